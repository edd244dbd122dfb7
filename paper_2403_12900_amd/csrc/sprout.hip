// C ABI of the decode library (include/sprout.h): argument validation, the
// host-side slot table, and the launch sequences of a decode step and of a
// prefill chunk.
//
// A decode step (one token row per active request) enqueues on the model's
// stream:
//   k_embed                      token rows -> fp32 residual x, QKV input (three parts)
//   per layer:
//     k_stream_gemm_qkv<EpiQKV>  RMSNorm . Wqkv, RoPE, q out, k/v appended to the paged cache
//     k_attn_decode (+merge)     softmax(q K^T / sqrt(hd)) V over the row's cached positions
//     k_stream_gemm<EpiResid>    x += o Wo^T
//     k_stream_gemm<EpiSwiGLU>   h = SiLU(RMSNorm(x) W1^T) * (RMSNorm(x) W3^T)
//     k_stream_gemm<EpiResid>    x += h W2^T (and the next QKV input)
//   k_stream_gemm<EpiLogits>     RMSNorm(x) Wlm^T, per-tile greedy candidates
//   k_argmax_final               tok[slot] = lowest index of the row maximum
// A prefill chunk (up to 4096 prompt rows of one or more requests) runs the
// same layer stack on tiled, compute-bound kernels:
//   k_embed_rows; per layer k_row_rscale, k_tile_gemm<EpiQKVRows> (query
//   tiles, then key and value tiles),
//   k_attn_prefill (causal, 16 queries per MFMA), k_tile_gemm<EpiResidRows>,
//   k_row_rscale, k_tile_gemm<EpiSwiGLURows>, k_tile_gemm<EpiResidRows>;
//   then k_gather_rows of the rows that end a prompt, and the decode LM head.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <type_traits>
#include <vector>

#include "attn_kernels.h"
#include "gemm_kernels.h"
#include "host_state.h"
#include "prefill_kernels.h"
#include "step_kernels.h"
#include "wgen_kernels.h"

using namespace sprk;

static_assert(spr::kPrefillRows == sprk::kPrefillRows, "prefill chunk size");
static_assert(spr::kMaxRows == sprk::kRows, "decode pass size");

// Scratch of spr_decode_step_static_scratch: a fixed array in device memory,
// one per device that loads the library, held until the process ends.
// Regions: split partials (of attention, or of the projections' split-K
// slices), arrival counters, LM-head greedy candidates.  Host code never passes the array's name to a kernel (on the
// host it is only a stand-in symbol): it resolves the array's device address
// once per device at init (static_scratch_address) and passes that.
constexpr size_t kStaticPartBytes = size_t{16} << 20;
constexpr size_t kStaticCntBytes = size_t{64} << 10;
constexpr size_t kStaticAmaxBytes = (size_t{8} << 20) - kStaticCntBytes;
constexpr size_t kStaticScratchBytes = kStaticPartBytes + kStaticCntBytes + kStaticAmaxBytes;  // 24 MiB
__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

struct spr_model {
  spr::Dims d{};
  spr::Layout lay{};
  char* ws = nullptr;
  hipStream_t st = nullptr;
  spr::SlotTable tab;
  std::vector<int32_t> bt_row;
  // A failure that leaves the model unusable (a HIP error, or a failed device
  // check of an earlier step): every later call returns it.
  spr_status sticky = SPR_OK;
  std::string sticky_msg;
  uint64_t seed = 0;
  // Decode attention work-groups resident at once (CUs x occupancy).
  int attn_slots = 1024;
  // Device-side error flag in mapped pinned host memory (host and device
  // views): kernels set a bit when a step met an input they cannot honour (a
  // token id outside the vocabulary, a logits row with no finite maximum);
  // the next call on the model reports it.
  int* err_host = nullptr;
  int* err_dev = nullptr;
  // Device address of this device's static scratch array (see `scratch`).
  char* static_scratch = nullptr;
  ~spr_model() {
    if (err_host != nullptr) (void)hipHostFree(err_host);
  }
};

namespace {

thread_local std::string g_err;

spr_status fail(spr_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

spr_status hip_fail(spr_model* m, const char* what, hipError_t e) {
  const std::string msg = std::string(what) + ": " + hipGetErrorString(e);
  if (m) {
    m->sticky = SPR_ERR_HIP;
    m->sticky_msg = "an earlier HIP error left the model unusable; release it (" + msg + ")";
  }
  return fail(SPR_ERR_HIP, msg);
}

#define SPR_HIP(m, expr)                               \
  do {                                                 \
    hipError_t e_ = (expr);                            \
    if (e_ != hipSuccess) return hip_fail(m, #expr, e_); \
  } while (0)

#define SPR_LAUNCHED(m, what)                          \
  do {                                                 \
    hipError_t e_ = hipGetLastError();                 \
    if (e_ != hipSuccess) return hip_fail(m, what, e_); \
  } while (0)

// Device address of `scratch` on each device, resolved once per device with
// that device current.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_addr[kMaxDevices] = {};

hipError_t static_scratch_address(int dev, char** out) {
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_addr[dev] == nullptr) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_addr[dev] = static_cast<char*>(p);
  }
  *out = g_scratch_addr[dev];
  return hipSuccess;
}

uint64_t stream_key(uint64_t seed, int tensor, int layer) {
  return sm_output(seed, 1u + 256u * static_cast<uint64_t>(tensor) + static_cast<uint64_t>(layer));
}

int ceil_div(int a, int b) { return (a + b - 1) / b; }

unsigned grid1(int64_t threads) { return static_cast<unsigned>((threads + 255) / 256); }

MatSpec mat_spec(const spr::Dims& d, int kind, int layer, uint64_t seed) {
  MatSpec s{};
  s.kind = kind;
  s.H = d.H;
  s.Hkv = d.Hkv;
  s.hd = d.hd;
  s.f = d.f;
  s.d = d.d;
  s.V = d.V;
  switch (kind) {
    case MK_QKV:
      s.NT = d.nt_qkv; s.KB = d.kb_d; s.K = d.d;
      s.key[0] = stream_key(seed, 1, layer);
      s.key[1] = stream_key(seed, 2, layer);
      s.key[2] = stream_key(seed, 3, layer);
      break;
    case MK_O:
      s.NT = d.nt_o; s.KB = d.kb_o; s.K = d.o_in;
      s.key[0] = stream_key(seed, 4, layer);
      break;
    case MK_W13:
      s.NT = d.nt_13; s.KB = d.kb_d; s.K = d.d;
      s.key[0] = stream_key(seed, 5, layer);
      s.key[1] = stream_key(seed, 6, layer);
      break;
    case MK_W2:
      s.NT = d.nt_2; s.KB = d.kb_f; s.K = d.f;
      s.key[0] = stream_key(seed, 7, layer);
      break;
    default:
      s.NT = d.nt_lm; s.KB = d.kb_d; s.K = d.d;
      s.key[0] = stream_key(seed, 8, 0);
  }
  return s;
}

struct Ptrs {
  char* ws;
  const spr::Layout* l;
  char* wqkv(int layer) const { return ws + l->off_wqkv + l->wqkv * layer; }
  char* wo(int layer) const { return ws + l->off_wo + l->wo * layer; }
  char* w13(int layer) const { return ws + l->off_w13 + l->w13 * layer; }
  char* w2(int layer) const { return ws + l->off_w2 + l->w2 * layer; }
  char* wlm() const { return ws + l->off_wlm; }
  char* emb() const { return ws + l->off_emb; }
  char* kc(int layer) const { return ws + l->off_kc + l->kv_layer_stride * layer; }
  char* vc(int layer) const { return ws + l->off_vc + l->kv_layer_stride * layer; }
  int32_t* bt() const { return reinterpret_cast<int32_t*>(ws + l->off_bt); }
  float* x() const { return reinterpret_cast<float*>(ws + l->off_x); }
  char* act(int i) const { return ws + (i == 0 ? l->off_act0 : l->off_act1); }
  float* q() const { return reinterpret_cast<float*>(ws + l->off_q); }
  float* part() const { return reinterpret_cast<float*>(ws + l->off_part); }
  int32_t* cnt() const { return reinterpret_cast<int32_t*>(ws + l->off_cnt); }
  float2* amax() const { return reinterpret_cast<float2*>(ws + l->off_amax); }
  float2* rope() const { return reinterpret_cast<float2*>(ws + l->off_rope); }
  PrefillRow* prow() const { return reinterpret_cast<PrefillRow*>(ws + l->off_prow); }
  PrefillTile* ptile() const { return reinterpret_cast<PrefillTile*>(ws + l->off_ptile); }
  float* rs() const { return reinterpret_cast<float*>(ws + l->off_rs); }
};

// Per-pass scratch of a decode forward: attention split partials (at most
// max_splits splits), split arrival counters (zero between launches) and the
// LM head's per-tile greedy candidates.  Either regions of the model's
// workspace or of the static scratch array (spr_decode_step_static_scratch).
struct DecodeScratch {
  float* part;
  int32_t* cnt;
  float2* amax;
  int max_splits;
  size_t part_floats;  // capacity of part
  int n_cnt;           // capacity of cnt
};

DecodeScratch workspace_scratch(const spr_model* m) {
  Ptrs p{m->ws, &m->lay};
  return DecodeScratch{p.part(), p.cnt(), p.amax(), spr::kMaxSplits, m->lay.part_floats, m->lay.n_cnt};
}

// Room for split-K partials and arrival counters (see SplitK): the regions of
// the attention split partials and counters, which hold what any pass's
// split-K launches need (spr::split_need) and which every launch that uses
// them leaves zero.
struct SplitRoom {
  float* part = nullptr;  // null: no split-K
  int32_t* cnt = nullptr;
  size_t part_floats = 0;
  int n_cnt = 0;
};

SplitRoom split_room(const DecodeScratch& sc) { return SplitRoom{sc.part, sc.cnt, sc.part_floats, sc.n_cnt}; }

template <class P>
spr_status init_weights(spr_model* m) {
  const spr::Dims& d = m->d;
  Ptrs p{m->ws, &m->lay};
  auto tiled = [&](char* dst, int kind, int layer) -> spr_status {
    const MatSpec s = mat_spec(d, kind, layer, m->seed);
    const int64_t threads = static_cast<int64_t>(s.NT) * s.KB * 64;
    k_init_tiled<P><<<grid1(threads), 256, 0, m->st>>>(reinterpret_cast<uint4*>(dst), s);
    SPR_LAUNCHED(m, "k_init_tiled");
    return SPR_OK;
  };
  spr_status st;
  for (int l = 0; l < d.L; ++l) {
    if ((st = tiled(p.wqkv(l), MK_QKV, l)) != SPR_OK) return st;
    if ((st = tiled(p.wo(l), MK_O, l)) != SPR_OK) return st;
    if ((st = tiled(p.w13(l), MK_W13, l)) != SPR_OK) return st;
    if ((st = tiled(p.w2(l), MK_W2, l)) != SPR_OK) return st;
  }
  if ((st = tiled(p.wlm(), MK_LM, 0)) != SPR_OK) return st;
  const int64_t ne = static_cast<int64_t>(d.V) * d.d;
  k_init_rowmajor<P><<<grid1(ne), 256, 0, m->st>>>(reinterpret_cast<typename P::elem*>(p.emb()), ne,
                                                    stream_key(m->seed, 0, 0));
  SPR_LAUNCHED(m, "k_init_rowmajor");
  return SPR_OK;
}

// Activation format of the QKV projection's input: all 24 bits of the fp32
// residual for bf16 models (three parts), the plain format otherwise.
template <class P>
using QKVIn = std::conditional_t<std::is_same_v<P, BF16>, BF16x3, P>;

// Rows of one forward pass.
struct RowSet {
  int n = 0;
  int slot[kRows];
  int pos[kRows];
  int out_row[kRows];
  int tok[kRows];
  int hist_idx[kRows];  // token-history index of the row's token, -1 = none
};

// Whether an epilogue is a residual update (O and down).
template <class E>
struct IsResid : std::false_type {};
template <class F>
struct IsResid<EpiResid<F>> : std::true_type {};

// Split-K pays (see SplitK) once a work-group's activation range holds at
// least this many K-block parts per 16-row tile (at two parts, 384 KiB of
// activations per work-group at 16 rows): measured on the 7B projections at
// 12-32 rows, it is then 1-7 us faster per launch; below (O and gate/up at
// 9-16 rows) the slices' publication costs more than it saves.
constexpr int kSplitMinParts = 384;

// Split-K launch (see SplitK) of S slices per group of RT tiles, WAVES waves
// per work-group; false (nothing launched) when the tiles do not divide into
// groups or the room is too small.
template <class P, int JT, int WAVES, int RT, int S, int U, class Epi>
bool launch_split(hipStream_t st, int NT, const uint4* w, const uint4* x, int KB, const Epi& epi,
                  const SplitRoom& room) {
  const int groups = NT / RT;
  if (room.part == nullptr || NT % RT != 0 || groups > room.n_cnt ||
      static_cast<size_t>(groups) * S * SplitKPairs<JT, RT, Epi::kNorm>::value * 128 > room.part_floats)
    return false;
  k_stream_gemm_split<P, JT, WAVES, Epi, RT, U, S><<<groups * S, WAVES * 64, 0, st>>>(
      w, x, KB, 16 * JT, epi.n_rows, epi, SplitK{room.part, room.cnt});
  return true;
}

// Launch shape of a projection, from sweeps over the 7B projection shapes on
// MI355X at 1..32 rows:
//   * at 9..32 rows, where a work-group's activation range holds at least
//     kSplitMinParts K-block parts per tile: split-K across work-groups (for
//     the 7B shapes down at 9..32 rows, O and gate/up at 17..32); never the
//     LM head;
//   * wide projections (>= 1024 16-row tiles: gate/up, LM head) at up to 32
//     rows: one-wave work-groups, each streaming two whole tiles over the
//     full K -- long contiguous streams and no cross-wave reduction;
//   * projections of 512..1023 tiles at 17..64 rows: four waves split K for
//     two tiles, so each activation fragment feeds two weight fragments;
//   * everything else: four waves split K for one tile.
// PK: packed rows (at most 8 rows, two activation parts per fragment).
template <class P, int JT, bool PK, class Epi>
void launch_gemm_shape(hipStream_t st, int NT, const uint4* w, const uint4* x, int KB, const Epi& epi,
                       const SplitRoom& room) {
  const int Rp = 16 * JT, n = epi.n_rows;
  constexpr int XF = StreamFrags<P, PK>::value;  // activation fragments per K-block and tile
  if constexpr (!PK && JT <= 2) {
    // Past 8 rows, with enough activation bytes per work-group: split-K.
    // Shapes from sweeps of the 7B projections at 12-32 rows.
    if (KB * JT * P::parts >= kSplitMinParts) {
      if constexpr (IsResid<Epi>::value) {
        // O and down: two tiles per group, four slices of two waves.
        if (launch_split<P, JT, 2, spr::kSplitO.rt, spr::kSplitO.s, 4>(st, NT, w, x, KB, epi, room)) return;
      } else if constexpr (std::is_same_v<Epi, EpiSwiGLU<P>>) {
        // gate/up: four tiles per group, two one-wave slices.
        if (launch_split<P, JT, 1, spr::kSplitGU.rt, spr::kSplitGU.s, 4>(st, NT, w, x, KB, epi, room)) return;
      }
    }
  }
  if constexpr (JT <= 2) {
    if (NT >= 1024 && NT % 2 == 0) {
      constexpr int U = XF == 3 ? (JT == 1 ? 4 : 2) : (JT == 1 ? 8 : 4);
      k_stream_gemm<P, JT, 1, Epi, 2, U, true, PK><<<NT / 2, 64, 0, st>>>(w, x, KB, Rp, n, epi);
      return;
    }
  }
  if constexpr (JT >= 2 && JT <= 4) {
    if (NT >= 512 && NT % 2 == 0) {
      k_stream_gemm<P, JT, 4, Epi, 2, StreamDepth<2 * JT * P::parts>::value, true><<<NT / 2, 256, 0, st>>>(
          w, x, KB, Rp, n, epi);
      return;
    }
  }
  k_stream_gemm<P, JT, 4, Epi, 1, StreamDepth<JT * XF>::value, true, PK><<<NT, 256, 0, st>>>(w, x, KB, Rp, n, epi);
}

// QKV of bf16 models (three-part input, see k_stream_gemm_qkv): four waves
// splitting K of one tile per work-group with packed rows (at most 8); at
// 9..32 rows split-K across work-groups; without room for its partials, two
// tiles per work-group (measured on the 7B shape at 16 rows: 1.2% less
// decode-step time than one).
template <int JT, bool PK, class Epi>
void launch_qkv_shape(hipStream_t st, int NT, const uint4* w, const uint4* x, int KB, const Epi& epi,
                      const SplitRoom& room) {
  const int Rp = 16 * JT, n = epi.n_rows;
  const int q_tiles = epi.H * epi.hd / 16;
  if constexpr (!PK && JT <= 2) {
    // Past 8 rows: split-K, four tiles per group, four slices of two waves
    // (9-16 rows) or one (17-32 rows); from sweeps of the 7B QKV projection.
    constexpr int RT = spr::kSplitQKV.rt, S = spr::kSplitQKV.s, WV = JT == 1 ? 2 : 1;
    const int groups = NT / RT;
    if (KB * JT * 3 >= kSplitMinParts && room.part != nullptr && NT % RT == 0 && q_tiles % RT == 0 &&
        groups <= room.n_cnt &&
        static_cast<size_t>(groups) * S * SplitKPairs<JT, RT, true>::value * 128 <= room.part_floats) {
      k_stream_gemm_qkv<JT, WV, Epi, RT, 4, 4, false, S>
          <<<groups * S, WV * 64, 0, st>>>(w, x, KB, Rp, n, epi, q_tiles, SplitK{room.part, room.cnt});
      return;
    }
  }
  if constexpr (!PK && JT <= 4) {
    if (NT % 2 == 0 && q_tiles % 2 == 0) {
      k_stream_gemm_qkv<JT, 4, Epi, 2, StreamDepth<2 * JT * 2>::value, StreamDepth<2 * JT * 3>::value, false>
          <<<NT / 2, 256, 0, st>>>(w, x, KB, Rp, n, epi, q_tiles);
      return;
    }
  }
  if constexpr (JT == 8) {  // (more rows than a decode pass holds) every tile takes all three parts
    k_stream_gemm<BF16x3, JT, 4, Epi, 1, StreamDepth<JT * 3>::value, true><<<NT, 256, 0, st>>>(w, x, KB, Rp, n, epi);
  } else {
    constexpr int X2 = StreamFrags<BF16, PK>::value, X3 = StreamFrags<BF16x3, PK>::value;
    k_stream_gemm_qkv<JT, 4, Epi, 1, StreamDepth<JT * X2>::value, StreamDepth<JT * X3>::value, PK>
        <<<NT, 256, 0, st>>>(w, x, KB, Rp, n, epi, q_tiles);
  }
}

template <class P, class Epi>
spr_status launch_gemm(spr_model* m, int NT, const char* W, const char* X, int KB, int JT, const Epi& epi,
                       const SplitRoom& room = {}) {
  const uint4* w = reinterpret_cast<const uint4*>(W);
  const uint4* x = reinterpret_cast<const uint4*>(X);
  if constexpr (P::parts == 3) {
    switch (JT) {
      case 1:
        if (epi.n_rows <= 8) {
          launch_qkv_shape<1, true>(m->st, NT, w, x, KB, epi, room);
        } else {
          launch_qkv_shape<1, false>(m->st, NT, w, x, KB, epi, room);
        }
        break;
      case 2: launch_qkv_shape<2, false>(m->st, NT, w, x, KB, epi, room); break;
      case 4: launch_qkv_shape<4, false>(m->st, NT, w, x, KB, epi, room); break;
      case 8: launch_qkv_shape<8, false>(m->st, NT, w, x, KB, epi, room); break;
      default:
        return fail(SPR_ERR_INVALID_ARG, "internal: unsupported row-tile count");
    }
    SPR_LAUNCHED(m, "k_stream_gemm_qkv");
    return SPR_OK;
  }
  switch (JT) {
    case 1:
      if constexpr (P::parts >= 2) {
        if (epi.n_rows <= 8) {
          launch_gemm_shape<P, 1, true>(m->st, NT, w, x, KB, epi, room);
          break;
        }
      }
      launch_gemm_shape<P, 1, false>(m->st, NT, w, x, KB, epi, room);
      break;
    case 2: launch_gemm_shape<P, 2, false>(m->st, NT, w, x, KB, epi, room); break;
    case 4: launch_gemm_shape<P, 4, false>(m->st, NT, w, x, KB, epi, room); break;
    case 8: launch_gemm_shape<P, 8, false>(m->st, NT, w, x, KB, epi, room); break;
    default:
      return fail(SPR_ERR_INVALID_ARG, "internal: unsupported row-tile count");
  }
  SPR_LAUNCHED(m, "k_stream_gemm");
  return SPR_OK;
}

template <class P, class KP, int HD>
spr_status launch_attention(spr_model* m, const AttnArgs& a) {
  k_attn_decode<KP, P, HD><<<dim3(a.Hkv, a.split_start[a.n_rows]), 256, 0, m->st>>>(a);
  SPR_LAUNCHED(m, "k_attn_decode");
  return SPR_OK;
}

// Attention arguments of one layer over rs (kv splits of bpw blocks per wave).
template <class P, class KP>
AttnArgs attention_args(spr_model* m, int l, const RowSet& rs, const RowSlotPos& sp, int Rp, int bpw, void* act,
                        const DecodeScratch& sc) {
  const spr::Dims& d = m->d;
  Ptrs p{m->ws, &m->lay};
  AttnArgs a{};
  a.q = p.q();
  a.kc = p.kc(l);
  a.vc = p.vc(l);
  a.bt = p.bt();
  a.act = act;
  a.part = sc.part;
  a.cnt = sc.cnt;
  a.n_rows = rs.n;
  a.H = d.H;
  a.Hkv = d.Hkv;
  a.G = d.G;
  a.mb = d.mb;
  a.bpw = bpw;
  a.Rp = Rp;
  a.qscale = static_cast<float>(1.4426950408889634 / std::sqrt(static_cast<double>(d.hd)));
  a.rows = sp;
  a.split_start[0] = 0;
  for (int r = 0; r < rs.n; ++r) a.split_start[r + 1] = a.split_start[r] + ceil_div((rs.pos[r] + 1 + 15) / 16, 4 * bpw);
  return a;
}

// Decode attention work-groups resident per CU (0 = unavailable).
template <class P, class KP>
int attn_blocks_per_cu(const spr::Dims& d) {
  int o = 0;
  const void* k = d.hd == 128 ? reinterpret_cast<const void*>(&k_attn_decode<KP, P, 128>)
                              : reinterpret_cast<const void*>(&k_attn_decode<KP, P, 64>);
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&o, k, 256, 0) != hipSuccess) o = 0;
  return o;
}

// One forward pass over rs (rows: slot, position, emitted logits row).
// tok_in != null: the inputs are tok_in[slot]; otherwise rs.tok.  Emitting
// rows write their greedy token to tok_out[slot].
template <class P, class KP>
spr_status forward(spr_model* m, const RowSet& rs, const int32_t* tok_in, int32_t* tok_out, float* logits,
                   int32_t* hist, const DecodeScratch& sc) {
  const spr::Dims& d = m->d;
  Ptrs p{m->ws, &m->lay};
  const int n = rs.n;
  const int JT = n <= 16 ? 1 : n <= 32 ? 2 : n <= 64 ? 4 : 8;
  const int Rp = 16 * JT;
  using E = typename P::elem;
  RowSlotPos sp;
  std::memcpy(sp.slot, rs.slot, sizeof(sp.slot));
  std::memcpy(sp.pos, rs.pos, sizeof(sp.pos));

  {
    EmbedArgs ea{};
    ea.emb = p.emb();
    ea.tok_dev = tok_in;
    ea.x = p.x();
    ea.act = p.act(0);
    ea.err = m->err_dev;
    ea.n_rows = n;
    ea.d = d.d;
    ea.V = d.V;
    ea.Rp = Rp;
    std::memcpy(ea.slot, rs.slot, sizeof(ea.slot));
    std::memcpy(ea.tok, rs.tok, sizeof(ea.tok));
    k_embed<QKVIn<P>><<<dim3(ceil_div(d.d / 4, 64), n), 64, 0, m->st>>>(ea);
    SPR_LAUNCHED(m, "k_embed");
  }

  // KV splits: a work-group covers 4 * bpw blocks of one (row, KV head), a
  // run of bpw blocks per wave.  bpw stays 1 until the pass has more blocks
  // than the resident waves (4 per work-group) take at once.  Rounding each
  // row up to whole splits can still leave more work-groups than stay
  // resident; then runs up to twice as long per wave that fit them into one
  // round are taken (measured on 7B, 12-28 rows of 400 positions: 3-15 us
  // less per layer), but not longer ones (a batch whose longest row would
  // need them: one long run then sets the time).  bpw grows further only
  // while the splits exceed the partial buffer.
  int total_blk = 0;
  for (int r = 0; r < n; ++r) total_blk += (rs.pos[r] + 1 + 15) / 16;
  int bpw = ceil_div(total_blk * d.Hkv, 4 * m->attn_slots);
  if (bpw < 1) bpw = 1;
  auto count_splits = [&](int w) {
    int t = 0;
    for (int r = 0; r < n; ++r) t += ceil_div((rs.pos[r] + 1 + 15) / 16, 4 * w);
    return t;
  };
  {
    int fit = bpw;
    while (count_splits(fit) * d.Hkv > m->attn_slots && count_splits(fit) > n && fit < 2 * bpw) ++fit;
    if (count_splits(fit) * d.Hkv <= m->attn_slots) bpw = fit;
  }
  while (count_splits(bpw) > sc.max_splits) ++bpw;
  // A row's splits are merged by its last arriving split, kMergeChunk
  // partials per round of loads: keep every row within one round (measured
  // on 7B at one row of 1024 positions: 17 splits 11.5 us, 9 splits 10.1 us).
  for (int r = 0; r < n; ++r)
    while (ceil_div((rs.pos[r] + 1 + 15) / 16, 4 * bpw) > kMergeChunk) ++bpw;

  const SplitRoom room = split_room(sc);
  spr_status st;
  for (int l = 0; l < d.L; ++l) {
    {
      EpiQKV<P, KP> e{};
      e.n_rows = n;
      e.H = d.H;
      e.Hkv = d.Hkv;
      e.hd = d.hd;
      e.mb = d.mb;
      e.dnorm = d.d;
      e.eps = d.eps;
      e.q = p.q();
      e.kc = reinterpret_cast<typename KP::elem*>(p.kc(l));
      e.vc = reinterpret_cast<typename KP::elem*>(p.vc(l));
      e.bt = p.bt();
      e.rope = p.rope();
      e.rows = sp;
      if ((st = launch_gemm<QKVIn<P>>(m, d.nt_qkv, p.wqkv(l), p.act(0), d.kb_d, JT, e, room)) != SPR_OK) return st;
    }
    {
      const AttnArgs a = attention_args<P, KP>(m, l, rs, sp, Rp, bpw, p.act(1), sc);
      st = d.hd == 128 ? launch_attention<P, KP, 128>(m, a) : launch_attention<P, KP, 64>(m, a);
      if (st != SPR_OK) return st;
    }
    {
      EpiResid<P> e{n, d.d, Rp, p.x(), reinterpret_cast<E*>(p.act(0))};
      if ((st = launch_gemm<P>(m, d.nt_o, p.wo(l), p.act(1), d.kb_o, JT, e, room)) != SPR_OK) return st;
    }
    {
      EpiSwiGLU<P> e{n, d.d, Rp, d.eps, reinterpret_cast<E*>(p.act(1))};
      if ((st = launch_gemm<P>(m, d.nt_13, p.w13(l), p.act(0), d.kb_d, JT, e, room)) != SPR_OK) return st;
    }
    if (l + 1 < d.L) {  // the new residual is the next layer's QKV input
      EpiResid<QKVIn<P>> e{n, d.d, Rp, p.x(), reinterpret_cast<E*>(p.act(0))};
      if ((st = launch_gemm<P>(m, d.nt_2, p.w2(l), p.act(1), d.kb_f, JT, e, room)) != SPR_OK) return st;
    } else {            // ... or the LM head's
      EpiResid<P> e{n, d.d, Rp, p.x(), reinterpret_cast<E*>(p.act(0))};
      if ((st = launch_gemm<P>(m, d.nt_2, p.w2(l), p.act(1), d.kb_f, JT, e, room)) != SPR_OK) return st;
    }
  }
  {
    EpiLogits<P> e{};
    e.n_rows = n;
    e.V = d.V;
    e.dnorm = d.d;
    e.eps = d.eps;
    e.logits = logits;
    e.part = sc.amax;
    std::memcpy(e.out_row, rs.out_row, sizeof(e.out_row));
    if ((st = launch_gemm<P>(m, d.nt_lm, p.wlm(), p.act(0), d.kb_d, JT, e)) != SPR_OK) return st;
  }
  {
    ArgmaxArgs a{};
    a.part = sc.amax;
    a.tok_dev = tok_out;
    a.n_tiles = d.nt_lm;
    a.err = m->err_dev;
    std::memcpy(a.slot, rs.slot, sizeof(a.slot));
    std::memcpy(a.out_row, rs.out_row, sizeof(a.out_row));
    std::memcpy(a.hist_idx, rs.hist_idx, sizeof(a.hist_idx));
    a.hist = hist;
    k_argmax_final<<<n, 256, 0, m->st>>>(a);
    SPR_LAUNCHED(m, "k_argmax_final");
  }
  return SPR_OK;
}

// Launches one projection of `layer` over n rows (see spr_time_projection).
template <class P>
spr_status launch_projection(spr_model* m, int projection, int layer, int n) {
  const spr::Dims& d = m->d;
  Ptrs p{m->ws, &m->lay};
  const SplitRoom room = split_room(workspace_scratch(m));
  const int JT = n <= 16 ? 1 : n <= 32 ? 2 : n <= 64 ? 4 : 8;
  const int Rp = 16 * JT;
  using E = typename P::elem;
  switch (projection) {
    case 1: {
      EpiResid<P> e{n, d.d, Rp, p.x(), reinterpret_cast<E*>(p.act(0))};
      return launch_gemm<P>(m, d.nt_o, p.wo(layer), p.act(1), d.kb_o, JT, e, room);
    }
    case 2: {
      EpiSwiGLU<P> e{n, d.d, Rp, d.eps, reinterpret_cast<E*>(p.act(1))};
      return launch_gemm<P>(m, d.nt_13, p.w13(layer), p.act(0), d.kb_d, JT, e, room);
    }
    case 3: {  // as in every layer but the last
      EpiResid<QKVIn<P>> e{n, d.d, Rp, p.x(), reinterpret_cast<E*>(p.act(0))};
      return launch_gemm<P>(m, d.nt_2, p.w2(layer), p.act(1), d.kb_f, JT, e, room);
    }
    default: {
      EpiLogits<P> e{};
      e.n_rows = n;
      e.V = d.V;
      e.dnorm = d.d;
      e.eps = d.eps;
      e.logits = nullptr;
      e.part = p.amax();
      for (int r = 0; r < kRows; ++r) e.out_row[r] = -1;
      return launch_gemm<P>(m, d.nt_lm, p.wlm(), p.act(0), d.kb_d, JT, e);
    }
  }
}

// One prefill chunk: C rows (rows[] on the device), n_tiles attention query
// tiles (ptile[] on the device), and the rows that end a prompt: emit_row[k]
// (chunk row) emits request emit_out[k]'s first token into tok[emit_slot[k]]
// and, when a history buffer is given, into hist[emit_hist[k]] (-1 = none).
struct PrefillChunk {
  int C = 0, n_tiles = 0, n_emit = 0;
  int emit_row[kRows], emit_out[kRows], emit_slot[kRows], emit_hist[kRows];
};

template <class P, class KP, int HD>
void launch_attn_prefill(spr_model* m, int layer, const PrefillChunk& ch, int Rp) {
  const spr::Dims& d = m->d;
  Ptrs p{m->ws, &m->lay};
  const float qscale = static_cast<float>(1.4426950408889634 / std::sqrt(static_cast<double>(d.hd)));
  k_attn_prefill<KP, P, HD><<<dim3(ch.n_tiles, d.H), 256, 0, m->st>>>(p.q(), p.kc(layer), p.vc(layer), p.bt(),
                                                                       p.ptile(), p.act(1), d.H, d.Hkv, d.mb, Rp,
                                                                       qscale);
}

// Tile shape of a prefill projection: 256 x 256 eight-wave work-groups when
// that gives at least one per CU (256; measured 3% faster on 7B-shape 4096-row
// chunks than requiring 512), else 128 x 128 when that gives at least 512,
// else 64 features x 128 rows, else 64 x 64.
// Three-part activations (QKV) take 256 features x 128 rows instead of 256 x
// 256: the larger tile's three LDS stages would need 192 KiB.
// LP: parts per K-block of the activation record X (P::parts used).
template <class P, class Epi, int LP = P::parts>
void launch_tile_gemm(hipStream_t st, const char* W, const char* X, int NT, int KB, int Rp, const Epi& e) {
  const uint4* w = reinterpret_cast<const uint4*>(W);
  const uint4* x = reinterpret_cast<const uint4*>(X);
  const int mt = Rp / 128;
  if constexpr (P::parts == 3) {
    if (ceil_div(NT, 16) * mt >= 256) {
      k_tile_gemm<P, 16, 8, Epi, 8, LP><<<dim3(ceil_div(NT, 16), mt), 512, 0, st>>>(w, x, NT, KB, Rp, e);
      return;
    }
  } else {
    if (ceil_div(NT, 16) * ceil_div(Rp, 256) >= 256) {
      k_tile_gemm<P, 16, 16, Epi, 8, LP><<<dim3(ceil_div(NT, 16), ceil_div(Rp, 256)), 512, 0, st>>>(w, x, NT, KB, Rp,
                                                                                                    e);
      return;
    }
  }
  if (ceil_div(NT, 8) * mt >= 512) {
    k_tile_gemm<P, 8, 8, Epi, 4, LP><<<dim3(ceil_div(NT, 8), mt), 256, 0, st>>>(w, x, NT, KB, Rp, e);
  } else if (ceil_div(NT, 4) * mt >= 512) {
    k_tile_gemm<P, 4, 8, Epi, 4, LP><<<dim3(ceil_div(NT, 4), mt), 256, 0, st>>>(w, x, NT, KB, Rp, e);
  } else {
    k_tile_gemm<P, 4, 4, Epi, 4, LP><<<dim3(ceil_div(NT, 4), Rp / 64), 256, 0, st>>>(w, x, NT, KB, Rp, e);
  }
}

template <class P, class KP>
spr_status prefill_pass(spr_model* m, const PrefillChunk& ch, int32_t* tok, float* logits, int32_t* hist) {
  const spr::Dims& d = m->d;
  Ptrs p{m->ws, &m->lay};
  using E = typename P::elem;
  const int C = ch.C;
  const int Rp = 128 * ceil_div(C, 128);
  const dim3 grid_d(ceil_div(d.d / 4, 64), C);
  k_embed_rows<QKVIn<P>><<<grid_d, 64, 0, m->st>>>(reinterpret_cast<const E*>(p.emb()), p.prow(), p.x(),
                                                   reinterpret_cast<E*>(p.act(0)), d.d, d.V, Rp);
  SPR_LAUNCHED(m, "k_embed_rows");
  for (int l = 0; l < d.L; ++l) {
    k_row_rscale<<<ceil_div(C, 4), 256, 0, m->st>>>(p.x(), p.rs(), C, d.d, d.eps);
    {
      EpiQKVRows<P, KP> e{};
      e.M = C;
      e.H = d.H;
      e.Hkv = d.Hkv;
      e.hd = d.hd;
      e.mb = d.mb;
      e.q = p.q();
      e.kc = reinterpret_cast<typename KP::elem*>(p.kc(l));
      e.vc = reinterpret_cast<typename KP::elem*>(p.vc(l));
      e.bt = p.bt();
      e.rope = p.rope();
      e.rows = p.prow();
      e.rs = p.rs();
      e.nt_base = 0;
      if constexpr (QKVIn<P>::parts == 3) {
        // Query tiles take hi + mid of the three-part record (and the larger
        // two-part tiles), key and value tiles all three parts.
        const int q_tiles = d.H * d.hd / 16;
        launch_tile_gemm<P, EpiQKVRows<P, KP>, 3>(m->st, p.wqkv(l), p.act(0), q_tiles, d.kb_d, Rp, e);
        e.nt_base = q_tiles;
        const char* wkv = p.wqkv(l) + static_cast<size_t>(q_tiles) * d.kb_d * 64 * sizeof(uint4);
        launch_tile_gemm<QKVIn<P>>(m->st, wkv, p.act(0), d.nt_qkv - q_tiles, d.kb_d, Rp, e);
      } else {
        launch_tile_gemm<QKVIn<P>>(m->st, p.wqkv(l), p.act(0), d.nt_qkv, d.kb_d, Rp, e);
      }
    }
    if (d.hd == 128) {
      launch_attn_prefill<P, KP, 128>(m, l, ch, Rp);
    } else {
      launch_attn_prefill<P, KP, 64>(m, l, ch, Rp);
    }
    {
      EpiResidRows<P> e{C, d.d, Rp, p.x(), reinterpret_cast<E*>(p.act(0))};
      launch_tile_gemm<P>(m->st, p.wo(l), p.act(1), d.nt_o, d.kb_o, Rp, e);
    }
    k_row_rscale<<<ceil_div(C, 4), 256, 0, m->st>>>(p.x(), p.rs(), C, d.d, d.eps);
    {
      EpiSwiGLURows<P> e{C, Rp, p.rs(), reinterpret_cast<E*>(p.act(1))};
      launch_tile_gemm<P>(m->st, p.w13(l), p.act(0), d.nt_13, d.kb_d, Rp, e);
    }
    {  // the new residual is the next layer's QKV input (the prompt's last rows reach the LM head from x)
      EpiResidRows<QKVIn<P>> e{C, d.d, Rp, p.x(), reinterpret_cast<E*>(p.act(0))};
      launch_tile_gemm<P>(m->st, p.w2(l), p.act(1), d.nt_2, d.kb_f, Rp, e);
    }
    SPR_LAUNCHED(m, "prefill layer");
  }
  if (ch.n_emit == 0) return SPR_OK;
  const int n = ch.n_emit;
  const int JT = n <= 16 ? 1 : n <= 32 ? 2 : n <= 64 ? 4 : 8;
  {
    GatherArgs g{};
    g.x = p.x();
    g.act = p.act(1);
    g.d = d.d;
    g.Rp = 16 * JT;
    g.n = n;
    for (int k = 0; k < n; ++k) g.src[k] = ch.emit_row[k];
    k_gather_rows<P><<<dim3(ceil_div(d.d / 4, 64), n), 64, 0, m->st>>>(g);
    SPR_LAUNCHED(m, "k_gather_rows");
  }
  spr_status st;
  {
    EpiLogits<P> e{};
    e.n_rows = n;
    e.V = d.V;
    e.dnorm = d.d;
    e.eps = d.eps;
    e.logits = logits;
    e.part = p.amax();
    for (int k = 0; k < kRows; ++k) e.out_row[k] = k < n ? ch.emit_out[k] : -1;
    if ((st = launch_gemm<P>(m, d.nt_lm, p.wlm(), p.act(1), d.kb_d, JT, e)) != SPR_OK) return st;
  }
  {
    ArgmaxArgs a{};
    a.part = p.amax();
    a.tok_dev = tok;
    a.n_tiles = d.nt_lm;
    a.err = m->err_dev;
    for (int k = 0; k < kRows; ++k) {
      a.slot[k] = k < n ? ch.emit_slot[k] : 0;
      a.out_row[k] = k < n ? ch.emit_out[k] : -1;
      a.hist_idx[k] = k < n ? ch.emit_hist[k] : -1;
    }
    a.hist = hist;
    k_argmax_final<<<n, 256, 0, m->st>>>(a);
    SPR_LAUNCHED(m, "k_argmax_final");
  }
  return SPR_OK;
}

spr_status prefill_any(spr_model* m, const PrefillChunk& ch, int32_t* tok, float* logits, int32_t* hist) {
  if (m->d.dtype == SPR_F32) return prefill_pass<F32, F32>(m, ch, tok, logits, hist);
  return m->d.kv_dtype == SPR_BF16 ? prefill_pass<BF16, BF16>(m, ch, tok, logits, hist)
                                   : prefill_pass<BF16, F32>(m, ch, tok, logits, hist);
}

spr_status forward_any(spr_model* m, const RowSet& rs, const int32_t* tok_in, int32_t* tok_out, float* logits,
                       int32_t* hist, const DecodeScratch& sc) {
  if (m->d.dtype == SPR_F32) return forward<F32, F32>(m, rs, tok_in, tok_out, logits, hist, sc);
  return m->d.kv_dtype == SPR_BF16 ? forward<BF16, BF16>(m, rs, tok_in, tok_out, logits, hist, sc)
                                   : forward<BF16, F32>(m, rs, tok_in, tok_out, logits, hist, sc);
}

// Device check bits (EmbedArgs / ArgmaxArgs `err`), reported by the next call.
std::string device_check_message(int bits) {
  std::string s = "a device check failed on an earlier call:";
  if (bits & kErrTokenRange) s += " a token id outside [0, vocab) was fed (it was read as a clamped id);";
  if (bits & kErrLogits) s += " a logits row had no finite maximum (its token was set to 0);";
  return s + " the model's state is unreliable; release it";
}

spr_status check_model(spr_model* m) {
  if (m == nullptr) return fail(SPR_ERR_INVALID_ARG, "model is null");
  if (m->sticky == SPR_OK && m->err_host != nullptr) {
    const int bits = *reinterpret_cast<volatile int*>(m->err_host);
    if (bits != 0) {
      m->sticky = SPR_ERR_DEVICE_CHECK;
      m->sticky_msg = device_check_message(bits);
    }
  }
  if (m->sticky != SPR_OK) return fail(m->sticky, m->sticky_msg);
  return SPR_OK;
}

// Device part of a prefill whose slots the table has already reserved:
// uploads the slots' block-table rows, then runs the prompts (request i:
// prompts[i][0 .. seq_lens[i])) in chunks of up to kPrefillRows rows in
// request order; a prompt may span chunks (its later rows attend to the
// positions an earlier chunk cached).  Request i's first token goes to
// tok[slots[i]], its logits to row i of `logits` (if non-null), and to
// hist[hist_idx[i]] (if hist is non-null and hist_idx[i] >= 0).  The host
// tables stay alive until the final synchronize.
spr_status prefill_device(spr_model* m, int n, const int32_t* slots, const int32_t* const* prompts,
                          const int32_t* seq_lens, int32_t* tok, float* logits, int32_t* hist,
                          const int32_t* hist_idx) {
  Ptrs p{m->ws, &m->lay};
  spr_status st;
  std::vector<int32_t> rows(static_cast<size_t>(n) * m->d.mb);
  for (int i = 0; i < n; ++i) m->tab.block_row(slots[i], rows.data() + static_cast<size_t>(i) * m->d.mb);
  for (int i = 0; i < n; ++i)
    SPR_HIP(m, hipMemcpyAsync(p.bt() + static_cast<size_t>(slots[i]) * m->d.mb,
                              rows.data() + static_cast<size_t>(i) * m->d.mb, m->d.mb * sizeof(int32_t),
                              hipMemcpyHostToDevice, m->st));
  std::vector<std::vector<PrefillRow>> row_tabs;
  std::vector<std::vector<PrefillTile>> tile_tabs;
  PrefillChunk ch;
  std::vector<PrefillRow> chunk_rows;
  std::vector<PrefillTile> tiles;
  auto flush = [&]() -> spr_status {
    if (chunk_rows.empty()) return SPR_OK;
    ch.C = static_cast<int>(chunk_rows.size());
    ch.n_tiles = static_cast<int>(tiles.size());
    if (ch.n_tiles > spr::kPrefillTiles) return fail(SPR_ERR_INVALID_ARG, "internal: prefill tile table overflow");
    row_tabs.push_back(std::move(chunk_rows));
    tile_tabs.push_back(std::move(tiles));
    chunk_rows = {};
    tiles = {};
    SPR_HIP(m, hipMemcpyAsync(p.prow(), row_tabs.back().data(), row_tabs.back().size() * sizeof(PrefillRow),
                              hipMemcpyHostToDevice, m->st));
    SPR_HIP(m, hipMemcpyAsync(p.ptile(), tile_tabs.back().data(), tile_tabs.back().size() * sizeof(PrefillTile),
                              hipMemcpyHostToDevice, m->st));
    spr_status s2 = prefill_any(m, ch, tok, logits, hist);
    ch = PrefillChunk{};
    return s2;
  };
  for (int i = 0; i < n; ++i) {
    int pos = 0;
    while (pos < seq_lens[i]) {
      if (static_cast<int>(chunk_rows.size()) == spr::kPrefillRows) {
        if ((st = flush()) != SPR_OK) return st;
      }
      // The next segment of request i that fits this chunk, in query tiles of 64.
      const int seg = std::min(seq_lens[i] - pos, spr::kPrefillRows - static_cast<int>(chunk_rows.size()));
      const int row0 = static_cast<int>(chunk_rows.size());
      for (int k = 0; k < seg; ++k) chunk_rows.push_back(PrefillRow{slots[i], pos + k, prompts[i][pos + k], 0});
      for (int k = 0; k < seg; k += 64) tiles.push_back(PrefillTile{slots[i], row0 + k, std::min(64, seg - k), pos + k});
      pos += seg;
      if (pos == seq_lens[i]) {
        ch.emit_row[ch.n_emit] = row0 + seg - 1;
        ch.emit_out[ch.n_emit] = i;
        ch.emit_slot[ch.n_emit] = slots[i];
        ch.emit_hist[ch.n_emit] = hist != nullptr && hist_idx != nullptr ? hist_idx[i] : -1;
        ++ch.n_emit;
      }
    }
  }
  if ((st = flush()) != SPR_OK) return st;
  SPR_HIP(m, hipStreamSynchronize(m->st));
  return SPR_OK;
}

// Device side of spr_serve: runs the scheduler's prefill and decode calls on
// the kernels above; request r's token k lands in out[off[r] + k].  With an
// EOS id, each call's tokens (the slot-indexed token buffer) are copied
// asynchronously into pinned host memory, and end_iteration reads the
// previous iteration's copies, so the host waits only for work that finished
// while the current iteration runs.  An event closes every iteration; each
// iteration's device time is later shared equally by the requests it served.
struct GpuServe : spr::ServeDevice {
  spr_model* m = nullptr;
  const spr::ServeRequest* reqs = nullptr;
  const int64_t* off = nullptr;
  int32_t* tok = nullptr;
  int32_t* out = nullptr;
  int eos_id = -1;
  int32_t* pin = nullptr;             // pinned [2 parities][2 phases][max_slots]
  hipEvent_t snap[2] = {nullptr, nullptr};
  struct Row {
    int slot, req, idx;
  };
  std::vector<Row> rows[2][2];        // [parity][0 prefill, 1 decode]
  bool pending = false;               // the previous iteration has copies to read
  int par = 0;
  std::vector<hipEvent_t> ev_iter;    // end of each iteration
  std::vector<std::vector<int>> served;  // requests each iteration served
  std::vector<int> cur;

  spr_status snapshot(int phase) {
    SPR_HIP(m, hipMemcpyAsync(pin + (par * 2 + phase) * m->d.S, tok, m->d.S * sizeof(int32_t),
                              hipMemcpyDeviceToHost, m->st));
    return SPR_OK;
  }

  spr_status prefill(int n, const int32_t* slots, const int32_t* req) override {
    std::vector<const int32_t*> prompts(n);
    std::vector<int32_t> lens(n), hidx(n);
    for (int i = 0; i < n; ++i) {
      prompts[i] = reqs[req[i]].tokens;
      lens[i] = reqs[req[i]].n_tokens;
      hidx[i] = static_cast<int32_t>(off[req[i]]);
      cur.push_back(req[i]);
    }
    spr_status st = prefill_device(m, n, slots, prompts.data(), lens.data(), tok, nullptr, out, hidx.data());
    if (st != SPR_OK || eos_id < 0) return st;
    for (int i = 0; i < n; ++i) rows[par][0].push_back(Row{slots[i], req[i], 0});
    return snapshot(0);
  }

  spr_status decode(int n, const int32_t* slots, const int32_t* lens, const int32_t* req,
                    const int32_t* produced) override {
    RowSet rs;
    rs.n = n;
    for (int r = 0; r < kRows; ++r) {
      const bool v = r < n;
      rs.slot[r] = v ? slots[r] : 0;
      rs.pos[r] = v ? lens[r] : 0;
      rs.out_row[r] = v ? r : -1;
      rs.tok[r] = 0;
      rs.hist_idx[r] = v ? static_cast<int>(off[req[r]] + produced[r]) : -1;
    }
    for (int i = 0; i < n; ++i) cur.push_back(req[i]);
    spr_status st = forward_any(m, rs, tok, tok, nullptr, out, workspace_scratch(m));
    if (st != SPR_OK || eos_id < 0) return st;
    for (int i = 0; i < n; ++i) rows[par][1].push_back(Row{slots[i], req[i], produced[i]});
    return snapshot(1);
  }

  // Appends the EOS hits among the copies of parity q (already complete).
  void scan(int q, std::vector<std::pair<int, int>>* eos) {
    for (int ph = 0; ph < 2; ++ph) {
      for (const Row& r : rows[q][ph])
        if (pin[(q * 2 + ph) * m->d.S + r.slot] == eos_id) eos->emplace_back(r.req, r.idx);
      rows[q][ph].clear();
    }
  }

  spr_status end_iteration(bool final, std::vector<std::pair<int, int>>* eos) override {
    hipEvent_t e = nullptr;
    SPR_HIP(m, hipEventCreate(&e));
    ev_iter.push_back(e);
    served.push_back(std::move(cur));
    cur.clear();
    SPR_HIP(m, hipEventRecord(e, m->st));
    if (eos_id < 0) return SPR_OK;
    SPR_HIP(m, hipEventRecord(snap[par], m->st));
    if (pending) {
      SPR_HIP(m, hipEventSynchronize(snap[par ^ 1]));
      scan(par ^ 1, eos);
    }
    if (final) {
      SPR_HIP(m, hipEventSynchronize(snap[par]));
      scan(par, eos);
      pending = false;
      return SPR_OK;
    }
    pending = true;
    par ^= 1;
    return SPR_OK;
  }
};


}  // namespace

extern "C" {

size_t spr_workspace_bytes(const spr_config* cfg) {
  if (cfg == nullptr) return 0;
  spr::Dims d;
  std::string err;
  if (!spr::derive(*cfg, &d, &err)) return 0;
  return spr::layout(d).total;
}

spr_status spr_init(const spr_config* cfg, uint64_t seed, void* dev_ws, size_t ws_bytes, void* hip_stream,
                    spr_model** out) {
  g_err.clear();
  if (cfg == nullptr || out == nullptr) return fail(SPR_ERR_INVALID_ARG, "init: cfg and out must not be null");
  *out = nullptr;
  spr::Dims d;
  std::string err;
  if (!spr::derive(*cfg, &d, &err)) return fail(SPR_ERR_INVALID_ARG, "init: " + err);
  const spr::Layout lay = spr::layout(d);
  if (dev_ws == nullptr || (reinterpret_cast<uintptr_t>(dev_ws) & 255) != 0)
    return fail(SPR_ERR_WORKSPACE, "init: workspace must be a non-null, 256-byte aligned device pointer");
  if (ws_bytes < lay.total)
    return fail(SPR_ERR_WORKSPACE, "init: workspace has " + std::to_string(ws_bytes) + " bytes, " +
                                       std::to_string(lay.total) + " needed");
  spr_model* m = new spr_model();
  m->d = d;
  m->lay = lay;
  m->ws = static_cast<char*>(dev_ws);
  m->st = static_cast<hipStream_t>(hip_stream);
  m->seed = seed;
  m->tab.init(d);
  m->bt_row.assign(d.mb, 0);
  spr_status st = d.dtype == SPR_BF16 ? init_weights<BF16>(m) : init_weights<F32>(m);
  if (st != SPR_OK) {
    delete m;
    return st;
  }
  Ptrs p{m->ws, &m->lay};
  // RoPE table: angle = pos * base^(-2i/hd), evaluated in double, stored as fp32 (cos, sin).
  std::vector<float> rope(static_cast<size_t>(d.max_ctx) * d.hd);
  for (int pos = 0; pos < d.max_ctx; ++pos)
    for (int i = 0; i < d.hd / 2; ++i) {
      const double theta = std::pow(static_cast<double>(d.rope_base), -2.0 * i / d.hd);
      const double ang = pos * theta;
      rope[(static_cast<size_t>(pos) * (d.hd / 2) + i) * 2] = static_cast<float>(std::cos(ang));
      rope[(static_cast<size_t>(pos) * (d.hd / 2) + i) * 2 + 1] = static_cast<float>(std::sin(ang));
    }
  hipError_t e = hipMemcpyAsync(p.rope(), rope.data(), rope.size() * sizeof(float), hipMemcpyHostToDevice, m->st);
  if (e == hipSuccess) e = hipMemsetAsync(p.bt(), 0, static_cast<size_t>(d.S) * d.mb * sizeof(int32_t), m->st);
  if (e == hipSuccess) e = hipMemsetAsync(p.act(0), 0, lay.act_bytes, m->st);
  if (e == hipSuccess) e = hipMemsetAsync(p.cnt(), 0, static_cast<size_t>(spr::kMaxRows) * d.Hkv * sizeof(int32_t), m->st);
  if (e == hipSuccess) e = hipMemsetAsync(p.act(1), 0, lay.act_bytes, m->st);
  if (e == hipSuccess) e = hipMemsetAsync(p.x(), 0, static_cast<size_t>(spr::kPrefillRows) * d.d * sizeof(float), m->st);
  // The device error flag: mapped pinned host memory, written by kernels only
  // when a check fails and read by the host at the start of every call.
  if (e == hipSuccess) e = hipHostMalloc(reinterpret_cast<void**>(&m->err_host), sizeof(int), hipHostMallocMapped);
  if (e == hipSuccess) {
    *m->err_host = 0;
    e = hipHostGetDevicePointer(reinterpret_cast<void**>(&m->err_dev), m->err_host, 0);
  }
  // Decode attention sizes its KV splits by the work-groups resident at once.
  if (e == hipSuccess) {
    int dev = 0, ncu = 0;
    e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess) e = static_scratch_address(dev, &m->static_scratch);
    const int attn_per_cu = d.dtype == SPR_F32 ? attn_blocks_per_cu<F32, F32>(d)
                            : d.kv_dtype == SPR_BF16 ? attn_blocks_per_cu<BF16, BF16>(d)
                                                     : attn_blocks_per_cu<BF16, F32>(d);
    if (e == hipSuccess && attn_per_cu >= 1) m->attn_slots = attn_per_cu * ncu;
  }
  if (e == hipSuccess) e = hipStreamSynchronize(m->st);
  if (e != hipSuccess) {
    hip_fail(nullptr, "init", e);
    delete m;
    return SPR_ERR_HIP;
  }
  *out = m;
  return SPR_OK;
}

spr_status spr_prefill(spr_model* m, int32_t n, const int32_t* slots, const int32_t* tokens, const int32_t* seq_lens,
                       const int32_t* stop_lens, int32_t* tok, float* logits, int32_t* retired) {
  g_err.clear();
  spr_status st = check_model(m);
  if (st != SPR_OK) return st;
  if (slots == nullptr || tokens == nullptr || seq_lens == nullptr || stop_lens == nullptr || tok == nullptr)
    return fail(SPR_ERR_INVALID_ARG, "prefill: slots, tokens, seq_lens, stop_lens and tok must not be null");
  std::string err;
  if ((st = m->tab.check_prefill(n, slots, seq_lens, stop_lens, &err)) != SPR_OK) return fail(st, err);
  int64_t total = 0;
  for (int i = 0; i < n; ++i) total += seq_lens[i];
  for (int64_t t = 0; t < total; ++t)
    if (tokens[t] < 0 || tokens[t] >= m->d.V) return fail(SPR_ERR_INVALID_ARG, "prefill: token id out of range");

  m->tab.commit_prefill(n, slots, seq_lens, stop_lens, retired);
  std::vector<const int32_t*> prompts(n);
  int64_t t = 0;
  for (int i = 0; i < n; ++i) {
    prompts[i] = tokens + t;
    t += seq_lens[i];
  }
  return prefill_device(m, n, slots, prompts.data(), seq_lens, tok, logits, nullptr, nullptr);
}

spr_status spr_decode_step(spr_model* m, int32_t n_active, const int32_t* slots, const int32_t* lens, int32_t* tok,
                           float* logits, int32_t* retired) {
  g_err.clear();
  spr_status st = check_model(m);
  if (st != SPR_OK) return st;
  if (slots == nullptr || lens == nullptr || tok == nullptr)
    return fail(SPR_ERR_INVALID_ARG, "decode_step: slots, lens and tok must not be null");
  std::string err;
  if ((st = m->tab.check_decode(n_active, slots, lens, &err)) != SPR_OK) return fail(st, err);
  RowSet rs;
  rs.n = n_active;
  for (int r = 0; r < kRows; ++r) {
    const bool v = r < n_active;
    rs.slot[r] = v ? slots[r] : 0;
    rs.pos[r] = v ? lens[r] : 0;
    rs.out_row[r] = v ? r : -1;
    rs.tok[r] = 0;
    rs.hist_idx[r] = -1;
  }
  if ((st = forward_any(m, rs, tok, tok, logits, nullptr, workspace_scratch(m))) != SPR_OK) return st;
  m->tab.commit_decode(n_active, slots, retired);
  return SPR_OK;
}

spr_status spr_decode_step_static_scratch(spr_model* m, int32_t n_active, const int32_t* slots, const int32_t* lens,
                                          int32_t* tok, float* logits, int32_t* retired) {
  g_err.clear();
  spr_status st = check_model(m);
  if (st != SPR_OK) return st;
  if (slots == nullptr || lens == nullptr || tok == nullptr)
    return fail(SPR_ERR_INVALID_ARG, "decode_step_static_scratch: slots, lens and tok must not be null");
  const spr::Dims& d = m->d;
  const size_t per_split = static_cast<size_t>(d.H) * (d.hd + 4) * sizeof(float);
  const int max_splits = static_cast<int>(std::min<size_t>(spr::kMaxSplits, kStaticPartBytes / per_split));
  const spr::SplitNeed sn = spr::split_need(d);
  if (static_cast<size_t>(spr::kMaxRows) * d.Hkv * sizeof(int32_t) > kStaticCntBytes ||
      static_cast<size_t>(d.nt_lm) * spr::kMaxRows * sizeof(float2) > kStaticAmaxBytes || max_splits < n_active ||
      sn.part_floats * sizeof(float) > kStaticPartBytes ||
      static_cast<size_t>(sn.counters) * sizeof(int32_t) > kStaticCntBytes)
    return fail(SPR_ERR_INVALID_ARG, "decode_step_static_scratch: the model or batch exceeds the 24 MiB static "
                                     "scratch (at most 128 KV heads, vocab <= 130048, n_heads * (head_dim + 4) "
                                     "* 4 * n_active <= 16 MiB, d_ff <= 30840 and (n_heads + 2 * n_kv_heads) * "
                                     "head_dim <= 30840)");
  std::string err;
  if ((st = m->tab.check_decode(n_active, slots, lens, &err)) != SPR_OK) return fail(st, err);
  RowSet rs;
  rs.n = n_active;
  for (int r = 0; r < kRows; ++r) {
    const bool v = r < n_active;
    rs.slot[r] = v ? slots[r] : 0;
    rs.pos[r] = v ? lens[r] : 0;
    rs.out_row[r] = v ? r : -1;
    rs.tok[r] = 0;
    rs.hist_idx[r] = -1;
  }
  DecodeScratch sc{reinterpret_cast<float*>(m->static_scratch),
                   reinterpret_cast<int32_t*>(m->static_scratch + kStaticPartBytes),
                   reinterpret_cast<float2*>(m->static_scratch + kStaticPartBytes + kStaticCntBytes),
                   max_splits,
                   kStaticPartBytes / sizeof(float),
                   static_cast<int>(kStaticCntBytes / sizeof(int32_t))};
  // Every call shares the array: the attention split counters and the
  // projections' split-K counters must start at zero (a fill kernel, which a
  // graph capture may record).
  const int ncnt = std::max(n_active * d.Hkv, spr::split_need(d).counters);
  k_zero_i32<<<ceil_div(ncnt, 256), 256, 0, m->st>>>(sc.cnt, ncnt);
  SPR_LAUNCHED(m, "k_zero_i32");
  if ((st = forward_any(m, rs, tok, tok, logits, nullptr, sc)) != SPR_OK) return st;
  m->tab.commit_decode(n_active, slots, retired);
  return SPR_OK;
}

spr_status spr_rewind_slot(spr_model* m, int32_t slot, int32_t len, int32_t produced) {
  g_err.clear();
  spr_status st = check_model(m);
  if (st != SPR_OK) return st;
  std::string err;
  if ((st = m->tab.check_rewind(slot, len, produced, &err)) != SPR_OK) return fail(st, err);
  m->tab.commit_rewind(slot, len, produced);
  return SPR_OK;
}

spr_status spr_free_slot(spr_model* m, int32_t slot) {
  g_err.clear();
  spr_status st = check_model(m);
  if (st != SPR_OK) return st;
  std::string err;
  if ((st = m->tab.check_free(slot, &err)) != SPR_OK) return fail(st, err);
  m->tab.commit_free(slot);
  return SPR_OK;
}

spr_status spr_slot_info(const spr_model* m, int32_t slot, int32_t* len, int32_t* produced, int32_t* stop_len) {
  if (m == nullptr || len == nullptr || produced == nullptr || stop_len == nullptr)
    return fail(SPR_ERR_INVALID_ARG, "slot_info: null argument");
  if (slot < 0 || slot >= m->d.S) return fail(SPR_ERR_INVALID_ARG, "slot_info: slot id out of range");
  const spr::Slot& s = m->tab.slot(slot);
  *len = s.state == spr::kFree ? -1 : s.len;
  *produced = s.produced;
  *stop_len = s.stop;
  return SPR_OK;
}

int32_t spr_free_blocks(const spr_model* m) { return m == nullptr ? -1 : m->tab.free_blocks(); }

spr_status spr_export_weight_rows(spr_model* m, int32_t tensor, int32_t layer, int32_t row0, int32_t nrows,
                                  float* out) {
  g_err.clear();
  spr_status st = check_model(m);
  if (st != SPR_OK) return st;
  const spr::Dims& d = m->d;
  if (out == nullptr) return fail(SPR_ERR_INVALID_ARG, "export: out must not be null");
  if (tensor < 0 || tensor > 8) return fail(SPR_ERR_INVALID_ARG, "export: tensor id must be in [0, 8]");
  const bool per_layer = tensor >= 1 && tensor <= 7;
  if (per_layer ? (layer < 0 || layer >= d.L) : layer != 0) return fail(SPR_ERR_INVALID_ARG, "export: bad layer");
  static const int kind_of[9] = {-1, MK_QKV, MK_QKV, MK_QKV, MK_O, MK_W13, MK_W13, MK_W2, MK_LM};
  static const int which_of[9] = {0, 0, 1, 2, 0, 0, 1, 0, 0};
  int rows_total, cols;
  switch (tensor) {
    case 0: case 8: rows_total = d.V; cols = d.d; break;
    case 1: rows_total = d.H * d.hd; cols = d.d; break;
    case 2: case 3: rows_total = d.Hkv * d.hd; cols = d.d; break;
    case 4: rows_total = d.d; cols = d.o_in; break;
    case 5: case 6: rows_total = d.f; cols = d.d; break;
    default: rows_total = d.d; cols = d.f;
  }
  if (row0 < 0 || nrows < 1 || static_cast<int64_t>(row0) + nrows > rows_total)
    return fail(SPR_ERR_INVALID_ARG, "export: row range outside the matrix");
  Ptrs p{m->ws, &m->lay};
  const int64_t count = static_cast<int64_t>(nrows) * cols;
  const bool bf = d.dtype == SPR_BF16;
  if (tensor == 0) {
    if (bf)
      k_export_rowmajor<BF16><<<grid1(count), 256, 0, m->st>>>(reinterpret_cast<const uint16_t*>(p.emb()), cols,
                                                               row0, nrows, out);
    else
      k_export_rowmajor<F32><<<grid1(count), 256, 0, m->st>>>(reinterpret_cast<const float*>(p.emb()), cols, row0,
                                                              nrows, out);
  } else {
    const MatSpec s = mat_spec(d, kind_of[tensor], per_layer ? layer : 0, m->seed);
    const char* base = tensor <= 3 ? p.wqkv(layer) : tensor == 4 ? p.wo(layer) : tensor <= 6 ? p.w13(layer)
                                                   : tensor == 7 ? p.w2(layer) : p.wlm();
    if (bf)
      k_export_tiled<BF16><<<grid1(count), 256, 0, m->st>>>(reinterpret_cast<const uint16_t*>(base), s,
                                                            which_of[tensor], row0, nrows, out);
    else
      k_export_tiled<F32><<<grid1(count), 256, 0, m->st>>>(reinterpret_cast<const float*>(base), s,
                                                           which_of[tensor], row0, nrows, out);
  }
  SPR_LAUNCHED(m, "export");
  return SPR_OK;
}

spr_status spr_test_write_lm_head_row(spr_model* m, int32_t dst, int32_t src, float fill) {
  g_err.clear();
  spr_status st = check_model(m);
  if (st != SPR_OK) return st;
  const spr::Dims& d = m->d;
  if (dst < 0 || dst >= d.V || src >= d.V)
    return fail(SPR_ERR_INVALID_ARG, "test_write_lm_head_row: dst in [0, vocab), src < vocab");
  Ptrs p{m->ws, &m->lay};
  if (d.dtype == SPR_BF16)
    k_write_tiled_row<BF16><<<ceil_div(d.d, 256), 256, 0, m->st>>>(reinterpret_cast<uint16_t*>(p.wlm()), d.kb_d, d.d,
                                                                    dst, src, fill);
  else
    k_write_tiled_row<F32><<<ceil_div(d.d, 256), 256, 0, m->st>>>(reinterpret_cast<float*>(p.wlm()), d.kb_d, d.d, dst,
                                                                   src, fill);
  SPR_LAUNCHED(m, "k_write_tiled_row");
  SPR_HIP(m, hipStreamSynchronize(m->st));
  return SPR_OK;
}

spr_status spr_time_read_ceiling(spr_model* m, int32_t reps, double* gbps, uint64_t* bytes) {
  g_err.clear();
  spr_status st = check_model(m);
  if (st != SPR_OK) return st;
  if (gbps == nullptr || bytes == nullptr) return fail(SPR_ERR_INVALID_ARG, "time_read_ceiling: null output");
  if (reps < 1 || reps > 1000) return fail(SPR_ERR_INVALID_ARG, "time_read_ceiling: reps in [1, 1000]");
  // Every weight matrix a decode step streams: all layers' projections and the LM head.
  const size_t nbytes = m->lay.off_emb - m->lay.off_wqkv;
  const uint4* base = reinterpret_cast<const uint4*>(m->ws + m->lay.off_wqkv);
  int dev = 0, ncu = 0;
  SPR_HIP(m, hipGetDevice(&dev));
  SPR_HIP(m, hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev));
  hipEvent_t e0, e1;
  SPR_HIP(m, hipEventCreate(&e0));
  hipError_t e = hipEventCreate(&e1);
  if (e != hipSuccess) {
    (void)hipEventDestroy(e0);
    return hip_fail(m, "hipEventCreate", e);
  }
  Ptrs p{m->ws, &m->lay};
  uint32_t* sink = reinterpret_cast<uint32_t*>(p.amax());
  e = hipEventRecord(e0, m->st);
  for (int r = 0; r < reps && e == hipSuccess; ++r) {
    k_read_stream<<<ncu * 8, 256, 0, m->st>>>(base, nbytes / 16, sink);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipEventRecord(e1, m->st);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (e != hipSuccess) return hip_fail(m, "time_read_ceiling", e);
  *bytes = static_cast<uint64_t>(nbytes);
  *gbps = static_cast<double>(nbytes) * reps / (static_cast<double>(ms) * 1e-3) / 1e9;
  return SPR_OK;
}

spr_status spr_time_projection(spr_model* m, int32_t projection, int32_t n_rows, int32_t reps, float* avg_us) {
  g_err.clear();
  spr_status st = check_model(m);
  if (st != SPR_OK) return st;
  if (avg_us == nullptr) return fail(SPR_ERR_INVALID_ARG, "time_projection: avg_us must not be null");
  if (projection < 1 || projection > 4)
    return fail(SPR_ERR_INVALID_ARG, "time_projection: projection must be 1 (O), 2 (gate/up), 3 (down) or 4 (LM head)");
  if (n_rows < 1 || n_rows > kRows || reps < 1 || reps > 100000)
    return fail(SPR_ERR_INVALID_ARG, "time_projection: n_rows in [1, 128] and reps in [1, 100000]");
  hipEvent_t e0, e1;
  SPR_HIP(m, hipEventCreate(&e0));
  hipError_t e = hipEventCreate(&e1);
  if (e != hipSuccess) {
    (void)hipEventDestroy(e0);
    return hip_fail(m, "hipEventCreate", e);
  }
  e = hipEventRecord(e0, m->st);
  // Launch r uses layer r mod n_layers, so the weights streamed are the whole
  // model's share of this projection, as in a decode step, and a matrix that
  // would fit in the last-level cache is not re-read from it.
  for (int r = 0; r < reps && e == hipSuccess && st == SPR_OK; ++r)
    st = m->d.dtype == SPR_BF16 ? launch_projection<BF16>(m, projection, r % m->d.L, n_rows)
                                : launch_projection<F32>(m, projection, r % m->d.L, n_rows);
  if (e == hipSuccess && st == SPR_OK) e = hipEventRecord(e1, m->st);
  if (e == hipSuccess && st == SPR_OK) e = hipEventSynchronize(e1);
  float ms = 0.f;
  if (e == hipSuccess && st == SPR_OK) e = hipEventElapsedTime(&ms, e0, e1);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (st != SPR_OK) return st;
  if (e != hipSuccess) return hip_fail(m, "time_projection", e);
  *avg_us = 1000.f * ms / static_cast<float>(reps);
  return SPR_OK;
}

spr_status spr_serve(spr_model* m, int32_t n, const spr_request* reqs, int32_t max_active, int32_t eos_id,
                     int32_t* tok, int32_t* out, int32_t* lengths, spr_serve_stats* stats) {
  g_err.clear();
  spr_status st = check_model(m);
  if (st != SPR_OK) return st;
  if (n < 0 || (n > 0 && (reqs == nullptr || tok == nullptr || out == nullptr)))
    return fail(SPR_ERR_INVALID_ARG, "serve: n must be >= 0, and reqs, tok and out non-null");
  if (eos_id >= m->d.V) return fail(SPR_ERR_INVALID_ARG, "serve: eos_id must be < vocab (or negative: none)");
  std::vector<spr::ServeRequest> rq(n);
  std::vector<int64_t> off(static_cast<size_t>(n) + 1, 0);
  for (int i = 0; i < n; ++i) {
    if (reqs[i].level < 0 || reqs[i].level >= SPR_MAX_LEVELS)
      return fail(SPR_ERR_INVALID_ARG, "serve: level must be in [0, SPR_MAX_LEVELS)");
    rq[i] = spr::ServeRequest{reqs[i].tokens, reqs[i].n_tokens, reqs[i].stop_len, reqs[i].arrival};
    off[i + 1] = off[i] + std::max(reqs[i].stop_len, 0);
  }
  if (off[n] > INT32_MAX) return fail(SPR_ERR_INVALID_ARG, "serve: too many output tokens");
  GpuServe dev;
  dev.m = m;
  dev.reqs = rq.data();
  dev.off = off.data();
  dev.tok = tok;
  dev.out = out;
  dev.eos_id = eos_id < 0 ? -1 : eos_id;
  hipEvent_t start = nullptr;
  struct Cleanup {  // releases what this call created, on every path
    GpuServe* d;
    hipEvent_t* start;
    ~Cleanup() {
      for (hipEvent_t e : d->ev_iter) (void)hipEventDestroy(e);
      for (hipEvent_t e : d->snap)
        if (e) (void)hipEventDestroy(e);
      if (*start) (void)hipEventDestroy(*start);
      if (d->pin) (void)hipHostFree(d->pin);
    }
  } cleanup{&dev, &start};
  SPR_HIP(m, hipEventCreate(&start));
  if (dev.eos_id >= 0) {
    SPR_HIP(m, hipHostMalloc(reinterpret_cast<void**>(&dev.pin), 4 * m->d.S * sizeof(int32_t), hipHostMallocDefault));
    for (int i = 0; i < 2; ++i) SPR_HIP(m, hipEventCreateWithFlags(&dev.snap[i], hipEventDisableTiming));
  }
  SPR_HIP(m, hipEventRecord(start, m->st));
  spr::ServeCounters c;
  std::vector<int32_t> len;
  std::string err;
  st = spr::serve(m->tab, m->d, n, rq.data(), max_active, dev, &c, &len, &err);
  if (st != SPR_OK) return err.empty() ? st : fail(st, err);
  SPR_HIP(m, hipStreamSynchronize(m->st));
  if (lengths != nullptr)
    for (int i = 0; i < n; ++i) lengths[i] = len[i];
  if (stats != nullptr) {
    // Each iteration's device time, shared equally by the requests it served.
    std::vector<double> sec(n, 0.0);
    double total = 0.0;
    hipEvent_t prev = start;
    for (size_t it = 0; it < dev.ev_iter.size(); ++it) {
      float ms = 0.f;
      SPR_HIP(m, hipEventElapsedTime(&ms, prev, dev.ev_iter[it]));
      prev = dev.ev_iter[it];
      total += ms * 1e-3;
      const auto& who = dev.served[it];
      for (int r : who) sec[r] += ms * 1e-3 / static_cast<double>(who.size());
    }
    *stats = spr_serve_stats{};
    stats->iterations = c.iterations;
    stats->decode_steps = c.decode_steps;
    stats->prefill_calls = c.prefill_calls;
    stats->decode_tokens = c.decode_tokens;
    stats->max_batch = c.max_batch;
    stats->mean_batch = c.mean_batch;
    stats->device_seconds = total;
    for (int i = 0; i < n; ++i) {
      const int lv = reqs[i].level;
      stats->level_requests[lv] += 1;
      stats->level_tokens[lv] += len[i];
      stats->level_seconds[lv] += sec[i];
    }
    for (int lv = 0; lv < SPR_MAX_LEVELS; ++lv) {
      if (stats->level_requests[lv] == 0) continue;
      stats->level_tokens[lv] /= stats->level_requests[lv];
      stats->level_seconds[lv] /= stats->level_requests[lv];
    }
  }
  return SPR_OK;
}

spr_status spr_release(spr_model* m) {
  if (m == nullptr) return fail(SPR_ERR_INVALID_ARG, "release: model is null");
  delete m;
  return SPR_OK;
}

const char* spr_last_error(void) { return g_err.c_str(); }

}  // extern "C"
