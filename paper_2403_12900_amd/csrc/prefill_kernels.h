// Prefill: the prompt of every new request runs through the model in chunks
// of up to kPrefillRows token rows, filling the KV cache (Section II-A: the
// prompt's keys and values are computed once and cached; generation follows).
// Unlike decode, each weight byte now meets hundreds of rows, so the
// projections are compute-bound: a tiled MFMA GEMM stages output tiles of up
// to 256 x 256 through LDS.  Attention is causal over each request's own
// positions; a wave's 16 MFMA columns are 16 consecutive query positions of
// one request and head, and the four waves of a work-group share each K/V
// tile they read from LDS, so every tile read feeds up to 64 queries.
#pragma once

#include <utility>

#include "attn_kernels.h"

namespace sprk {

constexpr int kPrefillRows = 4096;  // token rows per prefill chunk

// One token row of a chunk.
struct PrefillRow {
  int slot, pos, tok, pad;
};

// Up to 64 consecutive rows of one request (positions pos0 .. pos0 + n - 1
// at chunk rows row0 .. row0 + n - 1): one attention query tile.
struct PrefillTile {
  int slot, row0, n, pos0;
};

// x = E[tok], and its activation record (K-block-major, Rp rows).
template <class P>
__global__ __launch_bounds__(64) void k_embed_rows(const typename P::elem* __restrict__ emb,
                                                   const PrefillRow* __restrict__ rows, float* x,
                                                   typename P::elem* act, int d, int V, int Rp) {
  const int b = blockIdx.y;
  const int n0 = 4 * (blockIdx.x * 64 + threadIdx.x);
  if (n0 >= d) return;
  const int t = min(max(rows[b].tok, 0), V - 1);
  const typename P::elem* e = emb + static_cast<size_t>(t) * d + n0;
  const float v0 = P::to_f32(e[0]), v1 = P::to_f32(e[1]), v2 = P::to_f32(e[2]), v3 = P::to_f32(e[3]);
  *reinterpret_cast<float4*>(x + static_cast<size_t>(b) * d + n0) = make_float4(v0, v1, v2, v3);
  store_act4<P>(act, Rp, b, n0, v0, v1, v2, v3);
}

// RMSNorm scale of each row (unit gains): rs[b] = 1 / sqrt(mean(x_b^2) + eps).
// One wave per row.
__global__ __launch_bounds__(256) void k_row_rscale(const float* __restrict__ x, float* rs, int M, int d, float eps) {
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (b >= M) return;
  const float* xr = x + static_cast<size_t>(b) * d;
  float s = 0.f;
  for (int k = 4 * lane; k < d; k += 256) {
    const float4 v = *reinterpret_cast<const float4*>(xr + k);
    s = fmaf(v.x, v.x, fmaf(v.y, v.y, fmaf(v.z, v.z, fmaf(v.w, v.w, s))));
  }
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o);
  if (lane == 0) rs[b] = rsqrtf(s / static_cast<float>(d) + eps);
}

typedef __attribute__((address_space(1))) void global_void;
typedef __attribute__((address_space(3))) void lds_void;

// Waits until at most N vector-memory operations of this wave are in flight
// (expcnt and lgkmcnt not waited on).
template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// 16-byte LDS read issued as plain ds_read_b128.  The compiler treats LDS
// that global_load_lds fills as possibly still in flight and, at loop
// back-edges, would wait for every load in flight (vmcnt(0)) before any LDS
// read; the kernel's own vmcnt wait plus barrier already orders the read, so
// the read bypasses that tracking.  The caller waits with lds_reads_done()
// before using the results.
__device__ __forceinline__ u32x4_t lds_read16(const uint4* p) {
  u32x4_t v;
  const uint32_t a = static_cast<uint32_t>(reinterpret_cast<size_t>((lds_void*)p));
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(a));
  return v;
}
__device__ __forceinline__ void lds_reads_done() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
// Calls f(std::integral_constant<int, j>) for j = 0 .. N - 1 in order.
template <class F, int... J>
__device__ __forceinline__ void static_for_seq(F& f, std::integer_sequence<int, J...>) {
  (f(std::integral_constant<int, J>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F& f) {
  static_for_seq(f, std::make_integer_sequence<int, N>{});
}

// Waits until at most N of this wave's LDS reads are in flight (they return
// in issue order, so every read but the last N has landed).
template <int N>
__device__ __forceinline__ void lds_reads_left() {
  static_assert(N >= 0 && N < 16, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
}
// Ties a value read by lds_read16 to a point after lds_reads_done(): volatile
// asm statements keep their order, so no use of v can move above the wait.
__device__ __forceinline__ void lds_value_ready(u32x4_t& v) { asm volatile("" : "+v"(v)); }

// Work-group barrier for LDS filled by global_load_lds: each wave first waits
// for its own loads (vmcnt), so after the barrier every wave's fragments of
// that stage are in LDS.  No memory fence: a workgroup fence here would wait
// for every load in flight (vmcnt(0)), including the stages being prefetched.
// The empty asm statements keep the compiler from moving LDS accesses across.
__device__ __forceinline__ void lds_stage_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Tiled projection: out[b][n] = sum_k W[n][k] x[b][k] for rows b < M, fused
// with the op that follows (Epi).  A work-group computes TN weight tiles (16
// output features each) x TM row tiles (16 rows each) with NW waves, each
// owning a WN x WM block of 16 x 16 MFMA tiles.  Per K-block the work-group's
// operands -- TN weight fragments and TM x parts activation fragments, 1 KiB
// each -- go from global memory straight into LDS (global_load_lds, no
// register staging) in MFMA lane order: weight fragments are stored that way,
// and for activation fragments lane r + 16 g fetches row r's K-group g.  Three
// LDS stages (three separate arrays, so the compiler tracks each stage's
// loads on its own) keep two K-blocks in flight; each K-block costs one
// barrier: wait for its own loads, barrier (which also frees the stage read
// one K-block earlier), issue the loads two K-blocks ahead, multiply.  Weight
// tiles past NT re-read tile NT - 1 and row tiles past Rp re-read the last
// one; neither is stored.
// The operands a K-block moves from L2 into LDS, TN + parts x TM fragments,
// bound these kernels before MFMA does: the largest shape (256 features x 256
// rows, eight waves) moves half the bytes per product of 128 x 128.
template <int TN, int TM, int NW>
struct TileShape {
  static constexpr int GN = NW == 8 ? 2 : TN == 4 && TM == 8 ? 1 : 2;  // waves along features
  static constexpr int GM = NW / GN;                                  // waves along rows
  static constexpr int WN = TN / GN, WM = TM / GM;
  static_assert(GN * GM == NW && WN * GN == TN && WM * GM == TM, "tile shape");
};

// LP: parts per K-block of the activation record (the first P::parts are used).
template <class P, int TN, int TM, class Epi, int NW = 4, int LP = P::parts>
__global__ __launch_bounds__(NW * 64) void k_tile_gemm(const uint4* __restrict__ W, const uint4* __restrict__ X,
                                                       int NT, int KB, int Rp, Epi epi) {
  constexpr int PARTS = P::parts;
  static_assert(LP >= PARTS, "the record holds the parts used");
  constexpr int NFRAG = TN + TM * PARTS;
  static_assert(NFRAG % NW == 0, "fragments per stage must split over the waves");
  constexpr int L = NFRAG / NW;  // loads per wave per stage
  using TS = TileShape<TN, TM, NW>;
  constexpr int WN = TS::WN, WM = TS::WM;
  __shared__ uint4 st0[NFRAG][64];
  __shared__ uint4 st1[NFRAG][64];
  __shared__ uint4 st2[NFRAG][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // Work-groups go to the eight XCDs in turn (linear id mod 8), and each XCD
  // has its own L2.  XCD x takes the contiguous range of tiles from x * total
  // / 8 in an order that runs over groups of four row tiles, the row tile
  // fastest: the 32 work-groups an XCD holds at a time then cover 8 weight
  // tiles x 4 row tiles and fetch about 256 KB of operands per K-block instead
  // of up to 1.5 MB.
  int nt0, m0;
  {
    const int total = gridDim.x * gridDim.y, b = blockIdx.y * gridDim.x + blockIdx.x;
    const int q = total / 8, r = total % 8, x = b % 8, j = b / 8;
    const int t = x * q + min(x, r) + j;
    const int gm = gridDim.y % 4 == 0 ? 4 : 1;
    const int per_group = gm * gridDim.x;
    const int mg = t / per_group, rem = t % per_group;
    nt0 = (rem / gm) * TN;
    m0 = (mg * gm + rem % gm) * TM * 16;
  }
  const int wn = wave % TS::GN, wm = wave / TS::GN;
  const size_t xpart = static_cast<size_t>(Rp) * 4;  // uint4 per (K-block, part)
  const int xlane = (lane & 15) * 4 + (lane >> 4);   // uint4 of an activation fragment MFMA lane `lane` needs

  auto issue = [&](int kb, uint4(*dst)[64]) {
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const int f = wave + NW * i;
      const uint4* src;
      if (f < TN) {
        const int nt = min(nt0 + f, NT - 1);
        src = W + (static_cast<size_t>(nt) * KB + kb) * 64 + lane;
      } else {
        const int a = f - TN, q = a / TM, tt = a % TM;
        const int r0 = min(m0 + 16 * tt, Rp - 16);
        src = X + (static_cast<size_t>(kb) * LP + q) * xpart + static_cast<size_t>(r0) * 4 + xlane;
      }
      __builtin_amdgcn_global_load_lds((global_void*)src, (lds_void*)&dst[f][0], 16, 0, 0);
    }
  };

  f32x4_t acc[WN][WM];
#pragma unroll
  for (int i = 0; i < WN; ++i)
#pragma unroll
    for (int j = 0; j < WM; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // K-block kb: its loads are the oldest in flight; the next K-block's (if
  // any) may stay in flight.  Then the stage read at kb - 1 is free for kb + 2.
  auto step = [&](int kb, uint4(*cur)[64], uint4(*next)[64]) {
    if (kb + 1 < KB) {
      wait_vmem<L>();
    } else {
      wait_vmem<0>();
    }
    lds_stage_barrier();
    if (kb + 2 < KB) issue(kb + 2, next);
    // Reads in the order the products use them: the weight fragments, then
    // the activation fragments of row tile 0, 1, ...  The products of row
    // tile j start once its reads have landed, while the later tiles' reads
    // are still in flight.
    u32x4_t a[WN], b[WM][PARTS];
#pragma unroll
    for (int i = 0; i < WN; ++i) a[i] = lds_read16(&cur[wn * WN + i][lane]);
#pragma unroll
    for (int j = 0; j < WM; ++j)
#pragma unroll
      for (int q = 0; q < PARTS; ++q) b[j][q] = lds_read16(&cur[TN + q * TM + wm * WM + j][lane]);
    auto row_tile = [&](auto jc) {
      constexpr int j = decltype(jc)::value;
      lds_reads_left<(WM - 1 - j) * PARTS>();
      if constexpr (j == 0) {
#pragma unroll
        for (int i = 0; i < WN; ++i) lds_value_ready(a[i]);
      }
#pragma unroll
      for (int q = 0; q < PARTS; ++q) lds_value_ready(b[j][q]);
#pragma unroll
      for (int i = 0; i < WN; ++i)
#pragma unroll
        for (int q = 0; q < PARTS; ++q)
          acc[i][j] = P::mma(acc[i][j], __builtin_bit_cast(uint4, a[i]), __builtin_bit_cast(uint4, b[j][q]));
      // Keep these products ahead of the next tile's wait (the scheduler
      // would otherwise sink them below it).
      __builtin_amdgcn_sched_barrier(0);
    };
    static_for<WM>(row_tile);
  };

  issue(0, st0);
  if (KB > 1) issue(1, st1);
  for (int kb = 0; kb < KB; kb += 3) {
    step(kb, st0, st2);
    if (kb + 1 < KB) step(kb + 1, st1, st0);
    if (kb + 2 < KB) step(kb + 2, st2, st1);
  }
#pragma unroll
  for (int i = 0; i < WN; ++i) {
    const int nt = nt0 + wn * WN + i;
    if (nt >= NT) continue;
#pragma unroll
    for (int j = 0; j < WM; ++j) epi.apply_tile(nt, m0 + 16 * (wm * WM + j), acc[i][j], lane);
  }
}

// QKV epilogue: RMSNorm scale, RoPE on q and k, q to the attention input,
// k and v appended to the paged KV cache (same tile orders as decode).
template <class P, class KP = P>
struct EpiQKVRows {
  int M, H, Hkv, hd, mb;
  int nt_base;                    // weight tile of the launch's tile 0 (the launch may cover part of QKV)
  float* q;                       // [rows][H * hd]
  typename KP::elem* kc;
  typename KP::elem* vc;
  const int32_t* bt;
  const float2* rope;
  const PrefillRow* rows;
  const float* rs;

  __device__ __forceinline__ void apply_tile(int nt, int m0, const f32x4_t& acc, int lane) const {
    const int b = m0 + (lane & 15);
    if (b >= M) return;
    const int n0 = 16 * (nt_base + nt) + 4 * (lane >> 4);
    const int qr = H * hd, kr = Hkv * hd;
    const float s = rs[b];
    float v0 = acc[0] * s, v1 = acc[1] * s, v2 = acc[2] * s, v3 = acc[3] * s;
    const PrefillRow row = rows[b];
    const int p = row.pos;
    if (n0 < qr + kr) {
      const int dd = (n0 < qr ? n0 : n0 - qr) % hd;
      const float4 cs = *reinterpret_cast<const float4*>(rope + static_cast<size_t>(p) * (hd / 2) + dd / 2);
      const float a0 = v0 * cs.x - v1 * cs.y, a1 = v0 * cs.y + v1 * cs.x;
      const float a2 = v2 * cs.z - v3 * cs.w, a3 = v2 * cs.w + v3 * cs.z;
      v0 = a0;
      v1 = a1;
      v2 = a2;
      v3 = a3;
    }
    if (n0 < qr) {
      *reinterpret_cast<float4*>(q + static_cast<size_t>(b) * qr + n0) = make_float4(v0, v1, v2, v3);
      return;
    }
    const int blk = bt[static_cast<size_t>(row.slot) * mb + (p >> 4)];
    const int off = p & 15;
    if (n0 < qr + kr) {
      const int m = n0 - qr, kvh = m / hd, dd = m % hd;
      typename KP::elem* dst = kc + (static_cast<size_t>(blk) * Hkv + kvh) * 16 * hd + ktile_offset<KP>(off, dd);
      dst[0] = KP::from_f32(v0);
      dst[1] = KP::from_f32(v1);
      dst[2] = KP::from_f32(v2);
      dst[3] = KP::from_f32(v3);
    } else {
      const int m = n0 - qr - kr, kvh = m / hd, dd = m % hd;
      typename KP::elem* dst = vc + (static_cast<size_t>(blk) * Hkv + kvh) * 16 * hd;
      dst[vtile_offset<KP>(off, dd)] = KP::from_f32(v0);
      dst[vtile_offset<KP>(off, dd + 1)] = KP::from_f32(v1);
      dst[vtile_offset<KP>(off, dd + 2)] = KP::from_f32(v2);
      dst[vtile_offset<KP>(off, dd + 3)] = KP::from_f32(v3);
    }
  }
};

// O and down projections: residual add, new residual as the next activation.
template <class P>
struct EpiResidRows {
  int M, d, Rp;
  float* x;
  typename P::elem* act;

  __device__ __forceinline__ void apply_tile(int nt, int m0, const f32x4_t& acc, int lane) const {
    const int b = m0 + (lane & 15);
    if (b >= M) return;
    const int n0 = 16 * nt + 4 * (lane >> 4);
    float4* xp = reinterpret_cast<float4*>(x + static_cast<size_t>(b) * d + n0);
    float4 xv = *xp;
    xv.x += acc[0];
    xv.y += acc[1];
    xv.z += acc[2];
    xv.w += acc[3];
    *xp = xv;
    store_act4<P>(act, Rp, b, n0, xv.x, xv.y, xv.z, xv.w);
  }
};

// Gate/up (interleaved rows): RMSNorm scale, h = SiLU(gate) * up.
template <class P>
struct EpiSwiGLURows {
  int M, Rp;
  const float* rs;
  typename P::elem* act;

  __device__ __forceinline__ void apply_tile(int nt, int m0, const f32x4_t& acc, int lane) const {
    const int b = m0 + (lane & 15);
    if (b >= M) return;
    const int j0 = 8 * nt + 2 * (lane >> 4);
    const float s = rs[b];
    const float g0 = acc[0] * s, g1 = acc[1] * s, u0 = acc[2] * s, u1 = acc[3] * s;
    act_store<P>(act, Rp, b, j0, g0 / (1.f + __expf(-g0)) * u0);
    act_store<P>(act, Rp, b, j0 + 1, g1 / (1.f + __expf(-g1)) * u1);
  }
};

// Causal attention over each query tile's own request.  Work-group (tile of
// up to 64 consecutive rows of one request, query head): wave w owns rows
// 16 w .. 16 w + 15 as its 16 MFMA columns.  The work-group walks the KV blocks
// up to the tile's last position once.  Each block's K and V tiles come from
// global memory once, straight into LDS, and all four waves multiply their
// columns against them; the next block's loads are in flight while the
// current one is used (two LDS buffers, two barriers per block).  Sharing a
// block among 64 queries instead of 16 cuts the cache reads that bound this
// kernel fourfold.  A wave skips blocks that start after its last position;
// block 0 holds position 0, so every column's running maximum is finite after
// it.  Columns past the tile's rows repeat its last row and are not stored.
template <class P, class AP, int HD>
__global__ __launch_bounds__(256) void k_attn_prefill(const float* __restrict__ q, const void* kcv, const void* vcv,
                                                      const int32_t* __restrict__ bt,
                                                      const PrefillTile* __restrict__ tiles, void* actv, int H,
                                                      int Hkv, int mb, int Rp, float qscale) {
  using E = typename P::elem;
  using Blk = KVBlock<P, HD>;
  constexpr bool kBf16 = sizeof(E) == 2;
  constexpr int NF = Blk::NF, NV = Blk::NV;
  constexpr int NE = HD / 16;
  constexpr int KU = NF * 64, KVU = (NF + NV) * 64;  // uint4 of a block's K tile, of its K and V tiles
  constexpr int PER = KVU / 256;                     // uint4 each thread stages per block
  static_assert(KVU % 256 == 0, "a block's K and V tiles split evenly over the work-group");
  __shared__ uint4 skv[2][KVU];
  const PrefillTile tile = tiles[blockIdx.x];
  const int hq = blockIdx.y, kvh = hq / (H / Hkv);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = lane & 15, g = lane >> 4;
  const int r0 = 16 * wave;                            // the wave's first row of the tile
  const int rw = min(16, tile.n - r0);                 // its rows (none if <= 0)
  const int cq = rw > 0 ? r0 + (c < rw ? c : rw - 1) : tile.n - 1;
  const int pc = tile.pos0 + cq;                       // this column's position
  const int wave_last = tile.pos0 + (rw > 0 ? r0 + rw - 1 : 0);
  const int max_pos = tile.pos0 + tile.n - 1;
  const int nblk = (max_pos >> 4) + 1;
  const int32_t* btrow = bt + static_cast<size_t>(tile.slot) * mb;
  const E* kc = static_cast<const E*>(kcv);
  const E* vc = static_cast<const E*>(vcv);
  int ids = lane < nblk ? btrow[lane] : 0;             // block ids of blocks [i0, i0 + 64)

  // Block i's K and V tiles, straight from global memory into LDS buffer buf
  // (global_load_lds; no registers), thread t moving uint4 t, t + 256, ...
  // The block's id is lane (i mod 64) of ids.
  auto issue = [&](int i, int buf) __attribute__((always_inline)) {
    const int blk = __builtin_amdgcn_readlane(ids, i & 63);
    const size_t off = (static_cast<size_t>(blk) * Hkv + kvh) * 16 * HD;
    const uint4* kt = reinterpret_cast<const uint4*>(kc + off);
    const uint4* vt = reinterpret_cast<const uint4*>(vc + off);
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int idx = tid + 256 * p;
      const uint4* src = idx < KU ? kt + idx : vt + (idx - KU);
      __builtin_amdgcn_global_load_lds((global_void*)src, (lds_void*)&skv[buf][256 * p + 64 * wave], 16, 0, 0);
    }
  };

  uint4 qh[NF], ql[NF];
  {
    const float* qp = q + (static_cast<size_t>(tile.row0 + cq) * H + hq) * HD + g * P::per16;
    float4 qv[NF][P::per16 / 4];
#pragma unroll
    for (int f = 0; f < NF; ++f)
#pragma unroll
      for (int j4 = 0; j4 < P::per16 / 4; ++j4) qv[f][j4] = *reinterpret_cast<const float4*>(qp + f * P::kblk + 4 * j4);
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      union {
        uint4 u;
        E e[P::per16];
      } vh, vl;
#pragma unroll
      for (int j = 0; j < P::per16; ++j) {
        const float4 t = qv[f][j / 4];
        const float v = (j % 4 == 0 ? t.x : j % 4 == 1 ? t.y : j % 4 == 2 ? t.z : t.w) * qscale;
        vh.e[j] = P::from_f32(v);
        vl.e[j] = P::from_f32(v - P::to_f32(vh.e[j]));
      }
      qh[f] = vh.u;
      ql[f] = vl.u;
    }
  }

  f32x4_t O[NE];
#pragma unroll
  for (int e = 0; e < NE; ++e) O[e] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  issue(0, 0);
  for (int i = 0; i < nblk; ++i) {
    const int cur = i & 1;
    // The next block goes into the other buffer, which every wave finished
    // reading before the previous block's closing barrier.
    if (i + 1 < nblk) {
      if (((i + 1) & 63) == 0) ids = i + 1 + lane < nblk ? btrow[i + 1 + lane] : 0;
      issue(i + 1, cur ^ 1);
      wait_vmem<PER>();  // this thread's loads of block i have landed
    } else {
      wait_vmem<0>();
    }
    lds_stage_barrier();  // every thread's loads of block i have landed
    if (rw > 0 && i * 16 <= wave_last) {  // wave-uniform: the block has keys some column sees
      Blk B;
      u32x4_t kr[NF], vr[NV];
#pragma unroll
      for (int f = 0; f < NF; ++f) kr[f] = lds_read16(&skv[cur][f * 64 + lane]);
#pragma unroll
      for (int v = 0; v < NV; ++v) vr[v] = lds_read16(&skv[cur][KU + v * 64 + lane]);
      lds_reads_done();
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        lds_value_ready(kr[f]);
        B.kf[f] = __builtin_bit_cast(uint4, kr[f]);
      }
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        lds_value_ready(vr[v]);
        B.vf[v] = __builtin_bit_cast(uint4, vr[v]);
      }
      f32x4_t S = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        S = P::mma(S, B.kf[f], qh[f]);
        if constexpr (kBf16) S = P::mma(S, B.kf[f], ql[f]);
      }
      if (i * 16 + 15 > tile.pos0 + r0) {  // block reaches past the wave's first position: causal mask
        const int valid = pc - (i * 16 + 4 * g) + 1;
#pragma unroll
        for (int r = 0; r < 4; ++r) S[r] = r < valid ? S[r] : -INFINITY;
      }
      if (i == nblk - 1) B.mask_v(max_pos - (i * 16 + 4 * g) + 1);
      float mb2 = fmaxf(fmaxf(S[0], S[1]), fmaxf(S[2], S[3]));
      mb2 = fmaxf(mb2, __shfl_xor(mb2, 16));
      mb2 = fmaxf(mb2, __shfl_xor(mb2, 32));
      const float m_new = fmaxf(m_run, mb2);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
      float p[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) p[r] = __builtin_amdgcn_exp2f(S[r] - m_use);
      l_run = l_run * alpha + ((p[0] + p[1]) + (p[2] + p[3]));
      if (i != 0 && __ballot(m_new != m_run) != 0) {
#pragma unroll
        for (int e = 0; e < NE; ++e) {
          O[e][0] *= alpha;
          O[e][1] *= alpha;
          O[e][2] *= alpha;
          O[e][3] *= alpha;
        }
      }
      m_run = m_new;
      B.pv(O, p);
    }
    lds_stage_barrier();  // buffer cur is free for block i + 2
  }
  if (rw <= 0) return;
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  if (c >= rw) return;
  const float inv = 1.f / l_run;
  typename AP::elem* act = static_cast<typename AP::elem*>(actv);
#pragma unroll
  for (int e = 0; e < NE; ++e)
    store_act4<AP>(act, Rp, tile.row0 + r0 + c, hq * HD + 16 * e + 4 * g, O[e][0] * inv, O[e][1] * inv,
                   O[e][2] * inv, O[e][3] * inv);
}

// Rows src[k] of the residual as rows k of an activation record (Rp rows),
// for the LM head of the rows that emit a token.
struct GatherArgs {
  const float* x;
  void* act;
  int d, Rp, n;
  int src[kRows];
};
template <class P>
__global__ __launch_bounds__(64) void k_gather_rows(GatherArgs a) {
  const int k = blockIdx.y;
  const int n0 = 4 * (blockIdx.x * 64 + threadIdx.x);
  if (n0 >= a.d || k >= a.n) return;
  const float4 v = *reinterpret_cast<const float4*>(a.x + static_cast<size_t>(a.src[k]) * a.d + n0);
  store_act4<P>(static_cast<typename P::elem*>(a.act), a.Rp, k, n0, v.x, v.y, v.z, v.w);
}

}  // namespace sprk
