// Weight-streaming projection for decode: y[b][n] = sum_k W[n][k] x[b][k] for
// every active row b, with the op that follows fused into the epilogue.
//
// Decode reads every weight byte once per step while the batch is at most a
// few dozen rows, so the kernel is HBM-bound (intensity = rows flop/byte, far
// below the MFMA ridge).  MFMA is used as the dot-product engine because the
// tiles come straight from HBM in the operand layout, not because the
// kernel needs its throughput:
//   * one work-group per RT 16-row output tiles; its waves split the K-blocks,
//     each streaming contiguous 1 KiB weight fragments with 16-byte loads;
//   * the activations (rows x K, K-block-major, see act_offset) are the MFMA
//     B operand: one wave load reads 1 KiB of consecutive bytes (16 rows x 64
//     bytes of one part), and lanes of rows past the batch re-read row 0, so
//     a batch of one moves one row's bytes;
//   * a work-group may own RT row tiles, so each activation fragment feeds RT
//     weight fragments (fewer activation bytes per weight byte);
//   * bf16 activations come as hi + lo parts (two MFMAs per fragment), which
//     keeps the activation side of every product near fp32 precision; the
//     QKV projection's input comes as hi + mid + lo (all 24 bits, three
//     MFMAs), since its keys and values are rounded into a bf16 cache;
//   * per-wave accumulators are summed through LDS in a fixed order, so the
//     result is bitwise reproducible.
// RMSNorm (unit gains) of the input is fused: the sum of squares of each row
// is accumulated from the activation fragments already in registers (on
// MFMA, see k_stream_gemm), and 1/sqrt(mean + eps) scales the accumulator in
// the epilogue.
#pragma once

#include "device_common.h"

namespace sprk {

constexpr int kRows = 128;      // token rows per pass

struct RowSlotPos {
  int slot[kRows];
  int pos[kRows];
};

// Fragments each wave loads per pipeline stage, by MFMA work per K-block
// (row tiles x activation tiles x parts): more in flight when registers allow.
template <int XW>
struct StreamDepth {
  static constexpr int value = XW <= 3 ? 8 : XW <= 6 ? 4 : 2;
};

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// Weight fragment load; streaming (nontemporal) loads keep the once-read
// weights from displacing activations in the caches.
template <bool kStream>
__device__ __forceinline__ uint4 load_weight(const uint4* p) {
  if constexpr (kStream) {
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
  } else {
    return *p;
  }
}

// Activation fragments per K-block and 16-row tile: one per part, or, with
// packed rows (PK: at most 8 rows, JT = 1), two parts per fragment -- lanes
// of columns 0-7 carry part 2f of rows 0-7 and lanes of columns 8-15 part
// 2f + 1 of the same rows, so a batch of at most 8 rows spends half the MFMA
// columns and activation loads of the unpacked form.
template <class P, bool PK>
struct StreamFrags {
  static constexpr int value = PK ? (P::parts + 1) / 2 : P::parts;
};

// One work-group computes RT consecutive 16-row output tiles for all rows;
// its WAVES waves split the K-blocks, and each activation fragment a wave
// loads feeds RT weight fragments.
template <int JT, int RT, int UH, int XF>
struct StreamStage {
  uint4 a[UH][RT];                 // weight fragments
  uint4 x[UH][JT][XF];             // activation fragments
};

// Gram accumulator entries.  Entry (i, j) of a 16 x 16 MFMA accumulator sits
// in lane j + 16 * (i / 4), register i % 4.  gram_pick(g, lane) is the
// register each lane offers, g[lane % 4]; gram_entry(pick, i, j) then reads
// entry (i, j) for any i = j (mod 4), in particular the diagonal.
__device__ __forceinline__ float gram_pick(const f32x4_t& gm, int lane) {
  const int r = lane & 3;
  return r == 0 ? gm[0] : r == 1 ? gm[1] : r == 2 ? gm[2] : gm[3];
}
__device__ __forceinline__ float gram_entry(float pick, int i, int j) { return __shfl(pick, j + 16 * (i >> 2)); }

// One work-group computes RT consecutive 16-row output tiles for all rows;
// its WAVES waves split the K-blocks, and each activation fragment a wave
// loads feeds RT weight fragments.  Loads are software-pipelined: a wave
// issues the next stage of UH K-blocks before computing the current one, so
// its requests stay in flight while it computes.  For epilogues that apply
// RMSNorm, the rows' sums of squares come from MFMA too: the Gram product
// X^T X of each activation fragment with itself has them on its diagonal.
// For bf16 activations (x = hi + lo) that is hi.hi + 2 hi.lo, two MFMAs: the
// diagonal of hi.lo equals that of lo.hi, and lo.lo (at most 2^-18 of the
// sum) is left out.  With three parts (x = hi + mid + lo) it is hi.hi +
// 2 hi.mid + mid.mid + 2 hi.lo, four MFMAs; the terms left out (mid.lo,
// lo.lo) are at most 2^-24 of the sum.  Packed rows need fewer: the Gram
// product of the fragment (hi | lo) with itself holds hi.hi on its diagonal
// and hi.lo at (c, c + 8); that of (hi | mid) also holds mid.mid at (c + 8,
// c + 8), and (hi | mid) times (lo | 0) gives hi.lo on the diagonal.  The
// products themselves leave part 0 (and 2) of row c in accumulator column c
// and part 1 in column c + 8, which the epilogue adds.
// LDS floats the cross-wave reduction of stream_gemm_tiles needs.
template <int JT, int WAVES, int RT>
struct StreamRed {
  static constexpr int floats = WAVES > 1 ? (WAVES - 1) * JT * (4 * RT + 1) * 64 : 1;
};

// The two pipeline stages of a wave's stream (U K-blocks in flight).
template <class P, int JT, int RT, int U, bool PK>
using StreamStageOf = StreamStage<JT, RT, (U / 2 > 0 ? U / 2 : 1), StreamFrags<P, PK>::value>;

// Split-K across work-groups.  With more than 8 rows every work-group reads
// the whole activation of its K range, and O and down have only 256 tiles:
// one tile per work-group means each CU re-reads the full activation (at 32
// rows and two parts, four activation bytes per weight byte).  With S > 1
// the S work-groups of a group of RT tiles each take a contiguous 1/S of the
// K-blocks, so RT can be S times larger at the same work-group count and
// each activation fragment feeds RT weight fragments.  Each work-group
// publishes its partial sums (and the rows' partial sums of squares) with
// agent-coherent stores and counts itself in; the last to arrive adds the S
// partials in slice order -- the same order whichever arrives last, so the
// result stays bitwise reproducible -- and runs the epilogue.  No work-group
// waits on another.
struct SplitK {
  float* part;    // [group][slice][pair][64 lanes][2] floats
  int32_t* cnt;   // [group] arrived slices; zero between launches
};

// Floats each lane publishes per slice (accumulators, then sums of squares),
// rounded up to whole 8-byte pairs.
template <int JT, int RT, bool kNorm>
struct SplitKPairs {
  static constexpr int value = (RT * JT * 4 + (kNorm ? JT : 0) + 1) / 2;
};

// The body of k_stream_gemm as a device function: the WAVES waves of the
// calling work-group compute row tiles nt0 .. nt0 + RT - 1; red is LDS of
// StreamRed<JT, WAVES, RT>::floats floats.  With WAVES > 1 every wave of the
// work-group must call it (it synchronises the work-group).  s0, s1 are the
// pipeline stages.  PK: packed rows (n_rows <= 8, JT = 1, two or three parts).
// LP: parts per K-block of the activation record (at least P::parts; the
// first P::parts are used).
template <class P, int JT, int WAVES, class Epi, int RT, int U, bool kStream, bool PK, int LP = P::parts, int S = 1>
__device__ __forceinline__ void stream_gemm_tiles(const uint4* __restrict__ W, const uint4* __restrict__ X, int KB,
                                                  int Rp, int n_rows, const Epi& epi, int nt0, int wave, int lane,
                                                  float* red, StreamStageOf<P, JT, RT, U, PK>& s0,
                                                  StreamStageOf<P, JT, RT, U, PK>& s1, const SplitK& sk = {},
                                                  int slice = 0) {
  constexpr int PARTS = P::parts;
  static_assert(!PK || (JT == 1 && PARTS >= 2), "packed rows: one tile of at most 8 rows, two or three parts");
  static_assert(LP >= PARTS, "the record holds the parts used");
  static_assert(S == 1 || !PK, "split-K is for unpacked rows");
  constexpr int XF = StreamFrags<P, PK>::value;
  constexpr int UH = U / 2 > 0 ? U / 2 : 1;
  using Stage = StreamStageOf<P, JT, RT, U, PK>;
  // This work-group's K-blocks (its slice), split among its waves.
  const int ks0 = (KB * slice) / S, ks1 = (KB * (slice + 1)) / S;
  const int kb0 = ks0 + ((ks1 - ks0) * wave) / WAVES, kb1 = ks0 + ((ks1 - ks0) * (wave + 1)) / WAVES;
  // Gram accumulators per activation tile: hi.hi, then hi.lo (two parts) or
  // hi.mid, mid.mid, hi.lo (three parts); packed: (hi|lo)^2, or (hi|mid)^2
  // and (hi|mid).(lo|0).
  constexpr int NG = PK ? XF : PARTS == 3 ? 4 : PARTS;
  f32x4_t acc[RT][JT], gram[JT][NG];
#pragma unroll
  for (int j = 0; j < JT; ++j) {
#pragma unroll
    for (int t = 0; t < RT; ++t) acc[t][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < NG; ++i) gram[j][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }
  const uint4* wp = W + static_cast<size_t>(nt0) * KB * 64 + lane;
  const size_t wtile = static_cast<size_t>(KB) * 64;  // uint4 per row tile
  // This lane's uint4 offset within a K-block's activation record; fragment f
  // adds f * xstep.  Lanes of rows past n_rows read row 0 instead (the same
  // cache lines as a valid lane, so no extra traffic); their accumulator
  // columns are never stored, and MFMA columns do not mix, so the values they
  // read do not matter.  Packed: lane column c reads part 2 f + c / 8 of row
  // c % 8; for three parts, columns 8-15 of fragment 1 (part 3: the next
  // K-block's part 0, or past the last K-block's record, inside the buffer)
  // are zeroed after the load.
  const int xpart = Rp * 4;                  // uint4 per (K-block, part)
  const int xstep = PK ? 2 * xpart : xpart;  // uint4 between a lane's fragments
  int xoff[JT];
#pragma unroll
  for (int j = 0; j < JT; ++j) {
    if constexpr (PK) {
      const int c = lane & 15, r = c & 7;
      xoff[j] = (c >> 3) * xpart + (r < n_rows ? r : 0) * 4 + (lane >> 4);
    } else {
      const int b = 16 * j + (lane & 15);
      xoff[j] = (b < n_rows ? b : 0) * 4 + (lane >> 4);
    }
  }
  const bool zero_hi = PK && PARTS == 3 && (lane & 15) >= 8;  // packed (lo | 0): columns 8-15 are zero
  const size_t xblk = static_cast<size_t>(LP) * xpart;        // uint4 per K-block
  // Operands the epilogue reads from memory (residual, rotary table, block
  // table) are fetched now, by the wave that runs the epilogue, so their
  // latency hides under the weight stream instead of ending the kernel.
  typename Epi::Pre pre[RT];
  if (wave == 0) {
#pragma unroll
    for (int t = 0; t < RT; ++t) pre[t] = epi.template prefetch<JT>(nt0 + t, lane);
  }

  auto load1 = [&](Stage& st, int u, int kb) {
#pragma unroll
    for (int t = 0; t < RT; ++t) st.a[u][t] = load_weight<kStream>(wp + t * wtile + static_cast<size_t>(kb) * 64);
#pragma unroll
    for (int j = 0; j < JT; ++j)
#pragma unroll
      for (int f = 0; f < XF; ++f) st.x[u][j][f] = X[static_cast<size_t>(kb) * xblk + f * xstep + xoff[j]];
  };
  auto compute1 = [&](const Stage& st, int u) {
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      uint4 x[XF];
#pragma unroll
      for (int f = 0; f < XF; ++f) x[f] = st.x[u][j][f];
      if constexpr (PK && PARTS == 3) {
        x[1].x = zero_hi ? 0u : x[1].x;
        x[1].y = zero_hi ? 0u : x[1].y;
        x[1].z = zero_hi ? 0u : x[1].z;
        x[1].w = zero_hi ? 0u : x[1].w;
      }
#pragma unroll
      for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int f = 0; f < XF; ++f) acc[t][j] = P::mma(acc[t][j], st.a[u][t], x[f]);
      if constexpr (Epi::kNorm) {
        gram[j][0] = P::mma(gram[j][0], x[0], x[0]);
        if constexpr (PK) {
          if constexpr (XF == 2) gram[j][1] = P::mma(gram[j][1], x[0], x[1]);
        } else {
          if constexpr (PARTS >= 2) gram[j][1] = P::mma(gram[j][1], x[0], x[1]);
          if constexpr (PARTS == 3) {
            gram[j][2] = P::mma(gram[j][2], x[1], x[1]);
            gram[j][3] = P::mma(gram[j][3], x[0], x[2]);
          }
        }
      }
    }
  };
  auto load = [&](Stage& st, int kb) {
#pragma unroll
    for (int u = 0; u < UH; ++u) load1(st, u, kb + u);
  };
  auto compute = [&](const Stage& st) {
#pragma unroll
    for (int u = 0; u < UH; ++u) compute1(st, u);
  };

  const int nstage = (kb1 - kb0) / UH;
  if (nstage > 0) load(s0, kb0);
  for (int c = 0; c < nstage; c += 2) {
    if (c + 1 < nstage) load(s1, kb0 + (c + 1) * UH);
    compute(s0);
    if (c + 1 < nstage) {
      if (c + 2 < nstage) load(s0, kb0 + (c + 2) * UH);
      compute(s1);
    }
  }
  for (int kb = kb0 + nstage * UH; kb < kb1; ++kb) {
    load1(s0, 0, kb);
    compute1(s0, 0);
  }
  float ssq[JT];
#pragma unroll
  for (int j = 0; j < JT; ++j) {
    ssq[j] = 0.f;
    if constexpr (Epi::kNorm) {
      if constexpr (PK) {
        // Row c = lane column mod 8 (lanes of columns 8-15 compute row c's
        // again, unused).
        const int c = lane & 7;
        const float p0 = gram_pick(gram[j][0], lane);
        ssq[j] = gram_entry(p0, c, c);
        if constexpr (XF == 1) {
          ssq[j] += 2.f * gram_entry(p0, c, c + 8);
        } else {
          const float p1 = gram_pick(gram[j][1], lane);
          ssq[j] += 2.f * (gram_entry(p0, c, c + 8) + gram_entry(p1, c, c)) + gram_entry(p0, c + 8, c + 8);
        }
      } else {
        const int c = lane & 15;
        ssq[j] = gram_entry(gram_pick(gram[j][0], lane), c, c);
        if constexpr (PARTS == 2) ssq[j] += 2.f * gram_entry(gram_pick(gram[j][1], lane), c, c);
        if constexpr (PARTS == 3)
          ssq[j] += 2.f * (gram_entry(gram_pick(gram[j][1], lane), c, c) +
                           gram_entry(gram_pick(gram[j][3], lane), c, c)) +
                    gram_entry(gram_pick(gram[j][2], lane), c, c);
      }
    }
  }
  if constexpr (WAVES > 1) {
    // red[w - 1][j][4 t + c][lane], then the sums of squares at [.][j][4 RT][lane].
    auto at = [&](int w, int j, int i) -> float& { return red[((w * JT + j) * (4 * RT + 1) + i) * 64 + lane]; };
    if (wave > 0) {
#pragma unroll
      for (int j = 0; j < JT; ++j) {
#pragma unroll
        for (int t = 0; t < RT; ++t)
#pragma unroll
          for (int c = 0; c < 4; ++c) at(wave - 1, j, 4 * t + c) = acc[t][j][c];
        at(wave - 1, j, 4 * RT) = ssq[j];
      }
    }
    __syncthreads();
    if (wave != 0) return;
    for (int w = 0; w < WAVES - 1; ++w) {
#pragma unroll
      for (int j = 0; j < JT; ++j) {
#pragma unroll
        for (int t = 0; t < RT; ++t)
#pragma unroll
          for (int c = 0; c < 4; ++c) acc[t][j][c] += at(w, j, 4 * t + c);
        ssq[j] += at(w, j, 4 * RT);
      }
    }
  }
  if constexpr (S > 1) {
    // Publish this slice's partial, count it in; the last slice to arrive
    // sums all S in slice order and goes on to the epilogue.
    constexpr int NP = SplitKPairs<JT, RT, Epi::kNorm>::value;
    float v[2 * NP];
#pragma unroll
    for (int i = 0; i < 2 * NP; ++i) v[i] = 0.f;
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
      for (int j = 0; j < JT; ++j)
#pragma unroll
        for (int c = 0; c < 4; ++c) v[(t * JT + j) * 4 + c] = acc[t][j][c];
    if constexpr (Epi::kNorm) {
#pragma unroll
      for (int j = 0; j < JT; ++j) v[RT * JT * 4 + j] = ssq[j];
    }
    const int g = nt0 / RT;
    float* base = sk.part + static_cast<size_t>(g) * S * NP * 128 + 2 * lane;
#pragma unroll
    for (int i = 0; i < NP; ++i) store_coherent2(base + (static_cast<size_t>(slice) * NP + i) * 128, v[2 * i], v[2 * i + 1]);
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this slice's partial stores are complete
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    int last = 0;
    if (lane == 0) last = __hip_atomic_fetch_add(sk.cnt + g, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == S - 1;
    if (!__builtin_amdgcn_readfirstlane(last)) return;
    if (lane == 0) __hip_atomic_store(sk.cnt + g, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    float2 pv[S][NP];
#pragma unroll
    for (int q = 0; q < S; ++q)
#pragma unroll
      for (int i = 0; i < NP; ++i) pv[q][i] = load_coherent2(base + (static_cast<size_t>(q) * NP + i) * 128);
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      float2 a = pv[0][i];
#pragma unroll
      for (int q = 1; q < S; ++q) {
        a.x += pv[q][i].x;
        a.y += pv[q][i].y;
      }
      v[2 * i] = a.x;
      v[2 * i + 1] = a.y;
    }
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
      for (int j = 0; j < JT; ++j)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[t][j][c] = v[(t * JT + j) * 4 + c];
    if constexpr (Epi::kNorm) {
#pragma unroll
      for (int j = 0; j < JT; ++j) ssq[j] = v[RT * JT * 4 + j];
    }
  }
  if constexpr (PK) {
    // Row c's parts 0 (and 2) are in column c, part 1 in column c + 8.
    const int src = (lane & 48) | ((lane + 8) & 15);
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[t][0][c] += __shfl(acc[t][0][c], src);
  }
#pragma unroll
  for (int t = 0; t < RT; ++t) epi.template apply<JT>(nt0 + t, acc[t], ssq, lane, pre[t]);
}

template <class P, int JT, int WAVES, class Epi, int RT = 1, int U = StreamDepth<RT * JT * P::parts>::value,
          bool kStream = false, bool PK = false>
__global__ __launch_bounds__(WAVES * 64) void k_stream_gemm(const uint4* __restrict__ W, const uint4* __restrict__ X,
                                                            int KB, int Rp, int n_rows, Epi epi) {
  __shared__ float red[StreamRed<JT, WAVES, RT>::floats];
  StreamStageOf<P, JT, RT, U, PK> s0, s1;
  stream_gemm_tiles<P, JT, WAVES, Epi, RT, U, kStream, PK>(W, X, KB, Rp, n_rows, epi, blockIdx.x * RT,
                                                           __builtin_amdgcn_readfirstlane(threadIdx.x >> 6),
                                                           threadIdx.x & 63, red, s0, s1);
}

// k_stream_gemm with split-K across work-groups (see SplitK): work-group i
// takes slice i % S of group i / S, so the work-groups of one slice sit on
// the same XCDs (work-groups go to the XCDs round robin) and each XCD's L2
// holds only its slices' activations.
template <class P, int JT, int WAVES, class Epi, int RT, int U, int S>
__global__ __launch_bounds__(WAVES * 64) void k_stream_gemm_split(const uint4* __restrict__ W,
                                                                  const uint4* __restrict__ X, int KB, int Rp,
                                                                  int n_rows, Epi epi, SplitK sk) {
  __shared__ float red[StreamRed<JT, WAVES, RT>::floats];
  StreamStageOf<P, JT, RT, U, false> s0, s1;
  stream_gemm_tiles<P, JT, WAVES, Epi, RT, U, true, false, P::parts, S>(
      W, X, KB, Rp, n_rows, epi, (blockIdx.x / S) * RT, __builtin_amdgcn_readfirstlane(threadIdx.x >> 6),
      threadIdx.x & 63, red, s0, s1, sk, blockIdx.x % S);
}

// QKV projection of bf16 models over a three-part record: query tiles (the
// first q_tiles, a multiple of RT) take its first two parts -- hi and mid are
// the two-part form of the same values -- and key and value tiles, which are
// rounded into the bf16 cache, all three.  The branch is uniform per
// work-group.
// With S > 1, split-K across work-groups as in k_stream_gemm_split.
template <int JT, int WAVES, class Epi, int RT, int U2, int U3, bool PK, int S = 1>
__global__ __launch_bounds__(WAVES * 64) void k_stream_gemm_qkv(const uint4* __restrict__ W,
                                                                const uint4* __restrict__ X, int KB, int Rp,
                                                                int n_rows, Epi epi, int q_tiles, SplitK sk = {}) {
  __shared__ float red[StreamRed<JT, WAVES, RT>::floats];
  const int nt0 = (blockIdx.x / S) * RT, slice = blockIdx.x % S;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (nt0 < q_tiles) {
    StreamStageOf<BF16, JT, RT, U2, PK> s0, s1;
    stream_gemm_tiles<BF16, JT, WAVES, Epi, RT, U2, true, PK, 3, S>(W, X, KB, Rp, n_rows, epi, nt0, wave, lane, red,
                                                                    s0, s1, sk, slice);
  } else {
    StreamStageOf<BF16x3, JT, RT, U3, PK> s0, s1;
    stream_gemm_tiles<BF16x3, JT, WAVES, Epi, RT, U3, true, PK, 3, S>(W, X, KB, Rp, n_rows, epi, nt0, wave, lane,
                                                                      red, s0, s1, sk, slice);
  }
}

// Stores four consecutive features n0..n0+3 of row b into an activation buffer.
template <class P>
__device__ __forceinline__ void store_act4(typename P::elem* act, int Rp, int b, int n0, float v0, float v1, float v2,
                                           float v3) {
  act_store<P>(act, Rp, b, n0, v0);
  act_store<P>(act, Rp, b, n0 + 1, v1);
  act_store<P>(act, Rp, b, n0 + 2, v2);
  act_store<P>(act, Rp, b, n0 + 3, v3);
}

// QKV projection -> RMSNorm scale -> RoPE on q and k -> q to the attention
// input, k and v appended to the paged KV cache at the row's position.
// Per (block, KV head) the K tile is 16 positions x head_dim in MFMA fragment
// order (ktile_offset) and the V tile is transposed into the operand order of
// the P V product (vtile_offset), so the attention kernel reads both with
// 16-byte loads straight into MFMA operands.
template <class P, class KP = P>
struct EpiQKV {
  static constexpr bool kNorm = true;
  int n_rows, H, Hkv, hd, mb, dnorm;
  float eps;
  float* q;                     // [rows][H * hd]
  typename KP::elem* kc;        // this layer's K blocks (KV-cache format KP)
  typename KP::elem* vc;        // this layer's V blocks
  const int32_t* bt;            // [slots][mb]
  const float2* rope;           // [positions][hd / 2] (cos, sin)
  RowSlotPos rows;

  // Per row tile of a lane: the rotary (cos, sin) pairs of its four features
  // (q and k rows) and the KV block its position falls in (k and v rows).
  // Lanes of rows past n_rows fetch row 0's.
  struct Pre {
    float4 cs[kRows / 16];
    int blk[kRows / 16];
  };
  template <int JT>
  __device__ __forceinline__ Pre prefetch(int nt, int lane) const {
    Pre pr;
    const int n0 = 16 * nt + 4 * (lane >> 4);
    const int qr = H * hd, kr = Hkv * hd;
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      const int b = 16 * j + (lane & 15);
      const int bb = b < n_rows ? b : 0;
      const int p = rows.pos[bb];
      if (n0 < qr + kr) {
        const int dd = (n0 < qr ? n0 : n0 - qr) % hd;
        pr.cs[j] = *reinterpret_cast<const float4*>(rope + static_cast<size_t>(p) * (hd / 2) + dd / 2);
      }
      if (n0 >= qr) pr.blk[j] = bt[static_cast<size_t>(rows.slot[bb]) * mb + (p >> 4)];
    }
    return pr;
  }

  template <int JT>
  __device__ __forceinline__ void apply(int nt, const f32x4_t* acc, const float* ssq, int lane, const Pre& pr) const {
    const int n0 = 16 * nt + 4 * (lane >> 4);
    const int qr = H * hd, kr = Hkv * hd;
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      const int b = 16 * j + (lane & 15);
      if (b >= n_rows) continue;
      const float s = rsqrtf(ssq[j] / static_cast<float>(dnorm) + eps);
      float v0 = acc[j][0] * s, v1 = acc[j][1] * s, v2 = acc[j][2] * s, v3 = acc[j][3] * s;
      const int p = rows.pos[b];
      if (n0 < qr + kr) {
        const float2 c0 = make_float2(pr.cs[j].x, pr.cs[j].y), c1 = make_float2(pr.cs[j].z, pr.cs[j].w);
        const float a0 = v0 * c0.x - v1 * c0.y, a1 = v0 * c0.y + v1 * c0.x;
        const float a2 = v2 * c1.x - v3 * c1.y, a3 = v2 * c1.y + v3 * c1.x;
        v0 = a0;
        v1 = a1;
        v2 = a2;
        v3 = a3;
      }
      if (n0 < qr) {
        *reinterpret_cast<float4*>(q + static_cast<size_t>(b) * qr + n0) = make_float4(v0, v1, v2, v3);
        continue;
      }
      const int blk = pr.blk[j];
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
  }
};

// O and down projections: residual add, then the new residual in the
// activation format for the next projection.
template <class P>
struct EpiResid {
  static constexpr bool kNorm = false;
  int n_rows, d, Rp;
  float* x;                     // residual [rows][d]
  typename P::elem* act;        // next activation (K-block-major)

  // The residual values this lane updates (row 0's for rows past n_rows).
  // Each (row, feature) is read and written by one lane only.
  struct Pre {
    float4 x[kRows / 16];
  };
  template <int JT>
  __device__ __forceinline__ Pre prefetch(int nt, int lane) const {
    Pre pr;
    const int n0 = 16 * nt + 4 * (lane >> 4);
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      const int b = 16 * j + (lane & 15);
      const float* xp = x + static_cast<size_t>(b < n_rows ? b : 0) * d + n0;
      pr.x[j] = *reinterpret_cast<const float4*>(xp);
    }
    return pr;
  }

  template <int JT>
  __device__ __forceinline__ void apply(int nt, const f32x4_t* acc, const float*, int lane, const Pre& pr) const {
    const int n0 = 16 * nt + 4 * (lane >> 4);
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      const int b = 16 * j + (lane & 15);
      if (b >= n_rows) continue;
      float4* xp = reinterpret_cast<float4*>(x + static_cast<size_t>(b) * d + n0);
      float4 xv = pr.x[j];
      xv.x += acc[j][0];
      xv.y += acc[j][1];
      xv.z += acc[j][2];
      xv.w += acc[j][3];
      *xp = xv;
      store_act4<P>(act, Rp, b, n0, xv.x, xv.y, xv.z, xv.w);
    }
  }
};

// Gate/up projection (interleaved rows, see wgen_kernels.h): RMSNorm scale,
// then h = SiLU(gate) * up for two features per lane.
template <class P>
struct EpiSwiGLU {
  static constexpr bool kNorm = true;
  int n_rows, dnorm, Rp;
  float eps;
  typename P::elem* act;        // h, K-block-major over d_ff

  struct Pre {};
  template <int JT>
  __device__ __forceinline__ Pre prefetch(int, int) const {
    return {};
  }

  template <int JT>
  __device__ __forceinline__ void apply(int nt, const f32x4_t* acc, const float* ssq, int lane, const Pre&) const {
    const int j0 = 8 * nt + 2 * (lane >> 4);
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      const int b = 16 * j + (lane & 15);
      if (b >= n_rows) continue;
      const float s = rsqrtf(ssq[j] / static_cast<float>(dnorm) + eps);
      const float g0 = acc[j][0] * s, g1 = acc[j][1] * s, u0 = acc[j][2] * s, u1 = acc[j][3] * s;
      const float h0 = g0 / (1.f + __expf(-g0)) * u0;
      const float h1 = g1 / (1.f + __expf(-g1)) * u1;
      act_store<P>(act, Rp, b, j0, h0);
      act_store<P>(act, Rp, b, j0 + 1, h1);
    }
  }
};

// LM head: final RMSNorm scale, optional fp32 logits, and the per-tile greedy
// candidate (largest logit, lowest index on ties) of each row.
template <class P>
struct EpiLogits {
  static constexpr bool kNorm = true;
  int n_rows, V, dnorm;
  float eps;
  float* logits;                // [out_row][V] or null
  float2* part;                 // [tiles][kRows] (value, index bits)
  int out_row[kRows];           // logits row of each token row, -1 = none

  struct Pre {};
  template <int JT>
  __device__ __forceinline__ Pre prefetch(int, int) const {
    return {};
  }

  template <int JT>
  __device__ __forceinline__ void apply(int nt, const f32x4_t* acc, const float* ssq, int lane, const Pre&) const {
    const int n0 = 16 * nt + 4 * (lane >> 4);
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      const int b = 16 * j + (lane & 15);
      const bool vb = b < n_rows;
      const float s = rsqrtf(ssq[j] / static_cast<float>(dnorm) + eps);
      float best = -INFINITY;
      int bi = 0x7fffffff;
      int nan = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float z = acc[j][i] * s;
        const int n = n0 + i;
        if (n < V && z > best) {
          best = z;
          bi = n;
        }
        nan |= n < V && z != z;
        if (vb && logits != nullptr && n < V && out_row[b] >= 0) logits[static_cast<size_t>(out_row[b]) * V + n] = z;
      }
#pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        const float ob = __shfl_xor(best, o);
        const int oi = __shfl_xor(bi, o);
        nan |= __shfl_xor(nan, o);
        if (ob > best || (ob == best && oi < bi)) {
          best = ob;
          bi = oi;
        }
      }
      // A NaN logit makes the tile's candidate value NaN (k_argmax_final reports it).
      if ((lane >> 4) == 0 && vb)
        part[static_cast<size_t>(nt) * kRows + b] = make_float2(nan ? __int_as_float(0x7fc00000) : best, __int_as_float(bi));
    }
  }
};

}  // namespace sprk
