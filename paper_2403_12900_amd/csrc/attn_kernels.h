// Decode attention over the paged KV cache, one query position per row
// (Section II-A: each new token attends to the cached keys and values of all
// earlier tokens of its request, the directive prefix included).
//
// Work item = (row, KV split, KV head).  A workgroup of four waves covers the
// 16-position blocks of its split, each wave a contiguous run of bpw blocks.
// Per block, on MFMA:
//   S[t][h]  = K_tile(16 x hd) . Q^T(hd x 16)      -- t = position, h = query
//              head of the KV group (G <= 16 columns used; grouped-query heads
//              share the K/V tile they read once)
//   online softmax over t (column-wise max with wavefront shuffles, exp2 of
//   log2e-scaled scores)
//   O^T[e][h] += V^T_tile(hd x 16) . P(16 x 16)   -- P is the S accumulator
//              re-used in place as the B operand: no shuffle, no LDS
// The four waves are merged through LDS (log-sum-exp), each wave combining a
// quarter of the head dimensions.  A row whose context needs one split writes
// its output directly; otherwise each split publishes a partial (max, sum,
// unnormalised output) and counts itself in, and the split that arrives last
// merges them all (one launch; no work-group ever waits on another).  The
// grid holds only (row, split) pairs with work.
// bf16 keys are multiplied by q split into hi + lo bf16 parts, so the scores
// carry fp32-level precision of q.
#pragma once

#include "gemm_kernels.h"

namespace sprk {

struct AttnArgs {
  const float* q;         // [rows][H][hd], fp32
  const void* kc;         // this layer's K blocks [block][Hkv][16 x hd, ktile_offset order]
  const void* vc;         // this layer's V blocks [block][Hkv][16 x hd, vtile_offset order]
  const int32_t* bt;      // [slots][mb]
  void* act;              // output, K-block-major over H * hd
  float* part;            // [flat split][H][hd + 4]: m, l, -, -, o[hd]
  int32_t* cnt;           // [rows][Hkv] arrived splits; zero between launches
  int n_rows, H, Hkv, G, mb, bpw, Rp;
  float qscale;           // log2(e) / sqrt(hd)
  RowSlotPos rows;
  int split_start[kRows + 1];  // first flat split index of each row; [n_rows] = total
};

// Partials the last arriving split reads per round; the host keeps every
// row's split count within one round.
constexpr int kMergeChunk = 16;

template <class AP, int HD>
__device__ __forceinline__ void merge_splits(const AttnArgs& a, int b, int kvh, int f0, int ns);

// K and V of one 16-position block of one KV head, in registers: NF K
// operands and NV 16-byte V loads (two bf16 V^T operands or one fp32 operand
// each, see vtile_offset).  Each cached byte is read once per step, so the
// loads are streaming (nontemporal).
template <class P, int HD>
struct KVBlock {
  using E = typename P::elem;
  static constexpr int NF = HD / P::kblk;
  static constexpr int NV = HD * 16 * static_cast<int>(sizeof(E)) / 1024;
  uint4 kf[NF];
  uint4 vf[NV];

  __device__ __forceinline__ void load(const E* kc, const E* vc, size_t tile, int lane) {
    const uint4* kt = reinterpret_cast<const uint4*>(kc + tile * 16 * HD) + lane;
    const uint4* vt = reinterpret_cast<const uint4*>(vc + tile * 16 * HD) + lane;
#pragma unroll
    for (int f = 0; f < NF; ++f) kf[f] = load_weight<true>(kt + f * 64);
#pragma unroll
    for (int v = 0; v < NV; ++v) vf[v] = load_weight<true>(vt + v * 64);
  }

  // Positions past the context hold stale or never-written cache memory; they
  // get probability 0, but 0 * NaN would still poison the sum, so zero them.
  // `valid` = positions of this lane's four (4 g .. 4 g + 3) that are in context.
  __device__ __forceinline__ void mask_v(int valid) {
    if constexpr (sizeof(E) == 2) {
      const uint32_t m01 = valid >= 2 ? 0xFFFFFFFFu : valid == 1 ? 0xFFFFu : 0u;
      const uint32_t m23 = valid >= 4 ? 0xFFFFFFFFu : valid == 3 ? 0xFFFFu : 0u;
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        vf[v].x &= m01;
        vf[v].y &= m23;
        vf[v].z &= m01;
        vf[v].w &= m23;
      }
    } else {
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        vf[v].x = valid >= 1 ? vf[v].x : 0u;
        vf[v].y = valid >= 2 ? vf[v].y : 0u;
        vf[v].z = valid >= 3 ? vf[v].z : 0u;
        vf[v].w = valid >= 4 ? vf[v].w : 0u;
      }
    }
  }

  // O[e] (16 dims x 16 heads) += V^T(16 dims x 16 positions) . P(16 positions
  // x 16 heads), P given as this lane's four probabilities.  bf16: the
  // probabilities go in as hi + lo parts (two MFMAs per operand).
  __device__ __forceinline__ void pv(f32x4_t* O, const float* p) const {
    if constexpr (sizeof(E) == 2) {
      s16x4_t bh, bl;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const uint16_t h = f32_to_bf16_bits(p[r]);
        bh[r] = static_cast<short>(h);
        bl[r] = static_cast<short>(f32_to_bf16_bits(p[r] - bf16_bits_to_f32(h)));
      }
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const s16x4_t a0 = __builtin_bit_cast(s16x4_t, make_uint2(vf[v].x, vf[v].y));
        const s16x4_t a1 = __builtin_bit_cast(s16x4_t, make_uint2(vf[v].z, vf[v].w));
        O[2 * v] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a0, bh, O[2 * v], 0, 0, 0);
        O[2 * v] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a0, bl, O[2 * v], 0, 0, 0);
        O[2 * v + 1] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a1, bh, O[2 * v + 1], 0, 0, 0);
        O[2 * v + 1] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a1, bl, O[2 * v + 1], 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        O[v] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(vf[v].x), p[0], O[v], 0, 0, 0);
        O[v] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(vf[v].y), p[1], O[v], 0, 0, 0);
        O[v] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(vf[v].z), p[2], O[v], 0, 0, 0);
        O[v] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(vf[v].w), p[3], O[v], 0, 0, 0);
      }
    }
  }
};

// P is the KV-cache storage format (it also sets the MFMA operand type of q
// and of the probabilities); AP is the format of the output activation.
// Work-group (flat split f, KV head): row b and split s of f; blocks [s * 4
// bpw, min(nblk, (s + 1) * 4 bpw)); wave w takes the run of bpw blocks from
// s * 4 bpw + w * bpw.  A wave walks its blocks one at a time -- load K and
// V, scores, online-softmax update, P V -- with few registers, so that
// several waves per SIMD hide each other's memory latency (measured faster on
// MI355X than keeping two blocks in flight per wave at lower occupancy); the
// block ids of its run come in one vector load up front, so each block costs
// one memory round trip.  Branch conditions are wave-uniform; the partial
// last block of the context is masked by selects.
// LDS of one attention work item: the four waves' outputs and (max, sum).
template <int HD>
struct AttnSmem {
  f32x4_t so[4][HD / 16][64];
  float2 sml[4][64];
  int last;
};

// The body of k_attn_decode for work item (flat split f, KV head kvh), run by
// all four waves of the calling work-group.
template <class P, class AP, int HD>
__device__ __forceinline__ void attn_decode_unit(const AttnArgs& a, int f, int kvh, AttnSmem<HD>* sm) {
  using E = typename P::elem;
  using Blk = KVBlock<P, HD>;
  constexpr bool kBf16 = sizeof(E) == 2;
  constexpr int NF = Blk::NF;
  constexpr int NE = HD / 16;     // output operands (16 dims each)
  constexpr int EPW = NE / 4;     // output operands each wave merges and stores
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // Row of this work-group = number of rows whose splits all precede f (the
  // split starts increase), counted with one ballot per 64 rows.
  int b = 0;
  for (int r0 = 0; r0 < a.n_rows - 1; r0 += 64) {
    const int r = r0 + lane;
    b += __popcll(__ballot(r < a.n_rows - 1 && a.split_start[r + 1] <= f));
  }
  b = __builtin_amdgcn_readfirstlane(b);
  const int s = f - a.split_start[b];
  const int nsplit = a.split_start[b + 1] - a.split_start[b];
  const int pos = a.rows.pos[b];
  const int ctx = pos + 1;
  const int nblk = (ctx + 15) >> 4;
  const int h = lane & 15, g = lane >> 4;
  const bool hv = h < a.G;
  const int bpw = a.bpw;
  const int lo = min(nblk, (4 * s + wave) * bpw), hi = min(nblk, (4 * s + wave + 1) * bpw);
  const int32_t* btrow = a.bt + static_cast<size_t>(a.rows.slot[b]) * a.mb;
  int ids = lo + lane < hi ? btrow[lo + lane] : 0;  // block ids of the next 64 blocks of the run

  // Q^T operand (hi and lo parts for bf16), scaled so scores are in log2
  // units; fragment c, lane h + 16 g holds dims c * kblk + g * per16 + j,
  // matching the K tile order.
  // Lanes of padding columns (h >= G) read head kvh * G's q (a valid
  // address, so the loads are unconditional and vectorised) and zero it.
  uint4 qh[NF], ql[NF];
  {
    const float* qp = a.q + (static_cast<size_t>(b) * a.H + kvh * a.G + (hv ? h : 0)) * HD + g * P::per16;
    float4 qv[NF][P::per16 / 4];
#pragma unroll
    for (int c = 0; c < NF; ++c)
#pragma unroll
      for (int j4 = 0; j4 < P::per16 / 4; ++j4) qv[c][j4] = *reinterpret_cast<const float4*>(qp + c * P::kblk + 4 * j4);
    const float qs = hv ? a.qscale : 0.f;
#pragma unroll
    for (int c = 0; c < NF; ++c) {
      union {
        uint4 u;
        E e[P::per16];
      } vh, vl;
#pragma unroll
      for (int j = 0; j < P::per16; ++j) {
        const float4 t = qv[c][j / 4];
        const float v = (j % 4 == 0 ? t.x : j % 4 == 1 ? t.y : j % 4 == 2 ? t.z : t.w) * qs;
        vh.e[j] = P::from_f32(v);
        vl.e[j] = P::from_f32(v - P::to_f32(vh.e[j]));
      }
      qh[c] = vh.u;
      ql[c] = vl.u;
    }
  }

  f32x4_t O[NE];
#pragma unroll
  for (int e = 0; e < NE; ++e) O[e] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  const E* kc = static_cast<const E*>(a.kc);
  const E* vc = static_cast<const E*>(a.vc);

  for (int i = lo; i < hi; ++i) {
    const int k = i - lo;
    if ((k & 63) == 0 && k != 0) ids = i + lane < hi ? btrow[i + lane] : 0;
    Blk B;
    B.load(kc, vc, static_cast<size_t>(__builtin_amdgcn_readlane(ids, k & 63)) * a.Hkv + kvh, lane);
    f32x4_t S = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NF; ++c) {
      S = P::mma(S, B.kf[c], qh[c]);
      if constexpr (kBf16) S = P::mma(S, B.kf[c], ql[c]);
    }
    if (i == nblk - 1) {  // the block holding the context's last position
      const int valid = ctx - (i * 16 + 4 * g);
#pragma unroll
      for (int r = 0; r < 4; ++r) S[r] = r < valid ? S[r] : -INFINITY;
      B.mask_v(valid);
    }
    float mb = fmaxf(fmaxf(S[0], S[1]), fmaxf(S[2], S[3]));
    mb = fmaxf(mb, __shfl_xor(mb, 16));
    mb = fmaxf(mb, __shfl_xor(mb, 32));
    const float m_new = fmaxf(m_run, mb);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    float p[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) p[r] = __builtin_amdgcn_exp2f(S[r] - m_new);
    l_run = l_run * alpha + ((p[0] + p[1]) + (p[2] + p[3]));
    // O is still zero at the first block; later, rescale only if some
    // column's running maximum moved (alpha == 1 elsewhere).
    if (i != lo && __ballot(m_new != m_run) != 0) {
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
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);

  // Log-sum-exp merge of the four waves; wave w combines and stores output
  // operands [w * EPW, (w + 1) * EPW).  Wave 0 always holds at least one
  // block (its run starts the split), so M is finite; waves without blocks
  // carry m = -inf and weigh 0.
  sm->sml[wave][lane] = make_float2(m_run, l_run);
#pragma unroll
  for (int e = 0; e < NE; ++e) sm->so[wave][e][lane] = O[e];
  __syncthreads();
  float2 ml[4];
  float M = -INFINITY;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    ml[w] = sm->sml[w][lane];
    M = fmaxf(M, ml[w].x);
  }
  float cw[4], L = 0.f;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    cw[w] = __builtin_amdgcn_exp2f(ml[w].x - M);
    L += cw[w] * ml[w].y;
  }
  f32x4_t R[EPW];
#pragma unroll
  for (int k = 0; k < EPW; ++k) {
    R[k] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const f32x4_t o = sm->so[w][wave * EPW + k][lane];
#pragma unroll
      for (int r = 0; r < 4; ++r) R[k][r] += cw[w] * o[r];
    }
  }
  const int hq = kvh * a.G + h;
  if (nsplit == 1) {
    if (!hv) return;
    const float inv = 1.f / L;
    typename AP::elem* act = static_cast<typename AP::elem*>(a.act);
#pragma unroll
    for (int k = 0; k < EPW; ++k) {
      const int n0 = hq * HD + 16 * (wave * EPW + k) + 4 * g;
      store_act4<AP>(act, a.Rp, b, n0, R[k][0] * inv, R[k][1] * inv, R[k][2] * inv, R[k][3] * inv);
    }
    return;
  }
  // Several splits: publish this split's partial, then count it in.  Each
  // partial is written with agent-coherent stores and completed (vmcnt 0)
  // before the work-group's arrival is counted, so whichever split arrives
  // last reads every partial with agent-coherent loads: no cache write-back
  // and no wait on another work-group.
  if (hv) {
    float* pp = a.part + (static_cast<size_t>(f) * a.H + hq) * (HD + 4);
    if (wave == 0 && g == 0) store_coherent2(pp, M, L);
#pragma unroll
    for (int k = 0; k < EPW; ++k) {
      float* o = pp + 4 + 16 * (wave * EPW + k) + 4 * g;
      store_coherent2(o, R[k][0], R[k][1]);
      store_coherent2(o + 2, R[k][2], R[k][3]);
    }
  }
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's partial stores are complete
  __syncthreads();
  int32_t* cnt = a.cnt + b * a.Hkv + kvh;
  if (threadIdx.x == 0)
    sm->last = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == nsplit - 1;
  __syncthreads();
  if (!sm->last) return;
  if (threadIdx.x == 0) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  merge_splits<AP, HD>(a, b, kvh, a.split_start[b], nsplit);
}

// Grid (KV heads, flat splits): consecutive work-groups take the KV heads of
// one split, so the ones resident together read neighbouring tiles of the
// same blocks (measured 0.5% faster on the ragged 7B decode than splits
// first).
template <class P, class AP, int HD>
__global__ __launch_bounds__(256) void k_attn_decode(AttnArgs a) {
  __shared__ AttnSmem<HD> sm;
  attn_decode_unit<P, AP, HD>(a, blockIdx.y, blockIdx.x, &sm);
}

// Log-sum-exp merge of the nsplit partials of one (row, KV head), run by the
// split that arrived last.  Splits are taken kChunk at a time, all of a
// chunk's loads issued before any is combined (indexes past the last split
// re-read it and are then ignored).
template <class AP, int HD>
__device__ __forceinline__ void merge_splits(const AttnArgs& a, int b, int kvh, int f0, int ns) {
  constexpr int kChunk = kMergeChunk;
  typename AP::elem* act = static_cast<typename AP::elem*>(a.act);
  const size_t stride = static_cast<size_t>(a.H) * (HD + 4);
  for (int idx = threadIdx.x; idx < a.G * HD; idx += 256) {
    const int hq = kvh * a.G + idx / HD, dd = idx % HD;
    const float* pp = a.part + (static_cast<size_t>(f0) * a.H + hq) * (HD + 4);
    float M = -INFINITY, L = 0.f, Ov = 0.f;
    for (int t0 = 0; t0 < ns; t0 += kChunk) {
      float m[kChunk], l[kChunk], o[kChunk];
#pragma unroll
      for (int k = 0; k < kChunk; ++k) {
        const float* pt = pp + static_cast<size_t>(min(t0 + k, ns - 1)) * stride;
        const float2 ml = load_coherent2(pt);
        m[k] = ml.x;
        l[k] = ml.y;
        o[k] = __hip_atomic_load(pt + 4 + dd, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      float Mn = M;
#pragma unroll
      for (int k = 0; k < kChunk; ++k) Mn = t0 + k < ns ? fmaxf(Mn, m[k]) : Mn;
      const float sc = __builtin_amdgcn_exp2f(M - Mn);  // 0 while M = -inf
      L *= sc;
      Ov *= sc;
#pragma unroll
      for (int k = 0; k < kChunk; ++k) {
        const float c = t0 + k < ns ? __builtin_amdgcn_exp2f(m[k] - Mn) : 0.f;
        L += c * l[k];
        Ov += c * o[k];
      }
      M = Mn;
    }
    act_store<AP>(act, a.Rp, b, hq * HD + dd, Ov / L);
  }
}

}  // namespace sprk
