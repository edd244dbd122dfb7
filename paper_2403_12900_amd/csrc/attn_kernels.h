// Decode attention over the paged KV cache, one query position per row
// (Section II-A: each new token attends to the cached keys and values of all
// earlier tokens of its request, the directive prefix included).
//
// Work item = (row, KV split, KV head).  A workgroup of four waves walks the
// 16-position blocks of its split, wave w taking every fourth block.  Per
// block, on MFMA:
//   S[t][h]  = K_tile(16 x hd) . Q^T(hd x 16)      -- t = position, h = query
//              head of the KV group (G <= 16 columns used; grouped-query heads
//              share the K/V tile they read once)
//   online softmax over t (column-wise max with wavefront shuffles, exp2 of
//   log2e-scaled scores)
//   O^T[e][h] += V^T_tile(hd x 16) . P(16 x 16)   -- P is the S accumulator
//              re-used in place as the B operand: no shuffle, no LDS
// The four waves are merged through LDS (log-sum-exp).  A row whose context
// needs one split writes its output directly; otherwise each split writes a
// partial (max, sum, unnormalised output) and k_attn_merge combines them.
// The grid holds only (row, split) pairs with work.
// bf16 keys are multiplied by q split into hi + lo bf16 parts, so the scores
// carry fp32-level precision of q.
#pragma once

#include "gemm_kernels.h"

namespace sprk {

struct AttnArgs {
  const float* q;         // [rows][H][hd], fp32
  const void* kc;         // this layer's K blocks [block][Hkv][16 x hd in fragment order]
  const void* vc;         // this layer's V blocks [block][Hkv][hd][16]
  const int32_t* bt;      // [slots][mb]
  void* act;              // output, K-block-major over H * hd
  float* part;            // [rows][H][kSplitsMax][hd + 4]: m, l, -, -, o[hd]
  int n_rows, H, Hkv, G, mb, bps, Rp;
  float qscale;           // log2(e) / sqrt(hd)
  RowSlotPos rows;
  int split_start[kRows + 1];  // first flat split index of each row; [n_rows] = total
};

// Four consecutive positions of one V^T row (one dimension), as loaded.
template <class P>
struct VQuad;
template <>
struct VQuad<BF16> {
  uint2 raw;
  __device__ __forceinline__ void load(const uint16_t* v) {
    typedef unsigned int u2v __attribute__((ext_vector_type(2)));
    const u2v t = __builtin_nontemporal_load(reinterpret_cast<const u2v*>(v));
    raw = make_uint2(t.x, t.y);
  }
  // Positions past the context hold stale or never-written cache memory; they
  // get probability 0, but 0 * NaN would still poison the sum, so zero them.
  __device__ __forceinline__ void mask(int valid) {
    raw.x &= valid >= 2 ? 0xFFFFFFFFu : valid == 1 ? 0xFFFFu : 0u;
    raw.y &= valid >= 4 ? 0xFFFFFFFFu : valid == 3 ? 0xFFFFu : 0u;
  }
};
template <>
struct VQuad<F32> {
  uint4 raw;
  __device__ __forceinline__ void load(const float* v) { raw = load_weight<true>(reinterpret_cast<const uint4*>(v)); }
  __device__ __forceinline__ void mask(int valid) {
    raw.x = valid >= 1 ? raw.x : 0u;
    raw.y = valid >= 2 ? raw.y : 0u;
    raw.z = valid >= 3 ? raw.z : 0u;
    raw.w = valid >= 4 ? raw.w : 0u;
  }
};

// acc(16 dims x 16 heads) += V^T(16 dims x 16 positions) . P(16 positions x 16 heads).
// bf16: the probabilities go in as hi + lo parts (two MFMAs).
__device__ __forceinline__ f32x4_t mma_tok16(f32x4_t acc, const VQuad<BF16>& v, const float* p) {
  const s16x4_t a = __builtin_bit_cast(s16x4_t, v.raw);
  s16x4_t bh, bl;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const uint16_t h = f32_to_bf16_bits(p[r]);
    bh[r] = static_cast<short>(h);
    bl[r] = static_cast<short>(f32_to_bf16_bits(p[r] - bf16_bits_to_f32(h)));
  }
  acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, bh, acc, 0, 0, 0);
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, bl, acc, 0, 0, 0);
}

__device__ __forceinline__ f32x4_t mma_tok16(f32x4_t acc, const VQuad<F32>& v, const float* p) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(v.raw.x), p[0], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(v.raw.y), p[1], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(v.raw.z), p[2], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(v.raw.w), p[3], acc, 0, 0, 0);
  return acc;
}

// K and V of one 16-position block of one KV head, in registers.  Each cached
// byte is read once per step, so the loads are streaming (nontemporal).
template <class P, int HD>
struct KVBlock {
  using E = typename P::elem;
  static constexpr int NF = HD / P::kblk;  // K fragments (1 KiB each)
  static constexpr int NE = HD / 16;       // V^T fragments, 16 dims each
  uint4 kf[NF];
  VQuad<P> vq[NE];

  __device__ __forceinline__ void load(const E* kc, const E* vc, size_t tile, int lane) {
    const uint4* kt = reinterpret_cast<const uint4*>(kc + tile * 16 * HD) + lane;
#pragma unroll
    for (int f = 0; f < NF; ++f) kf[f] = load_weight<true>(kt + f * 64);
    const E* vt = vc + (tile * HD + (lane & 15)) * 16 + 4 * (lane >> 4);
#pragma unroll
    for (int e = 0; e < NE; ++e) vq[e].load(vt + e * 16 * 16);
  }
};

// P is the KV-cache storage format (it also sets the MFMA operand type of q
// and of the probabilities); AP is the format of the output activation.
// Work-group (split s, row b, KV head): blocks [s * bps, min(nblk, (s + 1) *
// bps)); wave w takes the contiguous run of bps / 4 blocks starting at
// w * bps / 4.  A wave walks its blocks one at a time -- load K and V, scores,
// online-softmax update, P V -- with few registers, so that several waves per
// SIMD hide each other's memory latency (measured faster on MI355X than
// keeping two blocks in flight per wave at lower occupancy).  Branch
// conditions are wave-uniform; the partial last block of the context is
// masked by selects.
template <class P, class AP, int HD>
__global__ __launch_bounds__(256) void k_attn_decode(AttnArgs a) {
  using E = typename P::elem;
  using Blk = KVBlock<P, HD>;
  constexpr bool kBf16 = sizeof(E) == 2;
  constexpr int NF = Blk::NF;
  constexpr int NE = Blk::NE;
  // Flat grid over the (row, split) pairs that have work: find this
  // work-group's row by binary search over the rows' first split index.
  const int f = blockIdx.x, kvh = blockIdx.y;
  int lo_r = 0, hi_r = a.n_rows - 1;
  while (lo_r < hi_r) {  // first row whose splits end after f
    const int mid = (lo_r + hi_r) >> 1;
    if (a.split_start[mid + 1] <= f) {
      lo_r = mid + 1;
    } else {
      hi_r = mid;
    }
  }
  const int b = lo_r;
  const int s = f - a.split_start[b];
  const int nsplit = a.split_start[b + 1] - a.split_start[b];
  const int pos = a.rows.pos[b];
  const int ctx = pos + 1;
  const int nblk = (ctx + 15) >> 4;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int h = lane & 15, g = lane >> 4;
  const bool hv = h < a.G;
  const int bpw = a.bps / 4;
  const int lo = min(nblk, s * a.bps + wave * bpw), hi = min(nblk, s * a.bps + (wave + 1) * bpw);
  const int32_t* btrow = a.bt + static_cast<size_t>(a.rows.slot[b]) * a.mb;

  // Q^T operand (hi and lo parts for bf16), scaled so scores are in log2
  // units; fragment c, lane h + 16 g holds dims c * kblk + g * per16 + j,
  // matching the K tile order.
  uint4 qh[NF], ql[NF];
  {
    const float* qp = a.q + (static_cast<size_t>(b) * a.H + kvh * a.G + (hv ? h : 0)) * HD + g * P::per16;
#pragma unroll
    for (int c = 0; c < NF; ++c) {
      union {
        uint4 u;
        E e[P::per16];
      } vh, vl;
#pragma unroll
      for (int j = 0; j < P::per16; ++j) {
        const float v = hv ? qp[c * P::kblk + j] * a.qscale : 0.f;
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
    Blk B;
    B.load(kc, vc, static_cast<size_t>(btrow[i]) * a.Hkv + kvh, lane);
    f32x4_t S = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      S = P::mma(S, B.kf[f], qh[f]);
      if constexpr (kBf16) S = P::mma(S, B.kf[f], ql[f]);
    }
    if (i == nblk - 1) {  // the block holding the context's last position
      const int valid = ctx - (i * 16 + 4 * g);
#pragma unroll
      for (int r = 0; r < 4; ++r) S[r] = r < valid ? S[r] : -INFINITY;
#pragma unroll
      for (int e = 0; e < NE; ++e) B.vq[e].mask(valid);
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
    m_run = m_new;
#pragma unroll
    for (int e = 0; e < NE; ++e) {
      O[e][0] *= alpha;
      O[e][1] *= alpha;
      O[e][2] *= alpha;
      O[e][3] *= alpha;
      O[e] = mma_tok16(O[e], B.vq[e], p);
    }
  }
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);

  __shared__ float sm[3][2 + 4 * NE][64];
  if (wave > 0) {
    sm[wave - 1][0][lane] = m_run;
    sm[wave - 1][1][lane] = l_run;
#pragma unroll
    for (int e = 0; e < NE; ++e)
#pragma unroll
      for (int r = 0; r < 4; ++r) sm[wave - 1][2 + 4 * e + r][lane] = O[e][r];
  }
  __syncthreads();
  const int hq = kvh * a.G + h;
  if (wave == 0) {
    // Wave 0 always holds at least one block (lo < nblk for s < nsplit), so
    // M is finite; waves without blocks carry m = -inf and weigh 0.
    float M = m_run;
    for (int w = 0; w < 3; ++w) M = fmaxf(M, sm[w][0][lane]);
    const float c0 = __builtin_amdgcn_exp2f(m_run - M);
    float L = l_run * c0;
#pragma unroll
    for (int e = 0; e < NE; ++e)
#pragma unroll
      for (int r = 0; r < 4; ++r) O[e][r] *= c0;
    for (int w = 0; w < 3; ++w) {
      const float cw = __builtin_amdgcn_exp2f(sm[w][0][lane] - M);
      L += cw * sm[w][1][lane];
#pragma unroll
      for (int e = 0; e < NE; ++e)
#pragma unroll
        for (int r = 0; r < 4; ++r) O[e][r] += cw * sm[w][2 + 4 * e + r][lane];
    }
    if (hv) {
      if (nsplit == 1) {
        const float inv = 1.f / L;
        typename AP::elem* act = static_cast<typename AP::elem*>(a.act);
#pragma unroll
        for (int e = 0; e < NE; ++e)
          store_act4<AP>(act, a.Rp, b, hq * HD + 16 * e + 4 * g, O[e][0] * inv, O[e][1] * inv, O[e][2] * inv,
                         O[e][3] * inv);
      } else {
        float* pp = a.part + ((static_cast<size_t>(b) * a.H + hq) * kSplitsMax + s) * (HD + 4);
        if (g == 0) {
          pp[0] = M;
          pp[1] = L;
        }
#pragma unroll
        for (int e = 0; e < NE; ++e)
          *reinterpret_cast<float4*>(pp + 4 + 16 * e + 4 * g) = make_float4(O[e][0], O[e][1], O[e][2], O[e][3]);
      }
    }
  }
}

// Log-sum-exp merge of the KV splits of one (row, KV head), for rows whose
// context needed more than one split; all splits' statistics and values are
// loaded before any is combined.  (A last-arriving split could merge instead
// of a second launch, but the device-scope release that needs -- a write-back
// of the XCD's L2 by every split -- measured ten times slower on MI355X.)
template <class AP, int HD>
__global__ __launch_bounds__(256) void k_attn_merge(AttnArgs a) {
  const int b = blockIdx.x, kvh = blockIdx.y;
  const int nsplit = a.split_start[b + 1] - a.split_start[b];
  if (nsplit <= 1) return;
  typename AP::elem* act = static_cast<typename AP::elem*>(a.act);
  for (int idx = threadIdx.x; idx < a.G * HD; idx += 256) {
    const int hm = kvh * a.G + idx / HD, dd = idx % HD;
    const float* pp = a.part + (static_cast<size_t>(b) * a.H + hm) * kSplitsMax * (HD + 4);
    float m[kSplitsMax], l[kSplitsMax], o[kSplitsMax];
#pragma unroll
    for (int t = 0; t < kSplitsMax; ++t) {
      const bool v = t < nsplit;
      m[t] = v ? pp[t * (HD + 4)] : -INFINITY;
      l[t] = v ? pp[t * (HD + 4) + 1] : 0.f;
      o[t] = v ? pp[t * (HD + 4) + 4 + dd] : 0.f;
    }
    float M = m[0];
#pragma unroll
    for (int t = 1; t < kSplitsMax; ++t) M = fmaxf(M, m[t]);
    float L = 0.f, Ov = 0.f;
#pragma unroll
    for (int t = 0; t < kSplitsMax; ++t) {
      const float c = __builtin_amdgcn_exp2f(m[t] - M);
      L += c * l[t];
      Ov += c * o[t];
    }
    act_store<AP>(act, a.Rp, b, hm * HD + dd, Ov / L);
  }
}

}  // namespace sprk
