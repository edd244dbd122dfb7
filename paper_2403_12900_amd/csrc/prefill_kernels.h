// Prefill: the prompt of every new request runs through the model in chunks
// of up to kPrefillRows token rows, filling the KV cache (Section II-A: the
// prompt's keys and values are computed once and cached; generation follows).
// Unlike decode, each weight byte now meets hundreds of rows, so the
// projections are compute-bound: a tiled MFMA GEMM stages 128 x 128 output
// tiles through LDS.  Attention is causal over each request's own positions;
// a wave's 16 MFMA columns are 16 consecutive query positions of one request
// and head, so every K/V tile read feeds 16 queries.
#pragma once

#include "attn_kernels.h"

namespace sprk {

constexpr int kPrefillRows = 1024;  // token rows per prefill chunk

// One token row of a chunk.
struct PrefillRow {
  int slot, pos, tok, pad;
};

// Up to 16 consecutive rows of one request (positions pos0 .. pos0 + n - 1
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

// Tiled projection: out[b][n] = sum_k W[n][k] x[b][k] for rows b < M, fused
// with the op that follows (Epi).  Work-group = 128 output features (8 weight
// tiles) x 128 rows; per K-block its 256 threads copy the 8 weight fragments
// and the 8 x parts activation fragments (1 KiB each) into LDS, and each wave
// multiplies a 64 x 64 quarter: 4 weight x 4 activation operands, all parts,
// 16 x parts MFMAs.  Two LDS stages: the next K-block's global loads are in
// flight while the current one is multiplied.  Activation fragments are
// stored to LDS in MFMA lane order (lane r + 16 g <- row r, K-group g), so
// every operand read is one conflict-free 16-byte LDS load.
template <class P, class Epi>
__global__ __launch_bounds__(256) void k_tile_gemm(const uint4* __restrict__ W, const uint4* __restrict__ X, int NT,
                                                   int KB, int Rp, Epi epi) {
  constexpr int PARTS = P::parts;
  constexpr int NFRAG = 8 + 8 * PARTS;  // fragments per K-block stage
  constexpr int PER = NFRAG / 4;        // fragments each thread copies
  __shared__ uint4 lds[2][NFRAG][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nt0 = blockIdx.x * 8, m0 = blockIdx.y * 128;
  const int fw = wave & 1, tw = wave >> 1;
  const size_t xpart = static_cast<size_t>(Rp) * 4;  // uint4 per (K-block, part)
  // Thread's copy duty: fragment wave + 4 i, lane `lane`.  Activation
  // fragments go to the LDS slot of MFMA lane (lane >> 2) + 16 (lane & 3).
  const int xslot = (lane >> 2) + 16 * (lane & 3);

  auto load = [&](uint4* r, int kb) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int f = wave + 4 * i;
      if (f < 8) {
        const int nt = nt0 + f;
        r[i] = nt < NT ? load_weight<true>(W + (static_cast<size_t>(nt) * KB + kb) * 64 + lane)
                       : make_uint4(0u, 0u, 0u, 0u);
      } else {
        const int a = f - 8, q = a >> 3, tt = a & 7;
        r[i] = X[(static_cast<size_t>(kb) * PARTS + q) * xpart + static_cast<size_t>(m0 + 16 * tt) * 4 + lane];
      }
    }
  };
  auto store = [&](int s, const uint4* r) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int f = wave + 4 * i;
      lds[s][f][f < 8 ? lane : xslot] = r[i];
    }
  };

  f32x4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  uint4 pre[PER];
  load(pre, 0);
  store(0, pre);
  __syncthreads();
  for (int kb = 0; kb < KB; ++kb) {
    const int s = kb & 1;
    if (kb + 1 < KB) load(pre, kb + 1);
    uint4 a[4], b[4][PARTS];
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = lds[s][fw * 4 + i][lane];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int q = 0; q < PARTS; ++q) b[j][q] = lds[s][8 + 8 * q + tw * 4 + j][lane];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int q = 0; q < PARTS; ++q) acc[i][j] = P::mma(acc[i][j], a[i], b[j][q]);
    if (kb + 1 < KB) store(s ^ 1, pre);
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int nt = nt0 + fw * 4 + i;
    if (nt >= NT) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) epi.apply_tile(nt, m0 + tw * 64 + 16 * j, acc[i][j], lane);
  }
}

// QKV epilogue: RMSNorm scale, RoPE on q and k, q to the attention input,
// k and v appended to the paged KV cache (same tile orders as decode).
template <class P, class KP = P>
struct EpiQKVRows {
  int M, H, Hkv, hd, mb;
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
    const int n0 = 16 * nt + 4 * (lane >> 4);
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

// Causal attention over each query tile's own request.  Work-group (tile,
// query head): the tile's 16 rows are the MFMA columns, the KV blocks up to
// the tile's last position are split into four contiguous runs, one per wave,
// merged through LDS as in decode.  Column c (position pos0 + c) sees
// positions <= pos0 + c; columns past the tile's rows repeat its last row and
// are not stored.  A wave whose run lies wholly after a column's position
// keeps that column at m = -inf, l = 0 and weighs 0 in the merge (wave 0's run
// starts at position 0, so every column's merged maximum is finite).
template <class P, class AP, int HD>
__global__ __launch_bounds__(256) void k_attn_prefill(const float* __restrict__ q, const void* kcv, const void* vcv,
                                                      const int32_t* __restrict__ bt,
                                                      const PrefillTile* __restrict__ tiles, void* actv, int H,
                                                      int Hkv, int mb, int Rp, float qscale) {
  using E = typename P::elem;
  using Blk = KVBlock<P, HD>;
  constexpr bool kBf16 = sizeof(E) == 2;
  constexpr int NF = Blk::NF;
  constexpr int NE = HD / 16;
  constexpr int EPW = NE / 4;
  const PrefillTile tile = tiles[blockIdx.x];
  const int hq = blockIdx.y, kvh = hq / (H / Hkv);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int c = lane & 15, g = lane >> 4;
  const int cq = c < tile.n ? c : tile.n - 1;
  const int pc = tile.pos0 + cq;                 // this column's position
  const int max_pos = tile.pos0 + tile.n - 1;
  const int nblk = (max_pos >> 4) + 1;
  const int lo = nblk * wave / 4, hi = nblk * (wave + 1) / 4;
  const int32_t* btrow = bt + static_cast<size_t>(tile.slot) * mb;
  int ids = lo + lane < hi ? btrow[lo + lane] : 0;

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
  const E* kc = static_cast<const E*>(kcv);
  const E* vc = static_cast<const E*>(vcv);
  for (int i = lo; i < hi; ++i) {
    const int k = i - lo;
    if ((k & 63) == 0 && k != 0) ids = i + lane < hi ? btrow[i + lane] : 0;
    Blk B;
    B.load(kc, vc, static_cast<size_t>(__builtin_amdgcn_readlane(ids, k & 63)) * Hkv + kvh, lane);
    f32x4_t S = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      S = P::mma(S, B.kf[f], qh[f]);
      if constexpr (kBf16) S = P::mma(S, B.kf[f], ql[f]);
    }
    if (i * 16 + 15 > tile.pos0) {  // block reaches past the tile's first position: causal mask
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
    if (k != 0 && __ballot(m_new != m_run) != 0) {
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

  __shared__ f32x4_t so[4][NE][64];
  __shared__ float2 sml[4][64];
  sml[wave][lane] = make_float2(m_run, l_run);
#pragma unroll
  for (int e = 0; e < NE; ++e) so[wave][e][lane] = O[e];
  __syncthreads();
  float2 ml[4];
  float M = -INFINITY;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    ml[w] = sml[w][lane];
    M = fmaxf(M, ml[w].x);
  }
  float cw[4], L = 0.f;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    cw[w] = __builtin_amdgcn_exp2f(ml[w].x - M);
    L += cw[w] * ml[w].y;
  }
  if (c >= tile.n) return;
  const float inv = 1.f / L;
  typename AP::elem* act = static_cast<typename AP::elem*>(actv);
#pragma unroll
  for (int k = 0; k < EPW; ++k) {
    f32x4_t R = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const f32x4_t o = so[w][wave * EPW + k][lane];
#pragma unroll
      for (int r = 0; r < 4; ++r) R[r] += cw[w] * o[r];
    }
    store_act4<AP>(act, Rp, tile.row0 + c, hq * HD + 16 * (wave * EPW + k) + 4 * g, R[0] * inv, R[1] * inv,
                   R[2] * inv, R[3] * inv);
  }
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
