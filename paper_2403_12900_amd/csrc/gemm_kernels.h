// Weight-streaming projection for decode: y[b][n] = sum_k W[n][k] x[b][k] for
// every active row b, with the op that follows fused into the epilogue.
//
// Decode reads every weight byte once per step while the batch is at most a
// few dozen rows, so the kernel is HBM-bound (intensity = rows flop/byte, far
// below the MFMA ridge).  MFMA is used as the dot-product engine because the
// tiles come straight from HBM in the operand layout, not because the
// kernel needs its throughput:
//   * one workgroup per 16-row output tile; its waves split the K-blocks, each
//     streaming contiguous 1 KiB weight fragments with 16-byte loads;
//   * the activations (rows x K, K-block-major records of 64-byte runs, see
//     act_record) are the MFMA B operand: a lane reads 16 contiguous bytes of
//     one row, and rows past the batch are not read at all, so a batch of one
//     reads one row;
//   * bf16 activations come as hi + lo parts (two MFMAs per fragment), which
//     keeps the activation side of every product near fp32 precision;
//   * per-wave accumulators are summed through LDS in a fixed order, so the
//     result is bitwise reproducible.
// RMSNorm (unit gains) of the input is fused: the sum of squares of each row
// is accumulated from the activation fragments already in registers, and
// 1/sqrt(mean + eps) scales the accumulator in the epilogue.
#pragma once

#include "device_common.h"

namespace sprk {

constexpr int kRows = 128;      // token rows per pass
constexpr int kSplitsMax = 16;  // decode-attention KV splits per (row, head)

struct RowSlotPos {
  int slot[kRows];
  int pos[kRows];
};

template <class P, int JT, int WAVES, class Epi>
__global__ __launch_bounds__(WAVES * 64) void k_stream_gemm(const uint4* __restrict__ W, const uint4* __restrict__ X,
                                                            int KB, int Rp, int n_rows, Epi epi) {
  const int nt = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int kb0 = (KB * wave) / WAVES, kb1 = (KB * (wave + 1)) / WAVES;
  f32x4_t acc[JT];
  float ssq[JT];
#pragma unroll
  for (int j = 0; j < JT; ++j) {
    acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    ssq[j] = 0.f;
  }
  const uint4* wp = W + static_cast<size_t>(nt) * KB * 64 + lane;
  // Activation record (kb, row) = PARTS runs of 64 bytes; lane reads 16 bytes of each.
  constexpr int PARTS = P::parts;
  constexpr int REC = 4 * PARTS;  // uint4 per record
  const uint4* xp = X + (lane & 15) * REC + (lane >> 4);
  bool rv[JT];  // rows past n_rows are never read: their lanes feed zeros
#pragma unroll
  for (int j = 0; j < JT; ++j) rv[j] = 16 * j + (lane & 15) < n_rows;
  const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
  constexpr int XW = JT * PARTS;
  constexpr int U = XW <= 2 ? 8 : XW <= 4 ? 4 : 2;
  int kb = kb0;
  for (; kb + U <= kb1; kb += U) {
    uint4 a[U], x[U][JT][PARTS];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      a[u] = wp[static_cast<size_t>(kb + u) * 64];
#pragma unroll
      for (int j = 0; j < JT; ++j)
#pragma unroll
        for (int q = 0; q < PARTS; ++q)
          x[u][j][q] = rv[j] ? xp[(static_cast<size_t>(kb + u) * Rp + 16 * j) * REC + 4 * q] : zero;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int j = 0; j < JT; ++j) {
#pragma unroll
        for (int q = 0; q < PARTS; ++q) acc[j] = P::mma(acc[j], a[u], x[u][j][q]);
        if constexpr (Epi::kNorm) ssq[j] += P::sumsq(x[u][j][0], x[u][j][PARTS - 1]);
      }
    }
  }
  for (; kb < kb1; ++kb) {
    const uint4 a = wp[static_cast<size_t>(kb) * 64];
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      uint4 x[PARTS];
#pragma unroll
      for (int q = 0; q < PARTS; ++q) x[q] = rv[j] ? xp[(static_cast<size_t>(kb) * Rp + 16 * j) * REC + 4 * q] : zero;
#pragma unroll
      for (int q = 0; q < PARTS; ++q) acc[j] = P::mma(acc[j], a, x[q]);
      if constexpr (Epi::kNorm) ssq[j] += P::sumsq(x[0], x[PARTS - 1]);
    }
  }
  if constexpr (WAVES > 1) {
    __shared__ float red[WAVES - 1][JT][5][64];
    if (wave > 0) {
#pragma unroll
      for (int j = 0; j < JT; ++j) {
#pragma unroll
        for (int c = 0; c < 4; ++c) red[wave - 1][j][c][lane] = acc[j][c];
        red[wave - 1][j][4][lane] = ssq[j];
      }
    }
    __syncthreads();
    if (wave != 0) return;
    for (int w = 0; w < WAVES - 1; ++w) {
#pragma unroll
      for (int j = 0; j < JT; ++j) {
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[j][c] += red[w][j][c][lane];
        ssq[j] += red[w][j][4][lane];
      }
    }
  }
  if constexpr (Epi::kNorm) {
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      ssq[j] += __shfl_xor(ssq[j], 16);
      ssq[j] += __shfl_xor(ssq[j], 32);
    }
  }
  epi.template apply<JT>(nt, acc, ssq, lane);
}

// Stores four consecutive features n0..n0+3 of row b into a K-block-major activation buffer.
template <class P>
__device__ __forceinline__ void store_act4(typename P::elem* act, int Rp, int b, int n0, float v0, float v1, float v2,
                                           float v3) {
  typename P::elem* rec = act_record<P>(act, Rp, b, n0);
  const int kk = n0 % P::kblk;
  P::store_act(rec, kk, v0);
  P::store_act(rec, kk + 1, v1);
  P::store_act(rec, kk + 2, v2);
  P::store_act(rec, kk + 3, v3);
}

// QKV projection -> RMSNorm scale -> RoPE on q and k -> q to the attention
// input, k and v appended to the paged KV cache at the row's position.
// K block layout [block][kv_head][16 positions][head_dim]; V is stored
// transposed per block, [block][kv_head][head_dim][16 positions], so the
// attention kernel reads 4 consecutive positions of one dimension as one
// MFMA operand.
template <class P>
struct EpiQKV {
  static constexpr bool kNorm = true;
  int n_rows, H, Hkv, hd, mb, dnorm;
  float eps;
  float* q;                     // [rows][H * hd]
  typename P::elem* kc;         // this layer's K blocks
  typename P::elem* vc;         // this layer's V blocks
  const int32_t* bt;            // [slots][mb]
  const float2* rope;           // [positions][hd / 2] (cos, sin)
  RowSlotPos rows;

  template <int JT>
  __device__ __forceinline__ void apply(int nt, const f32x4_t* acc, const float* ssq, int lane) const {
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
        const int dd = (n0 < qr ? n0 : n0 - qr) % hd;
        const float2* rp = rope + static_cast<size_t>(p) * (hd / 2) + dd / 2;
        const float2 c0 = rp[0], c1 = rp[1];
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
      const int blk = bt[static_cast<size_t>(rows.slot[b]) * mb + (p >> 4)];
      const int off = p & 15;
      if (n0 < qr + kr) {
        const int m = n0 - qr, kvh = m / hd, dd = m % hd;
        typename P::elem* dst = kc + ((static_cast<size_t>(blk) * Hkv + kvh) * 16 + off) * hd + dd;
        dst[0] = P::from_f32(v0);
        dst[1] = P::from_f32(v1);
        dst[2] = P::from_f32(v2);
        dst[3] = P::from_f32(v3);
      } else {
        const int m = n0 - qr - kr, kvh = m / hd, dd = m % hd;
        typename P::elem* dst = vc + ((static_cast<size_t>(blk) * Hkv + kvh) * hd + dd) * 16 + off;
        dst[0] = P::from_f32(v0);
        dst[16] = P::from_f32(v1);
        dst[32] = P::from_f32(v2);
        dst[48] = P::from_f32(v3);
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

  template <int JT>
  __device__ __forceinline__ void apply(int nt, const f32x4_t* acc, const float*, int lane) const {
    const int n0 = 16 * nt + 4 * (lane >> 4);
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      const int b = 16 * j + (lane & 15);
      if (b >= n_rows) continue;
      float4* xp = reinterpret_cast<float4*>(x + static_cast<size_t>(b) * d + n0);
      float4 xv = *xp;
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

  template <int JT>
  __device__ __forceinline__ void apply(int nt, const f32x4_t* acc, const float* ssq, int lane) const {
    const int j0 = 8 * nt + 2 * (lane >> 4);
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      const int b = 16 * j + (lane & 15);
      if (b >= n_rows) continue;
      const float s = rsqrtf(ssq[j] / static_cast<float>(dnorm) + eps);
      const float g0 = acc[j][0] * s, g1 = acc[j][1] * s, u0 = acc[j][2] * s, u1 = acc[j][3] * s;
      const float h0 = g0 / (1.f + __expf(-g0)) * u0;
      const float h1 = g1 / (1.f + __expf(-g1)) * u1;
      typename P::elem* rec = act_record<P>(act, Rp, b, j0);
      P::store_act(rec, j0 % P::kblk, h0);
      P::store_act(rec, j0 % P::kblk + 1, h1);
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

  template <int JT>
  __device__ __forceinline__ void apply(int nt, const f32x4_t* acc, const float* ssq, int lane) const {
    const int n0 = 16 * nt + 4 * (lane >> 4);
#pragma unroll
    for (int j = 0; j < JT; ++j) {
      const int b = 16 * j + (lane & 15);
      const bool vb = b < n_rows;
      const float s = rsqrtf(ssq[j] / static_cast<float>(dnorm) + eps);
      float best = -INFINITY;
      int bi = 0x7fffffff;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float z = acc[j][i] * s;
        const int n = n0 + i;
        if (n < V && z > best) {
          best = z;
          bi = n;
        }
        if (vb && logits != nullptr && n < V && out_row[b] >= 0) logits[static_cast<size_t>(out_row[b]) * V + n] = z;
      }
#pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        const float ob = __shfl_xor(best, o);
        const int oi = __shfl_xor(bi, o);
        if (ob > best || (ob == best && oi < bi)) {
          best = ob;
          bi = oi;
        }
      }
      if ((lane >> 4) == 0 && vb) part[static_cast<size_t>(nt) * kRows + b] = make_float2(best, __int_as_float(bi));
    }
  }
};

}  // namespace sprk
