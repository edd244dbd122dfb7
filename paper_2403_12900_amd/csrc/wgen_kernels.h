// Weight initialisation straight into the tiled layouts the streaming GEMM
// reads, and the inverse read-back of logical rows.
//
// Tiled layout of a projection W[N][K] (N outputs, K inputs): 16-row tiles
// nt, K-blocks kb; fragment (nt, kb) is 1 KiB at ((nt * KB + kb) * 64 + lane)
// * 16 bytes, lane = r + 16 g holding W[16 nt + r][kb * kblk + g * per16 + j],
// j < per16.  Rows and columns past N, K are zero.
//
// Fused matrices:
//   QKV  rows 0..H hd-1 = Wq, then Wk, then Wv (one GEMM, one pass over x).
//   W13  tile nt covers features 8 nt .. 8 nt + 7; tile row 4 a + i holds gate
//        (W1) row 8 nt + 2 a + i for i < 2 and up (W3) row 8 nt + 2 a + i - 2
//        for i >= 2, so one lane's four accumulator rows are gate and up of
//        two features and SiLU(gate) * up needs no data exchange.
#pragma once

#include "device_common.h"

namespace sprk {

enum MatKind { MK_QKV = 0, MK_O = 1, MK_W13 = 2, MK_W2 = 3, MK_LM = 4 };

struct MatSpec {
  int kind, NT, KB, K;       // tiles, K-blocks, logical K
  int H, Hkv, hd, f, d, V;
  uint64_t key[3];           // generator streams: QKV q/k/v, W13 gate/up, others key[0]
};

// Logical (stream index, row) of physical row n; false for padding rows.
__device__ __forceinline__ bool phys_row(const MatSpec& s, int n, int* which, int* row) {
  switch (s.kind) {
    case MK_QKV: {
      const int qr = s.H * s.hd, kr = s.Hkv * s.hd;
      if (n < qr) { *which = 0; *row = n; return true; }
      if (n < qr + kr) { *which = 1; *row = n - qr; return true; }
      *which = 2; *row = n - qr - kr;
      return *row < kr;
    }
    case MK_W13: {
      const int r = n & 15, a = r >> 2, i = r & 3;
      *row = 8 * (n >> 4) + 2 * a + (i & 1);
      *which = i < 2 ? 0 : 1;
      return *row < s.f;
    }
    case MK_O:
    case MK_W2:
      *which = 0; *row = n;
      return n < s.d;
    default:
      *which = 0; *row = n;
      return n < s.V;
  }
}

template <class P>
__global__ __launch_bounds__(256) void k_init_tiled(uint4* __restrict__ out, MatSpec s) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t nfrag = static_cast<int64_t>(s.NT) * s.KB;
  if (idx >= nfrag * 64) return;
  const int lane = static_cast<int>(idx & 63);
  const int64_t frag = idx >> 6;
  const int nt = static_cast<int>(frag / s.KB), kb = static_cast<int>(frag % s.KB);
  const int n = 16 * nt + (lane & 15);
  const int k0 = kb * P::kblk + (lane >> 4) * P::per16;
  int which = 0, row = 0;
  const bool valid = phys_row(s, n, &which, &row);
  union {
    uint4 u;
    typename P::elem e[P::per16];
  } v;
#pragma unroll
  for (int j = 0; j < P::per16; ++j) {
    const int k = k0 + j;
    v.e[j] = (valid && k < s.K) ? weight_elem<P>(s.key[which], static_cast<uint64_t>(row) * s.K + k)
                                : P::from_f32(0.f);
  }
  out[idx] = v.u;
}

// Row-major [rows][cols] table (the embedding).
template <class P>
__global__ __launch_bounds__(256) void k_init_rowmajor(typename P::elem* __restrict__ out, int64_t count,
                                                       uint64_t key) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < count) out[i] = weight_elem<P>(key, static_cast<uint64_t>(i));
}

// Reads logical rows [row0, row0 + nrows) of stream `which` of a tiled matrix
// back as fp32: out[r][c], c < s.K.
template <class P>
__global__ __launch_bounds__(256) void k_export_tiled(const typename P::elem* __restrict__ w, MatSpec s, int which,
                                                      int row0, int nrows, float* __restrict__ out) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= static_cast<int64_t>(nrows) * s.K) return;
  const int r = static_cast<int>(i / s.K) + row0, c = static_cast<int>(i % s.K);
  int n;
  switch (s.kind) {
    case MK_QKV:
      n = r + (which >= 1 ? s.H * s.hd : 0) + (which == 2 ? s.Hkv * s.hd : 0);
      break;
    case MK_W13: {
      const int t = r >> 3, a = (r & 7) >> 1, i2 = r & 1;
      n = 16 * t + 4 * a + i2 + (which == 1 ? 2 : 0);
      break;
    }
    default:
      n = r;
  }
  const int nt = n >> 4, kb = c / P::kblk, kk = c % P::kblk;
  const int lane = (n & 15) + 16 * (kk / P::per16);
  const int64_t at = ((static_cast<int64_t>(nt) * s.KB + kb) * 64 + lane) * P::per16 + kk % P::per16;
  out[i] = P::to_f32(w[at]);
}

template <class P>
__global__ __launch_bounds__(256) void k_export_rowmajor(const typename P::elem* __restrict__ w, int cols, int row0,
                                                         int nrows, float* __restrict__ out) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= static_cast<int64_t>(nrows) * cols) return;
  out[i] = P::to_f32(w[static_cast<int64_t>(row0) * cols + i]);
}

// Overwrites LM-head row dst of the tiled matrix (one thread per element of
// the row): with row src when src >= 0, else with `fill` rounded to the
// storage format.  A test aid (planted ties, poisoned rows).
template <class P>
__global__ __launch_bounds__(256) void k_write_tiled_row(typename P::elem* __restrict__ w, int KB, int K, int dst,
                                                         int src, float fill) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= K) return;
  const int kb = c / P::kblk, kk = c % P::kblk;
  auto at = [&](int n) {
    const int lane = (n & 15) + 16 * (kk / P::per16);
    return ((static_cast<int64_t>(n >> 4) * KB + kb) * 64 + lane) * P::per16 + kk % P::per16;
  };
  w[at(dst)] = src >= 0 ? w[at(src)] : P::from_f32(fill);
}

}  // namespace sprk
