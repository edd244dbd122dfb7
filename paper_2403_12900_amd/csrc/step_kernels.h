// Per-step kernels around the layer stack: token embedding and the final
// greedy token (lowest index among equal maxima).
#pragma once

#include "gemm_kernels.h"

namespace sprk {

// Bits of the device check flag (mapped host memory; the host reports a
// nonzero flag at the next call).
constexpr int kErrTokenRange = 1;  // a fed token id outside [0, V)
constexpr int kErrLogits = 2;      // a logits row with a NaN or no finite maximum

// Sets bit `bit` of the flag.  The flag lives in host memory, so this is a
// plain load and store (no read-modify-write atomic over the host link); two
// kernels racing to set different bits may leave only one, and the flag is
// still nonzero.  Runs only on the error path.
__device__ __forceinline__ void raise_check(int* err, int bit) {
  const int v = __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  __hip_atomic_store(err, v | bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

struct EmbedArgs {
  const void* emb;          // [V][d] row-major
  const int32_t* tok_dev;   // device tokens indexed by slot, or null: use tok[]
  float* x;                 // residual [rows][d]
  void* act;                // first activation, K-block-major over d
  int* err;                 // device check flag (kErrTokenRange)
  int n_rows, d, V, Rp;
  int slot[kRows];
  int tok[kRows];
};

// A token outside [0, V) (only possible when a caller forces one through
// device memory) raises kErrTokenRange, so the next call on the model fails;
// the read itself is clamped into the table.
template <class P>
__global__ __launch_bounds__(64) void k_embed(EmbedArgs a) {
  const int b = blockIdx.y;
  const int n0 = 4 * (blockIdx.x * 64 + threadIdx.x);
  if (n0 >= a.d) return;
  int t = a.tok_dev != nullptr ? a.tok_dev[a.slot[b]] : a.tok[b];
  if (t < 0 || t >= a.V) {
    if (n0 == 0) raise_check(a.err, kErrTokenRange);
    t = min(max(t, 0), a.V - 1);
  }
  const typename P::elem* e = static_cast<const typename P::elem*>(a.emb) + static_cast<size_t>(t) * a.d + n0;
  const float v0 = P::to_f32(e[0]), v1 = P::to_f32(e[1]), v2 = P::to_f32(e[2]), v3 = P::to_f32(e[3]);
  *reinterpret_cast<float4*>(a.x + static_cast<size_t>(b) * a.d + n0) = make_float4(v0, v1, v2, v3);
  store_act4<P>(static_cast<typename P::elem*>(a.act), a.Rp, b, n0, v0, v1, v2, v3);
}

struct ArgmaxArgs {
  const float2* part;       // [tiles][kRows] (value, index bits)
  int32_t* tok_dev;         // written at the row's slot
  int32_t* hist;            // or null: token history, written at hist_idx[row] when >= 0
  int* err;                 // device check flag (kErrLogits)
  int n_tiles;
  int slot[kRows];
  int out_row[kRows];       // -1: row emits no token
  int hist_idx[kRows];
};

__device__ __forceinline__ void better_of(float& v, int& i, float ov, int oi) {
  if (ov > v || (ov == v && oi < i)) {
    v = ov;
    i = oi;
  }
}

// A tile whose logits held a NaN reports a NaN candidate value (EpiLogits).
// A row with such a tile, or with no finite maximum, raises kErrLogits and
// gets token 0.
__global__ __launch_bounds__(256) void k_argmax_final(ArgmaxArgs a) {
  const int b = blockIdx.x;
  if (a.out_row[b] < 0) return;
  float v = -INFINITY;
  int idx = 0x7fffffff;
  int bad = 0;
  for (int t = threadIdx.x; t < a.n_tiles; t += 256) {
    const float2 p = a.part[static_cast<size_t>(t) * kRows + b];
    bad |= p.x != p.x;
    better_of(v, idx, p.x, __float_as_int(p.y));
  }
  bad = __syncthreads_or(bad);
  for (int o = 32; o >= 1; o >>= 1) better_of(v, idx, __shfl_xor(v, o), __shfl_xor(idx, o));
  __shared__ float sv[4];
  __shared__ int si[4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    sv[wave] = v;
    si[wave] = idx;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w) better_of(v, idx, sv[w], si[w]);
    if (bad || !(fabsf(v) <= 3.402823466e38f)) {
      raise_check(a.err, kErrLogits);
      idx = 0;
    }
    a.tok_dev[a.slot[b]] = idx;
    if (a.hist != nullptr && a.hist_idx[b] >= 0) a.hist[a.hist_idx[b]] = idx;
  }
}

// out[0 .. n) = 0.
__global__ __launch_bounds__(256) void k_zero_i32(int32_t* out, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) out[i] = 0;
}

// Streaming read of n16 16-byte words with the projections' load form
// (nontemporal 16-byte loads, kReadUnroll in flight per thread): the read
// rate this memory path reaches with no arithmetic attached.  Full chunks of
// 256 * kReadUnroll words run unpredicated; the tail is read word by word.
// The XOR of every word read goes to sink only when it equals a fixed
// constant, so no load can be dropped and the store practically never runs.
constexpr int kReadUnroll = 8;
__global__ __launch_bounds__(256) void k_read_stream(const uint4* __restrict__ p, size_t n16, uint32_t* sink) {
  constexpr size_t kChunk = 256 * kReadUnroll;
  const size_t full = n16 / kChunk;
  uint32_t acc = 0;
  for (size_t c = blockIdx.x; c < full; c += gridDim.x) {
    const uint4* q = p + c * kChunk + threadIdx.x;
    uint4 v[kReadUnroll];
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) v[u] = load_weight<true>(q + u * 256);
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  if (blockIdx.x == 0)
    for (size_t k = full * kChunk + threadIdx.x; k < n16; k += 256) {
      const uint4 v = p[k];
      acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
  if (acc == 0x9e3779b9u) sink[0] = acc;
}

}  // namespace sprk
