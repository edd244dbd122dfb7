// Device-side types and helpers for gfx950 (CDNA4): element formats, 16-byte
// operand fragments and the MFMA forms the kernels use.
//
// Fragment convention (both dtypes): one MFMA operand fragment is 64 lanes x
// 16 bytes.  Lane l = r + 16 g holds row (or column) r of a 16-wide tile and
// the g-th quarter of a K-block: 8 bf16 or 4 fp32 elements.  A K-block is
// therefore 32 bf16 or 16 fp32 elements.  Any consistent assignment of K
// indices to (lane group, element) gives the same dot products, so the weight
// tiles, the activation buffers and the attention K/V tiles only have to agree
// with each other.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sprk {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(short)))) short s16x4_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// Agent-coherent 8-byte store and load (relaxed device-scope atomics): a
// work-group on any XCD reads the stored value once the storing wave's vmcnt
// has drained, without a write-back of the storing XCD's L2.
__device__ __forceinline__ void store_coherent2(float* p, float x, float y) {
  const uint64_t v = static_cast<uint64_t>(__float_as_uint(x)) | (static_cast<uint64_t>(__float_as_uint(y)) << 32);
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 load_coherent2(const float* p) {
  const uint64_t v = __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return make_float2(__uint_as_float(static_cast<uint32_t>(v)), __uint_as_float(static_cast<uint32_t>(v >> 32)));
}

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));  // round to nearest even
}

// bf16 storage: 16-bit elements, 32 per K-block, MFMA 16x16x32.  An
// activation (an MFMA B operand) is carried as two bf16 parts, hi = bf16(v)
// and lo = bf16(v - hi), so the product with a bf16 weight keeps about 16
// significant bits of the fp32 activation.
struct BF16 {
  using elem = uint16_t;
  static constexpr int kblk = 32;
  static constexpr int per16 = 8;   // elements per 16 bytes
  static constexpr int parts = 2;   // activation parts (hi, lo)
  static __device__ __forceinline__ elem from_f32(float f) { return f32_to_bf16_bits(f); }
  static __device__ __forceinline__ float to_f32(elem e) { return bf16_bits_to_f32(e); }

  // acc += A(16 x 32) * B(32 x 16) for one fragment pair.
  static __device__ __forceinline__ f32x4_t mma(f32x4_t acc, uint4 a, uint4 b) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                   acc, 0, 0, 0);
  }
};

// bf16 weights whose activations come in three bf16 parts, hi = bf16(v),
// mid = bf16(v - hi) and lo = bf16(v - hi - mid): every significant bit of
// the fp32 activation (three MFMAs per fragment).  The QKV projection takes
// its input this way because its keys and values are rounded into a bf16
// cache, where an input error becomes a whole bf16 step of the elements it
// moves across a rounding boundary; with 16-bit inputs those steps, not the
// fp32 arithmetic, would set the distance to exact arithmetic.
struct BF16x3 : BF16 {
  static constexpr int parts = 3;
};

// fp32 storage: 16 elements per K-block, four MFMA 16x16x4 per fragment pair.
struct F32 {
  using elem = float;
  static constexpr int kblk = 16;
  static constexpr int per16 = 4;
  static constexpr int parts = 1;
  static __device__ __forceinline__ elem from_f32(float f) { return f; }
  static __device__ __forceinline__ float to_f32(elem e) { return e; }

  static __device__ __forceinline__ f32x4_t mma(f32x4_t acc, uint4 a, uint4 b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
    return acc;
  }
};

// Activation buffers (the MFMA B operand of the next projection) are
// K-block-major: K-block kb of part q (hi, then mid / lo) of row b is a 64-byte run at
// element offset ((kb * parts + q) * Rp + b) * kblk, Rp = padded rows.  The
// 16 rows of one part of one K-block are therefore 1 KiB of consecutive
// bytes, which is exactly what one 16-byte-per-lane load of a wave reads.
template <class P>
__device__ __forceinline__ size_t act_offset(int Rp, int b, int k, int part) {
  return (static_cast<size_t>(k / P::kblk * P::parts + part) * Rp + b) * P::kblk + k % P::kblk;
}

// A K tile of the KV cache (16 positions x head_dim) is stored in MFMA
// fragment order, as the A operand of scores = K . q^T: fragment c covers
// dims [c * kblk, (c + 1) * kblk), lane t + 16 g holds position t and dims
// c * kblk + g * per16 + j, j < per16.  One fragment is 1 KiB of consecutive
// bytes, so each wave load of a K tile is fully coalesced.
template <class P>
__device__ __forceinline__ int ktile_offset(int t, int dd) {
  return ((dd / P::kblk) * 64 + ((dd % P::kblk) / P::per16) * 16 + t) * P::per16 + dd % P::per16;
}

// A V tile (16 positions x head_dim) is stored transposed, as the A operand
// of O^T += V^T . P: in the operand for dims [16 e, 16 e + 16), lane r + 16 g
// holds dim 16 e + r at positions 4 g .. 4 g + 3.  For bf16 the 8-byte
// pieces of operands 2 c and 2 c + 1 of one lane are adjacent, so a lane
// fetches both with one 16-byte load; for fp32 a lane's 16 bytes are one
// operand.  Either way lane l's bytes of load v sit at byte (v * 64 + l) * 16
// of the tile, and every wave load reads 1 KiB of consecutive bytes.
template <class P>
__device__ __forceinline__ int vtile_offset(int t, int dd) {
  const int r = dd & 15, g = t >> 2, i = t & 3;
  if constexpr (P::per16 == 8) {
    return ((((dd >> 5) * 4 + g) * 16 + r) * 2 + ((dd >> 4) & 1)) * 4 + i;
  } else {
    return (((dd >> 4) * 4 + g) * 16 + r) * 4 + i;
  }
}

// Stores activation value v of row b, feature k as its P::parts parts: each
// part is the storage rounding of what the earlier parts leave (exact fp32
// differences).
template <class P>
__device__ __forceinline__ void act_store(typename P::elem* act, int Rp, int b, int k, float v) {
  float r = v;
#pragma unroll
  for (int q = 0; q < P::parts; ++q) {
    const typename P::elem e = P::from_f32(r);
    act[act_offset<P>(Rp, b, k, q)] = e;
    r -= P::to_f32(e);
  }
}

// ---------------------------------------------------------------------------
// Counter-based N(0, 0.02) weight draw.  SplitMix64 (Steele, Lea, Flood,
// OOPSLA 2014): the n-th output of a stream seeded with s is
// mix(s + n * 0x9E3779B97F4A7C15).  A matrix (tensor t, layer l) uses the
// stream whose seed is output 1 + 256 t + l of the stream seeded with the
// model seed; its element with row-major index e sums the eight 16-bit lanes
// of outputs 2e+1 and 2e+2 (an Irwin-Hall sum with mean 262140), and the
// weight is fp32(sum - 262140) * 0x1.91530cp-22 (std 0.02), rounded to the
// storage format.  Integer steps and one IEEE multiply: bit-exact anywhere.
// ---------------------------------------------------------------------------
__host__ __device__ __forceinline__ uint64_t sm_mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__host__ __device__ __forceinline__ uint64_t sm_output(uint64_t seed, uint64_t n) {
  return sm_mix64(seed + n * 0x9E3779B97F4A7C15ull);
}

__device__ __forceinline__ uint32_t lanes16_sum(uint64_t r) {
  return static_cast<uint32_t>(r & 0xFFFF) + static_cast<uint32_t>((r >> 16) & 0xFFFF) +
         static_cast<uint32_t>((r >> 32) & 0xFFFF) + static_cast<uint32_t>(r >> 48);
}

__device__ __forceinline__ float weight_draw(uint64_t stream, uint64_t e) {
  const uint32_t s = lanes16_sum(sm_output(stream, 2 * e + 1)) + lanes16_sum(sm_output(stream, 2 * e + 2));
  return static_cast<float>(static_cast<int32_t>(s) - 262140) * 0x1.91530cp-22f;
}

template <class P>
__device__ __forceinline__ typename P::elem weight_elem(uint64_t stream, uint64_t e) {
  return P::from_f32(weight_draw(stream, e));
}

__device__ __forceinline__ float wave_max(float v) {
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

}  // namespace sprk
