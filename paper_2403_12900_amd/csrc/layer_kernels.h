// Persistent decode layer: the five phases of one transformer layer over a
// decode pass -- QKV projection (RMSNorm, RoPE, KV append), attention, O
// projection (+ residual), gate/up projection (RMSNorm, SwiGLU), down
// projection (+ residual) -- in one launch of G resident work-groups, with a
// grid barrier between phases instead of a kernel boundary.  The projection
// phases use the per-kernel path's launch shapes (four-wave one-tile units;
// one-wave two-tile units for a wide gate/up), except that QKV at 17-32 rows
// keeps one-tile units where the per-kernel path pairs tiles; the attention
// splits are fitted to the grid so they run in one round.  The phases after a
// barrier issue their first weight loads while the barrier completes.
//
// Coherence inside the launch (the XCDs' L2 caches are not coherent with one
// another, and no release fence is used):
//   * everything a later phase reads is written with agent-coherent stores
//     (q, the KV append, attention outputs and partials, the residual x, the
//     activation records), and every wave drains its vmcnt before the barrier;
//   * each phase reads its activation record from a buffer no work-group has
//     read earlier in the launch (QKV: act_in, O: act_attn, gate/up: act_mid,
//     down: act_h; down writes act_out = act_in for the next launch), so no
//     XCD can hold a stale line of it; the kernel start invalidates what
//     earlier launches left in the caches;
//   * the residual x, read and rewritten by two phases, is read with
//     agent-coherent loads.
#pragma once

#include "attn_kernels.h"

namespace sprk {

// Grid barrier words (uint32, each group 256 bytes apart): arrival counters
// 0 .. kBarCounters-1, the top counter, then kBarCounters copies of the
// release word (work-group w polls copy w mod kBarCounters, so no single
// memory channel serves every poll).
constexpr int kBarCounters = 32;
constexpr int kBarWords = 64 * (2 * kBarCounters + 1);
// Sleep between polls, in units of 64 clocks.
constexpr int kBarSleep = 8;
// Polls of the release word before a barrier gives up (about a second).
constexpr int kBarSpinLimit = 1 << 20;

struct LayerArgs {
  const uint4* wqkv;
  const uint4* wo;
  const uint4* w13;
  const uint4* w2;
  const uint4* act_in;    // QKV input (K-block-major over d)
  const uint4* act_attn;  // O input: attention output (written through attn.act)
  const uint4* act_mid;   // gate/up input: residual after O (written through o.act)
  const uint4* act_h;     // down input: SwiGLU output (written through gu.act)
  int n_rows, Rp;
  int nt_qkv, nt_o, nt_13, nt_2, kb_d, kb_o, kb_f;
  int n_units;            // attention work items: flat splits x KV heads
  unsigned* bar;          // kBarWords words, zero at model start
  unsigned gen0;          // barrier generations gen0 + 1 .. gen0 + 4 are this launch's
  int spin_limit;         // polls before a barrier gives up (kBarSpinLimit)
  int* err;               // host-visible flag, set when a barrier times out
  AttnArgs attn;
};

// Grid barrier over the gridDim.x work-groups of a persistent launch, in two
// halves.  grid_arrive: every wave's stores before it have completed (the
// work-group barrier drains each wave's vmcnt), then the work-group is
// counted in.  Arrivals are spread over kBarCounters counters (work-group w
// arrives at counter w mod C); the work-group completing a counter arrives at
// the top counter, and the one completing that publishes generation gen in
// every copy of the release word.  Between the halves a work-group may issue
// loads that do not depend on the other work-groups' results (the next
// phase's weights).  grid_wait: one lane per work-group polls its copy of the
// release word, sleeping kBarSleep between polls, and the work-group proceeds
// once it reads gen.  Counts accumulate over launches: counter c holds
// per_c * gen after barrier gen, so the grid size must not change between
// launches that share the words.  A wait that has not seen gen after
// spin_limit polls, or once another one has timed out, sets *err and lets
// its work-group through: the launch still ends, and the host reports the
// failure.
__device__ __forceinline__ void grid_arrive(unsigned* words, unsigned gen) {
  __syncthreads();
  if (threadIdx.x == 0) {
    const int G = gridDim.x;
    const int C = G < kBarCounters ? G : kBarCounters;
    const int c = blockIdx.x % C;
    const unsigned per_c = static_cast<unsigned>((G - c + C - 1) / C);
    unsigned* top = words + 64 * kBarCounters;
    unsigned* rel0 = top + 64;
    const unsigned old = __hip_atomic_fetch_add(words + 64 * c, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (old + 1 == per_c * gen) {
      const unsigned t = __hip_atomic_fetch_add(top, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (t + 1 == static_cast<unsigned>(C) * gen)
        for (int k = 0; k < kBarCounters; ++k)
          __hip_atomic_store(rel0 + 64 * k, gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

__device__ __forceinline__ void grid_wait(unsigned* words, unsigned gen, int* err, int spin_limit) {
  if (threadIdx.x == 0) {
    const unsigned* rel = words + 64 * (kBarCounters + 1) + 64 * (blockIdx.x % kBarCounters);
    int spins = 0;
    while (static_cast<int>(__hip_atomic_load(rel, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) - gen) < 0) {
      if ((++spins & 63) == 0) {
        if (__hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) != 0) break;
        if (spins >= spin_limit) {
          __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
          break;
        }
      }
      __builtin_amdgcn_s_sleep(kBarSleep);
    }
  }
  __syncthreads();
}

__device__ __forceinline__ void grid_barrier(unsigned* words, unsigned gen, int* err, int spin_limit) {
  grid_arrive(words, gen);
  grid_wait(words, gen, err, spin_limit);
}

// One projection over the persistent grid.  kWide: one-wave units of two
// row tiles over the full K (unit u on wave u / G of work-group u mod G), the
// per-kernel path's shape for wide projections; otherwise four-wave units of
// one row tile, the waves splitting K (unit u on work-group u mod G).  Each
// phase compiles only its own shape, which keeps the kernel's register
// budget at that of its largest phase.
template <class P, int JT, bool kWide, class Epi>
__device__ __forceinline__ void gemm_phase(const uint4* W, const uint4* X, int NT, int KB, int Rp, int n_rows,
                                           const Epi& epi, float* red) {
  const int G = gridDim.x;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  // The lane index is made opaque in each iteration, so that nothing derived
  // from it is hoisted out of the unit loop and kept live across units (which
  // would raise the register budget above the one-unit kernel's).
  constexpr int WAVES = kWide ? 1 : 4, RT = kWide ? 2 : 1;
  constexpr int U = kWide ? (JT == 1 ? 8 : 4) : StreamDepth<JT * P::parts>::value;
  StreamStageOf<P, JT, RT, U> s0, s1;
  for (int u = kWide ? blockIdx.x + G * wave : blockIdx.x; u < (kWide ? NT / 2 : NT); u += kWide ? 4 * G : G) {
    if constexpr (!kWide) __syncthreads();  // the previous unit's reduction has been read
    int ln = lane;
    asm volatile("" : "+v"(ln));
    stream_gemm_tiles<P, JT, WAVES, Epi, RT, U, true>(W, X, KB, Rp, n_rows, epi, RT * u, kWide ? 0 : wave, ln, red,
                                                      s0, s1);
  }
}

// A projection phase that follows a grid barrier: each wave's first unit has
// its first two weight stages issued between the barrier's arrival and its
// wait, so the weight stream is already in flight when the barrier opens.
template <class P, int JT, bool kWide, class Epi>
__device__ __forceinline__ void gemm_phase_after(const uint4* W, const uint4* X, int NT, int KB, int Rp, int n_rows,
                                                 const Epi& epi, float* red, unsigned* bar, unsigned gen, int* err,
                                                 int spin_limit) {
  const int G = gridDim.x;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  constexpr int WAVES = kWide ? 1 : 4, RT = kWide ? 2 : 1;
  constexpr int U = kWide ? (JT == 1 ? 8 : 4) : StreamDepth<JT * P::parts>::value;
  const int u0 = kWide ? blockIdx.x + G * wave : blockIdx.x;
  const int nu = kWide ? NT / 2 : NT, step = kWide ? 4 * G : G;
  const int kw = kWide ? 0 : wave;
  StreamStageOf<P, JT, RT, U> s0, s1;
  grid_arrive(bar, gen);
  if (u0 < nu) stream_prefetch_weights<P, JT, WAVES, RT, U, true>(W, KB, RT * u0, kw, lane, s0, s1);
  grid_wait(bar, gen, err, spin_limit);
  if (u0 < nu)
    stream_gemm_tiles<P, JT, WAVES, Epi, RT, U, true, 2>(W, X, KB, Rp, n_rows, epi, RT * u0, kw, lane, red, s0, s1);
  for (int u = u0 + step; u < nu; u += step) {
    if constexpr (!kWide) __syncthreads();
    int ln = lane;
    asm volatile("" : "+v"(ln));
    stream_gemm_tiles<P, JT, WAVES, Epi, RT, U, true>(W, X, KB, Rp, n_rows, epi, RT * u, kw, ln, red, s0, s1);
  }
}

// The attention work items over the persistent grid (item u on work-group u
// mod G; items are (flat split, KV head) in the per-kernel grid's order).
template <class KP, class P, int HD>
__device__ __forceinline__ void attn_phase(const AttnArgs& at, int n_units, AttnSmem<HD>* sm) {
  const int F = n_units / at.Hkv;
  for (int u = blockIdx.x; u < n_units; u += gridDim.x) {
    __syncthreads();  // the previous item's LDS has been read
    attn_decode_unit<KP, P, HD, true>(at, u % F, u / F, sm);
  }
}

// LDS floats of gemm_phase's reduction (four waves, one row tile).
template <int JT>
struct LayerRed {
  static constexpr int floats = StreamRed<JT, 4, 1>::floats;
};

// Epilogues of one layer in the activation format P and KV format KP.
template <class P, class KP>
struct LayerEpis {
  EpiQKV<P, KP, true> qkv;
  EpiResid<P, true> o;
  EpiSwiGLU<P, true> gu;
  EpiResid<P, true> down;
};

// kWideGU: the gate/up projection has an even number of at least 1024 row
// tiles (one-wave two-tile units); every other phase uses four-wave units.
template <class P, class KP, int HD, int JT, bool kWideGU>
__global__ __launch_bounds__(256, 3) void k_decode_layer(LayerArgs a, LayerEpis<P, KP> e) {
  __shared__ AttnSmem<HD> sm_attn;
  __shared__ float red[LayerRed<JT>::floats];
  gemm_phase<P, JT, false>(a.wqkv, a.act_in, a.nt_qkv, a.kb_d, a.Rp, a.n_rows, e.qkv, red);
  grid_barrier(a.bar, a.gen0 + 1, a.err, a.spin_limit);
  attn_phase<KP, P, HD>(a.attn, a.n_units, &sm_attn);
  gemm_phase_after<P, JT, false>(a.wo, a.act_attn, a.nt_o, a.kb_o, a.Rp, a.n_rows, e.o, red, a.bar, a.gen0 + 2, a.err,
                                 a.spin_limit);
  gemm_phase_after<P, JT, kWideGU>(a.w13, a.act_mid, a.nt_13, a.kb_d, a.Rp, a.n_rows, e.gu, red, a.bar, a.gen0 + 3,
                                   a.err, a.spin_limit);
  gemm_phase_after<P, JT, false>(a.w2, a.act_h, a.nt_2, a.kb_f, a.Rp, a.n_rows, e.down, red, a.bar, a.gen0 + 4,
                                 a.err, a.spin_limit);
}

}  // namespace sprk
