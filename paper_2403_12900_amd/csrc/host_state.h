// Host-side state of a decode model: derived dimensions, the workspace layout,
// argument validation and the slot / KV-block bookkeeping.  Pure C++ (no HIP):
// the same translation unit is linked into the device library and into a
// host-only test library.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>
#include <utility>
#include <vector>

#include "../../include/sprout.h"

namespace spr {

constexpr int kKvBlock = 16;     // positions per KV block
constexpr int kMaxRows = 128;    // token rows per decode pass (and LM-head rows of a prefill chunk)
// Token rows per prefill chunk.  Chunks fill up in request order.  At 7B
// shapes, 32 prompts of 8427 tokens in all ran 14% faster in 4096-row chunks
// than in 1024-row ones (more work-groups per projection), and 2% faster than
// in three equal chunks.
constexpr int kPrefillRows = 4096;
constexpr int kPrefillTiles = kPrefillRows / 16 + 64;  // attention query tiles per chunk, 64 rows or fewer each
constexpr int kMaxSplits = 2048; // KV splits over all rows of one pass (decode attention)
constexpr int kFragBytes = 1024; // one MFMA operand fragment: 64 lanes x 16 bytes

struct Dims {
  int L, d, H, Hkv, hd, f, V, G;
  int dtype, esize, kblk;          // element bytes; elements per K-block (32 bf16 / 16 fp32)
  int kv_dtype, kv_esize;          // KV-cache storage format
  int qkv_rows, o_in;              // (H + 2 Hkv) hd, H hd
  int nt_qkv, nt_o, nt_13, nt_2, nt_lm;  // 16-row output tiles (gate/up: 8 features per tile)
  int kb_d, kb_o, kb_f, kb_max;    // K-blocks of the inputs d, H hd, d_ff
  int S, max_ctx, mb, nb;          // slots, positions, blocks per slot, pool blocks
  float rope_base, eps;
};

// Split-K shapes of the decode projections past 8 rows (16-row tiles per
// group, K slices): O and down, gate/up, QKV.
struct SplitShape {
  int rt, s;
};
constexpr SplitShape kSplitO{2, 4}, kSplitGU{4, 2}, kSplitQKV{4, 4};

// Bounds on what the split-K launches of any decode pass of the model use:
// partial-sum floats and arrival counters.
struct SplitNeed {
  size_t part_floats;
  int counters;
};
SplitNeed split_need(const Dims& d);

struct Layout {
  size_t wqkv, wo, w13, w2;        // per-layer strides of the tiled weights (bytes)
  size_t off_wqkv, off_wo, off_w13, off_w2, off_wlm, off_emb;
  size_t off_rope, off_kc, off_vc, kv_layer_stride, off_bt;
  size_t off_x, off_act0, off_act1, act_bytes, off_q, off_part, off_cnt, off_amax;
  size_t part_floats;              // capacity of the partials region (attention splits, split-K)
  int n_cnt;                       // capacity of the counters region
  size_t off_prow, off_ptile, off_rs;  // prefill chunk: row table, query tiles, RMSNorm scales
  size_t total;
};

bool derive(const spr_config& c, Dims* d, std::string* err);
Layout layout(const Dims& d);

enum SlotState { kFree = 0, kActive = 1, kFinished = 2 };

struct Slot {
  SlotState state = kFree;
  int len = -1, produced = 0, stop = 0;
  std::vector<int32_t> blocks;
};

class SlotTable {
 public:
  void init(const Dims& d);
  int free_blocks() const { return static_cast<int>(free_.size()); }
  const Slot& slot(int s) const { return slots_[s]; }

  // Validation (no state change).  Return SPR_OK or an error with *err set.
  spr_status check_prefill(int n, const int32_t* slots, const int32_t* seq_lens, const int32_t* stop_lens,
                           std::string* err) const;
  spr_status check_decode(int n, const int32_t* slots, const int32_t* lens, std::string* err) const;
  spr_status check_rewind(int slot, int len, int produced, std::string* err) const;
  spr_status check_free(int slot, std::string* err) const;

  // State changes; callers validate first.  commit_prefill reserves blocks
  // and returns the block-table rows it filled.
  void commit_prefill(int n, const int32_t* slots, const int32_t* seq_lens, const int32_t* stop_lens,
                      int32_t* retired);
  void commit_decode(int n, const int32_t* slots, int32_t* retired);
  void commit_rewind(int slot, int len, int produced);
  void commit_free(int slot);

  // Block-table row of a slot, padded with 0 to `mb` entries.
  void block_row(int slot, int32_t* row) const;

  // KV blocks a request of this prompt and stop length reserves.
  static int blocks_for(int seq_len, int stop_len) { return (seq_len + stop_len - 1 + kKvBlock - 1) / kKvBlock; }

 private:
  Dims d_{};
  std::vector<Slot> slots_;
  std::vector<int32_t> free_;   // stack of free block ids
};

// ---------------------------------------------------------------------------
// Continuous (iteration-level) batching over the slot table.  Requests wait
// in arrival order; every scheduler iteration
//   1. admits waiting requests whose arrival iteration has come, first come
//      first served, into free slots while fewer than max_active requests are
//      in flight and the KV pool can reserve their blocks (a request that
//      does not fit yet holds back the ones behind it);
//   2. prefills the admitted requests together (each emits its first token);
//   3. runs one decode step over every request still generating;
//   4. retires requests that produced their stop length and frees their slots
//      and blocks at once, for the next iteration's admissions;
//   5. retires requests whose token in the previous iteration was the EOS id
//      (Section II-A: generation ends at EOS or at the preset limit).  The
//      device reports EOS one iteration late, so the host never waits for the
//      iteration it has just enqueued; such a request runs one extra decode
//      row, inside the KV blocks it reserved, whose token is discarded.
// Iterations with nothing in flight jump to the next arrival.  The device
// work goes through ServeDevice, so the policy runs unchanged on the host
// alone (tests) or over the GPU kernels (spr_serve).
// ---------------------------------------------------------------------------
struct ServeRequest {
  const int32_t* tokens;  // prompt (directive prefix ++ user prompt)
  int n_tokens, stop_len;
  int arrival;            // first scheduler iteration it may be admitted in
};

struct ServeCounters {
  int64_t iterations = 0, decode_steps = 0, prefill_calls = 0, decode_tokens = 0;
  int max_batch = 0;
  double mean_batch = 0.0;  // mean decode-step batch
};

class ServeDevice {
 public:
  int iteration = 0;  // scheduler iteration of the next call (set by serve)
  virtual ~ServeDevice() = default;
  // Prefill requests req[k] into slots[k] (already reserved in the table);
  // each emits its token 0.
  virtual spr_status prefill(int n, const int32_t* slots, const int32_t* req) = 0;
  // One decode step; row k: slot, cached positions, request, index of the
  // token the step produces for it.
  virtual spr_status decode(int n, const int32_t* slots, const int32_t* lens, const int32_t* req,
                            const int32_t* produced) = 0;
  // Called after each iteration's device work.  Appends to *eos the (request,
  // token index) pairs whose token was the EOS id in the previous iteration;
  // with final = true (once, after the last iteration), in the last one too.
  virtual spr_status end_iteration(bool final, std::vector<std::pair<int, int>>* eos) = 0;
};

// Runs the whole request list.  Needs every slot free on entry; leaves every
// slot free on success.  SPR_ERR_INVALID_ARG for a malformed request or one
// the KV pool could never hold; errors of the device calls are returned as is.
// lengths (may be null) receives each request's generated tokens: up to and
// including its first EOS, else its stop length.
spr_status serve(SlotTable& tab, const Dims& d, int n, const ServeRequest* reqs, int max_active, ServeDevice& dev,
                 ServeCounters* counters, std::vector<int32_t>* lengths, std::string* err);

}  // namespace spr
