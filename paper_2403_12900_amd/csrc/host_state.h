// Host-side state of a decode model: derived dimensions, the workspace layout,
// argument validation and the slot / KV-block bookkeeping.  Pure C++ (no HIP):
// the same translation unit is linked into the device library and into a
// host-only test library.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/sprout.h"

namespace spr {

constexpr int kKvBlock = 16;     // positions per KV block
constexpr int kMaxRows = 128;    // token rows per decode pass (and LM-head rows of a prefill chunk)
constexpr int kPrefillRows = 1024;  // token rows per prefill chunk
constexpr int kPrefillTiles = kPrefillRows / 16 + 64;  // attention query tiles per chunk (segments add one each)
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

struct Layout {
  size_t wqkv, wo, w13, w2;        // per-layer strides of the tiled weights (bytes)
  size_t off_wqkv, off_wo, off_w13, off_w2, off_wlm, off_emb;
  size_t off_rope, off_kc, off_vc, kv_layer_stride, off_bt;
  size_t off_x, off_act0, off_act1, act_bytes, off_q, off_part, off_amax;
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

 private:
  Dims d_{};
  std::vector<Slot> slots_;
  std::vector<int32_t> free_;   // stack of free block ids
};

}  // namespace spr
