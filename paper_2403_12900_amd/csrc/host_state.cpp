// Host-side bookkeeping of the decode model (see host_state.h).
#include "host_state.h"

#include <utility>

#include <algorithm>
#include <cmath>
#include <limits>

namespace spr {

namespace {

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

int ceil_div(int a, int b) { return (a + b - 1) / b; }

bool fail(std::string* err, const std::string& msg) {
  if (err) *err = msg;
  return false;
}

}  // namespace

bool derive(const spr_config& c, Dims* out, std::string* err) {
  if (c.n_layers < 1 || c.n_layers > 255) return fail(err, "n_layers must be in [1, 255]");
  if (c.head_dim != 64 && c.head_dim != 128) return fail(err, "head_dim must be 64 or 128");
  if (c.n_heads < 1 || c.n_kv_heads < 1 || c.n_heads % c.n_kv_heads != 0)
    return fail(err, "n_heads must be a positive multiple of n_kv_heads");
  if (c.n_heads / c.n_kv_heads > 16) return fail(err, "n_heads / n_kv_heads must be <= 16");
  if (c.d_model < 16 || c.d_model % 16 != 0) return fail(err, "d_model must be a positive multiple of 16");
  if (c.d_ff < 1 || c.vocab < 1) return fail(err, "d_ff and vocab must be >= 1");
  if (c.dtype != SPR_F32 && c.dtype != SPR_BF16) return fail(err, "dtype must be SPR_F32 or SPR_BF16");
  if (c.kv_dtype != SPR_F32 && c.kv_dtype != SPR_BF16) return fail(err, "kv_dtype must be SPR_F32 or SPR_BF16");
  if (c.dtype == SPR_F32 && c.kv_dtype != SPR_F32) return fail(err, "fp32 models keep an fp32 KV cache");
  if (c.kv_block != kKvBlock) return fail(err, "kv_block must be 16");
  if (c.max_slots < 1 || c.max_slots > 64) return fail(err, "max_slots must be in [1, 64]");
  if (c.max_ctx < 1 || c.max_ctx > (1 << 20)) return fail(err, "max_ctx must be in [1, 2^20]");
  if (c.kv_blocks < 1) return fail(err, "kv_blocks must be >= 1");
  if (!(c.rope_base > 0.0f) || !std::isfinite(c.rope_base)) return fail(err, "rope_base must be positive");
  if (!(c.rms_eps >= 0.0f) || !std::isfinite(c.rms_eps)) return fail(err, "rms_eps must be >= 0");
  if (static_cast<int64_t>(c.n_heads) * c.head_dim > (1 << 20) || c.d_ff > (1 << 24) || c.d_model > (1 << 20) ||
      c.vocab > (1 << 24))
    return fail(err, "dimension too large");
  Dims d{};
  d.L = c.n_layers;
  d.d = c.d_model;
  d.H = c.n_heads;
  d.Hkv = c.n_kv_heads;
  d.hd = c.head_dim;
  d.f = c.d_ff;
  d.V = c.vocab;
  d.G = c.n_heads / c.n_kv_heads;
  d.dtype = c.dtype;
  d.esize = c.dtype == SPR_BF16 ? 2 : 4;
  d.kblk = c.dtype == SPR_BF16 ? 32 : 16;
  d.kv_dtype = c.kv_dtype;
  d.kv_esize = c.kv_dtype == SPR_BF16 ? 2 : 4;
  d.qkv_rows = (d.H + 2 * d.Hkv) * d.hd;
  d.o_in = d.H * d.hd;
  d.nt_qkv = d.qkv_rows / 16;
  d.nt_o = d.d / 16;
  d.nt_13 = ceil_div(d.f, 8);
  d.nt_2 = d.d / 16;
  d.nt_lm = ceil_div(d.V, 16);
  d.kb_d = ceil_div(d.d, d.kblk);
  d.kb_o = ceil_div(d.o_in, d.kblk);
  d.kb_f = ceil_div(d.f, d.kblk);
  d.kb_max = d.kb_d;
  if (d.kb_o > d.kb_max) d.kb_max = d.kb_o;
  if (d.kb_f > d.kb_max) d.kb_max = d.kb_f;
  d.S = c.max_slots;
  d.max_ctx = c.max_ctx;
  d.mb = ceil_div(c.max_ctx, kKvBlock);
  d.nb = c.kv_blocks;
  d.rope_base = c.rope_base;
  d.eps = c.rms_eps;
  *out = d;
  return true;
}

Layout layout(const Dims& d) {
  Layout l{};
  const size_t F = kFragBytes;
  l.wqkv = align256(static_cast<size_t>(d.nt_qkv) * d.kb_d * F);
  l.wo = align256(static_cast<size_t>(d.nt_o) * d.kb_o * F);
  l.w13 = align256(static_cast<size_t>(d.nt_13) * d.kb_d * F);
  l.w2 = align256(static_cast<size_t>(d.nt_2) * d.kb_f * F);
  size_t off = 0;
  auto take = [&off](size_t bytes) {
    size_t at = off;
    off += align256(bytes);
    return at;
  };
  l.off_wqkv = take(l.wqkv * d.L);
  l.off_wo = take(l.wo * d.L);
  l.off_w13 = take(l.w13 * d.L);
  l.off_w2 = take(l.w2 * d.L);
  l.off_wlm = take(static_cast<size_t>(d.nt_lm) * d.kb_d * F);
  l.off_emb = take(static_cast<size_t>(d.V) * d.d * d.esize);
  l.off_rope = take(static_cast<size_t>(d.max_ctx) * (d.hd / 2) * 2 * sizeof(float));
  l.kv_layer_stride = static_cast<size_t>(d.nb) * d.Hkv * kKvBlock * d.hd * d.kv_esize;
  l.off_kc = take(l.kv_layer_stride * d.L);
  l.off_vc = take(l.kv_layer_stride * d.L);
  l.off_bt = take(static_cast<size_t>(d.S) * d.mb * sizeof(int32_t));
  // Per-row buffers hold a whole prefill chunk (decode passes use the first rows).
  l.off_x = take(static_cast<size_t>(kPrefillRows) * d.d * sizeof(float));
  // Activation records carry hi + lo parts for bf16 models, and the QKV
  // input (d features) hi + mid + lo.
  const size_t act_blocks = d.dtype == SPR_BF16
                                ? std::max(2 * static_cast<size_t>(d.kb_max), 3 * static_cast<size_t>(d.kb_d))
                                : static_cast<size_t>(d.kb_max);
  l.act_bytes = act_blocks * kPrefillRows * d.kblk * d.esize;
  l.off_act0 = take(l.act_bytes);
  l.off_act1 = take(l.act_bytes);
  l.off_q = take(static_cast<size_t>(kPrefillRows) * d.H * d.hd * sizeof(float));
  // Partials of decode attention's KV splits, or of the projections' split-K
  // slices (never both in one launch).
  const SplitNeed sn = split_need(d);
  l.part_floats = std::max(static_cast<size_t>(kMaxSplits) * d.H * (d.hd + 4), sn.part_floats);
  l.off_part = take(l.part_floats * sizeof(float));
  // Arrival counters: decode attention's, one per (row, KV head), or the
  // split-K groups'; zero between launches.
  l.n_cnt = std::max(kMaxRows * d.Hkv, sn.counters);
  l.off_cnt = take(static_cast<size_t>(l.n_cnt) * sizeof(int32_t));
  l.off_amax = take(static_cast<size_t>(d.nt_lm) * kMaxRows * 2 * sizeof(float));
  l.off_prow = take(static_cast<size_t>(kPrefillRows) * 4 * sizeof(int32_t));
  l.off_ptile = take(static_cast<size_t>(kPrefillTiles) * 4 * sizeof(int32_t));
  l.off_rs = take(static_cast<size_t>(kPrefillRows) * sizeof(float));
  l.total = off;
  return l;
}

SplitNeed split_need(const Dims& d) {
  // The largest partials come at 32 rows (two 16-row activation tiles): per
  // group and slice, 64 lanes x (rt x 2 x 4 accumulators, plus 2 sums of
  // squares for the normed projections) floats in whole pairs.
  auto need = [](int nt, SplitShape sh, bool norm) {
    const size_t pairs = (sh.rt * 2 * 4 + (norm ? 2 : 0) + 1) / 2;
    return SplitNeed{static_cast<size_t>(nt / sh.rt) * sh.s * pairs * 128, nt / sh.rt};
  };
  SplitNeed out{0, 0};
  for (const SplitNeed& n : {need(d.nt_o, kSplitO, false), need(d.nt_2, kSplitO, false),
                             need(d.nt_13, kSplitGU, true), need(d.nt_qkv, kSplitQKV, true)}) {
    out.part_floats = std::max(out.part_floats, n.part_floats);
    out.counters = std::max(out.counters, n.counters);
  }
  return out;
}

void SlotTable::init(const Dims& d) {
  d_ = d;
  slots_.assign(d.S, Slot{});
  free_.clear();
  free_.reserve(d.nb);
  for (int b = d.nb - 1; b >= 0; --b) free_.push_back(b);  // block 0 is handed out first
}

spr_status SlotTable::check_prefill(int n, const int32_t* slots, const int32_t* seq_lens, const int32_t* stop_lens,
                                    std::string* err) const {
  if (n < 1 || n > d_.S) {
    *err = "prefill: n must be in [1, max_slots]";
    return SPR_ERR_INVALID_ARG;
  }
  std::vector<char> seen(d_.S, 0);
  int64_t need = 0;
  for (int i = 0; i < n; ++i) {
    const int s = slots[i];
    if (s < 0 || s >= d_.S) {
      *err = "prefill: slot id out of range";
      return SPR_ERR_INVALID_ARG;
    }
    if (seen[s]) {
      *err = "prefill: slot listed twice";
      return SPR_ERR_INVALID_ARG;
    }
    seen[s] = 1;
    if (slots_[s].state != kFree) {
      *err = "prefill: slot " + std::to_string(s) + " is not free";
      return SPR_ERR_STATE;
    }
    if (seq_lens[i] < 1 || stop_lens[i] < 1) {
      *err = "prefill: seq_len and stop_len must be >= 1";
      return SPR_ERR_INVALID_ARG;
    }
    const int64_t positions = static_cast<int64_t>(seq_lens[i]) + stop_lens[i] - 1;
    if (positions > d_.max_ctx) {
      *err = "prefill: seq_len + stop_len - 1 exceeds max_ctx";
      return SPR_ERR_INVALID_ARG;
    }
    need += (positions + kKvBlock - 1) / kKvBlock;
  }
  if (need > static_cast<int64_t>(free_.size())) {
    *err = "prefill: KV pool has " + std::to_string(free_.size()) + " free blocks, " + std::to_string(need) +
           " needed";
    return SPR_ERR_KV_FULL;
  }
  return SPR_OK;
}

void SlotTable::commit_prefill(int n, const int32_t* slots, const int32_t* seq_lens, const int32_t* stop_lens,
                               int32_t* retired) {
  for (int i = 0; i < n; ++i) {
    Slot& sl = slots_[slots[i]];
    const int positions = seq_lens[i] + stop_lens[i] - 1;
    const int nblk = (positions + kKvBlock - 1) / kKvBlock;
    sl.blocks.clear();
    for (int b = 0; b < nblk; ++b) {
      sl.blocks.push_back(free_.back());
      free_.pop_back();
    }
    sl.len = seq_lens[i];
    sl.produced = 1;
    sl.stop = stop_lens[i];
    sl.state = sl.produced >= sl.stop ? kFinished : kActive;
    if (retired) retired[i] = sl.state == kFinished ? 1 : 0;
  }
}

spr_status SlotTable::check_decode(int n, const int32_t* slots, const int32_t* lens, std::string* err) const {
  if (n < 1 || n > d_.S) {
    *err = "decode_step: n_active must be in [1, max_slots]";
    return SPR_ERR_INVALID_ARG;
  }
  std::vector<char> seen(d_.S, 0);
  for (int i = 0; i < n; ++i) {
    const int s = slots[i];
    if (s < 0 || s >= d_.S) {
      *err = "decode_step: slot id out of range";
      return SPR_ERR_INVALID_ARG;
    }
    if (seen[s]) {
      *err = "decode_step: slot listed twice";
      return SPR_ERR_INVALID_ARG;
    }
    seen[s] = 1;
    const Slot& sl = slots_[s];
    if (sl.state != kActive) {
      *err = "decode_step: slot " + std::to_string(s) + (sl.state == kFree ? " is free" : " has finished");
      return SPR_ERR_STATE;
    }
    if (lens[i] != sl.len) {
      *err = "decode_step: slot " + std::to_string(s) + " has " + std::to_string(sl.len) + " cached positions, " +
             std::to_string(lens[i]) + " given";
      return SPR_ERR_STATE;
    }
  }
  return SPR_OK;
}

void SlotTable::commit_decode(int n, const int32_t* slots, int32_t* retired) {
  for (int i = 0; i < n; ++i) {
    Slot& sl = slots_[slots[i]];
    sl.len += 1;
    sl.produced += 1;
    const bool done = sl.produced >= sl.stop;
    if (done) sl.state = kFinished;
    if (retired) retired[i] = done ? 1 : 0;
  }
}

spr_status SlotTable::check_rewind(int slot, int len, int produced, std::string* err) const {
  if (slot < 0 || slot >= d_.S) {
    *err = "rewind: slot id out of range";
    return SPR_ERR_INVALID_ARG;
  }
  const Slot& sl = slots_[slot];
  if (sl.state == kFree) {
    *err = "rewind: slot is free";
    return SPR_ERR_STATE;
  }
  const int prompt = sl.len - sl.produced + 1;
  if (produced < 1 || produced > sl.produced || len != prompt + produced - 1) {
    *err = "rewind: need 1 <= produced <= current and len == prompt + produced - 1";
    return SPR_ERR_INVALID_ARG;
  }
  return SPR_OK;
}

void SlotTable::commit_rewind(int slot, int len, int produced) {
  Slot& sl = slots_[slot];
  sl.len = len;
  sl.produced = produced;
  sl.state = produced >= sl.stop ? kFinished : kActive;
}

spr_status SlotTable::check_free(int slot, std::string* err) const {
  if (slot < 0 || slot >= d_.S) {
    *err = "free_slot: slot id out of range";
    return SPR_ERR_INVALID_ARG;
  }
  if (slots_[slot].state == kFree) {
    *err = "free_slot: slot is already free";
    return SPR_ERR_STATE;
  }
  return SPR_OK;
}

void SlotTable::commit_free(int slot) {
  Slot& sl = slots_[slot];
  for (auto it = sl.blocks.rbegin(); it != sl.blocks.rend(); ++it) free_.push_back(*it);
  sl = Slot{};
}

void SlotTable::block_row(int slot, int32_t* row) const {
  const Slot& sl = slots_[slot];
  for (int b = 0; b < d_.mb; ++b) row[b] = b < static_cast<int>(sl.blocks.size()) ? sl.blocks[b] : 0;
}

spr_status serve(SlotTable& tab, const Dims& d, int n, const ServeRequest* reqs, int max_active, ServeDevice& dev,
                 ServeCounters* counters, std::vector<int32_t>* lengths, std::string* err) {
  if (n < 0 || (n > 0 && reqs == nullptr)) {
    *err = "serve: n must be >= 0 and requests non-null";
    return SPR_ERR_INVALID_ARG;
  }
  if (max_active < 1 || max_active > d.S) {
    *err = "serve: max_active must be in [1, max_slots]";
    return SPR_ERR_INVALID_ARG;
  }
  for (int s = 0; s < d.S; ++s) {
    if (tab.slot(s).state != kFree) {
      *err = "serve: every slot must be free";
      return SPR_ERR_STATE;
    }
  }
  for (int i = 0; i < n; ++i) {
    const ServeRequest& r = reqs[i];
    if (r.tokens == nullptr || r.n_tokens < 1 || r.stop_len < 1 || r.arrival < 0) {
      *err = "serve: request " + std::to_string(i) + " is malformed";
      return SPR_ERR_INVALID_ARG;
    }
    for (int t = 0; t < r.n_tokens; ++t) {
      if (r.tokens[t] < 0 || r.tokens[t] >= d.V) {
        *err = "serve: request " + std::to_string(i) + " has a token id out of range";
        return SPR_ERR_INVALID_ARG;
      }
    }
    if (static_cast<int64_t>(r.n_tokens) + r.stop_len - 1 > d.max_ctx ||
        SlotTable::blocks_for(r.n_tokens, r.stop_len) > tab.free_blocks()) {
      *err = "serve: request " + std::to_string(i) + " can never fit (max_ctx or KV pool)";
      return SPR_ERR_INVALID_ARG;
    }
  }
  struct Live {
    int slot, req, len, produced;
  };
  std::vector<Live> live;
  std::vector<char> busy(d.S, 0);
  std::vector<int32_t> length(n);
  for (int i = 0; i < n; ++i) length[i] = reqs[i].stop_len;
  std::vector<std::pair<int, int>> eos;
  auto note_eos = [&]() {  // record EOS lengths; retire requests still in flight
    for (const auto& e : eos) {
      if (e.second + 1 < length[e.first]) length[e.first] = e.second + 1;
      for (size_t i = 0; i < live.size(); ++i) {
        if (live[i].req == e.first) {
          tab.commit_free(live[i].slot);
          busy[live[i].slot] = 0;
          live.erase(live.begin() + static_cast<std::ptrdiff_t>(i));
          break;
        }
      }
    }
    eos.clear();
  };
  ServeCounters c;
  int64_t batch_sum = 0;
  int q = 0;
  int it = 0;
  std::vector<int32_t> s0, s1, s2, s3, s4, ret;
  while (q < n || !live.empty()) {
    dev.iteration = it;
    // 1-2: admissions and their prefill.
    s0.clear();
    s1.clear();
    s2.clear();
    s3.clear();
    int reserve = 0;
    while (q < n && reqs[q].arrival <= it && static_cast<int>(live.size() + s0.size()) < max_active) {
      const int need = SlotTable::blocks_for(reqs[q].n_tokens, reqs[q].stop_len);
      if (need > tab.free_blocks() - reserve) break;
      int slot = 0;
      while (busy[slot]) ++slot;
      busy[slot] = 1;
      reserve += need;
      s0.push_back(slot);
      s1.push_back(q);
      s2.push_back(reqs[q].n_tokens);
      s3.push_back(reqs[q].stop_len);
      ++q;
    }
    if (!s0.empty()) {
      const int k = static_cast<int>(s0.size());
      spr_status st = tab.check_prefill(k, s0.data(), s2.data(), s3.data(), err);
      if (st != SPR_OK) return st;
      ret.assign(k, 0);
      tab.commit_prefill(k, s0.data(), s2.data(), s3.data(), ret.data());
      if ((st = dev.prefill(k, s0.data(), s1.data())) != SPR_OK) return st;
      ++c.prefill_calls;
      for (int i = 0; i < k; ++i) {
        if (ret[i]) {
          tab.commit_free(s0[i]);
          busy[s0[i]] = 0;
        } else {
          live.push_back(Live{s0[i], s1[i], s2[i], 1});
        }
      }
    }
    // 3-4: one decode step, retirements.
    if (!live.empty()) {
      const int k = static_cast<int>(live.size());
      s0.resize(k);
      s1.resize(k);
      s2.resize(k);
      s4.resize(k);
      for (int i = 0; i < k; ++i) {
        s0[i] = live[i].slot;
        s1[i] = live[i].len;
        s2[i] = live[i].req;
        s4[i] = live[i].produced;
      }
      spr_status st = tab.check_decode(k, s0.data(), s1.data(), err);
      if (st != SPR_OK) return st;
      if ((st = dev.decode(k, s0.data(), s1.data(), s2.data(), s4.data())) != SPR_OK) return st;
      ret.assign(k, 0);
      tab.commit_decode(k, s0.data(), ret.data());
      ++c.decode_steps;
      c.decode_tokens += k;
      batch_sum += k;
      if (k > c.max_batch) c.max_batch = k;
      std::vector<Live> keep;
      keep.reserve(k);
      for (int i = 0; i < k; ++i) {
        Live l = live[i];
        l.len += 1;
        l.produced += 1;
        if (ret[i]) {
          tab.commit_free(l.slot);
          busy[l.slot] = 0;
        } else {
          keep.push_back(l);
        }
      }
      live.swap(keep);
    }
    spr_status st = dev.end_iteration(false, &eos);
    if (st != SPR_OK) return st;
    note_eos();
    ++c.iterations;
    ++it;
    if (live.empty() && q < n && reqs[q].arrival > it) it = reqs[q].arrival;  // idle until the next arrival
  }
  spr_status st = dev.end_iteration(true, &eos);
  if (st != SPR_OK) return st;
  note_eos();
  c.mean_batch = c.decode_steps > 0 ? static_cast<double>(batch_sum) / c.decode_steps : 0.0;
  if (counters) *counters = c;
  if (lengths) *lengths = length;
  return SPR_OK;
}

}  // namespace spr
