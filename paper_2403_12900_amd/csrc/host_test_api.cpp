// Host-only C entry points over the slot table and workspace layout, built
// with g++ into a separate test library so the bookkeeping that every
// spr_prefill / spr_decode_step call runs before enqueueing work can be
// exercised without a GPU.  Not part of the device library.
#include <string>
#include <vector>

#include "host_state.h"

namespace {
thread_local std::string g_err;
struct Host {
  spr::Dims d;
  spr::SlotTable tab;
};
}  // namespace

extern "C" {

size_t sprh_workspace_bytes(const spr_config* cfg) {
  spr::Dims d;
  std::string err;
  if (cfg == nullptr || !spr::derive(*cfg, &d, &err)) {
    g_err = err;
    return 0;
  }
  return spr::layout(d).total;
}

void* sprh_new(const spr_config* cfg) {
  spr::Dims d;
  std::string err;
  if (cfg == nullptr || !spr::derive(*cfg, &d, &err)) {
    g_err = err;
    return nullptr;
  }
  Host* h = new Host();
  h->d = d;
  h->tab.init(d);
  return h;
}

void sprh_delete(void* h) { delete static_cast<Host*>(h); }

int sprh_prefill(void* hp, int n, const int32_t* slots, const int32_t* seq, const int32_t* stop, int32_t* retired) {
  Host* h = static_cast<Host*>(hp);
  spr_status st = h->tab.check_prefill(n, slots, seq, stop, &g_err);
  if (st == SPR_OK) h->tab.commit_prefill(n, slots, seq, stop, retired);
  return st;
}

int sprh_decode(void* hp, int n, const int32_t* slots, const int32_t* lens, int32_t* retired) {
  Host* h = static_cast<Host*>(hp);
  spr_status st = h->tab.check_decode(n, slots, lens, &g_err);
  if (st == SPR_OK) h->tab.commit_decode(n, slots, retired);
  return st;
}

int sprh_rewind(void* hp, int slot, int len, int produced) {
  Host* h = static_cast<Host*>(hp);
  spr_status st = h->tab.check_rewind(slot, len, produced, &g_err);
  if (st == SPR_OK) h->tab.commit_rewind(slot, len, produced);
  return st;
}

int sprh_free(void* hp, int slot) {
  Host* h = static_cast<Host*>(hp);
  spr_status st = h->tab.check_free(slot, &g_err);
  if (st == SPR_OK) h->tab.commit_free(slot);
  return st;
}

int sprh_free_blocks(void* hp) { return static_cast<Host*>(hp)->tab.free_blocks(); }

int sprh_slot(void* hp, int slot, int32_t* len, int32_t* produced, int32_t* stop, int32_t* state) {
  const spr::Slot& s = static_cast<Host*>(hp)->tab.slot(slot);
  *len = s.len;
  *produced = s.produced;
  *stop = s.stop;
  *state = s.state;
  return 0;
}

void sprh_block_row(void* hp, int slot, int32_t* row) { static_cast<Host*>(hp)->tab.block_row(slot, row); }

const char* sprh_last_error(void) { return g_err.c_str(); }

// Runs the serving scheduler over a device that only records, per produced
// token (request r's token k at out index off[r] + k): the scheduler
// iteration (iter_out), the slot (slot_out) and the call that produced it
// (call_out: calls are numbered from 0, prefill and decode alike), and per
// decode call its batch size (batch_out, up to max_calls).  Token k of
// request eos_req[j] is taken to be the EOS id when k == eos_idx[j]
// (j < n_eos).  lengths_out[r] receives the scheduler's length of request r.
// counters[0..4] = iterations, decode steps, prefill calls, decode tokens,
// max batch.
int sprh_serve(void* hp, int n, const int32_t* n_tokens, const int32_t* stop, const int32_t* arrival, int max_active,
               int n_eos, const int32_t* eos_req, const int32_t* eos_idx, int32_t* iter_out, int32_t* slot_out,
               int32_t* call_out, int32_t* batch_out, int max_calls, int32_t* lengths_out, int64_t* counters) {
  Host* h = static_cast<Host*>(hp);
  std::vector<int32_t> off(n + 1, 0);
  int max_tok = 1;
  for (int i = 0; i < n; ++i) {
    off[i + 1] = off[i] + stop[i];
    if (n_tokens[i] > max_tok) max_tok = n_tokens[i];
  }
  std::vector<int32_t> zeros(max_tok, 0);  // prompt ids are irrelevant to the schedule
  std::vector<spr::ServeRequest> reqs(n);
  for (int i = 0; i < n; ++i) reqs[i] = spr::ServeRequest{zeros.data(), n_tokens[i], stop[i], arrival[i]};
  struct Rec : spr::ServeDevice {
    const int32_t* off = nullptr;
    int32_t *iter_out = nullptr, *slot_out = nullptr, *call_out = nullptr, *batch_out = nullptr;
    int max_calls = 0, calls = 0, decodes = 0;
    std::vector<std::pair<int, int>> eos_set, cur, prev;
    void put(int req, int k, int slot) {
      iter_out[off[req] + k] = iteration;
      slot_out[off[req] + k] = slot;
      call_out[off[req] + k] = calls;
      cur.emplace_back(req, k);
    }
    void hits(const std::vector<std::pair<int, int>>& v, std::vector<std::pair<int, int>>* eos) const {
      for (const auto& t : v)
        for (const auto& e : eos_set)
          if (e == t) eos->push_back(t);
    }
    spr_status end_iteration(bool final, std::vector<std::pair<int, int>>* eos) override {
      hits(prev, eos);
      if (final) {
        hits(cur, eos);
        cur.clear();
      }
      prev.swap(cur);
      cur.clear();
      return SPR_OK;
    }
    spr_status prefill(int m, const int32_t* slots, const int32_t* req) override {
      for (int i = 0; i < m; ++i) put(req[i], 0, slots[i]);
      ++calls;
      return SPR_OK;
    }
    spr_status decode(int m, const int32_t* slots, const int32_t*, const int32_t* req,
                      const int32_t* produced) override {
      for (int i = 0; i < m; ++i) put(req[i], produced[i], slots[i]);
      if (decodes < max_calls) batch_out[decodes] = m;
      ++decodes;
      ++calls;
      return SPR_OK;
    }
  } rec;
  rec.off = off.data();
  rec.iter_out = iter_out;
  rec.slot_out = slot_out;
  rec.call_out = call_out;
  rec.batch_out = batch_out;
  rec.max_calls = max_calls;
  for (int j = 0; j < n_eos; ++j) rec.eos_set.emplace_back(eos_req[j], eos_idx[j]);
  spr::ServeCounters c;
  std::vector<int32_t> lengths;
  const spr_status st = spr::serve(h->tab, h->d, n, reqs.data(), max_active, rec, &c, &lengths, &g_err);
  for (int i = 0; i < n && st == SPR_OK; ++i) lengths_out[i] = lengths[i];
  counters[0] = c.iterations;
  counters[1] = c.decode_steps;
  counters[2] = c.prefill_calls;
  counters[3] = c.decode_tokens;
  counters[4] = c.max_batch;
  return st;
}
}
