// Host-only C entry points over the slot table and workspace layout, built
// with g++ into a separate test library so the bookkeeping that every
// spr_prefill / spr_decode_step call runs before enqueueing work can be
// exercised without a GPU.  Not part of the device library.
#include <string>

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
}
