// CPU-only shim over the host-side protocol (pw_state.cpp) for the test suite:
// the same allocator and requant / commit / reclaim state machine the library
// runs, driven by a simulated event clock instead of HIP events. No device
// memory is touched; a "launch" only records what would be enqueued.
#include <cstdint>
#include <set>
#include <string>
#include <vector>

#include "pw.h"
#include "pw_state.hpp"

namespace {

struct FakeEvents : pw::EventOps {
  uintptr_t next = 1;
  std::set<uintptr_t> live, completed;
  void* create() override {
    live.insert(next);
    return reinterpret_cast<void*>(next++);
  }
  void destroy(void* ev) override { live.erase(reinterpret_cast<uintptr_t>(ev)); }
  bool done(void* ev) override { return completed.count(reinterpret_cast<uintptr_t>(ev)) != 0; }
};

struct Handle {
  FakeEvents ev;
  pw::LayerState st;
  Handle(const pw_layer_desc& d, uint64_t bytes) : st(d, bytes, &ev) {}
};

thread_local std::string g_msg;

}  // namespace

extern "C" {

const char* pwt_last_error(void) { return g_msg.c_str(); }

void* pwt_create(const pw_layer_desc* d, uint64_t pool_bytes) {
  if (!pw::LayerState::valid_desc(*d, &g_msg)) return nullptr;
  return new Handle(*d, pool_bytes);
}

void pwt_destroy(void* h) { delete static_cast<Handle*>(h); }

int pwt_load(void* hv, int e, int proj, int rb, int bits) {
  Handle* h = static_cast<Handle*>(hv);
  pw_page_entry ent{};
  pw_status s = h->st.plan_load(e, proj, rb, bits, &ent, &g_msg);
  if (s == PW_OK) h->st.finish_load(e, proj, rb, ent);
  return s;
}

int pwt_load_apl(void* hv, int e, int proj, int rb, int bits) {
  Handle* h = static_cast<Handle*>(hv);
  pw_page_entry ent{};
  pw_status s = h->st.plan_load_apl(e, proj, rb, bits, &ent, &g_msg);
  if (s == PW_OK) h->st.finish_load(e, proj, rb, ent);
  return s;
}

// Requantize a batch; on success returns the batch's (simulated) event id.
int pwt_requant(void* hv, int n, const int* e, const int* proj, const int* rb, const int* nb,
                uint64_t* delta_total, uint64_t* event_id) {
  Handle* h = static_cast<Handle*>(hv);
  struct P { int e, proj, rb; pw_page_entry src, dst; };
  std::vector<P> plan;
  std::set<size_t> seen;
  uint64_t tot = 0;
  *event_id = 0;
  for (int i = 0; i < n; ++i) {
    P p{e[i], proj[i], rb[i], {}, {}};
    uint64_t d = 0;
    pw_status s = PW_OK;
    if (!h->st.check_block(p.e, p.proj, p.rb, &g_msg)) s = PW_EINVAL;
    else if (!seen.insert(h->st.index(p.e, p.proj, p.rb)).second) { g_msg = "duplicate"; s = PW_EINVAL; }
    else s = h->st.plan_requant(p.e, p.proj, p.rb, nb[i], &p.src, &p.dst, &d, &g_msg);
    if (s != PW_OK) {
      for (const P& q : plan) h->st.abort_slot(q.dst, q.proj);
      return s;
    }
    if (p.dst.bits == 0) continue;
    tot += d;
    plan.push_back(p);
  }
  *delta_total = tot;
  if (plan.empty()) return PW_OK;
  void* ev = h->ev.create();
  h->st.ref_event(ev);
  for (const P& p : plan) h->st.add_pending(p.e, p.proj, p.rb, p.dst, ev);
  h->st.unref_event(ev);
  *event_id = reinterpret_cast<uintptr_t>(ev);
  return PW_OK;
}

// Commit all pending blocks; returns the commit event id (0 if none).
uint64_t pwt_commit(void* hv, int* n) {
  Handle* h = static_cast<Handle*>(hv);
  *n = static_cast<int>(h->st.pending().size());
  if (*n == 0) return 0;
  void* cev = h->ev.create();
  h->st.committed(cev);
  return reinterpret_cast<uintptr_t>(cev);
}

void pwt_complete(void* hv, uint64_t ev) { static_cast<Handle*>(hv)->ev.completed.insert(ev); }

uint64_t pwt_reclaim(void* hv) { return static_cast<Handle*>(hv)->st.reclaim(); }

int pwt_entry(void* hv, int e, int proj, int rb, pw_page_entry* out) {
  Handle* h = static_cast<Handle*>(hv);
  if (!h->st.check_block(e, proj, rb, &g_msg)) return PW_EINVAL;
  *out = h->st.mirror[h->st.index(e, proj, rb)];
  return PW_OK;
}

void pwt_stats(void* hv, uint64_t* used, uint64_t* free_b, uint64_t* largest, uint64_t* live_events) {
  Handle* h = static_cast<Handle*>(hv);
  *used = h->st.alloc.used();
  *free_b = h->st.alloc.free_bytes();
  *largest = h->st.alloc.largest_free();
  *live_events = h->ev.live.size();
}

void pwt_set_host_pool(void* hv, uint64_t bytes) { static_cast<Handle*>(hv)->st.set_host_pool(bytes); }

// Offload a batch (the library's order: plan all, then register under one
// event); returns the status and the batch's event id (0: nothing copied).
int pwt_offload(void* hv, int n, const int* e, const int* proj, const int* rb, uint64_t* event_id) {
  Handle* h = static_cast<Handle*>(hv);
  struct P { int e, proj, rb; pw_page_entry src; uint64_t off; };
  std::vector<P> plan;
  std::set<size_t> seen;
  *event_id = 0;
  for (int i = 0; i < n; ++i) {
    P p{e[i], proj[i], rb[i], {}, 0};
    bool same = false;
    pw_status s = PW_OK;
    if (!h->st.check_block(p.e, p.proj, p.rb, &g_msg)) s = PW_EINVAL;
    else if (!seen.insert(h->st.index(p.e, p.proj, p.rb)).second) { g_msg = "duplicate"; s = PW_EINVAL; }
    else s = h->st.plan_offload(p.e, p.proj, p.rb, &p.src, &p.off, &same, &g_msg);
    if (s != PW_OK) {
      for (const P& q : plan) h->st.halloc.release(q.off, h->st.entry_bytes(q.proj, q.src));
      return s;
    }
    if (!same) plan.push_back(p);
  }
  if (plan.empty()) return PW_OK;
  void* ev = h->ev.create();
  h->st.ref_event(ev);
  for (const P& p : plan)
    h->st.finish_offload(p.e, p.proj, p.rb, p.off, p.src.bits, (p.src.rsv & 0xFF) == PW_FMT_APL, ev);
  h->st.unref_event(ev);
  *event_id = reinterpret_cast<uintptr_t>(ev);
  return PW_OK;
}

int pwt_reload(void* hv, int n, const int* e, const int* proj, const int* rb, uint64_t* added,
               uint64_t* event_id) {
  Handle* h = static_cast<Handle*>(hv);
  struct P { int e, proj, rb; pw_page_entry dst; pw::HostCopy hc; };
  std::vector<P> plan;
  std::set<size_t> seen;
  uint64_t tot = 0;
  *event_id = 0;
  *added = 0;
  for (int i = 0; i < n; ++i) {
    P p{e[i], proj[i], rb[i], {}, {}};
    uint64_t a = 0;
    pw_status s = PW_OK;
    if (!h->st.check_block(p.e, p.proj, p.rb, &g_msg)) s = PW_EINVAL;
    else if (!seen.insert(h->st.index(p.e, p.proj, p.rb)).second) { g_msg = "duplicate"; s = PW_EINVAL; }
    else s = h->st.plan_reload(p.e, p.proj, p.rb, &p.dst, &p.hc, &a, &g_msg);
    if (s != PW_OK) {
      for (const P& q : plan) h->st.abort_slot(q.dst, q.proj);
      return s;
    }
    tot += a;
    plan.push_back(p);
  }
  if (plan.empty()) return PW_OK;
  void* ev = h->ev.create();
  h->st.ref_event(ev);
  for (const P& p : plan) h->st.add_reload_pending(p.e, p.proj, p.rb, p.dst, ev);
  h->st.unref_event(ev);
  *added = tot;
  *event_id = reinterpret_cast<uintptr_t>(ev);
  return PW_OK;
}

int pwt_drop_host_copy(void* hv, int e, int proj, int rb) {
  Handle* h = static_cast<Handle*>(hv);
  if (!h->st.check_block(e, proj, rb, &g_msg)) return PW_EINVAL;
  h->st.drop_host_copy(e, proj, rb);
  return PW_OK;
}

// Host copy of a block: bitwidth (0: none), slot offset and its transfer event.
int pwt_host_copy(void* hv, int e, int proj, int rb, int* bits, uint64_t* off, uint64_t* event_id) {
  Handle* h = static_cast<Handle*>(hv);
  if (!h->st.check_block(e, proj, rb, &g_msg)) return PW_EINVAL;
  const pw::HostCopy& c = h->st.host[h->st.index(e, proj, rb)];
  *bits = c.bits;
  *off = c.off;
  *event_id = reinterpret_cast<uintptr_t>(c.ev);
  return PW_OK;
}

void pwt_host_stats(void* hv, uint64_t* capacity, uint64_t* used) {
  Handle* h = static_cast<Handle*>(hv);
  *capacity = h->st.halloc.capacity();
  *used = h->st.halloc.used();
}

int pwt_all_present(void* hv) { return static_cast<Handle*>(hv)->st.all_present() ? 1 : 0; }

}  // extern "C"
