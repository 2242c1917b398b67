// Host-side state of a paged layer: the slot allocator inside the caller's
// pool, the host mirror of the page table and the requant / commit / reclaim
// protocol. Plain C++ with no HIP dependency: events are reached through the
// EventOps interface, which the library backs with HIP events and the CPU
// tests back with a simulated clock.
//
// Protocol (Sec. 3.1 offload order, Sec. 3.3 asynchronous page movement):
//   requant   -> a fresh slot is allocated and filled on a side stream; the
//                committed entry is unchanged (state REQUANT_PENDING);
//   commit    -> after the requant's event, the new entry is published on the
//                main stream; the old slot is retired, tagged with the commit
//                event (its last possible reader precedes that event);
//   reclaim   -> retired slots whose commit event completed go back to the
//                free list, so the bytes Delta = M^b - M^b' (Eq. 3) become
//                available to the caller (e.g. for KV-cache blocks).
// Host copies (Sec. 3.1 page states, offload order):
//   offload   -> the committed page is copied to a slot of the caller's
//                host pool (device-to-host on a stream); the block keeps its
//                GPU page, and its host copy becomes usable once the copy's
//                event completed;
//   reload    -> a host copy of a higher bitwidth goes back into a fresh
//                device slot (host-to-device on a stream, after the offload
//                finished); the block is pending like a requant and the
//                raised entry is published by the next commit;
//   drop      -> the host slot is freed once its last transfer completed.
#pragma once

#include <cstdint>
#include <map>
#include <string>
#include <vector>

#include "pw.h"

namespace pw {

constexpr uint64_t kSlotAlign = 256;

// First-fit allocator over byte offsets [0, capacity), 256-byte granules,
// coalescing neighbours on release.
class SlotAllocator {
 public:
  explicit SlotAllocator(uint64_t capacity);
  bool alloc(uint64_t bytes, uint64_t* off);
  void release(uint64_t off, uint64_t bytes);
  uint64_t capacity() const { return cap_; }
  uint64_t used() const { return used_; }
  uint64_t free_bytes() const { return cap_ - used_; }
  uint64_t largest_free() const;
  static uint64_t round_up(uint64_t b) { return (b + kSlotAlign - 1) / kSlotAlign * kSlotAlign; }

 private:
  std::map<uint64_t, uint64_t> free_;  // offset -> length
  uint64_t cap_;
  uint64_t used_ = 0;
};

struct EventOps {
  virtual ~EventOps() {}
  virtual void* create() = 0;          // nullptr on failure
  virtual void destroy(void* ev) = 0;
  virtual bool done(void* ev) = 0;     // true once the recorded work completed
};

// A block's copy in host memory.
struct HostCopy {
  uint64_t off = 0;      // byte offset in the host pool
  uint8_t bits = 0;      // bitwidth of the copy; 0: none
  uint8_t apl = 0;       // 1: a nested bit-plane page (planes and LUTs)
  void* ev = nullptr;    // the last transfer that touches the slot (reference held)
};

class LayerState {
 public:
  LayerState(const pw_layer_desc& d, uint64_t pool_bytes, EventOps* ev);
  ~LayerState();

  static bool valid_desc(const pw_layer_desc& d, std::string* err);

  const pw_layer_desc desc;
  int nrb_max;
  size_t n_entries;

  size_t index(int e, int proj, int rb) const {
    return (static_cast<size_t>(e) * 3 + proj) * nrb_max + rb;
  }
  int kdim(int proj) const { return proj == PW_DOWN ? desc.F : desc.H; }
  int rows(int proj) const { return proj == PW_DOWN ? desc.H : desc.F; }
  int nrb(int proj) const { return rows(proj) / desc.R; }
  uint64_t code_bytes(int proj, int bits) const;   // bytes of values / codes
  uint64_t page_bytes(int proj, int bits) const;   // Eq. 3's M^b
  // Nested bit-plane pages: b planes of R K / 8 bytes and the LUTs up to b.
  uint64_t apl_bytes(int proj, int bits) const;
  uint64_t entry_bytes(int proj, const pw_page_entry& e) const {
    return (e.rsv & 0xFF) == PW_FMT_APL ? apl_bytes(proj, e.bits) : page_bytes(proj, e.bits);
  }
  uint64_t host_bytes(int proj, const HostCopy& h) const {
    return h.apl ? apl_bytes(proj, h.bits) : page_bytes(proj, h.bits);
  }
  // A pending entry that reuses its block's slot (a bit-plane drop) carries
  // this flag until it is published.
  static constexpr uint16_t kInPlace = 0x100;
  static pw_page_entry published(pw_page_entry e) {
    e.rsv = static_cast<uint16_t>(e.rsv & ~kInPlace);
    return e;
  }
  size_t n_apl = 0;                // present nested bit-plane pages

  bool check_block(int e, int proj, int rb, std::string* err) const;
  bool all_present() const { return n_present == n_pages; }

  // Loading an absent page: reserve a slot and describe the new entry.
  pw_status plan_load(int e, int proj, int rb, int bits, pw_page_entry* ent, std::string* err);
  pw_status plan_load_apl(int e, int proj, int rb, int bits, pw_page_entry* ent, std::string* err);
  void finish_load(int e, int proj, int rb, const pw_page_entry& ent);
  void abort_slot(const pw_page_entry& ent, int proj);

  // Requantization to a lower bitwidth into a fresh slot.
  pw_status plan_requant(int e, int proj, int rb, int new_bits, pw_page_entry* src,
                         pw_page_entry* dst, uint64_t* delta, std::string* err);
  void add_pending(int e, int proj, int rb, const pw_page_entry& dst, void* ev);

  // Host pool and host copies.
  bool has_host_pool() const { return halloc.capacity() > 0; }
  void set_host_pool(uint64_t bytes) { halloc = SlotAllocator(bytes); }
  // Offload the committed page of a block: a fresh host slot (*host_off) for
  // *src's page; *same = true (no work) if a copy at the committed bitwidth
  // exists already.
  pw_status plan_offload(int e, int proj, int rb, pw_page_entry* src, uint64_t* host_off, bool* same,
                         std::string* err);
  void finish_offload(int e, int proj, int rb, uint64_t host_off, int bits, bool apl, void* ev);
  // Reload a block from its host copy into a fresh device slot (*dst), the
  // copy being of a higher bitwidth than the committed page; *added receives
  // M^b' - M^b.
  pw_status plan_reload(int e, int proj, int rb, pw_page_entry* dst, HostCopy* hc, uint64_t* added,
                        std::string* err);
  void add_reload_pending(int e, int proj, int rb, const pw_page_entry& dst, void* ev);
  // Forget a block's host copy; its slot is freed by reclaim once its last
  // transfer completed.
  void drop_host_copy(int e, int proj, int rb);

  struct Pending {
    size_t idx;
    int proj;
    pw_page_entry next;
    void* ev;   // requant / reload done event (shared by a batch; reference counted)
  };
  struct Retired {
    uint64_t off, bytes;
    void* ev;   // commit event (shared; reference counted)
  };

  const std::vector<Pending>& pending() const { return pending_; }
  // Publish all pending entries in the mirror; old slots retire on commit_ev.
  void committed(void* commit_ev);
  // Free retired slots whose event completed; returns bytes freed.
  uint64_t reclaim();

  void ref_event(void* ev);
  void unref_event(void* ev);

  std::vector<pw_page_entry> mirror;
  SlotAllocator alloc;
  std::vector<HostCopy> host;      // per table index
  SlotAllocator halloc{0};         // host pool (capacity 0: none)
  size_t n_pages = 0;
  size_t n_present = 0;

 private:
  EventOps* evops_;
  std::vector<Pending> pending_;
  std::vector<Retired> retired_;
  std::vector<Retired> hretired_;  // host slots waiting for their last transfer
  std::map<void*, int> refs_;
};

}  // namespace pw
