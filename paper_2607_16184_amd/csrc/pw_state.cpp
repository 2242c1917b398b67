// Host-side slot allocator and page-table protocol (see pw_state.hpp).
#include "pw_state.hpp"

#include <algorithm>

namespace pw {

SlotAllocator::SlotAllocator(uint64_t capacity) : cap_(capacity / kSlotAlign * kSlotAlign) {
  if (cap_) free_[0] = cap_;
}

bool SlotAllocator::alloc(uint64_t bytes, uint64_t* off) {
  const uint64_t need = round_up(bytes);
  if (need == 0) return false;
  for (auto it = free_.begin(); it != free_.end(); ++it) {
    if (it->second >= need) {
      *off = it->first;
      const uint64_t rest = it->second - need;
      const uint64_t start = it->first + need;
      free_.erase(it);
      if (rest) free_[start] = rest;
      used_ += need;
      return true;
    }
  }
  return false;
}

void SlotAllocator::release(uint64_t off, uint64_t bytes) {
  const uint64_t len = round_up(bytes);
  used_ -= len;
  auto next = free_.lower_bound(off);
  uint64_t start = off, end = off + len;
  if (next != free_.end() && next->first == end) {
    end += next->second;
    next = free_.erase(next);
  }
  if (next != free_.begin()) {
    auto prev = std::prev(next);
    if (prev->first + prev->second == start) {
      start = prev->first;
      free_.erase(prev);
    }
  }
  free_[start] = end - start;
}

uint64_t SlotAllocator::largest_free() const {
  uint64_t m = 0;
  for (const auto& kv : free_) m = std::max(m, kv.second);
  return m;
}

bool LayerState::valid_desc(const pw_layer_desc& d, std::string* err) {
  auto bad = [&](const char* m) { *err = m; return false; };
  if (d.E <= 0 || d.H <= 0 || d.F <= 0 || d.R <= 0 || d.G <= 0) return bad("non-positive layer dimension");
  if (d.act != PW_F16 && d.act != PW_BF16) return bad("act must be PW_F16 or PW_BF16");
  if (d.sdt != PW_F16 && d.sdt != PW_BF16) return bad("sdt must be PW_F16 or PW_BF16");
  if (d.R % 64) return bad("R must be a multiple of 64");
  if (d.F % d.R || d.H % d.R) return bad("F and H must be multiples of R");
  if (d.F % 128 || d.H % 128) return bad("F and H must be multiples of 128");
  // the kernels index groups by shifts and masks: G is a power of two
  if (d.G != 64 && d.G != 128 && d.G != 256 && d.G != 512) return bad("G must be 64, 128, 256 or 512");
  if (d.F % d.G || d.H % d.G) return bad("G must divide F and H");
  if (static_cast<int64_t>(d.F) * d.H >= (int64_t(1) << 31)) return bad("F*H too large");
  return true;
}

LayerState::LayerState(const pw_layer_desc& d, uint64_t pool_bytes, EventOps* ev)
    : desc(d), alloc(pool_bytes), evops_(ev) {
  nrb_max = std::max(d.F, d.H) / d.R;
  n_entries = static_cast<size_t>(d.E) * 3 * nrb_max;
  mirror.assign(n_entries, pw_page_entry{0, 0, 0, PW_PAGE_ABSENT, 0, 0});
  host.assign(n_entries, HostCopy{});
  n_pages = static_cast<size_t>(d.E) * (2 * (d.F / d.R) + d.H / d.R);
}

LayerState::~LayerState() {
  for (auto& kv : refs_) evops_->destroy(kv.first);
}

uint64_t LayerState::code_bytes(int proj, int bits) const {
  const uint64_t rk = static_cast<uint64_t>(desc.R) * kdim(proj);
  return bits == 16 ? 2 * rk : bits == 8 ? rk : rk / 2;
}

uint64_t LayerState::page_bytes(int proj, int bits) const {
  const uint64_t sz = bits == 16 ? 0 : 4ull * desc.R * (kdim(proj) / desc.G);
  return code_bytes(proj, bits) + sz;
}

uint64_t LayerState::apl_bytes(int proj, int bits) const {
  const uint64_t rk8 = static_cast<uint64_t>(desc.R) * kdim(proj) / 8;
  const uint64_t lut4 = 32ull * desc.R, lut8 = 512ull * desc.R;
  return bits == 8 ? 8 * rk8 + lut4 + lut8 : 4 * rk8 + lut4;
}

bool LayerState::check_block(int e, int proj, int rb, std::string* err) const {
  if (e < 0 || e >= desc.E) { *err = "expert index out of range"; return false; }
  if (proj < 0 || proj > 2) { *err = "projection must be PW_GATE, PW_UP or PW_DOWN"; return false; }
  if (rb < 0 || rb >= nrb(proj)) { *err = "row-block index out of range"; return false; }
  return true;
}

pw_status LayerState::plan_load(int e, int proj, int rb, int bits, pw_page_entry* ent,
                                std::string* err) {
  if (!check_block(e, proj, rb, err)) return PW_EINVAL;
  if (bits != 16 && bits != 8 && bits != 4) { *err = "bits must be 16, 8 or 4"; return PW_EINVAL; }
  if (mirror[index(e, proj, rb)].bits != 0) { *err = "page already present"; return PW_EBUSY; }
  uint64_t off = 0;
  if (!alloc.alloc(page_bytes(proj, bits), &off)) { *err = "pool exhausted"; return PW_ENOMEM; }
  ent->data_off = off;
  ent->sz_off = bits == 16 ? 0 : off + code_bytes(proj, bits);
  ent->bits = static_cast<uint8_t>(bits);
  ent->state = PW_PAGE_RESIDENT;
  ent->rsv = 0;
  ent->gen = 1;
  return PW_OK;
}

pw_status LayerState::plan_load_apl(int e, int proj, int rb, int bits, pw_page_entry* ent, std::string* err) {
  if (!check_block(e, proj, rb, err)) return PW_EINVAL;
  if (bits != 8 && bits != 4) { *err = "nested bit-plane pages hold 8 or 4 bits"; return PW_EINVAL; }
  if (desc.R % 16 || kdim(proj) % 128) { *err = "R must be a multiple of 16 and K of 128"; return PW_EINVAL; }
  if (mirror[index(e, proj, rb)].bits != 0) { *err = "page already present"; return PW_EBUSY; }
  uint64_t off = 0;
  if (!alloc.alloc(apl_bytes(proj, bits), &off)) { *err = "pool exhausted"; return PW_ENOMEM; }
  ent->data_off = off;
  ent->sz_off = off + 4 * (static_cast<uint64_t>(desc.R) * kdim(proj) / 8);   // LUT_4
  ent->bits = static_cast<uint8_t>(bits);
  ent->state = PW_PAGE_RESIDENT;
  ent->rsv = PW_FMT_APL;
  ent->gen = 1;
  return PW_OK;
}

void LayerState::finish_load(int e, int proj, int rb, const pw_page_entry& ent) {
  mirror[index(e, proj, rb)] = ent;
  ++n_present;
  if ((ent.rsv & 0xFF) == PW_FMT_APL) ++n_apl;
}

void LayerState::abort_slot(const pw_page_entry& ent, int proj) {
  if (ent.rsv & kInPlace) return;   // a plane drop allocated nothing
  alloc.release(ent.data_off, entry_bytes(proj, ent));
}

pw_status LayerState::plan_requant(int e, int proj, int rb, int new_bits, pw_page_entry* src,
                                   pw_page_entry* dst, uint64_t* delta, std::string* err) {
  *delta = 0;
  if (!check_block(e, proj, rb, err)) return PW_EINVAL;
  if (new_bits != 16 && new_bits != 8 && new_bits != 4) { *err = "bits must be 16, 8 or 4"; return PW_EINVAL; }
  const pw_page_entry& cur = mirror[index(e, proj, rb)];
  if (cur.bits == 0) { *err = "page not present"; return PW_ESTATE; }
  if (cur.state != PW_PAGE_RESIDENT) { *err = "a requantization or reload of this block is pending"; return PW_EBUSY; }
  if (new_bits == cur.bits) return PW_OK;
  if (new_bits > cur.bits) {
    *err = "raising a bitwidth needs a reload from a host copy (pw_reload_block)";
    return PW_EUNSUPPORTED;
  }
  if ((cur.rsv & 0xFF) == PW_FMT_APL) {
    // nested bit-planes: 8 -> 4 keeps planes 0-3 and LUT_4 where they are;
    // the page tail (planes 4-7, LUT_8) is freed after the commit
    if (cur.bits != 8 || new_bits != 4) { *err = "nested bit-plane pages go from 8 to 4 bits only"; return PW_EUNSUPPORTED; }
    *src = cur;
    *dst = cur;
    dst->bits = 4;
    dst->rsv = static_cast<uint16_t>(PW_FMT_APL | kInPlace);
    dst->gen = cur.gen + 1;
    *delta = apl_bytes(proj, 8) - apl_bytes(proj, 4);
    return PW_OK;
  }
  uint64_t off = 0;
  if (!alloc.alloc(page_bytes(proj, new_bits), &off)) { *err = "pool exhausted"; return PW_ENOMEM; }
  *src = cur;
  dst->data_off = off;
  dst->sz_off = off + code_bytes(proj, new_bits);
  dst->bits = static_cast<uint8_t>(new_bits);
  dst->state = PW_PAGE_RESIDENT;
  dst->rsv = 0;
  dst->gen = cur.gen + 1;
  *delta = page_bytes(proj, cur.bits) - page_bytes(proj, new_bits);
  return PW_OK;
}

void LayerState::ref_event(void* ev) { ++refs_[ev]; }

void LayerState::unref_event(void* ev) {
  auto it = refs_.find(ev);
  if (it == refs_.end()) return;
  if (--it->second == 0) {
    evops_->destroy(ev);
    refs_.erase(it);
  }
}

void LayerState::add_pending(int e, int proj, int rb, const pw_page_entry& dst, void* ev) {
  const size_t idx = index(e, proj, rb);
  mirror[idx].state = PW_PAGE_REQUANT_PENDING;
  pending_.push_back(Pending{idx, proj, dst, ev});
  ref_event(ev);
}

void LayerState::committed(void* commit_ev) {
  for (const Pending& p : pending_) {
    pw_page_entry& cur = mirror[p.idx];
    if (p.next.rsv & kInPlace) {
      const uint64_t keep = apl_bytes(p.proj, p.next.bits);
      retired_.push_back(Retired{cur.data_off + keep, apl_bytes(p.proj, cur.bits) - keep, commit_ev});
    } else {
      retired_.push_back(Retired{cur.data_off, entry_bytes(p.proj, cur), commit_ev});
    }
    ref_event(commit_ev);
    cur = published(p.next);
    unref_event(p.ev);
  }
  pending_.clear();
}

uint64_t LayerState::reclaim() {
  uint64_t freed = 0;
  std::vector<Retired> keep;
  for (const Retired& r : retired_) {
    if (evops_->done(r.ev)) {
      alloc.release(r.off, r.bytes);
      freed += SlotAllocator::round_up(r.bytes);
      unref_event(r.ev);
    } else {
      keep.push_back(r);
    }
  }
  retired_.swap(keep);
  std::vector<Retired> hkeep;
  for (const Retired& r : hretired_) {
    if (!r.ev || evops_->done(r.ev)) {
      halloc.release(r.off, r.bytes);
      if (r.ev) unref_event(r.ev);
    } else {
      hkeep.push_back(r);
    }
  }
  hretired_.swap(hkeep);
  return freed;
}

pw_status LayerState::plan_offload(int e, int proj, int rb, pw_page_entry* src, uint64_t* host_off, bool* same,
                                   std::string* err) {
  *same = false;
  if (!check_block(e, proj, rb, err)) return PW_EINVAL;
  if (!has_host_pool()) { *err = "no host pool (pw_layer_set_host_pool)"; return PW_ESTATE; }
  const size_t idx = index(e, proj, rb);
  const pw_page_entry& cur = mirror[idx];
  if (cur.bits == 0) { *err = "page not present"; return PW_ESTATE; }
  if (cur.state != PW_PAGE_RESIDENT) { *err = "a requantization or reload of this block is pending"; return PW_EBUSY; }
  const bool apl = (cur.rsv & 0xFF) == PW_FMT_APL;
  if (host[idx].bits == cur.bits && (host[idx].apl != 0) == apl) {
    *same = true;
    return PW_OK;
  }
  // the copy is the committed page: a bit-plane page's planes and LUTs of its
  // committed precision (the 8-bit page, or the 4-bit prefix)
  uint64_t off = 0;
  if (!halloc.alloc(entry_bytes(proj, cur), &off)) { *err = "host pool exhausted"; return PW_ENOMEM; }
  *src = cur;
  *host_off = off;
  return PW_OK;
}

void LayerState::finish_offload(int e, int proj, int rb, uint64_t host_off, int bits, bool apl, void* ev) {
  drop_host_copy(e, proj, rb);   // a copy at another bitwidth is replaced
  HostCopy& h = host[index(e, proj, rb)];
  h.off = host_off;
  h.bits = static_cast<uint8_t>(bits);
  h.apl = apl ? 1 : 0;
  h.ev = ev;
  ref_event(ev);
}

pw_status LayerState::plan_reload(int e, int proj, int rb, pw_page_entry* dst, HostCopy* hc, uint64_t* added,
                                  std::string* err) {
  *added = 0;
  if (!check_block(e, proj, rb, err)) return PW_EINVAL;
  const size_t idx = index(e, proj, rb);
  const pw_page_entry& cur = mirror[idx];
  if (cur.bits == 0) { *err = "page not present"; return PW_ESTATE; }
  if (cur.state != PW_PAGE_RESIDENT) { *err = "a requantization or reload of this block is pending"; return PW_EBUSY; }
  const HostCopy& h = host[idx];
  if (h.bits == 0) { *err = "the block has no host copy"; return PW_ESTATE; }
  if (h.bits <= cur.bits) { *err = "the host copy is not of a higher bitwidth"; return PW_EUNSUPPORTED; }
  if ((h.apl != 0) != ((cur.rsv & 0xFF) == PW_FMT_APL)) {
    *err = "the host copy and the committed page are of different formats";
    return PW_EUNSUPPORTED;
  }
  uint64_t off = 0;
  if (!alloc.alloc(host_bytes(proj, h), &off)) { *err = "pool exhausted"; return PW_ENOMEM; }
  dst->data_off = off;
  if (h.apl) {
    // the full page comes back; LUT_4 follows planes 0-3 as in a loaded page
    dst->sz_off = off + 4 * (static_cast<uint64_t>(desc.R) * kdim(proj) / 8);
    dst->rsv = PW_FMT_APL;
  } else {
    dst->sz_off = h.bits == 16 ? 0 : off + code_bytes(proj, h.bits);
    dst->rsv = 0;
  }
  dst->bits = h.bits;
  dst->state = PW_PAGE_RESIDENT;
  dst->gen = cur.gen + 1;
  *hc = h;
  *added = host_bytes(proj, h) - entry_bytes(proj, cur);
  return PW_OK;
}

void LayerState::add_reload_pending(int e, int proj, int rb, const pw_page_entry& dst, void* ev) {
  const size_t idx = index(e, proj, rb);
  mirror[idx].state = PW_PAGE_RELOAD_PENDING;
  pending_.push_back(Pending{idx, proj, dst, ev});
  ref_event(ev);
  // the host slot is read by this transfer: it stays allocated until the transfer completed
  HostCopy& h = host[idx];
  ref_event(ev);
  if (h.ev) unref_event(h.ev);
  h.ev = ev;
}

void LayerState::drop_host_copy(int e, int proj, int rb) {
  HostCopy& h = host[index(e, proj, rb)];
  if (h.bits == 0) return;
  hretired_.push_back(Retired{h.off, host_bytes(proj, h), h.ev});   // the reference moves along
  h = HostCopy{};
}

}  // namespace pw
