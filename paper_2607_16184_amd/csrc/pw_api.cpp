// C ABI of libpagedweight.so (declared in include/pw.h).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <set>
#include <string>
#include <vector>

#include "pw.h"
#include "pw_internal.hpp"
#include "pw_state.hpp"

namespace {

thread_local std::string g_err;

pw_status fail(pw_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

pw_status hip_fail(hipError_t e, const char* what) {
  return fail(PW_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

}  // namespace

namespace pw {
pw_status set_error(pw_status s, const char* msg) { return fail(s, msg); }
}  // namespace pw

namespace {

struct HipEvents : pw::EventOps {
  void* create() override {
    hipEvent_t ev = nullptr;
    if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) return nullptr;
    return ev;
  }
  void destroy(void* ev) override { (void)hipEventDestroy(static_cast<hipEvent_t>(ev)); }
  bool done(void* ev) override { return hipEventQuery(static_cast<hipEvent_t>(ev)) == hipSuccess; }
};

struct ProfRec {
  int phase;
  hipEvent_t a, b;
};

}  // namespace

struct pw_layer {
  HipEvents evops;
  pw::LayerState st;
  uint8_t* pool;
  pw_page_entry* table;
  uint8_t* host_pool = nullptr;   // caller's pinned host memory for page copies
  int n_shared = 0;               // the last n_shared experts are shared experts
  // a stream of the layer's device on which the second expert chain or the
  // shared experts' GEMMs run beside the others, and its fork/join events
  hipStream_t side = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  bool prof = false;
  std::vector<ProfRec> recs;
  double tot_ms[PW_NPHASE] = {};
  int64_t cnt[PW_NPHASE] = {};
  int chains = 2;                 // concurrent expert chains of a decode-sized GEMM call

  pw_layer(const pw_layer_desc& d, void* p, size_t bytes, pw_page_entry* t)
      : st(d, bytes, &evops), pool(static_cast<uint8_t*>(p)), table(t) {}
};

namespace {

// Records a timing event pair around one launch when profiling is enabled.
struct ProfScope {
  pw_layer* L;
  int phase;
  hipStream_t st;
  hipEvent_t a = nullptr, b = nullptr;
  ProfScope(pw_layer* l, int ph, hipStream_t s) : L(l), phase(ph), st(s) {
    if (L && L->prof && hipEventCreate(&a) == hipSuccess && hipEventCreate(&b) == hipSuccess)
      (void)hipEventRecord(a, st);
  }
  ~ProfScope() {
    if (a && b) {
      (void)hipEventRecord(b, st);
      L->recs.push_back(ProfRec{phase, a, b});
    }
  }
};

bool mult_of_256(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 255u) == 0; }

// Pool offsets travel to the requant kernel as 32-bit counts of 256 bytes.
constexpr uint64_t kMaxPoolBytes = uint64_t(1) << 40;

// Device workspace layout of pw_moe_paged_gemm.
enum class GemmPath { kDecode, kStream, kTiled };

// One expert range of a call, run by its own GEMM launches: the routed
// experts [0, E - n_shared), and the shared experts (the last n_shared, each
// used by every token). Its kernel path, the decode kernels' slot tiles per
// pass and the down projection's K splits follow the range's own slots.
struct RangePlan {
  int e0, ne;          // experts [e0, e0 + ne)
  size_t S;            // slots routed to them
  GemmPath path;
  int nsplit, kb_per_split, mtb;
};

struct WsLayout {
  size_t h_off, h_bytes, op_off, op_bytes, total;
  RangePlan r[2];      // routed, shared (ne = 0 without shared experts)
};

// Which GEMM kernels serve a range, from its expected slots per expert
// S / ne: up to 48, the decode kernels (weights streamed in registers, exact
// code-domain arithmetic, up to four 16-slot tiles per pass); up to 127, the
// streaming kernel with 64-slot tiles; from 128, the LDS-tiled 256 x 256
// kernel. The shared experts of a decode-sized batch are a few experts with a
// few hundred slots each: where the tiled kernel's tiles would not give every
// CU a workgroup, the streaming kernel's smaller tiles spread their work. The
// last two need 32/64-row staging inside one page, 128-row down blocks and
// 32-bit activation row offsets (and the tiled kernel 256-row down blocks).
constexpr size_t kCUs = 256;

GemmPath pick_path(const pw_layer_desc& d, size_t S, size_t S_all, int ne, bool apl, bool shared) {
  const size_t expect = (S + ne - 1) / ne;
  const bool fits = S_all * d.F * 2 < (size_t(1) << 32) && S_all * d.H * 2 < (size_t(1) << 32);
  const bool tiles = fits && d.G >= 64 && d.R % 64 == 0 && d.F % 128 == 0;
  // nested bit-plane pages are read by the streaming kernel only
  if (apl) return GemmPath::kStream;
  if (expect >= 128 && tiles && d.H % 256 == 0) {
    const size_t tiled_wgs = static_cast<size_t>(ne) * ((expect + 255) / 256) * (d.F / 128);
    return shared && tiled_wgs < kCUs ? GemmPath::kStream : GemmPath::kTiled;
  }
  if (expect > 48 && tiles && d.H % 128 == 0) return GemmPath::kStream;
  return GemmPath::kDecode;
}

RangePlan plan_range(const pw_layer_desc& d, int e0, int ne, size_t S, size_t S_all, bool apl) {
  RangePlan r{};
  r.e0 = e0;
  r.ne = ne;
  r.S = S;
  if (ne <= 0) {
    r.nsplit = 1;
    r.kb_per_split = d.F / 128;
    r.mtb = 1;
    return r;
  }
  const int nkbF = d.F / 128;
  const int expect = static_cast<int>((S + ne - 1) / ne);
  r.path = pick_path(d, S, S_all, ne, apl, e0 > 0);
  // The decode kernels split the down projection's K = F when too few
  // (expert, 64-row block) units exist to fill the chip; deterministic in
  // (desc, T, K). At four slot tiles a workgroup covers 256 rows, so fewer
  // workgroups result, and that is kept: with that many slots per expert the
  // fp32 partials of a split cost more than the fuller chip gains.
  int nsplit = 1;
  if (r.path == GemmPath::kDecode && S <= 4096) {
    const size_t active = std::min<size_t>(ne, S);
    const size_t units = active * (d.H / 64);
    nsplit = static_cast<int>(std::max<size_t>(1, std::min<size_t>(8, 2048 / std::max<size_t>(units, 1))));
  }
  // likewise the streaming kernel with 32-slot tiles (bit-plane layers at
  // decode sizes): 128-row down workgroups, two per CU
  if (r.path == GemmPath::kStream && apl && expect <= 24 && S <= 4096) {
    const size_t active = std::min<size_t>(ne, S);
    const size_t units = active * (d.H / 128);
    nsplit = static_cast<int>(std::max<size_t>(1, std::min<size_t>(8, 1024 / std::max<size_t>(units, 1))));
  }
  // and the tiled kernel in two when its down tiles (256 rows x 256 slots,
  // one workgroup per CU) would run fewer than three rounds on the chip (the
  // last, partly filled round then weighs less; three or four splits add
  // more partial-sum traffic than they save)
  if (r.path == GemmPath::kTiled) {
    const size_t tiles = (S / 256 + static_cast<size_t>(ne)) * (d.H / 256);
    nsplit = tiles < 3 * kCUs ? 2 : 1;
  }
  nsplit = std::min(nsplit, nkbF);
  // a split holds whole quantization groups (G = 256, 512 span 2, 4 blocks)
  const int bpg = d.G > 128 ? d.G / 128 : 1;
  r.kb_per_split = ((nkbF + nsplit - 1) / nsplit + bpg - 1) / bpg * bpg;
  r.nsplit = (nkbF + r.kb_per_split - 1) / r.kb_per_split;
  // slot tiles per pass of the decode kernels: 1, 2 or 4 (with 4, a wave
  // streams two 16-row weight tiles)
  r.mtb = expect <= 12 ? 1 : expect <= 20 ? 2 : 4;
  return r;
}

WsLayout ws_layout(const pw_layer_desc& d, int T, int K, bool apl, int n_shared) {
  WsLayout w{};
  const size_t S = static_cast<size_t>(T) * K;
  const size_t S_sh = static_cast<size_t>(T) * n_shared;
  w.r[0] = plan_range(d, 0, d.E - n_shared, S - S_sh, S, apl);
  w.r[1] = plan_range(d, d.E - n_shared, n_shared, S_sh, S, apl);
  auto al = [](size_t b) { return (b + 255) / 256 * 256; };
  w.h_off = 0;
  w.h_bytes = al(S * d.F * 2);
  w.op_off = w.h_bytes;
  w.op_bytes = al(static_cast<size_t>(std::max(w.r[0].nsplit, w.r[1].nsplit)) * S * d.H * 4);
  w.total = w.h_bytes + w.op_bytes;
  return w;
}

// Waits until the work already enqueued on `st` has finished, so that slots
// its kernels or copies write can be released after a later step of the same
// call failed (a failing call must not hand out memory still being written).
void drain(hipStream_t st) { (void)hipStreamSynchronize(st); }

pw_status check_hip_last(const char* what) {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? PW_OK : hip_fail(e, what);
}

// Load-time quantization (or 16-bit layout) of pages from 16-bit values, each
// job with its own K, up to kMaxQJobs per launch (profiled with the requant
// phase).
pw_status run_qjobs(pw_layer* L, const std::vector<pw::QJob>& jobs, hipStream_t st) {
  const pw_layer_desc& d = L->st.desc;
  const int span = d.G > 128 ? d.G / 128 : 1;
  for (size_t base = 0; base < jobs.size(); base += pw::kMaxQJobs) {
    pw::QJobBatch b{};
    b.n_jobs = static_cast<int>(std::min<size_t>(pw::kMaxQJobs, jobs.size() - base));
    b.R = d.R;
    b.G = d.G;
    b.act = d.act;
    b.sdt = d.sdt;
    uint32_t items = 0;
    for (int j = 0; j < b.n_jobs; ++j) {
      b.job[j] = jobs[base + j];
      b.job[j].item_base = items;
      items += static_cast<uint32_t>(d.R / 16) * static_cast<uint32_t>((b.job[j].K / 128) / span);
    }
    b.total_items = items;
    ProfScope ps(L, PW_PH_REQUANT, st);
    hipError_t e = pw::launch_qjobs(b, st);
    if (e != hipSuccess) return hip_fail(e, "page quantization launch");
  }
  return PW_OK;
}

// Requant of pool pages, grouped by (source, destination) bitwidths in the
// plan's order, kMaxRqJobs pages per launch. The kernel finds a page's
// scale/zero block right after its codes (the slot layout of the allocator).
struct RqPlanned {
  pw_page_entry src, dst;
  int proj;
};
pw_status run_requant(pw_layer* L, const std::vector<RqPlanned>& jobs, hipStream_t st) {
  const pw_layer_desc& d = L->st.desc;
  static const int kPairs[3][2] = {{16, 8}, {16, 4}, {8, 4}};
  if (d.H / 128 > 65535 || d.F / 128 > 65535)
    return fail(PW_EUNSUPPORTED, "requant: H and F must stay below 2^23 (16-bit block counts)");
  for (const RqPlanned& j : jobs) {
    bool known = false;
    for (const auto& pr : kPairs) known = known || (j.src.bits == pr[0] && j.dst.bits == pr[1]);
    if (!known) return fail(PW_EUNSUPPORTED, "requant supports 16 -> 8, 16 -> 4 and 8 -> 4 only");
    const bool sz_follows = (j.src.bits == 16 || j.src.sz_off == j.src.data_off + L->st.code_bytes(j.proj, j.src.bits)) &&
                            j.dst.sz_off == j.dst.data_off + L->st.code_bytes(j.proj, j.dst.bits);
    if (!sz_follows || (j.src.data_off | j.dst.data_off) % 256 != 0)
      return fail(PW_EINVAL, "requant: a slot is not laid out as codes then scale/zero words on a 256-byte boundary");
  }
  for (const auto& pr : kPairs) {
    pw::RqBatch b{};
    b.pool = L->pool;
    b.R = d.R;
    b.G = d.G;
    b.kb[0] = static_cast<uint16_t>(d.H / 128);
    b.kb[1] = static_cast<uint16_t>(d.F / 128);
    auto flush = [&]() -> pw_status {
      if (b.n_jobs == 0) return PW_OK;
      ProfScope ps(L, PW_PH_REQUANT, st);
      hipError_t e = pw::launch_requant(b, pr[0], pr[1], d.act, d.sdt, st);
      b.n_jobs = 0;
      for (uint32_t& w : b.kbit) w = 0u;
      return e == hipSuccess ? PW_OK : hip_fail(e, "requant launch");
    };
    for (const RqPlanned& j : jobs) {
      if (j.src.bits != pr[0] || j.dst.bits != pr[1]) continue;
      const int n = b.n_jobs++;
      b.src[n] = static_cast<uint32_t>(j.src.data_off / 256);
      b.dst[n] = static_cast<uint32_t>(j.dst.data_off / 256);
      if (j.proj == PW_DOWN) b.kbit[n >> 5] |= 1u << (n & 31);
      if (b.n_jobs == pw::kMaxRqJobs) {
        pw_status s = flush();
        if (s != PW_OK) return s;
      }
    }
    pw_status s = flush();
    if (s != PW_OK) return s;
  }
  return PW_OK;
}

pw_status write_entries(pw_layer* L, const std::vector<std::pair<size_t, pw_page_entry>>& w,
                        hipStream_t st) {
  for (size_t base = 0; base < w.size(); base += pw::kMaxEntryWrites) {
    pw::EntryWrites ew{};
    ew.n = static_cast<int>(std::min<size_t>(pw::kMaxEntryWrites, w.size() - base));
    for (int i = 0; i < ew.n; ++i) {
      ew.idx[i] = static_cast<uint32_t>(w[base + i].first);
      ew.ent[i] = w[base + i].second;
    }
    hipError_t e = pw::launch_entry_writes(L->table, ew, st);
    if (e != hipSuccess) return hip_fail(e, "page-table write");
  }
  return PW_OK;
}

// The layer's own stream and its fork/join events, created on the pool's
// device (default priority; no implicit synchronization with the null
// stream: the fork/join events order it).
hipError_t ensure_side(pw_layer* L) {
  if (L->side) return hipSuccess;
  hipPointerAttribute_t attr{};
  hipError_t e = hipPointerGetAttributes(&attr, L->pool);
  int cur = -1;
  if (e == hipSuccess) e = hipGetDevice(&cur);
  if (e == hipSuccess && attr.device != cur) e = hipSetDevice(attr.device);
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&L->side, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&L->fork, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&L->join, hipEventDisableTiming);
  if (cur >= 0 && attr.device != cur) (void)hipSetDevice(cur);
  if (e != hipSuccess) {
    if (L->side) (void)hipStreamDestroy(L->side);
    if (L->fork) (void)hipEventDestroy(L->fork);
    if (L->join) (void)hipEventDestroy(L->join);
    L->side = nullptr;
    L->fork = L->join = nullptr;
  }
  return e;
}

}  // namespace

extern "C" {

const char* pw_last_error(void) { return g_err.c_str(); }

const char* pw_status_str(pw_status s) {
  switch (s) {
    case PW_OK: return "PW_OK";
    case PW_EINVAL: return "PW_EINVAL";
    case PW_ENOMEM: return "PW_ENOMEM";
    case PW_EBUSY: return "PW_EBUSY";
    case PW_EUNSUPPORTED: return "PW_EUNSUPPORTED";
    case PW_EHIP: return "PW_EHIP";
    case PW_ESTATE: return "PW_ESTATE";
  }
  return "unknown";
}

size_t pw_table_entries(const pw_layer_desc* d) {
  if (!d || d->R <= 0) return 0;
  return static_cast<size_t>(d->E) * 3 * (std::max(d->F, d->H) / d->R);
}

pw_status pw_page_bytes(const pw_layer_desc* d, int proj, int bits, size_t* bytes) {
  std::string err;
  if (!d || !bytes) return fail(PW_EINVAL, "null argument");
  if (!pw::LayerState::valid_desc(*d, &err)) return fail(PW_EINVAL, err);
  if (proj < 0 || proj > 2) return fail(PW_EINVAL, "bad projection");
  if (bits != 16 && bits != 8 && bits != 4) return fail(PW_EINVAL, "bits must be 16, 8 or 4");
  const uint64_t K = proj == PW_DOWN ? d->F : d->H;
  const uint64_t rk = static_cast<uint64_t>(d->R) * K;
  *bytes = bits == 16 ? 2 * rk : (bits == 8 ? rk : rk / 2) + 4ull * d->R * (K / d->G);
  return PW_OK;
}

pw_status pw_layer_create(const pw_layer_desc* d, void* pool_dev, size_t pool_bytes,
                          pw_page_entry* table_dev, pw_layer** out) {
  std::string err;
  if (!d || !out || !pool_dev || !table_dev) return fail(PW_EINVAL, "null argument");
  *out = nullptr;
  if (!pw::LayerState::valid_desc(*d, &err)) return fail(PW_EINVAL, err);
  if (!mult_of_256(pool_dev)) return fail(PW_EINVAL, "pool must be 256-byte aligned");
  if (static_cast<uint64_t>(pool_bytes) > kMaxPoolBytes) return fail(PW_EINVAL, "pool larger than 2^40 bytes");
  if (reinterpret_cast<uintptr_t>(table_dev) & 7u) return fail(PW_EINVAL, "table must be 8-byte aligned");
  pw_layer* L = new pw_layer(*d, pool_dev, pool_bytes, table_dev);
  hipError_t e = pw::launch_clear_table(table_dev, L->st.n_entries, nullptr);
  if (e == hipSuccess) e = hipStreamSynchronize(nullptr);
  if (e != hipSuccess) {
    delete L;
    return hip_fail(e, "clearing the page table");
  }
  e = ensure_side(L);
  if (e != hipSuccess) {
    delete L;
    return hip_fail(e, "creating the layer's stream");
  }
  *out = L;
  return PW_OK;
}

pw_status pw_layer_destroy(pw_layer* L) {
  if (!L) return PW_OK;
  for (auto& r : L->recs) {
    (void)hipEventSynchronize(r.b);
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  if (L->side) {
    (void)hipStreamSynchronize(L->side);
    (void)hipStreamDestroy(L->side);
  }
  if (L->fork) (void)hipEventDestroy(L->fork);
  if (L->join) (void)hipEventDestroy(L->join);
  delete L;
  return PW_OK;
}

pw_status pw_layer_load_page(pw_layer* L, int e, int proj, int rb, int bits, const void* rows16,
                             void* stream) {
  if (!L || !rows16) return fail(PW_EINVAL, "null argument");
  std::string err;
  pw_page_entry ent{};
  pw_status s = L->st.plan_load(e, proj, rb, bits, &ent, &err);
  if (s != PW_OK) return fail(s, err);
  hipStream_t st = static_cast<hipStream_t>(stream);
  // 16-bit: the rows are laid out as tiles; 8/4-bit: quantized into tiles
  pw::QJob j{};
  j.K = L->st.kdim(proj);
  j.src = static_cast<const uint8_t*>(rows16);
  j.dst = L->pool + ent.data_off;
  j.dst_sz = bits == 16 ? nullptr : L->pool + ent.sz_off;
  j.dst_bits = static_cast<uint8_t>(bits);
  j.src_plain = 1;
  s = run_qjobs(L, {j}, st);
  if (s == PW_OK) s = write_entries(L, {{L->st.index(e, proj, rb), ent}}, st);
  if (s != PW_OK) {
    drain(st);
    L->st.abort_slot(ent, proj);
    return s;
  }
  L->st.finish_load(e, proj, rb, ent);
  return PW_OK;
}

static size_t apl_job_bytes(const pw_layer* L) {
  const pw_layer_desc& d = L->st.desc;
  const size_t R = static_cast<size_t>(d.R), Kmax = static_cast<size_t>(std::max(d.H, d.F));
  return (R * Kmax + R * pw::kAplScratchRow + 255) / 256 * 256;
}

pw_status pw_apl_workspace_bytes(const pw_layer* L, int n, size_t* bytes) {
  if (!L || !bytes || n < 0) return fail(PW_EINVAL, "bad argument");
  *bytes = static_cast<size_t>(std::min(n, pw::kMaxAplJobs)) * apl_job_bytes(L);
  return PW_OK;
}

pw_status pw_layer_load_pages_apl(pw_layer* L, int n, const int* e, const int* proj, const int* rb,
                                  const int* bits, const void* const* rows16, void* ws, size_t ws_bytes,
                                  void* stream) {
  if (!L || n < 0 || (n > 0 && (!e || !proj || !rb || !bits || !rows16 || !ws))) return fail(PW_EINVAL, "bad argument");
  if (n == 0) return PW_OK;
  const size_t jb = apl_job_bytes(L);
  if (ws_bytes < static_cast<size_t>(std::min(n, pw::kMaxAplJobs)) * jb)
    return fail(PW_ENOMEM, "workspace smaller than pw_apl_workspace_bytes");
  if (!mult_of_256(ws)) return fail(PW_EINVAL, "workspace must be 256-byte aligned");
  std::string err;
  std::set<size_t> seen;
  std::vector<pw_page_entry> ents(n);
  auto rollback = [&](int upto) {
    for (int i = 0; i < upto; ++i) L->st.abort_slot(ents[i], proj[i]);
  };
  for (int i = 0; i < n; ++i) {
    if (!rows16[i] || (reinterpret_cast<uintptr_t>(rows16[i]) & 1u)) {
      rollback(i);
      return fail(PW_EINVAL, "null or misaligned source rows");
    }
    pw_status s = L->st.plan_load_apl(e[i], proj[i], rb[i], bits[i], &ents[i], &err);
    if (s == PW_OK && !seen.insert(L->st.index(e[i], proj[i], rb[i])).second) {
      L->st.abort_slot(ents[i], proj[i]);
      s = PW_EINVAL;
      err = "a block appears twice in the batch";
    }
    if (s != PW_OK) {
      rollback(i);
      return fail(s, err);
    }
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* wsb = static_cast<uint8_t*>(ws);
  for (int base = 0; base < n; base += pw::kMaxAplJobs) {
    pw::AplBatch b{};
    b.n_jobs = std::min(pw::kMaxAplJobs, n - base);
    b.R = L->st.desc.R;
    b.act = L->st.desc.act;
    uint32_t rows = 0;
    for (int j = 0; j < b.n_jobs; ++j) {
      const int i = base + j;
      pw::AplJob& J = b.job[j];
      J.src = static_cast<const uint16_t*>(rows16[i]);
      J.page = L->pool + ents[i].data_off;
      J.codes = wsb + static_cast<size_t>(j) * jb;
      J.scratch = J.codes + static_cast<size_t>(b.R) * std::max(L->st.desc.H, L->st.desc.F);
      J.row_base = rows;
      J.K = L->st.kdim(proj[i]);
      J.bits = bits[i];
      rows += static_cast<uint32_t>(b.R);
    }
    b.total_rows = rows;
    hipError_t he = pw::launch_apl_quant(b, st);
    if (he == hipSuccess) he = pw::launch_apl_pack(b, st);
    if (he != hipSuccess) {
      drain(st);
      rollback(n);
      return hip_fail(he, "bit-plane quantization launch");
    }
  }
  std::vector<std::pair<size_t, pw_page_entry>> w;
  for (int i = 0; i < n; ++i) w.push_back({L->st.index(e[i], proj[i], rb[i]), ents[i]});
  pw_status s = write_entries(L, w, st);
  if (s != PW_OK) {
    drain(st);
    rollback(n);
    return s;
  }
  for (int i = 0; i < n; ++i) L->st.finish_load(e[i], proj[i], rb[i], ents[i]);
  return PW_OK;
}

pw_status pw_route_topk_shared(const float* logits, int T, int E, int K, int renorm, int n_shared,
                               const float* shared_gate, int32_t* ids, float* w, int32_t* offsets,
                               int32_t* sorted_slot, int32_t* slot_pos, void* stream) {
  if (T < 0 || E < 1 || K < 1 || K > E || K > 16 || n_shared < 0 || E + n_shared > 256)
    return fail(PW_EINVAL, "need 1 <= K <= E, K <= 16, n_shared >= 0, E + n_shared <= 256, T >= 0");
  const int Kt = K + n_shared;
  if (static_cast<int64_t>(T) * Kt >= (int64_t(1) << 31)) return fail(PW_EINVAL, "T*K too large");
  if (!offsets || (T > 0 && (!logits || !ids || !w || !sorted_slot || !slot_pos)))
    return fail(PW_EINVAL, "null argument");
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (pw::route_permute_fits(T, E, K, n_shared)) {
    // small batches: one launch routes and permutes
    hipError_t e = pw::launch_route_permute(logits, T, E, K, renorm, n_shared, shared_gate, ids, w, offsets,
                                            sorted_slot, slot_pos, st);
    return e == hipSuccess ? PW_OK : hip_fail(e, "router launch");
  }
  hipError_t e = pw::launch_route_topk(logits, T, E, K, renorm, n_shared, shared_gate, ids, w, st);
  if (e != hipSuccess) return hip_fail(e, "router launch");
  e = pw::launch_permute(ids, T, Kt, E + n_shared, offsets, sorted_slot, slot_pos, st);
  if (e != hipSuccess) return hip_fail(e, "permute launch");
  return PW_OK;
}

pw_status pw_route_topk(const float* logits, int T, int E, int K, int renorm, int32_t* ids,
                        float* w, int32_t* offsets, int32_t* sorted_slot, int32_t* slot_pos,
                        void* stream) {
  return pw_route_topk_shared(logits, T, E, K, renorm, 0, nullptr, ids, w, offsets, sorted_slot, slot_pos,
                              stream);
}


pw_status pw_layer_set_chains(pw_layer* L, int chains) {
  if (!L) return fail(PW_EINVAL, "null layer");
  if (chains != 1 && chains != 2) return fail(PW_EINVAL, "chains must be 1 or 2");
  L->chains = chains;
  return PW_OK;
}

pw_status pw_layer_set_shared_experts(pw_layer* L, int n_shared) {
  if (!L) return fail(PW_EINVAL, "null layer");
  if (n_shared < 0 || n_shared >= L->st.desc.E)
    return fail(PW_EINVAL, "need 0 <= n_shared < E (at least one routed expert)");
  L->n_shared = n_shared;
  return PW_OK;
}

pw_status pw_probe_read(const void* buf, size_t bytes, int nblocks, uint32_t* out, void* stream) {
  constexpr size_t kUnit = 8 * 4096;   // one round of the probe's loads per workgroup
  if (!buf || !out || nblocks < 1 || nblocks > (1 << 20)) return fail(PW_EINVAL, "need buf, out and 1 <= nblocks <= 2^20");
  if (bytes == 0 || bytes % (kUnit * static_cast<size_t>(nblocks)) != 0)
    return fail(PW_EINVAL, "bytes must be a positive multiple of nblocks * 32768");
  hipError_t e = pw::launch_probe_read(buf, bytes, nblocks, out, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? PW_OK : hip_fail(e, "read probe launch");
}

pw_status pw_probe_mfma(int iters, int nblocks, float* out, void* stream) {
  if (!out || iters < 1 || nblocks < 1 || nblocks > (1 << 20))
    return fail(PW_EINVAL, "need out, iters >= 1 and 1 <= nblocks <= 2^20");
  hipError_t e = pw::launch_probe_mfma(iters, nblocks, out, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? PW_OK : hip_fail(e, "MFMA probe launch");
}

pw_status pw_routing_stats(const void* rows, pw_dtype act, int n_rows, int dim, int rows_by_position,
                           const float* topk_w, const int32_t* offsets, const int32_t* sorted_slot, int T, int E,
                           int K, double* norm2_ws, double* stats, int accumulate, void* stream) {
  if (T < 0 || E < 1 || K < 1 || K > E || E > 4096) return fail(PW_EINVAL, "need T >= 0, 1 <= K <= E <= 4096");
  if (static_cast<int64_t>(T) * K >= (int64_t(1) << 31)) return fail(PW_EINVAL, "T*K too large");
  if (act != PW_F16 && act != PW_BF16) return fail(PW_EINVAL, "act must be PW_F16 or PW_BF16");
  const int want = rows_by_position ? T * K : T;
  if (n_rows != want) return fail(PW_EINVAL, rows_by_position ? "n_rows must be T*K" : "n_rows must be T");
  if (dim < 8 || dim % 8 != 0) return fail(PW_EINVAL, "dim must be a positive multiple of 8");
  if (!offsets || !stats || (T > 0 && (!rows || !topk_w || !sorted_slot || !norm2_ws)))
    return fail(PW_EINVAL, "null argument");
  if (reinterpret_cast<uintptr_t>(rows) & 15u) return fail(PW_EINVAL, "rows must be 16-byte aligned");
  hipError_t e = pw::launch_routing_stats(static_cast<const uint16_t*>(rows), act, n_rows, dim, rows_by_position,
                                          topk_w, offsets, sorted_slot, T * K, E, K, norm2_ws, stats, accumulate,
                                          static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "routing statistics launch");
  return PW_OK;
}

pw_status pw_workspace_bytes(const pw_layer* L, int T, int K, size_t* gemm_ws) {
  if (!L || !gemm_ws || T < 0 || K < 1) return fail(PW_EINVAL, "bad argument");
  if (L->n_shared > 0 && K <= L->n_shared) return fail(PW_EINVAL, "K must exceed the shared experts");
  *gemm_ws = ws_layout(L->st.desc, T, K, L->st.n_apl > 0, L->n_shared).total;
  return PW_OK;
}

pw_status pw_moe_paged_gemm(const pw_layer* Lc, const void* x, int T, int K, const float* topk_w,
                            const int32_t* offsets, const int32_t* sorted_slot,
                            const int32_t* slot_pos, void* y, int out_fp32, void* ws,
                            size_t ws_bytes, void* stream) {
  pw_layer* L = const_cast<pw_layer*>(Lc);
  if (!L) return fail(PW_EINVAL, "null layer");
  if (T < 0 || K < 1 || K > L->st.desc.E) return fail(PW_EINVAL, "need T >= 0 and 1 <= K <= E");
  if (L->n_shared > 0 && K <= L->n_shared)
    return fail(PW_EINVAL, "K counts the routed and the shared columns: it must exceed the shared experts");
  if (T == 0) return PW_OK;
  if (!x || !topk_w || !offsets || !sorted_slot || !slot_pos || !y || !ws)
    return fail(PW_EINVAL, "null argument");
  if (!L->st.all_present()) return fail(PW_ESTATE, "every page of the layer must be loaded");
  if (static_cast<int64_t>(T) * K >= (int64_t(1) << 31)) return fail(PW_EINVAL, "T*K too large");
  {
    // the GEMM kernels address activation and SwiGLU rows with 32-bit byte offsets
    const uint64_t S = static_cast<uint64_t>(T) * K, lim = uint64_t(1) << 32;
    if (S * L->st.desc.F * 2 >= lim || S * L->st.desc.H * 2 >= lim)
      return fail(PW_EUNSUPPORTED, "T*K*max(F,H)*2 must stay below 2^32 (split the batch)");
  }
  const WsLayout wl = ws_layout(L->st.desc, T, K, L->st.n_apl > 0, L->n_shared);
  if (L->st.n_apl > 0) {
    const pw_layer_desc& dd = L->st.desc;
    const size_t S = static_cast<size_t>(T) * K;
    if (!(S * dd.F * 2 < (size_t(1) << 32) && S * dd.H * 2 < (size_t(1) << 32)) || dd.R % 64 || dd.G < 64 ||
        dd.H % 128)
      return fail(PW_EUNSUPPORTED, "nested bit-plane pages need the streaming kernel's shapes");
  }
  if (ws_bytes < wl.total) return fail(PW_ENOMEM, "workspace smaller than pw_workspace_bytes");
  if (!mult_of_256(ws)) return fail(PW_EINVAL, "workspace must be 256-byte aligned");
  if ((reinterpret_cast<uintptr_t>(x) & 15u) || (reinterpret_cast<uintptr_t>(y) & 15u))
    return fail(PW_EINVAL, "x and y must be 16-byte aligned");
  const pw_layer_desc& d = L->st.desc;
  pw::GemmArgs a{};
  a.pool = L->pool;
  a.table = L->table;
  a.x = static_cast<const uint16_t*>(x);
  a.offsets = offsets;
  a.sorted_slot = sorted_slot;
  a.slot_pos = slot_pos;
  a.topk_w = topk_w;
  a.h = reinterpret_cast<uint16_t*>(static_cast<uint8_t*>(ws) + wl.h_off);
  a.opart = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + wl.op_off);
  a.y = y;
  a.E = d.E;
  a.H = d.H;
  a.F = d.F;
  a.R = d.R;
  a.G = d.G;
  a.nrb_max = L->st.nrb_max;
  a.topk = K;
  a.T = T;
  a.S = T * K;
  a.out_fp32 = out_fp32 ? 1 : 0;
  a.act = d.act;
  a.sdt = d.sdt;
  a.apl = L->st.n_apl > 0 ? 1 : 0;
  a.n_shared = L->n_shared;
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = hipSuccess;
  // Routed experts, then shared experts: each range with its own kernels.
  // Launch units: with shared experts, the shared range runs on the layer's
  // own stream beside the routed one (its few workgroups share the chip with
  // the routed ones instead of running alone after them); without, a
  // decode-sized routed range runs as two chains of gate/up then down over
  // the two halves of its experts, the second on the layer's stream, so that
  // the boundary between one chain's phases overlaps the other's GEMMs. The
  // layer's stream is forked from `stream` and joined back before the
  // combine. Units write disjoint rows of h and of the partials.
  struct Unit {
    RangePlan r;
    hipStream_t s;
  };
  Unit units[2];
  int nu = 0;
  const bool shared_fork = L->chains == 2 && L->side && wl.r[0].ne > 0 && wl.r[1].ne > 0;
  const bool split_routed =
      L->chains == 2 && L->side && wl.r[1].ne <= 0 && wl.r[0].path == GemmPath::kDecode && wl.r[0].ne >= 2;
  if (split_routed) {
    units[0] = Unit{wl.r[0], st};
    units[0].r.ne = wl.r[0].ne / 2;
    units[1] = Unit{wl.r[0], L->side};
    units[1].r.e0 = wl.r[0].e0 + units[0].r.ne;
    units[1].r.ne = wl.r[0].ne - units[0].r.ne;
    nu = 2;
  } else {
    for (int ri = 0; ri < 2; ++ri)
      if (wl.r[ri].ne > 0) units[nu++] = Unit{wl.r[ri], shared_fork && ri == 1 ? L->side : st};
  }
  const bool fork = shared_fork || split_routed;
  auto for_range = [&](const RangePlan& r) {
    a.e0 = r.e0;
    a.ne = r.ne;
    a.s_range = static_cast<int>(r.S);
    a.nsplit = r.nsplit;
    a.kb_per_split = r.kb_per_split;
    a.mtb = r.mtb;
  };
  const char* what = nullptr;
  {
    ProfScope span(L, PW_PH_GEMM, st);
    if (fork) {
      e = hipEventRecord(L->fork, st);
      if (e == hipSuccess) e = hipStreamWaitEvent(L->side, L->fork, 0);
      if (e != hipSuccess) return hip_fail(e, "forking the layer's stream");
    }
    for (int pass = 0; pass < 2 && e == hipSuccess; ++pass) {
      const bool gateup = pass == 0;
      for (int ui = 0; ui < nu && e == hipSuccess; ++ui) {
        const RangePlan& r = units[ui].r;
        for_range(r);
        hipStream_t rs = units[ui].s;
        ProfScope ps(L, gateup ? PW_PH_GATEUP : PW_PH_DOWN, rs);
        e = r.path == GemmPath::kTiled    ? pw::launch_tgemm(a, gateup, rs)
            : r.path == GemmPath::kStream ? pw::launch_sgemm(a, gateup, rs)
            : gateup                      ? pw::launch_gateup(a, rs)
                                          : pw::launch_down(a, rs);
        if (e != hipSuccess) what = gateup ? "gate/up launch" : "down launch";
      }
    }
    if (fork) {
      // joined even after a failed launch, so that `stream` never waits on a
      // branch that was left open
      hipError_t ej = hipEventRecord(L->join, L->side);
      if (ej == hipSuccess) ej = hipStreamWaitEvent(st, L->join, 0);
      if (e == hipSuccess && ej != hipSuccess) {
        e = ej;
        what = "joining the layer's stream";
      }
    }
  }
  if (e != hipSuccess) return hip_fail(e, what);
  a.nsplit = wl.r[0].nsplit;
  a.nsplit_sh = wl.r[1].nsplit;
  {
    ProfScope ps(L, PW_PH_COMBINE, st);
    e = pw::launch_combine(a, st);
  }
  if (e != hipSuccess) return hip_fail(e, "combine launch");
  return PW_OK;
}

pw_status pw_moe_paged_gemm_noalloc(const pw_layer* L, const void* x, int T, int K, const float* topk_w,
                                    const int32_t* offsets, const int32_t* sorted_slot, const int32_t* slot_pos,
                                    void* y, int out_fp32, void* stream) {
  if (!L) return fail(PW_EINVAL, "null layer");
  if (T < 0 || K < 1 || K > L->st.desc.E) return fail(PW_EINVAL, "need T >= 0 and 1 <= K <= E");
  if (L->n_shared > 0 && K <= L->n_shared) return fail(PW_EINVAL, "K must exceed the shared experts");
  if (T == 0) return PW_OK;
  if (static_cast<int64_t>(T) * K >= (int64_t(1) << 31)) return fail(PW_EINVAL, "T*K too large");
  const size_t need = ws_layout(L->st.desc, T, K, L->st.n_apl > 0, L->n_shared).total;
  if (need > pw::kStaticScratchBytes)
    return fail(PW_ENOMEM, "the call needs " + std::to_string(need) + " bytes of workspace, more than the " +
                               std::to_string(pw::kStaticScratchBytes) +
                               "-byte static scratch: use pw_moe_paged_gemm with a workspace");
  hipStream_t st = static_cast<hipStream_t>(stream);
  int dev = -1;
  hipError_t e = hipStreamGetDevice(st, &dev);
  if (e != hipSuccess) return hip_fail(e, "hipStreamGetDevice");
  void* ptr = nullptr;
  e = pw::static_scratch(dev, &ptr);
  if (e != hipSuccess) return hip_fail(e, "looking up the static scratch");
  return pw_moe_paged_gemm(L, x, T, K, topk_w, offsets, sorted_slot, slot_pos, y, out_fp32, ptr,
                           pw::kStaticScratchBytes, stream);
}

pw_status pw_requant_blocks(pw_layer* L, int n, const int* e, const int* proj, const int* rb,
                            const int* new_bits, void* side_stream, size_t* delta_total) {
  if (!L || n < 0 || (n > 0 && (!e || !proj || !rb || !new_bits)))
    return fail(PW_EINVAL, "bad argument");
  if (delta_total) *delta_total = 0;
  std::string err;
  struct Planned {
    int e, proj, rb;
    pw_page_entry src, dst;
  };
  std::vector<Planned> plan;
  std::set<size_t> seen;
  uint64_t delta_sum = 0;
  auto rollback = [&]() {
    for (const Planned& p : plan) L->st.abort_slot(p.dst, p.proj);
  };
  for (int i = 0; i < n; ++i) {
    Planned p{e[i], proj[i], rb[i], {}, {}};
    uint64_t delta = 0;
    std::string e2;
    if (!L->st.check_block(p.e, p.proj, p.rb, &e2)) {
      rollback();
      return fail(PW_EINVAL, e2);
    }
    if (!seen.insert(L->st.index(p.e, p.proj, p.rb)).second) {
      rollback();
      return fail(PW_EINVAL, "a block appears twice in the batch");
    }
    pw_status s = L->st.plan_requant(p.e, p.proj, p.rb, new_bits[i], &p.src, &p.dst, &delta, &err);
    if (s != PW_OK) {
      rollback();
      return fail(s, err);
    }
    if (delta == 0 && p.dst.bits == 0) continue;   // same bitwidth: nothing to do
    delta_sum += delta;
    plan.push_back(p);
  }
  if (plan.empty()) return PW_OK;
  hipStream_t st = static_cast<hipStream_t>(side_stream);
  // a device-to-host copy of a source page still in flight on another stream
  // must finish before the page can retire (commit waits on this batch)
  std::set<void*> waits;
  for (const Planned& p : plan) {
    void* hev = L->st.host[L->st.index(p.e, p.proj, p.rb)].ev;
    if (hev && !L->evops.done(hev)) waits.insert(hev);
  }
  for (void* w : waits) {
    hipError_t he = hipStreamWaitEvent(st, static_cast<hipEvent_t>(w), 0);
    if (he != hipSuccess) {
      rollback();
      return hip_fail(he, "hipStreamWaitEvent");
    }
  }
  // launches of up to kMaxRqJobs pages per bitwidth pair (pages of every
  // projection together, each with its K)
  std::vector<RqPlanned> jobs;
  for (const Planned& p : plan) {
    if (p.dst.rsv & pw::LayerState::kInPlace) continue;   // a bit-plane drop needs no kernel
    jobs.push_back(RqPlanned{p.src, p.dst, p.proj});
  }
  pw_status rs = run_requant(L, jobs, st);
  if (rs != PW_OK) {
    drain(st);
    rollback();
    return rs;
  }
  void* ev = L->evops.create();
  if (!ev) {
    drain(st);
    rollback();
    return fail(PW_EHIP, "hipEventCreate failed");
  }
  hipError_t he = hipEventRecord(static_cast<hipEvent_t>(ev), st);
  if (he != hipSuccess) {
    L->evops.destroy(ev);
    drain(st);
    rollback();
    return hip_fail(he, "hipEventRecord");
  }
  L->st.ref_event(ev);   // hold while the batch is registered
  for (const Planned& p : plan) L->st.add_pending(p.e, p.proj, p.rb, p.dst, ev);
  L->st.unref_event(ev);
  if (delta_total) *delta_total = delta_sum;
  return PW_OK;
}

pw_status pw_requant_block(pw_layer* L, int e, int proj, int rb, int new_bits, void* side_stream,
                           size_t* delta_bytes) {
  return pw_requant_blocks(L, 1, &e, &proj, &rb, &new_bits, side_stream, delta_bytes);
}

// ---------------------------------------------------------------------------
// Host copies of pages: offload (device -> host) and reload (host -> device)
// ---------------------------------------------------------------------------

pw_status pw_layer_set_host_pool(pw_layer* L, void* host_pool, size_t host_bytes) {
  if (!L || !host_pool || host_bytes == 0) return fail(PW_EINVAL, "bad argument");
  if (!mult_of_256(host_pool)) return fail(PW_EINVAL, "host pool must be 256-byte aligned");
  if (L->st.has_host_pool()) return fail(PW_EBUSY, "the layer already has a host pool");
  L->host_pool = static_cast<uint8_t*>(host_pool);
  L->st.set_host_pool(host_bytes);
  return PW_OK;
}

namespace {

// Records an event on `st` for a batch of transfers; nullptr (with the error
// set) on failure.
static void* record_event(pw_layer* L, hipStream_t st, pw_status* s) {
  void* ev = L->evops.create();
  if (!ev) {
    *s = fail(PW_EHIP, "hipEventCreate failed");
    return nullptr;
  }
  hipError_t he = hipEventRecord(static_cast<hipEvent_t>(ev), st);
  if (he != hipSuccess) {
    L->evops.destroy(ev);
    *s = hip_fail(he, "hipEventRecord");
    return nullptr;
  }
  return ev;
}

static bool check_batch(pw_layer* L, int n, const int* e, const int* proj, const int* rb, std::string* err) {
  std::set<size_t> seen;
  for (int i = 0; i < n; ++i) {
    if (!L->st.check_block(e[i], proj[i], rb[i], err)) return false;
    if (!seen.insert(L->st.index(e[i], proj[i], rb[i])).second) {
      *err = "a block appears twice in the batch";
      return false;
    }
  }
  return true;
}

}  // namespace

pw_status pw_offload_blocks(pw_layer* L, int n, const int* e, const int* proj, const int* rb, void* stream) {
  if (!L || n < 0 || (n > 0 && (!e || !proj || !rb))) return fail(PW_EINVAL, "bad argument");
  std::string err;
  if (!check_batch(L, n, e, proj, rb, &err)) return fail(PW_EINVAL, err);
  struct Planned {
    int e, proj, rb;
    pw_page_entry src;
    uint64_t host_off;
  };
  std::vector<Planned> plan;
  auto rollback = [&]() {
    for (const Planned& p : plan) L->st.halloc.release(p.host_off, L->st.entry_bytes(p.proj, p.src));
  };
  for (int i = 0; i < n; ++i) {
    Planned p{e[i], proj[i], rb[i], {}, 0};
    bool same = false;
    pw_status s = L->st.plan_offload(p.e, p.proj, p.rb, &p.src, &p.host_off, &same, &err);
    if (s != PW_OK) {
      rollback();
      return fail(s, err);
    }
    if (!same) plan.push_back(p);
  }
  if (plan.empty()) return PW_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  for (const Planned& p : plan) {
    hipError_t he = hipMemcpyAsync(L->host_pool + p.host_off, L->pool + p.src.data_off,
                                   L->st.entry_bytes(p.proj, p.src), hipMemcpyDeviceToHost, st);
    if (he != hipSuccess) {
      drain(st);
      rollback();
      return hip_fail(he, "device-to-host page copy");
    }
  }
  pw_status s = PW_OK;
  void* ev = record_event(L, st, &s);
  if (!ev) {
    drain(st);
    rollback();
    return s;
  }
  L->st.ref_event(ev);
  for (const Planned& p : plan)
    L->st.finish_offload(p.e, p.proj, p.rb, p.host_off, p.src.bits, (p.src.rsv & 0xFF) == PW_FMT_APL, ev);
  L->st.unref_event(ev);
  return PW_OK;
}

pw_status pw_offload_block(pw_layer* L, int e, int proj, int rb, void* stream) {
  return pw_offload_blocks(L, 1, &e, &proj, &rb, stream);
}

pw_status pw_reload_blocks(pw_layer* L, int n, const int* e, const int* proj, const int* rb, void* stream,
                           size_t* added_total) {
  if (!L || n < 0 || (n > 0 && (!e || !proj || !rb))) return fail(PW_EINVAL, "bad argument");
  if (added_total) *added_total = 0;
  std::string err;
  if (!check_batch(L, n, e, proj, rb, &err)) return fail(PW_EINVAL, err);
  struct Planned {
    int e, proj, rb;
    pw_page_entry dst;
    pw::HostCopy hc;
  };
  std::vector<Planned> plan;
  uint64_t added = 0;
  auto rollback = [&]() {
    for (const Planned& p : plan) L->st.abort_slot(p.dst, p.proj);
  };
  for (int i = 0; i < n; ++i) {
    Planned p{e[i], proj[i], rb[i], {}, {}};
    uint64_t a = 0;
    pw_status s = L->st.plan_reload(p.e, p.proj, p.rb, &p.dst, &p.hc, &a, &err);
    if (s != PW_OK) {
      rollback();
      return fail(s, err);
    }
    added += a;
    plan.push_back(p);
  }
  if (plan.empty()) return PW_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  // each host copy must have arrived before it is read back
  std::set<void*> waits;
  for (const Planned& p : plan)
    if (p.hc.ev && !L->evops.done(p.hc.ev)) waits.insert(p.hc.ev);
  for (void* w : waits) {
    hipError_t he = hipStreamWaitEvent(st, static_cast<hipEvent_t>(w), 0);
    if (he != hipSuccess) {
      rollback();
      return hip_fail(he, "hipStreamWaitEvent");
    }
  }
  for (const Planned& p : plan) {
    hipError_t he = hipMemcpyAsync(L->pool + p.dst.data_off, L->host_pool + p.hc.off,
                                   L->st.host_bytes(p.proj, p.hc), hipMemcpyHostToDevice, st);
    if (he != hipSuccess) {
      drain(st);
      rollback();
      return hip_fail(he, "host-to-device page copy");
    }
  }
  pw_status s = PW_OK;
  void* ev = record_event(L, st, &s);
  if (!ev) {
    drain(st);
    rollback();
    return s;
  }
  L->st.ref_event(ev);
  for (const Planned& p : plan) L->st.add_reload_pending(p.e, p.proj, p.rb, p.dst, ev);
  L->st.unref_event(ev);
  if (added_total) *added_total = added;
  return PW_OK;
}

pw_status pw_reload_block(pw_layer* L, int e, int proj, int rb, void* stream, size_t* added_bytes) {
  return pw_reload_blocks(L, 1, &e, &proj, &rb, stream, added_bytes);
}

pw_status pw_drop_host_copy(pw_layer* L, int e, int proj, int rb) {
  std::string err;
  if (!L) return fail(PW_EINVAL, "null layer");
  if (!L->st.check_block(e, proj, rb, &err)) return fail(PW_EINVAL, err);
  L->st.drop_host_copy(e, proj, rb);
  return PW_OK;
}

pw_status pw_host_copy_info(pw_layer* L, int e, int proj, int rb, int* bits, int* ready) {
  std::string err;
  if (!L) return fail(PW_EINVAL, "null layer");
  if (!L->st.check_block(e, proj, rb, &err)) return fail(PW_EINVAL, err);
  const pw::HostCopy& h = L->st.host[L->st.index(e, proj, rb)];
  if (bits) *bits = h.bits;
  if (ready) *ready = h.bits != 0 && (!h.ev || L->evops.done(h.ev)) ? 1 : 0;
  return PW_OK;
}

pw_status pw_host_pool_stats(const pw_layer* L, size_t* capacity, size_t* used) {
  if (!L) return fail(PW_EINVAL, "null layer");
  if (capacity) *capacity = L->st.halloc.capacity();
  if (used) *used = L->st.halloc.used();
  return PW_OK;
}

pw_status pw_planner_create_for_layer(const pw_layer* L, const double* sens, const pw_planner_config* cfg,
                                      pw_planner** out) {
  if (!L || !sens || !cfg || !out) return fail(PW_EINVAL, "bad argument");
  const size_t n = L->st.n_entries;
  std::vector<int> ex(n), ty(n);
  std::vector<uint64_t> nb(3 * n);
  for (int e = 0; e < L->st.desc.E; ++e)
    for (int p = 0; p < 3; ++p)
      for (int rb = 0; rb < L->st.nrb_max; ++rb) {
        const size_t i = L->st.index(e, p, rb);
        ex[i] = e;
        ty[i] = p == PW_DOWN ? 1 : 0;
        nb[3 * i] = L->st.page_bytes(p, 16);
        nb[3 * i + 1] = L->st.page_bytes(p, 8);
        nb[3 * i + 2] = L->st.page_bytes(p, 4);
      }
  return pw_planner_create(L->st.desc.E, static_cast<int>(n), ex.data(), ty.data(), nb.data(), sens, cfg, out);
}

namespace {

// Committed bitwidth per table entry; 0 for blocks past a projection's row
// blocks, absent pages and blocks with a pending requant or reload.
static std::vector<int> planner_bits(const pw_layer* L) {
  std::vector<int> q(L->st.n_entries, 0);
  for (int e = 0; e < L->st.desc.E; ++e)
    for (int p = 0; p < 3; ++p)
      for (int rb = 0; rb < L->st.nrb(p); ++rb) {
        const size_t i = L->st.index(e, p, rb);
        const pw_page_entry& ent = L->st.mirror[i];
        if (ent.state == PW_PAGE_RESIDENT) q[i] = ent.bits;
      }
  return q;
}

}  // namespace

pw_status pw_planner_step_layer(pw_planner* P, const pw_layer* L, int free_blocks, int free_threshold,
                                uint64_t kv_block_bytes, pw_plan_summary* out) {
  if (!P || !L) return fail(PW_EINVAL, "bad argument");
  if (pw::planner_units(P) != static_cast<int>(L->st.n_entries))
    return fail(PW_EINVAL, "planner was not made for this layer's table");
  const std::vector<int> q = planner_bits(L);
  return pw_planner_step(P, q.data(), free_blocks, free_threshold, kv_block_bytes, out);
}

pw_status pw_planner_apply(pw_planner* P, pw_layer* L, void* side_stream, size_t* delta_total) {
  if (!P || !L) return fail(PW_EINVAL, "bad argument");
  if (delta_total) *delta_total = 0;
  if (pw::planner_units(P) != static_cast<int>(L->st.n_entries))
    return fail(PW_EINVAL, "planner was not made for this layer's table");
  int n = 0;
  pw_status s = pw_planner_plan(P, -1, 0, 0, nullptr, nullptr, nullptr, nullptr, &n);
  if (s != PW_OK || n == 0) return s;
  std::vector<int> unit(n), from(n), to(n);
  s = pw_planner_plan(P, -1, 0, n, unit.data(), from.data(), to.data(), nullptr, &n);
  if (s != PW_OK) return s;
  const std::vector<int> q = planner_bits(L);
  std::vector<int> es, ps, rbs, nbits;
  for (int k = 0; k < n; ++k) {
    const int i = unit[k];
    if (q[i] != from[k]) return fail(PW_ESTATE, "the table changed since the planner step");
    const int rb = i % L->st.nrb_max, ep = i / L->st.nrb_max;
    es.push_back(ep / 3);
    ps.push_back(ep % 3);
    rbs.push_back(rb);
    nbits.push_back(to[k]);
  }
  return pw_requant_blocks(L, n, es.data(), ps.data(), rbs.data(), nbits.data(), side_stream, delta_total);
}

pw_status pw_commit(pw_layer* L, void* main_stream, int* n_committed) {
  if (!L) return fail(PW_EINVAL, "null layer");
  if (n_committed) *n_committed = 0;
  const auto& pend = L->st.pending();
  if (pend.empty()) return PW_OK;
  hipStream_t st = static_cast<hipStream_t>(main_stream);
  std::set<void*> evs;
  for (const auto& p : pend) evs.insert(p.ev);
  for (void* ev : evs) {
    hipError_t he = hipStreamWaitEvent(st, static_cast<hipEvent_t>(ev), 0);
    if (he != hipSuccess) return hip_fail(he, "hipStreamWaitEvent");
  }
  std::vector<std::pair<size_t, pw_page_entry>> w;
  for (const auto& p : pend) w.push_back({p.idx, pw::LayerState::published(p.next)});
  // On a failure after part of the table was rewritten, the device entries
  // are put back to the committed ones of the host mirror (which the failed
  // call leaves unchanged) before the error is returned.
  auto restore = [&]() {
    std::vector<std::pair<size_t, pw_page_entry>> old;
    for (const auto& p : pend) {
      pw_page_entry cur = L->st.mirror[p.idx];
      cur.state = PW_PAGE_RESIDENT;
      old.push_back({p.idx, cur});
    }
    const std::string keep = g_err;
    (void)write_entries(L, old, st);
    drain(st);
    g_err = keep;
  };
  pw_status s = write_entries(L, w, st);
  if (s != PW_OK) {
    restore();
    return s;
  }
  void* cev = L->evops.create();
  if (!cev) {
    restore();
    return fail(PW_EHIP, "hipEventCreate failed");
  }
  hipError_t he = hipEventRecord(static_cast<hipEvent_t>(cev), st);
  if (he != hipSuccess) {
    L->evops.destroy(cev);
    s = hip_fail(he, "hipEventRecord");
    restore();
    return s;
  }
  const int n = static_cast<int>(pend.size());
  L->st.committed(cev);
  if (n_committed) *n_committed = n;
  return PW_OK;
}

pw_status pw_reclaim(pw_layer* L, size_t* bytes_freed) {
  if (!L) return fail(PW_EINVAL, "null layer");
  const uint64_t f = L->st.reclaim();
  if (bytes_freed) *bytes_freed = f;
  return PW_OK;
}

pw_status pw_page_info(const pw_layer* L, int e, int proj, int rb, pw_page_entry* out) {
  std::string err;
  if (!L || !out) return fail(PW_EINVAL, "null argument");
  if (!L->st.check_block(e, proj, rb, &err)) return fail(PW_EINVAL, err);
  *out = L->st.mirror[L->st.index(e, proj, rb)];
  return PW_OK;
}

pw_status pw_pool_stats(const pw_layer* L, size_t* used, size_t* free_bytes, size_t* largest) {
  if (!L) return fail(PW_EINVAL, "null layer");
  if (used) *used = L->st.alloc.used();
  if (free_bytes) *free_bytes = L->st.alloc.free_bytes();
  if (largest) *largest = L->st.alloc.largest_free();
  return PW_OK;
}

pw_status pw_profile_enable(pw_layer* L, int on) {
  if (!L) return fail(PW_EINVAL, "null layer");
  L->prof = on != 0;
  return PW_OK;
}

pw_status pw_profile_read(pw_layer* L, double* total_ms, int64_t* count, int reset) {
  if (!L) return fail(PW_EINVAL, "null layer");
  for (auto& r : L->recs) {
    hipError_t he = hipEventSynchronize(r.b);
    float ms = 0.f;
    if (he == hipSuccess) he = hipEventElapsedTime(&ms, r.a, r.b);
    if (he != hipSuccess) return hip_fail(he, "profile event");
    L->tot_ms[r.phase] += ms;
    L->cnt[r.phase] += 1;
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  L->recs.clear();
  for (int i = 0; i < PW_NPHASE; ++i) {
    if (total_ms) total_ms[i] = L->tot_ms[i];
    if (count) count[i] = L->cnt[i];
    if (reset) {
      L->tot_ms[i] = 0;
      L->cnt[i] = 0;
    }
  }
  return PW_OK;
}

}  // extern "C"
