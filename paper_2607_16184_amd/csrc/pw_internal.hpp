// Kernel argument blocks and launchers shared by the C ABI (pw_api.cpp) and
// the HIP kernels (pw_kernels.hip). Internal to libpagedweight.so.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>
#include <string>

#include "pw.h"

namespace pw {

// One page quantized at load time from 16-bit values (or laid out as a
// 16-bit page) by the load-time kernel.
struct QJob {
  const uint8_t* src;      // source 16-bit values
  uint8_t* dst;            // destination values or code block
  uint8_t* dst_sz;         // destination scale/zero block
  uint32_t item_base;      // first work item of this job
  int K;                   // reduction length of the page's rows (H or F)
  uint8_t dst_bits;        // 16, 8 or 4
  uint8_t src_plain;       // 1: src is R x K row-major 16-bit values (not a pool page)
  uint8_t rsv[2];
};
constexpr int kMaxQJobs = 32;
// A job has (R / 16) tiles x (K / max(G, 128)) work items; job j's items
// start at job[j].item_base (increasing).
struct QJobBatch {
  QJob job[kMaxQJobs];
  int n_jobs;
  int R, G;                // rows, group size (same for the batch)
  int act, sdt;
  uint32_t total_items;
};

// Pages of one requant launch, all of one (source, destination) bitwidth
// pair. A page's slot and its scale/zero block (right after the codes) are
// at pool + 256 src[j] and pool + 256 dst[j]; bit j of kbit selects its K
// (kb[0] = H / 128 for gate/up pages, kb[1] = F / 128 for down pages). The
// whole batch travels as the kernel argument (under 4 KiB).
constexpr int kMaxRqJobs = 448;
struct RqBatch {
  uint8_t* pool;
  int n_jobs;
  int R, G;
  uint16_t kb[2];
  uint32_t kbit[kMaxRqJobs / 32];
  uint32_t src[kMaxRqJobs];
  uint32_t dst[kMaxRqJobs];
};
static_assert(sizeof(RqBatch) <= 4000, "requant batch must fit a 4 KiB kernel argument");

// Nested bit-plane quantization of whole blocks (one thread per row).
constexpr int kMaxAplJobs = 32;
// per-row float64 scratch: centroids of levels 4..8 (16 + 32 + 64 + 128 + 256),
// cluster counts (256 int32), sums (256), parent minima and maxima (128 each)
constexpr size_t kAplScratchRow = 496 * 8 + 256 * 4 + 256 * 8 + 128 * 8 * 2;
struct AplJob {
  const uint16_t* src;     // R x K 16-bit weights, row-major
  uint8_t* page;           // the page slot (planes and LUTs)
  uint8_t* codes;          // R x K bytes of workspace: 8-bit codes
  uint8_t* scratch;        // R x kAplScratchRow bytes of workspace
  uint32_t row_base;       // first global row of this job
  int K;
  int bits;                // 8 or 4
};
struct AplBatch {
  AplJob job[kMaxAplJobs];
  int n_jobs;
  int R;
  int act;
  uint32_t total_rows;
};

// Page-table writes performed by a kernel on the caller's stream.
constexpr int kMaxEntryWrites = 64;
struct EntryWrites {
  pw_page_entry ent[kMaxEntryWrites];
  uint32_t idx[kMaxEntryWrites];
  int n;
};

struct GemmArgs {
  const uint8_t* pool;
  const pw_page_entry* table;
  const uint16_t* x;          // [T,H] act
  const int32_t* offsets;     // [E+1]
  const int32_t* sorted_slot; // [S]
  const int32_t* slot_pos;    // [S]
  const float* topk_w;        // [T,K]
  uint16_t* h;                // [S,F] act, rows in sorted order
  float* opart;               // [nsplit][S][H] fp32 partial down outputs
  void* y;                    // [T,H] act or fp32
  int E, H, F, R, G, nrb_max;
  int topk, T, S;
  int nsplit, kb_per_split;   // down projection split over K = F (in 128-blocks)
  int out_fp32;
  int act, sdt;
  int mtb;                    // M tiles (of 16 slots) per pass: 1, 2 or 4
  int apl;                    // the layer holds nested bit-plane pages
  // experts [e0, e0 + ne) are the ones a GEMM launch covers, holding about
  // s_range of the S slots (routed and shared experts run as separate launches)
  int e0, ne, s_range;
  // combine: the last n_shared of the topk columns are shared-expert slots,
  // whose down projection ran with nsplit_sh K splits
  int n_shared, nsplit_sh;
};

// Routed top-K of E logits per token, then n_shared shared-expert columns
// (experts E .. E + n_shared - 1, weight shared_gate[t][j] or 1): rows of
// K + n_shared ids and weights.
hipError_t launch_route_topk(const float* logits, int T, int E, int K, int renorm, int n_shared,
                             const float* shared_gate, int32_t* ids, float* w, hipStream_t st);
// Both in one single-workgroup launch, for batches route_permute_fits admits.
bool route_permute_fits(int T, int E, int K, int n_shared);
hipError_t launch_route_permute(const float* logits, int T, int E, int K, int renorm, int n_shared,
                                const float* shared_gate, int32_t* ids, float* w, int32_t* offsets,
                                int32_t* sorted_slot, int32_t* slot_pos, hipStream_t st);
hipError_t launch_permute(const int32_t* ids, int T, int K, int E, int32_t* offsets,
                          int32_t* sorted_slot, int32_t* slot_pos, hipStream_t st);
hipError_t launch_qjobs(const QJobBatch& b, hipStream_t st);
// Requant of pool pages (16 -> 8, 16 -> 4 or 8 -> 4, every page of the batch
// the same pair); hipErrorInvalidValue for a batch the kernel cannot take.
hipError_t launch_requant(const RqBatch& b, int src_bits, int dst_bits, int act, int sdt, hipStream_t st);
hipError_t launch_entry_writes(pw_page_entry* table, const EntryWrites& w, hipStream_t st);
hipError_t launch_clear_table(pw_page_entry* table, size_t n, hipStream_t st);
hipError_t launch_gateup(const GemmArgs& a, hipStream_t st);
hipError_t launch_down(const GemmArgs& a, hipStream_t st);
hipError_t launch_combine(const GemmArgs& a, hipStream_t st);
// large per-expert slot counts: LDS-tiled GEMM (256 x 256 tiles)
hipError_t launch_tgemm(const GemmArgs& a, bool gateup, hipStream_t st);
// small and medium slot counts: register-streamed tiles of 16/32/64 slots
hipError_t launch_sgemm(const GemmArgs& a, bool gateup, hipStream_t st);
hipError_t launch_apl_quant(const AplBatch& b, hipStream_t st);
// ceiling probes: a plain streaming read and back-to-back bf16 MFMAs
hipError_t launch_probe_read(const void* buf, size_t bytes, int nblocks, uint32_t* out, hipStream_t st);
hipError_t launch_probe_mfma(int iters, int nblocks, float* out, hipStream_t st);
hipError_t launch_apl_pack(const AplBatch& b, hipStream_t st);
// Per-expert routing statistics (row norms, then a fixed-order reduction).
hipError_t launch_routing_stats(const uint16_t* rows, int act, int n_rows, int dim, int by_position,
                                const float* topk_w, const int32_t* offsets, const int32_t* sorted_slot, int S,
                                int E, int K, double* norm2, double* stats, int accumulate, hipStream_t st);

// Static device scratch of the allocation-free GEMM entry point: its
// capacity, and its device address on `device` (looked up once per GPU).
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
hipError_t static_scratch(int device, void** ptr);

// Error reporting of the C ABI (thread-local message, returned status).
pw_status set_error(pw_status s, const char* msg);
inline pw_status set_error(pw_status s, const std::string& msg) { return set_error(s, msg.c_str()); }
int planner_units(const pw_planner* p);

}  // namespace pw
