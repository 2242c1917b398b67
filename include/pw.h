/*
 * pw.h -- C ABI of libpagedweight.so: the paged mixed-bitwidth MoE expert
 * forward and runtime requantization of PagedWeight (arXiv 2607.16184),
 * written for AMD Instinct MI355X (gfx950).
 *
 * Model (Sec. 3.1): the routed experts' weights live as pages in one device
 * pool. A page is one row-block of one projection of one expert: R rows of
 * gate [F,H], up [F,H] or down [H,F] (row-major, a row is an output feature,
 * the reduction dimension K is contiguous). A page table holds one entry per
 * (expert, projection, row-block) with the page's committed bitwidth (16, 8
 * or 4; the paper's q_i) and its byte offsets in the pool. The kernels read
 * every block at its committed bitwidth (Sec. 3.3). Lowering a block's
 * bitwidth frees pool bytes Delta = M^b - M^b' (Eq. 3) that the caller can
 * hand to its KV cache; the lower bitwidth is committed before the old pages
 * are retired (Sec. 3.1 offload order; Sec. 3.3 safe boundaries).
 *
 * Page formats (the build's reading; the paper's own format is Any-Precision
 * bit-planes, which it pairs with per-bitwidth LUTs):
 *   8/4-bit pages are asymmetric group-wise round-to-nearest along K, group
 *   size G, one (scale, zero) pair of dtype sdt per (row, group); weight =
 *   z + c*s. 16-bit pages hold values of the activation dtype.
 *   Layout of every format: the page's R x K values are cut into tiles of 16
 *   rows x 128 values, stored tile after tile (row-tile major: tile (tau, b)
 *   at index tau*(K/128) + b). Inside a tile, value (r, k) with lc = r mod 16,
 *   i = (k mod 128) div 32, lg = (k mod 32) div 8, q = k mod 8 belongs to lane
 *   l = 16*lg + lc and step i:
 *     16-bit: 4096-byte tile, value at byte 1024*i + 16*l + 2*q;
 *     8-bit:  2048-byte tile, code at byte 1024*(i div 2) + 16*l + 8*(i mod 2) + q;
 *     4-bit:  1024-byte tile, code in the little-endian 32-bit word at byte
 *             16*l + 4*i, at bits [4t, 4t+4) for q = 2t and [16+4t, 20+4t)
 *             for q = 2t+1.
 *   Scale/zero block (8/4-bit, right after the codes): pair index g*R + r
 *   holds (scale, zero) of row r, group g, as two 16-bit values (scale in the
 *   low half of the 32-bit pair).
 *   Bytes: M16 = 2RK, M8 = RK + 4R(K/G), M4 = RK/2 + 4R(K/G).
 *   Quantizer: z = largest sdt value <= min(v); r = fl32(max(v) - z);
 *   r == 0 -> s = +0 and all codes 0; else s = smallest sdt value >= fl32(r/Q),
 *   one sdt step higher if fl32(s*Q) < r; c = clamp(rint(fl32(fl32(v-z)/s)),0,Q)
 *   with Q = 2^bits - 1; a zero result of a directed rounding is +0.
 *   A requantization 8 -> 4 starts from fl32(z + c*s).
 *
 * Memory ownership: the caller allocates every device buffer (pool, device
 * page table, workspaces, activations, outputs, routing arrays) and owns the
 * HIP streams. The library never allocates or frees device memory. It owns the
 * host mirror of the page table, the slot allocator inside the caller's pool
 * and the HIP events it creates.
 *
 * Errors: every call returns pw_status and never throws across the ABI. A
 * failing call leaves the table, pool and free lists unchanged; pw_last_error()
 * returns a message for the calling thread. Asynchronous HIP errors surface as
 * PW_EHIP on a later call. A layer handle is not thread-safe.
 *
 * Streams: `stream` arguments are hipStream_t handles passed as void*; NULL
 * is the null stream. Outputs are valid once the stream reaches the work.
 */
#ifndef PAGEDWEIGHT_PW_H
#define PAGEDWEIGHT_PW_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    PW_OK = 0,
    PW_EINVAL = 1,        /* bad argument, shape or size                      */
    PW_ENOMEM = 2,        /* pool or workspace too small                      */
    PW_EBUSY = 3,         /* a requantization or reload of the block pending  */
    PW_EUNSUPPORTED = 4,  /* e.g. raising a bitwidth (needs a reload)         */
    PW_EHIP = 5,          /* a HIP runtime call failed                        */
    PW_ESTATE = 6         /* layer not ready (a page is missing)              */
} pw_status;

typedef enum { PW_F16 = 0, PW_BF16 = 1 } pw_dtype;
typedef enum { PW_GATE = 0, PW_UP = 1, PW_DOWN = 2 } pw_proj;

/* Page states of the committed GPU page (Sec. 3.1 page state). A block may
 * also hold a copy in the caller's host pool (pw_offload_block); the table
 * entry always describes the GPU page the kernels read.                   */
enum { PW_PAGE_ABSENT = 0, PW_PAGE_RESIDENT = 1, PW_PAGE_REQUANT_PENDING = 2, PW_PAGE_RELOAD_PENDING = 3 };

/* Page formats (pw_page_entry.rsv): group-wise RTN codes with scale/zero
 * (16-bit pages are plain values), or nested bit-planes with per-row LUTs
 * (pw_layer_load_pages_apl).                                              */
enum { PW_FMT_RTN = 0, PW_FMT_APL = 1 };

/* One page-table entry (device array and host mirror). 24 bytes. */
typedef struct {
    uint64_t data_off;  /* byte offset of the page (values, code block or bit-planes) */
    uint64_t sz_off;    /* byte offset of the scale/zero block (RTN; 0 for 16-bit
                           pages) or of the 4-bit LUT (nested bit-planes)             */
    uint8_t bits;       /* committed bitwidth q_i: 16, 8, 4; 0 = absent               */
    uint8_t state;      /* PW_PAGE_*                                                  */
    uint16_t rsv;       /* page format, PW_FMT_*                                      */
    uint32_t gen;       /* bumped at every commit                                     */
} pw_page_entry;

/* Layer shape. act is the activation dtype (and the dtype of 16-bit pages);
 * sdt the dtype of scales and zeros. Constraints: R a multiple of 64;
 * F and H multiples of R and of 128; G one of 64, 128, 256, 512 dividing F
 * and H (PW_EINVAL otherwise).                                             */
typedef struct {
    int E, H, F, R, G;
    int act;
    int sdt;
} pw_layer_desc;

typedef struct pw_layer pw_layer;

/* Number of entries of the device page table: E * 3 * max(F, H) / R.
 * Entry (e, proj, rb) is at index (e*3 + proj) * (max(F,H)/R) + rb.        */
size_t pw_table_entries(const pw_layer_desc* desc);

/* Bytes of one page of projection `proj` at `bits` (Eq. 3's M_i^b). */
pw_status pw_page_bytes(const pw_layer_desc* desc, int proj, int bits, size_t* bytes);

/* Sec. 3.1 (weight page table: one row per block with its committed
 * bitwidth and memory size). Create a layer over a caller-owned pool
 * [pool_dev, pool_dev + pool_bytes) (256-byte aligned, at most 2^40 bytes)
 * and device table table_dev (pw_table_entries entries, 8-byte aligned). The
 * table is cleared to absent entries on the null stream, which is
 * synchronized. The layer also creates, on the pool's device, a stream of
 * its own (default priority) and two events, for the GEMM's concurrent
 * chains (pw_layer_set_chains) and shared experts.
 *   bad shape (see pw_layer_desc), null or misaligned pointers, a pool
 *   above 2^40 bytes: PW_EINVAL.
 *   clearing the table or creating the stream failed: PW_EHIP (no handle
 *   is returned).                                                          */
pw_status pw_layer_create(const pw_layer_desc* desc, void* pool_dev, size_t pool_bytes,
                          pw_page_entry* table_dev, pw_layer** out);

/* Destroy the handle (waits for the library's events). */
pw_status pw_layer_destroy(pw_layer* layer);

/* Sec. 3.1 (a block's page at its bitwidth q_i, placed in the pool and
 * described by its table row). Place page (e, proj, rb) into a fresh pool
 * slot at `bits`: rows16_dev holds the page's R x K 16-bit values (act dtype,
 * row-major, device memory, read on `stream`). 16 -> copied; 8/4 ->
 * quantized on the GPU. The table entry is written on `stream` after the
 * data; later work on another stream must be ordered after `stream`.
 *   bad block or bits: PW_EINVAL.  page present: PW_EBUSY.
 *   no free slot: PW_ENOMEM.  launch failed: PW_EHIP (the slot is released
 *   after `stream` drained).                                               */
pw_status pw_layer_load_page(pw_layer* layer, int e, int proj, int rb, int bits,
                             const void* rows16_dev, void* stream);

/* Router (Sec. 2.1 top-K routing) and token permutation (Sec. 3.3 dispatch).
 *   logits   [T,E] fp32 device, row-major
 *   topk_ids [T,K] int32 out: per token the K largest logits, ties to the
 *            lower expert index, in decreasing order
 *   topk_w   [T,K] fp32 out: renorm=1 softmax over the selected K logits;
 *            renorm=0 the full softmax probability of each selected expert
 *   offsets  [E+1] int32 out: exclusive scan of per-expert slot counts
 *   sorted_slot [T*K] int32 out: slots s = t*K + k grouped by expert, in
 *            increasing s within an expert
 *   slot_pos [T*K] int32 out: inverse permutation of sorted_slot
 * Constraints: 1 <= K <= E <= 256, K <= 16, T*K < 2^31 (PW_EINVAL
 * otherwise). T = 0 writes offsets only.                                    */
pw_status pw_route_topk(const float* logits, int T, int E, int K, int renorm,
                        int32_t* topk_ids, float* topk_w, int32_t* offsets,
                        int32_t* sorted_slot, int32_t* slot_pos, void* stream);

/* Shared experts (Table 1 lists MoE layers with experts every token uses
 * beside the routed ones: 60 routed + 4 shared, 128 routed + 1 shared; the
 * paper does not give their combination, read here as the routed sum plus
 * each shared expert's output times a per-token gate, 1 unless the caller
 * supplies one). A layer of E experts declares its last n_shared experts as
 * shared (0 <= n_shared < E; 0 by default; PW_EINVAL otherwise); its pages
 * are paged, quantized, requantized and committed like any other expert's.
 * Routing for such a layer comes from pw_route_topk_shared, and
 * pw_moe_paged_gemm is then called with K = routed top-K + n_shared: each
 * token's last n_shared columns must be the shared experts (in order), its
 * first columns routed experts only. The GEMM runs the routed and the shared
 * experts as separate launches, each with the kernels suited to its slots
 * per expert (a shared expert has T); the shared experts' launches go to a
 * stream of the layer's own, forked from the caller's stream and joined back
 * before the combine, so that they run beside the routed ones (under graph
 * capture: two branches; with pw_layer_set_chains(layer, 1), on the
 * caller's stream after them). That stream (default priority) and its two
 * events live on the pool's device (created with the layer by
 * pw_layer_create; pw_layer_destroy releases them). No GPU work; takes
 * effect for the next GEMM call.                                           */
pw_status pw_layer_set_shared_experts(pw_layer* layer, int n_shared);

/* Concurrent expert chains (Sec. 3.3 runs the MoE forward as one fused
 * kernel; here its gate/up and down phases are separate launches, and this
 * setting overlaps the boundary between them). With
 * chains = 2 (the default), when a call's experts run on the decode kernels
 * and the layer has no shared experts, they are split into two halves, each
 * a chain of gate/up then down: the first on the caller's stream, the
 * second on the layer's own stream (forked from the caller's and joined
 * back before the combine; under graph capture, two branches), so that the
 * phase boundary of one chain overlaps the other's GEMMs; a layer with
 * shared experts runs those on the layer's stream instead (see
 * pw_layer_set_shared_experts). chains = 1 launches everything on the
 * caller's stream, one launch after another (each kernel alone on the GPU,
 * as a per-kernel timing needs). Results are identical either way (each
 * expert's rows are computed by the same kernels). PW_EINVAL unless chains
 * is 1 or 2. No GPU work; takes effect for the next GEMM call.            */
pw_status pw_layer_set_chains(pw_layer* layer, int chains);

/* Router with shared experts: the top-K of pw_route_topk over the E routed
 * experts' logits ([T,E] fp32), and for every token n_shared more columns,
 * expert E + j with weight shared_gate[t * n_shared + j] (fp32 device
 * [T, n_shared]; NULL: weight 1). topk_ids and topk_w are [T, K + n_shared];
 * the permutation covers E + n_shared experts (offsets [E + n_shared + 1],
 * sorted_slot and slot_pos [T (K + n_shared)]).
 * Constraints: 1 <= K <= E, K <= 16, n_shared >= 0, E + n_shared <= 256,
 * T (K + n_shared) < 2^31 (PW_EINVAL otherwise).                           */
pw_status pw_route_topk_shared(const float* logits, int T, int E, int K, int renorm, int n_shared,
                               const float* shared_gate, int32_t* topk_ids, float* topk_w,
                               int32_t* offsets, int32_t* sorted_slot, int32_t* slot_pos, void* stream);

/* Workspace bytes pw_moe_paged_gemm needs for T tokens with top-K. */
pw_status pw_workspace_bytes(const pw_layer* layer, int T, int K, size_t* gemm_ws);

/* Paged expert forward and combine (Sec. 3.3): for each routed slot (t,k)
 * with expert e, o = W_down[e] (silu(W_gate[e] x_t) * W_up[e] x_t), each
 * block read at its committed bitwidth; y[t] = sum_k topk_w[t,k] * o, k
 * ascending, fp32 accumulation. The SwiGLU output is rounded to `act`
 * before the down projection.
 *   x [T,H] act device; y [T,H] act, or fp32 if out_fp32 != 0.
 *   topk_w, offsets, sorted_slot, slot_pos: as produced by pw_route_topk.
 *   ws: device workspace of at least pw_workspace_bytes bytes.
 * Requires every page of the layer to be present (PW_ESTATE otherwise).
 * Sizes: T*K < 2^31, and T*K*max(F, H)*2 < 2^32 (32-bit row offsets in the
 * kernels; PW_EUNSUPPORTED otherwise: split the batch).
 * Streams: the work is ordered after what `stream` already holds and y is
 * complete when `stream` passes the call; part of it may run on the layer's
 * own stream in between (pw_layer_set_chains), forked from and joined back
 * into `stream`, so the caller orders nothing else. The workspace is in use
 * until `stream` passes the call.
 * Deterministic: no floating-point atomics; a fixed summation order.      */
pw_status pw_moe_paged_gemm(const pw_layer* layer, const void* x, int T, int K,
                            const float* topk_w, const int32_t* offsets,
                            const int32_t* sorted_slot, const int32_t* slot_pos,
                            void* y, int out_fp32, void* ws, size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops or harnesses that forbid hipMalloc): the forward of
 * pw_moe_paged_gemm with its workspace taken from a static device array of
 * the library instead of `ws`, so the call allocates nothing. Arguments,
 * kernels and results are those of pw_moe_paged_gemm. The array holds
 * 64 MiB on each GPU the library runs on, from that GPU's first call until
 * the process ends; the GPU is the one `stream` belongs to. Every call on a
 * GPU shares its array and overwrites what the last call left there (no part
 * of it needs to start zeroed): calls that overlap on one GPU (two streams,
 * two threads) race, and the caller serializes them.
 *   workspace need (pw_workspace_bytes) above 64 MiB, e.g. prefill batches
 *   of large layers: PW_ENOMEM (use pw_moe_paged_gemm).  Other errors: as
 *   pw_moe_paged_gemm.                                                     */
pw_status pw_moe_paged_gemm_noalloc(const pw_layer* layer, const void* x, int T, int K,
                                    const float* topk_w, const int32_t* offsets,
                                    const int32_t* sorted_slot, const int32_t* slot_pos,
                                    void* y, int out_fp32, void* stream);

/* Runtime downshift of one block (Sec. 3.1 offload; Sec. 3.3 asynchronous
 * page movement): requantize page (e, proj, rb) from its committed bitwidth
 * b to new_bits < b into a fresh slot on `side_stream`. The committed entry
 * is unchanged until pw_commit. *delta_bytes receives Eq. 3's M^b - M^b'.
 *   new_bits == b: PW_OK, delta 0, no work.
 *   new_bits > b: PW_EUNSUPPORTED (raising is a reload from a host copy,
 *   pw_reload_block).  pending already: PW_EBUSY.
 *   no free slot: PW_ENOMEM.                                              */
pw_status pw_requant_block(pw_layer* layer, int e, int proj, int rb, int new_bits,
                           void* side_stream, size_t* delta_bytes);

/* Batched form of pw_requant_block over n blocks (one kernel launch per 448
 * blocks of one (old, new) bitwidth pair, pages of every projection
 * together). On error no block of the batch is left pending.
 * Ordering: the kernels read the source pages on side_stream; the caller
 * orders side_stream after the stream that loaded or last wrote them (the
 * library itself waits only for host-copy transfers of those pages).     */
pw_status pw_requant_blocks(pw_layer* layer, int n, const int* e, const int* proj,
                            const int* rb, const int* new_bits, void* side_stream,
                            size_t* delta_bytes_total);

/* Host copies of pages (Sec. 3.1: a page's higher-precision version moves to
 * CPU memory before its GPU copy is lowered, and comes back when the
 * bitwidth is raised again; pages are CPU-resident, GPU-resident or in
 * transfer).
 *
 * pw_layer_set_host_pool: hand the layer a host pool [host_pool, + host_bytes)
 * (256-byte aligned; page-locked memory, e.g. hipHostMalloc, for the copies
 * to run asynchronously). The caller owns it and keeps it alive until
 * pw_layer_destroy. Once per layer (PW_EBUSY after).                       */
pw_status pw_layer_set_host_pool(pw_layer* layer, void* host_pool, size_t host_bytes);

/* Copy the committed page of each block (codes and scale/zero, Eq. 3's M^b
 * bytes; for a nested bit-plane page its planes and LUTs of the committed
 * precision) into a fresh host slot, device-to-host on `stream`. The GPU page
 * and the table are unchanged. A host copy at another bitwidth is replaced;
 * one at the committed bitwidth makes the block a no-op. To lower a block in
 * the paper's order, offload it and then requantize it on the same stream
 * (a bit-plane page: drop its planes 8 -> 4).
 *   no host pool, page absent: PW_ESTATE.  requant/reload pending: PW_EBUSY.
 *   host pool full: PW_ENOMEM (no block of the batch is copied).           */
pw_status pw_offload_blocks(pw_layer* layer, int n, const int* e, const int* proj, const int* rb,
                            void* stream);
pw_status pw_offload_block(pw_layer* layer, int e, int proj, int rb, void* stream);

/* Raise each block back to the bitwidth of its host copy: a fresh device
 * slot is filled host-to-device on `stream` (after the offload's copy
 * finished); the block is pending (PW_PAGE_RELOAD_PENDING) until pw_commit
 * publishes the raised entry, and its old slot is then retired like a
 * requantized one. A bit-plane page comes back whole (planes 0-7 and both
 * LUTs from its 8-bit copy) as a bit-plane entry. *added_bytes_total (may be
 * NULL) receives the sum of M^b' - M^b. The host copy stays (drop it with
 * pw_drop_host_copy).
 *   no host copy, page absent: PW_ESTATE.  copy not of a higher bitwidth, or
 *   of another format than the committed page: PW_EUNSUPPORTED.  pending
 *   already: PW_EBUSY.  no free slot: PW_ENOMEM.                           */
pw_status pw_reload_blocks(pw_layer* layer, int n, const int* e, const int* proj, const int* rb,
                           void* stream, size_t* added_bytes_total);
pw_status pw_reload_block(pw_layer* layer, int e, int proj, int rb, void* stream, size_t* added_bytes);

/* Forget a block's host copy; its host slot is freed by pw_reclaim once the
 * last transfer that uses it completed. No copy: PW_OK.                    */
pw_status pw_drop_host_copy(pw_layer* layer, int e, int proj, int rb);

/* Bitwidth of a block's host copy (0: none) and whether its device-to-host
 * copy completed (*ready = 1).                                             */
pw_status pw_host_copy_info(pw_layer* layer, int e, int proj, int rb, int* bits, int* ready);

/* Host pool capacity and bytes in host slots. */
pw_status pw_host_pool_stats(const pw_layer* layer, size_t* capacity, size_t* used);

/* Sec. 3.3 (page movement becomes visible only at a safe boundary between
 * kernel steps) and Sec. 3.1 (offload order: the lower bitwidth is committed
 * before the old pages are freed). Publish every pending requantization and
 * reload, ordered on main_stream after its transfer finished: the device
 * entries are rewritten by a kernel on main_stream, the host mirror updated,
 * and the old slots retired until main_stream passes the commit. A GEMM
 * enqueued on main_stream before the commit reads the old entries, one after
 * it the new ones. *n_committed may be NULL.
 *   a launch or event failed: PW_EHIP; the device entries are put back to
 *   the committed ones and the blocks stay pending.                        */
pw_status pw_commit(pw_layer* layer, void* main_stream, int* n_committed);

/* Sec. 3.1 (freed weight pages go back to the memory the KV cache draws
 * from; Eq. 3's Delta = M^b - M^b' per lowered block). Return retired slots
 * whose commit has completed to the pool's free list (and dropped host slots
 * whose last transfer completed to the host pool). Never blocks.
 * *bytes_freed (may be NULL) receives the device bytes returned (whole
 * 256-byte granules; every page size of a valid layer is such a multiple). */
pw_status pw_reclaim(pw_layer* layer, size_t* bytes_freed);

/* Host-mirror view of one entry. */
pw_status pw_page_info(const pw_layer* layer, int e, int proj, int rb, pw_page_entry* out);

/* Pool occupancy: bytes in slots, free bytes, largest free range. */
pw_status pw_pool_stats(const pw_layer* layer, size_t* used, size_t* free_bytes,
                        size_t* largest_free);

/* Per-kernel timing with HIP events recorded on the kernels' own streams.
 * Phases: 0 gate/up GEMM, 1 down GEMM, 2 combine, 3 requant (one record per
 * launch), 4 the GEMM phases of a pw_moe_paged_gemm call as a whole (one
 * record per call, on the caller's stream, from before its first GEMM launch
 * to after the last one, every chain joined: with concurrent chains the
 * per-launch records of phases 0 and 1 overlap, this one does not).
 * pw_profile_read waits for the recorded events and returns the summed
 * milliseconds and counts per phase; reset != 0 clears them.              */
enum { PW_PH_GATEUP = 0, PW_PH_DOWN = 1, PW_PH_COMBINE = 2, PW_PH_REQUANT = 3, PW_PH_GEMM = 4, PW_NPHASE = 5 };
pw_status pw_profile_enable(pw_layer* layer, int on);
pw_status pw_profile_read(pw_layer* layer, double* total_ms, int64_t* count, int reset);

/* ------------------------------------------------------------------------
 * Nested bit-plane pages (any-precision weights, Sec. 2.2 and 3.1: a block's
 * b-bit code is the top b bits of its 8-bit code; bit-planes and one LUT per
 * row and precision; lowering drops bit-planes).
 * ---------------------------------------------------------------------- */

/* Quantize n blocks into nested bit-plane pages at 8 or 4 bits. rows16[i]
 * (a host array of device pointers) holds block i's R x K 16-bit weights
 * (act dtype, row-major). Per row, in float64 with sums in order of k: a
 * 4-bit seed of 16 centroids at lo + (hi - lo)(2j+1)/32 refined by 8 Lloyd
 * iterations (nearest centroid, ties to the lower index; empty clusters keep
 * their centroid), then four one-bit splits to 8 bits (each cluster's two
 * children start at (lo + mean)/2 and (mean + hi)/2 of its members and take
 * 4 Lloyd iterations among them); LUT_b = the level-b centroids rounded to
 * act (nearest even). Page layout of an R x K block at 8 bits (4 bits: the
 * first two parts): planes 0-3 (plane 0 = most significant code bit,
 * RK/8 bytes each) | LUT_4 (R x 16 act values) | planes 4-7 | LUT_8
 * (R x 256). Inside a plane, 16-row x 128-column tile t = rt (K/128) + kb
 * takes 256 bytes at 256 t: lane l's 32-bit word at 4 l holds, at bit
 * 8 i + q, the plane's bit of row 16 rt + l mod 16, column
 * 128 kb + 32 i + 8 (l div 16) + q. The entry's sz_off points at LUT_4;
 * rsv = PW_FMT_APL. Eq. 3: M^8 = RK + 32 R + 512 R, M^4 = RK/2 + 32 R.
 * ws: device workspace of pw_apl_workspace_bytes(n) bytes. Work is
 * enqueued on `stream`; the table entries are written there too.
 *   bits not 8 or 4, R not a multiple of 16: PW_EINVAL.  present: PW_EBUSY.
 *   pool full: PW_ENOMEM (no page of the batch is placed).
 * A layer holding such pages runs the streaming GEMM kernel for every batch
 * size; pw_requant_block takes them from 8 to 4 bits without a kernel (the
 * tail of the slot, planes 4-7 and LUT_8, is freed by pw_reclaim after the
 * commit); host copies of them are not supported (PW_EUNSUPPORTED).      */
pw_status pw_apl_workspace_bytes(const pw_layer* layer, int n, size_t* bytes);
pw_status pw_layer_load_pages_apl(pw_layer* layer, int n, const int* e, const int* proj, const int* rb,
                                  const int* bits, const void* const* rows16, void* ws, size_t ws_bytes,
                                  void* stream);

/* ------------------------------------------------------------------------
 * Routing statistics and the runtime planner (Sec. 3.2, Alg. 1).
 * ---------------------------------------------------------------------- */

/* Per-expert routing statistics of one step, for Eq. 1's routing mass and
 * the routed-input features of the prompt residual (Sec. 3.2). For each
 * expert e and each slot routed to it (sorted_slot[offsets[e] ..
 * offsets[e+1]), in that order), with r the slot's routing weight and |x|
 * the Euclidean norm of the slot's input row:
 *   stats[5 e + 0] = sum r        stats[5 e + 1] = number of slots
 *   stats[5 e + 2] = sum r |x|    stats[5 e + 3] = sum r |x|^2
 *   stats[5 e + 4] = max |x|
 * in float64 with a fixed summation order (bit-identical across runs).
 * rows: [n_rows][dim] 16-bit values of dtype act (16-byte aligned, dim a
 * multiple of 8). rows_by_position = 0: the row of slot s = t K + k is
 * token t (the gate/up input x, n_rows = T); 1: the row of the i-th slot
 * of the expert-major list is row i (the down input h, n_rows = T K).
 * norm2_ws: device workspace of n_rows doubles. accumulate != 0 adds to
 * stats (online statistics over steps) instead of overwriting it. All
 * pointers are device memory; work is enqueued on `stream`.
 *   bad sizes or pointers: PW_EINVAL.                                     */
pw_status pw_routing_stats(const void* rows, pw_dtype act, int n_rows, int dim, int rows_by_position,
                           const float* topk_w, const int32_t* offsets, const int32_t* sorted_slot,
                           int T, int E, int K, double* norm2_ws, double* stats, int accumulate,
                           void* stream);

/* The planner (host code; no GPU work). Units are the page-table blocks it
 * may lower; unit i belongs to expert unit_expert[i] and has linear-block
 * type unit_type[i] (0: gate_up, for the gate and up projections; 1: down).
 * unit_bytes[3 i + j] is Eq. 3's M^b of the unit for b = 16, 8, 4 (j = 0,
 * 1, 2) and unit_sens[3 i + j] the offline sensitivity s^b (Eq. 2).
 * Bitwidths step down one level at a time (16 -> 8 -> 4).
 *
 * Configuration (offline calibration results, Sec. 3.2 and 4.1):
 *   routing buckets: experts sorted by routing mass (descending, ties to the
 *     lower index); bucket j takes positions floor(E c_{j-1} + 1/2) ..
 *     floor(E c_j + 1/2), c_j the running sum of bucket_frac (the last
 *     bucket takes the rest); mult[j] is its damage multiplier;
 *   bitwidth-floor stages: floor_bits[s][j] is the lowest bitwidth bucket j
 *     may reach at stage s (stages relax the floors: the depth caps);
 *   prompt residual heads [u][t] (t = 0: 16 -> 8, t = 1: 8 -> 4): Eq. 5's
 *     w and a, Eq. 6's confidence c, strength alpha, clip [rho_min,
 *     rho_max]; Eq. 8's damage floor eps.                                  */
#define PW_PLAN_MAX_BUCKETS 8
#define PW_PLAN_MAX_STAGES 8
typedef struct {
    int n_buckets;
    double bucket_frac[PW_PLAN_MAX_BUCKETS];
    double mult[PW_PLAN_MAX_BUCKETS];
    int n_stages;
    int floor_bits[PW_PLAN_MAX_STAGES][PW_PLAN_MAX_BUCKETS];
    double alpha, rho_min, rho_max, eps;
    double head_w[2][2][3];
    double head_a[2][2];
    double head_c[2][2];
} pw_planner_config;

typedef struct pw_planner pw_planner;

/* Result of one planner step. */
typedef struct {
    uint64_t target;     /* Eq. 7's D                                          */
    uint64_t bytes;      /* bytes the selected plan releases (sum of Eq. 3)    */
    double damage;       /* sum of Eq. 8 over its steps                        */
    int triggered;       /* D > 0: a plan was selected                         */
    int stage;           /* stage of the selected plan (-1: none)              */
    int n_steps;         /* one-level steps in it                              */
    int n_units;         /* units it lowers                                    */
} pw_plan_summary;

/* Copies the unit tables; the planner keeps one candidate plan per stage (the
 * plan queue) between steps.
 *   bad sizes, types, bitwidth floors or fractions: PW_EINVAL.             */
pw_status pw_planner_create(int n_experts, int n_units, const int* unit_expert, const int* unit_type,
                            const uint64_t* unit_bytes, const double* unit_sens,
                            const pw_planner_config* cfg, pw_planner** out);
void pw_planner_destroy(pw_planner* p);

/* The batch-level observation (Sec. 3.2, batched serving): each request adds
 * its routing statistics (host copies of pw_routing_stats for the gate/up
 * input and, or NULL for zero features, the down input) with its KV-block
 * weight; masses and features are averaged with those weights.
 * pw_planner_clear_requests forgets them.                                 */
pw_status pw_planner_add_request(pw_planner* p, const double* stats_gate_up, const double* stats_down,
                                 double kv_weight);
pw_status pw_planner_clear_requests(pw_planner* p);

/* One step of Alg. 1: D from the KV pressure (Eq. 7), a greedy plan per
 * stage (steps by Eq. 8's damage per released byte, cheapest first, until
 * D is met), the queue refreshed; when D > 0 the selected plan is the
 * strictest stage's that meets D, else the one releasing the most bytes.
 * unit_bits[i] is the unit's committed bitwidth (16, 8 or 4; 0: skip).  */
pw_status pw_planner_step(pw_planner* p, const int* unit_bits, int free_blocks, int free_threshold,
                          uint64_t kv_block_bytes, pw_plan_summary* out);

/* The plan of stage `stage` (-1: the selected one) as one entry per unit,
 * in the order the units were first taken: unit, committed bitwidth,
 * final bitwidth, bytes released (M^from - M^to). *n receives the count;
 * at most max_n entries are written. With steps != 0 the one-level steps
 * are listed instead (from and to one level apart, in the order taken).  */
pw_status pw_planner_plan(const pw_planner* p, int stage, int steps, int max_n, int* unit, int* from_bits,
                          int* to_bits, uint64_t* bytes, int* n);

/* Layer helpers: units = every table entry (expert, proj, row block) in
 * table order (index (e * 3 + proj) * nrb_max + rb; entries past a
 * projection's row blocks are units with bits 0). sens: [entries][3].
 * pw_planner_step_layer takes the committed bitwidths from the layer's
 * host mirror (blocks with a pending requant or reload are skipped);
 * pw_planner_apply requantizes every unit of the selected plan to its
 * final bitwidth on side_stream (pw_requant_blocks), *delta_total
 * receiving the bytes released once committed.                          */
pw_status pw_planner_create_for_layer(const pw_layer* layer, const double* sens, const pw_planner_config* cfg,
                                      pw_planner** out);
pw_status pw_planner_step_layer(pw_planner* p, const pw_layer* layer, int free_blocks, int free_threshold,
                                uint64_t kv_block_bytes, pw_plan_summary* out);
pw_status pw_planner_apply(pw_planner* p, pw_layer* layer, void* side_stream, size_t* delta_total);

/* ---- Ceiling probes (diagnostics beside the hot path) ---------------------
 * What the device delivers, for reading the kernels' roofline fractions
 * against the achievable as well as the published peaks.
 *
 * pw_probe_read: nblocks workgroups of 256 threads each stream one
 * contiguous span of bytes / nblocks bytes of buf (device memory, caller-
 * owned, at least `bytes` long, 16-byte aligned) with 16-byte nontemporal
 * loads. bytes must be a positive multiple of nblocks * 32768. out: device,
 * 2 * nblocks uint32 (a completion flag per workgroup in out[nblocks..]).
 * Bytes read per launch = bytes. Time it with events on `stream`.
 *
 * pw_probe_mfma: nblocks workgroups of 8 waves (one per CU, by a 96 KiB
 * LDS request) issue independent v_mfma_f32_32x32x16_bf16 back to back:
 * each wave runs iters rounds of 4. out: device, nblocks floats. Flops per
 * launch = nblocks * 8 * iters * 4 * 32768.
 *
 * Errors: PW_EINVAL for the argument conditions above; PW_EHIP if the
 * launch fails.                                                           */
pw_status pw_probe_read(const void* buf, size_t bytes, int nblocks, uint32_t* out, void* stream);
pw_status pw_probe_mfma(int iters, int nblocks, float* out, void* stream);

const char* pw_last_error(void);
const char* pw_status_str(pw_status s);

#ifdef __cplusplus
}
#endif
#endif /* PAGEDWEIGHT_PW_H */
