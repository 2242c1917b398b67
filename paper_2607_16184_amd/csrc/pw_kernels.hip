// HIP kernels for gfx950 (CDNA4): router, token permutation, group-wise RTN
// quantize / requantize, page-table writes and the combine. The paged GEMMs
// are in pw_decode.hip (decode-size batches) and pw_tgemm.hip (streaming and
// LDS-tiled GEMMs for larger batches); all three read the tiled page format
// described in pw.h.
#include <algorithm>

#include "pw_device.hpp"
#include "pw_internal.hpp"

namespace pw {
namespace {

// ---------------------------------------------------------------------------
// Router: top-K per token (ties to the lower index) and routing weights
// ---------------------------------------------------------------------------

constexpr int kMaxTopK = 16;
constexpr int kRouteLogitsPerLane = 4;            // E <= 256

// Selection key of logit v of expert e: larger key = earlier in (value
// descending, expert ascending) order. The float's bits are mapped to an
// order-preserving unsigned value (-0 taken as +0, so the two tie like equal
// values), the expert index complemented below them; 0 is below every key.
__device__ __forceinline__ uint64_t route_key(float v, int e) {
  uint32_t u = __float_as_uint(v);
  if (u == 0x80000000u) u = 0u;
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (static_cast<uint64_t>(u) << 32) | (0xFFFFFFFFu - static_cast<uint32_t>(e));
}

template <int CTRL>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t x) {
  const uint32_t lo = static_cast<uint32_t>(
      __builtin_amdgcn_update_dpp(0, static_cast<int>(static_cast<uint32_t>(x)), CTRL, 0xF, 0xF, false));
  const uint32_t hi = static_cast<uint32_t>(
      __builtin_amdgcn_update_dpp(0, static_cast<int>(static_cast<uint32_t>(x >> 32)), CTRL, 0xF, 0xF, false));
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ __forceinline__ uint64_t max_u64(uint64_t a, uint64_t b) { return a > b ? a : b; }

// Largest key of the wave, the same in every lane: within each row of 16
// lanes by DPP exchanges (pairs, quads, half-row and row mirrors), then over
// the four rows' results read out as wave-uniform values.
__device__ __forceinline__ uint64_t wave_max_key(uint64_t k) {
  k = max_u64(k, dpp_u64<0xB1>(k));    // quad_perm 1,0,3,2
  k = max_u64(k, dpp_u64<0x4E>(k));    // quad_perm 2,3,0,1
  k = max_u64(k, dpp_u64<0x141>(k));   // row_half_mirror
  k = max_u64(k, dpp_u64<0x140>(k));   // row_mirror
  uint64_t best = 0;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(k), 16 * r);
    const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(k >> 32), 16 * r);
    best = max_u64(best, (static_cast<uint64_t>(hi) << 32) | lo);
  }
  return best;
}

// One wave per token: lane l holds logits l, l + 64, ...; K rounds of a
// wave-wide arg-max in (value descending, index ascending) order take the
// next expert each. The weights use the same fp32 arithmetic as a serial
// loop: m = the largest selected logit, a_k = exp(l_k - m), w_k = a_k / sum,
// with the sum taken in k order (renorm) or in expert order over all E (each
// lane computes the exponentials of its own logits, and the terms are added
// one lane after another: the serial loop's operations in its order).
// Rows of ids and w hold K + n_shared columns: the routed experts, then the
// shared experts E + j with weight gate[t n_shared + j] (1 without a gate).
// lds_ids (may be null): the token's row of ids also goes there.
__device__ __forceinline__ void route_token(const float* __restrict__ logits, int t, int E, int K, int renorm,
                                            int n_shared, const float* __restrict__ gate,
                                            int32_t* __restrict__ ids, float* __restrict__ w, int* lds_ids) {
  const int lane = lane_id();
  const float* l = logits + static_cast<size_t>(t) * E;
  uint64_t key[kRouteLogitsPerLane];
  float lv[kRouteLogitsPerLane];
#pragma unroll
  for (int q = 0; q < kRouteLogitsPerLane; ++q) {
    const int e = lane + 64 * q;
    lv[q] = e < E ? l[e] : 0.0f;
    key[q] = e < E ? route_key(lv[q], e) : 0ull;
  }
  float sv[kMaxTopK];
  int se[kMaxTopK];
#pragma unroll
  for (int k = 0; k < kMaxTopK; ++k) {
    if (k < K) {
      uint64_t mine = key[0];
#pragma unroll
      for (int q = 1; q < kRouteLogitsPerLane; ++q) mine = max_u64(mine, key[q]);
      const uint64_t best = wave_max_key(mine);
      const int be = static_cast<int>(0xFFFFFFFFu - static_cast<uint32_t>(best));
      const uint32_t u = static_cast<uint32_t>(best >> 32);
      se[k] = be;
      sv[k] = __uint_as_float((u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u);   // the logit (-0 read as +0)
#pragma unroll
      for (int q = 0; q < kRouteLogitsPerLane; ++q)
        if (lane + 64 * q == be) key[q] = 0ull;
    }
  }
  const float m = sv[0];
  float sum = 0.0f;
  if (renorm) {
    if (lane != 0) return;
    for (int k = 0; k < K; ++k) sum += expf(sv[k] - m);
  } else {
    // terms past E are +0 and leave the (positive) sum unchanged
#pragma unroll
    for (int q = 0; q < kRouteLogitsPerLane; ++q) {
      if (64 * q < E) {
        const int ex = __float_as_int(lane + 64 * q < E ? expf(lv[q] - m) : 0.0f);
#pragma unroll
        for (int j = 0; j < 64; ++j) sum += __int_as_float(__builtin_amdgcn_readlane(ex, j));
      }
    }
    if (lane != 0) return;
  }
  const int Kt = K + n_shared;
  const size_t row = static_cast<size_t>(t) * Kt;
#pragma unroll
  for (int k = 0; k < kMaxTopK; ++k) {
    if (k < K) {
      ids[row + k] = se[k];
      w[row + k] = expf(sv[k] - m) / sum;
      if (lds_ids) lds_ids[row + k] = se[k];
    }
  }
  for (int j = 0; j < n_shared; ++j) {
    ids[row + K + j] = E + j;
    w[row + K + j] = gate ? gate[static_cast<size_t>(t) * n_shared + j] : 1.0f;
    if (lds_ids) lds_ids[row + K + j] = E + j;
  }
}

__global__ __launch_bounds__(256) void k_route_topk(const float* __restrict__ logits, int T, int E,
                                                    int K, int renorm, int n_shared,
                                                    const float* __restrict__ gate, int32_t* __restrict__ ids,
                                                    float* __restrict__ w) {
  const int t = blockIdx.x * 4 + static_cast<int>(threadIdx.x >> 6);
  if (t >= T) return;   // wave-uniform
  route_token(logits, t, E, K, renorm, n_shared, gate, ids, w, nullptr);
}

// Token permutation, one workgroup per expert e. Each workgroup builds the
// full histogram (order-free LDS atomics on counts), so every expert's offset
// is known everywhere; wave q then owns the q-th quarter of the slots and
// places e's slots in it in slot order: a ballot per 64 slots gives the ranks,
// the counts of the earlier quarters the base. No order depends on timing.
constexpr int kPermThreads = 256;
constexpr int kMaxExperts = 256;

// Ballots of `e` over slots [q0, q1) in 8-block steps (loads in flight
// together); calls f(s, rank within the step's block, block mask) for e's slots
// and returns their count.
template <class F>
__device__ __forceinline__ int perm_scan(const int32_t* __restrict__ ids, int q0, int q1, int e, F&& f) {
  const int lane = lane_id();
  int c = 0;
  for (int base = q0; base < q1; base += 8 * 64) {
    int idb[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int s = base + 64 * q + lane;
      idb[q] = s < q1 ? ids[s] : -1;
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const unsigned long long m = __ballot(idb[q] == e);
      if (idb[q] == e) {
        const int r = static_cast<int>(__builtin_amdgcn_mbcnt_hi(
            static_cast<uint32_t>(m >> 32), __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(m), 0u)));
        f(base + 64 * q + lane, c + r);
      }
      c += __popcll(m);
    }
  }
  return c;
}

__global__ __launch_bounds__(kPermThreads) void k_permute(const int32_t* __restrict__ ids, int S,
                                                          int E, int32_t* __restrict__ offsets,
                                                          int32_t* __restrict__ sorted_slot,
                                                          int32_t* __restrict__ slot_pos) {
  __shared__ int cnt[kMaxExperts];
  __shared__ int qcnt[4];
  const int e = blockIdx.x, tid = threadIdx.x, wave = tid >> 6, lane = lane_id();
  for (int i = tid; i < E; i += kPermThreads) cnt[i] = 0;
  __syncthreads();
  // eight ids per thread in flight before their counts are added
  for (int s0 = tid; s0 < S; s0 += 8 * kPermThreads) {
    int id[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int s = s0 + j * kPermThreads;
      id[j] = s < S ? ids[s] : -1;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (id[j] >= 0 && id[j] < E) atomicAdd(&cnt[id[j]], 1);
  }
  const int per = ((S + 3) / 4 + 63) / 64 * 64;
  const int q0 = min(S, wave * per), q1 = min(S, q0 + per);
  const int mine = perm_scan(ids, q0, q1, e, [](int, int) {});
  if (lane == 0) qcnt[wave] = mine;
  __syncthreads();
  if (e == 0 && tid == 0) {
    int acc = 0;
    for (int x = 0; x < E; ++x) {
      offsets[x] = acc;
      acc += cnt[x];
    }
    offsets[E] = acc;
  }
  int base = 0;
  for (int x = 0; x < e; ++x) base += cnt[x];
  for (int w = 0; w < wave; ++w) base += qcnt[w];
  perm_scan(ids, q0, q1, e, [&](int s, int r) {
    sorted_slot[base + r] = s;
    slot_pos[s] = base + r;
  });
}

// Small batches (T (K + n_shared) <= kFusedMaxSlots, T E <= kFusedMaxLogits):
// routing and permutation in one workgroup, so one launch does both.
//  1. the batch's logits are staged in LDS (coalesced loads);
//  2. thread t selects token t's top K by a serial pass over its logits in
//     expert order, carrying each logit down a fixed K-entry list kept in
//     (value descending, index ascending) order (the order of the wave
//     arg-max), then forms the weights with the same fp32 arithmetic as
//     route_token;
//  3. wave c ranks the slots of chunk c (64 slots) among the chunk's slots of
//     the same expert (one ballot per distinct expert in the chunk) and
//     counts them per expert;
//  4. per expert the chunk counts become absolute starts (offsets plus the
//     earlier chunks), so slot s lands at start[chunk][expert] + rank: slots
//     of an expert in increasing s, as in the two-launch path.
constexpr int kFusedThreads = 1024;
constexpr int kFusedMaxSlots = 1024;
constexpr int kFusedChunks = kFusedMaxSlots / 64;
constexpr int kFusedMaxLogits = 8192;

template <int KL>
__device__ __forceinline__ void route_token_serial(const float* l, int t, int E, int K, int renorm, int n_shared,
                                                   const float* __restrict__ gate, int32_t* __restrict__ ids,
                                                   float* __restrict__ w, int* lds_ids) {
  float sv[KL];
  int se[KL];
#pragma unroll
  for (int k = 0; k < KL; ++k) {
    sv[k] = -__builtin_inff();
    se[k] = -1;
  }
  for (int e = 0; e < E; ++e) {
    float v = l[e];
    int x = e;
#pragma unroll
    for (int k = 0; k < KL; ++k) {
      // (value descending, index ascending): a new logit has the highest
      // index so far, a displaced entry may precede an equal one below it
      if (k < K && (se[k] < 0 || v > sv[k] || (v == sv[k] && x < se[k]))) {
        const float tv = sv[k];
        const int tx = se[k];
        sv[k] = v;
        se[k] = x;
        v = tv;
        x = tx;
      }
    }
  }
  const float m = sv[0];
  float sum = 0.0f;
  if (renorm) {
#pragma unroll
    for (int k = 0; k < KL; ++k)
      if (k < K) sum += expf(sv[k] - m);
  } else {
    for (int e = 0; e < E; ++e) sum += expf(l[e] - m);
  }
  const int Kt = K + n_shared;
  const size_t row = static_cast<size_t>(t) * Kt;
#pragma unroll
  for (int k = 0; k < KL; ++k) {
    if (k < K) {
      ids[row + k] = se[k];
      w[row + k] = expf(sv[k] - m) / sum;
      lds_ids[row + k] = se[k];
    }
  }
  for (int j = 0; j < n_shared; ++j) {
    ids[row + K + j] = E + j;
    w[row + K + j] = gate ? gate[static_cast<size_t>(t) * n_shared + j] : 1.0f;
    lds_ids[row + K + j] = E + j;
  }
}

// KL: the list length of the top-K selection (a power of two, at least K)
template <int KL>
__global__ __launch_bounds__(kFusedThreads) void k_route_permute(const float* __restrict__ logits, int T, int E,
                                                                 int K, int renorm, int n_shared,
                                                                 const float* __restrict__ gate,
                                                                 int32_t* __restrict__ ids, float* __restrict__ w,
                                                                 int32_t* __restrict__ offsets,
                                                                 int32_t* __restrict__ sorted_slot,
                                                                 int32_t* __restrict__ slot_pos) {
  __shared__ float s_lg[kFusedMaxLogits];
  __shared__ int s_ids[kFusedMaxSlots];
  __shared__ int s_rank[kFusedMaxSlots];
  __shared__ int cc[kFusedChunks][kMaxExperts];   // per chunk: count, then absolute start
  __shared__ int tot[kMaxExperts];
  const int tid = threadIdx.x, wave = tid >> 6, lane = lane_id();
  const int Et = E + n_shared, S = T * (K + n_shared);
  const int nchunk = (S + 63) / 64;
  for (int i = tid; i < T * E; i += kFusedThreads) s_lg[i] = logits[i];
  for (int i = tid; i < kFusedChunks * kMaxExperts; i += kFusedThreads) cc[i / kMaxExperts][i % kMaxExperts] = 0;
  __syncthreads();
  if (tid < T)
    route_token_serial<KL>(s_lg + static_cast<size_t>(tid) * E, tid, E, K, renorm, n_shared, gate, ids, w, s_ids);
  __syncthreads();
  if (wave < nchunk) {
    const int s = wave * 64 + lane;
    const bool live = s < S;
    const int id = live ? s_ids[s] : -1;
    unsigned long long todo = __ballot(live);
    int rank = 0;
    while (todo) {
      const int first = __ffsll(static_cast<long long>(todo)) - 1;
      const int e0 = __shfl(id, first);
      const unsigned long long m = __ballot(id == e0);
      if (id == e0) {
        rank = static_cast<int>(__builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(m >> 32),
                                                          __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(m), 0u)));
      }
      if (lane == first) cc[wave][e0] = __popcll(m);
      todo &= ~m;
    }
    if (live) s_rank[s] = rank;
  }
  __syncthreads();
  if (tid < Et) {
    int n = 0;
    for (int c = 0; c < nchunk; ++c) n += cc[c][tid];
    tot[tid] = n;
  }
  __syncthreads();
  if (tid < Et) {
    int start = 0;
    for (int x = 0; x < tid; ++x) start += tot[x];
    offsets[tid] = start;
    if (tid == Et - 1) offsets[Et] = start + tot[tid];
    for (int c = 0; c < nchunk; ++c) {
      const int n = cc[c][tid];
      cc[c][tid] = start;
      start += n;
    }
  }
  __syncthreads();
  for (int s = tid; s < S; s += kFusedThreads) {
    const int pos = cc[s >> 6][s_ids[s]] + s_rank[s];
    sorted_slot[pos] = s;
    slot_pos[s] = pos;
  }
}

// ---------------------------------------------------------------------------
// Group-wise RTN: quantization of 16-bit rows into a page at load time (or a
// 16-bit page's layout transform), and requantization of pool pages to fewer
// bits (k_requant, below).
//
// Page layout: tiles of 16 rows x 128 values stored tile after tile (row tile
// major); inside a tile, lane l = 16 lg + lc (row lc, k-run lg) of k-step i
// owns 16 contiguous bytes: 16-bit values at 1024 i + 16 l, 8-bit codes of
// steps 2u, 2u+1 at 1024 u + 16 l, the four 4-bit words at 16 l. A wave reads
// or writes a tile as contiguous 1 KB rows. One wave handles one row tile over
// one span of K (max(G,128) values); groups are reduced over the lane groups.
// ---------------------------------------------------------------------------


// Group layout along K: G = 64 (two groups per 128-block), G = 128 (one),
// G = 256 or 512 (one group spans 2 or 4 blocks). The activation dtype ACT,
// the scale dtype SDT and the group layout GK are template parameters of the
// kernels; the load-time kernel's destination bitwidth varies per job.
enum { kQG64 = 0, kQG128 = 1, kQGBig = 2 };

// The raw 16-byte pieces lane l holds of one 128-value block of a row tile,
// for every source format (16-bit: four pieces; 8-bit: two; 4-bit: one), plus
// the (scale, zero) word of each k-step's group for quantized sources (the
// load-time kernel reads 16-bit sources only; k_requant all three).
struct QRaw {
  u32x4 w[4];
  uint32_t sz[4];
};

// The lane's four 16-byte pieces of 16-bit block blk of row tile tau: from a
// 16-bit pool page (tile layout) or from R x K row-major rows (src_plain).
__device__ __forceinline__ void q_load(const QJob& job, int tau, int blk, QRaw& raw) {
  const int lane = lane_id(), lc = lane & 15, lg = lane >> 4;
  const int K = job.K, nkb = K / 128;
  const size_t tile = static_cast<size_t>(tau) * nkb + blk;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint8_t* src = job.src_plain
        ? job.src + (static_cast<size_t>(tau * 16 + lc) * K + blk * 128 + 32 * i + 8 * lg) * 2
        : job.src + tile * 4096 + 1024 * i + 16 * lane;
    raw.w[i] = *reinterpret_cast<const u32x4*>(src);
  }
}

// The 32 values (k-steps i = 0..3, 8 values each) lane l holds of the block,
// widened to fp32 (exactly).
template <int ACT>
__device__ __forceinline__ void q_read(const QJob& job, int tau, int blk, float (&v)[32]) {
  QRaw raw;
  q_load(job, tau, blk, raw);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      v[8 * i + 2 * q] = val16(raw.w[i][q], ACT);
      v[8 * i + 2 * q + 1] = val16(raw.w[i][q] >> 16, ACT);
    }
}

// (scale, zero) bit patterns of a group from its extremes (the quantizer's steps).
template <int SDT>
__device__ __forceinline__ void q_params(float lo, float hi, int Q, uint32_t* sb, uint32_t* zb) {
  *zb = round_down16(lo, SDT);
  const float z = val16(*zb, SDT);
  const float r = hi - z;
  *sb = 0u;
  if (r == 0.0f) return;
  *sb = round_up16(r / static_cast<float>(Q), SDT);
  if (val16(*sb, SDT) * static_cast<float>(Q) < r) *sb += 1u;   // s > 0: next value up
}

// One group's (scale, zero) as the code computation uses them. A zero scale
// (every code 0) takes rs = 0, so the fast quotient below is 0.
struct QGroup {
  float z, s, rs;   // zero, scale, approximate 1 / s
  bool fast;        // d * rs decides the code (s far from the fp32 range limits, or s = 0)
};
template <int SDT>
__device__ __forceinline__ QGroup q_group(uint32_t sb, uint32_t zb) {
  QGroup g;
  g.z = val16(zb, SDT);
  g.s = val16(sb, SDT);
  const bool zero = sb == 0u;
  g.rs = zero ? 0.0f : __builtin_amdgcn_rcpf(g.s);
  g.fast = zero || (g.s >= 0x1p-100f && g.s <= 0x1p100f);
  return g;
}

// c = clamp(rint(fl32(d / s)), 0, Q) with d = fl32(v - z), d / s in [0, Q]
// up to rounding. The quotient is first taken as d * rcp(s), within a few
// fp32 ulp (below 2^-14 for quotients up to 256) of the correctly rounded
// one, so it decides rint unless it lies within 2^-12 of a half-integer;
// there, and for extreme scales, the correctly rounded division decides.
// Either way the code equals the one of the plain definition.
__device__ __forceinline__ uint32_t q_code(float v, const QGroup& g, int Q) {
  const float d = v - g.z;
  const float qa = d * g.rs;
  float c = rintf(qa);
  if (!g.fast || fabsf(qa - c) > 0.5f - 0x1p-12f) c = rintf(d / g.s);
  return static_cast<uint32_t>(__builtin_amdgcn_fmed3f(c, 0.0f, static_cast<float>(Q)));
}

// Codes of one block from its values and its group parameters, stored in the
// destination page's tile layout; the (scale, zero) words are written by the
// caller. Group g0 covers k-steps 0-3 (G >= 128) or 0-1 and g1 2-3 (G = 64).
template <int SDT, int GK>
__device__ __forceinline__ void q_store_codes(const QJob& job, int tau, int blk, const float (&v)[32], uint32_t sb0,
                                              uint32_t zb0, uint32_t sb1, uint32_t zb1, int Q) {
  const int lane = lane_id();
  const QGroup g0 = q_group<SDT>(sb0, zb0), g1 = q_group<SDT>(sb1, zb1);
  uint32_t c[32];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const bool second = GK == kQG64 && i >= 2;
#pragma unroll
    for (int q = 0; q < 8; ++q) c[8 * i + q] = q_code(v[8 * i + q], second ? g1 : g0, Q);
  }
  const size_t tile = static_cast<size_t>(tau) * (job.K / 128) + blk;
  if (job.dst_bits == 8) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      u32x4 o;
#pragma unroll
      for (int w = 0; w < 4; ++w)
        o[w] = c[16 * u + 4 * w] | (c[16 * u + 4 * w + 1] << 8) | (c[16 * u + 4 * w + 2] << 16) |
               (c[16 * u + 4 * w + 3] << 24);
      *reinterpret_cast<u32x4*>(job.dst + tile * 2048 + 1024 * u + 16 * lane) = o;
    }
  } else {
    u32x4 o;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint32_t w = 0u;
#pragma unroll
      for (int t = 0; t < 4; ++t) w |= (c[8 * i + 2 * t] << (4 * t)) | (c[8 * i + 2 * t + 1] << (16 + 4 * t));
      o[i] = w;
    }
    *reinterpret_cast<u32x4*>(job.dst + tile * 1024 + 16 * lane) = o;
  }
}

// 16-bit destination: the block's values rounded to the activation dtype, in
// tile layout (a layout transform of a plain 16-bit source).
template <int ACT>
__device__ __forceinline__ void q_store16(const QJob& job, int tau, int blk, const float (&v)[32]) {
  const int lane = lane_id();
  const size_t tile = static_cast<size_t>(tau) * (job.K / 128) + blk;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    u32x4 o;
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q] = rne16(v[8 * i + 2 * q], ACT) | (rne16(v[8 * i + 2 * q + 1], ACT) << 16);
    *reinterpret_cast<u32x4*>(job.dst + tile * 4096 + 1024 * i + 16 * lane) = o;
  }
}

// Extremes of the block's group(s) across the row's four lane groups.
template <int GK>
__device__ __forceinline__ void q_extremes(const float (&v)[32], float& lo0, float& hi0, float& lo1, float& hi1) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      if (GK == kQG64 && i >= 2) {
        lo1 = fminf(lo1, v[8 * i + q]);
        hi1 = fmaxf(hi1, v[8 * i + q]);
      } else {
        lo0 = fminf(lo0, v[8 * i + q]);
        hi0 = fmaxf(hi0, v[8 * i + q]);
      }
    }
}

__device__ __forceinline__ void q_rowreduce(float& lo0, float& hi0, float& lo1, float& hi1) {
  // the row's other values sit in lanes lc + 16, lc + 32, lc + 48
#pragma unroll
  for (int m = 16; m <= 32; m <<= 1) {
    lo0 = fminf(lo0, __shfl_xor(lo0, m));
    hi0 = fmaxf(hi0, __shfl_xor(hi0, m));
    lo1 = fminf(lo1, __shfl_xor(lo1, m));
    hi1 = fmaxf(hi1, __shfl_xor(hi1, m));
  }
}

// Register-lean form of the one-block path (G <= 128): the block stays in
// its loaded words and each value is widened again where it is used (the
// group extremes, then the codes, each packed as soon as it is computed), so
// no 32-value fp32 array is live and more waves fit on a SIMD. The values are
// the same: a 16-bit value exactly, or fl32(z + c s).
template <int ACT, int SDT, int SRC>
__device__ __forceinline__ float q_elem(const QRaw& raw, int e) {
  const int i = e >> 3, q = e & 7;
  if constexpr (SRC == 16) {
    const uint32_t w = raw.w[i][q >> 1];
    return val16((q & 1) ? (w >> 16) : w, ACT);
  } else {
    uint32_t c;
    if constexpr (SRC == 8) c = (raw.w[e >> 4][(e >> 2) & 3] >> (8 * (e & 3))) & 0xFFu;
    else c = (raw.w[0][i] >> ((q & 1) ? 16 + 4 * (q >> 1) : 4 * (q >> 1))) & 15u;
    const float s = val16(raw.sz[i], SDT), z = val16(raw.sz[i] >> 16, SDT);
    return z + static_cast<float>(c) * s;   // c*s exact
  }
}

// One 16-bit block quantized to the job's destination (16: layout transform).
template <int ACT, int SDT, int GK>
__device__ __forceinline__ void q_block(const QJob& job, const QJobBatch& b, const QRaw& raw, int tau, int blk, int lg,
                                        int r, int Q) {
  constexpr int SRC = 16;
  const int lane = lane_id();
  const size_t tile = static_cast<size_t>(tau) * (job.K / 128) + blk;
  if (job.dst_bits == 16) {          // layout transform of a 16-bit page
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      u32x4 o;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        o[q] = rne16(q_elem<ACT, SDT, SRC>(raw, 8 * i + 2 * q), ACT) |
               (rne16(q_elem<ACT, SDT, SRC>(raw, 8 * i + 2 * q + 1), ACT) << 16);
      *reinterpret_cast<u32x4*>(job.dst + tile * 4096 + 1024 * i + 16 * lane) = o;
    }
    return;
  }
  float lo0 = __builtin_inff(), hi0 = -__builtin_inff(), lo1 = lo0, hi1 = hi0;
#pragma unroll
  for (int e = 0; e < 32; ++e) {
    const float v = q_elem<ACT, SDT, SRC>(raw, e);
    if (GK == kQG64 && e >= 16) {
      lo1 = fminf(lo1, v);
      hi1 = fmaxf(hi1, v);
    } else {
      lo0 = fminf(lo0, v);
      hi0 = fmaxf(hi0, v);
    }
  }
  q_rowreduce(lo0, hi0, lo1, hi1);
  uint32_t sb0, zb0, sb1 = 0u, zb1 = 0u;
  q_params<SDT>(lo0, hi0, Q, &sb0, &zb0);
  if (GK == kQG64) q_params<SDT>(lo1, hi1, Q, &sb1, &zb1);
  const QGroup g0 = q_group<SDT>(sb0, zb0), g1 = q_group<SDT>(sb1, zb1);
  auto code = [&](int e) { return q_code(q_elem<ACT, SDT, SRC>(raw, e), (GK == kQG64 && e >= 16) ? g1 : g0, Q); };
  if (job.dst_bits == 8) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      u32x4 o;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int e = 16 * u + 4 * w;
        o[w] = code(e) | (code(e + 1) << 8) | (code(e + 2) << 16) | (code(e + 3) << 24);
      }
      *reinterpret_cast<u32x4*>(job.dst + tile * 2048 + 1024 * u + 16 * lane) = o;
    }
  } else {
    u32x4 o;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint32_t w = 0u;
#pragma unroll
      for (int t = 0; t < 4; ++t) w |= (code(8 * i + 2 * t) << (4 * t)) | (code(8 * i + 2 * t + 1) << (16 + 4 * t));
      o[i] = w;
    }
    *reinterpret_cast<u32x4*>(job.dst + tile * 1024 + 16 * lane) = o;
  }
  if (lg == 0) {
    const int gi = GK == kQG64 ? 2 * blk : blk;
    *reinterpret_cast<uint32_t*>(job.dst_sz + (static_cast<size_t>(gi) * b.R + r) * 4) = sb0 | (zb0 << 16);
    if (GK == kQG64)
      *reinterpret_cast<uint32_t*>(job.dst_sz + (static_cast<size_t>(gi + 1) * b.R + r) * 4) = sb1 | (zb1 << 16);
  }
}

// Work item -> (job j, 16-row tile tau, span sp of max(G, 128) values); job
// j's items start at job[j].item_base.
struct QItem {
  int j, tau, sp;
};
__device__ __forceinline__ QItem q_item(const QJobBatch& b, uint32_t item, int span) {
  QItem it;
  int j = 0;
  while (j + 1 < b.n_jobs && item >= b.job[j + 1].item_base) ++j;   // wave-uniform
  const int nsp = (b.job[j].K / 128) / span;
  const int rem = static_cast<int>(item - b.job[j].item_base);
  it.j = j;
  it.tau = rem / nsp;
  it.sp = rem % nsp;
  return it;
}

// One wave per item: a 16-row tile over one span of K. G <= 128 (every group
// inside one block): one block, quantized from registers in one pass. G > 128:
// G / 128 blocks, two passes (the group's extremes, then the codes).
template <int ACT, int SDT, int GK>
__device__ __forceinline__ void qjobs_item(const QJobBatch& b) {
  const uint32_t item = blockIdx.x * 4u + (threadIdx.x >> 6);
  if (item >= b.total_items) return;
  const int lane = lane_id(), lc = lane & 15, lg = lane >> 4;
  const int R = b.R;
  const int span = GK == kQGBig ? b.G / 128 : 1;    // blocks per item
  const QItem it = q_item(b, item, span);
  const QJob& job = b.job[it.j];
  const int tau = it.tau, sp = it.sp;
  const int r = tau * 16 + lc;
  const int Q = (1 << job.dst_bits) - 1;
  if constexpr (GK != kQGBig) {
    QRaw raw;
    q_load(job, tau, sp, raw);
    q_block<ACT, SDT, GK>(job, b, raw, tau, sp, lg, r, Q);
    (void)R;
  } else {
    float v[32];
    if (job.dst_bits == 16) {
      for (int blk = sp * span; blk < (sp + 1) * span; ++blk) {
        q_read<ACT>(job, tau, blk, v);
        q_store16<ACT>(job, tau, blk, v);
      }
      return;
    }
    float lo0 = __builtin_inff(), hi0 = -__builtin_inff(), lo1 = lo0, hi1 = hi0;
    for (int blk = sp * span; blk < (sp + 1) * span; ++blk) {
      q_read<ACT>(job, tau, blk, v);
      q_extremes<GK>(v, lo0, hi0, lo1, hi1);
    }
    q_rowreduce(lo0, hi0, lo1, hi1);
    uint32_t sb0, zb0;
    q_params<SDT>(lo0, hi0, Q, &sb0, &zb0);
    for (int blk = sp * span; blk < (sp + 1) * span; ++blk) {
      q_read<ACT>(job, tau, blk, v);
      q_store_codes<SDT, GK>(job, tau, blk, v, sb0, zb0, 0u, 0u, Q);
    }
    if (lg == 0) *reinterpret_cast<uint32_t*>(job.dst_sz + (static_cast<size_t>(sp) * R + r) * 4) = sb0 | (zb0 << 16);
  }
}

template <int ACT, int SDT, int GK>
__global__ __launch_bounds__(256) void k_qjobs(const QJobBatch b) {
  qjobs_item<ACT, SDT, GK>(b);
}

// G = 128 (one group per block): the one-block path fits in 64 VGPRs, so
// eight waves per SIMD and 32 blocks per CU are in flight.
template <int ACT, int SDT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(8))) void k_qjobs_g128(const QJobBatch b) {
  qjobs_item<ACT, SDT, kQG128>(b);
}

// ---------------------------------------------------------------------------
// Requantization of pool pages to fewer bits (16 -> 8, 16 -> 4, 8 -> 4).
//
// A launch covers up to kMaxRqJobs pages of one (source, destination) pair
// of bitwidths. The grid is (spans / 4, row tiles, pages): the wave of span
// 4 blockIdx.x + w of row tile blockIdx.y of page blockIdx.z codes that
// 16-row x max(G, 128)-value piece, so it finds its work from its indices
// with no search. Waves past a page's last span exit at once. The bitwidths
// are template parameters: every wave runs one straight path, the kernel
// stays under 64 VGPRs and eight waves per SIMD keep their loads in flight.
// Pool addresses are formed in the global address space, so the loads and
// stores are plain global (not flat) accesses; source blocks and codes are
// touched once, so both move as nontemporal (streaming) accesses.
// ---------------------------------------------------------------------------

#define PW_GLOBAL __attribute__((address_space(1)))
typedef const PW_GLOBAL uint8_t* gsrc_t;
typedef PW_GLOBAL uint8_t* gdst_t;

template <int SRC, int GK>
__device__ __forceinline__ void rq_load(gsrc_t src, gsrc_t src_sz, size_t tile, int R, int G, int blk, int r,
                                        QRaw& raw) {
  const int lane = lane_id();
  if constexpr (SRC == 16) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      raw.w[i] = __builtin_nontemporal_load(reinterpret_cast<const PW_GLOBAL u32x4*>(src + tile * 4096 + 1024 * i + 16 * lane));
  } else {
#pragma unroll
    for (int u = 0; u < 2; ++u)
      raw.w[u] = __builtin_nontemporal_load(reinterpret_cast<const PW_GLOBAL u32x4*>(src + tile * 2048 + 1024 * u + 16 * lane));
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = GK == kQG64 ? 2 * blk + (i >> 1) : GK == kQG128 ? blk : (blk * 128) / G;
      raw.sz[i] = *reinterpret_cast<const PW_GLOBAL uint32_t*>(src_sz + (static_cast<size_t>(g) * R + r) * 4);
    }
  }
}

// The code of v as an integer-valued float (q_code without the conversion).
__device__ __forceinline__ float q_codef(float v, const QGroup& g, float Qf) {
  const float d = v - g.z;
  const float qa = d * g.rs;
  float c = rintf(qa);
  if (!g.fast || fabsf(qa - c) > 0.5f - 0x1p-12f) c = rintf(d / g.s);
  return __builtin_amdgcn_fmed3f(c, 0.0f, Qf);
}

// Codes of one block in the destination tile layout. A code is an integer in
// [0, Q], so the byte conversion of cvt_pk_u8_f32 is exact; each call places
// one code in a chosen byte of a word. 4-bit word of k-step i: nibble t holds
// code 8i + 2t and nibble 4 + t code 8i + 2t + 1, i.e. bytes [c0 c4 c1 c5]
// in the low nibbles and [c2 c6 c3 c7] in the high ones.
template <int DST, typename CF>
__device__ __forceinline__ void rq_store_codes(gdst_t dst, size_t tile, CF cf) {
  const int lane = lane_id();
  if constexpr (DST == 8) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      u32x4 o;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int e = 16 * u + 4 * w;
        uint32_t x = __builtin_amdgcn_cvt_pk_u8_f32(cf(e), 0, 0u);
        x = __builtin_amdgcn_cvt_pk_u8_f32(cf(e + 1), 1, x);
        x = __builtin_amdgcn_cvt_pk_u8_f32(cf(e + 2), 2, x);
        o[w] = __builtin_amdgcn_cvt_pk_u8_f32(cf(e + 3), 3, x);
      }
      __builtin_nontemporal_store(o, reinterpret_cast<PW_GLOBAL u32x4*>(dst + tile * 2048 + 1024 * u + 16 * lane));
    }
  } else {
    u32x4 o;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = 8 * i;
      uint32_t a = __builtin_amdgcn_cvt_pk_u8_f32(cf(e), 0, 0u);
      a = __builtin_amdgcn_cvt_pk_u8_f32(cf(e + 4), 1, a);
      a = __builtin_amdgcn_cvt_pk_u8_f32(cf(e + 1), 2, a);
      a = __builtin_amdgcn_cvt_pk_u8_f32(cf(e + 5), 3, a);
      uint32_t c = __builtin_amdgcn_cvt_pk_u8_f32(cf(e + 2), 0, 0u);
      c = __builtin_amdgcn_cvt_pk_u8_f32(cf(e + 6), 1, c);
      c = __builtin_amdgcn_cvt_pk_u8_f32(cf(e + 3), 2, c);
      c = __builtin_amdgcn_cvt_pk_u8_f32(cf(e + 7), 3, c);
      o[i] = a | (c << 4);
    }
    __builtin_nontemporal_store(o, reinterpret_cast<PW_GLOBAL u32x4*>(dst + tile * 1024 + 16 * lane));
  }
}

template <int ACT, int SDT, int GK, int SRC, int DST>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(8))) void k_requant(const RqBatch b) {
  const int j = blockIdx.z;
  const int nkb = ((b.kbit[j >> 5] >> (j & 31)) & 1u) ? b.kb[1] : b.kb[0];
  const int span = GK == kQGBig ? b.G / 128 : 1;   // blocks per wave
  const int sp = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (sp * span >= nkb) return;
  const int lane = lane_id(), lc = lane & 15, lg = lane >> 4;
  const int R = b.R, tau = blockIdx.y, r = tau * 16 + lc;
  constexpr float Qf = static_cast<float>((1 << DST) - 1);
  const size_t rk = static_cast<size_t>(R) * nkb * 128;   // values of the page
  gsrc_t src = (gsrc_t)b.pool + static_cast<size_t>(b.src[j]) * 256;   // generic to global: C-style casts
  gsrc_t src_sz = src + rk * SRC / 8;
  gdst_t dst = (gdst_t)b.pool + static_cast<size_t>(b.dst[j]) * 256;
  gdst_t dst_sz = dst + rk * DST / 8;
  const size_t row0 = static_cast<size_t>(tau) * nkb;   // first tile of the row tile
  float lo0 = __builtin_inff(), hi0 = -__builtin_inff(), lo1 = lo0, hi1 = hi0;
  if constexpr (GK != kQGBig) {
    QRaw raw;
    rq_load<SRC, GK>(src, src_sz, row0 + sp, R, b.G, sp, r, raw);
#pragma unroll
    for (int e = 0; e < 32; ++e) {
      const float v = q_elem<ACT, SDT, SRC>(raw, e);
      if (GK == kQG64 && e >= 16) {
        lo1 = fminf(lo1, v);
        hi1 = fmaxf(hi1, v);
      } else {
        lo0 = fminf(lo0, v);
        hi0 = fmaxf(hi0, v);
      }
    }
    q_rowreduce(lo0, hi0, lo1, hi1);
    uint32_t sb0, zb0, sb1 = 0u, zb1 = 0u;
    q_params<SDT>(lo0, hi0, static_cast<int>(Qf), &sb0, &zb0);
    if (GK == kQG64) q_params<SDT>(lo1, hi1, static_cast<int>(Qf), &sb1, &zb1);
    const QGroup g0 = q_group<SDT>(sb0, zb0), g1 = q_group<SDT>(sb1, zb1);
    rq_store_codes<DST>(dst, row0 + sp, [&](int e) {
      return q_codef(q_elem<ACT, SDT, SRC>(raw, e), (GK == kQG64 && e >= 16) ? g1 : g0, Qf);
    });
    if (lg == 0) {
      const int gi = GK == kQG64 ? 2 * sp : sp;
      *reinterpret_cast<PW_GLOBAL uint32_t*>(dst_sz + (static_cast<size_t>(gi) * R + r) * 4) = sb0 | (zb0 << 16);
      if (GK == kQG64)
        *reinterpret_cast<PW_GLOBAL uint32_t*>(dst_sz + (static_cast<size_t>(gi + 1) * R + r) * 4) = sb1 | (zb1 << 16);
    }
  } else {
    // G > 128: the group spans `span` blocks; its extremes first, then the
    // codes, each pass reading the blocks again
    for (int blk = sp * span; blk < (sp + 1) * span; ++blk) {
      QRaw raw;
      rq_load<SRC, GK>(src, src_sz, row0 + blk, R, b.G, blk, r, raw);
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        const float v = q_elem<ACT, SDT, SRC>(raw, e);
        lo0 = fminf(lo0, v);
        hi0 = fmaxf(hi0, v);
      }
    }
    q_rowreduce(lo0, hi0, lo1, hi1);
    uint32_t sb0, zb0;
    q_params<SDT>(lo0, hi0, static_cast<int>(Qf), &sb0, &zb0);
    const QGroup g0 = q_group<SDT>(sb0, zb0);
    for (int blk = sp * span; blk < (sp + 1) * span; ++blk) {
      QRaw raw;
      rq_load<SRC, GK>(src, src_sz, row0 + blk, R, b.G, blk, r, raw);
      rq_store_codes<DST>(dst, row0 + blk, [&](int e) { return q_codef(q_elem<ACT, SDT, SRC>(raw, e), g0, Qf); });
    }
    if (lg == 0) *reinterpret_cast<PW_GLOBAL uint32_t*>(dst_sz + (static_cast<size_t>(sp) * R + r) * 4) = sb0 | (zb0 << 16);
  }
}

__global__ void k_entry_writes(pw_page_entry* table, const EntryWrites w) {
  const int i = threadIdx.x;
  if (i < w.n) table[w.idx[i]] = w.ent[i];
}

__global__ void k_clear_table(pw_page_entry* table, size_t n) {
  for (size_t i = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; i < n;
       i += static_cast<size_t>(gridDim.x) * blockDim.x)
    table[i] = pw_page_entry{0, 0, 0, PW_PAGE_ABSENT, 0, 0};
}

// ---------------------------------------------------------------------------
// combine: y[t] = sum_k w[t,k] * sum_split opart[split][slot_pos[t,k]]
// (k ascending; the last n_shared columns are shared-expert slots, whose
// down projection has nsplit_sh K splits)
// ---------------------------------------------------------------------------

// A thread holds four outputs of token t. Columns are taken C at a time (C
// of 2, 4, 6, 8: the column count rounded up, at most 16 / NSP; NSP: the largest
// split count rounded up to 1, 2, 4 or 8): the partial rows of every split
// of those columns are all loaded before any is summed, so up to 16 loads of
// a thread are in flight together; the sums keep the order (splits ascending
// per column, columns ascending into y).
template <int NSP, int C>
__global__ __launch_bounds__(256) void k_combine(const GemmArgs a) {
  const int t = blockIdx.x;
  const int n = (blockIdx.y * 256 + threadIdx.x) * 4;
  if (n >= a.H) return;
  f32x4 y = {0.f, 0.f, 0.f, 0.f};
  const size_t row = static_cast<size_t>(t) * a.topk;
  for (int k0 = 0; k0 < a.topk; k0 += C) {
    int pos[C], nsp[C];
    float wk[C];
#pragma unroll
    for (int j = 0; j < C; ++j) {
      const int k = min(k0 + j, a.topk - 1);
      pos[j] = clampi(a.slot_pos[row + k], 0, a.S - 1);
      wk[j] = a.topk_w[row + k];
      nsp[j] = k0 + j >= a.topk ? 0 : k < a.topk - a.n_shared ? a.nsplit : a.nsplit_sh;
    }
    // unconditional loads (a split past the column's count reloads one of its
    // own rows and is not summed): no branch separates them from each other
    f32x4 part[C][NSP];
#pragma unroll
    for (int j = 0; j < C; ++j)
#pragma unroll
      for (int sp = 0; sp < NSP; ++sp) {
        const int spc = min(sp, max(nsp[j] - 1, 0));
        part[j][sp] = *reinterpret_cast<const f32x4*>(a.opart + (static_cast<size_t>(spc) * a.S + pos[j]) * a.H + n);
      }
#pragma unroll
    for (int j = 0; j < C; ++j) {
      if (k0 + j < a.topk) {
        f32x4 o = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int sp = 0; sp < NSP; ++sp)
          if (sp < nsp[j]) o += part[j][sp];
        y += wk[j] * o;
      }
    }
  }
  if (a.out_fp32) {
    *reinterpret_cast<f32x4*>(static_cast<float*>(a.y) + static_cast<size_t>(t) * a.H + n) = y;
  } else {
    u32x2 o;
    o[0] = rne16(y[0], a.act) | (rne16(y[1], a.act) << 16);
    o[1] = rne16(y[2], a.act) | (rne16(y[3], a.act) << 16);
    *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(a.y) + static_cast<size_t>(t) * a.H + n) = o;
  }
}

}  // namespace

namespace {

// ---------------------------------------------------------------------------
// Nested bit-plane pages: quantization of a block (one thread per row, every
// sum in order of k in float64, so the result is reproducible bit for bit)
// and the packing of its 8-bit codes into bit-planes in lane order.
// ---------------------------------------------------------------------------

// Nearest-even rounding of a double straight to the 16-bit format (one
// rounding): r = rint(x / q) q with q the format's spacing at x is exact.
__device__ __forceinline__ uint32_t rne16_d(double x, int fmt) {
  if (x == 0.0) return __builtin_signbit(x) ? 0x8000u : 0u;
  const int emin = fmt == PW_BF16 ? -126 : -14;
  const int frac = fmt == PW_BF16 ? 7 : 10;
  int e = 0;
  (void)frexp(x, &e);
  const int ex = e - 1 > emin ? e - 1 : emin;
  const double q = ldexp(1.0, ex - frac);
  const float r = static_cast<float>(rint(x / q) * q);
  return fmt == PW_BF16 ? (__float_as_uint(r) >> 16) : f16_rne(r);
}

__device__ __forceinline__ int apl_nearest16(const double (&c)[16], double x) {
  int jb = 0;
  double best = fabs(x - c[0]);
#pragma unroll
  for (int j = 1; j < 16; ++j) {
    const double d = fabs(x - c[j]);
    if (d < best) {
      best = d;
      jb = j;
    }
  }
  return jb;
}

// The whole row r of job J in one thread, in the oracle's order of steps
// (the reference form, used for rows whose sums could round).
template <int ACT>
__device__ void apl_quant_row_seq(const AplJob& J, int r, int R) {
#pragma clang fp contract(off)
  const int K = J.K;
  const uint16_t* v = J.src + static_cast<size_t>(r) * K;
  uint8_t* code = J.codes + static_cast<size_t>(r) * K;
  double* cent = reinterpret_cast<double*>(J.scratch + static_cast<size_t>(r) * kAplScratchRow);
  int* an = reinterpret_cast<int*>(cent + 496);
  double* as = reinterpret_cast<double*>(an + 256);
  double* pmin = as + 256;
  double* pmax = pmin + 128;
  const size_t rk8 = static_cast<size_t>(R) * K / 8;
  // 4-bit seed
  double lo = val16(v[0], ACT), hi = lo;
  for (int k = 1; k < K; ++k) {
    const double x = val16(v[k], ACT);
    lo = x < lo ? x : lo;
    hi = x > hi ? x : hi;
  }
  double c[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) c[j] = lo + (hi - lo) * ((2.0 * j + 1.0) / 32.0);
  for (int it = 0; it < 8; ++it) {
    double S[16];
    int N[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      S[j] = 0.0;
      N[j] = 0;
    }
    for (int k = 0; k < K; ++k) {
      const double x = val16(v[k], ACT);
      const int a = apl_nearest16(c, x);
#pragma unroll
      for (int j = 0; j < 16; ++j) {   // S never holds -0.0, so adding +0.0 leaves it unchanged
        S[j] += j == a ? x : 0.0;
        N[j] += j == a ? 1 : 0;
      }
    }
#pragma unroll
    for (int j = 0; j < 16; ++j)
      if (N[j] > 0) c[j] = S[j] / N[j];
  }
  for (int k = 0; k < K; ++k) code[k] = static_cast<uint8_t>(apl_nearest16(c, val16(v[k], ACT)));
  uint16_t* lut4 = reinterpret_cast<uint16_t*>(J.page + 4 * rk8) + static_cast<size_t>(r) * 16;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    cent[j] = c[j];
    lut4[j] = static_cast<uint16_t>(rne16_d(c[j], ACT));
  }
  if (J.bits != 8) {
    for (int k = 0; k < K; ++k) code[k] = static_cast<uint8_t>(code[k] << 4);
    return;
  }
  // one-bit splits to 8 bits
  double* cp = cent;          // parents (P of them)
  double* cc = cent + 16;     // children (2 P)
  for (int P = 16; P <= 128; P *= 2) {
    for (int p = 0; p < P; ++p) {
      an[p] = 0;
      as[p] = 0.0;
      pmin[p] = 0.0;
      pmax[p] = 0.0;
    }
    for (int k = 0; k < K; ++k) {
      const double x = val16(v[k], ACT);
      const int p = code[k];
      if (an[p] == 0) {
        pmin[p] = x;
        pmax[p] = x;
      } else {
        pmin[p] = x < pmin[p] ? x : pmin[p];
        pmax[p] = x > pmax[p] ? x : pmax[p];
      }
      an[p] += 1;
      as[p] += x;
    }
    for (int p = 0; p < P; ++p) {
      if (an[p] > 0) {
        const double m = as[p] / an[p];
        cc[2 * p] = (pmin[p] + m) / 2.0;
        cc[2 * p + 1] = (m + pmax[p]) / 2.0;
      } else {
        cc[2 * p] = cp[p];
        cc[2 * p + 1] = cp[p];
      }
    }
    for (int it = 0; it < 4; ++it) {
      for (int q = 0; q < 2 * P; ++q) {
        an[q] = 0;
        as[q] = 0.0;
      }
      for (int k = 0; k < K; ++k) {
        const double x = val16(v[k], ACT);
        const int p = code[k];
        const int ch = fabs(x - cc[2 * p + 1]) < fabs(x - cc[2 * p]) ? 1 : 0;
        an[2 * p + ch] += 1;
        as[2 * p + ch] += x;
      }
      for (int q = 0; q < 2 * P; ++q)
        if (an[q] > 0) cc[q] = as[q] / an[q];
    }
    for (int k = 0; k < K; ++k) {
      const double x = val16(v[k], ACT);
      const int p = code[k];
      code[k] = static_cast<uint8_t>(2 * p + (fabs(x - cc[2 * p + 1]) < fabs(x - cc[2 * p]) ? 1 : 0));
    }
    cp = cc;
    cc += 2 * P;
  }
  uint16_t* lut8 = reinterpret_cast<uint16_t*>(J.page + 8 * rk8 + 32 * static_cast<size_t>(R)) +
                   static_cast<size_t>(r) * 256;
  for (int j = 0; j < 256; ++j) lut8[j] = static_cast<uint16_t>(rne16_d(cp[j], ACT));
}

// ---------------------------------------------------------------------------
// The same quantizer with one 256-thread workgroup per row. Every float64 sum
// of the algorithm adds 16-bit values, which are integer multiples of the
// smallest value's unit (2^(e - 7) for bf16, 2^(e - 10) for fp16); when the
// row's largest magnitude times K stays within 2^53 of that unit, every
// partial sum of every subset is exact, so the sums come out bit-identical in
// any order: the workgroup accumulates them with LDS atomics. Minima and
// maxima do not depend on order either, and every other step (assignments,
// means, child centroids, LUT rounding) is per value or per cluster, so the
// row's codes and LUTs equal the one-thread form's bit for bit. A row that
// fails the bound (or has K > 16384) runs the one-thread form in thread 0.
// ---------------------------------------------------------------------------

constexpr int kAplThreads = 256;
constexpr int kAplPerThread = 64;                 // values per thread: K <= 16384

// Unit and magnitude exponents of a nonzero 16-bit value: x is a multiple of
// 2^unit and |x| < 2^(mag + 1). Non-finite values give mag = 4096 (no bound).
template <int ACT>
__device__ __forceinline__ void apl_exps(uint32_t h, int& unit, int& mag) {
  if constexpr (ACT == PW_BF16) {
    const int E = (h >> 7) & 0xFF;
    if (E == 0xFF) { unit = -4096; mag = 4096; return; }
    unit = E == 0 ? -133 : E - 134;
    mag = E == 0 ? -127 : E - 127;
  } else {
    const int E = (h >> 10) & 0x1F;
    if (E == 0x1F) { unit = -4096; mag = 4096; return; }
    unit = E == 0 ? -24 : E - 25;
    mag = E == 0 ? -15 : E - 15;
  }
}

// order-preserving 64-bit keys of doubles (for LDS integer min / max)
__device__ __forceinline__ unsigned long long apl_key(double x) {
  const unsigned long long u = static_cast<unsigned long long>(__double_as_longlong(x));
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}
__device__ __forceinline__ double apl_unkey(unsigned long long k) {
  const unsigned long long u = (k >> 63) ? (k & 0x7FFFFFFFFFFFFFFFull) : ~k;
  return __longlong_as_double(static_cast<long long>(u));
}

template <int ACT>
__global__ __launch_bounds__(kAplThreads) void k_apl_quant(const AplBatch b) {
#pragma clang fp contract(off)
  const uint32_t g = blockIdx.x;                   // the row of the batch
  if (g >= b.total_rows) return;
  int jb = 0;
  while (jb + 1 < b.n_jobs && b.job[jb + 1].row_base <= g) ++jb;
  const AplJob& J = b.job[jb];
  const int r = static_cast<int>(g - J.row_base), K = J.K, R = b.R, tid = threadIdx.x;
  __shared__ double s_sum[256];
  __shared__ int s_cnt[256];
  __shared__ unsigned long long s_min[128], s_max[128];
  __shared__ double s_cp[128], s_cc[256];
  __shared__ int s_unit, s_mag;
  const uint16_t* v = J.src + static_cast<size_t>(r) * K;
  const bool fits = K <= kAplThreads * kAplPerThread;
  // this thread's values k = tid + 256 i, held as 16-bit patterns
  uint32_t vh[kAplPerThread / 2];
  int umin = 4096, mmax = -4096;
  double lo = __builtin_inf(), hi = -__builtin_inf();
#pragma unroll
  for (int i = 0; i < kAplPerThread; ++i) {
    const int k = tid + kAplThreads * i;
    const uint32_t h = (fits && k < K) ? v[k] : 0u;
    if (i & 1) vh[i >> 1] |= h << 16;
    else vh[i >> 1] = h;
    if (fits && k < K) {
      const double x = val16(h, ACT);
      lo = x < lo ? x : lo;
      hi = x > hi ? x : hi;
      if ((h & 0x7FFFu) != 0u) {
        int u, m;
        apl_exps<ACT>(h, u, m);
        umin = min(umin, u);
        mmax = max(mmax, m);
      }
    }
  }
  if (tid == 0) {
    s_unit = 4096;
    s_mag = -4096;
    s_min[0] = ~0ull;
    s_max[0] = 0ull;
  }
  __syncthreads();
  atomicMin(&s_unit, umin);
  atomicMax(&s_mag, mmax);
  if (fits && tid < K) {
    atomicMin(&s_min[0], apl_key(lo));
    atomicMax(&s_max[0], apl_key(hi));
  }
  __syncthreads();
  int klog = 0;
  while ((1 << klog) < K) ++klog;
  // all values zero: every sum is +0.0, exact
  const bool exact = fits && (s_mag == -4096 || (s_mag + 1) - s_unit + klog <= 53);
  if (!exact) {
    if (tid == 0) apl_quant_row_seq<ACT>(J, r, R);
    return;
  }
  auto val = [&](int i) { return val16((vh[i >> 1] >> (16 * (i & 1))) & 0xFFFFu, ACT); };
  auto live = [&](int i) { return tid + kAplThreads * i < K; };
  lo = apl_unkey(s_min[0]);
  hi = apl_unkey(s_max[0]);
  // 4-bit seed: centroids in registers (every thread computes the same)
  double c[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) c[j] = lo + (hi - lo) * ((2.0 * j + 1.0) / 32.0);
  uint32_t cw[kAplPerThread / 4];                  // this thread's codes, 8 bits each
  for (int it = 0; it < 8; ++it) {
    double S[16];
    int N[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      S[j] = 0.0;
      N[j] = 0;
    }
#pragma unroll
    for (int i = 0; i < kAplPerThread; ++i) {
      if (!live(i)) continue;
      const double x = val(i);
      const int a = apl_nearest16(c, x);
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        S[j] += j == a ? x : 0.0;
        N[j] += j == a ? 1 : 0;
      }
    }
    if (tid < 16) {
      s_sum[tid] = 0.0;
      s_cnt[tid] = 0;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if (N[j] == 0) continue;
      atomicAdd(&s_sum[j], S[j]);
      atomicAdd(&s_cnt[j], N[j]);
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 16; ++j)
      if (s_cnt[j] > 0) c[j] = s_sum[j] / s_cnt[j];
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < kAplPerThread; ++i) {
    const uint32_t a = live(i) ? static_cast<uint32_t>(apl_nearest16(c, val(i))) : 0u;
    if ((i & 3) == 0) cw[i >> 2] = a;
    else cw[i >> 2] |= a << (8 * (i & 3));
  }
  auto code_of = [&](int i) { return static_cast<int>((cw[i >> 2] >> (8 * (i & 3))) & 0xFFu); };
  const size_t rk8 = static_cast<size_t>(R) * K / 8;
  uint16_t* lut4 = reinterpret_cast<uint16_t*>(J.page + 4 * rk8) + static_cast<size_t>(r) * 16;
  if (tid < 16) lut4[tid] = static_cast<uint16_t>(rne16_d(c[tid], ACT));
  uint8_t* code = J.codes + static_cast<size_t>(r) * K;
  if (J.bits != 8) {
#pragma unroll
    for (int i = 0; i < kAplPerThread; ++i)
      if (live(i)) code[tid + kAplThreads * i] = static_cast<uint8_t>(code_of(i) << 4);
    return;
  }
  if (tid < 16) s_cp[tid] = c[tid];
  // one-bit splits to 8 bits
  for (int P = 16; P <= 128; P *= 2) {
    if (tid < P) {
      s_cnt[tid] = 0;
      s_sum[tid] = 0.0;
      s_min[tid] = ~0ull;
      s_max[tid] = 0ull;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kAplPerThread; ++i) {
      if (!live(i)) continue;
      const double x = val(i);
      const int p = code_of(i);
      atomicAdd(&s_cnt[p], 1);
      atomicAdd(&s_sum[p], x);
      atomicMin(&s_min[p], apl_key(x));
      atomicMax(&s_max[p], apl_key(x));
    }
    __syncthreads();
    if (tid < P) {
      const int n = s_cnt[tid];
      if (n > 0) {
        const double m = s_sum[tid] / n;
        s_cc[2 * tid] = (apl_unkey(s_min[tid]) + m) / 2.0;
        s_cc[2 * tid + 1] = (m + apl_unkey(s_max[tid])) / 2.0;
      } else {
        s_cc[2 * tid] = s_cp[tid];
        s_cc[2 * tid + 1] = s_cp[tid];
      }
    }
    __syncthreads();
    for (int it = 0; it < 4; ++it) {
      s_cnt[tid] = 0;                              // 2P <= 256 children
      s_sum[tid] = 0.0;
      __syncthreads();
#pragma unroll
      for (int i = 0; i < kAplPerThread; ++i) {
        if (!live(i)) continue;
        const double x = val(i);
        const int p = code_of(i);
        const int q = 2 * p + (fabs(x - s_cc[2 * p + 1]) < fabs(x - s_cc[2 * p]) ? 1 : 0);
        atomicAdd(&s_cnt[q], 1);
        atomicAdd(&s_sum[q], x);
      }
      __syncthreads();
      if (tid < 2 * P && s_cnt[tid] > 0) s_cc[tid] = s_sum[tid] / s_cnt[tid];
      __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < kAplPerThread; ++i) {
      if (!live(i)) continue;
      const double x = val(i);
      const int p = code_of(i);
      const uint32_t q = static_cast<uint32_t>(2 * p + (fabs(x - s_cc[2 * p + 1]) < fabs(x - s_cc[2 * p]) ? 1 : 0));
      cw[i >> 2] = (cw[i >> 2] & ~(0xFFu << (8 * (i & 3)))) | (q << (8 * (i & 3)));
    }
    if (tid < 2 * P && P < 128) s_cp[tid] = s_cc[tid];
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < kAplPerThread; ++i)
    if (live(i)) code[tid + kAplThreads * i] = static_cast<uint8_t>(code_of(i));
  uint16_t* lut8 = reinterpret_cast<uint16_t*>(J.page + 8 * rk8 + 32 * static_cast<size_t>(R)) +
                   static_cast<size_t>(r) * 256;
  lut8[tid] = static_cast<uint16_t>(rne16_d(s_cc[tid], ACT));
}

// One thread per (job, plane, tile, lane) word: bit 8 i + q of lane l's word
// is plane j's bit of row 16 rt + l mod 16, column 128 kb + 32 i + 8 (l / 16) + q.
__global__ __launch_bounds__(256) void k_apl_pack(const AplBatch b) {
  const uint32_t g = blockIdx.x * 256u + threadIdx.x;
  // job of this word: the batch's words are laid out job after job
  uint32_t base = 0;
  int jb = -1;
  uint32_t words = 0;
  for (int j = 0; j < b.n_jobs; ++j) {
    words = static_cast<uint32_t>(b.job[j].bits) * (b.R / 16) * (b.job[j].K / 128) * 64;
    if (g < base + words) {
      jb = j;
      break;
    }
    base += words;
  }
  if (jb < 0) return;
  const AplJob& J = b.job[jb];
  const uint32_t w = g - base;
  const int nkb = J.K / 128;
  const uint32_t per_plane = static_cast<uint32_t>(b.R / 16) * nkb * 64;
  const int plane = static_cast<int>(w / per_plane);
  const uint32_t rest = w % per_plane;
  const int t = static_cast<int>(rest / 64), lane = static_cast<int>(rest % 64);
  const int rt = t / nkb, kb = t % nkb;
  const int row = 16 * rt + (lane & 15);
  const uint8_t* cr = J.codes + static_cast<size_t>(row) * J.K + 128 * kb + 8 * (lane >> 4);
  uint32_t word = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int q = 0; q < 8; ++q) word |= static_cast<uint32_t>((cr[32 * i + q] >> (7 - plane)) & 1u) << (8 * i + q);
  const size_t rk8 = static_cast<size_t>(b.R) * J.K / 8;
  const size_t pbase = plane < 4 ? plane * rk8 : 4 * rk8 + 32 * static_cast<size_t>(b.R) + (plane - 4) * rk8;
  reinterpret_cast<uint32_t*>(J.page + pbase)[static_cast<size_t>(t) * 64 + lane] = word;
}

}  // namespace

namespace {

// ---------------------------------------------------------------------------
// Routing statistics for the planner (Eq. 1's numerator and the routed-input
// features of Sec. 3.2), in float64 with a fixed summation order.
// ---------------------------------------------------------------------------

// One wave per row: squared Euclidean norm of a 16-bit row. Lane l sums the
// values l * 8 .. + 8 of every 512-value span in order, then a butterfly.
template <int ACT>
__global__ __launch_bounds__(256) void k_row_norm2(const uint16_t* rows, int n_rows, int dim, double* out) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= n_rows) return;
  const uint16_t* r = rows + static_cast<size_t>(row) * dim;
  double acc = 0.0;
  for (int k = lane * 8; k < dim; k += 512) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(r + k);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const double a = val16(v[q] & 0xFFFFu, ACT), b = val16(v[q] >> 16, ACT);
      acc += a * a;   // exact products of 16-bit values
      acc += b * b;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  if (lane == 0) out[row] = acc;
}

// One workgroup per expert: thread j takes the expert's slots j, j + 256, ...
// in order, then a fixed tree over the 256 partial sums.
__global__ __launch_bounds__(256) void k_expert_stats(const double* norm2, int by_position, const float* topk_w,
                                                      const int32_t* offsets, const int32_t* sorted_slot, int S,
                                                      int K, int n_rows, double* stats, int accumulate) {
  __shared__ double red[5][256];
  const int e = blockIdx.x, tid = threadIdx.x;
  const int o = clampi(offsets[e], 0, S);
  const int n = clampi(offsets[e + 1], o, S) - o;
  double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0, a4 = 0.0;
  for (int i = tid; i < n; i += 256) {
    const int slot = clampi(sorted_slot[o + i], 0, S - 1);
    const int row = clampi(by_position ? o + i : slot / K, 0, n_rows - 1);
    const double r = topk_w[slot];
    const double n2 = norm2[row];
    const double nn = sqrt(n2);
    a0 += r;
    a1 += 1.0;
    a2 += r * nn;
    a3 += r * n2;
    a4 = fmax(a4, nn);
  }
  red[0][tid] = a0;
  red[1][tid] = a1;
  red[2][tid] = a2;
  red[3][tid] = a3;
  red[4][tid] = a4;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (tid < s) {
#pragma unroll
      for (int c = 0; c < 4; ++c) red[c][tid] += red[c][tid + s];
      red[4][tid] = fmax(red[4][tid], red[4][tid + s]);
    }
    __syncthreads();
  }
  if (tid < 5) {
    const double v = red[tid][0];
    double* d = stats + 5 * static_cast<size_t>(e) + tid;
    *d = !accumulate ? v : tid == 4 ? fmax(*d, v) : *d + v;
  }
}

}  // namespace

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------

hipError_t launch_route_topk(const float* logits, int T, int E, int K, int renorm, int n_shared,
                             const float* shared_gate, int32_t* ids, float* w, hipStream_t st) {
  if (T <= 0) return hipSuccess;
  if (K > kMaxTopK || E > 64 * kRouteLogitsPerLane) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_route_topk, dim3((T + 3) / 4), dim3(256), 0, st, logits, T, E, K, renorm, n_shared,
                     shared_gate, ids, w);
  return hipGetLastError();
}

// The single-workgroup path's serial selection and per-expert prefixes grow
// with the expert count: measured at 4.9 us against about 6 us for the two
// launches with 8 experts and 64 tokens, but 29.5 us with 60 experts and 128
// tokens, so it serves layers of at most kFusedMaxExperts experts.
constexpr int kFusedMaxExperts = 32;

bool route_permute_fits(int T, int E, int K, int n_shared) {
  return T >= 1 && T * (K + n_shared) <= kFusedMaxSlots && T * E <= kFusedMaxLogits &&
         E + n_shared <= kFusedMaxExperts && K <= kMaxTopK;
}

hipError_t launch_route_permute(const float* logits, int T, int E, int K, int renorm, int n_shared,
                                const float* shared_gate, int32_t* ids, float* w, int32_t* offsets,
                                int32_t* sorted_slot, int32_t* slot_pos, hipStream_t st) {
  if (!route_permute_fits(T, E, K, n_shared)) return hipErrorInvalidValue;
  const dim3 g(1), b(kFusedThreads);
  if (K <= 2)
    hipLaunchKernelGGL(k_route_permute<2>, g, b, 0, st, logits, T, E, K, renorm, n_shared, shared_gate, ids, w,
                       offsets, sorted_slot, slot_pos);
  else if (K <= 4)
    hipLaunchKernelGGL(k_route_permute<4>, g, b, 0, st, logits, T, E, K, renorm, n_shared, shared_gate, ids, w,
                       offsets, sorted_slot, slot_pos);
  else if (K <= 8)
    hipLaunchKernelGGL(k_route_permute<8>, g, b, 0, st, logits, T, E, K, renorm, n_shared, shared_gate, ids, w,
                       offsets, sorted_slot, slot_pos);
  else
    hipLaunchKernelGGL(k_route_permute<16>, g, b, 0, st, logits, T, E, K, renorm, n_shared, shared_gate, ids, w,
                       offsets, sorted_slot, slot_pos);
  return hipGetLastError();
}

hipError_t launch_permute(const int32_t* ids, int T, int K, int E, int32_t* offsets,
                          int32_t* sorted_slot, int32_t* slot_pos, hipStream_t st) {
  hipLaunchKernelGGL(k_permute, dim3(E), dim3(kPermThreads), 0, st, ids, T * K, E, offsets,
                     sorted_slot, slot_pos);
  return hipGetLastError();
}

template <int ACT, int SDT>
static void qjobs_go(const QJobBatch& b, hipStream_t st) {
  const dim3 grid((b.total_items + 3) / 4), block(256);
  if (b.G == 64) hipLaunchKernelGGL((k_qjobs<ACT, SDT, kQG64>), grid, block, 0, st, b);
  else if (b.G == 128) hipLaunchKernelGGL((k_qjobs_g128<ACT, SDT>), grid, block, 0, st, b);
  else hipLaunchKernelGGL((k_qjobs<ACT, SDT, kQGBig>), grid, block, 0, st, b);
}

hipError_t launch_qjobs(const QJobBatch& b, hipStream_t st) {
  if (b.total_items == 0) return hipSuccess;
  if (b.act == PW_BF16) {
    if (b.sdt == PW_BF16) qjobs_go<PW_BF16, PW_BF16>(b, st);
    else qjobs_go<PW_BF16, PW_F16>(b, st);
  } else {
    if (b.sdt == PW_BF16) qjobs_go<PW_F16, PW_BF16>(b, st);
    else qjobs_go<PW_F16, PW_F16>(b, st);
  }
  return hipGetLastError();
}

template <int ACT, int SDT, int GK>
static void requant_go(const RqBatch& b, int src_bits, int dst_bits, dim3 grid, hipStream_t st) {
  const dim3 block(256);
  if (src_bits == 16 && dst_bits == 8)
    hipLaunchKernelGGL((k_requant<ACT, SDT, GK, 16, 8>), grid, block, 0, st, b);
  else if (src_bits == 16)
    hipLaunchKernelGGL((k_requant<ACT, SDT, GK, 16, 4>), grid, block, 0, st, b);
  else
    hipLaunchKernelGGL((k_requant<ACT, SDT, GK, 8, 4>), grid, block, 0, st, b);
}

template <int ACT, int SDT>
static void requant_g(const RqBatch& b, int src_bits, int dst_bits, dim3 grid, hipStream_t st) {
  if (b.G == 64) requant_go<ACT, SDT, kQG64>(b, src_bits, dst_bits, grid, st);
  else if (b.G == 128) requant_go<ACT, SDT, kQG128>(b, src_bits, dst_bits, grid, st);
  else requant_go<ACT, SDT, kQGBig>(b, src_bits, dst_bits, grid, st);
}

hipError_t launch_requant(const RqBatch& b, int src_bits, int dst_bits, int act, int sdt, hipStream_t st) {
  if (b.n_jobs == 0) return hipSuccess;
  const bool pair_ok = (src_bits == 16 && (dst_bits == 8 || dst_bits == 4)) || (src_bits == 8 && dst_bits == 4);
  if (!pair_ok || b.n_jobs < 0 || b.n_jobs > kMaxRqJobs || b.R <= 0 || b.R % 16 != 0 ||
      (b.G != 64 && b.G != 128 && b.G != 256 && b.G != 512))
    return hipErrorInvalidValue;
  const int span = b.G > 128 ? b.G / 128 : 1;
  uint32_t max_spans = 0;
  for (int j = 0; j < b.n_jobs; ++j) {
    const uint32_t kb = ((b.kbit[j >> 5] >> (j & 31)) & 1u) ? b.kb[1] : b.kb[0];
    if (kb == 0 || kb % span != 0) return hipErrorInvalidValue;
    max_spans = std::max<uint32_t>(max_spans, kb / span);
  }
  const dim3 grid((max_spans + 3) / 4, b.R / 16, b.n_jobs);
  if (act == PW_BF16) {
    if (sdt == PW_BF16) requant_g<PW_BF16, PW_BF16>(b, src_bits, dst_bits, grid, st);
    else requant_g<PW_BF16, PW_F16>(b, src_bits, dst_bits, grid, st);
  } else {
    if (sdt == PW_BF16) requant_g<PW_F16, PW_BF16>(b, src_bits, dst_bits, grid, st);
    else requant_g<PW_F16, PW_F16>(b, src_bits, dst_bits, grid, st);
  }
  return hipGetLastError();
}

hipError_t launch_entry_writes(pw_page_entry* table, const EntryWrites& w, hipStream_t st) {
  if (w.n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_entry_writes, dim3(1), dim3(kMaxEntryWrites), 0, st, table, w);
  return hipGetLastError();
}

hipError_t launch_clear_table(pw_page_entry* table, size_t n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  const unsigned blocks = static_cast<unsigned>(std::min<size_t>((n + 255) / 256, 1024));
  hipLaunchKernelGGL(k_clear_table, dim3(blocks), dim3(256), 0, st, table, n);
  return hipGetLastError();
}

hipError_t launch_combine(const GemmArgs& a, hipStream_t st) {
  if (a.T <= 0) return hipSuccess;
  const int nmax = a.n_shared > 0 && a.nsplit_sh > a.nsplit ? a.nsplit_sh : a.nsplit;
  if (nmax < 1 || nmax > 8) return hipErrorInvalidValue;
  const int nsp = nmax == 1 ? 1 : nmax == 2 ? 2 : nmax <= 4 ? 4 : 8;
  const int cols = std::min(a.topk <= 2 ? 2 : a.topk <= 4 ? 4 : a.topk <= 6 ? 6 : 8, 16 / nsp);
  const dim3 grid(a.T, (a.H / 4 + 255) / 256), block(256);
  switch (nsp * 16 + cols) {
    case 16 + 2: hipLaunchKernelGGL((k_combine<1, 2>), grid, block, 0, st, a); break;
    case 16 + 4: hipLaunchKernelGGL((k_combine<1, 4>), grid, block, 0, st, a); break;
    case 16 + 6: hipLaunchKernelGGL((k_combine<1, 6>), grid, block, 0, st, a); break;
    case 16 + 8: hipLaunchKernelGGL((k_combine<1, 8>), grid, block, 0, st, a); break;
    case 32 + 2: hipLaunchKernelGGL((k_combine<2, 2>), grid, block, 0, st, a); break;
    case 32 + 4: hipLaunchKernelGGL((k_combine<2, 4>), grid, block, 0, st, a); break;
    case 32 + 6: hipLaunchKernelGGL((k_combine<2, 6>), grid, block, 0, st, a); break;
    case 32 + 8: hipLaunchKernelGGL((k_combine<2, 8>), grid, block, 0, st, a); break;
    case 64 + 2: hipLaunchKernelGGL((k_combine<4, 2>), grid, block, 0, st, a); break;
    case 64 + 4: hipLaunchKernelGGL((k_combine<4, 4>), grid, block, 0, st, a); break;
    default: hipLaunchKernelGGL((k_combine<8, 2>), grid, block, 0, st, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_apl_quant(const AplBatch& b, hipStream_t st) {
  if (b.total_rows == 0) return hipSuccess;
  const dim3 grid(b.total_rows), block(kAplThreads);   // one workgroup per row
  if (b.act == PW_BF16)
    hipLaunchKernelGGL(k_apl_quant<PW_BF16>, grid, block, 0, st, b);
  else
    hipLaunchKernelGGL(k_apl_quant<PW_F16>, grid, block, 0, st, b);
  return hipGetLastError();
}

hipError_t launch_apl_pack(const AplBatch& b, hipStream_t st) {
  uint64_t words = 0;
  for (int j = 0; j < b.n_jobs; ++j)
    words += static_cast<uint64_t>(b.job[j].bits) * (b.R / 16) * (b.job[j].K / 128) * 64;
  if (words == 0) return hipSuccess;
  hipLaunchKernelGGL(k_apl_pack, dim3(static_cast<unsigned>((words + 255) / 256)), dim3(256), 0, st, b);
  return hipGetLastError();
}

hipError_t launch_routing_stats(const uint16_t* rows, int act, int n_rows, int dim, int by_position,
                                const float* topk_w, const int32_t* offsets, const int32_t* sorted_slot, int S,
                                int E, int K, double* norm2, double* stats, int accumulate, hipStream_t st) {
  if (n_rows > 0) {
    const dim3 grid((n_rows + 3) / 4);
    if (act == PW_BF16)
      hipLaunchKernelGGL(k_row_norm2<PW_BF16>, grid, dim3(256), 0, st, rows, n_rows, dim, norm2);
    else
      hipLaunchKernelGGL(k_row_norm2<PW_F16>, grid, dim3(256), 0, st, rows, n_rows, dim, norm2);
  }
  hipLaunchKernelGGL(k_expert_stats, dim3(E), dim3(256), 0, st, norm2, by_position, topk_w, offsets, sorted_slot, S,
                     K, n_rows, stats, accumulate);
  return hipGetLastError();
}

}  // namespace pw
