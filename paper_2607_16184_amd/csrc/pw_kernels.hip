// HIP kernels for gfx950 (CDNA4): router, token permutation, group-wise RTN
// quantize / requantize, the decode-size paged gate/up and down GEMMs and the
// combine. (The streaming and LDS-tiled GEMMs for larger batches are in
// pw_tgemm.hip.)
//
// GEMM layout. Each wave computes D[n][m] = sum_k W[n][k] * X[m][k] for 16
// weight rows n (the MFMA A operand) and 16 routed slots m (the B operand)
// with v_mfma_f32_16x16x32_{bf16,f16}. K is walked in blocks of 128; a block
// is four MFMA k-steps, and in k-step i lane group j (lanes 16j..16j+15)
// supplies k = 32i + 8j .. 32i + 8j + 7 of both operands. The page format
// stores a 16-row x 128-value tile in exactly this lane order (16 contiguous
// bytes per lane and k-step for 16-bit values), so every weight fragment is
// one or more 16-byte loads per lane of a contiguous 1 KB row.
//
// Quantized pages run in the code domain: the A operand is the code c itself
// as an exact 16-bit float (int8 codes through an exact conversion; int4
// codes, and int8 codes with fp16 activations, OR-ed into the mantissa of a
// constant OFF, giving OFF + c exactly). Per group of G along K the MFMA gives
// P = sum (c + OFF) x, and X = sum x comes from sums taken while the
// activations are staged; the group's scale s and zero z are then applied in
// fp32 on the accumulator: acc += s * P + (z - OFF * s) * X, which is
// sum (z + c s) x. Weights are never rounded: z + c*s enters exactly.
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

// One wave per token: lane l holds logits l, l + 64, ...; K rounds of a
// wave-wide arg-max in (value descending, index ascending) order take the
// next expert each. The weights use the same fp32 arithmetic as a serial
// loop: m = the largest selected logit, a_k = exp(l_k - m), w_k = a_k / sum,
// with the sum taken in k order (renorm) or in expert order over all E.
__global__ __launch_bounds__(256) void k_route_topk(const float* __restrict__ logits, int T, int E,
                                                    int K, int renorm, int32_t* __restrict__ ids,
                                                    float* __restrict__ w) {
  const int t = blockIdx.x * 4 + static_cast<int>(threadIdx.x >> 6);
  if (t >= T) return;   // wave-uniform
  const int lane = lane_id();
  const float* l = logits + static_cast<size_t>(t) * E;
  float v[kRouteLogitsPerLane];
  bool live[kRouteLogitsPerLane];
#pragma unroll
  for (int q = 0; q < kRouteLogitsPerLane; ++q) {
    const int e = lane + 64 * q;
    live[q] = e < E;
    v[q] = live[q] ? l[e] : 0.0f;
  }
  float sv[kMaxTopK];
  int se[kMaxTopK];
#pragma unroll
  for (int k = 0; k < kMaxTopK; ++k) {
    if (k < K) {
      float bv = 0.0f;
      int be = 0x7fffffff;
#pragma unroll
      for (int q = 0; q < kRouteLogitsPerLane; ++q) {
        const int e = lane + 64 * q;
        if (live[q] && (be == 0x7fffffff || v[q] > bv || (v[q] == bv && e < be))) {
          bv = v[q];
          be = e;
        }
      }
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) {
        const float ov = __shfl_xor(bv, off);
        const int oe = __shfl_xor(be, off);
        if (oe != 0x7fffffff && (be == 0x7fffffff || ov > bv || (ov == bv && oe < be))) {
          bv = ov;
          be = oe;
        }
      }
      sv[k] = bv;
      se[k] = be;
#pragma unroll
      for (int q = 0; q < kRouteLogitsPerLane; ++q)
        if (lane + 64 * q == be) live[q] = false;
    }
  }
  if (lane != 0) return;
  const float m = sv[0];
  float sum = 0.0f;
  if (renorm) {
    for (int k = 0; k < K; ++k) sum += expf(sv[k] - m);
  } else {
    for (int e = 0; e < E; ++e) sum += expf(l[e] - m);
  }
#pragma unroll
  for (int k = 0; k < kMaxTopK; ++k) {
    if (k < K) {
      ids[static_cast<size_t>(t) * K + k] = se[k];
      w[static_cast<size_t>(t) * K + k] = expf(sv[k] - m) / sum;
    }
  }
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
  for (int s = tid; s < S; s += kPermThreads) {
    const int id = ids[s];
    if (id >= 0 && id < E) atomicAdd(&cnt[id], 1);
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

// ---------------------------------------------------------------------------
// Group-wise RTN quantize / requantize / 16-bit layout transform.
//
// Page layout: tiles of 16 rows x 128 values stored tile after tile (row tile
// major); inside a tile, lane l = 16 lg + lc (row lc, k-run lg) of k-step i
// owns 16 contiguous bytes: 16-bit values at 1024 i + 16 l, 8-bit codes of
// steps 2u, 2u+1 at 1024 u + 16 l, the four 4-bit words at 16 l. A wave reads
// or writes a tile as contiguous 1 KB rows. One wave handles one row tile over
// one span of K (max(G,128) values); groups are reduced over the lane groups.
// ---------------------------------------------------------------------------


// The raw 16-byte pieces lane l holds of one 128-value block of a row tile,
// for every source format (16-bit: four pieces; 8-bit: two; 4-bit: one), plus
// the (scale, zero) word of each k-step's group for quantized sources.
struct QRaw {
  u32x4 w[4];
  uint32_t sz[4];
};

__device__ __forceinline__ void q_load(const QJob& job, const QJobBatch& b, int tau, int blk, QRaw& raw) {
  const int lane = lane_id(), lc = lane & 15, lg = lane >> 4;
  const int K = b.K, nkb = K / 128;
  const size_t tile = static_cast<size_t>(tau) * nkb + blk;
  if (job.src_bits == 16) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint8_t* src = job.src_plain
          ? job.src + (static_cast<size_t>(tau * 16 + lc) * K + blk * 128 + 32 * i + 8 * lg) * 2
          : job.src + tile * 4096 + 1024 * i + 16 * lane;
      raw.w[i] = *reinterpret_cast<const u32x4*>(src);
    }
    return;
  }
  if (job.src_bits == 8) {
#pragma unroll
    for (int u = 0; u < 2; ++u) raw.w[u] = *reinterpret_cast<const u32x4*>(job.src + tile * 2048 + 1024 * u + 16 * lane);
  } else {
    raw.w[0] = *reinterpret_cast<const u32x4*>(job.src + tile * 1024 + 16 * lane);
  }
  const int r = tau * 16 + lc;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int g = (blk * 128 + 32 * i) / b.G;
    raw.sz[i] = *reinterpret_cast<const uint32_t*>(job.src_sz + (static_cast<size_t>(g) * b.R + r) * 4);
  }
}

// The 32 values (k-steps i = 0..3, 8 values each) lane l holds of the block,
// widened to fp32: 16-bit values, or quantized codes dequantized as
// fl32(z + c s) (c s is exact in fp32).
__device__ __forceinline__ void q_widen(const QJob& job, const QJobBatch& b, const QRaw& raw, float (&v)[32]) {
  if (job.src_bits == 16) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v[8 * i + 2 * q] = val16(raw.w[i][q], b.act);
        v[8 * i + 2 * q + 1] = val16(raw.w[i][q] >> 16, b.act);
      }
    return;
  }
  uint32_t c[32];
  if (job.src_bits == 8) {
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int w = 0; w < 4; ++w)
#pragma unroll
        for (int q = 0; q < 4; ++q) c[16 * u + 4 * w + q] = (raw.w[u][w] >> (8 * q)) & 0xFFu;
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        c[8 * i + 2 * t] = (raw.w[0][i] >> (4 * t)) & 15u;
        c[8 * i + 2 * t + 1] = (raw.w[0][i] >> (16 + 4 * t)) & 15u;
      }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float s = val16(raw.sz[i], b.sdt), z = val16(raw.sz[i] >> 16, b.sdt);
#pragma unroll
    for (int q = 0; q < 8; ++q) v[8 * i + q] = z + static_cast<float>(c[8 * i + q]) * s;   // c*s exact
  }
}

__device__ __forceinline__ void q_read(const QJob& job, const QJobBatch& b, int tau, int blk, float (&v)[32]) {
  QRaw raw;
  q_load(job, b, tau, blk, raw);
  q_widen(job, b, raw, v);
}

// (scale, zero) bit patterns of a group from its extremes (the quantizer's steps).
__device__ __forceinline__ void q_params(float lo, float hi, int Q, int sdt, uint32_t* sb, uint32_t* zb) {
  *zb = round_down16(lo, sdt);
  const float z = val16(*zb, sdt);
  const float r = hi - z;
  *sb = 0u;
  if (r == 0.0f) return;
  *sb = round_up16(r / static_cast<float>(Q), sdt);
  if (val16(*sb, sdt) * static_cast<float>(Q) < r) *sb += 1u;   // s > 0: next value up
}

__device__ __forceinline__ uint32_t q_code(float v, uint32_t sb, uint32_t zb, int Q, int sdt) {
  if (sb == 0u) return 0u;
  const float d = v - val16(zb, sdt);
  const float c = rintf(d / val16(sb, sdt));
  return static_cast<uint32_t>(fminf(fmaxf(c, 0.0f), static_cast<float>(Q)));
}

// Codes of one block from its values and its group parameters, stored in the
// destination page's tile layout; the (scale, zero) words are written by the
// caller. Group g0 covers k-steps 0-3 (G >= 128) or 0-1 and g1 2-3 (G = 64).
__device__ __forceinline__ void q_store_codes(const QJob& job, const QJobBatch& b, int tau, int blk,
                                              const float (&v)[32], uint32_t sb0, uint32_t zb0, uint32_t sb1,
                                              uint32_t zb1, int Q) {
  const int lane = lane_id();
  uint32_t c[32];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const bool second = b.G == 64 && i >= 2;
#pragma unroll
    for (int q = 0; q < 8; ++q) c[8 * i + q] = q_code(v[8 * i + q], second ? sb1 : sb0, second ? zb1 : zb0, Q, b.sdt);
  }
  const size_t tile = static_cast<size_t>(tau) * (b.K / 128) + blk;
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

// Extremes of the block's group(s) across the row's four lane groups.
__device__ __forceinline__ void q_extremes(const float (&v)[32], int G, float& lo0, float& hi0, float& lo1,
                                           float& hi1) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      if (G == 64 && i >= 2) {
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

// One wave per item: a 16-row tile over NB consecutive 128-blocks (G <= 128),
// or over one span of G values (G > 128, NB = 1). With G <= 128 every group
// lies inside one block, so all NB blocks are loaded first (their loads in
// flight together) and each block is quantized from registers in one pass.
template <int NB>
__global__ __launch_bounds__(256) void k_qjobs(const QJobBatch b) {
  const uint32_t item = blockIdx.x * 4u + (threadIdx.x >> 6);
  if (item >= b.total_items) return;
  const int lane = lane_id(), lc = lane & 15, lg = lane >> 4;
  const int K = b.K, R = b.R, G = b.G, nkb = K / 128;
  const int span = G > 128 ? G / 128 : 1;          // blocks per group
  const int nsp = nkb / (span * NB);
  const int j = static_cast<int>(item / b.items_per_job);
  const int rem = static_cast<int>(item % b.items_per_job);
  const int tau = rem / nsp, sp = rem % nsp;
  const QJob& job = b.job[j];
  const int r = tau * 16 + lc;
  const int Q = (1 << job.dst_bits) - 1;
  float v[32];
  if (span == 1) {
    QRaw raw[NB];
#pragma unroll
    for (int n = 0; n < NB; ++n) q_load(job, b, tau, sp * NB + n, raw[n]);
#pragma unroll
    for (int n = 0; n < NB; ++n) {
      const int blk = sp * NB + n;
      q_widen(job, b, raw[n], v);
      if (job.dst_bits == 16) {      // layout transform of a 16-bit page
        const size_t tile = static_cast<size_t>(tau) * nkb + blk;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          u32x4 o;
#pragma unroll
          for (int q = 0; q < 4; ++q)
            o[q] = rne16(v[8 * i + 2 * q], b.act) | (rne16(v[8 * i + 2 * q + 1], b.act) << 16);
          *reinterpret_cast<u32x4*>(job.dst + tile * 4096 + 1024 * i + 16 * lane) = o;
        }
        continue;
      }
      float lo0 = __builtin_inff(), hi0 = -__builtin_inff(), lo1 = lo0, hi1 = hi0;
      q_extremes(v, G, lo0, hi0, lo1, hi1);
      q_rowreduce(lo0, hi0, lo1, hi1);
      uint32_t sb0, zb0, sb1 = 0u, zb1 = 0u;
      q_params(lo0, hi0, Q, b.sdt, &sb0, &zb0);
      if (G == 64) q_params(lo1, hi1, Q, b.sdt, &sb1, &zb1);
      q_store_codes(job, b, tau, blk, v, sb0, zb0, sb1, zb1, Q);
      if (lg == 0) {
        const int g0 = G == 64 ? 2 * blk : blk;
        *reinterpret_cast<uint32_t*>(job.dst_sz + (static_cast<size_t>(g0) * R + r) * 4) = sb0 | (zb0 << 16);
        if (G == 64)
          *reinterpret_cast<uint32_t*>(job.dst_sz + (static_cast<size_t>(g0 + 1) * R + r) * 4) = sb1 | (zb1 << 16);
      }
    }
    return;
  }
  // G > 128: one group spans several blocks; pass 1 finds its extremes, pass 2
  // re-reads the blocks for the codes
  if (job.dst_bits == 16) {
    for (int blk = sp * span; blk < (sp + 1) * span; ++blk) {
      q_read(job, b, tau, blk, v);
      const size_t tile = static_cast<size_t>(tau) * nkb + blk;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        u32x4 o;
#pragma unroll
        for (int q = 0; q < 4; ++q) o[q] = rne16(v[8 * i + 2 * q], b.act) | (rne16(v[8 * i + 2 * q + 1], b.act) << 16);
        *reinterpret_cast<u32x4*>(job.dst + tile * 4096 + 1024 * i + 16 * lane) = o;
      }
    }
    return;
  }
  float lo0 = __builtin_inff(), hi0 = -__builtin_inff(), lo1 = lo0, hi1 = hi0;
  for (int blk = sp * span; blk < (sp + 1) * span; ++blk) {
    q_read(job, b, tau, blk, v);
    q_extremes(v, G, lo0, hi0, lo1, hi1);
  }
  q_rowreduce(lo0, hi0, lo1, hi1);
  uint32_t sb0, zb0;
  q_params(lo0, hi0, Q, b.sdt, &sb0, &zb0);
  for (int blk = sp * span; blk < (sp + 1) * span; ++blk) {
    q_read(job, b, tau, blk, v);
    q_store_codes(job, b, tau, blk, v, sb0, zb0, 0u, 0u, Q);
  }
  if (lg == 0) *reinterpret_cast<uint32_t*>(job.dst_sz + (static_cast<size_t>(sp) * R + r) * 4) = sb0 | (zb0 << 16);
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
// Paged GEMM building blocks
// ---------------------------------------------------------------------------

// Code-domain offset of a page format (see the file comment).
template <int ACT, int B>
struct CodeOff {
  static constexpr float value = (B == 16) ? 0.0f : (ACT == PW_BF16 ? (B == 4 ? 128.0f : 0.0f) : 1024.0f);
};

template <int B> struct WF;
template <> struct WF<16> { u32x4 v[4]; };
template <> struct WF<8> { u32x4 v[2]; };
template <> struct WF<4> { u32x4 v[1]; };

// The lane's 16-byte pieces of 128-block blk of its row tile; `tile0` is the
// tile row's first tile plus 16 * lane.
template <int B>
__device__ __forceinline__ void wf_load(WF<B>& f, const uint8_t* tile0, int blk) {
  const uint8_t* p = tile0 + static_cast<size_t>(blk) * tile_bytes<B>();
#pragma unroll
  for (int i = 0; i < tile_bytes<B>() / 1024; ++i) f.v[i] = ld16_nt(p + 1024 * i);
}

// A operand of k-step i: eight 16-bit values (weights, or codes as floats).
template <int ACT, int B>
__device__ __forceinline__ u32x4 wf_op(const WF<B>& f, int i) {
  if constexpr (B == 16) {
    return f.v[i];
  } else if constexpr (B == 8) {
    const uint32_t d0 = f.v[i >> 1][(i & 1) * 2], d1 = f.v[i >> 1][(i & 1) * 2 + 1];
    u32x4 o;
    if constexpr (ACT == PW_BF16) {
      // bytes -> exact fp32 -> upper halves are the exact bf16 values
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const uint32_t d = q ? d1 : d0;
        const float c0 = static_cast<float>(d & 0xFFu), c1 = static_cast<float>((d >> 8) & 0xFFu);
        const float c2 = static_cast<float>((d >> 16) & 0xFFu), c3 = static_cast<float>(d >> 24);
        o[2 * q] = __builtin_amdgcn_perm(__float_as_uint(c1), __float_as_uint(c0), 0x07060302u);
        o[2 * q + 1] = __builtin_amdgcn_perm(__float_as_uint(c3), __float_as_uint(c2), 0x07060302u);
      }
    } else {
      // 0x64 high byte: fp16 1024 + c
      o[0] = __builtin_amdgcn_perm(0x64646464u, d0, 0x05010400u);
      o[1] = __builtin_amdgcn_perm(0x64646464u, d0, 0x05030402u);
      o[2] = __builtin_amdgcn_perm(0x64646464u, d1, 0x05010400u);
      o[3] = __builtin_amdgcn_perm(0x64646464u, d1, 0x05030402u);
    }
    return o;
  } else {
    const uint32_t w = f.v[0][i];
    const uint32_t magic = ACT == PW_BF16 ? 0x43004300u : 0x64006400u;   // 128 / 1024
    u32x4 o;
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q] = ((w >> (4 * q)) & 0x000F000Fu) | magic;
    return o;
  }
}

// acc += s * P + (z - OFF s) * X for the lane's four rows; P is cleared.
// X[t] is the group's activation sum for this lane's slot (tile t).
template <int ACT, int B, int NT>
__device__ __forceinline__ void group_fix(f32x4 (&acc)[NT], f32x4 (&p)[NT], const float (&xs)[NT], u32x4 sz,
                                          int sdt) {
  constexpr float off = CodeOff<ACT, B>::value;
  float s[4], zp[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    s[r] = val16(sz[r], sdt);
    zp[r] = val16(sz[r] >> 16, sdt) - off * s[r];
  }
#pragma unroll
  for (int t = 0; t < NT; ++t) {
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[t][r] += s[r] * p[t][r] + zp[r] * xs[t];
    p[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
}


// Scale/zero block: 16 bytes = (s, z) of the lane's four output rows.
__device__ __forceinline__ u32x4 sz_load(const uint8_t* szrow, int g, int R) {
  return ld16(szrow + static_cast<size_t>(g) * R * 4);
}

// ---------------------------------------------------------------------------
// Paged GEMM core: one wave streams 16 rows of one page over a K range.
//
// K is processed in chunks of kCK 128-blocks. The activation tile of a chunk
// (NT*16 slots x kCK*128 values) is staged by the whole workgroup into one of
// two LDS buffers; the MFMA B operand is read from LDS. Each wave keeps its
// page's weights for the next chunk in flight in registers while it computes
// the current one, so the only vector-memory traffic in the loop is the
// weight stream plus one activation chunk; every wait count is static.
// Per chunk c:  issue x(c+1) | issue w(c+1) | compute c | LDS <- x(c+1) | barrier
// ---------------------------------------------------------------------------

constexpr int kCK = 2;                            // 128-blocks per chunk
constexpr int kXRow = kCK * 128 * 2 + 16;         // LDS bytes per staged activation row

// Per chunk buffer: NT*16 staged rows, then NT*16 x (2 kCK) fp32 sums of
// 64-value half blocks (the code-domain X of each quantization group).
template <int NT>
constexpr int xbuf_bytes() { return NT * 16 * kXRow + NT * 16 * 2 * kCK * 4; }
template <int NT>
constexpr int lds_x_bytes() { return 2 * xbuf_bytes<NT>(); }

// Rolling register window of a wave's page: slot j holds one 128-block's
// weights (and its scale/zero pairs for quantized pages).
template <int B, int GPK>
struct Slot {
  WF<B> w;
  u32x4 sz[GPK];
};
template <int GPK>
struct Slot<16, GPK> {
  WF<16> w;
};
// Blocks kept in flight per wave: about 8-16 KiB of weights for every format.
template <int B> constexpr int window() { return B == 4 ? 8 : 4; }

template <int B, int GPK>
__device__ __forceinline__ void load_slot(Slot<B, GPK>& sl, const uint8_t* wrow, const uint8_t* szrow,
                                          int b, int lg, int G, int R) {
  wf_load<B>(sl.w, wrow, b);
  if constexpr (B != 16) {
#pragma unroll
    for (int q = 0; q < GPK; ++q) sl.sz[q] = sz_load(szrow, GPK == 2 ? 2 * b + q : (b * 128) / G, R);
  }
}

// The workgroup's activation rows for one chunk (NT*16 rows x kCK*128
// values): thread tid stages the 16-byte pieces q = tid + 256 j, i.e. row
// q / kPieces, piece q % kPieces. rowoff[j] are byte offsets of its rows.
constexpr int kPieces = kCK * 128 / 8;            // 16-byte pieces per row
constexpr int kRowsPerPass = 256 / kPieces;
template <int NT> constexpr int x_passes() { return NT * 16 / kRowsPerPass; }
__device__ __forceinline__ int x_row(int j) { return static_cast<int>(threadIdx.x) / kPieces + kRowsPerPass * j; }

template <int NT>
struct XStage {
  u32x4 v[x_passes<NT>()];
};

template <int NT>
__device__ __forceinline__ void x_fetch(XStage<NT>& s, const uint8_t* base, const uint32_t (&rowoff)[x_passes<NT>()],
                                        int kel, int K) {
  const int col = (threadIdx.x % kPieces) * 8;
  const int k = min(kel + col, K - 8);
#pragma unroll
  for (int j = 0; j < x_passes<NT>(); ++j) s.v[j] = ld16(base + rowoff[j] + static_cast<size_t>(k) * 2);
}

// Writes the staged rows and, per row, the sums of each 64-value half block
// (8 consecutive pieces held by 8 consecutive lanes).
template <int ACT, int NT>
__device__ __forceinline__ void x_store(const XStage<NT>& s, uint8_t* buf) {
  const int col = threadIdx.x % kPieces;
  float* sums = reinterpret_cast<float*>(buf + NT * 16 * kXRow);
#pragma unroll
  for (int j = 0; j < x_passes<NT>(); ++j) {
    *reinterpret_cast<u32x4*>(buf + x_row(j) * kXRow + col * 16) = s.v[j];
    float acc = 0.0f;
#pragma unroll
    for (int q = 0; q < 4; ++q) acc += val16(s.v[j][q], ACT) + val16(s.v[j][q] >> 16, ACT);
    acc += __shfl_xor(acc, 1);
    acc += __shfl_xor(acc, 2);
    acc += __shfl_xor(acc, 4);
    if ((col & 7) == 0) sums[x_row(j) * (2 * kCK) + (col >> 3)] = acc;
  }
}

// LDS stores of this wave complete, then a workgroup barrier (no memory fence:
// weight loads stay in flight across it).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
}

__device__ __forceinline__ bool group_end_g(int GPK, int G, int kb, int i) {
  return GPK == 2 ? ((i & 1) == 1) : (i == 3 && ((kb + 1) * 128) % G == 0);
}

// Four k-steps of one 128-block (absolute block index kb). xblk points at the
// block's 128 values inside the staged chunk; hsum at the chunk's half-block
// sums and hb0 is this block's first half block.
template <int ACT, int B, int NT, int GPK>
__device__ __forceinline__ void compute_block(const Slot<B, GPK>& sl, const uint8_t* xblk, const float* hsum, int hb0,
                                              int kb, int G, int sdt, f32x4 (&acc)[NT], f32x4 (&p)[NT],
                                              float (&xs)[NT]) {
  const int lane = lane_id(), lc = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const u32x4 aw = wf_op<ACT, B>(sl.w, i);
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const u32x4 bx = *reinterpret_cast<const u32x4*>(xblk + (t * 16 + lc) * kXRow + (32 * i + 8 * lg) * 2);
      if constexpr (B == 16) acc[t] = mma<ACT>(aw, bx, acc[t]);
      else p[t] = mma<ACT>(aw, bx, p[t]);
    }
    if constexpr (B != 16) {
      if constexpr (GPK == 2) {
        if (i & 1) {
#pragma unroll
          for (int t = 0; t < NT; ++t) xs[t] = hsum[(t * 16 + lc) * (2 * kCK) + hb0 + (i >> 1)];
          group_fix<ACT, B, NT>(acc, p, xs, sl.sz[i >> 1], sdt);
        }
      } else if (i == 3) {
#pragma unroll
        for (int t = 0; t < NT; ++t)
          xs[t] += hsum[(t * 16 + lc) * (2 * kCK) + hb0] + hsum[(t * 16 + lc) * (2 * kCK) + hb0 + 1];
        if (((kb + 1) * 128) % G == 0) {
          group_fix<ACT, B, NT>(acc, p, xs, sl.sz[0], sdt);
#pragma unroll
          for (int t = 0; t < NT; ++t) xs[t] = 0.0f;
        }
      }
    }
  }
}

// One wave: acc[t] = W[16 rows] . X[16 slots of tile t]^T over 128-blocks
// [kb0, kb1). Block b's weights are loaded window() blocks ahead into slot
// b mod window(); the activation chunk (kCK blocks) of chunk c sits in LDS
// buffer c mod 2. Per chunk c: fetch x(c+1) | compute and refill | LDS <- x(c+1)
// | barrier. Every load is unconditional (addresses clamped to the range), so
// all wait counts are static; the workgroup passes nchunk - 1 barriers here.
template <int ACT, int B, int NT, int GPK>
__device__ void wave_gemm(const GemmArgs& a, uint8_t* lds, const uint8_t* xbase, const uint32_t (&rowoff)[x_passes<NT>()],
                          int K, const uint8_t* wrow, const uint8_t* szrow, int kb0, int kb1, f32x4 (&acc)[NT]) {
  constexpr int W = window<B>();
  static_assert(W % kCK == 0, "window must cover whole chunks");
  const int lg = lane_id() >> 4;
  const int nkb = kb1 - kb0, kmax = kb1 - 1;
  const int nchunk = (nkb + kCK - 1) / kCK;
  f32x4 p[NT];
  float xs[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    acc[t] = p[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    xs[t] = 0.0f;
  }
  Slot<B, GPK> win[W];
  XStage<NT> xr;
  x_fetch<NT>(xr, xbase, rowoff, kb0 * 128, K);
#pragma unroll
  for (int j = 0; j < W; ++j) load_slot<B, GPK>(win[j], wrow, szrow, min(kb0 + j, kmax), lg, a.G, a.R);
  x_store<ACT, NT>(xr, lds);
  lds_barrier();
  for (int base = 0; base < nkb; base += W) {
#pragma unroll
    for (int j = 0; j < W; ++j) {
      const int b = base + j;                       // block index within the range
      const int c = b / kCK;                        // chunk
      uint8_t* buf = lds + (c & 1) * xbuf_bytes<NT>();
      if (j % kCK == 0) x_fetch<NT>(xr, xbase, rowoff, (kb0 + (c + 1) * kCK) * 128, K);
      if (b < nkb)
        compute_block<ACT, B, NT, GPK>(win[j], buf + (b % kCK) * 256,
                                       reinterpret_cast<const float*>(buf + NT * 16 * kXRow), 2 * (b % kCK),
                                       kb0 + b, a.G, a.sdt, acc, p, xs);
      load_slot<B, GPK>(win[j], wrow, szrow, min(kb0 + b + W, kmax), lg, a.G, a.R);
      if (j % kCK == kCK - 1 && c + 1 < nchunk) {
        x_store<ACT, NT>(xr, lds + ((c + 1) & 1) * xbuf_bytes<NT>());
        lds_barrier();
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

__device__ __forceinline__ int fmt_code(uint8_t bits) {
  return bits == 16 ? 0 : bits == 8 ? 1 : bits == 4 ? 2 : -1;
}

// ---------------------------------------------------------------------------
// gate/up: a workgroup covers 32 rows of gate and the same 32 rows of up for
// one expert; waves 0-1 stream gate, waves 2-3 stream up (each in its own
// page format); the SwiGLU output h = silu(g) * u meets through LDS.
// ---------------------------------------------------------------------------

template <int ACT, int NT, int GPK>
__device__ void gateup_unit(const GemmArgs& a, uint8_t* lds, int e, int off_e, int n_e, int r32) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = lane_id(), lc = lane & 15, lg = lane >> 4;
  const int proj = wave >> 1, wsub = wave & 1;
  const int f0 = r32 * 32 + 16 * wsub;
  const int rb = f0 / a.R, lr0 = f0 - rb * a.R;
  const pw_page_entry ent = a.table[(static_cast<size_t>(e) * 3 + proj) * a.nrb_max + rb];
  const int code = fmt_code(ent.bits);
  const int H = a.H;
  float* xch = reinterpret_cast<float*>(lds + lds_x_bytes<NT>());   // [2 waves][NT][64 lanes][4]
  for (int mb = 0; mb < n_e; mb += NT * 16) {
    const uint8_t* xbase = reinterpret_cast<const uint8_t*>(a.x);
    uint32_t rowoff[x_passes<NT>()];
#pragma unroll
    for (int j = 0; j < x_passes<NT>(); ++j) {
      const int m = clampi(mb + x_row(j), 0, n_e - 1);
      const int slot = clampi(a.sorted_slot[off_e + m], 0, a.S - 1);
      rowoff[j] = static_cast<uint32_t>(slot / a.topk) * static_cast<uint32_t>(H * 2);
    }
    f32x4 acc[NT];
    const int nkb = H / 128;
    if (code == 0) {
      const uint8_t* wrow = a.pool + ent.data_off + static_cast<size_t>(lr0 / 16) * (H / 128) * tile_bytes<16>() + 16 * lane;
      wave_gemm<ACT, 16, NT, GPK>(a, lds, xbase, rowoff, H, wrow, nullptr, 0, nkb, acc);
    } else if (code == 1) {
      const uint8_t* wrow = a.pool + ent.data_off + static_cast<size_t>(lr0 / 16) * (H / 128) * tile_bytes<8>() + 16 * lane;
      const uint8_t* szrow = a.pool + ent.sz_off + static_cast<size_t>(lr0 + 4 * lg) * 4;
      wave_gemm<ACT, 8, NT, GPK>(a, lds, xbase, rowoff, H, wrow, szrow, 0, nkb, acc);
    } else {
      const uint8_t* wrow = a.pool + ent.data_off + static_cast<size_t>(lr0 / 16) * (H / 128) * tile_bytes<4>() + 16 * lane;
      const uint8_t* szrow = a.pool + ent.sz_off + static_cast<size_t>(lr0 + 4 * lg) * 4;
      wave_gemm<ACT, 4, NT, GPK>(a, lds, xbase, rowoff, H, wrow, szrow, 0, nkb, acc);
    }
    if (proj == 0) {
#pragma unroll
      for (int t = 0; t < NT; ++t)
        *reinterpret_cast<f32x4*>(xch + ((wsub * NT + t) * 64 + lane) * 4) = acc[t];
    }
    lds_barrier();
    if (proj == 1) {
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const int m = mb + 16 * t + lc;
        if (m < n_e) {
          const f32x4 g = *reinterpret_cast<const f32x4*>(xch + ((wsub * NT + t) * 64 + lane) * 4);
          uint32_t hv[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) hv[r] = rne16(g[r] / (1.0f + expf(-g[r])) * acc[t][r], ACT);
          u32x2 o;
          o[0] = hv[0] | (hv[1] << 16);
          o[1] = hv[2] | (hv[3] << 16);
          *reinterpret_cast<u32x2*>(a.h + static_cast<size_t>(off_e + m) * a.F + f0 + 4 * lg) = o;
        }
      }
    }
    lds_barrier();
  }
}

template <int ACT, int NTMAX, int GPK>
__global__ __launch_bounds__(256) void k_gateup(const GemmArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[lds_x_bytes<NTMAX>() + 2 * NTMAX * 64 * 16];
  const int upe = a.F / 32;
  const int e = blockIdx.x / upe, r32 = blockIdx.x % upe;
  const int off_e = clampi(a.offsets[e], 0, a.S);
  const int n_e = clampi(a.offsets[e + 1], off_e, a.S) - off_e;
  if (n_e <= 0) return;
  // every page of the unit must be present; otherwise the whole group returns
  const int rb = (r32 * 32) / a.R;
  for (int p = 0; p < 2; ++p)
    if (fmt_code(a.table[(static_cast<size_t>(e) * 3 + p) * a.nrb_max + rb].bits) < 0) return;
  if (NTMAX == 1 || n_e <= 16) gateup_unit<ACT, 1, GPK>(a, lds, e, off_e, n_e, r32);
  else if (NTMAX == 2 || n_e <= 32) gateup_unit<ACT, (NTMAX < 2 ? NTMAX : 2), GPK>(a, lds, e, off_e, n_e, r32);
  else gateup_unit<ACT, NTMAX, GPK>(a, lds, e, off_e, n_e, r32);
}

// ---------------------------------------------------------------------------
// down: a workgroup covers 64 rows of one down page over one K split of F;
// fp32 partial sums per split, reduced by the combine.
// ---------------------------------------------------------------------------

template <int ACT, int NT, int GPK>
__device__ void down_unit(const GemmArgs& a, uint8_t* lds, int e, int off_e, int n_e, int r64, int split,
                          const pw_page_entry& ent) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = lane_id(), lc = lane & 15, lg = lane >> 4;
  const int F = a.F;
  const int n0 = r64 * 64 + 16 * wave;
  const int rb = n0 / a.R, lr0 = n0 - rb * a.R;
  const int kb0 = split * a.kb_per_split;
  const int kb1 = min(F / 128, kb0 + a.kb_per_split);
  if (kb0 >= kb1) return;
  const int code = fmt_code(ent.bits);
  for (int mb = 0; mb < n_e; mb += NT * 16) {
    const uint8_t* xbase = reinterpret_cast<const uint8_t*>(a.h);
    uint32_t rowoff[x_passes<NT>()];
#pragma unroll
    for (int j = 0; j < x_passes<NT>(); ++j) {
      const int m = clampi(mb + x_row(j), 0, n_e - 1);
      rowoff[j] = static_cast<uint32_t>(off_e + m) * static_cast<uint32_t>(F * 2);
    }
    f32x4 acc[NT];
    if (code == 0) {
      const uint8_t* wrow = a.pool + ent.data_off + static_cast<size_t>(lr0 / 16) * (F / 128) * tile_bytes<16>() + 16 * lane;
      wave_gemm<ACT, 16, NT, GPK>(a, lds, xbase, rowoff, F, wrow, nullptr, kb0, kb1, acc);
    } else if (code == 1) {
      const uint8_t* wrow = a.pool + ent.data_off + static_cast<size_t>(lr0 / 16) * (F / 128) * tile_bytes<8>() + 16 * lane;
      const uint8_t* szrow = a.pool + ent.sz_off + static_cast<size_t>(lr0 + 4 * lg) * 4;
      wave_gemm<ACT, 8, NT, GPK>(a, lds, xbase, rowoff, F, wrow, szrow, kb0, kb1, acc);
    } else {
      const uint8_t* wrow = a.pool + ent.data_off + static_cast<size_t>(lr0 / 16) * (F / 128) * tile_bytes<4>() + 16 * lane;
      const uint8_t* szrow = a.pool + ent.sz_off + static_cast<size_t>(lr0 + 4 * lg) * 4;
      wave_gemm<ACT, 4, NT, GPK>(a, lds, xbase, rowoff, F, wrow, szrow, kb0, kb1, acc);
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int m = mb + 16 * t + lc;
      if (m < n_e) {
        float* dst = a.opart + (static_cast<size_t>(split) * a.S + off_e + m) * a.H + r64 * 64 + 16 * wave + 4 * lg;
        *reinterpret_cast<f32x4*>(dst) = acc[t];
      }
    }
    lds_barrier();
  }
}

template <int ACT, int NTMAX, int GPK>
__global__ __launch_bounds__(256) void k_down(const GemmArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[lds_x_bytes<NTMAX>()];
  const int upe = a.H / 64;
  const int split = blockIdx.x % a.nsplit;
  const int rest = blockIdx.x / a.nsplit;
  const int e = rest / upe, r64 = rest % upe;
  const int off_e = clampi(a.offsets[e], 0, a.S);
  const int n_e = clampi(a.offsets[e + 1], off_e, a.S) - off_e;
  if (n_e <= 0) return;
  const int rb = (r64 * 64) / a.R;
  const pw_page_entry ent = a.table[(static_cast<size_t>(e) * 3 + PW_DOWN) * a.nrb_max + rb];
  if (fmt_code(ent.bits) < 0) return;
  if (NTMAX == 1 || n_e <= 16) down_unit<ACT, 1, GPK>(a, lds, e, off_e, n_e, r64, split, ent);
  else if (NTMAX == 2 || n_e <= 32) down_unit<ACT, (NTMAX < 2 ? NTMAX : 2), GPK>(a, lds, e, off_e, n_e, r64, split, ent);
  else down_unit<ACT, NTMAX, GPK>(a, lds, e, off_e, n_e, r64, split, ent);
}

// ---------------------------------------------------------------------------
// combine: y[t] = sum_k w[t,k] * sum_split opart[split][slot_pos[t,k]]
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void k_combine(const GemmArgs a) {
  const int t = blockIdx.x;
  const int n = (blockIdx.y * 256 + threadIdx.x) * 4;
  if (n >= a.H) return;
  f32x4 y = {0.f, 0.f, 0.f, 0.f};
  for (int k = 0; k < a.topk; ++k) {
    const int pos = clampi(a.slot_pos[static_cast<size_t>(t) * a.topk + k], 0, a.S - 1);
    f32x4 o = {0.f, 0.f, 0.f, 0.f};
    for (int sp = 0; sp < a.nsplit; ++sp)
      o += *reinterpret_cast<const f32x4*>(a.opart + (static_cast<size_t>(sp) * a.S + pos) * a.H + n);
    const float wk = a.topk_w[static_cast<size_t>(t) * a.topk + k];
    y += wk * o;
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

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------

hipError_t launch_route_topk(const float* logits, int T, int E, int K, int renorm, int32_t* ids,
                             float* w, hipStream_t st) {
  if (T <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_route_topk, dim3((T + 3) / 4), dim3(256), 0, st, logits, T, E, K, renorm, ids, w);
  return hipGetLastError();
}

hipError_t launch_permute(const int32_t* ids, int T, int K, int E, int32_t* offsets,
                          int32_t* sorted_slot, int32_t* slot_pos, hipStream_t st) {
  hipLaunchKernelGGL(k_permute, dim3(E), dim3(kPermThreads), 0, st, ids, T * K, E, offsets,
                     sorted_slot, slot_pos);
  return hipGetLastError();
}

hipError_t launch_qjobs(const QJobBatch& b, hipStream_t st) {
  if (b.total_items == 0) return hipSuccess;
  const dim3 grid((b.total_items + 3) / 4), block(256);
  if (b.nb == 4) hipLaunchKernelGGL(k_qjobs<4>, grid, block, 0, st, b);
  else if (b.nb == 2) hipLaunchKernelGGL(k_qjobs<2>, grid, block, 0, st, b);
  else hipLaunchKernelGGL(k_qjobs<1>, grid, block, 0, st, b);
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

template <int ACT, int GPK>
static hipError_t gemm_launch(const GemmArgs& a, bool gateup, hipStream_t st) {
  const dim3 block(256);
  if (gateup) {
    const dim3 grid(a.E * (a.F / 32));
    if (a.mtb == 1) hipLaunchKernelGGL((k_gateup<ACT, 1, GPK>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((k_gateup<ACT, 2, GPK>), grid, block, 0, st, a);
  } else {
    const dim3 grid(a.E * (a.H / 64) * a.nsplit);
    if (a.mtb == 1) hipLaunchKernelGGL((k_down<ACT, 1, GPK>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((k_down<ACT, 2, GPK>), grid, block, 0, st, a);
  }
  return hipGetLastError();
}

static hipError_t gemm_dispatch(const GemmArgs& a, bool gateup, hipStream_t st) {
  const bool g64 = a.G == 64;
  if (a.act == PW_BF16) return g64 ? gemm_launch<PW_BF16, 2>(a, gateup, st) : gemm_launch<PW_BF16, 1>(a, gateup, st);
  return g64 ? gemm_launch<PW_F16, 2>(a, gateup, st) : gemm_launch<PW_F16, 1>(a, gateup, st);
}

hipError_t launch_gateup(const GemmArgs& a, hipStream_t st) { return gemm_dispatch(a, true, st); }

hipError_t launch_down(const GemmArgs& a, hipStream_t st) { return gemm_dispatch(a, false, st); }

hipError_t launch_combine(const GemmArgs& a, hipStream_t st) {
  if (a.T <= 0) return hipSuccess;
  const dim3 grid(a.T, (a.H / 4 + 255) / 256), block(256);
  hipLaunchKernelGGL(k_combine, grid, block, 0, st, a);
  return hipGetLastError();
}

}  // namespace pw
