// Paged GEMM for large per-expert slot counts (prefill-sized batches), gfx950.
//
// A workgroup (4 waves) computes a 256-row x 256-slot tile of D = W X^T for
// one expert: gate/up tiles are 128 rows of gate plus the same 128 rows of up
// (SwiGLU applied in the epilogue), down tiles are 256 rows of the down
// projection. Each wave owns a 128 x 128 sub-tile (8 x 8 MFMA 16x16x32 tiles,
// 256 fp32 accumulators). K advances in stages of 64: the workgroup stages the
// weights, dequantized once to the activation dtype, and the activations into
// a double-buffered LDS stage of 64 KiB laid out in MFMA fragment order, so
// every operand read is a conflict-free 16-byte LDS load. For large slot
// counts dequantizing once per stage costs less VALU work than the decode
// kernels' code-domain correction, whose cost grows with the slot count; the
// quantized weight enters the MFMA rounded to the activation dtype.
#include "pw_device.hpp"
#include "pw_internal.hpp"

namespace pw {
namespace {

constexpr int kTM = 256;                    // slots per tile
constexpr int kTN = 256;                    // weight rows per tile
constexpr int kTK = 64;                     // K per stage (two MFMA k-steps)
constexpr int kWB = kTN * kTK * 2;          // 32 KiB of weights per stage
constexpr int kXB = kTM * kTK * 2;          // 32 KiB of activations per stage
constexpr int kSB = kWB + kXB;              // one stage buffer

// Fragment (tile, k-step) offset inside a stage buffer part: 16-row tiles of
// two 1 KiB k-step blocks, each in lane order (lane l: row l mod 16, k-run l / 16).
__device__ __forceinline__ int frag_off(int tile, int i) { return (tile * 2 + i) * 1024; }

// A wave's share of the weight stage: 64 rows (four 16-row tiles) of one page.
template <int B> struct WStage;
template <> struct WStage<16> { u32x4 v[8]; };                 // tile t, step i at v[2t + i]
template <> struct WStage<8> { u32x4 v[4]; uint32_t sz[4]; };  // tile t: steps 2hh, 2hh+1
template <> struct WStage<4> { u32x2 v[4]; uint32_t sz[4]; };  // tile t: words of steps 2hh, 2hh+1

struct XStageT {
  u32x4 v[8];
};

template <int B>
__device__ __forceinline__ void w_fetch(WStage<B>& w, const uint8_t* tile0, const uint8_t* szrow, int kb, int hh,
                                        int g, int nkb, int R) {
  const int lane = lane_id();
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const uint8_t* tp = tile0 + (static_cast<size_t>(t) * nkb + kb) * tile_bytes<B>() + 16 * lane;
    if constexpr (B == 16) {
      w.v[2 * t] = ld16_nt(tp + 2 * hh * 1024);
      w.v[2 * t + 1] = ld16_nt(tp + (2 * hh + 1) * 1024);
    } else if constexpr (B == 8) {
      w.v[t] = ld16_nt(tp + hh * 1024);
    } else {
      w.v[t] = *reinterpret_cast<const u32x2*>(tp + 8 * hh);
    }
  }
  if constexpr (B != 16) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
      w.sz[t] = *reinterpret_cast<const uint32_t*>(szrow + (static_cast<size_t>(g) * R + 16 * t) * 4);
  }
}

// 8 dequantized values (k-run of one k-step) -> four packed 16-bit words.
template <int ACT>
__device__ __forceinline__ u32x4 deq8(const uint32_t (&c)[8], uint32_t szw, int sdt) {
  const float s = val16(szw, sdt), z = val16(szw >> 16, sdt);
  u32x4 o;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float v0 = z + static_cast<float>(c[2 * q]) * s;       // fl32(z + c s)
    const float v1 = z + static_cast<float>(c[2 * q + 1]) * s;
    o[q] = rne16(v0, ACT) | (rne16(v1, ACT) << 16);
  }
  return o;
}

template <int ACT, int B>
__device__ __forceinline__ void w_store(const WStage<B>& w, uint8_t* wbuf, int tile_base, int sdt) {
  const int lane = lane_id();
#pragma unroll
  for (int t = 0; t < 4; ++t) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      u32x4 o;
      if constexpr (B == 16) {
        o = w.v[2 * t + i];
      } else {
        uint32_t c[8];
        if constexpr (B == 8) {
          const uint32_t d0 = w.v[t][2 * i], d1 = w.v[t][2 * i + 1];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            c[q] = (d0 >> (8 * q)) & 0xFFu;
            c[4 + q] = (d1 >> (8 * q)) & 0xFFu;
          }
        } else {
          const uint32_t d = w.v[t][i];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            c[2 * u] = (d >> (4 * u)) & 15u;
            c[2 * u + 1] = (d >> (16 + 4 * u)) & 15u;
          }
        }
        o = deq8<ACT>(c, w.sz[t], sdt);
      }
      *reinterpret_cast<u32x4*>(wbuf + frag_off(tile_base + t, i) + 16 * lane) = o;
    }
  }
}

// Activation stage: thread tid copies pieces q = tid + 256 j (slot row q / 8,
// 8-value piece q mod 8) into fragment order.
__device__ __forceinline__ void x_fetch_t(XStageT& x, const uint8_t* base, const uint32_t (&rowoff)[8], int k0) {
  const int p = threadIdx.x & 7;
#pragma unroll
  for (int j = 0; j < 8; ++j) x.v[j] = *reinterpret_cast<const u32x4*>(base + rowoff[j] + static_cast<size_t>(k0 + 8 * p) * 2);
}

__device__ __forceinline__ void x_store_t(const XStageT& x, uint8_t* xbuf) {
  const int p = threadIdx.x & 7, i = p >> 2, lg = p & 3;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int r = (threadIdx.x >> 3) + 32 * j;
    *reinterpret_cast<u32x4*>(xbuf + frag_off(r >> 4, i) + 16 * (16 * lg + (r & 15))) = x.v[j];
  }
}

template <int ACT>
__device__ __forceinline__ void stage_mma(const uint8_t* buf, int wn, int wm, f32x4 (&acc)[8][8]) {
  const int lane = lane_id();
  const uint8_t* wbuf = buf;
  const uint8_t* xbuf = buf + kWB;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    u32x4 b[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) b[u] = *reinterpret_cast<const u32x4*>(xbuf + frag_off(wm * 8 + u, i) + 16 * lane);
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const u32x4 at = *reinterpret_cast<const u32x4*>(wbuf + frag_off(wn * 8 + t, i) + 16 * lane);
#pragma unroll
      for (int u = 0; u < 8; ++u) acc[t][u] = mma<ACT>(at, b[u], acc[t][u]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// The K loop of one wave (its staging share is one page of format B): stage
// s + 1 is fetched while stage s feeds the MFMAs, then written to the other
// LDS buffer; one barrier per stage.
template <int ACT, int B>
__device__ void tile_loop(const GemmArgs& a, uint8_t* lds, const uint8_t* tile0, const uint8_t* szrow,
                          const uint8_t* xbase, const uint32_t (&rowoff)[8], int nkb, int wave, f32x4 (&acc)[8][8]) {
  const int wn = wave >> 1, wm = wave & 1;
#pragma unroll
  for (int t = 0; t < 8; ++t)
#pragma unroll
    for (int u = 0; u < 8; ++u) acc[t][u] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int nstage = nkb * 128 / kTK;
  auto group_of = [&](int st) { return a.G == 64 ? st : (st * kTK) / a.G; };
  WStage<B> ws;
  XStageT xs;
  w_fetch<B>(ws, tile0, szrow, 0, 0, group_of(0), nkb, a.R);
  x_fetch_t(xs, xbase, rowoff, 0);
  w_store<ACT, B>(ws, lds, 4 * wave, a.sdt);
  x_store_t(xs, lds + kWB);
  __syncthreads();
  for (int st = 0; st < nstage; ++st) {
    uint8_t* cur = lds + (st & 1) * kSB;
    uint8_t* nxt = lds + ((st + 1) & 1) * kSB;
    const bool more = st + 1 < nstage;
    if (more) {
      const int s1 = st + 1;
      w_fetch<B>(ws, tile0, szrow, s1 >> 1, s1 & 1, group_of(s1), nkb, a.R);
      x_fetch_t(xs, xbase, rowoff, s1 * kTK);
    }
    stage_mma<ACT>(cur, wn, wm, acc);
    if (more) {
      w_store<ACT, B>(ws, nxt, 4 * wave, a.sdt);
      x_store_t(xs, nxt + kWB);
    }
    __syncthreads();
  }
}

// Maps a tile index to (expert, first slot) from the routing offsets.
__device__ __forceinline__ bool tile_expert(const GemmArgs& a, int mt, int* e_out, int* off_e, int* n_e, int* m0) {
  for (int e = 0; e < a.E; ++e) {
    const int o = clampi(a.offsets[e], 0, a.S);
    const int n = clampi(a.offsets[e + 1], o, a.S) - o;
    const int cnt = (n + kTM - 1) / kTM;
    if (mt < cnt) {
      *e_out = e;
      *off_e = o;
      *n_e = n;
      *m0 = mt * kTM;
      return true;
    }
    mt -= cnt;
  }
  return false;
}

template <int ACT, bool GATEUP>
__global__ __launch_bounds__(256) void k_tgemm(const GemmArgs a, int nblk, int mtmax) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * kSB];
  // XCD-aware order: consecutive workgroups of one XCD take consecutive tiles,
  // which share a weight block (same rows, next slot tile) and its L2 lines.
  const int nwg = gridDim.x;
  const int per_xcd = nwg / 8;
  const int logical = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  const int nb = logical / mtmax, mt = logical % mtmax;
  if (nb >= nblk) return;
  int e, off_e, n_e, m0;
  if (!tile_expert(a, mt, &e, &off_e, &n_e, &m0)) return;

  const int tid = threadIdx.x, wave = tid >> 6, lane = lane_id(), lc = lane & 15, lg = lane >> 4;
  const int wn = wave >> 1, wm = wave & 1;
  const int K = GATEUP ? a.H : a.F;
  const int R = a.R;
  // this wave's 64 weight rows for the staging loader
  int proj, grow;
  if (GATEUP) {
    proj = wave >> 1;                       // waves 0,1: gate; 2,3: up
    grow = nb * 128 + 64 * (wave & 1);
  } else {
    proj = PW_DOWN;
    grow = nb * 256 + 64 * wave;
  }
  const int rb = grow / R, lr0 = grow - rb * R;
  const pw_page_entry ent = a.table[(static_cast<size_t>(e) * 3 + proj) * a.nrb_max + rb];
  const int bits = ent.bits;
  if (bits != 16 && bits != 8 && bits != 4) return;   // (the host checks that every page is present)
  const size_t tbytes = bits == 16 ? 4096 : bits == 8 ? 2048 : 1024;
  const uint8_t* tile0 = a.pool + ent.data_off + static_cast<size_t>(lr0 / 16) * (K / 128) * tbytes;
  const uint8_t* szrow = a.pool + ent.sz_off + static_cast<size_t>(lr0 + lc) * 4;
  // activation rows of this thread's staging pieces
  const uint8_t* xbase = GATEUP ? reinterpret_cast<const uint8_t*>(a.x) : reinterpret_cast<const uint8_t*>(a.h);
  uint32_t rowoff[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int m = clampi(m0 + (tid >> 3) + 32 * j, 0, n_e - 1);
    if (GATEUP) {
      const int slot = clampi(a.sorted_slot[off_e + m], 0, a.S - 1);
      rowoff[j] = static_cast<uint32_t>(slot / a.topk) * static_cast<uint32_t>(a.H * 2);
    } else {
      rowoff[j] = static_cast<uint32_t>(off_e + m) * static_cast<uint32_t>(a.F * 2);
    }
  }

  f32x4 acc[8][8];
  const int nkb = K / 128;
  if (bits == 16) tile_loop<ACT, 16>(a, lds, tile0, szrow, xbase, rowoff, nkb, wave, acc);
  else if (bits == 8) tile_loop<ACT, 8>(a, lds, tile0, szrow, xbase, rowoff, nkb, wave, acc);
  else tile_loop<ACT, 4>(a, lds, tile0, szrow, xbase, rowoff, nkb, wave, acc);

  if (GATEUP) {
    // gate waves (wn = 0) hand their 128 x 128 accumulators to the up waves
    float* xch = reinterpret_cast<float*>(lds) + wm * (8 * 8 * 64 * 4);
    if (wn == 0) {
#pragma unroll
      for (int t = 0; t < 8; ++t)
#pragma unroll
        for (int u = 0; u < 8; ++u) *reinterpret_cast<f32x4*>(xch + ((t * 8 + u) * 64 + lane) * 4) = acc[t][u];
    }
    __syncthreads();
    if (wn == 1) {
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int m = m0 + wm * 128 + u * 16 + lc;
        if (m < n_e) {
#pragma unroll
          for (int t = 0; t < 8; ++t) {
            const f32x4 g = *reinterpret_cast<const f32x4*>(xch + ((t * 8 + u) * 64 + lane) * 4);
            uint32_t hv[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) hv[r] = rne16(g[r] / (1.0f + expf(-g[r])) * acc[t][u][r], ACT);
            u32x2 o;
            o[0] = hv[0] | (hv[1] << 16);
            o[1] = hv[2] | (hv[3] << 16);
            *reinterpret_cast<u32x2*>(a.h + static_cast<size_t>(off_e + m) * a.F + nb * 128 + t * 16 + 4 * lg) = o;
          }
        }
      }
    }
  } else {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int m = m0 + wm * 128 + u * 16 + lc;
      if (m < n_e) {
#pragma unroll
        for (int t = 0; t < 8; ++t)
          *reinterpret_cast<f32x4*>(a.opart + static_cast<size_t>(off_e + m) * a.H + nb * 256 + wn * 128 + t * 16 + 4 * lg) =
              acc[t][u];
      }
    }
  }
}

}  // namespace

// Tile counts of the large-M path: weight blocks and an upper bound on slot tiles.
int tgemm_mtmax(int S, int E) { return (S + kTM - 1) / kTM + E; }

hipError_t launch_tgemm(const GemmArgs& a, bool gateup, hipStream_t st) {
  const int nblk = gateup ? a.F / 128 : a.H / 256;
  const int mtmax = tgemm_mtmax(a.S, a.E);
  const int n = (nblk * mtmax + 7) / 8 * 8;
  if (a.act == PW_BF16) {
    if (gateup) hipLaunchKernelGGL((k_tgemm<PW_BF16, true>), dim3(n), dim3(256), 0, st, a, nblk, mtmax);
    else hipLaunchKernelGGL((k_tgemm<PW_BF16, false>), dim3(n), dim3(256), 0, st, a, nblk, mtmax);
  } else {
    if (gateup) hipLaunchKernelGGL((k_tgemm<PW_F16, true>), dim3(n), dim3(256), 0, st, a, nblk, mtmax);
    else hipLaunchKernelGGL((k_tgemm<PW_F16, false>), dim3(n), dim3(256), 0, st, a, nblk, mtmax);
  }
  return hipGetLastError();
}

}  // namespace pw
