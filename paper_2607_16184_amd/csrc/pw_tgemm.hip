// Paged GEMM for large per-expert slot counts (prefill-sized batches), gfx950.
//
// A workgroup of 8 waves (two per SIMD) computes a 256-row x 256-slot tile of
// D = W X^T for one expert: gate/up tiles are 128 rows of gate plus the same
// 128 rows of up (SwiGLU applied in the epilogue), down tiles are 256 rows of
// the down projection. Wave (wn, wm), wn = wave / 4, wm = wave mod 4, owns
// rows 128 wn .. + 128 and slots 64 wm .. + 64: 4 x 2 MFMA 32x32x16 tiles,
// 128 fp32 accumulators. K advances in stages of 64 through a double-buffered
// LDS stage of 64 KiB in 32x32x16 fragment order (1 KiB per 32-row x 16-k
// fragment, lane order), so every operand read and staging write is a
// conflict-free 16-byte LDS access. Each wave stages 32 weight rows (one page,
// dequantized once to the activation dtype) and 32 slots.
//
// Schedule (ping-pong): the two waves of a SIMD belong to different halves
// (wn = 0 and wn = 1), and the wn = 1 half runs one barrier interval behind.
// Between two workgroup barriers one half issues 16 MFMAs from operands
// already in registers while the other half does memory work: LDS writes of
// the next stage, global loads two stages ahead, and the LDS reads of its next
// MFMA operands. So the matrix core of every SIMD is fed by one wave while the
// other waits on memory, and a global load has about four intervals to land.
// The quantized weight enters the MFMA as fl32(z + c s) rounded to the
// activation dtype.
#include "pw_device.hpp"
#include "pw_internal.hpp"

namespace pw {
namespace {

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kTM = 256;                    // slots per tile
constexpr int kTN = 256;                    // weight rows per tile
constexpr int kTK = 64;                     // K per stage (two MFMA k-steps)
constexpr int kWB = kTN * kTK * 2;          // 32 KiB of weights per stage
constexpr int kXB = kTM * kTK * 2;          // 32 KiB of activations per stage
constexpr int kSB = kWB + kXB;              // one stage buffer
constexpr int kGN = 4;                      // weight blocks per raster band
// s_getreg operand for HW_REG_HW_ID (register 4) bits 5:4, the wave's SIMD.
constexpr int kHwRegSimdId = 4 | (4 << 6) | ((2 - 1) << 11);

// Fragment (tile, k-step) offset inside a stage buffer part: 32-row tiles of
// four 1 KiB 16-k blocks, each in 32x32x16 operand lane order (lane l: row
// l mod 32, k-run l / 32 of eight values).
__device__ __forceinline__ int frag32(int tile, int ks) { return (tile * 4 + ks) * 1024; }

// A wave's weight share of a stage: 32 rows (two 16-row tiles) of one page as
// four fragments f = 2 * tile + step.
template <int B> struct WStage;
template <> struct WStage<16> { u32x4 v[4]; };                 // fragment f at v[f]
template <> struct WStage<8> { u32x4 v[2]; uint32_t sz[2]; };  // tile t: both steps
template <> struct WStage<4> { u32x2 v[2]; uint32_t sz[2]; };  // tile t: one word per step

// Nested bit-plane pages (format codes 108 and 104: 8 and 4 planes). Per row
// tile and 128-value block, lane l holds one 32-bit word per plane covering
// its four k-steps; `lut` points at the wave's 32 LUT rows staged in LDS.
// The LUT pointer is held in the LDS address space, so lookups are LDS reads
// with 32-bit addresses (a generic pointer would make them flat loads).
constexpr int kApl8 = 108, kApl4 = 104;
template <int B> constexpr int apl_planes() { return B == kApl8 ? 8 : 4; }
typedef const __attribute__((address_space(3))) uint16_t* lds_lut_t;
template <> struct WStage<kApl8> { uint32_t p[2][8]; int hh; lds_lut_t lut; };
template <> struct WStage<kApl4> { uint32_t p[2][4]; int hh; lds_lut_t lut; };

// A wave's activation share: slot tiles 2 * wave + j / 2, k-step j mod 2.
struct XStage {
  u32x4 v[4];
};

// Weights are re-read by the other slot tiles of the expert: plain (cached) loads.
// For nested bit-plane pages tile0 is the page base plus the wave's row-tile
// offset inside a plane, and szrow carries the wave's LUT rows in LDS.
template <int B>
__device__ __forceinline__ void w_fetch(WStage<B>& w, const uint8_t* tile0, const uint8_t* szrow, int kb, int hh,
                                        int g, int nkb, int R) {
  const int lane = lane_id();
  if constexpr (B == kApl8 || B == kApl4) {
    const size_t rk8 = static_cast<size_t>(R) * nkb * 16;
#pragma unroll
    for (int j = 0; j < apl_planes<B>(); ++j) {
      const size_t pb = j < 4 ? j * rk8 : 4 * rk8 + 32 * static_cast<size_t>(R) + (j - 4) * rk8;
#pragma unroll
      for (int t = 0; t < 2; ++t)
        w.p[t][j] = *reinterpret_cast<const uint32_t*>(tile0 + pb + (static_cast<size_t>(t) * nkb + kb) * 256 +
                                                       4 * lane);
    }
    w.hh = hh;
    w.lut = (lds_lut_t)szrow;   // szrow points into LDS for these pages (generic to LDS: a C-style cast)
    (void)g;
  } else {
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const uint8_t* tp = tile0 + (static_cast<size_t>(t) * nkb + kb) * tile_bytes<B>() + 16 * lane;
    if constexpr (B == 16) {
      w.v[2 * t] = ld16(tp + 2 * hh * 1024);
      w.v[2 * t + 1] = ld16(tp + (2 * hh + 1) * 1024);
    } else if constexpr (B == 8) {
      w.v[t] = ld16(tp + hh * 1024);
    } else {
      w.v[t] = *reinterpret_cast<const u32x2*>(tp + 8 * hh);
    }
  }
  if constexpr (B != 16) {
#pragma unroll
    for (int t = 0; t < 2; ++t)
      w.sz[t] = *reinterpret_cast<const uint32_t*>(szrow + (static_cast<size_t>(g) * R + 16 * t) * 4);
  }
  }
}

// Eight fp32 values -> four packed 16-bit words (round to nearest even).
template <int ACT>
__device__ __forceinline__ u32x4 pack8(const float (&v)[8]) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  typedef __bf16 b2 __attribute__((ext_vector_type(2)));
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  u32x4 o;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const f2 p = {v[2 * q], v[2 * q + 1]};
    if constexpr (ACT == PW_BF16)
      o[q] = __builtin_bit_cast(uint32_t, __builtin_convertvector(p, b2));
    else
      o[q] = __builtin_bit_cast(uint32_t, __builtin_convertvector(p, h2));
  }
  return o;
}

// Fragment f of the wave's weights in the activation dtype: quantized codes
// become fl32(z + c s) (c s is exact in fp32, so one fma rounds once).
template <int ACT, int SDT, int B>
__device__ __forceinline__ u32x4 w_piece(const WStage<B>& w, int f) {
  if constexpr (B == kApl8 || B == kApl4) {
    // plane j's eight bits of this k-step (byte bs of its word) go to byte
    // 7 - j of a 64-bit word (8-bit pages; 4-bit pages: byte 3 - j of a
    // 32-bit word), gathered with byte permutes; a bit transpose then brings
    // each element's plane bits together (plane 0 the most significant)
    const int t = f >> 1;
    const uint32_t bs = static_cast<uint32_t>(2 * w.hh + (f & 1));
    const uint32_t pair = 0x0C0C0000u | ((4u + bs) << 8) | bs;   // (S0.byte bs, S1.byte bs) -> bytes 1, 0
    const uint32_t hi = __builtin_amdgcn_perm(__builtin_amdgcn_perm(w.p[t][0], w.p[t][1], pair),
                                              __builtin_amdgcn_perm(w.p[t][2], w.p[t][3], pair), 0x05040100u);
    constexpr int nl = B == kApl8 ? 256 : 16;
    const lds_lut_t lut = w.lut + (16 * t + (lane_id() & 15)) * nl;
    uint32_t idx[8];
    if constexpr (B == kApl8) {
      const uint32_t lo = __builtin_amdgcn_perm(__builtin_amdgcn_perm(w.p[t][4], w.p[t][5], pair),
                                                __builtin_amdgcn_perm(w.p[t][6], w.p[t][7], pair), 0x05040100u);
      // 8 x 8 transpose (three delta swaps): element e's code in byte e
      uint64_t x = (static_cast<uint64_t>(hi) << 32) | lo;
      uint64_t y = (x ^ (x >> 7)) & 0x00AA00AA00AA00AAull;
      x = x ^ y ^ (y << 7);
      y = (x ^ (x >> 14)) & 0x0000CCCC0000CCCCull;
      x = x ^ y ^ (y << 14);
      y = (x ^ (x >> 28)) & 0x00000000F0F0F0F0ull;
      x = x ^ y ^ (y << 28);
#pragma unroll
      for (int e = 0; e < 8; ++e) idx[e] = static_cast<uint32_t>(x >> (8 * e)) & 0xFFu;
    } else {
      // 4 x 8 transpose: bit 8 r + e (row r = byte r, element e) goes to bit
      // 4 n + r with n = 4 e1 + 2 e0 + e2 (the bits of e rotated), which two
      // delta swaps of index bits (0 with 3, 1 with 4) do: element e's 4-bit
      // code in nibble n
      uint32_t x = hi;
      uint32_t y = (x ^ (x >> 7)) & 0x00AA00AAu;
      x = x ^ y ^ (y << 7);
      y = (x ^ (x >> 14)) & 0x0000CCCCu;
      x = x ^ y ^ (y << 14);
      constexpr int nib[8] = {0, 2, 4, 6, 1, 3, 5, 7};
#pragma unroll
      for (int e = 0; e < 8; ++e) idx[e] = (x >> (4 * nib[e])) & 0xFu;
    }
    u32x4 o;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      o[q] = static_cast<uint32_t>(lut[idx[2 * q]]) | (static_cast<uint32_t>(lut[idx[2 * q + 1]]) << 16);
    return o;
  } else if constexpr (B == 16) {
    return w.v[f];
  } else {
    const int t = f >> 1, i = f & 1;
    const float s = val16(w.sz[t], SDT), z = val16(w.sz[t] >> 16, SDT);
    float v[8];
    if constexpr (B == 8) {
      const uint32_t d0 = w.v[t][2 * i], d1 = w.v[t][2 * i + 1];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v[q] = __builtin_fmaf(static_cast<float>((d0 >> (8 * q)) & 0xFFu), s, z);
        v[4 + q] = __builtin_fmaf(static_cast<float>((d1 >> (8 * q)) & 0xFFu), s, z);
      }
    } else {
      // codes 2u at bits 4u, 2u + 1 at bits 16 + 4u: split the nibbles into bytes
      const uint32_t d = w.v[t][i];
      const uint32_t lo = d & 0x0F0F0F0Fu, hi = (d >> 4) & 0x0F0F0F0Fu;
      const uint32_t src[8] = {lo, lo >> 16, hi, hi >> 16, lo >> 8, lo >> 24, hi >> 8, hi >> 24};
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = __builtin_fmaf(static_cast<float>(src[q] & 0xFFu), s, z);
    }
    return pack8<ACT>(v);
  }
}

// lane l reads slot row l mod 16 of the fragment's tile, k-run l / 16
__device__ __forceinline__ void x_fetch(XStage& x, const uint8_t* const (&xrow)[2], int k0) {
  const int lg = lane_id() >> 4;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    x.v[j] = *reinterpret_cast<const u32x4*>(xrow[j >> 1] + static_cast<size_t>(k0 + 32 * (j & 1) + 8 * lg) * 2);
}

// Writes the wave's staged pieces (32 weight rows and 32 slots over the
// stage's 64 k) to a buffer in 32x32x16 fragment order. A loaded piece holds
// row 16 t + l mod 16 (t: 16-row half), k = 32 i + 8 (l / 16) .. + 7 (i: k-step
// of 32); it goes to 16-k block 2 i + (l / 16) / 2 at lane 16 t + l mod 16 +
// 32 ((l / 16) mod 2). Each group of 16 lanes writes 256 contiguous bytes.
template <int ACT, int SDT, int B>
__device__ __forceinline__ void stage_store(const WStage<B>& w, const XStage& x, uint8_t* buf, int wave) {
  const int lane = lane_id(), lc = lane & 15, lg = lane >> 4;
  uint8_t* d = buf + frag32(wave, lg >> 1) + 16 * (lc + 32 * (lg & 1));
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      *reinterpret_cast<u32x4*>(d + 2048 * i + 256 * t) = w_piece<ACT, SDT, B>(w, 2 * t + i);
      *reinterpret_cast<u32x4*>(d + kWB + 2048 * i + 256 * t) = x.v[2 * t + i];
    }
}

typedef float f32x16 __attribute__((ext_vector_type(16)));

template <int ACT>
__device__ __forceinline__ f32x16 mma32(u32x4 a, u32x4 b, f32x16 c) {
  if constexpr (ACT == PW_BF16)
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c,
                                                  0, 0, 0);
}

// MFMA operands of one half stage (two 16-k blocks) for the wave's 128 x 64
// sub-tile: four 32-row weight fragments and two 32-slot fragments per block.
struct Ops {
  u32x4 a[2][4];
  u32x4 b[2][2];
};

__device__ __forceinline__ void ops_read(Ops& o, const uint8_t* buf, int wn, int wm, int half) {
  const uint8_t* wb = buf + 16 * lane_id();
#pragma unroll
  for (int q = 0; q < 2; ++q) {
#pragma unroll
    for (int r = 0; r < 4; ++r) o.a[q][r] = ld16(wb + frag32(4 * wn + r, 2 * half + q));
#pragma unroll
    for (int c = 0; c < 2; ++c) o.b[q][c] = ld16(wb + kWB + frag32(2 * wm + c, 2 * half + q));
  }
}

template <int ACT>
__device__ __forceinline__ void ops_mma(const Ops& o, f32x16 (&acc)[4][2]) {
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int c = 0; c < 2; ++c) acc[r][c] = mma32<ACT>(o.a[q][r], o.b[q][c], acc[r][c]);
}

// Wait for this wave's LDS operations, then a workgroup barrier. There is no
// memory fence: the global loads of later stages stay in flight across it.
__device__ __forceinline__ void lds_sync() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
}

// The K loop of one wave (its weight share is one page of format B). Per
// stage s, in barrier intervals:
//   MMA(s, first half) | stage s+1 -> LDS, loads of stage s+2 issued,
//   operands of (s, second half) read | MMA(s, second half) | operands of
//   (s+1, first half) read.
// The wn = 1 half passes one extra barrier before its loop and the wn = 0 half
// one after, so the two halves alternate and every wave passes the same
// number of barriers. Stage s+1 is written into the buffer of stage s-1 two
// intervals after that buffer's last read, and first read two intervals
// after its last write.
template <int ACT, int SDT, int B>
__device__ __forceinline__ void tile_loop(uint8_t* lds, const uint8_t* tile0, const uint8_t* szrow,
                                          const uint8_t* const (&xrow)[2], int nkb, int kb0, int kb1, int R,
                                          int G, int wave, int wn, int wm, bool live, f32x16 (&acc)[4][2]) {
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[r][c][e] = 0.0f;
  // stages of 64 values over the 128-blocks [kb0, kb1); stage s of the row
  // is s0 + st
  const int nstage = (kb1 - kb0) * 128 / kTK;
  const int s0 = kb0 * 128 / kTK;
  auto group_of = [&](int st) { return G == 64 ? st : (st * kTK) / G; };
  WStage<B> ws;
  XStage xs;
  Ops op;
  w_fetch<B>(ws, tile0, szrow, s0 >> 1, s0 & 1, group_of(s0), nkb, R);
  x_fetch(xs, xrow, s0 * kTK);
  stage_store<ACT, SDT, B>(ws, xs, lds, wave);
  if (nstage > 1) {
    w_fetch<B>(ws, tile0, szrow, (s0 + 1) >> 1, (s0 + 1) & 1, group_of(s0 + 1), nkb, R);
    x_fetch(xs, xrow, (s0 + 1) * kTK);
  }
  lds_sync();
  if (live) ops_read(op, lds, wn, wm, 0);
  if (wn == 1) lds_sync();
  for (int st = 0; st < nstage; ++st) {
    const uint8_t* cur = lds + (st & 1) * kSB;
    uint8_t* nxt = lds + ((st + 1) & 1) * kSB;
    if (live) ops_mma<ACT>(op, acc);
    lds_sync();
    if (st + 1 < nstage) {
      stage_store<ACT, SDT, B>(ws, xs, nxt, wave);
      if (st + 2 < nstage) {
        const int s2 = s0 + st + 2;
        w_fetch<B>(ws, tile0, szrow, s2 >> 1, s2 & 1, group_of(s2), nkb, R);
        x_fetch(xs, xrow, s2 * kTK);
      }
    }
    if (live) ops_read(op, cur, wn, wm, 1);
    lds_sync();
    if (live) ops_mma<ACT>(op, acc);
    lds_sync();
    if (live && st + 1 < nstage) ops_read(op, nxt, wn, wm, 0);
    lds_sync();
  }
  if (wn == 0) lds_sync();
}


// Maps a tile index to (expert, first slot) from the routing offsets.
__device__ __forceinline__ bool tile_expert(const GemmArgs& a, int mt, int* e_out, int* off_e, int* n_e, int* m0) {
  for (int e = a.e0; e < a.e0 + a.ne; ++e) {
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

template <int ACT, int SDT, bool GATEUP>
__global__ __launch_bounds__(kThreads) void k_tgemm(const GemmArgs a, int nblk, int mtmax) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * kSB];
  __shared__ int simd_of[kWaves];
  // XCD-aware order: each XCD takes a contiguous range of tiles; inside it,
  // bands of kGN weight blocks step the weight block first, so the workgroups
  // resident on an XCD share both weight and slot tiles in its L2.
  const int per_xcd = gridDim.x / 8;
  const int logical = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  const int band = logical / (kGN * mtmax), inb = logical % (kGN * mtmax);
  const int nb = band * kGN + inb % kGN, mt = inb / kGN;
  if (nb >= nblk) return;
  if (!GATEUP && static_cast<int>(blockIdx.y) * a.kb_per_split >= a.F / 128) return;   // an empty K split
  int e, off_e, n_e, m0;
  if (!tile_expert(a, mt, &e, &off_e, &n_e, &m0)) return;

  const int wave = threadIdx.x >> 6, lane = lane_id(), lc = lane & 15;
  // Compute roles: the two waves of a SIMD take wn = 0 and wn = 1 (their rank
  // on the SIMD) and wm = the SIMD, so each SIMD holds one wave of each
  // ping-pong half whatever the wave placement. If a SIMD does not hold
  // exactly two waves, roles follow the wave index. Either way each role is
  // taken once; staging duties follow the wave index.
  if (lane == 0) simd_of[wave] = static_cast<int>(__builtin_amdgcn_s_getreg(kHwRegSimdId));
  __syncthreads();
  int wn = wave >> 2, wm = wave & 3;
  {
    const int mine = simd_of[wave];
    int cnt[4] = {0, 0, 0, 0}, rank = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const int sw = simd_of[w] & 3;
      cnt[sw] += 1;
      rank += (w < wave && sw == mine) ? 1 : 0;
    }
    if (cnt[0] == 2 && cnt[1] == 2 && cnt[2] == 2 && cnt[3] == 2) {
      wn = rank;
      wm = mine & 3;
    }
  }
  const int K = GATEUP ? a.H : a.F;
  const int R = a.R;
  // this wave's 32 weight rows for the staging loader
  int proj, grow;
  if (GATEUP) {
    proj = wave >> 2;                       // waves 0-3: gate; 4-7: up
    grow = nb * 128 + 32 * (wave & 3);
  } else {
    proj = PW_DOWN;
    grow = nb * 256 + 32 * wave;
  }
  const int rb = grow / R, lr0 = grow - rb * R;
  const pw_page_entry ent = a.table[(static_cast<size_t>(e) * 3 + proj) * a.nrb_max + rb];
  const int bits = ent.bits;
  const size_t tbytes = bits == 16 ? 4096 : bits == 8 ? 2048 : 1024;
  const uint8_t* tile0 = a.pool + ent.data_off + static_cast<size_t>(lr0 / 16) * (K / 128) * tbytes;
  const uint8_t* szrow = a.pool + ent.sz_off + static_cast<size_t>(lr0 + lc) * 4;
  // activation rows of this lane's staging fragments: slot tiles 2 * wave + j
  const uint8_t* xrow[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int m = clampi(m0 + (2 * wave + j) * 16 + lc, 0, n_e - 1);
    if (GATEUP) {
      const int slot = clampi(a.sorted_slot[off_e + m], 0, a.S - 1);
      xrow[j] = reinterpret_cast<const uint8_t*>(a.x) + static_cast<size_t>(slot / a.topk) * a.H * 2;
    } else {
      xrow[j] = reinterpret_cast<const uint8_t*>(a.h) + static_cast<size_t>(off_e + m) * a.F * 2;
    }
  }

  // The host checks that every page is present, so bits is 16, 8 or 4 here; a
  // wave never leaves early (the loop's barriers need all eight).
  f32x16 acc[4][2];
  // The down kernel keeps its accumulators in AGPRs (the MFMA's C/D operands
  // then leave the VGPR file to the staging wave of the same SIMD): naming an
  // AGPR in an empty asm statement makes the compiler pick that MFMA form.
  // It fits two waves per SIMD there (about 100 VGPRs + 128 AGPRs); the
  // gate/up kernel would not, and keeps the VGPR form.
  if constexpr (!GATEUP) asm volatile("" ::: "a0");
  const int nkb = K / 128;
  // the down projection may split K = F (grid y: the split; fp32 partials)
  const int split = GATEUP ? 0 : static_cast<int>(blockIdx.y);
  const int kb0 = GATEUP ? 0 : split * a.kb_per_split;
  const int kb1 = GATEUP ? nkb : min(nkb, kb0 + a.kb_per_split);
  // In an expert's ragged last tile, waves whose 64 slots all lie past the
  // expert's slots still stage their share and pass every barrier, but read
  // no operands and issue no MFMAs (their LDS bandwidth goes to the others).
  const bool live = m0 + wm * 64 < n_e;
  if (bits == 16) tile_loop<ACT, SDT, 16>(lds, tile0, szrow, xrow, nkb, kb0, kb1, R, a.G, wave, wn, wm, live, acc);
  else if (bits == 8) tile_loop<ACT, SDT, 8>(lds, tile0, szrow, xrow, nkb, kb0, kb1, R, a.G, wave, wn, wm, live, acc);
  else tile_loop<ACT, SDT, 4>(lds, tile0, szrow, xrow, nkb, kb0, kb1, R, a.G, wave, wn, wm, live, acc);

  // Accumulator element 4 q + r of tile (rt, ct) is row 32 rt + 8 q + 4 (lane / 32)
  // + r of the wave's 128 rows, slot 32 ct + lane mod 32 of its 64 slots.
  const int rsub = 4 * (lane >> 5), msub = lane & 31;
  if (GATEUP) {
    // gate waves (wn = 0) hand their 128 x 64 accumulators to the up wave of
    // the same slots through LDS (free once every wave has left the loop)
    f32x4* xch = reinterpret_cast<f32x4*>(lds) + wm * (4 * 2 * 4 * 64);
    if (wn == 0) {
#pragma unroll
      for (int rt = 0; rt < 4; ++rt)
#pragma unroll
        for (int ct = 0; ct < 2; ++ct)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            xch[((rt * 2 + ct) * 4 + q) * 64 + lane] =
                f32x4{acc[rt][ct][4 * q], acc[rt][ct][4 * q + 1], acc[rt][ct][4 * q + 2], acc[rt][ct][4 * q + 3]};
    }
    __syncthreads();
    if (wn == 1) {
#pragma unroll
      for (int ct = 0; ct < 2; ++ct) {
        const int m = m0 + wm * 64 + ct * 32 + msub;
        if (m < n_e) {
#pragma unroll
          for (int rt = 0; rt < 4; ++rt)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const f32x4 g = xch[((rt * 2 + ct) * 4 + q) * 64 + lane];
              uint32_t hv[4];
#pragma unroll
              for (int r = 0; r < 4; ++r) hv[r] = rne16(g[r] / (1.0f + expf(-g[r])) * acc[rt][ct][4 * q + r], ACT);
              u32x2 o;
              o[0] = hv[0] | (hv[1] << 16);
              o[1] = hv[2] | (hv[3] << 16);
              *reinterpret_cast<u32x2*>(a.h + static_cast<size_t>(off_e + m) * a.F + nb * 128 + rt * 32 + q * 8 +
                                        rsub) = o;
            }
        }
      }
    }
  } else {
#pragma unroll
    for (int ct = 0; ct < 2; ++ct) {
      const int m = m0 + wm * 64 + ct * 32 + msub;
      if (m < n_e) {
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            *reinterpret_cast<f32x4*>(a.opart + (static_cast<size_t>(split) * a.S + off_e + m) * a.H + nb * 256 + wn * 128 +
                                      rt * 32 + q * 8 + rsub) =
                f32x4{acc[rt][ct][4 * q], acc[rt][ct][4 * q + 1], acc[rt][ct][4 * q + 2], acc[rt][ct][4 * q + 3]};
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Streaming paged GEMM for small and medium per-expert slot counts (decode,
// fine-grained experts): HBM-bound, so the design goal is bytes in flight.
// A workgroup of 4 waves covers 128 weight rows (gate/up: 64 rows of gate and
// the same 64 rows of up; down: 128 rows) and MT slots of one expert. Each wave
// streams 32 rows of one page through a register ring of D stages (64 values
// of K each, about 8 KiB per wave for every format) and computes them against
// all MT slots itself, so weights never pass through LDS; the MT x 64 slice of
// activations is staged once per stage for the four waves. Quantized weights
// are dequantized in registers to fl32(z + c s) rounded to the activation
// dtype, as in the large-tile kernel.
// ---------------------------------------------------------------------------

template <int B> constexpr int sg_depth() { return B == 16 ? 2 : B == 8 || B == kApl8 ? 4 : 8; }
constexpr int kSgStagePad = 8;   // stage counts are padded to a multiple of every depth

template <int MT> constexpr int sg_xbuf() { return MT * kTK * 2; }            // one activation buffer
template <int MT> constexpr int sg_lds() { return 2 * sg_xbuf<MT>() + 4 * 1024; } // + a discard area

// The loop body has no branches (every load and store is unconditional, with
// clamped indices), so the compiler's wait counts stay static and the ring's
// D stages really are in flight.
// The wave's rows over 128-blocks [kb0, kb1) of the nkb blocks of a row.
template <int ACT, int SDT, int B, int MT>
__device__ __forceinline__ void sg_loop(uint8_t* lds, const uint8_t* tile0, const uint8_t* szrow,
                                        const uint8_t* xrow, int xf, int nkb, int kb0, int kb1, int R, int gshift,
                                        int wave, f32x4 (&acc)[2][MT / 16]) {
  constexpr int D = sg_depth<B>();
  constexpr int XF = MT >= 32 ? MT / 32 : 1;       // activation fragments per wave
  constexpr int XB = sg_xbuf<MT>();
  const int lane = lane_id(), lg = lane >> 4;
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int u = 0; u < MT / 16; ++u) acc[t][u] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int nstage = (kb1 - kb0) * 128 / kTK;
  const int st0 = kb0 * 128 / kTK;                 // first stage of the range within the row
  const int npad = (nstage + kSgStagePad - 1) / kSgStagePad * kSgStagePad;
  auto group_of = [&](int st) { return (st * kTK) >> gshift; };
  // waves past the tile's activation fragments write a discard area instead
  const int xoff = xf < MT / 8 ? 1024 * xf : 2 * XB + 1024 * wave - 1024 * xf;
  auto fetch_w = [&](WStage<B>& w, int st) {
    const int s = st0 + min(st, nstage - 1);
    w_fetch<B>(w, tile0, szrow, s >> 1, s & 1, group_of(s), nkb, R);
  };
  // activation fragment q of this wave: xf + q (slot tile (xf + q) / 2, k-step (xf + q) mod 2)
  auto fetch_x = [&](u32x4 (&xv)[XF], int st) {
    const int s = st0 + min(st, nstage - 1);
#pragma unroll
    for (int q = 0; q < XF; ++q)
      xv[q] = ld16(xrow + static_cast<size_t>(s * kTK + 32 * ((xf + q) & 1) + 8 * lg) * 2);
  };
  auto store_x = [&](const u32x4 (&xv)[XF], int b) {
    uint8_t* d = lds + (xf < MT / 8 ? b * XB : 0) + xoff + 16 * lane;
#pragma unroll
    for (int q = 0; q < XF; ++q) *reinterpret_cast<u32x4*>(d + 1024 * q) = xv[q];
  };
  WStage<B> ring[D];
  u32x4 xv[XF];
#pragma unroll
  for (int j = 0; j < D; ++j) fetch_w(ring[j], j);
  fetch_x(xv, 0);
  store_x(xv, 0);
  __syncthreads();
  for (int base = 0; base < npad; base += D) {
#pragma unroll
    for (int j = 0; j < D; ++j) {
      const int st = base + j;
      const uint8_t* cur = lds + (st & 1) * XB + 16 * lane;
      fetch_x(xv, st + 1);
      __builtin_amdgcn_sched_barrier(0);   // issue the activation load first: its wait ends the stage
      const bool live = st < nstage;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        u32x4 bx[MT / 16];
#pragma unroll
        for (int u = 0; u < MT / 16; ++u) bx[u] = ld16(cur + 1024 * (2 * u + i));
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          u32x4 aw = w_piece<ACT, SDT, B>(ring[j], 2 * t + i);
          if (!live) aw = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
          for (int u = 0; u < MT / 16; ++u) acc[t][u] = mma<ACT>(aw, bx[u], acc[t][u]);
        }
      }
      fetch_w(ring[j], st + D);
      store_x(xv, (st + 1) & 1);
      __syncthreads();
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// LUT rows of the four waves (32 rows x 256 values each) for nested bit-plane pages
constexpr int kSgLutWave = 32 * 256 * 2;

template <int ACT, int SDT, bool GATEUP, int MT, bool APL>
__global__ __launch_bounds__(256) void k_sgemm(const GemmArgs a, int nblk, int mtmax) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[sg_lds<MT>() + (APL ? 4 * kSgLutWave : 0)];
  // the down projection may split K = F into a.nsplit ranges (fp32 partials,
  // summed by the combine); split-major block order
  const int nsplit = GATEUP ? 1 : a.nsplit;
  const int per_split = gridDim.x / nsplit;
  const int split = blockIdx.x / per_split, bid = blockIdx.x % per_split;
  const int per_xcd = per_split / 8;
  const int logical = (bid % 8) * per_xcd + bid / 8;
  const int band = logical / (kGN * mtmax), inb = logical % (kGN * mtmax);
  const int nb = band * kGN + inb % kGN, mt = inb / kGN;
  if (nb >= nblk) return;
  int e = 0, off_e = 0, n_e = 0, m0 = 0;
  {
    int rest = mt;
    bool found = false;
    for (int x = a.e0; x < a.e0 + a.ne && !found; ++x) {
      const int o = clampi(a.offsets[x], 0, a.S);
      const int n = clampi(a.offsets[x + 1], o, a.S) - o;
      const int cnt = (n + MT - 1) / MT;
      if (rest < cnt) {
        e = x;
        off_e = o;
        n_e = n;
        m0 = rest * MT;
        found = true;
      } else {
        rest -= cnt;
      }
    }
    if (!found) return;
  }
  const int wave = threadIdx.x >> 6, lane = lane_id(), lc = lane & 15, lg = lane >> 4;
  const int K = GATEUP ? a.H : a.F;
  const int R = a.R;
  int proj, grow;
  if (GATEUP) {
    proj = wave >> 1;                       // waves 0-1: gate; 2-3: up
    grow = nb * 64 + 32 * (wave & 1);
  } else {
    proj = PW_DOWN;
    grow = nb * 128 + 32 * wave;
  }
  const int rb = grow / R, lr0 = grow - rb * R;
  const pw_page_entry ent = a.table[(static_cast<size_t>(e) * 3 + proj) * a.nrb_max + rb];
  const int bits = ent.bits;
  const bool apl_page = APL && (ent.rsv & 0xFF) == PW_FMT_APL;
  const size_t tbytes = apl_page ? 256 : bits == 16 ? 4096 : bits == 8 ? 2048 : 1024;
  const uint8_t* tile0 = a.pool + ent.data_off + static_cast<size_t>(lr0 / 16) * (K / 128) * tbytes;
  const uint8_t* szrow = a.pool + ent.sz_off + static_cast<size_t>(lr0 + lc) * 4;
  if (APL && apl_page) {
    // the wave's 32 LUT rows of the committed precision go to its LDS area
    const int nl = bits == 8 ? 256 : 16;
    const size_t rk8 = static_cast<size_t>(R) * K / 8;
    const uint8_t* src = a.pool + ent.sz_off + (bits == 8 ? 32 * static_cast<size_t>(R) + 4 * rk8 : 0) +
                         static_cast<size_t>(lr0) * nl * 2;
    uint8_t* dst = lds + sg_lds<MT>() + wave * kSgLutWave;
    for (int o = 16 * lane; o < 32 * nl * 2; o += 16 * 64)
      *reinterpret_cast<u32x4*>(dst + o) = *reinterpret_cast<const u32x4*>(src + o);
    szrow = dst;
  }
  // this wave's activation fragments start at xf = wave * XF (slot tile xf / 2)
  constexpr int XF = MT >= 32 ? MT / 32 : 1;
  const int xf = wave * XF;
  const int m = clampi(m0 + (xf >> 1) * 16 + lc, 0, n_e - 1);
  const uint8_t* xrow;
  if (GATEUP) {
    const int slot = clampi(a.sorted_slot[off_e + m], 0, a.S - 1);
    xrow = reinterpret_cast<const uint8_t*>(a.x) + static_cast<size_t>(slot / a.topk) * a.H * 2;
  } else {
    xrow = reinterpret_cast<const uint8_t*>(a.h) + static_cast<size_t>(off_e + m) * a.F * 2;
  }
  // The host checks that every page is present, so bits is 16, 8 or 4 here; a
  // wave never leaves early (the loop's barriers need all four).
  f32x4 acc[2][MT / 16];
  const int nkb = K / 128;
  const int kb0 = GATEUP ? 0 : split * a.kb_per_split;
  const int kb1 = GATEUP ? nkb : min(nkb, kb0 + a.kb_per_split);
  if (kb0 >= kb1) return;                         // (whole workgroup: no barrier passed yet)
  const int gshift = 31 - __builtin_clz(a.G);     // G is a power of two, at least 64
  if constexpr (APL) {
    if (apl_page) {
      if (bits == 8) sg_loop<ACT, SDT, kApl8, MT>(lds, tile0, szrow, xrow, xf, nkb, kb0, kb1, R, gshift, wave, acc);
      else sg_loop<ACT, SDT, kApl4, MT>(lds, tile0, szrow, xrow, xf, nkb, kb0, kb1, R, gshift, wave, acc);
    } else if (bits == 16) {
      sg_loop<ACT, SDT, 16, MT>(lds, tile0, szrow, xrow, xf, nkb, kb0, kb1, R, gshift, wave, acc);
    } else if (bits == 8) {
      sg_loop<ACT, SDT, 8, MT>(lds, tile0, szrow, xrow, xf, nkb, kb0, kb1, R, gshift, wave, acc);
    } else {
      sg_loop<ACT, SDT, 4, MT>(lds, tile0, szrow, xrow, xf, nkb, kb0, kb1, R, gshift, wave, acc);
    }
  } else {
    if (bits == 16) sg_loop<ACT, SDT, 16, MT>(lds, tile0, szrow, xrow, xf, nkb, kb0, kb1, R, gshift, wave, acc);
    else if (bits == 8) sg_loop<ACT, SDT, 8, MT>(lds, tile0, szrow, xrow, xf, nkb, kb0, kb1, R, gshift, wave, acc);
    else sg_loop<ACT, SDT, 4, MT>(lds, tile0, szrow, xrow, xf, nkb, kb0, kb1, R, gshift, wave, acc);
  }

  const int wr = wave & 1;
  if (GATEUP) {
    // gate waves hand their 32 x MT accumulators to the up wave of the same rows
    float* xch = reinterpret_cast<float*>(lds) + wr * (2 * (MT / 16) * 64 * 4);
    if (proj == PW_GATE) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int u = 0; u < MT / 16; ++u)
          *reinterpret_cast<f32x4*>(xch + ((t * (MT / 16) + u) * 64 + lane) * 4) = acc[t][u];
    }
    __syncthreads();
    if (proj == PW_UP) {
#pragma unroll
      for (int u = 0; u < MT / 16; ++u) {
        const int mm = m0 + u * 16 + lc;
        if (mm < n_e) {
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            const f32x4 g = *reinterpret_cast<const f32x4*>(xch + ((t * (MT / 16) + u) * 64 + lane) * 4);
            uint32_t hv[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) hv[r] = rne16(g[r] / (1.0f + expf(-g[r])) * acc[t][u][r], ACT);
            u32x2 o;
            o[0] = hv[0] | (hv[1] << 16);
            o[1] = hv[2] | (hv[3] << 16);
            *reinterpret_cast<u32x2*>(a.h + static_cast<size_t>(off_e + mm) * a.F + grow + t * 16 + 4 * lg) = o;
          }
        }
      }
    }
  } else {
#pragma unroll
    for (int u = 0; u < MT / 16; ++u) {
      const int mm = m0 + u * 16 + lc;
      if (mm < n_e) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
          *reinterpret_cast<f32x4*>(a.opart + (static_cast<size_t>(split) * a.S + off_e + mm) * a.H + grow + t * 16 +
                                    4 * lg) =
              acc[t][u];
      }
    }
  }
}

template <int ACT, int SDT, int MT>
void sgemm_go(const GemmArgs& a, bool gateup, hipStream_t st) {
  const int nblk = gateup ? a.F / 64 : a.H / 128;
  const int mtmax = (a.s_range + MT - 1) / MT + a.ne;
  const int n = ((nblk + kGN - 1) / kGN * kGN * mtmax + 7) / 8 * 8 * (gateup ? 1 : a.nsplit);
  if (a.apl) {
    if (gateup)
      hipLaunchKernelGGL((k_sgemm<ACT, SDT, true, MT, true>), dim3(n), dim3(256), 0, st, a, nblk, mtmax);
    else
      hipLaunchKernelGGL((k_sgemm<ACT, SDT, false, MT, true>), dim3(n), dim3(256), 0, st, a, nblk, mtmax);
  } else if (gateup) {
    hipLaunchKernelGGL((k_sgemm<ACT, SDT, true, MT, false>), dim3(n), dim3(256), 0, st, a, nblk, mtmax);
  } else {
    hipLaunchKernelGGL((k_sgemm<ACT, SDT, false, MT, false>), dim3(n), dim3(256), 0, st, a, nblk, mtmax);
  }
}

// Layers with nested bit-plane pages run this kernel at every batch size;
// at decode sizes (up to 24 expected slots per expert) 32-slot tiles halve
// the activation staging, and with the LUT rows the workgroup's LDS then fits
// twice per CU.
template <int ACT, int SDT>
void sgemm_mt(const GemmArgs& a, bool gateup, hipStream_t st) {
  const int expect = (a.s_range + a.ne - 1) / a.ne;
  if (a.apl && expect <= 24) sgemm_go<ACT, SDT, 32>(a, gateup, st);
  else sgemm_go<ACT, SDT, 64>(a, gateup, st);
}

template <int ACT, int SDT>
void tgemm_go(const GemmArgs& a, bool gateup, int n, int nblk, int mtmax, hipStream_t st) {
  if (gateup)
    hipLaunchKernelGGL((k_tgemm<ACT, SDT, true>), dim3(n), dim3(kThreads), 0, st, a, nblk, mtmax);
  else
    hipLaunchKernelGGL((k_tgemm<ACT, SDT, false>), dim3(n, a.nsplit), dim3(kThreads), 0, st, a, nblk, mtmax);
}

}  // namespace

// Tile counts of the large-M path: an upper bound on slot tiles.
int tgemm_mtmax(int S, int E) { return (S + kTM - 1) / kTM + E; }

hipError_t launch_tgemm(const GemmArgs& a, bool gateup, hipStream_t st) {
  if (a.ne <= 0) return hipSuccess;
  const int nblk = gateup ? a.F / 128 : a.H / 256;
  const int mtmax = tgemm_mtmax(a.s_range, a.ne);
  const int n = ((nblk + kGN - 1) / kGN * kGN * mtmax + 7) / 8 * 8;
  if (a.act == PW_BF16) {
    if (a.sdt == PW_BF16) tgemm_go<PW_BF16, PW_BF16>(a, gateup, n, nblk, mtmax, st);
    else tgemm_go<PW_BF16, PW_F16>(a, gateup, n, nblk, mtmax, st);
  } else {
    if (a.sdt == PW_BF16) tgemm_go<PW_F16, PW_BF16>(a, gateup, n, nblk, mtmax, st);
    else tgemm_go<PW_F16, PW_F16>(a, gateup, n, nblk, mtmax, st);
  }
  return hipGetLastError();
}

// Streaming path (64-slot tiles): per-expert slot counts between the decode
// kernels' range and the large-tile kernel's.
hipError_t launch_sgemm(const GemmArgs& a, bool gateup, hipStream_t st) {
  if (a.ne <= 0) return hipSuccess;
  if (a.act == PW_BF16) {
    if (a.sdt == PW_BF16) sgemm_mt<PW_BF16, PW_BF16>(a, gateup, st);
    else sgemm_mt<PW_BF16, PW_F16>(a, gateup, st);
  } else {
    if (a.sdt == PW_BF16) sgemm_mt<PW_F16, PW_BF16>(a, gateup, st);
    else sgemm_mt<PW_F16, PW_F16>(a, gateup, st);
  }
  return hipGetLastError();
}

}  // namespace pw
