// Decode-size paged GEMMs for gfx950 (CDNA4): gate/up with the fused SwiGLU,
// and down with fp32 partial sums per K split. Used while an expert holds at
// most a few 16-slot tiles; larger batches go to pw_tgemm.hip.
//
// GEMM layout. Each wave computes D[n][m] = sum_k W[n][k] * X[m][k] for RT
// tiles of 16 weight rows n (the MFMA A operand) against tiles of 16 routed
// slots m (the B operand) with v_mfma_f32_16x16x32_{bf16,f16}; each B fragment
// read from LDS feeds the RT row tiles. K is walked in blocks of 128; a block
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
#include "pw_device.hpp"
#include "pw_internal.hpp"

namespace pw {
namespace {

// Code-domain offset of a page format (see the file comment).
template <int ACT, int B>
struct CodeOff {
  static constexpr float value = (B == 16) ? 0.0f : (ACT == PW_BF16 ? (B == 4 ? 128.0f : 0.0f) : 1024.0f);
};

// Group layout along K: G = 64 (two groups per 128-block), G = 128 (one
// group per block), G = 256 or 512 (one group spans 2 or 4 blocks).
enum { kG64 = 0, kG128 = 1, kGBig = 2 };
template <int GK> constexpr int groups_per_block() { return GK == kG64 ? 2 : 1; }

// 16-bit value of dtype FMT in the low half of h, as fp32.
template <int FMT>
__device__ __forceinline__ float lo16(uint32_t h) {
  if constexpr (FMT == PW_BF16) return __uint_as_float(h << 16);
  else return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(h)));
}
template <int FMT>
__device__ __forceinline__ float hi16(uint32_t h) {
  if constexpr (FMT == PW_BF16) return __uint_as_float(h & 0xFFFF0000u);
  else return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(h >> 16)));
}

template <int B> struct WF;
template <> struct WF<16> { u32x4 v[4]; };
template <> struct WF<8> { u32x4 v[2]; };
template <> struct WF<4> { u32x4 v[1]; };

// The lane's 16-byte pieces of 128-block blk of its row tile. `tiles` is the
// row tile's first tile (wave-uniform), `loff` = 16 * lane.
template <int B>
__device__ __forceinline__ void wf_load(WF<B>& f, const uint8_t* tiles, uint32_t loff, int blk) {
  const uint8_t* p = tiles + static_cast<size_t>(blk) * tile_bytes<B>();
#pragma unroll
  for (int i = 0; i < tile_bytes<B>() / 1024; ++i) f.v[i] = ld16_nt(p + 1024 * i + loff);
}

// A operand of k-step i: eight 16-bit values (weights, or codes as floats).
// `magic` is OFF as a pair of 16-bit floats, held in a register so that the
// 4-bit unpack is one v_and_or_b32 per operand register.
template <int ACT, int B>
__device__ __forceinline__ u32x4 wf_op(const WF<B>& f, int i, uint32_t magic) {
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
    u32x4 o;
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q] = ((w >> (4 * q)) & 0x000F000Fu) | magic;
    return o;
  }
}

template <int ACT> constexpr uint32_t code_magic() { return ACT == PW_BF16 ? 0x43004300u : 0x64006400u; }

// acc += s * P + (z - OFF s) * X for the lane's four rows (two fused
// multiply-adds per row). X[t] is the group's activation sum for this lane's
// slot (tile t).
template <int ACT, int SDT, int B, int NT>
__device__ __forceinline__ void group_fix(f32x4 (&acc)[NT], const f32x4 (&p)[NT], const float (&xs)[NT], u32x4 sz) {
  constexpr float off = CodeOff<ACT, B>::value;
  float s[4], zp[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    s[r] = lo16<SDT>(sz[r]);
    zp[r] = __builtin_fmaf(-off, s[r], hi16<SDT>(sz[r]));
  }
#pragma unroll
  for (int t = 0; t < NT; ++t) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      acc[t][r] = __builtin_fmaf(s[r], p[t][r], acc[t][r]);
      acc[t][r] = __builtin_fmaf(zp[r], xs[t], acc[t][r]);
    }
  }
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

// A wave streams RT 16-row weight tiles: each B fragment read from LDS feeds
// RT MFMAs. RT = 1 for up to two slot tiles per expert (decode), RT = 2 for
// four (the LDS operand traffic per weight byte halves).
template <int NTMAX> constexpr int row_tiles() { return NTMAX >= 4 ? 2 : 1; }

// Rolling register window of a wave's page: slot j holds one 128-block of the
// wave's RT row tiles (and their scale/zero pairs for quantized pages).
template <int B, int GK, int RT>
struct Slot {
  WF<B> w[RT];
  u32x4 sz[RT][groups_per_block<GK>()];
};
template <int GK, int RT>
struct Slot<16, GK, RT> {
  WF<16> w[RT];
};
// Blocks kept in flight per wave: 4-16 KiB of weights. Small windows keep the
// kernels at three (RT = 1) or two (RT = 2) waves per SIMD, which hides more
// latency than deeper per-wave prefetch.
template <int B, int RT> constexpr int window() { return RT == 1 && B == 4 ? 4 : 2; }

// Where a wave's page rows live: wave-uniform bases plus per-lane offsets.
// Row tile rt of the wave starts rt * tstride bytes after `tiles` and its
// scale/zero pairs 64 * rt bytes after `sz`.
struct PageRows {
  const uint8_t* tiles;    // first tile of the wave's first 16-row tile row
  const uint8_t* sz;       // scale/zero pair of the wave's first row, group 0
  size_t tstride;          // bytes of one tile row: (K / 128) tiles
  uint32_t wlo, szlo;      // lane offsets: 16 * lane, 16 * (lane / 16)
  int R;                   // rows per page (pair stride between groups)
  int gshift;              // log2(G / 128) for G >= 128
};

template <int B, int GK, int RT>
__device__ __forceinline__ void load_slot(Slot<B, GK, RT>& sl, const PageRows& pr, int b) {
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) wf_load<B>(sl.w[rt], pr.tiles + rt * pr.tstride, pr.wlo, b);
  if constexpr (B != 16) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int q = 0; q < groups_per_block<GK>(); ++q) {
        const int g = GK == kG64 ? 2 * b + q : GK == kG128 ? b : (b >> pr.gshift);
        sl.sz[rt][q] = ld16(pr.sz + static_cast<size_t>(g) * pr.R * 4 + 64 * rt + pr.szlo);
      }
  }
}

// The workgroup's activation rows for one chunk (NT*16 rows x kCK*128
// values): thread tid stages the 16-byte pieces q = tid + 256 j, i.e. row
// q / kPieces, piece q % kPieces. rowoff[j] are byte offsets of its rows.
constexpr int kPieces = kCK * 128 / 8;            // 16-byte pieces per row
// NW waves per workgroup stage a chunk together: rows per pass and passes.
template <int NW> constexpr int rows_per_pass() { return 64 * NW / kPieces; }
template <int NT, int NW> constexpr int x_passes() { return NT * 16 / rows_per_pass<NW>(); }
template <int NW>
__device__ __forceinline__ int x_row(int j) {
  return static_cast<int>(threadIdx.x) / kPieces + rows_per_pass<NW>() * j;
}

template <int NT, int NW>
struct XStage {
  u32x4 v[x_passes<NT, NW>()];
};

template <int NT, int NW>
__device__ __forceinline__ void x_fetch(XStage<NT, NW>& s, const uint8_t* base,
                                        const uint32_t (&rowoff)[x_passes<NT, NW>()], int kel, int K) {
  const int col = (threadIdx.x % kPieces) * 8;
  const int k = min(kel + col, K - 8);
#pragma unroll
  for (int j = 0; j < x_passes<NT, NW>(); ++j) s.v[j] = ld16(base + rowoff[j] + static_cast<size_t>(k) * 2);
}

// Sum of the eight 16-bit values of a piece: four dot products with (1, 1).
// (Each pair is copied out with memcpy: a bit_cast of a vector element to a
// 2 x 16-bit vector has been compiled to a read of element 0 every time.)
template <int ACT>
__device__ __forceinline__ float piece_sum(u32x4 v) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
  const uint32_t one = ACT == PW_BF16 ? 0x3F803F80u : 0x3C003C00u;
  float acc = 0.0f;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t w = v[q];
    if constexpr (ACT == PW_BF16) {
      bf16x2 a, b;
      __builtin_memcpy(&a, &w, 4);
      __builtin_memcpy(&b, &one, 4);
      acc = __builtin_amdgcn_fdot2_f32_bf16(a, b, acc, false);
    } else {
      f16x2 a, b;
      __builtin_memcpy(&a, &w, 4);
      __builtin_memcpy(&b, &one, 4);
      acc = __builtin_amdgcn_fdot2(a, b, acc, false);
    }
  }
  return acc;
}

// Sum over the eight lanes 8j..8j+7 (DPP within quads, then half-row mirror).
__device__ __forceinline__ float sum8(float v) {
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false));  // row_half_mirror
  return v;
}

// Writes the staged rows and, when a quantized page reads them, per row the
// sums of each 64-value half block (8 consecutive pieces held by 8
// consecutive lanes).
template <int ACT, int NT, int NW>
__device__ __forceinline__ void x_store(const XStage<NT, NW>& s, uint8_t* buf, bool sums) {
  const int col = threadIdx.x % kPieces;
#pragma unroll
  for (int j = 0; j < x_passes<NT, NW>(); ++j)
    *reinterpret_cast<u32x4*>(buf + x_row<NW>(j) * kXRow + col * 16) = s.v[j];
  if (sums) {
    float* hs = reinterpret_cast<float*>(buf + NT * 16 * kXRow);
#pragma unroll
    for (int j = 0; j < x_passes<NT, NW>(); ++j) {
      const float acc = sum8(piece_sum<ACT>(s.v[j]));
      if ((col & 7) == 0) hs[x_row<NW>(j) * (2 * kCK) + (col >> 3)] = acc;
    }
  }
}

// LDS stores of this wave complete, then a workgroup barrier (no memory fence:
// weight loads stay in flight across it).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
}

// Four k-steps of one 128-block. xblk points at the block's 128 values inside
// the staged chunk; hsum at the chunk's half-block sums and hb0 is this
// block's first half block. gend: a G > 128 group ends with this block.
// A group's P starts from a zero accumulator in its first k-step.
template <int ACT, int SDT, int B, int NT, int GK, int RT>
__device__ __forceinline__ void compute_block(const Slot<B, GK, RT>& sl, const uint8_t* xblk, const float* hsum,
                                              int hb0, bool gend, uint32_t magic, f32x4 (&acc)[RT][NT],
                                              f32x4 (&p)[RT][NT], float (&xs)[NT]) {
  const int lane = lane_id(), lc = lane & 15, lg = lane >> 4;
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    u32x4 aw[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) aw[rt] = wf_op<ACT, B>(sl.w[rt], i, magic);
    const bool fresh = (GK == kG128 && i == 0) || (GK == kG64 && (i & 1) == 0);
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const u32x4 bx = *reinterpret_cast<const u32x4*>(xblk + (t * 16 + lc) * kXRow + (32 * i + 8 * lg) * 2);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        if constexpr (B == 16) acc[rt][t] = mma<ACT>(aw[rt], bx, acc[rt][t]);
        else p[rt][t] = mma<ACT>(aw[rt], bx, fresh ? zero : p[rt][t]);
      }
    }
    if constexpr (B != 16) {
      if constexpr (GK == kG64) {
        if (i & 1) {
#pragma unroll
          for (int t = 0; t < NT; ++t) xs[t] = hsum[(t * 16 + lc) * (2 * kCK) + hb0 + (i >> 1)];
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) group_fix<ACT, SDT, B, NT>(acc[rt], p[rt], xs, sl.sz[rt][i >> 1]);
        }
      } else if constexpr (GK == kG128) {
        if (i == 3) {
#pragma unroll
          for (int t = 0; t < NT; ++t)
            xs[t] = hsum[(t * 16 + lc) * (2 * kCK) + hb0] + hsum[(t * 16 + lc) * (2 * kCK) + hb0 + 1];
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) group_fix<ACT, SDT, B, NT>(acc[rt], p[rt], xs, sl.sz[rt][0]);
        }
      } else if (i == 3) {
#pragma unroll
        for (int t = 0; t < NT; ++t)
          xs[t] += hsum[(t * 16 + lc) * (2 * kCK) + hb0] + hsum[(t * 16 + lc) * (2 * kCK) + hb0 + 1];
        if (gend) {
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) {
            group_fix<ACT, SDT, B, NT>(acc[rt], p[rt], xs, sl.sz[rt][0]);
#pragma unroll
            for (int t = 0; t < NT; ++t) p[rt][t] = zero;
          }
#pragma unroll
          for (int t = 0; t < NT; ++t) xs[t] = 0.0f;
        }
      }
    }
  }
}

// One wave: acc[rt][t] = W[16 rows of tile rt] . X[16 slots of tile t]^T over 128-blocks
// [kb0, kb1). Block b's weights are loaded window() blocks ahead into slot
// b mod window(); the activation chunk (kCK blocks) of chunk c sits in LDS
// buffer c mod 2. Per chunk c: fetch x(c+1) | compute and refill | LDS <- x(c+1)
// | barrier. Every load is unconditional (addresses clamped to the range), so
// all wait counts are static; the workgroup passes nchunk - 1 barriers here.
// `sums`: some wave of the workgroup reads a quantized page (workgroup-uniform).
template <int ACT, int SDT, int B, int NT, int GK, int RT, int NW>
__device__ void wave_gemm(uint8_t* lds, const uint8_t* xbase, const uint32_t (&rowoff)[x_passes<NT, NW>()], int K,
                          const PageRows& pr, int kb0, int kb1, bool sums, f32x4 (&acc)[RT][NT]) {
  constexpr int W = window<B, RT>();
  static_assert(W % kCK == 0, "window must cover whole chunks");
  const int nkb = kb1 - kb0, kmax = kb1 - 1;
  const int nchunk = (nkb + kCK - 1) / kCK;
  const int gmask = (1 << pr.gshift) - 1;
  // OFF in a register: keeps the unpack's constant out of the instruction
  uint32_t magic = code_magic<ACT>();
  asm volatile("" : "+v"(magic));
  f32x4 p[RT][NT];
  float xs[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) acc[rt][t] = p[rt][t] = f32x4{0.f, 0.f, 0.f, 0.f};
    xs[t] = 0.0f;
  }
  Slot<B, GK, RT> win[W];
  XStage<NT, NW> xr;
  x_fetch<NT, NW>(xr, xbase, rowoff, kb0 * 128, K);
#pragma unroll
  for (int j = 0; j < W; ++j) load_slot<B, GK, RT>(win[j], pr, min(kb0 + j, kmax));
  x_store<ACT, NT, NW>(xr, lds, sums);
  lds_barrier();
  for (int base = 0; base < nkb; base += W) {
#pragma unroll
    for (int j = 0; j < W; ++j) {
      const int b = base + j;                       // block index within the range
      const int c = b / kCK;                        // chunk
      uint8_t* buf = lds + (c & 1) * xbuf_bytes<NT>();
      if (j % kCK == 0) x_fetch<NT, NW>(xr, xbase, rowoff, (kb0 + (c + 1) * kCK) * 128, K);
      if (b < nkb)
        compute_block<ACT, SDT, B, NT, GK, RT>(win[j], buf + (b % kCK) * 256,
                                           reinterpret_cast<const float*>(buf + NT * 16 * kXRow), 2 * (b % kCK),
                                           ((kb0 + b + 1) & gmask) == 0, magic, acc, p, xs);
      load_slot<B, GK, RT>(win[j], pr, min(kb0 + b + W, kmax));
      if (j % kCK == kCK - 1 && c + 1 < nchunk) {
        x_store<ACT, NT, NW>(xr, lds + ((c + 1) & 1) * xbuf_bytes<NT>(), sums);
        lds_barrier();
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

__device__ __forceinline__ int fmt_code(uint8_t bits) {
  return bits == 16 ? 0 : bits == 8 ? 1 : bits == 4 ? 2 : -1;
}

// Wave-uniform bases of the rows from local row lr0 of a page of reduction
// length K (row tile rt at tiles + rt * tstride).
template <int B>
__device__ __forceinline__ PageRows page_rows(const GemmArgs& a, const pw_page_entry& ent, int lr0, int K) {
  const int lane = lane_id();
  PageRows pr;
  pr.tstride = static_cast<size_t>(K / 128) * tile_bytes<B>();
  pr.tiles = a.pool + ent.data_off + static_cast<size_t>(lr0 / 16) * pr.tstride;
  pr.sz = a.pool + ent.sz_off + static_cast<size_t>(lr0) * 4;
  pr.wlo = 16u * static_cast<uint32_t>(lane);
  pr.szlo = 16u * static_cast<uint32_t>(lane >> 4);
  pr.R = a.R;
  pr.gshift = a.G > 128 ? 31 - __builtin_clz(a.G / 128) : 0;
  return pr;
}

// The wave's page in format B (16, 8 or 4), or B = 0: in the format its
// table entry names, chosen here.
template <int ACT, int SDT, int B, int NT, int GK, int RT, int NW>
__device__ __forceinline__ void page_gemm(const GemmArgs& a, const pw_page_entry& ent, int lr0, int K, uint8_t* lds,
                                          const uint8_t* xbase, const uint32_t (&rowoff)[x_passes<NT, NW>()], int kb0,
                                          int kb1, bool sums, f32x4 (&acc)[RT][NT]) {
  if constexpr (B != 0) {
    wave_gemm<ACT, SDT, B, NT, GK, RT, NW>(lds, xbase, rowoff, K, page_rows<B>(a, ent, lr0, K), kb0, kb1, sums, acc);
  } else {
    const int code = fmt_code(ent.bits);
    if (code == 0)
      wave_gemm<ACT, SDT, 16, NT, GK, RT, NW>(lds, xbase, rowoff, K, page_rows<16>(a, ent, lr0, K), kb0, kb1, sums,
                                              acc);
    else if (code == 1)
      wave_gemm<ACT, SDT, 8, NT, GK, RT, NW>(lds, xbase, rowoff, K, page_rows<8>(a, ent, lr0, K), kb0, kb1, sums,
                                             acc);
    else
      wave_gemm<ACT, SDT, 4, NT, GK, RT, NW>(lds, xbase, rowoff, K, page_rows<4>(a, ent, lr0, K), kb0, kb1, sums,
                                             acc);
  }
}

// ---------------------------------------------------------------------------
// gate/up: a workgroup of NW waves covers 8 RT NW rows of gate and the same
// rows of up for one expert; the first NW / 2 waves stream gate, the others
// up (16 RT rows each, each wave in its own page's format); the SwiGLU output
// h = silu(g) * u meets through LDS. NW = 8 at four slot tiles (each staged
// activation chunk then serves twice the weight rows), else 4.
// ---------------------------------------------------------------------------

template <int RT, int NW> constexpr int gu_rows() { return 8 * RT * NW; }    // gate (and up) rows per workgroup
template <int RT, int NW> constexpr int dn_rows() { return 16 * RT * NW; }   // down rows per workgroup

// [NW / 2 waves][RT][NT][64 lanes] f32x4 of the gate waves, in the activation
// buffers once every wave has finished its K loop.
template <int NT, int RT, int NW>
constexpr int xch_bytes() { return NW / 2 * RT * NT * 64 * 16; }
template <int NT, int RT, int NW>
constexpr int gu_lds_bytes() {
  return lds_x_bytes<NT>() > xch_bytes<NT, RT, NW>() ? lds_x_bytes<NT>() : xch_bytes<NT, RT, NW>();
}

template <int ACT, int SDT, int B, int NT, int GK, int RT, int NW>
__device__ void gateup_unit(const GemmArgs& a, uint8_t* lds, int e, int off_e, int n_e, int unit, bool sums) {
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int lane = lane_id(), lc = lane & 15, lg = lane >> 4;
  const int proj = wave / (NW / 2), wsub = wave % (NW / 2);
  const int f0 = unit * gu_rows<RT, NW>() + 16 * RT * wsub;   // the wave's first row
  const int rb = f0 / a.R, lr0 = f0 - rb * a.R;
  const pw_page_entry ent = a.table[(static_cast<size_t>(e) * 3 + proj) * a.nrb_max + rb];
  const int H = a.H;
  f32x4* xch = reinterpret_cast<f32x4*>(lds);
  for (int mb = 0; mb < n_e; mb += NT * 16) {
    const uint8_t* xbase = reinterpret_cast<const uint8_t*>(a.x);
    uint32_t rowoff[x_passes<NT, NW>()];
#pragma unroll
    for (int j = 0; j < x_passes<NT, NW>(); ++j) {
      const int m = clampi(mb + x_row<NW>(j), 0, n_e - 1);
      const int slot = clampi(a.sorted_slot[off_e + m], 0, a.S - 1);
      rowoff[j] = static_cast<uint32_t>(slot / a.topk) * static_cast<uint32_t>(H * 2);
    }
    f32x4 acc[RT][NT];
    page_gemm<ACT, SDT, B, NT, GK, RT, NW>(a, ent, lr0, H, lds, xbase, rowoff, 0, H / 128, sums, acc);
    lds_barrier();   // every wave is done with the activation buffers
    if (proj == 0) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int t = 0; t < NT; ++t) xch[((wsub * RT + rt) * NT + t) * 64 + lane] = acc[rt][t];
    }
    lds_barrier();
    if (proj == 1) {
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const int m = mb + 16 * t + lc;
        if (m < n_e) {
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) {
            const f32x4 g = xch[((wsub * RT + rt) * NT + t) * 64 + lane];
            uint32_t hv[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) hv[r] = rne16(g[r] / (1.0f + expf(-g[r])) * acc[rt][t][r], ACT);
            u32x2 o;
            o[0] = hv[0] | (hv[1] << 16);
            o[1] = hv[2] | (hv[3] << 16);
            *reinterpret_cast<u32x2*>(a.h + static_cast<size_t>(off_e + m) * a.F + f0 + 16 * rt + 4 * lg) = o;
          }
        }
      }
    }
    lds_barrier();
  }
}

// RT = 1: one code body that picks the format inside; RT = 2: each wave runs
// the whole unit in its own page's format (every format passes the same
// barriers), which keeps the register allocations of the three apart.
template <int ACT, int SDT, int NT, int GK, int RT, int NW>
__device__ __forceinline__ void gateup_any(int code, const GemmArgs& a, uint8_t* lds, int e, int off_e, int n_e,
                                           int unit, bool sums) {
  if constexpr (RT == 1) {
    gateup_unit<ACT, SDT, 0, NT, GK, RT, NW>(a, lds, e, off_e, n_e, unit, sums);
  } else {
    if (code == 0) gateup_unit<ACT, SDT, 16, NT, GK, RT, NW>(a, lds, e, off_e, n_e, unit, sums);
    else if (code == 1) gateup_unit<ACT, SDT, 8, NT, GK, RT, NW>(a, lds, e, off_e, n_e, unit, sums);
    else gateup_unit<ACT, SDT, 4, NT, GK, RT, NW>(a, lds, e, off_e, n_e, unit, sums);
  }
}

// Workgroups are dealt to the eight XCDs in turn (blockIdx mod 8), each XCD
// with its own L2. With many experts, the down projection gives all `per_e`
// workgroups of one expert to one XCD (XCD x runs experts x, x + 8, x + 16,
// ... in order), so the expert's h rows, which no other expert reads, are
// fetched into one L2 instead of eight (the gate/up activations are token
// rows that every XCD reads anyway). The grid holds ne * per_e workgroups.
__device__ __forceinline__ int xcd_expert_order(int b, int per_e, int ne) {
  if (ne < 32 || ne % 8 != 0) return b;
  const int x = b & 7, j = b >> 3;
  return (x + 8 * (j / per_e)) * per_e + j % per_e;
}

// NTMAX slot tiles per pass (1, 2 or 4); experts with fewer slots take fewer
// (at NTMAX = 4 also three).
template <int ACT, int SDT, int NTMAX, int GK, int NW>
__global__ __launch_bounds__(64 * NW) void k_gateup(const GemmArgs a) {
  constexpr int RT = row_tiles<NTMAX>();
  constexpr int GU = gu_rows<RT, NW>();
  __shared__ __attribute__((aligned(16))) uint8_t lds[gu_lds_bytes<NTMAX, RT, NW>()];
  const int upe = a.F / GU;
  const int e = a.e0 + static_cast<int>(blockIdx.x) / upe, unit = blockIdx.x % upe;
  const int off_e = clampi(a.offsets[e], 0, a.S);
  const int n_e = clampi(a.offsets[e + 1], off_e, a.S) - off_e;
  if (n_e <= 0) return;
  // every page of the unit (one, or several when it spans pages) must be
  // present; otherwise the whole group returns
  bool sums = false;
  for (int rb = (unit * GU) / a.R; rb <= (unit * GU + GU - 1) / a.R; ++rb) {
    const int cg = fmt_code(a.table[(static_cast<size_t>(e) * 3 + PW_GATE) * a.nrb_max + rb].bits);
    const int cu = fmt_code(a.table[(static_cast<size_t>(e) * 3 + PW_UP) * a.nrb_max + rb].bits);
    if (cg < 0 || cu < 0) return;
    sums = sums || cg != 0 || cu != 0;
  }
  // the format of this wave's own page (its 16 RT rows lie inside one page)
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int proj = wave / (NW / 2), f0 = unit * GU + 16 * RT * (wave % (NW / 2));
  const int code = fmt_code(a.table[(static_cast<size_t>(e) * 3 + proj) * a.nrb_max + f0 / a.R].bits);
  if (NTMAX == 1 || n_e <= 16) gateup_any<ACT, SDT, 1, GK, RT, NW>(code, a, lds, e, off_e, n_e, unit, sums);
  else if (NTMAX == 2 || n_e <= 32) gateup_any<ACT, SDT, 2, GK, RT, NW>(code, a, lds, e, off_e, n_e, unit, sums);
  else if (n_e <= 48) gateup_any<ACT, SDT, 3, GK, RT, NW>(code, a, lds, e, off_e, n_e, unit, sums);
  else gateup_any<ACT, SDT, (NTMAX > 2 ? NTMAX : 2), GK, RT, NW>(code, a, lds, e, off_e, n_e, unit, sums);
}

// ---------------------------------------------------------------------------
// down: a workgroup of NW waves covers 16 RT NW rows of the down projection
// (16 RT per wave; one or more pages) over one K split of F; fp32 partial
// sums per split, reduced by the combine.
// ---------------------------------------------------------------------------

template <int ACT, int SDT, int B, int NT, int GK, int RT, int NW>
__device__ void down_unit(const GemmArgs& a, uint8_t* lds, int e, int off_e, int n_e, int unit, int split,
                          bool sums) {
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int lane = lane_id(), lc = lane & 15, lg = lane >> 4;
  const int F = a.F;
  const int n0 = unit * dn_rows<RT, NW>() + 16 * RT * wave;   // the wave's first row
  const int rb = n0 / a.R, lr0 = n0 - rb * a.R;
  const pw_page_entry ent = a.table[(static_cast<size_t>(e) * 3 + PW_DOWN) * a.nrb_max + rb];
  const int kb0 = split * a.kb_per_split;
  const int kb1 = min(F / 128, kb0 + a.kb_per_split);
  for (int mb = 0; mb < n_e; mb += NT * 16) {
    const uint8_t* xbase = reinterpret_cast<const uint8_t*>(a.h);
    uint32_t rowoff[x_passes<NT, NW>()];
#pragma unroll
    for (int j = 0; j < x_passes<NT, NW>(); ++j) {
      const int m = clampi(mb + x_row<NW>(j), 0, n_e - 1);
      rowoff[j] = static_cast<uint32_t>(off_e + m) * static_cast<uint32_t>(F * 2);
    }
    f32x4 acc[RT][NT];
    page_gemm<ACT, SDT, B, NT, GK, RT, NW>(a, ent, lr0, F, lds, xbase, rowoff, kb0, kb1, sums, acc);
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int m = mb + 16 * t + lc;
      if (m < n_e) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          float* dst = a.opart + (static_cast<size_t>(split) * a.S + off_e + m) * a.H + n0 + 16 * rt + 4 * lg;
          *reinterpret_cast<f32x4*>(dst) = acc[rt][t];
        }
      }
    }
    lds_barrier();
  }
}

template <int ACT, int SDT, int NT, int GK, int RT, int NW>
__device__ __forceinline__ void down_any(int code, const GemmArgs& a, uint8_t* lds, int e, int off_e, int n_e,
                                         int unit, int split, bool sums) {
  if constexpr (RT == 1) {
    down_unit<ACT, SDT, 0, NT, GK, RT, NW>(a, lds, e, off_e, n_e, unit, split, sums);
  } else {
    if (code == 0) down_unit<ACT, SDT, 16, NT, GK, RT, NW>(a, lds, e, off_e, n_e, unit, split, sums);
    else if (code == 1) down_unit<ACT, SDT, 8, NT, GK, RT, NW>(a, lds, e, off_e, n_e, unit, split, sums);
    else down_unit<ACT, SDT, 4, NT, GK, RT, NW>(a, lds, e, off_e, n_e, unit, split, sums);
  }
}

template <int ACT, int SDT, int NTMAX, int GK, int NW>
__global__ __launch_bounds__(64 * NW) void k_down(const GemmArgs a) {
  constexpr int RT = row_tiles<NTMAX>();
  constexpr int DN = dn_rows<RT, NW>();
  __shared__ __attribute__((aligned(16))) uint8_t lds[lds_x_bytes<NTMAX>()];
  const int upe = a.H / DN;
  const int wg = xcd_expert_order(static_cast<int>(blockIdx.x), upe * a.nsplit, a.ne);
  const int split = wg % a.nsplit;
  const int rest = wg / a.nsplit;
  const int e = a.e0 + rest / upe, unit = rest % upe;
  const int off_e = clampi(a.offsets[e], 0, a.S);
  const int n_e = clampi(a.offsets[e + 1], off_e, a.S) - off_e;
  if (n_e <= 0) return;
  if (split * a.kb_per_split >= a.F / 128) return;
  // every page of the unit (one, or two when the unit spans pages) must be present
  bool sums = false;
  for (int rb = (unit * DN) / a.R; rb <= (unit * DN + DN - 1) / a.R; ++rb) {
    const int c = fmt_code(a.table[(static_cast<size_t>(e) * 3 + PW_DOWN) * a.nrb_max + rb].bits);
    if (c < 0) return;
    sums = sums || c != 0;
  }
  const int n0 = unit * DN + 16 * RT * __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int code = fmt_code(a.table[(static_cast<size_t>(e) * 3 + PW_DOWN) * a.nrb_max + n0 / a.R].bits);
  if (NTMAX == 1 || n_e <= 16) down_any<ACT, SDT, 1, GK, RT, NW>(code, a, lds, e, off_e, n_e, unit, split, sums);
  else if (NTMAX == 2 || n_e <= 32)
    down_any<ACT, SDT, 2, GK, RT, NW>(code, a, lds, e, off_e, n_e, unit, split, sums);
  else if (n_e <= 48) down_any<ACT, SDT, 3, GK, RT, NW>(code, a, lds, e, off_e, n_e, unit, split, sums);
  else down_any<ACT, SDT, (NTMAX > 2 ? NTMAX : 2), GK, RT, NW>(code, a, lds, e, off_e, n_e, unit, split, sums);
}

// Waves per workgroup: 8 at four slot tiles when the shapes divide into the
// larger units, else 4.
template <int NTMAX> constexpr int waves_for() { return NTMAX == 4 ? 8 : 4; }

template <int ACT, int SDT, int GK, int NTMAX, int NW>
void gemm_launch_nw(const GemmArgs& a, bool gateup, hipStream_t st) {
  constexpr int RT = row_tiles<NTMAX>();
  const dim3 block(64 * NW);
  if (gateup)
    hipLaunchKernelGGL((k_gateup<ACT, SDT, NTMAX, GK, NW>), dim3(a.ne * (a.F / gu_rows<RT, NW>())), block, 0, st, a);
  else
    hipLaunchKernelGGL((k_down<ACT, SDT, NTMAX, GK, NW>), dim3(a.ne * (a.H / dn_rows<RT, NW>()) * a.nsplit), block, 0,
                       st, a);
}

template <int ACT, int SDT, int GK, int NTMAX>
void gemm_launch_nt(const GemmArgs& a, bool gateup, hipStream_t st) {
  constexpr int RT = row_tiles<NTMAX>();
  constexpr int NW = waves_for<NTMAX>();
  if (NW != 4 && a.F % gu_rows<RT, NW>() == 0 && a.H % dn_rows<RT, NW>() == 0)
    gemm_launch_nw<ACT, SDT, GK, NTMAX, NW>(a, gateup, st);
  else
    gemm_launch_nw<ACT, SDT, GK, NTMAX, 4>(a, gateup, st);
}

template <int ACT, int SDT, int GK>
void gemm_launch(const GemmArgs& a, bool gateup, hipStream_t st) {
  if (a.mtb == 1) gemm_launch_nt<ACT, SDT, GK, 1>(a, gateup, st);
  else if (a.mtb == 2) gemm_launch_nt<ACT, SDT, GK, 2>(a, gateup, st);
  else gemm_launch_nt<ACT, SDT, GK, 4>(a, gateup, st);
}

template <int ACT, int SDT>
void gemm_dispatch_g(const GemmArgs& a, bool gateup, hipStream_t st) {
  if (a.G == 64) gemm_launch<ACT, SDT, kG64>(a, gateup, st);
  else if (a.G == 128) gemm_launch<ACT, SDT, kG128>(a, gateup, st);
  else gemm_launch<ACT, SDT, kGBig>(a, gateup, st);
}

hipError_t gemm_dispatch(const GemmArgs& a, bool gateup, hipStream_t st) {
  if (a.mtb != 1 && a.mtb != 2 && a.mtb != 4) return hipErrorInvalidValue;
  if (a.ne <= 0) return hipSuccess;
  if (a.act == PW_BF16) {
    if (a.sdt == PW_BF16) gemm_dispatch_g<PW_BF16, PW_BF16>(a, gateup, st);
    else gemm_dispatch_g<PW_BF16, PW_F16>(a, gateup, st);
  } else {
    if (a.sdt == PW_BF16) gemm_dispatch_g<PW_F16, PW_BF16>(a, gateup, st);
    else gemm_dispatch_g<PW_F16, PW_F16>(a, gateup, st);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gateup(const GemmArgs& a, hipStream_t st) { return gemm_dispatch(a, true, st); }

hipError_t launch_down(const GemmArgs& a, hipStream_t st) { return gemm_dispatch(a, false, st); }

}  // namespace pw
