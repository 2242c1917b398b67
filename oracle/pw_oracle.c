/*
 * CPU oracle for the paged mixed-bitwidth MoE expert forward and the runtime
 * requantization of PagedWeight (arXiv 2607.16184).
 *
 * TEST INFRASTRUCTURE ONLY. Nothing on the product path links, loads or calls
 * this file; only the test suite, the smoke check and the benchmark's CPU
 * baseline leg do. It shares no code, header, table or constant with the HIP
 * library: it is written from the paper and from the documented page format.
 *
 * What it computes, and where the paper defines it:
 *   - router: top-K of E logits per token, weights renormalised over the
 *     selected K (Sec. 2.1, MoE routing);
 *   - routing mass of an expert (Sec. 2.1, Eq. 1);
 *   - expert FFN per routed slot and routing-weighted output accumulation,
 *     reading each linear-block at its committed bitwidth (Sec. 3.3, fused
 *     mixed-precision MoE kernel; Sec. 3.1, one page-table row per block);
 *   - released bytes of a bitwidth reduction, Delta = M^b - M^b' (Sec. 3.1, Eq. 3).
 *
 * The paper's weight format is Any-Precision bit-planes; this build uses
 * asymmetric group-wise round-to-nearest pages instead, which the paper does
 * not describe. The quantizer below is that reading, step by step:
 *   z = largest 16-bit (sdt) value <= min(v); r = fl32(max(v) - z);
 *   r == 0 -> s = +0, all codes 0; else s = smallest sdt value >= fl32(r/Q),
 *   bumped one sdt step if fl32(s*Q) < r; c = clamp(rint(fl32(fl32(v-z)/s)), 0, Q);
 *   dequantized value = fl32(z + c*s).
 * Floating point that decides an integer code is done in fp32, exactly as
 * stated; everything else (FFN, softmax) is fp64.
 *
 * Build: gcc -O2 -std=c11 -fPIC -shared -fopenmp -ffp-contract=off
 */
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define FMT_F16 0
#define FMT_BF16 1

/* ------------------------------------------------------------------------- */
/* 16-bit floating point formats, decoded from the IEEE-754 field definitions */
/* ------------------------------------------------------------------------- */

/* binary16: 1 sign, 5 exponent (bias 15), 10 fraction bits.
 * bfloat16: 1 sign, 8 exponent (bias 127), 7 fraction bits.            */
double or_decode16(uint16_t h, int fmt) {
    int ebits = fmt == FMT_F16 ? 5 : 8;
    int fbits = fmt == FMT_F16 ? 10 : 7;
    int bias = (1 << (ebits - 1)) - 1;
    int sign = (h >> 15) & 1;
    int ex = (h >> fbits) & ((1 << ebits) - 1);
    int fr = h & ((1 << fbits) - 1);
    double v;
    if (ex == (1 << ebits) - 1) {
        v = fr ? NAN : INFINITY;
    } else if (ex == 0) {
        v = ldexp((double)fr, 1 - bias - fbits);             /* subnormal */
    } else {
        v = ldexp((double)((1 << fbits) + fr), ex - bias - fbits);
    }
    return sign ? -v : v;
}

/* All finite values of a format in increasing order, with one bit pattern each
 * (+0 stands for zero). Built once by sorting the decoded patterns.        */
typedef struct { double v; uint16_t bits; } tab_ent;
static tab_ent g_tab[2][65536];
static int g_tab_n[2] = {0, 0};
static double g_dec[2][65536];
static int g_dec_ready[2] = {0, 0};

static int cmp_ent(const void* a, const void* b) {
    double x = ((const tab_ent*)a)->v, y = ((const tab_ent*)b)->v;
    return x < y ? -1 : x > y ? 1 : 0;
}

static void build_tab(int fmt) {
    if (g_tab_n[fmt]) return;
    int n = 0;
    for (int h = 0; h < 65536; ++h) {
        double v = or_decode16((uint16_t)h, fmt);
        if (!isfinite(v)) continue;
        if (v == 0.0 && h != 0) continue;   /* keep +0 only */
        g_tab[fmt][n].v = v;
        g_tab[fmt][n].bits = (uint16_t)h;
        ++n;
    }
    qsort(g_tab[fmt], n, sizeof(tab_ent), cmp_ent);
    g_tab_n[fmt] = n;
}

static const double* dec_table(int fmt) {
    if (!g_dec_ready[fmt]) {
        for (int h = 0; h < 65536; ++h) g_dec[fmt][h] = or_decode16((uint16_t)h, fmt);
        g_dec_ready[fmt] = 1;
    }
    return g_dec[fmt];
}

/* index of the largest table value <= x (x finite, within range) */
static int tab_floor(int fmt, double x) {
    build_tab(fmt);
    int lo = 0, hi = g_tab_n[fmt] - 1;
    if (x < g_tab[fmt][0].v) return -1;
    while (lo < hi) {
        int mid = (lo + hi + 1) / 2;
        if (g_tab[fmt][mid].v <= x) lo = mid; else hi = mid - 1;
    }
    return lo;
}

/* largest representable value <= x */
uint16_t or_round_down16(float x, int fmt) {
    int i = tab_floor(fmt, (double)x);
    return g_tab[fmt][i < 0 ? 0 : i].bits;
}

/* smallest representable value >= x */
uint16_t or_round_up16(float x, int fmt) {
    int i = tab_floor(fmt, (double)x);
    if (i >= 0 && g_tab[fmt][i].v == (double)x) return g_tab[fmt][i].bits;
    int j = i + 1;
    if (j >= g_tab_n[fmt]) j = g_tab_n[fmt] - 1;
    return g_tab[fmt][j].bits;
}

/* next representable value above the value of h */
uint16_t or_next_up16(uint16_t h, int fmt) {
    double v = or_decode16(h, fmt);
    int i = tab_floor(fmt, v);
    int j = i + 1;
    if (j >= g_tab_n[fmt]) j = g_tab_n[fmt] - 1;
    return g_tab[fmt][j].bits;
}

/* nearest representable value, ties to the even bit pattern */
uint16_t or_round_nearest16(double x, int fmt) {
    build_tab(fmt);
    int i = tab_floor(fmt, x);
    if (i < 0) return g_tab[fmt][0].bits;
    if (i == g_tab_n[fmt] - 1 || g_tab[fmt][i].v == x) return g_tab[fmt][i].bits;
    double a = g_tab[fmt][i].v, b = g_tab[fmt][i + 1].v;
    double da = x - a, db = b - x;
    if (da < db) return g_tab[fmt][i].bits;
    if (db < da) return g_tab[fmt][i + 1].bits;
    /* exact tie: the pattern with an even last fraction bit */
    return (g_tab[fmt][i].bits & 1) ? g_tab[fmt][i + 1].bits : g_tab[fmt][i].bits;
}

/* Threads an OpenMP region of the oracle uses (1 without OpenMP). */
int or_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Set the threads later OpenMP regions of the oracle use (timing only). */
void or_set_threads(int n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Build the lookup tables of both formats (call once before any threads). */
void or_init(void) {
    build_tab(FMT_F16);
    build_tab(FMT_BF16);
    dec_table(FMT_F16);
    dec_table(FMT_BF16);
}

/* ------------------------------------------------------------------------- */
/* Group-wise asymmetric round-to-nearest quantizer and its inverse          */
/* ------------------------------------------------------------------------- */

/* Quantize n fp32 values to `bits` (8 or 4) with one (scale, zero) pair in
 * format sdt. Writes n codes, the scale and zero bit patterns.            */
void or_quantize_group(const float* v, int n, int bits, int sdt,
                       uint8_t* codes, uint16_t* s_out, uint16_t* z_out) {
    const int Q = (1 << bits) - 1;
    float lo = v[0], hi = v[0];
    for (int j = 1; j < n; ++j) {
        if (v[j] < lo) lo = v[j];
        if (v[j] > hi) hi = v[j];
    }
    uint16_t zb = or_round_down16(lo, sdt);
    float z = (float)or_decode16(zb, sdt);
    float r = hi - z;
    if (r == 0.0f) {
        *s_out = 0;
        *z_out = zb;
        for (int j = 0; j < n; ++j) codes[j] = 0;
        return;
    }
    float s0 = r / (float)Q;
    uint16_t sb = or_round_up16(s0, sdt);
    float s = (float)or_decode16(sb, sdt);
    if (s * (float)Q < r) {
        sb = or_next_up16(sb, sdt);
        s = (float)or_decode16(sb, sdt);
    }
    for (int j = 0; j < n; ++j) {
        float d = v[j] - z;
        float q = d / s;
        float c = rintf(q);
        if (c < 0.0f) c = 0.0f;
        if (c > (float)Q) c = (float)Q;
        codes[j] = (uint8_t)c;
    }
    *s_out = sb;
    *z_out = zb;
}

/* fl32(z + c*s); the product c*s is exact in fp32 */
float or_dequant(uint8_t c, uint16_t s, uint16_t z, int sdt) {
    float sf = (float)or_decode16(s, sdt);
    float zf = (float)or_decode16(z, sdt);
    float p = (float)c * sf;
    return zf + p;
}

/* Quantize an R x K page given as fp32 values (row-major) into unpacked codes
 * [R][K] and scale/zero [R][K/G].                                          */
void or_quantize_page_f32(const float* v, int R, int K, int G, int bits, int sdt,
                          uint8_t* codes, uint16_t* s, uint16_t* z) {
    int ng = K / G;
    for (int r = 0; r < R; ++r)
        for (int g = 0; g < ng; ++g)
            or_quantize_group(v + (size_t)r * K + (size_t)g * G, G, bits, sdt,
                              codes + (size_t)r * K + (size_t)g * G,
                              s + (size_t)r * ng + g, z + (size_t)r * ng + g);
}

/* Quantize a page of 16-bit values (format fmt16). */
void or_quantize_page16(const uint16_t* w16, int fmt16, int R, int K, int G, int bits,
                        int sdt, uint8_t* codes, uint16_t* s, uint16_t* z) {
    float* v = (float*)malloc(sizeof(float) * (size_t)R * K);
    for (size_t i = 0; i < (size_t)R * K; ++i) v[i] = (float)or_decode16(w16[i], fmt16);
    or_quantize_page_f32(v, R, K, G, bits, sdt, codes, s, z);
    free(v);
}

/* Requantize a quantized page (bits_in) to bits_out < bits_in: the source
 * values are its dequantized fp32 values, then the quantizer runs again.   */
void or_requant_page(const uint8_t* codes_in, const uint16_t* s_in, const uint16_t* z_in,
                     int R, int K, int G, int sdt, int bits_out,
                     uint8_t* codes_out, uint16_t* s_out, uint16_t* z_out) {
    int ng = K / G;
    float* v = (float*)malloc(sizeof(float) * (size_t)R * K);
    for (int r = 0; r < R; ++r)
        for (int k = 0; k < K; ++k) {
            size_t gi = (size_t)r * ng + k / G;
            v[(size_t)r * K + k] = or_dequant(codes_in[(size_t)r * K + k], s_in[gi], z_in[gi], sdt);
        }
    or_quantize_page_f32(v, R, K, G, bits_out, sdt, codes_out, s_out, z_out);
    free(v);
}

/* ------------------------------------------------------------------------- */
/* Page byte format (pool layout) -- encoder and decoder                      */
/* ------------------------------------------------------------------------- */
/*
 * A page of R rows x K values is cut into tiles of 16 rows x 128 values
 * (tile (tau, beta): rows [16 tau, 16 tau + 16), values [128 beta, 128 beta +
 * 128)), stored in the order tau-major, beta-minor. Inside a tile, value
 * (r, k) with lc = r mod 16, i = (k mod 128) div 32, lg = (k mod 32) div 8,
 * q = k mod 8 belongs to "lane" l = 16 lg + lc and "step" i:
 *   16-bit: tile of 4096 bytes; value at byte 1024 i + 16 l + 2 q.
 *   8-bit : tile of 2048 bytes; code at byte 1024 (i div 2) + 16 l + 8 (i mod 2) + q.
 *   4-bit : tile of 1024 bytes; code in the little-endian 32-bit word at byte
 *           16 l + 4 i, at bits [4t, 4t+4) if q = 2t and [16+4t, 20+4t) if q = 2t+1.
 * 8/4-bit pages are followed by the scale/zero block: for group g (K/G of
 * them) and row r, the pair (scale, zero) as two 16-bit values at pair index
 * g R + r.
 * Page bytes: M16 = 2RK, M8 = RK + 4R(K/G), M4 = RK/2 + 4R(K/G).
 */

uint64_t or_page_bytes(int R, int K, int G, int bits) {
    uint64_t rk = (uint64_t)R * K, sz = 4ull * R * (K / G);
    if (bits == 16) return 2 * rk;
    if (bits == 8) return rk + sz;
    return rk / 2 + sz;
}

/* Eq. 3: bytes released when a block goes from b to b' (b' < b). */
uint64_t or_delta_bytes(int R, int K, int G, int b, int bp) {
    return or_page_bytes(R, K, G, b) - or_page_bytes(R, K, G, bp);
}

/* Byte offset of value (r, k) in the code/value block, and for 4-bit codes
 * the bit position inside the 32-bit word starting at that offset. */
static uint64_t value_offset(int K, int bits, int r, int k, int* bitpos) {
    int tau = r / 16, lc = r % 16, beta = k / 128;
    int i = (k % 128) / 32, lg = (k % 32) / 8, q = k % 8, l = 16 * lg + lc;
    uint64_t tile = (uint64_t)tau * (K / 128) + beta;
    *bitpos = 0;
    if (bits == 16) return tile * 4096 + 1024 * i + 16 * l + 2 * q;
    if (bits == 8) return tile * 2048 + 1024 * (i / 2) + 16 * l + 8 * (i % 2) + q;
    *bitpos = (q % 2) ? 16 + 4 * (q / 2) : 4 * (q / 2);
    return tile * 1024 + 16 * l + 4 * i;
}

void or_encode_page16(const uint16_t* w16, int R, int K, uint8_t* out) {
    int bp;
    for (int r = 0; r < R; ++r)
        for (int k = 0; k < K; ++k) {
            uint64_t o = value_offset(K, 16, r, k, &bp);
            uint16_t v = w16[(size_t)r * K + k];
            out[o] = (uint8_t)(v & 255);
            out[o + 1] = (uint8_t)(v >> 8);
        }
}

void or_decode_page16(const uint8_t* in, int R, int K, uint16_t* w16) {
    int bp;
    for (int r = 0; r < R; ++r)
        for (int k = 0; k < K; ++k) {
            uint64_t o = value_offset(K, 16, r, k, &bp);
            w16[(size_t)r * K + k] = (uint16_t)(in[o] | (in[o + 1] << 8));
        }
}

void or_encode_page(const uint8_t* codes, const uint16_t* s, const uint16_t* z,
                    int R, int K, int G, int bits, uint8_t* out) {
    int ng = K / G, bp;
    size_t code_bytes = bits == 8 ? (size_t)R * K : (size_t)R * K / 2;
    memset(out, 0, code_bytes);
    for (int r = 0; r < R; ++r)
        for (int k = 0; k < K; ++k) {
            uint64_t o = value_offset(K, bits, r, k, &bp);
            uint8_t c = codes[(size_t)r * K + k];
            if (bits == 8) {
                out[o] = c;
            } else {
                uint32_t w = (uint32_t)out[o] | ((uint32_t)out[o + 1] << 8) |
                             ((uint32_t)out[o + 2] << 16) | ((uint32_t)out[o + 3] << 24);
                w |= (uint32_t)(c & 15) << bp;
                for (int b = 0; b < 4; ++b) out[o + b] = (uint8_t)(w >> (8 * b));
            }
        }
    uint8_t* szp = out + code_bytes;
    for (int g = 0; g < ng; ++g)
        for (int r = 0; r < R; ++r) {
            size_t pi = (size_t)g * R + r;
            uint16_t sv = s[(size_t)r * ng + g], zv = z[(size_t)r * ng + g];
            szp[4 * pi + 0] = (uint8_t)(sv & 255);
            szp[4 * pi + 1] = (uint8_t)(sv >> 8);
            szp[4 * pi + 2] = (uint8_t)(zv & 255);
            szp[4 * pi + 3] = (uint8_t)(zv >> 8);
        }
}

void or_decode_page(const uint8_t* in, int R, int K, int G, int bits,
                    uint8_t* codes, uint16_t* s, uint16_t* z) {
    int ng = K / G, bp;
    size_t code_bytes = bits == 8 ? (size_t)R * K : (size_t)R * K / 2;
    for (int r = 0; r < R; ++r)
        for (int k = 0; k < K; ++k) {
            uint64_t o = value_offset(K, bits, r, k, &bp);
            uint8_t c;
            if (bits == 8) {
                c = in[o];
            } else {
                uint32_t w = (uint32_t)in[o] | ((uint32_t)in[o + 1] << 8) |
                             ((uint32_t)in[o + 2] << 16) | ((uint32_t)in[o + 3] << 24);
                c = (uint8_t)((w >> bp) & 15);
            }
            codes[(size_t)r * K + k] = c;
        }
    const uint8_t* szp = in + code_bytes;
    for (int g = 0; g < ng; ++g)
        for (int r = 0; r < R; ++r) {
            size_t pi = (size_t)g * R + r;
            s[(size_t)r * ng + g] = (uint16_t)(szp[4 * pi] | (szp[4 * pi + 1] << 8));
            z[(size_t)r * ng + g] = (uint16_t)(szp[4 * pi + 2] | (szp[4 * pi + 3] << 8));
        }
}

/* ------------------------------------------------------------------------- */
/* Router and token permutation                                              */
/* ------------------------------------------------------------------------- */

/* Per token: the K experts with the largest logits (ties to the lower index),
 * and their routing weights. renorm=1: softmax over the selected K logits;
 * renorm=0: the full softmax probability of each selected expert.          */
void or_route(const float* logits, int T, int E, int K, int renorm,
              int32_t* ids, double* w) {
    char* taken = (char*)malloc((size_t)E);
    for (int t = 0; t < T; ++t) {
        const float* l = logits + (size_t)t * E;
        memset(taken, 0, (size_t)E);
        for (int k = 0; k < K; ++k) {
            int best = -1;
            for (int e = 0; e < E; ++e) {
                if (taken[e]) continue;
                if (best < 0 || l[e] > l[best]) best = e;
            }
            taken[best] = 1;
            ids[(size_t)t * K + k] = best;
        }
        double m = (double)l[ids[(size_t)t * K]];
        double denom = 0.0;
        if (renorm) {
            for (int k = 0; k < K; ++k) denom += exp((double)l[ids[(size_t)t * K + k]] - m);
        } else {
            for (int e = 0; e < E; ++e) denom += exp((double)l[e] - m);
        }
        for (int k = 0; k < K; ++k)
            w[(size_t)t * K + k] = exp((double)l[ids[(size_t)t * K + k]] - m) / denom;
    }
    free(taken);
}

/* Group the T*K routed slots (slot s = t*K + k) by expert: expert-major, and
 * in increasing slot order within an expert.                               */
void or_permute(const int32_t* ids, int T, int K, int E, int32_t* counts,
                int32_t* offsets, int32_t* sorted_slot, int32_t* slot_pos) {
    int S = T * K, i = 0;
    for (int e = 0; e < E; ++e) {
        counts[e] = 0;
        offsets[e] = i;
        for (int s = 0; s < S; ++s)
            if (ids[s] == e) {
                sorted_slot[i++] = s;
                counts[e]++;
            }
    }
    offsets[E] = i;
    for (int j = 0; j < S; ++j) slot_pos[sorted_slot[j]] = j;
}

/* Eq. 1: routing mass of each expert, sum of its routing weights over the
 * sum of all routing weights.                                               */
void or_routing_mass(const int32_t* ids, const double* w, int T, int K, int E, double* mass) {
    double total = 0.0;
    for (int e = 0; e < E; ++e) mass[e] = 0.0;
    for (int t = 0; t < T; ++t)
        for (int k = 0; k < K; ++k) {
            mass[ids[(size_t)t * K + k]] += w[(size_t)t * K + k];
            total += w[(size_t)t * K + k];
        }
    for (int e = 0; e < E; ++e) mass[e] /= total;
}

/* ------------------------------------------------------------------------- */
/* Paged MoE expert forward                                                  */
/* ------------------------------------------------------------------------- */

/* One projection of all experts: `rows` x `cols` per expert.
 *   w16:   16-bit values [E][rows][cols] (used where the page is 16-bit)
 *   bits:  committed bitwidth per page [E][rows/R]
 *   codes: unpacked codes [E][rows][cols] (used where the page is 8/4-bit)
 *   s, z:  scale/zero bit patterns [E][rows][cols/G]                        */
typedef struct {
    const uint16_t* w16;
    const int32_t* bits;
    const uint8_t* codes;
    const uint16_t* s;
    const uint16_t* z;
    int rows, cols;
    uint16_t* wr;   /* w_round: each quantized weight rounded once, or NULL */
} or_proj;

/* dot(row n of expert e's projection, v) with the weight read at its page's
 * committed bitwidth: the 16-bit value, or z + c*s (exact in fp64). With
 * w_round=1 a quantized weight is instead first rounded to fp32 and then to
 * the activation format (round to nearest even both times): the value a
 * kernel feeds to a 16-bit matrix unit after dequantizing in fp32.         */
/* The weight of row n, column j of a quantized page: z + c*s (exact in fp64). */
static double quant_weight(const or_proj* P, int e, int n, int j, int G, const double* dsdt) {
    int ng = P->cols / G;
    size_t base = ((size_t)e * P->rows + n) * P->cols;
    size_t sb = ((size_t)e * P->rows + n) * ng;
    return dsdt[P->z[sb + j / G]] + (double)P->codes[base + j] * dsdt[P->s[sb + j / G]];
}

/* The w_round reading of a quantized weight: rounded to fp32, then to the
 * activation format (round to nearest even both times), as a bit pattern. */
static uint16_t rounded_weight(const or_proj* P, int e, int n, int j, int G, const double* dsdt, int act) {
    return or_round_nearest16((double)(float)quant_weight(P, e, n, j, G, dsdt), act);
}

static double proj_row_dot(const or_proj* P, int e, int n, const double* v, int R, int G,
                           const double* d16, const double* dsdt, int w_round, int act) {
    int b = P->bits[(size_t)e * (P->rows / R) + n / R];
    size_t base = ((size_t)e * P->rows + n) * P->cols;
    double acc = 0.0;
    if (b == 16) {
        const uint16_t* w = P->w16 + base;
        for (int j = 0; j < P->cols; ++j) acc += d16[w[j]] * v[j];
    } else if (w_round && P->wr) {
        const uint16_t* w = P->wr + base;
        for (int j = 0; j < P->cols; ++j) acc += d16[w[j]] * v[j];
    } else {
        for (int j = 0; j < P->cols; ++j) {
            double wv = quant_weight(P, e, n, j, G, dsdt);
            if (w_round) wv = or_decode16(rounded_weight(P, e, n, j, G, dsdt, act), act);
            acc += wv * v[j];
        }
    }
    return acc;
}

/* w_round: every quantized weight of the experts in `used` rounded once up
 * front (the same values proj_row_dot would round per token), or NULL when
 * the memory is not there (proj_row_dot then rounds as it goes).           */
static uint16_t* round_all(const or_proj* P, const unsigned char* used, int E, int R, int G,
                           const double* dsdt, int act) {
    uint16_t* wr = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)E * P->rows * P->cols);
    if (!wr) return NULL;
    for (int e = 0; e < E; ++e) {
        if (!used[e]) continue;
#pragma omp parallel for schedule(static)
        for (int n = 0; n < P->rows; ++n) {
            if (P->bits[(size_t)e * (P->rows / R) + n / R] == 16) continue;
            uint16_t* w = wr + ((size_t)e * P->rows + n) * P->cols;
            for (int j = 0; j < P->cols; ++j) w[j] = rounded_weight(P, e, n, j, G, dsdt, act);
        }
    }
    return wr;
}

/* y[t] = sum_k w[t,k] * down_e( silu(gate_e(x_t)) * up_e(x_t) ), e = ids[t,k],
 * for the tokens listed in `tok` (n_tok of them). fp64 throughout; with
 * h_round=1 the SwiGLU output is rounded to the activation format before the
 * down projection; w_round as in proj_row_dot. y is [T][H] and only the
 * listed rows are written.                                                  */
void or_moe_forward(const uint16_t* x16, int T, int H, int F, int E, int K, int R, int G,
                    int act, int sdt, const int32_t* ids, const double* w,
                    const uint16_t* g16, const int32_t* gbits, const uint8_t* gcodes,
                    const uint16_t* gs, const uint16_t* gz,
                    const uint16_t* u16, const int32_t* ubits, const uint8_t* ucodes,
                    const uint16_t* us, const uint16_t* uz,
                    const uint16_t* d16w, const int32_t* dbits, const uint8_t* dcodes,
                    const uint16_t* ds, const uint16_t* dz,
                    int h_round, int w_round, const int32_t* tok, int n_tok, double* y) {
    (void)T;
    or_init();
    const double* d16 = dec_table(act);
    const double* dsdt = dec_table(sdt);
    or_proj PG = {g16, gbits, gcodes, gs, gz, F, H, NULL};
    or_proj PU = {u16, ubits, ucodes, us, uz, F, H, NULL};
    or_proj PD = {d16w, dbits, dcodes, ds, dz, H, F, NULL};
    if (w_round) {
        unsigned char* used = (unsigned char*)calloc((size_t)E, 1);
        if (used) {
            for (int ti = 0; ti < n_tok; ++ti)
                for (int k = 0; k < K; ++k) used[ids[(size_t)tok[ti] * K + k]] = 1;
            PG.wr = round_all(&PG, used, E, R, G, dsdt, act);
            PU.wr = round_all(&PU, used, E, R, G, dsdt, act);
            PD.wr = round_all(&PD, used, E, R, G, dsdt, act);
            free(used);
        }
    }
    double* xv = (double*)malloc(sizeof(double) * H);
    double* h = (double*)malloc(sizeof(double) * F);
    double* o = (double*)malloc(sizeof(double) * H);
    for (int ti = 0; ti < n_tok; ++ti) {
        int t = tok[ti];
        for (int j = 0; j < H; ++j) xv[j] = d16[x16[(size_t)t * H + j]];
        for (int n = 0; n < H; ++n) y[(size_t)t * H + n] = 0.0;
        for (int k = 0; k < K; ++k) {
            int e = ids[(size_t)t * K + k];
#pragma omp parallel for schedule(static)
            for (int f = 0; f < F; ++f) {
                double gv = proj_row_dot(&PG, e, f, xv, R, G, d16, dsdt, w_round, act);
                double uv = proj_row_dot(&PU, e, f, xv, R, G, d16, dsdt, w_round, act);
                double hv = gv / (1.0 + exp(-gv)) * uv;
                if (h_round) hv = or_decode16(or_round_nearest16(hv, act), act);
                h[f] = hv;
            }
#pragma omp parallel for schedule(static)
            for (int n = 0; n < H; ++n)
                o[n] = proj_row_dot(&PD, e, n, h, R, G, d16, dsdt, w_round, act);
            double wk = w[(size_t)t * K + k];
            for (int n = 0; n < H; ++n) y[(size_t)t * H + n] += wk * o[n];
        }
    }
    free(xv);
    free(h);
    free(o);
    free(PG.wr);
    free(PU.wr);
    free(PD.wr);
}
