/*
 * ssmq_oracle.c -- reference oracle for the quantized selective-state update.
 *
 * TEST INFRASTRUCTURE. This is a plain, slow, deliberately obvious CPU statement
 * of what the GPU library computes. Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load it; the product path never does. It
 * shares no code, header, table or constant with the HIP library.
 *
 * Paper: "Low-Discrepancy Dither for Quantized Recurrent State Caches".
 *
 * Representation choices (on purpose different from any bit-level trick):
 *   - every storage format is its sorted set of finite values, built by decoding
 *     each code from the format's definition (sign, exponent, mantissa fields);
 *   - rounding is a neighbour search in that set followed by the threshold test
 *     of eq. (dither), carried out with exact double-precision comparisons;
 *   - thresholds are the 32-bit Weyl accumulator of Appendix B ("Dithers",
 *     hardware form), a keyed integer hash for stochastic rounding, and the
 *     Philox4x32-10 counter-based generator for stochastic rounding.
 *
 * Floating-point order of the fused step (fp32, no contraction; this file must
 * be compiled with -ffp-contract=off):
 *   z      = fl32(dt * A)
 *   dA     = fl32(exp(z))                    (exp in double, then one rounding)
 *   dx     = fl32(dt * x_p)
 *   w      = fl32(dx * B_n)
 *   h_prev = decode(code)                    fp16 / bf16 / fp32: the code's value
 *          = fl32(v * s_old)                 E4M3, INT8, INT4: the code's value v
 *                                            times its group's old scale, in fp32
 *                                            (every format is simulated in FP32,
 *                                            Appendix B "Formats")
 *   h_new  = fma(dA, h_prev, w)              (one rounding)
 *   y_p    = sum_n C_n h_new + D x_p         (accumulated in double)
 * then h_new is written back under the chosen rounding rule.
 */
#include <float.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------- */
/* Identifiers (the oracle's own numbering; the Python wrapper maps names).  */
/* ------------------------------------------------------------------------- */
enum { ORC_FP16 = 0, ORC_BF16 = 1, ORC_E4M3 = 2, ORC_FP32 = 3, ORC_INT8 = 4, ORC_INT4 = 5 };
#define ORC_NFMT 6

/* Symmetric integer formats with a block scale (Section 2 "Low-precision
 * storage"; Appendix B "Formats"): INTb stores integers in [-qmax, qmax],
 * qmax = 2^(b-1) - 1, two's complement; INT4 packs two entries per byte, the
 * even entry in the low nibble. */
static int is_int(int f) { return f == ORC_INT8 || f == ORC_INT4; }
static int int_qmax(int f) { return f == ORC_INT8 ? 127 : 7; }
static int is_scaled(int f) { return f == ORC_E4M3 || is_int(f); }
enum { ORC_RTN = 0, ORC_SR = 1, ORC_WEYL = 2, ORC_PHILOX = 3 };

/* ------------------------------------------------------------------------- */
/* Storage formats as value sets (Section 2 "Low-precision storage";          */
/* Appendix B "Formats").                                                     */
/* ------------------------------------------------------------------------- */
typedef struct {
    int bits;          /* code width                                   */
    int ebits, mbits;  /* exponent / mantissa field widths             */
    int bias;          /* exponent bias                                */
    int ieee_special;  /* 1: all-ones exponent is Inf/NaN (fp16, bf16) */
                       /* 0: only S.1111.111 is NaN, no Inf (E4M3FN)   */
} fmt_def;

static const fmt_def FMT[3] = {
    {16, 5, 10, 15, 1},  /* IEEE binary16                        */
    {16, 8, 7, 127, 1},  /* bfloat16                             */
    {8, 4, 3, 7, 0},     /* OCP FP8 E4M3FN: max 448, no infinity */
};

/* Value of a code from the format definition. NaN codes give NaN. */
static double decode_fields(int f, uint32_t code) {
    const fmt_def *d = &FMT[f];
    uint32_t sign = (code >> (d->bits - 1)) & 1u;
    uint32_t e = (code >> d->mbits) & ((1u << d->ebits) - 1u);
    uint32_t m = code & ((1u << d->mbits) - 1u);
    uint32_t emax_field = (1u << d->ebits) - 1u;
    double v;
    if (d->ieee_special && e == emax_field) {
        v = (m == 0) ? INFINITY : NAN;
    } else if (!d->ieee_special && e == emax_field && m == (1u << d->mbits) - 1u) {
        v = NAN;
    } else if (e == 0) {
        v = ldexp((double)m, 1 - d->bias - d->mbits);            /* subnormal */
    } else {
        v = ldexp((double)((1u << d->mbits) + m), (int)e - d->bias - d->mbits);
    }
    return sign ? -v : v;
}

/*
 * The grid of a format: all finite values, ascending, one entry for zero. For
 * fp16/bf16 the grid is extended by one point on each side, max + top step,
 * whose code is the infinity of that sign: this is how a cast overflows, and
 * it is the upper neighbour of values just beyond the largest finite value.
 */
typedef struct {
    int n;
    double *val;
    uint32_t *code;
    uint32_t pos_zero, neg_zero, pos_nan, neg_nan;
    double max_finite;
} grid_t;

static grid_t GRID[3];
static int grid_ready = 0;

static int cmp_double_code(const void *a, const void *b) {
    const double *x = (const double *)a, *y = (const double *)b;
    return (*x > *y) - (*x < *y);
}

static void build_grid(int f) {
    const fmt_def *d = &FMT[f];
    uint32_t ncodes = 1u << d->bits;
    /* pairs (value, code) packed as two doubles for qsort */
    double *pairs = (double *)malloc(sizeof(double) * 2 * (ncodes + 2));
    int n = 0;
    double maxf = 0.0;
    uint32_t pinf = 0, ninf = 0;
    grid_t *g = &GRID[f];
    g->pos_zero = 0;
    g->neg_zero = 1u << (d->bits - 1);
    for (uint32_t c = 0; c < ncodes; ++c) {
        double v = decode_fields(f, c);
        if (isnan(v)) continue;
        if (isinf(v)) {
            if (v > 0) pinf = c; else ninf = c;
            continue;
        }
        if (v == 0.0 && c != g->pos_zero) continue; /* one zero entry (+0) */
        if (v > maxf) maxf = v;
        pairs[2 * n] = v;
        pairs[2 * n + 1] = (double)c;
        ++n;
    }
    if (d->ieee_special) {
        /* step between the two largest finite values */
        uint32_t maxcode = pinf - 1u;
        double top_step = decode_fields(f, maxcode) - decode_fields(f, maxcode - 1u);
        pairs[2 * n] = maxf + top_step; pairs[2 * n + 1] = (double)pinf; ++n;
        pairs[2 * n] = -(maxf + top_step); pairs[2 * n + 1] = (double)ninf; ++n;
    }
    qsort(pairs, (size_t)n, sizeof(double) * 2, cmp_double_code);
    g->n = n;
    g->val = (double *)malloc(sizeof(double) * (size_t)n);
    g->code = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)n);
    for (int i = 0; i < n; ++i) {
        g->val[i] = pairs[2 * i];
        g->code[i] = (uint32_t)pairs[2 * i + 1];
    }
    g->max_finite = maxf;
    /* canonical quiet NaN codes */
    if (f == ORC_FP16) { g->pos_nan = 0x7E00u; g->neg_nan = 0xFE00u; }
    if (f == ORC_BF16) { g->pos_nan = 0x7FC0u; g->neg_nan = 0xFFC0u; }
    if (f == ORC_E4M3) { g->pos_nan = 0x7Fu; g->neg_nan = 0xFFu; }
    free(pairs);
}

static void ensure_grids(void) {
    if (grid_ready) return;
    for (int f = 0; f < 3; ++f) build_grid(f);
    grid_ready = 1;
}

/* index of the largest grid value <= x (x within the grid's range) */
static int floor_index(const grid_t *g, double x) {
    int lo = 0, hi = g->n - 1;
    while (lo < hi) {
        int mid = lo + (hi - lo + 1) / 2;
        if (g->val[mid] <= x) lo = mid; else hi = mid - 1;
    }
    return lo;
}

static uint32_t f32_bits(float x) { uint32_t u; memcpy(&u, &x, 4); return u; }
static float bits_f32(uint32_t u) { float x; memcpy(&x, &u, 4); return x; }

/*
 * Round the fp32 value x into format f.
 *
 * Eq. (dither): Q_u(x) = s * floor(x / s + u), applied on the local grid
 * (Appendix B "Formats"). With lo <= x < hi the neighbouring grid values and
 * s = hi - lo, floor(x/s + u) picks hi exactly when x + u*s >= hi, i.e. when x
 * lies at or above the point hi - u*s. That point and the comparison are exact
 * in double (hi has at most 12 significant bits, u*s at most 24).
 *
 * RTN: nearest neighbour, exact ties to the even code (the hardware cast).
 * E4M3: x is first clamped to [-448, 448] (saturation, Appendix B "Formats").
 * A result of zero keeps the sign of x; NaN gives the canonical NaN code.
 */
static uint32_t round_to_format(int f, int rule, float xf, uint32_t U24) {
    const grid_t *g = &GRID[f];
    int neg = signbit(xf) != 0;
    if (isnan(xf)) return neg ? g->neg_nan : g->pos_nan;
    double x = (double)xf;
    if (f == ORC_E4M3) {
        if (x > g->max_finite) x = g->max_finite;
        if (x < -g->max_finite) x = -g->max_finite;
    } else {
        /* at or beyond the overflow point: infinity of the sign of x */
        if (x >= g->val[g->n - 1]) return g->code[g->n - 1];
        if (x <= g->val[0]) return g->code[0];
    }
    int k = floor_index(g, x);
    double lo = g->val[k];
    int pick;
    if (lo == x) {
        pick = k;
    } else {
        double hi = g->val[k + 1];
        if (rule == ORC_RTN) {
            double mid = 0.5 * (lo + hi);
            if (x < mid) pick = k;
            else if (x > mid) pick = k + 1;
            else pick = ((g->code[k] & 1u) == 0) ? k : k + 1;
        } else {
            double u = (double)U24 / 16777216.0;   /* u = U / 2^24 */
            pick = (x >= hi - u * (hi - lo)) ? k + 1 : k;
        }
    }
    if (g->val[pick] == 0.0) return neg ? g->neg_zero : g->pos_zero;
    return g->code[pick];
}

/*
 * Round the scaled fp32 value q onto the integer lattice {-qmax, ..., qmax}:
 * eq. (dither) with step 1, lo = floor(q) and hi = lo + 1 (exact in double, as
 * is hi - u for a 24-bit u). Values are clamped to [-qmax, qmax] first
 * (Appendix B "Formats"); the bounds are lattice points, so clamping before
 * or after rounding gives the same integer. RTN: nearest, exact ties to the
 * even integer (the same tie rule as the floating-point casts). NaN has no
 * integer code and is stored as 0. Returns the signed integer.
 */
static int32_t round_to_int(int qmax, int rule, float qf, uint32_t U24) {
    if (isnan(qf)) return 0;
    double x = (double)qf;
    if (x > qmax) x = qmax;
    if (x < -qmax) x = -qmax;
    double lo = floor(x);
    if (lo == x) return (int32_t)lo;
    double hi = lo + 1.0;
    if (rule == ORC_RTN) {
        double mid = lo + 0.5;
        if (x < mid) return (int32_t)lo;
        if (x > mid) return (int32_t)hi;
        return (fmod(lo, 2.0) == 0.0) ? (int32_t)lo : (int32_t)hi;
    }
    double u = (double)U24 / 16777216.0;
    return (x >= hi - u) ? (int32_t)hi : (int32_t)lo;
}

/* storage code of one integer entry (byte for INT8, nibble for INT4) and back */
static uint32_t int_code(int f, int32_t k) { return (uint32_t)k & (f == ORC_INT8 ? 0xFFu : 0xFu); }
static int32_t int_value(int f, uint32_t code) {
    if (f == ORC_INT8) return (int32_t)(int8_t)(uint8_t)code;
    code &= 0xFu;
    return (code & 0x8u) ? (int32_t)code - 16 : (int32_t)code;
}

/* ------------------------------------------------------------------------- */
/* Thresholds.                                                                */
/* ------------------------------------------------------------------------- */

/*
 * Weyl dither, hardware form (Appendix B "Dithers"): a 32-bit accumulator
 *   acc = A (r+1) + B (c+1) + L l + S sigma + t Phi   (mod 2^32),
 * whose top 24 bits are the threshold. A, B, L, S are the decimal constants of
 * the float form times 2^32, rounded to the nearest integer; Phi is the 32-bit
 * golden increment (Section 6.4 "Three silent pitfalls", Observation "Space-time aliasing").
 * r = i / block, c = i % block for the flat entry index i.
 */
static uint32_t W_A, W_B, W_L, W_S;
static const uint32_t W_PHI = 2654435769u;

static uint32_t from_unit(double frac) { return (uint32_t)llround(frac * 4294967296.0); }

static void ensure_weyl_constants(void) {
    W_A = from_unit(0.7548776662);
    W_B = from_unit(0.5698402910);
    W_L = from_unit(0.1234567);
    W_S = from_unit(0.3141592);
}

static uint32_t weyl_acc(uint64_t i, uint64_t block, uint32_t layer, uint32_t seed, uint32_t t) {
    uint64_t r = i / block, c = i % block;
    uint32_t acc = W_A * (uint32_t)(r + 1u) + W_B * (uint32_t)(c + 1u) + W_L * layer +
                   W_S * seed + W_PHI * t;
    return acc;
}

/*
 * Stochastic rounding by an integer hash (Appendix B "Decode regime", hash SR):
 * fmix32 is the MurmurHash3 32-bit finalizer; 0x9E3779B1 and 0x85EBCA77 are the
 * entry and step multipliers the paper gives. The elided remainder of the
 * paper's pre-hash is read as a per-(seed, layer, step) key, hashed before it
 * meets the entry term, so that each step draws a fresh bijection of entries.
 * The threshold is the top 24 bits of the hash.
 */
static uint32_t fmix32(uint32_t h) {
    h ^= h >> 16;
    h *= 0x85EBCA6Bu;
    h ^= h >> 13;
    h *= 0xC2B2AE35u;
    h ^= h >> 16;
    return h;
}

static uint32_t sr_key(uint32_t seed, uint32_t layer, uint32_t t) {
    uint32_t k = fmix32(seed);
    k = fmix32(k ^ (layer * 0xC2B2AE3Du));
    k = fmix32(k ^ (t * 0x85EBCA77u));
    return k;
}

/*
 * Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as
 * easy as 1, 2, 3", SC 2011), the counter-based generator behind the paper's SR
 * (Appendix B "Dithers": torch.rand and tl.rand). Ten rounds on a counter of
 * four 32-bit words under a two-word key; each round multiplies words 0 and 2
 * by the round constants, mixes the high halves with the other words and the
 * key, and the key is advanced by the Weyl increments between rounds.
 */
static void philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int r = 0; r < 10; ++r) {
        const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        c0 = hi1 ^ c1 ^ k0;
        c1 = lo1;
        c2 = hi0 ^ c3 ^ k1;
        c3 = lo0;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Philox SR threshold (this library's mapping): entry i at step t takes word
 * i mod 4 of Philox4x32-10(counter = (floor(i/4) mod 2^32, floor(i/4) >> 32, t, 0),
 * key = (seed, layer)), top 24 bits. */
static uint32_t philox_threshold24(uint32_t seed, uint32_t layer, uint32_t t, uint64_t i) {
    const uint64_t q = i >> 2;
    const uint32_t ctr[4] = {(uint32_t)q, (uint32_t)(q >> 32), t, 0u};
    const uint32_t key[2] = {seed, layer};
    uint32_t out[4];
    philox4x32_10(ctr, key, out);
    return out[i & 3u] >> 8;
}

static uint32_t threshold24(int rule, uint32_t seed, uint32_t layer, uint32_t t, uint64_t i,
                            uint64_t block) {
    if (rule == ORC_WEYL) return weyl_acc(i, block, layer, seed, t) >> 8;
    if (rule == ORC_SR) return fmix32((uint32_t)i * 0x9E3779B1u + sr_key(seed, layer, t)) >> 8;
    if (rule == ORC_PHILOX) return philox_threshold24(seed, layer, t, i);
    return 1u << 23; /* RTN: nominal u = 1/2 (rounding itself is nearest-even) */
}

/* ------------------------------------------------------------------------- */
/* Exported helpers.                                                          */
/* ------------------------------------------------------------------------- */
static void ensure_init(void) {
    ensure_grids();
    ensure_weyl_constants();
}

void orc_weyl_constants(uint32_t out[5]) {
    ensure_init();
    out[0] = W_A; out[1] = W_B; out[2] = W_L; out[3] = W_S; out[4] = W_PHI;
}

uint32_t orc_fmix32(uint32_t h) { return fmix32(h); }

void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
    philox4x32_10(ctr, key, out);
}

int orc_grid(int f, double *val, uint32_t *code, int cap) {
    ensure_init();
    if (is_int(f)) {
        const int q = int_qmax(f), n = 2 * q + 1;
        if (val && code)
            for (int i = 0; i < n && i < cap; ++i) { val[i] = i - q; code[i] = int_code(f, i - q); }
        return n;
    }
    if (f < 0 || f > 2) return -1;
    const grid_t *g = &GRID[f];
    if (val && code) {
        int n = g->n < cap ? g->n : cap;
        for (int i = 0; i < n; ++i) { val[i] = g->val[i]; code[i] = g->code[i]; }
    }
    return g->n;
}

double orc_decode(int f, uint32_t code) {
    if (f == ORC_FP32) return (double)bits_f32(code);
    if (is_int(f)) return (double)int_value(f, code);
    return decode_fields(f, code);
}

/* Position of a code in its format's value order (both zeros share one). */
int orc_code_rank(int f, uint32_t code) {
    ensure_init();
    if (is_int(f)) {
        int32_t k = int_value(f, code);
        return (k < -int_qmax(f)) ? -1 : k + int_qmax(f);  /* -128 / -8 are not codes */
    }
    double v = decode_fields(f, code);
    if (isnan(v)) return -1;
    const grid_t *g = &GRID[f];
    if (isinf(v)) {
        if (!FMT[f].ieee_special) return -1;
        return v > 0 ? g->n - 1 : 0;
    }
    return floor_index(g, v);
}

uint32_t orc_round(int f, int rule, float x, uint32_t U24) {
    ensure_init();
    if (f == ORC_FP32) return f32_bits(x);
    if (is_int(f)) return int_code(f, round_to_int(int_qmax(f), rule, x, U24 & 0xFFFFFFu));
    return round_to_format(f, rule, x, U24 & 0xFFFFFFu);
}

void orc_round_array(int f, int rule, int64_t n, const float *x, const uint32_t *U24,
                     uint32_t *out) {
    ensure_init();
    for (int64_t i = 0; i < n; ++i) out[i] = orc_round(f, rule, x[i], U24 ? U24[i] : (1u << 23));
}

uint32_t orc_threshold(int rule, uint32_t seed, uint32_t layer, uint32_t step, uint64_t i,
                       uint64_t block) {
    ensure_init();
    return threshold24(rule, seed, layer, step, i, block);
}

void orc_dither_fill(int rule, uint32_t seed, uint32_t layer, uint32_t step, uint64_t entry_base,
                     int64_t n, uint64_t block, uint32_t *out) {
    ensure_init();
    for (int64_t k = 0; k < n; ++k)
        out[k] = threshold24(rule, seed, layer, step, entry_base + (uint64_t)k, block);
}

/* ------------------------------------------------------------------------- */
/* Code storage helpers (codes are 1, 2 or 4 bytes per entry; INT4 packs two */
/* entries per byte, entry 2j in the low nibble of byte j).                   */
/* ------------------------------------------------------------------------- */
static int code_bytes(int f) {
    return (f == ORC_E4M3 || is_int(f)) ? 1 : (f == ORC_FP32 ? 4 : 2);
}

static uint32_t load_code(int f, const void *p, int64_t k) {
    if (f == ORC_INT4) return (((const uint8_t *)p)[k / 2] >> (4 * (k % 2))) & 0xFu;
    switch (code_bytes(f)) {
        case 1: return ((const uint8_t *)p)[k];
        case 2: return ((const uint16_t *)p)[k];
        default: return ((const uint32_t *)p)[k];
    }
}

static void store_code(int f, void *p, int64_t k, uint32_t c) {
    if (f == ORC_INT4) {
        uint8_t *b = (uint8_t *)p + k / 2;
        const int sh = 4 * (int)(k % 2);
        *b = (uint8_t)((*b & ~(0xFu << sh)) | ((c & 0xFu) << sh));
        return;
    }
    switch (code_bytes(f)) {
        case 1: ((uint8_t *)p)[k] = (uint8_t)c; break;
        case 2: ((uint16_t *)p)[k] = (uint16_t)c; break;
        default: ((uint32_t *)p)[k] = c; break;
    }
}

/* Stored code -> its exact value as fp32 (E4M3: without the group scale). */
static float code_value(int f, uint32_t code) {
    if (f == ORC_FP32) return bits_f32(code);
    if (is_int(f)) return (float)int_value(f, code);
    return (float)decode_fields(f, code); /* exact: every code is an fp32 value */
}

/*
 * Requantize n fp32 values into format f (Appendix B "Formats").
 * E4M3 and INT8/INT4 use one fp32 scale per group of `group` consecutive
 * entries, with qmax = 448 (E4M3), 127 (INT8) or 7 (INT4):
 *   m = max |h| over the group (NaN entries ignored), s = fl32(m / qmax);
 *   s below the smallest normal fp32 is stored as 0 and every code is a
 *   (signed, for E4M3) zero, NaN staying NaN in E4M3; otherwise r = fl32(1 / s)
 *   and each entry is rounded as q = fl32(h * r) on the E4M3 grid or the
 *   integer lattice.
 * Entry k uses the threshold of global index entry_base + k.
 * Returns 0, or -1 on bad arguments.
 */
int orc_requantize(int f, int rule, uint32_t seed, uint32_t layer, uint32_t step,
                   uint64_t entry_base, uint64_t block, int64_t n, int64_t group, const float *h,
                   void *codes, float *scale) {
    ensure_init();
    if (f < 0 || f >= ORC_NFMT || n < 0 || block == 0) return -1;
    if (!is_scaled(f)) {
        for (int64_t k = 0; k < n; ++k) {
            uint32_t U = threshold24(rule, seed, layer, step, entry_base + (uint64_t)k, block);
            store_code(f, codes, k, orc_round(f, rule, h[k], U));
        }
        return 0;
    }
    if (group <= 0 || n % group != 0) return -1;
    for (int64_t g0 = 0; g0 < n; g0 += group) {
        float m = 0.0f;
        for (int64_t k = g0; k < g0 + group; ++k) {
            float a = fabsf(h[k]);
            if (a > m) m = a;
        }
        const float qmax = (f == ORC_E4M3) ? 448.0f : (float)int_qmax(f);
        float s = m / qmax;
        if (!(s >= FLT_MIN)) s = 0.0f;
        scale[g0 / group] = s;
        float r = (s == 0.0f) ? 0.0f : 1.0f / s;
        for (int64_t k = g0; k < g0 + group; ++k) {
            uint32_t c;
            if (is_int(f)) {
                const uint32_t U =
                    threshold24(rule, seed, layer, step, entry_base + (uint64_t)k, block);
                c = (s == 0.0f) ? 0u : int_code(f, round_to_int(int_qmax(f), rule, h[k] * r, U));
            } else if (isnan(h[k])) {
                c = signbit(h[k]) ? GRID[ORC_E4M3].neg_nan : GRID[ORC_E4M3].pos_nan;
            } else if (s == 0.0f) {
                c = signbit(h[k]) ? GRID[ORC_E4M3].neg_zero : GRID[ORC_E4M3].pos_zero;
            } else {
                float q = h[k] * r;
                uint32_t U = threshold24(rule, seed, layer, step, entry_base + (uint64_t)k, block);
                c = round_to_format(ORC_E4M3, rule, q, U);
            }
            store_code(f, codes, k, c);
        }
    }
    return 0;
}

/*
 * One decode step of the selective-state recurrence, eq. (rec):
 * h <- exp(dt A) h + dt B x, y = C h + D x  (Appendix B "Runners").
 *
 * Layout (row-major, contiguous):
 *   state  [batch][nheads][headdim][dstate] codes, updated in place
 *   scale  E4M3, INT8, INT4: one fp32 per group of entries (group 0 = one head)
 *          INT4 state rows hold dstate / 2 bytes (dstate even)
 *   x      [batch][nheads][headdim]        dt [batch][nheads]
 *   A      [nheads] (a_per_state = 0, Mamba-2) or [nheads][dstate] (= 1, Mamba-1)
 *   B, C   [batch][ngroups][dstate]; head h uses group h / (nheads / ngroups)
 *   D      [nheads] or NULL (no skip term)
 *   y      [batch][nheads][headdim] in double (output)
 *   hnew   optional [batch][nheads][headdim][dstate] fp32 pre-rounding values
 * Mamba-1 is the case headdim = 1, ngroups = 1, a_per_state = 1, nheads = d_inner.
 * y is computed from the pre-rounding state. The state is then written back
 * under (rule, format) with the thresholds of global entry entry_base + flat index.
 * Returns 0, or -1 on bad arguments.
 */
/*
 * The decode-step operations on either side of the update, as in the Mamba
 * reference implementation the paper's runners follow for the convolution and
 * the gate (Appendix B "Runners"):
 *   step size   dt' = softplus(fl32(dt + dt_bias)), softplus(v) = log(1 + e^v)
 *               evaluated in double and rounded once (v itself above 20, where
 *               the two agree in fp32);
 *   gate        y' = y * silu(z), silu(z) = z / (1 + e^-z), in double;
 *   conv1d      the causal depthwise convolution's state shifts by one position
 *               and takes the new input; out = sum_i state_i w_i + bias, in
 *               double, optionally through silu.
 */
static float softplus_dt(float v) {
    if (v > 20.0f) return v;
    return (float)log1p(exp((double)v));
}

static double silu(double z) { return z / (1.0 + exp(-z)); }

int orc_state_update_ex(int f, int rule, uint32_t seed, uint32_t layer, uint32_t step,
                        uint64_t entry_base, uint64_t block, int64_t group, int64_t batch,
                        int64_t nheads, int64_t headdim, int64_t dstate, int64_t ngroups,
                        int a_per_state, void *state, float *scale, const float *x,
                        const float *dt, const float *dt_bias, int dt_softplus, const float *z,
                        const float *A, const float *B, const float *C, const float *D, double *y,
                        float *hnew);

int orc_state_update(int f, int rule, uint32_t seed, uint32_t layer, uint32_t step,
                     uint64_t entry_base, uint64_t block, int64_t group, int64_t batch,
                     int64_t nheads, int64_t headdim, int64_t dstate, int64_t ngroups,
                     int a_per_state, void *state, float *scale, const float *x, const float *dt,
                     const float *A, const float *B, const float *C, const float *D, double *y,
                     float *hnew) {
    return orc_state_update_ex(f, rule, seed, layer, step, entry_base, block, group, batch, nheads,
                               headdim, dstate, ngroups, a_per_state, state, scale, x, dt, NULL, 0,
                               NULL, A, B, C, D, y, hnew);
}

/* As orc_state_update, with dt' = (softplus if dt_softplus)(dt + dt_bias) per
 * (batch, head) (dt_bias [nheads] or NULL) and y gated by silu(z) (z shaped as
 * y, or NULL). */
int orc_state_update_ex(int f, int rule, uint32_t seed, uint32_t layer, uint32_t step,
                        uint64_t entry_base, uint64_t block, int64_t group, int64_t batch,
                        int64_t nheads, int64_t headdim, int64_t dstate, int64_t ngroups,
                        int a_per_state, void *state, float *scale, const float *x,
                        const float *dt, const float *dt_bias, int dt_softplus, const float *z,
                        const float *A, const float *B, const float *C, const float *D, double *y,
                        float *hnew) {
    ensure_init();
    if (f < 0 || f >= ORC_NFMT || batch < 0 || nheads <= 0 || headdim <= 0 || dstate <= 0 ||
        ngroups <= 0 || nheads % ngroups != 0 || block == 0)
        return -1;
    const int64_t head_size = headdim * dstate;
    const int64_t n_total = batch * nheads * head_size;
    if (f == ORC_INT4 && dstate % 2 != 0) return -1;
    if (is_scaled(f)) {
        if (group == 0) group = head_size;
        if (group < 0 || n_total % group != 0) return -1;
    }
    float *hn = (float *)malloc(sizeof(float) * (size_t)(n_total > 0 ? n_total : 1));
    const int64_t heads_per_group = nheads / ngroups;
    for (int64_t b = 0; b < batch; ++b) {
        for (int64_t hd = 0; hd < nheads; ++hd) {
            const int64_t g = hd / heads_per_group;
            float dtv = dt[b * nheads + hd];
            if (dt_bias) dtv = dtv + dt_bias[hd];
            if (dt_softplus) dtv = softplus_dt(dtv);
            const float *Bg = B + (b * ngroups + g) * dstate;
            const float *Cg = C + (b * ngroups + g) * dstate;
            const float Dv = D ? D[hd] : 0.0f;
            for (int64_t p = 0; p < headdim; ++p) {
                const int64_t row = (b * nheads + hd) * headdim + p;
                const float xv = x[row];
                const float dx = dtv * xv;
                double acc = 0.0;
                for (int64_t n = 0; n < dstate; ++n) {
                    const int64_t k = row * dstate + n;
                    const float a = a_per_state ? A[hd * dstate + n] : A[hd];
                    const float z = dtv * a;
                    const float dA = (float)exp((double)z);
                    const float v = code_value(f, load_code(f, state, k));
                    /* the stored value: scaled formats multiply by the old scale */
                    const float h_prev = is_scaled(f) ? v * scale[k / group] : v;
                    const float w = dx * Bg[n];
                    const float h_new = fmaf(dA, h_prev, w);
                    hn[k] = h_new;
                    acc += (double)Cg[n] * (double)h_new;
                }
                y[row] = acc + (double)Dv * (double)xv;
                if (z) y[row] *= silu((double)z[row]);
            }
        }
    }
    if (hnew) memcpy(hnew, hn, sizeof(float) * (size_t)n_total);
    int rc = orc_requantize(f, rule, seed, layer, step, entry_base, block, n_total, group, hn,
                            state, scale);
    free(hn);
    return rc;
}

/*
 * Checkpoint write with an fp32 state (Section 6.5 "Periodic checkpointing";
 * Appendix B "Decode regime", CC = 8: fp32 intermediate states, rounding at
 * every k-th write). The state holds fp32 values. One step of eq. (rec) is
 * taken in fp32 exactly as for the unrounded format (h_prev is the stored
 * value), then each new value is rounded onto the grid of format f under the
 * rule (scaled formats: group scale s as in orc_requantize) and stored back as
 * its fp32 value: decode(code), or fl32(code value * s). The group scales are
 * also written to `scale` when it is not NULL. Steps between checkpoints are
 * plain fp32 steps (orc_state_update with ORC_FP32).
 * Returns 0, or -1 on bad arguments.
 */
int orc_state_update_fp32_grid(int f, int rule, uint32_t seed, uint32_t layer, uint32_t step,
                               uint64_t entry_base, uint64_t block, int64_t group, int64_t batch,
                               int64_t nheads, int64_t headdim, int64_t dstate, int64_t ngroups,
                               int a_per_state, float *state, float *scale, const float *x,
                               const float *dt, const float *A, const float *B, const float *C,
                               const float *D, double *y) {
    ensure_init();
    if (f < 0 || f >= ORC_NFMT || f == ORC_FP32) return -1;
    const int64_t n_total = batch * nheads * headdim * dstate;
    if (is_scaled(f)) {
        if (group == 0) group = headdim * dstate;
        if (group <= 0 || n_total % group != 0) return -1;
    }
    int rc = orc_state_update(ORC_FP32, ORC_RTN, seed, layer, step, entry_base, block, 0, batch,
                              nheads, headdim, dstate, ngroups, a_per_state, state, NULL, x, dt, A,
                              B, C, D, y, NULL);
    if (rc != 0) return rc;
    const int64_t n_alloc = n_total > 0 ? n_total : 1;
    void *codes = calloc((size_t)n_alloc, 4);
    float *sc = is_scaled(f) ? (float *)calloc((size_t)(n_alloc / (group > 0 ? group : 1) + 1), 4)
                             : NULL;
    rc = orc_requantize(f, rule, seed, layer, step, entry_base, block, n_total, group, state,
                        codes, sc);
    if (rc == 0) {
        for (int64_t k = 0; k < n_total; ++k) {
            const float v = code_value(f, load_code(f, codes, k));
            state[k] = is_scaled(f) ? v * sc[k / group] : v;
        }
        if (scale && sc) memcpy(scale, sc, sizeof(float) * (size_t)(n_total / group));
    }
    free(codes);
    free(sc);
    return rc;
}

/*
 * Causal depthwise conv1d decode update (the reference's convolution state):
 * state [batch][channels][width] holds the last `width` inputs of each channel,
 * oldest first. The state shifts by one and takes x [batch][channels]; then
 * out[b][c] = sum_i state[b][c][i] * weight[c][i] + bias[c] (bias may be NULL),
 * accumulated in double, and passed through silu when `act` is 1.
 */
int orc_conv1d_update(int64_t batch, int64_t channels, int64_t width, float *state,
                      const float *x, const float *weight, const float *bias, int act,
                      double *out) {
    if (batch < 0 || channels <= 0 || width <= 0) return -1;
    for (int64_t b = 0; b < batch; ++b) {
        for (int64_t c = 0; c < channels; ++c) {
            float *s = state + (b * channels + c) * width;
            for (int64_t i = 0; i + 1 < width; ++i) s[i] = s[i + 1];
            s[width - 1] = x[b * channels + c];
            double acc = bias ? (double)bias[c] : 0.0;
            for (int64_t i = 0; i < width; ++i) acc += (double)s[i] * (double)weight[c * width + i];
            out[b * channels + c] = act ? silu(acc) : acc;
        }
    }
    return 0;
}

/*
 * Open-loop replay (Appendix B "Open-loop replay"; Section 6.2, the paragraph on
 * the recurrence alone): each entry i of a recorded trace carries its decays
 * a_t[i] and writes w_t[i], t = 1..T, and its FP32 state h_0[i] at the end of
 * prefill. Two trajectories are iterated side by side:
 *   reference  h_t  = fma(a_t, h_{t-1}, w_t)                     (fp32)
 *   stored     hq_0 = Q_0(h_0),   hq_t = Q_t(fma(a_t, hq_{t-1}, w_t))
 * Q_t requantizes the whole vector under (rule, format) with the thresholds of
 * global index entry_base + i and step step0 + t (orc_requantize, group scales
 * for E4M3/INT8/INT4), and returns the stored value: the code's value, times
 * its group scale in fp32 for the scaled formats. Per block k of block_steps
 * steps (steps k*block_steps + 1 .. (k+1)*block_steps; the last may be shorter)
 *   err[k][i] = sum (hq_t - h_t)^2,   ref[k][i] = sum h_t^2,
 * each term formed and added in double, in step order. Optional outputs (NULL
 * to skip): codes and scales of hq_T, and h_T.
 * Layout: a and w are [T][n]; err and ref are [ceil(T / block_steps)][n].
 * Returns 0, or -1 on bad arguments.
 */
int orc_replay(int f, int rule, uint32_t seed, uint32_t layer, uint32_t step0,
               uint64_t entry_base, uint64_t block, int64_t n, int64_t group, int64_t steps,
               int64_t block_steps, const float *h0, const float *a, const float *w,
               double *err, double *ref, void *codes_out, float *scale_out, float *h_final) {
    ensure_init();
    if (f < 0 || f >= ORC_NFMT || n < 0 || steps < 0 || block_steps < 1 || block == 0) return -1;
    if (is_scaled(f) && (group <= 0 || n % group != 0)) return -1;
    const int64_t n_alloc = n > 0 ? n : 1;
    float *x = (float *)malloc(sizeof(float) * (size_t)n_alloc);
    float *hq = (float *)malloc(sizeof(float) * (size_t)n_alloc);
    float *href = (float *)malloc(sizeof(float) * (size_t)n_alloc);
    void *codes = calloc((size_t)n_alloc, 4);
    float *sc = is_scaled(f) ? (float *)calloc((size_t)(n_alloc / group + 1), sizeof(float)) : NULL;
    int rc = 0;
    for (int64_t t = 0; t <= steps && rc == 0; ++t) {
        for (int64_t i = 0; i < n; ++i) {
            if (t == 0) {
                href[i] = h0[i];
                x[i] = h0[i];
            } else {
                const float at = a[(t - 1) * n + i], wt = w[(t - 1) * n + i];
                href[i] = fmaf(at, href[i], wt);
                x[i] = fmaf(at, hq[i], wt);
            }
        }
        rc = orc_requantize(f, rule, seed, layer, step0 + (uint32_t)t, entry_base, block, n, group,
                            x, codes, sc);
        if (rc != 0) break;
        for (int64_t i = 0; i < n; ++i) {
            const float v = code_value(f, load_code(f, codes, i));
            hq[i] = is_scaled(f) ? v * sc[i / group] : v;
        }
        if (t == 0) continue;
        const int64_t k = (t - 1) / block_steps;
        for (int64_t i = 0; i < n; ++i) {
            if ((t - 1) % block_steps == 0) {
                err[k * n + i] = 0.0;
                if (ref) ref[k * n + i] = 0.0;
            }
            const double d = (double)hq[i] - (double)href[i];
            err[k * n + i] += d * d;
            if (ref) ref[k * n + i] += (double)href[i] * (double)href[i];
        }
    }
    if (rc == 0) {
        if (codes_out) memcpy(codes_out, codes, f == ORC_INT4 ? (size_t)((n + 1) / 2)
                                                              : (size_t)(n * code_bytes(f)));
        if (scale_out && sc) memcpy(scale_out, sc, sizeof(float) * (size_t)(n / group));
        if (h_final) memcpy(h_final, href, sizeof(float) * (size_t)n);
    }
    free(x);
    free(hq);
    free(href);
    free(codes);
    free(sc);
    return rc;
}
