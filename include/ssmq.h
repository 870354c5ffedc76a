/*
 * ssmq.h -- quantized selective-state update for Mamba-style recurrent state
 * caches on AMD Instinct MI355X (gfx950).
 *
 * Method: "Low-Discrepancy Dither for Quantized Recurrent State Caches".
 * Each state entry follows h_t = a_t h_(t-1) + w_t (Section 2, eq. (rec)); the
 * update is computed in fp32 and rounded only when written back (Section 2,
 * "Low-precision storage") with one of three threshold rules of eq. (dither):
 * round-to-nearest, stochastic rounding, or the golden-ratio Weyl dither with
 * per-entry R2 offsets and an integer phase (Appendix B, "Dithers").
 *
 * Conventions shared by every entry point:
 *   - Data pointers are DEVICE pointers (HIP device memory) unless stated. The
 *     caller owns every buffer and keeps it alive until the work on `stream`
 *     has completed. Nothing is allocated or retained by the library.
 *   - `stream` is a hipStream_t passed as void*; NULL is the default stream.
 *     Every call only enqueues work and returns; completion is the caller's
 *     business (e.g. hipStreamSynchronize).
 *   - All arguments are validated on the host before any HIP call. A rejected
 *     call returns a non-zero status, touches no memory and leaves a message
 *     for ssmq_last_error(). A failed kernel launch returns SSMQ_EDEVICE.
 *   - A call with nothing to do (batch 0, or n / n_entries 0) checks its
 *     scalar arguments, returns SSMQ_OK and launches nothing; its pointer
 *     arguments are not read and may be NULL.
 *   - Tensors are contiguous and row-major, with the layouts given below.
 *   - Step, layer and seed arithmetic is modulo 2^32.
 *   - Calls on different streams that write the same memory race; the library
 *     holds no global mutable state and is otherwise thread-safe.
 */
#ifndef SSMQ_H
#define SSMQ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SSMQ_OK = 0,
    SSMQ_EINVAL = 1,       /* null pointer, bad size or bad enum value          */
    SSMQ_EUNSUPPORTED = 2, /* valid but not implemented (shape / group layout)  */
    SSMQ_EALIGN = 3,       /* a pointer misses its required alignment           */
    SSMQ_EDEVICE = 4       /* the HIP runtime reported an error                 */
} ssmq_status;

/* Rounding rules, eq. (dither): Q_u(x) = s floor(x/s + u) (Section 2). */
typedef enum {
    SSMQ_RTN = 0,  /* round to nearest, ties to even (the native cast)                  */
    SSMQ_SR = 1,   /* stochastic: u from a counter-based hash of (seed, layer, entry, t) */
    SSMQ_WEYL = 2, /* Weyl dither: u = top 24 bits of A(r+1)+B(c+1)+L l+S sigma+t Phi    */
    SSMQ_SR_PHILOX = 3 /* stochastic with Philox4x32-10 (the generator behind the paper's SR,
                          Appendix B "Dithers"; Salmon et al., SC 2011): entry i at step t
                          takes word i mod 4 of Philox(counter (i/4 mod 2^32, i/4 >> 32,
                          t, 0), key (seed, layer)), top 24 bits                         */
} ssmq_rule;

/* Storage formats (Section 2 "Low-precision storage"; Appendix B "Formats"). */
typedef enum {
    SSMQ_FP16 = 0,      /* IEEE binary16 codes, no scale                                 */
    SSMQ_BF16 = 1,      /* bfloat16 codes, no scale                                      */
    SSMQ_FP8_E4M3 = 2,  /* OCP E4M3FN codes with one fp32 scale per group, max 448,
                           saturating                                                    */
    SSMQ_FP32 = 3,      /* unrounded fp32 (a full-precision twin); the rule is ignored   */
    SSMQ_INT8 = 4,      /* symmetric INT8, one fp32 block scale per group, codes
                           -127..127 two's complement, one byte per entry              */
    SSMQ_INT4 = 5       /* symmetric INT4, one fp32 block scale per group, codes -7..7
                           two's complement, two entries per byte (even entry in the
                           low nibble)                                                 */
} ssmq_format;

/* Shape of one layer's state cache [batch][nheads][headdim][dstate]. */
typedef struct {
    int64_t batch;       /* sequences in the batch (0 is a valid no-op)                   */
    int32_t nheads;      /* Mamba-2 heads; Mamba-1: d_inner channels                      */
    int32_t headdim;     /* P rows per head; Mamba-1: 1                                   */
    int32_t dstate;      /* N, the state dimension                                        */
    int32_t ngroups;     /* groups sharing B and C; head h uses group h / (nheads/ngroups) */
    int32_t a_per_state; /* 0: A[nheads] (Mamba-2); 1: A[nheads][dstate] (Mamba-1)        */
} ssmq_dims;

/*
 * SSMQ_FLAG_FP32_STATE (ssmq_state_update only): a checkpoint write on an fp32
 * state, for periodic checkpointing (Section 6.5 "Periodic checkpointing";
 * Appendix B "Decode regime", CC = 8: fp32 intermediate states, rounding every
 * k-th write). `state` holds fp32 values, read as they are; each new value is
 * rounded onto the grid of q->format under q->rule (E4M3/INT8/INT4 with their
 * group scale) and stored back as the fp32 value of its code (times the scale).
 * The group scales are written to `state_scale` when it is not NULL. The steps
 * between checkpoints are ordinary SSMQ_FP32 steps. Scale groups must be powers
 * of two up to 1024 entries; q->format must not be SSMQ_FP32.
 */
enum { SSMQ_FLAG_FP32_STATE = 1 };

/* How the state is written back. */
typedef struct {
    int32_t rule;          /* ssmq_rule                                                    */
    int32_t format;        /* ssmq_format                                                  */
    int32_t dither_block;  /* Weyl offsets: block r = i / dither_block, position
                              c = i % dither_block of the flat entry index i; a power of
                              two. 16 for Mamba models, the state dimension for hybrids
                              (Section 2 "Low-precision storage")                           */
    int32_t scale_group;   /* E4M3, INT8, INT4: entries per fp32 scale, a power of two
                              >= 16 that divides headdim*dstate; 0 = one scale per head.
                              The paper's blocks: 16 (Mamba), 128 (hybrids)               */
    uint32_t seed;         /* sigma (Appendix B "Dithers"; SR key)                          */
    uint32_t layer;        /* l (Appendix B "Dithers"; SR key)                              */
    uint32_t step;         /* t, the integer phase counter (Section 6.4, "Computing the
                              phase in float32": an integer phase keeps every stream)      */
    uint32_t flags;        /* 0, or SSMQ_FLAG_FP32_STATE                                    */
    uint64_t entry_base;   /* global flat index of entry 0 of this tensor, a multiple of
                              16; lets a shard reproduce the unsharded thresholds           */
} ssmq_qparams;

/*
 * ssmq_state_update -- one decode step of the selective-state update, in place.
 *
 * Defines (Section 2, eq. (rec); Appendix B "Runners", Mamba-1 and Mamba-2):
 *   h_prev = decode(state)                 (E4M3, INT8, INT4: the fp32 product of the
 *                                           code value and the old group scale)
 *   dA     = exp(dt * A)                   (per head, or per (head, n) for Mamba-1)
 *   h_new  = dA * h_prev + (dt * x_p) * B_n
 *   y_p    = sum_n C_n * h_new + D * x_p   (from the unrounded h_new)
 *   state  = Q_u(h_new) under (rule, format); E4M3, INT8 and INT4 first set each
 *            group scale to max|h_new| / qmax (448, 127, 7) and round
 *            h_new * (1/scale) on their grid (Appendix B "Formats").
 * Entry i = entry_base + flat index uses threshold u_(i,step) (see ssmq_dither_fill).
 * Evaluation order: the scaled formats take dA * h_prev as fl32(dA * scale) * code
 * value (one rounding of the scaled decay per group, where the definition rounds
 * code value * scale per entry); h_new then differs from the definition's by at
 * most about one fp32 ulp, and a stored code only where h_new lies next to its
 * rounding point (fewer than one entry in 10^5 measured).
 *
 * Arguments (device pointers; alignment in brackets):
 *   state        [batch][nheads][headdim][dstate] codes (2 B fp16/bf16, 1 B E4M3
 *                and INT8, 4 B fp32, 1/2 B INT4), read and overwritten [16 B]
 *   state_scale  E4M3, INT8, INT4: [batch*nheads*headdim*dstate / group] fp32, read
 *                (old scales) and overwritten (new scales) [4 B]; NULL otherwise
 *   x            [batch][nheads][headdim] fp32 [4 B]
 *   dt           [batch][nheads] fp32, the step size after softplus [4 B]
 *   A            [nheads] [4 B] or [nheads][dstate] [16 B] fp32 (negative decay rates)
 *   B, C         [batch][ngroups][dstate] fp32 [16 B]
 *   D            [nheads] fp32, or NULL for no skip term [4 B]
 *   y            [batch][nheads][headdim] fp32, written [4 B]
 * Requirements: a state row splits into chunks (dstate % 8 == 0 for fp16/bf16,
 * % 16 for E4M3, INT8 and INT4, % 4 for fp32) whose count is a power of two
 * <= 64; nheads % ngroups == 0. Scale groups are either one head (when
 * headdim*dstate is 4096 to 131072 entries, a power of two, and A is per head)
 * or a power of two of at most 1024 entries. Other shapes return
 * SSMQ_EUNSUPPORTED.
 */
ssmq_status ssmq_state_update(const ssmq_dims* dims, const ssmq_qparams* q, void* state,
                              float* state_scale, const float* x, const float* dt,
                              const float* A, const float* B, const float* C, const float* D,
                              float* y, void* stream);

/*
 * The decode-step operations on either side of the update, fused into it
 * (Appendix B "Runners": conv and gating as in the Mamba reference):
 *   dt' = dt + dt_bias[head]                   (dt_bias non-NULL)
 *   dt' = softplus(dt') = log(1 + exp(dt'))    (dt_softplus = 1; evaluated in
 *         double and rounded once; values above 20 are kept as they are)
 *   y'  = y * silu(z) = y * z / (1 + exp(-z))  (z non-NULL, shaped as y)
 * The update then uses dt' in place of dt. The group-wise RMS normalization of
 * Mamba-2 spans heads and stays outside.
 */
typedef struct {
    const float* dt_bias;  /* [nheads] fp32 device pointer, or NULL [4 B]        */
    int32_t dt_softplus;   /* 0 or 1                                              */
    int32_t reserved;      /* must be 0                                           */
    const float* z;        /* [batch][nheads][headdim] fp32, or NULL [4 B]        */
} ssmq_step_opts;

/*
 * ssmq_state_update_ex -- ssmq_state_update with the decode-step options above
 * (opts may be NULL: then it is ssmq_state_update). Same arguments, layouts,
 * requirements and errors; opts pointers are device pointers.
 */
ssmq_status ssmq_state_update_ex(const ssmq_dims* dims, const ssmq_qparams* q,
                                 const ssmq_step_opts* opts, void* state, float* state_scale,
                                 const float* x, const float* dt, const float* A, const float* B,
                                 const float* C, const float* D, float* y, void* stream);

/*
 * ssmq_conv1d_update -- the causal depthwise convolution's decode step (the
 * Mamba reference's convolution state; Appendix B "Runners").
 *   conv_state [batch][channels][width] fp32, the last `width` inputs of each
 *              channel, oldest first; shifted by one and x appended, in place
 *   x          [batch][channels] fp32, the new input
 *   weight     [channels][width] fp32; bias [channels] fp32 or NULL
 *   out        [batch][channels] fp32: bias + sum_k state[k] weight[k], through
 *              silu when act = 1 (accumulated in fp32 by FMA, k ascending)
 * All device pointers, 4-byte aligned; 1 <= width <= 64; batch * channels < 2^32.
 * For Mamba-2 the channels are x, B and C side by side (d_inner + 2 ngroups dstate).
 */
ssmq_status ssmq_conv1d_update(int64_t batch, int32_t channels, int32_t width, float* conv_state,
                               const float* x, const float* weight, const float* bias,
                               int32_t act, float* out, void* stream);

/*
 * ssmq_requantize -- write fp32 values into a storage format under a rule.
 *
 * The rounding step alone (Section 2, eq. (dither); Appendix B "Formats"):
 * codes[k] = Q_u(h[k]) with the threshold of entry entry_base + k. For E4M3,
 * INT8 and INT4 each group of consecutive entries (q->scale_group, or head_size
 * when that is 0) gets scale[g] = fl32(max|h| / qmax) (qmax 448, 127, 7),
 * flushed to 0 below 2^-126 (then every code of the group is a zero), and codes
 * of fl32(h * fl32(1 / scale)) rounded on the E4M3 grid or the integer lattice
 * after saturation to +-qmax. For the float formats a result of zero keeps the
 * sign of its input and NaN gives the canonical NaN code; the integer formats
 * store NaN as 0 and round exact ties of RTN to the even integer.
 *
 * Arguments: n_entries >= 0; head_size > 0 (used only for scaled formats with
 * scale_group 0); h [n_entries] fp32 [16 B]; codes [n_entries] codes (INT4:
 * n_entries / 2 bytes) [16 B]; scale (E4M3, INT8, INT4) [n_entries / group]
 * fp32 (written), else NULL [4 B]. Scale groups must be multiples of 16 that
 * divide n_entries; entry_base must be a multiple of 16.
 */
ssmq_status ssmq_requantize(const ssmq_qparams* q, int64_t n_entries, int64_t head_size,
                            const float* h, void* codes, float* scale, void* stream);

/*
 * ssmq_dither_fill -- the 24-bit thresholds U (u = U / 2^24) of entries
 * entry_base .. entry_base + n - 1 at one (seed, layer, step).
 *
 *   SSMQ_WEYL: top 24 bits of (A(r+1) + B(c+1) + L layer + S seed + t Phi) mod 2^32,
 *              r = i / dither_block, c = i % dither_block; A, B, L, S are 2^32 times
 *              0.7548776662, 0.5698402910, 0.1234567, 0.3141592 rounded to nearest and
 *              Phi = 2654435769 (Appendix B "Dithers"; Section 6.4).
 *   SSMQ_SR:   top 24 bits of fmix32(i * 0x9E3779B1 + K) with the per-step key
 *              K = fmix32(fmix32(fmix32(seed) ^ layer * 0xC2B2AE3D) ^ t * 0x85EBCA77)
 *              (Appendix B "Decode regime", hash SR; fmix32 = MurmurHash3 finalizer).
 *   SSMQ_SR_PHILOX: top 24 bits of word i mod 4 of Philox4x32-10 with counter
 *              (floor(i/4) mod 2^32, floor(i/4) >> 32, t, 0) and key (seed, layer).
 *   SSMQ_RTN:  2^23 (u = 1/2) everywhere; nearest rounding breaks exact ties to even.
 * Arguments: n >= 0; dither_block a power of two; U24 [n] uint32 output [4 B];
 * any entry_base.
 */
ssmq_status ssmq_dither_fill(int32_t rule, uint32_t seed, uint32_t layer, uint32_t step,
                             uint64_t entry_base, int64_t n, int32_t dither_block,
                             uint32_t* U24, void* stream);

/*
 * ssmq_replay -- open-loop replay of recorded decays and writes under one rule
 * and format (Appendix B "Open-loop replay"; Section 6.2, on the recurrence
 * alone reproducing the gain): the error a rounding rule accumulates in the
 * state recurrence by itself, without the rest of the network.
 *
 * Defines, for each entry i of a trace of n entries and T = steps steps:
 *   reference  h_0 = h0[i],        h_t  = fma(a[t-1][i], h_(t-1), w[t-1][i])   (fp32)
 *   stored     hq_0 = Q_0(h0[i]),  hq_t = Q_t(fma(a[t-1][i], hq_(t-1), w[t-1][i]))
 * where Q_t is the write-back of ssmq_requantize under q (rule, format, dither
 * block, seed, layer, entry_base) at step q->step + t, returning the stored value:
 * the code's value, times its group scale in fp32 for E4M3, INT8 and INT4 (each
 * group of q->scale_group consecutive entries gets scale fl32(max|x| / qmax)).
 * For each block k of block_steps steps (steps k*block_steps + 1 ..
 * min((k+1)*block_steps, T)):
 *   err[k][i] = sum (hq_t - h_t)^2      ref[k][i] = sum h_t^2
 * each term formed in double from the fp32 values and added in step order.
 * The state error of a set of entries is sum err / sum ref over them.
 *
 * Arguments (device pointers; alignment in brackets):
 *   n            entries, a multiple of 4 (and of the scale group); 0 is a no-op
 *   steps        T >= 0; block_steps >= 1
 *   h0           [n] fp32, the state at the end of prefill [16 B]
 *   a, w         [T][n] fp32 decays and writes [16 B]
 *   err          [ceil(T / block_steps)][n] double, written [16 B]
 *   ref          as err, or NULL [16 B]
 *   codes        [n] codes of hq_T (2 B fp16/bf16, 1 B E4M3 and INT8, 4 B fp32, INT4
 *                two per byte), or NULL [16 B]
 *   scale        E4M3, INT8, INT4: [n / scale_group] scales of hq_T, or NULL [4 B]
 *   h_final      [n] fp32 h_T, or NULL [16 B]
 * q->scale_group: for the scaled formats a power of two from 4 to 256 entries
 * (the paper's blocks are 16 and 128); q->flags must be 0; q->entry_base is a
 * multiple of 16 as everywhere.
 */
ssmq_status ssmq_replay(const ssmq_qparams* q, int64_t n, int32_t steps, int32_t block_steps,
                        const float* h0, const float* a, const float* w, double* err, double* ref,
                        void* codes, float* scale, float* h_final, void* stream);

/* Static text for a status code. Never NULL. */
const char* ssmq_status_string(ssmq_status s);

/* Detail of the last non-OK status returned on this host thread ("" if none). */
const char* ssmq_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SSMQ_H */
