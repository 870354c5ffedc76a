// ssmq_device.hpp -- device primitives of the quantized state update (gfx950).
//
// Formats, thresholds and the dithered rounding of eq. (dither) (Section 2).
//
// The rule. Write |x| = s (K + F) on the local grid of the format (K integer,
// F in [0, 1)), u = U / 2^24 with U the 24-bit threshold. Eq. (dither) is a
// signed floor, s floor(x/s + u): a positive x rounds up iff u >= 1 - F, a
// negative x rounds away from zero iff u < F. With R the k dropped fraction
// bits, for k <= 24 both read "R + (U_e >> (24 - k)) >= 2^k" where U_e = U for
// x >= 0 and U_e = 2^24 - 1 - U for x < 0, i.e. the magnitude is rounded up
// iff adding U_e's top k bits to it carries. In a 32-bit threshold word thr
// (U = thr >> 8), U_e is the top 24 bits of thr ^ signmask(x).
//
// Fast paths (the gfx950 conversions, checked on the device against the exact
// rule): v_cvt_sr_{bf16,f16,fp8}_f32(x, r) round |x| up iff the top 24 bits of
// r, added as above, carry; fed r = thr ^ signmask they implement eq. (dither)
// wherever k <= 24. The plain casts and v_cvt_pk_fp8_f32 are round-to-nearest-
// even. What they do not cover goes to the exact software path below, inside a
// branch that is taken by a wave only when one of its lanes needs it:
//   bf16  nothing (k = 16 everywhere; NaN and Inf come out canonical);
//   fp16  the subnormal range |x| < 2^-14 (the conversion is not exact there);
//   E4M3  NaN (the conversion loses its sign) and |q| < 2^-10, where k > 24.
// E4M3 values are clamped to +-448 (saturation) before the stochastic
// conversions, which do not saturate.
//
// INT8 / INT4 (symmetric, block scale, Appendix B "Formats") round q = h / s
// on the integer lattice. With q24 = h * (2^24 / s) (exactly q * 2^24 whenever
// q is a normal float), X = floor(q24) and U the 24-bit threshold,
// floor(q + U / 2^24) = (X + U) >> 24 exactly: only the top 24 fraction bits of
// q can decide the comparison with a multiple of 2^-24. The low byte (nibble)
// of X + U shifted right by 24 is the stored code. Values are clamped to
// +-qmax first (the bounds are lattice points, so this is the saturation);
// NaN and |q| < 2^-126 (q24 then differs from q * 2^24) take the exact path.
//
// Exact software path. Normal ranges use the carry rule on the magnitude bits.
// Below the smallest normal of fp16 and E4M3 the grid step is fixed, |x| / step
// has an exact fp32 integer part I and fraction F, and the rule is the exact
// fp32 comparison F >= 1 - u (x >= 0) or F > u (x < 0).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ssmq_launch.hpp"

namespace ssmq {

enum Fmt : int { kFP16 = 0, kBF16 = 1, kE4M3 = 2, kFP32 = 3, kINT8 = 4, kINT4 = 5 };
enum Rule : int { kRTN = 0, kSR = 1, kWEYL = 2, kPHILOX = 3 };

// Weyl accumulator (Appendix B "Dithers", hardware form): 2^32 times
// 0.7548776662, 0.5698402910, 0.1234567, 0.3141592, rounded to nearest, and the
// 32-bit golden increment (Section 6.4 "Three silent pitfalls").
constexpr uint32_t kWeylA = 0xC13FA9A9u;
constexpr uint32_t kWeylB = 0x91E10DA6u;
constexpr uint32_t kWeylL = 0x1F9ADBB9u;
constexpr uint32_t kWeylS = 0x506CBCC2u;
constexpr uint32_t kWeylPhi = 0x9E3779B9u;
// Hash SR multipliers: entry and step (Appendix B "Decode regime"), layer.
constexpr uint32_t kSrEntry = 0x9E3779B1u;
constexpr uint32_t kSrStep = 0x85EBCA77u;
constexpr uint32_t kSrLayer = 0xC2B2AE3Du;

// MurmurHash3 32-bit finalizer.
__host__ __device__ inline uint32_t fmix32(uint32_t h) {
  h ^= h >> 16;
  h *= 0x85EBCA6Bu;
  h ^= h >> 13;
  h *= 0xC2B2AE35u;
  h ^= h >> 16;
  return h;
}

// Per-step threshold keys (host and device). Weyl: the entry-independent part
// A + B + L layer + S seed + Phi t of the accumulator; hash SR: the chained key
// fmix32(fmix32(fmix32(seed) ^ layer * kSrLayer) ^ t * kSrStep).
__host__ __device__ inline uint32_t weyl_step_key(uint32_t seed, uint32_t layer, uint32_t step) {
  return kWeylA + kWeylB + kWeylL * layer + kWeylS * seed + kWeylPhi * step;
}
__host__ __device__ inline uint32_t sr_seed_key(uint32_t seed, uint32_t layer) {
  return fmix32(fmix32(seed) ^ (layer * kSrLayer));
}
__host__ __device__ inline uint32_t sr_step_key(uint32_t seed_key, uint32_t step) {
  return fmix32(seed_key ^ (step * kSrStep));
}

// A chunk is the unit one lane loads and stores: V entries in CB bytes (16, or
// 8 for INT4). Scaled formats keep one fp32 scale per group of entries;
// qmax is the value the group maximum is mapped to.
template <int F> struct Traits;
template <> struct Traits<kFP16> { static constexpr int V = 8, CB = 16; static constexpr bool scaled = false; };
template <> struct Traits<kBF16> { static constexpr int V = 8, CB = 16; static constexpr bool scaled = false; };
template <> struct Traits<kFP32> { static constexpr int V = 4, CB = 16; static constexpr bool scaled = false; };
// zh = fl32(1 / qmax) and zl = fl32(1 / qmax - zh) serve the group-scale division.
template <> struct Traits<kE4M3> {
  static constexpr int V = 16, CB = 16; static constexpr bool scaled = true;
  static constexpr float qmax = 448.0f, zh = 0x1.24924ap-9f, zl = -0x1.b6db6ep-34f;
};
template <> struct Traits<kINT8> {
  static constexpr int V = 16, CB = 16; static constexpr bool scaled = true;
  static constexpr float qmax = 127.0f, zh = 0x1.020408p-7f, zl = 0x1.020408p-35f;
};
template <> struct Traits<kINT4> {
  static constexpr int V = 16, CB = 8; static constexpr bool scaled = true;
  static constexpr float qmax = 7.0f, zh = 0x1.24924ap-3f, zl = -0x1.b6db6ep-28f;
};
template <int F> constexpr bool is_int_fmt = (F == kINT8 || F == kINT4);

template <int CB> struct ChunkOf;
template <> struct ChunkOf<16> { using type = uint4; };
template <> struct ChunkOf<8> { using type = uint2; };
template <int F> using chunk_t = typename ChunkOf<Traits<F>::CB>::type;

// Byte offset of the chunk that starts at entry e (a multiple of V).
template <int F, typename I>
__host__ __device__ constexpr I chunk_bytes_at(I e) {
  return e / static_cast<I>(Traits<F>::V) * static_cast<I>(Traits<F>::CB);
}

typedef float v2f __attribute__((ext_vector_type(2)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));
typedef _Float16 v2h __attribute__((ext_vector_type(2)));
typedef unsigned int v4u __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// Thresholds. A chunk is V consecutive entries starting at a flat index e0 that
// is a multiple of V; entry k of the chunk uses thr_word(base(e0), off[k]) with
// off[k] precomputed on the host (Weyl: A (k >> lb) + B (k & (block-1)); SR:
// k * 0x9E3779B1).
// ---------------------------------------------------------------------------
template <int R>
__device__ inline uint32_t thr_base(uint64_t e0, const Thr& th) {
  if constexpr (R == kWEYL) {
    const uint32_t r = static_cast<uint32_t>(e0 >> th.lb);
    const uint32_t c = static_cast<uint32_t>(e0) & ((1u << th.lb) - 1u);
    return kWeylA * r + kWeylB * c + th.key;
  } else if constexpr (R == kSR) {
    return static_cast<uint32_t>(e0) * kSrEntry + th.key;
  } else {
    return 0u;
  }
}
template <int R>
__device__ inline uint32_t thr_word(uint32_t base, uint32_t off) {
  if constexpr (R == kWEYL) return base + off;
  else if constexpr (R == kSR) return fmix32(base + off);
  else return 0x80000000u;
}

// Philox4x32-10 (Salmon et al., SC 2011): ten rounds of two 32x32->64-bit
// products on a four-word counter, key advanced by the Weyl increments.
__device__ inline void philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                     uint32_t k0, uint32_t k1, uint32_t (&out)[4]) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = static_cast<uint64_t>(0xD2511F53u) * c0;
    const uint64_t p1 = static_cast<uint64_t>(0xCD9E8D57u) * c2;
    // three-input XORs in one v_bitop3_b32 each (truth table 0x96)
    const uint32_t n0 = __builtin_amdgcn_bitop3_b32(static_cast<uint32_t>(p1 >> 32), c1, k0, 0x96);
    const uint32_t n2 = __builtin_amdgcn_bitop3_b32(static_cast<uint32_t>(p0 >> 32), c3, k1, 0x96);
    c1 = static_cast<uint32_t>(p1);
    c3 = static_cast<uint32_t>(p0);
    c0 = n0;
    c2 = n2;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

// Thresholds of one chunk of N entries whose first flat index is e0: tg(k) is
// the 32-bit word of entry k (U = word >> 8). Weyl and hash SR derive it from
// a per-chunk base and the per-position offsets; Philox SR draws word
// (e0 + k) mod 4 of the block with counter ((e0 + k) / 4, step, 0) and key
// (seed, layer).
template <int R, int N>
struct ChunkThr {
  uint32_t base;
  const uint32_t* off;
  __device__ uint32_t operator()(int k) const { return thr_word<R>(base, off[k]); }
};
template <int N>
struct ChunkThr<kPHILOX, N> {
  uint32_t w[N];
  __device__ uint32_t operator()(int k) const { return w[k]; }
};

// The 32-bit threshold word of one entry with global flat index i.
template <int R>
__device__ inline uint32_t entry_thr(uint64_t i, const Thr& th) {
  if constexpr (R == kPHILOX) {
    const uint64_t q = i >> 2;
    uint32_t o[4];
    philox4x32_10(static_cast<uint32_t>(q), static_cast<uint32_t>(q >> 32), th.step, 0u, th.seed,
                  th.layer, o);
    const uint32_t j = static_cast<uint32_t>(i) & 3u;
    return j == 0 ? o[0] : (j == 1 ? o[1] : (j == 2 ? o[2] : o[3]));
  } else {
    return thr_word<R>(thr_base<R>(i, th), 0u);
  }
}

template <int R, int N>
__device__ inline ChunkThr<R, N> chunk_thr(uint64_t e0, const Thr& th, uint32_t base,
                                           const uint32_t* off) {
  if constexpr (R == kPHILOX) {
    static_assert(N % 4 == 0, "Philox blocks cover four entries");
    ChunkThr<R, N> t;
    const uint64_t q0 = e0 >> 2;
#pragma unroll
    for (int g = 0; g < N / 4; ++g) {
      const uint64_t q = q0 + static_cast<uint64_t>(g);
      uint32_t o[4];
      philox4x32_10(static_cast<uint32_t>(q), static_cast<uint32_t>(q >> 32), th.step, 0u,
                    th.seed, th.layer, o);
#pragma unroll
      for (int i = 0; i < 4; ++i) t.w[4 * g + i] = o[i];
    }
    return t;
  } else {
    return ChunkThr<R, N>{base, off};
  }
}

// thr ^ signmask(x) in the top 24 bits (the low byte is don't-care).
__device__ inline uint32_t signed_thr(uint32_t thr, float x) {
  return thr ^ static_cast<uint32_t>(static_cast<int32_t>(__float_as_uint(x)) >> 24);
}

// ---------------------------------------------------------------------------
// Exact software rounding fp32 -> code.
// ---------------------------------------------------------------------------
template <bool RTN>
__device__ inline uint32_t round_fixed_step(float T, uint32_t neg, uint32_t thr) {
  const float I = floorf(T);
  const float F = T - I;  // exact
  bool up;
  if constexpr (RTN) {
    up = (F > 0.5f) || (F == 0.5f && (static_cast<uint32_t>(I) & 1u));
  } else {
    const uint32_t U = thr >> 8;
    up = neg ? (F > static_cast<float>(U) * 0x1p-24f)
             : (F >= static_cast<float>(0x1000000u - U) * 0x1p-24f);
  }
  return static_cast<uint32_t>(I) + (up ? 1u : 0u);
}

template <bool RTN>
__device__ inline uint32_t round_bf16(float x, uint32_t thr) {
  const uint32_t b = __float_as_uint(x);
  uint32_t add;
  if constexpr (RTN) {
    add = 0x7FFFu + ((b >> 16) & 1u);
  } else {
    const uint32_t sm = static_cast<uint32_t>(static_cast<int32_t>(b) >> 31);
    add = (thr ^ sm) >> 16;
  }
  uint32_t c = (b + add) >> 16;
  if ((b & 0x7FFFFFFFu) > 0x7F800000u) c = ((b >> 16) & 0x8000u) | 0x7FC0u;
  return c;
}

template <bool RTN>
__device__ inline uint32_t round_fp16(float x, uint32_t thr) {
  const uint32_t b = __float_as_uint(x);
  const uint32_t sign = (b >> 16) & 0x8000u;
  const uint32_t m = b & 0x7FFFFFFFu;
  uint32_t c;
  if (m >= 0x38800000u) {  // |x| >= 2^-14: normal range (k = 13) or overflow
    uint32_t add;
    if constexpr (RTN) {
      add = 0xFFFu + ((m >> 13) & 1u);
    } else {
      const uint32_t sm = static_cast<uint32_t>(static_cast<int32_t>(b) >> 31);
      add = (thr ^ sm) >> 19;
    }
    c = min(((m + add) >> 13) - (112u << 10), 0x7C00u);
  } else {                 // subnormal grid, step 2^-24
    c = round_fixed_step<RTN>(__uint_as_float(m) * 16777216.0f, sign, thr);
  }
  if (m > 0x7F800000u) c = 0x7E00u;
  return c | sign;
}

template <bool RTN>
__device__ inline uint32_t round_e4m3(float q, uint32_t thr) {
  const uint32_t b = __float_as_uint(q);
  const uint32_t sign = (b >> 24) & 0x80u;
  uint32_t m = b & 0x7FFFFFFFu;
  if (m > 0x7F800000u) return 0x7Fu | sign;  // NaN
  m = min(m, 0x43E00000u);                   // saturate at 448
  uint32_t c;
  if (m >= 0x3C800000u) {  // |q| >= 2^-6: normal range (k = 20)
    uint32_t add;
    if constexpr (RTN) {
      add = 0x7FFFFu + ((m >> 20) & 1u);
    } else {
      const uint32_t sm = static_cast<uint32_t>(static_cast<int32_t>(b) >> 31);
      add = (thr ^ sm) >> 12;
    }
    c = ((m + add) >> 20) - 960u;
  } else {                 // subnormal grid, step 2^-9
    c = round_fixed_step<RTN>(__uint_as_float(m) * 512.0f, sign, thr);
  }
  return c | sign;
}

// INT lattice, exact: q = h / s clamped to [-qmax, qmax], then floor(q + u)
// via the exact fp32 fraction (RTN: nearest, ties to even); NaN -> 0. Returns
// the two's complement code in the low bits.
template <bool RTN>
__device__ inline uint32_t round_int(float q, uint32_t thr, float qmax) {
  if (q != q) return 0u;
  q = fminf(fmaxf(q, -qmax), qmax);
  int k;
  if constexpr (RTN) {
    k = static_cast<int>(__builtin_rintf(q));
  } else {
    const float I = floorf(q);
    const float Fr = q - I;  // exact
    const uint32_t U = thr >> 8;
    k = static_cast<int>(I) + (Fr >= static_cast<float>(0x1000000u - U) * 0x1p-24f ? 1 : 0);
  }
  return static_cast<uint32_t>(k);
}

template <int F, int R>
__device__ inline uint32_t round_code(float x, uint32_t thr) {
  constexpr bool rtn = (R == kRTN);
  if constexpr (F == kBF16) return round_bf16<rtn>(x, thr);
  else if constexpr (F == kFP16) return round_fp16<rtn>(x, thr);
  else if constexpr (F == kE4M3) return round_e4m3<rtn>(x, thr);
  else if constexpr (F == kINT8) return round_int<rtn>(x, thr, 127.0f) & 0xFFu;
  else if constexpr (F == kINT4) return round_int<rtn>(x, thr, 7.0f) & 0xFu;
  else return __float_as_uint(x);
}

// ---------------------------------------------------------------------------
// Chunk quantizers: one chunk of fp32 values -> its codes, fast path plus the
// exact path for rare entries (the unscaled float formats here, E4M3 and the
// integer formats, which also take the group's 1 / s, further below).
// ---------------------------------------------------------------------------
template <int F>
__device__ inline void patch_code(uint32_t (&w)[4], int k, uint32_t c) {
  constexpr int bits = Traits<F>::CB * 8 / Traits<F>::V;  // code width
  if constexpr (bits == 32) {
    w[k] = c;
  } else {
    constexpr int per = 32 / bits;
    const int i = k / per, sh = (k % per) * bits;
    const uint32_t mask = ((1u << bits) - 1u) << sh;
    w[i] = (w[i] & ~mask) | ((c << sh) & mask);
  }
}

template <int F, int R>
__device__ inline bool needs_exact_path(float v) {
  if constexpr (F == kE4M3) {
    if constexpr (R == kRTN) return v != v;                            // NaN
    else return !(__builtin_fabsf(v) >= 0x1p-10f);                     // NaN or k > 24
  } else if constexpr (F == kFP16) {
    if constexpr (R == kRTN) return false;
    else return __builtin_fabsf(v) < 0x1p-14f;                         // subnormal range
  } else {
    return false;
  }
}

// Does any value of the chunk need the exact path (fp16 below its normal range)?
// The small-magnitude test uses the chunk minimum (fminf ignores NaN).
template <int F, int R, int V>
__device__ inline bool chunk_is_rare(const float (&v)[V]) {
  if constexpr (F != kFP16 || R == kRTN) {
    return false;
  } else {
    float mn = __builtin_fabsf(v[0]);
#pragma unroll
    for (int k = 1; k < V; ++k) mn = fminf(mn, __builtin_fabsf(v[k]));
    return mn < 0x1p-14f;
  }
}

// Whether any of the chunk's values is NaN, for callers without a cheaper test.
template <int V>
__device__ inline bool chunk_has_nan(const float (&v)[V]) {
  bool n = false;
#pragma unroll
  for (int k = 0; k < V; k += 2) n |= __builtin_isunordered(v[k], v[k + 1]);
  return n;
}

// The unscaled float formats need no NaN test: their conversions give the
// canonical NaN (maybe_nan is accepted for a uniform interface).
template <int F, int R, typename TG>
__device__ inline uint4 quantize_chunk(const float (&v)[Traits<F>::V], const TG& tg,
                                       bool /*maybe_nan*/) {
  static_assert(F == kBF16 || F == kFP16 || F == kFP32, "unscaled float formats");
  uint32_t w[4];
  if constexpr (F == kFP32) {
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = __float_as_uint(v[i]);
    return make_uint4(w[0], w[1], w[2], w[3]);
  }
  if constexpr (F == kBF16) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v2bf p;
      if constexpr (R == kRTN) {
        p = (v2bf){static_cast<__bf16>(v[2 * i]), static_cast<__bf16>(v[2 * i + 1])};
      } else {
        // Both halves are written, so the destination's previous contents are
        // don't-care: it starts as the first threshold, which dies here.
        const uint32_t t0 = signed_thr(tg(2 * i), v[2 * i]);
        p = __builtin_amdgcn_cvt_sr_bf16_f32(__builtin_bit_cast(v2bf, t0), v[2 * i], t0, false);
        p = __builtin_amdgcn_cvt_sr_bf16_f32(
            p, v[2 * i + 1], signed_thr(tg(2 * i + 1), v[2 * i + 1]), true);
      }
      w[i] = __builtin_bit_cast(uint32_t, p);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v2h p;
      if constexpr (R == kRTN) {
        p = (v2h){static_cast<_Float16>(v[2 * i]), static_cast<_Float16>(v[2 * i + 1])};
      } else {
        const uint32_t t0 = signed_thr(tg(2 * i), v[2 * i]);
        p = __builtin_amdgcn_cvt_sr_f16_f32(__builtin_bit_cast(v2h, t0), v[2 * i], t0, false);
        p = __builtin_amdgcn_cvt_sr_f16_f32(
            p, v[2 * i + 1], signed_thr(tg(2 * i + 1), v[2 * i + 1]), true);
      }
      w[i] = __builtin_bit_cast(uint32_t, p);
    }
  }
  if (__builtin_amdgcn_ballot_w64(chunk_is_rare<F, R, Traits<F>::V>(v)) != 0) {
#pragma unroll
    for (int k = 0; k < Traits<F>::V; ++k) {
      if (needs_exact_path<F, R>(v[k])) patch_code<F>(w, k, round_code<F, R>(v[k], tg(k)));
    }
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// E4M3 chunk of 16 entries: h the fp32 values, r = fl32(1 / s) of their group.
// Values q = fl32(h r) exceed 448 only by the scale's own rounding (the scale
// maps the group maximum to 448): the stochastic conversions, which do not
// saturate, get q clamped with v_med3_f32 (clamping first is eq. (dither) on
// the saturated grid) unless the caller knows that no q of the group passes 448
// (clamp = false, wave-uniform: fl32(max|h| r) <= 448, rounding is monotonic);
// round-to-nearest needs no clamp below 464, which a scaled value never
// reaches. The exact path takes NaN (maybe_nan: a NaN may be among h) and
// |q| < 2^-10; since fl32(x r) is monotonic in x, the smallest |q| is
// fl32(min|h| r), one product per chunk.
template <int R, typename TG>
__device__ inline uint4 quantize_e4m3_chunk(const float (&h)[16], float r, const TG& tg,
                                            bool maybe_nan, bool clamp) {
  float q[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) q[k] = h[k] * r;
  // Philox SR always clamps: its generator already fills the registers that a
  // second code path would need.
  if (R != kRTN && (R == kPHILOX || clamp)) {
#pragma unroll
    for (int k = 0; k < 16; ++k) q[k] = __builtin_amdgcn_fmed3f(q[k], -448.0f, 448.0f);
  }
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int k = 4 * i;
    int d;  // all four bytes are written: the previous contents are don't-care
    if constexpr (R == kRTN) {
      d = __builtin_amdgcn_cvt_pk_fp8_f32(q[k], q[k + 1], static_cast<int>(__float_as_uint(q[k])), false);
      d = __builtin_amdgcn_cvt_pk_fp8_f32(q[k + 2], q[k + 3], d, true);
    } else {
      const uint32_t t0 = signed_thr(tg(k), q[k]);  // dies here
      d = __builtin_amdgcn_cvt_sr_fp8_f32(q[k], t0, static_cast<int>(t0), 0);
      d = __builtin_amdgcn_cvt_sr_fp8_f32(q[k + 1], signed_thr(tg(k + 1), q[k + 1]), d, 1);
      d = __builtin_amdgcn_cvt_sr_fp8_f32(q[k + 2], signed_thr(tg(k + 2), q[k + 2]), d, 2);
      d = __builtin_amdgcn_cvt_sr_fp8_f32(q[k + 3], signed_thr(tg(k + 3), q[k + 3]), d, 3);
    }
    w[i] = static_cast<uint32_t>(d);
  }
  bool rare = maybe_nan;
  if constexpr (R != kRTN) {
    // Started from +infinity, the chain is eight v_min3 with |h| as source
    // modifiers (from |h[0]| the compiler first canonicalises two values). A NaN in
    // h is caught by maybe_nan: it reaches the row's y.
    float mn = __builtin_inff();
#pragma unroll
    for (int k = 0; k < 16; ++k) mn = fminf(mn, __builtin_fabsf(h[k]));
    rare = rare || !(mn * r >= 0x1p-10f);
  }
  if (__builtin_amdgcn_ballot_w64(rare) != 0) {
    // The products are formed again here (r passed through an empty asm so that
    // they are not shared with q): q then needs no copy to survive the clamp.
    float rr = r;
    asm volatile("" : "+v"(rr));
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const float v = h[k] * rr;
      if (needs_exact_path<kE4M3, R>(v)) patch_code<kE4M3>(w, k, round_code<kE4M3, R>(v, tg(k)));
    }
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// Byte `b` of each of four words, packed little-end first (v_perm_b32).
template <int B>
__device__ inline uint32_t pack_bytes(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3) {
  constexpr uint32_t lo = (0x0C0Cu << 16) | ((4u + B) << 8) | B;  // {w0.b, w1.b, 0, 0}
  const uint32_t p01 = __builtin_amdgcn_perm(w1, w0, lo);
  const uint32_t p23 = __builtin_amdgcn_perm(w3, w2, lo);
  return __builtin_amdgcn_perm(p23, p01, 0x05040100u);
}

// INT8 / INT4 chunk of 16 entries. h: the fp32 values, r = fl32(1 / s) and
// r24 = 2^24 r of their group (r24 is infinite when 2^24 r overflows);
// maybe_nan: a NaN may be among h. Values are clamped to +-qmax before the
// floor (the bounds are lattice points, so this is the exact saturation).
template <int F, int R, typename TG>
__device__ inline chunk_t<F> quantize_int_chunk(const float (&h)[16], float r, float r24,
                                               const TG& tg, bool maybe_nan) {
  constexpr float qmax = Traits<F>::qmax;
  uint32_t S[16];
  bool rare = maybe_nan;
  if constexpr (R == kRTN) {
    // Adding 1.5 * 2^23 rounds the clamped q to an integer, ties to even (the
    // sum's ulp is 1), and leaves that integer's two's complement in the low
    // bits of the sum's encoding.
#pragma unroll
    for (int k = 0; k < 16; ++k)
      S[k] = __float_as_uint(__builtin_amdgcn_fmed3f(h[k] * r, -qmax, qmax) + 0x1.8p23f);
  } else {
    float mn = __builtin_inff();
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const float q24 = h[k] * r24;
      mn = fminf(mn, __builtin_fabsf(q24));
      int X;  // floor of the clamped value
      asm("v_cvt_flr_i32_f32 %0, %1"
          : "=v"(X)
          : "v"(__builtin_amdgcn_fmed3f(q24, -qmax * 0x1p24f, qmax * 0x1p24f)));
      S[k] = static_cast<uint32_t>(X) + (tg(k) >> 8);
    }
    rare = rare || !(mn >= 0x1p-102f) || !(r24 < __builtin_inff());
  }
  constexpr int B = (R == kRTN) ? 0 : 3;  // the byte that holds the code
  uint32_t w[4];
  if constexpr (F == kINT8) {
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = pack_bytes<B>(S[4 * i], S[4 * i + 1], S[4 * i + 2], S[4 * i + 3]);
  } else {
    // even entries' bytes in one word, odd entries' in another, then nibble-interleave
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int k = 8 * i;
      const uint32_t ev = pack_bytes<B>(S[k], S[k + 2], S[k + 4], S[k + 6]);
      const uint32_t od = pack_bytes<B>(S[k + 1], S[k + 3], S[k + 5], S[k + 7]);
      w[i] = (ev & 0x0F0F0F0Fu) | ((od << 4) & 0xF0F0F0F0u);
    }
    w[2] = w[3] = 0u;
  }
  if (__builtin_amdgcn_ballot_w64(rare) != 0) {
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      bool exact;
      if constexpr (R == kRTN) {
        exact = h[k] != h[k];
      } else {
        // NaN, q below the normal range (q24 then differs from q 2^24), or r24 overflowed
        exact = !(__builtin_fabsf(h[k] * r24) >= 0x1p-102f) || !(r24 < __builtin_inff());
      }
      if (exact) patch_code<F>(w, k, round_code<F, R>(h[k] * r, tg(k)));
    }
  }
  if constexpr (F == kINT8) return make_uint4(w[0], w[1], w[2], w[3]);
  else return make_uint2(w[0], w[1]);
}

// One chunk of fp32 values h -> codes, for every format: r = 1 / s of the
// chunk's group (ignored by unscaled formats).
template <int F, int R, typename TG>
__device__ inline chunk_t<F> quantize_any(const float (&h)[Traits<F>::V], float r, const TG& tg,
                                         bool maybe_nan, bool clamp = true) {
  if constexpr (is_int_fmt<F>) {
    return quantize_int_chunk<F, R>(h, r, r * 0x1p24f, tg, maybe_nan);
  } else if constexpr (F == kE4M3) {
    return quantize_e4m3_chunk<R>(h, r, tg, maybe_nan, clamp);
  } else {
    return quantize_chunk<F, R>(h, tg, maybe_nan);
  }
}

// The exact fp32 value of one code (E4M3 and INT without the group scale).
template <int F>
__device__ inline float code_value(uint32_t c) {
  if constexpr (F == kBF16) return __uint_as_float(c << 16);
  else if constexpr (F == kFP16) return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(c)));
  else if constexpr (F == kE4M3) return __builtin_amdgcn_cvt_f32_fp8(static_cast<int>(c), 0);
  else if constexpr (F == kINT8) return static_cast<float>(static_cast<int32_t>(c << 24) >> 24);
  else if constexpr (F == kINT4) return static_cast<float>(static_cast<int32_t>(c << 28) >> 28);
  else return __uint_as_float(c);
}

// ---------------------------------------------------------------------------
// Decoding code -> its exact value as fp32 (E4M3 without the group scale, via
// v_cvt_pk_f32_fp8, which decodes OCP E4M3 exactly).
// ---------------------------------------------------------------------------
template <int F>
__device__ inline void decode_chunk(const uint2& raw, float (&out)[Traits<F>::V]) {
  static_assert(F == kINT4, "8-byte chunks hold INT4 codes");
  const uint32_t w[2] = {raw.x, raw.y};
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j)
      out[8 * i + j] = static_cast<float>(static_cast<int32_t>(w[i] << (28 - 4 * j)) >> 28);
}

template <int F>
__device__ inline void decode_chunk(const uint4& raw, float (&out)[Traits<F>::V]) {
  const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if constexpr (F == kBF16) {
      out[2 * i] = __uint_as_float(w[i] << 16);
      out[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    } else if constexpr (F == kFP16) {
      const v2h p = __builtin_bit_cast(v2h, w[i]);
      out[2 * i] = static_cast<float>(p.x);
      out[2 * i + 1] = static_cast<float>(p.y);
    } else if constexpr (F == kE4M3) {
      const v2f lo = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w[i]), false);
      const v2f hi = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w[i]), true);
      out[4 * i] = lo.x;
      out[4 * i + 1] = lo.y;
      out[4 * i + 2] = hi.x;
      out[4 * i + 3] = hi.y;
    } else if constexpr (F == kINT8) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        out[4 * i + j] = static_cast<float>(static_cast<int8_t>(w[i] >> (8 * j)));
    } else {
      out[i] = __uint_as_float(w[i]);
    }
  }
}

// Group scale of a scaled format: s = fl32(m / qmax), flushed to zero below
// 2^-126. For m in [2^-112, FLT_MAX], fma(m, zh, fl32(m zl)) is the correctly
// rounded quotient (Brisebarre, Muller and Raina, "Accelerating correctly rounded
// floating-point division when the divisor is known in advance", 2004; checked
// here for every such fp32 m and qmax = 7, 127, 448); smaller or infinite m
// divide (a wave-uniform branch, taken only by waves that hold such a group).
template <int F>
__device__ inline float group_scale(float m) {
  float s = fmaf(m, Traits<F>::zh, m * Traits<F>::zl);
  const bool slow = !(m >= 0x1p-112f && m <= 3.40282347e38f);
  if (__builtin_amdgcn_ballot_w64(slow) != 0) {
    // The empty asm keeps the division inside the branch: hoisted out of it
    // (the compiler's choice for a cheap-looking fdiv), every group pays for it.
    float mm = m;
    asm volatile("" : "+v"(mm));
    if (slow) s = mm / Traits<F>::qmax;
  }
  return (s >= 1.17549435e-38f) ? s : 0.0f;
}

// r = fl32(1 / s) for a group scale s: 0 for s = 0 or s infinite; otherwise
// s lies in [2^-126, 2^126), where one Newton step from v_rcp_f32,
// fma(fma(-s, y0, 1), y0, y0), is the correctly rounded reciprocal (checked on
// the device for every fp32 value in that range).
__device__ inline float recip_scale(float s) {
  const float y0 = __builtin_amdgcn_rcpf(s);
  const float r = fmaf(fmaf(-s, y0, 1.0f), y0, y0);
  return (s > 0.0f && s < __builtin_inff()) ? r : 0.0f;
}

// ---------------------------------------------------------------------------
// Cross-lane reductions over aligned groups of `width` lanes (a power of two
// <= 64): DPP within 16-lane rows, then swizzles across rows.
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ inline float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                               CTRL, 0xF, 0xF, false));
}
constexpr int kQuadXor1 = 0xB1;     // quad_perm [1,0,3,2]
constexpr int kQuadXor2 = 0x4E;     // quad_perm [2,3,0,1]
constexpr int kHalfMirror = 0x141;  // lane i <-> 7 - i within 8
constexpr int kRowMirror = 0x140;   // lane i <-> 15 - i within 16

__device__ inline float lane_sum(float v, int width) {
  if (width >= 2) v += dpp_f<kQuadXor1>(v);
  if (width >= 4) v += dpp_f<kQuadXor2>(v);
  if (width >= 8) v += dpp_f<kHalfMirror>(v);
  if (width >= 16) v += dpp_f<kRowMirror>(v);
  if (width >= 32) v += __shfl_xor(v, 16, 64);
  if (width >= 64) v += __shfl_xor(v, 32, 64);
  return v;
}
template <int CTRL>
__device__ inline uint32_t dpp_u(uint32_t v) {
  return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), CTRL, 0xF, 0xF, false));
}
// Maximum of unsigned words (bit patterns of non-negative, non-NaN floats).
__device__ inline uint32_t lane_umax(uint32_t v, int width) {
  if (width >= 2) v = max(v, dpp_u<kQuadXor1>(v));
  if (width >= 4) v = max(v, dpp_u<kQuadXor2>(v));
  if (width >= 8) v = max(v, dpp_u<kHalfMirror>(v));
  if (width >= 16) v = max(v, dpp_u<kRowMirror>(v));
  if (width >= 32) v = max(v, static_cast<uint32_t>(__shfl_xor(static_cast<int>(v), 16, 64)));
  if (width >= 64) v = max(v, static_cast<uint32_t>(__shfl_xor(static_cast<int>(v), 32, 64)));
  return v;
}

// Streaming (nontemporal) 16- and 8-byte accesses for the state.
typedef unsigned int v2u __attribute__((ext_vector_type(2)));
template <typename C>
__device__ inline C load_stream(const void* p);
template <>
__device__ inline uint4 load_stream<uint4>(const void* p) {
  const v4u v = __builtin_nontemporal_load(static_cast<const v4u*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
template <>
__device__ inline uint2 load_stream<uint2>(const void* p) {
  const v2u v = __builtin_nontemporal_load(static_cast<const v2u*>(p));
  return make_uint2(v.x, v.y);
}
__device__ inline void store_stream(void* p, const uint4& v) {
  const v4u w = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(w, static_cast<v4u*>(p));
}
__device__ inline void store_stream(void* p, const uint2& v) {
  const v2u w = {v.x, v.y};
  __builtin_nontemporal_store(w, static_cast<v2u*>(p));
}

}  // namespace ssmq
