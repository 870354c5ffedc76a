// ssmq_device.hpp -- device primitives of the quantized state update (gfx950).
//
// Formats, thresholds and the dithered rounding of eq. (dither) (Section 2),
// written on bit patterns for the GPU. The rounding of a finite fp32 value x
// into a format whose grid drops k of x's fraction bits is decided in integer
// arithmetic:
//   eq. (dither) rounds the magnitude up exactly when u >= 1 - f (x > 0) or
//   u < f' (x < 0, f' the magnitude's fraction). With U = 2^24 u and R the k
//   dropped bits, for k <= 24 both cases read "R + (U_e >> (24 - k)) >= 2^k",
//   where U_e = U for x >= 0 and 2^24 - 1 - U for x < 0. Adding U_e >> (24-k)
//   to the magnitude and truncating therefore performs the rounding, carry into
//   the exponent included. In the 32-bit threshold word thr (U = thr >> 8),
//   U_e >> (24 - k) = (thr ^ signmask) >> (32 - k).
// The normal ranges of fp16 (k = 13), bf16 (k = 16) and E4M3 (k = 20) satisfy
// k <= 24. Below the smallest normal of fp16 and E4M3 the grid step is fixed,
// x / step has an exact fp32 integer part and fraction F, and the rule becomes
// the exact fp32 comparison F >= 1 - u (x >= 0) or F > u (x < 0).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ssmq_launch.hpp"

namespace ssmq {

enum Fmt : int { kFP16 = 0, kBF16 = 1, kE4M3 = 2, kFP32 = 3 };
enum Rule : int { kRTN = 0, kSR = 1, kWEYL = 2 };

// Weyl accumulator (Appendix B "Dithers", hardware form): 2^32 times
// 0.7548776662, 0.5698402910, 0.1234567, 0.3141592, rounded to nearest, and the
// 32-bit golden increment (Section 5.4).
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

template <int F> struct Traits;
template <> struct Traits<kFP16> { static constexpr int bytes = 2, V = 8; };
template <> struct Traits<kBF16> { static constexpr int bytes = 2, V = 8; };
template <> struct Traits<kE4M3> { static constexpr int bytes = 1, V = 16; };
template <> struct Traits<kFP32> { static constexpr int bytes = 4, V = 4; };

// ---------------------------------------------------------------------------
// Thresholds. A chunk is V consecutive entries starting at a flat index e0 that
// is a multiple of V; entry k of the chunk has index e0 + k.
// ---------------------------------------------------------------------------
// Weyl accumulator of entry e0 (without the (r+1), (c+1) ones, folded in key).
__device__ inline uint32_t weyl_base(uint64_t e0, const Thr& th) {
  const uint32_t r = static_cast<uint32_t>(e0 >> th.lb);
  const uint32_t c = static_cast<uint32_t>(e0) & ((1u << th.lb) - 1u);
  return kWeylA * r + kWeylB * c + th.key;
}
// Increment from entry e0 to e0 + k of an aligned chunk (valid when e0 is a
// multiple of the chunk size and the block is a power of two).
__device__ inline uint32_t weyl_off(uint32_t k, const Thr& th) {
  return kWeylA * (k >> th.lb) + kWeylB * (k & ((1u << th.lb) - 1u));
}

template <int R>
__device__ inline uint32_t thr_base(uint64_t e0, const Thr& th) {
  if constexpr (R == kWEYL) return weyl_base(e0, th);
  else if constexpr (R == kSR) return static_cast<uint32_t>(e0) * kSrEntry + th.key;
  else return 0u;
}
template <int R>
__device__ inline uint32_t thr_word(uint32_t base, uint32_t k, const Thr& th) {
  if constexpr (R == kWEYL) return base + weyl_off(k, th);
  else if constexpr (R == kSR) return fmix32(base + k * kSrEntry);
  else return 0x80000000u;
}

// ---------------------------------------------------------------------------
// Rounding fp32 -> code. thr: 32-bit threshold word, U = thr >> 8.
// ---------------------------------------------------------------------------
// Fixed-step region: |x| = T * step with T < 2^10 exact in fp32.
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

template <int F, int R>
__device__ inline uint32_t round_code(float x, uint32_t thr) {
  constexpr bool rtn = (R == kRTN);
  if constexpr (F == kBF16) return round_bf16<rtn>(x, thr);
  else if constexpr (F == kFP16) return round_fp16<rtn>(x, thr);
  else if constexpr (F == kE4M3) return round_e4m3<rtn>(x, thr);
  else return __float_as_uint(x);
}

// ---------------------------------------------------------------------------
// Decoding code -> fp32 (exact). E4M3 goes through the fp16 grid: the E4M3
// value of code c equals 256 times the binary16 value of
// ((c & 0x7F) << 7) | ((c & 0x80) << 8), subnormals included, so
// fl32(v * s) = fl32(fp16value * (256 s)) when 256 s is exact.
// ---------------------------------------------------------------------------
__device__ inline float fp16_bits_to_float(uint32_t h) {
  _Float16 v = __builtin_bit_cast(_Float16, static_cast<uint16_t>(h));
  return static_cast<float>(v);
}
template <int F>
__device__ inline float decode_code(uint32_t c, float s256) {
  if constexpr (F == kBF16) return __uint_as_float(c << 16);
  else if constexpr (F == kFP16) return fp16_bits_to_float(c);
  else if constexpr (F == kE4M3) {
    const float v = fp16_bits_to_float(((c & 0x7Fu) << 7) | ((c & 0x80u) << 8)) * s256;
    return ((c & 0x7Fu) == 0x7Fu) ? __uint_as_float(0x7FC00000u) : v;
  } else return __uint_as_float(c);
}

// Unpack / pack the codes of one 16-byte chunk.
template <int F>
__device__ inline uint32_t chunk_code(const uint4& raw, int k) {
  const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
  if constexpr (Traits<F>::bytes == 4) return w[k];
  else if constexpr (Traits<F>::bytes == 2) return (w[k >> 1] >> ((k & 1) * 16)) & 0xFFFFu;
  else return (w[k >> 2] >> ((k & 3) * 8)) & 0xFFu;
}
template <int F>
__device__ inline uint4 pack_chunk(const uint32_t (&c)[Traits<F>::V]) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if constexpr (Traits<F>::bytes == 4) w[i] = c[i];
    else if constexpr (Traits<F>::bytes == 2) w[i] = c[2 * i] | (c[2 * i + 1] << 16);
    else w[i] = c[4 * i] | (c[4 * i + 1] << 8) | (c[4 * i + 2] << 16) | (c[4 * i + 3] << 24);
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// E4M3 group scale: s = fl32(m / 448), flushed to zero below 2^-126.
__device__ inline float e4m3_scale(float m) {
  const float s = m / 448.0f;
  return (s >= 1.17549435e-38f) ? s : 0.0f;
}

}  // namespace ssmq
