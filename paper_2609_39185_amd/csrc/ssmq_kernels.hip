// ssmq_kernels.hip -- HIP kernels of the quantized selective-state update (gfx950).
//
// Kernels:
//   k_update_head  one 256-thread workgroup per (batch, head) tile of a Mamba-2
//                  state (scalar A per head): dequantize -> exp(dt A) -> FMA
//                  recurrence -> y = C h + D x -> (E4M3 group scale) -> threshold
//                  -> round -> store, all in registers; the state crosses HBM
//                  once each way (Section 2 eq. (rec) and eq. (dither);
//                  Appendix B "Runners", "Formats", "Dithers").
//   k_update_rows  the same step for any row layout (Mamba-1 with A per (channel,
//                  n), and Mamba-2 shapes that do not fill a head tile).
//   k_requant      fp32 -> codes for fp16 / bf16 / fp32, 16 entries per thread.
//   k_requant_e4m3 fp32 -> E4M3 codes with group scales, a wave per group.
//   k_dither_fill  the 24-bit thresholds themselves.
//
// Thread layout of the update kernels: a chunk is 16 bytes of codes (V entries
// of one state row). The LR = dstate / V chunks of a row sit in LR consecutive
// lanes of one wave, so C.h is a reduction over LR lanes and a row's B and C
// slice is fixed per lane.
#include "ssmq_device.hpp"

namespace ssmq {

__device__ inline float lane_sum(float v, int width) {
  for (int o = width >> 1; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ inline float lane_max(float v, int width) {
  for (int o = width >> 1; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

template <int F>
__device__ inline uint4 load_chunk(const void* base, int64_t entry) {
  return *reinterpret_cast<const uint4*>(static_cast<const uint8_t*>(base) +
                                         entry * Traits<F>::bytes);
}
template <int F>
__device__ inline void store_chunk(void* base, int64_t entry, uint4 v) {
  *reinterpret_cast<uint4*>(static_cast<uint8_t*>(base) + entry * Traits<F>::bytes) = v;
}

template <int V>
__device__ inline void load_floats(const float* p, float (&out)[V]) {
#pragma unroll
  for (int i = 0; i < V; i += 4) {
    const float4 v = *reinterpret_cast<const float4*>(p + i);
    out[i] = v.x; out[i + 1] = v.y; out[i + 2] = v.z; out[i + 3] = v.w;
  }
}

// Quantize the V fp32 values of one chunk (E4M3: times r = 1/scale first).
template <int F, int R>
__device__ inline uint4 quantize_chunk(const float (&h)[Traits<F>::V], float r, uint64_t e0,
                                       const Thr& th) {
  constexpr int V = Traits<F>::V;
  uint32_t c[V];
  const uint32_t base = thr_base<R>(e0, th);
#pragma unroll
  for (int k = 0; k < V; ++k) {
    const float v = (F == kE4M3) ? h[k] * r : h[k];
    c[k] = round_code<F, R>(v, thr_word<R>(base, static_cast<uint32_t>(k), th));
  }
  return pack_chunk<F>(c);
}

// ---------------------------------------------------------------------------
// Mamba-2 head tile: headdim * dstate = 256 * CPT * V entries per workgroup.
// ---------------------------------------------------------------------------
template <int F, int R, int CPT>
__global__ __launch_bounds__(256) void k_update_head(UpdateArgs a) {
  constexpr int V = Traits<F>::V;
  const int t = threadIdx.x;
  const int64_t tile = blockIdx.x;  // b * nheads + h
  const int hh = static_cast<int>(tile % a.nheads);
  const int64_t b = tile / a.nheads;
  const int g = hh / a.heads_per_group;
  const int cc = t & (a.lanes_per_row - 1);
  const int n0 = cc * V;
  const int r0 = t >> a.lr_shift;
  const int rows_per_pass = 256 >> a.lr_shift;
  const int64_t tile_base = tile * a.head_size;

  uint4 raw[CPT];
  float xv[CPT];
#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    const int p = j * rows_per_pass + r0;
    raw[j] = load_chunk<F>(a.state, tile_base + static_cast<int64_t>(p) * a.dstate + n0);
    xv[j] = a.x[tile * a.headdim + p];
  }
  float Bv[V], Cv[V];
  load_floats<V>(a.B + (b * a.ngroups + g) * a.dstate + n0, Bv);
  load_floats<V>(a.C + (b * a.ngroups + g) * a.dstate + n0, Cv);
  const float dtv = a.dt[tile];
  const float dA = static_cast<float>(exp(static_cast<double>(dtv * a.A[hh])));
  const float Dv = a.D ? a.D[hh] : 0.0f;

  // old E4M3 scales (times 256, see decode_code)
  float s256[CPT];
#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    s256[j] = 0.0f;
    if constexpr (F == kE4M3) {
      const int p = j * rows_per_pass + r0;
      const int64_t e = tile_base + static_cast<int64_t>(p) * a.dstate + n0;
      s256[j] = a.scale[e / a.group] * 256.0f;
    }
  }

  float h[CPT][V];
#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    const float dx = dtv * xv[j];
    float ys = 0.0f;
#pragma unroll
    for (int k = 0; k < V; ++k) {
      const float hp = decode_code<F>(chunk_code<F>(raw[j], k), s256[j]);
      const float w = dx * Bv[k];
      h[j][k] = fmaf(dA, hp, w);
      ys = fmaf(Cv[k], h[j][k], ys);
    }
    ys = lane_sum(ys, a.lanes_per_row);
    if (cc == 0) {
      const int p = j * rows_per_pass + r0;
      a.y[tile * a.headdim + p] = ys + Dv * xv[j];
    }
  }

  // E4M3 scales: per group of a.group entries (lanes_per_group lanes of one
  // pass), or one per tile (lanes_per_group == 0).
  float rr[CPT];
#pragma unroll
  for (int j = 0; j < CPT; ++j) rr[j] = 1.0f;
  if constexpr (F == kE4M3) {
    float m[CPT];
#pragma unroll
    for (int j = 0; j < CPT; ++j) {
      m[j] = 0.0f;
#pragma unroll
      for (int k = 0; k < V; ++k) m[j] = fmaxf(m[j], fabsf(h[j][k]));
    }
    if (a.lanes_per_group == 0) {
      __shared__ float red[4];
      float mm = m[0];
#pragma unroll
      for (int j = 1; j < CPT; ++j) mm = fmaxf(mm, m[j]);
      mm = lane_max(mm, 64);
      if ((t & 63) == 0) red[t >> 6] = mm;
      __syncthreads();
      mm = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
      const float s = e4m3_scale(mm);
      const float r = (s == 0.0f) ? 0.0f : 1.0f / s;
#pragma unroll
      for (int j = 0; j < CPT; ++j) rr[j] = r;
      if (t == 0) a.scale[tile] = s;
    } else {
#pragma unroll
      for (int j = 0; j < CPT; ++j) {
        const float mm = lane_max(m[j], a.lanes_per_group);
        const float s = e4m3_scale(mm);
        rr[j] = (s == 0.0f) ? 0.0f : 1.0f / s;
        const int p = j * rows_per_pass + r0;
        const int64_t e = tile_base + static_cast<int64_t>(p) * a.dstate + n0;
        if ((t & (a.lanes_per_group - 1)) == 0) a.scale[e / a.group] = s;
      }
    }
  }

#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    const int p = j * rows_per_pass + r0;
    const int64_t e = tile_base + static_cast<int64_t>(p) * a.dstate + n0;
    const uint4 out = quantize_chunk<F, R>(h[j], rr[j], a.entry_base + static_cast<uint64_t>(e),
                                           a.thr);
    store_chunk<F>(a.state, e, out);
  }
}

// ---------------------------------------------------------------------------
// Row kernel: any layout whose rows are LR = dstate / V chunks. Each thread
// handles CPT_ROWS chunks, q = (blockIdx * CPT_ROWS + j) * 256 + t.
// ---------------------------------------------------------------------------
constexpr int CPT_ROWS = 2;

template <int F, int R, bool A_PER_STATE>
__global__ __launch_bounds__(256) void k_update_rows(UpdateArgs a) {
  constexpr int V = Traits<F>::V;
  const int t = threadIdx.x;
  const int cc = t & (a.lanes_per_row - 1);
  const int n0 = cc * V;
#pragma unroll
  for (int j = 0; j < CPT_ROWS; ++j) {
    const int64_t q = (static_cast<int64_t>(blockIdx.x) * CPT_ROWS + j) * 256 + t;
    const bool live = q < a.n_chunks;  // whole rows are live or dead together
    const int64_t qq = live ? q : 0;
    const int64_t e = qq * V;
    const int64_t row = e / a.dstate;
    const int64_t bh = row / a.headdim;  // b * nheads + h
    const int hh = static_cast<int>(bh % a.nheads);
    const int64_t b = bh / a.nheads;
    const int g = hh / a.heads_per_group;
    const uint4 raw = load_chunk<F>(a.state, e);
    const float xv = a.x[row];
    const float dtv = a.dt[bh];
    const float Dv = a.D ? a.D[hh] : 0.0f;
    float Bv[V], Cv[V];
    load_floats<V>(a.B + (b * a.ngroups + g) * a.dstate + n0, Bv);
    load_floats<V>(a.C + (b * a.ngroups + g) * a.dstate + n0, Cv);
    float dA[V];
    if constexpr (A_PER_STATE) {
      float Av[V];
      load_floats<V>(a.A + static_cast<int64_t>(hh) * a.dstate + n0, Av);
#pragma unroll
      for (int k = 0; k < V; ++k) dA[k] = static_cast<float>(exp(static_cast<double>(dtv * Av[k])));
    } else {
      const float d = static_cast<float>(exp(static_cast<double>(dtv * a.A[hh])));
#pragma unroll
      for (int k = 0; k < V; ++k) dA[k] = d;
    }
    float s256 = 0.0f;
    if constexpr (F == kE4M3) s256 = a.scale[e / a.group] * 256.0f;
    const float dx = dtv * xv;
    float h[V];
    float ys = 0.0f;
#pragma unroll
    for (int k = 0; k < V; ++k) {
      const float hp = decode_code<F>(chunk_code<F>(raw, k), s256);
      const float w = dx * Bv[k];
      h[k] = fmaf(dA[k], hp, w);
      ys = fmaf(Cv[k], h[k], ys);
    }
    ys = lane_sum(ys, a.lanes_per_row);
    if (live && cc == 0) a.y[row] = ys + Dv * xv;
    float r = 1.0f;
    if constexpr (F == kE4M3) {
      float m = 0.0f;
#pragma unroll
      for (int k = 0; k < V; ++k) m = fmaxf(m, fabsf(h[k]));
      m = lane_max(m, a.lanes_per_group);
      const float s = e4m3_scale(m);
      r = (s == 0.0f) ? 0.0f : 1.0f / s;
      if (live && (t & (a.lanes_per_group - 1)) == 0) a.scale[e / a.group] = s;
    }
    if (live) {
      const uint4 out = quantize_chunk<F, R>(h, r, a.entry_base + static_cast<uint64_t>(e), a.thr);
      store_chunk<F>(a.state, e, out);
    }
  }
}

// ---------------------------------------------------------------------------
// Requantize (no scale): 16 entries per thread; the last partial chunk entry by entry.
// ---------------------------------------------------------------------------
template <int F, int R>
__global__ __launch_bounds__(256) void k_requant(RequantArgs a) {
  const int64_t q = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t e = q * 16;
  if (e >= a.n) return;
  const uint64_t ge = a.entry_base + static_cast<uint64_t>(e);
  if (e + 16 <= a.n) {
    float h[16];
    load_floats<16>(a.h + e, h);
    constexpr int V = Traits<F>::V;
#pragma unroll
    for (int part = 0; part < 16 / V; ++part) {
      float hv[V];
#pragma unroll
      for (int k = 0; k < V; ++k) hv[k] = h[part * V + k];
      const uint4 out = quantize_chunk<F, R>(hv, 1.0f, ge + part * V, a.thr);
      store_chunk<F>(a.codes, e + part * V, out);
    }
  } else {
    for (int64_t k = e; k < a.n; ++k) {
      const uint64_t gk = a.entry_base + static_cast<uint64_t>(k);
      const uint32_t c = round_code<F, R>(a.h[k], thr_word<R>(thr_base<R>(gk, a.thr), 0u, a.thr));
      if constexpr (Traits<F>::bytes == 2) static_cast<uint16_t*>(a.codes)[k] = static_cast<uint16_t>(c);
      else if constexpr (Traits<F>::bytes == 4) static_cast<uint32_t*>(a.codes)[k] = c;
      else static_cast<uint8_t*>(a.codes)[k] = static_cast<uint8_t>(c);
    }
  }
}

// ---------------------------------------------------------------------------
// Requantize to E4M3 with group scales. lanes_per_group lanes (a power of two
// <= 64) work on one group; a wave covers 64 / lanes_per_group groups per
// iteration and loops over the group's 16-entry chunks.
// ---------------------------------------------------------------------------
template <int R>
__global__ __launch_bounds__(256) void k_requant_e4m3(RequantArgs a) {
  const int lane = threadIdx.x & 63;
  const int LG = a.lanes_per_group;
  const int gpw = 64 / LG;
  const int sub = lane / LG;
  const int li = lane & (LG - 1);
  const int64_t chunks_per_group = a.group / 16;
  const int64_t n_groups = a.n / a.group;
  const int64_t wave = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  const int64_t nwaves = static_cast<int64_t>(gridDim.x) * 4;
  for (int64_t g0 = wave * gpw; g0 < n_groups; g0 += nwaves * gpw) {
    const int64_t grp = g0 + sub;
    const bool live = grp < n_groups;
    float m = 0.0f;
    if (live) {
      for (int64_t c = li; c < chunks_per_group; c += LG) {
        float h[16];
        load_floats<16>(a.h + grp * a.group + c * 16, h);
#pragma unroll
        for (int k = 0; k < 16; ++k) m = fmaxf(m, fabsf(h[k]));
      }
    }
    m = lane_max(m, LG);
    const float s = e4m3_scale(m);
    const float r = (s == 0.0f) ? 0.0f : 1.0f / s;
    if (live && li == 0) a.scale[grp] = s;
    if (live) {
      for (int64_t c = li; c < chunks_per_group; c += LG) {
        const int64_t e = grp * a.group + c * 16;
        float h[16];
        load_floats<16>(a.h + e, h);
        const uint4 out = quantize_chunk<kE4M3, R>(h, r, a.entry_base + static_cast<uint64_t>(e), a.thr);
        store_chunk<kE4M3>(a.codes, e, out);
      }
    }
  }
}

template <int R>
__global__ __launch_bounds__(256) void k_dither_fill(DitherArgs a) {
  const int64_t q = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t e = q * 4;
  if (e >= a.n) return;
  const int64_t lim = (a.n - e < 4) ? (a.n - e) : 4;
  for (int64_t k = 0; k < lim; ++k) {
    const uint64_t ge = a.entry_base + static_cast<uint64_t>(e + k);
    a.out[e + k] = (R == kRTN) ? (1u << 23) : (thr_word<R>(thr_base<R>(ge, a.thr), 0u, a.thr) >> 8);
  }
}

// ---------------------------------------------------------------------------
// Launchers.
// ---------------------------------------------------------------------------
template <int F, int R, int CPT>
static hipError_t launch_head_cpt(const UpdateArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((k_update_head<F, R, CPT>), dim3(static_cast<unsigned>(a.batch * a.nheads)),
                     dim3(256), 0, s, a);
  return hipGetLastError();
}

template <int F, int R>
static hipError_t launch_head_fr(const UpdateArgs& a, int cpt, hipStream_t s) {
  switch (cpt) {
    case 1: return launch_head_cpt<F, R, 1>(a, s);
    case 2: return launch_head_cpt<F, R, 2>(a, s);
    case 4: return launch_head_cpt<F, R, 4>(a, s);
    case 8: return launch_head_cpt<F, R, 8>(a, s);
    default: return hipErrorInvalidValue;
  }
}

template <int F, int R>
static hipError_t launch_rows_fr(const UpdateArgs& a, bool a_per_state, hipStream_t s) {
  const int64_t per_block = 256LL * CPT_ROWS;
  const unsigned grid = static_cast<unsigned>((a.n_chunks + per_block - 1) / per_block);
  if (a_per_state)
    hipLaunchKernelGGL((k_update_rows<F, R, true>), dim3(grid), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((k_update_rows<F, R, false>), dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <int F>
static hipError_t dispatch_update_f(const UpdateArgs& a, int rule, int kind, int cpt, bool aps,
                                    hipStream_t s) {
  switch (rule) {
    case kRTN: return kind == 0 ? launch_head_fr<F, kRTN>(a, cpt, s) : launch_rows_fr<F, kRTN>(a, aps, s);
    case kSR: return kind == 0 ? launch_head_fr<F, kSR>(a, cpt, s) : launch_rows_fr<F, kSR>(a, aps, s);
    default: return kind == 0 ? launch_head_fr<F, kWEYL>(a, cpt, s) : launch_rows_fr<F, kWEYL>(a, aps, s);
  }
}

hipError_t launch_update(const UpdateArgs& a, int format, int rule, int kind, int cpt,
                         bool a_per_state, hipStream_t s) {
  switch (format) {
    case kFP16: return dispatch_update_f<kFP16>(a, rule, kind, cpt, a_per_state, s);
    case kBF16: return dispatch_update_f<kBF16>(a, rule, kind, cpt, a_per_state, s);
    case kE4M3: return dispatch_update_f<kE4M3>(a, rule, kind, cpt, a_per_state, s);
    default: return dispatch_update_f<kFP32>(a, rule, kind, cpt, a_per_state, s);
  }
}

template <int F>
static hipError_t launch_requant_f(const RequantArgs& a, int rule, hipStream_t s) {
  const int64_t chunks = (a.n + 15) / 16;
  const unsigned grid = static_cast<unsigned>((chunks + 255) / 256);
  switch (rule) {
    case kRTN: hipLaunchKernelGGL((k_requant<F, kRTN>), dim3(grid), dim3(256), 0, s, a); break;
    case kSR: hipLaunchKernelGGL((k_requant<F, kSR>), dim3(grid), dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((k_requant<F, kWEYL>), dim3(grid), dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_requant(const RequantArgs& a, int format, int rule, hipStream_t s) {
  if (format == kE4M3) {
    const int64_t n_groups = a.n / a.group;
    const int64_t gpw = 64 / a.lanes_per_group;
    int64_t blocks = (n_groups + 4 * gpw - 1) / (4 * gpw);
    if (blocks > 65536) blocks = 65536;
    const unsigned grid = static_cast<unsigned>(blocks);
    switch (rule) {
      case kRTN: hipLaunchKernelGGL((k_requant_e4m3<kRTN>), dim3(grid), dim3(256), 0, s, a); break;
      case kSR: hipLaunchKernelGGL((k_requant_e4m3<kSR>), dim3(grid), dim3(256), 0, s, a); break;
      default: hipLaunchKernelGGL((k_requant_e4m3<kWEYL>), dim3(grid), dim3(256), 0, s, a); break;
    }
    return hipGetLastError();
  }
  switch (format) {
    case kFP16: return launch_requant_f<kFP16>(a, rule, s);
    case kBF16: return launch_requant_f<kBF16>(a, rule, s);
    default: return launch_requant_f<kFP32>(a, rule, s);
  }
}

hipError_t launch_dither(const DitherArgs& a, int rule, hipStream_t s) {
  const int64_t chunks = (a.n + 3) / 4;
  const unsigned grid = static_cast<unsigned>((chunks + 255) / 256);
  switch (rule) {
    case kRTN: hipLaunchKernelGGL((k_dither_fill<kRTN>), dim3(grid), dim3(256), 0, s, a); break;
    case kSR: hipLaunchKernelGGL((k_dither_fill<kSR>), dim3(grid), dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((k_dither_fill<kWEYL>), dim3(grid), dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

}  // namespace ssmq
