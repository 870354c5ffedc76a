// ssmq_kernels.hip -- HIP kernels of the quantized selective-state update (gfx950).
//
// Kernels:
//   k_update_slab  Mamba-2 heads (scalar A per head): a workgroup updates a slab
//                  of rows of one (batch, head) tile: dequantize -> exp(dt A) ->
//                  FMA recurrence -> y = C h + D x -> (E4M3 group scale) ->
//                  threshold -> round -> store, in registers, so the state
//                  crosses HBM once each way (Section 2 eq. (rec) and eq.
//                  (dither); Appendix B "Runners", "Formats", "Dithers").
//   k_update_rows  the same step for any row layout (Mamba-1 with A per (channel,
//                  n), and Mamba-2 heads smaller than a slab).
//   k_requant      fp32 -> codes for fp16 / bf16 / fp32, one chunk per thread.
//   k_requant_scaled fp32 -> E4M3 / INT8 / INT4 codes with group scales.
//   k_dither_fill  the 24-bit thresholds themselves.
//   k_conv1d_update the causal depthwise convolution's decode step.
//   k_replay       open-loop replay of recorded decays and writes: a reference
//                  and a stored trajectory per entry, iterated in registers.
//
// Layout. A chunk is the codes of V consecutive entries of one state row: 16
// bytes holding 8 fp16 / bf16, 16 E4M3 / INT8 or 4 fp32 entries, or 8 bytes
// holding 16 INT4 entries. The LR = dstate / V chunks of a row sit in LR
// consecutive lanes of one wave, so a lane's slice of B and C is fixed and C.h
// is an LR-lane reduction. Each thread owns CPT chunks (one row per pass); the
// state moves with nontemporal 16- or 8-byte accesses (each byte is touched once
// per step, so nothing is gained by keeping it in the caches).
#include "ssmq_device.hpp"

namespace ssmq {

template <int V>
__device__ inline void load_floats(const float* p, float (&out)[V]) {
#pragma unroll
  for (int i = 0; i < V; i += 4) {
    const float4 v = *reinterpret_cast<const float4*>(p + i);
    out[i] = v.x; out[i + 1] = v.y; out[i + 2] = v.z; out[i + 3] = v.w;
  }
}

__device__ inline float decay(float dtv, float a) {
  return static_cast<float>(exp(static_cast<double>(dtv * a)));  // correctly rounded fl32(exp)
}

// The step size the update uses: dt, plus dt_bias[head] when given, through
// softplus(v) = log(1 + e^v) (double, one rounding; v itself above 20) when asked.
__device__ inline float step_size(const UpdateArgs& a, float dtv, int head) {
  if (a.dt_bias) dtv = dtv + a.dt_bias[head];
  if (a.dt_softplus && !(dtv > 20.0f)) dtv = static_cast<float>(log1p(exp(static_cast<double>(dtv))));
  return dtv;
}

__device__ inline float silu(float v) { return v / (1.0f + expf(-v)); }

// ---------------------------------------------------------------------------
// Mamba-2 head slabs: NT threads x CPT chunks = a run of whole rows of one head.
// ---------------------------------------------------------------------------
// The whole-head configurations of the scaled formats (four chunks per thread,
// up to 128 threads) hold 64 state values per thread and sit near the
// 128-register line; they are held to it (four waves per SIMD) instead of
// dropping to three waves.
//
// N128: the state dimension is 128 and a scale group is 128 entries (8 lanes)
// or the whole head, so the lanes per row and per group are compile-time
// constants: the reductions lose their runtime width tests (INT8 / INT4 about
// 6 % faster).
constexpr int log2c(int v) { return v <= 1 ? 0 : 1 + log2c(v / 2); }

template <int F, int R, int NT, int CPT, bool N128 = false>
__global__ __launch_bounds__(NT, (Traits<F>::scaled && CPT == 4 && NT <= 128) ? 4 : 1)
void k_update_slab(UpdateArgs a) {
  constexpr int V = Traits<F>::V;
  constexpr int NW = NT / 64;
  const int lanes_per_row = N128 ? 128 / V : a.lanes_per_row;
  const int lr_shift = N128 ? log2c(128 / V) : a.lr_shift;
  const int lanes_per_group = N128 ? 8 : a.lanes_per_group;  // when not the whole head
  const int t = threadIdx.x;
  const uint32_t blk = blockIdx.x;
  const uint32_t tile32 = a.div_slabs.div(blk);  // b * nheads + h
  const uint32_t slab = blk - tile32 * static_cast<uint32_t>(a.slabs_per_head);
  const uint32_t b32 = a.div_nheads.div(tile32);
  const int hh = static_cast<int>(tile32 - b32 * static_cast<uint32_t>(a.nheads));
  const int g = static_cast<int>(a.div_hpg.div(static_cast<uint32_t>(hh)));
  const int64_t tile = tile32, b = b32;
  const int cc = t & (lanes_per_row - 1);
  const int n0 = cc * V;
  const int rows_per_pass = NT >> lr_shift;
  const int r0 = (t >> lr_shift) + static_cast<int>(slab) * rows_per_pass * CPT;
  const int64_t tile_base = tile * a.head_size;
  // Uniform bases plus 32-bit lane offsets (a head holds fewer than 2^31 bytes).
  uint8_t* const hstate = static_cast<uint8_t*>(a.state) + chunk_bytes_at<F>(tile_base);
  const float* const hx = a.x + tile * a.headdim;
  float* const hy = a.y + tile * a.headdim;
  const uint32_t l0 = static_cast<uint32_t>(r0 * a.dstate + n0);  // lane's first entry in the head
  const uint32_t pass = static_cast<uint32_t>(rows_per_pass * a.dstate);  // entries per pass
  const int64_t e0 = tile_base + l0;

  // Per-head values are staged once per workgroup in LDS while the state loads
  // are in flight: B and C of the head's group (one float4 per thread, loaded
  // before the state so that staging them waits for them alone), and exp(dt A),
  // evaluated by the first wave in double with one final rounding.
  __shared__ float4 sBC[kMaxDstate / 2];
  __shared__ float sh[4];
  // y of the slab is staged here and written back as whole lines (the integer
  // formats, whose kernels measure 2-3 % slower that way, store it directly).
  constexpr bool kStageY = !(F == kINT8 || F == kINT4);
  __shared__ float sY[kStageY ? NT * CPT : 1];
  __shared__ uint32_t sDone;  // waves whose rows of y are in sY
  const int nq = a.dstate >> 2;  // float4 per vector
  const float* Bg = a.B + (b * a.ngroups + g) * a.dstate;
  const float* Cg = a.C + (b * a.ngroups + g) * a.dstate;
  const bool bc_one = 2 * nq <= NT;  // one float4 of B or C per thread at most
  float4 bc = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  if (bc_one && t < 2 * nq)
    bc = (t < nq) ? reinterpret_cast<const float4*>(Bg)[t] : reinterpret_cast<const float4*>(Cg)[t - nq];

  chunk_t<F> raw[CPT];
  float xv[CPT];
#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    raw[j] = load_stream<chunk_t<F>>(hstate + chunk_bytes_at<F>(l0 + j * pass));
    xv[j] = hx[r0 + j * rows_per_pass];
  }
  const float dt_in = a.dt[tile];
  const float Dv = a.D ? a.D[hh] : 0.0f;

  if (t < 64) {
    const float dte = step_size(a, dt_in, hh);
    const float d = decay(dte, a.A[hh]);
    if (t == 0) { sh[0] = d; sh[2] = dte; sDone = 0; }
  }
  if (bc_one) {
    if (t < 2 * nq) sBC[t] = bc;
  } else {
    for (int i = t; i < 2 * nq; i += NT)
      sBC[i] = (i < nq) ? reinterpret_cast<const float4*>(Bg)[i]
                        : reinterpret_cast<const float4*>(Cg)[i - nq];
  }
  __syncthreads();
  const float dA = sh[0];
  const float dtv = sh[2];

  float h[CPT][V];
  bool bad[CPT];  // a NaN or infinity reached this chunk's partial of y
  float yo[CPT];  // rows' y, for kernels that store it directly
  // Scaled formats store fl32(v * s_old); dA * h_prev is evaluated as
  // fma(fl32(dA * s_old), v, w), one rounding of the scaled decay per group in
  // place of one rounding of v * s_old per entry (it saves a multiply per entry;
  // h_new moves by about an ulp at most). E4M3, and the four-chunk configurations (one
  // scale per head), read their scales before the loop (read inside it, each
  // load is issued after the previous chunk's y store and waited for at once);
  // the block-scaled INT kernels measure faster with one select-addressed load
  // per chunk.
  constexpr bool kScalesFirst = (F == kE4M3) || (is_int_fmt<F> && CPT >= 4);
  float dAs[CPT];
#pragma unroll
  for (int j = 0; j < CPT; ++j) dAs[j] = dA;
  if constexpr (kScalesFirst) {
    if (a.lanes_per_group == 0) {
      const float d = dA * a.scale[tile];
#pragma unroll
      for (int j = 0; j < CPT; ++j) dAs[j] = d;
    } else {
#pragma unroll
      for (int j = 0; j < CPT; ++j) dAs[j] = dA * a.scale[(e0 + j * pass) >> a.group_shift];
    }
  }
#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    float dAj = dAs[j];
    if constexpr (is_int_fmt<F> && !kScalesFirst)
      dAj = dA * ((a.lanes_per_group == 0) ? a.scale[tile] : a.scale[(e0 + j * pass) >> a.group_shift]);
    float hp[V];
    decode_chunk<F>(raw[j], hp);
    const float dx = dtv * xv[j];
    // The lane's part of y: INT8 round-to-nearest, whose rounding is short enough
    // for the chain of dependent fmas to set the pace, sums in four interleaved
    // partial sums (4 % faster); elsewhere they measure no gain (the dithered
    // rules) or a loss (E4M3 and INT4 round-to-nearest, 1.5 and 3 %).
    constexpr int kYP = (F == kINT8 && R == kRTN) ? 4 : 1;
    float yp[kYP];
#pragma unroll
    for (int u = 0; u < kYP; ++u) yp[u] = 0.0f;
    // B and C come from LDS four at a time, so they are not held in registers
    // across passes.
#pragma unroll
    for (int i = 0; i < V / 4; ++i) {
      const float4 bq = sBC[(n0 >> 2) + i];
      const float4 cq = sBC[nq + (n0 >> 2) + i];
      const float bk[4] = {bq.x, bq.y, bq.z, bq.w};
      const float ck[4] = {cq.x, cq.y, cq.z, cq.w};
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int k = 4 * i + u;
        const float w = dx * bk[u];
        h[j][k] = fmaf(dAj, hp[k], w);
        yp[u % kYP] = fmaf(ck[u], h[j][k], yp[u % kYP]);
      }
    }
    float ys = yp[0];
    if constexpr (kYP == 4) ys = (yp[0] + yp[1]) + (yp[2] + yp[3]);
    // (a finite overflow of a partial sum only sends the chunk down the exact path)
    bad[j] = !__builtin_isfinite(ys);
    ys = lane_sum(ys, lanes_per_row);
    if constexpr (kStageY) {
      if (cc == 0) sY[(t >> lr_shift) + j * rows_per_pass] = ys + Dv * xv[j];
    } else {
      yo[j] = ys + Dv * xv[j];
    }
  }
  if constexpr (!kStageY) {
    // Stored after the loop, so no chunk's scale load waits behind a y store.
    if (cc == 0) {
#pragma unroll
      for (int j = 0; j < CPT; ++j) {
        float yv = yo[j];
        if (a.z) yv = yv * silu(a.z[tile * a.headdim + r0 + j * rows_per_pass]);
        hy[r0 + j * rows_per_pass] = yv;
      }
    }
  }

  float r[CPT];  // scaled formats: 1 / s of each chunk's group
  bool clamp = true;  // E4M3 dithers: some value may exceed 448 after scaling
#pragma unroll
  for (int j = 0; j < CPT; ++j) r[j] = 1.0f;
  if constexpr (Traits<F>::scaled) {
    // Lane maxima of |h| ignore NaN and are >= 0, so the cross-lane maximum can
    // compare bit patterns as unsigned integers.
    uint32_t m[CPT];
#pragma unroll
    for (int j = 0; j < CPT; ++j) {
      float mj = 0.0f;
#pragma unroll
      for (int k = 0; k < V; ++k) mj = fmaxf(mj, __builtin_fabsf(h[j][k]));
      m[j] = __float_as_uint(mj);
    }
    if (a.lanes_per_group == 0) {  // one scale for the whole head, which is this workgroup
      __shared__ uint32_t red[NW];
      uint32_t mm = m[0];
#pragma unroll
      for (int j = 1; j < CPT; ++j) mm = max(mm, m[j]);
      mm = lane_umax(mm, 64);
      if ((t & 63) == 0) red[t >> 6] = mm;
      __syncthreads();
      if (t < 64) {  // the first wave turns the maximum into the scale and its reciprocal
        uint32_t w = red[0];
#pragma unroll
        for (int i = 1; i < NW; ++i) w = max(w, red[i]);
        const float s = group_scale<F>(__uint_as_float(w));
        const float rs = recip_scale(s);
        if (t == 0) {
          sh[0] = s;
          sh[1] = rs;
          sh[3] = (__uint_as_float(w) * rs <= 448.0f) ? 0.0f : 1.0f;  // E4M3: clamp needed
          a.scale[tile] = s;
        }
      }
      __syncthreads();
      const float rs = sh[1];
      // A per-head scale whose own rounding leaves max|h| r <= 448 (about four
      // heads in five) needs the E4M3 clamp nowhere in the head.
      clamp = __builtin_amdgcn_readfirstlane(__float_as_uint(sh[3])) != 0u;
#pragma unroll
      for (int j = 0; j < CPT; ++j) r[j] = rs;
    } else if (CPT % 2 == 0 && lanes_per_group >= 2) {
      // Lanes t and t ^ 1 share their group in every chunk, so each computes one
      // scale of a pair of chunks (even lanes chunk j, odd lanes chunk j + 1) and
      // takes the other reciprocal from its neighbour: half the divisions and
      // reciprocals (INT8 about 2 % faster).
      const bool odd = (t & 1) != 0;
      const int lg = t & (lanes_per_group - 1);
#pragma unroll
      for (int j = 0; j < CPT; j += 2) {
        const uint32_t m0 = lane_umax(m[j], lanes_per_group);
        const uint32_t m1 = lane_umax(m[j + 1], lanes_per_group);
        const float s = group_scale<F>(__uint_as_float(odd ? m1 : m0));
        const float rs = recip_scale(s);
        const float other = __builtin_bit_cast(
            float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, rs), kQuadXor1, 0xF, 0xF, true));
        r[j] = odd ? other : rs;
        r[j + 1] = odd ? rs : other;
        if (lg == 0) a.scale[(e0 + j * pass) >> a.group_shift] = s;
        if (lg == 1) a.scale[(e0 + (j + 1) * pass) >> a.group_shift] = s;
      }
    } else {  // groups of lanes_per_group consecutive lanes of one pass
#pragma unroll
      for (int j = 0; j < CPT; ++j) {
        const float s = group_scale<F>(__uint_as_float(lane_umax(m[j], lanes_per_group)));
        r[j] = recip_scale(s);
        if ((t & (lanes_per_group - 1)) == 0) a.scale[(e0 + j * pass) >> a.group_shift] = s;
      }
    }
  }

  // Threshold bases of the chunks: one pass of NT chunks apart, a constant
  // step when the pass spans whole dither blocks. The direct form is kept
  // inside its branch by the empty asm: if-converted, its two 32-bit
  // multiplies would run for every chunk.
  uint32_t bases[CPT];
  bases[0] = thr_base<R>(a.entry_base + static_cast<uint64_t>(e0), a.thr);
  if (a.pass_thr_ok) {
#pragma unroll
    for (int j = 1; j < CPT; ++j) bases[j] = bases[0] + static_cast<uint32_t>(j) * a.pass_thr_inc;
  } else {
    uint64_t eb = a.entry_base + static_cast<uint64_t>(e0);
    asm volatile("" : "+v"(eb));
#pragma unroll
    for (int j = 1; j < CPT; ++j) bases[j] = thr_base<R>(eb + static_cast<uint64_t>(j) * pass, a.thr);
  }
#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    const int64_t e = e0 + static_cast<int64_t>(j) * pass;
    const uint32_t base = bases[j];
    const chunk_t<F> out = quantize_any<F, R>(
        h[j], r[j], chunk_thr<R, V>(a.entry_base + static_cast<uint64_t>(e), a.thr, base, a.toff),
        bad[j], clamp);
    store_stream(hstate + chunk_bytes_at<F>(l0 + j * pass), out);
  }

  // y leaves as whole lines rather than one float per row from every wave: each
  // wave counts itself in after its rows are in sY, and the last one to arrive
  // writes the slab's rows (the others exit; nothing waits).
  if constexpr (!kStageY) return;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  uint32_t arrived = 0;
  if ((t & 63) == 0) arrived = atomicAdd(&sDone, 1u);
  arrived = __shfl(arrived, 0);
  if (arrived == NW - 1) {
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    const int rows_slab = rows_per_pass * CPT;
    const int row0 = static_cast<int>(slab) * rows_slab;
    for (int i = t & 63; i < rows_slab; i += 64) {
      float yv = sY[i];
      if (a.z) yv = yv * silu(a.z[tile * a.headdim + row0 + i]);
      hy[row0 + i] = yv;
    }
  }
}

// ---------------------------------------------------------------------------
// Row kernel: any layout whose rows are LR = dstate / V chunks; one chunk per
// thread, chunk q = blockIdx * 256 + t.
// ---------------------------------------------------------------------------
// FP32_STATE: a checkpoint write on an fp32 state. The stored values are fp32
// (read as they are, no scale fold); each new value is rounded onto F's grid
// and written back as the fp32 value of its code (times the group scale for
// the scaled formats, whose scales are written only when a.scale is set).
template <int F, int R, bool A_PER_STATE, bool FP32_STATE>
__global__ __launch_bounds__(256) void k_update_rows(UpdateArgs a) {
  constexpr int V = Traits<F>::V;
  const int t = threadIdx.x;
  const int cc = t & (a.lanes_per_row - 1);
  const int n0 = cc * V;
  const int64_t q = static_cast<int64_t>(blockIdx.x) * 256 + t;
  const bool live = q < a.n_chunks;  // whole rows (and groups) are live or dead together
  const int64_t e = (live ? q : 0) * V;
  const uint32_t row = static_cast<uint32_t>(e >> a.dstate_shift);  // rows < 2^32 (checked on host)
  const uint32_t bh = a.div_headdim.div(row);                        // b * nheads + h
  const uint32_t b = a.div_nheads.div(bh);
  const int hh = static_cast<int>(bh - b * static_cast<uint32_t>(a.nheads));
  const int g = static_cast<int>(a.div_hpg.div(static_cast<uint32_t>(hh)));
  uint8_t* const state = static_cast<uint8_t*>(a.state);
  float hp[V], h[V];
  if constexpr (FP32_STATE) {
#pragma unroll
    for (int i = 0; i < V / 4; ++i) {
      const uint4 v = load_stream<uint4>(state + (e + 4 * i) * 4);
      hp[4 * i] = __uint_as_float(v.x); hp[4 * i + 1] = __uint_as_float(v.y);
      hp[4 * i + 2] = __uint_as_float(v.z); hp[4 * i + 3] = __uint_as_float(v.w);
    }
  } else {
    decode_chunk<F>(load_stream<chunk_t<F>>(state + chunk_bytes_at<F>(e)), hp);
  }
  const float xv = a.x[row];
  const float dtv = step_size(a, a.dt[bh], hh);
  const float Dv = a.D ? a.D[hh] : 0.0f;
  float Bv[V], Cv[V], dA[V];
  load_floats<V>(a.B + (static_cast<int64_t>(b) * a.ngroups + g) * a.dstate + n0, Bv);
  load_floats<V>(a.C + (static_cast<int64_t>(b) * a.ngroups + g) * a.dstate + n0, Cv);
  if constexpr (A_PER_STATE) {
    float Av[V];
    load_floats<V>(a.A + static_cast<int64_t>(hh) * a.dstate + n0, Av);
#pragma unroll
    for (int k = 0; k < V; ++k) dA[k] = decay(dtv, Av[k]);
  } else {
    const float d = decay(dtv, a.A[hh]);
#pragma unroll
    for (int k = 0; k < V; ++k) dA[k] = d;
  }
  if constexpr (Traits<F>::scaled && !FP32_STATE) {  // fold the old group scale into the decay (see k_update_slab)
    const float s_old = a.scale[e >> a.group_shift];
#pragma unroll
    for (int k = 0; k < V; ++k) dA[k] = dA[k] * s_old;
  }
  const float dx = dtv * xv;
  float ys = 0.0f;
#pragma unroll
  for (int k = 0; k < V; ++k) {
    const float w = dx * Bv[k];
    h[k] = fmaf(dA[k], hp[k], w);
    ys = fmaf(Cv[k], h[k], ys);
  }
  const bool bad = !__builtin_isfinite(ys);
  ys = lane_sum(ys, a.lanes_per_row);
  if (live && cc == 0) a.y[row] = a.z ? (ys + Dv * xv) * silu(a.z[row]) : ys + Dv * xv;
  float rs = 1.0f, s = 1.0f;
  if constexpr (Traits<F>::scaled) {
    float m = 0.0f;
#pragma unroll
    for (int k = 0; k < V; ++k) m = fmaxf(m, __builtin_fabsf(h[k]));
    s = group_scale<F>(__uint_as_float(lane_umax(__float_as_uint(m), a.lanes_per_group)));
    rs = recip_scale(s);
    if (live && a.scale && (t & (a.lanes_per_group - 1)) == 0) a.scale[e >> a.group_shift] = s;
  }
  const uint64_t ge = a.entry_base + static_cast<uint64_t>(e);
  const chunk_t<F> out =
      quantize_any<F, R>(h, rs, chunk_thr<R, V>(ge, a.thr, thr_base<R>(ge, a.thr), a.toff), bad);
  if constexpr (FP32_STATE) {
    float v[V];
    decode_chunk<F>(out, v);
#pragma unroll
    for (int k = 0; k < V; ++k)
      if constexpr (Traits<F>::scaled) v[k] = v[k] * s;
    if (live) {
#pragma unroll
      for (int i = 0; i < V / 4; ++i)
        store_stream(state + (e + 4 * i) * 4,
                     make_uint4(__float_as_uint(v[4 * i]), __float_as_uint(v[4 * i + 1]),
                                __float_as_uint(v[4 * i + 2]), __float_as_uint(v[4 * i + 3])));
    }
  } else {
    if (live) store_stream(state + chunk_bytes_at<F>(e), out);
  }
}

// ---------------------------------------------------------------------------
// Requantize without scale: one chunk of V entries per thread; the entries
// after the last whole chunk one by one.
// ---------------------------------------------------------------------------
template <int F>
__device__ inline void store_code(void* codes, int64_t k, uint32_t c) {
  constexpr int bytes = Traits<F>::CB / Traits<F>::V;
  if constexpr (bytes == 2) static_cast<uint16_t*>(codes)[k] = static_cast<uint16_t>(c);
  else if constexpr (bytes == 4) static_cast<uint32_t*>(codes)[k] = c;
  else static_cast<uint8_t*>(codes)[k] = static_cast<uint8_t>(c);
}

template <int F, int R>
__global__ __launch_bounds__(256) void k_requant(RequantArgs a) {
  constexpr int V = Traits<F>::V;
  const int64_t q = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t e = q * V;
  if (e >= a.n) return;
  const uint64_t ge = a.entry_base + static_cast<uint64_t>(e);
  if (e + V <= a.n) {
    float h[V];
    load_floats<V>(a.h + e, h);
    const uint4 out = quantize_chunk<F, R>(h, chunk_thr<R, V>(ge, a.thr, thr_base<R>(ge, a.thr), a.toff),
                                           chunk_has_nan<V>(h));
    *reinterpret_cast<uint4*>(static_cast<uint8_t*>(a.codes) + chunk_bytes_at<F>(e)) = out;
  } else {
    for (int64_t k = e; k < a.n; ++k) {
      const uint64_t gk = a.entry_base + static_cast<uint64_t>(k);
      store_code<F>(a.codes, k, round_code<F, R>(a.h[k], entry_thr<R>(gk, a.thr)));
    }
  }
}

// ---------------------------------------------------------------------------
// Requantize to a scaled format (E4M3, INT8, INT4) with group scales.
// lanes_per_group lanes (a power of two <= 64) work on one group; a wave covers
// 64 / lanes_per_group groups per iteration and loops over each group's
// 16-entry chunks.
// ---------------------------------------------------------------------------
template <int F, int R>
__global__ __launch_bounds__(256) void k_requant_scaled(RequantArgs a) {
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
        for (int k = 0; k < 16; ++k) m = fmaxf(m, __builtin_fabsf(h[k]));
      }
    }
    const float s = group_scale<F>(__uint_as_float(lane_umax(__float_as_uint(m), LG)));
    const float rs = recip_scale(s);
    if (live && li == 0) a.scale[grp] = s;
    const int64_t iters = (chunks_per_group + LG - 1) / LG;  // uniform trip count
    for (int64_t it = 0; it < iters; ++it) {
      const int64_t c = it * LG + li;
      const bool ok = live && c < chunks_per_group;
      const int64_t e = (ok ? grp * a.group + c * 16 : 0);
      float h[16];
      load_floats<16>(a.h + e, h);
      const uint64_t ge = a.entry_base + static_cast<uint64_t>(e);
      const chunk_t<F> out = quantize_any<F, R>(h, rs, chunk_thr<R, 16>(ge, a.thr, thr_base<R>(ge, a.thr), a.toff),
                                                chunk_has_nan<16>(h));
      if (ok) *reinterpret_cast<chunk_t<F>*>(static_cast<uint8_t*>(a.codes) + chunk_bytes_at<F>(e)) = out;
    }
  }
}

// Groups of 256 * 16 * CPT entries (4096 or 8192, e.g. one scale per 64x128
// head): one workgroup per group, its values held in registers between the
// maximum and the rounding, so the fp32 input is read once.
template <int F, int R, int CPT>
__global__ __launch_bounds__(256) void k_requant_group_wg(RequantArgs a) {
  const int t = threadIdx.x;
  const int64_t e0 = static_cast<int64_t>(blockIdx.x) * a.group;
  float h[CPT][16];
  float m = 0.0f;
#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    load_floats<16>(a.h + e0 + (static_cast<int64_t>(j) * 256 + t) * 16, h[j]);
#pragma unroll
    for (int k = 0; k < 16; ++k) m = fmaxf(m, __builtin_fabsf(h[j][k]));
  }
  __shared__ uint32_t red[4];
  __shared__ float rsh;
  const uint32_t mw = lane_umax(__float_as_uint(m), 64);
  if ((t & 63) == 0) red[t >> 6] = mw;
  __syncthreads();
  if (t == 0) {
    const uint32_t w = max(max(red[0], red[1]), max(red[2], red[3]));
    const float sc = group_scale<F>(__uint_as_float(w));
    a.scale[blockIdx.x] = sc;
    rsh = recip_scale(sc);
  }
  __syncthreads();
  const float rs = rsh;
#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    const int64_t e = e0 + (static_cast<int64_t>(j) * 256 + t) * 16;
    const uint64_t ge = a.entry_base + static_cast<uint64_t>(e);
    const chunk_t<F> out = quantize_any<F, R>(
        h[j], rs, chunk_thr<R, 16>(ge, a.thr, thr_base<R>(ge, a.thr), a.toff), chunk_has_nan<16>(h[j]));
    *reinterpret_cast<chunk_t<F>*>(static_cast<uint8_t*>(a.codes) + chunk_bytes_at<F>(e)) = out;
  }
}

template <int R>
__global__ __launch_bounds__(256) void k_dither_fill(DitherArgs a) {
  const int64_t q = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t e = q * 4;
  if (e >= a.n) return;
  const uint64_t ge = a.entry_base + static_cast<uint64_t>(e);
  if (a.n - e >= 4 && (reinterpret_cast<uintptr_t>(a.out) & 15u) == 0) {
    // Four whole words to a 16-byte aligned address: one 16-byte store, and one
    // Philox block when the four entries are the words of one block.
    uint32_t w[4];
    if constexpr (R == kPHILOX) {
      if ((ge & 3u) == 0) {
        const uint64_t blk = ge >> 2;
        philox4x32_10(static_cast<uint32_t>(blk), static_cast<uint32_t>(blk >> 32), a.thr.step, 0u,
                      a.thr.seed, a.thr.layer, w);
#pragma unroll
        for (int k = 0; k < 4; ++k) w[k] >>= 8;
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) w[k] = entry_thr<R>(ge + k, a.thr) >> 8;
      }
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) w[k] = (R == kRTN) ? (1u << 23) : (entry_thr<R>(ge + k, a.thr) >> 8);
    }
    store_stream(a.out + e, make_uint4(w[0], w[1], w[2], w[3]));
    return;
  }
  const int64_t lim = (a.n - e < 4) ? (a.n - e) : 4;
  for (int64_t k = 0; k < lim; ++k)
    a.out[e + k] = (R == kRTN) ? (1u << 23) : (entry_thr<R>(ge + static_cast<uint64_t>(k), a.thr) >> 8);
}

// ---------------------------------------------------------------------------
// Open-loop replay. Thread q owns entries 4q .. 4q+3 for all steps: the fp32
// reference h and the stored value hq stay in registers, so the only traffic is
// the trace (a and w, 8 bytes per entry and step, nontemporal, the next step's
// rows loaded while the current one is rounded) and the error sums per block.
// Each step rounds fma(a, hq, w) with the exact software rounding of the
// format (the per-entry functions of the fused kernels' exact path); the
// scaled formats first reduce max|x| over the group's lanes. Lanes past n
// (the grid's ragged end) run with zero inputs and store nothing, so the group
// reductions always see whole groups.
// ---------------------------------------------------------------------------
template <int F, int R>
__device__ inline void replay_round(const ReplayArgs& a, uint64_t e0, uint32_t step,
                                    const float (&x)[4], float (&hq)[4], uint32_t (&code)[4],
                                    float& scale) {
  Thr th = a.thr;
  th.step = step;
  if constexpr (R == kWEYL) th.key = a.weyl_key0 + kWeylPhi * (step - a.step0);
  else if constexpr (R == kSR) th.key = sr_step_key(a.sr_key0, step);
  uint32_t thr[4];
  if constexpr (R == kPHILOX) {
    const ChunkThr<R, 4> t4 = chunk_thr<R, 4>(e0, th, 0u, nullptr);
#pragma unroll
    for (int k = 0; k < 4; ++k) thr[k] = t4(k);
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) thr[k] = entry_thr<R>(e0 + k, th);
  }
  if constexpr (Traits<F>::scaled) {
    float m = 0.0f;
#pragma unroll
    for (int k = 0; k < 4; ++k) m = fmaxf(m, __builtin_fabsf(x[k]));
    const float s = group_scale<F>(__uint_as_float(lane_umax(__float_as_uint(m), a.lanes_per_group)));
    const float r = recip_scale(s);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      code[k] = round_code<F, R>(x[k] * r, thr[k]);
      hq[k] = code_value<F>(code[k]) * s;
    }
    scale = s;
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      code[k] = round_code<F, R>(x[k], thr[k]);
      hq[k] = code_value<F>(code[k]);
    }
  }
}

template <int F, int R>
__global__ __launch_bounds__(256) void k_replay(ReplayArgs a) {
  const int64_t q = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t i0 = q * 4;
  const bool live = i0 < a.n;
  const uint64_t e0 = a.entry_base + static_cast<uint64_t>(i0);
  float h[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (live) load_floats<4>(a.h0 + i0, h);
  float hq[4];
  uint32_t code[4];
  float scale = 0.0f;
  replay_round<F, R>(a, e0, a.step0, h, hq, code, scale);

  double err[4] = {0.0, 0.0, 0.0, 0.0}, ref[4] = {0.0, 0.0, 0.0, 0.0};
  float an[4] = {0.0f, 0.0f, 0.0f, 0.0f}, wn[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (live && a.steps > 0) {
    const uint4 av = load_stream<uint4>(a.a + i0), wv = load_stream<uint4>(a.w + i0);
    an[0] = __uint_as_float(av.x); an[1] = __uint_as_float(av.y);
    an[2] = __uint_as_float(av.z); an[3] = __uint_as_float(av.w);
    wn[0] = __uint_as_float(wv.x); wn[1] = __uint_as_float(wv.y);
    wn[2] = __uint_as_float(wv.z); wn[3] = __uint_as_float(wv.w);
  }
  for (int32_t t = 1; t <= a.steps; ++t) {
    float at[4], wt[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) { at[k] = an[k]; wt[k] = wn[k]; }
    if (live && t < a.steps) {  // the next step's rows, in flight while this one rounds
      const int64_t off = static_cast<int64_t>(t) * a.n + i0;
      const uint4 av = load_stream<uint4>(a.a + off), wv = load_stream<uint4>(a.w + off);
      an[0] = __uint_as_float(av.x); an[1] = __uint_as_float(av.y);
      an[2] = __uint_as_float(av.z); an[3] = __uint_as_float(av.w);
      wn[0] = __uint_as_float(wv.x); wn[1] = __uint_as_float(wv.y);
      wn[2] = __uint_as_float(wv.z); wn[3] = __uint_as_float(wv.w);
    }
    float x[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      h[k] = fmaf(at[k], h[k], wt[k]);
      x[k] = fmaf(at[k], hq[k], wt[k]);
    }
    replay_round<F, R>(a, e0, a.step0 + static_cast<uint32_t>(t), x, hq, code, scale);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const double d = static_cast<double>(hq[k]) - static_cast<double>(h[k]);
      err[k] += d * d;
      ref[k] += static_cast<double>(h[k]) * static_cast<double>(h[k]);
    }
    if (t % a.block_steps == 0 || t == a.steps) {
      if (live) {
        const int64_t off = static_cast<int64_t>((t - 1) / a.block_steps) * a.n + i0;
        double2* pe = reinterpret_cast<double2*>(a.err + off);
        pe[0] = make_double2(err[0], err[1]);
        pe[1] = make_double2(err[2], err[3]);
        if (a.ref) {
          double2* pr = reinterpret_cast<double2*>(a.ref + off);
          pr[0] = make_double2(ref[0], ref[1]);
          pr[1] = make_double2(ref[2], ref[3]);
        }
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) { err[k] = 0.0; ref[k] = 0.0; }
    }
  }
  if (!live) return;
  if (a.codes) {
    if constexpr (F == kFP32) {
      *reinterpret_cast<uint4*>(static_cast<uint32_t*>(a.codes) + i0) =
          make_uint4(code[0], code[1], code[2], code[3]);
    } else if constexpr (F == kBF16 || F == kFP16) {
      *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.codes) + i0) =
          make_uint2(code[0] | (code[1] << 16), code[2] | (code[3] << 16));
    } else if constexpr (F == kINT4) {
      static_cast<uint16_t*>(a.codes)[i0 / 4] =
          static_cast<uint16_t>(code[0] | (code[1] << 4) | (code[2] << 8) | (code[3] << 12));
    } else {
      static_cast<uint32_t*>(a.codes)[i0 / 4] =
          code[0] | (code[1] << 8) | (code[2] << 16) | (code[3] << 24);
    }
  }
  if constexpr (Traits<F>::scaled) {
    if (a.scale && (threadIdx.x & (a.lanes_per_group - 1)) == 0)
      a.scale[static_cast<int64_t>(e0 - a.entry_base) >> a.group_shift] = scale;
  }
  if (a.h_final)
    *reinterpret_cast<float4*>(a.h_final + i0) = make_float4(h[0], h[1], h[2], h[3]);
}

// ---------------------------------------------------------------------------
// Causal depthwise conv1d decode update: thread i = b * channels + c shifts its
// channel's window by one, appends x[i] and writes
// out[i] = (silu)(bias[c] + sum_k window[k] * weight[c][k]).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_conv1d_update(ConvArgs a) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= a.n) return;
  const uint32_t c = static_cast<uint32_t>(i) - a.div_channels.div(static_cast<uint32_t>(i)) * a.channels;
  float* const st = a.state + i * a.width;
  const float* const w = a.weight + static_cast<int64_t>(c) * a.width;
  float acc = a.bias ? a.bias[c] : 0.0f;
  for (int k = 0; k < a.width; ++k) {
    const float v = (k + 1 < a.width) ? st[k + 1] : a.x[i];
    st[k] = v;
    acc = fmaf(v, w[k], acc);
  }
  a.out[i] = a.act ? silu(acc) : acc;
}

// ---------------------------------------------------------------------------
// Launchers.
// ---------------------------------------------------------------------------
template <int F, int R, int NT, int CPT, bool N128 = false>
static hipError_t launch_slab(const UpdateArgs& a, hipStream_t s) {
  const int64_t blocks = a.batch * a.nheads * a.slabs_per_head;
  hipLaunchKernelGGL((k_update_slab<F, R, NT, CPT, N128>), dim3(static_cast<unsigned>(blocks)),
                     dim3(NT), 0, s, a);
  return hipGetLastError();
}

template <int F, int R>
static hipError_t launch_slab_cfg(const UpdateArgs& a, int cfg, hipStream_t s) {
  if (a.n128) {  // the configurations the dispatch picks for 128-entry rows
    if constexpr (Traits<F>::scaled) {
      if (cfg == kSlab128x4) return launch_slab<F, R, 128, 4, true>(a, s);
      if (cfg == kSlab256x2) return launch_slab<F, R, 256, 2, true>(a, s);
    } else {
      if (cfg == kSlab512x2) return launch_slab<F, R, 512, 2, true>(a, s);
    }
  }
  switch (cfg) {
    case kSlab64x4: return launch_slab<F, R, 64, 4>(a, s);
    case kSlab128x4: return launch_slab<F, R, 128, 4>(a, s);
    case kSlab256x1: return launch_slab<F, R, 256, 1>(a, s);
    case kSlab256x2: return launch_slab<F, R, 256, 2>(a, s);
    case kSlab256x4: return launch_slab<F, R, 256, 4>(a, s);
    case kSlab512x2: return launch_slab<F, R, 512, 2>(a, s);
    case kSlab512x4: return launch_slab<F, R, 512, 4>(a, s);
    case kSlab1024x4: return launch_slab<F, R, 1024, 4>(a, s);
    case kSlab1024x8: return launch_slab<F, R, 1024, 8>(a, s);
    default: return hipErrorInvalidValue;
  }
}

template <int F, int R>
static hipError_t launch_rows(const UpdateArgs& a, bool a_per_state, hipStream_t s) {
  const unsigned grid = static_cast<unsigned>((a.n_chunks + 255) / 256);
  if (a.fp32_state) {
    if constexpr (F != kFP32) {
      if (a_per_state)
        hipLaunchKernelGGL((k_update_rows<F, R, true, true>), dim3(grid), dim3(256), 0, s, a);
      else
        hipLaunchKernelGGL((k_update_rows<F, R, false, true>), dim3(grid), dim3(256), 0, s, a);
    } else {
      return hipErrorInvalidValue;
    }
  } else if (a_per_state) {
    hipLaunchKernelGGL((k_update_rows<F, R, true, false>), dim3(grid), dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL((k_update_rows<F, R, false, false>), dim3(grid), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

template <int F, int R>
static hipError_t launch_update_fr(const UpdateArgs& a, int cfg, bool aps, hipStream_t s) {
  return cfg == kRowKernel ? launch_rows<F, R>(a, aps, s) : launch_slab_cfg<F, R>(a, cfg, s);
}

template <int F>
static hipError_t launch_update_f(const UpdateArgs& a, int rule, int cfg, bool aps, hipStream_t s) {
  switch (rule) {
    case kRTN: return launch_update_fr<F, kRTN>(a, cfg, aps, s);
    case kSR: return launch_update_fr<F, kSR>(a, cfg, aps, s);
    case kPHILOX: return launch_update_fr<F, kPHILOX>(a, cfg, aps, s);
    default: return launch_update_fr<F, kWEYL>(a, cfg, aps, s);
  }
}

hipError_t launch_update(const UpdateArgs& a, int format, int rule, int cfg, bool a_per_state,
                         hipStream_t s) {
  switch (format) {
    case kFP16: return launch_update_f<kFP16>(a, rule, cfg, a_per_state, s);
    case kBF16: return launch_update_f<kBF16>(a, rule, cfg, a_per_state, s);
    case kE4M3: return launch_update_f<kE4M3>(a, rule, cfg, a_per_state, s);
    case kINT8: return launch_update_f<kINT8>(a, rule, cfg, a_per_state, s);
    case kINT4: return launch_update_f<kINT4>(a, rule, cfg, a_per_state, s);
    default: return launch_update_f<kFP32>(a, rule, cfg, a_per_state, s);
  }
}

template <int F>
static hipError_t launch_requant_f(const RequantArgs& a, int rule, hipStream_t s) {
  constexpr int V = Traits<F>::V;
  const int64_t chunks = (a.n + V - 1) / V;
  const unsigned grid = static_cast<unsigned>((chunks + 255) / 256);
  switch (rule) {
    case kRTN: hipLaunchKernelGGL((k_requant<F, kRTN>), dim3(grid), dim3(256), 0, s, a); break;
    case kSR: hipLaunchKernelGGL((k_requant<F, kSR>), dim3(grid), dim3(256), 0, s, a); break;
    case kPHILOX: hipLaunchKernelGGL((k_requant<F, kPHILOX>), dim3(grid), dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((k_requant<F, kWEYL>), dim3(grid), dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

template <int F, int CPT>
static hipError_t launch_requant_group_wg(const RequantArgs& a, int rule, hipStream_t s) {
  const unsigned grid = static_cast<unsigned>(a.n / a.group);
  switch (rule) {
    case kRTN: hipLaunchKernelGGL((k_requant_group_wg<F, kRTN, CPT>), dim3(grid), dim3(256), 0, s, a); break;
    case kSR: hipLaunchKernelGGL((k_requant_group_wg<F, kSR, CPT>), dim3(grid), dim3(256), 0, s, a); break;
    case kPHILOX: hipLaunchKernelGGL((k_requant_group_wg<F, kPHILOX, CPT>), dim3(grid), dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((k_requant_group_wg<F, kWEYL, CPT>), dim3(grid), dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

template <int F>
static hipError_t launch_requant_scaled(const RequantArgs& a, int rule, hipStream_t s) {
  const int64_t n_groups = a.n / a.group;
  if (n_groups <= 0x7FFFFFFFLL) {
    if (a.group == 4096) return launch_requant_group_wg<F, 1>(a, rule, s);
    if (a.group == 8192) return launch_requant_group_wg<F, 2>(a, rule, s);
  }
  const int64_t gpw = 64 / a.lanes_per_group;
  int64_t blocks = (n_groups + 4 * gpw - 1) / (4 * gpw);
  if (blocks > 65536) blocks = 65536;
  const unsigned grid = static_cast<unsigned>(blocks);
  switch (rule) {
    case kRTN: hipLaunchKernelGGL((k_requant_scaled<F, kRTN>), dim3(grid), dim3(256), 0, s, a); break;
    case kSR: hipLaunchKernelGGL((k_requant_scaled<F, kSR>), dim3(grid), dim3(256), 0, s, a); break;
    case kPHILOX: hipLaunchKernelGGL((k_requant_scaled<F, kPHILOX>), dim3(grid), dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((k_requant_scaled<F, kWEYL>), dim3(grid), dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_requant(const RequantArgs& a, int format, int rule, hipStream_t s) {
  switch (format) {
    case kFP16: return launch_requant_f<kFP16>(a, rule, s);
    case kBF16: return launch_requant_f<kBF16>(a, rule, s);
    case kE4M3: return launch_requant_scaled<kE4M3>(a, rule, s);
    case kINT8: return launch_requant_scaled<kINT8>(a, rule, s);
    case kINT4: return launch_requant_scaled<kINT4>(a, rule, s);
    default: return launch_requant_f<kFP32>(a, rule, s);
  }
}

hipError_t launch_dither(const DitherArgs& a, int rule, hipStream_t s) {
  const int64_t chunks = (a.n + 3) / 4;
  const unsigned grid = static_cast<unsigned>((chunks + 255) / 256);
  switch (rule) {
    case kRTN: hipLaunchKernelGGL((k_dither_fill<kRTN>), dim3(grid), dim3(256), 0, s, a); break;
    case kSR: hipLaunchKernelGGL((k_dither_fill<kSR>), dim3(grid), dim3(256), 0, s, a); break;
    case kPHILOX: hipLaunchKernelGGL((k_dither_fill<kPHILOX>), dim3(grid), dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((k_dither_fill<kWEYL>), dim3(grid), dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

template <int F>
static hipError_t launch_replay_f(const ReplayArgs& a, int rule, hipStream_t s) {
  const unsigned grid = static_cast<unsigned>((a.n / 4 + 255) / 256);
  switch (rule) {
    case kRTN: hipLaunchKernelGGL((k_replay<F, kRTN>), dim3(grid), dim3(256), 0, s, a); break;
    case kSR: hipLaunchKernelGGL((k_replay<F, kSR>), dim3(grid), dim3(256), 0, s, a); break;
    case kPHILOX: hipLaunchKernelGGL((k_replay<F, kPHILOX>), dim3(grid), dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((k_replay<F, kWEYL>), dim3(grid), dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_replay(const ReplayArgs& a, int format, int rule, hipStream_t s) {
  switch (format) {
    case kFP16: return launch_replay_f<kFP16>(a, rule, s);
    case kBF16: return launch_replay_f<kBF16>(a, rule, s);
    case kE4M3: return launch_replay_f<kE4M3>(a, rule, s);
    case kINT8: return launch_replay_f<kINT8>(a, rule, s);
    case kINT4: return launch_replay_f<kINT4>(a, rule, s);
    default: return launch_replay_f<kFP32>(a, rule, s);
  }
}

hipError_t launch_conv1d(const ConvArgs& a, hipStream_t s) {
  const unsigned grid = static_cast<unsigned>((a.n + 255) / 256);
  hipLaunchKernelGGL(k_conv1d_update, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace ssmq
