// ssmq_abi.cpp -- the C ABI of include/ssmq.h: host-side validation, launch
// geometry and dispatch. Every check runs before the first HIP call, so a
// rejected call never touches the device.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "ssmq.h"
#include "ssmq_device.hpp"
#include "ssmq_launch.hpp"

namespace {

thread_local char g_last_error[512] = "";

ssmq_status fail(ssmq_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return s;
}

ssmq_status ok() {
  g_last_error[0] = '\0';
  return SSMQ_OK;
}

bool is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }
int log2i(int64_t v) {
  int r = 0;
  while ((int64_t{1} << r) < v) ++r;
  return r;
}
bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Entries per chunk (the unit one lane moves): 16 bytes of fp16/bf16/fp32 or
// E4M3/INT8 codes, 8 bytes of INT4 codes.
int chunk_entries(int format) {
  switch (format) {
    case SSMQ_FP16: case SSMQ_BF16: return 8;
    case SSMQ_FP32: return 4;
    default: return 16;
  }
}
bool is_scaled(int format) {
  return format == SSMQ_FP8_E4M3 || format == SSMQ_INT8 || format == SSMQ_INT4;
}

// Threshold parameters of one call (Appendix B "Dithers"; hash SR) and the
// offset of entry k within a chunk whose first flat index is a multiple of 16.
ssmq::Thr make_thr(int rule, uint32_t seed, uint32_t layer, uint32_t step, int32_t block,
                   uint32_t toff[16]) {
  ssmq::Thr th{};
  th.lb = static_cast<uint32_t>(log2i(block));
  th.seed = seed;
  th.layer = layer;
  th.step = step;
  const uint32_t mask = static_cast<uint32_t>(block) - 1u;
  for (uint32_t k = 0; k < 16; ++k) {
    if (rule == SSMQ_WEYL) toff[k] = ssmq::kWeylA * (k >> th.lb) + ssmq::kWeylB * (k & mask);
    else if (rule == SSMQ_SR) toff[k] = k * ssmq::kSrEntry;
    else toff[k] = 0u;
  }
  if (rule == SSMQ_WEYL) th.key = ssmq::weyl_step_key(seed, layer, step);
  else if (rule == SSMQ_SR) th.key = ssmq::sr_step_key(ssmq::sr_seed_key(seed, layer), step);
  return th;
}

ssmq_status check_qparams(const ssmq_qparams* q) {
  if (!q) return fail(SSMQ_EINVAL, "qparams is NULL");
  if (q->rule < SSMQ_RTN || q->rule > SSMQ_SR_PHILOX)
    return fail(SSMQ_EINVAL, "unknown rule %d", q->rule);
  if (q->format < SSMQ_FP16 || q->format > SSMQ_INT4)
    return fail(SSMQ_EINVAL, "unknown format %d", q->format);
  if ((q->flags & ~static_cast<uint32_t>(SSMQ_FLAG_FP32_STATE)) != 0)
    return fail(SSMQ_EINVAL, "unknown qparams.flags bits 0x%x", q->flags);
  if ((q->flags & SSMQ_FLAG_FP32_STATE) && q->format == SSMQ_FP32)
    return fail(SSMQ_EINVAL, "SSMQ_FLAG_FP32_STATE rounds onto another format's grid, not FP32");
  if (!is_pow2(q->dither_block) || q->dither_block > (1 << 30))
    return fail(SSMQ_EINVAL, "dither_block %d is not a power of two in [1, 2^30]", q->dither_block);
  if (q->entry_base % 16 != 0)
    return fail(SSMQ_EINVAL, "entry_base %llu is not a multiple of 16",
                static_cast<unsigned long long>(q->entry_base));
  if (q->scale_group < 0) return fail(SSMQ_EINVAL, "scale_group is negative");
  return SSMQ_OK;
}

bool mul_ok(int64_t a, int64_t b, int64_t* out) {
  if (a == 0 || b == 0) { *out = 0; return true; }
  if (a > INT64_MAX / b) return false;
  *out = a * b;
  return true;
}

}  // namespace

extern "C" {

const char* ssmq_status_string(ssmq_status s) {
  switch (s) {
    case SSMQ_OK: return "ok";
    case SSMQ_EINVAL: return "invalid argument";
    case SSMQ_EUNSUPPORTED: return "unsupported shape or layout";
    case SSMQ_EALIGN: return "misaligned pointer";
    case SSMQ_EDEVICE: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* ssmq_last_error(void) { return g_last_error; }

ssmq_status ssmq_state_update(const ssmq_dims* dims, const ssmq_qparams* q, void* state,
                              float* state_scale, const float* x, const float* dt,
                              const float* A, const float* B, const float* C, const float* D,
                              float* y, void* stream) {
  return ssmq_state_update_ex(dims, q, nullptr, state, state_scale, x, dt, A, B, C, D, y, stream);
}

ssmq_status ssmq_state_update_ex(const ssmq_dims* dims, const ssmq_qparams* q,
                                 const ssmq_step_opts* opts, void* state, float* state_scale,
                                 const float* x, const float* dt, const float* A, const float* B,
                                 const float* C, const float* D, float* y, void* stream) {
  if (!dims) return fail(SSMQ_EINVAL, "dims is NULL");
  if (opts && (opts->reserved != 0 || (opts->dt_softplus != 0 && opts->dt_softplus != 1)))
    return fail(SSMQ_EINVAL, "opts: dt_softplus must be 0 or 1 and reserved 0");
  if (opts && ((opts->dt_bias && !aligned(opts->dt_bias, 4)) || (opts->z && !aligned(opts->z, 4))))
    return fail(SSMQ_EALIGN, "dt_bias and z must be 4-byte aligned");
  ssmq_status st = check_qparams(q);
  if (st != SSMQ_OK) return st;
  const ssmq_dims& d = *dims;
  if (d.batch < 0) return fail(SSMQ_EINVAL, "batch %lld < 0", static_cast<long long>(d.batch));
  if (d.nheads < 1 || d.headdim < 1 || d.dstate < 1 || d.ngroups < 1)
    return fail(SSMQ_EINVAL, "nheads, headdim, dstate and ngroups must be >= 1");
  if (d.nheads % d.ngroups != 0)
    return fail(SSMQ_EINVAL, "nheads %d is not a multiple of ngroups %d", d.nheads, d.ngroups);
  if (d.a_per_state != 0 && d.a_per_state != 1)
    return fail(SSMQ_EINVAL, "a_per_state must be 0 or 1");
  const bool scaled = is_scaled(q->format);  // E4M3, INT8, INT4: one fp32 scale per group
  const bool fp32_state = (q->flags & SSMQ_FLAG_FP32_STATE) != 0;

  const int V = chunk_entries(q->format);
  if (d.dstate % V != 0 || !is_pow2(d.dstate / V) || d.dstate / V > 64)
    return fail(SSMQ_EUNSUPPORTED,
                "dstate %d: rows must be a power-of-two number (<= 64) of %d-entry chunks",
                d.dstate, V);
  int64_t head_size = 0, n_total = 0, bh = 0;
  if (!mul_ok(d.headdim, d.dstate, &head_size) || !mul_ok(d.batch, d.nheads, &bh) ||
      !mul_ok(bh, head_size, &n_total))
    return fail(SSMQ_EINVAL, "state size overflows int64");
  int64_t group = 0;
  if (scaled) {
    group = q->scale_group ? q->scale_group : head_size;
    if (group % 16 != 0 || group > head_size || head_size % group != 0)
      return fail(SSMQ_EINVAL, "scale_group %lld must be a multiple of 16 dividing headdim*dstate",
                  static_cast<long long>(group));
  }
  if (n_total == 0) return ok();  // nothing to do: the pointers are not read
  if (!state || !x || !dt || !A || !B || !C || !y)
    return fail(SSMQ_EINVAL, "state, x, dt, A, B, C and y must not be NULL");
  if (scaled && !state_scale && !fp32_state)
    return fail(SSMQ_EINVAL, "E4M3, INT8 and INT4 need state_scale");
  if (!aligned(state, 16) || !aligned(B, 16) || !aligned(C, 16) || (d.a_per_state && !aligned(A, 16)))
    return fail(SSMQ_EALIGN, "state, B, C (and A[nheads][dstate]) must be 16-byte aligned");
  if (!aligned(x, 4) || !aligned(dt, 4) || !aligned(A, 4) || !aligned(y, 4) ||
      (D && !aligned(D, 4)) || (state_scale && !aligned(state_scale, 4)))
    return fail(SSMQ_EALIGN, "fp32 arrays must be 4-byte aligned");

  ssmq::UpdateArgs a{};
  a.state = state; a.scale = state_scale; a.x = x; a.dt = dt; a.A = A; a.B = B; a.C = C;
  a.D = D; a.y = y;
  if (opts) {
    a.dt_bias = opts->dt_bias;
    a.dt_softplus = opts->dt_softplus;
    a.z = opts->z;
  }
  a.batch = d.batch; a.nheads = d.nheads; a.headdim = d.headdim; a.dstate = d.dstate;
  a.ngroups = d.ngroups; a.heads_per_group = d.nheads / d.ngroups;
  a.lanes_per_row = d.dstate / V; a.lr_shift = log2i(a.lanes_per_row);
  a.dstate_shift = log2i(d.dstate);
  a.head_size = head_size; a.n_chunks = n_total / V;
  a.entry_base = q->entry_base;
  a.thr = make_thr(q->rule, q->seed, q->layer, q->step, q->dither_block, a.toff);
  a.group_shift = scaled && is_pow2(group) ? log2i(group) : 0;
  const bool small_groups_ok = !scaled || (is_pow2(group / 16) && group / 16 <= 64);
  a.fp32_state = fp32_state ? 1 : 0;
  if (fp32_state && !small_groups_ok)
    return fail(SSMQ_EUNSUPPORTED,
                "with SSMQ_FLAG_FP32_STATE scale groups must be powers of two up to 1024 entries");

  // Slab kernels for per-head A: a workgroup owns whole rows of one head, two
  // chunks per thread (the whole head when it holds 1024 chunks or a multiple:
  // one decay and one B/C staging per head); with one scale per head (scaled
  // formats) the workgroup owns the whole head, four chunks per thread (fewer,
  // fuller threads amortise the per-workgroup scale reduction and its barriers).
  int cfg = -1;
  const int64_t head_chunks = head_size / V;
  if (d.a_per_state == 0 && scaled && group == head_size && !fp32_state) {
    switch (head_chunks) {
      case 256: cfg = ssmq::kSlab64x4; break;
      case 512: cfg = ssmq::kSlab128x4; break;
      case 1024: cfg = ssmq::kSlab256x4; break;
      case 2048: cfg = ssmq::kSlab512x4; break;
      case 4096: cfg = ssmq::kSlab1024x4; break;
      case 8192: cfg = ssmq::kSlab1024x8; break;
      default: break;
    }
    if (cfg >= 0) { a.slabs_per_head = 1; a.lanes_per_group = 0; }
  }
  if (cfg < 0 && d.a_per_state == 0 && small_groups_ok && head_chunks % 256 == 0 && !fp32_state) {
    cfg = (head_chunks % 1024 == 0) ? ssmq::kSlab512x2
          : (head_chunks % 512 == 0)  ? ssmq::kSlab256x2
                                      : ssmq::kSlab256x1;
    a.slabs_per_head = static_cast<int32_t>(
        head_chunks / (ssmq::kSlabThreads[cfg] * ssmq::kSlabChunks[cfg]));
    a.lanes_per_group = scaled ? static_cast<int32_t>(group / 16) : 1;
    // E4M3 block scales: four chunks per thread as with one scale per head
    // (measured 4-8 % faster; the INT kernels measure slower that way).
    if (q->format == SSMQ_FP8_E4M3 && head_chunks % 512 == 0) {
      cfg = ssmq::kSlab128x4;
      a.slabs_per_head = static_cast<int32_t>(head_chunks / 512);
    }
  }
  if (cfg >= 0)
    a.n128 = (d.dstate == 128 && (!scaled || a.lanes_per_group == 0 || a.lanes_per_group == 8)) ? 1 : 0;
  if (cfg >= 0) {  // threshold base advance per pass of NT chunks
    const int64_t step_entries = static_cast<int64_t>(ssmq::kSlabThreads[cfg]) * V;
    a.pass_thr_ok = 1;
    if (q->rule == SSMQ_WEYL) {
      a.pass_thr_ok = (step_entries % q->dither_block) == 0;
      a.pass_thr_inc = ssmq::kWeylA * static_cast<uint32_t>(step_entries >> a.thr.lb);
    } else if (q->rule == SSMQ_SR) {
      a.pass_thr_inc = static_cast<uint32_t>(step_entries) * ssmq::kSrEntry;
    }
  }
  if (cfg >= 0 && bh * a.slabs_per_head > 0x7FFFFFFFLL)
    return fail(SSMQ_EUNSUPPORTED, "state too large for one launch");
  a.div_nheads = ssmq::make_fastdiv(static_cast<uint32_t>(d.nheads));
  a.div_hpg = ssmq::make_fastdiv(static_cast<uint32_t>(a.heads_per_group));
  if (cfg >= 0) a.div_slabs = ssmq::make_fastdiv(static_cast<uint32_t>(a.slabs_per_head));
  if (cfg < 0) {
    if (!small_groups_ok)
      return fail(SSMQ_EUNSUPPORTED,
                  "scale group of %lld entries: supported are powers of two up to 1024 "
                  "entries, or one scale per head of 4096 to 131072 entries with A per head",
                  static_cast<long long>(group));
    if ((n_total >> a.dstate_shift) > 0xFFFFFFFFLL || (a.n_chunks + 255) / 256 > 0x7FFFFFFFLL)
      return fail(SSMQ_EUNSUPPORTED, "state too large for one launch");
    cfg = ssmq::kRowKernel;
    a.lanes_per_group = scaled ? static_cast<int32_t>(group / 16) : 1;
    a.div_headdim = ssmq::make_fastdiv(static_cast<uint32_t>(d.headdim));
  }
  hipError_t e = ssmq::launch_update(a, q->format, q->rule, cfg, d.a_per_state != 0,
                                     static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SSMQ_EDEVICE, "kernel launch: %s", hipGetErrorString(e));
  return ok();
}

ssmq_status ssmq_requantize(const ssmq_qparams* q, int64_t n_entries, int64_t head_size,
                            const float* h, void* codes, float* scale, void* stream) {
  ssmq_status st = check_qparams(q);
  if (st != SSMQ_OK) return st;
  if (n_entries < 0) return fail(SSMQ_EINVAL, "n_entries < 0");
  const bool scaled = is_scaled(q->format);  // E4M3, INT8, INT4
  int64_t group = 0;
  if (scaled) {
    group = q->scale_group ? q->scale_group : head_size;
    if (group <= 0 || group % 16 != 0)
      return fail(SSMQ_EINVAL, "scale group %lld must be a positive multiple of 16",
                  static_cast<long long>(group));
    if (n_entries % group != 0)
      return fail(SSMQ_EINVAL, "n_entries is not a multiple of the scale group");
  }
  if (n_entries == 0) return ok();
  if (!h || !codes || (scaled && !scale)) return fail(SSMQ_EINVAL, "h, codes (and scale) must not be NULL");
  if (!aligned(h, 16) || !aligned(codes, 16) || (scaled && !aligned(scale, 4)))
    return fail(SSMQ_EALIGN, "h and codes must be 16-byte aligned, scale 4-byte aligned");
  ssmq::RequantArgs a{};
  a.h = h; a.codes = codes; a.scale = scale; a.n = n_entries; a.group = group;
  a.entry_base = q->entry_base;
  a.thr = make_thr(q->rule, q->seed, q->layer, q->step, q->dither_block, a.toff);
  a.lanes_per_group = 64;
  if (scaled && group / 16 <= 64 && is_pow2(group / 16)) a.lanes_per_group = static_cast<int32_t>(group / 16);
  if (!scaled && (n_entries + 16 * 256 - 1) / (16 * 256) > 0x7FFFFFFFLL)
    return fail(SSMQ_EUNSUPPORTED, "too many entries for one launch");
  hipError_t e = ssmq::launch_requant(a, q->format, q->rule, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SSMQ_EDEVICE, "kernel launch: %s", hipGetErrorString(e));
  return ok();
}

ssmq_status ssmq_conv1d_update(int64_t batch, int32_t channels, int32_t width, float* conv_state,
                               const float* x, const float* weight, const float* bias,
                               int32_t act, float* out, void* stream) {
  if (batch < 0) return fail(SSMQ_EINVAL, "batch < 0");
  if (channels < 1 || width < 1 || width > 64)
    return fail(SSMQ_EINVAL, "channels must be >= 1 and width in [1, 64]");
  if (act != 0 && act != 1) return fail(SSMQ_EINVAL, "act must be 0 or 1");
  if (batch == 0) return ok();
  if (!conv_state || !x || !weight || !out)
    return fail(SSMQ_EINVAL, "conv_state, x, weight and out must not be NULL");
  if (!aligned(conv_state, 4) || !aligned(x, 4) || !aligned(weight, 4) || !aligned(out, 4) ||
      (bias && !aligned(bias, 4)))
    return fail(SSMQ_EALIGN, "conv1d arrays must be 4-byte aligned");
  int64_t n = 0;
  if (!mul_ok(batch, channels, &n) || n > 0xFFFFFFFFLL)
    return fail(SSMQ_EUNSUPPORTED, "batch * channels must be below 2^32");
  ssmq::ConvArgs a{};
  a.state = conv_state; a.x = x; a.weight = weight; a.bias = bias; a.out = out;
  a.n = n; a.channels = channels; a.width = width; a.act = act;
  a.div_channels = ssmq::make_fastdiv(static_cast<uint32_t>(channels));
  hipError_t e = ssmq::launch_conv1d(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SSMQ_EDEVICE, "kernel launch: %s", hipGetErrorString(e));
  return ok();
}

ssmq_status ssmq_dither_fill(int32_t rule, uint32_t seed, uint32_t layer, uint32_t step,
                             uint64_t entry_base, int64_t n, int32_t dither_block,
                             uint32_t* U24, void* stream) {
  if (rule < SSMQ_RTN || rule > SSMQ_SR_PHILOX) return fail(SSMQ_EINVAL, "unknown rule %d", rule);
  if (n < 0) return fail(SSMQ_EINVAL, "n < 0");
  if (!is_pow2(dither_block) || dither_block > (1 << 30))
    return fail(SSMQ_EINVAL, "dither_block %d is not a power of two in [1, 2^30]", dither_block);
  if (n == 0) return ok();
  if (!U24) return fail(SSMQ_EINVAL, "U24 is NULL");
  if (!aligned(U24, 4)) return fail(SSMQ_EALIGN, "U24 must be 4-byte aligned");
  if ((n + 1023) / 1024 > 0x7FFFFFFFLL) return fail(SSMQ_EUNSUPPORTED, "n too large for one launch");
  ssmq::DitherArgs a{};
  a.out = U24; a.n = n; a.entry_base = entry_base;
  uint32_t unused[16];
  a.thr = make_thr(rule, seed, layer, step, dither_block, unused);
  hipError_t e = ssmq::launch_dither(a, rule, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SSMQ_EDEVICE, "kernel launch: %s", hipGetErrorString(e));
  return ok();
}

ssmq_status ssmq_replay(const ssmq_qparams* q, int64_t n, int32_t steps, int32_t block_steps,
                        const float* h0, const float* a, const float* w, double* err, double* ref,
                        void* codes, float* scale, float* h_final, void* stream) {
  ssmq_status st = check_qparams(q);
  if (st != SSMQ_OK) return st;
  if (q->flags != 0) return fail(SSMQ_EINVAL, "the replay takes no flags");
  if (n < 0 || n % 4 != 0) return fail(SSMQ_EINVAL, "n = %lld is not a multiple of 4 >= 0",
                                       static_cast<long long>(n));
  if (steps < 0) return fail(SSMQ_EINVAL, "steps < 0");
  if (block_steps < 1) return fail(SSMQ_EINVAL, "block_steps < 1");
  const bool scaled = is_scaled(q->format);
  const int64_t group = q->scale_group;
  if (scaled && !(is_pow2(group) && group >= 4 && group <= 256))
    return fail(SSMQ_EUNSUPPORTED, "replay scale groups are powers of two from 4 to 256 entries");
  if (scaled && n % group != 0)
    return fail(SSMQ_EINVAL, "n must be a multiple of the scale group");
  if (n == 0) return ok();
  if (!h0 || (steps > 0 && (!a || !w || !err)))
    return fail(SSMQ_EINVAL, "h0, a, w and err are required");
  if (!aligned(h0, 16) || (a && !aligned(a, 16)) || (w && !aligned(w, 16)) ||
      (err && !aligned(err, 16)) || (ref && !aligned(ref, 16)) || (codes && !aligned(codes, 16)) ||
      (h_final && !aligned(h_final, 16)) || (scale && !aligned(scale, 4)))
    return fail(SSMQ_EALIGN, "h0, a, w, err, ref, codes and h_final must be 16-byte aligned");
  if ((n / 4 + 255) / 256 > 0x7FFFFFFFLL) return fail(SSMQ_EUNSUPPORTED, "n too large for one launch");
  ssmq::ReplayArgs r{};
  r.h0 = h0; r.a = a; r.w = w; r.err = err; r.ref = ref; r.codes = codes;
  r.scale = scaled ? scale : nullptr; r.h_final = h_final;
  r.n = n; r.steps = steps; r.block_steps = block_steps;
  r.lanes_per_group = scaled ? static_cast<int32_t>(group / 4) : 1;
  r.group_shift = scaled ? log2i(group) : 0;
  r.entry_base = q->entry_base;
  r.step0 = q->step;
  uint32_t unused[16];
  r.thr = make_thr(q->rule, q->seed, q->layer, q->step, q->dither_block, unused);
  r.weyl_key0 = ssmq::weyl_step_key(q->seed, q->layer, q->step);
  r.sr_key0 = ssmq::sr_seed_key(q->seed, q->layer);
  hipError_t e = ssmq::launch_replay(r, q->format, q->rule, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SSMQ_EDEVICE, "kernel launch: %s", hipGetErrorString(e));
  return ok();
}

}  // extern "C"
