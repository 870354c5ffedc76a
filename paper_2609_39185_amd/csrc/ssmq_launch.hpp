// ssmq_launch.hpp -- kernel argument blocks and launchers shared by the C ABI
// (host side) and the kernels. Internal to the library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ssmq {

// Per-launch threshold parameters.
struct Thr {
  uint32_t key;  // Weyl: A + B + L*layer + S*seed + Phi*t; SR: per-step key
  uint32_t lb;   // log2(dither_block)
  uint32_t seed, layer, step;  // Philox SR: key (seed, layer), counter word 2 = step
};

// Division of 32-bit unsigned integers by an invariant d >= 1 with one high
// multiply (Granlund and Montgomery, "Division by invariant integers using
// multiplication", 1994, Figure 4.1): with l = ceil(log2 d),
// m = floor(2^32 (2^l - d) / d) + 1, t = mulhi(m, n),
// n / d = (t + ((n - t) >> sh1)) >> sh2, sh1 = min(l, 1), sh2 = max(l - 1, 0).
struct FastDiv {
  uint32_t d, m, sh1, sh2;
  __host__ __device__ uint32_t div(uint32_t n) const {
    const uint32_t t = static_cast<uint32_t>((static_cast<uint64_t>(m) * n) >> 32);
    return (t + ((n - t) >> sh1)) >> sh2;
  }
};

inline FastDiv make_fastdiv(uint32_t d) {
  uint32_t l = 0;
  while ((uint64_t{1} << l) < d) ++l;
  FastDiv f;
  f.d = d;
  f.m = static_cast<uint32_t>(((uint64_t{1} << 32) * ((uint64_t{1} << l) - d)) / d + 1);
  f.sh1 = l < 1 ? l : 1;
  f.sh2 = l > 1 ? l - 1 : 0;
  return f;
}

// Launch configurations of the update: slab kernels (threads x chunks per
// thread) and the row kernel.
enum UpdateConfig : int {
  kSlab64x4 = 0, kSlab128x4, kSlab256x1, kSlab256x2, kSlab256x4, kSlab512x2, kSlab512x4,
  kSlab1024x4, kSlab1024x8, kRowKernel
};
constexpr int kSlabThreads[] = {64, 128, 256, 256, 256, 512, 512, 1024, 1024};
constexpr int kSlabChunks[] = {4, 4, 1, 2, 4, 2, 4, 4, 8};
constexpr int kMaxDstate = 1024;  // 64 lanes x 16 E4M3 entries per row

struct UpdateArgs {
  void* state;
  float* scale;
  const float* x;
  const float* dt;
  const float* A;
  const float* B;
  const float* C;
  const float* D;
  float* y;
  const float* dt_bias;     // [nheads] added to dt, or null
  const float* z;           // [batch][nheads][headdim] gate y <- y * silu(z), or null
  int32_t dt_softplus;      // dt <- softplus(dt + dt_bias)
  int64_t batch;
  int32_t nheads, headdim, dstate, ngroups;
  int32_t heads_per_group;
  int32_t lanes_per_row;    // dstate / V, a power of two <= 64
  int32_t lr_shift;         // log2(lanes_per_row)
  int32_t dstate_shift;     // log2(dstate)
  int32_t group_shift;      // E4M3: log2(entries per scale) when that is a power of two
  int32_t lanes_per_group;  // E4M3: group / 16 lanes; 0 = one scale per head slab
  int32_t slabs_per_head;   // slab kernels: workgroups per (batch, head) tile
  int64_t head_size;        // headdim * dstate
  int64_t n_chunks;         // total entries / V
  uint64_t entry_base;
  int32_t fp32_state;       // row kernel: fp32 state, values rounded onto F's grid (a checkpoint)
  Thr thr;
  uint32_t toff[16];        // threshold offset of entry k of a chunk
  uint32_t pass_thr_inc;    // slab kernels: threshold base increment per pass ...
  int32_t pass_thr_ok;      // ... when a pass advances by whole dither blocks (or SR)
  int32_t n128;             // slab kernels: dstate 128, groups of 128 entries or one head
  FastDiv div_headdim, div_nheads, div_hpg, div_slabs;  // index arithmetic
};

struct RequantArgs {
  const float* h;
  void* codes;
  float* scale;
  int64_t n;
  int64_t group;            // E4M3 entries per scale
  int32_t lanes_per_group;  // E4M3 lanes cooperating on one group
  uint64_t entry_base;
  Thr thr;
  uint32_t toff[16];
};

struct ConvArgs {
  float* state;             // [n][width]
  const float* x;           // [n]
  const float* weight;      // [channels][width]
  const float* bias;        // [channels] or null
  float* out;               // [n]
  int64_t n;                // batch * channels
  int32_t channels, width, act;
  FastDiv div_channels;
};

struct DitherArgs {
  uint32_t* out;
  int64_t n;
  uint64_t entry_base;
  Thr thr;
};

// Open-loop replay of recorded decays and writes: four entries per thread.
struct ReplayArgs {
  const float* h0;          // [n]
  const float* a;           // [steps][n]
  const float* w;           // [steps][n]
  double* err;              // [n_blocks][n]
  double* ref;              // [n_blocks][n] or null
  void* codes;              // final codes or null
  float* scale;             // final group scales or null
  float* h_final;           // final reference state or null
  int64_t n;                // entries, a multiple of 4
  int32_t steps, block_steps;
  int32_t lanes_per_group;  // scaled formats: group / 4, a power of two <= 64
  int32_t group_shift;      // log2(group)
  uint64_t entry_base;      // a multiple of 4
  uint32_t step0;           // step of the write of h0
  uint32_t weyl_key0;       // Weyl key at step0
  uint32_t sr_key0;         // hash SR seed-and-layer key
  Thr thr;                  // lb, seed, layer (key and step set per step)
};

hipError_t launch_replay(const ReplayArgs& a, int format, int rule, hipStream_t s);
hipError_t launch_update(const UpdateArgs& a, int format, int rule, int cfg, bool a_per_state,
                         hipStream_t s);
hipError_t launch_requant(const RequantArgs& a, int format, int rule, hipStream_t s);
hipError_t launch_dither(const DitherArgs& a, int rule, hipStream_t s);
hipError_t launch_conv1d(const ConvArgs& a, hipStream_t s);

}  // namespace ssmq
