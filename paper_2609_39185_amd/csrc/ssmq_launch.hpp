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
};

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
  int64_t batch;
  int32_t nheads, headdim, dstate, ngroups;
  int32_t heads_per_group;
  int32_t lanes_per_row;    // dstate / V, a power of two <= 64
  int32_t lr_shift;         // log2(lanes_per_row)
  int32_t group;            // E4M3 entries per scale
  int32_t lanes_per_group;  // E4M3: group / 16 lanes; 0 = one scale per head tile
  int64_t head_size;        // headdim * dstate
  int64_t n_chunks;         // total entries / V
  uint64_t entry_base;
  Thr thr;
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
};

struct DitherArgs {
  uint32_t* out;
  int64_t n;
  uint64_t entry_base;
  Thr thr;
};

// kind 0: head-tile kernel with `cpt` chunks per thread; kind 1: row kernel.
hipError_t launch_update(const UpdateArgs& a, int format, int rule, int kind, int cpt,
                         bool a_per_state, hipStream_t s);
hipError_t launch_requant(const RequantArgs& a, int format, int rule, hipStream_t s);
hipError_t launch_dither(const DitherArgs& a, int rule, hipStream_t s);

}  // namespace ssmq
