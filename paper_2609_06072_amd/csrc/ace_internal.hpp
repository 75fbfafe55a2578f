// Host-side declarations shared by the C-ABI layer and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/ace.h"
#include "ace_device.hpp"

namespace ace {

// One adapted projection as the kernels see it.
struct Problem {
  int dtype;       // ACE_F32 / ACE_BF16
  int per_pair;    // input mode
  int T, k, d_in, d_out;
  float alpha;
  const void* x;
  const void* A;
  const void* B;
  const float* pair_w;
  const ace_routing* rt;
  KeyTable keys;   // ranks and rank offsets of the n_keys adapters
  int r_max;
};

int permute_tokens_per_block(int k);
size_t permute_ws_bytes(int T, int k, int n_keys);
hipError_t launch_permute(const int32_t* ids, int T, int k, int E, const int32_t* e2g, int G,
                          int mode, int n_keys, const ace_routing* rt, void* ws,
                          hipStream_t stream);

hipError_t launch_fwd(const Problem& p, void* y, hipStream_t stream);

size_t bwd_ws_bytes(int T, int k, int d_in, int d_out, int R);
hipError_t launch_bwd(const Problem& p, const void* dy, void* dx, float* dA, float* dB, void* ws,
                      hipStream_t stream);

// Number of compute units of the current device (cached per device).
int device_cu_count();

}  // namespace ace
