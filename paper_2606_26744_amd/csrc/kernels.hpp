// Internal launchers of libhdf (not exported).  Each returns the first HIP error
// it meets; argument checking is done by the C-ABI layer before any launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace hdf {

// Compute units of the current device (cached per device).
int device_cu_count();

struct ReduceScalars {
  float eps, gate_scale, gate_offset;
  int per_path_norm;
};

hipError_t launch_hc_reduce(bool bf16, int m, const void* H, const void* Wg, const float* bg,
                            int64_t n_tok, int d, const ReduceScalars& sc, void* Y, float* alpha,
                            hipStream_t s);

hipError_t launch_accept(const int32_t* draft, int stride, const int32_t* target, int n_seq,
                         int K, int32_t* acc, int32_t* anchor, int32_t* offs, int32_t* toks,
                         hipStream_t s);

}  // namespace hdf
