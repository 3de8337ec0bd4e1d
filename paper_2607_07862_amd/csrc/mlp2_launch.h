// Internal interface between the C ABI (mlp2_api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>

#include "mlp2_device.hpp"

namespace mlp2 {

// A compiled kernel family: row block, GEMM1 / GEMM2 column-block widths and
// the number of GEMM1 weight operands (2 for SwiGLU).
struct KernelConfig {
  int bm, bn1, bn2, nb;
};

bool config_supported(const KernelConfig& c);
hipError_t pipelined_occupancy(const KernelConfig& c, int* blocks_per_cu);
hipError_t launch_sequential(const KernelConfig& c, const Args& a, hipStream_t stream);
hipError_t launch_pipelined(const KernelConfig& c, const Args& a, int grid, hipStream_t stream);

}  // namespace mlp2
