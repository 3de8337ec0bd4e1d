// Internal interface between the C ABI (mlp2_api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>

#include "mlp2_device.hpp"

namespace mlp2 {

// A compiled kernel family: row block, GEMM1 / GEMM2 column-block widths, the
// number of GEMM1 weight operands (2 for SwiGLU) and the LDS ring depth.
struct KernelConfig {
  int bm, bn1, bn2, nb, ns;
};

bool config_supported(const KernelConfig& c);
// Resident work-groups per CU of a kernel: which = 0 (GEMM1 phase), 1 (GEMM2 phase), 2 (pipelined),
// 3 (workqueue).
hipError_t occupancy(const KernelConfig& c, int which, int* blocks_per_cu);
// a1 / a2: arguments of the GEMM1 / GEMM2 launch (they differ only in `lists`).
hipError_t launch_sequential(const KernelConfig& c, const Args& a1, const Args& a2, const int grids[2], hipStream_t stream);
hipError_t launch_pipelined(const KernelConfig& c, const Args& a, int grid, hipStream_t stream);
hipError_t launch_workqueue(const KernelConfig& c, const Args& a, int grid, hipStream_t stream);

}  // namespace mlp2
