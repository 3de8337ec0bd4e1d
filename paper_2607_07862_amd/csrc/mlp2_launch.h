// Internal interface between the C ABI (mlp2_api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>

#include "mlp2_device.hpp"

namespace mlp2 {

// A compiled kernel family: row block, GEMM1 / GEMM2 column-block widths, the
// number of GEMM1 weight operands (2 for SwiGLU), the LDS ring depth, the
// waves per work-group (4 or 8) and the K depth of a stage (64 or 32).
struct KernelConfig {
  int bm, bn1, bn2, nb, ns, waves, bk;
  int wnt;  // weight loads with the non-temporal hint
};

bool config_supported(const KernelConfig& c);
// Resident work-groups per CU of a kernel: which = 0 (GEMM1 phase), 1 (GEMM2 phase), 2 (pipelined),
// 3 (workqueue), 4 (sentinel).
hipError_t occupancy(const KernelConfig& c, int which, int* blocks_per_cu);
// a1 / a2: arguments of the GEMM1 / GEMM2 launch (they differ only in `lists`); stages: 1 = the
// GEMM1 kernel, 2 = the GEMM2 kernel, 3 = both in that order.
hipError_t launch_sequential(const KernelConfig& c, const Args& a1, const Args& a2, const int grids[2], hipStream_t stream,
                             int stages);
hipError_t launch_pipelined(const KernelConfig& c, const Args& a, int grid, hipStream_t stream);
hipError_t launch_workqueue(const KernelConfig& c, const Args& a, int grid, hipStream_t stream);
hipError_t launch_sentinel(const KernelConfig& c, const Args& a, int grid, hipStream_t stream);

// ---- GEMM chain: Z_l = act(Z_{l-1} W_l), Y = Z_{L-1} W_L, no split-K.
constexpr int kChainMaxLayers = 8;
constexpr int kChainWidthUnit = 128;  // every width is a multiple of this
// Tile shapes of the chain kernel: 0 = 128 x 128 (four waves, two-stage ring), 1 = 64 x 64 (four
// waves, four stages), 2 = 256 x 256 (eight waves, two-stage ring).
constexpr int kChainTiles[3] = {128, 64, 256};

// One layer of a chain launch (passed by value with every launch).
struct ChainLayer {
  const uint16_t* A;         // input rows, row stride K: X or the previous layer's Z
  const uint16_t* W;         // [K, N]
  uint16_t* out;             // this layer's Z [Mpad, N], or Y [M, N] for the last layer
  const uint32_t* ready_in;  // the producing layer's ready counters (null: first layer)
  uint32_t* ready_out;       // this layer's ready counters (null: last layer)
  int K, N;
  int alast;                 // last input row a load may touch (rows past it are clamped to it)
  int act;                   // activation on the output (MLP2_ACT_IDENTITY or MLP2_ACT_GELU_TANH)
  int guard;                 // store rows < M only (the last layer writes Y)
};

// Arguments of a chain launch.  `a` carries the control words, claim lists,
// spin limit, M, Mb and the rank table (orderp, a.items1 ranks; entry =
// layer << 24 | tile with tile = nb * Mb + mb).
struct ChainArgs {
  Args a;
  ChainLayer layer[kChainMaxLayers];
  int wait;        // items wait on their producing layer's ready counters (one launch for all layers)
  int end_of_run;  // the run's last launch: it advances the epoch
};

hipError_t chain_occupancy(int tile, int* blocks_per_cu);
hipError_t launch_chain(int tile, const ChainArgs& c, int grid, hipStream_t stream);

}  // namespace mlp2
