// The allocation-free entry point: mlp2_run_noalloc.
//
// For callers that cannot allocate device memory (code under graph capture,
// tight serving loops, harnesses that forbid allocation): one call plans and
// runs Y = act(X W1) W2 with every piece of workspace the kernels need (the
// intermediate Z, split-K partials, ready and arrival counters, control
// words, rank tables) carved out of `scratch`, a static device array of
// kScratchBytes that each GPU the library runs on holds until the process
// ends.  Host code never passes the array's name to a kernel (in host code
// it is a stand-in, not a device address): the device address is taken once
// per device with hipGetSymbolAddress and kept in g_scratch.
//
// Each call clears the counter region and writes the rank tables with a
// small fill kernel on the caller's stream (no hipMemsetAsync, so a captured
// graph records kernels only), then enqueues the same kernels as mlp2_run.
// Every call on a GPU shares that GPU's array: calls that overlap on one GPU
// (two streams, or two host threads) race and give undefined results.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <mutex>

#include "../../include/mlp2.h"
#include "mlp2_plan_impl.h"

namespace mlp2 {

constexpr size_t kScratchBytes = (size_t)64 << 20;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) char scratch[kScratchBytes];

static void* g_scratch[kMaxDevices];   // device address of `scratch` on each device, once known
static int g_num_cus[kMaxDevices];     // compute units of each device
static std::mutex g_scratch_mutex;

// The calling thread's device: its scratch address and CU count, looked up
// on the first call on that device.  MLP2_OK or an error code.
static int scratch_for(int dev, char** base, int* num_cus) {
  if (dev < 0 || dev >= kMaxDevices) return MLP2_ERR_DEVICE;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch[dev]) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return MLP2_ERR_HIP;
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0) return MLP2_ERR_DEVICE;
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return MLP2_ERR_HIP;
    g_num_cus[dev] = prop.multiProcessorCount;
    g_scratch[dev] = ptr;
  }
  *base = (char*)g_scratch[dev];
  *num_cus = g_num_cus[dev];
  return MLP2_OK;
}

// Zero the counter region (every counter, scoreboard, queue slot and control
// word, the epoch included, so each call starts from a fresh plan's state) and
// write the rank tables: GEMM1 and GEMM2 items in id order (column blocks
// first), the pipelined table every GEMM1 item, then every GEMM2 item, then
// (GEMM2 split-K) every reduction item, which the GEMM2 table ends with too.
__global__ void k_noalloc_init(uint32_t* counters, int counter_words, uint32_t* order1, int items1, uint32_t* order2,
                               int items2, int items_red, uint32_t* orderp) {
  const int stride = (int)(gridDim.x * blockDim.x);
  for (int i = (int)(blockIdx.x * blockDim.x + threadIdx.x); i < counter_words; i += stride) counters[i] = 0u;
  for (int i = (int)(blockIdx.x * blockDim.x + threadIdx.x); i < items1 + items2 + items_red; i += stride) {
    if (i < items1) {
      order1[i] = (uint32_t)i;
      orderp[i] = (uint32_t)i;
    } else if (i < items1 + items2) {
      order2[i - items1] = (uint32_t)(i - items1);
      orderp[i] = 0x80000000u | (uint32_t)(i - items1);
    } else {
      order2[i - items1] = 0x40000000u | (uint32_t)(i - items1 - items2);
      orderp[i] = 0xc0000000u | (uint32_t)(i - items1 - items2);
    }
  }
}

}  // namespace mlp2

extern "C" int mlp2_run_noalloc(int64_t M, int64_t H, int64_t F, int act, int dtype, const void* X, const void* W1,
                                const void* W2, void* Y, void* stream, int mode) {
  using namespace mlp2;
  if (M < 1 || H < 1 || F < 1 || !X || !W1 || !W2 || !Y) return record_error(MLP2_ERR_INVALID_ARG);
  if (act < MLP2_ACT_IDENTITY || act > MLP2_ACT_SWIGLU || dtype != MLP2_DTYPE_BF16) return record_error(MLP2_ERR_INVALID_ARG);
  if (mode != MLP2_MODE_SEQUENTIAL && mode != MLP2_MODE_TILE_PIPELINED && mode != MLP2_MODE_WORKQUEUE)
    return record_error(MLP2_ERR_INVALID_ARG);
  if (M > (1 << 20) || H % 64 || F % 64 || H > (1 << 18) || F > (1 << 18)) return record_error(MLP2_ERR_UNSUPPORTED);
  if (((uintptr_t)X | (uintptr_t)W1 | (uintptr_t)W2 | (uintptr_t)Y) & 15u) return record_error(MLP2_ERR_ALIGNMENT);
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return record_error(MLP2_ERR_HIP);
  char* base = nullptr;
  int num_cus = 0;
  int rc = scratch_for(dev, &base, &num_cus);
  if (rc != MLP2_OK) return record_error(rc);

  // The plan lives on this call's stack; its tables are the column-first
  // order with every GEMM2 item after every GEMM1 item in the pipelined table.
  mlp2_plan_s p;
  mlp2_tuning_t tz;
  std::memset(&tz, 0, sizeof(tz));
  tz.lag = -1;
  rc = configure_plan(&p, M, H, F, act, tz, dev, num_cus);
  if (rc != MLP2_OK) return record_error(rc);
  PlanLayout L;
  if (plan_layout(&p, true, &L, false) > kScratchBytes) return record_error(MLP2_ERR_UNSUPPORTED);  // beyond the scratch
  bind_plan(&p, base, L, nullptr);
  p.ws = base;
  p.ws_bytes = L.bytes;

  hipStream_t s = (hipStream_t)stream;
  const int words = (int)((L.cnt_end - L.cnt_off) / 4);
  const int n = std::max(words, p.items1 + p.items2 + p.items_red);
  const int grid = std::min(1024, (n + 255) / 256);
  hipLaunchKernelGGL(k_noalloc_init, dim3(grid), dim3(256), 0, s, (uint32_t*)(base + L.cnt_off), words, p.order1,
                     p.items1, p.order2, p.items2, p.items_red, p.orderp);
  if (hipGetLastError() != hipSuccess) return record_error(MLP2_ERR_HIP);
  return launch_plan(&p, X, W1, W2, Y, p.Z, s, mode);
}
