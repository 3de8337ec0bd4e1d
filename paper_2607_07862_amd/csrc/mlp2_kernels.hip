// Kernels of the tile-pipelined two-layer MLP and their launchers.
//
//   k_gemm1      GEMM1 work items, one per work-group (sequential mode)
//   k_gemm2      GEMM2 work items, one per work-group (sequential mode)
//   k_pipelined  one persistent launch doing both (tile-pipelined mode)
//
// Both modes run the same item functions below, so they produce the same
// bits: the same tiles, the same ascending K order inside a tile, the same
// fixed-order split-K reduction and the same epilogues.  The pipelined launch
// differs only in *when* a GEMM2 item may read a K-slice of Z: as soon as the
// GEMM1 tile that produced it has signalled (Sec. III-A of the paper: the
// consumer runs once every producer tile it reads is complete).
//
// Scheduling of the pipelined launch: a global ticket hands out the GEMM1
// items first, in the order of the plan's order table (column-block-first by
// default, Sec. III-A.5: the first kernel may follow a predefined order), then
// the GEMM2 items.  A GEMM2 item only ever waits for GEMM1 items that were
// claimed before it by running work-groups that never wait, so the launch
// cannot deadlock whatever its grid size or residency.
#include "mlp2_device.hpp"
#include "mlp2_launch.h"

namespace mlp2 {

// ------------------------------------------------------------------ work items

template <class T, int NB>
__device__ __forceinline__ void gemm1_item(const Args& a, int id_in, uint32_t epoch, uint16_t* lds, int* s_flag) {
  const int id = uniform(id_in);
  const int tile = id / a.S1, s = id - (id / a.S1) * a.S1;
  const int mb = tile % a.Mb, nb = tile / a.Mb;
  const int m0 = mb * T::BM, n0 = nb * T::BN;
  const int kbeg = s * a.kc1;
  const int kend = min(a.H, kbeg + a.kc1);

  f32x4 acc[NB][T::TN][T::TM];
  const uint16_t* Bp[NB];
  Bp[0] = a.W1;
  if constexpr (NB == 2) Bp[1] = a.W1 + (long)a.H * a.F;
  NoWait nowait;
  mainloop<T, NB>(a.X, a.H, m0, a.M - 1, Bp, a.F, n0, kbeg, kend, acc, lds, nowait);

  if (a.S1 > 1) {
    store_partial<T, NB>(a.part1, tile, a.S1, s, acc);
    const bool last = arrive_last(a.cnt1 + tile, epoch, a.S1, s_flag);
    if (!last) return;  // uniform; no barrier follows in this item
    reduce_partials<T, NB>(a.part1, tile, a.S1, acc);
  }

  // Fused epilogue: activation in fp32, round to bf16, 16-byte stores of Z.
  FragPos<T> fp(m0, n0);
#pragma unroll
  for (int tm = 0; tm < T::TM; ++tm) {
#pragma unroll
    for (int tp = 0; tp < T::TN / 2; ++tp) {
      float v[8];
      if constexpr (NB == 2) {
        float gt[8], up[8];
        pair_values<T>(acc[0], tp, tm, gt);
        pair_values<T>(acc[1], tp, tm, up);
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = silu(gt[i]) * up[i];
      } else {
        pair_values<T>(acc[0], tp, tm, v);
        if (a.act == ACT_GELU_TANH) {
#pragma unroll
          for (int i = 0; i < 8; ++i) v[i] = gelu_tanh(v[i]);
        }
      }
      const long row = fp.row0 + 16 * tm;
      const int col = fp.col0 + 32 * tp;
      *reinterpret_cast<u32x4*>(a.Z + row * a.F + col) = pack_bf16x8(v);
    }
  }
  // Producer signal: Z tile complete and released, then ready[tile] += 1.
  if (tile != a.drop_signal) {
    signal_ready(a.ready + tile);
  } else {
    wait_all_mem();
    __syncthreads();
  }
}

// GEMM2 item p: split s = p / tiles2 (lower splits first: they read the
// column blocks of Z that complete first), tile = p % tiles2.
template <class T, bool WAIT>
__device__ __forceinline__ void gemm2_item(const Args& a, int p_in, uint32_t epoch, uint16_t* lds, int* s_flag) {
  const int p = uniform(p_in);
  const int tiles2 = a.Mb * a.Nb2;
  const int s = p / tiles2, tile = p - s * tiles2;
  const int mb = tile % a.Mb, nb = tile / a.Mb;
  const int m0 = mb * T::BM, n0 = nb * T::BN;
  const int kbeg = s * a.kc2;
  const int kend = min(a.F, kbeg + a.kc2);

  f32x4 acc[1][T::TN][T::TM];
  const uint16_t* Bp[1] = {a.W2};
  const int zlast = a.Mb * T::BM - 1;
  if constexpr (WAIT) {
    ReadyWait w{a.ready, a.ctrl + CTRL_ERROR, mb, a.Mb, a.bn1, epoch + 1u, a.spin_limit, -1};
    mainloop<T, 1>(a.Z, a.F, m0, zlast, Bp, a.H, n0, kbeg, kend, acc, lds, w);
  } else {
    NoWait nowait;
    mainloop<T, 1>(a.Z, a.F, m0, zlast, Bp, a.H, n0, kbeg, kend, acc, lds, nowait);
  }

  if (a.S2 > 1) {
    store_partial<T, 1>(a.part2, tile, a.S2, s, acc);
    const bool last = arrive_last(a.cnt2 + tile, epoch, a.S2, s_flag);
    if (!last) return;  // uniform; no barrier follows in this item
    reduce_partials<T, 1>(a.part2, tile, a.S2, acc);
  }

  FragPos<T> fp(m0, n0);
#pragma unroll
  for (int tm = 0; tm < T::TM; ++tm) {
    const int row = fp.row0 + 16 * tm;
    if (row < a.M) {
#pragma unroll
      for (int tp = 0; tp < T::TN / 2; ++tp) {
        float v[8];
        pair_values<T>(acc[0], tp, tm, v);
        *reinterpret_cast<u32x4*>(a.Y + (long)row * a.H + fp.col0 + 32 * tp) = pack_bf16x8(v);
      }
    }
  }
}

// The last work-group of a run's final kernel resets the ticket and the done
// count and advances the epoch (all stream-ordered before the next run).
__device__ __forceinline__ void finish_run(const Args& a, uint32_t epoch) {
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t old = __hip_atomic_fetch_add(a.ctrl + CTRL_DONE, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    if (old == gridDim.x - 1) {
      __hip_atomic_store(a.ctrl + CTRL_TICKET, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(a.ctrl + CTRL_DONE, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(a.ctrl + CTRL_EPOCH, epoch + 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// ------------------------------------------------------------------ kernels

template <int A, int B>
struct MaxI {
  static constexpr int value = A > B ? A : B;
};

template <class T1, int NB, class T2>
__global__ __launch_bounds__(kThreads) void k_gemm1(Args a) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[T1::template lds_elems<NB>()];
  __shared__ int s_flag;
  const uint32_t epoch = uniform(ld_relaxed(a.ctrl + CTRL_EPOCH));
  gemm1_item<T1, NB>(a, (int)a.order1[blockIdx.x], epoch, lds, &s_flag);
}

template <class T1, int NB, class T2>
__global__ __launch_bounds__(kThreads) void k_gemm2(Args a) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[T2::template lds_elems<1>()];
  __shared__ int s_flag;
  const uint32_t epoch = uniform(ld_relaxed(a.ctrl + CTRL_EPOCH));
  gemm2_item<T2, false>(a, blockIdx.x, epoch, lds, &s_flag);
  finish_run(a, epoch);
}

template <class T1, int NB, class T2>
__global__ __launch_bounds__(kThreads) void k_pipelined(Args a) {
  constexpr int kLds = MaxI<T1::template lds_elems<NB>(), T2::template lds_elems<1>()>::value;
  __shared__ __attribute__((aligned(16))) uint16_t lds[kLds];
  __shared__ int s_item, s_flag;
  const uint32_t epoch = uniform(ld_relaxed(a.ctrl + CTRL_EPOCH));
  const int total = a.items1 + a.items2;
  for (;;) {
    if (threadIdx.x == 0)
      s_item = (int)__hip_atomic_fetch_add(a.ctrl + CTRL_TICKET, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    const int p = uniform(s_item);
    __syncthreads();  // s_item is rewritten at the next ticket
    if (p >= total) break;
    if (p < a.items1)
      gemm1_item<T1, NB>(a, (int)a.order1[p], epoch, lds, &s_flag);
    else
      gemm2_item<T2, true>(a, p - a.items1, epoch, lds, &s_flag);
    __syncthreads();  // the item's last LDS reads complete before the next item's writes
  }
  finish_run(a, epoch);
}

// ------------------------------------------------------------------ dispatch table

template <int BM, int BN>
struct TileFor;
template <> struct TileFor<32, 64> { using type = Tile<32, 64, 2, 2>; };
template <> struct TileFor<32, 128> { using type = Tile<32, 128, 1, 4>; };
template <> struct TileFor<64, 64> { using type = Tile<64, 64, 2, 2>; };
template <> struct TileFor<64, 128> { using type = Tile<64, 128, 2, 2>; };
template <> struct TileFor<128, 64> { using type = Tile<128, 64, 2, 2>; };
template <> struct TileFor<128, 128> { using type = Tile<128, 128, 2, 2>; };

struct Entry {
  int bm, bn1, bn2, nb;
  const void* seq1;
  const void* seq2;
  const void* pipe;
};

#define MLP2_ENTRY(BM, BN1, BN2, NB)                                                                    \
  Entry {                                                                                               \
    BM, BN1, BN2, NB,                                                                                   \
        (const void*)&k_gemm1<typename TileFor<BM, BN1>::type, NB, typename TileFor<BM, BN2>::type>,    \
        (const void*)&k_gemm2<typename TileFor<BM, BN1>::type, NB, typename TileFor<BM, BN2>::type>,    \
        (const void*)&k_pipelined<typename TileFor<BM, BN1>::type, NB, typename TileFor<BM, BN2>::type> \
  }

static const Entry kEntries[] = {
    MLP2_ENTRY(32, 128, 128, 1), MLP2_ENTRY(32, 128, 64, 1), MLP2_ENTRY(32, 64, 128, 1), MLP2_ENTRY(32, 64, 64, 1),
    MLP2_ENTRY(64, 128, 128, 1), MLP2_ENTRY(64, 128, 64, 1), MLP2_ENTRY(64, 64, 128, 1), MLP2_ENTRY(64, 64, 64, 1),
    MLP2_ENTRY(128, 128, 128, 1), MLP2_ENTRY(128, 128, 64, 1), MLP2_ENTRY(128, 64, 128, 1), MLP2_ENTRY(128, 64, 64, 1),
    MLP2_ENTRY(32, 64, 128, 2), MLP2_ENTRY(32, 64, 64, 2), MLP2_ENTRY(64, 64, 128, 2), MLP2_ENTRY(64, 64, 64, 2),
    MLP2_ENTRY(128, 64, 128, 2), MLP2_ENTRY(128, 64, 64, 2),
};

static const Entry* find_entry(const KernelConfig& c) {
  for (const Entry& e : kEntries)
    if (e.bm == c.bm && e.bn1 == c.bn1 && e.bn2 == c.bn2 && e.nb == c.nb) return &e;
  return nullptr;
}

bool config_supported(const KernelConfig& c) { return find_entry(c) != nullptr; }

hipError_t pipelined_occupancy(const KernelConfig& c, int* blocks_per_cu) {
  const Entry* e = find_entry(c);
  if (!e) return hipErrorInvalidValue;
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, e->pipe, kThreads, 0);
}

hipError_t launch_sequential(const KernelConfig& c, const Args& a, hipStream_t stream) {
  const Entry* e = find_entry(c);
  if (!e) return hipErrorInvalidValue;
  void* args[] = {const_cast<Args*>(&a)};
  hipError_t err = hipLaunchKernel(e->seq1, dim3(a.items1), dim3(kThreads), args, 0, stream);
  if (err != hipSuccess) return err;
  return hipLaunchKernel(e->seq2, dim3(a.items2), dim3(kThreads), args, 0, stream);
}

hipError_t launch_pipelined(const KernelConfig& c, const Args& a, int grid, hipStream_t stream) {
  const Entry* e = find_entry(c);
  if (!e) return hipErrorInvalidValue;
  void* args[] = {const_cast<Args*>(&a)};
  return hipLaunchKernel(e->pipe, dim3(grid), dim3(kThreads), args, 0, stream);
}

}  // namespace mlp2
