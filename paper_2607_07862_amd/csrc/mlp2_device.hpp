// Device building blocks of the tile-pipelined two-layer MLP on gfx950.
//
//   * an LDS double-buffered bf16 MFMA tile mainloop (v_mfma_f32_16x16x32_bf16),
//     with the row-major weight tile read transposed out of LDS by
//     ds_read_b64_tr_b16;
//   * the fused epilogues: activation + bf16 store + ready signal for GEMM1,
//     bf16 store for GEMM2, and a deterministic split-K reduction;
//   * the flag primitives: release-increment of a ready counter by the
//     producer, bounded acquire-spin by the consumer (Sec. III-A: the
//     producer fences its data before it signals; the consumer polls before
//     it reads).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mlp2 {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4_t;

constexpr int kThreads = 256;  // four 64-wide waves per work-group
constexpr int kBK = 64;        // K depth of one LDS stage

// Control words of a plan (device memory, zero at plan creation).
enum {
  CTRL_EPOCH = 0,   // runs completed; read at kernel start, bumped by the run's last work-group
  CTRL_TICKET = 1,  // next work item of the pipelined launch
  CTRL_DONE = 2,    // work-groups of the run's final kernel that have finished
  CTRL_ERROR = 3,   // nonzero once a bounded flag wait gave up
  CTRL_WORDS = 16
};

enum { ACT_IDENTITY = 0, ACT_GELU_TANH = 1, ACT_SWIGLU = 2 };

struct Args {
  const uint16_t* X;   // [M, H]
  const uint16_t* W1;  // [H, F]  (SwiGLU: [2, H, F])
  const uint16_t* W2;  // [F, H]
  uint16_t* Y;         // [M, H]
  uint16_t* Z;         // [Mpad, F]
  float* part1;        // GEMM1 split-K partials (fragment-native), or null
  float* part2;        // GEMM2 split-K partials, or null
  uint32_t* cnt1;      // [tiles1] split-K arrival counters of GEMM1
  uint32_t* cnt2;      // [tiles2] split-K arrival counters of GEMM2
  uint32_t* ready;     // [tiles1] ready counters: tile (mb, nb1) at index nb1 * Mb + mb
  uint32_t* ctrl;      // CTRL_* words
  const uint32_t* order1;  // GEMM1 item order, length items1
  int M, H, F, act;
  int Mb, Nb1, Nb2;        // row blocks; GEMM1 / GEMM2 column blocks
  int S1, S2;              // split-K factors
  int kc1, kc2;            // K per split (multiples of kBK)
  int items1, items2;
  int bn1;                 // GEMM1 column-block width (ready-counter granularity along GEMM2's K)
  uint32_t spin_limit;
  int drop_signal;         // GEMM1 tile whose signal is skipped (failure injection), -1 = none
};

// ------------------------------------------------------------------ scalars

__device__ __forceinline__ uint32_t ld_relaxed(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// A value every lane of the wave holds (read from LDS after a barrier, or
// loaded from a wave-uniform address), moved to a scalar register so that
// branches on it are scalar branches.  Every branch that has a barrier on
// either side must be taken this way: the compiler cannot prove uniformity
// of an LDS or memory value by itself and would otherwise lay the code out as
// an exec-masked divergent region, in which waves can execute different
// numbers of s_barrier and deadlock the work-group.
__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ uint32_t uniform(uint32_t v) { return (uint32_t)__builtin_amdgcn_readfirstlane((int)v); }

// Every wave waits until its own outstanding memory operations are complete
// (stores acknowledged), so that a later agent-scope release by one lane of
// the work-group covers the data of all waves.
__device__ __forceinline__ void wait_all_mem() { __builtin_amdgcn_s_waitcnt(0); }

// e^{-t} through the hardware base-2 exponential.
__device__ __forceinline__ float exp_neg(float t) { return __builtin_amdgcn_exp2f(-1.4426950408889634f * t); }

// GELU (tanh form): 0.5 z (1 + tanh(y)) with y = sqrt(2/pi)(z + 0.044715 z^3).
// Uses the identity 0.5 (1 + tanh(y)) = 1 / (1 + e^{-2y}).
__device__ __forceinline__ float gelu_tanh(float z) {
  const float y = 0.7978845608028654f * (z + 0.044715f * z * z * z);
  return z / (1.0f + exp_neg(2.0f * y));
}

// SiLU: g / (1 + e^{-g}).
__device__ __forceinline__ float silu(float g) { return g / (1.0f + exp_neg(g)); }

__device__ __forceinline__ u32x4 pack_bf16x8(const float (&v)[8]) {
  bf16x8 b;
#pragma unroll
  for (int i = 0; i < 8; ++i) b[i] = (__bf16)v[i];  // round to nearest even
  return __builtin_bit_cast(u32x4, b);
}

// ------------------------------------------------------------------ tile geometry

// A work-group tile of BM rows (the M side: X or Z rows) by BN columns (the N
// side: W columns).  Four waves in a WM x WN grid; each wave owns a
// (BM/WM) x (BN/WN) sub-tile made of 16x16 MFMA blocks.
//
// The MFMA is issued with the *weight* fragment as its A operand and the
// activation fragment as its B operand, so each lane ends up holding output
// row (lane % 16) and, for a pair of adjacent blocks, 8 consecutive output
// columns: the epilogue stores 16 contiguous bytes per lane.
template <int BM_, int BN_, int WM_, int WN_>
struct Tile {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_;
  static_assert(WM * WN == 4, "four waves");
  static constexpr int MW = BM / WM;  // rows per wave
  static constexpr int NW = BN / WN;  // columns per wave
  static constexpr int TM = MW / 16;
  static constexpr int TN = NW / 16;
  static_assert(TM >= 1 && TN >= 2 && TN % 2 == 0, "wave tile shape");
  static constexpr int A_STRIDE = kBK + 8;  // LDS row of the activation tile [BM][kBK], padded
  static constexpr int B_STRIDE = BN + 16;  // LDS row of the weight tile [kBK][BN], padded
  static constexpr int A_ELEMS = BM * A_STRIDE;
  static constexpr int B_ELEMS = kBK * B_STRIDE;
  static constexpr int A_CHUNKS = BM * kBK / 8 / kThreads;  // 16-byte loads per thread
  static constexpr int B_CHUNKS = kBK * BN / 8 / kThreads;
  static_assert(A_CHUNKS >= 1 && B_CHUNKS >= 1, "tile too small for 256 threads");
  template <int NB>
  static constexpr int stage_elems() { return A_ELEMS + NB * B_ELEMS; }
  template <int NB>
  static constexpr int lds_elems() { return 2 * stage_elems<NB>(); }
};

// ------------------------------------------------------------------ mainloop

struct NoWait {
  __device__ __forceinline__ void operator()(int) {}
};

// acc[b][tn][tm] += sum over k in [kbeg, kend) of W_b[k][n] * A[m][k] for the
// tile at (m0, n0).  A rows past `mlast` are clamped to `mlast` (their results
// are never stored).  `wait(k)` runs before the activation operand of the
// stage starting at k is loaded (after its weight loads were issued).
template <class T, int NB, class Wait>
__device__ __forceinline__ void mainloop(const uint16_t* __restrict__ A, long lda, int m0, int mlast,
                                         const uint16_t* const (&Bp)[NB], long ldb, int n0, int kbeg, int kend,
                                         f32x4 (&acc)[NB][T::TN][T::TM], uint16_t* lds, Wait& wait) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % T::WM;
  const int wn = wave / T::WM;

#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int i = 0; i < T::TN; ++i)
#pragma unroll
      for (int j = 0; j < T::TM; ++j) acc[b][i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = (kend - kbeg) / kBK;
  if (nk <= 0) return;

  // global -> register staging
  u32x4 ra[T::A_CHUNKS];
  u32x4 rb[NB][T::B_CHUNKS];
  const uint16_t* a_src[T::A_CHUNKS];
  int a_lds[T::A_CHUNKS];
#pragma unroll
  for (int i = 0; i < T::A_CHUNKS; ++i) {
    const int q = tid + kThreads * i;
    const int row = q >> 3, c8 = q & 7;
    int gr = m0 + row;
    gr = gr > mlast ? mlast : gr;
    a_src[i] = A + (long)gr * lda + c8 * 8;
    a_lds[i] = row * T::A_STRIDE + c8 * 8;
  }
  constexpr int BC = T::BN / 8;  // 16-byte chunks per weight row
  long b_off[T::B_CHUNKS];
  int b_lds[T::B_CHUNKS];
#pragma unroll
  for (int i = 0; i < T::B_CHUNKS; ++i) {
    const int q = tid + kThreads * i;
    const int row = q / BC, c8 = q % BC;
    b_off[i] = (long)row * ldb + n0 + c8 * 8;
    b_lds[i] = row * T::B_STRIDE + c8 * 8;
  }

  auto gload = [&](int k) {
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int i = 0; i < T::B_CHUNKS; ++i)
        rb[b][i] = *reinterpret_cast<const u32x4*>(Bp[b] + (long)k * ldb + b_off[i]);
    wait(k);
#pragma unroll
    for (int i = 0; i < T::A_CHUNKS; ++i) ra[i] = *reinterpret_cast<const u32x4*>(a_src[i] + k);
  };
  auto sstore = [&](int s) {
    uint16_t* base = lds + s * T::template stage_elems<NB>();
#pragma unroll
    for (int i = 0; i < T::A_CHUNKS; ++i) *reinterpret_cast<u32x4*>(base + a_lds[i]) = ra[i];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int i = 0; i < T::B_CHUNKS; ++i)
        *reinterpret_cast<u32x4*>(base + T::A_ELEMS + b * T::B_ELEMS + b_lds[i]) = rb[b][i];
  };

  // Fragment addressing inside a stage.
  //   activation (MFMA B operand): lane holds A[row = l%16][k = 8(l/16) .. +7]  -> ds_read_b128
  //   weight (MFMA A operand): ds_read_b64_tr_b16 over 4 rows x 4 chunks per 16-lane group;
  //     lane 4r+c of group g addresses row 8g+r (+4 for the upper half), columns 8c + 4*t2 .. +3,
  //     and receives column (8*(i/4) + 4*t2 + i%4) of those 4 rows, i = lane % 16.
  const int a_frag = (wm * T::MW + (lane & 15)) * T::A_STRIDE + 8 * (lane >> 4);
  const int g = lane >> 4, r4 = (lane & 15) >> 2, c4 = lane & 3;
  const int b_frag = (8 * g + r4) * T::B_STRIDE + wn * T::NW + 8 * c4;

  auto compute = [&](int s) {
    const uint16_t* base = lds + s * T::template stage_elems<NB>();
#pragma unroll
    for (int ks = 0; ks < kBK / 32; ++ks) {
      bf16x8 xf[T::TM];
#pragma unroll
      for (int tm = 0; tm < T::TM; ++tm)
        xf[tm] = *reinterpret_cast<const bf16x8*>(base + a_frag + tm * 16 * T::A_STRIDE + ks * 32);
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const uint16_t* bb = base + T::A_ELEMS + b * T::B_ELEMS + b_frag + ks * 32 * T::B_STRIDE;
#pragma unroll
        for (int tp = 0; tp < T::TN / 2; ++tp) {
#pragma unroll
          for (int t2 = 0; t2 < 2; ++t2) {
            const uint16_t* p = bb + tp * 32 + t2 * 4;
            bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(p));
            bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(p + 4 * T::B_STRIDE));
            bf16x8 wf = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
            for (int tm = 0; tm < T::TM; ++tm)
              acc[b][2 * tp + t2][tm] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf, xf[tm], acc[b][2 * tp + t2][tm], 0, 0, 0);
          }
        }
      }
    }
  };

  gload(kbeg);
  sstore(0);
  __syncthreads();
  for (int it = 0; it < nk; ++it) {
    const int s = it & 1;
    if (it + 1 < nk) gload(kbeg + (it + 1) * kBK);
    compute(s);
    if (it + 1 < nk) sstore(s ^ 1);
    __syncthreads();
  }
}

// ------------------------------------------------------------------ fragment <-> tile coordinates

// Output coordinates held by this lane for block pair tp and row block tm:
// row  = m0 + wm*MW + 16*tm + lane%16
// cols = n0 + wn*NW + 32*tp + 8*(lane/16) + [0..8)
template <class T>
struct FragPos {
  int row0, col0;
  __device__ FragPos(int m0, int n0) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    row0 = m0 + (wave % T::WM) * T::MW + (lane & 15);
    col0 = n0 + (wave / T::WM) * T::NW + 8 * (lane >> 4);
  }
};

template <class T>
__device__ __forceinline__ void pair_values(const f32x4 (&a)[T::TN][T::TM], int tp, int tm, float (&v)[8]) {
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    v[r] = a[2 * tp][tm][r];
    v[4 + r] = a[2 * tp + 1][tm][r];
  }
}

// ------------------------------------------------------------------ split-K partials
//
// Partials are stored fragment-native: for work item (tile, split s) each
// wave writes its accumulators as contiguous 1 KB runs (64 lanes x 16 bytes),
// so the writes and the reducer's reads are fully coalesced.  The reducer of a
// tile has the same lane <-> element mapping as every split.

template <class T, int NB>
struct Partial {
  static constexpr int PER_WAVE = NB * T::TN * T::TM;            // f32x4 per lane
  static constexpr long PER_ITEM = 4L * PER_WAVE * 64;            // f32x4 per (tile, split)
  __device__ static f32x4* at(float* base, long tile, int S, int s) {
    return reinterpret_cast<f32x4*>(base) + (tile * S + s) * PER_ITEM + (long)(threadIdx.x >> 6) * PER_WAVE * 64 +
           (threadIdx.x & 63);
  }
};

template <class T, int NB>
__device__ __forceinline__ void store_partial(float* base, long tile, int S, int s, const f32x4 (&acc)[NB][T::TN][T::TM]) {
  f32x4* p = Partial<T, NB>::at(base, tile, S, s);
  int i = 0;
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int tn = 0; tn < T::TN; ++tn)
#pragma unroll
      for (int tm = 0; tm < T::TM; ++tm, ++i) p[i * 64] = acc[b][tn][tm];
}

// acc = sum over s = 0 .. S-1 of partial s, in that order (fixed, so the result
// does not depend on which split arrived last).
template <class T, int NB>
__device__ __forceinline__ void reduce_partials(const float* base, long tile, int S, f32x4 (&acc)[NB][T::TN][T::TM]) {
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int tn = 0; tn < T::TN; ++tn)
#pragma unroll
      for (int tm = 0; tm < T::TM; ++tm) acc[b][tn][tm] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < S; ++s) {
    const f32x4* p = Partial<T, NB>::at(const_cast<float*>(base), tile, S, s);
    int i = 0;
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int tn = 0; tn < T::TN; ++tn)
#pragma unroll
        for (int tm = 0; tm < T::TM; ++tm, ++i) acc[b][tn][tm] += p[i * 64];
  }
}

// Split-K arrival: all waves' partial stores complete, then one lane bumps the
// tile's counter (acq_rel, agent scope).  Returns true in every thread of the
// work-group that arrived last; that work-group then owns the reduction.
// The counter advances by S per run and is never reset: the last arriver is
// the one whose previous value is epoch * S + S - 1 (unsigned, wrap-safe).
__device__ __forceinline__ bool arrive_last(uint32_t* cnt, uint32_t epoch, int S, int* s_flag) {
  wait_all_mem();
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t old = __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    *s_flag = (old - epoch * (uint32_t)S) == (uint32_t)(S - 1);
  }
  __syncthreads();
  const bool last = uniform(*s_flag) != 0;
  __syncthreads();  // s_flag may be rewritten by the next arrival
  if (last) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  return last;
}

// ------------------------------------------------------------------ ready flags

// Producer side: every wave's Z stores are complete, then one lane performs
// an agent-scope release increment of the tile's ready counter.
__device__ __forceinline__ void signal_ready(uint32_t* flag) {
  wait_all_mem();
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_add(flag, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

// Consumer side: before loading Z columns [k, k + kBK) of row block mb, wait
// until the GEMM1 tile (mb, k / bn1) has signalled in this run, i.e. until its
// counter reaches epoch + 1 (compared wrap-safe).  Each wave polls for itself
// (uniform address, one request per poll), sleeps between polls, gives up after
// spin_limit polls (latching CTRL_ERROR), then performs an agent-scope acquire.
struct ReadyWait {
  const uint32_t* ready;
  uint32_t* err;  // CTRL_ERROR word
  int mb, Mb, bn1;
  uint32_t target;
  uint32_t spin_limit;
  int known;  // highest column block already acquired by this wave
  __device__ __forceinline__ void operator()(int k) {
    const int kb = k / bn1;
    if (kb <= known) return;
    const uint32_t* f = ready + (long)kb * Mb + mb;
    // Once any wait of this run has given up, no wave waits again: the run
    // finishes promptly and the error is reported by the host.
    if ((int32_t)(uniform(ld_relaxed(f)) - target) < 0 && uniform(ld_relaxed(err)) == 0u) {
      for (uint32_t polls = 0;; ++polls) {
        if (polls >= spin_limit) {
          if ((threadIdx.x & 63) == 0) __hip_atomic_fetch_or(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          known = 0x7fffffff;
          return;
        }
        __builtin_amdgcn_s_sleep(2);
        if ((int32_t)(uniform(ld_relaxed(f)) - target) >= 0) break;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    known = kb;
  }
};

}  // namespace mlp2
