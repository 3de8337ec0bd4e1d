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

template <class A, class B>
struct is_same_type {
  static constexpr bool value = false;
};
template <class A>
struct is_same_type<A, A> {
  static constexpr bool value = true;
};
template <bool V>
struct bool_constant {
  static constexpr bool value = V;
};

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4_t;

constexpr int kBK = 64;        // K granularity of the plans (split-K ranges); a plan whose tiles take
                               // 128-deep stages keeps its K ranges multiples of 128

// Words per 128-byte line.  Every counter that work-groups update with device-
// scope atomics sits on a line of its own: such atomics are performed at the
// memory side of the device, one at a time per line, so counters sharing a
// line would queue behind each other's traffic.
constexpr int kLine = 32;

// Control words of a plan (device memory, zero at plan creation), one per line.
enum {
  CTRL_EPOCH = 0,                  // runs completed; read at kernel start, bumped by the run's last work-group
  CTRL_ERROR = 1 * kLine,          // nonzero once a bounded flag wait gave up
  CTRL_DONE_ALL = 2 * kLine,       // claim lists of the current kernel whose work-groups have all finished
  CTRL_TICKET = 3 * kLine,         // CTRL_TICKET + l * kLine: next ticket of claim list l (up to 16 lists:
                                   // 8 per role when the pipelined launch splits the grid into roles)
  CTRL_DONE = 19 * kLine,          // CTRL_DONE + l * kLine: finished work-groups of claim list l
  CTRL_QHEAD = 35 * kLine,         // workqueue mode: next queue slot a consumer claims
  CTRL_QTAIL = 36 * kLine,         // workqueue mode: next queue slot a producer fills
  CTRL_EPOCH_WQ = 37 * kLine,      // workqueue runs completed (the scoreboards advance in those only)
  CTRL_EPOCH_SN = 38 * kLine,      // sentinel runs completed (their parity picks the intermediate buffer)
  CTRL_WORDS = 39 * kLine
};
__device__ __forceinline__ int ctrl_ticket(int l) { return CTRL_TICKET + l * kLine; }
__device__ __forceinline__ int ctrl_done(int l) { return CTRL_DONE + l * kLine; }

enum { ACT_IDENTITY = 0, ACT_GELU_TANH = 1, ACT_SWIGLU = 2 };

struct Args {
  const uint16_t* X;   // [M, H]
  const uint16_t* W1;  // [H, F]  (SwiGLU: [2, H, F])
  const uint16_t* W2;  // [F, H]
  uint16_t* Y;         // [M, H]
  uint16_t* Z;         // [Mpad, F]
  uint16_t* Zs;        // sentinel mode: two intermediates of [Mpad, F] each, zs_elems apart; sentinel runs
                       // alternate between them (the other one is refilled with sentinels meanwhile)
  long zs_elems;
  uint16_t* Zr;        // inside a sentinel run: the intermediate the next sentinel run uses (refilled with
                       // sentinels tile by tile); null otherwise
  float* part1;        // GEMM1 split-K partials (fragment-native), or null
  float* part2;        // GEMM2 split-K partials, or null
  uint32_t* cnt1;      // split-K arrival counters of GEMM1: tile t at word t * kLine
  uint32_t* cnt2;      // split-K arrival counters of GEMM2: tile t at word t * kLine
  uint32_t* ready;     // ready counters: tile (mb, nb1) at word (nb1 * Mb + mb) * kLine
  uint32_t* board;     // workqueue mode: scoreboard of GEMM2 unit q at word q * kLine
  uint32_t* queue;     // workqueue mode: ring of ready GEMM2 units, items2 + 1 slots (one per unit and
                       // run, and a spare)
  uint32_t* ctrl;      // CTRL_* words
  const uint32_t* order1;  // GEMM1 item per rank of the GEMM1 kernel, length items1
  const uint32_t* order2;  // GEMM2 item per rank of the GEMM2 kernel, length items2 + items_red
                           // (bit 30 set: reduction item)
  const uint32_t* orderp;  // item per rank of the pipelined kernel, length items1 + items2 + items_red
                           // (bit 31 set: GEMM2 item, bits 31 and 30: reduction item; else GEMM1 item id)
  int M, H, F, act;
  int Mb, Nb1, Nb2;        // row blocks; GEMM1 / GEMM2 column blocks
  int S1, S2;              // split-K factors
  int kc1, kc2;            // K per split (multiples of kBK)
  int items1, items2;      // GEMM1 / GEMM2 work items (tiles x split-K parts)
  int bn1;                 // GEMM1 column-block width (ready-counter granularity along GEMM2's K)
  uint32_t spin_limit;
  int drop_signal;         // GEMM1 tile whose signal is skipped (failure injection), -1 = none
  uint64_t* trace;         // per-work-group timing records (trace builds only), or null
  int trace_cap;           // records per work-group
  int trace_groups;        // work-groups per trace section (the largest grid of the plan)
  int lists;               // claim lists of the launch (1 or 8; work-group g claims from list g % lists)
  int first_static;        // work-groups g < first_static take rank g as their first item without a
                           // ticket (ranks below it are items that never wait); the others claim
  int p1;                  // pipelined launch: 0 = shared roles; else work-groups with g % 64 < p1 take
                           // GEMM1 items only (from order1) and the others GEMM2 items only (order2)
  int lists2;              // claim lists of the GEMM2 role (role split only; `lists` is the GEMM1 role's)
  int red2;                // GEMM2 split-K: 0 = the part that arrives last sums the tile; else the tile is
                           // summed by red2 reduction items (slices of its units), ranked after every GEMM2 item
  int items_red;           // reduction items of the launch (tiles2 * red2, or 0)
};

// ------------------------------------------------------------------ optional timing trace
//
// Built with -DMLP2_TRACE, thread 0 of every work-group records per item:
// {rank, start, mainloop end, split-K arrival released, siblings arrived, end,
// ring-wait ticks, flag-wait ticks} on the 100 MHz real-time counter.  Ring waits are the mainloop's waits for its own
// loads plus the stage barrier; flag waits are ready-counter and sibling waits.
// Without the macro every hook compiles to nothing.
#ifdef MLP2_TRACE
constexpr bool kTrace = true;
#else
constexpr bool kTrace = false;
#endif
constexpr int kTraceWords = 8;

struct TraceAcc {
  uint64_t ring = 0, flag = 0, t_main = 0, t_rel = 0, t_wait = 0;
  uint64_t c_start = 0;  // shader-clock counter at the item's start
};

__device__ __forceinline__ uint64_t trace_now() {
  if constexpr (kTrace) return __builtin_amdgcn_s_memrealtime();
  return 0;
}

// Shader-clock counter (core clock cycles): beside the real-time counter it
// gives the clock an item ran at.
__device__ __forceinline__ uint64_t trace_clock() {
  if constexpr (kTrace) return __builtin_amdgcn_s_memtime();
  return 0;
}

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
// side: W columns), staged through an NS-deep ring of LDS buffers of kBK rows
// of K each.  Four or eight 64-wide waves in a WM x WN grid; each wave owns a
// (BM/WM) x (BN/WN) sub-tile made of 16x16 MFMA blocks.  Eight waves let a
// large tile (256 x 256: a quarter of the operand bytes per flop of 128 x 128)
// keep two waves per SIMD, so that one wave's LDS reads overlap the other's
// products.
//
// The MFMA is issued with the *weight* fragment as its A operand and the
// activation fragment as its B operand, so each lane ends up holding output
// row (lane % 16) and, for a pair of adjacent blocks, 8 consecutive output
// columns: the epilogue stores 16 contiguous bytes per lane.
//
// LDS stage layout (bytes), both parts unpadded and XOR-swizzled in 16-byte
// chunks, because the direct-to-LDS loads write each wave's 1 KB contiguously
// (lane i -> bytes 16 i):
//   activation tile [BM][BK] bf16, rows of BK * 2 bytes, XOR-swizzled per
//     chunk (swz_a) so that the 16 rows read by one ds_read_b128 group land
//     in 16 distinct 4-bank groups;
//   weight tile [BK][BN] bf16 per operand: chunk c of row k at c ^ swzB(k),
//     which puts the 4 rows read by one ds_read_b64_tr_b16 group in
//     different banks.
template <int BM_, int BN_, int WM_, int WN_, int NS_, int BK_ = kBK, bool WNT_ = false>
struct Tile {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, NS = NS_;
  // Weight loads with the non-temporal hint (plans whose weights exceed the
  // last-level cache): the streamed weights then stop displacing the lines
  // that the activation loads reuse.
  static constexpr bool WNT = WNT_;
  // K depth of one stage: 64; 32 (half the bytes per stage, so a ring of the
  // same LDS holds twice the stages); or 128 (twice the products per stage
  // for the same per-stage costs: the wait, the barrier, the DMA issue and
  // the first fragment reads, which a small tile with one wave per SIMD pays
  // in series).  The activation tile's rows are BK * 2 bytes.
  static constexpr int BK = BK_;
  static_assert(BK == 128 || BK == 64 || BK == 32, "stage depth");
  static constexpr int ROW_BYTES = BK * 2;      // activation tile row pitch in LDS
  static constexpr int CHUNKS = BK / 8;         // 16-byte chunks per activation row
  static constexpr int NWAVES = WM * WN;
  static constexpr int THREADS = 64 * NWAVES;
  static_assert(NWAVES == 4 || NWAVES == 8, "four or eight waves");
  static_assert(BN == 64 || BN == 128 || BN == 256, "weight tile width");
  static_assert(NS >= 2, "at least double buffered");
  static constexpr int MW = BM / WM;  // rows per wave
  static constexpr int NW = BN / WN;  // columns per wave
  static constexpr int TM = MW / 16;
  static constexpr int TN = NW / 16;
  static_assert(TM >= 1 && TN >= 2 && TN % 2 == 0, "wave tile shape");
  static constexpr int A_BYTES = BM * BK * 2;
  static constexpr int B_BYTES = BK * BN * 2;
  static constexpr int A_DMA = A_BYTES / 1024 / NWAVES;  // 1 KB wave loads per wave and stage
  static constexpr int B_DMA = B_BYTES / 1024 / NWAVES;
  static_assert(A_DMA >= 1 && B_DMA >= 1 && A_BYTES % (1024 * NWAVES) == 0 && B_BYTES % (1024 * NWAVES) == 0,
                "every wave loads whole 1 KB pieces of both operands");
  template <int NB>
  static constexpr int stage_bytes() { return A_BYTES + NB * B_BYTES; }
  template <int NB>
  static constexpr int lds_bytes() { return NS * stage_bytes<NB>(); }
  template <int NB>
  static constexpr int dma_per_stage() { return A_DMA + NB * B_DMA; }
};

// Activation tile swizzle: 256-byte rows (BK = 128), one to a bank period,
// put chunk c of row r at c ^ (r & 15); 128-byte rows (BK = 64) at
// c ^ ((r >> 1) & 7); 64-byte rows (BK = 32), four to a bank period, at
// c ^ ((r >> 2) & 3).  Either way the 16 rows one ds_read_b128 group reads
// land in 16 distinct 4-bank groups.
template <int BK = kBK>
__device__ __forceinline__ int swz_a(int row) {
  return BK == 128 ? row & 15 : BK == 64 ? (row >> 1) & 7 : (row >> 2) & 3;
}
template <int BN>
__device__ __forceinline__ int swz_b(int k) {
  return BN >= 128 ? 4 * (k & 3) : 4 * ((k >> 1) & 1);
}

// One 16-byte-per-lane direct-to-LDS load: lane i reads 16 bytes at
// base + voff and writes them to LDS at lds_addr + 16 i.  Issued through
// inline assembly so that the compiler does not serialise every LDS read
// behind it (it cannot tell the ring's stages apart); completion is tracked
// explicitly with s_waitcnt vmcnt.  M0 carries the LDS address: it is an
// operand of the asm ("{m0}" constraint), so the compiler itself writes it and
// knows the register holds that value, and never has a value of its own there.
__device__ __forceinline__ void dma16(const void* base, uint32_t voff, uint32_t lds_addr) {
  asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(base), "{m0}"(lds_addr) : "memory");
}

// The same load at device scope (sc1, the scope bit of the compiler's own
// agent-scope atomic loads): it reads the device's point of coherence rather
// than a line the consumer's XCD L2 may hold.  The sentinel mode's consumers
// read the intermediate this way, since no release and acquire order it.
// The same load with the non-temporal hint (a streamed operand read once).
__device__ __forceinline__ void dma16_nt(const void* base, uint32_t voff, uint32_t lds_addr) {
  asm volatile("global_load_lds_dwordx4 %0, %1 nt" ::"v"(voff), "s"(base), "{m0}"(lds_addr) : "memory");
}

__device__ __forceinline__ void dma16_coherent(const void* base, uint32_t voff, uint32_t lds_addr) {
  asm volatile("global_load_lds_dwordx4 %0, %1 sc1" ::"v"(voff), "s"(base), "{m0}"(lds_addr) : "memory");
}

// ------------------------------------------------------------------ sentinel synchronisation
//
// Sec. V-A of the paper: instead of a fence and a flag per tile, the
// intermediate buffer holds a sentinel value before its producer writes it,
// and the consumer re-reads until no sentinel is left.  The sentinel is the
// bf16 pattern 0xFFFF (a NaN with every payload bit set).  The GEMM1 epilogue
// never writes it (canonicalize_z turns it into the canonical NaN 0x7FC0, in
// every mode, so the modes stay bit-identical), so an element still holding
// 0xFFFF has not been written yet; the check is per element, so a load that
// sees part of a 16-byte piece before the rest was written is caught too.
constexpr uint16_t kSentinel = 0xFFFF;

__device__ __forceinline__ bool has_sentinel(u32x4 v) {
  bool any = false;
#pragma unroll
  for (int i = 0; i < 4; ++i) any |= (v[i] & 0xFFFFu) == 0xFFFFu || (v[i] >> 16) == 0xFFFFu;
  return any;
}

__device__ __forceinline__ u32x4 canonicalize_z(u32x4 v) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if ((v[i] & 0xFFFFu) == 0xFFFFu) v[i] = (v[i] & 0xFFFF0000u) | 0x7FC0u;
    if ((v[i] >> 16) == 0xFFFFu) v[i] = (v[i] & 0xFFFFu) | 0x7FC00000u;
  }
  return v;
}

// A 16-byte piece of the intermediate stored at device scope without any
// fence: two 8-byte agent-scope relaxed atomic stores (each single-copy atomic).
__device__ __forceinline__ void store_coherent16(uint16_t* p, u32x4 v) {
  uint64_t* q = reinterpret_cast<uint64_t*>(p);
  __hip_atomic_store(q, (uint64_t)v[0] | ((uint64_t)v[1] << 32), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(q + 1, (uint64_t)v[2] | ((uint64_t)v[3] << 32), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Wait until at most n of this wave's vector-memory operations are outstanding.
template <int N>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait until this wave's loads of the current stage are complete while the
// `after` (<= A) stages issued behind it stay in flight.  `after` is uniform.
template <int PER, int A>
__device__ __forceinline__ void wait_stages_behind(int after) {
  if constexpr (A <= 0) {
    wait_vm<0>();
  } else {
    static_assert(A * PER <= 63, "vmcnt holds at most 63 outstanding loads");
    if (after >= A) wait_vm<A * PER>();
    else wait_stages_behind<PER, A - 1>(after);
  }
}

// ------------------------------------------------------------------ mainloop

// acc[b][tn][tm] = sum over k in [kbeg, kend) of W_b[k][n] * A[m][k] for the
// tile at (m0, n0).  A rows past `mlast` are clamped to `mlast` (their results
// are never stored).  `wait(k)` runs, in every wave, before the activation
// operand of the stage starting at k is requested (after its weight loads).
//
// Pipeline: stages k0, k0 + BK, ... are loaded NS - 1 ahead of use.  At
// iteration it a wave waits for its own loads of stage it, a barrier makes
// every wave's loads of stage it visible and retires every wave's reads of
// stage it - 1, then the loads of stage it + NS - 1 go into that freed buffer
// and stage it is multiplied.  Four-wave tiles with three or more stages read
// one stage ahead into registers instead (below), and keep NS stages loading.
// A stage check that does nothing (every mode but the sentinel mode).
struct NoCheck {
  static constexpr bool kCoherentA = false;
  template <class... X>
  __device__ __forceinline__ void operator()(X...) {}
};

template <class T, int NB, class Wait, class Check = NoCheck>
__device__ __forceinline__ void mainloop(const uint16_t* __restrict__ A, long lda, int m0, int mlast,
                                         const uint16_t* const (&Bp)[NB], long ldb, int n0, int kbeg, int kend,
                                         f32x4 (&acc)[NB][T::TN][T::TM], char* lds, Wait& wait, TraceAcc& tr,
                                         Check check = Check()) {
  // The thread index passes through an empty asm, so the compiler derives
  // this call's per-lane offsets here instead of hoisting them out of the
  // persistent item loop: in the pipelined kernel, whose items take one of
  // two tile shapes, hoisted offsets of both shapes would stay live across
  // the whole kernel and push the mainloop's accumulators out of registers.
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid));
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

  const int nk = (kend - kbeg) / T::BK;
  if (nk <= 0) return;

  const uint32_t lds_base = (uint32_t)(uintptr_t)lds;
  constexpr int SB = T::template stage_bytes<NB>();
  constexpr int PER_STAGE = T::template dma_per_stage<NB>();

  // DMA source offsets (bytes, relative to the tensor bases) at k = 0.
  uint32_t a_off[T::A_DMA];
#pragma unroll
  for (int j = 0; j < T::A_DMA; ++j) {
    const int ch = wave + T::NWAVES * j;  // 1 KB chunk = 8 rows of 128 B (4 of 256 B, 16 of 64 B)
    const int row = (1024 / T::ROW_BYTES) * ch + lane / T::CHUNKS;
    const int lc = (lane % T::CHUNKS) ^ swz_a<T::BK>(row);
    int gr = m0 + row;
    gr = gr > mlast ? mlast : gr;
    a_off[j] = (uint32_t)(((long)gr * lda + 8 * lc) * 2);
  }
  constexpr int CPR = T::BN / 8;      // 16-byte chunks per weight row
  constexpr int RPC = 64 / CPR;       // weight rows per 1 KB chunk
  uint32_t b_off[T::B_DMA];
#pragma unroll
  for (int j = 0; j < T::B_DMA; ++j) {
    const int ch = wave + T::NWAVES * j;
    const int row = RPC * ch + lane / CPR;
    const int lc = (lane % CPR) ^ swz_b<T::BN>(row);
    b_off[j] = (uint32_t)(((long)row * ldb + n0 + 8 * lc) * 2);
  }

  // A stage's loads: the activation rows first (measured on the gated GEMM1
  // operand stream without math, 256 activation rows and two 128-column
  // weight stripes per stage: 216 -> 202 us), except while a GEMM2 item may
  // still have to wait for its activation rows: then the weights first, so
  // they stream during the wait.  The order is fixed per loop, not chosen
  // per stage: in the plain stage loop (every tile but the four-wave tiles
  // with three or more stages, below) an item that waits runs its stages
  // in the weights-first loop until its wait has seen every producer of its K
  // range complete, then in the activation-first loop (gated 396 -> 388 us,
  // prefill 440 -> 421 us pipelined; a choice per stage inside one loop made
  // the one-launch kernels much slower: decode 74 -> 113 us).
  auto issue = [&](int st, auto weights_first) {
    const int k = kbeg + st * T::BK;
    const uint32_t sbase = lds_base + (uint32_t)((st % T::NS) * SB);
    auto weights = [&]() {
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int j = 0; j < T::B_DMA; ++j) {
          const uint32_t dst = uniform(sbase + (uint32_t)(T::A_BYTES + b * T::B_BYTES + (wave + T::NWAVES * j) * 1024));
          if constexpr (T::WNT)
            dma16_nt(Bp[b], b_off[j] + (uint32_t)((long)k * ldb * 2), dst);
          else
            dma16(Bp[b], b_off[j] + (uint32_t)((long)k * ldb * 2), dst);
        }
    };
    auto activations = [&]() {
#pragma unroll
      for (int j = 0; j < T::A_DMA; ++j) {
        if constexpr (Check::kCoherentA)
          dma16_coherent(A, a_off[j] + (uint32_t)(k * 2), uniform(sbase + (uint32_t)((wave + T::NWAVES * j) * 1024)));
        else
          dma16(A, a_off[j] + (uint32_t)(k * 2), uniform(sbase + (uint32_t)((wave + T::NWAVES * j) * 1024)));
      }
    };
    if constexpr (decltype(weights_first)::value) {
      weights();
      wait(k);  // covers the stage's columns [k, k + BK)
      activations();
    } else {
      activations();
      wait(k);  // returns at once (takes the next ticket at the last stage)
      weights();
    }
  };
  using WaitFirst = bool_constant<Wait::kBlocks>;  // weights first where the item may wait
  using ActFirst = bool_constant<false>;

  // Fragment addressing (bytes inside a stage).
  //   activation (MFMA B operand): lane holds A[row = l%16][k = 8(l/16) .. +7]  -> ds_read_b128
  //   weight (MFMA A operand): ds_read_b64_tr_b16 over 4 rows x 4 chunks per 16-lane group;
  //     lane 4r+c of group g addresses row 8g+r (+4 for the upper half), columns 8c + 4*t2 .. +3,
  //     and receives column (8*(i/4) + 4*t2 + i%4) of those 4 rows, i = lane % 16.
  const int arow = wm * T::MW + (lane & 15);
  int a_frag[T::BK / 32];  // K half ks: chunk 4 ks + lane / 16 of the row
#pragma unroll
  for (int ks = 0; ks < T::BK / 32; ++ks)
    a_frag[ks] = arow * T::ROW_BYTES + (((4 * ks + (lane >> 4)) ^ swz_a<T::BK>(arow)) << 4);
  const int g = lane >> 4, r4 = (lane & 15) >> 2, c4 = lane & 3;
  const int brow = 8 * g + r4;
  int b_frag[T::TN / 2];
#pragma unroll
  for (int tp = 0; tp < T::TN / 2; ++tp) {
    const int q = ((wn * T::NW + 32 * tp) >> 3) + c4;
    b_frag[tp] = T::A_BYTES + brow * (2 * T::BN) + ((q ^ swz_b<T::BN>(brow)) << 4);
  }

  // K slices of 32 per stage (BK / 32 of them).  With a two-stage ring every fragment of
  // the stage is read before its first product: the reads of the second
  // half and of the later column pairs then overlap the first products in
  // whatever code the mainloop is inlined into (the one-launch kernels' item
  // loop otherwise schedules one read pair ahead of its four products).
  // Deeper rings keep each half's reads next to its products.  Both orders
  // accumulate every output in the same sequence (first half, then second).
  auto weight_frag = [&](const char* base, int ks, int b, int i) {
    const char* p = base + b * T::B_BYTES + b_frag[i / 2] + ks * 32 * (2 * T::BN) + (i % 2) * 8;
    bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(p));
    bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(p + 4 * (2 * T::BN)));
    return (bf16x8)__builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  };
  auto act_frag = [&](const char* base, int ks, int tm) {
    return *reinterpret_cast<const bf16x8*>(base + a_frag[ks] + tm * 16 * T::ROW_BYTES);
  };
  auto compute = [&](int st) {
    const char* base = lds + (st % T::NS) * SB;
    if constexpr (T::NS == 2) {
      bf16x8 xf[T::BK / 32][T::TM];
      bf16x8 wf[T::BK / 32][NB][T::TN];
#pragma unroll
      for (int ks = 0; ks < T::BK / 32; ++ks) {
#pragma unroll
        for (int tm = 0; tm < T::TM; ++tm) xf[ks][tm] = act_frag(base, ks, tm);
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
          for (int i = 0; i < T::TN; ++i) wf[ks][b][i] = weight_frag(base, ks, b, i);
      }
#pragma unroll
      for (int ks = 0; ks < T::BK / 32; ++ks)
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
          for (int i = 0; i < T::TN; ++i)
#pragma unroll
            for (int tm = 0; tm < T::TM; ++tm)
              acc[b][i][tm] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[ks][b][i], xf[ks][tm], acc[b][i][tm], 0, 0, 0);
    } else {
#pragma unroll
      for (int ks = 0; ks < T::BK / 32; ++ks) {
        bf16x8 xf[T::TM];
#pragma unroll
        for (int tm = 0; tm < T::TM; ++tm) xf[tm] = act_frag(base, ks, tm);
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
          for (int i = 0; i < T::TN; ++i) {
            const bf16x8 wf = weight_frag(base, ks, b, i);
#pragma unroll
            for (int tm = 0; tm < T::TM; ++tm)
              acc[b][i][tm] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf, xf[tm], acc[b][i][tm], 0, 0, 0);
          }
      }
    }
  };

  // Own loads of stage st complete (the stages issued after it may stay in
  // flight), then every wave's: the barrier also retires every wave's reads
  // of the stages before st.
  auto resident = [&](int st) {
    const uint64_t t0 = trace_now();
    wait_stages_behind<PER_STAGE, T::NS - 2>(min(T::NS - 2, nk - 1 - st));
    if constexpr (!is_same_type<Check, NoCheck>::value) {
      // The stage's activation pieces this wave loaded are in LDS: check them
      // (and reload any piece that still holds a sentinel) before the barrier
      // hands the stage to the other waves.
      const int k = kbeg + st * T::BK;
      const uint32_t sbase = lds_base + (uint32_t)((st % T::NS) * SB);
      check.template operator()<T>(A, a_off, k, sbase, lds + (st % T::NS) * SB, wave, lane);
    }
    __syncthreads();
    if constexpr (kTrace) tr.ring += trace_now() - t0;
  };

  // Prologue: NS - 1 stages in flight.
#pragma unroll
  for (int st = 0; st < T::NS - 1; ++st)
    if (st < nk) issue(st, WaitFirst());

  if constexpr (T::NWAVES == 4 && T::NS >= 3) {
    // One wave per SIMD: nothing else on the SIMD hides a stage's LDS read
    // latency, so the fragments of stage it + 1 are read into a second set
    // of registers while stage it is multiplied.  Stage it's slot is free
    // once every wave holds its fragments (the barrier of stage it + 1), and
    // takes the loads of stage it + NS.  Same products in the same order.
    struct Frags {
      bf16x8 x[T::BK / 32][T::TM];
      bf16x8 w[T::BK / 32][NB][T::TN];
    };
    auto read = [&](Frags& f, int st) {
      const char* base = lds + (st % T::NS) * SB;
#pragma unroll
      for (int ks = 0; ks < T::BK / 32; ++ks) {
#pragma unroll
        for (int tm = 0; tm < T::TM; ++tm) f.x[ks][tm] = act_frag(base, ks, tm);
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
          for (int i = 0; i < T::TN; ++i) f.w[ks][b][i] = weight_frag(base, ks, b, i);
      }
    };
    auto mma = [&](const Frags& f) {
#pragma unroll
      for (int ks = 0; ks < T::BK / 32; ++ks)
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
          for (int i = 0; i < T::TN; ++i)
#pragma unroll
            for (int tm = 0; tm < T::TM; ++tm)
              acc[b][i][tm] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.w[ks][b][i], f.x[ks][tm], acc[b][i][tm], 0, 0, 0);
    };
    // Stage it is multiplied while stage it + 1 (< nk) is read.
    auto advance = [&](int it, Frags& cur, Frags& nxt, auto order) {
      resident(it + 1);
      if (it + T::NS < nk) issue(it + T::NS, order);
      read(nxt, it + 1);
      mma(cur);
    };
    resident(0);
    if (T::NS - 1 < nk) issue(T::NS - 1, WaitFirst());
    Frags fa, fb;
    read(fa, 0);
    // Two stages per trip, the fragment sets swapping roles; every trip reads
    // a next stage, so both sets keep their registers (no conditional read
    // merges into the products' control flow).
    // (One loop: a waiting item keeps the weights-first order throughout; a
    // second, activation-first loop after the item's producers were all seen
    // complete made these kernels slower: decode 76 -> 88 us.)
    int it = 0;
    for (; it + 2 < nk; it += 2) {
      advance(it, fa, fb, WaitFirst());
      advance(it + 1, fb, fa, WaitFirst());
    }
    if (it + 1 < nk) {  // two stages left
      advance(it, fa, fb, WaitFirst());
      mma(fb);
    } else {            // one stage left
      mma(fa);
    }
    __syncthreads();  // every wave is done reading the ring before it is reused
    return;
  }

  int it = 0;
  if constexpr (Wait::kBlocks) {
    for (; it < nk && !wait.all_known(); ++it) {
      resident(it);
      if (it + T::NS - 1 < nk) issue(it + T::NS - 1, WaitFirst());
      compute(it);
    }
  }
  for (; it < nk; ++it) {
    resident(it);
    if (it + T::NS - 1 < nk) issue(it + T::NS - 1, ActFirst());
    compute(it);
  }
  __syncthreads();  // every wave is done reading the ring before it is reused
}

// The sentinel mode's stage check (the consumer side of Sec. V-A): each wave
// reads back the activation pieces it loaded for the stage (16 bytes per lane
// per 1 KB piece), and reloads a piece, at device scope, while any lane still
// sees a sentinel element in it, sleeping between tries.  After spin_limit
// tries, or once another wait gave up, it latches CTRL_ERROR (bit 2) and
// stops; the kernel still exits and mlp2_check reports the timeout.
struct SentinelCheck {
  static constexpr bool kCoherentA = true;
  uint32_t* err;  // CTRL_ERROR word
  uint32_t spin_limit;
  TraceAcc* tr;   // re-read time is counted as flag-wait time (trace builds)
  template <class T>
  __device__ __forceinline__ void operator()(const uint16_t* A, const uint32_t (&a_off)[T::A_DMA], int k,
                                             uint32_t sbase, const char* stage, int wave, int lane) {
#pragma unroll
    for (int j = 0; j < T::A_DMA; ++j) {
      const int piece = (wave + T::NWAVES * j) * 1024;
      const uint64_t t0 = trace_now();
      for (uint32_t tries = 0;; ++tries) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(stage + piece + 16 * lane);
        if (__builtin_amdgcn_ballot_w64(has_sentinel(v)) == 0) {  // the same in every lane
          if constexpr (kTrace) {
            if (tries) tr->flag += trace_now() - t0;
          }
          break;
        }
        if (tries >= spin_limit || ((tries & 63u) == 63u && uniform(ld_relaxed(err)) != 0u)) {
          if (lane == 0) __hip_atomic_fetch_or(err, 4u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          break;
        }
        __builtin_amdgcn_s_sleep(2);
        dma16_coherent(A, a_off[j] + (uint32_t)(k * 2), uniform(sbase + (uint32_t)piece));
        wait_vm<0>();
      }
    }
  }
};

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
// With split-K, a tile's K range is cut into S parts computed by separate
// work items.  Each part stores its fp32 accumulators "fragment-native": lane
// l of wave w writes its f32x4 of block i at ((tile*S + s)*PER_ITEM +
// (w*PER_WAVE + i)*64 + l), so writes and reads are fully coalesced 1 KB runs.
// Each part then counts its arrival on the tile's counter; the part that
// arrives last (it reads the count just below the run's target) adds up the
// tile in "units" (a wave's pair of adjacent 16x16 blocks in one row block,
// for every weight operand) in the fixed order s = 0, 1, ..., S-1 and runs the
// tile's epilogue; the other parts go straight on to their next item.  No part
// ever waits for a sibling, and the order of the adds never depends on which
// part finished last, so every run and mode gives the same bits.

template <class T, int NB>
struct Partial {
  static constexpr int PER_WAVE = NB * T::TN * T::TM;  // f32x4 per lane
  static constexpr long PER_ITEM = (long)T::NWAVES * PER_WAVE * 64;  // f32x4 per (tile, split)
  static constexpr int UNITS = T::NWAVES * T::TM * (T::TN / 2); // (wave, tm, tp) triples per tile
  __device__ static long block_index(long tile, int S, int s, int w, int b, int tn, int tm) {
    return (tile * S + s) * PER_ITEM + ((long)w * PER_WAVE + ((b * T::TN + tn) * T::TM + tm)) * 64;
  }
};

template <class T, int NB>
__device__ __forceinline__ void store_partial(float* base, long tile, int S, int s, const f32x4 (&acc)[NB][T::TN][T::TM]) {
  f32x4* p = reinterpret_cast<f32x4*>(base) + Partial<T, NB>::block_index(tile, S, s, threadIdx.x >> 6, 0, 0, 0) +
             (threadIdx.x & 63);
  int i = 0;
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int tn = 0; tn < T::TN; ++tn)
#pragma unroll
      for (int tm = 0; tm < T::TM; ++tm, ++i) p[i * 64] = acc[b][tn][tm];
}

// A reduction unit: wave w's blocks (2 tp, tm) and (2 tp + 1, tm).
template <class T>
struct Unit {
  int w, tm, tp;
  __device__ Unit() = default;
  __device__ explicit Unit(int u) {
    constexpr int per_wave = T::TM * (T::TN / 2);
    w = u / per_wave;
    const int r = u - w * per_wave;
    tm = r / (T::TN / 2);
    tp = r - tm * (T::TN / 2);
  }
  // Output row and first of the 8 consecutive columns held by `lane` of this unit.
  __device__ int row(int m0, int lane) const { return m0 + (w % T::WM) * T::MW + 16 * tm + (lane & 15); }
  __device__ int col(int n0, int lane) const { return n0 + (w / T::WM) * T::NW + 32 * tp + 8 * (lane >> 4); }
};

// v[g][b][0..7] = sum over s = 0 .. S-1 (in that order) of the 8 values of
// unit ug[g] for weight operand b, as held by `lane` (the layout pair_values
// produces).  G units at a time and R parts per round keep 2*G*NB*R loads of
// one wave in flight together; slots past the last part load part S - 1
// again (in bounds) and are not added.
template <class T, int NB, int G>
__device__ __forceinline__ void reduce_units(const float* base, long tile, int S, const Unit<T> (&ug)[G], int lane,
                                             float (&v)[G][NB][8]) {
  const f32x4* p = reinterpret_cast<const f32x4*>(base);
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int i = 0; i < 8; ++i) v[g][b][i] = 0.f;
  constexpr int R = 8;
  for (int s = 0; s < S; s += R) {
    f32x4 q[R][G][NB][2];
#pragma unroll
    for (int h = 0; h < R; ++h) {
      const int sh = min(s + h, S - 1);
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
          for (int t2 = 0; t2 < 2; ++t2)
            q[h][g][b][t2] = p[Partial<T, NB>::block_index(tile, S, sh, ug[g].w, b, 2 * ug[g].tp + t2, ug[g].tm) + lane];
    }
#pragma unroll
    for (int h = 0; h < R; ++h) {
      if (s + h >= S) break;  // uniform
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            v[g][b][r] += q[h][g][b][0][r];
            v[g][b][4 + r] += q[h][g][b][1][r];
          }
    }
  }
}

// Release-increment of a counter after every wave's stores are complete
// (used for split-K arrivals and for the producer's ready signal).
__device__ __forceinline__ void release_add(uint32_t* cnt) {
  wait_all_mem();
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

// A split-K part's arrival: store the partial, then one agent-scope release
// increment of the tile's counter (after every wave's stores are complete).
// Returns true (uniformly) on the part that arrives last in this run, i.e.
// that reads `target - 1`; that part then reads the others' partials after a
// barrier and a work-group-scope acquire.  No agent-scope acquire is needed,
// for the reason given for Z with the ready waits below: each tile's
// partials (whole 1 KB runs, never sharing a line with another tile's) are
// read once per launch, only by the completing part, after every part has
// released them.
template <class T, int NB>
__device__ __forceinline__ bool arrive_split(float* part, uint32_t* cnt, long tile, int S, int s, uint32_t target,
                                             const f32x4 (&acc)[NB][T::TN][T::TM], int* s_slot, TraceAcc& tr) {
  store_partial<T, NB>(part, tile, S, s, acc);
  wait_all_mem();
  __syncthreads();
  if constexpr (kTrace) tr.t_rel = trace_now();
  if (threadIdx.x == 0) {
    const uint32_t old = __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    *s_slot = old == target - 1u;
  }
  __syncthreads();
  const bool last = uniform(*s_slot) != 0;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  __syncthreads();  // *s_slot may be rewritten
  if constexpr (kTrace) tr.t_wait = trace_now();
  return last;
}

// ------------------------------------------------------------------ claiming items

// The next item of a persistent work-group.  Claim list l = blockIdx % lists
// hands out the ranks l, l + lists, l + 2 lists, ... in increasing order: the
// first `skip` of them without a ticket (first items of the list's
// work-groups below Args::first_static), the rest through the list's ticket
// word.  Taking a ticket is a device-scope
// atomic whose result comes back from the memory side after a long round
// trip, so `issue` sends it as early as the protocol allows (thread 0 keeps
// the ticket in a register while the item runs) and `park` writes the rank
// to LDS at the end of the item, where the next iteration reads it after a
// barrier.  Every item calls `issue` exactly once, then `park`.
struct Claim {
  uint32_t* ticket;
  int base, stride, skip;
  uint32_t t;
  __device__ __forceinline__ void issue() {
    if (threadIdx.x == 0) t = __hip_atomic_fetch_add(ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __device__ __forceinline__ void park(int* s_next) const {
    if (threadIdx.x == 0) *s_next = base + stride * ((int)t + skip);
  }
};

// The mainloop hook of every item: the item's own wait for the stage at K
// offset k (if any), then, when the loads of the item's last stage are
// issued, the ticket for the work-group's next item.  The last stage's wait
// is the item's last wait, so the claim never precedes a wait of its item.
// The atomic's round trip overlaps the last stages and the epilogue, while
// the choice of the next item is still made late: a work-group that
// committed to its next item a whole item ahead would keep it from a
// work-group that frees up sooner, and lengthen the launch's tail.
struct NoWait {
  static constexpr bool kBlocks = false;  // never waits
  __device__ __forceinline__ bool all_known() const { return true; }
  __device__ __forceinline__ void operator()(int) {}
};

template <class Wait, class C = Claim>
struct ClaimAtLastStage {
  static constexpr bool kBlocks = Wait::kBlocks;
  Wait& wait;
  C* next;
  int k_last;  // K offset of the item's last stage
  __device__ __forceinline__ bool all_known() const { return wait.all_known(); }
  __device__ __forceinline__ void operator()(int k) {
    wait(k);
    if (k == k_last) next->issue();
  }
};

// The claim of an item whose successor comes from somewhere else (a
// workqueue consumer pops its next unit after the item).
struct NoClaim {
  __device__ __forceinline__ void issue() {}
  __device__ __forceinline__ void park(int*) const {}
};

// ------------------------------------------------------------------ ready flags

// Producer side (Sec. III-A: the producer fences its output, then signals):
// every wave's Z stores are complete, then one lane performs an agent-scope
// release increment of the tile's ready counter.
__device__ __forceinline__ void signal_ready(uint32_t* flag) { release_add(flag); }

// Consumer side: before loading Z columns [k, k + span) of row block mb (one
// stage), every GEMM1 tile (mb, kb) whose columns they overlap must have
// signalled in this run (once per tile and run), i.e. its counter must have
// reached epoch + 1 (compared wrap-safe).  A stage deeper than a GEMM1 tile
// is wide (128-deep stages over 64-column tiles) can need two tiles; the
// wait then repeats from the first tile still unknown.
//
// Wave 0 polls the first counter it needs; once that is ready it reads up to
// 64 consecutive counters of the item's K range in one vector load and takes
// the longest ready prefix (a ballot).  Between polls the wave sleeps; after
// spin_limit polls it gives up, latches CTRL_ERROR and stops waiting for the
// rest of the run.  The result reaches the other waves
// through LDS and a work-group barrier.  Every call is made by all waves with
// the same k.
//
// Visibility of Z.  The producer's agent-scope release writes its Z lines
// back from its XCD's L2 before the counter moves.  The consumer needs no
// agent-scope acquire (on this chip an invalidation of its XCD's whole L2,
// which throws away the lines every other work-group of the XCD is
// streaming, and measured several percent of a run where consumers wait
// often): a cache can only return a stale Z line if it already held that
// line, and none can.  Every launch starts with the caches invalidated, and
// within a launch a line of Z (128 bytes of one row in one 64-column block;
// rows and blocks are 128-byte aligned) is read only after the counter of
// the tile that writes it has been seen complete, by the work-group whose
// wait returned or by another that waited for it the same way.  The
// observing load is an atomic, so it reads the counter at the device's
// point of coherence; the Z loads are issued after it, in program order,
// and a work-group-scope acquire orders them for the compiler.
struct ReadyWait {
  static constexpr bool kBlocks = true;  // waits on ready counters before the activation loads
  const uint32_t* ready;
  uint32_t* err;  // CTRL_ERROR word
  int mb, Mb, bn1;
  int kb_last;    // last column block of this item's K range
  uint32_t target;
  uint32_t spin_limit;
  int* s_known;   // LDS broadcast slot
  int k_ready;    // K offsets below this are in column blocks this work-group has acquired (uniform)
  TraceAcc* tr;
  int span;       // K depth of one stage
  // Every producer of the item's K range was seen complete (uniform).
  __device__ __forceinline__ bool all_known() const { return k_ready == 0x7fffffff; }
  __device__ __forceinline__ void operator()(int k) {
    const int k_hi = k + span - 1;  // the stage's last column
    if (k_hi < k_ready) return;     // one compare per stage; the division below only on a miss
    const uint64_t t0 = trace_now();
    // Each round acquires at least the first unknown column block, or gives up
    // (k_ready then covers everything), so the loop ends.
    do acquire((k > k_ready ? k : k_ready) / bn1);
    while (k_hi >= k_ready);
    if constexpr (kTrace) tr->flag += trace_now() - t0;
  }
  // One poll-and-gather round from column block kb; updates k_ready.
  __device__ __forceinline__ void acquire(int kb) {
    if (uniform((int)(threadIdx.x >> 6)) == 0) {  // wave 0, as a scalar branch
      const int lane = threadIdx.x & 63;
      const int j = kb + lane;
      int hi = -1;
      if (uniform(ld_relaxed(err)) == 0u) {
        // Poll the first counter needed, every lane at the same address (one
        // request per poll: a long wait must not flood the memory side that
        // the running producers stream from); scalar loop, uniform exits.
        const uint32_t* first = ready + ((long)kb * Mb + mb) * kLine;
        uint64_t m = 0;
        for (uint32_t polls = 0;; ++polls) {
          const uint32_t v = ld_relaxed(first);
          m = __builtin_amdgcn_ballot_w64((int32_t)(v - target) >= 0);
          if ((m & 1u) || polls >= spin_limit) break;
          __builtin_amdgcn_s_sleep(2);
        }
        if (m & 1u) {
          // then the longest ready prefix of up to 64 counters in one gather
          // (counters only grow during a run, so the first is still ready)
          const uint32_t v = ld_relaxed(ready + ((long)(j <= kb_last ? j : kb_last) * Mb + mb) * kLine);
          m = __builtin_amdgcn_ballot_w64((j <= kb_last) & ((int32_t)(v - target) >= 0));
          // ~m == 0 (all 64 ready) must be taken apart: a count of trailing
          // zeros of 0 is undefined, and the scalar find-first-one the
          // compiler emits for it returns -1.
          hi = ~m ? kb + (int)__builtin_ctzll(~m) - 1 : kb + 63;
        } else if (lane == 0) {
          __hip_atomic_fetch_or(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
      if (lane == 0) *s_known = hi >= 0 ? hi : 0x7fffffff;
    }
    __syncthreads();
    const int known = uniform(*s_known);
    k_ready = known >= kb_last ? 0x7fffffff : (known + 1) * bn1;
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    // Every wave has read *s_known before wave 0 may write it again: the
    // pipeline prologue calls this back to back, with no other barrier between.
    __syncthreads();
  }
};

// ------------------------------------------------------------------ workqueue mode
//
// The paper's own consumer scheduling (Sec. III-A.2-3): a scoreboard per
// consumer unit counts its finished producers, and the producer that
// completes a unit's count pushes the unit onto a ring-buffer workqueue from
// which consumer work-groups pop whole units.  Here a unit is a GEMM2 item
// (tile, split-K part) and its producers are the GEMM1 tiles of its row
// block whose Z columns overlap its K range (a closed form, so no dependency
// array is stored).  Counts only grow, and only in workqueue runs: with w
// the number of earlier workqueue runs (CTRL_EPOCH_WQ), a unit with n
// producers reaches (w + 1) * n in this run.  (The producers also signal
// their ready counters, which thus advance once per run in every mode.)  A
// queue entry carries the low 8 bits of w + 1 above the unit id, so a
// consumer never takes a slot filled by an earlier run (every slot below
// the run's unit count is rewritten in every workqueue run).  Every unit has at least one producer (the plan
// makes S2 = ceil(F / kc2) parts, none of them empty), so every unit is
// pushed exactly once per run.

__device__ __forceinline__ uint32_t queue_tag(uint32_t wq_epoch) { return ((wq_epoch + 1u) & 0xffu) << 24; }

// Producer side: every wave's Z stores of the tile are complete, then wave 0
// increments the scoreboard of each unit that reads the tile, one unit per
// lane (agent-scope release: the tile's Z lines are written back before the
// count moves).  The units whose count this completes are pushed together:
// lane 0 reserves as many queue slots as the ballot has bits with one atomic
// (a tile that completes a whole split's units would otherwise pay one
// round trip per unit, one after the other), and each completing lane
// publishes its unit in its slot with a release store.  The queue has one spare slot
// past the run's unit count; a reservation beyond it (impossible: each unit
// completes once per run) would land there, no consumer reads it, and the
// unit's consumer would time out and report the error.
__device__ __forceinline__ void push_ready(const Args& a, int tile, uint32_t wq_epoch) {
  wait_all_mem();
  __syncthreads();
  if (uniform((int)(threadIdx.x >> 6)) == 0) {  // wave 0, as a scalar branch
    const int lane = threadIdx.x & 63;
    const int mb = tile % a.Mb, kb = tile / a.Mb;
    const int k0 = kb * a.bn1, k1 = min(a.F, k0 + a.bn1) - 1;  // the tile's Z columns
    const int s_lo = k0 / a.kc2, s_hi = k1 / a.kc2;            // the K ranges they fall in
    const int units = a.Nb2 * (s_hi - s_lo + 1);
    for (int i0 = 0; i0 < units; i0 += 64) {  // uniform trip count; one unit per lane
      const int i = i0 + lane;
      int q = 0;
      bool complete = false;
      if (i < units) {
        const int s = s_lo + i / a.Nb2, nb2 = i % a.Nb2;
        q = (nb2 * a.Mb + mb) * a.S2 + s;
        const int kbeg = s * a.kc2, kend = min(a.F, kbeg + a.kc2);
        const uint32_t n = (uint32_t)((kend - 1) / a.bn1 - kbeg / a.bn1 + 1);
        const uint32_t old =
            __hip_atomic_fetch_add(a.board + (long)q * kLine, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        complete = old + 1u == (wq_epoch + 1u) * n;
      }
      const uint64_t m = __builtin_amdgcn_ballot_w64(complete);
      if (m) {  // a scalar branch: m is the same in every lane
        uint32_t base = 0;
        if (lane == 0)
          base = __hip_atomic_fetch_add(a.ctrl + CTRL_QTAIL, (uint32_t)__builtin_popcountll(m), __ATOMIC_RELAXED,
                                        __HIP_MEMORY_SCOPE_AGENT);
        base = uniform(base);
        if (complete) {
          const uint32_t below = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
          __hip_atomic_store(a.queue + min(base + below, (uint32_t)a.items2), queue_tag(wq_epoch) | (uint32_t)q,
                             __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
    }
  }
}

// Consumer side: wave 0 claims the next queue slot and polls it (every lane
// at the same address, a scalar loop with uniform exits) until a producer of
// this run has filled it, sleeping between polls; after spin_limit polls, or
// once another wait gave up, it latches CTRL_ERROR and returns no unit.
// Returns the unit for every wave, or -1 once the run's units are all
// claimed.  Z visibility follows the ready counters' argument: every
// producer of the unit released its Z lines before its increment, the
// completing increment precedes the release store of the entry, and no L2
// holds a Z line before a consumer has seen its producers complete.
__device__ __forceinline__ int pop_ready(const Args& a, uint32_t wq_epoch, int* s_bcast) {
  if (uniform((int)(threadIdx.x >> 6)) == 0) {  // wave 0, as a scalar branch
    const int lane = threadIdx.x & 63;
    uint32_t h = 0;
    if (lane == 0) h = __hip_atomic_fetch_add(a.ctrl + CTRL_QHEAD, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    h = uniform(h);
    int q = -1;
    if (h < (uint32_t)a.items2) {
      const uint32_t want = uniform(queue_tag(wq_epoch));
      for (uint32_t polls = 0;; ++polls) {
        const uint32_t v = uniform(ld_relaxed(a.queue + h));
        if ((v & 0xff000000u) == want) {
          q = (int)(v & 0x00ffffffu);
          if (q >= a.items2) {  // not an entry any producer writes: give up loudly
            if (lane == 0) __hip_atomic_fetch_or(a.ctrl + CTRL_ERROR, 2u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            q = -1;
          }
          break;
        }
        if (polls >= a.spin_limit || ((polls & 63u) == 63u && uniform(ld_relaxed(a.ctrl + CTRL_ERROR)) != 0u)) {
          if (lane == 0) __hip_atomic_fetch_or(a.ctrl + CTRL_ERROR, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          break;
        }
        __builtin_amdgcn_s_sleep(2);
      }
    }
    if (lane == 0) *s_bcast = q;
  }
  __syncthreads();
  const int q = uniform(*s_bcast);
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  __syncthreads();  // every wave has read the slot before wave 0 writes it again
  return q;
}

}  // namespace mlp2
