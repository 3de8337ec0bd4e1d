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
// Scheduling of the pipelined launch: claim lists hand out the items of one
// rank table, the GEMM1 items in the order of the plan's order table
// (column-block-first by default, Sec. III-A.5: the first kernel may follow a
// predefined order) and each GEMM2 item after the GEMM1 items it reads.  A
// GEMM2 item only ever waits for lower-ranked GEMM1 items, which never wait,
// so the launch cannot deadlock whatever its grid size or residency (the
// argument is given with the kernels below).
#include "mlp2_device.hpp"
#include "mlp2_launch.h"

namespace mlp2 {

// ------------------------------------------------------------------ epilogues

// GEMM1 epilogue for one lane: activation in fp32 on the 8 consecutive values
// of row `row` from column `col`, round to bf16, one 16-byte store into Z.
template <int NB, bool SN = false>
__device__ __forceinline__ void store_z(const Args& a, long row, int col, const float (&v)[NB][8], bool keep = true) {
  float z[8];
  if constexpr (NB == 2) {
#pragma unroll
    for (int i = 0; i < 8; ++i) z[i] = silu(v[0][i]) * v[1][i];
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) z[i] = v[0][i];
    if (a.act == ACT_GELU_TANH) {
#pragma unroll
      for (int i = 0; i < 8; ++i) z[i] = gelu_tanh(z[i]);
    }
  }
  const u32x4 packed = canonicalize_z(pack_bf16x8(z));  // never the sentinel pattern
  if constexpr (SN) {
    // Sentinel mode: the piece goes straight to the device's point of
    // coherence, with no fence or flag after it; the same piece of the next
    // sentinel run's intermediate is refilled with sentinels.
    if (keep) store_coherent16(a.Z + row * a.F + col, packed);  // !keep: a dropped tile (failure injection)
    const u32x4 sent = {0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu};
    *reinterpret_cast<u32x4*>(a.Zr + row * a.F + col) = sent;
  } else {
    *reinterpret_cast<u32x4*>(a.Z + row * a.F + col) = packed;
  }
}

__device__ __forceinline__ void store_y(const Args& a, int row, int col, const float (&v)[8]) {
  if (row < a.M) *reinterpret_cast<u32x4*>(a.Y + (long)row * a.H + col) = pack_bf16x8(v);
}

// Claim lists.  Work-groups are placed on the XCDs round-robin by index, so
// with 8 lists (work-group g on list g % 8) every XCD takes every 8th item of
// the rank order: the same number of weight-streaming items per XCD (and per
// L2 and fabric link), while the chip as a whole still works through the
// ranks in order.  Work-groups g < first_static take rank g as their first
// item without a ticket (those ranks are items that never wait); list l then
// skips the ranks below first_static it would hand out.
//
// With a role split (Args::p1) the pipelined launch holds two sets of claim
// lists: the GEMM1 role's work-groups (g % 64 < p1) deal the GEMM1 order
// table's ranks over lists 0..7, the GEMM2 role's the GEMM2 order table's over
// lists 8..15.  A work-group's list is its index among its role's work-groups
// modulo the role's list count; with p1 a multiple of 8 that index is
// congruent to g modulo 8, so every XCD still takes every 8th item of each
// role.
struct ListPos {
  int role;   // -1 shared, 0 GEMM1 role, 1 GEMM2 role
  int i, n;   // this work-group's index among the work-groups of its set, and their number
  int lists;  // claim lists of the set
  int list;   // this work-group's list, as an index into the control words' ticket and done lines
};

__device__ __forceinline__ ListPos list_pos(const Args& a, bool roles) {
  const int g = (int)blockIdx.x, G = (int)gridDim.x;
  if (!roles) return ListPos{-1, g, G, a.lists, g % a.lists};
  const int q = g / 64, j = g % 64, full = G / 64, rem = G % 64;
  const int n1 = full * a.p1 + min(rem, a.p1);
  if (j < a.p1) return ListPos{0, q * a.p1 + j, n1, a.lists, (q * a.p1 + j) % a.lists};
  const int i = q * (64 - a.p1) + (j - a.p1);
  return ListPos{1, i, G - n1, a.lists2, 8 + i % a.lists2};
}

__device__ __forceinline__ Claim make_claim(const Args& a, bool roles) {
  const ListPos lp = list_pos(a, roles);
  const int l = lp.i % lp.lists;
  const int skip = lp.role < 0 && l < a.first_static ? (a.first_static - 1 - l) / lp.lists + 1 : 0;
  return Claim{a.ctrl + ctrl_ticket(lp.list), l, lp.lists, skip, 0u};
}

// ------------------------------------------------------------------ trace records (MLP2_TRACE builds)

// Layout of the trace buffer: per kernel section (0 = GEMM1 or pipelined
// kernel, 1 = GEMM2 kernel of the sequential mode; trace_groups work-groups
// per section) and work-group, one word
// with the item count, then trace_cap records of kTraceWords words: rank
// (high half) and item (low half: the order-table entry, bit 31 set for a
// GEMM2 item), start, mainloop end, two epilogue marks (a signalling GEMM1 tile: Z stores
// complete, ready counter released; a split-K part that leaves the tile to a
// sibling: partial stored, arrival counted; else 0 and 0), end, ring-wait
// ticks, flag-wait ticks.  Records past
// trace_cap are counted, not stored.  Written by thread 0 with plain stores.
__device__ __forceinline__ void tr_mark_mainloop(TraceAcc& tr) { tr.t_main = trace_now(); }

__device__ __forceinline__ void tr_record(const Args& a, int section, int n, int rank, uint32_t item,
                                          uint64_t t_start, const TraceAcc& tr) {
  if (a.trace == nullptr || threadIdx.x != 0) return;
  uint64_t* slot = a.trace + ((long)section * a.trace_groups + blockIdx.x) * (1 + (long)a.trace_cap * kTraceWords);
  slot[0] = (uint64_t)(n + 1);
  if (n >= a.trace_cap) return;
  uint64_t* r = slot + 1 + (long)n * kTraceWords;
  r[0] = ((uint64_t)(uint32_t)rank << 32) | item;
  r[1] = t_start;
  r[2] = tr.t_main;
  r[3] = tr.t_rel;
  r[4] = tr.t_wait;
  r[5] = trace_now();
  r[6] = ((trace_clock() - tr.c_start) << 32) | (uint32_t)tr.ring;  // core cycles | ring-wait ticks
  r[7] = tr.flag;
}

// The completing part's reduction: every unit of the tile, G units per wave
// at a time (two for one weight operand, one for two), handed to `epi` with
// the unit's summed values.
template <class T, int NB, class Epi>
__device__ __forceinline__ void reduce_epilogue(const float* part, long tile, int S, Epi&& epi) {
  constexpr int U = Partial<T, NB>::UNITS;
  constexpr int G = NB == 1 ? 2 : 1;
  static_assert(U % G == 0, "units per group");
  const int lane = threadIdx.x & 63;
  for (int u0 = uniform((int)(threadIdx.x >> 6)) * G; u0 < U; u0 += T::NWAVES * G) {
    Unit<T> ug[G];
#pragma unroll
    for (int g = 0; g < G; ++g) ug[g] = Unit<T>(u0 + g);
    float v[G][NB][8];
    reduce_units<T, NB, G>(part, tile, S, ug, lane, v);
#pragma unroll
    for (int g = 0; g < G; ++g) epi(ug[g], lane, v[g]);
  }
}

// One slice of a tile's reduction (reduction items): the tile's units in
// groups of G, the slice's groups dealt to the waves; the same sums, in the
// same order, as the completing part's reduction above.
template <class T, int NB, class Epi>
__device__ __forceinline__ void reduce_slice(const float* part, long tile, int S, int slice, int slices, Epi&& epi) {
  constexpr int U = Partial<T, NB>::UNITS;
  constexpr int G = NB == 1 ? 2 : 1;
  static_assert(U % G == 0, "units per group");
  const int per = U / G / slices;  // groups per slice (the plan makes `slices` divide U / G)
  const int lane = threadIdx.x & 63;
  for (int grp = uniform((int)(threadIdx.x >> 6)); grp < per; grp += T::NWAVES) {
    const int u0 = (slice * per + grp) * G;
    Unit<T> ug[G];
#pragma unroll
    for (int g = 0; g < G; ++g) ug[g] = Unit<T>(u0 + g);
    float v[G][NB][8];
    reduce_units<T, NB, G>(part, tile, S, ug, lane, v);
#pragma unroll
    for (int g = 0; g < G; ++g) epi(ug[g], lane, v[g]);
  }
}

// ------------------------------------------------------------------ work items
//
// Split-K epilogue, shared by both GEMMs: each part stores its partial and
// counts its arrival (arrive_split); the part that completes the tile sums
// all S partials in the fixed order s = 0..S-1 and runs the tile's epilogue,
// the others claim their next item at once.  A GEMM1 tile signals its ready
// counter once per run, after the tile's Z rows are stored.

// GEMM1 item id = tile * S1 + s, tile = nb * Mb + mb.  WQ: the completed
// tile also feeds the workqueue's scoreboards (wq_epoch: workqueue runs so far).
template <class T, int NB, bool WQ = false, bool SN = false>
__device__ __forceinline__ void gemm1_item(const Args& a, int id_in, uint32_t epoch, char* lds, int* s_slot,
                                           Claim& next, int* s_next, TraceAcc& tr, uint32_t wq_epoch = 0) {
  const int id = uniform(id_in);
  const int tile = id / a.S1, s = id - tile * a.S1;
  const int mb = tile % a.Mb, nb = tile / a.Mb;
  const int m0 = mb * T::BM, n0 = nb * T::BN;
  const int kbeg = s * a.kc1;
  const int kend = min(a.H, kbeg + a.kc1);

  f32x4 acc[NB][T::TN][T::TM];
  const uint16_t* Bp[NB];
  Bp[0] = a.W1;
  if constexpr (NB == 2) Bp[1] = a.W1 + (long)a.H * a.F;
  NoWait nowait;  // a GEMM1 item never waits
  ClaimAtLastStage<NoWait> hook{nowait, &next, kend - T::BK};
  mainloop<T, NB>(a.X, a.H, m0, a.M - 1, Bp, a.F, n0, kbeg, kend, acc, lds, hook, tr);
  if constexpr (kTrace) tr_mark_mainloop(tr);

  if (a.S1 == 1) {
    next.park(s_next);
    FragPos<T> fp(m0, n0);
#pragma unroll
    for (int tm = 0; tm < T::TM; ++tm)
#pragma unroll
      for (int tp = 0; tp < T::TN / 2; ++tp) {
        float v[NB][8];
#pragma unroll
        for (int b = 0; b < NB; ++b) pair_values<T>(acc[b], tp, tm, v[b]);
        store_z<NB, SN>(a, fp.row0 + 16 * tm, fp.col0 + 32 * tp, v, tile != a.drop_signal);
      }
  } else {
    const bool last = arrive_split<T, NB>(a.part1, a.cnt1 + (long)tile * kLine, tile, a.S1, s,
                                          (epoch + 1u) * (uint32_t)a.S1, acc, s_slot, tr);
    next.park(s_next);
    if (!last) return;
    reduce_epilogue<T, NB>(a.part1, tile, a.S1, [&](const Unit<T>& u, int lane, const float (&v)[NB][8]) {
      store_z<NB, SN>(a, u.row(m0, lane), u.col(n0, lane), v, tile != a.drop_signal);
    });
  }
  if constexpr (SN) return;  // no fence and no flag: consumers check the data itself
  // Producer signal (one per tile and run): the tile's Z rows are released, ready[tile] += 1.
  if constexpr (kTrace) {
    wait_all_mem();
    tr.t_rel = trace_now();
  }
  if (tile != a.drop_signal) {
    signal_ready(a.ready + (long)tile * kLine);
    if constexpr (WQ) push_ready(a, tile, wq_epoch);
  }
  if constexpr (kTrace) tr.t_wait = trace_now();
}

// GEMM2 item p = tile * S2 + s (the parts of a tile are adjacent tickets,
// see the kernels' deadlock argument).  WAIT: each K-slice of Z is consumed
// only after its GEMM1 tile has signalled.  The tile is HV column halves of
// T side by side (HV = 1 or 2): with HV = 2 the mainloop treats the halves
// as two weight operands (W2 at the tile's column and T::BN columns further
// on), the same instantiation the gated GEMM1 uses for its Wg and Wu, so a
// kernel that holds both item kinds carries one mainloop shape and one
// register budget.  Each output element still accumulates over K in the
// same order.
template <class T, int HV, bool WAIT, class C = Claim, bool SN = false>
__device__ __forceinline__ void gemm2_item(const Args& a, int p_in, uint32_t epoch, char* lds, int* s_slot,
                                           C& next, int* s_next, TraceAcc& tr, uint32_t ready_runs = 0) {
  const int p = uniform(p_in);
  const int tile = p / a.S2, s = p - (p / a.S2) * a.S2;
  const int mb = tile % a.Mb, nb = tile / a.Mb;
  const int m0 = mb * T::BM, n0 = nb * T::BN * HV;
  const int kbeg = s * a.kc2;
  const int kend = min(a.F, kbeg + a.kc2);

  f32x4 acc[HV][T::TN][T::TM];
  const uint16_t* Bp[HV];
#pragma unroll
  for (int h = 0; h < HV; ++h) Bp[h] = a.W2 + h * T::BN;
  const int zlast = a.Mb * T::BM - 1;
  if constexpr (SN) {
    // Sentinel mode: no ready counters; each stage's Z pieces are loaded at
    // device scope and checked for sentinels before the stage is used.
    NoWait nowait;
    ClaimAtLastStage<NoWait, C> hook{nowait, &next, kend - T::BK};
    SentinelCheck check{a.ctrl + CTRL_ERROR, a.spin_limit, &tr};
    mainloop<T, HV>(a.Z, a.F, m0, zlast, Bp, a.H, n0, kbeg, kend, acc, lds, hook, tr, check);
  } else if constexpr (WAIT) {
    // ready counters advance once per run of every mode but the sentinel mode
    ReadyWait w{a.ready, a.ctrl + CTRL_ERROR, mb, a.Mb, a.bn1, (kend - 1) / a.bn1, ready_runs + 1u, a.spin_limit,
                s_slot, 0, &tr, T::BK};
    ClaimAtLastStage<ReadyWait, C> hook{w, &next, kend - T::BK};
    mainloop<T, HV>(a.Z, a.F, m0, zlast, Bp, a.H, n0, kbeg, kend, acc, lds, hook, tr);
  } else {
    NoWait nowait;
    ClaimAtLastStage<NoWait, C> hook{nowait, &next, kend - T::BK};
    mainloop<T, HV>(a.Z, a.F, m0, zlast, Bp, a.H, n0, kbeg, kend, acc, lds, hook, tr);
  }
  if constexpr (kTrace) tr_mark_mainloop(tr);

  if (a.S2 == 1) {
    next.park(s_next);
    FragPos<T> fp(m0, n0);
#pragma unroll
    for (int h = 0; h < HV; ++h)
#pragma unroll
      for (int tm = 0; tm < T::TM; ++tm)
#pragma unroll
        for (int tp = 0; tp < T::TN / 2; ++tp) {
          float v[8];
          pair_values<T>(acc[h], tp, tm, v);
          store_y(a, fp.row0 + 16 * tm, fp.col0 + h * T::BN + 32 * tp, v);
        }
  } else if (a.red2 > 0) {
    // The tile is summed by its reduction items: store the partial and count
    // the arrival (a release), then on to the next item.
    store_partial<T, HV>(a.part2, tile, a.S2, s, acc);
    if constexpr (kTrace) {
      wait_all_mem();
      tr.t_rel = trace_now();
    }
    release_add(a.cnt2 + (long)tile * kLine);
    if constexpr (kTrace) tr.t_wait = trace_now();
    next.park(s_next);
  } else {
    const bool last = arrive_split<T, HV>(a.part2, a.cnt2 + (long)tile * kLine, tile, a.S2, s,
                                          (epoch + 1u) * (uint32_t)a.S2, acc, s_slot, tr);
    next.park(s_next);
    if (!last) return;
    reduce_epilogue<T, HV>(a.part2, tile, a.S2, [&](const Unit<T>& u, int lane, const float (&v)[HV][8]) {
#pragma unroll
      for (int h = 0; h < HV; ++h) store_y(a, u.row(m0, lane), u.col(n0, lane) + h * T::BN, v[h]);
    });
  }
}

// Reduction item r = tile * red2 + slice of a GEMM2 tile with split-K: wait
// until every part of the tile has arrived in this run (its arrival counter at
// (epoch + 1) * S2, compared wrap-safe; thread 0 polls, the group waits at a
// barrier), then sum the slice's units over the parts in the fixed order and
// store them.  Reduction items rank after every GEMM2 item, so they wait only
// for lower ranks, and the whole tile is summed by red2 work-groups at once
// instead of by the part that arrives last.  The partials need no agent-scope
// acquire, for the reason given at arrive_split (each slice's 1 KB runs are
// read once per launch, by one item, after every part released them).  A wait
// that gives up latches CTRL_ERROR (bit 0) and skips the sums; the kernel
// still drains and mlp2_check reports the timeout.
template <class T, int HV, class C = Claim>
__device__ __forceinline__ void reduce_item(const Args& a, int r_in, uint32_t epoch, int* s_slot, C& next, int* s_next,
                                            TraceAcc& tr) {
  const int r = uniform(r_in);
  const int tile = r / a.red2, slice = r - tile * a.red2;
  const int mb = tile % a.Mb, nb = tile / a.Mb;
  const int m0 = mb * T::BM, n0 = nb * T::BN * HV;
  const uint32_t* cnt = a.cnt2 + (long)tile * kLine;
  const uint32_t target = (epoch + 1u) * (uint32_t)a.S2;
  const uint64_t t0 = trace_now();
  if (threadIdx.x == 0) {
    int ok = 0;
    if (ld_relaxed(a.ctrl + CTRL_ERROR) == 0u) {
      for (uint32_t polls = 0;; ++polls) {
        if ((int32_t)(ld_relaxed(cnt) - target) >= 0) {
          ok = 1;
          break;
        }
        if (polls >= a.spin_limit) break;
        __builtin_amdgcn_s_sleep(2);
      }
      if (!ok) __hip_atomic_fetch_or(a.ctrl + CTRL_ERROR, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    *s_slot = ok;
  }
  __syncthreads();
  const bool ok = uniform(*s_slot) != 0;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  __syncthreads();  // *s_slot may be rewritten
  if constexpr (kTrace) {
    tr.flag += trace_now() - t0;
    tr_mark_mainloop(tr);
  }
  next.issue();  // after the item's only wait
  if (ok)
    reduce_slice<T, HV>(a.part2, tile, a.S2, slice, a.red2, [&](const Unit<T>& u, int lane, const float (&v)[HV][8]) {
#pragma unroll
      for (int h = 0; h < HV; ++h) store_y(a, u.row(m0, lane), u.col(n0, lane) + h * T::BN, v[h]);
    });
  next.park(s_next);
}

// Counter lifetime across kernels and runs.  The last work-group of each
// claim list to finish resets that list's ticket and done count (no
// work-group of the list claims again); the last list to finish resets the
// list count and, at the end of a run, advances the epoch.  Everything is
// stream-ordered before the plan's next kernel.  Spreading the done counts
// over the lists keeps the exit atomics, one per work-group, off a single
// line.
__device__ __forceinline__ void finish_kernel(const Args& a, bool roles, uint32_t epoch, bool end_of_run,
                                              bool wq_run = false, uint32_t wq_epoch = 0, bool sn_run = false,
                                              uint32_t sn_epoch = 0) {
  __syncthreads();
  if (threadIdx.x == 0) {
    const ListPos lp = list_pos(a, roles);
    const int l = lp.i % lp.lists;
    const uint32_t in_list = (uint32_t)((lp.n - 1 - l) / lp.lists + 1);
    const uint32_t old = __hip_atomic_fetch_add(a.ctrl + ctrl_done(lp.list), 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    if (old == in_list - 1u) {
      __hip_atomic_store(a.ctrl + ctrl_ticket(lp.list), 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(a.ctrl + ctrl_done(lp.list), 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const uint32_t lists_done =
          __hip_atomic_fetch_add(a.ctrl + CTRL_DONE_ALL, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
      const uint32_t all_lists = (uint32_t)(lp.role < 0 ? a.lists : a.lists + a.lists2);
      if (lists_done == all_lists - 1u) {
        __hip_atomic_store(a.ctrl + CTRL_DONE_ALL, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(a.ctrl + CTRL_QHEAD, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(a.ctrl + CTRL_QTAIL, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (wq_run) __hip_atomic_store(a.ctrl + CTRL_EPOCH_WQ, wq_epoch + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (sn_run) __hip_atomic_store(a.ctrl + CTRL_EPOCH_SN, sn_epoch + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (end_of_run) __hip_atomic_store(a.ctrl + CTRL_EPOCH, epoch + 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
}

// ------------------------------------------------------------------ kernels
//
// Every kernel is persistent: a work-group claims item ranks (Claim) until
// the kernel's items are exhausted.  Items in rank order:
//   PHASE_GEMM1:     GEMM1 items in the order table's order
//   PHASE_GEMM2:     GEMM2 items
//   PHASE_PIPELINED: the merged table: GEMM1 items in the same order, each
//                    GEMM2 item placed after every GEMM1 item it reads (plus
//                    a lag of about one grid), so that GEMM2 work starts while
//                    later GEMM1 items still run; GEMM2 items wait per K-slice.
// Claim list l holds the ranks congruent to l modulo `lists` and hands them
// out in increasing order.  The only waits are a GEMM2 item's waits for GEMM1
// tiles, which have lower ranks in every table (split-K parts never wait for
// each other).  A work-group takes the ticket for its next item only after the
// last wait of its current item.  First items taken without a ticket are items
// that never wait, so they finish whether or not their work-group is resident
// yet.  Take the lowest-ranked unfinished item u: every lower rank is
// finished, so if u is claimed its waits end and it finishes; if it is not,
// every claimed item of its list ranks below u and is finished, so a
// work-group of that list is free to claim it.  Hence no launch deadlocks for
// any grid with at least one work-group per list, whatever the residency.
//
//   PHASE_WORKQUEUE: GEMM1 items by rank as in PHASE_GEMM1; a work-group whose
//                    claim runs past them pops GEMM2 units from the device
//                    workqueue until every unit of the run is claimed.  It
//                    pops only once every GEMM1 item is claimed, and GEMM1
//                    items never wait, so every producer finishes and every
//                    claimed queue slot is filled: no deadlock either.

//   PHASE_SENTINEL:  the pipelined rank table and claims, with the Lamport-
//                    style synchronisation of Sec. V-A: GEMM1 items store Z at
//                    device scope with no fence and no ready counter; GEMM2
//                    items wait for nothing but re-read each stage's Z pieces
//                    while any still holds the sentinel.  A GEMM2 item still
//                    depends only on lower-ranked GEMM1 items, so the
//                    deadlock argument above holds unchanged.

enum { PHASE_GEMM1 = 0, PHASE_GEMM2 = 1, PHASE_PIPELINED = 2, PHASE_WORKQUEUE = 3, PHASE_SENTINEL = 4 };

template <int A, int B>
struct MaxI {
  static constexpr int value = A > B ? A : B;
};

template <class T1, int NB, class T2, int HV, int PHASE>
constexpr int kernel_lds() {
  return PHASE == PHASE_GEMM1   ? T1::template lds_bytes<NB>()
         : PHASE == PHASE_GEMM2 ? T2::template lds_bytes<HV>()
                                : MaxI<T1::template lds_bytes<NB>(), T2::template lds_bytes<HV>()>::value;
}

// Work-groups per CU the register budget must allow: two four-wave groups
// whenever two rings fit in LDS; eight-wave groups run one per CU (two
// waves per SIMD already).
template <class T1, int NB, class T2, int HV, int PHASE>
constexpr int min_blocks() {
  return kernel_lds<T1, NB, T2, HV, PHASE>() <= 80 * 1024 && T1::NWAVES == 4 ? 2 : 1;
}

// T1, NB: GEMM1 tile and weight operands; T2, HV: GEMM2 tile half and halves.
// Both item kinds run in the same work-groups, so their tiles have the same waves.
template <class T1, int NB, class T2, int HV, int PHASE>
__global__ __launch_bounds__(T1::THREADS, (min_blocks<T1, NB, T2, HV, PHASE>())) void k_mlp2(Args a) {
  static_assert(T1::THREADS == T2::THREADS, "one work-group shape for both item kinds");
  constexpr int kLds = kernel_lds<T1, NB, T2, HV, PHASE>();
  __shared__ __attribute__((aligned(1024))) char lds[kLds];
  __shared__ int s_item, s_slot;
  const uint32_t epoch = uniform(ld_relaxed(a.ctrl + CTRL_EPOCH));
  const uint32_t wq_epoch = PHASE == PHASE_WORKQUEUE ? uniform(ld_relaxed(a.ctrl + CTRL_EPOCH_WQ)) : 0u;
  // Sentinel runs alternate between two intermediates: this run's producers
  // write one and refill the other with sentinels for the next sentinel run.
  const uint32_t sn_epoch =
      PHASE == PHASE_SENTINEL || PHASE == PHASE_PIPELINED ? uniform(ld_relaxed(a.ctrl + CTRL_EPOCH_SN)) : 0u;
  // Earlier runs whose GEMM1 tiles signalled the ready counters: every run but the sentinel runs.
  const uint32_t ready_runs = epoch - sn_epoch;
  if constexpr (PHASE == PHASE_SENTINEL) {
    a.Z = a.Zs + (long)(sn_epoch & 1u) * a.zs_elems;
    a.Zr = a.Zs + (long)((sn_epoch + 1u) & 1u) * a.zs_elems;
  }
  // A role split (pipelined launch only): this work-group takes the items of
  // one kind, in that kind's order table; otherwise both kinds from one order.
  const ListPos lp = list_pos(a, PHASE == PHASE_PIPELINED && a.p1 > 0);
  const int g1 = PHASE == PHASE_GEMM2 || lp.role == 1 ? 0 : a.items1;
  const int g2 = (PHASE == PHASE_GEMM2 || PHASE == PHASE_PIPELINED || PHASE == PHASE_SENTINEL) && lp.role != 0 ? a.items2 : 0;
  // reduction items (ranked last) in the launches that sum split-K tiles with them
  const int gr = (PHASE == PHASE_GEMM2 || PHASE == PHASE_PIPELINED) && lp.role != 0 ? a.items_red : 0;
  const int total = g1 + g2 + gr;
  int p;
  if (lp.role < 0 && (int)blockIdx.x < a.first_static) {
    p = (int)blockIdx.x;
  } else {
    Claim first = make_claim(a, lp.role >= 0);
    first.issue();
    first.park(&s_item);
    __syncthreads();
    p = uniform(s_item);
  }
  int n_items = 0;
  for (;;) {
    if (p >= total) break;
    __syncthreads();  // every wave has read s_item before the item's claim rewrites it
    TraceAcc tr;
    if constexpr (kTrace) tr.c_start = trace_clock();
    const uint64_t t_start = trace_now();
    Claim next = make_claim(a, lp.role >= 0);
    uint32_t e;  // order-table entry: item id, bit 31 set for a GEMM2 item
    if constexpr (PHASE == PHASE_SENTINEL) {
      e = uniform(a.orderp[p]);
      if (e & 0x80000000u)
        gemm2_item<T2, HV, false, Claim, true>(a, (int)(e & 0x7fffffffu), epoch, lds, &s_slot, next, &s_item, tr);
      else
        gemm1_item<T1, NB, false, true>(a, (int)e, epoch, lds, &s_slot, next, &s_item, tr);
    } else if constexpr (PHASE == PHASE_PIPELINED) {
      e = lp.role < 0 ? uniform(a.orderp[p]) : lp.role == 0 ? uniform(a.order1[p]) : (uniform(a.order2[p]) | 0x80000000u);
      if ((e & 0xc0000000u) == 0xc0000000u)
        reduce_item<T2, HV>(a, (int)(e & 0x3fffffffu), epoch, &s_slot, next, &s_item, tr);
      else if (e & 0x80000000u)
        gemm2_item<T2, HV, true>(a, (int)(e & 0x7fffffffu), epoch, lds, &s_slot, next, &s_item, tr, ready_runs);
      else
        gemm1_item<T1, NB>(a, (int)e, epoch, lds, &s_slot, next, &s_item, tr);
    } else if constexpr (PHASE == PHASE_GEMM1 || PHASE == PHASE_WORKQUEUE) {
      e = uniform(a.order1[p]);
      gemm1_item<T1, NB, PHASE == PHASE_WORKQUEUE>(a, (int)e, epoch, lds, &s_slot, next, &s_item, tr, wq_epoch);
    } else {
      e = uniform(a.order2[p]);
      if (e & 0x40000000u)
        reduce_item<T2, HV>(a, (int)(e & 0x3fffffffu), epoch, &s_slot, next, &s_item, tr);
      else
        gemm2_item<T2, HV, false>(a, (int)e, epoch, lds, &s_slot, next, &s_item, tr);
      e |= 0x80000000u;
    }
    if constexpr (kTrace) tr_record(a, PHASE == PHASE_GEMM2 ? 1 : 0, n_items++, p, e, t_start, tr);
    __syncthreads();
    p = uniform(s_item);
  }
  if constexpr (PHASE == PHASE_WORKQUEUE) {
    __syncthreads();  // every wave is done with s_item before pop_ready rewrites it
    uint64_t t_pop = trace_now();  // a unit's trace starts when its work-group begins to pop it
    uint64_t c_pop = trace_clock();
    for (int q = pop_ready(a, wq_epoch, &s_item); q >= 0; q = pop_ready(a, wq_epoch, &s_item)) {
      TraceAcc tr;
      if constexpr (kTrace) tr.c_start = c_pop;
      if constexpr (kTrace) tr.flag = trace_now() - t_pop;  // waiting for the queue slot to fill
      NoClaim none;
      gemm2_item<T2, HV, false, NoClaim>(a, q, epoch, lds, &s_slot, none, &s_item, tr);
      if constexpr (kTrace) tr_record(a, 0, n_items++, -1, 0x80000000u | (uint32_t)q, t_pop, tr);
      __syncthreads();  // the item's divergent stores close, and s_item is free again
      t_pop = trace_now();
      c_pop = trace_clock();
    }
  }
  finish_kernel(a, lp.role >= 0, epoch, PHASE != PHASE_GEMM1, PHASE == PHASE_WORKQUEUE, wq_epoch,
                PHASE == PHASE_SENTINEL, sn_epoch);
}

// ------------------------------------------------------------------ dispatch table

// Tile shapes by (rows, columns, ring depth, waves); the stage depth is a
// parameter of the eight-wave shapes (TileForK).
template <int BM, int BN, int NS, int W = 4>
struct TileFor;
template <int NS> struct TileFor<32, 64, NS> { using type = Tile<32, 64, 2, 2, NS>; };
template <int NS> struct TileFor<32, 128, NS> { using type = Tile<32, 128, 1, 4, NS>; };
template <int NS> struct TileFor<64, 64, NS> { using type = Tile<64, 64, 2, 2, NS>; };
template <int NS> struct TileFor<64, 128, NS> { using type = Tile<64, 128, 2, 2, NS>; };
template <int NS> struct TileFor<128, 64, NS> { using type = Tile<128, 64, 2, 2, NS>; };
template <int NS> struct TileFor<128, 128, NS> { using type = Tile<128, 128, 2, 2, NS>; };
template <int NS> struct TileFor<128, 256, NS> { using type = Tile<128, 256, 2, 2, NS>; };
template <int NS> struct TileFor<64, 256, NS> { using type = Tile<64, 256, 1, 4, NS>; };
template <int NS> struct TileFor<32, 256, NS> { using type = Tile<32, 256, 1, 4, NS>; };
template <int NS> struct TileFor<256, 64, NS> { using type = Tile<256, 64, 4, 1, NS>; };
template <int NS> struct TileFor<256, 128, NS> { using type = Tile<256, 128, 4, 1, NS>; };
// eight waves
template <int NS> struct TileFor<256, 256, NS, 8> { using type = Tile<256, 256, 2, 4, NS>; };
template <int NS> struct TileFor<256, 128, NS, 8> { using type = Tile<256, 128, 4, 2, NS>; };
template <int NS> struct TileFor<256, 64, NS, 8> { using type = Tile<256, 64, 4, 2, NS>; };
template <int NS> struct TileFor<128, 256, NS, 8> { using type = Tile<128, 256, 2, 4, NS>; };
template <int NS> struct TileFor<128, 128, NS, 8> { using type = Tile<128, 128, 2, 4, NS>; };
template <int NS> struct TileFor<128, 64, NS, 8> { using type = Tile<128, 64, 4, 2, NS>; };
template <int NS> struct TileFor<64, 256, NS, 8> { using type = Tile<64, 256, 2, 4, NS>; };
template <int NS> struct TileFor<32, 256, NS, 8> { using type = Tile<32, 256, 1, 8, NS>; };
template <int BM, int BN, int NS, int W, int BK, bool WNT = false>
struct TileForK {
  using base = typename TileFor<BM, BN, NS, W>::type;
  using type = Tile<BM, BN, base::WM, base::WN, NS, BK, WNT>;
};

struct Entry {
  int bm, bn1, bn2, nb, ns, waves, bk, wnt;
  const void* seq1;
  const void* seq2;
  const void* pipe;
  const void* wq;
  const void* sn;
};

// GEMM2 of BN2 columns as one tile (HV = 1), or as two halves of BN2 / 2 that
// share the GEMM1 tile shape (HV = 2).
#define MLP2_K(BM, BN1, BN2, NB, NS, HV, W, BK, NT, PH)                                      \
  (const void*)&k_mlp2<typename TileForK<BM, BN1, NS, W, BK, NT>::type, NB,                   \
                       typename TileForK<BM, (BN2) / (HV), NS, W, BK, NT>::type, HV, PH>
#define MLP2_ENTRY_WKN(BM, BN1, BN2, NB, NS, HV, W, BK, NT)                                   \
  Entry {                                                                                     \
    BM, BN1, BN2, NB, NS, W, BK, NT, MLP2_K(BM, BN1, BN2, NB, NS, HV, W, BK, NT, PHASE_GEMM1), \
        MLP2_K(BM, BN1, BN2, NB, NS, HV, W, BK, NT, PHASE_GEMM2),                             \
        MLP2_K(BM, BN1, BN2, NB, NS, HV, W, BK, NT, PHASE_PIPELINED),                         \
        MLP2_K(BM, BN1, BN2, NB, NS, HV, W, BK, NT, PHASE_WORKQUEUE),                         \
        MLP2_K(BM, BN1, BN2, NB, NS, HV, W, BK, NT, PHASE_SENTINEL)                           \
  }
#define MLP2_ENTRY_WK(BM, BN1, BN2, NB, NS, HV, W, BK) MLP2_ENTRY_WKN(BM, BN1, BN2, NB, NS, HV, W, BK, false)
#define MLP2_ENTRY_W(BM, BN1, BN2, NB, NS, HV, W) MLP2_ENTRY_WK(BM, BN1, BN2, NB, NS, HV, W, 64)
#define MLP2_ENTRY_HV(BM, BN1, BN2, NB, NS, HV) MLP2_ENTRY_W(BM, BN1, BN2, NB, NS, HV, 4)
#define MLP2_ENTRY(BM, BN1, BN2, NB, NS) MLP2_ENTRY_HV(BM, BN1, BN2, NB, NS, 1)

static const Entry kEntries[] = {
    MLP2_ENTRY(32, 128, 128, 1, 4), MLP2_ENTRY(32, 128, 64, 1, 4), MLP2_ENTRY(32, 64, 128, 1, 4), MLP2_ENTRY(32, 64, 64, 1, 4),
    MLP2_ENTRY(64, 128, 128, 1, 4), MLP2_ENTRY(64, 128, 64, 1, 4), MLP2_ENTRY(64, 64, 128, 1, 4), MLP2_ENTRY(64, 64, 64, 1, 4),
    MLP2_ENTRY(128, 128, 128, 1, 4), MLP2_ENTRY(128, 128, 64, 1, 4), MLP2_ENTRY(128, 64, 128, 1, 4), MLP2_ENTRY(128, 64, 64, 1, 4),
    MLP2_ENTRY(32, 64, 128, 2, 4), MLP2_ENTRY(32, 64, 64, 2, 4), MLP2_ENTRY(64, 64, 128, 2, 4), MLP2_ENTRY(64, 64, 64, 2, 4),
    MLP2_ENTRY(128, 64, 128, 2, 4), MLP2_ENTRY(128, 64, 64, 2, 4),
    // shallower rings: two work-groups per CU
    MLP2_ENTRY(128, 128, 128, 1, 2), MLP2_ENTRY(128, 128, 128, 1, 3), MLP2_ENTRY(128, 64, 64, 1, 3),
    MLP2_ENTRY(64, 128, 128, 1, 3), MLP2_ENTRY(128, 64, 128, 2, 2), MLP2_ENTRY(32, 128, 128, 1, 3),
    // wide weight tiles: half the activation traffic per weight byte
    MLP2_ENTRY(128, 256, 256, 1, 3), MLP2_ENTRY(128, 256, 128, 1, 3), MLP2_ENTRY(128, 128, 256, 1, 3),
    MLP2_ENTRY(128, 256, 256, 1, 2), MLP2_ENTRY(32, 256, 256, 1, 4), MLP2_ENTRY(64, 256, 256, 1, 3),
    // 256-row blocks: the weights of a 129..256-row batch are streamed once; the
    // gated GEMM2 of 128 columns runs as two 64-column halves (the GEMM1 shape)
    MLP2_ENTRY_HV(256, 64, 128, 2, 3, 2), MLP2_ENTRY(256, 64, 64, 2, 3), MLP2_ENTRY(256, 128, 128, 1, 3),
    MLP2_ENTRY(256, 64, 64, 1, 3),
    // eight-wave work-groups: large tiles, two waves per SIMD
    MLP2_ENTRY_W(256, 256, 256, 1, 2, 1, 8), MLP2_ENTRY_W(256, 128, 128, 1, 3, 1, 8),
    MLP2_ENTRY_W(256, 256, 128, 1, 2, 1, 8), MLP2_ENTRY_W(256, 128, 256, 1, 2, 2, 8),
    MLP2_ENTRY_W(256, 128, 256, 2, 2, 2, 8), MLP2_ENTRY_W(256, 64, 128, 2, 3, 2, 8),
    // the gated tile with non-temporal weight loads (weights beyond the last-level cache)
    MLP2_ENTRY_WKN(256, 128, 256, 2, 2, 2, 8, 64, true),
    MLP2_ENTRY_W(128, 128, 128, 1, 4, 1, 8), MLP2_ENTRY_W(128, 256, 256, 1, 3, 1, 8),
    MLP2_ENTRY_W(128, 64, 64, 1, 4, 1, 8),
    // 32-deep stages: twice the ring depth in the same LDS (measured slower
    // than 64-deep stages on every workload: one barrier per half the work)
    MLP2_ENTRY_WK(256, 128, 256, 2, 4, 2, 8, 32), MLP2_ENTRY_WK(128, 64, 64, 1, 8, 1, 4, 32),
    // 128-deep stages for the weight-streaming shapes of one wave per SIMD
    MLP2_ENTRY_WK(128, 64, 64, 1, 3, 1, 4, 128), MLP2_ENTRY_WK(32, 64, 128, 1, 3, 1, 4, 128),
    MLP2_ENTRY_WK(32, 64, 64, 1, 4, 1, 4, 128), MLP2_ENTRY_WK(64, 64, 64, 1, 4, 1, 4, 128),
};

static const Entry* find_entry(const KernelConfig& c) {
  for (const Entry& e : kEntries)
    if (e.bm == c.bm && e.bn1 == c.bn1 && e.bn2 == c.bn2 && e.nb == c.nb && e.ns == c.ns && e.waves == c.waves &&
        e.bk == c.bk && e.wnt == c.wnt)
      return &e;
  return nullptr;
}

// ------------------------------------------------------------------ GEMM chain
//
// An L-layer chain Z_l = act(Z_{l-1} W_l), Y = Z_{L-1} W_L: the producer /
// consumer relation of the two-layer kernel at every layer boundary (Sec.
// III-A).  An item is a T output tile of one layer over its whole K: 256 x
// 256 over eight waves with a two-stage ring for chains of many rows, 128 x
// 128 over four waves (two work-groups per CU), or 64 x 64 with four stages
// for chains of few rows, whose larger tiles would leave most CUs idle.
// A middle layer's item consumes like a GEMM2 item (it waits per K-slice on
// the ready counters of the layer below, row block mb) and produces like a
// GEMM1 item (activation, its Z rows stored, then its own ready counter
// released).  The one-launch rank table places every item after all the
// items it reads (plus a lag of about one grid), so the deadlock argument of
// the two-layer kernels holds unchanged: an item waits only for lower ranks,
// and a work-group takes its next ticket only after its current item's last
// wait.  The sequential mode launches each layer's items on their own, in
// layer order, without waits; both modes run this item function.
using ChainT128 = TileFor<128, 128, 2>::type;
using ChainT64 = TileFor<64, 64, 4>::type;
using ChainT256 = TileFor<256, 256, 2, 8>::type;
static_assert(ChainT128::NWAVES == 4 && ChainT64::NWAVES == 4 && ChainT256::NWAVES == 8, "chain tile waves");

template <class T>
__device__ __forceinline__ void chain_item(const ChainArgs& c, int layer, int tile, uint32_t epoch, char* lds,
                                           int* s_slot, Claim& next, int* s_next, TraceAcc& tr) {
  const Args& a = c.a;
  const ChainLayer& L = c.layer[layer];
  const int mb = tile % a.Mb, nb = tile / a.Mb;
  const int m0 = mb * T::BM, n0 = nb * T::BN;
  const int K = L.K;
  f32x4 acc[1][T::TN][T::TM];
  const uint16_t* Bp[1] = {L.W};
  if (c.wait && L.ready_in) {
    ReadyWait w{L.ready_in, a.ctrl + CTRL_ERROR, mb, a.Mb, T::BN, (K - 1) / T::BN, epoch + 1u, a.spin_limit, s_slot,
                0, &tr, T::BK};
    ClaimAtLastStage<ReadyWait> hook{w, &next, K - T::BK};
    mainloop<T, 1>(L.A, K, m0, L.alast, Bp, L.N, n0, 0, K, acc, lds, hook, tr);
  } else {
    NoWait nowait;
    ClaimAtLastStage<NoWait> hook{nowait, &next, K - T::BK};
    mainloop<T, 1>(L.A, K, m0, L.alast, Bp, L.N, n0, 0, K, acc, lds, hook, tr);
  }
  if constexpr (kTrace) tr_mark_mainloop(tr);
  next.park(s_next);
  FragPos<T> fp(m0, n0);
#pragma unroll
  for (int tm = 0; tm < T::TM; ++tm)
#pragma unroll
    for (int tp = 0; tp < T::TN / 2; ++tp) {
      float v[8];
      pair_values<T>(acc[0], tp, tm, v);
      if (L.act == ACT_GELU_TANH) {
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = gelu_tanh(v[i]);
      }
      const int row = fp.row0 + 16 * tm, col = fp.col0 + 32 * tp;
      if (!L.guard || row < a.M) *reinterpret_cast<u32x4*>(L.out + (long)row * L.N + col) = pack_bf16x8(v);
    }
  // Producer signal (one per tile and run): this tile's output rows are released.
  if (L.ready_out) signal_ready(L.ready_out + (long)tile * kLine);
}

// Four-wave tiles run two work-groups per CU, the eight-wave tile one.
template <class T>
__global__ __launch_bounds__(T::THREADS, T::NWAVES == 4 ? 2 : 1) void k_mlp2_chain(ChainArgs c) {
  __shared__ __attribute__((aligned(1024))) char lds[T::template lds_bytes<1>()];
  __shared__ int s_item, s_slot;
  const Args& a = c.a;
  const uint32_t epoch = uniform(ld_relaxed(a.ctrl + CTRL_EPOCH));
  const int total = a.items1;
  int p;
  {
    Claim first = make_claim(a, false);
    first.issue();
    first.park(&s_item);
    __syncthreads();
    p = uniform(s_item);
  }
  int n_items = 0;
  for (;;) {
    if (p >= total) break;
    __syncthreads();  // every wave has read s_item before the item's claim rewrites it
    TraceAcc tr;
    if constexpr (kTrace) tr.c_start = trace_clock();
    const uint64_t t_start = trace_now();
    Claim next = make_claim(a, false);
    const uint32_t e = uniform(a.orderp[p]);
    chain_item<T>(c, (int)(e >> 24), (int)(e & 0xffffffu), epoch, lds, &s_slot, next, &s_item, tr);
    // trace entry: layer << 24 | tile; every launch of a run records into section 0
    if constexpr (kTrace) tr_record(a, 0, n_items++, p, e, t_start, tr);
    __syncthreads();
    p = uniform(s_item);
  }
  finish_kernel(a, false, epoch, c.end_of_run != 0);
}

static const void* chain_kernel(int tile) {
  return tile == 0   ? (const void*)&k_mlp2_chain<ChainT128>
         : tile == 1 ? (const void*)&k_mlp2_chain<ChainT64>
                     : (const void*)&k_mlp2_chain<ChainT256>;
}

static int chain_threads(int tile) { return tile == 2 ? ChainT256::THREADS : ChainT128::THREADS; }

hipError_t chain_occupancy(int tile, int* blocks_per_cu) {
  if (tile < 0 || tile > 2) return hipErrorInvalidValue;
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, chain_kernel(tile), chain_threads(tile), 0);
}

hipError_t launch_chain(int tile, const ChainArgs& c, int grid, hipStream_t stream) {
  if (tile < 0 || tile > 2) return hipErrorInvalidValue;
  void* args[] = {const_cast<ChainArgs*>(&c)};
  return hipLaunchKernel(chain_kernel(tile), dim3(grid), dim3(chain_threads(tile)), args, 0, stream);
}

bool config_supported(const KernelConfig& c) { return find_entry(c) != nullptr; }

hipError_t occupancy(const KernelConfig& c, int which, int* blocks_per_cu) {
  const Entry* e = find_entry(c);
  if (!e) return hipErrorInvalidValue;
  const void* k = which == 0 ? e->seq1 : which == 1 ? e->seq2 : which == 2 ? e->pipe : which == 3 ? e->wq : e->sn;
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, k, 64 * e->waves, 0);
}

hipError_t launch_sequential(const KernelConfig& c, const Args& a1, const Args& a2, const int grids[2],
                             hipStream_t stream, int stages) {
  const Entry* e = find_entry(c);
  if (!e) return hipErrorInvalidValue;
  if (stages & 1) {
    void* args1[] = {const_cast<Args*>(&a1)};
    const hipError_t err = hipLaunchKernel(e->seq1, dim3(grids[0]), dim3(64 * e->waves), args1, 0, stream);
    if (err != hipSuccess) return err;
  }
  if (stages & 2) {
    void* args2[] = {const_cast<Args*>(&a2)};
    return hipLaunchKernel(e->seq2, dim3(grids[1]), dim3(64 * e->waves), args2, 0, stream);
  }
  return hipSuccess;
}

hipError_t launch_pipelined(const KernelConfig& c, const Args& a, int grid, hipStream_t stream) {
  const Entry* e = find_entry(c);
  if (!e) return hipErrorInvalidValue;
  void* args[] = {const_cast<Args*>(&a)};
  return hipLaunchKernel(e->pipe, dim3(grid), dim3(64 * e->waves), args, 0, stream);
}

hipError_t launch_workqueue(const KernelConfig& c, const Args& a, int grid, hipStream_t stream) {
  const Entry* e = find_entry(c);
  if (!e) return hipErrorInvalidValue;
  void* args[] = {const_cast<Args*>(&a)};
  return hipLaunchKernel(e->wq, dim3(grid), dim3(64 * e->waves), args, 0, stream);
}

hipError_t launch_sentinel(const KernelConfig& c, const Args& a, int grid, hipStream_t stream) {
  const Entry* e = find_entry(c);
  if (!e) return hipErrorInvalidValue;
  void* args[] = {const_cast<Args*>(&a)};
  return hipLaunchKernel(e->sn, dim3(grid), dim3(64 * e->waves), args, 0, stream);
}

}  // namespace mlp2
