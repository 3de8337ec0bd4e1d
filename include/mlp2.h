/*
 * mlp2.h - C ABI of the tile-pipelined two-layer MLP for AMD MI355X (gfx950).
 *
 * The operation is the two-layer product that CTA-pipelining (arXiv
 * 2607.07862) uses as its workload (Sec. IV: Y = X A B standing for an LLM MLP
 * layer), with an activation between the layers:
 *
 *     Z = act(X . W1)        first GEMM, fused activation epilogue
 *     Y = Z . W2             second GEMM
 *
 * Three execution modes compute bit-identical Y:
 *   MLP2_MODE_SEQUENTIAL      GEMM1 then GEMM2, two kernels on the stream.
 *   MLP2_MODE_TILE_PIPELINED  one persistent launch; a GEMM2 work-group
 *                             consumes each K-slice of Z as soon as the GEMM1
 *                             tiles producing it have signalled a per-tile
 *                             ready counter (Sec. III-A: producer epilogue
 *                             fences, then signals; consumer prologue polls;
 *                             Sec. III-A.5 host organisation; Sec. III-B.2
 *                             persistent kernels fetching work tiles).
 *   MLP2_MODE_WORKQUEUE       one persistent launch with the paper's own
 *                             consumer scheduling (Sec. III-A.2-3): each
 *                             completed GEMM1 tile counts down the scoreboard
 *                             of every GEMM2 unit that reads it, the producer
 *                             completing a unit pushes it onto a device
 *                             ring-buffer workqueue, and work-groups that run
 *                             out of GEMM1 items pop whole units from it.
 *
 * Data layout (all device memory, row-major, bf16, 16-byte aligned):
 *   X   [M, H]            input activations             (caller owns)
 *   W1  [H, F]            first weight                  (caller owns)
 *       [2, H, F]         SwiGLU: Wg then Wu, packed    (caller owns)
 *   W2  [F, H]            second weight                 (caller owns)
 *   Y   [M, H]            output, fully overwritten     (caller owns)
 * Arithmetic: bf16 inputs, fp32 accumulation, fp32 activation, the
 * intermediate Z stored as bf16 (round to nearest even), bf16 output
 * (Sec. III-C and Sec. IV fix bf16 in/out with fp32 accumulation).
 *
 * Activations: identity; GELU tanh form 0.5 z (1 + tanh(sqrt(2/pi)(z + 0.044715 z^3)));
 * SwiGLU silu(X.Wg) * (X.Wu) with silu(g) = g / (1 + exp(-g)).
 *
 * The mlp2_chain_* entry points at the end run the same protocol over a
 * chain of L GEMMs (Z_l = act(Z_{l-1} . W_l), Y = Z_{L-1} . W_L), where the
 * middle layers both consume and produce.
 *
 * Error behaviour: every entry point validates its arguments on the host
 * before it enqueues anything; a failing call has no side effect and returns
 * a negative MLP2_ERR_* code (mlp2_plan returns NULL and records the code for
 * mlp2_last_error()).  Device-side failures (a bounded flag wait that timed
 * out) are latched in the plan and reported by mlp2_check().
 *
 * Threading: a plan may be used from one host thread at a time and must not
 * be run concurrently on two streams (its workspace is shared).  Different
 * plans are independent.
 */
#ifndef MLP2_H
#define MLP2_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct mlp2_plan_s* mlp2_plan_t; /* opaque; created by mlp2_plan, freed by mlp2_destroy */

enum mlp2_act { MLP2_ACT_IDENTITY = 0, MLP2_ACT_GELU_TANH = 1, MLP2_ACT_SWIGLU = 2 };
enum mlp2_dtype { MLP2_DTYPE_BF16 = 0 };
/* MLP2_MODE_SENTINEL is the pipelined launch with the Lamport-style
 * synchronisation the paper discusses as an alternative (Sec. V-A): GEMM1
 * tiles store the intermediate at device scope with no fence and no ready
 * counter, and GEMM2 work-groups re-read each K-slice of it while any element
 * still holds a sentinel (the bf16 pattern 0xFFFF, which the epilogue never
 * writes: it turns that NaN into 0x7FC0 in every mode).  The plan keeps two
 * intermediates for it that alternate run by run, each run refilling the other
 * with sentinels tile by tile, so no run pre-fills a whole buffer.  Same
 * results as the other modes, bit for bit.  Not for plans run in row groups
 * (MLP2_ERR_UNSUPPORTED).
 *
 * MLP2_MODE_STAGE1 / MLP2_MODE_STAGE2 enqueue the first or the second kernel
 * of the sequential mode alone, for callers that schedule the two stages
 * themselves (e.g. a micro-batch pipeline over chunks of rows on two streams,
 * one plan per chunk).  The caller orders a plan's STAGE2 after its STAGE1
 * (same stream, or an event), and the pair after the plan's previous run:
 * every STAGE1 is followed by its STAGE2 before the plan runs again (the
 * device epoch advances with STAGE2, so two STAGE1 runs in a row leave the
 * split-K arrival counts past their targets).  Together they compute what
 * MLP2_MODE_SEQUENTIAL computes, bit for bit.
 * Not for plans run in row groups (MLP2_ERR_UNSUPPORTED). */
enum mlp2_mode {
  MLP2_MODE_SEQUENTIAL = 0,
  MLP2_MODE_TILE_PIPELINED = 1,
  MLP2_MODE_WORKQUEUE = 2,
  MLP2_MODE_STAGE1 = 3,
  MLP2_MODE_STAGE2 = 4,
  MLP2_MODE_SENTINEL = 5
};

enum mlp2_status {
  MLP2_OK = 0,
  MLP2_ERR_INVALID_ARG = -1, /* null plan/pointer, bad enum, non-positive size, aliasing Y */
  MLP2_ERR_UNSUPPORTED = -2, /* sizes outside the supported range (H, F multiples of 64) */
  MLP2_ERR_ALIGNMENT = -3,   /* a data pointer not 16-byte aligned */
  MLP2_ERR_HIP = -4,         /* a HIP runtime call failed (allocation, launch) */
  MLP2_ERR_TIMEOUT = -5,     /* a bounded flag wait on the device gave up (see mlp2_check) */
  MLP2_ERR_DEVICE = -6       /* no usable gfx950 device, or the plan belongs to another device */
};

/* GEMM1 tile-ordering policies (Sec. III-A.5: the first kernel may take its
 * tiles from a predefined source order).  The base order is column-first:
 * whole column blocks of Z first, so GEMM2's K-slices complete in order, and
 * the row blocks of one column block (which share its weight columns) run
 * together.  The default refines it for plans with several row blocks and no
 * split-K: ranks r, r + 8, ... run on one XCD, and each wave of the grid's
 * worth of tiles (still whole column blocks) is dealt to the 8 XCDs as
 * near-square sub-blocks, so the operand slices a stage reads are shared
 * inside each XCD's L2; the GEMM2 kernel's items are dealt the same way.
 * With many row blocks whose activation and first weights exceed the 256 MB
 * last-level cache, the default is MLP2_ORDER_BANDED instead, and the
 * pipelined launch then places every GEMM2 item after every GEMM1 item
 * (overlapping only the tail): a band's GEMM2 items could start beside the
 * next band's GEMM1 items, but both weight matrices streaming at once no
 * longer fit that cache.  (Row-block-first halves, which let some GEMM2
 * items start before GEMM1 ends, measured slower at prefill size.) */
enum mlp2_order {
  MLP2_ORDER_AUTO = 0,         /* the default: row bands for many row blocks whose X and W1
                                  exceed the last-level cache; else XCD-grouped column-first
                                  with several row blocks and no split-K; else column-first    */
  MLP2_ORDER_COLUMN_FIRST = 1, /* every row block of column block 0, then column block 1, ... */
  MLP2_ORDER_ROW_FIRST = 2,    /* every column block of row block 0, then row block 1, ...    */
  MLP2_ORDER_REVERSED = 3,     /* column-first, last column block first (stress order)         */
  MLP2_ORDER_SHUFFLED = 4,     /* a seeded permutation (stress order)                          */
  MLP2_ORDER_BANDED = 5        /* bands of about a grid's worth of row blocks, all column blocks
                                  of a band before the next (both kernels); for many row blocks,
                                  where a wave of whole column blocks reads all of X             */
};

/* Optional tuning for mlp2_plan_ex; a zero field means "choose automatically". */
typedef struct mlp2_tuning {
  int bm;        /* row-block height shared by both GEMMs: 32, 64, 128 or 256            */
  int bn1;       /* GEMM1 column-block width (= GEMM2 K-slice granularity): 64, 128 or 256*/
  int splitk1;   /* GEMM1 split-K factor (>= 1)                                           */
  int bn2;       /* GEMM2 column-block width: 64, 128 or 256                              */
  int splitk2;   /* GEMM2 split-K factor (>= 1)                                           */
  int grid;      /* persistent grid of every launch (no more work-groups than fit the
                    device at once)                                                      */
  int order;     /* enum mlp2_order (0 = MLP2_ORDER_AUTO)                                 */
  int stages;    /* LDS ring depth of the tile mainloop (2, 3 or 4, as built for the shape)*/
  int row_group; /* rows per launch group: 0 = automatic (groups once Z of all rows exceeds
                    the 256 MB last-level cache), -1 = one launch over all rows, else a
                    multiple of 256 (groups of that many rows, the last one shorter)      */
  int waves;     /* 64-wide waves per work-group: 4 or 8 (as built for the tile shape)     */
  int lag;       /* pipelined mode, shared roles: ranks between a GEMM2 item and the last
                    GEMM1 item it reads in the claim order; 0 = automatic (one grid),
                    -1 = every GEMM2 item after every GEMM1 item                          */
  int p1;        /* pipelined mode: 0 = shared roles (every work-group takes both kinds of
                    item from one rank order); else work-groups with index g % 64 < p1
                    take only GEMM1 items and the others only GEMM2 items (a static
                    producer / consumer split of the grid, p1 in 1..63 of every 64)       */
  int bk;        /* K depth of one LDS stage: 64, 32 or 128 (as built for the shape; 128   */
                 /* only where H and F are multiples of 128)                               */
  int weights_nt; /* weight loads with the non-temporal hint: 0 = automatic (on when W1 and
                     W2 together exceed the 256 MiB last-level cache and the tile is built
                     with it), 1 = on (refused where not built), -1 = off                 */
} mlp2_tuning_t;

/* What a plan chose, for reports and tests. */
typedef struct mlp2_info {
  int64_t M, H, F;
  int act;
  int bm, bn1, splitk1, bn2, splitk2, bk;
  int row_blocks;        /* ceil(M / bm)                                    */
  int col_blocks1;       /* F / bn1                                         */
  int col_blocks2;       /* H / bn2                                         */
  int items1, items2;    /* GEMM1 / GEMM2 split items (tiles x splitk)       */
  int grid_pipelined;    /* persistent work-groups of the pipelined launch  */
  int occupancy;         /* resident work-groups per CU of that kernel      */
  int num_cus;
  int order;
  int64_t workspace_bytes;
  uint32_t spin_limit;
  int stages;            /* LDS ring depth                                  */
  int grid_gemm1;        /* persistent work-groups of the GEMM1 launch      */
  int grid_gemm2;        /* persistent work-groups of the GEMM2 launch      */
  int row_group;         /* rows per launch group (0: one launch over all rows);
                            the tile fields above are those of a whole group */
  int waves;             /* 64-wide waves per work-group                    */
  int lag;               /* pipelined rank-table lag in ranks (shared roles) */
  int p1;                /* static GEMM1 share of every 64 work-groups (0: shared roles) */
  int weights_nt;        /* 1: the weight loads carry the non-temporal hint  */
} mlp2_info_t;

/* Create a plan for Y[M,H] = act(X[M,H] . W1) . W2 on the current HIP device.
 * Requires 1 <= M <= 1<<20, H and F multiples of 64 in [64, 1<<18], act in
 * enum mlp2_act and dtype == MLP2_DTYPE_BF16, and every operand one launch
 * reads (X or a row group's X, Z, each weight matrix) below 4 GB: the loads
 * address an operand with 32-bit byte offsets (MLP2_ERR_UNSUPPORTED otherwise).  Allocates the workspace (the
 * bf16 intermediate Z, split-K partials, counters) on the current device.
 * Returns NULL on failure; mlp2_last_error() gives the code. */
mlp2_plan_t mlp2_plan(int64_t M, int64_t H, int64_t F, int act, int dtype);

/* As mlp2_plan with explicit tuning (NULL = automatic).  Invalid tuning
 * (a tile that does not divide H or F, bm not in the list, ...) fails with
 * MLP2_ERR_UNSUPPORTED. */
mlp2_plan_t mlp2_plan_ex(int64_t M, int64_t H, int64_t F, int act, int dtype, const mlp2_tuning_t* tuning);

/* Enqueue one evaluation on `stream` (a hipStream_t; NULL = the default
 * stream) in `mode`.  Asynchronous: no host synchronisation, no allocation.
 * X, W1, W2, Y are device pointers laid out as described above; Y must not
 * overlap any input.  Runs of one plan on one stream are ordered; the plan
 * keeps its counters consistent across runs and modes without host resets.
 * A plan with row groups (mlp2_info_t.row_group > 0) enqueues the mode's
 * launches once per group of rows, in row order; rows do not interact, and
 * every mode uses the same groups, so the modes still agree bit for bit. */
int mlp2_run(mlp2_plan_t plan, const void* X, const void* W1, const void* W2, void* Y, void* stream, int mode);

/* Free the plan and its workspace.  NULL-safe.  It first waits for all work on
 * the plan's device: the plan does not record which streams ran it, and no
 * kernel of it may still use the workspace when it is freed. */
void mlp2_destroy(mlp2_plan_t plan);

/* Code of the last failing call on this host thread (MLP2_OK if none). */
int mlp2_last_error(void);

/* A static, never-NULL description of a status code. */
const char* mlp2_strerror(int code);

/* After the caller has synchronised the stream: MLP2_OK, or MLP2_ERR_TIMEOUT
 * if a flag wait gave up during an earlier run.  On a timeout it clears the
 * latched error and resets the plan's counters so the plan is usable again
 * (the reset runs on the null stream, and the call waits for that stream
 * only). */
int mlp2_check(mlp2_plan_t plan);

/* Fill *out with what the plan chose. */
int mlp2_plan_info(mlp2_plan_t plan, mlp2_info_t* out);

/* Device pointer to the plan's bf16 intermediate Z, laid out [row_blocks*bm, F]
 * row-major (rows >= M are padding; with row groups, Z of every group at its
 * rows).  Valid until mlp2_destroy.  For tests and
 * diagnostics; NULL on a NULL plan. */
const void* mlp2_intermediate(mlp2_plan_t plan);

/* Debug and failure-injection knobs (tests only).  Keys:
 *   MLP2_OPT_SPIN_LIMIT   polls before a flag wait gives up (default ~1 s of polling)
 *   MLP2_OPT_DROP_SIGNAL  GEMM1 tile index whose ready signal is skipped (-1 = none); in the
 *                         sentinel mode the tile's intermediate stores are skipped instead
 *   MLP2_OPT_ORDER        enum mlp2_order (rebuilds the order table)
 *   MLP2_OPT_GRID         persistent grid of every launch (0 = automatic; else
 *                         at most the work-groups that fit the device at once)
 * Returns MLP2_OK or MLP2_ERR_INVALID_ARG. */
enum mlp2_option { MLP2_OPT_SPIN_LIMIT = 1, MLP2_OPT_DROP_SIGNAL = 2, MLP2_OPT_ORDER = 3, MLP2_OPT_GRID = 4 };
int mlp2_set_option(mlp2_plan_t plan, int key, int64_t value);

/* Per-item timing trace (diagnostics).  Only a library built with the
 * MLP2_TRACE macro records; an ordinary build returns MLP2_ERR_UNSUPPORTED
 * and its kernels carry no trace code.  `buffer` is caller-owned device
 * memory (8-byte aligned, NULL detaches) that later runs of the plan fill:
 * for section s (0 = the GEMM1 kernel or the pipelined kernel, 1 = the GEMM2
 * kernel of the sequential mode) and work-group g of that launch, the block
 * at uint64 offset (s * G + g) * (1 + 8 * records_per_group) holds the
 * item count, then one record per item of 8 uint64: the item's rank (high
 * 32 bits) and its order-table entry (low 32 bits: the GEMM1 item id
 * tile * S1 + s, or for a GEMM2 item 0x80000000 | (tile * S2 + s)), start,
 * mainloop end, two epilogue marks, end (times on the 100 MHz device
 * real-time counter; the marks are: for a GEMM1 tile that signals, its Z
 * stores complete and its ready counter released; for a split-K part that
 * does not complete its tile, its partial stored and its arrival counted;
 * 0 and 0 otherwise), the item's core clock cycles (shader-clock counter,
 * high 32 bits) above its ticks waiting for the tile loads of the
 * work-group's own ring (low 32 bits), ticks waiting for ready counters and
 * split-K siblings.  Items beyond records_per_group are counted, not stored.
 * G is the largest of the plan's grids (grid_pipelined, grid_gemm1,
 * grid_gemm2 of mlp2_plan_info; with row groups the records are those of
 * the last whole group's launches, the shorter last group records nothing); the buffer must hold
 * 2 * G * (1 + 8 * records_per_group) words.  Returns MLP2_OK, MLP2_ERR_INVALID_ARG
 * or MLP2_ERR_UNSUPPORTED. */
int mlp2_trace_attach(mlp2_plan_t plan, void* buffer, int records_per_group);

/* ---- Allocation-free run (for callers that cannot allocate device memory:
 * code under graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Plans and enqueues one evaluation of Y = act(X . W1) . W2 in
 * `mode` on `stream`, exactly as mlp2_plan + mlp2_run would with the
 * column-first tile order and every GEMM2 item after every GEMM1 item in the
 * pipelined rank table (mode: sequential, tile_pipelined or workqueue), and
 * calls no allocating routine: every piece of
 * workspace (Z, split-K partials, counters, rank tables) lives in a static
 * device array of 64 MiB that the library holds on each GPU it runs on until
 * the process ends.  Arguments and layouts as mlp2_plan / mlp2_run (device
 * pointers, row-major bf16, 16-byte aligned; the caller owns X, W1, W2, Y).
 * Returns MLP2_OK once enqueued; MLP2_ERR_UNSUPPORTED when the plan's
 * workspace exceeds the 64 MiB (e.g. the 70B gated MLP at 256 rows or a
 * prefill batch: use mlp2_plan for those), and the codes of mlp2_plan and
 * mlp2_run otherwise; mlp2_last_error() records the code.  Every call on a
 * device shares that device's array and starts by clearing its counters (a
 * small fill kernel on `stream`, no memset node), so calls that overlap on one
 * device (two streams or two host threads) race and give undefined results.
 * A flag wait that times out is not reported here (there is no plan to check):
 * the kernels still exit, and mlp2_run + mlp2_check diagnose such a case. */
int mlp2_run_noalloc(int64_t M, int64_t H, int64_t F, int act, int dtype, const void* X, const void* W1,
                     const void* W2, void* Y, void* stream, int mode);

/* ---- GEMM chain: the producer / consumer relation at every layer boundary
 * (Sec. III-A applied to a chain of GEMMs whose middle kernels both consume
 * and produce).  Z_0 = X [M, D_0]; Z_l = act(Z_{l-1} . W_l) for l < L;
 * Y = Z_{L-1} . W_L [M, D_L].  W_l is [D_{l-1}, D_l] row-major bf16; fp32
 * accumulation; the intermediates are stored as bf16 in the plan's
 * workspace.  Items are output tiles over their whole K: 256 x 256 (eight
 * waves) when every width D_1 .. D_L is a multiple of 256 and the narrowest
 * layer has a 256-row tile per CU, else 128 x 128, or 64 x 64 when the
 * narrowest layer would have fewer 128-row tiles than CUs; each layer's
 * tiles are dealt to the XCDs in sub-blocks of rows and columns.  Chains of
 * many rows run as back-to-back launches over row groups of about 2.2 T
 * multiply-adds each (once the rows reach two groups; rows do not interact,
 * so the result is that of one launch). */
typedef struct mlp2_chain_s* mlp2_chain_t; /* opaque; created by mlp2_chain_plan, freed by mlp2_chain_destroy */

/* Plan an L-layer chain on the current device.  dims holds L + 1 widths
 * D_0 .. D_L (host array, read during the call), each a multiple of 128 in
 * [128, 65536]; 1 <= L <= 8; 1 <= M <= 1<<20; X, every intermediate and
 * every weight below 4 GB per launch (32-bit load offsets); act is MLP2_ACT_IDENTITY or
 * MLP2_ACT_GELU_TANH (applied after every layer but the last); dtype
 * MLP2_DTYPE_BF16.  Allocates the intermediates, ready counters and rank
 * tables.  NULL on failure (mlp2_last_error: MLP2_ERR_INVALID_ARG for null or
 * non-positive arguments and other activations, MLP2_ERR_UNSUPPORTED for
 * sizes outside the ranges, MLP2_ERR_DEVICE, MLP2_ERR_HIP). */
mlp2_chain_t mlp2_chain_plan(int64_t M, int layers, const int64_t* dims, int act, int dtype);

/* Enqueue one evaluation on `stream` (a hipStream_t; NULL = the default
 * stream).  X, Y: device pointers ([M, D_0] and [M, D_L], 16-byte aligned; Y
 * must not overlap X or a weight); W: host array of L device pointers to the
 * weights (read during the call).  MLP2_MODE_SEQUENTIAL launches each
 * layer's items after the previous layer's launch; MLP2_MODE_TILE_PIPELINED
 * runs every layer in one persistent launch, each tile starting once the
 * tiles of the layer below that it reads have signalled.  Both modes give
 * the same bits.  Asynchronous; no allocation; runs of one plan on one
 * stream are ordered.  Returns MLP2_OK or MLP2_ERR_INVALID_ARG (also for
 * MLP2_MODE_WORKQUEUE), MLP2_ERR_ALIGNMENT, MLP2_ERR_DEVICE, MLP2_ERR_HIP. */
int mlp2_chain_run(mlp2_chain_t plan, const void* X, const void* const* W, void* Y, void* stream, int mode);

/* As mlp2_check, for a chain plan (after the caller has synchronised). */
int mlp2_chain_check(mlp2_chain_t plan);

/* Polls before a flag wait of a later run gives up (tests of the failure
 * path); MLP2_ERR_INVALID_ARG outside 1 .. 2^32 - 1. */
int mlp2_chain_set_spin_limit(mlp2_chain_t plan, int64_t polls);

/* Persistent work-groups of the chain's one-launch mode (of a whole row
 * group's launch with row groups); 0 for a NULL plan. */
int mlp2_chain_grid(mlp2_chain_t plan);

/* Per-item timing records of a chain plan (trace builds only; otherwise
 * MLP2_ERR_UNSUPPORTED), as mlp2_trace_attach with G = mlp2_chain_grid:
 * every launch of a run records into section 0 (the sequential mode's
 * per-layer launches one after another, so its buffer holds the last
 * layer's); an entry's low 32 bits are layer << 24 | tile; with row groups
 * the last whole group's launches record. */
int mlp2_chain_trace_attach(mlp2_chain_t plan, void* buffer, int records_per_group);

/* Free the chain plan and its workspace (synchronises the device first).  NULL-safe. */
void mlp2_chain_destroy(mlp2_chain_t plan);

#ifdef __cplusplus
}
#endif

#endif /* MLP2_H */
