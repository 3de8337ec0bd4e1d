// C ABI of the tile-pipelined two-layer MLP: planning, validation, launch.
//
// The plan fixes everything that does not change between runs (tile sizes,
// split-K factors, the GEMM1 order table, the persistent grid, the workspace)
// so that mlp2_run only validates pointers and enqueues kernels: no
// allocation, no host synchronisation, no memset (graph-capture safe).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <numeric>
#include <random>
#include <string>
#include <vector>

#include "../../include/mlp2.h"
#include "mlp2_launch.h"
#include "mlp2_plan_impl.h"

using mlp2::Args;
using mlp2::KernelConfig;

struct mlp2_chain_s {
  int64_t M = 0;
  int L = 0;
  int64_t dims[mlp2::kChainMaxLayers + 1] = {};
  int act = 0;
  int device = -1;
  int num_cus = 0;
  int tile = 0;                           // chain tile shape (index into kChainTiles)
  int bt = 0;                             // its rows and columns
  int Mb = 0;
  int items[mlp2::kChainMaxLayers] = {};  // tiles per layer: Mb * D_l / bt
  int total = 0;
  int grid = 0;
  uint32_t spin_limit = 1u << 20;
  void* ws = nullptr;
  size_t ws_bytes = 0;
  uint16_t* Z[mlp2::kChainMaxLayers] = {};        // output of layer l < L - 1, [Mb * 128, D_{l+1}]
  uint32_t* ready[mlp2::kChainMaxLayers] = {};    // ready counters of layer l < L - 1
  uint32_t* ctrl = nullptr;
  uint32_t* order_seq = nullptr;  // layer l's tiles at offset seq_off[l], column blocks first
  uint32_t* order_pipe = nullptr; // every item of every layer, after its producers
  int seq_off[mlp2::kChainMaxLayers] = {};
  size_t counters_off = 0, counters_bytes = 0;
  uint64_t* trace = nullptr;  // caller-owned timing buffer (trace builds)
  int trace_cap = 0;
  // Row groups (chain_group_rows): launches over whole groups of group_rows
  // rows (`group`) and over the remaining rows (`tail`), in row order.
  int64_t group_rows = 0;
  mlp2_chain_s* group = nullptr;
  mlp2_chain_s* tail = nullptr;
};

namespace {

thread_local int g_last_error = MLP2_OK;

int fail(int code) {
  g_last_error = code;
  return code;
}

}  // namespace

namespace mlp2 {
int record_error(int code) { return fail(code); }
}  // namespace mlp2

namespace {

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

int ceil_div(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

// Claim lists of a launch: one per XCD (8), or one per work-group for grids
// below 8, so that every list has a work-group.
int claim_lists(int grid) { return std::min(8, std::max(1, grid)); }

// Work-groups of the GEMM1 role in a pipelined launch of `grid` work-groups
// split with share p1 of every 64 (those with index g % 64 < p1).
int role1_groups(int p1, int grid) { return grid / 64 * p1 + std::min(grid % 64, p1); }

// A role split leaves work-groups in both roles (no split: always true).
bool roles_ok(int p1, int grid) {
  if (p1 == 0) return true;
  const int n1 = role1_groups(p1, grid);
  return n1 >= 1 && grid - n1 >= 1;
}

// Split K into S ranges of kc (a multiple of the stage depth): as many parts
// as keep the tile count times S within `want` items (one round of the
// persistent grid), each range at least `min_k` deep.  Returns S and sets *kc.
int choose_split(int64_t K, int tiles, int want, int min_k, int gran, int* kc) {
  int S = std::max(1, want / std::max(1, tiles));
  S = std::min<int64_t>(S, std::max<int64_t>(1, K / min_k));
  int64_t k = align_up((size_t)ceil_div(K, S), gran);
  *kc = (int)k;
  return ceil_div(K, k);
}

// XCD-grouped order of an Mb x N tile grid (tile = nb * Mb + mb), for plans
// with several row blocks.  A launch deals rank r to the work-groups of claim
// list r % 8, which all sit on XCD r % 8 (work-groups are dispatched to the 8
// XCDs round-robin), so the tiles at ranks x, x + 8, ... share XCD x's L2.
// Consecutive waves of `wave` tiles cover whole column blocks (every row
// block of C columns, so column blocks still complete in order); each wave
// is cut into 8 sub-blocks as close to square as the divisors of 8 allow, one
// per XCD, walked column-first.  Every stage of a wave then reads rows + cols
// distinct operand slices per XCD instead of (rows of the XCD) + C: an 8 x 8
// sub-block reads 16 slices where the plain column-first deal reads 2 + 32.
std::vector<uint32_t> xcd_grouped(int Mb, int N, int wave) {
  constexpr int kXcds = 8;
  std::vector<uint32_t> out;
  out.reserve((size_t)Mb * N);
  const int C = std::max(1, wave / Mb);
  std::vector<uint32_t> per[kXcds];
  for (int c0 = 0; c0 < N; c0 += C) {
    const int cw = std::min(C, N - c0);
    int best_r = 1, best_cost = INT32_MAX;
    for (int r = 1; r <= kXcds && r <= Mb; r *= 2) {
      const int cost = ceil_div(Mb, r) + ceil_div(cw, kXcds / r);
      if (cost < best_cost) { best_cost = cost; best_r = r; }
    }
    const int rows = ceil_div(Mb, best_r), cols = ceil_div(cw, kXcds / best_r);
    for (int x = 0; x < kXcds; ++x) {
      per[x].clear();
      const int rg = x % best_r, cg = x / best_r;
      for (int nb = c0 + cg * cols; nb < std::min(c0 + cw, c0 + (cg + 1) * cols); ++nb)
        for (int mb = rg * rows; mb < std::min(Mb, (rg + 1) * rows); ++mb) per[x].push_back((uint32_t)(nb * Mb + mb));
    }
    // Deal the wave: its j-th group of 8 ranks takes the j-th tile of every
    // sub-block; once a sub-block runs out (ragged edges), the rest close up.
    for (size_t j = 0;; ++j) {
      bool any = false;
      for (int x = 0; x < kXcds; ++x)
        if (j < per[x].size()) { out.push_back(per[x][j]); any = true; }
      if (!any) break;
    }
  }
  return out;
}

// Row bands: `band` consecutive row blocks with all their column blocks,
// band after band, each band dealt to the XCDs as xcd_grouped deals a grid.
// A band reads its rows of the activation once while the weights stay in the
// last-level cache, and the GEMM2 items of a band depend on that band only.
std::vector<uint32_t> banded(int Mb, int N, int wave, int band) {
  std::vector<uint32_t> out;
  out.reserve((size_t)Mb * N);
  for (int r0 = 0; r0 < Mb; r0 += band) {
    const int rb = std::min(band, Mb - r0);
    for (uint32_t t : xcd_grouped(rb, N, wave)) {
      const int nb = (int)t / rb, mb = (int)t % rb;
      out.push_back((uint32_t)(nb * Mb + r0 + mb));
    }
  }
  return out;
}

// Row blocks per band: about one wave of the grid's tiles.
int band_rows(int N, int wave) { return std::max(1, wave / std::max(1, N)); }

// Whether the plan's GEMM1 order is row bands: explicitly, or by default once
// X and W1 together exceed the 256 MB last-level cache with many row blocks
// (measured at 8192 x 8192 weights: from 16384 rows on; at 32768 rows bands
// take the sequential mode from 12.7 to 9.0 ms).
bool uses_bands(const mlp2_plan_s* p) {
  if (p->S1 != 1) return false;
  if (p->order == MLP2_ORDER_BANDED) return true;
  const int64_t nb = p->act == MLP2_ACT_SWIGLU ? 2 : 1;
  const int64_t x_w1 = (int64_t)p->M * p->H * 2 + nb * p->H * p->F * 2;
  return p->order == MLP2_ORDER_AUTO && p->Mb >= 32 && x_w1 > (int64_t)256 << 20;
}

// GEMM1 item order (the rank order of the GEMM1 kernel, and of the GEMM1
// items within the pipelined kernel).  Items are id = tile * S1 + s with
// tile = nb * Mb + mb; every policy orders tiles and keeps the S1 parts of a
// tile adjacent.  MLP2_ORDER_AUTO is the XCD-grouped column-first order when
// there are several row blocks and no split-K, else plain column-first.
void build_order(mlp2_plan_s* p, std::vector<uint32_t>& out) {
  std::vector<uint32_t> tiles;
  tiles.reserve((size_t)p->Mb * p->Nb1);
  auto tile = [&](int nb, int mb) { tiles.push_back((uint32_t)(nb * p->Mb + mb)); };
  switch (p->order) {
    case MLP2_ORDER_ROW_FIRST:
      for (int mb = 0; mb < p->Mb; ++mb)
        for (int nb = 0; nb < p->Nb1; ++nb) tile(nb, mb);
      break;
    case MLP2_ORDER_REVERSED:
      for (int nb = p->Nb1 - 1; nb >= 0; --nb)
        for (int mb = 0; mb < p->Mb; ++mb) tile(nb, mb);
      break;
    case MLP2_ORDER_BANDED:
    case MLP2_ORDER_AUTO:
      if (uses_bands(p)) {
        tiles = banded(p->Mb, p->Nb1, p->grid1, band_rows(p->Nb1, p->grid1));
        break;
      }
      if (p->Mb > 1 && p->S1 == 1 && p->order == MLP2_ORDER_AUTO) {
        tiles = xcd_grouped(p->Mb, p->Nb1, p->grid1);
        break;
      }
      [[fallthrough]];
    default:  // MLP2_ORDER_COLUMN_FIRST, and the base of the shuffled order
      for (int nb = 0; nb < p->Nb1; ++nb)
        for (int mb = 0; mb < p->Mb; ++mb) tile(nb, mb);
      if (p->order == MLP2_ORDER_SHUFFLED) {
        std::mt19937 rng(12345u);
        std::shuffle(tiles.begin(), tiles.end(), rng);
      }
      break;
  }
  out.clear();
  out.reserve(tiles.size() * p->S1);
  for (uint32_t t : tiles)
    for (int s = 0; s < p->S1; ++s) out.push_back(t * (uint32_t)p->S1 + (uint32_t)s);
}

// GEMM2 item order (ranks of the GEMM2 kernel; GEMM2 items of the pipelined
// table are placed in this order among equal keys): XCD-grouped under
// MLP2_ORDER_AUTO with several row blocks and no split-K, else item order
// (q = tile * S2 + s, tile = nb * Mb + mb).  No GEMM2 item waits in the
// GEMM2 kernel, so any order is valid there.
void build_order2(const mlp2_plan_s* p, std::vector<uint32_t>& out) {
  if (uses_bands(p) && p->S2 == 1) {  // the GEMM1 bands' rows, band by band
    const std::vector<uint32_t> t = banded(p->Mb, p->Nb2, p->grid2, band_rows(p->Nb1, p->grid1));
    out.assign(t.begin(), t.end());
    return;
  }
  if (p->order == MLP2_ORDER_AUTO && p->Mb > 1 && p->S2 == 1) {
    out = xcd_grouped(p->Mb, p->Nb2, p->grid2);
    return;
  }
  out.resize((size_t)p->items2);
  for (int q = 0; q < p->items2; ++q) out[(size_t)q] = (uint32_t)q;
}

// Rank table of the pipelined kernel: the GEMM1 items keep their order; GEMM2
// item q = tile * S2 + s goes right after rank h(q) + lag (after every GEMM1
// item, in the GEMM2 order table's sequence, when lag >= items1), where h(q)
// is the highest GEMM1 rank among the tiles its K range reads.  Every GEMM2 item thus
// ranks above every GEMM1 item it waits for (what the deadlock argument
// needs), and is claimed about `lag` claims after its last producer.
void build_merged(const mlp2_plan_s* p, const std::vector<uint32_t>& order1, const std::vector<uint32_t>& order2, int lag,
                  std::vector<uint32_t>& out) {
  std::vector<int64_t> last_rank((size_t)p->Mb * p->Nb1, -1);
  for (size_t r = 0; r < order1.size(); ++r) {
    const uint32_t t = order1[r] / (uint32_t)p->S1;
    last_rank[t] = std::max<int64_t>(last_rank[t], (int64_t)r);
  }
  struct Key {
    int64_t key;
    int kind;  // 0 = GEMM1, 1 = GEMM2
    uint32_t id;
  };
  std::vector<Key> keys;
  keys.reserve(order1.size() + (size_t)p->items2);
  for (size_t r = 0; r < order1.size(); ++r) keys.push_back({(int64_t)r, 0, order1[r]});
  for (const uint32_t q2 : order2) {
    const int q = (int)q2;
    const int tile = q / p->S2, s = q % p->S2;
    const int mb = tile % p->Mb;
    const int64_t kbeg = (int64_t)s * p->kc2, kend = std::min<int64_t>(p->F, kbeg + p->kc2);
    int64_t h = -1;
    for (int64_t kb = kbeg / p->kc.bn1; kb <= (kend - 1) / p->kc.bn1; ++kb) h = std::max(h, last_rank[kb * p->Mb + mb]);
    // With a lag of the whole GEMM1 list (row bands) every GEMM2 item gets the
    // key items1: they all follow GEMM1 in the GEMM2 order table's sequence
    // (its bands and XCD deal) instead of being sorted by their last
    // producer.  Otherwise the key keeps the order in which producers finish
    // (e.g. split-K parts whose producers end a round apart).  Every item
    // still ranks above its producers.
    const int64_t n1 = (int64_t)order1.size();
    keys.push_back({lag >= n1 ? n1 : h + lag, 1, (uint32_t)q});
  }
  std::stable_sort(keys.begin(), keys.end(), [](const Key& a, const Key& b) {
    return a.key != b.key ? a.key < b.key : a.kind < b.kind;
  });
  out.clear();
  out.reserve(keys.size());
  for (const Key& k : keys) out.push_back(k.kind ? (0x80000000u | k.id) : k.id);
}

bool is_gfx950(int dev) {
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return false;
  return std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + nb && y < x + na;
}

// Ranks between a GEMM2 item and the last GEMM1 item it reads in the
// pipelined rank table (the stage split of a launch whose work-groups take
// both kinds of item).  A tuning value, or every GEMM2 item after every
// GEMM1 item (tuning -1, row bands, or a GEMM1 list shorter than two grids:
// its second round is a partial tail that GEMM2 items should fill rather
// than delay), else one grid.  Measured over lags of 1, grid/4, grid/2,
// grid, 2 grids and all GEMM1 first on the five workloads and 8192^2 weights
// at 4096 rows: a lag below one grid claims GEMM2 items before the GEMM1
// items they wait for are running (up to 50 % slower); at or beyond one grid
// all are within a few percent, all-first ahead for the 1.75-round prefill
// GEMM1 (456 against 465 us) and one grid ahead for two and more rounds.
int merged_lag(const mlp2_plan_s* p) {
  const int grid = p->grid_override ? p->grid_override : p->grid;
  if (p->lag > 0) return p->lag;
  if (p->lag == -1 || uses_bands(p) || p->items1 < 2 * grid) return p->items1;
  return grid;
}

int upload_order(mlp2_plan_s* p) {
  std::vector<uint32_t> ord, ord2, merged;
  build_order(p, ord);
  build_order2(p, ord2);
  // With row bands every GEMM2 item goes after every GEMM1 item: bands would
  // let a band's GEMM2 items start beside the next band's GEMM1 items, but
  // then W1 and W2 stream at once and no longer fit the last-level cache
  // together (measured: 30-37 % slower than the sequential mode at 4096 to
  // 32768 rows); the launch then overlaps only the tail of GEMM1.
  const int lag = merged_lag(p);
  build_merged(p, ord, ord2, lag, merged);
  p->lead1 = 0;
  while (p->lead1 < (int64_t)merged.size() && !(merged[p->lead1] & 0x80000000u)) ++p->lead1;
  // Reduction items after everything else, tile by tile in the order in which
  // the tiles' first parts are ranked (so the first tiles to finish come first).
  if (p->items_red) {
    std::vector<char> seen((size_t)p->Mb * p->Nb2, 0);
    std::vector<uint32_t> red;
    red.reserve((size_t)p->items_red);
    for (const uint32_t q : ord2) {
      const int tile = (int)q / p->S2;
      if (seen[(size_t)tile]) continue;
      seen[(size_t)tile] = 1;
      for (int j = 0; j < p->red2; ++j) red.push_back((uint32_t)(tile * p->red2 + j));
    }
    for (const uint32_t r : red) {
      ord2.push_back(0x40000000u | r);
      merged.push_back(0xc0000000u | r);
    }
  }
  if (hipMemcpy(p->order1, ord.data(), ord.size() * sizeof(uint32_t), hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(p->order2, ord2.data(), ord2.size() * sizeof(uint32_t), hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(p->orderp, merged.data(), merged.size() * sizeof(uint32_t), hipMemcpyHostToDevice) != hipSuccess)
    return MLP2_ERR_HIP;
  return MLP2_OK;
}

}  // namespace

extern "C" {

int mlp2_last_error(void) { return g_last_error; }

const char* mlp2_strerror(int code) {
  switch (code) {
    case MLP2_OK: return "ok";
    case MLP2_ERR_INVALID_ARG: return "invalid argument";
    case MLP2_ERR_UNSUPPORTED: return "unsupported size or tuning";
    case MLP2_ERR_ALIGNMENT: return "pointer not 16-byte aligned";
    case MLP2_ERR_HIP: return "HIP runtime call failed";
    case MLP2_ERR_TIMEOUT: return "device flag wait timed out";
    case MLP2_ERR_DEVICE: return "no usable gfx950 device for this plan";
    default: return "unknown status code";
  }
}

}  // extern "C"

namespace {

mlp2_plan_s* make_plan(int64_t M, int64_t H, int64_t F, int act, const mlp2_tuning_t& tz, int dev,
                       const hipDeviceProp_t& prop, uint16_t* z_ext);
mlp2_plan_s* make_grouped(int64_t M, int64_t H, int64_t F, int act, const mlp2_tuning_t& tz, int dev,
                          const hipDeviceProp_t& prop, int64_t rows);
int64_t group_rows_for(int64_t M, int64_t F, const mlp2_tuning_t& tz);

}  // namespace

extern "C" {

mlp2_plan_t mlp2_plan_ex(int64_t M, int64_t H, int64_t F, int act, int dtype, const mlp2_tuning_t* t) {
  g_last_error = MLP2_OK;
  if (M < 1 || H < 1 || F < 1) { fail(MLP2_ERR_INVALID_ARG); return nullptr; }
  if (act < MLP2_ACT_IDENTITY || act > MLP2_ACT_SWIGLU) { fail(MLP2_ERR_INVALID_ARG); return nullptr; }
  if (dtype != MLP2_DTYPE_BF16) { fail(MLP2_ERR_INVALID_ARG); return nullptr; }
  if (M > (1 << 20) || H % 64 || F % 64 || H > (1 << 18) || F > (1 << 18)) {
    fail(MLP2_ERR_UNSUPPORTED);
    return nullptr;
  }
  mlp2_tuning_t tz;
  std::memset(&tz, 0, sizeof(tz));
  if (t) tz = *t;
  if (tz.bm < 0 || tz.bn1 < 0 || tz.bn2 < 0 || tz.splitk1 < 0 || tz.splitk2 < 0 || tz.grid < 0 || tz.order < 0 || tz.stages < 0 ||
      tz.order > MLP2_ORDER_BANDED || tz.row_group < -1 || (tz.row_group > 0 && tz.row_group % 256) ||
      (tz.waves != 0 && tz.waves != 4 && tz.waves != 8) || tz.lag < -1 || tz.p1 < 0 || tz.p1 > 63 || tz.p1 % 8 ||
      (tz.bk != 0 && tz.bk != 32 && tz.bk != 64 && tz.bk != 128) || tz.weights_nt < -1 || tz.weights_nt > 1) {
    fail(MLP2_ERR_UNSUPPORTED);
    return nullptr;
  }

  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || !is_gfx950(dev)) { fail(MLP2_ERR_DEVICE); return nullptr; }
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) { fail(MLP2_ERR_HIP); return nullptr; }
  const int64_t rows = group_rows_for(M, F, tz);
  return rows ? make_grouped(M, H, F, act, tz, dev, prop, rows) : make_plan(M, H, F, act, tz, dev, prop, nullptr);
}

}  // extern "C"

namespace {

// Rows per launch group: 0 runs the plan as one launch of each kernel.
// Automatic: once the bf16 Z of all rows exceeds the 256 MB last-level
// cache, groups of the most rows whose Z fits (a multiple of 256), at least
// 8192 of them.  Measured with 8192 x 8192 weights: at 32768 rows two
// groups of 16384 take the sequential mode from 9.4 to 8.2 ms and the
// pipelined one from 10.4 to 8.0 ms (one launch of the pipelined kernel
// over all rows loses its clock), while at 16384 rows one launch is best.
int64_t group_rows_for(int64_t M, int64_t F, const mlp2_tuning_t& tz) {
  if (tz.row_group == -1) return 0;
  if (tz.row_group > 0) return tz.row_group < M ? tz.row_group : 0;
  const int64_t fit = ((int64_t)256 << 20) / (F * 2) / 256 * 256;
  return fit >= 8192 && M > fit ? fit : 0;
}

// A plan over whole groups of `rows` rows plus one over the rest, sharing
// one Z of every row (with room for the last group's tile padding: groups
// of a multiple of 256 rows hold whole row blocks, so only the last one pads).
mlp2_plan_s* make_grouped(int64_t M, int64_t H, int64_t F, int act, const mlp2_tuning_t& tz, int dev,
                          const hipDeviceProp_t& prop, int64_t rows) {
  auto* p = new mlp2_plan_s();
  p->M = M; p->H = H; p->F = F; p->act = act; p->device = dev;
  p->num_cus = prop.multiProcessorCount;
  p->order = tz.order;
  p->group_rows = rows;
  p->ws_bytes = align_up((size_t)(M + 256) * F * 2, 256);
  if (hipMalloc(&p->ws, p->ws_bytes) != hipSuccess) {
    delete p;
    fail(MLP2_ERR_HIP);
    return nullptr;
  }
  p->Z = (uint16_t*)p->ws;
  const int64_t rest = M % rows;
  if (hipMemset(p->Z, 0, p->ws_bytes) != hipSuccess ||
      !(p->group = make_plan(rows, H, F, act, tz, dev, prop, p->Z)) ||
      (rest && !(p->tail = make_plan(rest, H, F, act, tz, dev, prop, p->Z)))) {
    const int code = g_last_error != MLP2_OK ? g_last_error : MLP2_ERR_HIP;
    mlp2_destroy(p);
    fail(code);
    return nullptr;
  }
  if (p->group->kc.bm > 256 || rows % p->group->kc.bm) {  // whole row blocks per group
    mlp2_destroy(p);
    fail(MLP2_ERR_UNSUPPORTED);
    return nullptr;
  }
  return p;
}

}  // namespace

namespace mlp2 {

// Everything a single-launch plan fixes before it has memory: tiles, split-K
// factors, grids, the stage split.  No allocation (occupancy queries only).
int configure_plan(mlp2_plan_s* p, int64_t M, int64_t H, int64_t F, int act, const mlp2_tuning_t& tz, int dev,
                   int num_cus) {
  const int nb = act == MLP2_ACT_SWIGLU ? 2 : 1;
  p->M = M; p->H = H; p->F = F; p->act = act; p->device = dev;
  p->num_cus = num_cus;

  // ---- tile choice by regime (each row chosen by measurement on MI355X).
  // Up to 256 rows the plan streams weights: one row block holds every row,
  // so each weight byte is read once, and split-K makes enough items.  At 32
  // and 64 rows the per-item costs (pipeline fill, epilogue, split-K arrival)
  // weigh more than idle CUs, so both GEMMs keep their K ranges deep; at 64
  // rows small tiles shorten the latency-bound critical path.  Beyond 256 rows (MFMA-bound): 128 x 128 tiles, two work-groups
  // per CU.
  int pref[6] = {0, 0, 0, 0, 4, 64};  // bm, bn1, bn2, ring depth, waves, stage depth
  int min_k1 = 256, min_k2 = 256;  // shallowest K range of one split-K part
  if (M <= 32) {
    // 128-column GEMM1 tiles: half the activation bytes per weight byte of
    // 64-column ones (one 70B tensor-parallel shard, 32 x 8192 x 3584:
    // 42.2 -> 39.4 us pipelined)
    pref[0] = 32; pref[1] = F % 128 == 0 ? 128 : 64; pref[2] = 128; pref[3] = 4;
    min_k1 = 2048;
    min_k2 = 1536;
  } else if (M <= 64) {
    pref[0] = 64; pref[1] = 64; pref[2] = 64; pref[3] = 4;
    min_k1 = min_k2 = 1024;
    // Too few 64-row GEMM1 tiles for a quarter of the CUs: 32-row tiles and
    // 512-deep K ranges double the items that run side by side (measured at
    // 64 x 512 x 2048: 16.4 -> 14.2 us pipelined, 17.8 -> 16.4 sequential).
    if ((int64_t)ceil_div(M, 64) * (F / 64) < p->num_cus / 4) {
      pref[0] = 32;
      min_k1 = min_k2 = 512;
    }
  } else if (M <= 128) {
    pref[0] = 128; pref[1] = 64; pref[2] = 64; pref[3] = 4;
  } else if (M <= 256) {
    pref[0] = 256; pref[1] = nb == 1 ? 128 : 64; pref[2] = 128; pref[3] = 3;
    // Gated: 128 columns of each of Wg and Wu per tile over eight waves, GEMM2
    // as two 128-column halves (two-stage ring): half the activation bytes per
    // weight byte of the four-wave 64-column tile (70B gated MLP, 256 rows:
    // 600 -> 410 us pipelined).
    if (nb == 2 && F % 128 == 0 && H % 256 == 0) {
      pref[1] = 128; pref[2] = 256; pref[3] = 2; pref[4] = 8;
    }
  } else {
    pref[0] = 128; pref[1] = 128; pref[2] = 128; pref[3] = 2;
    // 256 x 256 tiles over eight waves (a quarter of the operand bytes per flop
    // of 128 x 128) once they fill every CU: Llama-8B prefill 2048 rows
    // 523 -> 450 us pipelined, 8192 x 8192 weights at 8192 rows 2074 -> 1726 us.
    if (nb == 1 && F % 256 == 0 && H % 256 == 0 && (int64_t)ceil_div(M, 256) * (F / 256) >= p->num_cus) {
      pref[0] = 256; pref[1] = 256; pref[2] = 256; pref[3] = 2; pref[4] = 8;
    }
  }
  // Fallbacks when the preferred tiles do not divide F / H or are not built.
  const int w = pref[4];
  const int bk = pref[5];
  const int cand[][5] = {
      {pref[0], pref[1], pref[2], pref[3], w}, {pref[0], pref[1], 64, pref[3], w}, {pref[0], 64, 64, pref[3], w},
      {pref[0], pref[1], pref[2], 4, w},       {pref[0], pref[1], 64, 4, w},       {pref[0], 64, 64, 4, w},
      {pref[0], pref[1], pref[2], pref[3], 4}, {pref[0], pref[1], 64, pref[3], 4}, {pref[0], 64, 64, pref[3], 4},
      {pref[0], pref[1], pref[2], 4, 4},       {pref[0], pref[1], 64, 4, 4},       {pref[0], 64, 64, 4, 4},
      {128, 64, 64, 4, 4},                     {64, 64, 64, 4, 4},                 {32, 64, 64, 4, 4},
  };
  // Weight loads with the non-temporal hint once the two weight matrices
  // together exceed the 256 MiB last-level cache: streamed weights then stop
  // displacing the lines the activation and Z loads reuse (70B gated MLP,
  // 1.4 GB of weights, back-to-back runs: 390 -> 378 us pipelined,
  // 405 -> 390 us sequential; after a 1 GiB flush: 389 -> 393 us pipelined,
  // 405 -> 398 us sequential).  Where the weights fit, a warm run reads part
  // of them from that cache, and the hint loses it (decode 80 -> 101 us,
  // prefill 430 -> 452 us): off.
  const bool big_weights = (uint64_t)(nb + 1) * (uint64_t)H * (uint64_t)F * 2 > ((uint64_t)256 << 20);
  const int nt_first = tz.weights_nt == 1 || (tz.weights_nt == 0 && big_weights) ? 1 : 0;
  const int nt_last = tz.weights_nt == 1 ? 1 : 0;  // forced on: no fallback without it
  bool found = false;
  // The preferred stage depth first; the fallbacks with 64-deep stages; with
  // the hint where wanted and built, else without.
  for (int pass = 0; pass < 2 && !found; ++pass) {
    for (const auto& c : cand) {
      for (int nt = nt_first; nt >= nt_last && !found; --nt) {
        KernelConfig k{tz.bm ? tz.bm : c[0], tz.bn1 ? tz.bn1 : c[1], tz.bn2 ? tz.bn2 : c[2], nb,
                       tz.stages ? tz.stages : c[3], tz.waves ? tz.waves : c[4], tz.bk ? tz.bk : pass ? 64 : bk, nt};
        // 128-deep stages need every K range (H; F; the split-K parts) in whole stages
        if (F % k.bn1 == 0 && H % k.bn2 == 0 && (k.bk < 128 || (H % k.bk == 0 && F % k.bk == 0)) &&
            mlp2::config_supported(k)) {
          p->kc = k;
          found = true;
        }
      }
      if (found) break;
    }
  }
  if (!found) return MLP2_ERR_UNSUPPORTED;
  const int bm = p->kc.bm, bn1 = p->kc.bn1, bn2 = p->kc.bn2;
  p->Mb = ceil_div(M, bm);
  // The direct-to-LDS loads address each operand with a 32-bit byte offset
  // from its base: every operand one launch reads (X, Z, each weight matrix)
  // stays below 4 GB.
  const uint64_t lim = (uint64_t)1 << 32;
  if ((uint64_t)M * H * 2 >= lim || (uint64_t)p->Mb * bm * F * 2 >= lim || (uint64_t)H * F * 2 >= lim)
    return MLP2_ERR_UNSUPPORTED;
  p->Nb1 = (int)(F / bn1);
  p->Nb2 = (int)(H / bn2);
  int occ[5] = {0, 0, 0, 0, 0};
  for (int w = 0; w < 5; ++w) {
    if (mlp2::occupancy(p->kc, w, &occ[w]) != hipSuccess || occ[w] < 1) return MLP2_ERR_HIP;
  }
  const int tiles1 = p->Mb * p->Nb1, tiles2 = p->Mb * p->Nb2;
  const int gran = std::max(mlp2::kBK, p->kc.bk);  // split-K parts hold whole stages
  if (tz.splitk1) {
    p->kc1 = (int)align_up((size_t)ceil_div(H, tz.splitk1), gran);
    p->S1 = ceil_div(H, p->kc1);
  } else {
    p->S1 = choose_split(H, tiles1, occ[0] * p->num_cus, min_k1, gran, &p->kc1);
  }
  if (tz.splitk2) {
    p->kc2 = (int)align_up((size_t)ceil_div(F, tz.splitk2), gran);
    p->S2 = ceil_div(F, p->kc2);
  } else {
    p->S2 = choose_split(F, tiles2, occ[1] * p->num_cus, min_k2, gran, &p->kc2);
  }
  p->order = tz.order;
  p->lag = tz.lag;
  p->p1 = tz.p1;
  p->items1 = tiles1 * p->S1;
  p->items2 = tiles2 * p->S2;
  // A GEMM2 tile with split-K is summed by reduction items, one slice of its
  // units each, ranked after every GEMM2 item: the sums of the launch's last
  // round then run on as many work-groups as the tile has parts (up to a
  // power of two that divides the tile's bm * bn2 / 1024 unit groups)
  // instead of on the part that arrives last (70B gated MLP: the last
  // round's 32 tiles of 8 parts took 42 us each on one work-group: 383 ->
  // 364 us pipelined, 399 -> 378 us sequential).  Not where a tile's partials
  // are small (under 64 KiB: the extra items then cost more than the sums;
  // 64 x 512 x 2048, 32 KiB per tile: 16.2 -> 16.9 us).
  p->red2 = 0;
  if (p->S2 > 1 && (int64_t)p->S2 * p->kc.bm * p->kc.bn2 * 4 >= (64 << 10)) {
    const int groups = p->kc.bm * p->kc.bn2 / 1024;
    int r = 1;
    while (2 * r <= p->S2 && 2 * r <= groups) r *= 2;
    p->red2 = r > 1 ? r : 0;
  }
  p->items_red = p->red2 ? tiles2 * p->red2 : 0;

  p->occupancy = occ[2];
  p->max_grid = std::min(std::min(std::min(occ[0], occ[1]), std::min(occ[2], occ[3])), occ[4]) * p->num_cus;
  if (tz.grid > p->max_grid) return MLP2_ERR_UNSUPPORTED;
  p->grid_override = tz.grid;
  p->grid1 = std::min(occ[0] * p->num_cus, p->items1);
  p->grid2 = std::min(occ[1] * p->num_cus, p->items2);
  p->grid = std::min(std::min(std::min(occ[2], occ[3]), occ[4]) * p->num_cus, p->items1 + p->items2);
  if (!roles_ok(p->p1, tz.grid ? tz.grid : p->grid)) return MLP2_ERR_UNSUPPORTED;  // both roles need work-groups
  if (p->items2 >= (1 << 24) || p->items_red >= (1 << 24))
    return MLP2_ERR_UNSUPPORTED;  // workqueue entries hold a unit id in 24 bits; rank entries flag kinds in bits 30, 31
  return MLP2_OK;
}

// Byte offsets of the workspace parts of a configured plan (Z only when the
// plan owns it); returns the total size.
size_t plan_layout(const mlp2_plan_s* p, bool own_z, PlanLayout* L, bool with_zs) {
  const int nb = p->act == MLP2_ACT_SWIGLU ? 2 : 1;
  const int bm = p->kc.bm, bn1 = p->kc.bn1, bn2 = p->kc.bn2;
  const int tiles1 = p->Mb * p->Nb1, tiles2 = p->Mb * p->Nb2;
  const int64_t Mpad = (int64_t)p->Mb * bm;
  const int64_t F = p->F;
  const bool z_ext = !own_z;
  size_t off = 0;
  const size_t z_off = off;
  if (!z_ext) off = align_up(off + (size_t)Mpad * F * 2, 256);
  const size_t p1_off = off;
  if (p->S1 > 1) off = align_up(off + (size_t)p->items1 * nb * bm * bn1 * 4, 256);
  const size_t p2_off = off;
  if (p->S2 > 1) off = align_up(off + (size_t)p->items2 * bm * bn2 * 4, 256);
  const size_t cnt_off = off;
  const size_t line = mlp2::kLine * 4;  // one counter per 128-byte line
  const size_t c1_off = off;
  off = align_up(off + (size_t)tiles1 * line, 256);
  const size_t c2_off = off;
  off = align_up(off + (size_t)tiles2 * line, 256);
  const size_t r_off = off;
  off = align_up(off + (size_t)tiles1 * line, 256);
  const size_t b_off = off;
  off = align_up(off + (size_t)p->items2 * line, 256);
  const size_t q_off = off;
  off = align_up(off + ((size_t)p->items2 + 1) * 4, 256);
  const size_t ctrl_off = off;
  off = align_up(off + mlp2::CTRL_WORDS * 4, 256);
  const size_t cnt_end = off;
  const size_t ord_off = off;
  off = align_up(off + (size_t)p->items1 * 4, 256);
  const size_t ord2_off = off;
  off = align_up(off + ((size_t)p->items2 + p->items_red) * 4, 256);
  const size_t ordp_off = off;
  off = align_up(off + ((size_t)p->items1 + p->items2 + p->items_red) * 4, 256);
  const size_t zs_off = off;
  const size_t zs_bytes = with_zs ? align_up((size_t)2 * Mpad * F * 2, 256) : 0;
  off += zs_bytes;
  *L = PlanLayout{z_off, p1_off, p2_off, c1_off, c2_off, r_off, b_off, q_off, ctrl_off, cnt_off, cnt_end,
                  ord_off, ord2_off, ordp_off, zs_off, zs_bytes, off};
  return off;
}

// Points a configured plan's workspace fields into memory at `b` laid out by L
// (Z at z_ext when the plan does not own it).
void bind_plan(mlp2_plan_s* p, char* b, const PlanLayout& L, uint16_t* z_ext) {
  p->Z = z_ext ? z_ext : (uint16_t*)(b + L.z_off);
  p->z_external = z_ext != nullptr;
  p->part1 = p->S1 > 1 ? (float*)(b + L.p1_off) : nullptr;
  p->part2 = p->S2 > 1 ? (float*)(b + L.p2_off) : nullptr;
  p->cnt1 = (uint32_t*)(b + L.c1_off);
  p->cnt2 = (uint32_t*)(b + L.c2_off);
  p->ready = (uint32_t*)(b + L.r_off);
  p->board = (uint32_t*)(b + L.b_off);
  p->queue = (uint32_t*)(b + L.q_off);
  p->ctrl = (uint32_t*)(b + L.ctrl_off);
  p->order1 = (uint32_t*)(b + L.ord_off);
  p->order2 = (uint32_t*)(b + L.ord2_off);
  p->orderp = (uint32_t*)(b + L.ordp_off);
  p->Zs = L.zs_bytes ? (uint16_t*)(b + L.zs_off) : nullptr;
  p->counters_off = L.cnt_off;
  p->counters_bytes = L.cnt_end - L.cnt_off;
}

}  // namespace mlp2

namespace {

mlp2_plan_s* make_plan(int64_t M, int64_t H, int64_t F, int act, const mlp2_tuning_t& tz, int dev,
                       const hipDeviceProp_t& prop, uint16_t* z_ext) {
  auto* p = new mlp2_plan_s();
  const int rc = mlp2::configure_plan(p, M, H, F, act, tz, dev, prop.multiProcessorCount);
  if (rc != MLP2_OK) {
    delete p;
    fail(rc);
    return nullptr;
  }
  mlp2::PlanLayout L;
  p->ws_bytes = mlp2::plan_layout(p, z_ext == nullptr, &L);
  if (hipMalloc(&p->ws, p->ws_bytes) != hipSuccess) {
    delete p;
    fail(MLP2_ERR_HIP);
    return nullptr;
  }
  char* b = (char*)p->ws;
  mlp2::bind_plan(p, b, L, z_ext);
  const int64_t Mpad = (int64_t)p->Mb * p->kc.bm;
  if (hipMemset(b + L.cnt_off, 0, L.cnt_end - L.cnt_off) != hipSuccess ||
      (L.zs_bytes && hipMemset(b + L.zs_off, 0xFF, L.zs_bytes) != hipSuccess) ||  // sentinels everywhere
      (!z_ext && hipMemset(p->Z, 0, (size_t)Mpad * F * 2) != hipSuccess) ||
      upload_order(p) != MLP2_OK || hipDeviceSynchronize() != hipSuccess) {
    (void)hipFree(p->ws);
    delete p;
    fail(MLP2_ERR_HIP);
    return nullptr;
  }
  return p;
}

}  // namespace

extern "C" {

mlp2_plan_t mlp2_plan(int64_t M, int64_t H, int64_t F, int act, int dtype) {
  return mlp2_plan_ex(M, H, F, act, dtype, nullptr);
}

}  // extern "C"

namespace mlp2 {

// One evaluation of a single-launch plan (each kernel launched once) with
// its Z rows at Z.
int launch_plan(const mlp2_plan_s* p, const void* X, const void* W1, const void* W2, void* Y, uint16_t* Z, hipStream_t s,
                int mode) {
  Args a;
  a.X = (const uint16_t*)X;
  a.W1 = (const uint16_t*)W1;
  a.W2 = (const uint16_t*)W2;
  a.Y = (uint16_t*)Y;
  a.Z = Z;
  a.part1 = p->part1;
  a.part2 = p->part2;
  a.cnt1 = p->cnt1;
  a.cnt2 = p->cnt2;
  a.ready = p->ready;
  a.board = p->board;
  a.queue = p->queue;
  a.ctrl = p->ctrl;
  a.order1 = p->order1;
  a.order2 = p->order2;
  a.orderp = p->orderp;
  a.M = (int)p->M;
  a.H = (int)p->H;
  a.F = (int)p->F;
  a.act = p->act;
  a.Mb = p->Mb;
  a.Nb1 = p->Nb1;
  a.Nb2 = p->Nb2;
  a.S1 = p->S1;
  a.S2 = p->S2;
  a.kc1 = p->kc1;
  a.kc2 = p->kc2;
  a.items1 = p->items1;
  a.items2 = p->items2;
  a.bn1 = p->kc.bn1;
  a.spin_limit = p->spin_limit;
  a.drop_signal = p->drop_signal;
  a.trace = p->trace;
  a.trace_cap = p->trace_cap;
  a.p1 = 0;
  a.lists2 = 0;
  a.red2 = p->red2;  // the sequential GEMM2 kernel and the pipelined launch use reduction items
  a.items_red = p->items_red;
  a.Zs = p->Zs;
  a.zs_elems = (long)p->Mb * p->kc.bm * p->F;
  a.Zr = nullptr;

  const int go = p->grid_override;
  const int grids[2] = {go ? go : p->grid1, go ? go : p->grid2};
  const int gridp = go ? go : p->grid;
  a.trace_groups = std::max(std::max(grids[0], grids[1]), gridp);
  hipError_t err;
  // First items without tickets (Args::first_static): with one work-group
  // per CU, work-group g starts at once on rank g when rank g is an item that
  // never waits, which saves the round trip of a first claim and keeps the
  // first round's ranks in launch order.  (With two work-groups per CU,
  // measured at prefill size, claiming every item was faster.)
  auto statics = [&](int64_t never_wait_lead, int grid) -> int {
    return grid <= p->num_cus ? (int)std::min<int64_t>(grid, never_wait_lead) : 0;
  };
  if (mode == MLP2_MODE_SEQUENTIAL || mode == MLP2_MODE_STAGE1 || mode == MLP2_MODE_STAGE2) {
    a.lists = claim_lists(grids[0]);
    a.first_static = statics(p->items1, grids[0]);  // GEMM1 items never wait
    Args a2 = a;
    a2.lists = claim_lists(grids[1]);
    a2.first_static = statics(p->items2, grids[1]);  // nor do GEMM2 items of this mode
    const int stages = mode == MLP2_MODE_STAGE1 ? 1 : mode == MLP2_MODE_STAGE2 ? 2 : 3;
    err = mlp2::launch_sequential(p->kc, a, a2, grids, s, stages);
  } else if (mode == MLP2_MODE_TILE_PIPELINED) {
    if (p->p1) {  // role split: each role's work-groups claim from lists of their own
      const int n1 = role1_groups(p->p1, gridp);
      a.p1 = p->p1;
      a.lists = claim_lists(n1);
      a.lists2 = claim_lists(gridp - n1);
      a.first_static = 0;
    } else {
      a.lists = claim_lists(gridp);
      a.first_static = statics(p->lead1, gridp);
    }
    err = mlp2::launch_pipelined(p->kc, a, gridp, s);
  } else if (mode == MLP2_MODE_SENTINEL) {
    if (!p->Zs) return fail(MLP2_ERR_UNSUPPORTED);
    a.red2 = 0;  // its last parts sum the tiles (same order, same bits)
    a.items_red = 0;
    a.lists = claim_lists(gridp);
    a.first_static = statics(p->lead1, gridp);
    err = mlp2::launch_sentinel(p->kc, a, gridp, s);
  } else {
    a.red2 = 0;  // workqueue units: the last part sums the tile (same order, same bits)
    a.items_red = 0;
    a.lists = claim_lists(gridp);
    a.first_static = statics(p->items1, gridp);  // every ranked item is a GEMM1 item
    err = mlp2::launch_workqueue(p->kc, a, gridp, s);
  }
  if (err != hipSuccess) return fail(MLP2_ERR_HIP);
  return MLP2_OK;
}

}  // namespace mlp2

extern "C" {

int mlp2_run(mlp2_plan_t p, const void* X, const void* W1, const void* W2, void* Y, void* stream, int mode) {
  if (!p || !X || !W1 || !W2 || !Y) return fail(MLP2_ERR_INVALID_ARG);
  if (mode < MLP2_MODE_SEQUENTIAL || mode > MLP2_MODE_SENTINEL) return fail(MLP2_ERR_INVALID_ARG);
  // The two stages of a grouped plan cannot be enqueued apart (its whole
  // groups share one plan, whose split-K arrivals count one GEMM1 pass per
  // run), and its groups share no sentinel intermediates.
  if (p->group && (mode == MLP2_MODE_STAGE1 || mode == MLP2_MODE_STAGE2 || mode == MLP2_MODE_SENTINEL))
    return fail(MLP2_ERR_UNSUPPORTED);
  if (((uintptr_t)X | (uintptr_t)W1 | (uintptr_t)W2 | (uintptr_t)Y) & 15u) return fail(MLP2_ERR_ALIGNMENT);
  const int nb = p->act == MLP2_ACT_SWIGLU ? 2 : 1;
  const size_t xb = (size_t)p->M * p->H * 2, w1b = (size_t)nb * p->H * p->F * 2, w2b = (size_t)p->F * p->H * 2;
  if (overlaps(Y, xb, X, xb) || overlaps(Y, xb, W1, w1b) || overlaps(Y, xb, W2, w2b)) return fail(MLP2_ERR_INVALID_ARG);
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != p->device) return fail(MLP2_ERR_DEVICE);

  hipStream_t s = (hipStream_t)stream;
  if (!p->group) return mlp2::launch_plan(p, X, W1, W2, Y, p->Z, s, mode);
  // Row groups, in order on the stream: each group's launches read its rows
  // of X and write its rows of Z and Y.
  const int64_t R = p->group_rows;
  int64_t r0 = 0;
  for (; r0 + R <= p->M; r0 += R) {
    const int rc = mlp2::launch_plan(p->group, (const uint16_t*)X + r0 * p->H, W1, W2, (uint16_t*)Y + r0 * p->H, p->Z + r0 * p->F, s, mode);
    if (rc != MLP2_OK) return rc;
  }
  if (p->tail) return mlp2::launch_plan(p->tail, (const uint16_t*)X + r0 * p->H, W1, W2, (uint16_t*)Y + r0 * p->H, p->Z + r0 * p->F, s, mode);
  return MLP2_OK;
}

void mlp2_destroy(mlp2_plan_t p) {
  if (!p) return;
  mlp2_destroy(p->group);
  mlp2_destroy(p->tail);
  int cur = -1;
  (void)hipGetDevice(&cur);
  if (cur != p->device) (void)hipSetDevice(p->device);
  (void)hipDeviceSynchronize();
  (void)hipFree(p->ws);
  if (cur != p->device && cur >= 0) (void)hipSetDevice(cur);
  delete p;
}

int mlp2_check(mlp2_plan_t p) {
  if (!p) return fail(MLP2_ERR_INVALID_ARG);
  if (p->group) {  // every group's plan is checked (and recovered) in turn
    const int a = mlp2_check(p->group);
    const int b = p->tail ? mlp2_check(p->tail) : MLP2_OK;
    return a != MLP2_OK ? fail(a) : b != MLP2_OK ? fail(b) : MLP2_OK;
  }
  uint32_t ctrl[mlp2::CTRL_WORDS];
  if (hipMemcpy(ctrl, p->ctrl, sizeof(ctrl), hipMemcpyDeviceToHost) != hipSuccess) return fail(MLP2_ERR_HIP);
  if (ctrl[mlp2::CTRL_ERROR] == 0) return MLP2_OK;
  // Recover: counters and epoch back to zero, both sentinel intermediates
  // back to sentinels (the stream is idle by contract).
  const size_t zs_bytes = p->Zs ? (size_t)2 * p->Mb * p->kc.bm * p->F * 2 : 0;
  if (hipMemsetAsync((char*)p->ws + p->counters_off, 0, p->counters_bytes, nullptr) != hipSuccess ||
      (zs_bytes && hipMemsetAsync(p->Zs, 0xFF, zs_bytes, nullptr) != hipSuccess) ||
      hipStreamSynchronize(nullptr) != hipSuccess)
    return fail(MLP2_ERR_HIP);
  return fail(MLP2_ERR_TIMEOUT);
}

int mlp2_plan_info(mlp2_plan_t p, mlp2_info_t* out) {
  if (!p || !out) return fail(MLP2_ERR_INVALID_ARG);
  if (p->group) {  // what a whole group's launch chose, over this plan's rows
    const int rc = mlp2_plan_info(p->group, out);
    if (rc != MLP2_OK) return rc;
    out->M = p->M;
    out->row_blocks = (int)ceil_div(p->M, out->bm);
    out->order = p->order;
    out->workspace_bytes = (int64_t)(p->ws_bytes + p->group->ws_bytes + (p->tail ? p->tail->ws_bytes : 0));
    out->row_group = (int)p->group_rows;
    return MLP2_OK;
  }
  std::memset(out, 0, sizeof(*out));
  out->M = p->M;
  out->H = p->H;
  out->F = p->F;
  out->act = p->act;
  out->bm = p->kc.bm;
  out->bn1 = p->kc.bn1;
  out->splitk1 = p->S1;
  out->bn2 = p->kc.bn2;
  out->splitk2 = p->S2;
  out->bk = p->kc.bk;
  out->stages = p->kc.ns;
  out->row_blocks = p->Mb;
  out->col_blocks1 = p->Nb1;
  out->col_blocks2 = p->Nb2;
  out->items1 = p->items1;
  out->items2 = p->items2;
  out->grid_pipelined = p->grid_override ? p->grid_override : p->grid;
  out->grid_gemm1 = p->grid_override ? p->grid_override : p->grid1;
  out->grid_gemm2 = p->grid_override ? p->grid_override : p->grid2;
  out->occupancy = p->occupancy;
  out->num_cus = p->num_cus;
  out->order = p->order;
  out->workspace_bytes = (int64_t)p->ws_bytes;
  out->spin_limit = p->spin_limit;
  out->waves = p->kc.waves;
  out->lag = merged_lag(p);
  out->p1 = p->p1;
  out->weights_nt = p->kc.wnt;
  return MLP2_OK;
}

const void* mlp2_intermediate(mlp2_plan_t p) { return p ? p->Z : nullptr; }

}  // extern "C"

namespace {

// Whether a single-launch plan accepts `value` for option `key`.
bool option_valid(const mlp2_plan_s* p, int key, int64_t value) {
  switch (key) {
    case MLP2_OPT_SPIN_LIMIT: return value >= 1 && value <= 0xFFFFFFFFLL;
    case MLP2_OPT_DROP_SIGNAL: return value >= -1 && value < (int64_t)p->Mb * p->Nb1;
    case MLP2_OPT_ORDER: return value >= MLP2_ORDER_AUTO && value <= MLP2_ORDER_BANDED;
    case MLP2_OPT_GRID:  // 0 = automatic; a role split keeps work-groups in both roles
      return value >= 0 && value <= p->max_grid && roles_ok(p->p1, value ? (int)value : p->grid);
    default: return false;
  }
}

}  // namespace

extern "C" {

int mlp2_set_option(mlp2_plan_t p, int key, int64_t value) {
  if (!p) return fail(MLP2_ERR_INVALID_ARG);
  if (p->group) {  // every group's plan takes the option (a dropped signal: the whole groups')
    // The value is checked against both sub-plans before either changes, so
    // a value one of them refuses leaves the grouped plan as it was.
    const bool to_tail = p->tail && key != MLP2_OPT_DROP_SIGNAL;
    if (!option_valid(p->group, key, value) || (to_tail && !option_valid(p->tail, key, value)))
      return fail(MLP2_ERR_INVALID_ARG);
    int rc = mlp2_set_option(p->group, key, value);
    if (rc == MLP2_OK && to_tail) rc = mlp2_set_option(p->tail, key, value);
    if (rc == MLP2_OK && key == MLP2_OPT_ORDER) p->order = (int)value;
    return rc;
  }
  if (!option_valid(p, key, value)) return fail(MLP2_ERR_INVALID_ARG);
  switch (key) {
    case MLP2_OPT_SPIN_LIMIT:
      p->spin_limit = (uint32_t)value;
      return MLP2_OK;
    case MLP2_OPT_DROP_SIGNAL:
      p->drop_signal = (int)value;
      return MLP2_OK;
    case MLP2_OPT_ORDER:
      p->order = (int)value;
      if (hipDeviceSynchronize() != hipSuccess || upload_order(p) != MLP2_OK) return fail(MLP2_ERR_HIP);
      return MLP2_OK;
    default:  // MLP2_OPT_GRID: 0 = automatic, else 1 .. the work-groups that fit the device at once
      p->grid_override = (int)value;
      // the pipelined rank table places GEMM2 items about one grid after their producers
      if (hipDeviceSynchronize() != hipSuccess || upload_order(p) != MLP2_OK) return fail(MLP2_ERR_HIP);
      return MLP2_OK;
  }
}

int mlp2_trace_attach(mlp2_plan_t p, void* buffer, int records_per_group) {
  if (!p || (buffer && records_per_group < 1) || ((uintptr_t)buffer & 7u)) return fail(MLP2_ERR_INVALID_ARG);
  if (!mlp2::kTrace) return fail(MLP2_ERR_UNSUPPORTED);
  if (p->group) return mlp2_trace_attach(p->group, buffer, records_per_group);  // the whole groups' launches
  p->trace = (uint64_t*)buffer;
  p->trace_cap = buffer ? records_per_group : 0;
  return MLP2_OK;
}


}  // extern "C"

namespace {

// Tile order of one chain layer (tile = nb * Mb + mb): the XCD-grouped
// order of the two-layer plan's GEMMs when the chain has several row blocks
// (each XCD's L2 then serves a sub-block of rows and columns instead of
// every XCD reading every weight stripe), else column blocks in order.
std::vector<uint32_t> chain_layer_order(const mlp2_chain_s* p, int l) {
  const int nb = p->items[l] / p->Mb;
  if (p->Mb > 1) return xcd_grouped(p->Mb, nb, p->grid);
  std::vector<uint32_t> t((size_t)p->items[l]);
  for (int i = 0; i < p->items[l]; ++i) t[(size_t)i] = (uint32_t)i;
  return t;
}

// Rank table of the chain's one-launch mode.  Layer 0's tiles come in the
// layer order; each later layer is merged in layer by layer: the item of
// tile (mb, nb) goes right after rank h + lag of the table built so far,
// where h is the highest rank among the tiles of the layer below in row
// block mb (it reads all of them), and items of equal key keep their layer
// order.  Every item therefore ranks above all of its producers.
std::vector<uint32_t> chain_rank_table(const mlp2_chain_s* p, int lag) {
  std::vector<uint32_t> list = chain_layer_order(p, 0);
  for (int l = 1; l < p->L; ++l) {
    std::vector<int64_t> row_last((size_t)p->Mb, -1);  // highest rank of layer l - 1 per row block
    for (size_t r = 0; r < list.size(); ++r)
      if ((int)(list[r] >> 24) == l - 1) {
        const int mb = (int)(list[r] & 0xffffffu) % p->Mb;
        row_last[(size_t)mb] = std::max<int64_t>(row_last[(size_t)mb], (int64_t)r);
      }
    std::vector<std::pair<int64_t, uint32_t>> add;
    for (uint32_t t : chain_layer_order(p, l)) {
      const int64_t key = std::min<int64_t>(row_last[(size_t)(t % (uint32_t)p->Mb)] + lag, (int64_t)list.size() - 1);
      add.push_back({key, ((uint32_t)l << 24) | t});
    }
    std::stable_sort(add.begin(), add.end(), [](const std::pair<int64_t, uint32_t>& x, const std::pair<int64_t, uint32_t>& y) {
      return x.first < y.first;
    });
    std::vector<uint32_t> merged;
    merged.reserve(list.size() + add.size());
    size_t k = 0;
    for (size_t r = 0; r < list.size(); ++r) {
      merged.push_back(list[r]);
      while (k < add.size() && add[k].first == (int64_t)r) merged.push_back(add[k++].second);
    }
    list.swap(merged);
  }
  return list;
}

}  // namespace

extern "C" {

}  // extern "C"

namespace {

// Chain tile (an index into kChainTiles): 256 x 256 over eight waves when
// every layer's width is a multiple of 256 and the narrowest layer still
// has a tile per CU; else 128 x 128, unless the narrowest layer would then
// have fewer tiles than CUs: 64 x 64 (four times the items) for chains of
// few rows.
int chain_tile(int64_t M, int layers, const int64_t* dims, int cus) {
  int64_t narrowest = dims[1];
  bool wide = true;
  for (int l = 1; l <= layers; ++l) {
    narrowest = std::min(narrowest, dims[l]);
    wide = wide && dims[l] % 256 == 0;
  }
  if (wide && (int64_t)ceil_div(M, 256) * (narrowest / 256) >= cus) return 2;
  return (int64_t)ceil_div(M, 128) * (narrowest / 128) < cus ? 1 : 0;
}

// Multiply-adds per launch group of a chain (see chain_group_rows).
constexpr double kChainGroupMacs = 2.2e12;

// Rows per launch group of a chain: 0 runs each mode's launches over all
// rows.  Long one-launch runs lose their lead and their clock (as in the
// two-layer measurements); with 256 x 256 tiles the chain runs best in
// groups of about 4.4 TFLOP (2.2 T multiply-adds) per launch.  Four layers of
// 8192 x 8192, pipelined (sequential): at 16384 rows one launch 7.55 ms
// (7.29), groups of 4096 rows 7.31 (7.29), of 8192 rows 6.90 (6.99); at
// 32768 rows one launch 15.9 (15.9), groups of 4096 / 8192 / 16384 rows
// 14.4 / 14.1 / 14.7 (14.5 / 14.1 / 15.0).  It groups once the rows reach
// two such groups.
int64_t chain_group_rows(int64_t M, int layers, const int64_t* dims) {
  double macs = 0;
  for (int l = 0; l < layers; ++l) macs += (double)dims[l] * (double)dims[l + 1];
  const int64_t rows = (int64_t)(kChainGroupMacs / macs) / 256 * 256;
  return rows >= 256 && M >= 2 * rows ? rows : 0;
}

mlp2_chain_s* make_chain(int64_t M, int layers, const int64_t* dims, int act, int dev, const hipDeviceProp_t& prop) {
  const int tile = chain_tile(M, layers, dims, prop.multiProcessorCount);
  int occ = 0;
  if (mlp2::chain_occupancy(tile, &occ) != hipSuccess || occ < 1) { fail(MLP2_ERR_HIP); return nullptr; }

  auto* p = new mlp2_chain_s();
  p->M = M; p->L = layers; p->act = act; p->device = dev; p->num_cus = prop.multiProcessorCount;
  for (int l = 0; l <= layers; ++l) p->dims[l] = dims[l];
  p->tile = tile;
  p->bt = mlp2::kChainTiles[tile];
  p->Mb = ceil_div(M, p->bt);
  // 32-bit byte offsets of the direct-to-LDS loads: X, every intermediate
  // and every weight matrix stay below 4 GB.
  const uint64_t lim = (uint64_t)1 << 32;
  bool too_big = (uint64_t)M * dims[0] * 2 >= lim;
  for (int l = 0; l < layers; ++l) {
    too_big |= (uint64_t)dims[l] * dims[l + 1] * 2 >= lim;
    if (l + 1 < layers) too_big |= (uint64_t)p->Mb * p->bt * dims[l + 1] * 2 >= lim;
  }
  if (too_big) {
    delete p;
    fail(MLP2_ERR_UNSUPPORTED);
    return nullptr;
  }
  for (int l = 0; l < layers; ++l) {
    p->items[l] = (int)(p->Mb * (dims[l + 1] / p->bt));
    p->seq_off[l] = p->total;
    p->total += p->items[l];
  }
  if (p->Mb > (1 << 16) || p->total >= (1 << 24)) { delete p; fail(MLP2_ERR_UNSUPPORTED); return nullptr; }
  p->grid = std::min(occ * p->num_cus, p->total);

  // workspace: intermediates, then ready counters and control words (zeroed), then rank tables
  const int64_t Mpad = (int64_t)p->Mb * p->bt;
  const size_t line = mlp2::kLine * 4;
  size_t off = 0, z_off[mlp2::kChainMaxLayers] = {}, r_off[mlp2::kChainMaxLayers] = {};
  for (int l = 0; l + 1 < layers; ++l) {
    z_off[l] = off;
    off = align_up(off + (size_t)Mpad * dims[l + 1] * 2, 256);
  }
  const size_t cnt_off = off;
  for (int l = 0; l + 1 < layers; ++l) {
    r_off[l] = off;
    off = align_up(off + (size_t)p->items[l] * line, 256);
  }
  const size_t ctrl_off = off;
  off = align_up(off + mlp2::CTRL_WORDS * 4, 256);
  const size_t cnt_end = off;
  const size_t seq_off = off;
  off = align_up(off + (size_t)p->total * 4, 256);
  const size_t pipe_off = off;
  off = align_up(off + (size_t)p->total * 4, 256);
  p->ws_bytes = off;
  if (hipMalloc(&p->ws, p->ws_bytes) != hipSuccess) { delete p; fail(MLP2_ERR_HIP); return nullptr; }
  char* b = (char*)p->ws;
  for (int l = 0; l + 1 < layers; ++l) {
    p->Z[l] = (uint16_t*)(b + z_off[l]);
    p->ready[l] = (uint32_t*)(b + r_off[l]);
  }
  p->ctrl = (uint32_t*)(b + ctrl_off);
  p->order_seq = (uint32_t*)(b + seq_off);
  p->order_pipe = (uint32_t*)(b + pipe_off);
  p->counters_off = cnt_off;
  p->counters_bytes = cnt_end - cnt_off;
  std::vector<uint32_t> seq;
  for (int l = 0; l < layers; ++l)
    for (uint32_t t : chain_layer_order(p, l)) seq.push_back(((uint32_t)l << 24) | t);
  const std::vector<uint32_t> pipe = chain_rank_table(p, p->grid);
  if (hipMemset(b, 0, cnt_end) != hipSuccess ||
      hipMemcpy(p->order_seq, seq.data(), seq.size() * 4, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(p->order_pipe, pipe.data(), pipe.size() * 4, hipMemcpyHostToDevice) != hipSuccess ||
      hipDeviceSynchronize() != hipSuccess) {
    (void)hipFree(p->ws);
    delete p;
    fail(MLP2_ERR_HIP);
    return nullptr;
  }
  return p;
}

int launch_chain_plan(const mlp2_chain_s* p, const void* X, const void* const* W, void* Y, hipStream_t s, int mode);

}  // namespace

extern "C" {

mlp2_chain_t mlp2_chain_plan(int64_t M, int layers, const int64_t* dims, int act, int dtype) {
  g_last_error = MLP2_OK;
  if (M < 1 || layers < 1 || !dims || (act != MLP2_ACT_IDENTITY && act != MLP2_ACT_GELU_TANH) || dtype != MLP2_DTYPE_BF16) {
    fail(MLP2_ERR_INVALID_ARG);
    return nullptr;
  }
  if (layers > mlp2::kChainMaxLayers || M > (1 << 20)) { fail(MLP2_ERR_UNSUPPORTED); return nullptr; }
  for (int l = 0; l <= layers; ++l)
    if (dims[l] < mlp2::kChainWidthUnit || dims[l] % mlp2::kChainWidthUnit || dims[l] > (1 << 16)) {
      fail(dims[l] < 1 ? MLP2_ERR_INVALID_ARG : MLP2_ERR_UNSUPPORTED);
      return nullptr;
    }
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || !is_gfx950(dev)) { fail(MLP2_ERR_DEVICE); return nullptr; }
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) { fail(MLP2_ERR_HIP); return nullptr; }
  const int64_t rows = chain_group_rows(M, layers, dims);
  if (!rows) return make_chain(M, layers, dims, act, dev, prop);
  auto* p = new mlp2_chain_s();
  p->M = M; p->L = layers; p->act = act; p->device = dev; p->num_cus = prop.multiProcessorCount;
  for (int l = 0; l <= layers; ++l) p->dims[l] = dims[l];
  p->group_rows = rows;
  if (!(p->group = make_chain(rows, layers, dims, act, dev, prop)) ||
      (M % rows && !(p->tail = make_chain(M % rows, layers, dims, act, dev, prop)))) {
    const int code = g_last_error != MLP2_OK ? g_last_error : MLP2_ERR_HIP;
    mlp2_chain_destroy(p);
    fail(code);
    return nullptr;
  }
  return p;
}

int mlp2_chain_run(mlp2_chain_t p, const void* X, const void* const* W, void* Y, void* stream, int mode) {
  if (!p || !X || !W || !Y) return fail(MLP2_ERR_INVALID_ARG);
  if (mode != MLP2_MODE_SEQUENTIAL && mode != MLP2_MODE_TILE_PIPELINED) return fail(MLP2_ERR_INVALID_ARG);
  uintptr_t bits = (uintptr_t)X | (uintptr_t)Y;
  for (int l = 0; l < p->L; ++l) {
    if (!W[l]) return fail(MLP2_ERR_INVALID_ARG);
    bits |= (uintptr_t)W[l];
  }
  if (bits & 15u) return fail(MLP2_ERR_ALIGNMENT);
  const size_t yb = (size_t)p->M * p->dims[p->L] * 2;
  if (overlaps(Y, yb, X, (size_t)p->M * p->dims[0] * 2)) return fail(MLP2_ERR_INVALID_ARG);
  for (int l = 0; l < p->L; ++l)
    if (overlaps(Y, yb, W[l], (size_t)p->dims[l] * p->dims[l + 1] * 2)) return fail(MLP2_ERR_INVALID_ARG);
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != p->device) return fail(MLP2_ERR_DEVICE);
  hipStream_t s = (hipStream_t)stream;
  if (!p->group) return launch_chain_plan(p, X, W, Y, s, mode);
  // Row groups, in order on the stream: each group's launches read its rows of X and write its rows of Y.
  const int64_t R = p->group_rows, d0 = p->dims[0], dl = p->dims[p->L];
  int64_t r0 = 0;
  for (; r0 + R <= p->M; r0 += R) {
    const int rc = launch_chain_plan(p->group, (const uint16_t*)X + r0 * d0, W, (uint16_t*)Y + r0 * dl, s, mode);
    if (rc != MLP2_OK) return rc;
  }
  if (p->tail) return launch_chain_plan(p->tail, (const uint16_t*)X + r0 * d0, W, (uint16_t*)Y + r0 * dl, s, mode);
  return MLP2_OK;
}

}  // extern "C"

namespace {

// One evaluation of a chain plan without row groups.
int launch_chain_plan(const mlp2_chain_s* p, const void* X, const void* const* W, void* Y, hipStream_t s, int mode) {
  mlp2::ChainArgs c;
  std::memset(&c, 0, sizeof(c));
  Args& a = c.a;
  a.ctrl = p->ctrl;
  a.M = (int)p->M;
  a.Mb = p->Mb;
  a.spin_limit = p->spin_limit;
  a.drop_signal = -1;
  a.first_static = 0;
  a.trace = p->trace;
  a.trace_cap = p->trace_cap;
  a.trace_groups = p->grid;
  const int64_t Mpad = (int64_t)p->Mb * p->bt;
  for (int l = 0; l < p->L; ++l) {
    mlp2::ChainLayer& L = c.layer[l];
    L.A = l == 0 ? (const uint16_t*)X : p->Z[l - 1];
    L.W = (const uint16_t*)W[l];
    L.out = l == p->L - 1 ? (uint16_t*)Y : p->Z[l];
    L.ready_in = l == 0 ? nullptr : p->ready[l - 1];
    L.ready_out = l == p->L - 1 ? nullptr : p->ready[l];
    L.K = (int)p->dims[l];
    L.N = (int)p->dims[l + 1];
    L.alast = l == 0 ? (int)p->M - 1 : (int)Mpad - 1;
    L.act = l == p->L - 1 ? MLP2_ACT_IDENTITY : p->act;
    L.guard = l == p->L - 1;
  }
  if (mode == MLP2_MODE_TILE_PIPELINED) {
    a.orderp = p->order_pipe;
    a.items1 = p->total;
    a.lists = claim_lists(p->grid);
    c.wait = 1;
    c.end_of_run = 1;
    if (mlp2::launch_chain(p->tile, c, p->grid, s) != hipSuccess) return fail(MLP2_ERR_HIP);
    return MLP2_OK;
  }
  for (int l = 0; l < p->L; ++l) {  // one launch per layer, in order: the stream orders the layers
    const int grid = std::min(p->grid, p->items[l]);
    a.orderp = p->order_seq + p->seq_off[l];
    a.items1 = p->items[l];
    a.lists = claim_lists(grid);
    c.wait = 0;
    c.end_of_run = l == p->L - 1;
    if (mlp2::launch_chain(p->tile, c, grid, s) != hipSuccess) return fail(MLP2_ERR_HIP);
  }
  return MLP2_OK;
}

}  // namespace

extern "C" {

int mlp2_chain_check(mlp2_chain_t p) {
  if (!p) return fail(MLP2_ERR_INVALID_ARG);
  if (p->group) {
    const int a = mlp2_chain_check(p->group);
    const int b = p->tail ? mlp2_chain_check(p->tail) : MLP2_OK;
    return a != MLP2_OK ? fail(a) : b != MLP2_OK ? fail(b) : MLP2_OK;
  }
  uint32_t ctrl[mlp2::CTRL_WORDS];
  if (hipMemcpy(ctrl, p->ctrl, sizeof(ctrl), hipMemcpyDeviceToHost) != hipSuccess) return fail(MLP2_ERR_HIP);
  if (ctrl[mlp2::CTRL_ERROR] == 0) return MLP2_OK;
  if (hipMemsetAsync((char*)p->ws + p->counters_off, 0, p->counters_bytes, nullptr) != hipSuccess ||
      hipStreamSynchronize(nullptr) != hipSuccess)
    return fail(MLP2_ERR_HIP);
  return fail(MLP2_ERR_TIMEOUT);
}

int mlp2_chain_trace_attach(mlp2_chain_t p, void* buffer, int records_per_group) {
  if (!p || (buffer && records_per_group < 1) || ((uintptr_t)buffer & 7u)) return fail(MLP2_ERR_INVALID_ARG);
  if (!mlp2::kTrace) return fail(MLP2_ERR_UNSUPPORTED);
  if (p->group) return mlp2_chain_trace_attach(p->group, buffer, records_per_group);  // the whole groups' launches
  p->trace = (uint64_t*)buffer;
  p->trace_cap = buffer ? records_per_group : 0;
  return MLP2_OK;
}

int mlp2_chain_grid(mlp2_chain_t p) { return !p ? 0 : p->group ? mlp2_chain_grid(p->group) : p->grid; }

int mlp2_chain_set_spin_limit(mlp2_chain_t p, int64_t polls) {
  if (!p || polls < 1 || polls > 0xFFFFFFFFLL) return fail(MLP2_ERR_INVALID_ARG);
  p->spin_limit = (uint32_t)polls;
  if (p->group) (void)mlp2_chain_set_spin_limit(p->group, polls);
  if (p->tail) (void)mlp2_chain_set_spin_limit(p->tail, polls);
  return MLP2_OK;
}

void mlp2_chain_destroy(mlp2_chain_t p) {
  if (!p) return;
  mlp2_chain_destroy(p->group);
  mlp2_chain_destroy(p->tail);
  int cur = -1;
  (void)hipGetDevice(&cur);
  if (cur != p->device) (void)hipSetDevice(p->device);
  (void)hipDeviceSynchronize();
  (void)hipFree(p->ws);
  if (cur != p->device && cur >= 0) (void)hipSetDevice(cur);
  delete p;
}

}  // extern "C"
