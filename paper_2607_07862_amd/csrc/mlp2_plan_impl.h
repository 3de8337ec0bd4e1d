// Internal: the plan object and the steps of plan creation, shared by the
// C ABI (mlp2_api.cpp) and the allocation-free entry point (mlp2_noalloc.hip).
#pragma once

#include <cstddef>
#include <cstdint>

#include "../../include/mlp2.h"
#include "mlp2_launch.h"

struct mlp2_plan_s {
  int64_t M = 0, H = 0, F = 0;
  int act = 0;
  int device = -1;
  mlp2::KernelConfig kc{};
  int Mb = 0, Nb1 = 0, Nb2 = 0;
  int S1 = 1, S2 = 1, kc1 = 0, kc2 = 0;
  int items1 = 0, items2 = 0;
  int red2 = 0, items_red = 0;  // GEMM2 split-K: reduction items per tile (0: the last part sums) and in all
  int grid = 0, grid1 = 0, grid2 = 0, occupancy = 0, num_cus = 0;
  int grid_override = 0;
  int max_grid = 0;  // work-groups of every kernel of the plan that fit the device at once
  int order = MLP2_ORDER_AUTO;
  int lag = 0;  // pipelined rank-table lag (tuning; 0 = one grid, -1 = after every GEMM1 item)
  int p1 = 0;   // static GEMM1 share of every 64 work-groups of the pipelined launch (0 = shared roles)
  uint32_t spin_limit = 1u << 20;
  int drop_signal = -1;
  uint64_t* trace = nullptr;  // caller-owned timing buffer (trace builds)
  int trace_cap = 0;
  // workspace
  void* ws = nullptr;
  size_t ws_bytes = 0;
  uint16_t* Z = nullptr;
  uint16_t* Zs = nullptr;  // sentinel mode: two intermediates of Mpad x F, one after the other (or null)
  float* part1 = nullptr;
  float* part2 = nullptr;
  uint32_t* cnt1 = nullptr;
  uint32_t* cnt2 = nullptr;
  uint32_t* ready = nullptr;
  uint32_t* board = nullptr;
  uint32_t* queue = nullptr;
  uint32_t* ctrl = nullptr;
  uint32_t* order1 = nullptr;
  uint32_t* order2 = nullptr;
  uint32_t* orderp = nullptr;
  int64_t lead1 = 0;  // leading ranks of the pipelined table that are GEMM1 items (they never wait)
  size_t counters_off = 0, counters_bytes = 0;
  // Row groups (group_rows_for): a grouped plan runs as back-to-back launches
  // of `group` over whole groups of group_rows rows and of `tail` over the
  // remaining rows; every launch writes its rows of this plan's Z.
  int64_t group_rows = 0;
  mlp2_plan_s* group = nullptr;
  mlp2_plan_s* tail = nullptr;
  bool z_external = false;  // a group's plan: Z belongs to the grouped plan
};

namespace mlp2 {

// Byte offsets of a plan's workspace parts.  The counter region
// [cnt_off, cnt_end) holds every counter and control word that starts at zero.
struct PlanLayout {
  size_t z_off, p1_off, p2_off, c1_off, c2_off, r_off, b_off, q_off, ctrl_off, cnt_off, cnt_end, ord_off, ord2_off,
      ordp_off, zs_off, zs_bytes, bytes;
};

int configure_plan(mlp2_plan_s* p, int64_t M, int64_t H, int64_t F, int act, const mlp2_tuning_t& tz, int dev,
                   int num_cus);
// with_zs: room for the sentinel mode's two intermediates (zs_bytes, else 0).
size_t plan_layout(const mlp2_plan_s* p, bool own_z, PlanLayout* L, bool with_zs = true);
void bind_plan(mlp2_plan_s* p, char* base, const PlanLayout& L, uint16_t* z_ext);
int launch_plan(const mlp2_plan_s* p, const void* X, const void* W1, const void* W2, void* Y, uint16_t* Z,
                hipStream_t s, int mode);
// Records `code` as the calling thread's last error and returns it.
int record_error(int code);

}  // namespace mlp2
