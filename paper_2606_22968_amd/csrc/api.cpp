// Host side of libmocap_attn's device calls: argument validation, split
// planning and kernel dispatch.  Every check runs before anything is
// enqueued.  The host-only chunk planners live in plan.cpp.
#include "mocap_attn.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <mutex>
#include <queue>
#include <utility>
#include <vector>

#include "internal.h"

namespace {

// Magic number and shift for unsigned division by an invariant d >= 1, valid
// for dividends below 2^31: l = ceil(log2 d), m = floor(2^32 (2^l - d) / d) + 1,
// and n / d = (umulhi(n, m) + n) >> l (Granlund and Montgomery, 1994, round-up
// method; the sum cannot overflow 32 bits because umulhi(n, m) <= n < 2^31).
void block_divider(uint32_t d, uint32_t* magic, int32_t* shift) {
  int l = 0;
  while ((1ull << l) < d) ++l;
  *magic = (uint32_t)((((1ull << l) - d) << 32) / d + 1);
  *shift = l;
}

using mocap::kTileKeys;
using mocap::kAttnWaveRows;
using mocap::kAttnWaves;

constexpr int kMaxDevices = 64;
constexpr int64_t kMaxPositions = ((int64_t)1 << 31) - 128;
std::atomic<int> g_cu_count[kMaxDevices];  // 0 = not yet queried

bool aligned16(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15u) == 0; }

bool supported_head_dim(int d) { return d == 64 || d == 128; }

mocap_status device_cu_count(int* out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MOCAP_ERR_HIP;
  if (dev >= 0 && dev < kMaxDevices) {
    const int cached = g_cu_count[dev].load(std::memory_order_relaxed);
    if (cached > 0) {
      *out = cached;
      return MOCAP_OK;
    }
  }
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return MOCAP_ERR_HIP;
  if (dev >= 0 && dev < kMaxDevices) g_cu_count[dev].store(cus, std::memory_order_relaxed);
  *out = cus;
  return MOCAP_OK;
}

// Query heads per unit (four waves): 2 when the GQA group is even, else 1.
int heads_per_unit(int group) { return group % 2 == 0 ? 2 : 1; }

struct Plan {
  int hu;
  int row_groups;
  int pairs;
  int base_wgs;      // workgroups of one KV range
  int64_t prefix_tiles;
  int n_ranges;
  size_t ws_bytes;
  // Prefix tiles [remote_begin, remote_end) come from a second store.
  int64_t remote_begin = 0, remote_end = 0;
};

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

size_t workspace_for(int n_ranges, int64_t chunk_len, int h_q, int head_dim) {
  if (n_ranges <= 1) return 0;
  const size_t rows = (size_t)n_ranges * (size_t)h_q * (size_t)chunk_len;
  return round_up(rows * (size_t)head_dim * sizeof(float), 256) + round_up(rows * sizeof(float), 256);
}

// Time model of one launch, used to choose the number of KV ranges.
//   * A workgroup costs kTileUs per 64-key tile that both of its units
//     compute and kLoneTile times that for a tile only its longer unit
//     computes (one wave per SIMD), scaled by head_dim / 128, plus kGroupUs
//     of fixed work; one workgroup per compute unit at a time (the attention
//     kernel's LDS ring fills a CU).
//   * The launch time is the makespan of longest-first list scheduling of
//     all workgroups onto the compute units (the kernel orders its work items
//     longest first), plus, when split, the partial-result traffic (written
//     by the attention kernel, read by the merge) at kMergeBytesPerUs.
// The constants were measured on MI355X; only the ranking of candidate
// plans depends on them.
constexpr double kTileUs = 2.0;
constexpr double kGroupUs = 4.0;
constexpr double kMergeBytesPerUs = 3.0e6;
constexpr double kLaunchUs = 4.0;
constexpr double kLoneTile = 0.65;

double estimate_launch_us(int64_t prefix_len, int32_t chunk_len, int h_q, int head_dim, int head_blocks_total,
                          int row_groups, int rows_per_unit, int64_t prefix_tiles, int n_ranges, int slots,
                          bool adjacent) {
  std::vector<double> cost;
  const int pairs = (row_groups + 1) / 2;
  cost.reserve((size_t)head_blocks_total * pairs * n_ranges);
  const double tile_us = kTileUs * head_dim / 128.0;
  // Tiles the unit of row group rg visits in the range that holds the chunk's keys.
  auto unit_tiles = [&](int rg) -> int64_t {
    const int64_t row_end = std::min<int64_t>(chunk_len, (int64_t)(rg + 1) * rows_per_unit);
    const int64_t t0 = n_ranges == 1 ? 0 : prefix_len / kTileKeys;
    return (prefix_len + row_end + kTileKeys - 1) / kTileKeys - t0;
  };
  for (int q = 0; q < pairs; ++q) {
    // Mirrored pair q: row groups q and R-1-q; adjacent pair q: R-2-2q and R-1-2q.
    const int top = adjacent ? row_groups - 1 - 2 * q : row_groups - 1 - q;
    const int other = adjacent ? top - 1 : q;
    const int64_t a = unit_tiles(top);
    const int64_t b = (other < 0 || other == top) ? 0 : unit_tiles(other);
    const double us = (double)std::min(a, b) * tile_us + (double)(std::max(a, b) - std::min(a, b)) * kLoneTile * tile_us;
    for (int hb = 0; hb < head_blocks_total; ++hb) cost.push_back(us + kGroupUs);
  }
  if (n_ranges > 1) {
    const int parts = n_ranges - 1;
    for (int r = 0; r < parts; ++r) {
      const int64_t tiles = prefix_tiles * (r + 1) / parts - prefix_tiles * r / parts;
      for (int i = 0; i < head_blocks_total * pairs; ++i) cost.push_back(tiles * tile_us + kGroupUs);
    }
  }
  std::sort(cost.begin(), cost.end(), std::greater<double>());
  std::priority_queue<double, std::vector<double>, std::greater<double>> load;
  for (int i = 0; i < slots; ++i) load.push(0.0);
  double makespan = 0.0;
  for (double c : cost) {
    const double t = load.top() + c;
    load.pop();
    load.push(t);
    makespan = std::max(makespan, t);
  }
  double total = makespan + kLaunchUs;
  if (n_ranges > 1) {
    const double partial = (double)n_ranges * chunk_len * h_q * (head_dim + 1) * 4.0;
    total += 2.0 * partial / kMergeBytesPerUs + kLaunchUs;
  }
  return total;
}

// 0 = automatic pairing choice; MOCAP_PAIRING=mirrored (1) or adjacent (2).
int pairing_mode() {
  const char* force = std::getenv("MOCAP_PAIRING");
  if (force && std::strcmp(force, "mirrored") == 0) return 1;
  if (force && std::strcmp(force, "adjacent") == 0) return 2;
  return 0;
}

// The better of the two pairings of row groups in a workgroup (mirrored:
// q with R-1-q, every workgroup about equally long, the shorter unit idle
// for part of the diagonal; adjacent: 2q with 2q+1, both units busy nearly
// throughout, workgroups of different lengths balanced by longest-first
// scheduling when there are many per compute unit).  MOCAP_PAIRING=mirrored
// or =adjacent in the environment forces one (for tests).
double best_pairing_us(int64_t prefix_len, int32_t chunk_len, int h_q, int head_dim, int head_blocks_total,
                       int row_groups, int rows_per_unit, int64_t prefix_tiles, int n_ranges, int slots,
                       bool* adjacent_out) {
  const int mode = pairing_mode();
  const bool only_mirrored = mode == 1, only_adjacent = mode == 2;
  const double mirrored = only_adjacent ? INFINITY
                                        : estimate_launch_us(prefix_len, chunk_len, h_q, head_dim, head_blocks_total,
                                                             row_groups, rows_per_unit, prefix_tiles, n_ranges, slots,
                                                             false);
  const double adjacent = only_mirrored ? INFINITY
                                        : estimate_launch_us(prefix_len, chunk_len, h_q, head_dim, head_blocks_total,
                                                             row_groups, rows_per_unit, prefix_tiles, n_ranges, slots,
                                                             true);
  // Adjacent only when the model expects it to win clearly.
  const bool adj = only_adjacent || (!only_mirrored && adjacent < mirrored * 0.98);
  if (adjacent_out) *adjacent_out = adj;
  return adj ? adjacent : mirrored;
}

struct PlanKey {
  int64_t prefix_len;
  int32_t chunk_len, h_q, h_kv, head_dim, requested, slots;
  size_t ws_cap;
  int pairing;
  bool operator==(const PlanKey& o) const {
    return prefix_len == o.prefix_len && chunk_len == o.chunk_len && h_q == o.h_q && h_kv == o.h_kv &&
           head_dim == o.head_dim && requested == o.requested && slots == o.slots && ws_cap == o.ws_cap &&
           pairing == o.pairing;
  }
};

// Small cache of automatic choices (a chunk loop asks for the same shape in
// mocap_chunk_attn_workspace_size and in mocap_chunk_attn).
std::mutex g_plan_mutex;
constexpr int kPlanCache = 64;
PlanKey g_plan_keys[kPlanCache];
int g_plan_values[kPlanCache];
int g_plan_count = 0, g_plan_next = 0;

// Number of KV ranges to use.  A requested count is clamped to what the
// prefix allows; 0 picks, among the prefix cut into 1, 2, 4, 8 or 16 ranges
// of at least 4 tiles (plus the chunk's own range) whose workspace fits in
// ws_cap bytes, or no split at all, the plan with the smallest modelled
// launch time.
int choose_ranges(int64_t prefix_len, int32_t chunk_len, int h_q, int h_kv, int head_dim, int head_blocks_total,
                  int row_groups, int rows_per_unit, int64_t prefix_tiles, int requested, int slots,
                  size_t ws_cap) {
  if (prefix_tiles <= 0) return 1;
  if (requested >= 1) {
    if (requested == 1) return 1;
    const int64_t parts = requested - 1 < prefix_tiles ? requested - 1 : prefix_tiles;
    return (int)parts + 1;
  }
  const PlanKey key{prefix_len, chunk_len, h_q, h_kv, head_dim, requested, slots, ws_cap, pairing_mode()};
  {
    std::lock_guard<std::mutex> lock(g_plan_mutex);
    for (int i = 0; i < g_plan_count; ++i)
      if (g_plan_keys[i] == key) return g_plan_values[i];
  }
  int best = 1;
  double best_us = best_pairing_us(prefix_len, chunk_len, h_q, head_dim, head_blocks_total, row_groups,
                                   rows_per_unit, prefix_tiles, 1, slots, nullptr);
  const int64_t max_parts = std::min<int64_t>(16, prefix_tiles / 4);
  for (int64_t parts = 1; parts <= max_parts; parts *= 2) {
    if (workspace_for((int)parts + 1, chunk_len, h_q, head_dim) > ws_cap) break;
    const double us = best_pairing_us(prefix_len, chunk_len, h_q, head_dim, head_blocks_total, row_groups,
                                      rows_per_unit, prefix_tiles, (int)parts + 1, slots, nullptr);
    if (us < best_us * 0.98) {  // a split must pay for itself clearly
      best_us = us;
      best = (int)parts + 1;
    }
  }
  std::lock_guard<std::mutex> lock(g_plan_mutex);
  g_plan_keys[g_plan_next] = key;
  g_plan_values[g_plan_next] = best;
  g_plan_next = (g_plan_next + 1) % kPlanCache;
  if (g_plan_count < kPlanCache) ++g_plan_count;
  return best;
}

mocap_status make_plan(int64_t prefix_len, int32_t chunk_len, int32_t h_q, int32_t h_kv,
                       int32_t head_dim, int32_t num_splits, Plan* plan, size_t ws_cap = SIZE_MAX) {
  const int group = h_q / h_kv;
  plan->hu = heads_per_unit(group);
  const int rows_per_unit = kAttnWaveRows * (kAttnWaves / 2 / plan->hu);
  plan->row_groups = (int)((chunk_len + rows_per_unit - 1) / rows_per_unit);
  plan->pairs = (plan->row_groups + 1) / 2;
  const int64_t base = (int64_t)(h_q / plan->hu) * plan->pairs;
  if (base > (int64_t)1 << 24) return MOCAP_ERR_UNSUPPORTED;
  plan->base_wgs = (int)base;
  plan->prefix_tiles = (prefix_len + kTileKeys - 1) / kTileKeys;
  int cus = 0;
  if (num_splits == 0 && plan->prefix_tiles > 0) {
    const mocap_status st = device_cu_count(&cus);
    if (st != MOCAP_OK) return st;
  }
  plan->n_ranges = choose_ranges(prefix_len, chunk_len, h_q, h_kv, head_dim, h_q / plan->hu, plan->row_groups,
                                 rows_per_unit, plan->prefix_tiles, num_splits, cus, ws_cap);
  plan->ws_bytes = workspace_for(plan->n_ranges, chunk_len, h_q, head_dim);
  return MOCAP_OK;
}

mocap_status check_store(const mocap_kv_store* kv) {
  if (kv == nullptr) return MOCAP_ERR_INVALID_ARG;
  if (kv->num_blocks <= 0 || kv->block_size <= 0 || kv->h_kv <= 0 || kv->head_dim <= 0)
    return MOCAP_ERR_INVALID_ARG;
  if (!supported_head_dim(kv->head_dim)) return MOCAP_ERR_UNSUPPORTED;
  if (kv->block_size % kTileKeys != 0) return MOCAP_ERR_UNSUPPORTED;
  return MOCAP_OK;
}

mocap_status check_positions(const mocap_kv_store* kv, int32_t n_table, int64_t start, int32_t len) {
  if (start < 0 || len < 0 || n_table < 0) return MOCAP_ERR_INVALID_ARG;
  // Kernels index positions with 32-bit integers.
  if (start + (int64_t)len > kMaxPositions) return MOCAP_ERR_INVALID_ARG;
  const int64_t end = start + len;
  const int64_t blocks_needed = (end + kv->block_size - 1) / kv->block_size;
  if (blocks_needed > n_table) return MOCAP_ERR_INVALID_ARG;
  return MOCAP_OK;
}

// Checks shared by the attention entry points (first store, sizes, pointers).
mocap_status check_attn_args(const mocap_kv_store* kv, const int32_t* block_table, int32_t n_table, const void* q,
                             int64_t prefix_len, int32_t chunk_len, int32_t h_q, int32_t h_kv, int32_t head_dim,
                             float scale, const void* o, const float* lse, int32_t num_splits) {
  mocap_status st = check_store(kv);
  if (st != MOCAP_OK) return st;
  if (h_q <= 0 || h_kv <= 0 || h_q % h_kv != 0 || h_kv != kv->h_kv || head_dim != kv->head_dim)
    return MOCAP_ERR_INVALID_ARG;
  if (!(scale > 0.f) || !std::isfinite(scale)) return MOCAP_ERR_INVALID_ARG;
  if (num_splits < 0) return MOCAP_ERR_INVALID_ARG;
  st = check_positions(kv, n_table, prefix_len, chunk_len);
  if (st != MOCAP_OK) return st;
  if (chunk_len == 0) return MOCAP_OK;
  if (!kv->k_pool || !kv->v_pool || !block_table || !q || !o || !lse) return MOCAP_ERR_INVALID_ARG;
  if (!aligned16(kv->k_pool) || !aligned16(kv->v_pool) || !aligned16(block_table) || !aligned16(q) ||
      !aligned16(o) || !aligned16(lse))
    return MOCAP_ERR_INVALID_ARG;
  return MOCAP_OK;
}

// A second store's key range: whole 64-key tiles inside the prefix.
bool valid_remote_range(int64_t begin, int64_t end, int64_t prefix_len) {
  return begin >= 0 && begin <= end && end <= prefix_len && begin % kTileKeys == 0 && end % kTileKeys == 0;
}

// Pairing of row groups for a launch (best_pairing_us), cached per shape.
struct PairKey {
  int64_t prefix_len;
  int32_t chunk_len, h_q, h_kv, head_dim, n_ranges, slots, mode;
  bool operator==(const PairKey& o) const {
    return prefix_len == o.prefix_len && chunk_len == o.chunk_len && h_q == o.h_q && h_kv == o.h_kv &&
           head_dim == o.head_dim && n_ranges == o.n_ranges && slots == o.slots && mode == o.mode;
  }
};
PairKey g_pair_keys[kPlanCache];
bool g_pair_values[kPlanCache];
int g_pair_count = 0, g_pair_next = 0;

bool choose_pairing(const Plan& plan, int64_t prefix_len, int32_t chunk_len, int32_t h_q, int32_t h_kv,
                    int32_t head_dim, int cus) {
  if (plan.row_groups <= 2) return false;  // a single pair: both pairings are the same
  const PairKey key{prefix_len, chunk_len, h_q, h_kv, head_dim, plan.n_ranges, cus, pairing_mode()};
  {
    std::lock_guard<std::mutex> lock(g_plan_mutex);
    for (int i = 0; i < g_pair_count; ++i)
      if (g_pair_keys[i] == key) return g_pair_values[i];
  }
  const int rows_per_unit = kAttnWaveRows * (kAttnWaves / 2 / plan.hu);
  bool adjacent = false;
  best_pairing_us(prefix_len, chunk_len, h_q, head_dim, h_q / plan.hu, plan.row_groups, rows_per_unit,
                  plan.prefix_tiles, plan.n_ranges, std::max(cus, 1), &adjacent);
  std::lock_guard<std::mutex> lock(g_plan_mutex);
  g_pair_keys[g_pair_next] = key;
  g_pair_values[g_pair_next] = adjacent;
  g_pair_next = (g_pair_next + 1) % kPlanCache;
  if (g_pair_count < kPlanCache) ++g_pair_count;
  return adjacent;
}

// Launches the attention kernel (and the merge when the plan is split).
// Arguments have been validated; remote_kv is used only for the plan's
// second-store ranges.
mocap_status enqueue_attention(const mocap_kv_store* kv, const int32_t* block_table, const mocap_kv_store* remote_kv,
                               const int32_t* remote_table, const Plan& plan, const void* q, int64_t prefix_len,
                               int32_t chunk_len, int32_t h_q, int32_t h_kv, int32_t head_dim, float scale,
                               void* o, float* lse, void* workspace, size_t workspace_bytes, void* stream) {
  const int64_t total = (int64_t)plan.base_wgs * plan.n_ranges;
  if (total > 0x7fffffff) return MOCAP_ERR_UNSUPPORTED;
  if (plan.n_ranges > 1) {
    if (workspace == nullptr || !aligned16(workspace) || workspace_bytes < plan.ws_bytes)
      return MOCAP_ERR_WORKSPACE;
  }

  mocap::AttnLaunch p;
  p.q = static_cast<const uint16_t*>(q);
  p.k_pool = static_cast<const uint16_t*>(kv->k_pool);
  p.v_pool = static_cast<const uint16_t*>(kv->v_pool);
  p.table = block_table;
  p.k_pool_r = remote_kv ? static_cast<const uint16_t*>(remote_kv->k_pool) : nullptr;
  p.v_pool_r = remote_kv ? static_cast<const uint16_t*>(remote_kv->v_pool) : nullptr;
  p.table_r = remote_kv ? remote_table : nullptr;
  p.o = static_cast<uint16_t*>(o);
  p.lse = lse;
  p.prefix_len = (int32_t)prefix_len;
  p.prefix_tiles = (int32_t)plan.prefix_tiles;
  p.chunk_len = chunk_len;
  p.h_q = h_q;
  p.h_kv = h_kv;
  p.group = h_q / h_kv;
  p.heads_per_unit = plan.hu;
  p.row_groups = plan.row_groups;
  p.pairs = plan.pairs;
  {
    int cus = 0;
    const mocap_status st = device_cu_count(&cus);
    if (st != MOCAP_OK) return st;
    p.pair_adjacent = choose_pairing(plan, prefix_len, chunk_len, h_q, h_kv, head_dim, cus) ? 1 : 0;
  }
  p.block_size = kv->block_size;
  block_divider((uint32_t)kv->block_size, &p.block_magic, &p.block_shift);
  p.n_ranges = plan.n_ranges;
  p.remote_begin = (int32_t)plan.remote_begin;
  p.remote_end = (int32_t)plan.remote_end;
  p.total_wgs = (int)total;
  p.scale_log2 = (float)((double)scale * 1.4426950408889634);
  p.ws_o = nullptr;
  p.ws_lse = nullptr;
  if (plan.n_ranges > 1) {
    const size_t rows = (size_t)plan.n_ranges * (size_t)h_q * (size_t)chunk_len;
    p.ws_o = static_cast<float*>(workspace);
    p.ws_lse = reinterpret_cast<float*>(static_cast<char*>(workspace) +
                                        round_up(rows * (size_t)head_dim * sizeof(float), 256));
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (mocap::launch_chunk_attn(p, head_dim, s) != hipSuccess) return MOCAP_ERR_HIP;
  if (plan.n_ranges > 1) {
    mocap::MergeLaunch m;
    m.ws_o = p.ws_o;
    m.ws_lse = p.ws_lse;
    m.o = p.o;
    m.lse = lse;
    m.chunk_len = chunk_len;
    m.h_q = h_q;
    m.n_ranges = plan.n_ranges;
    if (mocap::launch_lse_merge(m, head_dim, s) != hipSuccess) return MOCAP_ERR_HIP;
  }
  return MOCAP_OK;
}

// Host-side check of the block-table entries that positions [first, end) use:
// each in [0, num_blocks), no two logical blocks on one physical block.
mocap_status check_table_entries(const int32_t* table, int32_t n_table, int64_t first, int64_t end,
                                 int32_t block_size, int32_t num_blocks, int32_t* bad_out) {
  if (bad_out) *bad_out = -1;
  if (first < 0 || end < first || block_size <= 0 || num_blocks <= 0 || n_table < 0) return MOCAP_ERR_INVALID_ARG;
  if (end == first) return MOCAP_OK;
  const int64_t b0 = first / block_size, b1 = (end + block_size - 1) / block_size;
  if (b1 > n_table || table == nullptr) return MOCAP_ERR_INVALID_ARG;
  std::vector<std::pair<int32_t, int64_t>> used;
  used.reserve((size_t)(b1 - b0));
  for (int64_t b = b0; b < b1; ++b) {
    if (table[b] < 0 || table[b] >= num_blocks) {
      if (bad_out) *bad_out = (int32_t)b;
      return MOCAP_ERR_INVALID_ARG;
    }
    used.emplace_back(table[b], b);
  }
  std::sort(used.begin(), used.end());
  for (size_t i = 1; i < used.size(); ++i) {
    if (used[i].first == used[i - 1].first) {
      if (bad_out) *bad_out = (int32_t)used[i].second;
      return MOCAP_ERR_INVALID_ARG;
    }
  }
  return MOCAP_OK;
}

// In a build with MOCAP_DEBUG_TABLES, every call copies the table entries it
// will use to the host (a synchronous copy) and checks them before anything
// is enqueued; a bad entry returns MOCAP_ERR_INVALID_ARG.
#ifdef MOCAP_DEBUG_TABLES
mocap_status debug_check_table(const int32_t* dev_table, int64_t first, int64_t end, const mocap_kv_store* kv) {
  if (end <= first) return MOCAP_OK;
  const int64_t b0 = first / kv->block_size, b1 = (end + kv->block_size - 1) / kv->block_size;
  std::vector<int32_t> host((size_t)b1, 0);
  if (hipMemcpy(host.data() + b0, dev_table + b0, (size_t)(b1 - b0) * sizeof(int32_t), hipMemcpyDeviceToHost) !=
      hipSuccess)
    return MOCAP_ERR_HIP;
  return check_table_entries(host.data(), (int32_t)b1, first, end, kv->block_size, kv->num_blocks, nullptr);
}
#define MOCAP_DEBUG_CHECK(table, first, end, kv)                              \
  do {                                                                        \
    const mocap_status debug_st_ = debug_check_table((table), (first), (end), (kv)); \
    if (debug_st_ != MOCAP_OK) return debug_st_;                              \
  } while (0)
#else
#define MOCAP_DEBUG_CHECK(table, first, end, kv) \
  do {                                           \
  } while (0)
#endif

// ---- Scratch of the allocation-free entry point ----
// Split partials of mocap_chunk_attn_noalloc live in this array: every device
// the library runs on holds its own copy until the process ends.  Host code
// never uses the array's name as an address: the device address comes from
// hipGetSymbolAddress, once per device, with that device current.
constexpr size_t kScratchBytes = MOCAP_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
std::atomic<void*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mutex;

mocap_status device_scratch(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MOCAP_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return MOCAP_ERR_UNSUPPORTED;
  void* ptr = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (ptr == nullptr) {
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    ptr = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (ptr == nullptr) {
      if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return MOCAP_ERR_HIP;
      g_scratch_ptr[dev].store(ptr, std::memory_order_release);
    }
  }
  *out = ptr;
  return MOCAP_OK;
}

}  // namespace

extern "C" {

const char* mocap_status_string(mocap_status status) {
  switch (status) {
    case MOCAP_OK: return "MOCAP_OK";
    case MOCAP_ERR_INVALID_ARG: return "MOCAP_ERR_INVALID_ARG";
    case MOCAP_ERR_UNSUPPORTED: return "MOCAP_ERR_UNSUPPORTED";
    case MOCAP_ERR_WORKSPACE: return "MOCAP_ERR_WORKSPACE";
    case MOCAP_ERR_HIP: return "MOCAP_ERR_HIP";
  }
  return "MOCAP_ERR_UNKNOWN";
}

mocap_status mocap_kv_append(const mocap_kv_store* kv, const int32_t* block_table, int32_t n_table,
                             int64_t start_pos, int32_t chunk_len, const void* k_chunk,
                             const void* v_chunk, void* stream) {
  mocap_status st = check_store(kv);
  if (st != MOCAP_OK) return st;
  st = check_positions(kv, n_table, start_pos, chunk_len);
  if (st != MOCAP_OK) return st;
  if (chunk_len == 0) return MOCAP_OK;
  if (!kv->k_pool || !kv->v_pool || !block_table || !k_chunk || !v_chunk) return MOCAP_ERR_INVALID_ARG;
  if (!aligned16(kv->k_pool) || !aligned16(kv->v_pool) || !aligned16(block_table) ||
      !aligned16(k_chunk) || !aligned16(v_chunk))
    return MOCAP_ERR_INVALID_ARG;
  MOCAP_DEBUG_CHECK(block_table, start_pos, start_pos + chunk_len, kv);

  mocap::AppendLaunch p;
  p.k_chunk = static_cast<const uint16_t*>(k_chunk);
  p.v_chunk = static_cast<const uint16_t*>(v_chunk);
  p.k_pool = static_cast<uint16_t*>(kv->k_pool);
  p.v_pool = static_cast<uint16_t*>(kv->v_pool);
  p.table = block_table;
  p.start_pos = start_pos;
  p.chunk_len = chunk_len;
  p.h_kv = kv->h_kv;
  p.block_size = kv->block_size;
  if (mocap::launch_kv_append(p, kv->head_dim, static_cast<hipStream_t>(stream)) != hipSuccess)
    return MOCAP_ERR_HIP;
  return MOCAP_OK;
}

mocap_status mocap_chunk_attn_workspace_size(int64_t prefix_len, int32_t chunk_len, int32_t h_q,
                                             int32_t h_kv, int32_t head_dim, int32_t num_splits,
                                             int32_t* splits_out, size_t* bytes_out) {
  if (bytes_out == nullptr) return MOCAP_ERR_INVALID_ARG;
  if (prefix_len < 0 || chunk_len < 0 || h_q <= 0 || h_kv <= 0 || h_q % h_kv != 0 || num_splits < 0)
    return MOCAP_ERR_INVALID_ARG;
  if (prefix_len + (int64_t)chunk_len > kMaxPositions) return MOCAP_ERR_INVALID_ARG;
  if (!supported_head_dim(head_dim)) return MOCAP_ERR_UNSUPPORTED;
  if (chunk_len == 0) {
    if (splits_out) *splits_out = 1;
    *bytes_out = 0;
    return MOCAP_OK;
  }
  Plan plan;
  const mocap_status st = make_plan(prefix_len, chunk_len, h_q, h_kv, head_dim, num_splits, &plan);
  if (st != MOCAP_OK) return st;
  if (splits_out) *splits_out = plan.n_ranges;
  *bytes_out = plan.ws_bytes;
  return MOCAP_OK;
}

mocap_status mocap_chunk_attn(const mocap_kv_store* kv, const int32_t* block_table, int32_t n_table,
                              const void* q, int64_t prefix_len, int32_t chunk_len, int32_t h_q,
                              int32_t h_kv, int32_t head_dim, float scale, void* o, float* lse,
                              void* workspace, size_t workspace_bytes, int32_t num_splits,
                              void* stream) {
  mocap_status st = check_attn_args(kv, block_table, n_table, q, prefix_len, chunk_len, h_q, h_kv, head_dim,
                                    scale, o, lse, num_splits);
  if (st != MOCAP_OK || chunk_len == 0) return st;
  MOCAP_DEBUG_CHECK(block_table, 0, prefix_len + chunk_len, kv);
  Plan plan;
  st = make_plan(prefix_len, chunk_len, h_q, h_kv, head_dim, num_splits, &plan);
  if (st != MOCAP_OK) return st;
  return enqueue_attention(kv, block_table, nullptr, nullptr, plan, q, prefix_len, chunk_len, h_q, h_kv,
                           head_dim, scale, o, lse, workspace, workspace_bytes, stream);
}

mocap_status mocap_check_block_table(const int32_t* block_table, int32_t n_table, int64_t first_pos,
                                     int64_t end_pos, int32_t block_size, int32_t num_blocks,
                                     int32_t* bad_index_out) {
  return check_table_entries(block_table, n_table, first_pos, end_pos, block_size, num_blocks, bad_index_out);
}

mocap_status mocap_chunk_attn_noalloc(const mocap_kv_store* kv, const int32_t* block_table, int32_t n_table,
                                      const void* q, int64_t prefix_len, int32_t chunk_len, int32_t h_q,
                                      int32_t h_kv, int32_t head_dim, float scale, void* o, float* lse,
                                      int32_t num_splits, void* stream) {
  mocap_status st = check_attn_args(kv, block_table, n_table, q, prefix_len, chunk_len, h_q, h_kv, head_dim,
                                    scale, o, lse, num_splits);
  if (st != MOCAP_OK || chunk_len == 0) return st;
  MOCAP_DEBUG_CHECK(block_table, 0, prefix_len + chunk_len, kv);
  Plan plan;
  st = make_plan(prefix_len, chunk_len, h_q, h_kv, head_dim, num_splits, &plan, kScratchBytes);
  if (st != MOCAP_OK) return st;
  if (plan.ws_bytes > kScratchBytes) return MOCAP_ERR_WORKSPACE;  // a forced split that does not fit
  void* ws = nullptr;
  if (plan.n_ranges > 1) {
    st = device_scratch(&ws);
    if (st != MOCAP_OK) return st;
  }
  return enqueue_attention(kv, block_table, nullptr, nullptr, plan, q, prefix_len, chunk_len, h_q, h_kv, head_dim,
                           scale, o, lse, ws, kScratchBytes, stream);
}

mocap_status mocap_chunk_attn_two_store_workspace_size(int64_t prefix_len, int32_t chunk_len, int32_t h_q,
                                                       int32_t h_kv, int32_t head_dim, int64_t remote_begin,
                                                       int64_t remote_end, int32_t num_splits,
                                                       int32_t* splits_out, size_t* bytes_out) {
  if (bytes_out == nullptr) return MOCAP_ERR_INVALID_ARG;
  if (prefix_len < 0 || chunk_len < 0 || h_q <= 0 || h_kv <= 0 || h_q % h_kv != 0 || num_splits < 0)
    return MOCAP_ERR_INVALID_ARG;
  if (prefix_len + (int64_t)chunk_len > kMaxPositions) return MOCAP_ERR_INVALID_ARG;
  if (!supported_head_dim(head_dim)) return MOCAP_ERR_UNSUPPORTED;
  if (!valid_remote_range(remote_begin, remote_end, prefix_len)) return MOCAP_ERR_INVALID_ARG;
  if (chunk_len == 0) {
    if (splits_out) *splits_out = 1;
    *bytes_out = 0;
    return MOCAP_OK;
  }
  Plan plan;
  const mocap_status st = make_plan(prefix_len, chunk_len, h_q, h_kv, head_dim, num_splits, &plan);
  if (st != MOCAP_OK) return st;
  if (splits_out) *splits_out = plan.n_ranges;
  *bytes_out = plan.ws_bytes;
  return MOCAP_OK;
}

mocap_status mocap_chunk_attn_two_store(const mocap_kv_store* kv, const int32_t* block_table, int32_t n_table,
                                        const mocap_kv_store* remote_kv, const int32_t* remote_table,
                                        int32_t n_remote_table, int64_t remote_begin, int64_t remote_end,
                                        const void* q, int64_t prefix_len, int32_t chunk_len, int32_t h_q,
                                        int32_t h_kv, int32_t head_dim, float scale, void* o, float* lse,
                                        void* workspace, size_t workspace_bytes, int32_t num_splits,
                                        void* stream) {
  mocap_status st = check_attn_args(kv, block_table, n_table, q, prefix_len, chunk_len, h_q, h_kv, head_dim,
                                    scale, o, lse, num_splits);
  if (st != MOCAP_OK) return st;
  if (!valid_remote_range(remote_begin, remote_end, prefix_len)) return MOCAP_ERR_INVALID_ARG;
  if (remote_begin == remote_end) {
    if (chunk_len == 0) return MOCAP_OK;
    MOCAP_DEBUG_CHECK(block_table, 0, prefix_len + chunk_len, kv);
    Plan plan;
    st = make_plan(prefix_len, chunk_len, h_q, h_kv, head_dim, num_splits, &plan);
    if (st != MOCAP_OK) return st;
    return enqueue_attention(kv, block_table, nullptr, nullptr, plan, q, prefix_len, chunk_len, h_q, h_kv,
                             head_dim, scale, o, lse, workspace, workspace_bytes, stream);
  }
  st = check_store(remote_kv);
  if (st != MOCAP_OK) return st;
  if (remote_kv->h_kv != kv->h_kv || remote_kv->head_dim != kv->head_dim ||
      remote_kv->block_size != kv->block_size)
    return MOCAP_ERR_INVALID_ARG;
  st = check_positions(remote_kv, n_remote_table, 0, (int32_t)remote_end);
  if (st != MOCAP_OK) return st;
  if (chunk_len == 0) return MOCAP_OK;
  if (!remote_kv->k_pool || !remote_kv->v_pool || !remote_table || !aligned16(remote_kv->k_pool) ||
      !aligned16(remote_kv->v_pool) || !aligned16(remote_table))
    return MOCAP_ERR_INVALID_ARG;
  MOCAP_DEBUG_CHECK(block_table, 0, remote_begin, kv);
  MOCAP_DEBUG_CHECK(block_table, remote_end, prefix_len + chunk_len, kv);
  MOCAP_DEBUG_CHECK(remote_table, remote_begin, remote_end, remote_kv);
  Plan plan;
  st = make_plan(prefix_len, chunk_len, h_q, h_kv, head_dim, num_splits, &plan);
  if (st != MOCAP_OK) return st;
  plan.remote_begin = remote_begin / kTileKeys;
  plan.remote_end = remote_end / kTileKeys;
  return enqueue_attention(kv, block_table, remote_kv, remote_table, plan, q, prefix_len, chunk_len, h_q, h_kv,
                           head_dim, scale, o, lse, workspace, workspace_bytes, stream);
}

}  // extern "C"
