// Host-side chunk planners of libmocap_attn (no device work): the closed-form
// balanced chunk plan and the latency-balanced chunk partitioning of the
// paper's Section 4.2 (Alg. 1: the dynamic program and the simulated-annealing
// refinement).
#include "mocap_attn.h"

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <vector>

namespace {

// Sizes shared by the LBCP planners: S a positive multiple of align, M
// chunks of at least one align unit, N >= 1 stages, and a table small
// enough to scan (M (S / align)^2 <= 2^31).
mocap_status check_lbcp_sizes(int64_t seq_len, int32_t num_chunks, int32_t num_stages, int32_t align) {
  if (seq_len <= 0 || num_chunks <= 0 || num_stages <= 0 || align <= 0) return MOCAP_ERR_INVALID_ARG;
  if (seq_len % align != 0 || (int64_t)num_chunks * align > seq_len) return MOCAP_ERR_INVALID_ARG;
  const int64_t U = seq_len / align;
  if (U > 0x7fffffff / align) return MOCAP_ERR_INVALID_ARG;
  if ((double)num_chunks * (double)U * (double)U > 2147483648.0) return MOCAP_ERR_UNSUPPORTED;
  return MOCAP_OK;
}

// A chunk-cost table [k - 1][s] (k units long, starting at unit s) must be
// finite and non-negative wherever k + s <= U.
bool valid_cost_table(const double* cost, int64_t U) {
  for (int64_t k = 1; k <= U; ++k)
    for (int64_t s = 0; s + k <= U; ++s) {
      const double t = cost[(size_t)(k - 1) * U + (size_t)s];
      if (!(t >= 0.0) || !std::isfinite(t)) return false;
    }
  return true;
}

// Alg. 1, first stage (Section 4.2): for chunk index m from M down to 1, start
// u from U - 1 down to 0 and length k upwards, combine EvaluateChunk(k, u)
// with the suffix state (m + 1, u + k) and keep the k minimising
// t'_sum + (N - 1) t'_max.  The suffix boundary is t = 0 at (M + 1, U) and
// infeasible elsewhere.
template <typename Eval>
mocap_status lbcp_dp(int64_t U, int M, int num_stages, int32_t align, Eval evaluate, int32_t* lengths_out,
                     double* t_max_out, double* t_sum_out) {
#pragma clang fp contract(off)
  const double stages_m1 = (double)(num_stages - 1);
  const double inf = INFINITY;
  std::vector<double> tmax((size_t)(M + 2) * (U + 1), inf), tsum((size_t)(M + 2) * (U + 1), inf);
  std::vector<int32_t> ss((size_t)(M + 2) * (U + 1), 0);
  auto at = [&](int m, int64_t u) { return (size_t)m * (U + 1) + (size_t)u; };
  tmax[at(M + 1, U)] = 0.0;
  tsum[at(M + 1, U)] = 0.0;
  for (int m = M; m >= 1; --m) {
    for (int64_t s = U - 1; s >= 0; --s) {
      double best_obj = inf;
      for (int64_t k = 1; k <= U - s - (M - m); ++k) {
        const size_t nxt = at(m + 1, s + k);
        if (tsum[nxt] == inf) continue;  // infeasible suffix
        const double t = evaluate(k, s);
        const double t_max = std::max(tmax[nxt], t);
        const double t_sum = tsum[nxt] + t;
        const double obj = t_sum + stages_m1 * t_max;
        if (obj < best_obj) {
          best_obj = obj;
          tmax[at(m, s)] = t_max;
          tsum[at(m, s)] = t_sum;
          ss[at(m, s)] = (int32_t)k;
        }
      }
    }
  }
  if (tsum[at(1, 0)] == inf) return MOCAP_ERR_INVALID_ARG;
  int64_t u = 0;
  for (int m = 1; m <= M; ++m) {
    const int32_t k = ss[at(m, u)];
    lengths_out[m - 1] = k * align;
    u += k;
  }
  if (t_max_out) *t_max_out = tmax[at(1, 0)];
  if (t_sum_out) *t_sum_out = tsum[at(1, 0)];
  return MOCAP_OK;
}

// SplitMix64 (Steele, Lea and Flood, 2014): a counter-based generator,
// x += 0x9E3779B97F4A7C15 then two xor-shift-multiply rounds.
struct SplitMix64 {
  uint64_t x;
  uint64_t next() {
    uint64_t z = (x += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  double uniform() { return (double)(next() >> 11) * (1.0 / 9007199254740992.0); }  // [0, 1), 53 bits
};

// ---- LBCP second stage under the serving model (EvaluatePrefill / EvaluateE2E) ----
//
// N identical stages run the chunk operations of Q queued requests, served in
// order in batches of B (the last one smaller).  Operation j of a batch of n
// requests takes t_j + (n - 1) max(t_j - e, 0): t_j is the table's latency of
// the chunk for one request, e the part a batch does not multiply.  Every
// stage takes the same time for an operation, so operation k completes on
// stage s at sum_{i<=k} t_i + (s - 1) max_{i<=k} t_i (the flow-shop recurrence
// in closed form).  A stage holds a batch's KV from the start of each of its
// chunks there until the batch completes on stage N (Section 3.1); the batch's
// KV must fit each stage's capacity, or, under MBKR's fixed cross-half pairing
// (Section 4.1), the pooled capacity of stages i and i + N/2.  Every step
// below follows the same order of floating-point operations as the oracle.
struct ServingModel {
  int64_t U;
  int M, N;
  int64_t align;
  const double* table;
  double e, kv_bytes, capacity;
  bool pairing;
  int max_batch, Q;
};

struct Op {
  int b, j, n;
  double t;
};

void batch_op_times(const ServingModel& sm, const std::vector<int64_t>& ss, int n, std::vector<double>& out) {
  out.clear();
  int64_t s = 0;
  for (int m = 0; m < sm.M; ++m) {
    const double t = sm.table[(size_t)(ss[m] - 1) * sm.U + (size_t)s];
    out.push_back(t + (double)(n - 1) * std::max(t - sm.e, 0.0));
    s += ss[m];
  }
}

void make_schedule(const ServingModel& sm, const std::vector<int64_t>& ss, int B, std::vector<Op>& ops) {
  ops.clear();
  std::vector<double> times;
  int b = 0;
  for (int left = sm.Q; left > 0; left -= std::min(B, left), ++b) {
    const int n = std::min(B, left);
    batch_op_times(sm, ss, n, times);
    for (int j = 0; j < sm.M; ++j) ops.push_back(Op{b, j, n, times[j]});
  }
}

// C[(s - 1) * K + k]: completion of operation k on stage s.
void completion_times(const std::vector<Op>& ops, int N, std::vector<double>& C) {
  const size_t K = ops.size();
  C.assign((size_t)N * K, 0.0);
  double acc = 0.0, mx = 0.0;
  for (size_t k = 0; k < K; ++k) {
    acc += ops[k].t;
    mx = std::max(mx, ops[k].t);
    for (int s = 1; s <= N; ++s) C[(size_t)(s - 1) * K + k] = acc + (double)(s - 1) * mx;
  }
}

struct KvEvent {
  double when;
  int kind;  // 0: a batch leaves (its KV is freed), 1: a chunk starts on a stage
  int s, b, j;
  int64_t delta;
  bool operator<(const KvEvent& o) const {
    if (when != o.when) return when < o.when;
    if (kind != o.kind) return kind < o.kind;
    if (s != o.s) return s < o.s;
    if (b != o.b) return b < o.b;
    return j < o.j;
  }
};

int64_t peak_kv_tokens(const ServingModel& sm, const std::vector<int64_t>& ss, const std::vector<Op>& ops,
                       const std::vector<double>& C, const int* stages, int n_stages) {
  const size_t K = ops.size();
  const int n_batches = ops.empty() ? 0 : ops.back().b + 1;
  std::vector<double> done(n_batches, 0.0);
  for (size_t k = 0; k < K; ++k) done[ops[k].b] = C[(size_t)(sm.N - 1) * K + k];
  std::vector<KvEvent> ev;
  ev.reserve((K + n_batches) * n_stages);
  for (int g = 0; g < n_stages; ++g) {
    const int s = stages[g];
    for (size_t k = 0; k < K; ++k)
      ev.push_back(KvEvent{C[(size_t)(s - 1) * K + k] - ops[k].t, 1, s, ops[k].b, ops[k].j,
                           (int64_t)ops[k].n * ss[ops[k].j] * sm.align});
  }
  for (int b = 0; b < n_batches; ++b)
    for (int g = 0; g < n_stages; ++g) ev.push_back(KvEvent{done[b], 0, stages[g], b, -1, 0});
  std::sort(ev.begin(), ev.end());
  std::vector<int64_t> held((size_t)(sm.N + 1) * n_batches, 0);
  int64_t cur = 0, peak = 0;
  for (const KvEvent& x : ev) {
    int64_t& h = held[(size_t)x.s * n_batches + x.b];
    if (x.kind == 0) {
      cur -= h;
      h = 0;
    } else {
      h += x.delta;
      cur += x.delta;
      peak = std::max(peak, cur);
    }
  }
  return peak;
}

bool batch_feasible(const ServingModel& sm, const std::vector<int64_t>& ss, int B) {
  std::vector<Op> ops;
  std::vector<double> C;
  make_schedule(sm, ss, B, ops);
  completion_times(ops, sm.N, C);
  if (sm.pairing) {
    for (int s = 1; s <= sm.N / 2; ++s) {
      const int pair[2] = {s, s + sm.N / 2};
      if (!((double)peak_kv_tokens(sm, ss, ops, C, pair, 2) * sm.kv_bytes <= 2.0 * sm.capacity)) return false;
    }
  } else {
    for (int s = 1; s <= sm.N; ++s) {
      if (!((double)peak_kv_tokens(sm, ss, ops, C, &s, 1) * sm.kv_bytes <= sm.capacity)) return false;
    }
  }
  return true;
}

double sum_then_max(const std::vector<double>& times, int N) {
  double acc = 0.0, mx = 0.0;
  for (double t : times) {
    acc += t;
    mx = std::max(mx, t);
  }
  return acc + (double)(N - 1) * mx;
}

// EvaluatePrefill: the largest feasible batch B' (0 if none) and T'_pre.
void evaluate_prefill(const ServingModel& sm, const std::vector<int64_t>& ss, int* B_out, double* t_pre) {
  int best = 0;
  for (int B = 1; B <= std::min(sm.max_batch, sm.Q); ++B)
    if (batch_feasible(sm, ss, B)) best = B;
  *B_out = best;
  if (best == 0) {
    *t_pre = INFINITY;
    return;
  }
  std::vector<double> times;
  batch_op_times(sm, ss, best, times);
  *t_pre = sum_then_max(times, sm.N);
}

// EvaluateE2E: completion time of the last of the Q requests in batches of B.
double evaluate_e2e(const ServingModel& sm, const std::vector<int64_t>& ss, int B) {
  if (B == 0) return INFINITY;
  std::vector<Op> ops;
  std::vector<double> C;
  make_schedule(sm, ss, B, ops);
  completion_times(ops, sm.N, C);
  return C[(size_t)(sm.N - 1) * ops.size() + ops.size() - 1];
}

mocap_status serving_model(int64_t seq_len, int32_t num_chunks, int32_t num_stages, int32_t align,
                           const double* chunk_cost, const mocap_lbcp_serving* serving, ServingModel* sm) {
  const mocap_status st = check_lbcp_sizes(seq_len, num_chunks, num_stages, align);
  if (st != MOCAP_OK) return st;
  if (chunk_cost == nullptr || serving == nullptr) return MOCAP_ERR_INVALID_ARG;
  const int64_t U = seq_len / align;
  if (!valid_cost_table(chunk_cost, U)) return MOCAP_ERR_INVALID_ARG;
  if (!(serving->fixed_cost >= 0.0) || !std::isfinite(serving->fixed_cost) || !(serving->kv_bytes_per_token > 0.0) ||
      !std::isfinite(serving->kv_bytes_per_token) || !(serving->stage_capacity > 0.0) ||
      !std::isfinite(serving->stage_capacity) || serving->max_batch < 1 || serving->max_batch > 4096 ||
      serving->requests < 1 || serving->requests > 4096 || (serving->pairing != 0 && serving->pairing != 1))
    return MOCAP_ERR_INVALID_ARG;
  if (serving->pairing && num_stages % 2 != 0) return MOCAP_ERR_INVALID_ARG;
  *sm = ServingModel{U, num_chunks, num_stages, align, chunk_cost, serving->fixed_cost,
                     serving->kv_bytes_per_token, serving->stage_capacity, serving->pairing != 0,
                     serving->max_batch, serving->requests};
  return MOCAP_OK;
}

mocap_status read_partition(const int32_t* lengths, int M, int32_t align, int64_t U, std::vector<int64_t>* ss) {
  if (lengths == nullptr) return MOCAP_ERR_INVALID_ARG;
  ss->assign(M, 0);
  int64_t total = 0;
  for (int m = 0; m < M; ++m) {
    if (lengths[m] <= 0 || lengths[m] % align != 0) return MOCAP_ERR_INVALID_ARG;
    (*ss)[m] = lengths[m] / align;
    total += (*ss)[m];
  }
  return total == U ? MOCAP_OK : MOCAP_ERR_INVALID_ARG;
}

}  // namespace

extern "C" {

mocap_status mocap_lbcp_evaluate(int64_t seq_len, int32_t num_chunks, int32_t num_stages, int32_t align,
                                 const double* chunk_cost, const mocap_lbcp_serving* serving,
                                 const int32_t* lengths, int32_t* batch_out, double* t_pre_out,
                                 double* t_e2e_out) {
#pragma clang fp contract(off)
  ServingModel sm;
  mocap_status st = serving_model(seq_len, num_chunks, num_stages, align, chunk_cost, serving, &sm);
  if (st != MOCAP_OK) return st;
  std::vector<int64_t> ss;
  st = read_partition(lengths, num_chunks, align, sm.U, &ss);
  if (st != MOCAP_OK) return st;
  int B = 0;
  double t_pre = 0.0;
  evaluate_prefill(sm, ss, &B, &t_pre);
  const double t = evaluate_e2e(sm, ss, B);
  if (batch_out) *batch_out = B;
  if (t_pre_out) *t_pre_out = t_pre;
  if (t_e2e_out) *t_e2e_out = t;
  return MOCAP_OK;
}

mocap_status mocap_lbcp_refine_e2e(int64_t seq_len, int32_t num_chunks, int32_t num_stages, int32_t align,
                                   const double* chunk_cost, const mocap_lbcp_serving* serving, double temp0,
                                   double temp_min, double alpha, int32_t rounds, uint64_t seed,
                                   int32_t* lengths_inout, int32_t* batch_out, double* t_pre_out,
                                   double* t_e2e_out) {
#pragma clang fp contract(off)
  ServingModel sm;
  mocap_status st = serving_model(seq_len, num_chunks, num_stages, align, chunk_cost, serving, &sm);
  if (st != MOCAP_OK) return st;
  if (!(temp0 > 0.0) || !(temp_min > 0.0) || !std::isfinite(temp0) || !(alpha > 0.0) || !(alpha < 1.0) ||
      rounds < 1)
    return MOCAP_ERR_INVALID_ARG;
  std::vector<int64_t> ss;
  st = read_partition(lengths_inout, num_chunks, align, sm.U, &ss);
  if (st != MOCAP_OK) return st;
  const int M = num_chunks;
  auto score = [&](const std::vector<int64_t>& x, int* B, double* t_pre) {
    evaluate_prefill(sm, x, B, t_pre);
    return evaluate_e2e(sm, x, *B);
  };
  SplitMix64 rng{seed};
  int B = 0;
  double t_pre = 0.0;
  double t_cur = score(ss, &B, &t_pre);
  std::vector<int64_t> best = ss, cand = ss;
  int best_B = B;
  double best_pre = t_pre, best_t = t_cur;
  for (double temp = temp0; temp > temp_min; temp *= alpha) {
    for (int r = 0; r < rounds; ++r) {
      if (M < 2) break;
      const int64_t j = 1 + (int64_t)(rng.next() % (uint64_t)(M - 1));
      const int64_t dir = (rng.next() & 1) ? 1 : -1;
      cand = ss;
      cand[j - 1] += dir;
      cand[j] -= dir;
      if (cand[j - 1] < 1 || cand[j] < 1) continue;
      int B_new = 0;
      double pre_new = 0.0;
      const double t_new = score(cand, &B_new, &pre_new);
      const double u = rng.uniform();
      if (t_new < t_cur || (std::isfinite(t_new) && u < std::exp(-(t_new - t_cur) / temp))) {
        ss = cand;
        B = B_new;
        t_pre = pre_new;
        t_cur = t_new;
      }
      if (t_cur < best_t) {
        best = ss;
        best_B = B;
        best_pre = t_pre;
        best_t = t_cur;
      }
    }
  }
  for (int m = 0; m < M; ++m) lengths_inout[m] = (int32_t)(best[m] * align);
  if (batch_out) *batch_out = best_B;
  if (t_pre_out) *t_pre_out = best_pre;
  if (t_e2e_out) *t_e2e_out = best_t;
  return MOCAP_OK;
}

mocap_status mocap_chunk_plan(int64_t seq_len, int32_t num_chunks, int32_t align, int32_t balanced,
                              int32_t* lengths_out) {
  if (seq_len <= 0 || num_chunks <= 0 || lengths_out == nullptr) return MOCAP_ERR_INVALID_ARG;
  if (seq_len > ((int64_t)1 << 40)) return MOCAP_ERR_INVALID_ARG;
  typedef __int128 i128;
  int64_t prev = 0;
  for (int c = 1; c <= num_chunks; ++c) {
    int64_t bound;
    if (c == num_chunks) {
      bound = seq_len;
    } else if (!balanced) {
      bound = (int64_t)((i128)c * seq_len / num_chunks);
    } else {
      if (align <= 0 || seq_len % align != 0) return MOCAP_ERR_INVALID_ARG;
      // Boundary in units of `align`: u = A sqrt(c / M) with A = seq_len / align.
      // The nearest integer k satisfies M (2k - 1)^2 <= 4 A^2 c < M (2k + 1)^2.
      const i128 A = seq_len / align;
      const i128 rhs = 4 * A * A * (i128)c;
      int64_t k = (int64_t)std::floor((double)A * std::sqrt((double)c / num_chunks) + 0.5);
      auto lower_ok = [&](int64_t kk) { return kk <= 0 || (i128)num_chunks * (2 * (i128)kk - 1) * (2 * (i128)kk - 1) <= rhs; };
      while (!lower_ok(k)) --k;
      while (lower_ok(k + 1)) ++k;
      const i128 edge = (i128)num_chunks * (2 * (i128)k - 1) * (2 * (i128)k - 1);
      if (k > 0 && edge == rhs) return MOCAP_ERR_INVALID_ARG;  // exact tie
      bound = k * (int64_t)align;
    }
    const int64_t len = bound - prev;
    if (len <= 0 || len > 0x7fffffff) return MOCAP_ERR_INVALID_ARG;
    lengths_out[c - 1] = (int32_t)len;
    prev = bound;
  }
  return MOCAP_OK;
}

mocap_status mocap_chunk_prefixes(const int32_t* lengths, int32_t num_chunks, int64_t* prefixes_out) {
  if (num_chunks < 0 || (num_chunks > 0 && (lengths == nullptr || prefixes_out == nullptr)))
    return MOCAP_ERR_INVALID_ARG;
  for (int c = 0; c < num_chunks; ++c)
    if (lengths[c] < 0) return MOCAP_ERR_INVALID_ARG;
  // P_c = L_0 + ... + L_{c-1}: at most 2^31 chunks of at most 2^31 - 1 tokens,
  // so the sum stays below 2^62.
  int64_t p = 0;
  for (int c = 0; c < num_chunks; ++c) {
    prefixes_out[c] = p;
    p += lengths[c];
  }
  return MOCAP_OK;
}

mocap_status mocap_lbcp_plan(int64_t seq_len, int32_t num_chunks, int32_t num_stages, int32_t align,
                             double cost_pair, double cost_token, double cost_chunk,
                             int32_t* lengths_out, double* t_max_out, double* t_sum_out) {
#pragma clang fp contract(off)
  if (!(cost_pair >= 0.0) || !(cost_token >= 0.0) || !(cost_chunk >= 0.0) || !std::isfinite(cost_pair) ||
      !std::isfinite(cost_token) || !std::isfinite(cost_chunk))
    return MOCAP_ERR_INVALID_ARG;
  const mocap_status st = check_lbcp_sizes(seq_len, num_chunks, num_stages, align);
  if (st != MOCAP_OK || lengths_out == nullptr) return st != MOCAP_OK ? st : MOCAP_ERR_INVALID_ARG;
  return lbcp_dp(seq_len / align, num_chunks, num_stages, align,
                 [&](int64_t k, int64_t s) {
                   const double c = (double)(k * align), p = (double)(s * align);
                   return cost_pair * (c * p + c * (c + 1.0) / 2.0) + cost_token * c + cost_chunk;
                 },
                 lengths_out, t_max_out, t_sum_out);
}

mocap_status mocap_lbcp_plan_table(int64_t seq_len, int32_t num_chunks, int32_t num_stages, int32_t align,
                                   const double* chunk_cost, int32_t* lengths_out, double* t_max_out,
                                   double* t_sum_out) {
#pragma clang fp contract(off)
  const mocap_status st = check_lbcp_sizes(seq_len, num_chunks, num_stages, align);
  if (st != MOCAP_OK) return st;
  if (chunk_cost == nullptr || lengths_out == nullptr) return MOCAP_ERR_INVALID_ARG;
  const int64_t U = seq_len / align;
  if (!valid_cost_table(chunk_cost, U)) return MOCAP_ERR_INVALID_ARG;
  return lbcp_dp(U, num_chunks, num_stages, align,
                 [&](int64_t k, int64_t s) { return chunk_cost[(size_t)(k - 1) * U + (size_t)s]; },
                 lengths_out, t_max_out, t_sum_out);
}

mocap_status mocap_lbcp_refine(int64_t seq_len, int32_t num_chunks, int32_t num_stages, int32_t align,
                               const double* chunk_cost, double temp0, double temp_min, double alpha,
                               int32_t rounds, uint64_t seed, int32_t* lengths_inout, double* latency_out) {
#pragma clang fp contract(off)
  mocap_status st = check_lbcp_sizes(seq_len, num_chunks, num_stages, align);
  if (st != MOCAP_OK) return st;
  if (chunk_cost == nullptr || lengths_inout == nullptr) return MOCAP_ERR_INVALID_ARG;
  if (!(temp0 > 0.0) || !(temp_min > 0.0) || !std::isfinite(temp0) || !(alpha > 0.0) || !(alpha < 1.0) ||
      rounds < 1)
    return MOCAP_ERR_INVALID_ARG;
  const int64_t U = seq_len / align;
  if (!valid_cost_table(chunk_cost, U)) return MOCAP_ERR_INVALID_ARG;
  const int M = num_chunks;
  // Chunk lengths in units of align; must be a valid partition of seq_len.
  std::vector<int64_t> ss(M);
  int64_t total = 0;
  for (int m = 0; m < M; ++m) {
    if (lengths_inout[m] <= 0 || lengths_inout[m] % align != 0) return MOCAP_ERR_INVALID_ARG;
    ss[m] = lengths_inout[m] / align;
    total += ss[m];
  }
  if (total != U) return MOCAP_ERR_INVALID_ARG;
  // Pipeline latency of a partition: sum of its chunk costs plus (N - 1)
  // times the largest (Alg. 1's first-stage objective, here evaluated
  // exactly on the whole partition).
  const double stages_m1 = (double)(num_stages - 1);
  auto latency = [&](const std::vector<int64_t>& x) {
    double t_sum = 0.0, t_max = 0.0;
    int64_t s = 0;
    for (int m = 0; m < M; ++m) {
      const double t = chunk_cost[(size_t)(x[m] - 1) * U + (size_t)s];
      t_sum += t;
      t_max = std::max(t_max, t);
      s += x[m];
    }
    return t_sum + stages_m1 * t_max;
  };
  SplitMix64 rng{seed};
  std::vector<int64_t> best = ss, cand = ss;
  double t_cur = latency(ss), t_best = t_cur;
  for (double temp = temp0; temp > temp_min; temp *= alpha) {
    for (int r = 0; r < rounds; ++r) {
      // Perturb: move one of the M - 1 inner boundaries by one unit, keeping
      // both neighbouring chunks non-empty (S and M are preserved).
      if (M < 2) break;
      const int64_t j = 1 + (int64_t)(rng.next() % (uint64_t)(M - 1));  // boundary between chunks j-1 and j
      const int64_t dir = (rng.next() & 1) ? 1 : -1;                     // +1 moves the boundary right
      cand = ss;
      cand[j - 1] += dir;
      cand[j] -= dir;
      if (cand[j - 1] < 1 || cand[j] < 1) continue;
      const double t_new = latency(cand);
      const double u = rng.uniform();
      if (t_new < t_cur || u < std::exp(-(t_new - t_cur) / temp)) {
        ss = cand;
        t_cur = t_new;
      }
      if (t_cur < t_best) {
        best = ss;
        t_best = t_cur;
      }
    }
  }
  for (int m = 0; m < M; ++m) lengths_inout[m] = (int32_t)(best[m] * align);
  if (latency_out) *latency_out = t_best;
  return MOCAP_OK;
}

}  // extern "C"
