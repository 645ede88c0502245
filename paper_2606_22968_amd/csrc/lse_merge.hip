// Combine split-KV partials by their log-sum-exp.
//
// When the keys of a chunk are cut into disjoint ranges, range r yields the
// normalised partial o_r and lse_r.  The full result is
//   lse = log(sum_r exp(lse_r)),   o = sum_r exp(lse_r - lse) * o_r,
// the same combination the paper's debtor stage needs after reading part of
// its KV from its partner and part locally (Section 4.1).
//
// One thread produces 4 consecutive head-dim outputs of one (row, head).
#include "internal.h"

#include <math.h>

namespace mocap {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

template <int D>
__global__ __launch_bounds__(kGroupThreads) void lse_merge_kernel(const MergeLaunch p) {
  constexpr int QUADS = D / 4;
  const int64_t idx = (int64_t)blockIdx.x * kGroupThreads + threadIdx.x;
  const int64_t rows = (int64_t)p.chunk_len * p.h_q;
  if (idx >= rows * QUADS) return;
  const int quad = (int)(idx % QUADS);
  const int64_t rh = idx / QUADS;       // row-major over (row, head)
  const int head = (int)(rh % p.h_q);
  const int64_t row = rh / p.h_q;
  const int64_t L = p.chunk_len;

  float m = -INFINITY;
  for (int r = 0; r < p.n_ranges; ++r) m = fmaxf(m, p.ws_lse[((int64_t)r * p.h_q + head) * L + row]);
  float z = 0.f;
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int r = 0; r < p.n_ranges; ++r) {
    const int64_t base = ((int64_t)r * p.h_q + head) * L + row;
    const float lr = p.ws_lse[base];
    if (lr == -INFINITY) continue;
    const float w = expf(lr - m);
    z += w;
    acc += w * *reinterpret_cast<const f32x4*>(p.ws_o + base * D + quad * 4);
  }
  const float inv = z > 0.f ? 1.f / z : 0.f;
  bf16x4 out;
#pragma unroll
  for (int e = 0; e < 4; ++e) out[e] = (__bf16)(acc[e] * inv);
  *reinterpret_cast<bf16x4*>(p.o + (row * p.h_q + head) * D + quad * 4) = out;
  if (quad == 0) p.lse[(int64_t)head * L + row] = z > 0.f ? m + logf(z) : -INFINITY;
}

}  // namespace

hipError_t launch_lse_merge(const MergeLaunch& p, int head_dim, hipStream_t stream) {
  const int64_t threads = (int64_t)p.chunk_len * p.h_q * (head_dim / 4);
  const dim3 grid((unsigned)((threads + kGroupThreads - 1) / kGroupThreads)), block(kGroupThreads);
  if (head_dim == 128) {
    hipLaunchKernelGGL(lse_merge_kernel<128>, grid, block, 0, stream, p);
  } else {
    hipLaunchKernelGGL(lse_merge_kernel<64>, grid, block, 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace mocap
