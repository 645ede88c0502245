// Append one chunk's keys/values to the block-addressed KV store.
//
// Each chunk produces new KV that later chunks keep reading (Section 2.2);
// under the paper's memory-balanced reallocation (Section 4.1) a stage first
// produces the chunk's KV and then places it, locally or at its partner, so
// the store is addressed through a block table.  This kernel is a pure
// bit copy:
//   K: [L][Hkv][D] -> k_pool[phys][h][slot][:]        (row per position)
//   V: [L][Hkv][D] -> v_pool[phys][h][:][slot]        (transposed per block)
// with phys = table[(P + t) / bs] and slot = (P + t) % bs.
//
// One workgroup moves 64 positions of one KV head.  K rows go straight out as
// 16-byte stores.  V goes through LDS so that the transposed stores cover
// consecutive slots of one head-dim row: 16 bytes per thread for a whole
// 64-aligned tile, 2 bytes per lane at ragged edges.
#include "internal.h"

namespace mocap {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int D>
__global__ __launch_bounds__(kGroupThreads) void kv_append_kernel(const AppendLaunch p) {
  constexpr int ROW_CHUNKS = D / 8;
  constexpr int PITCH = D + 2;  // LDS pitch in elements (odd number of words)
  __shared__ uint16_t vt[kTileKeys * PITCH];

  const int tid = threadIdx.x;
  const int t0 = blockIdx.x * kTileKeys;
  const int h = blockIdx.y;
  const int n_tok = min(kTileKeys, p.chunk_len - t0);

  for (int c = tid; c < kTileKeys * ROW_CHUNKS; c += kGroupThreads) {
    const int tok = c / ROW_CHUNKS;
    const int col = (c % ROW_CHUNKS) * 8;
    if (tok >= n_tok) continue;
    const int64_t t = t0 + tok;
    const int64_t pos = p.start_pos + t;
    const int64_t lb = pos / p.block_size;
    const int64_t slot = pos - lb * p.block_size;
    const int64_t phys = p.table[lb];
    const int64_t src = (t * p.h_kv + h) * D + col;
    const u32x4 kv = *reinterpret_cast<const u32x4*>(p.k_chunk + src);
    *reinterpret_cast<u32x4*>(p.k_pool + ((phys * p.h_kv + h) * p.block_size + slot) * D + col) = kv;
    const u32x4 vv = *reinterpret_cast<const u32x4*>(p.v_chunk + src);
    uint32_t* dst = reinterpret_cast<uint32_t*>(vt + tok * PITCH + col);
#pragma unroll
    for (int w = 0; w < 4; ++w) dst[w] = vv[w];
  }
  __syncthreads();

  const int64_t pos0 = p.start_pos + t0;
  if (n_tok == kTileKeys && pos0 % kTileKeys == 0) {
    // A whole aligned tile (one block holds it): each thread gathers 8
    // consecutive positions of one head-dim row and stores them as 16 bytes.
    const int64_t lb = pos0 / p.block_size;
    const int64_t slot0 = pos0 - lb * p.block_size;
    uint16_t* base = p.v_pool + ((int64_t)p.table[lb] * p.h_kv + h) * D * (int64_t)p.block_size + slot0;
    for (int c = tid; c < D * (kTileKeys / 8); c += kGroupThreads) {
      const int e = c / (kTileKeys / 8), g = c % (kTileKeys / 8);
      u32x4 out;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        out[j] = (uint32_t)vt[(g * 8 + 2 * j) * PITCH + e] | ((uint32_t)vt[(g * 8 + 2 * j + 1) * PITCH + e] << 16);
      *reinterpret_cast<u32x4*>(base + (int64_t)e * p.block_size + g * 8) = out;
    }
    return;
  }
  // Otherwise (ragged edges): lane -> position, wavefront -> head-dim rows.
  const int lane = tid & 63;
  const int wave = tid >> 6;
  if (lane < n_tok) {
    const int64_t pos = p.start_pos + t0 + lane;
    const int64_t lb = pos / p.block_size;
    const int64_t slot = pos - lb * p.block_size;
    const int64_t phys = p.table[lb];
    uint16_t* dst = p.v_pool + (phys * p.h_kv + h) * D * (int64_t)p.block_size + slot;
    for (int e = wave; e < D; e += kWavesPerGroup) dst[(int64_t)e * p.block_size] = vt[lane * PITCH + e];
  }
}

}  // namespace

hipError_t launch_kv_append(const AppendLaunch& p, int head_dim, hipStream_t stream) {
  const dim3 grid((p.chunk_len + kTileKeys - 1) / kTileKeys, p.h_kv), block(kGroupThreads);
  if (head_dim == 128) {
    hipLaunchKernelGGL(kv_append_kernel<128>, grid, block, 0, stream, p);
  } else {
    hipLaunchKernelGGL(kv_append_kernel<64>, grid, block, 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace mocap
