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
// One workgroup moves 64 positions of one KV head.  Every thread first issues
// all of its loads (the pools may alias nothing the loads read, but the
// compiler cannot know that, so loads placed after stores would wait for
// them), then writes its K rows out as 16-byte stores and scatters its V
// chunks into an LDS tile [D][64 positions].  After one barrier the tile
// leaves as 16-byte stores of 8 consecutive slots of one head-dim row (a
// whole 64-aligned tile), or 2-byte stores at ragged edges.
//
// LDS tile: row e holds the 64 positions of dim e (128 bytes); the 16-byte
// chunk q of row e (positions 8q .. 8q+7) is stored at chunk q ^ ((e / 8) % 8).
// A 2-byte write instruction then spreads its 16 dim rows over 8 chunk
// positions (at most two lanes of a wave per bank), and a 16-byte read
// instruction serves 16 lanes from two rows without conflicts.
#include "internal.h"

namespace mocap {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int v_slot(int e, int tok) { return (tok ^ (((e >> 3) & 7) << 3)); }

template <int D>
__global__ __launch_bounds__(kGroupThreads) void kv_append_kernel(const AppendLaunch p) {
  constexpr int ROW_CHUNKS = D / 8;                              // 16-byte chunks per position
  constexpr int PER = kTileKeys * ROW_CHUNKS / kGroupThreads;    // chunks per thread
  static_assert(PER * kGroupThreads == kTileKeys * ROW_CHUNKS, "whole tile per workgroup");
  __shared__ __attribute__((aligned(16))) uint16_t vt[D * kTileKeys];

  const int tid = threadIdx.x;
  const int t0 = blockIdx.x * kTileKeys;
  const int h = blockIdx.y;
  const int n_tok = min(kTileKeys, p.chunk_len - t0);
  const int64_t pos0 = p.start_pos + t0;
  // The 64 positions span at most two blocks (block_size is a multiple of 64).
  const int64_t lb0 = pos0 / p.block_size;
  const int64_t slot00 = pos0 - lb0 * p.block_size;
  const int split = (int)min<int64_t>(p.block_size - slot00, kTileKeys);  // positions [0, split) in lb0
  const int64_t phys0 = p.table[lb0];
  const int64_t phys1 = split < n_tok ? (int64_t)p.table[lb0 + 1] : phys0;

  u32x4 kr[PER], vr[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int c = j * kGroupThreads + tid;
    const int tok = c / ROW_CHUNKS, ch = c % ROW_CHUNKS;
    if (tok < n_tok) {
      const int64_t src = ((int64_t)(t0 + tok) * p.h_kv + h) * D + ch * 8;
      kr[j] = *reinterpret_cast<const u32x4*>(p.k_chunk + src);
      vr[j] = *reinterpret_cast<const u32x4*>(p.v_chunk + src);
    }
  }
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int c = j * kGroupThreads + tid;
    const int tok = c / ROW_CHUNKS, ch = c % ROW_CHUNKS;
    if (tok < n_tok) {
      const int64_t phys = tok < split ? phys0 : phys1;
      const int64_t slot = tok < split ? slot00 + tok : tok - split;
      *reinterpret_cast<u32x4*>(p.k_pool + ((phys * p.h_kv + h) * p.block_size + slot) * D + ch * 8) = kr[j];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int e = ch * 8 + 2 * w;
        vt[e * kTileKeys + v_slot(e, tok)] = (uint16_t)(vr[j][w] & 0xFFFFu);
        vt[(e + 1) * kTileKeys + v_slot(e + 1, tok)] = (uint16_t)(vr[j][w] >> 16);
      }
    }
  }
  __syncthreads();

  if (n_tok == kTileKeys && slot00 % kTileKeys == 0) {
    // A whole aligned tile (one block holds it): 8 consecutive slots of one
    // head-dim row per 16-byte store.
    uint16_t* base = p.v_pool + (phys0 * p.h_kv + h) * D * (int64_t)p.block_size + slot00;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int c = j * kGroupThreads + tid;
      const int e = c / (kTileKeys / 8), q = c % (kTileKeys / 8);
      const u32x4 out = *reinterpret_cast<const u32x4*>(vt + e * kTileKeys + v_slot(e, q * 8));
      *reinterpret_cast<u32x4*>(base + (int64_t)e * p.block_size + q * 8) = out;
    }
    return;
  }
  // Otherwise (ragged edges): lane -> position, wavefront -> head-dim rows.
  const int lane = tid & 63;
  const int wave = tid >> 6;
  if (lane < n_tok) {
    const int64_t phys = lane < split ? phys0 : phys1;
    const int64_t slot = lane < split ? slot00 + lane : lane - split;
    uint16_t* dst = p.v_pool + (phys * p.h_kv + h) * D * (int64_t)p.block_size + slot;
    for (int e = wave; e < D; e += kWavesPerGroup) dst[(int64_t)e * p.block_size] = vt[e * kTileKeys + v_slot(e, lane)];
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
