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
// One workgroup moves 32 positions of one KV head, one 16-byte chunk of K and
// one of V per thread (D / 8 threads per position: 512 threads for D = 128):
// many small workgroups keep more of the chip's load queues busy than a few
// large ones.  Each thread issues both loads first (the pools may alias
// nothing the loads read, but the compiler cannot know that, so a load placed
// after a store would wait for it), writes its K chunk out as one 16-byte
// store and scatters its V chunk into an LDS tile [D][32 positions].  After
// one barrier the tile leaves as 16-byte stores of 8 consecutive slots of one
// head-dim row (a whole 32-aligned tile), or 2-byte stores at ragged edges.
//
// LDS tile: 16-byte chunk (e, q) holds positions 8q .. 8q+7 of dim e and is
// stored at chunk slot (4 e + q) ^ ((e / 8) % 16).  For D = 128 a 2-byte
// write instruction (16 chunk columns ch, dims e = 8 ch + k, positions
// t, t+2, t+4, t+6) then lands in 16 distinct groups of four banks, one
// dword of each bank, and the 16 lanes that a 16-byte read serves at a time
// (chunks 16 m .. 16 m + 15) stay in distinct groups too: no bank conflicts.
// (D = 64 has 8 chunk columns and writes two lanes per bank.)
#include "internal.h"

namespace mocap {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kAppendTokens = 32;  // positions per workgroup (4 chunks of 8 per dim row)

template <int D>
constexpr int append_threads() { return kAppendTokens * (D / 8); }

// Element index of (dim e, position tok) in the tile.
__device__ __forceinline__ int v_index(int e, int tok) {
  return ((((e << 2) + (tok >> 3)) ^ ((e >> 3) & 15)) << 3) + (tok & 7);
}

template <int D>
__global__ __launch_bounds__(append_threads<D>()) void kv_append_kernel(const AppendLaunch p) {
  constexpr int T = kAppendTokens;
  constexpr int ROW_CHUNKS = D / 8;  // 16-byte chunks per position
  constexpr int NT = append_threads<D>();
  __shared__ __attribute__((aligned(16))) uint16_t vt[D * T];

  const int tid = threadIdx.x;
  const int t0 = blockIdx.x * T;
  const int h = blockIdx.y;
  const int n_tok = min(T, p.chunk_len - t0);
  const int64_t pos0 = p.start_pos + t0;
  // The 32 positions span at most two blocks (block_size is a multiple of 64).
  const int64_t lb0 = pos0 / p.block_size;
  const int64_t slot00 = pos0 - lb0 * p.block_size;
  const int split = (int)min<int64_t>(p.block_size - slot00, T);  // positions [0, split) in lb0
  const int64_t phys0 = p.table[lb0];
  const int64_t phys1 = split < n_tok ? (int64_t)p.table[lb0 + 1] : phys0;

  // Thread -> (position, chunk): the D / 8 lanes of a position read its
  // whole K and V rows, consecutive 16-byte pieces.  A wavefront takes every
  // other position of 2 * PW consecutive ones (wave pairs share them), so its
  // 2-byte tile writes cover all four dwords of each 16-byte chunk.
  constexpr int PW = 64 / ROW_CHUNKS;  // positions per wavefront
  const int wv = tid >> 6, wl = tid & 63;
  const int tok = (wv >> 1) * 2 * PW + (wv & 1) + 2 * (wl / ROW_CHUNKS), ch = wl % ROW_CHUNKS;
  if (tok < n_tok) {
    const int64_t src = ((int64_t)(t0 + tok) * p.h_kv + h) * D + ch * 8;
    const u32x4 kr = *reinterpret_cast<const u32x4*>(p.k_chunk + src);
    const u32x4 vr = *reinterpret_cast<const u32x4*>(p.v_chunk + src);
    const int64_t phys = tok < split ? phys0 : phys1;
    const int64_t slot = tok < split ? slot00 + tok : tok - split;
    *reinterpret_cast<u32x4*>(p.k_pool + ((phys * p.h_kv + h) * p.block_size + slot) * D + ch * 8) = kr;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const int e = ch * 8 + 2 * w;
      vt[v_index(e, tok)] = (uint16_t)(vr[w] & 0xFFFFu);
      vt[v_index(e + 1, tok)] = (uint16_t)(vr[w] >> 16);
    }
  }
  __syncthreads();

  if (n_tok == T && slot00 % T == 0) {
    // A whole aligned tile (one block holds it): thread -> (dim row e, chunk
    // q), 8 consecutive slots of one head-dim row per 16-byte store.
    uint16_t* base = p.v_pool + (phys0 * p.h_kv + h) * D * (int64_t)p.block_size + slot00;
    const int e = tid / (T / 8), q = tid % (T / 8);
    const u32x4 out = *reinterpret_cast<const u32x4*>(vt + v_index(e, q * 8));
    *reinterpret_cast<u32x4*>(base + (int64_t)e * p.block_size + q * 8) = out;
    return;
  }
  // Otherwise (ragged edges): thread -> (position, one of NT / T dim rows).
  const int lt = tid % T, lr = tid / T;
  if (lt < n_tok) {
    const int64_t phys = lt < split ? phys0 : phys1;
    const int64_t slot = lt < split ? slot00 + lt : lt - split;
    uint16_t* dst = p.v_pool + (phys * p.h_kv + h) * D * (int64_t)p.block_size + slot;
    for (int e = lr; e < D; e += NT / T) dst[(int64_t)e * p.block_size] = vt[v_index(e, lt)];
  }
}

}  // namespace

hipError_t launch_kv_append(const AppendLaunch& p, int head_dim, hipStream_t stream) {
  const dim3 grid((p.chunk_len + kAppendTokens - 1) / kAppendTokens, p.h_kv);
  if (head_dim == 128) {
    hipLaunchKernelGGL(kv_append_kernel<128>, grid, dim3(append_threads<128>()), 0, stream, p);
  } else {
    hipLaunchKernelGGL(kv_append_kernel<64>, grid, dim3(append_threads<64>()), 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace mocap
