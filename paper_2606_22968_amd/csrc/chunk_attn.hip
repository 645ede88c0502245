// Chunked causal prefill attention for gfx950 (CDNA4).
//
// One chunk's queries attend to the prefix keys (no mask) and to the chunk's
// own keys (causal), as in Section 2.2 of the paper; the work of the chunk
// grows with its prefix as Eq. (1) of Section 3.2 describes.
//
// Kernel structure
//   * A workgroup is 4 wavefronts.  Each wavefront owns 64 query rows of one
//     query head, kept in registers as the B operand of the score product.
//     The 4 wavefronts of a workgroup share one KV head (GQA packing): each
//     K/V tile staged in LDS serves all of them.
//   * K/V advance in tiles of 64 keys, copied global -> LDS directly
//     (global_load_lds_dwordx4, no staging registers) into two stages: tile
//     t+1 is in flight while tile t is consumed; one barrier per tile.
//   * Scores are computed transposed, S^T = K Q^T, with
//     v_mfma_f32_32x32x16_bf16: a lane's accumulator then holds one query and
//     16 keys, so row statistics need one cross-half exchange
//     (v_permlane32_swap) and the probabilities are already in the B-operand
//     layout of O^T += V^T P^T.  K rows are fetched in a bit-swapped order
//     (bits 2 and 3 of the row index exchanged) so that each lane's 8
//     probabilities of a P*V step belong to 8 consecutive keys, which are 16
//     contiguous bytes of the key-contiguous V layout.
//   * Online softmax in base 2 with scale*log2(e) folded into one FMA.
//   * Only tiles that straddle the causal diagonal or a range edge are
//     masked; tiles entirely above the diagonal are never visited.  Keys at or
//     beyond P+L (unwritten store memory) are zero-filled in LDS so a masked
//     probability of 0 never meets a NaN.
//   * Optional split of the prefix into ranges: each range writes normalised
//     fp32 partials and their log-sum-exp; lse_merge.hip combines them.
#include "internal.h"

#include <math.h>

namespace mocap {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float lane_pair_max(float x) {
  // v_permlane32_swap exchanges the upper half of one operand with the lower
  // half of the other; the max over both results is max(x[l], x[l ^ 32]).
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float lane_pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Row order of K inside a 32-key MFMA block: bits 2 and 3 swapped.
__device__ __forceinline__ int key_row_order(int m) {
  return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1);
}

struct WorkItem {
  int kv_head;
  int head0;      // first query head of the workgroup
  int row_group;  // index of the workgroup's block of rows
  int range;      // KV range index
};

// Workgroup ids are handed to the 8 XCDs round robin.  Renumber them so each
// XCD receives one contiguous run of logical items: consecutive items share a
// KV head, so the tiles they stream stay in that XCD's L2.  Within a KV head
// the logical order is range, then row group from the last (longest) one
// down, then the head blocks of the group.
__device__ __forceinline__ WorkItem decode_item(const AttnLaunch& p, int hw_id) {
  const int n = p.total_wgs;
  const int xcd = hw_id & 7, slot = hw_id >> 3;
  const int per = n >> 3, rem = n & 7;
  const int logical = xcd * per + min(xcd, rem) + slot;

  const int head_blocks = p.group / p.heads_per_wg;
  const int per_range = head_blocks * p.row_groups;
  const int per_kv = per_range * p.n_ranges;
  WorkItem w;
  w.kv_head = logical / per_kv;
  int r = logical - w.kv_head * per_kv;
  w.range = r / per_range;
  r -= w.range * per_range;
  w.row_group = p.row_groups - 1 - r / head_blocks;
  const int hb = r - (r / head_blocks) * head_blocks;
  w.head0 = w.kv_head * p.group + hb * p.heads_per_wg;
  return w;
}

// Rows keep a running maximum m (base-2 units) that only moves when a block's
// maximum exceeds it by more than kRescaleSlack; between moves the
// probabilities exp2(s - m) stay below 2^kRescaleSlack, which fp32 sums and
// bf16 probabilities hold without loss of relative precision.  The final
// normalisation uses the same m for numerator and denominator, so the result
// does not depend on when m moved.  The O accumulator is therefore rescaled
// only on those rare moves, and a 64-key tile can be consumed as two
// independent 32-key halves.
constexpr float kRescaleSlack = 8.0f;

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// LDS layout of one stage (no padding; 16-byte chunks XOR-swizzled so the
// MFMA operand reads of 8 consecutive lanes hit 8 different 16-byte bank
// groups):
//   K tile  [64 keys][D]      chunk c of key row r stored at c ^ k_swizzle(r)
//   V tile  [D][64 keys]      chunk c of dim row e stored at c ^ (e & 7)
// K operand reads take rows key_row_order(0..7) = {0,1,2,3,8,9,10,11} per
// 8 lanes; k_swizzle separates r from r + 8.
__device__ __forceinline__ int k_swizzle(int r) { return (r & 7) ^ ((r >> 1) & 4); }

template <int D>
__global__ __launch_bounds__(kGroupThreads, 1) void chunk_attn_kernel(const AttnLaunch p) {
  constexpr int KS = D / 16;                     // k-steps of the score product
  constexpr int MD = D / 32;                     // 32-wide blocks of the head dim
  constexpr int K_ROW_CHUNKS = D / 8;            // 16-byte chunks per K row
  constexpr int V_ROW_CHUNKS = kTileKeys / 8;    // 16-byte chunks per V^T row
  constexpr int K_ELEMS = kTileKeys * D;
  constexpr int BUF_ELEMS = 2 * K_ELEMS;         // K tile + V^T tile
  constexpr int LOADS = K_ELEMS / 8 / kGroupThreads;  // 1 KiB wave loads per operand

  __shared__ __attribute__((aligned(1024))) uint16_t lds[2 * BUF_ELEMS];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int half = lane >> 5;
  const int l32 = lane & 31;

  const WorkItem item = decode_item(p, blockIdx.x);
  const int P = p.prefix_len;
  const int L = p.chunk_len;
  const int hp = p.heads_per_wg;
  const int blocks_per_wg = kWavesPerGroup / hp;
  const int head = item.head0 + (wave % hp);
  const int row0 = (item.row_group * blocks_per_wg + wave / hp) * kWaveRows;
  const int wg_row_end = min(L, (item.row_group + 1) * blocks_per_wg * kWaveRows);

  // Key range [lo, hi) of this launch item.
  int lo, hi;
  if (p.n_ranges == 1) {
    lo = 0;
    hi = P + L;
  } else if (item.range < p.n_ranges - 1) {
    const int parts = p.n_ranges - 1;
    lo = (int)((int64_t)p.prefix_tiles * item.range / parts) * kTileKeys;
    hi = min((int)((int64_t)p.prefix_tiles * (item.range + 1) / parts) * kTileKeys, P);
  } else {
    lo = P;
    hi = P + L;
  }
  const int wg_hi = min(hi, P + wg_row_end);
  const int tile_begin = lo / kTileKeys;
  const int tile_end = (wg_hi + kTileKeys - 1) / kTileKeys;
  const int valid_end = P + L;

  // Rows of this wavefront.  Keys at or beyond my_key_hi are masked for all of
  // them; keys in [lo, full_vis_hi) are visible to all of them.
  const int my_rows = min(row0 + kWaveRows, L) - row0;
  const int my_key_hi = my_rows > 0 ? min(hi, P + row0 + my_rows) : INT32_MIN;
  const int full_vis_hi = min(hi, P + row0 + 1);

  // ---- Q fragments (B operand of S^T = K Q^T) ----
  bf16x8 qf[2][KS];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int row = row0 + nb * 32 + l32;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (row < L) {
        qf[nb][ks] = *reinterpret_cast<const bf16x8*>(
            p.q + ((int64_t)row * p.h_q + head) * D + ks * 16 + half * 8);
      } else {
        qf[nb][ks] = bf16x8{};
      }
    }
  }

  // ---- tile staging: global -> LDS directly (global_load_lds_dwordx4) ----
  // Wave instruction j writes LDS chunks [(j*4 + wave)*64, +64) of an operand;
  // lane i fills chunk (j*4 + wave)*64 + i and fetches the global chunk that
  // the swizzle maps there.
  const int64_t head_stride = (int64_t)D * p.block_size;  // elements per (block, head)
  int k_src[LOADS], v_src[LOADS];  // per-lane element offsets inside a tile
#pragma unroll
  for (int j = 0; j < LOADS; ++j) {
    const int chunk = (j * kWavesPerGroup + wave) * 64 + lane;
    const int kr = chunk / K_ROW_CHUNKS, kc = (chunk % K_ROW_CHUNKS) ^ k_swizzle(kr);
    k_src[j] = kr * D + kc * 8;
    const int vr = chunk / V_ROW_CHUNKS, vc = (chunk % V_ROW_CHUNKS) ^ (vr & 7);
    v_src[j] = vr * p.block_size + vc * 8;
  }
  auto issue_tile = [&](int buf, int t) {
    const int pos0 = t * kTileKeys;
    const int lb = pos0 / p.block_size;
    const int slot0 = pos0 - lb * p.block_size;
    const int64_t base = ((int64_t)p.table[lb] * p.h_kv + item.kv_head) * head_stride;
    const uint16_t* kb = p.k_pool + base + (int64_t)slot0 * D;
    const uint16_t* vb = p.v_pool + base + slot0;
    uint16_t* kl = lds + buf * BUF_ELEMS;
    uint16_t* vl = kl + K_ELEMS;
#pragma unroll
    for (int j = 0; j < LOADS; ++j) {
      const int dst = (j * kWavesPerGroup + wave) * 64 * 8;
      __builtin_amdgcn_global_load_lds(kb + k_src[j], (lds_ptr_t)(kl + dst), 16, 0, 0);
      __builtin_amdgcn_global_load_lds(vb + v_src[j], (lds_ptr_t)(vl + dst), 16, 0, 0);
    }
  };

  f32x16 oacc[MD][2];
#pragma unroll
  for (int md = 0; md < MD; ++md) {
    oacc[md][0] = f32x16{};
    oacc[md][1] = f32x16{};
  }
  float m_run[2] = {-INFINITY, -INFINITY};
  float l_run[2] = {0.f, 0.f};
  const float sl2 = p.scale_log2;
  const int k_row_lo = key_row_order(l32);          // K row within a 32-key half
  const int v_row_sw = l32 & 7;                      // V^T swizzle of this lane's dim rows

  if (tile_begin < tile_end) issue_tile(0, tile_begin);

  for (int t = tile_begin; t < tile_end; ++t) {
    const int buf = (t - tile_begin) & 1;
    const int tstart = t * kTileKeys;
    // Tile t has landed for this thread; the barrier makes it visible to all
    // and guarantees every wave is done with the buffer refilled next.
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    __syncthreads();
    if (tstart + kTileKeys > valid_end) {
      // Keys at or beyond P + L are unwritten store memory: clear their V
      // columns so a zero probability never multiplies a NaN.
      uint16_t* vl = lds + buf * BUF_ELEMS + K_ELEMS;
      const int first = valid_end - tstart;
      for (int idx = tid; idx < D * kTileKeys; idx += kGroupThreads) {
        const int e = idx / kTileKeys, key = idx % kTileKeys;
        if (key >= first) vl[e * kTileKeys + (((key >> 3) ^ (e & 7)) << 3) + (key & 7)] = 0;
      }
      __syncthreads();
    }
    if (t + 1 < tile_end) issue_tile(buf ^ 1, t + 1);

    if (tstart < my_key_hi) {
      const uint16_t* kl = lds + buf * BUF_ELEMS;
      const uint16_t* vl = kl + K_ELEMS;
      const bool need_mask = tstart < lo || tstart + kTileKeys > full_vis_hi;

#pragma unroll
      for (int sb = 0; sb < 2; ++sb) {
        // S^T = K Q^T for 32 keys x 64 queries.
        f32x16 s[2];
        s[0] = s[1] = f32x16{};
        const int kr = sb * 32 + k_row_lo;
        const uint16_t* krow = kl + kr * D;
        const int ksw = k_swizzle(kr);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(krow + (((ks * 2 + half) ^ ksw) << 3));
          s[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[0][ks], s[0], 0, 0, 0);
          s[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[1][ks], s[1], 0, 0, 0);
        }

        // Element i of the accumulator holds key sb*32 + (i/8)*16 + half*8 + i%8.
        if (need_mask) {
#pragma unroll
          for (int nb = 0; nb < 2; ++nb) {
            const int base = tstart + sb * 32 + half * 8;
            const int lim_lo = lo - base;
            const int lim_hi = min(hi, P + row0 + nb * 32 + l32 + 1) - base;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
              const int c = (i / 8) * 16 + (i % 8);
              if (c < lim_lo || c >= lim_hi) s[nb][i] = -INFINITY;
            }
          }
        }

        bf16x8 pb[2][2];
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
          float mx = s[nb][0];
#pragma unroll
          for (int i = 1; i < 16; ++i) mx = fmaxf(mx, s[nb][i]);
          mx = lane_pair_max(mx) * sl2;
          if (__builtin_amdgcn_ballot_w64(mx > m_run[nb] + kRescaleSlack) != 0) {
            const float m_new = fmaxf(m_run[nb], mx);
            const float alpha = __builtin_amdgcn_exp2f(m_run[nb] - (m_new == -INFINITY ? 0.f : m_new));
            l_run[nb] *= alpha;
#pragma unroll
            for (int md = 0; md < MD; ++md) oacc[md][nb] *= alpha;
            m_run[nb] = m_new;
          }
          const float neg_m = m_run[nb] == -INFINITY ? 0.f : -m_run[nb];
          float rs = 0.f;
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const float e = __builtin_amdgcn_exp2f(fmaf(s[nb][i], sl2, neg_m));
            rs += e;
            pb[nb][i / 8][i % 8] = (__bf16)e;
          }
          l_run[nb] += rs;
        }

        // O^T += V^T P^T over these 32 keys (2 k-steps of 16).
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          const int vchunk = ((sb * 2 + kk) * 2 + half) ^ v_row_sw;
#pragma unroll
          for (int md = 0; md < MD; ++md) {
            const bf16x8 a = *reinterpret_cast<const bf16x8*>(vl + (md * 32 + l32) * kTileKeys + (vchunk << 3));
            oacc[md][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[0][kk], oacc[md][0], 0, 0, 0);
            oacc[md][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[1][kk], oacc[md][1], 0, 0, 0);
          }
        }
      }
    }
  }

  // ---- epilogue ----
  const bool split = p.n_ranges > 1;
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const float l_tot = lane_pair_sum(l_run[nb]);
    const int row = row0 + nb * 32 + l32;
    if (row >= L) continue;
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const float row_lse = l_tot > 0.f ? (m_run[nb] + log2f(l_tot)) * kLn2 : -INFINITY;
    if (!split) {
      uint16_t* orow = p.o + ((int64_t)row * p.h_q + head) * D;
#pragma unroll
      for (int md = 0; md < MD; ++md) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          bf16x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = (__bf16)(oacc[md][nb][j * 4 + e] * inv);
          *reinterpret_cast<bf16x4*>(orow + md * 32 + j * 8 + half * 4) = v;
        }
      }
      if (half == 0) p.lse[(int64_t)head * L + row] = row_lse;
    } else {
      const int64_t base = ((int64_t)item.range * p.h_q + head) * L + row;
      float* orow = p.ws_o + base * D;
#pragma unroll
      for (int md = 0; md < MD; ++md) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          f32x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = oacc[md][nb][j * 4 + e] * inv;
          *reinterpret_cast<f32x4*>(orow + md * 32 + j * 8 + half * 4) = v;
        }
      }
      if (half == 0) p.ws_lse[base] = row_lse;
    }
  }
}

}  // namespace

hipError_t launch_chunk_attn(const AttnLaunch& p, int head_dim, hipStream_t stream) {
  const dim3 grid(p.total_wgs), block(kGroupThreads);
  if (head_dim == 128) {
    hipLaunchKernelGGL(chunk_attn_kernel<128>, grid, block, 0, stream, p);
  } else {
    hipLaunchKernelGGL(chunk_attn_kernel<64>, grid, block, 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace mocap
