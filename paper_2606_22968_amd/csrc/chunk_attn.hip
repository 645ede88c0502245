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

#include <type_traits>

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

// Softmax bookkeeping.  Each query row keeps a reference exponent m (base 2)
// and accumulates p = exp2(s * scale * log2(e) - m) without taking block
// maxima.  m is only a scale: the result sum(p v) / sum(p) does not depend on
// it as long as nothing overflows, and fp32/bf16 keep their relative
// precision over the whole exponent range.  m is fixed by the first block of
// the row that has a visible key, while nothing has been accumulated yet, so
// the O accumulator never needs rescaling.  A later block whose partial row
// sum exceeds 2^kSumLimitLog2 (a score more than ~60 binary orders above the
// first block's maximum, which ordinary attention scores never reach) marks
// the row; after the pass the workgroup re-runs its key range once with m
// raised to the largest such block maximum.  O is therefore only ever written
// by MFMAs inside the loop.
constexpr float kSumLimit = 1152921504606846976.0f;  // 2^60

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef const __attribute__((address_space(4))) int32_t* const_i32_ptr;

// LDS layout of one stage (no padding; 16-byte chunks XOR-swizzled).  A
// ds_read_b128 serves 16 lanes at a time from 64 four-byte banks, so each run
// of 16 lanes must touch 16 different 16-byte bank groups of a 256-byte
// window:
//   K tile  [64 keys][D]      chunk c of key row r stored at c ^ k_swizzle(r)
//   V tile  [D][64 keys]      chunk c of dim row e stored at c ^ v_swizzle(e)
// K operand reads take 16 distinct rows per 16 lanes (key_row_order is a
// permutation of each aligned group of 16); V operand reads take 16
// consecutive dim rows of 128 bytes, two per 256-byte window.
template <int D>
__device__ __forceinline__ int k_swizzle(int r) {
  return D == 128 ? (r & 15) : ((r >> 1) & 7);
}
__device__ __forceinline__ int v_swizzle(int e) { return (e >> 1) & 7; }

__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

template <int N>
__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  bf16x2 v;
  v[0] = (__bf16)a;
  v[1] = (__bf16)b;
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c, false);
}

template <int D>
__global__ __launch_bounds__(kGroupThreads, 1) void chunk_attn_kernel(const AttnLaunch p) {
  // Device pass only: the host pass needs just the launch stub, and these
  // gfx950 builtins do not exist for the host target.
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int KS = D / 16;                     // k-steps of the score product
  constexpr int MD = D / 32;                     // 32-wide blocks of the head dim
  constexpr int K_ROW_CHUNKS = D / 8;            // 16-byte chunks per K row
  constexpr int V_ROW_CHUNKS = kTileKeys / 8;    // 16-byte chunks per V^T row
  constexpr int K_ELEMS = kTileKeys * D;
  constexpr int BUF_ELEMS = 2 * K_ELEMS;         // K tile + V^T tile
  constexpr int LOADS = K_ELEMS / 8 / kGroupThreads;  // 1 KiB wave loads per operand
  constexpr int TILE_OPS = 2 * LOADS;            // DMA instructions per thread per tile
  constexpr int STAGES = 4;

  __shared__ __attribute__((aligned(1024))) uint16_t lds[STAGES * BUF_ELEMS];

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
  const int wg_row0 = item.row_group * blocks_per_wg * kWaveRows;
  const int row0 = wg_row0 + (wave / hp) * kWaveRows;
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
  // Tiles [fast_begin, fast_end) are visible to every row of the workgroup
  // and need no mask.  At most one masked tile precedes them (a range start
  // inside a tile); the rest follow (the causal diagonal, a range end).
  const int n_head = (lo % kTileKeys) != 0 ? 1 : 0;
  const int fast_begin = tile_begin + n_head;
  const int fast_end = max(fast_begin, min(tile_end, min(hi, P + wg_row0 + 1) / kTileKeys));
  const int n_fast = fast_end - fast_begin;
  const int n_tiles = tile_end - tile_begin;
  // Processing order: the unmasked tiles first, then the head tile, then the
  // tail; softmax accumulation does not depend on the order of key blocks.
  auto seq_tile = [&](int i) -> int {
    if (i < n_fast) return fast_begin + i;
    if (i < n_fast + n_head) return tile_begin;
    return fast_end + (i - n_fast - n_head);
  };

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
  // the swizzle maps there.  Block-table entries are read with scalar loads.
  const const_i32_ptr table = (const_i32_ptr)p.table;
  const int64_t head_stride = (int64_t)D * p.block_size;  // elements per (block, head)
  int k_src[LOADS], v_src[LOADS];  // per-lane element offsets inside a tile
#pragma unroll
  for (int j = 0; j < LOADS; ++j) {
    const int chunk = (j * kWavesPerGroup + wave) * 64 + lane;
    const int kr = chunk / K_ROW_CHUNKS, kc = (chunk % K_ROW_CHUNKS) ^ k_swizzle<D>(kr);
    k_src[j] = kr * D + kc * 8;
    const int vr = chunk / V_ROW_CHUNKS, vc = (chunk % V_ROW_CHUNKS) ^ v_swizzle(vr);
    v_src[j] = vr * p.block_size + vc * 8;
  }
  // Sequence position i of the tile order uses LDS stage i % STAGES.
  auto issue_seq = [&](int i) {
    const int t = seq_tile(i);
    const int pos0 = t * kTileKeys;
    const int lb = pos0 / p.block_size;
    const int slot0 = pos0 - lb * p.block_size;
    const int64_t base = ((int64_t)table[lb] * p.h_kv + item.kv_head) * head_stride;
    const uint16_t* kb = p.k_pool + base + (int64_t)slot0 * D;
    const uint16_t* vb = p.v_pool + base + slot0;
    uint16_t* kl = lds + (i % STAGES) * BUF_ELEMS;
    uint16_t* vl = kl + K_ELEMS;
#pragma unroll
    for (int j = 0; j < LOADS; ++j) {
      const int dst = (j * kWavesPerGroup + wave) * 64 * 8;
      __builtin_amdgcn_global_load_lds(kb + k_src[j], (lds_ptr_t)(kl + dst), 16, 0, 0);
      __builtin_amdgcn_global_load_lds(vb + v_src[j], (lds_ptr_t)(vl + dst), 16, 0, 0);
    }
  };
  // Make sequence tile i visible to all waves.  `later` = tiles issued after
  // it that may still be in flight.
  auto publish_seq = [&](int i, int later) {
    if (later >= 2) {
      wait_vmem<2 * TILE_OPS>();
    } else if (later == 1) {
      wait_vmem<TILE_OPS>();
    } else {
      wait_vmem<0>();
    }
    lds_barrier();
    const int tstart = seq_tile(i) * kTileKeys;
    if (tstart + kTileKeys > valid_end) {
      // Keys at or beyond P + L are unwritten store memory: clear their V
      // columns so a zero probability never multiplies a NaN.
      uint16_t* vl = lds + (i % STAGES) * BUF_ELEMS + K_ELEMS;
      const int first = valid_end - tstart;
      for (int idx = tid; idx < D * kTileKeys; idx += kGroupThreads) {
        const int e = idx / kTileKeys, key = idx % kTileKeys;
        if (key >= first) vl[e * kTileKeys + (((key >> 3) ^ v_swizzle(e)) << 3) + (key & 7)] = 0;
      }
      lds_barrier();
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
  const int v_row_sw = v_swizzle(l32);               // V^T swizzle of this lane's dim rows
  const uint32_t ones = 0x3F803F80u;                 // bf16 pair (1, 1)

  // ---- building blocks of one 32-key half block ----
  auto scores = [&](f32x16 (&s)[2], const uint16_t* kl, int sb) {
    const int kr = sb * 32 + k_row_lo;
    const uint16_t* krow = kl + kr * D;
    const int ksw = k_swizzle<D>(kr);
    bf16x8 kf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      kf[ks] = *reinterpret_cast<const bf16x8*>(krow + (((ks * 2 + half) ^ ksw) << 3));
    s[0] = s[1] = f32x16{};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      s[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[ks], qf[0][ks], s[0], 0, 0, 0);
      s[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[ks], qf[1][ks], s[1], 0, 0, 0);
    }
  };
  auto pv = [&](const uint16_t* vl, int sb, const uint32_t (&pk)[2][8]) {
    bf16x8 vf[2][MD];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int vchunk = ((sb * 2 + kk) * 2 + half) ^ v_row_sw;
#pragma unroll
      for (int md = 0; md < MD; ++md)
        vf[kk][md] = *reinterpret_cast<const bf16x8*>(vl + (md * 32 + l32) * kTileKeys + (vchunk << 3));
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const bf16x8 pb0 = __builtin_bit_cast(bf16x8, u32x4{pk[0][kk * 4], pk[0][kk * 4 + 1], pk[0][kk * 4 + 2], pk[0][kk * 4 + 3]});
      const bf16x8 pb1 = __builtin_bit_cast(bf16x8, u32x4{pk[1][kk * 4], pk[1][kk * 4 + 1], pk[1][kk * 4 + 2], pk[1][kk * 4 + 3]});
#pragma unroll
      for (int md = 0; md < MD; ++md) {
        oacc[md][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[kk][md], pb0, oacc[md][0], 0, 0, 0);
        oacc[md][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[kk][md], pb1, oacc[md][1], 0, 0, 0);
      }
    }
  };
  // Visibility of this lane's 16 keys of a half block for query block nb, one
  // bit per accumulator element i (key offset (i/8)*16 + half*8 + i%8 from
  // `base`): keys in [lo, hi) and at or before the query's position.
  auto visible_bits = [&](int base, int nb) -> uint32_t {
    const int a = lo - base;
    const int b = min(hi, P + row0 + nb * 32 + l32 + 1) - base;
    // The offsets (i/8)*16 + i%8 increase with i, so the visible elements
    // form one run [first_i(a), first_i(b)).
    auto first_i = [](int x) { return x <= 0 ? 0 : x <= 8 ? x : x <= 16 ? 8 : x <= 24 ? x - 8 : 16; };
    const int i0 = first_i(a), i1 = first_i(b);
    return i1 > i0 ? (((1u << i1) - 1u) & ~((1u << i0) - 1u)) : 0u;
  };
  // Probabilities of query block nb: p = exp2(s * sl2 - m) as bf16 pairs,
  // masked elements cleared on the packed words (NaN-safe), and their sum.
  auto probs = [&](const f32x16& s, uint32_t (&pk)[8], float& rs, int nb, bool masked, uint32_t vis) {
    const float neg_m = -m_run[nb];
#pragma unroll
    for (int i = 0; i < 16; i += 2) {
      const float e0 = __builtin_amdgcn_exp2f(fmaf(s[i], sl2, neg_m));
      const float e1 = __builtin_amdgcn_exp2f(fmaf(s[i + 1], sl2, neg_m));
      pk[i / 2] = pack_bf16x2(e0, e1);
    }
    if (masked) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t lo_half = (uint32_t)__builtin_amdgcn_sbfe((int)vis, 2 * j, 1);
        const uint32_t hi_half = (uint32_t)__builtin_amdgcn_sbfe((int)vis, 2 * j + 1, 1);
        pk[j] &= (lo_half & 0x0000FFFFu) | (hi_half & 0xFFFF0000u);
      }
    }
    float acc = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) acc = dot2_bf16(pk[j], ones, acc);
    rs = acc;
  };
  // Accept the half block's probabilities.  Rarely (first visible block of a
  // row, or an overflow) take the slow path: rows with nothing accumulated
  // adopt the block maximum as their reference exponent and recompute; rows
  // that have accumulated are marked for the re-run.  Partner lanes (l and
  // l ^ 32) hold the same row and always decide together.
  float m_cand[2] = {-INFINITY, -INFINITY};
  bool rerun = false;
  auto settle = [&](const f32x16 (&s)[2], uint32_t (&pk)[2][8], float (&rs)[2], const uint32_t (&vis)[2]) {
    const bool over = !(rs[0] <= kSumLimit) || !(rs[1] <= kSumLimit);
    if (__builtin_amdgcn_ballot_w64(over) != 0) {
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        const bool row_over = lane_pair_max(!(rs[nb] <= kSumLimit) ? 1.f : 0.f) > 0.f;
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if ((vis[nb] >> i) & 1u) mx = fmaxf(mx, s[nb][i]);
        mx = lane_pair_max(mx) * sl2;
        const bool fresh = lane_pair_sum(l_run[nb]) == 0.f;
        if (row_over && !fresh) {
          m_cand[nb] = fmaxf(m_cand[nb], mx);
          rerun = true;
        }
        if (row_over && fresh) m_run[nb] = mx;
        const float neg_m = m_run[nb] == -INFINITY ? 0.f : -m_run[nb];
        float acc = 0.f;
        uint32_t fixed[8];
#pragma unroll
        for (int i = 0; i < 16; i += 2) {
          const float e0 = ((vis[nb] >> i) & 1u) ? __builtin_amdgcn_exp2f(fmaf(s[nb][i], sl2, neg_m)) : 0.f;
          const float e1 = ((vis[nb] >> (i + 1)) & 1u) ? __builtin_amdgcn_exp2f(fmaf(s[nb][i + 1], sl2, neg_m)) : 0.f;
          fixed[i / 2] = pack_bf16x2(e0, e1);
          acc = dot2_bf16(fixed[i / 2], ones, acc);
        }
        if (row_over && fresh) {
#pragma unroll
          for (int j = 0; j < 8; ++j) pk[nb][j] = fixed[j];
          rs[nb] = acc;
        }
      }
    }
    l_run[0] += rs[0];
    l_run[1] += rs[1];
  };

  // ---- software pipeline over 32-key half blocks ----
  // Per tile t (halves 0 and 1) the MFMA stream is
  //   S1(t) | PV0(t) | S0(t+1) | PV1(t)
  // and each group overlaps the exp/pack work of one query block of the
  // half block whose scores are ready:
  //   S1(t): probs(S0(t), nb 1)      PV0(t): probs(S1(t), nb 0)
  //   S0(t+1): probs(S1(t), nb 1)    PV1(t): probs(S0(t+1), nb 0)
  // PV1(t) reads tile t after the barrier that publishes tile t+1, so the
  // stage of tile t-1 is the first one free for refilling (tile t+3).
  f32x16 s0[2], s1[2];
  uint32_t pk0[2][8], pk1[2][8];
  float rs0[2], rs1[2];
  uint32_t vis0[2] = {0xFFFFu, 0xFFFFu}, vis1[2] = {0xFFFFu, 0xFFFFu};

  auto masked_seq = [&](int i) { return i >= n_fast; };
  auto set_vis = [&](uint32_t (&vis)[2], int i, int sb) {
    if (masked_seq(i)) {
      const int base = seq_tile(i) * kTileKeys + sb * 32 + half * 8;
      vis[0] = visible_bits(base, 0);
      vis[1] = visible_bits(base, 1);
    } else {
      vis[0] = vis[1] = 0xFFFFu;
    }
  };

  // One tile of the pipeline.  MASK selects the masked variant of the
  // probability computation for the tiles touched by this step.
  auto step = [&](int i, auto mask_tag) {
    constexpr bool MASK = decltype(mask_tag)::value;
    const uint16_t* kl = lds + (i % STAGES) * BUF_ELEMS;
    const uint16_t* vl = kl + K_ELEMS;
    const bool has_next = i + 1 < n_tiles;
    // S1(t) | probs(S0(t), nb 1)
    scores(s1, kl, 1);
    probs(s0[1], pk0[1], rs0[1], 1, MASK, vis0[1]);
    settle(s0, pk0, rs0, vis0);
    // PV0(t) | probs(S1(t), nb 0)
    if (MASK) set_vis(vis1, i, 1);
    pv(vl, 0, pk0);
    probs(s1[0], pk1[0], rs1[0], 0, MASK, vis1[0]);
    // Publish tile t+1, refill the stage of tile t-1 with tile t+3.
    if (has_next) {
      publish_seq(i + 1, min(n_tiles - (i + 2), 1));
      if (i + 3 < n_tiles) issue_seq(i + 3);
    }
    // S0(t+1) | probs(S1(t), nb 1).  On the last tile the scores are
    // computed from the current stage and discarded.
    const uint16_t* kn = has_next ? lds + ((i + 1) % STAGES) * BUF_ELEMS : kl;
    scores(s0, kn, 0);
    probs(s1[1], pk1[1], rs1[1], 1, MASK, vis1[1]);
    settle(s1, pk1, rs1, vis1);
    // PV1(t) | probs(S0(t+1), nb 0)
    if (MASK && has_next) set_vis(vis0, i + 1, 0);
    pv(vl, 1, pk1);
    probs(s0[0], pk0[0], rs0[0], 0, MASK, vis0[0]);
  };

  __shared__ int rerun_flag;
  for (int pass = 0; pass < 2 && n_tiles > 0; ++pass) {
    if (tid == 0) rerun_flag = 0;
    issue_seq(0);
    if (n_tiles > 1) issue_seq(1);
    if (n_tiles > 2) issue_seq(2);
    publish_seq(0, min(n_tiles - 1, 2));
    set_vis(vis0, 0, 0);
    scores(s0, lds, 0);
    probs(s0[0], pk0[0], rs0[0], 0, masked_seq(0), vis0[0]);
    // Steps whose tile and next tile are both unmasked use the mask-free
    // variant; all others the masked one.
    int i = 0;
    for (; i + 1 < n_fast; ++i) step(i, std::integral_constant<bool, false>{});
    for (; i < n_tiles; ++i) step(i, std::integral_constant<bool, true>{});

    // Re-run the range if any row of the workgroup overflowed its reference
    // exponent (all DMA has drained: the last publish waited for vmcnt(0)).
    if (pass == 0 && __builtin_amdgcn_ballot_w64(rerun) != 0 && lane == 0) atomicOr(&rerun_flag, 1);
    lds_barrier();
    const bool again = rerun_flag != 0;
    lds_barrier();
    if (!again) break;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      m_run[nb] = fmaxf(m_run[nb], m_cand[nb]);
      m_cand[nb] = -INFINITY;
      l_run[nb] = 0.f;
#pragma unroll
      for (int md = 0; md < MD; ++md) oacc[md][nb] = f32x16{};
    }
    rerun = false;
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
#endif  // __HIP_DEVICE_COMPILE__
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
