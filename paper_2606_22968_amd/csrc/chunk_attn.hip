// Chunked causal prefill attention for gfx950 (CDNA4).
//
// One chunk's queries attend to the prefix keys (no mask) and to the chunk's
// own keys (causal), as in Section 2.2 of the paper; the work of the chunk
// grows with its prefix as Eq. (1) of Section 3.2 describes.
//
// Kernel structure
//   * A workgroup is 8 wavefronts, two per SIMD, each within 256 registers.
//     Each wavefront owns 32 query rows of one query head, kept in registers
//     as the B operand of the score product.  All wavefronts of a workgroup
//     share one KV head (GQA packing), so each K/V tile staged in LDS serves
//     every query head of the group.
//   * Causal balance: the workgroup's two units of four waves take two row
//     groups of the same query heads, r and R-1-r (mirrored, so every
//     workgroup carries about the same number of (row, key) pairs) or two
//     adjacent ones (when many workgroups per CU even out their lengths);
//     the host picks per launch.  Each wave follows its own key range and
//     treats the tiles all its rows see in full as unmasked.  In a mirrored
//     pair, the last tiles only the longer row group sees are shared: the
//     shorter group's wave stores its rows, takes over its partner's rows
//     and computes the second 32-key half of each such tile while the
//     partner computes the first; the two partial results meet in LDS.
//   * K/V advance in tiles of 64 keys, copied global -> LDS directly
//     (buffer_load_dwordx4 ... lds, no staging registers) into a 4-stage ring
//     (128 KiB at head_dim 128), prefetched two tiles ahead, one workgroup
//     barrier per tile.  Even tiles are copied by waves 0-3 and odd tiles by
//     waves 4-7, so each wave computes a tile's addresses every other tile.
//   * Software pipelining inside each wavefront, in two complementary orders
//     for the two waves of a SIMD.  Waves 0-3: tile k's scores (MFMAs only),
//     then tile k-1's P*V with tile k's exp/pack/row-sum work woven in at a
//     fixed ratio (two scores per MFMA, four at head_dim 64); the
//     probabilities alternate between two register buffers.  Waves 4-7: tile
//     k's scores with tile k-1's softmax work woven in (at raised wave
//     priority), then tile k-1's P*V alone.  So while one wave of a SIMD
//     interleaves vector work with its MFMAs, the other mostly issues MFMAs.
//     LDS operand fragments are read two or more MFMAs ahead.
//   * Scores are computed transposed, S^T = K Q^T, with
//     v_mfma_f32_32x32x16_bf16: a lane's accumulator then holds one query and
//     16 keys, so row statistics need one cross-half exchange
//     (v_permlane32_swap) and the probabilities are already in the B-operand
//     layout of O^T += V^T P^T.  K rows are fetched in a bit-swapped order
//     (bits 2 and 3 of the row index exchanged) so that each lane's 8
//     probabilities of a P*V step belong to 8 consecutive keys, which are 16
//     contiguous bytes of the key-contiguous V layout.
//   * Softmax in base 2 with scale*log2(e) folded into one FMA, without block
//     maxima (see the bookkeeping note below).  Each row keeps two sums: the
//     bf16 probabilities that feed P*V (added with v_dot2), which normalise O
//     so numerator and denominator agree, and the fp32 exponentials before
//     rounding, which give the log-sum-exp (a bf16 sum would carry the 2^-8
//     rounding of a dominant probability into the LSE).
//   * Only tiles that straddle the causal diagonal or a range edge are
//     masked (their hidden scores are set to -inf before the exponentials);
//     tiles entirely above the diagonal are never visited.  Keys at or beyond
//     P+L (unwritten store memory) are zero-filled in LDS so a probability of
//     0 never meets a NaN.
//   * Optional split of the prefix into ranges: each range writes normalised
//     fp32 partials and their log-sum-exp; lse_merge.hip combines them.
//   * A run of prefix tiles may come from a second store (a debtor stage's
//     remote KV portion, Section 4.1): the store is chosen per tile.
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
  int head0;        // first query head of both units
  int row_group_a;  // row group of waves 0-3
  int row_group_b;  // row group of waves 4-7 (-1: none)
  int range;        // KV range index
};

// Workgroup ids are handed to the 8 XCDs round robin.  Renumber them so each
// XCD receives one contiguous run of logical items: consecutive items share a
// KV head, so the tiles they stream stay in that XCD's L2.  Within a KV head
// the logical order is range, then row-group pair (pair q holds row groups q
// and R-1-q; the middle group of an odd R is alone), then the head blocks of
// the group.
__device__ __forceinline__ WorkItem decode_item(const AttnLaunch& p, int hw_id) {
  const int n = p.total_wgs;
  const int xcd = hw_id & 7, slot = hw_id >> 3;
  const int per = n >> 3, rem = n & 7;
  const int logical = xcd * per + min(xcd, rem) + slot;

  const int head_blocks = p.group / p.heads_per_unit;
  const int per_range = head_blocks * p.pairs;
  const int per_kv = per_range * p.n_ranges;
  WorkItem w;
  w.kv_head = logical / per_kv;
  int r = logical - w.kv_head * per_kv;
  w.range = r / per_range;
  r -= w.range * per_range;
  const int pair = r / head_blocks;
  const int hb = r - pair * head_blocks;
  // Unit A takes the lower row group of the pair, unit B the higher (-1: none).
  if (p.pair_adjacent) {
    const int top = p.row_groups - 1 - 2 * pair;
    w.row_group_a = top > 0 ? top - 1 : top;
    w.row_group_b = top > 0 ? top : -1;
  } else {
    w.row_group_a = pair;
    w.row_group_b = p.row_groups - 1 - pair;
    if (w.row_group_b == pair) w.row_group_b = -1;
  }
  w.head0 = w.kv_head * p.group + hb * p.heads_per_unit;
  return w;
}

// Softmax bookkeeping.  Each query row keeps a reference exponent m (base 2)
// and accumulates p = exp2(s * scale * log2(e) - m) without taking block
// maxima.  m is only a scale: the result sum(p v) / sum(p) does not depend on
// it as long as nothing overflows, and fp32/bf16 keep their relative
// precision over the whole exponent range.  m is fixed by the first block of
// the row that has a visible key, while nothing has been accumulated yet, so
// the O accumulator never needs rescaling.  A later block whose partial row
// sum exceeds kSumLimit = 2^60 (a score more than ~60 binary orders above the
// first block's maximum, which ordinary attention scores never reach) marks
// the row: its m is raised to that block's maximum, its O accumulator and
// row sums (all of earlier blocks, taken with the old m) are scaled by
// 2^(m_old - m_new), and the block's probabilities are recomputed before
// they reach the P*V product.  The loop itself never rescales.
constexpr float kSumLimit = 1152921504606846976.0f;  // 2^60

typedef __attribute__((address_space(3))) void* lds_ptr_t;
// Word 3 of a raw (untyped) buffer descriptor: 32-bit data format.
constexpr int kBufferWord3 = 0x00020000;
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

// s_waitcnt immediates in the gfx9 encoding (vmcnt in bits 3:0 and 15:14,
// expcnt in 6:4, lgkmcnt in 11:8).  Written as builtins, not inline
// assembly, so the compiler's own wait insertion knows what has completed.
constexpr int kWaitLgkm0 = 0xC07F;
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
  __builtin_amdgcn_s_barrier();
}

template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x70 | 0xF00);
}

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

// TWO: some prefix tiles come from the second store (a separate
// instantiation, so single-store launches carry no per-tile store choice).
template <int D, bool TWO>
__global__ __launch_bounds__(kAttnThreads, 2) void chunk_attn_kernel(const AttnLaunch p) {
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int KS = D / 16;
  constexpr int MD = D / 32;
  constexpr int K_ROW_CHUNKS = D / 8;
  constexpr int V_ROW_CHUNKS = kTileKeys / 8;
  constexpr int K_ELEMS = kTileKeys * D;
  constexpr int BUF_ELEMS = 2 * K_ELEMS;
  // Tile t is copied by the four waves of group t & 1 (waves 0-3 or 4-7).
  constexpr int LOADS = K_ELEMS / 8 / (kAttnThreads / 2);
  constexpr int STAGES = 4;

  __shared__ __attribute__((aligned(1024))) uint16_t lds[STAGES * BUF_ELEMS];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar registers
  const int half = lane >> 5;
  const int l32 = lane & 31;

  const WorkItem item = decode_item(p, blockIdx.x);
  const int P = p.prefix_len;
  const int L = p.chunk_len;
  // Waves 0-3 form unit A, waves 4-7 unit B (one wave of each per SIMD).
  const int hu = p.heads_per_unit;
  const int unit_rows = (kAttnWaves / 2 / hu) * kAttnWaveRows;
  const int uw = wave & 3;
  const int head = item.head0 + (uw % hu);
  const bool unit_b = (wave >> 2) != 0;
  // First row of this wave slot in row group rg, and whether any of its rows lies before L.
  auto slot_row0 = [&](int rg) { return max(rg, 0) * unit_rows + (uw / hu) * kAttnWaveRows; };
  auto slot_on = [&](int rg) { return rg >= 0 && rg * unit_rows + (uw / hu) * kAttnWaveRows < L; };
  const int my_rg = unit_b ? item.row_group_b : item.row_group_a;
  const bool wave_on = slot_on(my_rg);  // a wave whose rows all lie past L has nothing to do
  int row0 = slot_row0(my_rg);
  const int wg_row0 = item.row_group_a * unit_rows;
  const int wg_row_end = min(L, (max(item.row_group_a, item.row_group_b) + 1) * unit_rows);

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
  const int n_head = (lo % kTileKeys) != 0 ? 1 : 0;
  const int fast_begin = tile_begin + n_head;
  const int fast_end = max(fast_begin, min(tile_end, min(hi, P + wg_row0 + 1) / kTileKeys));
  const int n_fast = fast_end - fast_begin;
  const int n_tiles = tile_end - tile_begin;
  auto seq_tile = [&](int i) __attribute__((always_inline)) -> int {
    if (i < n_fast) return fast_begin + i;
    if (i < n_fast + n_head) return tile_begin;
    return fast_end + (i - n_fast - n_head);
  };
  // A wave's share of the sequence: the first n positions (the tiles its
  // rows see; tiles past them come last in the order above), and, among
  // them, the tiles every one of its rows sees in full (unmasked).
  auto share_of = [&](int r0, bool on) {
    const int w_tile_end = (min(hi, P + r0 + kAttnWaveRows) + kTileKeys - 1) / kTileKeys;
    return on ? n_tiles - max(0, tile_end - w_tile_end) : 0;
  };
  const int n_w = share_of(row0, wave_on);
  int w_full_end = min(hi, P + row0 + 1);
  // Mirrored pairs leave the unit with the shorter row group idle on the
  // last positions, which only the other unit's rows see.  When there are
  // at least kHelpTiles of them, the wave of the shorter unit moves over to
  // its partner's rows for those positions (the same wave slot of the other
  // unit: same head, same SIMD): the partner computes the first 32-key half
  // of each such tile, the helper the second, and the two partial results
  // are merged through LDS at the end.  Both waves derive the same plan.
  constexpr int kHelpTiles = 4;
  const bool merge_wg = !p.pair_adjacent && item.row_group_b >= 0;
  const int a_n_w = share_of(slot_row0(item.row_group_a), slot_on(item.row_group_a));
  const int partner_row0 = slot_row0(item.row_group_b);
  const int partner_n_w = share_of(partner_row0, slot_on(item.row_group_b));
  const bool help = merge_wg && partner_n_w - a_n_w >= kHelpTiles;
  const int help_from = a_n_w;
  auto masked_at = [&](int i) __attribute__((always_inline)) -> bool {
    const int t = seq_tile(i);
    return t * kTileKeys < lo || (t + 1) * kTileKeys > w_full_end;
  };

  // Q fragments of the current 32 rows (B operand of S^T = K Q^T).
  bf16x8 qf[KS];
  auto load_q = [&]() __attribute__((always_inline)) {
    const int row = row0 + l32;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (row < L) {
        qf[ks] = *reinterpret_cast<const bf16x8*>(p.q + ((int64_t)row * p.h_q + head) * D + ks * 16 + half * 8);
      } else {
        qf[ks] = bf16x8{};
      }
    }
  };
  load_q();


  const int64_t head_stride = (int64_t)D * p.block_size;
  const int my_group = wave >> 2;
  const int gwave = wave & 3;  // wave within its group of four
  // Copy j of a tile moves 16-byte chunk (j * 4 + gwave) * 64 + lane.  The
  // swizzled column of a chunk does not depend on j (j adds whole rows: 16 K
  // rows or 32 V dim rows), so one per-lane offset serves every copy and j
  // moves the scalar offset.
  int k_src, v_src;
  {
    const int chunk = gwave * 64 + lane;
    const int kr = chunk / K_ROW_CHUNKS, kc = (chunk % K_ROW_CHUNKS) ^ k_swizzle<D>(kr);
    k_src = (kr * D + kc * 8) * 2;
    const int vr = chunk / V_ROW_CHUNKS, vc = (chunk % V_ROW_CHUNKS) ^ v_swizzle(vr);
    v_src = (vr * p.block_size + vc * 8) * 2;
  }
  constexpr int K_ROWS_PER_COPY = kAttnThreads / 2 / K_ROW_CHUNKS;
  constexpr int V_ROWS_PER_COPY = kAttnThreads / 2 / V_ROW_CHUNKS;
  static_assert(K_ROWS_PER_COPY % 16 == 0 && V_ROWS_PER_COPY % 16 == 0, "copy stride keeps the swizzle");
  auto issue_seq = [&](int i) __attribute__((always_inline)) {
    if ((i & 1) != my_group) return;
    const int t = seq_tile(i);
    // Tiles [remote_begin, remote_end) live in the second store.
    const bool remote = TWO && t >= p.remote_begin && t < p.remote_end;
    const const_i32_ptr table = (const_i32_ptr)(remote ? p.table_r : p.table);
    const int pos0 = t * kTileKeys;
    const int lb = (int)((__umulhi((uint32_t)pos0, p.block_magic) + (uint32_t)pos0) >> p.block_shift);
    const int slot0 = pos0 - lb * p.block_size;
    const int64_t base = ((int64_t)table[lb] * p.h_kv + item.kv_head) * head_stride;
    const uint16_t* kb = (remote ? p.k_pool_r : p.k_pool) + base + (int64_t)slot0 * D;
    const uint16_t* vb = (remote ? p.v_pool_r : p.v_pool) + base + slot0;
    uint16_t* kl = lds + (i % STAGES) * BUF_ELEMS;
    uint16_t* vl = kl + K_ELEMS;
    // Buffer loads rather than global_load_lds: while a global (FLAT-encoded)
    // LDS copy is in flight, the compiler's wait insertion cannot count LDS
    // reads one by one and waits for all of them before each MFMA.
    const __amdgpu_buffer_rsrc_t kr = __builtin_amdgcn_make_buffer_rsrc((void*)kb, 0, -1, kBufferWord3);
    const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc((void*)vb, 0, -1, kBufferWord3);
#pragma unroll
    for (int j = 0; j < LOADS; ++j) {
      const int dst = (j * 4 + gwave) * 64 * 8;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(kr, (lds_ptr_t)(kl + dst), 16, k_src, j * K_ROWS_PER_COPY * D * 2,
                                               0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(vr, (lds_ptr_t)(vl + dst), 16, v_src,
                                               j * V_ROWS_PER_COPY * p.block_size * 2, 0, 0);
    }
  };
  // The group that copied tile i waits for its copies (the only ones it has in
  // flight: it copies its next tile only after this barrier); the other group
  // has just the following tile in flight and does not wait.
  auto publish_seq = [&](int i) __attribute__((always_inline)) {
    if ((i & 1) == my_group) wait_vmem<0>();
    lds_barrier();
    const int tstart = seq_tile(i) * kTileKeys;
    if (tstart + kTileKeys > valid_end) {
      uint16_t* vl = lds + (i % STAGES) * BUF_ELEMS + K_ELEMS;
      const int first = valid_end - tstart;
      for (int idx = tid; idx < D * kTileKeys; idx += kAttnThreads) {
        const int e = idx / kTileKeys, key = idx % kTileKeys;
        if (key >= first) vl[e * kTileKeys + (((key >> 3) ^ v_swizzle(e)) << 3) + (key & 7)] = 0;
      }
      lds_barrier();
    }
  };

  f32x16 oacc[MD];
#pragma unroll
  for (int md = 0; md < MD; ++md) oacc[md] = f32x16{};
  // l_run: sum of the bf16 probabilities (normalises O); f_run: sum of the
  // fp32 exponentials (the log-sum-exp).
  float m_run = -INFINITY, l_run = 0.f, f_run = 0.f;
  const float sl2 = p.scale_log2;
  int k_row_lo = key_row_order(l32);
  int v_row_sw = v_swizzle(l32);
  const uint32_t ones = 0x3F803F80u;

  auto visible_bits = [&](int base) __attribute__((always_inline)) -> uint32_t {
    const int a = lo - base;
    const int b = min(hi, P + row0 + l32 + 1) - base;
    auto first_i = [](int x) { return x <= 0 ? 0 : x <= 8 ? x : x <= 16 ? 8 : x <= 24 ? x - 8 : 16; };
    const int i0 = first_i(a), i1 = first_i(b);
    return i1 > i0 ? (((1u << i1) - 1u) & ~((1u << i0) - 1u)) : 0u;
  };

  // Pieces of one 64-key tile.  NH = 2 (nh2): the whole tile -- scores (16
  // MFMAs), probabilities of both 32-key halves, settle, P*V (16 MFMAs).
  // NH = 1 (nh1): only the 32-key half h0 (8 + 8 MFMAs), when two waves
  // share each tile's keys (their partial results are merged at the end).
  f32x16 s[2];
  uint32_t pk[2][2][8];  // [buffer][32-key half][packed pairs]: tile i uses buffer i % 2
  float rs[2], fs[2];  // per 32-key half: bf16 sum, fp32 sum
  auto scores = [&](auto nh, int i, bool masked, int h0, f32x16* s) __attribute__((always_inline)) {
    constexpr int NH = decltype(nh)::value;
    const uint16_t* kl = lds + (i % STAGES) * BUF_ELEMS;
    const int kr0 = h0 * 32 + k_row_lo, kr1 = 32 + k_row_lo;
    const uint16_t* krow0 = kl + kr0 * D;
    const uint16_t* krow1 = kl + kr1 * D;
    const int ksw0 = k_swizzle<D>(kr0), ksw1 = k_swizzle<D>(kr1);
    // The 32-key halves are independent accumulation chains; their K
    // fragments are read two k-steps ahead of the MFMAs that use them.
    auto kfrag = [&](const uint16_t* krow, int ksw, int ks) __attribute__((always_inline)) {
      return *reinterpret_cast<const bf16x8*>(krow + (((ks * 2 + half) ^ ksw) << 3));
    };
    bf16x8 a0[KS], a1[KS];
    a0[0] = kfrag(krow0, ksw0, 0);
    if constexpr (NH == 2) a1[0] = kfrag(krow1, ksw1, 0);
    a0[1] = kfrag(krow0, ksw0, 1);
    if constexpr (NH == 2) a1[1] = kfrag(krow1, ksw1, 1);
    s[0] = s[1] = f32x16{};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (ks + 2 < KS) {
        a0[ks + 2] = kfrag(krow0, ksw0, ks + 2);
        if constexpr (NH == 2) a1[ks + 2] = kfrag(krow1, ksw1, ks + 2);
      }
      s[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0[ks], qf[ks], s[0], 0, 0, 0);
      if constexpr (NH == 2) s[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks], qf[ks], s[1], 0, 0, 0);
    }
    // Issue order: the first 2 * NH fragment reads, then each MFMA followed
    // by the next read, so reads stay two k-steps ahead of their MFMAs.
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * NH, 1);  // LDS reads
#pragma unroll
    for (int k = 0; k < NH * KS; ++k) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);  // MFMA
      if (k + 2 * NH < NH * KS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 1);
    }
    if (masked) {
      // Hidden scores become -inf, so their probabilities are exactly 0.
      const int tstart = seq_tile(i) * kTileKeys;
#pragma unroll
      for (int sb = 0; sb < NH; ++sb) {
        const uint32_t vm = visible_bits(tstart + (h0 + sb) * 32 + half * 8);
#pragma unroll
        for (int i2 = 0; i2 < 16; ++i2) {
          const int keep = __builtin_amdgcn_sbfe((int)vm, i2, 1);
          s[sb][i2] = __int_as_float((__float_as_int(s[sb][i2]) & keep) | (~keep & (int)0xFF800000u));
        }
      }
    }
  };
  // Probabilities of the NH halves of scores ss into buffer b and their row sums.
  auto probs = [&](auto nh, const f32x16* ss, int b, float neg_m) __attribute__((always_inline)) {
    constexpr int NH = decltype(nh)::value;
#pragma unroll
    for (int sb = 0; sb < NH; ++sb) {
      float fa = 0.f;
#pragma unroll
      for (int i2 = 0; i2 < 16; i2 += 2) {
        const float e0 = __builtin_amdgcn_exp2f(fmaf(ss[sb][i2], sl2, neg_m));
        const float e1 = __builtin_amdgcn_exp2f(fmaf(ss[sb][i2 + 1], sl2, neg_m));
        pk[b][sb][i2 / 2] = pack_bf16x2(e0, e1);
        fa += e0 + e1;
      }
      fs[sb] = fa;
    }
#pragma unroll
    for (int sb = 0; sb < NH; ++sb) {
      float acc = 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j) acc = dot2_bf16(pk[b][sb][j], ones, acc);
      rs[sb] = acc;
    }
    if constexpr (NH == 1) rs[1] = fs[1] = 0.f;
  };
  // A row still without a reference exponent (m = -inf, exponent offset
  // +inf) has an infinite or NaN sum here, which sends it to the fresh branch.
  auto settle = [&](auto nh, const f32x16* ss, int b) __attribute__((always_inline)) {
    constexpr int NH = decltype(nh)::value;
    const bool over = !(rs[0] <= kSumLimit) || !(rs[1] <= kSumLimit);
    if (__builtin_amdgcn_ballot_w64(over) != 0) {
      const bool row_over = lane_pair_max(over ? 1.f : 0.f) > 0.f;
      // Largest score of the block (hidden ones are -inf).
      float mx = -INFINITY;
#pragma unroll
      for (int sb = 0; sb < NH; ++sb)
#pragma unroll
        for (int i2 = 0; i2 < 16; ++i2) mx = fmaxf(mx, ss[sb][i2]);
      mx = lane_pair_max(mx) * sl2;
      if (row_over) {
        // A row with nothing accumulated yet (m = -inf) just takes its
        // reference; otherwise everything accumulated so far is rescaled.
        if (lane_pair_sum(l_run) != 0.f) {
          const float f = __builtin_amdgcn_exp2f(m_run - mx);
#pragma unroll
          for (int md = 0; md < MD; ++md) oacc[md] *= f;
          l_run *= f;
          f_run *= f;
        }
        m_run = mx;
        probs(nh, ss, b, m_run == -INFINITY ? 0.f : -m_run);
      }
    }
    l_run += rs[0] + rs[1];
    f_run += fs[0] + fs[1];
  };
  // Tile i's P*V alone (probabilities from buffer b), V fragments read
  // AHEAD MFMAs before their use.
  auto pv = [&](auto nh, int i, int b, int h0) __attribute__((always_inline)) {
    constexpr int NH = decltype(nh)::value;
    const uint16_t* vl = lds + (i % STAGES) * BUF_ELEMS + K_ELEMS;
    auto vfrag = [&](int kl, int md) __attribute__((always_inline)) {
      const int vchunk = ((2 * h0 + kl) * 2 + half) ^ v_row_sw;
      return *reinterpret_cast<const bf16x8*>(vl + (md * 32 + l32) * kTileKeys + (vchunk << 3));
    };
    constexpr int NF = 2 * NH * MD, AHEAD = 3;
    bf16x8 vf[AHEAD + 1];
#pragma unroll
    for (int k = 0; k < AHEAD; ++k) vf[k] = vfrag(k / MD, k % MD);
#pragma unroll
    for (int k = 0; k < NF; ++k) {
      const int kl = k / MD, md = k % MD, sb = kl / 2, kk = kl % 2;
      if (k + AHEAD < NF) vf[(k + AHEAD) % (AHEAD + 1)] = vfrag((k + AHEAD) / MD, (k + AHEAD) % MD);
      const bf16x8 pb = __builtin_bit_cast(
          bf16x8, u32x4{pk[b][sb][kk * 4], pk[b][sb][kk * 4 + 1], pk[b][sb][kk * 4 + 2], pk[b][sb][kk * 4 + 3]});
      oacc[md] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[k % (AHEAD + 1)], pb, oacc[md], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // Tile i's P*V (probabilities from buffer bo) with the next tile's
  // probabilities (into buffer bn) woven in: after each MFMA, the
  // exponentials, packing and row sums of 8 * NH / (2 * NH * MD) score
  // pairs.  V fragments are read two MFMAs ahead.  The scheduling barrier
  // after each step keeps this order, which the compiler's scheduler would
  // otherwise collapse into all MFMAs first.
  auto pv_probs = [&](auto nh, int i, int bo, int bn, float neg_m, int h0) __attribute__((always_inline)) {
    constexpr int NH = decltype(nh)::value;
    const uint16_t* vl = lds + (i % STAGES) * BUF_ELEMS + K_ELEMS;
    auto vfrag = [&](int kl, int md) __attribute__((always_inline)) {
      const int vchunk = ((2 * h0 + kl) * 2 + half) ^ v_row_sw;
      return *reinterpret_cast<const bf16x8*>(vl + (md * 32 + l32) * kTileKeys + (vchunk << 3));
    };
    constexpr int NF = 2 * NH * MD, AHEAD = 2, NPAIRS = 8 * NH, PAIRS = NPAIRS / NF;
    bf16x8 vf[AHEAD + 1];
#pragma unroll
    for (int k = 0; k < AHEAD; ++k) vf[k] = vfrag(k / MD, k % MD);
    // Within the weave, a pair's pack trails its exponentials by two pairs
    // and its row-sum step by four, so no VALU instruction waits on the one
    // just before it.
    constexpr int LAG_PACK = 2, LAG_SUM = 4;
    float acc[2] = {0.f, 0.f}, facc[2] = {0.f, 0.f};
    float ex[NPAIRS][2];
    auto do_exp = [&](int pr) __attribute__((always_inline)) {
      const int nsb = pr / 8, j = pr % 8;
      ex[pr][0] = __builtin_amdgcn_exp2f(fmaf(s[nsb][2 * j], sl2, neg_m));
      ex[pr][1] = __builtin_amdgcn_exp2f(fmaf(s[nsb][2 * j + 1], sl2, neg_m));
    };
    auto do_pack = [&](int pr) __attribute__((always_inline)) {
      pk[bn][pr / 8][pr % 8] = pack_bf16x2(ex[pr][0], ex[pr][1]);
    };
    auto do_sum = [&](int pr) __attribute__((always_inline)) {
      acc[pr / 8] = dot2_bf16(pk[bn][pr / 8][pr % 8], ones, acc[pr / 8]);
      facc[pr / 8] += ex[pr][0] + ex[pr][1];
    };
#pragma unroll
    for (int k = 0; k < NF; ++k) {
      const int kl = k / MD, md = k % MD, sb = kl / 2, kk = kl % 2;
      if (k + AHEAD < NF) vf[(k + AHEAD) % (AHEAD + 1)] = vfrag((k + AHEAD) / MD, (k + AHEAD) % MD);
      const bf16x8 pb = __builtin_bit_cast(
          bf16x8, u32x4{pk[bo][sb][kk * 4], pk[bo][sb][kk * 4 + 1], pk[bo][sb][kk * 4 + 2], pk[bo][sb][kk * 4 + 3]});
      oacc[md] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[k % (AHEAD + 1)], pb, oacc[md], 0, 0, 0);
#pragma unroll
      for (int q = 0; q < PAIRS; ++q) {
        const int pr = k * PAIRS + q;
        do_exp(pr);
        if (pr >= LAG_PACK) do_pack(pr - LAG_PACK);
        if (pr >= LAG_SUM) do_sum(pr - LAG_SUM);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int pr = NPAIRS; pr < NPAIRS + LAG_SUM; ++pr) {
      if (pr - LAG_PACK < NPAIRS) do_pack(pr - LAG_PACK);
      do_sum(pr - LAG_SUM);
    }
    rs[0] = acc[0];
    rs[1] = acc[1];
    fs[0] = facc[0];
    fs[1] = facc[1];
  };
  // Barrier k, met by every wave at the top of tile k, publishes tile k and
  // frees the stage of tile k-2 (every wave has finished its P*V), which tile
  // k+2 refills.
  auto barrier_k = [&](int k) __attribute__((always_inline)) {
    publish_seq(k);
    if (k + 2 < n_tiles) issue_seq(k + 2);
  };
  // Position i of the sequence (probabilities into buffer b): scores, then
  // the previous tile's P*V with this tile's probabilities woven in, so one
  // wave keeps both the matrix and the vector units busy.
  auto step = [&](auto nh, int i, int b, int h0) __attribute__((always_inline)) {
    barrier_k(i);
    scores(nh, i, masked_at(i), h0, s);
    pv_probs(nh, i - 1, b ^ 1, b, -m_run, h0);
    settle(nh, s, b);
  };
  // Positions [from, to) of the sequence, meeting their barriers: the first
  // tile's scores and probabilities, the woven steps, and the last P*V.
  auto run_range = [&](auto nh, int from, int to, int h0) __attribute__((always_inline)) {
    barrier_k(from);
    scores(nh, from, masked_at(from), h0, s);
    probs(nh, s, 0, -m_run);
    settle(nh, s, 0);
    for (int i = from + 1; i < to; i += 2) {
      step(nh, i, 1, h0);
      if (i + 1 < to) step(nh, i + 1, 0, h0);
    }
    if ((to - 1 - from) & 1) {  // the last tile's probabilities are in buffer 1
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int j = 0; j < 8; ++j) pk[0][sb][j] = pk[1][sb][j];
    }
    pv(nh, to - 1, 0, h0);
  };
  // The order of the other unit (waves 4-7; wave w and w + 4 share a SIMD):
  // tile i's scores with tile i-1's exponentials, packing and row sums woven
  // in after each MFMA, then tile i-1's P*V alone.  One wave of each SIMD is
  // then in an MFMA-only phase while the other interleaves the softmax.
  f32x16 sc[2][2];  // [tile parity][32-key half]
  auto mask_scores = [&](auto nh, int i, f32x16* ss) __attribute__((always_inline)) {
    constexpr int NH = decltype(nh)::value;
    const int tstart = seq_tile(i) * kTileKeys;
#pragma unroll
    for (int sb = 0; sb < NH; ++sb) {
      const uint32_t vm = visible_bits(tstart + sb * 32 + half * 8);
#pragma unroll
      for (int i2 = 0; i2 < 16; ++i2) {
        const int keep = __builtin_amdgcn_sbfe((int)vm, i2, 1);
        ss[sb][i2] = __int_as_float((__float_as_int(ss[sb][i2]) & keep) | (~keep & (int)0xFF800000u));
      }
    }
  };
  // Tile i's scores into sn with the probabilities of tile i-1 (scores sp,
  // masked here first when tile i-1 straddles an edge) woven in.
  auto scores_probs = [&](auto nh, int i, f32x16* sn, f32x16* sp, float neg_m) __attribute__((always_inline)) {
    constexpr int NH = decltype(nh)::value;
    if (masked_at(i - 1)) mask_scores(nh, i - 1, sp);
    const uint16_t* kl = lds + (i % STAGES) * BUF_ELEMS;
    const int kr0 = k_row_lo, kr1 = 32 + k_row_lo;
    const uint16_t* krow0 = kl + kr0 * D;
    const uint16_t* krow1 = kl + kr1 * D;
    const int ksw0 = k_swizzle<D>(kr0), ksw1 = k_swizzle<D>(kr1);
    // MFMA k uses half k % NH at k-step k / NH; its K fragment is read AHEAD
    // MFMAs earlier.
    constexpr int NF = NH * KS, AHEAD = 2, NPAIRS = 8 * NH, PAIRS = NPAIRS / NF;
    static_assert(PAIRS * NF == NPAIRS, "whole score pairs per MFMA");
    auto kfrag = [&](int k) __attribute__((always_inline)) {
      const int sb = k % NH, ks = k / NH;
      const uint16_t* krow = sb == 0 ? krow0 : krow1;
      const int ksw = sb == 0 ? ksw0 : ksw1;
      return *reinterpret_cast<const bf16x8*>(krow + (((ks * 2 + half) ^ ksw) << 3));
    };
    bf16x8 kf[AHEAD + 1];
#pragma unroll
    for (int k = 0; k < AHEAD; ++k) kf[k] = kfrag(k);
    constexpr int LAG_PACK = 2, LAG_SUM = 4;
    float acc[2] = {0.f, 0.f}, facc[2] = {0.f, 0.f};
    float ex[NPAIRS][2];
    auto do_exp = [&](int pr) __attribute__((always_inline)) {
      const int psb = pr / 8, j = pr % 8;
      ex[pr][0] = __builtin_amdgcn_exp2f(fmaf(sp[psb][2 * j], sl2, neg_m));
      ex[pr][1] = __builtin_amdgcn_exp2f(fmaf(sp[psb][2 * j + 1], sl2, neg_m));
    };
    auto do_pack = [&](int pr) __attribute__((always_inline)) {
      pk[0][pr / 8][pr % 8] = pack_bf16x2(ex[pr][0], ex[pr][1]);
    };
    auto do_sum = [&](int pr) __attribute__((always_inline)) {
      acc[pr / 8] = dot2_bf16(pk[0][pr / 8][pr % 8], ones, acc[pr / 8]);
      facc[pr / 8] += ex[pr][0] + ex[pr][1];
    };
    sn[0] = sn[1] = f32x16{};
#pragma unroll
    for (int k = 0; k < NF; ++k) {
      const int sb = k % NH, ks = k / NH;
      if (k + AHEAD < NF) kf[(k + AHEAD) % (AHEAD + 1)] = kfrag(k + AHEAD);
      sn[sb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[k % (AHEAD + 1)], qf[ks], sn[sb], 0, 0, 0);
#pragma unroll
      for (int q = 0; q < PAIRS; ++q) {
        const int pr = k * PAIRS + q;
        do_exp(pr);
        if (pr >= LAG_PACK) do_pack(pr - LAG_PACK);
        if (pr >= LAG_SUM) do_sum(pr - LAG_SUM);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int pr = NPAIRS; pr < NPAIRS + LAG_SUM; ++pr) {
      if (pr - LAG_PACK < NPAIRS) do_pack(pr - LAG_PACK);
      do_sum(pr - LAG_SUM);
    }
    rs[0] = acc[0];
    rs[1] = acc[1];
    fs[0] = facc[0];
    fs[1] = facc[1];
  };
  // Position i in the other unit's order: tile i's scores (into sn) with the
  // probabilities of tile i-1 (scores sp) woven in, then tile i-1's P*V.  The
  // woven phase runs at raised wave priority, so its MFMAs issue as soon as
  // their operands are ready and the partner wave's MFMA-only phase fills the
  // gaps; at equal priority the older partner's back-to-back MFMAs held the
  // matrix unit and stalled this wave's in-order stream.
  auto step_b = [&](int i, f32x16* sn, f32x16* sp) __attribute__((always_inline)) {
    const std::integral_constant<int, 2> nh;
    barrier_k(i);
    __builtin_amdgcn_s_setprio(1);
    scores_probs(nh, i, sn, sp, -m_run);
    __builtin_amdgcn_s_setprio(0);
    settle(nh, sp, 0);
    pv(nh, i - 1, 0, 0);
  };
  // Positions [from, to) in the other unit's order (whole tiles).
  auto run_range_b = [&](int from, int to) __attribute__((always_inline)) {
    const std::integral_constant<int, 2> nh;
    barrier_k(from);
    scores(nh, from, false, 0, sc[0]);
    for (int i = from + 1; i < to; i += 2) {
      step_b(i, sc[1], sc[0]);
      if (i + 1 < to) step_b(i + 1, sc[0], sc[1]);
    }
    // The last tile's scores are in sc[1] after an odd number of steps.
    if ((to - 1 - from) & 1) {
#pragma unroll
      for (int sb = 0; sb < 2; ++sb) sc[0][sb] = sc[1][sb];
    }
    if (masked_at(to - 1)) mask_scores(nh, to - 1, sc[0]);
    probs(nh, sc[0], 0, -m_run);
    settle(nh, sc[0], 0);
    pv(nh, to - 1, 0, 0);
  };
  // O and LSE of the current rows (or their split partials).
  const bool split = p.n_ranges > 1;
  auto store_outputs = [&]() __attribute__((always_inline)) {
    const float l_tot = lane_pair_sum(l_run);
    const float f_tot = lane_pair_sum(f_run);
    const int row = row0 + l32;
    if (row < L) {
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
      const float row_lse = f_tot > 0.f ? (m_run + log2f(f_tot)) * kLn2 : -INFINITY;
      if (!split) {
        uint16_t* orow = p.o + ((int64_t)row * p.h_q + head) * D;
#pragma unroll
        for (int md = 0; md < MD; ++md) {
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            bf16x4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = (__bf16)(oacc[md][j * 4 + e] * inv);
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
            for (int e = 0; e < 4; ++e) v[e] = oacc[md][j * 4 + e] * inv;
            *reinterpret_cast<f32x4*>(orow + md * 32 + j * 8 + half * 4) = v;
          }
        }
        if (half == 0) p.ws_lse[base] = row_lse;
      }
    }
  };

  const std::integral_constant<int, 2> nh2;
  const std::integral_constant<int, 1> nh1;
  if (n_tiles > 0) {
    // Without this, values the first tile derives from these (its masks, its
    // LDS addresses) are computed once ahead of the loop and then occupy
    // registers through every later tile.
    asm volatile("" : "+s"(lo), "+s"(hi), "+v"(k_row_lo), "+v"(v_row_sw));
    issue_seq(0);
    if (n_tiles > 1) issue_seq(1);
    // Whole tiles: this wave's own positions, or, when the unit pair
    // shares the last positions, the positions before them.  Then the
    // shared positions: the helped wave keeps its rows and takes the first
    // 32-key half of each tile; the helping wave stores its own rows and
    // takes the second half for its partner's rows.  One copy of each loop
    // serves every wave.
    const int full_end = help ? help_from : n_w;
    int done = 0;  // positions whose barrier this wave has met
    if (full_end > 0) {
      if (unit_b) {
        run_range_b(0, full_end);
      } else {
        run_range(nh2, 0, full_end, 0);
      }
      done = full_end;
    }
    if (help) {
      if (!unit_b) {
        if (full_end > 0) store_outputs();
        row0 = partner_row0;
        w_full_end = min(hi, P + row0 + 1);
        load_q();
        m_run = -INFINITY;
        l_run = f_run = 0.f;
#pragma unroll
        for (int md = 0; md < MD; ++md) oacc[md] = f32x16{};
      }
      run_range(nh1, help_from, partner_n_w, unit_b ? 0 : 1);
      done = partner_n_w;
    }
    if (done == 0) {
      barrier_k(0);
      done = 1;
    }
    for (int i = done; i < n_tiles; ++i) barrier_k(i);
  }

  if (merge_wg) {
    // The helping wave hands its partial (O, m and both sums of the
    // partner's rows over the second key halves) to the partner through LDS,
    // which no tile occupies any more.
    constexpr int NV = MD * 16;
    float* mb = reinterpret_cast<float*>(lds) + uw * (NV + 3) * 64;
    lds_barrier();
    if (help && !unit_b) {
#pragma unroll
      for (int md = 0; md < MD; ++md)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          *reinterpret_cast<f32x4*>(mb + ((md * 4 + j) * 64 + lane) * 4) =
              f32x4{oacc[md][j * 4], oacc[md][j * 4 + 1], oacc[md][j * 4 + 2], oacc[md][j * 4 + 3]};
      mb[NV * 64 + lane] = m_run;
      mb[NV * 64 + 64 + lane] = l_run;
      mb[NV * 64 + 128 + lane] = f_run;
    }
    lds_barrier();
    if (help && unit_b) {
      const float m_a = mb[NV * 64 + lane];
      const float m = fmaxf(m_run, m_a);
      const float cb = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - m);
      const float ca = m_a == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_a - m);
#pragma unroll
      for (int md = 0; md < MD; ++md)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const f32x4 o_a = *reinterpret_cast<const f32x4*>(mb + ((md * 4 + j) * 64 + lane) * 4);
#pragma unroll
          for (int e = 0; e < 4; ++e) oacc[md][j * 4 + e] = oacc[md][j * 4 + e] * cb + o_a[e] * ca;
        }
      l_run = l_run * cb + mb[NV * 64 + 64 + lane] * ca;
      f_run = f_run * cb + mb[NV * 64 + 128 + lane] * ca;
      m_run = m;
    }
  }
  // Waves with rows left to write: their own (no help), or the partner's
  // merged rows (the wave that was helped); a helping wave stored its own.
  if (help ? unit_b : wave_on) store_outputs();
#endif  // __HIP_DEVICE_COMPILE__
}

}  // namespace

hipError_t launch_chunk_attn(const AttnLaunch& p, int head_dim, hipStream_t stream) {
  const dim3 grid(p.total_wgs), block(kAttnThreads);
  const bool two = p.remote_end > p.remote_begin;
  if (head_dim == 128) {
    if (two) {
      hipLaunchKernelGGL((chunk_attn_kernel<128, true>), grid, block, 0, stream, p);
    } else {
      hipLaunchKernelGGL((chunk_attn_kernel<128, false>), grid, block, 0, stream, p);
    }
  } else {
    if (two) {
      hipLaunchKernelGGL((chunk_attn_kernel<64, true>), grid, block, 0, stream, p);
    } else {
      hipLaunchKernelGGL((chunk_attn_kernel<64, false>), grid, block, 0, stream, p);
    }
  }
  return hipGetLastError();
}

}  // namespace mocap
