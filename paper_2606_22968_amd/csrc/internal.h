// Internal launch descriptions shared by the host API and the HIP kernels of
// libmocap_attn.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mocap {

constexpr int kTileKeys = 64;          // keys per KV tile (LDS stage)
constexpr int kAttnWaves = 8;          // wavefronts per attention workgroup
constexpr int kAttnWaveRows = 32;      // query rows owned by one attention wavefront
constexpr int kAttnThreads = 64 * kAttnWaves;
constexpr int kWavesPerGroup = 4;      // wavefronts per workgroup of the other kernels
constexpr int kGroupThreads = 64 * kWavesPerGroup;

// One launch of the attention kernel: every workgroup holds two units of four
// wavefronts; a unit owns `heads_per_unit` query heads of one GQA group times
// `32 * 4 / heads_per_unit` query rows (a row group).  The units of a
// workgroup take two row groups of the same heads, for one KV range: pair q
// is row groups q and row_groups - 1 - q (mirrored; the middle group of an
// odd count is alone), or row_groups - 2 - 2q and row_groups - 1 - 2q
// (adjacent, longest pair first; group 0 alone when the count is odd).
//
// KV ranges: n_ranges == 1 is the unsplit launch over [0, P + L); otherwise
// n_ranges - 1 ranges cut the prefix tiles [0, ceil(P / 64)) evenly (the
// last one ends at P), then the chunk's own keys [P, P + L).  Tile t holds
// keys [64 t, 64 t + 64); tiles [remote_begin, remote_end) are read from the
// second store, every other tile from the first.
struct AttnLaunch {
  const uint16_t* q;        // bf16 [L][Hq][D]
  const uint16_t* k_pool;   // bf16 [nb][Hkv][bs][D]
  const uint16_t* v_pool;   // bf16 [nb][Hkv][D][bs]
  const int32_t* table;     // logical block -> physical block
  const uint16_t* k_pool_r; // second store (same layout and block size), or null
  const uint16_t* v_pool_r;
  const int32_t* table_r;
  uint16_t* o;              // bf16 [L][Hq][D]         (unsplit)
  float* lse;               // fp32 [Hq][L]            (unsplit)
  float* ws_o;              // fp32 [R][Hq][L][D]      (split partials)
  float* ws_lse;            // fp32 [R][Hq][L]
  int32_t prefix_len;       // P (P + L < 2^31 - 128, checked on the host)
  int32_t prefix_tiles;     // ceil(P / 64)
  int32_t chunk_len;        // L
  int32_t h_q;
  int32_t h_kv;
  int32_t group;            // Hq / Hkv
  int32_t heads_per_unit;   // 2 or 1 (divides group)
  int32_t row_groups;       // ceil(L / rows_per_unit)
  int32_t pairs;            // ceil(row_groups / 2)
  int32_t pair_adjacent;    // 0 = mirrored pairs, 1 = adjacent pairs
  int32_t block_size;
  uint32_t block_magic;     // floor(n / block_size) = (umulhi(n, magic) + n) >> shift
  int32_t block_shift;      //   for 0 <= n < 2^31 (division by an invariant integer)
  int32_t n_ranges;         // 1 = unsplit; else prefix ranges + 1 chunk range
  int32_t remote_begin;     // tiles [remote_begin, remote_end) live in the second store
  int32_t remote_end;
  int32_t total_wgs;
  float scale_log2;         // scale * log2(e)
};

struct AppendLaunch {
  const uint16_t* k_chunk;  // bf16 [L][Hkv][D]
  const uint16_t* v_chunk;  // bf16 [L][Hkv][D]
  uint16_t* k_pool;
  uint16_t* v_pool;
  const int32_t* table;
  int64_t start_pos;
  int32_t chunk_len;
  int32_t h_kv;
  int32_t block_size;
};

struct MergeLaunch {
  const float* ws_o;        // fp32 [R][Hq][L][D]
  const float* ws_lse;      // fp32 [R][Hq][L]
  uint16_t* o;              // bf16 [L][Hq][D]
  float* lse;               // fp32 [Hq][L]
  int32_t chunk_len;
  int32_t h_q;
  int32_t n_ranges;
};

hipError_t launch_chunk_attn(const AttnLaunch& p, int head_dim, hipStream_t stream);
hipError_t launch_kv_append(const AppendLaunch& p, int head_dim, hipStream_t stream);
hipError_t launch_lse_merge(const MergeLaunch& p, int head_dim, hipStream_t stream);

}  // namespace mocap
