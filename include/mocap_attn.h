/*
 * mocap_attn.h -- C ABI of libmocap_attn: chunked causal prefill attention on
 * AMD Instinct MI355X (gfx950).
 *
 * The operation (MOCAP, Section 2.2 "Chunked Pipeline", and Eq. (1) of
 * Section 3.2): a long prompt of S tokens is cut into chunks; chunk c has
 * L_c query tokens and sits behind a prefix of P_c = L_1 + ... + L_{c-1}
 * tokens.  Its queries attend to the keys/values of every earlier chunk (the
 * prefix, no mask) and to its own keys under a causal mask, so chunk c costs
 * about L_c (P_c + L_c) -- the growth with P_c that the paper's
 * latency-balanced chunk partitioning (Section 4.2) compensates.  The
 * keys/values of earlier chunks stay resident between chunks; the paper's
 * memory-balanced KV reallocation (Section 4.1) moves part of them elsewhere,
 * which is why this library addresses them through a block table rather than
 * assuming one contiguous buffer.
 *
 * For query row i of chunk c (absolute position t = P_c + i), head h:
 *   kvh   = h / (h_q / h_kv)                      contiguous GQA groups
 *   s_j   = scale * <q_{i,h}, k_{j,kvh}>          for keys j = 0 .. t
 *   lse   = ln( sum_j exp(s_j) )
 *   o_i,h = sum_j exp(s_j - lse) * v_{j,kvh}
 * Inputs are bf16; products accumulate in fp32; softmax runs in fp32; the
 * probabilities are rounded to bf16 before the P*V product; O is rounded to
 * bf16 (round to nearest even); LSE is fp32.
 *
 * Conventions shared by every call
 *   - Tensor pointers are DEVICE pointers owned by the caller.  The library
 *     allocates no device memory and keeps no state across calls except small
 *     host caches (per-device compute-unit count, recent automatic split and
 *     pairing choices, per-device scratch addresses) and the static device scratch
 *     of mocap_chunk_attn_noalloc (MOCAP_NOALLOC_SCRATCH_BYTES per device,
 *     part of the loaded library image, never allocated by a call).
 *   - Calls enqueue work on `stream` (a hipStream_t passed as void*; NULL is
 *     the default stream) and return without synchronising.  A device-side
 *     fault shows up at the caller's next synchronisation.
 *   - Arguments are validated on the host before anything is enqueued; on any
 *     error status nothing is launched and nothing is written.
 *   - Position p of the sequence lives in logical block p / block_size at
 *     slot p % block_size; block_table[logical] gives the physical block.
 *     Table entries are trusted: each must lie in [0, num_blocks), and
 *     distinct positions must not share a slot.  mocap_check_block_table
 *     checks a host copy of a table; a library built with
 *     -DMOCAP_DEBUG_TABLES (build.py --debug-tables, libmocap_attn_debug.so)
 *     copies the entries each call will use to the host (a synchronous
 *     copy, so such a build cannot be used under graph capture) and returns
 *     MOCAP_ERR_INVALID_ARG, launching nothing, when one is out of range or
 *     two logical blocks share a physical block.
 *   - All device pointers must be 16-byte aligned.
 *   - The attention calls choose, per launch and from a time model, how the
 *     two halves of a workgroup pair up query rows; the environment variable
 *     MOCAP_PAIRING=mirrored or =adjacent forces one choice (for testing).
 *     Results agree with the oracle either way; they need not be bitwise
 *     equal between the two.
 */
#ifndef MOCAP_ATTN_H
#define MOCAP_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MOCAP_OK = 0,
  MOCAP_ERR_INVALID_ARG = 1, /* a malformed argument: nothing enqueued          */
  MOCAP_ERR_UNSUPPORTED = 2, /* well formed, but outside what the kernels do   */
  MOCAP_ERR_WORKSPACE = 3,   /* workspace missing or smaller than required     */
  MOCAP_ERR_HIP = 4          /* the HIP runtime reported an error              */
} mocap_status;

/*
 * A block-addressed KV store (host struct describing caller-owned device
 * memory).  Each physical block holds block_size consecutive positions of
 * all h_kv heads.
 *   k_pool : bf16 [num_blocks][h_kv][block_size][head_dim]   row per position
 *   v_pool : bf16 [num_blocks][h_kv][head_dim][block_size]   transposed inside
 *            each block, so one head-dim coordinate of consecutive positions
 *            is contiguous (the layout the P*V product consumes).
 * block_size must be a positive multiple of 64; head_dim is 64 or 128.
 */
typedef struct {
  void* k_pool;
  void* v_pool;
  int32_t num_blocks;
  int32_t block_size;
  int32_t h_kv;
  int32_t head_dim;
} mocap_kv_store;

/*
 * mocap_kv_append -- store one chunk's newly produced keys/values
 * (Section 2.2: the KV of earlier chunks stays live for later chunks;
 * Section 4.1: each stage first produces the chunk's new KV cache).
 *
 *   kv          store to write into (see mocap_kv_store)
 *   block_table device int32 [n_table], logical block -> physical block
 *   start_pos   P_c, absolute position of the chunk's first token (>= 0)
 *   chunk_len   L_c (>= 0); 0 is a no-op
 *   k_chunk     device bf16 [chunk_len][h_kv][head_dim]
 *   v_chunk     device bf16 [chunk_len][h_kv][head_dim]
 *   stream      hipStream_t or NULL
 *
 * Positions start_pos .. start_pos + chunk_len - 1 are written bit for bit;
 * nothing else in the pools changes.  Requires
 * ceil((start_pos + chunk_len) / block_size) <= n_table.
 * Errors: INVALID_ARG for null/misaligned pointers, negative sizes or a table
 * that is too short; UNSUPPORTED for head_dim or block_size outside the above;
 * HIP if the launch fails.
 */
mocap_status mocap_kv_append(const mocap_kv_store* kv, const int32_t* block_table, int32_t n_table,
                             int64_t start_pos, int32_t chunk_len, const void* k_chunk,
                             const void* v_chunk, void* stream);

/*
 * mocap_chunk_attn_workspace_size -- plan the KV split of one chunk and size
 * its workspace.
 *
 * The keys a chunk sees may be cut into ranges that are processed in
 * parallel and then combined by their log-sum-exp (the same combination a
 * debtor stage needs when it reads part of its KV remotely and part locally,
 * Section 4.1).  num_splits is the number of ranges: 1 = unsplit (no
 * workspace), n >= 2 = the prefix [0, P_c) cut into n - 1 ranges on 64-key
 * tile boundaries plus the chunk's own keys as the last range, 0 = let the
 * library choose from the shape and the current device's compute-unit count.
 * A requested count is clamped to what the prefix allows (1 when P_c = 0).
 *
 *   splits_out  (may be NULL) the number of ranges that will be used
 *   bytes_out   workspace bytes mocap_chunk_attn needs for this plan (0 when
 *               the plan is unsplit)
 * Errors: INVALID_ARG for a null bytes_out or malformed sizes; UNSUPPORTED
 * for head_dim not in {64, 128}; HIP if the device query fails (auto only).
 */
mocap_status mocap_chunk_attn_workspace_size(int64_t prefix_len, int32_t chunk_len, int32_t h_q,
                                             int32_t h_kv, int32_t head_dim, int32_t num_splits,
                                             int32_t* splits_out, size_t* bytes_out);

/*
 * mocap_chunk_attn -- causal attention of one chunk over its prefix and itself
 * (Section 2.2; cost c_i (p_i + c_i) by Eq. (1)).
 *
 *   kv, block_table, n_table  KV store holding positions [0, prefix_len +
 *               chunk_len): the chunk's own KV must already be appended, on
 *               this stream or otherwise ordered before this call
 *   q           device bf16 [chunk_len][h_q][head_dim]
 *   prefix_len  P_c (>= 0);  chunk_len  L_c (>= 0, 0 is a no-op)
 *   h_q, h_kv   query / KV head counts, h_q a multiple of h_kv, h_kv equal to
 *               kv->h_kv; head_dim equal to kv->head_dim
 *   scale       score scale, finite and > 0 (typically 1/sqrt(head_dim))
 *   o           device bf16 [chunk_len][h_q][head_dim]           (output)
 *   lse         device fp32 [h_q][chunk_len], natural log          (output)
 *   workspace   device scratch of workspace_bytes, or NULL when the plan is
 *               unsplit; its contents on entry do not matter
 *   num_splits  as in mocap_chunk_attn_workspace_size
 *   stream      hipStream_t or NULL
 *
 * The same (shape, num_splits, device) always gives the same plan and the
 * same bits, whatever physical blocks the table names.
 * Errors: INVALID_ARG for null/misaligned pointers, negative sizes, h_q not a
 * multiple of h_kv, head counts or head_dim that differ from the store, a
 * non-positive or non-finite scale, or a table shorter than
 * ceil((prefix_len + chunk_len) / block_size); UNSUPPORTED for head_dim not in
 * {64, 128} or block_size not a positive multiple of 64; WORKSPACE when the
 * plan needs more than workspace_bytes; HIP if a launch fails.
 */
mocap_status mocap_chunk_attn(const mocap_kv_store* kv, const int32_t* block_table, int32_t n_table,
                              const void* q, int64_t prefix_len, int32_t chunk_len, int32_t h_q,
                              int32_t h_kv, int32_t head_dim, float scale, void* o, float* lse,
                              void* workspace, size_t workspace_bytes, int32_t num_splits,
                              void* stream);

/*
 * mocap_chunk_attn_two_store -- mocap_chunk_attn for a chunk whose prefix KV
 * lives partly in a second store: the memory-balanced KV reallocation of
 * Section 4.1, where a debtor stage's KV accesses split into a remote portion
 * (held by its paired creditor stage) and a local portion.  The attention
 * kernel picks the store for every 64-key tile it loads, so the result does
 * not depend on where the range edges fall.
 *
 *   kv, block_table, n_table   the first ("local") store: it holds positions
 *               [0, remote_begin) and [remote_end, prefix_len + chunk_len),
 *               including the chunk's own KV; n_table >=
 *               ceil((prefix_len + chunk_len) / block_size)
 *   remote_kv, remote_table, n_remote_table   the second ("remote") store: it
 *               holds positions [remote_begin, remote_end); the same h_kv,
 *               head_dim and block_size as kv; its table is indexed by the
 *               same logical block numbers (position p in logical block
 *               p / block_size), so n_remote_table >= ceil(remote_end /
 *               block_size); only entries of blocks that overlap the range
 *               are read.  Its pools may be any memory the device can read
 *               (a peer device's HBM included).
 *   remote_begin, remote_end   multiples of 64 with 0 <= remote_begin <=
 *               remote_end <= prefix_len.  An empty range makes the call
 *               identical to mocap_chunk_attn (remote arguments unused, may
 *               be NULL).
 *   num_splits, workspace, other arguments   as in mocap_chunk_attn (the
 *               split plan is the same as for a single store).
 *
 * Each store is read only at the positions it holds, so the other store's
 * slots at those positions may hold anything (NaN included).  Results are
 * bitwise equal to mocap_chunk_attn's on a single store holding the same
 * keys and values, with the same num_splits.
 * Errors: as mocap_chunk_attn, plus INVALID_ARG for a malformed remote range,
 * a remote store that differs in h_kv, head_dim or block_size, or a remote
 * table that is too short or null.
 */
mocap_status mocap_chunk_attn_two_store(const mocap_kv_store* kv, const int32_t* block_table, int32_t n_table,
                                        const mocap_kv_store* remote_kv, const int32_t* remote_table,
                                        int32_t n_remote_table, int64_t remote_begin, int64_t remote_end,
                                        const void* q, int64_t prefix_len, int32_t chunk_len, int32_t h_q,
                                        int32_t h_kv, int32_t head_dim, float scale, void* o, float* lse,
                                        void* workspace, size_t workspace_bytes, int32_t num_splits,
                                        void* stream);

/*
 * mocap_chunk_attn_two_store_workspace_size -- the range count and workspace
 * bytes of mocap_chunk_attn_two_store: the same as
 * mocap_chunk_attn_workspace_size for the shape, after the remote range is
 * checked.  splits_out may be NULL.
 * Errors: INVALID_ARG for a null bytes_out, malformed sizes or remote range;
 * UNSUPPORTED for head_dim not in {64, 128}; HIP if the device query fails
 * (num_splits = 0 only).
 */
mocap_status mocap_chunk_attn_two_store_workspace_size(int64_t prefix_len, int32_t chunk_len, int32_t h_q,
                                                       int32_t h_kv, int32_t head_dim, int64_t remote_begin,
                                                       int64_t remote_end, int32_t num_splits,
                                                       int32_t* splits_out, size_t* bytes_out);

/*
 * mocap_chunk_plan -- chunk lengths for a prompt of seq_len tokens (host only,
 * no device work).
 *
 *   balanced = 0: uniform; boundary c at floor(c * seq_len / num_chunks).
 *   balanced = 1: every chunk gets the same causal attention work
 *     L_c (P_c + L_c / 2), the balancing goal behind Section 4.2's
 *     latency-balanced partitioning applied to the attention term of Eq. (1).
 *     Cumulative work up to boundary x is x^2 / 2, so boundary c sits at
 *     seq_len * sqrt(c / num_chunks), rounded to the nearest multiple of
 *     align (exact integer arithmetic).  seq_len must be a multiple of align.
 *   lengths_out host int32 [num_chunks]
 * Errors: INVALID_ARG for non-positive sizes, a null output, seq_len not a
 * multiple of align (balanced), an exact rounding tie, an empty chunk, or a
 * length that does not fit in int32.
 */
mocap_status mocap_chunk_plan(int64_t seq_len, int32_t num_chunks, int32_t align, int32_t balanced,
                              int32_t* lengths_out);

/*
 * mocap_chunk_prefixes -- prefix offsets of a chunk sequence (host only):
 * prefixes_out[c] = lengths[0] + ... + lengths[c - 1], the number of earlier
 * tokens every query of chunk c attends to (P_c above; Section 2.2, the p_i
 * of Eq. (1)).
 *
 *   lengths       host int32 [num_chunks], each >= 0
 *   prefixes_out  host int64 [num_chunks]; prefixes_out[0] = 0
 * Errors: INVALID_ARG for num_chunks < 0, a negative length, or a null array
 * with num_chunks > 0.
 */
mocap_status mocap_chunk_prefixes(const int32_t* lengths, int32_t num_chunks, int64_t* prefixes_out);

/*
 * mocap_lbcp_plan -- first stage of latency-balanced chunk partitioning
 * (Section 4.2, Alg. 1, the dynamic-programming initialisation), host only.
 *
 * Chooses num_chunks chunk lengths, each a positive multiple of align, that
 * sum to seq_len, by the dynamic program of Alg. 1: scanning chunk index m
 * from num_chunks down to 1, start s from the end down to 0 and length k
 * upwards, the cost t of a chunk of k starting at s is combined with the best
 * suffix state (m+1, s+k) into t'_max = max(t_max, t) and t'_sum = t_sum + t,
 * and the candidate minimising t'_sum + (num_stages - 1) * t'_max is kept.
 * The suffix boundary, which the paper leaves implicit, is t = 0 at
 * (num_chunks + 1, seq_len) and infeasible elsewhere.
 *
 * EvaluateChunk is the deterministic compute-latency model
 *   t(c, p) = cost_pair * (c p + c (c + 1) / 2) + cost_token * c + cost_chunk
 * for a chunk of c tokens behind p tokens: c p + c (c + 1) / 2 is the exact
 * number of causally visible (query, key) pairs, the attention term of
 * Eq. (1); cost_token covers work proportional to c (the GEMM term of
 * Eq. (1), appends); cost_chunk is a fixed cost per chunk.  The
 * coefficients are typically fitted to measured mocap_chunk_attn latency.
 *
 *   seq_len      S, a positive multiple of align
 *   num_chunks   M >= 1, with M * align <= S
 *   num_stages   N >= 1, pipeline stages of Alg. 1's objective
 *   lengths_out  host int32 [num_chunks]
 *   t_max_out, t_sum_out   (may be NULL) the plan's largest chunk cost and
 *                sum of chunk costs under the model
 * Work is O(M (S/align)^2); the call allocates host memory for its tables.
 * Errors: INVALID_ARG for non-positive sizes, a null lengths_out, S not a
 * multiple of align, M * align > S or negative/non-finite coefficients;
 * UNSUPPORTED when M (S/align)^2 exceeds 2^31 (the table would be too slow).
 */
mocap_status mocap_lbcp_plan(int64_t seq_len, int32_t num_chunks, int32_t num_stages, int32_t align,
                             double cost_pair, double cost_token, double cost_chunk,
                             int32_t* lengths_out, double* t_max_out, double* t_sum_out);

/*
 * mocap_lbcp_plan_table -- mocap_lbcp_plan with EvaluateChunk read from a
 * table instead of the three-coefficient model (host only).
 *
 *   chunk_cost  host double [U][U] with U = seq_len / align:
 *               chunk_cost[(k - 1) * U + s] is the latency of a chunk of
 *               k * align tokens starting at token s * align, for k >= 1 and
 *               s + k <= U (other entries are not read).  Typically measured
 *               latencies interpolated over a grid.
 * Other arguments and outputs as in mocap_lbcp_plan.
 * Errors: as mocap_lbcp_plan, plus INVALID_ARG for a null table or a read
 * entry that is negative or not finite.
 */
mocap_status mocap_lbcp_plan_table(int64_t seq_len, int32_t num_chunks, int32_t num_stages, int32_t align,
                                   const double* chunk_cost, int32_t* lengths_out, double* t_max_out,
                                   double* t_sum_out);

/*
 * mocap_lbcp_refine -- second stage of latency-balanced chunk partitioning
 * (Section 4.2, Alg. 1, the simulated-annealing refinement), host only.
 *
 * Starting from lengths_inout (typically the dynamic program's plan), the
 * temperature runs from temp0, multiplied by alpha after every `rounds`
 * perturbations, until it is no longer above temp_min.  A perturbation moves
 * one of the num_chunks - 1 inner chunk boundaries by one align unit
 * (seq_len and num_chunks preserved; a move that would empty a chunk is
 * skipped).  A candidate is accepted if its latency T' is lower, or with
 * probability exp(-(T' - T) / Temp); the best partition seen is returned.
 * Random draws come from SplitMix64 seeded with `seed`: for each
 * perturbation, one draw picks the boundary (draw mod (num_chunks - 1)), one
 * the direction (lowest bit), and, for a valid move, one uniform in [0, 1)
 * (the top 53 bits) the acceptance.
 *
 * The latency of a partition is its single-request prefill latency under
 * the same table: sum of chunk costs + (num_stages - 1) * largest chunk cost
 * (a single-request refinement; mocap_lbcp_refine_e2e adds the paper's
 * batch, memory and end-to-end terms).
 *
 *   chunk_cost     as in mocap_lbcp_plan_table
 *   temp0 > 0, temp_min > 0, 0 < alpha < 1, rounds >= 1
 *   lengths_inout  host int32 [num_chunks]: in, a partition of seq_len into
 *                  positive multiples of align; out, the best one found
 *   latency_out    (may be NULL) its latency
 * Errors: INVALID_ARG for malformed sizes, table, schedule or input
 * partition (nothing is written); UNSUPPORTED as in mocap_lbcp_plan.
 */
mocap_status mocap_lbcp_refine(int64_t seq_len, int32_t num_chunks, int32_t num_stages, int32_t align,
                               const double* chunk_cost, double temp0, double temp_min, double alpha,
                               int32_t rounds, uint64_t seed, int32_t* lengths_inout, double* latency_out);

/*
 * mocap_check_block_table -- check the entries of a block table (a HOST copy)
 * that positions [first_pos, end_pos) use: logical blocks first_pos /
 * block_size .. ceil(end_pos / block_size) - 1 must each name a physical
 * block in [0, num_blocks), and no two of them the same one (Section 4.1's
 * reallocation moves blocks; a table that maps two logical blocks onto one
 * physical block would make appends overwrite each other).  Host only.
 *
 *   block_table    host int32 [n_table]
 *   bad_index_out  (may be NULL) the first offending logical block, or -1
 * Returns MOCAP_OK, or MOCAP_ERR_INVALID_ARG for a bad entry, a table shorter
 * than the range needs, a null table for a non-empty range, or malformed
 * sizes.
 */
mocap_status mocap_check_block_table(const int32_t* block_table, int32_t n_table, int64_t first_pos,
                                     int64_t end_pos, int32_t block_size, int32_t num_blocks,
                                     int32_t* bad_index_out);

/*
 * The serving model of mocap_lbcp_evaluate and mocap_lbcp_refine_e2e: the
 * batch size, memory and end-to-end terms of Section 4.2's second stage
 * (EvaluatePrefill and EvaluateE2E of Alg. 1), which the paper names without
 * defining.  The readings this library takes:
 *   - N identical pipeline stages run the chunk operations of `requests`
 *     requests waiting at time 0, served in order in batches of B (the last
 *     one smaller); consecutive batches follow each other through the
 *     pipeline.  A chunk of a batch of n requests takes t + (n - 1) *
 *     max(t - fixed_cost, 0) on every stage, t being its table entry (the
 *     latency for one request) and fixed_cost the part of it a batch does
 *     not multiply.
 *   - A stage holds the KV of a batch's chunks from the start of each chunk
 *     on that stage until the batch leaves the last stage (Section 3.1:
 *     earlier stages hold theirs longer).  One request token occupies
 *     kv_bytes_per_token on a stage; each stage holds stage_capacity bytes of
 *     KV.  pairing = 0: every stage must fit its own capacity at all times;
 *     pairing = 1 (Section 4.1's memory-balanced reallocation with fixed
 *     cross-half pairing, N even): stage i and stage i + N/2 pool their
 *     capacities (a debtor spills to its partner).
 *   - EvaluatePrefill gives B', the largest batch in [1, min(max_batch,
 *     requests)] whose schedule fits (0 if none), and T'_pre, the prefill
 *     latency of one batch of B' (sum of its chunk times + (N - 1) times the
 *     largest); EvaluateE2E gives T', the completion time of the last of
 *     the requests served in batches of B' (the workload's end-to-end
 *     latency; requests / T' is its throughput; +infinity when B' = 0).
 */
typedef struct {
  double fixed_cost;          /* >= 0, in the units of the cost table        */
  double kv_bytes_per_token;  /* > 0                                          */
  double stage_capacity;      /* > 0, bytes of KV one stage holds             */
  int32_t pairing;            /* 0 or 1                                       */
  int32_t max_batch;          /* 1 .. 4096                                    */
  int32_t requests;           /* 1 .. 4096                                    */
} mocap_lbcp_serving;

/*
 * mocap_lbcp_evaluate -- EvaluatePrefill and EvaluateE2E of one partition
 * under the serving model above (host only).
 *
 *   chunk_cost  as in mocap_lbcp_plan_table
 *   serving     the serving model
 *   lengths     host int32 [num_chunks], a partition of seq_len into positive
 *               multiples of align
 *   batch_out, t_pre_out, t_e2e_out   (each may be NULL) B', T'_pre, T'
 * Errors: INVALID_ARG for malformed sizes, table, serving model (pairing with
 * odd num_stages included) or partition; UNSUPPORTED as in mocap_lbcp_plan.
 */
mocap_status mocap_lbcp_evaluate(int64_t seq_len, int32_t num_chunks, int32_t num_stages, int32_t align,
                                 const double* chunk_cost, const mocap_lbcp_serving* serving,
                                 const int32_t* lengths, int32_t* batch_out, double* t_pre_out,
                                 double* t_e2e_out);

/*
 * mocap_lbcp_refine_e2e -- second stage of latency-balanced chunk
 * partitioning (Section 4.2, Alg. 1's simulated annealing) under the serving
 * model: every candidate partition is scored by (B', T'_pre) =
 * EvaluatePrefill, T' = EvaluateE2E, and T' is minimised.  Perturbation,
 * acceptance, cooling and random draws are those of mocap_lbcp_refine (a
 * candidate with T' = +infinity is never accepted over a finite one).
 *
 *   lengths_inout  in: the start partition (typically the dynamic program's);
 *                  out: the best one found
 *   batch_out, t_pre_out, t_e2e_out   (each may be NULL) its B', T'_pre, T'
 * Other arguments as in mocap_lbcp_refine and mocap_lbcp_evaluate.
 * Errors: as mocap_lbcp_evaluate, plus INVALID_ARG for a malformed schedule.
 */
mocap_status mocap_lbcp_refine_e2e(int64_t seq_len, int32_t num_chunks, int32_t num_stages, int32_t align,
                                   const double* chunk_cost, const mocap_lbcp_serving* serving, double temp0,
                                   double temp_min, double alpha, int32_t rounds, uint64_t seed,
                                   int32_t* lengths_inout, int32_t* batch_out, double* t_pre_out,
                                   double* t_e2e_out);

/*
 * Bytes of the library's static device scratch used by
 * mocap_chunk_attn_noalloc (128 MiB, held on every device the library runs
 * on until the process ends).
 */
#define MOCAP_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)

/*
 * mocap_chunk_attn_noalloc -- mocap_chunk_attn without a workspace argument,
 * for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation).  The
 * split partials live in a static device array of MOCAP_NOALLOC_SCRATCH_BYTES
 * inside the library; the call allocates nothing (no hipMalloc, no hipFree,
 * no allocating library routine) and enqueues only kernel launches.
 *
 * Arguments, outputs and errors as in mocap_chunk_attn.  With num_splits = 0
 * the plan is the best automatic plan whose partials fit the scratch (the
 * same plan as mocap_chunk_attn's whenever that one fits); a requested
 * num_splits whose partials need more than MOCAP_NOALLOC_SCRATCH_BYTES
 * (see mocap_chunk_attn_workspace_size) returns MOCAP_ERR_WORKSPACE and
 * launches nothing.  For the same plan the results are bitwise equal to
 * mocap_chunk_attn's.
 *
 * Every call on a device shares that device's scratch, which keeps the last
 * call's contents (nothing needs clearing: every partial a call reads is
 * written earlier by the same call).  Calls that overlap on one device --
 * on different streams, or from different threads without ordering -- race
 * on the scratch; order them on one stream.  The first call on a device
 * looks up the scratch's device address (hipGetSymbolAddress) with that
 * device current; a failure returns MOCAP_ERR_HIP.
 */
mocap_status mocap_chunk_attn_noalloc(const mocap_kv_store* kv, const int32_t* block_table, int32_t n_table,
                                      const void* q, int64_t prefix_len, int32_t chunk_len, int32_t h_q,
                                      int32_t h_kv, int32_t head_dim, float scale, void* o, float* lse,
                                      int32_t num_splits, void* stream);

/* A static, human-readable name for a status code. */
const char* mocap_status_string(mocap_status status);

#ifdef __cplusplus
}
#endif

#endif /* MOCAP_ATTN_H */
