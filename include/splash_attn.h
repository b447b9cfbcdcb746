/*
 * libsplash_attn -- owner-local paged MLA decode attention for MI355X (gfx950).
 *
 * The operation (Sec. 3 "DOP: Computation"; Sec. 3 "Cost"; App. B "Per-Step
 * Cost Model"): an owner GPU holds its N_r = B*q current query rows for all H
 * heads, [N_r, H, d_q] with d_q = d_c + d_r = 576, and the whole latent history
 * of each request it owns, kept in pages.  For every row and every head it
 * attends over the complete causal prefix of that request's history (Sec. 4.1
 * "Handoff") and returns a d_z = d_c = 512 wide output per head.  MLA keeps one
 * head-shared latent row per token (Sec. 1), so one cache row [latent 512 |
 * rope 64] serves as the key of every head, and its first 512 entries serve as
 * the value.  DP-attention and DOP run this same owner-local core (App. B).
 *
 * For request b with history length s_b (s_b counts the current chunk,
 * 1 <= q_chunk <= s_b), chunk row i and head h, output row n = b*q_chunk + i:
 *   visible keys j = 0 .. s_b - q_chunk + i
 *   K_j  = pool row  block_table[b*max_pages_per_seq + j/64]*64 + j%64
 *          (fp8 cache: K_j = e4m3(code) * kv_scales[that row])
 *   z_j  = softmax_scale * <q[n,h,:], K_j>
 *   lse[n,h]   = ln sum_j exp(z_j)                (natural log, scaled logits)
 *   out[n,h,:] = sum_j exp(z_j - lse[n,h]) * K_j[0:512]
 *
 * Entry points: the whole step (splash_mla_attend), its phases (plan,
 * attend_units, combine_splits, run), the standalone LSE merge
 * (splash_mla_combine), and around the same core: one position shard of the
 * histories (splash_mla_attend_shard), attention over listed positions only
 * (splash_mla_attend_topk), and the DOP regroup of query and output rows
 * (splash_dop_*).
 *
 * Conventions for every entry point:
 *  - All tensor pointers are DEVICE pointers owned by the caller; the library
 *    never allocates or frees device memory in these calls and keeps no
 *    pointer after it returns.  `stream` is a hipStream_t (NULL: the null
 *    stream); all work is enqueued on it with no host synchronisation (except
 *    under SPLASH_FLAG_DEBUG_CHECK), so the calls can be captured in a graph.
 *  - Return value: SPLASH_OK or a negative status; no C++ exception crosses
 *    the boundary.  splash_status_string() names a status and
 *    splash_last_error() holds the last detailed message of the calling
 *    thread.
 *  - Device data is trusted on the fast path: seq_lens[b] < q_chunk or a
 *    block-table entry outside [0, num_pages) is undefined behaviour unless
 *    SPLASH_FLAG_DEBUG_CHECK is set, which validates them first.
 *  - Unused block-table slots (past ceil(s_b/64)) and pool rows past a
 *    history's end are never used in the result.
 */
#ifndef SPLASH_ATTN_H
#define SPLASH_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes -------------------------------------------------------- */
#define SPLASH_OK                        0
#define SPLASH_ERR_INVALID_ARGUMENT     (-1) /* null pointer, q_chunk<1, dims != 576/512, bad scale, bad device data */
#define SPLASH_ERR_UNSUPPORTED          (-2) /* H not in {16,32,...,128}, page size != 64, unknown kv dtype */
#define SPLASH_ERR_MISALIGNED           (-3) /* a tensor base pointer not 16-byte aligned */
#define SPLASH_ERR_WORKSPACE_TOO_SMALL  (-4)
#define SPLASH_ERR_HIP                  (-5) /* a HIP call or launch failed; see splash_last_error() */

/* ---- cache formats --------------------------------------------------------- */
#define SPLASH_KV_BF16      0  /* pool: [num_pages, 64, 576] bf16 */
#define SPLASH_KV_FP8_E4M3  1  /* pool: [num_pages, 64, 576] OCP E4M3 ("fn") bytes + kv_scales [num_pages, 64] fp32 */
/* Latent-row cache (App. B, theoretical scenarios for DCU and H200,
 * residency assumptions: FP8 latent with its scales and BF16 RoPE; the
 * paper fixes neither the split nor the scale granularity).  Pool:
 * [num_pages, 64, 656] bytes; a row is 512 OCP E4M3 latent codes, four
 * little-endian fp32 scales (scale t covers latent columns [128t, 128t+128))
 * and the 64 RoPE values as bf16: K[d] = e4m3(code[d]) * scale[d / 128] for
 * d < 512, K[512 + r] = rope[r].  Scales must be positive normal powers
 * of two no larger than 2^63 (the conversion uses only a scale's exponent,
 * and the weights take it as an exponent step); rows no history reaches may
 * hold anything.  Under SPLASH_FLAG_DEBUG_CHECK every entry point rejects a
 * reached (top-k: listed) row whose scale is not.  kv_scales is ignored.
 * Every attend entry point (whole histories, shards, top-k) and the gather
 * take it. */
#define SPLASH_KV_FP8_LATENT 2

/* ---- flags ------------------------------------------------------------------ */
#define SPLASH_FLAG_DEBUG_CHECK  1u  /* validate seq_lens / block table on the device first; synchronises `stream` */
#define SPLASH_FLAG_FORCE_SPLIT  2u  /* split every history into work units of `split_pages` pages */
/* fp8 caches (App. C: FP8 E4M3 KV): QK with K converted exactly to bf16 and
 * the bf16 MFMA's fp32 sums, instead of the default: K's own codes on the fp8
 * matrix pipe against the query split exactly into two E4M3 terms, faster
 * (config 5: attend 629 against 722 us, latent rows 697 against 772) with sums kept to about 2^-18 of sum |q_i k_i|, so a
 * score is off by up to about 2^-18 * softmax_scale * sum |q_i k_i|.  No
 * effect on the bf16 cache. */
#define SPLASH_FLAG_EXACT_QK     4u

#define SPLASH_DIM_QK     576
#define SPLASH_DIM_V      512
#define SPLASH_PAGE_SIZE  64
#define SPLASH_MAX_HEADS  128

/* Description of one call.  Sizes are element counts. */
typedef struct splash_mla_desc {
    int32_t batch;              /* B: requests owned by this GPU (0: idle owner, every call is a no-op) */
    int32_t num_heads;          /* H: query heads, a multiple of 16 in [16, 128] */
    int32_t dim_qk;             /* must be 576 = 512 latent + 64 rope */
    int32_t dim_v;              /* must be 512 */
    int32_t page_size;          /* must be 64 */
    int32_t max_pages_per_seq;  /* row stride of block_table (>= ceil(max s_b / 64)) */
    int32_t num_pages;          /* pages in the pool */
    int32_t kv_dtype;           /* SPLASH_KV_* */
    const float* kv_scales;     /* device [num_pages, 64] fp32 per-token scales; SPLASH_KV_FP8_E4M3 only, else ignored */
    float softmax_scale;        /* multiplies <q, k>; finite and > 0 (1/sqrt(192) for DeepSeek-V3 dims) */
    uint32_t flags;             /* SPLASH_FLAG_* */
    int32_t split_pages;        /* with SPLASH_FLAG_FORCE_SPLIT: pages per work unit, >= 1 */
} splash_mla_desc;

/*
 * Workspace.  One caller-allocated device buffer carries the plan (work list,
 * split offsets) and the partial results of split histories.
 * `max_partials` bounds how many partial results (one per work unit of a
 * split history, room for H x 512 fp32 each) the planner may use; <= 0 selects
 * SPLASH_DEFAULT_MAX_PARTIALS.  The planner never exceeds the capacity that
 * the passed ws_bytes provides: with too little room it splits less.
 * Layout (byte offsets from splash_mla_workspace_offsets, 256-byte aligned):
 *   [0] header int32[1152]: [1] number of work units, [2] partial slots
 *       used, [3] pages per unit chosen (0 for a fold plan), [4] debug
 *       status, [6] number of split tiles, [7] total pages, [8] most parts of
 *       a split tile, [9] workers of a fold plan (0: the queue, ordered
 *       longest unit first and dealt to the workers in a snake), [10] the fold
 *       plan's cap; from [64] the fold plan's first unit of each worker
 *       (workers + 1 entries).  [0] and [5] are written as 0 and unused.
 *   [1] work units int32[max_units][4] = {tile, first page, end page, slot},
 *       tile = b*q_chunk + i, slot = partial index or -1 (unit writes out/lse)
 *   [2] split offsets int32[B*q_chunk + 1] (partial slots of tile t are
 *       [off[t], off[t+1]); empty when the tile is a single unit)
 *   [3] split tiles int32[B*q_chunk] (the tiles with partials, ascending)
 *   [4] partial lse fp32 [max_partials, H]
 *   [5] partial out: room for fp32 [max_partials, H, 512]; the library keeps
 *       them as fp16 [max_partials, H, 512] (the first half of the region),
 *       each (slot, head) 128-column quarter q multiplied by 2^-e, with e
 *       byte q of uint32 [max_partials, H] right after them (e = 0 unless
 *       the quarter's largest magnitude reaches 2^15; then every stored
 *       value stays below 2^15).  Internal: only splash_mla_combine_splits
 *       reads them.
 */
#define SPLASH_DEFAULT_MAX_PARTIALS 1024
size_t splash_mla_workspace_size(int32_t batch, int32_t q_chunk, int32_t num_heads,
                                 int32_t max_partials);
/* Writes the six byte offsets above into offsets[6]; returns the total size. */
size_t splash_mla_workspace_offsets(int32_t batch, int32_t q_chunk, int32_t num_heads,
                                    int32_t max_partials, size_t* offsets);

/*
 * splash_mla_attend: the whole step -- plan, attend, combine -- on `stream`.
 *   q            bf16 [B*q_chunk, H, 576], row n = b*q_chunk + i, each head's 576
 *                entries packed [no-position 512 | rotary 64] (App. E)
 *   kv_pages     pool, see SPLASH_KV_*
 *   block_table  int32 [B, max_pages_per_seq]; logical page k of request b is
 *                physical page block_table[b*max_pages_per_seq + k]
 *   seq_lens     int32 [B], history length including the current chunk
 *   q_chunk      query rows per request (1: decode), 1 <= q_chunk <= seq_lens[b]
 *   out          bf16 [B*q_chunk, H, 512] (round to nearest even)
 *   lse          fp32 [B*q_chunk, H] natural-log LSE of the scaled logits; may be NULL
 * Results are deterministic: the same inputs give the same bits, independent
 * of page placement in the pool and of how units land on compute units.
 */
int splash_mla_attend(const void* q, const void* kv_pages, const int32_t* block_table,
                      const int32_t* seq_lens, int32_t q_chunk, void* out, float* lse,
                      const splash_mla_desc* desc, void* workspace, size_t ws_bytes,
                      void* stream);

/*
 * splash_mla_attend_noalloc: splash_mla_attend for callers that cannot
 * allocate device memory (code under graph capture, tight serving loops,
 * harnesses that forbid allocation): the same step on a workspace the
 * library owns, so the caller passes inputs and outputs only.
 *   The workspace is a device array of SPLASH_NOALLOC_SCRATCH_BYTES inside
 *   the library, one per GPU the library runs on, held until the process
 *   ends; its address is looked up once per device.  The call allocates
 *   nothing and enqueues only kernels on `stream`.
 *   Every call on one GPU shares that GPU's array: calls that overlap on one
 *   GPU (other streams, other threads) race and give undefined results;
 *   calls in one stream order are fine.  Nothing in the array needs to
 *   start at zero: the plan writes everything the later kernels read.
 *   Arguments as for splash_mla_attend.  Errors: as splash_mla_attend, plus
 *   SPLASH_ERR_WORKSPACE_TOO_SMALL when the batch's minimum workspace (its
 *   plan, plus the partials that histories longer than 1024 pages force)
 *   exceeds the array; with less room than splash_mla_attend's default
 *   workspace the planner splits less.  SPLASH_FLAG_DEBUG_CHECK is refused
 *   (SPLASH_ERR_UNSUPPORTED): its check reads a result back to the host.
 */
#define SPLASH_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
int splash_mla_attend_noalloc(const void* q, const void* kv_pages, const int32_t* block_table,
                              const int32_t* seq_lens, int32_t q_chunk, void* out, float* lse,
                              const splash_mla_desc* desc, void* stream);

/*
 * splash_mla_plan + splash_mla_run: the same step in two halves, so that a
 * plan made once per step (it depends only on seq_lens, q_chunk and desc) can
 * serve every layer.  splash_mla_run must see the workspace of a plan made
 * with the same seq_lens, q_chunk and desc, earlier in stream order.
 * The split heuristic (a cost-model argmin over candidate unit sizes, in the
 * spirit of Sec. 4.2's calibrated argmin) balances pages over the compute
 * units and splits a history only where that shortens the step.
 */
int splash_mla_plan(const int32_t* seq_lens, int32_t q_chunk, const splash_mla_desc* desc,
                    void* workspace, size_t ws_bytes, void* stream);
int splash_mla_run(const void* q, const void* kv_pages, const int32_t* block_table,
                   const int32_t* seq_lens, int32_t q_chunk, void* out, float* lse,
                   const splash_mla_desc* desc, void* workspace, size_t ws_bytes,
                   void* stream);

/*
 * splash_mla_attend_units + splash_mla_combine_splits: splash_mla_run in its
 * two launches.  attend_units processes every work unit of the plan: a tile
 * (query row with all heads) that is one unit writes its out/lse rows
 * directly; the units of a split tile write partials (fp16 with a
 * power-of-two scale, see the workspace layout) into the workspace.  combine_splits merges those partials into out/lse (its
 * arguments must match the attend_units call).  Same argument rules as
 * splash_mla_run.
 */
int splash_mla_attend_units(const void* q, const void* kv_pages, const int32_t* block_table,
                            const int32_t* seq_lens, int32_t q_chunk, void* out, float* lse,
                            const splash_mla_desc* desc, void* workspace, size_t ws_bytes,
                            void* stream);
int splash_mla_combine_splits(int32_t q_chunk, void* out, float* lse, const splash_mla_desc* desc,
                              void* workspace, size_t ws_bytes, void* stream);

/*
 * splash_mla_attend_topk: top-k (sparse) attention, the attention the paper's
 * sparse backend runs (each row attends a selected subset of its history,
 * chosen by an indexer that is not part of this library).  Row n =
 * b*q_chunk + i attends the token positions topk_idx[n][0 .. topk_count[n])
 * of request b's history, with the logits, values, softmax and LSE of
 * splash_mla_attend restricted to those keys:
 *   topk_idx    device int32 [B*q_chunk, topk]: positions, each in the row's
 *               visible prefix [0, seq_lens[b] - q_chunk + i]; entries past
 *               the count are not read.  A position listed twice counts twice.
 *   topk_count  device int32 [B*q_chunk], 0 <= count <= topk; a row with an
 *               empty list gets out = 0, lse = -inf.
 * Only the block-table entries of listed positions are read.  Lists longer
 * than 2048 entries are split into partials (the workspace needs room for
 * B*q_chunk*ceil(ceil(topk/64)/32) of them, else WORKSPACE_TOO_SMALL);
 * SPLASH_FLAG_FORCE_SPLIT takes split_pages <= 32 (groups of 64 entries).
 * SPLASH_FLAG_DEBUG_CHECK validates counts, positions and their pages.  Other
 * arguments as for splash_mla_attend.
 */
int splash_mla_attend_topk(const void* q, const void* kv_pages, const int32_t* block_table,
                           const int32_t* seq_lens, int32_t q_chunk, const int32_t* topk_idx,
                           const int32_t* topk_count, int32_t topk, void* out, float* lse,
                           const splash_mla_desc* desc, void* workspace, size_t ws_bytes,
                           void* stream);

/*
 * DOP regroup (Sec. 3 "DOP: Computation"; App. E, DOP transfer).  With
 * sharded projections, rank t of T holds all N current query rows for its
 * heads_local = H/T heads (global heads [t*H/T, (t+1)*H/T)); the owner of a
 * request needs that request's rows for all H heads.  A variable-size
 * all-to-all (not part of this library; its split sizes are the per-owner
 * row counts) moves one contiguous block between every pair.  These calls
 * build and take apart those blocks; rows keep their identity, heads their
 * order, and each packed query row carries the no-position part followed by
 * the rotary part.  All tensors are bf16, contiguous, 16-byte aligned
 * device buffers; row_order is a device int32 [num_rows] permutation of the
 * rows, grouped by owner (owner 0's rows first); it is not validated.
 *
 * splash_dop_pack_q (rank side, before attention):
 *   q_nope [num_rows, heads_local, 512], q_rope [num_rows, heads_local, 64]
 *   -> send [num_rows, heads_local, 576], send[k] = q_nope[row_order[k]] | q_rope[row_order[k]]
 * splash_dop_unpack_q (owner side): recv [num_ranks, owner_rows, heads_local,
 *   576] (rank t's block t) -> q_owner [owner_rows, num_ranks*heads_local, 576],
 *   q_owner[i][t*heads_local + h] = recv[t][i][h]
 * splash_dop_pack_out (owner side, after attention): out_owner [owner_rows,
 *   num_ranks*heads_local, 512] -> send [num_ranks, owner_rows, heads_local,
 *   512], send[t][i][h] = out_owner[i][t*heads_local + h]
 * splash_dop_unpack_out (rank side): recv [num_rows, heads_local, 512] in
 *   row_order -> out [num_rows, heads_local, 512], out[row_order[k]] = recv[k]
 *
 * Zero rows is a no-op (an owner with no rows still takes part in the
 * exchange).  Errors: INVALID_ARGUMENT for negative or zero sizes or NULL
 * buffers, MISALIGNED, UNSUPPORTED when rows * H * 72 reaches 2^31.
 */
int splash_dop_pack_q(const void* q_nope, const void* q_rope, const int32_t* row_order,
                      int32_t num_rows, int32_t heads_local, void* send, void* stream);
int splash_dop_unpack_q(const void* recv, int32_t num_ranks, int32_t owner_rows,
                        int32_t heads_local, void* q_owner, void* stream);
int splash_dop_pack_out(const void* out_owner, int32_t num_ranks, int32_t owner_rows,
                        int32_t heads_local, void* send, void* stream);
int splash_dop_unpack_out(const void* recv, const int32_t* row_order, int32_t num_rows,
                          int32_t heads_local, void* out, void* stream);

/*
 * splash_mla_attend_shard: the partial result of one position shard (App. E,
 * position-sharded CP: each rank holds a slice of a request's token history,
 * and the ranks' partial results are merged by their log-sum-exp).  For every
 * query row n = b*q_chunk + i and head h it attends over the keys of request
 * b in [key_begin[b], key_end[b]) that row n sees (j <= seq_lens[b] - q_chunk
 * + i), and writes the normalised fp32 output and its natural-log LSE into
 * slot b*num_shards + shard:
 *   part_out  fp32 [B*num_shards, q_chunk, H, 512]: rows of request b, shard k
 *             at slot b*num_shards + k (this call writes its shard's slots)
 *   part_lse  fp32 [B*num_shards, q_chunk, H]
 * A row that sees no key of the shard gets out = 0 and lse = -inf.  After the
 * num_shards calls (any order, same workspace reused), splash_mla_combine
 * with split_indptr[b] = b*num_shards merges them into the result over the
 * union of the shards: with shards that tile [0, seq_len) it equals
 * splash_mla_attend.
 *   key_begin, key_end  device int32 [B]; key_begin[b] a multiple of 64 (the
 *             shard starts on a page), 0 <= key_begin[b] <= key_end[b]; only
 *             the block-table entries of the shard's pages are read.
 * The workspace needs a partial slot per query row (max_partials >= B *
 * q_chunk, else SPLASH_ERR_WORKSPACE_TOO_SMALL).  Other arguments as for
 * splash_mla_attend; SPLASH_FLAG_FORCE_SPLIT is rejected (UNSUPPORTED), and
 * SPLASH_FLAG_DEBUG_CHECK also checks the key ranges.
 */
int splash_mla_attend_shard(const void* q, const void* kv_pages, const int32_t* block_table,
                            const int32_t* seq_lens, int32_t q_chunk, const int32_t* key_begin,
                            const int32_t* key_end, int32_t num_shards, int32_t shard, float* part_out,
                            float* part_lse, const splash_mla_desc* desc, void* workspace,
                            size_t ws_bytes, void* stream);

/*
 * splash_mla_combine: merge partial attention results over disjoint key sets
 * into the result over their union (the merge a position-sharded history
 * needs, App. E).  For request b, partial slots s in
 * [split_indptr[b], split_indptr[b+1]) each hold rows i < q_chunk:
 *   partials     fp32 [S_tot, q_chunk, H, 512], normalised outputs
 *   partial_lse  fp32 [S_tot, q_chunk, H]; -inf marks a part with no key
 *   L = ln sum_s exp(lse_s);  out = sum_s exp(lse_s - L) * partial_s
 *   out          bf16 [B*q_chunk, H, 512]; out_lse fp32 [B*q_chunk, H] or NULL
 * A request with no partial, or whose parts are all -inf, gets out = 0 and
 * lse = -inf.  split_indptr is a device int32 [B+1] array.
 */
int splash_mla_combine(const float* partials, const float* partial_lse,
                       const int32_t* split_indptr, int32_t batch, int32_t q_chunk,
                       int32_t num_heads, void* out, float* out_lse, void* stream);

/*
 * splash_mla_debug_gather (tests): copy every history, token by token, into
 * a dense buffer through the same page-address code the attention kernel
 * uses.  dense_out holds sum_b seq_lens[b] rows of the pool's row bytes
 * (1152 for bf16, 576 for fp8, 656 for latent rows), request after request.
 */
int splash_mla_debug_gather(const void* kv_pages, const int32_t* block_table,
                            const int32_t* seq_lens, const splash_mla_desc* desc,
                            void* dense_out, void* stream);

/*
 * splash_mla_plan_host: the planner run on the CPU over HOST seq_lens, for
 * tests and for callers that want to inspect a plan.  It computes exactly
 * what splash_mla_plan computes on the device for `num_workers` compute units
 * and `max_partials` partial slots.  units_out: int32 [max_units][4];
 * indptr_out: int32 [B*q_chunk + 1]; stats_out: int32[7] = {units, partial
 * slots used, pages per unit (0 for a fold plan), total pages, workers of a
 * fold plan (0: the queue, dealt to the workers in a snake), the pages a fold plan
 * lets a long history keep (the rest goes to a second worker), the most
 * parts of any split tile}; worker_start_out (may be NULL): int32
 * [num_workers + 1], for a fold plan the first unit of each worker (worker g
 * runs units [w[g], w[g+1])), untouched otherwise.  Returns SPLASH_OK, or
 * SPLASH_ERR_WORKSPACE_TOO_SMALL when max_units is too small.
 */
int splash_mla_plan_host(const int32_t* seq_lens_host, int32_t q_chunk,
                         const splash_mla_desc* desc, int32_t num_workers,
                         int32_t max_partials, int32_t* units_out, int32_t max_units,
                         int32_t* indptr_out, int32_t* stats_out, int32_t* worker_start_out);

/* Number of work units the workspace reserves: B*q_chunk + max_partials. */
int32_t splash_mla_max_units(int32_t batch, int32_t q_chunk, int32_t max_partials);

/* Compute units of the current device as the planner sees them (>= 1). */
int32_t splash_device_workers(void);

const char* splash_status_string(int status);
const char* splash_last_error(void);
const char* splash_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SPLASH_ATTN_H */
