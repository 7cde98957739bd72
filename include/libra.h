/*
 * libra.h -- C ABI of the MI355X (gfx950) Libra hot path.
 *
 * Libra (arXiv 2607.23250) balances document-masked causal attention over a
 * pool of fixed-token packed sequences by cutting it into SH-Tiles
 * (sequence block x query-head shard, Sec. 4.3.1, Eq. 5), costing every tile
 * by its exact causal pair count (Eq. 6) and placing tiles on the pool's
 * workers with a communication-aware greedy rule (Sec. 4.3.2, Algorithm 2).
 * This library exposes that path on one GPU:
 *
 *   libra_plan      host, integer: tiles, costs and the placement;
 *   libra_attn_fwd  device: O and the log-sum-exp for a list of tiles;
 *   libra_attn_bwd  device: dQ, dK, dV for the same tiles.
 *
 * Conventions shared by every entry point
 *   - Return 0 (LIBRA_OK) or a negative LIBRA_E* code; nothing throws across
 *     the ABI.  libra_strerror(code) names a code; libra_last_error() gives a
 *     thread-local description of the last failure on the calling thread.
 *   - Token positions are pool coordinates: packs are concatenated in pool
 *     order, samples in pack order.  cu_seqlens[j] is the first position of
 *     sample j, cu_seqlens[n] the pool size; pack_cu likewise for packs.
 *   - Tensors use the THD layout: row-major [rows][heads][head_dim].  K and V
 *     rows are pool positions; Q, O, dO and dQ rows are the rows listed by the
 *     tiles (q_row .. q_row + q_end - q_begin).  LSE is fp32 [h_q][n_q_rows].
 *   - Grouped-query heads map contiguously: kv_head = q_head / (h_q / h_kv).
 *   - The caller owns and allocates every buffer.  Device entry points take
 *     device pointers, enqueue work on `stream` (a hipStream_t; NULL is the
 *     default stream) and return without synchronizing.  They never allocate.
 *     Invalid arguments are rejected on the host before anything is enqueued.
 *     A kernel fault is reported by the caller's next synchronization.
 */
#ifndef LIBRA_H
#define LIBRA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  LIBRA_OK = 0,
  LIBRA_EINVAL = -1,        /* malformed arguments */
  LIBRA_ENOSPC = -2,        /* an output or workspace buffer is too small */
  LIBRA_EUNSUPPORTED = -3,  /* valid but not implemented (e.g. head_dim) */
  LIBRA_EOVERFLOW = -4,     /* an integer result does not fit its type */
  LIBRA_EHIP = -5           /* a HIP runtime call or kernel launch failed */
};

/* One SH-Tile (Eq. 5): sequence block x head shard. 56 bytes, naturally aligned. */
typedef struct libra_tile {
  int64_t q_begin;    /* first query position of the block (pool coordinates) */
  int64_t q_end;      /* one past the last position; q_end - q_begin <= B */
  int64_t q_row;      /* row of q_begin in the Q / O / dO / dQ / LSE buffers */
  int64_t cost;       /* Eq. 6: (h_q / H) * causal same-sample (q, k) pairs */
  int32_t head_begin; /* query heads [head_begin, head_end), width h_q / H */
  int32_t head_end;
  int32_t pack;       /* pack index in the pool */
  int32_t home;       /* Q-home worker q(t) (Sec. 4.3.2) */
  int32_t worker;     /* assigned worker sigma(t) from Algorithm 2 */
  int32_t id;         /* tile ID = pool_block_index * H + shard */
} libra_tile_t;

/* Plan parameters.  V = num_packs * cp virtual workers. */
typedef struct libra_plan_cfg {
  int32_t block_tokens;  /* B (>= 1) */
  int32_t head_shards;   /* H; must divide num_q_heads; h_kv % H == 0 or H % h_kv == 0 */
  int32_t num_packs;     /* P */
  int32_t cp;            /* CP degree; every pack length is a multiple of 2*cp */
  int32_t num_q_heads;   /* h_q */
  int32_t num_kv_heads;  /* h_kv; divides h_q */
  int32_t head_dim;      /* d (any value >= 1 for planning) */
  int32_t elem_bytes;    /* bytes per element of Q/K/V/O (2 for bf16) */
  int32_t tau_num;       /* tau = tau_num / tau_den (the paper fixes 3/100) */
  int32_t tau_den;
} libra_plan_cfg_t;

const char *libra_strerror(int code);
const char *libra_last_error(void);

/*
 * libra_plan -- SH-Tiles, Eq. 6 costs and Algorithm 2 placement (host only).
 *
 * Blocks of at most B tokens are cut at positions of each pack (no extra cut
 * at sample boundaries, the last block may be short); each block with each of
 * the H query-head shards is one tile (Sec. 4.3.1).  Tile cost, the KV groups
 * K(t) (Eq. 7) and the communication increment (Eq. 8) feed Algorithm 2 with
 * capacity C = (1 + tau) * sum(f) / V, evaluated exactly in integers.
 * Q-home: pack p is split into 2*cp equal chunks; chunk c is held by CP rank
 * c (c < cp) or 2*cp-1-c, and worker ids are p*cp + rank.  A worker initially
 * holds the KV groups of the samples lying wholly on it.  KV group bytes are
 * len * max(1, h_kv/H) * d * elem_bytes * 2; Q and O bytes are
 * rows * (h_q/H) * d * elem_bytes each.
 *
 *   lengths[num_samples], cu_seqlens[num_samples+1], pack_cu[num_packs+1]:
 *       host arrays; cu_seqlens[0] = 0, cu_seqlens[j+1]-cu_seqlens[j] =
 *       lengths[j] >= 1, pack boundaries fall on sample boundaries.
 *   q_ranges[2*num_q_ranges]: host [begin, end) pairs selecting the query
 *       rows present (whole blocks only, sorted, disjoint), or NULL for all.
 *       Rows are numbered in position order over the selected ranges.
 *       Absent blocks yield no tile but keep their place in the tile IDs.
 *   tiles[tiles_cap]: output in tile-ID order, or NULL to query the count.
 *   num_tiles: out, number of tiles (also set when tiles is NULL).
 *   worker_load[V]: out, Algorithm 2 load L_r of every worker (may be NULL).
 *   worker_bytes[V]: out, bytes every worker receives under the plan (may be
 *       NULL): the sum of Eq. 8 over the tiles placed on it, each evaluated
 *       when the tile was placed (KV groups not yet held, plus Q rows and
 *       outputs of tiles it does not home).
 * Errors: EINVAL (inconsistent inputs), ENOSPC (tiles_cap too small;
 * *num_tiles still holds the count), EOVERFLOW (a cost or byte count
 * overflows int64).  Reentrant; allocates only host memory it frees.
 */
int libra_plan(const libra_plan_cfg_t *cfg, const int64_t *lengths, int64_t num_samples,
               const int64_t *cu_seqlens, const int64_t *pack_cu, const int64_t *q_ranges,
               int32_t num_q_ranges, libra_tile_t *tiles, int64_t tiles_cap,
               int64_t *num_tiles, int64_t *worker_load, int64_t *worker_bytes);

/*
 * libra_vrsp -- Variance-Reduced Sequence Placement (Sec. 4.2, Algorithm 1;
 * host only).
 *
 * Forms K = num_seqs / pool_size sequence pools of exactly pool_size packed
 * sequences from one optimizer-step window.  Workload F_i = sum of squared
 * raw-sample lengths of sequence i (Eq. 4).  Sequences are taken in order
 * of decreasing F_i, ties by increasing index; each joins the pool of least
 * (load, pool index) among the pools holding fewer than pool_size
 * sequences.  The output concatenates the pools in pool-index order
 * (GA-major, pool-minor), each pool in placement order.
 *
 *   lengths[num_samples]: host array, the raw-sample lengths (>= 1) of all
 *       packed sequences of the window, sequence after sequence.
 *   seq_cu[num_seqs+1]: host array, sequence i holds samples
 *       [seq_cu[i], seq_cu[i+1]); seq_cu[0] = 0, seq_cu[num_seqs] =
 *       num_samples, nondecreasing.
 *   order[num_seqs]: out, original sequence indices in output order.
 *   pool_load[num_seqs / pool_size]: out, summed workload of each pool
 *       (may be NULL).
 *   seq_work[num_seqs]: out, F_i (may be NULL).
 * Errors: EINVAL (pool_size < 1 or not dividing num_seqs, inconsistent
 * offsets or lengths, NULL arguments), EOVERFLOW (a workload or pool load
 * overflows int64).  Reentrant; allocates only host memory it frees.
 */
int libra_vrsp(const int64_t *lengths, int64_t num_samples, const int64_t *seq_cu,
               int64_t num_seqs, int32_t pool_size, int64_t *order, int64_t *pool_load,
               int64_t *seq_work);

/*
 * libra_attn_workspace_size -- bytes of device workspace that
 * libra_attn_fwd (backward = 0) or libra_attn_bwd (backward = 1) needs for
 * these sizes.  Returns 0 for invalid sizes.
 */
size_t libra_attn_workspace_size(int64_t num_tiles, int64_t num_samples, int64_t n_q_rows,
                                 int64_t n_kv_rows, int32_t h_q, int32_t h_kv, int32_t head_dim,
                                 int32_t backward);

/*
 * libra_attn_fwd -- document-masked causal attention (Eq. 1 under the
 * block-diagonal causal mask of Sec. 2.3) for every (row, query head) covered
 * by the tiles:
 *     O   = softmax(q K^T * scale + M) V  over the keys of the row's own
 *           sample at sample-local positions <= the row's own,
 *     LSE = natural log of sum(exp(q K^T * scale)) over the same keys.
 *   q [n_q_rows][h_q][d], k, v [n_kv_rows][h_kv][d]: bf16, device.
 *   cu_seqlens [num_samples+1]: int64, device, as in libra_plan.
 *   tiles [num_tiles]: device copy of libra_plan output (only q_begin, q_end,
 *       q_row, head_begin, head_end are read).  Tiles must not overlap in
 *       (row, head); any subset of a plan (one worker's tiles) is valid.
 *   head_dim: 64 or 128 (else EUNSUPPORTED).  softmax_scale <= 0 means 1/sqrt(d).
 *   o [n_q_rows][h_q][d] bf16, lse [h_q][n_q_rows] fp32: device outputs; only
 *       covered (row, head) entries are written.
 *   workspace: device, >= libra_attn_workspace_size(..., 0) bytes, 256-byte
 *       aligned; contents are scratch.  It holds the work items and the
 *       split-K partial results (3072 slots of 128 rows x (d + 2) fp32, about
 *       200 MB at d = 128).
 * Split K: a call with fewer than two work items per workgroup (few rows and
 * heads against long samples) cuts its long items into key ranges that run in
 * parallel and merges their partial results (the online-softmax recurrence
 * across ranges); the result is the same up to the order of fp32 additions.
 * Rows and heads are processed independently of how tiles group them, so the
 * output does not depend on B, H or the worker a tile was placed on; it is
 * bit-identical across such groupings whenever no item is split.
 */
int libra_attn_fwd(const void *q, const void *k, const void *v, const int64_t *cu_seqlens,
                   int64_t num_samples, const libra_tile_t *tiles, int64_t num_tiles,
                   int64_t n_q_rows, int64_t n_kv_rows, int32_t h_q, int32_t h_kv,
                   int32_t head_dim, float softmax_scale, void *o, float *lse, void *workspace,
                   size_t workspace_bytes, void *stream);

/*
 * Tiles that do not lie inside the buffers a call describes (q_begin < 0,
 * q_end > n_kv_rows, empty ranges, rows past n_q_rows, heads outside
 * [0, h_q)) are skipped on the device: the call still returns LIBRA_OK and
 * computes every other tile exactly as without them.  The number skipped by
 * the last libra_attn_fwd or libra_attn_bwd call that used a workspace is an
 * int32 at byte offset LIBRA_WS_SKIPPED_OFFSET of that workspace (plus 1 if
 * the workspace's work-item list overflowed, which a workspace of
 * libra_attn_workspace_size bytes rules out).
 *
 * libra_attn_skipped_tiles -- copies that count to *count after the work
 * already enqueued on `stream` has finished (it synchronizes `stream`).
 *   workspace: the device workspace of that call (256-byte aligned).
 * Errors: EINVAL (NULL arguments), EHIP.
 *
 * Tiles that overlap in (row, head) are not detected.  Each copy is computed
 * in full: O, LSE and dQ of the shared pairs are written twice with the same
 * values, and dK / dV receive their contribution twice.  libra_plan never
 * produces overlapping tiles.
 */
#define LIBRA_WS_SKIPPED_OFFSET 16
int libra_attn_skipped_tiles(const void *workspace, int32_t *count, void *stream);

/*
 * libra_attn_fwd_noalloc -- libra_attn_fwd without a workspace argument, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation).  Same arguments,
 * semantics and errors as libra_attn_fwd, with the same kernels but without
 * split K (its partial slots would not fit), so its results equal
 * libra_attn_fwd's whenever that call splits no item; the work items live in
 * a device array built into the library, of LIBRA_FWD_NOALLOC_MAX_WORKSPACE
 * bytes, one per device, held until the process ends.  The call allocates
 * nothing and frees nothing (its first call on a device looks up that
 * device's array).
 *   Sizes whose work-item list (48 bytes per item, bounded from the sizes as
 *   for libra_attn_workspace_size) exceeds the array are rejected with
 *   LIBRA_ENOSPC before anything is enqueued (16 MiB covers, e.g., 65536
 *   query rows x 32 heads of a 1M-token pack).
 *   Every call on one device shares that device's array: calls that overlap
 *   in time on one device (different streams, or host threads) race and
 *   must be serialized by the caller.  Each call's preparation pass rewrites
 *   every part of the array it later reads, so nothing needs clearing
 *   between calls.  The skipped-tile count of these calls is not exposed.
 */
#define LIBRA_FWD_NOALLOC_MAX_WORKSPACE ((size_t)16 << 20)
int libra_attn_fwd_noalloc(const void *q, const void *k, const void *v,
                           const int64_t *cu_seqlens, int64_t num_samples,
                           const libra_tile_t *tiles, int64_t num_tiles, int64_t n_q_rows,
                           int64_t n_kv_rows, int32_t h_q, int32_t h_kv, int32_t head_dim,
                           float softmax_scale, void *o, float *lse, void *stream);

/* libra_attn_bwd flags */
#define LIBRA_BWD_ACCUMULATE_DKV 1u /* dk, dv are fp32 and are added to (not overwritten) */

/*
 * libra_attn_bwd -- gradients of sum(dO * O) for the rows and heads covered
 * by the tiles (the textbook attention backward; the paper's backward reuses
 * the forward assignment, Sec. 4.3.3):
 *     P = exp(q K^T * scale - LSE),  D = rowsum(dO * O),
 *     dV = P^T dO,  dS = P * (dO V^T - D),  dQ = scale * dS K,  dK = scale * dS^T q,
 * with dK / dV summed over the query heads of each KV head.
 *   q, k, v, o, dout: bf16 device tensors as in libra_attn_fwd; lse fp32 as
 *       returned by libra_attn_fwd for the same tiles.
 *   dq [n_q_rows][h_q][d] bf16: covered (row, head) entries are written.
 *   dk, dv [n_kv_rows][h_kv][d]: bf16, every element written (zero where no
 *       covered row attends); with LIBRA_BWD_ACCUMULATE_DKV they are fp32 and
 *       this call's contribution is added, so several disjoint tile sets
 *       (virtual workers) can be summed into one caller-zeroed buffer.
 *   workspace: >= libra_attn_workspace_size(..., 1) bytes, 256-byte aligned.
 * Precision: the dK / dV products take fp16 copies of q, dout, k and v, each
 * scaled by a power of two from its max |x| over what the products read, so
 * that P and dS round to 11 significant bits instead of bf16's 8; the scales
 * are undone exactly on output.  dQ's products take the bf16 inputs.
 * Inputs: every element of k and v in the samples the tiles touch, and of
 * q, dout, o and lse in the covered (row, head) pairs, must be finite.
 * Other rows of q, dout, o and lse are not read by the dK / dV products
 * (their fp16 copies hold zeros there).
 * Split K: the dQ products split their work items into key ranges as the
 * forward does, when the call's items would leave more than a tenth of the
 * workgroups idle; the parts' fp32 dQ and sums of dS are merged before the
 * dK / dV products read D.  The workspace holds those partial results too.
 */
int libra_attn_bwd(const void *q, const void *k, const void *v, const void *o, const float *lse,
                   const void *dout, const int64_t *cu_seqlens, int64_t num_samples,
                   const libra_tile_t *tiles, int64_t num_tiles, int64_t n_q_rows,
                   int64_t n_kv_rows, int32_t h_q, int32_t h_kv, int32_t head_dim,
                   float softmax_scale, void *dq, void *dk, void *dv, uint32_t flags,
                   void *workspace, size_t workspace_bytes, void *stream);

/*
 * Kernel timing (tracing aid).  libra_timing_enable(1) clears the records of
 * the calling thread and makes every later libra_attn_fwd / libra_attn_bwd
 * call on that thread record HIP events on its stream around its main
 * persistent kernels (the work-item kernels, not the small preparation
 * passes); libra_timing_enable(0) stops recording.  libra_timing_read waits
 * for the recorded events and returns the summed milliseconds and the number
 * of launches since the last enable of: which = 0, the forward kernel;
 * 1, the backward dK/dV kernel; 2, the backward dQ kernel.
 * Errors: EINVAL (bad `which`, NULL outputs), EHIP.
 */
int libra_timing_enable(int enable);
int libra_timing_read(int which, double *total_ms, int64_t *launches);

/*
 * Matrix-core reference loop (measurement aid): the bf16 MFMA throughput the
 * device sustains under load, reported beside the published dense peak.
 * libra_mfma_loop enqueues on `stream` one workgroup per compute unit, of
 * 4 waves (waves_per_simd = 1) or 8 (= 2, two waves on every SIMD); each wave
 * runs `iters` rounds of 4 independent v_mfma_f32_32x32x16_bf16 products
 * (32768 flops each) and does no other work.
 *   libra_mfma_loop_size: *record_words = uint64 words the record needs
 *       (3 per workgroup), *products_per_iter = products per round over the
 *       whole launch (flops of the launch = 32768 * iters * products_per_iter).
 *   record: device buffer of >= record_words uint64, owned by the caller;
 *       workgroup i writes record[3 i] = shader-clock cycles and
 *       record[3 i + 1] = 100 MHz wall-clock ticks of wave 0's loop (their
 *       ratio times 0.1 is the shader clock in GHz); record[3 i + 2] is not
 *       written.
 * The caller times the launch with events on the same stream.
 * Errors: EINVAL (waves_per_simd not 1 or 2, iters < 1, NULL pointers),
 * ENOSPC (record too small), EHIP.
 */
int libra_mfma_loop_size(int32_t waves_per_simd, int64_t *record_words,
                         int64_t *products_per_iter);
int libra_mfma_loop(int32_t waves_per_simd, int32_t iters, uint64_t *record,
                    int64_t record_words, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* LIBRA_H */
