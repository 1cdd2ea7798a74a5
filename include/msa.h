/*
 * msa.h -- C ABI of the Multi-Segment Attention (MSA) library for AMD
 * Instinct MI355X (gfx950).
 *
 * The operation (Sec. 4.1, Eq. 2 of the AsymCache paper, built on attention
 * as in Sec. 2.1, Eq. 1): the query tokens of each sequence sit in one or
 * more disjoint position segments -- recomputed evicted blocks, a new prompt
 * chunk, a decode token.  Their hidden states are concatenated and only the
 * attention needs the split indices (Sec. 4.1).  Each query at absolute
 * position p attends to exactly the keys at positions 0..p of its own
 * sequence (the "equivalent seq_len" of its token, Sec. 4.1), resident or
 * freshly written, read from a paged K/V cache through a block table (the
 * kernel extends PagedAttention, Sec. 5.3).  Query head h reads K/V head
 * h / (Hq / Hkv) (grouped-query attention, Sec. 2.1).
 *
 *   o[r, h, :] = sum_{j <= p_r} softmax_j(scale * <q[r, h], k_j>) * v_j
 *   lse[r, h]  = log sum_{j <= p_r} exp(scale * <q[r, h], k_j>)      (natural log)
 *
 * All segments of all sequences run in one plan and one kernel launch (the
 * paper's single fused launch, Sec. 4.1); long contexts may be split along
 * the keys and merged by log-sum-exp (an addition of this library, not in
 * the paper).
 *
 * Conventions
 *  - Element type: bfloat16 for q, k_cache, v_cache and o; float32 for lse.
 *  - Packed query order ("rows"): sequences in order; inside a sequence,
 *    segments in ascending position; inside a segment, ascending position.
 *    Output row r corresponds to input row r.  total_q = sum of seg_len.
 *  - q[r, h, c]   at q + r*q_stride_tok + h*q_stride_head + c
 *    o[r, h, c]   at o + r*o_stride_tok + h*o_stride_head + c
 *    lse[r, h]    at lse + r*num_q_heads + h              (contiguous)
 *    K of position j of sequence b, kv head g, channel c (token-major block):
 *        k_cache + blk*k_stride_block + g*k_stride_head + (j%bs)*k_stride_tok + c
 *    V (channel-major block: the 16 tokens of one channel are contiguous,
 *    the layout of vLLM's paged-attention V cache):
 *        v_cache + blk*v_stride_block + g*v_stride_head + c*v_stride_dim + (j%bs)
 *    where blk = block_table[b*max_blocks_per_seq + j/bs].
 *    Strides are in elements and must be multiples of 8 (16-byte vectors);
 *    all device pointers must be 16-byte aligned.
 *  - Ownership: the caller owns every tensor, the block table and the
 *    workspace.  A plan owns a small device buffer (allocated by msa_plan,
 *    uploaded asynchronously on the given stream) and its host copy; it is
 *    immutable, serves every layer of one batch step, and msa_forward may be
 *    called with it concurrently on different streams provided each call has
 *    its own workspace and output.
 *  - Errors: every function returns a status; MSA_OK is 0.  On
 *    MSA_ERR_INVALID_ARG, MSA_ERR_UNSUPPORTED and MSA_ERR_OUT_OF_MEMORY
 *    nothing was launched and no output was written.  MSA_ERR_DEVICE means
 *    a HIP call or launch failed: work enqueued before it in the same call
 *    (msa_forward's attention launch, when its merge launch fails) may have
 *    written part of the output.  msa_last_error() then returns a
 *    thread-local message.
 *  - Preconditions not checked on the hot path: the K/V of every query
 *    position are already in the cache; block_table[b][i] is a valid
 *    physical block for every i < ceil((max query position of b + 1) / bs);
 *    other block-table entries are never read; cache values at positions
 *    >= seq_kv_len[b] inside a referenced block are finite.  An entry outside
 *    [0, num_blocks) makes the kernels read outside the caches;
 *    msa_check_block_table validates a table against a plan (debug use).
 */
#ifndef MSA_H_
#define MSA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum msa_status {
  MSA_OK = 0,
  MSA_ERR_INVALID_ARG = 1,   /* malformed shapes, segments, pointers, sizes */
  MSA_ERR_UNSUPPORTED = 2,   /* valid but not built: head_dim, block size, ... */
  MSA_ERR_OUT_OF_MEMORY = 3, /* host or device allocation failed */
  MSA_ERR_DEVICE = 4         /* a HIP runtime call or kernel launch failed */
} msa_status;

/* Opaque plan handle (library-owned). */
typedef struct msa_plan_s *msa_plan_t;

/* Problem shape and tensor layout shared by every layer of a batch step. */
typedef struct msa_shape {
  int32_t num_seqs;           /* B >= 0 */
  int32_t num_q_heads;        /* Hq >= 1 */
  int32_t num_kv_heads;       /* Hkv >= 1, Hq % Hkv == 0, Hq / Hkv <= 256 */
  int32_t head_dim;           /* d: 64 or 128 */
  int32_t block_size;         /* bs: 16 */
  int32_t max_blocks_per_seq; /* row stride of block_table (entries) */
  int32_t num_blocks;         /* physical blocks in each cache */
  float scale;                /* softmax scale > 0, 1/sqrt(d) in the paper's Eq. 1 */
  int64_t q_stride_tok, q_stride_head;                 /* channel stride is 1 */
  int64_t o_stride_tok, o_stride_head;                 /* channel stride is 1 */
  int64_t k_stride_block, k_stride_head, k_stride_tok; /* channel stride is 1 */
  int64_t v_stride_block, v_stride_head, v_stride_dim; /* token stride is 1 */
} msa_shape;

/* Planner options; a zero field means "choose automatically". */
typedef struct msa_plan_opts {
  int32_t q_tile_tokens;   /* cap on query tokens per tile (<= tile rows / (Hq/Hkv)) */
  int32_t kv_split_tokens; /* force key splits of this many keys (multiple of 64) */
  int32_t flags;           /* MSA_PLAN_* bits */
  int32_t reserved[5];     /* must be zero */
} msa_plan_opts;

/* Build the plan on the host only: no device memory, no upload.  Such a plan
 * can be inspected (msa_plan_info, msa_plan_export) but not executed. */
#define MSA_PLAN_HOST_ONLY 1
/* Disable the cost-based automatic key splitting (forced splits still apply). */
#define MSA_PLAN_NO_AUTO_SPLIT 2
/* Force the tile width (query rows x heads per workgroup).  Without a flag
 * the planner takes:
 *   - 32-row tiles when no 128-row tile would hold more than 32 rows
 *     (decode-like plans: the four waves of a workgroup split the tile's
 *     keys and read K and V straight into registers, two workgroups per CU);
 *   - 256-row tiles (one workgroup per CU; each K/V step is loaded once for
 *     twice the rows) when the plan has many tiles and a long run of key
 *     steps per workgroup slot;
 *   - else 128-row tiles (two workgroups per CU: one's start-up and tail
 *     overlap the other's work).
 * The flags are exclusive.  32-row tiles need Hq / Hkv <= 32, 128-row tiles
 * Hq / Hkv <= 128 (else MSA_ERR_UNSUPPORTED). */
#define MSA_PLAN_TILE_ROWS_128 4
#define MSA_PLAN_TILE_ROWS_256 8
#define MSA_PLAN_TILE_ROWS_32 16
/* Carry every softmax weight into the P.V product as two bf16 terms,
 * hi = bf16(w) and lo = bf16(w - hi), as the default path does only on the
 * key step that holds each row's own position.  By default the weights of
 * earlier keys enter as bf16 numbers (each moved by up to 2^-8 of itself):
 * on inputs whose scores make a few keys carry a row's weight, this moves
 * the output by up to 2^-8 * sum_j p_j |v_j| (p_j the normalised weights)
 * before its own bf16 rounding.  With this flag the weights hold to about
 * 2^-17, at the cost of a second P.V product on every step and no
 * software pipelining: 1.3 to 1.5 times the time of a call on plans with
 * prefill rows, about the same on decode-like plans (bound by streaming
 * K/V).  The plan is otherwise the same. */
#define MSA_PLAN_PRECISE_WEIGHTS 32

/* Figures describing a plan. */
typedef struct msa_plan_info_t {
  int64_t total_q;          /* packed query rows */
  int64_t num_work;         /* attention work items (tiles x key ranges) */
  int64_t num_tiles;        /* query tiles x kv heads before key splitting */
  int64_t num_merge;        /* tiles whose keys were split (merge work items) */
  int64_t max_splits;       /* largest number of key splits of one tile */
  int64_t workspace_bytes;  /* bytes msa_forward needs in its workspace (may be 0) */
  double useful_flops;      /* 4 * d * Hq * sum_rows (p + 1): QK^T and PV, visible pairs */
  double tile_flops;        /* flops the tiles issue (waves holding rows), incl. masked waste */
  double planned_bytes;     /* Q + O + K/V bytes the executed tiles request */
  double min_bytes;         /* Q + O + K/V of visible keys once per (seq, kv head) */
  int64_t tile_rows;        /* rows per tile of this plan: 32, 128 or 256 */
  int64_t num_workgroups;   /* workgroups launched; each runs its own list of work items */
} msa_plan_info_t;

/*
 * msa_plan: validate the segment descriptors and build the work list.
 *
 * The paper runs the attention of all segments of all requests in one
 * kernel, handing it the segments' split indices; each query token finds its
 * "equivalent seq_len" (its causal limit) in a precomputed per-token array
 * (Sec. 4.1, Eq. 2).  msa_plan builds both once per batch step: the split
 * indices are seg_indptr / seg_start / seg_len, the per-token array is the
 * plan's row-position table (msa_plan_export), and the work list maps tiles
 * of query rows x KV heads x key ranges onto workgroups.
 *
 *   shape       problem shape and strides (host pointer, read during the call)
 *   seq_kv_len  [num_seqs] host: context length of each sequence, 0 <= L <=
 *               max_blocks_per_seq * block_size
 *   seg_indptr  [num_seqs + 1] host: segments of sequence b are
 *               seg_indptr[b] .. seg_indptr[b+1]-1; seg_indptr[0] == 0
 *   seg_start, seg_len  [seg_indptr[num_seqs]] host: segment = positions
 *               [start, start + len); len >= 1; sorted, disjoint (adjacent
 *               allowed) and inside [0, L) per sequence.  A sequence may
 *               have no segments.
 *   opts        may be NULL (all automatic)
 *   hip_stream  hipStream_t on which the plan's device buffer is uploaded
 *               (ignored with MSA_PLAN_HOST_ONLY); msa_forward calls on other
 *               streams must be ordered after this upload by the caller
 *   out         receives the plan; destroy with msa_plan_destroy
 *
 * Returns MSA_ERR_INVALID_ARG for malformed descriptors or shapes,
 * MSA_ERR_UNSUPPORTED for head_dim not in {64, 128}, block_size != 16,
 * Hq / Hkv > 256, Hq / Hkv > 128 with MSA_PLAN_TILE_ROWS_128, or Hq / Hkv > 32
 * with MSA_PLAN_TILE_ROWS_32;
 * MSA_ERR_OUT_OF_MEMORY; MSA_ERR_DEVICE.
 */
msa_status msa_plan(const msa_shape *shape, const int32_t *seq_kv_len, const int32_t *seg_indptr,
                    const int32_t *seg_start, const int32_t *seg_len, const msa_plan_opts *opts,
                    void *hip_stream, msa_plan_t *out);

/* msa_plan_info: figures of a plan (see msa_plan_info_t). */
msa_status msa_plan_info(msa_plan_t plan, msa_plan_info_t *info);

/*
 * msa_forward: run MSA for one layer: the attention of every packed query
 * row over the keys at positions 0..p of its sequence (Sec. 4.1, Eq. 2, on
 * attention as in Sec. 2.1, Eq. 1), read from the paged cache through the
 * block table (the kernel extends PagedAttention, Sec. 5.3), as one fused
 * launch for all segments (plus a log-sum-exp merge launch when the plan
 * split long key ranges).
 *
 *   q            device bf16 [total_q, Hq, d] (strided as in the shape)
 *   k_cache      device bf16, token-major blocks (see conventions)
 *   v_cache      device bf16, channel-major blocks
 *   block_table  device int32 [num_seqs * max_blocks_per_seq]
 *   o            device bf16 [total_q, Hq, d] output (strided)
 *   lse          device float32 [total_q, Hq] output, or NULL
 *   workspace    device buffer of at least msa_plan_info().workspace_bytes
 *                bytes (may be NULL when that is 0); contents need no
 *                initialisation and are clobbered
 *   hip_stream   hipStream_t on which all kernels are enqueued (no host sync)
 *
 * Returns MSA_ERR_INVALID_ARG for NULL or misaligned pointers, a too-small
 * workspace or a host-only plan; MSA_ERR_DEVICE if a launch fails (if the
 * merge launch fails, the attention launch before it may have written part
 * of o and lse).  The block table is not checked (see msa_check_block_table).
 */
msa_status msa_forward(msa_plan_t plan, const void *q, const void *k_cache, const void *v_cache,
                       const int32_t *block_table, void *o, float *lse, void *workspace,
                       size_t workspace_bytes, void *hip_stream);

/*
 * msa_forward_noalloc: msa_forward for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the workspace is a scratch array of
 * MSA_NOALLOC_WORKSPACE_BYTES inside the library, one per device, held
 * until the process ends.  The call allocates and frees nothing.  Arguments
 * and results are those of msa_forward without the workspace; the outputs
 * are bit-identical to msa_forward's.
 *
 * Every call on a device shares that device's array and leaves it holding
 * its partial results: calls that may overlap on one device (other streams,
 * other threads) race and must be ordered by the caller.  The first call on
 * each device looks the array's device address up (hipGetSymbolAddress,
 * with that device current) and keeps it; make that first call before
 * capturing a graph.
 *
 * Returns MSA_ERR_UNSUPPORTED, launching nothing, when the plan's workspace
 * (msa_plan_info().workspace_bytes) exceeds MSA_NOALLOC_WORKSPACE_BYTES;
 * otherwise the statuses of msa_forward.
 */
#define MSA_NOALLOC_WORKSPACE_BYTES (64ull << 20)
msa_status msa_forward_noalloc(msa_plan_t plan, const void *q, const void *k_cache,
                               const void *v_cache, const int32_t *block_table, void *o, float *lse,
                               void *hip_stream);

/*
 * msa_kv_append: write the fresh keys and values of every packed query row
 * into the paged cache, at the row's absolute position.  All segments'
 * tokens go through one forward pass (Sec. 4.1), so each layer produces K/V
 * for every packed row; they must sit in the PagedAttention-style cache
 * (Sec. 5.3) before msa_forward reads them (K/V of earlier segments are
 * keys of later ones).  Same plan, same row order as msa_forward.
 *
 *   k_new, v_new  device bf16 [total_q, Hkv, d]: element (r, g, c) at
 *                 k_new + r*k_new_stride_tok + g*k_new_stride_head + c
 *                 (likewise v_new with its own strides; channel stride 1;
 *                 strides in elements, positive multiples of 8)
 *   block_table   device int32 [num_seqs * max_blocks_per_seq]
 *   k_cache, v_cache  device caches in the layout of the conventions above
 *   hip_stream    hipStream_t on which the kernel is enqueued (no host sync)
 *
 * Row r (sequence b, position p) writes K[blk, g, p % 16, :] and
 * V[blk, g, :, p % 16] for every kv head g, blk = block_table[b][p / 16].
 * Nothing else in the caches is written.  A row whose block-table entry is
 * outside [0, num_blocks) is skipped (not written).  No two rows may map to
 * the same cache slot (e.g. through physical blocks shared by sequences):
 * such writes race.  The new K/V must not overlap the caches.
 *
 * Returns MSA_ERR_INVALID_ARG for NULL or misaligned pointers, bad strides
 * or a host-only plan; MSA_ERR_DEVICE if the launch fails.  A plan with no
 * rows returns MSA_OK and launches nothing.
 */
msa_status msa_kv_append(msa_plan_t plan, const void *k_new, const void *v_new,
                         int64_t k_new_stride_tok, int64_t k_new_stride_head,
                         int64_t v_new_stride_tok, int64_t v_new_stride_head,
                         const int32_t *block_table, void *k_cache, void *v_cache,
                         void *hip_stream);

/*
 * msa_check_block_table: debug-only validation of a block table against a
 * plan, before msa_forward or msa_kv_append use it.  The paged cache of
 * PagedAttention (Sec. 5.3) maps each sequence's logical blocks to physical
 * ones; the kernels trust that mapping, and an entry outside [0, num_blocks)
 * makes them read (or, for msa_forward, fault) outside the caches.
 *
 * Reads exactly the entries the plan's kernels read: for sequence b,
 * logical blocks 0 .. ceil((P_b + 1) / block_size) - 1, where P_b is the
 * largest query position of b (no entry if b has no query rows).
 *
 *   block_table  [num_seqs * max_blocks_per_seq] int32, row stride
 *                max_blocks_per_seq (host or device memory, per location)
 *   location     MSA_TABLE_HOST: a host pointer, read directly;
 *                MSA_TABLE_DEVICE: a device pointer; the entries are copied
 *                to the host on hip_stream, which is then synchronised (the
 *                copy is ordered after earlier work on that stream)
 *   hip_stream   hipStream_t for the copy (ignored for host tables)
 *
 * Works on host-only plans too.  Returns MSA_OK when every entry read lies
 * in [0, num_blocks); MSA_ERR_INVALID_ARG for the first entry that does not,
 * in sequence order then logical-block order, with msa_last_error() naming
 * the sequence, the logical block and the value; MSA_ERR_INVALID_ARG for a
 * NULL or misaligned table or a bad location; MSA_ERR_DEVICE if the copy
 * fails; MSA_ERR_OUT_OF_MEMORY.  Nothing is written.
 */
#define MSA_TABLE_HOST 0
#define MSA_TABLE_DEVICE 1
msa_status msa_check_block_table(msa_plan_t plan, const int32_t *block_table, int32_t location,
                                 void *hip_stream);

/* msa_plan_destroy: free a plan.  The caller must have synchronised every
 * stream that used it.  NULL is accepted. */
void msa_plan_destroy(msa_plan_t plan);

/* msa_last_error: thread-local text describing the last non-OK status
 * returned on this thread ("" if none).  Valid until the next call. */
const char *msa_last_error(void);

/*
 * msa_plan_export: host copies of a plan's device tables, for testing and
 * inspection.  Any output pointer may be NULL.
 *   row_pos  [total_q] int32: absolute position of each packed row
 *   work     [num_work * 8] int32: per work item {seq, kv_head, row0, nrows,
 *            kv_lo, kv_hi, out_slot, wg}; rows row0 .. row0+nrows-1 of
 *            sequence seq, keys [kv_lo, kv_hi); out_slot -1 writes the final
 *            output, else the workspace slot of a partial result; wg is the
 *            workgroup that runs it (items of one workgroup are adjacent, in
 *            run order, workgroups ascending; workgroup i runs on XCD i % 8)
 *   merge    [num_merge * 8] int32: per split tile {seq, kv_head, row0, nrows,
 *            nsplit, slot0, 0, 0}: slots slot0 .. slot0+nsplit-1 in key order
 */
msa_status msa_plan_export(msa_plan_t plan, int32_t *row_pos, int32_t *work, int32_t *merge);

#ifdef __cplusplus
}
#endif

#endif /* MSA_H_ */
