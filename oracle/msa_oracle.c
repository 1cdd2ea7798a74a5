/*
 * msa_oracle.c -- plain, slow CPU oracle for Multi-Segment Attention (MSA).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or helper with the GPU library; it parses its own inputs.
 *
 * What it computes (the plain definition, written out):
 *   Attention (Sec. 2.1, Eq. 1):  O = softmax(Q K^T / sqrt(d_k)) V, with the
 *   scale passed in as an argument.
 *   Multi-Segment Attention (Sec. 4.1, Eq. 2): the query tokens of one
 *   sequence sit in several disjoint position segments; the output is the
 *   concatenation, segment by segment, of attention of that segment's queries
 *   over the sequence's keys.  Read as causal by absolute position: the query
 *   at absolute position p sees exactly the keys at positions 0..p of its own
 *   sequence, whether they are resident cached blocks or freshly computed
 *   tokens of an earlier segment (Sec. 4.1: each thread gets an "equivalent
 *   seq_len" for its token from a precomputed array).
 *   Grouped-query attention (Sec. 2.1 names GQA): query head h reads K/V head
 *   h / (Hq / Hkv).
 *   The keys and values live in a paged cache addressed through a block table
 *   (Sec. 5.3: the kernel extends PagedAttention), block size bs:
 *     K of position j of sequence b, kv head g, channel c:
 *        k_cache[blk*ksb + g*ksh + (j%bs)*kst + c],   blk = block_table[b][j/bs]
 *     V (channel-major inside a block):
 *        v_cache[blk*vsb + g*vsh + c*vsd + (j%bs)]
 *
 *   The cache write before the attention (msa_oracle_kv_append): every packed
 *   row's fresh key and value go to the slot of its absolute position.
 *
 * Precision: inputs are bf16 bit patterns, widened exactly; every product,
 * sum, exponential and division is done in IEEE double, in the order the
 * definition is written (keys ascending, channels ascending).
 *
 * Packed query order: sequences in order; inside a sequence, segments in the
 * given (ascending, disjoint) order; inside a segment, ascending position.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define MSA_ORACLE_OK 0
#define MSA_ORACLE_BAD_ARG 1
#define MSA_ORACLE_NO_MEM 3

static double bf16_to_double(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

typedef struct {
  /* problem */
  int32_t num_q_heads, num_kv_heads, head_dim, block_size, max_blocks_per_seq;
  double scale;
  const uint16_t *q;
  int64_t qst, qsh;
  const uint16_t *k;
  int64_t ksb, ksh, kst;
  const uint16_t *v;
  int64_t vsb, vsh, vsd;
  const int32_t *block_table;
  /* row -> (sequence, absolute position), built by walking the segments */
  const int32_t *row_seq;
  const int32_t *row_pos;
  /* work list */
  const int64_t *item_row;  /* NULL: item i is (row i / Hq, head i % Hq) */
  const int32_t *item_head;
  int64_t n_items;
  int32_t max_pos;
  double *out_o;   /* [n_items][head_dim] */
  double *out_lse; /* [n_items] */
  /* threading */
  int32_t num_threads, tid;
  int32_t failed;
} job_t;

/* One (query row, query head): the definition, term by term. */
static void one_row(const job_t *J, int64_t row, int32_t h, double *s, double *o,
                    double *lse) {
  const int32_t d = J->head_dim, bs = J->block_size;
  const int32_t b = J->row_seq[row], p = J->row_pos[row];
  const int32_t g = h / (J->num_q_heads / J->num_kv_heads);
  const uint16_t *qv = J->q + row * J->qst + (int64_t)h * J->qsh;
  const int32_t *bt = J->block_table + (int64_t)b * J->max_blocks_per_seq;

  /* scores s_j = scale * <q, k_j> for every visible key j = 0..p */
  double m = -INFINITY;
  for (int32_t j = 0; j <= p; ++j) {
    const int64_t blk = bt[j / bs];
    const uint16_t *kv = J->k + blk * J->ksb + (int64_t)g * J->ksh + (int64_t)(j % bs) * J->kst;
    double dot = 0.0;
    for (int32_t c = 0; c < d; ++c) dot += bf16_to_double(qv[c]) * bf16_to_double(kv[c]);
    s[j] = J->scale * dot;
    if (s[j] > m) m = s[j];
  }
  /* softmax weights w_j = exp(s_j - m), l = sum_j w_j, o = sum_j w_j v_j / l */
  double l = 0.0;
  for (int32_t c = 0; c < d; ++c) o[c] = 0.0;
  for (int32_t j = 0; j <= p; ++j) {
    const double w = exp(s[j] - m);
    l += w;
    const int64_t blk = bt[j / bs];
    const uint16_t *vv = J->v + blk * J->vsb + (int64_t)g * J->vsh + (j % bs);
    for (int32_t c = 0; c < d; ++c) o[c] += w * bf16_to_double(vv[(int64_t)c * J->vsd]);
  }
  for (int32_t c = 0; c < d; ++c) o[c] /= l;
  *lse = m + log(l);
}

static void *worker(void *arg) {
  job_t *J = (job_t *)arg;
  double *s = (double *)malloc(sizeof(double) * ((size_t)J->max_pos + 1));
  if (!s) {
    J->failed = 1;
    return NULL;
  }
  /* static, interleaved split of the items: results do not depend on it */
  for (int64_t i = J->tid; i < J->n_items; i += J->num_threads) {
    int64_t row;
    int32_t h;
    if (J->item_row) {
      row = J->item_row[i];
      h = J->item_head[i];
    } else {
      row = i / J->num_q_heads;
      h = (int32_t)(i % J->num_q_heads);
    }
    one_row(J, row, h, s, J->out_o + i * J->head_dim, J->out_lse + i);
  }
  free(s);
  return NULL;
}

/*
 * msa_oracle_total_rows: number of packed query rows (sum of segment
 * lengths), or -1 if the descriptors are malformed.
 */
int64_t msa_oracle_total_rows(int32_t num_seqs, const int32_t *seg_indptr,
                              const int32_t *seg_len) {
  int64_t t = 0;
  for (int32_t b = 0; b < num_seqs; ++b)
    for (int32_t s = seg_indptr[b]; s < seg_indptr[b + 1]; ++s) {
      if (seg_len[s] < 0) return -1;
      t += seg_len[s];
    }
  return t;
}

/*
 * msa_oracle_forward: exact MSA for a list of (row, head) items.
 *
 * item_row / item_head == NULL computes every row and head; then item i is
 * (row i / Hq, head i % Hq) and out_o is [total_rows][Hq][d], out_lse is
 * [total_rows][Hq].  Otherwise out_o is [n_items][d] and out_lse [n_items].
 * Strides are in elements.  Returns 0, or a nonzero code for inputs that
 * break the definition's preconditions (nothing is then written).
 */
int msa_oracle_forward(int32_t num_seqs, int32_t num_q_heads, int32_t num_kv_heads,
                       int32_t head_dim, int32_t block_size, int32_t max_blocks_per_seq,
                       int32_t num_blocks, double scale, const int32_t *seq_kv_len,
                       const int32_t *seg_indptr, const int32_t *seg_start,
                       const int32_t *seg_len, const uint16_t *q, int64_t q_stride_tok,
                       int64_t q_stride_head, const uint16_t *k_cache, int64_t k_stride_block,
                       int64_t k_stride_head, int64_t k_stride_tok, const uint16_t *v_cache,
                       int64_t v_stride_block, int64_t v_stride_head, int64_t v_stride_dim,
                       const int32_t *block_table, const int64_t *item_row,
                       const int32_t *item_head, int64_t n_items, double *out_o,
                       double *out_lse, int32_t num_threads) {
  if (num_seqs < 0 || num_q_heads <= 0 || num_kv_heads <= 0 ||
      num_q_heads % num_kv_heads != 0 || head_dim <= 0 || block_size <= 0)
    return MSA_ORACLE_BAD_ARG;
  const int64_t total = msa_oracle_total_rows(num_seqs, seg_indptr, seg_len);
  if (total < 0) return MSA_ORACLE_BAD_ARG;

  int32_t *row_seq = (int32_t *)malloc(sizeof(int32_t) * (size_t)(total + 1));
  int32_t *row_pos = (int32_t *)malloc(sizeof(int32_t) * (size_t)(total + 1));
  if (!row_seq || !row_pos) {
    free(row_seq);
    free(row_pos);
    return MSA_ORACLE_NO_MEM;
  }
  /* walk the segments: packed row r <-> (sequence, absolute position) */
  int64_t r = 0;
  int32_t max_pos = 0;
  int bad = 0;
  for (int32_t b = 0; b < num_seqs && !bad; ++b) {
    int32_t prev_end = 0;
    for (int32_t s = seg_indptr[b]; s < seg_indptr[b + 1]; ++s) {
      if (seg_len[s] < 1 || seg_start[s] < prev_end ||
          (int64_t)seg_start[s] + seg_len[s] > seq_kv_len[b] ||
          (int64_t)seq_kv_len[b] > (int64_t)max_blocks_per_seq * block_size) {
        bad = 1;
        break;
      }
      for (int32_t t = 0; t < seg_len[s]; ++t) {
        row_seq[r] = b;
        row_pos[r] = seg_start[s] + t;
        if (row_pos[r] > max_pos) max_pos = row_pos[r];
        ++r;
      }
      prev_end = seg_start[s] + seg_len[s];
    }
  }
  /* every block the definition reads must exist */
  for (int64_t i = 0; i < total && !bad; ++i) {
    const int32_t *bt = block_table + (int64_t)row_seq[i] * max_blocks_per_seq;
    for (int32_t jb = 0; jb <= row_pos[i] / block_size; ++jb)
      if (bt[jb] < 0 || bt[jb] >= num_blocks) {
        bad = 1;
        break;
      }
  }
  if (item_row) {
    for (int64_t i = 0; i < n_items && !bad; ++i)
      if (item_row[i] < 0 || item_row[i] >= total || item_head[i] < 0 ||
          item_head[i] >= num_q_heads)
        bad = 1;
  } else {
    n_items = total * num_q_heads;
  }
  if (bad) {
    free(row_seq);
    free(row_pos);
    return MSA_ORACLE_BAD_ARG;
  }

  if (num_threads < 1) num_threads = 1;
  if (n_items < num_threads) num_threads = n_items > 0 ? (int32_t)n_items : 1;
  job_t *jobs = (job_t *)calloc((size_t)num_threads, sizeof(job_t));
  pthread_t *th = (pthread_t *)calloc((size_t)num_threads, sizeof(pthread_t));
  if (!jobs || !th) {
    free(jobs);
    free(th);
    free(row_seq);
    free(row_pos);
    return MSA_ORACLE_NO_MEM;
  }
  for (int32_t t = 0; t < num_threads; ++t) {
    job_t *J = &jobs[t];
    J->num_q_heads = num_q_heads;
    J->num_kv_heads = num_kv_heads;
    J->head_dim = head_dim;
    J->block_size = block_size;
    J->max_blocks_per_seq = max_blocks_per_seq;
    J->scale = scale;
    J->q = q;
    J->qst = q_stride_tok;
    J->qsh = q_stride_head;
    J->k = k_cache;
    J->ksb = k_stride_block;
    J->ksh = k_stride_head;
    J->kst = k_stride_tok;
    J->v = v_cache;
    J->vsb = v_stride_block;
    J->vsh = v_stride_head;
    J->vsd = v_stride_dim;
    J->block_table = block_table;
    J->row_seq = row_seq;
    J->row_pos = row_pos;
    J->item_row = item_row;
    J->item_head = item_head;
    J->n_items = n_items;
    J->max_pos = max_pos;
    J->out_o = out_o;
    J->out_lse = out_lse;
    J->num_threads = num_threads;
    J->tid = t;
  }
  int failed = 0;
  if (num_threads == 1) {
    worker(&jobs[0]);
  } else {
    int32_t started = 0;
    for (; started < num_threads; ++started)
      if (pthread_create(&th[started], NULL, worker, &jobs[started]) != 0) break;
    /* threads that could not start run inline, same items, same results */
    for (int32_t t = started; t < num_threads; ++t) worker(&jobs[t]);
    for (int32_t t = 0; t < started; ++t) pthread_join(th[t], NULL);
  }
  for (int32_t t = 0; t < num_threads; ++t) failed |= jobs[t].failed;
  free(jobs);
  free(th);
  free(row_seq);
  free(row_pos);
  return failed ? MSA_ORACLE_NO_MEM : MSA_ORACLE_OK;
}

/*
 * msa_oracle_kv_append: the cache write that precedes attention.  All
 * segments' tokens go through one forward pass (Sec. 4.1), which yields the
 * key and value of every packed row; each is stored in the paged cache
 * (Sec. 5.3, PagedAttention's block table) at the row's absolute position:
 *   K[blk, g, p % bs, c] = k_new[r, g, c],  V[blk, g, c, p % bs] = v_new[r, g, c]
 *   for every kv head g and channel c, blk = block_table[b][p / bs].
 * A row whose block-table entry is outside [0, num_blocks) has no slot and
 * writes nothing.  Rows are written in packed order.  Returns 0, or a nonzero
 * code (nothing written) when the segments break the layout's rules.
 */
int msa_oracle_kv_append(int32_t num_seqs, int32_t num_kv_heads, int32_t head_dim,
                         int32_t block_size, int32_t max_blocks_per_seq, int32_t num_blocks,
                         const int32_t *seq_kv_len, const int32_t *seg_indptr,
                         const int32_t *seg_start, const int32_t *seg_len,
                         const uint16_t *k_new, int64_t kn_stride_tok, int64_t kn_stride_head,
                         const uint16_t *v_new, int64_t vn_stride_tok, int64_t vn_stride_head,
                         uint16_t *k_cache, int64_t k_stride_block, int64_t k_stride_head,
                         int64_t k_stride_tok, uint16_t *v_cache, int64_t v_stride_block,
                         int64_t v_stride_head, int64_t v_stride_dim,
                         const int32_t *block_table) {
  if (num_seqs < 0 || num_kv_heads <= 0 || head_dim <= 0 || block_size <= 0)
    return MSA_ORACLE_BAD_ARG;
  /* the same segment rules as the attention */
  for (int32_t b = 0; b < num_seqs; ++b) {
    int32_t prev_end = 0;
    for (int32_t s = seg_indptr[b]; s < seg_indptr[b + 1]; ++s) {
      if (seg_len[s] < 1 || seg_start[s] < prev_end ||
          (int64_t)seg_start[s] + seg_len[s] > seq_kv_len[b] ||
          (int64_t)seq_kv_len[b] > (int64_t)max_blocks_per_seq * block_size)
        return MSA_ORACLE_BAD_ARG;
      prev_end = seg_start[s] + seg_len[s];
    }
  }
  int64_t r = 0;
  for (int32_t b = 0; b < num_seqs; ++b)
    for (int32_t s = seg_indptr[b]; s < seg_indptr[b + 1]; ++s)
      for (int32_t t = 0; t < seg_len[s]; ++t, ++r) {
        const int32_t p = seg_start[s] + t;
        const int32_t blk = block_table[(int64_t)b * max_blocks_per_seq + p / block_size];
        if (blk < 0 || blk >= num_blocks) continue;
        const int32_t off = p % block_size;
        for (int32_t g = 0; g < num_kv_heads; ++g)
          for (int32_t c = 0; c < head_dim; ++c) {
            k_cache[blk * k_stride_block + g * k_stride_head + off * k_stride_tok + c] =
                k_new[r * kn_stride_tok + g * kn_stride_head + c];
            v_cache[blk * v_stride_block + g * v_stride_head + c * v_stride_dim + off] =
                v_new[r * vn_stride_tok + g * vn_stride_head + c];
          }
      }
  return MSA_ORACLE_OK;
}
