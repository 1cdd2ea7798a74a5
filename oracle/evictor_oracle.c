/*
 * evictor_oracle.c -- plain, slow CPU oracle of the computation-aware block
 * evictor.  TEST INFRASTRUCTURE ONLY (same rules as msa_oracle.c: only the
 * tests, the smoke check and the benchmark's CPU-baseline leg load it; it
 * shares nothing with the library).
 *
 * The definition, evaluated from scratch at every eviction:
 *   Eq. 3: evict the block B that minimises f_B(t) * dT_B;
 *   Eq. 9: f_B(t) = min(exp(-tau / alpha), exp(-(tau - tau0) / beta)),
 *          tau = t - (time B was last released);
 *   Alg. 1: the second segment is scaled by the online coefficient lambda
 *          (initially given), i.e. the weight is min(w1, lambda * w2);
 *   Eq. 10: a lifespan update tau sets lambda = exp((tau - tau0)/beta - tau/alpha).
 * The minimum is taken over ln(weight) = min(-tau/alpha, ln lambda -
 * (tau - tau0)/beta) + ln dT, which orders blocks exactly as the weight does
 * (the logarithm is increasing) but cannot underflow.  Ties go to the
 * smaller block id.  Every block is kept in a plain array and scanned.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#define OP_ADD 0
#define OP_REMOVE 1
#define OP_EVICT 2
#define OP_LIFESPAN 3

typedef struct {
  int64_t id;
  double t_last, cost;
} oracle_block_t;

static int64_t find(const oracle_block_t *b, int64_t n, int64_t id) {
  for (int64_t i = 0; i < n; ++i)
    if (b[i].id == id) return i;
  return -1;
}

/*
 * msa_oracle_evictor_replay: apply n_ops operations (codes above; the same
 * argument arrays as the library's replay) and write the id of each evicted
 * block to evicted[i] (-1 for other ops).  Returns 0, or 1 + the index of the
 * first operation that the definition cannot apply (adding a present block,
 * removing an absent one, evicting from an empty set, a non-positive cost),
 * or -1 when out of memory.
 */
int64_t msa_oracle_evictor_replay(double alpha, double beta, double tau0, double lambda,
                                  int64_t n_ops, const int32_t *op, const int64_t *id,
                                  const double *t, const double *cost, int64_t *evicted) {
  oracle_block_t *b = NULL;
  int64_t n = 0, cap = 0;
  double log_lambda = log(lambda);
  int64_t rc = 0;
  for (int64_t i = 0; i < n_ops && rc == 0; ++i) {
    evicted[i] = -1;
    if (op[i] == OP_ADD) {
      if (!(cost[i] > 0) || find(b, n, id[i]) >= 0) {
        rc = i + 1;
        break;
      }
      if (n == cap) {
        cap = cap ? 2 * cap : 64;
        oracle_block_t *nb = (oracle_block_t *)realloc(b, (size_t)cap * sizeof *b);
        if (!nb) {
          rc = -1;
          break;
        }
        b = nb;
      }
      b[n].id = id[i];
      b[n].t_last = t[i];
      b[n].cost = cost[i];
      ++n;
    } else if (op[i] == OP_REMOVE) {
      const int64_t k = find(b, n, id[i]);
      if (k < 0) {
        rc = i + 1;
        break;
      }
      b[k] = b[n - 1];
      --n;
    } else if (op[i] == OP_EVICT) {
      if (n == 0) {
        rc = i + 1;
        break;
      }
      int64_t best = -1;
      double best_w = 0;
      for (int64_t k = 0; k < n; ++k) {
        const double tau = t[i] - b[k].t_last;
        const double seg1 = -tau / alpha;
        const double seg2 = log_lambda - (tau - tau0) / beta;
        const double w = (seg1 < seg2 ? seg1 : seg2) + log(b[k].cost);
        if (best < 0 || w < best_w || (w == best_w && b[k].id < b[best].id)) {
          best = k;
          best_w = w;
        }
      }
      evicted[i] = b[best].id;
      b[best] = b[n - 1];
      --n;
    } else if (op[i] == OP_LIFESPAN) {
      log_lambda = (t[i] - tau0) / beta - t[i] / alpha;
    } else {
      rc = i + 1;
    }
  }
  free(b);
  return rc;
}
