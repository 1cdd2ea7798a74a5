/*
 * msa_evictor.h -- C ABI of the computation-aware KV block evictor (Sec. 4.2,
 * Alg. 1 of the AsymCache paper), the host-side control plane that decides
 * which cached blocks become the non-contiguous segments MSA recomputes.
 *
 * Policy.  A cached block B that no running request uses (reference count
 * zero) has a recomputation cost dT_B > 0 (Sec. 4.3, Eq. 5 / Eq. 7: it grows
 * with the block's position) and a frequency value (Sec. 4.4, Eq. 9)
 *
 *     f_B(t) = min( exp(-tau_B(t) / alpha), lambda * exp(-(tau_B(t) - tau0) / beta) )
 *
 * with tau_B(t) = t - t_last(B), the time since the block was last released
 * (reading of this library: the paper does not define tau_B(t) beyond "time
 * since access"; lambda is the online coefficient of Sec. 5.1, initially 1).
 * An eviction takes the block of least expected cost f_B(t) * dT_B (Eq. 3);
 * ties go to the smaller block id.
 *
 * Structure (Alg. 1).  Each exponential segment keeps the order of any two
 * blocks fixed over time (the order-preserving rule, Eq. 8; the paper's
 * appendix shows only exponentials do).  Each segment therefore keeps its
 * own ordered tree keyed by a time-invariant log weight:
 *     key1 = t_last / alpha + ln dT,   key2 = t_last / beta + ln dT
 * An eviction compares the two trees' minima at time t.  Every call is
 * O(log n).  With MSA_EVICTOR_LINEAR the same policy runs as an O(n) scan
 * (the linear-time baseline of Sec. 4.5).
 *
 * Times are in any consistent unit (e.g. seconds), costs in any positive unit.
 * The evictor is not thread-safe: serialise calls on one handle.
 */
#ifndef MSA_EVICTOR_H_
#define MSA_EVICTOR_H_

#include <stdint.h>

#include "msa.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct msa_evictor_s *msa_evictor_t;

/* Evaluate the policy by scanning every block (O(n) per eviction). */
#define MSA_EVICTOR_LINEAR 1

typedef struct msa_evictor_params {
  double alpha;  /* decay constant of the first segment, > 0 */
  double beta;   /* decay constant after the lifespan, > 0 */
  double tau0;   /* horizontal shift of the second segment */
  double lambda; /* initial online coefficient, > 0 (the paper starts at 1) */
  int32_t flags; /* MSA_EVICTOR_* bits */
  int32_t reserved[3]; /* must be zero */
} msa_evictor_params;

/* msa_evictor_create: an empty evictor.  MSA_ERR_INVALID_ARG for
 * non-positive or non-finite alpha, beta or lambda, non-finite tau0, unknown
 * flags or non-zero reserved fields. */
msa_status msa_evictor_create(const msa_evictor_params *params, msa_evictor_t *out);

/* msa_evictor_destroy: free the evictor (NULL accepted). */
void msa_evictor_destroy(msa_evictor_t ev);

/* msa_evictor_add (Alg. 1, ADD): block_id's reference count became zero at
 * time t_last; it is now evictable with recomputation cost `cost`.
 * MSA_ERR_INVALID_ARG if the id is already present, cost is not finite and
 * > 0, or t_last is not finite. */
msa_status msa_evictor_add(msa_evictor_t ev, int64_t block_id, double t_last, double cost);

/* msa_evictor_remove (Alg. 1, REMOVE): block_id was hit by a new request
 * and is no longer evictable.  MSA_ERR_INVALID_ARG if it is not present. */
msa_status msa_evictor_remove(msa_evictor_t ev, int64_t block_id);

/* msa_evictor_evict (Alg. 1, EVICT): remove and return in *block_id the block
 * of least expected cost at time t_now.  MSA_ERR_INVALID_ARG when empty or
 * t_now is not finite. */
msa_status msa_evictor_evict(msa_evictor_t ev, double t_now, int64_t *block_id);

/* msa_evictor_set_lambda: the online coefficient (Sec. 5.1), > 0. */
msa_status msa_evictor_set_lambda(msa_evictor_t ev, double lambda);

/* msa_evictor_set_lifespan: lambda <- exp((tau - tau0) / beta - tau / alpha)
 * (Eq. 10), which puts the turning point of f at the observed average
 * lifespan tau (>= 0, finite).  *lambda_out (may be NULL) receives lambda. */
msa_status msa_evictor_set_lifespan(msa_evictor_t ev, double tau, double *lambda_out);

/* msa_evictor_size: number of evictable blocks (0 for NULL). */
int64_t msa_evictor_size(msa_evictor_t ev);

/* msa_evictor_log_weight: ln(f_B(t) * dT_B) of a present block at time t.
 * MSA_ERR_INVALID_ARG if absent. */
msa_status msa_evictor_log_weight(msa_evictor_t ev, int64_t block_id, double t, double *out);

/* Operation codes of msa_evictor_replay. */
#define MSA_EVICTOR_OP_ADD 0      /* (id, t_last, cost) */
#define MSA_EVICTOR_OP_REMOVE 1   /* (id) */
#define MSA_EVICTOR_OP_EVICT 2    /* (t_now) -> evicted id */
#define MSA_EVICTOR_OP_LIFESPAN 3 /* (tau in t) */

/*
 * msa_evictor_replay: apply n operations in order (host arrays of n entries;
 * `id` is read for ADD / REMOVE, `t` for ADD / EVICT / LIFESPAN, `cost` for
 * ADD).  evicted[i] receives the id returned by an EVICT op (-1 for other
 * ops).  Stops at the first failing op: returns its status and writes its
 * index to *failed_at (may be NULL; -1 on success).  For driving traces
 * without per-call overhead.
 */
msa_status msa_evictor_replay(msa_evictor_t ev, int64_t n, const int32_t *op, const int64_t *id,
                              const double *t, const double *cost, int64_t *evicted,
                              int64_t *failed_at);

#ifdef __cplusplus
}
#endif

#endif /* MSA_EVICTOR_H_ */
