// evictor.cpp -- the computation-aware block evictor declared in
// include/msa_evictor.h (Sec. 4.2, Alg. 1).
//
// Each evictable block carries two time-invariant log weights.  At time t the
// two segments of the frequency function (Sec. 4.4) give
//     ln w1(B, t) = key1(B) - t / alpha,   key1 = t_last / alpha + ln dT
//     ln w2(B, t) = key2(B) - t / beta + tau0 / beta,   key2 = t_last / beta + ln dT
// and the block's weight is min(w1, lambda * w2).  Within one segment the
// order of two blocks never changes with t (the shift -t/alpha is common), so
// each segment keeps an ordered set of (key, id); the block of least weight is
// the minimum of one of the two sets.  Log weights avoid the underflow of
// exp(-tau / beta) for long-idle blocks.
#include <cmath>
#include <cstdint>
#include <new>
#include <set>
#include <string>
#include <unordered_map>
#include <utility>
#include <vector>

#include "errors.h"
#include "msa_evictor.h"

namespace {

msa_status ev_error(msa_status st, const char* msg) {
  msa::set_last_error(msg);
  return st;
}

struct Entry {
  double key1, key2;
  size_t slot;  // position in the dense array (linear mode)
};

struct Dense {
  int64_t id;
  double key1, key2;
};

}  // namespace

struct msa_evictor_s {
  double alpha, beta, tau0, log_lambda;
  bool linear;
  std::unordered_map<int64_t, Entry> blocks;
  std::set<std::pair<double, int64_t>> tree1, tree2;  // ordered by (key, id)
  std::vector<Dense> dense;                           // linear mode: all blocks, any order

  // ln(f_B(t) * dT_B) from the stored keys.
  double log_weight(double key1, double key2, double t) const {
    const double a = key1 - t / alpha;
    const double b = log_lambda + key2 + (tau0 - t) / beta;
    return a < b ? a : b;
  }

  void erase(int64_t id, const Entry& e) {
    if (linear) {
      const size_t s = e.slot;
      dense[s] = dense.back();
      blocks[dense[s].id].slot = s;
      dense.pop_back();
    } else {
      tree1.erase({e.key1, id});
      tree2.erase({e.key2, id});
    }
    blocks.erase(id);
  }

  int64_t pick(double t) const {
    if (linear) {
      int64_t best = -1;
      double bw = 0;
      for (const Dense& d : dense) {
        const double w = log_weight(d.key1, d.key2, t);
        if (best < 0 || w < bw || (w == bw && d.id < best)) {
          best = d.id;
          bw = w;
        }
      }
      return best;
    }
    const auto& m1 = *tree1.begin();
    const auto& m2 = *tree2.begin();
    const double w1 = m1.first - t / alpha;
    const double w2 = log_lambda + m2.first + (tau0 - t) / beta;
    if (w1 < w2) return m1.second;
    if (w2 < w1) return m2.second;
    return m1.second < m2.second ? m1.second : m2.second;
  }
};

extern "C" {

msa_status msa_evictor_create(const msa_evictor_params* p, msa_evictor_t* out) {
  if (!out) return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_create: out is null");
  *out = nullptr;
  if (!p) return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_create: params is null");
  if (!std::isfinite(p->alpha) || !(p->alpha > 0) || !std::isfinite(p->beta) || !(p->beta > 0) ||
      !std::isfinite(p->lambda) || !(p->lambda > 0) || !std::isfinite(p->tau0))
    return ev_error(MSA_ERR_INVALID_ARG,
                    "msa_evictor_create: alpha, beta, lambda must be finite and > 0; tau0 finite");
  if (p->flags & ~MSA_EVICTOR_LINEAR)
    return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_create: unknown flags");
  for (int i = 0; i < 3; ++i)
    if (p->reserved[i]) return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_create: reserved != 0");
  msa_evictor_s* ev = new (std::nothrow) msa_evictor_s();
  if (!ev) return ev_error(MSA_ERR_OUT_OF_MEMORY, "msa_evictor_create: allocation failed");
  ev->alpha = p->alpha;
  ev->beta = p->beta;
  ev->tau0 = p->tau0;
  ev->log_lambda = std::log(p->lambda);
  ev->linear = (p->flags & MSA_EVICTOR_LINEAR) != 0;
  *out = ev;
  return MSA_OK;
}

void msa_evictor_destroy(msa_evictor_t ev) { delete ev; }

msa_status msa_evictor_add(msa_evictor_t ev, int64_t block_id, double t_last, double cost) {
  if (!ev) return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_add: null evictor");
  if (!std::isfinite(t_last) || !std::isfinite(cost) || !(cost > 0))
    return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_add: t_last must be finite, cost finite and > 0");
  try {
    auto ins = ev->blocks.emplace(block_id, Entry{});
    if (!ins.second) return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_add: block already present");
    Entry& e = ins.first->second;
    const double log_cost = std::log(cost);
    e.key1 = t_last / ev->alpha + log_cost;
    e.key2 = t_last / ev->beta + log_cost;
    if (ev->linear) {
      e.slot = ev->dense.size();
      ev->dense.push_back(Dense{block_id, e.key1, e.key2});
    } else {
      ev->tree1.emplace(e.key1, block_id);
      ev->tree2.emplace(e.key2, block_id);
    }
  } catch (const std::bad_alloc&) {
    ev->blocks.erase(block_id);
    return ev_error(MSA_ERR_OUT_OF_MEMORY, "msa_evictor_add: allocation failed");
  }
  return MSA_OK;
}

msa_status msa_evictor_remove(msa_evictor_t ev, int64_t block_id) {
  if (!ev) return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_remove: null evictor");
  auto it = ev->blocks.find(block_id);
  if (it == ev->blocks.end()) return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_remove: block not present");
  const Entry e = it->second;
  ev->erase(block_id, e);
  return MSA_OK;
}

msa_status msa_evictor_evict(msa_evictor_t ev, double t_now, int64_t* block_id) {
  if (!ev || !block_id) return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_evict: null argument");
  if (!std::isfinite(t_now)) return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_evict: t_now not finite");
  if (ev->blocks.empty()) return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_evict: no evictable block");
  const int64_t id = ev->pick(t_now);
  const Entry e = ev->blocks.at(id);
  ev->erase(id, e);
  *block_id = id;
  return MSA_OK;
}

msa_status msa_evictor_set_lambda(msa_evictor_t ev, double lambda) {
  if (!ev) return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_set_lambda: null evictor");
  if (!std::isfinite(lambda) || !(lambda > 0))
    return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_set_lambda: lambda must be finite and > 0");
  ev->log_lambda = std::log(lambda);
  return MSA_OK;
}

msa_status msa_evictor_set_lifespan(msa_evictor_t ev, double tau, double* lambda_out) {
  if (!ev) return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_set_lifespan: null evictor");
  if (!std::isfinite(tau) || tau < 0)
    return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_set_lifespan: tau must be finite and >= 0");
  ev->log_lambda = (tau - ev->tau0) / ev->beta - tau / ev->alpha;
  if (lambda_out) *lambda_out = std::exp(ev->log_lambda);
  return MSA_OK;
}

int64_t msa_evictor_size(msa_evictor_t ev) { return ev ? (int64_t)ev->blocks.size() : 0; }

msa_status msa_evictor_log_weight(msa_evictor_t ev, int64_t block_id, double t, double* out) {
  if (!ev || !out) return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_log_weight: null argument");
  auto it = ev->blocks.find(block_id);
  if (it == ev->blocks.end()) return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_log_weight: block not present");
  *out = ev->log_weight(it->second.key1, it->second.key2, t);
  return MSA_OK;
}

msa_status msa_evictor_replay(msa_evictor_t ev, int64_t n, const int32_t* op, const int64_t* id,
                              const double* t, const double* cost, int64_t* evicted,
                              int64_t* failed_at) {
  if (failed_at) *failed_at = -1;
  if (!ev || n < 0 || (n > 0 && (!op || !id || !t || !cost || !evicted)))
    return ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_replay: null or negative argument");
  for (int64_t i = 0; i < n; ++i) {
    msa_status st;
    evicted[i] = -1;
    switch (op[i]) {
      case MSA_EVICTOR_OP_ADD: st = msa_evictor_add(ev, id[i], t[i], cost[i]); break;
      case MSA_EVICTOR_OP_REMOVE: st = msa_evictor_remove(ev, id[i]); break;
      case MSA_EVICTOR_OP_EVICT: st = msa_evictor_evict(ev, t[i], &evicted[i]); break;
      case MSA_EVICTOR_OP_LIFESPAN: st = msa_evictor_set_lifespan(ev, t[i], nullptr); break;
      default: st = ev_error(MSA_ERR_INVALID_ARG, "msa_evictor_replay: unknown op code");
    }
    if (st != MSA_OK) {
      if (failed_at) *failed_at = i;
      return st;
    }
  }
  return MSA_OK;
}

}  // extern "C"
