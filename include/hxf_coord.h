/*
 * hxf_coord.h -- C ABI of the global coordinator's decisions across instances.
 *
 * The paper schedules at two levels: a global coordinator assigns each LLM
 * request of a workflow to one of N model instances (workload-balanced
 * dispatch, Section 4.1), and each instance orders its own queue (Section 4.2,
 * hxf.h).  The dispatch weight alpha is tuned online from tail latency
 * (Section 4.3).  This header holds the per-decision arithmetic of those two
 * sections; the event loop that calls it (arrivals, stage completions, the
 * sliding window, the alpha grid replay) is host code above the library.
 *
 * Conventions are those of hxf.h: int return codes (HXF_OK or a negative
 * HXF_E* code), int64 microseconds, no allocation visible to the caller, no
 * exception crossing the boundary.  Every function here is host-only.
 */
#ifndef HXF_COORD_H
#define HXF_COORD_H

#include <stdint.h>

#include "hxf.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Queueing cost of the instance, Section 4.1 (the sum over the instance's queue of the
 * requests' compute-cost estimates): the sum of t_comp over every request submitted to
 * this instance that has not finished or been cancelled, queued or running (a running
 * request still holds batch slots and tokens that a new one would wait for, so each
 * counts at its full estimate: the maximal queueing time).  HXF_EINVAL on null pointers. */
int hxf_queue_cost(hxf_instance* inst, int64_t* t_queue_us);

/* Compute-cost estimate t_comp (Section 4.1) of a request of l_in prefill tokens and
 * l_out output tokens on this instance's cost model (hxf_sched_cfg.cost_ps).
 * HXF_EINVAL on a null pointer or a negative length. */
int hxf_request_cost(hxf_instance* inst, int32_t l_in, int32_t l_out, int64_t* t_comp_us);

/* hxf_submit with the SLO budget of Section 4.2 computed from instance-average costs:
 * every cost in the budget (this request's and the later stages' in req->rest) is the
 * mean over n_instances instances, floor(sum of their unfloored estimates / n_instances),
 * where cost_sum_ps (host, 4 int64) is the n_instances instances' cost coefficients summed
 * element-wise.  The urgency key still uses this instance's own t_comp.  With
 * n_instances = 1 and this instance's coefficients it equals hxf_submit.  HXF_EINVAL if
 * n_instances < 1 or cost_sum_ps is null; otherwise the errors of hxf_submit. */
int hxf_submit_shared(hxf_instance* inst, const hxf_stage_req* req, int64_t now_us, const int64_t* cost_sum_ps,
                      int32_t n_instances, uint64_t* out_id);

/* Workload-balanced dispatch, Section 4.1: the index m in [0, n) maximising
 *   score(m) = (1 - alpha) * beta / max(t_queue_us[m], 1) - alpha * t_comp_us[m],
 * evaluated in IEEE double without fused multiply-adds as
 *   a = (1 - alpha) * (beta / q);  b = alpha * c;  score = a - b.
 * A queue of zero counts as one microsecond (the clock's resolution), so every empty
 * instance gets the same, largest queue reward and the compute term picks among them.
 * Ties go to the lowest index.  t_comp_us, t_queue_us: host arrays of n int64 (us);
 * beta: the deployment constant C_ref * Q_ref (us^2).  HXF_EINVAL if n < 1, a pointer is
 * null, alpha is outside [0, 1] or beta is negative or not finite. */
int hxf_wb_select(int32_t n, const int64_t* t_comp_us, const int64_t* t_queue_us, double alpha, double beta,
                  int32_t* out_index);

/* One-sided two-sample t-test of Section 4.3 (H1: the new window's latencies are larger
 * on average than the reference window's), in Welch's form (no equal-variance
 * assumption):
 *   t = (mean_new - mean_ref) / sqrt(v_new/n_new + v_ref/n_ref)   (v: sample variances),
 *   dof by the Welch-Satterthwaite formula, p = P(T_dof >= t) from the Student t
 *   distribution (regularised incomplete beta, evaluated by its continued fraction).
 * If both variances are zero: t = +inf and p = 0 when mean_new > mean_ref, else t = 0
 * (or -inf) and p = 1; dof is then n_new + n_ref - 2.
 * x_new, x_ref: host arrays of doubles.  HXF_EINVAL if either has fewer than 2 values, a
 * pointer is null, or a value is not finite. */
int hxf_ttest_greater(const double* x_new, int32_t n_new, const double* x_ref, int32_t n_ref, double* t_stat,
                      double* dof, double* p_value);

#ifdef __cplusplus
}
#endif
#endif /* HXF_COORD_H */
