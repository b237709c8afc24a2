// Decisions of the global coordinator (include/hxf_coord.h): workload-balanced
// instance selection (Section 4.1) and the latency-regression t-test that
// triggers alpha re-tuning (Section 4.3).  Host code only.
#include <cmath>
#include <limits>

#include "hxf_coord.h"

// The score and the statistics are specified operation by operation; no fused
// multiply-adds, so that every compiler and the host reference round alike.
#pragma clang fp contract(off)

namespace {

// Regularised incomplete beta function I_x(a, b) for a, b > 0, with y = 1 - x
// supplied separately so that neither tail loses digits to cancellation.  The
// continued fraction of I_x(a, b) (coefficients d_{2m+1} = -(a+m)(a+b+m)x /
// ((a+2m)(a+2m+1)), d_{2m} = m(b-m)x / ((a+2m-1)(a+2m))) is summed by the modified
// Lentz method on the side where it converges quickly, x < (a+1)/(a+b+2); the other
// side uses I_x(a, b) = 1 - I_y(b, a).
double cont_frac(double a, double b, double x) {
  const double tiny = 1e-300, eps = 1e-16;
  double f = tiny, c = tiny, d = 0.0;
  for (int k = 1; k <= 2000; ++k) {
    double num;
    if (k == 1) {
      num = 1.0;
    } else {
      const int j = k - 1;   // index of the coefficient d_j
      const double m = (double)(j / 2);
      if (j % 2 == 1) num = -((a + m) * (a + b + m) * x) / ((a + 2.0 * m) * (a + 2.0 * m + 1.0));
      else num = (m * (b - m) * x) / ((a + 2.0 * m - 1.0) * (a + 2.0 * m));
    }
    d = 1.0 + num * d;
    if (std::fabs(d) < tiny) d = tiny;
    c = 1.0 + num / c;
    if (std::fabs(c) < tiny) c = tiny;
    d = 1.0 / d;
    const double delta = c * d;
    f *= delta;
    if (k > 1 && std::fabs(delta - 1.0) < eps) break;
  }
  return f;
}

double inc_beta(double a, double b, double x, double y) {
  if (x <= 0.0) return 0.0;
  if (y <= 0.0) return 1.0;
  const double log_front = std::lgamma(a + b) - std::lgamma(a) - std::lgamma(b) + a * std::log(x) + b * std::log(y);
  const double front = std::exp(log_front);
  if (x < (a + 1.0) / (a + b + 2.0)) return front * cont_frac(a, b, x) / a;
  return 1.0 - front * cont_frac(b, a, y) / b;
}

// P(T >= t) for Student's t with dof degrees of freedom:
// P(T >= |t|) = I_{dof/(dof+t^2)}(dof/2, 1/2) / 2.
double t_upper_tail(double t, double dof) {
  if (std::isinf(t)) return t > 0 ? 0.0 : 1.0;
  const double t2 = t * t;
  const double x = dof / (dof + t2), y = t2 / (dof + t2);
  const double half_tail = 0.5 * inc_beta(0.5 * dof, 0.5, x, y);
  return t >= 0.0 ? half_tail : 1.0 - half_tail;
}

void mean_var(const double* v, int32_t n, double* mean, double* var) {
  double s = 0.0;
  for (int32_t i = 0; i < n; ++i) s += v[i];
  const double m = s / (double)n;
  double q = 0.0;
  for (int32_t i = 0; i < n; ++i) {
    const double e = v[i] - m;
    q += e * e;
  }
  *mean = m;
  *var = q / (double)(n - 1);
}

}  // namespace

extern "C" {

int hxf_wb_select(int32_t n, const int64_t* t_comp_us, const int64_t* t_queue_us, double alpha, double beta,
                  int32_t* out_index) {
  if (n < 1 || !t_comp_us || !t_queue_us || !out_index) return HXF_EINVAL;
  if (!(alpha >= 0.0 && alpha <= 1.0) || !(beta >= 0.0) || std::isinf(beta)) return HXF_EINVAL;
  double best = -std::numeric_limits<double>::infinity();
  int32_t arg = 0;
  for (int32_t m = 0; m < n; ++m) {
    const double q = (double)(t_queue_us[m] > 1 ? t_queue_us[m] : 1);
    const double reward = (1.0 - alpha) * (beta / q);
    const double cost = alpha * (double)t_comp_us[m];
    const double score = reward - cost;
    if (m == 0 || score > best) {
      best = score;
      arg = m;
    }
  }
  *out_index = arg;
  return HXF_OK;
}

int hxf_ttest_greater(const double* x_new, int32_t n_new, const double* x_ref, int32_t n_ref, double* t_stat,
                      double* dof, double* p_value) {
  if (!x_new || !x_ref || !t_stat || !dof || !p_value || n_new < 2 || n_ref < 2) return HXF_EINVAL;
  for (int32_t i = 0; i < n_new; ++i)
    if (!std::isfinite(x_new[i])) return HXF_EINVAL;
  for (int32_t i = 0; i < n_ref; ++i)
    if (!std::isfinite(x_ref[i])) return HXF_EINVAL;
  double m1, v1, m2, v2;
  mean_var(x_new, n_new, &m1, &v1);
  mean_var(x_ref, n_ref, &m2, &v2);
  const double s1 = v1 / (double)n_new, s2 = v2 / (double)n_ref;
  const double se2 = s1 + s2;
  if (se2 == 0.0) {
    *dof = (double)(n_new + n_ref - 2);
    if (m1 > m2) {
      *t_stat = std::numeric_limits<double>::infinity();
      *p_value = 0.0;
    } else {
      *t_stat = m1 == m2 ? 0.0 : -std::numeric_limits<double>::infinity();
      *p_value = 1.0;
    }
    return HXF_OK;
  }
  const double t = (m1 - m2) / std::sqrt(se2);
  const double den = (s1 * s1) / (double)(n_new - 1) + (s2 * s2) / (double)(n_ref - 1);
  const double nu = (se2 * se2) / den;
  *t_stat = t;
  *dof = nu;
  *p_value = t_upper_tail(t, nu);
  return HXF_OK;
}

}  // extern "C"
