// Runtime-adaptive proposal-length controller (Section 3.2, Eq. (1)):
// host-side scalar logic between the lookup and the verify step.
//
// Objective of a length l at retrieval similarity s:
//     J(l) = T(l) / (A(l, s) + 1)
// T: predicted iteration latency, exp of a quadratic in u = l / l_max fitted
//    to log-latency observations by exponentially weighted recursive least
//    squares;
// A: expected accepted proposal tokens, the sum over j <= l of the
//    probability that the first j tokens all pass, from two logistic models
//    over (1, s, j / l_max): the first token, and token j >= 2 given j - 1.
// One pass over l carries the running prefix probability and the running
// sum, so the whole objective row costs O(l_max).
#include <cmath>
#include <cstring>
#include <new>

#include "pf_internal.h"

static_assert(sizeof(pf_ctl_params) == 32, "pf_ctl_params layout");
static_assert(sizeof(pf_ctl_state) == 168, "pf_ctl_state layout");

namespace {

using pf::fail;
using pf::ok;

// logistic function without overflow for either sign of z
inline double logistic(double z) {
  if (z >= 0.0) return 1.0 / (1.0 + std::exp(-z));
  const double e = std::exp(z);
  return e / (1.0 + e);
}

inline double dot3(const double *w, double a, double b, double c) {
  double t = 0.0;
  t += w[0] * a;
  t += w[1] * b;
  t += w[2] * c;
  return t;
}

pf_status check_params(const pf_ctl_params *p) {
  if (!p) return fail(PF_EINVAL, "pf_ctl: null params");
  if (p->l_max < 1 || p->l_max > PF_MAX_DRAFT)
    return fail(PF_EINVAL, "pf_ctl: l_max %d outside 1..%d", p->l_max, PF_MAX_DRAFT);
  if (p->explore_every < 0) return fail(PF_EINVAL, "pf_ctl: explore_every < 0");
  if (!(p->lr > 0.0) || !std::isfinite(p->lr)) return fail(PF_EINVAL, "pf_ctl: lr must be > 0");
  if (!(p->forget > 0.0 && p->forget <= 1.0))
    return fail(PF_EINVAL, "pf_ctl: forget must lie in (0, 1]");
  if (!(p->prior_var > 0.0) || !std::isfinite(p->prior_var))
    return fail(PF_EINVAL, "pf_ctl: prior_var must be > 0");
  return ok();
}

// the objective for l = 0..L into J (J may be null); returns the first argmin
int objective_row(const pf_ctl *c, double s, int L, double *J) {
  const double lm = c->p.l_max;
  const double *th = c->st.theta;
  double prefix = 1.0, acc = 0.0;
  int best = 0;
  double best_j = 0.0;
  for (int l = 0; l <= L; ++l) {
    if (l >= 1) {
      const double *w = l == 1 ? c->st.w_first : c->st.w_cont;
      prefix *= logistic(dot3(w, 1.0, s, l / lm));
      acc += prefix;
    }
    const double u = l / lm;
    const double j = std::exp(dot3(th, 1.0, u, u * u)) / (acc + 1.0);
    if (J) J[l] = j;
    if (l == 0 || j < best_j) {
      best = l;
      best_j = j;
    }
  }
  return best;
}

void logistic_step(double *w, double lr, double x1, double x2, bool y) {
  const double g = lr * ((y ? 1.0 : 0.0) - logistic(dot3(w, 1.0, x1, x2)));
  w[0] += g;
  w[1] += g * x1;
  w[2] += g * x2;
}

// one recursive-least-squares update of log T on (1, u, u^2)
void latency_step(pf_ctl_state &st, double lam, double u, double y) {
  const double x[3] = {1.0, u, u * u};
  double Px[3];
  for (int r = 0; r < 3; ++r) Px[r] = dot3(st.P + 3 * r, x[0], x[1], x[2]);
  const double den = lam + dot3(x, Px[0], Px[1], Px[2]);
  double k[3];
  for (int r = 0; r < 3; ++r) k[r] = Px[r] / den;
  const double err = y - dot3(st.theta, x[0], x[1], x[2]);
  for (int r = 0; r < 3; ++r) st.theta[r] += k[r] * err;
  for (int r = 0; r < 3; ++r)
    for (int q = 0; q < 3; ++q) st.P[3 * r + q] = (st.P[3 * r + q] - k[r] * Px[q]) / lam;
}

int range_of(const pf_ctl *c, int32_t avail) {
  int L = avail < c->p.l_max ? avail : c->p.l_max;
  return L < 0 ? 0 : L;
}

}  // namespace

extern "C" {

pf_status pf_ctl_create(const pf_ctl_params *params, pf_ctl **out) {
  if (!out) return fail(PF_EINVAL, "pf_ctl_create: null out");
  *out = nullptr;
  if (pf_status r = check_params(params)) return r;
  pf_ctl *c = new (std::nothrow) pf_ctl;
  if (!c) return fail(PF_ENOMEM, "pf_ctl_create: out of host memory");
  std::memset(c, 0, sizeof(*c));
  c->p = *params;
  for (int r = 0; r < 3; ++r) c->st.P[4 * r] = params->prior_var;
  *out = c;
  return ok();
}

void pf_ctl_destroy(pf_ctl *ctl) { delete ctl; }

pf_status pf_ctl_get_state(const pf_ctl *ctl, pf_ctl_state *out) {
  if (!ctl || !out) return fail(PF_EINVAL, "pf_ctl_get_state: null pointer");
  *out = ctl->st;
  return ok();
}

pf_status pf_ctl_set_state(pf_ctl *ctl, const pf_ctl_state *in) {
  if (!ctl || !in) return fail(PF_EINVAL, "pf_ctl_set_state: null pointer");
  const double *v = in->w_first;  // the 18 doubles: w_first .. P
  for (int i = 0; i < 18; ++i)
    if (!std::isfinite(v[i])) return fail(PF_EINVAL, "pf_ctl_set_state: non-finite state");
  if (in->n_choose < 0 || in->n_explore < 0 || in->n_observe < 0)
    return fail(PF_EINVAL, "pf_ctl_set_state: negative counter");
  ctl->st = *in;
  return ok();
}

pf_status pf_ctl_objective(const pf_ctl *ctl, double s, int32_t avail, double *objective_out,
                           int32_t *best_out) {
  if (!ctl) return fail(PF_EINVAL, "pf_ctl_objective: null controller");
  if (!std::isfinite(s)) return fail(PF_EINVAL, "pf_ctl_objective: similarity not finite");
  const int best = objective_row(ctl, s, range_of(ctl, avail), objective_out);
  if (best_out) *best_out = best;
  return ok();
}

pf_status pf_ctl_choose(pf_ctl *ctl, double s, int32_t avail, int32_t *l_out) {
  if (!ctl || !l_out) return fail(PF_EINVAL, "pf_ctl_choose: null pointer");
  if (!std::isfinite(s)) return fail(PF_EINVAL, "pf_ctl_choose: similarity not finite");
  const int L = range_of(ctl, avail);
  int l = objective_row(ctl, s, L, nullptr);
  pf_ctl_state &st = ctl->st;
  ++st.n_choose;
  const int every = ctl->p.explore_every;
  if (every > 0 && L > 0 && st.n_choose % every == 0) {
    // alternate between the neighbour above and the one below
    const int step = (st.n_explore % 2 == 0) ? 1 : -1;
    int nb = l + step;
    if (nb < 0 || nb > L) nb = l - step;
    ++st.n_explore;
    l = nb;
  }
  *l_out = l;
  return ok();
}

pf_status pf_ctl_observe(pf_ctl *ctl, int32_t l, double s, int32_t accepted, double latency_ms) {
  if (!ctl) return fail(PF_EINVAL, "pf_ctl_observe: null controller");
  if (l < 0 || l > ctl->p.l_max)
    return fail(PF_EINVAL, "pf_ctl_observe: length %d outside 0..%d", l, ctl->p.l_max);
  if (accepted < 0 || accepted > l)
    return fail(PF_EINVAL, "pf_ctl_observe: accepted %d outside 0..%d", accepted, l);
  if (!(latency_ms > 0.0) || !std::isfinite(latency_ms))
    return fail(PF_EINVAL, "pf_ctl_observe: latency must be finite and > 0");
  if (!std::isfinite(s)) return fail(PF_EINVAL, "pf_ctl_observe: similarity not finite");
  pf_ctl_state &st = ctl->st;
  const double lm = ctl->p.l_max;
  if (l >= 1) {
    logistic_step(st.w_first, ctl->p.lr, s, 1.0 / lm, accepted >= 1);
    // token j is a sample of the conditional model only while every earlier
    // token was accepted: j = 2 .. min(l, accepted + 1)
    const int last = accepted + 1 < l ? accepted + 1 : l;
    for (int j = 2; j <= last; ++j) logistic_step(st.w_cont, ctl->p.lr, s, j / lm, accepted >= j);
  }
  latency_step(st, ctl->p.forget, l / lm, std::log(latency_ms));
  ++st.n_observe;
  return ok();
}

}  // extern "C"
