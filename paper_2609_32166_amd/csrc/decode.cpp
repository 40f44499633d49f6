// One decoding iteration of Section 3.2 driven from the host: the paper's
// retrieval, the proposal-length choice of Eq. (1), single-pass verification
// and the commit, optionally the memory update (the iteration's tokens and
// their contexts appended to the store), then the next iteration's query key
// and the controller's update from what was observed.
//
// The host needs two facts from the device per iteration (the retrieved
// proposal before choosing its length, the accepted length after the step),
// so the iteration synchronises twice, through a pinned staging buffer of the
// model. Everything between the two reads is enqueued back to back.
#include <chrono>
#include <cstring>

#include "pf_internal.h"

static_assert(sizeof(pf_iteration) == 40, "pf_iteration layout");

using pf::fail;
using pf::ok;

namespace {

constexpr size_t kStageBytes = 4096;
static_assert(sizeof(pf_draft) + sizeof(pf_verify_result) <= kStageBytes, "stage size");

#define DCHK(call)                                                                      \
  do {                                                                                  \
    hipError_t e_ = (call);                                                             \
    if (e_ != hipSuccess) return fail(PF_EHIP, "%s: %s", #call, hipGetErrorString(e_)); \
  } while (0)

}  // namespace

extern "C" {

pf_status pf_decode_iteration(pf_model *m, pf_kv_cache *kv, pf_context *ctx, pf_store *store,
                              const pf_keyproj *kp, pf_ctl *ctl, int32_t l_fixed, int32_t append,
                              int8_t *q_dev, pf_draft *draft_dev, pf_verify_result *res_dev,
                              pf_iteration *out, pf_stream s) {
  const auto t0 = std::chrono::steady_clock::now();
  if (!m || !kv || !ctx || !store || !kp || !q_dev || !draft_dev || !res_dev || !out)
    return fail(PF_EINVAL, "pf_decode_iteration: null pointer");
  if (!ctl && (l_fixed < 0 || l_fixed > PF_MAX_DRAFT))
    return fail(PF_EINVAL, "pf_decode_iteration: l_fixed %d not in [0,%d]", l_fixed, PF_MAX_DRAFT);
  hipStream_t hs = (hipStream_t)s;
  if (!m->stage) DCHK(hipHostMalloc(&m->stage, kStageBytes, hipHostMallocDefault));
  pf_draft *d = (pf_draft *)m->stage;
  pf_verify_result *r = (pf_verify_result *)((char *)m->stage + sizeof(pf_draft));

  // retrieval: the longest proposal the choice may use
  const int k_max = ctl ? ctl->p.l_max : l_fixed;
  if (pf_status e = pf_draft_lookup_cosine(store, ctx, q_dev, k_max, 0, 1, PF_MAX_DRAFT,
                                           draft_dev, s))
    return e;
  DCHK(hipMemcpyAsync(d, draft_dev, sizeof(pf_draft), hipMemcpyDeviceToHost, hs));
  DCHK(hipStreamSynchronize(hs));
  const int n_found = d->n_found;
  const int avail = d->n_nodes - 1;
  const double sim = n_found > 0 ? (double)d->cand_score[0] : 0.0;

  // Eq. (1), or the fixed length; no eligible entry: a greedy pass
  int l = 0;
  if (n_found > 0) {
    if (ctl) {
      if (pf_status e = pf_ctl_choose(ctl, sim, avail, &l)) return e;
    } else {
      l = l_fixed < avail ? l_fixed : avail;
    }
  }
  const int rows = l + 1;
  if (pf_status e = pf_verify_step(m, kv, draft_dev, rows, 0, nullptr, res_dev, s)) return e;
  if (pf_status e = pf_kv_commit(kv, res_dev, ctx, s)) return e;
  if (append) {
    if (pf_status e = pf_store_append_verified(store, m, kp, res_dev, s)) return e;
  }
  if (pf_status e = pf_verify_query_key(m, kp, res_dev, q_dev, s)) return e;
  DCHK(hipMemcpyAsync(r, res_dev, sizeof(pf_verify_result), hipMemcpyDeviceToHost, hs));
  DCHK(hipStreamSynchronize(hs));

  // the commit grew both bounds by the verify rows; the lengths grew by
  // accepted + 1 (pf_kv_commit checked the context capacity for all rows)
  const int grown = r->accept_len + 1;
  kv->host_bound -= rows - grown;
  ctx->host_bound -= rows - grown;
  if (append) store->log_host_bound -= rows - grown;

  const double ms =
      std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
  out->n_found = n_found;
  out->avail = avail;
  out->l = l;
  out->accepted = r->accept_len;
  out->bonus = r->bonus;
  out->status = r->status;
  out->s = sim;
  out->ms = ms;
  if (ctl) {
    if (pf_status e = pf_ctl_observe(ctl, l, sim, r->accept_len, ms)) return e;
  }
  return ok();
}

}  // extern "C"
