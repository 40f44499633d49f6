// C-ABI layer of libpf: argument checks, the experience-store builder, model
// creation (weight packing) and the launch sequence of one verify step.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "kernels.h"

using namespace pf;

thread_local LaunchTimer *pf::t_launch_timer = nullptr;

static_assert(sizeof(pf_draft) == 1384, "pf_draft layout");
static_assert(sizeof(pf_verify_result) == 808, "pf_verify_result layout");

static thread_local std::string g_err;

pf_status pf::fail(pf_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

pf_status pf::ok() {
  g_err.clear();
  return PF_OK;
}

namespace {

#define HIPCHK(call)                                                                   \
  do {                                                                                 \
    hipError_t e_ = (call);                                                            \
    if (e_ != hipSuccess) return fail(PF_EHIP, "%s: %s", #call, hipGetErrorString(e_)); \
  } while (0)

inline hipStream_t st(pf_stream s) { return (hipStream_t)s; }
inline int64_t roundup(int64_t a, int64_t b) { return (a + b - 1) / b * b; }
inline bool is_bf16(const pf_model *m) { return m->cfg.dtype == PF_DTYPE_BF16; }
inline int frag_k_of(const pf_model *m) { return is_bf16(m) ? 32 : 16; }

Packed geom(int64_t N, int64_t K, int kf) {
  Packed p;
  p.N = N;
  p.K = K;
  p.NT = (N + 15) / 16;
  p.KFr = (K + kf - 1) / kf;
  return p;
}

// split-K factor for a partial-sum GEMM, from its shape and the CU count
// only (never the row count, so every row's summation order is fixed): the
// smallest factor from about one block per CU up whose blocks (counted at two
// n tiles per block) fill the CUs evenly, at least 7/8 of the slots of the
// busiest CU count in use, with at least two fragments per wave. Measured on
// both models: 7B O and down 3 -> 4 splits (336 -> 448 blocks; 33 rows:
// down 30.6 -> 25.8 us, O 9.0 -> 7.9; 17 rows: down 32.7 -> 27.2); 3B keeps
// 4 (256 blocks), where 6 costs O 4.6 -> 5.9 us and down 11.2 -> 12.7.
int splits_for(int64_t nblocks, int64_t KFr, int cus) {
  int64_t cap = KFr / 8;
  if (cap < 1) cap = 1;
  if (cus < 1) cus = 1;
  const int64_t s0 = (cus + nblocks - 1) / nblocks;
  for (int64_t s = s0; s <= cap; ++s) {
    const int64_t b = nblocks * s, per_cu = (b + cus - 1) / cus;
    if (8 * b >= 7 * per_cu * cus) return (int)s;
  }
  return (int)(s0 < cap ? s0 : cap);
}

// blocks of a partial-sum GEMM counted at two n tiles per block whatever the
// row count, so the split factor (and with it every row's summation order)
// does not depend on how many rows a step verifies
int64_t partial_blocks(const Packed &p) {
  const int nt = gemm_tiles_per_block(EPI_PARTIAL, 1);
  return (p.NT + nt - 1) / nt;
}

constexpr int kMaxSplitsAttn = 64;

// Collects one (start, stop) event pair per kernel launched while installed,
// tagged with the profiling kind current at the launch.
struct Prof final : LaunchTimer {
  std::vector<hipEvent_t> ev;
  std::vector<int> kind;
  int cur = -1;
  bool events(hipEvent_t *start, hipEvent_t *stop) override {
    hipError_t r = hipEventCreateWithFlags(start, hipEventDisableSystemFence);
    if (r == hipSuccess) {
      r = hipEventCreateWithFlags(stop, hipEventDisableSystemFence);
      if (r != hipSuccess) (void)hipEventDestroy(*start);
    }
    if (r != hipSuccess) {
      if (err == hipSuccess) err = r;
      return false;
    }
    ev.push_back(*start);
    ev.push_back(*stop);
    kind.push_back(cur);
    return true;
  }
  ~Prof() override {
    for (hipEvent_t e : ev) (void)hipEventDestroy(e);
  }
};

// Installs a timer for the lifetime of the scope (no-op for a null timer).
struct TimerScope {
  explicit TimerScope(LaunchTimer *t) { t_launch_timer = t; }
  ~TimerScope() { t_launch_timer = nullptr; }
};

template <typename T> pf_status dev_alloc(T **p, int64_t bytes, int64_t *total) {
  if (bytes <= 0) bytes = 16;
  if (hipMalloc((void **)p, (size_t)bytes) != hipSuccess) {
    *p = nullptr;
    return fail(PF_ENOMEM, "hipMalloc of %lld bytes failed", (long long)bytes);
  }
  if (total) *total += bytes;
  return PF_OK;
}

void prefill_free(pf_model *m) {
  void *ptrs[] = {m->pre_x, m->pre_y, m->pre_rope, m->pre_apo, m->pre_apml, m->pre_xn,
                  m->pre_qb, m->pre_attn, m->pre_act, m->pre_rowinfo, m->pre_status,
                  m->pre_part, m->pre_xb};
  for (void *p : ptrs)
    if (p) (void)hipFree(p);
  m->pre_x = m->pre_y = m->pre_rope = m->pre_apo = m->pre_apml = m->pre_part = nullptr;
  m->pre_xn = m->pre_qb = m->pre_attn = m->pre_act = m->pre_xb = nullptr;
  m->pre_rowinfo = m->pre_status = nullptr;
  m->pre_rows = 0;
}

void model_free(pf_model *m) {
  if (!m) return;
  prefill_free(m);
  void *ptrs[] = {m->wqkv, m->wo, m->wgu, m->wd, m->lm, m->embed, m->attn_norm, m->ffn_norm,
                  m->final_norm, m->inv_freq, m->x, m->xn, m->ssq, m->qb, m->attn, m->act, m->part,
                  m->apart_o, m->apart_ml, m->amax, m->rope, m->rowinfo, m->pred, m->flags};
  for (void *p : ptrs)
    if (p) (void)hipFree(p);
  if (m->stage) (void)hipHostFree(m->stage);
  delete m;
}

}  // namespace

extern "C" {

const char *pf_last_error(void) { return g_err.c_str(); }
const char *pf_version(void) { return "pf 0.1 gfx950"; }

// ---------------------------------------------------------------------------
// context
// ---------------------------------------------------------------------------

pf_status pf_context_init(pf_context *ctx, int32_t *tokens_dev, int32_t *len_dev, int64_t capacity,
                          int64_t len, pf_stream s) {
  if (!ctx || !tokens_dev || !len_dev) return fail(PF_EINVAL, "pf_context_init: null pointer");
  if (capacity < 1 || len < 0 || len > capacity || capacity > INT32_MAX)
    return fail(PF_EINVAL, "pf_context_init: bad capacity %lld / len %lld", (long long)capacity,
                (long long)len);
  ctx->tokens = tokens_dev;
  ctx->len = len_dev;
  ctx->capacity = capacity;
  ctx->host_bound = len;
  HIPCHK(launch_set_int(len_dev, (int32_t)len, st(s)));
  return ok();
}

pf_status pf_context_sync_bound(pf_context *ctx, pf_stream s) {
  if (!ctx || !ctx->len) return fail(PF_EINVAL, "pf_context_sync_bound: null pointer");
  int32_t v = 0;
  HIPCHK(hipMemcpyAsync(&v, ctx->len, 4, hipMemcpyDeviceToHost, st(s)));
  HIPCHK(hipStreamSynchronize(st(s)));
  ctx->host_bound = v;
  return ok();
}

// ---------------------------------------------------------------------------
// store
// ---------------------------------------------------------------------------

pf_status pf_store_build(const int32_t *tokens, const int64_t *offs, int64_t n_seqs, int32_t ngram,
                         pf_stream s, pf_store **out) {
  if (!out) return fail(PF_EINVAL, "pf_store_build: null out");
  *out = nullptr;
  if (!offs || n_seqs < 0) return fail(PF_EINVAL, "pf_store_build: bad offsets");
  if (ngram < 1 || ngram > 8) return fail(PF_EINVAL, "pf_store_build: ngram %d not in [1,8]", ngram);
  if (offs[0] != 0) return fail(PF_EINVAL, "pf_store_build: offsets[0] must be 0");
  for (int64_t i = 0; i < n_seqs; ++i)
    if (offs[i + 1] < offs[i]) return fail(PF_EINVAL, "pf_store_build: offsets not monotonic");
  const int64_t T = offs[n_seqs];
  if (T > 0 && !tokens) return fail(PF_EINVAL, "pf_store_build: null tokens");
  if (T >= ((int64_t)1 << 31)) return fail(PF_EUNSUPPORTED, "pf_store_build: T >= 2^31");

  // eligible entries: n-gram inside the sequence and p < last position
  std::vector<int32_t> pos, rem;
  for (int64_t q = 0; q < n_seqs; ++q) {
    const int64_t a = offs[q], last = offs[q + 1] - 1;
    for (int64_t p = a + ngram - 1; p < last; ++p) {
      pos.push_back((int32_t)p);
      rem.push_back((int32_t)(last - p));
    }
  }
  const int64_t E = (int64_t)pos.size();
  int nb_log2 = 0;
  while (((int64_t)1 << nb_log2) < E && nb_log2 < 28) ++nb_log2;
  const int64_t nb = (int64_t)1 << nb_log2;
  std::vector<uint32_t> bk(E);
  std::vector<int32_t> off(nb + 1, 0);
  for (int64_t i = 0; i < E; ++i) {
    bk[i] = ngram_hash(tokens + pos[i] - ngram + 1, ngram) & (uint32_t)(nb - 1);
    off[bk[i] + 1]++;
  }
  for (int64_t b = 0; b < nb; ++b) off[b + 1] += off[b];
  std::vector<int32_t> fill(off.begin(), off.end() - 1);
  std::vector<int32_t> epos(E), erem(E);
  for (int64_t i = 0; i < E; ++i) {
    int32_t at = fill[bk[i]]++;
    epos[at] = pos[i];
    erem[at] = rem[i];
  }

  pf_store *S = new pf_store();
  S->T = T;
  S->E = E;
  S->h_tokens.assign(tokens, tokens + T);
  S->h_last.resize(T);
  for (int64_t q = 0; q < n_seqs; ++q)
    for (int64_t p = offs[q]; p < offs[q + 1]; ++p) S->h_last[p] = (int32_t)(offs[q + 1] - 1);
  S->nb_log2 = nb_log2;
  S->ngram = ngram;
  pf_status r = PF_OK;
  if ((r = dev_alloc(&S->tokens, T * 4, nullptr)) || (r = dev_alloc(&S->ent_pos, E * 4, nullptr)) ||
      (r = dev_alloc(&S->ent_rem, E * 4, nullptr)) ||
      (r = dev_alloc(&S->bucket_off, (nb + 1) * 4, nullptr))) {
    pf_store_destroy(S);
    return r;
  }
  hipStream_t hs = st(s);
  hipError_t e = hipSuccess;
  if (T) e = hipMemcpyAsync(S->tokens, tokens, T * 4, hipMemcpyHostToDevice, hs);
  if (e == hipSuccess && E) e = hipMemcpyAsync(S->ent_pos, epos.data(), E * 4, hipMemcpyHostToDevice, hs);
  if (e == hipSuccess && E) e = hipMemcpyAsync(S->ent_rem, erem.data(), E * 4, hipMemcpyHostToDevice, hs);
  if (e == hipSuccess)
    e = hipMemcpyAsync(S->bucket_off, off.data(), (nb + 1) * 4, hipMemcpyHostToDevice, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);  // host vectors die here
  if (e != hipSuccess) {
    pf_store_destroy(S);
    return fail(PF_EHIP, "pf_store_build: copy failed: %s", hipGetErrorString(e));
  }
  *out = S;
  return ok();
}

static void store_free_keys(pf_store *S) {
  void *ptrs[] = {S->keys, S->tok_off, S->cpos, S->crem, S->cnk, S->cpart, S->cpart_elig};
  for (void *p : ptrs)
    if (p) (void)hipFree(p);
  S->keys = nullptr;
  S->tok_off = S->cpos = S->crem = S->cnk = S->cpart_elig = nullptr;
  S->cpart = nullptr;
  S->Ec = 0;
  S->n_tok = 0;
}

static void store_free_log(pf_store *S) {
  void *ptrs[] = {S->log_state, S->log_seq, S->log_nk, S->seq_end, S->row_keys};
  for (void *p : ptrs)
    if (p) (void)hipFree(p);
  S->log_state = S->log_seq = S->log_nk = S->seq_end = nullptr;
  S->row_keys = nullptr;
  S->cap_log = S->max_log_seqs = 0;
  S->log_host_bound = 0;
  S->log_seqs_host = 0;
}

void pf_store_destroy(pf_store *S) {
  if (!S) return;
  store_free_log(S);
  if (S->tokens) (void)hipFree(S->tokens);
  if (S->ent_pos) (void)hipFree(S->ent_pos);
  if (S->ent_rem) (void)hipFree(S->ent_rem);
  if (S->bucket_off) (void)hipFree(S->bucket_off);
  store_free_keys(S);
  delete S;
}

int64_t pf_store_size(const pf_store *S) { return S ? S->T : -1; }

// ---------------------------------------------------------------------------
// cosine retrieval
// ---------------------------------------------------------------------------

pf_status pf_keyproj_create(const float *R, int32_t hidden, pf_keyproj **out) {
  if (!out) return fail(PF_EINVAL, "pf_keyproj_create: null out");
  *out = nullptr;
  if (!R) return fail(PF_EINVAL, "pf_keyproj_create: null projection");
  if (hidden < 16 || hidden > kKeyMaxHidden)
    return fail(PF_EINVAL, "pf_keyproj_create: hidden %d not in [16, %d]", hidden, kKeyMaxHidden);
  pf_keyproj *kp = new pf_keyproj();
  kp->H = hidden;
  kp->Lc = (int32_t)roundup((hidden + 15) / 16, 4);
  const int64_t nrc = (int64_t)PF_KEY_DIM * 16 * kp->Lc;
  std::vector<float> rc((size_t)nrc, 0.f);
  for (int j = 0; j < PF_KEY_DIM; ++j)
    for (int c = 0; c < 16; ++c)
      for (int t = 0; t < kp->Lc; ++t) {
        const int k = c + 16 * t;
        if (k < hidden) rc[((size_t)j * 16 + c) * kp->Lc + t] = R[(size_t)j * hidden + k];
      }
  pf_status r = PF_OK;
  if ((r = dev_alloc(&kp->Rc, nrc * 4, nullptr)) ||
      (r = dev_alloc(&kp->v, (int64_t)kKeyBatch * PF_KEY_DIM * 8, nullptr))) {
    pf_keyproj_destroy(kp);
    return r;
  }
  hipError_t e = hipMemcpy(kp->Rc, rc.data(), (size_t)nrc * 4, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    pf_keyproj_destroy(kp);
    return fail(PF_EHIP, "pf_keyproj_create: copy failed: %s", hipGetErrorString(e));
  }
  *out = kp;
  return ok();
}

void pf_keyproj_destroy(pf_keyproj *kp) {
  if (!kp) return;
  if (kp->Rc) (void)hipFree(kp->Rc);
  if (kp->v) (void)hipFree(kp->v);
  delete kp;
}

// keys of n rows in batches that fit a projection work buffer of kKeyBatch
// rows (the projection's own, or the given one)
static pf_status encode_rows(const pf_keyproj *kp, bool bf16, bool packed, const void *h,
                             int64_t ld, int64_t n, int8_t *keys, hipStream_t hs,
                             double *work = nullptr) {
  double *v = work ? work : kp->v;
  const size_t esz = bf16 ? 2 : 4;
  for (int64_t b = 0; b < n; b += kKeyBatch) {
    const int nb = (int)std::min<int64_t>(kKeyBatch, n - b);
    if (packed) {
      // rows b.. of the packed verify activations: batches start on 16-row
      // tiles (kKeyBatch is a multiple of 16), so shift by whole tiles
      const int kf = bf16 ? 32 : 16;
      const char *hb = (const char *)h + (size_t)(b / 16) * (size_t)(ld / kf) * 1024;
      HIPCHK(launch_key_project(bf16, true, kp->Rc, kp->H, kp->Lc, hb, ld, nb, nullptr, v, hs));
    } else {
      HIPCHK(launch_key_project(bf16, false, kp->Rc, kp->H, kp->Lc,
                                (const char *)h + (size_t)b * ld * esz, ld, nb, nullptr, v, hs));
    }
    HIPCHK(launch_key_quant(v, nb, keys + b * PF_KEY_DIM, hs));
  }
  return PF_OK;
}

pf_status pf_key_encode(const pf_keyproj *kp, const void *h, int32_t dtype, int64_t ld, int64_t n,
                        int8_t *keys, pf_stream s) {
  if (!kp || (n > 0 && (!h || !keys))) return fail(PF_EINVAL, "pf_key_encode: null pointer");
  if (dtype != PF_DTYPE_F32 && dtype != PF_DTYPE_BF16)
    return fail(PF_EINVAL, "pf_key_encode: dtype %d", dtype);
  if (n < 0 || n > (1 << 20)) return fail(PF_EINVAL, "pf_key_encode: n %lld out of range", (long long)n);
  if (ld < kp->H) return fail(PF_EINVAL, "pf_key_encode: ld %lld < hidden %d", (long long)ld, kp->H);
  if (pf_status r = encode_rows(kp, dtype == PF_DTYPE_BF16, false, h, ld, n, keys, st(s))) return r;
  return ok();
}

pf_status pf_key_encode_static(const pf_keyproj *kp, const void *h, int32_t dtype, int64_t ld,
                               int64_t n, int8_t *keys, pf_stream s) {
  if (!kp || (n > 0 && (!h || !keys))) return fail(PF_EINVAL, "pf_key_encode_static: null pointer");
  if (dtype != PF_DTYPE_F32 && dtype != PF_DTYPE_BF16)
    return fail(PF_EINVAL, "pf_key_encode_static: dtype %d", dtype);
  if (n < 0 || n > (1 << 20))
    return fail(PF_EINVAL, "pf_key_encode_static: n %lld out of range [0, 2^20]", (long long)n);
  if (ld < kp->H)
    return fail(PF_EINVAL, "pf_key_encode_static: ld %lld < hidden %d", (long long)ld, kp->H);
  double *work = nullptr;
  int64_t elems = 0;
  HIPCHK(key_scratch(&work, &elems));
  if (elems < (int64_t)kKeyBatch * PF_KEY_DIM)
    return fail(PF_EINVAL, "pf_key_encode_static: static buffer of %lld values below one batch",
                (long long)elems);
  if (pf_status r = encode_rows(kp, dtype == PF_DTYPE_BF16, false, h, ld, n, keys, st(s), work))
    return r;
  return ok();
}

pf_status pf_store_attach_keys(pf_store *S, const int8_t *keys, pf_stream s) {
  if (!S) return fail(PF_EINVAL, "pf_store_attach_keys: null store");
  if (S->T > 0 && !keys) return fail(PF_EINVAL, "pf_store_attach_keys: null keys");
  if (S->log_state) return fail(PF_ESTATE, "pf_store_attach_keys: the store has an append region");
  const int64_t T = S->T;
  // entries p < b(p), grouped by token, ascending p within a token
  int32_t n_tok = 1;
  for (int64_t p = 0; p < T; ++p) n_tok = std::max(n_tok, S->h_tokens[p] + 1);
  std::vector<int32_t> off((size_t)n_tok + 1, 0);
  for (int64_t p = 0; p < T; ++p)
    if (p < S->h_last[p] && S->h_tokens[p] >= 0) off[(size_t)S->h_tokens[p] + 1]++;
  for (int32_t t = 0; t < n_tok; ++t) off[(size_t)t + 1] += off[t];
  const int64_t Ec = off[n_tok];
  std::vector<int32_t> fill(off.begin(), off.end() - 1), cpos(Ec), crem(Ec), cnk(Ec);
  for (int64_t p = 0; p < T; ++p) {
    if (!(p < S->h_last[p] && S->h_tokens[p] >= 0)) continue;
    const int32_t at = fill[S->h_tokens[p]]++;
    cpos[at] = (int32_t)p;
    crem[at] = S->h_last[p] - (int32_t)p;
    int32_t nk = 0;
    for (int j = 0; j < PF_KEY_DIM; ++j) nk += (int32_t)keys[p * PF_KEY_DIM + j] * keys[p * PF_KEY_DIM + j];
    cnk[at] = nk;
  }
  store_free_keys(S);
  pf_status r = PF_OK;
  if ((r = dev_alloc(&S->keys, T * PF_KEY_DIM, nullptr)) ||
      (r = dev_alloc(&S->tok_off, ((int64_t)n_tok + 1) * 4, nullptr)) ||
      (r = dev_alloc(&S->cpos, std::max<int64_t>(Ec, 1) * 4, nullptr)) ||
      (r = dev_alloc(&S->crem, std::max<int64_t>(Ec, 1) * 4, nullptr)) ||
      (r = dev_alloc(&S->cnk, std::max<int64_t>(Ec, 1) * 4, nullptr)) ||
      (r = dev_alloc(&S->cpart, (int64_t)kCosScanBlocks * PF_MAX_CAND * 16, nullptr)) ||
      (r = dev_alloc(&S->cpart_elig, (int64_t)kCosScanBlocks * 4, nullptr))) {
    store_free_keys(S);
    return r;
  }
  hipStream_t hs = st(s);
  hipError_t e = hipSuccess;
  if (T) e = hipMemcpyAsync(S->keys, keys, T * PF_KEY_DIM, hipMemcpyHostToDevice, hs);
  if (e == hipSuccess)
    e = hipMemcpyAsync(S->tok_off, off.data(), ((size_t)n_tok + 1) * 4, hipMemcpyHostToDevice, hs);
  if (e == hipSuccess && Ec) e = hipMemcpyAsync(S->cpos, cpos.data(), Ec * 4, hipMemcpyHostToDevice, hs);
  if (e == hipSuccess && Ec) e = hipMemcpyAsync(S->crem, crem.data(), Ec * 4, hipMemcpyHostToDevice, hs);
  if (e == hipSuccess && Ec) e = hipMemcpyAsync(S->cnk, cnk.data(), Ec * 4, hipMemcpyHostToDevice, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);  // host vectors die here
  if (e != hipSuccess) {
    store_free_keys(S);
    return fail(PF_EHIP, "pf_store_attach_keys: copy failed: %s", hipGetErrorString(e));
  }
  S->Ec = Ec;
  S->n_tok = n_tok;
  return ok();
}

pf_status pf_draft_lookup_cosine(const pf_store *S, const pf_context *ctx, const int8_t *q,
                                 int32_t k_max, int32_t tree, int32_t n_cand, int32_t max_nodes,
                                 pf_draft *draft, pf_stream s) {
  if (!S || !ctx || !ctx->tokens || !ctx->len || !draft || !q)
    return fail(PF_EINVAL, "pf_draft_lookup_cosine: null pointer");
  if (!S->tok_off) return fail(PF_ESTATE, "pf_draft_lookup_cosine: store has no keys");
  if (k_max < 0 || k_max > PF_MAX_DRAFT)
    return fail(PF_EINVAL, "pf_draft_lookup_cosine: k_max %d not in [0,%d]", k_max, PF_MAX_DRAFT);
  if (tree != 0 && tree != 1) return fail(PF_EINVAL, "pf_draft_lookup_cosine: tree must be 0 or 1");
  if (n_cand < 1 || n_cand > PF_MAX_CAND || (!tree && n_cand != 1))
    return fail(PF_EINVAL, "pf_draft_lookup_cosine: n_cand %d invalid", n_cand);
  if (tree && (max_nodes < 1 || max_nodes > PF_MAX_TREE_NODES))
    return fail(PF_EINVAL, "pf_draft_lookup_cosine: max_nodes %d not in [1,%d]", max_nodes,
                PF_MAX_TREE_NODES);
  if (ctx->host_bound < 1) return fail(PF_ESTATE, "pf_draft_lookup_cosine: empty context");
  CosArgs a;
  a.tokens = S->tokens;
  a.keys = S->keys;
  a.tok_off = S->tok_off;
  a.ent_pos = S->cpos;
  a.ent_rem = S->crem;
  a.ent_nk = S->cnk;
  a.n_tok = S->n_tok;
  a.ctx = ctx->tokens;
  a.ctx_len = ctx->len;
  a.q = q;
  a.k_max = k_max;
  a.tree = tree;
  a.n_cand = n_cand;
  a.max_nodes = tree ? max_nodes : PF_MAX_DRAFT;
  a.part = S->cpart;
  a.part_elig = S->cpart_elig;
  a.draft = draft;
  a.log_state = S->log_state;
  a.log_seq = S->log_seq;
  a.log_nk = S->log_nk;
  a.seq_end = S->seq_end;
  a.T_base = (int32_t)S->T;
  HIPCHK(launch_cos_lookup(a, st(s)));
  return ok();
}

// ---------------------------------------------------------------------------
// online memory update: append region, appends, compaction
// ---------------------------------------------------------------------------

pf_status pf_store_reserve(pf_store *S, int64_t capacity, int32_t max_seqs, pf_stream s) {
  if (!S) return fail(PF_EINVAL, "pf_store_reserve: null store");
  if (!S->tok_off) return fail(PF_ESTATE, "pf_store_reserve: attach keys first");
  if (S->log_state) return fail(PF_ESTATE, "pf_store_reserve: the store already has an append region");
  if (capacity < 1 || max_seqs < 1 || S->T + capacity >= ((int64_t)1 << 31) ||
      capacity > ((int64_t)1 << 28))
    return fail(PF_EINVAL, "pf_store_reserve: capacity %lld / sequences %d out of range",
                (long long)capacity, max_seqs);
  const int64_t T = S->T, N = T + capacity;
  int32_t *tokens = nullptr;
  int8_t *keys = nullptr;
  pf_status r = PF_OK;
  if ((r = dev_alloc(&tokens, N * 4, nullptr))) return r;
  if ((r = dev_alloc(&keys, N * PF_KEY_DIM, nullptr))) {
    (void)hipFree(tokens);
    return r;
  }
  hipStream_t hs = st(s);
  hipError_t e = hipSuccess;
  if (T) e = hipMemcpyAsync(tokens, S->tokens, T * 4, hipMemcpyDeviceToDevice, hs);
  if (e == hipSuccess && T)
    e = hipMemcpyAsync(keys, S->keys, T * PF_KEY_DIM, hipMemcpyDeviceToDevice, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  if (e != hipSuccess) {
    (void)hipFree(tokens);
    (void)hipFree(keys);
    return fail(PF_EHIP, "pf_store_reserve: copy failed: %s", hipGetErrorString(e));
  }
  (void)hipFree(S->tokens);
  (void)hipFree(S->keys);
  S->tokens = tokens;
  S->keys = keys;
  if ((r = dev_alloc(&S->log_state, 2 * 4, nullptr)) ||
      (r = dev_alloc(&S->log_seq, capacity * 4, nullptr)) ||
      (r = dev_alloc(&S->log_nk, capacity * 4, nullptr)) ||
      (r = dev_alloc(&S->seq_end, (int64_t)max_seqs * 4, nullptr)) ||
      (r = dev_alloc(&S->row_keys, (int64_t)kRowPad * PF_KEY_DIM, nullptr))) {
    store_free_log(S);
    return r;
  }
  e = hipMemsetAsync(S->log_state, 0, 2 * 4, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  if (e != hipSuccess) {
    store_free_log(S);
    return fail(PF_EHIP, "pf_store_reserve: %s", hipGetErrorString(e));
  }
  S->cap_log = (int32_t)capacity;
  S->max_log_seqs = max_seqs;
  return ok();
}

pf_status pf_store_begin_sequence(pf_store *S, pf_stream s) {
  if (!S) return fail(PF_EINVAL, "pf_store_begin_sequence: null store");
  if (!S->log_state) return fail(PF_ESTATE, "pf_store_begin_sequence: no append region");
  if (S->log_seqs_host >= S->max_log_seqs)
    return fail(PF_ECAPACITY, "pf_store_begin_sequence: %d sequences already opened",
                S->log_seqs_host);
  HIPCHK(launch_store_begin(S->log_state, S->seq_end, (int32_t)S->T, st(s)));
  ++S->log_seqs_host;
  return ok();
}

static pf_status append_check(const pf_store *S, int32_t n_max, const char *fn) {
  if (!S->log_state) return fail(PF_ESTATE, "%s: no append region", fn);
  if (S->log_seqs_host < 1) return fail(PF_ESTATE, "%s: no open sequence", fn);
  if (S->log_host_bound + n_max > S->cap_log)
    return fail(PF_ECAPACITY, "%s: appended bound %lld + %d > capacity %d", fn,
                (long long)S->log_host_bound, n_max, S->cap_log);
  return PF_OK;
}

pf_status pf_store_append(pf_store *S, const int32_t *tokens, const int8_t *keys,
                          const int32_t *n_dev, int32_t n_max, pf_stream s) {
  if (!S || !tokens || !keys || !n_dev) return fail(PF_EINVAL, "pf_store_append: null pointer");
  if (n_max < 0) return fail(PF_EINVAL, "pf_store_append: n_max < 0");
  if (pf_status r = append_check(S, n_max, "pf_store_append")) return r;
  if (((uintptr_t)keys & 15) != 0) return fail(PF_EINVAL, "pf_store_append: keys not 16-byte aligned");
  AppendArgs a{};
  a.tokens = S->tokens;
  a.keys = S->keys;
  a.log_state = S->log_state;
  a.log_seq = S->log_seq;
  a.log_nk = S->log_nk;
  a.seq_end = S->seq_end;
  a.T_base = (int32_t)S->T;
  a.cap = S->cap_log;
  a.tok_src = tokens;
  a.key_src = keys;
  a.n_dev = n_dev;
  a.n_max = n_max;
  a.res = nullptr;
  HIPCHK(launch_store_append(a, st(s)));
  S->log_host_bound += n_max;
  return ok();
}

pf_status pf_store_append_verified(pf_store *S, const pf_model *m, const pf_keyproj *kp,
                                   const pf_verify_result *res, pf_stream s) {
  if (!S || !m || !kp || !res) return fail(PF_EINVAL, "pf_store_append_verified: null pointer");
  const int rows = m->last_rows;
  if (rows < 1) return fail(PF_ESTATE, "pf_store_append_verified: no verify step yet");
  if (pf_status r = append_check(S, rows, "pf_store_append_verified")) return r;
  if (pf_status r = pf_verify_row_keys(m, kp, rows, S->row_keys, s)) return r;
  AppendArgs a{};
  a.tokens = S->tokens;
  a.keys = S->keys;
  a.log_state = S->log_state;
  a.log_seq = S->log_seq;
  a.log_nk = S->log_nk;
  a.seq_end = S->seq_end;
  a.T_base = (int32_t)S->T;
  a.cap = S->cap_log;
  a.key_src = S->row_keys;
  a.n_max = rows;
  a.res = res;
  HIPCHK(launch_store_append(a, st(s)));
  S->log_host_bound += rows;
  return ok();
}

pf_status pf_store_appended(pf_store *S, pf_stream s, int64_t *n_out) {
  if (!S || !n_out) return fail(PF_EINVAL, "pf_store_appended: null pointer");
  *n_out = 0;
  if (!S->log_state) return ok();
  int32_t st2[2];
  HIPCHK(hipMemcpyAsync(st2, S->log_state, 8, hipMemcpyDeviceToHost, st(s)));
  HIPCHK(hipStreamSynchronize(st(s)));
  S->log_host_bound = st2[0];
  *n_out = st2[0];
  return ok();
}

pf_status pf_store_compact(pf_store *S, int64_t budget, pf_stream s) {
  if (!S) return fail(PF_EINVAL, "pf_store_compact: null store");
  if (!S->tok_off) return fail(PF_ESTATE, "pf_store_compact: the store has no keys");
  if (budget < 0) return fail(PF_EINVAL, "pf_store_compact: budget < 0");
  hipStream_t hs = st(s);
  const int64_t T = S->T;
  int32_t lst[2] = {0, 0};
  std::vector<int32_t> ends;
  if (S->log_state) {
    HIPCHK(hipMemcpyAsync(lst, S->log_state, 8, hipMemcpyDeviceToHost, hs));
    HIPCHK(hipStreamSynchronize(hs));
    ends.resize((size_t)std::max(lst[1], 0));
    if (lst[1] > 0)
      HIPCHK(hipMemcpyAsync(ends.data(), S->seq_end, (size_t)lst[1] * 4, hipMemcpyDeviceToHost, hs));
  }
  const int64_t N = T + lst[0];
  std::vector<int32_t> tok((size_t)N);
  std::vector<int8_t> keys((size_t)N * PF_KEY_DIM);
  if (N) {
    HIPCHK(hipMemcpyAsync(tok.data(), S->tokens, N * 4, hipMemcpyDeviceToHost, hs));
    HIPCHK(hipMemcpyAsync(keys.data(), S->keys, N * PF_KEY_DIM, hipMemcpyDeviceToHost, hs));
  }
  HIPCHK(hipStreamSynchronize(hs));
  // sequences in store order: the built ones, then the appended ones
  std::vector<std::pair<int64_t, int64_t>> seqs;  // [start, end)
  for (int64_t p = 0; p < T;) {
    const int64_t e = (int64_t)S->h_last[p] + 1;
    seqs.push_back({p, e});
    p = e;
  }
  int64_t start = T;
  for (int32_t q = 0; q < lst[1]; ++q) {
    const int64_t e = (int64_t)ends[q] + 1;
    if (e > start) seqs.push_back({start, e});
    start = std::max(start, e);
  }
  // evict the oldest sequences while over the budget (0: no budget)
  int64_t total = 0;
  for (auto &q : seqs) total += q.second - q.first;
  size_t first = 0;
  while (budget > 0 && total > budget && first < seqs.size()) {
    total -= seqs[first].second - seqs[first].first;
    ++first;
  }
  std::vector<int32_t> ntok;
  std::vector<int8_t> nkeys;
  std::vector<int64_t> offs{0};
  for (size_t i = first; i < seqs.size(); ++i) {
    for (int64_t p = seqs[i].first; p < seqs[i].second; ++p) ntok.push_back(tok[(size_t)p]);
    nkeys.insert(nkeys.end(), keys.begin() + seqs[i].first * PF_KEY_DIM,
                 keys.begin() + seqs[i].second * PF_KEY_DIM);
    offs.push_back((int64_t)ntok.size());
  }
  pf_store *R = nullptr;
  if (pf_status r = pf_store_build(ntok.data(), offs.data(), (int64_t)offs.size() - 1, S->ngram, s, &R))
    return r;
  pf_status r = pf_store_attach_keys(R, nkeys.data(), s);
  if (r == PF_OK && S->log_state) r = pf_store_reserve(R, S->cap_log, S->max_log_seqs, s);
  if (r != PF_OK) {
    pf_store_destroy(R);
    return r;
  }
  std::swap(*S, *R);
  pf_store_destroy(R);
  return ok();
}

pf_status pf_draft_lookup(const pf_store *S, const pf_context *ctx, int32_t k_max, int32_t tree,
                          int32_t n_cand, int32_t max_nodes, pf_draft *draft, pf_stream s) {
  if (!S || !ctx || !ctx->tokens || !ctx->len || !draft)
    return fail(PF_EINVAL, "pf_draft_lookup: null pointer");
  if (k_max < 0 || k_max > PF_MAX_DRAFT)
    return fail(PF_EINVAL, "pf_draft_lookup: k_max %d not in [0,%d]", k_max, PF_MAX_DRAFT);
  if (tree != 0 && tree != 1) return fail(PF_EINVAL, "pf_draft_lookup: tree must be 0 or 1");
  if (n_cand < 1 || n_cand > PF_MAX_CAND || (!tree && n_cand != 1))
    return fail(PF_EINVAL, "pf_draft_lookup: n_cand %d invalid", n_cand);
  if (tree && (max_nodes < 1 || max_nodes > PF_MAX_TREE_NODES))
    return fail(PF_EINVAL, "pf_draft_lookup: max_nodes %d not in [1,%d]", max_nodes,
                PF_MAX_TREE_NODES);
  if (ctx->host_bound < 1) return fail(PF_ESTATE, "pf_draft_lookup: empty context");
  LookupArgs a;
  a.tokens = S->tokens;
  a.ent_pos = S->ent_pos;
  a.ent_rem = S->ent_rem;
  a.bucket_off = S->bucket_off;
  a.nb_log2 = S->nb_log2;
  a.ngram = S->ngram;
  a.ctx = ctx->tokens;
  a.ctx_len = ctx->len;
  a.k_max = k_max;
  a.tree = tree;
  a.n_cand = n_cand;
  a.max_nodes = tree ? max_nodes : PF_MAX_DRAFT;
  a.draft = draft;
  HIPCHK(launch_lookup(a, st(s)));
  return ok();
}

// ---------------------------------------------------------------------------
// model
// ---------------------------------------------------------------------------

pf_status pf_model_create(const pf_model_config *cfg, const pf_model_weights *w, pf_stream s,
                          pf_model **out) {
  if (!out) return fail(PF_EINVAL, "pf_model_create: null out");
  *out = nullptr;
  if (!cfg || !w) return fail(PF_EINVAL, "pf_model_create: null config or weights");
  const pf_model_config c = *cfg;
  if (c.dtype != PF_DTYPE_F32 && c.dtype != PF_DTYPE_BF16)
    return fail(PF_EINVAL, "pf_model_create: unknown dtype %d", c.dtype);
  if (c.n_layers < 1 || c.hidden < 16 || c.n_heads < 1 || c.n_kv_heads < 1 || c.ffn < 16 ||
      c.vocab < 16)
    return fail(PF_EINVAL, "pf_model_create: bad sizes");
  if (c.head_dim != 64 && c.head_dim != 128)
    return fail(PF_EUNSUPPORTED, "pf_model_create: head_dim %d not in {64,128}", c.head_dim);
  if (c.n_heads % c.n_kv_heads || c.n_heads / c.n_kv_heads > 8)
    return fail(PF_EUNSUPPORTED, "pf_model_create: n_heads/n_kv_heads must be an integer <= 8");
  if (c.hidden % 16 || c.ffn % 16 || c.vocab % 16)
    return fail(PF_EUNSUPPORTED, "pf_model_create: hidden, ffn, vocab must be multiples of 16");
  if (!(c.rms_eps >= 0) || !(c.rope_theta > 0)) return fail(PF_EINVAL, "pf_model_create: eps/theta");
  if (!w->embed || !w->lm_head || !w->wqkv || !w->wo || !w->wgu || !w->wd || !w->attn_norm ||
      !w->ffn_norm || !w->final_norm)
    return fail(PF_EINVAL, "pf_model_create: null weight pointer");

  pf_model *m = new pf_model();
  m->cfg = c;
  const bool bf = c.dtype == PF_DTYPE_BF16;
  m->esz = bf ? 2 : 4;
  const int kf = bf ? 32 : 16;
  const int64_t L = c.n_layers, H = c.hidden, q = (int64_t)c.n_heads * c.head_dim,
                kv = (int64_t)c.n_kv_heads * c.head_dim, F = c.ffn, V = c.vocab;
  m->pqkv = geom(q + 2 * kv, H, kf);
  m->po = geom(H, q, kf);
  m->pgu = geom(2 * F, H, kf);
  m->pd = geom(H, F, kf);
  m->plm = geom(V, H, kf);
  if (m->plm.bytes() >= ((int64_t)1 << 31) || m->pgu.bytes() >= ((int64_t)1 << 31)) {
    model_free(m);
    return fail(PF_EUNSUPPORTED, "pf_model_create: a packed matrix exceeds 2 GiB");
  }
  int64_t tot = 0;
  pf_status r = PF_OK;
#define ALLOC(ptr, bytes)                          \
  if ((r = dev_alloc(&(ptr), (bytes), &tot))) {    \
    model_free(m);                                 \
    return r;                                      \
  }
  ALLOC(m->wqkv, m->pqkv.bytes() * L);
  ALLOC(m->wo, m->po.bytes() * L);
  ALLOC(m->wgu, m->pgu.bytes() * L);
  ALLOC(m->wd, m->pd.bytes() * L);
  ALLOC(m->lm, m->plm.bytes());
  ALLOC(m->embed, V * H * m->esz);
  ALLOC(m->attn_norm, L * H * 4);
  ALLOC(m->ffn_norm, L * H * 4);
  ALLOC(m->final_norm, H * 4);
  ALLOC(m->inv_freq, (c.head_dim / 2) * 8);
  // step work buffers
  const int64_t Hp = roundup(H, kf), qp = roundup(q, kf), Fp = roundup(F, kf);
  int64_t part = 0;
  {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        cus > 0)
      m->wave_slots = 4 * cus;
  }
  const Packed *pg[] = {&m->pqkv, &m->po, &m->pd};
  for (const Packed *p : pg) {
    int64_t nb = partial_blocks(*p);
    int64_t e = (int64_t)splits_for(nb, p->KFr, m->wave_slots / 4) * kRowPad * p->NT * 16;
    if (e > part) part = e;
  }
  m->part_elems = part;
  m->apart_rows = (int64_t)c.n_heads * kMaxSplitsAttn * kRowPad;
  m->amax_elems = ((m->plm.NT + 3) / 4) * kRowPad;
  ALLOC(m->x, kRowPad * H * 4);
  ALLOC(m->xn, kRowPad * Hp * m->esz);
  ALLOC(m->ssq, (int64_t)kRowPad * kMaxNormSlices * 4);
  ALLOC(m->qb, kRowPad * q * m->esz);
  ALLOC(m->attn, kRowPad * qp * m->esz);
  ALLOC(m->act, kRowPad * Fp * m->esz);
  ALLOC(m->part, part * 4);
  ALLOC(m->apart_o, m->apart_rows * c.head_dim * 4);
  ALLOC(m->apart_ml, m->apart_rows * 2 * 4);
  ALLOC(m->amax, m->amax_elems * (int64_t)sizeof(ArgmaxPart));
  ALLOC(m->rope, kRowPad * c.head_dim * 4);
  ALLOC(m->rowinfo, kRowPad * 4 * 4 + kRowPad * 8);
  ALLOC(m->pred, 2 * kRowPad * 4);
  ALLOC(m->flags, 64);
#undef ALLOC
  m->bytes = tot;

  hipStream_t hs = st(s);
  hipError_t e = hipSuccess;
  void *zero[] = {m->x, m->xn, m->qb, m->attn, m->act, m->ssq};
  int64_t zb[] = {kRowPad * H * 4, kRowPad * Hp * m->esz, kRowPad * q * m->esz,
                  kRowPad * qp * m->esz, kRowPad * Fp * m->esz, (int64_t)kRowPad * kMaxNormSlices * 4};
  for (int i = 0; i < 6 && e == hipSuccess; ++i) e = hipMemsetAsync(zero[i], 0, zb[i], hs);
  if (e == hipSuccess) e = launch_pack(w->wqkv, q + 2 * kv, H, L, (q + 2 * kv) * H, bf, m->pqkv, m->wqkv, hs,
                                           c.head_dim);
  if (e == hipSuccess) e = launch_pack(w->wo, H, q, L, H * q, bf, m->po, m->wo, hs);
  if (e == hipSuccess) e = launch_pack(w->wgu, 2 * F, H, L, 2 * F * H, bf, m->pgu, m->wgu, hs);
  if (e == hipSuccess) e = launch_pack(w->wd, H, F, L, H * F, bf, m->pd, m->wd, hs);
  if (e == hipSuccess) e = launch_pack(w->lm_head, V, H, 1, V * H, bf, m->plm, m->lm, hs);
  if (e == hipSuccess) e = hipMemcpyAsync(m->embed, w->embed, V * H * m->esz, hipMemcpyDeviceToDevice, hs);
  if (e == hipSuccess) e = hipMemcpyAsync(m->attn_norm, w->attn_norm, L * H * 4, hipMemcpyDeviceToDevice, hs);
  if (e == hipSuccess) e = hipMemcpyAsync(m->ffn_norm, w->ffn_norm, L * H * 4, hipMemcpyDeviceToDevice, hs);
  if (e == hipSuccess) e = hipMemcpyAsync(m->final_norm, w->final_norm, H * 4, hipMemcpyDeviceToDevice, hs);
  std::vector<double> invf(c.head_dim / 2);
  for (int i = 0; i < c.head_dim / 2; ++i)
    invf[i] = std::pow(c.rope_theta, -2.0 * (double)i / (double)c.head_dim);
  if (e == hipSuccess)
    e = hipMemcpyAsync(m->inv_freq, invf.data(), invf.size() * 8, hipMemcpyHostToDevice, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  if (e != hipSuccess) {
    model_free(m);
    return fail(PF_EHIP, "pf_model_create: %s", hipGetErrorString(e));
  }
  *out = m;
  return ok();
}

void pf_model_destroy(pf_model *m) { model_free(m); }
int64_t pf_model_bytes(const pf_model *m) { return m ? m->bytes : -1; }

// ---------------------------------------------------------------------------
// KV cache
// ---------------------------------------------------------------------------

int64_t pf_kv_bytes(const pf_model *m, int64_t capacity) {
  if (!m || capacity < 0) return -1;
  return (int64_t)m->cfg.n_layers * 2 * m->cfg.n_kv_heads * capacity * m->cfg.head_dim * m->esz;
}

pf_status pf_kv_init(pf_kv_cache *kv, const pf_model *m, void *data, int32_t *len_dev,
                     int64_t capacity) {
  if (!kv || !m || !data || !len_dev) return fail(PF_EINVAL, "pf_kv_init: null pointer");
  if (capacity < 64 || capacity % 64 || capacity > INT32_MAX)
    return fail(PF_EINVAL, "pf_kv_init: capacity %lld must be a positive multiple of 64",
                (long long)capacity);
  kv->data = data;
  kv->len = len_dev;
  kv->capacity = capacity;
  kv->host_bound = 0;
  kv->n_layers = m->cfg.n_layers;
  kv->n_kv_heads = m->cfg.n_kv_heads;
  kv->head_dim = m->cfg.head_dim;
  kv->dtype = m->cfg.dtype;
  kv->pending = 0;
  kv->pending_tree = 0;
  return ok();
}

static pf_status kv_check(const pf_kv_cache *kv, const char *fn) {
  if (!kv || !kv->data || !kv->len) return fail(PF_EINVAL, "%s: null cache", fn);
  if (kv->capacity < 64 || kv->capacity % 64) return fail(PF_EINVAL, "%s: bad capacity", fn);
  return PF_OK;
}

pf_status pf_kv_import(pf_kv_cache *kv, const void *src, int64_t n, pf_stream s) {
  if (pf_status r = kv_check(kv, "pf_kv_import")) return r;
  if (!src && n > 0) return fail(PF_EINVAL, "pf_kv_import: null source");
  if (n < 0 || n > kv->capacity) return fail(PF_ECAPACITY, "pf_kv_import: %lld rows", (long long)n);
  if (n > 0)
    HIPCHK(launch_kv_copy(kv->dtype == PF_DTYPE_BF16, true, kv->data, src, nullptr, kv->n_layers,
                          kv->n_kv_heads, kv->head_dim, kv->capacity, 0, n, st(s)));
  HIPCHK(launch_set_int(kv->len, (int32_t)n, st(s)));
  kv->host_bound = n;
  kv->pending = 0;
  return ok();
}

pf_status pf_kv_export(const pf_kv_cache *kv, void *dst, int64_t start, int64_t n, pf_stream s) {
  if (pf_status r = kv_check(kv, "pf_kv_export")) return r;
  if (!dst || start < 0 || n < 0 || start + n > kv->capacity)
    return fail(PF_EINVAL, "pf_kv_export: bad range");
  if (n > 0)
    HIPCHK(launch_kv_copy(kv->dtype == PF_DTYPE_BF16, false, kv->data, nullptr, dst, kv->n_layers,
                          kv->n_kv_heads, kv->head_dim, kv->capacity, start, n, st(s)));
  return ok();
}

pf_status pf_kv_set_len(pf_kv_cache *kv, int64_t len, pf_stream s) {
  if (pf_status r = kv_check(kv, "pf_kv_set_len")) return r;
  if (len < 0 || len > kv->capacity) return fail(PF_ECAPACITY, "pf_kv_set_len: %lld", (long long)len);
  HIPCHK(launch_set_int(kv->len, (int32_t)len, st(s)));
  kv->host_bound = len;
  kv->pending = 0;
  return ok();
}

pf_status pf_kv_sync_bound(pf_kv_cache *kv, pf_stream s) {
  if (pf_status r = kv_check(kv, "pf_kv_sync_bound")) return r;
  int32_t v = 0;
  HIPCHK(hipMemcpyAsync(&v, kv->len, 4, hipMemcpyDeviceToHost, st(s)));
  HIPCHK(hipStreamSynchronize(st(s)));
  kv->host_bound = v;
  kv->pending = 0;
  return ok();
}

// ---------------------------------------------------------------------------
// verify step
// ---------------------------------------------------------------------------

static pf_status model_kv_match(const pf_model *m, const pf_kv_cache *kv, const char *fn) {
  if (kv->n_layers != m->cfg.n_layers || kv->n_kv_heads != m->cfg.n_kv_heads ||
      kv->head_dim != m->cfg.head_dim || kv->dtype != m->cfg.dtype)
    return fail(PF_EINVAL, "%s: cache does not match the model", fn);
  return PF_OK;
}

// Launch one kernel of the step, tagged with its profiling kind; with
// only_kind >= 0 the launches of every other kind are skipped.
#define PROF(k, call)                                                            \
  do {                                                                           \
    if (prof) prof->cur = (k);                                                   \
    if (only_kind < 0 || only_kind == (k)) HIPCHK(call);                         \
  } while (0)

// Keys per attention key range. Ranges start at multiples of this length,
// and the length depends on the row count of the step only through the key
// bound's band, so a query row is reduced over the same ranges in the same
// order whatever rows share its step: a verify row reproduces, bit for bit,
// the single-row step at its position (greedy decoding), except when the two
// steps' key bounds fall in different bands. The length is five 32-key (bf16;
// 16-key fp32) chunks per range (measured best: shorter ranges add splits and
// waves, longer ones leave the kernel's straight-line part), doubled until
// the ranges of one query row per head fit the resident waves (one per SIMD)
// and the combine's 64 lanes.
static int attn_range_keys(int64_t keys_max, bool bf, int nq, int wave_slots) {
  int max_splits = wave_slots / nq;
  if (max_splits > kMaxSplitsAttn) max_splits = kMaxSplitsAttn;
  if (max_splits < 1) max_splits = 1;
  int64_t chunk = 5 * (bf ? 32 : 16);
  while ((keys_max + chunk - 1) / chunk > max_splits) chunk *= 2;
  return (int)chunk;
}

// Grouped attention (bf16, head_dim 128): keys per range, a multiple of the
// 64-key phase, sized so that one KV head has at most T ranges, T = the
// resident blocks (two per compute unit) over four row groups per KV head,
// at most the combine's 64. The length depends on the row count only
// through the key bound (ceil(keys / (64 T)) changes every 64 T keys), so a
// verify row reproduces the single-row step at its position bit for bit
// unless the two key bounds straddle such a step.
static int attn_gq_range_keys(int64_t keys_max, int nkv, int cus) {
  int target = 2 * cus / (4 * (nkv > 0 ? nkv : 1));
  if (target > kMaxSplitsAttn) target = kMaxSplitsAttn;
  if (target < 1) target = 1;
  const int64_t per = (keys_max + target - 1) / target;
  // whole 64-key phases of the kernel: a range that ends half way through a
  // phase costs the phase anyway (3B: 96 -> 128 keys, 43 -> 33 ranges, 264 ->
  // 216 blocks; 3B tree 616 -> 504 blocks, within the resident 512)
  return (int)(((per + 63) / 64) * 64);
}

// Probabilities enter the grouped attention's value product as two bf16
// terms (the rounding residue of the first as the second).
constexpr bool kAttnHiLo = true;

static pf_status verify_impl(pf_model *m, pf_kv_cache *kv, const pf_draft *draft, int32_t rows,
                             int32_t tree, float *logits, pf_verify_result *res, pf_stream s,
                             Prof *prof, float *resid = nullptr, int only_kind = -1) {
  if (!m || !draft || !res) return fail(PF_EINVAL, "pf_verify_step: null pointer");
  if (pf_status r = kv_check(kv, "pf_verify_step")) return r;
  if (pf_status r = model_kv_match(m, kv, "pf_verify_step")) return r;
  if (tree != 0 && tree != 1) return fail(PF_EINVAL, "pf_verify_step: tree must be 0 or 1");
  if (rows < 1 || rows > (tree ? 64 : kMaxRows))
    return fail(PF_EINVAL, "pf_verify_step: rows %d out of range", rows);
  if (kv->host_bound < 0 || kv->host_bound + rows > kv->capacity)
    return fail(PF_ECAPACITY, "pf_verify_step: cache bound %lld + %d rows > capacity %lld",
                (long long)kv->host_bound, rows, (long long)kv->capacity);
  const pf_model_config &c = m->cfg;
  const bool bf = is_bf16(m);
  const int kf = frag_k_of(m);
  const int L = c.n_layers, H = c.hidden, hd = c.head_dim, nq = c.n_heads, nkv = c.n_kv_heads;
  const int64_t q = (int64_t)nq * hd, kvd = (int64_t)nkv * hd, F = c.ffn, V = c.vocab;
  const int64_t Hp = roundup(H, kf), qp = roundup(q, kf), Fp = roundup(F, kf);
  const int M = rows, MT = (rows + 15) / 16;
  hipStream_t hs = st(s);
  TimerScope timer_scope(prof);
  const float eps = (float)c.rms_eps;
  uint64_t *rowmask = (uint64_t *)(m->rowinfo + kRowPad * 4);

  m->last_rows = rows;
  StepArgs sa;
  sa.draft = draft;
  sa.res = res;
  sa.kv_len = kv->len;
  sa.rows = rows;
  sa.tree = tree;
  sa.L = L; sa.H = H; sa.nq = nq; sa.nkv = nkv; sa.hd = hd; sa.F = (int)F; sa.V = (int)V;
  sa.eps = eps;
  sa.inv_freq = m->inv_freq;
  sa.rowinfo = m->rowinfo;
  sa.rowmask = rowmask;
  sa.rope = m->rope;
  PROF(0, launch_prep(sa, hs));
  // the norms inside the layer stack leave their scale to the next projection
  // (x * gain in xn, sums of squares in ssq); the final norm, whose rows are
  // also read by the retrieval keys, writes normalised rows
  const int nss = norm_slices(H);
  RowScale rsc{m->ssq, nss, H, eps};
  PROF(0, launch_embed_norm(bf, m->embed, m->rowinfo, M, H, m->attn_norm, eps, m->x, m->xn, Hp,
                            true, m->ssq, hs));
  if (resid && only_kind < 0) HIPCHK(launch_copy_rows(m->x, M, H, resid, hs));

  // attention geometry: key ranges over P + rows keys (P <= host bound)
  const int64_t keys_max = kv->host_bound + rows;
  const bool gq = attn_gq_supported(bf, hd);
  const int chunk = gq ? attn_gq_range_keys(keys_max, nkv, m->wave_slots / 4)
                       : attn_range_keys(keys_max, bf, nq, m->wave_slots);
  const int n_splits = (int)((keys_max + chunk - 1) / chunk);
  // rows beyond one wave's tiles take more waves per range; those waves then
  // reduce several consecutive ranges each, to stay within the resident waves
  const int row_groups = (MT + attn_tiles_per_wave(MT) - 1) / attn_tiles_per_wave(MT);
  const int64_t slots = (int64_t)m->wave_slots * attn_waves_per_simd(MT);
  const int per_wave = (int)(((int64_t)nq * row_groups * n_splits + slots - 1) / slots);

  for (int l = 0; l < L; ++l) {
    // QKV projection, RoPE and the KV append in one kernel
    QkvArgs qa{};
    qa.W = (const char *)m->wqkv + (int64_t)l * m->pqkv.bytes();
    qa.W_bytes = m->pqkv.bytes();
    qa.KFr = m->pqkv.KFr;
    qa.X = m->xn;
    qa.ldx = Hp;
    qa.rs = rsc;
    if (l == 0) qa.rs.nss = 1;  // the embedding norm's one sum per row
    qa.M = M;
    qa.nq = nq;
    qa.nkv = nkv;
    qa.hd = hd;
    qa.rope = m->rope;
    qa.kv_len = kv->len;
    qa.qbuf = m->qb;
    qa.ldq = q;
    qa.cache = kv->data;
    qa.layer = l;
    qa.cap = kv->capacity;
    PROF(1, launch_gemm_qkv(bf, MT, qa, m->wave_slots / 4, hs));
    // attention
    AttnArgs at{};
    at.q = m->qb;
    at.ldq = q;
    at.cache = kv->data;
    at.plane = kv->capacity * hd;
    at.cap = kv->capacity;
    at.layer = l;
    at.n_kv = nkv;
    at.group = nq / nkv;
    at.head_dim = hd;
    at.M = M;
    at.rowpad = kRowPad;
    at.kv_len = kv->len;
    at.n_splits = n_splits;
    at.chunk_keys = chunk;
    at.per_wave = per_wave;
    at.keys_bound = (int)keys_max;
    at.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)hd));
    at.tree = tree;
    at.anc = rowmask;
    at.part_o = m->apart_o;
    at.part_ml = m->apart_ml;
    at.out = m->attn;
    at.ldout = qp;
    at.out_packed = 1;
    PROF(3, gq ? launch_attn_gq(at, kAttnHiLo, hs) : launch_attn(bf, MT, at, hs));
    // output projection + residual + FFN norm
    GemmArgs go{};
    go.W = (const char *)m->wo + (int64_t)l * m->po.bytes();
    go.W_bytes = m->po.bytes();
    go.KFr = m->po.KFr;
    go.NTtot = m->po.NT;
    go.X = m->attn;
    go.ldx = qp;
    go.M = M;
    go.splits = splits_for(partial_blocks(m->po), m->po.KFr, m->wave_slots / 4);
    go.out = m->part;
    go.ldo = H;
    PROF(4, launch_gemm(bf, EPI_PARTIAL, MT, go, m->wave_slots / 4, hs));
    PROF(5, launch_residual_norm_deferred(bf, m->part, go.splits, kRowPad, M, H, H,
                                         m->ffn_norm + (int64_t)l * H, m->x, m->xn, Hp, m->ssq, hs));
    // gate/up + SwiGLU
    GemmArgs gg{};
    gg.W = (const char *)m->wgu + (int64_t)l * m->pgu.bytes();
    gg.W_bytes = m->pgu.bytes();
    gg.KFr = m->pgu.KFr;
    gg.NTtot = m->pgu.NT;
    gg.X = m->xn;
    gg.ldx = Hp;
    gg.M = M;
    gg.splits = 1;
    gg.act = m->act;
    gg.ldact = Fp;
    gg.up_tile_off = F / 16;
    gg.rs = rsc;
    PROF(6, launch_gemm(bf, EPI_SWIGLU, MT, gg, m->wave_slots / 4, hs));
    // down projection + residual + next norm
    GemmArgs gd{};
    gd.W = (const char *)m->wd + (int64_t)l * m->pd.bytes();
    gd.W_bytes = m->pd.bytes();
    gd.KFr = m->pd.KFr;
    gd.NTtot = m->pd.NT;
    gd.X = m->act;
    gd.ldx = Fp;
    gd.M = M;
    gd.splits = splits_for(partial_blocks(m->pd), m->pd.KFr, m->wave_slots / 4);
    gd.out = m->part;
    gd.ldo = H;
    PROF(7, launch_gemm(bf, EPI_PARTIAL, MT, gd, m->wave_slots / 4, hs));
    if (l + 1 < L)
      PROF(5, launch_residual_norm_deferred(bf, m->part, gd.splits, kRowPad, M, H, H,
                                           m->attn_norm + (int64_t)(l + 1) * H, m->x, m->xn, Hp,
                                           m->ssq, hs));
    else
      PROF(5, launch_residual_norm(bf, m->part, gd.splits, kRowPad, M, H, H, m->final_norm, eps,
                                  m->x, m->xn, Hp, true, hs));
    if (resid && only_kind < 0)
      HIPCHK(launch_copy_rows(m->x, M, H, resid + (int64_t)(l + 1) * M * H, hs));
  }
  // lm_head + greedy argmax partials
  GemmArgs gl{};
  gl.W = m->lm;
  gl.W_bytes = m->plm.bytes();
  gl.KFr = m->plm.KFr;
  gl.NTtot = m->plm.NT;
  gl.X = m->xn;
  gl.ldx = Hp;
  gl.M = M;
  gl.splits = 1;
  gl.amax = m->amax;
  gl.logits = logits;
  gl.ldlog = V;
  PROF(8, launch_gemm(bf, EPI_ARGMAX, MT, gl, m->wave_slots / 4, hs));
  const int nparts = (int)((m->plm.NT + gemm_tiles_per_block(EPI_ARGMAX, MT) - 1) /
                           gemm_tiles_per_block(EPI_ARGMAX, MT));
  PROF(9, launch_argmax_accept(m->amax, nparts, rows, tree, draft, m->pred, res, hs));
  if (only_kind < 0) {
    kv->pending = rows;
    kv->pending_tree = tree;
  }
  return ok();
}

pf_status pf_verify_step(pf_model *m, pf_kv_cache *kv, const pf_draft *draft, int32_t rows,
                         int32_t tree, float *logits, pf_verify_result *res, pf_stream s) {
  return verify_impl(m, kv, draft, rows, tree, logits, res, s, nullptr);
}

pf_status pf_verify_kernel_repeat(pf_model *m, pf_kv_cache *kv, const pf_draft *draft,
                                  int32_t rows, int32_t tree, int32_t kind,
                                  pf_verify_result *res, pf_stream s) {
  if (kind < 0 || kind >= PF_PROF_MARKER)
    return fail(PF_EINVAL, "pf_verify_kernel_repeat: kind %d out of range", kind);
  return verify_impl(m, kv, draft, rows, tree, nullptr, res, s, nullptr, nullptr, kind);
}

pf_status pf_read_stream(const void *buf, int64_t bytes, uint32_t *sink, pf_stream s) {
  if (!buf || !sink) return fail(PF_EINVAL, "pf_read_stream: null pointer");
  if (((uintptr_t)buf & 15) || bytes <= 0 || bytes % 16384 || bytes >= ((int64_t)1 << 31))
    return fail(PF_EINVAL, "pf_read_stream: %lld bytes at %p (16-byte aligned multiple of 16 KiB, "
                "below 2 GiB)", (long long)bytes, buf);
  int dev = 0, cus = 0;
  HIPCHK(hipGetDevice(&dev));
  HIPCHK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  HIPCHK(launch_read_stream(buf, (uint32_t)bytes, cus, sink, st(s)));
  return ok();
}

pf_status pf_verify_step_trace(pf_model *m, pf_kv_cache *kv, const pf_draft *draft, int32_t rows,
                               int32_t tree, float *logits, pf_verify_result *res, float *resid,
                               pf_stream s) {
  if (!resid) return fail(PF_EINVAL, "pf_verify_step_trace: null residual buffer");
  return verify_impl(m, kv, draft, rows, tree, logits, res, s, nullptr, resid);
}

pf_status pf_verify_step_profiled(pf_model *m, pf_kv_cache *kv, const pf_draft *draft,
                                  int32_t rows, int32_t tree, float *logits, pf_verify_result *res,
                                  pf_stream s, double *ms_out, int32_t *count_out) {
  if (!ms_out || !count_out) return fail(PF_EINVAL, "pf_verify_step_profiled: null outputs");
  // Hold the stream until the whole step is enqueued, so that the timed
  // kernels run back to back as in a graph replay rather than waiting on
  // host submission (the hold is released on every path, and is bounded by
  // 500 ms of wall clock on the device in any case).
  int dev = 0, rate_khz = 0;
  HIPCHK(hipGetDevice(&dev));
  HIPCHK(hipDeviceGetAttribute(&rate_khz, hipDeviceAttributeWallClockRate, dev));
  int32_t *flag = nullptr;
  HIPCHK(hipHostMalloc((void **)&flag, 64, hipHostMallocCoherent));
  struct Release {
    int32_t *f;
    hipStream_t s;
    ~Release() {
      __atomic_store_n(f, 1, __ATOMIC_SEQ_CST);
      (void)hipStreamSynchronize(s);
      (void)hipHostFree(f);
    }
  } release{flag, st(s)};
  __atomic_store_n(flag, 0, __ATOMIC_SEQ_CST);
  HIPCHK(launch_hold(flag, (uint64_t)rate_khz * 500, st(s)));
  Prof prof;
  // the cost of an event pair itself: pairs recorded with no work between
  constexpr int kMarkerPairs = 16;
  prof.cur = PF_PROF_MARKER;
  for (int i = 0; i < kMarkerPairs; ++i) {
    hipEvent_t e0, e1;
    if (!prof.events(&e0, &e1)) break;
    HIPCHK(hipEventRecord(e0, st(s)));
    HIPCHK(hipEventRecord(e1, st(s)));
  }
  pf_status r = verify_impl(m, kv, draft, rows, tree, logits, res, s, &prof);
  __atomic_store_n(flag, 1, __ATOMIC_SEQ_CST);
  if (r != PF_OK) return r;
  HIPCHK(prof.err);
  HIPCHK(hipStreamSynchronize(st(s)));
  std::vector<float> ms(prof.kind.size());
  double marker = 0.0;
  int n_marker = 0;
  for (size_t i = 0; i < prof.kind.size(); ++i) {
    HIPCHK(hipEventElapsedTime(&ms[i], prof.ev[2 * i], prof.ev[2 * i + 1]));
    if (prof.kind[i] == PF_PROF_MARKER) {
      marker += ms[i];
      ++n_marker;
    }
  }
  const double per_pair = n_marker ? marker / n_marker : 0.0;
  for (size_t i = 0; i < prof.kind.size(); ++i) {
    const int k = prof.kind[i];
    if (k < 0 || k >= PF_PROF_KINDS) continue;
    ms_out[k] += k == PF_PROF_MARKER ? ms[i] : std::max(0.0, ms[i] - per_pair);
    count_out[k] += 1;
  }
  return ok();
}

pf_status pf_verify_query_key(const pf_model *m, const pf_keyproj *kp, const pf_verify_result *res,
                              int8_t *q, pf_stream s) {
  if (!m || !kp || !res || !q) return fail(PF_EINVAL, "pf_verify_query_key: null pointer");
  if (kp->H != m->cfg.hidden)
    return fail(PF_EINVAL, "pf_verify_query_key: projection hidden %d != model hidden %d", kp->H,
                m->cfg.hidden);
  const bool bf = is_bf16(m);
  const int64_t Hp = roundup(m->cfg.hidden, frag_k_of(m));
  hipStream_t hs = st(s);
  HIPCHK(launch_key_project(bf, true, kp->Rc, kp->H, kp->Lc, m->xn, Hp, 1, res, kp->v, hs));
  HIPCHK(launch_key_quant(kp->v, 1, q, hs));
  return ok();
}

pf_status pf_verify_row_keys(const pf_model *m, const pf_keyproj *kp, int32_t rows, int8_t *keys,
                             pf_stream s) {
  if (!m || !kp || !keys) return fail(PF_EINVAL, "pf_verify_row_keys: null pointer");
  if (kp->H != m->cfg.hidden)
    return fail(PF_EINVAL, "pf_verify_row_keys: projection hidden %d != model hidden %d", kp->H,
                m->cfg.hidden);
  if (rows < 1 || rows > kMaxRows)
    return fail(PF_EINVAL, "pf_verify_row_keys: rows %d out of range", rows);
  const int64_t Hp = roundup(m->cfg.hidden, frag_k_of(m));
  if (pf_status r = encode_rows(kp, is_bf16(m), true, m->xn, Hp, rows, keys, st(s))) return r;
  return ok();
}

pf_status pf_kv_commit(pf_kv_cache *kv, const pf_verify_result *res, pf_context *ctx,
                       pf_stream s) {
  if (!res) return fail(PF_EINVAL, "pf_kv_commit: null result");
  if (pf_status r = kv_check(kv, "pf_kv_commit")) return r;
  if (kv->pending <= 0) return fail(PF_ESTATE, "pf_kv_commit: no verify step to commit");
  if (ctx && (!ctx->tokens || !ctx->len)) return fail(PF_EINVAL, "pf_kv_commit: bad context");
  if (ctx && ctx->host_bound + kv->pending > ctx->capacity)
    return fail(PF_ECAPACITY, "pf_kv_commit: context bound %lld + %d > capacity %lld",
                (long long)ctx->host_bound, kv->pending, (long long)ctx->capacity);
  HIPCHK(launch_commit(kv->dtype == PF_DTYPE_BF16, res, kv->data, kv->n_layers, kv->n_kv_heads,
                       kv->head_dim, kv->capacity, kv->pending_tree, kv->len,
                       ctx ? ctx->tokens : nullptr,
                       ctx ? ctx->len : nullptr, ctx ? ctx->capacity : 0, st(s)));
  kv->host_bound += kv->pending;
  if (ctx) ctx->host_bound += kv->pending;
  kv->pending = 0;
  kv->pending_tree = 0;
  return ok();
}

pf_status pf_kv_carry(pf_kv_cache *kv, const pf_model *m, int32_t n_spans, const int64_t *src,
                      const int64_t *dst, const int64_t *len, pf_stream s) {
  if (!m) return fail(PF_EINVAL, "pf_kv_carry: null model");
  if (pf_status r = kv_check(kv, "pf_kv_carry")) return r;
  if (pf_status r = model_kv_match(m, kv, "pf_kv_carry")) return r;
  if (kv->pending) return fail(PF_ESTATE, "pf_kv_carry: a verify step is not committed");
  if (n_spans < 0 || (n_spans > 0 && (!src || !dst || !len)))
    return fail(PF_EINVAL, "pf_kv_carry: bad span arrays");
  if (kv->head_dim / 2 > kCarryMaxHalf)
    return fail(PF_EUNSUPPORTED, "pf_kv_carry: head_dim %d too large", kv->head_dim);
  if (kv->capacity * kv->head_dim * (kv->dtype == PF_DTYPE_BF16 ? 2 : 4) >= ((int64_t)1 << 31))
    return fail(PF_EUNSUPPORTED, "pf_kv_carry: one cache plane must stay below 2 GiB");
  for (int32_t i = 0; i < n_spans; ++i) {
    if (len[i] < 0 || src[i] < 0 || dst[i] < 0 || len[i] > kv->capacity ||
        src[i] > kv->capacity - len[i] || dst[i] > kv->capacity - len[i])
      return fail(PF_EINVAL, "pf_kv_carry: span %d (src %lld, dst %lld, len %lld) outside capacity %lld",
                  i, (long long)src[i], (long long)dst[i], (long long)len[i],
                  (long long)kv->capacity);
  }
  CarryArgs a{};
  a.cache = kv->data;
  a.L = kv->n_layers;
  a.nkv = kv->n_kv_heads;
  a.hd = kv->head_dim;
  a.cap = kv->capacity;
  a.inv_freq = m->inv_freq;
  const bool bf = kv->dtype == PF_DTYPE_BF16;
  for (int32_t i = 0; i < n_spans; ++i) {
    const int64_t d = dst[i] - src[i], n = len[i];
    if (d == 0 || n == 0) continue;  // rotation by zero: nothing moves
    // pieces whose source and destination do not overlap, in the order that
    // reads every source slot before it is overwritten (memmove)
    const int64_t piece = std::min<int64_t>(n, d > 0 ? d : -d);
    const int64_t pieces = (n + piece - 1) / piece;
    for (int64_t k = 0; k < pieces; ++k) {
      const int64_t j = d > 0 ? pieces - 1 - k : k;  // right shift: last piece first
      const int64_t off = j * piece;
      a.src = src[i] + off;
      a.dst = dst[i] + off;
      a.n = (int)std::min<int64_t>(piece, n - off);
      a.delta = d;
      HIPCHK(launch_kv_carry(bf, a, st(s)));
    }
  }
  return ok();
}

constexpr int kPrefillSplits = 8;

// bf16 chunks take the LDS-staged 32x32 kernel; fp32 the register-fed one
static hipError_t prefill_gemm(bool bf, int epi, const BigGemmArgs &a, hipStream_t s) {
  return bf ? launch_gemm_pre(epi, a, s) : launch_gemm_big(false, epi, a, s);
}

// split-K factor of a bf16 prefill GEMM with a narrow output: about one
// block (256 W rows x 128 X rows) per CU, at least eight stages (16
// fragments) a split
constexpr int kPreSplitsMax = 8;
static int prefill_splits(int64_t n_tiles16, int64_t rows_pad, int64_t KFr, int cus) {
  const int64_t blocks = ((n_tiles16 + 15) / 16) * (rows_pad / 128);
  int64_t sp = cus / blocks;
  const int64_t cap = std::min<int64_t>(kPreSplitsMax, KFr / 16);
  if (sp > cap) sp = cap;
  return sp < 1 ? 1 : (int)sp;
}

static pf_status prefill_alloc(pf_model *m, int64_t rows) {
  if (m->pre_rows >= rows) return PF_OK;
  prefill_free(m);
  const pf_model_config &c = m->cfg;
  const int kf = frag_k_of(m);
  const int64_t R = roundup(rows, 128), H = c.hidden, q = (int64_t)c.n_heads * c.head_dim,
                kv = (int64_t)c.n_kv_heads * c.head_dim;
  const int64_t Hp = roundup(H, kf), qp = roundup(q, kf), Fp = roundup(c.ffn, kf);
  pf_status r;
#define PALLOC(ptr, bytes)                       \
  if ((r = dev_alloc(&(ptr), (bytes), nullptr))) { \
    prefill_free(m);                             \
    return r;                                    \
  }
  PALLOC(m->pre_x, R * H * 4);
  PALLOC(m->pre_y, R * (q + 2 * kv) * 4);
  PALLOC(m->pre_rope, R * c.head_dim * 4);
  PALLOC(m->pre_apo, (int64_t)c.n_heads * kPrefillSplits * R * c.head_dim * 4);
  PALLOC(m->pre_apml, (int64_t)c.n_heads * kPrefillSplits * R * 2 * 4);
  PALLOC(m->pre_xn, R * Hp * m->esz);
  PALLOC(m->pre_qb, R * q * m->esz);
  PALLOC(m->pre_attn, R * qp * m->esz);
  PALLOC(m->pre_act, R * Fp * m->esz);
  PALLOC(m->pre_rowinfo, R * 4 * 4);
  PALLOC(m->pre_status, 64);
  if (m->cfg.dtype == PF_DTYPE_BF16) {
    PALLOC(m->pre_part, (int64_t)kPreSplitsMax * R * std::max<int64_t>(q + 2 * kv, H) * 4);
    PALLOC(m->pre_xb, R * Hp * 2);
  }
#undef PALLOC
  // zero padding columns and rows stay zero: the norms write columns < H and
  // the GEMM epilogues skip rows past the chunk
  void *zero[] = {m->pre_xn, m->pre_qb, m->pre_attn, m->pre_act, m->pre_status, m->pre_xb};
  int64_t zb[] = {R * Hp * m->esz, R * q * m->esz, R * qp * m->esz, R * Fp * m->esz, 64, R * Hp * 2};
  for (int i = 0; i < 6; ++i)
    if (zero[i]) HIPCHK(hipMemset(zero[i], 0, zb[i]));
  HIPCHK(hipDeviceSynchronize());
  m->pre_rows = R;
  return PF_OK;
}

pf_status pf_prefill(pf_model *m, pf_kv_cache *kv, const int32_t *tokens, int32_t n, int32_t chunk,
                     float *logits_last, pf_stream s) {
  if (!m || !tokens) return fail(PF_EINVAL, "pf_prefill: null pointer");
  if (pf_status r = kv_check(kv, "pf_prefill")) return r;
  if (pf_status r = model_kv_match(m, kv, "pf_prefill")) return r;
  if (n < 1 || chunk < 1 || chunk > 4096)
    return fail(PF_EINVAL, "pf_prefill: n %d / chunk %d out of range", n, chunk);
  if (kv->pending) return fail(PF_ESTATE, "pf_prefill: a verify step is not committed");
  if (kv->host_bound + n > kv->capacity)
    return fail(PF_ECAPACITY, "pf_prefill: cache bound %lld + %d > capacity %lld",
                (long long)kv->host_bound, n, (long long)kv->capacity);
  const int C = chunk < n ? chunk : n;
  if (pf_status r = prefill_alloc(m, C)) return r;
  const pf_model_config &c = m->cfg;
  const bool bf = is_bf16(m);
  const int kf = frag_k_of(m);
  const int L = c.n_layers, H = c.hidden, hd = c.head_dim, nq = c.n_heads, nkv = c.n_kv_heads;
  const int64_t q = (int64_t)nq * hd, kvd = (int64_t)nkv * hd, F = c.ffn, V = c.vocab;
  const int64_t Hp = roundup(H, kf), qp = roundup(q, kf), Fp = roundup(F, kf);
  const int R = (int)m->pre_rows;
  const float eps = (float)c.rms_eps;
  hipStream_t hs = st(s);
  const uint64_t *rowmask = (const uint64_t *)(m->rowinfo + kRowPad * 4);

  for (int c0 = 0; c0 < n; c0 += C) {
    const int rows = n - c0 < C ? n - c0 : C;
    HIPCHK(launch_prefill_rows(tokens + c0, rows, (int)V, kv->len, m->inv_freq, hd, m->pre_rowinfo,
                               m->pre_rope, m->pre_status, hs));
    HIPCHK(launch_embed_norm(bf, m->embed, m->pre_rowinfo, rows, H, m->attn_norm, eps, m->pre_x,
                             m->pre_xn, Hp, false, nullptr, hs));
    const int64_t keys_max = kv->host_bound + c0 + rows;
    // key ranges: the staged kernel takes enough of them for about two of
    // its blocks per CU; the other path a fixed 8
    const bool staged = attn_prefill_supported(bf, hd, nq / nkv);
    int ck;
    if (staged) {
      // two four-wave blocks per CU; a KV head's query heads take one block
      // per four
      const int blocks = nkv * ((rows + 31) / 32) * ((nq / nkv + 3) / 4);
      int want = (2 * (m->wave_slots / 4) + blocks - 1) / blocks;
      if (want > kPrefillSplits) want = kPrefillSplits;
      ck = (int)roundup((keys_max + want - 1) / want, 64);
      if (ck < 256) ck = 256;
    } else {
      ck = (int)roundup((keys_max + kPrefillSplits - 1) / kPrefillSplits, 32);
      if (ck < 128) ck = 128;
    }
    const int nsp = (int)((keys_max + ck - 1) / ck);
    for (int l = 0; l < L; ++l) {
      BigGemmArgs g{};
      g.W = (const char *)m->wqkv + (int64_t)l * m->pqkv.bytes();
      g.W_bytes = m->pqkv.bytes();
      g.KFr = m->pqkv.KFr;
      g.NTtot = m->pqkv.NT;
      g.X = m->pre_xn;
      g.ldx = Hp;
      g.x_rows = R;
      g.M = rows;
      g.ldy = q + 2 * kvd;
      // bf16: split-K partials, added by the epilogue kernel in split order
      g.splits = bf ? prefill_splits(m->pqkv.NT, R, m->pqkv.KFr, m->wave_slots / 4) : 1;
      g.y = bf ? m->pre_part : m->pre_y;
      g.ystride = (int64_t)R * g.ldy;
      HIPCHK(prefill_gemm(bf, BIG_STORE, g, hs));
      HIPCHK(launch_qkv_post(bf, g.y, g.splits, R, rows, nq, nkv, hd, q + 2 * kvd, m->pre_rope,
                             kv->len, m->pre_qb, q, kv->data, l, kv->capacity, hs));
      AttnArgs at{};
      at.q = m->pre_qb;
      at.ldq = q;
      at.cache = kv->data;
      at.plane = kv->capacity * hd;
      at.cap = kv->capacity;
      at.layer = l;
      at.n_kv = nkv;
      at.group = nq / nkv;
      at.head_dim = hd;
      at.M = rows;
      at.rowpad = R;
      at.kv_len = kv->len;
      at.n_splits = nsp;
      at.chunk_keys = ck;
      at.per_wave = 1;
      at.keys_bound = (int)keys_max;
      at.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)hd));
      at.tree = 0;
      at.anc = rowmask;
      at.part_o = m->pre_apo;
      at.part_ml = m->pre_apml;
      at.out = m->pre_attn;
      at.ldout = qp;
      if (staged)
        HIPCHK(launch_attn_prefill(at, hs));
      else
        HIPCHK(launch_attn(bf, (rows + 15) / 16, at, hs));
      BigGemmArgs go{};
      go.W = (const char *)m->wo + (int64_t)l * m->po.bytes();
      go.W_bytes = m->po.bytes();
      go.KFr = m->po.KFr;
      go.NTtot = m->po.NT;
      go.X = m->pre_attn;
      go.ldx = qp;
      go.x_rows = R;
      go.M = rows;
      go.ldy = H;
      if (bf) {  // split-K partials; the norm kernel adds them to the residual
        go.splits = prefill_splits(m->po.NT, R, m->po.KFr, m->wave_slots / 4);
        go.y = m->pre_part;
        go.ystride = (int64_t)R * H;
        HIPCHK(prefill_gemm(bf, BIG_STORE, go, hs));
        // the FFN input goes out in the 32-row packed layout of the SwiGLU GEMM
        HIPCHK(launch_residual_norm(bf, m->pre_part, go.splits, R, rows, H, H,
                                    m->ffn_norm + (int64_t)l * H, eps, m->pre_x, m->pre_xb, Hp, 2,
                                    hs));
      } else {
        go.y = m->pre_x;
        HIPCHK(prefill_gemm(bf, BIG_RESID, go, hs));
        HIPCHK(launch_residual_norm(bf, nullptr, 0, R, rows, H, H, m->ffn_norm + (int64_t)l * H,
                                    eps, m->pre_x, m->pre_xn, Hp, false, hs));
      }
      BigGemmArgs gg{};
      gg.W = (const char *)m->wgu + (int64_t)l * m->pgu.bytes();
      gg.W_bytes = m->pgu.bytes();
      gg.KFr = m->pgu.KFr;
      gg.NTtot = m->pgu.NT;
      gg.X = m->pre_xn;
      gg.ldx = Hp;
      gg.x_rows = R;
      gg.M = rows;
      gg.act = m->pre_act;
      gg.ldact = Fp;
      gg.up_tile_off = F / 16;
      if (bf) {
        gg.X = m->pre_xb;
        HIPCHK(launch_gemm_ffn(gg, hs));
      } else {
        HIPCHK(prefill_gemm(bf, BIG_SWIGLU, gg, hs));
      }
      BigGemmArgs gd{};
      gd.W = (const char *)m->wd + (int64_t)l * m->pd.bytes();
      gd.W_bytes = m->pd.bytes();
      gd.KFr = m->pd.KFr;
      gd.NTtot = m->pd.NT;
      gd.X = m->pre_act;
      gd.ldx = Fp;
      gd.x_rows = R;
      gd.M = rows;
      gd.ldy = H;
      const float *next_gain = l + 1 < L ? m->attn_norm + (int64_t)(l + 1) * H : m->final_norm;
      if (bf) {
        gd.splits = prefill_splits(m->pd.NT, R, m->pd.KFr, m->wave_slots / 4);
        gd.y = m->pre_part;
        gd.ystride = (int64_t)R * H;
        HIPCHK(prefill_gemm(bf, BIG_STORE, gd, hs));
        HIPCHK(launch_residual_norm(bf, m->pre_part, gd.splits, R, rows, H, H, next_gain, eps,
                                    m->pre_x, m->pre_xn, Hp, false, hs));
      } else {
        gd.y = m->pre_x;
        HIPCHK(prefill_gemm(bf, BIG_RESID, gd, hs));
        HIPCHK(launch_residual_norm(bf, nullptr, 0, R, rows, H, H, next_gain, eps, m->pre_x,
                                    m->pre_xn, Hp, false, hs));
      }
    }
    HIPCHK(launch_add_int(kv->len, rows, hs));
    if (c0 + rows == n && logits_last) {
      // last token: final-norm row -> lm_head (one row through the verify GEMM)
      HIPCHK(launch_pack_row(bf, (const char *)m->pre_xn + (int64_t)(rows - 1) * Hp * m->esz, m->xn,
                             Hp, hs));
      GemmArgs gl{};
      gl.W = m->lm;
      gl.W_bytes = m->plm.bytes();
      gl.KFr = m->plm.KFr;
      gl.NTtot = m->plm.NT;
      gl.X = m->xn;
      gl.ldx = Hp;
      gl.M = 1;
      gl.splits = 1;
      gl.amax = m->amax;
      gl.logits = logits_last;
      gl.ldlog = V;
      HIPCHK(launch_gemm(bf, EPI_ARGMAX, 1, gl, m->wave_slots / 4, hs));
    }
  }
  kv->host_bound += n;
  return ok();
}

}  // extern "C"
