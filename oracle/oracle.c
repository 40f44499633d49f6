/*
 * CPU oracle for the retrieval-drafted verify step. TEST INFRASTRUCTURE ONLY:
 * only the tests, the smoke check and the benchmark's CPU-baseline leg may
 * load this library. It shares no code with the HIP path.
 *
 * Everything is computed in fp64 with plain loops, in the order the paper
 * states the method (arXiv 2609.32166, Section 3.2 "Experience-Guided
 * Adaptive Decoding"):
 *   - the decoding experience memory is one shared token array with an
 *     output-sequence boundary b per entry; a proposal starting after
 *     position p may use positions p+1 .. min(p+l, b) only (Sec. 3.2,
 *     "Decoding experience memory", the [A,B,C | D,E] example);
 *   - an entry is eligible only if its stored token matches the current
 *     token and p < b; no eligible entry means an ordinary greedy pass
 *     (Sec. 3.2, "Context-compatible retrieval");
 *   - one forward pass over the current token and the proposal gives l+1
 *     greedy predictions; the longest matching proposal prefix is accepted
 *     plus the model's own next token (Sec. 3.2, "Single-pass token
 *     verification").
 * The n-gram match key and the (length, position) rank that replace the
 * hidden-state cosine ranking, the token tree and the decoder architecture
 * (RMSNorm, RoPE, grouped-query attention, SwiGLU) are the workload's
 * readings; they are listed with the other readings in the design notes.
 *
 * Precision contract (bf16 models): weights, cached K/V and the activations
 * at these points are bf16, round-to-nearest-even: RMSNorm outputs, Q/K/V
 * after RoPE, the attention output, the SwiGLU output. All other values
 * (residual stream, norms, softmax, logits) stay fp64 here; logits are
 * handed out as fp32 and greedy decisions are taken on those fp32 values.
 */
#include "oracle.h"

#include <math.h>
#include <omp.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Number formats                                                            */
/* ------------------------------------------------------------------------ */

double or_bf16_to_double(uint16_t h) {
  uint32_t b = (uint32_t)h << 16;
  float f;
  memcpy(&f, &b, 4);
  return (double)f;
}

/* Round a double directly to the nearest bf16 value (8 significant bits),
 * ties to even, by clearing the low 45 fraction bits of the binary64
 * pattern. Results outside the binary32 exponent range are not needed here. */
double or_round_bf16(double x) {
  if (!isfinite(x) || x == 0.0) return x;
  uint64_t b;
  memcpy(&b, &x, 8);
  uint64_t lsb = (b >> 45) & 1u;
  b += ((uint64_t)1 << 44) - 1 + lsb;
  b &= ~(((uint64_t)1 << 45) - 1);
  double r;
  memcpy(&r, &b, 8);
  return r;
}

uint16_t or_double_to_bf16_bits(double x) {
  double r = or_round_bf16(x);
  float f = (float)r; /* exact: r has 8 significant bits */
  uint32_t b;
  memcpy(&b, &f, 4);
  return (uint16_t)(b >> 16);
}

static inline double rnd(const or_model *m, double x) { return m->bf16 ? or_round_bf16(x) : x; }

static inline double wget(const or_model *m, const void *p, int64_t i) {
  return m->bf16 ? or_bf16_to_double(((const uint16_t *)p)[i]) : (double)((const float *)p)[i];
}

/* ------------------------------------------------------------------------ */
/* Building blocks (exported so the tests can pin each one)                  */
/* ------------------------------------------------------------------------ */

/* RMSNorm: y_k = x_k / sqrt(mean_k(x^2) + eps) * g_k. */
void or_rmsnorm(const double *x, const float *g, int n, double eps, double *y) {
  double ss = 0.0;
  for (int k = 0; k < n; ++k) ss += x[k] * x[k];
  double inv = 1.0 / sqrt(ss / n + eps);
  for (int k = 0; k < n; ++k) y[k] = x[k] * inv * (double)g[k];
}

/* Rotary embedding, rotate-half pairing: dimension i < d/2 is paired with
 * i + d/2 and rotated by angle pos * theta^(-2i/d). In place. */
void or_rope(double *v, int d, double pos, double theta) {
  int h = d / 2;
  for (int i = 0; i < h; ++i) {
    double ang = pos * pow(theta, -2.0 * (double)i / (double)d);
    double c = cos(ang), s = sin(ang);
    double a = v[i], b = v[i + h];
    v[i] = a * c - b * s;
    v[i + h] = a * s + b * c;
  }
}

/* SiLU-gated linear unit of one pair: silu(g) * u, silu(g) = g / (1 + e^-g). */
double or_swiglu(double g, double u) { return g / (1.0 + exp(-g)) * u; }

/* Dense layer y[m][n] = sum_k x[m][k] * W[n][k] for W stored [N][K] in the
 * model's weight format. Parallel over output features. */
static void linear(const or_model *m, const void *W, int64_t N, int64_t K, int M,
                   const double *x, double *y) {
#pragma omp parallel
  {
    double *row = (double *)malloc(sizeof(double) * (size_t)K);
#pragma omp for schedule(static)
    for (int64_t n = 0; n < N; ++n) {
      for (int64_t k = 0; k < K; ++k) row[k] = wget(m, W, n * K + k);
      for (int r = 0; r < M; ++r) {
        const double *xr = x + (int64_t)r * K;
        double acc = 0.0;
        for (int64_t k = 0; k < K; ++k) acc += xr[k] * row[k];
        y[(int64_t)r * N + n] = acc;
      }
    }
    free(row);
  }
}

/* Exported dense layer for a plain fp32 or bf16 matrix (test access). */
void or_linear(const void *W, int is_bf16, int64_t N, int64_t K, int M, const double *x,
               double *y) {
  or_model m;
  memset(&m, 0, sizeof m);
  m.bf16 = is_bf16;
  linear(&m, W, N, K, M, x, y);
}

/* Softmax attention of one query row over `nk` keys:
 *   out = sum_t softmax_t(q . k_t * scale) v_t,
 * with keys/values given as row pointers (NULL-free), length d. */
void or_attend(const double *q, const double *const *keys, const double *const *vals, int64_t nk,
               int d, double scale, double *out) {
  double *s = (double *)malloc(sizeof(double) * (size_t)(nk > 0 ? nk : 1));
  double mx = -INFINITY;
  for (int64_t t = 0; t < nk; ++t) {
    double acc = 0.0;
    for (int i = 0; i < d; ++i) acc += q[i] * keys[t][i];
    s[t] = acc * scale;
    if (s[t] > mx) mx = s[t];
  }
  double den = 0.0;
  for (int64_t t = 0; t < nk; ++t) {
    s[t] = exp(s[t] - mx);
    den += s[t];
  }
  for (int i = 0; i < d; ++i) out[i] = 0.0;
  for (int64_t t = 0; t < nk; ++t) {
    double p = s[t] / den;
    for (int i = 0; i < d; ++i) out[i] += p * vals[t][i];
  }
  free(s);
}

/* ------------------------------------------------------------------------ */
/* Decoder forward                                                           */
/* ------------------------------------------------------------------------ */

/*
 * One decoder layer l over M new rows, in place on the residual stream x
 * [M][H] (fp64).
 *
 *   kv_prefix  cached K/V of positions 0..P-1, logical layout
 *              [L][2][nkv][P][hd] in the model's storage format
 *   kv_extra   further cached K/V rows that every new row sees, fp64 values
 *              (already rounded to the storage format), [L][2][nkv][E][hd]
 *   pos[M]     absolute RoPE positions of the new rows
 *   vis[M*M]   vis[j*M+i] != 0 iff new row j attends to new row i (j sees
 *              itself; causal for a linear draft, ancestors for a tree)
 *   kv_new     [L][2][nkv][M][hd] fp64 K/V of the new rows (layer l's part
 *              is written); NULL ok
 */
void or_layer(const or_model *m, int l, const void *kv_prefix, int64_t P, const double *kv_extra,
              int64_t E, int M, const int64_t *pos, const uint8_t *vis, double *x,
              double *kv_new) {
  const int H = m->H, nq = m->nq, nkv = m->nkv, hd = m->hd, F = m->F;
  const int qd = nq * hd, kvd = nkv * hd, nqkv = qd + 2 * kvd, grp = nq / nkv;
  const double scale = 1.0 / sqrt((double)hd);

  double *xn = (double *)malloc(sizeof(double) * (size_t)M * H);
  double *qkv = (double *)malloc(sizeof(double) * (size_t)M * nqkv);
  double *att = (double *)malloc(sizeof(double) * (size_t)M * qd);
  double *tmp = (double *)malloc(sizeof(double) * (size_t)M * H);
  double *gu = (double *)malloc(sizeof(double) * (size_t)M * 2 * F);
  double *act = (double *)malloc(sizeof(double) * (size_t)M * F);
  double *pk = (double *)malloc(sizeof(double) * (size_t)nkv * (P > 0 ? P : 1) * hd);
  double *pv = (double *)malloc(sizeof(double) * (size_t)nkv * (P > 0 ? P : 1) * hd);

  /* attention sub-layer input: RMSNorm, rounded */
  for (int r = 0; r < M; ++r) {
    or_rmsnorm(x + (int64_t)r * H, m->attn_norm + (int64_t)l * H, H, m->eps, xn + (int64_t)r * H);
    for (int k = 0; k < H; ++k) xn[(int64_t)r * H + k] = rnd(m, xn[(int64_t)r * H + k]);
  }
  linear(m, (const char *)m->wqkv + (size_t)l * nqkv * H * (m->bf16 ? 2 : 4), nqkv, H, M, xn,
         qkv);
  /* RoPE on every query and key head, then round Q, K, V */
  for (int r = 0; r < M; ++r) {
    double *row = qkv + (int64_t)r * nqkv;
    for (int h = 0; h < nq + nkv; ++h) or_rope(row + h * hd, hd, (double)pos[r], m->theta);
    for (int i = 0; i < nqkv; ++i) row[i] = rnd(m, row[i]);
  }
  if (kv_new) {
    for (int r = 0; r < M; ++r)
      for (int g = 0; g < nkv; ++g)
        for (int i = 0; i < hd; ++i) {
          const double *row = qkv + (int64_t)r * nqkv;
          kv_new[((((int64_t)l * 2 + 0) * nkv + g) * M + r) * hd + i] = row[qd + g * hd + i];
          kv_new[((((int64_t)l * 2 + 1) * nkv + g) * M + r) * hd + i] = row[qd + kvd + g * hd + i];
        }
  }
  /* cached prefix of this layer as fp64 */
  for (int g = 0; g < nkv; ++g)
    for (int64_t t = 0; t < P; ++t)
      for (int i = 0; i < hd; ++i) {
        int64_t src_k = ((((int64_t)l * 2 + 0) * nkv + g) * P + t) * hd + i;
        int64_t src_v = ((((int64_t)l * 2 + 1) * nkv + g) * P + t) * hd + i;
        pk[((int64_t)g * P + t) * hd + i] = wget(m, kv_prefix, src_k);
        pv[((int64_t)g * P + t) * hd + i] = wget(m, kv_prefix, src_v);
      }
  /* grouped-query attention: query head h reads KV head h / grp; keys in
     position order: prefix, extra rows, visible new rows */
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int r = 0; r < M; ++r)
    for (int h = 0; h < nq; ++h) {
      int g = h / grp;
      int64_t cap = P + E + M;
      const double **ks = (const double **)malloc(sizeof(double *) * (size_t)cap);
      const double **vs = (const double **)malloc(sizeof(double *) * (size_t)cap);
      int64_t nk = 0;
      for (int64_t t = 0; t < P; ++t, ++nk) {
        ks[nk] = pk + ((int64_t)g * P + t) * hd;
        vs[nk] = pv + ((int64_t)g * P + t) * hd;
      }
      for (int64_t e = 0; e < E; ++e, ++nk) {
        ks[nk] = kv_extra + ((((int64_t)l * 2 + 0) * nkv + g) * E + e) * hd;
        vs[nk] = kv_extra + ((((int64_t)l * 2 + 1) * nkv + g) * E + e) * hd;
      }
      for (int i = 0; i < M; ++i) {
        if (!vis[(int64_t)r * M + i]) continue;
        ks[nk] = qkv + (int64_t)i * nqkv + qd + g * hd;
        vs[nk] = qkv + (int64_t)i * nqkv + qd + kvd + g * hd;
        ++nk;
      }
      double *o = att + (int64_t)r * qd + h * hd;
      or_attend(qkv + (int64_t)r * nqkv + h * hd, ks, vs, nk, hd, scale, o);
      for (int i = 0; i < hd; ++i) o[i] = rnd(m, o[i]);
      free(ks);
      free(vs);
    }
  /* output projection + residual */
  linear(m, (const char *)m->wo + (size_t)l * H * qd * (m->bf16 ? 2 : 4), H, qd, M, att, tmp);
  for (int64_t i = 0; i < (int64_t)M * H; ++i) x[i] += tmp[i];
  /* feed-forward sub-layer */
  for (int r = 0; r < M; ++r) {
    or_rmsnorm(x + (int64_t)r * H, m->ffn_norm + (int64_t)l * H, H, m->eps, xn + (int64_t)r * H);
    for (int k = 0; k < H; ++k) xn[(int64_t)r * H + k] = rnd(m, xn[(int64_t)r * H + k]);
  }
  linear(m, (const char *)m->wgu + (size_t)l * 2 * F * H * (m->bf16 ? 2 : 4), 2 * (int64_t)F, H,
         M, xn, gu);
  for (int r = 0; r < M; ++r)
    for (int j = 0; j < F; ++j) {
      double g = gu[(int64_t)r * 2 * F + j], u = gu[(int64_t)r * 2 * F + F + j];
      act[(int64_t)r * F + j] = rnd(m, or_swiglu(g, u));
    }
  linear(m, (const char *)m->wd + (size_t)l * H * F * (m->bf16 ? 2 : 4), H, F, M, act, tmp);
  for (int64_t i = 0; i < (int64_t)M * H; ++i) x[i] += tmp[i];

  free(xn); free(qkv); free(att); free(tmp); free(gu); free(act); free(pk); free(pv);
}

/*
 * Final RMSNorm (rounded as it enters the lm_head) and the lm_head of M rows
 * of the last layer's residual stream x [M][H]. hidden [M][H] (NULL ok)
 * receives the lm_head input; logits [M][V] fp32 (NULL ok).
 */
void or_head(const or_model *m, const double *x, int M, float *logits, double *hidden) {
  const int H = m->H;
  const int64_t V = m->V;
  double *xn = (double *)malloc(sizeof(double) * (size_t)(M > 0 ? M : 1) * H);
  for (int r = 0; r < M; ++r) {
    or_rmsnorm(x + (int64_t)r * H, m->final_norm, H, m->eps, xn + (int64_t)r * H);
    for (int k = 0; k < H; ++k) xn[(int64_t)r * H + k] = rnd(m, xn[(int64_t)r * H + k]);
  }
  if (hidden)
    for (int64_t i = 0; i < (int64_t)M * H; ++i) hidden[i] = xn[i];
  if (logits) {
    double *lg = (double *)malloc(sizeof(double) * (size_t)(M > 0 ? M : 1) * V);
    linear(m, m->lm_head, V, H, M, xn, lg);
    for (int64_t i = 0; i < (int64_t)M * V; ++i) logits[i] = (float)lg[i];
    free(lg);
  }
  free(xn);
}

/*
 * Forward pass of M new rows over a cached context: token embedding, the L
 * decoder layers (or_layer), then the final norm and lm_head (or_head).
 *
 *   kv_prefix, P, kv_extra, E, pos, vis: as for or_layer
 *   tok[M]     token ids of the new rows
 *   logits     [M][V] fp32 for rows >= logits_from (others untouched); NULL ok
 *   kv_new     [L][2][nkv][M][hd] fp64 K/V of the new rows; NULL ok
 *   hidden     [M][H] final-layer states (the final RMSNorm output, rounded
 *              as it enters the lm_head) for rows >= logits_from; NULL ok
 *   resid      [L+1][M][H] residual stream: the embeddings, then the stream
 *              after each layer; NULL ok
 * Returns 0.
 */
int or_forward(const or_model *m, const void *kv_prefix, int64_t P, const double *kv_extra,
               int64_t E, int M, const int32_t *tok, const int64_t *pos, const uint8_t *vis,
               int logits_from, float *logits, double *kv_new, double *hidden, double *resid) {
  const int L = m->L, H = m->H;
  const int64_t V = m->V;
  double *x = (double *)calloc((size_t)M * H, sizeof(double));

  /* token embedding */
  for (int r = 0; r < M; ++r)
    for (int k = 0; k < H; ++k) x[(int64_t)r * H + k] = wget(m, m->embed, (int64_t)tok[r] * H + k);
  if (resid) memcpy(resid, x, sizeof(double) * (size_t)M * H);

  for (int l = 0; l < L; ++l) {
    or_layer(m, l, kv_prefix, P, kv_extra, E, M, pos, vis, x, kv_new);
    if (resid) memcpy(resid + (int64_t)(l + 1) * M * H, x, sizeof(double) * (size_t)M * H);
  }

  if ((logits || hidden) && logits_from < M) {
    int nr = M - logits_from;
    or_head(m, x + (int64_t)logits_from * H, nr,
            logits ? logits + (int64_t)logits_from * V : NULL,
            hidden ? hidden + (int64_t)logits_from * H : NULL);
  }
  free(x);
  return 0;
}

/* Greedy choice on fp32 logits: the largest value, the lowest index among
 * equal values; NaN never wins. Returns -1 if every value is NaN. */
int32_t or_argmax(const float *v, int64_t n) {
  int64_t best = -1;
  for (int64_t i = 0; i < n; ++i) {
    if (isnan(v[i])) continue;
    if (best < 0 || v[i] > v[best]) best = i;
  }
  return (int32_t)best;
}

/* ------------------------------------------------------------------------ */
/* Retrieval over the decoding experience memory (exhaustive scan)           */
/* ------------------------------------------------------------------------ */

/*
 * Every store position p is an entry. It is eligible when
 *   - the n tokens ending at p lie inside one output sequence and equal the
 *     last n context tokens (the last of which is the current token), and
 *   - p < b(p), b(p) being the last position of p's output sequence.
 * Its proposal is tokens p+1 .. p+len with len = min(k_max, b(p) - p).
 * Entries rank by (len, p), larger first; the best `n_cand` are returned in
 * rank order. Returns the number found.
 */
int or_lookup_candidates(const int32_t *tokens, const int64_t *seq_off, int64_t n_seqs,
                         int ngram, const int32_t *ctx, int64_t ctx_len, int k_max, int n_cand,
                         int64_t *cand_pos, int32_t *cand_len) {
  int found = 0;
  if (ctx_len < ngram || ngram < 1 || n_cand < 1) return 0;
  const int32_t *q = ctx + ctx_len - ngram;
  for (int64_t s = 0; s < n_seqs; ++s) {
    int64_t a = seq_off[s], b = seq_off[s + 1] - 1; /* b: last position */
    for (int64_t p = a + ngram - 1; p < b; ++p) {
      int match = 1;
      for (int i = 0; i < ngram; ++i)
        if (tokens[p - ngram + 1 + i] != q[i]) { match = 0; break; }
      if (!match) continue;
      int64_t rem = b - p;
      int32_t len = (int32_t)(rem < k_max ? rem : k_max);
      /* insert into the sorted top list */
      int at = found;
      while (at > 0 && (cand_len[at - 1] < len || (cand_len[at - 1] == len && cand_pos[at - 1] < p)))
        --at;
      if (at >= n_cand) continue;
      int last = found < n_cand ? found : n_cand - 1;
      for (int i = last; i > at; --i) {
        cand_len[i] = cand_len[i - 1];
        cand_pos[i] = cand_pos[i - 1];
      }
      cand_len[at] = len;
      cand_pos[at] = p;
      if (found < n_cand) ++found;
    }
  }
  return found;
}

/*
 * Draft nodes. Node 0 is the current token (depth 0). A linear draft is the
 * best candidate's proposal as a chain. A tree merges the candidates in rank
 * order into a prefix-shared token trie: each token walks to the existing
 * child with that token or creates a new child (children in creation order);
 * creation stops for good once `max_nodes` non-root nodes exist.
 * anc[i] has bit u set for every ancestor-or-self u of node i (i < 64).
 * Returns the node count.
 */
int or_build_draft(const int32_t *tokens, const int64_t *cand_pos, const int32_t *cand_len,
                   int n_found, int32_t cur_token, int tree, int max_nodes, int32_t *node_tok,
                   int32_t *parent, int32_t *depth, uint64_t *anc) {
  int n = 1;
  node_tok[0] = cur_token;
  parent[0] = -1;
  depth[0] = 0;
  anc[0] = 1u;
  if (!tree) {
    if (n_found > 0) {
      for (int i = 0; i < cand_len[0]; ++i) {
        node_tok[n] = tokens[cand_pos[0] + 1 + i];
        parent[n] = n - 1;
        depth[n] = n;
        anc[n] = n < 64 ? (anc[n - 1] | ((uint64_t)1 << n)) : 0;
        ++n;
      }
    }
    return n;
  }
  int full = 0;
  for (int c = 0; c < n_found && !full; ++c) {
    int cur = 0;
    for (int i = 0; i < cand_len[c]; ++i) {
      int32_t t = tokens[cand_pos[c] + 1 + i];
      int child = -1;
      for (int u = 1; u < n; ++u)
        if (parent[u] == cur && node_tok[u] == t) { child = u; break; }
      if (child < 0) {
        if (n - 1 >= max_nodes) { full = 1; break; }
        child = n++;
        node_tok[child] = t;
        parent[child] = cur;
        depth[child] = depth[cur] + 1;
        anc[child] = anc[cur] | ((uint64_t)1 << child);
      }
      cur = child;
    }
  }
  return n;
}

/*
 * Retrieval keys (Section 4, "Memory and retrieval": the final-layer states
 * are normalized and reduced to 256-dimensional int8 keys by one fixed random
 * projection). h is the final-layer state as it enters the lm_head (the final
 * RMSNorm output). The projection is v = R h with R [kd][H] row-major: each
 * component is one plain fp64 sum over k = 0 .. H-1 in index order, every
 * product and every partial sum rounded separately (no fused operations).
 * The key is the symmetric int8 quantisation of v with a per-vector scale:
 * code_j = round-half-even(v_j * 127 / max_i |v_i|); an all-zero v gives the
 * zero key. (A positive rescaling of h changes neither the direction nor,
 * up to rounding, the codes, so no further normalisation is applied.)
 * Another summation order of the same projection can move a code by one only
 * where v_j * 127 / max_i |v_i| lies within that order's rounding error of a
 * half-integer.
 */
__attribute__((optimize("fp-contract=off")))
void or_key_project(const double *R, int kd, int H, const double *h, int64_t n, double *v) {
  for (int64_t r = 0; r < n; ++r) {
    const double *hr = h + r * H;
    for (int j = 0; j < kd; ++j) {
      volatile double acc = 0.0;
      for (int k = 0; k < H; ++k) {
        volatile double p = R[(int64_t)j * H + k] * hr[k];
        acc = acc + p;
      }
      v[r * kd + j] = acc;
    }
  }
}

void or_key_encode(const double *R, int kd, int H, const double *h, int64_t n, int8_t *out) {
  double *v = (double *)malloc(sizeof(double) * (size_t)kd);
  for (int64_t r = 0; r < n; ++r) {
    or_key_project(R, kd, H, h + r * H, 1, v);
    double mx = 0.0;
    for (int j = 0; j < kd; ++j)
      if (fabs(v[j]) > mx) mx = fabs(v[j]);
    for (int j = 0; j < kd; ++j) {
      double c = mx > 0.0 ? rint((v[j] * 127.0) / mx) : 0.0;
      if (c > 127.0) c = 127.0;
      if (c < -127.0) c = -127.0;
      out[r * kd + j] = (int8_t)c;
    }
  }
  free(v);
}

/*
 * Cosine order of two entries against one query, decided exactly: cos is
 * dot / sqrt(|q|^2 |k|^2) with integer dot products and squared norms.
 * Positive cosines rank above zero (a zero dot product or a zero key) and
 * zero above negative; two positives compare dot_a^2 |k_b|^2 against
 * dot_b^2 |k_a|^2 (the query norm is common), two negatives the other way.
 * Returns > 0 if a ranks above b, < 0 if below, 0 if equal.
 */
static int cos_cmp(int64_t da, int64_t na, int64_t db, int64_t nb) {
  int ca = da > 0 ? 2 : (da == 0 ? 1 : 0);
  int cb = db > 0 ? 2 : (db == 0 ? 1 : 0);
  if (ca != cb) return ca - cb;
  if (ca == 1) return 0;
  __int128 l = (__int128)da * da * nb, r = (__int128)db * db * na;
  int c = l > r ? 1 : (l < r ? -1 : 0);
  return ca == 2 ? c : -c;
}

/*
 * Cosine retrieval (Section 3.2, "Context-compatible retrieval"): among the
 * entries p whose stored token equals the query token y and that precede
 * their output-sequence boundary (p < b(p)), rank by cosine similarity of
 * the int8 keys (cos_cmp), then by the proposal length min(k_max, b(p) - p),
 * then by p, larger first. Writes the best n_cand in rank order with their
 * cosine (fp64, 0 for a zero key) and returns how many were found.
 */
int or_cos_candidates(const int32_t *tokens, const int64_t *seq_off, int64_t n_seqs,
                      const int8_t *keys, int kd, int32_t y, const int8_t *qkey, int k_max,
                      int n_cand, int64_t *cand_pos, int32_t *cand_len, double *cand_cos) {
  int found = 0;
  int64_t nq = 0;
  for (int j = 0; j < kd; ++j) nq += (int64_t)qkey[j] * qkey[j];
  int64_t cdot[8], cnk[8];
  if (n_cand < 1 || n_cand > 8) return 0;
  for (int64_t s = 0; s < n_seqs; ++s) {
    int64_t a = seq_off[s], b = seq_off[s + 1] - 1; /* b: last position */
    for (int64_t p = a; p < b; ++p) {
      if (tokens[p] != y) continue;
      int64_t dot = 0, nk = 0;
      for (int j = 0; j < kd; ++j) {
        dot += (int64_t)qkey[j] * keys[p * kd + j];
        nk += (int64_t)keys[p * kd + j] * keys[p * kd + j];
      }
      int64_t rem = b - p;
      int32_t len = (int32_t)(rem < k_max ? rem : k_max);
      /* insert into the sorted top list */
      int at = found;
      while (at > 0) {
        int c = cos_cmp(dot, nk, cdot[at - 1], cnk[at - 1]);
        int above = c > 0 || (c == 0 && (len > cand_len[at - 1] ||
                                         (len == cand_len[at - 1] && p > cand_pos[at - 1])));
        if (!above) break;
        --at;
      }
      if (at >= n_cand) continue;
      int last = found < n_cand ? found : n_cand - 1;
      for (int i = last; i > at; --i) {
        cand_len[i] = cand_len[i - 1];
        cand_pos[i] = cand_pos[i - 1];
        cdot[i] = cdot[i - 1];
        cnk[i] = cnk[i - 1];
      }
      cand_len[at] = len;
      cand_pos[at] = p;
      cdot[at] = dot;
      cnk[at] = nk;
      if (found < n_cand) ++found;
    }
  }
  for (int i = 0; i < found; ++i)
    cand_cos[i] = (nq > 0 && cnk[i] > 0) ? (double)cdot[i] / sqrt((double)nq * (double)cnk[i]) : 0.0;
  return found;
}

void or_set_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }
int or_get_threads(void) { return omp_get_max_threads(); }
