/*
 * pf.h -- C ABI of the retrieval-drafted verify step for MI355X (gfx950).
 *
 * One decoding iteration of Experience-Guided Adaptive Decoding (arXiv
 * 2609.32166, Section 3.2) is
 *     pf_draft_lookup -> pf_verify_step -> pf_kv_commit
 * on one HIP stream, with every input and output resident in device memory
 * and no host synchronisation between the calls. pf_prefill covers the
 * prompt-prefix carryover of Section 3.4 (resume after a reused prefix).
 *
 * Conventions
 *  - Every call returns a pf_status and never throws. On error the message
 *    of pf_last_error() (thread-local, valid until the next pf_* call on the
 *    thread) says what was wrong.
 *  - Argument errors are detected on the host before anything is launched.
 *  - "device" pointers are HIP device memory of the current device; "host"
 *    pointers are ordinary process memory read during the call only.
 *  - Work is enqueued on the caller's stream (a hipStream_t passed as
 *    pf_stream; NULL is the legacy default stream). Outputs are valid after
 *    the stream has been synchronised.
 *  - The caller owns every pointer it passes; the library owns the handles
 *    it creates (pf_store, pf_model) and frees them in the destroy calls.
 *  - pf_draft_lookup, pf_verify_step and pf_kv_commit allocate nothing and
 *    do not synchronise: the step can be captured into a HIP graph. A model
 *    holds one set of step work buffers, so steps on one model must not
 *    overlap (serialise them on one stream).
 */
#ifndef PF_H
#define PF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t pf_status;
#define PF_OK 0
#define PF_EINVAL (-1)       /* bad argument (null pointer, size out of range) */
#define PF_ENOMEM (-2)       /* device allocation failed (create calls only) */
#define PF_EHIP (-3)         /* a HIP runtime call failed */
#define PF_ECAPACITY (-4)    /* KV cache or context capacity would be exceeded */
#define PF_ESTATE (-5)       /* object in the wrong state for the call */
#define PF_EUNSUPPORTED (-6) /* shape or dtype the library does not handle */

#define PF_DTYPE_F32 0
#define PF_DTYPE_BF16 1

/* The proposal length is capped at 64 (Section 4, "Memory and retrieval");
 * a draft holds the current token plus at most 64 proposal tokens. */
#define PF_MAX_DRAFT 64
#define PF_MAX_NODES 65
#define PF_MAX_CAND 4
#define PF_MAX_TREE_NODES 63 /* non-root nodes of a tree draft */

typedef void *pf_stream; /* hipStream_t */

typedef struct pf_store pf_store;
typedef struct pf_model pf_model;

const char *pf_last_error(void);
const char *pf_version(void);

/* ------------------------------------------------------------------------ */
/* Draft record (device memory, written by pf_draft_lookup)                  */
/* ------------------------------------------------------------------------ */

/*
 * Node 0 is the current token (the last context token). Linear drafts are a
 * chain: node i (1 <= i < n_nodes) is proposal token i, parent i-1, depth i.
 * Tree drafts merge up to PF_MAX_CAND proposals into a prefix-shared token
 * trie; anc[i] has bit u set for every ancestor-or-self u of node i.
 */
typedef struct pf_draft {
  int32_t n_nodes;   /* 1 + number of proposal tokens (1: no proposal) */
  int32_t tree;      /* 1 if built as a tree */
  int32_t n_found;   /* candidates returned (0..n_cand) */
  int32_t n_eligible;/* eligible store entries seen for the query */
  int32_t token[PF_MAX_NODES];
  int32_t parent[PF_MAX_NODES]; /* -1 for the root */
  int32_t depth[PF_MAX_NODES];
  int32_t reserved0;
  uint64_t anc[PF_MAX_NODES];
  int32_t cand_len[PF_MAX_CAND];  /* proposal length of candidate c */
  int64_t cand_pos[PF_MAX_CAND];  /* store position p of candidate c */
  float cand_score[PF_MAX_CAND];  /* cosine similarity of candidate c (cosine
                                     lookup; 0 for the n-gram lookup) */
} pf_draft;

/* Verify result (device memory, written by pf_verify_step). */
typedef struct pf_verify_result {
  int32_t accept_len;  /* l_acc: accepted proposal tokens */
  int32_t bonus;       /* the model's own token after the accepted prefix */
  int32_t rows;        /* verify rows used */
  int32_t status;      /* 0, or PF_VSTATUS_* bits */
  int64_t kv_base;     /* cache length the step appended after (P) */
  int32_t path[PF_MAX_NODES];       /* node at depth d of the accepted path, d <= accept_len */
  int32_t pred[PF_MAX_NODES];       /* greedy token predicted at each row */
  int32_t out_tokens[PF_MAX_NODES]; /* accept_len accepted tokens, then the bonus */
  int32_t reserved0;
} pf_verify_result;

#define PF_VSTATUS_NAN 1        /* a row's logits held NaN (NaN never wins argmax) */
#define PF_VSTATUS_CTX_FULL 2   /* context buffer too small for the commit */
#define PF_VSTATUS_BAD_TOKEN 4  /* a row's token id was outside [0, vocab); id 0 was used */

/* ------------------------------------------------------------------------ */
/* Decoding context (tokens of prompt and output so far, on the device)     */
/* ------------------------------------------------------------------------ */

typedef struct pf_context {
  int32_t *tokens;    /* device [capacity] */
  int32_t *len;       /* device int32: tokens in use; tokens[len-1] is the current token */
  int64_t capacity;
  int64_t host_bound; /* host upper bound of *len, maintained by the library */
} pf_context;

/* Describe a context buffer whose first `len` tokens are already on the
 * device; sets *len_dev = len (async on s) and host_bound = len. */
pf_status pf_context_init(pf_context *ctx, int32_t *tokens_dev, int32_t *len_dev, int64_t capacity,
                          int64_t len, pf_stream s);
/* Synchronise s and tighten host_bound to the device length. */
pf_status pf_context_sync_bound(pf_context *ctx, pf_stream s);

/* ------------------------------------------------------------------------ */
/* Experience store (Section 3.2, "Decoding experience memory")             */
/* ------------------------------------------------------------------------ */

/*
 * Build the store from prior output sequences appended once to a shared
 * token array. tokens_host[T] holds all sequences back to back;
 * seq_offsets_host[n_seqs+1] are their start offsets (offsets[0] = 0,
 * offsets[n_seqs] = T). An entry at position p is eligible for an n-gram
 * query when the n tokens ending at p lie inside p's sequence and p < b(p),
 * b(p) being the last position of that sequence. The host arrays are copied;
 * the store owns its device copy. ngram in [1, 8]; T < 2^31.
 */
pf_status pf_store_build(const int32_t *tokens_host, const int64_t *seq_offsets_host,
                         int64_t n_seqs, int32_t ngram, pf_stream s, pf_store **out);
void pf_store_destroy(pf_store *store);
int64_t pf_store_size(const pf_store *store); /* tokens T */

/*
 * Draft lookup. The query is the last `ngram` context tokens (ending with the
 * current token). Every eligible entry p proposes tokens p+1..p+len with
 * len = min(k_max, b(p) - p) (truncated at the boundary, Section 3.2).
 * Entries rank by (len, p), larger first. Linear (tree = 0): the best entry's
 * proposal. Tree (tree = 1): the best n_cand proposals merged in rank order
 * into a trie of at most max_nodes non-root nodes. A context shorter than
 * ngram, or no eligible entry, gives an empty proposal (n_nodes = 1), which
 * verifies as an ordinary greedy step. Requires *ctx->len >= 1.
 * k_max in [0, 64]; n_cand in [1, 4] (1 if linear); max_nodes in [1, 63].
 * draft_dev: device pf_draft, written asynchronously on s.
 */
pf_status pf_draft_lookup(const pf_store *store, const pf_context *ctx, int32_t k_max,
                          int32_t tree, int32_t n_cand, int32_t max_nodes, pf_draft *draft_dev,
                          pf_stream s);

/* ------------------------------------------------------------------------ */
/* Cosine retrieval over final-layer states (Section 3.2 "Context-compatible */
/* retrieval"; Section 4 "Memory and retrieval")                            */
/* ------------------------------------------------------------------------ */

/* Entries are indexed by the decoder's final-layer state h (the final RMSNorm
 * output as it enters the lm_head), mapped to PF_KEY_DIM int8 codes through
 * a fixed random projection R [PF_KEY_DIM][hidden]. */
#define PF_KEY_DIM 256

typedef struct pf_keyproj pf_keyproj;

/* Copy the projection R_host ([PF_KEY_DIM][hidden] fp32 values, row-major)
 * to the device. hidden in [16, 8192]. */
pf_status pf_keyproj_create(const float *R_host, int32_t hidden, pf_keyproj **out);
void pf_keyproj_destroy(pf_keyproj *kp);

/*
 * Keys of n states (Section 4, "Memory and retrieval": a fixed random
 * projection of the final-layer state to 256 dimensions, int8): h_dev
 * [n][ld] (PF_DTYPE_F32 or PF_DTYPE_BF16 values, the first `hidden` of each
 * row used) -> keys_dev int8 [n][PF_KEY_DIM]. v = R h in fp64 (each
 * component summed as 16 interleaved fused multiply-add chains, chain c
 * taking k = c, c+16, ..., the chains added in order c = 0..15), then
 * code_j = round-half-even(v_j * 127 / max|v|), the zero key for v = 0.
 * Another fp64 summation order gives the same codes except where
 * v_j * 127 / max|v| lies within the orders' rounding error of a
 * half-integer. n in [0, 2^20]; ld >= hidden. The fp64 projections of each
 * batch of 64 rows pass through the projection's work buffer (allocated by
 * pf_keyproj_create): calls with one projection on overlapping streams race.
 */
pf_status pf_key_encode(const pf_keyproj *kp, const void *h_dev, int32_t dtype, int64_t ld,
                        int64_t n, int8_t *keys_dev, pf_stream s);

/*
 * pf_key_encode for callers that cannot allocate (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * kernels and the same keys, but the fp64 projections of each batch of 64
 * rows pass through a static device buffer of the library (64 x PF_KEY_DIM
 * doubles, 128 KiB, one per GPU, held until the process ends) instead of the
 * projection's work buffer. Calls nothing that allocates. Every call on one
 * GPU shares that buffer, which keeps the last batch's projections: calls
 * that overlap on one GPU (on different streams or host threads) race. The
 * buffer is written in full before it is read, so no clearing is needed.
 * Arguments and errors as for pf_key_encode (n in [0, 2^20]).
 */
pf_status pf_key_encode_static(const pf_keyproj *kp, const void *h_dev, int32_t dtype, int64_t ld,
                               int64_t n, int8_t *keys_dev, pf_stream s);

/*
 * Give a store its cosine index: keys_host int8 [T][PF_KEY_DIM], the key of
 * the state that produced each stored token (T = pf_store_size). An entry is
 * a position p that precedes its output-sequence boundary (p < b(p)); the
 * entries are grouped by their stored token. Replaces a previous index. The
 * host array is copied.
 */
pf_status pf_store_attach_keys(pf_store *store, const int8_t *keys_host, pf_stream s);

/*
 * Cosine draft lookup. The query is (y, q): y the current token (the last
 * context token, on the device) and q_dev int8 [PF_KEY_DIM] the key of the
 * state that predicted it. Eligible entries are those whose stored token is
 * y (and p < b(p)). They rank by cosine similarity of the keys, decided
 * exactly in integers (a positive cosine above zero -- a zero dot product or
 * a zero key -- above a negative one; within a sign by dot^2 / |key|^2), then
 * by proposal length min(k_max, b(p) - p), then by p, larger first. Drafts
 * are built as in pf_draft_lookup (linear, or a trie of the best n_cand);
 * cand_score holds each candidate's cosine. No eligible entry gives an
 * empty proposal. Requires pf_store_attach_keys and *ctx->len >= 1.
 */
pf_status pf_draft_lookup_cosine(const pf_store *store, const pf_context *ctx,
                                 const int8_t *q_dev, int32_t k_max, int32_t tree, int32_t n_cand,
                                 int32_t max_nodes, pf_draft *draft_dev, pf_stream s);

/* ------------------------------------------------------------------------ */
/* Model                                                                    */
/* ------------------------------------------------------------------------ */

typedef struct pf_model_config {
  int32_t n_layers, hidden, n_heads, n_kv_heads, head_dim, ffn, vocab;
  int32_t dtype;     /* PF_DTYPE_F32 or PF_DTYPE_BF16 (weights, cache, activations) */
  double rope_theta; /* rotate-half RoPE, angle pos * theta^(-2i/head_dim) */
  double rms_eps;
} pf_model_config;

/*
 * Device pointers to the caller's weights, row-major, in the model dtype
 * except the norm gains (fp32). L = n_layers, H = hidden, q = n_heads *
 * head_dim, kv = n_kv_heads * head_dim, F = ffn, V = vocab.
 *   embed [V][H], lm_head [V][H]
 *   wqkv [L][q+2kv][H]  rows: query heads, then key heads, then value heads
 *   wo   [L][H][q]
 *   wgu  [L][2F][H]     rows: gate, then up
 *   wd   [L][H][F]
 *   attn_norm, ffn_norm [L][H]; final_norm [H]
 * pf_model_create copies everything into library-owned buffers (weights in a
 * tiled layout for the matrix cores); the caller may free its copies after
 * the stream has been synchronised.
 */
typedef struct pf_model_weights {
  const void *embed, *lm_head, *wqkv, *wo, *wgu, *wd;
  const float *attn_norm, *ffn_norm, *final_norm;
} pf_model_weights;

/* Requirements: head_dim in {64, 128}; n_heads % n_kv_heads == 0; hidden,
 * q, F multiples of 16; vocab multiple of 16. */
pf_status pf_model_create(const pf_model_config *cfg, const pf_model_weights *w, pf_stream s,
                          pf_model **out);
void pf_model_destroy(pf_model *model);
/* Device bytes held by the model (weights + work buffers). */
int64_t pf_model_bytes(const pf_model *model);

/* ------------------------------------------------------------------------ */
/* KV cache (caller-owned device buffer with this layout)                   */
/* ------------------------------------------------------------------------ */

/*
 * Per layer l and KV head g, a key plane and a value plane of
 * capacity*head_dim elements each, in the model dtype, together the array
 * [n_layers][2][n_kv][capacity][head_dim]:
 *   keys   at ((l*2 + 0)*n_kv + g) * capacity*head_dim, element [slot][i]
 *   values at ((l*2 + 1)*n_kv + g) * capacity*head_dim, element [slot][i]
 * Slot t holds position t. *len is the committed length; slots >= *len are
 * dead. capacity must be a multiple of 64.
 */
typedef struct pf_kv_cache {
  void *data;         /* device, pf_kv_bytes() bytes */
  int32_t *len;       /* device int32 */
  int64_t capacity;
  int64_t host_bound; /* host upper bound of *len, maintained by the library */
  int32_t n_layers, n_kv_heads, head_dim, dtype;
  int32_t pending;      /* rows appended by the last verify, not yet committed */
  int32_t pending_tree; /* 1 if that verify was a tree draft */
} pf_kv_cache;

int64_t pf_kv_bytes(const pf_model *model, int64_t capacity);
pf_status pf_kv_init(pf_kv_cache *kv, const pf_model *model, void *data_dev, int32_t *len_dev,
                     int64_t capacity);
/* Copy a prefix given in the logical layout [L][2][n_kv][n][head_dim]
 * (device) into slots 0..n-1 and set the length to n. */
pf_status pf_kv_import(pf_kv_cache *kv, const void *src_dev, int64_t n, pf_stream s);
/* Copy slots start..start+n-1 out in the logical layout [L][2][n_kv][n][head_dim]. */
pf_status pf_kv_export(const pf_kv_cache *kv, void *dst_dev, int64_t start, int64_t n,
                       pf_stream s);
/* Set the committed length (rolls back whole steps; len <= capacity). */
pf_status pf_kv_set_len(pf_kv_cache *kv, int64_t len, pf_stream s);
/* Synchronise s and tighten host_bound to the device length (the bound
 * otherwise grows by the verify rows at every commit). */
pf_status pf_kv_sync_bound(pf_kv_cache *kv, pf_stream s);

/* ------------------------------------------------------------------------ */
/* Verify step (Section 3.2, "Single-pass token verification")              */
/* ------------------------------------------------------------------------ */

/*
 * One decoder forward over `rows` rows: node j of the draft (row 0 the
 * current token; rows >= n_nodes are padding: token 0, never accepted, never
 * attended by real rows) at position P + depth(j), P = *kv->len. Each row
 * attends to the cached prefix 0..P-1 and to the draft rows it may see:
 * rows <= j for a linear draft, ancestors-or-self for a tree. K/V of row j
 * are appended at slot P + j. Greedy prediction per row (largest fp32 logit,
 * lowest index on ties, NaN never wins), then acceptance of the longest
 * proposal prefix that matches the predictions plus the model's next token.
 * rows = k_max + 1 for linear drafts (<= 65), max_nodes + 1 for trees (<= 64),
 * at least the draft's n_nodes. logits_dev: NULL or device fp32
 * [rows][vocab] receiving the logits. res_dev: device pf_verify_result.
 * Fails with PF_ECAPACITY if host_bound + rows > capacity.
 */
pf_status pf_verify_step(pf_model *model, pf_kv_cache *kv, const pf_draft *draft_dev,
                         int32_t rows, int32_t tree, float *logits_dev,
                         pf_verify_result *res_dev, pf_stream s);

/*
 * Profiling variant of pf_verify_step: the same work, timed per kernel. The
 * stream is first held by a wait kernel (released by the host once the whole
 * step is enqueued, and bounded by 500 ms of device wall clock in any case),
 * so the kernels run back to back instead of waiting on host submission.
 * Every launch is bracketed by a pair of fenceless HIP events; the cost of a
 * pair itself is measured in the same call from pairs recorded with no work
 * between (kind PF_PROF_MARKER: their total ms and their number) and is
 * subtracted from every launch. The call synchronises s, then adds each
 * launch's duration in ms to ms_out[kind] and 1 to count_out[kind] (host
 * arrays of PF_PROF_KINDS entries, caller-initialised). Allocates events and
 * a pinned flag: not for graph capture.
 */
#define PF_PROF_KINDS 11
#define PF_PROF_SETUP 0     /* row setup, embedding + first RMSNorm */
#define PF_PROF_QKV 1       /* QKV projection */
#define PF_PROF_QKV_POST 2  /* split-K reduction, RoPE, KV append */
#define PF_PROF_ATTN 3      /* verify attention + split merge */
#define PF_PROF_O 4         /* output projection */
#define PF_PROF_NORM 5      /* residual add + RMSNorm */
#define PF_PROF_GATE_UP 6   /* gate/up projection + SwiGLU */
#define PF_PROF_DOWN 7      /* down projection */
#define PF_PROF_LM_HEAD 8   /* lm_head + argmax partials */
#define PF_PROF_ACCEPT 9    /* argmax reduction + acceptance */
#define PF_PROF_MARKER 10   /* empty event pairs (calibration, not subtracted) */
pf_status pf_verify_step_profiled(pf_model *model, pf_kv_cache *kv, const pf_draft *draft_dev,
                                  int32_t rows, int32_t tree, float *logits_dev,
                                  pf_verify_result *res_dev, pf_stream s, double *ms_out,
                                  int32_t *count_out);

/*
 * Benchmark hook: enqueues only the launches of one profiling kind (one of
 * PF_PROF_SETUP .. PF_PROF_ACCEPT) that pf_verify_step would make for these
 * arguments, every layer's, on the step's own buffers, so that one kernel's
 * duration can be timed in isolation (e.g. captured in a graph). The outputs
 * are meaningless, nothing becomes pending for pf_kv_commit, and the cache
 * slots P.. may be overwritten. Argument checks and errors as for
 * pf_verify_step; kind out of range: PF_EINVAL.
 */
pf_status pf_verify_kernel_repeat(pf_model *model, pf_kv_cache *kv, const pf_draft *draft_dev,
                                  int32_t rows, int32_t tree, int32_t kind,
                                  pf_verify_result *res_dev, pf_stream s);

/*
 * Calibration for the benchmark's roofline: reads `bytes` of device memory at
 * buf_dev (16-byte aligned, a multiple of 16 KiB) once with a plain streaming
 * kernel (one 256-thread block per compute unit, every wave keeping eight
 * 16-byte loads per lane in flight) and writes a checksum word to sink_dev,
 * so that the time of the call is the device's achievable HBM read rate.
 */
pf_status pf_read_stream(const void *buf_dev, int64_t bytes, uint32_t *sink_dev, pf_stream s);

/*
 * Test-mode variant of pf_verify_step: the same step, plus a copy of the
 * residual stream (the fp32 state every decoder layer adds its attention and
 * feed-forward outputs to, Section 3.2's verification forward) into resid_dev,
 * device fp32 [n_layers + 1][rows][hidden]: entry 0 holds the token
 * embeddings, entry l + 1 the stream after layer l (the input of the final
 * norm for l = n_layers - 1). It lets a test drive a reference from the
 * device's own input of each layer. resid_dev must not be NULL; the other
 * arguments and errors are those of pf_verify_step. The copies are extra
 * launches on s (allocates nothing).
 */
pf_status pf_verify_step_trace(pf_model *model, pf_kv_cache *kv, const pf_draft *draft_dev,
                               int32_t rows, int32_t tree, float *logits_dev,
                               pf_verify_result *res_dev, float *resid_dev, pf_stream s);

/*
 * Retrieval keys from the last verify step's final-layer states (they stay
 * in the model's work buffers until its next verify step or prefill).
 * pf_verify_query_key: the key of the row whose prediction is the bonus token
 * (node path[accept_len]), i.e. the query of the next iteration (Section 3.2:
 * the final token of an iteration and the state that produced it form the
 * next retrieval query). pf_verify_row_keys: the keys of rows 0..rows-1 (the
 * contexts of the verified tokens, for adding them to the store). The model's
 * hidden size must equal the projection's. keys int8 device memory.
 */
pf_status pf_verify_query_key(const pf_model *model, const pf_keyproj *kp,
                              const pf_verify_result *res_dev, int8_t *q_dev, pf_stream s);
pf_status pf_verify_row_keys(const pf_model *model, const pf_keyproj *kp, int32_t rows,
                             int8_t *keys_dev, pf_stream s);

/*
 * Commit the accepted rows (Section 3.2: the iteration advances the output
 * by l_acc + 1 tokens). Linear: the accepted rows already sit at slots
 * P..P+l_acc; the length becomes P + l_acc + 1 and later slots are dead
 * (rollback of the rejected rows). Tree: the rows of the accepted path are
 * moved to slots P..P+l_acc first. ctx (nullable): the accepted tokens and
 * the bonus token are appended, so the bonus becomes the current token.
 */
pf_status pf_kv_commit(pf_kv_cache *kv, const pf_verify_result *res_dev, pf_context *ctx,
                       pf_stream s);

/* ------------------------------------------------------------------------ */
/* Prompt-prefix carryover prefill (Section 3.4)                            */
/* ------------------------------------------------------------------------ */

/*
 * Rolling-image KV-state carryover (Section 3.4): for s = 0..n_spans-1 in
 * order, the cached tokens at slots src[s]..src[s]+len[s]-1 move to slots
 * dst[s]..dst[s]+len[s]-1. A key cached at position m becomes
 * R(m') R(m)^-1 K at m' = m + dst[s] - src[s] (R: the model's rotary
 * embedding; evaluated as the rotation by m' - m, angles in fp64, the
 * rotation in fp32, rounded to the cache dtype); values move unchanged.
 * Every span reads the cache as the earlier spans left it, and a span whose
 * source and destination overlap behaves as a memmove (it runs as pieces of
 * |dst - src| tokens, one launch each). Slots are read whether or not they
 * lie below the cache length, which the call does not change: a step that
 * keeps a prefix sets the length (pf_kv_set_len) to prefill the new tokens
 * between and after the carried spans. src, dst, len: host arrays; every
 * span must lie inside the capacity. Errors: PF_EINVAL (spans), PF_ESTATE (a
 * verify step not committed), PF_EUNSUPPORTED (head_dim > 256, or one cache
 * plane, capacity * head_dim elements, of 2 GiB or more). Allocates nothing,
 * does not synchronise.
 */
pf_status pf_kv_carry(pf_kv_cache *kv, const pf_model *model, int32_t n_spans, const int64_t *src,
                      const int64_t *dst, const int64_t *len, pf_stream s);

/*
 * Run n new tokens (device int32) through the decoder after the cached
 * prefix P = *kv->len, in causal chunks of `chunk` rows, appending their K/V
 * at slots P..P+n-1 and setting the length to P+n. logits_last_dev: NULL or
 * device fp32 [vocab] for the last new token. Needs host_bound + n <= capacity.
 */
pf_status pf_prefill(pf_model *model, pf_kv_cache *kv, const int32_t *tokens_dev, int32_t n,
                     int32_t chunk, float *logits_last_dev, pf_stream s);

/* ------------------------------------------------------------------------ */
/* Online memory update (Section 3.2, step 6; decoding-memory budget,       */
/* Section 5.6)                                                             */
/* ------------------------------------------------------------------------ */

/*
 * After each decoding iteration the tokens it appended and the contexts that
 * produced them join the decoding memory. The store (with keys attached)
 * gets an append region: positions T .. T + capacity - 1 of its token and
 * key arrays, in appended output sequences. The cosine lookup sees appended
 * positions like built ones: eligible when the token matches and the
 * position precedes its sequence's last position; the open sequence's last
 * position is its newest token, so every append makes the previous one
 * eligible. The n-gram lookup sees only built positions. A store with an
 * append region ranks exactly like a store built from the same sequences
 * (tests compare the two).
 *
 * pf_store_reserve: create the region (capacity positions, at most max_seqs
 *   sequences); needs keys attached; once per store (pf_store_attach_keys
 *   then fails with PF_ESTATE). Synchronises s.
 * pf_store_begin_sequence: open a new, empty output sequence (the previous
 *   one is closed); PF_ECAPACITY past max_seqs.
 * pf_store_append: append *n_dev tokens (device int32, at most n_max) with
 *   their keys (device int8 [n][256], 16-byte aligned) to the open sequence.
 * pf_store_append_verified: append the last verify step's out_tokens[0 ..
 *   accept_len] with the keys of the rows that produced them (rows path[j],
 *   from the model's final-layer states; the projection as in
 *   pf_verify_row_keys), device-side, with no host synchronisation.
 * Both appends fail with PF_ESTATE without an open sequence and with
 *   PF_ECAPACITY when the host's bound on appended positions (grown by n_max
 *   or the verify rows per call, made exact by pf_store_appended) would pass
 *   the capacity.
 * pf_store_appended: synchronise s, return the appended positions.
 * pf_store_compact: synchronise s and rebuild the store from its sequences
 *   (built, then appended, in order), evicting the oldest sequences while
 *   more than `budget` positions remain (0: no budget); the append region is
 *   recreated empty with no open sequence. The store's size (pf_store_size)
 *   then counts the kept positions.
 */
pf_status pf_store_reserve(pf_store *store, int64_t capacity, int32_t max_seqs, pf_stream s);
pf_status pf_store_begin_sequence(pf_store *store, pf_stream s);
pf_status pf_store_append(pf_store *store, const int32_t *tokens_dev, const int8_t *keys_dev,
                          const int32_t *n_dev, int32_t n_max, pf_stream s);
pf_status pf_store_append_verified(pf_store *store, const pf_model *model, const pf_keyproj *kp,
                                   const pf_verify_result *res_dev, pf_stream s);
pf_status pf_store_appended(pf_store *store, pf_stream s, int64_t *n_out);
pf_status pf_store_compact(pf_store *store, int64_t budget, pf_stream s);

/* ------------------------------------------------------------------------ */
/* Proposal-length controller (Section 3.2, "Runtime-adaptive proposal-     */
/* length controller", Eq. (1))                                             */
/* ------------------------------------------------------------------------ */

/*
 * Host-side, fp64. For an eligible retrieval of similarity s (the draft's
 * cand_score[0] for the cosine lookup) whose proposal holds `avail` tokens,
 * the length l in 0..L, L = min(l_max, avail), that minimises
 *     J(l) = T(l) / (A(l, s) + 1)
 * (ties: the shorter). l = 0 is a greedy pass; verify with rows = l + 1 (the
 * verify step ignores draft nodes at or beyond `rows`).
 *   A(l, s) = sum_{j=1..l} prod_{i=1..j} q_i, the expected accepted proposal
 *     tokens; q_1 = sigmoid(w_first . (1, s, 1/l_max)) is the first token's
 *     acceptance probability and q_j = sigmoid(w_cont . (1, s, j/l_max)) the
 *     probability that token j >= 2 passes given that token j-1 did.
 *   T(l) = exp(theta . (1, u, u^2)), u = l/l_max: the predicted iteration
 *     latency in ms.
 * pf_ctl_observe learns from one finished iteration that proposed l tokens
 * at similarity s, accepted `accepted` of them and took latency_ms: one
 * logistic-regression gradient step (w += lr * (y - q) * x) for the first
 * token when l >= 1 and for each token j = 2..min(l, accepted+1) (y: token j
 * accepted), then one recursive-least-squares step of log(latency_ms) on
 * (1, u, u^2) with forgetting factor `forget` (from theta = 0, covariance
 * prior_var * I). Every explore_every-th pf_ctl_choose (0: never) returns a
 * neighbour of the best length instead, alternately the one above and the
 * one below (the other one where that leaves 0..L; none when L = 0).
 * Errors: PF_EINVAL for a null pointer, a parameter out of its range, a
 * non-finite similarity or latency, or an observation with accepted outside
 * 0..l or l outside 0..l_max. A controller is not thread-safe.
 */
typedef struct pf_ctl_params {
  int32_t l_max;         /* 1..64 */
  int32_t explore_every; /* >= 0 */
  double lr;             /* > 0 */
  double forget;         /* (0, 1] */
  double prior_var;      /* > 0 */
} pf_ctl_params;

typedef struct pf_ctl_state {
  double w_first[3];
  double w_cont[3];
  double theta[3];
  double P[9]; /* latency-fit covariance, row-major */
  int64_t n_choose, n_explore, n_observe;
} pf_ctl_state;

typedef struct pf_ctl pf_ctl;

pf_status pf_ctl_create(const pf_ctl_params *params, pf_ctl **out);
void pf_ctl_destroy(pf_ctl *ctl);
pf_status pf_ctl_get_state(const pf_ctl *ctl, pf_ctl_state *out);
/* Replace the estimator states and counters (all values finite, counters >= 0). */
pf_status pf_ctl_set_state(pf_ctl *ctl, const pf_ctl_state *in);
/* J(0..L) into objective_out (NULL, or host double[L + 1]) and the argmin
 * into best_out (nullable); changes nothing. */
pf_status pf_ctl_objective(const pf_ctl *ctl, double s, int32_t avail, double *objective_out,
                           int32_t *best_out);
pf_status pf_ctl_choose(pf_ctl *ctl, double s, int32_t avail, int32_t *l_out);
pf_status pf_ctl_observe(pf_ctl *ctl, int32_t l, double s, int32_t accepted, double latency_ms);

/* ------------------------------------------------------------------------ */
/* One decoding iteration, host-driven (Section 3.2, steps 2-7)             */
/* ------------------------------------------------------------------------ */

typedef struct pf_iteration {
  int32_t n_found;  /* eligible entries the retrieval ranked (0: greedy pass) */
  int32_t avail;    /* tokens of the retrieved proposal (cut at its boundary and the cap) */
  int32_t l;        /* proposal length verified (rows = l + 1) */
  int32_t accepted; /* l_acc */
  int32_t bonus;    /* the model's token after the accepted prefix: the new current token */
  int32_t status;   /* pf_verify_result.status */
  double s;         /* cosine similarity of the retrieved entry (0 when none) */
  double ms;        /* host wall time of the whole call */
} pf_iteration;

/*
 * Cosine retrieval for the current token with query key q_dev (linear
 * proposal, cap ctl's l_max, or l_fixed without a controller) -> the length
 * l: Eq. (1) through pf_ctl_choose, or min(l_fixed, retrieved length), or 0
 * when nothing is eligible -> pf_verify_step over l + 1 rows ->
 * pf_kv_commit (appends the accepted tokens and the bonus to ctx) -> with
 * append != 0, pf_store_append_verified (the memory update of step 6) ->
 * pf_verify_query_key into q_dev (the next iteration's query) -> with a
 * controller, pf_ctl_observe(l, s, accepted, ms) (also for greedy passes,
 * which teach the latency fit T(0)). ctl: nullable. store must have keys
 * attached; the projection's hidden size must be the model's. draft_dev,
 * res_dev: device buffers the iteration writes. The call synchronises s
 * twice (after the retrieval and at the end) and tightens kv and ctx
 * host bounds to the exact lengths; on the model's first call it allocates
 * a small pinned host buffer, so it is not for graph capture. Errors: those
 * of the calls it makes, PF_EINVAL for null pointers or l_fixed outside
 * 0..64.
 */
pf_status pf_decode_iteration(pf_model *model, pf_kv_cache *kv, pf_context *ctx, pf_store *store,
                              const pf_keyproj *kp, pf_ctl *ctl, int32_t l_fixed, int32_t append,
                              int8_t *q_dev, pf_draft *draft_dev, pf_verify_result *res_dev,
                              pf_iteration *out, pf_stream s);

#ifdef __cplusplus
}
#endif
#endif /* PF_H */
