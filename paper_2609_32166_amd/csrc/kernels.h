// Host-side launchers of the HIP kernels (internal to libpf).
#pragma once

#include <utility>

#include "pf_internal.h"

namespace pf {

// Kernel timing for the profiled verify step. While a timer is installed on
// the calling thread, every launch is bracketed by its own pair of events
// recorded on the launch stream (created without the system-scope fence, so
// a marker does not write back and invalidate the caches). A failure to
// create events is kept in the timer and reported by its owner.
struct LaunchTimer {
  hipError_t err = hipSuccess;
  virtual bool events(hipEvent_t *start, hipEvent_t *stop) = 0;
  virtual ~LaunchTimer() = default;
};
extern thread_local LaunchTimer *t_launch_timer;

template <typename... P, typename... A>
inline hipError_t launch_k(void (*k)(P...), dim3 grid, dim3 block, hipStream_t s, A &&...args) {
  hipEvent_t e0, e1;
  LaunchTimer *t = t_launch_timer;
  const bool timed = t && t->events(&e0, &e1);
  if (timed) {
    hipError_t r = hipEventRecord(e0, s);
    if (r != hipSuccess) return r;
  }
  k<<<grid, block, 0, s>>>(std::forward<A>(args)...);
  hipError_t r = hipGetLastError();
  if (r != hipSuccess || !timed) return r;
  return hipEventRecord(e1, s);
}

// Returns the error of a launch helper from the enclosing launcher.
#define PF_TRY(...)                          \
  do {                                       \
    hipError_t e_ = (__VA_ARGS__);           \
    if (e_ != hipSuccess) return e_;         \
  } while (0)

// Buffer-resource loads: 16-byte loads whose byte offset is checked against
// the resource size; an offset past the end returns zeros and fetches
// nothing. Used for ragged K ranges without branches.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef unsigned v4u __attribute__((ext_vector_type(4)));
constexpr uint32_t kOOB = 0x80000000u;
constexpr int kRsrcWord3 = 0x00020000;  // gfx9-family raw buffer descriptor word 3

__device__ inline rsrc_t make_rsrc(const void *p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes,
                                           kRsrcWord3);
}
__device__ inline uint4 bload16(rsrc_t r, uint32_t off) {
  v4u v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
  return make_uint4(v.x, v.y, v.z, v.w);
}
// Same, with the non-temporal cache policy: for data read exactly once per
// launch (weight streams), so it does not displace reused lines in L2.
constexpr int kPolicyNT = 2;
__device__ inline uint4 bload16_stream(rsrc_t r, uint32_t off) {
  v4u v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kPolicyNT);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Deferred RMSNorm scale of the verify step. RMSNorm(x) W^T equals
// inv(x) * ((x * gain) W^T), the product with the gains elementwise and
// inv(x) = 1 / sqrt(mean(x^2) + eps) one number per row, so the norms inside
// the layer stack write x * gain (rounded to the
// model dtype) as the next projection's operand, together with partial sums of
// squares of x, one per slice of kNormSlice columns, at ssq[row * nss +
// slice]; the projection adds a row's slices in slice order and multiplies
// that row's sums by inv before its epilogue. The rounding to the model dtype
// then comes before the per-row scale instead of after it. Spreading a row
// over several norm blocks is what this buys: one block per row moved a whole
// row of partials through a single compute unit.
constexpr int kNormSlice = 512;     // columns per norm block (wider rows: more per block)
constexpr int kMaxNormSlices = 8;
struct RowScale {
  const float *ssq;  // [rows][nss] partial sums of squares
  int nss;           // slices per row (1..kMaxNormSlices)
  int H;             // row length
  float eps;
};
inline int norm_slices(int H) {
  const int n = (H + kNormSlice - 1) / kNormSlice;
  return n < kMaxNormSlices ? n : kMaxNormSlices;
}

// The block's rows' deferred scales into LDS (invl[row], rows < M): thread t
// < M adds row t's slices in slice order, and the epilogue reads one LDS
// value per row after its barrier instead of computing the scale once per
// output tile. The QKV kernel issues the loads before its product loop's
// first loads and finishes right after them (the oldest loads in flight, so
// their wait costs nothing beyond the first products' own wait; issued later,
// its loop's fixed wait counts would also wait for them); the gate/up kernel
// issues them after its first loads and finishes in the epilogue (measured
// 0.5 us faster per 7B launch, the same at 3B). Buffer loads: slices past nss
// and rows past M read zeros, with no branch around a load.
struct RowInv {
  float v[kMaxNormSlices];
  __device__ void issue(const RowScale &r, int M) {
    const int t = (int)threadIdx.x;
    const rsrc_t rr = make_rsrc(r.ssq, (uint32_t)(M * r.nss * 4));
#pragma unroll
    for (int g = 0; g < kMaxNormSlices; ++g)
      v[g] = __builtin_bit_cast(
          float, __builtin_amdgcn_raw_buffer_load_b32(
                     rr, t < M && g < r.nss ? (t * r.nss + g) * 4 : (int)kOOB, 0, 0));
  }
  __device__ void finish(const RowScale &r, int M, float *invl) const {
    float ss = 0.f;
#pragma unroll
    for (int g = 0; g < kMaxNormSlices; ++g)
      if (g < r.nss) ss += v[g];
    const int t = (int)threadIdx.x;
    if (t < M) invl[t] = 1.0f / sqrtf(ss / (float)r.H + r.eps);
  }
};

enum GemmEpi { EPI_PARTIAL = 0, EPI_SWIGLU = 1, EPI_ARGMAX = 2 };

struct GemmArgs {
  const void *W;      // packed fragments of one matrix
  int64_t W_bytes;    // bytes of that packed matrix (< 2^31)
  int64_t KFr;        // k fragments
  int64_t NTtot;      // n tiles (16 rows of W each) of the output
  const void *X;      // activations [kRowPad][ldx], model dtype
  int64_t ldx;        // elements per activation row (multiple of the fragment k)
  int M;              // valid rows
  int splits;         // split-K factor (grid.y)
  // EPI_PARTIAL: out[(split*kRowPad + m)*ldo + n]
  float *out;
  int64_t ldo;
  // EPI_SWIGLU: act[m*ldact + n] = silu(inv*gate)*(inv*up), gate tile t, up tile
  // t + up_tile_off, inv the row's deferred RMSNorm scale (X holds x * gain)
  void *act;
  int64_t ldact;
  int64_t up_tile_off;
  RowScale rs;
  // EPI_ARGMAX: amax[blockIdx.x*kRowPad + m]; optional logits[m*ldlog + n]
  ArgmaxPart *amax;
  float *logits;
  int64_t ldlog;
};

// QKV projection with RoPE and the KV append fused (qkv.hip): one block per
// pair of 16-column tiles half a head apart, K split over the block's waves
struct QkvArgs {
  const void *W;        // packed fused QKV weights of one layer
  int64_t W_bytes, KFr;
  const void *X;        // fragment-packed rows x * gain (RMSNorm scale deferred)
  int64_t ldx;
  RowScale rs;          // the rows' deferred RMSNorm scale, applied to the sums
  int M;                // valid rows
  int nq, nkv, hd;
  const float *rope;    // [kRowPad][hd/2][2] cos, sin of each row's position
  const int32_t *kv_len;
  void *qbuf;           // [kRowPad][ldq] queries after RoPE
  int64_t ldq;
  void *cache;          // KV cache: keys and values at slot P + row
  int layer;
  int64_t cap;
};
// cus: compute units of the device (the block shape depends on the model's
// tile count against it, never on the rows)
hipError_t launch_gemm_qkv(bool bf16, int mt, const QkvArgs &a, int cus, hipStream_t s);

struct AttnArgs {
  const void *q;        // [kRowPad][ldq] queries after RoPE
  int64_t ldq;
  const void *cache;    // KV cache data
  int64_t plane;        // capacity * head_dim
  int64_t cap;          // capacity
  int layer, n_kv, group, head_dim;
  int M;                // query rows (verify rows or prefill chunk rows)
  int rowpad;           // row stride of q and of the partial buffers (>= rows, rows of q
                        // past M must be readable)
  const int32_t *kv_len;  // P (device)
  int n_splits;         // key ranges, one partial result each
  int chunk_keys;       // keys per range (multiple of the chunk, 32 bf16 / 16 fp32)
  int per_wave;         // consecutive key ranges one wave reduces (>= 1)
  int keys_bound;       // host upper bound on P + M (loads stay below it)
  float scale_log2;     // log2(e) / sqrt(head_dim)
  int tree;
  const uint64_t *anc;  // [kRowPad] draft-key visibility of each row (tree)
  float *part_o;        // [n_heads][n_splits][kRowPad][head_dim]
  float *part_ml;       // [n_heads][n_splits][kRowPad][2]
  void *out;            // [kRowPad][ldout] attention output (model dtype)
  int64_t ldout;
  int out_packed;       // out in the fragment-packed activation layout
};

hipError_t launch_attn(bool bf16, int rt, const AttnArgs &a, hipStream_t s);
// merge of the key-range partials (head_dim 128, at most 64 ranges)
hipError_t launch_attn_combine(bool bf16, const AttnArgs &a, hipStream_t s);
// Grouped verify attention (attn_gq.hip; bf16, head_dim 128): one block per
// (KV head, key range of chunk_keys keys, row group) over the group's
// query heads x rows, K/V chunks staged in LDS; then the partial combine.
// hilo: probabilities enter the value product as two bf16 terms.
bool attn_gq_supported(bool bf16, int head_dim);
int attn_gq_tiles(int group, int rows);
int attn_gq_row_groups(int group, int rows);
hipError_t launch_attn_gq(const AttnArgs &a, bool hilo, hipStream_t s);
// Prefill attention with LDS-staged K/V tiles shared by a KV head's query
// heads (bf16, head_dim 128, 4..8 query heads per KV head; chunk_keys a
// multiple of 64), followed by the partial combine.
bool attn_prefill_supported(bool bf16, int head_dim, int group);
hipError_t launch_attn_prefill(const AttnArgs &a, hipStream_t s);
// Query tiles (16 rows) per attention wave for rt tiles, and the waves each
// SIMD holds at that footprint: one or two tiles fit two waves per SIMD,
// three tiles one; more tiles are spread over waves of three (five tiles)
// or two.
inline int attn_tiles_per_wave(int rt) { return rt <= 2 ? rt : (rt == 3 || rt == 5) ? 3 : 2; }
inline int attn_waves_per_simd(int rt) { return attn_tiles_per_wave(rt) == 3 ? 1 : 2; }

// step kernels (step.hip)
struct StepArgs {
  const pf_draft *draft;
  pf_verify_result *res;
  int32_t *kv_len;
  int rows, tree;
  int L, H, nq, nkv, hd, F, V;
  float eps;
  const double *inv_freq;
  int32_t *rowinfo;     // [kRowPad][4] token, depth, valid, 0
  uint64_t *rowmask;    // [kRowPad]
  float *rope;          // [kRowPad][hd/2][2]
};
hipError_t launch_prep(const StepArgs &a, hipStream_t s);
// ssq null: xn = RMSNorm(x) * gain; otherwise xn = x * gain and ssq[row] the
// row's sum of squares (the deferred scale, one slice per row)
hipError_t launch_embed_norm(bool bf16, const void *embed, const int32_t *rowinfo, int M, int H,
                             const float *gain, float eps, float *x, void *xn, int64_t ldxn,
                             int packed, float *ssq, hipStream_t s);
hipError_t launch_qkv_post(bool bf16, const float *part, int splits, int rowpad, int M, int nq,
                           int nkv, int hd, int64_t ldpart, const float *rope, const int32_t *kv_len,
                           void *qbuf, int64_t ldq, void *cache, int layer, int64_t cap,
                           hipStream_t s);
// packed: the xn layout (xn_index: 0 row-major, 1 verify fragment-packed,
// 2 prefill 32-row packed, bf16 only)
hipError_t launch_residual_norm(bool bf16, const float *part, int splits, int rowpad, int M, int H,
                                int64_t ldpart, const float *gain, float eps, float *x, void *xn,
                                int64_t ldxn, int packed, hipStream_t s);
// The same with the RMSNorm scale deferred (verify rows, xn fragment-packed):
// x += partials, xn = x * gain elementwise, ssq[row * norm_slices(H) +
// slice] = the slice's sum of squares of x; one block per (row, slice)
hipError_t launch_residual_norm_deferred(bool bf16, const float *part, int splits, int rowpad, int M,
                                         int H, int64_t ldpart, const float *gain, float *x,
                                         void *xn, int64_t ldxn, float *ssq, hipStream_t s);
// prefill rows: tokens[i] at position P + i (P = *kv_len), RoPE table, rowinfo
hipError_t launch_prefill_rows(const int32_t *tokens, int n, int V, const int32_t *kv_len,
                               const double *inv_freq, int hd, int32_t *rowinfo, float *rope,
                               int32_t *status, hipStream_t s);
hipError_t launch_add_int(int32_t *p, int32_t v, hipStream_t s);
// dst[r][c] = x[r][c] for the first `rows` rows of the fp32 residual stream
// (row stride H in both)
hipError_t launch_copy_rows(const float *x, int rows, int H, float *dst, hipStream_t s);
// plain streaming read of bytes (< 2^31) at buf over `blocks` 256-thread blocks
hipError_t launch_read_stream(const void *buf, uint32_t bytes, int blocks, uint32_t *sink,
                              hipStream_t s);
hipError_t launch_pack_row(bool bf16, const void *src, void *dst, int64_t ld, hipStream_t s);

// tiled GEMM for prefill chunks (gemm_big.hip): Y[M x N] = X[M x K] W^T,
// 128 x 128 block tiles, epilogues below
enum BigEpi { BIG_STORE = 0, BIG_RESID = 1, BIG_SWIGLU = 2 };
struct BigGemmArgs {
  const void *W;
  int64_t W_bytes;
  int64_t KFr, NTtot;
  const void *X;
  int64_t ldx;
  int64_t x_rows;       // rows allocated in X (multiple of 128)
  int M;                // valid rows
  float *y;             // BIG_STORE: y[m*ldy + n]; BIG_RESID: y[m*ldy + n] += result
  int64_t ldy;
  void *act;            // BIG_SWIGLU: act[m*ldact + n]
  int64_t ldact;
  int64_t up_tile_off;  // BIG_SWIGLU: up tile index offset (F/16)
  // launch_gemm_pre, BIG_STORE only: split K over grid.z; split z stores its
  // partial sums at y + z * ystride (0 or 1: no split)
  int splits;
  int64_t ystride;
};
hipError_t launch_gemm_big(bool bf16, int epi, const BigGemmArgs &a, hipStream_t s);
// bf16 prefill GEMM: W streamed into the matrix operands, X staged in LDS,
// 32x32 matrix instructions
// (prefill_gemm.hip); needs x_rows % 128 == 0 and ldx % 32 == 0
hipError_t launch_gemm_pre(int epi, const BigGemmArgs &a, hipStream_t s);
// bf16 prefill SwiGLU GEMM over whole chunks (prefill_gemm.hip): X in the
// 32-row packed layout (xb32_off), x_rows % 32 == 0, ldx >= 32 * KFr
hipError_t launch_gemm_ffn(const BigGemmArgs &a, hipStream_t s);
hipError_t launch_argmax_accept(const ArgmaxPart *amax, int nparts, int rows, int tree,
                                const pf_draft *draft, int32_t *pred, pf_verify_result *res,
                                hipStream_t s);
hipError_t launch_commit(bool bf16, const pf_verify_result *res, void *cache, int L, int nkv,
                         int hd, int64_t cap, int tree, int32_t *kv_len, int32_t *ctx_tokens,
                         int32_t *ctx_len, int64_t ctx_cap, hipStream_t s);
hipError_t launch_kv_copy(bool bf16, bool import_, void *cache, const void *logical_src,
                          void *logical_dst, int L, int nkv, int hd, int64_t cap, int64_t start,
                          int64_t n, hipStream_t s);
hipError_t launch_set_int(int32_t *p, int32_t v, hipStream_t s);
hipError_t launch_hold(const int32_t *flag, uint64_t max_ticks, hipStream_t s);

// rolling-image carryover (carry.hip): one span whose source and destination
// slots do not overlap
constexpr int kCarryMaxHalf = 128;  // head_dim / 2 at most
struct CarryArgs {
  void *cache;              // KV cache data (layout of pf_kv_cache)
  int L, nkv, hd;
  int64_t cap;              // slots per plane
  int64_t src, dst;         // first source / destination slot
  int n;                    // tokens
  int64_t delta;            // m' - m = dst - src
  const double *inv_freq;   // [hd/2] theta^(-2i/hd)
};
hipError_t launch_kv_carry(bool bf16, const CarryArgs &a, hipStream_t s);

// lookup (lookup.hip)
struct LookupArgs {
  const int32_t *tokens;
  const int32_t *ent_pos, *ent_rem, *bucket_off;
  int nb_log2, ngram;
  const int32_t *ctx, *ctx_len;
  int k_max, tree, n_cand, max_nodes;
  pf_draft *draft;
};
hipError_t launch_lookup(const LookupArgs &a, hipStream_t s);

// Draft nodes from ranked candidates, built by a whole block of 256 threads
// (every thread calls it with the same arguments): the candidates' proposal
// tokens are staged in LDS in parallel, one thread builds the nodes there
// (node 0 is the current token; linear: the best candidate's proposal as a
// chain; tree: the candidates merged in rank order into a prefix-shared trie,
// children in creation order, creation stopping for good once max_nodes
// non-root nodes exist), and the block writes every node slot of d (unused
// slots zero, parent -1). Returns the node count.
__device__ inline int build_draft_block(pf_draft *d, const int32_t *tokens, int32_t cur_token,
                                        const int *cand_pos, const int *cand_len, int found,
                                        int tree, int max_nodes) {
  __shared__ int32_t ct[PF_MAX_CAND][PF_MAX_DRAFT];
  __shared__ int32_t ntok[PF_MAX_NODES], npar[PF_MAX_NODES], ndep[PF_MAX_NODES];
  __shared__ uint64_t nanc[PF_MAX_NODES];
  __shared__ int s_nn;
  const int tid = threadIdx.x;
  for (int t = tid; t < PF_MAX_CAND * PF_MAX_DRAFT; t += blockDim.x) {
    const int c = t / PF_MAX_DRAFT, i = t % PF_MAX_DRAFT;
    ct[c][i] = (c < found && i < cand_len[c]) ? tokens[cand_pos[c] + 1 + i] : 0;
  }
  __syncthreads();
  if (tid == 0) {
    int nn = 1;
    ntok[0] = cur_token;
    npar[0] = -1;
    ndep[0] = 0;
    nanc[0] = 1ull;
    if (!tree) {
      if (found > 0) {
        for (int i = 0; i < cand_len[0]; ++i) {
          ntok[nn] = ct[0][i];
          npar[nn] = nn - 1;
          ndep[nn] = nn;
          nanc[nn] = nn < 64 ? (nanc[nn - 1] | (1ull << nn)) : 0ull;
          ++nn;
        }
      }
    } else {
      bool full = false;
      for (int c = 0; c < found && !full; ++c) {
        int cur = 0;
        for (int i = 0; i < cand_len[c]; ++i) {
          const int t = ct[c][i];
          int child = -1;
          for (int u = 1; u < nn; ++u)
            if (npar[u] == cur && ntok[u] == t) {
              child = u;
              break;
            }
          if (child < 0) {
            if (nn - 1 >= max_nodes) {
              full = true;
              break;
            }
            child = nn++;
            ntok[child] = t;
            npar[child] = cur;
            ndep[child] = ndep[cur] + 1;
            nanc[child] = nanc[cur] | (1ull << child);
          }
          cur = child;
        }
      }
    }
    s_nn = nn;
  }
  __syncthreads();
  const int nn = s_nn;
  for (int j = tid; j < PF_MAX_NODES; j += blockDim.x) {
    const bool u = j < nn;
    d->token[j] = u ? ntok[j] : 0;
    d->parent[j] = u ? npar[j] : -1;
    d->depth[j] = u ? ndep[j] : 0;
    d->anc[j] = u ? nanc[j] : 0ull;
  }
  return nn;
}

// cosine retrieval (keys.hip)
constexpr int kKeyDim = PF_KEY_DIM;
constexpr int kKeyRowsPerBlock = 2;   // rows per projection block
constexpr int kKeyMaxHidden = 8192;   // padded hidden sizes the projection stages in LDS
constexpr int kKeyBatch = 64;         // rows per projection launch (work buffer)
constexpr int kCosScanBlocks = 256;   // blocks of the cosine scan
struct CosArgs {
  const int32_t *tokens;
  const int8_t *keys;                  // [T][kKeyDim]
  const int32_t *tok_off;              // [n_tok + 1]
  const int32_t *ent_pos, *ent_rem, *ent_nk;
  int n_tok;
  const int32_t *ctx, *ctx_len;
  const int8_t *q;                     // [kKeyDim]
  int k_max, tree, n_cand, max_nodes;
  int4 *part;                          // [kCosScanBlocks][PF_MAX_CAND] (dot, nk, len, pos)
  int32_t *part_elig;                  // [kCosScanBlocks]
  pf_draft *draft;
  // append region (null log_state: none): entries T_base + i, i < log_state[0]
  const int32_t *log_state;            // [0] appended positions, [1] sequences opened
  const int32_t *log_seq, *log_nk;     // per appended position: sequence, key norm^2
  const int32_t *seq_end;              // per appended sequence: its last position
  int32_t T_base;
};
hipError_t launch_cos_lookup(const CosArgs &a, hipStream_t s);

// append region updates (keys.hip). Open a sequence; append n tokens with
// their keys to the open sequence: n = *n_dev (at most n_max) from
// tok_src / key_src rows, or, with res, the verified iteration's
// out_tokens[0..accept_len] with key rows res->path[j] of key_src.
struct AppendArgs {
  int32_t *tokens;                     // store tokens [T_base + cap]
  int8_t *keys;                        // store keys [T_base + cap][kKeyDim]
  int32_t *log_state, *log_seq, *log_nk, *seq_end;
  int32_t T_base, cap;
  const int32_t *tok_src;
  const int8_t *key_src;
  const int32_t *n_dev;
  int32_t n_max;
  const pf_verify_result *res;
};
hipError_t launch_store_begin(int32_t *log_state, int32_t *seq_end, int32_t T_base, hipStream_t s);
hipError_t launch_store_append(const AppendArgs &a, hipStream_t s);
// v[r][j] (fp64) of rows of h: plain [n][ld] rows, or rows of the packed
// verify activations (ld = padded hidden); with sel, the single row
// sel->path[sel->accept_len]. Rc: the projection chain-major (pf_keyproj).
hipError_t launch_key_project(bool bf16, bool packed, const float *Rc, int H, int Lc,
                              const void *h, int64_t ld, int n, const pf_verify_result *sel,
                              double *v, hipStream_t s);
hipError_t launch_key_quant(const double *v, int n, int8_t *keys, hipStream_t s);
// Device address of the static projection buffer (one batch of kKeyBatch
// rows) on the current device, and its size in doubles.
hipError_t key_scratch(double **out, int64_t *elems);

// Packs W [N][K] (per layer) into MFMA fragments. rope_hd > 0 packs the rows
// of each rope_hd-row head RoPE-paired: 16-row tile t of a head holds
// dimensions 8t..8t+7, then rope_hd/2 + 8t..rope_hd/2 + 8t+7.
hipError_t launch_pack(const void *src, int64_t N, int64_t K, int64_t layers, int64_t src_layer_stride,
                       bool bf16, const Packed &geom, void *dst, hipStream_t s, int rope_hd = 0);
// Column of dimension d (0 <= d < hd) of a head in a RoPE-paired packed output.
__host__ __device__ inline int rope_paired_col(int d, int hd) {
  const int half = hd / 2, e = d < half ? d : d - half;
  return (e / 8) * 16 + (e % 8) + (d < half ? 0 : 8);
}

// Tiles per block along N for each epilogue.
int gemm_tiles_per_block(int epi, int mt);  // argmax; partial-sum counted at two
// W tiles per block of a partial-sum projection (ntiles 16-row tiles, splits)
int gemm_partial_tiles(int mt, int64_t ntiles, int splits, int cus);
// gate/up pairs per block for a model with gate_tiles 16-row gate tiles
int gemm_swiglu_pairs(int mt, int64_t gate_tiles, int cus);
// cus: compute units of the device (gate/up's block shape depends on the
// model's tiles against it)
hipError_t launch_gemm(bool bf16, int epi, int mt, const GemmArgs &a, int cus, hipStream_t s);

}  // namespace pf
