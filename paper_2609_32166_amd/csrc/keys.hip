// Retrieval keys and cosine lookup over the decoding experience memory
// (Section 3.2, "Context-compatible retrieval"; Section 4, "Memory and
// retrieval": final-layer states mapped to 256-dimensional int8 keys by a
// fixed random projection).
//
// Keys. v = R h in fp64. Each component is 16 interleaved fused
// multiply-add chains (chain c: k = c, c+16, ...), added in order at the end;
// a 16-lane group of a wave runs the 16 chains of one (row, component), so the
// summation order, and with it every code, is fixed. code = round-half-even(
// v * 127 / max|v|).
//
// Lookup. The entries of one token (grouped at store build) are scanned by a
// grid of blocks; every thread keeps its best few entries under an exact
// integer order (cosine sign class, then dot^2 * |k'|^2 against dot'^2 * |k|^2,
// then proposal length, then position), blocks reduce theirs in LDS, and one
// block merges the block results and builds the draft.
#include <mutex>

#include "kernels.h"

namespace pf {

// ---------------------------------------------------------------------------
// key projection and quantisation
// ---------------------------------------------------------------------------

template <typename T> __device__ inline double hval(const T *h, int64_t i);
template <> __device__ inline double hval<float>(const float *h, int64_t i) { return (double)h[i]; }
template <> __device__ inline double hval<bf16_t>(const bf16_t *h, int64_t i) {
  return (double)bf16_to_f32(h[i].bits);
}

// grid (kKeyDim / 16, ceil(n / kKeyRowsPerBlock)), 256 threads: thread
// (jj = tid / 16, c = tid % 16) runs chain c of component j = 16 * blockIdx.x
// + jj for the block's rows. Rc is chain-major, [kKeyDim][16][Lc] with Lc a
// multiple of 4 and zeros past the end of K, so a lane streams its chain with
// 16-byte loads; the block's rows are staged in LDS (zeros past H), where a
// zero weight times a zero state leaves the chain unchanged.
template <typename T, bool PACKED>
__global__ __launch_bounds__(256) void k_key_project(const float *Rc, int H, int Lc, const T *h,
                                                     int64_t ld, int n,
                                                     const pf_verify_result *sel, double *v) {
  constexpr int RB = kKeyRowsPerBlock;
  __shared__ float hs[RB][kKeyMaxHidden];
  const int tid = threadIdx.x;
  const int jj = tid >> 4, c = tid & 15;
  const int j = blockIdx.x * 16 + jj;
  const int r0 = blockIdx.y * RB;
  const int Kp = 16 * Lc;  // padded K
  for (int r = 0; r < RB; ++r) {
    const bool live = r0 + r < n;
    const int row = sel ? sel->path[sel->accept_len] : r0 + r;
    for (int k = tid; k < Kp; k += 256) {
      float x = 0.f;
      if (live && k < H)
        x = (float)hval<T>(h, PACKED ? act_off<T>(row, k, ld) : (int64_t)row * ld + k);
      hs[r][k] = x;
    }
  }
  __syncthreads();
  double acc[RB];
#pragma unroll
  for (int r = 0; r < RB; ++r) acc[r] = 0.0;
  const float4 *rc = (const float4 *)(Rc + ((int64_t)j * 16 + c) * Lc);
#pragma unroll 8
  for (int t4 = 0; t4 < Lc / 4; ++t4) {
    const float4 w = rc[t4];
    const float we[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int k = c + 16 * (4 * t4 + e);
#pragma unroll
      for (int r = 0; r < RB; ++r) acc[r] = fma((double)we[e], (double)hs[r][k], acc[r]);
    }
  }
  // add the 16 chains of each (row, component) in order c = 0..15
  __shared__ double part[RB][16][16];
#pragma unroll
  for (int r = 0; r < RB; ++r) part[r][jj][c] = acc[r];
  __syncthreads();
  if (c < RB && r0 + c < n) {
    const int r = c;
    double sum = part[r][jj][0];
#pragma unroll
    for (int t = 1; t < 16; ++t) sum += part[r][jj][t];
    v[(int64_t)(r0 + r) * kKeyDim + j] = sum;
  }
}

// one block of kKeyDim threads per row
__global__ __launch_bounds__(kKeyDim) void k_key_quant(const double *v, int8_t *keys) {
  const int r = blockIdx.x, j = threadIdx.x;
  const double x = v[(int64_t)r * kKeyDim + j];
  __shared__ double sm[kKeyDim / 64];
  double m = fabs(x);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) m = fmax(m, __shfl_xor(m, o, 64));
  if ((j & 63) == 0) sm[j >> 6] = m;
  __syncthreads();
  m = sm[0];
#pragma unroll
  for (int w = 1; w < kKeyDim / 64; ++w) m = fmax(m, sm[w]);
  double code = m > 0.0 ? rint((x * 127.0) / m) : 0.0;
  code = fmin(fmax(code, -127.0), 127.0);
  keys[(int64_t)r * kKeyDim + j] = (int8_t)code;
}

hipError_t launch_key_project(bool bf16, bool packed, const float *Rc, int H, int Lc,
                              const void *h, int64_t ld, int n, const pf_verify_result *sel,
                              double *v, hipStream_t s) {
  if (n < 1) return hipSuccess;
  if (16 * Lc > kKeyMaxHidden || 16 * Lc < H || Lc % 4) return hipErrorInvalidValue;
  const dim3 grid(kKeyDim / 16, (n + kKeyRowsPerBlock - 1) / kKeyRowsPerBlock);
  if (bf16) {
    if (packed)
      return launch_k(k_key_project<bf16_t, true>, grid, 256, s, Rc, H, Lc, (const bf16_t *)h, ld,
                      n, sel, v);
    return launch_k(k_key_project<bf16_t, false>, grid, 256, s, Rc, H, Lc, (const bf16_t *)h, ld,
                    n, sel, v);
  }
  if (packed)
    return launch_k(k_key_project<float, true>, grid, 256, s, Rc, H, Lc, (const float *)h, ld, n,
                    sel, v);
  return launch_k(k_key_project<float, false>, grid, 256, s, Rc, H, Lc, (const float *)h, ld, n,
                  sel, v);
}

// Static projection buffer of pf_key_encode_static: one batch of fp64
// projections in a file-scope device array, so that entry point allocates
// nothing. In host code the array's name is only a stand-in for its symbol;
// its device address, different on every GPU, is looked up once per device
// (with that device current) and kept.
static __device__ __align__(256) double scratch[kKeyBatch * kKeyDim];
constexpr int kMaxDevices = 64;
static double *g_scratch_ptr[kMaxDevices];
static std::mutex g_scratch_mu;

hipError_t key_scratch(double **out, int64_t *elems) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    double *p = nullptr;
    e = hipGetSymbolAddress((void **)&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  *elems = (int64_t)kKeyBatch * kKeyDim;
  return hipSuccess;
}

hipError_t launch_key_quant(const double *v, int n, int8_t *keys, hipStream_t s) {
  if (n < 1) return hipSuccess;
  return launch_k(k_key_quant, n, kKeyDim, s, v, keys);
}

// ---------------------------------------------------------------------------
// cosine lookup
// ---------------------------------------------------------------------------

// A candidate: dot product with the query, squared norm of its key, proposal
// length and position (pos < 0: none).
struct CosCand {
  int dot, nk, len, pos;
};

__device__ inline CosCand no_cand() { return CosCand{0, 0, 0, -1}; }

// dot^2 * nk as a 128-bit (hi, lo) pair (dot^2 < 2^45, nk < 2^23)
__device__ inline void sq_times(int dot, int nk, uint64_t &hi, uint64_t &lo) {
  const uint64_t d2 = (uint64_t)((int64_t)dot * dot);
  lo = d2 * (uint64_t)nk;
  hi = __umul64hi(d2, (uint64_t)nk);
}

// > 0: a ranks above b
__device__ inline int cand_cmp(const CosCand &a, const CosCand &b) {
  if ((a.pos < 0) != (b.pos < 0)) return a.pos < 0 ? -1 : 1;
  if (a.pos < 0) return 0;
  const int ca = a.dot > 0 ? 2 : (a.dot == 0 ? 1 : 0);
  const int cb = b.dot > 0 ? 2 : (b.dot == 0 ? 1 : 0);
  if (ca != cb) return ca - cb;
  if (ca != 1) {
    uint64_t lh, ll, rh, rl;
    sq_times(a.dot, b.nk, lh, ll);
    sq_times(b.dot, a.nk, rh, rl);
    if (lh != rh || ll != rl) {
      const bool gt = lh > rh || (lh == rh && ll > rl);
      return (ca == 2) == gt ? 1 : -1;
    }
  }
  if (a.len != b.len) return a.len > b.len ? 1 : -1;
  if (a.pos != b.pos) return a.pos > b.pos ? 1 : -1;
  return 0;
}

__device__ inline int wave_sum_int(int v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ inline int4 pack_cand(const CosCand &c) { return make_int4(c.dot, c.nk, c.len, c.pos); }
__device__ inline CosCand unpack_cand(int4 v) { return CosCand{v.x, v.y, v.z, v.w}; }

// Block-wide selection of the best n_cand of the items[256 * NI] in LDS
// (each a candidate or none), in rank order, into out[]. Tree reduction per
// round over (item index) with the exact order; the winner is removed.
// The rounds are unrolled to the largest candidate count so that out[] is
// indexed by constants and stays in registers.
template <int NI>
__device__ int select_top(int4 *items, int n_cand, CosCand (&out)[PF_MAX_CAND], int *wins) {
  const int tid = threadIdx.x;
  int found = 0;
#pragma unroll
  for (int r = 0; r < PF_MAX_CAND; ++r) {
    if (r >= n_cand) break;  // uniform over the block
    // each thread's best of its NI items
    int bi = tid * NI;
    CosCand b = unpack_cand(items[bi]);
#pragma unroll
    for (int i = 1; i < NI; ++i) {
      CosCand x = unpack_cand(items[tid * NI + i]);
      if (cand_cmp(x, b) > 0) {
        b = x;
        bi = tid * NI + i;
      }
    }
    wins[tid] = bi;
    __syncthreads();
    for (int st = 128; st >= 1; st >>= 1) {
      if (tid < st) {
        const CosCand x = unpack_cand(items[wins[tid + st]]);
        const CosCand y = unpack_cand(items[wins[tid]]);
        if (cand_cmp(x, y) > 0) wins[tid] = wins[tid + st];
      }
      __syncthreads();
    }
    const int w = wins[0];
    const CosCand best = unpack_cand(items[w]);
    __syncthreads();
    if (best.pos < 0) break;
    out[r] = best;  // r == found: every earlier round found one
    found = r + 1;
    if (tid == 0) items[w] = pack_cand(no_cand());
    __syncthreads();
  }
  return found;
}

// grid kCosScanBlocks x 256: each block scans its share of the query token's
// entries and writes its best n_cand (and how many entries it saw)
__global__ __launch_bounds__(256) void k_cos_scan(CosArgs a) {
  __shared__ uint4 qs[kKeyDim / 16];
  __shared__ int4 items[256 * PF_MAX_CAND];
  __shared__ int wins[256];
  __shared__ int welig[4];
  const int tid = threadIdx.x;
  const int len = *a.ctx_len;
  const int y = len >= 1 ? a.ctx[len - 1] : -1;
  int e0 = 0, e1 = 0;
  if (y >= 0 && y < a.n_tok) {
    e0 = a.tok_off[y];
    e1 = a.tok_off[y + 1];
  }
  if (tid < kKeyDim / 16) qs[tid] = ((const uint4 *)a.q)[tid];
  __syncthreads();

  CosCand top[PF_MAX_CAND];
#pragma unroll
  for (int c = 0; c < PF_MAX_CAND; ++c) top[c] = no_cand();
  int cnt = 0;
  auto consider = [&](int p, int nk, int rem) {
    const uint4 *kp = (const uint4 *)(a.keys + (int64_t)p * kKeyDim);
    int dot = 0;
#pragma unroll
    for (int w = 0; w < kKeyDim / 16; ++w) {
      const uint4 kv = kp[w], qv = qs[w];
      dot = __builtin_amdgcn_sdot4((int)kv.x, (int)qv.x, dot, false);
      dot = __builtin_amdgcn_sdot4((int)kv.y, (int)qv.y, dot, false);
      dot = __builtin_amdgcn_sdot4((int)kv.z, (int)qv.z, dot, false);
      dot = __builtin_amdgcn_sdot4((int)kv.w, (int)qv.w, dot, false);
    }
    CosCand x{dot, nk, min(a.k_max, rem), p};
    ++cnt;
    // insert into the sorted thread-local list
#pragma unroll
    for (int c = 0; c < PF_MAX_CAND; ++c) {
      if (c < a.n_cand && cand_cmp(x, top[c]) > 0) {
        const CosCand t = top[c];
        top[c] = x;
        x = t;
      }
    }
  };
  for (int i = e0 + blockIdx.x * 256 + tid; i < e1; i += kCosScanBlocks * 256)
    consider(a.ent_pos[i], a.ent_nk[i], a.ent_rem[i]);
  // appended positions: token match and p < b(p), b(p) the last position of
  // p's sequence (the open sequence's grows with every append)
  if (a.log_state && y >= 0) {
    const int n_log = a.log_state[0];
    for (int i = blockIdx.x * 256 + tid; i < n_log; i += kCosScanBlocks * 256) {
      const int p = a.T_base + i;
      if (a.tokens[p] != y) continue;
      const int b = a.seq_end[a.log_seq[i]];
      if (p < b) consider(p, a.log_nk[i], b - p);
    }
  }
#pragma unroll
  for (int c = 0; c < PF_MAX_CAND; ++c) items[tid * PF_MAX_CAND + c] = pack_cand(top[c]);
  cnt = wave_sum_int(cnt);
  if ((tid & 63) == 0) welig[tid >> 6] = cnt;
  __syncthreads();
  CosCand best[PF_MAX_CAND];
  const int found = select_top<PF_MAX_CAND>(items, a.n_cand, best, wins);
  if (tid == 0) {
    for (int c = 0; c < PF_MAX_CAND; ++c)
      a.part[blockIdx.x * PF_MAX_CAND + c] = pack_cand(c < found ? best[c] : no_cand());
    a.part_elig[blockIdx.x] = welig[0] + welig[1] + welig[2] + welig[3];
  }
}

// one block: merge the block results (kCosScanBlocks * PF_MAX_CAND items) and
// build the draft
__global__ __launch_bounds__(256) void k_cos_reduce(CosArgs a) {
  static_assert(kCosScanBlocks == 256, "one reduce thread per scan block");
  __shared__ int4 items[256 * PF_MAX_CAND];
  __shared__ int wins[256];
  __shared__ int selig[4], snq[4];
  const int tid = threadIdx.x;
  pf_draft *d = a.draft;
#pragma unroll
  for (int c = 0; c < PF_MAX_CAND; ++c)
    items[tid * PF_MAX_CAND + c] = a.part[tid * PF_MAX_CAND + c];
  const int e = wave_sum_int(a.part_elig[tid]);
  const int qv = (int)a.q[tid];  // kKeyDim == blockDim
  const int nqw = wave_sum_int(qv * qv);
  if ((tid & 63) == 0) {
    selig[tid >> 6] = e;
    snq[tid >> 6] = nqw;
  }
  __syncthreads();
  CosCand best[PF_MAX_CAND];
  const int found = select_top<PF_MAX_CAND>(items, a.n_cand, best, wins);
  int cpos[PF_MAX_CAND], clen[PF_MAX_CAND];
  for (int c = 0; c < PF_MAX_CAND; ++c) {
    const bool ok = c < found;
    cpos[c] = ok ? best[c].pos : -1;
    clen[c] = ok ? best[c].len : 0;
  }
  const int len = *a.ctx_len;
  const int nn = build_draft_block(d, a.tokens, len >= 1 ? a.ctx[len - 1] : 0, cpos, clen, found,
                                   a.tree, a.max_nodes);
  if (tid != 0) return;
  const int nq = snq[0] + snq[1] + snq[2] + snq[3];
  for (int c = 0; c < PF_MAX_CAND; ++c) {
    const bool ok = c < found;
    d->cand_len[c] = clen[c];
    d->cand_pos[c] = cpos[c];
    d->cand_score[c] = ok && nq > 0 && best[c].nk > 0
                           ? (float)((double)best[c].dot / sqrt((double)nq * (double)best[c].nk))
                           : 0.f;
  }
  d->n_found = found;
  d->n_eligible = selig[0] + selig[1] + selig[2] + selig[3];
  d->tree = a.tree;
  d->n_nodes = nn;
}

// open a sequence in the append region: it starts empty at the next
// position (last position = start - 1 until something is appended)
__global__ void k_store_begin(int32_t *log_state, int32_t *seq_end, int32_t T_base) {
  if (threadIdx.x != 0) return;
  const int sq = log_state[1];
  seq_end[sq] = T_base + log_state[0] - 1;
  log_state[1] = sq + 1;
}

// one block: append to the open sequence (the host keeps the region and the
// sequence table large enough)
__global__ __launch_bounds__(256) void k_store_append(AppendArgs a) {
  const int tid = threadIdx.x;
  const int len0 = a.log_state[0];
  const int sq = a.log_state[1] - 1;
  int n = a.res ? a.res->accept_len + 1 : *a.n_dev;
  n = max(0, min(n, min(a.n_max, a.cap - len0)));
  if (sq < 0) n = 0;  // no open sequence
  for (int j = tid; j < n; j += blockDim.x) {
    const int p = a.T_base + len0 + j;
    const int row = a.res ? a.res->path[j] : j;
    a.tokens[p] = a.res ? a.res->out_tokens[j] : a.tok_src[j];
    const int4 *src = (const int4 *)(a.key_src + (int64_t)row * kKeyDim);
    int4 *dst = (int4 *)(a.keys + (int64_t)p * kKeyDim);
    int nk = 0;
#pragma unroll
    for (int w = 0; w < kKeyDim / 16; ++w) {
      const int4 v = src[w];
      dst[w] = v;
      nk = __builtin_amdgcn_sdot4(v.x, v.x, nk, false);
      nk = __builtin_amdgcn_sdot4(v.y, v.y, nk, false);
      nk = __builtin_amdgcn_sdot4(v.z, v.z, nk, false);
      nk = __builtin_amdgcn_sdot4(v.w, v.w, nk, false);
    }
    a.log_seq[len0 + j] = sq;
    a.log_nk[len0 + j] = nk;
  }
  __syncthreads();
  if (tid == 0 && n > 0) {
    a.log_state[0] = len0 + n;
    a.seq_end[sq] = a.T_base + len0 + n - 1;
  }
}

hipError_t launch_store_begin(int32_t *log_state, int32_t *seq_end, int32_t T_base,
                              hipStream_t s) {
  return launch_k(k_store_begin, 1, 64, s, log_state, seq_end, T_base);
}

hipError_t launch_store_append(const AppendArgs &a, hipStream_t s) {
  return launch_k(k_store_append, 1, 256, s, a);
}

hipError_t launch_cos_lookup(const CosArgs &a, hipStream_t s) {
  PF_TRY(launch_k(k_cos_scan, kCosScanBlocks, 256, s, a));
  return launch_k(k_cos_reduce, 1, 256, s, a);
}

}  // namespace pf
