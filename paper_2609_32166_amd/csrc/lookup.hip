// Draft lookup over the decoding experience memory.
//
// The store keeps, per n-gram hash bucket, the eligible entries p (the n
// tokens ending at p lie inside p's output sequence and p < b(p)) and
// rem(p) = b(p) - p. One block scans the query's bucket: each lane takes one
// entry, confirms the n tokens, and forms the rank key
// ((min(k_max, rem) + 1) << 40) | p; a wave max-reduction and a cross-wave
// step in LDS pick the best key, repeated with an exclusion bound for the
// top candidates of a tree. Matches are counted with wavefront ballots.
#include "kernels.h"

namespace pf {

__device__ inline unsigned long long wave_max_u64(unsigned long long v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    unsigned long long w = __shfl_xor(v, o, 64);
    v = w > v ? w : v;
  }
  return v;
}

__global__ __launch_bounds__(256) void k_lookup(LookupArgs a) {
  __shared__ int32_t q[8];
  __shared__ unsigned long long wbest[4];
  __shared__ unsigned long long cand[PF_MAX_CAND];
  __shared__ int welig[4];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int len = *a.ctx_len;
  const int n = a.ngram;
  const bool have = len >= n && n >= 1 && a.k_max >= 0;
  if (tid < n && have) q[tid] = a.ctx[len - n + tid];
  pf_draft *d = a.draft;
  __syncthreads();

  int b0 = 0, b1 = 0;
  if (have) {
    const uint32_t bk = ngram_hash(q, n) & ((1u << a.nb_log2) - 1u);
    b0 = a.bucket_off[bk];
    b1 = a.bucket_off[bk + 1];
  }
  const int rounds = a.tree ? a.n_cand : 1;
  unsigned long long bound = ~0ull;
  int found = 0, nelig = 0;
  for (int r = 0; r < rounds; ++r) {
    unsigned long long best = 0;
    int cnt = 0;
    for (int base = b0; base < b1; base += 256) {
      const int i = base + tid;
      bool elig = false;
      unsigned long long key = 0;
      if (i < b1) {
        const int p = a.ent_pos[i];
        elig = true;
        for (int t = 0; t < n; ++t)
          if (a.tokens[p - n + 1 + t] != q[t]) {
            elig = false;
            break;
          }
        if (elig) {
          const int L = min(a.k_max, a.ent_rem[i]);
          key = ((unsigned long long)(L + 1) << 40) | (unsigned long long)p;
        }
      }
      const unsigned long long ball = __ballot(elig);
      cnt += __popcll(ball);
      if (elig && key < bound && key > best) best = key;
    }
    best = wave_max_u64(best);
    if (lane == 0) {
      wbest[w] = best;
      welig[w] = cnt;
    }
    __syncthreads();
    unsigned long long bb = wbest[0];
    for (int k = 1; k < 4; ++k) bb = wbest[k] > bb ? wbest[k] : bb;
    if (r == 0) nelig = welig[0] + welig[1] + welig[2] + welig[3];
    __syncthreads();
    if (bb == 0) break;
    if (tid == 0) cand[found] = bb;
    ++found;
    bound = bb;
  }
  __syncthreads();

  int cpos[PF_MAX_CAND], clen[PF_MAX_CAND];
  for (int c = 0; c < PF_MAX_CAND; ++c) {
    const bool ok = c < found;
    clen[c] = ok ? (int)(cand[c] >> 40) - 1 : 0;
    cpos[c] = ok ? (int)(cand[c] & ((1ull << 40) - 1)) : -1;
  }
  const int nn = build_draft_block(d, a.tokens, len >= 1 ? a.ctx[len - 1] : 0, cpos, clen, found,
                                   a.tree, a.max_nodes);
  if (tid != 0) return;
  d->n_found = found;
  d->n_eligible = nelig;
  d->tree = a.tree;
  for (int c = 0; c < PF_MAX_CAND; ++c) {
    d->cand_len[c] = clen[c];
    d->cand_pos[c] = c < found ? (int64_t)cpos[c] : -1;
    d->cand_score[c] = 0.f;
  }
  d->n_nodes = nn;
}

hipError_t launch_lookup(const LookupArgs &a, hipStream_t s) {
  PF_TRY(launch_k(k_lookup, 1, 256, s, a));
  return hipGetLastError();
}

}  // namespace pf
