// Grouped verify attention for bf16 models with head_dim 128: one block per
// (KV head, key range, row group). The rows of a block are "virtual rows":
// every (query head of the KV group, draft row) pair, head-major, so the
// group's query heads share one copy of each K/V chunk. A chunk (32 keys:
// 8 KiB of keys, 8 KiB of values, both [slot][head_dim] rows in the cache) is
// loaded once per block by all 256 threads into registers two chunks ahead,
// stored into one of three LDS stages (values transposed on the way, so the
// value product reads eight consecutive keys of one dimension per lane), and
// read from there by the four waves, each of which holds RT 16-row tiles of
// virtual rows. Per wave and chunk the arithmetic is that of
// the per-head kernel (attn.hip): S^T = K Q^T with the permuted key rows, the
// log2-domain online softmax with the deferred rescale, then O^T += V^T P^T.
// With HILO the probabilities enter the value product as two bf16 terms
// (p = hi + lo, lo = the rounding residue of hi), so the product sees them to
// about 16 significant bits instead of 8.
//
// Key ranges are a fixed number of chunks that depends only on the key
// bound's band (chosen by the host), and every range is reduced from fresh
// accumulators, so a row's result does not depend on the other rows of the
// step. Each block writes one partial (o, max, sum) per virtual row in the
// layout k_attn_combine reads.
#include "kernels.h"

namespace pf {

namespace {

constexpr int GQ_HD = 128;
constexpr int GQ_KC = 32;                          // keys per chunk
// Staged keys: [key][16-byte granule g ^ swz(key)] rows of 256 bytes; staged
// values: [dim][32 keys] rows padded to 80 bytes. The swizzle spreads the 16
// keys one operand read touches (keys 0-3, 8-11, 16-19, 24-27 plus 4 for the
// second group) over 16 distinct granules, and the 80-byte value rows put
// the 16 dimensions of a read on distinct banks, so neither read conflicts.
constexpr int GQ_KROW = GQ_HD * 2;                 // 256
constexpr int GQ_VROW = GQ_KC * 2 + 16;            // 80
constexpr int GQ_KBYTES = GQ_KC * GQ_KROW;         // 8192
constexpr int GQ_STAGE = GQ_KBYTES + GQ_HD * GQ_VROW;  // 18432
__device__ inline int gq_swz(int key) { return (key & 15) ^ ((key >> 4) << 2); }
constexpr int GQ_NST = 3;                          // LDS stages

__device__ inline uint4 pack8_bf16(const float *p) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  typedef __bf16 b2 __attribute__((ext_vector_type(2)));
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f2){p[2 * i], p[2 * i + 1]}, b2));
  return make_uint4(w[0], w[1], w[2], w[3]);
}

__device__ __forceinline__ float gq_row_max4(float x) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float gq_row_sum4(float x) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Two blocks per compute unit (two waves per SIMD, so one wave's products
// overlap the other's softmax): at most 256 registers a wave.
template <int RT, bool HILO>
__global__ __launch_bounds__(256, 2) void k_attn_gq(AttnArgs a, int row_groups) {
  constexpr int E = 8;          // bf16 per 16-byte lane chunk
  constexpr int KF = 32;        // dims per MFMA step
  constexpr int NDS = GQ_HD / KF;   // 4 dim steps of S
  constexpr int NDT = GQ_HD / 16;   // 8 dim tiles of O
  __shared__ __attribute__((aligned(16))) unsigned char lds[GQ_NST * GQ_STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, q = lane >> 4;
  // block -> (KV head g, key range kr, row group rg); the row groups of one
  // (g, kr) share its chunks, so they sit on one XCD (blocks are dispatched
  // round-robin over the 8 XCDs)
  const int b = blockIdx.x, xcd = b & 7, slot = b >> 3;
  const int rg = slot % row_groups;
  const int wk = (slot / row_groups) * 8 + xcd;
  if (wk >= a.n_kv * a.n_splits) return;
  const int g = wk / a.n_splits, kr = wk % a.n_splits;
  const int M = a.M, G = a.group, V = G * M;

  const int k0 = kr * a.chunk_keys;
  const int kb = min(k0 + a.chunk_keys, a.keys_bound);
  const int nchunks = kb > k0 ? (kb - k0 + GQ_KC - 1) / GQ_KC : 0;

  // K/V planes of (layer, g)
  const bf16_t *kplane = (const bf16_t *)a.cache + ((int64_t)(a.layer * 2 + 0) * a.n_kv + g) * a.plane;
  const bf16_t *vplane = (const bf16_t *)a.cache + ((int64_t)(a.layer * 2 + 1) * a.n_kv + g) * a.plane;
  const uint32_t plane_bytes = (uint32_t)(a.plane * 2);
  const rsrc_t kr_ = make_rsrc(kplane, plane_bytes);
  const rsrc_t vr_ = make_rsrc(vplane, plane_bytes);

  // chunk loads: thread tid carries K pieces tid, tid + 256 (key = p / 16,
  // 16-byte piece p % 16 of its row) and the V pieces of keys 2 kp, 2 kp + 1
  // (kp = tid % 16) at dimensions 8 dg .. 8 dg + 7 (dg = tid / 16)
  uint4 pa[4], pb[4];
  const int kp = tid & 15, dg = tid >> 4;
  auto issue = [&](uint4 *pr, int c) {
    const int kc = k0 + c * GQ_KC;
    const bool in = c < nchunks;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int p = tid + 256 * i;
      const int key = kc + (p >> 4);
      pr[i] = bload16(kr_, in && key < kb ? (uint32_t)(((int64_t)key * GQ_HD + (p & 15) * E) * 2) : kOOB);
      const int vk = kc + 2 * kp + i;
      pr[2 + i] = bload16(vr_, in && vk < kb ? (uint32_t)(((int64_t)vk * GQ_HD + dg * E) * 2) : kOOB);
    }
  };
  // values of keys at or past the cache end are zeroed (those slots are not
  // initialised for this step; a zero probability must not meet a NaN)
  int kend = 0;
  auto stash = [&](const uint4 *pr, int c, int stage) {
    const int kc = k0 + c * GQ_KC;
    unsigned char *st = lds + stage * GQ_STAGE;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int p = tid + 256 * i, key = p >> 4;
      *(uint4 *)(st + key * GQ_KROW + (((p & 15) ^ gq_swz(key)) * 16)) = pr[i];
    }
    const int v0 = kc + 2 * kp;
    const uint4 a0 = v0 < kend ? pr[2] : make_uint4(0, 0, 0, 0);
    const uint4 a1 = v0 + 1 < kend ? pr[3] : make_uint4(0, 0, 0, 0);
    const uint32_t x0[4] = {a0.x, a0.y, a0.z, a0.w}, x1[4] = {a1.x, a1.y, a1.z, a1.w};
    unsigned char *vt = st + GQ_KBYTES + kp * 4;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const uint32_t lo = (x0[e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
      const uint32_t hi = (x1[e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
      *(uint32_t *)(vt + (dg * E + e) * GQ_VROW) = lo | (hi << 16);
    }
  };

  issue(pa, 0);
  issue(pb, 1);

  // query fragments and per-row visibility of the wave's virtual rows
  const int vbase = (rg * 4 + wid) * RT * 16;
  uint4 qf[RT][NDS];
  int jrow[RT], hrow[RT];
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    const int v = vbase + t * 16 + (lane & 15);
    const bool real = v < V;
    const int hl = real ? v / M : 0, j = real ? v % M : 0;
    jrow[t] = real ? j : -1;
    hrow[t] = g * G + hl;
    const bf16_t *qrow = (const bf16_t *)a.q + (int64_t)j * a.ldq + hrow[t] * GQ_HD;
#pragma unroll
    for (int d = 0; d < NDS; ++d)
      qf[t][d] = real ? *(const uint4 *)(qrow + d * KF + q * E) : make_uint4(0, 0, 0, 0);
  }
  const int P = *a.kv_len;
  kend = P + M;
  const int k1 = min(k0 + a.chunk_keys, kend);
  int lim[RT];
  uint64_t anc[RT];
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    const int j = jrow[t] < 0 ? 0 : jrow[t];
    lim[t] = jrow[t] < 0 ? 0 : (a.tree ? k1 : min(k1, P + j + 1));
    anc[t] = a.tree ? a.anc[j] : 0ull;
  }

  float m_run[RT], l_run[RT];
  f32x4 o[RT][NDT];
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    m_run[t] = -INFINITY;
    l_run[t] = 0.f;
#pragma unroll
    for (int u = 0; u < NDT; ++u) o[t][u] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  stash(pa, 0, 0);
  issue(pa, 2);
  stash(pb, 1, 1);
  issue(pb, 3);
  __syncthreads();

  const float sc = a.scale_log2;
  constexpr float kSlack = 8.f;  // log2 headroom of the reference maximum
  const int r = lane & 15;
  // Scores of chunk c: S^T = K Q^T (keys permuted so that lane quarter q ends
  // up with keys q*E .. q*E + E - 1 of its row). Issued one chunk ahead of
  // the softmax that uses them, so the matrix products of chunk c + 1 run
  // while the vector units do chunk c's softmax.
  auto qk = [&](int c, int stage, float (&sv)[RT][E]) {
    const int kc = k0 + c * GQ_KC;
    if (c >= nchunks || kc >= k1) return;  // uniform over the block
    const unsigned char *st = lds + stage * GQ_STAGE;
    uint4 kf[2][NDS];
#pragma unroll
    for (int cg = 0; cg < 2; ++cg) {
      const int kl = E * (r >> 2) + 4 * cg + (r & 3);
#pragma unroll
      for (int d = 0; d < NDS; ++d)
        kf[cg][d] = *(const uint4 *)(st + kl * GQ_KROW + (((4 * d + q) ^ gq_swz(kl)) * 16));
    }
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
      for (int cg = 0; cg < 2; ++cg) {
        f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int d = 0; d < NDS; ++d) acc = mma<bf16_t>(kf[cg][d], qf[t][d], acc);
#pragma unroll
        for (int i = 0; i < 4; ++i) sv[t][4 * cg + i] = acc[i];
      }
  };
  // softmax of chunk c and O^T += V^T P^T
  auto soft_pv = [&](int c, int stage, float (&sin)[RT][E]) {
    const int kc = k0 + c * GQ_KC;
    if (c >= nchunks || kc >= k1) return;  // uniform over the block
    const unsigned char *st = lds + stage * GQ_STAGE;
    auto vfrag = [&](int u) {
      return *(const uint4 *)(st + GQ_KBYTES + (u * 16 + r) * GQ_VROW + q * 16);
    };
    const int kl0 = kc + q * E;  // first key of this lane's score chunk
    const bool all_visible = kc + GQ_KC <= min(P, k1);
#pragma unroll
    for (int t = 0; t < RT; ++t) {
      float sv[E];
#pragma unroll
      for (int e = 0; e < E; ++e) sv[e] = sin[t][e];
      if (!all_visible) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const int key = kl0 + e;
          bool vis = key < lim[t];
          if (a.tree) vis &= (key < P) | (((anc[t] >> ((key - P) & 63)) & 1ull) != 0);
          sv[e] = vis ? sv[e] : -INFINITY;
        }
      }
      float cmax = fmaxf(fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3])),
                         fmaxf(fmaxf(sv[4], sv[5]), fmaxf(sv[6], sv[7])));
      cmax = gq_row_max4(cmax);
      // the reference maximum of a row moves only when that row outgrows it
      // (rows that did not grow scale by exactly 1)
      const bool grow = m_run[t] == -INFINITY ? cmax > -INFINITY : (cmax - m_run[t]) * sc > kSlack;
      if (__any(grow)) {
        const float m_new = grow ? fmaxf(m_run[t], cmax) : m_run[t];
        const float alpha = grow ? __builtin_amdgcn_exp2f((m_run[t] - m_new) * sc) : 1.f;
        l_run[t] *= alpha;
#pragma unroll
        for (int u = 0; u < NDT; ++u) o[t][u] *= alpha;
        m_run[t] = m_new;
      }
      const float msc = m_run[t] == -INFINITY ? 0.f : m_run[t] * sc;
      float p[E];
#pragma unroll
      for (int e = 0; e < E; ++e) p[e] = __builtin_amdgcn_exp2f(fmaf(sv[e], sc, -msc));  // exp2(-inf) = 0
      l_run[t] += ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
      const uint4 phi = pack8_bf16(p);
      uint4 plo = make_uint4(0, 0, 0, 0);
      if (HILO) {
        float lo[E];
        const uint32_t w[4] = {phi.x, phi.y, phi.z, phi.w};
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const uint32_t h16 = (w[e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
          lo[e] = p[e] - __uint_as_float(h16 << 16);
        }
        plo = pack8_bf16(lo);
      }
#pragma unroll
      for (int u = 0; u < NDT; ++u) {
        const uint4 vf = vfrag(u);
        o[t][u] = mma<bf16_t>(vf, phi, o[t][u]);
        if (HILO) o[t][u] = mma<bf16_t>(vf, plo, o[t][u]);
      }
    }
  };

  float sA[RT][E], sB[RT][E];
  qk(0, 0, sA);
  for (int c = 0; c < nchunks; c += 2) {
    qk(c + 1, (c + 1) % GQ_NST, sB);
    soft_pv(c, c % GQ_NST, sA);
    stash(pa, c + 2, (c + 2) % GQ_NST);
    issue(pa, c + 4);
    __syncthreads();
    qk(c + 2, (c + 2) % GQ_NST, sA);
    soft_pv(c + 1, (c + 1) % GQ_NST, sB);
    stash(pb, c + 3, (c + 3) % GQ_NST);
    issue(pb, c + 5);
    __syncthreads();
  }

  // partial of key range kr: lane holds O^T[d = u*16 + 4q + i][row lane%16]
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    const float l = gq_row_sum4(l_run[t]);
    const int j = jrow[t];
    if (j >= 0) {
      float *po = a.part_o + (((int64_t)hrow[t] * a.n_splits + kr) * a.rowpad + j) * GQ_HD;
#pragma unroll
      for (int u = 0; u < NDT; ++u)
        *(float4 *)(po + u * 16 + 4 * q) = make_float4(o[t][u][0], o[t][u][1], o[t][u][2], o[t][u][3]);
      if (q == 0) {
        float *pml = a.part_ml + (((int64_t)hrow[t] * a.n_splits + kr) * a.rowpad + j) * 2;
        pml[0] = m_run[t] == -INFINITY ? -INFINITY : m_run[t] * sc;
        pml[1] = l;
      }
    }
  }
}

}  // namespace

// Tiles per wave: one (16 virtual rows per wave, 64 per block); a step's
// virtual rows are spread over row groups of blocks, each with its own K/V
// chunks from L2. Two tiles per wave (half the blocks) and twice the key
// ranges measured the same or slower on the 7B step (20.7-25.7 us).
int attn_gq_tiles(int group, int rows) {
  (void)group;
  (void)rows;
  return 1;
}

int attn_gq_row_groups(int group, int rows) {
  const int v = group * rows;
  const int per = 64 * attn_gq_tiles(group, rows);
  return (v + per - 1) / per;
}

bool attn_gq_supported(bool bf16, int head_dim) { return bf16 && head_dim == GQ_HD; }

template <bool HILO>
static hipError_t launch_gq(const AttnArgs &a, hipStream_t s) {
  const int rt = attn_gq_tiles(a.group, a.M);
  const int rgs = attn_gq_row_groups(a.group, a.M);
  const int works = a.n_kv * a.n_splits;
  dim3 grid(8 * rgs * ((works + 7) / 8));
  switch (rt) {
    case 1: PF_TRY(launch_k(k_attn_gq<1, HILO>, grid, dim3(256), s, a, rgs)); break;
    default: return hipErrorInvalidValue;
  }
  return hipSuccess;
}

hipError_t launch_attn_gq(const AttnArgs &a, bool hilo, hipStream_t s) {
  if (!attn_gq_supported(true, a.head_dim) || a.chunk_keys % GQ_KC != 0 || a.M < 1 ||
      a.n_splits < 1 || a.plane * 2 >= (int64_t)1 << 31 || a.keys_bound < 0)
    return hipErrorInvalidValue;
  PF_TRY(hilo ? launch_gq<true>(a, s) : launch_gq<false>(a, s));
  return launch_attn_combine(true, a, s);
}

}  // namespace pf
