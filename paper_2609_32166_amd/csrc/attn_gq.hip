// Grouped verify attention for bf16 models with head_dim 128: one block per
// (KV head, key range, row group). The rows of a block are "virtual rows":
// every (query head of the KV group, draft row) pair, head-major, so the
// group's query heads share one copy of each K/V chunk. A chunk (32 keys:
// 8 KiB of keys, 8 KiB of values, both [slot][head_dim] rows in the cache) is
// loaded once per block by all 256 threads into registers a phase ahead,
// stored into LDS row-major as in the cache, and read from there by the four
// waves, each of which holds one 16-row tile of virtual rows (the value
// product's operand, eight keys of one dimension per lane, through
// transposing LDS reads). Per
// wave and chunk: S^T = K Q^T with the permuted key rows, the log2-domain
// online softmax with the deferred rescale, then O^T += V^T P^T, two chunks
// per phase. The probabilities enter the value product as two bf16 terms
// (p = hi + lo, lo = the rounding residue of hi), so the product sees them to
// about 16 significant bits instead of 8 (HILO; without it, one term).
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
// Staged keys: [key] rows of 256 bytes padded to 272, so the 16 consecutive
// keys one operand read touches start on 16 distinct 16-byte bank groups.
// Staged values: [key] rows padded to 288 bytes, so the four keys x 32 bytes
// one 16-lane group of a transposing read touches fall on distinct banks.
constexpr int GQ_KROW = GQ_HD * 2 + 16;            // 272
constexpr int GQ_VROW = GQ_HD * 2 + 32;            // 288: value rows [key][dim], padded
constexpr int GQ_KBYTES = GQ_KC * GQ_KROW;         // 8704
constexpr int GQ_STAGE = GQ_KBYTES + GQ_KC * GQ_VROW;  // 17920
constexpr int GQ_CHUNK_BYTES = GQ_KC * GQ_HD * 2;  // 8192 bytes of one plane per chunk

__device__ inline uint4 pack8_bf16(const float *p) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  typedef __bf16 b2 __attribute__((ext_vector_type(2)));
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f2){p[2 * i], p[2 * i + 1]}, b2));
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// Value operand from two transposing 64-bit LDS reads (gfx950
// ds_read_b64_tr_b16: within a group of 16 lanes the lanes' four 16-bit
// elements are concatenated, A[4 s + e], and lane i receives A[i + 16 j]),
// elements 0-3 from the first address, 4-7 from the second.
typedef short gq_v4s __attribute__((ext_vector_type(4)));
__device__ inline uint4 gq_read_tr(const unsigned char *p0, const unsigned char *p1) {
  const gq_v4s a = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) gq_v4s *)(const_cast<unsigned char *>(p0)));
  const gq_v4s b = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) gq_v4s *)(const_cast<unsigned char *>(p1)));
  const uint2 x = __builtin_bit_cast(uint2, a), y = __builtin_bit_cast(uint2, b);
  return make_uint4(x.x, x.y, y.x, y.y);
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

// The whole offset goes in the vector operand: the descriptor's bound checks
// that operand (plus the instruction's constant), not the scalar offset.
__device__ __forceinline__ uint4 gq_load(rsrc_t r, uint32_t off) {
  v4u v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// A phase takes two 32-key chunks (two LDS stages of two chunks each, one
// barrier and one stash per 64 keys) and one softmax update for both, so the
// two chunks' exponentials, packs and value products are independent work
// for the wave. The reference maximum moves only when a row outgrows it over
// the phase's 64 keys. Two blocks per compute unit (two waves per SIMD): at
// most 256 registers a wave.
template <bool HILO>
__global__ __launch_bounds__(256, 2) void k_attn_gq(AttnArgs a, int row_groups) {
  constexpr int E = 8;          // bf16 per 16-byte lane chunk
  constexpr int KF = 32;        // dims per MFMA step
  constexpr int NDS = GQ_HD / KF;   // 4 dim steps of S
  constexpr int NDT = GQ_HD / 16;   // 8 dim tiles of O
  constexpr int PH = 2 * GQ_STAGE;  // bytes of one stage (two chunks)
  __shared__ __attribute__((aligned(16))) unsigned char lds[2 * PH];

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, q = lane >> 4;
  const int b = blockIdx.x, xcd = b & 7, slot = b >> 3;
  const int rg = slot % row_groups;
  const int wk = (slot / row_groups) * 8 + xcd;
  if (wk >= a.n_kv * a.n_splits) return;
  const int g = wk / a.n_splits, kr = wk % a.n_splits;
  const int M = a.M, G = a.group, V = G * M;

  const int k0 = kr * a.chunk_keys;
  const int kb = min(k0 + a.chunk_keys, a.keys_bound);
  const int nchunks = kb > k0 ? (kb - k0 + GQ_KC - 1) / GQ_KC : 0;

  const int64_t roff = (int64_t)k0 * GQ_HD;
  const bf16_t *kplane = (const bf16_t *)a.cache + ((int64_t)(a.layer * 2 + 0) * a.n_kv + g) * a.plane + roff;
  const bf16_t *vplane = (const bf16_t *)a.cache + ((int64_t)(a.layer * 2 + 1) * a.n_kv + g) * a.plane + roff;
  const rsrc_t kr_ = make_rsrc(kplane, (uint32_t)max(kb - k0, 0) * (GQ_HD * 2));

  uint4 pr[2][4];  // the next phase's two chunks in flight
  const int kp = tid & 15, dg = tid >> 4;
  const uint32_t koff = (uint32_t)tid * 16u;
  const uint32_t voff = koff;
  auto issue_k = [&](uint4 *r4, int c) {
    const uint32_t so = (uint32_t)c * GQ_CHUNK_BYTES;
    r4[0] = gq_load(kr_, koff + so);
    r4[1] = gq_load(kr_, koff + so + 4096u);
  };
  auto issue_v = [&](rsrc_t vr, uint4 *r4, int c) {
    const uint32_t so = (uint32_t)c * GQ_CHUNK_BYTES;
    r4[2] = gq_load(vr, voff + so);
    r4[3] = gq_load(vr, voff + so + 4096u);
  };
  {
    const rsrc_t vr0 = make_rsrc(vplane, (uint32_t)max(kb - k0, 0) * (GQ_HD * 2));
    issue_k(pr[0], 0);
    issue_v(vr0, pr[0], 0);
    issue_k(pr[1], 1);
    issue_v(vr0, pr[1], 1);
  }
  const int P = *a.kv_len;
  const int kend = P + M;
  const rsrc_t vr_ = make_rsrc(vplane, (uint32_t)max(min(kb, kend) - k0, 0) * (GQ_HD * 2));

  const int kst = (tid >> 4) * GQ_KROW + (tid & 15) * 16;
  const int vst = GQ_KBYTES + (tid >> 4) * GQ_VROW + (tid & 15) * 16;
  const int r = lane & 15;
  const int kld = r * GQ_KROW + q * 16;
  // value operand of lane quarter q: the probabilities' keys 4q..4q+3 and
  // 16+4q..16+4q+3 of the chunk (the score layout). Transposing reads: source
  // lane s of quarter q points at key 4q + s / 4 (+16 for the second read),
  // dims 16u + 4 (s % 4) .. + 3, so lane i receives dim 16u + i of the four
  // keys
  const int vld = GQ_KBYTES + (4 * q + (r >> 2)) * GQ_VROW + 8 * (r & 3);
  // chunk i (0, 1) of stage sg
  auto stash = [&](const uint4 *r4, int sg, int i, int zero_from) {
    unsigned char *st = lds + sg * PH + i * GQ_STAGE;
    *(uint4 *)(st + kst) = r4[0];
    *(uint4 *)(st + kst + 16 * GQ_KROW) = r4[1];
    *(uint4 *)(st + vst) = (tid >> 4) < zero_from ? r4[2] : make_uint4(0, 0, 0, 0);
    *(uint4 *)(st + vst + 16 * GQ_VROW) = (tid >> 4) + 16 < zero_from ? r4[3] : make_uint4(0, 0, 0, 0);
  };

  // query fragments and visibility of the wave's 16 virtual rows
  const int v = (rg * 4 + wid) * 16 + (lane & 15);
  const bool real = v < V;
  const int hl = real ? v / M : 0, jr = real ? v % M : 0;
  const int jrow = real ? jr : -1;
  const int hrow = g * G + hl;
  uint4 qf[NDS];
  {
    const bf16_t *qrow = (const bf16_t *)a.q + (int64_t)jr * a.ldq + hrow * GQ_HD;
#pragma unroll
    for (int d = 0; d < NDS; ++d) qf[d] = real ? *(const uint4 *)(qrow + d * KF + q * E) : make_uint4(0, 0, 0, 0);
  }
  const int k1 = min(k0 + a.chunk_keys, kend);
  const int lim = jrow < 0 ? 0 : (a.tree ? k1 : min(k1, P + jr + 1));
  const uint64_t anc = a.tree ? a.anc[jr] : 0ull;

  float m_run = -INFINITY, l_run = 0.f;
  f32x4 o[NDT];
#pragma unroll
  for (int u = 0; u < NDT; ++u) o[u] = f32x4{0.f, 0.f, 0.f, 0.f};

  stash(pr[0], 0, 0, kend - k0);
  stash(pr[1], 0, 1, kend - k0 - GQ_KC);
  issue_k(pr[0], 2);
  issue_v(vr_, pr[0], 2);
  issue_k(pr[1], 3);
  issue_v(vr_, pr[1], 3);
  __syncthreads();

  const float sc = a.scale_log2;
  constexpr float kSlack = 8.f;
  // scores of chunk i of stage sg: lane quarter c of row lane % 16 gets keys
  // 4c..4c+3 and 16+4c..16+4c+3 of the chunk
  auto qk = [&](int sg, int i, float (&sv)[E]) {
    const unsigned char *st = lds + sg * PH + i * GQ_STAGE + kld;
    uint4 kf[2][NDS];
#pragma unroll
    for (int cg = 0; cg < 2; ++cg)
#pragma unroll
      for (int d = 0; d < NDS; ++d) kf[cg][d] = *(const uint4 *)(st + cg * 16 * GQ_KROW + d * 64);
#pragma unroll
    for (int cg = 0; cg < 2; ++cg) {
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int d = 0; d < NDS; ++d) acc = mma<bf16_t>(kf[cg][d], qf[d], acc);
#pragma unroll
      for (int e = 0; e < 4; ++e) sv[4 * cg + e] = acc[e];
    }
  };
  auto mask = [&](int kc, float (&sv)[E]) {
    const int kl0 = kc + q * 4;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int key = kl0 + (e & 3) + 16 * (e >> 2);
      bool vis = key < lim;
      if (a.tree) vis &= (key < P) | (((anc >> ((key - P) & 63)) & 1ull) != 0);
      sv[e] = vis ? sv[e] : -INFINITY;
    }
  };
  auto pv = [&](int sg, int i, const float (&p)[E]) {
    const unsigned char *st = lds + sg * PH + i * GQ_STAGE + vld;
    uint4 vf[NDT];
#pragma unroll
    for (int u = 0; u < NDT; ++u) vf[u] = gq_read_tr(st + 32 * u, st + 32 * u + 16 * GQ_VROW);
    const uint4 phi = pack8_bf16(p);
    uint4 plo = make_uint4(0, 0, 0, 0);
    if (HILO) {
      float lo[E];
      const uint32_t w[4] = {phi.x, phi.y, phi.z, phi.w};
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const uint32_t h = (e & 1) ? (w[e >> 1] & 0xFFFF0000u) : (w[e >> 1] << 16);
        lo[e] = p[e] - __uint_as_float(h);
      }
      plo = pack8_bf16(lo);
    }
#pragma unroll
    for (int u = 0; u < NDT; ++u) {
      o[u] = mma<bf16_t>(vf[u], phi, o[u]);
      if (HILO) o[u] = mma<bf16_t>(vf[u], plo, o[u]);
    }
  };

  for (int c = 0; c < nchunks; c += 2) {
    const int sg = (c >> 1) & 1;
    const int kcA = k0 + c * GQ_KC, kcB = kcA + GQ_KC;
    const bool vA = kcA < k1, vB = c + 1 < nchunks && kcB < k1;  // uniform over the block
    if (vA) {
      float sA[E], sB[E];
      qk(sg, 0, sA);
      if (vB) {
        qk(sg, 1, sB);
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) sB[e] = -INFINITY;
      }
      if (!(kcB + GQ_KC <= min(P, k1))) {
        mask(kcA, sA);
        if (vB) mask(kcB, sB);
      }
      float cmax = fmaxf(fmaxf(fmaxf(fmaxf(sA[0], sA[1]), fmaxf(sA[2], sA[3])),
                               fmaxf(fmaxf(sA[4], sA[5]), fmaxf(sA[6], sA[7]))),
                         fmaxf(fmaxf(fmaxf(sB[0], sB[1]), fmaxf(sB[2], sB[3])),
                               fmaxf(fmaxf(sB[4], sB[5]), fmaxf(sB[6], sB[7]))));
      cmax = gq_row_max4(cmax);
      const bool grow = m_run == -INFINITY ? cmax > -INFINITY : (cmax - m_run) * sc > kSlack;
      if (__any(grow)) {
        const float m_new = grow ? fmaxf(m_run, cmax) : m_run;
        const float alpha = grow ? __builtin_amdgcn_exp2f((m_run - m_new) * sc) : 1.f;
        l_run *= alpha;
#pragma unroll
        for (int u = 0; u < NDT; ++u) o[u] *= alpha;
        m_run = m_new;
      }
      const float msc = m_run == -INFINITY ? 0.f : m_run * sc;
      float pA[E], pB[E];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        pA[e] = __builtin_amdgcn_exp2f(fmaf(sA[e], sc, -msc));  // exp2(-inf) = 0
        pB[e] = __builtin_amdgcn_exp2f(fmaf(sB[e], sc, -msc));
      }
      l_run += (((pA[0] + pA[1]) + (pA[2] + pA[3])) + ((pA[4] + pA[5]) + (pA[6] + pA[7]))) +
               (((pB[0] + pB[1]) + (pB[2] + pB[3])) + ((pB[4] + pB[5]) + (pB[6] + pB[7])));
      pv(sg, 0, pA);
      if (vB) pv(sg, 1, pB);
    }
    // the next phase's chunks into the other stage, the one after into registers
    stash(pr[0], sg ^ 1, 0, GQ_KC);
    stash(pr[1], sg ^ 1, 1, GQ_KC);
    issue_k(pr[0], c + 4);
    issue_v(vr_, pr[0], c + 4);
    issue_k(pr[1], c + 5);
    issue_v(vr_, pr[1], c + 5);
    __syncthreads();
  }

  const float l = gq_row_sum4(l_run);
  if (jrow >= 0) {
    float *po = a.part_o + (((int64_t)hrow * a.n_splits + kr) * a.rowpad + jrow) * GQ_HD;
#pragma unroll
    for (int u = 0; u < NDT; ++u)
      *(float4 *)(po + u * 16 + 4 * q) = make_float4(o[u][0], o[u][1], o[u][2], o[u][3]);
    if (q == 0) {
      float *pml = a.part_ml + (((int64_t)hrow * a.n_splits + kr) * a.rowpad + jrow) * 2;
      pml[0] = m_run == -INFINITY ? -INFINITY : m_run * sc;
      pml[1] = l;
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
  if (rt != 1) return hipErrorInvalidValue;
  PF_TRY(launch_k(k_attn_gq<HILO>, grid, dim3(256), s, a, rgs));
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
