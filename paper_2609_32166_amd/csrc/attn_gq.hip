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
// Staged keys: [key] rows of 256 bytes padded to 272, so the 16 consecutive
// keys one operand read touches start on 16 distinct 16-byte bank groups.
// Staged values: [dim] rows of the chunk's 32 keys (80 bytes with padding, so
// the 16 dimensions of a read fall on distinct bank groups), keys permuted
// within the row to match the score layout: key k = 16a + 4c + b sits at
// position 8c + 4a + b, so lane quarter c finds the eight keys its
// probabilities belong to (4c..4c+3 and 16+4c..16+4c+3) in one 16-byte read.
constexpr int GQ_KROW = GQ_HD * 2 + 16;            // 272
constexpr int GQ_VROW = GQ_KC * 2 + 16;            // 80
constexpr int GQ_KBYTES = GQ_KC * GQ_KROW;         // 8704
constexpr int GQ_STAGE = GQ_KBYTES + GQ_HD * GQ_VROW;  // 18944
constexpr int GQ_NST = 3;                          // LDS stages
constexpr int GQ_CHUNK_BYTES = GQ_KC * GQ_HD * 2;  // 8192 bytes of one plane per chunk
__device__ constexpr int gq_vpos(int k) { return ((k >> 2) & 3) * 8 + (k >> 4) * 4 + (k & 3); }

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

// The whole offset goes in the vector operand: the descriptor's bound checks
// that operand (plus the instruction's constant), not the scalar offset.
__device__ __forceinline__ uint4 gq_load(rsrc_t r, uint32_t off) {
  v4u v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
  return make_uint4(v.x, v.y, v.z, v.w);
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

  // K/V rows of the range in (layer, g): buffer resources based at its
  // first key and bounded at its last (keys, which masking hides past the
  // cache end) or at the cache end (values: slots past it are not
  // initialised for this step and a zero probability must not meet a NaN),
  // so loads past either bound return zeros without a select
  const int64_t roff = (int64_t)k0 * GQ_HD;
  const bf16_t *kplane = (const bf16_t *)a.cache + ((int64_t)(a.layer * 2 + 0) * a.n_kv + g) * a.plane + roff;
  const bf16_t *vplane = (const bf16_t *)a.cache + ((int64_t)(a.layer * 2 + 1) * a.n_kv + g) * a.plane + roff;
  const rsrc_t kr_ = make_rsrc(kplane, (uint32_t)max(kb - k0, 0) * (GQ_HD * 2));

  // chunk loads: thread tid carries K pieces tid, tid + 256 (16-byte piece
  // p % 16 of key p / 16) and the V pieces of keys 2 kp, 2 kp + 1 (kp = tid %
  // 16) at dimensions 8 dg .. 8 dg + 7 (dg = tid / 16)
  uint4 pa[4], pb[4];
  const int kp = tid & 15, dg = tid >> 4;
  const uint32_t koff = (uint32_t)tid * 16u;
  const uint32_t voff = (uint32_t)(2 * kp * GQ_HD + dg * E) * 2u;
  auto issue_k = [&](uint4 *pr, int c) {
    const uint32_t so = (uint32_t)c * GQ_CHUNK_BYTES;
    pr[0] = gq_load(kr_, koff + so);
    pr[1] = gq_load(kr_, koff + so + 4096u);
  };
  // the first two chunks' values are fetched before the cache length is
  // known (bounded at the range end) and zeroed past the cache end on the way
  // into LDS; later chunks use the resource bounded at the cache end
  auto issue_v = [&](rsrc_t vr, uint4 *pr, int c) {
    const uint32_t so = (uint32_t)c * GQ_CHUNK_BYTES;
    pr[2] = gq_load(vr, voff + so);
    pr[3] = gq_load(vr, voff + so + GQ_HD * 2u);
  };
  {
    const rsrc_t vr0 = make_rsrc(vplane, (uint32_t)max(kb - k0, 0) * (GQ_HD * 2));
    issue_k(pa, 0);
    issue_v(vr0, pa, 0);
    issue_k(pb, 1);
    issue_v(vr0, pb, 1);
  }
  const int P = *a.kv_len;
  const int kend = P + M;
  const rsrc_t vr_ = make_rsrc(vplane, (uint32_t)max(min(kb, kend) - k0, 0) * (GQ_HD * 2));
  auto issue = [&](uint4 *pr, int c) {
    issue_k(pr, c);
    issue_v(vr_, pr, c);
  };

  // LDS addresses: stores of a thread's pieces, operand reads of a lane
  const int kst = (tid >> 4) * GQ_KROW + (tid & 15) * 16;          // key piece tid
  const int vst = GQ_KBYTES + 8 * dg * GQ_VROW + gq_vpos(2 * kp) * 2;  // dim 8 dg, keys 2kp, 2kp+1
  const int r = lane & 15;
  const int kld = r * GQ_KROW + q * 16;                             // key r (+16 cg), granule q (+4 d)
  const int vld = GQ_KBYTES + r * GQ_VROW + q * 16;                 // dim r (+16 u), keys of quarter q
  auto stash = [&](const uint4 *pr, int stage, int zero_from) {
    unsigned char *st = lds + stage * GQ_STAGE;
    *(uint4 *)(st + kst) = pr[0];
    *(uint4 *)(st + kst + 16 * GQ_KROW) = pr[1];
    // zero_from: first key (relative to the chunk) whose values are zeroed
    // here (only the first two chunks need it)
    const uint4 a0 = 2 * kp < zero_from ? pr[2] : make_uint4(0, 0, 0, 0);
    const uint4 a1 = 2 * kp + 1 < zero_from ? pr[3] : make_uint4(0, 0, 0, 0);
    const uint32_t x0[4] = {a0.x, a0.y, a0.z, a0.w};
    const uint32_t x1[4] = {a1.x, a1.y, a1.z, a1.w};
#pragma unroll
    for (int e = 0; e < E; ++e) {
      // low half: key 2kp, high half: key 2kp + 1, at dimension 8 dg + e
      const uint32_t w = (e & 1) ? __builtin_amdgcn_perm(x1[e >> 1], x0[e >> 1], 0x07060302u)
                                 : __builtin_amdgcn_perm(x1[e >> 1], x0[e >> 1], 0x05040100u);
      *(uint32_t *)(st + vst + e * GQ_VROW) = w;
    }
  };

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

  stash(pa, 0, kend - k0);
  issue(pa, 2);
  stash(pb, 1, kend - k0 - GQ_KC);
  issue(pb, 3);
  __syncthreads();

  const float sc = a.scale_log2;
  constexpr float kSlack = 8.f;  // log2 headroom of the reference maximum
  // Scores of chunk c: S^T = K Q^T over two 16-key tiles; lane quarter c of
  // row lane % 16 ends up with keys 4c..4c+3 (first tile) and 16+4c..16+4c+3
  // (second tile). Issued one chunk ahead of the softmax that uses them, so
  // the matrix products of chunk c + 1 run while the vector units do chunk
  // c's softmax.
  auto load_k = [&](int stage, uint4 (&kf)[2][NDS]) {
    const unsigned char *st = lds + stage * GQ_STAGE + kld;
#pragma unroll
    for (int cg = 0; cg < 2; ++cg)
#pragma unroll
      for (int d = 0; d < NDS; ++d) kf[cg][d] = *(const uint4 *)(st + cg * 16 * GQ_KROW + d * 64);
  };
  auto load_v = [&](int stage, uint4 (&vf)[NDT]) {
    const unsigned char *st = lds + stage * GQ_STAGE + vld;
#pragma unroll
    for (int u = 0; u < NDT; ++u) vf[u] = *(const uint4 *)(st + u * 16 * GQ_VROW);
  };
  auto qk = [&](int c, const uint4 (&kf)[2][NDS], float (&sv)[RT][E]) {
    const int kc = k0 + c * GQ_KC;
    if (c >= nchunks || kc >= k1) return;  // uniform over the block
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
  auto soft_pv = [&](int c, const uint4 (&vf)[NDT], float (&sin)[RT][E]) {
    const int kc = k0 + c * GQ_KC;
    if (c >= nchunks || kc >= k1) return;  // uniform over the block
    const int kl0 = kc + q * 4;  // keys kl0 + (e & 3) + 16 (e >> 2) of this lane's scores
    const bool all_visible = kc + GQ_KC <= min(P, k1);
#pragma unroll
    for (int t = 0; t < RT; ++t) {
      float sv[E];
#pragma unroll
      for (int e = 0; e < E; ++e) sv[e] = sin[t][e];
      if (!all_visible) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const int key = kl0 + (e & 3) + 16 * (e >> 2);
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
          const uint32_t h = (e & 1) ? (w[e >> 1] & 0xFFFF0000u) : (w[e >> 1] << 16);
          lo[e] = p[e] - __uint_as_float(h);
        }
        plo = pack8_bf16(lo);
      }
#pragma unroll
      for (int u = 0; u < NDT; ++u) {
        o[t][u] = mma<bf16_t>(vf[u], phi, o[t][u]);
        if (HILO) o[t][u] = mma<bf16_t>(vf[u], plo, o[t][u]);
      }
    }
  };

  // One phase: the LDS reads of chunk c + 1's keys and chunk c's values go
  // out first, then chunk c + 1's score products, chunk c's softmax and
  // value products, the stash of chunk c + 2 and the loads of chunk c + 4.
  float sA[RT][E], sB[RT][E];
  {
    uint4 kf[2][NDS];
    load_k(0, kf);
    qk(0, kf, sA);
  }
  auto phase = [&](int c, float (&scur)[RT][E], float (&snext)[RT][E], uint4 *pr) {
    uint4 kf[2][NDS], vf[NDT];
    load_k((c + 1) % GQ_NST, kf);
    load_v(c % GQ_NST, vf);
    qk(c + 1, kf, snext);
    soft_pv(c, vf, scur);
    stash(pr, (c + 2) % GQ_NST, GQ_KC);
    issue(pr, c + 4);
    __syncthreads();
  };
  for (int c = 0; c < nchunks; c += 2) {
    phase(c, sA, sB, pa);
    phase(c + 1, sB, sA, pb);
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
