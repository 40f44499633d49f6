// Grouped-query verify attention. Each query row (draft node j, head h)
// attends to the cached keys 0..P-1 and to the draft keys P..P+M-1 it may
// see (causal for a linear draft, ancestors-or-self for a tree).
//
// Work split: one wave per (key range, query head, 32 query rows); the heads
// of a group read the same K/V fragments, which they share through L2. The
// host sizes the ranges so that every wave of the launch is resident at once
// (one wave per SIMD at this register footprint). The loop body is kept
// small (every wave runs it only a few times, so instruction fetch of a long
// unrolled body would dominate). Keys are processed in chunks of 4*E (32 bf16 / 16 fp32). S^T = K Q^T is formed
// with K as the MFMA A operand, permuting which key each A row carries so
// that, after the MFMA, lane quarter q holds the scores of keys q*E..q*E+E-1
// of its query row (column). That is exactly the B-operand layout of
// O^T += V^T P^T; a lane's V^T fragment (E consecutive keys of one
// dimension, from the [slot][dim] value rows of the cache) is gathered with
// E element loads. The
// online softmax runs in the log2 domain in fp32; probabilities enter the PV
// product in the model dtype. Each block writes an unnormalised partial
// (o, running max, running sum) per row; k_attn_combine merges the splits.
#include "kernels.h"

namespace pf {

// E probabilities in [0, 1] -> one 16-byte MFMA operand chunk in the model
// dtype (bf16: hardware round-to-nearest-even conversion).
template <typename T> __device__ inline uint4 pack_probs(const float *p);
template <> __device__ inline uint4 pack_probs<float>(const float *p) {
  return make_uint4(__float_as_uint(p[0]), __float_as_uint(p[1]), __float_as_uint(p[2]),
                    __float_as_uint(p[3]));
}
template <> __device__ inline uint4 pack_probs<bf16_t>(const float *p) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  typedef __bf16 b2 __attribute__((ext_vector_type(2)));
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f2){p[2 * i], p[2 * i + 1]}, b2));
  return make_uint4(w[0], w[1], w[2], w[3]);
}
// The rounding residue of eight bf16-packed probabilities as a second bf16
// operand: the value product takes each probability as hi + lo, about 16
// significant bits (the precision contract rounds no probability).
__device__ inline uint4 pack_probs_lo(const float *p, const uint4 &hi) {
  const uint32_t w[4] = {hi.x, hi.y, hi.z, hi.w};
  float lo[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint32_t h = (e & 1) ? (w[e >> 1] & 0xFFFF0000u) : (w[e >> 1] << 16);
    lo[e] = p[e] - __uint_as_float(h);
  }
  return pack_probs<bf16_t>(lo);
}

// E consecutive keys key0 .. key0 + E - 1 of dimension dim from [slot][hd]
// value rows, packed as one 16-byte operand chunk (key0 + e in element e);
// in == false loads nothing and gives zeros.
template <typename T> __device__ inline uint4 gather_vt(rsrc_t r, bool in, int key0, int dim, int hd);
template <> __device__ inline uint4 gather_vt<float>(rsrc_t r, bool in, int key0, int dim, int hd) {
  uint32_t w[4];
#pragma unroll
  for (int e = 0; e < 4; ++e)
    w[e] = __builtin_amdgcn_raw_buffer_load_b32(
        r, in ? (int)(((int64_t)(key0 + e) * hd + dim) * 4) : (int)kOOB, 0, 0);
  return make_uint4(w[0], w[1], w[2], w[3]);
}
template <> __device__ inline uint4 gather_vt<bf16_t>(rsrc_t r, bool in, int key0, int dim, int hd) {
  uint32_t h[8];
#pragma unroll
  for (int e = 0; e < 8; ++e)
    h[e] = __builtin_amdgcn_raw_buffer_load_b16(
        r, in ? (int)(((int64_t)(key0 + e) * hd + dim) * 2) : (int)kOOB, 0, 0);
  return make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                    h[6] | (h[7] << 16));
}

// Keeps the first n (0..E) elements of a 16-byte chunk and zeroes the rest.
template <typename T> __device__ inline uint4 keep_first(uint4 v, int n) {
  constexpr int E = Elem<T>::E, PER = E / 4;  // elements per 32-bit word
  uint32_t m[4];
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    if (PER == 1) {
      m[w] = w < n ? 0xFFFFFFFFu : 0u;
    } else {
      m[w] = (2 * w < n ? 0x0000FFFFu : 0u) | (2 * w + 1 < n ? 0xFFFF0000u : 0u);
    }
  }
  return make_uint4(v.x & m[0], v.y & m[1], v.z & m[2], v.w & m[3]);
}

// Max / sum over the four lanes that hold the same MFMA row (lanes l, l^16,
// l^32, l^48) with the cross-row lane swaps (no LDS round trip): a swap of
// x with itself leaves each lane x and its partner's x in the two results.
__device__ __forceinline__ float row_max4(float x) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float row_sum4(float x) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

template <typename T, int RT, int HD, int WPE = 1, int NS = 2>
__global__ __launch_bounds__(64, WPE) void k_attn(AttnArgs a) {
  constexpr int E = Elem<T>::E;
  constexpr int KF = 4 * E;       // d per MFMA step, keys per chunk
  constexpr int KC = 4 * E;       // keys per chunk
  constexpr int NDS = HD / KF;    // d steps for S
  constexpr int NDT = HD / 16;    // d tiles of O
  constexpr int NCG = E / 4;      // key sub-groups per chunk
  const int lane = threadIdx.x & 63;
  const int q = lane >> 4;
  // XCD-aware placement: blocks are dispatched round-robin over the 8 XCDs,
  // so the `group` query heads that read the same (KV head, key range) get
  // block ids of equal residue mod 8 and share one L2.
  // A wave reduces per_wave consecutive key ranges, one after the other,
  // and writes one partial per range: every range is reduced from fresh
  // accumulators in the same order whichever wave takes it, so the result
  // does not depend on how ranges are spread over waves.
  const int b = blockIdx.x;
  const int xcd = b & 7, j = b >> 3;
  const int hl = j % a.group;
  const int nwr = (a.n_splits + a.per_wave - 1) / a.per_wave;  // wave ranges per KV head
  const int w = (j / a.group) * 8 + xcd;  // (KV head, wave range) work id
  if (w >= a.n_kv * nwr) return;
  const int g = w / nwr;
  const int s0 = (w % nwr) * a.per_wave;  // first key range of this wave
  const int h = g * a.group + hl;
  const int row0 = blockIdx.y * RT * 16;  // first query row of this wave

  const int M = a.M;
  const int k0 = s0 * a.chunk_keys;
  const int kw = k0 + a.per_wave * a.chunk_keys;  // end of the wave's keys
  const int cps = a.chunk_keys / KC;              // chunks per key range
  // Loads are bounded by the host's upper bound on P + M, so they are issued
  // without waiting for the device-side length; keys past the true end are
  // masked once P has arrived.
  const int kb = min(kw, a.keys_bound);
  const int nchunks = kb > k0 ? (kb - k0 + KC - 1) / KC : 0;

  float m_run[RT], l_run[RT];
  f32x4 o[RT][NDT];
#pragma unroll
  for (int r = 0; r < RT; ++r) {
    m_run[r] = -INFINITY;
    l_run[r] = 0.f;
#pragma unroll
    for (int t = 0; t < NDT; ++t) o[r][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // query fragments: row j = r*16 + lane%16, dims ds*KF + q*E .. +E
  uint4 qf[RT][NDS];
#pragma unroll
  for (int r = 0; r < RT; ++r) {
    const int jr = min(row0 + r * 16 + (lane & 15), a.rowpad - 1);
    const T *qrow = (const T *)a.q + (int64_t)jr * a.ldq + h * HD;
#pragma unroll
    for (int d = 0; d < NDS; ++d) qf[r][d] = *(const uint4 *)(qrow + d * KF + q * E);
  }
  const T *kplane = (const T *)a.cache + ((int64_t)(a.layer * 2 + 0) * a.n_kv + g) * a.plane;
  const T *vplane = (const T *)a.cache + ((int64_t)(a.layer * 2 + 1) * a.n_kv + g) * a.plane;
  const uint32_t plane_bytes = (uint32_t)(a.plane * sizeof(T));
  const rsrc_t kr = make_rsrc(kplane, plane_bytes);
  const rsrc_t vr = make_rsrc(vplane, plane_bytes);
  const float sc = a.scale_log2;

  // K/V chunk slots. NS >= 2: compute one chunk while the others' loads are
  // in flight. NS == 1: one slot, the next chunk's K issued as soon as the
  // score products have read the current one and its V after the value
  // products (fewer live registers). Chunks past the range load out of the
  // resource (zeros, no traffic).
  uint4 kf[NS][NCG][NDS], vf[NS][NDT];
  auto load_k = [&](int slot, int c) {
    const int kc = k0 + c * KC;
    const bool in = c < nchunks;
#pragma unroll
    for (int cg = 0; cg < NCG; ++cg) {
      const int r = lane & 15;
      const int key = kc + E * (r >> 2) + 4 * cg + (r & 3);
#pragma unroll
      for (int d = 0; d < NDS; ++d)
        kf[slot][cg][d] =
            bload16(kr, in ? (uint32_t)(((int64_t)key * HD + d * KF + q * E) * sizeof(T)) : kOOB);
    }
  };
  auto load_v = [&](int slot, int c) {
    const int kc = k0 + c * KC;
    const bool in = c < nchunks;
#pragma unroll
    for (int t = 0; t < NDT; ++t)
      vf[slot][t] = gather_vt<T>(vr, in, kc + q * E, t * 16 + (lane & 15), HD);
  };
  auto load = [&](int slot, int c) {
    load_k(slot, c);
    load_v(slot, c);
  };
#pragma unroll
  for (int u = 0; u < NS; ++u) {
    load(u, u);
    __builtin_amdgcn_sched_barrier(0);
  }

  // visibility: key < lim[r] (linear drafts: draft key P + i is seen by rows
  // j >= i), and for a tree also ancestor-or-self among the draft keys
  const int P = *a.kv_len;
  const int kend = P + M;
  const int k1 = min(kw, kend);
  int lim[RT];
  uint64_t anc[RT];
#pragma unroll
  for (int r = 0; r < RT; ++r) {
    const int jq = row0 + r * 16 + (lane & 15);
    lim[r] = a.tree ? k1 : min(k1, P + jq + 1);
    anc[r] = a.tree ? a.anc[min(jq, a.rowpad - 1)] : 0ull;
  }

  // Online softmax with a deferred rescale: m_run is a row's reference
  // maximum (raw score units) that only moves when the row's maximum exceeds
  // it by more than 2^8 in probability, so probabilities stay below 256 and
  // the accumulators are rescaled a handful of times per range instead of
  // per chunk. The result equals the usual update up to rounding.
  constexpr float kSlack = 8.f;  // log2 headroom of the reference maximum
  auto compute = [&](int slot, int c) {
    const int kc = k0 + c * KC;
    if (c >= nchunks || kc >= k1) return;  // uniform over the wave
    const int kl = kc + q * E;             // first key of this lane's chunk
    float sv[RT][E];
#pragma unroll
    for (int r = 0; r < RT; ++r)
#pragma unroll
      for (int cg = 0; cg < NCG; ++cg) {
        f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int d = 0; d < NDS; ++d) acc = mma<T>(kf[slot][cg][d], qf[r][d], acc);
#pragma unroll
        for (int i = 0; i < 4; ++i) sv[r][4 * cg + i] = acc[i];
      }
    if constexpr (NS == 1) load_k(0, c + 1);
    // value columns of keys past the end of the cache are zeroed (not
    // initialised there; a zero probability must not meet a NaN)
    if (kc + KC > kend) {
      const int n = min(max(kend - kl, 0), E);
#pragma unroll
      for (int t = 0; t < NDT; ++t) vf[slot][t] = keep_first<T>(vf[slot][t], n);
    }
    const bool all_visible = kc + KC <= min(P, k1);  // cached prefix only (uniform)
#pragma unroll
    for (int r = 0; r < RT; ++r) {
      if (!all_visible) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const int key = kl + e;
          bool vis = key < lim[r];
          if (a.tree) vis &= (key < P) | (((anc[r] >> ((key - P) & 63)) & 1ull) != 0);
          sv[r][e] = vis ? sv[r][e] : -INFINITY;
        }
      }
      float cmax = sv[r][0];
#pragma unroll
      for (int e = 1; e < E; ++e) cmax = fmaxf(cmax, sv[r][e]);
      cmax = row_max4(cmax);
      // move the reference of the rows that outgrew it. The branch is taken
      // by the whole wave, but every row decides for itself (the others keep
      // their reference and scale by exactly 1), so a row's arithmetic never
      // depends on the other rows of its tile.
      const bool grow = m_run[r] == -INFINITY ? cmax > -INFINITY : (cmax - m_run[r]) * sc > kSlack;
      if (__any(grow)) {
        const float m_new = grow ? fmaxf(m_run[r], cmax) : m_run[r];
        const float alpha =
            grow ? __builtin_amdgcn_exp2f((m_run[r] - m_new) * sc) : 1.f;  // exp2(-inf) = 0
        l_run[r] *= alpha;
#pragma unroll
        for (int t = 0; t < NDT; ++t) o[r][t] *= alpha;
        m_run[r] = m_new;
      }
      const float msc = m_run[r] == -INFINITY ? 0.f : m_run[r] * sc;
      float p[E], psum = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        p[e] = __builtin_amdgcn_exp2f(fmaf(sv[r][e], sc, -msc));  // exp2(-inf) = 0
        psum += p[e];
      }
      l_run[r] += psum;
      const uint4 pu = pack_probs<T>(p);
#pragma unroll
      for (int t = 0; t < NDT; ++t) o[r][t] = mma<T>(vf[slot][t], pu, o[r][t]);
      if constexpr (sizeof(T) == 2) {
        const uint4 pl = pack_probs_lo(p, pu);
#pragma unroll
        for (int t = 0; t < NDT; ++t) o[r][t] = mma<T>(vf[slot][t], pl, o[r][t]);
      }
    }
    if constexpr (NS == 1) load_v(0, c + 1);
  };
  // write the partial of key range sp and restart the accumulators: lane
  // holds O^T[d = t*16 + 4q + i][row lane%16]
  auto flush = [&](int sp) {
    float *po = a.part_o + (((int64_t)h * a.n_splits + sp) * a.rowpad) * HD;
    float *pml = a.part_ml + (((int64_t)h * a.n_splits + sp) * a.rowpad) * 2;
#pragma unroll
    for (int r = 0; r < RT; ++r) {
      const float l = row_sum4(l_run[r]);
      const int jq = row0 + r * 16 + (lane & 15);
      if (jq < M) {
#pragma unroll
        for (int t = 0; t < NDT; ++t)
          *(float4 *)(po + (int64_t)jq * HD + t * 16 + 4 * q) =
              make_float4(o[r][t][0], o[r][t][1], o[r][t][2], o[r][t][3]);
        if (q == 0) {  // (max, sum) in the log2-scaled units the combine uses
          pml[jq * 2 + 0] = m_run[r] == -INFINITY ? -INFINITY : m_run[r] * sc;
          pml[jq * 2 + 1] = l;
        }
      }
      m_run[r] = -INFINITY;
      l_run[r] = 0.f;
#pragma unroll
      for (int t = 0; t < NDT; ++t) o[r][t] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  };
  int sp = s0, next_flush = cps - 1;  // key range being reduced, its last chunk
  auto step = [&](int slot, int c) {
    compute(slot, c);
    if (c == next_flush && c < nchunks) {  // uniform over the wave
      flush(sp++);
      next_flush += cps;
    }
  };

  // The first kStraight chunks run as straight-line code (no loop-carried
  // accumulators to shuffle between register files); longer ranges continue
  // in a loop. Compute of a chunk past the range returns at once.
  constexpr int kStraight = NS * ((6 + NS - 1) / NS);
  if constexpr (NS == 1) {
#pragma unroll
    for (int c = 0; c < kStraight; ++c) {
      step(0, c);
      __builtin_amdgcn_sched_barrier(0);
    }
    for (int c = kStraight; c < nchunks; ++c) {
      step(0, c);
      __builtin_amdgcn_sched_barrier(0);
    }
  } else {
#pragma unroll
    for (int c = 0; c < kStraight; c += NS) {
#pragma unroll
      for (int u = 0; u < NS; ++u) {
        step(u, c + u);
        load(u, c + u + NS);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    for (int c = kStraight; c < nchunks; c += NS) {
#pragma unroll
      for (int u = 0; u < NS; ++u) {
        step(u, c + u);
        load(u, c + u + NS);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  // the last range ends before a whole number of chunks (key bound)
  if (nchunks % cps != 0) flush(sp);
}

// Merge the key-range partials of one (row, head) and round the result. Four
// waves: wave w takes splits w, w + 4, ... (up to 16 each) and loads their
// outputs before anything waits (they do not depend on the cache length,
// which only decides how many splits count); wave 0's lane s reads split s's
// (max, sum). Each wave adds its splits in index order, then the four waves'
// sums are added in wave order, so the result does not depend on timing.
template <typename T, int HD>
__global__ __launch_bounds__(256) void k_attn_combine(AttnArgs a) {
  // A split's partial row (HD floats) is read by HD/4 lanes with 16-byte
  // loads, so one wave load covers SPW splits; wave w takes splits w, w + 4,
  // ... (up to 64 in all). Sums per dimension: over a lane's splits in
  // order, then over the lanes holding the same dimensions (xor pattern, in
  // fixed order), then over the waves 0..3.
  constexpr int LPS = HD / 4;     // lanes per split row
  constexpr int SPW = 64 / LPS;   // splits per wave load
  constexpr int NUI = 16 / SPW;   // wave loads per lane (16 splits per wave)
  const int j = blockIdx.x, h = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int sub = lane / LPS, c4 = lane % LPS;
  const float *pml = a.part_ml + ((int64_t)h * a.n_splits * a.rowpad) * 2;
  const float *po = a.part_o + ((int64_t)h * a.n_splits * a.rowpad) * HD;
  const int ns = a.n_splits;
  float4 v[NUI];
#pragma unroll
  for (int u = 0; u < NUI; ++u) {
    const int sp = wid + 4 * (u * SPW + sub);
    v[u] = sp < ns ? *(const float4 *)(po + ((int64_t)sp * a.rowpad + j) * HD + 4 * c4)
                   : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  float mv = -INFINITY, lv = 0.f;
  if (wid == 0 && lane < ns) {
    mv = pml[((int64_t)lane * a.rowpad + j) * 2];
    lv = pml[((int64_t)lane * a.rowpad + j) * 2 + 1];
  }
  const int P = *a.kv_len;
  const int used = min(ns, (P + a.M + a.chunk_keys - 1) / a.chunk_keys);
  __shared__ float ws[64];
  __shared__ float s_den;
  __shared__ float4 red[4][LPS];
  if (wid == 0) {
    // splits past the used ones hold stale data: weight zero, outputs skipped
    const float m = lane < used ? mv : -INFINITY, l = lane < used ? lv : 0.f;
    const float mx = wave_max(m);
    const float w = m == -INFINITY ? 0.f : exp2f(m - mx);
    const float den = wave_sum(w * l);
    ws[lane] = w;
    if (lane == 0) s_den = den;
  }
  __syncthreads();
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int u = 0; u < NUI; ++u) {
    const int sp = wid + 4 * (u * SPW + sub);
    if (sp < used) {
      const float w = ws[sp];
      acc.x += w * v[u].x;
      acc.y += w * v[u].y;
      acc.z += w * v[u].z;
      acc.w += w * v[u].w;
    }
  }
  // lanes c4 + LPS * sub hold the same dimensions: add them in sub order
#pragma unroll
  for (int o = LPS; o < 64; o <<= 1) {
    float4 b;
    b.x = __shfl_xor(acc.x, o, 64);
    b.y = __shfl_xor(acc.y, o, 64);
    b.z = __shfl_xor(acc.z, o, 64);
    b.w = __shfl_xor(acc.w, o, 64);
    const bool low = (lane & o) == 0;  // the lower sub keeps its sum first
    acc = low ? make_float4(acc.x + b.x, acc.y + b.y, acc.z + b.z, acc.w + b.w)
              : make_float4(b.x + acc.x, b.y + acc.y, b.z + acc.z, b.w + acc.w);
  }
  if (sub == 0) red[wid][c4] = acc;
  __syncthreads();
  if (wid != 0 || sub != 0) return;
  const float den = s_den;
  const float4 r0 = red[0][c4], r1 = red[1][c4], r2 = red[2][c4], r3 = red[3][c4];
  const float tot[4] = {((r0.x + r1.x) + r2.x) + r3.x, ((r0.y + r1.y) + r2.y) + r3.y,
                        ((r0.z + r1.z) + r2.z) + r3.z, ((r0.w + r1.w) + r2.w) + r3.w};
  T *out = (T *)a.out;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int d = 4 * c4 + i;
    const int64_t k = h * HD + d;
    Elem<T>::store(out, a.out_packed ? act_off<T>(j, k, a.ldout) : (int64_t)j * a.ldout + k,
                   tot[i] / den);
  }
}

// ---------------------------------------------------------------------------
// Prefill attention (bf16, head_dim 128, 4..8 query heads per KV head): a
// chunk's rows all attend to the long reused prefix, so the work is a dense
// contraction and K/V tiles are worth staging. One block of four waves per
// (KV head, key range, 32-row query tile, four of the KV head's query
// heads); its waves are those query heads, all on the same 32 rows, so one
// LDS copy of each 64-key K and V^T tile serves them. Two such blocks fit a
// CU, one computing while the other waits for its tiles. Per wave and tile: S^T = K Q^T as two 32-key halves of eight
// 32x32x16 products (K rows permuted so that each lane ends up with eight
// consecutive keys of its query row per 16-key step, the B-operand layout of
// the value product), the online softmax in fp32 with the reference-maximum
// rescale of the verify kernel, then O^T += V^T P^T. K and V tiles are staged
// row-major as they sit in the cache; the V^T operand comes from transposing
// LDS reads. Loads of the next tile are in flight while the current one is
// multiplied. Each block writes one
// partial per (row, head) for k_attn_combine.
// ---------------------------------------------------------------------------

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ inline f32x16 mma32(const uint4 &a, const uint4 &b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Key (within a 32-key half tile) carried by row i of the score product's A
// operand. The product leaves value v of lane l at output row
// 8*(v/4) + 4*(l/32) + v%4; with this assignment that row holds key
// 16*(v/8) + 8*(l/32) + v%8.
__device__ inline int score_key(int i) {
  const int g = i >> 3, half = (i >> 2) & 1, r = i & 3;
  return 16 * (g >> 1) + 8 * half + 4 * (g & 1) + r;
}

constexpr int kPreKeys = 64;  // keys per staged tile

// Two transposing 64-bit LDS reads (gfx950 ds_read_b64_tr_b16), the first
// giving elements 0-3 of the 16-byte operand, the second elements 4-7.
typedef short v4s16 __attribute__((ext_vector_type(4)));
__device__ inline uint4 lds_read_tr16x2(const char *p0, const char *p1) {
  const v4s16 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4s16 *)(const_cast<char *>(p0)));
  const v4s16 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4s16 *)(const_cast<char *>(p1)));
  const uint2 x = __builtin_bit_cast(uint2, a), y = __builtin_bit_cast(uint2, b);
  return make_uint4(x.x, x.y, y.x, y.y);
}

}  // namespace

__global__ __launch_bounds__(256, 2) void k_attn_prefill(AttnArgs a) {
  constexpr int HD = 128;
  constexpr int nthr = 256;  // four waves: up to four of the KV head's query heads
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int r32 = lane & 31, hh = lane >> 5;
  // blocks of one (KV head, key range) pair get ids of equal residue mod 8:
  // they run on one XCD and share its L2 copy of the range's K/V. A KV head
  // with more than four query heads takes two blocks per row tile, so two
  // independent blocks share every CU.
  const int rtiles = (a.M + 31) / 32;
  const int nsub = (a.group + 3) / 4;
  const int npairs = a.n_kv * a.n_splits;
  const int b = blockIdx.x, rest = b >> 3;
  const int t = rest % rtiles, sub = (rest / rtiles) % nsub;
  const int p = (rest / rtiles / nsub) * 8 + (b & 7);
  if (p >= npairs) return;
  const int g = p / a.n_splits, sp = p % a.n_splits;
  const int hl = sub * 4 + wid;        // query head within the group
  const bool head = hl < a.group;      // a wave past the group only helps load
  const int h = g * a.group + min(hl, a.group - 1);
  const int j0 = t * 32;

  // query fragments: lane holds Q[row j0 + r32][16*ds + 8*hh .. +8]
  uint4 qf[HD / 16];
  {
    const int jr = min(j0 + r32, a.rowpad - 1);
    const bf16_t *qrow = (const bf16_t *)a.q + (int64_t)jr * a.ldq + h * HD + 8 * hh;
#pragma unroll
    for (int ds = 0; ds < HD / 16; ++ds) qf[ds] = *(const uint4 *)(qrow + 16 * ds);
  }
  const bf16_t *kplane = (const bf16_t *)a.cache + ((int64_t)(a.layer * 2 + 0) * a.n_kv + g) * a.plane;
  const bf16_t *vplane = (const bf16_t *)a.cache + ((int64_t)(a.layer * 2 + 1) * a.n_kv + g) * a.plane;
  const rsrc_t kr = make_rsrc(kplane, (uint32_t)(a.plane * 2));
  const rsrc_t vr = make_rsrc(vplane, (uint32_t)(a.plane * 2));
  const float sc = a.scale_log2;

  // keys of this block: its range, cut at the last row's causal bound
  const int P = *a.kv_len;
  const int kend = P + a.M;
  const int k_lo = sp * a.chunk_keys;
  const int k_hi = min(min(k_lo + a.chunk_keys, P + min(j0 + 32, a.M)), kend);
  const int ntiles = k_hi > k_lo ? (k_hi - k_lo + kPreKeys - 1) / kPreKeys : 0;

  // staged tiles, keys and values alike: [key][16-byte chunk ^ (key & 15)]
  // (row-major as in the cache, the swizzle keeps the lanes of an operand
  // read on distinct banks). Keys or values at or past the cache end load as
  // zeros (out of range), so a zero probability never meets an
  // uninitialised NaN.
  static_assert(kPreKeys * HD / 8 == 4 * nthr, "four 16-byte chunks of K and of V per thread");
  __shared__ uint4 lk[2][kPreKeys][HD / 8];
  __shared__ uint4 lv[2][kPreKeys][HD / 8];
  uint4 gk[4], gv[4];
  auto gload = [&](int kt) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int idx = tid + r * nthr;
      const int key = kt + (idx >> 4), c = idx & 15;
      const uint32_t off = key < kend ? (uint32_t)(((int64_t)key * HD + c * 8) * 2) : kOOB;
      gk[r] = bload16(kr, off);
      gv[r] = bload16(vr, off);
    }
  };
  auto lstore = [&](int buf, int kt) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int idx = tid + r * nthr;
      const int key = idx >> 4, c = idx & 15;
      lk[buf][key][c ^ (key & 15)] = gk[r];
      lv[buf][key][c ^ (key & 15)] = gv[r];
    }
  };
  // The value product needs V^T: lane l of the A operand holds dimension
  // d = 32 dt + l % 32 of eight consecutive keys. Two transposing LDS reads
  // give them (gfx950: within a group of 16 lanes, the lanes' four 16-bit
  // elements are concatenated, A[4 s + e], and lane i receives A[i + 16 j],
  // j = 0..3). Source lane s of group G points at key kb + s / 4, dimensions
  // d0 + 4 (s % 4) .. + 3 with d0 = 32 dt + 16 (G % 2), kb = the step's first
  // key + 8 (G / 2) (+ 4 for the second read), so lane i receives dimension
  // d0 + i of keys kb .. kb + 3. voff: byte offsets within a 16-key step.
  uint32_t voff[HD / 32][2];
  {
    const int s16 = lane & 15, G = lane >> 4;
#pragma unroll
    for (int dt = 0; dt < HD / 32; ++dt)
#pragma unroll
      for (int rr = 0; rr < 2; ++rr) {
        const int kl = 8 * (G >> 1) + 4 * rr + (s16 >> 2);  // key within the step (0..15)
        const int chunk = (4 * dt + 2 * (G & 1) + ((s16 & 3) >> 1)) ^ kl;
        voff[dt][rr] = (uint32_t)(kl * HD * 2 + chunk * 16 + (s16 & 1) * 8);
      }
  }

  float m_run = -INFINITY, l_run = 0.f;
  f32x16 o[HD / 32];
#pragma unroll
  for (int dt = 0; dt < HD / 32; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[dt][v] = 0.f;
  const int row = j0 + r32;
  const int lim = min(P + row + 1, kend);  // keys visible to this lane's row
  constexpr float kSlack = 8.f;

  if (ntiles > 0) {
    gload(k_lo);
    lstore(0, k_lo);
  }
  __syncthreads();
  for (int it = 0; it < ntiles; ++it) {
    const int buf = it & 1, kt = k_lo + it * kPreKeys;
    if (it + 1 < ntiles) gload(kt + kPreKeys);
    if (head) {
    f32x16 s[2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
      for (int v = 0; v < 16; ++v) s[st][v] = 0.f;
      const int kl = st * 32 + score_key(r32);
#pragma unroll
      for (int ds = 0; ds < HD / 16; ++ds)
        s[st] = mma32(lk[buf][kl][(2 * ds + hh) ^ (kl & 15)], qf[ds], s[st]);
    }
    // lane value v of half st is key kt + 32*st + 16*(v/8) + 8*hh + v%8
    if (kt + kPreKeys > P + j0 + 1) {  // some key past the first row's bound (uniform)
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = kt + 32 * st + 16 * (v >> 3) + 8 * hh + (v & 7);
          s[st][v] = key < lim ? s[st][v] : -INFINITY;
        }
    }
    float cmax = s[0][0];
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int v = 0; v < 16; ++v) cmax = fmaxf(cmax, s[st][v]);
    {  // the row's other 32 keys sit in lane l ^ 32
      auto x = __builtin_amdgcn_permlane32_swap(__float_as_uint(cmax), __float_as_uint(cmax), false,
                                                false);
      cmax = fmaxf(__uint_as_float(x[0]), __uint_as_float(x[1]));
    }
    const bool grow = m_run == -INFINITY ? cmax > -INFINITY : (cmax - m_run) * sc > kSlack;
    if (__any(grow)) {
      const float m_new = grow ? fmaxf(m_run, cmax) : m_run;
      const float alpha = grow ? __builtin_amdgcn_exp2f((m_run - m_new) * sc) : 1.f;
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < HD / 32; ++dt) o[dt] *= alpha;
      m_run = m_new;
    }
    const float msc = m_run == -INFINITY ? 0.f : m_run * sc;
    uint4 pb[2][2], pl[2][2];  // P^T operand of each 16-key step, as hi + lo
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        float pv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          pv[e] = __builtin_amdgcn_exp2f(fmaf(s[st][8 * s2 + e], sc, -msc));
          l_run += pv[e];
        }
        pb[st][s2] = pack_probs<bf16_t>(pv);
        pl[st][s2] = pack_probs_lo(pv, pb[st][s2]);
      }
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
        for (int dt = 0; dt < HD / 32; ++dt) {
          const char *step = (const char *)&lv[buf][32 * st + 16 * s2][0];
          const uint4 vv = lds_read_tr16x2(step + voff[dt][0], step + voff[dt][1]);
          o[dt] = mma32(vv, pb[st][s2], o[dt]);
          o[dt] = mma32(vv, pl[st][s2], o[dt]);
        }
    }
    if (it + 1 < ntiles) lstore(buf ^ 1, kt + kPreKeys);
    __syncthreads();
  }

  // partial of this key range: lane holds O^T[d = 32*dt + 8*(v/4) + 4*hh + v%4][row]
  {
    auto x = __builtin_amdgcn_permlane32_swap(__float_as_uint(l_run), __float_as_uint(l_run), false,
                                              false);
    l_run = __uint_as_float(x[0]) + __uint_as_float(x[1]);
  }
  if (head && row < a.M) {
    const int64_t slot = ((int64_t)h * a.n_splits + sp) * a.rowpad + row;
    float *po = a.part_o + slot * HD;
#pragma unroll
    for (int dt = 0; dt < HD / 32; ++dt)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4)
        *(float4 *)(po + 32 * dt + 8 * q4 + 4 * hh) =
            make_float4(o[dt][4 * q4], o[dt][4 * q4 + 1], o[dt][4 * q4 + 2], o[dt][4 * q4 + 3]);
    if (hh == 0) {
      a.part_ml[slot * 2 + 0] = m_run == -INFINITY ? -INFINITY : m_run * sc;
      a.part_ml[slot * 2 + 1] = l_run;
    }
  }
}

// Merge the key-range partials of the prefill attention: few ranges (at most
// kPrefillMaxSplits) and many (row, head) pairs, so a half-wave takes one
// pair. Lane c holds dimensions 4c .. 4c + 3; every lane reads the ranges'
// (max, sum) itself (the same addresses across the half-wave) and adds the
// weighted outputs in range order, so the result does not depend on timing.
constexpr int kPrefillMaxSplits = 8;
template <int HD>
__global__ __launch_bounds__(256) void k_attn_combine_rows(AttnArgs a) {
  constexpr int LPP = HD / 4;     // lanes per (row, head) pair
  constexpr int PPB = 256 / LPP;  // pairs per block
  const int nh = a.n_kv * a.group;
  const int pair = blockIdx.x * PPB + (int)threadIdx.x / LPP, c4 = threadIdx.x % LPP;
  if (pair >= a.M * nh) return;
  const int j = pair / nh, h = pair % nh;
  const int ns = a.n_splits;
  const int P = *a.kv_len;
  // ranges past the used ones hold stale data: skipped
  const int used = min(ns, (P + a.M + a.chunk_keys - 1) / a.chunk_keys);
  const float *pml = a.part_ml + ((int64_t)h * ns * a.rowpad + j) * 2;
  const float *po = a.part_o + ((int64_t)h * ns * a.rowpad + j) * HD + 4 * c4;
  float4 v[kPrefillMaxSplits];
  float m[kPrefillMaxSplits], l[kPrefillMaxSplits];
#pragma unroll
  for (int sp = 0; sp < kPrefillMaxSplits; ++sp) {
    if (sp < used) {
      v[sp] = *(const float4 *)(po + (int64_t)sp * a.rowpad * HD);
      m[sp] = pml[(int64_t)sp * a.rowpad * 2];
      l[sp] = pml[(int64_t)sp * a.rowpad * 2 + 1];
    }
  }
  float mx = -INFINITY;
#pragma unroll
  for (int sp = 0; sp < kPrefillMaxSplits; ++sp)
    if (sp < used) mx = fmaxf(mx, m[sp]);
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  float den = 0.f;
#pragma unroll
  for (int sp = 0; sp < kPrefillMaxSplits; ++sp) {
    if (sp < used) {
      const float w = m[sp] == -INFINITY ? 0.f : exp2f(m[sp] - mx);
      den += w * l[sp];
      acc.x += w * v[sp].x;
      acc.y += w * v[sp].y;
      acc.z += w * v[sp].z;
      acc.w += w * v[sp].w;
    }
  }
  const float r[4] = {acc.x / den, acc.y / den, acc.z / den, acc.w / den};
  bf16_t *out = (bf16_t *)a.out;
  const int64_t k = (int64_t)h * HD + 4 * c4;
  if (a.out_packed) {
#pragma unroll
    for (int i = 0; i < 4; ++i) Elem<bf16_t>::store(out, act_off<bf16_t>(j, k + i, a.ldout), r[i]);
  } else {
    uint2 pk;
    pk.x = (uint32_t)f32_to_bf16(r[0]) | ((uint32_t)f32_to_bf16(r[1]) << 16);
    pk.y = (uint32_t)f32_to_bf16(r[2]) | ((uint32_t)f32_to_bf16(r[3]) << 16);
    *(uint2 *)(out + (int64_t)j * a.ldout + k) = pk;
  }
}

bool attn_prefill_supported(bool bf16, int head_dim, int group) {
  return bf16 && head_dim == 128 && group >= 4 && group <= 8;
}

hipError_t launch_attn_prefill(const AttnArgs &a, hipStream_t s) {
  if (!attn_prefill_supported(true, a.head_dim, a.group) || a.chunk_keys % kPreKeys != 0 ||
      a.M < 1 || a.plane * 2 >= (int64_t)1 << 31 || a.n_splits < 1 ||
      a.n_splits > kPrefillMaxSplits || (!a.out_packed && a.ldout % 4 != 0))
    return hipErrorInvalidValue;
  const int rtiles = (a.M + 31) / 32;
  const int npairs = a.n_kv * a.n_splits;
  const int nsub = (a.group + 3) / 4;
  dim3 grid(8 * ((npairs + 7) / 8) * rtiles * nsub);
  PF_TRY(launch_k(k_attn_prefill, grid, dim3(256), s, a));
  const int pairs = a.M * a.n_kv * a.group;
  PF_TRY(launch_k(k_attn_combine_rows<128>, dim3((pairs + 7) / 8), 256, s, a));
  return hipGetLastError();
}

template <typename T, int HD>
static hipError_t attn_t(int rt, const AttnArgs &a, hipStream_t s) {
  const int per = attn_tiles_per_wave(rt);
  const int groups = (rt + per - 1) / per;
  if (a.chunk_keys % (4 * Elem<T>::E) != 0 || a.keys_bound < 0 || a.per_wave < 1)
    return hipErrorInvalidValue;
  const int works = a.n_kv * ((a.n_splits + a.per_wave - 1) / a.per_wave);
  dim3 grid(8 * a.group * ((works + 7) / 8), groups), block(64);
  switch (per) {
    case 1: PF_TRY(launch_k(k_attn<T, 1, HD, 2, 1>, grid, block, s, a)); break;
    case 2: PF_TRY(launch_k(k_attn<T, 2, HD, 2, 1>, grid, block, s, a)); break;
    case 3: PF_TRY(launch_k(k_attn<T, 3, HD, 1, 1>, grid, block, s, a)); break;
    default: return hipErrorInvalidValue;
  }
  PF_TRY(launch_k(k_attn_combine<T, HD>, dim3(a.M, a.n_kv * a.group), 256, s, a));
  return hipGetLastError();
}

hipError_t launch_attn_combine(bool bf16, const AttnArgs &a, hipStream_t s) {
  if (a.head_dim != 128 || a.n_splits > 64) return hipErrorInvalidValue;
  if (bf16)
    PF_TRY(launch_k(k_attn_combine<bf16_t, 128>, dim3(a.M, a.n_kv * a.group), 256, s, a));
  else
    PF_TRY(launch_k(k_attn_combine<float, 128>, dim3(a.M, a.n_kv * a.group), 256, s, a));
  return hipGetLastError();
}

hipError_t launch_attn(bool bf16, int rt, const AttnArgs &a, hipStream_t s) {
  if (a.head_dim == 128) return bf16 ? attn_t<bf16_t, 128>(rt, a, s) : attn_t<float, 128>(rt, a, s);
  if (a.head_dim == 64) return bf16 ? attn_t<bf16_t, 64>(rt, a, s) : attn_t<float, 64>(rt, a, s);
  return hipErrorInvalidValue;
}

}  // namespace pf
