// Grouped-query verify attention. Each query row (draft node j, head h)
// attends to the cached keys 0..P-1 and to the draft keys P..P+M-1 it may
// see (causal for a linear draft, ancestors-or-self for a tree).
//
// Work split: one wave per (key range, query head); the heads of a group read
// the same K/V fragments, which they share through L2. Keys
// are processed in chunks of 4*E (32 bf16 / 16 fp32). S^T = K Q^T is formed
// with K as the MFMA A operand, permuting which key each A row carries so
// that, after the MFMA, lane quarter q holds the scores of keys q*E..q*E+E-1
// of its query row (column). That is exactly the B-operand layout of
// O^T += V^T P^T, and values are stored transposed ([dim][slot]) in the
// cache, so the V^T fragment of a lane is one contiguous 16-byte load. The
// online softmax runs in the log2 domain in fp32; probabilities enter the PV
// product in the model dtype. Each block writes an unnormalised partial
// (o, running max, running sum) per row; k_attn_combine merges the splits.
#include "kernels.h"

namespace pf {

template <typename T, int RT, int HD>
__global__ __launch_bounds__(64) void k_attn(AttnArgs a) {
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
  const int b = blockIdx.x;
  const int xcd = b & 7, j = b >> 3;
  const int hl = j % a.group;
  const int w = (j / a.group) * 8 + xcd;  // (KV head, key range) work id
  if (w >= a.n_kv * a.n_splits) return;
  const int g = w / a.n_splits;
  const int s = w % a.n_splits;
  const int h = g * a.group + hl;
  const int row0 = blockIdx.y * RT * 16;  // first query row of this wave

  const int P = *a.kv_len;
  const int M = a.M;
  const int kend = P + M;
  const int k0 = s * a.chunk_keys;
  const int k1 = min(k0 + a.chunk_keys, kend);

  float *po = a.part_o + (((int64_t)h * a.n_splits + s) * a.rowpad) * HD;
  float *pml = a.part_ml + (((int64_t)h * a.n_splits + s) * a.rowpad) * 2;

  float m_run[RT], l_run[RT];
  f32x4 o[RT][NDT];
#pragma unroll
  for (int r = 0; r < RT; ++r) {
    m_run[r] = -INFINITY;
    l_run[r] = 0.f;
#pragma unroll
    for (int t = 0; t < NDT; ++t) o[r][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  if (k0 < k1) {
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
    const int nchunks = (k1 - k0 + KC - 1) / KC;

    // two chunk slots: compute one while the other's K/V loads are in flight.
    // Chunks past the range load out of the resource (zeros, no traffic) and
    // their keys are masked, so they add nothing.
    uint4 kf[2][NCG][NDS], vf[2][NDT];
    auto load = [&](int slot, int c) {
      const int kc = k0 + c * KC;
      const bool in = c < nchunks;
#pragma unroll
      for (int cg = 0; cg < NCG; ++cg) {
        const int r = lane & 15;
        const int key = kc + E * (r >> 2) + 4 * cg + (r & 3);
#pragma unroll
        for (int d = 0; d < NDS; ++d)
          kf[slot][cg][d] = bload16(
              kr, in ? (uint32_t)(((int64_t)key * HD + d * KF + q * E) * sizeof(T)) : kOOB);
      }
#pragma unroll
      for (int t = 0; t < NDT; ++t)
        vf[slot][t] = bload16(
            vr, in ? (uint32_t)(((int64_t)(t * 16 + (lane & 15)) * a.cap + kc + q * E) * sizeof(T))
                   : kOOB);
    };
    auto compute = [&](int slot, int c) {
      const int kc = k0 + c * KC;
      if (kc + KC > kend) {  // zero value columns of keys past the end of the cache
#pragma unroll
        for (int t = 0; t < NDT; ++t) {
          union {
            uint4 v;
            T e[E];
          } u;
          u.v = vf[slot][t];
#pragma unroll
          for (int e = 0; e < E; ++e)
            if (kc + q * E + e >= kend) memset(&u.e[e], 0, sizeof(T));
          vf[slot][t] = u.v;
        }
      }
#pragma unroll
      for (int r = 0; r < RT; ++r) {
        const int j = row0 + r * 16 + (lane & 15);  // query row of this lane
        float sv[E];
#pragma unroll
        for (int cg = 0; cg < NCG; ++cg) {
          f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int d = 0; d < NDS; ++d) acc = mma<T>(kf[slot][cg][d], qf[r][d], acc);
#pragma unroll
          for (int i = 0; i < 4; ++i) sv[4 * cg + i] = acc[i];
        }
        // keys of this lane: kc + q*E + e, e = 4*cg + i
        float cmax = -INFINITY;
        if (kc + KC <= min(P, k1)) {  // cached prefix only: every key visible
#pragma unroll
          for (int e = 0; e < E; ++e) {
            sv[e] *= sc;
            cmax = fmaxf(cmax, sv[e]);
          }
        } else {
#pragma unroll
          for (int e = 0; e < E; ++e) {
            const int key = kc + q * E + e;
            bool vis = key < k1;
            if (vis && key >= P) {
              const int di = key - P;
              vis = a.tree ? (j < 64 && ((a.anc[j] >> di) & 1ull)) : (di <= j);
            }
            sv[e] = vis ? sv[e] * sc : -INFINITY;
            cmax = fmaxf(cmax, sv[e]);
          }
        }
        cmax = fmaxf(cmax, __shfl_xor(cmax, 16, 64));
        cmax = fmaxf(cmax, __shfl_xor(cmax, 32, 64));
        const float m_new = fmaxf(m_run[r], cmax);
        const float alpha = m_new == -INFINITY ? 1.f : exp2f(m_run[r] - m_new);
        union {
          uint4 v;
          T e[E];
        } pu;
        float psum = 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const float p = sv[e] == -INFINITY ? 0.f : exp2f(sv[e] - m_new);
          Elem<T>::store(pu.e, e, p);
          psum += p;
        }
        l_run[r] = l_run[r] * alpha + psum;
        m_run[r] = m_new;
#pragma unroll
        for (int t = 0; t < NDT; ++t) {
          o[r][t] *= alpha;
          o[r][t] = mma<T>(vf[slot][t], pu.v, o[r][t]);
        }
      }
    };
    load(0, 0);
    __builtin_amdgcn_sched_barrier(0);
    load(1, 1);
    __builtin_amdgcn_sched_barrier(0);
    for (int c = 0; c < nchunks; c += 2) {
      compute(0, c);
      load(0, c + 2);
      __builtin_amdgcn_sched_barrier(0);
      compute(1, c + 1);
      load(1, c + 3);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // write the partial: lane holds O^T[d = t*16 + 4q + i][row lane%16]
#pragma unroll
  for (int r = 0; r < RT; ++r) {
    float l = l_run[r];
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    const int j = row0 + r * 16 + (lane & 15);
    if (j >= M) continue;
#pragma unroll
    for (int t = 0; t < NDT; ++t)
      *(float4 *)(po + (int64_t)j * HD + t * 16 + 4 * q) =
          make_float4(o[r][t][0], o[r][t][1], o[r][t][2], o[r][t][3]);
    if (q == 0) {
      pml[j * 2 + 0] = m_run[r];
      pml[j * 2 + 1] = l;
    }
  }
}

// Merge the key-range partials of one (row, head) and round the result:
// lane s reads split s's (max, sum); the output sum over splits keeps eight
// loads in flight per lane.
template <typename T, int HD>
__global__ __launch_bounds__(64) void k_attn_combine(AttnArgs a) {
  const int j = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
  const float *pml = a.part_ml + ((int64_t)h * a.n_splits * a.rowpad) * 2;
  const float *po = a.part_o + ((int64_t)h * a.n_splits * a.rowpad) * HD;
  const int P = *a.kv_len;
  const int used = min(a.n_splits, (P + a.M + a.chunk_keys - 1) / a.chunk_keys);
  float m = -INFINITY, l = 0.f;
  if (lane < used) {
    m = pml[((int64_t)lane * a.rowpad + j) * 2];
    l = pml[((int64_t)lane * a.rowpad + j) * 2 + 1];
  }
  const float mx = wave_max(m);
  const float w = m == -INFINITY ? 0.f : exp2f(m - mx);
  const float den = wave_sum(w * l);
  __shared__ float ws[64];
  ws[lane] = w;
  __syncthreads();
  float acc[HD / 64];
#pragma unroll
  for (int i = 0; i < HD / 64; ++i) acc[i] = 0.f;
  int s = 0;
  for (; s + 8 <= used; s += 8) {
    float v[8][HD / 64];
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int i = 0; i < HD / 64; ++i)
        v[u][i] = po[((int64_t)(s + u) * a.rowpad + j) * HD + lane + 64 * i];
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int i = 0; i < HD / 64; ++i) acc[i] += ws[s + u] * v[u][i];
  }
  for (; s < used; ++s)
#pragma unroll
    for (int i = 0; i < HD / 64; ++i)
      acc[i] += ws[s] * po[((int64_t)s * a.rowpad + j) * HD + lane + 64 * i];
  T *out = (T *)a.out + (int64_t)j * a.ldout + h * HD;
#pragma unroll
  for (int i = 0; i < HD / 64; ++i) Elem<T>::store(out, lane + 64 * i, acc[i] / den);
}

template <typename T, int HD>
static hipError_t attn_t(int rt, const AttnArgs &a, hipStream_t s) {
  // at most three 16-row query tiles per wave (register budget); more rows
  // are spread over blockIdx.z
  const int per = rt <= 3 ? rt : 2;
  const int groups = (rt + per - 1) / per;
  const int works = a.n_kv * a.n_splits;
  dim3 grid(8 * a.group * ((works + 7) / 8), groups), block(64);
  switch (per) {
    case 1: k_attn<T, 1, HD><<<grid, block, 0, s>>>(a); break;
    case 2: k_attn<T, 2, HD><<<grid, block, 0, s>>>(a); break;
    case 3: k_attn<T, 3, HD><<<grid, block, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  k_attn_combine<T, HD><<<dim3(a.M, a.n_kv * a.group), 64, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_attn(bool bf16, int rt, const AttnArgs &a, hipStream_t s) {
  if (a.head_dim == 128) return bf16 ? attn_t<bf16_t, 128>(rt, a, s) : attn_t<float, 128>(rt, a, s);
  if (a.head_dim == 64) return bf16 ? attn_t<bf16_t, 64>(rt, a, s) : attn_t<float, 64>(rt, a, s);
  return hipErrorInvalidValue;
}

}  // namespace pf
