// Fused skinny GEMM for the verify step, one launch per projection:
//
//   prologue  stage this block's slice of X (rows 0..MT*16-1, its k range) in
//             LDS -- either a bf16 activation copy, or the fp32 residual
//             stream normalised on the fly: bf16(x * rsqrt(mean(x^2)+eps) * g),
//             with mean(x^2) summed from per-column-group partial sums the
//             producer of x left behind (so no separate RMSNorm launch)
//   main      4 waves, each streaming its own 2 weight tiles (16 rows x 32 k
//             per 1 KiB fragment, contiguous) through a ring of fragment
//             slots into the MFMA A operand; X fragments come from LDS
//   epilogue  split-K partials to global memory; the last block of a column
//             group to arrive (device-scope counter, no waiting) reduces the
//             splits in a fixed order and applies the group epilogue:
//             QKV  -> RoPE, round, queries out, K/V appended to the cache
//             RESID-> residual add into x, per-group sum of squares
//             SWIGLU-> silu(gate) * up, rounded
//
// Two block layouts. SwiGLU: a block owns 4 gate tiles and their 4 up tiles
// (one pair per wave, all waves on the block's k range, X reused 4x from
// LDS). QKV / output / down projections (N in the low thousands): a block owns
// one tile pair and its 4 waves split the block's k range four ways, reducing
// through LDS; the narrow column group keeps the split count -- and so the
// last block's reduction -- small. For QKV the pair is tiles j and j+4 of one
// head, so RoPE's (i, i + head_dim/2) pairs stay inside the group.
#include "kernels.h"

namespace pf {

namespace {
constexpr int kU = 6;        // fragment slots per wave
constexpr int kXPad = 16;    // bytes of padding per LDS row (bank spread)
__device__ inline float silu(float g) { return g / (1.0f + expf(-g)); }
}  // namespace

template <typename T, int MT, int EPI, int XS>
__global__ __launch_bounds__(256) void k_fgemm(FusedArgs a) {
  constexpr int E = Elem<T>::E;
  constexpr int KF = 4 * E;
  extern __shared__ __align__(16) unsigned char lds[];
  const int lane = threadIdx.x & 63;
  const int wid = threadIdx.x >> 6;
  const int grp = blockIdx.x;
  const int s = blockIdx.y;
  const int64_t r0 = (int64_t)s * a.KFr / a.splits, r1 = (int64_t)(s + 1) * a.KFr / a.splits;
  const int nfr = (int)(r1 - r0);
  const int xrow = nfr * 64 + kXPad;  // LDS bytes per X row

  constexpr bool WIDE = EPI == FEPI_SWIGLU;
  // weight tiles of this wave and its k fragments [f0, f1) (relative to r0)
  int64_t tile[2];
  bool tv[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    if (EPI == FEPI_SWIGLU) {
      const int64_t gt = (int64_t)grp * 4 + wid;  // gate tile
      tile[j] = j == 0 ? gt : gt + a.up_tile_off;
      tv[j] = gt < a.up_tile_off;
    } else if (EPI == FEPI_QKV) {
      // head grp/(hd/32), tiles j0 and j0 + hd/32 of that head
      const int half_tiles = a.hd / 32;
      const int64_t head = grp / half_tiles, j0 = grp % half_tiles;
      tile[j] = head * (a.hd / 16) + j0 + j * half_tiles;
      tv[j] = tile[j] < a.NTtot;
    } else {
      tile[j] = (int64_t)grp * 2 + j;
      tv[j] = tile[j] < a.NTtot;
    }
  }
  const int f0 = WIDE ? 0 : wid * nfr / 4, f1 = WIDE ? nfr : (wid + 1) * nfr / 4;
  const int nw = f1 - f0;
  const rsrc_t wr = make_rsrc(a.W, (uint32_t)a.W_bytes);
  uint32_t wbase[2];
#pragma unroll
  for (int j = 0; j < 2; ++j)
    wbase[j] = tv[j] ? (uint32_t)(((tile[j] * a.KFr + r0 + f0) * 64 + lane) * 16) : kOOB;

  // start the weight stream before staging X: the weights do not depend on it
  uint4 wv[kU][2];
  auto load = [&](int u, int i) {
    const bool in = i < nw;
#pragma unroll
    for (int j = 0; j < 2; ++j)
      wv[u][j] = bload16(wr, in && wbase[j] != kOOB ? wbase[j] + (uint32_t)i * 1024u : kOOB);
  };
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    load(u, u);
    __builtin_amdgcn_sched_barrier(0);
  }

  // ---- stage X rows 0..MT*16-1, k elements [r0*KF, r1*KF) into LDS ----
  {
    const int nrow = MT * 16;
    const int kbase = (int)(r0 * KF);
    const int chunks = nfr * 4;  // 16-byte chunks per row
    if (XS == XS_NORM) {
      __shared__ float inv_s[80];
      if (threadIdx.x < nrow) {
        const int m = threadIdx.x;
        float ss = 0.f;
        if (m < a.M)
          for (int t = 0; t < a.ss_groups; ++t) ss += a.ss[t * kRowPad + m];
        inv_s[m] = m < a.M ? 1.0f / sqrtf(ss / (float)a.H + a.eps) : 0.f;
      }
      __syncthreads();
      for (int c = threadIdx.x; c < nrow * chunks; c += 256) {
        const int m = c / chunks, ch = c % chunks;
        const int k0 = kbase + ch * E;
        union {
          uint4 v;
          T e[E];
        } u;
        const float inv = inv_s[m];
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const int k = k0 + e;
          const float v = (m < a.M && k < a.H) ? a.xf[(int64_t)m * a.H + k] * inv * a.gain[k] : 0.f;
          Elem<T>::store(u.e, e, v);
        }
        *(uint4 *)(lds + m * xrow + ch * 16) = u.v;
      }
    } else {
      const T *xb = (const T *)a.xb;
      for (int c = threadIdx.x; c < nrow * chunks; c += 256) {
        const int m = c / chunks, ch = c % chunks;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (m < a.M) v = *(const uint4 *)(xb + (int64_t)m * a.ldx + kbase + ch * E);
        *(uint4 *)(lds + m * xrow + ch * 16) = v;
      }
    }
    __syncthreads();
  }

  // ---- main loop ----
  f32x4 acc[MT][2];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[m][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int q = lane >> 4;
  const unsigned char *xl = lds + (lane & 15) * xrow + q * 16 + f0 * 64;
  for (int i = 0; i < nw; i += kU) {
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      // past the k range the weight slot holds zeros (out-of-bounds loads),
      // so the product adds nothing; the X read is clamped into the slice
      const int f = i + u < nw ? i + u : (nw > 0 ? nw - 1 : 0);
      uint4 xv[MT];
#pragma unroll
      for (int m = 0; m < MT; ++m) xv[m] = *(const uint4 *)(xl + m * 16 * xrow + f * 64);
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[m][j] = mma<T>(wv[u][j], xv[m], acc[m][j]);
      load(u, i + kU + u);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  if (!WIDE) {
    // the four waves hold partial sums over different k quarters: reduce in
    // LDS (fixed order) into wave 0
    __shared__ f32x4 red[3][MT][2][64];
    __syncthreads();
    if (wid > 0) {
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int j = 0; j < 2; ++j) red[wid - 1][m][j][lane] = acc[m][j];
    }
    __syncthreads();
    if (wid == 0) {
#pragma unroll
      for (int w = 0; w < 3; ++w)
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
          for (int j = 0; j < 2; ++j) acc[m][j] += red[w][m][j][lane];
    }
  }

  // ---- split partials: lane holds D[n = tile*16 + 4q + i][row = m*16 + lane%16] ----
  float *part = a.part + (int64_t)s * kRowPad * a.ldpart;
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    if (!WIDE && wid != 0) break;
    const int row = m * 16 + (lane & 15);
    if (row >= a.M) continue;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (!tv[j]) continue;
      const int64_t col = tile[j] * 16 + 4 * q;
      *(float4 *)(part + (int64_t)row * a.ldpart + col) =
          make_float4(acc[m][j][0], acc[m][j][1], acc[m][j][2], acc[m][j][3]);
    }
  }

  // ---- the last block of this column group reduces and finishes it ----
  __shared__ int is_last;
  __syncthreads();
  if (threadIdx.x == 0) {
    int last = 1;
    if (a.splits > 1) {
      __threadfence();
      const unsigned old = atomicAdd(&a.counters[grp], 1u);
      last = old == (unsigned)(a.splits - 1);
      if (last) {
        __threadfence();
        atomicExch(&a.counters[grp], 0u);  // ready for the next launch
      }
    }
    is_last = last;
  }
  __syncthreads();
  if (!is_last) return;

  const int M = a.M;
  // sum of the split partials of (row m, column c), eight loads in flight
  auto colsum = [&](int m, int64_t c) {
    const float *p = a.part + (int64_t)m * a.ldpart + c;
    const int64_t st = (int64_t)kRowPad * a.ldpart;
    float v = 0.f;
    int sp = 0;
    for (; sp + 8 <= a.splits; sp += 8) {
      float t[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) t[u] = p[(sp + u) * st];
#pragma unroll
      for (int u = 0; u < 8; ++u) v += t[u];
    }
    for (; sp < a.splits; ++sp) v += p[sp * st];
    return v;
  };
  if (EPI == FEPI_QKV) {
    // columns of tile 0 (i) and tile 1 (i + hd/2) of one head: RoPE pairs
    const int hd = a.hd, half = hd / 2;
    const int64_t qd = (int64_t)a.nq * hd, kvd = (int64_t)a.nkv * hd;
    const int P = *a.kv_len;
    const int64_t plane = a.cap * hd;
    const int64_t hc = (tile[0] / (hd / 16)) * hd;  // first column of the head
    const int ib = (int)(tile[0] * 16 - hc);        // first pair index of the group
    for (int t = threadIdx.x; t < M * 16; t += 256) {
      const int m = t / 16, i = ib + t % 16;
      const float va = colsum(m, hc + i), vb = colsum(m, hc + i + half);
      const int64_t slot = P + m;
      if (hc < qd + kvd) {
        const float cs = a.rope[((int64_t)m * half + i) * 2 + 0];
        const float sn = a.rope[((int64_t)m * half + i) * 2 + 1];
        const float ra = va * cs - vb * sn, rb = va * sn + vb * cs;
        if (hc < qd) {
          T *qo = (T *)a.qout + (int64_t)m * qd + hc;
          Elem<T>::store(qo, i, ra);
          Elem<T>::store(qo, i + half, rb);
        } else {
          const int g = (int)((hc - qd) / hd);
          T *kp = (T *)a.cache + ((int64_t)(a.layer * 2 + 0) * a.nkv + g) * plane + slot * hd;
          Elem<T>::store(kp, i, ra);
          Elem<T>::store(kp, i + half, rb);
        }
      } else {
        const int g = (int)((hc - qd - kvd) / hd);
        T *vp = (T *)a.cache + ((int64_t)(a.layer * 2 + 1) * a.nkv + g) * plane;
        Elem<T>::store(vp, (int64_t)i * a.cap + slot, va);
        Elem<T>::store(vp, (int64_t)(i + half) * a.cap + slot, vb);
      }
    }
  } else if (EPI == FEPI_RESID) {
    // x[:, 32 columns of this group] += sum of splits; per-row sum of squares
    const int64_t c0 = (int64_t)grp * 32;
    for (int m = wid; m < M; m += 4) {
      float acc2 = 0.f;
      if (lane < 32) {
        const float v = a.xf[(int64_t)m * a.H + c0 + lane] + colsum(m, c0 + lane);
        a.xf[(int64_t)m * a.H + c0 + lane] = v;
        acc2 = v * v;
      }
      acc2 = wave_sum(acc2);
      if (lane == 0) a.ss_out[grp * kRowPad + m] = acc2;
    }
  } else {  // FEPI_SWIGLU: gate tiles grp*4..+3 (64 columns) and their up tiles
    const int64_t c0 = (int64_t)grp * 64;
    const int ncol = (int)min((int64_t)64, a.up_tile_off * 16 - c0);
    const int64_t F = a.up_tile_off * 16;
    for (int t = threadIdx.x; t < M * ncol; t += 256) {
      const int m = t / ncol, c = t % ncol;
      const float g = colsum(m, c0 + c), u = colsum(m, F + c0 + c);
      Elem<T>::store((T *)a.act, (int64_t)m * a.ldact + c0 + c, silu(g) * u);
    }
  }
}

int64_t fgemm_groups(int epi, int64_t NTtot, int64_t up_tile_off) {
  return epi == FEPI_SWIGLU ? (up_tile_off + 3) / 4 : (NTtot + 1) / 2;
}

int fgemm_lds_bytes(bool bf16, int mt, int64_t KFr, int splits) {
  (void)bf16;
  const int64_t nfr = (KFr + splits - 1) / splits;
  return (int)(mt * 16 * (nfr * 64 + kXPad));
}

template <typename T, int EPI, int XS>
static hipError_t fg_mt(int mt, const FusedArgs &a, dim3 grid, int lds, hipStream_t s) {
  switch (mt) {
    case 1: k_fgemm<T, 1, EPI, XS><<<grid, 256, lds, s>>>(a); break;
    case 2: k_fgemm<T, 2, EPI, XS><<<grid, 256, lds, s>>>(a); break;
    case 3: k_fgemm<T, 3, EPI, XS><<<grid, 256, lds, s>>>(a); break;
    case 4: k_fgemm<T, 4, EPI, XS><<<grid, 256, lds, s>>>(a); break;
    case 5: k_fgemm<T, 5, EPI, XS><<<grid, 256, lds, s>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T, int EPI, int XS>
static hipError_t fg_attr() {
  const void *ks[] = {(const void *)k_fgemm<T, 1, EPI, XS>, (const void *)k_fgemm<T, 2, EPI, XS>,
                      (const void *)k_fgemm<T, 3, EPI, XS>, (const void *)k_fgemm<T, 4, EPI, XS>,
                      (const void *)k_fgemm<T, 5, EPI, XS>};
  for (const void *k : ks) {
    hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, kFgemmMaxLds);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t fgemm_init() {
  hipError_t e;
  if ((e = fg_attr<bf16_t, FEPI_QKV, XS_NORM>()) != hipSuccess) return e;
  if ((e = fg_attr<bf16_t, FEPI_SWIGLU, XS_NORM>()) != hipSuccess) return e;
  if ((e = fg_attr<bf16_t, FEPI_RESID, XS_BF16>()) != hipSuccess) return e;
  if ((e = fg_attr<float, FEPI_QKV, XS_NORM>()) != hipSuccess) return e;
  if ((e = fg_attr<float, FEPI_SWIGLU, XS_NORM>()) != hipSuccess) return e;
  return fg_attr<float, FEPI_RESID, XS_BF16>();
}

template <typename T>
static hipError_t fg_t(int epi, int xs, int mt, const FusedArgs &a, hipStream_t s) {
  const int64_t groups = fgemm_groups(epi, a.NTtot, a.up_tile_off);
  dim3 grid((unsigned)groups, (unsigned)a.splits);
  const int lds = fgemm_lds_bytes(sizeof(T) == 2, mt, a.KFr, a.splits);
  if (epi == FEPI_QKV) return fg_mt<T, FEPI_QKV, XS_NORM>(mt, a, grid, lds, s);
  if (epi == FEPI_SWIGLU) return fg_mt<T, FEPI_SWIGLU, XS_NORM>(mt, a, grid, lds, s);
  if (xs == XS_BF16) return fg_mt<T, FEPI_RESID, XS_BF16>(mt, a, grid, lds, s);
  return hipErrorInvalidValue;
}

hipError_t launch_fgemm(bool bf16, int epi, int xs, int mt, const FusedArgs &a, hipStream_t s) {
  return bf16 ? fg_t<bf16_t>(epi, xs, mt, a, s) : fg_t<float>(epi, xs, mt, a, s);
}

// x[m] = embed[token m]; per-group (32 columns) sums of squares of x
template <typename T>
__global__ __launch_bounds__(256) void k_embed_ss(const T *embed, const int32_t *rowinfo, int H,
                                                  float *x, float *ss) {
  const int m = blockIdx.x;
  const int tok = rowinfo[m * 4];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  float *xr = x + (int64_t)m * H;
  for (int g = wid; g < H / 32; g += 4) {
    float acc2 = 0.f;
    if (lane < 32) {
      const int c = g * 32 + lane;
      const float v = Elem<T>::load(embed, (int64_t)tok * H + c);
      xr[c] = v;
      acc2 = v * v;
    }
    acc2 = wave_sum(acc2);
    if (lane == 0) ss[g * kRowPad + m] = acc2;
  }
}

hipError_t launch_embed_ss(bool bf16, const void *embed, const int32_t *rowinfo, int M, int H,
                           float *x, float *ss, hipStream_t s) {
  if (bf16)
    k_embed_ss<bf16_t><<<M, 256, 0, s>>>((const bf16_t *)embed, rowinfo, H, x, ss);
  else
    k_embed_ss<float><<<M, 256, 0, s>>>((const float *)embed, rowinfo, H, x, ss);
  return hipGetLastError();
}

// xn = bf16(x * rsqrt(mean(x^2) + eps) * gain) from the per-group sums
template <typename T>
__global__ __launch_bounds__(256) void k_norm_ss(const float *x, const float *ss, int groups,
                                                 int H, const float *gain, float eps, T *xn,
                                                 int64_t ldxn) {
  const int m = blockIdx.x;
  float t = 0.f;
  for (int g = 0; g < groups; ++g) t += ss[g * kRowPad + m];
  const float inv = 1.0f / sqrtf(t / (float)H + eps);
  for (int k = threadIdx.x; k < H; k += 256)
    Elem<T>::store(xn + (int64_t)m * ldxn, k, x[(int64_t)m * H + k] * inv * gain[k]);
}

hipError_t launch_norm_ss(bool bf16, const float *x, const float *ss, int groups, int M, int H,
                          const float *gain, float eps, void *xn, int64_t ldxn, hipStream_t s) {
  if (bf16)
    k_norm_ss<bf16_t><<<M, 256, 0, s>>>(x, ss, groups, H, gain, eps, (bf16_t *)xn, ldxn);
  else
    k_norm_ss<float><<<M, 256, 0, s>>>(x, ss, groups, H, gain, eps, (float *)xn, ldxn);
  return hipGetLastError();
}

}  // namespace pf
