// Tiled GEMM for prefill chunks: Y[M x N] = X[M x K] * W[N x K]^T with M in
// the hundreds, compute-bound. A block of 4 waves owns a 128 (rows of X) x
// 128 (rows of W) tile; each wave a 64 x 64 quarter, i.e. 4 x 4 MFMA 16x16
// accumulators. W comes from the same packed fragments as the verify GEMM
// (one contiguous 1 KiB load per 16 rows x one k fragment, straight into the
// MFMA A operand); X rows go into the B operand. The k loop is a ring of kU
// fragment slots with the load order pinned, as in the verify GEMM.
#include "kernels.h"

namespace pf {

namespace {
constexpr int kU = 3;
__device__ inline float silu(float g) { return g / (1.0f + expf(-g)); }
}  // namespace

template <typename T, int EPI>
__global__ __launch_bounds__(256) void k_gemm_big(BigGemmArgs a) {
  constexpr int E = Elem<T>::E;
  constexpr int MT = 4, NT = 4;
  const int lane = threadIdx.x & 63;
  const int wid = threadIdx.x >> 6;
  const int wm = wid & 1, wn = wid >> 1;
  const int64_t row0 = (int64_t)blockIdx.y * 128 + wm * 64;

  int64_t tile[NT];
  bool tv[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    if (EPI == BIG_SWIGLU) {
      // block covers gate tiles 4*bx .. 4*bx+3 and the matching up tiles;
      // wave wn takes two gate tiles (j = 0, 1) and their up tiles (j = 2, 3)
      const int64_t gt = (int64_t)blockIdx.x * 4 + wn * 2 + (j & 1);
      tile[j] = j < 2 ? gt : gt + a.up_tile_off;
      tv[j] = gt < a.up_tile_off;
    } else {
      tile[j] = (int64_t)blockIdx.x * 8 + wn * 4 + j;
      tv[j] = tile[j] < a.NTtot;
    }
  }
  const rsrc_t wr = make_rsrc(a.W, (uint32_t)a.W_bytes);
  const rsrc_t xr = make_rsrc(a.X, (uint32_t)(a.x_rows * a.ldx * sizeof(T)));
  uint32_t wbase[NT], xbase[MT];
#pragma unroll
  for (int j = 0; j < NT; ++j)
    wbase[j] = tv[j] ? (uint32_t)((tile[j] * a.KFr * 64 + lane) * 16) : kOOB;
#pragma unroll
  for (int m = 0; m < MT; ++m)
    xbase[m] = (uint32_t)(((row0 + m * 16 + (lane & 15)) * a.ldx + (lane >> 4) * E) * sizeof(T));

  f32x4 acc[MT][NT];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[m][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int64_t n = a.KFr;
  uint4 wv[kU][NT], xv[kU][MT];
  auto load = [&](int u, int64_t i) {
    const bool in = i < n;
#pragma unroll
    for (int j = 0; j < NT; ++j)
      wv[u][j] = bload16(wr, in && wbase[j] != kOOB ? wbase[j] + (uint32_t)(i * 1024) : kOOB);
#pragma unroll
    for (int m = 0; m < MT; ++m)
      xv[u][m] = bload16(xr, in ? xbase[m] + (uint32_t)(i * 4 * E * sizeof(T)) : kOOB);
  };
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    load(u, u);
    __builtin_amdgcn_sched_barrier(0);
  }
  for (int64_t i = 0; i < n; i += kU) {
#pragma unroll
    for (int u = 0; u < kU; ++u) {
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[m][j] = mma<T>(wv[u][j], xv[u][m], acc[m][j]);
      load(u, i + kU + u);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // lane holds D[n = tile*16 + 4q + i][row = row0 + m*16 + lane%16]
  const int q = lane >> 4;
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const int64_t row = row0 + m * 16 + (lane & 15);
    if (row >= a.M) continue;
    if (EPI == BIG_SWIGLU) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        if (!tv[j]) continue;
        const int64_t col = tile[j] * 16 + 4 * q;
        T *dst = (T *)a.act + row * a.ldact + col;
#pragma unroll
        for (int i = 0; i < 4; ++i) Elem<T>::store(dst, i, silu(acc[m][j][i]) * acc[m][j + 2][i]);
      }
    } else {
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        if (!tv[j]) continue;
        const int64_t col = tile[j] * 16 + 4 * q;
        float4 *dst = (float4 *)(a.y + row * a.ldy + col);
        float4 v = make_float4(acc[m][j][0], acc[m][j][1], acc[m][j][2], acc[m][j][3]);
        if (EPI == BIG_RESID) {
          const float4 o = *dst;
          v.x += o.x;
          v.y += o.y;
          v.z += o.z;
          v.w += o.w;
        }
        *dst = v;
      }
    }
  }
}

template <typename T>
static hipError_t big_t(int epi, const BigGemmArgs &a, hipStream_t s) {
  const unsigned gy = (unsigned)((a.M + 127) / 128);
  if (epi == BIG_SWIGLU) {
    dim3 grid((unsigned)((a.up_tile_off + 3) / 4), gy);
    PF_TRY(launch_k(k_gemm_big<T, BIG_SWIGLU>, grid, 256, s, a));
  } else {
    dim3 grid((unsigned)((a.NTtot + 7) / 8), gy);
    if (epi == BIG_STORE)
      PF_TRY(launch_k(k_gemm_big<T, BIG_STORE>, grid, 256, s, a));
    else
      PF_TRY(launch_k(k_gemm_big<T, BIG_RESID>, grid, 256, s, a));
  }
  return hipGetLastError();
}

hipError_t launch_gemm_big(bool bf16, int epi, const BigGemmArgs &a, hipStream_t s) {
  return bf16 ? big_t<bf16_t>(epi, a, s) : big_t<float>(epi, a, s);
}

}  // namespace pf
