// Prefill GEMM (bf16): Y[M x N] = X[M x K] * W[N x K]^T for chunks of a few
// hundred rows, compute-bound. A block of 4 waves owns 128 rows of W (eight
// 16-row fragment tiles) by 128 rows of X; each wave a 64 x 64 quarter as
// 2 x 2 tiles of the 32 x 32 x 16 bf16 matrix instruction. Both operands are
// staged through LDS, two k fragments (64 k) per stage, double-buffered:
// the next stage's global loads are in flight while the current stage is
// multiplied. Narrow outputs split K over grid.z into partial sums that the
// following reduction kernel adds in split order. W keeps the packed
// fragment layout in LDS (a lane's 16-byte operand chunk is one contiguous
// read); X rows are stored with their 16-byte chunks XOR-swizzled by row, so
// the 32 rows a matrix instruction reads hit different banks.
#include "kernels.h"

namespace pf {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ inline f32x16 mma32(const uint4 &a, const uint4 &b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ inline float silu_f(float g) { return g / (1.0f + expf(-g)); }

// LDS slot of the 16-row W tile holding rows 16*half .. of a wave's n-group
__device__ inline int wave_slot(int epi, int wn, int g, int half) {
  return epi == BIG_SWIGLU ? (g == 0 ? 2 * wn + half : 4 + 2 * wn + half) : 4 * wn + 2 * g + half;
}

template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_pre(BigGemmArgs a) {
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm = wid & 1, wn = wid >> 1;
  // the block's eight W tiles, in LDS slot order
  int64_t wt[8];
  bool wvld[8];
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    if (EPI == BIG_SWIGLU) {
      const int64_t g = (int64_t)blockIdx.x * 4 + (s & 3);
      wt[s] = s < 4 ? g : g + a.up_tile_off;
      wvld[s] = g < a.up_tile_off;
    } else {
      wt[s] = (int64_t)blockIdx.x * 8 + s;
      wvld[s] = wt[s] < a.NTtot;
    }
  }
  const int64_t row0 = (int64_t)blockIdx.y * 128;
  // k fragments of this block's split (grid.z; one split without)
  const int64_t S = a.splits > 1 ? a.splits : 1;
  const int64_t kf_lo = blockIdx.z * a.KFr / S, kf_hi = (blockIdx.z + 1) * a.KFr / S;
  float *const y = a.y + (S > 1 ? blockIdx.z * a.ystride : 0);
  const rsrc_t wr = make_rsrc(a.W, (uint32_t)a.W_bytes);
  const rsrc_t xr = make_rsrc(a.X, (uint32_t)(a.x_rows * a.ldx * 2));

  __shared__ uint4 lw[2][8][2][64];  // stage, slot, fragment in the stage, lane chunk
  __shared__ uint4 lx[2][128][8];    // stage, row, swizzled 16-byte chunk
  const int64_t nst = (kf_hi - kf_lo + 1) / 2;

  // global loads of one stage: four W and four X chunks per thread
  uint4 gw[4], gx[4];
  auto gload = [&](int64_t st) {
    const int64_t kf0 = kf_lo + st * 2;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int idx = tid + 256 * r;
      const int frag = idx >> 6, ln = idx & 63;
      const int s = frag >> 1, kk = frag & 1;
      // fragments past the split's range load zeros (W), so the X chunks
      // there add nothing
      const bool in = wvld[s] && kf0 + kk < kf_hi;
      gw[r] = bload16(wr, in ? (uint32_t)(((wt[s] * a.KFr + kf0 + kk) * 64 + ln) * 16) : kOOB);
      const int row = idx >> 3, ch = idx & 7;
      const int64_t k = kf0 * 32 + ch * 8;
      gx[r] = bload16(xr, k < a.ldx ? (uint32_t)(((row0 + row) * a.ldx + k) * 2) : kOOB);
    }
  };
  auto lstore = [&](int b) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int idx = tid + 256 * r;
      const int frag = idx >> 6, ln = idx & 63;
      lw[b][frag >> 1][frag & 1][ln] = gw[r];
      const int row = idx >> 3, ch = idx & 7;
      lx[b][row][ch ^ (row & 7)] = gx[r];
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int g = 0; g < 2; ++g)
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[g][t][v] = 0.f;

  const int r32 = lane & 31, hi = lane >> 5;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int64_t st = 0; st < nst; ++st) {
    const int b = (int)(st & 1);
    if (st + 1 < nst) gload(st + 1);
#pragma unroll
    for (int h = 0; h < 4; ++h) {  // 16-k steps: fragment h / 2, half h % 2
      const int kk = h >> 1, kq = 2 * (h & 1) + hi;
      uint4 A[2], B[2];
#pragma unroll
      for (int g = 0; g < 2; ++g) A[g] = lw[b][wave_slot(EPI, wn, g, r32 >> 4)][kk][kq * 16 + (lane & 15)];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int row = wm * 64 + t * 32 + r32;
        B[t] = lx[b][row][(kk * 4 + kq) ^ (row & 7)];
      }
#pragma unroll
      for (int g = 0; g < 2; ++g)
#pragma unroll
        for (int t = 0; t < 2; ++t) acc[g][t] = mma32(A[g], B[t], acc[g][t]);
    }
    if (st + 1 < nst) lstore(b ^ 1);
    __syncthreads();
  }

  // lane holds D[n = 8*(v/4) + 4*hi + v%4 of its n-group][token = r32 of its token group]
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int64_t row = row0 + wm * 64 + t * 32 + r32;
    if (row >= a.M) continue;
#pragma unroll
    for (int q = 0; q < 4; ++q) {  // four consecutive n per group of four values
      const int i = 8 * q + 4 * hi;    // n within the 32-row group
      if (EPI == BIG_SWIGLU) {
        const int s = wave_slot(EPI, wn, 0, i >> 4);
        if (!wvld[s]) continue;
        const int64_t col = wt[s] * 16 + (i & 15);
        bf16_t *dst = (bf16_t *)a.act + row * a.ldact + col;
#pragma unroll
        for (int u = 0; u < 4; ++u)
          Elem<bf16_t>::store(dst, u, silu_f(acc[0][t][4 * q + u]) * acc[1][t][4 * q + u]);
      } else {
#pragma unroll
        for (int g = 0; g < 2; ++g) {
          const int s = wave_slot(EPI, wn, g, i >> 4);
          if (!wvld[s]) continue;
          const int64_t col = wt[s] * 16 + (i & 15);
          float4 *dst = (float4 *)(y + row * a.ldy + col);
          float4 v = make_float4(acc[g][t][4 * q], acc[g][t][4 * q + 1], acc[g][t][4 * q + 2],
                                 acc[g][t][4 * q + 3]);
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
}

}  // namespace

hipError_t launch_gemm_pre(int epi, const BigGemmArgs &a, hipStream_t s) {
  if (a.x_rows % 128 != 0 || a.ldx % 32 != 0) return hipErrorInvalidValue;
  if (a.splits > 1 && (epi != BIG_STORE || a.splits > a.KFr)) return hipErrorInvalidValue;
  const unsigned gy = (unsigned)((a.M + 127) / 128);
  const unsigned gz = a.splits > 1 ? (unsigned)a.splits : 1u;
  if (epi == BIG_SWIGLU) {
    dim3 grid((unsigned)((a.up_tile_off + 3) / 4), gy);
    PF_TRY(launch_k(k_gemm_pre<BIG_SWIGLU>, grid, 256, s, a));
  } else {
    dim3 grid((unsigned)((a.NTtot + 7) / 8), gy, gz);
    if (epi == BIG_STORE)
      PF_TRY(launch_k(k_gemm_pre<BIG_STORE>, grid, 256, s, a));
    else
      PF_TRY(launch_k(k_gemm_pre<BIG_RESID>, grid, 256, s, a));
  }
  return hipGetLastError();
}

}  // namespace pf
