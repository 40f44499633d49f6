// Prefill GEMM (bf16): Y[M x N] = X[M x K] * W[N x K]^T for chunks of a few
// hundred rows, compute-bound. A block of 4 waves owns 256 rows of W (sixteen
// 16-row fragment tiles) by 128 rows of X; each wave 64 W rows x the 128 X
// rows, as 2 x 4 tiles of the 32 x 32 x 16 bf16 matrix instruction.
//
// W goes from HBM straight into the A operands: the packed fragment layout
// makes a lane's 16-byte chunk of a 32-row tile one contiguous read, and each
// W element is used by one wave only, so staging it in LDS would only add LDS
// traffic. Each wave keeps a ring of D 16-k steps of W loads in flight. X
// rows are shared by the four waves: they are staged in LDS, 64 k per stage,
// double-buffered, with their 16-byte chunks XOR-swizzled by row so the 32
// rows an operand read touches hit different banks.
//
// Blocks that read the same W slice (the X row blocks of one W tile and
// split) get consecutive ids of one residue mod 8, so they run at the same
// time on one XCD and the slice comes from HBM once into that XCD's L2.
// Narrow outputs split K into partial sums that the following reduction
// kernel adds in split order.
#include "kernels.h"

namespace pf {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ inline f32x16 mma32(const uint4 &a, const uint4 &b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ inline float silu_f(float g) { return g / (1.0f + expf(-g)); }

// grid geometry: gx W tiles (256 rows; SwiGLU: 128 gate + 128 up rows) by gy
// X row blocks by gz K splits
struct PreGrid {
  int gx, gy, gz;
};

template <int EPI, int D, int MINB>
__global__ __launch_bounds__(256, MINB) void k_gemm_pre(BigGemmArgs a, PreGrid pg) {
  static_assert(D % 4 == 0, "the W ring holds whole stages");
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int r32 = lane & 31, hi = lane >> 5;
  // block id -> (W tile and split, X row block); see the header
  const int bj = blockIdx.x >> 3;
  const int wq = (bj / pg.gy) * 8 + (blockIdx.x & 7);
  if (wq >= pg.gx * pg.gz) return;
  const int bx = wq % pg.gx, by = bj % pg.gy, bz = wq / pg.gx;

  // first 16-row tile of the wave's two 32-row A tiles
  int64_t t0[2];
  bool tv[2];
  if (EPI == BIG_SWIGLU) {
    const int64_t g = (int64_t)bx * 8 + 2 * wid;  // gate tiles g, g + 1 and their up tiles
    t0[0] = g;
    t0[1] = g + a.up_tile_off;
    tv[0] = tv[1] = g < a.up_tile_off;
  } else {
    const int64_t g = (int64_t)bx * 16 + 4 * wid;
    t0[0] = g;
    t0[1] = g + 2;
    tv[0] = g < a.NTtot;
    tv[1] = g + 2 < a.NTtot;
  }
  const int64_t row0 = (int64_t)by * 128;
  const int64_t S = pg.gz;
  const int64_t kf_lo = bz * a.KFr / S, kf_hi = (bz + 1) * a.KFr / S;
  float *const y = a.y + (S > 1 ? bz * a.ystride : 0);
  const rsrc_t wr = make_rsrc(a.W, (uint32_t)a.W_bytes);
  const rsrc_t xr = make_rsrc(a.X, (uint32_t)(a.x_rows * a.ldx * 2));
  const int64_t nsteps = 2 * (kf_hi - kf_lo);  // 16-k steps
  const int64_t nst = (nsteps + 3) / 4;        // 64-k stages

  // A operand of step i: row r32 of the 32-row tile (16-row tile t0 + r32/16,
  // its row r32 % 16), k = 16 * (i % 2) + 8 * hi .. + 8 of fragment i / 2.
  // Tiles past the matrix read out of the resource: zeros.
  uint32_t wbase[2];
#pragma unroll
  for (int g = 0; g < 2; ++g)
    wbase[g] = (uint32_t)(((t0[g] + (r32 >> 4)) * a.KFr + kf_lo) * 1024 + (lane & 15) * 16 + hi * 256);
  uint4 ring[D][2];
  auto wload = [&](int slot, int64_t i) {
    const bool in = i < nsteps;
#pragma unroll
    for (int g = 0; g < 2; ++g)
      ring[slot][g] =
          bload16_stream(wr, in && tv[g] ? wbase[g] + (uint32_t)((i >> 1) * 1024 + (i & 1) * 512) : kOOB);
  };

  __shared__ uint4 lx[2][128][8];  // stage, row, swizzled 16-byte chunk
  uint4 gx[4];
  auto gload = [&](int64_t st) {
    const int64_t kf0 = kf_lo + st * 2;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int idx = tid + 256 * r;
      const int row = idx >> 3, ch = idx & 7;
      const int64_t k = kf0 * 32 + ch * 8;
      // chunks past the split's k range load zeros
      const bool in = kf0 + (ch >> 2) < kf_hi && k < a.ldx;
      gx[r] = bload16(xr, in ? (uint32_t)(((row0 + row) * a.ldx + k) * 2) : kOOB);
    }
  };
  auto lstore = [&](int b) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int idx = tid + 256 * r;
      const int row = idx >> 3, ch = idx & 7;
      lx[b][row][ch ^ (row & 7)] = gx[r];
    }
  };

  f32x16 acc[2][4];
#pragma unroll
  for (int g = 0; g < 2; ++g)
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[g][t][v] = 0.f;

  // B operands of a 16-k step, two sets: the next step's are read from LDS
  // before this step's products issue
  uint4 bq[2][4];
  auto readb = [&](int b, int h, int set) {
    const int kk = h >> 1, kq = 2 * (h & 1) + hi;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int row = t * 32 + r32;
      bq[set][t] = lx[b][row][(kk * 4 + kq) ^ (row & 7)];
    }
  };
  // stage st, its W steps in ring slots slot0 .. slot0 + 3
  auto stage = [&](int64_t st, int b, int slot0) {
    if (st + 1 < nst) gload(st + 1);
    readb(b, 0, 0);
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      if (h < 3) readb(b, h + 1, (h + 1) & 1);
      __builtin_amdgcn_sched_barrier(0);
      const int slot = (slot0 + h) % D;
#pragma unroll
      for (int g = 0; g < 2; ++g)
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[g][t] = mma32(ring[slot][g], bq[h & 1][t], acc[g][t]);
      wload(slot, st * 4 + h + D);
      // keep the refill right behind its slot's products
      __builtin_amdgcn_sched_barrier(0);
    }
    if (st + 1 < nst) lstore(b ^ 1);
    __syncthreads();
  };

#pragma unroll
  for (int i = 0; i < D; ++i) wload(i, i);
  gload(0);
  lstore(0);
  __syncthreads();
  // whole ring turns with static slots, then the remaining stages
  constexpr int SR = D / 4;
  int64_t st = 0;
  for (; st + SR <= nst; st += SR) {
#pragma unroll
    for (int u = 0; u < SR; ++u) stage(st + u, (int)((st + u) & 1), 4 * u);
  }
#pragma unroll
  for (int u = 0; u < SR - 1; ++u)
    if (st + u < nst) stage(st + u, (int)((st + u) & 1), 4 * u);

  // lane holds D[n = 8*(v/4) + 4*hi + v%4 of its 32-row A tile][token = r32 of its B tile]
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int64_t row = row0 + t * 32 + r32;
    if (row >= a.M) continue;
#pragma unroll
    for (int q = 0; q < 4; ++q) {  // four consecutive n per group of four values
      const int i = 8 * q + 4 * hi;  // n within the 32-row tile
      if (EPI == BIG_SWIGLU) {
        if (t0[0] + (i >> 4) >= a.up_tile_off) continue;
        bf16_t *dst = (bf16_t *)a.act + row * a.ldact + t0[0] * 16 + i;
#pragma unroll
        for (int u = 0; u < 4; ++u)
          Elem<bf16_t>::store(dst, u, silu_f(acc[0][t][4 * q + u]) * acc[1][t][4 * q + u]);
      } else {
#pragma unroll
        for (int g = 0; g < 2; ++g) {
          if (t0[g] + (i >> 4) >= a.NTtot) continue;
          float4 *dst = (float4 *)(y + row * a.ldy + t0[g] * 16 + i);
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
  if (a.x_rows % 128 != 0 || a.ldx % 32 != 0 || a.W_bytes >= ((int64_t)1 << 31) ||
      a.x_rows * a.ldx * 2 >= ((int64_t)1 << 31))
    return hipErrorInvalidValue;
  if (a.splits > 1 && (epi != BIG_STORE || a.splits > a.KFr)) return hipErrorInvalidValue;
  PreGrid pg;
  pg.gy = (int)((a.M + 127) / 128);
  pg.gz = a.splits > 1 ? a.splits : 1;
  pg.gx = epi == BIG_SWIGLU ? (int)((a.up_tile_off + 7) / 8) : (int)((a.NTtot + 15) / 16);
  const dim3 grid(8u * (unsigned)((pg.gx * pg.gz + 7) / 8) * (unsigned)pg.gy);
  // SwiGLU: a short W ring and two blocks per CU; the split projections: a
  // longer ring at one block per CU (measured best for each)
  if (epi == BIG_SWIGLU)
    PF_TRY(launch_k(k_gemm_pre<BIG_SWIGLU, 4, 2>, grid, 256, s, a, pg));
  else if (epi == BIG_STORE)
    PF_TRY(launch_k(k_gemm_pre<BIG_STORE, 8, 1>, grid, 256, s, a, pg));
  else
    PF_TRY(launch_k(k_gemm_pre<BIG_RESID, 8, 1>, grid, 256, s, a, pg));
  return hipGetLastError();
}

}  // namespace pf
