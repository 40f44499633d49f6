// Skinny GEMM for the verify step: Y[M x N] = X[M x K] * W[N x K]^T with
// M <= 80 rows (the current token plus the draft) and N, K in the thousands.
// The work is bound by streaming W from HBM once; the matrix cores only have
// to keep up. W is pre-packed so every wave load is one contiguous 1 KiB
// fragment (16 rows x 32 bf16 or 16 fp32 columns), which goes straight into
// the MFMA A operand; X rows go into the B operand. Each block of 4 waves owns
// NT n-tiles and one K range (split-K), the waves split that range four ways
// and reduce through LDS in a fixed order, so results are deterministic.
#include "kernels.h"

namespace pf {

// ---------------------------------------------------------------------------
// weight packing
// ---------------------------------------------------------------------------

// Source row of packed row n when the rows are attention heads of rope_hd
// dimensions packed RoPE-paired: tile t of a head (16 rows) holds dimensions
// 8t .. 8t+7 and their rotation partners rope_hd/2 + 8t .. rope_hd/2 + 8t+7,
// so a 16-column output tile can be rotated without its neighbours.
__device__ inline int64_t rope_paired_row(int64_t n, int rope_hd) {
  const int64_t head = n / rope_hd;
  const int w = (int)(n % rope_hd), t = w / 16, c = w % 16;
  const int dim = c < 8 ? 8 * t + c : rope_hd / 2 + 8 * t + (c - 8);
  return head * rope_hd + dim;
}

template <typename T>
__global__ void k_pack(const T *__restrict__ src, int64_t N, int64_t K, int64_t KFr,
                       int64_t NT, int64_t layers, int64_t src_layer_stride, int rope_hd,
                       uint4 *__restrict__ dst) {
  constexpr int E = Elem<T>::E;
  constexpr int KF = 4 * E;
  const int64_t per_layer = NT * KFr * 64;
  const int64_t total = per_layer * layers;
  for (int64_t c = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; c < total;
       c += (int64_t)gridDim.x * blockDim.x) {
    int64_t l = c / per_layer, r = c % per_layer;
    int lane = (int)(r & 63);
    int64_t frag = r >> 6;
    int64_t nt = frag / KFr, kf = frag % KFr;
    int64_t n = nt * 16 + (lane & 15);
    int64_t k0 = kf * KF + (lane >> 4) * E;
    union {
      uint4 v;
      T e[E];
    } u;
    const int64_t ns = rope_hd > 0 ? rope_paired_row(n, rope_hd) : n;
    const T *row = src + l * src_layer_stride + ns * K;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      int64_t k = k0 + e;
      if (n < N && ns < N && k < K) {
        u.e[e] = row[k];
      } else {
        memset(&u.e[e], 0, sizeof(T));
      }
    }
    dst[c] = u.v;
  }
}

hipError_t launch_pack(const void *src, int64_t N, int64_t K, int64_t layers,
                       int64_t src_layer_stride, bool bf16, const Packed &g, void *dst,
                       hipStream_t s, int rope_hd) {
  if (rope_hd > 0 && (rope_hd % 16 != 0 || N % rope_hd != 0)) return hipErrorInvalidValue;
  int64_t total = g.NT * g.KFr * 64 * layers;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (bf16)
    PF_TRY(launch_k(k_pack<bf16_t>, (unsigned)blocks, 256, s, (const bf16_t *)src, N, K, g.KFr, g.NT, layers,
                                                    src_layer_stride, rope_hd, (uint4 *)dst));
  else
    PF_TRY(launch_k(k_pack<float>, (unsigned)blocks, 256, s, (const float *)src, N, K, g.KFr, g.NT, layers,
                                                   src_layer_stride, rope_hd, (uint4 *)dst));
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// GEMM
// ---------------------------------------------------------------------------


// n tiles per block. Each X load instruction costs about as much as a W
// load whatever its bytes, so the more X tiles (rows) a step has, the more W
// tiles a block should meet each X fragment with. The partial-sum projections
// take NP = 2 or 4 W tiles (gemm_partial_tiles), gate/up NP gate/up pairs
// (gemm_swiglu_pairs), both chosen on the host from the model's tiles against
// the CUs; the lm_head takes four. Per tile the sums are the same: a tile's k
// range and its split of the range over the waves do not depend on how many
// tiles share the block.
template <int EPI, int MT, int NP> struct EpiTiles {
  static constexpr int NT = EPI == EPI_ARGMAX ? 4 : EPI == EPI_SWIGLU ? 2 * NP : NP;
  static constexpr int kU = NT >= 6 ? 3 : NT >= 4 ? 4 : 6;  // fragment slots in flight per wave
  // three pairs at three X tiles run two blocks per CU (206 registers)
  static constexpr int MinBlocks = EPI == EPI_SWIGLU && NP == 3 && MT == 3 ? 2 : 1;
};

__device__ inline float silu(float g) { return g / (1.0f + expf(-g)); }

template <typename T, int MT, int EPI, int NP>
__global__ __launch_bounds__(256, (EpiTiles<EPI, MT, NP>::MinBlocks)) void k_gemm(GemmArgs a) {
  constexpr int NT = EpiTiles<EPI, MT, NP>::NT;
  constexpr int kU = EpiTiles<EPI, MT, NP>::kU;
  constexpr int E = Elem<T>::E;
  const int lane = threadIdx.x & 63;
  const int wid = threadIdx.x >> 6;

  // n tiles of this block
  int64_t tile[NT];
  bool tv[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    if (EPI == EPI_SWIGLU) {  // gate tiles first, then their up tiles
      constexpr int PR = NT / 2;
      const int64_t t = (int64_t)blockIdx.x * PR + j % PR;
      tile[j] = j < PR ? t : t + a.up_tile_off;
      tv[j] = t < a.up_tile_off;
    } else {
      tile[j] = (int64_t)blockIdx.x * NT + j;
      tv[j] = tile[j] < a.NTtot;
    }
  }

  // k fragment range of this wave
  const int64_t s = blockIdx.y;
  const int64_t r0 = s * a.KFr / a.splits, r1 = (s + 1) * a.KFr / a.splits;
  const int64_t f0 = r0 + wid * (r1 - r0) / 4, f1 = r0 + (wid + 1) * (r1 - r0) / 4;
  const int64_t n = f1 - f0;

  const rsrc_t wr = make_rsrc(a.W, (uint32_t)a.W_bytes);
  const rsrc_t xr = make_rsrc(a.X, (uint32_t)(kRowPad * a.ldx * sizeof(T)));
  uint32_t wbase[NT], xbase[MT];
#pragma unroll
  for (int j = 0; j < NT; ++j)
    wbase[j] = tv[j] ? (uint32_t)(((tile[j] * a.KFr + f0) * 64 + lane) * 16) : kOOB;
  // X is fragment-packed: fragment (m, f) is 64 lanes x 16 B, contiguous.
  // Rows past M are padding of the last 16-row tile: their lanes load
  // nothing (out-of-bounds offset gives zeros without memory traffic).
  const int64_t xkfr = a.ldx / (4 * E);
#pragma unroll
  for (int m = 0; m < MT; ++m)
    xbase[m] = m * 16 + (lane & 15) < a.M ? (uint32_t)(((m * xkfr + f0) * 64 + lane) * 16) : kOOB;

  f32x4 acc[MT][NT];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[m][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  // ring of kU fragment slots: compute slot u, then refill it with the
  // fragment kU positions ahead. Loads past the wave's range go out of the
  // buffer resource's bounds and return zeros without memory traffic, so the
  // loop body is straight-line and the wait counts stay static.
  uint4 wv[kU][NT], xv[kU][MT];
  auto load = [&](int u, int64_t i) {
    const bool in = i < n;
#pragma unroll
    for (int j = 0; j < NT; ++j)
      wv[u][j] = bload16_stream(wr, in && wbase[j] != kOOB ? wbase[j] + (uint32_t)(i * 1024) : kOOB);
#pragma unroll
    for (int m = 0; m < MT; ++m)
      xv[u][m] = bload16(xr, in && xbase[m] != kOOB ? xbase[m] + (uint32_t)(i * 1024) : kOOB);
  };
  // SwiGLU: the rows' deferred RMSNorm scales (see RowInv)
  __shared__ float invl[EPI == EPI_SWIGLU ? kRowPad : 1];
  RowInv ri;
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    load(u, u);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (EPI == EPI_SWIGLU) ri.issue(a.rs, a.M);
  __builtin_amdgcn_sched_barrier(0);
  for (int64_t i = 0; i < n; i += kU) {
#pragma unroll
    for (int u = 0; u < kU; ++u) {
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[m][j] = mma<T>(wv[u][j], xv[u][m], acc[m][j]);
      load(u, i + kU + u);
      // keep slot order: the refill of slot u must not sink below later slots,
      // or the next pass would have to wait for every load in flight
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // lane holds D[n = tile*16 + 4*q + i][row = m*16 + lane%16], q = lane/16
  const int q = lane >> 4;
  if (EPI != EPI_ARGMAX) {
    // every wave stores its partial sums; wave w then finishes the outputs
    // w, w + 4, ... of the block, adding the four waves' sums in wave order
    __shared__ f32x4 red[4][MT][NT][64];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int j = 0; j < NT; ++j) red[wid][m][j][lane] = acc[m][j];
    if (EPI == EPI_SWIGLU) ri.finish(a.rs, a.M, invl);
    __syncthreads();
    auto sum4 = [&](int m, int j) {
      f32x4 v = red[0][m][j][lane];
#pragma unroll
      for (int w = 1; w < 4; ++w) v += red[w][m][j][lane];
      return v;
    };
    if (EPI == EPI_PARTIAL) {
#pragma unroll
      for (int k = 0; k < MT * NT; ++k) {
        const int m = k / NT, j = k % NT;
        const int row = m * 16 + (lane & 15);
        if (k % 4 != wid || row >= a.M || !tv[j]) continue;
        const f32x4 v = sum4(m, j);
        const int64_t col = tile[j] * 16 + 4 * q;
        *(float4 *)(a.out + (s * kRowPad + row) * a.ldo + col) = make_float4(v[0], v[1], v[2], v[3]);
      }
    } else {  // EPI_SWIGLU
      constexpr int PR = NT / 2;
#pragma unroll
      for (int k = 0; k < MT * PR; ++k) {
        const int m = k / PR, p = k % PR;
        const int row = m * 16 + (lane & 15);
        if (k % 4 != wid || row >= a.M || !tv[p]) continue;
        const f32x4 g = sum4(m, p), u = sum4(m, p + PR);
        const float inv = invl[row];
        // act is the next GEMM's X: fragment-packed; the four columns stay in
        // one E-element chunk
        const int64_t col = tile[p] * 16 + 4 * q;
        T *dst = (T *)a.act + act_off<T>(row, col, a.ldact);
#pragma unroll
        for (int i = 0; i < 4; ++i) Elem<T>::store(dst, i, silu(g[i] * inv) * (u[i] * inv));
      }
    }
    return;
  }

  // argmax: reduce the four waves' partial sums in LDS (fixed order: wave 0..3)
  __shared__ f32x4 red[3][MT][NT][64];
  if (wid > 0) {
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int j = 0; j < NT; ++j) red[wid - 1][m][j][lane] = acc[m][j];
  }
  __syncthreads();
  if (wid != 0) return;
#pragma unroll
  for (int w = 0; w < 3; ++w)
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int j = 0; j < NT; ++j) acc[m][j] += red[w][m][j][lane];

  {
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      int row = m * 16 + (lane & 15);
      float bv = -INFINITY;
      int bi = 0x7FFFFFFF;
      int nan = 0;
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        if (!tv[j]) continue;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = acc[m][j][i];
          int idx = (int)(tile[j] * 16 + 4 * q + i);
          if (v != v) {
            nan = 1;
            continue;
          }
          if (v > bv || (v == bv && idx < bi)) {
            bv = v;
            bi = idx;
          }
        }
      }
      if (a.logits && row < a.M) {
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          if (!tv[j]) continue;
          int64_t col = tile[j] * 16 + 4 * q;
          *(float4 *)(a.logits + (int64_t)row * a.ldlog + col) =
              make_float4(acc[m][j][0], acc[m][j][1], acc[m][j][2], acc[m][j][3]);
        }
      }
      // reduce over the four lane quarters that share this row
#pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        float ov = __shfl_xor(bv, o, 64);
        int oi = __shfl_xor(bi, o, 64);
        nan |= __shfl_xor(nan, o, 64);
        if (ov > bv || (ov == bv && oi < bi)) {
          bv = ov;
          bi = oi;
        }
      }
      if (q == 0 && row < a.M) {
        ArgmaxPart p;
        p.v = bv;
        p.idx = bi;
        p.nan = nan;
        p.pad = 0;
        a.amax[(int64_t)blockIdx.x * kRowPad + row] = p;
      }
    }
  }
}

int gemm_tiles_per_block(int epi, int mt) {
  (void)mt;
  return epi == EPI_ARGMAX ? 4 : 2;  // argmax; partial-sum projections counted at two
}

// W tiles per block of a partial-sum projection: four at three X tiles, and
// at two or more while the four-tile blocks (ntiles/4 x splits) still fill
// 7/8 of the CUs; two otherwise. Measured: 7B (224 tiles, 4 splits) at 17
// rows down 27.2 -> 23.9 us and O 9.0 -> 7.1 us with four; 3B (128 tiles)
// keeps two (four at 8 splits: down 11.2 -> 11.8 us).
int gemm_partial_tiles(int mt, int64_t ntiles, int splits, int cus) {
  if (mt == 3) return 4;
  const int64_t b4 = (ntiles + 3) / 4 * splits;
  return mt >= 2 && 8 * b4 >= 7 * (int64_t)cus ? 4 : 2;
}

// Gate/up pairs per block: the fewest of three or five whose blocks fit one
// per CU (five only up to three X tiles, whose epilogue then fills 120 KB of
// LDS), else three at three X tiles where those blocks fit two per CU (X reuse
// matters most there), else one: many small blocks fill the CUs evenly.
// Measured: 3B (688 gate tiles) three pairs, at 17 rows 19.4 -> 18.1 us and
// at 49 rows 25.0 -> 19.5 us against one; 7B (1184) five pairs (237 blocks),
// at 33 rows 52.4 us with three -> 49.3 us, at 17 rows 49.2 us with one ->
// 48.1 us.
int gemm_swiglu_pairs(int mt, int64_t gate_tiles, int cus) {
  const int64_t b3 = (gate_tiles + 2) / 3, b5 = (gate_tiles + 4) / 5;
  if (b3 <= cus) return 3;
  if (mt <= 3 && b5 <= cus) return 5;
  if (mt == 3 && b3 <= 2 * (int64_t)cus) return 3;
  return 1;
}

template <typename T, int EPI, int NP>
static hipError_t launch_t(int mt, const GemmArgs &a, dim3 grid, hipStream_t s) {
  // five gate/up pairs exist up to three X tiles only (LDS)
  constexpr bool wide = EPI == EPI_SWIGLU && NP == 5;
  switch (mt) {
    case 1: return launch_k(k_gemm<T, 1, EPI, NP>, grid, 256, s, a);
    case 2: return launch_k(k_gemm<T, 2, EPI, NP>, grid, 256, s, a);
    case 3: return launch_k(k_gemm<T, 3, EPI, NP>, grid, 256, s, a);
    case 4:
      if constexpr (!wide) return launch_k(k_gemm<T, 4, EPI, NP>, grid, 256, s, a);
      return hipErrorInvalidValue;
    case 5:
      if constexpr (!wide) return launch_k(k_gemm<T, 5, EPI, NP>, grid, 256, s, a);
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm(bool bf16, int epi, int mt, const GemmArgs &a, int cus, hipStream_t s) {
  if (epi == EPI_SWIGLU) {
    if (!a.rs.ssq || a.rs.nss < 1 || a.rs.nss > kMaxNormSlices || a.M < 1 || a.M > kRowPad)
      return hipErrorInvalidValue;
    const int np = gemm_swiglu_pairs(mt, a.up_tile_off, cus);
    const dim3 grid((unsigned)((a.up_tile_off + np - 1) / np), (unsigned)a.splits);
    if (np == 3) return bf16 ? launch_t<bf16_t, EPI_SWIGLU, 3>(mt, a, grid, s)
                             : launch_t<float, EPI_SWIGLU, 3>(mt, a, grid, s);
    if (np == 5) return bf16 ? launch_t<bf16_t, EPI_SWIGLU, 5>(mt, a, grid, s)
                             : launch_t<float, EPI_SWIGLU, 5>(mt, a, grid, s);
    return bf16 ? launch_t<bf16_t, EPI_SWIGLU, 1>(mt, a, grid, s) : launch_t<float, EPI_SWIGLU, 1>(mt, a, grid, s);
  }
  if (epi == EPI_PARTIAL) {
    const int nt = gemm_partial_tiles(mt, a.NTtot, a.splits, cus);
    const dim3 grid((unsigned)((a.NTtot + nt - 1) / nt), (unsigned)a.splits);
    if (nt == 4) return bf16 ? launch_t<bf16_t, EPI_PARTIAL, 4>(mt, a, grid, s)
                             : launch_t<float, EPI_PARTIAL, 4>(mt, a, grid, s);
    return bf16 ? launch_t<bf16_t, EPI_PARTIAL, 2>(mt, a, grid, s) : launch_t<float, EPI_PARTIAL, 2>(mt, a, grid, s);
  }
  const int tpb = gemm_tiles_per_block(epi, mt);
  const dim3 grid((unsigned)((a.NTtot + tpb - 1) / tpb), (unsigned)a.splits);
  return bf16 ? launch_t<bf16_t, EPI_ARGMAX, 0>(mt, a, grid, s) : launch_t<float, EPI_ARGMAX, 0>(mt, a, grid, s);
}

}  // namespace pf
