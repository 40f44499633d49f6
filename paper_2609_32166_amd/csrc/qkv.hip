// QKV projection of the verify step with its epilogue in the same kernel:
// the sums for a pair of 16-column tiles half a head apart are reduced
// inside the block (its waves split K, added in a fixed order), rotated
// (RoPE pairs dimension d with d + head_dim/2), and written where the next
// kernels read them: queries row-major for the attention, keys and values
// into the cache at slot P + row. No split-K partials and no separate
// epilogue kernel.
#include "kernels.h"

namespace pf {

namespace {

// Eight waves per block for every row count: the K split, and so the order
// of the sums, must not depend on the rows (a verify row reproduces the
// single-row step bit for bit). Sixteen measured slower (3B 9.8 vs 7.7 us).
// Fragment loads in flight per wave: eight up to two row tiles (a 3B wave's
// whole range at once: 6.85 -> 6.33 us), six beyond (registers). The slot
// count does not change the order in which a wave adds its fragments.
constexpr int kQkvWaves = 8;
template <int MT> constexpr int qkv_slots() { return MT <= 2 ? 8 : 6; }

template <typename T, int MT>
__global__ __launch_bounds__(64 * kQkvWaves) void k_gemm_qkv(QkvArgs a) {
  constexpr int NW = kQkvWaves;
  constexpr int kU = qkv_slots<MT>();  // fragment slots in flight per wave
  constexpr int E = Elem<T>::E;
  const int lane = threadIdx.x & 63;
  const int wid = threadIdx.x >> 6;
  const int half_tiles = a.hd / 32;  // 16-column tiles per rotation half
  const int hh = blockIdx.x / half_tiles, jt = blockIdx.x % half_tiles;
  const int64_t tA = (int64_t)hh * (a.hd / 16) + jt, tB = tA + half_tiles;

  // this wave's k fragments (the whole K is split over the block's waves)
  const int64_t f0 = wid * a.KFr / NW, f1 = (wid + 1) * a.KFr / NW;
  const int64_t n = f1 - f0;
  const rsrc_t wr = make_rsrc(a.W, (uint32_t)a.W_bytes);
  const rsrc_t xr = make_rsrc(a.X, (uint32_t)(kRowPad * a.ldx * sizeof(T)));
  const uint32_t wbase[2] = {(uint32_t)(((tA * a.KFr + f0) * 64 + lane) * 16),
                             (uint32_t)(((tB * a.KFr + f0) * 64 + lane) * 16)};
  uint32_t xbase[MT];
  const int64_t xkfr = a.ldx / (4 * E);
#pragma unroll
  for (int m = 0; m < MT; ++m)
    xbase[m] = m * 16 + (lane & 15) < a.M ? (uint32_t)(((m * xkfr + f0) * 64 + lane) * 16) : kOOB;

  // Epilogue: thread t < 256 owns one (row, RoPE pair) of each row tile;
  // queries, keys and values all run along the dimension (row-major
  // stores). Its cache length and RoPE factors are read before the products,
  // so their latency hides behind the loop.
  const int half = a.hd / 2;
  const int kind = hh < a.nq ? 0 : (hh < a.nq + a.nkv ? 1 : 2);  // query, key, value head
  const int et = threadIdx.x;
  const int er = (et >> 4) & 15;  // row within the tile
  const int ec = et & 15;         // column within the tile
  const int ed = jt * 16 + ec;                             // dimension in the first half
  int P = 0;
  float rc[MT], rs[MT];
  if (et < 256) {
    P = *a.kv_len;
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const int row = min(m * 16 + er, a.M - 1);
      rc[m] = kind == 2 ? 1.f : a.rope[((int64_t)row * half + ed) * 2 + 0];
      rs[m] = kind == 2 ? 0.f : a.rope[((int64_t)row * half + ed) * 2 + 1];
    }
  }

  f32x4 acc[MT][2];
#pragma unroll
  for (int m = 0; m < MT; ++m) acc[m][0] = acc[m][1] = f32x4{0.f, 0.f, 0.f, 0.f};
  uint4 wv[kU][2], xv[kU][MT];
  auto load = [&](int u, int64_t i) {
    const bool in = i < n;
#pragma unroll
    for (int t = 0; t < 2; ++t)
      wv[u][t] = bload16_stream(wr, in ? wbase[t] + (uint32_t)(i * 1024) : kOOB);
#pragma unroll
    for (int m = 0; m < MT; ++m)
      xv[u][m] = bload16(xr, in && xbase[m] != kOOB ? xbase[m] + (uint32_t)(i * 1024) : kOOB);
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
        for (int t = 0; t < 2; ++t) acc[m][t] = mma<T>(wv[u][t], xv[u][m], acc[m][t]);
      load(u, i + kU + u);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // fixed-order reduction over the waves, one row tile at a time: every wave
  // writes its sums, then each epilogue thread adds its output's eight wave
  // sums in wave order, rotates the pair and stores it
  __shared__ f32x4 red[NW][2][64];
  const int64_t plane = a.cap * a.hd;
  // lane of the MFMA output holding (row er, column ec), and its element
  const int src_lane = er + 16 * (ec >> 2), src_i = ec & 3;
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    red[wid][0][lane] = acc[m][0];
    red[wid][1][lane] = acc[m][1];
    __syncthreads();
    const int row = m * 16 + er;
    if (et < 256 && row < a.M) {
      float x = red[0][0][src_lane][src_i], y = red[0][1][src_lane][src_i];
#pragma unroll
      for (int w = 1; w < NW; ++w) {
        x += red[w][0][src_lane][src_i];
        y += red[w][1][src_lane][src_i];
      }
      const int64_t slot = P + row;
      if (kind == 2) {
        T *vp = (T *)a.cache + ((int64_t)(a.layer * 2 + 1) * a.nkv + (hh - a.nq - a.nkv)) * plane +
                slot * a.hd;
        Elem<T>::store(vp, ed, x);
        Elem<T>::store(vp, ed + half, y);
      } else {
        const float c = rc[m], sn = rs[m];
        // explicit FMAs: every row-count instantiation rounds the rotation the
        // same way (left to contraction, two instantiations may differ)
        const float rx = fmaf(x, c, -(y * sn)), ry = fmaf(x, sn, y * c);
        T *dst = kind == 0 ? (T *)a.qbuf + (int64_t)row * a.ldq + (int64_t)hh * a.hd
                           : (T *)a.cache + ((int64_t)(a.layer * 2 + 0) * a.nkv + (hh - a.nq)) * plane +
                                 slot * a.hd;
        Elem<T>::store(dst, ed, rx);
        Elem<T>::store(dst, ed + half, ry);
      }
    }
    __syncthreads();
  }
}

template <typename T>
hipError_t launch_t(int mt, const QkvArgs &a, hipStream_t s) {
  const unsigned blocks = (unsigned)((a.nq + 2 * a.nkv) * (a.hd / 32));
  switch (mt) {
    case 1: return launch_k(k_gemm_qkv<T, 1>, blocks, 64 * kQkvWaves, s, a);
    case 2: return launch_k(k_gemm_qkv<T, 2>, blocks, 64 * kQkvWaves, s, a);
    case 3: return launch_k(k_gemm_qkv<T, 3>, blocks, 64 * kQkvWaves, s, a);
    case 4: return launch_k(k_gemm_qkv<T, 4>, blocks, 64 * kQkvWaves, s, a);
    case 5: return launch_k(k_gemm_qkv<T, 5>, blocks, 64 * kQkvWaves, s, a);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_gemm_qkv(bool bf16, int mt, const QkvArgs &a, hipStream_t s) {
  if (a.hd % 32 != 0) return hipErrorInvalidValue;
  PF_TRY(bf16 ? launch_t<bf16_t>(mt, a, s) : launch_t<float>(mt, a, s));
  return hipGetLastError();
}

}  // namespace pf
