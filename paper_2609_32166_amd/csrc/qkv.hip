// QKV projection of the verify step with its epilogue in the same kernel.
// The fused weight is packed RoPE-paired (a 16-row tile of a head holds
// dimensions 8t..8t+7 and their partners half a head on), so every output
// tile can be rotated on its own. A block takes one or two consecutive tiles
// of a head; its waves split K and their sums are reduced inside the block in
// a fixed order, rotated (RoPE pairs dimension d with d + head_dim/2), and
// written where the next kernels read them: queries row-major for the
// attention, keys and values into the cache at slot P + row. No split-K
// partials and no separate epilogue kernel.
#include "kernels.h"

namespace pf {

namespace {

// Tiles per block and waves per block are chosen by the model's shape only,
// never by the row count: the K split, and so the order of the sums, must
// not depend on the rows (a verify row reproduces the single-row step bit for
// bit). Fragment loads in flight per wave: eight, six with two tiles and
// three or more row tiles (registers). The slot count does not change the
// order in which a wave adds its fragments.
template <int MT, int NTL> constexpr int qkv_slots() { return NTL == 1 || MT <= 2 ? 8 : 6; }

template <typename T, int MT, int NTL, int NW>
__global__ __launch_bounds__(64 * NW) void k_gemm_qkv(QkvArgs a) {
  constexpr int kU = qkv_slots<MT, NTL>();  // fragment slots in flight per wave
  constexpr int E = Elem<T>::E;
  const int lane = threadIdx.x & 63;
  const int wid = threadIdx.x >> 6;
  const int th = a.hd / 16;                        // tiles per head
  const int hh = blockIdx.x / (th / NTL);          // head (queries, then keys, then values)
  const int jt0 = (blockIdx.x % (th / NTL)) * NTL;  // first tile of the block within the head
  const int64_t t0 = (int64_t)hh * th + jt0;

  // this wave's k fragments (the whole K is split over the block's waves)
  const int64_t f0 = wid * a.KFr / NW, f1 = (wid + 1) * a.KFr / NW;
  const int64_t n = f1 - f0;
  const rsrc_t wr = make_rsrc(a.W, (uint32_t)a.W_bytes);
  const rsrc_t xr = make_rsrc(a.X, (uint32_t)(kRowPad * a.ldx * sizeof(T)));
  uint32_t wbase[NTL];
#pragma unroll
  for (int i = 0; i < NTL; ++i) wbase[i] = (uint32_t)((((t0 + i) * a.KFr + f0) * 64 + lane) * 16);
  uint32_t xbase[MT];
  const int64_t xkfr = a.ldx / (4 * E);
#pragma unroll
  for (int m = 0; m < MT; ++m)
    xbase[m] = m * 16 + (lane & 15) < a.M ? (uint32_t)(((m * xkfr + f0) * 64 + lane) * 16) : kOOB;

  // Epilogue: thread t < 128 NTL owns RoPE pair p of row r of the block's
  // tile i (consecutive threads, consecutive dimensions). Its cache length and
  // RoPE factors are read before the products, so their latency hides behind
  // the loop.
  const int half = a.hd / 2;
  const int kind = hh < a.nq ? 0 : (hh < a.nq + a.nkv ? 1 : 2);  // query, key, value head
  const int et = threadIdx.x;
  const int ei = et >> 7, er = (et >> 3) & 15, ep = et & 7;
  const int ed = (jt0 + ei) * 8 + ep;  // dimension in the first half
  const bool eact = et < 128 * NTL;
  int P = 0;
  float rc[MT], rs[MT];
  if (eact) {
    P = *a.kv_len;
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const int row = min(m * 16 + er, a.M - 1);
      rc[m] = kind == 2 ? 1.f : a.rope[((int64_t)row * half + ed) * 2 + 0];
      rs[m] = kind == 2 ? 0.f : a.rope[((int64_t)row * half + ed) * 2 + 1];
    }
  }

  f32x4 acc[MT][NTL];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int i = 0; i < NTL; ++i) acc[m][i] = f32x4{0.f, 0.f, 0.f, 0.f};
  uint4 wv[kU][NTL], xv[kU][MT];
  auto load = [&](int u, int64_t i) {
    const bool in = i < n;
#pragma unroll
    for (int t = 0; t < NTL; ++t)
      wv[u][t] = bload16_stream(wr, in ? wbase[t] + (uint32_t)(i * 1024) : kOOB);
#pragma unroll
    for (int m = 0; m < MT; ++m)
      xv[u][m] = bload16(xr, in && xbase[m] != kOOB ? xbase[m] + (uint32_t)(i * 1024) : kOOB);
  };
  // the rows' deferred RMSNorm scales (see RowInv)
  __shared__ float invl[kRowPad];
  RowInv ri;
  ri.issue(a.rs, a.M);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    load(u, u);
    __builtin_amdgcn_sched_barrier(0);
  }
  ri.finish(a.rs, a.M, invl);
  __builtin_amdgcn_sched_barrier(0);
  for (int64_t i = 0; i < n; i += kU) {
#pragma unroll
    for (int u = 0; u < kU; ++u) {
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int t = 0; t < NTL; ++t) acc[m][t] = mma<T>(wv[u][t], xv[u][m], acc[m][t]);
      load(u, i + kU + u);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // fixed-order reduction over the waves, one row tile at a time: every wave
  // writes its sums, then each epilogue thread adds its pair's NW wave sums in
  // wave order, rotates the pair and stores it
  __shared__ f32x4 red[NW][NTL][64];
  const int64_t plane = a.cap * a.hd;
  // MFMA output lanes of (row er, column ep) and (row er, column ep + 8)
  const int xl = er + 16 * (ep >> 2), yl = er + 16 * (2 + (ep >> 2)), ec = ep & 3;
#pragma unroll
  for (int m = 0; m < MT; ++m) {
#pragma unroll
    for (int i = 0; i < NTL; ++i) red[wid][i][lane] = acc[m][i];
    __syncthreads();
    const int row = m * 16 + er;
    if (eact && row < a.M) {
      float x = red[0][ei][xl][ec], y = red[0][ei][yl][ec];
#pragma unroll
      for (int w = 1; w < NW; ++w) {
        x += red[w][ei][xl][ec];
        y += red[w][ei][yl][ec];
      }
      const float inv = invl[row];  // written before the loop, visible after the barrier
      x *= inv;
      y *= inv;
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

// Block shape per model: one tile and four waves while the tiles fit the
// compute units once (every compute unit streams its own weights); two tiles
// and eight waves beyond, where one tile per block would leave a second
// round of blocks.
template <typename T, int NTL, int NW>
hipError_t launch_mt(int mt, const QkvArgs &a, unsigned blocks, hipStream_t s) {
  switch (mt) {
    case 1: return launch_k(k_gemm_qkv<T, 1, NTL, NW>, blocks, 64 * NW, s, a);
    case 2: return launch_k(k_gemm_qkv<T, 2, NTL, NW>, blocks, 64 * NW, s, a);
    case 3: return launch_k(k_gemm_qkv<T, 3, NTL, NW>, blocks, 64 * NW, s, a);
    case 4: return launch_k(k_gemm_qkv<T, 4, NTL, NW>, blocks, 64 * NW, s, a);
    case 5: return launch_k(k_gemm_qkv<T, 5, NTL, NW>, blocks, 64 * NW, s, a);
    default: return hipErrorInvalidValue;
  }
}

template <typename T>
hipError_t launch_t(int mt, const QkvArgs &a, int cus, hipStream_t s) {
  const int tiles = (a.nq + 2 * a.nkv) * (a.hd / 16);
  if (tiles <= cus) return launch_mt<T, 1, 4>(mt, a, (unsigned)tiles, s);
  return launch_mt<T, 2, 8>(mt, a, (unsigned)(tiles / 2), s);
}

}  // namespace

hipError_t launch_gemm_qkv(bool bf16, int mt, const QkvArgs &a, int cus, hipStream_t s) {
  if (a.hd % 32 != 0 || !a.rs.ssq || a.rs.nss < 1 || a.rs.nss > kMaxNormSlices || a.M < 1 ||
      a.M > kRowPad)
    return hipErrorInvalidValue;
  PF_TRY(bf16 ? launch_t<bf16_t>(mt, a, cus, s) : launch_t<float>(mt, a, cus, s));
  return hipGetLastError();
}

}  // namespace pf
