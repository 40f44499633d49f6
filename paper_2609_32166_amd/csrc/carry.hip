// Rolling-image KV-state carryover (Section 3.4): move one span of cached
// tokens to new slots, re-rotating the keys from position m to m' and
// copying the values. A launch handles a span whose source and destination
// slots do not overlap; the host splits overlapping spans.
//
// Grid: x over the span's work, y over the (layer, KV head) planes, z = 0
// keys, 1 values. Keys and values are both [slot][head_dim] rows: whole rows
// move with 16-byte accesses on both sides, the keys rotated on the way.
#include <algorithm>

#include "kernels.h"

namespace pf {

namespace {

// Element e of a 16-byte chunk held in registers, read and written with
// shifts and selects (indexing the chunk through a pointer would put it in
// scratch memory). e is a compile-time constant after unrolling.
__device__ inline uint32_t chunk_word(const uint4 &v, int w) {
  return w == 0 ? v.x : w == 1 ? v.y : w == 2 ? v.z : v.w;
}
__device__ inline void chunk_put_word(uint4 &v, int w, uint32_t x) {
  if (w == 0) v.x = x;
  else if (w == 1) v.y = x;
  else if (w == 2) v.z = x;
  else v.w = x;
}
template <typename T> struct Chunk;
template <> struct Chunk<float> {
  __device__ static float get(const uint4 &v, int e) { return __uint_as_float(chunk_word(v, e)); }
  __device__ static void set(uint4 &v, int e, float f) { chunk_put_word(v, e, __float_as_uint(f)); }
};
template <> struct Chunk<bf16_t> {
  __device__ static float get(const uint4 &v, int e) {
    return bf16_to_f32((uint16_t)(chunk_word(v, e >> 1) >> (16 * (e & 1))));
  }
  __device__ static void set(uint4 &v, int e, float f) {
    const int sh = 16 * (e & 1);
    const uint32_t w = chunk_word(v, e >> 1);
    chunk_put_word(v, e >> 1, (w & ~(0xFFFFu << sh)) | ((uint32_t)f32_to_bf16(f) << sh));
  }
};

template <typename T>
__global__ __launch_bounds__(256) void k_kv_carry(CarryArgs a) {
  constexpr int VE = 16 / (int)sizeof(T);  // elements per 16-byte access
  const int l = blockIdx.y / a.nkv, g = blockIdx.y % a.nkv;
  const int64_t plane = a.cap * a.hd;
  T *cache = (T *)a.cache;
  if (blockIdx.z == 0) {
    // keys: rotation by delta * theta_i (R(m') R(m)^-1 with m' - m = delta);
    // angles in fp64, as the verify step forms them
    const int h = a.hd / 2;
    __shared__ float cs[kCarryMaxHalf], sn[kCarryMaxHalf];
    for (int i = threadIdx.x; i < h; i += blockDim.x) {
      const double ang = (double)a.delta * a.inv_freq[i];
      cs[i] = (float)cos(ang);
      sn[i] = (float)sin(ang);
    }
    __syncthreads();
    T *kp = cache + ((int64_t)(l * 2 + 0) * a.nkv + g) * plane;
    const int gk = h / VE;  // 16-byte groups of the first half of a row
    const int items = a.n * gk;
    for (int w = blockIdx.x * blockDim.x + threadIdx.x; w < items; w += gridDim.x * blockDim.x) {
      const int tok = w / gk, grp = w % gk;
      const T *s = kp + (a.src + tok) * a.hd + grp * VE;
      T *d = kp + (a.dst + tok) * a.hd + grp * VE;
      const uint4 lo = *(const uint4 *)s, hi = *(const uint4 *)(s + h);
      uint4 olo = lo, ohi = hi;
#pragma unroll
      for (int e = 0; e < VE; ++e) {
        const int i = grp * VE + e;
        const float xv = Chunk<T>::get(lo, e), yv = Chunk<T>::get(hi, e);
        Chunk<T>::set(olo, e, xv * cs[i] - yv * sn[i]);
        Chunk<T>::set(ohi, e, xv * sn[i] + yv * cs[i]);
      }
      *(uint4 *)d = olo;
      *(uint4 *)(d + h) = ohi;
    }
    return;
  }
  // values: rows copied unchanged
  const T *vs = cache + ((int64_t)(l * 2 + 1) * a.nkv + g) * plane;
  T *vd = cache + ((int64_t)(l * 2 + 1) * a.nkv + g) * plane;
  const int gv = a.hd / VE;  // 16-byte groups of a row
  const int items = a.n * gv;
  for (int w = blockIdx.x * blockDim.x + threadIdx.x; w < items; w += gridDim.x * blockDim.x) {
    const int tok = w / gv, grp = w % gv;
    *(uint4 *)(vd + (a.dst + tok) * a.hd + grp * VE) =
        *(const uint4 *)(vs + (a.src + tok) * a.hd + grp * VE);
  }
}

}  // namespace

hipError_t launch_kv_carry(bool bf16, const CarryArgs &a, hipStream_t s) {
  const int ve = bf16 ? 8 : 4;
  const int64_t plane_bytes = a.cap * a.hd * (bf16 ? 2 : 4);
  if (a.hd % (2 * ve) != 0 || a.hd / 2 > kCarryMaxHalf || a.n < 1 ||
      plane_bytes >= ((int64_t)1 << 31))
    return hipErrorInvalidValue;
  const int64_t k_items = (int64_t)a.n * (a.hd / 2 / ve);
  const int64_t v_items = (int64_t)a.n * (a.hd / ve);
  const int64_t bx = std::min<int64_t>((std::max(k_items, v_items) + 255) / 256, 1024);
  const dim3 grid((unsigned)bx, (unsigned)(a.L * a.nkv), 2);
  if (bf16)
    PF_TRY(launch_k(k_kv_carry<bf16_t>, grid, 256, s, a));
  else
    PF_TRY(launch_k(k_kv_carry<float>, grid, 256, s, a));
  return hipGetLastError();
}

}  // namespace pf
