// Rolling-image KV-state carryover (Section 3.4): move one span of cached
// tokens to new slots, re-rotating the keys from position m to m' and
// copying the values. A launch handles a span whose source and destination
// slots do not overlap; the host splits overlapping spans.
//
// Grid: x over the span's work, y over the (layer, KV head) planes, z = 0
// keys, 1 values. Keys: whole rows move, 16-byte accesses on both sides.
// Values (stored [head_dim][slot]): every 16-byte destination chunk is
// assembled from the two aligned source chunks around it with a byte funnel
// shift (the shift is the same for the whole launch), so both sides use
// aligned 16-byte accesses whatever the distance; chunks at the span's ends
// store only their elements inside it.
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
  __device__ static void put_raw(float *p, const uint32_t (&o)[4], int e) { p[0] = __uint_as_float(o[e]); }
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
  __device__ static void put_raw(bf16_t *p, const uint32_t (&o)[4], int e) {
    p[0].bits = (uint16_t)(o[e >> 1] >> (16 * (e & 1)));
  }
};

template <typename T>
__global__ __launch_bounds__(256) void k_kv_carry(CarryArgs a) {
  constexpr int VE = 16 / (int)sizeof(T);  // elements per 16-byte access
  constexpr int ESZ = (int)sizeof(T);
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
  // values
  T *vp = cache + ((int64_t)(l * 2 + 1) * a.nkv + g) * plane;
  const rsrc_t vr = make_rsrc(vp, (uint32_t)(plane * ESZ));
  const int64_t c0 = a.dst / VE, c1 = (a.dst + a.n + VE - 1) / VE;  // destination chunks
  const int nch = (int)(c1 - c0);
  // source element of a chunk's first element sits r elements past an
  // aligned chunk boundary; r is the same for every chunk
  const int r = (int)(((-a.delta) % VE + VE) % VE);
  const int sb = r * ESZ, q = sb >> 2, bsh = sb & 3;  // byte shift, as dwords + bytes
  const int items = a.hd * nch;
  for (int w = blockIdx.x * blockDim.x + threadIdx.x; w < items; w += gridDim.x * blockDim.x) {
    const int i = w / nch;
    const int64_t d0 = (c0 + w % nch) * VE;  // destination slot of the chunk
    const int64_t a0 = d0 - a.delta - r;      // aligned source slot below it
    const int64_t off = (int64_t)i * a.cap + a0;
    const uint4 A = bload16(vr, off >= 0 ? (uint32_t)(off * ESZ) : kOOB);
    const uint4 B = bload16(vr, off + VE >= 0 ? (uint32_t)((off + VE) * ESZ) : kOOB);
    // source words q .. q + 4 of the two chunks, as named registers (an
    // array indexed by q would be placed in scratch memory)
    uint32_t w0, w1, w2, w3, w4;
    switch (q) {  // uniform over the launch
      case 0: w0 = A.x; w1 = A.y; w2 = A.z; w3 = A.w; w4 = B.x; break;
      case 1: w0 = A.y; w1 = A.z; w2 = A.w; w3 = B.x; w4 = B.y; break;
      case 2: w0 = A.z; w1 = A.w; w2 = B.x; w3 = B.y; w4 = B.z; break;
      default: w0 = A.w; w1 = B.x; w2 = B.y; w3 = B.z; w4 = B.w; break;
    }
    uint32_t o[4];
    o[0] = bsh ? __builtin_amdgcn_alignbyte(w1, w0, bsh) : w0;
    o[1] = bsh ? __builtin_amdgcn_alignbyte(w2, w1, bsh) : w1;
    o[2] = bsh ? __builtin_amdgcn_alignbyte(w3, w2, bsh) : w2;
    o[3] = bsh ? __builtin_amdgcn_alignbyte(w4, w3, bsh) : w3;
    T *drow = vp + (int64_t)i * a.cap;
    if (d0 >= a.dst && d0 + VE <= a.dst + a.n) {
      *(uint4 *)(drow + d0) = make_uint4(o[0], o[1], o[2], o[3]);
    } else {
#pragma unroll
      for (int e = 0; e < VE; ++e)
        if (d0 + e >= a.dst && d0 + e < a.dst + a.n) Chunk<T>::put_raw(drow + d0 + e, o, e);
    }
  }
}

}  // namespace

hipError_t launch_kv_carry(bool bf16, const CarryArgs &a, hipStream_t s) {
  const int ve = bf16 ? 8 : 4;
  const int64_t plane_bytes = a.cap * a.hd * (bf16 ? 2 : 4);
  if (a.hd % (2 * ve) != 0 || a.hd / 2 > kCarryMaxHalf || a.n < 1 || a.cap % ve != 0 ||
      plane_bytes >= ((int64_t)1 << 31))
    return hipErrorInvalidValue;
  const int64_t k_items = (int64_t)a.n * (a.hd / 2 / ve);
  const int64_t v_items = (int64_t)a.hd * (a.n / ve + 2);
  const int64_t bx = std::min<int64_t>((std::max(k_items, v_items) + 255) / 256, 1024);
  const dim3 grid((unsigned)bx, (unsigned)(a.L * a.nkv), 2);
  if (bf16)
    PF_TRY(launch_k(k_kv_carry<bf16_t>, grid, 256, s, a));
  else
    PF_TRY(launch_k(k_kv_carry<float>, grid, 256, s, a));
  return hipGetLastError();
}

}  // namespace pf
