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
      const T *x = (const T *)&lo, *y = (const T *)&hi;
      uint4 olo, ohi;
      T *ox = (T *)&olo, *oy = (T *)&ohi;
#pragma unroll
      for (int e = 0; e < VE; ++e) {
        const int i = grp * VE + e;
        const float xv = Elem<T>::load(x, e), yv = Elem<T>::load(y, e);
        Elem<T>::store(ox, e, xv * cs[i] - yv * sn[i]);
        Elem<T>::store(oy, e, xv * sn[i] + yv * cs[i]);
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
    const uint32_t wv[8] = {A.x, A.y, A.z, A.w, B.x, B.y, B.z, B.w};
    uint32_t o[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      uint32_t lo = 0, hi = 0;
      switch (q) {  // uniform over the launch
        case 0: lo = wv[k]; hi = wv[k + 1]; break;
        case 1: lo = wv[k + 1]; hi = wv[k + 2]; break;
        case 2: lo = wv[k + 2]; hi = wv[k + 3]; break;
        default: lo = wv[k + 3]; hi = wv[k + 4]; break;
      }
      o[k] = bsh ? __builtin_amdgcn_alignbyte(hi, lo, bsh) : lo;
    }
    T *drow = vp + (int64_t)i * a.cap;
    if (d0 >= a.dst && d0 + VE <= a.dst + a.n) {
      *(uint4 *)(drow + d0) = make_uint4(o[0], o[1], o[2], o[3]);
    } else {
      const T *ov = (const T *)o;
#pragma unroll
      for (int e = 0; e < VE; ++e)
        if (d0 + e >= a.dst && d0 + e < a.dst + a.n) drow[d0 + e] = ov[e];
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
