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
#include <type_traits>

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

// ---------------------------------------------------------------------------
// SwiGLU projection of a whole chunk, act = silu(X Wg^T) * (X Wu^T), as one
// pass over the chunk's rows: a block owns NJ gate tiles of 16 columns for up
// to 512 rows of X, so the 7B-class FFN (1184 gate tiles) takes 237 blocks,
// one per CU, in a single round. The block's W rows form NJ 32-row A tiles,
// each the 16 gate rows over the 16 up rows of the same columns, so a lane's
// gate and up sums of one output sit in the same accumulator (values v and
// v + 8). Each of the 8 waves owns 64 rows of X (two 32-row B tiles): 16 NJ
// accumulator tiles of 32x32 per block, 10 per wave.
//
// W is read by all eight waves: it goes from HBM straight into LDS (16-byte
// load-to-LDS instructions, no registers), 64 k a stage, three stage buffers
// with the loads two stages ahead; the packed fragments are copied as they
// are, so a 16-lane group's operand read is 256 contiguous bytes. X is read by
// one wave only: it comes straight from the 32-row packed layout into the B
// operands, one 1 KiB load per tile and 16-k step, six steps in flight.
//
// Loads complete in issue order as far as the wait counter is concerned, so
// waiting for an X load also waits for every W load issued before it: the W
// loads of a stage go out right after the first X refill of the stage two
// before, which gives them seven steps. Every stage issues the same loads
// (zero-fill offsets past the matrix), so one wait count before each barrier
// is exact, and the barrier is a bare s_barrier: a block-wide fence would
// wait for every load in flight, the X ring included.
// ---------------------------------------------------------------------------

// s_waitcnt immediate (gfx9 encoding) that waits until at most n vector
// memory loads are outstanding and leaves the other counters alone
constexpr int vmcnt_imm(int n) { return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14); }

// A-operand reads of the SwiGLU kernel, issued as plain LDS reads the
// compiler does not track: it cannot always prove that a read of the current
// stage misses the buffer the load-to-LDS instructions are filling, and then
// waits for every load in flight before the read. lds_wait<N> waits until at
// most N LDS operations are outstanding (they complete in order; anything
// else outstanding only makes the wait stricter) and passes the operand
// through, so the products that use it cannot move above the wait.
// (These and the load-to-LDS builtin below are compiled in the device pass
// only: in the host pass they keep the kernel's launch stub from being
// emitted, without an error.)
typedef unsigned v4u __attribute__((ext_vector_type(4)));
template <int OFF> __device__ inline v4u lds_read16(uint32_t addr) {
  v4u r = {0u, 0u, 0u, 0u};
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF) : "memory");
#endif
  return r;
}
template <int N> __device__ inline void lds_wait(v4u &r) {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(r) : "i"(N) : "memory");
#endif
}
// 16-byte load from a buffer resource straight into LDS: the wave's 64 lanes
// write their 16 bytes contiguously from the wave-uniform address `lds`; an
// offset past the resource writes zeros and fetches nothing
__device__ inline void bload16_lds(rsrc_t r, void *lds, uint32_t off) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void *)lds, 16, off,
                                           0, 0, kPolicyNT);
#endif
}
__device__ inline uint32_t lds_addr(const void *p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)p;
}
__device__ inline f32x16 mma32v(v4u a, const uint4 &b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
template <int I, int N, typename F> __device__ inline void static_for(F &&f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

template <int NJ>
__global__ __launch_bounds__(512, 1) void k_gemm_ffn(BigGemmArgs a) {
  constexpr int D = 6;                       // X ring: 16-k steps in flight
  constexpr int WPT = (NJ * 256 + 511) / 512;  // 16-byte W chunks per thread and stage
  constexpr int WSTAGE = WPT * 512;          // chunks a stage buffer holds
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int r32 = lane & 31, hi = lane >> 5;
  const int64_t gate_tiles = a.up_tile_off;
  const int64_t g0 = (int64_t)blockIdx.x * NJ;
  const int64_t xrow0 = (int64_t)blockIdx.y * 512 + wid * 64;
  const bool active = xrow0 < a.x_rows;  // wave-uniform
  const int64_t KFr = a.KFr, ksteps = 2 * KFr, nst = (KFr + 1) / 2;
  const rsrc_t wr = make_rsrc(a.W, (uint32_t)a.W_bytes);
  const rsrc_t xr = make_rsrc(a.X, (uint32_t)(a.x_rows * a.ldx * 2));

  // stage chunk c: A tile c >> 8, gate (0) or up (1) half (c >> 7) & 1, byte
  // (c & 127) * 16 of the two fragments' 2 KiB. Chunks past NJ * 256 (the
  // stage is padded to whole rounds of 512) and tiles past the FFN load
  // zeros, so every thread issues the same loads.
  __shared__ uint4 lw0[WSTAGE], lw1[WSTAGE], lw2[WSTAGE];
  uint32_t woff[WPT];
  bool wval[WPT];
#pragma unroll
  for (int i = 0; i < WPT; ++i) {
    const int c = tid + 512 * i;
    const int64_t g = g0 + (c >> 8);
    wval[i] = c < NJ * 256 && g < gate_tiles;
    const int64_t t = g + (((c >> 7) & 1) ? gate_tiles : 0);
    woff[i] = wval[i] ? (uint32_t)(t * KFr * 1024 + (c & 127) * 16) : 0u;
  }
  // a wave's load-to-LDS writes its 64 lanes' 16 bytes contiguously from
  // the wave-uniform address it is given
  auto wload = [&](uint4 *buf, int64_t st) {
#pragma unroll
    for (int i = 0; i < WPT; ++i) {
      const int c = tid + 512 * i;
      // stages past the end, and the second fragment of an odd last stage
      const bool in = wval[i] && st < nst && 2 * st + ((c & 127) >> 6) < KFr;
      bload16_lds(wr, buf + 512 * i + 64 * wid, in ? woff[i] + (uint32_t)(st * 2048) : kOOB);
    }
  };

  // B operand of 16-k step i, tile u: lane's 16 bytes of the 1 KiB chunk
  const int64_t ldk = a.ldx >> 4;
  const uint32_t xbase = (uint32_t)((xrow0 >> 5) * ldk * 1024 + lane * 16);
  uint4 xq[D][2];
  auto xload = [&](int slot, int64_t i) {
    const bool in = active && i < ksteps;
#pragma unroll
    for (int u = 0; u < 2; ++u)
      xq[slot][u] = bload16(xr, in ? xbase + (uint32_t)((u * ldk + i) * 1024) : kOOB);
  };
  // A operand of step s of a stage, tile j: row r32 (gate rows 0-15, up rows
  // 16-31), k = 16 (s % 2) + 8 hi .. + 8 of fragment s / 2; byte address
  // lane part + j * 4096 + (s / 2) * 1024 + (s % 2) * 512 of the stage buffer
  const uint32_t alane = (uint32_t)((r32 >> 4) * 2048 + hi * 256 + (r32 & 15) * 16);

  f32x16 acc[NJ][2];
#pragma unroll
  for (int j = 0; j < NJ; ++j)
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[j][u][v] = 0.f;

  // loads issued after the W loads of stage st + 1 by the end of stage st:
  // the last three X refills of stage st - 1, the first X refill and the W
  // loads of stage st, its last three X refills (the prologue issues more
  // after stage 1's, so the same count waits a little early there)
  constexpr int kAfterW = 2 * 3 + 2 + WPT + 2 * 3;
  wload(lw0, 0);
  wload(lw1, 1);
#pragma unroll
  for (int i = 0; i < D; ++i) xload(i, i);
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(WPT + 2 * D));
  __builtin_amdgcn_s_barrier();

  // stage st reads buffer st % 3; within a run of three stages starting at a
  // multiple of three, its X slots are (4 u + s) % D
  auto run = [&](auto uc, const uint4 *cur, uint4 *ahead, int64_t st) {
    constexpr int u = decltype(uc)::value;
    const uint32_t abase = lds_addr(cur) + alane;
    static_for<0, 4>([&](auto sc) {
      constexpr int s = decltype(sc)::value;
      constexpr int slot = (4 * u + s) % D;
      if (active) {
        v4u af[NJ];
        static_for<0, NJ>([&](auto jc) {
          constexpr int j = decltype(jc)::value;
          af[j] = lds_read16<j * 4096 + (s >> 1) * 1024 + (s & 1) * 512>(abase);
        });
        static_for<0, NJ>([&](auto jc) {
          constexpr int j = decltype(jc)::value;
          lds_wait<NJ - 1 - j>(af[j]);
#pragma unroll
          for (int t = 0; t < 2; ++t) acc[j][t] = mma32v(af[j], xq[slot][t], acc[j][t]);
          // each operand's products right behind its own wait
          __builtin_amdgcn_sched_barrier(0);
        });
      }
      xload(slot, st * 4 + s + D);
      if (s == 0) wload(ahead, st + 2);
    });
    // stage st + 1's W is in LDS for every wave; this stage's reads are done
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(kAfterW));
    __builtin_amdgcn_s_barrier();
  };
  auto stage = [&](auto uc, int64_t st) {
    constexpr int u = decltype(uc)::value;
    run(uc, u == 0 ? lw0 : u == 1 ? lw1 : lw2, u == 0 ? lw2 : u == 1 ? lw0 : lw1, st);
  };
  int64_t st = 0;
  for (; st + 3 <= nst; st += 3) {
    stage(std::integral_constant<int, 0>{}, st);
    stage(std::integral_constant<int, 1>{}, st + 1);
    stage(std::integral_constant<int, 2>{}, st + 2);
  }
  if (st < nst) stage(std::integral_constant<int, 0>{}, st);
  if (st + 1 < nst) stage(std::integral_constant<int, 1>{}, st + 1);
  if (!active) return;

  // lane holds D[n = 8 (v / 4) + 4 hi + v % 4][row r32 of its B tile]: gate
  // column n for v < 8, its up partner at v + 8
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int64_t g = g0 + j;
    if (g >= gate_tiles) continue;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int64_t row = xrow0 + 32 * u + r32;
      if (row >= a.M) continue;
      bf16_t *dst = (bf16_t *)a.act + row * a.ldact + g * 16 + 4 * hi;
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        uint2 pk;
        uint32_t h[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          h[e] = f32_to_bf16(silu_f(acc[j][u][4 * q + e]) * acc[j][u][8 + 4 * q + e]);
        pk.x = h[0] | (h[1] << 16);
        pk.y = h[2] | (h[3] << 16);
        *(uint2 *)(dst + 8 * q) = pk;
      }
    }
  }
}

}  // namespace

hipError_t launch_gemm_ffn(const BigGemmArgs &a, hipStream_t s) {
  constexpr int NJ = 5;
  if (a.x_rows % 32 != 0 || a.ldx % 32 != 0 || a.ldx < 32 * a.KFr || a.ldact % 4 != 0 ||
      a.W_bytes >= ((int64_t)1 << 31) || a.x_rows * a.ldx * 2 >= ((int64_t)1 << 31) ||
      a.up_tile_off < 1 || a.M > a.x_rows)
    return hipErrorInvalidValue;
  const dim3 grid((unsigned)((a.up_tile_off + NJ - 1) / NJ), (unsigned)((a.x_rows + 511) / 512));
  PF_TRY(launch_k(k_gemm_ffn<NJ>, grid, 512, s, a));
  return hipGetLastError();
}

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
