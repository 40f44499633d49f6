// Internal definitions shared by the HIP kernels and the C-ABI layer of
// libpf. gfx950 (CDNA4) only: 64-wide wavefronts, MFMA 16x16 tiles.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "pf.h"

namespace pf {

// status helpers of the C ABI: fail() records the message returned by
// pf_last_error() and returns st; ok() clears it
pf_status fail(pf_status st, const char *fmt, ...);
pf_status ok();

// ---------------------------------------------------------------------------
// element types
// ---------------------------------------------------------------------------

struct bf16_t {
  uint16_t bits;
};

__host__ __device__ inline float bf16_to_f32(uint16_t h) {
  return __uint_as_float((uint32_t)h << 16);
}

// Round-to-nearest-even fp32 -> bf16 (NaN stays a quiet NaN).
__host__ __device__ inline uint16_t f32_to_bf16(float f) {
  uint32_t b = __float_as_uint(f);
  if ((b & 0x7F800000u) == 0x7F800000u && (b & 0x007FFFFFu)) return 0x7FC0;
  b += 0x7FFFu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
  static constexpr int E = 4;  // elements per 16-byte lane chunk
  __device__ static float load(const float *p, int64_t i) { return p[i]; }
  __device__ static float to_f32(float v) { return v; }
  __device__ static float round(float v) { return v; }  // fp32 models keep fp32
  __device__ static void store(float *p, int64_t i, float v) { p[i] = v; }
};
template <> struct Elem<bf16_t> {
  static constexpr int E = 8;
  __device__ static float load(const bf16_t *p, int64_t i) { return bf16_to_f32(p[i].bits); }
  __device__ static float round(float v) { return bf16_to_f32(f32_to_bf16(v)); }
  __device__ static void store(bf16_t *p, int64_t i, float v) { p[i].bits = f32_to_bf16(v); }
};

// k elements covered by one 16-byte-per-lane fragment of a wave (4 lane
// quarters x E elements).
template <typename T> constexpr int frag_k() { return 4 * Elem<T>::E; }

// Activation layout read by the skinny verify GEMM ("fragment-packed"): for
// every 16-row tile and every k fragment, the 64 lanes' E-element chunks are
// stored contiguously (lane = row % 16 + 16 * quarter), so one wave's operand
// fragment is a single coalesced 1 KiB load. `ld` is the padded row length, a
// multiple of 4E; the buffer size equals that of a row-major [rows][ld] array.
template <typename T> __device__ inline int64_t act_off(int row, int64_t k, int64_t ld) {
  constexpr int E = Elem<T>::E, KF = 4 * E;
  return (((int64_t)(row >> 4) * (ld / KF) + k / KF) * 64 + ((k % KF) / E) * 16 + (row & 15)) * E +
         k % E;
}

// bf16 activation layout read by the prefill SwiGLU GEMM ("32-row packed"):
// for every 32-row tile and every 16-k step, the 64 lanes' 8-element chunks of
// the 32x32x16 matrix instruction's B operand are stored contiguously (lane =
// row % 32 + 32 * (k / 8 % 2)), so a wave's operand is one 1 KiB load. `ld`
// is the padded row length (a multiple of 32); the size equals that of a
// row-major [rows][ld] array with rows a multiple of 32.
__host__ __device__ inline int64_t xb32_off(int row, int64_t k, int64_t ld) {
  return (((int64_t)(row >> 5) * (ld >> 4) + (k >> 4)) * 64 + ((k >> 3) & 1) * 32 + (row & 31)) * 8 +
         (k & 7);
}

// ---------------------------------------------------------------------------
// MFMA step: D(16x16) += A(16 x KF) * B(KF x 16) where every lane supplies
// one 16-byte chunk of A and of B. Lane l carries row l%16 of A and column
// l%16 of B; its chunk covers the k slots of lane quarter l/16. The output
// lane l holds D[4*(l/16)+i][l%16], i = 0..3. Any consistent assignment of
// k indices to (quarter, element) gives the same contraction.
// ---------------------------------------------------------------------------

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ inline f32x4 mma16(float, const uint4 &a, const uint4 &b, f32x4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
  return c;
}

__device__ inline f32x4 mma16(bf16_t, const uint4 &a, const uint4 &b, f32x4 c) {
  bf16x8 av = __builtin_bit_cast(bf16x8, a);
  bf16x8 bv = __builtin_bit_cast(bf16x8, b);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, c, 0, 0, 0);
}

template <typename T> __device__ inline f32x4 mma(const uint4 &a, const uint4 &b, f32x4 c) {
  return mma16(T{}, a, b, c);
}

// ---------------------------------------------------------------------------
// wave helpers
// ---------------------------------------------------------------------------

__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// ---------------------------------------------------------------------------
// packed weight layout for the skinny GEMM
//
// W [N][K] row-major is stored as fragments of 16 rows x KF columns; fragment
// (nt, kf) is 64 lanes x 16 bytes, contiguous, lane = (n % 16) + 16 * q where
// q = (k % KF) / E, element e = k % E. Rows >= N and columns >= K are zero.
// ---------------------------------------------------------------------------

struct Packed {
  void *data = nullptr;
  int64_t N = 0, K = 0;  // logical
  int64_t NT = 0;        // n-tiles of 16 rows
  int64_t KFr = 0;       // k fragments
  int64_t bytes() const { return NT * KFr * 1024; }
};

// Step work buffers sized for the largest verify (65 rows, padded to 80).
constexpr int kMaxRows = 65;
constexpr int kRowPad = 80;

struct ArgmaxPart {
  float v;
  int32_t idx;
  int32_t nan;
  int32_t pad;
};

}  // namespace pf

// internal model object
struct pf_model {
  pf_model_config cfg;
  int esz;  // bytes per element
  // packed weights, one Packed per layer for wqkv/wo/wgu/wd (contiguous arrays)
  void *wqkv = nullptr, *wo = nullptr, *wgu = nullptr, *wd = nullptr, *lm = nullptr;
  pf::Packed pqkv, po, pgu, pd, plm;  // per-layer geometry (data = first layer)
  void *embed = nullptr;
  float *attn_norm = nullptr, *ffn_norm = nullptr, *final_norm = nullptr;
  double *inv_freq = nullptr;
  // step work buffers
  float *x = nullptr;        // [kRowPad][H] residual stream
  void *xn = nullptr;        // [kRowPad][Kpad(H)] normalised activations (inside the verify
                             // layer stack: x * gain, the RMSNorm scale deferred)
  float *ssq = nullptr;      // [kRowPad][nss] the deferred scale's partial sums of squares
  void *qb = nullptr;        // [kRowPad][q] queries after RoPE
  void *attn = nullptr;      // [kRowPad][Kpad(q)] attention output
  void *act = nullptr;       // [kRowPad][Kpad(F)] SwiGLU output
  float *part = nullptr;     // split-K partial sums
  int64_t part_elems = 0;
  float *apart_o = nullptr;  // attention partial outputs
  float *apart_ml = nullptr; // attention partial (max, sum)
  int64_t apart_rows = 0;    // capacity in (head, split, row) units
  int wave_slots = 1024;     // SIMDs of the device: waves resident at once at 1 per SIMD
  pf::ArgmaxPart *amax = nullptr;  // lm_head argmax partials
  int64_t amax_elems = 0;
  float *rope = nullptr;     // [kRowPad][head_dim/2][2] cos, sin of the step's rows
  int32_t *rowinfo = nullptr;// [kRowPad][4]: token, position offset (depth), valid, pad
  int32_t *pred = nullptr;   // [kRowPad]
  int32_t *flags = nullptr;  // [4] device status words
  int64_t bytes = 0;
  // prefill work buffers (allocated on first use, sized for pre_rows rows)
  int64_t pre_rows = 0;
  float *pre_x = nullptr, *pre_y = nullptr, *pre_rope = nullptr, *pre_apo = nullptr,
        *pre_apml = nullptr;
  void *pre_xn = nullptr, *pre_qb = nullptr, *pre_attn = nullptr, *pre_act = nullptr;
  int32_t *pre_rowinfo = nullptr, *pre_status = nullptr;
  float *pre_part = nullptr;  // split-K partial sums of the bf16 prefill GEMMs
  void *pre_xb = nullptr;     // bf16: FFN input rows in the 32-row packed layout
  // pinned host staging of the decode iteration (draft and result copies),
  // allocated on its first use
  void *stage = nullptr;
  int32_t last_rows = 0;  // rows of the last verify step
};

// proposal-length controller: parameters and estimator states
struct pf_ctl {
  pf_ctl_params p;
  pf_ctl_state st;
};

struct pf_store {
  int32_t *tokens = nullptr;     // [T]
  int32_t *ent_pos = nullptr;    // [E] eligible positions grouped by bucket
  int32_t *ent_rem = nullptr;    // [E] b(p) - p
  int32_t *bucket_off = nullptr; // [nb + 1]
  int64_t T = 0, E = 0;
  int32_t nb_log2 = 0;
  int32_t ngram = 0;
  // cosine index (pf_store_attach_keys): entries p < b(p) grouped by token
  int8_t *keys = nullptr;        // [T][PF_KEY_DIM]
  int32_t *tok_off = nullptr;    // [n_tok + 1]
  int32_t *cpos = nullptr;       // [Ec] positions, ascending within a token
  int32_t *crem = nullptr;       // [Ec] b(p) - p
  int32_t *cnk = nullptr;        // [Ec] squared norm of the key
  int4 *cpart = nullptr;         // lookup scratch: per-block best candidates
  int32_t *cpart_elig = nullptr; // lookup scratch: per-block eligible counts
  int64_t Ec = 0;
  int32_t n_tok = 0;
  // host copies kept for attaching keys: tokens and each position's
  // sequence-last position b(p)
  std::vector<int32_t> h_tokens, h_last;
  // append region (pf_store_reserve): positions T .. T + cap_log - 1 of the
  // token and key arrays, filled by appends to the open sequence
  int32_t cap_log = 0, max_log_seqs = 0;
  int32_t *log_state = nullptr;  // device [2]: appended positions, sequences opened
  int32_t *log_seq = nullptr;    // [cap_log] sequence of each appended position
  int32_t *log_nk = nullptr;     // [cap_log] squared key norm
  int32_t *seq_end = nullptr;    // [max_log_seqs] last position of each appended sequence
  int8_t *row_keys = nullptr;    // [kRowPad][PF_KEY_DIM] keys of a verify step's rows
  int64_t log_host_bound = 0;    // host upper bound of log_state[0]
  int32_t log_seqs_host = 0;     // sequences opened
};

struct pf_keyproj {
  float *Rc = nullptr;   // [PF_KEY_DIM][16][Lc]: R[j][c + 16 t] at [j][c][t], zeros past H
  double *v = nullptr;   // work: projections of one batch of rows
  int32_t H = 0, Lc = 0;
};

namespace pf {
// n-gram hash used by the store builder (host) and the lookup kernel.
__host__ __device__ inline uint32_t ngram_hash(const int32_t *t, int n) {
  uint32_t h = 2166136261u;
  for (int i = 0; i < n; ++i) {
    h ^= (uint32_t)t[i];
    h *= 16777619u;
  }
  h ^= h >> 16;
  h *= 0x85EBCA6Bu;
  h ^= h >> 13;
  h *= 0xC2B2AE35u;
  h ^= h >> 16;
  return h;
}
}  // namespace pf
