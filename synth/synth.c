/*
 * Seeded synthetic input generator.
 *
 * This file produces the bulk random tensors (weights, KV prefixes) that both
 * the oracle and the HIP path consume. It contains none of the decoding
 * method's arithmetic: only a counter-based random stream and the conversion
 * of its draws to the storage formats (fp32, bf16 bit patterns).
 *
 * Random stream: SplitMix64 (Steele, Lea, Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014), used in counter mode:
 *   draw(key, i) = mix64(key + (i + 1) * GOLDEN)
 * where mix64 is the SplitMix64 output finaliser. Every element is a pure
 * function of (key, index), so any thread split gives identical bytes.
 *
 * Normals: Box-Muller on pairs of 53-bit uniforms; element 2j takes the
 * cosine branch of pair j, element 2j+1 the sine branch.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <string.h>

#define SY_GOLDEN 0x9E3779B97F4A7C15ULL

static inline uint64_t sy_mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

uint64_t sy_draw(uint64_t key, uint64_t i) { return sy_mix64(key + (i + 1) * SY_GOLDEN); }

/* Stream key for (seed, tensor id). */
uint64_t sy_key(uint64_t seed, uint64_t tensor_id) {
  return sy_mix64(sy_mix64(seed + SY_GOLDEN) ^ (tensor_id * 0xD1B54A32D192ED03ULL));
}

static inline double sy_unit(uint64_t key, uint64_t i) {
  return (double)(sy_draw(key, i) >> 11) * (1.0 / 9007199254740992.0); /* [0,1) */
}

static inline double sy_normal_at(uint64_t key, uint64_t idx) {
  uint64_t pair = idx >> 1;
  double u1 = sy_unit(key, 2 * pair);
  double u2 = sy_unit(key, 2 * pair + 1);
  double r = sqrt(-2.0 * log(1.0 - u1)); /* 1-u1 in (0,1] */
  double a = 6.283185307179586476925286766559 * u2;
  return (idx & 1) ? r * sin(a) : r * cos(a);
}

/* fp32 -> bf16 bit pattern, round to nearest even; NaN -> quiet NaN. */
static inline uint16_t sy_f32_to_bf16(float f) {
  uint32_t b;
  memcpy(&b, &f, 4);
  if ((b & 0x7F800000u) == 0x7F800000u && (b & 0x007FFFFFu)) return 0x7FC0;
  b += 0x7FFFu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}

typedef struct {
  uint64_t key;
  int64_t begin, end;
  double mean, std;
  void *out;
  int kind; /* 0: f32 normal, 1: bf16 normal, 2: f32 bf16-representable normal */
} sy_job;

static void *sy_worker(void *arg) {
  sy_job *j = (sy_job *)arg;
  for (int64_t i = j->begin; i < j->end; ++i) {
    float v = (float)(j->mean + j->std * sy_normal_at(j->key, (uint64_t)i));
    if (j->kind == 0) {
      ((float *)j->out)[i] = v;
    } else {
      uint16_t h = sy_f32_to_bf16(v);
      if (j->kind == 1) {
        ((uint16_t *)j->out)[i] = h;
      } else {
        uint32_t b = (uint32_t)h << 16;
        memcpy(&((float *)j->out)[i], &b, 4);
      }
    }
  }
  return NULL;
}

static void sy_run(uint64_t key, int64_t n, double mean, double std, void *out, int kind,
                   int threads) {
  if (threads < 1) threads = 1;
  if (threads > 256) threads = 256;
  if (n < 65536) threads = 1;
  pthread_t tid[256];
  sy_job jobs[256];
  int64_t chunk = (n + threads - 1) / threads;
  chunk = (chunk + 1) & ~(int64_t)1; /* keep Box-Muller pairs within one job */
  int started = 0;
  for (int t = 0; t < threads; ++t) {
    int64_t b = (int64_t)t * chunk, e = b + chunk;
    if (b >= n) break;
    if (e > n) e = n;
    jobs[t] = (sy_job){key, b, e, mean, std, out, kind};
    if (threads == 1) {
      sy_worker(&jobs[t]);
    } else {
      pthread_create(&tid[t], NULL, sy_worker, &jobs[t]);
      ++started;
    }
  }
  for (int t = 0; t < started; ++t) pthread_join(tid[t], NULL);
}

/* out[i] = mean + std * N(0,1)_i as fp32. */
void sy_normal_f32(uint64_t key, int64_t n, double mean, double std, float *out, int threads) {
  sy_run(key, n, mean, std, out, 0, threads);
}

/* out[i] = bf16_rne(mean + std * N(0,1)_i), stored as raw bf16 bits. */
void sy_normal_bf16(uint64_t key, int64_t n, double mean, double std, uint16_t *out,
                    int threads) {
  sy_run(key, n, mean, std, out, 1, threads);
}

/* Same values as sy_normal_bf16 but widened back to fp32 (exactly representable). */
void sy_normal_bf16_as_f32(uint64_t key, int64_t n, double mean, double std, float *out,
                           int threads) {
  sy_run(key, n, mean, std, out, 2, threads);
}

/* Raw 64-bit draws for indices [first, first+n). */
void sy_draws(uint64_t key, uint64_t first, int64_t n, uint64_t *out) {
  for (int64_t i = 0; i < n; ++i) out[i] = sy_draw(key, first + (uint64_t)i);
}
