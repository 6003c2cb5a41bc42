/*
 * Seeded synthetic inputs for the atomic-expert layer.
 *
 * This module only draws numbers. It holds none of the layer's arithmetic, and
 * both the GPU path and the oracle receive the same host buffers it fills.
 *
 * Generator (counter based, so any element can be drawn on its own):
 *   - SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
 *     generators", OOPSLA 2014): the n-th output (n >= 1) of the stream seeded
 *     with s is mix(s + n * 0x9E3779B97F4A7C15) with the published mix
 *     constants below.
 *   - The stream of tensor `stream` under `seed` is seeded with
 *     key = first output of the SplitMix64 stream seeded with seed * 256 + stream.
 *   - Element number c of a tensor consumes outputs 6c+1 .. 6c+6 of its stream.
 *     Each 64-bit output gives two 24-bit uniforms (bits 63..40 and 39..16).
 *   - A standard-normal stand-in is the Irwin-Hall sum of those twelve
 *     uniforms, centred: z = (S - 6 * 2^24) / 2^24 with S = sum of the twelve
 *     24-bit integers. It has mean 0 and variance 1 (up to 2^-24 terms) and is
 *     bounded by |z| < 6.
 *   - The stored value is (float)((double)(S - 6 * 2^24) * (scale * 2^-24)):
 *     one rounding in double, then one to float. For bf16 outputs the float is
 *     rounded to nearest-even on its upper 16 bits.
 * The arithmetic is integer, plus IEEE double multiplication, so the values
 * are the same on every machine.
 */
#include <stdint.h>
#include <string.h>
#include <pthread.h>

#define SM64_GAMMA 0x9E3779B97F4A7C15ULL

static inline uint64_t sm64_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

uint64_t synth_stream_key(uint64_t seed, uint32_t stream) {
  return sm64_mix(seed * 256ULL + (uint64_t)stream + SM64_GAMMA);
}

/* Centred Irwin-Hall integer sum for element `c` of the stream `key`. */
static inline int64_t ih12_centred(uint64_t key, uint64_t c) {
  int64_t s = 0;
  uint64_t n = 6ULL * c + 1ULL;
  for (int j = 0; j < 6; ++j) {
    uint64_t w = sm64_mix(key + (n + (uint64_t)j) * SM64_GAMMA);
    s += (int64_t)(w >> 40);
    s += (int64_t)((w >> 16) & 0xFFFFFFULL);
  }
  return s - 6LL * (1LL << 24);
}

static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

typedef struct {
  uint64_t key;
  const int64_t* rows;    /* NULL: rows first_row, first_row + 1, ... */
  int64_t first_row;
  int64_t row_begin, row_end; /* local row range of this worker */
  int64_t row_len;
  const double* row_scale;    /* NULL or indexed by global row id */
  double scale;
  int out_bf16;
  void* out;
} fill_job;

static void* fill_worker(void* arg) {
  const fill_job* j = (const fill_job*)arg;
  const double two_m24 = 1.0 / 16777216.0;
  for (int64_t r = j->row_begin; r < j->row_end; ++r) {
    int64_t grow = j->rows ? j->rows[r] : j->first_row + r;
    double s = j->scale * two_m24;
    if (j->row_scale) s = j->scale * j->row_scale[grow] * two_m24;
    uint64_t c0 = (uint64_t)grow * (uint64_t)j->row_len;
    for (int64_t m = 0; m < j->row_len; ++m) {
      float f = (float)((double)ih12_centred(j->key, c0 + (uint64_t)m) * s);
      int64_t o = r * j->row_len + m;
      if (j->out_bf16)
        ((uint16_t*)j->out)[o] = f32_to_bf16_rne(f);
      else
        ((float*)j->out)[o] = f;
    }
  }
  return 0;
}

/*
 * Fill `n_rows` rows of `row_len` elements. Row r of the output holds global
 * row rows[r] (or first_row + r when rows is NULL); element m of global row g
 * is element g * row_len + m of the tensor's stream. The value is
 * scale * row_scale[g] * z (row_scale may be NULL, meaning 1).
 */
void synth_fill_rows(uint64_t seed, uint32_t stream, const int64_t* rows,
                     int64_t first_row, int64_t n_rows, int64_t row_len,
                     const double* row_scale, double scale, int out_bf16,
                     void* out, int n_threads) {
  if (n_rows <= 0 || row_len <= 0) return;
  if (n_threads < 1) n_threads = 1;
  if (n_threads > 64) n_threads = 64;
  if ((int64_t)n_threads > n_rows) n_threads = (int)n_rows;
  pthread_t th[64];
  fill_job jobs[64];
  uint64_t key = synth_stream_key(seed, stream);
  for (int i = 0; i < n_threads; ++i) {
    fill_job* j = &jobs[i];
    j->key = key;
    j->rows = rows;
    j->first_row = first_row;
    j->row_begin = n_rows * i / n_threads;
    j->row_end = n_rows * (i + 1) / n_threads;
    j->row_len = row_len;
    j->row_scale = row_scale;
    j->scale = scale;
    j->out_bf16 = out_bf16;
    j->out = out;
  }
  for (int i = 1; i < n_threads; ++i) pthread_create(&th[i], 0, fill_worker, &jobs[i]);
  fill_worker(&jobs[0]);
  for (int i = 1; i < n_threads; ++i) pthread_join(th[i], 0);
}

/* Raw SplitMix64 output n (n >= 1) of the stream seeded with s; exposed so the
 * generator can be checked against the published definition. */
uint64_t synth_splitmix64_output(uint64_t s, uint64_t n) {
  return sm64_mix(s + n * SM64_GAMMA);
}
