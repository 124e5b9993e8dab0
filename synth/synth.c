/*
 * Seeded synthetic KV caches shaped like a streaming video MLLM's cache.
 *
 * This module only draws random numbers and lays them out; it holds none of
 * the compression method's arithmetic. Both the CPU oracle and the GPU path
 * consume the bytes it writes.
 *
 * Random numbers are counter based, so any element can be drawn on its own
 * and the fill parallelises over threads without changing a single bit:
 *   u64 = splitmix64_mix(seed_state(seed, tag) + (counter + 1) * GOLDEN)
 * where splitmix64_mix is the output function of SplitMix64 (Steele, Lea and
 * Flood, "Fast splittable pseudorandom number generators", OOPSLA 2014).
 * A uniform in (0, 1] takes the top 53 bits; a standard normal is the cosine
 * branch of the Box-Muller transform over the uniforms at counters 2i, 2i+1.
 *
 * Keys follow a per-patch AR(1) process along the frame axis:
 *   K[0] ~ N(0,1),  K[f] = rho_q * K[f-1] + sqrt(1 - rho_q^2) * eps_f,
 * carried in fp64 and stored rounded (fp64 -> fp32 -> bf16, each step
 * round-to-nearest-even). Values are N(0,1) elements times one
 * LogNormal(0, sigma_l) scale per row.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define GOLDEN 0x9E3779B97F4A7C15ULL

enum { TAG_RHO = 1, TAG_STATIC = 2, TAG_K = 3, TAG_VZ = 5, TAG_VSCALE = 6 };
enum { SYN_BF16 = 0, SYN_F32 = 1 };

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static inline uint64_t seed_state(uint64_t seed, uint64_t tag) {
  return mix64(seed * GOLDEN + 0x632BE59BD9B4E019ULL) ^ (tag * 0xD1B54A32D192ED03ULL);
}

static inline uint64_t draw(uint64_t state, uint64_t counter) {
  return mix64(state + (counter + 1) * GOLDEN);
}

/* uniform in (0, 1] */
static inline double unif(uint64_t state, uint64_t counter) {
  return ((double)(draw(state, counter) >> 11) + 1.0) * (1.0 / 9007199254740992.0);
}

static inline double normal(uint64_t state, uint64_t counter) {
  double u1 = unif(state, 2 * counter);
  double u2 = unif(state, 2 * counter + 1);
  return sqrt(-2.0 * log(u1)) * cos(6.283185307179586476925 * u2);
}

static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)(u >> 16); /* inf/nan: not produced here */
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7fffu + lsb;
  return (uint16_t)(u >> 16);
}

static inline void store(void* out, int dtype, int64_t i, double x) {
  float f = (float)x;
  if (dtype == SYN_BF16)
    ((uint16_t*)out)[i] = f32_to_bf16_rne(f);
  else
    ((float*)out)[i] = f;
}

/* counter layout: (lh << 40) | (frame << 20) | within-frame offset */
static inline uint64_t ctr(int64_t lh, int64_t f, int64_t off) {
  return ((uint64_t)lh << 40) | ((uint64_t)f << 20) | (uint64_t)off;
}

/* Per-patch AR(1) coefficient: with probability static_frac the patch is
 * static (rho = static_rho), otherwise rho ~ U(lo, hi). */
void synth_rho(uint64_t seed, int32_t p, double static_frac, double static_rho, double lo, double hi,
               double* rho) {
  uint64_t s_static = seed_state(seed, TAG_STATIC), s_rho = seed_state(seed, TAG_RHO);
  for (int32_t q = 0; q < p; ++q) {
    double us = unif(s_static, (uint64_t)q);
    double ur = unif(s_rho, (uint64_t)q);
    rho[q] = (us <= static_frac) ? static_rho : lo + (hi - lo) * ur;
  }
}

/*
 * Keys of frames [f0, f0 + nf) for every (layer, head), written as rows
 * out[lh * slice_stride + row0 + (f - f0) * p + q][d]. Rows whose stream
 * position f * p + q is >= row_limit are skipped (partial last frame), and so
 * is the recurrence update for them (they are never read back).
 * state[lh][q][d] holds K[f-1] in fp64 and is updated; it is ignored for f = 0.
 */
int synth_keys(uint64_t seed, int32_t LH, int32_t p, int32_t D, const double* rho, int32_t f0, int32_t nf,
               int64_t row_limit, double* state, void* out, int64_t slice_stride_rows, int64_t row0,
               int32_t dtype) {
  if (p <= 0 || D <= 0 || (int64_t)p * D >= (1 << 20) || f0 < 0 || f0 + nf >= (1 << 20)) return -1;
  uint64_t sk = seed_state(seed, TAG_K);
#pragma omp parallel for collapse(2) schedule(static)
  for (int32_t lh = 0; lh < LH; ++lh) {
    for (int32_t q = 0; q < p; ++q) {
      double a = rho[q], b = sqrt(1.0 - rho[q] * rho[q]);
      for (int32_t f = f0; f < f0 + nf; ++f) {
        if ((int64_t)f * p + q >= row_limit) break;
        int64_t orow = (int64_t)lh * slice_stride_rows + row0 + (int64_t)(f - f0) * p + q;
        double* st = state + ((int64_t)lh * p + q) * D;
        for (int32_t d = 0; d < D; ++d) {
          double e = normal(sk, ctr(lh, f, (int64_t)q * D + d));
          double k = (f == 0) ? e : a * st[d] + b * e;
          st[d] = k;
          store(out, dtype, orow * D + d, k);
        }
      }
    }
  }
  return 0;
}

/*
 * Values of frames [f0, f0 + nf): V = z * exp(sigma_l * g), z ~ N(0,1) per
 * element, g ~ N(0,1) per row. sigma has one entry per layer (LH = L * H).
 */
int synth_values(uint64_t seed, int32_t L, int32_t H, int32_t p, int32_t D, const double* sigma, int32_t f0,
                 int32_t nf, int64_t row_limit, void* out, int64_t slice_stride_rows, int64_t row0,
                 int32_t dtype) {
  if (p <= 0 || D <= 0 || (int64_t)p * D >= (1 << 20) || f0 < 0 || f0 + nf >= (1 << 20)) return -1;
  uint64_t sz = seed_state(seed, TAG_VZ), ss = seed_state(seed, TAG_VSCALE);
  int32_t LH = L * H;
#pragma omp parallel for collapse(2) schedule(static)
  for (int32_t lh = 0; lh < LH; ++lh) {
    for (int32_t f = f0; f < f0 + nf; ++f) {
      double sg = sigma[lh / H];
      for (int32_t q = 0; q < p; ++q) {
        if ((int64_t)f * p + q >= row_limit) break;
        int64_t orow = (int64_t)lh * slice_stride_rows + row0 + (int64_t)(f - f0) * p + q;
        double scale = exp(sg * normal(ss, ctr(lh, f, q)));
        for (int32_t d = 0; d < D; ++d) {
          double z = normal(sz, ctr(lh, f, (int64_t)q * D + d));
          store(out, dtype, orow * D + d, z * scale);
        }
      }
    }
  }
  return 0;
}

/* Fresh-cache metadata: row x of every slice holds frame x / p, patch x % p. */
void synth_fresh_meta(int32_t LH, int64_t S, int64_t n, int32_t p, int32_t* frame_idx, int32_t* patch_idx) {
#pragma omp parallel for schedule(static)
  for (int32_t lh = 0; lh < LH; ++lh) {
    for (int64_t x = 0; x < S; ++x) {
      int64_t i = (int64_t)lh * S + x;
      frame_idx[i] = x < n ? (int32_t)(x / p) : -1;
      patch_idx[i] = x < n ? (int32_t)(x % p) : -1;
    }
  }
}

/* Raw draws, exposed so tests can check the generator's own statistics. */
void synth_normals(uint64_t seed, uint64_t tag, uint64_t c0, int64_t count, double* out) {
  uint64_t s = seed_state(seed, tag);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < count; ++i) out[i] = normal(s, c0 + (uint64_t)i);
}
