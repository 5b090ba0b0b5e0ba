/*
 * Seeded synthetic input generator, host implementation.
 *
 * This file holds no arithmetic of the scoring method. It turns
 * (seed, stream, element index) into a storage value, and it is the
 * single source of inputs for both the fp64 oracle and the GPU path.
 * synth_device.hip implements the same definition for the GPU; the two
 * are required to agree bit for bit (checked by the test suite).
 *
 * Definition
 * ----------
 *   mix(z)       SplitMix64 finaliser (Steele, Lea, Flood, "Fast splittable
 *                pseudorandom number generators", OOPSLA 2014; constants of
 *                Vigna's reference splitmix64.c).
 *   key          mix(mix(seed + G) + stream * G),  G = 0x9E3779B97F4A7C15
 *   word(n)      mix(key + (n + 1) * G)            (SplitMix64 state n+1)
 *   normal(i)    Irwin-Hall sum of twelve 16-bit uniforms taken from
 *                word(3i), word(3i+1), word(3i+2):
 *                    z = (S - 393210) / 65536      (exact in double)
 *                mean 0, variance 1 - 2^-32, support [-6, 6].
 *   value(i)     mean + std * z, in double (product rounded, then sum
 *                rounded; no fused multiply-add), then rounded to the
 *                storage type: fp32 by round-to-nearest-even, bf16 by
 *                round-to-nearest-even from that fp32.
 *   fp8 tiles    a tile of T consecutive normals z_i (index t*T + i) gets a
 *                scale s and codes q_i = E4M3FN(z_i / s) rounded to nearest
 *                even (saturating at 448; no NaN is produced). Scale mode 0:
 *                s = 2^e, the smallest power of two with amax / s <= 448;
 *                mode 1: s = fp32(amax / 448) (1 for an all-zero tile), so
 *                that the tile's largest value maps to the top of the e4m3
 *                range; z_i / s is one correctly rounded double division.
 *
 * Only integer operations and correctly rounded IEEE basic operations are
 * used, so every platform that follows IEEE 754 gives identical bits.
 * Build with contraction off (-ffp-contract=off).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define SYN_GAMMA 0x9E3779B97F4A7C15ULL

static inline uint64_t syn_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

uint64_t synth_key(uint64_t seed, uint64_t stream) {
  return syn_mix(syn_mix(seed + SYN_GAMMA) + stream * SYN_GAMMA);
}

static inline uint64_t syn_word(uint64_t key, uint64_t n) {
  return syn_mix(key + (n + 1) * SYN_GAMMA);
}

static inline uint32_t syn_sum4(uint64_t w) {
  return (uint32_t)(w & 0xFFFF) + (uint32_t)((w >> 16) & 0xFFFF) +
         (uint32_t)((w >> 32) & 0xFFFF) + (uint32_t)(w >> 48);
}

static inline double syn_normal(uint64_t key, uint64_t i) {
  uint32_t s = syn_sum4(syn_word(key, 3 * i)) + syn_sum4(syn_word(key, 3 * i + 1)) +
               syn_sum4(syn_word(key, 3 * i + 2));
  return ((double)s - 393210.0) * (1.0 / 65536.0);
}

static inline uint16_t syn_f32_to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

/* value(i) for i in [offset, offset + n): dtype 0 = fp32, 1 = bf16, 2 = fp64 */
void synth_fill_normal(void *out, int64_t n, uint64_t seed, uint64_t stream, int64_t offset,
                       double mean, double stdv, int dtype) {
  uint64_t key = synth_key(seed, stream);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    double z = syn_normal(key, (uint64_t)(offset + i));
    double prod = stdv * z;
    double v = mean + prod;
    if (dtype == 0) {
      ((float *)out)[i] = (float)v;
    } else if (dtype == 1) {
      ((uint16_t *)out)[i] = syn_f32_to_bf16((float)v);
    } else {
      ((double *)out)[i] = v;
    }
  }
}

/* E4M3FN encode of x (finite, |x| <= 448 after scaling) with round to nearest even. */
static uint8_t syn_e4m3_rne(double x) {
  uint8_t sign = 0;
  if (x < 0) {
    sign = 0x80;
    x = -x;
  }
  if (x >= 448.0) return sign | 0x7E;
  /* find the binade: normal numbers 2^(e-7) * (1 + m/8), e in 1..15; subnormals 2^-6 * m/8 */
  int e;
  double fr = frexp(x, &e); /* x = fr * 2^e, fr in [0.5, 1) ; exact */
  int unb = e - 1;          /* x = 1.xxx * 2^unb */
  double step;
  if (unb < -6) {
    step = ldexp(1.0, -9); /* subnormal spacing 2^-6 / 8 */
  } else {
    step = ldexp(1.0, unb - 3);
  }
  (void)fr;
  double q = x / step; /* exact: step is a power of two */
  double fl = floor(q);
  double rem = q - fl;
  uint64_t m = (uint64_t)fl;
  if (rem > 0.5 || (rem == 0.5 && (m & 1))) m += 1;
  /* value = m * step; re-encode */
  double val = (double)m * step;
  if (val == 0.0) return sign;
  if (val >= 448.0) return sign | 0x7E;
  int e2;
  frexp(val, &e2);
  int ub = e2 - 1;
  if (ub < -6) {
    /* subnormal: val = k * 2^-9, k in 1..7 */
    uint32_t k = (uint32_t)(val * 512.0);
    return sign | (uint8_t)k;
  }
  uint32_t exp_field = (uint32_t)(ub + 7);
  double mant = val / ldexp(1.0, ub) - 1.0; /* in [0, 1), multiple of 1/8 */
  uint32_t mf = (uint32_t)(mant * 8.0);
  return sign | (uint8_t)((exp_field << 3) | mf);
}

/* Tiles t in [tile0, tile0 + ntiles), each of T elements: codes and scales (scale_mode 0:
 * powers of two; 1: amax / 448). */
void synth_fill_fp8_tiles(uint8_t *codes, float *scales, int64_t ntiles, int64_t T, uint64_t seed,
                          uint64_t stream, int64_t tile0, int scale_mode) {
  uint64_t key = synth_key(seed, stream);
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < ntiles; ++t) {
    uint64_t base = (uint64_t)(tile0 + t) * (uint64_t)T;
    double amax = 0.0;
    for (int64_t i = 0; i < T; ++i) {
      double a = fabs(syn_normal(key, base + (uint64_t)i));
      if (a > amax) amax = a;
    }
    if (scale_mode == 1) {
      float sf = amax > 0.0 ? (float)(amax / 448.0) : 1.0f;
      scales[t] = sf;
      for (int64_t i = 0; i < T; ++i)
        codes[t * T + i] = syn_e4m3_rne(syn_normal(key, base + (uint64_t)i) / (double)sf);
      continue;
    }
    /* smallest e with amax <= 448 * 2^e; 448 = 0.875 * 2^9 and amax = f * 2^ea, f in [0.5, 1) */
    int e = -30;
    if (amax > 0.0) {
      int ea;
      double f = frexp(amax, &ea);
      e = (f <= 0.875) ? ea - 9 : ea - 8;
    }
    double s = ldexp(1.0, e);
    scales[t] = (float)s;
    for (int64_t i = 0; i < T; ++i) {
      double z = syn_normal(key, base + (uint64_t)i);
      codes[t * T + i] = syn_e4m3_rne(ldexp(z, -e));
    }
  }
}

/* Raw 64-bit words word(offset .. offset+n) (for integer recipes: lengths, permutations). */
void synth_words(uint64_t *out, int64_t n, uint64_t seed, uint64_t stream, int64_t offset) {
  uint64_t key = synth_key(seed, stream);
  for (int64_t i = 0; i < n; ++i) out[i] = syn_word(key, (uint64_t)(offset + i));
}
