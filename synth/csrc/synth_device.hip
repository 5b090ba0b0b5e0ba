// Seeded synthetic input generator, GPU implementation.
//
// Same definition as synth_host.c (SplitMix64 counter words, Irwin-Hall
// normals, round-to-nearest-even storage rounding, fp8 tile scales as powers
// of two or amax / 448); it exists so that multi-GB inputs can be written straight into
// HBM. It holds no arithmetic of the scoring method. The test suite checks
// that both implementations produce identical bits.
//
// Built with -ffp-contract=off: the double product and sum that form each
// value must round separately, exactly as on the host.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#define SYN_GAMMA 0x9E3779B97F4A7C15ULL

__host__ __device__ static inline uint64_t syn_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static uint64_t syn_key(uint64_t seed, uint64_t stream) {
  return syn_mix(syn_mix(seed + SYN_GAMMA) + stream * SYN_GAMMA);
}

__device__ static inline uint32_t syn_sum4(uint64_t w) {
  return (uint32_t)(w & 0xFFFF) + (uint32_t)((w >> 16) & 0xFFFF) +
         (uint32_t)((w >> 32) & 0xFFFF) + (uint32_t)(w >> 48);
}

__device__ static inline double syn_normal(uint64_t key, uint64_t i) {
  uint32_t s = syn_sum4(syn_mix(key + (3 * i + 1) * SYN_GAMMA)) +
               syn_sum4(syn_mix(key + (3 * i + 2) * SYN_GAMMA)) +
               syn_sum4(syn_mix(key + (3 * i + 3) * SYN_GAMMA));
  return ((double)s - 393210.0) * (1.0 / 65536.0);
}

__device__ static inline uint16_t syn_f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__global__ void syn_fill_normal_kernel(void *out, int64_t n, uint64_t key, int64_t offset,
                                       double mean, double stdv, int dtype) {
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    double z = syn_normal(key, (uint64_t)(offset + i));
    double prod = __dmul_rn(stdv, z);
    double v = __dadd_rn(mean, prod);
    if (dtype == 0) {
      ((float *)out)[i] = __double2float_rn(v);
    } else if (dtype == 1) {
      ((uint16_t *)out)[i] = syn_f32_to_bf16(__double2float_rn(v));
    } else {
      ((double *)out)[i] = v;
    }
  }
}

__device__ static uint8_t syn_e4m3_rne(double x) {
  uint8_t sign = 0;
  if (x < 0) {
    sign = 0x80;
    x = -x;
  }
  if (x >= 448.0) return sign | 0x7E;
  int e;
  frexp(x, &e);
  int unb = e - 1;
  double step = (unb < -6) ? ldexp(1.0, -9) : ldexp(1.0, unb - 3);
  double q = ldexp(x, -ilogb(step));
  double fl = floor(q);
  double rem = q - fl;
  uint64_t m = (uint64_t)fl;
  if (rem > 0.5 || (rem == 0.5 && (m & 1))) m += 1;
  double val = ldexp((double)m, ilogb(step));
  if (val == 0.0) return sign;
  if (val >= 448.0) return sign | 0x7E;
  int e2;
  frexp(val, &e2);
  int ub = e2 - 1;
  if (ub < -6) {
    uint32_t k = (uint32_t)ldexp(val, 9);
    return sign | (uint8_t)k;
  }
  uint32_t exp_field = (uint32_t)(ub + 7);
  double mant = ldexp(val, -ub) - 1.0;
  uint32_t mf = (uint32_t)ldexp(mant, 3);
  return sign | (uint8_t)((exp_field << 3) | mf);
}

// One 64-lane wave per tile: amax by a wave reduction (max is order-free), then codes.
__global__ void syn_fill_fp8_kernel(uint8_t *codes, float *scales, int64_t ntiles, int64_t T,
                                    uint64_t key, int64_t tile0, int scale_mode) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t t = wave; t < ntiles; t += nwaves) {
    uint64_t base = (uint64_t)(tile0 + t) * (uint64_t)T;
    double amax = 0.0;
    for (int64_t i = lane; i < T; i += 64) amax = fmax(amax, fabs(syn_normal(key, base + i)));
    for (int off = 32; off > 0; off >>= 1) amax = fmax(amax, __shfl_xor(amax, off, 64));
    if (scale_mode == 1) {
      const float sf = amax > 0.0 ? (float)(amax / 448.0) : 1.0f;
      if (lane == 0) scales[t] = sf;
      for (int64_t i = lane; i < T; i += 64)
        codes[t * T + i] = syn_e4m3_rne(syn_normal(key, base + i) / (double)sf);
      continue;
    }
    int e = -30;
    if (amax > 0.0) {
      int ea;
      double f = frexp(amax, &ea);
      e = (f <= 0.875) ? ea - 9 : ea - 8;
    }
    if (lane == 0) scales[t] = (float)ldexp(1.0, e);
    for (int64_t i = lane; i < T; i += 64)
      codes[t * T + i] = syn_e4m3_rne(ldexp(syn_normal(key, base + i), -e));
  }
}

extern "C" {

// dtype 0 = fp32, 1 = bf16, 2 = fp64. `out` is device memory of n elements. Returns a hipError_t.
int synth_dev_fill_normal(void *out, int64_t n, uint64_t seed, uint64_t stream, int64_t offset,
                          double mean, double stdv, int dtype, void *stream_handle) {
  if (n <= 0) return 0;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(syn_fill_normal_kernel, dim3((unsigned)blocks), dim3(256), 0,
                     (hipStream_t)stream_handle, out, n, syn_key(seed, stream), offset, mean, stdv,
                     dtype);
  return (int)hipGetLastError();
}

int synth_dev_fill_fp8_tiles(uint8_t *codes, float *scales, int64_t ntiles, int64_t T, uint64_t seed,
                             uint64_t stream, int64_t tile0, int scale_mode, void *stream_handle) {
  if (ntiles <= 0) return 0;
  int64_t blocks = (ntiles + 3) / 4;  // 4 waves per block
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(syn_fill_fp8_kernel, dim3((unsigned)blocks), dim3(256), 0,
                     (hipStream_t)stream_handle, codes, scales, ntiles, T, syn_key(seed, stream),
                     tile0, scale_mode);
  return (int)hipGetLastError();
}

}  // extern "C"
