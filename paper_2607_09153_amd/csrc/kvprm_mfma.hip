// Matrix-core (MFMA, v_mfma_f32_16x16x32_bf16) kernels of the verify-token pass for gfx950:
// the projection GEMVs over bf16 weights and the split-L paged attention over bf16 / fp8 caches.
//
// Precision: weights and cache values enter the matrix cores exactly (bf16, or e4m3 widened to
// bf16, which is exact). The fp32 operands on the other side (activations, queries, softmax
// probabilities) are split as x = hi + lo with hi = bf16(x), lo = bf16(x - hi), and both halves
// are multiplied, so products carry ~16 significant bits and accumulate in fp32.
//
// MFMA 16x16x32 operand layout used throughout (lane l, c = l / 16, n = l % 16):
//   A (16 x 32): lane holds row n, reduction slots 8c .. 8c+7
//   B (32 x 16): lane holds column n, reduction slots 8c .. 8c+7
//   D (16 x 16): lane holds rows 4c .. 4c+3 of column n
// Reduction slots are paired between A and B by (c, element), so any assignment of the
// contracted index to slots is valid as long as both operands use the same one.
#include <math.h>

#include "kvprm_internal.h"

namespace kvprm {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ floatx4 mfma16(const uint4 &a, const uint4 &b, const floatx4 &c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// round-to-nearest-even fp32 -> bf16 bits (finite inputs)
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ void split_hi_lo(float x, uint32_t &hi, uint32_t &lo) {
  hi = bf16_rne(x);
  lo = bf16_rne(x - __uint_as_float(hi << 16));
}

__device__ __forceinline__ uint32_t pack2(uint32_t a, uint32_t b) { return a | (b << 16); }

// ------------------------------------------------------------------------------- GEMV operand

// Activation operand of the projection GEMV, in B-operand order:
//   buf[(kb * NT + t) * 64 + lane] = 8 bf16 for k = 32 kb + 8 (lane / 16) + i, column
//   t * 16 + lane % 16.
// Column -> (candidate, half): with Bp == 8 (NT == 1) columns 0..7 are the hi halves and 8..15
// the lo halves of candidates 0..7; otherwise columns [0, Bp) are hi and [Bp, 2 Bp) lo.
// u = in (optionally RMS-normalised: in * rsqrt(mean(in^2) + eps) * gamma, with the sum of
// squares taken from the per-256-row partials ss).
__global__ __launch_bounds__(256) void k_act_prep(const float *in, int K, const void *gamma,
                                                  int wdt, const float *ss, int nss, float eps,
                                                  int B, int Bp, int NT, uint4 *buf) {
  const int idx = blockIdx.x * 256 + threadIdx.x;
  const int total = (K / 32) * NT * 64;
  if (idx >= total) return;
  const int lane = idx & 63;
  const int t = (idx >> 6) % NT;
  const int kb = (idx >> 6) / NT;
  const int col = t * 16 + (lane & 15);
  const int lo_half = (col >= Bp) ? 1 : 0;
  const int cand = col - lo_half * Bp;
  uint32_t h16[8];
  if (cand < B) {
    float inv = 1.f;
    if (gamma) {
      float s = 0.f;
      for (int i = 0; i < nss; ++i) s += ss[(size_t)i * B + cand];
      inv = 1.0f / sqrtf(s / (float)K + eps);
    }
    const int k0 = kb * 32 + 8 * (lane >> 4);
    const float *src = in + (size_t)cand * K + k0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      float u = src[i];
      if (gamma) {
        const float gm = wdt ? __uint_as_float((uint32_t)((const uint16_t *)gamma)[k0 + i] << 16)
                             : ((const float *)gamma)[k0 + i];
        u = u * inv * gm;
      }
      uint32_t hi, lo;
      split_hi_lo(u, hi, lo);
      h16[i] = lo_half ? lo : hi;
    }
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) h16[i] = 0;
  }
  buf[idx] = make_uint4(pack2(h16[0], h16[1]), pack2(h16[2], h16[3]), pack2(h16[4], h16[5]),
                        pack2(h16[6], h16[7]));
}

// ------------------------------------------------------------------------------- GEMV (MFMA)

// part[ks][row][b] = sum over the k-slice of W[row][k] u_b[k]. Each wave owns MT consecutive
// 16-row tiles; per 32-wide k-block it loads MT weight tiles straight from HBM into A-operand
// registers (16 bytes per lane, rows n, k 8c..8c+7) and NT activation tiles (L2-resident, 1 KiB
// per wave-load), and issues MT * NT MFMAs. hi/lo halves are added in the epilogue.
template <int MT, int NT>
__global__ __launch_bounds__(256) void k_gemv_mfma(GemvSegs segs, int rows_total, int K, int kslice,
                                                   const uint4 *act, int B, int Bp, float *part) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rt0 = (blockIdx.x * 4 + wave) * MT;
  const int ks = blockIdx.y;
  const int k0 = ks * kslice;
  const int nkb = min(kslice, K - k0) >> 5;
  if (rt0 * 16 >= rows_total) return;
  const uint16_t *wrow[MT];
  bool valid[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const int r = (rt0 + m) * 16 + (lane & 15);
    valid[m] = (rt0 + m) * 16 < rows_total;
    int seg = 0, base = 0;
    while (seg < segs.nseg - 1 && r >= base + segs.rows[seg]) base += segs.rows[seg++];
    wrow[m] = (const uint16_t *)segs.w[seg] + (size_t)(valid[m] ? r - base : 0) * K + k0 +
              8 * (lane >> 4);
  }
  floatx4 acc[MT][NT];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[m][t] = floatx4{0.f, 0.f, 0.f, 0.f};
  const uint4 *ap = act + (size_t)(k0 >> 5) * NT * 64 + lane;
#pragma unroll 4
  for (int kb = 0; kb < nkb; ++kb) {
    uint4 a[MT], bv[NT];
#pragma unroll
    for (int m = 0; m < MT; ++m)
      a[m] = valid[m] ? *(const uint4 *)(wrow[m] + kb * 32) : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int t = 0; t < NT; ++t) bv[t] = ap[(size_t)(kb * NT + t) * 64];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[m][t] = mfma16(a[m], bv[t], acc[m][t]);
  }
  const int n = lane & 15, c4 = (lane >> 4) * 4;
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    if (!valid[m]) continue;
    const int rbase = (rt0 + m) * 16 + c4;
    if (NT == 1) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float v = acc[m][0][i] + __shfl_xor(acc[m][0][i], 8, 64);
        if (n < 8 && n < B) part[((size_t)ks * rows_total + rbase + i) * B + n] = v;
      }
    } else {
#pragma unroll
      for (int t = 0; t < NT / 2; ++t) {
        const int cand = t * 16 + n;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float v = acc[m][t][i] + acc[m][t + NT / 2][i];
          if (cand < B) part[((size_t)ks * rows_total + rbase + i) * B + cand] = v;
        }
      }
    }
  }
}

int gemv_nt(int B) { return B <= 8 ? 1 : 2 * ((B + 15) / 16); }
int gemv_bp(int B) { return B <= 8 ? 8 : 16 * ((B + 15) / 16); }

// Split-K plan for the MFMA GEMV: enough waves to cover the chip, k-slices of whole 32-blocks.
void gemv_split(int rows, int K, int B, int &kslice, int &ksplit) {
  const int NT = gemv_nt(B);
  const int MT = NT >= 2 ? 2 : 1;
  const int waves_per_split = (rows / 16 + MT - 1) / MT;
  const int target = 3072;
  int want = (target + waves_per_split - 1) / waves_per_split;
  const int nkb = K / 32;
  if (want < 1) want = 1;
  if (want > nkb) want = nkb;
  const int kb_per = (nkb + want - 1) / want;
  kslice = kb_per * 32;
  ksplit = (K + kslice - 1) / kslice;
}

hipError_t launch_gemv_mfma(const Dims &dm, const Plan &p, const GemvSegs &segs, int K,
                            int kslice, int ksplit, const float *in, const void *gamma,
                            const float *ss, float *part, uint4 *actbuf, hipStream_t s) {
  const int B = p.B, NT = gemv_nt(B), Bp = gemv_bp(B);
  const int total = (K / 32) * NT * 64;
  hipLaunchKernelGGL(k_act_prep, dim3((total + 255) / 256), dim3(256), 0, s, in, K, gamma, dm.wdt,
                     ss, p.nss, dm.eps, B, Bp, NT, actbuf);
  int rows = 0;
  for (int i = 0; i < segs.nseg; ++i) rows += segs.rows[i];
  const int rt = rows / 16;
#define KVPRM_GEMV(MT_, NT_)                                                                  \
  hipLaunchKernelGGL((k_gemv_mfma<MT_, NT_>), dim3((rt + 4 * MT_ - 1) / (4 * MT_), ksplit),   \
                     dim3(256), 0, s, segs, rows, K, kslice, (const uint4 *)actbuf, B, Bp, part)
  switch (NT) {
    case 1: KVPRM_GEMV(1, 1); break;
    case 2: KVPRM_GEMV(2, 2); break;
    case 4: KVPRM_GEMV(2, 4); break;
    case 6: KVPRM_GEMV(2, 6); break;
    case 8: KVPRM_GEMV(2, 8); break;
    default: return hipErrorInvalidValue;
  }
#undef KVPRM_GEMV
  return hipGetLastError();
}

// ------------------------------------------------------------------------------- attention (MFMA)

template <bool HIGH>
__device__ __forceinline__ uint32_t fp8x2_to_bf16x2(uint32_t word) {
  // two OCP e4m3 codes -> two fp32 (exact) -> upper halves are the exact bf16 values
  const auto f = __builtin_amdgcn_cvt_pk_f32_fp8((int)word, HIGH);
  return (__float_as_uint(f[0]) >> 16) | (__float_as_uint(f[1]) & 0xFFFF0000u);
}

// One block (4 waves) per (chunk of kChunkPages pages, kv-head j, candidate b) over the
// candidate's private pages. Each wave takes page pairs (32 tokens): S = K Q^T on the matrix
// cores (A = the K tile, 16 tokens x 32 dims; B = the g query heads as columns, in three bf16
// terms),
// online softmax per head in registers (a lane holds 4 tokens of one head per page), then
// O^T += V^T P^T (A = V^T rows of 16 dims x 32 tokens read straight from the dimension-major V
// tile, B = P^T hi and lo). The four waves merge through LDS and write one unnormalised partial
// (acc, m, l) per q-head. Slots at or beyond L_b are masked in S and zeroed in V (they may hold
// anything, NaN included).
template <int KVT, int D>
__global__ __launch_bounds__(256) void k_attn_mfma(const void *kpool, const void *vpool,
                                                   const float *kscale, const float *vscale,
                                                   int nkv, int g, const int32_t *page_table,
                                                   int max_pages, const int32_t *lengths,
                                                   GroupTable gt, int nch, const float *q,
                                                   float *apart, int nq) {
  constexpr int NKB = D / 32;  // 32-dim blocks of q.k
  constexpr int NDB = D / 16;  // 16-dim blocks of the output
  constexpr int EB = KVT == 1 ? 2 : 1;
  constexpr size_t TILE = (size_t)kPage * D * EB;
  __shared__ int phys_s[kChunkPages];
  __shared__ float ksc_s[kChunkPages], vsc_s[kChunkPages];
  __shared__ float red_m[4][16], red_l[4][16];
  __shared__ float red_acc[4][D][17];

  const int c = blockIdx.x, j = blockIdx.y, b = blockIdx.z;
  const int L = lengths[b];
  const int npages = (L + kPage - 1) / kPage;
  int first = 0;
  for (int gi = 0; gi < gt.n; ++gi)
    if (b >= gt.start[gi] && b < gt.start[gi + 1]) first = gt.prefix_pages[gi];
  const int p0 = first + c * kChunkPages;
  float *outbase = apart + (((size_t)b * nq + (size_t)j * g) * nch + c) * (D + 2);
  const size_t hstride = (size_t)nch * (D + 2);
  if (p0 >= npages) {
    for (int i = threadIdx.x; i < g * (D + 2); i += 256) {
      const int h = i / (D + 2), e = i - h * (D + 2);
      outbase[h * hstride + e] = (e == D) ? -INFINITY : 0.f;
    }
    return;
  }
  const int np = min(npages, p0 + kChunkPages) - p0;
  if (threadIdx.x < np) {
    const int ph = page_table[(size_t)b * max_pages + p0 + threadIdx.x];
    phys_s[threadIdx.x] = ph;
    if (KVT == 2) {
      ksc_s[threadIdx.x] = kscale[(size_t)ph * nkv + j];
      vsc_s[threadIdx.x] = vscale[(size_t)ph * nkv + j];
    }
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 15, cq = lane >> 4;

  // query operands of head n (zero columns for n >= g), split in three bf16 terms so that the
  // scores keep fp32-level accuracy even for very large logits
  uint4 qhi[NKB], qmd[NKB], qlo[NKB];
  {
    const float *qr = q + ((size_t)b * nq + (size_t)j * g + (n < g ? n : 0)) * D;
#pragma unroll
    for (int kk = 0; kk < NKB; ++kk) {
      uint32_t h[8], md[8], l[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        int dim;
        if (KVT == 1)
          dim = kk * 32 + 8 * cq + i;
        else
          dim = 16 * (4 * (kk >> 1) + cq) + 8 * (kk & 1) + i;
        const float v = (n < g) ? qr[dim] : 0.f;
        uint32_t rest;
        split_hi_lo(v, h[i], rest);
        split_hi_lo(v - __uint_as_float(h[i] << 16), md[i], l[i]);
      }
      qhi[kk] = make_uint4(pack2(h[0], h[1]), pack2(h[2], h[3]), pack2(h[4], h[5]), pack2(h[6], h[7]));
      qmd[kk] = make_uint4(pack2(md[0], md[1]), pack2(md[2], md[3]), pack2(md[4], md[5]),
                           pack2(md[6], md[7]));
      qlo[kk] = make_uint4(pack2(l[0], l[1]), pack2(l[2], l[3]), pack2(l[4], l[5]), pack2(l[6], l[7]));
    }
  }
  __syncthreads();

  const float rs = 1.0f / sqrtf((float)D);
  float m_run = -INFINITY, l_run = 0.f;
  floatx4 acc[NDB];
#pragma unroll
  for (int nb = 0; nb < NDB; ++nb) acc[nb] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int npairs = (np + 1) >> 1;
  for (int pp = wave; pp < npairs; pp += 4) {
    const int la = 2 * pp, lb = 2 * pp + 1;
    const bool hasB = lb < np;
    const int pa = phys_s[la];
    const int pb = hasB ? phys_s[lb] : pa;
    const char *kA = (const char *)kpool + ((size_t)pa * nkv + j) * TILE;
    const char *kB = (const char *)kpool + ((size_t)pb * nkv + j) * TILE;
    const char *vA = (const char *)vpool + ((size_t)pa * nkv + j) * TILE;
    const char *vB = (const char *)vpool + ((size_t)pb * nkv + j) * TILE;
    // ---- loads
    uint4 KA[NKB], KB[NKB];
    uint2 VA[NDB], VB[NDB];
    if (KVT == 1) {
#pragma unroll
      for (int kk = 0; kk < NKB; ++kk) {
        KA[kk] = *(const uint4 *)(kA + (size_t)(kk * 64 + lane) * 16);
        KB[kk] = *(const uint4 *)(kB + (size_t)(kk * 64 + lane) * 16);
      }
#pragma unroll
      for (int nb = 0; nb < NDB; ++nb) {
        VA[nb] = *(const uint2 *)(vA + (size_t)(nb * 16 + n) * 32 + cq * 8);
        VB[nb] = *(const uint2 *)(vB + (size_t)(nb * 16 + n) * 32 + cq * 8);
      }
    } else {
      uint4 ra[NKB / 2], rb[NKB / 2];
#pragma unroll
      for (int kp = 0; kp < NKB / 2; ++kp) {
        ra[kp] = *(const uint4 *)(kA + (size_t)(kp * 64 + lane) * 16);
        rb[kp] = *(const uint4 *)(kB + (size_t)(kp * 64 + lane) * 16);
      }
      uint32_t wa[NDB], wb[NDB];
#pragma unroll
      for (int nb = 0; nb < NDB; ++nb) {
        wa[nb] = *(const uint32_t *)(vA + (size_t)(nb * 16 + n) * 16 + cq * 4);
        wb[nb] = *(const uint32_t *)(vB + (size_t)(nb * 16 + n) * 16 + cq * 4);
      }
#pragma unroll
      for (int kp = 0; kp < NKB / 2; ++kp) {
        KA[2 * kp] = make_uint4(fp8x2_to_bf16x2<false>(ra[kp].x), fp8x2_to_bf16x2<true>(ra[kp].x),
                                fp8x2_to_bf16x2<false>(ra[kp].y), fp8x2_to_bf16x2<true>(ra[kp].y));
        KA[2 * kp + 1] = make_uint4(fp8x2_to_bf16x2<false>(ra[kp].z), fp8x2_to_bf16x2<true>(ra[kp].z),
                                    fp8x2_to_bf16x2<false>(ra[kp].w), fp8x2_to_bf16x2<true>(ra[kp].w));
        KB[2 * kp] = make_uint4(fp8x2_to_bf16x2<false>(rb[kp].x), fp8x2_to_bf16x2<true>(rb[kp].x),
                                fp8x2_to_bf16x2<false>(rb[kp].y), fp8x2_to_bf16x2<true>(rb[kp].y));
        KB[2 * kp + 1] = make_uint4(fp8x2_to_bf16x2<false>(rb[kp].z), fp8x2_to_bf16x2<true>(rb[kp].z),
                                    fp8x2_to_bf16x2<false>(rb[kp].w), fp8x2_to_bf16x2<true>(rb[kp].w));
      }
#pragma unroll
      for (int nb = 0; nb < NDB; ++nb) {
        VA[nb] = make_uint2(fp8x2_to_bf16x2<false>(wa[nb]), fp8x2_to_bf16x2<true>(wa[nb]));
        VB[nb] = make_uint2(fp8x2_to_bf16x2<false>(wb[nb]), fp8x2_to_bf16x2<true>(wb[nb]));
      }
    }
    // ---- scores: lane holds tokens 4cq + i of pages la and lb for head n
    floatx4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < NKB; ++kk) {
      sa = mfma16(KA[kk], qhi[kk], sa);
      sa = mfma16(KA[kk], qmd[kk], sa);
      sa = mfma16(KA[kk], qlo[kk], sa);
      sb = mfma16(KB[kk], qhi[kk], sb);
      sb = mfma16(KB[kk], qmd[kk], sb);
      sb = mfma16(KB[kk], qlo[kk], sb);
    }
    const float sca = (KVT == 2) ? ksc_s[la] * rs : rs;
    const float scb = (KVT == 2) ? ksc_s[hasB ? lb : la] * rs : rs;
    const int ta = (p0 + la) * kPage + 4 * cq, tb = (p0 + lb) * kPage + 4 * cq;
    float s[8];
    bool ok[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ok[i] = ta + i < L;
      ok[4 + i] = hasB && (tb + i < L);
      s[i] = ok[i] ? sa[i] * sca : -INFINITY;
      s[4 + i] = ok[4 + i] ? sb[i] * scb : -INFINITY;
    }
    float mx = s[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) mx = fmaxf(mx, s[i]);
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);  // finite: token 0 of page la is always valid
    const float alpha = expf(m_run - m_new);
    m_run = m_new;
    float pv[8], psum = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      pv[i] = ok[i] ? expf(s[i] - m_new) : 0.f;
      psum += pv[i];
    }
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int nb = 0; nb < NDB; ++nb) {
      acc[nb][0] *= alpha;
      acc[nb][1] *= alpha;
      acc[nb][2] *= alpha;
      acc[nb][3] *= alpha;
    }
    if (KVT == 2) {
      const float va_s = vsc_s[la], vb_s = vsc_s[hasB ? lb : la];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pv[i] *= va_s;
        pv[4 + i] *= vb_s;
      }
    }
    uint32_t ph[8], pl[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) split_hi_lo(pv[i], ph[i], pl[i]);
    const uint4 Phi = make_uint4(pack2(ph[0], ph[1]), pack2(ph[2], ph[3]), pack2(ph[4], ph[5]),
                                 pack2(ph[6], ph[7]));
    const uint4 Plo = make_uint4(pack2(pl[0], pl[1]), pack2(pl[2], pl[3]), pack2(pl[4], pl[5]),
                                 pack2(pl[6], pl[7]));
    // zero V entries of masked tokens (their slots may hold NaN)
    const uint32_t ma0 = (ok[0] ? 0xFFFFu : 0u) | (ok[1] ? 0xFFFF0000u : 0u);
    const uint32_t ma1 = (ok[2] ? 0xFFFFu : 0u) | (ok[3] ? 0xFFFF0000u : 0u);
    const uint32_t mb0 = (ok[4] ? 0xFFFFu : 0u) | (ok[5] ? 0xFFFF0000u : 0u);
    const uint32_t mb1 = (ok[6] ? 0xFFFFu : 0u) | (ok[7] ? 0xFFFF0000u : 0u);
#pragma unroll
    for (int nb = 0; nb < NDB; ++nb) {
      const uint4 vop = make_uint4(VA[nb].x & ma0, VA[nb].y & ma1, VB[nb].x & mb0, VB[nb].y & mb1);
      acc[nb] = mfma16(vop, Phi, acc[nb]);
      acc[nb] = mfma16(vop, Plo, acc[nb]);
    }
  }
  // ---- merge the four waves
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  if (lane < 16) {
    red_m[wave][n] = m_run;
    red_l[wave][n] = l_run;
  }
#pragma unroll
  for (int nb = 0; nb < NDB; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i) red_acc[wave][nb * 16 + 4 * cq + i][n] = acc[nb][i];
  __syncthreads();
  for (int e = threadIdx.x; e < g * D; e += 256) {
    const int h = e / D, d = e - h * D;
    float M = red_m[0][h];
#pragma unroll
    for (int w = 1; w < 4; ++w) M = fmaxf(M, red_m[w][h]);
    float a = 0.f, l = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float f = (red_m[w][h] == -INFINITY) ? 0.f : expf(red_m[w][h] - M);
      a += f * red_acc[w][d][h];
      l += f * red_l[w][h];
    }
    outbase[h * hstride + d] = a;
    if (d == 0) {
      outbase[h * hstride + D] = M;
      outbase[h * hstride + D + 1] = l;
    }
  }
}

hipError_t launch_attn_mfma(const Dims &dm, const Plan &p, const char *kp, const char *vp,
                            const float *ksc, const float *vsc, const int32_t *page_table,
                            const int32_t *lengths, const GroupTable &gt, const float *q,
                            float *apart, hipStream_t s) {
  dim3 grid(p.nch, dm.nkv, p.B);
#define KVPRM_ATTM(KVT, D)                                                                   \
  hipLaunchKernelGGL((k_attn_mfma<KVT, D>), grid, dim3(256), 0, s, kp, vp, ksc, vsc, dm.nkv, \
                     dm.g, page_table, p.max_pages, lengths, gt, p.nch, q, apart, dm.nq)
  if (dm.kvdt == 1) {
    if (dm.d == 64) KVPRM_ATTM(1, 64);
    else KVPRM_ATTM(1, 128);
  } else {
    if (dm.d == 64) KVPRM_ATTM(2, 64);
    else KVPRM_ATTM(2, 128);
  }
#undef KVPRM_ATTM
  return hipGetLastError();
}

}  // namespace kvprm
