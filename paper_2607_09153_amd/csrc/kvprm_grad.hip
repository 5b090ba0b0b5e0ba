// Backward pass of the verify-token readout with respect to the key/value cache (gfx950), for
// KV Steering (appendix: gradient steps on the cache that lower -log P(+)).
//
// The forward pass (the matrix-core pipeline) saves, per layer, the residual stream entering
// the layer and after the attention block, q / k_self / v_self of the verify token, the
// attention output o and the log-sum-exp of every head's softmax (the token's own key
// included), and the gate / up pre-activations. Then, from the reward head back to layer 0:
//
//   head:       dz = sigmoid(z) - 1, through the final RMSNorm            -> dx
//   FFN:        dh = W_down^T dx; SwiGLU derivative -> (d gate, d up);
//               du2 = [W_gate; W_up]^T (d gate, d up); RMSNorm backward    -> dx_mid
//   attention:  do = W_o^T dx_mid; per cached token t and head h of kv-head j:
//               p = exp(q.K_t / sqrt(d) - lse_h), ds = p (do_h.V_t - do_h.o_h),
//               dK_t = sum_h ds q_h / sqrt(d), dV_t = sum_h p do_h, dq_h += ds K_t / sqrt(d);
//               the same for the token's own key; rotary backward;
//               du1 = [W_q; W_k; W_v]^T (dq, dk, dv); RMSNorm backward  -> dx_in
//
// The transposed products read the packed bf16 weight tiles once and run on the matrix cores
// (each tile turned around by a product with a 0/1 selector, then contracted with d in bf16
// hi + lo terms). All reductions have a fixed order.
#include <math.h>
#include <string.h>

#include "kvprm_internal.h"

namespace kvprm {

namespace {

__device__ __forceinline__ float bf(uint32_t h) { return __uint_as_float(h << 16); }

__device__ __forceinline__ float ldw(const void *p, size_t i) {
  return bf(((const uint16_t *)p)[i]);
}

__device__ __forceinline__ uint16_t bf16_round(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// sum over the N lanes of an aligned N-lane group (N a power of two <= 64)
template <int N>
__device__ __forceinline__ float sum_lanes(float v) {
#pragma unroll
  for (int off = N / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Sum over a block of NTHR threads (multiple of 64); every thread gets the result.
template <int NTHR>
__device__ __forceinline__ float block_sum(float v, float *red) {
  v = wave_sum(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int w = 0; w < NTHR / 64; ++w) s += red[w];
  return s;
}

__device__ __forceinline__ uint4 ld_nt(const uint4 *p) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 v = __builtin_nontemporal_load((const u32x4 *)p);
  return make_uint4(v.x, v.y, v.z, v.w);
}

constexpr float kLog2e = 1.4426950408889634f;

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short shortx4 __attribute__((ext_vector_type(4)));

// Matrix-core products (lane l, c = l / 16, n = l % 16; D = accumulator):
//   16x16x32: A lane holds row n, reduction slots 8c .. 8c+7; B lane holds column n, the same
//             slots; D lane holds rows 4c .. 4c+3 of column n
//   16x16x16: as above with reduction slots 4c .. 4c+3
// Any assignment of the contracted index to slots works if A and B use the same one.
__device__ __forceinline__ floatx4 mma32(const uint4 &a, const uint4 &b, const floatx4 &c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
__device__ __forceinline__ floatx4 mma16(const uint2 &a, const uint2 &b, const floatx4 &c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(shortx4, a),
                                                   __builtin_bit_cast(shortx4, b), c, 0, 0, 0);
}

// x = hi + lo with hi, lo bf16 (nearest-even each): hi * y + lo * y keeps ~16 bits of x
__device__ __forceinline__ void split_bf16(float x, uint32_t &hi, uint32_t &lo) {
  hi = bf16_round(x);
  lo = bf16_round(x - bf(hi));
}

}  // namespace

// ------------------------------------------------------------------------------- head, norms

// Reward head backward for one candidate per block: z = w_r . (x r gamma) + b_r with
// r = 1/sqrt(mean(x^2) + eps); the loss -log sigmoid(z) has dz = sigmoid(z) - 1, and
// dx = dz (r gamma w_r - (r^3 / H) x sum_i gamma_i w_r,i x_i).
__global__ __launch_bounds__(256) void k_head_bwd(const float *x, const void *gam, const void *wr,
                                                  float rb, int H, float eps, float *dx,
                                                  float *dxT, int B) {
  __shared__ float red[4];
  const int b = blockIdx.x;
  const float *xb = x + (size_t)b * H;
  float sq = 0.f, dot = 0.f;
  for (int i = threadIdx.x; i < H; i += 256) {
    const float v = xb[i];
    sq += v * v;
    dot += v * ldw(gam, i) * ldw(wr, i);
  }
  sq = block_sum<256>(sq, red);
  dot = block_sum<256>(dot, red);
  const float r = 1.0f / sqrtf(sq / (float)H + eps);
  const float z = dot * r + rb;
  const float dz = 1.0f / (1.0f + expf(-z)) - 1.0f;
  const float c = r * r * r / (float)H * dot;
  for (int i = threadIdx.x; i < H; i += 256) {
    const float v = dz * (r * ldw(gam, i) * ldw(wr, i) - c * xb[i]);
    dx[(size_t)b * H + i] = v;
    dxT[(size_t)i * kDPad + b] = v;
  }
}

// RMSNorm backward plus the residual path, one candidate per block:
// out = res + r (gamma dy) - (r^3 / H) x sum_i gamma_i dy_i x_i (out may be res), also written
// transposed to outT [H][kDPad]. Each thread keeps its inputs in registers between the two
// passes (H <= kGradMaxHidden).
constexpr int kRmsPer = kGradMaxHidden / 1024;
__global__ __launch_bounds__(1024) void k_rms_bwd(const float *x, const void *gam, const float *dy,
                                                  const float *res, float *out, float *outT, int B,
                                                  int H, float eps) {
  __shared__ float red[16];
  const int b = blockIdx.x;
  const size_t o = (size_t)b * H;
  float xv[kRmsPer], gd[kRmsPer];
  float sq = 0.f, dot = 0.f;
#pragma unroll
  for (int k = 0; k < kRmsPer; ++k) {
    const int i = threadIdx.x + k * 1024;
    xv[k] = i < H ? x[o + i] : 0.f;
    gd[k] = i < H ? ldw(gam, i) * dy[o + i] : 0.f;
  }
#pragma unroll
  for (int k = 0; k < kRmsPer; ++k) {
    sq += xv[k] * xv[k];
    dot += gd[k] * xv[k];
  }
  sq = block_sum<1024>(sq, red);
  dot = block_sum<1024>(dot, red);
  const float r = 1.0f / sqrtf(sq / (float)H + eps);
  const float c = r * r * r / (float)H * dot;
#pragma unroll
  for (int k = 0; k < kRmsPer; ++k) {
    const int i = threadIdx.x + k * 1024;
    if (i < H) {
      const float v = res[o + i] + r * gd[k] - c * xv[k];
      out[o + i] = v;
      outT[(size_t)i * kDPad + b] = v;
    }
  }
}

// ------------------------------------------------------------------------------- W^T d

// y[b][k] = sum over the stacked rows r of W[r][k] d[r][b] for packed bf16 matrices (1 KiB
// blocks, block kb * (rows_i / 16) + t, lane l holding W[16 t + l % 16][32 kb + 8 (l / 16) + i]).
// Block = 4 waves on 4 consecutive 32-input blocks kb of one row split (kTgemvWindow tiles at
// most); the split's d rows are staged once in LDS, and each wave streams the contiguous weight
// blocks of its kb with two batches of U tiles in flight. Partials: part[split][b][k].
struct TgemvArgs {
  const void *w[3];
  int seg_tiles[3];  // row tiles of each segment
  int nseg;
  int K;             // inputs (columns) of every segment
  const float *d;    // [stacked rows][kDPad] (columns >= B ignored)
  int B;
  int tiles, tps, nsplit;  // stacked row tiles, tiles per split, splits
  float *part;       // [nsplit][B][K]
};

// The product runs on the matrix cores. Its contraction runs over rows while a tile lane holds
// 8 inputs of one row, so each tile is first turned around by a product with a 0/1 selector:
// S_h[k][n] = 1 where k = 16 h + n gives D[r][n] = W[r][16 h + n] exactly (one bf16 weight
// times 1 per output), with lane (n, c) holding rows 4c .. 4c+3 of input 16 h + n, which is the
// B operand of a 16x16x16 product over the tile's 16 rows. Its A operand holds d, staged once
// per split in LDS in that layout: slot m < 8 the hi bf16 term of candidate m's d, slot 8 + m
// the lo term (zero for candidates past B and for tiles past the split), so the tile costs four
// matrix-core products instead of 64 FMAs per lane. The accumulator lane (n, c) holds slots
// 4c .. 4c+3 of input 16 h + n; a candidate's hi and lo sums (lanes c and c + 2) are added at the
// end.
template <int U>
__global__ __launch_bounds__(256) void k_tgemv_mx(TgemvArgs a) {
  constexpr int NT = kTgemvWindow + 2 * U;  // staged tiles (the last 2U only ever zero)
  __shared__ uint2 dop_s[NT][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nkb = a.K >> 5;
  const int bps = (nkb + 3) >> 2;  // blocks per split
  const int split = blockIdx.x / bps;
  const int kb = (blockIdx.x - split * bps) * 4 + w;
  const bool act = kb < nkb;  // wave-uniform
  const int n = lane & 15, c = lane >> 4;
  const int t0 = split * a.tps, t1 = min(a.tiles, t0 + a.tps);
  const int cum1 = a.nseg > 1 ? a.seg_tiles[0] : a.tiles;
  const int cum2 = a.nseg > 2 ? a.seg_tiles[0] + a.seg_tiles[1] : a.tiles;
  auto load = [&](int t, uint4 *wv) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int tt = min(t + u, t1 - 1);  // past the end: repeat the last tile (its d is zero)
      const int sg = tt >= cum2 ? 2 : (tt >= cum1 ? 1 : 0);
      const int base = sg == 0 ? 0 : (sg == 1 ? cum1 : cum2);
      wv[u] = ld_nt((const uint4 *)a.w[sg] + ((size_t)kb * a.seg_tiles[sg] + (tt - base)) * 64 + lane);
    }
  };
  uint4 wa[U], wb[U];
  if (act) load(t0, wa);  // in flight while d is staged
  // staging: item (tile tl, row group q) reads rows 16 (t0 + tl) + 4q .. + 3 and writes the hi
  // and lo operands of every candidate for lanes 16 q + m and 16 q + 8 + m
  for (int it = threadIdx.x; it < NT * 4; it += 256) {
    const int tl = it >> 2, q = it & 3;
    float dv[4][8];
    const bool live = tl < t1 - t0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float4 v0 = make_float4(0.f, 0.f, 0.f, 0.f), v1 = v0;
      if (live) {
        const float4 *dr = (const float4 *)(a.d + ((size_t)(t0 + tl) * 16 + 4 * q + i) * kDPad);
        v0 = dr[0];
        v1 = dr[1];
      }
      dv[i][0] = v0.x; dv[i][1] = v0.y; dv[i][2] = v0.z; dv[i][3] = v0.w;
      dv[i][4] = v1.x; dv[i][5] = v1.y; dv[i][6] = v1.z; dv[i][7] = v1.w;
    }
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      uint32_t hi[4], lo[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float v = m < a.B ? dv[i][m] : 0.f;
        hi[i] = bf16_round(v);
        lo[i] = bf16_round(v - bf(hi[i]));
      }
      dop_s[tl][16 * q + m] = make_uint2(hi[0] | (hi[1] << 16), hi[2] | (hi[3] << 16));
      dop_s[tl][16 * q + 8 + m] = make_uint2(lo[0] | (lo[1] << 16), lo[2] | (lo[3] << 16));
    }
  }
  __syncthreads();
  if (!act) return;
  // selector operands: B lane (n, c) holds slots 8c .. 8c+7 of column n; 1.0 where 8c + i = 16 h + n
  uint4 sel[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    uint32_t wd[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t e0 = (8 * c + 2 * j == 16 * h + n) ? 0x3F80u : 0u;
      const uint32_t e1 = (8 * c + 2 * j + 1 == 16 * h + n) ? 0x3F80u : 0u;
      wd[j] = e0 | (e1 << 16);
    }
    sel[h] = make_uint4(wd[0], wd[1], wd[2], wd[3]);
  }
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
  floatx4 acc[2] = {zero, zero};
  auto comp = [&](int t, const uint4 *wv) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint2 aop = dop_s[t + u - t0][lane];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const floatx4 tr = mma32(wv[u], sel[h], zero);  // exact: one weight per output
        const uint2 bop = make_uint2((__float_as_uint(tr[0]) >> 16) | (__float_as_uint(tr[1]) & 0xFFFF0000u),
                                     (__float_as_uint(tr[2]) >> 16) | (__float_as_uint(tr[3]) & 0xFFFF0000u));
        acc[h] = mma16(aop, bop, acc[h]);
      }
    }
  };
  for (int t = t0; t < t1; t += 2 * U) {
    load(t + U, wb);
    __builtin_amdgcn_sched_barrier(0);
    comp(t, wa);
    __builtin_amdgcn_sched_barrier(0);
    load(t + 2 * U, wa);
    __builtin_amdgcn_sched_barrier(0);
    comp(t + U, wb);
    __builtin_amdgcn_sched_barrier(0);
  }
  // hi + lo of candidate 4c + i (c < 2) from lanes c and c + 2
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[h][i] += __shfl_xor(acc[h][i], 32, 64);
  if (c < 2) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int b = 4 * c + i;
      if (b < a.B) {
        float *dst = a.part + ((size_t)split * a.B + b) * a.K + kb * 32 + n;
        dst[0] = acc[0][i];
        dst[16] = acc[1][i];
      }
    }
  }
}

// Sum of the splits, in split order: y[b][k] = sum_s part[s][b][k]. With SWIGLU the sum is the
// gradient dh of the SwiGLU output h = silu(a) c (a, c the saved gate / up pre-activations,
// gu[b][0..F) and gu[b][F..2F)), and the kernel writes the stacked d vector of the gate/up
// products: out[f][b] = dh c silu'(a), out[F + f][b] = dh silu(a) (rows of kDPad columns).
template <bool SWIGLU>
__global__ __launch_bounds__(256) void k_tgemv_sum(const float *part, int nsplit, int B, int K,
                                                   const float *gu, float *out) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= B * K) return;
  float s = 0.f;
  for (int i = 0; i < nsplit; ++i) s += part[(size_t)i * B * K + e];
  if (!SWIGLU) {
    out[e] = s;
    return;
  }
  const int b = e / K, f = e - b * K;
  const float av = gu[(size_t)b * 2 * K + f], cv = gu[(size_t)b * 2 * K + K + f];
  const float sg = 1.0f / (1.0f + expf(-av));
  const float silu = av * sg;
  const float dsilu = sg * (1.0f + av * (1.0f - sg));
  out[(size_t)f * kDPad + b] = s * cv * dsilu;
  out[(size_t)(K + f) * kDPad + b] = s * silu;
}

// ------------------------------------------------------------------------------- attention

// The verify token's own key, per (candidate, kv-head j): for the g heads h of j,
// Dh = do_h . o_h, p = exp(q_h . k_self / sqrt(d) - lse_h), ds = p (do_h . v_self - Dh);
// dk_self = sum_h ds q_h / sqrt(d), dv_self = sum_h p do_h, dq_h = ds k_self / sqrt(d).
// One thread per dimension.
template <int D>
__global__ __launch_bounds__(D) void k_attn_bwd_self(const float *q, const float *ks,
                                                     const float *vs, const float *o,
                                                     const float *lse, const float *dout, int nq,
                                                     int nkv, float *Dh, float *dq_self,
                                                     float *dk_self, float *dv_self) {
  __shared__ float red[D / 64];
  const int b = blockIdx.x, j = blockIdx.y, m = threadIdx.x;
  const int g = nq / nkv;
  const float sc = 1.0f / sqrtf((float)D);
  const float kv = ks[((size_t)b * nkv + j) * D + m], vv = vs[((size_t)b * nkv + j) * D + m];
  float dk = 0.f, dv = 0.f;
  for (int hh = 0; hh < g; ++hh) {
    const int h = j * g + hh;
    const size_t r = ((size_t)b * nq + h) * D + m;
    const float qv = q[r], dov = dout[r];
    const float Dv = block_sum<D>(dov * o[r], red);
    const float s = block_sum<D>(qv * kv, red) * sc;
    const float dp = block_sum<D>(dov * vv, red);
    const float p = expf(s - lse[(size_t)b * nq + h]);
    const float ds = p * (dp - Dv);
    dk += ds * qv * sc;
    dv += p * dov;
    dq_self[r] = ds * kv * sc;
    if (m == 0) Dh[(size_t)b * nq + h] = Dv;
  }
  dk_self[((size_t)b * nkv + j) * D + m] = dk;
  dv_self[((size_t)b * nkv + j) * D + m] = dv;
}

struct AttnBwdArgs {
  char *kp, *vp;               // this layer's pools (bf16), updated in place when steering
  float *gk, *gv;              // this layer's gradient pools (fp32, pool element order) or null
  float eta;                   // steering step (in place) when gk is null
  const int32_t *page_table;
  int max_pages;
  const int32_t *lengths;
  int nkv, nq, CP, nch;        // chunk length in pages, chunk slots per (candidate, head)
  const float *q, *dout, *lse, *Dh;  // [B][nq][D], [B][nq][D], [B][nq], [B][nq]
  float *dq_part;              // [B][nq][nch][D]
};

// Attention backward over the cache on the matrix cores (bf16 cache). Block = W waves of one
// (candidate b, kv-head j); wave w walks the CP pages of chunk W x + w of b. Per page of 16
// cached tokens, with the g q-heads of j as the other side of every product (padded to 16):
//   S^T = Q K^T              16x16x32 over the dims (A = q in three bf16 terms, B = the K tile
//                            as loaded)
//   dP^T = dO V^T            over the dims (B = the V tile read back from LDS token-major)
//   P = exp(S / sqrt(d) - lse), dS = P (dP - D)      lane = token, its 4 heads in registers
//   dV = P dO                16x16x16 over the heads: a lane ends with 4 consecutive slots of
//                            two dims, i.e. its own 16 bytes of the V tile
//   dK^T = (q / sqrt(d))^T dS^T   over the heads: 4 consecutive dims of one token per lane
//   dQ += dS^T K             over the tokens (dS transposed and K read dims-major through LDS)
// fp32 operands enter as bf16 hi + lo. The q / dO operands with the heads as the reduction index
// are built once per block in LDS. Slots at or beyond L get zero gradient (their stored values
// may be anything, NaN included, and are masked before every product that mixes tokens).
template <int D, int W>
__global__ __launch_bounds__(64 * W) void k_attn_bwd_mx(AttnBwdArgs a) {
  constexpr int NKB = D / 32, NDB = D / 16;
  constexpr int TILE = kPage * D;  // elements of a tile
  constexpr int TL = TILE / 512;   // 16-byte pieces of a tile per lane (= NKB)
  constexpr int DST = 20;          // row stride (elements) of the dS transpose
  static_assert(TL == NKB, "tile pieces per lane");
  __shared__ uint4 qT_s[NDB][64];            // lane (dim 16 nb + n, c): heads 4c.. of q / sqrt(d), hi.xy lo.zw
  __shared__ uint4 dO_s[NDB][64];            // the same for dO
  __shared__ uint4 qa_s[3][NKB][64];         // lane (head n, c): dims 32 kk + 8c .. of q, three terms
  __shared__ uint4 oa_s[2][NKB][64];         // the same for dO, two terms
  __shared__ uint4 kt_s[W][TL * 64];         // the page's K tile as stored
  __shared__ uint4 vt_s[W][TL * 64];         // the page's V tile as stored
  __shared__ uint16_t ds_s[W][2][16 * DST];  // dS^T hi, lo: [head][token]
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int n = lane & 15, c = lane >> 4;
  const int b = blockIdx.y, j = blockIdx.z;
  const int nq = a.nq, g = nq / a.nkv;
  const int L = a.lengths[b];
  const int npages = (L + kPage - 1) / kPage;
  if ((int)blockIdx.x * W * a.CP >= npages) return;  // the whole block
  const float sc = 1.0f / sqrtf((float)D);
  const size_t hb = (size_t)b * nq + (size_t)j * g;  // row of the first q-head of kv-head j
  for (int e = threadIdx.x; e < NDB * 64; e += 64 * W) {
    const int nb = e >> 6, ln = e & 63;
    const int m = 16 * nb + (ln & 15), c4 = 4 * (ln >> 4);
    uint32_t qh[4], ql[4], oh[4], ol[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool hv = c4 + i < g;
      const size_t r = (hb + (hv ? c4 + i : 0)) * D + m;
      split_bf16(hv ? a.q[r] * sc : 0.f, qh[i], ql[i]);
      split_bf16(hv ? a.dout[r] : 0.f, oh[i], ol[i]);
    }
    qT_s[nb][ln] = make_uint4(qh[0] | qh[1] << 16, qh[2] | qh[3] << 16, ql[0] | ql[1] << 16,
                              ql[2] | ql[3] << 16);
    dO_s[nb][ln] = make_uint4(oh[0] | oh[1] << 16, oh[2] | oh[3] << 16, ol[0] | ol[1] << 16,
                              ol[2] | ol[3] << 16);
  }
  // q (three terms) and dO (two) with the dims as reduction index, lane = head n
  for (int e = threadIdx.x; e < NKB * 64; e += 64 * W) {
    const int kk = e >> 6, ln = e & 63, hn = ln & 15, c8 = 8 * (ln >> 4);
    const bool hv = hn < g;
    const float *qr = a.q + (hb + (hv ? hn : 0)) * D + 32 * kk + c8;
    const float *orow = a.dout + (hb + (hv ? hn : 0)) * D + 32 * kk + c8;
    uint32_t h[8], md[8], lo[8], oh[8], ol[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float qv = hv ? qr[i] : 0.f;
      uint32_t rest;
      split_bf16(qv, h[i], rest);
      split_bf16(qv - bf(h[i]), md[i], lo[i]);
      split_bf16(hv ? orow[i] : 0.f, oh[i], ol[i]);
    }
    qa_s[0][kk][ln] = make_uint4(h[0] | h[1] << 16, h[2] | h[3] << 16, h[4] | h[5] << 16, h[6] | h[7] << 16);
    qa_s[1][kk][ln] = make_uint4(md[0] | md[1] << 16, md[2] | md[3] << 16, md[4] | md[5] << 16,
                                 md[6] | md[7] << 16);
    qa_s[2][kk][ln] = make_uint4(lo[0] | lo[1] << 16, lo[2] | lo[3] << 16, lo[4] | lo[5] << 16,
                                 lo[6] | lo[7] << 16);
    oa_s[0][kk][ln] = make_uint4(oh[0] | oh[1] << 16, oh[2] | oh[3] << 16, oh[4] | oh[5] << 16,
                                 oh[6] | oh[7] << 16);
    oa_s[1][kk][ln] = make_uint4(ol[0] | ol[1] << 16, ol[2] | ol[3] << 16, ol[4] | ol[5] << 16,
                                 ol[6] | ol[7] << 16);
  }
  float lse2[4], Dh4[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int h = 4 * c + i;
    lse2[i] = h < g ? a.lse[hb + h] * kLog2e : 0.f;
    Dh4[i] = h < g ? a.Dh[hb + h] : 0.f;
  }
  floatx4 dq[NDB];
#pragma unroll
  for (int nb = 0; nb < NDB; ++nb) dq[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
  __syncthreads();  // block operands ready; no other barrier below (every LDS region after this
                    // is private to one wave, whose LDS accesses execute in program order)
  const int chunk = blockIdx.x * W + wv;
  const int pw0 = chunk * a.CP, pw1 = min(npages, pw0 + a.CP);
  if (pw0 >= pw1) return;
  uint4 *ks = kt_s[wv], *vs = vt_s[wv];
  const uint16_t *ks16 = (const uint16_t *)ks, *vs16 = (const uint16_t *)vs;
  uint16_t *dsh = ds_s[wv][0], *dsl = ds_s[wv][1];
  const float rs2 = kLog2e * sc;
  const int32_t *prow = a.page_table + (size_t)b * a.max_pages;
  const uint4 *kp4 = (const uint4 *)a.kp, *vp4 = (const uint4 *)a.vp;
  size_t toff = ((size_t)prow[pw0] * a.nkv + j) * TILE;  // element offset of the next tile
  uint4 kn[TL], vn[TL];
#pragma unroll
  for (int t = 0; t < TL; ++t) {
    kn[t] = ld_nt(kp4 + toff / 8 + t * 64 + lane);
    vn[t] = ld_nt(vp4 + toff / 8 + t * 64 + lane);
  }
  for (int pi = pw0; pi < pw1; ++pi) {
    const size_t tcur = toff;
    uint4 kr[TL], vr[TL];
#pragma unroll
    for (int t = 0; t < TL; ++t) {
      kr[t] = kn[t];
      vr[t] = vn[t];
    }
    if (pi + 1 < pw1) {  // the next page's tiles are in flight while this one is computed
      toff = ((size_t)prow[pi + 1] * a.nkv + j) * TILE;
#pragma unroll
      for (int t = 0; t < TL; ++t) {
        kn[t] = ld_nt(kp4 + toff / 8 + t * 64 + lane);
        vn[t] = ld_nt(vp4 + toff / 8 + t * 64 + lane);
      }
    }
#pragma unroll
    for (int t = 0; t < TL; ++t) {
      ks[t * 64 + lane] = kr[t];
      vs[t * 64 + lane] = vr[t];
    }
    // S^T and dP^T: lane = token n of the page, rows = heads 4c .. 4c+3
    floatx4 st = {0.f, 0.f, 0.f, 0.f}, dpt = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < NKB; ++kk) {
      st = mma32(qa_s[0][kk][lane], kr[kk], st);
      st = mma32(qa_s[1][kk][lane], kr[kk], st);
      st = mma32(qa_s[2][kk][lane], kr[kk], st);
    }
#pragma unroll
    for (int kk = 0; kk < NKB; ++kk) {
      // V element (slot n, dim m) of the stored tile (bf16: x = 8, r = 2)
      uint32_t e[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int m = 32 * kk + 8 * c + i;
        e[i] = vs16[((((m >> 5) * 4 + (n >> 2)) * 16 + (m & 15)) * 2 + ((m >> 4) & 1)) * 4 + (n & 3)];
      }
      const uint4 vb = make_uint4(e[0] | e[1] << 16, e[2] | e[3] << 16, e[4] | e[5] << 16,
                                  e[6] | e[7] << 16);
      dpt = mma32(oa_s[0][kk][lane], vb, dpt);
      dpt = mma32(oa_s[1][kk][lane], vb, dpt);
    }
    const int t0 = pi * kPage;
    const bool tv = t0 + n < L;
    uint32_t ph[4], pl[4], sh[4], sl[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool ok = tv && 4 * c + i < g;
      const float p = ok ? __builtin_amdgcn_exp2f(st[i] * rs2 - lse2[i]) : 0.f;
      const float ds = ok ? p * (dpt[i] - Dh4[i]) : 0.f;
      split_bf16(p, ph[i], pl[i]);
      split_bf16(ds, sh[i], sl[i]);
      dsh[(4 * c + i) * DST + n] = (uint16_t)sh[i];
      dsl[(4 * c + i) * DST + n] = (uint16_t)sl[i];
    }
    const uint2 Ph = make_uint2(ph[0] | ph[1] << 16, ph[2] | ph[3] << 16);
    const uint2 Pl = make_uint2(pl[0] | pl[1] << 16, pl[2] | pl[3] << 16);
    const uint2 Sh = make_uint2(sh[0] | sh[1] << 16, sh[2] | sh[3] << 16);
    const uint2 Sl = make_uint2(sl[0] | sl[1] << 16, sl[2] | sl[3] << 16);
    // dV, two 16-dim blocks at a time: lane = dim 16 nb + n, rows = slots 4c .. 4c+3, which is
    // the lane's own 16-byte piece t of the V tile
#pragma unroll
    for (int t = 0; t < TL; ++t) {
      floatx4 dv[2];
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const uint4 ob = dO_s[2 * t + r][lane];
        const uint2 oh = make_uint2(ob.x, ob.y), ol = make_uint2(ob.z, ob.w);
        floatx4 v = {0.f, 0.f, 0.f, 0.f};
        v = mma16(Ph, oh, v);
        v = mma16(Ph, ol, v);
        v = mma16(Pl, oh, v);
        dv[r] = v;
      }
      if (a.gk) {
        float *gv = a.gv + tcur + (size_t)(t * 64 + lane) * 8;
        *(float4 *)gv = make_float4(dv[0][0], dv[0][1], dv[0][2], dv[0][3]);
        *(float4 *)(gv + 4) = make_float4(dv[1][0], dv[1][1], dv[1][2], dv[1][3]);
      } else {
        const uint32_t w[4] = {vr[t].x, vr[t].y, vr[t].z, vr[t].w};
        uint32_t nw[4];
#pragma unroll
        for (int q2 = 0; q2 < 4; ++q2) {
          uint32_t out = 0;
#pragma unroll
          for (int hb2 = 0; hb2 < 2; ++hb2) {
            const int i = (q2 & 1) * 2 + hb2;  // slot 4c + i, dim block r = q2 / 2
            const uint32_t old16 = (w[q2] >> (16 * hb2)) & 0xFFFFu;
            const uint32_t new16 =
                t0 + 4 * c + i < L ? bf16_round(bf(old16) - a.eta * dv[q2 >> 1][i]) : old16;
            out |= new16 << (16 * hb2);
          }
          nw[q2] = out;
        }
        ((uint4 *)((uint16_t *)a.vp + tcur))[t * 64 + lane] = make_uint4(nw[0], nw[1], nw[2], nw[3]);
      }
    }
    // dK^T: lane = token n, rows = dims 16 nb + 4c .. +3 (half of a 16-byte group of the K tile)
#pragma unroll
    for (int nb = 0; nb < NDB; ++nb) {
      const uint4 qb = qT_s[nb][lane];
      const uint2 qh = make_uint2(qb.x, qb.y), ql = make_uint2(qb.z, qb.w);
      floatx4 k = {0.f, 0.f, 0.f, 0.f};
      k = mma16(qh, Sh, k);
      k = mma16(qh, Sl, k);
      k = mma16(ql, Sh, k);
      const int m = 16 * nb + 4 * c;
      const int idx = ((m >> 3) * 16 + n) * 8 + (m & 7);
      if (a.gk) {
        *(float4 *)(a.gk + tcur + idx) = make_float4(k[0], k[1], k[2], k[3]);
      } else if (tv) {
        const uint2 old = *(const uint2 *)(ks16 + idx);
        const uint32_t o4[4] = {old.x & 0xFFFFu, old.x >> 16, old.y & 0xFFFFu, old.y >> 16};
        uint32_t nv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) nv[i] = bf16_round(bf(o4[i]) - a.eta * k[i]);
        *(uint2 *)((uint16_t *)a.kp + tcur + idx) = make_uint2(nv[0] | nv[1] << 16, nv[2] | nv[3] << 16);
      }
    }
    // dQ += dS^T K: A = dS^T (lane = head n, slots = tokens 4c .. 4c+3), B = K (lane = dim
    // 16 nb + n, the same tokens; slots past L zeroed)
    const uint2 Ah = *(const uint2 *)(dsh + n * DST + 4 * c);
    const uint2 Al = *(const uint2 *)(dsl + n * DST + 4 * c);
#pragma unroll
    for (int nb = 0; nb < NDB; ++nb) {
      const int m = 16 * nb + n;
      uint32_t kv4[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int s2 = 4 * c + i;
        const uint32_t v = ks16[((m >> 3) * 16 + s2) * 8 + (m & 7)];
        kv4[i] = t0 + s2 < L ? v : 0u;
      }
      const uint2 kb = make_uint2(kv4[0] | kv4[1] << 16, kv4[2] | kv4[3] << 16);
      dq[nb] = mma16(Ah, kb, dq[nb]);
      dq[nb] = mma16(Al, kb, dq[nb]);
    }
  }
  // this chunk's dq partial: lane = dim 16 nb + n, rows = heads 4c .. 4c+3
#pragma unroll
  for (int nb = 0; nb < NDB; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (4 * c + i < g)
        a.dq_part[((hb + 4 * c + i) * a.nch + chunk) * D + 16 * nb + n] = dq[nb][i] * sc;
}

// dq of every head (the own-key term, then the chunk partials: four groups of consecutive
// chunks, each added in order by its own threads, the groups in order), the rotary backward of
// dq and dk_self (the transposed rotation by the same angles), and the stacked d vector of the
// q/k/v products: rows [0, nq d) dq, then n_kv d of dk, then n_kv d of dv; layout
// [row][kDPad].
template <int D>
__global__ __launch_bounds__(2 * D) void k_attn_bwd_merge(const float *dq_part, int nch,
                                                          const int32_t *lengths, int CP,
                                                          const float *dq_self,
                                                          const float *dk_self,
                                                          const float *dv_self, const float *rope,
                                                          int nq, int nkv, int B, float *dqkv) {
  constexpr int HD = D / 2, NGRP = 4;  // threads: NGRP groups of HD (dims i and i + HD)
  __shared__ float red_s[NGRP][2][HD];
  const int b = blockIdx.x, h = blockIdx.y;  // h < nq: q-head; else kv-head (block-uniform)
  const int i = threadIdx.x % HD, grp = threadIdx.x / HD;
  const float cs = rope[((size_t)b * HD + i) * 2], sn = rope[((size_t)b * HD + i) * 2 + 1];
  float y1, y2;
  size_t row;
  if (h < nq) {
    // chunk partials: group grp adds its quarter of the chunks in order, eight loads in flight;
    // then the quarters are added in group order
    const int L = lengths[b];
    const int nc = ((L + kPage - 1) / kPage + CP - 1) / CP;
    const int per = (nc + NGRP - 1) / NGRP;
    const int c0 = min(nc, grp * per), c1 = min(nc, c0 + per);
    const float *pp = dq_part + ((size_t)b * nq + h) * nch * D;
    float a1 = 0.f, a2 = 0.f;
    int c = c0;
    for (; c + 8 <= c1; c += 8) {
      float u1[8], u2[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        u1[k] = pp[(size_t)(c + k) * D + i];
        u2[k] = pp[(size_t)(c + k) * D + i + HD];
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        a1 += u1[k];
        a2 += u2[k];
      }
    }
    for (; c < c1; ++c) {
      a1 += pp[(size_t)c * D + i];
      a2 += pp[(size_t)c * D + i + HD];
    }
    red_s[grp][0][i] = a1;
    red_s[grp][1][i] = a2;
    __syncthreads();
    if (grp != 0) return;
    y1 = dq_self[((size_t)b * nq + h) * D + i];
    y2 = dq_self[((size_t)b * nq + h) * D + i + HD];
#pragma unroll
    for (int k = 0; k < NGRP; ++k) {
      y1 += red_s[k][0][i];
      y2 += red_s[k][1][i];
    }
    row = (size_t)h * D;
  } else if (grp != 0) {
    return;
  } else if (h < nq + nkv) {
    const int j = h - nq;
    y1 = dk_self[((size_t)b * nkv + j) * D + i];
    y2 = dk_self[((size_t)b * nkv + j) * D + i + HD];
    row = (size_t)nq * D + (size_t)j * D;
  } else {
    const int j = h - nq - nkv;
    dqkv[((size_t)(nq + nkv) * D + (size_t)j * D + i) * kDPad + b] =
        dv_self[((size_t)b * nkv + j) * D + i];
    dqkv[((size_t)(nq + nkv) * D + (size_t)j * D + i + HD) * kDPad + b] =
        dv_self[((size_t)b * nkv + j) * D + i + HD];
    return;
  }
  // forward: (a, c) -> (a cos - c sin, c cos + a sin); backward is the transpose
  dqkv[(row + i) * kDPad + b] = y1 * cs + y2 * sn;
  dqkv[(row + i + HD) * kDPad + b] = y2 * cs - y1 * sn;
}

// ------------------------------------------------------------------------------- sequencing

// Row splits of a transposed product: about 2048 waves (8 per compute unit, one round) and at
// most kTgemvWindow tiles per split; the tile count per split is then evened out.
int grad_tgemv_splits(int K, int tiles) {
  const int nkb = K / 32;
  int nsplit = 2048 / nkb;
  const int need = (tiles + kTgemvWindow - 1) / kTgemvWindow;
  if (nsplit < need) nsplit = need;
  if (nsplit > tiles) nsplit = tiles;
  if (nsplit > kGradMaxSplits) nsplit = kGradMaxSplits;
  if (nsplit < 1) nsplit = 1;
  const int tps = (tiles + nsplit - 1) / nsplit;
  return (tiles + tps - 1) / tps;
}

// out = W^T d over stacked segments (rows[i] rows each, packed, K inputs): the split partials
// and their sum; with swiglu the sum is turned into the gate/up d vector (see k_tgemv_sum).
static hipError_t tgemv(const Plan &p, const void *const w[3], const int rows[3], int nseg, int K,
                        const float *d, float *part, float *out, const float *gu, bool swiglu,
                        hipStream_t s) {
  TgemvArgs a;
  memset(&a, 0, sizeof a);
  int tiles = 0;
  for (int i = 0; i < nseg; ++i) {
    a.w[i] = w[i];
    a.seg_tiles[i] = rows[i] / 16;
    tiles += rows[i] / 16;
  }
  a.nseg = nseg;
  a.K = K;
  a.d = d;
  a.B = p.B;
  a.tiles = tiles;
  a.nsplit = grad_tgemv_splits(K, tiles);
  a.tps = (tiles + a.nsplit - 1) / a.nsplit;
  a.part = part;
  if (a.tps > kTgemvWindow) return hipErrorInvalidValue;  // more rows than the splits allow
  const int bps = (K / 32 + 3) / 4;
  // batches of 2 tiles (ragged 32k steering step: 15.02-15.05 ms; 4: 15.12-15.15, 8: 15.21-15.22,
  // 1: 15.68, 16: 16.5)
  hipLaunchKernelGGL(k_tgemv_mx<2>, dim3(bps * a.nsplit), dim3(256), 0, s, a);
  const int n = p.B * K;
  if (swiglu)
    hipLaunchKernelGGL(k_tgemv_sum<true>, dim3((n + 255) / 256), dim3(256), 0, s, part, a.nsplit,
                       p.B, K, gu, out);
  else
    hipLaunchKernelGGL(k_tgemv_sum<false>, dim3((n + 255) / 256), dim3(256), 0, s, part, a.nsplit,
                       p.B, K, gu, out);
  return hipGetLastError();
}

hipError_t launch_backward(const Dims &dm, const Plan &p, const Workspace &w, const GradSave &sv,
                           const kvprm_layer_weights *layers, const void *final_norm,
                           const void *reward_w, float reward_b, char *kpool, char *vpool,
                           size_t layer_bytes, const int32_t *page_table, const int32_t *lengths,
                           int CP, int chunks, float *grad_k, float *grad_v, float eta,
                           hipStream_t s) {
  const int B = p.B, H = dm.H, F = dm.F, D = dm.d, nq = dm.nq, nkv = dm.nkv;
  hipError_t e;
#define KVPRM_CHECK()                       \
  do {                                      \
    if ((e = hipGetLastError()) != hipSuccess) return e; \
  } while (0)
  hipLaunchKernelGGL(k_head_bwd, dim3(B), dim3(256), 0, s, w.x, final_norm, reward_w, reward_b, H,
                     dm.eps, sv.dx, sv.dxT, B);
  KVPRM_CHECK();
  const size_t qd = (size_t)B * nq * D, kd = (size_t)B * nkv * D;
  const size_t elems = layer_bytes / 2;  // bf16 elements of one layer's pool
  for (int l = dm.layers - 1; l >= 0; --l) {
    const kvprm_layer_weights &W = layers[l];
    const float *x_in = sv.x_in + (size_t)l * B * H, *x_mid = sv.x_mid + (size_t)l * B * H;
    const float *q = sv.q + l * qd, *ks = sv.ks + l * kd, *vs = sv.vs + l * kd;
    const float *o = sv.o + l * qd, *lse = sv.lse + (size_t)l * B * nq;
    const float *gu = sv.gu + (size_t)l * B * 2 * F;
    // FFN: dh = W_down^T dx -> (d gate, d up) -> du2 = [W_gate; W_up]^T (.) -> dx_mid
    {
      const void *wd[3] = {W.w_down, nullptr, nullptr};
      const int rd[3] = {H, 0, 0};
      if ((e = tgemv(p, wd, rd, 1, F, sv.dxT, sv.part, sv.dgu, gu, true, s)) != hipSuccess) return e;
      const void *wgu[3] = {W.w_gate, W.w_up, nullptr};
      const int rgu[3] = {F, F, 0};
      if ((e = tgemv(p, wgu, rgu, 2, H, sv.dgu, sv.part, sv.du, nullptr, false, s)) != hipSuccess)
        return e;
      hipLaunchKernelGGL(k_rms_bwd, dim3(B), dim3(1024), 0, s, x_mid, W.ffn_norm, sv.du, sv.dx,
                         sv.dxm, sv.dxmT, B, H, dm.eps);
      KVPRM_CHECK();
    }
    // attention: do = W_o^T dx_mid; the own key; the cached keys and values; dq -> du1 -> dx
    {
      const void *wo[3] = {W.wo, nullptr, nullptr};
      const int ro[3] = {H, 0, 0};
      if ((e = tgemv(p, wo, ro, 1, nq * D, sv.dxmT, sv.part, sv.dout, nullptr, false, s)) !=
          hipSuccess)
        return e;
      if (D == 64)
        hipLaunchKernelGGL(k_attn_bwd_self<64>, dim3(B, nkv), dim3(64), 0, s, q, ks, vs, o, lse,
                           sv.dout, nq, nkv, sv.Dh, sv.dq_self, sv.dk_self, sv.dv_self);
      else
        hipLaunchKernelGGL(k_attn_bwd_self<128>, dim3(B, nkv), dim3(128), 0, s, q, ks, vs, o, lse,
                           sv.dout, nq, nkv, sv.Dh, sv.dq_self, sv.dk_self, sv.dv_self);
      KVPRM_CHECK();
      AttnBwdArgs a;
      memset(&a, 0, sizeof a);
      a.kp = kpool + layer_bytes * l;
      a.vp = vpool + layer_bytes * l;
      a.gk = grad_k ? grad_k + elems * l : nullptr;
      a.gv = grad_v ? grad_v + elems * l : nullptr;
      a.eta = eta;
      a.page_table = page_table;
      a.max_pages = p.max_pages;
      a.lengths = lengths;
      a.nkv = nkv;
      a.nq = nq;
      a.CP = CP;
      a.nch = p.nch;
      a.q = q;
      a.dout = sv.dout;
      a.lse = lse;
      a.Dh = sv.Dh;
      a.dq_part = sv.dq_part;
      constexpr int WB = 8;  // waves (chunks) per block of the matrix-core backward
      const dim3 grid((chunks + WB - 1) / WB, B, nkv);
      if (D == 64)
        hipLaunchKernelGGL((k_attn_bwd_mx<64, WB>), grid, dim3(64 * WB), 0, s, a);
      else
        hipLaunchKernelGGL((k_attn_bwd_mx<128, WB>), grid, dim3(64 * WB), 0, s, a);
      KVPRM_CHECK();
      if (D == 64)
        hipLaunchKernelGGL(k_attn_bwd_merge<64>, dim3(B, nq + 2 * nkv), dim3(128), 0, s,
                           sv.dq_part, p.nch, lengths, CP, sv.dq_self, sv.dk_self, sv.dv_self,
                           w.rope, nq, nkv, B, sv.dqkv);
      else
        hipLaunchKernelGGL(k_attn_bwd_merge<128>, dim3(B, nq + 2 * nkv), dim3(256), 0, s,
                           sv.dq_part, p.nch, lengths, CP, sv.dq_self, sv.dk_self, sv.dv_self,
                           w.rope, nq, nkv, B, sv.dqkv);
      KVPRM_CHECK();
      const void *wqkv[3] = {W.wq, W.wk, W.wv};
      const int rqkv[3] = {nq * D, nkv * D, nkv * D};
      if ((e = tgemv(p, wqkv, rqkv, 3, H, sv.dqkv, sv.part, sv.du, nullptr, false, s)) != hipSuccess)
        return e;
      hipLaunchKernelGGL(k_rms_bwd, dim3(B), dim3(1024), 0, s, x_in, W.attn_norm, sv.du, sv.dxm,
                         sv.dx, sv.dxT, B, H, dm.eps);
      KVPRM_CHECK();
    }
  }
#undef KVPRM_CHECK
  return hipSuccess;
}

}  // namespace kvprm
