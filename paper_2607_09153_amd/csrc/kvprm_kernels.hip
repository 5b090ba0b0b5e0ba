// HIP kernels of the verify-token pass (gfx950). Vector-ALU versions for every dtype; the
// matrix-core (MFMA) kernels for bf16 weights and bf16/fp8 caches live in kvprm_mfma.hip
// (projections) and kvprm_attn.hip (attention).
//
// Per layer the pass runs: RMSNorm+QKV projection (split-K partials) -> sum partials + rotary
// -> split-L paged attention partials -> log-sum-exp merge with the token's own key -> output
// projection -> residual add -> RMSNorm+gate/up projection -> SwiGLU -> down projection ->
// residual add; after the last layer the final RMSNorm and the reward head.
// Every reduction has a fixed order, so results are bitwise reproducible run to run.
#include <math.h>

#include "kvprm_internal.h"

namespace kvprm {

// ------------------------------------------------------------------------------- helpers

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

__device__ __forceinline__ float load_scalar(const void *p, size_t i, int wdt) {
  return wdt ? bf16_bits_to_f32(((const uint16_t *)p)[i]) : ((const float *)p)[i];
}

// OCP E4M3FN code -> fp32 (exact). Exponent 0: subnormal m/8 * 2^-6.
__device__ __forceinline__ float e4m3_to_f32(uint32_t c) {
  uint32_t s = (c & 0x80u) << 24;
  uint32_t e = (c >> 3) & 0xFu;
  uint32_t m = c & 0x7u;
  float v;
  if (e == 0) {
    v = (float)m * 0.001953125f;  // m * 2^-9
  } else {
    v = __uint_as_float(((e + 120u) << 23) | (m << 20));
  }
  if (e == 15u && m == 7u) v = __uint_as_float(0x7FC00000u);
  return __uint_as_float(__float_as_uint(v) | s);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

// Sum over a 256-thread block; every thread gets the result. red must hold 4 floats.
__device__ __forceinline__ float block_sum256(float v, float *red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

// ------------------------------------------------------------------------------- plan

// Split-K plan of a matrix-core GEMV, in whole 32-wide input blocks: about 32 blocks per wave
// (long contiguous weight streams), but at least ~2048 waves in all and at least 4 blocks per
// slice. With one operand column tile the slice's operand is staged in LDS (1 KiB per block,
// <= 32 KiB); with more tiles the kernel reads it from memory.
static GemvPlan gemv_plan(int rows, int K, int B) {
  GemvPlan g;
  g.rows = rows;
  g.K = K;
  const int nt = gemv_nt(B);
  const int mt = gemv_mt(nt, rows);
  const int waves = (rows / 16 + mt - 1) / mt;
  const int nkb = K / 32;
  int want = (nkb + 31) / 32;
  const int want_par = (2048 + waves - 1) / waves;
  if (want < want_par) want = want_par;
  if (want > nkb / 4) want = nkb / 4;
  if (want < 1) want = 1;
  const int kb_per = (nkb + want - 1) / want;  // <= 32 unless the slice count is capped
  g.kslice = kb_per * 32;
  g.ksplit = (K + g.kslice - 1) / g.kslice;
  return g;
}

// Split-K plan of k_resid_split (wpb row tiles per block, batches of U input blocks): as many
// input slices as leave about one block per compute unit, each slice a whole number of batches.
static GemvPlan resid_split_plan(int rows, int K, int wpb, int U) {
  GemvPlan g;
  g.rows = rows;
  g.K = K;
  const int groups = (rows / 16 + wpb - 1) / wpb;
  const int nkb = K / 32;
  int want = 256 / groups;
  if (want < 1) want = 1;
  const int kb_per = ((nkb + want - 1) / want + U - 1) / U * U;
  g.kslice = kb_per * 32;
  g.ksplit = (nkb + kb_per - 1) / kb_per;
  return g;
}

static size_t partial_elems(const GemvPlan &g) {
  return (size_t)((g.ksplit + 3) & ~3) * g.rows;
}

Plan make_plan(const Dims &dm, int Breal, int max_pages, int lora_rank, int depth) {
  Plan p{};
  const int B = Breal * depth;  // rows of the pass (verify tokens of all candidates)
  p.B = B;
  p.Breal = Breal;
  p.kq = depth;
  p.max_pages = max_pages;
  p.lora_rank = lora_rank;
  // Matrix-core attention chunk: the longest of 16, 32, 64 pages that still gives at least 160
  // work items (of 256 compute units) for a batch that fills its page table (longer chunks
  // stream longer page runs per wave: measured faster even with some units idle), and at most
  // kMaxChunks - 2 chunks per candidate.
  p.cshift = 6;
  while (p.cshift > 4 && (long long)Breal * max_pages < (160LL << p.cshift)) --p.cshift;

  // chunk slots: chunks of max_pages at the shortest chunk (16 pages: the call may pick shorter
  // chunks than the plan from the host lengths) plus one (a shared prefix that ends inside a
  // chunk adds one), for whichever attention path runs
  const int n_mx = ((max_pages + 15) >> 4) + 1;
  const int n_valu = (max_pages + kChunkPagesValu - 1) / kChunkPagesValu + 1;
  p.nch = dm.kvdt == 0 ? n_valu : n_mx;
  size_t m = 0;
  if (dm.wdt == 1) {
    // sums of squares per 16-row tile (written by the fused projections' epilogues); split-K
    // partials only for the adapter's A-factor products
    p.rb = 16;
    p.nt = gemv_nt(B);
    p.bp = gemv_bp(B);
    if (lora_rank > 0) {
      // A-factor products: rows = adapter rank per segment, input = the group's input width
      p.g_la[LORA_QKV] = gemv_plan(3 * lora_rank, dm.H, B);
      p.g_la[LORA_O] = gemv_plan(lora_rank, dm.nq * dm.d, B);
      p.g_la[LORA_GU] = gemv_plan(2 * lora_rank, dm.H, B);
      p.g_la[LORA_DOWN] = gemv_plan(lora_rank, dm.F, B);
      for (const GemvPlan &g : p.g_la) m = partial_elems(g) > m ? partial_elems(g) : m;
    }
    // the fused q/k/v kernel has one block per rotary tile pair; with more pairs than compute
    // units (320 at H = 8192, 64/8 heads) a second round leaves most of the chip idle, and the
    // split-K product with its finish kernel measured faster (28.3 vs 29.1 ms per call there)
    const int pairs = (dm.nq + 2 * dm.nkv) * (dm.d / 32);
    if (pairs > 256 && lora_rank == 0) {
      p.qkv_split = 1;
      p.g_qkv = gemv_plan((dm.nq + 2 * dm.nkv) * dm.d, dm.H, B);
      m = partial_elems(p.g_qkv) > m ? partial_elems(p.g_qkv) : m;
    }
    // Split-K projections (k_resid_split + a finish kernel): a fused kernel's block owns whole
    // rows over the whole input and reads the whole operand (NT KiB per input block) from L2,
    // for H / 16 row tiles (224 at the 7B shape, under one block per compute unit); the split
    // blocks share each operand batch over 8 row tiles and cover all compute units, at the cost
    // of one more launch. Measured per call: the down projection for every batch size (ragged
    // 32k 4.79-4.82 -> 4.73-4.76 ms, 7B batch of 16 3.86 -> 3.59), q/k/v too for 9-16 rows (3.57),
    // all three for 9-16 rows with at least 512 row tiles (large fp8 24.6 -> 23.7) and for more
    // than 16 rows (beam 7.92 -> 6.74 with output and down, 6.8 -> 6.75 with q/k/v).
    {
      // input blocks per batch of k_resid_split; with one column tile 16 where the input widths
      // divide (ragged 32k 4.75 -> 4.69 ms per call against 8), else 8
      int U = 4;
      if (p.nt == 1) U = (dm.nq * dm.d / 32) % 16 == 0 && (dm.F / 32) % 16 == 0 ? 16 : 8;
      // bits: 1 down, 2 output, 4 q/k/v
      const int mask = p.nt >= 4 ? 7 : p.nt == 2 ? (dm.H / 16 >= 512 ? 7 : 5) : 1;
      if ((dm.nq * dm.d / 32) % U == 0 && (dm.F / 32) % U == 0) {
        // (8 row tiles per block measured faster than 16: 6.74 against 6.79 ms per call of the
        // 64-candidate beam)
        p.rs_wpb = 8;
        p.rs_u = U;
        p.rs_d = mask & 1;
        p.rs_o = (mask >> 1) & 1;
        p.g_rs_o = resid_split_plan(dm.H, dm.nq * dm.d, p.rs_wpb, U);
        p.g_rs_d = resid_split_plan(dm.H, dm.F, p.rs_wpb, U);
        if ((mask & 4) && (dm.H / 32) % U == 0 && (dm.nq + 2 * dm.nkv) * (dm.d / 2) >= 64) {
          p.rs_qkv = 1;
          p.g_rs_qkv = resid_split_plan((dm.nq + 2 * dm.nkv) * dm.d, dm.H, p.rs_wpb, U);
        }
        for (const GemvPlan *g : {&p.g_rs_o, &p.g_rs_d, &p.g_rs_qkv}) {
          // (with an adapter, one more slice: its B-factor tail)
          const size_t e = (size_t)(g->ksplit + (lora_rank > 0 ? 1 : 0)) * g->rows;
          m = e > m ? e : m;
        }
      }
    }
  } else {
    // vector-ALU GEMV: the activation slice of all B candidates is staged in LDS (<= 32 KiB)
    p.rb = 256;
    auto slice = [&](int K) {
      int s = (8192 / (B > 0 ? B : 1)) & ~63;
      if (s < 64) s = 64;
      if (s > K) s = K;
      return s;
    };
    p.kslice_qkv = slice(dm.H);
    p.kslice_o = slice(dm.nq * dm.d);
    p.kslice_gu = slice(dm.H);
    p.kslice_d = slice(dm.F);
    p.ks_qkv = (dm.H + p.kslice_qkv - 1) / p.kslice_qkv;
    p.ks_o = (dm.nq * dm.d + p.kslice_o - 1) / p.kslice_o;
    p.ks_gu = (dm.H + p.kslice_gu - 1) / p.kslice_gu;
    p.ks_d = (dm.F + p.kslice_d - 1) / p.kslice_d;
    const size_t e[4] = {(size_t)p.ks_qkv * (dm.nq + 2 * dm.nkv) * dm.d, (size_t)p.ks_o * dm.H,
                         (size_t)p.ks_gu * 2 * dm.F, (size_t)p.ks_d * dm.H};
    for (size_t v : e) m = v > m ? v : m;
  }
  p.nss = (dm.H + p.rb - 1) / p.rb;
  p.part_elems = m * (size_t)B;
  return p;
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

Workspace carve(const Dims &dm, const Plan &p, void *base) {
  Workspace w{};
  char *c = (char *)base;
  size_t off = 0;
  auto take = [&](size_t elems) {
    float *r = base ? (float *)(c + off) : nullptr;
    off += align256(elems * sizeof(float));
    return r;
  };
  const size_t B = (size_t)p.B;
  w.x = take(B * dm.H);
  w.ss = take((size_t)p.nss * B);
  w.part = take(p.part_elems);
  w.q = take(B * dm.nq * dm.d);
  w.kself = take(B * dm.nkv * dm.d);
  w.vself = take(B * dm.nkv * dm.d);
  w.apart = take(B * dm.nq * (size_t)p.nch * (dm.d + 2));
  w.o = take(B * dm.nq * dm.d);
  w.hffn = take(B * dm.F);
  if (dm.wdt == 1) {
    const size_t per_k = (size_t)p.nt * 64 * 8 / 32;  // bf16 elements per input of an operand
    w.rope = take(B * dm.d);
    w.opA = (uint16_t *)take((per_k * dm.H + 1) / 2);
    w.opO = (uint16_t *)take((per_k * dm.nq * dm.d + 1) / 2);
    w.opD = (uint16_t *)take((per_k * dm.F + 1) / 2);
    if (p.lora_rank > 0) w.topd = (uint16_t *)take((per_k * 3 * p.lora_rank + 1) / 2);
  }
  w.bytes = off;
  return w;
}

// Workspace of the backward pass, after the forward's (see GradSave).
GradSave carve_grad(const Dims &dm, const Plan &p, void *base) {
  GradSave g{};
  char *c = (char *)base;
  size_t off = 0;
  auto take = [&](size_t elems) {
    float *r = base ? (float *)(c + off) : nullptr;
    off += align256(elems * sizeof(float));
    return r;
  };
  const size_t B = (size_t)p.B, NL = (size_t)dm.layers, H = dm.H, F = dm.F, d = dm.d;
  const size_t nq = dm.nq, nkv = dm.nkv;
  g.x_in = take(NL * B * H);
  g.x_mid = take(NL * B * H);
  g.q = take(NL * B * nq * d);
  g.ks = take(NL * B * nkv * d);
  g.vs = take(NL * B * nkv * d);
  g.o = take(NL * B * nq * d);
  g.lse = take(NL * B * nq);
  g.gu = take(NL * B * 2 * F);
  g.dx = take(B * H);
  g.dxT = take(kDPad * H);
  g.dxm = take(B * H);
  g.dxmT = take(kDPad * H);
  g.du = take(B * H);
  g.dgu = take(2 * F * kDPad);
  g.dout = take(B * nq * d);
  g.Dh = take(B * nq);
  g.dq_self = take(B * nq * d);
  g.dk_self = take(B * nkv * d);
  g.dv_self = take(B * nkv * d);
  g.dqkv = take((nq + 2 * nkv) * d * kDPad);
  g.dq_part = take(B * nq * (size_t)p.nch * d);
  // split partials of the four transposed products
  size_t part = 0;
  const size_t cand[4][2] = {{F, H / 16}, {H, 2 * F / 16}, {nq * d, H / 16},
                             {H, (nq + 2 * nkv) * d / 16}};
  for (const auto &kt : cand) {
    const size_t n = (size_t)grad_tgemv_splits((int)kt[0], (int)kt[1]) * B * kt[0];
    part = n > part ? n : part;
  }
  g.part = take(part);
  g.bytes = off;
  return g;
}

// ------------------------------------------------------------------------------- init

// x[b] = e_v for every candidate (the verify token's embedding); ss = its sum of squares per
// 256-row block.
__global__ __launch_bounds__(256) void k_init(float *x, float *ss, const void *ev, int wdt, int B,
                                              int H) {
  __shared__ float red[4];
  const int r = blockIdx.x * 256 + threadIdx.x;
  float v = (r < H) ? load_scalar(ev, r, wdt) : 0.f;
  if (r < H)
    for (int b = 0; b < B; ++b) x[(size_t)b * H + r] = v;
  float t = block_sum256(v * v, red);
  if (threadIdx.x == 0)
    for (int b = 0; b < B; ++b) ss[(size_t)blockIdx.x * B + b] = t;
}

hipError_t launch_init(const Dims &dm, const Plan &p, const Workspace &w, const void *verify_embed,
                       hipStream_t s) {
  hipLaunchKernelGGL(k_init, dim3(p.nss), dim3(256), 0, s, w.x, w.ss, verify_embed, dm.wdt, p.B,
                     dm.H);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------- GEMV (VALU)

// One thread per output row; the block's K-slice of the (normalised) activations of all
// candidates sits in LDS and is read as broadcasts. Partials: part[ks][row][b].
template <int WDT>
__global__ __launch_bounds__(256) void k_gemv_valu(GemvSegs segs, int rows_total, int K, int kslice,
                                                   const float *in, const void *gamma,
                                                   const float *ss, int nss, float eps, int B,
                                                   float *part) {
  extern __shared__ float u_s[];  // [B][kslice]
  __shared__ float inv_s[256];
  const int k0 = blockIdx.y * kslice;
  const int kn = min(kslice, K - k0);
  if (gamma) {
    for (int b = threadIdx.x; b < B; b += 256) {
      float t = 0.f;
      for (int i = 0; i < nss; ++i) t += ss[(size_t)i * B + b];
      inv_s[b] = 1.0f / sqrtf(t / (float)K + eps);
    }
    __syncthreads();
  }
  for (int i = threadIdx.x; i < B * kn; i += 256) {
    const int b = i / kn, k = i - b * kn;
    float v = in[(size_t)b * K + k0 + k];
    if (gamma) v = v * inv_s[b] * load_scalar(gamma, k0 + k, WDT);
    u_s[b * kslice + k] = v;
  }
  __syncthreads();
  const int r = blockIdx.x * 256 + threadIdx.x;
  if (r >= rows_total) return;
  int seg = 0, base = 0;
  while (seg < segs.nseg - 1 && r >= base + segs.rows[seg]) base += segs.rows[seg++];
  const size_t roff = (size_t)(r - base) * K + k0;
  constexpr int NB = 8;
  for (int b0 = 0; b0 < B; b0 += NB) {
    float acc[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[j] = 0.f;
    if (WDT == 1) {
      const uint4 *wp = (const uint4 *)((const uint16_t *)segs.w[seg] + roff);
      for (int k = 0; k < kn; k += 8) {
        uint4 wv = wp[k >> 3];
        float wf[8] = {bf16_bits_to_f32(wv.x & 0xFFFF), bf16_bits_to_f32(wv.x >> 16),
                       bf16_bits_to_f32(wv.y & 0xFFFF), bf16_bits_to_f32(wv.y >> 16),
                       bf16_bits_to_f32(wv.z & 0xFFFF), bf16_bits_to_f32(wv.z >> 16),
                       bf16_bits_to_f32(wv.w & 0xFFFF), bf16_bits_to_f32(wv.w >> 16)};
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          if (b0 + j < B) {
            const float *u = u_s + (b0 + j) * kslice + k;
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[j] += wf[e] * u[e];
          }
        }
      }
    } else {
      const float4 *wp = (const float4 *)((const float *)segs.w[seg] + roff);
      for (int k = 0; k < kn; k += 4) {
        float4 wv = wp[k >> 2];
        float wf[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          if (b0 + j < B) {
            const float *u = u_s + (b0 + j) * kslice + k;
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[j] += wf[e] * u[e];
          }
        }
      }
    }
    float *out = part + ((size_t)blockIdx.y * rows_total + r) * B;
#pragma unroll
    for (int j = 0; j < NB; ++j)
      if (b0 + j < B) out[b0 + j] = acc[j];
  }
}

hipError_t launch_gemv(const Dims &dm, const Plan &p, const GemvSegs &segs, int K, int kslice,
                       int ksplit, const float *in, const void *gamma, const float *ss,
                       float *part, hipStream_t s) {
  int rows = 0;
  for (int i = 0; i < segs.nseg; ++i) rows += segs.rows[i];
  dim3 grid((rows + 255) / 256, ksplit);
  size_t lds = (size_t)p.B * kslice * sizeof(float);
  if (dm.wdt == 1)
    hipLaunchKernelGGL(k_gemv_valu<1>, grid, dim3(256), lds, s, segs, rows, K, kslice, in, gamma,
                       ss, p.nss, dm.eps, p.B, part);
  else
    hipLaunchKernelGGL(k_gemv_valu<0>, grid, dim3(256), lds, s, segs, rows, K, kslice, in, gamma,
                       ss, p.nss, dm.eps, p.B, part);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------- q/k/v + rotary

// Sums the split-K partials of the fused q|k|v projection and rotates q and k at position L_b
// (rotate-half: pair (i, i + d/2) by angle L_b * theta^(-2i/d), evaluated in fp64).
__global__ void k_qkv_finish(const float *part, int ksplit, int rows_total, int B, int nq, int nkv,
                             int d, float theta, const int32_t *lengths, float *q, float *ks,
                             float *vs) {
  const int b = blockIdx.x, head = blockIdx.y, i = threadIdx.x;  // i < d/2
  const int r0 = head * d + i, r1 = r0 + d / 2;
  float a = 0.f, c = 0.f;
  for (int k = 0; k < ksplit; ++k) {
    a += part[((size_t)k * rows_total + r0) * B + b];
    c += part[((size_t)k * rows_total + r1) * B + b];
  }
  float oa = a, oc = c;
  if (head < nq + nkv) {
    const double pos = (double)lengths[b];
    const double inv = pow((double)theta, (-2.0 * (double)i) / (double)d);
    double sn, cs;
    sincos(pos * inv, &sn, &cs);
    oa = (float)((double)a * cs - (double)c * sn);
    oc = (float)((double)c * cs + (double)a * sn);
  }
  float *dst;
  if (head < nq)
    dst = q + ((size_t)b * nq + head) * d;
  else if (head < nq + nkv)
    dst = ks + ((size_t)b * nkv + (head - nq)) * d;
  else
    dst = vs + ((size_t)b * nkv + (head - nq - nkv)) * d;
  dst[i] = oa;
  dst[i + d / 2] = oc;
}

hipError_t launch_qkv_finish(const Dims &dm, const Plan &p, const Workspace &w,
                             const int32_t *lengths, hipStream_t s) {
  const int rows = (dm.nq + 2 * dm.nkv) * dm.d;
  hipLaunchKernelGGL(k_qkv_finish, dim3(p.B, dm.nq + 2 * dm.nkv), dim3(dm.d / 2), 0, s, w.part,
                     p.ks_qkv, rows, p.B, dm.nq, dm.nkv, dm.d, dm.theta, lengths, w.q, w.kself,
                     w.vself);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------- attention (VALU)

template <int KVT>
__device__ __forceinline__ float kv_elem(const void *tile, int idx) {
  if (KVT == 0) return ((const float *)tile)[idx];
  if (KVT == 1) return bf16_bits_to_f32(((const uint16_t *)tile)[idx]);
  return e4m3_to_f32(((const uint8_t *)tile)[idx]);
}

// One block per (chunk of kChunkPagesValu pages, kv-head j, candidate b) over the candidate's
// private pages [first_page, npages). Writes unnormalised partials for the g q-heads of j:
// acc = sum_t e^{s_t - m} V_t, m = max_t s_t, l = sum_t e^{s_t - m}; an empty chunk writes
// m = -inf, l = 0.
template <int KVT, int D>
__global__ __launch_bounds__(256) void k_attn_valu(const void *kpool, const void *vpool,
                                                   const float *kscale, const float *vscale,
                                                   int nkv, int g, const int32_t *page_table,
                                                   int max_pages, const int32_t *lengths,
                                                   GroupTable gt, int nch, const float *q,
                                                   float *apart, int nq) {
  constexpr int EB = KVT == 0 ? 4 : (KVT == 1 ? 2 : 1);
  constexpr int X = 16 / EB;
  constexpr int T = kChunkPagesValu * kPage;  // tokens per chunk
  constexpr int NT = 256 / D;             // token groups in the PV phase
  __shared__ float q_s[16][D];
  __shared__ float s_s[16][T];
  __shared__ float acc_s[NT][16][D];
  __shared__ float ml_s[16][2];
  __shared__ int phys_s[kChunkPagesValu];
  __shared__ float ksc_s[kChunkPagesValu], vsc_s[kChunkPagesValu];

  const int c = blockIdx.x, j = blockIdx.y, b = blockIdx.z;
  const int L = lengths[b];
  const int npages = (L + kPage - 1) / kPage;
  int first = 0;
  for (int gi = 0; gi < gt.n; ++gi)
    if (b >= gt.start[gi] && b < gt.start[gi + 1]) first = gt.prefix_pages[gi];
  const int p0 = first + c * kChunkPagesValu;
  float *outbase = apart + (((size_t)b * nq + (size_t)j * g) * nch + c) * (D + 2);
  const size_t hstride = (size_t)nch * (D + 2);
  if (p0 >= npages) {
    for (int i = threadIdx.x; i < g * (D + 2); i += 256) {
      const int h = i / (D + 2), e = i - h * (D + 2);
      outbase[h * hstride + e] = (e == D) ? -INFINITY : 0.f;
    }
    return;
  }
  const int p1 = min(npages, p0 + kChunkPagesValu);
  const int tok0 = p0 * kPage;
  const int ntok = min(L, p1 * kPage) - tok0;
  for (int i = threadIdx.x; i < g * D; i += 256) {
    const int h = i / D, m = i - h * D;
    q_s[h][m] = q[((size_t)b * nq + j * g + h) * D + m];
  }
  for (int i = threadIdx.x; i < p1 - p0; i += 256) {
    const int ph = page_table[(size_t)b * max_pages + p0 + i];
    phys_s[i] = ph;
    if (KVT == 2) {
      ksc_s[i] = kscale[(size_t)ph * nkv + j];
      vsc_s[i] = vscale[(size_t)ph * nkv + j];
    }
  }
  __syncthreads();
  const float rs = 1.0f / sqrtf((float)D);
  // scores
  for (int t = threadIdx.x; t < T; t += 256) {
    float s[16];
#pragma unroll
    for (int h = 0; h < 16; ++h) s[h] = 0.f;
    if (t < ntok) {
      const int pg = t / kPage, slot = t % kPage;
      const char *tile = (const char *)kpool + ((size_t)phys_s[pg] * nkv + j) * (kPage * D) * EB;
      for (int m0 = 0; m0 < D; m0 += X) {
#pragma unroll
        for (int e = 0; e < X; ++e) {
          const float kv = kv_elem<KVT>(tile, ((m0 / X) * kPage + slot) * X + e);
#pragma unroll
          for (int h = 0; h < 16; ++h)
            if (h < g) s[h] += q_s[h][m0 + e] * kv;
        }
      }
      const float sc = (KVT == 2) ? ksc_s[pg] * rs : rs;
#pragma unroll
      for (int h = 0; h < 16; ++h)
        if (h < g) s_s[h][t] = s[h] * sc;
    } else {
#pragma unroll
      for (int h = 0; h < 16; ++h)
        if (h < g) s_s[h][t] = -INFINITY;
    }
  }
  __syncthreads();
  // softmax statistics per head: one wave per head
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int h = wv; h < g; h += 4) {
    float m = -INFINITY;
    for (int t = lane; t < T; t += 64) m = fmaxf(m, s_s[h][t]);
    m = wave_max(m);
    float l = 0.f;
    for (int t = lane; t < T; t += 64) {
      const float pv = (t < ntok) ? expf(s_s[h][t] - m) : 0.f;
      s_s[h][t] = pv;
      l += pv;
    }
    l = wave_sum(l);
    if (lane == 0) {
      ml_s[h][0] = m;
      ml_s[h][1] = l;
    }
  }
  __syncthreads();
  // P V: thread (dim m, token group tg)
  {
    const int m = threadIdx.x % D, tg = threadIdx.x / D;
    float acc[16];
#pragma unroll
    for (int h = 0; h < 16; ++h) acc[h] = 0.f;
    const int npg = p1 - p0;
    for (int pg = tg; pg < npg; pg += NT) {
      const char *tile = (const char *)vpool + ((size_t)phys_s[pg] * nkv + j) * (kPage * D) * EB;
      const float vsc = (KVT == 2) ? vsc_s[pg] : 1.f;
      const int nslot = min(kPage, ntok - pg * kPage);
      constexpr int R = X / 4;
      const int vbase = (((m / (16 * R)) * 4) * 16 + m % 16) * R + (m / 16) % R;
      for (int sl = 0; sl < nslot; ++sl) {
        // V tile: ((((m / 16R) * 4 + s / 4) * 16 + m % 16) * R + (m / 16) % R) * 4 + s % 4
        const float v = kv_elem<KVT>(tile, (vbase + (sl / 4) * 16 * R) * 4 + sl % 4) * vsc;
        const int t = pg * kPage + sl;
#pragma unroll
        for (int h = 0; h < 16; ++h)
          if (h < g) acc[h] += s_s[h][t] * v;
      }
    }
#pragma unroll
    for (int h = 0; h < 16; ++h)
      if (h < g) acc_s[tg][h][m] = acc[h];
  }
  __syncthreads();
  for (int i = threadIdx.x; i < g * D; i += 256) {
    const int h = i / D, m = i - h * D;
    float a = 0.f;
    for (int tg = 0; tg < NT; ++tg) a += acc_s[tg][h][m];
    outbase[h * hstride + m] = a;
  }
  if (threadIdx.x < g) {
    outbase[threadIdx.x * hstride + D] = ml_s[threadIdx.x][0];
    outbase[threadIdx.x * hstride + D + 1] = ml_s[threadIdx.x][1];
  }
}

// Log-sum-exp merge of the chunk partials with the token's own key/value:
// m = max(m_c, s_self), o = (sum_c e^{m_c - m} acc_c + e^{s_self - m} v_self) /
//                           (sum_c e^{m_c - m} l_c + e^{s_self - m}).
template <int D>
__global__ __launch_bounds__(D) void k_merge(const float *apart, int nch, GroupTable gt,
                                             const float *q,
                                             const float *kself, const float *vself,
                                             const int32_t *lengths, float *o, int nq, int nkv,
                                             int g) {
  __shared__ float red[2];
  const int b = blockIdx.x, h = blockIdx.y, m = threadIdx.x;
  const int j = h / g;
  float prod = q[((size_t)b * nq + h) * D + m] * kself[((size_t)b * nkv + j) * D + m];
  prod = wave_sum(prod);
  if (D > 64) {
    if ((m & 63) == 0) red[m >> 6] = prod;
    __syncthreads();
    prod = red[0] + red[1];
  }
  const float s_self = prod * (1.0f / sqrtf((float)D));
  const int L = lengths[b];
  const int npages = (L + kPage - 1) / kPage;
  int first = 0;
  for (int gi = 0; gi < gt.n; ++gi)
    if (b >= gt.start[gi] && b < gt.start[gi + 1]) first = gt.prefix_pages[gi];
  const int nc = (npages - first + kChunkPagesValu - 1) / kChunkPagesValu;
  const float *pb = apart + ((size_t)b * nq + h) * nch * (D + 2);
  float mx = s_self;
  for (int c = 0; c < nc; ++c) mx = fmaxf(mx, pb[(size_t)c * (D + 2) + D]);
  float es = expf(s_self - mx);
  float l = es;
  float acc = es * vself[((size_t)b * nkv + j) * D + m];
  for (int c = 0; c < nc; ++c) {
    const float *pc = pb + (size_t)c * (D + 2);
    const float f = expf(pc[D] - mx);
    l += f * pc[D + 1];
    acc += f * pc[m];
  }
  o[((size_t)b * nq + h) * D + m] = acc / l;
}

static hipError_t launch_merge(const Dims &dm, const Plan &p, const Workspace &w,
                               const GroupTable &gt, const int32_t *lengths, const float *q,
                               const float *kself, const float *vself, float *o, hipStream_t s) {
  if (dm.d == 64)
    hipLaunchKernelGGL(k_merge<64>, dim3(p.B, dm.nq), dim3(64), 0, s, w.apart, p.nch, gt, q,
                       kself, vself, lengths, o, dm.nq, dm.nkv, dm.g);
  else
    hipLaunchKernelGGL(k_merge<128>, dim3(p.B, dm.nq), dim3(128), 0, s, w.apart, p.nch, gt, q,
                       kself, vself, lengths, o, dm.nq, dm.nkv, dm.g);
  return hipGetLastError();
}

hipError_t launch_attention(const Dims &dm, const Plan &p, const Workspace &w, int layer,
                            const void *kpool, const void *vpool, const float *kscale,
                            const float *vscale, int num_pages, const int32_t *page_table,
                            const int32_t *lengths, const GroupTable &gt, const float *q,
                            const float *kself, const float *vself, float *o, hipStream_t s,
                            bool merge) {
  const int EB = dm.kvdt == 0 ? 4 : (dm.kvdt == 1 ? 2 : 1);
  const size_t layer_elems = (size_t)num_pages * dm.nkv * kPage * dm.d;
  const char *kp = (const char *)kpool + layer_elems * EB * layer;
  const char *vp = (const char *)vpool + layer_elems * EB * layer;
  const float *ksc = kscale ? kscale + (size_t)layer * num_pages * dm.nkv : nullptr;
  const float *vsc = vscale ? vscale + (size_t)layer * num_pages * dm.nkv : nullptr;
  if (dm.kvdt != 0)  // matrix-core kernels (bf16 and fp8 caches)
    return launch_attn_mx(dm, p, w, kp, vp, ksc, vsc, page_table, lengths, gt, q, kself, vself, o,
                          nullptr, s, merge);
  dim3 grid(p.nch, dm.nkv, p.B);
#define KVPRM_ATT(KVT, D)                                                                     \
  hipLaunchKernelGGL((k_attn_valu<KVT, D>), grid, dim3(256), 0, s, kp, vp, ksc, vsc, dm.nkv, \
                     dm.g, page_table, p.max_pages, lengths, gt, p.nch, q, w.apart, dm.nq)
  if (dm.d == 64) {
    if (dm.kvdt == 0) KVPRM_ATT(0, 64);
    else if (dm.kvdt == 1) KVPRM_ATT(1, 64);
    else KVPRM_ATT(2, 64);
  } else {
    if (dm.kvdt == 0) KVPRM_ATT(0, 128);
    else if (dm.kvdt == 1) KVPRM_ATT(1, 128);
    else KVPRM_ATT(2, 128);
  }
#undef KVPRM_ATT
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !merge) return e;
  return launch_merge(dm, p, w, gt, lengths, q, kself, vself, o, s);
}

// ------------------------------------------------------------------------------- residual

// x[b][r] += sum_ks part[ks][r][b]; ss[blk][b] = sum over the block's rows of x^2.
__global__ __launch_bounds__(256) void k_residual(float *x, const float *part, int ksplit, float *ss,
                                                  int B, int H) {
  __shared__ float red[4][64];
  const int r = blockIdx.x * 256 + threadIdx.x;
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int b0 = 0; b0 < B; b0 += 64) {
    for (int bb = 0; bb < 64 && b0 + bb < B; ++bb) {
      const int b = b0 + bb;
      float v = 0.f;
      if (r < H) {
        float a = 0.f;
        for (int k = 0; k < ksplit; ++k) a += part[((size_t)k * H + r) * B + b];
        v = x[(size_t)b * H + r] + a;
        x[(size_t)b * H + r] = v;
      }
      const float t = wave_sum(v * v);
      if (lane == 0) red[wv][bb] = t;
    }
    __syncthreads();
    if (threadIdx.x < 64 && b0 + threadIdx.x < B)
      ss[(size_t)blockIdx.x * B + b0 + threadIdx.x] =
          (red[0][threadIdx.x] + red[1][threadIdx.x]) + (red[2][threadIdx.x] + red[3][threadIdx.x]);
    __syncthreads();
  }
}

hipError_t launch_residual(const Dims &dm, const Plan &p, const Workspace &w, int ksplit,
                           hipStream_t s) {
  hipLaunchKernelGGL(k_residual, dim3(p.nss), dim3(256), 0, s, w.x, w.part, ksplit, w.ss, p.B,
                     dm.H);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------- SwiGLU

// h[b][f] = silu(gate) * up, gate/up = sums of the split-K partials of rows f and F + f.
__global__ __launch_bounds__(256) void k_swiglu(const float *part, int ksplit, float *h, int B,
                                                int F) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (size_t)B * F) return;
  const int f = (int)(i / B), b = (int)(i - (size_t)f * B);
  float gs = 0.f, us = 0.f;
  for (int k = 0; k < ksplit; ++k) {
    gs += part[((size_t)k * 2 * F + f) * B + b];
    us += part[((size_t)k * 2 * F + F + f) * B + b];
  }
  h[(size_t)b * F + f] = gs / (1.0f + expf(-gs)) * us;
}

hipError_t launch_swiglu(const Dims &dm, const Plan &p, const Workspace &w, int ksplit,
                         hipStream_t s) {
  const size_t n = (size_t)p.B * dm.F;
  hipLaunchKernelGGL(k_swiglu, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, w.part, ksplit,
                     w.hffn, p.B, dm.F);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------- reward head

// z_b = w_r . (x_b / sqrt(mean(x_b^2) + eps) * gamma_f) + b_r; P(+) = sigmoid(z_b). One pass
// over x_b: sum(x^2) and sum(x gamma_f w_r) together (the RMS scale is a common factor of the
// dot product), four rows per thread in flight.
__global__ __launch_bounds__(256) void k_head(const float *x, int H, float eps, const void *gam,
                                              const void *wr, int wdt, float rb, float *scores,
                                              float *logits, int kq) {
  __shared__ float red[4];
  const int b = blockIdx.x;
  const float *xb = x + ((size_t)b * kq + kq - 1) * H;  // the candidate's last verify token
  float sq = 0.f, dot = 0.f;
  int r = threadIdx.x;
  for (; r + 3 * 256 < H; r += 4 * 256) {
    float v[4], gw[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      v[u] = xb[r + u * 256];
      gw[u] = load_scalar(gam, r + u * 256, wdt) * load_scalar(wr, r + u * 256, wdt);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      sq += v[u] * v[u];
      dot += v[u] * gw[u];
    }
  }
  for (; r < H; r += 256) {
    const float v = xb[r];
    sq += v * v;
    dot += v * (load_scalar(gam, r, wdt) * load_scalar(wr, r, wdt));
  }
  sq = block_sum256(sq, red);
  dot = block_sum256(dot, red);
  if (threadIdx.x == 0) {
    const float inv = 1.0f / sqrtf(sq / (float)H + eps);
    const float z = dot * inv + rb;
    float pz;
    if (z >= 0.f) {
      pz = 1.0f / (1.0f + expf(-z));
    } else {
      const float ez = expf(z);
      pz = ez / (1.0f + ez);
    }
    scores[b] = pz;
    if (logits) logits[b] = z;
  }
}

hipError_t launch_head(const Dims &dm, const Plan &p, const Workspace &w, const void *final_norm,
                       const void *reward_w, float reward_b, float *scores, float *logits,
                       hipStream_t s) {
  hipLaunchKernelGGL(k_head, dim3(p.Breal), dim3(256), 0, s, w.x, dm.H, dm.eps, final_norm,
                     reward_w, dm.wdt, reward_b, scores, logits, p.kq);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------- cache packing

// Token-major cache tiles ([page_size][d] values, slot-major) -> the stored K or V tile layout.
// One block per tile (grid-stride over tiles): the tile is read into LDS with 16-byte loads,
// then every thread assembles 16-byte output groups in output order and stores them, so both
// the reads and the writes are contiguous. EB = element bytes; x = 16 / EB values per group.
//   K group (m / x) * 16 + s holds dims m .. m + x - 1 of slot s (a contiguous source run);
//   V group ((m / (16 r)) * 4 + s / 4) * 16 + m % 16 holds slots 4 (s / 4) .. + 3 of the r dims
//   m % 16 + 16 i (i < r) of the 16 r-dim block, as [i][slot % 4] (r = x / 4).
template <int EB, bool V>
__global__ __launch_bounds__(256) void k_pack_kv(const uint4 *__restrict__ src, uint4 *__restrict__ dst,
                                                 int64_t ntiles, int d) {
  extern __shared__ uint4 tile_s[];
  constexpr int X = 16 / EB, R = X / 4;
  const int groups = 16 * d / X;  // 16-byte groups per tile
  const unsigned char *tb = (const unsigned char *)tile_s;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const uint4 *sp = src + t * groups;
    for (int i = threadIdx.x; i < groups; i += 256) tile_s[i] = sp[i];
    __syncthreads();
    for (int gi = threadIdx.x; gi < groups; gi += 256) {
      uint4 out;
      if (!V) {
        const int s = gi & 15, mb = gi >> 4;  // slot, x-dim block
        out = tile_s[s * (d / X) + mb];
      } else {
        const int mm = gi & 15, sq = (gi >> 4) & 3, blk = gi >> 6;
        unsigned char *ob = (unsigned char *)&out;
#pragma unroll
        for (int i = 0; i < R; ++i)
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const int m = blk * 16 * R + i * 16 + mm, sl = 4 * sq + k;
#pragma unroll
            for (int e = 0; e < EB; ++e) ob[(i * 4 + k) * EB + e] = tb[(sl * d + m) * EB + e];
          }
      }
      dst[t * groups + gi] = out;
    }
    __syncthreads();
  }
}

hipError_t launch_pack_kv(const void *src, void *dst, int64_t ntiles, int d, int eb, bool v,
                          hipStream_t s) {
  const size_t lds = (size_t)16 * d * eb;
  int64_t blocks = ntiles < 65536 ? ntiles : 65536;
  const dim3 grid((unsigned)blocks), block(256);
  const uint4 *a = (const uint4 *)src;
  uint4 *b = (uint4 *)dst;
#define KVPRM_PK(E_)                                                                    \
  if (v) hipLaunchKernelGGL((k_pack_kv<E_, true>), grid, block, lds, s, a, b, ntiles, d); \
  else hipLaunchKernelGGL((k_pack_kv<E_, false>), grid, block, lds, s, a, b, ntiles, d)
  switch (eb) {
    case 4: KVPRM_PK(4); break;
    case 2: KVPRM_PK(2); break;
    case 1: KVPRM_PK(1); break;
    default: return hipErrorInvalidValue;
  }
#undef KVPRM_PK
  return hipGetLastError();
}

// ------------------------------------------------------------------------------- diagnostics

// Streaming read of n16 16-byte words: grid-stride, four non-temporal loads in flight per
// thread, the words folded into an XOR that each wave adds to *sink with one atomic, so that the
// loads cannot be removed (and a test can check that every word was read once). The reference
// ceiling for the kernels' HBM fractions.
__global__ __launch_bounds__(256) void k_stream_read(const uint4 *buf, size_t n16, uint32_t *sink) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const size_t stride = (size_t)gridDim.x * 256;
  size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  uint32_t acc = 0;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    u32x4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = __builtin_nontemporal_load((const u32x4 *)(buf + i + u * stride));
#pragma unroll
    for (int u = 0; u < 4; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n16; i += stride) {
    const u32x4 v = __builtin_nontemporal_load((const u32x4 *)(buf + i));
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, off, 64);
  if ((threadIdx.x & 63) == 0) atomicXor(sink, acc);
}

hipError_t launch_stream_read(const void *buf, size_t bytes, uint32_t *sink, hipStream_t s) {
  // 512 blocks of 4 waves: the fastest shape of a plain streaming read on this chip (256 blocks
  // leave the memory system short of requests, 1024 and more add contention)
  hipLaunchKernelGGL(k_stream_read, dim3(512), dim3(256), 0, s, (const uint4 *)buf, bytes / 16,
                     sink);
  return hipGetLastError();
}

}  // namespace kvprm
