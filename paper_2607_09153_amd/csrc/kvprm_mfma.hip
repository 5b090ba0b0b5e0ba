// Matrix-core (MFMA, v_mfma_f32_16x16x32_bf16) pipeline of the verify-token pass for gfx950,
// used with bf16 weights and bf16 or fp8 (OCP e4m3) caches: the projections and their fused
// element-wise steps (this file) and the attention kernels (kvprm_attn.hip). Per layer:
//
//   q/k/v projection, RMSNorm scale and rotary in its epilogue      -> q, k_self, v_self
//   attention (split-L paged partials) -> merge with the token's own key (-> o, as operand)
//   output projection + residual (x += .., sums of squares, operand x * gamma_ffn)
//   gate/up projection + SwiGLU (RMSNorm scale, silu(g) * u, operand of the down projection)
//   down projection + residual (x += .., sums of squares, operand x * gamma_attn of the next layer)
//
// Each projection block owns whole output rows: its waves split the input range and add their
// sums in a fixed order, so results are bitwise reproducible. RMSNorm is applied as a
// per-candidate scale after the product: W (x * gamma * r) = r * (W (x * gamma)),
// r = 1/sqrt(mean(x^2) + eps). The split-K GEMV (k-partials, then a finish kernel) serves the
// A factors of unmerged adapters.
//
// Precision: weights and cache values enter the matrix cores exactly (bf16, or e4m3 widened to
// bf16, which is exact). The fp32 operands on the other side are split into bf16 terms,
// x = hi + lo (three terms for queries), and every term is multiplied, so products keep about
// fp32 accuracy and accumulate in fp32.
//
// MFMA 16x16x32 operand layout used throughout (lane l, c = l / 16, n = l % 16):
//   A (16 x 32): lane holds row n, reduction slots 8c .. 8c+7
//   B (32 x 16): lane holds column n, reduction slots 8c .. 8c+7
//   D (16 x 16): lane holds rows 4c .. 4c+3 of column n
// Reduction slots are paired between A and B by (c, element), so any assignment of the
// contracted index to slots is valid as long as both operands use the same one.
//
// Activation operand of a GEMV ("operand buffer"): for k-block kb (32 inputs), column tile t
// and lane, 8 bf16 = inputs 32 kb + 8 (lane / 16) + i of column 16 t + lane % 16. Columns: with
// Bp == 8 (batch <= 8, one tile) columns 0..7 hold the hi halves and 8..15 the lo halves of
// candidates 0..7; otherwise columns [0, Bp) are hi and [Bp, 2 Bp) lo (Bp = batch rounded up
// to 16). Columns of absent candidates only ever reach outputs that are discarded.
#include <math.h>
#include <string.h>

#include "kvprm_internal.h"
#include "kvprm_mx_common.h"

namespace kvprm {

// operand column tiles for B candidates: one (hi in columns 0..7, lo in 8..15) up to 8, else
// hi and lo tiles of 16 candidates each
int gemv_nt(int B) { return B <= 8 ? 1 : 2 * ((B + 15) / 16); }
// row tiles per wave of the split-K GEMV: two (sharing each operand load) for several operand
// column tiles and many rows; one otherwise (more waves for the short projections)
int gemv_mt(int nt, int rows) { return nt >= 2 && rows >= 8192 ? 2 : 1; }
int gemv_bp(int B) { return B <= 8 ? 8 : 16 * ((B + 15) / 16); }

// ------------------------------------------------------------------------------- init

// x_b = e_v, the sums of squares per RB-row block, the QKV operand e_v * gamma_attn(0), and the
// rotary table cos/sin(L_b theta^(-2i/d)) (angles in fp64).
__global__ __launch_bounds__(256) void k_init_mx(float *x, float *ss, int RB, const void *ev,
                                                 const void *gamma0, int wdt, int B, int H,
                                                 uint16_t *opA, int NT, int Bp,
                                                 const int32_t *lengths, int kq, float theta,
                                                 int d, float *rope, float *xsave) {
  __shared__ float red[4];
  const int r0 = blockIdx.x * RB;
  const int nr = min(RB, H - r0);
  float sq = 0.f;
  for (int idx = threadIdx.x; idx < nr * B; idx += 256) {  // (row, candidate) pairs
    const int i = idx % nr, b = idx / nr;
    const int r = r0 + i;
    const float v = ld_w(ev, r, wdt);
    if (b == 0) sq += v * v;
    x[(size_t)b * H + r] = v;
    if (xsave) xsave[(size_t)b * H + r] = v;
    store_operand(opA, NT, Bp, r, b, v * ld_w(gamma0, r, wdt));
  }
  sq = bsum(sq, red);
  if (threadIdx.x < B) ss[(size_t)blockIdx.x * B + threadIdx.x] = sq;
  // the rotary table over all blocks' threads (one fp64 angle each: a single block took 18 us
  // for 64 rows)
  for (int e = blockIdx.x * 256 + threadIdx.x; e < B * (d / 2); e += gridDim.x * 256) {
    // row b is verify token b % kq of candidate b / kq, at position L + b % kq
    const int b = e / (d / 2), i = e - b * (d / 2);
    const double inv = pow((double)theta, (-2.0 * (double)i) / (double)d);
    double sn, cs;
    sincos((double)(lengths[b / kq] + b % kq) * inv, &sn, &cs);
    rope[2 * e] = (float)cs;
    rope[2 * e + 1] = (float)sn;
  }
}

// ------------------------------------------------------------------------------- GEMV

struct GemvArgs {
  const void *w[3];  // weight segments [rows_i][K], row-major, stacked in order
  int seg_rows[3];
  int nseg;
  int rows, K, kslice, ksplit;
  const uint4 *act;  // operand buffer of the input
  int B;
  float *part;  // [rows][B][ksp] k-partials, ksp = ksplit rounded up to 4
  int ksp;
};

// part[row][b][ks] = sum over k-slice ks of W[row][k] u_b[k], W in the packed tile layout
// (1 KiB per 32-input block and 16-row tile, input block major, in A-operand lane order): one
// load instruction reads 1 KiB, and the waves working on one k-slice sweep a contiguous region
// together, input block by input block. Each wave owns MT row tiles. The weights stream in
// batches of U input blocks, double buffered: the next batch's loads are in flight while the
// current batch's MT * NT * U MFMAs run, and the first batch is issued before the block copies
// its k-slice of the operand (NT column tiles) into LDS. The hi and lo halves of each candidate
// are added before the partial is stored.
template <int MT, int NT, int U, int WPB, bool DIRECT>
__global__ __launch_bounds__(64 * WPB) void k_gemv_mx(GemvArgs a) {
  extern __shared__ uint4 act_s[];  // the block's k-slice of the operand: nkb * NT * 64 entries
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int ks = blockIdx.y;
  const int k0 = ks * a.kslice;
  const int nkb = min(a.kslice, a.K - k0) >> 5;
  const int tile0 = (blockIdx.x * WPB + wave) * MT;
  const int B = a.B;
  const bool active = tile0 * 16 < a.rows;
  const uint4 *wt[MT];
  size_t kstride[MT];  // uint4 entries between consecutive input blocks of a tile
  bool valid[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const int tile = tile0 + m;
    valid[m] = tile * 16 < a.rows;
    int seg = 0, base = 0;
    while (seg < a.nseg - 1 && tile * 16 >= base + a.seg_rows[seg]) base += a.seg_rows[seg++];
    const int lt = valid[m] ? tile - base / 16 : 0;
    const size_t ntiles = (size_t)a.seg_rows[seg] / 16;
    kstride[m] = ntiles * 64;
    wt[m] = (const uint4 *)a.w[seg] + ((size_t)(k0 >> 5) * ntiles + lt) * 64 + lane;
  }
  // Rows of an absent tile read tile 0 of their segment and are never stored.
  auto load_batch = [&](int kb, uint4 (&av)[U][MT]) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int m = 0; m < MT; ++m) av[u][m] = ld_stream(&wt[m][(size_t)(kb + u) * kstride[m]]);
  };
  const uint4 *ap = (DIRECT ? a.act + (size_t)(k0 >> 5) * NT * 64 : act_s) + lane;
  floatx4 acc[MT][NT];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[m][t] = floatx4{0.f, 0.f, 0.f, 0.f};
  auto mma_batch = [&](int kb, const uint4 (&av)[U][MT]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      uint4 bv[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) bv[t] = ap[((kb + u) * NT + t) * 64];
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[m][t] = mfma16(av[u][m], bv[t], acc[m][t]);
    }
  };
  const int nbat = nkb / U;
  uint4 a0[U][MT], a1[U][MT];
  if (active && nbat > 0) load_batch(0, a0);
  if (!DIRECT) {
    const uint4 *src = a.act + (size_t)(k0 >> 5) * NT * 64;
    for (int i = threadIdx.x; i < nkb * NT * 64; i += 64 * WPB) act_s[i] = src[i];
    __syncthreads();
  }
  if (!active) return;
  // pairs of batches; a prefetch past the last batch repeats the last one (an L2 hit) so that
  // the loop has no conditional loads
  int i = 0;
  for (; i + 2 <= nbat; i += 2) {
    load_batch((i + 1) * U, a1);
    __builtin_amdgcn_sched_barrier(0);
    mma_batch(i * U, a0);
    __builtin_amdgcn_sched_barrier(0);
    load_batch(min(i + 2, nbat - 1) * U, a0);
    __builtin_amdgcn_sched_barrier(0);
    mma_batch((i + 1) * U, a1);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (i < nbat) mma_batch(i * U, a0);
  for (int kb = nbat * U; kb < nkb; ++kb) {
    uint4 av[MT], bv[NT];
#pragma unroll
    for (int m = 0; m < MT; ++m) av[m] = ld_stream(&wt[m][(size_t)kb * kstride[m]]);
#pragma unroll
    for (int t = 0; t < NT; ++t) bv[t] = ap[(kb * NT + t) * 64];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[m][t] = mfma16(av[m], bv[t], acc[m][t]);
  }
  const int n = lane & 15, c4 = (lane >> 4) * 4;
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    if (!valid[m]) continue;
    const int rbase = (tile0 + m) * 16 + c4;
    if (NT == 1) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float v = acc[m][0][i] + __shfl_xor(acc[m][0][i], 8, 64);
        if (n < 8 && n < B) a.part[((size_t)(rbase + i) * B + n) * a.ksp + ks] = v;
      }
    } else {
#pragma unroll
      for (int t = 0; t < NT / 2; ++t) {
        const int cand = t * 16 + n;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float v = acc[m][t][i] + acc[m][t + NT / 2][i];
          if (cand < B) a.part[((size_t)(rbase + i) * B + cand) * a.ksp + ks] = v;
        }
      }
    }
  }
}

// Sum of the k-partials of output row idx = r * B + b, contiguous, added in k order, in two
// steps so that callers can issue every load of a kernel before the first add: ksum_load issues
// the first NMAX 16-byte loads unconditionally (indices past the row's last group repeat it
// and are not added), ksum_add adds them and loads any groups beyond NMAX itself.
template <int NMAX>
__device__ __forceinline__ void ksum_load(const float *__restrict__ part, int ksp, size_t idx,
                                          float4 (&v)[NMAX]) {
  const float4 *pp = (const float4 *)(part + idx * ksp);
  const int n4 = ksp >> 2;
#pragma unroll
  for (int i = 0; i < NMAX; ++i) v[i] = pp[min(i, n4 - 1)];
}

template <int NMAX>
__device__ __forceinline__ float ksum_add(const float *__restrict__ part, int ksp, int ksplit,
                                          size_t idx, const float4 (&v)[NMAX]) {
  const int n4 = ksp >> 2;
  float s = 0.f;
  auto add4 = [&](const float4 &w, int k) {
    s += k < ksplit ? w.x : 0.f;
    s += k + 1 < ksplit ? w.y : 0.f;
    s += k + 2 < ksplit ? w.z : 0.f;
    s += k + 3 < ksplit ? w.w : 0.f;
  };
#pragma unroll
  for (int i = 0; i < NMAX; ++i)
    if (i < n4) add4(v[i], 4 * i);
  const float4 *pp = (const float4 *)(part + idx * ksp);
  for (int i = NMAX; i < n4; ++i) add4(pp[i], 4 * i);
  return s;
}

// NMAX for ksum: the number of 16-byte groups of a partial row, rounded up to 1, 2, 4 or 8.
static int ksum_nmax(int ksp) {
  const int n4 = ksp >> 2;
  return n4 <= 1 ? 1 : n4 <= 2 ? 2 : n4 <= 4 ? 4 : 8;
}


// v += ss[i][b] for i = i0, i0 + P, ... < nss, in that order, eight loads in flight at a time.
__device__ __forceinline__ void rms_tail(const float *__restrict__ ss, int B, int b, int i0, int P,
                                         int nss, float &v) {
  int i = i0;
  for (; i + 7 * P < nss; i += 8 * P) {
    float t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) t[u] = ss[(size_t)(i + u * P) * B + b];
#pragma unroll
    for (int u = 0; u < 8; ++u) v += t[u];
  }
  for (; i < nss; i += P) v += ss[(size_t)i * B + b];
}

// RMSNorm scales r_b = 1 / sqrt(mean(x_b^2) + eps) from the per-row-block sums of squares
// ss[i][b], by one wave (B <= 8), without LDS or barriers: with Bq = B rounded up to a power
// of two, lane l sums rows l / Bq, l / Bq + 64 / Bq, ... of candidate l % Bq (32 loads issued by
// wave_rms_load, any further rows in wave_rms_finish), a butterfly over the lanes of equal
// l % Bq completes the sums (identical in every lane and block), and each lane takes its own
// candidate's.
struct WaveRmsLoads {
  float v[32];
};

__device__ __forceinline__ void wave_rms_load(const float *__restrict__ ss, int nss, int B,
                                              WaveRmsLoads &ld) {
  const int lane = threadIdx.x & 63;
  int Bq = 1;
  while (Bq < B) Bq <<= 1;
  const int P = 64 / Bq;
  const int bl = lane & (Bq - 1), part = lane / Bq;
  const bool ok = bl < B;
#pragma unroll
  for (int u = 0; u < 32; ++u) {
    const int i = part + u * P;
    const bool in = ok && i < nss;
    const float t = ss[(size_t)(in ? i : 0) * B + (ok ? bl : 0)];
    ld.v[u] = in ? t : 0.f;
  }
}

__device__ __forceinline__ float wave_rms_finish(const float *__restrict__ ss, int nss, int B, int b,
                                                 int H, float eps, const WaveRmsLoads &ld) {
  const int lane = threadIdx.x & 63;
  int Bq = 1;
  while (Bq < B) Bq <<= 1;
  const int P = 64 / Bq;
  const int bl = lane & (Bq - 1), part = lane / Bq;
  float v = 0.f;
#pragma unroll
  for (int u = 0; u < 32; ++u) v += ld.v[u];
  if (bl < B) rms_tail(ss, B, bl, part + 32 * P, P, nss, v);
  for (int off = Bq; off < 64; off <<= 1) v += __shfl_xor(v, off, 64);
  const float tot = __shfl(v, b, 64);
  return 1.0f / sqrtf(tot / (float)H + eps);
}

// r_b = 1 / sqrt(mean(x_b^2) + eps) for every candidate, computed by a whole block of NTHR
// threads from the per-row-block sums of squares ss[i][b] into inv_s[b]: with Bq = B rounded up
// to a power of two, thread t sums rows t / Bq, t / Bq + NTHR / Bq, ... of candidate t % Bq,
// and the NTHR / Bq partial sums of each candidate are added in a fixed order, so every block
// gets identical values. rms_load issues a thread's first 16 loads (unconditional, clamped,
// zero past the end) so that callers can start them early; rms_finish adds any further rows,
// reduces, and contains two barriers.
struct RmsLoads {
  float v[16];
};

template <int NTHR>
__device__ __forceinline__ void rms_load(const float *__restrict__ ss, int nss, int B,
                                         RmsLoads &ld) {
  const int t = threadIdx.x;
  int Bq = 1;
  while (Bq < B) Bq <<= 1;
  const int P = NTHR / Bq;
  const int b = t & (Bq - 1), part = t / Bq;
  const bool ok = b < B;
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    const int i = part + u * P;
    const bool in = ok && i < nss;
    const float x = ss[(size_t)(in ? i : 0) * B + (ok ? b : 0)];
    ld.v[u] = in ? x : 0.f;
  }
}

template <int NTHR>
__device__ __forceinline__ void rms_finish(const float *__restrict__ ss, int nss, int B, int H,
                                           float eps, const RmsLoads &ld, float *part_s,
                                           float *inv_s) {
  const int t = threadIdx.x;
  int Bq = 1;
  while (Bq < B) Bq <<= 1;
  const int P = NTHR / Bq;
  const int b = t & (Bq - 1), part = t / Bq;
  float v = 0.f;
#pragma unroll
  for (int u = 0; u < 16; ++u) v += ld.v[u];
  if (b < B) rms_tail(ss, B, b, part + 16 * P, P, nss, v);
  part_s[t] = v;
  __syncthreads();
  if (t < B) {
    float s = 0.f;
    for (int k = 0; k < P; ++k) s += part_s[k * Bq + t];
    inv_s[t] = 1.0f / sqrtf(s / (float)H + eps);
  }
  __syncthreads();
}

// ------------------------------------------------------------- GEMV with fused epilogue

// The projections and the element-wise steps that follow them run in one kernel: a block owns
// MT row tiles over the whole input; its WPB waves split the input blocks into contiguous ranges
// (weights double buffered in batches of U, the operand read from memory), each wave adds the
// hi and lo halves of every candidate (B <= 8: columns b and 8 + b of the one operand tile;
// otherwise tiles g and NT/2 + g hold the hi and lo halves of candidates 16 g .. 16 g + 15),
// the waves' sums are added in LDS in a fixed order, and wave g applies the epilogue to the
// complete outputs of candidate group g, so no split-K partials cross a kernel boundary.
//   EPI_RESID:  one tile: x += y, the tile's sums of squares per candidate, next operand
//               x * gamma (if gamma).
//   EPI_SWIGLU: gate tile t and up tile t: h = silu(r g) * (r u) as the down operand.
//   EPI_ROPE:   tile t and tile t + d/32 of one q/k/v head (the two halves of its rotary
//               pairs): q, k_self, v_self = rotary(r y) written as fp32 (no rotation for v).
enum { EPI_RESID = 1, EPI_SWIGLU = 2, EPI_ROPE = 3 };

struct FusedArgs {
  const void *w[3];  // weight segments (packed layout), stacked rows
  int seg_rows[3];
  int nseg;
  int K;
  const uint4 *act;  // operand [K / 32][NT][64]
  int B;
  // epilogue
  float *x;                  // residual [B][H] (RESID)
  float *xsave;              // a copy of the updated residual (RESID, may be null)
  int H;
  float *ss;                 // sums of squares: written per 16-row tile (RESID), read (SWIGLU)
  int nss;
  float eps;
  const void *gamma;         // bf16 gain of the next RMSNorm (RESID), may be null
  uint16_t *op;              // next operand (RESID, SWIGLU)
  int NT, Bp;                // layout of the next operand
  int F;
  // adapter tail (tkb > 0): tkb more input blocks from the segments' B factors (packed
  // [rows_i][32 tkb], null = no adapter) with operand slot i of tact as input
  const void *tw[3];
  const uint4 *tact;
  int tkb, tstride;
  float *save;  // SWIGLU: gate / up pre-activations [B][2F] (may be null)
  // ROPE: outputs [B][nq | nkv][d] and the rotary table [B][d/2][cos, sin]
  float *q, *ks, *vs;
  const float *rope;
  int nq, nkv, d;
};

template <int MT, int NT, int WPB, int U, int EPI>
__global__ __launch_bounds__(64 * WPB) void k_gemv_fused(FusedArgs a) {
  constexpr int NG = NT == 1 ? 1 : NT / 2;  // candidate groups
  static_assert(NG <= WPB, "one wave per candidate group in the epilogue");
  __shared__ floatx4 red_s[WPB][MT][NG][64];
  __shared__ float part_s[64 * WPB];
  __shared__ float inv_s[64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int B = a.B;
  // global row tiles of this block
  int tile[MT];
  tile[0] = blockIdx.x;
  if (EPI == EPI_RESID)  // MT consecutive row tiles
#pragma unroll
    for (int m = 0; m < MT; ++m) tile[m] = blockIdx.x * MT + m;
  if (EPI == EPI_SWIGLU && MT > 1) tile[MT - 1] = blockIdx.x + a.F / 16;
  if (EPI == EPI_ROPE) {  // block = (head, tile of the head's first half)
    const int half = a.d / 32;
    tile[0] = (blockIdx.x / half) * (a.d / 16) + blockIdx.x % half;
    tile[MT - 1] = tile[0] + half;
  }
  const uint4 *wt[MT];
  size_t kstride[MT];
  int segm[MT], ltm[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    int seg = 0, base = 0;
    while (seg < a.nseg - 1 && tile[m] * 16 >= base + a.seg_rows[seg]) base += a.seg_rows[seg++];
    const size_t ntiles = (size_t)a.seg_rows[seg] / 16;
    kstride[m] = ntiles * 64;
    wt[m] = (const uint4 *)a.w[seg] + (size_t)(tile[m] - base / 16) * 64 + lane;
    segm[m] = seg;
    ltm[m] = tile[m] - base / 16;
  }
  // this wave's input blocks [kb0, kb1)
  const int nkb = a.K >> 5;
  const int per = (nkb + WPB - 1) / WPB;
  const int kb0 = min(nkb, wave * per), kb1 = min(nkb, kb0 + per);
  const uint4 *ap = a.act + lane;
  // the epilogue's sums of squares are fetched now and used after the product: by wave 0
  // alone for one column tile (B <= 8), by the whole block for two
  WaveRmsLoads wl;
  RmsLoads rl;
  constexpr bool RMS = EPI == EPI_SWIGLU || EPI == EPI_ROPE;  // RMSNorm scale in the epilogue
  if (RMS && NT == 1 && wave == 0) wave_rms_load(a.ss, a.nss, B, wl);
  if (RMS && NT >= 2) rms_load<64 * WPB>(a.ss, a.nss, B, rl);
  floatx4 acc[MT][NT];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[m][t] = floatx4{0.f, 0.f, 0.f, 0.f};
  auto load_batch = [&](int kb, uint4(&av)[U][MT], uint4(&bv)[U][NT]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int m = 0; m < MT; ++m) av[u][m] = ld_stream(&wt[m][(size_t)(kb + u) * kstride[m]]);
#pragma unroll
      for (int t = 0; t < NT; ++t) bv[u][t] = ap[((size_t)(kb + u) * NT + t) * 64];
    }
  };
  auto mma_batch = [&](const uint4(&av)[U][MT], const uint4(&bv)[U][NT]) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[m][t] = mfma16(av[u][m], bv[u][t], acc[m][t]);
  };
  const int nbat = (kb1 - kb0) / U;
  if (nbat > 0) {
    uint4 a0[U][MT], a1[U][MT], b0[U][NT], b1[U][NT];
    load_batch(kb0, a0, b0);
    int i = 0;
    for (; i + 2 <= nbat; i += 2) {
      load_batch(kb0 + (i + 1) * U, a1, b1);
      __builtin_amdgcn_sched_barrier(0);
      mma_batch(a0, b0);
      __builtin_amdgcn_sched_barrier(0);
      load_batch(kb0 + min(i + 2, nbat - 1) * U, a0, b0);
      __builtin_amdgcn_sched_barrier(0);
      mma_batch(a1, b1);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (i < nbat) mma_batch(a0, b0);
  }
  for (int kb = kb0 + nbat * U; kb < kb1; ++kb) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const uint4 bv = ap[((size_t)kb * NT + t) * 64];
#pragma unroll
      for (int m = 0; m < MT; ++m)
        acc[m][t] = mfma16(ld_stream(&wt[m][(size_t)kb * kstride[m]]), bv, acc[m][t]);
    }
  }
  // adapter tail: B_seg (scale * A_seg u), its tkb input blocks spread over the waves
  if (a.tkb > 0) {
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const uint4 *bw = (const uint4 *)a.tw[segm[m]];
      if (!bw) continue;
      bw += (size_t)ltm[m] * 64 + lane;
      const uint4 *tp = a.tact + (size_t)segm[m] * a.tstride + lane;
      for (int kb = wave; kb < a.tkb; kb += WPB) {
        const uint4 av = ld_stream(&bw[(size_t)kb * kstride[m]]);
#pragma unroll
        for (int t = 0; t < NT; ++t)
          acc[m][t] = mfma16(av, tp[((size_t)kb * NT + t) * 64], acc[m][t]);
      }
    }
  }
  // hi + lo, then the waves' sums in LDS
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int gi = 0; gi < NG; ++gi) {
      floatx4 v;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        v[i] = NT == 1 ? acc[m][0][i] + __shfl_xor(acc[m][0][i], 8, 64)
                       : acc[m][gi][i] + acc[m][gi + NG][i];
      red_s[wave][m][gi][lane] = v;
    }
  __syncthreads();
  if (RMS && NT >= 2) rms_finish<64 * WPB>(a.ss, a.nss, B, a.H, a.eps, rl, part_s, inv_s);
  if (wave >= NG) return;
  const int gi = wave;
  // fixed-order sum over the waves; lane (n, cq) holds rows 4 cq .. 4 cq + 3 of candidate n of
  // group gi
  const int n = lane & 15, cq = lane >> 4;
  float y[MT][4];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    floatx4 tt = red_s[0][m][gi][lane];
#pragma unroll
    for (int w = 1; w < WPB; ++w) {
      const floatx4 v = red_s[w][m][gi][lane];
      tt[0] += v[0];
      tt[1] += v[1];
      tt[2] += v[2];
      tt[3] += v[3];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) y[m][i] = tt[i];
  }
  const int cand = NT == 1 ? n : 16 * gi + n;
  const bool cand_ok = NT == 1 ? (n < 8 && n < B) : cand < B;
  const int b = cand_ok ? cand : 0;
  if (EPI == EPI_RESID) {
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      float sq = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = tile[m] * 16 + 4 * cq + i;
        float xv = 0.f;
        if (cand_ok) {
          xv = a.x[(size_t)b * a.H + r] + y[m][i];
          a.x[(size_t)b * a.H + r] = xv;
          if (a.xsave) a.xsave[(size_t)b * a.H + r] = xv;
          if (a.gamma) store_operand(a.op, a.NT, a.Bp, r, b, xv * ld_bf16(a.gamma, r));
        }
        sq += xv * xv;
      }
      // rows of the tile: the 4 lane groups cq, in a fixed order
      sq += __shfl_xor(sq, 16, 64);
      sq += __shfl_xor(sq, 32, 64);
      if (cand_ok && cq == 0) a.ss[(size_t)tile[m] * B + b] = sq;
    }
  } else if (EPI == EPI_ROPE) {
    const float inv = NT == 1 ? wave_rms_finish(a.ss, a.nss, B, b, a.H, a.eps, wl) : inv_s[b];
    const int d = a.d, hd = d / 2;
    const int head = tile[0] / (d / 16);
    const bool rot = head < a.nq + a.nkv;  // q and k heads rotate, v heads do not
    float *dst = head < a.nq ? a.q + ((size_t)b * a.nq + head) * d
                 : head < a.nq + a.nkv ? a.ks + ((size_t)b * a.nkv + head - a.nq) * d
                                       : a.vs + ((size_t)b * a.nkv + head - a.nq - a.nkv) * d;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int di = tile[0] * 16 + 4 * cq + i - head * d;  // dimension in the first half
      const float y1 = y[0][i] * inv, y2 = y[MT - 1][i] * inv;
      const float2 csn = *(const float2 *)(a.rope + ((size_t)b * hd + di) * 2);
      if (cand_ok) {
        dst[di] = rot ? y1 * csn.x - y2 * csn.y : y1;
        dst[di + hd] = rot ? y2 * csn.x + y1 * csn.y : y2;
      }
    }
  } else {  // EPI_SWIGLU
    const float inv = NT == 1 ? wave_rms_finish(a.ss, a.nss, B, b, a.H, a.eps, wl) : inv_s[b];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int f = tile[0] * 16 + 4 * cq + i;
      const float gv = y[0][i] * inv, uv = y[MT - 1][i] * inv;
      if (cand_ok) store_operand(a.op, a.NT, a.Bp, f, b, gv / (1.0f + expf(-gv)) * uv);
      if (cand_ok && a.save) {
        a.save[(size_t)b * 2 * a.F + f] = gv;
        a.save[(size_t)b * 2 * a.F + a.F + f] = uv;
      }
    }
  }
}

// Gate/up + SwiGLU for 16 candidates or fewer whose input is a whole number of batches. Every input
// block brings NT KiB of operand for 2 KiB of gate/up weights, and k_gemv_fused, whose waves
// split the input range, reads each operand tile from L2 once per wave. Here the waves of a block
// own whole row tiles over the full input range instead (waves 0 .. WPB/2 - 1 gate tiles t0 + w,
// the others the matching up tiles) and share every input block's operand tiles through LDS,
// read from L2 once per block; the launcher sizes blocks so that each compute unit holds at most
// one where possible. Batches of U input blocks are double buffered: while the matrix cores work on
// batch i (operand from one LDS buffer, weights in registers), batch i+1's operand tiles go into
// the other buffer and batch i+2's loads are issued. Each output is a complete sum over the
// input (added in a different order than k_gemv_fused's); the up waves hand their sums to the
// gate waves through LDS for the SwiGLU epilogue.
template <int NT, int WPB, int U>
__global__ __launch_bounds__(64 * WPB, 4) void k_gateup_wide(FusedArgs a) {
  // candidate groups: with one column tile (B <= 8) columns b and 8 + b hold the hi and lo
  // halves of candidate b; otherwise tiles g and NT/2 + g those of candidates 16 g .. 16 g + 15
  constexpr int NG = NT == 1 ? 1 : NT / 2;
  constexpr int HALF = WPB / 2;      // gate/up tile pairs per block
  constexpr int PIECES = U * NT * 64;                     // 16-byte operand pieces per batch
  constexpr int PER = (PIECES + 64 * WPB - 1) / (64 * WPB);  // per thread (the last partly)
  constexpr bool EVEN = PER * 64 * WPB == PIECES;
  // the up waves' sums (HALF x NG x 64 float4) go through the two operand buffers (2 x U x NT x
  // 64 16-byte entries)
  static_assert(2 * U * NT >= HALF * NG, "the up sums fit in the operand buffers");
  __shared__ uint4 op_s[2][U * NT * 64];
  __shared__ float part_s[64 * WPB];
  __shared__ float inv_s[64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int B = a.B;
  const int ntf = a.F / 16;
  const bool up = wave >= HALF;
  const int pair = (int)blockIdx.x * HALF + (up ? wave - HALF : wave);
  const bool own = pair < ntf;
  const int tl = own ? pair : ntf - 1;  // past the end: repeat the last tile (results unused)
  const size_t kstride = (size_t)ntf * 64;
  const uint4 *wp = (const uint4 *)a.w[up ? 1 : 0] + (size_t)tl * 64 + lane;
  const int nbat = (a.K >> 5) / U;  // the launcher guarantees K / 32 % U == 0
  RmsLoads rl;
  rms_load<64 * WPB>(a.ss, a.nss, B, rl);
  floatx4 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  uint4 wa[U], wb[U];
  u32x4 ov[PER];
  auto load_w = [&](int bat, uint4(&w)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) w[u] = ld_stream(&wp[(size_t)(bat * U + u) * kstride]);
  };
  // (the staging registers are plain vectors passed explicitly: as uint4 captured by reference
  // they were kept in scratch memory)
  auto load_op = [&](int bat, u32x4(&o)[PER]) {  // operand [K/32][NT][64]: a batch is U * NT * 64
    const u32x4 *src = (const u32x4 *)a.act + (size_t)bat * PIECES;  // pieces
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = threadIdx.x + i * 64 * WPB;
      o[i] = src[EVEN || e < PIECES ? e : PIECES - 1];  // (a piece past the batch is not stored)
    }
  };
  auto store_op = [&](int buf, const u32x4(&o)[PER]) {
    u32x4 *dst = (u32x4 *)&op_s[buf][0];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = threadIdx.x + i * 64 * WPB;
      if (EVEN || e < PIECES) dst[e] = o[i];
    }
  };
  auto mma = [&](int buf, const uint4(&w)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[t] = mfma16(w[u], op_s[buf][(u * NT + t) * 64 + lane], acc[t]);
  };
  // batch i's operand is loaded into registers one batch before it is stored to LDS, and its
  // weights two batches before they are used, so that each load has a whole batch of products
  // and a barrier to arrive
  load_op(0, ov);
  store_op(0, ov);
  load_w(0, wa);
  if (nbat > 1) {
    load_op(1, ov);
    load_w(1, wb);
  }
  __syncthreads();
  for (int bat = 0; bat < nbat; bat += 2) {  // block-uniform trip counts and barriers
    mma(0, wa);
    if (bat + 1 < nbat) store_op(1, ov);  // buffer 1 was last read before the previous barrier
    if (bat + 2 < nbat) {
      load_op(bat + 2, ov);
      load_w(bat + 2, wa);
    }
    __syncthreads();
    if (bat + 1 >= nbat) break;
    mma(1, wb);
    if (bat + 2 < nbat) store_op(0, ov);
    if (bat + 3 < nbat) {
      load_op(bat + 3, ov);
      load_w(bat + 3, wb);
    }
    __syncthreads();
  }
  // adapter tail: B_seg (scale * A_seg u) of this wave's segment, operands from L2
  const int seg = up ? 1 : 0;
  if (a.tkb > 0 && a.tw[seg]) {
    const uint4 *bw = (const uint4 *)a.tw[seg] + (size_t)tl * 64 + lane;
    const uint4 *tp = a.tact + (size_t)seg * a.tstride + lane;
    for (int kb = 0; kb < a.tkb; ++kb) {
      const uint4 av = ld_stream(&bw[(size_t)kb * kstride]);
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[t] = mfma16(av, tp[((size_t)kb * NT + t) * 64], acc[t]);
    }
  }
  // hi + lo per candidate group; the up waves leave theirs in LDS (the operand buffers are free:
  // the last barrier of the loop follows their last read)
  float4 *xch = (float4 *)&op_s[0][0];  // [HALF][NG][64]
  float hl[NG][4];  // hi + lo (every lane, before any branch: the one-tile case shuffles)
#pragma unroll
  for (int gi = 0; gi < NG; ++gi)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      hl[gi][i] = NT == 1 ? acc[0][i] + __shfl_xor(acc[0][i], 8, 64) : acc[gi][i] + acc[gi + NG][i];
  if (up) {
#pragma unroll
    for (int gi = 0; gi < NG; ++gi)
      xch[((wave - HALF) * NG + gi) * 64 + lane] = make_float4(hl[gi][0], hl[gi][1], hl[gi][2], hl[gi][3]);
  }
  rms_finish<64 * WPB>(a.ss, a.nss, B, a.H, a.eps, rl, part_s, inv_s);  // has barriers
  if (up || !own) return;
  const int n = lane & 15, cq = lane >> 4;
#pragma unroll
  for (int gi = 0; gi < NG; ++gi) {
    const int cand = NT == 1 ? n : 16 * gi + n;
    if (cand >= B || (NT == 1 && n >= 8)) continue;
    const float inv = inv_s[cand];
    const float4 uvv = xch[(wave * NG + gi) * 64 + lane];
    const float uv4[4] = {uvv.x, uvv.y, uvv.z, uvv.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int f = tl * 16 + 4 * cq + i;
      const float gv = hl[gi][i] * inv;
      const float uv = uv4[i] * inv;
      store_operand(a.op, a.NT, a.Bp, f, cand, gv / (1.0f + expf(-gv)) * uv);
      if (a.save) {
        a.save[(size_t)cand * 2 * a.F + f] = gv;
        a.save[(size_t)cand * 2 * a.F + a.F + f] = uv;
      }
    }
  }
}

// Gate/up + SwiGLU for more than 16 candidates (NT >= 4 column tiles). With NT operand tiles per
// input block a wave that owns one row tile reads NT KiB of operand from LDS for each KiB of
// weights; here wave w of the block owns gate/up tile pair blockIdx.x WPB + w whole, so each
// operand tile it reads from LDS feeds two products (the gate's and the up's) and the SwiGLU
// epilogue needs no exchange between waves. Staging as in k_gateup_wide: batches of U input
// blocks of the operand double buffered in LDS, the weights two batches ahead in registers.
template <int NT, int WPB, int U>
__global__ __launch_bounds__(64 * WPB, 1) void k_gateup_pair(FusedArgs a) {
  constexpr int NG = NT / 2;
  constexpr int PIECES = U * NT * 64;
  constexpr int PER = (PIECES + 64 * WPB - 1) / (64 * WPB);
  constexpr bool EVEN = PER * 64 * WPB == PIECES;
  __shared__ uint4 op_s[2][U * NT * 64];
  __shared__ float part_s[64 * WPB];
  __shared__ float inv_s[64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int B = a.B;
  const int ntf = a.F / 16;
  const int pair = (int)blockIdx.x * WPB + wave;
  const bool own = pair < ntf;
  const int tl = own ? pair : ntf - 1;  // past the end: repeat the last pair (results unused)
  const size_t kstride = (size_t)ntf * 64;
  const uint4 *wpg = (const uint4 *)a.w[0] + (size_t)tl * 64 + lane;
  const uint4 *wpu = (const uint4 *)a.w[1] + (size_t)tl * 64 + lane;
  const int nbat = (a.K >> 5) / U;  // the launcher guarantees K / 32 % U == 0
  RmsLoads rl;
  rms_load<64 * WPB>(a.ss, a.nss, B, rl);
  floatx4 acc[2][NT];
#pragma unroll
  for (int m = 0; m < 2; ++m)
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[m][t] = floatx4{0.f, 0.f, 0.f, 0.f};
  uint4 wa[2][U], wb[2][U];
  u32x4 ov[PER];
  auto load_w = [&](int bat, uint4(&w)[2][U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      w[0][u] = ld_stream(&wpg[(size_t)(bat * U + u) * kstride]);
      w[1][u] = ld_stream(&wpu[(size_t)(bat * U + u) * kstride]);
    }
  };
  auto load_op = [&](int bat, u32x4(&o)[PER]) {
    const u32x4 *src = (const u32x4 *)a.act + (size_t)bat * PIECES;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = threadIdx.x + i * 64 * WPB;
      o[i] = src[EVEN || e < PIECES ? e : PIECES - 1];
    }
  };
  auto store_op = [&](int buf, const u32x4(&o)[PER]) {
    u32x4 *dst = (u32x4 *)&op_s[buf][0];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = threadIdx.x + i * 64 * WPB;
      if (EVEN || e < PIECES) dst[e] = o[i];
    }
  };
  // the products of batch buf with weights w; each input block's weight registers are reloaded
  // with batch nb's as soon as its products are issued, so that the weight stream does not wait
  // for the whole batch of products
  // (the operand tiles of input block u + 1 are read from LDS while block u's products issue)
  auto mma = [&](int buf, uint4(&w)[2][U], int nb) {
    uint4 o[2][NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) o[0][t] = op_s[buf][t * 64 + lane];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (u + 1 < U) {
#pragma unroll
        for (int t = 0; t < NT; ++t) o[(u + 1) & 1][t] = op_s[buf][((u + 1) * NT + t) * 64 + lane];
      }
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        acc[0][t] = mfma16(w[0][u], o[u & 1][t], acc[0][t]);
        acc[1][t] = mfma16(w[1][u], o[u & 1][t], acc[1][t]);
      }
      if (nb < nbat) {
        w[0][u] = ld_stream(&wpg[(size_t)(nb * U + u) * kstride]);
        w[1][u] = ld_stream(&wpu[(size_t)(nb * U + u) * kstride]);
      }
    }
  };
  load_op(0, ov);
  store_op(0, ov);
  load_w(0, wa);
  if (nbat > 1) {
    load_op(1, ov);
    load_w(1, wb);
  }
  __syncthreads();
  for (int bat = 0; bat < nbat; bat += 2) {  // block-uniform trip counts and barriers
    mma(0, wa, bat + 2);
    if (bat + 1 < nbat) store_op(1, ov);
    if (bat + 2 < nbat) load_op(bat + 2, ov);
    __syncthreads();
    if (bat + 1 >= nbat) break;
    mma(1, wb, bat + 3);
    if (bat + 2 < nbat) store_op(0, ov);
    if (bat + 3 < nbat) load_op(bat + 3, ov);
    __syncthreads();
  }
  // adapter tail: B_seg (scale * A_seg u) of each segment, operands from L2
  if (a.tkb > 0) {
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      if (!a.tw[m]) continue;
      const uint4 *bw = (const uint4 *)a.tw[m] + (size_t)tl * 64 + lane;
      const uint4 *tp = a.tact + (size_t)m * a.tstride + lane;
      for (int kb = 0; kb < a.tkb; ++kb) {
        const uint4 av = ld_stream(&bw[(size_t)kb * kstride]);
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[m][t] = mfma16(av, tp[((size_t)kb * NT + t) * 64], acc[m][t]);
      }
    }
  }
  rms_finish<64 * WPB>(a.ss, a.nss, B, a.H, a.eps, rl, part_s, inv_s);  // has barriers
  if (!own) return;
  const int n = lane & 15, cq = lane >> 4;
#pragma unroll
  for (int gi = 0; gi < NG; ++gi) {
    const int cand = 16 * gi + n;
    if (cand >= B) continue;
    const float inv = inv_s[cand];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int f = tl * 16 + 4 * cq + i;
      const float gv = (acc[0][gi][i] + acc[0][gi + NG][i]) * inv;
      const float uv = (acc[1][gi][i] + acc[1][gi + NG][i]) * inv;
      store_operand(a.op, a.NT, a.Bp, f, cand, gv / (1.0f + expf(-gv)) * uv);
      if (a.save) {
        a.save[(size_t)cand * 2 * a.F + f] = gv;
        a.save[(size_t)cand * 2 * a.F + a.F + f] = uv;
      }
    }
  }
}

// Split-K projection (q/k/v, output, down) for more than 16 candidates. At NT >= 4 column tiles
// every input block brings NT KiB of operand for each 1 KiB weight tile, and a block that owns
// one row tile (or tile pair) over the whole input (k_gemv_fused) pulls its whole operand from
// L2 for a few hundredth of the weights. Here block (g, ks) owns row tiles g WPB .. g WPB + WPB
// - 1 (one per wave; the rows may stack up to three weight segments) over input slice ks: each
// batch of U input blocks of the operand is staged once in LDS and read by all WPB waves (double
// buffered, loaded one batch ahead; the weights two batches ahead, as in k_gateup_wide), and the
// plan sizes the grid at about one block per compute unit. Each wave writes its tile's slice
// sums (hi + lo) to part[ks][candidate][row]; k_resid_split_fin (output, down: the residual
// epilogue) or k_qkv_split_fin (q/k/v: RMSNorm scale and rotation) adds the slices in order.
struct SplitArgs {
  const void *w[3];  // packed weight segments (e.g. q, k, v), stacked rows
  int seg_rows[3];
  int nseg;
  int rows, nkb;     // row count (all segments), input blocks of 32
  int kb_per;        // input blocks per slice (a multiple of U)
  const uint4 *act;  // operand [K / 32][NT][64]
  int B;
  float *part;       // [ksplit (+ 1 with an adapter)][B][rows]
  // adapter tail (tkb > 0): slice ksplit (the grid's last) runs the tkb input blocks of the
  // segments' B factors (packed [rows_i][32 tkb], null = no adapter) against operand slot i of
  // tact, as k_gemv_fused's tail does
  int ksplit;
  const void *tw[3];
  const uint4 *tact;
  int tkb, tstride;
};

template <int NT, int WPB, int U>
__global__ __launch_bounds__(64 * WPB) void k_resid_split(SplitArgs a) {
  // candidate groups: one column tile (B <= 8) holds the hi and lo halves of candidate b in
  // columns b and 8 + b; otherwise tiles g and NG + g those of candidates 16 g .. 16 g + 15
  constexpr int NG = NT == 1 ? 1 : NT / 2;
  constexpr int PIECES = U * NT * 64;  // 16-byte operand pieces per batch
  constexpr int PER = PIECES / (64 * WPB);
  static_assert(PER >= 1 && PER * 64 * WPB == PIECES, "operand batch split evenly over the block");
  __shared__ uint4 op_s[2][U * NT * 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int ks = blockIdx.y;
  const int kb0 = ks * a.kb_per;
  const int nbat = min(a.kb_per, a.nkb - kb0) / U;
  const int tile = (int)blockIdx.x * WPB + wave;
  const bool own = tile < a.rows / 16;
  const int tl = own ? tile : a.rows / 16 - 1;  // past the end: repeat the last tile (not stored)
  int seg = 0, base = 0;  // the tile's weight segment
  while (seg < a.nseg - 1 && tl * 16 >= base + a.seg_rows[seg]) base += a.seg_rows[seg++];
  const size_t ntiles = (size_t)a.seg_rows[seg] / 16;
  const size_t kstride = ntiles * 64;
  const uint4 *wp = (const uint4 *)a.w[seg] + ((size_t)kb0 * ntiles + (tl - base / 16)) * 64 + lane;
  const u32x4 *src = (const u32x4 *)a.act + (size_t)kb0 * NT * 64 + threadIdx.x;
  floatx4 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  if (ks == a.ksplit) {  // the adapter tail slice (block-uniform: no barriers on this path)
    const uint4 *bw = (const uint4 *)a.tw[seg];
    if (bw && own) {
      bw += (size_t)(tl - base / 16) * 64 + lane;
      const uint4 *tp = a.tact + (size_t)seg * a.tstride + lane;
      for (int kb = 0; kb < a.tkb; ++kb) {
        const uint4 av = ld_stream(&bw[(size_t)kb * kstride]);
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[t] = mfma16(av, tp[((size_t)kb * NT + t) * 64], acc[t]);
      }
    }
  } else {
  uint4 wa[U], wb[U];
  u32x4 ov[PER];
  auto load_w = [&](int bat, uint4(&w)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) w[u] = ld_stream(&wp[(size_t)(bat * U + u) * kstride]);
  };
  auto load_op = [&](int bat, u32x4(&o)[PER]) {
#pragma unroll
    for (int i = 0; i < PER; ++i) o[i] = src[(size_t)bat * PIECES + i * 64 * WPB];
  };
  auto store_op = [&](int buf, const u32x4(&o)[PER]) {
    u32x4 *dst = (u32x4 *)&op_s[buf][0] + threadIdx.x;
#pragma unroll
    for (int i = 0; i < PER; ++i) dst[i * 64 * WPB] = o[i];
  };
  auto mma = [&](int buf, const uint4(&w)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[t] = mfma16(w[u], op_s[buf][(u * NT + t) * 64 + lane], acc[t]);
  };
  if (nbat > 0) {
    load_op(0, ov);
    store_op(0, ov);
    load_w(0, wa);
    if (nbat > 1) {
      load_op(1, ov);
      load_w(1, wb);
    }
  }
  __syncthreads();
  for (int bat = 0; bat < nbat; bat += 2) {  // block-uniform trip counts and barriers
    mma(0, wa);
    if (bat + 1 < nbat) store_op(1, ov);  // buffer 1 was last read before the previous barrier
    if (bat + 2 < nbat) {
      load_op(bat + 2, ov);
      load_w(bat + 2, wa);
    }
    __syncthreads();
    if (bat + 1 >= nbat) break;
    mma(1, wb);
    if (bat + 2 < nbat) store_op(0, ov);
    if (bat + 3 < nbat) {
      load_op(bat + 3, ov);
      load_w(bat + 3, wb);
    }
    __syncthreads();
  }
  }
  if (!own) return;  // (whole waves)
  // lane (n, cq) holds rows 4 cq .. 4 cq + 3 of the tile for column n
  const int n = lane & 15, cq = lane >> 4;
#pragma unroll
  for (int gi = 0; gi < NG; ++gi) {
    float hl[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      hl[i] = NT == 1 ? acc[0][i] + __shfl_xor(acc[0][i], 8, 64) : acc[gi][i] + acc[gi + NG][i];
    const int cand = NT == 1 ? n : 16 * gi + n;
    if (cand >= a.B || (NT == 1 && n >= 8)) continue;
    *(float4 *)(a.part + ((size_t)ks * a.B + cand) * a.rows + tile * 16 + 4 * cq) =
        make_float4(hl[0], hl[1], hl[2], hl[3]);
  }
}

// Residual epilogue of k_resid_split, one output (candidate b, row r) per thread, e = b H + r:
// y = the slice sums added in slice order, x += y, the next operand x * gamma (if gamma), and the
// sum of squares of the new x over each 16-row tile (16 consecutive lanes, a fixed shuffle order).
__global__ __launch_bounds__(256) void k_resid_split_fin(const float *__restrict__ part, int ksplit,
                                                         float *x, float *xsave, float *ss, int H,
                                                         int B, const void *gamma, uint16_t *op,
                                                         int NT, int Bp) {
  const int e = (int)blockIdx.x * 256 + threadIdx.x;
  if (e >= B * H) return;  // (whole 16-lane groups: H is a multiple of 16)
  const int b = e / H, r = e - b * H;
  const size_t stride = (size_t)B * H;
  float y = 0.f;
#pragma unroll 8
  for (int k = 0; k < ksplit; ++k) y += part[(size_t)k * stride + e];
  const float xv = x[e] + y;
  x[e] = xv;
  if (xsave) xsave[e] = xv;
  if (gamma) store_operand(op, NT, Bp, r, b, xv * ld_bf16(gamma, r));
  float sq = xv * xv;
  sq += __shfl_xor(sq, 1, 64);
  sq += __shfl_xor(sq, 2, 64);
  sq += __shfl_xor(sq, 4, 64);
  sq += __shfl_xor(sq, 8, 64);
  if ((r & 15) == 0) ss[(size_t)(r >> 4) * B + b] = sq;
}

// Rotary epilogue of the split q/k/v product (k_resid_split over the stacked q, k, v rows), one
// rotary pair (candidate b, head, i < d/2) per thread, consecutive threads on consecutive i: the
// slice sums of rows r and r + d/2 of the head added in slice order, times the candidate's
// RMSNorm scale (its sums of squares added by one wave: lane-strided, then a fixed butterfly),
// rotated (q and k heads; v heads are not) and stored as q, k_self or v_self (fp32).
__global__ __launch_bounds__(256) void k_qkv_split_fin(const float *__restrict__ part, int ksplit,
                                                       const float *__restrict__ ss, int nss,
                                                       int H, float eps, int B, int nq, int nkv,
                                                       int d, const float *__restrict__ rope,
                                                       float *__restrict__ q, float *__restrict__ ks,
                                                       float *__restrict__ vs) {
  const int hd = d / 2, nh = nq + 2 * nkv, rows = nh * d;
  const int e = (int)blockIdx.x * 256 + threadIdx.x;
  const bool act = e < B * nh * hd;
  const int ec = act ? e : 0;
  const int b = ec / (nh * hd), rem = ec - b * (nh * hd);
  const int head = rem / hd, i = rem - head * hd;
  const int r = head * d + i;
  // the wave's candidates: b of its first and last active lanes (a wave spans at most two, as
  // nh * hd >= 64); the sums of squares of both are added lane-strided by the whole wave
  const size_t stride = (size_t)B * rows;
  float y1 = 0.f, y2 = 0.f;
  const float *p1 = part + (size_t)b * rows + r;
#pragma unroll 8
  for (int k = 0; k < ksplit; ++k) {
    y1 += p1[(size_t)k * stride];
    y2 += p1[(size_t)k * stride + hd];
  }
  // (the wave's lanes hold nondecreasing candidates; the inactive tail takes the first one)
  int b1 = act ? b : 0;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) b1 = max(b1, __shfl_xor(b1, off, 64));
  const int lane = threadIdx.x & 63;
  const int b0 = __shfl(b, 0, 64);
  float s0 = 0.f, s1 = 0.f;
  for (int t = lane; t < nss; t += 64) {
    s0 += ss[(size_t)t * B + b0];
    if (b1 != b0) s1 += ss[(size_t)t * B + b1];
  }
  s0 = wsum(s0);
  s1 = wsum(s1);
  const float inv = 1.0f / sqrtf((b == b0 ? s0 : s1) / (float)H + eps);
  if (!act) return;
  const float2 csn = *(const float2 *)(rope + ((size_t)b * hd + i) * 2);
  const float x1 = y1 * inv, x2 = y2 * inv;
  const bool rot = head < nq + nkv;
  float *dst = head < nq ? q + ((size_t)b * nq + head) * d
               : head < nq + nkv ? ks + ((size_t)b * nkv + (head - nq)) * d
                                 : vs + ((size_t)b * nkv + (head - nq - nkv)) * d;
  dst[i] = rot ? x1 * csn.x - x2 * csn.y : x1;
  dst[i + hd] = rot ? x2 * csn.x + x1 * csn.y : x2;
}

__global__ __launch_bounds__(256) void k_pack_weight(const uint4 *src, uint4 *dst, int64_t rows,
                                                     int64_t K) {
  const int64_t ngroups = rows * K / 8;
  const int64_t ntiles = rows / 16;
  for (int64_t gidx = (int64_t)blockIdx.x * 256 + threadIdx.x; gidx < ngroups;
       gidx += (int64_t)gridDim.x * 256) {
    const int64_t l = gidx & 63, blk = gidx >> 6;
    const int64_t kb = blk / ntiles, t = blk - kb * ntiles;
    const int64_t r = 16 * t + (l & 15), k = 32 * kb + 8 * (l >> 4);
    dst[gidx] = src[(r * K + k) / 8];
  }
}

hipError_t launch_pack_weight(const void *src, void *dst, int64_t rows, int64_t K, hipStream_t s) {
  const int64_t ngroups = rows * K / 8;
  int64_t blocks = (ngroups + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_pack_weight, dim3((unsigned)blocks), dim3(256), 0, s, (const uint4 *)src,
                     (uint4 *)dst, rows, K);
  return hipGetLastError();
}

hipError_t launch_init_mx(const Dims &dm, const Plan &p, const Workspace &w, const void *ev,
                          const void *gamma0, const int32_t *lengths, hipStream_t s,
                          float *xsave) {
  hipLaunchKernelGGL(k_init_mx, dim3(p.nss), dim3(256), 0, s, w.x, w.ss, p.rb, ev, gamma0, dm.wdt,
                     p.B, dm.H, w.opA, p.nt, p.bp, lengths, p.kq, dm.theta, dm.d, w.rope, xsave);
  return hipGetLastError();
}

static hipError_t launch_gemv_mx(const Plan &p, const GemvPlan &gp, const void *w0, int r0,
                                 const void *w1, int r1, const void *w2, int r2,
                                 const uint16_t *act, float *part, hipStream_t s) {
  GemvArgs a;
  memset(&a, 0, sizeof a);
  a.w[0] = w0;
  a.w[1] = w1;
  a.w[2] = w2;
  a.seg_rows[0] = r0;
  a.seg_rows[1] = r1;
  a.seg_rows[2] = r2;
  a.nseg = w2 ? 3 : (w1 ? 2 : 1);
  a.rows = gp.rows;
  a.K = gp.K;
  a.kslice = gp.kslice;
  a.ksplit = gp.ksplit;
  a.act = (const uint4 *)act;
  a.B = p.B;
  a.part = part;
  a.ksp = (gp.ksplit + 3) & ~3;
  const int mt = gemv_mt(p.nt, gp.rows);
  // 4 waves per block; the operand k-slice is staged in LDS for one column tile and read
  // straight from memory (L2) for more (measured faster than staging it: LDS would cap
  // residency, and an LDS-streamed variant with 8 row tiles per block measured slower)
  constexpr int WPB = 4;
  const bool direct = p.nt >= 2;
  dim3 grid((gp.rows / 16 + WPB * mt - 1) / (WPB * mt), gp.ksplit);
  const size_t lds = direct ? 0 : (size_t)(gp.kslice / 32) * p.nt * 64 * sizeof(uint4);
#define KVPRM_G(MT_, NT_, U_)                                                                  \
  if (direct)                                                                                  \
    hipLaunchKernelGGL((k_gemv_mx<MT_, NT_, U_, WPB, true>), grid, dim3(64 * WPB), lds, s, a); \
  else                                                                                         \
    hipLaunchKernelGGL((k_gemv_mx<MT_, NT_, U_, WPB, false>), grid, dim3(64 * WPB), lds, s, a)
#define KVPRM_G2(NT_, U_) \
  if (mt == 2) {          \
    KVPRM_G(2, NT_, U_);  \
  } else {                \
    KVPRM_G(1, NT_, U_);  \
  }
  switch (p.nt) {
    case 1: KVPRM_G(1, 1, 4); break;
    case 2: KVPRM_G2(2, 4); break;
    case 4: KVPRM_G2(4, 2); break;
    case 6: KVPRM_G2(6, 2); break;
    case 8: KVPRM_G2(8, 2); break;
    default: return hipErrorInvalidValue;
  }
#undef KVPRM_G2
#undef KVPRM_G
  return hipGetLastError();
}

static int ksp_of(const GemvPlan &g) { return (g.ksplit + 3) & ~3; }

static FusedArgs fused_args(const Dims &dm, const Plan &p, const Workspace &w, int K,
                            const uint16_t *act);
static void set_tail(FusedArgs &a, const Plan &p, const Workspace &w, const LoraTail &tail);

// q, k_self, v_self in one launch: a block owns both halves of the rotary pairs of one head
// (tiles t and t + d/32) over the whole input and rotates them in its epilogue.
static hipError_t launch_qkv_rope_fused(const Dims &dm, const Plan &p, const Workspace &w,
                                        const void *wq, const void *wk, const void *wv,
                                        const LoraTail &tail, hipStream_t s) {
  FusedArgs a = fused_args(dm, p, w, dm.H, w.opA);
  set_tail(a, p, w, tail);
  a.w[0] = wq;
  a.w[1] = wk;
  a.w[2] = wv;
  a.seg_rows[0] = dm.nq * dm.d;
  a.seg_rows[1] = dm.nkv * dm.d;
  a.seg_rows[2] = dm.nkv * dm.d;
  a.nseg = 3;
  a.q = w.q;
  a.ks = w.kself;
  a.vs = w.vself;
  a.rope = w.rope;
  a.nq = dm.nq;
  a.nkv = dm.nkv;
  a.d = dm.d;
  const dim3 grid((dm.nq + 2 * dm.nkv) * (dm.d / 32));
  switch (p.nt) {
    case 1: hipLaunchKernelGGL((k_gemv_fused<2, 1, 8, 4, EPI_ROPE>), grid, dim3(64 * 8), 0, s, a); break;
    case 2: hipLaunchKernelGGL((k_gemv_fused<2, 2, 8, 4, EPI_ROPE>), grid, dim3(64 * 8), 0, s, a); break;
    case 4: hipLaunchKernelGGL((k_gemv_fused<2, 4, 8, 2, EPI_ROPE>), grid, dim3(64 * 8), 0, s, a); break;
    case 6: hipLaunchKernelGGL((k_gemv_fused<2, 6, 8, 1, EPI_ROPE>), grid, dim3(64 * 8), 0, s, a); break;
    case 8: hipLaunchKernelGGL((k_gemv_fused<2, 8, 8, 1, EPI_ROPE>), grid, dim3(64 * 8), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// q, k_self, v_self from the split-K partials of the stacked q/k/v product: the k-partials of
// rows r and r + d/2 of a head (the two halves of a rotary pair) added in k order, the RMSNorm
// scale of the candidate, the rotation (q and k heads) at the candidate's position. One thread
// per (row pair, candidate).
template <int NMAX>
__global__ __launch_bounds__(256) void k_qkv_fin_mx(const float *__restrict__ part, int ksp,
                                                    int ksplit, const float *__restrict__ ss,
                                                    int nss, int H, float eps, int B, int nq,
                                                    int nkv, int d, const float *__restrict__ rope,
                                                    float *__restrict__ q, float *__restrict__ ks,
                                                    float *__restrict__ vs) {
  __shared__ float part_s[256], inv_s[64];
  const int hd = d / 2;
  const int e = blockIdx.x * 256 + threadIdx.x;
  const bool act = e < (nq + 2 * nkv) * hd * B;
  const int ec = act ? e : 0;
  const int pr = ec / B, b = ec - pr * B;
  const int head = pr / hd, i = pr - head * hd;
  const int r = head * d + i;
  const size_t i1 = (size_t)r * B + b, i2 = (size_t)(r + hd) * B + b;
  float4 v1[NMAX], v2[NMAX];
  ksum_load<NMAX>(part, ksp, i1, v1);
  ksum_load<NMAX>(part, ksp, i2, v2);
  const float2 csn = *(const float2 *)(rope + ((size_t)b * hd + i) * 2);
  RmsLoads rl;
  rms_load<256>(ss, nss, B, rl);
  rms_finish<256>(ss, nss, B, H, eps, rl, part_s, inv_s);  // has barriers: every thread
  const float x1 = ksum_add<NMAX>(part, ksp, ksplit, i1, v1);
  const float x2 = ksum_add<NMAX>(part, ksp, ksplit, i2, v2);
  if (!act) return;
  const float inv = inv_s[b];
  const float y1 = x1 * inv, y2 = x2 * inv;
  const bool rot = head < nq + nkv;
  float *dst = head < nq ? q + ((size_t)b * nq + head) * d
               : head < nq + nkv ? ks + ((size_t)b * nkv + (head - nq)) * d
                                 : vs + ((size_t)b * nkv + (head - nq - nkv)) * d;
  dst[i] = rot ? y1 * csn.x - y2 * csn.y : y1;
  dst[i + hd] = rot ? y2 * csn.x + y1 * csn.y : y2;
}

static hipError_t launch_split(const Plan &p, const Workspace &w, const GemvPlan &g,
                               const void *w0, int r0, const void *w1, int r1, const void *w2,
                               int r2, const uint16_t *act, const LoraTail &tail, hipStream_t s);

hipError_t launch_qkv_mx(const Dims &dm, const Plan &p, const Workspace &w, const void *wq,
                         const void *wk, const void *wv, const LoraTail &tail, hipStream_t s) {
  if (p.rs_qkv) {  // split-K product (+ the adapter tail slice) and the rotary finish
    hipError_t e = launch_split(p, w, p.g_rs_qkv, wq, dm.nq * dm.d, wk, dm.nkv * dm.d, wv,
                                dm.nkv * dm.d, w.opA, tail, s);
    if (e != hipSuccess) return e;
    const int n = p.B * (dm.nq + 2 * dm.nkv) * (dm.d / 2);
    hipLaunchKernelGGL(k_qkv_split_fin, dim3((n + 255) / 256), dim3(256), 0, s, w.part,
                       p.g_rs_qkv.ksplit + (tail.tkb > 0 ? 1 : 0), w.ss, p.nss, dm.H, dm.eps,
                       p.B, dm.nq, dm.nkv, dm.d, w.rope, w.q, w.kself, w.vself);
    return hipGetLastError();
  }
  if (!p.qkv_split || tail.tkb > 0) return launch_qkv_rope_fused(dm, p, w, wq, wk, wv, tail, s);
  hipError_t e = launch_gemv_mx(p, p.g_qkv, wq, dm.nq * dm.d, wk, dm.nkv * dm.d, wv,
                                dm.nkv * dm.d, w.opA, w.part, s);
  if (e != hipSuccess) return e;
  const int n = (dm.nq + 2 * dm.nkv) * (dm.d / 2) * p.B;
  const int ksp = ksp_of(p.g_qkv);
#define KVPRM_F(NM)                                                                           \
  hipLaunchKernelGGL(k_qkv_fin_mx<NM>, dim3((n + 255) / 256), dim3(256), 0, s, w.part, ksp,   \
                     p.g_qkv.ksplit, w.ss, p.nss, dm.H, dm.eps, p.B, dm.nq, dm.nkv, dm.d,     \
                     w.rope, w.q, w.kself, w.vself)
  switch (ksum_nmax(ksp)) {
    case 1: KVPRM_F(1); break;
    case 2: KVPRM_F(2); break;
    case 4: KVPRM_F(4); break;
    default: KVPRM_F(8); break;
  }
#undef KVPRM_F
  return hipGetLastError();
}

// scale * (sum of the k-partials) of adapter row r (segment r / rank, index r % rank) for
// candidate b, stored into operand slot slot[segment] of topd. One thread per (row, candidate).
template <int NMAX>
__global__ __launch_bounds__(256) void k_lora_fin(const float *__restrict__ part, int ksp,
                                                  int ksplit, int rows, int B, int rank, int3 slot,
                                                  float scale, uint16_t *topd, int NT, int Bp,
                                                  size_t slot_elems) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= rows * B) return;
  float4 v[NMAX];
  ksum_load<NMAX>(part, ksp, (size_t)e, v);
  const float sum = ksum_add<NMAX>(part, ksp, ksplit, (size_t)e, v);
  const int r = e / B, b = e - r * B;
  const int seg = r / rank, k = r - seg * rank;
  const int sl = seg == 0 ? slot.x : (seg == 1 ? slot.y : slot.z);
  store_operand(topd + (size_t)sl * slot_elems, NT, Bp, k, b, scale * sum);
}

hipError_t launch_lora_a(const Dims &dm, const Plan &p, const Workspace &w, int group,
                         const void *const a[3], float scale, const uint16_t *act, hipStream_t s) {
  (void)dm;
  const void *seg[3] = {nullptr, nullptr, nullptr};
  int slot[3] = {0, 0, 0}, n = 0;
  for (int i = 0; i < 3; ++i)
    if (a[i]) {
      seg[n] = a[i];
      slot[n++] = i;
    }
  if (n == 0) return hipSuccess;
  const int r = p.lora_rank;
  GemvPlan g = p.g_la[group];
  g.rows = n * r;
  hipError_t e = launch_gemv_mx(p, g, seg[0], r, seg[1], n > 1 ? r : 0, seg[2], n > 2 ? r : 0,
                                act, w.part, s);
  if (e != hipSuccess) return e;
  const int cnt = g.rows * p.B;
  const size_t slot_elems = (size_t)(r / 32) * p.nt * 64 * 8;
  const int3 sl = make_int3(slot[0], slot[1], slot[2]);
#define KVPRM_L(NM)                                                                            \
  hipLaunchKernelGGL(k_lora_fin<NM>, dim3((cnt + 255) / 256), dim3(256), 0, s, w.part,         \
                     ksp_of(g), g.ksplit, g.rows, p.B, r, sl, scale, w.topd, p.nt, p.bp,       \
                     slot_elems)
  switch (ksum_nmax(ksp_of(g))) {
    case 1: KVPRM_L(1); break;
    case 2: KVPRM_L(2); break;
    case 4: KVPRM_L(4); break;
    default: KVPRM_L(8); break;
  }
#undef KVPRM_L
  return hipGetLastError();
}

static void set_tail(FusedArgs &a, const Plan &p, const Workspace &w, const LoraTail &tail) {
  for (int i = 0; i < 3; ++i) a.tw[i] = tail.b[i];
  a.tact = (const uint4 *)w.topd;
  a.tkb = tail.tkb;
  a.tstride = tail.tkb * p.nt * 64;
}

// fused projections
static hipError_t launch_resid_fused(const Plan &p, const FusedArgs &a, int tiles, hipStream_t s) {
  const dim3 grid(tiles);
  // two row tiles per wave, one operand read for both, when that still leaves a block for every
  // compute unit: two candidate tiles (9 to 16 candidates) and at least 512 row tiles (H = 8192:
  // 28.9 -> 26.7 ms per call of the large fp8 workload)
  if (p.nt == 2 && tiles % 2 == 0 && tiles >= 512) {
    hipLaunchKernelGGL((k_gemv_fused<2, 2, 8, 4, EPI_RESID>), dim3(tiles / 2), dim3(512), 0, s, a);
    return hipGetLastError();
  }
  switch (p.nt) {
    // (8 waves with batches of 2 input blocks: 9.2 -> 8.7 us per output projection of the
    // ragged batch of 8, against 16 x 4, 8 x 4, 16 x 2 and 16 x 1)
    case 1: hipLaunchKernelGGL((k_gemv_fused<1, 1, 8, 2, EPI_RESID>), grid, dim3(64 * 8), 0, s, a); break;
    // batches of 2 input blocks (74 registers): 4.20 -> 4.15 ms per call of the 7B batch of 16
    case 2: hipLaunchKernelGGL((k_gemv_fused<1, 2, 8, 2, EPI_RESID>), grid, dim3(64 * 8), 0, s, a); break;
    case 4: hipLaunchKernelGGL((k_gemv_fused<1, 4, 8, 2, EPI_RESID>), grid, dim3(64 * 8), 0, s, a); break;
    case 6: hipLaunchKernelGGL((k_gemv_fused<1, 6, 8, 1, EPI_RESID>), grid, dim3(64 * 8), 0, s, a); break;
    case 8: hipLaunchKernelGGL((k_gemv_fused<1, 8, 16, 1, EPI_RESID>), grid, dim3(64 * 16), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// k_resid_split over the plan's slices, then k_resid_split_fin (next operand into w.opA)
static hipError_t launch_split(const Plan &p, const Workspace &w, const GemvPlan &g,
                               const void *w0, int r0, const void *w1, int r1, const void *w2,
                               int r2, const uint16_t *act, const LoraTail &tail, hipStream_t s) {
  SplitArgs a;
  memset(&a, 0, sizeof a);
  a.w[0] = w0;
  a.w[1] = w1;
  a.w[2] = w2;
  a.seg_rows[0] = r0;
  a.seg_rows[1] = r1;
  a.seg_rows[2] = r2;
  a.nseg = w2 ? 3 : (w1 ? 2 : 1);
  a.rows = g.rows;
  a.nkb = g.K / 32;
  a.kb_per = g.kslice / 32;
  a.act = (const uint4 *)act;
  a.B = p.B;
  a.part = w.part;
  a.ksplit = g.ksplit;
  for (int i = 0; i < 3; ++i) a.tw[i] = tail.b[i];
  a.tact = (const uint4 *)w.topd;
  a.tkb = tail.tkb;
  a.tstride = tail.tkb * p.nt * 64;
  // (the plan's slices are whole batches of p.rs_u input blocks: U, or 8 or 16 with one column tile)
  constexpr int U = 4, WPB = 8;
  if (p.rs_wpb != WPB || (p.nt > 1 && p.rs_u != U)) return hipErrorInvalidValue;
  const dim3 grid((g.rows / 16 + WPB - 1) / WPB, g.ksplit + (tail.tkb > 0 ? 1 : 0));
  switch (p.nt) {
    case 1:
      if (p.rs_u == 16)
        hipLaunchKernelGGL((k_resid_split<1, WPB, 16>), grid, dim3(64 * WPB), 0, s, a);
      else if (p.rs_u == 8)
        hipLaunchKernelGGL((k_resid_split<1, WPB, 8>), grid, dim3(64 * WPB), 0, s, a);
      else
        return hipErrorInvalidValue;
      break;
    case 2: hipLaunchKernelGGL((k_resid_split<2, WPB, U>), grid, dim3(64 * WPB), 0, s, a); break;
    case 4: hipLaunchKernelGGL((k_resid_split<4, WPB, U>), grid, dim3(64 * WPB), 0, s, a); break;
    case 6: hipLaunchKernelGGL((k_resid_split<6, WPB, U>), grid, dim3(64 * WPB), 0, s, a); break;
    case 8: hipLaunchKernelGGL((k_resid_split<8, WPB, U>), grid, dim3(64 * WPB), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

static hipError_t launch_resid_split(const Dims &dm, const Plan &p, const Workspace &w,
                                     const GemvPlan &g, const void *wt, const uint16_t *act,
                                     const LoraTail &tail, const void *gamma, float *xsave,
                                     hipStream_t s) {
  hipError_t e = launch_split(p, w, g, wt, dm.H, nullptr, 0, nullptr, 0, act, tail, s);
  if (e != hipSuccess) return e;
  const int n = p.B * dm.H;
  hipLaunchKernelGGL(k_resid_split_fin, dim3((n + 255) / 256), dim3(256), 0, s, w.part,
                     g.ksplit + (tail.tkb > 0 ? 1 : 0), w.x, xsave, w.ss, dm.H, p.B, gamma,
                     w.opA, p.nt, p.bp);
  return hipGetLastError();
}

static FusedArgs fused_args(const Dims &dm, const Plan &p, const Workspace &w, int K,
                            const uint16_t *act) {
  FusedArgs a;
  memset(&a, 0, sizeof a);
  a.K = K;
  a.act = (const uint4 *)act;
  a.B = p.B;
  a.x = w.x;
  a.H = dm.H;
  a.ss = w.ss;
  a.nss = p.nss;
  a.eps = dm.eps;
  a.NT = p.nt;
  a.Bp = p.bp;
  a.F = dm.F;
  return a;
}

hipError_t launch_oproj_fused(const Dims &dm, const Plan &p, const Workspace &w, const void *wo,
                              const void *gamma_ffn, const LoraTail &tail, hipStream_t s,
                              float *xsave) {
  if (p.rs_o) return launch_resid_split(dm, p, w, p.g_rs_o, wo, w.opO, tail, gamma_ffn, xsave, s);
  FusedArgs a = fused_args(dm, p, w, dm.nq * dm.d, w.opO);
  a.xsave = xsave;
  set_tail(a, p, w, tail);
  a.w[0] = wo;
  a.seg_rows[0] = dm.H;
  a.nseg = 1;
  a.gamma = gamma_ffn;
  a.op = w.opA;
  return launch_resid_fused(p, a, dm.H / 16, s);
}

hipError_t launch_gateup_fused(const Dims &dm, const Plan &p, const Workspace &w, const void *wg,
                               const void *wu, const LoraTail &tail, hipStream_t s,
                               float *save_gu) {
  FusedArgs a = fused_args(dm, p, w, dm.H, w.opA);
  set_tail(a, p, w, tail);
  a.save = save_gu;
  a.w[0] = wg;
  a.w[1] = wu;
  a.seg_rows[0] = dm.F;
  a.seg_rows[1] = dm.F;
  a.nseg = 2;
  a.op = w.opD;
  const dim3 grid(dm.F / 16);
  // Shared-operand kernel (k_gateup_wide): HALF gate/up tile pairs per block (2 HALF waves),
  // chosen so that every compute unit gets at most one block where possible: with 4 pairs, the
  // 1184 pairs of the 7B shape make 296 blocks, and the 40 compute units holding two set the
  // kernel's length (beam: 5 pairs, 237 blocks: 8.42 -> 7.90 ms per call).
  constexpr int UW = 4;  // batch depth
  const int pairs = dm.F / 16;
  int half = (pairs + 255) / 256;
  half = half < 4 ? 4 : (half > 8 ? 8 : half);
  const dim3 wgrid((pairs + half - 1) / half);
  const bool wide = (dm.H / 32) % UW == 0;
  // more than 16 candidates: one gate/up pair per wave (k_gateup_pair), as many pairs per block
  // as k_gateup_wide's (beam batch of 64: 6.75 -> 6.59 ms per call)
  if (wide && p.nt >= 4) {
#define KVPRM_GP(NT_)                                                                                 \
  switch (half) {                                                                                  \
    case 4: hipLaunchKernelGGL((k_gateup_pair<NT_, 4, UW>), wgrid, dim3(256), 0, s, a); break;      \
    case 5: hipLaunchKernelGGL((k_gateup_pair<NT_, 5, UW>), wgrid, dim3(320), 0, s, a); break;      \
    case 6: hipLaunchKernelGGL((k_gateup_pair<NT_, 6, UW>), wgrid, dim3(384), 0, s, a); break;      \
    case 7: hipLaunchKernelGGL((k_gateup_pair<NT_, 7, UW>), wgrid, dim3(448), 0, s, a); break;      \
    default: hipLaunchKernelGGL((k_gateup_pair<NT_, 8, UW>), wgrid, dim3(512), 0, s, a); break;     \
  }
    if (p.nt == 4) KVPRM_GP(4)
    else if (p.nt == 6) KVPRM_GP(6)
    else KVPRM_GP(8)
#undef KVPRM_GP
    return hipGetLastError();
  }
#define KVPRM_GW(NT_)                                                                                \
  switch (half) {                                                                                 \
    case 4: hipLaunchKernelGGL((k_gateup_wide<NT_, 8, UW>), wgrid, dim3(512), 0, s, a); break;     \
    case 5: hipLaunchKernelGGL((k_gateup_wide<NT_, 10, UW>), wgrid, dim3(640), 0, s, a); break;    \
    case 6: hipLaunchKernelGGL((k_gateup_wide<NT_, 12, UW>), wgrid, dim3(768), 0, s, a); break;    \
    case 7: hipLaunchKernelGGL((k_gateup_wide<NT_, 14, UW>), wgrid, dim3(896), 0, s, a); break;    \
    default: hipLaunchKernelGGL((k_gateup_wide<NT_, 16, UW>), wgrid, dim3(1024), 0, s, a); break;  \
  }
  // with balanced blocks it is also the faster choice for 16 candidates or fewer (7B batch of 16:
  // 4.15 -> 3.86 ms per call; ragged batch of 8: about 2% faster); an input that is not a whole
  // number of batches takes k_gemv_fused
  if (wide) {
    if (p.nt == 1) KVPRM_GW(1)
    else KVPRM_GW(2)
    return hipGetLastError();
  }
  switch (p.nt) {
    case 1: hipLaunchKernelGGL((k_gemv_fused<2, 1, 4, 4, EPI_SWIGLU>), grid, dim3(64 * 4), 0, s, a); break;
    case 2: hipLaunchKernelGGL((k_gemv_fused<2, 2, 4, 4, EPI_SWIGLU>), grid, dim3(64 * 4), 0, s, a); break;
    case 4: hipLaunchKernelGGL((k_gemv_fused<2, 4, 4, 2, EPI_SWIGLU>), grid, dim3(64 * 4), 0, s, a); break;
    case 6: hipLaunchKernelGGL((k_gemv_fused<2, 6, 4, 1, EPI_SWIGLU>), grid, dim3(64 * 4), 0, s, a); break;
    case 8: hipLaunchKernelGGL((k_gemv_fused<2, 8, 4, 1, EPI_SWIGLU>), grid, dim3(64 * 4), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
#undef KVPRM_GW
  return hipGetLastError();
}

hipError_t launch_down_fused(const Dims &dm, const Plan &p, const Workspace &w, const void *wd,
                             const void *gamma_next, const LoraTail &tail, hipStream_t s,
                             float *xsave) {
  if (p.rs_d) return launch_resid_split(dm, p, w, p.g_rs_d, wd, w.opD, tail, gamma_next, xsave, s);
  FusedArgs a = fused_args(dm, p, w, dm.F, w.opD);
  a.xsave = xsave;
  set_tail(a, p, w, tail);
  a.w[0] = wd;
  a.seg_rows[0] = dm.H;
  a.nseg = 1;
  a.gamma = gamma_next;
  a.op = w.opA;
  return launch_resid_fused(p, a, dm.H / 16, s);
}

}  // namespace kvprm
