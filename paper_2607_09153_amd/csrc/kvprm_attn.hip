// Matrix-core attention of the verify-token pass for gfx950 (bf16 or fp8 e4m3 caches): the
// split-L paged chunk kernel over private pages (k_attn_mx), the shared-prefix kernel
// (k_prefix_mx) and the log-sum-exp merge with the token's own key (k_merge_mx).
#include <hip/hip_runtime.h>
#include <math.h>
#include <string.h>

#include <type_traits>

#include "kvprm_internal.h"
#include "kvprm_mx_common.h"

namespace kvprm {

// ------------------------------------------------------------------------------- attention

template <bool HIGH>
__device__ __forceinline__ uint32_t fp8x2_to_bf16x2(uint32_t word) {
  // two OCP e4m3 codes (bytes 0, 1 or 2, 3) -> two bf16 in one instruction; every e4m3 value is
  // a bf16 value and the scale is 1, so the conversion is exact
  typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
  const bf16x2v v = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(word, 1.0f, HIGH);
  return __builtin_bit_cast(uint32_t, v);
}

// Lane i's value of v, for a wave-uniform i (a scalar read of one lane: no LDS round trip).
__device__ __forceinline__ int lane_value(int v, int i) { return __builtin_amdgcn_readlane(v, i); }
__device__ __forceinline__ float lane_value(float v, int i) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), i));
}

// Raw registers of one page pair of one kv-head, in tile byte order (16 bytes per lane and
// instruction): K tiles of pages A and B, then their V tiles. bf16 uses D/32 of each, fp8 D/64.
template <int D>
struct PairRaw {
  uint4 k[2][D / 32];
  uint4 v[2][D / 32];
};

// Loads a pair from tile base pointers: global memory read once (STREAM, non-temporal), or LDS.
template <int KVT, int D, bool STREAM>
__device__ __forceinline__ void load_pair_raw(const uint4 *kA, const uint4 *kB, const uint4 *vA,
                                              const uint4 *vB, int lane, PairRaw<D> &r) {
  constexpr int N = KVT == 1 ? D / 32 : D / 64;
#pragma unroll
  for (int i = 0; i < N; ++i) {
    if (STREAM) {
      r.k[0][i] = ld_stream(kA + i * 64 + lane);
      r.k[1][i] = ld_stream(kB + i * 64 + lane);
      r.v[0][i] = ld_stream(vA + i * 64 + lane);
      r.v[1][i] = ld_stream(vB + i * 64 + lane);
    } else {
      r.k[0][i] = kA[i * 64 + lane];
      r.k[1][i] = kB[i * 64 + lane];
      r.v[0][i] = vA[i * 64 + lane];
      r.v[1][i] = vB[i * 64 + lane];
    }
  }
}

// Raw pair -> bf16 MFMA operands. K: lane holds token lane % 16, 8 dims per 32-dim block
// (bf16: dims 32kk + 8c + i; fp8: dims 16 (4 (kk/2) + c) + 8 (kk%2) + i). V (tile stores 4
// consecutive slots of r dims 16 apart): VA[nb] = slots 4c..4c+3 of dim 16 nb + lane % 16.
template <int KVT, int D>
__device__ __forceinline__ void unpack_pair(const PairRaw<D> &r, uint4 *KA, uint4 *KB, uint2 *VA,
                                            uint2 *VB) {
  constexpr int NKB = D / 32, NDB = D / 16;
  if (KVT == 1) {
#pragma unroll
    for (int kk = 0; kk < NKB; ++kk) {
      KA[kk] = r.k[0][kk];
      KB[kk] = r.k[1][kk];
    }
#pragma unroll
    for (int q2 = 0; q2 < NDB / 2; ++q2) {
      VA[2 * q2] = make_uint2(r.v[0][q2].x, r.v[0][q2].y);
      VA[2 * q2 + 1] = make_uint2(r.v[0][q2].z, r.v[0][q2].w);
      VB[2 * q2] = make_uint2(r.v[1][q2].x, r.v[1][q2].y);
      VB[2 * q2 + 1] = make_uint2(r.v[1][q2].z, r.v[1][q2].w);
    }
  } else {
#pragma unroll
    for (int kp = 0; kp < NKB / 2; ++kp) {
      const uint4 ra = r.k[0][kp], rb = r.k[1][kp];
      KA[2 * kp] = make_uint4(fp8x2_to_bf16x2<false>(ra.x), fp8x2_to_bf16x2<true>(ra.x),
                              fp8x2_to_bf16x2<false>(ra.y), fp8x2_to_bf16x2<true>(ra.y));
      KA[2 * kp + 1] = make_uint4(fp8x2_to_bf16x2<false>(ra.z), fp8x2_to_bf16x2<true>(ra.z),
                                  fp8x2_to_bf16x2<false>(ra.w), fp8x2_to_bf16x2<true>(ra.w));
      KB[2 * kp] = make_uint4(fp8x2_to_bf16x2<false>(rb.x), fp8x2_to_bf16x2<true>(rb.x),
                              fp8x2_to_bf16x2<false>(rb.y), fp8x2_to_bf16x2<true>(rb.y));
      KB[2 * kp + 1] = make_uint4(fp8x2_to_bf16x2<false>(rb.z), fp8x2_to_bf16x2<true>(rb.z),
                                  fp8x2_to_bf16x2<false>(rb.w), fp8x2_to_bf16x2<true>(rb.w));
    }
#pragma unroll
    for (int q4 = 0; q4 < NDB / 4; ++q4) {
      const uint32_t wa[4] = {r.v[0][q4].x, r.v[0][q4].y, r.v[0][q4].z, r.v[0][q4].w};
      const uint32_t wb[4] = {r.v[1][q4].x, r.v[1][q4].y, r.v[1][q4].z, r.v[1][q4].w};
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        VA[4 * q4 + jj] = make_uint2(fp8x2_to_bf16x2<false>(wa[jj]), fp8x2_to_bf16x2<true>(wa[jj]));
        VB[4 * q4 + jj] = make_uint2(fp8x2_to_bf16x2<false>(wb[jj]), fp8x2_to_bf16x2<true>(wb[jj]));
      }
    }
  }
}

// Query operands of one column (zero when absent), split in three bf16 terms so that the
// scores keep fp32-level accuracy even for very large logits. The dim order matches the K
// operand of the cache dtype.
template <int KVT, int D>
__device__ __forceinline__ void load_query_ops(const float *qr, bool present, int cq, uint4 *qhi,
                                               uint4 *qmd, uint4 *qlo) {
  constexpr int NKB = D / 32;
#pragma unroll
  for (int kk = 0; kk < NKB; ++kk) {
    uint32_t h[8], md[8], l[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int dim = (KVT == 1) ? kk * 32 + 8 * cq + i : 16 * (4 * (kk >> 1) + cq) + 8 * (kk & 1) + i;
      const float v = present ? qr[dim] : 0.f;
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

// One online-softmax step over a page pair for the 16 columns (queries) of a wave:
// S = K Q^T (lane holds tokens 4c + i of pages A and B for column lane % 16; q0, q1, q2 = the
// query's hi, mid, lo bf16 terms, three MFMAs per 32-dim block), running max and sum, then
// O^T += V^T P^T with P split hi + lo (two MFMAs per 16-dim block). Scores arrive scaled by
// log2(e) (sca, scb include it), so the running max m_run is in log2 units and p = 2^(s - m).
// ok[] marks valid tokens: masked tokens get p = 0 and, with MASKV, their V entries are zeroed,
// since slots past a candidate's length may hold NaN (a caller that knows every masked slot holds
// finite data passes MASKV = false). vsa / vsb scale P for fp8 V.
template <int D, bool MASKV = true>
__device__ __forceinline__ void online_step(const uint4 *KA, const uint4 *KB, const uint2 *VA,
                                            const uint2 *VB, const uint4 *q0, const uint4 *q1,
                                            const uint4 *q2, const bool *ok, float sca, float scb,
                                            float vsa, float vsb, float &m_run, float &l_run,
                                            floatx4 *acc) {
  constexpr int NKB = D / 32, NDB = D / 16;
  floatx4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kk = 0; kk < NKB; ++kk) {
    sa = mfma16(KA[kk], q0[kk], sa);
    sa = mfma16(KA[kk], q1[kk], sa);
    sa = mfma16(KA[kk], q2[kk], sa);
    sb = mfma16(KB[kk], q0[kk], sb);
    sb = mfma16(KB[kk], q1[kk], sb);
    sb = mfma16(KB[kk], q2[kk], sb);
  }
  float sv[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    sv[i] = ok[i] ? sa[i] * sca : -INFINITY;
    sv[4 + i] = ok[4 + i] ? sb[i] * scb : -INFINITY;
  }
  float mx = sv[0];
#pragma unroll
  for (int i = 1; i < 8; ++i) mx = fmaxf(mx, sv[i]);
  mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  const float m_new = fmaxf(m_run, mx);  // finite once any valid token has been seen
  const float alpha = (m_new == -INFINITY) ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
  m_run = m_new;
  float pv[8], psum = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    pv[i] = ok[i] ? __builtin_amdgcn_exp2f(sv[i] - m_new) : 0.f;
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
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    pv[i] *= vsa;
    pv[4 + i] *= vsb;
  }
  uint32_t ph[4], pl[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) split2(pv[2 * i], pv[2 * i + 1], ph[i], pl[i]);
  const uint4 Phi = make_uint4(ph[0], ph[1], ph[2], ph[3]);
  const uint4 Plo = make_uint4(pl[0], pl[1], pl[2], pl[3]);
  const uint32_t ma0 = (ok[0] ? 0xFFFFu : 0u) | (ok[1] ? 0xFFFF0000u : 0u);
  const uint32_t ma1 = (ok[2] ? 0xFFFFu : 0u) | (ok[3] ? 0xFFFF0000u : 0u);
  const uint32_t mb0 = (ok[4] ? 0xFFFFu : 0u) | (ok[5] ? 0xFFFF0000u : 0u);
  const uint32_t mb1 = (ok[6] ? 0xFFFFu : 0u) | (ok[7] ? 0xFFFF0000u : 0u);
#pragma unroll
  for (int nb = 0; nb < NDB; ++nb) {
    const uint4 vop = MASKV ? make_uint4(VA[nb].x & ma0, VA[nb].y & ma1, VB[nb].x & mb0, VB[nb].y & mb1)
                            : make_uint4(VA[nb].x, VA[nb].y, VB[nb].x, VB[nb].y);
    acc[nb] = mfma16(vop, Phi, acc[nb]);
    acc[nb] = mfma16(vop, Plo, acc[nb]);
  }
}

// Stores a wave's partial for column n (acc rows d = 16 nb + 4 cq + i; 64 bytes per head and
// 16-dim block across the 4 lanes of the column) and its m (given in log2 units), l.
template <int D>
__device__ __forceinline__ void store_partial(float *hb, int cq, const floatx4 *acc, float m_run,
                                              float l_run) {
  constexpr int NDB = D / 16;
#pragma unroll
  for (int nb = 0; nb < NDB; ++nb)
    *(float4 *)(hb + nb * 16 + 4 * cq) = make_float4(acc[nb][0], acc[nb][1], acc[nb][2], acc[nb][3]);
  if (cq == 0) *(float2 *)(hb + D) = make_float2(m_run * kLn2, l_run);  // m back to natural units
}

struct AttnArgs {
  const char *kp, *vp;     // this layer's pools
  const float *ksc, *vsc;  // this layer's fp8 scales (or null)
  int nkv, g, nq;
  const int32_t *page_table;
  int max_pages;
  const int32_t *lengths;
  GroupTable gt;
  int nch;
  const float *q, *kself, *vself;
  float *apart;   // [B][nq][nch][D + 2]: per chunk the acc row, then m, then l; a candidate's
                  // shared-prefix chunks come first, its private chunks after them
  float *o;       // [B][nq][D] fp32 output (may be null)
  uint16_t *op;   // operand buffer of the output projection (may be null)
  int NT, Bp;
  float *lse;     // [B][nq] log-sum-exp of each softmax, own keys included (may be null)
  int kq;         // verify tokens per candidate: row v = token v % kq of candidate v / kq; q,
                  // k_self, v_self, partials and o are per row, lengths and page table per
                  // candidate, group ranges in rows
};

// One block per (chunk of pages, candidate b) over the candidate's private pages,
// one wave per kv-head j, so the n_kv tiles of a page (contiguous in the pool) are read together.
// Each wave walks the chunk two pages (32 tokens) at a time: S = K Q^T on the matrix cores
// (A = the K tile, 16 tokens x 32 dims; B = the g query heads of j as columns, in three bf16
// terms), online softmax per head in registers (a lane holds 4 tokens of one head per page),
// then O^T += V^T P^T (A = V^T, 16 dims x 32 tokens; the V tile stores 4 consecutive slots of
// a dimension together, so one 16-byte load per lane feeds 2 (bf16) or 4 (fp8) A operands; B =
// P^T hi and lo). The wave writes its unnormalised partial (acc, m, l) per q-head.
// Slots at or beyond L_b are masked in S and zeroed in V (they may hold anything, NaN included).
template <int KVT, int D>
__global__ __launch_bounds__(64 * kMaxKvHeadsMx) void k_attn_mx(AttnArgs a) {
  constexpr int NKB = D / 32;  // 32-dim blocks of q.k
  constexpr int NDB = D / 16;  // 16-dim blocks of the output
  constexpr int EB = KVT == 1 ? 2 : 1;
  constexpr size_t TILE = (size_t)kPage * D * EB;
  const int c = blockIdx.x, b = blockIdx.y;  // chunk, candidate
  const int j = threadIdx.x >> 6;
  const int nkv = a.nkv, g = a.g, nq = a.nq, kq = a.kq;
  const int L = a.lengths[b];
  const int npages = (L + kPage - 1) / kPage;
  int first = 0;
  for (int gi = 0; gi < a.gt.n; ++gi)
    if (b * kq >= a.gt.start[gi] && b * kq < a.gt.start[gi + 1]) first = a.gt.prefix_pages[gi];
  const int CP = 1 << a.gt.cshift_private;
  const int ncp = (first + (1 << a.gt.cshift_prefix) - 1) >> a.gt.cshift_prefix;  // prefix chunks
  const int p0 = first + c * CP;
  if (p0 >= npages) return;
  const int np = min(npages, p0 + CP) - p0;
  const int lane = threadIdx.x & 63;
  const int n = lane & 15, cq = lane >> 4;
  // each wave reads the chunk's page ids itself into lane registers (lane i holds page i and,
  // for fp8, its scales) and fetches them with scalar lane reads: no LDS, no barrier
  const int ph_l = lane < np ? a.page_table[(size_t)b * a.max_pages + p0 + lane] : 0;
  float ksc_l = 0.f, vsc_l = 0.f;
  if (KVT == 2 && lane < np) {
    ksc_l = a.ksc[(size_t)ph_l * nkv + j];
    vsc_l = a.vsc[(size_t)ph_l * nkv + j];
  }
  const int npairs = (np + 1) >> 1;
  auto load_pair = [&](int pp, PairRaw<D> &r) {
    // indices past the chunk are clamped to its last page: those tokens are masked anyway
    const int pa = lane_value(ph_l, min(2 * pp, np - 1));
    const int pb = lane_value(ph_l, min(2 * pp + 1, np - 1));
    load_pair_raw<KVT, D, true>((const uint4 *)(a.kp + ((size_t)pa * nkv + j) * TILE),
                          (const uint4 *)(a.kp + ((size_t)pb * nkv + j) * TILE),
                          (const uint4 *)(a.vp + ((size_t)pa * nkv + j) * TILE),
                          (const uint4 *)(a.vp + ((size_t)pb * nkv + j) * TILE), lane, r);
  };
  PairRaw<D> r0, r1;
  load_pair(0, r0);  // in flight while the queries are prepared

  // column n: verify token n / g of this candidate, q-head j g + n % g (kq g <= 16 columns)
  const bool colv = n < kq * g;
  const int ti = colv ? n / g : 0, hh = colv ? n - (n / g) * g : 0;
  const size_t row = (size_t)b * kq + ti;
  uint4 q0[NKB], q1[NKB], q2[NKB];
  load_query_ops<KVT, D>(a.q + (row * nq + (size_t)j * g + hh) * D, colv, cq, q0, q1, q2);
  const float rs = kLog2e / sqrtf((float)D);  // scores in log2 units
  float m_run = -INFINITY, l_run = 0.f;
  floatx4 acc[NDB];
#pragma unroll
  for (int nb = 0; nb < NDB; ++nb) acc[nb] = floatx4{0.f, 0.f, 0.f, 0.f};

  auto compute_pair = [&](int pp, const PairRaw<D> &r, auto maskv) {
    const int la = min(2 * pp, np - 1), lb = 2 * pp + 1;
    const bool hasA = 2 * pp < np, hasB = lb < np;
    uint4 KA[NKB], KB[NKB];
    uint2 VA[NDB], VB[NDB];
    unpack_pair<KVT, D>(r, KA, KB, VA, VB);
    const int ta = (p0 + la) * kPage + 4 * cq, tb = (p0 + lb) * kPage + 4 * cq;
    bool ok[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ok[i] = hasA && (ta + i < L);
      ok[4 + i] = hasB && (tb + i < L);
    }
    const int lbc = hasB ? lb : la;
    const float sca = (KVT == 2) ? lane_value(ksc_l, la) * rs : rs;
    const float scb = (KVT == 2) ? lane_value(ksc_l, lbc) * rs : rs;
    const float vsa = (KVT == 2) ? lane_value(vsc_l, la) : 1.f;
    const float vsb = (KVT == 2) ? lane_value(vsc_l, lbc) : 1.f;
    online_step<D, decltype(maskv)::value>(KA, KB, VA, VB, q0, q1, q2, ok, sca, scb, vsa, vsb,
                                           m_run, l_run, acc);
  };
  // a branch-free loop over an even number of pairs: the pair past the end (if any) is fully
  // masked, and loads past the end repeat the last page (an L2 hit), so that wait counts never
  // cover the loads in flight for the next pair
  // (scheduling barriers keep each pair's loads ahead of the previous pair's arithmetic, so that
  // the waits inside a compute step cover only its own, older loads)
  // Only the chunk holding the candidate's last page can hold slots past L_b (which may be
  // NaN); every page of the other chunks is full, and their pairs past the end repeat a full
  // page (finite, with p = 0), so their V operands need no masking. fp8 pages, whose step is
  // bound by vector instructions rather than HBM, get a loop copy without it (for bf16 the
  // second copy would cost more registers than the masking costs time).
  auto chunk_loop = [&](auto maskv) {
    for (int pp = 0; pp < npairs; pp += 2) {
      load_pair(pp + 1, r1);
      __builtin_amdgcn_sched_barrier(0);
      compute_pair(pp, r0, maskv);
      __builtin_amdgcn_sched_barrier(0);
      load_pair(pp + 2, r0);
      __builtin_amdgcn_sched_barrier(0);
      compute_pair(pp + 1, r1, maskv);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  if (KVT == 2 && p0 + np < npages)
    chunk_loop(std::integral_constant<bool, false>{});
  else
    chunk_loop(std::integral_constant<bool, true>{});
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  if (colv)
    store_partial<D>(a.apart + ((row * nq + (size_t)j * g + hh) * a.nch + ncp + c) * (D + 2), cq,
                     acc, m_run, l_run);
}

// Shared-prefix attention: the members of a prefix group share the physical pages of their
// first prefix_pages pages, which are read once for all of them. One block per (prefix chunk c,
// kv-head j, column block) with up to 16 waves; the columns are (member, q-head of j) pairs,
// 16 per wave (e.g. 2 members x 7 heads). The pair's K and V tiles (one head) are staged in LDS
// once per block, double buffered, and every wave runs the online step on them with its own
// columns. Partials go to the members' chunk slots [0, ncp).
template <int KVT, int D>
__global__ __launch_bounds__(64 * kPrefixWaves) void k_prefix_mx(AttnArgs a) {
  constexpr int NKB = D / 32, NDB = D / 16;
  constexpr int EB = KVT == 1 ? 2 : 1;
  constexpr int TILE16 = kPage * D * EB / 16;  // uint4 entries per tile
  __shared__ uint4 stage_s[2][4][TILE16];      // [buffer][K A, K B, V A, V B]
  const int c = blockIdx.x, j = blockIdx.y;
  // group and column block of this block
  int grp = 0;
  while (grp < a.gt.n - 1 && (int)blockIdx.z >= a.gt.colblock_start[grp + 1]) ++grp;
  const int cb = blockIdx.z - a.gt.colblock_start[grp];
  const int m0 = a.gt.start[grp], members = a.gt.start[grp + 1] - m0;
  const int ppages = a.gt.prefix_pages[grp];
  const int CP = 1 << a.gt.cshift_prefix;
  const int p0 = c * CP;
  if (p0 >= ppages) return;
  const int np = min(ppages, p0 + CP) - p0;
  const int npairs = (np + 1) >> 1;
  const int nkv = a.nkv, g = a.g, nq = a.nq;
  constexpr int nthr = 64 * kPrefixWaves;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 15, cq = lane >> 4;
  const int col = (cb * kPrefixWaves + wave) * 16 + n;  // (member, head) column
  const int mem = col / g, hh = col - mem * g;
  const bool present = mem < members;
  const int bcand = m0 + (present ? mem : 0);
  // page ids and fp8 scales of the chunk (from the first member's table row), in lanes
  const int ph_l = lane < np ? a.page_table[(size_t)(m0 / a.kq) * a.max_pages + p0 + lane] : 0;
  float ksc_l = 1.f, vsc_l = 1.f;
  if (KVT == 2 && lane < np) {
    ksc_l = a.ksc[(size_t)ph_l * nkv + j];
    vsc_l = a.vsc[(size_t)ph_l * nkv + j];
  }
  // cooperative staging: thread t copies entries t, t + nthr, ... of the pair's 4 tiles. NPF
  // pairs are in flight in registers (a ring, unrolled so that its indices are constants);
  // the pair being computed sits in one of two LDS buffers. Fetches past the last pair repeat
  // it (an L2 hit), so that no load is conditional.
  constexpr int PER = (4 * TILE16 + nthr - 1) / nthr;
  constexpr int NPF = KVT == 2 ? 2 : 4;  // pairs in flight (fp8 unpacking needs the registers)
  struct Stage {
    uint4 v[PER];
  };
  auto fetch = [&](int pp) __attribute__((always_inline)) {
    Stage st;
    pp = min(pp, npairs - 1);
    const int pa = lane_value(ph_l, min(2 * pp, np - 1));
    const int pb = lane_value(ph_l, min(2 * pp + 1, np - 1));
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = min((int)threadIdx.x + u * nthr, 4 * TILE16 - 1);
      const int t = e / TILE16, o = e - t * TILE16;
      const char *pool = t < 2 ? a.kp : a.vp;
      const int pg = (t & 1) ? pb : pa;
      st.v[u] = ((const uint4 *)(pool + ((size_t)pg * nkv + j) * TILE16 * 16))[o];
    }
    return st;
  };
  auto stash = [&](int buf, const Stage &src) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = threadIdx.x + u * nthr;
      if (e < 4 * TILE16) (&stage_s[buf][0][0])[e] = src.v[u];
    }
  };
  // the ring of NPF register buffers is four named values, so that every index is a constant
  Stage s0 = fetch(0), s1 = fetch(1), s2, s3;
  if (NPF == 4) {
    s2 = fetch(2);
    s3 = fetch(3);
  }
  uint4 qhi[NKB], qmd[NKB], qlo[NKB];
  load_query_ops<KVT, D>(a.q + ((size_t)bcand * nq + (size_t)j * g + hh) * D, present, cq, qhi,
                         qmd, qlo);
  stash(0, s0);
  __syncthreads();
  const float rs = kLog2e / sqrtf((float)D);  // scores in log2 units
  float m_run = -INFINITY, l_run = 0.f;
  floatx4 acc[NDB];
#pragma unroll
  for (int nb = 0; nb < NDB; ++nb) acc[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
  // step pp: refill the buffer pair pp left (with pair pp + NPF), compute pair pp from LDS, and
  // stash pair pp + 1 (fetched NPF - 1 steps earlier) into the other LDS buffer
  auto step = [&](int pp, Stage &mine, const Stage &next) __attribute__((always_inline)) {
    mine = fetch(pp + NPF);
    const int buf = pp & 1;
    PairRaw<D> r;
    load_pair_raw<KVT, D, false>(stage_s[buf][0], stage_s[buf][1], stage_s[buf][2], stage_s[buf][3],
                                 lane, r);
    uint4 KA[NKB], KB[NKB];
    uint2 VA[NDB], VB[NDB];
    unpack_pair<KVT, D>(r, KA, KB, VA, VB);
    const int la = 2 * pp, lb = 2 * pp + 1;
    const bool hasB = lb < np;
    bool ok[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ok[i] = true;  // prefix pages are full
      ok[4 + i] = hasB;
    }
    const int lbc = hasB ? lb : la;
    const float sca = (KVT == 2) ? lane_value(ksc_l, la) * rs : rs;
    const float scb = (KVT == 2) ? lane_value(ksc_l, lbc) * rs : rs;
    const float vsa = (KVT == 2) ? lane_value(vsc_l, la) : 1.f;
    const float vsb = (KVT == 2) ? lane_value(vsc_l, lbc) : 1.f;
    online_step<D>(KA, KB, VA, VB, qhi, qmd, qlo, ok, sca, scb, vsa, vsb, m_run, l_run, acc);
    if (pp + 1 < npairs) stash(buf ^ 1, next);
    __syncthreads();
  };
  for (int pb = 0; pb < npairs; pb += NPF) {
    if (NPF == 2) {
      step(pb, s0, s1);
      if (pb + 1 >= npairs) break;
      step(pb + 1, s1, s0);
    } else {
      step(pb, s0, s1);
      if (pb + 1 >= npairs) break;
      step(pb + 1, s1, s2);
      if (pb + 2 >= npairs) break;
      step(pb + 2, s2, s3);
      if (pb + 3 >= npairs) break;
      step(pb + 3, s3, s0);
    }
  }
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  if (present)
    store_partial<D>(a.apart + (((size_t)bcand * nq + (size_t)j * g + hh) * a.nch + c) * (D + 2),
                     cq, acc, m_run, l_run);
}

// Log-sum-exp merge of the chunk partials of one (candidate b, q-head h) with the token's own
// key/value: m = max(s_self, m_c),
//   o = (e^{s_self - m} v_self + sum_c e^{m_c - m} acc_c) / (e^{s_self - m} + sum_c e^{m_c - m} l_c).
// One block of NTHR threads per (b, h): thread (s, d) owns output dimension d for the chunks
// c = s, s + S, ... (S = NTHR / D subsets). Every load is issued at entry (the first 16 chunk
// rows of each subset go to registers), so the merge costs about one memory round trip; the
// subsets are added in a fixed order. Writes o (fp32) and/or the output projection's operand.
template <int D, int NTHR>
__global__ __launch_bounds__(NTHR) void k_merge_mx(AttnArgs a) {
  constexpr int S = NTHR / D;   // chunk subsets
  constexpr int NW = NTHR / 64;  // waves
  constexpr int R = 16;
  __shared__ float m_s[kMaxChunks], f_s[kMaxChunks];
  __shared__ float red[3][NW];
  __shared__ float sub_s[S][D];
  __shared__ float sself_s[16];
  const int b = blockIdx.x, h = blockIdx.y, t = threadIdx.x;  // row (candidate, verify token)
  const int lane = t & 63, wave = t >> 6;
  const int sub = t / D, dd = t - sub * D;
  const int j = h / a.g;
  const int kq = a.kq, cand = b / kq, tok = b - cand * kq;
  const int L = a.lengths[cand];
  const int npages = (L + kPage - 1) / kPage;
  int first = 0;
  for (int gi = 0; gi < a.gt.n; ++gi)
    if (b >= a.gt.start[gi] && b < a.gt.start[gi + 1]) first = a.gt.prefix_pages[gi];
  // shared-prefix chunks, then private chunks
  const int sp = a.gt.cshift_prefix, sv = a.gt.cshift_private;
  const int nc = ((first + (1 << sp) - 1) >> sp) + ((npages - first + (1 << sv) - 1) >> sv);
  const float *base = a.apart + ((size_t)b * a.nq + h) * a.nch * (D + 2);
  float rv[R];
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const int c = sub + S * i;
    rv[i] = c < nc ? base[(size_t)c * (D + 2) + dd] : 0.f;
  }
  float mx = -INFINITY;
  for (int c = t; c < nc; c += NTHR) {
    const float m = base[(size_t)c * (D + 2) + D];
    m_s[c] = m;
    f_s[c] = base[(size_t)c * (D + 2) + D + 1];  // l_c for now
    mx = fmaxf(mx, m);
  }
  // the verify tokens' own keys: this row's token attends to tokens 0..tok of its candidate
  // (rows cand kq + i); s_i = q . k_self_i / sqrt(D), one wave per key
  const size_t row0 = (size_t)cand * kq;
  const float *qr = a.q + ((size_t)b * a.nq + h) * D;
  for (int i = wave; i <= tok; i += NW) {
    const float *kr = a.kself + ((row0 + i) * a.nkv + j) * D;
    float dot = 0.f;
#pragma unroll
    for (int u = 0; u < D / 64; ++u) dot += qr[lane + 64 * u] * kr[lane + 64 * u];
    dot = wsum(dot);
    if (lane == 0) sself_s[i] = dot * (1.0f / sqrtf((float)D));
  }
  mx = wmax(mx);
  if (lane == 0) red[1][wave] = mx;
  __syncthreads();
  float M = -INFINITY;
  for (int i = 0; i <= tok; ++i) M = fmaxf(M, sself_s[i]);
#pragma unroll
  for (int w = 0; w < NW; ++w) M = fmaxf(M, red[1][w]);
  float ls = 0.f;
  for (int c = t; c < nc; c += NTHR) {
    const float f = expf(m_s[c] - M);
    ls += f * f_s[c];
    f_s[c] = f;
  }
  ls = wsum(ls);
  if (lane == 0) red[2][wave] = ls;
  __syncthreads();
  float lsum = 0.f;
#pragma unroll
  for (int w = 0; w < NW; ++w) lsum += red[2][w];
  float acc = 0.f;
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const int c = sub + S * i;
    if (c < nc) acc += f_s[c] * rv[i];
  }
  for (int c = sub + S * R; c < nc; c += S) acc += f_s[c] * base[(size_t)c * (D + 2) + dd];
  sub_s[sub][dd] = acc;
  __syncthreads();
  if (sub != 0) return;
  float tot = 0.f;
#pragma unroll
  for (int k = 0; k < S; ++k) tot += sub_s[k][dd];
  float es_sum = 0.f;
  for (int i = 0; i <= tok; ++i) {
    const float es = expf(sself_s[i] - M);
    es_sum += es;
    tot += es * a.vself[((row0 + i) * a.nkv + j) * D + dd];
  }
  const float ov = tot / (lsum + es_sum);
  if (a.lse && dd == 0) a.lse[(size_t)b * a.nq + h] = M + logf(lsum + es_sum);
  if (a.o) a.o[((size_t)b * a.nq + h) * D + dd] = ov;
  if (a.op) store_operand(a.op, a.NT, a.Bp, h * D + dd, b, ov);
}

hipError_t launch_attn_mx(const Dims &dm, const Plan &p, const Workspace &w, const char *kp,
                          const char *vp, const float *ksc, const float *vsc,
                          const int32_t *page_table, const int32_t *lengths, const GroupTable &gt,
                          const float *q, const float *kself, const float *vself, float *o,
                          uint16_t *op, hipStream_t s, bool merge, float *lse) {
  AttnArgs a;
  memset(&a, 0, sizeof a);
  a.lse = lse;
  a.kp = kp;
  a.vp = vp;
  a.ksc = ksc;
  a.vsc = vsc;
  a.nkv = dm.nkv;
  a.g = dm.g;
  a.nq = dm.nq;
  a.page_table = page_table;
  a.max_pages = p.max_pages;
  a.lengths = lengths;
  a.gt = gt;
  a.nch = p.nch;
  a.q = q;
  a.kself = kself;
  a.vself = vself;
  a.apart = w.apart;
  a.o = o;
  a.op = op;
  a.NT = p.nt;
  a.Bp = p.bp;
  a.kq = p.kq;
  if (gt.n > 0) {
    dim3 pgrid(gt.prefix_chunks, dm.nkv, gt.colblock_start[gt.n]);
#define KVPRM_P(KVT, D) \
  hipLaunchKernelGGL((k_prefix_mx<KVT, D>), pgrid, dim3(64 * kPrefixWaves), 0, s, a)
    if (dm.kvdt == 1) {
      if (dm.d == 64) KVPRM_P(1, 64);
      else KVPRM_P(1, 128);
    } else {
      if (dm.d == 64) KVPRM_P(2, 64);
      else KVPRM_P(2, 128);
    }
#undef KVPRM_P
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  dim3 grid(gt.private_chunks > 0 ? gt.private_chunks : p.nch - 1, p.Breal);
#define KVPRM_A(KVT, D) hipLaunchKernelGGL((k_attn_mx<KVT, D>), grid, dim3(64 * dm.nkv), 0, s, a)
  if (dm.kvdt == 1) {
    if (dm.d == 64) KVPRM_A(1, 64);
    else KVPRM_A(1, 128);
  } else {
    if (dm.d == 64) KVPRM_A(2, 64);
    else KVPRM_A(2, 128);
  }
#undef KVPRM_A
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !merge) return e;
  // 256 threads per (row, q-head) when each of their 256 / D chunk subsets has at most 8 of the
  // row's chunks (16 at d_h = 128: per merge 5.2 -> 5.1 us for the 7B batch of 16, 6.4 -> 5.9 us
  // for the large fp8 batch; rows of 32 chunks, as in the ragged 32k batch, take 5.3 us against
  // 5.0-5.1 with 512) or when there are more rows than four 512-thread blocks per compute unit
  // hold (the 64-candidate beam: 1792 rows), so that they all run in one round; 512 otherwise
  // (a row's chunks: its group prefix's and its private pages'; without host lengths, the
  // plan's chunk slots)
  const int row_chunks = gt.private_chunks > 0 ? gt.prefix_chunks + gt.private_chunks : p.nch;
  const bool small = p.B * dm.nq > 1024 || row_chunks <= (256 / dm.d) * 8;
  const dim3 mgrid(p.B, dm.nq);
  if (dm.d == 64) {
    if (small) hipLaunchKernelGGL((k_merge_mx<64, 256>), mgrid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_merge_mx<64, 512>), mgrid, dim3(512), 0, s, a);
  } else {
    if (small) hipLaunchKernelGGL((k_merge_mx<128, 256>), mgrid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_merge_mx<128, 512>), mgrid, dim3(512), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace kvprm
