// Internal declarations shared by the C-ABI layer and the HIP kernels of libkvprm.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvprm {

// Shape of the model as the kernels see it.
struct Dims {
  int layers, H, nq, nkv, d, F, g;
  float theta, eps;
  int wdt;   // 0 fp32, 1 bf16
  int kvdt;  // 0 fp32, 1 bf16, 2 fp8 e4m3
};

// Prefix-sharing groups, passed by value to the attention kernels (no host->device copy).
constexpr int kMaxGroups = 64;
struct GroupTable {
  int n;                         // 0 = no sharing
  int start[kMaxGroups + 1];     // candidate ranges
  int prefix_pages[kMaxGroups];  // shared pages of each group
};

// Attention split: each work item covers kChunkPages pages of one (candidate, kv-head).
constexpr int kChunkPages = 32;
constexpr int kPage = 16;

// Workspace carve-up (all offsets 256-byte aligned).
struct Workspace {
  float *x;        // [B][H] residual stream
  float *ss;       // [nss][B] partial sums of squares of x
  float *part;     // GEMV split-K partials [ksplit][rows][B]
  float *q;        // [B][nq][d]
  float *kself;    // [B][nkv][d]
  float *vself;    // [B][nkv][d]
  float *apart;    // attention partials [B][nq][nch][d + 2] (acc..., m, l)
  float *o;        // [B][nq * d]
  float *hffn;     // [B][F]
  uint4 *act;      // activation operand of the MFMA GEMV (bf16 hi/lo, B-operand order)
  size_t bytes;
};

struct Plan {
  int B, max_pages, nch;      // nch = chunks per (candidate, kv-head) at max_pages
  int nss;                    // blocks of 256 rows in H
  int ks_qkv, ks_o, ks_gu, ks_d;  // split-K counts
  int kslice_qkv, kslice_o, kslice_gu, kslice_d;
  size_t part_elems;
  size_t act_bytes;
};

// MFMA GEMV helpers (kvprm_mfma.hip)
int gemv_nt(int B);
int gemv_bp(int B);
void gemv_split(int rows, int K, int B, int &kslice, int &ksplit);

Plan make_plan(const Dims &dm, int B, int max_pages);
Workspace carve(const Dims &dm, const Plan &p, void *base);

// Kernel launchers (return hipGetLastError()).
hipError_t launch_init(const Dims &dm, const Plan &p, const Workspace &w, const void *verify_embed,
                       hipStream_t s);
// Y partials = W_seg . u, u = in (optionally RMS-normalised with gamma using ss). Up to three
// row segments with their own weight pointers (e.g. q, k, v).
struct GemvSegs {
  const void *w[3];
  int rows[3];
  int nseg;
};
hipError_t launch_gemv(const Dims &dm, const Plan &p, const GemvSegs &segs, int K, int kslice,
                       int ksplit, const float *in, const void *gamma, const float *ss,
                       float *part, uint4 *actbuf, hipStream_t s);
hipError_t launch_gemv_mfma(const Dims &dm, const Plan &p, const GemvSegs &segs, int K,
                            int kslice, int ksplit, const float *in, const void *gamma,
                            const float *ss, float *part, uint4 *actbuf, hipStream_t s);
hipError_t launch_attn_mfma(const Dims &dm, const Plan &p, const char *kp, const char *vp,
                            const float *ksc, const float *vsc, const int32_t *page_table,
                            const int32_t *lengths, const GroupTable &gt, const float *q,
                            float *apart, hipStream_t s);
hipError_t launch_qkv_finish(const Dims &dm, const Plan &p, const Workspace &w,
                             const int32_t *lengths, hipStream_t s);
hipError_t launch_attention(const Dims &dm, const Plan &p, const Workspace &w, int layer,
                            const void *kpool, const void *vpool, const float *kscale,
                            const float *vscale, int num_pages, const int32_t *page_table,
                            const int32_t *lengths, const GroupTable &gt, const float *q,
                            const float *kself, const float *vself, float *o, hipStream_t s);
hipError_t launch_residual(const Dims &dm, const Plan &p, const Workspace &w, int ksplit,
                           hipStream_t s);
hipError_t launch_swiglu(const Dims &dm, const Plan &p, const Workspace &w, int ksplit,
                         hipStream_t s);
hipError_t launch_head(const Dims &dm, const Plan &p, const Workspace &w, const void *final_norm,
                       const void *reward_w, float reward_b, float *scores, float *logits,
                       hipStream_t s);

}  // namespace kvprm
