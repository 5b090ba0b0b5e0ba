// Internal declarations shared by the C-ABI layer and the HIP kernels of libkvprm.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/kvprm.h"

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
constexpr int kPrefixWaves = 7;  // waves per shared-prefix block (16 columns each; 7 x 16 = 112
                                 // columns = 16 members x 7 heads at the 7B shape, so the 448
                                 // columns of a 64-candidate beam fill 4 blocks exactly)
struct GroupTable {
  int n;                               // 0 = no sharing
  int start[kMaxGroups + 1];           // candidate ranges
  int prefix_pages[kMaxGroups];        // shared pages of each group
  int colblock_start[kMaxGroups + 1];  // shared-prefix column blocks of the groups, cumulative
  int prefix_chunks;                   // chunks of the longest group prefix
  int private_chunks;                  // chunk grid of the private pages (0 = from max_pages)
  int cshift_prefix, cshift_private;   // chunk lengths (1 << shift pages) of the two kernels
};

// Attention split: each work item covers one chunk of pages of one candidate (and kv-head).
// The matrix-core kernels take the chunk length from the plan (16, 32 or 64 pages); the
// vector-ALU kernels use kChunkPagesValu.
constexpr int kChunkPagesValu = 32;
constexpr int kMaxChunks = 1024;  // chunk partials one merge handles
constexpr int kMaxKvHeadsMx = 8;  // matrix-core attention: one wave per kv-head in a block
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
  float *hffn;     // [B][F] (vector-ALU path)
  uint16_t *topd;  // adapter operand slots [3][rank / 32][NT][64][8] bf16 (scale * A u)
  // matrix-core path
  float *rope;       // [B][d/2][2] cos, sin of the verify position
  uint16_t *opA;     // GEMV operands (bf16 hi/lo): QKV and gate/up input (K = H)
  uint16_t *opO;     //   output projection input (K = n_q d)
  uint16_t *opD;     //   down projection input (K = F)
  size_t bytes;
};

struct GemvPlan {
  int rows, K, kslice, ksplit;
};

// Adapter of one projection group (q/k/v, o, gate/up or down) of one layer.
struct LoraTail {
  const void *b[3];  // B factor of each segment (packed [rows_i][rank]); null = no adapter
  int tkb;           // rank / 32; 0 = no tail
};

struct Plan {
  // B = rows of the pass: candidates x verify tokens per candidate (kq, the depth-k readout);
  // row v is verify token v % kq of candidate v / kq. Breal = candidates.
  int B, max_pages, nch;      // nch = chunk slots per (row, q-head), see make_plan
  int kq, Breal;
  int cshift;                 // matrix-core attention chunk from (B, max_pages): 1 << cshift pages
  int nss;                    // row blocks of H that carry partial sums of squares
  int rb;                     // rows per such block
  // vector-ALU path
  int ks_qkv, ks_o, ks_gu, ks_d;  // split-K counts
  int kslice_qkv, kslice_o, kslice_gu, kslice_d;
  // matrix-core path
  int nt, bp;                 // operand column tiles and padded batch
  // low-rank adapter (0 = none): the split-K plans of the A-factor products of the q/k/v,
  // output, gate/up and down groups
  int lora_rank;
  GemvPlan g_la[4];
  // q/k/v as a split-K product and a finish kernel (RMSNorm scale, rotary) instead of the fused
  // kernel, for shapes with more rotary tile pairs than compute units (no adapter)
  int qkv_split;
  GemvPlan g_qkv;
  // projections as split-K products whose blocks share each operand batch in LDS
  // (k_resid_split: rs_wpb row tiles per block, kslice / 32 input blocks per slice, an adapter's
  // B-factor tail as one more slice) and a finish kernel, by batch size; 0 = the fused kernels
  int rs_wpb;
  int rs_u;        // input blocks per operand batch of k_resid_split (4, or 8 / 16 at one column tile)
  int rs_o, rs_d;  // output / down projection split
  GemvPlan g_rs_o, g_rs_d;
  int rs_qkv;  // the q/k/v product the same way, with a rotary finish (k_qkv_split_fin)
  GemvPlan g_rs_qkv;
  size_t part_elems;
};

enum { LORA_QKV = 0, LORA_O = 1, LORA_GU = 2, LORA_DOWN = 3 };

// Backward pass for KV steering (kvprm_grad.hip): activations the forward pass saves per layer
// (B rows each) and the backward scratch. Vectors that enter a transposed product are
// [row][kDPad]; the others [B][width].
constexpr int kGradMaxSplits = 64;  // row splits of a transposed product
constexpr int kDPad = 8;            // columns of a transposed product's d rows (batch <= 8)
constexpr int kGradMaxHidden = 16384;  // hidden size the RMSNorm backward holds in registers
constexpr int kTgemvWindow = 144;      // row tiles of one split of a transposed product (its d
                                        // rows, 72 KiB, are staged in LDS)
struct GradSave {
  float *x_in, *x_mid;           // [N_L][B][H] residual stream entering the layer / after attention
  float *q, *ks, *vs, *o;        // [N_L][B][n_q | n_kv][d] (q, k_self after rotary)
  float *lse;                    // [N_L][B][n_q] log-sum-exp of each head's softmax (own key incl.)
  float *gu;                     // [N_L][B][2F] gate / up pre-activations
  float *dx, *dxT, *dxm, *dxmT;  // [B][H] and [H][kDPad]: residual gradient after / inside
  float *du;                     // [B][H]
  float *dgu;                    // [2F][kDPad]
  float *dout;                   // [B][n_q d]
  float *Dh;                     // [B][n_q]
  float *dq_self;                // [B][n_q][d]
  float *dk_self, *dv_self;      // [B][n_kv][d]
  float *dqkv;                   // [(n_q + 2 n_kv) d][kDPad]
  float *dq_part;                // [B][n_q][nch][d]
  float *part;                   // transposed-product split partials
  size_t bytes;
};
int grad_tgemv_splits(int K, int tiles);
GradSave carve_grad(const Dims &dm, const Plan &p, void *base);
hipError_t launch_backward(const Dims &dm, const Plan &p, const Workspace &w, const GradSave &sv,
                           const kvprm_layer_weights *layers, const void *final_norm,
                           const void *reward_w, float reward_b, char *kpool, char *vpool,
                           size_t layer_bytes, const int32_t *page_table, const int32_t *lengths,
                           int CP, int chunks, float *grad_k, float *grad_v, float eta,
                           hipStream_t s);

// matrix-core helpers (kvprm_mfma.hip; the attention launcher is in kvprm_attn.hip)
int gemv_nt(int B);
int gemv_bp(int B);
int gemv_mt(int nt, int rows);
hipError_t launch_pack_weight(const void *src, void *dst, int64_t rows, int64_t K, hipStream_t s);
hipError_t launch_stream_read(const void *buf, size_t bytes, uint32_t *sink, hipStream_t s);
// token-major cache tiles -> the stored K (v = false) or V tile layout; eb = element bytes
hipError_t launch_pack_kv(const void *src, void *dst, int64_t ntiles, int d, int eb, bool v,
                          hipStream_t s);

Plan make_plan(const Dims &dm, int B, int max_pages, int lora_rank = 0, int depth = 1);
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
                       float *part, hipStream_t s);
// matrix-core pipeline (bf16 weights)
// xsave (optional): a copy of the residual stream x as initialised
hipError_t launch_init_mx(const Dims &dm, const Plan &p, const Workspace &w, const void *ev,
                          const void *gamma0, const int32_t *lengths, hipStream_t s,
                          float *xsave = nullptr);
hipError_t launch_qkv_mx(const Dims &dm, const Plan &p, const Workspace &w, const void *wq,
                         const void *wk, const void *wv, const LoraTail &tail, hipStream_t s);
// scale * A u of one projection group's adapters into the operand slots w.topd (slot i =
// segment i; a[i] null = segment without adapter): a split-K GEMV and a finish kernel
hipError_t launch_lora_a(const Dims &dm, const Plan &p, const Workspace &w, int group,
                         const void *const a[3], float scale, const uint16_t *act, hipStream_t s);
// fused projections: no split-K partials, the element-wise step after the output, gate/up and
// down projections runs in the epilogue
// xsave (optional, output and down projections): a copy of the updated residual stream
hipError_t launch_oproj_fused(const Dims &dm, const Plan &p, const Workspace &w, const void *wo,
                              const void *gamma_ffn, const LoraTail &tail, hipStream_t s,
                              float *xsave = nullptr);
hipError_t launch_gateup_fused(const Dims &dm, const Plan &p, const Workspace &w, const void *wg,
                               const void *wu, const LoraTail &tail, hipStream_t s,
                               float *save_gu = nullptr);
hipError_t launch_down_fused(const Dims &dm, const Plan &p, const Workspace &w, const void *wd,
                             const void *gamma_next, const LoraTail &tail, hipStream_t s,
                             float *xsave = nullptr);
hipError_t launch_attn_mx(const Dims &dm, const Plan &p, const Workspace &w, const char *kp,
                          const char *vp, const float *ksc, const float *vsc,
                          const int32_t *page_table, const int32_t *lengths, const GroupTable &gt,
                          const float *q, const float *kself, const float *vself, float *o,
                          uint16_t *op, hipStream_t s, bool merge = true, float *lse = nullptr);
hipError_t launch_qkv_finish(const Dims &dm, const Plan &p, const Workspace &w,
                             const int32_t *lengths, hipStream_t s);
hipError_t launch_attention(const Dims &dm, const Plan &p, const Workspace &w, int layer,
                            const void *kpool, const void *vpool, const float *kscale,
                            const float *vscale, int num_pages, const int32_t *page_table,
                            const int32_t *lengths, const GroupTable &gt, const float *q,
                            const float *kself, const float *vself, float *o, hipStream_t s,
                            bool merge = true);
hipError_t launch_residual(const Dims &dm, const Plan &p, const Workspace &w, int ksplit,
                           hipStream_t s);
hipError_t launch_swiglu(const Dims &dm, const Plan &p, const Workspace &w, int ksplit,
                         hipStream_t s);
hipError_t launch_head(const Dims &dm, const Plan &p, const Workspace &w, const void *final_norm,
                       const void *reward_w, float reward_b, float *scores, float *logits,
                       hipStream_t s);

}  // namespace kvprm
