// C ABI of libkvprm: argument validation, workspace carving and launch sequencing of the
// verify-token pass. Nothing here allocates device memory; only the debug check of the page
// table (KVPRM_DEBUG=1 at kvprm_create) synchronises the host.
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/kvprm.h"
#include "kvprm_internal.h"

using namespace kvprm;

struct kvprm_handle_s {
  kvprm_model_desc desc;
  Dims dm;
  bool debug;  // KVPRM_DEBUG=1 at creation: check device page ids on the host before each call
};

static thread_local std::string g_err;

static kvprm_status fail(kvprm_status st, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
static kvprm_status fail(kvprm_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

static kvprm_status ok() {
  g_err.clear();
  return KVPRM_OK;
}

#define HIP_TRY(expr, what)                                                                  \
  do {                                                                                       \
    hipError_t e_ = (expr);                                                                  \
    if (e_ != hipSuccess) return fail(KVPRM_E_HIP, "%s: %s", what, hipGetErrorString(e_)); \
  } while (0)

extern "C" {

const char *kvprm_last_error(void) { return g_err.c_str(); }

kvprm_status kvprm_create(const kvprm_model_desc *d, kvprm_handle *out) {
  if (!d || !out) return fail(KVPRM_E_INVALID, "kvprm_create: null argument");
  if (d->num_layers < 1 || d->hidden < 1 || d->num_q_heads < 1 || d->num_kv_heads < 1 ||
      d->head_dim < 1 || d->ffn_dim < 1)
    return fail(KVPRM_E_INVALID, "kvprm_create: sizes must be positive");
  if (d->num_q_heads % d->num_kv_heads != 0)
    return fail(KVPRM_E_INVALID, "kvprm_create: num_q_heads %% num_kv_heads != 0");
  if (!(d->rms_eps >= 0.f) || !(d->rope_theta > 0.f))
    return fail(KVPRM_E_INVALID, "kvprm_create: rms_eps must be >= 0 and rope_theta > 0");
  if (d->page_size != 16) return fail(KVPRM_E_UNSUPPORTED, "kvprm_create: page_size must be 16");
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(KVPRM_E_UNSUPPORTED, "kvprm_create: head_dim must be 64 or 128");
  if (d->num_q_heads / d->num_kv_heads > 16)
    return fail(KVPRM_E_UNSUPPORTED, "kvprm_create: at most 16 query heads per kv-head");
  if (d->kv_dtype != KVPRM_F32 && d->num_kv_heads > kMaxKvHeadsMx)
    return fail(KVPRM_E_UNSUPPORTED, "kvprm_create: at most %d kv-heads with bf16/fp8 caches",
                kMaxKvHeadsMx);
  if (d->hidden % 64 != 0 || d->ffn_dim % 64 != 0 || (d->num_q_heads * d->head_dim) % 64 != 0)
    return fail(KVPRM_E_UNSUPPORTED, "kvprm_create: hidden, ffn_dim, n_q*d_h must be multiples of 64");
  const bool f32 = d->weight_dtype == KVPRM_F32 && d->kv_dtype == KVPRM_F32;
  const bool bf = d->weight_dtype == KVPRM_BF16 &&
                  (d->kv_dtype == KVPRM_BF16 || d->kv_dtype == KVPRM_FP8_E4M3);
  if (!f32 && !bf)
    return fail(KVPRM_E_UNSUPPORTED,
                "kvprm_create: dtype pair must be (F32, F32), (BF16, BF16) or (BF16, FP8_E4M3)");
  kvprm_handle h = new (std::nothrow) kvprm_handle_s;
  if (!h) return fail(KVPRM_E_INTERNAL, "kvprm_create: out of host memory");
  h->desc = *d;
  Dims &m = h->dm;
  m.layers = d->num_layers;
  m.H = d->hidden;
  m.nq = d->num_q_heads;
  m.nkv = d->num_kv_heads;
  m.d = d->head_dim;
  m.F = d->ffn_dim;
  m.g = d->num_q_heads / d->num_kv_heads;
  m.theta = d->rope_theta;
  m.eps = d->rms_eps;
  m.wdt = d->weight_dtype == KVPRM_BF16 ? 1 : 0;
  m.kvdt = d->kv_dtype == KVPRM_F32 ? 0 : (d->kv_dtype == KVPRM_BF16 ? 1 : 2);
  const char *dbg = getenv("KVPRM_DEBUG");
  h->debug = dbg && dbg[0] && strcmp(dbg, "0") != 0;
  *out = h;
  return ok();
}

kvprm_status kvprm_destroy(kvprm_handle h) {
  delete h;
  return ok();
}

static kvprm_status check_batch(const kvprm_handle h, const kvprm_batch *b, const char *fn) {
  if (!b) return fail(KVPRM_E_INVALID, "%s: null batch", fn);
  if (b->batch < 0) return fail(KVPRM_E_INVALID, "%s: batch < 0", fn);
  if (b->batch == 0) return KVPRM_OK;
  if (b->batch > 256) return fail(KVPRM_E_UNSUPPORTED, "%s: at most 256 candidates per call", fn);
  if (h->dm.wdt == 1 && b->batch > 64)
    return fail(KVPRM_E_UNSUPPORTED, "%s: at most 64 candidates per call with bf16 weights", fn);
  if (!b->page_table || !b->lengths) return fail(KVPRM_E_INVALID, "%s: null page_table or lengths", fn);
  if (b->max_pages < 1) return fail(KVPRM_E_INVALID, "%s: max_pages < 1", fn);
  // chunk slots per candidate: one per chunk of max_pages, plus one where a shared prefix
  // splits a chunk (chunks of 16 pages at the shortest, 32 on the vector-ALU path)
  const int max_mp = (kMaxChunks - 2) * (h->dm.kvdt == 0 ? kChunkPagesValu : 16);
  if (b->max_pages > max_mp)
    return fail(KVPRM_E_UNSUPPORTED, "%s: max_pages above %d", fn, max_mp);
  const int cap = b->max_pages * h->desc.page_size;
  if (b->lengths_host)
    for (int i = 0; i < b->batch; ++i)
      if (b->lengths_host[i] < 0 || b->lengths_host[i] > cap)
        return fail(KVPRM_E_INVALID, "%s: lengths[%d] = %d outside [0, %d]", fn, i,
                    b->lengths_host[i], cap);
  if (b->num_groups < 0) return fail(KVPRM_E_INVALID, "%s: num_groups < 0", fn);
  if (b->num_groups > 0) {
    const int *s = b->group_start_host, *pl = b->group_prefix_len_host;
    if (!s || !pl) return fail(KVPRM_E_INVALID, "%s: null group arrays", fn);
    if (!b->lengths_host)
      return fail(KVPRM_E_INVALID, "%s: the prefix-sharing hint needs lengths_host", fn);
    if (s[0] != 0 || s[b->num_groups] != b->batch)
      return fail(KVPRM_E_INVALID, "%s: groups must tile [0, batch)", fn);
    for (int g = 0; g < b->num_groups; ++g) {
      if (s[g + 1] <= s[g]) return fail(KVPRM_E_INVALID, "%s: group %d is empty or unordered", fn, g);
      if (pl[g] < 0 || pl[g] % h->desc.page_size != 0 || pl[g] > cap)
        return fail(KVPRM_E_INVALID, "%s: group %d prefix %d not a page multiple in [0, %d]", fn,
                    g, pl[g], cap);
      if (b->lengths_host)
        for (int i = s[g]; i < s[g + 1]; ++i)
          if (b->lengths_host[i] < pl[g])
            return fail(KVPRM_E_INVALID, "%s: candidate %d shorter than its group prefix", fn, i);
    }
  }
  return KVPRM_OK;
}

static kvprm_status check_cache(const kvprm_handle h, const kvprm_kv_cache *c, const char *fn) {
  if (!c || !c->k_pages || !c->v_pages) return fail(KVPRM_E_INVALID, "%s: null cache pool", fn);
  if (c->num_pages < 1) return fail(KVPRM_E_INVALID, "%s: num_pages < 1", fn);
  if (h->dm.kvdt == 2 && (!c->k_scale || !c->v_scale))
    return fail(KVPRM_E_INVALID, "%s: fp8 cache needs k_scale and v_scale", fn);
  return KVPRM_OK;
}

// Debug mode only: copy lengths and the page table to the host (on the call's stream, then
// wait) and check every read entry against [0, num_pages), every length against the table and
// against lengths_host (when given: the launch grids are sized from it), and, for the calls
// that write per-page results (distinct_pages: gradients and steering), that no physical page
// is read by two candidates.
static kvprm_status check_pages_debug(const kvprm_handle h, const kvprm_kv_cache *c,
                                      const kvprm_batch *b, hipStream_t s, const char *fn,
                                      bool distinct_pages = false) {
  if (!h->debug) return KVPRM_OK;
  std::vector<int32_t> len(b->batch), pt((size_t)b->batch * b->max_pages);
  if (hipMemcpyAsync(len.data(), b->lengths, len.size() * 4, hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipMemcpyAsync(pt.data(), b->page_table, pt.size() * 4, hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return fail(KVPRM_E_HIP, "%s: debug copy of the page table failed", fn);
  const int cap = b->max_pages * h->desc.page_size;
  std::vector<int32_t> owner(distinct_pages ? (size_t)c->num_pages : 0, -1);
  for (int i = 0; i < b->batch; ++i) {
    if (len[i] < 0 || len[i] > cap)
      return fail(KVPRM_E_INVALID, "%s: lengths[%d] = %d outside [0, %d]", fn, i, len[i], cap);
    if (b->lengths_host && b->lengths_host[i] != len[i])
      return fail(KVPRM_E_INVALID, "%s: lengths_host[%d] = %d differs from lengths[%d] = %d", fn,
                  i, b->lengths_host[i], i, len[i]);
    const int np = (len[i] + h->desc.page_size - 1) / h->desc.page_size;
    for (int k = 0; k < np; ++k) {
      const int32_t id = pt[(size_t)i * b->max_pages + k];
      if (id < 0 || id >= c->num_pages)
        return fail(KVPRM_E_INVALID, "%s: page_table[%d][%d] = %d outside [0, %d)", fn, i, k, id,
                    c->num_pages);
      if (distinct_pages) {
        if (owner[id] >= 0)
          return fail(KVPRM_E_INVALID, "%s: page %d is read by candidates %d and %d", fn, id,
                      owner[id], i);
        owner[id] = i;
      }
    }
  }
  return KVPRM_OK;
}

static size_t ws_bytes_for(const kvprm_handle h, const kvprm_batch *b) {
  Plan p = make_plan(h->dm, b->batch, b->max_pages);
  return carve(h->dm, p, nullptr).bytes;
}

kvprm_status kvprm_workspace_size(kvprm_handle h, const kvprm_batch *b, size_t *bytes) {
  if (!h || !bytes) return fail(KVPRM_E_INVALID, "kvprm_workspace_size: null argument");
  kvprm_status st = check_batch(h, b, "kvprm_workspace_size");
  if (st != KVPRM_OK) return st;
  *bytes = b->batch == 0 ? 0 : ws_bytes_for(h, b);
  return ok();
}

static kvprm_status check_ws(const kvprm_handle h, const kvprm_batch *b, void *ws, size_t n,
                             const char *fn) {
  const size_t need = ws_bytes_for(h, b);
  if (!ws || n < need)
    return fail(KVPRM_E_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, need,
                ws ? n : (size_t)0);
  if (((uintptr_t)ws & 255) != 0) return fail(KVPRM_E_WORKSPACE, "%s: workspace not 256-byte aligned", fn);
  return KVPRM_OK;
}

// Longest chunk (16, 32 or 64 pages) that leaves at least 160 work items for `pages` pages.
static int chunk_shift_for(long long pages) {
  int sh = 6;
  while (sh > 4 && pages < (160LL << sh)) --sh;
  return sh;
}

// Launch table of the attention kernels. The prefix-sharing hint is used by the matrix-core
// attention only (fp32 caches take the vector-ALU path, which reads every page per candidate)
// and only for up to kMaxGroups groups; otherwise it is ignored, which changes nothing but
// speed. With lengths on the host, the chunk lengths are chosen from the pages each kernel
// actually reads (private pages; group prefixes times their column blocks and kv-heads), and
// the chunk grid of the private pages is sized to the longest private range; without them the
// plan's chunk (from batch and max_pages) serves both.
static GroupTable group_table(const kvprm_handle h, const kvprm_batch *b, const Plan &p) {
  GroupTable gt;
  memset(&gt, 0, sizeof gt);
  gt.cshift_prefix = gt.cshift_private = p.cshift;
  const bool share = h->dm.kvdt != 0 && b->num_groups > 0 && b->num_groups <= kMaxGroups;
  const int kq = p.kq;  // group ranges are kept in rows (candidates x verify tokens)
  if (share) {
    gt.n = b->num_groups;
    for (int i = 0; i <= gt.n; ++i) gt.start[i] = b->group_start_host[i] * kq;
    const int cols_per_block = 16 * kPrefixWaves;
    long long items = 0;  // prefix pages x column blocks (per kv-head)
    for (int i = 0; i < gt.n; ++i) {
      const int pp = b->group_prefix_len_host[i] / kPage;
      const int members = gt.start[i + 1] - gt.start[i];
      gt.prefix_pages[i] = pp;
      const int blocks = pp > 0 ? (members * h->dm.g + cols_per_block - 1) / cols_per_block : 0;
      gt.colblock_start[i + 1] = gt.colblock_start[i] + blocks;
      items += (long long)pp * blocks;
    }
    // the hint requires host lengths (checked), so the chunks follow the actual work
    gt.cshift_prefix = chunk_shift_for(items * h->dm.nkv);
    for (int i = 0; i < gt.n; ++i) {
      const int ch = (gt.prefix_pages[i] + (1 << gt.cshift_prefix) - 1) >> gt.cshift_prefix;
      if (ch > gt.prefix_chunks) gt.prefix_chunks = ch;
    }
  }
  if (b->lengths_host) {
    long long priv_total = 0;
    for (int i = 0; i < b->batch; ++i) {
      int first = 0;
      for (int k = 0; k < gt.n; ++k)
        if (i * kq >= gt.start[k] && i * kq < gt.start[k + 1]) first = gt.prefix_pages[k];
      priv_total += (b->lengths_host[i] + kPage - 1) / kPage - first;
    }
    gt.cshift_private = chunk_shift_for(priv_total);
    const int CP = 1 << gt.cshift_private;
    int most = 1;
    for (int i = 0; i < b->batch; ++i) {
      int first = 0;
      for (int k = 0; k < gt.n; ++k)
        if (i * kq >= gt.start[k] && i * kq < gt.start[k + 1]) first = gt.prefix_pages[k];
      const int priv = (b->lengths_host[i] + kPage - 1) / kPage - first;
      const int ch = (priv + CP - 1) / CP;
      if (ch > most) most = ch;
    }
    gt.private_chunks = most;
  }
  return gt;
}

static kvprm_status check_readout(const kvprm_handle h, const kvprm_readout_weights *wts,
                                  const char *fn) {
  if (!wts || !wts->layers || !wts->verify_embed || !wts->final_norm || !wts->reward_w)
    return fail(KVPRM_E_INVALID, "%s: null readout weights", fn);
  for (int l = 0; l < h->dm.layers; ++l) {
    const kvprm_layer_weights &W = wts->layers[l];
    if (!W.attn_norm || !W.wq || !W.wk || !W.wv || !W.wo || !W.ffn_norm || !W.w_gate ||
        !W.w_up || !W.w_down)
      return fail(KVPRM_E_INVALID, "%s: null weight in layer %d", fn, l);
  }
  return KVPRM_OK;
}

static kvprm_status check_lora_rank(const kvprm_handle h, int32_t rank, const char *fn) {
  if (h->dm.wdt != 1)
    return fail(KVPRM_E_UNSUPPORTED, "%s: unmerged adapters need bf16 weights", fn);
  if (rank < 32 || rank > 512 || rank % 32 != 0)
    return fail(KVPRM_E_INVALID, "%s: adapter rank %d is not a multiple of 32 in [32, 512]", fn,
                rank);
  return KVPRM_OK;
}

static kvprm_status check_lora(const kvprm_handle h, const kvprm_lora *lora, const char *fn) {
  if (!lora || !lora->layers) return fail(KVPRM_E_INVALID, "%s: null adapter", fn);
  kvprm_status st = check_lora_rank(h, lora->rank, fn);
  if (st != KVPRM_OK) return st;
  if (!(lora->scale == lora->scale)) return fail(KVPRM_E_INVALID, "%s: adapter scale is NaN", fn);
  static const char *names[7] = {"q", "k", "v", "o", "gate", "up", "down"};
  for (int l = 0; l < h->dm.layers; ++l) {
    const kvprm_layer_lora &L = lora->layers[l];
    const kvprm_lora_factors f[7] = {L.q, L.k, L.v, L.o, L.gate, L.up, L.down};
    for (int i = 0; i < 7; ++i)
      if ((f[i].a == nullptr) != (f[i].b == nullptr))
        return fail(KVPRM_E_INVALID, "%s: layer %d adapter %s has one factor null", fn, l,
                    names[i]);
  }
  return KVPRM_OK;
}

// The matrix-core pipeline (bf16 weights), per layer: the q/k/v projection with the RMSNorm
// scale and the rotary embedding in its epilogue, the attention chunk kernel(s) and their merge,
// then the output, gate/up and down projections with their element-wise steps fused. The down
// projection (all batch sizes), q/k/v (more than 8 rows) and the output projection (more than 16
// rows, or large shapes) run instead as split-K products with a finish kernel each: seven to
// nine launches per layer (one more with shared prefixes). With an adapter, each
// projection group that has one first computes scale * A u (a split-K GEMV and its finish) and
// the projection adds B (scale * A u) as a tail of its input range.
// With sv, the activations the backward pass needs are kept per layer (GradSave).
static kvprm_status score_mx(const kvprm_handle h, const kvprm_kv_cache *cache,
                             const kvprm_batch *b, const kvprm_readout_weights *wts,
                             const kvprm_lora *lora, const Plan &p, const Workspace &w,
                             const GroupTable &gt, float *scores, float *logits, hipStream_t s,
                             const GradSave *sv = nullptr) {
  const Dims &dm = h->dm;
  const int EB = dm.kvdt == 0 ? 4 : (dm.kvdt == 1 ? 2 : 1);
  const size_t layer_bytes = (size_t)cache->num_pages * dm.nkv * kPage * dm.d * EB;
  const size_t layer_scales = (size_t)cache->num_pages * dm.nkv;
  const int tkb = lora ? lora->rank / 32 : 0;
  const LoraTail none{{nullptr, nullptr, nullptr}, 0};
  auto tail_of = [&](const void *b0, const void *b1, const void *b2) {
    LoraTail t{{b0, b1, b2}, (b0 || b1 || b2) ? tkb : 0};
    return t;
  };
  HIP_TRY(launch_init_mx(dm, p, w, wts->verify_embed, wts->layers[0].attn_norm, b->lengths, s,
                         sv ? sv->x_in : nullptr),
          "init");
  const size_t qd = (size_t)p.B * dm.nq * dm.d, kd = (size_t)p.B * dm.nkv * dm.d;
  for (int l = 0; l < dm.layers; ++l) {
    const kvprm_layer_weights &W = wts->layers[l];
    const void *gamma_next = l + 1 < dm.layers ? wts->layers[l + 1].attn_norm : nullptr;
    Workspace wl = w;  // with sv: q, k_self, v_self written to the layer's saved copies
    float *o_save = nullptr, *lse_save = nullptr, *gu_save = nullptr;
    if (sv) {  // (the residual stream entering the layer was saved by the previous epilogue)
      wl.q = sv->q + l * qd;
      wl.kself = sv->ks + l * kd;
      wl.vself = sv->vs + l * kd;
      o_save = sv->o + l * qd;
      lse_save = sv->lse + (size_t)l * p.B * dm.nq;
      gu_save = sv->gu + (size_t)l * p.B * 2 * dm.F;
    }
    LoraTail t_qkv = none, t_o = none, t_gu = none, t_d = none;
    if (lora) {
      const kvprm_layer_lora &A = lora->layers[l];
      t_qkv = tail_of(A.q.b, A.k.b, A.v.b);
      t_o = tail_of(A.o.b, nullptr, nullptr);
      t_gu = tail_of(A.gate.b, A.up.b, nullptr);
      t_d = tail_of(A.down.b, nullptr, nullptr);
      const void *a_qkv[3] = {A.q.a, A.k.a, A.v.a};
      HIP_TRY(launch_lora_a(dm, p, w, LORA_QKV, a_qkv, lora->scale, w.opA, s), "q/k/v adapter");
    }
    HIP_TRY(launch_qkv_mx(dm, p, wl, W.wq, W.wk, W.wv, t_qkv, s), "qkv projection");
    HIP_TRY(launch_attn_mx(dm, p, w, (const char *)cache->k_pages + layer_bytes * l,
                           (const char *)cache->v_pages + layer_bytes * l,
                           cache->k_scale ? cache->k_scale + layer_scales * l : nullptr,
                           cache->v_scale ? cache->v_scale + layer_scales * l : nullptr,
                           b->page_table, b->lengths, gt, wl.q, wl.kself, wl.vself, o_save,
                           w.opO, s, true, lse_save),
            "attention");
    if (lora && t_o.tkb) {
      const void *a_o[3] = {lora->layers[l].o.a, nullptr, nullptr};
      HIP_TRY(launch_lora_a(dm, p, w, LORA_O, a_o, lora->scale, w.opO, s), "output adapter");
    }
    HIP_TRY(launch_oproj_fused(dm, p, w, W.wo, W.ffn_norm, t_o, s,
                               sv ? sv->x_mid + (size_t)l * p.B * dm.H : nullptr),
            "output projection");
    if (lora && t_gu.tkb) {
      const void *a_gu[3] = {lora->layers[l].gate.a, lora->layers[l].up.a, nullptr};
      HIP_TRY(launch_lora_a(dm, p, w, LORA_GU, a_gu, lora->scale, w.opA, s), "gate/up adapter");
    }
    HIP_TRY(launch_gateup_fused(dm, p, w, W.w_gate, W.w_up, t_gu, s, gu_save),
            "gate/up projection");
    if (lora && t_d.tkb) {
      const void *a_d[3] = {lora->layers[l].down.a, nullptr, nullptr};
      HIP_TRY(launch_lora_a(dm, p, w, LORA_DOWN, a_d, lora->scale, w.opD, s), "down adapter");
    }
    HIP_TRY(launch_down_fused(dm, p, w, W.w_down, gamma_next, t_d, s,
                              sv && l + 1 < dm.layers ? sv->x_in + (size_t)(l + 1) * p.B * dm.H
                                                      : nullptr),
            "down projection");
  }
  HIP_TRY(launch_head(dm, p, w, wts->final_norm, wts->reward_w, wts->reward_b, scores, logits, s),
          "reward head");
  return KVPRM_OK;
}

static kvprm_status check_options(const kvprm_handle h, const kvprm_batch *b, const kvprm_lora *lora,
                                  int32_t depth, const char *fn) {
  if (depth < 1) return fail(KVPRM_E_INVALID, "%s: depth %d < 1", fn, depth);
  if (depth > 1) {
    if (h->dm.wdt != 1)
      return fail(KVPRM_E_UNSUPPORTED, "%s: a depth-k readout needs bf16 weights", fn);
    if (depth * h->dm.g > 16)
      return fail(KVPRM_E_UNSUPPORTED, "%s: depth %d x %d query heads per kv-head exceeds 16", fn,
                  depth, h->dm.g);
    if (b && (long long)b->batch * depth > 64)
      return fail(KVPRM_E_UNSUPPORTED, "%s: batch %d x depth %d exceeds 64 rows", fn, b->batch,
                  depth);
  }
  if (lora) return check_lora(h, lora, fn);
  return KVPRM_OK;
}

static size_t ws_bytes_ex(const kvprm_handle h, const kvprm_batch *b, const kvprm_lora *lora,
                          int32_t depth) {
  const Plan p = make_plan(h->dm, b->batch, b->max_pages, lora ? lora->rank : 0, depth);
  return carve(h->dm, p, nullptr).bytes;
}

// Every scoring entry point: validation, then the matrix-core pipeline (bf16 weights) or the
// vector-ALU one (fp32 weights; no adapter, depth 1).
static kvprm_status score_impl(kvprm_handle h, const kvprm_kv_cache *cache, const kvprm_batch *b,
                               const kvprm_readout_weights *wts, const kvprm_lora *lora,
                               int32_t depth, void *workspace, size_t ws_bytes, float *scores,
                               float *logits, void *stream, const char *fn) {
  if (!h) return fail(KVPRM_E_INVALID, "%s: null handle", fn);
  kvprm_status st = check_batch(h, b, fn);
  if (st != KVPRM_OK) return st;
  if ((st = check_options(h, b, lora, depth, fn)) != KVPRM_OK) return st;
  if (b->batch == 0) return ok();
  if ((st = check_cache(h, cache, fn)) != KVPRM_OK) return st;
  if ((st = check_readout(h, wts, fn)) != KVPRM_OK) return st;
  if (!scores) return fail(KVPRM_E_INVALID, "%s: null scores", fn);
  const size_t need = ws_bytes_ex(h, b, lora, depth);
  if (!workspace || ws_bytes < need)
    return fail(KVPRM_E_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, need,
                workspace ? ws_bytes : (size_t)0);
  if (((uintptr_t)workspace & 255) != 0)
    return fail(KVPRM_E_WORKSPACE, "%s: workspace not 256-byte aligned", fn);
  if ((st = check_pages_debug(h, cache, b, (hipStream_t)stream, fn)) != KVPRM_OK) return st;

  const Dims &dm = h->dm;
  hipStream_t s = (hipStream_t)stream;
  const Plan p = make_plan(dm, b->batch, b->max_pages, lora ? lora->rank : 0, depth);
  const Workspace w = carve(dm, p, workspace);
  const GroupTable gt = group_table(h, b, p);
  if (dm.wdt == 1) {
    if ((st = score_mx(h, cache, b, wts, lora, p, w, gt, scores, logits, s)) != KVPRM_OK)
      return st;
    return ok();
  }
  // vector-ALU pipeline (fp32 weights)
  HIP_TRY(launch_init(dm, p, w, wts->verify_embed, s), "init");
  for (int l = 0; l < dm.layers; ++l) {
    const kvprm_layer_weights &W = wts->layers[l];
    GemvSegs qkv{{W.wq, W.wk, W.wv}, {dm.nq * dm.d, dm.nkv * dm.d, dm.nkv * dm.d}, 3};
    HIP_TRY(launch_gemv(dm, p, qkv, dm.H, p.kslice_qkv, p.ks_qkv, w.x, W.attn_norm, w.ss, w.part, s),
            "qkv projection");
    HIP_TRY(launch_qkv_finish(dm, p, w, b->lengths, s), "rotary");
    HIP_TRY(launch_attention(dm, p, w, l, cache->k_pages, cache->v_pages, cache->k_scale,
                             cache->v_scale, cache->num_pages, b->page_table, b->lengths, gt, w.q,
                             w.kself, w.vself, w.o, s),
            "attention");
    GemvSegs wo{{W.wo, nullptr, nullptr}, {dm.H, 0, 0}, 1};
    HIP_TRY(launch_gemv(dm, p, wo, dm.nq * dm.d, p.kslice_o, p.ks_o, w.o, nullptr, nullptr, w.part, s),
            "output projection");
    HIP_TRY(launch_residual(dm, p, w, p.ks_o, s), "residual");
    GemvSegs gu{{W.w_gate, W.w_up, nullptr}, {dm.F, dm.F, 0}, 2};
    HIP_TRY(launch_gemv(dm, p, gu, dm.H, p.kslice_gu, p.ks_gu, w.x, W.ffn_norm, w.ss, w.part, s),
            "gate/up projection");
    HIP_TRY(launch_swiglu(dm, p, w, p.ks_gu, s), "swiglu");
    GemvSegs dn{{W.w_down, nullptr, nullptr}, {dm.H, 0, 0}, 1};
    HIP_TRY(launch_gemv(dm, p, dn, dm.F, p.kslice_d, p.ks_d, w.hffn, nullptr, nullptr, w.part, s),
            "down projection");
    HIP_TRY(launch_residual(dm, p, w, p.ks_d, s), "residual");
  }
  HIP_TRY(launch_head(dm, p, w, wts->final_norm, wts->reward_w, wts->reward_b, scores, logits, s),
          "reward head");
  return ok();
}

kvprm_status kvprm_score(kvprm_handle h, const kvprm_kv_cache *cache, const kvprm_batch *b,
                         const kvprm_readout_weights *wts, void *workspace, size_t ws_bytes,
                         float *scores, float *logits, void *stream) {
  return score_impl(h, cache, b, wts, nullptr, 1, workspace, ws_bytes, scores, logits, stream,
                    "kvprm_score");
}

// ---------------------------------------------------------------- allocation-free scoring

// Workspace of kvprm_score_static: one array per GPU, held by the library's code object on every
// device it is loaded on until the process ends. Host code never uses this name as an address
// (on the host it is a stand-in, not device memory): the device address of the current device's
// copy comes from hipGetSymbolAddress and is kept in g_static_ws.
static __device__ __align__(256) unsigned char scratch[KVPRM_STATIC_WORKSPACE_BYTES];

constexpr int kMaxDevices = 64;
static std::mutex g_static_mu;
static void *g_static_ws[kMaxDevices];

// The current device's copy of `scratch` (resolved once per device, with that device current);
// a non-null stream must belong to the current device.
static kvprm_status static_workspace(hipStream_t s, void **ptr, const char *fn) {
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev), "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(KVPRM_E_UNSUPPORTED, "%s: device %d outside [0, %d)", fn, dev, kMaxDevices);
  if (s) {
    hipDevice_t sdev = -1;
    HIP_TRY(hipStreamGetDevice(s, &sdev), "hipStreamGetDevice");
    if (sdev != dev)
      return fail(KVPRM_E_INVALID, "%s: the stream belongs to device %d, device %d is current", fn,
                  (int)sdev, dev);
  }
  std::lock_guard<std::mutex> lock(g_static_mu);
  if (!g_static_ws[dev]) {
    void *p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
    if (!p || ((uintptr_t)p & 255) != 0)
      return fail(KVPRM_E_INTERNAL, "%s: static workspace address %p is not 256-byte aligned", fn, p);
    g_static_ws[dev] = p;
  }
  *ptr = g_static_ws[dev];
  return KVPRM_OK;
}

kvprm_status kvprm_score_static(kvprm_handle h, const kvprm_kv_cache *cache, const kvprm_batch *b,
                                const kvprm_readout_weights *wts, float *scores, float *logits,
                                void *stream) {
  const char *fn = "kvprm_score_static";
  if (!h) return fail(KVPRM_E_INVALID, "%s: null handle", fn);
  kvprm_status st = check_batch(h, b, fn);
  if (st != KVPRM_OK) return st;
  if (b->batch == 0) return ok();
  const size_t need = ws_bytes_for(h, b);
  if (need > (size_t)KVPRM_STATIC_WORKSPACE_BYTES)
    return fail(KVPRM_E_WORKSPACE, "%s: the batch needs %zu bytes of workspace, the static one holds %zu",
                fn, need, (size_t)KVPRM_STATIC_WORKSPACE_BYTES);
  void *ws = nullptr;
  if ((st = static_workspace((hipStream_t)stream, &ws, fn)) != KVPRM_OK) return st;
  return score_impl(h, cache, b, wts, nullptr, 1, ws, (size_t)KVPRM_STATIC_WORKSPACE_BYTES, scores,
                    logits, stream, fn);
}

kvprm_status kvprm_workspace_size_lora(kvprm_handle h, const kvprm_batch *b, int32_t rank,
                                       size_t *bytes) {
  const char *fn = "kvprm_workspace_size_lora";
  if (!h || !bytes) return fail(KVPRM_E_INVALID, "%s: null argument", fn);
  kvprm_status st = check_lora_rank(h, rank, fn);
  if (st != KVPRM_OK) return st;
  if ((st = check_batch(h, b, fn)) != KVPRM_OK) return st;
  if (b->batch == 0) {
    *bytes = 0;
    return ok();
  }
  const Plan p = make_plan(h->dm, b->batch, b->max_pages, rank);
  *bytes = carve(h->dm, p, nullptr).bytes;
  return ok();
}

kvprm_status kvprm_score_lora(kvprm_handle h, const kvprm_kv_cache *cache, const kvprm_batch *b,
                              const kvprm_readout_weights *base, const kvprm_lora *lora,
                              void *workspace, size_t ws_bytes, float *scores, float *logits,
                              void *stream) {
  const char *fn = "kvprm_score_lora";
  if (!h) return fail(KVPRM_E_INVALID, "%s: null handle", fn);
  if (!lora) return fail(KVPRM_E_INVALID, "%s: null adapter", fn);
  return score_impl(h, cache, b, base, lora, 1, workspace, ws_bytes, scores, logits, stream, fn);
}

kvprm_status kvprm_workspace_size_ex(kvprm_handle h, const kvprm_batch *b,
                                     const kvprm_score_options *opt, size_t *bytes) {
  const char *fn = "kvprm_workspace_size_ex";
  if (!h || !bytes) return fail(KVPRM_E_INVALID, "%s: null argument", fn);
  kvprm_status st = check_batch(h, b, fn);
  if (st != KVPRM_OK) return st;
  const kvprm_lora *lora = opt ? opt->lora : nullptr;
  const int32_t depth = opt ? opt->depth : 1;
  if ((st = check_options(h, b, lora, depth, fn)) != KVPRM_OK) return st;
  *bytes = b->batch == 0 ? 0 : ws_bytes_ex(h, b, lora, depth);
  return ok();
}

kvprm_status kvprm_score_ex(kvprm_handle h, const kvprm_kv_cache *cache, const kvprm_batch *b,
                            const kvprm_readout_weights *wts, const kvprm_score_options *opt,
                            void *workspace, size_t ws_bytes, float *scores, float *logits,
                            void *stream) {
  return score_impl(h, cache, b, wts, opt ? opt->lora : nullptr, opt ? opt->depth : 1, workspace,
                    ws_bytes, scores, logits, stream, "kvprm_score_ex");
}

// ------------------------------------------------------------------ gradients and steering

static size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

static kvprm_status check_grad(const kvprm_handle h, const kvprm_batch *b, const char *fn) {
  if (h->dm.wdt != 1 || h->dm.kvdt != 1)
    return fail(KVPRM_E_UNSUPPORTED, "%s: cache gradients need bf16 weights and a bf16 cache", fn);
  if (b->batch > 8) return fail(KVPRM_E_UNSUPPORTED, "%s: at most 8 candidates", fn);
  if (h->dm.H > kGradMaxHidden)
    return fail(KVPRM_E_UNSUPPORTED, "%s: hidden size above %d", fn, kGradMaxHidden);
  // the row tiles of the transposed gate/up and q/k/v products must fit the splits
  const int max_rows = kGradMaxSplits * kTgemvWindow * 8;
  if (h->dm.F > max_rows || (h->dm.nq + 2 * h->dm.nkv) * h->dm.d > max_rows)
    return fail(KVPRM_E_UNSUPPORTED, "%s: ffn_dim or (n_q + 2 n_kv) d_h above %d", fn, max_rows);
  if (b->num_groups != 0)
    return fail(KVPRM_E_INVALID, "%s: candidates must not share cache pages (no prefix hint)", fn);
  return KVPRM_OK;
}

static size_t grad_ws_bytes(const kvprm_handle h, const kvprm_batch *b) {
  const Plan p = make_plan(h->dm, b->batch, b->max_pages);
  return align_up(carve(h->dm, p, nullptr).bytes) + carve_grad(h->dm, p, nullptr).bytes;
}

kvprm_status kvprm_workspace_size_grad(kvprm_handle h, const kvprm_batch *b, size_t *bytes) {
  const char *fn = "kvprm_workspace_size_grad";
  if (!h || !bytes) return fail(KVPRM_E_INVALID, "%s: null argument", fn);
  kvprm_status st = check_batch(h, b, fn);
  if (st != KVPRM_OK) return st;
  if (b->batch == 0) {
    *bytes = 0;
    return ok();
  }
  if ((st = check_grad(h, b, fn)) != KVPRM_OK) return st;
  *bytes = grad_ws_bytes(h, b);
  return ok();
}

// `steps` rounds of forward (activations saved) and backward; with grad_k / grad_v the
// backward writes the gradient (one round), otherwise it steps the cache in place by -eta.
static kvprm_status grad_impl(kvprm_handle h, const kvprm_kv_cache *cache, const kvprm_batch *b,
                              const kvprm_readout_weights *wts, void *workspace, size_t ws_bytes,
                              float *scores, float *grad_k, float *grad_v, float eta,
                              int32_t steps, float *scores_after, void *stream, const char *fn) {
  if (!h) return fail(KVPRM_E_INVALID, "%s: null handle", fn);
  kvprm_status st = check_batch(h, b, fn);
  if (st != KVPRM_OK) return st;
  if (b->batch == 0) return ok();
  if ((st = check_grad(h, b, fn)) != KVPRM_OK) return st;
  if ((st = check_cache(h, cache, fn)) != KVPRM_OK) return st;
  if ((st = check_readout(h, wts, fn)) != KVPRM_OK) return st;
  const size_t need = grad_ws_bytes(h, b);
  if (!workspace || ws_bytes < need)
    return fail(KVPRM_E_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, need,
                workspace ? ws_bytes : (size_t)0);
  if (((uintptr_t)workspace & 255) != 0)
    return fail(KVPRM_E_WORKSPACE, "%s: workspace not 256-byte aligned", fn);
  if ((st = check_pages_debug(h, cache, b, (hipStream_t)stream, fn, true)) != KVPRM_OK) return st;
  const Dims &dm = h->dm;
  hipStream_t s = (hipStream_t)stream;
  const Plan p = make_plan(dm, b->batch, b->max_pages);
  const Workspace w = carve(dm, p, workspace);
  const GradSave sv = carve_grad(dm, p, (char *)workspace + align_up(w.bytes));
  const GroupTable gt = group_table(h, b, p);
  // the backward attention walks 16-page chunks (partial slots of the plan are sized for them)
  const int CP = 16;
  const int chunks = p.nch - 1;
  const size_t layer_bytes = (size_t)cache->num_pages * dm.nkv * kPage * dm.d * 2;
  for (int t = 0; t < steps; ++t) {
    // scores of the cache as it enters each step; the caller's array holds the first
    if ((st = score_mx(h, cache, b, wts, nullptr, p, w, gt, t == 0 ? scores : sv.Dh, nullptr, s,
                       &sv)) != KVPRM_OK)
      return st;
    HIP_TRY(launch_backward(dm, p, w, sv, wts->layers, wts->final_norm, wts->reward_w,
                            wts->reward_b, (char *)cache->k_pages, (char *)cache->v_pages,
                            layer_bytes, b->page_table, b->lengths, CP, chunks, grad_k, grad_v,
                            eta, s),
            "backward");
  }
  if (scores_after)
    if ((st = score_mx(h, cache, b, wts, nullptr, p, w, gt, scores_after, nullptr, s)) != KVPRM_OK)
      return st;
  return ok();
}

kvprm_status kvprm_score_grad(kvprm_handle h, const kvprm_kv_cache *cache, const kvprm_batch *b,
                              const kvprm_readout_weights *weights, void *workspace,
                              size_t ws_bytes, float *scores, float *grad_k, float *grad_v,
                              void *stream) {
  const char *fn = "kvprm_score_grad";
  if (!scores || !grad_k || !grad_v) return fail(KVPRM_E_INVALID, "%s: null output", fn);
  return grad_impl(h, cache, b, weights, workspace, ws_bytes, scores, grad_k, grad_v, 0.f, 1,
                   nullptr, stream, fn);
}

kvprm_status kvprm_steer(kvprm_handle h, const kvprm_kv_cache *cache, const kvprm_batch *b,
                         const kvprm_readout_weights *weights, float eta, int32_t steps,
                         void *workspace, size_t ws_bytes, float *scores_before,
                         float *scores_after, void *stream) {
  const char *fn = "kvprm_steer";
  if (!scores_before || !scores_after) return fail(KVPRM_E_INVALID, "%s: null output", fn);
  if (steps < 1) return fail(KVPRM_E_INVALID, "%s: steps %d < 1", fn, steps);
  if (!(eta == eta)) return fail(KVPRM_E_INVALID, "%s: eta is NaN", fn);
  return grad_impl(h, cache, b, weights, workspace, ws_bytes, scores_before, nullptr, nullptr,
                   eta, steps, scores_after, stream, fn);
}

kvprm_status kvprm_pack_weight(const void *src, void *dst, int64_t rows, int64_t K, void *stream) {
  const char *fn = "kvprm_pack_weight";
  if (!src || !dst) return fail(KVPRM_E_INVALID, "%s: null pointer", fn);
  if (rows <= 0 || K <= 0 || rows % 16 != 0 || K % 32 != 0)
    return fail(KVPRM_E_INVALID, "%s: rows %% 16 and K %% 32 must be 0 (rows=%lld, K=%lld)", fn,
                (long long)rows, (long long)K);
  const uintptr_t a = (uintptr_t)src, b = (uintptr_t)dst, n = (uintptr_t)(rows * K * 2);
  if (a < b + n && b < a + n) return fail(KVPRM_E_INVALID, "%s: src and dst overlap", fn);
  if ((a | b) & 15) return fail(KVPRM_E_INVALID, "%s: pointers must be 16-byte aligned", fn);
  HIP_TRY(launch_pack_weight(src, dst, rows, K, (hipStream_t)stream), "pack");
  return ok();
}

kvprm_status kvprm_pack_kv(const void *src, void *dst, int64_t num_tiles, int32_t head_dim,
                           kvprm_dtype dtype, kvprm_kv_part part, void *stream) {
  const char *fn = "kvprm_pack_kv";
  if (num_tiles < 0) return fail(KVPRM_E_INVALID, "%s: num_tiles < 0", fn);
  if (head_dim != 64 && head_dim != 128)
    return fail(KVPRM_E_UNSUPPORTED, "%s: head_dim must be 64 or 128", fn);
  if (dtype != KVPRM_F32 && dtype != KVPRM_BF16 && dtype != KVPRM_FP8_E4M3)
    return fail(KVPRM_E_INVALID, "%s: unknown dtype %d", fn, (int)dtype);
  if (part != KVPRM_KEYS && part != KVPRM_VALUES)
    return fail(KVPRM_E_INVALID, "%s: part must be KVPRM_KEYS or KVPRM_VALUES", fn);
  if (num_tiles == 0) return ok();
  if (!src || !dst) return fail(KVPRM_E_INVALID, "%s: null pointer", fn);
  const int eb = dtype == KVPRM_F32 ? 4 : (dtype == KVPRM_BF16 ? 2 : 1);
  const uintptr_t a = (uintptr_t)src, b = (uintptr_t)dst;
  const uintptr_t n = (uintptr_t)num_tiles * 16 * (uintptr_t)head_dim * (uintptr_t)eb;
  if (a < b + n && b < a + n) return fail(KVPRM_E_INVALID, "%s: src and dst overlap", fn);
  if ((a | b) & 15) return fail(KVPRM_E_INVALID, "%s: pointers must be 16-byte aligned", fn);
  HIP_TRY(launch_pack_kv(src, dst, num_tiles, head_dim, eb, part == KVPRM_VALUES,
                         (hipStream_t)stream),
          "pack kv");
  return ok();
}

kvprm_status kvprm_stream_read(const void *buf, size_t bytes, uint32_t *sink, void *stream) {
  const char *fn = "kvprm_stream_read";
  if (!buf || !sink) return fail(KVPRM_E_INVALID, "%s: null pointer", fn);
  if (bytes == 0 || bytes % 16 != 0)
    return fail(KVPRM_E_INVALID, "%s: bytes must be a positive multiple of 16", fn);
  if ((uintptr_t)buf & 15) return fail(KVPRM_E_INVALID, "%s: buf must be 16-byte aligned", fn);
  if ((uintptr_t)sink & 3) return fail(KVPRM_E_INVALID, "%s: sink must be 4-byte aligned", fn);
  HIP_TRY(launch_stream_read(buf, bytes, sink, (hipStream_t)stream), "stream read");
  return ok();
}

kvprm_status kvprm_attention(kvprm_handle h, const kvprm_kv_cache *cache, const kvprm_batch *b,
                             int32_t layer, const float *q, const float *k_self,
                             const float *v_self, void *workspace, size_t ws_bytes, float *o,
                             void *stream) {
  const char *fn = "kvprm_attention";
  if (!h) return fail(KVPRM_E_INVALID, "%s: null handle", fn);
  kvprm_status st = check_batch(h, b, fn);
  if (st != KVPRM_OK) return st;
  if (b->batch == 0) return ok();
  if ((st = check_cache(h, cache, fn)) != KVPRM_OK) return st;
  if (layer < 0 || layer >= h->dm.layers)
    return fail(KVPRM_E_INVALID, "%s: layer %d outside [0, %d)", fn, layer, h->dm.layers);
  if (!q || !k_self || !v_self || !o) return fail(KVPRM_E_INVALID, "%s: null q/k_self/v_self/o", fn);
  if ((st = check_ws(h, b, workspace, ws_bytes, fn)) != KVPRM_OK) return st;
  if ((st = check_pages_debug(h, cache, b, (hipStream_t)stream, fn)) != KVPRM_OK) return st;
  const Dims &dm = h->dm;
  const Plan p = make_plan(dm, b->batch, b->max_pages);
  const Workspace w = carve(dm, p, workspace);
  HIP_TRY(launch_attention(dm, p, w, layer, cache->k_pages, cache->v_pages, cache->k_scale,
                           cache->v_scale, cache->num_pages, b->page_table, b->lengths,
                           group_table(h, b, p), q, k_self, v_self, o, (hipStream_t)stream),
          "attention");
  return ok();
}

kvprm_status kvprm_attention_partials(kvprm_handle h, const kvprm_kv_cache *cache,
                                      const kvprm_batch *b, int32_t layer, const float *q,
                                      void *workspace, size_t ws_bytes, void *stream) {
  const char *fn = "kvprm_attention_partials";
  if (!h) return fail(KVPRM_E_INVALID, "%s: null handle", fn);
  kvprm_status st = check_batch(h, b, fn);
  if (st != KVPRM_OK) return st;
  if (b->batch == 0) return ok();
  if ((st = check_cache(h, cache, fn)) != KVPRM_OK) return st;
  if (layer < 0 || layer >= h->dm.layers)
    return fail(KVPRM_E_INVALID, "%s: layer %d outside [0, %d)", fn, layer, h->dm.layers);
  if (!q) return fail(KVPRM_E_INVALID, "%s: null q", fn);
  if ((st = check_ws(h, b, workspace, ws_bytes, fn)) != KVPRM_OK) return st;
  if ((st = check_pages_debug(h, cache, b, (hipStream_t)stream, fn)) != KVPRM_OK) return st;
  const Dims &dm = h->dm;
  const Plan p = make_plan(dm, b->batch, b->max_pages);
  const Workspace w = carve(dm, p, workspace);
  HIP_TRY(launch_attention(dm, p, w, layer, cache->k_pages, cache->v_pages, cache->k_scale,
                           cache->v_scale, cache->num_pages, b->page_table, b->lengths,
                           group_table(h, b, p), q, nullptr, nullptr, nullptr,
                           (hipStream_t)stream, false),
          "attention partials");
  return ok();
}

}  // extern "C"
