// hs_api.cpp — the C ABI of libhs (include/hs.h): argument/state checks on
// host mirrors, workspace ownership, and the per-step launch sequence.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>

#include "hs_internal.h"

namespace hs {

thread_local std::string g_err;

int fail(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

}  // namespace hs

using namespace hs;

namespace {

#define HIP_TRY(expr)                                                                      \
  do {                                                                                     \
    hipError_t e_ = (expr);                                                                \
    if (e_ != hipSuccess) return fail(HS_E_DEVICE, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

int dtype_bytes(int dt) { return dt == HS_F32 ? 4 : 2; }

// Light checks needed by the size formula alone.
bool shape_ok(const hs_config *c) {
  return c && c->n_layers > 0 && c->n_kv_heads > 0 && c->head_dim > 0 && c->d_model > 0 && c->dtype >= HS_F32 &&
         c->dtype <= HS_BF16;
}

int check_config(const hs_config *c) {
  if (!shape_ok(c)) return fail(HS_E_INVALID, "config: non-positive size or unknown dtype");
  if (c->n_heads <= 0 || c->ffn_dim <= 0 || c->vocab <= 0)
    return fail(HS_E_INVALID, "config: non-positive n_heads/ffn_dim/vocab");
  if (c->n_heads % c->n_kv_heads) return fail(HS_E_INVALID, "config: n_heads %% n_kv_heads != 0");
  if (c->head_dim % 32) return fail(HS_E_INVALID, "config: head_dim / 2 must be a multiple of 16");
  const int group = c->n_heads / c->n_kv_heads;
  if (!attn_supported(c->dtype, c->head_dim, group))
    return fail(HS_E_INVALID, "config: head_dim %d with %d query heads per KV head is not supported", c->head_dim,
                group);
  const int ce = 16 / dtype_bytes(c->dtype);
  if (c->d_model % ce || (c->n_heads * c->head_dim) % ce || c->ffn_dim % ce)
    return fail(HS_E_INVALID, "config: d_model, n_heads*head_dim and ffn_dim must be multiples of %d", ce);
  if (c->rope_kind != HS_ROPE_1D && c->rope_kind != HS_ROPE_M3) return fail(HS_E_INVALID, "config: rope_kind");
  if (c->rope_kind == HS_ROPE_M3) {
    const int *s = c->mrope_section;
    if (s[0] < 0 || s[1] < 0 || s[2] < 0 || s[0] + s[1] + s[2] != c->head_dim / 2)
      return fail(HS_E_INVALID, "config: M-RoPE sections must sum to head_dim / 2");
  }
  if (!(c->rope_theta > 0.f) || !(c->rms_eps >= 0.f)) return fail(HS_E_INVALID, "config: rope_theta/rms_eps");
  if (c->qkv_bias != 0 && c->qkv_bias != 1) return fail(HS_E_INVALID, "config: qkv_bias");
  return HS_OK;
}

// Attention work decomposition for nq queries of at most max_len positions.
// A work group covers one (query, KV head) and S consecutive positions.  The
// positions of a pair are cut into splits until there are about four work
// groups per CU, but no further than one batch of K/V loads per wave (round =
// ATTN_WAVES x positions per wave-wide load x loads per batch; a matrix-core
// wave takes 16 positions per tile and ATTN_MMA_BATCH tiles per batch); S is
// a multiple of the positions one work-group iteration covers.  Many pairs
// keep one split each.
void split_policy(int nq, int n_kv, int group, int head_dim, int dtype, int max_len, int *S, int *n_split) {
  const int ce = dtype == HS_F32 ? 4 : 8;
  const bool mma = attn_uses_mma(dtype, group);  // 16-position tiles per wave
  const int step = ATTN_WAVES * (mma ? 16 : 64 * ce / head_dim);
  const int round = step * (mma ? ATTN_MMA_BATCH : attn_batch(group));
  const int64_t pairs = (int64_t)nq * n_kv;
  // (two per CU instead of four: Qwen-shaped batch 16, 8 splits against 16,
  // 3.625 against 3.577 ms per step)
  const int want = (int)std::max<int64_t>(1, (1024 + pairs - 1) / pairs);
  const int by_round = std::max(1, (max_len + round - 1) / round);
  const int ns = std::min(std::min(want, by_round), ATTN_MAX_SPLITS);
  int s = (max_len + ns - 1) / ns;
  s = (s + step - 1) / step * step;
  *S = s;
  *n_split = (max_len + s - 1) / s;
}

int64_t kv_request_elems(const hs_config &c, int cap) {
  return 2ll * c.n_layers * c.n_kv_heads * (int64_t)c.head_dim * cap;
}

// A handle works with any model of the same configuration whose max_ctx
// covers its capacities (each model brings its own weights and workspaces),
// e.g. several copies of the weights.
bool kv_matches(const hs_kv *kv, const hs_model *m) {
  return kv && m && kv->m && std::memcmp(&kv->m->cfg, &m->cfg, sizeof(hs_config)) == 0 && kv->max_cap <= m->max_ctx;
}

KvRef kv_ref(const hs_kv *kv) {
  return KvRef{kv->buf,   kv->d_base, kv->d_toff, kv->d_bt,  kv->d_cap,
               kv->d_len, kv->d_act,  kv->batch,  kv->ntab, kv->pool ? 1 : 0};
}

KvPool kv_pool(const hs_kv *kv) {
  return KvPool{kv->d_base, kv->d_toff,  kv->d_cap, kv->d_len,   kv->d_rope,       kv->d_ready,
                kv->d_nblk, kv->d_stack, kv->d_top, kv->m->status, kv->d_act, kv->block_tokens,
                kv->block_elems};
}

int blocks_for(const hs_kv *kv, int len) { return (len + kv->block_tokens - 1) / kv->block_tokens; }

// The split policy; a pooled cache's splits are whole multiples of
// POOL_SPAN positions, the longest batch of loads of any attention kernel, so
// that no batch crosses a block (blocks are multiples of it too).
constexpr int POOL_SPAN = 256;
void kv_split_policy(const hs_config &c, bool pool, int nq, int max_len, int *S, int *ns) {
  split_policy(nq, c.n_kv_heads, c.n_heads / c.n_kv_heads, c.head_dim, c.dtype, max_len, S, ns);
  if (!pool) return;
  *S = (*S + POOL_SPAN - 1) / POOL_SPAN * POOL_SPAN;
  *ns = (max_len + *S - 1) / *S;
}

// the decode columns' dispatch order, longest first; every request grows by
// one position per step, so it holds until the batch changes
hipError_t rebuild_order(hs_kv *kv, hipStream_t st) {
  return launch_build_order(kv->d_len, kv->pool ? kv->d_act : nullptr, kv->n_active, kv->d_order, st);
}

// the ready requests, in order, as the decode columns (pooled caches)
hipError_t rebuild_active(hs_kv *kv, hipStream_t st) {
  kv->act_host.clear();
  for (int r = 0; r < kv->batch; ++r)
    if (kv->ready[r]) kv->act_host.push_back(r);
  kv->n_active = (int)kv->act_host.size();
  const hipError_t e = launch_build_act(kv->d_ready, kv->batch, kv->d_act, st);
  return e != hipSuccess ? e : rebuild_order(kv, st);
}

void free_model(hs_model *m) {
  if (!m) return;
  void *ptrs[] = {m->x,      m->q,      m->attn,    m->act,      m->hnorm,  m->splitk, m->xlast,
                  m->pk_dev, m->logits, m->part_o, m->part_ml, m->rope_tab, m->status};
  for (void *p : ptrs)
    if (p) (void)hipFree(p);
  delete m;
}

// The device scratch one pass works in: the residual stream, the q,
// attention, SwiGLU and normalised-row activations, the K-split and
// attention-split partials, and the logits the LM head writes when the caller
// passes no buffer.  Normally the model's workspaces (hs_model_create);
// hs_decode_step_static carves them from a static device array instead.
struct StepWs {
  float *x;
  void *q, *attn, *act, *hnorm;
  float *splitk;
  int64_t splitk_floats;
  float *part_o, *part_ml;
  float *logits;
};

StepWs model_ws(const hs_model *m) {
  return StepWs{m->x, m->q, m->attn, m->act, m->hnorm, m->splitk, m->splitk_floats, m->part_o, m->part_ml, m->logits};
}

// The launches of one pass over ncols activation rows held in ws.x: decode
// (one row per request, prefill = 0) or prefill (the packed rows of the
// requests in pk).  Each member launches one kernel.
struct Step {
  hs_model *m;
  hs_kv *kv;
  int ncols, prefill;
  PackedRows pk;
  const int *rope_pos;
  int rope_ld;
  int S, n_split;
  hipStream_t st;
  StepWs ws;

  // K splits the residual projection over K inputs leaves in ws.splitk for
  // the next RMSNorm to add: in decode, when the projection reads its
  // activations from memory and that norm runs in its own kernel (0: it adds
  // into ws.x itself)
  int defer(int K) const {
    const hs_config &c = m->cfg;
    return prefill ? 0 : resid_defer_splits(c.dtype, ncols, K, c.d_model, ws.splitk_floats);
  }
  int o_defer() const {
    const hs_config &c = m->cfg;
    return combine_fused() ? 0 : defer(c.n_heads * c.head_dim);
  }
  int down_defer() const { return defer(m->cfg.ffn_dim); }

  // pend: splits of partials the previous residual projection left pending
  hipError_t qkv(int l, int pend) const {
    const hs_config &c = m->cfg;
    const hs_layer_weights &W = m->layers[l];
    GemmArgs g{};
    g.w[0] = W.wq;
    g.w[1] = W.wk;
    g.w[2] = W.wv;
    if (c.qkv_bias) {
      g.bias[0] = W.bq;
      g.bias[1] = W.bk;
      g.bias[2] = W.bv;
    }
    g.rows[0] = c.n_heads * c.head_dim;
    g.rows[1] = g.rows[2] = c.n_kv_heads * c.head_dim;
    g.K = c.d_model;
    g.ncols = ncols;
    g.x = ws.x;
    g.gain = W.attn_norm;
    g.h_work = ws.hnorm;
    g.eps = c.rms_eps;
    g.pend = (const double *)ws.splitk;
    g.pend_s = pend;
    g.out = ws.q;
    g.ld_out = c.n_heads * c.head_dim;
    g.head_dim = c.head_dim;
    g.n_heads = c.n_heads;
    g.n_kv = c.n_kv_heads;
    g.kv = kv_ref(kv);
    g.layer = l;
    g.prefill = prefill;
    g.pk = m->pk_dev;
    g.rope_pos = rope_pos;
    g.rope_ld = rope_ld;
    g.rope_m3 = c.rope_kind == HS_ROPE_M3;
    g.sec0 = c.mrope_section[0];
    g.sec1 = c.mrope_section[0] + c.mrope_section[1];
    g.rope_tab = m->rope_tab;
    g.rope_max = m->max_ctx;
    g.status = m->status;
    g.splitk_ws = ws.splitk;
    g.splitk_cap = ws.splitk_floats;
    return launch_gemm(c.dtype, PRO_NORM, kv->pool ? EPI_QKV_PAGED : EPI_QKV, g, st);
  }

  AttnArgs attn_args(int l) const {
    const hs_config &c = m->cfg;
    AttnArgs a{};
    a.q = ws.q;
    a.ld_q = c.n_heads * c.head_dim;
    a.kv = kv_ref(kv);
    a.layer = l;
    a.n_heads = c.n_heads;
    a.n_kv = c.n_kv_heads;
    a.prefill = prefill;
    a.pk = m->pk_dev;
    a.prefill_tiles = pk.tcu[pk.n];
    a.prefill_pairs = 0;
    for (int i = 0; i < pk.n; ++i) a.prefill_pairs += (pk.tcu[i + 1] - pk.tcu[i] + 1) / 2;
    a.S = S;
    a.n_split = n_split;
    a.part_o = ws.part_o;
    a.part_ml = ws.part_ml;
    a.scale = (float)(1.0 / std::sqrt((double)c.head_dim));
    a.order = !prefill && ncols > 1 ? kv->d_order : nullptr;
    a.out = ws.attn;
    // in the layout the O projection reads
    a.out_packed = gemm_x_packed(c.dtype, ncols, c.n_heads * c.head_dim) ? 1 : 0;
    return a;
  }

  hipError_t attn(int l) const {
    const hs_config &c = m->cfg;
    if (prefill && attn_prefill_on_mma(c.dtype))
      return launch_attention_prefill(c.dtype, c.head_dim, c.n_heads / c.n_kv_heads, ncols, attn_args(l), st);
    return launch_attention(c.dtype, c.head_dim, c.n_heads / c.n_kv_heads, ncols, attn_args(l), st);
  }

  // the split combine runs in the O projection's prologue when it fits there
  bool combine_fused() const {
    const hs_config &c = m->cfg;
    return gemm_combine_fusable(c.dtype, ncols, c.n_heads * c.head_dim, c.n_heads, n_split);
  }

  // launches nothing with a single split or a fused combine
  hipError_t combine(int l) const {
    const hs_config &c = m->cfg;
    if (n_split <= 1 || combine_fused()) return hipSuccess;
    return launch_combine(c.dtype, c.head_dim, ncols, attn_args(l), st);
  }

  hipError_t residual(const void *w, int K, const void *x, int x_packed, int defer_s) const {
    const hs_config &c = m->cfg;
    GemmArgs o{};
    o.defer = defer_s;
    o.w[0] = w;
    o.rows[0] = c.d_model;
    o.K = K;
    o.ncols = ncols;
    o.x = x;
    o.x_packed = x_packed;
    o.resid = ws.x;
    o.ld_resid = c.d_model;
    o.splitk_ws = ws.splitk;
    o.splitk_cap = ws.splitk_floats;
    return launch_gemm(c.dtype, PRO_PLAIN, EPI_RESID, o, st);
  }

  hipError_t oproj(int l) const {
    const hs_config &c = m->cfg;
    const int ko = c.n_heads * c.head_dim;
    if (!combine_fused())
      return residual(m->layers[l].wo, ko, ws.attn, gemm_x_packed(c.dtype, ncols, ko) ? 1 : 0, o_defer());
    GemmArgs o{};
    o.w[0] = m->layers[l].wo;
    o.rows[0] = c.d_model;
    o.K = c.n_heads * c.head_dim;
    o.ncols = ncols;
    o.part_o = ws.part_o;
    o.part_ml = ws.part_ml;
    o.n_split = n_split;
    o.head_dim = c.head_dim;
    o.n_heads = c.n_heads;
    o.resid = ws.x;
    o.ld_resid = c.d_model;
    return launch_gemm(c.dtype, PRO_COMBINE, EPI_RESID, o, st);
  }

  hipError_t gateup(int l, int pend) const {
    const hs_config &c = m->cfg;
    const hs_layer_weights &W = m->layers[l];
    GemmArgs u{};
    u.w[0] = W.w_gate;
    u.w[1] = W.w_up;
    u.rows[0] = u.rows[1] = c.ffn_dim;
    u.K = c.d_model;
    u.ncols = ncols;
    u.x = ws.x;
    u.gain = W.mlp_norm;
    u.h_work = ws.hnorm;
    u.eps = c.rms_eps;
    u.pend = (const double *)ws.splitk;
    u.pend_s = pend;
    u.out = ws.act;
    // in the layout the down projection reads
    u.out_packed = gemm_x_packed(c.dtype, ncols, c.ffn_dim) ? 1 : 0;
    u.ld_out = c.ffn_dim;
    return launch_gemm(c.dtype, PRO_NORM, EPI_SWIGLU, u, st);
  }

  hipError_t down(int l) const {
    const hs_config &c = m->cfg;
    return residual(m->layers[l].w_down, c.ffn_dim, ws.act, gemm_x_packed(c.dtype, ncols, c.ffn_dim) ? 1 : 0,
                    down_defer());
  }

  // final RMSNorm + LM head over ncols rows starting at x_rows (pend: as
  // for qkv, the rows being ws.x)
  hipError_t head(const float *x_rows, float *logits, int pend) const {
    const hs_config &c = m->cfg;
    GemmArgs g{};
    g.w[0] = m->w.lm_head;
    g.rows[0] = c.vocab;
    g.K = c.d_model;
    g.ncols = ncols;
    g.x = x_rows;
    g.gain = m->w.final_norm;
    g.h_work = ws.hnorm;
    g.eps = c.rms_eps;
    g.pend = (const double *)ws.splitk;
    g.pend_s = pend;
    g.out = logits;
    g.ld_out = c.vocab;
    return launch_gemm(c.dtype, PRO_NORM, EPI_STORE, g, st);
  }

  // every layer; the last down projection's partials (down_defer()) stay
  // pending for the caller
  int layers() const {
    for (int l = 0; l < m->cfg.n_layers; ++l) {
      HIP_TRY(qkv(l, l ? down_defer() : 0));
      HIP_TRY(attn(l));
      HIP_TRY(combine(l));
      HIP_TRY(oproj(l));
      HIP_TRY(gateup(l, o_defer()));
      HIP_TRY(down(l));
    }
    return HS_OK;
  }
};

// The decode pass of a handle (checks that every request can take a step).
// A decode step runs over the handle's active requests: every request of a
// contiguous cache (all must be prefilled), the ready requests of a pool.
int decode_step_args(hs_model *m, hs_kv *kv, hipStream_t st, Step *out, int *blocks_needed = nullptr) {
  const hs_config &c = m->cfg;
  const int B = kv->n_active;
  if (B <= 0) return fail(HS_E_STATE, "decode: no prefilled request");
  if (B > m->max_batch) return fail(HS_E_INVALID, "decode: batch %d exceeds max_batch %d", B, m->max_batch);
  int need = 0;
  for (int b : kv->act_host) {
    if (!kv->ready[b]) return fail(HS_E_STATE, "decode: request %d is not prefilled", b);
    if (kv->len[b] >= kv->cap[b]) return fail(HS_E_CAPACITY, "decode: request %d is full (%d positions)", b, kv->cap[b]);
    if (kv->pool) need += blocks_for(kv, kv->len[b] + 1) - kv->nblk[b];
  }
  if (kv->pool && need > kv->free_blocks)
    return fail(HS_E_CAPACITY, "decode: the pool has %d free blocks, the step needs %d", kv->free_blocks, need);
  if (blocks_needed) *blocks_needed = need;
  int S, ns;
  kv_split_policy(c, kv->pool, B, kv->max_cap, &S, &ns);
  if (ns > 1 && (int64_t)B * c.n_heads * ns > m->part_entries)
    return fail(HS_E_INVALID, "decode: attention workspace too small");
  *out = Step{m, kv, B, 0, PackedRows{}, kv->d_rope, B, S, ns, st, model_ws(m)};
  return HS_OK;
}

// Prefill of n requests (§5.4: the language prefill from the transferred
// embedding rows).  Their rows are packed request by request; the requests are
// taken in order, in passes of at most PACK_MAX requests whose rows fit the row
// workspaces, and each pass runs every layer once over all its rows.
int prefill_requests(hs_model *m, hs_kv *kv, int n, const int32_t *reqs, const void *emb, const int32_t *text_ids,
                     const int32_t *s_text, const int32_t *pos_thw, float *last_logits, int32_t *first_tokens,
                     hs_stream_t stream, const char *fn) {
  if (!kv_matches(kv, m)) return fail(HS_E_INVALID, "%s: model/handle mismatch", fn);
  if (!m->w.lm_head) return fail(HS_E_STATE, "%s: model has no LM head", fn);
  if (!first_tokens) return fail(HS_E_INVALID, "%s: first_token is NULL", fn);
  if (n <= 0 || n > kv->batch || !reqs || !s_text) return fail(HS_E_INVALID, "%s: bad request list", fn);
  const hs_config &c = m->cfg;
  int64_t total = 0, total_v = 0, total_t = 0, blocks = 0;
  std::vector<char> seen(kv->batch, 0);
  for (int i = 0; i < n; ++i) {
    const int req = reqs[i];
    if (req < 0 || req >= kv->batch) return fail(HS_E_INVALID, "%s: request %d out of range", fn, req);
    if (seen[req]) return fail(HS_E_INVALID, "%s: request %d listed twice", fn, req);
    seen[req] = 1;
    if (s_text[i] < 0) return fail(HS_E_INVALID, "%s: negative s_text", fn);
    if (kv->pool && kv->cap[req] == 0) return fail(HS_E_STATE, "%s: slot %d holds no admitted request", fn, req);
    const int s_ctx = kv->n_v[req] + s_text[i];
    if (s_ctx <= 0) return fail(HS_E_INVALID, "%s: empty context", fn);
    if (kv->ready[req] || kv->len[req] != 0) return fail(HS_E_STATE, "%s: request %d is not empty", fn, req);
    if (s_ctx > kv->cap[req])
      return fail(HS_E_CAPACITY, "%s: context %d exceeds capacity %d", fn, s_ctx, kv->cap[req]);
    total += s_ctx;
    total_v += kv->n_v[req];
    total_t += s_text[i];
    if (kv->pool) blocks += blocks_for(kv, s_ctx) - kv->nblk[req];
  }
  if (kv->pool && blocks > kv->free_blocks)
    return fail(HS_E_CAPACITY, "%s: the pool has %d free blocks, the contexts need %lld", fn, kv->free_blocks,
                (long long)blocks);
  if ((total_v > 0 && !emb) || (total_t > 0 && !text_ids))
    return fail(HS_E_INVALID, "%s: missing embedding rows or text ids", fn);
  if (((uintptr_t)emb) % 16) return fail(HS_E_INVALID, "%s: emb must be 16-byte aligned", fn);
  if (c.rope_kind == HS_ROPE_M3 && !pos_thw) return fail(HS_E_INVALID, "%s: M-RoPE needs pos_thw", fn);
  if (c.rope_kind == HS_ROPE_1D && pos_thw) return fail(HS_E_INVALID, "%s: 1-D RoPE takes no pos_thw", fn);
  if (total > INT32_MAX) return fail(HS_E_INVALID, "%s: too many rows", fn);
  hipStream_t st = (hipStream_t)stream;
  const int b = dtype_bytes(c.dtype);
  // without a caller logits buffer, a pass's logits go to the [max_batch][V] workspace
  const int max_np = last_logits ? PACK_MAX : std::min(PACK_MAX, m->max_batch);
  int64_t voff = 0, toff = 0, roff = 0;
  for (int i0 = 0; i0 < n;) {
    PackedRows pk{};
    int rows = 0;
    while (i0 + pk.n < n && pk.n < max_np) {
      const int k = i0 + pk.n, s_ctx = kv->n_v[reqs[k]] + s_text[k];
      if (pk.n > 0 && rows + s_ctx > m->rows) break;  // one request always fits (s_ctx <= max_ctx <= rows)
      pk.req[pk.n] = reqs[k];
      pk.cu[pk.n] = rows;
      rows += s_ctx;
      ++pk.n;
    }
    pk.cu[pk.n] = rows;
    const int qpt = attn_prefill_rows_per_tile(c.n_heads / c.n_kv_heads);
    for (int k = 0; k < pk.n; ++k) pk.tcu[k + 1] = pk.tcu[k] + (pk.cu[k + 1] - pk.cu[k] + qpt - 1) / qpt;
    HIP_TRY(launch_set_packed(m->pk_dev, pk, st));
    if (kv->pool) {  // blocks for the pass's contexts
      KvReserve r{};
      r.n = pk.n;
      for (int k = 0; k < pk.n; ++k) {
        r.req[k] = pk.req[k];
        r.target[k] = pk.cu[k + 1] - pk.cu[k];
      }
      HIP_TRY(launch_kv_reserve(kv_pool(kv), r, 0, st));
    }
    for (int k = 0; k < pk.n; ++k) {
      const int nv = kv->n_v[pk.req[k]], nt = s_text[i0 + k];
      HIP_TRY(launch_prefill_rows(c.dtype, (const char *)emb + voff * c.d_model * b, nv, m->w.embed, c.vocab,
                                  c.d_model, text_ids ? text_ids + toff : nullptr, nt, m->x + (int64_t)pk.cu[k] * c.d_model,
                                  m->status, st));
      voff += nv;
      toff += nt;
    }
    // every row is its own query over the rows before it in its request; no
    // splits (S covers the longest request)
    Step pre{m, kv, rows, 1, pk, pos_thw ? pos_thw + roff : nullptr, (int)total, rows, 1, st, model_ws(m)};
    const int rc = pre.layers();
    if (rc) return rc;
    HIP_TRY(launch_gather_last(m->x, c.d_model, pk, m->xlast, st));
    float *lg = last_logits ? last_logits + (int64_t)i0 * c.vocab : m->logits;
    Step last = pre;
    last.ncols = pk.n;
    HIP_TRY(last.head(m->xlast, lg, 0));
    HIP_TRY(launch_argmax(lg, c.vocab, c.vocab, pk.n, first_tokens + i0, nullptr, nullptr, nullptr, 0, st));
    for (int k = 0; k < pk.n; ++k)
      HIP_TRY(launch_prefill_finish(kv->d_len, kv->d_rope, kv->d_ready, pk.req[k], pk.cu[k + 1] - pk.cu[k],
                                    pos_thw ? pos_thw + roff + pk.cu[k] : nullptr, (int)total, st));
    for (int k = 0; k < pk.n; ++k) {
      const int req = pk.req[k], s_ctx = pk.cu[k + 1] - pk.cu[k];
      kv->len[req] = s_ctx;
      kv->ready[req] = 1;
      if (kv->pool) {
        kv->free_blocks -= blocks_for(kv, s_ctx) - kv->nblk[req];
        kv->nblk[req] = blocks_for(kv, s_ctx);
      }
    }
    roff += rows;
    i0 += pk.n;
  }
  HIP_TRY(kv->pool ? rebuild_active(kv, st) : rebuild_order(kv, st));
  return HS_OK;
}

}  // namespace

extern "C" {

const char *hs_last_error(void) { return g_err.c_str(); }

int hs_kv_bytes(const hs_config *cfg, int64_t n_v, int64_t s_text, uint64_t *kv_bytes, uint64_t *emb_bytes) {
  if (!shape_ok(cfg)) return fail(HS_E_INVALID, "hs_kv_bytes: bad config");
  if (n_v < 0 || s_text < 0) return fail(HS_E_INVALID, "hs_kv_bytes: negative length");
  const uint64_t factors[] = {2, (uint64_t)cfg->n_layers, (uint64_t)cfg->n_kv_heads, (uint64_t)cfg->head_dim,
                              (uint64_t)n_v + (uint64_t)s_text, (uint64_t)dtype_bytes(cfg->dtype)};
  uint64_t kv = 1, emb = 0;
  for (uint64_t f : factors)
    if (__builtin_mul_overflow(kv, f, &kv)) return fail(HS_E_INVALID, "hs_kv_bytes: size overflows 64 bits");
  if (__builtin_mul_overflow((uint64_t)n_v, (uint64_t)cfg->d_model, &emb) ||
      __builtin_mul_overflow(emb, (uint64_t)dtype_bytes(cfg->dtype), &emb))
    return fail(HS_E_INVALID, "hs_kv_bytes: size overflows 64 bits");
  if (kv_bytes) *kv_bytes = kv;
  if (emb_bytes) *emb_bytes = emb;
  return HS_OK;
}

int hs_packed_bytes(int32_t dtype, int64_t rows, int64_t cols, uint64_t *bytes) {
  if (!bytes || dtype < HS_F32 || dtype > HS_BF16 || rows <= 0 || cols <= 0)
    return fail(HS_E_INVALID, "hs_packed_bytes: bad argument");
  if (cols % (16 / dtype_bytes(dtype))) return fail(HS_E_INVALID, "hs_packed_bytes: cols must fill 16-byte chunks");
  *bytes = (uint64_t)packed_elems(dtype, rows, cols) * dtype_bytes(dtype);
  return HS_OK;
}

int hs_pack_matrix(int32_t dtype, const void *src, int64_t rows, int64_t cols, void *dst, hs_stream_t stream) {
  uint64_t bytes;
  int rc = hs_packed_bytes(dtype, rows, cols, &bytes);
  if (rc) return rc;
  if (!src || !dst || ((uintptr_t)src | (uintptr_t)dst) % 16)
    return fail(HS_E_INVALID, "hs_pack_matrix: NULL or misaligned pointer");
  if (cols > INT32_MAX) return fail(HS_E_INVALID, "hs_pack_matrix: cols too large");
  HIP_TRY(launch_pack(dtype, src, rows, cols, dst, 0, (hipStream_t)stream));
  return HS_OK;
}

int hs_pack_matrix_heads(int32_t dtype, const void *src, int64_t rows, int64_t cols, int32_t head_dim, void *dst,
                         hs_stream_t stream) {
  uint64_t bytes;
  int rc = hs_packed_bytes(dtype, rows, cols, &bytes);
  if (rc) return rc;
  if (!src || !dst || ((uintptr_t)src | (uintptr_t)dst) % 16)
    return fail(HS_E_INVALID, "hs_pack_matrix_heads: NULL or misaligned pointer");
  if (cols > INT32_MAX) return fail(HS_E_INVALID, "hs_pack_matrix_heads: cols too large");
  if (head_dim <= 0 || head_dim % 16 || rows % head_dim)
    return fail(HS_E_INVALID, "hs_pack_matrix_heads: head_dim %d must be a positive multiple of 16 dividing rows",
                head_dim);
  HIP_TRY(launch_pack(dtype, src, rows, cols, dst, head_dim, (hipStream_t)stream));
  return HS_OK;
}

int hs_model_create(const hs_config *cfg, const hs_weights *w, int32_t max_batch, int32_t max_ctx, hs_model **out) {
  if (!out) return fail(HS_E_INVALID, "hs_model_create: out is NULL");
  *out = nullptr;
  int rc = check_config(cfg);
  if (rc) return rc;
  if (!w || !w->embed || !w->layers) return fail(HS_E_INVALID, "hs_model_create: missing embed/layers");
  if (((uintptr_t)w->embed | (uintptr_t)w->lm_head) % 16)
    return fail(HS_E_INVALID, "hs_model_create: embed and lm_head must be 16-byte aligned");
  if (w->lm_head && !w->final_norm) return fail(HS_E_INVALID, "hs_model_create: lm_head without final_norm");
  if (max_batch <= 0 || max_ctx <= 0) return fail(HS_E_INVALID, "hs_model_create: max_batch/max_ctx must be > 0");
  for (int l = 0; l < cfg->n_layers; ++l) {
    const hs_layer_weights &L = w->layers[l];
    if (!L.attn_norm || !L.wq || !L.wk || !L.wv || !L.wo || !L.mlp_norm || !L.w_gate || !L.w_up || !L.w_down)
      return fail(HS_E_INVALID, "hs_model_create: layer %d has a NULL weight", l);
    if (cfg->qkv_bias && (!L.bq || !L.bk || !L.bv))
      return fail(HS_E_INVALID, "hs_model_create: layer %d lacks q/k/v bias", l);
  }
  hs_model *m = new (std::nothrow) hs_model();
  if (!m) return fail(HS_E_DEVICE, "hs_model_create: out of host memory");
  m->cfg = *cfg;
  m->w = *w;
  m->layers.assign(w->layers, w->layers + cfg->n_layers);
  m->w.layers = m->layers.data();
  m->max_batch = max_batch;
  m->max_ctx = max_ctx;
  if (hipGetDevice(&m->device) != hipSuccess) {
    free_model(m);
    return fail(HS_E_DEVICE, "hs_model_create: no HIP device");
  }
  const hs_config &c = *cfg;
  const int b = dtype_bytes(c.dtype), hd = c.head_dim, nh = c.n_heads;
  const int64_t rows = std::max(max_batch, max_ctx);
  m->rows = rows;

  // attention partial capacity: the largest (queries x heads x splits) any
  // decode batch <= max_batch with capacities <= max_ctx, or any prefill of
  // <= max_ctx rows, can ask for
  int64_t entries = 0;
  const int group = c.n_heads / c.n_kv_heads;
  for (int nq = 1; nq <= max_batch; ++nq) {
    int S, ns;
    for (int len = 1; len <= max_ctx; len += std::max(1, len / 64)) {
      split_policy(nq, c.n_kv_heads, group, hd, c.dtype, len, &S, &ns);
      if (ns > 1) entries = std::max(entries, (int64_t)nq * nh * ns);
    }
    split_policy(nq, c.n_kv_heads, group, hd, c.dtype, max_ctx, &S, &ns);
    if (ns > 1) entries = std::max(entries, (int64_t)nq * nh * ns);
  }
  m->part_entries = entries;
  m->splitk_floats = (int64_t)SPLITK_MAX * max_batch * std::max(c.d_model, (c.n_heads + 2 * c.n_kv_heads) * c.head_dim);

  struct Alloc {
    void **p;
    size_t bytes;
  } allocs[] = {
      {(void **)&m->x, (size_t)rows * c.d_model * 4},
      {&m->q, (size_t)rows * nh * hd * b},
      {&m->attn, (size_t)act_elems(rows, nh * hd) * b},
      {&m->act, (size_t)act_elems(rows, c.ffn_dim) * b},
      {&m->hnorm, (size_t)act_elems(rows, c.d_model) * b},
      {(void **)&m->splitk, (size_t)m->splitk_floats * 4},
      {(void **)&m->xlast, (size_t)PACK_MAX * c.d_model * 4},
      {(void **)&m->pk_dev, sizeof(PackedRows)},
      {(void **)&m->logits, w->lm_head ? (size_t)max_batch * c.vocab * 4 : 0},
      {(void **)&m->part_o, (size_t)std::max<int64_t>(entries, 1) * hd * 4},
      {(void **)&m->part_ml, (size_t)std::max<int64_t>(entries, 1) * 2 * 4},
      {(void **)&m->rope_tab, (size_t)max_ctx * (hd / 2) * 2 * 4},
      {(void **)&m->status, 4},
  };
  for (auto &a : allocs) {
    if (!a.bytes) continue;
    if (hipMalloc(a.p, a.bytes) != hipSuccess) {
      free_model(m);
      return fail(HS_E_DEVICE, "hs_model_create: hipMalloc of %zu bytes failed", a.bytes);
    }
  }
  // RoPE table: pair i at position p turns by p * theta^(-2i/d_h); angle and
  // cos/sin in fp64, stored as fp32
  std::vector<float> tab((size_t)max_ctx * (hd / 2) * 2);
  for (int p = 0; p < max_ctx; ++p)
    for (int i = 0; i < hd / 2; ++i) {
      const double inv = std::pow((double)c.rope_theta, -(double)(2 * i) / (double)hd);
      const double ang = (double)p * inv;
      tab[((size_t)p * (hd / 2) + i) * 2] = (float)std::cos(ang);
      tab[((size_t)p * (hd / 2) + i) * 2 + 1] = (float)std::sin(ang);
    }
  // activations read in the packed layout are read in whole k-blocks of 128,
  // past K against zero weight rows: those elements must hold finite values
  // (they are never written, so cleared once here)
  if (hipMemcpy(m->rope_tab, tab.data(), tab.size() * 4, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemset(m->status, 0, 4) != hipSuccess || hipMemset(m->attn, 0, (size_t)act_elems(rows, nh * hd) * b) ||
      hipMemset(m->act, 0, (size_t)act_elems(rows, c.ffn_dim) * b) ||
      hipMemset(m->hnorm, 0, (size_t)act_elems(rows, c.d_model) * b)) {
    free_model(m);
    return fail(HS_E_DEVICE, "hs_model_create: initial copies failed");
  }
  *out = m;
  return HS_OK;
}

int hs_model_free(hs_model *m) {
  if (!m) return fail(HS_E_INVALID, "hs_model_free: NULL");
  free_model(m);
  return HS_OK;
}

int hs_model_status(hs_model *m, int32_t *flags) {
  if (!m || !flags) return fail(HS_E_INVALID, "hs_model_status: NULL argument");
  HIP_TRY(hipDeviceSynchronize());
  HIP_TRY(hipMemcpy(flags, m->status, 4, hipMemcpyDeviceToHost));
  HIP_TRY(hipMemset(m->status, 0, 4));
  return HS_OK;
}

int hs_kv_alloc(hs_model *m, int32_t batch, const int32_t *n_v, const int32_t *capacity, void *dev_buf,
                uint64_t buf_bytes, hs_kv **out) {
  if (!out) return fail(HS_E_INVALID, "hs_kv_alloc: out is NULL");
  *out = nullptr;
  if (!m || !n_v || !capacity || !dev_buf) return fail(HS_E_INVALID, "hs_kv_alloc: NULL argument");
  if (batch <= 0) return fail(HS_E_INVALID, "hs_kv_alloc: batch must be > 0");
  const hs_config &c = m->cfg;
  const int b = dtype_bytes(c.dtype);
  uint64_t total = 0;
  for (int i = 0; i < batch; ++i) {
    if (n_v[i] < 0 || capacity[i] <= 0 || n_v[i] > capacity[i] || capacity[i] > m->max_ctx)
      return fail(HS_E_INVALID, "hs_kv_alloc: request %d has n_v %d, capacity %d (max_ctx %d)", i, n_v[i],
                  capacity[i], m->max_ctx);
    total += (uint64_t)kv_request_elems(c, capacity[i]) * b;
  }
  if (buf_bytes < total)
    return fail(HS_E_BUFFER, "hs_kv_alloc: buffer holds %llu bytes, layout needs %llu",
                (unsigned long long)buf_bytes, (unsigned long long)total);
  if (((uintptr_t)dev_buf) % 16) return fail(HS_E_INVALID, "hs_kv_alloc: buffer must be 16-byte aligned");
  hs_kv *kv = new (std::nothrow) hs_kv();
  if (!kv) return fail(HS_E_DEVICE, "hs_kv_alloc: out of host memory");
  kv->m = m;
  kv->batch = batch;
  kv->buf = dev_buf;
  kv->buf_bytes = buf_bytes;
  kv->n_v.assign(n_v, n_v + batch);
  kv->cap.assign(capacity, capacity + batch);
  kv->len.assign(batch, 0);
  kv->rope.assign(batch, 0);
  kv->ready.assign(batch, 0);
  kv->base.resize(batch);
  int64_t off = 0;
  for (int i = 0; i < batch; ++i) {
    kv->base[i] = off;
    off += kv_request_elems(c, capacity[i]);
    kv->max_cap = std::max(kv->max_cap, capacity[i]);
  }
  // one block per request: the block table is the base offsets, the block
  // size the capacity; every request is a decode column
  std::vector<int> ident(batch);
  for (int i = 0; i < batch; ++i) ident[i] = i;
  kv->ntab = batch;
  kv->n_active = batch;
  kv->act_host = ident;
  bool ok = hipMalloc(&kv->d_base, batch * 8) == hipSuccess && hipMalloc(&kv->d_cap, batch * 4) == hipSuccess &&
            hipMalloc(&kv->d_len, batch * 4) == hipSuccess && hipMalloc(&kv->d_rope, batch * 4) == hipSuccess &&
            hipMalloc(&kv->d_toff, batch * 4) == hipSuccess && hipMalloc(&kv->d_act, batch * 4) == hipSuccess &&
            hipMalloc(&kv->d_ready, batch * 4) == hipSuccess && hipMalloc(&kv->d_order, batch * 4) == hipSuccess;
  ok = ok && hipMemcpy(kv->d_base, kv->base.data(), batch * 8, hipMemcpyHostToDevice) == hipSuccess &&
       hipMemcpy(kv->d_cap, kv->cap.data(), batch * 4, hipMemcpyHostToDevice) == hipSuccess &&
       hipMemcpy(kv->d_toff, ident.data(), batch * 4, hipMemcpyHostToDevice) == hipSuccess &&
       hipMemcpy(kv->d_act, ident.data(), batch * 4, hipMemcpyHostToDevice) == hipSuccess &&
       hipMemcpy(kv->d_order, ident.data(), batch * 4, hipMemcpyHostToDevice) == hipSuccess &&
       hipMemset(kv->d_len, 0, batch * 4) == hipSuccess && hipMemset(kv->d_rope, 0, batch * 4) == hipSuccess &&
       hipMemset(kv->d_ready, 0, batch * 4) == hipSuccess;
  kv->d_bt = kv->d_cap;
  if (!ok) {
    hs_kv_free(kv);
    return fail(HS_E_DEVICE, "hs_kv_alloc: metadata allocation failed");
  }
  *out = kv;
  return HS_OK;
}

int hs_kv_free(hs_kv *kv) {
  if (!kv) return fail(HS_E_INVALID, "hs_kv_free: NULL");
  void *ptrs[] = {kv->d_base,  kv->d_cap,   kv->d_len,  kv->d_rope, kv->d_toff, kv->d_act, kv->d_order,
                  kv->d_ready, kv->d_stack, kv->d_top, kv->d_nblk, kv->d_bt == kv->d_cap ? nullptr : kv->d_bt};
  for (void *p : ptrs)
    if (p) (void)hipFree(p);
  delete kv;
  return HS_OK;
}

int hs_kv_pool_create(hs_model *m, int32_t slots, int32_t block_tokens, void *dev_buf, uint64_t buf_bytes,
                      hs_kv **out) {
  if (!out) return fail(HS_E_INVALID, "hs_kv_pool_create: out is NULL");
  *out = nullptr;
  if (!m || !dev_buf) return fail(HS_E_INVALID, "hs_kv_pool_create: NULL argument");
  const hs_config &c = m->cfg;
  if (c.dtype == HS_F32) return fail(HS_E_INVALID, "hs_kv_pool_create: pooled caches take 16-bit storage");
  if (slots <= 0 || slots > 4096) return fail(HS_E_INVALID, "hs_kv_pool_create: slots must be in 1..4096");
  if (block_tokens < POOL_SPAN || block_tokens > 16384 || (block_tokens & (block_tokens - 1)))
    return fail(HS_E_INVALID, "hs_kv_pool_create: block_tokens must be a power of two in 256..16384");
  if (((uintptr_t)dev_buf) % 16) return fail(HS_E_INVALID, "hs_kv_pool_create: buffer must be 16-byte aligned");
  const int64_t block_elems = kv_request_elems(c, block_tokens);
  const uint64_t block_bytes = (uint64_t)block_elems * dtype_bytes(c.dtype);
  const uint64_t n_blocks = buf_bytes / block_bytes;
  if (n_blocks < 1 || n_blocks > (1u << 30))
    return fail(HS_E_BUFFER, "hs_kv_pool_create: buffer holds %llu blocks of %llu bytes",
                (unsigned long long)n_blocks, (unsigned long long)block_bytes);
  // attention partials for the block-aligned splits: a pooled split is the
  // unpooled one rounded up to whole POOL_SPANs, so it never needs more
  // partials than hs_model_create sized for (and nothing here reallocates a
  // workspace that a captured decode graph may hold)
  for (int nq = 1; nq <= std::min(slots, m->max_batch); ++nq) {
    int S, ns;
    kv_split_policy(c, true, nq, m->max_ctx, &S, &ns);
    if (ns > 1 && (int64_t)nq * c.n_heads * ns > m->part_entries)
      return fail(HS_E_INVALID, "hs_kv_pool_create: %d queries x %d splits exceed the model's attention workspace",
                  nq, ns);
  }
  hs_kv *kv = new (std::nothrow) hs_kv();
  if (!kv) return fail(HS_E_DEVICE, "hs_kv_pool_create: out of host memory");
  kv->m = m;
  kv->batch = slots;
  kv->buf = dev_buf;
  kv->buf_bytes = buf_bytes;
  kv->pool = true;
  kv->block_tokens = block_tokens;
  kv->block_elems = block_elems;
  kv->n_blocks = (int)n_blocks;
  kv->free_blocks = (int)n_blocks;
  kv->max_blocks = (m->max_ctx + block_tokens - 1) / block_tokens;
  kv->ntab = slots * kv->max_blocks;
  kv->n_v.assign(slots, 0);
  kv->cap.assign(slots, 0);
  kv->len.assign(slots, 0);
  kv->rope.assign(slots, 0);
  kv->ready.assign(slots, 0);
  kv->nblk.assign(slots, 0);
  kv->n_active = 0;
  std::vector<int64_t> tab(kv->ntab, -1);
  std::vector<int> toff(slots), bt(slots, block_tokens), stack(n_blocks);
  for (int i = 0; i < slots; ++i) toff[i] = i * kv->max_blocks;
  for (uint64_t i = 0; i < n_blocks; ++i) stack[i] = (int)i;
  const int top = (int)n_blocks;
  const size_t sb = (size_t)slots * 4;
  bool ok = hipMalloc(&kv->d_base, (size_t)kv->ntab * 8) == hipSuccess && hipMalloc(&kv->d_cap, sb) == hipSuccess &&
            hipMalloc(&kv->d_len, sb) == hipSuccess && hipMalloc(&kv->d_rope, sb) == hipSuccess &&
            hipMalloc(&kv->d_toff, sb) == hipSuccess && hipMalloc(&kv->d_bt, sb) == hipSuccess &&
            hipMalloc(&kv->d_act, sb) == hipSuccess && hipMalloc(&kv->d_ready, sb) == hipSuccess &&
            hipMalloc(&kv->d_order, sb) == hipSuccess &&
            hipMalloc(&kv->d_nblk, sb) == hipSuccess && hipMalloc(&kv->d_stack, n_blocks * 4) == hipSuccess &&
            hipMalloc(&kv->d_top, 4) == hipSuccess;
  ok = ok && hipMemcpy(kv->d_base, tab.data(), (size_t)kv->ntab * 8, hipMemcpyHostToDevice) == hipSuccess &&
       hipMemcpy(kv->d_toff, toff.data(), sb, hipMemcpyHostToDevice) == hipSuccess &&
       hipMemcpy(kv->d_bt, bt.data(), sb, hipMemcpyHostToDevice) == hipSuccess &&
       hipMemcpy(kv->d_stack, stack.data(), n_blocks * 4, hipMemcpyHostToDevice) == hipSuccess &&
       hipMemcpy(kv->d_top, &top, 4, hipMemcpyHostToDevice) == hipSuccess &&
       hipMemset(kv->d_cap, 0, sb) == hipSuccess && hipMemset(kv->d_len, 0, sb) == hipSuccess &&
       hipMemset(kv->d_rope, 0, sb) == hipSuccess && hipMemset(kv->d_act, 0, sb) == hipSuccess &&
       hipMemset(kv->d_order, 0, sb) == hipSuccess &&
       hipMemset(kv->d_ready, 0, sb) == hipSuccess && hipMemset(kv->d_nblk, 0, sb) == hipSuccess;
  if (!ok) {
    hs_kv_free(kv);
    return fail(HS_E_DEVICE, "hs_kv_pool_create: metadata allocation failed");
  }
  *out = kv;
  return HS_OK;
}

int hs_kv_admit(hs_kv *kv, int32_t slot, int32_t n_v, int32_t capacity, hs_stream_t stream) {
  if (!kv || !kv->pool) return fail(HS_E_INVALID, "hs_kv_admit: not a pooled cache");
  if (slot < 0 || slot >= kv->batch) return fail(HS_E_INVALID, "hs_kv_admit: slot %d out of range", slot);
  if (kv->cap[slot] != 0) return fail(HS_E_STATE, "hs_kv_admit: slot %d is in use", slot);
  if (n_v < 0 || capacity <= 0 || n_v > capacity || capacity > kv->m->max_ctx)
    return fail(HS_E_INVALID, "hs_kv_admit: n_v %d, capacity %d (max_ctx %d)", n_v, capacity, kv->m->max_ctx);
  HIP_TRY(launch_set_int(kv->d_cap + slot, capacity, (hipStream_t)stream));
  kv->n_v[slot] = n_v;
  kv->cap[slot] = capacity;
  kv->max_cap = std::max(kv->max_cap, capacity);
  return HS_OK;
}

int hs_kv_release(hs_kv *kv, int32_t slot, hs_stream_t stream) {
  if (!kv || !kv->pool) return fail(HS_E_INVALID, "hs_kv_release: not a pooled cache");
  if (slot < 0 || slot >= kv->batch) return fail(HS_E_INVALID, "hs_kv_release: slot %d out of range", slot);
  if (kv->cap[slot] == 0) return fail(HS_E_STATE, "hs_kv_release: slot %d is empty", slot);
  hipStream_t st = (hipStream_t)stream;
  HIP_TRY(launch_kv_release(kv_pool(kv), slot, st));
  HIP_TRY(launch_set_int(kv->d_cap + slot, 0, st));
  const bool was_ready = kv->ready[slot];
  kv->free_blocks += kv->nblk[slot];
  kv->nblk[slot] = 0;
  kv->n_v[slot] = kv->cap[slot] = kv->len[slot] = kv->rope[slot] = 0;
  kv->ready[slot] = 0;
  if (was_ready) HIP_TRY(rebuild_active(kv, st));
  return HS_OK;
}

int hs_stream_read(const void *buf, uint64_t bytes, uint32_t *sink, int32_t blocks, hs_stream_t stream) {
  if (!buf || !sink || blocks <= 0 || bytes == 0 || bytes % 16 || ((uintptr_t)buf) % 16)
    return fail(HS_E_INVALID, "hs_stream_read: bad argument");
  HIP_TRY(launch_stream_read(buf, bytes, sink, blocks, (hipStream_t)stream));
  return HS_OK;
}

int hs_kv_pool_blocks(const hs_kv *kv, int32_t *free_blocks, int32_t *n_blocks) {
  if (!kv || !kv->pool) return fail(HS_E_INVALID, "hs_kv_pool_blocks: not a pooled cache");
  if (free_blocks) *free_blocks = kv->free_blocks;
  if (n_blocks) *n_blocks = kv->n_blocks;
  return HS_OK;
}

int hs_prefill_embeddings(hs_model *m, hs_kv *kv, int32_t req, const void *emb, const int32_t *text_ids,
                          int32_t s_text, const int32_t *pos_thw, float *last_logits, int32_t *first_token,
                          hs_stream_t stream) {
  return prefill_requests(m, kv, 1, &req, emb, text_ids, &s_text, pos_thw, last_logits, first_token, stream,
                          "hs_prefill_embeddings");
}

int hs_prefill_batch(hs_model *m, hs_kv *kv, int32_t n, const int32_t *reqs, const void *emb,
                     const int32_t *text_ids, const int32_t *s_text, const int32_t *pos_thw, float *last_logits,
                     int32_t *first_tokens, hs_stream_t stream) {
  return prefill_requests(m, kv, n, reqs, emb, text_ids, s_text, pos_thw, last_logits, first_tokens, stream,
                          "hs_prefill_batch");
}

int hs_model_reserve_rows(hs_model *m, int64_t rows) {
  if (!m) return fail(HS_E_INVALID, "hs_model_reserve_rows: model is NULL");
  if (rows <= 0 || rows > (1 << 24)) return fail(HS_E_INVALID, "hs_model_reserve_rows: rows %lld out of range", (long long)rows);
  if (rows <= m->rows) return HS_OK;
  const hs_config &c = m->cfg;
  const int b = dtype_bytes(c.dtype), nhd = c.n_heads * c.head_dim;
  void *fresh[5] = {nullptr, nullptr, nullptr, nullptr, nullptr};
  const size_t bytes[5] = {(size_t)rows * c.d_model * 4, (size_t)rows * nhd * b, (size_t)act_elems(rows, nhd) * b,
                           (size_t)act_elems(rows, c.ffn_dim) * b, (size_t)act_elems(rows, c.d_model) * b};
  for (int i = 0; i < 5; ++i)
    if (hipMalloc(&fresh[i], bytes[i]) != hipSuccess) {
      for (void *p : fresh)
        if (p) (void)hipFree(p);
      return fail(HS_E_DEVICE, "hs_model_reserve_rows: hipMalloc of %zu bytes failed", bytes[i]);
    }
  // the old buffers may still be in use by queued work; the packed-layout
  // activations start cleared (as in hs_model_create)
  if (hipDeviceSynchronize() != hipSuccess || hipMemset(fresh[2], 0, bytes[2]) != hipSuccess ||
      hipMemset(fresh[3], 0, bytes[3]) != hipSuccess || hipMemset(fresh[4], 0, bytes[4]) != hipSuccess) {
    for (void *p : fresh) (void)hipFree(p);
    return fail(HS_E_DEVICE, "hs_model_reserve_rows: device synchronisation failed");
  }
  void **slots[5] = {(void **)&m->x, &m->q, &m->attn, &m->act, &m->hnorm};
  for (int i = 0; i < 5; ++i) {
    (void)hipFree(*slots[i]);
    *slots[i] = fresh[i];
  }
  m->rows = rows;
  return HS_OK;
}

// One decode step (hs_decode_step); ovr, when given, replaces the model's
// workspaces as the step's scratch.
static int decode_impl(hs_model *m, hs_kv *kv, const int32_t *tokens_in, int32_t *tokens_out, float *logits,
                       float *hidden_out, hs_stream_t stream, const StepWs *ovr, const char *fn) {
  if (!kv_matches(kv, m)) return fail(HS_E_INVALID, "%s: model/handle mismatch", fn);
  if (!tokens_in) return fail(HS_E_INVALID, "%s: tokens_in is NULL", fn);
  const hs_config &c = m->cfg;
  if (m->w.lm_head) {
    if (!tokens_out) return fail(HS_E_INVALID, "%s: tokens_out is NULL", fn);
    if (tokens_out == tokens_in) return fail(HS_E_INVALID, "%s: tokens_out aliases tokens_in", fn);
  } else if (logits) {
    return fail(HS_E_INVALID, "%s: model has no LM head, logits must be NULL", fn);
  }
  hipStream_t st = (hipStream_t)stream;
  Step step;
  int need = 0;
  int rc = decode_step_args(m, kv, st, &step, &need);
  if (rc) return rc;
  if (ovr) step.ws = *ovr;
  const int B = kv->n_active;
  // a pooled request entering a new block takes it now, on the device
  if (kv->pool) HIP_TRY(launch_kv_reserve(kv_pool(kv), KvReserve{}, B, st));
  const int *act = kv->pool ? kv->d_act : nullptr;  // a contiguous cache decodes request c in column c
  HIP_TRY(launch_embed(c.dtype, m->w.embed, c.vocab, c.d_model, tokens_in, act, B, step.ws.x, m->status, st));
  rc = step.layers();
  if (rc) return rc;
  // the last down projection's pending partials: added by the final norm,
  // else here
  const int pend = step.down_defer();
  if (m->w.lm_head) {
    float *lg = logits ? logits : step.ws.logits;
    HIP_TRY(step.head(step.ws.x, lg, pend));
    HIP_TRY(launch_argmax(lg, c.vocab, c.vocab, B, tokens_out, act, kv->d_len, kv->d_rope, 1, st));
  } else {
    if (pend) HIP_TRY(launch_resid_pending((const double *)step.ws.splitk, pend, B, c.d_model, step.ws.x, st));
    HIP_TRY(launch_advance(kv->d_len, kv->d_rope, act, B, st));
  }
  if (hidden_out)
    HIP_TRY(hipMemcpyAsync(hidden_out, step.ws.x, (size_t)B * c.d_model * 4, hipMemcpyDeviceToDevice, st));
  for (int b : kv->act_host) {
    if (kv->pool) {
      const int k = blocks_for(kv, kv->len[b] + 1) - kv->nblk[b];
      kv->nblk[b] += k;
      kv->free_blocks -= k;
    }
    kv->len[b] += 1;
  }
  return HS_OK;
}

int hs_decode_step(hs_model *m, hs_kv *kv, const int32_t *tokens_in, int32_t *tokens_out, float *logits,
                   float *hidden_out, hs_stream_t stream) {
  return decode_impl(m, kv, tokens_in, tokens_out, logits, hidden_out, stream, nullptr, "hs_decode_step");
}

// ---- the decode step with its scratch in a static device array ----
//
// scratch is a file-scope device array; every GPU the library runs on holds
// its own copy until the process ends.  In host code its name is a stand-in,
// not a device address: each device's address is looked up once, with that
// device current, and only that address is handed to kernels and copies.
static __device__ __align__(256) unsigned char scratch[HS_STATIC_SCRATCH_BYTES];

namespace {
constexpr int SCRATCH_MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[SCRATCH_MAX_DEVICES] = {};

// the current device's copy of the scratch array (looked up once per device)
int scratch_ptr(int dev, void **out) {
  if (dev < 0 || dev >= SCRATCH_MAX_DEVICES) return fail(HS_E_INVALID, "hs_decode_step_static: device %d", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(HS_E_DEVICE, "hs_decode_step_static: hipGetSymbolAddress: %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return HS_OK;
}
}  // namespace

extern "C" int hs_decode_step_static(hs_model *m, hs_kv *kv, const int32_t *tokens_in, int32_t *tokens_out,
                                     float *logits, float *hidden_out, hs_stream_t stream) {
  static const char *fn = "hs_decode_step_static";
  if (!kv_matches(kv, m)) return fail(HS_E_INVALID, "%s: model/handle mismatch", fn);
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return fail(HS_E_DEVICE, "%s: no current device", fn);
  if (dev != m->device) return fail(HS_E_INVALID, "%s: the current device %d is not the model's (%d)", fn, dev,
                                    m->device);
  const hs_config &c = m->cfg;
  const int B = kv->n_active;
  if (B <= 0) return fail(HS_E_STATE, "%s: no prefilled request", fn);
  int S, ns;
  kv_split_policy(c, kv->pool, B, kv->max_cap, &S, &ns);
  // the step's scratch, carved in 256-byte aligned pieces
  const int64_t b = dtype_bytes(c.dtype), nhd = (int64_t)c.n_heads * c.head_dim;
  const int64_t qkv_rows = (int64_t)(c.n_heads + 2 * c.n_kv_heads) * c.head_dim;
  const int64_t splitk_floats = (int64_t)SPLITK_MAX * B * std::max<int64_t>(c.d_model, qkv_rows);
  const int64_t entries = ns > 1 ? (int64_t)B * c.n_heads * ns : 1;
  const uint64_t sizes[10] = {(uint64_t)B * c.d_model * 4,
                              (uint64_t)(B * nhd * b),
                              (uint64_t)(act_elems(B, nhd) * b),
                              (uint64_t)(act_elems(B, c.ffn_dim) * b),
                              (uint64_t)(act_elems(B, c.d_model) * b),
                              (uint64_t)splitk_floats * 4,
                              (uint64_t)entries * c.head_dim * 4,
                              (uint64_t)entries * 2 * 4,
                              (m->w.lm_head && !logits) ? (uint64_t)B * c.vocab * 4 : 0u,
                              0u};
  uint64_t offs[10], total = 0;
  for (int i = 0; i < 10; ++i) {
    offs[i] = total;
    total += (sizes[i] + 255) / 256 * 256;
  }
  if (total > HS_STATIC_SCRATCH_BYTES)
    return fail(HS_E_INVALID, "%s: this step needs %llu bytes of scratch, the static array holds %llu", fn,
                (unsigned long long)total, (unsigned long long)HS_STATIC_SCRATCH_BYTES);
  void *base = nullptr;
  int rc = scratch_ptr(dev, &base);
  if (rc) return rc;
  char *p = (char *)base;
  StepWs ws{(float *)(p + offs[0]), p + offs[1], p + offs[2], p + offs[3], p + offs[4], (float *)(p + offs[5]),
            splitk_floats, (float *)(p + offs[6]), (float *)(p + offs[7]),
            sizes[8] ? (float *)(p + offs[8]) : nullptr};
  // The array keeps whatever the last call left.  The activations read in the
  // packed layout are read in whole k-blocks of 128 elements, past K up to
  // the block's end, against weight rows that are zero there: those elements
  // must hold finite values, so a K that is not a multiple of 128 has its
  // buffer cleared first.  Everything else a step reads it writes first.
  hipStream_t st = (hipStream_t)stream;
  const int64_t ks[3] = {nhd, c.ffn_dim, c.d_model};
  void *bufs[3] = {ws.attn, ws.act, ws.hnorm};
  for (int i = 0; i < 3; ++i)
    if (ks[i] % 128 && gemm_x_packed(c.dtype, B, (int)ks[i]))
      HIP_TRY(launch_zero(bufs[i], sizes[2 + i], st));
  return decode_impl(m, kv, tokens_in, tokens_out, logits, hidden_out, stream, &ws, fn);
}

int hs_replay_kernels(hs_model *m, hs_kv *kv, int32_t kind, int32_t count, hs_stream_t stream) {
  if (!kv_matches(kv, m)) return fail(HS_E_INVALID, "hs_replay_kernels: model/handle mismatch");
  if (count < 0) return fail(HS_E_INVALID, "hs_replay_kernels: negative count");
  hipStream_t st = (hipStream_t)stream;
  Step step;
  int rc = decode_step_args(m, kv, st, &step);
  if (rc) return rc;
  const int L = m->cfg.n_layers;
  if (kind == HS_K_HEAD && !m->w.lm_head) return fail(HS_E_STATE, "hs_replay_kernels: model has no LM head");
  if (kind == HS_K_COMBINE && step.n_split <= 1)
    return fail(HS_E_STATE, "hs_replay_kernels: this batch runs attention in one split");
  for (int i = 0; i < count; ++i) {
    const int l = i % L;
    hipError_t e;
    switch (kind) {
      case HS_K_QKV: e = step.qkv(l, l ? step.down_defer() : 0); break;
      case HS_K_ATTN: e = step.attn(l); break;
      case HS_K_COMBINE: e = step.combine(l); break;
      case HS_K_OPROJ: e = step.oproj(l); break;
      case HS_K_GATEUP: e = step.gateup(l, step.o_defer()); break;
      case HS_K_DOWN: e = step.down(l); break;
      case HS_K_HEAD: e = step.head(m->x, m->logits, step.down_defer()); break;
      default: return fail(HS_E_INVALID, "hs_replay_kernels: kind %d cannot be replayed", kind);
    }
    HIP_TRY(e);
  }
  return HS_OK;
}

int hs_kv_lengths(const hs_kv *kv, int32_t *host_len) {
  if (!kv || !host_len) return fail(HS_E_INVALID, "hs_kv_lengths: NULL argument");
  HIP_TRY(hipDeviceSynchronize());
  HIP_TRY(hipMemcpy(host_len, kv->d_len, kv->batch * 4, hipMemcpyDeviceToHost));
  return HS_OK;
}

int hs_kv_sync(hs_kv *kv) {
  if (!kv) return fail(HS_E_INVALID, "hs_kv_sync: NULL handle");
  HIP_TRY(hipDeviceSynchronize());
  HIP_TRY(hipMemcpy(kv->len.data(), kv->d_len, kv->batch * 4, hipMemcpyDeviceToHost));
  HIP_TRY(hipMemcpy(kv->rope.data(), kv->d_rope, kv->batch * 4, hipMemcpyDeviceToHost));
  if (kv->pool) {
    HIP_TRY(hipMemcpy(kv->nblk.data(), kv->d_nblk, kv->batch * 4, hipMemcpyDeviceToHost));
    HIP_TRY(hipMemcpy(&kv->free_blocks, kv->d_top, 4, hipMemcpyDeviceToHost));
  }
  return HS_OK;
}

// The byte ranges of the cache buffer that hold rows pos0 .. pos0 + n - 1 of
// (req, layer, K|V, head), one per block they touch (host-side layout; a pooled
// cache's block starts are read from the device).
static int kv_slabs(const hs_kv *kv, int32_t req, int32_t layer, int32_t kv_sel, int32_t head, int32_t pos0,
                    int32_t n, const void *p, std::vector<std::pair<int64_t, size_t>> *out) {
  if (!kv || !p) return fail(HS_E_INVALID, "kv copy: NULL argument");
  const hs_config &c = kv->m->cfg;
  if (req < 0 || req >= kv->batch || layer < 0 || layer >= c.n_layers || kv_sel < 0 || kv_sel > 1 || head < 0 ||
      head >= c.n_kv_heads || pos0 < 0 || n < 0 || pos0 + (int64_t)n > kv->cap[req])
    return fail(HS_E_INVALID, "kv copy: (req %d, layer %d, kv %d, head %d, pos %d + %d) outside the cache", req, layer,
                kv_sel, head, pos0, n);
  const int b = dtype_bytes(c.dtype);
  const int bt = kv->pool ? kv->block_tokens : kv->cap[req];
  std::vector<int64_t> starts;
  if (kv->pool) {
    starts.resize(kv->max_blocks);
    HIP_TRY(hipDeviceSynchronize());
    HIP_TRY(hipMemcpy(starts.data(), kv->d_base + (int64_t)req * kv->max_blocks, kv->max_blocks * 8,
                      hipMemcpyDeviceToHost));
  } else {
    starts.assign(1, kv->base[req]);
  }
  out->clear();
  for (int p0 = pos0; p0 < pos0 + n;) {
    const int blk = p0 / bt, in_blk = std::min(pos0 + n, (blk + 1) * bt) - p0;
    if (starts[blk] < 0) return fail(HS_E_INVALID, "kv copy: position %d of request %d has no block", p0, req);
    const int64_t elem =
        starts[blk] + ((int64_t)((layer * 2 + kv_sel) * c.n_kv_heads + head) * bt + p0 - blk * bt) * c.head_dim;
    out->push_back({elem * b, (size_t)in_blk * c.head_dim * b});
    p0 += in_blk;
  }
  return HS_OK;
}

int hs_kv_write(hs_kv *kv, int32_t req, int32_t layer, int32_t kv_sel, int32_t head, int32_t pos0, int32_t n,
                const void *src, int32_t src_is_device) {
  std::vector<std::pair<int64_t, size_t>> slabs;
  int rc = kv_slabs(kv, req, layer, kv_sel, head, pos0, n, src, &slabs);
  if (rc) return rc;
  HIP_TRY(hipDeviceSynchronize());
  size_t done = 0;
  for (auto &sl : slabs) {
    HIP_TRY(hipMemcpy((char *)kv->buf + sl.first, (const char *)src + done, sl.second,
                      src_is_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice));
    done += sl.second;
  }
  HIP_TRY(hipDeviceSynchronize());
  return HS_OK;
}

int hs_kv_read(const hs_kv *kv, int32_t req, int32_t layer, int32_t kv_sel, int32_t head, int32_t pos0, int32_t n,
               void *dst, int32_t dst_is_device) {
  std::vector<std::pair<int64_t, size_t>> slabs;
  int rc = kv_slabs(kv, req, layer, kv_sel, head, pos0, n, dst, &slabs);
  if (rc) return rc;
  HIP_TRY(hipDeviceSynchronize());
  size_t done = 0;
  for (auto &sl : slabs) {
    HIP_TRY(hipMemcpy((char *)dst + done, (const char *)kv->buf + sl.first, sl.second,
                      dst_is_device ? hipMemcpyDeviceToDevice : hipMemcpyDeviceToHost));
    done += sl.second;
  }
  return HS_OK;
}

int hs_kv_set_length(hs_kv *kv, int32_t req, int32_t len, int32_t rope_pos) {
  if (!kv) return fail(HS_E_INVALID, "hs_kv_set_length: NULL");
  if (req < 0 || req >= kv->batch || len < 0 || len > kv->cap[req] || rope_pos < 0)
    return fail(HS_E_INVALID, "hs_kv_set_length: bad request/length");
  if (kv->pool) {  // blocks to cover the new length
    const int need = blocks_for(kv, len) - kv->nblk[req];
    if (need > kv->free_blocks)
      return fail(HS_E_CAPACITY, "hs_kv_set_length: the pool has %d free blocks, %d needed", kv->free_blocks, need);
    if (need > 0) {
      KvReserve r{};
      r.n = 1;
      r.req[0] = req;
      r.target[0] = len;
      HIP_TRY(launch_kv_reserve(kv_pool(kv), r, 0, nullptr));
      kv->nblk[req] += need;
      kv->free_blocks -= need;
    }
  }
  const int ready = len > 0;
  HIP_TRY(hipDeviceSynchronize());
  HIP_TRY(hipMemcpy(kv->d_len + req, &len, 4, hipMemcpyHostToDevice));
  HIP_TRY(hipMemcpy(kv->d_rope + req, &rope_pos, 4, hipMemcpyHostToDevice));
  HIP_TRY(hipMemcpy(kv->d_ready + req, &ready, 4, hipMemcpyHostToDevice));
  kv->len[req] = len;
  kv->rope[req] = rope_pos;
  kv->ready[req] = ready;
  HIP_TRY(kv->pool ? rebuild_active(kv, nullptr) : rebuild_order(kv, nullptr));
  HIP_TRY(hipDeviceSynchronize());
  return HS_OK;
}

}  // extern "C"
