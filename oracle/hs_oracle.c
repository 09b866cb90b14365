/*
 * hs_oracle.c — plain CPU oracle for the language-decode step of
 * modality-disaggregated MLLM serving (arXiv 2603.12707).
 *
 * TEST INFRASTRUCTURE ONLY: used by the test suite, the smoke check and the
 * benchmark's CPU-baseline leg, never by the product path.  It shares no code
 * with the HIP library.  Precision and scope are described in hs_oracle.h.
 *
 * Paper anchors:
 *   - Eq. 1 (§4.1): D_KV = 2 * L * n_kv * d_h * s_ctx * b.
 *   - Embedding-size display (§4.1): D_emb = N_v * d * b.
 *   - Theorem 1 / Eq. 2 (§4.2): s_ctx = N_v + s_text.
 *   - §2 and Eq. 5 (§4.3): decode streams the weights and the KV cache from
 *     HBM once per generated token; each token appends one K and one V row
 *     per layer (§4 opening paragraph).
 *   - §5.1: the language model consumes the projected embedding [1, N_v, d]
 *     as its first N_v input rows.
 *   - §6.1 "Models": LLaVA-1.5-7B (Vicuna-7B backbone, MHA, 32 layers, 32 KV
 *     heads) and Qwen2.5-VL (GQA backbone, 28 layers, 4 KV heads).
 * The decoder layer itself is the standard pre-RMSNorm LLaMA layer; the paper
 * does not write it out.
 */
#include "hs_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#define OR_OK 0
#define OR_E_INVALID (-1)
#define OR_E_CAPACITY (-2)
#define OR_E_STATE (-4)

/* ------------------------------------------------------------------------ */
/* Storage formats.                                                          */
/* ------------------------------------------------------------------------ */

/* IEEE binary32 -> binary16, round to nearest, ties to even. */
uint16_t or_f32_to_f16_bits(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  uint32_t sign = (u >> 16) & 0x8000u;
  uint32_t ex = (u >> 23) & 0xFFu;
  uint32_t man = u & 0x7FFFFFu;
  if (ex == 0xFFu) return (uint16_t)(sign | 0x7C00u | (man ? 0x200u : 0u));
  int32_t e = (int32_t)ex - 127 + 15;
  if (e >= 31) return (uint16_t)(sign | 0x7C00u);
  if (e <= 0) {
    /* result is a binary16 subnormal (or zero); value = man * 2^(e - 14)
       units of 2^-24 once the implicit bit is restored */
    if (e < -10) return (uint16_t)sign;
    man |= 0x800000u;
    int shift = 14 - e;
    uint32_t h = man >> shift;
    uint32_t rem = man & ((1u << shift) - 1u);
    uint32_t half = 1u << (shift - 1);
    if (rem > half || (rem == half && (h & 1u))) h++;
    return (uint16_t)(sign | h);
  }
  uint32_t h = ((uint32_t)e << 10) | (man >> 13);
  uint32_t rem = man & 0x1FFFu;
  if (rem > 0x1000u || (rem == 0x1000u && (h & 1u))) h++;
  return (uint16_t)(sign | h);
}

/* IEEE binary32 -> bfloat16, round to nearest, ties to even. */
uint16_t or_f32_to_bf16_bits(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  if (((u >> 23) & 0xFFu) == 0xFFu && (u & 0x7FFFFFu)) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

static float f16_bits_to_f32(uint16_t h) {
  uint32_t sign = ((uint32_t)h & 0x8000u) << 16;
  uint32_t ex = ((uint32_t)h >> 10) & 0x1Fu;
  uint32_t man = (uint32_t)h & 0x3FFu;
  uint32_t u;
  if (ex == 0) {
    if (man == 0) {
      u = sign;
    } else { /* subnormal: man * 2^-24 */
      float f = (float)man * 5.9604644775390625e-08f;
      memcpy(&u, &f, 4);
      u |= sign;
    }
  } else if (ex == 31) {
    u = sign | 0x7F800000u | (man << 13);
  } else {
    u = sign | ((ex - 15 + 127) << 23) | (man << 13);
  }
  float f;
  memcpy(&f, &u, 4);
  return f;
}

static float bf16_bits_to_f32(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

static float g_f16_table[65536];
static int g_f16_table_ready = 0;

static void f16_table_init(void) {
  if (g_f16_table_ready) return;
  for (uint32_t i = 0; i < 65536u; ++i) g_f16_table[i] = f16_bits_to_f32((uint16_t)i);
  g_f16_table_ready = 1;
}

float or_load(int32_t dtype, const void *p, int64_t i) {
  if (dtype == OR_F32) return ((const float *)p)[i];
  uint16_t h = ((const uint16_t *)p)[i];
  return dtype == OR_F16 ? f16_bits_to_f32(h) : bf16_bits_to_f32(h);
}

/* R(.): round an fp32 value to the storage dtype and back. */
float or_round(int32_t dtype, float x) {
  if (dtype == OR_F16) return f16_bits_to_f32(or_f32_to_f16_bits(x));
  if (dtype == OR_BF16) return bf16_bits_to_f32(or_f32_to_bf16_bits(x));
  return x;
}

static int64_t dtype_bytes(int32_t dtype) { return dtype == OR_F32 ? 4 : 2; }

/* Sequential fp64 dot product of an fp32 vector with row `row` of a
 * row-major [*, K] matrix in the storage dtype. */
static double dot_row(int32_t dtype, const void *w, int64_t row, int32_t K, const float *h) {
  double acc = 0.0;
  if (dtype == OR_F32) {
    const float *r = (const float *)w + row * (int64_t)K;
    for (int32_t k = 0; k < K; ++k) acc += (double)h[k] * (double)r[k];
  } else if (dtype == OR_F16) {
    const uint16_t *r = (const uint16_t *)w + row * (int64_t)K;
    for (int32_t k = 0; k < K; ++k) acc += (double)h[k] * (double)g_f16_table[r[k]];
  } else {
    const uint16_t *r = (const uint16_t *)w + row * (int64_t)K;
    for (int32_t k = 0; k < K; ++k) acc += (double)h[k] * (double)bf16_bits_to_f32(r[k]);
  }
  return acc;
}

/* ------------------------------------------------------------------------ */
/* Eq. 1 and the embedding-size display (§4.1).                              */
/* ------------------------------------------------------------------------ */
int or_transfer_bytes(const or_config *c, int64_t n_v, int64_t s_text, uint64_t *kv_bytes,
                      uint64_t *emb_bytes) {
  if (!c || n_v < 0 || s_text < 0 || c->n_layers <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0 ||
      c->d_model <= 0 || c->dtype < OR_F32 || c->dtype > OR_BF16)
    return OR_E_INVALID;
  uint64_t b = (uint64_t)dtype_bytes(c->dtype);
  uint64_t s_ctx = (uint64_t)n_v + (uint64_t)s_text;
  if (kv_bytes)
    *kv_bytes = 2ull * (uint64_t)c->n_layers * (uint64_t)c->n_kv_heads * (uint64_t)c->head_dim * s_ctx * b;
  if (emb_bytes) *emb_bytes = (uint64_t)n_v * (uint64_t)c->d_model * b;
  return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Building blocks.                                                          */
/* ------------------------------------------------------------------------ */

/* h = R(x / sqrt(mean(x^2) + eps) * g) */
void or_rmsnorm(int32_t d, const float *x, const void *gain, int32_t dtype, float eps, float *h_out) {
  double ss = 0.0;
  for (int32_t k = 0; k < d; ++k) ss += (double)x[k] * (double)x[k];
  double rsq = 1.0 / sqrt(ss / (double)d + (double)eps);
  for (int32_t k = 0; k < d; ++k)
    h_out[k] = or_round(dtype, (float)((double)x[k] * rsq * (double)or_load(dtype, gain, k)));
}

/* Rotary embedding, rotate-half form: frequency pair i couples elements i and
 * i + d_h/2 and turns them by pos * theta^(-2i/d_h).  Angle and cos/sin are
 * evaluated in fp64 and rounded to fp32. */
void or_rope_cos_sin(float theta, int32_t head_dim, int32_t pair, int32_t pos, float *c, float *s) {
  double inv = pow((double)theta, -(double)(2 * pair) / (double)head_dim);
  double ang = (double)pos * inv;
  *c = (float)cos(ang);
  *s = (float)sin(ang);
}

static int32_t rope_pos_of_pair(const or_config *c, int32_t pair, const int32_t pos3[3]) {
  if (c->rope_kind != OR_ROPE_M3) return pos3[0];
  if (pair < c->mrope_section[0]) return pos3[0];
  if (pair < c->mrope_section[0] + c->mrope_section[1]) return pos3[1];
  return pos3[2];
}

/* Rotates one head vector (length d_h, fp32) in place; no storage rounding. */
void or_rope_rotate(const or_config *c, float *vec, const int32_t pos3[3]) {
  int32_t half = c->head_dim / 2;
  for (int32_t i = 0; i < half; ++i) {
    float cs, sn;
    or_rope_cos_sin(c->rope_theta, c->head_dim, i, rope_pos_of_pair(c, i, pos3), &cs, &sn);
    double x1 = vec[i], x2 = vec[i + half];
    vec[i] = (float)(x1 * (double)cs - x2 * (double)sn);
    vec[i + half] = (float)(x2 * (double)cs + x1 * (double)sn);
  }
}

/* o = softmax(q K^T / sqrt(d_h)) V over n_t tokens, in fp64, rounded to fp32. */
void or_attention(int32_t n_t, int32_t d_h, const float *q, const float *k, int64_t k_stride,
                  const float *v, int64_t v_stride, float *o_out) {
  double *p = (double *)malloc(sizeof(double) * (size_t)(n_t > 0 ? n_t : 1));
  double scale = 1.0 / sqrt((double)d_h);
  double m = -INFINITY;
  for (int32_t t = 0; t < n_t; ++t) {
    double dot = 0.0;
    for (int32_t e = 0; e < d_h; ++e) dot += (double)q[e] * (double)k[t * k_stride + e];
    p[t] = dot * scale;
    if (p[t] > m) m = p[t];
  }
  double l = 0.0;
  for (int32_t t = 0; t < n_t; ++t) {
    p[t] = exp(p[t] - m);
    l += p[t];
  }
  for (int32_t e = 0; e < d_h; ++e) {
    double acc = 0.0;
    for (int32_t t = 0; t < n_t; ++t) acc += p[t] * (double)v[t * v_stride + e];
    o_out[e] = (float)(acc / l);
  }
  free(p);
}

float or_silu(float z) { return (float)((double)z / (1.0 + exp(-(double)z))); }

/* Greedy selection: the largest logit, lowest index among equals; -1 on NaN
 * or empty input. */
int32_t or_argmax(int32_t n, const float *v) {
  if (n <= 0) return -1;
  int32_t best = 0;
  for (int32_t i = 0; i < n; ++i) {
    if (isnan(v[i])) return -1;
    if (v[i] > v[best]) best = i;
  }
  return best;
}

/* ------------------------------------------------------------------------ */
/* Request state.                                                            */
/* ------------------------------------------------------------------------ */
static int config_ok(const or_config *c) {
  if (c->n_layers <= 0 || c->d_model <= 0 || c->n_heads <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0 ||
      c->ffn_dim <= 0 || c->vocab <= 0)
    return 0;
  if (c->n_heads % c->n_kv_heads != 0 || c->head_dim % 2 != 0) return 0;
  if (c->dtype < OR_F32 || c->dtype > OR_BF16) return 0;
  if (c->rope_kind == OR_ROPE_M3 &&
      c->mrope_section[0] + c->mrope_section[1] + c->mrope_section[2] != c->head_dim / 2)
    return 0;
  return 1;
}

static int64_t kv_index(const or_config *c, const or_seq *s, int32_t layer, int32_t kv_sel, int32_t pos,
                        int32_t head) {
  return ((((int64_t)layer * 2 + kv_sel) * s->cap + pos) * c->n_kv_heads + head) * c->head_dim;
}

int or_seq_init(const or_model *m, or_seq *s, int32_t cap) {
  if (!m || !s || cap <= 0 || !config_ok(&m->cfg)) return OR_E_INVALID;
  const or_config *c = &m->cfg;
  size_t n = (size_t)c->n_layers * 2u * (size_t)cap * (size_t)c->n_kv_heads * (size_t)c->head_dim;
  s->kv = (float *)calloc(n, sizeof(float));
  if (!s->kv) return OR_E_INVALID;
  s->cap = cap;
  s->len = 0;
  s->rope_pos = 0;
  f16_table_init();
  return OR_OK;
}

void or_seq_free(or_seq *s) {
  if (s && s->kv) free(s->kv);
  if (s) s->kv = NULL;
}

int or_seq_write_kv(const or_model *m, or_seq *s, int32_t layer, int32_t kv_sel, int32_t head, int32_t pos0,
                    int32_t n, const float *src) {
  const or_config *c = &m->cfg;
  if (layer < 0 || layer >= c->n_layers || kv_sel < 0 || kv_sel > 1 || head < 0 || head >= c->n_kv_heads ||
      pos0 < 0 || n < 0 || pos0 + n > s->cap)
    return OR_E_INVALID;
  for (int32_t t = 0; t < n; ++t) {
    float *dst = s->kv + kv_index(c, s, layer, kv_sel, pos0 + t, head);
    for (int32_t e = 0; e < c->head_dim; ++e) dst[e] = or_round(c->dtype, src[(int64_t)t * c->head_dim + e]);
  }
  return OR_OK;
}

int or_seq_read_kv(const or_model *m, const or_seq *s, int32_t layer, int32_t kv_sel, int32_t head, int32_t pos0,
                   int32_t n, float *dst) {
  const or_config *c = &m->cfg;
  if (layer < 0 || layer >= c->n_layers || kv_sel < 0 || kv_sel > 1 || head < 0 || head >= c->n_kv_heads ||
      pos0 < 0 || n < 0 || pos0 + n > s->cap)
    return OR_E_INVALID;
  for (int32_t t = 0; t < n; ++t) {
    const float *src = s->kv + kv_index(c, s, layer, kv_sel, pos0 + t, head);
    memcpy(dst + (int64_t)t * c->head_dim, src, sizeof(float) * (size_t)c->head_dim);
  }
  return OR_OK;
}

int or_seq_set_len(or_seq *s, int32_t len, int32_t rope_pos) {
  if (len < 0 || len > s->cap) return OR_E_INVALID;
  s->len = len;
  s->rope_pos = rope_pos;
  return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* One row through every layer.                                              */
/* ------------------------------------------------------------------------ */

/* Runs the row x_in (fp32, length d) at position index s->len through all
 * layers, appending its K/V rows; optional outputs are the final residual
 * (before the final norm) and the LM-head logits. */
int or_forward_row(const or_model *m, or_seq *s, const float *x_in, const int32_t pos3[3], float *hidden_out,
                   float *logits_out) {
  const or_config *c = &m->cfg;
  if (!config_ok(c)) return OR_E_INVALID;
  if (s->len >= s->cap) return OR_E_CAPACITY;
  f16_table_init();
  const int32_t d = c->d_model, hd = c->head_dim, nh = c->n_heads, nkv = c->n_kv_heads, F = c->ffn_dim;
  const int32_t g = nh / nkv, dt = c->dtype, pos = s->len;
  const int64_t kv_row = (int64_t)nkv * hd; /* stride between positions */

  float *x = (float *)malloc(sizeof(float) * (size_t)d);
  float *h = (float *)malloc(sizeof(float) * (size_t)d);
  float *q = (float *)malloc(sizeof(float) * (size_t)nh * hd);
  float *kk = (float *)malloc(sizeof(float) * (size_t)nkv * hd);
  float *vv = (float *)malloc(sizeof(float) * (size_t)nkv * hd);
  float *o = (float *)malloc(sizeof(float) * (size_t)nh * hd);
  float *a = (float *)malloc(sizeof(float) * (size_t)F);
  memcpy(x, x_in, sizeof(float) * (size_t)d);

  for (int32_t l = 0; l < c->n_layers; ++l) {
    const or_layer *W = &m->layers[l];
    /* attention block */
    or_rmsnorm(d, x, W->attn_norm, dt, c->rms_eps, h);
    for (int32_t r = 0; r < nh * hd; ++r)
      q[r] = (float)(dot_row(dt, W->wq, r, d, h) + (c->qkv_bias ? (double)or_load(dt, W->bq, r) : 0.0));
    for (int32_t r = 0; r < nkv * hd; ++r) {
      kk[r] = (float)(dot_row(dt, W->wk, r, d, h) + (c->qkv_bias ? (double)or_load(dt, W->bk, r) : 0.0));
      vv[r] = (float)(dot_row(dt, W->wv, r, d, h) + (c->qkv_bias ? (double)or_load(dt, W->bv, r) : 0.0));
    }
    for (int32_t hh = 0; hh < nh; ++hh) or_rope_rotate(c, q + (int64_t)hh * hd, pos3);
    for (int32_t j = 0; j < nkv; ++j) or_rope_rotate(c, kk + (int64_t)j * hd, pos3);
    for (int32_t r = 0; r < nh * hd; ++r) q[r] = or_round(dt, q[r]);
    for (int32_t j = 0; j < nkv; ++j) {
      float *kd = s->kv + kv_index(c, s, l, 0, pos, j);
      float *vd = s->kv + kv_index(c, s, l, 1, pos, j);
      for (int32_t e = 0; e < hd; ++e) {
        kd[e] = or_round(dt, kk[(int64_t)j * hd + e]);
        vd[e] = or_round(dt, vv[(int64_t)j * hd + e]);
      }
    }
    for (int32_t hh = 0; hh < nh; ++hh) {
      int32_t j = hh / g; /* query head hh reads KV head floor(hh / g) */
      or_attention(pos + 1, hd, q + (int64_t)hh * hd, s->kv + kv_index(c, s, l, 0, 0, j), kv_row,
                   s->kv + kv_index(c, s, l, 1, 0, j), kv_row, o + (int64_t)hh * hd);
    }
    for (int32_t r = 0; r < nh * hd; ++r) o[r] = or_round(dt, o[r]);
    for (int32_t n = 0; n < d; ++n) x[n] = (float)((double)x[n] + dot_row(dt, W->wo, n, nh * hd, o));

    /* MLP block */
    or_rmsnorm(d, x, W->mlp_norm, dt, c->rms_eps, h);
    for (int32_t j = 0; j < F; ++j) {
      float gate = (float)dot_row(dt, W->w_gate, j, d, h);
      float up = (float)dot_row(dt, W->w_up, j, d, h);
      double silu = (double)gate / (1.0 + exp(-(double)gate));
      a[j] = or_round(dt, (float)(silu * (double)up));
    }
    for (int32_t n = 0; n < d; ++n) x[n] = (float)((double)x[n] + dot_row(dt, W->w_down, n, F, a));
  }
  s->len += 1;

  if (hidden_out) memcpy(hidden_out, x, sizeof(float) * (size_t)d);
  if (logits_out && m->lm_head) {
    or_rmsnorm(d, x, m->final_norm, dt, c->rms_eps, h);
    for (int32_t v = 0; v < c->vocab; ++v) logits_out[v] = (float)dot_row(dt, m->lm_head, v, d, h);
  }
  free(x);
  free(h);
  free(q);
  free(kk);
  free(vv);
  free(o);
  free(a);
  return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Prefill from the projected embedding, then greedy decode.                 */
/* ------------------------------------------------------------------------ */

/* Rows 0..n_v-1 are the vision embedding rows, rows n_v..n_v+s_text-1 the
 * text-token embeddings.  1-D RoPE uses position r for row r; M-RoPE takes
 * the (t, h, w) ids of row r from pos_thw[0..2][r].  The next decode position
 * is s_ctx for 1-D RoPE and max(pos_thw) + 1 for M-RoPE. */
int or_prefill(const or_model *m, or_seq *s, const void *emb, int32_t n_v, const int32_t *text_ids, int32_t s_text,
               const int32_t *pos_thw, float *last_logits, int32_t *first_token) {
  const or_config *c = &m->cfg;
  if (!config_ok(c) || n_v < 0 || s_text < 0 || n_v + s_text <= 0) return OR_E_INVALID;
  if ((n_v > 0 && !emb) || (s_text > 0 && !text_ids)) return OR_E_INVALID;
  if (c->rope_kind == OR_ROPE_M3 && !pos_thw) return OR_E_INVALID;
  if (s->len != 0) return OR_E_STATE;
  const int32_t d = c->d_model, s_ctx = n_v + s_text;
  if (s_ctx > s->cap) return OR_E_CAPACITY;
  for (int32_t t = 0; t < s_text; ++t)
    if (text_ids[t] < 0 || text_ids[t] >= c->vocab) return OR_E_INVALID;

  float *x = (float *)malloc(sizeof(float) * (size_t)d);
  float *logits = m->lm_head ? (float *)malloc(sizeof(float) * (size_t)c->vocab) : NULL;
  int rc = OR_OK;
  for (int32_t r = 0; r < s_ctx && rc == OR_OK; ++r) {
    for (int32_t k = 0; k < d; ++k)
      x[k] = r < n_v ? or_load(c->dtype, emb, (int64_t)r * d + k)
                     : or_load(c->dtype, m->embed, (int64_t)text_ids[r - n_v] * d + k);
    int32_t pos3[3];
    if (c->rope_kind == OR_ROPE_M3) {
      pos3[0] = pos_thw[r];
      pos3[1] = pos_thw[s_ctx + r];
      pos3[2] = pos_thw[2 * s_ctx + r];
    } else {
      pos3[0] = pos3[1] = pos3[2] = r;
    }
    rc = or_forward_row(m, s, x, pos3, NULL, r == s_ctx - 1 ? logits : NULL);
  }
  if (rc == OR_OK) {
    if (c->rope_kind == OR_ROPE_M3) {
      int32_t mx = pos_thw[0];
      for (int64_t i = 0; i < 3 * (int64_t)s_ctx; ++i)
        if (pos_thw[i] > mx) mx = pos_thw[i];
      s->rope_pos = mx + 1;
    } else {
      s->rope_pos = s_ctx;
    }
    if (logits) {
      if (last_logits) memcpy(last_logits, logits, sizeof(float) * (size_t)c->vocab);
      if (first_token) *first_token = or_argmax(c->vocab, logits);
    } else if (first_token) {
      *first_token = -1;
    }
  }
  free(x);
  free(logits);
  return rc;
}

/* One greedy decode step: embeds token_in at the next position, appends its
 * K/V rows and returns the argmax of the logits. */
int or_decode(const or_model *m, or_seq *s, int32_t token_in, float *logits, float *hidden, int32_t *token_out) {
  const or_config *c = &m->cfg;
  if (!config_ok(c)) return OR_E_INVALID;
  if (token_in < 0 || token_in >= c->vocab) return OR_E_INVALID;
  if (s->len == 0) return OR_E_STATE;
  if (s->len >= s->cap) return OR_E_CAPACITY;
  const int32_t d = c->d_model;
  float *x = (float *)malloc(sizeof(float) * (size_t)d);
  float *lg = NULL;
  if (m->lm_head) lg = logits ? logits : (float *)malloc(sizeof(float) * (size_t)c->vocab);
  for (int32_t k = 0; k < d; ++k) x[k] = or_load(c->dtype, m->embed, (int64_t)token_in * d + k);
  int32_t pos3[3] = {s->rope_pos, s->rope_pos, s->rope_pos};
  int rc = or_forward_row(m, s, x, pos3, hidden, lg);
  if (rc == OR_OK) {
    s->rope_pos += 1;
    if (token_out) *token_out = lg ? or_argmax(c->vocab, lg) : -1;
  }
  if (lg && lg != logits) free(lg);
  free(x);
  return rc;
}
