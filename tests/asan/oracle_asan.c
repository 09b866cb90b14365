/*
 * Drives every entry point of the CPU oracle on small models (each storage
 * dtype, both RoPE kinds, with and without q/k/v bias and LM head), including
 * the argument and state errors, for a build with AddressSanitizer and
 * UndefinedBehaviorSanitizer (tests/test_sanitize.py).  Weights are filled from
 * a xorshift generator: memory safety, not values, is what this run checks.
 * Prints "ok" and returns 0 when every call returned what it should.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "hs_oracle.h"

static uint64_t g_state = 88172645463325252ull;
static float rnd(void) {
  g_state ^= g_state << 13;
  g_state ^= g_state >> 7;
  g_state ^= g_state << 17;
  return (float)((double)(g_state >> 11) / 9007199254740992.0) * 2.f - 1.f;
}

static void *arr(int32_t dtype, int64_t n, float mean, float scale) {
  const size_t b = dtype == OR_F32 ? 4 : 2;
  void *p = malloc((size_t)n * b);
  for (int64_t i = 0; i < n; ++i) {
    const float v = mean + scale * rnd();
    if (dtype == OR_F32) ((float *)p)[i] = v;
    else if (dtype == OR_F16) ((uint16_t *)p)[i] = or_f32_to_f16_bits(v);
    else ((uint16_t *)p)[i] = or_f32_to_bf16_bits(v);
  }
  return p;
}

static int g_fail = 0;
#define EXPECT(cond)                                                 \
  do {                                                               \
    if (!(cond)) {                                                   \
      fprintf(stderr, "%s:%d: expected %s\n", __FILE__, __LINE__, #cond); \
      g_fail = 1;                                                    \
    }                                                                \
  } while (0)

static void run(int32_t dtype, int32_t rope_kind, int32_t bias, int32_t with_head) {
  or_config c;
  memset(&c, 0, sizeof c);
  c.n_layers = 2;
  c.d_model = 72;
  c.n_heads = 4;
  c.n_kv_heads = 2;
  c.head_dim = 16;
  c.ffn_dim = 100;
  c.vocab = 53;
  c.rope_theta = 10000.f;
  c.rms_eps = 1e-5f;
  c.rope_kind = rope_kind;
  if (rope_kind == OR_ROPE_M3) {
    c.mrope_section[0] = 2;
    c.mrope_section[1] = 3;
    c.mrope_section[2] = 3;
  }
  c.qkv_bias = bias;
  c.dtype = dtype;
  const int32_t d = c.d_model, qd = c.n_heads * c.head_dim, kd = c.n_kv_heads * c.head_dim, F = c.ffn_dim;
  or_layer layers[2];
  for (int l = 0; l < 2; ++l) {
    or_layer *L = &layers[l];
    L->attn_norm = arr(dtype, d, 1.f, 0.1f);
    L->wq = arr(dtype, (int64_t)qd * d, 0.f, 0.1f);
    L->wk = arr(dtype, (int64_t)kd * d, 0.f, 0.1f);
    L->wv = arr(dtype, (int64_t)kd * d, 0.f, 0.1f);
    L->bq = bias ? arr(dtype, qd, 0.f, 0.1f) : NULL;
    L->bk = bias ? arr(dtype, kd, 0.f, 0.1f) : NULL;
    L->bv = bias ? arr(dtype, kd, 0.f, 0.1f) : NULL;
    L->wo = arr(dtype, (int64_t)d * qd, 0.f, 0.1f);
    L->mlp_norm = arr(dtype, d, 1.f, 0.1f);
    L->w_gate = arr(dtype, (int64_t)F * d, 0.f, 0.1f);
    L->w_up = arr(dtype, (int64_t)F * d, 0.f, 0.1f);
    L->w_down = arr(dtype, (int64_t)d * F, 0.f, 0.1f);
  }
  or_model m;
  m.cfg = c;
  m.embed = arr(dtype, (int64_t)c.vocab * d, 0.f, 1.f);
  m.final_norm = with_head ? arr(dtype, d, 1.f, 0.1f) : NULL;
  m.lm_head = with_head ? arr(dtype, (int64_t)c.vocab * d, 0.f, 0.1f) : NULL;
  m.layers = layers;

  uint64_t kvb = 0, eb = 0;
  EXPECT(or_transfer_bytes(&c, 9, 4, &kvb, &eb) == 0);
  EXPECT(or_transfer_bytes(&c, -1, 4, &kvb, &eb) != 0);

  const int32_t n_v = 9, s_text = 4, n_dec = 5, cap = n_v + s_text + n_dec;
  void *emb = arr(dtype, (int64_t)n_v * d, 0.f, 1.f);
  int32_t ids[4] = {1, 52, 0, 17};
  int32_t pos[3 * 13];
  for (int r = 0; r < n_v + s_text; ++r) {  /* a 3 x 3 image, then text */
    const int img = r < n_v;
    pos[r] = img ? 0 : r - n_v + 3;
    pos[13 + r] = img ? r / 3 : r - n_v + 3;
    pos[26 + r] = img ? r % 3 : r - n_v + 3;
  }
  const int32_t *pthw = rope_kind == OR_ROPE_M3 ? pos : NULL;
  float *logits = (float *)malloc(sizeof(float) * (size_t)c.vocab);
  float *hidden = (float *)malloc(sizeof(float) * (size_t)d);
  int32_t tok = -1;

  or_seq s, t;
  EXPECT(or_seq_init(&m, &s, cap) == 0);
  EXPECT(or_decode(&m, &s, 3, logits, hidden, &tok) != 0);          /* not prefilled */
  int32_t bad_ids[4] = {1, 53, 0, 2};
  EXPECT(or_prefill(&m, &s, emb, n_v, bad_ids, s_text, pthw, logits, &tok) != 0);  /* id out of range */
  EXPECT(or_prefill(&m, &s, emb, n_v, ids, s_text, pthw, with_head ? logits : NULL, &tok) == 0);
  EXPECT(or_prefill(&m, &s, emb, n_v, ids, s_text, pthw, logits, &tok) != 0);      /* already prefilled */
  EXPECT(tok == (with_head ? tok : -1));
  for (int k = 0; k < n_dec; ++k) {
    const int32_t in = with_head ? tok : k % c.vocab;
    EXPECT(or_decode(&m, &s, in, with_head ? logits : NULL, hidden, &tok) == 0);
  }
  EXPECT(or_decode(&m, &s, 0, NULL, NULL, NULL) != 0);                /* full */
  EXPECT(or_decode(&m, &s, -1, NULL, NULL, NULL) != 0);               /* id out of range */

  /* the cache copied row by row into a second sequence, then one more step on each */
  EXPECT(or_seq_init(&m, &t, cap + 1) == 0);
  float *rows = (float *)malloc(sizeof(float) * (size_t)cap * c.head_dim);
  for (int l = 0; l < c.n_layers; ++l)
    for (int sel = 0; sel < 2; ++sel)
      for (int h = 0; h < c.n_kv_heads; ++h) {
        EXPECT(or_seq_read_kv(&m, &s, l, sel, h, 0, cap, rows) == 0);
        EXPECT(or_seq_write_kv(&m, &t, l, sel, h, 0, cap, rows) == 0);
      }
  EXPECT(or_seq_read_kv(&m, &s, 2, 0, 0, 0, 1, rows) != 0);
  EXPECT(or_seq_read_kv(&m, &s, 0, 2, 0, 0, 1, rows) != 0);
  EXPECT(or_seq_read_kv(&m, &s, 0, 0, 2, 0, 1, rows) != 0);
  EXPECT(or_seq_read_kv(&m, &s, 0, 0, 0, cap, 1, rows) != 0);
  EXPECT(or_seq_write_kv(&m, &t, 0, 0, 0, cap, 2, rows) != 0);
  EXPECT(or_seq_set_len(&t, cap + 2, 0) != 0);
  EXPECT(or_seq_set_len(&t, cap, s.rope_pos) == 0);
  EXPECT(or_decode(&m, &t, 5, with_head ? logits : NULL, hidden, &tok) == 0);

  /* building blocks on their own */
  float hv[72];
  float xv[72];
  for (int k = 0; k < d; ++k) xv[k] = rnd();
  or_rmsnorm(d, xv, layers[0].attn_norm, dtype, c.rms_eps, hv);
  float cs = 0.f, sn = 0.f;
  or_rope_cos_sin(c.rope_theta, c.head_dim, 3, 11, &cs, &sn);
  const int32_t p3[3] = {4, 5, 6};
  or_rope_rotate(&c, hv, p3);
  float q[16], kk[3 * 16], vv[3 * 16], o[16];
  for (int e = 0; e < 16; ++e) q[e] = rnd();
  for (int e = 0; e < 48; ++e) {
    kk[e] = rnd();
    vv[e] = rnd();
  }
  or_attention(3, 16, q, kk, 16, vv, 16, o);
  EXPECT(or_argmax(d, hv) >= 0);
  (void)or_silu(0.5f);

  free(rows);
  or_seq_free(&s);
  or_seq_free(&t);
  free(logits);
  free(hidden);
  free(emb);
  for (int l = 0; l < 2; ++l) {
    or_layer *L = &layers[l];
    const void *ps[] = {L->attn_norm, L->wq, L->wk, L->wv, L->bq, L->bk, L->bv, L->wo, L->mlp_norm, L->w_gate,
                        L->w_up, L->w_down};
    for (size_t i = 0; i < sizeof ps / sizeof ps[0]; ++i) free((void *)ps[i]);
  }
  free((void *)m.embed);
  free((void *)m.final_norm);
  free((void *)m.lm_head);
}

int main(void) {
  for (int32_t dtype = OR_F32; dtype <= OR_BF16; ++dtype)
    for (int32_t rope = OR_ROPE_1D; rope <= OR_ROPE_M3; ++rope)
      for (int32_t bias = 0; bias <= 1; ++bias)
        for (int32_t head = 0; head <= 1; ++head) run(dtype, rope, bias, head);
  if (g_fail) return 1;
  printf("ok\n");
  return 0;
}
