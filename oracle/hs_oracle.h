/*
 * hs_oracle.h — declarations of the CPU oracle for the language-decode step of
 * modality-disaggregated MLLM serving (arXiv 2603.12707).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may include, link or
 * call this code: only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg use it.  It shares no code, header, table or constant with
 * the HIP library.
 *
 * What it computes: a LLaMA-style pre-RMSNorm decoder (RoPE, SwiGLU MLP,
 * untied LM head) fed first with projected vision-embedding rows and then with
 * text-token embeddings, run one row at a time in causal order, followed by
 * greedy decode.  The paper names the models (Vicuna-7B backbone with MHA,
 * 32 layers, 32 KV heads; a GQA backbone with 28 layers and 4 KV heads, §6.1
 * "Models") but never writes the layer out; the plain textbook definition is
 * used.  The KV-cache and embedding sizes follow Eq. 1 and the embedding-size
 * display of §4.1.
 *
 * Precision: every value the method holds (residual stream, logits, RoPE
 * tables) is fp32; values written to storage (normalised activations, q/k/v
 * after RoPE, attention output, SwiGLU output) are rounded to the storage
 * dtype with round-to-nearest-even.  Every dot product and reduction is
 * evaluated in fp64 in sequential index order and rounded once.
 *
 * Single-threaded, no SIMD intrinsics, no blocking: slow on purpose.
 */
#ifndef HS_ORACLE_H
#define HS_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { OR_F32 = 0, OR_F16 = 1, OR_BF16 = 2 };
enum { OR_ROPE_1D = 0, OR_ROPE_M3 = 1 };

typedef struct or_config {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab;
  float rope_theta, rms_eps;
  int32_t rope_kind;        /* OR_ROPE_1D or OR_ROPE_M3 */
  int32_t mrope_section[3]; /* frequency-pair counts per (t, h, w) section */
  int32_t qkv_bias;         /* 1: q/k/v projections carry a bias vector */
  int32_t dtype;            /* storage dtype of weights, KV and activations */
} or_config;

/* Per-layer weights, row-major nn.Linear layout [out_features, in_features],
 * all in the storage dtype. */
typedef struct or_layer {
  const void *attn_norm;          /* [d] */
  const void *wq, *wk, *wv;       /* [n_h*d_h, d], [n_kv*d_h, d], [n_kv*d_h, d] */
  const void *bq, *bk, *bv;       /* biases or NULL */
  const void *wo;                 /* [d, n_h*d_h] */
  const void *mlp_norm;           /* [d] */
  const void *w_gate, *w_up;      /* [F, d] */
  const void *w_down;             /* [d, F] */
} or_layer;

typedef struct or_model {
  or_config cfg;
  const void *embed;              /* [V, d] */
  const void *final_norm;         /* [d]; unused when lm_head is NULL */
  const void *lm_head;            /* [V, d] or NULL (layer stack only) */
  const or_layer *layers;         /* [n_layers] */
} or_model;

/* One request's state: its own KV cache (fp32 array holding storage-rounded
 * values, layout [layer][K|V][pos][kv_head][d_h]), its length and the RoPE
 * position of the next decoded token. */
typedef struct or_seq {
  int32_t cap, len, rope_pos;
  float *kv;
} or_seq;

/* ---- Eq. 1 and the embedding-size display (§4.1), Theorem 1 (§4.2) ---- */
int or_transfer_bytes(const or_config *c, int64_t n_v, int64_t s_text,
                      uint64_t *kv_bytes, uint64_t *emb_bytes);

/* ---- element access and storage rounding ---- */
float or_load(int32_t dtype, const void *p, int64_t i);
float or_round(int32_t dtype, float x);
uint16_t or_f32_to_f16_bits(float x);
uint16_t or_f32_to_bf16_bits(float x);

/* ---- building blocks (exposed for the pin tests) ---- */
void or_rmsnorm(int32_t d, const float *x, const void *gain, int32_t dtype,
                float eps, float *h_out);
void or_rope_cos_sin(float theta, int32_t head_dim, int32_t pair, int32_t pos,
                     float *c, float *s);
void or_rope_rotate(const or_config *c, float *vec, const int32_t pos3[3]);
void or_attention(int32_t n_t, int32_t d_h, const float *q, const float *k,
                  int64_t k_stride, const float *v, int64_t v_stride,
                  float *o_out);
float or_silu(float z);
int32_t or_argmax(int32_t n, const float *v);

/* ---- whole model ---- */
int or_seq_init(const or_model *m, or_seq *s, int32_t cap);
void or_seq_free(or_seq *s);
int or_seq_write_kv(const or_model *m, or_seq *s, int32_t layer, int32_t kv_sel,
                    int32_t head, int32_t pos0, int32_t n, const float *src);
int or_seq_read_kv(const or_model *m, const or_seq *s, int32_t layer,
                   int32_t kv_sel, int32_t head, int32_t pos0, int32_t n,
                   float *dst);
int or_seq_set_len(or_seq *s, int32_t len, int32_t rope_pos);

int or_forward_row(const or_model *m, or_seq *s, const float *x_in,
                   const int32_t pos3[3], float *hidden_out, float *logits_out);
int or_prefill(const or_model *m, or_seq *s, const void *emb, int32_t n_v,
               const int32_t *text_ids, int32_t s_text, const int32_t *pos_thw,
               float *last_logits, int32_t *first_token);
int or_decode(const or_model *m, or_seq *s, int32_t token_in, float *logits,
              float *hidden, int32_t *token_out);

#ifdef __cplusplus
}
#endif
#endif
