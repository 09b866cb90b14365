// hs_internal.h — private structures of libhs shared by the host API and the
// kernel launchers.  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "hs.h"

namespace hs {

// Arguments of the weight-streaming GEMM  Y[c][n] = sum_k X[c][k] * W[n][k].
// Columns c are activation rows (decode requests or prefill rows); rows n are
// output features.  Row tiles of 16 are enumerated over up to three matrices.
// The rows of one prefill pass: up to PACK_MAX requests, their rows packed
// request by request.  Request i of the pass is KV request req[i] and owns the
// rows cu[i] .. cu[i + 1] - 1, its positions 0 .. cu[i + 1] - cu[i] - 1.
// tcu is set by the prefill attention launcher: request i's query tiles are
// tcu[i] .. tcu[i + 1] - 1.
constexpr int PACK_MAX = 32;
struct PackedRows {
  int n;
  int cu[PACK_MAX + 1];
  int req[PACK_MAX];
  int tcu[PACK_MAX + 1];
};

struct GemmArgs {
  const void *w[3];
  const void *bias[3];
  int rows[3];
  int K;
  int ncols;
  // prologue: plain activations (model dtype [ncols][K]), the fp32 residual
  // stream [ncols][K] normalised with gain[K] and eps, or the attention output
  // [ncols][n_heads * head_dim] combined from n_split split partials
  const void *x;
  const void *gain;
  float eps;
  void *h_work;          // PRO_NORM over many columns: normalised rows, model dtype [ncols][K]
  const float *part_o;   // [ncols][n_heads][n_split][head_dim]
  const float *part_ml;  // [ncols][n_heads][n_split][2]
  int n_split;
  // epilogue outputs
  void *out;    // logits fp32 / SwiGLU output / q after RoPE, row stride ld_out
  int ld_out;
  float *resid; // residual stream fp32 [ncols][ld_resid], updated in place
  int ld_resid;
  // residual epilogue split over K: fp32 partials [k_split][ncols][rows[0]]
  // (workspace of splitk_cap floats), summed into resid in split order
  float *splitk_ws;
  int64_t splitk_cap;
  int k_split;  // set by the launcher
  // q/k/v epilogue: RoPE and KV append
  int head_dim, n_heads, n_kv;
  void *kv;
  const int64_t *kv_base;
  const int *kv_cap;
  const int *kv_len;
  int layer;
  int prefill;         // 0: decode (column = request, position = len); 1: prefill rows described by pk
  PackedRows pk;
  int kv_nreq;         // entries of kv_base / kv_cap
  const int *rope_pos; // decode: [ncols]; prefill M-RoPE: [3][rope_ld] (section-major); prefill 1-D: NULL
  int rope_ld;
  int rope_m3;
  int sec0, sec1;      // M-RoPE section boundaries (pairs)
  const float *rope_tab;
  int rope_max;
  int *status;
  // set by the launcher: work groups per column group, and column groups
  int n_groups, n_colg;
};

enum { PRO_PLAIN = 0, PRO_NORM = 1, PRO_COMBINE = 2 };
// most K splits of a residual GEMM over many columns
constexpr int SPLITK_MAX = 4;
// the attention combine runs in the projection's prologue for at most this
// many splits (and activations that fit the prologue's LDS copy)
constexpr int COMBINE_FUSE_SPLITS = 8;

// waves per attention work group
constexpr int ATTN_WAVES = 4;
// position groups per batch of K/V loads of one attention wave: fewer when
// the query-head group's accumulators take more registers
constexpr int attn_batch(int group) { return group <= 2 ? 8 : 4; }
// query-head groups of 4 or more in 16-bit storage run on the matrix cores,
// in tiles of 16 positions per wave, ATTN_MMA_BATCH tiles per batch of loads
constexpr bool attn_uses_mma(int dtype, int group) { return dtype != HS_F32 && group >= 4; }
constexpr int ATTN_MMA_BATCH = 2;
constexpr int ATTN_MAX_SPLITS = 256;
enum { EPI_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_QKV = 3 };

struct AttnArgs {
  const void *q;
  int ld_q;
  const void *kv;
  const int64_t *kv_base;
  const int *kv_cap;
  const int *kv_len;
  int layer;
  int n_heads, n_kv;
  int prefill;     // 0: decode (query = request, length = len + 1); 1: prefill rows described by pk
  PackedRows pk;   // prefill: query row r of request i has length r - cu[i] + 1
  int S;           // positions per split
  int n_split;     // splits per (query, kv head)
  float *part_o;   // [nq][n_heads][n_split][head_dim]
  float *part_ml;  // [nq][n_heads][n_split][2]
  float scale;
  void *out;       // combined output, model dtype [nq][n_heads * head_dim]
};

hipError_t launch_gemm(int dtype, int pro, int epi, const GemmArgs &a, hipStream_t st);
// whether launch_gemm takes PRO_COMBINE for these shapes
bool gemm_combine_fusable(int dtype, int ncols, int K, int n_heads, int n_split);
hipError_t launch_pack(int dtype, const void *src, int64_t rows, int64_t cols, void *dst, int pair_hd,
                       hipStream_t st);
int64_t packed_elems(int dtype, int64_t rows, int64_t cols);
hipError_t launch_attention(int dtype, int head_dim, int group, int nq, const AttnArgs &a, hipStream_t st);
hipError_t launch_combine(int dtype, int head_dim, int nq, const AttnArgs &a, hipStream_t st);
// causal prefill attention over the packed rows of a.pk (nrows in all), 16-bit storage
bool attn_prefill_on_mma(int dtype);
hipError_t launch_attention_prefill(int dtype, int head_dim, int group, int nrows, const AttnArgs &a,
                                    hipStream_t st);
hipError_t launch_embed(int dtype, const void *embed, int vocab, int d, const int *tokens, int n, float *x,
                        int *status, hipStream_t st);
hipError_t launch_prefill_rows(int dtype, const void *emb, int n_v, const void *embed, int vocab, int d,
                               const int *ids, int s_text, float *x, int *status, hipStream_t st);
hipError_t launch_argmax(const float *logits, int vocab, int ld, int n, int *tokens_out, int *len, int *rope_pos,
                         int advance, hipStream_t st);
hipError_t launch_advance(int *len, int *rope_pos, int n, hipStream_t st);
// len[req] = s_ctx and the next RoPE position; pos_thw: [3][ld] section-major, this request's s_ctx columns
hipError_t launch_prefill_finish(int *len, int *rope_pos, int req, int s_ctx, const int *pos_thw, int ld,
                                 hipStream_t st);
// out[i] = x[pk.cu[i + 1] - 1] for the pk.n requests (rows of d floats)
hipError_t launch_gather_last(const float *x, int d, const PackedRows &pk, float *out, hipStream_t st);

bool attn_supported(int dtype, int head_dim, int group);

}  // namespace hs

struct hs_model {
  hs_config cfg;
  hs_weights w;
  std::vector<hs_layer_weights> layers;
  int device = 0;
  int max_batch = 0, max_ctx = 0;
  int64_t rows = 0;         // capacity of the row workspaces below (max_rows)
  int64_t part_entries = 0; // capacity of the attention partial buffers in (query, head, split) entries
  // workspaces (device)
  float *x = nullptr;       // [max_rows][d] residual stream
  void *q = nullptr;        // [max_rows][n_h * d_h] q after RoPE
  void *attn = nullptr;     // [max_rows][n_h * d_h] attention output
  void *act = nullptr;      // [max_rows][F] SwiGLU output
  void *hnorm = nullptr;    // [max_rows][d] normalised rows for GEMMs over many columns
  float *splitk = nullptr;  // [SPLITK_MAX][max_batch][d] residual GEMM partials
  int64_t splitk_floats = 0;
  float *xlast = nullptr;   // [PACK_MAX][d] last rows of the requests of a prefill pass
  float *logits = nullptr;  // [max_batch][V] (used when the caller passes no logits buffer)
  float *part_o = nullptr;
  float *part_ml = nullptr;
  float *rope_tab = nullptr; // [max_ctx][d_h / 2][2]
  int *status = nullptr;
};

struct hs_kv {
  hs_model *m = nullptr;
  int batch = 0;
  void *buf = nullptr;
  uint64_t buf_bytes = 0;
  std::vector<int> n_v, cap, len, rope;
  std::vector<int64_t> base;
  std::vector<char> ready;
  int max_cap = 0;
  int64_t *d_base = nullptr;
  int *d_cap = nullptr, *d_len = nullptr, *d_rope = nullptr;
};
