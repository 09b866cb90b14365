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

// Where the cache rows of request (slot) r live.  Its positions are cut into
// blocks of bt[r] positions; block k starts at element tab[toff[r] + k] of the
// cache buffer (negative: not allocated) and holds, for every (layer l, K|V s,
// KV head j), bt[r] consecutive rows of head_dim elements:
//   element(l, s, j, p, e) = tab[toff[r] + p / bt[r]]
//                            + (((l * 2 + s) * n_kv + j) * bt[r] + p % bt[r]) * head_dim + e.
// A contiguous cache is one block per request (bt = capacity).  In a decode
// step, column c is request act[c].
struct KvRef {
  void *buf;
  const int64_t *tab;
  const int *toff, *bt, *cap, *len, *act;
  int nreq, ntab;  // entries of toff / bt / cap / len, and of tab
  int paged;       // 0: one block per request (toff[r] = r, bt = cap, act[c] = c)
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
  int x_packed;          // x in the packed activation layout (packed_x_index) instead of rows
  void *h_work;          // PRO_NORM over many columns: normalised rows, model dtype [ncols][K]
  const float *part_o;   // [ncols][n_heads][n_split][head_dim]
  const float *part_ml;  // [ncols][n_heads][n_split][2]
  int n_split;
  // epilogue outputs
  void *out;    // logits fp32 / SwiGLU output / q after RoPE, row stride ld_out
  int ld_out;
  int out_packed;  // SwiGLU output in the packed activation layout (K = rows[0])
  float *resid; // residual stream fp32 [ncols][ld_resid], updated in place
  int ld_resid;
  // residual epilogue split over K: fp32 partials [k_split][ncols][rows[0]]
  // (workspace of splitk_cap floats), summed into resid in split order
  float *splitk_ws;
  int64_t splitk_cap;
  int k_split;  // set by the launcher
  // residual epilogue left to the next normalisation: the K-split partials
  // go to splitk_ws as fp64 [defer][ncols][rows[0]] (2 floats of the
  // workspace each) and resid is not touched
  int defer;
  // PRO_NORM: pending fp64 partials of the previous residual projection,
  // [pend_s][ncols][K], added into the residual rows x (which are rewritten)
  // before they are normalised
  const double *pend;
  int pend_s;
  // q/k/v epilogue: RoPE and KV append
  int head_dim, n_heads, n_kv;
  KvRef kv;
  int layer;
  int prefill;           // 0: decode (column = request, position = len); 1: prefill rows described by *pk
  const PackedRows *pk;  // device copy of the pass's rows (prefill)
  const int *rope_pos; // decode: [requests]; prefill M-RoPE: [3][rope_ld] (section-major); prefill 1-D: NULL
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
#ifndef HS_STATIC_SCRATCH_BYTES
#define HS_STATIC_SCRATCH_BYTES (64ull << 20)
#endif
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
// EPI_QKV_PAGED: the q/k/v epilogue for a cache of several blocks per request
// EPI_PART: the residual epilogue as K-split partials (GemmArgs::defer)
enum { EPI_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_QKV = 3, EPI_QKV_PAGED = 4, EPI_PART = 5 };
constexpr bool epi_qkv(int e) { return e == EPI_QKV || e == EPI_QKV_PAGED; }

struct AttnArgs {
  const void *q;
  int ld_q;
  KvRef kv;
  int layer;
  int n_heads, n_kv;
  int prefill;     // 0: decode (query = column c, request act[c], length = len + 1); 1: prefill rows in *pk
  const PackedRows *pk;  // device copy; query row r of request i has length r - cu[i] + 1
  int prefill_tiles;     // prefill: query tiles in all (pk->tcu[pk->n])
  int prefill_pairs;     // prefill: pairs of one request's consecutive query tiles, sum of ceil(tiles / 2)
  int S;           // positions per split (pooled caches: a multiple of 256)
  const int *order;  // decode: work-group row z serves column order[z] (longest first); NULL: z
  int n_split;     // splits per (query, kv head)
  float *part_o;   // [nq][n_heads][n_split][head_dim]
  float *part_ml;  // [nq][n_heads][n_split][2]
  float scale;
  int out_packed;  // out in the packed activation layout (the O projection reads it so)
  void *out;       // combined output, model dtype [nq][n_heads * head_dim]
};

hipError_t launch_gemm(int dtype, int pro, int epi, const GemmArgs &a, hipStream_t st);
// whether a GEMM over ncols columns with K-long 16-bit activations reads them
// from memory through MFMA-operand loads (2..32 columns that the LDS copy
// cannot hold); its producer then writes them in the packed activation layout
bool gemm_x_packed(int dtype, int ncols, int K);
// K splits a residual projection over K inputs leaves pending for the next
// RMSNorm over d_model (0: it adds into the residual rows itself); cap is
// the floats of the partials workspace
int resid_defer_splits(int dtype, int ncols, int K, int d_model, int64_t cap);
// x[col][0..rows) += the pending fp64 partials [k_split][ncols][rows]
// summed in split order (the sum k_rmsnorm applies), for a pass that ends
// without a normalisation
hipError_t launch_resid_pending(const double *part, int k_split, int ncols, int rows, float *x, hipStream_t st);
// elements an activation buffer of `rows` rows of K needs, the packed layout
// of up to 32 columns included
int64_t act_elems(int64_t rows, int64_t K);
// whether launch_gemm takes PRO_COMBINE for these shapes
bool gemm_combine_fusable(int dtype, int ncols, int K, int n_heads, int n_split);
hipError_t launch_pack(int dtype, const void *src, int64_t rows, int64_t cols, void *dst, int pair_hd,
                       hipStream_t st);
int64_t packed_elems(int dtype, int64_t rows, int64_t cols);
hipError_t launch_attention(int dtype, int head_dim, int group, int nq, const AttnArgs &a, hipStream_t st);
hipError_t launch_combine(int dtype, int head_dim, int nq, const AttnArgs &a, hipStream_t st);
// causal prefill attention over the packed rows of *a.pk (nrows in all), 16-bit storage; query
// tiles of 16 / group rows
int attn_prefill_rows_per_tile(int group);
bool attn_prefill_on_mma(int dtype);
hipError_t launch_attention_prefill(int dtype, int head_dim, int group, int nrows, const AttnArgs &a,
                                    hipStream_t st);
// x[c] = E[tokens[act[c]]] (act NULL: tokens[c])
hipError_t launch_embed(int dtype, const void *embed, int vocab, int d, const int *tokens, const int *act, int n,
                        float *x, int *status, hipStream_t st);
hipError_t launch_prefill_rows(int dtype, const void *emb, int n_v, const void *embed, int vocab, int d,
                               const int *ids, int s_text, float *x, int *status, hipStream_t st);
// row c's argmax to tokens_out[act[c]] (act NULL: [c]); with advance, that
// request's length and RoPE position += 1
hipError_t launch_argmax(const float *logits, int vocab, int ld, int n, int *tokens_out, const int *act, int *len,
                         int *rope_pos, int advance, hipStream_t st);
hipError_t launch_advance(int *len, int *rope_pos, const int *act, int n, hipStream_t st);
// len[req] = s_ctx, the next RoPE position, ready[req] = 1; pos_thw: [3][ld]
// section-major, this request's s_ctx columns
hipError_t launch_prefill_finish(int *len, int *rope_pos, int *ready, int req, int s_ctx, const int *pos_thw, int ld,
                                 hipStream_t st);

// Block pool of a KV handle: a stack of free block ids on the device, and per
// request the count of blocks it holds (its table entries toff[r] ..).
struct KvPool {
  int64_t *tab;
  const int *toff, *cap;
  int *len, *rope, *ready, *nblk, *stack, *top, *status;
  const int *act;
  int bt;              // positions per block
  int64_t block_elems; // elements per block
};
// requests and the lengths their blocks must cover
struct KvReserve {
  int n;
  int req[PACK_MAX];
  int target[PACK_MAX];
};
// Gives requests the blocks that cover positions [0, target): the listed ones
// (decode_n == 0), or the decode step's columns act[0 .. decode_n) with target
// len + 1 (capped at capacity).  A shortfall sets status bit 4 and leaves
// those requests' entries unallocated.
hipError_t launch_kv_reserve(const KvPool &p, const KvReserve &r, int decode_n, hipStream_t st);
// returns request req's blocks to the stack and empties it (length 0, not ready)
hipError_t launch_kv_release(const KvPool &p, int req, hipStream_t st);
// order = the n decode columns by decreasing length (ties: lower column
// first); column c is request act[c] (act NULL: c)
hipError_t launch_build_order(const int *len, const int *act, int n, int *order, hipStream_t st);
// reads bytes (a multiple of 16) from buf; one word per work group to sink[blocks]
hipError_t launch_stream_read(const void *buf, uint64_t bytes, uint32_t *sink, int blocks, hipStream_t st);
// *p = v, in stream order
hipError_t launch_set_int(int *p, int v, hipStream_t st);
// zeroes bytes (a multiple of 16, 16-byte aligned) at p, in stream order
hipError_t launch_zero(void *p, uint64_t bytes, hipStream_t st);
// act = the ready requests in order (n requests)
hipError_t launch_build_act(const int *ready, int n, int *act, hipStream_t st);
// *dst = v, in stream order (the rows of a prefill pass, for the kernels that read them)
hipError_t launch_set_packed(PackedRows *dst, const PackedRows &v, hipStream_t st);
// out[i] = x[pk.cu[i + 1] - 1] for the pk.n requests (rows of d floats)
hipError_t launch_gather_last(const float *x, int d, const PackedRows &pk, float *out, hipStream_t st);

bool attn_supported(int dtype, int head_dim, int group);

// records the thread's error message (hs_last_error) and returns code
int fail(int code, const char *fmt, ...);

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
  float *splitk = nullptr;  // [SPLITK_MAX][max_batch][max(d, q|k|v rows)] K-split GEMM partials
  int64_t splitk_floats = 0;
  float *xlast = nullptr;   // [PACK_MAX][d] last rows of the requests of a prefill pass
  hs::PackedRows *pk_dev = nullptr;  // the rows of the current prefill pass
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
  int64_t *d_base = nullptr;  // block table (contiguous: one block start per request)
  int *d_cap = nullptr, *d_len = nullptr, *d_rope = nullptr;
  int *d_toff = nullptr, *d_bt = nullptr, *d_act = nullptr, *d_ready = nullptr;
  int *d_order = nullptr;  // decode columns, longest first
  int ntab = 0;
  int n_active = 0;  // decode columns
  // block pool (handles from hs_kv_pool_create)
  bool pool = false;
  int block_tokens = 0, n_blocks = 0, max_blocks = 0, free_blocks = 0;
  int64_t block_elems = 0;
  int *d_stack = nullptr, *d_top = nullptr, *d_nblk = nullptr;
  std::vector<int> nblk;     // blocks held per request (host mirror)
  std::vector<int> act_host; // decode columns' requests (host mirror of d_act)
};
