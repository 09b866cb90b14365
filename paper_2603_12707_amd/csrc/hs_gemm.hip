// hs_gemm.hip — weight-streaming MFMA GEMM of the decode step (gfx950) and the
// packing of weight matrices into the layout it streams.
//
// Decode reads every weight byte once per generated token (§2; Eq. 5 of §4.3
// models decode time as the streamed weight bytes over HBM bandwidth), so the
// GEMM is organised as one sequential pass over a packed copy of each matrix:
// a 16-row x 256-byte tile slice is stored as 1 KB in MFMA lane order, so that
// every wave-wide load instruction reads 1 KB of contiguous HBM.
#include "hs_device.h"

#include <algorithm>

namespace hs {
namespace {

using namespace dev;

// ---------------------------------------------------------------------------
// packed layout
// ---------------------------------------------------------------------------
// A row-major [N, K] matrix becomes tiles of 16 rows; each tile is a sequence
// of k-blocks of 16 chunks (16 x CE elements, 256 bytes per row); k-block kb
// of tile t is four 1 KB sub-blocks s, and lane l = 16 * lq + li of sub-block
// s holds the 16-byte chunk kc = 16 * kb + 4 * s + lq of row 16 * t + li.
// Rows past N and chunks past K are zero.  With pair_hd > 0 the rows form
// heads of pair_hd rows, and packed row 2 j of a head holds its row j,
// packed row 2 j + 1 its row j + pair_hd / 2 (the two rows RoPE rotates
// together end up in the same lane of an MFMA output tile).
template <int DT>
__global__ __launch_bounds__(256) void k_pack(const void *src, void *dst, int64_t N, int K, int nkb,
                                              int64_t total, int pair_hd) {
  constexpr int CE = Ty<DT>::CE;
  using S = typename Ty<DT>::S;
  for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int lane = (int)(i & 63), s = (int)((i >> 6) & 3);
    const int64_t rest = i >> 8;
    const int kb = (int)(rest % nkb);
    const int64_t tile = rest / nkb;
    int64_t row = tile * 16 + (lane & 15);
    if (pair_hd > 0) {
      const int64_t head = row / pair_hd;
      const int p = (int)(row - head * pair_hd);
      row = head * pair_hd + ((p & 1) ? pair_hd / 2 + p / 2 : p / 2);
    }
    const int kc = kb * 16 + s * 4 + (lane >> 4);
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (row < N && (int64_t)kc * CE < K) v = ld16((const S *)src + row * K + (int64_t)kc * CE);
    *(u32x4 *)((S *)dst + i * CE) = v;
  }
}

// ---------------------------------------------------------------------------
// row tiles
// ---------------------------------------------------------------------------
// q/k/v: R consecutive tiles of the q, k, v matrices taken in turn (their
// rows packed in head-paired order); SwiGLU pairs row j of the gate and of
// the up projection; the other epilogues take R consecutive tiles.
// rows of a K-split GEMM's partials: the residual rows, or q|k|v rows in turn
__host__ __device__ inline int split_rows(const GemmArgs &a, int epi) {
  return epi_qkv(epi) ? (a.n_heads + 2 * a.n_kv) * a.head_dim : a.rows[0];
}

template <int EPI, int R>
__device__ __forceinline__ void tile_map(const GemmArgs &a, int g, int *mat, int *row0) {
  if constexpr (epi_qkv(EPI)) {
    const int tq = a.n_heads * a.head_dim / 16, tk = a.n_kv * a.head_dim / 16;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      int m = 0, t = g * R + r;
      if (t >= tq) {
        t -= tq;
        m = 1;
        if (t >= tk) {
          t -= tk;
          m = 2;
        }
      }
      mat[r] = m;
      row0[r] = 16 * t;  // past the v rows for a partial last group
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    mat[0] = 0;
    mat[1] = 1;
    row0[0] = row0[1] = 16 * g;
  } else {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      mat[r] = 0;
      row0[r] = 16 * (R * g + r);
    }
  }
}

// PK: the SwiGLU output goes to the packed activation layout where a.out_packed
// says so (the down projection reads it so, which happens at 2..32 columns,
// the widths k_gemm serves; the kernels for wider GEMMs never write it)
template <int DT, int EPI, int R, bool PK = false>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs &a, const int *mat, const int *row0, const f32x4 *v,
                                              int col, int rr) {
  if constexpr (EPI == EPI_STORE) {
    float *o = (float *)a.out + (int64_t)col * a.ld_out;
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = row0[r] + rr + e;
        if (row < a.rows[mat[r]]) o[row] = v[r][e];
      }
  } else if constexpr (EPI == EPI_RESID) {
    float *x = a.resid + (int64_t)col * a.ld_resid;
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = row0[r] + rr + e;
        if (row < a.rows[mat[r]]) x[row] += v[r][e];
      }
  } else if constexpr (EPI == EPI_SWIGLU) {
    const bool packed = PK && a.out_packed;
    const int nkb_o = (a.rows[0] / 8 + 15) / 16;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int j = row0[0] + rr + e;
      if (j < a.rows[0]) {
        const float g = v[0][e], u = v[1][e];
        const int64_t at = packed ? packed_x_index(col, j, nkb_o) : (int64_t)col * a.ld_out + j;
        st_elem<DT>(a.out, at, g / (1.0f + expf(-g)) * u);
      }
    }
  }
}

// q/k/v epilogue inputs of one thread (one output column, packed rows
// rr..rr+3 of each of its R tiles: RoPE pairs (j, j + d_h/2) and
// (j + 1, j + 1 + d_h/2)), read ahead of the main loop: the KV position,
// capacity and base of the column's request and the RoPE position of each
// pair first; the cos/sin entries and the biases once those positions are in.
// Every read goes through a buffer range, so none sits behind a branch.
template <int R>
struct QkvIn {
  int pos, cap, bt;
  int64_t base;  // start of the block holding pos (negative: none)
  int p[R][2];
  float cs[R][2], sn[R][2], b1[R][2], b2[R][2];
};

template <int DT, int R, bool PAGED>
__device__ __forceinline__ void qkv_fetch_ids(const GemmArgs &a, const int *mat, const int *row0, int col, int rr,
                                              bool ok, QkvIn<R> &in) {
  const bool dec = !a.prefill;
  const KvRef &kv = a.kv;
  // decode: column col is request act[col]; prefill: the packed row's request
  // and its position in that request
  int req = 0, ppos = 0;
  if (!dec) {
    const int i = packed_request(a.pk, col);
    req = a.pk->req[i];
    ppos = col - a.pk->cu[i];
  }
  const uint32_t nb = (uint32_t)kv.nreq * 4u;
  if constexpr (PAGED) {
    const rsrc_t ar = make_rsrc(kv.act, dec ? (uint32_t)a.ncols * 4u : 0u);
    if (dec) req = (int)bld4(ar, ok ? (uint32_t)col * 4u : BUF_OOB);
  } else if (dec) {
    req = col;
  }
  const rsrc_t lr = make_rsrc(kv.len, dec ? nb : 0u), cr = make_rsrc(kv.cap, nb);
  const rsrc_t br = make_rsrc(kv.tab, (uint32_t)kv.ntab * 8u);
  const rsrc_t pr = make_rsrc(a.rope_pos, dec ? nb : (a.rope_m3 ? 3u * a.rope_ld * 4u : 0u));
  const uint32_t ro = ok ? (uint32_t)req * 4u : BUF_OOB;
  const uint32_t pl = bld4(lr, dec ? ro : BUF_OOB);
  in.cap = (int)bld4(cr, ro);
  if constexpr (PAGED) {  // the block holding the position
    const rsrc_t or_ = make_rsrc(kv.toff, nb), tr = make_rsrc(kv.bt, nb);
    const int toff = (int)bld4(or_, ro);
    in.bt = max(1, (int)bld4(tr, ro));
    in.pos = dec ? (int)pl : ppos;
    const u32x2 bb = bld8(br, ok && in.pos < in.cap ? (uint32_t)(toff + in.pos / in.bt) * 8u : BUF_OOB);
    in.base = ok && in.pos < in.cap ? (int64_t)(((uint64_t)bb[1] << 32) | bb[0]) : -1;
  } else {  // one block per request: its start, read beside the length
    const u32x2 bb = bld8(br, ok ? (uint32_t)req * 8u : BUF_OOB);
    in.bt = in.cap;
    in.pos = dec ? (int)pl : ppos;
    in.base = ok && in.pos < in.cap ? (int64_t)(((uint64_t)bb[1] << 32) | bb[0]) : -1;
  }
  const int hd = a.head_dim;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int j0 = (row0[r] % hd + rr) >> 1;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int i = j0 + e, sec = i < a.sec0 ? 0 : (i < a.sec1 ? 1 : 2);
      const bool rot = ok && mat[r] < 2 && (dec || a.rope_m3);
      const uint32_t pv = bld4(pr, rot ? (uint32_t)(dec ? req : sec * a.rope_ld + col) * 4u : BUF_OOB);
      in.p[r][e] = (dec || a.rope_m3) ? (int)pv : in.pos;
    }
  }
}

template <int DT, int R>
__device__ __forceinline__ void qkv_fetch_tab(const GemmArgs &a, const int *mat, const int *row0, int rr, bool ok,
                                              QkvIn<R> &in) {
  const int hd = a.head_dim, half = hd >> 1;
  const rsrc_t tr = make_rsrc(a.rope_tab, (uint32_t)a.rope_max * half * 8u);
  constexpr int SB = DT == HS_F32 ? 4 : 2;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int m = mat[r], head = row0[r] / hd, j0 = (row0[r] - head * hd + rr) >> 1;
    const bool live = ok && row0[r] < a.rows[m];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int p = min(max(in.p[r][e], 0), a.rope_max - 1);
      const u32x2 t = bld8(tr, live && m < 2 ? (uint32_t)(p * half + j0 + e) * 8u : BUF_OOB);
      in.cs[r][e] = __uint_as_float(t[0]);
      in.sn[r][e] = __uint_as_float(t[1]);
    }
    const rsrc_t bq = make_rsrc(a.bias[m], a.bias[m] ? (uint32_t)a.rows[m] * SB : 0u);
    const uint32_t o1 = (uint32_t)(head * hd + j0) * SB, o2 = (uint32_t)(head * hd + half + j0) * SB;
    if constexpr (DT == HS_F32) {
      const u32x2 v1 = bld8(bq, live ? o1 : BUF_OOB), v2 = bld8(bq, live ? o2 : BUF_OOB);
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        in.b1[r][e] = __uint_as_float(v1[e]);
        in.b2[r][e] = __uint_as_float(v2[e]);
      }
    } else {
      const uint32_t v1 = bld4(bq, live ? o1 : BUF_OOB), v2 = bld4(bq, live ? o2 : BUF_OOB);
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const uint32_t h1 = (v1 >> (16 * e)) & 0xFFFFu, h2 = (v2 >> (16 * e)) & 0xFFFFu;
        in.b1[r][e] = DT == HS_F16 ? f16_to_f32(h1) : bf16_to_f32(h1);
        in.b2[r][e] = DT == HS_F16 ? f16_to_f32(h2) : bf16_to_f32(h2);
      }
    }
  }
}

// bias, RoPE on q and k, then R(q) to the q workspace and k, v rows appended
// to the cache at the request's position
template <int DT, int R, bool PAGED>
__device__ __forceinline__ void qkv_store(const GemmArgs &a, const int *mat, const int *row0, const f32x4 *v, int col,
                                          int rr, const QkvIn<R> &in) {
  constexpr int B = DT == HS_F32 ? 4 : 2;
  const int hd = a.head_dim, half = hd >> 1;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int m = mat[r];
    if (row0[r] >= a.rows[m]) continue;
    const int head = row0[r] / hd, j0 = (row0[r] - head * hd + rr) >> 1;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int i = j0 + e;  // frequency pair, < d_h / 2
      const float v1 = v[r][2 * e] + in.b1[r][e], v2 = v[r][2 * e + 1] + in.b2[r][e];
      float o1 = v1, o2 = v2;
      if (m < 2) {
        o1 = v1 * in.cs[r][e] - v2 * in.sn[r][e];
        o2 = v2 * in.cs[r][e] + v1 * in.sn[r][e];
      }
      if (m == 0) {
        void *q = (char *)a.out + ((int64_t)col * a.ld_out + head * hd) * B;
        st_elem<DT>(q, i, o1);
        st_elem<DT>(q, i + half, o2);
      } else if (in.base >= 0) {
        const int pin = PAGED ? in.pos % in.bt : in.pos;  // position within its block
        const int64_t off = in.base + ((int64_t)((a.layer * 2 + (m == 2 ? 1 : 0)) * a.n_kv + head) * in.bt + pin) * hd;
        st_elem<DT>(a.kv.buf, off + i, o1);
        st_elem<DT>(a.kv.buf, off + i + half, o2);
      }
    }
  }

}

// fp64 sum over the 64 lanes of a wave; every lane gets it.
__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

// fp64 sum over the 64 * NW threads of a work group; every thread gets it.
template <int NW>
__device__ __forceinline__ double block_sum(double v, double *s_part) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  v = wave_sum_f64(v);
  __syncthreads();
  if (lane == 0) s_part[wave] = v;
  __syncthreads();
  double t = 0.0;
#pragma unroll
  for (int w = 0; w < NW; ++w) t += s_part[w];
  return t;
}

__device__ __forceinline__ double sumsq_f64(f32x4 v) {
  return (double)v[0] * v[0] + (double)v[1] * v[1] + (double)v[2] * v[2] + (double)v[3] * v[3];
}

// Normalised activations h = x * rs * gain for the 4 consecutive k values of
// one float4 of x, rounded to the storage dtype and written to the LDS copy.
template <int DT>
__device__ __forceinline__ void put_h(unsigned char *s_x, int64_t at, f32x4 v, float rs, const float *g) {
  float h[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) h[e] = v[e] * rs * g[e];
  if constexpr (DT == HS_F32) {
    *(f32x4 *)((float *)s_x + at) = f32x4{h[0], h[1], h[2], h[3]};
  } else {
    uint32_t w0, w1;
    if constexpr (DT == HS_F16) {
      w0 = f32_to_f16(h[0]) | (f32_to_f16(h[1]) << 16);
      w1 = f32_to_f16(h[2]) | (f32_to_f16(h[3]) << 16);
    } else {
      w0 = f32_to_bf16(h[0]) | (f32_to_bf16(h[1]) << 16);
      w1 = f32_to_bf16(h[2]) | (f32_to_bf16(h[3]) << 16);
    }
    *(u32x2 *)((uint16_t *)s_x + at) = u32x2{w0, w1};
  }
}

// 4 gain values starting at element k (k a multiple of 4)
template <int DT>
__device__ __forceinline__ void gain4(rsrc_t gr, int k, bool ok, float *g) {
  if constexpr (DT == HS_F32) {
    const u32x4 v = bld16(gr, ok ? (uint32_t)k * 4u : BUF_OOB);
#pragma unroll
    for (int e = 0; e < 4; ++e) g[e] = __uint_as_float(v[e]);
  } else {
    const u32x2 v = bld8(gr, ok ? (uint32_t)k * 2u : BUF_OOB);
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      g[2 * e] = DT == HS_F16 ? f16_to_f32(v[e] & 0xFFFFu) : bf16_to_f32(v[e] & 0xFFFFu);
      g[2 * e + 1] = DT == HS_F16 ? f16_to_f32(v[e] >> 16) : bf16_to_f32(v[e] >> 16);
    }
  }
}

// RMSNorm of fp32 residual rows into the storage dtype, one work group per
// row: h = R(x * rs * gain), rs = 1 / sqrt(mean(x^2) + eps) with the sum of
// squares in fp64 -- the normalisation the GEMM prologue applies when it
// stages its columns itself, done once for GEMMs over more columns.  The
// row's first 4096 elements and their gains are requested together and stay
// in registers from the sum of squares to the scaling (one memory round trip);
// a longer row reads the rest twice.
// PS > 0: the previous residual projection left its PS K-split partials
// pend[s][row][k] in fp64; x + R32(p_0 + ... + p_{PS-1}) (summed in split
// order in fp64, rounded once: the rounding of the projection's own residual
// epilogue) is the residual row, written back to x and normalised.  The
// longer-row passes recompute it rather than read back what this thread
// stored.
template <int DT, int PS>
__global__ __launch_bounds__(256) void k_rmsnorm(float *x, const void *gain, float eps, int K, void *h, int packed,
                                                const double *pend, int ncols) {
  constexpr int NV = 4;  // 16-byte chunks per thread held in registers
  constexpr int SB = DT == HS_F32 ? 4 : 2;
  float *xr = x + (int64_t)blockIdx.x * K;
  const rsrc_t xq = make_rsrc(xr, (uint32_t)K * 4u);
  const rsrc_t gr = make_rsrc(gain, (uint32_t)K * SB);
  rsrc_t pq[PS > 0 ? PS : 1];
#pragma unroll
  for (int s = 0; s < PS; ++s) pq[s] = make_rsrc(pend + ((int64_t)s * ncols + blockIdx.x) * K, (uint32_t)K * 8u);
  // partials of elements k..k+3: two 16-byte loads per split
  using P4 = u32x4[2];
  auto pend4 = [&](int k, bool ok, P4 (&p)[PS > 0 ? PS : 1]) {
#pragma unroll
    for (int s = 0; s < PS; ++s)
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) p[s][hf] = bld16(pq[s], ok ? (uint32_t)k * 8u + hf * 16u : BUF_OOB);
  };
  // the residual row's elements k..k+3 (in range: k < K)
  auto row4 = [&](f32x4 v, const P4 (&p)[PS > 0 ? PS : 1]) -> f32x4 {
    if constexpr (PS > 0) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        double t = 0.0;
#pragma unroll
        for (int s = 0; s < PS; ++s) {
          const uint32_t lo = p[s][e >> 1][2 * (e & 1)], hi = p[s][e >> 1][2 * (e & 1) + 1];
          const double d = __builtin_bit_cast(double, (uint64_t)lo | ((uint64_t)hi << 32));
          t = s ? t + d : d;
        }
        v[e] += (float)t;
      }
    }
    return v;
  };
  __shared__ double s_part[4];
  f32x4 xv[NV];
  P4 pv[NV][PS > 0 ? PS : 1];
  float gv[NV][4];
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    const int k = (u * 256 + (int)threadIdx.x) * 4;
    xv[u] = __builtin_bit_cast(f32x4, bld16(xq, k < K ? (uint32_t)k * 4u : BUF_OOB));
    pend4(k, k < K, pv[u]);
    gain4<DT>(gr, k, k < K, gv[u]);
  }
#pragma unroll
  for (int u = 0; u < NV; ++u) xv[u] = row4(xv[u], pv[u]);  // zeros past K
  double ss = 0.0;
#pragma unroll
  for (int u = 0; u < NV; ++u) ss += sumsq_f64(xv[u]);
  for (int k = (NV * 256 + (int)threadIdx.x) * 4; k < K; k += 1024) {
    P4 p[PS > 0 ? PS : 1];
    pend4(k, true, p);
    ss += sumsq_f64(row4(*(const f32x4 *)(xr + k), p));
  }
  const float rs = (float)(1.0 / sqrt(block_sum<4>(ss, s_part) / (double)K + (double)eps));
  const int nkb = (K / 8 + 15) / 16;
  // (packed: the 4 elements stay consecutive, k being a multiple of 4)
  auto at = [&](int k) { return packed ? packed_x_index((int)blockIdx.x, k, nkb) : (int64_t)blockIdx.x * K + k; };
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    const int k = (u * 256 + (int)threadIdx.x) * 4;
    if (k < K) {
      if constexpr (PS > 0) *(f32x4 *)(xr + k) = xv[u];
      put_h<DT>((unsigned char *)h, at(k), xv[u], rs, gv[u]);
    }
  }
  for (int k = (NV * 256 + (int)threadIdx.x) * 4; k < K; k += 1024) {
    float g[4];
    gain4<DT>(gr, k, true, g);
    P4 p[PS > 0 ? PS : 1];
    pend4(k, true, p);
    const f32x4 v = row4(*(const f32x4 *)(xr + k), p);
    if constexpr (PS > 0) *(f32x4 *)(xr + k) = v;
    put_h<DT>((unsigned char *)h, at(k), v, rs, g);
  }
}

// Y[c][n] = sum_k X[c][k] W[n][k] over R row tiles and NT column tiles of 16.
//
// The NW waves of a work group split the packed k-blocks round robin, so that
// together they read consecutive kilobytes.  Each wave keeps a ring of two
// groups of U k-blocks of weight loads in flight (non-temporal: every weight
// byte is read once per step); a group is refilled as soon as its MFMAs are
// issued.  The loads are raw buffer reads whose ranges end where the data
// ends, so that no load sits behind a branch; the ring runs a whole number
// of rounds, and groups past the wave's last k-block read zeros.
// X comes from a copy in LDS (XS = 1: the work group's columns are few; with
// PRO_NORM the copy holds the normalised activations, with the first column's
// x requested before the weights; with PRO_COMBINE the attention output
// rebuilt from its split partials), or from the activation rows in global
// memory (PRO_PLAIN, XS = 0), requested with the weights.  The waves' partial
// tiles are summed in a fixed order through LDS and handed to the epilogue.
// PK: the SwiGLU output in the packed layout; XP: activations read from
// memory in the packed layout (a.out_packed, a.x_packed).
// EPI_PART: work group b takes the k-blocks of split b mod a.k_split (a
// contiguous range, the splits as equal as whole k-blocks allow) of row
// group b / a.k_split and stores its tile, summed in fp64, as that split's
// fp64 partial.
template <int DT, int R, int NT, int NW, int U, int PRO, int XS, int EPI, bool PK, bool XP>
__global__ __launch_bounds__(64 * NW) void k_gemm(GemmArgs a) {
  static_assert(PRO == PRO_PLAIN || XS == 1, "only plain activations are read from global memory");
  using S = typename Ty<DT>::S;
  constexpr int CE = Ty<DT>::CE;
  constexpr int SB = (int)sizeof(S);
  constexpr int D = 2;  // groups of weight loads in flight per wave
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int li = lane & 15, lq = lane >> 4;
  // The kernel arguments the first loads are built from, fetched in one
  // round trip (fetched where first read, behind the column-group branch,
  // they took three before the first weight load).
  {
    const int n_colg = a.n_colg, n_groups = a.n_groups, K0 = a.K, ncols = a.ncols;
    const int r0 = a.rows[0], r1 = a.rows[1], r2 = a.rows[2];
    const void *w0 = a.w[0], *w1 = a.w[1], *w2 = a.w[2], *x = a.x, *gain = a.gain;
    asm volatile("" ::"s"(n_colg), "s"(n_groups), "s"(K0), "s"(ncols), "s"(r0), "s"(r1), "s"(r2), "s"(w0), "s"(w1),
                 "s"(w2), "s"(x), "s"(gain));
    if constexpr (epi_qkv(EPI) || PRO == PRO_COMBINE) {  // the q/k/v row map; the split partials
      const int hd = a.head_dim, nh = a.n_heads, nkv = a.n_kv, nsp = a.n_split;
      const float *po = a.part_o, *pm = a.part_ml;
      asm volatile("" ::"s"(hd), "s"(nh), "s"(nkv), "s"(nsp), "s"(po), "s"(pm));
    }
  }
  // Over several column groups the grid is one-dimensional and ordered so
  // that the column groups of a row group take consecutive slots of one XCD
  // (work groups are dealt to the 8 XCDs round robin): the later groups then
  // read the row group's weights from that XCD's L2 instead of HBM.
  int grp = blockIdx.x, cgi = 0;
  if (a.n_colg > 1) {
    const int slot = (int)blockIdx.x >> 3;
    cgi = slot % a.n_colg;
    grp = (slot / a.n_colg) * 8 + ((int)blockIdx.x & 7);
    if (grp >= a.n_groups) return;
  }
  const int col0 = cgi * 16 * NT;
  const int K = a.K, kchunks = K / CE, nkb = (kchunks + 15) >> 4;
  const int nst = min(a.ncols - col0, 16 * NT);
  // the k-blocks [kb_lo, kb_hi) of this work group
  int sp = 0, kb_lo = 0, kb_hi = nkb;
  if constexpr (EPI == EPI_PART) {
    const int ks = a.k_split, per = (nkb + ks - 1) / ks;
    sp = grp % ks;
    grp /= ks;
    kb_lo = min(nkb, sp * per);
    kb_hi = min(nkb, kb_lo + per);
  }

  int mat[R], row0[R];
  tile_map<EPI, R>(a, grp, mat, row0);
  // one range per row tile: its packed k-blocks (4 KB each); empty past the matrix
  rsrc_t wr[R];
#pragma unroll
  for (int r = 0; r < R; ++r)
    wr[r] = make_rsrc((const S *)a.w[mat[r]] + (int64_t)(row0[r] >> 4) * nkb * 256 * CE,
                      row0[r] < a.rows[mat[r]] ? (uint32_t)nkb * 4096u : 0u);
  // group g of this wave: k-blocks kb_lo + wave + (g * U + u) * NW
  auto load_w = [&](u32x4 (&wv)[U][R][4], int g) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kb = kb_lo + wave + (g * U + u) * NW;
      const uint32_t off = kb < kb_hi ? (uint32_t)kb * 4096u + (uint32_t)lane * 16u : BUF_OOB;
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int r = 0; r < R; ++r) wv[u][r][s] = bld16_stream(wr[r], off + s * 1024u);
    }
  };

  const rsrc_t gr = make_rsrc(a.gain, PRO == PRO_NORM ? (uint32_t)K * SB : 0u);
  // x of the work group's columns: fp32 residual rows (PRO_NORM) or activation rows
  const rsrc_t xr = PRO == PRO_NORM ? make_rsrc((const float *)a.x + (int64_t)col0 * K, (uint32_t)nst * K * 4u)
                    : XP          ? make_rsrc((const S *)a.x + (int64_t)(col0 >> 4) * nkb * 256 * CE,
                                              (uint32_t)((nst + 15) >> 4) * nkb * 4096u)
                                  : make_rsrc((const S *)a.x + (int64_t)col0 * K, (uint32_t)nst * K * SB);
  __shared__ double s_part[NW];
  extern __shared__ __align__(16) unsigned char s_x[];  // XS: activations [nst][K]

  // requested before the weights so that the prologue waits for them alone
  constexpr int PER = 4;
  f32x4 xv[PER];
  float gv[PER][4];
  u32x4 xc[PER];
  // PRO_COMBINE: float4 item i of the staged activations is elements
  // k = 4 (i mod K/4) .. +3 of column i / (K/4), i.e. of head k / head_dim.
  // The split weights e^(m_s - M) and the denominator of each (column, head)
  // pair are computed once, by thread `pair`, into LDS.
  constexpr int PERC = 2, NSF = COMBINE_FUSE_SPLITS;
  f32x4 co[PRO == PRO_COMBINE ? PERC : 1][NSF];
  float cm[NSF], cl[NSF];
  const int ns = a.n_split, hd = a.head_dim;
  const int npair = nst * a.n_heads;
  const rsrc_t por = make_rsrc(a.part_o + (int64_t)col0 * a.n_heads * ns * hd,
                               PRO == PRO_COMBINE ? (uint32_t)npair * ns * hd * 4u : 0u);
  const rsrc_t pmr = make_rsrc(a.part_ml + (int64_t)col0 * a.n_heads * ns * 2,
                               PRO == PRO_COMBINE ? (uint32_t)npair * ns * 8u : 0u);
  __shared__ float s_cw[PRO == PRO_COMBINE ? 64 * NW : 1][NSF + 1];  // weights, then the denominator
  auto combine_load = [&](int item, f32x4 (&o)[NSF]) {
    const int c = item / (K / 4), k = (item - c * (K / 4)) * 4;
    const int h = k / hd, e = k - h * hd;
    const bool ok = item < nst * (K / 4);
    const int base = (c * a.n_heads + h) * ns;
#pragma unroll
    for (int sp = 0; sp < NSF; ++sp)
      o[sp] = __builtin_bit_cast(f32x4, bld16(por, ok && sp < ns ? (uint32_t)((base + sp) * hd + e) * 4u : BUF_OOB));
  };
  auto combine_ml = [&]() {
    const int pair = threadIdx.x;
#pragma unroll
    for (int sp = 0; sp < NSF; ++sp) {
      const u32x2 ml = bld8(pmr, pair < npair && sp < ns ? (uint32_t)(pair * ns + sp) * 8u : BUF_OOB);
      cm[sp] = __uint_as_float(ml[0]);
      cl[sp] = __uint_as_float(ml[1]);
    }
  };
  // M = max_s m_s, w_s = e^(m_s - M), den = sum_s w_s l_s in split order (the
  // arithmetic of the separate combine kernel)
  auto combine_weights = [&]() {
    const int pair = threadIdx.x;
    if (pair >= npair) return;
    float M = -INFINITY;
#pragma unroll
    for (int sp = 0; sp < NSF; ++sp)
      if (sp < ns) M = fmaxf(M, cm[sp]);
    float den = 0.f;
#pragma unroll
    for (int sp = 0; sp < NSF; ++sp)
      if (sp < ns) {
        const float w = expf(cm[sp] - M);
        s_cw[pair][sp] = w;
        den += w * cl[sp];
      }
    s_cw[pair][NSF] = den;
  };
  // o = sum_s w_s o_s / den, rounded to the storage dtype
  auto combine_store = [&](int item, const f32x4 (&o)[NSF]) {
    if (item >= nst * (K / 4)) return;
    const int c = item / (K / 4), h = (item - c * (K / 4)) * 4 / hd;
    const float *w = s_cw[c * a.n_heads + h];
    float num[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int sp = 0; sp < NSF; ++sp)
      if (sp < ns)
#pragma unroll
        for (int e = 0; e < 4; ++e) num[e] += w[sp] * o[sp][e];
    float h4[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) h4[e] = num[e] / w[NSF];
    const int64_t at = (int64_t)item * 4;  // staged rows are contiguous [nst][K]
    if constexpr (DT == HS_F32) {
      *(f32x4 *)((float *)s_x + at) = f32x4{h4[0], h4[1], h4[2], h4[3]};
    } else {
      uint32_t w0, w1;
      if constexpr (DT == HS_F16) {
        w0 = f32_to_f16(h4[0]) | (f32_to_f16(h4[1]) << 16);
        w1 = f32_to_f16(h4[2]) | (f32_to_f16(h4[3]) << 16);
      } else {
        w0 = f32_to_bf16(h4[0]) | (f32_to_bf16(h4[1]) << 16);
        w1 = f32_to_bf16(h4[2]) | (f32_to_bf16(h4[3]) << 16);
      }
      *(u32x2 *)((uint16_t *)s_x + at) = u32x2{w0, w1};
    }
  };
  if constexpr (XS == 1 && PRO == PRO_NORM) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int k = (u * 64 * NW + (int)threadIdx.x) * 4;
      xv[u] = __builtin_bit_cast(f32x4, bld16(xr, k < K ? (uint32_t)k * 4u : BUF_OOB));
      gain4<DT>(gr, k, k < K, gv[u]);
    }
  } else if constexpr (PRO == PRO_COMBINE) {
    // split maxima and sums of one (column, head) pair per thread, and the
    // split partials of the first PERC float4 items of every thread
    combine_ml();
#pragma unroll
    for (int i = 0; i < PERC; ++i) combine_load(i * 64 * NW + (int)threadIdx.x, co[i]);
  } else if constexpr (XS == 1) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int i = u * 64 * NW + (int)threadIdx.x;  // 16-byte chunk of the staged rows
      xc[u] = bld16(xr, i < nst * kchunks ? (uint32_t)i * 16u : BUF_OOB);
    }
  }

  // chunk kc of column 16 t + li of the work group; zero past the data
  auto load_x = [&](int t, int kc) -> u32x4 {
    const int c = 16 * t + li;
    const bool ok = c < nst && kc < kchunks;
    if constexpr (XS == 1) {
      const u32x4 v = *(const u32x4 *)((const S *)s_x + (ok ? (int64_t)c * K + (int64_t)kc * CE : 0));
      return ok ? v : u32x4{0u, 0u, 0u, 0u};
    } else {
      // packed: chunk kc of column tile col0 / 16 + t is lane 16 * (kc mod 4) + li
      // of sub-block kc / 4
      const uint32_t at = XP ? ((((uint32_t)(t * nkb) + (uint32_t)(kc >> 4)) * 4u + (uint32_t)((kc >> 2) & 3)) * 64u +
                                (uint32_t)((kc & 3) * 16 + li)) * 16u
                             : (uint32_t)(c * K + kc * CE) * SB;
      return bld16(xr, ok ? at : BUF_OOB);
    }
  };

  // activations from global memory at two column tiles or fewer travel in a
  // ring of their own, each group's chunks requested just before its weights
  constexpr bool XRING = XS == 0 && NT <= 2;
  u32x4 xq[XRING ? D : 1][U][NT][4];
  auto load_xg = [&](u32x4 (&xv)[U][NT][4], int g) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kb = kb_lo + wave + (g * U + u) * NW;
      // past the split's range: past the data (zeros, like the weights)
      const int kc0 = EPI != EPI_PART || kb < kb_hi ? kb * 16 : kchunks;
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int t = 0; t < NT; ++t) xv[u][t][s] = load_x(t, kc0 + s * 4 + lq);
    }
  };
  // residual epilogue: the 4 rows of x this thread adds into, read now (no
  // other work group writes them) so the epilogue does not wait for them
  constexpr bool XPRE = EPI == EPI_RESID && R == 1 && NT * 64 <= 64 * NW;
  f32x4 xres = f32x4{0.f, 0.f, 0.f, 0.f};
  if constexpr (XPRE) {
    const int it = (int)threadIdx.x, c = 16 * (it >> 6) + (it & 15), rr = 4 * ((it & 63) >> 4);
    const rsrc_t xrr = make_rsrc(a.resid, (uint32_t)a.ncols * a.ld_resid * 4u);
    xres = __builtin_bit_cast(
        f32x4, bld16(xrr, it < NT * 64 && col0 + c < a.ncols ? (uint32_t)((col0 + c) * a.ld_resid + row0[0] + rr) * 4u
                                                              : BUF_OOB));
  }

  // q/k/v epilogue: ids now, table entries and biases after the prologue
  static_assert(!epi_qkv(EPI) || NT * 64 <= 64 * NW, "one epilogue item per thread");
  QkvIn<R> qin;
  const int ep_col = col0 + 16 * ((int)threadIdx.x >> 6) + ((int)threadIdx.x & 15);
  const int ep_rr = 4 * (((int)threadIdx.x & 63) >> 4);
  const bool ep_ok = (int)threadIdx.x < NT * 64 && ep_col < a.ncols;
  if constexpr (epi_qkv(EPI)) qkv_fetch_ids<DT, R, EPI == EPI_QKV_PAGED>(a, mat, row0, ep_col, ep_rr, ep_ok, qin);

  u32x4 w[D][U][R][4];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    if constexpr (XRING) load_xg(xq[d], d);
    load_w(w[d], d);
  }

  if constexpr (PRO == PRO_NORM && XS == 1) {
    // one pass over each staged column; the first column's x (already
    // requested) stays in registers between its sum of squares and its
    // scaling, in the same straight-line code as its loads
    auto stage = [&](int c) {
      double ss = 0.0;
#pragma unroll
      for (int u = 0; u < PER; ++u) ss += sumsq_f64(xv[u]);
      for (int k = (PER * 64 * NW + (int)threadIdx.x) * 4; k < K; k += 256 * NW)  // columns longer than one pass
        ss += sumsq_f64(__builtin_bit_cast(f32x4, bld16(xr, (uint32_t)(c * K + k) * 4u)));
      const float rs = (float)(1.0 / sqrt(block_sum<NW>(ss, s_part) / (double)K + (double)a.eps));
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const int k = (u * 64 * NW + (int)threadIdx.x) * 4;
        if (k < K) put_h<DT>(s_x, (int64_t)c * K + k, xv[u], rs, gv[u]);
      }
      for (int k = (PER * 64 * NW + (int)threadIdx.x) * 4; k < K; k += 256 * NW) {
        float g[4];
        gain4<DT>(gr, k, true, g);
        put_h<DT>(s_x, (int64_t)c * K + k,
                  __builtin_bit_cast(f32x4, bld16(xr, (uint32_t)(c * K + k) * 4u)), rs, g);
      }
    };
    stage(0);
    for (int c = 1; c < nst; ++c) {
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const int k = (u * 64 * NW + (int)threadIdx.x) * 4;
        xv[u] = __builtin_bit_cast(f32x4, bld16(xr, k < K ? (uint32_t)(c * K + k) * 4u : BUF_OOB));
      }
      stage(c);
    }
    __syncthreads();
  } else if constexpr (PRO == PRO_COMBINE) {
    combine_weights();
    __syncthreads();
#pragma unroll
    for (int i = 0; i < PERC; ++i) combine_store(i * 64 * NW + (int)threadIdx.x, co[i]);
    for (int item = PERC * 64 * NW + (int)threadIdx.x; item < nst * (K / 4); item += 64 * NW) {
      f32x4 o[NSF];
      combine_load(item, o);
      combine_store(item, o);
    }
    __syncthreads();
  } else if constexpr (XS == 1) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int i = u * 64 * NW + (int)threadIdx.x;
      if (i < nst * kchunks) *(u32x4 *)(s_x + (int64_t)i * 16) = xc[u];
    }
    for (int i = PER * 64 * NW + (int)threadIdx.x; i < nst * kchunks; i += 64 * NW)
      *(u32x4 *)(s_x + (int64_t)i * 16) = bld16(xr, (uint32_t)i * 16u);
    __syncthreads();
  }


  if constexpr (epi_qkv(EPI)) qkv_fetch_tab<DT, R>(a, mat, row0, ep_rr, ep_ok, qin);

  // The MFMAs of one k-group accumulate in fp32 from zero; with ACC64 each
  // group's tile is then added into fp64 accumulators, so that fp32 rounding
  // only ever acts on sums of 4 * U * 32 products (where the registers allow).
  constexpr bool ACC64 = R * NT <= 2 || EPI == EPI_PART;
  f32x4 acc[R][NT];
  double acc64[ACC64 ? R : 1][ACC64 ? NT : 1][4];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      acc[r][t] = f32x4{0.f, 0.f, 0.f, 0.f};
      if constexpr (ACC64)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc64[r][t][e] = 0.0;
    }

  const int nk = kb_hi - kb_lo;
  const int nblk = wave < nk ? (nk - 1 - wave) / NW + 1 : 0;  // k-blocks of this wave
  const int ng = (nblk + U - 1) / U;
  for (int g0 = 0; g0 < ng; g0 += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int g = g0 + d;
      u32x4 xl[XRING ? 1 : U][XRING ? 1 : NT][4];
      if constexpr (!XRING) load_xg(xl, g);
      auto &xb = [&]() -> auto & {
        if constexpr (XRING) return xq[d];
        else return xl;
      }();
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
          for (int r = 0; r < R; ++r)
#pragma unroll
            for (int t = 0; t < NT; ++t) acc[r][t] = mma<DT>(w[d][u][r][s], xb[u][t][s], acc[r][t]);
      if constexpr (ACC64) {
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
          for (int t = 0; t < NT; ++t) {
#pragma unroll
            for (int e = 0; e < 4; ++e) acc64[r][t][e] += (double)acc[r][t][e];
            acc[r][t] = f32x4{0.f, 0.f, 0.f, 0.f};
          }
      }
      if constexpr (XRING) load_xg(xq[d], g + D);
      load_w(w[d], g + D);
      // keep the next group's MFMAs (which wait for its loads) below this refill
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // fixed-order sum of the waves' partial tiles through LDS
  __shared__ __align__(16) unsigned char s_red_raw[NW * R * NT * 64 * (ACC64 ? 32 : 16)];
  double *s_red64 = (double *)s_red_raw;  // [NW][R][NT][4][64]
  f32x4 *s_red = (f32x4 *)s_red_raw;      // [NW][R][NT][64]
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      if constexpr (ACC64) {
#pragma unroll
        for (int e = 0; e < 4; ++e) s_red64[(((wave * R + r) * NT + t) * 4 + e) * 64 + lane] = acc64[r][t][e];
      } else {
        s_red[((wave * R + r) * NT + t) * 64 + lane] = acc[r][t];
      }
    }
  __syncthreads();
  for (int item = threadIdx.x; item < NT * 64; item += 64 * NW) {
    const int t = item >> 6, ln = item & 63;
    f32x4 v[R];
    double vd[EPI == EPI_PART ? R : 1][4];  // EPI_PART: the fp64 sums themselves
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if constexpr (ACC64) {
        double sum[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
        for (int w2 = 0; w2 < NW; ++w2)
#pragma unroll
          for (int e = 0; e < 4; ++e) sum[e] += s_red64[(((w2 * R + r) * NT + t) * 4 + e) * 64 + ln];
        v[r] = f32x4{(float)sum[0], (float)sum[1], (float)sum[2], (float)sum[3]};
        if constexpr (EPI == EPI_PART)
#pragma unroll
          for (int e = 0; e < 4; ++e) vd[r][e] = sum[e];
      } else {
        v[r] = s_red[((0 * R + r) * NT + t) * 64 + ln];
#pragma unroll
        for (int w2 = 1; w2 < NW; ++w2) v[r] += s_red[((w2 * R + r) * NT + t) * 64 + ln];
      }
    }
    const int col = col0 + 16 * t + (ln & 15);
    if constexpr (XPRE) {
      if (col < a.ncols) {
        float *x = a.resid + (int64_t)col * a.ld_resid;
        const int row = row0[0] + 4 * (ln >> 4);
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (row + e < a.rows[0]) x[row + e] = xres[e] + v[0][e];
      }
    } else if constexpr (epi_qkv(EPI)) {
      if (col < a.ncols) qkv_store<DT, R, EPI == EPI_QKV_PAGED>(a, mat, row0, v, col, 4 * (ln >> 4), qin);
    } else if constexpr (EPI == EPI_PART) {
      if (col < a.ncols) {
        double *o = (double *)a.splitk_ws + ((int64_t)sp * a.ncols + col) * a.rows[0];
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int row = row0[r] + 4 * (ln >> 4) + e;
            if (row < a.rows[0]) o[row] = vd[r][e];
          }
      }
    } else {
      if (col < a.ncols) gemm_epilogue<DT, EPI, R, PK>(a, mat, row0, v, col, 4 * (ln >> 4));
    }
  }
}

// Many columns (B > 32, and prefill): Y = X W^T as a tiled GEMM.  A work group
// owns WR x RTW row tiles and WC x CTW column tiles; wave (wr, wc) computes
// its RTW x CTW output tiles over the whole K, so there is no reduction
// between waves and every weight operand feeds CTW MFMAs and every activation
// operand RTW.  Operands go straight from global memory into MFMA registers,
// one 32-element k step (a 1 KB weight sub-block per row tile, 16 bytes per
// lane per column tile) at a time, through a ring of two steps.  SwiGLU work
// groups hold gate tiles in their first RTW / 2 rows of each wave and the
// matching up tiles in the rest.  Activations are plain rows of the storage
// dtype (normalised once by k_rmsnorm when the projection has a norm).
// Accumulation is fp32 over the whole K.
template <int DT, int RTW, int CTW, int WR, int WC, int EPI>
__global__ __launch_bounds__(64 * WR * WC) void k_gemm_tile(GemmArgs a) {
  using S = typename Ty<DT>::S;
  constexpr int CE = Ty<DT>::CE;
  constexpr int SB = (int)sizeof(S);
  constexpr int D = 2;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wr = wave / WC, wc = wave % WC;
  const int li = lane & 15, lq = lane >> 4;
  const int K = a.K, kchunks = K / CE, nkb = (kchunks + 15) >> 4, nsb = nkb * 4;
  // XCD-aware order: the column groups of a row group are consecutive slots of one XCD
  int rg = blockIdx.x, cg = 0;
  if (a.n_colg > 1) {
    const int slot = (int)blockIdx.x >> 3;
    cg = slot % a.n_colg;
    rg = (slot / a.n_colg) * 8 + ((int)blockIdx.x & 7);
    if (rg >= a.n_groups) return;
  }
  int mat[RTW], row0[RTW];
#pragma unroll
  for (int r = 0; r < RTW; ++r) {
    if constexpr (EPI == EPI_SWIGLU) {
      constexpr int H = RTW / 2;
      mat[r] = r < H ? 0 : 1;
      row0[r] = 16 * ((rg * WR + wr) * H + (r % H));
    } else if constexpr (epi_qkv(EPI)) {
      const int tq = a.n_heads * a.head_dim / 16, tk = a.n_kv * a.head_dim / 16;
      int m = 0, t = (rg * WR + wr) * RTW + r;
      if (t >= tq) {
        t -= tq;
        m = 1;
        if (t >= tk) {
          t -= tk;
          m = 2;
        }
      }
      mat[r] = m;
      row0[r] = 16 * t;
    } else {
      mat[r] = 0;
      row0[r] = 16 * ((rg * WR + wr) * RTW + r);
    }
  }
  rsrc_t wres[RTW];
#pragma unroll
  for (int r = 0; r < RTW; ++r)
    wres[r] = make_rsrc((const S *)a.w[mat[r]] + (int64_t)(row0[r] >> 4) * nkb * 256 * CE,
                        row0[r] < a.rows[mat[r]] ? (uint32_t)nkb * 4096u : 0u);
  const rsrc_t xres = make_rsrc(a.x, (uint32_t)a.ncols * K * SB);
  const int colw = (cg * WC + wc) * CTW * 16;  // first column of the wave
  auto load = [&](u32x4 (&wv)[RTW], u32x4 (&xv)[CTW], int st) {
    const bool in = st < nsb;
    const uint32_t wo = (uint32_t)(st >> 2) * 4096u + (uint32_t)(st & 3) * 1024u + (uint32_t)lane * 16u;
#pragma unroll
    for (int r = 0; r < RTW; ++r) wv[r] = bld16_stream(wres[r], in ? wo : BUF_OOB);
    const int kc = (st >> 2) * 16 + (st & 3) * 4 + lq;
#pragma unroll
    for (int c = 0; c < CTW; ++c) {
      const int col = colw + 16 * c + li;
      xv[c] = bld16(xres, in && col < a.ncols && kc < kchunks ? (uint32_t)(col * K + kc * CE) * SB : BUF_OOB);
    }
  };
  f32x4 acc[RTW][CTW];
#pragma unroll
  for (int r = 0; r < RTW; ++r)
#pragma unroll
    for (int c = 0; c < CTW; ++c) acc[r][c] = f32x4{0.f, 0.f, 0.f, 0.f};
  u32x4 wv[D][RTW], xv[D][CTW];
#pragma unroll
  for (int d = 0; d < D; ++d) load(wv[d], xv[d], d);
  for (int s0 = 0; s0 < nsb; s0 += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
#pragma unroll
      for (int r = 0; r < RTW; ++r)
#pragma unroll
        for (int c = 0; c < CTW; ++c) acc[r][c] = mma<DT>(wv[d][r], xv[d][c], acc[r][c]);
      load(wv[d], xv[d], s0 + d + D);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  const int rr = 4 * lq;
#pragma unroll
  for (int c = 0; c < CTW; ++c) {
    const int col = colw + 16 * c + li;
    if (col >= a.ncols) continue;
    if constexpr (EPI == EPI_SWIGLU) {
      constexpr int H = RTW / 2;
#pragma unroll
      for (int r = 0; r < H; ++r) {
        const int m2[2] = {0, 1}, r2[2] = {row0[r], row0[r + H]};
        const f32x4 v2[2] = {acc[r][c], acc[r + H][c]};
        gemm_epilogue<DT, EPI_SWIGLU, 2>(a, m2, r2, v2, col, rr);
      }
    } else if constexpr (epi_qkv(EPI)) {
#pragma unroll
      for (int r = 0; r < RTW; ++r) {
        QkvIn<1> in;
        qkv_fetch_ids<DT, 1, EPI == EPI_QKV_PAGED>(a, &mat[r], &row0[r], col, rr, true, in);
        qkv_fetch_tab<DT, 1>(a, &mat[r], &row0[r], rr, true, in);
        qkv_store<DT, 1, EPI == EPI_QKV_PAGED>(a, &mat[r], &row0[r], &acc[r][c], col, rr, in);
      }
    } else {
#pragma unroll
      for (int r = 0; r < RTW; ++r) gemm_epilogue<DT, EPI, 1>(a, &mat[r], &row0[r], &acc[r][c], col, rr);
    }
  }
}

// Many columns (prefill rows, large batches) with both operands shared
// through LDS: a work group of 8 waves (4 x 2) owns RTG row tiles (SwiGLU:
// RTG/2 gate and the RTG/2 matching up tiles) by CTG column tiles, each wave
// RTG/4 x CTG/2 of them.  K advances in stages of two 32-element sub-blocks:
// the stage's weight sub-blocks (1 KB each, contiguous in the packed layout)
// and activation sub-blocks are staged in LDS in MFMA operand order, and each
// wave reads the operands of its output tiles from there (16 B per lane,
// conflict free).  Global loads run two stages ahead through registers, LDS
// is double buffered.  fp32 accumulation.
constexpr int LG_NW = 8;
template <int DT, int EPI, int RTG, int CTG>
__global__ __launch_bounds__(64 * LG_NW) void k_gemm_lds(GemmArgs a) {
  using S = typename Ty<DT>::S;
  constexpr int CE = Ty<DT>::CE;
  constexpr int SB = (int)sizeof(S);
  constexpr int RTW = RTG / 4, CTW = CTG / 2;        // tiles per wave
  constexpr int WSUB = RTG * 2, XSUB = CTG * 2;      // 1 KB sub-blocks per stage
  constexpr int WPT = WSUB / LG_NW, XPT = XSUB / LG_NW;  // of them moved per thread
  static_assert(WSUB % LG_NW == 0 && XSUB % LG_NW == 0, "stage split over the waves");
  static_assert(EPI != EPI_SWIGLU || RTW % 2 == 0, "gate/up pairs per wave");
  __shared__ __align__(16) u32x4 s_w[2][WSUB * 64];
  __shared__ __align__(16) u32x4 s_x[2][XSUB * 64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wr = wave >> 1, wc = wave & 1;
  const int li = lane & 15, lq = lane >> 4;
  const int K = a.K, kchunks = K / CE, nkb = (kchunks + 15) >> 4, nsb = nkb * 4;
  // XCD-aware order: the (column group, K split) units of a row group are
  // consecutive slots of one XCD
  const int nks = a.k_split > 1 ? a.k_split : 1, nu = a.n_colg * nks;
  int rg = blockIdx.x, cg = 0, ks = 0;
  if (nu > 1) {
    const int slot = (int)blockIdx.x >> 3, u = slot % nu;
    cg = u % a.n_colg;
    ks = u / a.n_colg;
    rg = (slot / nu) * 8 + ((int)blockIdx.x & 7);
    if (rg >= a.n_groups) return;
  }
  // this work group's K range, in 32-element sub-blocks [g_begin, g_end)
  const int kb_split = (nkb + nks - 1) / nks;
  const int g_begin = ks * kb_split * 4, g_end = min(nsb, (ks + 1) * kb_split * 4);
  const int nstage = g_end > g_begin ? (g_end - g_begin + 1) / 2 : 0;
  // row tile t of the work group (wave t / RTW) -> matrix and first row
  auto tile_of = [&](int t, int &m, int &r0) {
    if constexpr (EPI == EPI_SWIGLU) {
      constexpr int H = RTW / 2;
      const int w = t / RTW, k = t % RTW;
      m = k < H ? 0 : 1;
      r0 = 16 * (rg * (RTG / 2) + w * H + k % H);
    } else if constexpr (epi_qkv(EPI)) {
      const int tq = a.n_heads * a.head_dim / 16, tk = a.n_kv * a.head_dim / 16;
      int mm = 0, u = rg * RTG + t;
      if (u >= tq) {
        u -= tq;
        mm = 1;
        if (u >= tk) {
          u -= tk;
          mm = 2;
        }
      }
      m = mm;
      r0 = 16 * u;  // past the v rows for a partial last group
    } else {
      m = 0;
      r0 = 16 * (rg * RTG + t);
    }
  };
  const int colg0 = cg * CTG * 16;
  const rsrc_t xres = make_rsrc(a.x, (uint32_t)a.ncols * K * SB);
  // stage loads: thread (wave, lane) moves lane `lane` of sub-blocks
  // wave + 8 u; sub-block b of a stage is row tile (column tile) b / 2, k
  // sub-block b % 2 of the stage, so every buffer resource is wave-uniform
  rsrc_t wres[WPT];
#pragma unroll
  for (int u = 0; u < WPT; ++u) {
    const int t = (wave + LG_NW * u) >> 1;
    int m, r0;
    tile_of(t, m, r0);
    wres[u] = make_rsrc((const S *)a.w[m] + (int64_t)(r0 >> 4) * nkb * 256 * CE,
                        r0 < a.rows[m] ? (uint32_t)nkb * 4096u : 0u);
  }
  auto gload = [&](u32x4 (&wv)[WPT], u32x4 (&xv)[XPT], int st) {
#pragma unroll
    for (int u = 0; u < WPT; ++u) {
      const int g = g_begin + st * 2 + ((wave + LG_NW * u) & 1);
      wv[u] = bld16_stream(wres[u], g < g_end ? (uint32_t)(g >> 2) * 4096u + (uint32_t)(g & 3) * 1024u +
                                                    (uint32_t)lane * 16u
                                              : BUF_OOB);
    }
#pragma unroll
    for (int u = 0; u < XPT; ++u) {
      const int sbk = wave + LG_NW * u, ct = sbk >> 1, g = g_begin + st * 2 + (sbk & 1);
      const int col = colg0 + ct * 16 + li, kc = g * 4 + lq;
      xv[u] = bld16(xres, g < g_end && col < a.ncols && kc < kchunks ? (uint32_t)(col * K + kc * CE) * SB : BUF_OOB);
    }
  };
  auto lstore = [&](const u32x4 (&wv)[WPT], const u32x4 (&xv)[XPT], int buf) {
#pragma unroll
    for (int u = 0; u < WPT; ++u) s_w[buf][(wave + LG_NW * u) * 64 + lane] = wv[u];
#pragma unroll
    for (int u = 0; u < XPT; ++u) s_x[buf][(wave + LG_NW * u) * 64 + lane] = xv[u];
  };

  f32x4 acc[RTW][CTW];
#pragma unroll
  for (int r = 0; r < RTW; ++r)
#pragma unroll
    for (int c = 0; c < CTW; ++c) acc[r][c] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 ra_w[WPT], ra_x[XPT], rb_w[WPT], rb_x[XPT];
  gload(ra_w, ra_x, 0);
  lstore(ra_w, ra_x, 0);
  gload(ra_w, ra_x, 1);
  gload(rb_w, rb_x, 2);
  __syncthreads();
  for (int st0 = 0; st0 < nstage; st0 += 2) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int st = st0 + h, buf = h;  // stage st sits in LDS buffer st % 2
      if (st < nstage) {
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) {
          u32x4 av[RTW], bv[CTW];
#pragma unroll
          for (int r = 0; r < RTW; ++r) av[r] = s_w[buf][((wr * RTW + r) * 2 + sub) * 64 + lane];
#pragma unroll
          for (int c = 0; c < CTW; ++c) bv[c] = s_x[buf][((wc * CTW + c) * 2 + sub) * 64 + lane];
#pragma unroll
          for (int r = 0; r < RTW; ++r)
#pragma unroll
            for (int c = 0; c < CTW; ++c) acc[r][c] = mma<DT>(av[r], bv[c], acc[r][c]);
        }
      }
      // stage st + 1 (in registers since two stages ago) into the other
      // buffer, then request stage st + 3 into the registers it leaves
      if (h == 0) {
        lstore(ra_w, ra_x, 1);
        gload(ra_w, ra_x, st + 3);
      } else {
        lstore(rb_w, rb_x, 0);
        gload(rb_w, rb_x, st + 3);
      }
      __syncthreads();
    }
  }

  const int rr = 4 * lq;
  int mat[RTW], row0[RTW];
#pragma unroll
  for (int r = 0; r < RTW; ++r) tile_of(wr * RTW + r, mat[r], row0[r]);
#pragma unroll
  for (int c = 0; c < CTW; ++c) {
    const int col = colg0 + (wc * CTW + c) * 16 + li;
    if (col >= a.ncols) continue;
    if constexpr (EPI == EPI_SWIGLU) {
      constexpr int H = RTW / 2;
#pragma unroll
      for (int r = 0; r < H; ++r) {
        const int m2[2] = {0, 1}, r2[2] = {row0[r], row0[r + H]};
        const f32x4 v2[2] = {acc[r][c], acc[r + H][c]};
        gemm_epilogue<DT, EPI_SWIGLU, 2>(a, m2, r2, v2, col, rr);
      }
    } else if ((EPI == EPI_RESID || epi_qkv(EPI)) && nks > 1) {
      // K split: this split's fp32 partial over the output rows (q/k/v:
      // the q, k and v rows in turn), finished by a second kernel
      const int prows = split_rows(a, EPI);
      float *o = a.splitk_ws + ((int64_t)ks * a.ncols + col) * prows;
#pragma unroll
      for (int r = 0; r < RTW; ++r)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int row = 16 * (rg * RTG + wr * RTW + r) + rr + e;
          if (row < prows) o[row] = acc[r][c][e];
        }
    } else if constexpr (epi_qkv(EPI)) {
#pragma unroll
      for (int r = 0; r < RTW; ++r) {
        QkvIn<1> in;
        qkv_fetch_ids<DT, 1, EPI == EPI_QKV_PAGED>(a, &mat[r], &row0[r], col, rr, true, in);
        qkv_fetch_tab<DT, 1>(a, &mat[r], &row0[r], rr, true, in);
        qkv_store<DT, 1, EPI == EPI_QKV_PAGED>(a, &mat[r], &row0[r], &acc[r][c], col, rr, in);
      }
    } else {
#pragma unroll
      for (int r = 0; r < RTW; ++r) gemm_epilogue<DT, EPI, 1>(a, &mat[r], &row0[r], &acc[r][c], col, rr);
    }
  }
}

// The q/k/v epilogue after a K split: sums the partials of four q|k|v rows
// of one column in split order, then bias, RoPE, R(q) and the K/V append as
// in the GEMM's own epilogue.
template <int DT, bool PAGED>
__global__ __launch_bounds__(256) void k_qkv_split_epilogue(GemmArgs a) {
  const int prows = split_rows(a, EPI_QKV), n4 = prows / 4;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)a.ncols * n4) return;
  const int col = (int)(i / n4), row = (int)(i % n4) * 4;
  const int64_t slice = (int64_t)a.ncols * prows;
  const float *part = a.splitk_ws + (int64_t)col * prows + row;
  f32x4 v = *(const f32x4 *)part;
  for (int k = 1; k < a.k_split; ++k) v += *(const f32x4 *)(part + k * slice);
  // the row's matrix and tile, as the GEMM maps q|k|v row tiles
  const int tq = a.n_heads * a.head_dim / 16, tk = a.n_kv * a.head_dim / 16;
  int m = 0, t = row / 16;
  if (t >= tq) {
    t -= tq;
    m = 1;
    if (t >= tk) {
      t -= tk;
      m = 2;
    }
  }
  const int r0 = 16 * t, rr = row % 16;
  QkvIn<1> in;
  qkv_fetch_ids<DT, 1, PAGED>(a, &m, &r0, col, rr, true, in);
  qkv_fetch_tab<DT, 1>(a, &m, &r0, rr, true, in);
  qkv_store<DT, 1, PAGED>(a, &m, &r0, &v, col, rr, in);
}

// x[col][row] += the K-split partials of (col, row), in split order; four
// rows per thread (rows % 4 == 0)
__global__ __launch_bounds__(256) void k_splitk_sum(const float *part, int k_split, int ncols, int rows, float *x,
                                                   int ld_x) {
  const int n4 = rows / 4;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)ncols * n4) return;
  const int col = (int)(i / n4), row = (int)(i % n4) * 4;
  const int64_t slice = (int64_t)ncols * rows;
  f32x4 s = *(const f32x4 *)(part + (int64_t)col * rows + row);
  for (int k = 1; k < k_split; ++k) s += *(const f32x4 *)(part + k * slice + (int64_t)col * rows + row);
  f32x4 *xp = (f32x4 *)(x + (int64_t)col * ld_x + row);
  *xp += s;
}

// x[col][row] += R32(the fp64 K-split partials of (col, row) summed in split
// order), one element per thread: the pending residual sum of a pass that
// ends without a normalisation
__global__ __launch_bounds__(256) void k_resid_pending(const double *part, int k_split, int ncols, int rows, float *x) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x, slice = (int64_t)ncols * rows;
  if (i >= slice) return;
  double t = part[i];
  for (int k = 1; k < k_split; ++k) t += part[k * slice + i];
  x[i] += (float)t;
}

// ---------------------------------------------------------------------------
// weight-stationary GEMM for a few hundred columns
// ---------------------------------------------------------------------------
// At 129..256 columns (decode at a large batch) every weight row meets all
// columns, so a wave that owns WS_RT row tiles of a work unit takes their
// weights straight from memory into registers (a ring WS_DEPTH stages deep,
// non-temporal loads) and never shares them: only the activations go through
// LDS.  A work group = WS_NWC consumer waves (one task of WS_RT row tiles x
// WS_CT column tiles each) + WS_NP producer waves that stage the activations
// of each 64-element K stage into a double buffer.  Consumers read each
// activation sub-block from LDS a few ahead of its MFMAs (scheduling groups
// keep the reads WS_PF operands ahead) and meet the producers at one barrier
// per stage.  The grid is one work group per CU looping over work units
// (row-task group, column group); the column groups of one row group land on
// the same XCD, where the later ones read the weights from L2.  Taken for the
// tall matrices that need no K split, gate/up and the LM head: at the
// batch-256 Qwen-shaped layer gate/up takes 100-107 us against 146 for the
// LDS-staged kernel.  The short ones (q/k/v, O, down) measured slower here
// even split into 4-8 K ranges (O 47-55 us against 33, down 89 against 73):
// each wave waits for its own weights once per stage, so with few work units
// the latency of the weight stream is exposed.
// Five consumers: the Qwen-shaped gate/up at batch 256 is 240 work units on
// 256 CUs (six made 208 units, leaving 48 CUs idle: 103.7 against 95.5 us).
// A ring three stages deep spills at two waves per SIMD.
constexpr int WS_RT = 4, WS_CT = 8, WS_NWC = 5, WS_NP = 2, WS_DEPTH = 2, WS_PF = 3, WS_GRID = 256;
constexpr int WS_MIN_COLS = 129, WS_MAX_COLS = 256;

// one work-group barrier once this wave's LDS accesses are complete; the
// global loads in flight (the weight ring) are not waited for
__device__ __forceinline__ void ws_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// row tile r of task t -> matrix and first row (SwiGLU: WS_RT/2 gate tiles,
// then the matching up tiles)
template <int EPI>
__device__ __forceinline__ void ws_tile(int t, int r, int &m, int &r0) {
  if constexpr (EPI == EPI_SWIGLU) {
    constexpr int H = WS_RT / 2;
    m = r < H ? 0 : 1;
    r0 = 16 * (t * H + r % H);
  } else {
    m = 0;
    r0 = 16 * (t * WS_RT + r);
  }
}

template <int DT, int EPI>
__global__ __launch_bounds__(64 * (WS_NWC + WS_NP)) __attribute__((amdgpu_waves_per_eu(2, 2)))
void k_gemm_ws(GemmArgs a) {
  using S = typename Ty<DT>::S;
  constexpr int CE = Ty<DT>::CE;
  constexpr int SB = (int)sizeof(S);
  constexpr int RT = WS_RT, CT = WS_CT, NWC = WS_NWC, NP = WS_NP, DEPTH = WS_DEPTH, PF = WS_PF;
  constexpr int XE = 2 * CT, XPT = XE / NP, NB = 2 * CT;
  constexpr int UNR = DEPTH % 2 == 0 ? DEPTH : 2 * DEPTH;  // stages per unrolled round
  static_assert(XE % NP == 0 && PF <= NB, "stage split");
  static_assert(EPI == EPI_SWIGLU || EPI == EPI_STORE, "tall matrices without a K split");
  __shared__ __align__(16) u32x4 s_x[2][XE * 64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int li = lane & 15, lq = lane >> 4;
  const int K = a.K, kchunks = K / CE, nkb = (kchunks + 15) >> 4, nsb = nkb * 4;
  const int per_task = EPI == EPI_SWIGLU ? RT / 2 : RT;
  const int n_task = ((a.rows[0] + 15) / 16 + per_task - 1) / per_task;
  const int n_rg = (n_task + NWC - 1) / NWC, n_rg8 = (n_rg + 7) / 8 * 8;
  const int n_cg = (a.ncols + 16 * CT - 1) / (16 * CT);
  const int n_units = n_rg8 * n_cg;
  const rsrc_t xres = make_rsrc(a.x, (uint32_t)a.ncols * K * SB);
  const int g_begin = 0, g_end = nsb, nstage = (nsb + 1) / 2;
  for (int unit = blockIdx.x; unit < n_units; unit += gridDim.x) {
    // unit = ((row group / 8) * n_cg + column group) * 8 + row group % 8
    const int lo = unit & 7, v = unit >> 3;
    const int cg = v % n_cg, rg = (v / n_cg) * 8 + lo;
    if (rg >= n_rg) continue;
    const int cnt = min(NWC, n_task - rg * NWC);
    const int colg0 = cg * CT * 16;
    if (wave >= NWC) {
      // producer: activation sub-block e = sub * CT + column tile of each stage
      const int pw = wave - NWC;
      u32x4 xr[XPT];
      auto xload = [&](int st) {
#pragma unroll
        for (int i = 0; i < XPT; ++i) {
          const int e = pw + NP * i, sub = e / CT, ct = e % CT, g = g_begin + st * 2 + sub;
          const int col = colg0 + ct * 16 + li, kc = g * 4 + lq;
          xr[i] = bld16(xres, g < g_end && col < a.ncols && kc < kchunks ? (uint32_t)(col * K + kc * CE) * SB : BUF_OOB);
        }
      };
      auto xstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < XPT; ++i) s_x[buf][(pw + NP * i) * 64 + lane] = xr[i];
      };
      xload(0);
      xstore(0);
      xload(1);
      for (int st0 = 0; st0 < nstage; st0 += 2) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          if (st0 + h < nstage) {
            ws_barrier();
            xstore(h ^ 1);
            xload(st0 + h + 2);
          }
        }
      }
      ws_barrier();
    } else if (wave < cnt) {
      const int task = rg * NWC + wave;
      int mat[RT], row0[RT];
      rsrc_t wres[RT];
#pragma unroll
      for (int r = 0; r < RT; ++r) {
        ws_tile<EPI>(task, r, mat[r], row0[r]);
        wres[r] = make_rsrc((const S *)a.w[mat[r]] + (int64_t)(row0[r] >> 4) * nkb * 256 * CE,
                            row0[r] < a.rows[mat[r]] ? (uint32_t)nkb * 4096u : 0u);
      }
      u32x4 wq[DEPTH][2][RT];
      auto wload = [&](int slot, int st) {
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) {
          const int g = g_begin + st * 2 + sub;
#pragma unroll
          for (int r = 0; r < RT; ++r)
            wq[slot][sub][r] = bld16_stream(wres[r], g < g_end ? (uint32_t)g * 1024u + (uint32_t)lane * 16u : BUF_OOB);
        }
      };
      f32x4 acc[RT][CT];
#pragma unroll
      for (int r = 0; r < RT; ++r)
#pragma unroll
        for (int c = 0; c < CT; ++c) acc[r][c] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < DEPTH; ++s) wload(s, s);
      auto stage = [&](int st, int slot, int buf) {
        ws_barrier();
        u32x4 bq[PF];
#pragma unroll
        for (int j = 0; j < PF; ++j) bq[j] = s_x[buf][j * 64 + lane];
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const u32x4 b = bq[j % PF];
          if (j + PF < NB) bq[j % PF] = s_x[buf][(j + PF) * 64 + lane];
          const int sub = j / CT, c = j % CT;
#pragma unroll
          for (int r = 0; r < RT; ++r) acc[r][c] = mma<DT>(wq[slot][sub][r], b, acc[r][c]);
        }
        // PF operand reads ahead, then RT MFMAs and one read per operand
        __builtin_amdgcn_sched_group_barrier(0x100, PF, 0);
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          __builtin_amdgcn_sched_group_barrier(0x008, RT, 0);
          if (j + PF < NB) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        wload(slot, st + DEPTH);
      };
      // whole rounds of UNR stages with no guard, so that the waits for the
      // weight ring count its loads exactly; then the remaining stages
      int st0 = 0;
      for (; st0 + UNR <= nstage; st0 += UNR) {
#pragma unroll
        for (int h = 0; h < UNR; ++h) stage(st0 + h, h % DEPTH, h & 1);
      }
#pragma unroll
      for (int h = 0; h < UNR; ++h)
        if (st0 + h < nstage) stage(st0 + h, h % DEPTH, h & 1);
      ws_barrier();

      const int rr = 4 * lq;
#pragma unroll
      for (int c = 0; c < CT; ++c) {
        const int col = colg0 + c * 16 + li;
        if (col >= a.ncols) continue;
        if constexpr (EPI == EPI_SWIGLU) {
          constexpr int H = RT / 2;
#pragma unroll
          for (int r = 0; r < H; ++r) {
            const int m2[2] = {0, 1}, r2[2] = {row0[r], row0[r + H]};
            const f32x4 v2[2] = {acc[r][c], acc[r + H][c]};
            gemm_epilogue<DT, EPI_SWIGLU, 2>(a, m2, r2, v2, col, rr);
          }
        } else {
#pragma unroll
          for (int r = 0; r < RT; ++r) gemm_epilogue<DT, EPI, 1>(a, &mat[r], &row0[r], &acc[r][c], col, rr);
        }
      }
    } else {
      // no task in this unit: the same barriers
      for (int st = 0; st < nstage; ++st) ws_barrier();
      ws_barrier();
    }
  }
}

// ---------------------------------------------------------------------------
// launch shapes
// ---------------------------------------------------------------------------
constexpr int XS_MAX_BYTES = 32 * 1024;  // LDS for normalised activations

template <int DT, int R, int NT, int NW, int U, int PRO, int XS, int EPI>
hipError_t gemm_launch(const GemmArgs &a, int n_groups, size_t shmem, hipStream_t st) {
  GemmArgs g = a;
  g.n_groups = n_groups;
  g.n_colg = (a.ncols + 16 * NT - 1) / (16 * NT);
  const int blocks = g.n_colg > 1 ? (n_groups + 7) / 8 * 8 * g.n_colg : n_groups;
  // the packed layouts get instantiations of their own, so the usual
  // row-major loads and stores carry no branch
  if constexpr (DT != HS_F32) {
    if constexpr (EPI == EPI_SWIGLU)
      if (a.out_packed) {
        if constexpr (XS == 0)
          if (a.x_packed) {
            HS_LAUNCH((k_gemm<DT, R, NT, NW, U, PRO, XS, EPI, true, true>), dim3(blocks), dim3(64 * NW), shmem, st, g);
            return hipGetLastError();
          }
        HS_LAUNCH((k_gemm<DT, R, NT, NW, U, PRO, XS, EPI, true, false>), dim3(blocks), dim3(64 * NW), shmem, st, g);
        return hipGetLastError();
      }
    if constexpr (XS == 0)
      if (a.x_packed) {
        HS_LAUNCH((k_gemm<DT, R, NT, NW, U, PRO, XS, EPI, false, true>), dim3(blocks), dim3(64 * NW), shmem, st, g);
        return hipGetLastError();
      }
  }
  HS_LAUNCH((k_gemm<DT, R, NT, NW, U, PRO, XS, EPI, false, false>), dim3(blocks), dim3(64 * NW), shmem, st, g);
  return hipGetLastError();
}

// Launch shape per epilogue.  Work groups of 4 waves when the activations are
// staged in LDS (the batch-1 down projection 16.3 against 16.9 µs with 8; the
// O projection with the split combine keeps 8), of 2-4 when they are read from
// memory (gemm_global_r).  One k-block per group,
// two for the LM head at one staged column tile.
// Columns staged in LDS (few): one row tile per work group (R = 1; SwiGLU 2).
// Activations read from global memory: every row tile of a work group reuses
// the activation chunks it loads, so q/k/v and the LM head take as many row
// tiles per work group as keep the grid large (LM head 4; q/k/v 4 while that
// leaves >= 192 work groups, else 2 while >= 128), the residual projections 1.
template <int DT, int EPI, int R, int NW, int NT>
hipError_t gemm_global(const GemmArgs &p, int tiles16, hipStream_t st) {
  const int n_groups = EPI == EPI_SWIGLU ? tiles16 : (tiles16 + R - 1) / R;
  return gemm_launch<DT, R, NT, NW, 1, PRO_PLAIN, 0, EPI>(p, n_groups, 0, st);
}

// Waves per work group: 2 for q/k/v, the LM head and, at one column tile,
// SwiGLU (batch 16, Qwen-shaped: gate/up 47.3 against 49.6 µs with 4 waves,
// q/k/v 14.2 against 14.9); SwiGLU over two column tiles 1 (batch 32,
// LLaVA-shaped: 38.2 against 39.5 with 4; one wave at one tile: 48.8).  The
// residual projections take 4 at one column tile and 2 at two (batch 16: O 7.8
// against 8.8 µs with 8, down 27.3 against 27.9; batch 32: down 22.5 against
// 24.4).
template <int DT, int EPI, int NT>
hipError_t gemm_global_r(const GemmArgs &p, int tiles16, hipStream_t st) {
  constexpr int NW = EPI == EPI_RESID ? (NT == 1 ? 4 : 2) : EPI != EPI_SWIGLU ? 2 : NT == 1 ? 2 : 1;
  if constexpr (EPI == EPI_SWIGLU) return gemm_global<DT, EPI, 2, NW, NT>(p, tiles16, st);
  else if constexpr (EPI == EPI_RESID) return gemm_global<DT, EPI, 1, NW, NT>(p, tiles16, st);
  else if constexpr (EPI == EPI_STORE) return gemm_global<DT, EPI, 4, NW, NT>(p, tiles16, st);
  else {
    if (tiles16 % 4 == 0 && tiles16 / 4 >= 192) return gemm_global<DT, EPI, 4, NW, NT>(p, tiles16, st);
    if (tiles16 % 2 == 0 && tiles16 / 2 >= 128) return gemm_global<DT, EPI, 2, NW, NT>(p, tiles16, st);
    return gemm_global<DT, EPI, 1, NW, NT>(p, tiles16, st);
  }
}

// Tiled GEMM launch: work-group tiles of WR*RTW row tiles by WC*CTW column
// tiles (SwiGLU: RTW/2 gate and RTW/2 up tiles per wave).
template <int DT, int RTW, int CTW, int WR, int WC, int EPI>
hipError_t gemm_tile_launch(const GemmArgs &a, int tiles16, hipStream_t st) {
  GemmArgs g = a;
  const int rows_per_group = EPI == EPI_SWIGLU ? WR * RTW / 2 : WR * RTW;
  g.n_groups = (tiles16 + rows_per_group - 1) / rows_per_group;
  g.n_colg = (a.ncols + 16 * WC * CTW - 1) / (16 * WC * CTW);
  const int blocks = g.n_colg > 1 ? (g.n_groups + 7) / 8 * 8 * g.n_colg : g.n_groups;
  HS_LAUNCH((k_gemm_tile<DT, RTW, CTW, WR, WC, EPI>), dim3(blocks), dim3(64 * WR * WC), 0, st, g);
  return hipGetLastError();
}

// work groups of the LDS kernel with RTG x CTG tiles (and k_split K splits)
template <int EPI, int RTG, int CTG>
int lds_groups(const GemmArgs &a, int tiles16, int k_split, int &n_groups, int &n_colg) {
  const int rows_per_group = EPI == EPI_SWIGLU ? RTG / 2 : RTG;
  n_groups = (tiles16 + rows_per_group - 1) / rows_per_group;
  n_colg = (a.ncols + 16 * CTG - 1) / (16 * CTG);
  const int nu = n_colg * k_split;
  return nu > 1 ? (n_groups + 7) / 8 * 8 * nu : n_groups;
}

// after a GEMM that split K: the kernel that sums the partials into the
// residual stream, or into the q/k/v epilogue
template <int DT, int EPI>
hipError_t split_finish(const GemmArgs &g, hipStream_t st) {
  const int64_t n = (int64_t)g.ncols * (split_rows(g, EPI) / 4);
  if constexpr (epi_qkv(EPI)) {
    HS_LAUNCH((k_qkv_split_epilogue<DT, EPI == EPI_QKV_PAGED>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
              g);
  } else {
    HS_LAUNCH(k_splitk_sum, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, g.splitk_ws, g.k_split, g.ncols,
              g.rows[0], g.resid, g.ld_resid);
  }
  return hipGetLastError();
}

template <int DT, int EPI, int RTG, int CTG>
hipError_t gemm_lds_launch(const GemmArgs &a, int tiles16, int k_split, hipStream_t st) {
  GemmArgs g = a;
  g.k_split = k_split;
  const int blocks = lds_groups<EPI, RTG, CTG>(a, tiles16, k_split, g.n_groups, g.n_colg);
  HS_LAUNCH((k_gemm_lds<DT, EPI, RTG, CTG>), dim3(blocks), dim3(64 * LG_NW), 0, st, g);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess || k_split <= 1) return e;
  return split_finish<DT, EPI>(g, st);
}

template <int DT, int EPI>
hipError_t gemm_ws_launch(const GemmArgs &a, hipStream_t st) {
  HS_LAUNCH((k_gemm_ws<DT, EPI>), dim3(WS_GRID), dim3(64 * (WS_NWC + WS_NP)), 0, st, a);
  return hipGetLastError();
}

// Many columns.  Where the work-group tile of 16 x 8 row x column tiles (wave
// tiles of 4 x 4, half the LDS reads per MFMA) still gives LDS_BIG_GROUPS
// work groups, it is taken (prefill gate/up at 640 rows: 159 against 191 us;
// with the threshold at 200 instead of 384 the 640-row q/k/v takes it too,
// and the LLaVA-shaped prefill went from 21.1 to 20.2 ms).  From
// WIDE_COLS columns on, 16 x 16 tiles (wave tiles of 4 x 8: 0.375 KB of LDS
// reads per MFMA instead of 0.5; 128 KB of LDS) where they give as many work
// groups; below that the 256-column groups pad too much (gate/up at 640
// rows: 240 against 172 us).
// A GEMM (residual or q/k/v) with fewer than SPLITK_BELOW work groups
// splits K (up to SPLITK_MAX ways, at least 4 k-blocks each) when the
// partials fit the workspace.  Otherwise the LDS-staged kernel from
// LDS_MIN_GROUPS work groups up, and below that the register-tiled kernel,
// whose smaller work groups spread narrow matrices over more CUs (measured
// crossover: between 64 and 80 work groups of the LDS kernel).
constexpr int LDS_MIN_GROUPS = 72, LDS_BIG_GROUPS = 200, SPLITK_BELOW = 128, SPLITK_TARGET = 256, WIDE_COLS = 2048;
template <int DT, int EPI>
hipError_t gemm_tiled(const GemmArgs &p, int tiles16, hipStream_t st) {
  if constexpr (DT != HS_F32 && (EPI == EPI_SWIGLU || EPI == EPI_STORE))
    if (p.ncols >= WS_MIN_COLS && p.ncols <= WS_MAX_COLS) return gemm_ws_launch<DT, EPI>(p, st);
  int ng, nc;
  if (p.ncols >= WIDE_COLS && lds_groups<EPI, 16, 16>(p, tiles16, 1, ng, nc) >= LDS_BIG_GROUPS)
    return gemm_lds_launch<DT, EPI, 16, 16>(p, tiles16, 1, st);
  if (lds_groups<EPI, 16, 8>(p, tiles16, 1, ng, nc) >= LDS_BIG_GROUPS)
    return gemm_lds_launch<DT, EPI, 16, 8>(p, tiles16, 1, st);
  const int blocks = lds_groups<EPI, 8, 8>(p, tiles16, 1, ng, nc);
  if constexpr (EPI == EPI_RESID || epi_qkv(EPI)) {
    const int nkb = (p.K / Ty<DT>::CE + 15) / 16;
    int ks = blocks < SPLITK_BELOW ? std::min(std::min(SPLITK_MAX, (SPLITK_TARGET + blocks - 1) / blocks), nkb / 4) : 1;
    if (ks > 1) {
      const int per = (nkb + ks - 1) / ks;
      ks = (nkb + per - 1) / per;  // no empty split
    }
    const int prows = split_rows(p, EPI);
    if (ks > 1 && p.splitk_ws && prows % 4 == 0 && (int64_t)ks * p.ncols * prows <= p.splitk_cap)
      return gemm_lds_launch<DT, EPI, 8, 8>(p, tiles16, ks, st);
  }
  if (blocks >= LDS_MIN_GROUPS) return gemm_lds_launch<DT, EPI, 8, 8>(p, tiles16, 1, st);
  if constexpr (EPI == EPI_SWIGLU) return gemm_tile_launch<DT, 4, 4, 2, 2, EPI>(p, tiles16, st);
  else if constexpr (EPI == EPI_RESID) return gemm_tile_launch<DT, 2, 2, 1, 4, EPI>(p, tiles16, st);
  else return gemm_tile_launch<DT, 2, 4, 2, 2, EPI>(p, tiles16, st);
}

// A residual projection that leaves its sum to the next RMSNorm
// (resid_defer_splits): two row tiles per work group of 2 waves and K split
// in two, as many work groups as one row tile each over the whole K (the
// activation chunks a work group loads feed twice the MFMAs).  Batch 16,
// Qwen-shaped: down 22.8 against 27.0 us, O 6.2 against 7.0; batch 32,
// LLaVA-shaped: down 18.1 against 21.4, O 8.1 against 9.1 (kernels alone).
constexpr int DEFER_SPLITS = 2;
template <int DT>
hipError_t gemm_defer(const GemmArgs &a, int tiles16, int tiles, hipStream_t st) {
  if (DT == HS_F32 || !a.x_packed || tiles > 2 || a.defer != DEFER_SPLITS || !a.splitk_ws ||
      2 * (int64_t)a.defer * a.ncols * a.rows[0] > a.splitk_cap)
    return hipErrorInvalidValue;
  GemmArgs g = a;
  g.k_split = a.defer;
  const int n_groups = (tiles16 + 1) / 2 * a.defer;
  if (tiles <= 1) return gemm_launch<DT, 2, 1, 2, 1, PRO_PLAIN, 0, EPI_PART>(g, n_groups, 0, st);
  return gemm_launch<DT, 2, 2, 2, 1, PRO_PLAIN, 0, EPI_PART>(g, n_groups, 0, st);
}

template <int DT, int PRO, int EPI>
hipError_t gemm_shape(const GemmArgs &a, hipStream_t st) {
  // row tiles of 16 (SwiGLU: of one of its two matrices)
  const int tiles16 = epi_qkv(EPI) ? (a.n_heads + 2 * a.n_kv) * a.head_dim / 16 : (a.rows[0] + 15) / 16;
  const int tiles = (a.ncols + 15) / 16;
  const int b = DT == HS_F32 ? 4 : 2;
  const size_t xs = (size_t)a.ncols * a.K * b;
  if constexpr (EPI == EPI_RESID && PRO == PRO_PLAIN)
    if (a.defer) {
      if constexpr (DT == HS_F32) return hipErrorInvalidValue;
      else return gemm_defer<DT>(a, tiles16, tiles, st);
    }
  if (tiles <= 1 && xs <= XS_MAX_BYTES) {
    if (a.pend_s) return hipErrorInvalidValue;  // pending partials are added by k_rmsnorm alone
    constexpr int R = EPI == EPI_SWIGLU ? 2 : 1;
    constexpr int NW = 4;
    constexpr int U = EPI == EPI_STORE ? 2 : 1;
    return gemm_launch<DT, R, 1, NW, U, PRO, 1, EPI>(a, tiles16, xs, st);
  }
  GemmArgs p = a;
  if constexpr (PRO == PRO_NORM) {
    // more columns than the prologue stages: normalise them once, then read
    // them as plain activations (in the packed layout where the GEMM reads
    // them through MFMA-operand loads)
    p.x_packed = gemm_x_packed(DT, a.ncols, a.K) ? 1 : 0;
    float *x = (float *)a.x;  // rewritten with the pending partials added
    if (a.pend_s == 0)
      HS_LAUNCH((k_rmsnorm<DT, 0>), dim3(a.ncols), dim3(256), 0, st, x, a.gain, a.eps, a.K, a.h_work, p.x_packed,
                nullptr, a.ncols);
    else if (a.pend_s == DEFER_SPLITS && a.pend)
      HS_LAUNCH((k_rmsnorm<DT, DEFER_SPLITS>), dim3(a.ncols), dim3(256), 0, st, x, a.gain, a.eps, a.K, a.h_work,
                p.x_packed, a.pend, a.ncols);
    else
      return hipErrorInvalidValue;
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    p.x = a.h_work;
  }
  if (tiles <= 1) return gemm_global_r<DT, EPI, 1>(p, tiles16, st);
  if (tiles <= 2) return gemm_global_r<DT, EPI, 2>(p, tiles16, st);
  return gemm_tiled<DT, EPI>(p, tiles16, st);
}

// the combine prologue: one column tile whose activations fit the LDS copy
template <int DT>
hipError_t gemm_combine(const GemmArgs &a, hipStream_t st) {
  const size_t xs = (size_t)a.ncols * a.K * (DT == HS_F32 ? 4 : 2);
  return gemm_launch<DT, 1, 1, 8, 1, PRO_COMBINE, 1, EPI_RESID>(a, (a.rows[0] + 15) / 16, xs, st);
}

template <int DT>
hipError_t gemm_dt(int pro, int epi, const GemmArgs &a, hipStream_t st) {
  if (pro == PRO_COMBINE && epi == EPI_RESID) return gemm_combine<DT>(a, st);
  if (pro == PRO_NORM && epi == EPI_QKV) return gemm_shape<DT, PRO_NORM, EPI_QKV>(a, st);
  if constexpr (DT != HS_F32)  // pooled caches hold 16-bit storage only
    if (pro == PRO_NORM && epi == EPI_QKV_PAGED) return gemm_shape<DT, PRO_NORM, EPI_QKV_PAGED>(a, st);
  if (pro == PRO_NORM && epi == EPI_SWIGLU) return gemm_shape<DT, PRO_NORM, EPI_SWIGLU>(a, st);
  if (pro == PRO_NORM && epi == EPI_STORE) return gemm_shape<DT, PRO_NORM, EPI_STORE>(a, st);
  if (pro == PRO_PLAIN && epi == EPI_RESID) return gemm_shape<DT, PRO_PLAIN, EPI_RESID>(a, st);
  return hipErrorInvalidValue;
}

}  // namespace

bool gemm_x_packed(int dtype, int ncols, int K) {
  // the launch shape's choice: activations staged in LDS (one column tile
  // that fits the copy), from memory (two column tiles at most), or the
  // tiled kernels
  if (dtype == HS_F32 || ncols <= 0) return false;
  const int tiles = (ncols + 15) / 16;
  return tiles <= 2 && !(tiles <= 1 && (size_t)ncols * K * 2 <= XS_MAX_BYTES);
}

int resid_defer_splits(int dtype, int ncols, int K, int d_model, int64_t cap) {
  // the projection reads its activations from memory (k_gemm over 2..32
  // columns), the next normalisation runs in k_rmsnorm (its columns do not
  // fit the prologue's LDS copy), every split holds a k-block, whole float4
  // rows, and the fp64 partials fit the workspace
  if (!gemm_x_packed(dtype, ncols, K)) return 0;
  const int tiles = (ncols + 15) / 16;
  if (tiles <= 1 && (size_t)ncols * d_model * 2 <= XS_MAX_BYTES) return 0;
  if ((K / 8 + 15) / 16 < DEFER_SPLITS || d_model % 4) return 0;
  if (2 * (int64_t)DEFER_SPLITS * ncols * d_model > cap) return 0;
  return DEFER_SPLITS;
}

hipError_t launch_resid_pending(const double *part, int k_split, int ncols, int rows, float *x, hipStream_t st) {
  if (ncols <= 0 || rows <= 0 || k_split <= 0) return hipSuccess;
  const int64_t n = (int64_t)ncols * rows;
  HS_LAUNCH(k_resid_pending, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, part, k_split, ncols, rows, x);
  return hipGetLastError();
}

int64_t act_elems(int64_t rows, int64_t K) { return std::max(rows * K, (int64_t)32 * ((K + 127) / 128 * 128)); }

hipError_t launch_gemm(int dtype, int pro, int epi, const GemmArgs &a, hipStream_t st) {
  if (a.ncols <= 0 || a.rows[0] <= 0) return hipSuccess;
  switch (dtype) {
    case HS_F32: return gemm_dt<HS_F32>(pro, epi, a, st);
    case HS_F16: return gemm_dt<HS_F16>(pro, epi, a, st);
    case HS_BF16: return gemm_dt<HS_BF16>(pro, epi, a, st);
  }
  return hipErrorInvalidValue;
}

bool gemm_combine_fusable(int dtype, int ncols, int K, int n_heads, int n_split) {
  const size_t b = dtype == HS_F32 ? 4 : 2;
  return n_split > 1 && n_split <= COMBINE_FUSE_SPLITS && ncols >= 1 && ncols <= 16 && K % 4 == 0 &&
         (size_t)ncols * K * b <= XS_MAX_BYTES && ncols * n_heads <= 64 * 8;
}

int64_t packed_elems(int dtype, int64_t rows, int64_t cols) {
  const int ce = dtype == HS_F32 ? 4 : 8;
  const int64_t nkb = (cols / ce + 15) / 16;
  return ((rows + 15) / 16) * nkb * 256 * ce;
}

hipError_t launch_pack(int dtype, const void *src, int64_t rows, int64_t cols, void *dst, int pair_hd,
                       hipStream_t st) {
  const int ce = dtype == HS_F32 ? 4 : 8;
  const int nkb = (int)((cols / ce + 15) / 16);
  const int64_t total = ((rows + 15) / 16) * nkb * 256;
  if (total <= 0) return hipSuccess;
  const int grid = (int)std::min<int64_t>((total + 255) / 256, 65536);
  switch (dtype) {
    case HS_F32: HS_LAUNCH(k_pack<HS_F32>, dim3(grid), dim3(256), 0, st, src, dst, rows, (int)cols, nkb, total, pair_hd); break;
    case HS_F16: HS_LAUNCH(k_pack<HS_F16>, dim3(grid), dim3(256), 0, st, src, dst, rows, (int)cols, nkb, total, pair_hd); break;
    case HS_BF16: HS_LAUNCH(k_pack<HS_BF16>, dim3(grid), dim3(256), 0, st, src, dst, rows, (int)cols, nkb, total, pair_hd); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace hs
