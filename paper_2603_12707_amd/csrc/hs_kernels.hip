// hs_kernels.hip — gfx950 kernels of the language-decode step (arXiv 2603.12707):
// weight-streaming MFMA GEMM with fused RMSNorm prologue and RoPE + KV-append /
// SwiGLU / residual / logits epilogues, split-K flash-decoding attention with
// its combine, embedding gather and greedy selection.
//
// The paper characterises decode as the phase that streams the model weights
// and the KV cache from HBM once per generated token (§2; Eq. 5 of §4.3, where
// decode time is the streamed bytes over HBM bandwidth) and grows the cache by
// one K and one V row per layer per token (Eq. 1, §4.1).  Every kernel here is
// therefore organised around one coalesced pass over those bytes.
#include "hs_internal.h"

#include <cmath>

namespace hs {

thread_local LaunchEvents g_launch_events;

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// every launch carries the timing hook's events (null when untimed)
#define HS_LAUNCH(kernel, grid, block, shmem, stream, ...)                                                        \
  hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, g_launch_events.start, g_launch_events.stop, 0, \
                        __VA_ARGS__)

// ---------------------------------------------------------------------------
// storage dtypes
// ---------------------------------------------------------------------------
template <int DT>
struct Ty;
template <>
struct Ty<HS_F32> {
  using S = float;
  static constexpr int CE = 4;  // elements per 16-byte chunk
};
template <>
struct Ty<HS_F16> {
  using S = uint16_t;
  static constexpr int CE = 8;
};
template <>
struct Ty<HS_BF16> {
  using S = uint16_t;
  static constexpr int CE = 8;
};

__device__ __forceinline__ float f16_to_f32(uint32_t u) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)u);
}
__device__ __forceinline__ uint32_t f32_to_f16(float f) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)f);  // v_cvt_f16_f32, round to nearest even
}
__device__ __forceinline__ float bf16_to_f32(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x7FFFFFu)) return (u >> 16) | 0x40u;
  u += 0x7FFFu + ((u >> 16) & 1u);  // round to nearest even
  return u >> 16;
}

template <int DT>
__device__ __forceinline__ float ld_elem(const void *p, int64_t i) {
  if constexpr (DT == HS_F32) return ((const float *)p)[i];
  else if constexpr (DT == HS_F16) return f16_to_f32(((const uint16_t *)p)[i]);
  else return bf16_to_f32(((const uint16_t *)p)[i]);
}

// R(.): store an fp32 value in the storage dtype
template <int DT>
__device__ __forceinline__ void st_elem(void *p, int64_t i, float v) {
  if constexpr (DT == HS_F32) ((float *)p)[i] = v;
  else if constexpr (DT == HS_F16) ((uint16_t *)p)[i] = (uint16_t)f32_to_f16(v);
  else ((uint16_t *)p)[i] = (uint16_t)f32_to_bf16(v);
}

// 16-byte chunk -> CE floats
template <int DT>
__device__ __forceinline__ void unpack(u32x4 w, float *f) {
  if constexpr (DT == HS_F32) {
#pragma unroll
    for (int e = 0; e < 4; ++e) f[e] = __uint_as_float(w[e]);
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if constexpr (DT == HS_F16) {
        f[2 * e] = f16_to_f32(w[e] & 0xFFFFu);
        f[2 * e + 1] = f16_to_f32(w[e] >> 16);
      } else {
        f[2 * e] = bf16_to_f32(w[e] & 0xFFFFu);
        f[2 * e + 1] = bf16_to_f32(w[e] >> 16);
      }
    }
  }
}

// CE floats -> 16-byte chunk, rounding to the storage dtype
template <int DT>
__device__ __forceinline__ u32x4 pack(const float *f) {
  u32x4 w;
  if constexpr (DT == HS_F32) {
#pragma unroll
    for (int e = 0; e < 4; ++e) w[e] = __float_as_uint(f[e]);
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if constexpr (DT == HS_F16) w[e] = f32_to_f16(f[2 * e]) | (f32_to_f16(f[2 * e + 1]) << 16);
      else w[e] = f32_to_bf16(f[2 * e]) | (f32_to_bf16(f[2 * e + 1]) << 16);
    }
  }
  return w;
}

// One 16x16 output tile += A(16 x k) * B(k x 16) over the k values held in a
// 16-byte chunk per lane.  Lane l supplies row (A) / column (B) l % 16 and the
// k sub-range of lane group l / 16; A and B use the same k mapping, so the
// order of k inside the contraction is immaterial.
template <int DT>
__device__ __forceinline__ f32x4 mma(u32x4 a, u32x4 b, f32x4 c) {
  if constexpr (DT == HS_F16) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                  0, 0);
  } else if constexpr (DT == HS_BF16) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
  } else {
    f32x4 av = __builtin_bit_cast(f32x4, a), bv = __builtin_bit_cast(f32x4, b);
#pragma unroll
    for (int e = 0; e < 4; ++e) c = __builtin_amdgcn_mfma_f32_16x16x4f32(av[e], bv[e], c, 0, 0, 0);
    return c;
  }
}

__device__ __forceinline__ u32x4 ld16(const void *p) { return *(const u32x4 *)p; }
__device__ __forceinline__ u32x4 ld16_stream(const void *p) {
  return __builtin_nontemporal_load((const u32x4 *)p);
}

// ---------------------------------------------------------------------------
// cross-lane reductions (DPP within 16-lane rows, then across rows)
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float,
                            __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
constexpr int DPP_QUAD_1032 = 0xB1;    // quad_perm [1,0,3,2]
constexpr int DPP_QUAD_2301 = 0x4E;    // quad_perm [2,3,0,1]
constexpr int DPP_ROW_HALF_MIRROR = 0x141;
constexpr int DPP_ROW_MIRROR = 0x140;

// sum over aligned groups of N lanes (N = 8, 16, 32, 64); every lane gets it
template <int N>
__device__ __forceinline__ float group_sum(float v) {
  v += dpp<DPP_QUAD_1032>(v);
  v += dpp<DPP_QUAD_2301>(v);
  v += dpp<DPP_ROW_HALF_MIRROR>(v);
  if constexpr (N >= 16) v += dpp<DPP_ROW_MIRROR>(v);
  if constexpr (N >= 32) v += __shfl_xor(v, 16);
  if constexpr (N >= 64) v += __shfl_xor(v, 32);
  return v;
}
__device__ __forceinline__ float wave_sum(float v) { return group_sum<64>(v); }
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp<DPP_QUAD_1032>(v));
  v = fmaxf(v, dpp<DPP_QUAD_2301>(v));
  v = fmaxf(v, dpp<DPP_ROW_HALF_MIRROR>(v));
  v = fmaxf(v, dpp<DPP_ROW_MIRROR>(v));
  v = fmaxf(v, __shfl_xor(v, 16));
  v = fmaxf(v, __shfl_xor(v, 32));
  return v;
}

// ---------------------------------------------------------------------------
// weight-streaming GEMM
// ---------------------------------------------------------------------------

// Row tiles of work group g.  The q/k/v epilogue pairs rows i and i + d_h/2
// of one head (the two halves RoPE rotates together); SwiGLU pairs row j of
// the gate and of the up projection.
template <int EPI, int R>
__device__ __forceinline__ void tile_map(const GemmArgs &a, int g, int *mat, int *row0) {
  if constexpr (EPI == EPI_QKV) {
    const int hd = a.head_dim, gph = hd / 32;
    int m = 0, rem = g;
    if (rem >= a.n_heads * gph) {
      rem -= a.n_heads * gph;
      m = 1;
      if (rem >= a.n_kv * gph) {
        rem -= a.n_kv * gph;
        m = 2;
      }
    }
    const int head = rem / gph, i0 = (rem % gph) * 16;
    mat[0] = mat[1] = m;
    row0[0] = head * hd + i0;
    row0[1] = head * hd + i0 + hd / 2;
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

template <int DT, int EPI, int R>
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
    void *o = (char *)a.out + (int64_t)col * a.ld_out * (DT == HS_F32 ? 4 : 2);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int j = row0[0] + rr + e;
      if (j < a.rows[0]) {
        const float g = v[0][e], u = v[1][e];
        st_elem<DT>(o, j, g / (1.0f + expf(-g)) * u);
      }
    }
  } else {  // EPI_QKV
    const int m = mat[0], hd = a.head_dim, half = hd >> 1;
    const int head = row0[0] / hd, i0 = row0[0] - head * hd;
    int req, pos;
    if (a.prefill_req < 0) {
      req = col;
      pos = a.kv_len[col];
    } else {
      req = a.prefill_req;
      pos = col;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int i = i0 + rr + e;  // frequency pair, < d_h / 2
      float v1 = v[0][e], v2 = v[1][e];
      if (a.bias[m]) {
        v1 += ld_elem<DT>(a.bias[m], head * hd + i);
        v2 += ld_elem<DT>(a.bias[m], head * hd + i + half);
      }
      float o1 = v1, o2 = v2;
      if (m < 2) {
        int p;
        if (a.prefill_req < 0) p = a.rope_pos[col];
        else if (!a.rope_m3) p = col;
        else p = a.rope_pos[(i < a.sec0 ? 0 : (i < a.sec1 ? 1 : 2)) * a.ncols + col];
        p = min(max(p, 0), a.rope_max - 1);
        const float cs = a.rope_tab[((int64_t)p * half + i) * 2], sn = a.rope_tab[((int64_t)p * half + i) * 2 + 1];
        o1 = v1 * cs - v2 * sn;
        o2 = v2 * cs + v1 * sn;
      }
      if (m == 0) {
        void *q = (char *)a.out + ((int64_t)col * a.ld_out + head * hd) * (DT == HS_F32 ? 4 : 2);
        st_elem<DT>(q, i, o1);
        st_elem<DT>(q, i + half, o2);
      } else {
        const int cap = a.kv_cap[req];
        if (pos < cap) {
          const int64_t off =
              a.kv_base[req] + ((int64_t)((a.layer * 2 + (m == 2 ? 1 : 0)) * a.n_kv + head) * cap + pos) * hd;
          st_elem<DT>(a.kv, off + i, o1);
          st_elem<DT>(a.kv, off + i + half, o2);
        }
      }
    }
  }
}

// Y[c][n] = sum_k X[c][k] W[n][k] for R row tiles of 16 and NT column tiles
// of 16.  NW waves split K into interleaved 256-byte blocks; each lane streams
// 16-byte chunks of W (non-temporal: every weight byte is read once per step)
// and of X (re-read from L2), then the waves' partial tiles are summed in a
// fixed order through LDS and handed to the epilogue.
template <int DT, int R, int NT, int NW, int PRO, int EPI>
__global__ __launch_bounds__(64 * NW) void k_gemm(GemmArgs a) {
  using S = typename Ty<DT>::S;
  constexpr int CE = Ty<DT>::CE;
  constexpr int U = NT <= 2 ? 2 : 1;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int li = lane & 15, lq = lane >> 4;
  const int col0 = blockIdx.y * 16 * NT;
  const int K = a.K, kchunks = K / CE, nkb = (kchunks + 15) >> 4;

  int mat[R], row0[R];
  tile_map<EPI, R>(a, blockIdx.x, mat, row0);
  const S *wp[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int row = row0[r] + li;
    wp[r] = row < a.rows[mat[r]] ? (const S *)a.w[mat[r]] + (int64_t)row * K : nullptr;
  }

  __shared__ float s_rsq[16 * NT];
  if constexpr (PRO == PRO_NORM) {
    const float *x = (const float *)a.x;
    for (int c = wave; c < 16 * NT; c += NW) {
      const int col = col0 + c;
      float ss = 0.f;
      if (col < a.ncols) {
        const float *xr = x + (int64_t)col * K;
        for (int k = lane * 4; k < K; k += 256) {
          const f32x4 v = *(const f32x4 *)(xr + k);
          ss += v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
        }
      }
      ss = wave_sum(ss);
      if (lane == 0) s_rsq[c] = 1.0f / sqrtf(ss / (float)K + a.eps);
    }
    __syncthreads();
  }

  auto load_x = [&](int t, int kc) -> u32x4 {
    const int col = col0 + 16 * t + li;
    if (col >= a.ncols || kc >= kchunks) return u32x4{0u, 0u, 0u, 0u};
    if constexpr (PRO == PRO_PLAIN) {
      return ld16((const S *)a.x + (int64_t)col * K + (int64_t)kc * CE);
    } else {
      const float *xr = (const float *)a.x + (int64_t)col * K + (int64_t)kc * CE;
      const float rs = s_rsq[16 * t + li];
      float xv[CE], gv[CE], h[CE];
      unpack<HS_F32>(ld16(xr), xv);
      if constexpr (CE == 8) unpack<HS_F32>(ld16(xr + 4), xv + 4);
      unpack<DT>(ld16((const S *)a.gain + (int64_t)kc * CE), gv);
#pragma unroll
      for (int e = 0; e < CE; ++e) h[e] = xv[e] * rs * gv[e];
      return pack<DT>(h);
    }
  };

  f32x4 acc[R][NT];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[r][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int kb0 = wave; kb0 < nkb; kb0 += NW * U) {
    u32x4 wa[U][R][4], xb[U][NT][4];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kb = kb0 + u * NW;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const int kc = kb * 16 + lq * 4 + s;
#pragma unroll
        for (int r = 0; r < R; ++r)
          wa[u][r][s] = (wp[r] && kc < kchunks) ? ld16_stream(wp[r] + (int64_t)kc * CE) : u32x4{0u, 0u, 0u, 0u};
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kb = kb0 + u * NW;
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int t = 0; t < NT; ++t) xb[u][t][s] = load_x(t, kb * 16 + lq * 4 + s);
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
          for (int t = 0; t < NT; ++t) acc[r][t] = mma<DT>(wa[u][r][s], xb[u][t][s], acc[r][t]);
  }

  __shared__ f32x4 s_red[NW][R][NT][64];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int t = 0; t < NT; ++t) s_red[wave][r][t][lane] = acc[r][t];
  __syncthreads();
  for (int item = threadIdx.x; item < NT * 64; item += 64 * NW) {
    const int t = item >> 6, ln = item & 63;
    f32x4 v[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      v[r] = s_red[0][r][t][ln];
#pragma unroll
      for (int w = 1; w < NW; ++w) v[r] += s_red[w][r][t][ln];
    }
    const int col = col0 + 16 * t + (ln & 15);
    if (col < a.ncols) gemm_epilogue<DT, EPI, R>(a, mat, row0, v, col, 4 * (ln >> 4));
  }
}

// ---------------------------------------------------------------------------
// split-K flash-decoding attention
// ---------------------------------------------------------------------------
// One work group = (split, kv head j, query).  Its four waves stream the
// split's K rows (16-byte chunks, LPT lanes per position), score them against
// the G query heads of KV head j, form the split's softmax statistics and
// stream the V rows once for all G heads.  Outputs are the unnormalised
// partial o, the split max m and sum l.
template <int DT, int HD, int G>
__global__ __launch_bounds__(256) void k_attn(AttnArgs a) {
  using S = typename Ty<DT>::S;
  constexpr int CE = Ty<DT>::CE;
  constexpr int LPT = HD / CE;
  constexpr int TPW = 64 / LPT;
  const int split = blockIdx.x, j = blockIdx.y, qi = blockIdx.z;
  int req, L;
  if (a.prefill_req < 0) {
    req = qi;
    L = a.kv_len[qi] + 1;
  } else {
    req = a.prefill_req;
    L = qi + 1;
  }
  const int cap = a.kv_cap[req];
  L = min(L, cap);
  const int t0 = split * a.S;
  if (t0 >= L) return;
  const int n = min(a.S, L - t0);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tg = lane / LPT, c = lane % LPT;
  const S *Kp = (const S *)a.kv + a.kv_base[req] + (int64_t)((a.layer * 2) * a.n_kv + j) * cap * HD;
  const S *Vp = (const S *)a.kv + a.kv_base[req] + (int64_t)((a.layer * 2 + 1) * a.n_kv + j) * cap * HD;

  float qf[G][CE];
#pragma unroll
  for (int h = 0; h < G; ++h)
    unpack<DT>(ld16((const S *)a.q + (int64_t)qi * a.ld_q + (j * G + h) * HD + c * CE), qf[h]);

  __shared__ float s_p[G][ATTN_SMAX];
  __shared__ float s_m[G], s_l[G];
  __shared__ float s_o[4][G][HD];

  // scores

  for (int b = wave * TPW; b < n; b += 4 * TPW) {
    const int tt = b + tg;
    const bool valid = tt < n;
    float kf[CE];
    if (valid) unpack<DT>(ld16(Kp + (int64_t)(t0 + tt) * HD + c * CE), kf);
    else
#pragma unroll
      for (int e = 0; e < CE; ++e) kf[e] = 0.f;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float d = 0.f;
#pragma unroll
      for (int e = 0; e < CE; ++e) d += qf[h][e] * kf[e];
      d = group_sum<LPT>(d);
      if (valid && c == 0) s_p[h][tt] = d * a.scale;
    }
  }
  __syncthreads();

  // split softmax statistics
  for (int h = wave; h < G; h += 4) {
    float mx = -INFINITY;
    for (int i = lane; i < n; i += 64) mx = fmaxf(mx, s_p[h][i]);
    mx = wave_max(mx);
    float l = 0.f;
    for (int i = lane; i < n; i += 64) {
      const float p = expf(s_p[h][i] - mx);
      s_p[h][i] = p;
      l += p;
    }
    l = wave_sum(l);
    if (lane == 0) {
      s_m[h] = mx;
      s_l[h] = l;
    }
  }
  __syncthreads();

  // p . V
  float o[G][CE];
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < CE; ++e) o[h][e] = 0.f;

  for (int b = wave * TPW; b < n; b += 4 * TPW) {
    const int tt = b + tg;
    if (tt < n) {
      float vf[CE];
      unpack<DT>(ld16(Vp + (int64_t)(t0 + tt) * HD + c * CE), vf);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float p = s_p[h][tt];
#pragma unroll
        for (int e = 0; e < CE; ++e) o[h][e] += p * vf[e];
      }
    }
  }
#pragma unroll
  for (int off = LPT; off < 64; off <<= 1)
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < CE; ++e) o[h][e] += __shfl_xor(o[h][e], off);
  if (tg == 0)
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < CE; ++e) s_o[wave][h][c * CE + e] = o[h][e];
  __syncthreads();

  const int64_t pbase = ((int64_t)qi * a.n_heads + j * G) * a.n_split + split;
  for (int idx = threadIdx.x; idx < G * HD; idx += 256) {
    const int h = idx / HD, e = idx - h * HD;
    const float v = s_o[0][h][e] + s_o[1][h][e] + s_o[2][h][e] + s_o[3][h][e];
    a.part_o[(pbase + (int64_t)h * a.n_split) * HD + e] = v;
  }
  if (threadIdx.x < G) {
    const int h = threadIdx.x;
    a.part_ml[(pbase + (int64_t)h * a.n_split) * 2] = s_m[h];
    a.part_ml[(pbase + (int64_t)h * a.n_split) * 2 + 1] = s_l[h];
  }
}

// o = sum_s e^(m_s - M) o_s / sum_s e^(m_s - M) l_s over the splits that hold
// positions, in split order; rounded to the storage dtype.
template <int DT, int HD>
__global__ __launch_bounds__(HD) void k_combine(AttnArgs a) {
  const int h = blockIdx.x, qi = blockIdx.y, e = threadIdx.x;
  int req, L;
  if (a.prefill_req < 0) {
    req = qi;
    L = a.kv_len[qi] + 1;
  } else {
    req = a.prefill_req;
    L = qi + 1;
  }
  L = min(L, a.kv_cap[req]);
  const int ns = (L + a.S - 1) / a.S;
  const int64_t base = ((int64_t)qi * a.n_heads + h) * a.n_split;
  float M = -INFINITY;
  for (int s = 0; s < ns; ++s) M = fmaxf(M, a.part_ml[(base + s) * 2]);
  float num = 0.f, den = 0.f;
  for (int s = 0; s < ns; ++s) {
    const float w = expf(a.part_ml[(base + s) * 2] - M);
    num += w * a.part_o[(base + s) * HD + e];
    den += w * a.part_ml[(base + s) * 2 + 1];
  }
  st_elem<DT>(a.out, ((int64_t)qi * a.n_heads + h) * HD + e, num / den);
}

// ---------------------------------------------------------------------------
// embeddings, selection, bookkeeping
// ---------------------------------------------------------------------------
template <int DT>
__global__ __launch_bounds__(256) void k_embed(const void *E, int V, int d, const int *tok, float *x, int *status) {
  const int b = blockIdx.x;
  int t = tok[b];
  if (t < 0 || t >= V) {
    if (threadIdx.x == 0) atomicOr(status, 1);
    t = 0;
  }
  for (int k = threadIdx.x; k < d; k += 256) x[(int64_t)b * d + k] = ld_elem<DT>(E, (int64_t)t * d + k);
}

template <int DT>
__global__ __launch_bounds__(256) void k_prefill_rows(const void *emb, int n_v, const void *E, int V, int d,
                                                      const int *ids, float *x, int *status) {
  const int r = blockIdx.x;
  const void *src;
  int64_t row;
  if (r < n_v) {
    src = emb;
    row = r;
  } else {
    int t = ids[r - n_v];
    if (t < 0 || t >= V) {
      if (threadIdx.x == 0) atomicOr(status, 1);
      t = 0;
    }
    src = E;
    row = t;
  }
  for (int k = threadIdx.x; k < d; k += 256) x[(int64_t)r * d + k] = ld_elem<DT>(src, row * d + k);
}

// Greedy selection: largest logit, lowest index among equals (NaN never wins).
__global__ __launch_bounds__(1024) void k_argmax(const float *logits, int V, int ld, int *out, int *len, int *rope,
                                                 int advance) {
  const int b = blockIdx.x;
  const float *lg = logits + (int64_t)b * ld;
  float bv = -INFINITY;
  int bi = 0x7FFFFFFF;
  for (int i = threadIdx.x; i < V; i += 1024) {
    const float v = lg[i];
    if (v > bv) {
      bv = v;
      bi = i;
    }
  }
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(bv, off);
    const int oi = __shfl_xor(bi, off);
    if (ov > bv || (ov == bv && oi < bi)) {
      bv = ov;
      bi = oi;
    }
  }
  __shared__ float s_v[16];
  __shared__ int s_i[16];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    s_v[wave] = bv;
    s_i[wave] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 16; ++w)
      if (s_v[w] > bv || (s_v[w] == bv && s_i[w] < bi)) {
        bv = s_v[w];
        bi = s_i[w];
      }
    out[b] = bi == 0x7FFFFFFF ? 0 : bi;
    if (advance) {
      len[b] += 1;
      rope[b] += 1;
    }
  }
}

__global__ void k_advance(int *len, int *rope, int n) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < n) {
    len[b] += 1;
    rope[b] += 1;
  }
}

__global__ __launch_bounds__(256) void k_prefill_finish(int *len, int *rope, int req, int s_ctx, const int *pos_thw) {
  int mx = s_ctx - 1;
  if (pos_thw) {
    mx = 0x80000000;
    for (int i = threadIdx.x; i < 3 * s_ctx; i += 256) mx = max(mx, pos_thw[i]);
    for (int off = 32; off >= 1; off >>= 1) mx = max(mx, __shfl_xor(mx, off));
    __shared__ int s_mx[4];
    if ((threadIdx.x & 63) == 0) s_mx[threadIdx.x >> 6] = mx;
    __syncthreads();
    mx = max(max(s_mx[0], s_mx[1]), max(s_mx[2], s_mx[3]));
  }
  if (threadIdx.x == 0) {
    len[req] = s_ctx;
    rope[req] = mx + 1;
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <int DT, int R, int NT, int PRO, int EPI>
hipError_t gemm_launch(const GemmArgs &a, int n_groups, hipStream_t st) {
  constexpr int NW = 4;
  const dim3 grid(n_groups, (a.ncols + 16 * NT - 1) / (16 * NT));
  HS_LAUNCH((k_gemm<DT, R, NT, NW, PRO, EPI>), grid, dim3(64 * NW), 0, st, a);
  return hipGetLastError();
}

template <int DT, int PRO, int EPI>
hipError_t gemm_nt(const GemmArgs &a, int n_groups, hipStream_t st) {
  constexpr int R = EPI == EPI_RESID ? 1 : 2;
  const int tiles = (a.ncols + 15) / 16;
  if (tiles <= 1) return gemm_launch<DT, R, 1, PRO, EPI>(a, n_groups, st);
  if (tiles <= 2) return gemm_launch<DT, R, 2, PRO, EPI>(a, n_groups, st);
  return gemm_launch<DT, R, 4, PRO, EPI>(a, n_groups, st);
}

template <int DT>
hipError_t gemm_dt(int pro, int epi, const GemmArgs &a, int n_groups, hipStream_t st) {
  if (pro == PRO_NORM && epi == EPI_QKV) return gemm_nt<DT, PRO_NORM, EPI_QKV>(a, n_groups, st);
  if (pro == PRO_NORM && epi == EPI_SWIGLU) return gemm_nt<DT, PRO_NORM, EPI_SWIGLU>(a, n_groups, st);
  if (pro == PRO_NORM && epi == EPI_STORE) return gemm_nt<DT, PRO_NORM, EPI_STORE>(a, n_groups, st);
  if (pro == PRO_PLAIN && epi == EPI_RESID) return gemm_nt<DT, PRO_PLAIN, EPI_RESID>(a, n_groups, st);
  return hipErrorInvalidValue;
}

template <int DT, int HD>
hipError_t attn_hd(int group, int nq, const AttnArgs &a, hipStream_t st) {
  const dim3 grid(a.n_split, a.n_kv, nq);
  switch (group) {
    case 1: HS_LAUNCH((k_attn<DT, HD, 1>), grid, dim3(256), 0, st, a); break;
    case 2: HS_LAUNCH((k_attn<DT, HD, 2>), grid, dim3(256), 0, st, a); break;
    case 4: HS_LAUNCH((k_attn<DT, HD, 4>), grid, dim3(256), 0, st, a); break;
    case 7: HS_LAUNCH((k_attn<DT, HD, 7>), grid, dim3(256), 0, st, a); break;
    case 8: HS_LAUNCH((k_attn<DT, HD, 8>), grid, dim3(256), 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int DT>
hipError_t attn_dt(int head_dim, int group, int nq, const AttnArgs &a, hipStream_t st) {
  if (head_dim == 64) return attn_hd<DT, 64>(group, nq, a, st);
  if (head_dim == 128) return attn_hd<DT, 128>(group, nq, a, st);
  return hipErrorInvalidValue;
}

template <int DT>
hipError_t combine_dt(int head_dim, int nq, const AttnArgs &a, hipStream_t st) {
  const dim3 grid(a.n_heads, nq);
  if (head_dim == 64) HS_LAUNCH((k_combine<DT, 64>), grid, dim3(64), 0, st, a);
  else if (head_dim == 128) HS_LAUNCH((k_combine<DT, 128>), grid, dim3(128), 0, st, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace

bool attn_supported(int dtype, int head_dim, int group) {
  (void)dtype;
  return (head_dim == 64 || head_dim == 128) && (group == 1 || group == 2 || group == 4 || group == 7 || group == 8);
}

hipError_t launch_gemm(int dtype, int pro, int epi, const GemmArgs &a, int n_groups, hipStream_t st) {
  if (n_groups <= 0 || a.ncols <= 0) return hipSuccess;
  switch (dtype) {
    case HS_F32: return gemm_dt<HS_F32>(pro, epi, a, n_groups, st);
    case HS_F16: return gemm_dt<HS_F16>(pro, epi, a, n_groups, st);
    case HS_BF16: return gemm_dt<HS_BF16>(pro, epi, a, n_groups, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_attention(int dtype, int head_dim, int group, int nq, const AttnArgs &a, hipStream_t st) {
  if (nq <= 0) return hipSuccess;
  switch (dtype) {
    case HS_F32: return attn_dt<HS_F32>(head_dim, group, nq, a, st);
    case HS_F16: return attn_dt<HS_F16>(head_dim, group, nq, a, st);
    case HS_BF16: return attn_dt<HS_BF16>(head_dim, group, nq, a, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_combine(int dtype, int head_dim, int nq, const AttnArgs &a, hipStream_t st) {
  if (nq <= 0) return hipSuccess;
  switch (dtype) {
    case HS_F32: return combine_dt<HS_F32>(head_dim, nq, a, st);
    case HS_F16: return combine_dt<HS_F16>(head_dim, nq, a, st);
    case HS_BF16: return combine_dt<HS_BF16>(head_dim, nq, a, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_embed(int dtype, const void *embed, int vocab, int d, const int *tokens, int n, float *x, int *status,
                        hipStream_t st) {
  if (n <= 0) return hipSuccess;
  switch (dtype) {
    case HS_F32: HS_LAUNCH(k_embed<HS_F32>, dim3(n), dim3(256), 0, st, embed, vocab, d, tokens, x, status); break;
    case HS_F16: HS_LAUNCH(k_embed<HS_F16>, dim3(n), dim3(256), 0, st, embed, vocab, d, tokens, x, status); break;
    case HS_BF16: HS_LAUNCH(k_embed<HS_BF16>, dim3(n), dim3(256), 0, st, embed, vocab, d, tokens, x, status); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_prefill_rows(int dtype, const void *emb, int n_v, const void *embed, int vocab, int d,
                               const int *ids, int s_text, float *x, int *status, hipStream_t st) {
  const int rows = n_v + s_text;
  if (rows <= 0) return hipSuccess;
  switch (dtype) {
    case HS_F32: HS_LAUNCH(k_prefill_rows<HS_F32>, dim3(rows), dim3(256), 0, st, emb, n_v, embed, vocab, d, ids, x, status); break;
    case HS_F16: HS_LAUNCH(k_prefill_rows<HS_F16>, dim3(rows), dim3(256), 0, st, emb, n_v, embed, vocab, d, ids, x, status); break;
    case HS_BF16: HS_LAUNCH(k_prefill_rows<HS_BF16>, dim3(rows), dim3(256), 0, st, emb, n_v, embed, vocab, d, ids, x, status); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_argmax(const float *logits, int vocab, int ld, int n, int *tokens_out, int *len, int *rope_pos,
                         int advance, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  HS_LAUNCH(k_argmax, dim3(n), dim3(1024), 0, st, logits, vocab, ld, tokens_out, len, rope_pos, advance);
  return hipGetLastError();
}

hipError_t launch_advance(int *len, int *rope_pos, int n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  HS_LAUNCH(k_advance, dim3((n + 255) / 256), dim3(256), 0, st, len, rope_pos, n);
  return hipGetLastError();
}

hipError_t launch_prefill_finish(int *len, int *rope_pos, int req, int s_ctx, const int *pos_thw, hipStream_t st) {
  HS_LAUNCH(k_prefill_finish, dim3(1), dim3(256), 0, st, len, rope_pos, req, s_ctx, pos_thw);
  return hipGetLastError();
}

}  // namespace hs
