// hs_attn.hip — split-K flash-decoding attention over the per-request KV
// cache (gfx950), and the combine of its splits.
//
// Each generated token attends over all cached positions of its request, so
// decode streams the KV cache from HBM once per token (§2); the cache holds
// 2 * L * n_kv * d_h * s_ctx elements per request (Eq. 1, §4.1).  Work is
// split along the positions so that short batches still fill the GPU.
#include "hs_device.h"

namespace hs {
namespace {

using namespace dev;

// ---------------------------------------------------------------------------
// split-K flash-decoding attention
// ---------------------------------------------------------------------------
// Online-softmax state of one query head over a set of positions: running
// max m, sum l = sum_t e^(s_t - m) and unnormalised output o = sum_t e^(s_t - m) v_t.
__device__ __forceinline__ float merge_weight(float m_part, float m_all) {
  return m_part == -INFINITY ? 0.f : expf(m_part - m_all);
}

// One work group = (split, KV head j, query).  Each of its NW waves walks
// its share of the split's positions (LPT lanes per position, one 16-byte
// chunk of the K row and of the V row per lane); loads are issued a block of
// UB position groups ahead of their use (double-buffered), and every position
// group keeps an online softmax for the G query heads of KV head j.  The
// groups are merged with lane shuffles, the waves through LDS.  With a single
// split the work group writes the normalised output, otherwise the split's
// unnormalised partial o, its max m and its sum l.
template <int DT, int HD, int G, int NW>
__global__ __launch_bounds__(64 * NW) void k_attn(AttnArgs a) {
  using S = typename Ty<DT>::S;
  constexpr int CE = Ty<DT>::CE;
  constexpr int LPT = HD / CE;
  constexpr int TPW = 64 / LPT;           // positions per wave-wide load
  constexpr int STEP = NW * TPW;          // positions per work-group iteration
  constexpr int UB = G <= 2 ? 8 : 4;      // iterations per block of loads
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
  const int ns = (L + a.S - 1) / a.S;
  const int n_it = (n + STEP - 1) / STEP;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tg = lane / LPT, c = lane % LPT;
  const S *Kp = (const S *)a.kv + a.kv_base[req] + (int64_t)((a.layer * 2) * a.n_kv + j) * cap * HD + c * CE;
  const S *Vp = (const S *)a.kv + a.kv_base[req] + (int64_t)((a.layer * 2 + 1) * a.n_kv + j) * cap * HD + c * CE;

  float qf[G][CE];
#pragma unroll
  for (int h = 0; h < G; ++h)
    unpack<DT>(ld16((const S *)a.q + (int64_t)qi * a.ld_q + (j * G + h) * HD + c * CE), qf[h]);

  float m[G], l[G], o[G][CE];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = -INFINITY;
    l[h] = 0.f;
#pragma unroll
    for (int e = 0; e < CE; ++e) o[h][e] = 0.f;
  }
  for (int it0 = 0; it0 < n_it; it0 += UB) {
    // all K and V chunks of the block are requested before any is used
    u32x4 kr[UB], vr[UB];
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int tt = (it0 + u) * STEP + wave * TPW + tg;
      if (it0 + u < n_it && tt < n) {
        kr[u] = ld16(Kp + (int64_t)(t0 + tt) * HD);
        vr[u] = ld16(Vp + (int64_t)(t0 + tt) * HD);
      } else {
        kr[u] = vr[u] = u32x4{0u, 0u, 0u, 0u};
      }
    }
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int tt = (it0 + u) * STEP + wave * TPW + tg;
      const bool valid = it0 + u < n_it && tt < n;
      float kf[CE], vf[CE];
      unpack<DT>(kr[u], kf);
      unpack<DT>(vr[u], vf);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        float d = 0.f;
#pragma unroll
        for (int e = 0; e < CE; ++e) d += qf[h][e] * kf[e];
        d = group_sum<LPT>(d);
        if (valid) {
          const float sc = d * a.scale;
          const float mn = fmaxf(m[h], sc);
          const float corr = merge_weight(m[h], mn);
          const float p = expf(sc - mn);
          l[h] = l[h] * corr + p;
#pragma unroll
          for (int e = 0; e < CE; ++e) o[h][e] = o[h][e] * corr + p * vf[e];
          m[h] = mn;
        }
      }
    }
  }
  // merge the TPW position groups of the wave (lanes with the same chunk c)
#pragma unroll
  for (int off = LPT; off < 64; off <<= 1) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float m2 = __shfl_xor(m[h], off), l2 = __shfl_xor(l[h], off);
      const float mn = fmaxf(m[h], m2);
      const float w1 = merge_weight(m[h], mn), w2 = merge_weight(m2, mn);
      l[h] = l[h] * w1 + l2 * w2;
#pragma unroll
      for (int e = 0; e < CE; ++e) o[h][e] = o[h][e] * w1 + __shfl_xor(o[h][e], off) * w2;
      m[h] = mn;
    }
  }
  __shared__ float s_m[NW][G], s_l[NW][G];
  __shared__ float s_o[NW][G][HD];
  if (tg == 0)
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < CE; ++e) s_o[wave][h][c * CE + e] = o[h][e];
  if (lane == 0)
#pragma unroll
    for (int h = 0; h < G; ++h) {
      s_m[wave][h] = m[h];
      s_l[wave][h] = l[h];
    }
  __syncthreads();

  const int64_t qh = (int64_t)qi * a.n_heads + j * G;  // first (query, head) row of this group
  for (int idx = threadIdx.x; idx < G * HD; idx += 64 * NW) {
    const int h = idx / HD, e = idx - h * HD;
    float M = s_m[0][h];
#pragma unroll
    for (int w = 1; w < NW; ++w) M = fmaxf(M, s_m[w][h]);
    float num = 0.f, den = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float wt = merge_weight(s_m[w][h], M);
      num += wt * s_o[w][h][e];
      den += wt * s_l[w][h];
    }
    if (ns == 1) {
      st_elem<DT>(a.out, (qh + h) * HD + e, num / den);
    } else {
      a.part_o[((qh + h) * a.n_split + split) * HD + e] = num;
      if (e == 0) {
        a.part_ml[((qh + h) * a.n_split + split) * 2] = M;
        a.part_ml[((qh + h) * a.n_split + split) * 2 + 1] = den;
      }
    }
  }
}

// o = sum_s e^(m_s - M) o_s / sum_s e^(m_s - M) l_s over the splits that hold
// positions, in split order; rounded to the storage dtype.  Queries whose
// positions fit one split were finished by the attention kernel.
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
  if (ns <= 1) return;
  const int64_t base = ((int64_t)qi * a.n_heads + h) * a.n_split;
  __shared__ float s_m[ATTN_MAX_SPLITS], s_w[ATTN_MAX_SPLITS];
  __shared__ float s_den;
  for (int sp = e; sp < ns; sp += HD) s_m[sp] = a.part_ml[(base + sp) * 2];
  __syncthreads();
  float M = -INFINITY;
  for (int sp = 0; sp < ns; ++sp) M = fmaxf(M, s_m[sp]);
  for (int sp = e; sp < ns; sp += HD) s_w[sp] = expf(s_m[sp] - M);
  __syncthreads();
  if (e == 0) {
    float den = 0.f;
    for (int sp = 0; sp < ns; ++sp) den += s_w[sp] * a.part_ml[(base + sp) * 2 + 1];
    s_den = den;
  }
  float num = 0.f;
  for (int sp = 0; sp < ns; ++sp) num += s_w[sp] * a.part_o[(base + sp) * HD + e];
  __syncthreads();
  st_elem<DT>(a.out, ((int64_t)qi * a.n_heads + h) * HD + e, num / s_den);
}

template <int DT, int HD>
hipError_t attn_hd(int group, int nq, const AttnArgs &a, hipStream_t st) {
  const dim3 grid(a.n_split, a.n_kv, nq);
  const bool wide = a.waves == ATTN_WAVES_WIDE;
  switch (group) {
    case 1:
      if (wide) HS_LAUNCH((k_attn<DT, HD, 1, ATTN_WAVES_WIDE>), grid, dim3(64 * ATTN_WAVES_WIDE), 0, st, a);
      else HS_LAUNCH((k_attn<DT, HD, 1, ATTN_WAVES>), grid, dim3(64 * ATTN_WAVES), 0, st, a);
      break;
    case 2:
      if (wide) HS_LAUNCH((k_attn<DT, HD, 2, ATTN_WAVES_WIDE>), grid, dim3(64 * ATTN_WAVES_WIDE), 0, st, a);
      else HS_LAUNCH((k_attn<DT, HD, 2, ATTN_WAVES>), grid, dim3(64 * ATTN_WAVES), 0, st, a);
      break;
    case 4: HS_LAUNCH((k_attn<DT, HD, 4, ATTN_WAVES>), grid, dim3(64 * ATTN_WAVES), 0, st, a); break;
    case 7: HS_LAUNCH((k_attn<DT, HD, 7, ATTN_WAVES>), grid, dim3(64 * ATTN_WAVES), 0, st, a); break;
    case 8: HS_LAUNCH((k_attn<DT, HD, 8, ATTN_WAVES>), grid, dim3(64 * ATTN_WAVES), 0, st, a); break;
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
  if (nq <= 0 || a.n_split <= 1) return hipSuccess;
  switch (dtype) {
    case HS_F32: return combine_dt<HS_F32>(head_dim, nq, a, st);
    case HS_F16: return combine_dt<HS_F16>(head_dim, nq, a, st);
    case HS_BF16: return combine_dt<HS_BF16>(head_dim, nq, a, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace hs
