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
// chunk of the K row and of the V row per lane), requesting the chunks of UB
// position groups at once; the split policy sizes splits so that one such
// batch usually covers a wave's share.  Every position group keeps an online
// softmax for the G query heads of KV head j.  The groups are merged with
// lane shuffles, the waves through LDS.  With a single split the work group
// writes the normalised output; otherwise every split writes its unnormalised
// partial o, its max m and its sum l, a split past the query's positions
// writing the neutral (o = 0, m = -inf, l = 0).
// K/V are read through buffer ranges that end at the split's last position,
// so that no load sits behind a branch.
template <int DT, int HD, int G, int NW>
__global__ __launch_bounds__(64 * NW) void k_attn(AttnArgs a) {
  using S = typename Ty<DT>::S;
  constexpr int CE = Ty<DT>::CE;
  constexpr int SB = (int)sizeof(S);
  constexpr int LPT = HD / CE;
  constexpr int TPW = 64 / LPT;           // positions per wave-wide load
  constexpr int STEP = NW * TPW;          // positions per work-group iteration
  constexpr int UB = attn_batch(G);       // iterations per batch of loads
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
  const int64_t qh = (int64_t)qi * a.n_heads + j * G;  // first (query, head) row of this group
  if (t0 >= L) {
    for (int idx = threadIdx.x; idx < G * HD; idx += 64 * NW) {
      const int h = idx / HD, e = idx - h * HD;
      a.part_o[((qh + h) * a.n_split + split) * HD + e] = 0.f;
      if (e == 0) {
        a.part_ml[((qh + h) * a.n_split + split) * 2] = -INFINITY;
        a.part_ml[((qh + h) * a.n_split + split) * 2 + 1] = 0.f;
      }
    }
    return;
  }
  const int n = min(a.S, L - t0);
  const int n_it = (n + STEP - 1) / STEP;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int tg = lane / LPT, c = lane % LPT;
  const S *kbase = (const S *)a.kv + a.kv_base[req] + ((int64_t)((a.layer * 2) * a.n_kv + j) * cap + t0) * HD;
  const S *vbase = (const S *)a.kv + a.kv_base[req] + ((int64_t)((a.layer * 2 + 1) * a.n_kv + j) * cap + t0) * HD;
  const rsrc_t kr = make_rsrc(kbase, (uint32_t)n * HD * SB), vr = make_rsrc(vbase, (uint32_t)n * HD * SB);

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
    // all K and V chunks of the batch are requested before any is used;
    // positions past the split read zeros
    u32x4 kc[UB], vc[UB];
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const uint32_t off = (uint32_t)((it0 + u) * STEP + wave * TPW + tg) * (HD * SB) + (uint32_t)c * 16u;
      kc[u] = bld16_stream(kr, off);
      vc[u] = bld16_stream(vr, off);
    }
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int tt = (it0 + u) * STEP + wave * TPW + tg;
      const bool valid = tt < n;
      float kf[CE], vf[CE];
      unpack<DT>(kc[u], kf);
      unpack<DT>(vc[u], vf);
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
    if (a.n_split == 1) {
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

// o = sum_s e^(m_s - M) o_s / sum_s e^(m_s - M) l_s over the n_split splits
// of one (query, head), in split order (empty splits have weight zero);
// rounded to the storage dtype.  NSF > 0: at most NSF splits, whose partials
// are all requested at once.
template <int DT, int HD, int NSF>
__global__ __launch_bounds__(HD) void k_combine(AttnArgs a) {
  const int h = blockIdx.x, qi = blockIdx.y, e = threadIdx.x;
  const int ns = a.n_split;
  const int64_t base = ((int64_t)qi * a.n_heads + h) * ns;
  float num = 0.f, den = 0.f;
  if constexpr (NSF > 0) {
    const rsrc_t mr = make_rsrc(a.part_ml + base * 2, (uint32_t)ns * 8u);
    const rsrc_t orr = make_rsrc(a.part_o + base * HD, (uint32_t)ns * HD * 4u);
    float m[NSF], l[NSF], o[NSF];
#pragma unroll
    for (int sp = 0; sp < NSF; ++sp) {
      const u32x2 ml = bld8(mr, (uint32_t)sp * 8u);
      m[sp] = __uint_as_float(ml[0]);
      l[sp] = __uint_as_float(ml[1]);
      o[sp] = __uint_as_float(bld4(orr, (uint32_t)(sp * HD + e) * 4u));
    }
    float M = -INFINITY;
#pragma unroll
    for (int sp = 0; sp < NSF; ++sp)
      if (sp < ns) M = fmaxf(M, m[sp]);
#pragma unroll
    for (int sp = 0; sp < NSF; ++sp)
      if (sp < ns) {
        const float w = expf(m[sp] - M);
        den += w * l[sp];
        num += w * o[sp];
      }
  } else {
    __shared__ float s_m[ATTN_MAX_SPLITS], s_w[ATTN_MAX_SPLITS];
    for (int sp = e; sp < ns; sp += HD) s_m[sp] = a.part_ml[(base + sp) * 2];
    __syncthreads();
    float M = -INFINITY;
    for (int sp = 0; sp < ns; ++sp) M = fmaxf(M, s_m[sp]);
    for (int sp = e; sp < ns; sp += HD) s_w[sp] = expf(s_m[sp] - M);
    __syncthreads();
    for (int sp = 0; sp < ns; ++sp) {
      den += s_w[sp] * a.part_ml[(base + sp) * 2 + 1];
      num += s_w[sp] * a.part_o[(base + sp) * HD + e];
    }
  }
  st_elem<DT>(a.out, ((int64_t)qi * a.n_heads + h) * HD + e, num / den);
}

template <int DT, int HD>
hipError_t attn_hd(int group, int nq, const AttnArgs &a, hipStream_t st) {
  const dim3 grid(a.n_split, a.n_kv, nq), block(64 * ATTN_WAVES);
  switch (group) {
    case 1: HS_LAUNCH((k_attn<DT, HD, 1, ATTN_WAVES>), grid, block, 0, st, a); break;
    case 2: HS_LAUNCH((k_attn<DT, HD, 2, ATTN_WAVES>), grid, block, 0, st, a); break;
    case 4: HS_LAUNCH((k_attn<DT, HD, 4, ATTN_WAVES>), grid, block, 0, st, a); break;
    case 7: HS_LAUNCH((k_attn<DT, HD, 7, ATTN_WAVES>), grid, block, 0, st, a); break;
    case 8: HS_LAUNCH((k_attn<DT, HD, 8, ATTN_WAVES>), grid, block, 0, st, a); break;
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

template <int DT, int HD>
hipError_t combine_hd(int nq, const AttnArgs &a, hipStream_t st) {
  const dim3 grid(a.n_heads, nq), block(HD);
  if (a.n_split <= 8) HS_LAUNCH((k_combine<DT, HD, 8>), grid, block, 0, st, a);
  else if (a.n_split <= 16) HS_LAUNCH((k_combine<DT, HD, 16>), grid, block, 0, st, a);
  else HS_LAUNCH((k_combine<DT, HD, 0>), grid, block, 0, st, a);
  return hipGetLastError();
}

template <int DT>
hipError_t combine_dt(int head_dim, int nq, const AttnArgs &a, hipStream_t st) {
  if (head_dim == 64) return combine_hd<DT, 64>(nq, a, st);
  if (head_dim == 128) return combine_hd<DT, 128>(nq, a, st);
  return hipErrorInvalidValue;
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
