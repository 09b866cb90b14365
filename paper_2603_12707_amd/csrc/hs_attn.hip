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

}  // namespace hs
