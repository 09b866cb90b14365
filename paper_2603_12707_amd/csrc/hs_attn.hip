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

// element (row, c) of the combined output: rows of n_heads * head_dim, or the
// packed activation layout the O projection reads at 2..32 columns
__device__ __forceinline__ int64_t attn_out_at(const AttnArgs &a, int64_t row, int c, int hd) {
  const int K = a.n_heads * hd;
  return a.out_packed ? packed_x_index((int)row, c, (K / 8 + 15) / 16) : row * K + c;
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
// so that no load sits behind a branch.  In a cache of several blocks per
// request (PAGED) a batch of loads always lies in one block and gets a range
// of its own, the block's start read one batch ahead.  In decode, work-group
// row z serves the z-th longest request (a.order).
template <int DT, int HD, int G, int NW, bool PAGED>
__global__ __launch_bounds__(64 * NW) void k_attn(AttnArgs a) {
  using S = typename Ty<DT>::S;
  constexpr int CE = Ty<DT>::CE;
  constexpr int SB = (int)sizeof(S);
  constexpr int LPT = HD / CE;
  constexpr int TPW = 64 / LPT;           // positions per wave-wide load
  constexpr int STEP = NW * TPW;          // positions per work-group iteration
  constexpr int UB = attn_batch(G);       // iterations per batch of loads
  // decode: the longest requests' work groups are dispatched first
  const int split = blockIdx.x, j = blockIdx.y, qi = a.order ? a.order[blockIdx.z] : (int)blockIdx.z;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int tg = lane / LPT, c = lane % LPT;
  // the query chunks are requested first (also by a split past the end,
  // which does not use them) and unpacked once the batch's K/V loads are in
  // flight, so their latency overlaps the cache metadata and K/V loads
  u32x4 qraw[G];
#pragma unroll
  for (int h = 0; h < G; ++h) qraw[h] = ld16((const S *)a.q + (int64_t)qi * a.ld_q + (j * G + h) * HD + c * CE);
  // the request's length, capacity and (contiguous cache) first element,
  // requested together
  // (16-bit storage prefills through k_attn_prefill: here a.prefill is set
  // for fp32 alone, and the 16-bit kernels compile the decode path only)
  int req, last;  // last: the query's position
  if (DT != HS_F32 || !a.prefill) {
    req = PAGED ? a.kv.act[qi] : qi;
    last = a.kv.len[req];
  } else {
    const int i = packed_request(a.pk, qi);
    req = a.pk->req[i];
    last = qi - a.pk->cu[i];
  }
  const int cap = a.kv.cap[req];
  const int64_t b_req = PAGED ? 0 : a.kv.tab[req];
  // the three loads issued together, one wait (a paged cache reads its block
  // table in the loop, whose loads the pin would turn into vector loads)
  if constexpr (!PAGED) asm volatile("" ::"s"(last), "s"(cap), "s"(b_req));
  const int L = min(last + 1, cap);
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
  // one block per request: the split's rows are one range.  Several blocks:
  // each batch of loads (a whole number of which fills a block) reads the
  // block holding it, whose start is read one batch ahead.
  int64_t ko = 0, vo = 0;
  int bt = 0, toff = 0;
  int64_t kin = 0, vin = 0, b_next = 0;
  if constexpr (PAGED) {
    bt = a.kv.bt[req];
    toff = a.kv.toff[req];
    kin = (int64_t)((a.layer * 2) * a.n_kv + j) * bt * HD;
    vin = kin + (int64_t)a.n_kv * bt * HD;
    b_next = a.kv.tab[toff + t0 / bt];
  } else {
    ko = b_req + ((int64_t)((a.layer * 2) * a.n_kv + j) * cap + t0) * HD;
    vo = ko + (int64_t)a.n_kv * cap * HD;
  }
  const uint32_t nbytes = (uint32_t)n * HD * SB;
  const rsrc_t kr = make_rsrc((const S *)a.kv.buf + max(ko, (int64_t)0), nbytes);
  const rsrc_t vr = make_rsrc((const S *)a.kv.buf + max(vo, (int64_t)0), nbytes);

  float qf[G][CE];

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
    rsrc_t kb = kr, vb = vr;
    int rel = 0;
    bool blk_ok = true;  // a paged batch's block is held (a pool that ran dry leaves it unheld)
    if constexpr (PAGED) {
      const int64_t b0 = b_next;
      blk_ok = b0 >= 0;
      const int pb = t0 + it0 * STEP, pn = pb + UB * STEP;
      b_next = pn < t0 + n ? a.kv.tab[toff + pn / bt] : 0;
      const int64_t at = max(b0, (int64_t)0) + (int64_t)(pb % bt) * HD;
      const uint32_t bytes = b0 < 0 ? 0u : (uint32_t)min(UB * STEP, n - it0 * STEP) * HD * SB;
      kb = make_rsrc((const S *)a.kv.buf + at + kin, bytes);
      vb = make_rsrc((const S *)a.kv.buf + at + vin, bytes);
      rel = it0 * STEP;
    }
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const uint32_t off = (uint32_t)((it0 + u) * STEP - rel + wave * TPW + tg) * (HD * SB) + (uint32_t)c * 16u;
      kc[u] = bld16_stream(kb, off);
      vc[u] = bld16_stream(vb, off);
    }
    // opaque to the compiler: keeps the unpack (and its wait) here, behind the loads
#pragma unroll
    for (int h = 0; h < G; ++h) {
      asm volatile("" : "+v"(qraw[h]));
      unpack<DT>(qraw[h], qf[h]);
    }
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int tt = (it0 + u) * STEP + wave * TPW + tg;
      const bool valid = tt < n && blk_ok;  // positions of an unheld block are masked
      float kf[CE], vf[CE];
      unpack<DT>(kc[u], kf);
      unpack<DT>(vc[u], vf);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        float d = 0.f;
#pragma unroll
        for (int e = 0; e < CE; ++e) d += qf[h][e] * kf[e];
        d = group_sum<LPT>(d);
        // branch-free update: a position past the split (zero K/V rows)
        // leaves the state as it is (a branch here let the compiler move a
        // V load behind it, with a wait for every load in flight)
        const float sc = valid ? d * a.scale : -INFINITY;
        const float mn = fmaxf(m[h], sc);
        const float corr = merge_weight(m[h], mn);
        const float p = valid ? expf(sc - mn) : 0.f;
        l[h] = l[h] * corr + p;
#pragma unroll
        for (int e = 0; e < CE; ++e) o[h][e] = o[h][e] * corr + p * vf[e];
        m[h] = mn;
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
      st_elem<DT>(a.out, attn_out_at(a, qi, (j * G + h) * HD + e, HD), num / den);
    } else {
      a.part_o[((qh + h) * a.n_split + split) * HD + e] = num;
      if (e == 0) {
        a.part_ml[((qh + h) * a.n_split + split) * 2] = M;
        a.part_ml[((qh + h) * a.n_split + split) * 2 + 1] = den;
      }
    }
  }
}

// storage-dtype parts the softmax probabilities enter the PV product as
template <int DT>
constexpr int P_PARTS = DT == HS_BF16 ? 3 : 2;

// Attention for query-head groups of 4..16 heads on the matrix cores.  One
// work group = (split, KV head j, query), as above; each wave takes tiles of 16
// consecutive positions.  Per tile, the scores of the tile's positions for all
// heads of the group are S^T = K Q^T (16 positions x 16 head slots, MFMA
// 16x16x32: exact products of the stored 16-bit values, fp32 sums).  A lane
// then holds the scores of positions 4 q .. 4 q + 3 (q = lane / 16) for head
// lane % 16 -- exactly the B-operand layout of the 16x16x16 MFMA that updates
// O^T (d x heads) += V^T P^T, so the online-softmax probabilities feed the
// matrix cores from registers.  That MFMA takes 16-bit operands, so P enters
// as the sum of storage-dtype parts, p = hi + lo (+ lo2) with hi = R(p),
// lo = R(p - hi), lo2 = R(p - hi - lo), one MFMA each: the products with the
// stored V values are exact and p keeps ~22 (fp16, two parts) or ~24 (bf16,
// three parts) significant bits, against fp32 in the definition (a single
// rounding of p to bf16 doubled the error of o and, over 28 layers, the
// error of the residual stream; two bf16 parts left the Qwen-shaped logits
// 1.8 % from the oracle, three 1.2 %).  l sums the parts, so o stays a
// weighted mean of the V rows.  For the V^T operand a lane loads
// chunk c = lane % 16 of the 4 positions it covers, and output row c of d-tile
// dt is element d = 8 c + dt, which a lane gathers from its four chunks.
// The waves merge through LDS as in k_attn.
template <int DT, int HD, int G, int NW, bool PAGED>
__global__ __launch_bounds__(64 * NW) void k_attn_mma(AttnArgs a) {
  static_assert(DT != HS_F32 && G <= 16 && (HD == 64 || HD == 128), "16-bit storage, at most 16 heads per group");
  constexpr int SB = 2;
  constexpr int CPR = HD / 8;         // 16-byte chunks per row
  constexpr int KK = HD / 32;         // 32-wide k steps of the scores
  constexpr int UB = ATTN_MMA_BATCH;  // tiles per batch of loads
  constexpr int STEP = NW * 16;       // positions per work-group iteration
  // decode: the longest requests' work groups are dispatched first
  const int split = blockIdx.x, j = blockIdx.y, qi = a.order ? a.order[blockIdx.z] : (int)blockIdx.z;
  // (16-bit storage prefills through k_attn_prefill: here a.prefill is set
  // for fp32 alone, and the 16-bit kernels compile the decode path only)
  int req, last;  // last: the query's position
  if (DT != HS_F32 || !a.prefill) {
    req = PAGED ? a.kv.act[qi] : qi;
    last = a.kv.len[req];
  } else {
    const int i = packed_request(a.pk, qi);
    req = a.pk->req[i];
    last = qi - a.pk->cu[i];
  }
  // the request's length, capacity and (contiguous cache) first element,
  // requested together, one wait
  const int cap = a.kv.cap[req];
  const int64_t b_req = PAGED ? 0 : a.kv.tab[req];
  if constexpr (!PAGED) asm volatile("" ::"s"(last), "s"(cap), "s"(b_req));  // as in k_attn
  const int L = min(last + 1, cap);
  const int t0 = split * a.S;
  const int64_t qh = (int64_t)qi * a.n_heads + j * G;
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
  const int li = lane & 15, lg = lane >> 4;
  // one block per request: the split's rows are one range.  Several blocks:
  // each batch of loads (a whole number of which fills a block) reads the
  // block holding it, whose start is read one batch ahead.
  int64_t ko = 0, vo = 0;
  int bt = 0, toff = 0;
  int64_t kin = 0, vin = 0, b_next = 0;
  if constexpr (PAGED) {
    bt = a.kv.bt[req];
    toff = a.kv.toff[req];
    kin = (int64_t)((a.layer * 2) * a.n_kv + j) * bt * HD;
    vin = kin + (int64_t)a.n_kv * bt * HD;
    b_next = a.kv.tab[toff + t0 / bt];
  } else {
    ko = b_req + ((int64_t)((a.layer * 2) * a.n_kv + j) * cap + t0) * HD;
    vo = ko + (int64_t)a.n_kv * cap * HD;
  }
  const uint32_t nbytes = (uint32_t)n * HD * SB;
  const rsrc_t kr = make_rsrc((const uint16_t *)a.kv.buf + max(ko, (int64_t)0), nbytes);
  const rsrc_t vr = make_rsrc((const uint16_t *)a.kv.buf + max(vo, (int64_t)0), nbytes);

  // Q^T operand: head lane % 16 of the group (zero past G), k = 32 kk + 8 q ..
  u32x4 qb[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk)
    qb[kk] = li < G ? ld16((const uint16_t *)a.q + (int64_t)qi * a.ld_q + (j * G + li) * HD + (kk * 4 + lg) * 8)
                    : u32x4{0u, 0u, 0u, 0u};

  float m = -INFINITY, l = 0.f;
  f32x4 o[8];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int it0 = 0; it0 < n_it; it0 += UB) {
    // every K and V chunk of the batch is requested before any is used;
    // positions past the split read zeros
    u32x4 kc[UB][KK], vc[UB][4];
    rsrc_t kb = kr, vb = vr;
    int rel = 0;
    bool blk_ok = true;  // as in k_attn
    if constexpr (PAGED) {
      const int64_t b0 = b_next;
      blk_ok = b0 >= 0;
      const int pb = t0 + it0 * STEP, pn = pb + UB * STEP;
      b_next = pn < t0 + n ? a.kv.tab[toff + pn / bt] : 0;
      const int64_t at = max(b0, (int64_t)0) + (int64_t)(pb % bt) * HD;
      const uint32_t bytes = b0 < 0 ? 0u : (uint32_t)min(UB * STEP, n - it0 * STEP) * HD * SB;
      kb = make_rsrc((const uint16_t *)a.kv.buf + at + kin, bytes);
      vb = make_rsrc((const uint16_t *)a.kv.buf + at + vin, bytes);
      rel = it0 * STEP;
    }
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int p0 = ((it0 + u) * NW + wave) * 16 - rel;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk)
        kc[u][kk] = bld16_stream(kb, (uint32_t)((p0 + li) * HD + (kk * 4 + lg) * 8) * SB);
#pragma unroll
      for (int i = 0; i < 4; ++i)
        vc[u][i] = bld16_stream(vb, li < CPR ? (uint32_t)((p0 + 4 * lg + i) * HD + li * 8) * SB : BUF_OOB);
    }
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int p0 = ((it0 + u) * NW + wave) * 16;
      f32x4 sc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) sc = mma<DT>(kc[u][kk], qb[kk], sc);
      float sv[4];
      float tmax = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        sv[i] = p0 + 4 * lg + i < n && blk_ok ? sc[i] * a.scale : -INFINITY;
        tmax = fmaxf(tmax, sv[i]);
      }
      tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
      const float mn = fmaxf(m, tmax);
      const float corr = m == -INFINITY ? 0.f : __expf(m - mn);
      float pr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) pr[i] = sv[i] == -INFINITY ? 0.f : __expf(sv[i] - mn);
      // the PV operands: p = hi + lo (+ lo2 in bf16) in the storage dtype;
      // l sums the parts
      u32x2 ph = u32x2{0u, 0u}, pl = u32x2{0u, 0u}, pt = u32x2{0u, 0u};
      float ps = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t hb = DT == HS_F16 ? f32_to_f16(pr[i]) : f32_to_bf16(pr[i]);
        const float hf = DT == HS_F16 ? f16_to_f32(hb) : bf16_to_f32(hb);
        const uint32_t lb = DT == HS_F16 ? f32_to_f16(pr[i] - hf) : f32_to_bf16(pr[i] - hf);
        const float lf = DT == HS_F16 ? f16_to_f32(lb) : bf16_to_f32(lb);
        if constexpr (P_PARTS<DT> == 3) {
          const uint32_t tb = f32_to_bf16(pr[i] - hf - lf);
          ps += hf + lf + bf16_to_f32(tb);
          pt[i >> 1] |= tb << (16 * (i & 1));
        } else {
          ps += hf + lf;
        }
        ph[i >> 1] |= hb << (16 * (i & 1));
        pl[i >> 1] |= lb << (16 * (i & 1));
      }
      ps += __shfl_xor(ps, 16);
      ps += __shfl_xor(ps, 32);
      l = l * corr + ps;
      m = mn;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        o[dt] *= corr;
        // V^T rows: element dt of chunk lane % 16 of the 4 positions
        const int w = dt >> 1, sh = 16 * (dt & 1);
        u32x2 av;
        av[0] = ((vc[u][0][w] >> sh) & 0xFFFFu) | (((vc[u][1][w] >> sh) & 0xFFFFu) << 16);
        av[1] = ((vc[u][2][w] >> sh) & 0xFFFFu) | (((vc[u][3][w] >> sh) & 0xFFFFu) << 16);
        o[dt] = mma16<DT>(av, ph, o[dt]);
        o[dt] = mma16<DT>(av, pl, o[dt]);
        if constexpr (P_PARTS<DT> == 3) o[dt] = mma16<DT>(av, pt, o[dt]);
      }
    }
  }

  __shared__ float s_m[NW][16], s_l[NW][16];
  __shared__ float s_o[NW][16][HD + 1];
  if (lg == 0) {
    s_m[wave][li] = m;
    s_l[wave][li] = l;
  }
#pragma unroll
  for (int dt = 0; dt < 8; ++dt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int d = (4 * lg + i) * 8 + dt;
      if (d < HD) s_o[wave][li][d] = o[dt][i];
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
      st_elem<DT>(a.out, attn_out_at(a, qi, (j * G + h) * HD + e, HD), num / den);
    } else {
      a.part_o[((qh + h) * a.n_split + split) * HD + e] = num;
      if (e == 0) {
        a.part_ml[((qh + h) * a.n_split + split) * 2] = M;
        a.part_ml[((qh + h) * a.n_split + split) * 2 + 1] = den;
      }
    }
  }
}

// Prefill attention on the matrix cores (causal: row r of the request attends
// to rows 0..r).  The 16 MFMA columns of a query tile hold QPT = 16 / G
// consecutive query rows x the G query heads of KV head j.  A work group
// takes two consecutive query tiles of one request; its NW waves walk the key
// tiles of 16 positions up to the pair's last row between them, each K/V tile
// loaded once for both query tiles, masking the keys past each row, each wave
// with an online softmax per query tile; the waves' states merge through LDS
// at the end.  Operand layouts and the split of p into storage-dtype parts
// are those of k_attn_mma, so the K/V rows a wave loads serve 2 x QPT x G
// (query, head) pairs at once.
// Slack (in units of the natural-log score) by which a column's scores may
// pass the running maximum before it is raised: exp(s - m) stays below e^8.
constexpr float RESCALE_SLACK = 8.f;

template <int DT, int HD, int G, int NW>
__global__ __launch_bounds__(64 * NW, 2) void k_attn_prefill(AttnArgs a) {
  static_assert(DT != HS_F32 && G <= 16 && (HD == 64 || HD == 128), "16-bit storage, at most 16 heads per group");
  constexpr int SB = 2;
  constexpr int CPR = HD / 8;
  constexpr int KK = HD / 32;
  constexpr int UB = ATTN_MMA_BATCH;
  constexpr int QPT = 16 / G;  // query rows per tile
  constexpr int QT = 2;        // query tiles per work group
  static_assert(NW >= QT, "one merging wave per query tile");
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int li = lane & 15, lg = lane >> 4;
  // The work group's item w = (KV head j, tile pair pp).  Work groups are
  // dealt to the 8 XCDs round robin; the order below gives each XCD one run
  // of consecutive items, so that the query tiles of a head, which all read
  // its K/V rows, share that XCD's L2.  Within a head the last pairs come
  // first, so that the long causal rows start early.
  const int np = a.prefill_pairs;
  const int total = np * a.n_kv, nq = total >> 3, nr = total & 7;
  const int xcd = (int)blockIdx.x & 7;
  const int w = (xcd < nr ? xcd * (nq + 1) : nr * (nq + 1) + (xcd - nr) * nq) + ((int)blockIdx.x >> 3);
  const int j = w / np;
  const int pp = np - 1 - (w - j * np);
  // packed request i holds pairs [pbase_i, pbase_i + ceil(tiles_i / 2))
  const PackedRows *pk = a.pk;
  int pi = 0, pbase = 0;
  for (int k = 0; k + 1 < pk->n; ++k) {
    const int npk = (pk->tcu[k + 1] - pk->tcu[k] + 1) >> 1;
    if (pi == k && pp >= pbase + npk) {
      pbase += npk;
      pi = k + 1;
    }
  }
  const int roff = pk->cu[pi], nrows = pk->cu[pi + 1] - roff;
  const int ntiles = pk->tcu[pi + 1] - pk->tcu[pi];
  const int req = pk->req[pi];
  const int lt0 = 2 * (pp - pbase);  // the pair's tiles lt0, lt0 + 1 of the request (the second may not exist)
  const int sh = li % G;             // the lane column's head
  int sq[QT];
  bool slot[QT];
#pragma unroll
  for (int s = 0; s < QT; ++s) {
    sq[s] = (lt0 + s) * QPT + li / G;  // the lane column's query position in tile s
    slot[s] = lt0 + s < ntiles && li < QPT * G && sq[s] < nrows;
  }
  const int qlast = min(min(lt0 + QT, ntiles) * QPT - 1, nrows - 1);  // the pair's last row
  const int n_kt = qlast / 16 + 1;                                   // key tiles
  // key tiles are read block by block (a block holds a whole number of tiles)
  const int bt = a.kv.bt[req], toff = a.kv.toff[req];
  const int64_t kin = (int64_t)((a.layer * 2) * a.n_kv + j) * bt * HD, vin = kin + (int64_t)a.n_kv * bt * HD;
  const uint16_t *buf = (const uint16_t *)a.kv.buf;

  u32x4 qb[QT][KK];
#pragma unroll
  for (int s = 0; s < QT; ++s)
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
      qb[s][kk] = slot[s] ? ld16((const uint16_t *)a.q + (int64_t)(roff + sq[s]) * a.ld_q + (j * G + sh) * HD +
                                 (kk * 4 + lg) * 8)
                          : u32x4{0u, 0u, 0u, 0u};

  float m[QT], l[QT];
  f32x4 o[QT][8];
#pragma unroll
  for (int s = 0; s < QT; ++s) {
    m[s] = -INFINITY;
    l[s] = 0.f;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[s][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // Key tiles in batches of UB per wave: the wave takes tiles kt0 + u NW +
  // wave.  Past the pair's last key every load is empty and reads as zero.
  constexpr int STEP = UB * NW;
  for (int kt0 = 0; kt0 < n_kt; kt0 += STEP) {
    u32x4 kc[UB][KK], vc[UB][4];
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int p0 = (kt0 + u * NW + wave) * 16, blk = p0 / bt, pb = p0 - blk * bt;
      const int64_t b0 = p0 <= qlast ? a.kv.tab[toff + blk] : -1;
      // rows of the block up to the pair's last query position; past them, zeros
      const uint32_t nbytes = b0 < 0 ? 0u : (uint32_t)min(bt, qlast + 1 - blk * bt) * HD * SB;
      const rsrc_t kr = make_rsrc(buf + max(b0, (int64_t)0) + kin, nbytes);
      const rsrc_t vr = make_rsrc(buf + max(b0, (int64_t)0) + vin, nbytes);
#pragma unroll
      for (int kk = 0; kk < KK; ++kk)
        kc[u][kk] = bld16(kr, (uint32_t)((pb + li) * HD + (kk * 4 + lg) * 8) * SB);
#pragma unroll
      for (int i = 0; i < 4; ++i)
        vc[u][i] = bld16(vr, li < CPR ? (uint32_t)((pb + 4 * lg + i) * HD + li * 8) * SB : BUF_OOB);
    }
    // scores of the batch's key tiles for both query tiles, their chains
    // interleaved (past a row every score is masked and the state stays)
    f32x4 sc[QT][UB];
#pragma unroll
    for (int s = 0; s < QT; ++s)
#pragma unroll
      for (int u = 0; u < UB; ++u) sc[s][u] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
#pragma unroll
      for (int s = 0; s < QT; ++s)
#pragma unroll
        for (int u = 0; u < UB; ++u) sc[s][u] = mma<DT>(kc[u][kk], qb[s][kk], sc[s][u]);
    u32x2 ph[QT][UB], pl[QT][UB], pt[QT][UB];
#pragma unroll
    for (int s = 0; s < QT; ++s) {
      float sv[UB][4];
      float tmax = -INFINITY;
#pragma unroll
      for (int u = 0; u < UB; ++u)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int p = (kt0 + u * NW + wave) * 16 + 4 * lg + i;
          sv[u][i] = slot[s] && p <= sq[s] ? sc[s][u][i] * a.scale : -INFINITY;
          tmax = fmaxf(tmax, sv[u][i]);
        }
      // o / l does not depend on the reference m as long as exp(s - m) stays
      // in range.  m, the same for the four lanes of a column, is raised to
      // the column's maximum (and o, l rescaled) only when some score of the
      // wave passes it by more than RESCALE_SLACK.
      if (__ballot(tmax > m[s] + RESCALE_SLACK)) {
        tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
        tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
        const float mn = fmaxf(m[s], tmax);
        const float corr = m[s] == -INFINITY ? 0.f : __expf(m[s] - mn);
        l[s] *= corr;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) o[s][dt] *= corr;
        m[s] = mn;
      }
#pragma unroll
      for (int u = 0; u < UB; ++u) {
        ph[s][u] = u32x2{0u, 0u};
        pl[s][u] = u32x2{0u, 0u};
        pt[s][u] = u32x2{0u, 0u};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float pr = sv[u][i] == -INFINITY ? 0.f : __expf(sv[u][i] - m[s]);
          const uint32_t hb = DT == HS_F16 ? f32_to_f16(pr) : f32_to_bf16(pr);
          const float hf = DT == HS_F16 ? f16_to_f32(hb) : bf16_to_f32(hb);
          const uint32_t lb = DT == HS_F16 ? f32_to_f16(pr - hf) : f32_to_bf16(pr - hf);
          const float lf = DT == HS_F16 ? f16_to_f32(lb) : bf16_to_f32(lb);
          if constexpr (P_PARTS<DT> == 3) {  // this lane's keys only
            const uint32_t tb = f32_to_bf16(pr - hf - lf);
            l[s] += hf + lf + bf16_to_f32(tb);
            pt[s][u][i >> 1] |= tb << (16 * (i & 1));
          } else {
            l[s] += hf + lf;
          }
          ph[s][u][i >> 1] |= hb << (16 * (i & 1));
          pl[s][u][i >> 1] |= lb << (16 * (i & 1));
        }
      }
    }
#pragma unroll
    for (int u = 0; u < UB; ++u)
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        // the 16-bit element dt of keys 4 lg .. 4 lg + 3, low half first
        const int w2 = dt >> 1;
        const uint32_t sel = dt & 1 ? 0x07060302u : 0x05040100u;
        u32x2 av;
        av[0] = __builtin_amdgcn_perm(vc[u][1][w2], vc[u][0][w2], sel);
        av[1] = __builtin_amdgcn_perm(vc[u][3][w2], vc[u][2][w2], sel);
#pragma unroll
        for (int s = 0; s < QT; ++s) {
          o[s][dt] = mma16<DT>(av, ph[s][u], o[s][dt]);
          o[s][dt] = mma16<DT>(av, pl[s][u], o[s][dt]);
          if constexpr (P_PARTS<DT> == 3) o[s][dt] = mma16<DT>(av, pt[s][u], o[s][dt]);
        }
      }
  }
  // l so far covers this lane's keys; the column's sum adds the four lanes
#pragma unroll
  for (int s = 0; s < QT; ++s) {
    l[s] += __shfl_xor(l[s], 16);
    l[s] += __shfl_xor(l[s], 32);
  }
  // merge the waves' states in wave order: M = max m_w, o = sum_w e^(m_w - M) o_w,
  // l = sum_w e^(m_w - M) l_w; wave s merges query tile s
  __shared__ float s_ml[NW][QT][2][64];
  __shared__ f32x4 s_o[NW][QT][8][64];
#pragma unroll
  for (int s = 0; s < QT; ++s) {
    s_ml[wave][s][0][lane] = m[s];
    s_ml[wave][s][1][lane] = l[s];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) s_o[wave][s][dt][lane] = o[s][dt];
  }
  __syncthreads();
  if (wave >= QT) return;
  const int ms = wave;  // wave-uniform
  bool my_slot = false;
  int my_sq = 0;
#pragma unroll
  for (int s = 0; s < QT; ++s)
    if (s == ms) {
      my_slot = slot[s];
      my_sq = sq[s];
    }
  if (!my_slot) return;
  float M = s_ml[0][ms][0][lane];
#pragma unroll
  for (int w2 = 1; w2 < NW; ++w2) M = fmaxf(M, s_ml[w2][ms][0][lane]);
  float L = 0.f;
  f32x4 O[8];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) O[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int w2 = 0; w2 < NW; ++w2) {
    const float mw = s_ml[w2][ms][0][lane];
    const float wt = mw == -INFINITY ? 0.f : __expf(mw - M);
    L += wt * s_ml[w2][ms][1][lane];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) O[dt] += wt * s_o[w2][ms][dt][lane];
  }
  // lane (c, q) holds rows d = (4 q + i) * 8 + dt of its column's output
  const int64_t orow = roff + my_sq;
  const int ocol = (j * G + sh) * HD;
#pragma unroll
  for (int dt = 0; dt < 8; ++dt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int d = (4 * lg + i) * 8 + dt;
      if (d < HD) st_elem<DT>(a.out, attn_out_at(a, orow, ocol + d, HD), O[dt][i] / L);
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
  st_elem<DT>(a.out, attn_out_at(a, qi, h * HD + e, HD), num / den);
}

template <int DT, int HD, bool PAGED>
hipError_t attn_hd(int group, int nq, const AttnArgs &a, hipStream_t st) {
  if (DT != HS_F32 && a.prefill) return hipErrorInvalidValue;  // 16-bit prefill runs k_attn_prefill
  const dim3 grid(a.n_split, a.n_kv, nq), block(64 * ATTN_WAVES);
  switch (group) {
    case 1: HS_LAUNCH((k_attn<DT, HD, 1, ATTN_WAVES, PAGED>), grid, block, 0, st, a); break;
    case 2: HS_LAUNCH((k_attn<DT, HD, 2, ATTN_WAVES, PAGED>), grid, block, 0, st, a); break;
    case 4:
      if constexpr (DT == HS_F32) HS_LAUNCH((k_attn<DT, HD, 4, ATTN_WAVES, PAGED>), grid, block, 0, st, a);
      else HS_LAUNCH((k_attn_mma<DT, HD, 4, ATTN_WAVES, PAGED>), grid, block, 0, st, a);
      break;
    case 7:
      if constexpr (DT == HS_F32) HS_LAUNCH((k_attn<DT, HD, 7, ATTN_WAVES, PAGED>), grid, block, 0, st, a);
      else HS_LAUNCH((k_attn_mma<DT, HD, 7, ATTN_WAVES, PAGED>), grid, block, 0, st, a);
      break;
    case 8:
      if constexpr (DT == HS_F32) HS_LAUNCH((k_attn<DT, HD, 8, ATTN_WAVES, PAGED>), grid, block, 0, st, a);
      else HS_LAUNCH((k_attn_mma<DT, HD, 8, ATTN_WAVES, PAGED>), grid, block, 0, st, a);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int DT>
hipError_t attn_dt(int head_dim, int group, int nq, const AttnArgs &a, hipStream_t st) {
  // pooled caches hold 16-bit storage only
  if constexpr (DT != HS_F32) {
    if (a.kv.paged) {
      if (head_dim == 64) return attn_hd<DT, 64, true>(group, nq, a, st);
      if (head_dim == 128) return attn_hd<DT, 128, true>(group, nq, a, st);
      return hipErrorInvalidValue;
    }
  }
  if (head_dim == 64) return attn_hd<DT, 64, false>(group, nq, a, st);
  if (head_dim == 128) return attn_hd<DT, 128, false>(group, nq, a, st);
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

template <int DT, int HD>
hipError_t prefill_hd(int group, const AttnArgs &a, hipStream_t st) {
  constexpr int NW = 4;  // waves per query tile, taking its key tiles round robin
  const dim3 grid(a.prefill_pairs * a.n_kv), block(64 * NW);
  switch (group) {
    case 1: HS_LAUNCH((k_attn_prefill<DT, HD, 1, NW>), grid, block, 0, st, a); break;
    case 2: HS_LAUNCH((k_attn_prefill<DT, HD, 2, NW>), grid, block, 0, st, a); break;
    case 4: HS_LAUNCH((k_attn_prefill<DT, HD, 4, NW>), grid, block, 0, st, a); break;
    case 7: HS_LAUNCH((k_attn_prefill<DT, HD, 7, NW>), grid, block, 0, st, a); break;
    case 8: HS_LAUNCH((k_attn_prefill<DT, HD, 8, NW>), grid, block, 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

bool attn_prefill_on_mma(int dtype) { return dtype != HS_F32; }

int attn_prefill_rows_per_tile(int group) { return 16 / group; }

hipError_t launch_attention_prefill(int dtype, int head_dim, int group, int nrows, const AttnArgs &a,
                                    hipStream_t st) {
  if (nrows <= 0 || a.prefill_tiles <= 0) return hipSuccess;
  if (dtype == HS_F16) return head_dim == 64 ? prefill_hd<HS_F16, 64>(group, a, st)
                                             : prefill_hd<HS_F16, 128>(group, a, st);
  if (dtype == HS_BF16) return head_dim == 64 ? prefill_hd<HS_BF16, 64>(group, a, st)
                                              : prefill_hd<HS_BF16, 128>(group, a, st);
  return hipErrorInvalidValue;
}

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
