// hs_misc.hip — embedding gather, prefill input rows, greedy selection and
// length bookkeeping kernels of the decode engine (gfx950).
#include "hs_device.h"

namespace hs {
namespace {

using namespace dev;

// ---------------------------------------------------------------------------
// embeddings, selection, bookkeeping
// ---------------------------------------------------------------------------
// Copies one embedding row (model dtype) into the fp32 residual stream, one
// 16-byte chunk per thread and step, all loads issued before the stores.
template <int DT>
__device__ __forceinline__ void copy_row(const void *__restrict__ src, float *__restrict__ dst, int d) {
  constexpr int CE = Ty<DT>::CE;
  using S = typename Ty<DT>::S;
  constexpr int PER = 4;  // chunks per thread per pass
  for (int base = 0; base < d; base += 256 * CE * PER) {
    u32x4 v[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int k = base + (u * 256 + threadIdx.x) * CE;
      v[u] = k < d ? ld16((const S *)src + k) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int k = base + (u * 256 + threadIdx.x) * CE;
      if (k < d) {
        float f[CE];
        unpack<DT>(v[u], f);
#pragma unroll
        for (int e = 0; e < CE; e += 4) *(f32x4 *)(dst + k + e) = f32x4{f[e], f[e + 1], f[e + 2], f[e + 3]};
      }
    }
  }
}

template <int DT>
__global__ __launch_bounds__(256) void k_embed(const void *E, int V, int d, const int *tok, const int *act, float *x,
                                               int *status) {
  const int b = blockIdx.x;
  int t = tok[act ? act[b] : b];
  if (t < 0 || t >= V) {
    if (threadIdx.x == 0) atomicOr(status, 1);
    t = 0;
  }
  constexpr int B = DT == HS_F32 ? 4 : 2;
  copy_row<DT>((const char *)E + (int64_t)t * d * B, x + (int64_t)b * d, d);
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
  constexpr int B = DT == HS_F32 ? 4 : 2;
  copy_row<DT>((const char *)src + row * d * B, x + (int64_t)r * d, d);
}

// Greedy selection: largest logit, lowest index among equals (NaN never wins).
// Each thread scans indices i = tid + 1024 k in order, eight loads at a time.
__global__ __launch_bounds__(1024) void k_argmax(const float *__restrict__ logits, int V, int ld, int *out,
                                                 const int *act, int *len, int *rope, int advance) {
  const int b = blockIdx.x;
  const float *lg = logits + (int64_t)b * ld;
  float bv = -INFINITY;
  int bi = 0x7FFFFFFF;
  constexpr int PER = 8;
  for (int base = 0; base < V; base += 1024 * PER) {
    float v[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int i = base + u * 1024 + threadIdx.x;
      v[u] = i < V ? lg[i] : -INFINITY;
    }
#pragma unroll
    for (int u = 0; u < PER; ++u)
      if (v[u] > bv) {
        bv = v[u];
        bi = base + u * 1024 + threadIdx.x;
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
    const int r = act ? act[b] : b;
    out[r] = bi == 0x7FFFFFFF ? 0 : bi;
    if (advance) {
      len[r] += 1;
      rope[r] += 1;
    }
  }
}

__global__ void k_advance(int *len, int *rope, const int *act, int n) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < n) {
    const int r = act ? act[b] : b;
    len[r] += 1;
    rope[r] += 1;
  }
}

__global__ __launch_bounds__(256) void k_prefill_finish(int *len, int *rope, int *ready, int req, int s_ctx,
                                                        const int *pos_thw, int ld) {
  int mx = s_ctx - 1;
  if (pos_thw) {
    mx = 0x80000000;
    for (int i = threadIdx.x; i < 3 * s_ctx; i += 256) mx = max(mx, pos_thw[(i / s_ctx) * ld + i % s_ctx]);
    for (int off = 32; off >= 1; off >>= 1) mx = max(mx, __shfl_xor(mx, off));
    __shared__ int s_mx[4];
    if ((threadIdx.x & 63) == 0) s_mx[threadIdx.x >> 6] = mx;
    __syncthreads();
    mx = max(max(s_mx[0], s_mx[1]), max(s_mx[2], s_mx[3]));
  }
  if (threadIdx.x == 0) {
    len[req] = s_ctx;
    rope[req] = mx + 1;
    ready[req] = 1;
  }
}

// exclusive prefix sum over the 256 threads of the work group; *total gets the sum
__device__ int block_scan(int v, int *s_tmp, int *total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc = v;
  for (int off = 1; off < 64; off <<= 1) {
    const int o = __shfl_up(inc, off);
    if (lane >= off) inc += o;
  }
  if (lane == 63) s_tmp[wave] = inc;
  __syncthreads();
  int before = 0, all = 0;
  for (int w = 0; w < 4; ++w) {
    before += w < wave ? s_tmp[w] : 0;
    all += s_tmp[w];
  }
  __syncthreads();
  *total = all;
  return before + inc - v;
}

// Block allocation: each listed request takes the blocks between what it holds
// and what covers its target length, from the top of the free stack, in list
// order (a prefix sum hands out disjoint stack ranges, so no atomics).
__global__ __launch_bounds__(256) void k_kv_reserve(KvPool p, KvReserve r, int decode_n) {
  __shared__ int s_tmp[4];
  __shared__ int s_top, s_used;
  if (threadIdx.x == 0) s_top = *p.top;
  __syncthreads();
  const int n = decode_n > 0 ? decode_n : r.n;
  for (int c0 = 0; c0 < n; c0 += 256) {
    const int c = c0 + threadIdx.x;
    int req = -1, need = 0, held = 0;
    if (c < n) {
      req = decode_n > 0 ? p.act[c] : r.req[c];
      const int target = decode_n > 0 ? min(p.len[req] + 1, p.cap[req]) : r.target[c];
      held = p.nblk[req];
      need = max(0, (target + p.bt - 1) / p.bt - held);
    }
    int total;
    const int off = block_scan(need, s_tmp, &total);
    const int top = s_top;
    if (threadIdx.x == 0) s_used = 0;
    __syncthreads();
    // offsets grow along the list, so the requests served are a prefix of it
    if (need > 0) {
      if (off + need <= top) {
        for (int k = 0; k < need; ++k) {
          const int blk = p.stack[top - 1 - off - k];
          p.tab[p.toff[req] + held + k] = (int64_t)blk * p.block_elems;
        }
        p.nblk[req] = held + need;
        atomicMax(&s_used, off + need);
      } else {
        atomicOr(p.status, 4);  // pool exhausted: the request keeps unallocated entries
      }
    }
    __syncthreads();
    if (threadIdx.x == 0) s_top = top - s_used;
    __syncthreads();
  }
  if (threadIdx.x == 0) *p.top = s_top;
}

__global__ __launch_bounds__(256) void k_kv_release(KvPool p, int req) {
  const int held = p.nblk[req], top = *p.top;
  for (int k = threadIdx.x; k < held; k += 256) {
    const int64_t start = p.tab[p.toff[req] + k];
    p.stack[top + k] = (int)(start / p.block_elems);
    p.tab[p.toff[req] + k] = -1;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    *p.top = top + held;
    p.nblk[req] = 0;
    p.len[req] = 0;
    p.rope[req] = 0;
    p.ready[req] = 0;
  }
}

// Column c's rank is the number of columns ahead of it: longer, or as long
// with a lower index.  n^2 comparisons in one work group (n <= a few
// thousand, once per change of the batch).
__global__ __launch_bounds__(256) void k_build_order(const int *len, const int *act, int n, int *order) {
  for (int c = threadIdx.x; c < n; c += 256) {
    const int lc = len[act ? act[c] : c];
    int rank = 0;
    for (int o = 0; o < n; ++o) {
      const int lo = len[act ? act[o] : o];
      rank += lo > lc || (lo == lc && o < c);
    }
    order[rank] = c;
  }
}

// A plain streaming read (the HBM read rate the kernels are measured
// against): each work group reads 32 KB of consecutive bytes per round, each
// wave eight wave-wide 16-byte non-temporal loads of 1 KB, the rounds
// grid-strided; folded into one word per work group so that nothing is
// skipped.  (Loads strided by the whole grid, each a different DRAM page,
// read 4 GiB at 6.47 TB/s against 7.05 for this pattern.)
__global__ __launch_bounds__(256) void k_stream_read(const u32x4 *p, int64_t n16, uint32_t *sink) {
  constexpr int LPW = 8;                   // 1 KB loads per wave per round
  constexpr int64_t ROUND = 4 * LPW * 64;  // 16-byte words per work-group round
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t step = (int64_t)gridDim.x * ROUND;
  u32x4 acc = u32x4{0u, 0u, 0u, 0u};
  int64_t base = (int64_t)blockIdx.x * ROUND;
  for (; base + ROUND <= n16; base += step) {
    u32x4 v[LPW];
#pragma unroll
    for (int u = 0; u < LPW; ++u) v[u] = ld16_stream(p + base + (wave * LPW + u) * 64 + lane);
#pragma unroll
    for (int u = 0; u < LPW; ++u) acc ^= v[u];
  }
  if (base < n16)  // the last, partial round
    for (int u = 0; u < LPW; ++u) {
      const int64_t i = base + (wave * LPW + u) * 64 + lane;
      if (i < n16) acc ^= ld16_stream(p + i);
    }
  uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
  for (int off = 32; off >= 1; off >>= 1) x ^= __shfl_xor(x, off);
  __shared__ uint32_t s_x[4];
  if ((threadIdx.x & 63) == 0) s_x[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = s_x[0] ^ s_x[1] ^ s_x[2] ^ s_x[3];
}

__global__ void k_set_int(int *p, int v) {
  if (threadIdx.x == 0) *p = v;
}

// zeroes n16 16-byte words (grid-strided vector stores)
__global__ __launch_bounds__(256) void k_zero(u32x4 *p, int64_t n16) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += (int64_t)gridDim.x * 256)
    p[i] = u32x4{0u, 0u, 0u, 0u};
}

__global__ __launch_bounds__(256) void k_build_act(const int *ready, int n, int *act) {
  __shared__ int s_tmp[4];
  int base = 0;
  for (int c0 = 0; c0 < n; c0 += 256) {
    const int c = c0 + threadIdx.x;
    const int f = c < n && ready[c] ? 1 : 0;
    int total;
    const int off = block_scan(f, s_tmp, &total);
    if (f) act[base + off] = c;
    base += total;
  }
}

__global__ __launch_bounds__(128) void k_set_packed(PackedRows v, PackedRows *dst) {
  constexpr int N = (int)(sizeof(PackedRows) / 4);
  const int *src = (const int *)&v;
  for (int i = threadIdx.x; i < N; i += 128) ((int *)dst)[i] = src[i];
}

__global__ __launch_bounds__(256) void k_gather_last(const float *x, int d, PackedRows pk, float *out) {
  const float *src = x + (int64_t)(pk.cu[blockIdx.x + 1] - 1) * d;
  float *dst = out + (int64_t)blockIdx.x * d;
  for (int i = threadIdx.x; i < d; i += 256) dst[i] = src[i];
}

}  // namespace

hipError_t launch_embed(int dtype, const void *embed, int vocab, int d, const int *tokens, const int *act, int n,
                        float *x, int *status, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  switch (dtype) {
    case HS_F32: HS_LAUNCH(k_embed<HS_F32>, dim3(n), dim3(256), 0, st, embed, vocab, d, tokens, act, x, status); break;
    case HS_F16: HS_LAUNCH(k_embed<HS_F16>, dim3(n), dim3(256), 0, st, embed, vocab, d, tokens, act, x, status); break;
    case HS_BF16: HS_LAUNCH(k_embed<HS_BF16>, dim3(n), dim3(256), 0, st, embed, vocab, d, tokens, act, x, status); break;
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

hipError_t launch_argmax(const float *logits, int vocab, int ld, int n, int *tokens_out, const int *act, int *len,
                         int *rope_pos, int advance, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  HS_LAUNCH(k_argmax, dim3(n), dim3(1024), 0, st, logits, vocab, ld, tokens_out, act, len, rope_pos, advance);
  return hipGetLastError();
}

hipError_t launch_advance(int *len, int *rope_pos, const int *act, int n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  HS_LAUNCH(k_advance, dim3((n + 255) / 256), dim3(256), 0, st, len, rope_pos, act, n);
  return hipGetLastError();
}

hipError_t launch_kv_reserve(const KvPool &p, const KvReserve &r, int decode_n, hipStream_t st) {
  if (decode_n <= 0 && r.n <= 0) return hipSuccess;
  HS_LAUNCH(k_kv_reserve, dim3(1), dim3(256), 0, st, p, r, decode_n);
  return hipGetLastError();
}

hipError_t launch_kv_release(const KvPool &p, int req, hipStream_t st) {
  HS_LAUNCH(k_kv_release, dim3(1), dim3(256), 0, st, p, req);
  return hipGetLastError();
}

hipError_t launch_build_order(const int *len, const int *act, int n, int *order, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  HS_LAUNCH(k_build_order, dim3(1), dim3(256), 0, st, len, act, n, order);
  return hipGetLastError();
}

hipError_t launch_stream_read(const void *buf, uint64_t bytes, uint32_t *sink, int blocks, hipStream_t st) {
  HS_LAUNCH(k_stream_read, dim3(blocks), dim3(256), 0, st, (const u32x4 *)buf, (int64_t)(bytes / 16), sink);
  return hipGetLastError();
}

hipError_t launch_set_int(int *p, int v, hipStream_t st) {
  HS_LAUNCH(k_set_int, dim3(1), dim3(64), 0, st, p, v);
  return hipGetLastError();
}

hipError_t launch_zero(void *p, uint64_t bytes, hipStream_t st) {
  const int64_t n16 = (int64_t)(bytes / 16);
  if (n16 <= 0) return hipSuccess;
  const int grid = (int)std::min<int64_t>((n16 + 255) / 256, 1024);
  HS_LAUNCH(k_zero, dim3(grid), dim3(256), 0, st, (u32x4 *)p, n16);
  return hipGetLastError();
}

hipError_t launch_build_act(const int *ready, int n, int *act, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  HS_LAUNCH(k_build_act, dim3(1), dim3(256), 0, st, ready, n, act);
  return hipGetLastError();
}

hipError_t launch_prefill_finish(int *len, int *rope_pos, int *ready, int req, int s_ctx, const int *pos_thw, int ld,
                                 hipStream_t st) {
  HS_LAUNCH(k_prefill_finish, dim3(1), dim3(256), 0, st, len, rope_pos, ready, req, s_ctx, pos_thw, ld);
  return hipGetLastError();
}

hipError_t launch_set_packed(PackedRows *dst, const PackedRows &v, hipStream_t st) {
  HS_LAUNCH(k_set_packed, dim3(1), dim3(128), 0, st, v, dst);
  return hipGetLastError();
}

hipError_t launch_gather_last(const float *x, int d, const PackedRows &pk, float *out, hipStream_t st) {
  if (pk.n <= 0) return hipSuccess;
  HS_LAUNCH(k_gather_last, dim3(pk.n), dim3(256), 0, st, x, d, pk, out);
  return hipGetLastError();
}

}  // namespace hs
