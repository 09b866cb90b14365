// hs_device.h — device-side helpers shared by the gfx950 kernels of libhs:
// storage dtypes and their round-to-nearest-even conversions, 16-byte chunk
// (un)packing, the MFMA tile update and DPP/shuffle reductions.
#pragma once

#include "hs_internal.h"

#include <cmath>
#include <type_traits>

#define HS_LAUNCH(kernel, grid, block, shmem, stream, ...) \
  hipLaunchKernelGGL(kernel, grid, block, shmem, stream, __VA_ARGS__)

namespace hs {
namespace dev {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

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

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

// The 16x16x16 MFMA: lane l supplies row (A) / column (B) l % 16 and the
// 4 k values 4 (l / 16) .. + 3 of its 8-byte operand.
template <int DT>
__device__ __forceinline__ f32x4 mma16(u32x2 a, u32x2 b, f32x4 c) {
  if constexpr (DT == HS_F16) {
    return __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(f16x4, a), __builtin_bit_cast(f16x4, b), c, 0, 0,
                                                 0);
  } else {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(bf16x4, a), __builtin_bit_cast(bf16x4, b), c,
                                                     0, 0, 0);
  }
}

__device__ __forceinline__ u32x4 ld16(const void *p) { return *(const u32x4 *)p; }
__device__ __forceinline__ u32x4 ld16_stream(const void *p) {
  return __builtin_nontemporal_load((const u32x4 *)p);
}

// Packed activation layout (16-bit storage): column c, element k of a matrix
// of K-long columns sits where the MFMA B operand wants it -- per 16-column
// tile and 128-element k-block, four 1 KB sub-blocks of 32 elements, lane
// 16 * (k / 8 mod 4) + c mod 16 holding 8 consecutive elements -- so a wave
// reads one sub-block of a column tile as 1 KB of consecutive bytes.
__host__ __device__ inline int64_t packed_x_index(int c, int k, int nkb) {
  return ((((int64_t)(c >> 4) * nkb + (k >> 7)) * 4 + ((k >> 5) & 3)) * 64 + (((k >> 3) & 3) << 4) + (c & 15)) * 8 +
         (k & 7);
}

// ---------------------------------------------------------------------------
// raw buffer reads
// ---------------------------------------------------------------------------
// A buffer resource covers the byte range [base, base + bytes); a read at an
// offset past it returns zeros without touching memory.  Loads that may fall
// outside their data therefore need no branch, which keeps the compiler's
// count of outstanding loads exact (a branch around a load makes it wait for
// all of them).  Ranges stay below BUF_OOB, the offset used for "no data".
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr uint32_t BUF_OOB = 0x80000000u;
constexpr int BUF_WORD3 = 0x00020000;  // raw access, 32-bit data format
__device__ __forceinline__ rsrc_t make_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, BUF_WORD3);
}
__device__ __forceinline__ u32x4 bld16(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
// non-temporal: data read once per step (the weight stream)
__device__ __forceinline__ u32x4 bld16_stream(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 2));
}
__device__ __forceinline__ uint32_t bld4(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
__device__ __forceinline__ u32x2 bld8(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
}

// request (index into pk) of packed prefill row `row`
__device__ __forceinline__ int packed_request(const PackedRows *pk, int row) {
  int i = 0;
  for (int k = 1; k < pk->n; ++k) i += row >= pk->cu[k];
  return i;
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


}  // namespace dev
}  // namespace hs
