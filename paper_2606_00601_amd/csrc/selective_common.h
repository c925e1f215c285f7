// selective_common.h -- helpers of the fused selective scan kernels: raw-bits
// registers for fp32 / bf16 inputs and their exact widening to fp32.
#pragma once

#include "sw_internal.h"

namespace sw {

__device__ __forceinline__ int64_t imin(int64_t a, int64_t b) { return a < b ? a : b; }

template <typename IN>
struct Elt;
template <>
struct Elt<float> {
  static __device__ __forceinline__ uint32_t raw(const float* __restrict__ p, int64_t i) {
    return __float_as_uint(p[i]);
  }
};
template <>
struct Elt<uint16_t> {
  static __device__ __forceinline__ uint32_t raw(const uint16_t* __restrict__ p, int64_t i) {
    return p[i];
  }
};

// Cache policy of a buffer access (the `aux` operand of the raw buffer
// builtins): SW_NT marks it non-temporal -- for data a kernel reads or writes
// once, so that it does not displace lines other workgroups read again (B and
// C of a batch).  Only where one instruction covers whole 128-byte lines: a
// line read in parts by successive instructions measured slower with it.
constexpr int SW_NT = 2;

// Raw registers for COUNT consecutive elements of type IN.
template <typename IN, int COUNT>
struct RawVec {
  static constexpr int W = (COUNT * (int)sizeof(IN) + 3) / 4;
  uint32_t w[W];
  // from a 16-byte (W % 4 == 0) or 8-byte aligned address
  __device__ __forceinline__ void load_vec(const IN* __restrict__ p) {
    if constexpr (W % 4 == 0) {
#pragma unroll
      for (int q = 0; q < W / 4; ++q) {
        const uint4 v = reinterpret_cast<const uint4*>(p)[q];
        w[4 * q] = v.x;
        w[4 * q + 1] = v.y;
        w[4 * q + 2] = v.z;
        w[4 * q + 3] = v.w;
      }
    } else {
      static_assert(W % 2 == 0, "8-byte granularity");
#pragma unroll
      for (int q = 0; q < W / 2; ++q) {
        const uint2 v = reinterpret_cast<const uint2*>(p)[q];
        w[2 * q] = v.x;
        w[2 * q + 1] = v.y;
      }
    }
  }
  // from a raw buffer resource at byte offset `off` (16- or 8-byte aligned),
  // with cache policy POL; bytes outside the resource's range read as zero
  template <int POL = 0>
  __device__ __forceinline__ void load_buf(__amdgpu_buffer_rsrc_t rs, int32_t off) {
    if constexpr (W % 4 == 0) {
#pragma unroll
      for (int q = 0; q < W / 4; ++q) {
        const uint4 v =
            __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, off + 16 * q, 0, POL));
        w[4 * q] = v.x;
        w[4 * q + 1] = v.y;
        w[4 * q + 2] = v.z;
        w[4 * q + 3] = v.w;
      }
    } else if constexpr (W == 1) {
      w[0] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, POL));
    } else {
      static_assert(W % 2 == 0, "8-byte granularity");
#pragma unroll
      for (int q = 0; q < W / 2; ++q) {
        const uint2 v =
            __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(rs, off + 8 * q, 0, POL));
        w[2 * q] = v.x;
        w[2 * q + 1] = v.y;
      }
    }
  }
  // element i as fp32 (bf16 widened exactly)
  __device__ __forceinline__ float get(int i) const {
    if constexpr (sizeof(IN) == 4) {
      return __uint_as_float(w[i]);
    } else {
      return (i & 1) ? bf16_hi(w[i >> 1]) : bf16_lo(w[i >> 1]);
    }
  }
  // element i from raw bits (element-wise path)
  __device__ __forceinline__ void set(int i, uint32_t bits) {
    if constexpr (sizeof(IN) == 4) {
      w[i] = bits;
    } else if (i & 1) {
      w[i >> 1] = (w[i >> 1] & 0xffffu) | (bits << 16);
    } else {
      w[i >> 1] = (w[i >> 1] & 0xffff0000u) | (bits & 0xffffu);
    }
  }
};

// 16- and 8-byte payloads of raw buffer stores
typedef unsigned int sw_u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int sw_u32x2 __attribute__((ext_vector_type(2)));

// Raw buffer resource over `bytes` bytes from `base` (stride 0, the gfx9
// default data format): loads at byte offsets past the range return zero
// instead of faulting, and stores there are dropped.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}

}  // namespace sw
