// selective_common.h -- helpers shared by the two layouts of the fused
// selective scan (selective_scan.hip, selective_scan_rows.hip): raw-bits
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

}  // namespace sw
