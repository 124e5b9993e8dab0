// Device helpers shared by the compression-pass kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ipv {

constexpr int kWave = 64;

// Workspace header: the device error word lives in the first 256 bytes.
constexpr size_t kWsHeader = 256;

struct alignas(16) Raw16 {
  uint32_t w[4];
};

// 16 bytes of a row, decoded to fp32. EPL = elements per 16-byte lane chunk.
template <typename T>
struct Lane;

template <>
struct Lane<uint16_t> {  // bf16 bit patterns
  static constexpr int EPL = 8;
  __device__ static inline void decode(const Raw16& r, float* f) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = __uint_as_float(r.w[i] << 16);
      f[2 * i + 1] = __uint_as_float(r.w[i] & 0xffff0000u);
    }
  }
};

template <>
struct Lane<float> {
  static constexpr int EPL = 4;
  __device__ static inline void decode(const Raw16& r, float* f) {
#pragma unroll
    for (int i = 0; i < 4; ++i) f[i] = __uint_as_float(r.w[i]);
  }
};

__device__ inline Raw16 load16(const void* p) { return *reinterpret_cast<const Raw16*>(p); }

__device__ inline void store16(void* p, const Raw16& v) { *reinterpret_cast<Raw16*>(p) = v; }

// Sum over aligned groups of G lanes (G a power of two <= 64).
template <int G>
__device__ inline float group_sum(float v) {
#pragma unroll
  for (int m = G / 2; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}

__device__ inline void raise_error(uint32_t* err, uint32_t bits) {
  if (err) atomicOr(err, bits);
}

// fp32 -> uint32 whose unsigned order is the float order; -0.0 maps like +0.0.
__device__ inline uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Workgroups are dispatched round-robin over the 8 XCDs (id % 8). Renumber
// them so that consecutive logical ids share an XCD and its L2: logical =
// (id % 8) * per_xcd + id / 8. The grid must be padded to a multiple of 8;
// logical ids >= the real count return early.
__device__ inline uint32_t xcd_logical_id(uint32_t id, uint32_t grid) {
  const uint32_t per_xcd = grid / 8u;
  return (id % 8u) * per_xcd + id / 8u;
}

}  // namespace ipv
