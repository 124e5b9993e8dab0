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
// dot / sumsq: the dot product of two 16-byte chunks / the sum of squares of
// one, accumulated in fp32 (bf16 pairs by the packed bf16 dot instruction:
// each bf16 product is exact in fp32).
template <typename T>
struct Lane;

typedef __bf16 Bf16x2 __attribute__((ext_vector_type(2)));

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
  __device__ static inline float dot(const Raw16& a, const Raw16& b) {
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(Bf16x2, a.w[i]), __builtin_bit_cast(Bf16x2, b.w[i]),
                                            acc, false);
    return acc;
  }
  __device__ static inline float sumsq(const Raw16& r) { return dot(r, r); }
};

template <>
struct Lane<float> {
  static constexpr int EPL = 4;
  __device__ static inline void decode(const Raw16& r, float* f) {
#pragma unroll
    for (int i = 0; i < 4; ++i) f[i] = __uint_as_float(r.w[i]);
  }
  __device__ static inline float dot(const Raw16& a, const Raw16& b) {
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) acc += __uint_as_float(a.w[i]) * __uint_as_float(b.w[i]);
    return acc;
  }
  __device__ static inline float sumsq(const Raw16& r) { return dot(r, r); }
};

// Hardware square root and reciprocal square root (about 1 ulp): the scores
// need 1e-3 relative accuracy, not the correctly rounded sequences.
__device__ inline float fast_sqrt(float x) { return __builtin_amdgcn_sqrtf(x); }
__device__ inline float fast_rsqrt(float x) { return __builtin_amdgcn_rsqf(x); }

__device__ inline Raw16 load16(const void* p) { return *reinterpret_cast<const Raw16*>(p); }

// Buffer loads: a resource covers [base, base + bytes); a load past the end
// returns zeros instead of faulting, so bounds need no branch (branches around
// loads make the compiler wait for each load before the next is issued).
constexpr int kBufferDword3 = 0x00020000;  // raw 32-bit data (gfx9 family)

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kBufferDword3);
}

// Cache-policy operand of a buffer load that streams data read once
// (gfx950 encoding of the nontemporal bit).
constexpr int kNontemporal = 2;

// Nontemporal (streaming) store: compacted rows are not read again in the
// pass, and storing them this way keeps them from lingering as dirty lines
// that a later kernel's reads would have to write back first.
typedef uint32_t U32x4 __attribute__((ext_vector_type(4)));
__device__ inline void store16(void* p, const Raw16& v) {
  const U32x4 x = {v.w[0], v.w[1], v.w[2], v.w[3]};
  __builtin_nontemporal_store(x, reinterpret_cast<U32x4*>(p));
}

// ---- cross-lane moves
// DPP moves run in the vector ALU; __shfl_* goes through the LDS crossbar
// (ds_bpermute) with far longer latency. DPP controls (GFX9 encoding):
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppRowShr = 0x110;     // + k: row_shr:k (within rows of 16 lanes)
constexpr int kDppRowMirror = 0x140;  // lane l <- 15 - l within a row
constexpr int kDppHalfMirror = 0x141; // lane l <- 7 - l within each 8 lanes
constexpr int kDppQuadMirror = 0x1B;  // quad_perm [3,2,1,0]: lane l <- 3 - l within each 4 lanes

template <int CTRL, bool BOUND_ZERO = false>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xf, 0xf, BOUND_ZERO);
}

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __uint_as_float(dpp_u32<CTRL>(__float_as_uint(v)));
}

// Sum over aligned groups of G lanes (G a power of two <= 64); every lane of
// a group gets the group's sum, the same in all of them. The first steps
// pair lanes whose values are equal within smaller groups, so a mirror is an
// exchange with the other half: xor 1, xor 2, (0..3 <-> 4..7), (0..7 <-> 8..15),
// then xor 16 and xor 32 through the crossbar. A group is inactive as a whole
// or active as a whole.
template <int G>
__device__ __forceinline__ float group_sum(float v) {
  if (G >= 2) v += dpp_f32<kDppXor1>(v);
  if (G >= 4) v += dpp_f32<kDppXor2>(v);
  if (G >= 8) v += dpp_f32<kDppHalfMirror>(v);
  if (G >= 16) v += dpp_f32<kDppRowMirror>(v);
  if (G >= 32) v += __shfl_xor(v, 16, kWave);
  if (G >= 64) v += __shfl_xor(v, 32, kWave);
  return v;
}

// Reduce-scatter of four rows' partial sums over an aligned group of G lanes
// (G a power of two, 4 <= G <= 64): v[u][m] is this lane's part of value m of
// row u. On return the lane holds out[m] = the group's total of value m for
// row scatter_row<G>(lane), the same in all G / 4 lanes that hold that row.
// Two exchange steps halve the rows a lane keeps (it adds the partner's part
// of the rows it keeps and hands over the others): partners are the lane
// mirrored across the group's halves, then across its quarters; the quarter
// of lanes that ends up with one row then sums over its own lanes. Groups
// wider than 16 lanes first fold onto 16 through the crossbar.
template <int G>
__device__ __forceinline__ int scatter_row(int lane) {
  constexpr int H = G > 16 ? 16 : G;
  return ((lane & (H / 2)) ? 2 : 0) + ((lane & (H / 4)) ? 1 : 0);
}

template <int G, int M>
__device__ __forceinline__ void reduce_scatter4(float (&v)[4][M], float (&out)[M], int lane) {
  static_assert(G >= 4 && G <= 64 && (G & (G - 1)) == 0, "group of 4..64 lanes");
  if (G >= 32) {
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int m = 0; m < M; ++m) {
        v[u][m] += __shfl_xor(v[u][m], 16, kWave);
        if (G == 64) v[u][m] += __shfl_xor(v[u][m], 32, kWave);
      }
  }
  constexpr int H = G > 16 ? 16 : G;
  // mirror across halves, then across quarters, of an H-lane group
  constexpr int MA = H == 16 ? kDppRowMirror : (H == 8 ? kDppHalfMirror : kDppXor2);
  constexpr int MB = H == 16 ? kDppHalfMirror : (H == 8 ? kDppQuadMirror : kDppXor1);
  const bool hi_a = (lane & (H / 2)) != 0, hi_b = (lane & (H / 4)) != 0;
  float w[2][M];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int m = 0; m < M; ++m) {
      const float keep = hi_a ? v[2 + j][m] : v[j][m];
      const float give = hi_a ? v[j][m] : v[2 + j][m];
      w[j][m] = keep + dpp_f32<MA>(give);
    }
#pragma unroll
  for (int m = 0; m < M; ++m) {
    const float keep = hi_b ? w[1][m] : w[0][m];
    const float give = hi_b ? w[0][m] : w[1][m];
    out[m] = keep + dpp_f32<MB>(give);
    if (H == 16) {
      out[m] += dpp_f32<kDppXor1>(out[m]);
      out[m] += dpp_f32<kDppXor2>(out[m]);
    } else if (H == 8) {
      out[m] += dpp_f32<kDppXor1>(out[m]);
    }
  }
}

// Inclusive prefix sum over the 64 lanes of a fully active wave: a
// Hillis-Steele scan within each row of 16 lanes, then the totals of the
// rows below are added.
__device__ __forceinline__ int32_t wave_inclusive_scan(int32_t v) {
  v += (int32_t)dpp_u32<kDppRowShr + 1, true>((uint32_t)v);
  v += (int32_t)dpp_u32<kDppRowShr + 2, true>((uint32_t)v);
  v += (int32_t)dpp_u32<kDppRowShr + 4, true>((uint32_t)v);
  v += (int32_t)dpp_u32<kDppRowShr + 8, true>((uint32_t)v);
  const int32_t r0 = __builtin_amdgcn_readlane(v, 15);
  const int32_t r1 = __builtin_amdgcn_readlane(v, 31);
  const int32_t r2 = __builtin_amdgcn_readlane(v, 47);
  const int lane = (int)(threadIdx.x % kWave);
  return v + (lane >= 16 ? r0 : 0) + (lane >= 32 ? r1 : 0) + (lane >= 48 ? r2 : 0);
}

// Minimum and maximum over the 64 lanes of a fully active wave (uniform result).
__device__ __forceinline__ void wave_min_max(uint32_t& mn, uint32_t& mx) {
  mn = min(mn, dpp_u32<kDppXor1>(mn));
  mx = max(mx, dpp_u32<kDppXor1>(mx));
  mn = min(mn, dpp_u32<kDppXor2>(mn));
  mx = max(mx, dpp_u32<kDppXor2>(mx));
  mn = min(mn, dpp_u32<kDppHalfMirror>(mn));
  mx = max(mx, dpp_u32<kDppHalfMirror>(mx));
  mn = min(mn, dpp_u32<kDppRowMirror>(mn));
  mx = max(mx, dpp_u32<kDppRowMirror>(mx));
  uint32_t a = (uint32_t)__builtin_amdgcn_readlane((int)mn, 0), b = (uint32_t)__builtin_amdgcn_readlane((int)mx, 0);
#pragma unroll
  for (int r = 16; r < kWave; r += 16) {
    a = min(a, (uint32_t)__builtin_amdgcn_readlane((int)mn, r));
    b = max(b, (uint32_t)__builtin_amdgcn_readlane((int)mx, r));
  }
  mn = a;
  mx = b;
}

// Exclusive prefix sum over the workgroup in thread order (one barrier);
// *total gets the sum. `tot` is used by this scan only.
template <int NT>
__device__ __forceinline__ int32_t block_exclusive_scan(int32_t v, int32_t* tot, int32_t* total) {
  constexpr int NW = NT / kWave;
  const int tid = threadIdx.x, lane = tid % kWave, w = tid / kWave;
  const int32_t incl = wave_inclusive_scan(v);
  if (lane == kWave - 1) tot[w] = incl;
  __syncthreads();
  int32_t off = 0, sum = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const int32_t t = tot[i];
    off += i < w ? t : 0;
    sum += t;
  }
  *total = sum;
  return incl - v + off;
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

// Division by a divisor d fixed for a launch, as a multiply-high and two
// shifts with a magic number computed on the host (Granlund and Montgomery,
// "Division by invariant integers using multiplication", 1994): exact for
// every 32-bit x. With l = ceil(log2 d), m = floor(2^32 (2^l - d) / d) + 1:
//   t = mulhi(x, m),  x / d = (t + ((x - t) >> 1)) >> (l - 1);
// d = 1 uses m = 0 and no shifts.
struct FastDiv {
  uint32_t d, m, s1, s2;
};

inline FastDiv make_fastdiv(uint32_t d) {
  FastDiv f{d, 0u, 0u, 0u};
  if (d > 1) {
    uint32_t l = 0;
    while ((1ull << l) < d) ++l;
    f.m = (uint32_t)(((1ull << 32) * ((1ull << l) - d)) / d + 1);
    f.s1 = 1;
    f.s2 = l - 1;
  }
  return f;
}

__device__ __forceinline__ uint32_t fast_div(uint32_t x, const FastDiv& f) {
  const uint32_t t = __umulhi(x, f.m);
  return (t + ((x - t) >> f.s1)) >> f.s2;
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
