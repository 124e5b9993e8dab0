// In-place, order-preserving compaction (Sec. 3.1; Algorithm 1 step (5)):
// row j <- row keep[j] for j < C, for K, V, frame_idx and patch_idx.
//
// Safety of doing it in place: keep is ascending, so keep[j] >= j. Output
// rows are processed in chunks [j0, j0 + CH) by ONE workgroup walking its
// chunks in order. A chunk reads rows keep[j] >= j0 and writes rows < j0 + CH;
// every later chunk reads only rows >= j0 + CH. So once all of a chunk's
// loads have landed (wait on the memory counter, then a workgroup barrier) its
// stores cannot clobber anything still to be read, and the next chunk's
// loads may be issued while those stores drain. Independent walks run per
// (slice, tensor, column block): columns never alias across walks.
#pragma once

#include "ipv_device.hpp"

namespace ipv {

template <int RB>  // bytes per row
struct CompactCfg {
  static constexpr int CB = RB < 128 ? RB : 128;  // bytes per column block
  static constexpr int NCB = RB / CB;             // column blocks per row
  static constexpr int LPP = CB / 16;             // lanes per row piece
  static constexpr int RPS = 256 / LPP;           // rows per step
  static constexpr int U = 8;                     // steps per chunk
  static constexpr int CH = RPS * U;              // rows per chunk
};

// grid: slices * 2 * NCB workgroups; work w -> (slice, tensor K/V, column block)
template <int RB>
__global__ __launch_bounds__(256) void k_compact(char* __restrict__ K, char* __restrict__ V,
                                                 int32_t* __restrict__ frame_idx, int32_t* __restrict__ patch_idx,
                                                 int64_t S, int32_t n, int32_t budget,
                                                 const int32_t* __restrict__ keep_idx, uint32_t* err) {
  using C = CompactCfg<RB>;
  constexpr int LPP = C::LPP, RPS = C::RPS, U = C::U;
  const int64_t w = blockIdx.x;
  const int64_t slice = w / (2 * C::NCB);
  const int t = (int)((w / C::NCB) % 2);
  const int cb = (int)(w % C::NCB);
  char* base = (t == 0 ? K : V) + slice * S * RB + cb * C::CB;
  const bool meta = (t == 0 && cb == 0);
  int32_t* fr = frame_idx + slice * S;
  int32_t* pa = patch_idx + slice * S;
  const int32_t* keep = keep_idx + slice * budget;
  const int tid = threadIdx.x, sub = tid / LPP, lane = tid % LPP;

#pragma unroll 1
  for (int64_t j0 = 0; j0 < budget; j0 += C::CH) {
    Raw16 buf[U];
    int32_t src[U], mf[U], mp[U];
    bool bad = false;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t j = j0 + u * RPS + sub;
      src[u] = -1;
      if (j < budget) {
        const int32_t s = keep[j];
        if (s < j || s >= n) {
          bad = true;
        } else if (s != j) {
          src[u] = s;
          buf[u] = load16(base + (int64_t)s * RB + lane * 16);
          if (meta && lane == 0) {
            mf[u] = fr[s];
            mp[u] = pa[s];
          }
        }
      }
    }
    if (bad && lane == 0) raise_error(err, 8u);
    // Use every loaded register in an opaque statement: the compiler must wait
    // for each load's data here, before the barrier, and cannot sink a load
    // past it. After the barrier every wave's loads of this chunk have landed.
#pragma unroll
    for (int u = 0; u < U; ++u) asm volatile("" ::"v"(buf[u].w[0]), "v"(mf[u]), "v"(mp[u]));
    __syncthreads();
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t j = j0 + u * RPS + sub;
      if (src[u] >= 0) {
        store16(base + j * RB + lane * 16, buf[u]);
        if (meta && lane == 0) {
          fr[j] = mf[u];
          pa[j] = mp[u];
        }
      }
    }
  }
}

}  // namespace ipv
