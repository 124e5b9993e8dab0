// Keep-set selection (Algorithm 1 steps (3)-(5); Sec. 3.3), one workgroup of
// 1024 threads per (stream, layer, head) slice.
//
// Thread t owns the RPT consecutive rows [t*RPT, (t+1)*RPT); its per-row flags
// live in 64-bit masks and its scores in registers. Each stage picks the top k
// of its candidates with an MSB-first radix select over order-preserving
// 32-bit keys (four 8-bit digits, an LDS histogram per digit), which yields
// the k-th largest key theta and how many of the k must come from keys equal
// to theta; those go to the lowest row indices through an exclusive scan of
// per-thread equal counts in row order. Ties are therefore broken exactly as
// "higher score first, then lower row index".
#pragma once

#include "ipv_device.hpp"

namespace ipv {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;

struct SelShared {
  uint32_t hist[256];
  int32_t wave_tot[kSelWaves];
  int32_t wave_off[kSelWaves];
  int32_t total;
  int32_t digit;
  int32_t above;
};

__device__ inline int32_t wave_inclusive_scan(int32_t v, int lane) {
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int32_t t = __shfl_up(v, d, kWave);
    if (lane >= d) v += t;
  }
  return v;
}

// Exclusive prefix sum over the workgroup in thread order; *total gets the sum.
__device__ inline int32_t block_exclusive_scan(int32_t v, SelShared& sh, int32_t* total) {
  const int tid = threadIdx.x, lane = tid % kWave, w = tid / kWave;
  const int32_t incl = wave_inclusive_scan(v, lane);
  if (lane == kWave - 1) sh.wave_tot[w] = incl;
  __syncthreads();
  if (w == 0) {
    const int32_t t = lane < kSelWaves ? sh.wave_tot[lane] : 0;
    const int32_t ti = wave_inclusive_scan(t, lane);
    if (lane < kSelWaves) sh.wave_off[lane] = ti - t;
    if (lane == kSelWaves - 1) sh.total = ti;
  }
  __syncthreads();
  const int32_t res = incl - v + sh.wave_off[w];
  *total = sh.total;
  __syncthreads();
  return res;
}

// Top-k of the candidate rows (bits of `cand`) by key; returns the mask of
// picked rows of this thread. k must not exceed the number of candidates.
template <int RPT>
__device__ uint64_t radix_top(const uint32_t (&key)[RPT], uint64_t cand, int32_t k, SelShared& sh) {
  if (k <= 0) return 0;
  const int tid = threadIdx.x;
  uint32_t prefix = 0, pmask = 0;
  int32_t remaining = k;
#pragma unroll 1
  for (int shift = 24; shift >= 0; shift -= 8) {
    if (tid < 256) sh.hist[tid] = 0;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < RPT; ++i)
      if (((cand >> i) & 1ull) && (key[i] & pmask) == prefix) atomicAdd(&sh.hist[(key[i] >> shift) & 255u], 1u);
    __syncthreads();
    if (tid < kWave) {
      // lane l holds digits 255-4l .. 252-4l, so lane order is descending digit order
      const int lane = tid;
      int32_t c[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) c[j] = (int32_t)sh.hist[255 - 4 * lane - j];
      const int32_t s = c[0] + c[1] + c[2] + c[3];
      const int32_t incl = wave_inclusive_scan(s, lane);
      const int32_t excl = incl - s;
      if (excl < remaining && remaining <= incl) {
        int32_t above = excl;
        int j = 0;
        while (above + c[j] < remaining) above += c[j++];
        sh.digit = 255 - 4 * lane - j;
        sh.above = above;
      }
    }
    __syncthreads();
    remaining -= sh.above;
    prefix |= (uint32_t)sh.digit << shift;
    pmask |= 255u << shift;
    __syncthreads();  // the next digit rewrites sh.digit / sh.above
  }
  // keys > prefix are in; `remaining` of the keys == prefix, lowest rows first
  int32_t eq = 0;
#pragma unroll
  for (int i = 0; i < RPT; ++i) eq += ((cand >> i) & 1ull) && key[i] == prefix;
  int32_t tot;
  int32_t taken = block_exclusive_scan(eq, sh, &tot);
  uint64_t pick = 0;
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    if (!((cand >> i) & 1ull)) continue;
    if (key[i] > prefix) {
      pick |= 1ull << i;
    } else if (key[i] == prefix) {
      if (taken < remaining) pick |= 1ull << i;
      ++taken;
    }
  }
  return pick;
}

template <int RPT>
__device__ inline void load_keys(const float* __restrict__ s, int64_t row0, int32_t n, uint64_t cand,
                                 uint32_t (&key)[RPT], uint32_t* err) {
  bool nan = false;
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const float v = row0 + i < n ? s[row0 + i] : 0.f;
    nan |= ((cand >> i) & 1ull) && (v != v);
    key[i] = order_key(v);
  }
  if (nan) raise_error(err, 16u);
}

template <int RPT>
__global__ __launch_bounds__(kSelThreads) void k_select(const float* __restrict__ tar, const float* __restrict__ van,
                                                        const int32_t* __restrict__ frame_idx, int64_t S, int32_t n,
                                                        int32_t budget, int32_t tar_total, int32_t r,
                                                        int32_t* __restrict__ keep_idx, uint32_t* err) {
  __shared__ SelShared sh;
  const int tid = threadIdx.x;
  const int64_t slice = blockIdx.x;
  const int64_t base = slice * S;
  const int64_t row0 = (int64_t)tid * RPT;
  int32_t* keep = keep_idx + slice * budget;

  const int64_t thr = (int64_t)frame_idx[base + n - 1] - r + 1;
  uint64_t valid = 0, recent = 0;
  int32_t prev = (row0 > 0 && row0 <= n) ? frame_idx[base + row0 - 1] : INT32_MIN;
  int32_t bad = 0;
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    if (row0 + i < n) {
      const int32_t f = frame_idx[base + row0 + i];
      valid |= 1ull << i;
      if ((int64_t)f >= thr) recent |= 1ull << i;
      bad |= f < prev;
      prev = f;
    }
  }
  int32_t n_recent, n_bad;
  block_exclusive_scan(__popcll(recent), sh, &n_recent);
  block_exclusive_scan(bad, sh, &n_bad);
  if (n_bad || n_recent > budget) {
    // metadata breaks the cache invariants: report, and keep rows 0..C-1 in place
    if (tid == 0) raise_error(err, n_bad ? 2u : 4u);
    for (int32_t j = tid; j < budget; j += kSelThreads) keep[j] = j;
    return;
  }
  const int32_t b_tar = max(0, tar_total - n_recent);
  const int32_t b_van = budget - n_recent - b_tar;

  uint32_t key[RPT];
  const uint64_t past = valid & ~recent;
  uint64_t pick_t = 0, pick_v = 0;
  if (b_tar > 0) {
    load_keys<RPT>(tar + base, row0, n, past, key, err);
    pick_t = radix_top<RPT>(key, past, b_tar, sh);
  }
  if (b_van > 0) {
    load_keys<RPT>(van + base, row0, n, past & ~pick_t, key, err);
    pick_v = radix_top<RPT>(key, past & ~pick_t, b_van, sh);
  }
  const uint64_t kept = recent | pick_t | pick_v;
  int32_t total;
  int32_t pos = block_exclusive_scan(__popcll(kept), sh, &total);
  if (total != budget && tid == 0) raise_error(err, 16u);  // only reachable with NaN keys
#pragma unroll
  for (int i = 0; i < RPT; ++i)
    if (((kept >> i) & 1ull) && pos < budget) keep[pos++] = (int32_t)(row0 + i);
}

}  // namespace ipv
