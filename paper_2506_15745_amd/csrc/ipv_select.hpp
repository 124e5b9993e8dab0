// Keep-set selection (Algorithm 1 steps (3)-(5); Sec. 3.3), one workgroup of
// NT threads per (stream, layer, head) slice.
//
// Thread t owns the RPT consecutive rows [t*RPT, (t+1)*RPT). All of its frame
// ids and both score columns are loaded at once (16-byte loads), turned into
// order-preserving 32-bit keys (-0.0 equal to +0.0) and kept in registers.
//
// Each stage picks the top k of its candidates with an MSB-first radix
// select over the keys: 8-bit digits starting below the bits that all the
// candidates share, an LDS histogram per digit (two buffers, alternating, so
// a digit costs two barriers), stopping as soon as the threshold bin holds
// exactly the keys still needed. Keys above the threshold prefix are in;
// among keys equal to it, an exclusive scan of per-thread counts in row order
// lets the lowest row indices in first. That is exactly "higher score first,
// then lower row index".
#pragma once

#include "ipv_device.hpp"

namespace ipv {

template <int NT>
struct SelShared {
  static constexpr int NW = NT / kWave;
  uint32_t hist[2][256];
  int32_t wave_tot[NW];
  int32_t wave_off[NW];
  uint32_t wave_min[NW], wave_max[NW];
  int32_t total;
  int32_t digit;
  int32_t above;
  int32_t done;
  int32_t first_recent;
  int32_t bad;
};

// Exclusive prefix sum over the workgroup in thread order; *total gets the sum.
template <int NT>
__device__ __forceinline__ int32_t block_exclusive_scan(int32_t v, SelShared<NT>& sh, int32_t* total) {
  constexpr int NW = NT / kWave;
  const int tid = threadIdx.x, lane = tid % kWave, w = tid / kWave;
  const int32_t incl = wave_inclusive_scan(v);
  if (lane == kWave - 1) sh.wave_tot[w] = incl;
  __syncthreads();
  if (w == 0) {
    const int32_t t = lane < NW ? sh.wave_tot[lane] : 0;
    const int32_t ti = wave_inclusive_scan(t);
    if (lane < NW) sh.wave_off[lane] = ti - t;
    if (lane == NW - 1) sh.total = ti;
  }
  __syncthreads();
  const int32_t res = incl - v + sh.wave_off[w];
  *total = sh.total;
  __syncthreads();
  return res;
}

// Top-k of the candidate rows (bits of `cand`) by key; returns this thread's
// picks. 0 < k <= number of candidates.
template <int NT, int RPT>
__device__ __forceinline__ uint64_t radix_top(const uint32_t (&key)[RPT], uint64_t cand, int32_t k, SelShared<NT>& sh) {
  constexpr int NW = NT / kWave;
  const int tid = threadIdx.x, lane = tid % kWave, w = tid / kWave;
  // bits shared by every candidate key
  uint32_t mn = 0xffffffffu, mx = 0u;
#pragma unroll
  for (int i = 0; i < RPT; ++i)
    if ((cand >> i) & 1ull) {
      mn = min(mn, key[i]);
      mx = max(mx, key[i]);
    }
  wave_min_max(mn, mx);
  if (lane == 0) {
    sh.wave_min[w] = mn;
    sh.wave_max[w] = mx;
  }
  if (tid < 256) sh.hist[0][tid] = 0u;
  __syncthreads();
  mn = sh.wave_min[0];
  mx = sh.wave_max[0];
#pragma unroll
  for (int i = 1; i < NW; ++i) {
    mn = min(mn, sh.wave_min[i]);
    mx = max(mx, sh.wave_max[i]);
  }
  const int common = (mn == mx) ? 32 : __clz((int)(mn ^ mx));
  uint32_t pmask = common == 0 ? 0u : (common == 32 ? 0xffffffffu : 0xffffffffu << (32 - common));
  uint32_t prefix = mn & pmask;
  int32_t remaining = k;
  int cur = 0;
#pragma unroll 1
  for (int top = 32 - common; top > 0; top -= 8) {
    const int shift = max(0, top - 8);
    const uint32_t dmask = (1u << (top - shift)) - 1u;
#pragma unroll
    for (int i = 0; i < RPT; ++i)
      if (((cand >> i) & 1ull) && (key[i] & pmask) == prefix) atomicAdd(&sh.hist[cur][(key[i] >> shift) & dmask], 1u);
    if (tid < 256) sh.hist[cur ^ 1][tid] = 0u;  // the next digit's buffer
    __syncthreads();
    if (w == 0) {
      // lane l holds digits 255-4l .. 252-4l: lane order is descending digit order
      int32_t c[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) c[j] = (int32_t)sh.hist[cur][255 - 4 * lane - j];
      const int32_t s = c[0] + c[1] + c[2] + c[3];
      const int32_t incl = wave_inclusive_scan(s);
      const int32_t excl = incl - s;
      if (excl < remaining && remaining <= incl) {
        int32_t above = excl;
        int j = 0;
        while (above + c[j] < remaining) above += c[j++];
        sh.digit = 255 - 4 * lane - j;
        sh.above = above;
        sh.done = (above + c[j] == remaining);  // the threshold bin is taken whole
      }
    }
    __syncthreads();
    remaining -= sh.above;
    prefix |= (uint32_t)sh.digit << shift;
    pmask |= dmask << shift;
    cur ^= 1;
    if (sh.done) break;
  }
  // masked keys above the prefix are in; `remaining` of those equal to it go
  // to the lowest rows (all of them when the loop stopped early)
  int32_t eq = 0;
#pragma unroll
  for (int i = 0; i < RPT; ++i) eq += ((cand >> i) & 1ull) && (key[i] & pmask) == prefix;
  int32_t tot;
  int32_t taken = block_exclusive_scan<NT>(eq, sh, &tot);
  uint64_t pick = 0;
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    if (!((cand >> i) & 1ull)) continue;
    const uint32_t mk = key[i] & pmask;
    if (mk > prefix) {
      pick |= 1ull << i;
    } else if (mk == prefix) {
      if (taken < remaining) pick |= 1ull << i;
      ++taken;
    }
  }
  return pick;
}

// Rows [row0, row0 + RPT) of one slice's column (S rows of 4 bytes); rows at
// or past S read as 0. VEC: rows are 16-byte aligned (S % 4 == 0), so a run
// lies wholly inside or wholly past the column and loads 16 bytes at a time.
template <int RPT, bool VEC>
__device__ __forceinline__ void load_row_run(const void* __restrict__ col, int64_t S, int64_t row0,
                                             uint32_t (&out)[RPT]) {
  const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(col, (uint32_t)(S * 4));
  if (VEC) {
#pragma unroll
    for (int i = 0; i < RPT; i += 4) {
      const auto v = __builtin_amdgcn_raw_buffer_load_b128(rs, (uint32_t)((row0 + i) * 4), 0, 0);
      out[i] = v[0];
      out[i + 1] = v[1];
      out[i + 2] = v[2];
      out[i + 3] = v[3];
    }
  } else {
#pragma unroll
    for (int i = 0; i < RPT; ++i) out[i] = __builtin_amdgcn_raw_buffer_load_b32(rs, (uint32_t)((row0 + i) * 4), 0, 0);
  }
}

// One slice with NT threads. VEC: every slice's row 0 is 16-byte aligned
// (capacity % 4 == 0) so row runs load 16 bytes at a time.
template <int NT, int RPT, bool VEC>
__device__ __forceinline__ void select_slice(const float* __restrict__ tar, const float* __restrict__ van,
                             const int32_t* __restrict__ frame_idx, int64_t S, int32_t n, int32_t budget,
                             int32_t tar_total, int32_t r, int32_t* __restrict__ keep_idx,
                             uint32_t* err, int64_t slice, SelShared<NT>& sh) {
  const int tid = threadIdx.x;
  const int64_t base = slice * S;
  const int64_t row0 = (int64_t)tid * RPT;
  int32_t* keep = keep_idx + slice * budget;

  // all loads are issued up front; with many rows per thread the VaN column
  // waits until the TaR stage is done, to stay within the register budget
  constexpr bool kEarlyVan = RPT <= 16;
  uint32_t fr[RPT], kt[RPT], kv[RPT];
  load_row_run<RPT, VEC>(frame_idx + base, S, row0, fr);
  load_row_run<RPT, VEC>(tar + base, S, row0, kt);
  if (kEarlyVan) load_row_run<RPT, VEC>(van + base, S, row0, kv);
  const __amdgpu_buffer_rsrc_t frs = buffer_rsrc(frame_idx + base, (uint32_t)(S * 4));
  const int32_t last = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(frs, (uint32_t)(n - 1) * 4u, 0, 0);
  const int32_t prev_row = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(frs, (uint32_t)max(row0 - 1, (int64_t)0) * 4u,
                                                                          0, 0);
  const int32_t before = row0 > 0 ? prev_row : INT32_MIN;
  if (tid == 0) {
    sh.first_recent = n;
    sh.bad = 0;
  }
  __syncthreads();

  const int64_t thr = (int64_t)last - r + 1;
  uint64_t valid = 0, recent = 0;
  int32_t prev = before;
  bool bad = false, nan_t = false, nan_v = false;
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    if (row0 + i < n) {
      const int32_t f = (int32_t)fr[i];
      valid |= 1ull << i;
      const bool rec = (int64_t)f >= thr;
      if (rec) recent |= 1ull << i;
      if (rec && (int64_t)prev < thr) sh.first_recent = (int32_t)(row0 + i);  // the window's first row
      bad |= f < prev;
      prev = f;
      nan_t |= !rec && __uint_as_float(kt[i]) != __uint_as_float(kt[i]);
      if (kEarlyVan) nan_v |= !rec && __uint_as_float(kv[i]) != __uint_as_float(kv[i]);
    }
    kt[i] = order_key(__uint_as_float(kt[i]));
    if (kEarlyVan) kv[i] = order_key(__uint_as_float(kv[i]));
  }
  if (bad) sh.bad = 1;
  __syncthreads();
  // with non-decreasing frame ids the window is the suffix starting at first_recent
  const int32_t n_recent = n - sh.first_recent;
  const bool broken = sh.bad || n_recent > budget;
  if (broken) {
    // metadata breaks the cache invariants: report, and keep rows 0..C-1 in place
    if (tid == 0) raise_error(err, sh.bad ? 2u : 4u);
    for (int32_t j = tid; j < budget; j += NT) keep[j] = j;
  } else {
    const int32_t b_tar = max(0, tar_total - n_recent);
    const int32_t b_van = budget - n_recent - b_tar;
    const uint64_t past = valid & ~recent;
    uint64_t pick_t = 0, pick_v = 0;
    if (b_tar > 0) {
      if (nan_t) raise_error(err, 16u);
      pick_t = radix_top<NT, RPT>(kt, past, b_tar, sh);
    }
    if (b_van > 0) {
      if (!kEarlyVan) {
        load_row_run<RPT, VEC>(van + base, S, row0, kv);
#pragma unroll
        for (int i = 0; i < RPT; ++i) {
          nan_v |= ((past >> i) & 1ull) && __uint_as_float(kv[i]) != __uint_as_float(kv[i]);
          kv[i] = order_key(__uint_as_float(kv[i]));
        }
      }
      if (nan_v) raise_error(err, 16u);
      pick_v = radix_top<NT, RPT>(kv, past & ~pick_t, b_van, sh);
    }
    const uint64_t kept = recent | pick_t | pick_v;
    int32_t total;
    int32_t pos = block_exclusive_scan<NT>(__popcll(kept), sh, &total);
    if (total != budget && tid == 0) raise_error(err, 16u);  // only reachable with NaN keys
#pragma unroll
    for (int i = 0; i < RPT; ++i)
      if (((kept >> i) & 1ull) && pos < budget) keep[pos++] = (int32_t)(row0 + i);
  }
  __syncthreads();  // the caller may reuse sh
}

template <int NT, int RPT, bool VEC>
__global__ __launch_bounds__(NT) void k_select(const float* __restrict__ tar, const float* __restrict__ van,
                                               const int32_t* __restrict__ frame_idx, int64_t S, int32_t n,
                                               int32_t budget, int32_t tar_total, int32_t r,
                                               int32_t* __restrict__ keep_idx, uint32_t* err) {
  __shared__ SelShared<NT> sh;
  select_slice<NT, RPT, VEC>(tar, van, frame_idx, S, n, budget, tar_total, r, keep_idx, err, blockIdx.x, sh);
}

}  // namespace ipv
