// Consecutive-frame TaR: a past key is compared with one key only, the key at
// its patch position in the closest earlier frame that still holds that
// position (Sec. 3.1 measures static patches between adjacent frames; Tab. 5
// contrasts TaR variants). Score -cos(K[x], K[prev(x)]), 0 with no such row.
//
// Two kernels:
//   k_prev_rows       one 1024-thread block per slice takes the rows in chunks
//                     of 1024 and writes prev(x) (or -1) for every valid row;
//                     it also publishes the slice's first recent row and,
//                     optionally, zeroes the slice's compaction flags.
//   k_adjacent_sweep  the bandwidth part: for each past row, K[x] and
//                     K[prev(x)] (and V[x] when VaN is fused), one dot product
//                     and two norms per row.
#pragma once

#include "ipv_device.hpp"
#include "ipv_scores.hpp"  // the VaN tiles that share the walk's launch

namespace ipv {

constexpr int kPrevThreads = 1024;
constexpr int kPrevMaxPositions = 8192;

// prev(x), with frame ids non-decreasing along the rows: the latest row y < x
// at x's patch position whose frame is older than x's. The rows are taken in
// chunks of 1024, one row per thread. Inside a chunk the rows are bucketed by
// position with a counting sort in LDS (an atomic rank per row, an exclusive
// scan over the p counters, a scatter), so a row finds the latest earlier row
// of its position in the same chunk by looking through its own bucket only
// (about 1024 / p entries); if there is none, `last[q]` (the latest row at q
// in the chunks before) is the answer, and the row that is the last of its
// bucket updates `last[q]` for the next chunk. A second row with the same
// (frame, patch) pair, a frame id that decreases, or a patch id outside
// [0, p) sets an error bit; such metadata gives no defined prev.
//
// The chunk's frame ids are double-buffered in LDS; a chunk costs six
// barriers and no global-memory round trip (the next chunk's loads are in
// flight meanwhile). One slice's walk is one block of kPrevThreads threads.
__device__ __forceinline__ void prev_rows_block(int64_t slice, const int32_t* __restrict__ frame_idx,
                                                const int32_t* __restrict__ patch_idx, int64_t S, int32_t n,
                                                int32_t r, int32_t p, int32_t* __restrict__ prev,
                                                int32_t* __restrict__ first_recent, uint32_t* err,
                                                uint32_t* __restrict__ zero, int32_t zero_per_slice) {
  constexpr int NT = kPrevThreads;
  constexpr int BPT = (kPrevMaxPositions + 1 + NT - 1) / NT;  // scan entries per thread
  __shared__ int32_t last[kPrevMaxPositions];
  __shared__ int32_t cnt[kPrevMaxPositions + 1];  // counts, then bucket starts (cnt[p] = rows bucketed)
  __shared__ int32_t bucket[NT];
  __shared__ int32_t cfr[2][NT];  // chunk frame ids, double-buffered
  __shared__ int32_t scan_tot[NT / kWave];
  // carry: frame id of the previous chunk's last row, and the row its frame starts at
  __shared__ int32_t carry_frame, carry_start;
  const int tid = threadIdx.x;
  const int64_t base = slice * S;
  if (zero)
    for (int i = tid; i < zero_per_slice; i += NT) zero[slice * zero_per_slice + i] = 0u;
  for (int q = tid; q < p; q += NT) last[q] = -1;
  for (int q = tid; q <= p; q += NT) cnt[q] = 0;
  if (tid == 0) {
    carry_frame = INT32_MIN;
    carry_start = 0;
  }
  const int64_t thr = (int64_t)frame_idx[base + n - 1] - r + 1;
  uint32_t ebits = 0;
  int32_t nf = frame_idx[base + min((int64_t)tid, (int64_t)n - 1)];
  int32_t np = patch_idx[base + min((int64_t)tid, (int64_t)n - 1)];
  int b = 0;
  for (int64_t c0 = 0; c0 < n; c0 += NT, b ^= 1) {
    const int64_t x = c0 + tid;
    const bool valid = x < n;
    const int32_t f = nf, q = np;
    const bool inq = valid && q >= 0 && q < p;
    cfr[b][tid] = f;
    __syncthreads();  // (A) chunk metadata visible; counters zero
    {  // the next chunk's metadata is on its way meanwhile
      const int64_t xn = min(c0 + NT + tid, (int64_t)n - 1);
      nf = frame_idx[base + xn];
      np = patch_idx[base + xn];
    }
    const int32_t rank = inq ? atomicAdd(&cnt[q], 1) : 0;
    __syncthreads();  // (B) counts complete
    {  // exclusive scan of cnt[0..p] in place: thread t owns entries [t*BPT, (t+1)*BPT)
      int32_t v[BPT], sum = 0;
#pragma unroll
      for (int i = 0; i < BPT; ++i) {
        const int e = tid * BPT + i;
        v[i] = e <= p ? cnt[e] : 0;
        sum += v[i];
      }
      int32_t total;
      int32_t run = block_exclusive_scan<NT>(sum, scan_tot, &total);
#pragma unroll
      for (int i = 0; i < BPT; ++i) {
        const int e = tid * BPT + i;
        if (e <= p) cnt[e] = run;
        run += v[i];
      }
    }
    __syncthreads();  // (C) bucket starts visible
    if (inq) bucket[cnt[q] + rank] = tid;
    __syncthreads();  // (D) buckets filled
    const int32_t cf = carry_frame, cs = carry_start;
    const int cnt_rows = (int)min((int64_t)NT, (int64_t)n - c0);
    int32_t pred = -1;
    bool last_of_bucket = true;
    if (valid) {
      const int32_t fprev = tid > 0 ? cfr[b][tid - 1] : cf;
      if (f < fprev) ebits |= 2u;
      if ((int64_t)f >= thr && (int64_t)fprev < thr) first_recent[slice] = (int32_t)x;
      if (!inq) {
        ebits |= 1u;
      } else {
        // the latest row of this chunk before x at position q
        int hit = -1;
        const int lo = cnt[q], hi = cnt[q + 1];
        for (int i = lo; i < hi; ++i) {
          const int e = bucket[i];
          if (e < tid) hit = max(hit, e);
          last_of_bucket &= e <= tid;
        }
        const bool past = (int64_t)f < thr;
        if (hit >= 0) {
          if (cfr[b][hit] < f) {
            if (past) pred = (int32_t)(c0 + hit);
          } else {
            ebits |= 2u;  // the same (frame, patch) pair twice
          }
        } else {
          const int32_t L = last[q];
          if (L >= 0 && f == cf && L >= cs) ebits |= 2u;  // twice, across the chunk boundary
          else if (past) pred = L;
        }
      }
      prev[base + x] = pred;
    }
    __syncthreads();  // (E) every row has read last[], the buckets and the carry
    if (inq && last_of_bucket) last[q] = (int32_t)x;
    for (int e = tid; e <= p; e += NT) cnt[e] = 0;
    const int32_t fl = cfr[b][cnt_rows - 1];
    if (tid == cnt_rows - 1) carry_frame = fl;
    // the row where the last row's frame starts, if it starts in this chunk
    if (valid && f == fl && (tid > 0 ? cfr[b][tid - 1] != fl : cf != fl)) carry_start = (int32_t)x;
  }
  if (ebits) raise_error(err, ebits);
}

// grid: one block per slice
__global__ __launch_bounds__(kPrevThreads) void k_prev_rows(const int32_t* __restrict__ frame_idx,
                                                            const int32_t* __restrict__ patch_idx, int64_t S,
                                                            int32_t n, int32_t r, int32_t p,
                                                            int32_t* __restrict__ prev,
                                                            int32_t* __restrict__ first_recent, uint32_t* err,
                                                            uint32_t* __restrict__ zero, int32_t zero_per_slice) {
  prev_rows_block(blockIdx.x, frame_idx, patch_idx, S, n, r, p, prev, first_recent, err, zero, zero_per_slice);
}

// The prev-row walk and the VaN tiles of the sweep in one launch (VaN needs
// no prev rows, so V streams while the walks run): blocks [0, prev_padded)
// walk one slice each (those at or past `slices` return at once), the rest
// hold four VaN tiles of 256 threads each, XCD-mapped like the sweep.
// prev_padded is a multiple of 8, so tile block i + prev_padded runs on XCD
// i % 8.
template <typename T, int D>
__global__ __launch_bounds__(kPrevThreads) void k_prev_van(const T* __restrict__ V, const int32_t* __restrict__ frame_idx,
    const int32_t* __restrict__ patch_idx, int64_t S, int32_t n, int32_t r, int32_t p, int32_t* __restrict__ prev,
    int32_t* __restrict__ first_recent, uint32_t* err, uint32_t* __restrict__ zero, int32_t zero_per_slice,
    uint32_t prev_padded, uint32_t slices, float* __restrict__ van, TileGrid g) {
  if (blockIdx.x < prev_padded) {
    if (blockIdx.x < slices)
      prev_rows_block(blockIdx.x, frame_idx, patch_idx, S, n, r, p, prev, first_recent, err, zero, zero_per_slice);
    return;
  }
  using C = SweepCfg<T, D>;
  const uint32_t quad = xcd_logical_id(blockIdx.x - prev_padded, g.blocks);
  const uint32_t logical = quad * 4u + threadIdx.x / 256u;
  if (logical >= g.n_work) return;
  const uint32_t tile = fast_div(logical, g.col_blocks);
  const uint32_t colblock = logical - tile * g.col_blocks.d;
  const uint32_t slice = fast_div(tile, g.frame_blocks);
  const uint32_t f0 = (tile - slice * g.frame_blocks.d) * C::U;
  sweep_tile<T, D, false, true>(V, V, patch_idx, S, n, p, nullptr, n, nullptr, van, err, slice, f0, colblock,
                                threadIdx.x % 256u);
}

// TaR of the past rows against their prev rows. Rows are processed in
// natural order: a block covers GROUPS * U consecutive rows, GROUPS rows
// (contiguous bytes) per step, one lane group of LPR lanes (16 bytes each)
// per row. K[x] (past rows only) loads go out with the prev(x) loads;
// K[prev(x)] follows once prev(x) is known. Branch-free buffer loads: a lane
// with nothing to read uses an offset past the end.
template <typename T, int D>
__global__ __launch_bounds__(256) void k_adjacent_sweep(const T* __restrict__ K, const int32_t* __restrict__ prev,
                                                        int64_t S, int32_t n, const int32_t* __restrict__ first_recent,
                                                        float* __restrict__ tar, int32_t blocks_per_slice,
                                                        uint32_t n_work) {
  constexpr int EPL = Lane<T>::EPL, LPR = D / EPL, GROUPS = 256 / LPR, U = 4;
  constexpr uint32_t kSkip = 0xfffffff0u;
  constexpr uint32_t RB = D * (uint32_t)sizeof(T);
  const uint32_t logical = xcd_logical_id(blockIdx.x, gridDim.x);
  if (logical >= n_work) return;
  const int64_t slice = logical / blocks_per_slice;
  const int64_t r0 = (int64_t)(logical % blocks_per_slice) * GROUPS * U;
  const int tid = threadIdx.x, g = tid / LPR, lane = tid % LPR;
  const int64_t base = slice * S;
  const int32_t rec = first_recent[slice];
  const uint32_t lo = (uint32_t)lane * EPL * (uint32_t)sizeof(T);
  const __amdgpu_buffer_rsrc_t krs = buffer_rsrc(K + base * D, (uint32_t)S * RB);
  const __amdgpu_buffer_rsrc_t prs = buffer_rsrc(prev + base, (uint32_t)(S * 4));
  int32_t y[U];
  Raw16 kx[U], ky[U];
  auto load = [](const __amdgpu_buffer_rsrc_t& rs, uint32_t off, Raw16& out) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0);
    out.w[0] = v[0];
    out.w[1] = v[1];
    out.w[2] = v[2];
    out.w[3] = v[3];
  };
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t x = r0 + u * GROUPS + g;
    const bool past = x < n && x < rec;
    const int32_t yl = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(prs, past ? (uint32_t)x * 4u : kSkip, 0, 0);
    y[u] = past ? yl : -1;
    load(krs, past ? (uint32_t)x * RB + lo : kSkip, kx[u]);
  }
#pragma unroll
  for (int u = 0; u < U; ++u) load(krs, y[u] >= 0 ? (uint32_t)y[u] * RB + lo : kSkip, ky[u]);
  float tsc[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const float dot = group_sum<LPR>(Lane<T>::dot(kx[u], ky[u]));
    const float aa = group_sum<LPR>(Lane<T>::sumsq(kx[u]));
    const float cc = group_sum<LPR>(Lane<T>::sumsq(ky[u]));
    float sc = (y[u] >= 0 && aa != 0.f && cc != 0.f) ? -(dot * fast_rsqrt(aa) * fast_rsqrt(cc)) : 0.f;  // NaN stays NaN
    if (sc == 0.f) sc = 0.f;  // -0.0 -> +0.0
    tsc[u] = sc;
  }
  if (lane < U) {
    const int64_t x = r0 + lane * GROUPS + g;
    if (x < n) tar[base + x] = lane == 0 ? tsc[0] : lane == 1 ? tsc[1] : lane == 2 ? tsc[2] : tsc[3];
  }
}

}  // namespace ipv
