// Keep-set selection (Algorithm 1 steps (3)-(5); Sec. 3.3), one workgroup per
// (stream, layer, head) slice, or per (stream, layer) when the heads share one
// keep set. A workgroup has as many waves as its rows need, at most NT / 64
// (the host fits the launch); per-wave LDS slots of absent waves hold neutral
// values, so loops over all NT / 64 slots see only the present ones.
//
// Variants: a reversed stage (the TaR Reverse / VaN Reverse rows of Tab. 5)
// complements its keys, so the same top-k takes the lowest scores, ties still
// to the lowest rows. Head-shared selection ranks, per row, the fp32 sum of
// the layer's head scores taken in head order, checks that every head holds
// the same frame ids, and writes the one keep set to every head.
//
// Thread t owns the RPT consecutive rows [t*RPT, (t+1)*RPT). All of its frame
// ids and both score columns are loaded at once (16-byte buffer loads),
// turned into order-preserving 32-bit keys (-0.0 equal to +0.0) and kept in
// registers.
//
// Each stage picks the top k of its candidates with an MSB-first radix
// select over the keys: 8-bit digits starting below the bits that all the
// candidates share, an LDS histogram per digit, stopping as soon as the
// threshold bin holds exactly the keys still needed. Keys above the threshold
// prefix are in; if the bits run out first, the keys equal to it go to the
// lowest row indices (an exclusive scan of per-thread counts in row order).
// That is exactly "higher score first, then lower row index".
//
// Latency is set by the number of workgroup barriers, so:
//   * the block-wide minimum and maximum of both stages' keys come out of the
//     barrier that also publishes the window start (the VaN range is taken
//     over all past rows, a superset of its candidates, which still bounds
//     their common prefix);
//   * a digit costs two barriers: after the histogram's, wave 0 alone reads
//     it and finds the threshold digit, and publishes it for the second.
//     (Every wave repeating the scan saves that barrier but costs more: four
//     waves share a SIMD, so sixteen copies of the scan queue for issue.)
//     Histograms rotate over three LDS buffers, so a buffer is cleared only
//     after the barrier that follows its last reader;
//   * each histogram has kHistCopies copies, lane l adding into copy
//     l % kHistCopies, so lanes of one wave that hit the same bin mostly hit
//     different words in different banks;
//   * scans take one barrier: each wave adds up the wave totals it needs;
//   * the keep set is gathered in LDS in output order, kStageRows positions
//     at a time, then written with consecutive stores.
#pragma once

#include "ipv_device.hpp"

namespace ipv {

// A histogram is kHistCopies copies of 256 bins, copy-major with a skew of
// kHistSkew words so that the copies of one bin sit in different LDS banks:
// word copy * kHistStride + bin.
constexpr int kHistCopies = 4;
constexpr int kHistSkew = 4;
constexpr int kHistStride = 256 + kHistSkew;
constexpr int kHistWords = kHistCopies * kHistStride;
constexpr int kStageRows = 8192;  // keep-set positions gathered in LDS per round of stores

template <int NT>
struct SelShared {
  static constexpr int NW = NT / kWave;
  alignas(16) uint32_t hist[3][kHistWords];
  uint32_t wave_min[2][NW], wave_max[2][NW];  // [TaR, VaN] key ranges per wave
  uint32_t late_min[NW], late_max[NW];        // VaN range when its keys load late
  uint32_t wave_bad[NW];
  int32_t wave_tot[3][NW];                    // [TaR ties, VaN ties, output positions]
  int32_t first_recent;
  int32_t dig[3];                             // a digit's threshold digit, keys above it, keys in it
  int32_t stage[kStageRows];                  // the keep set in output order
};

// Neutral per-wave slots for the waves the launch does not have.
template <int NT>
__device__ __forceinline__ void neutral_missing_waves(SelShared<NT>& sh) {
  const int t = threadIdx.x, nw = (int)(blockDim.x / kWave);
  if (t >= nw && t < NT / kWave) {
    sh.wave_min[0][t] = sh.wave_min[1][t] = sh.late_min[t] = 0xffffffffu;
    sh.wave_max[0][t] = sh.wave_max[1][t] = sh.late_max[t] = 0u;
    sh.wave_bad[t] = 0u;
    sh.wave_tot[0][t] = sh.wave_tot[1][t] = sh.wave_tot[2][t] = 0;
  }
}

// State of one stage's digit loop, the same in every thread.
struct Radix {
  uint32_t prefix, pmask;
  int32_t remaining;
  bool done;
};

// The digit loop for the top k of `cand` keys whose common bits are those of
// [mn, mx]. `buf` is the rotating histogram counter (shared by both stages).
template <int NT, int RPT>
__device__ __forceinline__ Radix radix_digits(const uint32_t (&key)[RPT], uint64_t cand, int32_t k, uint32_t mn,
                                              uint32_t mx, SelShared<NT>& sh, int& buf) {
  const int tid = threadIdx.x, lane = tid % kWave;
  const int common = (mn == mx) ? 32 : __clz((int)(mn ^ mx));
  Radix R;
  R.pmask = common == 0 ? 0u : (common == 32 ? 0xffffffffu : 0xffffffffu << (32 - common));
  R.prefix = mn & R.pmask;
  R.remaining = k;
  R.done = false;
  const int copy = lane % kHistCopies;
#pragma unroll 1
  for (int top = 32 - common; top > 0 && !R.done; top -= 8) {
    const int shift = max(0, top - 8);
    const uint32_t dmask = (1u << (top - shift)) - 1u;
    uint32_t* h = sh.hist[buf];
#pragma unroll
    for (int i = 0; i < RPT; ++i)
      if (((cand >> i) & 1ull) && (key[i] & R.pmask) == R.prefix)
        atomicAdd(&h[copy * kHistStride + ((key[i] >> shift) & dmask)], 1u);
    // the next digit's buffer, last read two digits ago
    uint32_t* nxt = sh.hist[buf == 2 ? 0 : buf + 1];
    for (int i = tid; i < kHistWords; i += (int)blockDim.x) nxt[i] = 0u;
    __syncthreads();
    if (tid < kWave) {
      // wave 0: lane l holds digits 255-4l .. 252-4l (descending digit order),
      // read as one 16-byte run of bins 252-4l .. 255-4l per copy
      int32_t c[4] = {0, 0, 0, 0};
#pragma unroll
      for (int cp = 0; cp < kHistCopies; ++cp) {
        const uint4 v = *reinterpret_cast<const uint4*>(h + cp * kHistStride + 252 - 4 * lane);
        c[0] += (int32_t)v.w;
        c[1] += (int32_t)v.z;
        c[2] += (int32_t)v.y;
        c[3] += (int32_t)v.x;
      }
      const int32_t s = c[0] + c[1] + c[2] + c[3];
      const int32_t incl = wave_inclusive_scan(s);
      const int32_t excl = incl - s;
      // the lane holding the threshold digit: the one whose run of bins
      // reaches the remaining count (exactly one lane)
      if (excl < R.remaining && R.remaining <= incl) {
        int32_t above = excl, j = 0;
        while (j < 3 && above + c[j] < R.remaining) above += c[j++];
        sh.dig[0] = 255 - 4 * lane - j;
        sh.dig[1] = above;
        sh.dig[2] = j == 0 ? c[0] : (j == 1 ? c[1] : (j == 2 ? c[2] : c[3]));
      }
    }
    __syncthreads();
    const int32_t d = sh.dig[0], a = sh.dig[1], cnt = sh.dig[2];
    R.remaining -= a;
    R.prefix |= (uint32_t)d << shift;
    R.pmask |= dmask << shift;
    R.done = cnt == R.remaining;  // the threshold bin is taken whole
    buf = buf == 2 ? 0 : buf + 1;
  }
  return R;
}

// This thread's picks among `cand` after the digit loop. Ties on the full
// key (the loop ran out of bits) go to the lowest rows.
template <int NT, int RPT>
__device__ __forceinline__ uint64_t radix_picks(const uint32_t (&key)[RPT], uint64_t cand, const Radix& R,
                                                int32_t* tie_tot) {
  uint64_t pick = 0, eq = 0;
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    if (!((cand >> i) & 1ull)) continue;
    const uint32_t mk = key[i] & R.pmask;
    if (mk > R.prefix) pick |= 1ull << i;
    if (mk == R.prefix) eq |= 1ull << i;
  }
  if (R.done) return pick | eq;
  int32_t tot;
  int32_t taken = block_exclusive_scan<NT>(__popcll(eq), tie_tot, &tot);
#pragma unroll
  for (int i = 0; i < RPT; ++i)
    if ((eq >> i) & 1ull) {
      if (taken < R.remaining) pick |= 1ull << i;
      ++taken;
    }
  return pick;
}

// Block-wide min and max of this thread's candidate keys (one barrier).
template <int NT, int RPT>
__device__ __forceinline__ void block_min_max(const uint32_t (&key)[RPT], uint64_t cand, SelShared<NT>& sh,
                                              uint32_t& mn, uint32_t& mx) {
  constexpr int NW = NT / kWave;
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
  mn = 0xffffffffu;
  mx = 0u;
#pragma unroll
  for (int i = 0; i < RPT; ++i)
    if ((cand >> i) & 1ull) {
      mn = min(mn, key[i]);
      mx = max(mx, key[i]);
    }
  wave_min_max(mn, mx);
  if (lane == 0) {
    sh.late_min[w] = mn;
    sh.late_max[w] = mx;
  }
  __syncthreads();
  // lane i reads wave i's range, a wave reduction combines them
  mn = lane < NW ? sh.late_min[lane] : 0xffffffffu;
  mx = lane < NW ? sh.late_max[lane] : 0u;
  wave_min_max(mn, mx);
}

// Rows [row0, row0 + RPT) of one slice's column (S rows of 4 bytes); rows at
// or past S read as 0, and so does every row when `present` is false (an
// empty resource). VEC: rows are 16-byte aligned (S % 4 == 0), so a run lies
// wholly inside or wholly past the column and loads 16 bytes at a time.
template <int RPT, bool VEC>
__device__ __forceinline__ void load_row_run(const void* __restrict__ col, int64_t S, int64_t row0,
                                             uint32_t (&out)[RPT], bool present = true) {
  const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(col, present ? (uint32_t)(S * 4) : 0u);
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

// Heads after the first whose runs are loaded together (the rest of a
// layer's heads in one round trip when a thread holds few rows).
template <int RPT>
constexpr int head_batch() { return RPT <= 8 ? 3 : 1; }

// A score run summed over `heads` consecutive slices (column stride S) in
// fp32, head 0 first, starting from +0 (the order the keep decision is
// defined in); heads == 1 is the slice's own run. Absent heads of a batch
// read as +0, which leaves every sum unchanged.
template <int RPT, bool VEC>
__device__ __forceinline__ void load_score_run(const float* __restrict__ col, int64_t S, int32_t heads, int64_t row0,
                                               uint32_t (&out)[RPT]) {
  constexpr int G = head_batch<RPT>();
  load_row_run<RPT, VEC>(col, S, row0, out);
  if (heads == 1) return;
#pragma unroll
  for (int i = 0; i < RPT; ++i) out[i] = __float_as_uint(0.f + __uint_as_float(out[i]));
#pragma unroll 1
  for (int32_t h = 1; h < heads; h += G) {
    uint32_t t[G][RPT];
#pragma unroll
    for (int g = 0; g < G; ++g) load_row_run<RPT, VEC>(col + min(h + g, heads - 1) * S, S, row0, t[g], h + g < heads);
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int i = 0; i < RPT; ++i) out[i] = __float_as_uint(__uint_as_float(out[i]) + __uint_as_float(t[g][i]));
  }
}

// Head-shared selection: true if some head's frame ids differ from head 0's
// on this thread's rows.
template <int RPT, bool VEC>
__device__ __forceinline__ bool heads_differ(const int32_t* __restrict__ fr0, int64_t S, int32_t heads, int64_t row0,
                                             int32_t n, const uint32_t (&fr)[RPT]) {
  constexpr int G = head_batch<RPT>();
  bool diff = false;
#pragma unroll 1
  for (int32_t h = 1; h < heads; h += G) {
    uint32_t t[G][RPT];
#pragma unroll
    for (int g = 0; g < G; ++g) load_row_run<RPT, VEC>(fr0 + min(h + g, heads - 1) * S, S, row0, t[g], h + g < heads);
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int i = 0; i < RPT; ++i) diff |= h + g < heads && row0 + i < n && t[g][i] != fr[i];
  }
  return diff;
}

// Writes the keep set: `kept` marks this thread's kept rows among its RPT
// rows from row0, `pos` is the number of kept rows before them. `put(j, row)`
// stores output position j. The set is gathered in LDS in output order,
// kStageRows positions at a time, so that the global stores are consecutive
// across the block.
template <int NT, int RPT, typename Put>
__device__ __forceinline__ void write_keep(uint64_t kept, int32_t pos, int32_t budget, int64_t row0,
                                           SelShared<NT>& sh, Put put) {
  for (int32_t lo = 0; lo < budget; lo += kStageRows) {
    const int32_t hi = min(budget, lo + kStageRows);
    int32_t q = pos;
#pragma unroll
    for (int i = 0; i < RPT; ++i)
      if (((kept >> i) & 1ull) && q < budget) {
        if (q >= lo && q < hi) sh.stage[q - lo] = (int32_t)(row0 + i);
        ++q;
      }
    __syncthreads();
    for (int32_t j = threadIdx.x; j < hi - lo; j += (int32_t)blockDim.x) put(lo + j, sh.stage[j]);
    if (hi < budget) __syncthreads();  // the next positions reuse the stage
  }
}

// One group of `heads` slices (1: a slice of its own) with NT threads. VEC:
// every slice's row 0 is 16-byte aligned (capacity % 4 == 0) so row runs
// load 16 bytes at a time. tflip / vflip: 0, or ~0 for a reversed stage.
template <int NT, int RPT, bool VEC>
__device__ __forceinline__ void select_slice(const float* __restrict__ tar, const float* __restrict__ van,
                             const int32_t* __restrict__ frame_idx, int64_t S, int32_t n, int32_t budget,
                             int32_t tar_total, int32_t r, int32_t* __restrict__ keep_idx,
                             uint32_t* err, int64_t slice, int32_t heads, uint32_t tflip, uint32_t vflip,
                             SelShared<NT>& sh) {
  constexpr int NW = NT / kWave;
  const int tid = threadIdx.x, lane = tid % kWave, w = tid / kWave;
  const int64_t base = slice * S;
  const int64_t row0 = (int64_t)tid * RPT;
  int32_t* keep = keep_idx + slice * budget;
  // every head of the group gets the same keep set
  auto put = [&](int32_t j, int32_t row) {
    if (heads == 1) {
      keep[j] = row;
      return;
    }
    for (int32_t h = 0; h < heads; ++h) keep[(int64_t)h * budget + j] = row;
  };

  // all loads are issued up front; with many rows per thread the VaN column
  // waits until the TaR stage is done, to stay within the register budget
  constexpr bool kEarlyVan = RPT <= 16;
  uint32_t fr[RPT], kt[RPT], kv[RPT];
  load_row_run<RPT, VEC>(frame_idx + base, S, row0, fr);
  load_score_run<RPT, VEC>(tar + base, S, heads, row0, kt);
  if (kEarlyVan) load_score_run<RPT, VEC>(van + base, S, heads, row0, kv);
  const __amdgpu_buffer_rsrc_t frs = buffer_rsrc(frame_idx + base, (uint32_t)(S * 4));
  const int32_t last = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(frs, (uint32_t)(n - 1) * 4u, 0, 0);
  const int32_t prev_row = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(frs, (uint32_t)max(row0 - 1, (int64_t)0) * 4u,
                                                                          0, 0);
  const int32_t before = row0 > 0 ? prev_row : INT32_MIN;
  for (int i = tid; i < kHistWords; i += (int)blockDim.x) sh.hist[0][i] = 0u;
  neutral_missing_waves<NT>(sh);

  const int64_t thr = (int64_t)last - r + 1;
  uint64_t valid = 0, recent = 0;
  int32_t prev = before;
  bool bad = heads > 1 && heads_differ<RPT, VEC>(frame_idx + base, S, heads, row0, n, fr);
  bool nan_t = false, nan_v = false;
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    if (row0 + i < n) {
      const int32_t f = (int32_t)fr[i];
      valid |= 1ull << i;
      const bool rec = (int64_t)f >= thr;
      if (rec) recent |= 1ull << i;
      // the window's first row: with any frame ids, at least one row has a
      // recent frame and a non-recent predecessor (or is row 0); with
      // non-decreasing ids exactly one
      if (rec && (int64_t)prev < thr) sh.first_recent = (int32_t)(row0 + i);
      bad |= f < prev;
      prev = f;
      nan_t |= !rec && __uint_as_float(kt[i]) != __uint_as_float(kt[i]);
      if (kEarlyVan) nan_v |= !rec && __uint_as_float(kv[i]) != __uint_as_float(kv[i]);
    }
    kt[i] = order_key(__uint_as_float(kt[i])) ^ tflip;
    if (kEarlyVan) kv[i] = order_key(__uint_as_float(kv[i])) ^ vflip;
  }
  const uint64_t past = valid & ~recent;
  // key ranges of both stages over the past rows, and the frame check
  uint32_t tmn = 0xffffffffu, tmx = 0u, vmn = 0xffffffffu, vmx = 0u;
#pragma unroll
  for (int i = 0; i < RPT; ++i)
    if ((past >> i) & 1ull) {
      tmn = min(tmn, kt[i]);
      tmx = max(tmx, kt[i]);
      if (kEarlyVan) {
        vmn = min(vmn, kv[i]);
        vmx = max(vmx, kv[i]);
      }
    }
  wave_min_max(tmn, tmx);
  if (kEarlyVan) wave_min_max(vmn, vmx);
  const bool wbad = __ballot(bad) != 0;
  if (lane == 0) {
    sh.wave_min[0][w] = tmn;
    sh.wave_max[0][w] = tmx;
    sh.wave_min[1][w] = vmn;
    sh.wave_max[1][w] = vmx;
    sh.wave_bad[w] = wbad;
  }
  __syncthreads();
  bool any_bad = false;
  // lane i reads wave i's ranges, wave reductions combine them
  tmn = lane < NW ? sh.wave_min[0][lane] : 0xffffffffu;
  tmx = lane < NW ? sh.wave_max[0][lane] : 0u;
  vmn = lane < NW ? sh.wave_min[1][lane] : 0xffffffffu;
  vmx = lane < NW ? sh.wave_max[1][lane] : 0u;
  wave_min_max(tmn, tmx);
  wave_min_max(vmn, vmx);
  any_bad = __ballot(lane < NW && sh.wave_bad[lane] != 0) != 0;
  // with non-decreasing frame ids the window is the suffix starting at first_recent
  const int32_t n_recent = n - sh.first_recent;
  const bool broken = any_bad || n_recent > budget;
  if (broken) {
    // metadata breaks the cache invariants: report, and keep rows 0..C-1 in place
    if (tid == 0) raise_error(err, any_bad ? 2u : 4u);
    for (int32_t j = tid; j < budget; j += (int32_t)blockDim.x) put(j, j);
    return;
  }
  const int32_t b_tar = max(0, tar_total - n_recent);
  const int32_t b_van = budget - n_recent - b_tar;
  uint64_t pick_t = 0, pick_v = 0;
  int buf = 0;
  if (b_tar > 0) {
    if (nan_t) raise_error(err, 16u);
    const Radix R = radix_digits<NT, RPT>(kt, past, b_tar, tmn, tmx, sh, buf);
    pick_t = radix_picks<NT, RPT>(kt, past, R, sh.wave_tot[0]);
  }
  if (b_van > 0) {
    const uint64_t cand = past & ~pick_t;
    if (!kEarlyVan) {
      load_score_run<RPT, VEC>(van + base, S, heads, row0, kv);
#pragma unroll
      for (int i = 0; i < RPT; ++i) {
        nan_v |= ((past >> i) & 1ull) && __uint_as_float(kv[i]) != __uint_as_float(kv[i]);
        kv[i] = order_key(__uint_as_float(kv[i])) ^ vflip;
      }
      block_min_max<NT, RPT>(kv, cand, sh, vmn, vmx);
    }
    if (nan_v) raise_error(err, 16u);
    const Radix R = radix_digits<NT, RPT>(kv, cand, b_van, vmn, vmx, sh, buf);
    pick_v = radix_picks<NT, RPT>(kv, cand, R, sh.wave_tot[1]);
  }
  const uint64_t kept = recent | pick_t | pick_v;
  int32_t total;
  int32_t pos = block_exclusive_scan<NT>(__popcll(kept), sh.wave_tot[2], &total);
  if (total != budget && tid == 0) raise_error(err, 16u);  // only reachable with NaN keys
  write_keep<NT, RPT>(kept, pos, budget, row0, sh, put);
}

// ---------------------------------------------------------------- Uniform Select
// The frame-sampling baseline of the KV-compression comparison (appendix, KV
// cache compression details: frames at regular intervals, every token of a
// taken frame), from frame ids alone. The recent window is kept; the past
// rows [0, |P|) hold q frames, numbered 0..q-1 in row order; the past budget
// b = C - |R| buys k = ceil(b * q / |P|) frames at ranks floor(j * q / k). A
// frame of rank i is taken iff some j * q / k lies in [i, i + 1), i.e.
// ceil(i * k / q) * q < (i + 1) * k. The b past rows kept are the taken
// frames' rows in row order, then (if those hold fewer than b rows) the
// lowest other past rows. Two block scans: frame starts give each row its
// rank, taken rows give each row its place among them; a row's place among
// the other past rows is its index minus the taken rows before it, since the
// past is a prefix of the slice.
__device__ __forceinline__ bool uniform_taken(int64_t rank, int64_t k, int64_t q) {
  return (rank * k + q - 1) / q * q < (rank + 1) * k;
}

template <int NT, int RPT, bool VEC>
__device__ __forceinline__ void uniform_slice(const int32_t* __restrict__ frame_idx, int64_t S, int32_t n,
                                              int32_t budget, int32_t r, int32_t* __restrict__ keep_idx,
                                              uint32_t* err, int64_t slice, int32_t heads, uint32_t* __restrict__ zero,
                                              int32_t zero_per_slice, SelShared<NT>& sh) {
  constexpr int NW = NT / kWave;
  const int tid = threadIdx.x, lane = tid % kWave, w = tid / kWave;
  const int64_t base = slice * S;
  const int64_t row0 = (int64_t)tid * RPT;
  int32_t* keep = keep_idx + slice * budget;
  auto put = [&](int32_t j, int32_t row) {
    for (int32_t h = 0; h < heads; ++h) keep[(int64_t)h * budget + j] = row;
  };
  // no score kernel runs before this selection in a pass: it zeroes the
  // compaction flags of its slices (zero_per_slice words each) instead
  if (zero)
    for (int64_t i = tid; i < (int64_t)heads * zero_per_slice; i += (int64_t)blockDim.x)
      zero[slice * zero_per_slice + i] = 0u;

  neutral_missing_waves<NT>(sh);
  uint32_t fr[RPT];
  load_row_run<RPT, VEC>(frame_idx + base, S, row0, fr);
  const __amdgpu_buffer_rsrc_t frs = buffer_rsrc(frame_idx + base, (uint32_t)(S * 4));
  const int32_t last = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(frs, (uint32_t)(n - 1) * 4u, 0, 0);
  const int32_t before = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(
      frs, (uint32_t)max(row0 - 1, (int64_t)0) * 4u, 0, 0);
  const int64_t thr = (int64_t)last - r + 1;
  uint64_t valid = 0, recent = 0, start = 0;
  bool bad = heads > 1 && heads_differ<RPT, VEC>(frame_idx + base, S, heads, row0, n, fr);
  int32_t prev = before;
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    if (row0 + i < n) {
      const int32_t f = (int32_t)fr[i];
      const bool first = row0 + i == 0;
      valid |= 1ull << i;
      const bool rec = (int64_t)f >= thr;
      if (rec) recent |= 1ull << i;
      if (rec && (first || (int64_t)prev < thr)) sh.first_recent = (int32_t)(row0 + i);
      if (first || f != prev) start |= 1ull << i;
      bad |= !first && f < prev;
      prev = f;
    }
  }
  const bool wbad = __ballot(bad) != 0;
  if (lane == 0) sh.wave_bad[w] = wbad;
  __syncthreads();
  bool any_bad = false;
#pragma unroll
  for (int i = 0; i < NW; ++i) any_bad |= sh.wave_bad[i] != 0;
  const int32_t n_past = sh.first_recent;
  const int32_t n_recent = n - n_past;
  if (any_bad || n_recent > budget) {
    if (tid == 0) raise_error(err, any_bad ? 2u : 4u);
    for (int32_t j = tid; j < budget; j += (int32_t)blockDim.x) put(j, j);
    return;
  }
  const uint64_t past = valid & ~recent;
  const int32_t b = budget - n_recent;
  uint64_t pick = 0;
  if (b > 0) {
    // each row's frame rank among the past frames
    int32_t q32;
    const int32_t rank0 = block_exclusive_scan<NT>(__popcll(start & past), sh.wave_tot[0], &q32);
    const int64_t q = q32;
    const int64_t k = ((int64_t)b * q + n_past - 1) / n_past;
    uint64_t taken = 0;
    int64_t rank = rank0 - 1;  // the frame this thread's first row continues, if it is no start
    bool tk = rank >= 0 && uniform_taken(rank, k, q);
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      if (!((past >> i) & 1ull)) continue;
      if ((start >> i) & 1ull) tk = uniform_taken(++rank, k, q);
      if (tk) taken |= 1ull << i;
    }
    // places among the taken rows, and among the other past rows
    int32_t total;
    int32_t tpos = block_exclusive_scan<NT>(__popcll(taken), sh.wave_tot[1], &total);
    const int32_t fill = b - total;  // other past rows needed (if positive)
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      if (!((past >> i) & 1ull)) continue;
      if ((taken >> i) & 1ull) {
        if (tpos < b) pick |= 1ull << i;
        ++tpos;
      } else if (row0 + i - tpos < fill) {
        pick |= 1ull << i;
      }
    }
  }
  const uint64_t kept = recent | pick;
  int32_t total;
  int32_t pos = block_exclusive_scan<NT>(__popcll(kept), sh.wave_tot[2], &total);
  write_keep<NT, RPT>(kept, pos, budget, row0, sh, put);
}

// grid: one block per group of `heads` consecutive slices (heads > 1: every
// head must hold the same frame ids and receives the same keep set).
// zero (may be null): zero_per_slice words per slice to clear
template <int NT, int RPT, bool VEC>
__global__ __launch_bounds__(NT) void k_select_uniform(const int32_t* __restrict__ frame_idx, int64_t S, int32_t n,
                                                       int32_t budget, int32_t r, int32_t* __restrict__ keep_idx,
                                                       uint32_t* err, int32_t heads, uint32_t* __restrict__ zero,
                                                       int32_t zero_per_slice) {
  __shared__ SelShared<NT> sh;
  uniform_slice<NT, RPT, VEC>(frame_idx, S, n, budget, r, keep_idx, err, (int64_t)blockIdx.x * heads, heads, zero,
                              zero_per_slice, sh);
}

// grid: one block per group of `heads` consecutive slices
template <int NT, int RPT, bool VEC>
__global__ __launch_bounds__(NT) void k_select(const float* __restrict__ tar, const float* __restrict__ van,
                                               const int32_t* __restrict__ frame_idx, int64_t S, int32_t n,
                                               int32_t budget, int32_t tar_total, int32_t r,
                                               int32_t* __restrict__ keep_idx, uint32_t* err, int32_t heads,
                                               uint32_t tflip, uint32_t vflip) {
  __shared__ SelShared<NT> sh;
  select_slice<NT, RPT, VEC>(tar, van, frame_idx, S, n, budget, tar_total, r, keep_idx, err,
                             (int64_t)blockIdx.x * heads, heads, tflip, vflip, sh);
}

}  // namespace ipv
