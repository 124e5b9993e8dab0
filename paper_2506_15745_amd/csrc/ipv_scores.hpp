// Scoring kernels of the compression pass: the recent-key table, the row
// sweep (TaR and VaN tiles), and the layer-adaptive VaN pooling. A pass that
// needs both scores runs the table and the VaN tiles in one launch, then the
// TaR tiles.
//
// TaR (Sec. 3.1, TaR equation) averages cos(K[x], K[y]) over the recent rows y
// at x's patch position. Cosine is linear in the unit vectors, so
//   -(1/r_q) sum_y cos(K[x], K[y]) = -(K[x]/|K[x]|) . m_q,
//   m_q = (1/r_q) sum_y K[y]/|K[y]|   (zero keys contribute the zero vector),
// and the sweep reads each past key once against a per-slice table of m_q
// (fp32, p x D) that the first kernel builds from the recent window.
#pragma once

#include "ipv_device.hpp"

namespace ipv {

// ---------------------------------------------------------------- recent-key table
// One block of NT threads per (slice, GROUPS = NT / LPR patch positions).
// Each lane group of LPR lanes owns one patch position q and sums the unit
// recent keys at q in frame order (deterministic), then scales by 1/r_q.
// Positions with no recent key get m_q = 0, which makes their TaR score 0.
// slot (LDS, GROUPS * r ints): slot[g * r + (frame - first recent frame)] =
// row of that key, or -1. The block with q0 == 0 also publishes the slice's
// first recent row, which the sweep uses to skip recent keys.
//
// Latency: every global load that does not depend on another is issued
// before any result is used. A recent frame holds at most p rows, so the
// window lies in the last r*p rows, t0 = n - r*p onwards; when those rows are
// r whole frames in patch order (a cache that was filled frame by frame since
// the last compaction), the key of recent frame j at position q is row
// t0 + j*p + q. The first kSpecFrames of those rows are loaded before the
// window is scanned, and used if the scan's slot table names the same rows;
// otherwise (or for later frames) the keys are loaded from the slot rows.
constexpr int kSpecFrames = 4;  // = the batch size of the summing loop below
constexpr int kScanBatch = 4;

template <typename T, int D, int NT>
__device__ __forceinline__ void table_block(const T* __restrict__ K, const int32_t* __restrict__ frame_idx,
                            const int32_t* __restrict__ patch_idx, int64_t S, int32_t n, int32_t r, int32_t p,
                            int64_t slice, int32_t q0, float* __restrict__ table, int32_t* __restrict__ first_recent,
                            uint32_t* err, int32_t* slot) {
  constexpr int EPL = Lane<T>::EPL;
  constexpr int LPR = D / EPL;
  constexpr int GROUPS = NT / LPR;
  const int tid = threadIdx.x;
  const int32_t q1 = min(p, q0 + GROUPS);
  const int64_t base = slice * S;
  const int g = tid / LPR, lane = tid % LPR;
  const int32_t q = q0 + g;
  const int64_t t0 = max((int64_t)0, (int64_t)n - (int64_t)r * p);

  // Loads take clamped (in-range) indices instead of branches, so that they
  // are all in flight together; values of clamped loads are never used. The
  // window scan reads NT * kScanBatch rows per batch (the whole window in the
  // usual case); its loads are issued first, then the speculative key loads,
  // and an empty asm statement takes the scan values, so the scan waits for
  // its own loads only and the compiler cannot move them into the branches
  // below. Errors are collected in a register and raised once.
  int32_t f[kScanBatch], fprev[kScanBatch], pq[kScanBatch];
  auto load_batch = [&](int64_t tb) {
#pragma unroll
    for (int b = 0; b < kScanBatch; ++b) {
      const int64_t t = min(tb + (int64_t)b * NT + tid, (int64_t)n - 1);
      f[b] = frame_idx[base + t];
      pq[b] = patch_idx[base + t];
      fprev[b] = frame_idx[base + max(t - 1, t0)];
    }
  };
  const int64_t thr = (int64_t)frame_idx[base + n - 1] - r + 1;
  uint32_t ebits = 0;
  auto scan_batch = [&](int64_t tb) {
#pragma unroll
    for (int b = 0; b < kScanBatch; ++b) asm volatile("" ::"v"(f[b]), "v"(pq[b]), "v"(fprev[b]));
#pragma unroll
    for (int b = 0; b < kScanBatch; ++b) {
      const int64_t t = tb + (int64_t)b * NT + tid;
      if (t >= n || f[b] < thr) continue;
      // the window's first row: the one recent row whose predecessor is not
      // recent (or the scan start); with non-decreasing frame ids there is one
      if (q0 == 0 && (t == t0 || fprev[b] < thr)) first_recent[slice] = (int32_t)t;
      const int64_t fo = (int64_t)f[b] - thr;
      if (pq[b] < 0 || pq[b] >= p) {
        ebits |= 1u;
      } else if (fo >= r) {  // a frame id above the last row's: ids decrease somewhere
        ebits |= 2u;
      } else if (pq[b] >= q0 && pq[b] < q1) {
        if (atomicExch(&slot[(pq[b] - q0) * r + fo], (int32_t)t) != -1) ebits |= 2u;
      }
    }
  };
  load_batch(t0);
  Raw16 spec[kSpecFrames];
#pragma unroll
  for (int j = 0; j < kSpecFrames; ++j) {
    const int64_t x = min(t0 + (int64_t)j * p + q, (int64_t)n - 1);
    spec[j] = load16(K + (base + x) * D + lane * EPL);
  }
  // the slot table is cleared while the loads are in flight
  for (int i = tid; i < GROUPS * r; i += NT) slot[i] = -1;
  __syncthreads();
  scan_batch(t0);
  for (int64_t tb = t0 + (int64_t)NT * kScanBatch; tb < n; tb += (int64_t)NT * kScanBatch) {
    load_batch(tb);
    scan_batch(tb);
  }
  if (ebits) raise_error(err, ebits);
  __syncthreads();

  float acc[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) acc[i] = 0.f;
  int cnt = 0;
  if (q < q1) {
    // batches of 4 independent key loads, summed in frame order
    for (int j0 = 0; j0 < r; j0 += 4) {
      Raw16 raw[4];
      int32_t y[4];
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int j = j0 + b;
        y[b] = j < r ? slot[g * r + j] : -1;
        if (y[b] < 0) continue;  // uniform within the lane group
        if (j0 == 0 && y[b] == t0 + (int64_t)b * p + q)  // b < kSpecFrames: a fixed register
          raw[b] = spec[b];
        else
          raw[b] = load16(K + (base + y[b]) * D + lane * EPL);
      }
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        if (y[b] < 0) continue;
        ++cnt;
        float f[EPL];
        Lane<T>::decode(raw[b], f);
        const float ss = group_sum<LPR>(Lane<T>::sumsq(raw[b]));
        const float inv = ss > 0.f ? fast_rsqrt(ss) : 0.f;
#pragma unroll
        for (int i = 0; i < EPL; ++i) acc[i] += f[i] * inv;
      }
    }
    const float scale = cnt ? 1.f / (float)cnt : 0.f;
    float* out = table + ((int64_t)slice * p + q) * D + lane * EPL;
#pragma unroll
    for (int i = 0; i < EPL; i += 4)
      *reinterpret_cast<float4*>(out + i) = make_float4(acc[i] * scale, acc[i + 1] * scale, acc[i + 2] * scale,
                                                        acc[i + 3] * scale);
  }
}

// Table block `tb` of the grid: slice tb / blocks_per_slice, GROUPS patch
// positions from (tb % blocks_per_slice) * GROUPS. zero (optional): the first
// block of each slice also zeroes zero_per_slice words at
// zero + slice * zero_per_slice (the compaction flags of a pass, saving a
// launch). `slot`: GROUPS * r ints of LDS.
template <typename T, int D>
__device__ __forceinline__ void table_grid_block(uint32_t tb, const T* __restrict__ K,
                                                 const int32_t* __restrict__ frame_idx,
                                                 const int32_t* __restrict__ patch_idx, int64_t S, int32_t n,
                                                 int32_t r, int32_t p, int32_t blocks_per_slice,
                                                 float* __restrict__ table, int32_t* __restrict__ first_recent,
                                                 uint32_t* err, uint32_t* __restrict__ zero, int32_t zero_per_slice,
                                                 int32_t* slot) {
  constexpr int GROUPS = 256 / (D / Lane<T>::EPL);
  const int64_t slice = tb / blocks_per_slice;
  const int32_t q0 = (int32_t)(tb % blocks_per_slice) * GROUPS;
  if (zero && q0 == 0)
    for (int i = threadIdx.x; i < zero_per_slice; i += 256) zero[slice * zero_per_slice + i] = 0u;
  table_block<T, D, 256>(K, frame_idx, patch_idx, S, n, r, p, slice, q0, table, first_recent, err, slot);
}

template <typename T, int D>
__global__ __launch_bounds__(256) void k_recent_table(const T* __restrict__ K, const int32_t* __restrict__ frame_idx,
                                                      const int32_t* __restrict__ patch_idx, int64_t S, int32_t n,
                                                      int32_t r, int32_t p, int32_t blocks_per_slice,
                                                      float* __restrict__ table, int32_t* __restrict__ first_recent,
                                                      uint32_t* err, uint32_t* __restrict__ zero,
                                                      int32_t zero_per_slice) {
  extern __shared__ int32_t slot[];
  table_grid_block<T, D>(blockIdx.x, K, frame_idx, patch_idx, S, n, r, p, blocks_per_slice, table, first_recent, err,
                         zero, zero_per_slice, slot);
}

// ---------------------------------------------------------------- TaR / VaN row sweep
// Rows are tiled over the (frame, patch) plane of the row space: row x is
// taken as frame x / p, patch x % p. This covers every row exactly once for
// any layout, and it is the true position of every row in a cache filled with
// whole frames. A tile is GROUPS consecutive patch columns by U frames; each
// lane group (LPR lanes, 16 bytes per lane) owns one column, so for every
// frame step the workgroup reads GROUPS consecutive rows (contiguous bytes).
//
// A column's U rows normally share one patch, hence one m vector: the group
// fetches m for the column's own patch position at the same time as the K/V
// loads (no dependence on patch_idx), then checks every row's real patch_idx
// and fetches the right m vector for any row where the two differ. The result
// never depends on the layout; only the number of m fetches does.
//
// Rows at or after first_recent (the start of the recent window, published
// per slice by the table kernel) are recent: TaR 0 and no K read. A tile can
// score both (TAR and VAN) or one of them; the library runs the two halves as
// separate launches, since the VaN half does not wait for the table.
template <typename T, int D>
struct SweepCfg {
  static constexpr int EPL = Lane<T>::EPL;
  static constexpr int LPR = D / EPL;
  static constexpr int GROUPS = 256 / LPR;
  static constexpr int U = 4;
};

// Where a launch's tiles are: work item w (after the XCD renumbering) is
// column block w % col_blocks of frame block (w / col_blocks) % frame_blocks
// of slice w / (col_blocks * frame_blocks); the divisions are magic-number
// multiplies, so a tile finds its place in a few scalar instructions.
struct TileGrid {
  FastDiv col_blocks, frame_blocks;
  uint32_t n_work;
  uint32_t blocks;  // tile blocks of the launch (a multiple of 8), the XCD renumbering's grid
};

// One tile: 256 threads (tid in [0, 256)), columns [colblock * GROUPS, +GROUPS),
// frames [f0, f0 + U). rec = the slice's first recent row. Row indices are
// 32-bit (a slice holds at most 65536 rows).
template <typename T, int D, bool TAR, bool VAN>
__device__ __forceinline__ void sweep_tile(const T* __restrict__ K, const T* __restrict__ V,
                                           const int32_t* __restrict__ patch_idx, int64_t S, uint32_t n, uint32_t p,
                                           const float* __restrict__ table, uint32_t rec, float* __restrict__ tar,
                                           float* __restrict__ van, uint32_t* err, uint32_t slice, uint32_t f0,
                                           uint32_t colblock, int tid) {
  using C = SweepCfg<T, D>;
  constexpr int EPL = C::EPL, LPR = C::LPR, GROUPS = C::GROUPS, U = C::U;
  const uint32_t col = colblock * GROUPS + tid / LPR;
  const int lane = tid % LPR;
  if (col >= p) return;  // the whole lane group idles: it is in no cross-lane sum
  const int64_t base = (int64_t)slice * S;
  if (!TAR) rec = n;
  const uint32_t past_end = min(n, rec);  // rows [0, past_end) are past (TaR); VaN scores rows [0, n)

  // Every load is a buffer load issued without a branch (a lane with nothing
  // to read uses an offset past the end and gets zeros); the patch ids of
  // the column's U rows come from one load per lane: lane l reads row l % 4,
  // and a DPP broadcast inside each quad hands row u's id to every lane.
  static_assert(U == 4 && LPR % 4 == 0, "patch-id broadcast over quads");
  constexpr uint32_t kSkip = 0xfffffff0u;
  constexpr uint32_t RB = D * (uint32_t)sizeof(T);
  const uint32_t lo = (uint32_t)lane * EPL * (uint32_t)sizeof(T);
  int32_t pq_mine = 0;
  if (TAR) {
    const __amdgpu_buffer_rsrc_t prs = buffer_rsrc(patch_idx + base, (uint32_t)(S * 4));
    const uint32_t xm = (f0 + (lane & 3)) * p + col;
    pq_mine = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(prs, xm < past_end ? xm * 4u : kSkip, 0, 0);
  }
  Raw16 kr[U], vr[U];
  const __amdgpu_buffer_rsrc_t krs = buffer_rsrc(K + base * D, (uint32_t)S * RB);
  const __amdgpu_buffer_rsrc_t vrs = buffer_rsrc(V + base * D, (uint32_t)S * RB);
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const uint32_t x = (f0 + u) * p + col;
    if (TAR) {
      // nontemporal: each past key is read once by the pass's scoring
      const auto k = __builtin_amdgcn_raw_buffer_load_b128(krs, x < past_end ? x * RB + lo : kSkip, 0, kNontemporal);
      kr[u].w[0] = k[0];
      kr[u].w[1] = k[1];
      kr[u].w[2] = k[2];
      kr[u].w[3] = k[3];
    }
    if (VAN) {
      const auto v = __builtin_amdgcn_raw_buffer_load_b128(vrs, x < n ? x * RB + lo : kSkip, 0, 0);
      vr[u].w[0] = v[0];
      vr[u].w[1] = v[1];
      vr[u].w[2] = v[2];
      vr[u].w[3] = v[3];
    }
  }
  // the m vector of the column's own position, fetched with the K loads
  float4 ms[EPL / 4];
  const bool any_past = TAR && f0 * p + col < past_end;
  if (TAR) {
    // the resource base must be uniform: the slice's table, lane offset in the offset
    const __amdgpu_buffer_rsrc_t mrs = buffer_rsrc(table + (int64_t)slice * p * D, p * D * 4u);
#pragma unroll
    for (int i = 0; i < EPL / 4; ++i) {
      const auto m = __builtin_amdgcn_raw_buffer_load_b128(
          mrs, any_past ? (col * D + lane * EPL + 4 * i) * 4u : kSkip, 0, 0);
      ms[i] = make_float4(__uint_as_float(m[0]), __uint_as_float(m[1]), __uint_as_float(m[2]),
                          __uint_as_float(m[3]));
    }
  }
  int32_t pq[U];
  if (TAR) {
    pq[0] = (int32_t)dpp_u32<0x00>((uint32_t)pq_mine);
    pq[1] = (int32_t)dpp_u32<0x55>((uint32_t)pq_mine);
    pq[2] = (int32_t)dpp_u32<0xAA>((uint32_t)pq_mine);
    pq[3] = (int32_t)dpp_u32<0xFF>((uint32_t)pq_mine);
  }
  // Each lane's partial sums of the U rows are reduce-scattered over the lane
  // group, so that a lane ends up with the totals of one row (scatter_row)
  // and the lanes that hold row u store it: one store instruction per wave.
  constexpr int Q = (LPR > 16 ? 16 : LPR) / 4;  // lanes per row after the scatter
  const int my_row = scatter_row<LPR>(lane);
  const uint32_t x_mine = (f0 + my_row) * p + col;
  const bool storer = lane < 16 && lane % Q == 0 && x_mine < n;
  if (VAN) {
    float part[U][1];
#pragma unroll
    for (int u = 0; u < U; ++u) part[u][0] = (f0 + u) * p + col < n ? Lane<T>::sumsq(vr[u]) : 0.f;
    float tot[1];
    reduce_scatter4<LPR, 1>(part, tot, lane);
    if (storer) van[base + x_mine] = fast_sqrt(tot[0]);
  }
  if (TAR) {
    float part[U][2];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t x = (f0 + u) * p + col;
      const bool past = x < past_end;
      const int32_t q = pq[u];
      const bool ok = past && q >= 0 && q < (int32_t)p;
      if (past && !ok && lane == 0) raise_error(err, 1u);
      float4 m[EPL / 4];
#pragma unroll
      for (int i = 0; i < EPL / 4; ++i) m[i] = ms[i];
      if (ok && q != (int32_t)col) {  // the row is not at its frame-plane position: exact lookup
        const float* mq = table + ((int64_t)slice * p + q) * D + lane * EPL;
#pragma unroll
        for (int i = 0; i < EPL / 4; ++i) m[i] = *reinterpret_cast<const float4*>(mq + 4 * i);
      }
      float dot = 0.f, kk = 0.f;
      if (ok) {
        float f[EPL];
        Lane<T>::decode(kr[u], f);
#pragma unroll
        for (int i = 0; i < EPL; i += 4) {
          const float4 mv = m[i / 4];
          dot += f[i] * mv.x + f[i + 1] * mv.y + f[i + 2] * mv.z + f[i + 3] * mv.w;
        }
        kk = Lane<T>::sumsq(kr[u]);
      }
      part[u][0] = dot;
      part[u][1] = kk;
    }
    float tot[2];
    reduce_scatter4<LPR, 2>(part, tot, lane);
    float sc = tot[1] != 0.f ? -(tot[0] * fast_rsqrt(tot[1])) : 0.f;  // a NaN key gives NaN, as in exact arithmetic
    if (sc == 0.f) sc = 0.f;  // -0.0 -> +0.0
    if (storer) tar[base + x_mine] = x_mine < past_end ? sc : 0.f;
  }
}

// The kernel arguments a tile needs, all read in the first round of scalar
// loads (an empty asm statement that takes them as operands keeps the
// compiler from spreading the loads over several dependent rounds).
#define IPV_ARGS_NOW(...) asm volatile("" ::__VA_ARGS__)

// grid: padded to a multiple of 8; work w = (slice * frame_blocks + frame block) * col_blocks + column block.
// sure_past: rows below it are past whatever the frame ids say (n - r * p:
// the window holds at most r frames of at most p rows), so a tile that ends
// there does not wait for the slice's window start.
template <typename T, int D, bool TAR, bool VAN>
__global__ __launch_bounds__(256) void k_score_sweep(const T* __restrict__ K, const T* __restrict__ V,
                                                     const int32_t* __restrict__ patch_idx, int64_t S, int32_t n,
                                                     int32_t p, const float* __restrict__ table,
                                                     const int32_t* __restrict__ first_recent,
                                                     float* __restrict__ tar, float* __restrict__ van,
                                                     uint32_t* err, TileGrid g, int32_t sure_past) {
  using C = SweepCfg<T, D>;
  IPV_ARGS_NOW("s"(K), "s"(V), "s"(patch_idx), "s"(S), "s"(n), "s"(p), "s"(table), "s"(first_recent), "s"(tar),
               "s"(van), "s"(g.col_blocks.m), "s"(g.frame_blocks.m), "s"(g.n_work), "s"(g.blocks), "s"(sure_past));
  const uint32_t logical = xcd_logical_id(blockIdx.x, g.blocks);
  if (logical >= g.n_work) return;
  const uint32_t tile = fast_div(logical, g.col_blocks);
  const uint32_t colblock = logical - tile * g.col_blocks.d;
  const uint32_t slice = fast_div(tile, g.frame_blocks);
  const uint32_t f0 = (tile - slice * g.frame_blocks.d) * C::U;
  const bool tail = (int64_t)(f0 + C::U) * p > sure_past;
  const uint32_t rec = TAR && tail ? (uint32_t)first_recent[slice] : (uint32_t)n;
  sweep_tile<T, D, TAR, VAN>(K, V, patch_idx, S, n, p, table, rec, tar, van, err, slice, f0, colblock, threadIdx.x);
}

// The recent-key table and the VaN half of the sweep in one launch. The VaN
// scores need no table, so their tiles can run while the table is built:
// blocks [0, table_padded) are table blocks (those at or past table_real
// return at once), dispatched first so that they all start together; the
// rest are VaN tiles, XCD-mapped like the sweep, which take the slots the
// table blocks leave and stream V meanwhile. The TaR half of the sweep reads
// the table, so it is the next launch. table_padded is a multiple of 8, so
// tile block i + table_padded runs on XCD i % 8.
template <typename T, int D>
__global__ __launch_bounds__(256) void k_table_van(const T* __restrict__ K, const T* __restrict__ V,
                                                   const int32_t* __restrict__ frame_idx,
                                                   const int32_t* __restrict__ patch_idx, int64_t S, int32_t n,
                                                   int32_t r, int32_t p, int32_t blocks_per_slice,
                                                   uint32_t table_padded, uint32_t table_real,
                                                   float* __restrict__ table, int32_t* __restrict__ first_recent,
                                                   uint32_t* err, uint32_t* __restrict__ zero, int32_t zero_per_slice,
                                                   float* __restrict__ van, TileGrid g) {
  extern __shared__ int32_t slot[];
  if (blockIdx.x < table_padded) {
    if (blockIdx.x < table_real)
      table_grid_block<T, D>(blockIdx.x, K, frame_idx, patch_idx, S, n, r, p, blocks_per_slice, table, first_recent,
                             err, zero, zero_per_slice, slot);
    return;
  }
  using C = SweepCfg<T, D>;
  IPV_ARGS_NOW("s"(V), "s"(S), "s"(n), "s"(p), "s"(van), "s"(g.col_blocks.m), "s"(g.frame_blocks.m),
               "s"(g.n_work), "s"(g.blocks));
  const uint32_t logical = xcd_logical_id(blockIdx.x - table_padded, g.blocks);
  if (logical >= g.n_work) return;
  const uint32_t tile = fast_div(logical, g.col_blocks);
  const uint32_t colblock = logical - tile * g.col_blocks.d;
  const uint32_t slice = fast_div(tile, g.frame_blocks);
  const uint32_t f0 = (tile - slice * g.frame_blocks.d) * C::U;
  sweep_tile<T, D, false, true>(K, V, patch_idx, S, n, p, table, n, nullptr, van, err, slice, f0, colblock,
                                threadIdx.x);
}

// ---------------------------------------------------------------- adaptive pooling
// The pooling kernels run kPoolThreads threads a workgroup (the CV also runs
// in 256-thread blocks beside the TaR tiles); a thread takes rows tid,
// tid + threads, ... and issues kPoolBatch of their loads at once (buffer
// loads: rows past n read as zero and are left out).
constexpr int kPoolThreads = 1024;
constexpr int kPoolBatch = 8;
constexpr int kPoolHeads = 4;  // the CV loads this many heads' rows at once

// Sum over the NT threads of a workgroup in a fixed order: a butterfly inside
// each wave, then the wave totals in wave order. Every thread gets the sum.
// red: one slot per wave, free again when this returns.
template <int NT>
__device__ __forceinline__ double pool_block_sum(double v, double* red) {
  constexpr int NW = NT / kWave;
#pragma unroll
  for (int off = kWave / 2; off >= 1; off /= 2) v += __shfl_xor(v, off);
  if (threadIdx.x % kWave == 0) red[threadIdx.x / kWave] = v;
  __syncthreads();
  double t = 0.0;
#pragma unroll
  for (int i = 0; i < NW; ++i) t += red[i];
  __syncthreads();
  return t;
}

// Per (stream, layer) bl: CV of all H * n VaN values in fp64, two passes
// (mean, then squared deviations), each a fixed-order reduction; window k
// from the thresholds, written to pool_ws[bl] (and pool_out[bl] if given).
// NT threads (tid in [0, NT)); red: NT / 64 doubles of LDS.
template <int NT>
__device__ __forceinline__ void pool_cv_block(const float* __restrict__ van, int64_t S, int32_t n, int32_t H,
                                              double tau1, double tau2, double tau3, int32_t* __restrict__ pool_ws,
                                              int32_t* __restrict__ pool_out, int64_t bl, int tid, double* red) {
  constexpr int U = kPoolBatch;
  const double count = (double)H * (double)n;
  // Pass `second`: the sum of the values, else of their squared deviations
  // from `mean`. Loads go out kPoolHeads heads x kPoolBatch rows at a time
  // (a missing head reads from an empty resource: zeros, left out).
  auto sweep = [&](bool second, double mean) -> double {
    double acc = 0.0;
    for (int32_t h0 = 0; h0 < H; h0 += kPoolHeads) {
      __amdgpu_buffer_rsrc_t rs[kPoolHeads];
#pragma unroll
      for (int g = 0; g < kPoolHeads; ++g)
        rs[g] = buffer_rsrc(van + (bl * H + min(h0 + g, H - 1)) * S, h0 + g < H ? (uint32_t)n * 4u : 0u);
      for (int32_t x0 = tid; x0 < n; x0 += NT * U) {
        float t[kPoolHeads][U];
#pragma unroll
        for (int g = 0; g < kPoolHeads; ++g)
#pragma unroll
          for (int u = 0; u < U; ++u)
            t[g][u] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs[g], (uint32_t)(x0 + u * NT) * 4u, 0, 0));
#pragma unroll
        for (int g = 0; g < kPoolHeads; ++g)
#pragma unroll
          for (int u = 0; u < U; ++u)
            if (h0 + g < H && x0 + u * NT < n) {
              const double d = second ? (double)t[g][u] - mean : (double)t[g][u];
              acc += second ? d * d : d;
            }
      }
    }
    return acc;
  };
  const double mean = pool_block_sum<NT>(sweep(false, 0.0), red) / count;
  const double v = sweep(true, mean);
  const double sd = sqrt(pool_block_sum<NT>(v, red) / count);
  if (tid == 0) {
    const double cv = mean == 0.0 ? 0.0 : sd / mean;
    const int32_t k = cv < tau1 ? 7 : cv < tau2 ? 5 : cv < tau3 ? 3 : 1;
    pool_ws[bl] = k;
    if (pool_out) pool_out[bl] = k;
  }
}

// One workgroup per (stream, layer).
__global__ __launch_bounds__(kPoolThreads) void k_pool_cv(const float* __restrict__ van, int64_t S, int32_t n,
                                                          int32_t H, double tau1, double tau2, double tau3,
                                                          int32_t* __restrict__ pool_ws,
                                                          int32_t* __restrict__ pool_out) {
  __shared__ double red[kPoolThreads / kWave];
  pool_cv_block<kPoolThreads>(van, S, n, H, tau1, tau2, tau3, pool_ws, pool_out, blockIdx.x, threadIdx.x, red);
}

// The k x k window mean is separable: every cell first gets the sum and count
// of the present cells (value >= 0) in its row of the window (hsum, hcnt),
// then a row adds those of the window's rows, top to bottom. Cells outside
// the grid are masked (a masked term adds exactly +0).
template <int HALF>
__device__ __forceinline__ void window_row(const float* cell, float* hsum, uint8_t* hcnt, int32_t c, int32_t p,
                                           int32_t grid_w, const FastDiv& pdiv, const FastDiv& wdiv) {
  const int32_t qq = c - (int32_t)fast_div((uint32_t)c, pdiv) * p;
  const int32_t cj = qq - (int32_t)fast_div((uint32_t)qq, wdiv) * grid_w, row0 = c - cj;
  float sum = 0.f;
  int cnt = 0;
#pragma unroll
  for (int dj = -HALF; dj <= HALF; ++dj) {
    const int32_t j = cj + dj;
    const bool inside = (uint32_t)j < (uint32_t)grid_w;
    const float v = cell[inside ? row0 + j : c];
    const bool use = inside && v >= 0.f;
    sum += use ? v : 0.f;
    cnt += use;
  }
  hsum[c] = sum;
  hcnt[c] = (uint8_t)cnt;
}

template <int HALF>
__device__ __forceinline__ float window_col(const float* hsum, const uint8_t* hcnt, int32_t fo, int32_t q, int32_t p,
                                            int32_t grid_h, int32_t grid_w, const FastDiv& wdiv) {
  const int32_t ci = (int32_t)fast_div((uint32_t)q, wdiv), c = fo * p + q;
  float sum = 0.f;
  int cnt = 0;
#pragma unroll
  for (int di = -HALF; di <= HALF; ++di) {
    const int32_t i = ci + di;
    const bool inside = (uint32_t)i < (uint32_t)grid_h;
    const int32_t at = inside ? c + di * grid_w : c;
    sum += inside ? hsum[at] : 0.f;
    cnt += inside ? hcnt[at] : 0;
  }
  return sum / (float)cnt;
}

// One workgroup per slice. Frames are handled FR at a time: their raw VaN
// values are scattered into an LDS grid (absent cells hold -1), then every
// row of those frames averages the present cells of its k x k window (the
// separable sums above) and overwrites its own score. Rows of later frames
// still hold raw values. Each round starts at the smallest frame id not yet
// covered, so the loop runs at most once per present frame whatever the ids
// are. Rows whose patch id is outside the grid keep their raw value. A
// thread's first kPoolBatch rows (all of them when n <= kPoolThreads *
// kPoolBatch) are loaded once and kept in registers for every pass; later
// rows are loaded again in each pass.
constexpr int kPoolCells = 8192;

__global__ __launch_bounds__(kPoolThreads) void k_pool_apply(float* __restrict__ van,
                                                             const int32_t* __restrict__ frame_idx,
                                                             const int32_t* __restrict__ patch_idx, int64_t S,
                                                             int32_t n, int32_t H, int32_t grid_h, int32_t grid_w,
                                                             const int32_t* __restrict__ pool_ws, FastDiv pdiv,
                                                             FastDiv wdiv) {
  constexpr int NT = kPoolThreads, U = kPoolBatch, NW = NT / kWave;
  __shared__ float cell[kPoolCells];
  __shared__ float hsum[kPoolCells];
  __shared__ uint8_t hcnt[kPoolCells];
  __shared__ int32_t wmin[NW];
  __shared__ int32_t slots;  // frame slots of the round that hold a row
  const int tid = threadIdx.x;
  const int64_t slice = blockIdx.x;
  const int32_t k = pool_ws[slice / H];
  if (k != 3 && k != 5 && k != 7) return;  // 1: no pooling
  const int32_t p = grid_h * grid_w, FR = kPoolCells / p;
  const int64_t base = slice * S;
  const __amdgpu_buffer_rsrc_t frs = buffer_rsrc(frame_idx + base, (uint32_t)n * 4u);
  const __amdgpu_buffer_rsrc_t prs = buffer_rsrc(patch_idx + base, (uint32_t)n * 4u);
  const __amdgpu_buffer_rsrc_t vrs = buffer_rsrc(van + base, (uint32_t)n * 4u);
  float* vcol = van + base;

  int32_t f0[U], q0[U];
  float v0[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const uint32_t off = (uint32_t)(tid + u * NT) * 4u;
    f0[u] = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(frs, off, 0, 0);
    q0[u] = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(prs, off, 0, 0);
    v0[u] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(vrs, off, 0, 0));
  }
  // rows x0 + u * NT of batch b (b == 0: the registers above); rows past n read as 0
  auto rows = [&](int32_t b, int32_t x0, int32_t (&f)[U], int32_t (&q)[U], float (&v)[U], bool need_v) {
    if (b == 0) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        f[u] = f0[u];
        q[u] = q0[u];
        v[u] = v0[u];
      }
      return;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t off = (uint32_t)(x0 + u * NT) * 4u;
      f[u] = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(frs, off, 0, 0);
      q[u] = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(prs, off, 0, 0);
      v[u] = need_v ? __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(vrs, off, 0, 0)) : 0.f;
    }
  };

  // the smallest frame id at or above `lower` (INT32_MAX: none); its barrier
  // also ends every thread's use of `cell` before the next round clears it
  auto next_start = [&](int64_t lower) -> int32_t {
    int32_t mine = INT32_MAX;
    for (int32_t b = 0, x0 = tid; x0 < n; ++b, x0 += NT * U) {
      int32_t f[U], q[U];
      float v[U];
      rows(b, x0, f, q, v, false);
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (x0 + u * NT < n && (int64_t)f[u] >= lower) mine = min(mine, f[u]);
    }
#pragma unroll
    for (int off = kWave / 2; off >= 1; off /= 2) mine = min(mine, __shfl_xor(mine, off));
    if (tid % kWave == 0) wmin[tid / kWave] = mine;
    __syncthreads();
    int32_t m = INT32_MAX;
#pragma unroll
    for (int i = 0; i < NW; ++i) m = min(m, wmin[i]);
    __syncthreads();
    return m;
  };

  for (int32_t fb = next_start(INT64_MIN); fb != INT32_MAX; fb = next_start((int64_t)fb + FR)) {
    for (int i = tid; i < FR * p; i += NT) cell[i] = -1.f;
    if (tid == 0) slots = 0;
    __syncthreads();
    int32_t top = 0;  // 1 + the highest slot this thread fills
    for (int32_t b = 0, x0 = tid; x0 < n; ++b, x0 += NT * U) {
      int32_t f[U], q[U];
      float v[U];
      rows(b, x0, f, q, v, true);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t fo = (int64_t)f[u] - fb;
        if (x0 + u * NT < n && fo >= 0 && fo < FR && q[u] >= 0 && q[u] < p) {
          cell[fo * p + q[u]] = v[u];
          top = max(top, (int32_t)fo + 1);
        }
      }
    }
#pragma unroll
    for (int off = kWave / 2; off >= 1; off /= 2) top = max(top, __shfl_xor(top, off));
    if (tid % kWave == 0) atomicMax(&slots, top);
    __syncthreads();
    // window rows of the filled slots only
    const int32_t cells = slots * p;
    for (int c = tid; c < cells; c += NT) {
      if (k == 7) window_row<3>(cell, hsum, hcnt, c, p, grid_w, pdiv, wdiv);
      else if (k == 5) window_row<2>(cell, hsum, hcnt, c, p, grid_w, pdiv, wdiv);
      else window_row<1>(cell, hsum, hcnt, c, p, grid_w, pdiv, wdiv);
    }
    __syncthreads();
    for (int32_t b = 0, x0 = tid; x0 < n; ++b, x0 += NT * U) {
      int32_t f[U], q[U];
      float v[U];
      rows(b, x0, f, q, v, false);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t fo = (int64_t)f[u] - fb;
        if (x0 + u * NT >= n || fo < 0 || fo >= FR || q[u] < 0 || q[u] >= p) continue;
        const int32_t slot = (int32_t)fo;
        vcol[x0 + u * NT] = k == 7   ? window_col<3>(hsum, hcnt, slot, q[u], p, grid_h, grid_w, wdiv)
                            : k == 5 ? window_col<2>(hsum, hcnt, slot, q[u], p, grid_h, grid_w, wdiv)
                                     : window_col<1>(hsum, hcnt, slot, q[u], p, grid_h, grid_w, wdiv);
      }
    }
  }
}

// ---------------------------------------------------------------- TaR tiles with the pooling CV
// The TaR half of the sweep with the CV of the layer-adaptive pooling beside
// it (the VaN scores are final after the previous launch): blocks
// [0, cv_padded) compute the CV of (stream, layer) blockIdx.x (those at or
// past cv_real return at once), the rest are TaR tiles as in k_score_sweep.
// cv_padded is a multiple of 8, so tile block i + cv_padded runs on XCD i % 8.
template <typename T, int D>
__global__ __launch_bounds__(256) void k_tar_sweep_cv(const T* __restrict__ K, const int32_t* __restrict__ patch_idx,
                                                      int64_t S, int32_t n, int32_t p, const float* __restrict__ table,
                                                      const int32_t* __restrict__ first_recent,
                                                      float* __restrict__ tar, uint32_t* err, TileGrid g,
                                                      int32_t sure_past, const float* __restrict__ van, int32_t H,
                                                      double tau1, double tau2, double tau3,
                                                      int32_t* __restrict__ pool_ws, uint32_t cv_padded,
                                                      uint32_t cv_real) {
  __shared__ double red[256 / kWave];
  if (blockIdx.x < cv_padded) {
    if (blockIdx.x < cv_real)
      pool_cv_block<256>(van, S, n, H, tau1, tau2, tau3, pool_ws, nullptr, blockIdx.x, threadIdx.x, red);
    return;
  }
  using C = SweepCfg<T, D>;
  const uint32_t logical = xcd_logical_id(blockIdx.x - cv_padded, g.blocks);
  if (logical >= g.n_work) return;
  const uint32_t tile = fast_div(logical, g.col_blocks);
  const uint32_t colblock = logical - tile * g.col_blocks.d;
  const uint32_t slice = fast_div(tile, g.frame_blocks);
  const uint32_t f0 = (tile - slice * g.frame_blocks.d) * C::U;
  const bool tail = (int64_t)(f0 + C::U) * p > sure_past;
  const uint32_t rec = tail ? (uint32_t)first_recent[slice] : (uint32_t)n;
  sweep_tile<T, D, true, false>(K, nullptr, patch_idx, S, n, p, table, rec, tar, nullptr, err, slice, f0, colblock,
                                threadIdx.x);
}

}  // namespace ipv
