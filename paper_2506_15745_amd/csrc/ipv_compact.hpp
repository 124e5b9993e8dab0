// In-place, order-preserving compaction (Sec. 3.1; Algorithm 1 step (5)):
// row j <- row keep[j] for j < C, for K, V, frame_idx and patch_idx.
//
// The rows of a slice form independent "walks": each column block of K (up
// to CBMAX bytes of every row), each of V, and the metadata pair. A walk's
// output rows are cut into chunks of CH rows and every chunk is one
// workgroup, so the whole copy runs
// in parallel. The in-place hazard: a chunk writes rows [c0, c1) that an
// earlier chunk of the same walk may still have to read (keep[j] >= j, so a
// chunk's sources lie at or after its own rows, never before). Hence:
//   1. workgroups are numbered chunk-major (all walks' chunk 0, then chunk 1,
//      ...), so every chunk a workgroup can depend on has a lower id;
//   2. a workgroup loads its source rows into registers, waits until they
//      have landed in every wave, and sets its chunk's "loaded" flag;
//   3. it waits for the flags of the earlier chunks of its walk whose
//      source range overlaps [c0, c1), then stores.
// Workgroups are dispatched in increasing id order (round-robin over the
// XCDs, in order within each), so the lowest unfinished workgroup is always
// resident and every chunk it waits for has already set its flag: the
// waits always end. A chunk's flag depends only on its own loads. The spin
// is bounded all the same; on expiry the chunk reports IPV_DEV_WAIT_TIMEOUT
// and does not store.
//
// The flags (one uint32 per chunk, in the workspace) must be zero when the
// kernel starts; k_clear_flags (or, in a full pass, the table kernel) zeroes
// them.
#pragma once

#include "ipv_device.hpp"

namespace ipv {

constexpr uint32_t kSpinLimit = 1u << 20;

// bytes per row, threads per chunk, rows per chunk, largest column block
template <int RB, int NT, int CHR, int CBMAX>
struct CompactCfg {
  static constexpr int CH = CHR;                      // rows per chunk
  static constexpr int CB = RB < CBMAX ? RB : CBMAX;  // bytes per column block
  static constexpr int NCB = RB / CB;                 // column blocks per row
  static constexpr int LPP = CB / 16;                 // lanes per row piece
  static constexpr int RPS = NT / LPP;                // rows per step
  static constexpr int U = CH / RPS;                  // steps per chunk
  static constexpr int MPT = 2 * CH / NT;             // metadata walk: 2 arrays x CH rows over NT threads
  static constexpr int PARTS = 2 * NCB + 1;           // walks per slice: K blocks, V blocks, metadata
  static_assert(U >= 1 && U * RPS == CH, "chunk shape");
  static_assert(MPT >= 1 && MPT * NT == 2 * CH && CH % kWave == 0, "metadata walk shape");
};

__device__ inline uint32_t load_flag(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ inline void store_flag(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Zero `count` words.
__global__ void k_clear_flags(uint32_t* flags, int64_t count) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) flags[i] = 0u;
}

// Chunk k of walk `part` of `slice` with NT threads. wflags: the walk's flags
// (one per chunk, zero at kernel start). ok_sh: one word of LDS.
template <int RB, int NT, int CHR, int CBMAX>
__device__ __forceinline__ void compact_chunk(char* __restrict__ K, char* __restrict__ V, int32_t* __restrict__ frame_idx,
                              int32_t* __restrict__ patch_idx, int64_t S, int32_t n, int32_t budget,
                              const int32_t* __restrict__ keep_idx, uint32_t* err, uint32_t* wflags,
                              int64_t slice, int part, uint32_t k, uint32_t* ok_sh) {
  using C = CompactCfg<RB, NT, CHR, CBMAX>;
  constexpr int LPP = C::LPP, RPS = C::RPS, U = C::U, CH = C::CH, MPT = C::MPT;
  const int tid = threadIdx.x;
  const int64_t c0 = (int64_t)k * CH;
  const int64_t c1 = min((int64_t)budget, c0 + CH);
  const int32_t* keep = keep_idx + slice * budget;
  const bool data = part < 2 * C::NCB;

  // 1. loads: first every keep index of the chunk, then every source row,
  // each batch issued at once. Buffer loads need no branches: a lane with
  // nothing to load reads past the end of the resource, which returns zeros
  // without touching memory.
  constexpr uint32_t kSkip = 0xfffffff0u;
  const __amdgpu_buffer_rsrc_t krs = buffer_rsrc(keep, (uint32_t)budget * 4u);
  Raw16 buf[U];
  int32_t src[U];
  int32_t mval[MPT], msrc[MPT];
  bool bad = false;
  char* base = nullptr;
  const int sub = tid / LPP, lane = tid % LPP;
  const uint32_t col = (uint32_t)((part % C::NCB) * C::CB + lane * 16);  // byte offset in a row
  if (data) {
    base = (part < C::NCB ? K : V) + slice * S * RB;
    const __amdgpu_buffer_rsrc_t drs = buffer_rsrc(base, (uint32_t)(S * RB));
    int32_t kj[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t j = c0 + u * RPS + sub;
      kj[u] = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(krs, j < c1 ? (uint32_t)j * 4u : kSkip, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t j = c0 + u * RPS + sub;
      const int32_t s = kj[u];
      const bool in = j < c1;
      bad |= in && (s < j || s >= n);
      src[u] = (in && s > j && s < n) ? s : -1;
      const auto v = __builtin_amdgcn_raw_buffer_load_b128(drs, src[u] >= 0 ? (uint32_t)src[u] * RB + col : kSkip, 0, 0);
      buf[u].w[0] = v[0];
      buf[u].w[1] = v[1];
      buf[u].w[2] = v[2];
      buf[u].w[3] = v[3];
    }
  } else {
    // element e = tid + i * NT: array e / CH (frame ids, patch ids), row e % CH;
    // CH is a multiple of the wave size, so the array is uniform per wave
    int32_t kj[MPT];
#pragma unroll
    for (int i = 0; i < MPT; ++i) {
      const int64_t j = c0 + (tid + i * NT) % CH;
      kj[i] = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(krs, j < c1 ? (uint32_t)j * 4u : kSkip, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < MPT; ++i) {
      const int e = __builtin_amdgcn_readfirstlane(tid + i * NT);
      const __amdgpu_buffer_rsrc_t mrs = buffer_rsrc((e < CH ? frame_idx : patch_idx) + slice * S, (uint32_t)(S * 4));
      const int64_t j = c0 + (tid + i * NT) % CH;
      const bool in = j < c1;
      const int32_t s = kj[i];
      bad |= in && (s < j || s >= n);
      msrc[i] = (in && s > j && s < n) ? s : -1;
      mval[i] = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(mrs, msrc[i] >= 0 ? (uint32_t)msrc[i] * 4u : kSkip, 0, 0);
    }
  }
  if (bad) raise_error(err, 8u);
  // Use every loaded register in an opaque statement: the compiler must wait
  // for each load's data here, before the barrier. After the barrier every
  // wave's loads of this chunk have landed.
#pragma unroll
  for (int u = 0; u < U; ++u) asm volatile("" ::"v"(buf[u].w[0]));
#pragma unroll
  for (int i = 0; i < MPT; ++i) asm volatile("" ::"v"(mval[i]));
  __syncthreads();

  // 2. publish
  if (tid == 0) store_flag(&wflags[k], 1u);

  // 3. wait for the earlier chunks of this walk that read rows in [c0, c1)
  if (tid < kWave) {
    bool ok = true;
    for (uint32_t j0 = 0; j0 < k && ok; j0 += kWave) {
      const uint32_t jc = j0 + tid;
      bool need = false;
      if (jc < k) {
        const int32_t lo = keep[(int64_t)jc * CH];
        const int32_t hi = keep[min((int64_t)budget, (int64_t)(jc + 1) * CH) - 1];
        need = hi >= c0 && lo < c1;
      }
      for (uint32_t spins = 0;; ++spins) {
        const bool pending = need && load_flag(&wflags[jc]) == 0u;
        if (__ballot(pending) == 0) break;
        if (spins >= kSpinLimit) {
          ok = false;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
    if (tid == 0) *ok_sh = ok;
  }
  __syncthreads();

  // 4. store
  if (*ok_sh) {
    if (data) {
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (src[u] >= 0) store16(base + (c0 + u * RPS + sub) * RB + col, buf[u]);
    } else {
#pragma unroll
      for (int i = 0; i < MPT; ++i) {
        const int e = tid + i * NT;
        if (msrc[i] >= 0) ((e < CH ? frame_idx : patch_idx) + slice * S)[c0 + e % CH] = mval[i];
      }
    }
  } else if (tid == 0) {
    raise_error(err, 32u);
  }
}

// grid: slices * PARTS * n_chunks workgroups of NT threads, id = chunk * walks + walk
template <int RB, int NT, int CHR, int CBMAX>
__global__ __launch_bounds__(NT) void k_compact(char* __restrict__ K, char* __restrict__ V,
                                                int32_t* __restrict__ frame_idx, int32_t* __restrict__ patch_idx,
                                                int64_t S, int32_t n, int32_t budget,
                                                const int32_t* __restrict__ keep_idx, uint32_t* err,
                                                uint32_t* flags, uint32_t n_chunks) {
  using C = CompactCfg<RB, NT, CHR, CBMAX>;
  __shared__ uint32_t ok_sh;
  const uint32_t walks = gridDim.x / n_chunks;
  const uint32_t k = blockIdx.x / walks, w = blockIdx.x % walks;
  compact_chunk<RB, NT, CHR, CBMAX>(K, V, frame_idx, patch_idx, S, n, budget, keep_idx, err, flags + (int64_t)w * n_chunks,
                        w / C::PARTS, (int)(w % C::PARTS), k, &ok_sh);
}

}  // namespace ipv
