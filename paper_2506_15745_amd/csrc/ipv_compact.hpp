// In-place, order-preserving compaction (Sec. 3.1; Algorithm 1 step (5)):
// row j <- row keep[j] for j < C, for K, V, frame_idx and patch_idx.
//
// The rows of a slice form independent "walks": each column block of K (up
// to CBMAX bytes of every row), each of V, and the metadata pair. A walk's
// output rows are cut into chunks of CH rows and every chunk is one
// workgroup, so the whole copy runs in parallel. The in-place hazard: a chunk
// writes rows [c0, c1) that an earlier chunk of the same walk may still have
// to read (keep is strictly ascending, so keep[j] >= j: a chunk's sources lie
// at or after its own rows, never before). Hence:
//   1. a workgroup draws its chunk number from a ticket counter of its walk,
//      so every lower chunk of the walk belongs to a workgroup that is
//      already running, whatever order the hardware dispatches them in;
//   2. it loads its source rows into registers, waits until they have landed
//      in every wave, and sets its chunk's "loaded" flag;
//   3. it waits for the flags of the earlier chunks of its walk whose source
//      range overlaps [c0, c1), then stores.
// A chunk's flag depends only on its own loads, and every chunk it waits for
// holds a slot and sets its flag without waiting itself, so the waits end.
// The spin is bounded all the same (a workspace shared by overlapping calls
// breaks the counters); on expiry the chunk reports IPV_DEV_WAIT_TIMEOUT and
// does not store.
//
// Workgroups are numbered chunk-major (all walks' chunk 0, then chunk 1, ...),
// and workgroup id / walks is the chunk a workgroup draws when the dispatcher
// starts them in id order, as it does: the loads of that chunk are issued
// together with the ticket draw and kept if the ticket matches, so the draw
// adds no latency; a workgroup that draws another chunk loads that one.
//
// The wait rule needs each chunk's source rows to lie between its first and
// last keep entries, i.e. keep strictly ascending. A chunk that finds a keep
// entry outside [j, n) or not above the one before reports IPV_DEV_BAD_KEEP
// and stores nothing.
//
// Per walk the workspace holds one flag per chunk and then the ticket
// counter, all zero when the kernel starts; k_clear_flags (or, in a full
// pass, the first kernel: the table or prev-row launch, or the Uniform Select
// selection) zeroes them.
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
  static constexpr int NW = NT / kWave;
  static_assert(U >= 1 && U * RPS == CH, "chunk shape");
  static_assert(MPT >= 1 && MPT * NT == 2 * CH && CH % kWave == 0, "metadata walk shape");
  static_assert(CH <= NT, "one thread per row checks the keep order");
};

// Words of one walk's workspace: a flag per chunk, then the ticket counter.
__host__ __device__ inline int64_t walk_words(int64_t n_chunks) { return n_chunks + 1; }

template <int NT, int CHR>
struct CompactShared {
  int32_t keep[CHR + 1];  // keep[c0 - 1] (or -1), then the chunk's keep entries
  uint32_t wave_bad[NT / kWave];
  uint32_t ticket;
  uint32_t ok;
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

// Walk `part` of `slice` with NT threads; wflags: the walk's n_chunks flags,
// then its ticket counter. kexp: the chunk this workgroup draws when
// workgroups start in id order.
template <int RB, int NT, int CHR, int CBMAX>
__device__ __forceinline__ void compact_walk(char* __restrict__ K, char* __restrict__ V,
                                             int32_t* __restrict__ frame_idx, int32_t* __restrict__ patch_idx,
                                             int64_t S, int32_t n, int32_t budget,
                                             const int32_t* __restrict__ keep_idx, uint32_t* err, uint32_t* wflags,
                                             uint32_t n_chunks, int64_t slice, int part, uint32_t kexp,
                                             CompactShared<NT, CHR>& sh) {
  using C = CompactCfg<RB, NT, CHR, CBMAX>;
  constexpr int LPP = C::LPP, RPS = C::RPS, U = C::U, CH = C::CH, MPT = C::MPT;
  const int tid = threadIdx.x, wave = tid / kWave;
  const int32_t* keep = keep_idx + slice * budget;
  const bool data = part < 2 * C::NCB;

  // the ticket: drawn first, so its round trip overlaps the loads below
  uint32_t drawn = 0;
  if (tid == 0) drawn = atomicAdd(&wflags[n_chunks], 1u);

  // Loads of chunk k: first every keep index of the chunk, then every source
  // row, each batch issued at once. Buffer loads need no branches: a lane with
  // nothing to load reads past the end of the resource, which returns zeros
  // without touching memory. Only keep entries in (j, n) are followed (j:
  // nothing to move); the order check comes after the first barrier.
  constexpr uint32_t kSkip = 0xfffffff0u;
  const __amdgpu_buffer_rsrc_t krs = buffer_rsrc(keep, (uint32_t)budget * 4u);
  Raw16 buf[U];
  int32_t src[U];
  int32_t mval[MPT], msrc[MPT];
  char* base = nullptr;
  const int sub = tid / LPP, lane = tid % LPP;
  const uint32_t col = (uint32_t)((part % C::NCB) * C::CB + lane * 16);  // byte offset in a row
  auto load_chunk = [&](uint32_t k) {
    const int64_t c0 = (int64_t)k * CH;
    const int64_t c1 = min((int64_t)budget, c0 + CH);
    if (tid == 0) {
      const int32_t before = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(
          krs, c0 > 0 ? (uint32_t)(c0 - 1) * 4u : kSkip, 0, 0);
      sh.keep[0] = c0 > 0 ? before : -1;
    }
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
        src[u] = (j < c1 && s > j && s < n) ? s : -1;
        // nontemporal: the pass reads each kept row once here and not again
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(drs, src[u] >= 0 ? (uint32_t)src[u] * RB + col : kSkip,
                                                             0, kNontemporal);
        buf[u].w[0] = v[0];
        buf[u].w[1] = v[1];
        buf[u].w[2] = v[2];
        buf[u].w[3] = v[3];
        if (lane == 0) sh.keep[1 + u * RPS + sub] = s;
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
        const __amdgpu_buffer_rsrc_t mrs =
            buffer_rsrc((e < CH ? frame_idx : patch_idx) + slice * S, (uint32_t)(S * 4));
        const int64_t j = c0 + (tid + i * NT) % CH;
        const int32_t s = kj[i];
        msrc[i] = (j < c1 && s > j && s < n) ? s : -1;
        mval[i] =
            (int32_t)__builtin_amdgcn_raw_buffer_load_b32(mrs, msrc[i] >= 0 ? (uint32_t)msrc[i] * 4u : kSkip, 0, 0);
        if (tid + i * NT < CH) sh.keep[1 + tid + i * NT] = s;
      }
    }
    // Use every loaded register in an opaque statement: the compiler must
    // wait for each load's data here, before the barrier that follows. After
    // that barrier every wave's loads of this chunk have landed.
#pragma unroll
    for (int u = 0; u < U; ++u) asm volatile("" ::"v"(buf[u].w[0]));
#pragma unroll
    for (int i = 0; i < MPT; ++i) asm volatile("" ::"v"(mval[i]));
  };

  load_chunk(kexp);
  if (tid == 0) sh.ticket = drawn;
  __syncthreads();
  const uint32_t k = sh.ticket;
  if (k >= n_chunks) {  // the counter was not zero: a workspace shared by overlapping calls
    if (tid == 0) raise_error(err, 32u);
    return;
  }
  if (k != kexp) {  // uniform: this workgroup drew another chunk than its id suggests
    load_chunk(k);
    __syncthreads();
  }
  const int64_t c0 = (int64_t)k * CH;
  const int64_t c1 = min((int64_t)budget, c0 + CH);

  // 2. the keep order of this chunk: row c0 + tid against the row before it
  {
    const int64_t j = c0 + tid;
    bool bad = false;
    if (tid < CH && j < c1) {
      const int32_t s = sh.keep[1 + tid], before = sh.keep[tid];
      bad = s < j || s >= n || s <= before;
    }
    const bool wbad = __ballot(bad) != 0;
    if (tid % kWave == 0) sh.wave_bad[wave] = wbad;
  }

  // 3. publish, then wait for the earlier chunks of this walk that read rows in [c0, c1)
  if (tid == 0) store_flag(&wflags[k], 1u);
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
    if (tid == 0) sh.ok = ok;
  }
  __syncthreads();
  bool any_bad = false;
#pragma unroll
  for (int i = 0; i < CH / kWave; ++i) any_bad |= sh.wave_bad[i] != 0;

  // 4. store
  if (sh.ok && !any_bad) {
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
    raise_error(err, any_bad ? 8u : 32u);
  }
}

// grid: slices * PARTS * n_chunks workgroups of NT threads; walk = id % walks,
// expected chunk = id / walks (walks: a magic-number divisor from the host).
// flags: walk_words(n_chunks) words per walk.
template <int RB, int NT, int CHR, int CBMAX>
__global__ __launch_bounds__(NT) void k_compact(char* __restrict__ K, char* __restrict__ V,
                                                int32_t* __restrict__ frame_idx, int32_t* __restrict__ patch_idx,
                                                int64_t S, int32_t n, int32_t budget,
                                                const int32_t* __restrict__ keep_idx, uint32_t* err,
                                                uint32_t* flags, uint32_t n_chunks, FastDiv walks) {
  using C = CompactCfg<RB, NT, CHR, CBMAX>;
  __shared__ CompactShared<NT, CHR> sh;
  // every argument in the first round of scalar loads
  asm volatile("" ::"s"(K), "s"(V), "s"(frame_idx), "s"(patch_idx), "s"(S), "s"(n), "s"(budget), "s"(keep_idx),
               "s"(err), "s"(flags), "s"(n_chunks), "s"(walks.d), "s"(walks.m), "s"(walks.s2));
  const uint32_t kexp = fast_div(blockIdx.x, walks), w = blockIdx.x - kexp * walks.d;
  compact_walk<RB, NT, CHR, CBMAX>(K, V, frame_idx, patch_idx, S, n, budget, keep_idx, err,
                                   flags + (int64_t)w * walk_words(n_chunks), n_chunks, w / C::PARTS,
                                   (int)(w % C::PARTS), kexp, sh);
}

}  // namespace ipv
