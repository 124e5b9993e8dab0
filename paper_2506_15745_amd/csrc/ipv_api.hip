// C ABI of the compression pass: argument validation, workspace layout and
// kernel launches. Every check that the host can make happens before the
// first launch, so a rejected call enqueues nothing and touches no buffer.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <mutex>
#include <vector>

#include "../../include/ipv.h"
#include "ipv_adjacent.hpp"
#include "ipv_compact.hpp"
#include "ipv_scores.hpp"
#include "ipv_select.hpp"

using namespace ipv;

#define IPV_TRY(x)               \
  do {                           \
    const ipv_status _s = (x);   \
    if (_s != IPV_OK) return _s; \
  } while (0)

namespace {

constexpr int32_t kMaxRows = 65536;  // select: 1024 threads x 64 row flags
constexpr int64_t kMaxWindowRows = 65536;        // r * p: recent rows scanned per table block
constexpr int32_t kMaxRecentFrames = 256;
static_assert(kPrevMaxPositions >= kPoolCells, "the prev-row walk holds one entry per patch position");
constexpr int kCompactThreads = 1024;
constexpr int kCompactRows = 512;      // rows per compaction chunk
constexpr int kCompactColBytes = 256;  // largest column block a compaction walk copies

struct Dims {
  int64_t B, L, H, S, D, p, slices;
  int32_t gh, gw, dtype;
  int64_t elem;  // bytes per element
};

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

ipv_status check_shape(const ipv_shape* s, Dims* d) {
  if (!s) return IPV_ERR_NULL;
  if (s->dtype != IPV_BF16 && s->dtype != IPV_F32) return IPV_ERR_DTYPE;
  if (s->streams < 1 || s->layers < 1 || s->kv_heads < 1 || s->capacity < 1 || s->grid_h < 1 || s->grid_w < 1)
    return IPV_ERR_SHAPE;
  if (s->head_dim != 32 && s->head_dim != 64 && s->head_dim != 128 && s->head_dim != 256) return IPV_ERR_SHAPE;
  const int64_t p = (int64_t)s->grid_h * s->grid_w;
  if (p > kPoolCells) return IPV_ERR_SHAPE;
  d->B = s->streams;
  d->L = s->layers;
  d->H = s->kv_heads;
  d->S = s->capacity;
  d->D = s->head_dim;
  d->p = p;
  d->slices = d->B * d->L * d->H;
  d->gh = s->grid_h;
  d->gw = s->grid_w;
  d->dtype = s->dtype;
  d->elem = s->dtype == IPV_BF16 ? 2 : 4;
  if (d->slices > (int64_t)INT32_MAX / 8) return IPV_ERR_SHAPE;
  // buffer loads address one slice's rows with 32-bit byte offsets
  if (d->S * d->D * d->elem > (int64_t)UINT32_MAX - 16) return IPV_ERR_SHAPE;
  return IPV_OK;
}

ipv_status check_mode(uint32_t mode) { return (mode & ~(uint32_t)IPV_MODE_ALL) ? IPV_ERR_ARG : IPV_OK; }

// Uniform Select decides from frame ids: no score buffers are read or written
bool scores_needed(uint32_t mode) { return (mode & IPV_UNIFORM_SELECT) == 0; }

ipv_status check_rows(const Dims& d, int32_t n) {
  if (n < 1 || n > d.S || n > kMaxRows) return IPV_ERR_SHAPE;
  return IPV_OK;
}

ipv_status check_recent(const Dims& d, int32_t r) {
  if (r < 1 || r > kMaxRecentFrames) return IPV_ERR_ARG;
  if ((int64_t)r * d.p > kMaxWindowRows) return IPV_ERR_ARG;
  return IPV_OK;
}

// A pass keeps budget rows of n: 1 <= budget <= n. Whether the budget also
// holds the recent window |R| depends on the frame ids, which only the device
// reads: the selection reports a larger window (IPV_DEV_RECENT_OVER).
ipv_status check_budget(int32_t n, int32_t budget) {
  return (budget < 1 || budget > n) ? IPV_ERR_BUDGET : IPV_OK;
}

// The continual-compression loop runs many passes without reading the device
// between them, so it asks for a budget that holds any window the cache can
// have: |R| <= min(n, r * p) (a frame holds each patch position at most once).
ipv_status check_loop_budget(const Dims& d, int32_t n, int32_t budget, int32_t r) {
  IPV_TRY(check_budget(n, budget));
  return budget < std::min<int64_t>(n, (int64_t)r * d.p) ? IPV_ERR_BUDGET : IPV_OK;
}

// ------------------------------------------------------------ workspace layout
// [0, 256)                 device error word (uint32) + padding
// table  slices * p * D    fp32 m_q vectors of the recent window; in the
//                          consecutive-frame TaR mode the same region holds
//                          prev(x) per row instead (slices * S int32)
// first  slices            int32 first recent row of each slice
// pool   B * L             int32 pooling window per (stream, layer)
// flags  walks * (chunks+1) per compaction walk: a uint32 per chunk (1 once its
//                          rows are loaded), then the walk's ticket counter
size_t up256(size_t x) { return (x + 255) / 256 * 256; }
int64_t compact_parts(const Dims& d) { return 2 * std::max<int64_t>(1, d.D * d.elem / kCompactColBytes) + 1; }
int64_t max_chunks(const Dims& d) { return (d.S + kCompactRows - 1) / kCompactRows; }
size_t table_offset() { return kWsHeader; }
size_t table_bytes(const Dims& d) {
  return std::max((size_t)(d.slices * d.p * d.D) * sizeof(float), (size_t)(d.slices * d.S) * sizeof(int32_t));
}
size_t first_offset(const Dims& d) { return up256(table_offset() + table_bytes(d)); }
size_t pool_offset(const Dims& d) { return up256(first_offset(d) + (size_t)d.slices * sizeof(int32_t)); }
size_t flags_offset(const Dims& d) { return up256(pool_offset(d) + (size_t)(d.B * d.L) * sizeof(int32_t)); }
size_t ws_total(const Dims& d) {
  return up256(flags_offset(d) + (size_t)(d.slices * compact_parts(d) * walk_words(max_chunks(d))) * sizeof(uint32_t));
}

ipv_status check_ws(const Dims& d, const void* ws, size_t ws_bytes) {
  if (!ws) return IPV_ERR_WORKSPACE;
  if (!aligned(ws, 256)) return IPV_ERR_ALIGN;
  if (ws_bytes < ws_total(d)) return IPV_ERR_WORKSPACE;
  return IPV_OK;
}

uint32_t* err_word(void* ws) { return reinterpret_cast<uint32_t*>(ws); }
float* ws_table(void* ws) { return reinterpret_cast<float*>(static_cast<char*>(ws) + table_offset()); }
int32_t* ws_prev(void* ws) { return reinterpret_cast<int32_t*>(static_cast<char*>(ws) + table_offset()); }
int32_t* ws_first(void* ws, const Dims& d) {
  return reinterpret_cast<int32_t*>(static_cast<char*>(ws) + first_offset(d));
}
uint32_t* ws_flags(void* ws, const Dims& d) {
  return reinterpret_cast<uint32_t*>(static_cast<char*>(ws) + flags_offset(d));
}
int32_t* ws_pool(void* ws, const Dims& d) {
  return reinterpret_cast<int32_t*>(static_cast<char*>(ws) + pool_offset(d));
}

ipv_status launched() { return hipGetLastError() == hipSuccess ? IPV_OK : IPV_ERR_HIP; }

// blocks: the launch's tile blocks (after any blocks of another role that come first)
TileGrid tile_grid(int32_t col_blocks, int32_t frame_blocks, uint32_t work, uint32_t blocks) {
  return TileGrid{make_fastdiv((uint32_t)col_blocks), make_fastdiv((uint32_t)frame_blocks), work, blocks};
}

uint32_t pad8(uint32_t x) { return (x + 7u) / 8u * 8u; }

// ------------------------------------------------------------ launchers
ipv_status no_mark() { return IPV_OK; }

// K == nullptr: VaN only; V == nullptr: TaR only. With both, the first launch
// builds what TaR needs (the recent-key table, or in the consecutive-frame
// mode the prev rows) with the VaN tiles beside it, and the second scores
// TaR. between(): runs after the first launch (the table, the prev rows, or
// nothing for VaN only), before the sweep that follows.
// zero_chunks > 0: the first kernel also zeroes the compaction flags for a
// compaction of zero_chunks chunks per walk that follows in the same pass.
// adjacent: consecutive-frame TaR (IPV_TAR_ADJACENT)
// cv_tau (may be null): with both scores and the recent-key table, the TaR
// launch also computes the pooling CV and window of every (stream, layer)
// (k_pool_apply must follow); ignored otherwise.
template <typename T, int D, typename Between>
ipv_status run_scores(const Dims& d, const void* K, const void* V, const int32_t* fr, const int32_t* pa, int32_t n,
                      int32_t r, float* tar, float* van, void* ws, hipStream_t st, Between between,
                      int64_t zero_chunks, bool adjacent, const double* cv_tau) {
  const bool do_tar = K != nullptr, do_van = V != nullptr;
  uint32_t* zero = zero_chunks > 0 ? ws_flags(ws, d) : nullptr;
  const int32_t zero_per_slice = (int32_t)(compact_parts(d) * walk_words(zero_chunks));
  if (do_tar && adjacent) {
    if (do_van) {
      // prev-row walks and VaN tiles in one launch
      using C = SweepCfg<T, D>;
      const int32_t col_blocks = (int32_t)((d.p + C::GROUPS - 1) / C::GROUPS);
      const int32_t frame_blocks = (int32_t)(((n + d.p - 1) / d.p + C::U - 1) / C::U);
      const uint32_t work = (uint32_t)(d.slices * frame_blocks * col_blocks);
      const uint32_t prev_padded = pad8((uint32_t)d.slices);
      k_prev_van<T, D><<<dim3(prev_padded + pad8((work + 3) / 4)), dim3(kPrevThreads), 0, st>>>(
          static_cast<const T*>(V), fr, pa, d.S, n, r, (int32_t)d.p, ws_prev(ws), ws_first(ws, d), err_word(ws),
          zero, zero_per_slice, prev_padded, (uint32_t)d.slices, van,
          tile_grid(col_blocks, frame_blocks, work, pad8((work + 3) / 4)));
    } else {
      k_prev_rows<<<dim3((uint32_t)d.slices), dim3(kPrevThreads), 0, st>>>(
          fr, pa, d.S, n, r, (int32_t)d.p, ws_prev(ws), ws_first(ws, d), err_word(ws), zero, zero_per_slice);
    }
    IPV_TRY(between());
    // then the TaR rows
    constexpr int ROWS = 256 / (D / Lane<T>::EPL) * 4;
    const int32_t bps = (n + ROWS - 1) / ROWS;
    const uint32_t work = (uint32_t)(d.slices * bps);
    k_adjacent_sweep<T, D><<<dim3(pad8(work)), dim3(256), 0, st>>>(static_cast<const T*>(K), ws_prev(ws), d.S, n,
                                                                   ws_first(ws, d), tar, bps, work);
    return launched();
  }
  constexpr int GROUPS = 256 / (D / Lane<T>::EPL);
  const int32_t blocks = (int32_t)((d.p + GROUPS - 1) / GROUPS);
  const size_t lds = (size_t)GROUPS * r * sizeof(int32_t);
  const uint32_t table_real = (uint32_t)(d.slices * blocks);
  using C = SweepCfg<T, D>;
  const int32_t col_blocks = (int32_t)((d.p + C::GROUPS - 1) / C::GROUPS);
  const int32_t frame_blocks = (int32_t)(((n + d.p - 1) / d.p + C::U - 1) / C::U);
  const uint32_t work = (uint32_t)(d.slices * frame_blocks * col_blocks);
  const dim3 grid(pad8(work)), block(256);
  const T* k = static_cast<const T*>(K);
  const T* v = static_cast<const T*>(V);
  int32_t* first = ws_first(ws, d);
  // rows certainly before the recent window (it holds at most r * p rows)
  const int32_t sure_past = (int32_t)std::max<int64_t>(0, (int64_t)n - (int64_t)r * d.p);
  if (do_tar && do_van) {
    // table and VaN tiles in one launch, then the TaR tiles
    const uint32_t table_padded = pad8(table_real);
    k_table_van<T, D><<<dim3(table_padded + pad8(work)), block, lds, st>>>(
        k, v, fr, pa, d.S, n, r, (int32_t)d.p, blocks, table_padded, table_real, ws_table(ws), first, err_word(ws),
        zero, zero_per_slice, van, tile_grid(col_blocks, frame_blocks, work, pad8(work)));
    IPV_TRY(between());
    if (cv_tau) {
      const uint32_t cv_real = (uint32_t)(d.B * d.L), cv_padded = pad8(cv_real);
      k_tar_sweep_cv<T, D><<<dim3(cv_padded + pad8(work)), block, 0, st>>>(
          k, pa, d.S, n, (int32_t)d.p, ws_table(ws), first, tar, err_word(ws),
          tile_grid(col_blocks, frame_blocks, work, pad8(work)), sure_past, van, (int32_t)d.H, cv_tau[0], cv_tau[1],
          cv_tau[2], ws_pool(ws, d), cv_padded, cv_real);
      return launched();
    }
    k_score_sweep<T, D, true, false><<<grid, block, 0, st>>>(k, v, pa, d.S, n, (int32_t)d.p, ws_table(ws), first,
                                                             tar, van, err_word(ws),
                                                             tile_grid(col_blocks, frame_blocks, work, pad8(work)), sure_past);
    return launched();
  }
  if (do_tar)
    k_recent_table<T, D><<<dim3(table_real), block, lds, st>>>(k, fr, pa, d.S, n, r, (int32_t)d.p, blocks,
                                                               ws_table(ws), first, err_word(ws), zero,
                                                               zero_per_slice);
  IPV_TRY(between());
  if (do_tar)
    k_score_sweep<T, D, true, false><<<grid, block, 0, st>>>(k, v, pa, d.S, n, (int32_t)d.p, ws_table(ws), first,
                                                             tar, van, err_word(ws),
                                                             tile_grid(col_blocks, frame_blocks, work, pad8(work)), sure_past);
  else
    k_score_sweep<T, D, false, true><<<grid, block, 0, st>>>(k, v, pa, d.S, n, (int32_t)d.p, ws_table(ws), first,
                                                             tar, van, err_word(ws),
                                                             tile_grid(col_blocks, frame_blocks, work, pad8(work)), n);
  return launched();
}

template <typename Between = ipv_status (*)()>
ipv_status scores(const Dims& d, const void* K, const void* V, const int32_t* fr, const int32_t* pa, int32_t n,
                  int32_t r, float* tar, float* van, void* ws, hipStream_t st, Between between = no_mark,
                  int64_t zero_chunks = 0, bool adjacent = false, const double* cv_tau = nullptr) {
#define IPV_SCORES(T, DD)                                                                                        \
  if (d.D == DD)                                                                                                 \
    return run_scores<T, DD>(d, K, V, fr, pa, n, r, tar, van, ws, st, between, zero_chunks, adjacent, cv_tau);
  if (d.dtype == IPV_BF16) {
    IPV_SCORES(uint16_t, 32) IPV_SCORES(uint16_t, 64) IPV_SCORES(uint16_t, 128) IPV_SCORES(uint16_t, 256)
  } else {
    IPV_SCORES(float, 32) IPV_SCORES(float, 64) IPV_SCORES(float, 128) IPV_SCORES(float, 256)
  }
#undef IPV_SCORES
  return IPV_ERR_SHAPE;
}

// cv_done: the TaR launch has computed the windows already (k_tar_sweep_cv)
ipv_status pool_d(const Dims& d, const double* tau, float* van, const int32_t* fr, const int32_t* pa, int32_t n,
                  int32_t* pool_out, void* ws, hipStream_t st, bool cv_done = false) {
  if (!cv_done)
    k_pool_cv<<<dim3((uint32_t)(d.B * d.L)), dim3(kPoolThreads), 0, st>>>(van, d.S, n, (int32_t)d.H, tau[0], tau[1],
                                                                          tau[2], ws_pool(ws, d), pool_out);
  k_pool_apply<<<dim3((uint32_t)d.slices), dim3(kPoolThreads), 0, st>>>(
      van, fr, pa, d.S, n, (int32_t)d.H, d.gh, d.gw, ws_pool(ws, d), make_fastdiv((uint32_t)d.p),
      make_fastdiv((uint32_t)d.gw));
  return launched();
}

__global__ void k_fill_i32(int32_t* p, int64_t count, int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) p[i] = v;
}

constexpr int kSelThreads = 1024;  // most threads of a selection workgroup
constexpr int64_t kComputeUnits = 256;  // MI355X

// Threads of a selection workgroup: whole waves for the n rows at RPT rows a
// thread, at most kSelThreads (the caller picks RPT >= n / kSelThreads).
uint32_t sel_threads(int32_t n, int RPT) {
  const int32_t t = (n + RPT - 1) / RPT;
  return (uint32_t)std::min(kSelThreads, (t + 63) / 64 * 64);
}

// mode: the reverse bits complement a stage's keys; IPV_HEAD_SHARED gives one
// block (and one keep set) to each (stream, layer)
template <int RPT>
ipv_status run_select(const Dims& d, const float* tar, const float* van, const int32_t* fr, int32_t n, int32_t budget,
                      int32_t tar_total, int32_t r, int32_t* keep, uint32_t* err, hipStream_t st, uint32_t mode) {
  const int32_t heads = (mode & IPV_HEAD_SHARED) ? (int32_t)d.H : 1;
  const uint32_t tflip = (mode & IPV_TAR_REVERSE) ? 0xffffffffu : 0u;
  const uint32_t vflip = (mode & IPV_VAN_REVERSE) ? 0xffffffffu : 0u;
  const dim3 grid((uint32_t)(d.slices / heads)), block(sel_threads(n, RPT));
  // 16-byte row-run loads need every slice to start 16-byte aligned
  if (d.S % 4 == 0)
    k_select<kSelThreads, RPT, true><<<grid, block, 0, st>>>(tar, van, fr, d.S, n, budget, tar_total, r, keep, err,
                                                             heads, tflip, vflip);
  else
    k_select<kSelThreads, RPT, false><<<grid, block, 0, st>>>(tar, van, fr, d.S, n, budget, tar_total, r, keep, err,
                                                              heads, tflip, vflip);
  return launched();
}

// Uniform Select: one block per slice, or per (stream, layer) with
// IPV_HEAD_SHARED. zero (may be null): the blocks also zero zero_per_slice
// words per slice there (the compaction flags of the pass).
template <int RPT>
ipv_status run_uniform(const Dims& d, const int32_t* fr, int32_t n, int32_t budget, int32_t r, int32_t* keep,
                       uint32_t* err, hipStream_t st, uint32_t mode, uint32_t* zero, int32_t zero_per_slice) {
  const int32_t heads = (mode & IPV_HEAD_SHARED) ? (int32_t)d.H : 1;
  const dim3 grid((uint32_t)(d.slices / heads)), block(sel_threads(n, RPT));
  if (d.S % 4 == 0)
    k_select_uniform<kSelThreads, RPT, true><<<grid, block, 0, st>>>(fr, d.S, n, budget, r, keep, err, heads, zero,
                                                                     zero_per_slice);
  else
    k_select_uniform<kSelThreads, RPT, false><<<grid, block, 0, st>>>(fr, d.S, n, budget, r, keep, err, heads, zero,
                                                                      zero_per_slice);
  return launched();
}

// zero / zero_per_slice: as for run_uniform (used by Uniform Select only)
ipv_status select(const Dims& d, const float* tar, const float* van, const int32_t* fr, int32_t n, int32_t budget,
                  int32_t tar_total, int32_t r, int32_t* keep, uint32_t* err, hipStream_t st, uint32_t mode,
                  uint32_t* zero = nullptr, int32_t zero_per_slice = 0) {
  const int32_t rpt = (n + kSelThreads - 1) / kSelThreads;
  // A block of up to 8 rows a thread (832 threads for 6272 rows) holds a CU
  // alone; with more blocks than CUs, 16 rows a thread (half the threads)
  // lets three blocks share a CU, which ends sooner although each block takes
  // longer (16-stream 7B-class batch: 65 against 93 us).
  const int64_t groups = d.slices / ((mode & IPV_HEAD_SHARED) ? d.H : 1);
  const bool many = groups > kComputeUnits && rpt <= 8;
  if (mode & IPV_UNIFORM_SELECT) {
    if (many) return run_uniform<16>(d, fr, n, budget, r, keep, err, st, mode, zero, zero_per_slice);
    if (rpt <= 4) return run_uniform<4>(d, fr, n, budget, r, keep, err, st, mode, zero, zero_per_slice);
    if (rpt <= 8) return run_uniform<8>(d, fr, n, budget, r, keep, err, st, mode, zero, zero_per_slice);
    if (rpt <= 16) return run_uniform<16>(d, fr, n, budget, r, keep, err, st, mode, zero, zero_per_slice);
    if (rpt <= 32) return run_uniform<32>(d, fr, n, budget, r, keep, err, st, mode, zero, zero_per_slice);
    return run_uniform<64>(d, fr, n, budget, r, keep, err, st, mode, zero, zero_per_slice);
  }
  if (many) return run_select<16>(d, tar, van, fr, n, budget, tar_total, r, keep, err, st, mode);
  if (rpt <= 4) return run_select<4>(d, tar, van, fr, n, budget, tar_total, r, keep, err, st, mode);
  if (rpt <= 8) return run_select<8>(d, tar, van, fr, n, budget, tar_total, r, keep, err, st, mode);
  if (rpt <= 12) return run_select<12>(d, tar, van, fr, n, budget, tar_total, r, keep, err, st, mode);
  if (rpt <= 16) return run_select<16>(d, tar, van, fr, n, budget, tar_total, r, keep, err, st, mode);
  if (rpt <= 32) return run_select<32>(d, tar, van, fr, n, budget, tar_total, r, keep, err, st, mode);
  return run_select<64>(d, tar, van, fr, n, budget, tar_total, r, keep, err, st, mode);
}

int64_t compact_chunks(int32_t budget) { return (budget + kCompactRows - 1) / kCompactRows; }

// flags_zeroed: an earlier kernel of the pass (the table or prev-row launch, or
// the uniform selection) has zeroed the flags already
template <int RB>
ipv_status run_compact(const Dims& d, void* K, void* V, int32_t* fr, int32_t* pa, int32_t n, const int32_t* keep,
                       int32_t budget, void* ws, hipStream_t st, bool flags_zeroed) {
  using C = CompactCfg<RB, kCompactThreads, kCompactRows, kCompactColBytes>;
  const uint32_t chunks = (uint32_t)compact_chunks(budget);
  const int64_t total = d.slices * C::PARTS * chunks;
  if (!flags_zeroed) {
    const int64_t words = d.slices * C::PARTS * walk_words(chunks);
    k_clear_flags<<<dim3((uint32_t)((words + 255) / 256)), dim3(256), 0, st>>>(ws_flags(ws, d), words);
  }
  k_compact<RB, kCompactThreads, kCompactRows, kCompactColBytes><<<dim3((uint32_t)total), dim3(kCompactThreads), 0, st>>>(
      static_cast<char*>(K), static_cast<char*>(V), fr, pa, d.S, n, budget, keep, err_word(ws), ws_flags(ws, d),
      chunks, make_fastdiv((uint32_t)(d.slices * C::PARTS)));
  return launched();
}

ipv_status compact(const Dims& d, void* K, void* V, int32_t* fr, int32_t* pa, int32_t n, const int32_t* keep,
                   int32_t budget, void* ws, hipStream_t st, bool flags_zeroed = false) {
  switch (d.D * d.elem) {
    case 64: return run_compact<64>(d, K, V, fr, pa, n, keep, budget, ws, st, flags_zeroed);
    case 128: return run_compact<128>(d, K, V, fr, pa, n, keep, budget, ws, st, flags_zeroed);
    case 256: return run_compact<256>(d, K, V, fr, pa, n, keep, budget, ws, st, flags_zeroed);
    case 512: return run_compact<512>(d, K, V, fr, pa, n, keep, budget, ws, st, flags_zeroed);
    case 1024: return run_compact<1024>(d, K, V, fr, pa, n, keep, budget, ws, st, flags_zeroed);
  }
  return IPV_ERR_SHAPE;
}

// ------------------------------------------------------------ append
// `frames` consecutive frames of `rows` rows each into rows
// [n, n + frames * rows) of every slice. Block row blockIdx.y takes slices
// blockIdx.y, + gridDim.y, ...; in a slice, a grid-stride loop over the 16-byte
// pieces of the new rows in destination order (contiguous), then their
// metadata: frame frame_id + j for the rows of frame j, patch first_patch +
// the row's place in its frame. Source frame j of slice s starts at byte
// j * frame_stride + s * rows * RB. The caller keeps frames * rows * RB within
// the slice's 32-bit byte range (n + frames * rows <= S).
__global__ __launch_bounds__(256) void k_append(const char* __restrict__ Kn, const char* __restrict__ Vn,
                                                char* __restrict__ K, char* __restrict__ V,
                                                int32_t* __restrict__ fr, int32_t* __restrict__ pa, int64_t S,
                                                int32_t n, int32_t rows, int32_t frames, int64_t frame_stride,
                                                int64_t RB, int32_t frame_id, int32_t first_patch, int64_t slices) {
  const uint32_t per_frame = (uint32_t)rows * (uint32_t)(RB / 16);
  const uint32_t pieces = (uint32_t)frames * per_frame, meta = (uint32_t)frames * (uint32_t)rows;
  const uint32_t first = blockIdx.x * blockDim.x + threadIdx.x, step = gridDim.x * blockDim.x;
  for (int64_t slice = blockIdx.y; slice < slices; slice += gridDim.y) {
    const char* ks = Kn + slice * rows * RB;
    const char* vs = Vn + slice * rows * RB;
    char* kd = K + (slice * S + n) * RB;
    char* vd = V + (slice * S + n) * RB;
    for (uint32_t e = first; e < pieces; e += step) {
      const uint32_t j = e / per_frame;
      const int64_t src = (int64_t)j * frame_stride + (int64_t)(e - j * per_frame) * 16;
      store16(kd + (int64_t)e * 16, load16(ks + src));
      store16(vd + (int64_t)e * 16, load16(vs + src));
    }
    for (uint32_t e = first; e < meta; e += step) {
      const uint32_t j = e / (uint32_t)rows;
      fr[slice * S + n + e] = frame_id + (int32_t)j;
      pa[slice * S + n + e] = first_patch + (int32_t)(e - j * (uint32_t)rows);
    }
  }
}

int32_t floor_share(double alpha, int32_t budget) { return (int32_t)std::floor(alpha * (double)budget); }

ipv_status check_tau(const double* tau) {
  if (!tau) return IPV_OK;
  for (int i = 0; i < 3; ++i)
    if (!std::isfinite(tau[i])) return IPV_ERR_ARG;
  if (!(tau[0] <= tau[1] && tau[1] <= tau[2])) return IPV_ERR_ARG;
  return IPV_OK;
}

// ------------------------------------------------------------ per-stream row counts
// Every call takes n_tokens as a host array of B row counts. The work is
// launched once per maximal run of consecutive streams with the same count
// (one run for a batch at one fill level); a stream with 0 rows is left alone.
// A run is a contiguous sub-batch: the same layouts with fewer streams, so the
// kernels see one count, and the runs reuse the workspace one after another
// on the stream.
Dims sub_batch(const Dims& d, int64_t nb) {
  Dims s = d;
  s.B = nb;
  s.slices = nb * d.L * d.H;
  return s;
}

template <typename T>
T* at_stream(T* p, int64_t b0, int64_t per_stream_elems) {
  return p ? p + b0 * per_stream_elems : p;
}

// fn(sub-batch dims, first stream, row count) for every run with a non-zero count
template <typename F>
ipv_status for_each_run(const Dims& d, const int32_t* n_tokens, F fn) {
  for (int64_t b = 0; b < d.B;) {
    const int32_t n = n_tokens[b];
    int64_t e = b + 1;
    while (e < d.B && n_tokens[e] == n) ++e;
    if (n > 0) IPV_TRY(fn(sub_batch(d, e - b), b, n));
    b = e;
  }
  return IPV_OK;
}

// every count in [0, min(S, kMaxRows)]; `each` checks the non-zero ones further
template <typename F>
ipv_status check_counts(const Dims& d, const int32_t* n_tokens, F each) {
  if (!n_tokens) return IPV_ERR_NULL;
  for (int64_t b = 0; b < d.B; ++b) {
    const int32_t n = n_tokens[b];
    if (n < 0 || n > d.S || n > kMaxRows) return IPV_ERR_SHAPE;
    if (n > 0) IPV_TRY(each(n));
  }
  return IPV_OK;
}

ipv_status no_check(int32_t) { return IPV_OK; }

// loop: the budget check of the continual-compression loop (check_loop_budget)
ipv_status check_pass_args(const Dims& d, const int32_t* n_tokens, int32_t budget, double alpha, int32_t r,
                           const double* cv_tau, uint32_t mode, bool loop = false) {
  IPV_TRY(check_recent(d, r));
  if (!(alpha >= 0.0 && alpha <= 1.0)) return IPV_ERR_ARG;
  IPV_TRY(check_counts(d, n_tokens, [&](int32_t n) {
    return loop ? check_loop_budget(d, n, budget, r) : check_budget(n, budget);
  }));
  IPV_TRY(check_tau(cv_tau));
  return check_mode(mode);
}

// the whole pass on one run; events (may be NULL) as in ipv_compress_timed
ipv_status compress_run(const Dims& d, void* K, void* V, int32_t* fr, int32_t* pa, int32_t n, int32_t budget,
                        double alpha, int32_t r, uint32_t mode, const double* cv_tau, float* tar, float* van,
                        int32_t* keep, void* ws, hipStream_t st, const ipv_events* events) {
  auto mark = [&](int i) -> ipv_status {
    if (!events || !events->at[i]) return IPV_OK;
    return hipEventRecord(static_cast<hipEvent_t>(events->at[i]), st) == hipSuccess ? IPV_OK : IPV_ERR_HIP;
  };
  const bool uniform = (mode & IPV_UNIFORM_SELECT) != 0;  // no scores: frame ids decide
  const bool adjacent = (mode & IPV_TAR_ADJACENT) != 0;
  // with the recent-key table, the pooling CV runs in the TaR launch
  const bool cv_fused = cv_tau && !uniform && !adjacent;
  IPV_TRY(mark(0));
  if (uniform)
    IPV_TRY(mark(1));
  else
    IPV_TRY(scores(d, K, V, fr, pa, n, r, tar, van, ws, st, [&]() { return mark(1); }, compact_chunks(budget),
                   adjacent, cv_fused ? cv_tau : nullptr));
  IPV_TRY(mark(2));
  if (cv_tau && !uniform) IPV_TRY(pool_d(d, cv_tau, van, fr, pa, n, nullptr, ws, st, cv_fused));
  IPV_TRY(mark(3));
  // the score launches zero the compaction's flags; without them the uniform selection does
  IPV_TRY(select(d, tar, van, fr, n, budget, floor_share(alpha, budget), r, keep, err_word(ws), st, mode,
                 uniform ? ws_flags(ws, d) : nullptr,
                 (int32_t)(compact_parts(d) * walk_words(compact_chunks(budget)))));
  IPV_TRY(mark(4));
  IPV_TRY(compact(d, K, V, fr, pa, n, keep, budget, ws, st, true));
  return mark(5);
}

// per-stream element counts of the arrays
int64_t kv_bytes_per_stream(const Dims& d) { return d.L * d.H * d.S * d.D * d.elem; }
int64_t rows_per_stream(const Dims& d) { return d.L * d.H * d.S; }

// Frames [0, frames) of K_new / V_new (frame j at byte j * frame_stride; in
// a frame the batch's [B, L, H, rows, D] layout) appended to every stream
// after its n_tokens[b] rows; one launch per run of equal counts (an empty
// stream appends at row 0 like any other). Arguments checked by the caller.
ipv_status append_frames(const Dims& d, void* K, void* V, int32_t* frame_idx, int32_t* patch_idx,
                         const int32_t* n_tokens, const void* K_new, const void* V_new, int32_t rows, int32_t frames,
                         int64_t frame_stride, int32_t frame_id, int32_t first_patch, hipStream_t st) {
  const int64_t RB = d.D * d.elem;
  const int64_t kb = kv_bytes_per_stream(d), rs = rows_per_stream(d), nb = d.L * d.H * (int64_t)rows * RB;
  const int64_t pieces = (int64_t)frames * rows * (RB / 16);
  for (int64_t b = 0; b < d.B;) {
    const int32_t n = n_tokens[b];
    int64_t e = b + 1;
    while (e < d.B && n_tokens[e] == n) ++e;
    const int64_t slices = (e - b) * d.L * d.H;
    const dim3 grid((uint32_t)std::min<int64_t>((pieces + 255) / 256, 256), (uint32_t)std::min<int64_t>(slices, 65535));
    k_append<<<grid, dim3(256), 0, st>>>(static_cast<const char*>(K_new) + b * nb,
                                         static_cast<const char*>(V_new) + b * nb, static_cast<char*>(K) + b * kb,
                                         static_cast<char*>(V) + b * kb, frame_idx + b * rs, patch_idx + b * rs, d.S, n,
                                         rows, frames, frame_stride, RB, frame_id, first_patch, slices);
    IPV_TRY(launched());
    b = e;
  }
  return IPV_OK;
}

}  // namespace

extern "C" {

ipv_status ipv_workspace_bytes(const ipv_shape* shape, size_t* bytes) {
  Dims d;
  IPV_TRY(check_shape(shape, &d));
  if (!bytes) return IPV_ERR_NULL;
  *bytes = ws_total(d);
  return IPV_OK;
}

ipv_status ipv_tar_scores(const ipv_shape* shape, const void* K, const int32_t* frame_idx, const int32_t* patch_idx,
                          const int32_t* n_tokens, int32_t recent_frames, uint32_t mode, float* tar, void* ws,
                          size_t ws_bytes, void* stream) {
  Dims d;
  IPV_TRY(check_shape(shape, &d));
  if (!K || !frame_idx || !patch_idx || !tar) return IPV_ERR_NULL;
  if (!aligned(K, 16) || !aligned(frame_idx, 16) || !aligned(patch_idx, 16) || !aligned(tar, 16)) return IPV_ERR_ALIGN;
  IPV_TRY(check_counts(d, n_tokens, no_check));
  IPV_TRY(check_recent(d, recent_frames));
  IPV_TRY(check_mode(mode));
  IPV_TRY(check_ws(d, ws, ws_bytes));
  const int64_t kb = kv_bytes_per_stream(d), rs = rows_per_stream(d);
  return for_each_run(d, n_tokens, [&](const Dims& s, int64_t b0, int32_t n) {
    return scores(s, static_cast<const char*>(K) + b0 * kb, nullptr, frame_idx + b0 * rs, patch_idx + b0 * rs, n,
                  recent_frames, tar + b0 * rs, nullptr, ws, static_cast<hipStream_t>(stream), no_mark, 0,
                  (mode & IPV_TAR_ADJACENT) != 0);
  });
}

ipv_status ipv_van_scores(const ipv_shape* shape, const void* V, const int32_t* frame_idx, const int32_t* patch_idx,
                          const int32_t* n_tokens, const double* cv_tau, float* van, int32_t* pool_size, void* ws,
                          size_t ws_bytes, void* stream) {
  Dims d;
  IPV_TRY(check_shape(shape, &d));
  if (!V || !frame_idx || !patch_idx || !van) return IPV_ERR_NULL;
  if (!aligned(V, 16) || !aligned(frame_idx, 16) || !aligned(patch_idx, 16) || !aligned(van, 16)) return IPV_ERR_ALIGN;
  if (pool_size && !aligned(pool_size, 4)) return IPV_ERR_ALIGN;
  IPV_TRY(check_counts(d, n_tokens, no_check));
  IPV_TRY(check_tau(cv_tau));
  IPV_TRY(check_ws(d, ws, ws_bytes));
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t kb = kv_bytes_per_stream(d), rs = rows_per_stream(d);
  return for_each_run(d, n_tokens, [&](const Dims& s, int64_t b0, int32_t n) -> ipv_status {
    const int32_t* fr = frame_idx + b0 * rs;
    const int32_t* pa = patch_idx + b0 * rs;
    float* vn = van + b0 * rs;
    int32_t* ps = at_stream(pool_size, b0, d.L);
    IPV_TRY(scores(s, nullptr, static_cast<const char*>(V) + b0 * kb, fr, pa, n, 1, nullptr, vn, ws, st));
    if (cv_tau) return pool_d(s, cv_tau, vn, fr, pa, n, ps, ws, st);
    if (ps) {
      const int64_t cnt = s.B * s.L;
      k_fill_i32<<<dim3((uint32_t)((cnt + 255) / 256)), dim3(256), 0, st>>>(ps, cnt, 1);
      return launched();
    }
    return IPV_OK;
  });
}

ipv_status ipv_select(const ipv_shape* shape, const float* tar, const float* van, const int32_t* frame_idx,
                      const int32_t* n_tokens, int32_t budget, double alpha, int32_t recent_frames, uint32_t mode,
                      int32_t* keep_idx, void* ws, size_t ws_bytes, void* stream) {
  Dims d;
  IPV_TRY(check_shape(shape, &d));
  if (!frame_idx || !keep_idx || (scores_needed(mode) && (!tar || !van))) return IPV_ERR_NULL;
  if (!aligned(tar, 16) || !aligned(van, 16) || !aligned(frame_idx, 16) || !aligned(keep_idx, 16)) return IPV_ERR_ALIGN;
  IPV_TRY(check_pass_args(d, n_tokens, budget, alpha, recent_frames, nullptr, mode));
  IPV_TRY(check_ws(d, ws, ws_bytes));
  const int64_t rs = rows_per_stream(d), ks = d.L * d.H * (int64_t)budget;
  return for_each_run(d, n_tokens, [&](const Dims& s, int64_t b0, int32_t n) {
    return select(s, at_stream(tar, b0, rs), at_stream(van, b0, rs), frame_idx + b0 * rs, n, budget,
                  floor_share(alpha, budget),
                  recent_frames, keep_idx + b0 * ks, err_word(ws), static_cast<hipStream_t>(stream), mode);
  });
}

ipv_status ipv_compact(const ipv_shape* shape, void* K, void* V, int32_t* frame_idx, int32_t* patch_idx,
                       const int32_t* n_tokens, const int32_t* keep_idx, int32_t budget, void* ws, size_t ws_bytes,
                       void* stream) {
  Dims d;
  IPV_TRY(check_shape(shape, &d));
  if (!K || !V || !frame_idx || !patch_idx || !keep_idx) return IPV_ERR_NULL;
  if (!aligned(K, 16) || !aligned(V, 16) || !aligned(frame_idx, 16) || !aligned(patch_idx, 16) ||
      !aligned(keep_idx, 16))
    return IPV_ERR_ALIGN;
  IPV_TRY(check_counts(d, n_tokens, [&](int32_t n) { return budget < 1 || budget > n ? IPV_ERR_BUDGET : IPV_OK; }));
  IPV_TRY(check_ws(d, ws, ws_bytes));
  const int64_t kb = kv_bytes_per_stream(d), rs = rows_per_stream(d), ks = d.L * d.H * (int64_t)budget;
  return for_each_run(d, n_tokens, [&](const Dims& s, int64_t b0, int32_t n) {
    return compact(s, static_cast<char*>(K) + b0 * kb, static_cast<char*>(V) + b0 * kb, frame_idx + b0 * rs,
                   patch_idx + b0 * rs, n, keep_idx + b0 * ks, budget, ws, static_cast<hipStream_t>(stream));
  });
}

}  // extern "C"

namespace {

// Every host check of a whole pass except the workspace's.
ipv_status check_compress(const ipv_shape* shape, Dims* d, const void* K, const void* V, const int32_t* frame_idx,
                          const int32_t* patch_idx, const int32_t* n_tokens, int32_t budget, double alpha,
                          int32_t recent_frames, uint32_t mode, const double* cv_tau, const float* tar,
                          const float* van, const int32_t* keep_idx) {
  IPV_TRY(check_shape(shape, d));
  if (!K || !V || !frame_idx || !patch_idx || !keep_idx || (scores_needed(mode) && (!tar || !van)))
    return IPV_ERR_NULL;
  if (!aligned(K, 16) || !aligned(V, 16) || !aligned(frame_idx, 16) || !aligned(patch_idx, 16) ||
      !aligned(tar, 16) || !aligned(van, 16) || !aligned(keep_idx, 16))
    return IPV_ERR_ALIGN;
  return check_pass_args(*d, n_tokens, budget, alpha, recent_frames, cv_tau, mode);
}

// ------------------------------------------------------------ allocation-free pass
// ipv_compress_noalloc's workspace: one array per GPU, allocated with the
// library's code object when it is loaded on that GPU and held until the
// process ends. Host code never passes `scratch` itself to a kernel (on the
// host the name is only a stand-in): it passes the device address that
// hipGetSymbolAddress returns for the current GPU, looked up on the first
// call on that GPU and kept per device.
constexpr size_t kScratchBytes = (size_t)96 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// The scratch array of the current device; the stream must belong to it.
ipv_status scratch_of(hipStream_t st, void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return IPV_ERR_HIP;
  if (st) {
    hipDevice_t sdev = -1;
    if (hipStreamGetDevice(st, &sdev) != hipSuccess) return IPV_ERR_HIP;
    if ((int)sdev != dev) return IPV_ERR_ARG;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return IPV_ERR_HIP;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return IPV_OK;
}

__global__ void k_copy_word(uint32_t* dst, const uint32_t* src) {
  if (threadIdx.x == 0) *dst = *src;
}

}  // namespace

extern "C" {

ipv_status ipv_compress_noalloc(const ipv_shape* shape, void* K, void* V, int32_t* frame_idx, int32_t* patch_idx,
                                const int32_t* n_tokens, int32_t budget, double alpha, int32_t recent_frames,
                                uint32_t mode, const double* cv_tau, float* tar, float* van, int32_t* keep_idx,
                                uint32_t* device_errors, void* stream) {
  Dims d;
  IPV_TRY(check_compress(shape, &d, K, V, frame_idx, patch_idx, n_tokens, budget, alpha, recent_frames, mode,
                         cv_tau, tar, van, keep_idx));
  if (ws_total(d) > kScratchBytes) return IPV_ERR_WORKSPACE;
  if (device_errors && !aligned(device_errors, 4)) return IPV_ERR_ALIGN;
  hipStream_t st = static_cast<hipStream_t>(stream);
  void* ws = nullptr;
  IPV_TRY(scratch_of(st, &ws));
  // the error word starts at zero (a kernel, not a memset, so the call can be
  // captured into a graph); everything else the pass reads it writes first
  k_fill_i32<<<dim3(1), dim3(64), 0, st>>>(static_cast<int32_t*>(ws), 1, 0);
  IPV_TRY(launched());
  IPV_TRY(ipv_compress_timed(shape, K, V, frame_idx, patch_idx, n_tokens, budget, alpha, recent_frames, mode,
                             cv_tau, tar, van, keep_idx, ws, kScratchBytes, stream, nullptr));
  if (device_errors) {
    k_copy_word<<<dim3(1), dim3(64), 0, st>>>(device_errors, err_word(ws));
    return launched();
  }
  return IPV_OK;
}

ipv_status ipv_compress_timed(const ipv_shape* shape, void* K, void* V, int32_t* frame_idx, int32_t* patch_idx,
                              const int32_t* n_tokens, int32_t budget, double alpha, int32_t recent_frames,
                              uint32_t mode, const double* cv_tau, float* tar, float* van, int32_t* keep_idx,
                              void* ws, size_t ws_bytes, void* stream, const ipv_events* events) {
  Dims d;
  IPV_TRY(check_compress(shape, &d, K, V, frame_idx, patch_idx, n_tokens, budget, alpha, recent_frames, mode,
                         cv_tau, tar, van, keep_idx));
  IPV_TRY(check_ws(d, ws, ws_bytes));
  const int64_t kb = kv_bytes_per_stream(d), rs = rows_per_stream(d), ks = d.L * d.H * (int64_t)budget;
  return for_each_run(d, n_tokens, [&](const Dims& s, int64_t b0, int32_t n) {
    return compress_run(s, static_cast<char*>(K) + b0 * kb, static_cast<char*>(V) + b0 * kb, frame_idx + b0 * rs,
                        patch_idx + b0 * rs, n, budget, alpha, recent_frames, mode, cv_tau, at_stream(tar, b0, rs),
                        at_stream(van, b0, rs), keep_idx + b0 * ks, ws, static_cast<hipStream_t>(stream), events);
  });
}

ipv_status ipv_compress(const ipv_shape* shape, void* K, void* V, int32_t* frame_idx, int32_t* patch_idx,
                        const int32_t* n_tokens, int32_t budget, double alpha, int32_t recent_frames, uint32_t mode,
                        const double* cv_tau, float* tar, float* van, int32_t* keep_idx, void* ws, size_t ws_bytes,
                        void* stream) {
  return ipv_compress_timed(shape, K, V, frame_idx, patch_idx, n_tokens, budget, alpha, recent_frames, mode, cv_tau,
                            tar, van, keep_idx, ws, ws_bytes, stream, nullptr);
}

ipv_status ipv_append(const ipv_shape* shape, void* K, void* V, int32_t* frame_idx, int32_t* patch_idx,
                      const int32_t* n_tokens, const void* K_new, const void* V_new, int32_t rows, int32_t frame_id,
                      int32_t first_patch, void* stream) {
  Dims d;
  IPV_TRY(check_shape(shape, &d));
  if (!K || !V || !frame_idx || !patch_idx || !K_new || !V_new || !n_tokens) return IPV_ERR_NULL;
  if (!aligned(K, 16) || !aligned(V, 16) || !aligned(frame_idx, 16) || !aligned(patch_idx, 16) ||
      !aligned(K_new, 16) || !aligned(V_new, 16))
    return IPV_ERR_ALIGN;
  if (rows < 1) return IPV_ERR_SHAPE;
  for (int64_t b = 0; b < d.B; ++b)
    if (n_tokens[b] < 0 || (int64_t)n_tokens[b] + rows > d.S) return IPV_ERR_SHAPE;
  if (first_patch < 0 || (int64_t)first_patch + rows > d.p) return IPV_ERR_ARG;
  return append_frames(d, K, V, frame_idx, patch_idx, n_tokens, K_new, V_new, rows, 1, 0, frame_id, first_patch,
                       static_cast<hipStream_t>(stream));
}

ipv_status ipv_ckv_step(const ipv_shape* shape, void* K, void* V, int32_t* frame_idx, int32_t* patch_idx,
                        const int32_t* n_tokens, const void* K_new, const void* V_new, int32_t rows, int32_t frame_id,
                        int32_t first_patch, int32_t mem_cap, int32_t budget, double alpha, int32_t recent_frames,
                        uint32_t mode, const double* cv_tau, float* tar, float* van, int32_t* keep_idx, void* ws,
                        size_t ws_bytes, int32_t* n_out, int32_t* compressed, void* stream) {
  Dims d;
  IPV_TRY(check_shape(shape, &d));
  if (!n_out || !compressed || !n_tokens) return IPV_ERR_NULL;
  if (mem_cap < 1 || mem_cap > d.S) return IPV_ERR_SHAPE;
  if (budget > mem_cap) return IPV_ERR_BUDGET;
  // the row counts after the append; the streams that reach the cap run the pass
  std::vector<int32_t> after((size_t)d.B), pass((size_t)d.B);
  bool any = false;
  for (int64_t b = 0; b < d.B; ++b) {
    if (n_tokens[b] < 0 || n_tokens[b] >= mem_cap) return IPV_ERR_SHAPE;
    after[b] = n_tokens[b] + rows;
    pass[b] = after[b] >= mem_cap ? after[b] : 0;
    any |= pass[b] > 0;
  }
  if (any) {
    // every argument of the pass is checked before the append is enqueued
    if (!keep_idx || !K || !V || !frame_idx || !patch_idx || (scores_needed(mode) && (!tar || !van)))
      return IPV_ERR_NULL;
    if (!aligned(tar, 16) || !aligned(van, 16) || !aligned(keep_idx, 16)) return IPV_ERR_ALIGN;
    IPV_TRY(check_pass_args(d, pass.data(), budget, alpha, recent_frames, cv_tau, mode, true));
    IPV_TRY(check_ws(d, ws, ws_bytes));
  }
  IPV_TRY(ipv_append(shape, K, V, frame_idx, patch_idx, n_tokens, K_new, V_new, rows, frame_id, first_patch, stream));
  if (any)
    IPV_TRY(ipv_compress(shape, K, V, frame_idx, patch_idx, pass.data(), budget, alpha, recent_frames, mode, cv_tau,
                         tar, van, keep_idx, ws, ws_bytes, stream));
  for (int64_t b = 0; b < d.B; ++b) {
    n_out[b] = pass[b] > 0 ? budget : after[b];
    compressed[b] = pass[b] > 0;
  }
  return IPV_OK;
}

ipv_status ipv_ckv_stream(const ipv_shape* shape, void* K, void* V, int32_t* frame_idx, int32_t* patch_idx,
                          int32_t* n_tokens, const void* frames_K, const void* frames_V, int32_t n_frames,
                          int32_t rows, int32_t first_frame_id, int32_t mem_cap, int32_t budget, double alpha,
                          int32_t recent_frames, uint32_t mode, const double* cv_tau, float* tar, float* van,
                          int32_t* keep_idx, void* ws, size_t ws_bytes, int32_t* passes, void* stream) {
  Dims d;
  IPV_TRY(check_shape(shape, &d));
  if (!n_tokens || !passes || !frames_K || !frames_V || !K || !V || !frame_idx || !patch_idx) return IPV_ERR_NULL;
  if (!aligned(K, 16) || !aligned(V, 16) || !aligned(frame_idx, 16) || !aligned(patch_idx, 16) ||
      !aligned(frames_K, 16) || !aligned(frames_V, 16))
    return IPV_ERR_ALIGN;
  if (n_frames < 0 || rows < 1 || mem_cap < 1 || mem_cap > d.S) return IPV_ERR_SHAPE;
  if (budget > mem_cap) return IPV_ERR_BUDGET;
  if ((int64_t)first_frame_id + n_frames > INT32_MAX || rows > d.p) return IPV_ERR_ARG;
  // every step is checked on the host before the first one is enqueued: the
  // row counts of the whole stretch follow from the counts, rows and cap alone
  std::vector<int32_t> n(n_tokens, n_tokens + d.B), after((size_t)d.B), pass((size_t)d.B);
  bool any_pass = false;
  for (int32_t f = 0; f < n_frames; ++f) {
    bool any = false;
    for (int64_t b = 0; b < d.B; ++b) {
      if (n[b] < 0 || n[b] >= mem_cap || (int64_t)n[b] + rows > d.S) return IPV_ERR_SHAPE;
      after[b] = n[b] + rows;
      pass[b] = after[b] >= mem_cap ? after[b] : 0;
      any |= pass[b] > 0;
    }
    if (any) IPV_TRY(check_pass_args(d, pass.data(), budget, alpha, recent_frames, cv_tau, mode, true));
    any_pass |= any;
    for (int64_t b = 0; b < d.B; ++b) n[b] = pass[b] > 0 ? budget : after[b];
  }
  if (any_pass) {
    if (!keep_idx || (scores_needed(mode) && (!tar || !van))) return IPV_ERR_NULL;
    if (!aligned(tar, 16) || !aligned(van, 16) || !aligned(keep_idx, 16)) return IPV_ERR_ALIGN;
    IPV_TRY(check_ws(d, ws, ws_bytes));
  }
  const int64_t frame_bytes = d.slices * rows * d.D * d.elem;
  const char* fk = static_cast<const char*>(frames_K);
  const char* fv = static_cast<const char*>(frames_V);
  for (int64_t b = 0; b < d.B; ++b) passes[b] = 0;
  std::vector<int32_t> n_out((size_t)d.B), fired((size_t)d.B);
  for (int32_t f = 0; f < n_frames;) {
    // frames [f, g) bring no stream to the cap: one append launch (per run of
    // equal counts) for all of them; frame g is a step with its pass
    int64_t until = INT64_MAX;  // frames until the first stream reaches the cap, that frame included
    for (int64_t b = 0; b < d.B; ++b) until = std::min<int64_t>(until, (mem_cap - n_tokens[b] + rows - 1) / rows);
    const int32_t g = (int32_t)std::min<int64_t>(n_frames, f + until - 1);
    if (g > f) {
      IPV_TRY(append_frames(d, K, V, frame_idx, patch_idx, n_tokens, fk + f * frame_bytes, fv + f * frame_bytes, rows,
                            g - f, frame_bytes, first_frame_id + f, 0, static_cast<hipStream_t>(stream)));
      for (int64_t b = 0; b < d.B; ++b) n_tokens[b] += (g - f) * rows;
    }
    if (g < n_frames) {
      IPV_TRY(ipv_ckv_step(shape, K, V, frame_idx, patch_idx, n_tokens, fk + g * frame_bytes, fv + g * frame_bytes, rows,
                           first_frame_id + g, 0, mem_cap, budget, alpha, recent_frames, mode, cv_tau, tar, van,
                           keep_idx, ws, ws_bytes, n_out.data(), fired.data(), stream));
      for (int64_t b = 0; b < d.B; ++b) {
        n_tokens[b] = n_out[b];
        passes[b] += fired[b];
      }
    }
    f = g + 1;
  }
  return IPV_OK;
}

ipv_status ipv_clear_device_errors(void* ws, size_t ws_bytes, void* stream) {
  if (!ws) return IPV_ERR_NULL;
  if (!aligned(ws, 256)) return IPV_ERR_ALIGN;
  if (ws_bytes < kWsHeader) return IPV_ERR_WORKSPACE;
  k_fill_i32<<<dim3(1), dim3(64), 0, static_cast<hipStream_t>(stream)>>>(static_cast<int32_t*>(ws), 1, 0);
  return launched();
}

ipv_status ipv_read_device_errors(const void* ws, size_t ws_bytes, void* stream, uint32_t* flags) {
  if (!ws || !flags) return IPV_ERR_NULL;
  if (!aligned(ws, 256)) return IPV_ERR_ALIGN;
  if (ws_bytes < kWsHeader) return IPV_ERR_WORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (hipMemcpyAsync(flags, ws, sizeof(uint32_t), hipMemcpyDeviceToHost, st) != hipSuccess) return IPV_ERR_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return IPV_ERR_HIP;
  return IPV_OK;
}

const char* ipv_status_str(ipv_status s) {
  switch (s) {
    case IPV_OK: return "ok";
    case IPV_ERR_NULL: return "a required pointer is NULL";
    case IPV_ERR_ALIGN: return "a pointer is not aligned as required";
    case IPV_ERR_SHAPE: return "unsupported or inconsistent shape";
    case IPV_ERR_DTYPE: return "unsupported dtype";
    case IPV_ERR_BUDGET: return "budget outside [1, n] (continual-compression loop: [min(n, r*p), n])";
    case IPV_ERR_ARG: return "invalid argument (alpha, recent_frames or cv_tau)";
    case IPV_ERR_WORKSPACE: return "workspace missing or too small";
    case IPV_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

}  // extern "C"
