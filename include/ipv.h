/*
 * ipv.h -- C ABI of the InfiniPot-V KV-cache compression pass for AMD MI355X
 * (gfx950). InfiniPot-V: "Memory-Constrained KV Cache Compression for
 * Streaming Video Understanding" (arXiv 2506.15745).
 *
 * When a streaming video model's KV cache reaches its memory cap |M|, the pass
 * shrinks every (stream, layer, KV head) slice to a budget of C rows:
 *
 *   ipv_tar_scores   Temporal-axis Redundancy score of every past row
 *                    (Sec. 3.1, TaR equation)
 *   ipv_van_scores   Value-Norm score of every row, optionally average-pooled
 *                    with a layer-adaptive window (Sec. 3.2; Algorithm 2)
 *   ipv_select       keep set: recent window + TaR picks + VaN picks
 *                    (Algorithm 1 steps (3)-(5); Sec. 3.3)
 *   ipv_compact      in-place, order-preserving gather of the kept rows
 *                    (Sec. 3.1; Algorithm 1 step (5))
 *   ipv_compress     the four steps above, in order, on one stream
 *   ipv_append       add a frame's rows to the cache (Algorithm 1 step (1))
 *   ipv_ckv_step     append, then compress when the memory cap is reached
 *   ipv_ckv_stream   many frames through that loop in one call
 *
 * A `mode` argument (IPV_MODE_* bits, 0 = the method as published) selects the
 * variants of the paper's ablation (Tab. 5: TaR Reverse, VaN Reverse, TaR
 * between consecutive frames) and the head-shared reading of the scores.
 *
 * ---------------------------------------------------------------- layouts
 * A cache holds B streams x L layers x H KV heads; each (b, l, h) "slice" has
 * a row capacity S of which rows [0, n_tokens[b]) are valid. n_tokens is a
 * HOST array of B row counts (streams fill at their own pace); a stream with
 * 0 rows is left alone by every call except ipv_append. The work is launched
 * once per maximal run of consecutive streams with the same count, so a batch
 * at one fill level is one launch per kernel. All row-major:
 *   K, V        [B, L, H, S, D] elements of `dtype` (bf16 or fp32), device
 *   frame_idx   [B, L, H, S] int32, device: frame id of each row
 *   patch_idx   [B, L, H, S] int32, device: patch position in [0, grid_h*grid_w)
 *   tar, van    [B, L, H, S] fp32, device (only rows [0, n) are written)
 *   keep_idx    [B, L, H, C] int32, device, strictly ascending row indices
 *   pool_size   [B, L] int32, device (pooling window chosen per layer)
 * Frame ids must not decrease along the rows of a slice, and a frame holds
 * each patch position at most once. This holds for a cache that appends whole
 * frames and is only ever compacted by this library (compaction is stable).
 * The recent window is every row whose frame id is >= F - r + 1, where F is
 * the frame id of row n-1 (a partial last frame counts as a frame).
 * Scores accumulate in fp32: a K or V row's squared norm must lie in the
 * fp32 range (finite, and normal unless the row is zero): element magnitudes
 * up to about 1e18 for D = 128. Beyond that the norm overflows and the
 * scores that involve the row are not meaningful; below it precision is
 * lost.
 *
 * Pointer alignment: K, V, tar, van, frame_idx, patch_idx, keep_idx 16 bytes;
 * the workspace 256 bytes.
 *
 * Workspace: ipv_workspace_bytes(shape) bytes of device memory. Calls that
 * share a workspace must not overlap in time.
 *
 * ---------------------------------------------------------------- ownership
 * The caller allocates and owns every buffer, including the workspace
 * (size from ipv_workspace_bytes). The library allocates no device memory,
 * keeps no state between calls and is thread-safe for distinct buffers.
 * `stream` is a hipStream_t (NULL: the default stream). Every call only
 * enqueues work on `stream` and returns; results are visible after the
 * stream is synchronised.
 *
 * ---------------------------------------------------------------- errors
 * Host-checkable argument errors return a non-zero ipv_status before
 * anything is enqueued and leave every buffer untouched. Problems that only
 * the device can see (metadata breaking the invariants above, a recent window
 * larger than the budget, a keep_idx that is not strictly ascending in [0, n),
 * a NaN score) set bits in the workspace's device error word
 * (IPV_DEV_*); the kernels stay in bounds, skip the offending rows and carry
 * on. Read the word with ipv_read_device_errors, reset it with
 * ipv_clear_device_errors. IPV_ERR_HIP means a launch failed (a stream error
 * is also reported by the next HIP call on that stream).
 */
#ifndef IPV_H
#define IPV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  IPV_OK = 0,
  IPV_ERR_NULL = 1,        /* a required pointer is NULL */
  IPV_ERR_ALIGN = 2,       /* a pointer breaks the alignment rules above */
  IPV_ERR_SHAPE = 3,       /* bad B/L/H/D/S/grid, a row count outside [0, S], or a size the kernels do not cover */
  IPV_ERR_DTYPE = 4,       /* dtype is neither IPV_BF16 nor IPV_F32 */
  IPV_ERR_BUDGET = 5,      /* budget outside [1, n]; ipv_ckv_step / ipv_ckv_stream: outside [min(n, r*p), n] */
  IPV_ERR_ARG = 6,         /* alpha outside [0, 1], recent_frames < 1, bad cv_tau */
  IPV_ERR_WORKSPACE = 7,   /* workspace missing or smaller than ipv_workspace_bytes */
  IPV_ERR_HIP = 8          /* the HIP runtime reported an error */
} ipv_status;

typedef enum { IPV_BF16 = 0, IPV_F32 = 1 } ipv_dtype;

/* Device error word bits (accumulated with atomic OR until cleared). */
enum {
  IPV_DEV_BAD_PATCH = 1u,      /* patch_idx outside [0, p): the row scored 0 / was left out of pooling */
  IPV_DEV_BAD_FRAMES = 2u,     /* frame ids decrease, a (frame, patch) pair repeats in the window (in any
                                  row with IPV_TAR_ADJACENT), or heads differ with IPV_HEAD_SHARED */
  IPV_DEV_RECENT_OVER = 4u,    /* recent window |R| larger than the budget: keep_idx set to 0..C-1 (the
                                  compaction then moves nothing) */
  IPV_DEV_BAD_KEEP = 8u,       /* keep_idx[j] outside [j, n) or not above keep_idx[j-1]: the compaction
                                  chunk (512 rows) holding row j was not moved */
  IPV_DEV_NAN = 16u,           /* a candidate score is NaN: its rank is unspecified */
  IPV_DEV_WAIT_TIMEOUT = 32u   /* compaction: a chunk's bounded wait expired or its walk's counters were
                                  not zero (a workspace shared by overlapping calls); its rows were not
                                  moved */
};

/*
 * Variant bits of the `mode` argument. Calls ignore the bits that do not
 * concern their step and reject unknown bits with IPV_ERR_ARG.
 */
enum {
  /* the TaR stage keeps the b_T past rows with the LOWEST tar (Tab. 5, TaR Reverse) */
  IPV_TAR_REVERSE = 1u,
  /* the VaN stage keeps the b_V rows with the LOWEST van (Tab. 5, VaN Reverse; Sec. 3.2) */
  IPV_VAN_REVERSE = 2u,
  /* TaR between consecutive frames (Sec. 3.1 and its figure on static patches of
     adjacent frames): a past row x at position q is compared with the one row
     at q in the latest earlier frame that holds q:
       tar[x] = -cos(K[x], K[y]),  0 if no earlier frame holds q. */
  IPV_TAR_ADJACENT = 4u,
  /* one keep set per (stream, layer) (the head-free s(t, i, j) and K[:, I, :] of
     Sec. 3.1-3.3): each stage ranks, per row, the sum over the layer's heads of
     their scores (fp32, heads added in order 0..H-1 starting from +0); every head
     must hold the same frame ids and receives the same keep_idx row. */
  IPV_HEAD_SHARED = 8u,
  /* Uniform Select, the frame-sampling baseline of the paper's KV-compression
     comparison (appendix, KV cache compression details: frames at regular
     intervals, every token of a taken frame). No scores: the recent window is
     kept, and the past budget b = C - |R| goes to the q past frames (numbered
     0..q-1 in row order, |P| past rows) at ranks floor(j * q / k),
     k = ceil(b * q / |P|): their rows in row order up to b, then, if those
     frames hold fewer than b rows, the lowest other past rows. tar and van are
     neither read nor written (they may be NULL) and alpha is unused; the
     other variant bits do not apply, and with IPV_HEAD_SHARED every head must
     hold the same frame ids (all heads then keep the same rows). */
  IPV_UNIFORM_SELECT = 16u,
  IPV_MODE_ALL = 31u
};

typedef struct {
  int32_t streams;   /* B >= 1 */
  int32_t layers;    /* L >= 1 */
  int32_t kv_heads;  /* H >= 1 */
  int32_t head_dim;  /* D: 32, 64, 128 or 256 */
  int32_t capacity;  /* S: row stride of a slice, S >= n */
  int32_t grid_h;    /* patch grid of a frame: p = grid_h * grid_w tokens per frame */
  int32_t grid_w;
  int32_t dtype;     /* ipv_dtype of K and V */
} ipv_shape;

/* Bytes of device workspace every call on this shape needs (>= 256). */
ipv_status ipv_workspace_bytes(const ipv_shape* shape, size_t* bytes);

/*
 * TaR score (Sec. 3.1, TaR equation). For a past row x at patch position q:
 *   tar[x] = -(1/r_q) * sum over the r_q recent rows y at position q of cos(K[x], K[y])
 * with cos = 0 when either key is zero, and tar[x] = 0 when r_q = 0 (a
 * position missing from a partial recent frame). Recent rows get 0. -0.0 is
 * written as +0.0. fp32 accumulation. Requires 1 <= r <= 256 and r * p <= 65536.
 * mode & IPV_TAR_ADJACENT: the consecutive-frame score described at that bit.
 */
ipv_status ipv_tar_scores(const ipv_shape* shape, const void* K, const int32_t* frame_idx,
                          const int32_t* patch_idx, const int32_t* n_tokens, int32_t recent_frames, uint32_t mode,
                          float* tar, void* ws, size_t ws_bytes, void* stream);

/*
 * VaN score (Sec. 3.2): van[x] = ||V[x]||_2 for every valid row, fp32.
 * With cv_tau (host pointer to three doubles tau1 <= tau2 <= tau3) the scores
 * are pooled per layer (Algorithm 2): CV = std/mean over all heads and valid
 * rows of the layer (population std), window k = 7 if CV < tau1, 5 if
 * CV < tau2, 3 if CV < tau3, else 1; each row's score becomes the mean over
 * the rows of its own frame and slice whose grid cell lies in the k x k window
 * around its cell (stride 1, cells outside the grid or absent are skipped).
 * cv_tau NULL: no pooling. pool_size (device, [B, L], may be NULL) receives k.
 */
ipv_status ipv_van_scores(const ipv_shape* shape, const void* V, const int32_t* frame_idx,
                          const int32_t* patch_idx, const int32_t* n_tokens, const double* cv_tau, float* van,
                          int32_t* pool_size, void* ws, size_t ws_bytes, void* stream);

/*
 * Keep set of `budget` = C rows per slice (Algorithm 1 steps (3)-(5); Sec. 3.3):
 *   b_T = max(0, floor(alpha * C) - |R|),  b_V = C - |R| - b_T   (floor taken in double)
 *   T = the b_T past rows with the highest tar, V = the b_V past rows outside T
 *   with the highest van; equal scores go to the lower row index, -0.0 == +0.0.
 *   keep_idx = R u T u V in ascending order.
 * Requires 1 <= C <= n and n <= 65536. The window |R| comes from the frame
 * ids on the device: when |R| > C the slice's keep_idx is 0..C-1 and
 * IPV_DEV_RECENT_OVER is raised.
 * mode: IPV_TAR_REVERSE / IPV_VAN_REVERSE take a stage's lowest scores (ties
 * still to the lower row index); IPV_HEAD_SHARED selects once per layer.
 */
ipv_status ipv_select(const ipv_shape* shape, const float* tar, const float* van, const int32_t* frame_idx,
                      const int32_t* n_tokens, int32_t budget, double alpha, int32_t recent_frames, uint32_t mode,
                      int32_t* keep_idx, void* ws, size_t ws_bytes, void* stream);

/*
 * In-place compaction (Sec. 3.1; Algorithm 1 step (5)): for j < C, row j of
 * K, V, frame_idx and patch_idx becomes a bit copy of row keep_idx[j]. Each
 * slice's keep_idx must be strictly ascending with entries in [0, n) (so
 * keep_idx[j] >= j), as ipv_select writes it; a chunk of 512 rows holding an
 * entry that breaks this is not moved and raises IPV_DEV_BAD_KEEP. Rows
 * [C, S) are left unspecified and free for new frames. The caller then sets
 * n_tokens[b] = C for every stream with n_tokens[b] > 0.
 * All chunks of all slices are copied in parallel; a chunk stores only after
 * every earlier chunk that reads its rows has loaded them (flags and a ticket
 * counter per walk in ws, zeroed by the call).
 */
ipv_status ipv_compact(const ipv_shape* shape, void* K, void* V, int32_t* frame_idx, int32_t* patch_idx,
                       const int32_t* n_tokens, const int32_t* keep_idx, int32_t budget, void* ws, size_t ws_bytes,
                       void* stream);

/* The whole pass: ipv_tar_scores, ipv_van_scores, ipv_select, ipv_compact,
   each with the same mode (with IPV_TAR_ADJACENT the VaN scores are computed
   in the same sweep as the consecutive-frame TaR scores). */
ipv_status ipv_compress(const ipv_shape* shape, void* K, void* V, int32_t* frame_idx, int32_t* patch_idx,
                        const int32_t* n_tokens, int32_t budget, double alpha, int32_t recent_frames, uint32_t mode,
                        const double* cv_tau, float* tar, float* van, int32_t* keep_idx, void* ws,
                        size_t ws_bytes, void* stream);

/*
 * ipv_compress with per-kernel timing: each non-NULL entry of `at` is a
 * hipEvent_t (created by the caller) recorded on `stream` at a step boundary:
 *   at[0] before the recent-key table   at[1] before the TaR/VaN sweep
 *   (IPV_TAR_ADJACENT: before the prev-row walk, before the adjacent sweep)
 *   at[2] before pooling                at[3] before selection
 *   at[4] before compaction             at[5] after compaction
 * Elapsed time between consecutive events is that step's device time. With
 * several runs of equal row counts the events are recorded in each run, so
 * they end up timing the last run.
 */
typedef struct {
  void* at[6];
} ipv_events;

ipv_status ipv_compress_timed(const ipv_shape* shape, void* K, void* V, int32_t* frame_idx, int32_t* patch_idx,
                              const int32_t* n_tokens, int32_t budget, double alpha, int32_t recent_frames,
                              uint32_t mode, const double* cv_tau, float* tar, float* van, int32_t* keep_idx,
                              void* ws, size_t ws_bytes, void* stream, const ipv_events* events);

/*
 * ipv_compress for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same pass and the same kernels, with the workspace taken from a 96 MiB
 * array that the library holds on each GPU it runs on (from the first call on
 * that GPU until the process ends) instead of a caller buffer. The call itself
 * allocates nothing. Shapes whose ipv_workspace_bytes exceeds 96 MiB are
 * refused with IPV_ERR_WORKSPACE (the 7B- and 72B-class caches fit; a batch of
 * 16 7B-class streams does not). The stream must belong to the current device
 * (IPV_ERR_ARG otherwise). device_errors (device, 4-byte aligned, may be NULL)
 * receives the pass's device error word (IPV_DEV_* bits), which the call
 * clears first. All calls on one GPU share its array: calls that overlap in
 * time on one GPU (other streams, other host threads) race and must not be
 * made; calls in sequence on one stream are fine.
 */
ipv_status ipv_compress_noalloc(const ipv_shape* shape, void* K, void* V, int32_t* frame_idx, int32_t* patch_idx,
                                const int32_t* n_tokens, int32_t budget, double alpha, int32_t recent_frames,
                                uint32_t mode, const double* cv_tau, float* tar, float* van, int32_t* keep_idx,
                                uint32_t* device_errors, void* stream);

/*
 * Append new rows to every slice (Algorithm 1 step (1): the tokens of a new
 * frame, or part of one, join the cache after prefill). Rows
 * [n_tokens[b], n_tokens[b] + rows) of each slice of stream b receive K_new / V_new
 * ([B, L, H, rows, D], same dtype as the cache, device, 16-byte aligned),
 * frame_idx = frame_id and patch_idx = first_patch + i for the i-th new row.
 * Needs n_tokens[b] >= 0, rows >= 1, n_tokens[b] + rows <= S and
 * first_patch + rows <= p. Stream b's row count becomes n_tokens[b] + rows.
 */
ipv_status ipv_append(const ipv_shape* shape, void* K, void* V, int32_t* frame_idx, int32_t* patch_idx,
                      const int32_t* n_tokens, const void* K_new, const void* V_new, int32_t rows, int32_t frame_id,
                      int32_t first_patch, void* stream);

/*
 * One iteration of continual KV cache compression (Algorithm 1; Sec. 3):
 * append the new rows to every stream (ipv_append), and compress to `budget`
 * rows every stream that then holds len >= mem_cap rows (ipv_compress with
 * the given alpha, recent_frames, mode and cv_tau; the other streams are left
 * alone). n_out[b] and compressed[b] (host arrays of B) receive each stream's
 * row count after the step and whether its pass ran.
 * Needs budget <= mem_cap <= S and n_tokens[b] < mem_cap (the previous step
 * left every stream below the cap). A pass that runs needs budget >=
 * min(len, r * p), the largest window a cache of len rows can hold, since the
 * loop does not read the device between passes. Positions: the cache holds keys before the
 * rotary position encoding and compaction keeps the order of the kept rows,
 * so after every step row j takes position j at decoding, which stays below
 * mem_cap + rows (appendix, positional-encoding details); no position array
 * is stored.
 */
ipv_status ipv_ckv_step(const ipv_shape* shape, void* K, void* V, int32_t* frame_idx, int32_t* patch_idx,
                        const int32_t* n_tokens, const void* K_new, const void* V_new, int32_t rows, int32_t frame_id,
                        int32_t first_patch, int32_t mem_cap, int32_t budget, double alpha, int32_t recent_frames,
                        uint32_t mode, const double* cv_tau, float* tar, float* van, int32_t* keep_idx, void* ws, size_t ws_bytes,
                        int32_t* n_out, int32_t* compressed, void* stream);

/*
 * A whole stretch of a stream through the loop above, driven from the host
 * library with no round trip per frame: for f = 0 .. n_frames-1, the
 * equivalent of ipv_ckv_step with K_new / V_new = frame f of frames_K /
 * frames_V ([n_frames, B, L, H, rows, D], device, 16-byte aligned), frame id
 * first_frame_id + f and first_patch 0. n_tokens (host, [B]) holds the row
 * counts on entry and receives them on return; passes (host, [B]) receives how
 * many times each stream was compressed. The frames between two passes go
 * out as one append launch (the result is that of one append per frame).
 * Every step is checked before the first is enqueued (the counts of the
 * whole stretch follow from the counts, rows, mem_cap and budget), so a
 * rejected call enqueues nothing. The only error that can come after the
 * first launch is IPV_ERR_HIP (the runtime refused a launch or a copy);
 * n_tokens and passes then describe the frames enqueued before it. The work
 * of all frames shares tar, van, keep_idx and the workspace, which hold the
 * last pass's values on return. Problems only the device sees (IPV_DEV_* bits)
 * accumulate in the workspace's error word over all passes of the call and do
 * not stop it: read the word with ipv_read_device_errors after the call.
 */
ipv_status ipv_ckv_stream(const ipv_shape* shape, void* K, void* V, int32_t* frame_idx, int32_t* patch_idx,
                          int32_t* n_tokens, const void* frames_K, const void* frames_V, int32_t n_frames,
                          int32_t rows, int32_t first_frame_id, int32_t mem_cap, int32_t budget, double alpha,
                          int32_t recent_frames, uint32_t mode, const double* cv_tau, float* tar, float* van,
                          int32_t* keep_idx, void* ws, size_t ws_bytes, int32_t* passes, void* stream);

/* Reset the workspace's device error word (a small kernel on `stream`). */
ipv_status ipv_clear_device_errors(void* ws, size_t ws_bytes, void* stream);

/* Synchronise `stream` and copy the device error word to *flags (host). */
ipv_status ipv_read_device_errors(const void* ws, size_t ws_bytes, void* stream, uint32_t* flags);

/* Static description of a status code. */
const char* ipv_status_str(ipv_status status);

#ifdef __cplusplus
}
#endif
#endif /* IPV_H */
