/*
 * CPU oracle of the InfiniPot-V KV-cache compression pass.
 *
 * TEST INFRASTRUCTURE ONLY. This file exists to check the GPU library. Only
 * the test suite, the package's smoke check and the benchmark's CPU-baseline
 * leg may load it; the product path never calls it and shares no code with it.
 *
 * It is plain and slow on purpose: scalar loops, fp64 accumulation, one
 * (stream, layer, head) slice at a time (OpenMP only spreads whole slices over
 * threads). Stored elements are decoded exactly (bf16 bits << 16 is an exact
 * float). Each function follows the paper's own definition of its step:
 *
 *   recent/past split   Sec. 3.1 (last r frames kept whole); Algorithm 1 step (2)
 *   TaR score           Sec. 3.1, TaR equation: minus the mean cosine between a
 *                       past key and the keys at the same patch position in the
 *                       r recent frames
 *   VaN score           Sec. 3.2: L2 norm of the value vector
 *   adaptive pooling    Sec. 3.2 "Layer-wise Adaptive Pooling"; Algorithm 2
 *                       (mean/std/CV of the layer's VaN, pooling size g(CV) from
 *                       thresholds tau1 < tau2 < tau3, AveragePool2d)
 *   selection           Algorithm 1 steps (3)-(5) and Sec. 3.3: TaR budget
 *                       floor(alpha*C) - |recent|, VaN fills the rest, the
 *                       recent window is always kept
 *   compaction          Sec. 3.1 / Algorithm 1 step (5): K <- K[I], V <- V[I]
 *
 * Variants (Tab. 5 ablation rows and the head-shared reading of the scores),
 * chosen by the `mode` bits:
 *   IPVO_TAR_REVERSE    the TaR stage keeps the lowest TaR scores (TaR Reverse)
 *   IPVO_VAN_REVERSE    the VaN stage keeps the lowest VaN scores (VaN Reverse)
 *   IPVO_TAR_ADJACENT   a past key is compared with the key at its patch
 *                       position in the closest earlier frame that still has
 *                       one (consecutive-frame similarity, Sec. 3.1 and its
 *                       figure on static patches between adjacent frames),
 *                       instead of with the r recent frames
 *   IPVO_HEAD_SHARED    one keep set per (stream, layer): each stage ranks the
 *                       fp32 sum over the layer's heads of their scores (the
 *                       head-free s(t, i, j) and K[:, I, :] of Sec. 3.1-3.3),
 *                       and every head keeps the same rows
 *   IPVO_UNIFORM        Uniform Select, the frame-sampling baseline of the
 *                       KV-compression comparison (appendix, KV cache
 *                       compression details): past frames at regular
 *                       intervals, all of their rows, no scores
 *
 * Readings where the paper is silent (documented with the design notes):
 *   - cos(a, b) = 0 when |a||b| = 0; a patch with no key in the recent window
 *     scores 0; -0.0 is written as +0.0.
 *   - scores are per (stream, layer, KV head); the keep set is per slice.
 *   - VaN candidates exclude rows already picked by TaR, so the kept count is
 *     exactly C; ties go to the lower row index; kept rows stay in order.
 *   - the recent window is every row whose frame id is >= F - r + 1, F being
 *     the frame id of the last valid row (a partial last frame counts as one).
 *   - pooling: stride 1, floor(k/2) cells each side, mean over the cells of
 *     the same frame that are present and inside the grid; CV uses the
 *     population standard deviation over all heads and rows of the layer.
 *
 * Layouts (row-major): K, V [B, L, H, S, D] (dtype 0 = bf16 bits, 1 = fp32);
 * frame_idx, patch_idx int32 [B, L, H, S]; scores [B, L, H, S]; rows [0, n)
 * are valid in every slice.
 */
#define _GNU_SOURCE
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int32_t streams, layers, kv_heads, head_dim, capacity, grid_h, grid_w, dtype;
} ipvo_shape;

typedef struct {
  int32_t n_recent, b_tar, b_van, pad;
  float cut_tar, cut_van; /* score of the last row picked by each stage (NaN if the stage picks none) */
} ipvo_select_info;

enum { IPVO_OK = 0, IPVO_ERR_ARG = -1, IPVO_ERR_META = -2, IPVO_ERR_BUDGET = -3, IPVO_ERR_NAN = -4 };
enum {
  IPVO_TAR_REVERSE = 1,
  IPVO_VAN_REVERSE = 2,
  IPVO_TAR_ADJACENT = 4,
  IPVO_HEAD_SHARED = 8,
  IPVO_UNIFORM = 16,
  IPVO_MODES = 31
};

static int shape_ok(const ipvo_shape* s, int32_t n) {
  if (!s) return 0;
  if (s->streams < 1 || s->layers < 1 || s->kv_heads < 1 || s->head_dim < 1) return 0;
  if (s->grid_h < 1 || s->grid_w < 1 || (s->dtype != 0 && s->dtype != 1)) return 0;
  if (n < 1 || n > s->capacity) return 0;
  return 1;
}

static int64_t n_slices(const ipvo_shape* s) { return (int64_t)s->streams * s->layers * s->kv_heads; }

/* element e of row x in slice sl, decoded exactly */
static double elem(const ipvo_shape* s, const void* base, int64_t sl, int64_t x, int32_t e) {
  int64_t i = (sl * s->capacity + x) * s->head_dim + e;
  if (s->dtype == 1) return (double)((const float*)base)[i];
  uint32_t bits = (uint32_t)((const uint16_t*)base)[i] << 16;
  float f;
  memcpy(&f, &bits, 4);
  return (double)f;
}

int32_t ipvo_max_threads(void) { return omp_get_max_threads(); }

/* Threads for the slice loops that follow (the benchmark's single-thread
 * timing); the arithmetic of each slice does not depend on it. */
void ipvo_set_threads(int32_t threads) { omp_set_num_threads(threads > 0 ? threads : 1); }

/*
 * Recent window of one slice (Sec. 3.1; Algorithm 1 step (2)): rows whose
 * frame id is one of the r latest, counted from the last valid row's frame.
 * Writes is_recent[0..n) and returns |R|, or -1 if the metadata breaks the
 * cache's invariants (frame ids must not decrease along the rows, so the
 * window is a suffix).
 */
static int32_t recent_window(const int32_t* fr, int32_t n, int32_t r, unsigned char* is_recent) {
  int32_t last = fr[n - 1];
  int64_t thr = (int64_t)last - r + 1;
  int32_t count = 0;
  for (int32_t x = 0; x < n; ++x) {
    if (x > 0 && fr[x] < fr[x - 1]) return -1;
    is_recent[x] = (unsigned char)(fr[x] >= thr);
    count += is_recent[x];
  }
  return count;
}

static double cosine(const ipvo_shape* s, const void* K, int64_t sl, int64_t a, int64_t b) {
  double dot = 0.0, na = 0.0, nb = 0.0;
  for (int32_t e = 0; e < s->head_dim; ++e) {
    double ka = elem(s, K, sl, a, e), kb = elem(s, K, sl, b, e);
    dot += ka * kb;
    na += ka * ka;
    nb += kb * kb;
  }
  double den = sqrt(na) * sqrt(nb);
  return den == 0.0 ? 0.0 : dot / den;
}

/*
 * TaR score (Sec. 3.1, TaR equation; Algorithm 2's loop over past patches):
 * for a past row x at patch position q, minus the mean of cos(K[x], K[y]) over
 * the recent rows y at the same position q. Recent rows get 0 (they are kept
 * regardless). Rows [n, S) are not written.
 * IPVO_TAR_ADJACENT: minus cos(K[x], K[y]) for the one row y at position q
 * whose frame is the latest frame before x's that has a row at q (0 if no
 * earlier frame has one).
 */
int ipvo_tar_scores(const ipvo_shape* s, const void* K, const int32_t* frame_idx, const int32_t* patch_idx,
                    int32_t n, int32_t recent_frames, uint32_t mode, double* tar) {
  if (!shape_ok(s, n) || !K || !frame_idx || !patch_idx || !tar || recent_frames < 1) return IPVO_ERR_ARG;
  if (mode & ~(uint32_t)IPVO_MODES) return IPVO_ERR_ARG;
  const int32_t p = s->grid_h * s->grid_w;
  int err = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
  for (int64_t sl = 0; sl < n_slices(s); ++sl) {
    const int32_t* fr = frame_idx + sl * s->capacity;
    const int32_t* pa = patch_idx + sl * s->capacity;
    double* out = tar + sl * s->capacity;
    unsigned char* rec = malloc((size_t)n);
    int32_t nr = recent_window(fr, n, recent_frames, rec);
    if (nr < 0) { err |= 1; free(rec); continue; }
    for (int32_t x = 0; x < n; ++x) {
      if (pa[x] < 0 || pa[x] >= p) err |= 1;
      /* consecutive-frame TaR needs each (frame, patch) pair at most once */
      if (mode & IPVO_TAR_ADJACENT)
        for (int32_t y = x - 1; y >= 0 && fr[y] == fr[x]; --y)
          if (pa[y] == pa[x]) err |= 1;
      if (rec[x]) { out[x] = 0.0; continue; }
      double sum = 0.0;
      int32_t count = 0;
      if (mode & IPVO_TAR_ADJACENT) {
        /* frame ids do not decrease along the rows: walk back to the first
           row at position q that lies in an earlier frame */
        for (int32_t y = x - 1; y >= 0; --y)
          if (pa[y] == pa[x] && fr[y] < fr[x]) {
            sum = cosine(s, K, sl, x, y);
            count = 1;
            break;
          }
      } else {
        for (int32_t y = n - nr; y < n; ++y) {
          if (pa[y] != pa[x]) continue;
          sum += cosine(s, K, sl, x, y);
          count += 1;
        }
      }
      double v = count ? -(sum / count) : 0.0;
      out[x] = (v == 0.0) ? 0.0 : v; /* -0.0 -> +0.0 */
    }
    free(rec);
  }
  return err ? IPVO_ERR_META : IPVO_OK;
}

/* Pooling size from the layer's coefficient of variation (Algorithm 2, g). */
static int32_t pool_size_of(double cv, const double* tau) {
  if (cv < tau[0]) return 7;
  if (cv < tau[1]) return 5;
  if (cv < tau[2]) return 3;
  return 1;
}

/*
 * VaN score (Sec. 3.2): ||V[x]||_2 for every valid row. With thresholds tau
 * the scores are then average-pooled per layer (Algorithm 2): CV_l = std/mean
 * of all VaN values of layer l (all heads, all valid rows; population std),
 * k = g(CV_l), and each row's score becomes the mean VaN over the rows of the
 * same slice and frame whose grid cell lies in the k x k window centred on
 * its own cell. pool_size[b, l] receives k (1 without tau) when non-NULL.
 */
int ipvo_van_scores(const ipvo_shape* s, const void* V, const int32_t* frame_idx, const int32_t* patch_idx,
                    int32_t n, const double* cv_tau, double* van, int32_t* pool_size) {
  if (!shape_ok(s, n) || !V || !frame_idx || !patch_idx || !van) return IPVO_ERR_ARG;
  if (cv_tau && !(cv_tau[0] <= cv_tau[1] && cv_tau[1] <= cv_tau[2])) return IPVO_ERR_ARG;
  const int32_t p = s->grid_h * s->grid_w, gw = s->grid_w, gh = s->grid_h;
  const int64_t S = s->capacity, H = s->kv_heads;
  int err = 0;

#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t sl = 0; sl < n_slices(s); ++sl) {
    for (int32_t x = 0; x < n; ++x) {
      double ss = 0.0;
      for (int32_t e = 0; e < s->head_dim; ++e) {
        double v = elem(s, V, sl, x, e);
        ss += v * v;
      }
      van[sl * S + x] = sqrt(ss);
    }
  }

  const int64_t layers_total = (int64_t)s->streams * s->layers;
  for (int64_t bl = 0; bl < layers_total; ++bl) {
    int32_t k = 1;
    if (cv_tau) {
      double sum = 0.0, cnt = (double)H * n;
      for (int64_t h = 0; h < H; ++h)
        for (int32_t x = 0; x < n; ++x) sum += van[(bl * H + h) * S + x];
      double mean = sum / cnt, var = 0.0;
      for (int64_t h = 0; h < H; ++h)
        for (int32_t x = 0; x < n; ++x) {
          double d = van[(bl * H + h) * S + x] - mean;
          var += d * d;
        }
      double sd = sqrt(var / cnt);
      double cv = mean == 0.0 ? 0.0 : sd / mean;
      k = pool_size_of(cv, cv_tau);
    }
    if (pool_size) pool_size[bl] = k;
    if (k == 1) continue;
    const int32_t half = k / 2;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
    for (int64_t h = 0; h < H; ++h) {
      const int64_t sl = bl * H + h;
      const int32_t* fr = frame_idx + sl * S;
      const int32_t* pa = patch_idx + sl * S;
      double* raw = malloc(sizeof(double) * (size_t)n);
      double* cell = malloc(sizeof(double) * (size_t)p);
      unsigned char* present = malloc((size_t)p);
      memcpy(raw, van + sl * S, sizeof(double) * (size_t)n);
      int32_t a = 0;
      while (a < n) {
        /* one frame: rows [a, b) share frame_idx[a] */
        int32_t b = a;
        while (b < n && fr[b] == fr[a]) ++b;
        if (b < n && fr[b] < fr[a]) err |= 1;
        memset(present, 0, (size_t)p);
        for (int32_t y = a; y < b; ++y) {
          if (pa[y] < 0 || pa[y] >= p || present[pa[y]]) { err |= 1; continue; }
          present[pa[y]] = 1;
          cell[pa[y]] = raw[y];
        }
        for (int32_t x = a; x < b; ++x) {
          if (pa[x] < 0 || pa[x] >= p) continue;
          int32_t ci = pa[x] / gw, cj = pa[x] % gw;
          double sum = 0.0;
          int32_t count = 0;
          for (int32_t i = ci - half; i <= ci + half; ++i) {
            if (i < 0 || i >= gh) continue;
            for (int32_t j = cj - half; j <= cj + half; ++j) {
              if (j < 0 || j >= gw || !present[i * gw + j]) continue;
              sum += cell[i * gw + j];
              count += 1;
            }
          }
          van[sl * S + x] = sum / count;
        }
        a = b;
      }
      free(raw);
      free(cell);
      free(present);
    }
  }
  return err ? IPVO_ERR_META : IPVO_OK;
}

/* Top-k order: higher score first, equal scores by lower row index. */
static int by_score_desc(const void* pa, const void* pb, void* ctx) {
  const float* sc = (const float*)ctx;
  int32_t a = *(const int32_t*)pa, b = *(const int32_t*)pb;
  if (sc[a] > sc[b]) return -1;
  if (sc[a] < sc[b]) return 1;
  return (a > b) - (a < b);
}

/* Reverse order (the ablation's reversed stages): lower score first, equal
   scores by lower row index. */
static int by_score_asc(const void* pa, const void* pb, void* ctx) {
  const float* sc = (const float*)ctx;
  int32_t a = *(const int32_t*)pa, b = *(const int32_t*)pb;
  if (sc[a] < sc[b]) return -1;
  if (sc[a] > sc[b]) return 1;
  return (a > b) - (a < b);
}

/*
 * Uniform Select (appendix, KV cache compression details: frames taken at
 * regular intervals with every token of each taken frame). With the recent
 * window R kept as in the other modes, the past rows P = [0, n - |R|) hold q
 * distinct frame ids; number them 0..q-1 in row order. The past budget
 * b = C - |R| buys k = ceil(b * q / |P|) frames (b in frames of the past's
 * average size, rounded up), taken at ranks floor(j * q / k), j = 0..k-1
 * (steps of q / k >= 1 frames from the oldest). The b past rows kept are the
 * rows of the taken frames in row order (the last one cut short when b is not
 * a whole number of frames), then, if those frames hold fewer than b rows
 * (frames that lost rows to earlier passes), the lowest past rows of the
 * other frames. Writes keep[x] = 1 for the b picks.
 */
static void uniform_pick(const int32_t* fr, int32_t n_past, int32_t b, unsigned char* keep) {
  if (b <= 0) return;
  /* rank of each past row's frame */
  int32_t* rank = malloc(sizeof(int32_t) * (size_t)(n_past > 0 ? n_past : 1));
  int32_t q = 0;
  for (int32_t x = 0; x < n_past; ++x) {
    if (x == 0 || fr[x] != fr[x - 1]) ++q;
    rank[x] = q - 1;
  }
  const int64_t k = ((int64_t)b * q + n_past - 1) / n_past;
  unsigned char* taken = calloc((size_t)q, 1);
  for (int64_t j = 0; j < k; ++j) taken[(j * q) / k] = 1;
  int32_t left = b;
  for (int32_t x = 0; x < n_past && left > 0; ++x)
    if (taken[rank[x]]) {
      keep[x] = 1;
      --left;
    }
  for (int32_t x = 0; x < n_past && left > 0; ++x)
    if (!taken[rank[x]]) {
      keep[x] = 1;
      --left;
    }
  free(taken);
  free(rank);
}

/*
 * One keep set from one pair of fp32 score columns and one frame column.
 * Returns an error bit (0 on success) and fills keep_idx[0..budget) and *inf.
 */
static int select_one(const float* st, const float* sv, const int32_t* fr, int32_t n, int32_t budget,
                      int32_t tar_budget_total, int32_t recent_frames, uint32_t mode, int32_t* keep_idx,
                      ipvo_select_info* info) {
  unsigned char* rec = malloc((size_t)n);
  unsigned char* keep = calloc((size_t)n, 1);
  int32_t* order = malloc(sizeof(int32_t) * (size_t)n);
  int err = 0;
  int32_t nr = recent_window(fr, n, recent_frames, rec);
  ipvo_select_info inf = {nr, 0, 0, 0, NAN, NAN};
  if (nr < 0) err |= 2;
  else if (nr > budget) err |= 4;
  else if (mode & IPVO_UNIFORM) {
    /* the window is a suffix: the past rows are [0, n - nr) */
    inf.b_van = budget - nr;
    for (int32_t x = 0; x < n; ++x) keep[x] = rec[x];
    uniform_pick(fr, n - nr, budget - nr, keep);
    int32_t j = 0;
    for (int32_t x = 0; x < n; ++x)
      if (keep[x]) keep_idx[j++] = x;
    if (j != budget) err |= 16;
  } else {
    for (int32_t x = 0; x < n; ++x)
      if (!rec[x] && (isnan(st[x]) || isnan(sv[x]))) err |= 8;
    int32_t bt = tar_budget_total - nr;
    if (bt < 0) bt = 0;
    int32_t bv = budget - nr - bt;
    inf.b_tar = bt;
    inf.b_van = bv;
    for (int32_t x = 0; x < n; ++x) keep[x] = rec[x];
    /* TaR stage over the past rows */
    int32_t m = 0;
    for (int32_t x = 0; x < n; ++x)
      if (!rec[x]) order[m++] = x;
    qsort_r(order, (size_t)m, sizeof(int32_t), (mode & IPVO_TAR_REVERSE) ? by_score_asc : by_score_desc,
            (void*)st);
    for (int32_t i = 0; i < bt; ++i) keep[order[i]] = 1;
    if (bt > 0) inf.cut_tar = st[order[bt - 1]];
    /* VaN stage over the past rows TaR did not pick */
    m = 0;
    for (int32_t x = 0; x < n; ++x)
      if (!keep[x]) order[m++] = x;
    qsort_r(order, (size_t)m, sizeof(int32_t), (mode & IPVO_VAN_REVERSE) ? by_score_asc : by_score_desc,
            (void*)sv);
    for (int32_t i = 0; i < bv; ++i) keep[order[i]] = 1;
    if (bv > 0) inf.cut_van = sv[order[bv - 1]];
    int32_t j = 0;
    for (int32_t x = 0; x < n; ++x)
      if (keep[x]) keep_idx[j++] = x;
    if (j != budget) err |= 16;
  }
  *info = inf;
  free(rec);
  free(keep);
  free(order);
  return err;
}

/*
 * Keep-set selection (Algorithm 1 steps (3)-(5); Sec. 3.3). Scores are fp32,
 * the precision the GPU decides in. With R the recent window:
 *   b_T = max(0, floor(alpha * C) - |R|),  b_V = C - |R| - b_T
 *   T = the b_T past rows with the highest TaR score
 *   V = the b_V past rows outside T with the highest VaN score
 *   keep = R u T u V, ascending.
 * tar_budget_total = floor(alpha * C) computed by the caller in double.
 * IPVO_TAR_REVERSE / IPVO_VAN_REVERSE: that stage takes the lowest scores.
 * IPVO_HEAD_SHARED: per (stream, layer), the scores of heads 0..H-1 are added
 * in that order in fp32, every head must hold the same frame ids, and the one
 * keep set (and info) is written for every head.
 * IPVO_UNIFORM: the past rows come from frames at regular intervals
 * (uniform_pick); the scores are not read and may be NULL.
 */
int ipvo_select(const ipvo_shape* s, const float* tar, const float* van, const int32_t* frame_idx, int32_t n,
                int32_t budget, int32_t tar_budget_total, int32_t recent_frames, uint32_t mode, int32_t* keep_idx,
                ipvo_select_info* info) {
  const int uniform = (mode & IPVO_UNIFORM) != 0;
  if (!shape_ok(s, n) || (!uniform && (!tar || !van)) || !frame_idx || !keep_idx || recent_frames < 1)
    return IPVO_ERR_ARG;
  if (mode & ~(uint32_t)IPVO_MODES) return IPVO_ERR_ARG;
  if (budget < 1 || budget > n || tar_budget_total < 0 || tar_budget_total > budget) return IPVO_ERR_BUDGET;
  const int64_t S = s->capacity;
  /* slices that share one keep set; Uniform Select reads frame ids only, the same in every head */
  const int32_t G = (mode & IPVO_HEAD_SHARED) && !uniform ? s->kv_heads : 1;
  int err = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
  for (int64_t grp = 0; grp < n_slices(s) / G; ++grp) {
    const int64_t sl0 = grp * G;
    ipvo_select_info inf;
    if (G == 1) {
      err |= select_one(uniform ? NULL : tar + sl0 * S, uniform ? NULL : van + sl0 * S, frame_idx + sl0 * S, n,
                        budget, tar_budget_total, recent_frames, mode, keep_idx + sl0 * budget, &inf);
    } else {
      float* st = malloc(sizeof(float) * (size_t)n);
      float* sv = malloc(sizeof(float) * (size_t)n);
      for (int32_t x = 0; x < n; ++x) {
        float a = 0.0f, b = 0.0f;
        for (int32_t h = 0; h < G; ++h) {
          a += tar[(sl0 + h) * S + x];
          b += van[(sl0 + h) * S + x];
          if (frame_idx[(sl0 + h) * S + x] != frame_idx[sl0 * S + x]) err |= 2;
        }
        st[x] = a;
        sv[x] = b;
      }
      err |= select_one(st, sv, frame_idx + sl0 * S, n, budget, tar_budget_total, recent_frames, mode,
                        keep_idx + sl0 * budget, &inf);
      for (int32_t h = 1; h < G; ++h)
        memcpy(keep_idx + (sl0 + h) * budget, keep_idx + sl0 * budget, sizeof(int32_t) * (size_t)budget);
      free(st);
      free(sv);
    }
    if (info)
      for (int32_t h = 0; h < G; ++h) info[sl0 + h] = inf;
  }
  if (uniform && (mode & IPVO_HEAD_SHARED)) {
    /* one keep set per layer: every head must hold the same frame ids (then
       every head's keep set, computed from them alone, is the same) */
    const int32_t H = s->kv_heads;
    for (int64_t sl = 0; sl < n_slices(s); ++sl)
      for (int32_t x = 0; x < n; ++x)
        if (frame_idx[sl * S + x] != frame_idx[(sl - sl % H) * S + x]) err |= 2;
  }
  if (err & 2) return IPVO_ERR_META;
  if (err & 4) return IPVO_ERR_BUDGET;
  if (err & 8) return IPVO_ERR_NAN;
  return err ? IPVO_ERR_META : IPVO_OK;
}

/*
 * Compaction (Algorithm 1 step (5)): row j of K, V, frame_idx and patch_idx
 * becomes row keep[j], for j < C, as a bit copy through a separate buffer.
 * Rows [C, S) are left as they were.
 */
int ipvo_compact(const ipvo_shape* s, void* K, void* V, int32_t* frame_idx, int32_t* patch_idx, int32_t n,
                 const int32_t* keep_idx, int32_t budget) {
  if (!shape_ok(s, n) || !K || !V || !frame_idx || !patch_idx || !keep_idx) return IPVO_ERR_ARG;
  if (budget < 1 || budget > n) return IPVO_ERR_BUDGET;
  const int64_t S = s->capacity;
  const size_t row = (size_t)s->head_dim * (s->dtype == 1 ? 4 : 2);
  int err = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
  for (int64_t sl = 0; sl < n_slices(s); ++sl) {
    const int32_t* keep = keep_idx + sl * budget;
    char* tk = malloc(row * (size_t)budget);
    char* tv = malloc(row * (size_t)budget);
    int32_t* tf = malloc(sizeof(int32_t) * (size_t)budget);
    int32_t* tp = malloc(sizeof(int32_t) * (size_t)budget);
    char* kb = (char*)K + (size_t)sl * S * row;
    char* vb = (char*)V + (size_t)sl * S * row;
    int ok = 1;
    for (int32_t j = 0; j < budget; ++j)
      if (keep[j] < 0 || keep[j] >= n) ok = 0;
    if (ok) {
      for (int32_t j = 0; j < budget; ++j) {
        memcpy(tk + row * j, kb + row * (size_t)keep[j], row);
        memcpy(tv + row * j, vb + row * (size_t)keep[j], row);
        tf[j] = frame_idx[sl * S + keep[j]];
        tp[j] = patch_idx[sl * S + keep[j]];
      }
      memcpy(kb, tk, row * (size_t)budget);
      memcpy(vb, tv, row * (size_t)budget);
      memcpy(frame_idx + sl * S, tf, sizeof(int32_t) * (size_t)budget);
      memcpy(patch_idx + sl * S, tp, sizeof(int32_t) * (size_t)budget);
    } else {
      err |= 1;
    }
    free(tk);
    free(tv);
    free(tf);
    free(tp);
  }
  return err ? IPVO_ERR_ARG : IPVO_OK;
}

/*
 * The whole pass in the paper's order (Algorithm 1 steps (2)-(5)): TaR and
 * VaN scores in fp64, rounded to fp32 for the selection, then compaction in
 * place. tar/van/keep_idx/info may be NULL (scratch is allocated here).
 */
int ipvo_compress(const ipvo_shape* s, void* K, void* V, int32_t* frame_idx, int32_t* patch_idx, int32_t n,
                  int32_t budget, int32_t tar_budget_total, int32_t recent_frames, uint32_t mode,
                  const double* cv_tau, float* tar_out, float* van_out, int32_t* keep_out, ipvo_select_info* info) {
  if (!shape_ok(s, n)) return IPVO_ERR_ARG;
  const int64_t cells = n_slices(s) * s->capacity;
  double* tar = calloc((size_t)cells, sizeof(double));
  double* van = calloc((size_t)cells, sizeof(double));
  float* tf = tar_out ? tar_out : calloc((size_t)cells, sizeof(float));
  float* vf = van_out ? van_out : calloc((size_t)cells, sizeof(float));
  int32_t* keep = keep_out ? keep_out : malloc(sizeof(int32_t) * (size_t)(n_slices(s) * budget));
  int rc = IPVO_OK;
  if (!(mode & IPVO_UNIFORM)) {  /* Uniform Select scores nothing */
    rc = ipvo_tar_scores(s, K, frame_idx, patch_idx, n, recent_frames, mode, tar);
    if (rc == IPVO_OK) rc = ipvo_van_scores(s, V, frame_idx, patch_idx, n, cv_tau, van, NULL);
  }
  if (rc == IPVO_OK) {
    for (int64_t sl = 0; sl < n_slices(s); ++sl)
      for (int32_t x = 0; x < n; ++x) {
        tf[sl * s->capacity + x] = (float)tar[sl * s->capacity + x];
        vf[sl * s->capacity + x] = (float)van[sl * s->capacity + x];
      }
    rc = ipvo_select(s, tf, vf, frame_idx, n, budget, tar_budget_total, recent_frames, mode, keep, info);
  }
  if (rc == IPVO_OK) rc = ipvo_compact(s, K, V, frame_idx, patch_idx, n, keep, budget);
  free(tar);
  free(van);
  if (!tar_out) free(tf);
  if (!van_out) free(vf);
  if (!keep_out) free(keep);
  return rc;
}
