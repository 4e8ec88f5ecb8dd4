// Host side of the C ABI declared in include/conduit.h: argument checks,
// workspace layout, and the launch sequence of each entry point.  Every check
// runs before the first HIP call, so a rejected call enqueues nothing.
#include "conduit.h"

#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <string>

#include "common.h"

using namespace conduit;

// bf16 scoring reads the span's queries with 32-bit byte offsets.
constexpr int64_t kMaxSpanBytes = int64_t(1) << 31;

// Epoch of a statistics launch's merge marks (never 0): a mark written
// under another epoch counts as unset, so the workspace needs no clearing
// between calls.
uint32_t next_merge_epoch() {
  static std::atomic<uint32_t> epoch{0};
  uint32_t e;
  do e = ++epoch;
  while (e == 0);
  return e;
}

// Whether the column-sum workgroups rebuild the split statistics rows
// themselves (small spans and caches) rather than the statistics kernel
// merging each block once.
bool colsum_fuses_lse(int32_t lse_ns, int64_t n_pair, int32_t n_vis) {
  return lse_ns > 1 && lse_ns <= kLseRegSplits && n_pair <= kColsumMaxLsePairs &&
         (n_vis + kColsumKeysPerBlock - 1) / kColsumKeysPerBlock <= kColsumFuseMaxBlocks;
}

namespace {

thread_local std::string g_last_error;

conduit_status fail(conduit_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

conduit_status hip_fail(hipError_t e, const char *what) {
  return fail(CONDUIT_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

conduit_status ok() {
  g_last_error.clear();
  return CONDUIT_OK;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int esize(int32_t dtype) { return dtype == CONDUIT_BF16 ? 2 : 4; }

conduit_status check_kv(const conduit_kv *kv) {
  if (!kv) return fail(CONDUIT_ERR_INVALID_ARG, "kv is NULL");
  if (kv->dtype != CONDUIT_F32 && kv->dtype != CONDUIT_BF16)
    return fail(CONDUIT_ERR_INVALID_ARG, "kv->dtype %d is not a conduit_dtype", kv->dtype);
  if (!kv->k || !kv->v) return fail(CONDUIT_ERR_INVALID_ARG, "kv->k or kv->v is NULL");
  if (!aligned16(kv->k) || !aligned16(kv->v))
    return fail(CONDUIT_ERR_INVALID_ARG, "kv->k and kv->v must be 16-byte aligned");
  if (kv->n_ctx < 1) return fail(CONDUIT_ERR_INVALID_ARG, "kv->n_ctx = %d < 1", kv->n_ctx);
  if (kv->n_kv_heads < 1 || kv->n_q_heads < 1)
    return fail(CONDUIT_ERR_INVALID_ARG, "head counts must be >= 1");
  if (kv->n_kv_heads > 256)
    return fail(CONDUIT_ERR_UNSUPPORTED, "n_kv_heads %d (supported: up to 256)", kv->n_kv_heads);
  if (kv->n_q_heads % kv->n_kv_heads != 0)
    return fail(CONDUIT_ERR_INVALID_ARG, "n_q_heads %d is not a multiple of n_kv_heads %d",
                kv->n_q_heads, kv->n_kv_heads);
  if (kv->head_dim != 64 && kv->head_dim != 128)
    return fail(CONDUIT_ERR_UNSUPPORTED, "head_dim %d (supported: 64, 128)", kv->head_dim);
  const int64_t row = (int64_t)kv->n_kv_heads * kv->head_dim;
  if (kv->k_stride < row || kv->v_stride < row)
    return fail(CONDUIT_ERR_INVALID_ARG, "token strides (%lld, %lld) below a row of %lld elements",
                (long long)kv->k_stride, (long long)kv->v_stride, (long long)row);
  if ((kv->k_stride * esize(kv->dtype)) % 16 || (kv->v_stride * esize(kv->dtype)) % 16)
    return fail(CONDUIT_ERR_INVALID_ARG, "token strides must be multiples of 16 bytes");
  if (kv->k_stride * esize(kv->dtype) >= kMaxStrideBytes || kv->v_stride * esize(kv->dtype) >= kMaxStrideBytes)
    return fail(CONDUIT_ERR_UNSUPPORTED, "token strides of %lld / %lld bytes (supported: below 32 MiB)",
                (long long)(kv->k_stride * esize(kv->dtype)), (long long)(kv->v_stride * esize(kv->dtype)));
  if (!kv->block_table) {
    if (kv->page_size != 0 || kv->n_pages != 0)
      return fail(CONDUIT_ERR_INVALID_ARG, "page_size and n_pages must be 0 without a block table");
    return CONDUIT_OK;
  }
  const int32_t ps = kv->page_size;
  if (ps < 1 || (ps & (ps - 1)) != 0)
    return fail(CONDUIT_ERR_INVALID_ARG, "page_size %d is not a power of two", ps);
  if (ps < 64 || ps > (1 << 20))
    return fail(CONDUIT_ERR_UNSUPPORTED, "page_size %d (supported: powers of two from 64 to 2^20)", ps);
  if (kv->n_pages < 1) return fail(CONDUIT_ERR_INVALID_ARG, "n_pages = %d < 1", kv->n_pages);
  if (reinterpret_cast<uintptr_t>(kv->block_table) % 4)
    return fail(CONDUIT_ERR_INVALID_ARG, "block_table must be 4-byte aligned");
  return CONDUIT_OK;
}

// Token -> cache row addressing of a checked descriptor.
KvPages pages_of(const conduit_kv *kv) {
  KvPages pg{};
  if (kv->block_table) {
    pg.table = kv->block_table;
    pg.shift = __builtin_ctz((unsigned)kv->page_size);
    pg.n_pages = kv->n_pages;
  }
  return pg;
}

// The image table; `limit` is the first position that may not hold visual tokens.
conduit_status check_images(const conduit_images *img, int64_t limit, ImageTable *tbl) {
  if (!img) return fail(CONDUIT_ERR_INVALID_ARG, "img is NULL");
  if (img->n_images < 1) return fail(CONDUIT_ERR_INVALID_ARG, "n_images = %d < 1", img->n_images);
  if (img->n_images > CONDUIT_MAX_IMAGES)
    return fail(CONDUIT_ERR_UNSUPPORTED, "n_images = %d > %d", img->n_images, CONDUIT_MAX_IMAGES);
  if (!img->img_pos || !img->img_off) return fail(CONDUIT_ERR_INVALID_ARG, "image arrays are NULL");
  const int K = img->n_images;
  if (img->img_off[0] != 0) return fail(CONDUIT_ERR_INVALID_ARG, "img_off[0] must be 0");
  int64_t prev_end = 0;
  for (int j = 0; j < K; ++j) {
    const int64_t n_j = (int64_t)img->img_off[j + 1] - img->img_off[j];
    if (n_j < 1) return fail(CONDUIT_ERR_INVALID_ARG, "image %d is empty or img_off decreases", j);
    if (img->img_pos[j] < prev_end)
      return fail(CONDUIT_ERR_INVALID_ARG, "image %d at position %d overlaps or is out of order", j,
                  img->img_pos[j]);
    prev_end = (int64_t)img->img_pos[j] + n_j;
    if (prev_end > limit)
      return fail(CONDUIT_ERR_INVALID_ARG, "image %d ends at %lld, beyond %lld", j, (long long)prev_end,
                  (long long)limit);
  }
  if (img->n_vis != img->img_off[K])
    return fail(CONDUIT_ERR_INVALID_ARG, "n_vis %d != img_off[n_images] %d", img->n_vis, img->img_off[K]);
  if (tbl) {
    memset(tbl, 0, sizeof(*tbl));
    tbl->n_images = K;
    tbl->n_vis = img->n_vis;
    for (int j = 0; j < K; ++j) tbl->pos[j] = img->img_pos[j];
    for (int j = 0; j <= K; ++j) tbl->off[j] = img->img_off[j];
  }
  return CONDUIT_OK;
}

// Workspace of the bf16 attention plan (see AttnPlan) and its partials.
struct PlanLayout {
  size_t pb_info, pb_base, items, hdr, part_m, part_l, part_o;
  int32_t n_pb, max_items;
};

int64_t attn_blocks(int64_t n_rows, int32_t group, bool with_values) {
  const int64_t ppb = attn_pairs_per_block(with_values);
  return (n_rows * group + ppb - 1) / ppb;
}

template <typename Take>
PlanLayout plan_layout(const conduit_kv *kv, int64_t n_rows, bool with_values, Take &&take, int32_t layers = 1) {
  PlanLayout P{};
  const int32_t group = kv->n_q_heads / kv->n_kv_heads;
  const int64_t n_pb = attn_blocks(n_rows, group, with_values);
  const int64_t max_items = attn_max_items(n_pb, kv->n_kv_heads, with_values);
  const int64_t slots = max_items * attn_pairs_per_block(with_values) * layers;  // layer l's partials l * max_items slots on
  P.n_pb = (int32_t)n_pb;
  P.max_items = (int32_t)max_items;
  P.pb_info = take((size_t)n_pb * 16);
  P.pb_base = take((size_t)n_pb * 4);
  P.items = take((size_t)max_items * 16);
  P.hdr = take(16);
  P.part_m = take((size_t)slots * 4);
  P.part_l = take((size_t)slots * 4);
  P.part_o = take(with_values ? (size_t)slots * kv->head_dim * 2 : 0);  // bf16
  return P;
}

AttnPlan plan_at(void *ws, const PlanLayout &P);
conduit_status check_layers(const conduit_kv *kvs, int32_t n_layers);

struct ScoreLayout {
  size_t row_b, colsum, vsq, done, merge_flag, f32_ml, total;
  PlanLayout plan;
};

// layers: the layers one launch covers (the multi-layer scoring); each has
// its own row LSEs, statistics partials, column sums and norms.
ScoreLayout score_layout(const conduit_kv *kv, int32_t n_q, int32_t n_vis, int32_t layers = 1) {
  ScoreLayout L{};
  const int64_t rows = (int64_t)n_q * kv->n_q_heads;
  const bool bf16 = kv->dtype == CONDUIT_BF16;
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t at = off; off = align_up(off + bytes, 256); return at; };
  L.row_b = take((size_t)rows * 4 * layers);
  if (bf16) L.plan = plan_layout(kv, n_q, false, take, layers);
  L.colsum = take((size_t)kv->n_kv_heads * n_vis * 4 * layers);
  L.vsq = take((size_t)kv->n_kv_heads * n_vis * 4 * layers);
  if (bf16) L.done = take((size_t)(n_vis + kColsumKeysPerBlock - 1) / kColsumKeysPerBlock * 4);
  if (bf16) L.merge_flag = take((size_t)L.plan.max_items * 4 * layers);
  if (!bf16) {  // the fp32 statistics' key splits
    const int32_t ns = f32_attn_splits(n_q, kv->n_q_heads, kv->n_ctx);
    L.f32_ml = ns > 1 ? take((size_t)ns * rows * 8) : 0;
  }
  L.total = off;
  return L;
}

struct RefreshLayout {
  size_t f32_ml, f32_o, total;
  PlanLayout plan;
};

// layers: the layers one attention launch covers (the multi-layer refresh).
// fp32: the key splits' partials, if the rows are split.
RefreshLayout refresh_layout(const conduit_kv *kv, int32_t k, int32_t layers = 1) {
  RefreshLayout L{};
  if (k <= 0) return L;
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t at = off; off = align_up(off + bytes, 256); return at; };
  if (kv->dtype == CONDUIT_BF16) {
    L.plan = plan_layout(kv, k, true, take, layers);
  } else {
    const int32_t ns = f32_attn_splits(k, kv->n_q_heads, kv->n_ctx);
    if (ns > 1) {
      const size_t pairs = (size_t)k * kv->n_q_heads;
      L.f32_ml = take(ns * pairs * 8);
      L.f32_o = take(ns * pairs * kv->head_dim * 4);
    }
  }
  L.total = off;
  return L;
}

// The fp32 attention's outputs, with the key splits' partials in ws when
// f32_attn_splits cuts the rows' keys (ml_off / o_off: their workspace offsets).
DirectOut f32_out(const conduit_kv *kv, int64_t n_rows, float *row_b, float *lse_out, void *o_out, void *ws,
                  size_t ml_off, size_t o_off) {
  DirectOut out{row_b, lse_out, static_cast<float *>(o_out), 1, 0, nullptr, nullptr, 1};
  const int32_t ns = f32_attn_splits(n_rows, kv->n_q_heads, kv->n_ctx);
  if (ns > 1) {
    const int32_t tiles = (kv->n_ctx + 63) / 64;
    out.n_split = ns;
    out.chunk = (tiles + ns - 1) / ns * 64;
    out.part_ml = reinterpret_cast<float2 *>(static_cast<char *>(ws) + ml_off);
    out.part_o = o_out ? reinterpret_cast<float *>(static_cast<char *>(ws) + o_off) : nullptr;
  }
  return out;
}

conduit_status check_ws(const void *ws, size_t ws_bytes, size_t need) {
  if (ws_bytes < need)
    return fail(CONDUIT_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", ws_bytes, need);
  if (need > 0 && (!ws || (reinterpret_cast<uintptr_t>(ws) & 255u)))
    return fail(CONDUIT_ERR_INVALID_ARG, "workspace must be non-NULL and 256-byte aligned");
  return CONDUIT_OK;
}

char *at(void *ws, size_t off) { return static_cast<char *>(ws) + off; }

AttnPlan plan_at(void *ws, const PlanLayout &P) {
  AttnPlan a{};
  a.pb_info = reinterpret_cast<int4 *>(at(ws, P.pb_info));
  a.pb_base = reinterpret_cast<int32_t *>(at(ws, P.pb_base));
  a.items = reinterpret_cast<int4 *>(at(ws, P.items));
  a.hdr = reinterpret_cast<int32_t *>(at(ws, P.hdr));
  a.n_pb = P.n_pb;
  a.max_items = P.max_items;
  return a;
}

// Kernel timing state of one thread.  Events are created on first use and
// kept for the life of the thread (never destroyed: the HIP runtime may be
// gone when thread-local destructors run at exit).
struct ProfRecord {
  const char *name;
  hipEvent_t start, stop;
};
struct ProfState {
  bool enabled = false;
  int count = 0;       // launches recorded
  int created = 0;     // event pairs created
  ProfRecord rec[CONDUIT_PROFILE_MAX];
};
thread_local ProfState *g_prof = nullptr;

}  // namespace

ProfScope::ProfScope(const char *name, hipStream_t s) : slot_(-1), stream_(s) {
  ProfState *st = g_prof;
  if (!st || !st->enabled || st->count >= CONDUIT_PROFILE_MAX) return;
  const int i = st->count;
  if (i >= st->created) {
    if (hipEventCreate(&st->rec[i].start) != hipSuccess) return;
    if (hipEventCreate(&st->rec[i].stop) != hipSuccess) {
      (void)hipEventDestroy(st->rec[i].start);
      return;
    }
    st->created = i + 1;
  }
  if (hipEventRecord(st->rec[i].start, s) != hipSuccess) return;
  st->rec[i].name = name;
  slot_ = i;
  st->count = i + 1;
}

ProfScope::~ProfScope() {
  if (slot_ >= 0) (void)hipEventRecord(g_prof->rec[slot_].stop, stream_);
}

extern "C" {

conduit_status conduit_profile_enable(int32_t enabled) {
  if (!g_prof) {
    if (!enabled) return ok();
    g_prof = new ProfState();
  }
  if (enabled) g_prof->count = 0;
  g_prof->enabled = enabled != 0;
  return ok();
}

int32_t conduit_profile_count(void) { return g_prof ? g_prof->count : 0; }

conduit_status conduit_profile_read(int32_t i, const char **name, float *ms) {
  if (!name || !ms) return fail(CONDUIT_ERR_INVALID_ARG, "name and ms are required");
  if (!g_prof || i < 0 || i >= g_prof->count)
    return fail(CONDUIT_ERR_INVALID_ARG, "launch %d not recorded (%d recorded)", i, conduit_profile_count());
  const ProfRecord &r = g_prof->rec[i];
  hipError_t e = hipEventSynchronize(r.stop);
  if (e != hipSuccess) return hip_fail(e, "profile event");
  e = hipEventElapsedTime(ms, r.start, r.stop);
  if (e != hipSuccess) return hip_fail(e, "profile elapsed time");
  *name = r.name;
  return ok();
}


int64_t conduit_budget(int64_t n_vis, int64_t r_num, int64_t r_den) {
  if (n_vis < 0 || r_den <= 0 || r_num < 0 || r_num > r_den) return -1;
  return (int64_t)(((__int128)r_num * n_vis) / r_den);
}

size_t conduit_score_workspace_bytes(const conduit_kv *kv, int32_t n_q, const conduit_images *img) {
  if (!kv || !img || n_q < 1 || kv->n_kv_heads < 1 || kv->n_q_heads < kv->n_kv_heads || img->n_vis < 1)
    return 0;
  return score_layout(kv, n_q, img->n_vis).total;
}

conduit_status conduit_score(const conduit_kv *kv, const void *q, int32_t n_q, int32_t q_pos0,
                             const conduit_images *img, conduit_norm norm, conduit_agg agg, float scale,
                             const float *row_lse_in, float *row_lse_out, const float *vnorm_in,
                             float *s_acc, float *a_acc, int32_t accumulate, float *a_out, float *vnorm_out,
                             void *ws, size_t ws_bytes, hipStream_t stream) {
  conduit_status st = check_kv(kv);
  if (st) return st;
  if (!q || !aligned16(q)) return fail(CONDUIT_ERR_INVALID_ARG, "q must be non-NULL and 16-byte aligned");
  if (n_q < 1) return fail(CONDUIT_ERR_INVALID_ARG, "n_q = %d < 1", n_q);
  if (q_pos0 < 0 || (int64_t)q_pos0 + n_q > kv->n_ctx)
    return fail(CONDUIT_ERR_INVALID_ARG, "span [%d, %lld) outside the cache of %d tokens", q_pos0,
                (long long)q_pos0 + n_q, kv->n_ctx);
  if (norm != CONDUIT_NORM_CAUSAL_ROW && norm != CONDUIT_NORM_VISUAL_ONLY)
    return fail(CONDUIT_ERR_INVALID_ARG, "norm %d is not a conduit_norm", (int)norm);
  if (agg != CONDUIT_AGG_MEAN && agg != CONDUIT_AGG_RMS)
    return fail(CONDUIT_ERR_INVALID_ARG, "agg %d is not a conduit_agg", (int)agg);
  if (!(scale > 0.f) || scale == __builtin_inff()) return fail(CONDUIT_ERR_INVALID_ARG, "scale must be finite and > 0");
  if (!s_acc || !a_acc) return fail(CONDUIT_ERR_INVALID_ARG, "s_acc and a_acc are required");
  if (accumulate != 0 && accumulate != 1) return fail(CONDUIT_ERR_INVALID_ARG, "accumulate must be 0 or 1");
  ImageTable tbl;
  st = check_images(img, q_pos0, &tbl);
  if (st) return st;
  const bool bf16 = kv->dtype == CONDUIT_BF16;
  if (bf16 && attn_blocks(n_q, kv->n_q_heads / kv->n_kv_heads, false) > kAttnPlanMaxBlocks)
    return fail(CONDUIT_ERR_UNSUPPORTED, "n_q * n_q_heads / n_kv_heads = %lld exceeds %lld",
                (long long)n_q * (kv->n_q_heads / kv->n_kv_heads),
                (long long)kAttnPlanMaxBlocks * attn_pairs_per_block(false));
  if (bf16 && (int64_t)n_q * kv->n_q_heads * kv->head_dim * 2 >= kMaxSpanBytes)
    return fail(CONDUIT_ERR_UNSUPPORTED, "the span's queries (%lld bytes) must stay below 2^31 bytes",
                (long long)n_q * kv->n_q_heads * kv->head_dim * 2);
  const ScoreLayout L = score_layout(kv, n_q, img->n_vis);
  st = check_ws(ws, ws_bytes, L.total);
  if (st) return st;

  const int D = kv->head_dim;
  const float scale_log2 = scale * kLog2e;
  float *row_b = reinterpret_cast<float *>(at(ws, L.row_b));
  const bool vis_only = norm == CONDUIT_NORM_VISUAL_ONLY;

  int32_t lse_ns = 0;
  bool fuse_lse = false;
  DirectOut f32_stats{};  // fp32: the statistics' outputs (key splits merged by the column sums)
  hipError_t e;
  // bf16: the column-sum workgroups count their arrivals per key block and
  // the last one finalizes it; the kernel before them clears the counters.
  int32_t *done = bf16 ? reinterpret_cast<int32_t *>(at(ws, L.done)) : nullptr;
  const int32_t n_done = (img->n_vis + kColsumKeysPerBlock - 1) / kColsumKeysPerBlock;
  if (row_lse_in) {
    e = launch_lse_to_b(row_lse_in, row_b, n_q * kv->n_q_heads, done, bf16 ? n_done : 0, stream);
    if (e != hipSuccess) return hip_fail(e, "lse_to_b");
    if (row_lse_out) {
      e = hipMemcpyAsync(row_lse_out, row_lse_in, (size_t)n_q * kv->n_q_heads * 4, hipMemcpyDeviceToDevice,
                         stream);
      if (e != hipSuccess) return hip_fail(e, "copy row_lse");
    }
  } else {
    AttnParams ap{};
    ap.k = kv->k;
    ap.v = kv->v;
    ap.k_stride = kv->k_stride;
    ap.v_stride = kv->v_stride;
    ap.pages = pages_of(kv);
    ap.n_kv_heads = kv->n_kv_heads;
    ap.group = kv->n_q_heads / kv->n_kv_heads;
    ap.n_q_heads = kv->n_q_heads;
    ap.n_ctx = kv->n_ctx;
    ap.q = q;
    ap.n_rows = n_q;
    ap.row_pos = nullptr;
    ap.q_pos0 = q_pos0;
    ap.vis_only = vis_only ? 1 : 0;
    ap.tbl = tbl;
    ap.scale_log2 = scale_log2;
    ap.row_b = row_b;
    ap.lse_out = row_lse_out;
    if (bf16) {
      ap.plan = plan_at(ws, L.plan);
      ap.part_m = reinterpret_cast<float *>(at(ws, L.plan.part_m));
      ap.part_l = reinterpret_cast<float *>(at(ws, L.plan.part_l));
      // split rows: merged by the column-sum workgroups, or else by the
      // statistics kernel's last split of each block (no merge launch)
      lse_ns = attn_span_splits(ap, attn_pairs_per_block(false), 1);
      fuse_lse = colsum_fuses_lse(lse_ns, (int64_t)n_q * ap.group, img->n_vis);
      if (!fuse_lse) {
        ap.merge_flag = reinterpret_cast<uint32_t *>(at(ws, L.merge_flag));
        ap.epoch = next_merge_epoch();
      }
      ap.skip_merge = 1;
      ap.zero_i32 = done;
      ap.zero_n = n_done;
      e = launch_attn(ap, D, false, stream);
      if (e != hipSuccess) return hip_fail(e, "row statistics");
    } else {
      // split rows are merged by the column sums (below), not by a launch
      f32_stats = f32_out(kv, n_q, row_b, row_lse_out, nullptr, ws, L.f32_ml, 0);
      f32_stats.merge = 0;
      e = launch_attn_f32(ap, f32_stats, D, false, stream);
      if (e != hipSuccess) return hip_fail(e, "row statistics");
    }
  }

  ColsumParams cs{};
  cs.k = kv->k;
  cs.v = kv->v;
  cs.k_stride = kv->k_stride;
  cs.v_stride = kv->v_stride;
  cs.pages = pages_of(kv);
  cs.n_kv_heads = kv->n_kv_heads;
  cs.group = kv->n_q_heads / kv->n_kv_heads;
  cs.n_q_heads = kv->n_q_heads;
  cs.q = q;
  cs.n_q = n_q;
  cs.row_b = row_b;
  cs.tbl = tbl;
  cs.n_vis = img->n_vis;
  cs.scale_log2 = scale_log2;
  cs.colsum_part = reinterpret_cast<float *>(at(ws, L.colsum));
  cs.vsq_part = reinterpret_cast<float *>(at(ws, L.vsq));
  cs.vnorm_in = vnorm_in;

  FinalizeParams fp{};
  fp.colsum_part = cs.colsum_part;
  fp.vsq_part = cs.vsq_part;
  fp.vnorm_in = vnorm_in;
  fp.rms = agg == CONDUIT_AGG_RMS;
  fp.n_kv_heads = kv->n_kv_heads;
  fp.n_vis = img->n_vis;
  fp.n_rows_f = (float)((int64_t)n_q * kv->n_q_heads);
  fp.accumulate = accumulate;
  fp.s_acc = s_acc;
  fp.a_acc = a_acc;
  fp.a_out = a_out;
  fp.vnorm_out = vnorm_out;

  if (f32_stats.n_split > 1) {
    cs.f32_ml = f32_stats.part_ml;
    cs.lse_ns = f32_stats.n_split;
    cs.lse_out = row_lse_out;
  }
  if (fuse_lse) {
    cs.lse_part_m = reinterpret_cast<float *>(at(ws, L.plan.part_m));
    cs.lse_part_l = reinterpret_cast<float *>(at(ws, L.plan.part_l));
    cs.lse_ns = lse_ns;
    cs.lse_ppb = attn_pairs_per_block(false);
    cs.lse_out = row_lse_out;
  }
  cs.done = done;
  cs.fin = fp;
  e = launch_colsum(cs, D, bf16, agg == CONDUIT_AGG_RMS, stream);
  if (e != hipSuccess) return hip_fail(e, "column sums");
  if (!done) {
    e = launch_finalize(fp, stream);
    if (e != hipSuccess) return hip_fail(e, "finalize");
  }
  return ok();
}

size_t conduit_score_layers_workspace_bytes(const conduit_kv *kv, int32_t n_q, const conduit_images *img,
                                           int32_t n_layers) {
  if (n_layers < 1 || n_layers > CONDUIT_MAX_LAYERS) return 0;
  const size_t one = conduit_score_workspace_bytes(kv, n_q, img);
  if (one == 0 || n_layers == 1 || kv->dtype != CONDUIT_BF16) return one;
  return score_layout(kv, n_q, img->n_vis, std::min<int32_t>(n_layers, kMaxLayerBatch)).total;
}

conduit_status conduit_score_layers(const conduit_kv *kvs, int32_t n_layers, const void *const *q, int32_t n_q,
                                    int32_t q_pos0, const conduit_images *img, conduit_norm norm,
                                    conduit_agg agg, float scale, const float *const *vnorm_in, float *s_acc,
                                    float *a_acc, int32_t accumulate, void *ws, size_t ws_bytes,
                                    hipStream_t stream) {
  conduit_status st = check_layers(kvs, n_layers);
  if (st) return st;
  const conduit_kv *kv = &kvs[0];
  if (!q) return fail(CONDUIT_ERR_INVALID_ARG, "q is NULL");
  for (int32_t l = 0; l < n_layers; ++l)
    if (!q[l] || !aligned16(q[l])) return fail(CONDUIT_ERR_INVALID_ARG, "q[%d] must be non-NULL and 16-byte aligned", l);
  if (n_q < 1) return fail(CONDUIT_ERR_INVALID_ARG, "n_q = %d < 1", n_q);
  if (q_pos0 < 0 || (int64_t)q_pos0 + n_q > kv->n_ctx)
    return fail(CONDUIT_ERR_INVALID_ARG, "span [%d, %lld) outside the cache of %d tokens", q_pos0,
                (long long)q_pos0 + n_q, kv->n_ctx);
  if (norm != CONDUIT_NORM_CAUSAL_ROW && norm != CONDUIT_NORM_VISUAL_ONLY)
    return fail(CONDUIT_ERR_INVALID_ARG, "norm %d is not a conduit_norm", (int)norm);
  if (agg != CONDUIT_AGG_MEAN && agg != CONDUIT_AGG_RMS)
    return fail(CONDUIT_ERR_INVALID_ARG, "agg %d is not a conduit_agg", (int)agg);
  if (!(scale > 0.f) || scale == __builtin_inff()) return fail(CONDUIT_ERR_INVALID_ARG, "scale must be finite and > 0");
  if (!s_acc || !a_acc) return fail(CONDUIT_ERR_INVALID_ARG, "s_acc and a_acc are required");
  if (accumulate != 0 && accumulate != 1) return fail(CONDUIT_ERR_INVALID_ARG, "accumulate must be 0 or 1");
  ImageTable tbl;
  st = check_images(img, q_pos0, &tbl);
  if (st) return st;
  const bool bf16 = kv->dtype == CONDUIT_BF16;
  if (n_layers == 1 || !bf16) {  // fp32 (or one layer): the per-layer calls
    const size_t need = conduit_score_workspace_bytes(kv, n_q, img);
    st = check_ws(ws, ws_bytes, need);
    if (st) return st;
    for (int32_t l = 0; l < n_layers; ++l) {
      st = conduit_score(&kvs[l], q[l], n_q, q_pos0, img, norm, agg, scale, nullptr, nullptr,
                         vnorm_in ? vnorm_in[l] : nullptr, s_acc, a_acc, l > 0 ? 1 : accumulate, nullptr, nullptr, ws,
                         ws_bytes, stream);
      if (st) return st;
    }
    return ok();
  }
  if (attn_blocks(n_q, kv->n_q_heads / kv->n_kv_heads, false) > kAttnPlanMaxBlocks)
    return fail(CONDUIT_ERR_UNSUPPORTED, "n_q * n_q_heads / n_kv_heads = %lld exceeds %lld",
                (long long)n_q * (kv->n_q_heads / kv->n_kv_heads),
                (long long)kAttnPlanMaxBlocks * attn_pairs_per_block(false));
  if ((int64_t)n_q * kv->n_q_heads * kv->head_dim * 2 >= kMaxSpanBytes)
    return fail(CONDUIT_ERR_UNSUPPORTED, "the span's queries (%lld bytes) must stay below 2^31 bytes",
                (long long)n_q * kv->n_q_heads * kv->head_dim * 2);
  const int32_t nb_max = std::min<int32_t>(n_layers, kMaxLayerBatch);
  const ScoreLayout L = score_layout(kv, n_q, img->n_vis, nb_max);
  st = check_ws(ws, ws_bytes, L.total);
  if (st) return st;

  const int D = kv->head_dim;
  const int64_t rows = (int64_t)n_q * kv->n_q_heads;
  const float scale_log2 = scale * kLog2e;
  float *row_b = reinterpret_cast<float *>(at(ws, L.row_b));
  int32_t *done = reinterpret_cast<int32_t *>(at(ws, L.done));
  const int32_t n_done = (img->n_vis + kColsumKeysPerBlock - 1) / kColsumKeysPerBlock;

  AttnParams ap{};
  ap.k = kv->k;
  ap.v = kv->v;
  ap.k_stride = kv->k_stride;
  ap.v_stride = kv->v_stride;
  ap.pages = pages_of(kv);
  ap.n_kv_heads = kv->n_kv_heads;
  ap.group = kv->n_q_heads / kv->n_kv_heads;
  ap.n_q_heads = kv->n_q_heads;
  ap.n_ctx = kv->n_ctx;
  ap.q = q[0];
  ap.n_rows = n_q;
  ap.q_pos0 = q_pos0;
  ap.vis_only = norm == CONDUIT_NORM_VISUAL_ONLY ? 1 : 0;
  ap.tbl = tbl;
  ap.scale_log2 = scale_log2;
  ap.plan = plan_at(ws, L.plan);
  ap.part_m = reinterpret_cast<float *>(at(ws, L.plan.part_m));
  ap.part_l = reinterpret_cast<float *>(at(ws, L.plan.part_l));
  ap.skip_merge = 1;  // merged by the column sums or by the statistics kernel (split count per launch, below)
  ap.zero_i32 = done;
  ap.zero_n = n_done;

  ColsumParams cs{};
  cs.k = kv->k;
  cs.v = kv->v;
  cs.k_stride = kv->k_stride;
  cs.v_stride = kv->v_stride;
  cs.pages = pages_of(kv);
  cs.n_kv_heads = kv->n_kv_heads;
  cs.group = ap.group;
  cs.n_q_heads = kv->n_q_heads;
  cs.q = q[0];
  cs.n_q = n_q;
  cs.row_b = row_b;
  cs.tbl = tbl;
  cs.n_vis = img->n_vis;
  cs.scale_log2 = scale_log2;
  cs.colsum_part = reinterpret_cast<float *>(at(ws, L.colsum));
  cs.vsq_part = reinterpret_cast<float *>(at(ws, L.vsq));
  cs.done = done;
  FinalizeParams fp{};
  fp.colsum_part = cs.colsum_part;
  fp.vsq_part = cs.vsq_part;
  fp.rms = agg == CONDUIT_AGG_RMS;
  fp.n_kv_heads = kv->n_kv_heads;
  fp.n_vis = img->n_vis;
  fp.n_rows_f = (float)rows;
  fp.s_acc = s_acc;
  fp.a_acc = a_acc;

  // Per batch of up to 16 layers: one statistics launch (which also clears
  // the finalize counters and merges its split rows) and one column-sum launch whose last workgroup per
  // key block finalizes the batch's layers in order onto s_acc and A.
  for (int32_t l0 = 0; l0 < n_layers; l0 += kMaxLayerBatch) {
    LayerTable lt{};
    lt.n = std::min<int32_t>(kMaxLayerBatch, n_layers - l0);
    for (int32_t i = 0; i < lt.n; ++i) {
      lt.k[i] = kvs[l0 + i].k;
      lt.v[i] = kvs[l0 + i].v;
      lt.q[i] = q[l0 + i];
      lt.rowb[i] = row_b + i * rows;
      lt.vnorm[i] = vnorm_in ? vnorm_in[l0 + i] : nullptr;
    }
    // The statistics' split count depends on the launch's layer count; the
    // column sums rebuild the split rows themselves when they can, otherwise
    // the statistics kernel merges them (each launch marks afresh).
    const int32_t lse_ns = attn_span_splits(ap, attn_pairs_per_block(false), lt.n);
    const bool fuse_lse = colsum_fuses_lse(lse_ns, (int64_t)n_q * ap.group, img->n_vis);
    ap.merge_flag = fuse_lse ? nullptr : reinterpret_cast<uint32_t *>(at(ws, L.merge_flag));
    if (!fuse_lse) ap.epoch = next_merge_epoch();
    cs.lse_part_m = fuse_lse ? ap.part_m : nullptr;
    cs.lse_part_l = fuse_lse ? ap.part_l : nullptr;
    cs.lse_ns = fuse_lse ? lse_ns : 0;
    cs.lse_ppb = fuse_lse ? attn_pairs_per_block(false) : 0;
    cs.lse_layer_stride = fuse_lse ? (int64_t)L.plan.max_items * attn_pairs_per_block(false) : 0;
    hipError_t e = launch_attn(ap, D, false, stream, &lt);
    if (e != hipSuccess) return hip_fail(e, "row statistics");
    fp.accumulate = (l0 > 0 || accumulate) ? 1 : 0;
    cs.fin = fp;
    e = launch_colsum(cs, D, true, agg == CONDUIT_AGG_RMS, stream, &lt);
    if (e != hipSuccess) return hip_fail(e, "column sums");
  }
  return ok();
}

conduit_status conduit_score_noalloc(const conduit_kv *kv, const void *q, int32_t n_q, int32_t q_pos0,
                                     const conduit_images *img, conduit_norm norm, conduit_agg agg, float scale,
                                     const float *row_lse_in, float *row_lse_out, const float *vnorm_in,
                                     float *s_acc, float *a_acc, int32_t accumulate, float *a_out,
                                     float *vnorm_out, hipStream_t stream) {
  static_assert(kStaticScoreScratchBytes == CONDUIT_SCORE_NOALLOC_MAX_BYTES, "scratch size");
  // A size query of 0 means an argument conduit_score rejects on its own
  // (a valid call always needs scratch, so with none it cannot pass the
  // checks); otherwise the call must fit the fixed scratch.
  const size_t need = conduit_score_workspace_bytes(kv, n_q, img);
  if (need == 0)
    return conduit_score(kv, q, n_q, q_pos0, img, norm, agg, scale, row_lse_in, row_lse_out, vnorm_in, s_acc,
                         a_acc, accumulate, a_out, vnorm_out, nullptr, 0, stream);
  if (need > kStaticScoreScratchBytes)
    return fail(CONDUIT_ERR_UNSUPPORTED,
                "this scoring call needs %zu bytes of scratch; conduit_score_noalloc holds at most %zu "
                "(use conduit_score with a caller workspace)",
                need, kStaticScoreScratchBytes);
  void *scratch = nullptr;
  const hipError_t e = static_score_scratch(&scratch);
  if (e != hipSuccess) return hip_fail(e, "static scratch address");
  return conduit_score(kv, q, n_q, q_pos0, img, norm, agg, scale, row_lse_in, row_lse_out, vnorm_in, s_acc, a_acc,
                       accumulate, a_out, vnorm_out, scratch, kStaticScoreScratchBytes, stream);
}

conduit_status conduit_value_norms(const conduit_kv *kv, const conduit_images *img, float *vnorm_out,
                                   hipStream_t stream) {
  conduit_status st = check_kv(kv);
  if (st) return st;
  if (!vnorm_out) return fail(CONDUIT_ERR_INVALID_ARG, "vnorm_out is NULL");
  ImageTable tbl;
  st = check_images(img, kv->n_ctx, &tbl);
  if (st) return st;
  hipError_t e = launch_value_norms(kv->v, kv->v_stride, pages_of(kv), kv->n_kv_heads * kv->head_dim,
                                    kv->dtype == CONDUIT_BF16, tbl, vnorm_out, stream);
  if (e != hipSuccess) return hip_fail(e, "value norms");
  return ok();
}

namespace {

struct ResidualLayout {
  size_t row_b, vnorm, part, total;
  int32_t n_splits, tiles_per_split, pairs_pad;
};

ResidualLayout residual_layout(const conduit_kv *kv, int32_t n_q, int32_t n_vis, int32_t n_samples, bool iso) {
  ResidualLayout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t at = off; off = align_up(off + bytes, 256); return at; };
  L.row_b = take((size_t)n_q * kv->n_q_heads * 4);
  if (iso) L.vnorm = take((size_t)n_vis * 4);
  if (kv->dtype == CONDUIT_BF16) {
    const int64_t pairs = (int64_t)n_q * (kv->n_q_heads / kv->n_kv_heads);
    const int64_t n_pb = (pairs + kResidualPairs - 1) / kResidualPairs;
    const int tiles = (n_vis + kAttnKeyTile - 1) / kAttnKeyTile;
    const int64_t base = n_pb * kv->n_kv_heads * n_samples;
    int splits = (int)std::min<int64_t>((kResidualTargetBlocks + base - 1) / base,
                                        std::max(1, tiles / kResidualMinTiles));
    splits = std::max(splits, (tiles + kResidualMaxTiles - 1) / kResidualMaxTiles);
    splits = std::max(1, splits);
    L.tiles_per_split = (tiles + splits - 1) / splits;
    L.n_splits = (tiles + L.tiles_per_split - 1) / L.tiles_per_split;
    L.pairs_pad = (int32_t)(n_pb * kResidualPairs);
    L.part = take((size_t)n_samples * L.n_splits * kv->n_kv_heads * L.pairs_pad * kv->head_dim * 4);
  }
  L.total = off;
  return L;
}

}  // namespace

size_t conduit_residual_workspace_bytes(const conduit_kv *kv, int32_t n_q, const conduit_images *img,
                                        int32_t n_samples, int32_t iso) {
  if (!kv || !img || n_q < 1 || n_samples < 1 || kv->n_kv_heads < 1 || kv->n_q_heads < kv->n_kv_heads ||
      img->n_vis < 1 || (kv->head_dim != 64 && kv->head_dim != 128))
    return 0;
  return residual_layout(kv, n_q, img->n_vis, n_samples, iso != 0).total;
}

conduit_status conduit_residual_error(const conduit_kv *kv, const void *q, int32_t n_q, int32_t q_pos0,
                                      const conduit_images *img, float scale, const float *row_lse_in,
                                      const uint8_t *refreshed, const void *z, int32_t n_samples, float kappa,
                                      float *err_out, void *ws, size_t ws_bytes, hipStream_t stream) {
  conduit_status st = check_kv(kv);
  if (st) return st;
  if (!q || !aligned16(q)) return fail(CONDUIT_ERR_INVALID_ARG, "q must be non-NULL and 16-byte aligned");
  if (n_q < 1) return fail(CONDUIT_ERR_INVALID_ARG, "n_q = %d < 1", n_q);
  if (q_pos0 < 0 || (int64_t)q_pos0 + n_q > kv->n_ctx)
    return fail(CONDUIT_ERR_INVALID_ARG, "span [%d, %lld) outside the cache of %d tokens", q_pos0,
                (long long)q_pos0 + n_q, kv->n_ctx);
  if (!(scale > 0.f) || scale == __builtin_inff()) return fail(CONDUIT_ERR_INVALID_ARG, "scale must be finite and > 0");
  if (!row_lse_in) return fail(CONDUIT_ERR_INVALID_ARG, "row_lse_in is required (conduit_score's row_lse_out)");
  if (!refreshed) return fail(CONDUIT_ERR_INVALID_ARG, "refreshed is required");
  if (!err_out) return fail(CONDUIT_ERR_INVALID_ARG, "err_out is required");
  const bool iso = z != nullptr;
  if (iso) {
    if (!aligned16(z)) return fail(CONDUIT_ERR_INVALID_ARG, "z must be 16-byte aligned");
    if (n_samples < 1) return fail(CONDUIT_ERR_INVALID_ARG, "n_samples = %d < 1", n_samples);
    if (!(kappa > 0.f) || kappa == __builtin_inff())
      return fail(CONDUIT_ERR_INVALID_ARG, "kappa must be finite and > 0");
  } else if (n_samples != 1) {
    return fail(CONDUIT_ERR_INVALID_ARG, "the projected error (z = NULL) takes n_samples = 1");
  }
  if ((int64_t)n_samples * kv->n_kv_heads > 65535)
    return fail(CONDUIT_ERR_UNSUPPORTED, "n_samples * n_kv_heads = %lld > 65535",
                (long long)n_samples * kv->n_kv_heads);
  if ((int64_t)n_samples * n_q * kv->n_q_heads > INT32_MAX)
    return fail(CONDUIT_ERR_UNSUPPORTED, "n_samples * n_q * n_q_heads exceeds 2^31 - 1");
  ImageTable tbl;
  st = check_images(img, q_pos0, &tbl);
  if (st) return st;
  const ResidualLayout L = residual_layout(kv, n_q, img->n_vis, n_samples, iso);
  st = check_ws(ws, ws_bytes, L.total);
  if (st) return st;
  char *w = static_cast<char *>(ws);
  const bool bf16 = kv->dtype == CONDUIT_BF16;
  ResidualParams rp{};
  rp.k = kv->k;
  rp.k_stride = kv->k_stride;
  rp.pages = pages_of(kv);
  rp.disp = iso ? z : kv->v;
  rp.disp_stride = kv->v_stride;
  rp.vnorm = iso ? reinterpret_cast<float *>(w + L.vnorm) : nullptr;
  rp.sigma_scale = iso ? kappa / sqrtf((float)(kv->n_kv_heads * kv->head_dim)) : 1.f;
  rp.refreshed = refreshed;
  rp.q = q;
  rp.n_q = n_q;
  rp.n_q_heads = kv->n_q_heads;
  rp.n_kv_heads = kv->n_kv_heads;
  rp.group = kv->n_q_heads / kv->n_kv_heads;
  rp.n_vis = img->n_vis;
  rp.n_samples = n_samples;
  rp.row_b = reinterpret_cast<float *>(w + L.row_b);
  rp.scale_log2 = scale * kLog2e;
  rp.tbl = tbl;
  rp.n_splits = L.n_splits;
  rp.tiles_per_split = L.tiles_per_split;
  rp.pairs_pad = L.pairs_pad;
  rp.part = bf16 ? reinterpret_cast<float *>(w + L.part) : nullptr;
  rp.err_out = err_out;
  hipError_t e = launch_lse_to_b(row_lse_in, reinterpret_cast<float *>(w + L.row_b), n_q * kv->n_q_heads, nullptr, 0,
                                 stream);
  if (e != hipSuccess) return hip_fail(e, "row statistics");
  if (iso) {
    e = launch_value_norms(kv->v, kv->v_stride, pages_of(kv), kv->n_kv_heads * kv->head_dim, bf16, tbl,
                           reinterpret_cast<float *>(w + L.vnorm), stream);
    if (e != hipSuccess) return hip_fail(e, "value norms");
  }
  e = launch_residual(rp, kv->head_dim, bf16, stream);
  if (e != hipSuccess) return hip_fail(e, "residual error");
  return ok();
}

namespace {
// Workspace of conduit_select_topk: the exchange area of the multi-workgroup
// top-k (when n_vis uses it), then s_hat when the caller keeps none.
size_t select_ws_need(int32_t n_vis, bool with_shat) {
  if (n_vis < 1) return 0;
  const size_t multi = select_uses_multi(n_vis) ? select_multi_layout().total : 0;
  return multi + (with_shat ? 0 : align_up((size_t)n_vis * 4, 256));
}
}  // namespace

size_t conduit_select_workspace_bytes(int32_t n_vis, int32_t n_images) {
  (void)n_images;
  return select_ws_need(n_vis, false);
}

conduit_status conduit_select_topk(const float *s_acc, const float *a_acc, int32_t n_layers,
                                   const conduit_images *img, float lambda, conduit_rule rule, int32_t k,
                                   int32_t *idx_out, int32_t *pos_out, uint8_t *mask_out, float *shat_out,
                                   float *c_out, int32_t *quota_out, void *ws, size_t ws_bytes,
                                   hipStream_t stream) {
  if (!s_acc || !a_acc) return fail(CONDUIT_ERR_INVALID_ARG, "s_acc and a_acc are required");
  if (n_layers < 1) return fail(CONDUIT_ERR_INVALID_ARG, "n_layers = %d < 1", n_layers);
  if (!(lambda >= 0.f && lambda <= 1.f)) return fail(CONDUIT_ERR_INVALID_ARG, "lambda must lie in [0, 1]");
  if (rule != CONDUIT_RANK_COMPOSITE && rule != CONDUIT_RANK_ATTENTION && rule != CONDUIT_RANK_EXPLICIT)
    return fail(CONDUIT_ERR_INVALID_ARG, "rule %d is not a conduit_rule", (int)rule);
  conduit_status st = check_images(img, INT32_MAX, nullptr);
  if (st) return st;
  ImageTable tbl;
  check_images(img, INT32_MAX, &tbl);
  if (k < 0 || k > img->n_vis) return fail(CONDUIT_ERR_INVALID_ARG, "k = %d outside [0, n_vis = %d]", k, img->n_vis);
  if (k > 0 && (!idx_out || !pos_out)) return fail(CONDUIT_ERR_INVALID_ARG, "idx_out and pos_out are required");
  const size_t need = select_ws_need(img->n_vis, shat_out != nullptr);
  if (k > 0) {
    st = check_ws(ws, ws_bytes, need);
    if (st) return st;
  }
  hipError_t e;
  if (k == 0) {  // Algorithm 1 early exit: the all-zero mask
    if (mask_out) {
      e = launch_clear_u8(mask_out, img->n_vis, stream);
      if (e != hipSuccess) return hip_fail(e, "clear mask");
    }
    if (rule == CONDUIT_RANK_EXPLICIT && quota_out) {
      e = launch_clear_u8(reinterpret_cast<uint8_t *>(quota_out), (int64_t)img->n_images * 4, stream);
      if (e != hipSuccess) return hip_fail(e, "clear quotas");
    }
    return ok();
  }
  SelectParams sp{};
  // The attention-only rule ranks A where the composite ranks s (Table 5's drop-value-norm ablation).
  sp.s_acc = rule == CONDUIT_RANK_ATTENTION ? a_acc : s_acc;
  sp.a_acc = a_acc;
  sp.n_layers = n_layers;
  sp.lambda = lambda;
  sp.k = k;
  sp.idx_out = idx_out;
  sp.pos_out = pos_out;
  sp.mask_out = mask_out;
  const size_t multi = select_uses_multi(img->n_vis) ? select_multi_layout().total : 0;
  sp.multi = multi ? ws : nullptr;
  sp.shat = shat_out ? shat_out : reinterpret_cast<float *>(static_cast<char *>(ws) + multi);
  sp.c_out = c_out;
  sp.quota_out = quota_out;
  e = rule == CONDUIT_RANK_EXPLICIT ? launch_select_explicit(sp, tbl, stream) : launch_select(sp, tbl, stream);
  if (e != hipSuccess) return hip_fail(e, "select");
  return ok();
}

namespace {

ScatterParams scatter_params(const conduit_kv *kv, const int32_t *pos, int32_t k, const void *k_new,
                             const void *v_new, void *k_old_out, void *v_old_out) {
  ScatterParams sp{};
  sp.k = kv->k;
  sp.v = kv->v;
  sp.k_stride_bytes = kv->k_stride * esize(kv->dtype);
  sp.v_stride_bytes = kv->v_stride * esize(kv->dtype);
  sp.pages = pages_of(kv);
  sp.n_ctx = kv->n_ctx;
  sp.row_bytes = kv->n_kv_heads * kv->head_dim * esize(kv->dtype);
  sp.pos = pos;
  sp.n_rows = k;
  sp.k_new = k_new;
  sp.v_new = v_new;
  sp.k_old = k_old_out;
  sp.v_old = v_old_out;
  return sp;
}

// Checks of a refresh of k rows (k > 0) and its workspace.
conduit_status check_refresh(const conduit_kv *kv, const void *q_sel, const int32_t *pos, int32_t k,
                             void *o_out, void *ws, size_t ws_bytes) {
  if (!pos) return fail(CONDUIT_ERR_INVALID_ARG, "pos is NULL");
  if (!q_sel || !aligned16(q_sel) || !o_out || !aligned16(o_out))
    return fail(CONDUIT_ERR_INVALID_ARG, "q_sel and o_out must be non-NULL and 16-byte aligned");
  if (kv->dtype == CONDUIT_BF16 && attn_blocks(k, kv->n_q_heads / kv->n_kv_heads, true) > kAttnPlanMaxBlocks)
    return fail(CONDUIT_ERR_UNSUPPORTED, "k * n_q_heads / n_kv_heads = %lld exceeds %lld",
                (long long)k * (kv->n_q_heads / kv->n_kv_heads),
                (long long)kAttnPlanMaxBlocks * attn_pairs_per_block(true));
  return check_ws(ws, ws_bytes, refresh_layout(kv, k).total);
}

// Refresh attention of the rows at pos (the plan and partials in ws for bf16).
AttnParams refresh_params(const conduit_kv *kv, const void *q_sel, const int32_t *pos, int32_t k, float scale,
                          void *o_out, float *lse_out, void *ws) {
  AttnParams ap{};
  ap.k = kv->k;
  ap.v = kv->v;
  ap.k_stride = kv->k_stride;
  ap.v_stride = kv->v_stride;
  ap.pages = pages_of(kv);
  ap.n_kv_heads = kv->n_kv_heads;
  ap.group = kv->n_q_heads / kv->n_kv_heads;
  ap.n_q_heads = kv->n_q_heads;
  ap.n_ctx = kv->n_ctx;
  ap.q = q_sel;
  ap.n_rows = k;
  ap.row_pos = pos;
  ap.q_pos0 = 0;
  ap.vis_only = 0;
  ap.scale_log2 = scale * kLog2e;
  ap.lse_out = lse_out;
  ap.o_out = o_out;
  if (kv->dtype == CONDUIT_BF16) {
    const RefreshLayout L = refresh_layout(kv, k);
    ap.plan = plan_at(ws, L.plan);
    ap.part_m = reinterpret_cast<float *>(at(ws, L.plan.part_m));
    ap.part_l = reinterpret_cast<float *>(at(ws, L.plan.part_l));
    ap.part_o = reinterpret_cast<u16 *>(at(ws, L.plan.part_o));
  }
  return ap;
}

}  // namespace

conduit_status conduit_scatter_kv(const conduit_kv *kv, const int32_t *pos, int32_t k, const void *k_new,
                                  const void *v_new, void *k_old_out, void *v_old_out, hipStream_t stream) {
  conduit_status st = check_kv(kv);
  if (st) return st;
  if (k < 0 || k > kv->n_ctx) return fail(CONDUIT_ERR_INVALID_ARG, "k = %d outside [0, n_ctx]", k);
  if (k == 0) return ok();
  if (!pos) return fail(CONDUIT_ERR_INVALID_ARG, "pos is NULL");
  if (!k_new || !v_new || !aligned16(k_new) || !aligned16(v_new))
    return fail(CONDUIT_ERR_INVALID_ARG, "k_new and v_new must be non-NULL and 16-byte aligned");
  if ((k_old_out && !aligned16(k_old_out)) || (v_old_out && !aligned16(v_old_out)))
    return fail(CONDUIT_ERR_INVALID_ARG, "k_old_out and v_old_out must be 16-byte aligned");
  const ScatterParams sp = scatter_params(kv, pos, k, k_new, v_new, k_old_out, v_old_out);
  hipError_t e = launch_scatter(sp, stream);
  if (e != hipSuccess) return hip_fail(e, "scatter");
  return ok();
}

size_t conduit_refresh_workspace_bytes(const conduit_kv *kv, int32_t k) {
  if (!kv || k < 1 || kv->n_kv_heads < 1 || kv->n_q_heads < kv->n_kv_heads || kv->n_ctx < 1) return 0;
  if (kv->head_dim != 64 && kv->head_dim != 128) return 0;
  return refresh_layout(kv, k).total;
}

conduit_status conduit_refresh_attn(const conduit_kv *kv, const void *q_sel, const int32_t *pos, int32_t k,
                                    float scale, void *o_out, float *lse_out, void *ws, size_t ws_bytes,
                                    hipStream_t stream) {
  conduit_status st = check_kv(kv);
  if (st) return st;
  if (k < 0 || k > kv->n_ctx) return fail(CONDUIT_ERR_INVALID_ARG, "k = %d outside [0, n_ctx]", k);
  if (!(scale > 0.f) || scale == __builtin_inff()) return fail(CONDUIT_ERR_INVALID_ARG, "scale must be finite and > 0");
  if (k == 0) return ok();
  st = check_refresh(kv, q_sel, pos, k, o_out, ws, ws_bytes);
  if (st) return st;
  const AttnParams ap = refresh_params(kv, q_sel, pos, k, scale, o_out, lse_out, ws);
  hipError_t e;
  if (kv->dtype == CONDUIT_BF16) {
    e = launch_attn(ap, kv->head_dim, true, stream);
  } else {
    const RefreshLayout L = refresh_layout(kv, k);
    const DirectOut out = f32_out(kv, k, nullptr, lse_out, o_out, ws, L.f32_ml, L.f32_o);
    e = launch_attn_f32(ap, out, kv->head_dim, true, stream);
  }
  if (e != hipSuccess) return hip_fail(e, "refresh attention");
  return ok();
}

conduit_status conduit_merge_refresh_attn(const conduit_kv *kv, const int32_t *pos, int32_t k, const void *k_new,
                                          const void *v_new, const void *q_sel, float scale, void *o_out,
                                          float *lse_out, void *ws, size_t ws_bytes, hipStream_t stream) {
  conduit_status st = check_kv(kv);
  if (st) return st;
  if (k < 0 || k > kv->n_ctx) return fail(CONDUIT_ERR_INVALID_ARG, "k = %d outside [0, n_ctx]", k);
  if (!(scale > 0.f) || scale == __builtin_inff()) return fail(CONDUIT_ERR_INVALID_ARG, "scale must be finite and > 0");
  if (k == 0) return ok();
  if (!k_new || !v_new || !aligned16(k_new) || !aligned16(v_new))
    return fail(CONDUIT_ERR_INVALID_ARG, "k_new and v_new must be non-NULL and 16-byte aligned");
  st = check_refresh(kv, q_sel, pos, k, o_out, ws, ws_bytes);
  if (st) return st;
  const ScatterParams sp = scatter_params(kv, pos, k, k_new, v_new, nullptr, nullptr);
  const AttnParams ap = refresh_params(kv, q_sel, pos, k, scale, o_out, lse_out, ws);
  hipError_t e;
  if (kv->dtype == CONDUIT_BF16) {
    e = launch_merge_refresh(ap, sp, kv->head_dim, stream);
  } else {
    e = launch_scatter(sp, stream);
    if (e == hipSuccess) {
      const RefreshLayout L = refresh_layout(kv, k);
      const DirectOut out = f32_out(kv, k, nullptr, lse_out, o_out, ws, L.f32_ml, L.f32_o);
      e = launch_attn_f32(ap, out, kv->head_dim, true, stream);
    }
  }
  if (e != hipSuccess) return hip_fail(e, "merge and refresh attention");
  return ok();
}

namespace {

// The layers of one request: every descriptor valid and shaped like kvs[0]
// (only the k and v pointers may differ).
conduit_status check_layers(const conduit_kv *kvs, int32_t n_layers) {
  if (!kvs) return fail(CONDUIT_ERR_INVALID_ARG, "kvs is NULL");
  if (n_layers < 1 || n_layers > CONDUIT_MAX_LAYERS)
    return fail(CONDUIT_ERR_INVALID_ARG, "n_layers = %d outside [1, %d]", n_layers, CONDUIT_MAX_LAYERS);
  for (int32_t l = 0; l < n_layers; ++l) {
    const conduit_status st = check_kv(&kvs[l]);
    if (st) return st;
    const conduit_kv &a = kvs[0], &b = kvs[l];
    if (a.dtype != b.dtype || a.n_kv_heads != b.n_kv_heads || a.n_q_heads != b.n_q_heads ||
        a.head_dim != b.head_dim || a.n_ctx != b.n_ctx || a.k_stride != b.k_stride || a.v_stride != b.v_stride ||
        a.block_table != b.block_table || a.page_size != b.page_size || a.n_pages != b.n_pages)
      return fail(CONDUIT_ERR_INVALID_ARG, "layer %d's cache is not shaped like layer 0's", l);
  }
  return CONDUIT_OK;
}

conduit_status check_layer_ptrs(const void *const *ptrs, int32_t n_layers, const char *what, bool nullable) {
  if (!ptrs) return nullable ? CONDUIT_OK : fail(CONDUIT_ERR_INVALID_ARG, "%s is NULL", what);
  for (int32_t l = 0; l < n_layers; ++l) {
    if (!ptrs[l] && nullable) continue;
    if (!ptrs[l] || !aligned16(ptrs[l]))
      return fail(CONDUIT_ERR_INVALID_ARG, "%s[%d] must be non-NULL and 16-byte aligned", what, l);
  }
  return CONDUIT_OK;
}

}  // namespace

conduit_status conduit_scatter_kv_layers(const conduit_kv *kvs, int32_t n_layers, const int32_t *pos, int32_t k,
                                         const void *const *k_new, const void *const *v_new, hipStream_t stream) {
  conduit_status st = check_layers(kvs, n_layers);
  if (st) return st;
  const conduit_kv *kv = &kvs[0];
  if (k < 0 || k > kv->n_ctx) return fail(CONDUIT_ERR_INVALID_ARG, "k = %d outside [0, n_ctx]", k);
  if (k == 0) return ok();
  if (!pos) return fail(CONDUIT_ERR_INVALID_ARG, "pos is NULL");
  st = check_layer_ptrs(k_new, n_layers, "k_new", false);
  if (st) return st;
  st = check_layer_ptrs(v_new, n_layers, "v_new", false);
  if (st) return st;
  ScatterParams sp{};
  sp.k_stride_bytes = kv->k_stride * esize(kv->dtype);
  sp.v_stride_bytes = kv->v_stride * esize(kv->dtype);
  sp.pages = pages_of(kv);
  sp.n_ctx = kv->n_ctx;
  sp.row_bytes = kv->n_kv_heads * kv->head_dim * esize(kv->dtype);
  sp.pos = pos;
  sp.n_rows = k;
  for (int32_t l0 = 0; l0 < n_layers; l0 += kMaxLayerBatch) {
    ScatterLayers sl{};
    sl.n = std::min<int32_t>(kMaxLayerBatch, n_layers - l0);
    for (int32_t i = 0; i < sl.n; ++i) {
      sl.k[i] = kvs[l0 + i].k;
      sl.v[i] = kvs[l0 + i].v;
      sl.k_new[i] = k_new[l0 + i];
      sl.v_new[i] = v_new[l0 + i];
    }
    const hipError_t e = launch_scatter_layers(sp, sl, stream);
    if (e != hipSuccess) return hip_fail(e, "scatter");
  }
  return ok();
}

size_t conduit_refresh_layers_workspace_bytes(const conduit_kv *kv, int32_t k, int32_t n_layers) {
  if (n_layers < 1 || n_layers > CONDUIT_MAX_LAYERS) return 0;
  const size_t one = conduit_refresh_workspace_bytes(kv, k);
  if (one == 0 || n_layers == 1) return one;
  return refresh_layout(kv, k, std::min<int32_t>(n_layers, kMaxLayerBatch)).total;
}

conduit_status conduit_refresh_attn_layers(const conduit_kv *kvs, int32_t n_layers, const void *const *q_sel,
                                           const int32_t *pos, int32_t k, float scale, void *const *o_out,
                                           float *const *lse_out, void *ws, size_t ws_bytes, hipStream_t stream) {
  conduit_status st = check_layers(kvs, n_layers);
  if (st) return st;
  const conduit_kv *kv = &kvs[0];
  if (k < 0 || k > kv->n_ctx) return fail(CONDUIT_ERR_INVALID_ARG, "k = %d outside [0, n_ctx]", k);
  if (!(scale > 0.f) || scale == __builtin_inff()) return fail(CONDUIT_ERR_INVALID_ARG, "scale must be finite and > 0");
  if (k == 0) return ok();
  if (!pos) return fail(CONDUIT_ERR_INVALID_ARG, "pos is NULL");
  st = check_layer_ptrs(q_sel, n_layers, "q_sel", false);
  if (st) return st;
  st = check_layer_ptrs(reinterpret_cast<const void *const *>(o_out), n_layers, "o_out", false);
  if (st) return st;
  if (n_layers == 1)
    return conduit_refresh_attn(kv, q_sel[0], pos, k, scale, o_out[0], lse_out ? lse_out[0] : nullptr, ws, ws_bytes,
                                stream);
  if (kv->dtype == CONDUIT_BF16 && attn_blocks(k, kv->n_q_heads / kv->n_kv_heads, true) > kAttnPlanMaxBlocks)
    return fail(CONDUIT_ERR_UNSUPPORTED, "k * n_q_heads / n_kv_heads = %lld exceeds %lld",
                (long long)k * (kv->n_q_heads / kv->n_kv_heads),
                (long long)kAttnPlanMaxBlocks * attn_pairs_per_block(true));
  const RefreshLayout L = refresh_layout(kv, k, std::min<int32_t>(n_layers, kMaxLayerBatch));
  st = check_ws(ws, ws_bytes, L.total);
  if (st) return st;
  if (kv->dtype != CONDUIT_BF16) {  // fp32: the per-layer calls, one after the other on the workspace
    for (int32_t l = 0; l < n_layers; ++l) {
      st = conduit_refresh_attn(&kvs[l], q_sel[l], pos, k, scale, o_out[l], lse_out ? lse_out[l] : nullptr, ws,
                                ws_bytes, stream);
      if (st) return st;
    }
    return ok();
  }
  AttnParams ap{};
  ap.k = kv->k;
  ap.v = kv->v;
  ap.k_stride = kv->k_stride;
  ap.v_stride = kv->v_stride;
  ap.pages = pages_of(kv);
  ap.n_kv_heads = kv->n_kv_heads;
  ap.group = kv->n_q_heads / kv->n_kv_heads;
  ap.n_q_heads = kv->n_q_heads;
  ap.n_ctx = kv->n_ctx;
  ap.q = q_sel[0];
  ap.n_rows = k;
  ap.row_pos = pos;
  ap.scale_log2 = scale * kLog2e;
  ap.o_out = o_out[0];
  ap.plan = plan_at(ws, L.plan);
  ap.part_m = reinterpret_cast<float *>(at(ws, L.plan.part_m));
  ap.part_l = reinterpret_cast<float *>(at(ws, L.plan.part_l));
  ap.part_o = reinterpret_cast<u16 *>(at(ws, L.plan.part_o));
  // One plan (it depends on the rows only), then one attention and one
  // merge launch per kMaxLayerBatch layers.
  for (int32_t l0 = 0; l0 < n_layers; l0 += kMaxLayerBatch) {
    LayerTable lt{};
    lt.n = std::min<int32_t>(kMaxLayerBatch, n_layers - l0);
    for (int32_t i = 0; i < lt.n; ++i) {
      lt.k[i] = kvs[l0 + i].k;
      lt.v[i] = kvs[l0 + i].v;
      lt.q[i] = q_sel[l0 + i];
      lt.o[i] = o_out[l0 + i];
      lt.lse[i] = lse_out ? lse_out[l0 + i] : nullptr;
    }
    const hipError_t e = launch_attn(ap, kv->head_dim, true, stream, &lt, l0 > 0);
    if (e != hipSuccess) return hip_fail(e, "refresh attention");
  }
  return ok();
}

const char *conduit_status_str(conduit_status status) {
  switch (status) {
    case CONDUIT_OK: return "CONDUIT_OK";
    case CONDUIT_ERR_INVALID_ARG: return "CONDUIT_ERR_INVALID_ARG";
    case CONDUIT_ERR_UNSUPPORTED: return "CONDUIT_ERR_UNSUPPORTED";
    case CONDUIT_ERR_WORKSPACE: return "CONDUIT_ERR_WORKSPACE";
    case CONDUIT_ERR_HIP: return "CONDUIT_ERR_HIP";
  }
  return "CONDUIT_ERR_UNKNOWN";
}

const char *conduit_last_error(void) { return g_last_error.c_str(); }

const char *conduit_version(void) { return "conduit-gfx950 0.1.0"; }

}  // extern "C"
