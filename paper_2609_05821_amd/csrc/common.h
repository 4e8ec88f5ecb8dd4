// Internal declarations shared by the HIP kernels and the host layer of
// libconduit (gfx950 only).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace conduit {

typedef uint16_t u16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));  // 16-byte register moves
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kMaxImages = 256;

// Image table passed by value in kernel arguments (2 KB).
struct ImageTable {
  int32_t n_images;
  int32_t n_vis;
  int32_t pos[kMaxImages];      // first sequence position of image j
  int32_t off[kMaxImages + 1];  // visual-index offsets
};

// The image table staged in LDS by a workgroup, for per-key lookups.
struct ImageLds {
  int32_t n_images;
  int32_t pos[kMaxImages];
  int32_t off[kMaxImages + 1];
};

// Cooperative copy of the table into LDS; the caller synchronises after it.
__device__ __forceinline__ void image_table_to_lds(const ImageTable &t, ImageLds &s, int tid, int nthreads) {
  const int n = t.n_images;
  for (int j = tid; j <= n; j += nthreads) {
    s.off[j] = t.off[j];
    if (j < n) s.pos[j] = t.pos[j];
  }
  if (tid == 0) s.n_images = n;
}

// Sequence position of visual index t (0 <= t < n_vis): image j is the last
// one with off[j] <= t.  T is ImageLds or ImageTable.
template <typename T>
__device__ __forceinline__ int vis_position(const T &s, int t) {
  int lo = 0, hi = s.n_images - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (s.off[mid] <= t) lo = mid;
    else hi = mid - 1;
  }
  return s.pos[lo] + (t - s.off[lo]);
}

// Whether sequence position q holds a visual token.
template <typename T>
__device__ __forceinline__ bool is_visual(const T &s, int q) {
  int lo = 0, hi = s.n_images - 1;  // last image with pos[j] <= q
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (s.pos[mid] <= q) lo = mid;
    else hi = mid - 1;
  }
  return q >= s.pos[lo] && q < s.pos[lo] + (s.off[lo + 1] - s.off[lo]);
}

// ---------------------------------------------------------------------------
// Device helpers
// ---------------------------------------------------------------------------
__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

template <typename T>
__device__ __forceinline__ u32x4 ld16(const T *p) { return *reinterpret_cast<const u32x4 *>(p); }
template <typename T>
__device__ __forceinline__ void st16(T *p, u32x4 v) { *reinterpret_cast<u32x4 *>(p) = v; }

__device__ __forceinline__ float bf16_to_f32(u16 b) {
  return __builtin_bit_cast(float, static_cast<uint32_t>(b) << 16);
}

// fp32 -> bf16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ u16 f32_to_bf16(float f) {
  return __builtin_bit_cast(u16, static_cast<__bf16>(f));
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Maximum of a value and its partner lane (lane ^ 32), in every lane:
// v_permlane32_swap exchanges the two 32-lane halves.
__device__ __forceinline__ float half_max(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__builtin_bit_cast(float, (uint32_t)r[0]), __builtin_bit_cast(float, (uint32_t)r[1]));
}

__device__ __forceinline__ float half_sum(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __builtin_bit_cast(float, (uint32_t)r[0]) + __builtin_bit_cast(float, (uint32_t)r[1]);
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}

// Cache row of a token.  A paged cache keeps token t in row
// table[t >> shift] * 2^shift + (t mod 2^shift) of its page pool; without a
// table the row is t.  Table entries are clamped into the pool, so a bad
// entry cannot send an access outside it.
struct KvPages {
  const int32_t *table;     // nullable: contiguous cache
  int32_t shift;            // log2 of the page size
  int32_t n_pages;          // pages in the pool
};

__device__ __forceinline__ int64_t kv_row(const KvPages &pg, int t) {
  if (!pg.table) return t;
  const int page = min(max(pg.table[t >> pg.shift], 0), pg.n_pages - 1);
  return ((int64_t)page << pg.shift) | (t & ((1 << pg.shift) - 1));
}

// Block-table reads for pipelined loops: a buffer load returns 0 for a read
// past the resource's record count instead of touching memory, so the read is
// unconditional (no branch, hence no early wait on every load in flight).  A
// contiguous cache gets 0 records and a 31-bit in-page mask, so the row is the
// token itself.
// gfx9 raw buffer resource, word 3: 32-bit data format, no swizzle.
constexpr int kRawBufferWord3 = 0x00020000;

// Buffer resource over `bytes` bytes from p: loads address it with 32-bit
// per-lane byte offsets (one VGPR each, the base stays scalar), and a read
// past the end returns 0 instead of touching memory.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void *p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, bytes, kRawBufferWord3);
}

__device__ __forceinline__ u32x4 buffer_ld16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

struct KvPageReader {
  __amdgpu_buffer_rsrc_t rsrc;
  int32_t shift;
  int32_t last_page;
};

__device__ __forceinline__ KvPageReader page_reader(const KvPages &pg, int n_ctx) {
  KvPageReader r;
  if (pg.table) {
    const int entries = ((n_ctx - 1) >> pg.shift) + 1;
    r.rsrc = buffer_rsrc(pg.table, entries * 4);
    r.shift = pg.shift;
    r.last_page = pg.n_pages - 1;
  } else {
    r.rsrc = buffer_rsrc(nullptr, 0);
    r.shift = 31;
    r.last_page = 0;
  }
  return r;
}

// Page entry of token t (raw; 0 past the table).
__device__ __forceinline__ int read_page(const KvPageReader &r, int t) {
  return __builtin_amdgcn_raw_buffer_load_b32(r.rsrc, (t >> r.shift) * 4, 0, 0);
}

// Cache row of token t from its raw page entry.
__device__ __forceinline__ int64_t page_row(const KvPageReader &r, int page, int t) {
  const int pg = min(max(page, 0), r.last_page);
  return ((int64_t)pg << r.shift) | (int64_t)((uint32_t)t & ((1u << r.shift) - 1u));
}

// The A operand of O^T += V^T P^T for one 16-key MFMA step, read from the
// row-major V tile with two transposing LDS reads (ds_read_b64_tr_b16): in
// each group of 16 lanes, lane 4j + q reads 4 head dims of key j and lane
// 4q + r receives dim 4q + r of keys 0..3.  Lane (m, h) of the wave ends up
// with keys 4h + 0..3 and 8 + 4h + 0..3 of the step for head dim m, the
// order in which the S^T accumulator holds them (so P needs no shuffle).
typedef short short4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) short4 lds_short4;

typedef short short8 __attribute__((ext_vector_type(8)));

// Element offset, inside a V tile with row stride VS, of the 4 dims this
// lane reads for the first half of an MFMA step (keys 0..7); the second
// half (keys 8..15) is 8 rows further.
template <int VS>
__device__ __forceinline__ int v_operand_lane_offset(int lane) {
  const int s = lane & 15, h = lane >> 5, dgrp = (lane >> 4) & 1;
  return (4 * h + (s >> 2)) * VS + 16 * dgrp + 4 * (s & 3);
}

template <int VS>
__device__ __forceinline__ bf16x8 v_operand(const u16 *at) {
  const short4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4 *)(at));
  const short4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4 *)(at + 8 * VS));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Interleaved V tile: key 8a + 4b + c of every 16-key block (a, b in {0, 1},
// c in 0..3) is stored in row 8b + 2c + a of the block.  The four rows that
// one 32-lane half of a transposing read touches are then two rows apart, so
// with a row stride of 8 (mod 32) dwords they start 16 banks apart and cover
// the 64 banks once (with the plain order every bank is hit twice).  The
// operand registers are the same as with the plain order.
__device__ __forceinline__ int v_interleaved_key(int row16) {
  return 8 * (row16 & 1) + 4 * ((row16 >> 3) & 1) + ((row16 >> 1) & 3);
}

template <int VS>
__device__ __forceinline__ int v_operand_lane_offset_il(int lane) {
  const int s = lane & 15, h = lane >> 5, dgrp = (lane >> 4) & 1;
  return (8 * h + 2 * (s >> 2)) * VS + 16 * dgrp + 4 * (s & 3);
}

template <int VS>
__device__ __forceinline__ bf16x8 v_operand_il(const u16 *at) {
  const short4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4 *)(at));
  const short4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4 *)(at + VS));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Wave-wide reductions and scans through DPP lane moves (no LDS round trip,
// unlike a shuffle).
template <int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t old, uint32_t x) {
  // lanes whose source is outside the row, or whose row is masked off, keep `old`
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)x, CTRL, ROW_MASK, 0xf, false);
}
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;  // lane i <- lane 7-i within 8
constexpr int kDppMirror = 0x140;      // lane i <- lane 15-i within 16
constexpr int kDppBcast15 = 0x142;     // lane 15 of each row -> the next row
constexpr int kDppBcast31 = 0x143;     // lane 31 -> rows 2 and 3
constexpr int kDppShr1 = 0x111;        // row_shr:n = 0x110 + n

// Reduction of one value per lane with an associative, commutative op of
// identity `id`; the result is uniform.  Fixed order: quads, eights,
// sixteens, then the four rows into lane 63.
template <class Op>
__device__ __forceinline__ uint32_t wave_reduce(uint32_t x, uint32_t id, Op op) {
  x = op(x, dpp_mov<kDppXor1>(id, x));
  x = op(x, dpp_mov<kDppXor2>(id, x));
  x = op(x, dpp_mov<kDppHalfMirror>(id, x));
  x = op(x, dpp_mov<kDppMirror>(id, x));
  x = op(x, dpp_mov<kDppBcast15, 0xA>(id, x));
  x = op(x, dpp_mov<kDppBcast31, 0xC>(id, x));
  return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}
__device__ __forceinline__ float wave_fsum(float x) {
  return __builtin_bit_cast(float, wave_reduce(__builtin_bit_cast(uint32_t, x), 0u, [](uint32_t a, uint32_t b) {
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b));
  }));
}
// Inclusive prefix sum over the wave (modulo 2^32).
__device__ __forceinline__ uint32_t wave_inclusive_sum(uint32_t x) {
  x += dpp_mov<kDppShr1>(0u, x);
  x += dpp_mov<kDppShr1 + 1>(0u, x);
  x += dpp_mov<kDppShr1 + 3>(0u, x);
  x += dpp_mov<kDppShr1 + 7>(0u, x);
  x += dpp_mov<kDppBcast15, 0xA>(0u, x);
  x += dpp_mov<kDppBcast31, 0xC>(0u, x);
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// ---------------------------------------------------------------------------
// Kernel parameter blocks
// ---------------------------------------------------------------------------

// Causal attention of a set of query rows against one layer's cache.  Used for
// the row statistics of the scoring pass (no values) and for the refresh
// attention of the selected rows (with values).
// Work plan of the bf16 attention, built on the device from the row
// positions (attn_plan_kernel).  A block is `ppb` consecutive (row, head)
// pairs of one KV head; its causal key range [0, maxpos] is cut into n_s
// near-equal splits of `chunk` keys.  An item is one (KV head, block, split);
// items are listed largest first and each has a partial slot.
struct AttnPlan {
  int4 *pb_info;            // [n_pb] {maxpos, minpos, n_s, chunk}
  int32_t *pb_base;         // [n_pb] slot of split 0 for KV head 0
  int4 *items;              // [max_items] {kv head, block, split, slot}
  int32_t *hdr;             // {n_items, slots per KV head}
  int32_t n_pb;
  int32_t max_items;
  // Rows at q_pos0 + r (the scoring span): the plan is closed-form instead,
  // every block cut into uniform_ns near-equal splits, item i = (block,
  // KV head, split) = ((block * n_kv_heads + head) * uniform_ns + split),
  // its own partial slot.  0 = the device-built plan above.
  int32_t uniform_ns;
  int32_t uniform_items;
};

// Causal attention of a set of query rows against one layer's cache.  Used for
// the row statistics of the scoring pass (no values) and for the refresh
// attention of the selected rows (with values).
struct AttnParams {
  const void *k;
  const void *v;
  int64_t k_stride;         // elements between cache rows
  int64_t v_stride;
  KvPages pages;            // token -> cache row (pages hold >= 64 rows)
  int32_t n_kv_heads;
  int32_t group;            // n_q_heads / n_kv_heads
  int32_t n_q_heads;
  int32_t n_ctx;
  const void *q;            // [n_rows][n_q_heads][D]
  int32_t n_rows;
  const int32_t *row_pos;   // nullable: row r sits at q_pos0 + r
  int32_t q_pos0;
  int32_t vis_only;         // statistics only: keys restricted to visual tokens (tbl)
  float scale_log2;         // logit scale * log2(e)
  AttnPlan plan;            // bf16 path
  float *part_m;            // [max_items][ppb] running max (log2 units)
  float *part_l;            // [max_items][ppb] softmax denominator
  u16 *part_o;              // [max_items][ppb][D] bf16: the split's output O_s / l_s (values only)
  // Final outputs, written directly by blocks whose keys form one split.
  float *row_b;             // nullable [n_rows * H_q]: log2-domain log-sum-exp
  float *lse_out;           // nullable [n_rows * H_q]: natural-log log-sum-exp
  void *o_out;              // [n_rows][H_q][D] bf16 (values only)
  ImageTable tbl;           // read when vis_only
  int32_t skip_merge;       // host side: no merge launch (merged in the kernel, or by the caller)
  int32_t *zero_i32;        // nullable: cleared by the kernel (counters of a later kernel)
  int32_t zero_n;
  // Statistics with the closed-form plan (nullable): one mark per partial
  // slot, set to the call's epoch by the item that wrote the slot; the item
  // that finds every split of its block marked merges the block into
  // row_b / lse_out.  Marks of another epoch count as unset, so they need no
  // clearing.
  uint32_t *merge_flag;
  uint32_t epoch;
};

// Per-layer pointers of a launch that covers several layers of one request
// (the same rows, shapes and plan in every layer).  n = 0: one layer, the
// pointers of the parameter block are used.  Split partials of layer l sit
// l * max_items slots further on.
constexpr int kMaxLayerBatch = 16;
struct LayerTable {
  const void *k[kMaxLayerBatch];
  const void *v[kMaxLayerBatch];
  const void *q[kMaxLayerBatch];
  void *o[kMaxLayerBatch];           // refresh outputs
  float *lse[kMaxLayerBatch];        // nullable: natural-log LSE outputs
  float *rowb[kMaxLayerBatch];       // nullable: log2-domain row LSE (statistics)
  const float *vnorm[kMaxLayerBatch];  // nullable: value-norm tables (column sums)
  int32_t n;
};

// Device-coherent store of a partial (written through to where every XCD
// reads it), so that a later workgroup of the same kernel can read it with
// device-scope loads, without a device-scope cache write-back.
__device__ __forceinline__ void store_coherent(float *q, float v) {
  __hip_atomic_store(q, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Entry l of one of a LayerTable's pointer arrays, as a chain of selects.  An
// index that is not a compile-time constant into an array of a kernel
// parameter makes the compiler copy the whole parameter to per-lane scratch
// memory (2 KB per lane here, reloaded all through the kernel).
template <class T>
__device__ __forceinline__ T layer_entry(T const (&a)[kMaxLayerBatch], int l) {
  T r = a[0];
#pragma unroll
  for (int i = 1; i < kMaxLayerBatch; ++i) r = l == i ? a[i] : r;
  return r;
}

// Merge of split partials into final outputs (blocks with n_s > 1).
struct CombineParams {
  int32_t n_rows;
  int32_t n_q_heads;
  int32_t group;
  int32_t ppb;
  AttnPlan plan;
  const float *part_m;
  const float *part_l;
  const u16 *part_o;        // nullable (statistics only): bf16 O_s / l_s
  float *row_b;             // nullable [n_rows * H_q]: log2-domain log-sum-exp
  float *lse_out;           // nullable [n_rows * H_q]: natural-log log-sum-exp
  void *o_out;              // nullable [n_rows][H_q][D] bf16
};

// Outputs of the fp32 path.  With n_split > 1 each (row, head) pair's key
// range is cut into n_split ranges of `chunk` keys (whole tiles), processed by
// separate workgroups that write partials (part_ml: [n_split][pairs] of
// {m, l}; part_o: [n_split][pairs][D], unnormalised), merged by a second
// launch into the outputs.
struct DirectOut {
  float *row_b;
  float *lse_out;
  float *o_out;
  int32_t n_split;
  int32_t chunk;
  float2 *part_ml;
  float *part_o;
  int32_t merge;  // 0: the partials are merged by the caller's next kernel
};
// Key splits of the fp32 attention for n_rows rows of n_q_heads heads over a
// cache of n_ctx keys: enough workgroups to cover the chip about twice (four
// rows per workgroup), at least two tiles per split, at most 8 splits.
constexpr int kF32RowsPerBlock = 4;
inline int32_t f32_attn_splits(int64_t n_rows, int32_t n_q_heads, int32_t n_ctx) {
  const int64_t blocks = (n_rows + kF32RowsPerBlock - 1) / kF32RowsPerBlock * n_q_heads;
  const int64_t tiles = ((int64_t)n_ctx + 63) / 64;
  int64_t ns = (512 + blocks - 1) / blocks;
  ns = ns < 8 ? ns : 8;
  ns = ns < tiles / 2 ? ns : tiles / 2;
  return (int32_t)(ns > 1 ? ns : 1);
}


struct FinalizeParams {
  const float *colsum_part;
  const float *vsq_part;
  const float *vnorm_in;    // nullable: value norms given
  int32_t n_kv_heads;
  int32_t n_vis;
  float n_rows_f;           // n_q * n_q_heads, as float
  int32_t rms;              // a = sqrt(colsum / n_rows) (Eq. 4) instead of the mean
  int32_t accumulate;
  float *s_acc;
  float *a_acc;
  float *a_out;             // nullable
  float *vnorm_out;         // nullable
};

struct ColsumParams {
  const void *k;
  const void *v;
  int64_t k_stride;
  int64_t v_stride;
  KvPages pages;
  int32_t n_kv_heads;
  int32_t group;
  int32_t n_q_heads;
  const void *q;            // [n_q][n_q_heads][D]
  int32_t n_q;
  const float *row_b;       // [n_q * n_q_heads] log2-domain log-sum-exp
  ImageTable tbl;           // visual index -> sequence position
  int32_t n_vis;
  float scale_log2;
  float *colsum_part;       // [n_kv_heads][n_vis]: sum of alpha (or alpha^2 for RMS)
  float *vsq_part;          // [n_kv_heads][n_vis]
  const float *vnorm_in;    // nullable: value norms given, V not read
  // Row log-sum-exp rebuilt from the statistics pass's split partials (its
  // closed-form plan: lse_ns <= kLseRegSplits splits of lse_ppb-pair blocks)
  // instead of read from row_b; the first key block also writes lse_out
  // (natural log).
  const float *lse_part_m;
  const float *lse_part_l;
  int32_t lse_ns;
  int32_t lse_ppb;
  float *lse_out;
  int64_t lse_layer_stride;  // several layers: statistics partial slots per layer
  // fp32: the statistics' key splits ({m, l} per pair, lse_ns of them),
  // merged here instead of read from row_b (the first key block writes
  // lse_out).
  const float2 *f32_ml;
  // nullable: arrival counters, one per key block, cleared beforehand; the
  // last KV head's workgroup of a key block finalizes its keys (fin).
  int32_t *done;
  FinalizeParams fin;
};

struct SelectParams {
  const float *s_acc;
  const float *a_acc;
  int32_t n_layers;
  float lambda;
  int32_t k;
  int32_t *idx_out;
  int32_t *pos_out;
  uint8_t *mask_out;        // nullable
  float *shat;              // [n_vis]: caller's shat_out or workspace
  float *c_out;             // nullable
  int32_t *quota_out;       // nullable (explicit rule)
  void *multi;              // exchange area of the multi-workgroup top-k (select_multi_bytes)
};

// Multi-workgroup top-k: kSelMultiKeys visual tokens per workgroup (1024
// threads x 4), between kSelSingleMax + 1 and kSelMultiMaxWg * kSelMultiKeys
// tokens.  Its exchange area holds the arrival flags of the grid barriers,
// the per-workgroup image partial sums and digit histograms.
constexpr int kSelMultiKeys = 4096;
constexpr int kSelMultiMaxWg = 32;
constexpr int kSelMultiBarriers = 3;  // one after each of the three digit passes
constexpr int kSelDigitBins = 2048;
struct SelectMultiLayout {
  size_t flags, gpart, ghist, total;
};
constexpr SelectMultiLayout select_multi_layout() {
  SelectMultiLayout L{};
  L.flags = 0;
  L.gpart = 256 * ((kSelMultiBarriers * kSelMultiMaxWg * 4 + 255) / 256);
  L.ghist = L.gpart + 256 * (((kSelMultiMaxWg + kMaxImages) * 4 + 255) / 256);
  L.total = L.ghist + (size_t)3 * kSelMultiMaxWg * kSelDigitBins * 4;
  return L;
}
constexpr int kSelSingleMax = 16384;  // one workgroup up to here
constexpr bool select_uses_multi(int n_vis) {
  return n_vis > kSelSingleMax && n_vis <= kSelMultiMaxWg * kSelMultiKeys;
}

struct ScatterParams {
  void *k;
  void *v;
  int64_t k_stride_bytes;
  int64_t v_stride_bytes;
  KvPages pages;
  int32_t n_ctx;            // positions are clamped to [0, n_ctx)
  int32_t row_bytes;        // n_kv_heads * head_dim * element size
  const int32_t *pos;
  int32_t n_rows;
  const void *k_new;
  const void *v_new;
  void *k_old;              // nullable
  void *v_old;              // nullable
};

// One selected row of the cache merge, by one wave: 16-byte chunks of its K
// and V (after copying the stale ones out, when asked).
__device__ __forceinline__ void scatter_row(const ScatterParams &p, int row, int lane) {
  const int64_t pos = kv_row(p.pages, min(max(p.pos[row], 0), p.n_ctx - 1));  // cache row
  const int nch = p.row_bytes / 16;
  char *kdst = static_cast<char *>(p.k) + pos * p.k_stride_bytes;
  char *vdst = static_cast<char *>(p.v) + pos * p.v_stride_bytes;
  const char *ksrc = static_cast<const char *>(p.k_new) + (int64_t)row * p.row_bytes;
  const char *vsrc = static_cast<const char *>(p.v_new) + (int64_t)row * p.row_bytes;
  for (int c = lane; c < nch; c += 64) {
    const u32x4 kn = ld16(ksrc + 16 * c);
    const u32x4 vn = ld16(vsrc + 16 * c);
    if (p.k_old) st16(static_cast<char *>(p.k_old) + (int64_t)row * p.row_bytes + 16 * c, ld16(kdst + 16 * c));
    if (p.v_old) st16(static_cast<char *>(p.v_old) + (int64_t)row * p.row_bytes + 16 * c, ld16(vdst + 16 * c));
    st16(kdst + 16 * c, kn);
    st16(vdst + 16 * c, vn);
  }
}

// Per-layer cache and fresh-row pointers of a multi-layer merge.
struct ScatterLayers {
  void *k[kMaxLayerBatch];
  void *v[kMaxLayerBatch];
  const void *k_new[kMaxLayerBatch];
  const void *v_new[kMaxLayerBatch];
  int32_t n;
};

// Residual value-write error of a refresh set: for each displacement sample
// m and (span row, query head) pair, || sum over non-refreshed visual t of
// alpha_t xi_t ||^2 with alpha from the row's known log-sum-exp.  The bf16
// path writes per-split partial sums of the residual vector, which a second
// kernel adds in split order and squares.
struct ResidualParams {
  const void *k;
  int64_t k_stride;
  KvPages pages;
  const void *disp;         // iso: z [M][n_vis][H_kv][D]; projected: the V cache
  int64_t disp_stride;      // projected: elements between V cache rows
  const float *vnorm;       // iso: ||V_t|| [n_vis]; projected: nullptr
  float sigma_scale;        // iso: kappa / sqrt(H_kv * D)
  const uint8_t *refreshed; // [n_vis]: 1 = in the refresh set (left out)
  const void *q;            // [n_q][n_q_heads][D]
  int32_t n_q;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t group;
  int32_t n_vis;
  int32_t n_samples;
  const float *row_b;       // [n_q * n_q_heads] log2-domain log-sum-exp
  float scale_log2;
  ImageTable tbl;
  int32_t n_splits;         // bf16: key splits
  int32_t tiles_per_split;  // bf16: 64-key tiles per split
  int32_t pairs_pad;        // bf16: pair slots per KV head (blocks of 256)
  float *part;              // bf16: [M][n_splits][n_kv_heads][pairs_pad][D]
  float *err_out;           // [M][n_q][n_q_heads]
};

// Brackets one kernel launch with HIP events when kernel timing is enabled
// on the calling thread (conduit_profile_enable); otherwise does nothing.
class ProfScope {
 public:
  ProfScope(const char *name, hipStream_t s);
  ~ProfScope();
  ProfScope(const ProfScope &) = delete;
  ProfScope &operator=(const ProfScope &) = delete;

 private:
  int slot_;
  hipStream_t stream_;
};

// ---------------------------------------------------------------------------
// Launchers (host side, defined next to their kernels).  Each returns the
// status of the launch.
// ---------------------------------------------------------------------------
// bf16 attention: plan, persistent attention over the plan's items, merge.
// lt (nullable): several layers in one launch of each kernel; plan_ready:
// the device plan was built by an earlier call on the same rows and
// workspace, so no plan launch.
hipError_t launch_attn(const AttnParams &p, int head_dim, bool with_values, hipStream_t s,
                       const LayerTable *lt = nullptr, bool plan_ready = false);
hipError_t launch_attn_f32(const AttnParams &p, const DirectOut &out, int head_dim,
                           bool with_values, hipStream_t s);
// lse_in (natural log) to the log2 domain; also clears zero_i32[0, zero_n).
hipError_t launch_lse_to_b(const float *lse_in, float *row_b, int32_t n, int32_t *zero_i32, int32_t zero_n,
                           hipStream_t s);
// Split count of the closed-form plan the statistics pass uses for rows at
// q_pos0 + r (pairs per block ppb), as launch_attn picks it.
int attn_uniform_splits(const AttnParams &p, int ppb, int target);
// Split count of the scoring span's statistics for `layers` layers in one
// launch (attn_uniform_splits' count for one).
int attn_span_splits(const AttnParams &p, int ppb, int layers);
// lt (nullable, bf16 only): several layers in one launch (grid z = layer).
hipError_t launch_colsum(const ColsumParams &p, int head_dim, bool bf16, bool rms, hipStream_t s,
                         const LayerTable *lt = nullptr);
hipError_t launch_value_norms(const void *v, int64_t v_stride, const KvPages &pages, int32_t row_elems,
                              bool bf16, const ImageTable &tbl, float *out, hipStream_t s);
hipError_t launch_finalize(const FinalizeParams &p, hipStream_t s);
hipError_t launch_select(const SelectParams &p, const ImageTable &tbl, hipStream_t s);
hipError_t launch_select_explicit(const SelectParams &p, const ImageTable &tbl, hipStream_t s);
hipError_t launch_clear_u8(uint8_t *p, int64_t n, hipStream_t s);
hipError_t launch_scatter(const ScatterParams &p, hipStream_t s);
// Cache merge of the rows and their refresh attention (bf16): the plan and the
// merge in one launch, then the attention and the split merge.
hipError_t launch_merge_refresh(const AttnParams &p, const ScatterParams &sp, int head_dim, hipStream_t s);
hipError_t launch_scatter_layers(const ScatterParams &p, const ScatterLayers &sl, hipStream_t s);
hipError_t launch_residual(const ResidualParams &p, int head_dim, bool bf16, hipStream_t s);

// Size of the fixed device scratch behind conduit_score_noalloc (must equal
// CONDUIT_SCORE_NOALLOC_MAX_BYTES of conduit.h).
constexpr size_t kStaticScoreScratchBytes = size_t(16) << 20;
// Device address of that scratch on the current device, resolved with
// hipGetSymbolAddress on the first call per device and kept.
hipError_t static_score_scratch(void **out);

// Residual-error tiling: 256 pairs of one KV head per workgroup (8 waves),
// 64 visual keys per tile, at least this many tiles per key split.
constexpr int kResidualPairs = 256;
constexpr int kResidualMinTiles = 8;
constexpr int kResidualTargetBlocks = 512;
constexpr int kResidualMaxTiles = 32;   // key metadata of a split is held in LDS

// Tiling shared by the host layer (workspace sizing) and the kernels.
// (row, head) pairs per attention workgroup: 256 with values (refresh,
// 8 waves, one workgroup per CU), 128 for the statistics-only variant
// (4 waves, two workgroups per CU).
constexpr int attn_pairs_per_block(bool with_values) { return with_values ? 256 : 128; }
// Persistent attention grid: one resident workgroup slot per grid entry on
// the 256 CUs of an MI355X.
constexpr int attn_grid(bool with_values) { return with_values ? 256 : 512; }
// The plan aims at this many items per grid slot: finer items balance the
// CUs better, coarser ones write fewer partials and pay the per-item start
// (query load, first tile) less often.  Statistics tiles are cheap (no PV),
// so that variant keeps coarser items.
constexpr int attn_plan_rounds(bool with_values) { return with_values ? 2 : 1; }
constexpr int kAttnPlanMinTiles = 8;     // smallest split, in key tiles
constexpr int kAttnPlanMaxBlocks = 4096; // pair blocks per KV head the planner holds
// Items the plan aims at: `rounds` per grid slot; with values also at least
// two per pair block and KV head, so that long causal ranges are always cut
// (with more blocks than the grid takes per round and no splits, one block
// longer than a workgroup's share of the tiles sets the kernel's time).
constexpr int64_t attn_plan_target(int64_t n_pb, int64_t n_kv_heads, bool with_values) {
  const int64_t base = (int64_t)attn_grid(with_values) * attn_plan_rounds(with_values);
  return with_values && 2 * n_pb * n_kv_heads > base ? 2 * n_pb * n_kv_heads : base;
}
// Upper bound on the items of one plan: sum_b ceil(tiles_b / T) over blocks
// and KV heads, with T >= total tiles / target.
constexpr int64_t attn_max_items(int64_t n_pb, int64_t n_kv_heads, bool with_values) {
  return attn_plan_target(n_pb, n_kv_heads, with_values) + n_pb * n_kv_heads;
}
constexpr int kAttnKeyTile = 64;         // keys per LDS tile
constexpr int64_t kMaxStrideBytes = int64_t(1) << 25;  // row strides below 32 MiB: a key tile spans < 2 GiB
constexpr int kColsumKeysPerBlock = 256;  // visual keys per workgroup
// Split statistics rows are merged by every column-sum workgroup (in LDS,
// from registers) when the span has at most kColsumMaxLsePairs pairs per KV
// head, at most kLseRegSplits splits and at most kColsumFuseMaxBlocks key
// blocks (so few workgroups repeat it); otherwise the statistics kernel
// merges them once.
constexpr int kColsumMaxLsePairs = 4096;
constexpr int kLseRegSplits = 24;
constexpr int kColsumFuseMaxBlocks = 64;

}  // namespace conduit
