// Causal attention of query rows over one layer's KV cache, gfx950.
//
// Two users:
//  * the scoring pass needs, for every span row, the log-sum-exp of its
//    softmax over the row's key domain before the visual column sums of
//    Eq. 6 can be normalised (statistics only, no values);
//  * the selective recompute needs, for every selected visual row, causal
//    attention over the merged fresh/stale cache (values included).
//
// bf16 path, three launches:
//  1. attn_plan_kernel (one workgroup) reads the row positions and cuts the
//     work into items: a block of (row, head) pairs of one KV head times a
//     split of the block's causal key range.  Splits are near-equal, with the
//     smallest split size whose item count fits one or two items per resident
//     workgroup; items are listed largest first.
//  2. attn_bf16_kernel runs a persistent grid (one 8-wave workgroup per CU
//     with values, two 4-wave ones without) that walks the item list in
//     snake order, so every CU gets a similar share of tiles.  Per 64-key
//     tile, K is staged row-major and V row-major with its rows interleaved
//     within 16-key blocks (read back through transposing LDS reads free of
//     bank conflicts); with values by direct-to-LDS loads into five K
//     and four V stages, two tiles per barrier; statistics only through
//     registers, one tile per barrier.  Each wave computes
//     S^T = K Q^T with v_mfma_f32_32x32x16_bf16 so that every lane holds 16
//     keys of one pair column and the online softmax runs in-lane; the
//     probabilities feed O^T = V^T P^T straight from the accumulator
//     registers.  The loop is software-pipelined by 32-key sub-tiles: the S^T
//     products of the next sub-tile are issued while the current one is
//     exponentiated.  A block whose keys form a single split writes its final
//     outputs; otherwise each split writes (m, l, O) partials in the log2
//     domain.
//  3. combine_kernel merges the partials of split blocks in a fixed order
//     (deterministic, no atomics).
#include <algorithm>
#include <climits>
#include <type_traits>

#include "common.h"

namespace conduit {
namespace {

constexpr int KT = kAttnKeyTile;
constexpr float kNegInf = -__builtin_inff();
constexpr float kMInit = -1e30f;  // initial running maximum (log2 units)
// Statistics: the running maximum only moves when a sub-tile's maximum
// exceeds it by more than this many log2 units; probabilities stay below 2^8
// and l is rescaled rarely.  Exact: l and the final normaliser share it.
constexpr float kRescaleSlack = 8.f;
// Statistics: split partials a merging workgroup loads at once per pair.
constexpr int kMergeLoads = 16;

// LDS tiles.  K rows are D + 8 elements apart (16 bytes of padding: the 16
// lanes of an S^T operand read cover 16 rows in distinct banks); V rows are
// D + 16 apart and read through transposing LDS reads.  Both pitches make a
// tile a whole number of 1 KB direct-to-LDS transfers.
template <int D>
struct TileGeom {
  static constexpr int kPitch = D + 8, vPitch = D + 16;
  static constexpr int kXfer = KT * kPitch * 2 / 1024, vXfer = KT * vPitch * 2 / 1024;
  static_assert(KT * kPitch * 2 % 1024 == 0 && KT * vPitch * 2 % 1024 == 0, "whole 1 KB transfers");
};

// With values: five K and four V tile stages filled by direct-to-LDS loads
// (160.8 KB at d = 128).  Statistics only: three register-staged K tiles, the
// key-domain bits and the image table.
template <bool Stats>
struct StatsLds {
  uint64_t okmask[4];  // key-domain filter per K stage, bit = key
  ImageLds img;        // visual-only statistics: the image table
};
template <>
struct StatsLds<false> {};

template <int D, bool PV>
struct AttnSmem : StatsLds<!PV> {
  alignas(16) u16 k[PV ? 5 : 4][KT][TileGeom<D>::kPitch];
  alignas(16) u16 v[PV ? 4 : 1][PV ? KT : 1][TileGeom<D>::vPitch];
};

// One 1 KB direct-to-LDS transfer: lane l's 16 bytes at byte voff of the
// buffer land at LDS byte lds_addr + 16 l.  Written as assembly so that the
// compiler's wait insertion does not make every later LDS read wait for it;
// completion is awaited explicitly (vm_wait) before the barrier that
// publishes a tile.
__device__ __forceinline__ void lds_dma16(__amdgpu_buffer_rsrc_t r, uint32_t lds_addr, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds_addr), "v"(voff), "s"(r)
               : "memory", "m0");
}

// s_waitcnt vmcnt(N), expcnt and lgkmcnt left open (gfx9 encoding).
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__device__ __forceinline__ int row_position(const int32_t *row_pos, int q_pos0, int r) {
  return row_pos ? row_pos[r] : q_pos0 + r;
}

// Closed-form plan of rows at q_pos0 + r: block pb's {maxpos, minpos, n_s,
// chunk} (positions clamped to the cache, n_s near-equal splits).
__device__ __forceinline__ int4 uniform_block_info(int pb, int ppb, int group, int n_rows, int q_pos0,
                                                   int n_ctx, int ns) {
  const int64_t p0 = (int64_t)pb * ppb;
  const int64_t p1 = min(p0 + ppb, (int64_t)n_rows * group) - 1;
  const int minpos = min(q_pos0 + (int)(p0 / group), n_ctx - 1);
  const int maxpos = min(q_pos0 + (int)(p1 / group), n_ctx - 1);
  const int tiles = maxpos / KT + 1;
  return make_int4(maxpos, minpos, ns, ((tiles + ns - 1) / ns) * KT);
}



// Builds the work plan from the row positions (see AttnPlan).  One
// workgroup of 1024 threads; blocks and histogram bins live in LDS.
struct PlanArgs {
  const int32_t *row_pos;  // nullable: row r sits at q_pos0 + r
  int32_t q_pos0;
  int32_t n_rows;
  int32_t group;
  int32_t n_kv_heads;
  int32_t n_ctx;
  int32_t ppb;             // pairs per block
  int32_t target_items;    // grid slots * rounds
  AttnPlan plan;
};

constexpr int kPlanThreads = 1024;
constexpr int kPlanWaves = kPlanThreads / 64;
constexpr int kPlanBins = 2048;  // (size class, KV head) bins; larger sizes share the top class

// Exclusive prefix sum over the block (one call per kernel: s_wave is not
// reused, so no trailing barrier).
__device__ int plan_exclusive_scan(int x, int *s_wave, int &total) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int inc = (int)wave_inclusive_sum((uint32_t)x);
  if (lane == 63) s_wave[w] = inc;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int i = 0; i < kPlanWaves; ++i) {
    const int v = s_wave[i];
    before += i < w ? v : 0;
    all += v;
  }
  total = all;
  return before + inc - x;
}

__device__ __forceinline__ void build_plan(const PlanArgs &a) {
  __shared__ int s_max[kAttnPlanMaxBlocks], s_min[kAttnPlanMaxBlocks];
  __shared__ int s_base[kAttnPlanMaxBlocks + 1], s_ct[kAttnPlanMaxBlocks];
  __shared__ int s_bin[kPlanBins];   // per size class: count, then base
  __shared__ int s_rank[kPlanBins];  // per (size class, KV head): items placed
  __shared__ int s_wave[kPlanWaves];
  __shared__ int s_count;
  const int tid = threadIdx.x;
  const int n_pb = a.plan.n_pb;
  const int G = a.group;
  for (int b = tid; b < n_pb; b += kPlanThreads) {
    s_max[b] = 0;
    s_min[b] = 0x7fffffff;
  }
  for (int i = tid; i < kPlanBins; i += kPlanThreads) s_bin[i] = 0;
  if (tid == 0) s_count = 0;
  __syncthreads();

  // Position range of every block: each row updates the blocks its G pairs
  // fall in.  Positions are clamped to the cache, so no key tile of the plan
  // lies outside it.
  for (int r0 = 0; r0 < a.n_rows; r0 += 4 * kPlanThreads) {
    int rp[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int r = r0 + tid + u * kPlanThreads;
      rp[u] = r < a.n_rows ? (a.row_pos ? a.row_pos[r] : a.q_pos0 + r) : 0;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int r = r0 + tid + u * kPlanThreads;
      if (r >= a.n_rows) continue;
      const int pos = min(max(rp[u], 0), a.n_ctx - 1);
      const int64_t p0 = (int64_t)r * G;
      for (int64_t b = p0 / a.ppb; b <= (p0 + G - 1) / a.ppb; ++b) {
        atomicMax(&s_max[b], pos);
        atomicMin(&s_min[b], pos);
      }
    }
  }
  __syncthreads();

  // Items are ordered by size class, larger first; within a class the KV
  // heads alternate (item r of head h at class base + r * n_kv + h), so with
  // workgroup g on XCD g mod 8 each XCD's L2 serves few heads at a time.
  const int max_class = kPlanBins / a.n_kv_heads - 1;
  // Wave 0 alone sizes the splits (wave-level reductions, no barriers);
  // lane l owns blocks [l * per, (l + 1) * per).
  if (tid < 64) {
    const int lane = tid;
    const int per = (n_pb + 63) / 64;
    const int b0 = min(lane * per, n_pb), b1 = min(b0 + per, n_pb);
    int max_tiles = 0;
    for (int b = b0; b < b1; ++b) max_tiles = max(max_tiles, s_max[b] / kAttnKeyTile + 1);
    max_tiles = (int)wave_reduce((uint32_t)max_tiles, 0u, [](uint32_t x, uint32_t y) { return x > y ? x : y; });

    // Split size T: the smallest T >= kAttnPlanMinTiles whose item count
    // n_kv * sum_b ceil(tiles_b / T) fits the target (bisection; the count
    // does not grow with T).  Past T = max_tiles no block splits any more.
    auto count_items = [&](int T) {
      int my = 0;
      for (int b = b0; b < b1; ++b) my += (s_max[b] / kAttnKeyTile + T) / T;  // ceil(tiles / T)
      my = (int)wave_reduce((uint32_t)my, 0u, [](uint32_t x, uint32_t y) { return x + y; });
      return (long long)my * a.n_kv_heads;
    };
    int lo = kAttnPlanMinTiles, hi = max(kAttnPlanMinTiles, max_tiles);
    while (lo < hi) {
      const int mid = lo + (hi - lo) / 2;
      if (count_items(mid) <= a.target_items) hi = mid;
      else lo = mid + 1;
    }
    const int T = lo;

    // Splits per block: n_s = ceil(tiles / T) near-equal splits of ct <= T
    // tiles; all but the last hold ct tiles, the last at least one.  Sizes
    // go into a histogram (one count per KV head).
    int my_ns = 0;
    for (int b = b0; b < b1; ++b) my_ns += (s_max[b] / kAttnKeyTile + T) / T;
    const int inc = (int)wave_inclusive_sum((uint32_t)my_ns);
    int base = inc - my_ns;
    for (int b = b0; b < b1; ++b) {
      const int tiles = s_max[b] / kAttnKeyTile + 1;
      const int ns = (tiles + T - 1) / T;
      const int ct = (tiles + ns - 1) / ns;
      const int last = tiles - (ns - 1) * ct;
      s_base[b] = base;
      s_ct[b] = ct;
      a.plan.pb_info[b] = make_int4(s_max[b], min(max(s_min[b], 0), a.n_ctx - 1), ns, ct * kAttnKeyTile);
      a.plan.pb_base[b] = base;
      base += ns;
      // every KV head has the same splits: one count per size class
      if (ns > 1) atomicAdd(&s_bin[min(ct, max_class)], ns - 1);
      atomicAdd(&s_bin[min(last, max_class)], 1);
    }
    if (lane == 63) {
      s_base[n_pb] = inc;  // S
      s_count = inc;
    }
  }
  __syncthreads();
  const int S = s_count;

  // Largest first: the base of a size class counts the items of larger
  // classes (all heads).
  constexpr int kBinsPer = kPlanBins / kPlanThreads;
  int cnt[kBinsPer], my_cnt = 0;
#pragma unroll
  for (int i = 0; i < kBinsPer; ++i) {
    cnt[i] = s_bin[kPlanBins - 1 - (tid * kBinsPer + i)] * a.n_kv_heads;
    my_cnt += cnt[i];
  }
  int n_items;
  int off = plan_exclusive_scan(my_cnt, s_wave, n_items);
#pragma unroll
  for (int i = 0; i < kBinsPer; ++i) {
    s_bin[kPlanBins - 1 - (tid * kBinsPer + i)] = off;
    s_rank[kPlanBins - 1 - (tid * kBinsPer + i)] = 0;
    off += cnt[i];
  }
  __syncthreads();

  // One thread per item id = h * S + base_b + s (its partial slot); the
  // block is found by bisection over the bases.
  for (int id = tid; id < n_items; id += kPlanThreads) {
    const int h = id / S, rem = id - h * S;
    int l2 = 0, h2 = n_pb - 1;  // last block with base <= rem
    while (l2 < h2) {
      const int mid = (l2 + h2 + 1) >> 1;
      if (s_base[mid] <= rem) l2 = mid;
      else h2 = mid - 1;
    }
    const int b = l2, sp = rem - s_base[b];
    const int nsb = s_base[b + 1] - s_base[b], ct = s_ct[b];
    const int size = sp + 1 < nsb ? ct : (s_max[b] / kAttnKeyTile + 1) - (nsb - 1) * ct;
    const int cls = min(size, max_class);
    const int at = s_bin[cls] + atomicAdd(&s_rank[cls * a.n_kv_heads + h], 1) * a.n_kv_heads + h;
    if (at < a.plan.max_items) a.plan.items[at] = make_int4(h, b, sp, id);
  }
  if (tid == 0) {
    a.plan.hdr[0] = min(n_items, a.plan.max_items);
    a.plan.hdr[1] = S;
  }
}

__global__ __launch_bounds__(kPlanThreads) void attn_plan_kernel(PlanArgs a) { build_plan(a); }

// The plan (workgroup 0) and the cache merge of the same rows (the other
// workgroups, one wave per row) in one launch: they are independent, and the
// attention that follows needs both.
__global__ __launch_bounds__(kPlanThreads) void plan_scatter_kernel(PlanArgs a, ScatterParams sp) {
  if (blockIdx.x == 0) {
    build_plan(a);
    return;
  }
  const int row = (blockIdx.x - 1) * kPlanWaves + (threadIdx.x >> 6);
  if (row < sp.n_rows) scatter_row(sp, row, threadIdx.x & 63);
}

// W waves per workgroup, each owning 32 (row, head) pair columns.  With
// values (refresh) W = 8: two waves per SIMD and 256 pairs sharing each K/V
// tile; statistics only W = 4 with two workgroups per CU.  The grid is
// persistent: workgroup g takes items g, 2G' - 1 - g, 2G' + g, ... of the
// plan (G' = grid size), i.e. snake order over a largest-first list.
// ML: several layers per launch (LayerTable); item i of the launch is plan
// item i mod n of layer i / n (n plan items): layer after layer, each largest
// item first, so the running workgroups share one or two layers' K/V in the
// last-level cache.
template <int D, bool PV, int W, bool UNI, bool ML = false>
__global__ __launch_bounds__(W * 64, 8 / W) void attn_bf16_kernel(AttnParams p, LayerTable lt) {
  constexpr int kThreads = W * 64;
  constexpr int kPairs = W * 32;  // (row, head) pairs per block
  constexpr int KS = D / 16;      // MFMA k-steps over the head dimension
  constexpr int DT = D / 32;      // 32-row tiles of O^T
  __shared__ AttnSmem<D, PV> sm;
  __shared__ int s_restart;  // attempt id of the item being restarted (see kHeadroom)
  __shared__ int s_last;     // statistics: this workgroup holds the last split of its block

  const int G = p.group;
  const int n_pairs = p.n_rows * G;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 31, half = lane >> 5;
  if (p.zero_i32)
    for (int i = blockIdx.x * kThreads + tid; i < p.zero_n; i += gridDim.x * kThreads) p.zero_i32[i] = 0;
  const u16 *Kg = static_cast<const u16 *>(p.k);
  const u16 *Vg = static_cast<const u16 *>(p.v);
  const int n_layers = ML ? lt.n : 1;
  const KvPageReader pr = page_reader(p.pages, p.n_ctx);
  using Geo = TileGeom<D>;
  const int v_lane = v_operand_lane_offset_il<Geo::vPitch>(lane);  // PV operand reads (interleaved V rows)
  // Direct-to-LDS staging (with values): a tile's K transfers are numbered
  // 0..kXfer-1 and its V transfers kXfer..kXfer+vXfer-1; wave w issues
  // transfers w, w + 8, ...  Lane l of transfer x fills LDS byte 16 l of it,
  // i.e. one 16-byte chunk of a padded row; lanes that land in the padding
  // point past the buffer's end, so they fetch nothing and write zeros.
  // xoff[s] is lane l's byte offset inside the tile for transfer wave + 8 s
  // (head offset added per item; the padding offset stays out of range).
  constexpr int kXferAll = Geo::kXfer + Geo::vXfer;
  constexpr uint32_t kPadOff = 0x80000000u;  // beyond any tile resource (< 2 GiB): reads as 0
  constexpr int kXferUsed = PV ? kXferAll : Geo::kXfer;  // statistics only: K tiles alone
  constexpr int kSlots = (kXferUsed + W - 1) / W;
  uint32_t xoff0[kSlots];
#pragma unroll
  for (int sl = 0; sl < kSlots; ++sl) {
    const int x = wave + W * sl;
    const bool isk = x < Geo::kXfer;
    const int pitch_b = 2 * (isk ? Geo::kPitch : Geo::vPitch);
    const int b = (isk ? x : x - Geo::kXfer) * 1024 + 16 * lane;
    const int lrow = b / pitch_b, ch = (b % pitch_b) / 16;
    // V rows are stored interleaved: LDS row lrow holds this key of the tile
    const int row = isk ? lrow : (lrow & ~15) | v_interleaved_key(lrow & 15);
    xoff0[sl] = ch < D / 8 ? (uint32_t)(((int64_t)row * (isk ? p.k_stride : p.v_stride) + 8 * ch) * 2) : kPadOff;
  }
  const u16 *Qg = static_cast<const u16 *>(p.q);
  void *o_out = p.o_out;
  float *lse_out = p.lse_out;
  float *row_b = p.row_b;
  const float c = p.scale_log2;
  // UNI: the closed-form plan of contiguous rows (no plan loads at all).
  constexpr bool uniform = UNI;
  const int n_plan_items = uniform ? p.plan.uniform_items : min(p.plan.hdr[0], p.plan.max_items);
  const int n_items = n_plan_items * n_layers;

  const int grid = gridDim.x, g = blockIdx.x;
  if (tid == 0) s_restart = 0;
  int attempt_id = 0;
  if constexpr (!PV) {
    if (p.vis_only) {
      image_table_to_lds(p.tbl, sm.img, tid, kThreads);
      __syncthreads();
    }
  }

  for (int round = 0;; ++round) {
    const int lidx = round * grid + ((round & 1) ? grid - 1 - g : g);
    if (lidx >= n_items) break;
    const int idx = ML ? lidx % n_plan_items : lidx;  // plan item
    int64_t slot_off = 0;  // partial slots of this item's layer
    int layer = 0;
    if constexpr (ML) {
      layer = lidx / n_plan_items;
      Kg = static_cast<const u16 *>(lt.k[layer]);
      Vg = static_cast<const u16 *>(lt.v[layer]);
      Qg = static_cast<const u16 *>(lt.q[layer]);
      o_out = lt.o[layer];
      lse_out = lt.lse[layer];
      row_b = lt.rowb[layer];
      slot_off = (int64_t)layer * p.plan.max_items;
    }
    const int uns = p.plan.uniform_ns;
    const int4 item = uniform ? make_int4((idx / uns) % p.n_kv_heads, idx / (uns * p.n_kv_heads), idx % uns, idx)
                              : p.plan.items[idx];  // {kv head, block, split, slot}
    const int kvh = item.x, pb = item.y;
    if (kvh < 0 || kvh >= p.n_kv_heads || pb < 0 || pb >= p.plan.n_pb || item.w < 0 ||
        item.w >= p.plan.max_items)
      continue;
    const int4 info = uniform ? uniform_block_info(pb, kPairs, G, p.n_rows, p.q_pos0, p.n_ctx, uns)
                              : p.plan.pb_info[pb];  // {maxpos, minpos, n_s, chunk}
    const int kbeg = item.z * info.w;
    const int kend = min(kbeg + info.w, info.x + 1);
    const int minpos = info.y;
    const bool single = info.z == 1;
    if (kbeg >= kend) continue;
    const int pair0 = pb * kPairs;

    // The pair column owned by this lane.
    const int pair = pair0 + wave * 32 + col;
    const bool valid = pair < n_pairs;
    const int r = valid ? pair / G : 0;
    const int gpair = r * p.n_q_heads + kvh * G + (valid ? pair % G : 0);
    const int rp = valid ? row_position(p.row_pos, p.q_pos0, r) : -1;
    bf16x8 qreg[KS];
    {
      const u16 *qrow = Qg + (int64_t)gpair * D + 8 * half;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        qreg[ks] = as_bf16x8(valid ? ld16(qrow + ks * 16) : u32x4{0, 0, 0, 0});
    }

    // Statistics only (visual-only domain): one bit per key of the tile at
    // t0 in K stage st, set by wave 0 beside the tile's transfers.
    auto okmask_tile = [&](int st, int t0) __attribute__((always_inline)) {
      if constexpr (!PV) {
        if (p.vis_only && wave == 0) {
          const int kp = t0 + lane;
          const uint64_t bits = __ballot(kp < kend && is_visual(sm.img, kp));
          if (lane == 0) sm.okmask[st] = bits;
        }
      }
    };
    // This wave's transfers of the K tile at t0 (row0; rows at or past kend
    // read as 0 through the resource bound) into K stage st, or (with values)
    // of the V tile into V stage st.  A tile that does not exist still
    // gets its transfers (zero-length resource), so every iteration issues
    // the same count per wave.
    const uint32_t head_b = (uint32_t)(kvh * D * 2);
    auto dma_tile = [&](bool isk, int st, int t0, int64_t row0) __attribute__((always_inline)) {
      {
        const int rows = min(max(kend - t0, 0), KT);
        // the resource must sit in scalar registers: its inputs are uniform,
        // which readfirstlane makes explicit
        const uint64_t ga = (uint64_t)(uintptr_t)(isk ? Kg + row0 * p.k_stride : Vg + row0 * p.v_stride);
        const uint64_t gu = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(ga >> 32)) << 32) |
                            (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)ga);
        const int nbytes = __builtin_amdgcn_readfirstlane((int)(rows * (isk ? p.k_stride : p.v_stride) * 2));
        const auto rs = buffer_rsrc(reinterpret_cast<const void *>((uintptr_t)gu), nbytes);
        const uint32_t base = isk ? (uint32_t)(uintptr_t)&sm.k[st][0][0] : (uint32_t)(uintptr_t)&sm.v[PV ? st : 0][0][0];
#pragma unroll
        for (int sl = 0; sl < kSlots; ++sl) {
          const int x = wave + W * sl;
          if (isk ? x < Geo::kXfer : (x >= Geo::kXfer && x < kXferAll))
            lds_dma16(rs, __builtin_amdgcn_readfirstlane(base + (isk ? x : x - Geo::kXfer) * 1024),
                      xoff0[sl] == kPadOff ? kPadOff : xoff0[sl] + head_b);
        }
      }
    };

    // Running maximum (log2 units) starts finite, so exp2(c*s - m) needs no
    // special case: masked logits are -inf and give 0; the first tile with a
    // visible key always moves m.
    float m = kMInit, l = 0.f;
    f32x16 o[DT];

    // S^T of one 32-key sub-tile: K operands from LDS, 8 chained MFMAs.
    auto scores = [&](int buf, int sub) __attribute__((always_inline)) {
      bf16x8 ka[KS];
      const u16 *krow = &sm.k[buf][sub * 32 + col][8 * half];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) ka[ks] = as_bf16x8(ld16(krow + ks * 16));
      f32x16 sc = f32x16{};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[ks], qreg[ks], sc, 0, 0, 0);
      return sc;
    };
    // Tiles that need a key filter: causal / split end, and the key domain.
    auto tile_masked = [&](int t0) __attribute__((always_inline)) {
      return (!PV && p.vis_only) || t0 + KT > kend || t0 + KT - 1 > minpos;
    };
    // Key filter of sub-tile `sub` of the tile at t0 (K buffer buf).
    auto mask_sub = [&](f32x16 &sc, int buf, int t0, int sub) __attribute__((always_inline)) {
      const int lim = min(kend - 1, rp) - t0 - 4 * half;  // last visible key of the tile, lane-relative
      // key-domain filter (statistics of visual-only scoring): the tile's
      // bits from this lane's first key on
      uint64_t dom = ~0ull;
      if constexpr (!PV) dom = (sm.okmask[buf] | (p.vis_only ? 0ull : ~0ull)) >> (4 * half);
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int kl = sub * 32 + 8 * (v >> 2) + (v & 3);  // + 4 * half
        bool ok = kl <= lim;
        if constexpr (!PV) ok = ok & (((dom >> kl) & 1ull) != 0);
        sc[v] = ok ? sc[v] : kNegInf;
      }
    };
    auto sub_max = [&](const f32x16 &sc) __attribute__((always_inline)) {
      float x = kNegInf;
#pragma unroll
      for (int v = 0; v < 16; ++v) x = fmaxf(x, sc[v]);
      return half_max(x) * c;
    };

    // Software-pipelined main loop over 64-key tiles of two 32-key
    // sub-tiles, one barrier per tile.  Each sub-step issues the S^T products
    // of the next sub-tile while it exponentiates the current one
    // (independent work in one instruction stream, so the matrix core and
    // the VALU overlap), then O^T += V^T P^T of the current sub-tile while it
    // takes the next one's maximum.  Iteration t reads K(t), K(t+1) and V(t).
    // With values the tiles arrive by direct-to-LDS loads into a four-stage
    // ring, K three tiles ahead and V two (each wave waits for the transfers
    // it issued one iteration earlier before the barrier); statistics only
    // stage K through registers one tile ahead (three K buffers).
    // Block-table entries of 64 consecutive tiles are read at once, one per
    // lane, and each tile takes its entry with a lane read; only every 64th
    // tile waits for the table.
    int page_vec = 0, page_base = -64;
    auto tile_row = [&](int t0) __attribute__((always_inline)) {
      const int ti = t0 / KT;
      if (ti - page_base >= 64) {
        page_base = ti;
        page_vec = read_page(pr, (ti + (tid & 63)) * KT);
        vm_wait<0>();  // here, not before every lane read (the tile transfers are invisible to the compiler)
      }
      return page_row(pr, __builtin_amdgcn_readlane(page_vec, ti - page_base), t0);
    };
    auto row_of = [&](int t0) __attribute__((always_inline)) { return t0 < kend ? tile_row(t0) : (int64_t)0; };

    // With values, the probabilities of an item are taken against one
    // reference maximum per pair column, fixed for the item: the first
    // sub-tile's maximum (kMInit if none of its keys is visible: then no key
    // of the split is).  The result is exact for any reference (O, l and the
    // final normaliser share it); the reference only has to keep
    // 2^(c s - m) in range.  A later sub-tile whose maximum exceeds the
    // reference by more than kHeadroom (2^32: sums over any key range stay
    // far inside fp32) marks the workgroup for a restart of the item with
    // the largest maximum seen so far as the reference.  A restart is taken
    // at a barrier, so every wave takes it; each restart is triggered by a
    // sub-tile beyond the previous trigger, so an item restarts at most once
    // per iteration.  Without a running-maximum rescale the sub-steps have no
    // branch on the probabilities, and O^T is written by matrix products
    // only.  Statistics only keep an online maximum (their rescale is one
    // multiply; with the visual-only domain the first keys of a split are
    // often outside it, which a fixed reference would turn into restarts).
    constexpr float kHeadroom = 32.f;
    constexpr float kHeadroomSum = 4294967296.f;  // 2^kHeadroom
    float m_seen = kMInit;
    bool over = false;
    for (int attempt = 0;; ++attempt) {
    l = 0.f;
    page_base = -64;
    // Statistics over every key of the causal range take a fixed reference
    // in their first attempt like the values path; after a restart, or with
    // the visual-only domain, they keep the online maximum.
    const bool fixed_ref = PV ? attempt == 0 : attempt == 0 && !p.vis_only;
    if constexpr (!PV) m = kMInit;
    if constexpr (PV) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) o[dt] = f32x16{};
    }
    if constexpr (PV) {
      // K(0..2), V(0..1); tiles past kend arrive as zeros
      const int64_t r0 = tile_row(kbeg), r1 = row_of(kbeg + KT), r2 = row_of(kbeg + 2 * KT);
      dma_tile(true, 0, kbeg, r0);
      dma_tile(false, 0, kbeg, r0);
      dma_tile(true, 1, kbeg + KT, r1);
      dma_tile(false, 1, kbeg + KT, r1);
      dma_tile(true, 2, kbeg + 2 * KT, r2);
      vm_wait<0>();
    } else {
      // K(0..2); tiles past kend arrive as zeros
      const int64_t r0 = tile_row(kbeg), r1 = row_of(kbeg + KT), r2 = row_of(kbeg + 2 * KT);
      dma_tile(true, 0, kbeg, r0);
      okmask_tile(0, kbeg);
      dma_tile(true, 1, kbeg + KT, r1);
      okmask_tile(1, kbeg + KT);
      dma_tile(true, 2, kbeg + 2 * KT, r2);
      okmask_tile(2, kbeg + 2 * KT);
      vm_wait<0>();
    }
    __syncthreads();
    f32x16 sa = scores(0, 0), sb;
    if (PV || fixed_ref) {
      if (tile_masked(kbeg)) mask_sub(sa, 0, kbeg, 0);
      m = fmaxf(fmaxf(sub_max(sa), m_seen), kMInit);
      m_seen = m;
      over = false;
    }
    // One sub-step.  cur holds S^T of the current sub-tile (sub-tile csub of
    // the tile at ct0, K stage cbuf; its V rows are vsub*32.. of V stage
    // vst); the S^T products of the next sub-tile (K stage kbn, rows
    // ksub*32..; after the last sub-tile: discarded) are issued into nxt.
    // The key filter of cur comes first, so everything after it is one basic
    // block: the compiler then places the exponentials of cur among the
    // matrix products of nxt instead of sinking them past a later branch.
    // exact_tag std::false_type (a first attempt with a fixed reference)
    // only checks that the sub-tile's probabilities stay below 2^kHeadroom
    // in sum, which any sub-tile exceeding the reference by more than
    // kHeadroom violates.  std::true_type: with values every sub-tile's
    // maximum is tracked against the reference (the attempts after a
    // restart); statistics keep the online maximum.
    auto sub_step = [&](auto exact_tag, f32x16 &cur, f32x16 &nxt, int kbn, int ksub, int vst, int vsub,
                        bool cur_masked, int cbuf, int ct0, int csub) __attribute__((always_inline)) {
      constexpr bool kExact = decltype(exact_tag)::value;
      if (cur_masked) mask_sub(cur, cbuf, ct0, csub);
      nxt = scores(kbn, ksub);
      float alpha = 1.f;
      if constexpr (PV) {
        if constexpr (kExact) {
          const float mx = sub_max(cur);
          m_seen = fmaxf(m_seen, mx);
          over = over || mx > m + kHeadroom;
        }
      } else if constexpr (kExact) {
        const float mx = sub_max(cur);
        const bool grow = mx > m + kRescaleSlack;
        alpha = grow ? fast_exp2(m - mx) : 1.f;
        m = grow ? mx : m;
      }
      // probabilities of the current sub-tile; fp32 row sum (the
      // log-sum-exp output needs it to 1e-4; summing the bf16-rounded
      // probabilities is off by up to 2^-9 when few terms dominate)
      const float neg_m = -m;
#pragma unroll
      for (int v = 0; v < 16; ++v) cur[v] = fast_exp2(fmaf(cur[v], c, neg_m));
      float psum = 0.f;
#pragma unroll
      for (int v = 0; v < 16; ++v) psum += cur[v];
      if constexpr (!kExact) over = over || !(psum <= kHeadroomSum);  // inf included
      l = PV || !kExact ? l + psum : l * alpha + psum;
      // l is needed only after the loop; this empty statement makes it (and
      // so this sub-tile's exponentials) due here, so the compiler does not
      // sink them past the next sub-step's key filter.
      asm volatile("" ::"v"(l));
      if constexpr (PV) {
        bf16x8 pk[2];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
          for (int e = 0; e < 8; ++e) pk[ks][e] = static_cast<__bf16>(cur[8 * ks + e]);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          bf16x8 va[DT];
#pragma unroll
          for (int dt = 0; dt < DT; ++dt)
            va[dt] = v_operand_il<Geo::vPitch>(&sm.v[vst][vsub * 32 + ks * 16][dt * 32] + v_lane);
#pragma unroll
          for (int dt = 0; dt < DT; ++dt)
            o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[dt], pk[ks], o[dt], 0, 0, 0);
        }
      }
    };
    const int gen = ++attempt_id;  // the workgroup's attempts in order (uniform, never repeats)
    bool restart = false;
    if constexpr (PV) {
      // Two tiles (t, t+1) per barrier.  K stages rotate mod 5 and V stages
      // mod 4: the iteration reads K(t..t+2) and V(t..t+1) while K(t+3),
      // K(t+4), V(t+2) and V(t+3) arrive; they are awaited before the
      // barrier, one iteration after they were issued.  A tile t+1 past kend
      // arrives as zeros and is masked whole.  The last iteration issues no
      // transfers: only a next iteration would read them.
      // The first attempt checks the probability sums, a restart tracks the
      // maxima (below).
      auto tiles = [&](auto exact_tag) __attribute__((always_inline)) {
      int t0 = kbeg, ks = 0, vs = 0;  // stages of tile t
      for (;;) {
        const int k1 = ks + 1 == 5 ? 0 : ks + 1, k2 = k1 + 1 == 5 ? 0 : k1 + 1;
        const int k3 = k2 + 1 == 5 ? 0 : k2 + 1, k4 = k3 + 1 == 5 ? 0 : k3 + 1;
        const int v1 = (vs + 1) & 3, v2 = (vs + 2) & 3, v3 = (vs + 3) & 3;
        const bool more2 = t0 + 2 * KT < kend;  // the next iteration exists
        if (more2) {
          const int64_t r2 = row_of(t0 + 2 * KT), r3 = row_of(t0 + 3 * KT), r4 = row_of(t0 + 4 * KT);
          dma_tile(false, v2, t0 + 2 * KT, r2);
          dma_tile(false, v3, t0 + 3 * KT, r3);
          dma_tile(true, k3, t0 + 3 * KT, r3);
          dma_tile(true, k4, t0 + 4 * KT, r4);
        }
        const bool m0 = tile_masked(t0), m1 = tile_masked(t0 + KT);
        sub_step(exact_tag, sa, sb, ks, 1, vs, 0, m0, ks, t0, 0);       // S(t,1)   | P(t,0) V
        sub_step(exact_tag, sb, sa, k1, 0, vs, 1, m0, ks, t0, 1);       // S(t+1,0) | P(t,1) V
        sub_step(exact_tag, sa, sb, k1, 1, v1, 0, m1, k1, t0 + KT, 0);  // S(t+1,1) | P(t+1,0) V
        sub_step(exact_tag, sb, sa, k2, 0, v1, 1, m1, k1, t0 + KT, 1);  // S(t+2,0) | P(t+1,1) V
        if (__ballot(over) != 0 && lane == 0) s_restart = gen;
        vm_wait<0>();
        __syncthreads();
        restart = s_restart == gen;
        if (!more2 || restart) break;
        t0 += 2 * KT;
        ks = k2;
        vs = v2;
      }
      };
      if (fixed_ref) tiles(std::false_type{});
      else tiles(std::true_type{});
    } else {
      // One tile per barrier, K stages mod 4: iteration t reads K(t) and
      // K(t+1) while K(t+2) is complete and K(t+3) arrives.  Before the
      // barrier a wave waits until at most kSlots of its transfers are
      // outstanding: all of K(t+2)'s, so only K(t+3)'s may remain.  K(t+3)
      // is issued only if iteration t+2 exists (the first to read it);
      // otherwise the wave waits for all of its transfers.
      auto tiles = [&](auto exact_tag) __attribute__((always_inline)) {
      constexpr bool kExact = decltype(exact_tag)::value;
      int t0 = kbeg, st = 0;  // K stage of tile t
      for (;;) {
        const bool more = t0 + KT < kend;
        const bool need3 = t0 + 2 * KT < kend;  // iteration t+2 exists
        const int st1 = (st + 1) & 3, st3 = (st + 3) & 3;
        if (need3) {
          dma_tile(true, st3, t0 + 3 * KT, row_of(t0 + 3 * KT));
          okmask_tile(st3, t0 + 3 * KT);
        }
        const bool m0 = tile_masked(t0);
        sub_step(exact_tag, sa, sb, st, 1, 0, 0, m0, st, t0, 0);   // S(t,1)   | P(t,0)
        sub_step(exact_tag, sb, sa, st1, 0, 0, 0, m0, st, t0, 1);  // S(t+1,0) | P(t,1)
        if constexpr (!kExact) {
          if (__ballot(over) != 0 && lane == 0) s_restart = gen;
        }
        if (need3) vm_wait<kSlots - 1>();
        else vm_wait<0>();
        __syncthreads();
        if constexpr (!kExact) restart = s_restart == gen;
        if (!more || restart) break;
        t0 += KT;
        st = st1;
      }
      };
      if (fixed_ref) tiles(std::false_type{});
      else tiles(std::true_type{});
      vm_wait<0>();  // the last transfers (zero tiles) land before the stages are reused
    }

    if (!restart) break;
    }  // attempts

    // ---- outputs: final values for a single-split block, else partials ----
    const float l_tot = l + __shfl_xor(l, 32, 64);
    if (valid) {
      if (single) {
        const float b = m + __log2f(l_tot);
        if (half == 0) {
          if (row_b) row_b[gpair] = b;
          if (lse_out) lse_out[gpair] = b * kLn2;
        }
      } else {
        const int64_t idx2 = (item.w + slot_off) * kPairs + wave * 32 + col;
        if (half == 0) {
          if (!PV && p.merge_flag) {  // read by another workgroup of this kernel
            store_coherent(p.part_m + idx2, m);
            store_coherent(p.part_l + idx2, l_tot);
          } else {
            p.part_m[idx2] = m;
            p.part_l[idx2] = l_tot;
          }
        }
      }
    }
    if constexpr (PV) {
      // O / l of a single-split block, else the split's own output O_s / l_s
      // (a convex combination of V rows; l = 0, no visible key in the split,
      // gives 0), in bf16.  A lane holds 4-dim pieces of its pair column, so
      // the rows are assembled in LDS (pair-major, the K stages: no tile is
      // read any more) and written out 16 bytes per lane, each pair's row
      // contiguous.
      static_assert(kPairs * Geo::kPitch <= (int)(sizeof(sm.k) / 2), "output rows fit the K stages");
      u16 *orow = &sm.k[0][0][0];
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          uint2 w;
          w.x = (uint32_t)f32_to_bf16(o[dt][4 * g4] * inv) | ((uint32_t)f32_to_bf16(o[dt][4 * g4 + 1] * inv) << 16);
          w.y = (uint32_t)f32_to_bf16(o[dt][4 * g4 + 2] * inv) | ((uint32_t)f32_to_bf16(o[dt][4 * g4 + 3] * inv) << 16);
          *reinterpret_cast<uint2 *>(orow + (wave * 32 + col) * Geo::kPitch + dt * 32 + 8 * g4 + 4 * half) = w;
        }
      __syncthreads();
      constexpr int kChunks = D / 8;  // 16-byte pieces of a row
      // rows of the item's pairs: O rows (row, head) or consecutive partial rows
      u16 *const obase = single ? static_cast<u16 *>(o_out) : p.part_o + (item.w + slot_off) * kPairs * D;
#pragma unroll 2
      for (int i = 0; i < kPairs * kChunks / kThreads; ++i) {
        const int c = tid + kThreads * i;
        const int pl = c / kChunks, ch = c % kChunks;
        const int pr = pair0 + pl;
        if (pr < n_pairs) {
          const u32x4 v = *reinterpret_cast<const u32x4 *>(orow + pl * Geo::kPitch + ch * 8);
          const int64_t row = single ? (int64_t)(pr / G) * p.n_q_heads + kvh * G + pr % G : pl;
          *reinterpret_cast<u32x4 *>(obase + row * D + ch * 8) = v;
        }
      }
      __syncthreads();  // the next item's transfers overwrite these rows
    }

    // Statistics with the closed-form plan: each split item of a block,
    // once its partials are stored device-coherently and waited for, marks
    // its slot with the call's epoch and then reads the marks of the block's
    // other splits; one that finds them all set merges the block's splits in
    // split order, b = M + log2(sum_s l_s 2^(m_s - M)), into row_b / lse_out.
    // The last item to mark always finds them set; if two items both do,
    // they write the same values.
    if constexpr (!PV) {
      if (p.merge_flag && !single) {
        const int ns = info.z;
        const int64_t slot0 = ((int64_t)pb * p.n_kv_heads + kvh) * ns + slot_off;
        __builtin_amdgcn_s_waitcnt(0);  // this wave's partial stores are complete
        __syncthreads();
        if (tid == 0)
          __hip_atomic_store(p.merge_flag + item.w + slot_off, p.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __builtin_amdgcn_s_waitcnt(0);  // the mark is stored before the others are read
        if (wave == 0) {
          bool all = true;
          for (int s0 = 0; s0 < ns; s0 += 64) {
            const int sp = s0 + lane;
            const uint32_t f = sp < ns ? __hip_atomic_load(p.merge_flag + slot0 + sp, __ATOMIC_RELAXED,
                                                           __HIP_MEMORY_SCOPE_AGENT)
                                       : p.epoch;
            all = all && __ballot(f != p.epoch) == 0;
          }
          if (lane == 0) s_last = all;
        }
        __syncthreads();
        if (s_last) {
          for (int j = tid; j < kPairs; j += kThreads) {
            const int pair = pair0 + j;
            if (pair >= n_pairs) continue;
            const int gp = (pair / G) * p.n_q_heads + kvh * G + pair % G;
            // kMergeLoads splits' partials are loaded at once (indices
            // clamped, so every load is issued), then reduced in order
            auto ld = [&](const float *a, int sp) __attribute__((always_inline)) {
              return __hip_atomic_load(a + (slot0 + min(sp, ns - 1)) * kPairs + j, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
            };
            float mv[kMergeLoads], lv[kMergeLoads];
            float M = kNegInf, L = 0.f;
            for (int s0 = 0; s0 < ns; s0 += kMergeLoads) {
#pragma unroll
              for (int i = 0; i < kMergeLoads; ++i) mv[i] = ld(p.part_m, s0 + i);
#pragma unroll
              for (int i = 0; i < kMergeLoads; ++i) M = s0 + i < ns ? fmaxf(M, mv[i]) : M;
            }
            for (int s0 = 0; s0 < ns; s0 += kMergeLoads) {
              if (ns > kMergeLoads) {  // else the one batch is still in registers
#pragma unroll
                for (int i = 0; i < kMergeLoads; ++i) mv[i] = ld(p.part_m, s0 + i);
              }
#pragma unroll
              for (int i = 0; i < kMergeLoads; ++i) lv[i] = ld(p.part_l, s0 + i);
#pragma unroll
              for (int i = 0; i < kMergeLoads; ++i) L = s0 + i < ns ? L + fast_exp2(mv[i] - M) * lv[i] : L;
            }
            const float b = M + __log2f(L);
            if (row_b) row_b[gp] = b;
            if (lse_out) lse_out[gp] = b * kLn2;
          }
        }
      }
    }
  }
}

// Merge split partials of blocks with n_s > 1: M = max m_s,
// L = sum l_s 2^(m_s - M), O = sum l_s 2^(m_s - M) Ohat_s / L, splits in
// order, where Ohat_s = O_s / l_s is the split's own output, kept in bf16 (a
// convex combination of V rows, so its relative rounding error stays 2^-9
// and the merged row, a convex combination of the Ohat_s, keeps it).
// With values a thread merges 16 head dims of one pair (the whole grid is
// resident at once); statistics only, one thread per pair.  The m_s, l_s and
// Ohat_s of up to kMergeBatch splits are loaded together and folded into a
// running maximum, so a thread waits on two round trips to memory for
// n_s <= kMergeBatch (plan entry, then the partials); for such blocks the
// sums are exactly those of the two-pass formula above.
constexpr int kMergeBatch = 4;
constexpr int kMergeDims = 16;
template <int D>
__global__ __launch_bounds__(256) void combine_kernel(CombineParams p, LayerTable lt) {
  static_assert(D % kMergeDims == 0, "whole 16-dim slices");
  constexpr int NC = D / kMergeDims;
  if (lt.n > 0) {  // layer blockIdx.y of a multi-layer launch
    const int l = blockIdx.y;
    const int64_t off = (int64_t)l * p.plan.max_items * p.ppb;
    p.part_m += off;
    p.part_l += off;
    if (p.part_o) p.part_o += off * D;
    p.o_out = lt.o[l];
    p.lse_out = lt.lse[l];
    p.row_b = lt.rowb[l];
  }
  const int64_t n_gp = (int64_t)p.n_rows * p.n_q_heads;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const bool values = p.part_o != nullptr;
  const int64_t gp = values ? gid / NC : gid;
  const int c = values ? (int)(gid % NC) : 0;
  if (gp >= n_gp) return;
  const int r = (int)(gp / p.n_q_heads), hq = (int)(gp % p.n_q_heads);
  const int h = hq / p.group;
  const int64_t pair = (int64_t)r * p.group + hq % p.group;
  const int pb = (int)(pair / p.ppb), j = (int)(pair % p.ppb);
  const bool uniform = p.plan.uniform_ns > 0;
  const int ns = uniform ? p.plan.uniform_ns : p.plan.pb_info[pb].z;
  if (ns <= 1) return;  // written by the attention kernel
  const int64_t slot0 = uniform ? ((int64_t)pb * (p.n_q_heads / p.group) + h) * ns
                                : (int64_t)h * p.plan.hdr[1] + p.plan.pb_base[pb];
  if (slot0 + ns > p.plan.max_items) return;  // never for a plan within its bound
  const int64_t idx0 = slot0 * p.ppb + j;
  // Split s contributes W_s = 2^(m_s - M) l_s and W_s * Ohat_s, with Ohat_s
  // its normalised output (bf16) and M the running maximum of the m_s.
  float M = kNegInf, L = 0.f;
  float acc[kMergeDims];
#pragma unroll
  for (int e = 0; e < kMergeDims; ++e) acc[e] = 0.f;
  for (int s0 = 0; s0 < ns; s0 += kMergeBatch) {
    float mb[kMergeBatch], lb[kMergeBatch];
    u32x4 ob[kMergeBatch][2];
#pragma unroll
    for (int i = 0; i < kMergeBatch; ++i) {
      const bool in = s0 + i < ns;
      const int64_t idx = idx0 + (int64_t)(s0 + i) * p.ppb;
      mb[i] = in ? p.part_m[idx] : kNegInf;
      lb[i] = in ? p.part_l[idx] : 0.f;
#pragma unroll
      for (int q = 0; q < 2; ++q)
        ob[i][q] = in && values ? ld16(p.part_o + idx * D + kMergeDims * c + 8 * q) : u32x4{0, 0, 0, 0};
    }
    float Mn = M;
#pragma unroll
    for (int i = 0; i < kMergeBatch; ++i) Mn = fmaxf(Mn, mb[i]);  // finite: split s0 exists
    const float rs = fast_exp2(M - Mn);                             // 0 on the first batch
    L *= rs;
#pragma unroll
    for (int e = 0; e < kMergeDims; ++e) acc[e] *= rs;
#pragma unroll
    for (int i = 0; i < kMergeBatch; ++i) {
      if (s0 + i < ns) {
        const float w = fast_exp2(mb[i] - Mn) * lb[i];  // m >= kMInit is finite
        L += w;
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const uint32_t x = ob[i][q][u];
            acc[8 * q + 2 * u] += w * __builtin_bit_cast(float, x << 16);
            acc[8 * q + 2 * u + 1] += w * __builtin_bit_cast(float, x & 0xffff0000u);
          }
      }
    }
    M = Mn;
  }
  const float b = M + __log2f(L);
  if (c == 0) {
    if (p.row_b) p.row_b[gp] = b;
    if (p.lse_out) p.lse_out[gp] = b * kLn2;
  }
  if (values) {
    const float inv = 1.f / L;
    u16 *out = static_cast<u16 *>(p.o_out) + gp * D + kMergeDims * c;
#pragma unroll
    for (int q = 0; q < kMergeDims / 4; ++q) {
      uint2 w;
      w.x = (uint32_t)f32_to_bf16(acc[4 * q] * inv) | ((uint32_t)f32_to_bf16(acc[4 * q + 1] * inv) << 16);
      w.y = (uint32_t)f32_to_bf16(acc[4 * q + 2] * inv) | ((uint32_t)f32_to_bf16(acc[4 * q + 3] * inv) << 16);
      *reinterpret_cast<uint2 *>(out + 4 * q) = w;
    }
  }
}

// fp32 path.  A workgroup of four waves takes four consecutive rows of one
// query head (one wave per (row, head) pair); they share every 64-key tile of
// K (and V), which is staged in LDS by coalesced 16-byte loads.  For the
// logits, lane j of a wave takes key t0 + j of the tile: its K row is read
// from LDS (rows padded to D + 4 floats, so the lanes' rows start in
// different banks) and the query is held in registers.  The probabilities go
// through LDS, so that lane e accumulates output dims e, e + 64, ... over the
// tile's V rows.  The next tile's K/V chunks are loaded into registers while
// the current one is used, and the queries sit in LDS (read as broadcasts).
// Online softmax in the log2 domain, fp32 throughout.  With few rows the
// key range is cut into splits of whole tiles (blockIdx.z; see
// f32_attn_splits): each writes its (m, l) and unnormalised output, merged in
// split order by attn_f32_merge_kernel (or, for the statistics, by the fp32
// column sums).  Otherwise the final outputs are written directly.
constexpr int kF32Rows = kF32RowsPerBlock;
template <int D, bool PV>
__global__ __launch_bounds__(kF32Rows * 64) void attn_f32_kernel(AttnParams p, DirectOut out) {
  constexpr int KP = D + 4;
  constexpr int PER = D / 64;
  constexpr int CH = KT * D / 4 / (kF32Rows * 64);  // 16-byte chunks per thread and tile
  static_assert(CH * kF32Rows * 64 * 4 == KT * D, "whole chunks");
  __shared__ alignas(16) float ks[KT][KP];
  __shared__ alignas(16) float vsm[PV ? KT : 1][PV ? D : 4];
  __shared__ float ps[kF32Rows][KT];
  __shared__ alignas(16) float qsm[kF32Rows][D];
  __shared__ int s_maxpos;
  __shared__ ImageLds img;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int r = blockIdx.x * kF32Rows + wave, hq = blockIdx.y, kvh = hq / p.group;
  const bool valid = r < p.n_rows;
  const int rpos = valid ? min(row_position(p.row_pos, p.q_pos0, r), p.n_ctx - 1) : -1;
  const int64_t gp = (int64_t)(valid ? r : 0) * p.n_q_heads + hq;
  const float *Kg = static_cast<const float *>(p.k);
  const float *Vg = static_cast<const float *>(p.v);
  if (tid == 0) s_maxpos = -1;
  if (p.vis_only) image_table_to_lds(p.tbl, img, tid, kF32Rows * 64);
  __syncthreads();
  if (lane == 0) atomicMax(&s_maxpos, rpos);
  if (lane < D / 4) {
    const float *q = static_cast<const float *>(p.q) + gp * D;
    *reinterpret_cast<f32x4 *>(&qsm[wave][4 * lane]) =
        valid ? *reinterpret_cast<const f32x4 *>(q + 4 * lane) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // A tile's chunks (rows past the cache repeat its last row; they are
  // masked), loaded into registers one tile ahead.
  f32x4 kq[CH], vq[PV ? CH : 1];
  auto load_tile = [&](int t0) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int cidx = tid + kF32Rows * 64 * i;
      const int row = cidx / (D / 4), c4 = cidx % (D / 4);
      const int64_t src = kv_row(p.pages, min(t0 + row, p.n_ctx - 1));
      kq[i] = *reinterpret_cast<const f32x4 *>(Kg + src * p.k_stride + kvh * D + 4 * c4);
      if constexpr (PV) vq[i] = *reinterpret_cast<const f32x4 *>(Vg + src * p.v_stride + kvh * D + 4 * c4);
    }
  };
  __syncthreads();
  const int maxpos = s_maxpos;
  // this workgroup's keys: split blockIdx.z of the range, or all of it
  const bool split = out.n_split > 1;
  const int kb = split ? (int)blockIdx.z * out.chunk : 0;
  const int kend = split ? min(maxpos + 1, kb + out.chunk) : maxpos + 1;
  float m = kNegInf, l = 0.f, o[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) o[i] = 0.f;
  if (kb < kend) load_tile(kb);
  for (int t0 = kb; t0 < kend; t0 += KT) {
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int cidx = tid + kF32Rows * 64 * i;
      const int row = cidx / (D / 4), c4 = cidx % (D / 4);
      *reinterpret_cast<f32x4 *>(&ks[row][4 * c4]) = kq[i];
      if constexpr (PV) *reinterpret_cast<f32x4 *>(&vsm[row][4 * c4]) = vq[i];
    }
    __syncthreads();
    if (t0 + KT < kend) load_tile(t0 + KT);
    const int key = t0 + lane;
    const bool vis = key <= rpos && key < kend && (!p.vis_only || is_visual(img, key));
    float d4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int e = 0; e < D; e += 4) {
      const f32x4 kk = *reinterpret_cast<const f32x4 *>(&ks[lane][e]);
      const f32x4 qq = *reinterpret_cast<const f32x4 *>(&qsm[wave][e]);
#pragma unroll
      for (int u = 0; u < 4; ++u) d4[u] = fmaf(qq[u], kk[u], d4[u]);
    }
    const float dot = (d4[0] + d4[1]) + (d4[2] + d4[3]);
    const float z = vis ? dot * p.scale_log2 : kNegInf;
    const float m_new = fmaxf(m, wave_max(z));
    const float m_use = m_new == kNegInf ? 0.f : m_new;
    const float alpha = fast_exp2(m - m_use);
    const float pj = fast_exp2(z - m_use);
    l = l * alpha + wave_sum(pj);
    m = m_new;
    if constexpr (PV) {
      ps[wave][lane] = pj;  // read back by this wave only; LDS keeps a wave's accesses in order
#pragma unroll
      for (int i = 0; i < PER; ++i) o[i] *= alpha;
#pragma unroll 8
      for (int j = 0; j < KT; ++j) {
        const float pjj = ps[wave][j];
#pragma unroll
        for (int i = 0; i < PER; ++i) o[i] = fmaf(pjj, vsm[j][lane + 64 * i], o[i]);
      }
    }
    __syncthreads();
  }
  if (!valid) return;
  if (split) {  // the split's (m, l) and unnormalised output, merged below
    const int64_t idx = (int64_t)blockIdx.z * p.n_rows * p.n_q_heads + gp;
    if (lane == 0) out.part_ml[idx] = make_float2(m, l);
    if constexpr (PV) {
#pragma unroll
      for (int i = 0; i < PER; ++i) out.part_o[idx * D + lane + 64 * i] = o[i];
    }
    return;
  }
  const float b = m + __log2f(l);
  if (lane == 0) {
    if (out.row_b) out.row_b[gp] = b;
    if (out.lse_out) out.lse_out[gp] = b * kLn2;
  }
  if constexpr (PV) {
    const float inv = 1.f / l;
    float *dst = out.o_out + gp * D;
#pragma unroll
    for (int i = 0; i < PER; ++i) dst[lane + 64 * i] = o[i] * inv;
  }
}

// Merge of the fp32 key splits, in split order: M = max m_s,
// L = sum l_s 2^(m_s - M), O = sum o_s 2^(m_s - M) / L (o_s unnormalised,
// relative to m_s).  One thread per (pair, output dim), or per pair without
// values.  Every pair sees at least one key, so M is finite.
template <int D, bool PV>
__global__ __launch_bounds__(256) void attn_f32_merge_kernel(int64_t n_gp, DirectOut out) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t gp = PV ? gid / D : gid;
  const int d = PV ? (int)(gid % D) : 0;
  if (gp >= n_gp) return;
  float M = kNegInf;
  for (int sp = 0; sp < out.n_split; ++sp) M = fmaxf(M, out.part_ml[sp * n_gp + gp].x);
  float L = 0.f, acc = 0.f;
  for (int sp = 0; sp < out.n_split; ++sp) {
    const float2 ml = out.part_ml[sp * n_gp + gp];
    const float w = ml.y > 0.f ? fast_exp2(ml.x - M) : 0.f;  // an empty split adds nothing
    L = fmaf(w, ml.y, L);
    if constexpr (PV) acc = fmaf(w, out.part_o[(sp * n_gp + gp) * D + d], acc);
  }
  const float b = M + __log2f(L);
  if (d == 0) {
    if (out.row_b) out.row_b[gp] = b;
    if (out.lse_out) out.lse_out[gp] = b * kLn2;
  }
  if constexpr (PV) out.o_out[gp * D + d] = acc / L;
}

__global__ void lse_to_b_kernel(const float *lse, float *b, int n, int32_t *zero_i32, int zero_n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) b[i] = lse[i] * kLog2e;
  if (zero_i32)
    for (int z = i; z < zero_n; z += gridDim.x * blockDim.x) zero_i32[z] = 0;
}

}  // namespace

// Split count of the closed-form plan for rows at q_pos0 + r: about the
// device plan's item target, at least kAttnPlanMinTiles tiles per split of
// the shortest block, and no empty split in any block.
int attn_uniform_splits(const AttnParams &p, int ppb, int target) {
  const int64_t n_pairs = (int64_t)p.n_rows * p.group;
  const int n_pb = (int)((n_pairs + ppb - 1) / ppb);
  int min_tiles = INT32_MAX;
  auto tiles_of = [&](int b) {
    const int64_t last = std::min<int64_t>((int64_t)(b + 1) * ppb, n_pairs) - 1;
    const int maxpos = std::min(p.q_pos0 + (int)(last / p.group), p.n_ctx - 1);
    return maxpos / KT + 1;
  };
  for (int b = 0; b < n_pb; ++b) min_tiles = std::min(min_tiles, tiles_of(b));
  int ns = std::max(1, target / std::max(1, n_pb * p.n_kv_heads));
  ns = std::min(ns, std::max(1, min_tiles / kAttnPlanMinTiles));
  auto all_nonempty = [&](int n) {
    for (int b = 0; b < n_pb; ++b) {
      const int t = tiles_of(b);
      if ((int64_t)((t + n - 1) / n) * (n - 1) >= t) return false;
    }
    return true;
  };
  while (ns > 1 && !all_nonempty(ns)) --ns;
  return ns;
}

// Split count of the scoring span's statistics with `layers` layers in one
// launch.  One layer takes attn_uniform_splits' count.  With several, every
// split count multiplies into layers * blocks * KV heads items, so fewer
// splits fill the grid: among the counts up to the one-layer count that
// leave no split empty, the one with the least estimated time, i.e. grid
// rounds times (tiles per split + kSpanItemTiles, an item's fixed start and
// end in tiles), the smaller count on ties.
int attn_span_splits(const AttnParams &p, int ppb, int layers) {
  const int ns1 = attn_uniform_splits(p, ppb, attn_grid(false) * attn_plan_rounds(false));
  if (layers <= 1) return ns1;
  constexpr int kSpanItemTiles = 4;
  const int64_t n_pairs = (int64_t)p.n_rows * p.group;
  const int64_t n_pb = (n_pairs + ppb - 1) / ppb;
  auto tiles_of = [&](int64_t b) {
    const int64_t last = std::min<int64_t>((b + 1) * ppb, n_pairs) - 1;
    const int maxpos = std::min(p.q_pos0 + (int)(last / p.group), p.n_ctx - 1);
    return maxpos / KT + 1;
  };
  const int max_tiles = tiles_of(n_pb - 1);  // positions grow with the row
  auto all_nonempty = [&](int n) {
    for (int64_t b = 0; b < n_pb; ++b) {
      const int t = tiles_of(b);
      if ((int64_t)((t + n - 1) / n) * (n - 1) >= t) return false;
    }
    return true;
  };
  int best = ns1;
  int64_t best_cost = INT64_MAX;
  for (int ns = 1; ns <= ns1; ++ns) {
    if (ns > 1 && !all_nonempty(ns)) continue;
    const int64_t items = (int64_t)layers * n_pb * p.n_kv_heads * ns;
    const int64_t rounds = (items + attn_grid(false) - 1) / attn_grid(false);
    const int64_t cost = rounds * ((max_tiles + ns - 1) / ns + kSpanItemTiles);
    if (cost < best_cost) {
      best_cost = cost;
      best = ns;
    }
  }
  return best;
}

namespace {

// The plan's arguments for rows with positions (layers: the layers of one
// launch, 0 for one).
PlanArgs plan_args(const AttnParams &p, bool with_values, int layers) {
  PlanArgs pa{};
  pa.row_pos = p.row_pos;
  pa.q_pos0 = p.q_pos0;
  pa.n_rows = p.n_rows;
  pa.group = p.group;
  pa.n_kv_heads = p.n_kv_heads;
  pa.n_ctx = p.n_ctx;
  pa.ppb = attn_pairs_per_block(with_values);
  // With several layers per launch every plan item runs once per layer, so
  // when one layer's unsplit items do not fill the grid the plan needs
  // proportionally fewer splits.  Layers that fill it on their own keep the
  // one-layer plan: the launch then walks the layers one after the other
  // like separate launches would (their K/V do not all fit in the last-level
  // cache at once; unsplit items of very different lengths would spread the
  // workgroups over several layers).
  const int64_t one_layer = attn_plan_target(p.plan.n_pb, p.n_kv_heads, with_values);
  pa.target_items = (int32_t)(layers > 0 && (int64_t)p.plan.n_pb * p.n_kv_heads < attn_grid(with_values)
                                  ? std::max<int64_t>(1, one_layer / layers) : one_layer);
  pa.plan = p.plan;
  return pa;
}

}  // namespace

hipError_t launch_attn(const AttnParams &p_in, int head_dim, bool with_values, hipStream_t s, const LayerTable *lt,
                       bool plan_ready) {
  const LayerTable lt0 = lt ? *lt : LayerTable{};
  const bool ml = lt0.n > 0;
  const int ppb = attn_pairs_per_block(with_values);
  AttnParams p = p_in;
  if (!p.row_pos && !with_values) {  // the scoring span: closed-form plan, no plan launch
    const int ns = attn_span_splits(p, ppb, ml ? lt0.n : 1);
    const int64_t n_pb = ((int64_t)p.n_rows * p.group + ppb - 1) / ppb;
    p.plan.uniform_ns = ns;
    p.plan.uniform_items = (int32_t)(n_pb * p.n_kv_heads * ns);
  } else {
    p.plan.uniform_ns = 0;
    p.plan.uniform_items = 0;
  }
  const PlanArgs pa = plan_args(p, with_values, lt0.n);
  hipError_t e = hipSuccess;
  if (p.plan.uniform_ns == 0 && !plan_ready) {
    ProfScope ps("attn_plan", s);
    attn_plan_kernel<<<1, kPlanThreads, 0, s>>>(pa);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }

  const int grid = attn_grid(with_values);
  {
    ProfScope ps(with_values ? "attn_values" : "attn_stats", s);
    // the closed-form plan only serves the statistics of the scoring span
    const bool uni = p.plan.uniform_ns > 0 && !with_values;
    if (ml && !with_values && !uni) return hipErrorInvalidValue;  // several layers: refresh or scoring span
    if (head_dim == 128) {
      if (ml && !with_values) attn_bf16_kernel<128, false, 4, true, true><<<grid, 4 * 64, 0, s>>>(p, lt0);
      else if (ml) attn_bf16_kernel<128, true, 8, false, true><<<grid, 8 * 64, 0, s>>>(p, lt0);
      else if (with_values) attn_bf16_kernel<128, true, 8, false><<<grid, 8 * 64, 0, s>>>(p, lt0);
      else if (uni) attn_bf16_kernel<128, false, 4, true><<<grid, 4 * 64, 0, s>>>(p, lt0);
      else attn_bf16_kernel<128, false, 4, false><<<grid, 4 * 64, 0, s>>>(p, lt0);
    } else {
      if (ml && !with_values) attn_bf16_kernel<64, false, 4, true, true><<<grid, 4 * 64, 0, s>>>(p, lt0);
      else if (ml) attn_bf16_kernel<64, true, 8, false, true><<<grid, 8 * 64, 0, s>>>(p, lt0);
      else if (with_values) attn_bf16_kernel<64, true, 8, false><<<grid, 8 * 64, 0, s>>>(p, lt0);
      else if (uni) attn_bf16_kernel<64, false, 4, true><<<grid, 4 * 64, 0, s>>>(p, lt0);
      else attn_bf16_kernel<64, false, 4, false><<<grid, 4 * 64, 0, s>>>(p, lt0);
    }
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;

  if (p.skip_merge) return hipSuccess;  // merged by the caller's next kernel
  CombineParams cp{};
  cp.n_rows = p.n_rows;
  cp.n_q_heads = p.n_q_heads;
  cp.group = p.group;
  cp.ppb = ppb;
  cp.plan = p.plan;
  cp.part_m = p.part_m;
  cp.part_l = p.part_l;
  cp.part_o = with_values ? p.part_o : nullptr;
  cp.row_b = p.row_b;
  cp.lse_out = p.lse_out;
  cp.o_out = with_values ? p.o_out : nullptr;
  const int64_t n_gp = (int64_t)p.n_rows * p.n_q_heads;
  const int64_t n = with_values ? n_gp * (head_dim / kMergeDims) : n_gp;
  const dim3 blocks((unsigned)((n + 255) / 256), ml ? (unsigned)lt0.n : 1u);
  ProfScope ps("attn_merge", s);
  if (head_dim == 128) combine_kernel<128><<<blocks, 256, 0, s>>>(cp, lt0);
  else combine_kernel<64><<<blocks, 256, 0, s>>>(cp, lt0);
  return hipGetLastError();
}

hipError_t launch_merge_refresh(const AttnParams &p, const ScatterParams &sp, int head_dim, hipStream_t s) {
  {
    ProfScope ps("plan_scatter", s);
    const unsigned blocks = 1u + (unsigned)((sp.n_rows + kPlanWaves - 1) / kPlanWaves);
    plan_scatter_kernel<<<blocks, kPlanThreads, 0, s>>>(plan_args(p, true, 0), sp);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return launch_attn(p, head_dim, true, s, nullptr, /*plan_ready=*/true);
}

hipError_t launch_attn_f32(const AttnParams &p, const DirectOut &out, int head_dim,
                           bool with_values, hipStream_t s) {
  const int ns = out.n_split > 1 ? out.n_split : 1;
  {
    ProfScope ps("attn_f32", s);
    const dim3 grid((p.n_rows + kF32Rows - 1) / kF32Rows, p.n_q_heads, ns);
    if (head_dim == 128) {
      if (with_values) attn_f32_kernel<128, true><<<grid, kF32Rows * 64, 0, s>>>(p, out);
      else attn_f32_kernel<128, false><<<grid, kF32Rows * 64, 0, s>>>(p, out);
    } else {
      if (with_values) attn_f32_kernel<64, true><<<grid, kF32Rows * 64, 0, s>>>(p, out);
      else attn_f32_kernel<64, false><<<grid, kF32Rows * 64, 0, s>>>(p, out);
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || ns == 1 || !out.merge) return e;
  ProfScope ps("attn_f32_merge", s);
  const int64_t n_gp = (int64_t)p.n_rows * p.n_q_heads;
  const int64_t n = with_values ? n_gp * head_dim : n_gp;
  const unsigned blocks = (unsigned)((n + 255) / 256);
  if (head_dim == 128) {
    if (with_values) attn_f32_merge_kernel<128, true><<<blocks, 256, 0, s>>>(n_gp, out);
    else attn_f32_merge_kernel<128, false><<<blocks, 256, 0, s>>>(n_gp, out);
  } else {
    if (with_values) attn_f32_merge_kernel<64, true><<<blocks, 256, 0, s>>>(n_gp, out);
    else attn_f32_merge_kernel<64, false><<<blocks, 256, 0, s>>>(n_gp, out);
  }
  return hipGetLastError();
}

hipError_t launch_lse_to_b(const float *lse_in, float *row_b, int32_t n, int32_t *zero_i32, int32_t zero_n,
                           hipStream_t s) {
  ProfScope ps("lse_to_b", s);
  lse_to_b_kernel<<<(n + 255) / 256, 256, 0, s>>>(lse_in, row_b, n, zero_i32, zero_n);
  return hipGetLastError();
}

}  // namespace conduit
