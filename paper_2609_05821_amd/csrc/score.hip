// Scoring pass kernels, gfx950 (Sec. 3.3 Eq. 6-7; Algorithm 1 scoring loop).
// Visual keys are located through the image table (copied into LDS), so no
// index map is built beforehand.
//
// Once every span row's log-sum-exp b_r (log2 domain) is known, the visual
// column sums of Eq. 6 are  sum_r 2^(c * <q_r, k_t> - b_r)  with
// c = scale * log2(e).  A workgroup owns 256 visual keys of one KV head and
// streams all (span token, grouped head) rows of that head past them:
// S = Q K^T with v_mfma_f32_32x32x16_bf16 puts one key column in each lane
// (16 rows per lane), so the column sums accumulate in-lane.  The same
// workgroup reads its keys' V rows once for the value-norm proxy (the norm of
// the concatenated cached heads), so the cache is read once per layer.
// Per-KV-head partials are reduced in a fixed order by the finalize kernel,
// which also applies the 1/(n_q H_q) mean and accumulates the layer into
// s = sum_l a v and A = sum_l a (Eq. 7).
#include <type_traits>

#include "common.h"

namespace conduit {
namespace {

constexpr float kInf = __builtin_inff();

constexpr int kColsumThreads = 512;   // 8 waves x 32 keys

// Q rows stream through LDS in chunks of kQChunk (span token, head) rows,
// double-buffered: the next chunk's global loads (unconditional, clamped
// addresses) are in flight while the current chunk's kQChunk / 32 MFMA row
// tiles and exponentials run, one barrier per chunk.  The V rows for the
// value norms are fetched during the last chunk and consumed at the end.
constexpr int kQChunk = 256;

// Finalize of one visual token: fixed-order sum over KV heads, the mean (or
// RMS) over rows and heads, the value norm, s = a v and the layer
// accumulation of Eq. 7.
// COHERENT: the partials were written by other workgroups of the running
// kernel with device-coherent stores, and are read the same way.
template <bool COHERENT = false>
__device__ __forceinline__ void finalize_token(const FinalizeParams &p, int t) {
  auto ld = [](const float *q) {
    return COHERENT ? __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : *q;
  };
  float cs = 0.f, sq = 0.f;
  for (int h = 0; h < p.n_kv_heads; ++h) {
    cs += ld(p.colsum_part + (int64_t)h * p.n_vis + t);
    if (!p.vnorm_in) sq += ld(p.vsq_part + (int64_t)h * p.n_vis + t);
  }
  const float a = p.rms ? sqrtf(cs / p.n_rows_f) : cs / p.n_rows_f;
  const float v = p.vnorm_in ? p.vnorm_in[t] : sqrtf(sq);
  const float s = a * v;
  if (p.accumulate) {
    p.s_acc[t] += s;
    p.a_acc[t] += a;
  } else {
    p.s_acc[t] = s;
    p.a_acc[t] = a;
  }
  if (p.a_out) p.a_out[t] = a;
  if (p.vnorm_out) p.vnorm_out[t] = v;
}


// The workgroups of the n_kv_heads KV heads of one key block each count
// their arrival once their partials are stored (device-coherent stores,
// waited for before the count); the last to arrive finalizes the block's
// keys, reading every head's partials in head order with device-coherent
// loads, as the finalize kernel does.  The counters are cleared by the kernel
// that runs before this one.  (A device-scope release/acquire fence pair per
// workgroup would write back and invalidate the XCD's L2 each time, which
// costs more than the separate finalize launch.)
// With several layers in the launch (nb > 0) the last of the nb * n_kv_heads
// workgroups of a key block finalizes every layer in layer order: the same
// fp32 additions, in the same order, as one finalize per layer.
__device__ __forceinline__ void finalize_layers_token(const FinalizeParams &p, const LayerTable &lt, int nb, int t) {
  const int64_t stride = (int64_t)p.n_kv_heads * p.n_vis;
  float s_acc = 0.f, a_acc = 0.f;
  for (int l = 0; l < nb; ++l) {
    float cs = 0.f, sq = 0.f;
    const float *vn = layer_entry(lt.vnorm, l);
    for (int h = 0; h < p.n_kv_heads; ++h) {
      const int64_t i = l * stride + (int64_t)h * p.n_vis + t;
      cs += __hip_atomic_load(const_cast<float *>(p.colsum_part + i), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (!vn) sq += __hip_atomic_load(const_cast<float *>(p.vsq_part + i), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    const float a = p.rms ? sqrtf(cs / p.n_rows_f) : cs / p.n_rows_f;
    const float v = vn ? vn[t] : sqrtf(sq);
    const float sv = a * v;
    if (l == 0 && !p.accumulate) {
      s_acc = sv;
      a_acc = a;
    } else {
      if (l == 0) {
        s_acc = p.s_acc[t];
        a_acc = p.a_acc[t];
      }
      s_acc += sv;
      a_acc += a;
    }
  }
  p.s_acc[t] = s_acc;
  p.a_acc[t] = a_acc;
}

__device__ __forceinline__ void finalize_when_last(const ColsumParams &p, const LayerTable &lt, int tid,
                                                   int n_threads) {
  __shared__ int s_last;
  __builtin_amdgcn_s_waitcnt(0);  // this wave's partial stores are complete
  __syncthreads();
  const int arrivals = p.n_kv_heads * (lt.n > 0 ? lt.n : 1);
  if (tid == 0)
    s_last = __hip_atomic_fetch_add(p.done + blockIdx.x, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
             arrivals - 1;
  __syncthreads();
  if (!s_last) return;
  for (int i = tid; i < kColsumKeysPerBlock; i += n_threads) {
    const int t = blockIdx.x * kColsumKeysPerBlock + i;
    if (t >= p.n_vis) continue;
    if (lt.n > 0) finalize_layers_token(p.fin, lt, lt.n, t);
    else finalize_token<true>(p.fin, t);
  }
}

// RMS: accumulate alpha^2 (Eq. 4's surrogate) instead of alpha.
// FUSE: the row log-sum-exps are rebuilt from the statistics partials into
// LDS (the split merge of the statistics pass, same order and arithmetic).
// lt.n > 0: several layers, layer blockIdx.z (the statistics partials, column
// sums and norms of layer l sit l strides further on).
template <int D, bool RMS, bool FUSE>
__global__ __launch_bounds__(kColsumThreads) void colsum_bf16_kernel(ColsumParams p, LayerTable lt) {
  constexpr int KS = D / 16;
  // This layer's pointers, in locals: p itself stays unwritten (a written
  // kernel parameter holding the image table would be copied to scratch).
  const bool ml = lt.n > 0;
  const int layer = ml ? (int)blockIdx.z : 0;
  const int64_t part_off = (int64_t)layer * p.n_kv_heads * p.n_vis;
  const int64_t lse_off = p.lse_part_m ? layer * p.lse_layer_stride : 0;
  const void *k_l = ml ? layer_entry(lt.k, layer) : p.k;
  const void *v_l = ml ? layer_entry(lt.v, layer) : p.v;
  const void *q_l = ml ? layer_entry(lt.q, layer) : p.q;
  const float *row_b = ml ? layer_entry(lt.rowb, layer) : p.row_b;
  const float *vnorm_in = ml ? layer_entry(lt.vnorm, layer) : p.vnorm_in;
  float *colsum_part = p.colsum_part + part_off;
  float *vsq_part = p.vsq_part + part_off;
  const float *lse_part_m = p.lse_part_m ? p.lse_part_m + lse_off : nullptr;
  const float *lse_part_l = p.lse_part_m ? p.lse_part_l + lse_off : nullptr;
  float *lse_out = ml ? nullptr : p.lse_out;
  constexpr int QCH = kQChunk * D / 8;       // 16-byte chunks in a Q chunk
  constexpr int CPT = QCH / kColsumThreads;  // per thread
  constexpr int VPT = kColsumKeysPerBlock * D / 8 / kColsumThreads;  // V chunks per thread
  static_assert(QCH % kColsumThreads == 0, "Q chunk split");
  __shared__ alignas(16) u16 qs[2][kQChunk][D + 8];
  __shared__ alignas(16) float bs[2][kQChunk];
  __shared__ ImageLds img;
  __shared__ float b_all[FUSE ? kColsumMaxLsePairs : 1];
  __shared__ int64_t s_row[kColsumKeysPerBlock];  // cache row of each key of the block

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 31, half = lane >> 5;
  const int kvh = blockIdx.y;
  const int G = p.group;
  const int n_pair = p.n_q * G;
  const int nch = (n_pair + kQChunk - 1) / kQChunk;
  const u16 *Kg = static_cast<const u16 *>(k_l);
  const u16 *Vg = static_cast<const u16 *>(v_l);
  const u16 *Qg = static_cast<const u16 *>(q_l);

  // Chunk c into registers.  Item i of a thread is pair row
  // c * kQChunk + tid / (D/8) + i * kRowStep, i.e. span row qq[i] and head
  // rr[i] of the group (pair = qq * G + rr), kept from chunk to chunk by
  // adding kQChunk = q_step * G + r_step.  The loads go through a buffer
  // resource bounded by the span's queries, so rows past n_pair read as
  // zeros (and their b as +inf when stored).
  constexpr int kRowStep = kColsumThreads / (D / 8);
  const int q_step = kQChunk / G, r_step = kQChunk % G;
  int qq[CPT], rr[CPT];
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int pr0 = tid / (D / 8) + kRowStep * i;
    qq[i] = pr0 / G;
    rr[i] = pr0 % G;
  }
  int qb = tid / G, rb = tid % G;  // statistics row of this thread (tid < kQChunk)
  const auto q_rsrc = buffer_rsrc(Qg, p.n_q * p.n_q_heads * D * 2);
  const auto b_rsrc = buffer_rsrc(row_b, FUSE ? 0 : p.n_q * p.n_q_heads * 4);
  const uint32_t lane_b = (tid % (D / 8)) * 16;
  auto next_rows = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      rr[i] += r_step;
      qq[i] += q_step;
      if (rr[i] >= G) {
        rr[i] -= G;
        ++qq[i];
      }
    }
    rb += r_step;
    qb += q_step;
    if (rb >= G) {
      rb -= G;
      ++qb;
    }
  };
  auto load_chunk = [&](u32x4 (&qv)[CPT], float &bv) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < CPT; ++i)
      qv[i] = buffer_ld16(q_rsrc, (uint32_t)((qq[i] * p.n_q_heads + kvh * G + rr[i]) * D) * 2u + lane_b);
    if (!FUSE && tid < kQChunk)
      bv = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                         b_rsrc, (uint32_t)(qb * p.n_q_heads + kvh * G + rb) * 4u, 0, 0));
  };
  auto store_chunk = [&](int c, int buf, const u32x4 (&qv)[CPT], float bv) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int cidx = tid + kColsumThreads * i;
      st16(&qs[buf][cidx / (D / 8)][(cidx % (D / 8)) * 8], qv[i]);
    }
    if (tid < kQChunk) {
      const int pr = c * kQChunk + tid;
      bs[buf][tid] = pr < n_pair ? (FUSE ? b_all[pr] : bv) : kInf;  // 2^-inf = 0
    }
  };

  u32x4 qv[CPT];
  float bv = kInf;
  load_chunk(qv, bv);

  // FUSE: b = M + log2(sum_s l_s 2^(m_s - M)) over the splits of the row's
  // block, s ascending, exactly as the statistics merge computes it.  The
  // host fuses only up to kLseRegSplits splits: they are read in one pass
  // (indices clamped, so every read is issued unconditionally) and reduced
  // from registers, two rows per thread and pass (a second row past n_pair
  // reads the last row instead and is not stored).  Split sp of a row sits
  // sp * lse_ppb floats after split 0: a scalar offset of the load, the
  // same for every lane.  The first pass's reads go out before the image
  // table and the K rows: they hit in the cache the statistics kernel just
  // wrote, and reads issued after the K rows would wait for them (the memory
  // counter returns in order).
  const int ns = p.lse_ns;
  const auto m_rsrc = buffer_rsrc(lse_part_m, FUSE ? 0x7fffffff : 0);
  const auto l_rsrc = buffer_rsrc(lse_part_l, FUSE ? 0x7fffffff : 0);
  const uint32_t split_b = (uint32_t)p.lse_ppb * 4u;
  float mv[FUSE ? 2 : 1][FUSE ? kLseRegSplits : 1], lv[FUSE ? 2 : 1][FUSE ? kLseRegSplits : 1];
  // Spans of at most kLseFewSplits splits read only that many (the tag
  // gives the count read); the rest read all kLseRegSplits, clamped.
  constexpr int kLseFewSplits = 8;
  const bool few_splits = ns <= kLseFewSplits;
  auto lse_issue = [&](int pr0, auto nsm_tag) __attribute__((always_inline)) {
    constexpr int NSM = decltype(nsm_tag)::value;
    if constexpr (FUSE) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int pr = min(pr0 + u * kColsumThreads, n_pair - 1);
        const int pb = pr / p.lse_ppb, j = pr % p.lse_ppb;
        const int64_t slot0 = ((int64_t)pb * p.n_kv_heads + kvh) * ns;
        const uint32_t row_b0 = (uint32_t)(slot0 * p.lse_ppb + j) * 4u;
#pragma unroll
        for (int sp = 0; sp < NSM; ++sp) {
          const uint32_t so = (uint32_t)min(sp, ns - 1) * split_b;
          mv[u][sp] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(m_rsrc, row_b0, so, 0));
          lv[u][sp] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(l_rsrc, row_b0, so, 0));
        }
      }
    }
  };
  auto lse_reduce = [&](int pr0, auto nsm_tag) __attribute__((always_inline)) {
    constexpr int NSM = decltype(nsm_tag)::value;
    if constexpr (FUSE) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int pr = pr0 + u * kColsumThreads;
        float M = -kInf, L = 0.f;
#pragma unroll
        for (int sp = 0; sp < NSM; ++sp) M = sp < ns ? fmaxf(M, mv[u][sp]) : M;
#pragma unroll
        for (int sp = 0; sp < NSM; ++sp) L = sp < ns ? L + fast_exp2(mv[u][sp] - M) * lv[u][sp] : L;
        const float b = M + __log2f(L);
        if (pr < n_pair) {
          b_all[pr] = b;
          if (blockIdx.x == 0 && lse_out) lse_out[(pr / G) * p.n_q_heads + kvh * G + pr % G] = b * kLn2;
        }
      }
    }
  };
  using FewTag = std::integral_constant<int, kLseFewSplits>;
  using AllTag = std::integral_constant<int, kLseRegSplits>;
  if (FUSE && n_pair > 0) {
    if (few_splits) lse_issue(tid, FewTag{});
    else lse_issue(tid, AllTag{});
  }

  image_table_to_lds(p.tbl, img, tid, kColsumThreads);
  __syncthreads();
  // This lane's key column, held as the B operand for every row tile.
  const int t = blockIdx.x * kColsumKeysPerBlock + wave * 32 + col;
  const bool tvalid = t < p.n_vis;
  bf16x8 kreg[KS];
  {
    // the key's cache row (page lookup included), also kept for the V rows
    const int64_t row = kv_row(p.pages, vis_position(img, tvalid ? t : p.n_vis - 1));
    if (half == 0) s_row[wave * 32 + col] = row;
    const u16 *krow = Kg + row * p.k_stride + kvh * D + 8 * half;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kreg[ks] = as_bf16x8(ld16(krow + ks * 16));
  }
  // V rows of the block's keys for the value norms, 16 bytes per item (not
  // read when the norms are given).  They are loaded during the last Q
  // chunk, so that they do not compete with the K rows and the first chunk
  // for memory bandwidth at the start; their addresses are formed after the
  // first chunk is staged, from the rows the K loads resolved.
  const bool read_v = vnorm_in == nullptr;
  u32x4 vv[VPT];
  const u16 *vsrc[VPT];
  auto load_v = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < VPT; ++i) vv[i] = read_v ? ld16(vsrc[i]) : u32x4{0, 0, 0, 0};
  };
  const int v_chunk = nch - 1;  // no chunk load (and wait) follows
  if constexpr (FUSE) {
    if (few_splits) {
      if (n_pair > 0) lse_reduce(tid, FewTag{});
      for (int pr0 = tid + 2 * kColsumThreads; pr0 < n_pair; pr0 += 2 * kColsumThreads) {
        lse_issue(pr0, FewTag{});
        lse_reduce(pr0, FewTag{});
      }
    } else {
      if (n_pair > 0) lse_reduce(tid, AllTag{});
      for (int pr0 = tid + 2 * kColsumThreads; pr0 < n_pair; pr0 += 2 * kColsumThreads) {
        lse_issue(pr0, AllTag{});
        lse_reduce(pr0, AllTag{});
      }
    }
    __syncthreads();
  }
  store_chunk(0, 0, qv, bv);
  __syncthreads();
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    const int vi = tid + kColsumThreads * i;  // key vi / (D/8) of the block (rows past n_vis repeat the last)
    vsrc[i] = Vg + s_row[vi / (D / 8)] * p.v_stride + kvh * D + (vi % (D / 8)) * 8;
  }

  float colsum = 0.f;
  for (int c = 0; c < nch; ++c) {
    const int buf = c & 1;
    const bool more = c + 1 < nch;
    if (more) {
      next_rows();
      load_chunk(qv, bv);
    }
    if (c == v_chunk) load_v();
    const int rows = min(kQChunk, n_pair - c * kQChunk);
    auto row_step = [&](int r0) __attribute__((always_inline)) {
      f32x16 acc0 = f32x16{}, acc1 = f32x16{};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 a0 = as_bf16x8(ld16(&qs[buf][r0 + col][ks * 16 + 8 * half]));
        const bf16x8 a1 = as_bf16x8(ld16(&qs[buf][r0 + 32 + col][ks * 16 + 8 * half]));
        acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, kreg[ks], acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, kreg[ks], acc1, 0, 0, 0);
      }
      // lane (col, half), register v holds row 8*(v/4) + 4*half + v%4 of its tile
      float part0 = 0.f, part1 = 0.f;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 b0 = *reinterpret_cast<const f32x4 *>(&bs[buf][r0 + 8 * g + 4 * half]);
        const f32x4 b1 = *reinterpret_cast<const f32x4 *>(&bs[buf][r0 + 32 + 8 * g + 4 * half]);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          // alpha = 2^(c z - b); RMS sums alpha^2 = 2^(2 (c z - b))
          const float z0 = fmaf(acc0[4 * g + i], p.scale_log2, -b0[i]);
          const float z1 = fmaf(acc1[4 * g + i], p.scale_log2, -b1[i]);
          part0 += fast_exp2(RMS ? 2.f * z0 : z0);
          part1 += fast_exp2(RMS ? 2.f * z1 : z1);
        }
      }
      colsum += part0 + part1;
    };
    // A full chunk's row steps unrolled: one step's products are independent
    // of the previous step's exponentials, so the two overlap.
    if (rows == kQChunk) {
#pragma unroll
      for (int r0 = 0; r0 < kQChunk; r0 += 64) row_step(r0);
    } else {
      for (int r0 = 0; r0 < rows; r0 += 64) row_step(r0);
    }
    if (more) store_chunk(c + 1, buf ^ 1, qv, bv);
    __syncthreads();
  }
  colsum += __shfl_xor(colsum, 32, 64);
  if (half == 0 && tvalid) store_coherent(colsum_part + (int64_t)kvh * p.n_vis + t, colsum);

  // Value-norm proxy: this head's share of ||V_t||^2.  Item vi covers
  // dims (vi % (D/8))*8 .. +7 of key vi / (D/8); the D/8 items of a key sit
  // in consecutive lanes and are summed with lane shuffles.
  static_assert((D / 8) <= 64 && 64 % (D / 8) == 0, "key items within a wave");
#pragma unroll
  for (int i = 0; read_v && i < VPT; ++i) {
    float sq = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = __builtin_bit_cast(float, vv[i][e] << 16);
      const float hi = __builtin_bit_cast(float, vv[i][e] & 0xffff0000u);
      sq = fmaf(lo, lo, sq);
      sq = fmaf(hi, hi, sq);
    }
#pragma unroll
    for (int o = 1; o < D / 8; o <<= 1) sq += __shfl_xor(sq, o, 64);
    const int vi = tid + kColsumThreads * i;
    const int tv = blockIdx.x * kColsumKeysPerBlock + vi / (D / 8);
    if (vi % (D / 8) == 0 && tv < p.n_vis) store_coherent(vsq_part + (int64_t)kvh * p.n_vis + tv, sq);
  }
  if (p.done) finalize_when_last(p, lt, tid, kColsumThreads);
}

// fp32 path: one wave per 64 visual keys of one KV head.  Lane j holds the
// K row of key j in registers; the (span token, grouped head) query rows and
// their log-sum-exps pass through LDS in chunks of 64 (loaded coalesced, read
// as broadcasts), and the lane sums 2^(c z - b) (or its square) over them.
// The lane's V row gives its share of ||V_t||^2.
template <int D>
__global__ __launch_bounds__(64) void colsum_f32_kernel(ColsumParams p, bool rms) {
  __shared__ alignas(16) float qs[64][D];
  __shared__ float bs[64];
  const int lane = threadIdx.x;
  const int t = blockIdx.x * 64 + lane;
  const int kvh = blockIdx.y;
  const bool tvalid = t < p.n_vis;
  const float *Kg = static_cast<const float *>(p.k);
  const float *Vg = static_cast<const float *>(p.v);
  const float *Qg = static_cast<const float *>(p.q);
  const int64_t pos = kv_row(p.pages, vis_position(p.tbl, tvalid ? t : p.n_vis - 1));  // cache row
  float kr[D];
#pragma unroll
  for (int e = 0; e < D; e += 4) {
    const f32x4 x = *reinterpret_cast<const f32x4 *>(Kg + pos * p.k_stride + kvh * D + e);
    kr[e] = x[0];
    kr[e + 1] = x[1];
    kr[e + 2] = x[2];
    kr[e + 3] = x[3];
  }
  // The V row's share of ||V_t||^2, loaded with the K row (in flight during
  // the first query chunk).
  float sq = 0.f;
  if (!p.vnorm_in) {
    const float *vr = Vg + pos * p.v_stride + kvh * D;
#pragma unroll
    for (int e = 0; e < D; e += 4) {
      const f32x4 x = *reinterpret_cast<const f32x4 *>(vr + e);
#pragma unroll
      for (int u = 0; u < 4; ++u) sq = fmaf(x[u], x[u], sq);
    }
  }
  const int G = p.group, n_pair = p.n_q * G;
  float colsum = 0.f;
  for (int c0 = 0; c0 < n_pair; c0 += 64) {
    const int rows = min(64, n_pair - c0);
    for (int cidx = lane; cidx < rows * (D / 4); cidx += 64) {
      const int rr = cidx / (D / 4), c4 = cidx % (D / 4), pr = c0 + rr;
      const int64_t qrow = (int64_t)(pr / G) * p.n_q_heads + kvh * G + pr % G;
      *reinterpret_cast<f32x4 *>(&qs[rr][4 * c4]) = *reinterpret_cast<const f32x4 *>(Qg + qrow * D + 4 * c4);
    }
    if (lane < rows) {
      const int pr = c0 + lane;
      const int64_t gq = (int64_t)(pr / G) * p.n_q_heads + kvh * G + pr % G;
      if (p.f32_ml) {
        // the statistics' key splits, merged as their merge launch would:
        // b = M + log2(sum_s l_s 2^(m_s - M)), splits in order
        const int64_t n_gp = (int64_t)p.n_q * p.n_q_heads;
        float M = -kInf;
        for (int sp = 0; sp < p.lse_ns; ++sp) M = fmaxf(M, p.f32_ml[sp * n_gp + gq].x);
        float L = 0.f;
        for (int sp = 0; sp < p.lse_ns; ++sp) {
          const float2 ml = p.f32_ml[sp * n_gp + gq];
          const float w = ml.y > 0.f ? fast_exp2(ml.x - M) : 0.f;
          L = fmaf(w, ml.y, L);
        }
        const float b = M + __log2f(L);
        if (blockIdx.x == 0 && p.lse_out) p.lse_out[gq] = b * kLn2;
        bs[lane] = b;
      } else {
        bs[lane] = p.row_b[gq];
      }
    }
    __syncthreads();
    for (int rr = 0; rr < rows; ++rr) {
      float d4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int e = 0; e < D; e += 4) {
        const f32x4 qq = *reinterpret_cast<const f32x4 *>(&qs[rr][e]);
#pragma unroll
        for (int u = 0; u < 4; ++u) d4[u] = fmaf(qq[u], kr[e + u], d4[u]);
      }
      const float dot = (d4[0] + d4[1]) + (d4[2] + d4[3]);
      const float z = fmaf(dot, p.scale_log2, -bs[rr]);
      colsum += fast_exp2(rms ? 2.f * z : z);
    }
    __syncthreads();
  }
  if (!tvalid) return;
  p.colsum_part[(int64_t)kvh * p.n_vis + t] = colsum;
  if (!p.vnorm_in) p.vsq_part[(int64_t)kvh * p.n_vis + t] = sq;
}

__global__ void finalize_kernel(FinalizeParams p) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t < p.n_vis) finalize_token<false>(p, t);
}

// Value-norm table (Eq. 7's proxy, tabulated when the cache is built): one
// wave per visual token sums the squares of its row_elems cached values
// (all KV heads concatenated), 16 bytes per lane and step.
template <bool BF16>
__global__ __launch_bounds__(256) void value_norms_kernel(const void *v, int64_t v_stride, KvPages pages,
                                                          int row_elems, ImageTable tbl, float *out) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (t >= tbl.n_vis) return;
  constexpr int EPC = BF16 ? 8 : 4;  // elements per 16-byte chunk
  const char *row = static_cast<const char *>(v) + kv_row(pages, vis_position(tbl, t)) * v_stride * (BF16 ? 2 : 4);
  float sq = 0.f;
  for (int c = lane; c < row_elems / EPC; c += 64) {
    const u32x4 w = ld16(row + 16 * c);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (BF16) {
        const float lo = __builtin_bit_cast(float, w[e] << 16);
        const float hi = __builtin_bit_cast(float, w[e] & 0xffff0000u);
        sq = fmaf(lo, lo, sq);
        sq = fmaf(hi, hi, sq);
      } else {
        // The element goes through a scalar first: hipcc compiled a bit_cast
        // of the vector-element lvalue itself into a read of element 0.
        const uint32_t u = w[e];
        const float x = __builtin_bit_cast(float, u);
        sq = fmaf(x, x, sq);
      }
    }
  }
  sq = wave_sum(sq);
  if (lane == 0) out[t] = sqrtf(sq);
}

}  // namespace

hipError_t launch_value_norms(const void *v, int64_t v_stride, const KvPages &pages, int32_t row_elems,
                              bool bf16, const ImageTable &tbl, float *out, hipStream_t s) {
  ProfScope ps("value_norms", s);
  const int blocks = (tbl.n_vis + 3) / 4;
  if (bf16) value_norms_kernel<true><<<blocks, 256, 0, s>>>(v, v_stride, pages, row_elems, tbl, out);
  else value_norms_kernel<false><<<blocks, 256, 0, s>>>(v, v_stride, pages, row_elems, tbl, out);
  return hipGetLastError();
}

hipError_t launch_colsum(const ColsumParams &p, int head_dim, bool bf16, bool rms, hipStream_t s,
                         const LayerTable *lt) {
  const LayerTable lt0 = lt ? *lt : LayerTable{};
  if (bf16) {
    dim3 grid((p.n_vis + kColsumKeysPerBlock - 1) / kColsumKeysPerBlock, p.n_kv_heads, lt0.n > 0 ? lt0.n : 1);
    ProfScope ps("colsum", s);
    const bool fuse = p.lse_part_m != nullptr;
    if (head_dim == 128) {
      if (fuse) {
        if (rms) colsum_bf16_kernel<128, true, true><<<grid, kColsumThreads, 0, s>>>(p, lt0);
        else colsum_bf16_kernel<128, false, true><<<grid, kColsumThreads, 0, s>>>(p, lt0);
      } else {
        if (rms) colsum_bf16_kernel<128, true, false><<<grid, kColsumThreads, 0, s>>>(p, lt0);
        else colsum_bf16_kernel<128, false, false><<<grid, kColsumThreads, 0, s>>>(p, lt0);
      }
    } else {
      if (fuse) {
        if (rms) colsum_bf16_kernel<64, true, true><<<grid, kColsumThreads, 0, s>>>(p, lt0);
        else colsum_bf16_kernel<64, false, true><<<grid, kColsumThreads, 0, s>>>(p, lt0);
      } else {
        if (rms) colsum_bf16_kernel<64, true, false><<<grid, kColsumThreads, 0, s>>>(p, lt0);
        else colsum_bf16_kernel<64, false, false><<<grid, kColsumThreads, 0, s>>>(p, lt0);
      }
    }
  } else {
    dim3 grid((p.n_vis + 63) / 64, p.n_kv_heads);
    ProfScope ps("colsum_f32", s);
    if (head_dim == 128) colsum_f32_kernel<128><<<grid, 64, 0, s>>>(p, rms);
    else colsum_f32_kernel<64><<<grid, 64, 0, s>>>(p, rms);
  }
  return hipGetLastError();
}

hipError_t launch_finalize(const FinalizeParams &p, hipStream_t s) {
  ProfScope ps("finalize", s);
  finalize_kernel<<<(p.n_vis + 255) / 256, 256, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace conduit
