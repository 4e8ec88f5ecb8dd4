// Residual value-write error of a refresh set, gfx950 (Eq. 3 of the local
// residual-staleness model; App. D.1 isotropic Monte Carlo displacements and
// App. D.3 projected error).
//
// For displacement sample m, span row i and query head h the residual is
//   y = sum over visual t not in T of alpha_{i,h,t} xi^(m)_t[kv(h)],
// with alpha the cached-key attention of the scoring pass (normalised by the
// row's log-sum-exp, which the caller supplies), and the kernel reports
// ||y||^2.  xi is either kappa ||V_t|| / sqrt(H_kv D) * z_t (z given) or the
// cached value itself (stale values zeroed, App. D.3).
//
// The bf16 path is one MFMA pass per (key split, 256-pair block, KV head,
// sample): S^T = K Q^T for 64 visual keys, alpha = 2^(c s - b) straight from
// the known log-sum-exp (no running maximum), and y^T += Xi^T alpha^T with the
// displacement tile staged row-major in LDS (scaled at staging) and read
// through transposing LDS reads; refreshed keys and keys past the last
// visual token get a zero displacement row.  Partial y
// per split go to the workspace; residual_sum_kernel adds them in split order
// and squares.
#include <type_traits>

#include "common.h"

namespace conduit {
namespace {

constexpr int KT = kAttnKeyTile;
constexpr int kThreads = 512;   // 8 waves, 32 pairs each

template <int D>
struct ResidualSmem {
  alignas(16) u16 k[2][KT][D + 8];   // K rows of the tile's visual keys
  alignas(16) u16 x[2][KT][D + 32];  // displacement tile, one row per key (PV operand reads transpose)
  int64_t row[kResidualMaxTiles * KT];   // cache row of each key of the split
  float scale[kResidualMaxTiles * KT];   // displacement scale: sigma_t, 1, or 0 (refreshed)
  ImageLds img;
};

template <int D>
__global__ __launch_bounds__(kThreads, 1) void residual_bf16_kernel(ResidualParams p) {
  constexpr int KS = D / 16;                     // MFMA k-steps over the head dim
  constexpr int DT = D / 32;                     // 32-row tiles of y^T
  constexpr int KCH = KT * D / 8 / kThreads;     // 16-byte K (and displacement) chunks per thread
  static_assert(KCH >= 1 && KT * D / 8 == KCH * kThreads, "staging covers the tile");
  __shared__ ResidualSmem<D> sm;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 31, half = lane >> 5;
  const int split = blockIdx.x, pb = blockIdx.y;
  const int kvh = blockIdx.z % p.n_kv_heads, m = blockIdx.z / p.n_kv_heads;
  const int G = p.group;
  const int n_pairs = p.n_q * G;
  const u16 *Kg = static_cast<const u16 *>(p.k);
  const u16 *Xg = static_cast<const u16 *>(p.disp);
  const float c = p.scale_log2;
  const bool iso = p.vnorm != nullptr;
  const int v_lane = v_operand_lane_offset<D + 32>(lane);

  image_table_to_lds(p.tbl, sm.img, tid, kThreads);

  // The pair column owned by this lane; its query and log-sum-exp.
  const int pair = pb * kResidualPairs + wave * 32 + col;
  const bool valid = pair < n_pairs;
  const int r = valid ? pair / G : 0;
  const int gpair = r * p.n_q_heads + kvh * G + (valid ? pair % G : 0);
  bf16x8 qreg[KS];
  {
    const u16 *qrow = static_cast<const u16 *>(p.q) + (int64_t)gpair * D + 8 * half;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qreg[ks] = as_bf16x8(valid ? ld16(qrow + ks * 16) : u32x4{0, 0, 0, 0});
  }
  const float b = valid ? p.row_b[gpair] : 0.f;

  const int tv_beg = split * p.tiles_per_split * KT;
  const int tv_end = min(tv_beg + p.tiles_per_split * KT, p.n_vis);
  __syncthreads();  // image table in LDS
  // Per-key metadata of the split, resolved once: the tile loop then reads
  // only LDS before its global loads (a dependent global read there would
  // make every tile wait for the loads already in flight).
  for (int j = tid; j < tv_end - tv_beg; j += kThreads) {
    const int tv = tv_beg + j;
    sm.row[j] = kv_row(p.pages, vis_position(sm.img, tv));
    sm.scale[j] = p.refreshed[tv] ? 0.f : (iso ? p.vnorm[tv] * p.sigma_scale : 1.f);
  }
  __syncthreads();
  const int last = max(tv_end - tv_beg - 1, 0);

  // Two register sets: tiles are loaded two ahead of the one computing, so
  // each load has two tiles' compute to arrive.
  u32x4 rk[2][KCH];
  u32x4 rx[2][KCH];
  float sx[2][KCH];
  // Global -> register set R for the tile of visual keys tv0 .. tv0 + 63.
  auto load_tile = [&](int tv0, auto set) __attribute__((always_inline)) {
    constexpr int R = decltype(set)::value;
    const int j0 = tv0 - tv_beg;
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int cidx = tid + kThreads * i;
      const int jr = j0 + cidx / (D / 8), j = min(jr, last);
      const int dc = (cidx % (D / 8)) * 8;
      rk[R][i] = ld16(Kg + sm.row[j] * p.k_stride + kvh * D + dc);
      const int64_t off = iso ? (((int64_t)m * p.n_vis + tv_beg + j) * p.n_kv_heads + kvh) * D
                              : sm.row[j] * p.disp_stride + kvh * D;
      rx[R][i] = ld16(Xg + off + dc);
      sx[R][i] = jr <= last ? sm.scale[j] : 0.f;
    }
  };
  // Registers -> LDS: K rows as loaded; the displacement scaled and rounded
  // to bf16, row-major.
  auto store_tile = [&](int buf, auto set) __attribute__((always_inline)) {
    constexpr int R = decltype(set)::value;
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int cidx = tid + kThreads * i;
      st16(&sm.k[buf][cidx / (D / 8)][(cidx % (D / 8)) * 8], rk[R][i]);
    }
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int cidx = tid + kThreads * i;
      u32x4 w;
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        const uint32_t u = rx[R][i][e2];
        const float lo = __builtin_bit_cast(float, u << 16) * sx[R][i];
        const float hi = __builtin_bit_cast(float, u & 0xffff0000u) * sx[R][i];
        w[e2] = (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
      }
      st16(&sm.x[buf][cidx / (D / 8)][(cidx % (D / 8)) * 8], w);
    }
  };

  f32x16 y[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) y[dt] = f32x16{};

  auto tile = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      const u16 *krow = &sm.k[buf][sub * 32 + col][8 * half];
      f32x16 sc = f32x16{};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(ld16(krow + ks * 16)), qreg[ks], sc, 0, 0, 0);
      // alpha = 2^(c s - b); b is the row's whole log-sum-exp, so alpha <= 1
      bf16x8 pk[2];
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int e = 0; e < 8; ++e) pk[ks][e] = static_cast<__bf16>(fast_exp2(fmaf(sc[8 * ks + e], c, -b)));
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const bf16x8 xa = v_operand<D + 32>(&sm.x[buf][sub * 32 + ks * 16][dt * 32] + v_lane);
          y[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xa, pk[ks], y[dt], 0, 0, 0);
        }
    }
  };

  constexpr std::integral_constant<int, 0> S0{};
  constexpr std::integral_constant<int, 1> S1{};
  const int n_t = (tv_end - tv_beg + KT - 1) / KT;
  if (n_t > 0) {
    // LDS buffer b holds the tile being computed; register set 1 - b holds
    // the next tile and set b receives the one after it.
    // Loads are unconditional (past the split's end they repeat its last
    // tile and are never stored), so each wait covers only the older set.
    auto tile_at = [&](int i) { return tv_beg + min(i, n_t - 1) * KT; };
    load_tile(tile_at(0), S0);
    load_tile(tile_at(1), S1);
    store_tile(0, S0);
    __syncthreads();
    for (int i = 0; i < n_t; i += 2) {
      load_tile(tile_at(i + 2), S0);
      tile(0);
      if (i + 1 < n_t) store_tile(1, S1);
      __syncthreads();
      if (i + 1 >= n_t) break;
      load_tile(tile_at(i + 3), S1);
      tile(1);
      if (i + 2 < n_t) store_tile(0, S0);
      __syncthreads();
    }
  }

  // Partial residual of this split: lane (pair, half) holds dims
  // dt*32 + 8*g4 + 4*half + 0..3 of its pair.
  if (valid) {
    float *dst = p.part + ((((int64_t)m * p.n_splits + split) * p.n_kv_heads + kvh) * p.pairs_pad + pair) * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        f32x4 v4;
#pragma unroll
        for (int i = 0; i < 4; ++i) v4[i] = y[dt][4 * g4 + i];
        *reinterpret_cast<f32x4 *>(dst + dt * 32 + 8 * g4 + 4 * half) = v4;
      }
  }
}

// One wave per (sample, KV head, pair): the split partials added in split
// order, then the squared norm.
template <int D>
__global__ __launch_bounds__(256) void residual_sum_kernel(ResidualParams p) {
  constexpr int PER = D / 64;
  const int n_pairs = p.n_q * p.group;
  const int64_t wid = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (wid >= (int64_t)p.n_samples * p.n_kv_heads * n_pairs) return;
  const int pair = (int)(wid % n_pairs);
  const int kvh = (int)((wid / n_pairs) % p.n_kv_heads);
  const int m = (int)(wid / ((int64_t)n_pairs * p.n_kv_heads));
  float yv[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) yv[i] = 0.f;
  for (int s = 0; s < p.n_splits; ++s) {
    const float *src = p.part + ((((int64_t)m * p.n_splits + s) * p.n_kv_heads + kvh) * p.pairs_pad + pair) * D;
#pragma unroll
    for (int i = 0; i < PER; ++i) yv[i] += src[lane + 64 * i];
  }
  float sq = 0.f;
#pragma unroll
  for (int i = 0; i < PER; ++i) sq = fmaf(yv[i], yv[i], sq);
  sq = wave_sum(sq);
  if (lane == 0) {
    const int r = pair / p.group, h = kvh * p.group + pair % p.group;
    p.err_out[((int64_t)m * p.n_q + r) * p.n_q_heads + h] = sq;
  }
}

// fp32 path: one wave per (sample, span row, query head) over all visual
// keys, 64 keys per step, the residual accumulated per lane over D/64 dims.
template <int D>
__global__ __launch_bounds__(64) void residual_f32_kernel(ResidualParams p) {
  constexpr int PER = D / 64;
  __shared__ float qs[D];
  const int64_t gid = blockIdx.x;  // (m * n_q + r) * n_q_heads + h
  const int lane = threadIdx.x;
  const int h = (int)(gid % p.n_q_heads);
  const int r = (int)((gid / p.n_q_heads) % p.n_q);
  const int m = (int)(gid / ((int64_t)p.n_q_heads * p.n_q));
  const int kvh = h / p.group;
  const float *Kg = static_cast<const float *>(p.k);
  const float *Xg = static_cast<const float *>(p.disp);
  const bool iso = p.vnorm != nullptr;
  const float *q = static_cast<const float *>(p.q) + ((int64_t)r * p.n_q_heads + h) * D;
  for (int e = lane; e < D; e += 64) qs[e] = q[e];
  __syncthreads();
  const float b = p.row_b[(int64_t)r * p.n_q_heads + h];
  float yv[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) yv[i] = 0.f;
  for (int base = 0; base < p.n_vis; base += 64) {
    const int t = base + lane;
    float a = 0.f;
    if (t < p.n_vis && p.refreshed[t] == 0) {
      const float *kr = Kg + kv_row(p.pages, vis_position(p.tbl, t)) * p.k_stride + kvh * D;
      float dot = 0.f;
#pragma unroll 8
      for (int e = 0; e < D; ++e) dot = fmaf(qs[e], kr[e], dot);
      a = fast_exp2(fmaf(dot, p.scale_log2, -b)) * (iso ? p.vnorm[t] * p.sigma_scale : 1.f);
    }
    const int nk = min(64, p.n_vis - base);
    for (int j = 0; j < nk; ++j) {
      const float aj = __shfl(a, j, 64);
      if (aj == 0.f) continue;  // uniform: every lane reads the same aj
      const int tj = base + j;
      const float *xr = iso ? Xg + (((int64_t)m * p.n_vis + tj) * p.n_kv_heads + kvh) * D
                            : Xg + kv_row(p.pages, vis_position(p.tbl, tj)) * p.disp_stride + kvh * D;
#pragma unroll
      for (int i = 0; i < PER; ++i) yv[i] = fmaf(aj, xr[lane + 64 * i], yv[i]);
    }
  }
  float sq = 0.f;
#pragma unroll
  for (int i = 0; i < PER; ++i) sq = fmaf(yv[i], yv[i], sq);
  sq = wave_sum(sq);
  if (lane == 0) p.err_out[gid] = sq;
}

}  // namespace

hipError_t launch_residual(const ResidualParams &p, int head_dim, bool bf16, hipStream_t s) {
  if (bf16) {
    const int n_pb = p.pairs_pad / kResidualPairs;
    dim3 grid(p.n_splits, n_pb, p.n_kv_heads * p.n_samples);
    const int64_t waves = (int64_t)p.n_samples * p.n_kv_heads * p.n_q * p.group;
    {
      ProfScope ps("residual", s);
      if (head_dim == 128) residual_bf16_kernel<128><<<grid, kThreads, 0, s>>>(p);
      else residual_bf16_kernel<64><<<grid, kThreads, 0, s>>>(p);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    ProfScope ps("residual_sum", s);
    const unsigned blocks = (unsigned)((waves + 3) / 4);
    if (head_dim == 128) residual_sum_kernel<128><<<blocks, 256, 0, s>>>(p);
    else residual_sum_kernel<64><<<blocks, 256, 0, s>>>(p);
  } else {
    ProfScope ps("residual_f32", s);
    const unsigned blocks = (unsigned)((int64_t)p.n_samples * p.n_q * p.n_q_heads);
    if (head_dim == 128) residual_f32_kernel<128><<<blocks, 64, 0, s>>>(p);
    else residual_f32_kernel<64><<<blocks, 64, 0, s>>>(p);
  }
  return hipGetLastError();
}

}  // namespace conduit
