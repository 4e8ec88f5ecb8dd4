// Causal attention of query rows over one layer's KV cache, gfx950.
//
// Two users:
//  * the scoring pass needs, for every span row, the log-sum-exp of its
//    softmax over the row's key domain before the visual column sums of
//    Eq. 6 can be normalised (statistics only, no values);
//  * the selective recompute needs, for every selected visual row, causal
//    attention over the merged fresh/stale cache (values included).
//
// bf16 path: workgroups of 8 waves (two per SIMD, so one wave's MFMAs overlap
// the other's softmax) own 256 (row, head) pairs of one KV head (grouped heads
// share the K/V tiles) and one key split.  Per 64-key tile, double-buffered in
// LDS with the next tile's global loads in flight, K is staged row-major and
// V transposed; each wave computes
// S^T = K Q^T with v_mfma_f32_32x32x16_bf16 so that every lane holds 16 keys
// of one pair column and the online softmax runs in-lane; the probabilities
// feed O^T = V^T P^T straight from the accumulator registers.  Splits write
// (m, l, O) partials in the log2 domain that a combine kernel merges in a
// fixed order (deterministic, no atomics).
#include "common.h"

namespace conduit {
namespace {

constexpr int KT = kAttnKeyTile;
constexpr float kNegInf = -__builtin_inff();
constexpr float kMInit = -1e30f;  // initial running maximum (log2 units)

template <int D>
struct AttnSmem {
  alignas(16) u16 k[2][KT][D + 8];   // K tiles, one row per key (+16 B pad against bank conflicts)
  alignas(16) u16 vt[2][D][KT + 8];  // V^T tiles, keys in MFMA-operand order
  uint64_t okmask[2];                // key-domain filter per tile, bit = key
  int maxpos, minpos;
};

__device__ __forceinline__ int row_position(const int32_t *row_pos, int q_pos0, int r) {
  return row_pos ? row_pos[r] : q_pos0 + r;
}

// Slot of key `kl` (0..63) of a tile inside a V^T row.  The S^T accumulator
// gives lane half h, register v the key 8*(v/4) + 4*h + (v%4) of a 32-key
// sub-tile; the PV product consumes registers 8*ks..8*ks+7 as one 16-deep
// k-step, so those eight keys are stored contiguously per lane half.
__device__ __forceinline__ int vt_slot(int kl) {
  const int sub = kl >> 5, w = kl & 31, ks = w >> 4, r = w & 15;
  const int h = (r & 7) >> 2, e = 4 * (r >> 3) + (r & 3);
  return sub * 32 + ks * 16 + h * 8 + e;
}

// Global -> register staging of one key tile (issued a tile ahead).
template <int D, bool PV, int W>
struct TileRegs {
  static constexpr int kThreads = W * 64;
  static constexpr int KCH = KT * D / 8 / kThreads;    // 16-byte K chunks per thread
  static constexpr int VIT = (KT / 2) * (D / 8);       // 2-key x 8-dim V items
  static constexpr int VPT = VIT >= kThreads ? VIT / kThreads : 1;  // items per thread
  u32x4 k[KCH];
  u32x4 v[PV ? 2 : 1];
  uint8_t ok;
};

// The running maximum only moves when a sub-tile's maximum exceeds it by more
// than this many log2 units; probabilities stay below 2^8 and O, l are
// rescaled rarely.  Exact: O, l and the final normaliser share the reference.
constexpr float kRescaleSlack = 8.f;

// W waves per workgroup, each owning 32 (row, head) pair columns.  With
// values (refresh) W = 8: two waves per SIMD and 256 pairs sharing each K/V
// tile; statistics only W = 4 with two workgroups per CU.
template <int D, bool PV, int W>
__global__ __launch_bounds__(W * 64, 8 / W) void attn_bf16_kernel(AttnParams p) {
  constexpr int kThreads = W * 64;
  constexpr int KS = D / 16;   // MFMA k-steps over the head dimension
  constexpr int DT = D / 32;   // 32-row tiles of O^T
  using Regs = TileRegs<D, PV, W>;
  __shared__ AttnSmem<D> sm;

  // Blocks of later rows see more keys: launch them first.
  constexpr int kPairs = W * 32;  // (row, head) pairs per workgroup
  const int split = blockIdx.x, pb = gridDim.y - 1 - blockIdx.y, kvh = blockIdx.z;
  const int G = p.group;
  const int n_pairs = p.n_rows * G;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 31, half = lane >> 5;
  const int pair0 = pb * kPairs;

  // Position range of this block's rows bounds its keys and its masking.
  if (tid == 0) {
    sm.maxpos = -1;
    sm.minpos = 0x7fffffff;
  }
  __syncthreads();
  {
    const int r_first = pair0 / G;
    const int r_last = (min(pair0 + kPairs, n_pairs) - 1) / G;
    for (int r = r_first + tid; r <= r_last; r += kThreads) {
      const int rp = row_position(p.row_pos, p.q_pos0, r);
      atomicMax(&sm.maxpos, rp);
      atomicMin(&sm.minpos, rp);
    }
  }
  __syncthreads();
  const int kbeg = split * p.chunk;
  const int kend = min(kbeg + p.chunk, sm.maxpos + 1);
  const int minpos = sm.minpos;
  if (kbeg >= kend) return;

  const u16 *Kg = static_cast<const u16 *>(p.k);
  const u16 *Vg = static_cast<const u16 *>(p.v);
  const u16 *Qg = static_cast<const u16 *>(p.q);
  const float c = p.scale_log2;

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

  // Per-thread offsets of its staging chunks inside a key tile; a tile's
  // base moves by KT rows, and only a partial last tile clamps its rows.
  int64_t koff[Regs::KCH];
#pragma unroll
  for (int i = 0; i < Regs::KCH; ++i) {
    const int cidx = tid + kThreads * i;
    koff[i] = (int64_t)(cidx / (D / 8)) * p.k_stride + kvh * D + (cidx % (D / 8)) * 8;
  }
  // V items: item = tid + kThreads * i; key pair fastest, so each half-wave
  // later writes 32 different keys of one V^T row (32 different LDS banks).
  constexpr int VPT = Regs::VPT;
  const bool v_active = Regs::VIT >= kThreads || tid < Regs::VIT;
  int v_kpair[VPT], v_dc[VPT];
  int64_t voff[VPT][2];
#pragma unroll
  for (int it = 0; it < VPT; ++it) {
    const int item = tid + kThreads * it;
    v_kpair[it] = item % (KT / 2);
    v_dc[it] = item / (KT / 2);
#pragma unroll
    for (int i = 0; i < 2; ++i)
      voff[it][i] = (int64_t)(v_kpair[it] * 2 + i) * p.v_stride + kvh * D + v_dc[it] * 8;
  }

  u32x4 rk[Regs::KCH];
  u32x4 rv[PV ? VPT : 1][2];
  bool rok = false;
  auto load_tile = [&](int t0) __attribute__((always_inline)) {
    const u16 *kb = Kg + (int64_t)t0 * p.k_stride;
    const u16 *vb = Vg + (int64_t)t0 * p.v_stride;
    if (t0 + KT <= kend) {
#pragma unroll
      for (int i = 0; i < Regs::KCH; ++i) rk[i] = ld16(kb + koff[i]);
      if constexpr (PV) {
        if (v_active) {
#pragma unroll
          for (int it = 0; it < VPT; ++it)
#pragma unroll
            for (int i = 0; i < 2; ++i) rv[it][i] = ld16(vb + voff[it][i]);
        }
      }
    } else {  // partial tile: rows past kend repeat the last row (masked later)
#pragma unroll
      for (int i = 0; i < Regs::KCH; ++i) {
        const int cidx = tid + kThreads * i;
        const int kp = min(t0 + cidx / (D / 8), kend - 1);
        rk[i] = ld16(Kg + (int64_t)kp * p.k_stride + kvh * D + (cidx % (D / 8)) * 8);
      }
      if constexpr (PV) {
        if (v_active) {
#pragma unroll
          for (int it = 0; it < VPT; ++it)
#pragma unroll
            for (int i = 0; i < 2; ++i) {
              const int kp = min(t0 + v_kpair[it] * 2 + i, kend - 1);
              rv[it][i] = ld16(Vg + (int64_t)kp * p.v_stride + kvh * D + v_dc[it] * 8);
            }
        }
      }
    }
    if (!PV && p.key_ok && tid < KT) {
      const int kp = t0 + tid;
      rok = kp < kend && p.key_ok[kp] != 0;
    }
  };
  auto store_tile = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < Regs::KCH; ++i) {
      const int cidx = tid + kThreads * i;
      st16(&sm.k[buf][cidx / (D / 8)][(cidx % (D / 8)) * 8], rk[i]);
    }
    if constexpr (PV) {
      if (v_active) {
#pragma unroll
        for (int it = 0; it < VPT; ++it) {
          const int slot = vt_slot(v_kpair[it] * 2);
          const u32x4 w0 = rv[it][0], w1 = rv[it][1];
#pragma unroll
          for (int e2 = 0; e2 < 4; ++e2) {
            // dims 2*e2 (low halves) and 2*e2+1 (high halves) of the two keys
            *reinterpret_cast<uint32_t *>(&sm.vt[buf][v_dc[it] * 8 + 2 * e2][slot]) =
                (w0[e2] & 0xffffu) | (w1[e2] << 16);
            *reinterpret_cast<uint32_t *>(&sm.vt[buf][v_dc[it] * 8 + 2 * e2 + 1][slot]) =
                (w0[e2] >> 16) | (w1[e2] & 0xffff0000u);
          }
        }
      }
    }
    if (!PV && p.key_ok && tid < KT) {  // wave 0: one bit per key of the tile
      const uint64_t bits = __ballot(rok != 0);
      if (tid == 0) sm.okmask[buf] = bits;
    }
  };

  // Running maximum (log2 units) starts finite, so exp2(c*s - m) needs no
  // special case: masked logits are -inf and give 0; the first valid
  // sub-tile always moves m.
  float m = kMInit, l = 0.f;
  f32x16 o[DT];
  if constexpr (PV) {
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[dt] = f32x16{};
  }

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

  // Online softmax of one sub-tile, then O^T += V^T P^T.
  auto softmax_pv = [&](f32x16 sc, int buf, int sub, int t0, bool masked) __attribute__((always_inline)) {
    if (masked) {  // branch-free: causal / split end and the key domain
      const int lim = min(kend - 1, rp) - t0;  // last visible key of the tile
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int kl = sub * 32 + 8 * (v >> 2) + 4 * half + (v & 3);
        bool ok = kl <= lim;
        if constexpr (!PV) {  // key-domain filter: statistics of visual-only scoring
          const uint64_t dom = p.key_ok ? sm.okmask[buf] : ~0ull;
          ok = ok & (((dom >> kl) & 1ull) != 0);
        }
        sc[v] = ok ? sc[v] : kNegInf;
      }
    }
    float mx = kNegInf;
#pragma unroll
    for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sc[v]);
    mx = half_max(mx) * c;
    const bool grow = mx > m + kRescaleSlack;
    const float alpha = grow ? fast_exp2(m - mx) : 1.f;
    m = grow ? mx : m;
    const float neg_m = -m;
#pragma unroll
    for (int v = 0; v < 16; ++v) sc[v] = fast_exp2(fmaf(sc[v], c, neg_m));
    if constexpr (PV) {
      bf16x8 pk[2];
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int e = 0; e < 8; ++e) pk[ks][e] = static_cast<__bf16>(sc[8 * ks + e]);
      // fp32 row sum (the log-sum-exp output needs it to 1e-4; summing the
      // bf16-rounded probabilities is off by up to 2^-9 when few terms dominate)
      float psum = 0.f;
#pragma unroll
      for (int v = 0; v < 16; ++v) psum += sc[v];
      l = l * alpha + psum;
      if (__ballot(grow)) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[dt] *= alpha;
      }
      bf16x8 va[2][DT];
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          va[ks][dt] = as_bf16x8(ld16(&sm.vt[buf][dt * 32 + col][sub * 32 + ks * 16 + 8 * half]));
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[ks][dt], pk[ks], o[dt], 0, 0, 0);
    } else {
      float psum = 0.f;
#pragma unroll
      for (int v = 0; v < 16; ++v) psum += sc[v];
      l = l * alpha + psum;
    }
  };

  // Double-buffered main loop: the next tile's global loads are in flight
  // while the current tile computes; one barrier per tile.  Both sub-tiles'
  // S^T MFMAs are issued before the first softmax, so the VALU work of one
  // sub-tile runs while the matrix core still works on the other.
  load_tile(kbeg);
  store_tile(0);
  __syncthreads();
  int buf = 0;
  for (int t0 = kbeg; t0 < kend; t0 += KT) {
    const bool more = t0 + KT < kend;
    if (more) load_tile(t0 + KT);
    const bool masked = (!PV && p.key_ok != nullptr) || t0 + KT > kend || t0 + KT - 1 > minpos;
    const f32x16 s0 = scores(buf, 0);
    const f32x16 s1 = scores(buf, 1);
    softmax_pv(s0, buf, 0, t0, masked);
    softmax_pv(s1, buf, 1, t0, masked);
    if (more) store_tile(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }

  // ---- write this split's partials ----
  const int64_t n_gp = (int64_t)p.n_rows * p.n_q_heads;
  const float l_tot = l + __shfl_xor(l, 32, 64);
  if (valid) {
    const int64_t idx = (int64_t)split * n_gp + gpair;
    if (half == 0) {
      p.part_m[idx] = m;
      p.part_l[idx] = l_tot;
    }
    if constexpr (PV) {
      float *dst = p.part_o + idx * D;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          f32x4 w = {o[dt][4 * g], o[dt][4 * g + 1], o[dt][4 * g + 2], o[dt][4 * g + 3]};
          *reinterpret_cast<f32x4 *>(dst + dt * 32 + 8 * g + 4 * half) = w;
        }
    }
  }
}

// Merge split partials: M = max m_s, L = sum l_s 2^(m_s - M),
// O = sum O_s 2^(m_s - M) / L.  Splits 0..pos/chunk hold the row's keys.
template <int D>
__global__ __launch_bounds__(256) void combine_kernel(CombineParams p) {
  constexpr int NC = D / 4;
  const int64_t n_gp = (int64_t)p.n_rows * p.n_q_heads;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const bool values = p.part_o != nullptr;
  const int64_t gp = values ? gid / NC : gid;
  const int c = values ? (int)(gid % NC) : 0;
  if (gp >= n_gp) return;
  const int r = (int)(gp / p.n_q_heads);
  const int pos = p.row_pos ? p.row_pos[r] : p.q_pos0 + r;
  const int ns = pos / p.chunk + 1;
  float M = kNegInf;
  for (int s = 0; s < ns; ++s) M = fmaxf(M, p.part_m[s * n_gp + gp]);
  float L = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < ns; ++s) {
    const float ms = p.part_m[s * n_gp + gp];
    const float w = fast_exp2(ms - M);  // m >= kMInit is finite
    L += w * p.part_l[s * n_gp + gp];
    if (values) acc += w * *reinterpret_cast<const f32x4 *>(p.part_o + (s * n_gp + gp) * D + 4 * c);
  }
  const float b = M + __log2f(L);
  if (c == 0) {
    if (p.row_b) p.row_b[gp] = b;
    if (p.lse_out) p.lse_out[gp] = b * kLn2;
  }
  if (values) {
    const float inv = 1.f / L;
    if (p.o_bf16) {
      u16 *out = static_cast<u16 *>(p.o_out) + gp * D + 4 * c;
      uint2 w;
      w.x = (uint32_t)f32_to_bf16(acc[0] * inv) | ((uint32_t)f32_to_bf16(acc[1] * inv) << 16);
      w.y = (uint32_t)f32_to_bf16(acc[2] * inv) | ((uint32_t)f32_to_bf16(acc[3] * inv) << 16);
      *reinterpret_cast<uint2 *>(out) = w;
    } else {
      *reinterpret_cast<f32x4 *>(static_cast<float *>(p.o_out) + gp * D + 4 * c) = acc * inv;
    }
  }
}

// fp32 path: one wave per (row, head) pair over the whole causal key range,
// 64 keys per step (one per lane), written straight to the final outputs.
template <int D, bool PV>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnParams p, CombineParams out) {
  constexpr int PER = D / 64;
  __shared__ float qs[D];
  const int64_t gp = blockIdx.x;
  const int lane = threadIdx.x;
  const int r = (int)(gp / p.n_q_heads), hq = (int)(gp % p.n_q_heads), kvh = hq / p.group;
  const int rpos = row_position(p.row_pos, p.q_pos0, r);
  const float *Kg = static_cast<const float *>(p.k);
  const float *Vg = static_cast<const float *>(p.v);
  const float *q = static_cast<const float *>(p.q) + gp * D;
  for (int e = lane; e < D; e += 64) qs[e] = q[e];
  __syncthreads();
  float m = kNegInf, l = 0.f, o[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) o[i] = 0.f;
  for (int base = 0; base <= rpos; base += 64) {
    const int kp = base + lane;
    const bool ok = kp <= rpos && (p.key_ok == nullptr || p.key_ok[kp]);
    float z = kNegInf;
    if (ok) {
      const float *kr = Kg + (int64_t)kp * p.k_stride + kvh * D;
      float dot = 0.f;
#pragma unroll 8
      for (int e = 0; e < D; ++e) dot = fmaf(qs[e], kr[e], dot);
      z = dot * p.scale_log2;
    }
    const float m_new = fmaxf(m, wave_max(z));
    const float m_use = (m_new == kNegInf) ? 0.f : m_new;
    const float alpha = fast_exp2(m - m_use);
    const float e = fast_exp2(z - m_use);
    l = l * alpha + wave_sum(e);
    m = m_new;
    if constexpr (PV) {
#pragma unroll
      for (int i = 0; i < PER; ++i) o[i] *= alpha;
      const int nk = min(64, rpos - base + 1);
      for (int j = 0; j < nk; ++j) {
        const float pj = __shfl(e, j, 64);
        const float *vr = Vg + (int64_t)(base + j) * p.v_stride + kvh * D;
#pragma unroll
        for (int i = 0; i < PER; ++i) o[i] = fmaf(pj, vr[lane + 64 * i], o[i]);
      }
    }
  }
  const float b = m + __log2f(l);
  if (lane == 0) {
    if (out.row_b) out.row_b[gp] = b;
    if (out.lse_out) out.lse_out[gp] = b * kLn2;
  }
  if constexpr (PV) {
    const float inv = 1.f / l;
    float *dst = static_cast<float *>(out.o_out) + gp * D;
#pragma unroll
    for (int i = 0; i < PER; ++i) dst[lane + 64 * i] = o[i] * inv;
  }
}

__global__ void lse_to_b_kernel(const float *lse, float *b, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) b[i] = lse[i] * kLog2e;
}

}  // namespace

hipError_t launch_attn(const AttnParams &p, int head_dim, bool bf16, bool with_values, hipStream_t s) {
  const int n_pairs = p.n_rows * p.group;
  if (!bf16) return hipErrorInvalidValue;
  // refresh: 8 waves (256 pairs share each K/V tile); statistics: 4 waves,
  // two workgroups per CU (many short splits)
  const dim3 grid_v(p.n_split, (n_pairs + attn_pairs_per_block(true) - 1) / attn_pairs_per_block(true),
                    p.n_kv_heads);
  const dim3 grid_s(p.n_split, (n_pairs + attn_pairs_per_block(false) - 1) / attn_pairs_per_block(false),
                    p.n_kv_heads);
  if (head_dim == 128) {
    if (with_values) attn_bf16_kernel<128, true, 8><<<grid_v, 8 * 64, 0, s>>>(p);
    else attn_bf16_kernel<128, false, 4><<<grid_s, 4 * 64, 0, s>>>(p);
  } else {
    if (with_values) attn_bf16_kernel<64, true, 8><<<grid_v, 8 * 64, 0, s>>>(p);
    else attn_bf16_kernel<64, false, 4><<<grid_s, 4 * 64, 0, s>>>(p);
  }
  return hipGetLastError();
}

hipError_t launch_combine(const CombineParams &p, int head_dim, hipStream_t s) {
  const int64_t n_gp = (int64_t)p.n_rows * p.n_q_heads;
  const int64_t n = p.part_o ? n_gp * (head_dim / 4) : n_gp;
  const int blocks = (int)((n + 255) / 256);
  if (head_dim == 128) combine_kernel<128><<<blocks, 256, 0, s>>>(p);
  else combine_kernel<64><<<blocks, 256, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_attn_f32(const AttnParams &p, const CombineParams &out, int head_dim,
                           bool with_values, hipStream_t s) {
  const int64_t n_gp = (int64_t)p.n_rows * p.n_q_heads;
  if (head_dim == 128) {
    if (with_values) attn_f32_kernel<128, true><<<n_gp, 64, 0, s>>>(p, out);
    else attn_f32_kernel<128, false><<<n_gp, 64, 0, s>>>(p, out);
  } else {
    if (with_values) attn_f32_kernel<64, true><<<n_gp, 64, 0, s>>>(p, out);
    else attn_f32_kernel<64, false><<<n_gp, 64, 0, s>>>(p, out);
  }
  return hipGetLastError();
}

hipError_t launch_lse_to_b(const float *lse_in, float *row_b, int32_t n, hipStream_t s) {
  lse_to_b_kernel<<<(n + 255) / 256, 256, 0, s>>>(lse_in, row_b, n);
  return hipGetLastError();
}

}  // namespace conduit
