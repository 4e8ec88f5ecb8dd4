// Causal attention of query rows over one layer's KV cache, gfx950.
//
// Two users:
//  * the scoring pass needs, for every span row, the log-sum-exp of its
//    softmax over the row's key domain before the visual column sums of
//    Eq. 6 can be normalised (statistics only, no values);
//  * the selective recompute needs, for every selected visual row, causal
//    attention over the merged fresh/stale cache (values included).
//
// bf16 path: workgroups of 4 waves own 256 (row, head) pairs of one KV head
// (grouped heads share the K/V tiles) and one key split.  Per 64-key tile,
// K is staged in LDS row-major and V transposed; each wave computes
// S^T = K Q^T with v_mfma_f32_32x32x16_bf16 so that every lane holds 16 keys
// of one pair column and the online softmax runs in-lane; the probabilities
// feed O^T = V^T P^T straight from the accumulator registers.  Splits write
// (m, l, O) partials in the log2 domain that a combine kernel merges in a
// fixed order (deterministic, no atomics).
#include "common.h"

namespace conduit {
namespace {

constexpr int kThreads = 256;
constexpr int KT = kAttnKeyTile;
constexpr float kNegInf = -__builtin_inff();

template <int D>
struct AttnSmem {
  u16 k[KT][D + 8];   // K tile, one row per key (+16 B pad against bank conflicts)
  u16 vt[D][KT + 8];  // V^T tile, keys in MFMA-operand order
  uint8_t ok[KT];     // key-domain filter for the tile
  int maxpos;
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

template <int D, bool PV>
__global__ __launch_bounds__(kThreads, 1) void attn_bf16_kernel(AttnParams p) {
  constexpr int KS = D / 16;   // MFMA k-steps over the head dimension
  constexpr int DT = D / 32;   // 32-row tiles of O^T
  __shared__ AttnSmem<D> sm;

  const int split = blockIdx.x, pb = blockIdx.y, kvh = blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 31, half = lane >> 5;
  const int G = p.group;
  const int n_pairs = p.n_rows * G;
  const int pair0 = pb * kAttnPairsPerBlock;

  // Largest position among this block's rows bounds its key range.
  if (tid == 0) sm.maxpos = -1;
  __syncthreads();
  {
    const int r_first = pair0 / G;
    const int r_last = (min(pair0 + kAttnPairsPerBlock, n_pairs) - 1) / G;
    for (int r = r_first + tid; r <= r_last; r += kThreads)
      atomicMax(&sm.maxpos, row_position(p.row_pos, p.q_pos0, r));
  }
  __syncthreads();
  const int kbeg = split * p.chunk;
  const int kend = min(kbeg + p.chunk, sm.maxpos + 1);
  if (kbeg >= kend) return;

  const u16 *Kg = static_cast<const u16 *>(p.k);
  const u16 *Vg = static_cast<const u16 *>(p.v);
  const u16 *Qg = static_cast<const u16 *>(p.q);

  // Pair columns owned by this lane: two 32-wide tiles per wave.
  int rp[2], gpair[2];
  bool valid[2];
  bf16x8 qreg[2][KS];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    const int pair = pair0 + wave * 64 + nt * 32 + col;
    valid[nt] = pair < n_pairs;
    const int r = valid[nt] ? pair / G : 0;
    const int hq = kvh * G + (valid[nt] ? pair % G : 0);
    gpair[nt] = r * p.n_q_heads + hq;
    rp[nt] = valid[nt] ? row_position(p.row_pos, p.q_pos0, r) : -1;
    const u16 *qrow = Qg + (int64_t)gpair[nt] * D + 8 * half;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      uint4 v = valid[nt] ? *reinterpret_cast<const uint4 *>(qrow + ks * 16) : make_uint4(0, 0, 0, 0);
      qreg[nt][ks] = as_bf16x8(v);
    }
  }

  float m[2] = {kNegInf, kNegInf}, l[2] = {0.f, 0.f};
  f32x16 o[2][DT];
  if constexpr (PV) {
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) o[nt][dt] = f32x16{};
  }

  for (int t0 = kbeg; t0 < kend; t0 += KT) {
    __syncthreads();  // previous tile fully consumed
    // ---- stage K (row-major) ----
    constexpr int KCH = KT * D / 8;  // 16-byte chunks in a K tile
#pragma unroll
    for (int c = tid; c < KCH; c += kThreads) {
      const int key = c / (D / 8), dc = c % (D / 8);
      const int kp = t0 + key;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (kp < kend) v = *reinterpret_cast<const uint4 *>(Kg + (int64_t)kp * p.k_stride + kvh * D + dc * 8);
      *reinterpret_cast<uint4 *>(&sm.k[key][dc * 8]) = v;
    }
    // ---- stage V transposed: a thread takes 4 consecutive keys x 8 dims ----
    if constexpr (PV) {
      constexpr int VIT = (KT / 4) * (D / 8);
      for (int c = tid; c < VIT; c += kThreads) {
        const int dc = c % (D / 8), quad = c / (D / 8);
        u16 vals[4][8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int kp = t0 + quad * 4 + i;
          uint4 v = make_uint4(0, 0, 0, 0);
          if (kp < kend) v = *reinterpret_cast<const uint4 *>(Vg + (int64_t)kp * p.v_stride + kvh * D + dc * 8);
          *reinterpret_cast<uint4 *>(vals[i]) = v;
        }
        const int slot = vt_slot(quad * 4);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          uint2 w;
          w.x = (uint32_t)vals[0][e] | ((uint32_t)vals[1][e] << 16);
          w.y = (uint32_t)vals[2][e] | ((uint32_t)vals[3][e] << 16);
          *reinterpret_cast<uint2 *>(&sm.vt[dc * 8 + e][slot]) = w;
        }
      }
    }
    if (tid < KT) {
      const int kp = t0 + tid;
      sm.ok[tid] = (kp < kend) && (p.key_ok == nullptr || p.key_ok[kp]);
    }
    __syncthreads();

    // ---- S^T = K Q^T for two 32-key sub-tiles x two pair tiles ----
    f32x16 s[2][2];
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      s[sub][0] = f32x16{};
      s[sub][1] = f32x16{};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 a = as_bf16x8(*reinterpret_cast<const uint4 *>(&sm.k[sub * 32 + col][ks * 16 + 8 * half]));
        s[sub][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[0][ks], s[sub][0], 0, 0, 0);
        s[sub][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[1][ks], s[sub][1], 0, 0, 0);
      }
    }

    // ---- online softmax, in-lane over 32 keys per pair column ----
    bf16x8 pk[2][2][2];  // [sub][nt][ks] probabilities as PV operands
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      float mx = kNegInf;
#pragma unroll
      for (int sub = 0; sub < 2; ++sub)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int kl = sub * 32 + 8 * (v >> 2) + 4 * half + (v & 3);
          const bool ok = sm.ok[kl] && (t0 + kl <= rp[nt]);
          const float z = ok ? s[sub][nt][v] * p.scale_log2 : kNegInf;
          s[sub][nt][v] = z;
          mx = fmaxf(mx, z);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m[nt], mx);
      const float m_use = (m_new == kNegInf) ? 0.f : m_new;
      const float alpha = fast_exp2(m[nt] - m_use);
      float psum = 0.f;
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float e = fast_exp2(s[sub][nt][v] - m_use);
          s[sub][nt][v] = e;
          psum += e;
        }
        if constexpr (PV) {
#pragma unroll
          for (int ks = 0; ks < 2; ++ks) {
            bf16x8 b;
#pragma unroll
            for (int e = 0; e < 8; ++e) b[e] = static_cast<__bf16>(s[sub][nt][8 * ks + e]);
            pk[sub][nt][ks] = b;
          }
        }
      }
      l[nt] = l[nt] * alpha + psum;
      m[nt] = m_new;
      if constexpr (PV) {
        if (alpha != 1.f) {
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) o[nt][dt] *= alpha;
        }
      }
    }

    // ---- O^T += V^T P^T ----
    if constexpr (PV) {
#pragma unroll
      for (int sub = 0; sub < 2; ++sub)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) {
            const bf16x8 a = as_bf16x8(
                *reinterpret_cast<const uint4 *>(&sm.vt[dt * 32 + col][sub * 32 + ks * 16 + 8 * half]));
            o[0][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pk[sub][0][ks], o[0][dt], 0, 0, 0);
            o[1][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pk[sub][1][ks], o[1][dt], 0, 0, 0);
          }
    }
  }

  // ---- write this split's partials ----
  const int64_t n_gp = (int64_t)p.n_rows * p.n_q_heads;
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    const float l_tot = l[nt] + __shfl_xor(l[nt], 32, 64);
    if (!valid[nt]) continue;
    const int64_t idx = (int64_t)split * n_gp + gpair[nt];
    if (half == 0) {
      p.part_m[idx] = m[nt];
      p.part_l[idx] = l_tot;
    }
    if constexpr (PV) {
      float *dst = p.part_o + idx * D;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          f32x4 w = {o[nt][dt][4 * g], o[nt][dt][4 * g + 1], o[nt][dt][4 * g + 2], o[nt][dt][4 * g + 3]};
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
    const float w = (ms == kNegInf) ? 0.f : fast_exp2(ms - M);
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
  dim3 grid(p.n_split, (n_pairs + kAttnPairsPerBlock - 1) / kAttnPairsPerBlock, p.n_kv_heads);
  if (!bf16) return hipErrorInvalidValue;
  if (head_dim == 128) {
    if (with_values) attn_bf16_kernel<128, true><<<grid, kThreads, 0, s>>>(p);
    else attn_bf16_kernel<128, false><<<grid, kThreads, 0, s>>>(p);
  } else {
    if (with_values) attn_bf16_kernel<64, true><<<grid, kThreads, 0, s>>>(p);
    else attn_bf16_kernel<64, false><<<grid, kThreads, 0, s>>>(p);
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
