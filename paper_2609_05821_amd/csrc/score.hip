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

// Q row blocks stream through two LDS slots; block x is fetched into
// register set x mod 3, three blocks ahead of its use, so the global load
// latency hides behind the MFMA and exponential work of the blocks in
// between (one barrier per block).
constexpr int kQAhead = 3;

template <int D>
__global__ __launch_bounds__(kColsumThreads) void colsum_bf16_kernel(ColsumParams p) {
  constexpr int KS = D / 16;
  constexpr int QCH = 32 * D / 8;       // 16-byte chunks in a 32-row Q block
  __shared__ alignas(16) u16 qs[2][32][D + 8];
  __shared__ alignas(16) float bs[2][32];
  __shared__ ImageLds img;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 31, half = lane >> 5;
  const int kvh = blockIdx.y;
  const int G = p.group;
  const int n_pair = p.n_q * G;
  const int nblk = (n_pair + 31) / 32;
  const u16 *Kg = static_cast<const u16 *>(p.k);
  const u16 *Vg = static_cast<const u16 *>(p.v);
  const u16 *Qg = static_cast<const u16 *>(p.q);

  // Cooperative load of row block `blk` (32 (span token, head) rows).
  auto load_q = [&](int blk, u32x4 &qv, float &bv) __attribute__((always_inline)) {
    if (blk >= nblk) return;
    if (tid < QCH) {
      const int row = tid / (D / 8), dc = tid % (D / 8);
      const int pr = blk * 32 + row;
      qv = u32x4{0, 0, 0, 0};
      if (pr < n_pair) {
        const int i = pr / G, hq = kvh * G + pr % G;
        qv = ld16(Qg + ((int64_t)i * p.n_q_heads + hq) * D + dc * 8);
      }
    }
    if (tid < 32) {
      const int pr = blk * 32 + tid;
      bv = kInf;  // padding rows contribute 2^-inf = 0
      if (pr < n_pair) bv = p.row_b[(pr / G) * p.n_q_heads + kvh * G + pr % G];
    }
  };
  auto store_q = [&](int slot, const u32x4 &qv, float bv) __attribute__((always_inline)) {
    if (tid < QCH) st16(&qs[slot][tid / (D / 8)][(tid % (D / 8)) * 8], qv);
    if (tid < 32) bs[slot][tid] = bv;
  };

  u32x4 qv[kQAhead];
  float bv[kQAhead];
#pragma unroll
  for (int i = 0; i < kQAhead; ++i) {
    qv[i] = u32x4{0, 0, 0, 0};
    bv[i] = kInf;
    load_q(i, qv[i], bv[i]);
  }

  // This lane's key column, held as the B operand for every row block.
  image_table_to_lds(p.tbl, img, tid, kColsumThreads);
  __syncthreads();
  const int t = blockIdx.x * kColsumKeysPerBlock + wave * 32 + col;
  const bool tvalid = t < p.n_vis;
  bf16x8 kreg[KS];
  {
    const u16 *krow = Kg + (int64_t)(tvalid ? vis_position(img, t) : 0) * p.k_stride + kvh * D + 8 * half;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      kreg[ks] = as_bf16x8(tvalid ? ld16(krow + ks * 16) : u32x4{0, 0, 0, 0});
  }
  store_q(0, qv[0], bv[0]);
  load_q(kQAhead, qv[0], bv[0]);
  __syncthreads();

  float colsum = 0.f;
  // Block b: compute from slot b & 1, then store block b + 1 (register set
  // (b + 1) % 3) into the other slot and fetch block b + 4 into that set.
  auto step = [&](int b, auto j_tag) __attribute__((always_inline)) {
    constexpr int J = decltype(j_tag)::value;  // == (b + 1) % 3
    if (b >= nblk) return;
    const int slot = b & 1;
    f32x16 acc = f32x16{};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const bf16x8 a = as_bf16x8(ld16(&qs[slot][col][ks * 16 + 8 * half]));
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, kreg[ks], acc, 0, 0, 0);
    }
    // lane (col, half), register v holds row 8*(v/4) + 4*half + v%4
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4 bb = *reinterpret_cast<const f32x4 *>(&bs[slot][8 * g + 4 * half]);
#pragma unroll
      for (int i = 0; i < 4; ++i) colsum += fast_exp2(fmaf(acc[4 * g + i], p.scale_log2, -bb[i]));
    }
    if (b + 1 < nblk) {
      store_q(slot ^ 1, qv[J], bv[J]);
      load_q(b + 1 + kQAhead, qv[J], bv[J]);
    }
    __syncthreads();
  };
  for (int b = 0; b < nblk; b += 3) {
    step(b, std::integral_constant<int, 1>{});
    step(b + 1, std::integral_constant<int, 2>{});
    step(b + 2, std::integral_constant<int, 0>{});
  }
  colsum += __shfl_xor(colsum, 32, 64);
  if (half == 0 && tvalid) p.colsum_part[(int64_t)kvh * p.n_vis + t] = colsum;

  // Value-norm proxy: this head's share of ||V_t||^2, two threads per key.
  {
    const int kk = tid >> 1, part = tid & 1;
    const int tv = blockIdx.x * kColsumKeysPerBlock + kk;
    float sq = 0.f;
    if (tv < p.n_vis) {
      const u16 *vrow = Vg + (int64_t)vis_position(img, tv) * p.v_stride + kvh * D + part * (D / 2);
#pragma unroll
      for (int c = 0; c < D / 16; ++c) {
        const u32x4 ws = ld16(vrow + c * 8);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float lo = __builtin_bit_cast(float, ws[e] << 16);
          const float hi = __builtin_bit_cast(float, ws[e] & 0xffff0000u);
          sq = fmaf(lo, lo, sq);
          sq = fmaf(hi, hi, sq);
        }
      }
    }
    sq += __shfl_xor(sq, 1, 64);
    if (part == 0 && tv < p.n_vis) p.vsq_part[(int64_t)kvh * p.n_vis + tv] = sq;
  }
}

// fp32 path: one thread per (visual key, KV head).
template <int D>
__global__ __launch_bounds__(64) void colsum_f32_kernel(ColsumParams p) {
  const int t = blockIdx.x * 64 + threadIdx.x;
  const int kvh = blockIdx.y;
  if (t >= p.n_vis) return;
  const float *Kg = static_cast<const float *>(p.k);
  const float *Vg = static_cast<const float *>(p.v);
  const float *Qg = static_cast<const float *>(p.q);
  const int64_t pos = vis_position(p.tbl, t);
  float kr[D];
#pragma unroll
  for (int e = 0; e < D; ++e) kr[e] = Kg[pos * p.k_stride + kvh * D + e];
  float colsum = 0.f;
  const int n_pair = p.n_q * p.group;
  for (int pr = 0; pr < n_pair; ++pr) {
    const int i = pr / p.group, hq = kvh * p.group + pr % p.group;
    const float *q = Qg + ((int64_t)i * p.n_q_heads + hq) * D;
    float dot = 0.f;
#pragma unroll
    for (int e = 0; e < D; ++e) dot = fmaf(q[e], kr[e], dot);
    colsum += fast_exp2(fmaf(dot, p.scale_log2, -p.row_b[(int64_t)i * p.n_q_heads + hq]));
  }
  float sq = 0.f;
  const float *vr = Vg + pos * p.v_stride + kvh * D;
#pragma unroll 8
  for (int e = 0; e < D; ++e) sq = fmaf(vr[e], vr[e], sq);
  p.colsum_part[(int64_t)kvh * p.n_vis + t] = colsum;
  p.vsq_part[(int64_t)kvh * p.n_vis + t] = sq;
}

__global__ void finalize_kernel(FinalizeParams p) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= p.n_vis) return;
  float cs = 0.f, sq = 0.f;
  for (int h = 0; h < p.n_kv_heads; ++h) {
    cs += p.colsum_part[(int64_t)h * p.n_vis + t];
    sq += p.vsq_part[(int64_t)h * p.n_vis + t];
  }
  const float a = cs / p.n_rows_f;
  const float v = sqrtf(sq);
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

}  // namespace

hipError_t launch_colsum(const ColsumParams &p, int head_dim, bool bf16, hipStream_t s) {
  if (bf16) {
    dim3 grid((p.n_vis + kColsumKeysPerBlock - 1) / kColsumKeysPerBlock, p.n_kv_heads);
    ProfScope ps("colsum", s);
    if (head_dim == 128) colsum_bf16_kernel<128><<<grid, kColsumThreads, 0, s>>>(p);
    else colsum_bf16_kernel<64><<<grid, kColsumThreads, 0, s>>>(p);
  } else {
    dim3 grid((p.n_vis + 63) / 64, p.n_kv_heads);
    ProfScope ps("colsum_f32", s);
    if (head_dim == 128) colsum_f32_kernel<128><<<grid, 64, 0, s>>>(p);
    else colsum_f32_kernel<64><<<grid, 64, 0, s>>>(p);
  }
  return hipGetLastError();
}

hipError_t launch_finalize(const FinalizeParams &p, hipStream_t s) {
  ProfScope ps("finalize", s);
  finalize_kernel<<<(p.n_vis + 255) / 256, 256, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace conduit
