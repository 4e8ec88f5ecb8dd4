// Image reweighting and global top-k, gfx950 (Sec. 3.4 Eq. 8-9, Sec. 3.5
// Eq. 10-11, the tail of Algorithm 1).
//
// One workgroup of 1024 threads:
//  1. g_j = sum_{t in V_j} A_t / (|L| n_j): one wave per image, lane-strided
//     partial sums and a butterfly reduction (fixed order);
//  2. g_bar and c_j = (1 - lambda) + lambda g_j / g_bar  (c_j = 1 if g_bar = 0);
//  3. s_hat_t = (s_t / |L|) c_pi(t), written once;
//  4. the k-th largest s_hat by radix select on the fp32 bit patterns
//     (s_hat >= 0, so unsigned bit order is value order): the bits every key
//     shares first (block AND/OR), then 11-bit passes over the rest with LDS
//     histograms (integer atomics: exact);
//  5. ordered compaction: everything above the threshold plus the first
//     `need` entries equal to it in index order (ties to the lower index),
//     with one block scan of both counts, so idx/pos come out ascending.
// The explicit-quota rule (select_explicit_kernel) shares steps 1-2.
#include "common.h"

namespace conduit {
namespace {

constexpr int kSelThreads = 1024;
constexpr int kWaves = kSelThreads / 64;

__device__ __forceinline__ uint32_t order_key(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  return u == 0x80000000u ? 0u : u;  // -0 ranks as +0
}

// Exclusive scan of one int per thread over the block; also returns the total.
__device__ int block_exclusive_scan(int x, int *s_wave, int &total) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int inc = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(inc, o, 64);
    if (lane >= o) inc += y;
  }
  if (lane == 63) s_wave[w] = inc;
  __syncthreads();
  if (w == 0) {
    int v = lane < kWaves ? s_wave[lane] : 0;
#pragma unroll
    for (int o = 1; o < kWaves; o <<= 1) {
      const int y = __shfl_up(v, o, 64);
      if (lane >= o) v += y;
    }
    if (lane < kWaves) s_wave[lane] = v;
  }
  __syncthreads();
  const int excl = inc - x + (w > 0 ? s_wave[w - 1] : 0);
  total = s_wave[kWaves - 1];
  __syncthreads();
  return excl;
}

// Bitwise AND and OR of one value per thread over the block in one
// exchange (every thread gets both).
__device__ void block_and_or(uint32_t &a, uint32_t &o, int *s_a, int *s_o) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    a &= __shfl_xor(a, off, 64);
    o |= __shfl_xor(o, off, 64);
  }
  if (lane == 0) {
    s_a[w] = (int)a;
    s_o[w] = (int)o;
  }
  __syncthreads();
  a = 0xffffffffu;
  o = 0;
  for (int i = 0; i < kWaves; ++i) {
    a &= (uint32_t)s_a[i];
    o |= (uint32_t)s_o[i];
  }
  __syncthreads();
}

// Bitwise AND / OR of one value per thread over the block (every thread
// gets the result).
__device__ uint32_t block_and(uint32_t x, int *s_wave) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x &= __shfl_xor(x, o, 64);
  if (lane == 0) s_wave[w] = (int)x;
  __syncthreads();
  uint32_t r = 0xffffffffu;
  for (int i = 0; i < kWaves; ++i) r &= (uint32_t)s_wave[i];
  __syncthreads();
  return r;
}

__device__ uint32_t block_or(uint32_t x, int *s_wave) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x |= __shfl_xor(x, o, 64);
  if (lane == 0) s_wave[w] = (int)x;
  __syncthreads();
  uint32_t r = 0;
  for (int i = 0; i < kWaves; ++i) r |= (uint32_t)s_wave[i];
  __syncthreads();
  return r;
}

constexpr int kSelBatch = 8;  // strided scores loaded together per thread
constexpr int kSelSeg = 16;   // consecutive scores loaded together in the compaction
__global__ __launch_bounds__(kSelThreads) void select_kernel(SelectParams p, ImageTable tbl) {
  __shared__ float s_g[kMaxImages];
  __shared__ float s_c[kMaxImages];
  __shared__ int hist[2048];
  __shared__ int s_wave[kWaves];
  __shared__ int s_wave2[kWaves];
  __shared__ int s_bin, s_above;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = tbl.n_vis, K = tbl.n_images;
  const float n_layers = (float)p.n_layers;

  // 1. per-image mean attention (each lane sums its tokens in order)
  for (int j = wave; j < K; j += kWaves) {
    const int lo = tbl.off[j], hi = tbl.off[j + 1];
    float acc = 0.f;
    for (int t0 = lo + lane; t0 < hi; t0 += 64 * kSelBatch) {
      float v[kSelBatch];
#pragma unroll
      for (int u = 0; u < kSelBatch; ++u) v[u] = t0 + 64 * u < hi ? p.a_acc[t0 + 64 * u] : 0.f;
#pragma unroll
      for (int u = 0; u < kSelBatch; ++u)
        if (t0 + 64 * u < hi) acc += v[u];
    }
    acc = wave_sum(acc);
    if (lane == 0) s_g[j] = acc / (n_layers * (float)(hi - lo));
  }
  __syncthreads();
  // 2. coefficients
  if (wave == 0) {
    float acc = 0.f;
    for (int j = lane; j < K; j += 64) acc += s_g[j];
    const float g_bar = wave_sum(acc) / (float)K;
    for (int j = lane; j < K; j += 64) {
      // (1 - lambda) + lambda * x adds two non-negative terms, so it keeps full
      // relative precision even for c << 1; x == 1 (one image, or an image at
      // the mean) gives exactly 1.
      const float x = s_g[j] / g_bar;
      const float c = (g_bar == 0.f || x == 1.f) ? 1.f : (1.f - p.lambda) + p.lambda * x;
      s_c[j] = c;
      if (p.c_out) p.c_out[j] = c;
    }
  }
  __syncthreads();
  // 3. composite scores
  for (int j = wave; j < K; j += kWaves) {
    const int lo = tbl.off[j], hi = tbl.off[j + 1];
    const float c = s_c[j];
    for (int t0 = lo + lane; t0 < hi; t0 += 64 * kSelBatch) {
      float v[kSelBatch];
#pragma unroll
      for (int u = 0; u < kSelBatch; ++u) v[u] = t0 + 64 * u < hi ? p.s_acc[t0 + 64 * u] : 0.f;
#pragma unroll
      for (int u = 0; u < kSelBatch; ++u)
        if (t0 + 64 * u < hi) p.shat[t0 + 64 * u] = (v[u] / n_layers) * c;
    }
  }
  __syncthreads();

  // 4. radix select of the k-th largest key.  The bits every key shares
  // come first (block AND/OR); the rest are resolved 11 bits per pass, so
  // the first digit spreads over the bits that vary (scores in a narrow
  // range share their sign and high exponent bits, and a digit made of
  // those would send nearly every LDS atomic to a few bins).
  // Loops over the scores load kSelBatch of them before using any (one
  // memory round trip per batch instead of one per score).
  uint32_t k_and = 0xffffffffu, k_or = 0;
  for (int t0 = tid; t0 < n; t0 += kSelBatch * kSelThreads) {
    float v[kSelBatch];
#pragma unroll
    for (int u = 0; u < kSelBatch; ++u) v[u] = t0 + u * kSelThreads < n ? p.shat[t0 + u * kSelThreads] : 0.f;
#pragma unroll
    for (int u = 0; u < kSelBatch; ++u)
      if (t0 + u * kSelThreads < n) {
        const uint32_t key = order_key(v[u]);
        k_and &= key;
        k_or |= key;
      }
  }
  block_and_or(k_and, k_or, s_wave, s_wave2);
  const uint32_t varying = k_and ^ k_or;
  uint32_t prefix = k_and, pmask = 0xffffffffu;
  int kk = p.k;
  const int top = varying ? 31 - __builtin_clz(varying) : -1;
  if (varying) {
    pmask = top == 31 ? 0u : ~((2u << top) - 1u);  // shared high bits
    prefix = k_and & pmask;
  }
  for (int hi = top; hi >= 0; hi -= 11) {  // digit = bits hi .. hi-10 (fewer at the end)
    const int sh = hi - 10, nb = 2048;
    for (int b = tid; b < nb; b += kSelThreads) hist[b] = 0;
    __syncthreads();
    for (int t0 = tid; t0 < n; t0 += kSelBatch * kSelThreads) {
      float v[kSelBatch];
#pragma unroll
      for (int u = 0; u < kSelBatch; ++u) v[u] = t0 + u * kSelThreads < n ? p.shat[t0 + u * kSelThreads] : 0.f;
#pragma unroll
      for (int u = 0; u < kSelBatch; ++u) {
        const uint32_t key = order_key(v[u]);
        if (t0 + u * kSelThreads < n && (key & pmask) == prefix)
          atomicAdd(&hist[(sh >= 0 ? key >> sh : key << (-sh)) & (nb - 1)], 1);
      }
    }
    __syncthreads();
    // thread tid owns bins in descending order: nb-1-per*tid .. nb-per*(tid+1)
    const int per = nb / kSelThreads;
    int local = 0;
    for (int i = 0; i < per; ++i) local += hist[nb - 1 - per * tid - i];
    int total;
    int run = block_exclusive_scan(local, s_wave, total);
    for (int i = 0; i < per; ++i) {
      const int b = nb - 1 - per * tid - i;
      const int h = hist[b];
      if (run < kk && run + h >= kk) {
        s_bin = b;
        s_above = run;
      }
      run += h;
    }
    __syncthreads();
    if (sh >= 0) {
      prefix |= (uint32_t)s_bin << sh;
      pmask |= (uint32_t)(nb - 1) << sh;
    } else {  // last, partial digit
      prefix |= (uint32_t)s_bin >> (-sh);
      pmask |= (uint32_t)(nb - 1) >> (-sh);
    }
    kk -= s_above;
    __syncthreads();
  }
  const uint32_t tau = prefix;
  const int need_eq = kk;  // entries equal to tau to take, lowest indices first

  // 5. ordered compaction over contiguous per-thread segments
  const int seg = (n + kSelThreads - 1) / kSelThreads;
  const int lo = min(n, tid * seg), hi = min(n, lo + seg);
  int gt = 0, eq = 0;
  for (int t0 = lo; t0 < hi; t0 += kSelSeg) {
    float v[kSelSeg];
#pragma unroll
    for (int u = 0; u < kSelSeg; ++u) v[u] = t0 + u < hi ? p.shat[t0 + u] : 0.f;
#pragma unroll
    for (int u = 0; u < kSelSeg; ++u)
      if (t0 + u < hi) {
        const uint32_t key = order_key(v[u]);
        gt += key > tau;
        eq += key == tau;
      }
  }
  int total;
  const int eq_before = block_exclusive_scan(eq, s_wave, total);
  const int take_eq = max(0, min(eq, need_eq - eq_before));
  int out = block_exclusive_scan(gt + take_eq, s_wave, total);
  int j = 0;  // image of the segment start
  if (lo < hi) {
    int a = 0, b = K - 1;
    while (a < b) {
      const int mid = (a + b + 1) >> 1;
      if (tbl.off[mid] <= lo) a = mid; else b = mid - 1;
    }
    j = a;
  }
  int eq_seen = 0;
  for (int t0 = lo; t0 < hi; t0 += kSelSeg) {
    float v[kSelSeg];
#pragma unroll
    for (int u = 0; u < kSelSeg; ++u) v[u] = t0 + u < hi ? p.shat[t0 + u] : 0.f;
#pragma unroll
    for (int u = 0; u < kSelSeg; ++u) {
      const int t = t0 + u;
      if (t >= hi) break;
      while (t >= tbl.off[j + 1]) ++j;
      const uint32_t key = order_key(v[u]);
      bool sel = key > tau;
      if (key == tau) {
        sel = eq_seen < take_eq;
        ++eq_seen;
      }
      if (p.mask_out) p.mask_out[t] = sel ? 1 : 0;
      if (sel && out < p.k) {
        p.idx_out[out] = t;
        p.pos_out[out] = tbl.pos[j] + (t - tbl.off[j]);
        ++out;
      }
    }
  }
}

// Steps 1-2 with the image table (s_off) in LDS: g_j into s_g (one wave per
// image, lane-strided partial sums, butterfly reduction: a fixed order), then
// g_bar and c_j = (1 - lambda) + lambda g_j / g_bar into s_c, exactly 1 where
// g_j = g_bar or g_bar = 0.  All 1024 threads take part; ends synchronised.
// PRE: `pre` holds the first 16 x 64 values of image `wave`, loaded by the
// caller at kernel start (the same values in the same order).
template <bool PRE>
__device__ __forceinline__ void image_coefficients(const SelectParams &p, int K, const int *s_off, float *s_g,
                                                   float *s_c, bool write_c, const float (&pre)[16]) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float n_layers = (float)p.n_layers;
  for (int j = wave; j < K; j += kWaves) {
    const int a = s_off[j], b = s_off[j + 1];
    float tot = 0.f;
    for (int t0 = a; t0 < b; t0 += 16 * 64) {  // 16 independent loads per round
      float v[16];
      const bool use_pre = PRE && j == wave && t0 == a;
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int t = t0 + 64 * u + lane;
        v[u] = use_pre ? pre[u] : (t < b ? p.a_acc[t] : 0.f);
      }
#pragma unroll
      for (int u = 0; u < 16; ++u) tot += v[u];
    }
    tot = wave_sum(tot);
    if (lane == 0) s_g[j] = tot / (n_layers * (float)(b - a));
  }
  __syncthreads();
  if (wave == 0) {
    float acc = 0.f;
    for (int j = lane; j < K; j += 64) acc += s_g[j];
    const float g_bar = wave_sum(acc) / (float)K;
    for (int j = lane; j < K; j += 64) {
      const float x = s_g[j] / g_bar;
      const float c = (g_bar == 0.f || x == 1.f) ? 1.f : (1.f - p.lambda) + p.lambda * x;
      s_c[j] = c;
      if (write_c && p.c_out) p.c_out[j] = c;
    }
  }
  __syncthreads();
}

// Register-resident variant for n_vis <= 1024 * PER: thread t owns visual
// tokens [t*PER, t*PER + PER), so scores are read once and the compaction is
// in index order without re-reading.  The radix select first fixes the bits
// every key shares (block AND/OR), then resolves the rest 11 bits per pass
// with one shared 2,048-bin LDS histogram: below the shared prefix the
// digits spread over the varying exponent and high mantissa bits, so LDS
// atomics rarely collide.
template <int PER>
__global__ __launch_bounds__(kSelThreads) void select_regs_kernel(SelectParams p, ImageTable tbl) {
  constexpr int kBits = 11, kBins = 1 << kBits;
  __shared__ float s_g[kMaxImages];
  __shared__ float s_c[kMaxImages];
  __shared__ int s_off[kMaxImages + 1];
  __shared__ int s_delta[kMaxImages];  // position - visual index, per image
  __shared__ int hist[kBins];
  __shared__ int s_wave[kWaves];
  __shared__ int s_wave2[kWaves];
  __shared__ int s_bin, s_above;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = tbl.n_vis, K = tbl.n_images;
  const float n_layers = (float)p.n_layers;
  const float inv_layers = 1.f / n_layers;

  // Image `wave`'s first attention values, in flight with the scores below.
  float pre[16];
  {
    const int a = wave < K ? tbl.off[wave] : 0, b = wave < K ? tbl.off[wave + 1] : 0;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int t = a + 64 * u + lane;
      pre[u] = t < b ? p.a_acc[t] : 0.f;
    }
  }
  // The radix histogram starts cleared; afterwards each pass clears the bins
  // it has read.
  for (int b = tid; b < kBins; b += kSelThreads) hist[b] = 0;

  // The image table moves to LDS (per-lane lookups would otherwise be
  // dependent loads from the kernel-argument segment).
  for (int j = tid; j <= K; j += kSelThreads) {
    s_off[j] = tbl.off[j];
    if (j < K) s_delta[j] = tbl.pos[j] - tbl.off[j];
  }
  // This thread's tokens [lo, lo + cnt): their scores load while the
  // per-image means are computed.
  const int lo = min(n, tid * PER), cnt = min(n, lo + PER) - lo;
  const bool whole = cnt == PER;
  float sv[PER];
  if (whole) {  // 16-byte loads, all in flight at once
#pragma unroll
    for (int e = 0; e < PER; e += 4) {
      const f32x4 v4 = *reinterpret_cast<const f32x4 *>(p.s_acc + lo + e);
      sv[e] = v4[0];
      sv[e + 1] = v4[1];
      sv[e + 2] = v4[2];
      sv[e + 3] = v4[3];
    }
  } else {
#pragma unroll
    for (int e = 0; e < PER; ++e) sv[e] = e < cnt ? p.s_acc[lo + e] : 0.f;
  }
  __syncthreads();

  // 1-2. per-image mean attention and coefficients
  image_coefficients<true>(p, K, s_off, s_g, s_c, true, pre);

  // 3. composite scores (s / |L|) * c_pi(t) of this thread's tokens
  int j0 = 0;  // image of the first token
  if (cnt > 0) {
    int a = 0, b = K - 1;
    while (a < b) {
      const int mid = (a + b + 1) >> 1;
      if (s_off[mid] <= lo) a = mid; else b = mid - 1;
    }
    j0 = a;
  }
  uint32_t key[PER];
  {
    int j = j0, next = s_off[j0 + 1];
    float c = s_c[j0];
    float sh[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      if (e < cnt) {
        while (lo + e >= next) {
          ++j;
          next = s_off[j + 1];
          c = s_c[j];
        }
      }
      sh[e] = (sv[e] * inv_layers) * c;
      key[e] = order_key(sh[e]);
    }
    if (p.shat) {
      if (whole) {
#pragma unroll
        for (int e = 0; e < PER; e += 4)
          *reinterpret_cast<f32x4 *>(p.shat + lo + e) = f32x4{sh[e], sh[e + 1], sh[e + 2], sh[e + 3]};
      } else {
#pragma unroll
        for (int e = 0; e < PER; ++e)
          if (e < cnt) p.shat[lo + e] = sh[e];
      }
    }
  }

  // 4. radix select of the k-th largest key
  uint32_t k_and = 0xffffffffu, k_or = 0;
#pragma unroll
  for (int e = 0; e < PER; ++e)
    if (e < cnt) {
      k_and &= key[e];
      k_or |= key[e];
    }
  block_and_or(k_and, k_or, s_wave, s_wave2);
  const uint32_t varying = k_and ^ k_or;  // bits that differ between keys
  uint32_t prefix = k_and, pmask = 0xffffffffu;
  int kk = p.k;
  if (varying) {
    const int top = 31 - __builtin_clz(varying);
    pmask = top == 31 ? 0u : ~((2u << top) - 1u);  // shared high bits
    prefix = k_and & pmask;
    for (int hi = top; hi >= 0; hi -= kBits) {  // digit = bits hi .. hi-10 (fewer at the end)
      const int sh = hi - (kBits - 1);
#pragma unroll
      for (int e = 0; e < PER; ++e)
        if (e < cnt && (key[e] & pmask) == prefix)
          atomicAdd(&hist[(sh >= 0 ? key[e] >> sh : key[e] << (-sh)) & (kBins - 1)], 1);
      __syncthreads();
      // thread tid owns bins kBins-1-2*tid, kBins-2-2*tid (descending)
      const int b0 = kBins - 1 - 2 * tid;
      const int h0 = hist[b0], h1 = hist[b0 - 1];
      hist[b0] = 0;  // cleared for the next pass (only this thread reads them)
      hist[b0 - 1] = 0;
      int total;
      const int run = block_exclusive_scan(h0 + h1, s_wave, total);
      if (run < kk && run + h0 >= kk) {
        s_bin = b0;
        s_above = run;
      } else if (run + h0 < kk && run + h0 + h1 >= kk) {
        s_bin = b0 - 1;
        s_above = run + h0;
      }
      __syncthreads();
      if (sh >= 0) {
        prefix |= (uint32_t)s_bin << sh;
        pmask |= (uint32_t)(kBins - 1) << sh;
      } else {  // last, partial digit
        prefix |= (uint32_t)s_bin >> (-sh);
        pmask |= (uint32_t)(kBins - 1) >> (-sh);
      }
      kk -= s_above;
    }
  }
  const uint32_t tau = prefix;
  const int need_eq = kk;  // entries equal to tau to take, lowest indices first

  // 5. ordered compaction
  int gt = 0, eq = 0;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    gt += (e < cnt) && key[e] > tau;
    eq += (e < cnt) && key[e] == tau;
  }
  // One scan of both counts (each < 2^16 for n_vis <= 32,768): the equal
  // entries taken before this thread are min(eq_before, need_eq).
  int total;
  const int packed = block_exclusive_scan((eq << 16) | gt, s_wave, total);
  const int eq_before = (int)((uint32_t)packed >> 16), gt_before = packed & 0xffff;
  const int take_eq = max(0, min(eq, need_eq - eq_before));
  int out = gt_before + min(eq_before, need_eq);
  int j = j0, next = cnt > 0 ? s_off[j0 + 1] : 0, delta = cnt > 0 ? s_delta[j0] : 0, eq_seen = 0;
  uint32_t mword[(PER + 3) / 4] = {};
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    if (e < cnt) {
      const int t = lo + e;
      while (t >= next) {
        ++j;
        next = s_off[j + 1];
        delta = s_delta[j];
      }
      bool sel = key[e] > tau;
      if (key[e] == tau) {
        sel = eq_seen < take_eq;
        ++eq_seen;
      }
      mword[e >> 2] |= (sel ? 1u : 0u) << (8 * (e & 3));
      if (sel && out < p.k) {
        p.idx_out[out] = t;
        p.pos_out[out] = t + delta;
        ++out;
      }
    }
  }
  if (p.mask_out) {
    if (whole && (reinterpret_cast<uintptr_t>(p.mask_out) & 15) == 0 && PER % 16 == 0) {
#pragma unroll
      for (int w = 0; w < PER / 4; w += 4)
        *reinterpret_cast<u32x4 *>(p.mask_out + lo + 4 * w) = u32x4{mword[w], mword[w + 1], mword[w + 2], mword[w + 3]};
    } else {
#pragma unroll
      for (int e = 0; e < PER; ++e)
        if (e < cnt) p.mask_out[lo + e] = (mword[e >> 2] >> (8 * (e & 3))) & 1u;
    }
  }
}

// Explicit per-image quotas: one workgroup per image.  Every workgroup
// derives the same c_j (steps 1-2) and the same quotas k_j ~ c_j n_j:
// largest remainder in float32, image order, shares capped at n_j with the
// surplus re-apportioned, all-zero weights falling back to n_j, remaining
// seats to the largest fractional parts (ties to the lower image).
// Workgroup j then keeps the k_j largest s_t of image j: the k_j-th largest
// key by bisection on the fp32 bit patterns (s >= 0), then everything above
// it plus the lowest-index entries equal to it, compacted in index order
// behind the quotas of the images before j.
__global__ __launch_bounds__(kSelThreads) void select_explicit_kernel(SelectParams p, ImageTable tbl) {
  __shared__ float s_g[kMaxImages];
  __shared__ float s_c[kMaxImages];
  __shared__ float s_share[kMaxImages];
  __shared__ float s_frac[kMaxImages];
  __shared__ int s_off[kMaxImages + 1];
  __shared__ int s_delta[kMaxImages];
  __shared__ int s_quota[kMaxImages];
  __shared__ int s_live[kMaxImages];
  __shared__ int s_wave[kWaves];
  __shared__ float s_total;
  __shared__ int s_left, s_capped, s_bysize, s_rest;

  const int tid = threadIdx.x;
  const int K = tbl.n_images, jimg = blockIdx.x;
  for (int j = tid; j <= K; j += kSelThreads) {
    s_off[j] = tbl.off[j];
    if (j < K) {
      s_delta[j] = tbl.pos[j] - tbl.off[j];
      s_quota[j] = 0;
      s_live[j] = 1;
    }
  }
  if (tid == 0) s_left = p.k;
  __syncthreads();
  const float no_pre[16] = {};
  image_coefficients<false>(p, K, s_off, s_g, s_c, jimg == 0, no_pre);

  // quotas
  for (;;) {
    if (tid == 0) {
      float total = 0.f;
      for (int j = 0; j < K; ++j)
        if (s_live[j]) total = __fadd_rn(total, __fmul_rn(s_c[j], (float)(s_off[j + 1] - s_off[j])));
      int by_size = total == 0.f;
      if (by_size) {
        total = 0.f;
        for (int j = 0; j < K; ++j)
          if (s_live[j]) total = __fadd_rn(total, (float)(s_off[j + 1] - s_off[j]));
      }
      s_total = total;
      s_bysize = by_size;
      s_capped = 0;
    }
    __syncthreads();
    const float total = s_total;
    const float left = (float)s_left;
    for (int j = tid; j < K; j += kSelThreads) {
      if (!s_live[j]) continue;
      const float nj = (float)(s_off[j + 1] - s_off[j]);
      const float w = s_bysize ? nj : __fmul_rn(s_c[j], nj);
      const float share = __fdiv_rn(__fmul_rn(left, w), total);
      s_share[j] = share;
      if (share >= nj) atomicAdd(&s_capped, 1);
    }
    __syncthreads();
    if (s_capped == 0) break;
    for (int j = tid; j < K; j += kSelThreads) {
      const int nj = s_off[j + 1] - s_off[j];
      if (s_live[j] && s_share[j] >= (float)nj) {
        s_quota[j] = nj;
        s_live[j] = 0;
        atomicSub(&s_left, nj);
      }
    }
    __syncthreads();
  }
  if (tid == 0) s_rest = s_left;
  __syncthreads();
  for (int j = tid; j < K; j += kSelThreads) {
    s_frac[j] = -1.f;
    if (!s_live[j]) continue;
    const int nj = s_off[j + 1] - s_off[j];
    const int base = min((int)floorf(s_share[j]), nj);
    s_quota[j] = base;
    s_frac[j] = __fsub_rn(s_share[j], (float)base);
    atomicSub(&s_rest, base);
  }
  __syncthreads();
  {
    int plus[(kMaxImages + kSelThreads - 1) / kSelThreads] = {};
    for (int j = tid, i = 0; j < K; j += kSelThreads, ++i) {
      const int nj = s_off[j + 1] - s_off[j];
      if (!s_live[j] || s_quota[j] >= nj) continue;
      int rank = 0;  // candidates ahead of j: larger fraction, or equal and lower index
      for (int u = 0; u < K; ++u) {
        const int nu = s_off[u + 1] - s_off[u];
        if (!s_live[u] || s_quota[u] >= nu) continue;
        rank += s_frac[u] > s_frac[j] || (s_frac[u] == s_frac[j] && u < j);
      }
      plus[i] = rank < s_rest;
    }
    __syncthreads();
    for (int j = tid, i = 0; j < K; j += kSelThreads, ++i) s_quota[j] += plus[i];
  }
  __syncthreads();
  if (jimg == 0 && p.quota_out)
    for (int j = tid; j < K; j += kSelThreads) p.quota_out[j] = s_quota[j];

  // selection inside image jimg
  const int a = s_off[jimg], b = s_off[jimg + 1];
  const int kq = s_quota[jimg];
  int out0 = 0;
  for (int j = 0; j < jimg; ++j) out0 += s_quota[j];
  const float inv_layers = 1.f / (float)p.n_layers;
  const float cj = s_c[jimg];
  auto block_count = [&](uint32_t thr, bool strict) {
    int c = 0;
    for (int t = a + tid; t < b; t += kSelThreads) {
      const uint32_t key = order_key(p.s_acc[t]);
      c += strict ? key > thr : key >= thr;
    }
    int total;
    (void)block_exclusive_scan(c, s_wave, total);
    return total;
  };
  uint32_t thr = 0;
  if (kq > 0) {
    for (int bit = 31; bit >= 0; --bit) {
      const uint32_t cand = thr | (1u << bit);
      if (block_count(cand, false) >= kq) thr = cand;
    }
  }
  const int need_eq = kq > 0 ? kq - block_count(thr, true) : 0;
  int eq_base = 0, sel_base = 0;
  for (int t0 = a; t0 < b; t0 += kSelThreads) {
    const int t = t0 + tid;
    const bool live = t < b;
    const float sv = live ? p.s_acc[t] : 0.f;
    const uint32_t key = order_key(sv);
    const bool gt = live && kq > 0 && key > thr;
    const bool eq = live && kq > 0 && key == thr;
    int n_eq, n_sel;
    const int eq_before = eq_base + block_exclusive_scan(eq ? 1 : 0, s_wave, n_eq);
    const bool sel = gt || (eq && eq_before < need_eq);
    const int rank = sel_base + block_exclusive_scan(sel ? 1 : 0, s_wave, n_sel);
    if (live) {
      if (sel && rank < kq && out0 + rank < p.k) {
        p.idx_out[out0 + rank] = t;
        p.pos_out[out0 + rank] = t + s_delta[jimg];
      }
      if (p.mask_out) p.mask_out[t] = sel ? 1 : 0;
      if (p.shat) p.shat[t] = (sv * inv_layers) * cj;
    }
    eq_base += n_eq;
    sel_base += n_sel;
  }
}

__global__ void clear_u8_kernel(uint8_t *p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

}  // namespace

hipError_t launch_select(const SelectParams &p, const ImageTable &tbl, hipStream_t s) {
  ProfScope ps("select", s);
  if (tbl.n_vis <= kSelThreads * 16) select_regs_kernel<16><<<1, kSelThreads, 0, s>>>(p, tbl);
  else if (tbl.n_vis <= kSelThreads * 32) select_regs_kernel<32><<<1, kSelThreads, 0, s>>>(p, tbl);
  else select_kernel<<<1, kSelThreads, 0, s>>>(p, tbl);
  return hipGetLastError();
}

hipError_t launch_select_explicit(const SelectParams &p, const ImageTable &tbl, hipStream_t s) {
  ProfScope ps("select_explicit", s);
  select_explicit_kernel<<<tbl.n_images, kSelThreads, 0, s>>>(p, tbl);
  return hipGetLastError();
}

hipError_t launch_clear_u8(uint8_t *p, int64_t n, hipStream_t s) {
  ProfScope ps("clear_mask", s);
  clear_u8_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(p, n);
  return hipGetLastError();
}

}  // namespace conduit
