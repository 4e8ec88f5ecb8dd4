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

// image of visual token t (s_off in LDS, K images)
__device__ __forceinline__ int image_of(const int *s_off, int K, int t) {
  int a = 0, b = K - 1;
  while (a < b) {
    const int mid = (a + b + 1) >> 1;
    if (s_off[mid] <= t) a = mid; else b = mid - 1;
  }
  return a;
}

// Block-wide scans exchange one value per wave through LDS behind a single
// barrier.  Each call site has its own LDS slots (or alternates between two),
// so no trailing barrier is needed before reuse.
// Exclusive prefix sum over the block in thread order (modulo 2^32: exact
// whenever the true prefix fits); `total` gets the block sum.  `slot`:
// kWaves LDS words for this call.
__device__ __forceinline__ uint32_t block_exclusive_sum(uint32_t x, uint32_t *slot, uint32_t &total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const uint32_t inc = wave_inclusive_sum(x);
  if (lane == 63) slot[w] = inc;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int i = 0; i < kWaves; ++i) {
    const uint32_t v = slot[i];
    before += i < w ? v : 0u;
    all += v;
  }
  total = all;
  return before + inc - x;
}
__device__ __forceinline__ uint32_t block_exclusive_sum(uint32_t x, uint32_t *slot) {
  uint32_t total;
  return block_exclusive_sum(x, slot, total);
}

// Register-resident top-k for n_vis <= 1024 * PER: thread t owns visual
// tokens [t*PER, t*PER + PER), so every score is read once and the
// compaction is in index order without re-reading.  All reductions and scans
// are DPP-based; the steps are
//  1. g_j: each thread sums its A values image by image (token order) into
//     LDS slot (thread + image) - unique, because a thread's images never
//     precede its predecessor's - then one wave per image adds the slots of
//     the threads that overlap it, in thread order;
//  2. g_bar over the images (every wave, the same order, so the same bits)
//     and c_j into LDS;
//  3. s_hat and its order keys;
//  4. radix select: the bits every key shares (block AND/OR), then 11-bit
//     digits over the rest with one LDS histogram, stopping as soon as the
//     chosen bin holds exactly the entries still needed;
//  5. ordered compaction of everything above the prefix found plus the
//     first `need` entries equal to it (ties to the lower index): the
//     selected indices go to LDS at their output rank, then out to idx/pos
//     in coalesced stores.
template <int PER>
__global__ __launch_bounds__(kSelThreads) void select_regs_kernel(SelectParams p, ImageTable tbl) {
  constexpr int kBits = 11, kBins = 1 << kBits;
  static_assert(PER % 4 == 0 && PER * kSelThreads <= 65536, "counts are packed in 16 bits");
  __shared__ int s_idx[PER * kSelThreads];
  __shared__ float s_g[kMaxImages];
  __shared__ float s_c[kMaxImages];
  __shared__ int s_off[kMaxImages + 1];
  __shared__ int s_delta[kMaxImages];  // position - visual index, per image
  __shared__ float s_part[kSelThreads + kMaxImages];
  __shared__ int hist[kBins];
  __shared__ uint32_t s_andor[2][kWaves];
  __shared__ uint32_t s_scan[3][kWaves];
  __shared__ int s_pick[2][3];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = tbl.n_vis, K = tbl.n_images;
  const float n_layers = (float)p.n_layers;
  const float inv_layers = 1.f / n_layers;
  const int lo = min(n, tid * PER), cnt = min(n, lo + PER) - lo;
  const bool vec = cnt == PER && ((reinterpret_cast<uintptr_t>(p.s_acc) | reinterpret_cast<uintptr_t>(p.a_acc) |
                                   reinterpret_cast<uintptr_t>(p.shat)) & 15) == 0;
  auto load = [&](const float *src, float (&v)[PER]) __attribute__((always_inline)) {
    if (vec) {
#pragma unroll
      for (int e = 0; e < PER; e += 4) {
        const f32x4 x = *reinterpret_cast<const f32x4 *>(src + lo + e);
        v[e] = x[0];
        v[e + 1] = x[1];
        v[e + 2] = x[2];
        v[e + 3] = x[3];
      }
    } else {
#pragma unroll
      for (int e = 0; e < PER; ++e) v[e] = e < cnt ? src[lo + e] : 0.f;
    }
  };
  float sv[PER];
  {
    float av[PER];
    load(p.a_acc, av);
    load(p.s_acc, sv);
    for (int j = tid; j <= K; j += kSelThreads) {
      s_off[j] = tbl.off[j];
      if (j < K) s_delta[j] = tbl.pos[j] - tbl.off[j];
    }
    for (int b = tid; b < kBins; b += kSelThreads) hist[b] = 0;
    __syncthreads();
    // 1. this thread's A, summed per image in token order
    if (cnt > 0) {
      int a = 0, b = K - 1;  // image of the first token
      while (a < b) {
        const int mid = (a + b + 1) >> 1;
        if (s_off[mid] <= lo) a = mid; else b = mid - 1;
      }
      int j = a, next = s_off[a + 1];
      float acc = 0.f;
      if (next >= lo + cnt) {  // one image
#pragma unroll
        for (int e = 0; e < PER; ++e) acc += e < cnt ? av[e] : 0.f;
      } else {
#pragma unroll
        for (int e = 0; e < PER; ++e) {
          if (e < cnt) {
            if (lo + e >= next) {  // images are non-empty: the next token starts image j + 1
              s_part[tid + j] = acc;
              acc = 0.f;
              ++j;
              next = s_off[j + 1];
            }
            acc += av[e];
          }
        }
      }
      s_part[tid + j] = acc;
    }
  }
  __syncthreads();
  for (int j = wave; j < K; j += kWaves) {
    const int a = s_off[j], b = s_off[j + 1];
    float acc = 0.f;
    for (int t = a / PER + lane; t <= (b - 1) / PER; t += 64) acc += s_part[t + j];
    acc = wave_fsum(acc);
    if (lane == 0) s_g[j] = acc / (n_layers * (float)(b - a));
  }
  __syncthreads();
  // 2. g_bar and the coefficients
  float gacc = 0.f;
  for (int j = lane; j < K; j += 64) gacc += s_g[j];
  const float g_bar = wave_fsum(gacc) / (float)K;
  for (int j = tid; j < K; j += kSelThreads) {
    // (1 - lambda) + lambda * x adds two non-negative terms, so it keeps full
    // relative precision even for c << 1; x == 1 (one image, or an image at
    // the mean) gives exactly 1.
    const float x = s_g[j] / g_bar;
    const float c = (g_bar == 0.f || x == 1.f) ? 1.f : (1.f - p.lambda) + p.lambda * x;
    s_c[j] = c;
    if (p.c_out) p.c_out[j] = c;
  }
  __syncthreads();

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
  uint32_t key[PER];  // takes the place of sv: each score is stored, then only its key is kept
  {
    int j = j0, next = s_off[j0 + 1];
    float c = s_c[j0];
    const bool one_image = next >= lo + cnt;
#pragma unroll
    for (int e = 0; e < PER; e += 4) {
      f32x4 sh;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (!one_image && e + u < cnt && lo + e + u >= next) {
          ++j;
          next = s_off[j + 1];
          c = s_c[j];
        }
        sh[u] = (sv[e + u] * inv_layers) * c;
        key[e + u] = order_key(sh[u]);
      }
      if (p.shat) {
        if (vec) {
          *reinterpret_cast<f32x4 *>(p.shat + lo + e) = sh;
        } else {
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (e + u < cnt) p.shat[lo + e + u] = sh[u];
        }
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
  k_and = wave_reduce(k_and, 0xffffffffu, [](uint32_t a, uint32_t b) { return a & b; });
  k_or = wave_reduce(k_or, 0u, [](uint32_t a, uint32_t b) { return a | b; });
  if (lane == 0) {
    s_andor[0][wave] = k_and;
    s_andor[1][wave] = k_or;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kWaves; ++i) {
    k_and &= s_andor[0][i];
    k_or |= s_andor[1][i];
  }
  const uint32_t varying = k_and ^ k_or;  // bits that differ between keys
  uint32_t prefix = k_and, pmask = 0xffffffffu;
  int kk = p.k;
  if (varying) {
    const int top = 31 - __builtin_clz(varying);
    pmask = top == 31 ? 0u : ~((2u << top) - 1u);  // shared high bits
    prefix = k_and & pmask;
    for (int hi = top, pass = 0; hi >= 0; hi -= kBits, ++pass) {  // digit = bits hi .. hi-10 (fewer at the end)
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
      const int run = (int)block_exclusive_sum((uint32_t)(h0 + h1), s_scan[pass & 1]);
      int *pick = s_pick[pass & 1];
      if (run < kk && run + h0 >= kk) {
        pick[0] = b0;
        pick[1] = run;
        pick[2] = run + h0 == kk;  // the bin is exactly what is still needed
      } else if (run + h0 < kk && run + h0 + h1 >= kk) {
        pick[0] = b0 - 1;
        pick[1] = run + h0;
        pick[2] = run + h0 + h1 == kk;
      }
      __syncthreads();
      const uint32_t bin = (uint32_t)pick[0];
      if (sh >= 0) {
        prefix |= bin << sh;
        pmask |= (uint32_t)(kBins - 1) << sh;
      } else {  // last, partial digit
        prefix |= bin >> (-sh);
        pmask |= (uint32_t)(kBins - 1) >> (-sh);
      }
      kk -= pick[1];
      if (pick[2]) break;
    }
  }
  // The selection: keys whose masked bits exceed the prefix, then the first
  // `need_eq` (in index order) whose masked bits equal it.  After the last
  // digit the mask is complete and the prefix is the k-th largest key.
  const int need_eq = kk;

  // 5. ordered compaction
  int gt = 0, eq = 0;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const uint32_t m = key[e] & pmask;
    gt += (e < cnt) && m > prefix;
    eq += (e < cnt) && m == prefix;
  }
  // One scan of both counts (each prefix < 2^16 for n_vis <= 65,536): the
  // equal entries taken before this thread are min(eq_before, need_eq).
  const uint32_t packed = block_exclusive_sum(((uint32_t)eq << 16) | (uint32_t)gt, s_scan[2]);
  const int eq_before = (int)(packed >> 16), gt_before = (int)(packed & 0xffffu);
  const int take_eq = max(0, min(eq, need_eq - eq_before));
  int out = gt_before + min(eq_before, need_eq);
  int eq_seen = 0;
  uint32_t mword[4] = {};
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    bool sel = false;
    if (e < cnt) {
      const uint32_t m = key[e] & pmask;
      sel = m > prefix;
      if (m == prefix) {
        sel = eq_seen < take_eq;
        ++eq_seen;
      }
      if (sel && out < p.k) s_idx[out++] = lo + e;
    }
    mword[(e >> 2) & 3] |= (sel ? 1u : 0u) << (8 * (e & 3));
    if (p.mask_out && (e & 15) == 15) {  // 16 mask bytes per store
      const int base = e - 15;
      if (vec && (reinterpret_cast<uintptr_t>(p.mask_out) & 15) == 0) {
        *reinterpret_cast<u32x4 *>(p.mask_out + lo + base) = u32x4{mword[0], mword[1], mword[2], mword[3]};
      } else {
        for (int u = 0; u < 16; ++u)
          if (base + u < cnt) p.mask_out[lo + base + u] = (mword[u >> 2] >> (8 * (u & 3))) & 1u;
      }
      mword[0] = mword[1] = mword[2] = mword[3] = 0u;
    }
  }
  if constexpr (PER % 16 != 0) {
    if (p.mask_out)
      for (int u = 0; u < PER % 16; ++u)
        if (PER - PER % 16 + u < cnt)
          p.mask_out[lo + PER - PER % 16 + u] = (mword[u >> 2] >> (8 * (u & 3))) & 1u;
  }
  __syncthreads();
  for (int i = tid; i < p.k; i += kSelThreads) {
    const int t = s_idx[i];
    p.idx_out[i] = t;
    p.pos_out[i] = t + s_delta[image_of(s_off, K, t)];
  }
}

// ---------------------------------------------------------------------------
// Multi-workgroup top-k for kSelMultiKeys < n_vis <= kSelMultiMaxWg *
// kSelMultiKeys: workgroup b owns visual tokens [4096 b, 4096 b + 4096), four
// consecutive ones per thread (16-byte loads), so the per-token work and the
// scattered output stores spread over G = ceil(n_vis / 4096) CUs.
//  select_partials_kernel: each workgroup sums its A values per image in
//    token order (threads, then the threads of each image in order) into
//    slot (b + image) of the exchange area - unique, as for threads - and
//    clears the barrier flags of the next kernel.
//  select_multi_kernel: every workgroup adds the partials of each image in
//    workgroup order (so all derive the same g_j, g_bar and c_j bits), forms
//    its keys and writes s_hat, then the radix select runs on fixed digits
//    (bits 31-21, 20-10, 9-0 of the key): per pass each workgroup publishes
//    its local histogram, passes a grid barrier and adds all G histograms in
//    workgroup order, so every workgroup picks the same bin; the passes stop
//    once the bin holds exactly what is still needed.  The published
//    histograms also give each workgroup the number of selected entries of
//    the workgroups before it, so it writes its outputs in index order with
//    no further exchange.
// A grid barrier is a flag per workgroup in device memory (set after a
// device-scope release, polled with device-scope loads and an acquire): all
// G <= 32 workgroups are resident at once on a 256-CU device.  The wait is
// bounded (about a second); a workgroup that gives up goes on, so the kernel
// always ends, and its outputs are then not meaningful.
// ---------------------------------------------------------------------------
constexpr int kSelMultiPer = kSelMultiKeys / kSelThreads;
constexpr uint32_t kSelSpinLimit = 1u << 20;

__device__ __forceinline__ void grid_arrive_wait(uint32_t *flags, int G) {
  __syncthreads();  // every wave's stores of this phase are done
  if (threadIdx.x == 0) {
    __threadfence();  // release them at device scope
    __hip_atomic_store(flags + blockIdx.x, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    if (lane < G) {
      uint32_t spins = 0;
      while (__hip_atomic_load(flags + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u) {
        if (++spins > kSelSpinLimit) break;
        __builtin_amdgcn_s_sleep(2);
      }
    }
    __threadfence();  // acquire the other workgroups' stores
  }
  __syncthreads();
}

__global__ __launch_bounds__(kSelThreads) void select_partials_kernel(SelectParams p, ImageTable tbl) {
  constexpr int PER = kSelMultiPer;
  __shared__ int s_off[kMaxImages + 1];
  __shared__ float s_part[kSelThreads + kMaxImages];
  const SelectMultiLayout L = select_multi_layout();
  char *ws = static_cast<char *>(p.multi);
  float *gpart = reinterpret_cast<float *>(ws + L.gpart);
  uint32_t *flags = reinterpret_cast<uint32_t *>(ws + L.flags);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, b = blockIdx.x;
  const int n = tbl.n_vis, K = tbl.n_images;
  const int base = b * kSelMultiKeys, end = min(n, base + kSelMultiKeys);
  const int lo = min(end, base + tid * PER), cnt = min(end, lo + PER) - lo;
  float av[PER];
  if (cnt == PER && (reinterpret_cast<uintptr_t>(p.a_acc) & 15) == 0) {
    const f32x4 x = *reinterpret_cast<const f32x4 *>(p.a_acc + lo);
#pragma unroll
    for (int e = 0; e < PER; ++e) av[e] = x[e];
  } else {
#pragma unroll
    for (int e = 0; e < PER; ++e) av[e] = e < cnt ? p.a_acc[lo + e] : 0.f;
  }
  for (int j = tid; j <= K; j += kSelThreads) s_off[j] = tbl.off[j];
  if (b == 0)
    for (int i = tid; i < kSelMultiBarriers * kSelMultiMaxWg; i += kSelThreads) flags[i] = 0u;
  __syncthreads();
  if (cnt > 0) {
    int j = image_of(s_off, K, lo), next = s_off[j + 1];
    float acc = 0.f;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      if (e < cnt) {
        if (lo + e >= next) {  // images are non-empty: the next token starts image j + 1
          s_part[tid + j] = acc;
          acc = 0.f;
          ++j;
          next = s_off[j + 1];
        }
        acc += av[e];
      }
    }
    s_part[tid + j] = acc;
  }
  __syncthreads();
  // this workgroup's partial of every image it overlaps, threads in order
  const int j_first = image_of(s_off, K, base), j_last = image_of(s_off, K, end - 1);
  for (int j = j_first + wave; j <= j_last; j += kWaves) {
    const int t0 = (max(s_off[j], base) - base) / PER, t1 = (min(s_off[j + 1], end) - 1 - base) / PER;
    float acc = 0.f;
    for (int t = t0 + lane; t <= t1; t += 64) acc += s_part[t + j];
    acc = wave_fsum(acc);
    if (lane == 0) gpart[b + j] = acc;
  }
}

// GMAX >= gridDim.x bounds the unrolled histogram merge.
template <int GMAX>
__global__ __launch_bounds__(kSelThreads) void select_multi_kernel(SelectParams p, ImageTable tbl) {
  constexpr int PER = kSelMultiPer;
  __shared__ float s_g[kMaxImages];
  __shared__ float s_c[kMaxImages];
  __shared__ int s_off[kMaxImages + 1];
  __shared__ int s_delta[kMaxImages];
  __shared__ float s_gpart[kSelMultiMaxWg + kMaxImages];
  __shared__ int hist[kSelDigitBins];
  __shared__ uint32_t s_scan[4][kWaves];
  __shared__ int s_pick[2][4];
  const SelectMultiLayout L = select_multi_layout();
  char *ws = static_cast<char *>(p.multi);
  const float *gpart = reinterpret_cast<const float *>(ws + L.gpart);
  int *ghist = reinterpret_cast<int *>(ws + L.ghist);
  uint32_t *flags = reinterpret_cast<uint32_t *>(ws + L.flags);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, b = blockIdx.x, G = gridDim.x;
  const int n = tbl.n_vis, K = tbl.n_images;
  const float n_layers = (float)p.n_layers;
  const float inv_layers = 1.f / n_layers;
  const int base = b * kSelMultiKeys, end = min(n, base + kSelMultiKeys);
  const int lo = min(end, base + tid * PER), cnt = min(end, lo + PER) - lo;
  const bool vec = cnt == PER && ((reinterpret_cast<uintptr_t>(p.s_acc) | reinterpret_cast<uintptr_t>(p.shat)) & 15) == 0;
  float sv[PER];
  if (vec) {
    const f32x4 x = *reinterpret_cast<const f32x4 *>(p.s_acc + lo);
#pragma unroll
    for (int e = 0; e < PER; ++e) sv[e] = x[e];
  } else {
#pragma unroll
    for (int e = 0; e < PER; ++e) sv[e] = e < cnt ? p.s_acc[lo + e] : 0.f;
  }
  for (int j = tid; j <= K; j += kSelThreads) {
    s_off[j] = tbl.off[j];
    if (j < K) s_delta[j] = tbl.pos[j] - tbl.off[j];
  }
  for (int i = tid; i < kSelDigitBins; i += kSelThreads) hist[i] = 0;
  // the partials (slots never written are never read)
  if (tid < G + K) s_gpart[tid] = gpart[tid];
  __syncthreads();
  // 1. g_j: the workgroup partials of image j, in workgroup order
  for (int j = wave; j < K; j += kWaves) {
    const int a = s_off[j], e = s_off[j + 1];
    float acc = 0.f;
    for (int w = a / kSelMultiKeys + lane; w <= (e - 1) / kSelMultiKeys; w += 64) acc += s_gpart[w + j];
    acc = wave_fsum(acc);
    if (lane == 0) s_g[j] = acc / (n_layers * (float)(e - a));
  }
  __syncthreads();
  // 2. g_bar (every wave, same order) and c_j
  float gacc = 0.f;
  for (int j = lane; j < K; j += 64) gacc += s_g[j];
  const float g_bar = wave_fsum(gacc) / (float)K;
  for (int j = tid; j < K; j += kSelThreads) {
    const float x = s_g[j] / g_bar;
    const float c = (g_bar == 0.f || x == 1.f) ? 1.f : (1.f - p.lambda) + p.lambda * x;
    s_c[j] = c;
    if (b == 0 && p.c_out) p.c_out[j] = c;
  }
  __syncthreads();
  // 3. keys of this thread's tokens
  const int j0 = cnt > 0 ? image_of(s_off, K, lo) : 0;
  uint32_t key[PER];
  {
    int j = j0, next = s_off[j0 + 1];
    float c = s_c[j0];
    f32x4 sh;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      if (e < cnt && lo + e >= next) {
        ++j;
        next = s_off[j + 1];
        c = s_c[j];
      }
      sh[e] = (sv[e] * inv_layers) * c;
      key[e] = order_key(sh[e]);
    }
    if (p.shat) {
      if (vec) {
        *reinterpret_cast<f32x4 *>(p.shat + lo) = sh;
      } else {
#pragma unroll
        for (int e = 0; e < PER; ++e)
          if (e < cnt) p.shat[lo + e] = sh[e];
      }
    }
  }
  // 4. radix select on fixed digits.  The histograms also give the
  // compaction's offsets: the entries of workgroups before this one above
  // the final threshold are, summed over the passes, those of their
  // published bins above each pass's pick (gt_prior, one share per thread),
  // and those equal to it are their count in the last pick.
  uint32_t prefix = 0, pmask = 0;
  int kk = p.k, gt_prior = 0, eq_prior = 0;
  for (int pass = 0; pass < 3; ++pass) {
    const int sh = pass == 0 ? 21 : pass == 1 ? 10 : 0;
    const uint32_t dmask = pass == 2 ? 0x3ffu : 0x7ffu;
#pragma unroll
    for (int e = 0; e < PER; ++e)
      if (e < cnt && (key[e] & pmask) == prefix) atomicAdd(&hist[(key[e] >> sh) & dmask], 1);
    __syncthreads();
    // thread tid owns bins 2047-2*tid, 2046-2*tid (descending)
    const int b0 = kSelDigitBins - 1 - 2 * tid;
    int *mine = ghist + ((size_t)pass * kSelMultiMaxWg + b) * kSelDigitBins;
    *reinterpret_cast<int2 *>(mine + b0 - 1) = int2{hist[b0 - 1], hist[b0]};
    hist[b0] = 0;
    hist[b0 - 1] = 0;
    grid_arrive_wait(flags + pass * kSelMultiMaxWg, G);
    int2 v[GMAX];  // all loads in flight together
#pragma unroll
    for (int w = 0; w < GMAX; ++w)
      if (w < G) v[w] = *reinterpret_cast<const int2 *>(ghist + ((size_t)pass * kSelMultiMaxWg + w) * kSelDigitBins + b0 - 1);
    int h0 = 0, h1 = 0, q0 = 0, q1 = 0;  // all workgroups / those before this one
#pragma unroll
    for (int w = 0; w < GMAX; ++w)  // workgroup order
      if (w < G) {
        h0 += v[w].y;
        h1 += v[w].x;
        if (w < b) {
          q0 += v[w].y;
          q1 += v[w].x;
        }
      }
    const int run = (int)block_exclusive_sum((uint32_t)(h0 + h1), s_scan[pass & 1]);
    int *pick = s_pick[pass & 1];
    if (run < kk && run + h0 >= kk) {
      pick[0] = b0;
      pick[1] = run;
      pick[2] = run + h0 == kk;
      pick[3] = q0;
    } else if (run + h0 < kk && run + h0 + h1 >= kk) {
      pick[0] = b0 - 1;
      pick[1] = run + h0;
      pick[2] = run + h0 + h1 == kk;
      pick[3] = q1;
    }
    __syncthreads();
    const int bin = pick[0];
    gt_prior += (b0 > bin ? q0 : 0) + (b0 - 1 > bin ? q1 : 0);
    eq_prior = pick[3];
    prefix |= (uint32_t)bin << sh;
    pmask |= dmask << sh;
    kk -= pick[1];
    if (pick[2]) break;
  }
  const int need_eq = kk;

  // 5. ordered compaction: counts in the workgroup, then across workgroups
  int gt = 0, eq = 0;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const uint32_t m = key[e] & pmask;
    gt += (e < cnt) && m > prefix;
    eq += (e < cnt) && m == prefix;
  }
  // one block exclusive scan of the packed counts (< 2^16 entries per
  // workgroup) and of the prior workgroups' share, whose block total is
  // their count above the threshold
  const uint32_t packed = block_exclusive_sum(((uint32_t)eq << 16) | (uint32_t)gt, s_scan[2]);
  uint32_t gt_wg;
  (void)block_exclusive_sum((uint32_t)gt_prior, s_scan[3], gt_wg);
  const int eq_before = eq_prior + (int)(packed >> 16), gt_before = (int)gt_wg + (int)(packed & 0xffffu);
  const int take_eq = max(0, min(eq, need_eq - eq_before));
  int out = gt_before + min(eq_before, need_eq);
  int j = j0, next = cnt > 0 ? s_off[j0 + 1] : 0, delta = cnt > 0 ? s_delta[j0] : 0, eq_seen = 0;
  uint32_t mword = 0;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    if (e < cnt) {
      const int t = lo + e;
      if (t >= next) {
        ++j;
        next = s_off[j + 1];
        delta = s_delta[j];
      }
      const uint32_t m = key[e] & pmask;
      bool sel = m > prefix;
      if (m == prefix) {
        sel = eq_seen < take_eq;
        ++eq_seen;
      }
      mword |= (sel ? 1u : 0u) << (8 * e);
      if (sel && out < p.k) {
        p.idx_out[out] = t;
        p.pos_out[out] = t + delta;
        ++out;
      }
    }
  }
  if (p.mask_out) {
    if (cnt == PER && (reinterpret_cast<uintptr_t>(p.mask_out) & 3) == 0) {
      *reinterpret_cast<uint32_t *>(p.mask_out + lo) = mword;
    } else {
      for (int e = 0; e < cnt; ++e) p.mask_out[lo + e] = (mword >> (8 * e)) & 1u;
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
  const int n = tbl.n_vis;
  if (n <= kSelThreads * 4) {
    select_regs_kernel<4><<<1, kSelThreads, 0, s>>>(p, tbl);
  } else if (n <= kSelThreads * 16) {  // faster in one workgroup up to here
    select_regs_kernel<16><<<1, kSelThreads, 0, s>>>(p, tbl);
  } else if (select_uses_multi(n)) {
    if (!p.multi) return hipErrorInvalidValue;
    const int G = (n + kSelMultiKeys - 1) / kSelMultiKeys;
    select_partials_kernel<<<G, kSelThreads, 0, s>>>(p, tbl);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (G <= 4) select_multi_kernel<4><<<G, kSelThreads, 0, s>>>(p, tbl);
    else if (G <= 8) select_multi_kernel<8><<<G, kSelThreads, 0, s>>>(p, tbl);
    else if (G <= 16) select_multi_kernel<16><<<G, kSelThreads, 0, s>>>(p, tbl);
    else select_multi_kernel<32><<<G, kSelThreads, 0, s>>>(p, tbl);
  } else {
    select_kernel<<<1, kSelThreads, 0, s>>>(p, tbl);
  }
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
