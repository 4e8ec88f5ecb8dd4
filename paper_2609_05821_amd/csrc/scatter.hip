// Cache merge for the selective recompute, gfx950: the selected rows take
// their recomputed K/V, every other row is reused in place (Sec. 3).  One
// wave per selected row moves 16-byte chunks of K and V; when asked, the
// stale rows are copied out first so the merge can be undone.  The layers of
// one request can go in one launch (one grid row per layer).
#include "common.h"

namespace conduit {
namespace {

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

__global__ __launch_bounds__(256) void scatter_kernel(ScatterParams p) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row < p.n_rows) scatter_row(p, row, threadIdx.x & 63);
}

// Several layers of one request, layer blockIdx.y (same rows and shapes).
__global__ __launch_bounds__(256) void scatter_layers_kernel(ScatterParams p, ScatterLayers sl) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= p.n_rows) return;
  const int l = blockIdx.y;
  p.k = sl.k[l];
  p.v = sl.v[l];
  p.k_new = sl.k_new[l];
  p.v_new = sl.v_new[l];
  scatter_row(p, row, threadIdx.x & 63);
}

}  // namespace

hipError_t launch_scatter(const ScatterParams &p, hipStream_t s) {
  ProfScope ps("scatter", s);
  scatter_kernel<<<(p.n_rows + 3) / 4, 256, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_scatter_layers(const ScatterParams &p, const ScatterLayers &sl, hipStream_t s) {
  ProfScope ps("scatter", s);
  scatter_layers_kernel<<<dim3((p.n_rows + 3) / 4, sl.n), 256, 0, s>>>(p, sl);
  return hipGetLastError();
}

}  // namespace conduit
