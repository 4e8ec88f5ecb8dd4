// Cache merge for the selective recompute, gfx950: the selected rows take
// their recomputed K/V, every other row is reused in place (Sec. 3).  One
// wave per selected row moves 16-byte chunks of K and V; when asked, the
// stale rows are copied out first so the merge can be undone.  The layers of
// one request can go in one launch (one grid row per layer).
#include "common.h"

namespace conduit {
namespace {

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
