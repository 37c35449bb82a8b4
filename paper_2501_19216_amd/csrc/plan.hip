// Device-side plan of the factorised forward (Thm. 3.3 with local origins):
// everything the layer needs besides the aggregation and the recouple is
// derived on the GPU, so the forward never waits for the device.
//
//   bounding box -> tile grid (one thread) -> tile of every atom ->
//   receiver order (graph, then Morton index of 4 A cells) ->
//   solid harmonics of every edge's sender about the receiver's tile centre
//   (fp64, rounded to fp32) and of every receiver (fp64).
//
// The CSR is read with clamped indices everywhere (row bounds to [0, E],
// senders to [0, n)), so a malformed graph gives wrong numbers, never an
// access outside the caller's buffers; e2f_validate_graph checks a graph.
#include <hip/hip_runtime.h>
#include <hipcub/hipcub.hpp>

#include <climits>

#include "e2f_launch.h"

namespace e2f {
namespace {

__device__ __forceinline__ int64_t clamp_edge(int64_t e, int64_t lo, int64_t hi) {
  return e < lo ? lo : (e > hi ? hi : e);
}

__device__ __forceinline__ int clamp_node(int j, int n) { return (unsigned)j < (unsigned)n ? j : 0; }

// Row bounds of receiver i, clamped so that 0 <= e0 <= e1 <= E.
__device__ __forceinline__ void row_bounds(const int64_t* __restrict__ row_ptr, int i, int64_t E, int64_t& e0,
                                           int64_t& e1) {
  e0 = clamp_edge(row_ptr[i], 0, E);
  e1 = clamp_edge(row_ptr[i + 1], e0, E);
}

// Centre of tile cell `cell` of the grid, in Angstrom (the grid's integer
// arithmetic on the 2^-16 A lattice, then one exact division).
__device__ __forceinline__ void tile_centre(const TileGridDev& g, int cell, double& ox, double& oy, double& oz) {
  const int cx = cell % g.dim[0], cy = (cell / g.dim[0]) % g.dim[1], cz = cell / (g.dim[0] * g.dim[1]);
  const int c[3] = {cx, cy, cz};
  double o[3];
#pragma unroll
  for (int k = 0; k < 3; ++k)
    o[k] = (double)(g.lo[k] + ((2 * (int64_t)c[k] + 1) * g.span[k]) / (2 * (int64_t)g.dim[k])) / kGrid;
  ox = o[0], oy = o[1], oz = o[2];
}

// All (L+1)^2 real solid harmonics of (x, y, z) from their monomial tables,
// each handed to sink(k, value).  Every lane walks the same table entries,
// so the loads are uniform.
template <int L, typename Sink>
__device__ __forceinline__ void sh_all(const DevTables& t, double x, double y, double z, Sink sink) {
  constexpr int NK = (L + 1) * (L + 1);
  for (int k = 0; k < NK; ++k) {
    double acc = 0.0;
    for (int e = t.sh_ptr[k]; e < t.sh_ptr[k + 1]; ++e) {
      const int pw = t.sh_pow[e];
      double m = t.sh_coef[e];
      for (int q = 0; q < (pw & 15); ++q) m *= x;
      for (int q = 0; q < ((pw >> 4) & 15); ++q) m *= y;
      for (int q = 0; q < ((pw >> 8) & 15); ++q) m *= z;
      acc += m;
    }
    sink(k, acc);
  }
}

__global__ void k_plan_init(int* __restrict__ st, unsigned* __restrict__ dmin) {
  if (threadIdx.x < 3) st[threadIdx.x] = INT_MAX;
  else if (threadIdx.x < 6) st[threadIdx.x] = INT_MIN;
  else if (threadIdx.x < kStatsInts) st[threadIdx.x] = 0;
  if (threadIdx.x == 0 && dmin) *dmin = 0x7f800000u;  // +inf
}

__global__ void k_plan_bbox(const float* __restrict__ pos, const int32_t* __restrict__ gid, int n,
                            int* __restrict__ st) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  for (int k = 0; k < 3; ++k) {
    const float x = pos[3 * i + k];
    if (!(fabsf(x) < 16384.0f)) {  // also catches NaN; the atom is then kept out of the box
      atomicOr(&st[7], 1);
      return;
    }
    const int X = __float2int_rn(x * 65536.0f);
    atomicMin(&st[k], X);
    atomicMax(&st[3 + k], X);
  }
  if (gid) {
    const int g = gid[i];
    if (g < 0) atomicOr(&st[7], 2);
    else atomicMax(&st[6], g);
  }
}

// Shortest nonzero edge length (fp32 bits; positive floats order like their
// bits), one atomic per wave.
__global__ void k_plan_dmin(const float* __restrict__ pos, const int32_t* __restrict__ rows,
                            const int32_t* __restrict__ col, int n, int64_t n_edges, unsigned* __restrict__ dmin) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  unsigned v = 0x7f800000u;
  if (e < n_edges) {
    const int i = clamp_node(rows[e], n), j = clamp_node(col[e], n);
    const float dx = pos[3 * i] - pos[3 * j], dy = pos[3 * i + 1] - pos[3 * j + 1], dz = pos[3 * i + 2] - pos[3 * j + 2];
    const float d = sqrtf(dx * dx + dy * dy + dz * dz);
    if (d > 0.0f && d < INFINITY) v = __float_as_uint(d);
  }
  for (int o = 32; o > 0; o >>= 1) v = min(v, (unsigned)__shfl_xor((int)v, o));
  if ((threadIdx.x & 63) == 0 && v != 0x7f800000u) atomicMin(dmin, v);
}

// One thread: the tile grid from the bounding box.  The side is `side`
// grid units, or, when dmin is given, at most dmin_scale times the shortest
// edge; at least 1/64 A, at most 1024 tiles per axis, and graphs x tiles
// below 2^31.
__global__ void k_plan_grid(const int* __restrict__ st, const unsigned* __restrict__ dmin, double side,
                            double dmin_scale, bool graphs, TileGridDev* __restrict__ g) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  int lo[3], hi[3];
  for (int k = 0; k < 3; ++k) {
    lo[k] = st[k], hi[k] = st[3 + k];
    if (lo[k] > hi[k]) lo[k] = hi[k] = 0;  // no finite position
  }
  if (dmin) {
    const float d = __uint_as_float(*dmin);
    if (d < INFINITY) side = fmin(side, dmin_scale * (double)d * kGrid);
  }
  side = fmax(side, kGrid / 64.0);
  const int64_t ngraph = graphs ? (int64_t)st[6] + 1 : 1;
  for (;;) {
    int64_t ncell = 1;
    for (int k = 0; k < 3; ++k) {
      g->lo[k] = lo[k];
      g->span[k] = (int64_t)hi[k] - lo[k] + 1;
      int64_t d = (int64_t)ceil((double)g->span[k] / side);
      d = d < 1 ? 1 : (d > 1024 ? 1024 : d);
      g->dim[k] = (int)d;
      ncell *= d;
    }
    if (ncell * ngraph < ((int64_t)1 << 31) || side > 1e18) {
      g->ncell = (int)ncell;
      break;
    }
    side *= 2.0;
  }
}

__device__ __forceinline__ int tile_axis(float x, const TileGridDev& g, int k) {
  const int64_t X = __float2int_rn(x * 65536.0f);
  int64_t q = (X - g.lo[k]) * g.dim[k] / g.span[k];
  return (int)(q < 0 ? 0 : (q > g.dim[k] - 1 ? g.dim[k] - 1 : q));
}

// tile_of[i] = graph * ncell + cell; keys for the receiver order: graph in
// the high 32 bits, then the Morton index of 4 A cells of the box.
__global__ void k_plan_tiles(const float* __restrict__ pos, const int32_t* __restrict__ gid, int n,
                             const TileGridDev* __restrict__ gp, int32_t* __restrict__ tile_of,
                             uint64_t* __restrict__ keys, int32_t* __restrict__ vals) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const TileGridDev g = *gp;
  const float p[3] = {pos[3 * i], pos[3 * i + 1], pos[3 * i + 2]};
  const int c0 = tile_axis(p[0], g, 0), c1 = tile_axis(p[1], g, 1), c2 = tile_axis(p[2], g, 2);
  const int graph = gid ? max(gid[i], 0) : 0;
  tile_of[i] = graph * g.ncell + (c2 * g.dim[1] + c1) * g.dim[0] + c0;
  uint32_t m = 0;
  for (int k = 0; k < 3; ++k) {
    int64_t c = ((int64_t)__float2int_rn(p[k] * 65536.0f) - g.lo[k]) / (int64_t)(4.0 * kGrid);
    c = c < 0 ? 0 : (c > 1023 ? 1023 : c);
    uint32_t v = (uint32_t)c;
    v = (v | (v << 16)) & 0x030000ff;
    v = (v | (v << 8)) & 0x0300f00f;
    v = (v | (v << 4)) & 0x030c30c3;
    v = (v | (v << 2)) & 0x09249249;
    m |= v << k;
  }
  keys[i] = ((uint64_t)(uint32_t)graph << 32) | m;
  vals[i] = i;
}

// Solid harmonics of every receiver about its tile centre, fp64 [n][nk].
template <int L>
__global__ __launch_bounds__(256) void k_plan_node_sh(DevTables t, const float* __restrict__ pos, int n,
                                                      const int32_t* __restrict__ tile_of,
                                                      const TileGridDev* __restrict__ gp, double* __restrict__ R) {
  constexpr int NK = (L + 1) * (L + 1);
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const TileGridDev g = *gp;
  double ox, oy, oz;
  tile_centre(g, tile_of[i] % g.ncell, ox, oy, oz);
  double* Ri = R + (size_t)i * NK;
  sh_all<L>(t, (double)pos[3 * i] - ox, (double)pos[3 * i + 1] - oy, (double)pos[3 * i + 2] - oz,
            [&](int k, double v) { Ri[k] = v; });
}

// Solid harmonics of every edge's sender about its receiver's tile centre,
// fp32 [E][nk] in CSR order.  A thread per edge (rows: the receiver of every
// edge), 256 consecutive edges per workgroup; the values pass through LDS so
// that the workgroup stores its 256 rows as one contiguous block.
template <int L>
__global__ __launch_bounds__(256) void k_plan_edge_sh(DevTables t, const float* __restrict__ pos,
                                                      const int32_t* __restrict__ rows,
                                                      const int32_t* __restrict__ col, int n, int64_t n_edges,
                                                      const int32_t* __restrict__ tile_of,
                                                      const TileGridDev* __restrict__ gp, float* __restrict__ Re) {
  constexpr int NK = (L + 1) * (L + 1), NKP = NK | 1;  // odd row stride: conflict-free LDS stores
  __shared__ float buf[256 * NKP];
  const int64_t e0 = (int64_t)blockIdx.x * 256, e = e0 + threadIdx.x;
  const int cnt = (int)min((int64_t)256, n_edges - e0);
  if (e < n_edges) {
    const TileGridDev g = *gp;
    const int i = clamp_node(rows[e], n), j = clamp_node(col[e], n);
    double ox, oy, oz;
    tile_centre(g, tile_of[i] % g.ncell, ox, oy, oz);
    float* b = buf + threadIdx.x * NKP;
    sh_all<L>(t, (double)pos[3 * j] - ox, (double)pos[3 * j + 1] - oy, (double)pos[3 * j + 2] - oz,
              [&](int k, double v) { b[k] = (float)v; });
  }
  __syncthreads();
  float* dst = Re + e0 * NK;
  for (int q = threadIdx.x; q < cnt * NK; q += 256) dst[q] = buf[(q / NK) * NKP + q % NK];
}

// The receiver of every edge (rows [E]), clamped like every CSR read.
// A wave per receiver, its lanes over the receiver's edges.
__global__ __launch_bounds__(256) void k_plan_edge_rows(const int64_t* __restrict__ row_ptr, int n, int64_t n_edges,
                                                        int32_t* __restrict__ rows) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (i >= n) return;
  int64_t e0, e1;
  row_bounds(row_ptr, i, n_edges, e0, e1);
  for (int64_t e = e0 + lane; e < e1; e += 64) rows[e] = i;
}

__global__ void k_fill(float* __restrict__ p, int64_t count, float v) {
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < count; q += (int64_t)gridDim.x * blockDim.x)
    p[q] = v;
}

// The centre of the bounding box (grid units halved exactly, as on the host
// before), in Angstrom; the box of no finite position is the origin.
__global__ void k_plan_centre(const int* __restrict__ st, double* __restrict__ org) {
  if (threadIdx.x < 3) {
    const int k = threadIdx.x;
    const bool empty = st[k] > st[3 + k];
    org[k] = empty ? 0.0 : (double)((((int64_t)st[k] + st[3 + k]) / 2)) / kGrid;
  }
}

// Graph check: bit 1 row_ptr[0] != 0, bit 2 a row end below its start,
// bit 4 row_ptr[n] != E, bit 8 a sender outside [0, n).
__global__ void k_validate_rows(const int64_t* __restrict__ row_ptr, int n, int64_t n_edges, int* __restrict__ bad) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i > n) return;
  int b = 0;
  if (i == 0 && row_ptr[0] != 0) b |= 1;
  if (i < n && row_ptr[i + 1] < row_ptr[i]) b |= 2;
  if (i == n && row_ptr[n] != n_edges) b |= 4;
  if (b) atomicOr(bad, b);
}

__global__ void k_validate_cols(const int32_t* __restrict__ col, int n, int64_t n_edges, int* __restrict__ bad) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  bool out = e < n_edges && (unsigned)col[e] >= (unsigned)n;
  if (__any(out) && (threadIdx.x & 63) == 0) atomicOr(bad, 8);
}

}  // namespace

hipError_t launch_plan_bbox(const float* pos, const int32_t* graph_id, int n, int* stats, unsigned* dmin,
                            hipStream_t s) {
  k_plan_init<<<1, 64, 0, s>>>(stats, dmin);
  if (n > 0) k_plan_bbox<<<(n + 255) / 256, 256, 0, s>>>(pos, graph_id, n, stats);
  return hipGetLastError();
}

hipError_t launch_plan_centre(const int* stats, double* origin, hipStream_t s) {
  k_plan_centre<<<1, 64, 0, s>>>(stats, origin);
  return hipGetLastError();
}

hipError_t launch_plan_dmin(const float* pos, const int32_t* rows, const int32_t* col, int n, int64_t n_edges,
                            unsigned* dmin, hipStream_t s) {
  const int64_t blocks = (n_edges + 255) / 256;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  if (blocks > 0) k_plan_dmin<<<(unsigned)blocks, 256, 0, s>>>(pos, rows, col, n, n_edges, dmin);
  return hipGetLastError();
}

hipError_t launch_plan_grid(const int* stats, const unsigned* dmin, double side, double dmin_scale, bool graphs,
                            TileGridDev* grid, hipStream_t s) {
  k_plan_grid<<<1, 64, 0, s>>>(stats, dmin, side, dmin_scale, graphs, grid);
  return hipGetLastError();
}

size_t plan_sort_tmp_bytes(int n) {
  size_t b = 0;
  hipcub::DeviceRadixSort::SortPairs(nullptr, b, (const uint64_t*)nullptr, (uint64_t*)nullptr,
                                     (const int32_t*)nullptr, (int32_t*)nullptr, n);
  return b;
}

hipError_t launch_plan_order(const float* pos, const int32_t* graph_id, int n, const TileGridDev* grid,
                             int32_t* tile_of, uint64_t* keys, uint64_t* keys_out, int32_t* vals, int32_t* order,
                             void* tmp, size_t tmp_bytes, hipStream_t s) {
  if (n == 0) return hipSuccess;
  k_plan_tiles<<<(n + 255) / 256, 256, 0, s>>>(pos, graph_id, n, grid, tile_of, keys, vals);
  size_t b = tmp_bytes;
  return hipcub::DeviceRadixSort::SortPairs(tmp, b, keys, keys_out, vals, order, n, 0, graph_id ? 64 : 30, s);
}

hipError_t launch_plan_sh(const DevTables& t, const float* pos, const int32_t* rows, const int32_t* col, int n,
                          int64_t n_edges, const int32_t* tile_of, const TileGridDev* grid, double* Rr, float* Re,
                          hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int64_t eblocks = (n_edges + 255) / 256;
  if (eblocks > 0x7fffffff) return hipErrorInvalidValue;
  switch (t.L) {
#define E2F_SH(LL)                                                                                          \
  case LL:                                                                                                  \
    k_plan_node_sh<LL><<<(n + 255) / 256, 256, 0, s>>>(t, pos, n, tile_of, grid, Rr);                       \
    if (eblocks > 0)                                                                                        \
      k_plan_edge_sh<LL><<<(unsigned)eblocks, 256, 0, s>>>(t, pos, rows, col, n, n_edges, tile_of, grid, Re); \
    break;
    E2F_SH(0) E2F_SH(1) E2F_SH(2) E2F_SH(3) E2F_SH(4) E2F_SH(5) E2F_SH(6)
#undef E2F_SH
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_plan_edge_rows(const int64_t* row_ptr, int n, int64_t n_edges, int32_t* rows, hipStream_t s) {
  if (n > 0) k_plan_edge_rows<<<(n + 3) / 4, 256, 0, s>>>(row_ptr, n, n_edges, rows);
  return hipGetLastError();
}

hipError_t launch_fill(float* p, int64_t count, float v, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((count + 255) / 256, 8192);
  k_fill<<<(unsigned)blocks, 256, 0, s>>>(p, count, v);
  return hipGetLastError();
}

hipError_t launch_validate_graph(const int64_t* row_ptr, const int32_t* col, int n, int64_t n_edges, int* bad,
                                 hipStream_t s) {
  k_fill<<<1, 64, 0, s>>>((float*)bad, 1, 0.0f);  // 0.0f has the bits of int 0
  k_validate_rows<<<(n + 1 + 255) / 256, 256, 0, s>>>(row_ptr, n, n_edges, bad);
  const int64_t blocks = (n_edges + 255) / 256;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  if (blocks > 0) k_validate_cols<<<(unsigned)blocks, 256, 0, s>>>(col, n, n_edges, bad);
  return hipGetLastError();
}

}  // namespace e2f
