// Radius graph on gfx950 (Alg. 1 step 2: D_ij = |r_i - r_j|, kept below the
// cutoff).  Cell list with integer cell coordinates on the 2^-16 A grid:
//   bbox (atomic min/max) -> cell counts -> exclusive scan -> cell members ->
//   per-atom neighbour count over the 27 cells (exact integer predicate; one
//   64-lane workgroup per atom) -> exclusive scan into row_ptr -> fill with
//   every row sorted in LDS (rows above 1024: fill, then a segmented sort).
// Only integer atomics are used, and the rows are sorted at the end, so the
// CSR is bitwise deterministic.
#include <hip/hip_runtime.h>
#include <hipcub/hipcub.hpp>

#include <algorithm>

#include "e2f_launch.h"

namespace e2f {
namespace {

__device__ __forceinline__ int grid_coord(float x) { return __float2int_rn(x * 65536.0f); }

// Bounding box on the grid (stats as in launch_bbox): each lane's atom, a
// reduction over the wave and the workgroup, then one atomic per workgroup
// and value.  An atom with a coordinate that is not finite or beyond
// +-16384 A sets bit 1 and stays out of the box; a negative graph id sets
// bit 2.
__global__ __launch_bounds__(256) void k_bbox(const float* __restrict__ pos, const int32_t* __restrict__ gid, int n,
                                              int* __restrict__ st) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  int lo[3] = {INT_MAX, INT_MAX, INT_MAX}, hi[3] = {INT_MIN, INT_MIN, INT_MIN}, gmax = 0, bad = 0;
  if (i < n) {
    float x[3];
    bool ok = true;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      x[k] = pos[3 * i + k];
      ok = ok && fabsf(x[k]) < 16384.0f;  // also false for NaN
    }
    if (ok) {
#pragma unroll
      for (int k = 0; k < 3; ++k) lo[k] = hi[k] = grid_coord(x[k]);
    } else {
      bad |= 1;
    }
    if (gid) {
      const int g = gid[i];
      if (g < 0) bad |= 2;
      else gmax = g;
    }
  }
  for (int o = 32; o > 0; o >>= 1) {  // every lane takes part
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      lo[k] = min(lo[k], __shfl_xor(lo[k], o));
      hi[k] = max(hi[k], __shfl_xor(hi[k], o));
    }
    gmax = max(gmax, __shfl_xor(gmax, o));
    bad |= __shfl_xor(bad, o);
  }
  __shared__ int part[4][8];  // the waves' results, then one atomic per workgroup and value
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
#pragma unroll
    for (int k = 0; k < 3; ++k) part[wave][k] = lo[k], part[wave][3 + k] = hi[k];
    part[wave][6] = gmax, part[wave][7] = bad;
  }
  __syncthreads();
  if (threadIdx.x < 8) {
    const int q = threadIdx.x;
    int v = part[0][q];
    for (int w = 1; w < (int)(blockDim.x >> 6); ++w) {
      const int u = part[w][q];
      v = q < 3 ? min(v, u) : (q < 7 ? max(v, u) : (v | u));
    }
    if (q < 3) {
      if (v != INT_MAX) atomicMin(&st[q], v);
    } else if (q < 6) {
      if (v != INT_MIN) atomicMax(&st[q], v);
    } else if (q == 6) {
      if (v > 0) atomicMax(&st[6], v);
    } else if (v) {
      atomicOr(&st[7], v);
    }
  }
}

__global__ void k_stats_init(int* st) {
  if (threadIdx.x < 3) st[threadIdx.x] = INT_MAX;
  else if (threadIdx.x < 6) st[threadIdx.x] = INT_MIN;
  else if (threadIdx.x < kStatsInts) st[threadIdx.x] = 0;
}

struct Grid {
  int lo0, lo1, lo2;
  int d0, d1, d2;
  int64_t side;
};

__device__ __forceinline__ int cell_axis(int X, int lo, int64_t side, int d) {
  int64_t c = ((int64_t)X - lo) / side;
  return (int)(c < d - 1 ? c : d - 1);
}

__global__ void k_cell_count(const float* __restrict__ pos, int n, Grid g, int* __restrict__ cell_of,
                             int* __restrict__ cell_cnt) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int cx = cell_axis(grid_coord(pos[3 * i]), g.lo0, g.side, g.d0);
  const int cy = cell_axis(grid_coord(pos[3 * i + 1]), g.lo1, g.side, g.d1);
  const int cz = cell_axis(grid_coord(pos[3 * i + 2]), g.lo2, g.side, g.d2);
  const int c = (cz * g.d1 + cy) * g.d0 + cx;
  cell_of[i] = c;
  atomicAdd(&cell_cnt[c], 1);
}

__global__ void k_cell_place(int n, const int* __restrict__ cell_of, const int* __restrict__ cell_start,
                             int* __restrict__ cell_fill, int* __restrict__ members) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int c = cell_of[i];
  members[cell_start[c] + atomicAdd(&cell_fill[c], 1)] = i;
}

// Count (out == nullptr) or write the neighbours of atom i.
template <bool WRITE>
__global__ void k_neighbors(const float* __restrict__ pos, const int32_t* __restrict__ gid, int n, double r2, Grid g,
                            const int* __restrict__ cell_of, const int* __restrict__ cell_start,
                            const int* __restrict__ members, int64_t* __restrict__ counts,
                            const int64_t* __restrict__ row_ptr, int32_t* __restrict__ out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int xi = grid_coord(pos[3 * i]), yi = grid_coord(pos[3 * i + 1]), zi = grid_coord(pos[3 * i + 2]);
  const int gi = gid ? gid[i] : 0;
  const int c = cell_of[i];
  const int cx = c % g.d0, cy = (c / g.d0) % g.d1, cz = c / (g.d0 * g.d1);
  int64_t cnt = 0;
  int64_t w = WRITE ? row_ptr[i] : 0;
  for (int dz = -1; dz <= 1; ++dz) {
    const int z = cz + dz;
    if (z < 0 || z >= g.d2) continue;
    for (int dy = -1; dy <= 1; ++dy) {
      const int y = cy + dy;
      if (y < 0 || y >= g.d1) continue;
      for (int dx = -1; dx <= 1; ++dx) {
        const int x = cx + dx;
        if (x < 0 || x >= g.d0) continue;
        const int cc = (z * g.d1 + y) * g.d0 + x;
        for (int q = cell_start[cc]; q < cell_start[cc + 1]; ++q) {
          const int j = members[q];
          if (j == i) continue;
          if (gid && gid[j] != gi) continue;
          const int64_t ddx = (int64_t)grid_coord(pos[3 * j]) - xi;
          const int64_t ddy = (int64_t)grid_coord(pos[3 * j + 1]) - yi;
          const int64_t ddz = (int64_t)grid_coord(pos[3 * j + 2]) - zi;
          const int64_t d2 = ddx * ddx + ddy * ddy + ddz * ddz;  // < 2^53 for cutoff <= 64 A
          if ((double)d2 < r2) {
            if (WRITE) out[w++] = j;
            else ++cnt;
          }
        }
      }
    }
  }
  if (!WRITE) counts[i] = cnt;
}

// One 64-lane workgroup per atom i: the members of the 27 cells around i are
// enumerated as one list through a prefix over the cells (lane c < 27 holds
// cell c), 64 candidates at a time.  Count: ballot totals, and the largest
// degree.  Fill: the row is collected in LDS, sorted there (bitonic) and
// written in ascending order; rows longer than kNlRowMax take the global
// segmented sort instead (the host picks the path from the largest degree).
constexpr int kNlRowMax = 1024;

__device__ __forceinline__ int wave_prefix_incl(int v, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(v, o);
    if (lane >= o) v += u;
  }
  return v;
}

template <bool WRITE>
__global__ __launch_bounds__(64) void k_neighbors_wave(const float* __restrict__ pos, const int32_t* __restrict__ gid,
                                                       int n, double r2, Grid g, const int* __restrict__ cell_of,
                                                       const int* __restrict__ cell_start,
                                                       const int* __restrict__ members, int64_t* __restrict__ counts,
                                                       int* __restrict__ max_degree,
                                                       const int64_t* __restrict__ row_ptr, int32_t* __restrict__ out) {
  __shared__ int32_t row[kNlRowMax];
  const int i = blockIdx.x, lane = threadIdx.x;
  const int xi = grid_coord(pos[3 * i]), yi = grid_coord(pos[3 * i + 1]), zi = grid_coord(pos[3 * i + 2]);
  const int gi = gid ? gid[i] : 0;
  const int c = cell_of[i];
  const int cx = c % g.d0, cy = (c / g.d0) % g.d1, cz = c / (g.d0 * g.d1);
  // lane q < 27: neighbour cell q (dx, dy, dz in -1..1), its first member and count
  int cs = 0, cn = 0;
  if (lane < 27) {
    const int x = cx + lane % 3 - 1, y = cy + (lane / 3) % 3 - 1, z = cz + lane / 9 - 1;
    if (x >= 0 && x < g.d0 && y >= 0 && y < g.d1 && z >= 0 && z < g.d2) {
      const int cc = (z * g.d1 + y) * g.d0 + x;
      cs = cell_start[cc];
      cn = cell_start[cc + 1] - cs;
    }
  }
  const int incl = wave_prefix_incl(cn, lane);
  const int total = __shfl(incl, 63);
  int found = 0;
  for (int t0 = 0; t0 < total; t0 += 64) {
    // every lane searches (the shuffles need the whole wave); lanes past the
    // list search for the last candidate and count nothing
    const int t = t0 + lane;
    const bool valid = t < total;
    const int tc = valid ? t : total - 1;
    // cell of candidate tc: the first q with incl[q] > tc, i.e. the number of
    // q with incl[q] <= tc (incl is nondecreasing and incl[26..63] = total >
    // tc).  Five fixed steps with no branch around the shuffles: every lane
    // of the wave takes part in each one (a lane that had left a data-dependent
    // loop would not supply its value).
    int lo = 0;
#pragma unroll
    for (int step = 16; step >= 1; step >>= 1) {
      const int v = __shfl(incl, lo + step - 1);
      lo += v <= tc ? step : 0;
    }
    const int cnl = __shfl(cn, lo), off = tc - (__shfl(incl, lo) - cnl), base = __shfl(cs, lo);
    const bool inr = off >= 0 && off < cnl;  // always true; keeps every read inside the cell
    const int j = inr ? members[base + off] : i;
    bool hit = false;
    if (valid && j != i && (!gid || gid[j] == gi)) {
      const int64_t ddx = (int64_t)grid_coord(pos[3 * j]) - xi;
      const int64_t ddy = (int64_t)grid_coord(pos[3 * j + 1]) - yi;
      const int64_t ddz = (int64_t)grid_coord(pos[3 * j + 2]) - zi;
      const int64_t d2 = ddx * ddx + ddy * ddy + ddz * ddz;  // < 2^53 for cutoff <= 64 A
      hit = (double)d2 < r2;
    }
    const uint64_t m = __ballot(hit);
    if (WRITE && hit) {
      const int rank = __popcll(m & ((1ull << lane) - 1));
      row[found + rank] = j;
    }
    found += __popcll(m);
  }
  if (!WRITE) {
    if (lane == 0) counts[i] = found;
    return;
  }
  __syncthreads();
  int p2 = 1;
  while (p2 < found) p2 <<= 1;
  for (int q = found + lane; q < p2; q += 64) row[q] = INT_MAX;
  __syncthreads();
  for (int size = 2; size <= p2; size <<= 1)
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int t = lane; t < p2 / 2; t += 64) {
        const int lo = 2 * t - (t & (stride - 1)), hi = lo + stride;
        const bool up = (lo & size) == 0;
        const int a = row[lo], b = row[hi];
        if ((a > b) == up) {
          row[lo] = b;
          row[hi] = a;
        }
      }
      __syncthreads();
    }
  const int64_t r0 = row_ptr[i];
  for (int q = lane; q < found; q += 64) out[r0 + q] = row[q];
}

__global__ void k_zero_last(int64_t* counts, int n) { counts[n] = 0; }

// Largest row length: a maximum per workgroup (wave shuffles, then the four
// waves through LDS), one atomic per workgroup.
__global__ __launch_bounds__(256) void k_degree_max(const int64_t* __restrict__ counts, int n,
                                                    int* __restrict__ max_degree) {
  __shared__ int wmax[4];
  int m = 0;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    m = max(m, (int)counts[i]);
  for (int o = 32; o > 0; o >>= 1) m = max(m, __shfl_xor(m, o));
  if ((threadIdx.x & 63) == 0) wmax[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) atomicMax(max_degree, max(max(wmax[0], wmax[1]), max(wmax[2], wmax[3])));
}

// ---------------------------------------------------------------- kNN graph
// k nearest neighbours (the sparse graphs of the scaling study, Sec. 4.1):
// row i holds the min(k, n_g - 1) atoms j != i of i's graph that come first
// in (squared distance on the 2^-16 A grid, index) order, by ascending index.
// Row sizes follow from the graph sizes alone (integer atomics); the rows
// are filled by one workgroup per receiver that streams every candidate,
// keeps those ahead of the current k-th (distance, index) pair in an LDS
// buffer and cuts the buffer back to k by a bitonic sort when it could
// overflow.  The result does not depend on the order of arrival.
constexpr int kKnnBuf = 2048;

__global__ void k_knn_graph_sizes(const int32_t* __restrict__ gid, int n, int* __restrict__ gsize) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) atomicAdd(&gsize[gid ? gid[i] : 0], 1);
}

__global__ void k_knn_row_sizes(const int32_t* __restrict__ gid, int n, int k, const int* __restrict__ gsize,
                                int64_t* __restrict__ counts) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) counts[i] = min(k, gsize[gid ? gid[i] : 0] - 1);
  if (i == 0) counts[n] = 0;
}

__device__ __forceinline__ bool knn_less(uint64_t da, int ja, uint64_t db, int jb) {
  return da < db || (da == db && ja < jb);
}

// bitonic sort of (d, j)[0, m) ascending, m a power of two, 256 threads
__device__ void knn_sort(uint64_t* d, int32_t* j, int m) {
  for (int size = 2; size <= m; size <<= 1)
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int t = threadIdx.x; t < m / 2; t += blockDim.x) {
        const int lo = 2 * t - (t & (stride - 1)), hi = lo + stride;
        const bool up = (lo & size) == 0;
        if (knn_less(d[hi], j[hi], d[lo], j[lo]) == up) {
          const uint64_t td = d[lo];
          d[lo] = d[hi];
          d[hi] = td;
          const int32_t tj = j[lo];
          j[lo] = j[hi];
          j[hi] = tj;
        }
      }
      __syncthreads();
    }
}

__global__ __launch_bounds__(256) void k_knn_fill(const float* __restrict__ pos, const int32_t* __restrict__ gid,
                                                  int n, int k, const int64_t* __restrict__ row_ptr,
                                                  int32_t* __restrict__ col) {
  __shared__ uint64_t bd[kKnnBuf];
  __shared__ int32_t bj[kKnnBuf];
  __shared__ int cnt;
  __shared__ uint64_t thr_d;
  __shared__ int thr_j;
  const int i = blockIdx.x, t = threadIdx.x;
  const int64_t r0 = row_ptr[i];
  const int m = (int)(row_ptr[i + 1] - r0);  // min(k, n_g - 1)
  if (m == 0) return;                          // uniform over the workgroup
  const int gi = gid ? gid[i] : 0;
  const int64_t xi = grid_coord(pos[3 * i]), yi = grid_coord(pos[3 * i + 1]), zi = grid_coord(pos[3 * i + 2]);
  if (t == 0) {
    cnt = 0;
    thr_d = ~0ull;
    thr_j = INT_MAX;
  }
  __syncthreads();
  for (int j0 = 0; j0 < n; j0 += blockDim.x) {
    const int j = j0 + t;
    if (j < n && j != i && (!gid || gid[j] == gi)) {
      const int64_t dx = grid_coord(pos[3 * j]) - xi, dy = grid_coord(pos[3 * j + 1]) - yi,
                    dz = grid_coord(pos[3 * j + 2]) - zi;
      const uint64_t d = (uint64_t)(dx * dx) + (uint64_t)(dy * dy) + (uint64_t)(dz * dz);
      if (knn_less(d, j, thr_d, thr_j)) {
        const int p = atomicAdd(&cnt, 1);  // < kKnnBuf: the buffer is cut below kKnnBuf - 256
        bd[p] = d;
        bj[p] = j;
      }
    }
    __syncthreads();
    const int c = cnt;  // the same in every thread: nobody appends before the next barrier
    __syncthreads();
    if (c > kKnnBuf - (int)blockDim.x || (j0 + (int)blockDim.x >= n && c > 0)) {
      for (int q = c + t; q < kKnnBuf; q += blockDim.x) {
        bd[q] = ~0ull;
        bj[q] = INT_MAX;
      }
      __syncthreads();
      knn_sort(bd, bj, kKnnBuf);
      if (t == 0) {
        cnt = min(c, k);
        if (c >= k) {
          thr_d = bd[k - 1];
          thr_j = bj[k - 1];
        }
      }
      __syncthreads();
    }
  }
  // the m nearest are bd/bj[0, m); write them by ascending index
  int p2 = 1;
  while (p2 < m) p2 <<= 1;
  for (int q = t; q < p2; q += blockDim.x) {
    bd[q] = 0;
    if (q >= m) bj[q] = INT_MAX;
  }
  __syncthreads();
  knn_sort(bd, bj, p2);
  for (int q = t; q < m; q += blockDim.x) col[r0 + q] = bj[q];
}

Grid to_grid(const CellGrid& cg) {
  return Grid{cg.lo[0], cg.lo[1], cg.lo[2], cg.dim[0], cg.dim[1], cg.dim[2], cg.side};
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

struct NlScratch {
  int* cell_of;
  int* cell_cnt;    // ncell + 1 (becomes the fill cursor)
  int* cell_start;  // ncell + 1
  int* members;
  int64_t* counts;  // n + 1
  void* scan_tmp;
  size_t scan_bytes;
};

size_t scan_bytes_cells(int64_t ncell) {
  size_t b = 0;
  hipcub::DeviceScan::ExclusiveSum(nullptr, b, (int*)nullptr, (int*)nullptr, (int)(ncell + 1));
  return b;
}
size_t scan_bytes_counts(int n) {
  size_t b = 0;
  hipcub::DeviceScan::ExclusiveSum(nullptr, b, (int64_t*)nullptr, (int64_t*)nullptr, n + 1);
  return b;
}

NlScratch carve(void* base, int n, const CellGrid& g) {
  char* p = (char*)base;
  NlScratch s;
  s.cell_of = (int*)p; p += align256(sizeof(int) * (size_t)n);
  s.cell_cnt = (int*)p; p += align256(sizeof(int) * (size_t)(g.ncell + 1));
  s.cell_start = (int*)p; p += align256(sizeof(int) * (size_t)(g.ncell + 1));
  s.members = (int*)p; p += align256(sizeof(int) * (size_t)n);
  s.counts = (int64_t*)p; p += align256(sizeof(int64_t) * (size_t)(n + 1));
  s.scan_bytes = std::max(scan_bytes_cells(g.ncell), scan_bytes_counts(n));
  s.scan_tmp = p;
  return s;
}

}  // namespace

hipError_t launch_bbox(const float* pos, const int32_t* graph_id, int n, int* stats, hipStream_t s) {
  k_stats_init<<<1, 64, 0, s>>>(stats);
  if (n > 0) k_bbox<<<(n + 255) / 256, 256, 0, s>>>(pos, graph_id, n, stats);
  return hipGetLastError();
}

size_t nl_scratch_bytes(int n, const CellGrid& g) {
  size_t b = 0;
  b += align256(sizeof(int) * (size_t)n);
  b += 2 * align256(sizeof(int) * (size_t)(g.ncell + 1));
  b += align256(sizeof(int) * (size_t)n);
  b += align256(sizeof(int64_t) * (size_t)(n + 1));
  b += align256(std::max(scan_bytes_cells(g.ncell), scan_bytes_counts(n)));
  return b;
}

hipError_t launch_nl_count(const float* pos, const int32_t* graph_id, int n, double r2, const CellGrid& cg,
                           void* scratch, int64_t* row_ptr, int* max_degree, hipStream_t st) {
  NlScratch s = carve(scratch, n, cg);
  Grid g = to_grid(cg);
  hipError_t e = hipMemsetAsync(s.cell_cnt, 0, sizeof(int) * (size_t)(cg.ncell + 1), st);
  if (e != hipSuccess) return e;
  const int blocks = (n + 255) / 256;
  k_cell_count<<<blocks, 256, 0, st>>>(pos, n, g, s.cell_of, s.cell_cnt);
  size_t tb = s.scan_bytes;
  e = hipcub::DeviceScan::ExclusiveSum(s.scan_tmp, tb, s.cell_cnt, s.cell_start, (int)(cg.ncell + 1), st);
  if (e != hipSuccess) return e;
  e = hipMemsetAsync(s.cell_cnt, 0, sizeof(int) * (size_t)(cg.ncell + 1), st);
  if (e != hipSuccess) return e;
  k_cell_place<<<blocks, 256, 0, st>>>(n, s.cell_of, s.cell_start, s.cell_cnt, s.members);
  if ((e = hipMemsetAsync(max_degree, 0, sizeof(int), st)) != hipSuccess) return e;
  k_neighbors_wave<false><<<n, 64, 0, st>>>(pos, graph_id, n, r2, g, s.cell_of, s.cell_start, s.members, s.counts,
                                            max_degree, nullptr, nullptr);
  k_degree_max<<<std::min((n + 255) / 256, 256), 256, 0, st>>>(s.counts, n, max_degree);
  k_zero_last<<<1, 1, 0, st>>>(s.counts, n);
  tb = s.scan_bytes;
  e = hipcub::DeviceScan::ExclusiveSum(s.scan_tmp, tb, s.counts, row_ptr, n + 1, st);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

size_t nl_sort_tmp_bytes(int n, int64_t E) {
  size_t b = 0;
  hipcub::DeviceSegmentedRadixSort::SortKeys(nullptr, b, (const int32_t*)nullptr, (int32_t*)nullptr, (int)E, n,
                                             (const int64_t*)nullptr, (const int64_t*)nullptr, 0, 32);
  return b;
}

hipError_t launch_nl_fill(const float* pos, const int32_t* graph_id, int n, double r2, const CellGrid& cg,
                          void* scratch, const int64_t* row_ptr, int32_t* unsorted, int32_t* col_idx, int64_t E,
                          int max_degree, void* sort_tmp, size_t sort_tmp_bytes, hipStream_t st) {
  NlScratch s = carve(scratch, n, cg);
  Grid g = to_grid(cg);
  if (max_degree <= kNlRowMax) {  // rows sorted in LDS
    k_neighbors_wave<true><<<n, 64, 0, st>>>(pos, graph_id, n, r2, g, s.cell_of, s.cell_start, s.members, nullptr,
                                             nullptr, row_ptr, col_idx);
    return hipGetLastError();
  }
  k_neighbors<true><<<(n + 255) / 256, 256, 0, st>>>(pos, graph_id, n, r2, g, s.cell_of, s.cell_start, s.members,
                                                    nullptr, row_ptr, unsorted);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  int bits = 1;
  while ((1LL << bits) < (int64_t)n) ++bits;
  size_t tb = sort_tmp_bytes;
  e = hipcub::DeviceSegmentedRadixSort::SortKeys(sort_tmp, tb, unsorted, col_idx, (int)E, n, row_ptr, row_ptr + 1, 0,
                                                 bits, st);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

size_t knn_scratch_bytes(int n, int ngraph) {
  return align256(sizeof(int) * (size_t)ngraph) + align256(sizeof(int64_t) * (size_t)(n + 1)) +
         align256(scan_bytes_counts(n));
}

hipError_t launch_knn_count(const int32_t* graph_id, int n, int k, int ngraph, void* scratch, int64_t* row_ptr,
                            hipStream_t s) {
  char* p = (char*)scratch;
  int* gsize = (int*)p;
  p += align256(sizeof(int) * (size_t)ngraph);
  int64_t* counts = (int64_t*)p;
  p += align256(sizeof(int64_t) * (size_t)(n + 1));
  void* tmp = p;
  hipError_t e = hipMemsetAsync(gsize, 0, sizeof(int) * (size_t)ngraph, s);
  if (e != hipSuccess) return e;
  k_knn_graph_sizes<<<(n + 255) / 256, 256, 0, s>>>(graph_id, n, gsize);
  k_knn_row_sizes<<<(n + 256) / 256, 256, 0, s>>>(graph_id, n, k, gsize, counts);
  size_t b = scan_bytes_counts(n);
  if ((e = hipcub::DeviceScan::ExclusiveSum(tmp, b, counts, row_ptr, n + 1, s)) != hipSuccess) return e;
  return hipGetLastError();
}

hipError_t launch_knn_fill(const float* pos, const int32_t* graph_id, int n, int k, const int64_t* row_ptr,
                           int32_t* col_idx, hipStream_t s) {
  if (n == 0) return hipSuccess;
  k_knn_fill<<<n, 256, 0, s>>>(pos, graph_id, n, k, row_ptr, col_idx);
  return hipGetLastError();
}

}  // namespace e2f
