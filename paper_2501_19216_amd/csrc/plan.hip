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

#include <algorithm>
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
    // floor((2c + 1) span / (2 dim)): the product is below 2^43 and the
    // divisor at most 2048, so the double quotient (below 2^32, error below
    // 2^-21) truncates to the integer division's result, which is at least
    // 1/2048 from the next integer
    o[k] = (double)(g.lo[k] + (int64_t)((double)((2 * (int64_t)c[k] + 1) * g.span[k]) / (double)(2 * g.dim[k]))) /
           kGrid;
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

// The same harmonics from the dense per-degree table: the powers of x, y
// and z once, then per degree l the monomials x^ex y^ey z^(l-ex-ey) at fixed
// register positions and each component as their dot product with its row
// (the table's loads are uniform over the wave).  Every loop bound is a
// constant of L, so the whole evaluation unrolls into straight-line fp64
// multiply-adds.
template <int L, typename Sink>
__device__ __forceinline__ void sh_dense(const DevTables& t, double x, double y, double z, Sink sink) {
  double px[L + 1], py[L + 1], pz[L + 1];
  px[0] = py[0] = pz[0] = 1.0;
#pragma unroll
  for (int a = 1; a <= L; ++a) px[a] = px[a - 1] * x, py[a] = py[a - 1] * y, pz[a] = pz[a - 1] * z;
  const double* __restrict__ c = t.sh_dense;
#pragma unroll
  for (int l = 0; l <= L; ++l) {
    double mono[sh_monos(L)];
    int q = 0;
#pragma unroll
    for (int ex = 0; ex <= l; ++ex)
#pragma unroll
      for (int ey = 0; ey <= l - ex; ++ey) mono[q++] = px[ex] * py[ey] * pz[l - ex - ey];
    const int M = sh_monos(l), off = sh_dense_off(l);
#pragma unroll
    for (int m = 0; m < 2 * l + 1; ++m) {
      double acc = 0.0;
#pragma unroll
      for (int k = 0; k < M; ++k) acc = fma(c[off + m * M + k], mono[k], acc);
      sink(l * l + m, acc);
    }
  }
}

__global__ void k_plan_init(int* __restrict__ st, unsigned* __restrict__ dmin) {
  if (threadIdx.x < 3) st[threadIdx.x] = INT_MAX;
  else if (threadIdx.x < 6) st[threadIdx.x] = INT_MIN;
  else if (threadIdx.x < kStatsInts) st[threadIdx.x] = 0;
  if (threadIdx.x == 0 && dmin) *dmin = 0x7f800000u;  // +inf
}

// One atom's part of the bounding box: its grid coordinates (lo = hi), or
// the empty box and error bit 1 when a coordinate is not finite or outside
// +-16384 A (the atom is then kept out of the box); its graph id g (or -1
// without graphs), or error bit 2 when negative.
__device__ __forceinline__ void atom_box(const float x[3], int g, bool has_graph, int lo[3], int hi[3], int& gmax,
                                         int& bad) {
  lo[0] = lo[1] = lo[2] = INT_MAX;
  hi[0] = hi[1] = hi[2] = INT_MIN;
  gmax = 0;
  bad = 0;
  const bool ok = fabsf(x[0]) < 16384.0f && fabsf(x[1]) < 16384.0f && fabsf(x[2]) < 16384.0f;  // false for NaN
  if (ok) {
#pragma unroll
    for (int k = 0; k < 3; ++k) lo[k] = hi[k] = __float2int_rn(x[k] * 65536.0f);
  } else {
    bad |= 1;
  }
  if (has_graph) {
    if (g < 0) bad |= 2;
    else gmax = g;
  }
}

// Reduction of atom_box over a wave (every lane takes part).
__device__ __forceinline__ void wave_box(int lo[3], int hi[3], int& gmax, int& bad) {
  for (int o = 32; o > 0; o >>= 1) {
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      lo[k] = min(lo[k], __shfl_xor(lo[k], o));
      hi[k] = max(hi[k], __shfl_xor(hi[k], o));
    }
    gmax = max(gmax, __shfl_xor(gmax, o));
    bad |= __shfl_xor(bad, o);
  }
}

// The bounding box on the grid: a wave reduction, the workgroup's waves
// through LDS, then one atomic per workgroup and value.
__global__ __launch_bounds__(256) void k_plan_bbox(const float* __restrict__ pos, const int32_t* __restrict__ gid,
                                                   int n, int* __restrict__ st) {
  __shared__ int part[4][8];
  const int i = blockIdx.x * blockDim.x + threadIdx.x, wave = threadIdx.x >> 6;
  int lo[3] = {INT_MAX, INT_MAX, INT_MAX}, hi[3] = {INT_MIN, INT_MIN, INT_MIN}, gmax = 0, bad = 0;
  if (i < n) {
    const float x[3] = {pos[3 * i], pos[3 * i + 1], pos[3 * i + 2]};
    atom_box(x, gid ? gid[i] : 0, gid != nullptr, lo, hi, gmax, bad);
  }
  wave_box(lo, hi, gmax, bad);  // every lane takes part
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

// Shortest nonzero edge length (fp32 bits; positive floats order like their
// bits): each thread takes a grid-stride share of the edges, the minimum is
// reduced over the wave and the workgroup, and one atomic per workgroup
// meets the others (one per wave made a 1.6 M-edge graph wait on 25,000
// atomics to a single word).
constexpr int kDminThreads = 256, kDminMaxBlocks = 2048;
__global__ __launch_bounds__(kDminThreads) void k_plan_dmin(const float* __restrict__ pos,
                                                            const int32_t* __restrict__ rows,
                                                            const int32_t* __restrict__ col, int n, int64_t n_edges,
                                                            unsigned* __restrict__ dmin) {
  __shared__ unsigned part[kDminThreads / 64];
  unsigned v = 0x7f800000u;
  for (int64_t e = (int64_t)blockIdx.x * kDminThreads + threadIdx.x; e < n_edges;
       e += (int64_t)gridDim.x * kDminThreads) {
    const int i = clamp_node(rows[e], n), j = clamp_node(col[e], n);
    const float dx = pos[3 * i] - pos[3 * j], dy = pos[3 * i + 1] - pos[3 * j + 1], dz = pos[3 * i + 2] - pos[3 * j + 2];
    const float d = sqrtf(dx * dx + dy * dy + dz * dz);
    if (d > 0.0f && d < INFINITY) v = min(v, __float_as_uint(d));
  }
  for (int o = 32; o > 0; o >>= 1) v = min(v, (unsigned)__shfl_xor((int)v, o));
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned m = part[0];
    for (int w = 1; w < kDminThreads / 64; ++w) m = min(m, part[w]);
    if (m != 0x7f800000u) atomicMin(dmin, m);
  }
}

// The tile grid from the bounding box st (as k_plan_bbox leaves it).  The
// side is `side` grid units, or, when dmin is given, at most dmin_scale
// times the shortest edge; at least 1/64 A and at most 1024 tiles per axis
// (so at most 2^30 tiles).  The tiles of every graph share the grid: a tile
// only places the local origin of the receivers in it.
__device__ void grid_from_box(const int* st, const unsigned* __restrict__ dmin, double side, double dmin_scale,
                              TileGridDev& g) {
  if (dmin) {
    const float d = __uint_as_float(*dmin);
    if (d < INFINITY) side = fmin(side, dmin_scale * (double)d * kGrid);
  }
  side = fmax(side, kGrid / 64.0);
  int64_t ncell = 1;
  for (int k = 0; k < 3; ++k) {
    int lo = st[k], hi = st[3 + k];
    if (lo > hi) lo = hi = 0;  // no finite position
    g.lo[k] = lo;
    g.span[k] = (int64_t)hi - lo + 1;
    int64_t d = (int64_t)ceil((double)g.span[k] / side);
    d = d < 1 ? 1 : (d > 1024 ? 1024 : d);
    g.dim[k] = (int)d;
    ncell *= d;
  }
  g.ncell = (int)ncell;
  g.pad = 0;
}

__global__ void k_plan_grid(const int* __restrict__ st, const unsigned* __restrict__ dmin, double side,
                            double dmin_scale, TileGridDev* __restrict__ g) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  TileGridDev v;
  grid_from_box(st, dmin, side, dmin_scale, v);
  *g = v;
}

__device__ __forceinline__ int tile_axis(float x, const TileGridDev& g, int k) {
  const int64_t X = __float2int_rn(x * 65536.0f);
  const int64_t q = (int64_t)((double)(X - g.lo[k]) * (double)g.dim[k] / (double)g.span[k]);
  return (int)(q < 0 ? 0 : (q > g.dim[k] - 1 ? g.dim[k] - 1 : q));
}

// Tile of an atom at p (its cell of the grid) and its key in the receiver
// order: the graph in the high 32 bits, then the Morton index of 4 A cells
// of the box.
__device__ __forceinline__ void tile_key(const float p[3], int graph, const TileGridDev& g, int32_t& tile,
                                         uint64_t& key) {
  const int c0 = tile_axis(p[0], g, 0), c1 = tile_axis(p[1], g, 1), c2 = tile_axis(p[2], g, 2);
  tile = (c2 * g.dim[1] + c1) * g.dim[0] + c0;
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
  key = ((uint64_t)(uint32_t)graph << 32) | m;
}

__global__ void k_plan_tiles(const float* __restrict__ pos, const int32_t* __restrict__ gid, int n,
                             const TileGridDev* __restrict__ gp, int32_t* __restrict__ tile_of,
                             uint64_t* __restrict__ keys, int32_t* __restrict__ vals) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const TileGridDev g = *gp;
  const float p[3] = {pos[3 * i], pos[3 * i + 1], pos[3 * i + 2]};
  tile_key(p, gid ? max(gid[i], 0) : 0, g, tile_of[i], keys[i]);
  vals[i] = i;
}

// The whole plan of a small graph (n <= kPlanSmallMax) in one workgroup of
// T threads (8 T >= n): bounding box, grid, tiles and keys (each thread
// loads its atoms tid + u T, u < 8, once, all loads in flight together),
// then the receivers sorted by key with a least-significant-digit radix sort
// in LDS.  A slot is one 64-bit word, Morton index << 13 | atom index; the
// passes take four bits at a time, first of the Morton index, then (with
// graphs) of the graph id, read through the slot's atom index (graph ids are
// more significant, as in the key of the large path), and a pass is skipped
// where every atom has the same digit.  Each pass is stable: thread t holds
// slots 8t .. 8t+7, and the slot of its u-th item with digit d is the count
// of smaller digits, plus the count of d in threads below t, plus the count
// of d in its own items before u.  So the order is the one the stable radix
// sort of the large path gives.  The slots past n hold the largest key and
// follow every atom.  st and *gout are written as by k_plan_bbox and
// k_plan_grid.
// LDS: slots [9 NS/8] u64 (slot s at s + s/8, so the eight consecutive slots
// of a lane start 72 bytes after the previous lane's), per-thread offset
// rows [T][17] u32, per-wave digit counts and their prefix over the waves
// [33][8] u32.
constexpr int kPlanIpt = 8;
constexpr int kPlanIdxBits = 13;  // atom index bits of a slot: kPlanSmallMax <= 2^13
constexpr int kPlanThreads = 1024;

__device__ __forceinline__ int plan_slot(int s) { return s + s / kPlanIpt; }

__global__ __launch_bounds__(kPlanThreads) void k_plan_small(const float* __restrict__ pos,
                                                             const int32_t* __restrict__ gid, int n,
                                                             const unsigned* __restrict__ dmin, double side,
                                                             double dmin_scale, int* __restrict__ st,
                                                             TileGridDev* __restrict__ gout,
                                                             int32_t* __restrict__ tile_of,
                                                             int32_t* __restrict__ order) {
  extern __shared__ uint64_t slot[];
  __shared__ int box[kStatsInts];
  __shared__ unsigned bits[4];  // OR and AND of the Morton indices, then of the graph ids
  __shared__ TileGridDev g;
  const int T = blockDim.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, NW = T / 64, NS = kPlanIpt * T;
  unsigned* offs = (unsigned*)(slot + plan_slot(NS));
  unsigned* wcnt = offs + 17 * T;  // [wave][8]: the wave's digit counts; [16 + wave][8]: those of the waves below
  if (tid < kStatsInts) box[tid] = tid < 3 ? INT_MAX : (tid < 6 ? INT_MIN : 0);
  if (tid < 4) bits[tid] = (tid & 1) ? ~0u : 0u;
  float x[kPlanIpt][3];
  int gv[kPlanIpt];
#pragma unroll
  for (int u = 0; u < kPlanIpt; ++u) {
    const int i = tid + u * T;
    const int c = i < n ? i : 0;  // unconditional loads (n >= 1), masked below
    x[u][0] = pos[3 * c], x[u][1] = pos[3 * c + 1], x[u][2] = pos[3 * c + 2];
    gv[u] = gid ? gid[c] : 0;
  }
  int lo[3] = {INT_MAX, INT_MAX, INT_MAX}, hi[3] = {INT_MIN, INT_MIN, INT_MIN}, gmax = 0, bad = 0;
#pragma unroll
  for (int u = 0; u < kPlanIpt; ++u) {
    if (tid + u * T >= n) continue;
    int l[3], h[3], gm, b;
    atom_box(x[u], gv[u], gid != nullptr, l, h, gm, b);
#pragma unroll
    for (int k = 0; k < 3; ++k) lo[k] = min(lo[k], l[k]), hi[k] = max(hi[k], h[k]);
    gmax = max(gmax, gm);
    bad |= b;
  }
  __syncthreads();  // box initialised
  wave_box(lo, hi, gmax, bad);
  if (lane == 0) {
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      atomicMin(&box[k], lo[k]);
      atomicMax(&box[3 + k], hi[k]);
    }
    atomicMax(&box[6], gmax);
    atomicOr(&box[7], bad);
  }
  __syncthreads();
  if (tid == 0) {
    TileGridDev v;
    grid_from_box(box, dmin, side, dmin_scale, v);
    g = v;
    *gout = v;
  }
  if (tid < kStatsInts) st[tid] = box[tid];
  __syncthreads();
  unsigned mor = 0, mand = ~0u, gor = 0, gand = ~0u;
#pragma unroll
  for (int u = 0; u < kPlanIpt; ++u) {
    const int i = tid + u * T;
    uint64_t w = (uint64_t)0x3fffffff << kPlanIdxBits | (uint64_t)i;  // past n: the largest Morton index
    if (i < n) {
      int32_t t;
      uint64_t key;
      tile_key(x[u], gid ? max(gv[u], 0) : 0, g, t, key);
      tile_of[i] = t;
      const unsigned m = (unsigned)key, gr = (unsigned)(key >> 32);
      mor |= m, mand &= m, gor |= gr, gand &= gr;
      w = (uint64_t)m << kPlanIdxBits | (uint64_t)i;
    }
    slot[plan_slot(i)] = w;
  }
  for (int o = 32; o > 0; o >>= 1) {
    mor |= __shfl_xor(mor, o), mand &= __shfl_xor(mand, o);
    gor |= __shfl_xor(gor, o), gand &= __shfl_xor(gand, o);
  }
  if (lane == 0) {
    atomicOr(&bits[0], mor);
    atomicAnd(&bits[1], mand);
    atomicOr(&bits[2], gor);
    atomicAnd(&bits[3], gand);
  }
  __syncthreads();
  const unsigned mdiff = bits[0] ^ bits[1], gdiff = gid ? bits[2] ^ bits[3] : 0u;
  // passes: digit p < 8 of the Morton index, then digit p - 8 of the graph id
  for (int p = 0; p < 16; ++p) {
    const unsigned dm = p < 8 ? mdiff : gdiff;
    const int sh = 4 * (p & 7);
    if (((dm >> sh) & 15u) == 0) continue;  // every atom has this digit: the pass keeps the order
    uint64_t w[kPlanIpt];
    int d[kPlanIpt], r[kPlanIpt];
    uint64_t c64 = 0;  // the thread's count of each digit, four bits each (at most 8)
#pragma unroll
    for (int u = 0; u < kPlanIpt; ++u) w[u] = slot[plan_slot(kPlanIpt * tid + u)];
#pragma unroll
    for (int u = 0; u < kPlanIpt; ++u) {
      if (p < 8) {
        d[u] = (int)(w[u] >> (kPlanIdxBits + sh)) & 15;
      } else {
        const int i = (int)(w[u] & ((1u << kPlanIdxBits) - 1));
        const unsigned gr = i < n ? (unsigned)max(gid[i], 0) : 0x7fffffffu;
        d[u] = (int)(gr >> sh) & 15;
      }
    }
#pragma unroll
    for (int u = 0; u < kPlanIpt; ++u) {
      r[u] = (int)(c64 >> (4 * d[u])) & 15;
      c64 += (uint64_t)1 << (4 * d[u]);
    }
    // counts of digits 2q and 2q+1 in the halves of word q, then an
    // inclusive scan over the wave (totals stay below 2^16)
    unsigned cw[8], inc[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      cw[q] = (unsigned)((c64 >> (8 * q)) & 15) | (unsigned)((c64 >> (8 * q + 4)) & 15) << 16;
      inc[q] = cw[q];
    }
    for (int o = 1; o < 64; o <<= 1) {
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const unsigned y = __shfl_up(inc[q], o);
        if (lane >= o) inc[q] += y;
      }
    }
    if (lane == 63) {
#pragma unroll
      for (int q = 0; q < 8; ++q) wcnt[wave * 8 + q] = inc[q];
    }
    __syncthreads();  // every slot loaded (the scatter below overwrites them) and the wave counts stored
    if (tid < 8) {    // prefix of the counts over the waves; entry NW holds the totals
      unsigned c[kPlanThreads / 64], a = 0;
#pragma unroll
      for (int wv = 0; wv < kPlanThreads / 64; ++wv) c[wv] = wv < NW ? wcnt[wv * 8 + tid] : 0u;
#pragma unroll
      for (int wv = 0; wv < kPlanThreads / 64; ++wv) {
        if (wv < NW) wcnt[(16 + wv) * 8 + tid] = a;
        a += c[wv];
      }
      wcnt[(16 + NW) * 8 + tid] = a;
    }
    __syncthreads();
    unsigned start = 0;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int sq = 16 * (q & 1);
      const unsigned own = (inc[q >> 1] - cw[q >> 1] + wcnt[(16 + wave) * 8 + (q >> 1)]) >> sq & 0xffffu;
      offs[17 * tid + q] = start + own;
      start += wcnt[(16 + NW) * 8 + (q >> 1)] >> sq & 0xffffu;
    }
#pragma unroll
    for (int u = 0; u < kPlanIpt; ++u) slot[plan_slot((int)offs[17 * tid + d[u]] + r[u])] = w[u];
    __syncthreads();  // slots placed; the wave counts are free again
  }
  for (int i = tid; i < n; i += T) order[i] = (int32_t)(slot[plan_slot(i)] & ((1u << kPlanIdxBits) - 1));
}

// Solid harmonics about each receiver's tile centre, in one launch: blocks
// below eblocks take 256 consecutive edges each, the harmonics of the
// edge's sender in fp32, Re [E][nk] in CSR order (rows: the receiver of
// every edge; a thread per edge, whose values pass through LDS so that the
// workgroup stores its 256 rows as one contiguous block); the blocks after
// take 256 receivers each, their own harmonics in fp64, R [n][nk].
template <int L>
__global__ __launch_bounds__(256) void k_plan_sh(DevTables t, const float* __restrict__ pos,
                                                 const int32_t* __restrict__ rows, const int32_t* __restrict__ col,
                                                 int n, int64_t n_edges, int64_t eblocks,
                                                 const int32_t* __restrict__ tile_of,
                                                 const TileGridDev* __restrict__ gp, float* __restrict__ Re,
                                                 double* __restrict__ R) {
  constexpr int NK = (L + 1) * (L + 1), NKP = NK | 1;  // odd row stride: conflict-free LDS stores
  __shared__ float buf[256 * NKP];
  const TileGridDev g = *gp;
  double ox, oy, oz;
  if (blockIdx.x >= eblocks) {  // a receiver's own harmonics (uniform over the workgroup)
    const int i = (int)((blockIdx.x - eblocks) * 256) + threadIdx.x;
    if (i >= n) return;
    tile_centre(g, tile_of[i], ox, oy, oz);
    double* Ri = R + (size_t)i * NK;
    sh_dense<L>(t, (double)pos[3 * i] - ox, (double)pos[3 * i + 1] - oy, (double)pos[3 * i + 2] - oz,
                [&](int k, double v) { Ri[k] = v; });
    return;
  }
  const int64_t e0 = (int64_t)blockIdx.x * 256, e = e0 + threadIdx.x;
  const int cnt = (int)min((int64_t)256, n_edges - e0);
  if (e < n_edges) {
    const int i = clamp_node(rows[e], n), j = clamp_node(col[e], n);
    tile_centre(g, tile_of[i], ox, oy, oz);
    float* b = buf + threadIdx.x * NKP;
    sh_dense<L>(t, (double)pos[3 * j] - ox, (double)pos[3 * j + 1] - oy, (double)pos[3 * j + 2] - oz,
                [&](int k, double v) { b[k] = (float)v; });
  }
  __syncthreads();
  float* dst = Re + e0 * NK;
  for (int q = threadIdx.x; q < cnt * NK; q += 256) dst[q] = buf[(q / NK) * NKP + q % NK];
}

// The receiver of every edge (rows [E]), clamped like every CSR read: a
// wave per receiver, its lanes over the receiver's edges, in the blocks
// below rblocks; with alpha, the blocks after copy the attention weights
// [E][H] head-major, alpha_hm [H][E] (a thread per edge).
__global__ __launch_bounds__(256) void k_plan_edge_rows(const int64_t* __restrict__ row_ptr, int n, int64_t n_edges,
                                                        int32_t* __restrict__ rows, int64_t rblocks,
                                                        const float* __restrict__ alpha, int H,
                                                        float* __restrict__ alpha_hm) {
  if (blockIdx.x >= rblocks) {
    const int64_t e = (blockIdx.x - rblocks) * 256 + threadIdx.x;
    if (e >= n_edges) return;
    for (int h = 0; h < H; ++h) alpha_hm[(int64_t)h * n_edges + e] = alpha[e * H + h];
    return;
  }
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

hipError_t launch_plan_init(int* stats, unsigned* dmin, hipStream_t s) {
  k_plan_init<<<1, 64, 0, s>>>(stats, dmin);
  return hipGetLastError();
}

hipError_t launch_plan_small(const float* pos, const int32_t* graph_id, int n, const unsigned* dmin, double side,
                             double dmin_scale, int* stats, TileGridDev* grid, int32_t* tile_of, int32_t* order,
                             hipStream_t s) {
  if (n <= 0 || n > kPlanSmallMax) return hipErrorInvalidValue;
  static_assert(kPlanSmallMax <= kPlanIpt * kPlanThreads, "one workgroup holds the small plan");
  static_assert(kPlanSmallMax <= (1 << kPlanIdxBits), "a slot holds the atom index");
  static_assert(kPlanThreads / 64 + 17 <= 33, "wave counts and their prefix fit 33 rows of 8");
  // 16 T >= n, whole waves
  const int T = std::max(64, (n + 64 * kPlanIpt - 1) / (64 * kPlanIpt) * 64);
  const int ns = kPlanIpt * T;
  const size_t lds = sizeof(uint64_t) * (size_t)(ns + ns / kPlanIpt) + sizeof(unsigned) * (17 * (size_t)T + 33 * 8);
  if (lds > 32768)
    if (hipError_t e = hipFuncSetAttribute((const void*)k_plan_small, hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)lds);
        e != hipSuccess)
      return e;
  k_plan_small<<<1, T, lds, s>>>(pos, graph_id, n, dmin, side, dmin_scale, stats, grid, tile_of, order);
  return hipGetLastError();
}

hipError_t launch_plan_centre(const int* stats, double* origin, hipStream_t s) {
  k_plan_centre<<<1, 64, 0, s>>>(stats, origin);
  return hipGetLastError();
}

hipError_t launch_plan_dmin(const float* pos, const int32_t* rows, const int32_t* col, int n, int64_t n_edges,
                            unsigned* dmin, hipStream_t s) {
  const int64_t blocks = std::min<int64_t>((n_edges + kDminThreads - 1) / kDminThreads, kDminMaxBlocks);
  if (blocks > 0) k_plan_dmin<<<(unsigned)blocks, kDminThreads, 0, s>>>(pos, rows, col, n, n_edges, dmin);
  return hipGetLastError();
}

hipError_t launch_plan_grid(const int* stats, const unsigned* dmin, double side, double dmin_scale,
                            TileGridDev* grid, hipStream_t s) {
  k_plan_grid<<<1, 64, 0, s>>>(stats, dmin, side, dmin_scale, grid);
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
  const int64_t eblocks = (n_edges + 255) / 256, blocks = eblocks + (n + 255) / 256;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  switch (t.L) {
#define E2F_SH(LL)                                                                                             \
  case LL:                                                                                                     \
    k_plan_sh<LL><<<(unsigned)blocks, 256, 0, s>>>(t, pos, rows, col, n, n_edges, eblocks, tile_of, grid, Re, Rr); \
    break;
    E2F_SH(0) E2F_SH(1) E2F_SH(2) E2F_SH(3) E2F_SH(4) E2F_SH(5) E2F_SH(6)
#undef E2F_SH
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_plan_edge_rows(const int64_t* row_ptr, int n, int64_t n_edges, int32_t* rows, const float* alpha,
                                 int H, float* alpha_hm, hipStream_t s) {
  const int64_t rblocks = (n + 3) / 4, ablocks = alpha && alpha_hm ? (n_edges + 255) / 256 : 0;
  if (rblocks + ablocks > 0x7fffffff) return hipErrorInvalidValue;
  if (rblocks + ablocks > 0)
    k_plan_edge_rows<<<(unsigned)(rblocks + ablocks), 256, 0, s>>>(row_ptr, n, n_edges, rows, rblocks,
                                                                  ablocks ? alpha : nullptr, H, alpha_hm);
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
