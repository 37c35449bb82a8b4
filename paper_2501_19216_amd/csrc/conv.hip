// HIP kernels of the Wigner-6j convolution (Thm. 3.3, Alg. 1) and of the
// per-edge baseline (Def. 3.1) for gfx950.
//
// Data layout (HBM):
//   feat  [N][nk][C]        float32, nk = (L+1)^2
//   R     [items][nk]       float64 solid harmonics of p = r - origin
//   T     [pairs][dimT][C]  float32 j-side products, one row per (tile, sender)
//   S     [N][dimT][C]      float32 aggregated products per receiver
//   y/out [N][nk][C]        float32
// Channels are innermost everywhere, so every row gather in the aggregation
// and every per-node product reads contiguous, coalesced channel vectors.
// No floating-point atomics anywhere: each output element has one writer.
#include <hip/hip_runtime.h>
#include <hip/hip_bf16.h>
#include <hipcub/hipcub.hpp>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <type_traits>
#include <utility>

#include "e2f_launch.h"

namespace e2f {
namespace {

// ------------------------------------------------------------ solid harmonics
// Component k of R(p) as the explicit polynomial sum_t coef_t x^ex y^ey z^ez.
template <typename F>
__device__ __forceinline__ F sh_poly(const DevTables& t, int k, F x, F y, F z) {
  F acc = 0;
  for (int e = t.sh_ptr[k]; e < t.sh_ptr[k + 1]; ++e) {
    const int pw = t.sh_pow[e];
    F m = (F)t.sh_coef[e];
    for (int q = 0; q < (pw & 15); ++q) m *= x;
    for (int q = 0; q < ((pw >> 4) & 15); ++q) m *= y;
    for (int q = 0; q < ((pw >> 8) & 15); ++q) m *= z;
    acc += m;
  }
  return acc;
}

// Gradient of one solid harmonic from its monomials: d/dx of c x^a y^b z^e
// is c a x^(a-1) y^b z^e (no term when a = 0).
template <typename F>
__device__ __forceinline__ void sh_poly_grad(const DevTables& t, int k, F x, F y, F z, F& gx, F& gy, F& gz) {
  // per monomial one power loop per coordinate: b^(n-1) (1 for n = 0, where
  // the derivative's factor n is 0), then b^n = b^(n-1) b selected without a
  // branch
  auto pm1 = [](F b, int n) {
    F r = 1;
    for (int q = 1; q < n; ++q) r *= b;
    return r;
  };
  gx = 0, gy = 0, gz = 0;
  for (int e = t.sh_ptr[k]; e < t.sh_ptr[k + 1]; ++e) {
    const int pw = t.sh_pow[e];
    const int ex = pw & 15, ey = (pw >> 4) & 15, ez = (pw >> 8) & 15;
    const F c = (F)t.sh_coef[e];
    const F xm = pm1(x, ex), ym = pm1(y, ey), zm = pm1(z, ez);
    const F X = ex > 0 ? xm * x : (F)1, Y = ey > 0 ? ym * y : (F)1, Z = ez > 0 ? zm * z : (F)1;
    gx += c * (F)ex * xm * Y * Z;
    gy += c * (F)ey * X * ym * Z;
    gz += c * (F)ez * X * Y * zm;
  }
}

__global__ void k_sh(DevTables t, const float* __restrict__ pos, const int32_t* __restrict__ node_of,
                     const double* __restrict__ origins_d, const float* __restrict__ origins_f,
                     const int32_t* __restrict__ origin_id, int origin_mod, int n, double* __restrict__ out_d,
                     float* __restrict__ out_f) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= (int64_t)n * t.nk) return;
  const int item = (int)(gid / t.nk), k = (int)(gid % t.nk);
  const int node = node_of ? node_of[item] : item;
  double ox = 0.0, oy = 0.0, oz = 0.0;
  const int oi = origin_id ? origin_id[item] % origin_mod : 0;
  if (origins_d) {
    ox = origins_d[3 * oi];
    oy = origins_d[3 * oi + 1];
    oz = origins_d[3 * oi + 2];
  } else if (origins_f) {
    ox = origins_f[3 * oi];
    oy = origins_f[3 * oi + 1];
    oz = origins_f[3 * oi + 2];
  }
  const double v = sh_poly<double>(t, k, (double)pos[3 * node] - ox, (double)pos[3 * node + 1] - oy,
                                   (double)pos[3 * node + 2] - oz);
  if (out_d) out_d[gid] = v;
  else out_f[gid] = (float)v;
}

// ------------------------------------------------------------ j-side node TP
// T[item][r][c] = sum_al M[r][al] h_node^(a)[al][c] for the rows r of degree a,
// with the per-node matrix M[r][al] = sum_be C^{d de}_{a al, b be} R^(b)_be(p)
// built once per item in float64 (cost independent of C).  The product runs on
// v_mfma_f32_16x16x4f32: tiles of 16 rows of one degree a (so they share the
// K operand h^(a), 2a+1 values padded to a multiple of 4) by 16 channels.
// T is stored head-major, T[item][c / dh][r][c % dh] (dh = C: plain [r][c]).
typedef float v4f __attribute__((ext_vector_type(4)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

// Build one chunk of a per-node matrix into LDS from its schedule (see
// Schedule): coalesced, independent loads; each thread sums its slots.
__device__ __forceinline__ void run_schedule(const int* __restrict__ meta, const double* __restrict__ coef, int K,
                                             const double* Rl, float* dst) {
  // eight entries' loads issued before the first is used (the schedule sits
  // in L2: each batch costs one load latency), then their eight R values
  // read from LDS together; entries past K are zeros
  double acc = 0.0;
  const int t = threadIdx.x;
  for (int k0 = 0; k0 < K; k0 += 8) {
    int m[8];
    double c[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const bool ok = k0 + u < K;
      m[u] = ok ? meta[(k0 + u) * kSchedThreads + t] : 0;
      c[u] = ok ? coef[(k0 + u) * kSchedThreads + t] : 0.0;
    }
    double rv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) rv[u] = Rl[(m[u] >> 20) & 127];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      acc += c[u] * rv[u];
      if (m[u] < 0) {
        dst[m[u] & 0xfffff] = (float)acc;
        acc = 0.0;
      }
    }
  }
}

// Per item (a sender under its tile's origin): the whole per-node matrix
// M^(a)[row][al] = sum_b C^{d de}_{a al, b be} R^(b)_be(p) of every degree a
// is built once in LDS from one fixed schedule, stored transposed (al-major,
// rows padded to 16 mod 32 floats), and h is staged in LDS (rows padded the
// same way) when it fits.  The products then need no global load, so the T
// stores never hold up a wait:
//     T[row][c] = sum_al M^(a)[row][al] h^(a)[al][c]
// on v_mfma_f32_16x16x4f32 with A = h^T (16 channels x 4 al), B = M^T
// (4 al x 16 rows); each lane ends with 4 consecutive channels of one row,
// stored as one float4 (a wave writes 16 whole rows of 64 bytes per head).
// NW waves share one per-node matrix: the first kSchedThreads threads build it,
// all of them run the products (at high L the matrix leaves room for one
// workgroup per CU, so more waves per workgroup keep the stores in flight).
template <int L, int NW>
__global__ __launch_bounds__(NW * 64) void k_node_tp(DevTables t, const double* __restrict__ R,
                                                 const int32_t* __restrict__ node_of, const float* __restrict__ feat,
                                                 int C, int dh, int hs, float* __restrict__ T) {
  constexpr int NK = (L + 1) * (L + 1);
  extern __shared__ float sm[];  // M (t.tp_mo[L+1] floats), then h if staged (hs > 0)
  __shared__ double Rl[NK];
  const int item = blockIdx.x;
  const int node = node_of ? node_of[item] : item;
  if (threadIdx.x < NK) Rl[threadIdx.x] = R[(size_t)item * NK + threadIdx.x];
  const int msize = t.tp_mo[L + 1];
  float* Mt = sm;
  const float* h = feat + (size_t)node * NK * C;
  int hstride = C;
  if (hs > 0) {
    float* hl = sm + ((msize + 3) & ~3);
    const int c4 = C / 4;
    for (int q = threadIdx.x; q < NK * c4; q += blockDim.x)
      ((float4*)hl)[(q / c4) * (hs / 4) + q % c4] = ((const float4*)h)[q];
    h = hl;
    hstride = hs;
  }
  for (int q = threadIdx.x; q < msize; q += blockDim.x) Mt[q] = 0.0f;
  __syncthreads();
  if (threadIdx.x < kSchedThreads) run_schedule(t.tp_meta, t.tp_coef, t.tp_k[0], Rl, Mt);
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int l16 = lane & 15, k4 = lane >> 4;
  const int NT = (C + 15) / 16;
  float* Tp = T + (size_t)item * t.dimT * C;
#pragma unroll
  for (int a = 0; a <= L; ++a) {
    const int KA = 2 * a + 1, KP = (KA + 3) & ~3;
    const int ra0 = t.a_row_start[a], rows = t.a_row_start[a + 1] - ra0;
    const int rs = t.tp_rs[a];
    const float* Ma = Mt + t.tp_mo[a];
    const int nrt = (rows + 15) / 16;
    for (int task = wave; task < nrt * NT; task += NW) {
      const int rt = task / NT, nt = task % NT;
      const int ca = nt * 16 + l16;  // A operand channel
      const float* hc = h + (ca < C ? ca : 0);
      v4f acc = {0.f, 0.f, 0.f, 0.f};
      for (int ks = 0; ks < KP / 4; ++ks) {
        const int k = 4 * ks + k4, kc = min(k, KA - 1);  // k >= KA: weight 0
        const float hv = hc[(a * a + kc) * hstride];
        const float av = k < KA ? hv : 0.0f;
        const float bv = Ma[kc * rs + rt * 16 + l16];
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc, 0, 0, 0);
      }
      // acc[v] = T[row rt*16 + l16][channel nt*16 + 4*k4 + v]
      const int row = rt * 16 + l16, c0 = nt * 16 + 4 * k4;
      if (row < rows && c0 < C)
        *(float4*)(Tp + (size_t)(c0 / dh) * t.dimT * dh + (size_t)(ra0 + row) * dh + c0 % dh) =
            make_float4(acc[0], acc[1], acc[2], acc[3]);
    }
  }
}

// ------------------------------------------------------------ receiver blocks
// Receivers are cut into blocks of G consecutive entries of the spatial
// order.  For each block the plan lists the union U_b of the T rows its
// edges read (sorted, unique) and, for every edge, the position of its T row
// in U_b.  Rows are sorted by sender and the pairs of a tile are numbered by
// ascending sender, so every receiver's edges are in ascending U_b position.
constexpr int kUnionMax = 8192;  // G * (largest degree) must fit

__global__ void k_block_edges(const int64_t* __restrict__ row_ptr, const int32_t* __restrict__ order, int n, int G,
                              int nblk, int32_t* __restrict__ blk_count) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= nblk) return;
  int64_t c = 0;
  for (int r = b * G; r < min(n, (b + 1) * G); ++r) c += row_ptr[order[r] + 1] - row_ptr[order[r]];
  blk_count[b] = (int32_t)c;
}

__global__ __launch_bounds__(256) void k_block_union(const int64_t* __restrict__ row_ptr,
                                                     const int32_t* __restrict__ col_pair,
                                                     const int32_t* __restrict__ order, int n, int G,
                                                     const int32_t* __restrict__ blk_off,
                                                     int32_t* __restrict__ uni, int32_t* __restrict__ ucount,
                                                     int32_t* __restrict__ edge_slot) {
  extern __shared__ int32_t ush[];
  int32_t* keys = ush;               // [kUnionMax]
  int32_t* ukeys = ush + kUnionMax;  // [kUnionMax]
  __shared__ int32_t off[65];
  __shared__ int32_t part[256];
  const int b = blockIdx.x;
  const int r0 = b * G, nr = min(G, n - r0);
  if (threadIdx.x == 0) {
    int32_t o = 0;
    for (int r = 0; r < nr; ++r) {
      off[r] = o;
      const int i = order[r0 + r];
      o += (int32_t)(row_ptr[i + 1] - row_ptr[i]);
    }
    off[nr] = o;
  }
  __syncthreads();
  const int total = off[nr];  // <= kUnionMax, guaranteed by the host's choice of G
  int p2 = 1;
  while (p2 < total) p2 <<= 1;
  for (int r = 0; r < nr; ++r) {
    const int64_t rs = row_ptr[order[r0 + r]];
    for (int t = threadIdx.x; t < off[r + 1] - off[r]; t += blockDim.x) keys[off[r] + t] = col_pair[rs + t];
  }
  for (int k = total + threadIdx.x; k < p2; k += blockDim.x) keys[k] = 0x7fffffff;
  __syncthreads();
  // bitonic sort of keys[0, p2)
  for (int size = 2; size <= p2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int k = threadIdx.x; k < p2 / 2; k += blockDim.x) {
        const int lo = 2 * k - (k & (stride - 1));
        const int hi = lo + stride;
        const bool up = (lo & size) == 0;
        const int32_t x = keys[lo], y = keys[hi];
        if ((x > y) == up) {
          keys[lo] = y;
          keys[hi] = x;
        }
      }
      __syncthreads();
    }
  }
  // unique: each thread owns a contiguous run of `per` sorted keys
  const int per = (total + blockDim.x - 1) / blockDim.x;
  const int k0 = threadIdx.x * per, k1 = min(total, k0 + per);
  int cnt = 0;
  for (int k = k0; k < k1; ++k) cnt += (k == 0 || keys[k] != keys[k - 1]);
  part[threadIdx.x] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t s = 0;
    for (int t = 0; t < (int)blockDim.x; ++t) {
      const int32_t v = part[t];
      part[t] = s;
      s += v;
    }
    ucount[b] = s;
    off[64] = s;
  }
  __syncthreads();
  int w = part[threadIdx.x];
  for (int k = k0; k < k1; ++k)
    if (k == 0 || keys[k] != keys[k - 1]) {
      ukeys[w] = keys[k];
      uni[blk_off[b] + w] = keys[k];
      ++w;
    }
  __syncthreads();
  const int nu = off[64];
  // position of every edge's T row in the union
  for (int r = 0; r < nr; ++r) {
    const int64_t rs = row_ptr[order[r0 + r]];
    for (int t = threadIdx.x; t < off[r + 1] - off[r]; t += blockDim.x) {
      const int32_t key = col_pair[rs + t];
      int lo = 0, hi = nu;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (ukeys[mid] < key) lo = mid + 1;
        else hi = mid;
      }
      edge_slot[rs + t] = lo;
    }
  }
}

// ------------------------------------------------------------ aggregation
// S[i][q] = sum_{e in row i} alpha[e][head(q)] T[col_pair[e]][q].
//
// MFMA form.  For a block of 16 spatially consecutive receivers and the union
// U_b of their T rows, and for one head h:
//     S_b,h [16 x cols] = A_b,h [16 x |U_b|] . T_{U_b},h [|U_b| x cols],
// where A_b,h[r][u] is the attention weight of the edge (receiver r, union row
// u) or 0; each workgroup assembles A_b,h in LDS from alpha and edge_slot.  v_mfma_f32_16x16x4f32 takes A as 16 receivers x 4 union rows and
// B as 4 union rows x 16 columns of head h, so every T element loaded from
// L2 is used by all 16 receivers inside the matrix core instead of being
// gathered once per edge.  The columns of head h are enumerated as
// m = delta*dh + t (t < dh) and cut into groups of 16; T and S are stored
// head-major ([row][head][delta][t]), so one head's columns are contiguous
// and a wave's 8 groups read 512 contiguous bytes of each T row.  A wave owns
// kAggGroups groups of one head of one block and walks U_b four rows at a time.
// Accumulation order is fixed (deterministic).
constexpr int kXcds = 8;
constexpr int kPiece = 512;  // union rows staged in LDS at a time

template <int NQ, int NS, int WV>
__global__ __launch_bounds__(64 * WV) void k_aggregate_mfma(const float* __restrict__ T, int pair_base,
                                                        const int32_t* __restrict__ uni,
                                                        const int32_t* __restrict__ blk_off,
                                                        const int32_t* __restrict__ ucount,
                                                        const int64_t* __restrict__ row_ptr,
                                                        const int32_t* __restrict__ order,
                                                        const int32_t* __restrict__ edge_slot,
                                                        const float* __restrict__ alpha_hm, int64_t n_edges,
                                                        int n, int nblk, int bpx, int by_task,
                                                        int ntg, int ntgw, int dimT, int C, int dh, int H,
                                                        float* __restrict__ S) {
  __shared__ int64_t ubl[kPiece];     // float4 offset of each union row of the piece in T
  __shared__ float4 Al4[kPiece * 4];  // Al[slot][receiver]: A operand of head h
  const float* Al = (const float*)Al4;
  // workgroup = (block b, column task); the blocks of one XCD are contiguous
  // in space and the column tasks are the slow index, so the workgroups in
  // flight on an XCD share T rows through its L2
  const int bid = blockIdx.x;
  const int xcd = bid % kXcds, local = bid / kXcds;
  const int b = by_task ? local % nblk : xcd * bpx + local % bpx;
  const int wtask = by_task ? (local / nblk) * kXcds + xcd : local / bpx;
  if (b >= nblk || wtask >= H * ntgw) return;  // uniform over the workgroup
  const int h = wtask / ntgw;
  const float* ah = alpha_hm ? alpha_hm + (int64_t)h * n_edges : nullptr;  // head h's weights, by edge
  const int tg = (wtask % ntgw) * WV + (int)(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int j = lane & 15, k = lane >> 4;
  const int64_t W4 = (int64_t)dimT * C / 4;
  const int hcols = dimT * dh;
  // MFMA group g = 4q + u reads column m = (tg*NQ + q)*64 + 4j + u of head h,
  // so lane j loads the float4 at 4j covering its four groups.  Columns past
  // the head's end load column 0 of the head instead (never stored).
  constexpr int kAggGroups = 4 * NQ;
  int c4[NQ];
  bool cvalid[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int m0 = (tg * NQ + q) * 64 + 4 * j;
    cvalid[q] = tg < ntg && m0 < hcols;
    c4[q] = (h * hcols + (cvalid[q] ? m0 : 0)) / 4;
  }
  v4f acc[kAggGroups];
#pragma unroll
  for (int g = 0; g < kAggGroups; ++g) acc[g] = (v4f){0.f, 0.f, 0.f, 0.f};
  const int nu = ucount[b];
  const int32_t* ub = uni + blk_off[b];
  // the A operand is built by threads 0..255, 16 per receiver
  const int rr = threadIdx.x >> 4, rl = threadIdx.x & 15;
  int64_t e0 = 0, e1 = 0;
  if (rr < 16 && b * 16 + rr < n) {
    const int i = order[b * 16 + rr];
    e0 = row_ptr[i];
    e1 = row_ptr[i + 1];
  }
  // senders are ascending in every row, so a receiver's edges reach the union
  // slots in ascending order: each thread keeps a cursor over its edges
  // (stride 16) and every piece continues from it
  int64_t ecur = e0 + rl;
  const float4* T4 = (const float4*)T;
  const bool active = tg < ntg;  // uniform over the wave
  // Union rows 4 at a time (lane row k); rows past the piece take weight 0
  // and re-read its last row.  NS register stages: while the MFMAs of one
  // step run, the loads of the next NS-1 steps are in flight.
  float4 bst[NS][NQ];
  float ast[NS];
  auto load = [&](int s0, int np, float4* bv, float& a) {
    const int sl = s0 + k, sc = min(sl, np - 1);  // clamped reads, no branch
    const float av = Al[sc * 16 + j];
    a = sl < np ? av : 0.0f;
    const float4* trow = T4 + ubl[sc];
#pragma unroll
    for (int q = 0; q < NQ; ++q) bv[q] = trow[c4[q]];
  };
  auto mma = [&](const float4* bv, float a) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      acc[4 * q + 0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, bv[q].x, acc[4 * q + 0], 0, 0, 0);
      acc[4 * q + 1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, bv[q].y, acc[4 * q + 1], 0, 0, 0);
      acc[4 * q + 2] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, bv[q].z, acc[4 * q + 2], 0, 0, 0);
      acc[4 * q + 3] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, bv[q].w, acc[4 * q + 3], 0, 0, 0);
    }
  };
  for (int p0 = 0; p0 < nu; p0 += kPiece) {
    const int np = min(nu - p0, kPiece);
    // staging: the piece's 64-bit T row offsets and A = the attention
    // weights of the block's edges whose union slot falls in the piece,
    // scattered into a zeroed LDS tile.  All global loads of a batch are
    // issued (clamped indexes, no branch) before the first store.
    {
      constexpr int kNT = 64 * WV, kU = kPiece / kNT;
      static_assert(kPiece % kNT == 0, "piece must split evenly over the threads");
      constexpr int kEB = 4;  // edges per thread per batch (16 threads per receiver)
      __syncthreads();
      const int t = threadIdx.x;
      int32_t uu[kU];
#pragma unroll
      for (int u = 0; u < kU; ++u) uu[u] = ub[p0 + min(t + kNT * u, np - 1)];
      int sl[kEB];
      float av[kEB];
      auto load_edges = [&](int64_t eb) {
#pragma unroll
        for (int u = 0; u < kEB; ++u) {
          const int64_t ec = min(eb + 16 * u, e1 - 1);
          sl[u] = edge_slot[ec] - p0;
          av[u] = ah ? ah[ec] : 1.0f;
        }
      };
      if (ecur < e1) load_edges(ecur);
#pragma unroll
      for (int u = 0; u < kU; ++u) ubl[t + kNT * u] = (int64_t)(uu[u] - pair_base) * W4;
      for (int q = t; q < 4 * np; q += kNT) Al4[q] = make_float4(0.f, 0.f, 0.f, 0.f);
      __syncthreads();
      // earlier pieces took every slot below p0; the first edge past this
      // piece is where the next one starts (the loop bound does not depend on
      // loaded data, so the next batch's loads need not wait for this one's)
      float* Alw = (float*)Al4;
      int64_t nxt = e1;
      for (int64_t eb = ecur; eb < e1; eb += 16 * kEB) {
        if (eb != ecur) load_edges(eb);
#pragma unroll
        for (int u = 0; u < kEB; ++u) {
          const int64_t ev = eb + 16 * u;
          if (ev < e1) {
            if (sl[u] >= np) nxt = min(nxt, ev);
            else if (sl[u] >= 0) Alw[sl[u] * 16 + rr] = av[u];
          }
        }
      }
      ecur = nxt;
      __syncthreads();
    }
    if (!active) continue;  // no barrier below
    // Steps of 4 rows, NS per iteration (the last iteration is padded with
    // zero-weight steps); the body has no branch, so each wait covers only
    // the oldest stage, and sched_barrier keeps the scheduler from sinking
    // a prefetch to its use.
#pragma unroll
    for (int st = 0; st < NS - 1; ++st) load(4 * st, np, bst[st], ast[st]);
    const int nit = (np + 4 * NS - 1) / (4 * NS);
    for (int it = 0; it < nit; ++it) {
#pragma unroll
      for (int st = 0; st < NS; ++st) {
        const int ls = (st + NS - 1) % NS;
        load(4 * (it * NS + st + NS - 1), np, bst[ls], ast[ls]);
        __builtin_amdgcn_sched_barrier(0);
        mma(bst[st], ast[st]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  if (!active) return;
  // acc[4q+u][v] = S[receiver 4k+v of the block][column (tg*NQ+q)*64 + 4j + u]
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int r = b * 16 + 4 * k + v;
    if (r >= n) continue;
    float4* srow = (float4*)S + (int64_t)order[r] * W4;  // S rows by receiver
#pragma unroll
    for (int q = 0; q < NQ; ++q)
      if (cvalid[q]) srow[c4[q]] = make_float4(acc[4 * q][v], acc[4 * q + 1][v], acc[4 * q + 2][v], acc[4 * q + 3][v]);
  }
}

// Fallback for receivers with more than 512 neighbours: one wave per
// receiver and 1 KB column chunk, rows read from L2 (receivers in spatial
// order, XCD-contiguous mapping).
constexpr int kAggRecv = 4;
constexpr int kAggChunk4 = 64;

__global__ __launch_bounds__(64 * kAggRecv) void k_aggregate_rows(const float4* __restrict__ T, int pair_base,
                                                                  const int64_t* __restrict__ row_ptr,
                                                                  const int32_t* __restrict__ col_pair,
                                                                  const float* __restrict__ alpha,
                                                                  const int32_t* __restrict__ order, int n, int W4,
                                                                  int nchunk, int ngroups, int gpx, int C, int dh,
                                                                  int H, float4* __restrict__ S) {
  const int bid = blockIdx.x;
  const int xcd = bid % kXcds, local = bid / kXcds;
  const int group = xcd * gpx + local % gpx;
  const int chunk = local / gpx;
  if (group >= ngroups || chunk >= nchunk) return;
  const int r = group * kAggRecv + (int)(threadIdx.x >> 6);
  const int q = chunk * kAggChunk4 + (int)(threadIdx.x & 63);
  if (r >= n || q >= W4) return;
  const int i = order[r];
  const int head = (int)(((int64_t)q * 4) / ((int64_t)W4 * 4 / H));  // head-major rows
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  const int64_t e0 = row_ptr[i], e1 = row_ptr[i + 1];
#pragma unroll 4
  for (int64_t e = e0; e < e1; ++e) {
    const float a = alpha ? alpha[e * H + head] : 1.0f;
    const float4 v = T[(size_t)(col_pair[e] - pair_base) * W4 + q];
    acc.x += a * v.x;
    acc.y += a * v.y;
    acc.z += a * v.z;
    acc.w += a * v.w;
  }
  S[(size_t)i * W4 + q] = acc;  // S rows by receiver
}

// ------------------------------------------------------------ aggregation of the node products
// The j-side product is linear, so the aggregation can run on the uncoupled
// products and the coupling follow per receiver:
//   S_i^(a,b,d)[de][c] = sum_j alpha_ij [h_j^(a) (x) R^(b)(p_j)]^(d)_de[c]
//                      = sum_{al,be} C^{d de}_{a al, b be} G_i[(b,be)][(a,al)][c],
//   G_i[be][q][c]      = sum_j alpha_ij,h(c) R_be(p_j) h_j[q][c].
// Per (receiver, head) G_i is one dense product on v_mfma_f32_16x16x4f32:
// M = the (L+1)^2 components be of R (padded to 16), K = the receiver's
// neighbours four at a time, N = the (L+1)^2 * dh columns (q, t) of head h,
// with A = alpha * R staged in LDS per chunk of edges and B = the neighbours'
// features read from L2.  There are no structural zeros (only the padding of
// M), and the operands are the features h (not one T row per tile and
// sender).  G then sits in LDS and the coupling to S uses the node product's
// CG tables (row -> slots al -> entries (be, C)); S is written head-major, as
// the recouple reads it.
constexpr int kOuterEdges = 128;  // edges staged per chunk
// register pipeline of the products: kOuterStages - 1 steps ahead (3 measured
// faster than 4 and 5: 6.47, 6.52, 6.62 ms at 20k atoms, L = 4)
constexpr int kOuterStages = 3;

// Staging of one chunk of ne <= EC edges from edge c0 for the products:
// Al[nb * AS + be] = alpha_e R_be(p_j) of the chunk's edge nb for the 4
// ceil(ne / 4) rows the steps read (zeros past ne and for be >= NK), jl[nb]
// = its sender for nb < EC (edge c0 past ne, and 0 for an index outside
// [0, n_nodes): no read leaves the caller's buffers), times jmul (a row
// stride; the product is stored as unsigned 32 bits).  alpha_h is the head's
// row of the head-major weights (NULL: all ones).  Consecutive threads take
// consecutive components of one edge (contiguous R loads, conflict-free LDS
// stores); four values per thread in flight, loads before stores.  Needs
// blockDim.x >= EC; the caller synchronises before and after.
template <int NK, int MP, int AS, int EC>
__device__ __forceinline__ void stage_chunk(const float* __restrict__ Re, const float* __restrict__ alpha_h,
                                            const int32_t* __restrict__ col, int64_t c0, int ne, int n_nodes,
                                            float* __restrict__ Al, int* __restrict__ jl, unsigned jmul = 1) {
  const int nsl = 4 * ((ne + 3) / 4) * MP;
  int jv = threadIdx.x < EC ? col[c0 + ((int)threadIdx.x < ne ? threadIdx.x : 0)] : 0;
  jv = (unsigned)jv < (unsigned)n_nodes ? jv : 0;
  for (int base = threadIdx.x; base < nsl; base += 4 * blockDim.x) {
    float av[4], rv[4];
    bool okv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = base + u * blockDim.x, nb = idx / MP, be = idx % MP;
      okv[u] = idx < nsl && nb < ne && be < NK;
      const int64_t e = c0 + (nb < ne ? nb : 0);
      av[u] = alpha_h ? alpha_h[e] : 1.0f;
      rv[u] = Re[(size_t)e * NK + (be < NK ? be : 0)];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = base + u * blockDim.x;
      if (idx < nsl) Al[(idx / MP) * AS + idx % MP] = okv[u] ? av[u] * rv[u] : 0.0f;
    }
  }
  if (threadIdx.x < EC) jl[threadIdx.x] = (int)((unsigned)jv * jmul);
}

// The j-side coupling of one receiver's G (in LDS, rows of GS floats) into
// its S rows of one head (Sr, rows of dh floats), from a thread-balanced
// schedule: group g walks its entries k*cgroups + g, four channels per
// thread (tq), CB entries at a time (their schedule reads, then their G
// reads, then the sums; past ck: entry 0 with coefficient 0, never the last
// of a row).  Packed entries (PK) hold a 9-bit row and the index of their
// coefficient in coef; otherwise coef runs beside meta and the row has 12
// bits.  CB = 8 above L = 4, where the schedule (120 KB at L = 6) is read
// from L2 by every receiver and head: half the round trips (234.4 vs 237.7
// ms at 200k atoms, L = 6); 4 below (no gain there).
template <bool PK, int CB>
__device__ __forceinline__ void couple_rows(const int* __restrict__ meta, const float* __restrict__ coef, int ck,
                                            int cgroups, int g, int tq, const float* G, int GS, int dh,
                                            float* __restrict__ Sr) {
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int k0 = 0; k0 < ck; k0 += CB) {
    int m[CB];
    float c[CB];
    float4 gv[CB];
#pragma unroll
    for (int u = 0; u < CB; ++u) {
      const bool ok = k0 + u < ck;
      m[u] = ok ? meta[(k0 + u) * cgroups + g] : 0;
      if (!PK) c[u] = ok ? coef[(k0 + u) * cgroups + g] : 0.0f;
    }
    if (PK) {
#pragma unroll
      for (int u = 0; u < CB; ++u) {
        const float cv = coef[(m[u] >> 21) & 1023];
        c[u] = k0 + u < ck ? cv : 0.0f;
      }
    }
#pragma unroll
    for (int u = 0; u < CB; ++u) gv[u] = *(const float4*)(G + ((m[u] >> 6) & 63) * GS + (m[u] & 63) * dh + 4 * tq);
#pragma unroll
    for (int u = 0; u < CB; ++u) {
      v.x += c[u] * gv[u].x, v.y += c[u] * gv[u].y, v.z += c[u] * gv[u].z, v.w += c[u] * gv[u].w;
      if (m[u] < 0) {
        *(float4*)(Sr + ((m[u] >> 12) & (PK ? 511 : 4095)) * dh + 4 * tq) = v;
        v = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
  }
}

template <int L, int NTWM, int LB>
__global__ __launch_bounds__(LB) void k_outer_agg(DevTables t, const float* __restrict__ Re,
                                                    const int64_t* __restrict__ row_ptr,
                                                    const int32_t* __restrict__ col,
                                                    const float* __restrict__ alpha_hm, int64_t n_edges,
                                                    const float* __restrict__ feat, const int32_t* __restrict__ order,
                                                    const int* __restrict__ cmeta, const float* __restrict__ ccoef,
                                                    const int* __restrict__ pmeta, const float* __restrict__ ptab,
                                                    int ntab, int ck, int cgroups, int work_floats, int n, int nrx,
                                                    int rpw, int C, int H, int hdiv, int n_nodes,
                                                    float* __restrict__ S) {
  constexpr int NK = (L + 1) * (L + 1), MT = (NK + 15) / 16, MP = 16 * MT;
  constexpr int EC = kOuterEdges;
  extern __shared__ float sm[];
  // rows of AS = MP + 16 floats: the four rows an MFMA step reads (one per
  // lane group k4) start 48 banks apart, so the operand reads are
  // conflict-free
  constexpr int AS = MP + 16;
  float* Al = sm;                   // [EC][AS]: Al[nb*AS + be] = alpha * R_be of the chunk's edge nb
  int* jl = (int*)(sm + EC * AS);   // [EC]: sender of the edge (clamped past the chunk)
  float* G = sm;                    // [NK][GS], after the products (reuses the staging space)
  // the coupling schedule, staged once in LDS after the work space when
  // work_floats > 0 (else read from global memory): packed entries and their
  // coefficient table when ntab > 0, else entries and coefficients
  if (work_floats > 0 && ntab > 0) {
    for (int q = threadIdx.x; q < ck * cgroups; q += blockDim.x) ((int*)(sm + work_floats))[q] = pmeta[q];
    for (int q = threadIdx.x; q < ntab; q += blockDim.x) sm[work_floats + ck * cgroups + q] = ptab[q];
  } else if (work_floats > 0) {
    for (int q = threadIdx.x; q < ck * cgroups; q += blockDim.x) {
      ((int*)(sm + work_floats))[q] = cmeta[q];
      sm[work_floats + ck * cgroups + q] = ccoef[q];
    }
  }
  const int dh = C / H, NC = NK * dh, NT = (NC + 15) / 16, GS = NC + 4;
  // workgroup -> (rpw consecutive receivers, head h); the receivers of one
  // XCD are contiguous in the spatial order and their heads consecutive
  const int bid = blockIdx.x, xcd = bid % 8, local = bid / 8;
  const int h = local % H, rfirst = xcd * nrx + (local / H) * rpw;
  const int rlast = min(min(rfirst + rpw, (xcd + 1) * nrx), n);  // uniform over the workgroup
  const int NW = blockDim.x >> 6, wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int l16 = lane & 15, k4 = lane >> 4;
  // the wave's column blocks cb = wave + NW u (u < NTWM/4) of 64 columns:
  // tile w of block u holds the columns cb*64 + 4 l16 + w, so lane l16 reads
  // the four consecutive columns 4 l16 .. 4 l16 + 3 (one q, as 4 | dh) as
  // one float4
  constexpr int NB = NTWM / 4;
  int off[NB];
  bool cok[NB], tlive[NB];
#pragma unroll
  for (int u = 0; u < NB; ++u) {
    const int cb = wave + NW * u, nn = cb * 64 + 4 * l16;
    tlive[u] = __builtin_amdgcn_readfirstlane(cb * 64 < NC ? 1 : 0) != 0;  // uniform over the wave
    cok[u] = nn < NC;
    const int q = cok[u] ? nn / dh : 0, tt = cok[u] ? nn % dh : 0;
    off[u] = q * C + h * dh + tt;
  }
  (void)NT;
  for (int r = rfirst; r < rlast; ++r) {
  const int i = order[r];
  v4f acc[MT][NTWM];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int w = 0; w < NTWM; ++w) acc[mt][w] = (v4f){0.f, 0.f, 0.f, 0.f};
  // row bounds clamped to [0, E] (a malformed graph cannot move a read
  // outside the caller's buffers)
  const int64_t rb0 = row_ptr[i], rb1 = row_ptr[i + 1];
  const int64_t e0 = rb0 < 0 ? 0 : (rb0 > n_edges ? n_edges : rb0);
  const int64_t e1 = rb1 < e0 ? e0 : (rb1 > n_edges ? n_edges : rb1);
  __syncthreads();  // the previous receiver's coupling has read G (and the schedule is staged)
  for (int64_t c0 = e0; c0 < e1; c0 += EC) {
    const int ne = (int)min((int64_t)EC, e1 - c0);
    __syncthreads();
    stage_chunk<NK, MP, AS, EC>(Re, alpha_hm ? alpha_hm + (int64_t)(h / hdiv) * n_edges : nullptr, col, c0, ne,
                                n_nodes, Al, jl);
    __syncthreads();
    const int ns = (ne + 3) / 4;
    // three-stage pipeline: the features of steps st+1, st+2 are loaded
    // while the MFMAs of step st run
    // Each stage holds both operands of a step: A (the lane's two rows of
    // alpha R from LDS) and B (the features), so no wait precedes the MFMAs.
    // Rows 4 st + k4 < 4 ns <= EC hold alpha R (zeros past ne); steps past ns
    // read row EC - 1 and a valid sender and are never multiplied.  Columns
    // past NC read column 0 (valid) and their results are never stored.
    float aq[kOuterStages][MT];
    float4 bq[kOuterStages][NB];
    auto loadb = [&](int st, float* a, float4* b) {
      const int nb = min(4 * st + k4, EC - 1);
      const float* hj = feat + (size_t)jl[nb] * NK * C;
#pragma unroll
      for (int u = 0; u < NB; ++u) b[u] = *(const float4*)(hj + off[u]);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) a[mt] = Al[nb * AS + mt * 16 + l16];
    };
    auto mma = [&](const float* a, const float4* b) {
#pragma unroll
      for (int u = 0; u < NB; ++u) {
        if (!tlive[u]) continue;  // scalar: uniform over the wave
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          acc[mt][4 * u + 0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[mt], b[u].x, acc[mt][4 * u + 0], 0, 0, 0);
          acc[mt][4 * u + 1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[mt], b[u].y, acc[mt][4 * u + 1], 0, 0, 0);
          acc[mt][4 * u + 2] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[mt], b[u].z, acc[mt][4 * u + 2], 0, 0, 0);
          acc[mt][4 * u + 3] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[mt], b[u].w, acc[mt][4 * u + 3], 0, 0, 0);
        }
      }
    };
#pragma unroll
    for (int u = 0; u + 1 < kOuterStages; ++u) loadb(u, aq[u], bq[u]);
    for (int st = 0; st < ns; st += kOuterStages) {
#pragma unroll
      for (int u = 0; u < kOuterStages; ++u) {
        const int w = (u + kOuterStages - 1) % kOuterStages;
        loadb(st + u + kOuterStages - 1, aq[w], bq[w]);
        __builtin_amdgcn_sched_barrier(0);
        if (u == 0 || st + u < ns) mma(aq[u], bq[u]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  __syncthreads();  // the staging space becomes G
  // acc[mt][4u + w][v] = G[be = mt*16 + 4 k4 + v][n = cb*64 + 4 l16 + w]:
  // one float4 per (block, tile row, v)
#pragma unroll
  for (int u = 0; u < NB; ++u) {
    if (!cok[u]) continue;
    const int nn = (wave + NW * u) * 64 + 4 * l16;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int be = mt * 16 + 4 * k4 + v;
        if (be < NK)
          *(float4*)(G + be * GS + nn) =
              make_float4(acc[mt][4 * u][v], acc[mt][4 * u + 1][v], acc[mt][4 * u + 2][v], acc[mt][4 * u + 3][v]);
      }
  }
  __syncthreads();
  // j-side coupling: S[row][tt] = sum over the row's entries of C * G[be][q dh + tt]
  float* Sr = S + (size_t)r * t.dimT * C + (size_t)h * t.dimT * dh;
  const int dq = dh >> 2, g = threadIdx.x / dq, tq = threadIdx.x % dq;
  constexpr int CB = L > 4 ? 8 : 4;  // schedule entries per batch
  if (g < cgroups) {
    if (work_floats > 0 && ntab > 0)
      couple_rows<true, CB>((const int*)(sm + work_floats), sm + work_floats + ck * cgroups, ck, cgroups, g, tq, G,
                            GS, dh, Sr);
    else if (work_floats > 0)
      couple_rows<false, CB>((const int*)(sm + work_floats), sm + work_floats + ck * cgroups, ck, cgroups, g, tq,
                             G, GS, dh, Sr);
    else
      couple_rows<false, CB>(cmeta, ccoef, ck, cgroups, g, tq, G, GS, dh, Sr);
  }
  }  // receivers of the workgroup
}

// ------------------------------------------------------------ fused recouple
// Up to L = 4 with heads of 16 channels the recouple is applied where G is
// made: per receiver the matrix F_i = Q_i CG (the j-side coupling composed
// with the i-side recouple, built once per receiver by k_fuse_build) takes
// the aggregated uncoupled products straight to the output,
//     y_i[k][h*16 + t] = sum_{be, q} F_i[k][be, q] G_i^h[be][q][t],
// so neither the coupled S_i nor a second kernel's read of it exists.

// F_i = sum_x R_x(p_i) K_x in float64, rounded once to float: a workgroup
// builds kFuseRecv receivers' rows (the receivers order[r0 ..] of the slice,
// row r0 + b), each thread a set of positions; position p sums its entries
// fidx/fcoef[fptr[p] .. fptr[p+1]).
constexpr int kFuseRecv = 16;
__global__ __launch_bounds__(256) void k_fuse_build(const int* __restrict__ fptr, const int* __restrict__ fidx,
                                                    const double* __restrict__ fcoef, int np, int nk,
                                                    const double* __restrict__ R, const int32_t* __restrict__ order,
                                                    int nb, float* __restrict__ F) {
  __shared__ double Rl[kFuseRecv][(kFuseMaxL + 1) * (kFuseMaxL + 1)];
  const int r0 = blockIdx.x * kFuseRecv;
  const int nr = min(kFuseRecv, nb - r0);
  for (int q = threadIdx.x; q < kFuseRecv * nk; q += blockDim.x) {
    const int b = q / nk, x = q % nk;
    Rl[b][x] = b < nr ? R[(size_t)order[r0 + b] * nk + x] : 0.0;
  }
  __syncthreads();
  for (int p = threadIdx.x; p < np; p += blockDim.x) {
    double acc[kFuseRecv];
#pragma unroll
    for (int b = 0; b < kFuseRecv; ++b) acc[b] = 0.0;
    const int e1 = fptr[p + 1];
    for (int e = fptr[p]; e < e1; ++e) {
      const double c = fcoef[e];
      const int x = fidx[e];
#pragma unroll
      for (int b = 0; b < kFuseRecv; ++b) acc[b] += c * Rl[b][x];
    }
#pragma unroll
    for (int b = 0; b < kFuseRecv; ++b)
      if (b < nr) F[(size_t)(r0 + b) * np + p] = (float)acc[b];
  }
}


// x = hi + mid + lo exactly, each part a bfloat16 rounded to nearest even
// (8 + 8 + 8 significant bits hold a float's 24), returned as bit patterns.
// The products of the split operands that reach 2^-24 relative (hi hi,
// hi mid, mid hi, hi lo, mid mid, lo hi) are exact in float and summed in
// float by the matrix cores, so six bf16 products stand in for one float
// product within float rounding.
__device__ __forceinline__ void split_bf16x3(float x, unsigned& hi, unsigned& mid, unsigned& lo) {
  const __bf16 h = (__bf16)x;
  const float r = x - (float)h;
  const __bf16 m = (__bf16)r;
  const __bf16 l = (__bf16)(r - (float)m);
  hi = __builtin_bit_cast(unsigned short, h);
  mid = __builtin_bit_cast(unsigned short, m);
  lo = __builtin_bit_cast(unsigned short, l);
}

// The fused aggregation's groups of components, one product wave each: NG =
// ceil(NK / 4) groups of at most four, as even as possible (NK = 25: 4, 4, 4,
// 4, 3, 3, 3), so that two product waves sharing a SIMD hold at most 7 of the
// 25 component tiles; group g holds the components fuse_g0(NK, g) ..
// fuse_g0(NK, g) + fuse_gn(NK, g) - 1.
__host__ __device__ constexpr int fuse_gn(int nk, int g) {
  return nk / ((nk + 3) / 4) + (g < nk % ((nk + 3) / 4) ? 1 : 0);
}
__host__ __device__ constexpr int fuse_g0(int nk, int g) {
  return g * (nk / ((nk + 3) / 4)) + (g < nk % ((nk + 3) / 4) ? g : nk % ((nk + 3) / 4));
}
static_assert(fuse_g0(25, 6) + fuse_gn(25, 6) == 25 && fuse_gn(25, 3) == 4 && fuse_gn(25, 4) == 3,
              "groups of 25 components: 4, 4, 4, 4, 3, 3, 3");
static_assert(fuse_g0(16, 3) == 12 && fuse_gn(16, 3) == 4 && fuse_g0(9, 2) == 6 && fuse_gn(1, 0) == 1,
              "groups of 16, 9 and 1 components");

// The features in the order of the fused aggregation's B operand, each value
// split into three bfloat16 parts: per node and head of 16 channels, the
// groups of components above (slot i of group g: component fuse_g0(NK, g) +
// i, zero from fuse_gn(NK, g) on), each group [t][i] (t the channel in the
// head): a uint4 of the four components' hi | mid << 16
// and, in the second array (same index), a uint2 of their lo parts
// (components 0, 1 in the first word, low half first).  Lane t of a wave
// reads its group's four components with one 16-byte and one 8-byte load; a
// group of 16 lanes reads 256 + 128 contiguous bytes.
__global__ void k_feat_qmajor3(const float* __restrict__ feat, int n, int nk, int C, int ng,
                               uint4* __restrict__ hm, uint2* __restrict__ lo) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // (node, head, group, t)
  const int H = C / 16;
  if (q >= (int64_t)n * H * ng * 16) return;
  const int t = (int)(q % 16);
  const int64_t r = q / 16;
  const int g = (int)(r % ng), h = (int)(r / ng % H);
  const int64_t j = r / ((int64_t)ng * H);
  const float* src = feat + (size_t)j * nk * C + h * 16 + t;
  unsigned a[4], b[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    unsigned x, y, z;
    split_bf16x3(i < fuse_gn(nk, g) ? src[(size_t)(fuse_g0(nk, g) + i) * C] : 0.0f, x, y, z);
    a[i] = x | y << 16;
    b[i] = z;
  }
  hm[q] = make_uint4(a[0], a[1], a[2], a[3]);
  lo[q] = make_uint2(b[0] | b[1] << 16, b[2] | b[3] << 16);
}

// The aggregation with the recouple applied in registers.  Work split as in
// k_outer_agg (a workgroup: rpw consecutive receivers of one head h of 16
// channels), but tile w of wave v holds the 16 channels t = l16 of one
// component q = fuse_g0(NK, v) + w, so that after the products the accumulator element
// s of a lane (l16, k4), G[16 mt + 4 k4 + s][q][l16], is exactly the B
// operand of K step s of F_i G when the K index of that step is ordered as
// be = 16 mt + 4 k4 + s; F_i is stored in the matching order.  Each wave sums
// its components' share of y (rows 16 rt + 4 k4 + v, channel l16); the
// shares meet in LDS and one pass stores the head's 16 channels of y_i.
//
// The workgroup walks its receivers' chunks of up to kOuterEdges edges (an
// isolated receiver is one empty chunk).  Waves 0 .. NG-1 multiply (wave v:
// the fuse_gn(NK, v) components of group v); the last wave stages: while the others multiply
// chunk k from one LDS buffer it loads chunk k+1 (alpha, R of the edges, the
// senders) and writes alpha R and the senders' offsets into the other, so
// the products never wait for a chunk's loads.  One barrier per chunk (two
// more after a receiver's last chunk, for the shares of y, which reuse the
// finished buffer).
// The K rows of G and F (KR of them; the plain layer: KR = NK, row be the
// component be of R(p_j)) may stack several filter degrees of alpha / D^f:
// segment s of the K rows (from sg.start[s]) holds the components be =
// row - start of R(p_j) weighted by alpha_hm[s], so that one gather of the
// senders serves several degrees.
// register pipeline of the fused products: kFuseStages - 1 steps ahead
constexpr int kFuseStages = 3;
constexpr int kFuseRows = kOuterEdges + 4 * (2 * kFuseStages - 2);  // staging rows with the prefetch padding

template <int L, int LB, int KR>
__global__ __launch_bounds__(LB) void k_outer_fused(const float* __restrict__ Re, const int64_t* __restrict__ row_ptr,
                                                    const int32_t* __restrict__ col, FusedSegs sg, int64_t n_edges,
                                                    const uint4* __restrict__ fhm, const uint2* __restrict__ flo,
                                                    const int32_t* __restrict__ order, const float* __restrict__ F,
                                                    int n, int nrx, int rpw, int C, int H, int hdiv, int n_nodes,
                                                    bool accumulate, float* __restrict__ y) {
  constexpr int NK = (L + 1) * (L + 1), MT = (NK + 15) / 16, MP = 16 * MT;  // rows k of y and F
  constexpr int MK = (KR + 15) / 16, MPK = 16 * MK;                         // K rows of G and F
  constexpr int EC = kOuterEdges;
  // staging row stride in words: two words per component (a 64-bit read per
  // lane), odd rows rotated by 16 components where 2 MP is a multiple of 64,
  // so rows 4 st + k4 of one step alternate between the two halves of the
  // banks
  constexpr int AS = 2 * MPK;
  constexpr int ROT = (2 * MPK) % 64 == 0 ? 16 : 0;
  constexpr int QB = fuse_qblock(NK, KR), FS = fuse_stride(NK, KR);
  constexpr int NG = (NK + 3) / 4;  // groups of at most four components (fuse_gn): one product wave each
  // rows EC .. SR-1 of a buffer are padding (zero weights, sender offset 0):
  // the last iteration of the step loop starts at a step st <= ns - 1 and
  // loads up to step st + 2 (kFuseStages - 1) ahead, i.e. rows up to
  // 4 (ns - 1 + 2 (kFuseStages - 1)) + 3 <= EC + 8 kFuseStages - 9
  constexpr int SR = kFuseRows, SB = SR * AS;
  static_assert(SR - EC >= 8 * kFuseStages - 8, "padding rows must cover the prefetch past a full chunk");
  static_assert(NG * MP * 16 <= SB, "the shares of y must fit one staging buffer");
  constexpr int RPI = 64 / MPK;           // rows the staging wave covers per pass (lane: K row lane % MPK)
  constexpr int ITER = EC / RPI;          // passes over a full chunk
  extern __shared__ float sm[];
  float* Alb = sm;                        // [2][SR][AS] alpha R of the chunk's edges, split (zero past its rows)
  int* job = (int*)(sm + 2 * SB);         // [2][SR] the senders' offsets in the re-laid features
  float* sa = sm + 2 * SB + 2 * SR;       // [sg.n][EC] the staging wave's copy of the chunk's weights
  const int bid = blockIdx.x, xcd = bid % 8, local = bid / 8;
  const int h = local % H, rfirst = xcd * nrx + (local / H) * rpw;
  const int rlast = min(min(rfirst + rpw, (xcd + 1) * nrx), n);  // uniform over the workgroup
  if (rfirst >= rlast) return;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int l16 = lane & 15, k4 = lane >> 4;
  const bool stager = wave == NG;  // uniform over the wave
  // a product wave's live tiles (the components q0 .. q0 + nl - 1 of its
  // group) and the lane's entry of a sender: its wave's group, channel t = l16
  const int nl = stager ? 0 : __builtin_amdgcn_readfirstlane(fuse_gn(NK, wave));
  const int q0 = stager ? 0 : fuse_g0(NK, wave);
  const unsigned fstride = (unsigned)(H * NG * 16);
  const unsigned foff = (unsigned)((h * NG + min(wave, NG - 1)) * 16 + l16);
  for (int q = threadIdx.x; q < 2 * (SR - EC) * AS; q += blockDim.x) {
    const int b = q / ((SR - EC) * AS);
    Alb[b * SB + EC * AS + q % ((SR - EC) * AS)] = 0.0f;
  }
  for (int q = threadIdx.x; q < 2 * (SR - EC); q += blockDim.x) job[(q / (SR - EC)) * SR + EC + q % (SR - EC)] = 0;
  // edge range of receiver row r (clamped to [0, E]: a malformed graph
  // cannot move a read outside the caller's buffers)
  auto bounds = [&](int r, int64_t& e0, int64_t& e1) {
    const int i = order[r];
    const int64_t rb0 = row_ptr[i], rb1 = row_ptr[i + 1];
    e0 = rb0 < 0 ? 0 : (rb0 > n_edges ? n_edges : rb0);
    e1 = rb1 < e0 ? e0 : (rb1 > n_edges ? n_edges : rb1);
  };
  // the staging wave: chunk [c0, c0 + ne) into buffer b.  Every sender
  // offset below EC is written (0 past ne); the weight rows read by the
  // chunk's steps (4 ceil(ne / 4)) are written whole, zero past ne and in
  // the columns NK .. MP-1.  Lane: component be = lane % MP of rows
  // rs + RPI it; the R values load in batches of BT rows per lane, the next
  // batch in flight while the current one is stored (clamped addresses, so
  // the loads are unconditional; an empty chunk loads none).
  auto stage = [&](int64_t c0, int ne, int b) {
    float* Al = Alb + b * SB;
    int* jo = job + b * SR;
    if (ne == 0) {  // an isolated receiver: zero weights, sender offsets 0
#pragma unroll
      for (int u = 0; u < EC / 64; ++u) {
#pragma unroll
        for (int sgm = 0; sgm < kFusedSegs; ++sgm)
          if (sgm < sg.n) sa[sgm * EC + lane + 64 * u] = 0.0f;
        jo[lane + 64 * u] = 0;
      }
      return;
    }
    // unconditional loads (the compiler can then keep every batch in flight):
    // the weights and harmonics of edges c0 .. c0 + EC - 1 lie inside their
    // arrays, which carry kEdgePad rows of padding past the last edge (a
    // missing weight array reads the harmonics instead); the caller's senders
    // are read at a clamped index.  Rows past ne are masked by selects.
    float av[kFusedSegs][EC / 64];
    int jv[EC / 64];
#pragma unroll
    for (int u = 0; u < EC / 64; ++u) {
      const int nb = lane + 64 * u;
#pragma unroll
      for (int sgm = 0; sgm < kFusedSegs; ++sgm) {
        if (sgm >= sg.n) break;
        const float* ah = sg.alpha_hm[sgm] ? sg.alpha_hm[sgm] + (int64_t)(h / hdiv) * n_edges : nullptr;
        const float a = (ah ? ah : Re)[c0 + nb];
        av[sgm][u] = nb < ne ? (ah ? a : 1.0f) : 0.0f;
      }
      const int j = col[c0 + min(nb, ne - 1)];
      jv[u] = nb < ne && (unsigned)j < (unsigned)n_nodes ? j : 0;
    }
#pragma unroll
    for (int u = 0; u < EC / 64; ++u) {
#pragma unroll
      for (int sgm = 0; sgm < kFusedSegs; ++sgm)
        if (sgm < sg.n) sa[sgm * EC + lane + 64 * u] = av[sgm][u];
      jo[lane + 64 * u] = (int)((unsigned)jv[u] * fstride);
    }
    __builtin_amdgcn_wave_barrier();
    const int nrow = 4 * ((ne + 3) / 4);
    // the lane's position p = lane % MPK of the row holds K row kr (the K
    // order of F: within tile p / 16, row 16 (p / 16) + j at 4 (j / ks) +
    // j % ks), or nothing (zeros) where no row takes it; K row kr of segment
    // sgm is the harmonics' component kr - sg.start[sgm] with that segment's
    // weights
    const int p = lane % MPK, rs = lane / MPK;
    const int pt = p / 16, pk4 = (p % 16) / 4, ps = p % 4, ks = fuse_ks(KR, pt);
    const int pj = pk4 * ks + ps;
    const bool bok = pt * 16 < KR && ps < ks && pj < fuse_rows(KR, pt);
    const int kr = 16 * pt + pj;
    int seg = 0, s0 = 0;
#pragma unroll
    for (int sgm = 1; sgm < kFusedSegs; ++sgm)
      if (sgm < sg.n && kr >= sg.start[sgm]) {
        seg = sgm;
        s0 = sg.start[sgm];
      }
    const int be = bok ? kr - s0 : 0;  // the harmonics' component (< NK: checked by the launcher)
    const float* wsrc = sa + seg * EC;
    // the lane's rows rs + RPI (BT bt + k): one base per batch, immediate
    // offsets within it
    const float* src = Re + (size_t)(c0 + rs) * NK + be;
    constexpr int BT = 16, NBT = ITER / BT;
    static_assert(ITER % BT == 0, "batches must cover a chunk");
    static_assert(kEdgePad >= EC, "the per-edge arrays must be padded by a chunk");
    float cur[BT], nxt[BT];
    auto load = [&](int bt, float* d) {
      const float* sb = src + (size_t)bt * BT * RPI * NK;
#pragma unroll
      for (int k = 0; k < BT; ++k) d[k] = sb[k * RPI * NK];
    };
    load(0, cur);
#pragma unroll 1
    for (int bt = 0; bt < NBT && bt * BT * RPI < nrow; ++bt) {
      const bool more_rows = bt + 1 < NBT && (bt + 1) * BT * RPI < nrow;
      if (more_rows) load(bt + 1, nxt);
#pragma unroll
      for (int k = 0; k < BT; ++k) {
        const int nb = (bt * BT + k) * RPI + rs;
        const float w = cur[k] * wsrc[nb];
        const float v = bok && nb < ne ? w : 0.0f;
        if (nb < nrow) {
          // A of the split products: words hi | mid << 16 and hi | lo << 16
          unsigned hi, mid, lo;
          split_bf16x3(v, hi, mid, lo);
          ((uint2*)(Al + nb * AS))[(p + (nb & 1) * ROT) % MPK] = make_uint2(hi | mid << 16, hi | lo << 16);
        }
      }
      if (more_rows) {
#pragma unroll
        for (int k = 0; k < BT; ++k) cur[k] = nxt[k];
      }
    }
  };
  int r = rfirst;
  int64_t e0, e1;
  bounds(r, e0, e1);
  int64_t c0 = e0;
  if (stager) stage(c0, (int)min((int64_t)EC, e1 - c0), 0);
  __syncthreads();
  v4f acc[MK][4];
#pragma unroll
  for (int mt = 0; mt < MK; ++mt)
#pragma unroll
    for (int w = 0; w < 4; ++w) acc[mt][w] = (v4f){0.f, 0.f, 0.f, 0.f};
  for (int kb = 0;; kb ^= 1) {
    const int ne = (int)min((int64_t)EC, e1 - c0);  // 0 for an isolated receiver
    const bool last = c0 + EC >= e1;                 // the receiver's last chunk (uniform)
    int rn = r;
    int64_t c0n = c0 + EC, e0n = e0, e1n = e1;
    if (last) {
      rn = r + 1;
      if (rn < rlast) {
        bounds(rn, e0n, e1n);
        c0n = e0n;
      }
    }
    const bool more = rn < rlast;
    if (stager) {
      if (more) stage(c0n, (int)min((int64_t)EC, e1n - c0n), kb ^ 1);
    } else {
      const float* Al = Alb + kb * SB;
      const int* jo = job + kb * SR;
      const int ns = (ne + 3) / 4;
      // pipeline of the products: the operands of steps st+1, st+2 are
      // loaded while the MFMAs of step st run; steps past ns read rows of
      // zeros or stale weights with valid senders and are never multiplied.
      // NL (the wave's live tiles) is a constant of each copy of the loop.
      // The products are split: K of one v_mfma_f32_16x16x32_bf16 is 4
      // edges (k4) x 8 slots, six of them the cross products of the parts,
      //   A = {hi|mid, hi|lo, hi|mid, 0}, B = {hi|mid, mid|hi, lo|hi, 0}
      // (A from the staging words, B from the lane's uint4 / uint2 of the
      // sender), so a step is two loads, MT 64-bit LDS reads, two ALU
      // operations per tile and NL MT MFMAs of half the fp32 cost.
      auto products = [&](auto nlc) {
        constexpr int NL = decltype(nlc)::value;
        uint2 aq[kFuseStages][MK];
        uint4 bh[kFuseStages];
        uint2 bl[kFuseStages];
        auto loadb = [&](int st, uint2* a, uint4& h4, uint2& l2) {
          const int nb = min(4 * st + k4, SR - 1);  // < SR without the clamp (see SR)
          const unsigned o = (unsigned)jo[nb] + foff;
          h4 = fhm[o];
          l2 = flo[o];
          const uint2* row = (const uint2*)(Al + nb * AS);
#pragma unroll
          for (int mt = 0; mt < MK; ++mt) a[mt] = row[(mt * 16 + l16 + (nb & 1) * ROT) % MPK];
        };
        auto mma = [&](const uint2* a, const uint4& h4, const uint2& l2) {
          const unsigned hw[4] = {h4.x, h4.y, h4.z, h4.w};
          const unsigned lw[4] = {l2.x & 0xffffu, l2.x >> 16, l2.y & 0xffffu, l2.y >> 16};
#pragma unroll
          for (int w = 0; w < NL; ++w) {
            const v8bf bv =
                __builtin_bit_cast(v8bf, (v4u){hw[w], (hw[w] >> 16) | (hw[w] << 16), lw[w] | (hw[w] << 16), 0u});
#pragma unroll
            for (int mt = 0; mt < MK; ++mt) {
              const v8bf av = __builtin_bit_cast(v8bf, (v4u){a[mt].x, a[mt].y, a[mt].x, 0u});
              acc[mt][w] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc[mt][w], 0, 0, 0);
            }
          }
        };
#pragma unroll
        for (int u = 0; u + 1 < kFuseStages; ++u) loadb(u, aq[u], bh[u], bl[u]);
        for (int st = 0; st < ns; st += kFuseStages) {
#pragma unroll
          for (int u = 0; u < kFuseStages; ++u) {
            const int w = (u + kFuseStages - 1) % kFuseStages;
            loadb(st + u + kFuseStages - 1, aq[w], bh[w], bl[w]);
            __builtin_amdgcn_sched_barrier(0);
            if (u == 0 || st + u < ns) mma(aq[u], bh[u], bl[u]);
            __builtin_amdgcn_sched_barrier(0);
          }
        }
      };
      if (nl == 4) products(std::integral_constant<int, 4>{});
      else if (nl == 3) products(std::integral_constant<int, 3>{});
      else if (nl == 2) products(std::integral_constant<int, 2>{});
      else if (nl == 1) products(std::integral_constant<int, 1>{});
    }
    if (last) {
      // this wave's share of y_i: A = F_i (rows k, K = the K rows in the step
      // order above, zero past KR), B = the accumulators.  The F loads are
      // unconditional (lanes past a sub-block's rows or K values read a
      // valid element and take zero), so the wait counts stay exact; the
      // next component's values load while this one's MFMAs run.
      const float* Fr = F + (size_t)r * FS;
      v4f ya[MT];
#pragma unroll
      for (int rt = 0; rt < MT; ++rt) ya[rt] = (v4f){0.f, 0.f, 0.f, 0.f};
      auto recouple = [&](auto nlc) {
        constexpr int NL = decltype(nlc)::value;
        float4 fv[2][MT][MK];
        auto loadf = [&](int w, float4 (*f)[MK]) {
          const int q = q0 + w;  // < NK for w < NL
#pragma unroll
          for (int rt = 0; rt < MT; ++rt)
#pragma unroll
            for (int mt = 0; mt < MK; ++mt) {
              // (a 0/1 factor rather than a select: a value every lane uses
              // keeps the compiler from predicating the load)
              const bool ok = l16 < fuse_rows(NK, rt) && k4 < fuse_kc(KR, mt);
              const float z = ok ? 1.0f : 0.0f;
              const float4 v = *(const float4*)(Fr + q * QB + fuse_blk(NK, KR, rt, mt) +
                                                (ok ? (k4 * fuse_rows(NK, rt) + l16) * 4 : 0));
              f[rt][mt] = make_float4(v.x * z, v.y * z, v.z * z, v.w * z);
            }
        };
        // (scheduling barriers keep the next component's loads ahead of
        // this one's MFMAs; without them the loads sink to their first use
        // and every F block waits out a full L2 round trip)
        loadf(0, fv[0]);
#pragma unroll
        for (int w = 0; w < NL; ++w) {
          if (w + 1 < NL) loadf(w + 1, fv[(w + 1) & 1]);
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int mt = 0; mt < MK; ++mt)
#pragma unroll
            for (int rt = 0; rt < MT; ++rt) {
              // K steps s >= fuse_ks(KR, mt) hold no K row (zero F and G):
              // skipped (mt is a constant of the unrolled loop)
              const float4 f = fv[w & 1][rt][mt];
              ya[rt] = __builtin_amdgcn_mfma_f32_16x16x4f32(f.x, acc[mt][w][0], ya[rt], 0, 0, 0);
              if (fuse_ks(KR, mt) > 1)
                ya[rt] = __builtin_amdgcn_mfma_f32_16x16x4f32(f.y, acc[mt][w][1], ya[rt], 0, 0, 0);
              if (fuse_ks(KR, mt) > 2)
                ya[rt] = __builtin_amdgcn_mfma_f32_16x16x4f32(f.z, acc[mt][w][2], ya[rt], 0, 0, 0);
              if (fuse_ks(KR, mt) > 3)
                ya[rt] = __builtin_amdgcn_mfma_f32_16x16x4f32(f.w, acc[mt][w][3], ya[rt], 0, 0, 0);
            }
          __builtin_amdgcn_sched_barrier(0);
        }
      };
      if (nl == 4) recouple(std::integral_constant<int, 4>{});
      else if (nl == 3) recouple(std::integral_constant<int, 3>{});
      else if (nl == 2) recouple(std::integral_constant<int, 2>{});
      else if (nl == 1) recouple(std::integral_constant<int, 1>{});
      __syncthreads();  // every product wave is done with buffer kb: it takes the shares of y
      float* yp = Alb + kb * SB;  // [NG][MP][16]
      if (!stager) {
#pragma unroll
        for (int rt = 0; rt < MT; ++rt)
#pragma unroll
          for (int v = 0; v < 4; ++v) yp[(wave * MP + 16 * rt + 4 * k4 + v) * 16 + l16] = ya[rt][v];
      }
      __syncthreads();
      const int i = order[r];
      for (int idx = threadIdx.x; idx < NK * 16; idx += blockDim.x) {
        const int row = idx >> 4, t = idx & 15;
        float sum = 0.0f;
        for (int wv = 0; wv < NG; ++wv) sum += yp[(wv * MP + row) * 16 + t];
        float* yo = y + ((size_t)i * NK + row) * C + h * 16 + t;
        *yo = accumulate ? *yo + sum : sum;  // (accumulate: the sum over the filter degrees of alpha / D^f)
      }
#pragma unroll
      for (int mt = 0; mt < MK; ++mt)
#pragma unroll
        for (int w = 0; w < 4; ++w) acc[mt][w] = (v4f){0.f, 0.f, 0.f, 0.f};
    }
    if (!more) break;
    __syncthreads();  // buffer kb ^ 1 is staged; buffer kb (and the shares of y) is free
    r = rn;
    c0 = c0n;
    e0 = e0n;
    e1 = e1n;
  }
}

// ------------------------------------------------------------ i-side recouple
// y_i[k][c] = sum_r Q_i[k][r] S_i[r][c] over the T rows r, with the per-node
// matrix Q_i[(o,m)][(a,b,d,de)] = sum_u K(a,b,d,u,o) sum_ga C^{o m}_{u ga, d de}
// R^(u)_ga(p_i) summed in float64 into an fp32 LDS tile (rc_rows T rows at a
// time, from a fixed schedule) and the product on v_mfma_f32_16x16x4f32: 16
// output rows x 16 channels per tile, S_i read from HBM exactly once.

template <int L, int NTW>
__global__ __launch_bounds__(256) void k_recouple(DevTables t, const double* __restrict__ R,
                                                  const float* __restrict__ S, int64_t s_stride,
                                                  const int32_t* __restrict__ order, int C, int dh,
                                                  bool accumulate, float* __restrict__ y) {
  constexpr int NK = (L + 1) * (L + 1);
  constexpr int MT = (NK + 15) / 16;  // NTW: channel tiles per wave and pass
  constexpr int QS = rc_qstride(NK);
  constexpr int RR = rc_rows(NK);
  constexpr int ST = 8;                // 4-row steps per pipeline stage
  extern __shared__ float Qt[];        // Qt[r][k], RR rows of QS floats
  __shared__ double Rl[NK];
  const int i = order[blockIdx.x];  // S row blockIdx.x belongs to receiver i
  if (threadIdx.x < NK) Rl[threadIdx.x] = R[(size_t)i * NK + threadIdx.x];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int j = lane & 15, k4 = lane >> 4;
  const int dimT = t.dimT;
  const float* Si = S + (size_t)blockIdx.x * s_stride;  // s_stride 0: one S row shared by all
  const int NT = (C + 15) / 16;
  for (int ns = 0; ns < NT; ns += 4 * NTW) {
    // B operand: lane (j, k4) reads channel c(q) of row 4s + k4; channels
    // past C read channel 0 (never stored)
    const float* sb[NTW];
    bool cok[NTW];
#pragma unroll
    for (int q = 0; q < NTW; ++q) {
      const int c = (ns + wave + 4 * q) * 16 + j;
      cok[q] = c < C;
      const int cc = cok[q] ? c : 0;
      sb[q] = Si + (size_t)(cc / dh) * dimT * dh + cc % dh;
    }
    v4f acc[NTW][MT];
#pragma unroll
    for (int q = 0; q < NTW; ++q)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[q][mt] = (v4f){0.f, 0.f, 0.f, 0.f};
    for (int r0 = 0; r0 < dimT; r0 += RR) {
      const int rc = min(RR, dimT - r0);
      __syncthreads();
      for (int q = threadIdx.x; q < RR * QS; q += blockDim.x) Qt[q] = 0.0f;
      // Stages of ST steps in pairs; rows past the chunk read its last row
      // and take Q = 0.  No branch in the body, so each wait covers only the
      // older stage; sched_barrier keeps a prefetch from sinking to its use.
      // The first stage of S is loaded before the Q tile is built.
      float bA[ST][NTW], bB[ST][NTW];
      auto load = [&](int stg, float (*bv)[NTW]) {
#pragma unroll
        for (int u = 0; u < ST; ++u) {
          const int rl = min((stg * ST + u) * 4 + k4, rc - 1);
#pragma unroll
          for (int q = 0; q < NTW; ++q) bv[u][q] = sb[q][(size_t)(r0 + rl) * dh];
        }
      };
      load(0, bA);
      __syncthreads();
      const int ch = r0 / RR;
      run_schedule(t.rc_meta + t.rc_off[ch], t.rc_coef + t.rc_off[ch], t.rc_k[ch], Rl, Qt);
      __syncthreads();
      auto mma = [&](int stg, float (*bv)[NTW]) {
        // the stage's A values read from LDS together, then its MFMAs
        float a[ST][MT];
#pragma unroll
        for (int u = 0; u < ST; ++u) {
          const int rl = (stg * ST + u) * 4 + k4;
          const int rq = min(rl, RR - 1);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            const float qv = Qt[rq * QS + mt * 16 + j];
            a[u][mt] = rl < rc ? qv : 0.0f;
          }
        }
#pragma unroll
        for (int u = 0; u < ST; ++u)
#pragma unroll
          for (int q = 0; q < NTW; ++q)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
              acc[q][mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[u][mt], bv[u][q], acc[q][mt], 0, 0, 0);
      };
      const int nstage = (rc + 4 * ST - 1) / (4 * ST);
      for (int sp = 0; sp < nstage; sp += 2) {
        load(sp + 1, bB);
        __builtin_amdgcn_sched_barrier(0);
        mma(sp, bA);
        __builtin_amdgcn_sched_barrier(0);
        load(sp + 2, bA);
        __builtin_amdgcn_sched_barrier(0);
        mma(sp + 1, bB);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
#pragma unroll
    for (int q = 0; q < NTW; ++q) {
      const int c = (ns + wave + 4 * q) * 16 + j;
      if (!cok[q]) continue;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int row = mt * 16 + 4 * k4 + v;
          if (row < NK) {
            float* yp = y + ((size_t)i * NK + row) * C + c;
            *yp = accumulate ? *yp + acc[q][mt][v] : acc[q][mt][v];
          }
        }
    }
  }
}

// ------------------------------------------------------------ channel mixing
// out[row][c'] = sum_c W[o][c'][c] y[row][c] for the rows (i, m) of degree o:
// a tiled GEMM per degree, 64 rows x 64 output channels per block, 4x4
// outputs per thread.  With bf16 weights the inputs are rounded to bf16 and
// the products accumulate in fp32.
__device__ __forceinline__ float bf16_round(float x) { return __bfloat162float(__float2bfloat16(x)); }

template <bool BF16>
__global__ __launch_bounds__(256) void k_mix(const float* __restrict__ y, const void* __restrict__ Wv, int n, int nk,
                                             int o, int C, float* __restrict__ out) {
  __shared__ float Ys[16][64 + 1];
  __shared__ float Ws[16][64 + 1];
  const int nm = 2 * o + 1;
  const int64_t rows = (int64_t)n * nm;
  const int64_t r0 = (int64_t)blockIdx.x * 64;
  const int n0 = blockIdx.y * 64;
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  float acc[4][4] = {};
  auto row_addr = [&](int64_t r) -> int64_t {
    const int64_t i = r / nm, m = r % nm;
    return (i * nk + o * o + m) * (int64_t)C;
  };
  for (int k0 = 0; k0 < C; k0 += 16) {
    for (int q = threadIdx.x; q < 16 * 64; q += 256) {
      const int rr = q / 16, kk = q % 16;  // Y tile: 64 rows x 16 k
      const int64_t r = r0 + rr;
      float v = 0.0f;
      if (r < rows && k0 + kk < C) v = y[row_addr(r) + k0 + kk];
      Ys[kk][rr] = BF16 ? bf16_round(v) : v;
      const int nn = q / 16;  // W tile: 64 out channels x 16 k
      float w = 0.0f;
      if (n0 + nn < C && k0 + kk < C) {
        const size_t wi = ((size_t)o * C + n0 + nn) * C + k0 + kk;
        w = BF16 ? __bfloat162float(((const __hip_bfloat16*)Wv)[wi]) : ((const float*)Wv)[wi];
      }
      Ws[kk][nn] = w;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        a[u] = Ys[kk][ty * 4 + u];
        b[u] = Ws[kk][tx * 4 + u];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] += a[u] * b[v];
    }
    __syncthreads();
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int64_t r = r0 + ty * 4 + u;
    if (r >= rows) continue;
    const int64_t base = row_addr(r);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int cn = n0 + tx * 4 + v;
      if (cn < C) out[base + cn] = acc[u][v];
    }
  }
}

// MFMA channel mixing, used when C is a multiple of 16 up to 128.
// One workgroup of kMixWaves waves holds W^(o) in LDS (padded rows, so the
// 16-byte operand reads of 16 consecutive lanes hit distinct banks) and
// streams kMixGroups groups of 16*kMixWaves rows of irrep o. Each wave takes
// 16 rows and loads them once into registers as the B operand: lane (j, q)
// holds row j, channels 16s+4q..16s+4q+3. W^(o) rows are the A operand, read
// from LDS for every 16-channel output block; the reduction visits channel
// 16s+4q+u at step (s, u) on both operands. fp32: v_mfma_f32_16x16x4f32;
// bf16: y rounded to bf16 (nearest even) and v_mfma_f32_16x16x16bf16_1k,
// fp32 accumulation either way.
typedef short v4s __attribute__((ext_vector_type(4)));
struct MixGrid {
  int wg_start[kMaxL + 2];  // first workgroup of each irrep o, and the total
};
constexpr int kMixWaves = 8;
constexpr int kMixGroups = 4;
constexpr int kMixRowsPerWg = 16 * kMixWaves * kMixGroups;

__device__ __forceinline__ short bf16_bits(float x) {
  return (short)__bfloat16_as_ushort(__float2bfloat16(x));
}

template <bool BF16, int C16>
__global__ __launch_bounds__(64 * kMixWaves) void k_mix_mfma(const float* __restrict__ y, const void* __restrict__ Wv,
                                                            int n, int nk, int L, MixGrid g,
                                                            float* __restrict__ out) {
  constexpr int C = 16 * C16;
  constexpr int WS = BF16 ? C + 8 : C + 4;  // LDS row stride in elements
  extern __shared__ float mix_lds[];
  int o = 0;
  while (o < L && (int)blockIdx.x >= g.wg_start[o + 1]) ++o;
  const int nm = 2 * o + 1;
  const int64_t rows = (int64_t)n * nm;
  if (BF16) {
    uint16_t* Wl = (uint16_t*)mix_lds;
    const uint16_t* W = (const uint16_t*)Wv + (size_t)o * C * C;
    for (int q = threadIdx.x; q < C * C; q += blockDim.x) Wl[(q / C) * WS + q % C] = W[q];
  } else {
    const float* W = (const float*)Wv + (size_t)o * C * C;
    for (int q = threadIdx.x; q < C * C; q += blockDim.x) mix_lds[(q / C) * WS + q % C] = W[q];
  }
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int j = lane & 15, q4 = lane >> 4;
  const int64_t first = (int64_t)(blockIdx.x - g.wg_start[o]) * kMixRowsPerWg;
  for (int gi = 0; gi < kMixGroups; ++gi) {
    const int64_t r0 = first + (int64_t)(gi * kMixWaves + wave) * 16;
    if (r0 >= rows) break;  // uniform over the wave
    const int64_t r = r0 + j;
    const bool valid = r < rows;
    int64_t base = 0;
    if (valid) {
      const int64_t i = r / nm;
      base = (i * nk + o * o + (r - i * nm)) * C;
    }
    float4 yv[C16];
#pragma unroll
    for (int s = 0; s < C16; ++s)
      yv[s] = valid ? *(const float4*)(y + base + 16 * s + 4 * q4) : make_float4(0.f, 0.f, 0.f, 0.f);
    v4s yb[BF16 ? C16 : 1];
    if (BF16) {
#pragma unroll
      for (int s = 0; s < C16; ++s)
        yb[s] = (v4s){bf16_bits(yv[s].x), bf16_bits(yv[s].y), bf16_bits(yv[s].z), bf16_bits(yv[s].w)};
    }
#pragma unroll 2
    for (int cb = 0; cb < C16; ++cb) {
      v4f acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < C16; ++s) {
        if (BF16) {
          const v4s a = *(const v4s*)((const uint16_t*)mix_lds + (cb * 16 + j) * WS + 16 * s + 4 * q4);
          acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, yb[s], acc, 0, 0, 0);
        } else {
          const float4 a = *(const float4*)(mix_lds + (cb * 16 + j) * WS + 16 * s + 4 * q4);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, yv[s].x, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, yv[s].y, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, yv[s].z, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, yv[s].w, acc, 0, 0, 0);
        }
      }
      // acc[v] = out[row j][16cb + 4q + v]
      if (valid) *(float4*)(out + base + 16 * cb + 4 * q4) = make_float4(acc[0], acc[1], acc[2], acc[3]);
    }
  }
}

// ------------------------------------------------------------ backward
// Both per-edge products of the backward from one matrix product per
// (receiver, head).  The edge filter is linear in the solid harmonics,
// K_e[k][q] = sum_be R_be(r_e) Kc[be][k][q] with Kc the path-weighted filter
// coefficients, so the receiver's output gradient folds into
//   Z_i[be][q][c] = sum_k gy_i[k][c] Kc[be][k][q]
// and per head h one contraction over (q, c of h),
//   X_h[be][e] = sum_{q, c of h} Z_i[be][q][c] h_{j(e)}[q][c],
// gives both outputs of edge e = (i, j), r_e = r_i - r_j:
//   galpha[e][h] = sum_be R_be(r_e) X_h[be][e],
//   gedge[e][x]  = sum_be dR_be/dx(r_e) W[be][e],  W = sum_h alpha_eh X_h.
// The contraction runs on v_mfma_f32_16x16x4f32 with be as rows (MT tiles
// of 16), edges as columns (tiles of 16 edges; NTE tiles per wave, the
// wave's tiles are wave + NW et) and kappa = q dh + c as the reduction:
// step st covers kappa in [16 st, 16 st + 16), lane group k4 takes kappa =
// 16 st + 4 k4 .. + 3 (four channels of one row q, as 4 | dh) as one float4,
// and MFMA w of four uses component w.  LDS holds, per workgroup, the schedule of the Z
// sums (path weights folded in, staged once; read from global memory above
// L = 4, where it outgrows LDS), the head's slice of gy_i and Z
// for qc rows q at a time (Z[be][kappa - q0 dh]), with a row stride of
// qc dh + 4 or + 8 floats, an odd number of quadruples (the 16 rows be of an
// operand read start in distinct bank quadruples).  A workgroup takes
// rpw consecutive receivers; edge chunks of NW NTE 16 edges, Z rebuilt per
// chunk, head and row pass.  Each output element has one writer.
template <int L, int NTE, bool WA, bool WP, bool GT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void k_edge_geom(DevTables t, const float* __restrict__ pos,
                                                   const float* __restrict__ feat, const float* __restrict__ gy,
                                                   const int64_t* __restrict__ row_ptr,
                                                   const int32_t* __restrict__ col, const float* __restrict__ alpha,
                                                   int n, int rpw, int C, int H, int qc,
                                                   const int* __restrict__ gmeta, const float* __restrict__ gunit,
                                                   const int* __restrict__ goc, int gtot,
                                                   const float* __restrict__ Gt, int64_t n_edges,
                                                   float* __restrict__ galpha, float* __restrict__ gedge) {
  constexpr int NK = (L + 1) * (L + 1), MT = (NK + 15) / 16;
  constexpr bool STAGED = L <= 4;  // the schedule in LDS (it outgrows LDS above L = 4)
  extern __shared__ float4 sm4[];
  const int dh = C / H, dq = dh >> 2, ZS = qc * dh + (((qc * dh) >> 2) & 1 ? 8 : 4);
  float* gyl = (float*)sm4;  // [NK][dh]: gy_i of the head
  // STAGED: [gtot] schedule, [gtot] its coefficients times the path weights
  int* smeta = (int*)(gyl + NK * dh);
  float* sunit = gyl + NK * dh + gtot;
  float* Z = gyl + NK * dh + (STAGED ? 2 * gtot : 0);  // [NK be][ZS]: Z[be][qq][c] at be*ZS + qq*dh + c
  if (STAGED)
    for (int x = threadIdx.x; x < gtot; x += blockDim.x) {
      const int m = gmeta[x];
      smeta[x] = m;
      sunit[x] = gunit[x] * t.w_f[(m >> 18) & 511];
    }
  // workgroup -> rpw consecutive receivers; the receivers of one XCD are contiguous
  const int nxr = (n + 7) / 8, xcd = blockIdx.x % 8;
  const int rfirst = xcd * nxr + (blockIdx.x / 8) * rpw;
  const int rlast = min(min(rfirst + rpw, (xcd + 1) * nxr), n);  // uniform over the workgroup
  const int NW = blockDim.x >> 6, wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int l16 = lane & 15, k4 = lane >> 4;
  const int grp = threadIdx.x >> 2, sub = threadIdx.x & 3;  // kGeomGroups groups of four threads
  for (int i = rfirst; i < rlast; ++i) {
    const int64_t e0 = row_ptr[i], e1 = row_ptr[i + 1];
    const float xi = pos[3 * i], yi = pos[3 * i + 1], zi = pos[3 * i + 2];
    const float* gyi = gy + (size_t)i * NK * C;
    for (int64_t c0 = e0; c0 < e1; c0 += NW * NTE * 16) {
      const int ne = (int)min((int64_t)NW * NTE * 16, e1 - c0);
      const int ntiles = (ne + 15) / 16;
      int jn[NTE];
      bool ev[NTE], tlive[NTE];
#pragma unroll
      for (int et = 0; et < NTE; ++et) tlive[et] = __builtin_amdgcn_readfirstlane(wave + NW * et < ntiles ? 1 : 0) != 0;
      float dx[NTE], dy[NTE], dz[NTE];
      float Rv[NTE][MT][4];
      v4f W[NTE][MT];
#pragma unroll
      for (int et = 0; et < NTE; ++et) {
        const int nb = (wave + NW * et) * 16 + l16;
        ev[et] = nb < ne;
        jn[et] = col[c0 + (ev[et] ? nb : 0)];  // columns past ne read a valid sender, never stored
        dx[et] = xi - pos[3 * jn[et]], dy[et] = yi - pos[3 * jn[et] + 1], dz[et] = zi - pos[3 * jn[et] + 2];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          W[et][mt] = (v4f){0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int be = mt * 16 + 4 * k4 + v;
            Rv[et][mt][v] = (WA && be < NK) ? sh_poly<float>(t, be, dx[et], dy[et], dz[et]) : 0.0f;
          }
        }
      }
      for (int h = 0; h < H; ++h) {
        // every thread has passed a barrier since the last Z sums read gyl
        for (int x = threadIdx.x; x < NK * dq; x += blockDim.x)
          *(float4*)(gyl + 4 * x) = *(const float4*)(gyi + (size_t)(x / dq) * C + h * dh + 4 * (x % dq));
        v4f X[NTE][MT];
#pragma unroll
        for (int et = 0; et < NTE; ++et)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) X[et][mt] = (v4f){0.f, 0.f, 0.f, 0.f};
        for (int q0 = 0; q0 < NK; q0 += qc) {
          const int nq = min(qc, NK - q0);
          __syncthreads();  // gyl is staged; the previous steps have read Z
          {
            // Z rows of this pass: group grp walks its schedule entries, each
            // of its four threads takes the channel quads sub, sub + 4, ..
            const int ch = q0 / qc, off = goc[2 * ch], ck = goc[2 * ch + 1];
            for (int cq = sub; cq < dq && grp < kGeomGroups; cq += 4) {
              float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 4
              for (int k = 0; k < ck; ++k) {
                const int x = off + k * kGeomGroups + grp;
                const int m = STAGED ? smeta[x] : gmeta[x];
                const float cf = STAGED ? sunit[x] : gunit[x] * t.w_f[(m >> 18) & 511];
                const float4 g = *(const float4*)(gyl + (m & 63) * dh + 4 * cq);
                v.x += cf * g.x, v.y += cf * g.y, v.z += cf * g.z, v.w += cf * g.w;
                if (m < 0) {
                  *(float4*)(Z + ((m >> 6) & 63) * ZS + ((m >> 12) & 63) * dh + 4 * cq) = v;
                  v = make_float4(0.f, 0.f, 0.f, 0.f);
                }
              }
            }
          }
          __syncthreads();
          // three-stage pipeline: the features of steps st+1, st+2 load while
          // the MFMAs of st run
          const int nkap = nq * dh, nst = (nkap + 15) / 16;
          // each stage holds both operands of a step (A from LDS, B from the
          // senders' features), so no wait precedes the MFMAs
          // branch-free: clamped addresses, zeros selected after the loads
          auto loadb = [&](int st, float4* a, float4* b) {
            const int kap = 16 * min(st, nst - 1) + 4 * k4;
            const bool kok = kap < nkap;
            const unsigned kc = kok ? kap : 0;  // past the pass: a valid row, A = 0
            const unsigned q = q0 + kc / (unsigned)dh, c = kc % (unsigned)dh;
#pragma unroll
            for (int et = 0; et < NTE; ++et)
              b[et] = *(const float4*)(feat + ((size_t)jn[et] * NK + q) * C + h * dh + c);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
              const int be = mt * 16 + l16;
              const float4 z = *(const float4*)(Z + (be < NK ? be : 0) * ZS + kc);
              a[mt] = (be < NK && kok) ? z : make_float4(0.f, 0.f, 0.f, 0.f);
            }
          };
          auto mma = [&](const float4* a, const float4* b) {
#pragma unroll
            for (int et = 0; et < NTE; ++et) {
              if (!tlive[et]) continue;  // scalar: uniform over the wave
#pragma unroll
              for (int mt = 0; mt < MT; ++mt) {
                X[et][mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[mt].x, b[et].x, X[et][mt], 0, 0, 0);
                X[et][mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[mt].y, b[et].y, X[et][mt], 0, 0, 0);
                X[et][mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[mt].z, b[et].z, X[et][mt], 0, 0, 0);
                X[et][mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[mt].w, b[et].w, X[et][mt], 0, 0, 0);
              }
            }
          };
          float4 aA[MT], aB[MT], aC[MT], bA[NTE], bB[NTE], bC[NTE];
          loadb(0, aA, bA);
          loadb(1, aB, bB);
          for (int st = 0; st < nst; st += 3) {
            loadb(st + 2, aC, bC);
            __builtin_amdgcn_sched_barrier(0);
            mma(aA, bA);
            __builtin_amdgcn_sched_barrier(0);
            loadb(st + 3, aA, bA);
            __builtin_amdgcn_sched_barrier(0);
            if (st + 1 < nst) mma(aB, bB);
            __builtin_amdgcn_sched_barrier(0);
            loadb(st + 4, aB, bB);
            __builtin_amdgcn_sched_barrier(0);
            if (st + 2 < nst) mma(aC, bC);
            __builtin_amdgcn_sched_barrier(0);
          }
        }
        // lane (k4, l16) holds X_h[be = mt*16 + 4 k4 + v][edge column l16]
#pragma unroll
        for (int et = 0; et < NTE; ++et) {
          if (wave + NW * et >= ntiles) continue;  // uniform over the wave
          const int64_t e = c0 + (wave + NW * et) * 16 + l16;
          if (WA) {
            float p = 0.0f;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
              for (int v = 0; v < 4; ++v) p += Rv[et][mt][v] * X[et][mt][v];
            p += __shfl_xor(p, 16);
            p += __shfl_xor(p, 32);
            if (k4 == 0 && ev[et]) galpha[e * H + h] = p;
          }
          if (WP) {
            const float aw = (alpha && ev[et]) ? alpha[e * H + h] : 1.0f;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) W[et][mt] += aw * X[et][mt];
          }
        }
      }
      if (WP) {
#pragma unroll
        for (int et = 0; et < NTE; ++et) {
          if (wave + NW * et >= ntiles) continue;  // uniform over the wave
          float fx = 0.f, fy = 0.f, fz = 0.f;
          if (GT) {
            // the gradients from the per-edge table [3][NK][E] (consecutive
            // lanes l16 read consecutive edges)
            const int64_t ec = c0 + (ev[et] ? (wave + NW * et) * 16 + l16 : 0);
            const size_t plane = (size_t)NK * n_edges;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
              for (int v = 0; v < 4; ++v) {
                const int be = mt * 16 + 4 * k4 + v;
                if (be < NK) {
                  const float* gp = Gt + (size_t)be * n_edges + ec;
                  const float w = W[et][mt][v];
                  fx += gp[0] * w, fy += gp[plane] * w, fz += gp[2 * plane] * w;
                }
              }
          } else {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
              for (int v = 0; v < 4; ++v) {
                const int be = mt * 16 + 4 * k4 + v;
                if (be < NK) {
                  float gx, gyy, gz;
                  sh_poly_grad<float>(t, be, dx[et], dy[et], dz[et], gx, gyy, gz);
                  fx += gx * W[et][mt][v], fy += gyy * W[et][mt][v], fz += gz * W[et][mt][v];
                }
              }
          }
          fx += __shfl_xor(fx, 16), fy += __shfl_xor(fy, 16), fz += __shfl_xor(fz, 16);
          fx += __shfl_xor(fx, 32), fy += __shfl_xor(fy, 32), fz += __shfl_xor(fz, 32);
          if (k4 == 0 && ev[et]) {
            const int64_t e = c0 + (wave + NW * et) * 16 + l16;
            gedge[e * 3] = fx, gedge[e * 3 + 1] = fy, gedge[e * 3 + 2] = fz;
          }
        }
      }
    }
  }
}

// Per atom a: the forces of the edges it receives minus those it sends,
// each in ascending order (the sent edges through the transposed graph).
__global__ void k_force_gather(const int64_t* __restrict__ row_ptr, const int64_t* __restrict__ rowT,
                               const int32_t* __restrict__ perm, const float* __restrict__ gedge, int n,
                               float* __restrict__ gpos) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= (int64_t)n * 3) return;
  const int a = (int)(q / 3), x = (int)(q % 3);
  float s = 0.0f;
  for (int64_t e = row_ptr[a]; e < row_ptr[a + 1]; ++e) s += gedge[e * 3 + x];
  for (int64_t t = rowT[a]; t < rowT[a + 1]; ++t) s -= gedge[(int64_t)perm[t] * 3 + x];
  gpos[q] = s;
}

// transposed graph: rows[e] = receiver of edge e; counts of every sender
__global__ void k_edge_rows(const int64_t* __restrict__ row_ptr, int n, int32_t* __restrict__ rows) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) rows[e] = i;
}

__global__ void k_sender_counts(const int32_t* __restrict__ col, int64_t E, int n, int64_t* __restrict__ cnt,
                                int32_t* __restrict__ iota) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < E) {
    atomicAdd((unsigned long long*)&cnt[col[e]], 1ull);
    iota[e] = (int32_t)e;
  }
}

__global__ void k_transpose_gather(const int32_t* __restrict__ perm, const int32_t* __restrict__ rows,
                                   const float* __restrict__ alpha, int64_t E, int H, int32_t* __restrict__ colT,
                                   float* __restrict__ alphaT) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= E) return;
  const int64_t e = perm[t];
  colT[t] = rows[e];
  if (alpha)
    for (int h = 0; h < H; ++h) alphaT[t * H + h] = alpha[e * H + h];
}

// W^T[o][c][c'] = W[o][c'][c] (elements of `bytes` bytes)
template <typename E>
__global__ void k_transpose_mix(const E* __restrict__ W, int L1, int C, E* __restrict__ WT) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= (int64_t)L1 * C * C) return;
  const int64_t o = q / ((int64_t)C * C), r = q % ((int64_t)C * C);
  const int a = (int)(r / C), b = (int)(r % C);
  WT[(o * C + b) * C + a] = W[q];
}

// ------------------------------------------------------------ dense graphs
// Every atom attends to every other (the dense graphs of the scaling study,
// Sec. 4.1): the aggregation S_h = A_h T_h is a dense product with
// A_h[i][j] = alpha[i][j][h] for j != i and 0 on the diagonal.

// Global moments of the uncoupled products (App. G with every pair weighted
// alike): G[be][col] = sum_j R_be(p_j) h_j[col], col = q*C + c over the
// (L+1)^2 C columns of the features.  One thread per column, the (L+1)^2
// sums in fp64 registers over the atoms j = g, g + G, .. (in order) of group
// g = blockIdx.y; R of each atom is read by the whole workgroup (uniform).
template <int NK>
__global__ __launch_bounds__(256) void k_global_G_partial(const double* __restrict__ R, const float* __restrict__ feat,
                                                          int n, int cols, int G, double* __restrict__ part) {
  const int col = blockIdx.x * blockDim.x + threadIdx.x;
  const int g = blockIdx.y;
  const int cc = col < cols ? col : 0;  // columns past the end compute column 0, never stored
  double acc[NK];
#pragma unroll
  for (int b = 0; b < NK; ++b) acc[b] = 0.0;
  for (int j = g; j < n; j += G) {
    const double hv = (double)feat[(size_t)j * cols + cc];
    const double* Rj = R + (size_t)j * NK;
#pragma unroll
    for (int b = 0; b < NK; ++b) acc[b] += Rj[b] * hv;
  }
  if (col < cols)
#pragma unroll
    for (int b = 0; b < NK; ++b) part[((size_t)g * NK + b) * cols + col] = acc[b];
}

// G64 = sum over the groups in order; then the j-side coupling of the one
// global row: M[h][row][t] = sum over the row's entries of coef G64[be][q*C + c]
// (c = h*dh + t, the head-major layout of an S row).
__global__ void k_global_G_finish(const double* __restrict__ part, int64_t W, int G, double* __restrict__ G64) {
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (x >= W) return;
  double acc = 0.0;
  for (int g = 0; g < G; ++g) acc += part[(size_t)g * W + x];
  G64[x] = acc;
}

__global__ void k_global_couple(DevTables t, const double* __restrict__ G64, int C, int dh, float* __restrict__ M32) {
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (x >= (int64_t)t.dimT * C) return;
  const int row = (int)(x / C), c = (int)(x % C);
  double acc = 0.0;
  for (int e = t.ag_ptr[row]; e < t.ag_ptr[row + 1]; ++e) {
    const int gi = t.ag_idx[e];
    acc += (double)t.ag_coef[e] * G64[(size_t)(gi >> 6) * t.nk * C + (size_t)(gi & 63) * C + c];
  }
  M32[((size_t)(c / dh) * t.dimT + row) * dh + c % dh] = (float)acc;
}

// Per-degree attention weights alpha / D^f (Alg. 1), D = |r_i - r_j| in
// float64, head-major per f: alpha_f[(f*H + h)*E + e]; 0 for f > 0 at D = 0.
__global__ void k_alpha_dnorm(const float* __restrict__ pos, const int32_t* __restrict__ rows,
                              const int32_t* __restrict__ col, const float* __restrict__ alpha, int n,
                              int64_t n_edges, int H, int L, float* __restrict__ alpha_f) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= n_edges) return;
  const int i0 = rows[e], j0 = col[e];
  const int i = (unsigned)i0 < (unsigned)n ? i0 : 0, j = (unsigned)j0 < (unsigned)n ? j0 : 0;
  const double dx = (double)pos[3 * i] - pos[3 * j], dy = (double)pos[3 * i + 1] - pos[3 * j + 1],
               dz = (double)pos[3 * i + 2] - pos[3 * j + 2];
  const double D = sqrt(dx * dx + dy * dy + dz * dz);
  const double inv = D > 0.0 ? 1.0 / D : 0.0;
  double s = 1.0;
  for (int f = 0; f <= L; ++f) {
    for (int h = 0; h < H; ++h)
      alpha_f[((int64_t)f * H + h) * n_edges + e] = (float)((alpha ? (double)alpha[e * H + h] : 1.0) * s);
    s *= inv;
  }
}

// thread per edge: reads its H contiguous weights, writes one coalesced
// row segment per head
__global__ void k_alpha_head_major(const float* __restrict__ alpha, int64_t n_edges, int H,
                                   float* __restrict__ alpha_hm) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= n_edges) return;
  for (int h = 0; h < H; ++h) alpha_hm[(int64_t)h * n_edges + e] = alpha[e * H + h];
}

__global__ void k_iota(int n, int32_t* __restrict__ v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) v[i] = i;
}

// ------------------------------------------------------------ edge baseline
// Per receiver block: edges in batches of EB; for each edge the filter
// K[k][q] = sum_f w_afo sum_mf C^{o m}_{a al, f mf} R^(f)_mf(r_i - r_j) is built
// once in LDS (cost independent of C), then every channel applies it to h_j.
template <int L>
__global__ __launch_bounds__(128) void k_edge_tp(DevTables t, const float* __restrict__ pos,
                                                 const float* __restrict__ feat, const int64_t* __restrict__ row_ptr,
                                                 const int32_t* __restrict__ col, const float* __restrict__ alpha,
                                                 int C, int H, bool y_norm, int n_nodes, int64_t n_edges,
                                                 float* __restrict__ y) {
  constexpr int NK = (L + 1) * (L + 1);
  constexpr int EB = 4;
  extern __shared__ float sm[];
  float* Kl = sm;                 // [EB][NK*NK]
  float* Rl = sm + EB * NK * NK;  // [EB][NK]
  const int i = blockIdx.x;
  const int dh = C / H;
  // row bounds clamped to [0, E], senders to [0, n): a malformed graph
  // cannot move a read outside the caller's buffers
  const int64_t rb0 = row_ptr[i], rb1 = row_ptr[i + 1];
  const int64_t e0 = rb0 < 0 ? 0 : (rb0 > n_edges ? n_edges : rb0);
  const int64_t e1 = rb1 < e0 ? e0 : (rb1 > n_edges ? n_edges : rb1);
  auto sender = [&](int64_t e) {
    const int j = col[e];
    return (unsigned)j < (unsigned)n_nodes ? j : 0;
  };
  const float xi = pos[3 * i], yi = pos[3 * i + 1], zi = pos[3 * i + 2];
  for (int c0 = 0; c0 < C; c0 += blockDim.x) {
    const int c = c0 + threadIdx.x;
    const bool live = c < C;
    float acc[NK];
#pragma unroll
    for (int k = 0; k < NK; ++k) acc[k] = 0.0f;
    for (int64_t eb = e0; eb < e1; eb += EB) {
      const int nb = (e1 - eb) < EB ? (int)(e1 - eb) : EB;
      __syncthreads();
      for (int q = threadIdx.x; q < nb * NK; q += blockDim.x) {
        const int b = q / NK, k = q % NK;
        const int j = sender(eb + b);
        float dx = xi - pos[3 * j], dy = yi - pos[3 * j + 1], dz = zi - pos[3 * j + 2];
        if (y_norm) {  // R^(f)(r / D) = R^(f)(r) / D^f; the zero vector at D = 0
          const float D = sqrtf(dx * dx + dy * dy + dz * dz);
          const float sc = D > 0.0f ? 1.0f / D : 0.0f;
          dx *= sc, dy *= sc, dz *= sc;
        }
        Rl[q] = sh_poly<float>(t, k, dx, dy, dz);
      }
      __syncthreads();
      for (int q = threadIdx.x; q < nb * NK * NK; q += blockDim.x) {
        const int b = q / (NK * NK), s = q % (NK * NK);
        float v = 0.0f;
        for (int e = t.k_ptr[s]; e < t.k_ptr[s + 1]; ++e) v += t.k_coef[e] * Rl[b * NK + t.k_ridx[e]];
        Kl[q] = v;
      }
      __syncthreads();
      if (live) {
        for (int b = 0; b < nb; ++b) {
          const int j = sender(eb + b);
          const float a = alpha ? alpha[(eb + b) * H + c / dh] : 1.0f;
          float h[NK];
#pragma unroll
          for (int q = 0; q < NK; ++q) h[q] = a * feat[((size_t)j * NK + q) * C + c];
          const float* Kb = Kl + b * NK * NK;
#pragma unroll
          for (int k = 0; k < NK; ++k) {
            float s = 0.0f;
#pragma unroll
            for (int q = 0; q < NK; ++q) s += Kb[k * NK + q] * h[q];
            acc[k] += s;
          }
        }
      }
    }
    if (live) {
#pragma unroll
      for (int k = 0; k < NK; ++k) y[((size_t)i * NK + k) * C + c] = acc[k];
    }
  }
}

// Kernels whose dynamic LDS exceeds the 64 KB default must opt in (gfx950
// has 160 KB per CU).
template <typename K>
hipError_t allow_lds(K kernel, size_t bytes) {
  if (bytes <= 32768) return hipSuccess;
  return hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

}  // namespace

// ============================================================ launchers
hipError_t launch_sh(const DevTables& t, const float* pos, const int32_t* node_of, const double* origins_d,
                     const float* origins_f, const int32_t* origin_id, int origin_mod, int n, double* out_d,
                     float* out_f, hipStream_t s) {
  const int64_t total = (int64_t)n * t.nk;
  if (total == 0) return hipSuccess;
  k_sh<<<(unsigned)((total + 255) / 256), 256, 0, s>>>(t, pos, node_of, origins_d, origins_f, origin_id, origin_mod,
                                                        n, out_d, out_f);
  return hipGetLastError();
}

hipError_t launch_node_tp(const DevTables& t, const double* R, const int32_t* node_of, const float* feat,
                          int n_items, int C, int dh, float* T, hipStream_t s) {
  if (n_items == 0) return hipSuccess;
  // h staged in LDS with rows padded to 16 mod 32 floats when it is small
  int hs = (C + 15) / 16 * 16;
  if ((hs / 16) % 2 == 0) hs += 16;
  const size_t mbytes = sizeof(float) * (size_t)((t.tp_mo[t.L + 1] + 3) & ~3);
  const size_t hbytes = sizeof(float) * (size_t)t.nk * hs;
  if (hbytes > 32768) hs = 0;
  const size_t lds = mbytes + (hs > 0 ? hbytes : 0);
  static const int nw_env = [] {
    const char* v = getenv("E2F_TP_WAVES");
    return v ? atoi(v) : 0;
  }();
  // waves per workgroup: enough for 16 waves per CU at the number of
  // workgroups the LDS tile leaves room for (160 KB per CU)
  const int wg_cu = (int)std::max<size_t>(1, 163840 / std::max<size_t>(lds, 1));
  const int nw = nw_env == 4 || nw_env == 8 || nw_env == 16 ? nw_env : (wg_cu >= 4 ? 4 : (wg_cu >= 2 ? 8 : 16));
  switch (t.L * 32 + nw) {
#define E2F_CASE(LL, NW)                                                                                    \
  case LL * 32 + NW:                                                                                        \
    if (hipError_t e = allow_lds(k_node_tp<LL, NW>, lds); e != hipSuccess) return e;                        \
    k_node_tp<LL, NW><<<n_items, NW * 64, lds, s>>>(t, R, node_of, feat, C, dh, hs, T);                     \
    break;
#define E2F_CASES(LL) E2F_CASE(LL, 4) E2F_CASE(LL, 8) E2F_CASE(LL, 16)
    E2F_CASES(0) E2F_CASES(1) E2F_CASES(2) E2F_CASES(3) E2F_CASES(4) E2F_CASES(5) E2F_CASES(6)
#undef E2F_CASES
#undef E2F_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

namespace {
// Checks of the standalone aggregation's plan, one thread per receiver (in
// index order): bit 16 of *bad when a row's senders are not strictly
// ascending; *maxc = the largest edge count of a block of G consecutive
// receivers.  Row bounds are clamped to [0, n_edges].
__global__ void k_a3_checks(const int64_t* __restrict__ row_ptr, const int32_t* __restrict__ col, int n,
                            int64_t n_edges, int G, int* __restrict__ bad, int* __restrict__ maxc) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  auto clampe = [&](int64_t v) { return v < 0 ? (int64_t)0 : (v > n_edges ? n_edges : v); };
  const int64_t e0 = clampe(row_ptr[i]), e1 = max(e0, clampe(row_ptr[i + 1]));
  bool asc = true;
  for (int64_t e = e0 + 1; e < e1; ++e) asc = asc && col[e] > col[e - 1];
  if (!asc) atomicOr(bad, 16);
  if (i % G == 0) {
    const int last = min(n, i + G);
    const int64_t b0 = clampe(row_ptr[i]), b1 = max(b0, clampe(row_ptr[last]));
    atomicMax(maxc, (int)min(b1 - b0, (int64_t)0x7fffffff));
  }
}
// order: bit 32 of *bad unless every entry is in [0, n) and taken once
// (cnt: n ints, zero on entry)
__global__ void k_a3_order(const int32_t* __restrict__ order, int n, int* __restrict__ cnt, int* __restrict__ bad) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= n) return;
  const int i = order[r];
  if ((unsigned)i >= (unsigned)n) atomicOr(bad, 32);
  else if (atomicAdd(cnt + i, 1) != 0) atomicOr(bad, 32);
}
}  // namespace

hipError_t launch_a3_order_check(const int32_t* order, int n, int* cnt, int* bad, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipError_t e = launch_fill((float*)cnt, n, 0.0f, s);
  if (e != hipSuccess) return e;
  k_a3_order<<<(n + 255) / 256, 256, 0, s>>>(order, n, cnt, bad);
  return hipGetLastError();
}

hipError_t launch_a3_checks(const int64_t* row_ptr, const int32_t* col, int n, int64_t n_edges, int* bad,
                            int* maxc, hipStream_t s) {
  hipError_t e = launch_fill((float*)maxc, 1, 0.0f, s);
  if (e != hipSuccess || n == 0) return e;
  k_a3_checks<<<(n + 255) / 256, 256, 0, s>>>(row_ptr, col, n, n_edges, 16, bad, maxc);
  return hipGetLastError();
}

int a3_union_max() { return kUnionMax; }

size_t blocks_tmp_bytes(int nblk) {
  size_t b = 0;
  hipcub::DeviceScan::ExclusiveSum(nullptr, b, (const int32_t*)nullptr, (int32_t*)nullptr, nblk + 1);
  return b;
}

hipError_t launch_block_union(const int64_t* row_ptr, const int32_t* col_pair, const int32_t* order, int n,
                              int32_t* blk_count, int32_t* blk_off, int32_t* uni, int32_t* ucount, int32_t* edge_slot,
                              void* tmp, size_t tmp_bytes, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int G = 16;
  const int nblk = (n + G - 1) / G;
  // the scan's extra element, cleared by a fill kernel (0.0f has the bits of int 0)
  hipError_t e = launch_fill((float*)(blk_count + nblk), 1, 0.0f, s);
  if (e != hipSuccess) return e;
  if ((e = launch_fill((float*)(ucount + nblk), 1, 0.0f, s)) != hipSuccess) return e;
  k_block_edges<<<(nblk + 255) / 256, 256, 0, s>>>(row_ptr, order, n, G, nblk, blk_count);
  size_t b = tmp_bytes;
  if ((e = hipcub::DeviceScan::ExclusiveSum(tmp, b, blk_count, blk_off, nblk + 1, s)) != hipSuccess) return e;
  const size_t lds = 2 * sizeof(int32_t) * kUnionMax;
  if ((e = allow_lds(k_block_union, lds)) != hipSuccess) return e;
  k_block_union<<<nblk, 256, lds, s>>>(row_ptr, col_pair, order, n, G, blk_off, uni, ucount, edge_slot);
  return hipGetLastError();
}

hipError_t launch_aggregate(const float* T, int pair_base, const int64_t* row_ptr, const int32_t* col_pair,
                            const float* alpha, const float* alpha_hm, int64_t n_edges, int n_total,
                            const int32_t* order, const int32_t* uni, const int32_t* blk_off,
                            const int32_t* ucount, const int32_t* edge_slot, bool use_blocks, int n, int dimT, int C,
                            int H, float* S, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int dh = C / H;
  if (use_blocks) {
    // columns per wave: 64*NQ, register stages NS, waves per workgroup WV,
    // and a cap on workgroups per CU (through unused dynamic LDS; 0: none).
    // Measured: at a mean degree of ~80 (20k atoms, L=4) NQ=2 with four
    // workgroups per CU is fastest; at ~200 (200k atoms, L=6) NQ=4 with two
    // (the A-operand build of a workgroup grows with its block's edges).
    // E2F_AGG_CFG="NQ,NS,WV" and E2F_AGG_WGCU override (tuning).
    const bool dense_rows = n_edges >= (int64_t)128 * n_total;
    int nq = dense_rows ? 4 : 2, ns = 3, wv = 4;
    if (const char* cfg = getenv("E2F_AGG_CFG")) sscanf(cfg, "%d,%d,%d", &nq, &ns, &wv);
    static const int wgcu_env = [] {
      const char* v = getenv("E2F_AGG_WGCU");
      return v ? atoi(v) : -1;
    }();
    const int wgcu = wgcu_env >= 0 ? wgcu_env : (dense_rows ? 2 : 0);
    // XCD x takes the column tasks x, x+8, ... over every block, so each T
    // element is read by one XCD's L2 (blocks in space order within a task);
    // E2F_AGG_MAP=0 gives each XCD a contiguous range of blocks instead
    static const int by_task = [] {
      const char* v = getenv("E2F_AGG_MAP");
      return v ? atoi(v) : 1;
    }();
    const size_t static_lds = sizeof(int64_t) * kPiece + sizeof(float4) * kPiece * 4;
    const size_t pad = wgcu > 0 && (size_t)(163840 / wgcu) > static_lds ? 163840 / wgcu - static_lds - 256 : 0;
    const int nblk = (n + 15) / 16;
    const int ntg = (dimT * dh + 64 * nq - 1) / (64 * nq);
    const int ntgw = (ntg + wv - 1) / wv;
    const int bpx = (nblk + kXcds - 1) / kXcds;
    const int64_t blocks = by_task ? (int64_t)kXcds * ((H * ntgw + kXcds - 1) / kXcds) * nblk
                                   : (int64_t)kXcds * bpx * H * ntgw;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
#define E2F_AGG(NQ_, NS_, WV_)                                                                             \
  if (nq == NQ_ && ns == NS_ && wv == WV_) {                                                              \
    if (pad > 0)                                                                                          \
      if (hipError_t e = allow_lds(k_aggregate_mfma<NQ_, NS_, WV_>, pad); e != hipSuccess) return e;     \
    k_aggregate_mfma<NQ_, NS_, WV_><<<(unsigned)blocks, 64 * WV_, pad, s>>>(                              \
        T, pair_base, uni, blk_off, ucount, row_ptr, order, edge_slot, alpha_hm, n_edges, n, nblk, bpx,        \
        by_task, ntg,                                                                                     \
        ntgw, dimT, C, dh, H, S);                                                                         \
    return hipGetLastError();                                                                             \
  }
    E2F_AGG(2, 2, 4) E2F_AGG(2, 3, 4) E2F_AGG(2, 4, 4) E2F_AGG(2, 3, 8) E2F_AGG(2, 3, 2) E2F_AGG(4, 3, 4)
    E2F_AGG(4, 3, 8) E2F_AGG(6, 2, 4)
#undef E2F_AGG
    return hipErrorInvalidValue;
  }
  const int64_t W4 = (int64_t)dimT * C / 4;
  const int nchunk = (int)((W4 + kAggChunk4 - 1) / kAggChunk4);
  const int ngroups = (n + kAggRecv - 1) / kAggRecv;
  const int gpx = (ngroups + kXcds - 1) / kXcds;
  const int64_t blocks = (int64_t)kXcds * gpx * nchunk;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  k_aggregate_rows<<<(unsigned)blocks, 64 * kAggRecv, 0, s>>>((const float4*)T, pair_base, row_ptr, col_pair, alpha,
                                                              order, n,
                                                              (int)W4, nchunk, ngroups, gpx, C, dh, H, (float4*)S);
  return hipGetLastError();
}

namespace {
struct OuterShape {
  int nw = 0;
  size_t lds = 0;   // work space (staging, then G)
};
// column tiles per wave: 4 (measured faster than 8 at L = 4: more waves,
// fewer registers each); E2F_OUTER_NTW=8 selects 8 at L <= 4 (tuning)
int outer_ntw(int L) {
  static const int env = [] {
    const char* v = getenv("E2F_OUTER_NTW");
    return v ? atoi(v) : 0;
  }();
  return L > 4 ? 4 : (env == 4 || env == 8 ? env : 4);
}

OuterShape outer_shape(int L, int C, int H) {
  const int nk = (L + 1) * (L + 1), mp = 16 * ((nk + 15) / 16), dh = C / H;
  const int nc = nk * dh, nt = (nc + 63) / 64 * 4, ntwm = outer_ntw(L);  // tiles in whole 64-column blocks
  OuterShape o;
  o.nw = (nt + ntwm - 1) / ntwm;
  o.nw = std::max(o.nw, 2);  // the staging needs at least kOuterEdges threads
  o.lds = std::max(sizeof(float) * (size_t)kOuterEdges * (mp + 16) + sizeof(int) * kOuterEdges,
                   sizeof(float) * (size_t)nk * (nc + 4));
  return o;
}
}  // namespace

int outer_agg_groups(int L, int C, int H) { return 64 * outer_shape(L, C, H).nw / (C / H / 4); }

bool outer_agg_supported(int L, int C, int H) {
  const OuterShape o = outer_shape(L, C, H);
  return o.nw >= 1 && o.nw <= (outer_ntw(L) == 8 ? 8 : 16) && o.lds <= 160 * 1024;
}

hipError_t launch_outer_agg(const DevTables& t, const float* Re, const int64_t* row_ptr, const int32_t* col,
                            const float* alpha_hm, int64_t n_edges, const float* feat,
                            const int32_t* order, const int* cmeta, const float* ccoef, const int* pmeta,
                            const float* ptab, int ntab, int ck, int cgroups, int n, int C, int H, int hdiv,
                            int n_nodes, float* S, hipStream_t s) {
  if (n == 0) return hipSuccess;
  if (!outer_agg_supported(t.L, C, H) || cgroups != outer_agg_groups(t.L, C, H)) return hipErrorInvalidValue;
  const OuterShape o = outer_shape(t.L, C, H);
  // receivers per workgroup, and the coupling schedule in LDS when it fits
  // beside the work space with two workgroups per CU
  static const int rpw_env = [] {
    const char* v = getenv("E2F_OUTER_RPW");
    return v ? atoi(v) : 0;
  }();
  const int rpw = rpw_env > 0 ? rpw_env : 8;
  // the packed schedule (L <= 4) leaves room for three workgroups per CU at
  // L = 4, C = 128, H = 8; E2F_OUTER_PACKED=0 stages the unpacked one (tuning)
  static const bool packed_env = [] {
    const char* v = getenv("E2F_OUTER_PACKED");
    return !v || atoi(v) != 0;
  }();
  const bool packed = packed_env && ntab > 0 && pmeta && ptab;
  const size_t sched_b = packed ? sizeof(float) * ((size_t)ck * cgroups + ntab)
                                : sizeof(float) * 2 * (size_t)ck * cgroups;
  const bool sched_lds = o.lds + sched_b <= 80 * 1024;
  const int ntab_k = packed && sched_lds ? ntab : 0;
  const int work_floats = sched_lds ? (int)(o.lds / sizeof(float)) : 0;
  const size_t lds = o.lds + (sched_lds ? sched_b : 0);
  const int nrx = (n + kXcds - 1) / kXcds;
  const int64_t blocks = (int64_t)kXcds * ((nrx + rpw - 1) / rpw) * H;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  // launch bound 512 (up to 256 VGPRs) at L <= 4 with at most 8 waves; at
  // L = 5, 6 the bound 1024 keeps two workgroups per CU (170 VGPRs under
  // 512 allow one; 1024 spills a few and measures faster: 311 vs 404 ms for
  // 200k atoms, L = 6)
  const int lb = t.L <= 4 && o.nw <= 8 ? 512 : 1024;
  switch (t.L * 64 + outer_ntw(t.L) * 4 + (lb == 512 ? 0 : 1)) {
#define E2F_CASE(LL, NTWM, LB)                                                                              \
  case LL * 64 + NTWM * 4 + (LB == 512 ? 0 : 1):                                                            \
    if (hipError_t e = allow_lds(k_outer_agg<LL, NTWM, LB>, lds); e != hipSuccess) return e;                \
    k_outer_agg<LL, NTWM, LB><<<(unsigned)blocks, 64 * o.nw, lds, s>>>(t, Re, row_ptr, col,                 \
                                                                      alpha_hm, n_edges, feat, order, cmeta, \
                                                                      ccoef, pmeta, ptab, ntab_k, ck,        \
                                                                      cgroups, work_floats, n, nrx, rpw, C,  \
                                                                      H, hdiv, n_nodes, S);                  \
    break;
#define E2F_CASES(LL) E2F_CASE(LL, 4, 512) E2F_CASE(LL, 4, 1024)
    E2F_CASES(0) E2F_CASES(1) E2F_CASES(2) E2F_CASES(3) E2F_CASES(4) E2F_CASES(5) E2F_CASES(6)
    E2F_CASE(0, 8, 512) E2F_CASE(1, 8, 512) E2F_CASE(2, 8, 512) E2F_CASE(3, 8, 512) E2F_CASE(4, 8, 512)
#undef E2F_CASES
#undef E2F_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

int fuse_groups(int L) { return ((L + 1) * (L + 1) + 3) / 4; }

bool outer_fused_supported(int L, int C, int H, int64_t n_nodes) {
  return L >= 0 && L <= kFuseMaxL && H >= 1 && C == 16 * H &&
         (uint64_t)n_nodes * H * fuse_groups(L) * 16 <= 0xffffffffull;
}

hipError_t launch_fuse_build(int L, int nkr, const int* fptr, const int* fidx, const double* fcoef,
                             const double* R, const int32_t* order, int n, float* F, hipStream_t s) {
  if (n == 0) return hipSuccess;
  if (L < 0 || L > kFuseMaxL || nkr < 1) return hipErrorInvalidValue;
  const int nk = (L + 1) * (L + 1);
  k_fuse_build<<<(n + kFuseRecv - 1) / kFuseRecv, 256, 0, s>>>(fptr, fidx, fcoef, fuse_stride(nk, nkr), nk, R, order,
                                                                 n, F);
  return hipGetLastError();
}

hipError_t launch_feat_qmajor(int L, const float* feat, int n, int C, float* featq, hipStream_t s) {
  if (n == 0) return hipSuccess;
  if (C % 16) return hipErrorInvalidValue;
  const int64_t total = (int64_t)n * (C / 16) * fuse_groups(L) * 16;
  if ((total + 255) / 256 > 0x7fffffff) return hipErrorInvalidValue;
  k_feat_qmajor3<<<(unsigned)((total + 255) / 256), 256, 0, s>>>(feat, n, (L + 1) * (L + 1), C, fuse_groups(L),
                                                                  (uint4*)featq, (uint2*)featq + 2 * total);
  return hipGetLastError();
}

// (the stacked alpha / D^f passes: 5, 14 and 30 K rows at L = 1, 2, 3, and
// 30 at L = 4)
bool fused_krows_supported(int L, int nkr) {
  const int nk = (L + 1) * (L + 1);
  return L >= 0 && L <= kFuseMaxL && (nkr == nk || (L == 1 && nkr == 5) || (L == 2 && nkr == 14) || (L >= 3 && nkr == 30));
}

hipError_t launch_outer_fused(int L, int nkr, const float* Re, const int64_t* row_ptr, const int32_t* col,
                              const FusedSegs& sg, int64_t n_edges, const float* featq, const int32_t* order,
                              const float* F, int n, int C, int H, int hdiv, int n_nodes, bool accumulate, float* y,
                              hipStream_t s) {
  if (n == 0) return hipSuccess;
  if (!outer_fused_supported(L, C, H, n_nodes) || !fused_krows_supported(L, nkr)) return hipErrorInvalidValue;
  const int nk = (L + 1) * (L + 1), mpk = 16 * ((nkr + 15) / 16);
  // segments: start[0] = 0, increasing, each at most nk rows (the harmonics'
  // component kr - start stays below nk)
  if (sg.n < 1 || sg.n > kFusedSegs || sg.start[0] != 0) return hipErrorInvalidValue;
  for (int q = 0; q < sg.n; ++q) {
    const int end = q + 1 < sg.n ? sg.start[q + 1] : nkr;
    if (end <= sg.start[q] || end - sg.start[q] > nk) return hipErrorInvalidValue;
  }
  const int nw = (nk + 3) / 4 + 1;  // a product wave per group of four components, and the staging wave
  const size_t lds =
      sizeof(float) * (2 * (size_t)kFuseRows * 2 * mpk + 2 * (size_t)kFuseRows + (size_t)sg.n * kOuterEdges);
  const size_t nq = (size_t)n_nodes * H * fuse_groups(L) * 16;  // entries of the re-laid features
  const uint4* fhm = (const uint4*)featq;
  const uint2* flo = (const uint2*)(fhm + nq);
  static const int rpw_env = [] {
    const char* v = getenv("E2F_OUTER_RPW");
    return v ? atoi(v) : 0;
  }();
  const int rpw = rpw_env > 0 ? rpw_env : 8;
  const int nrx = (n + kXcds - 1) / kXcds;
  const int64_t blocks = (int64_t)kXcds * ((nrx + rpw - 1) / rpw) * H;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
#define E2F_LAUNCH(LL, KK)                                                                                     \
  do {                                                                                                         \
    if (hipError_t e = allow_lds(k_outer_fused<LL, 512, KK>, lds); e != hipSuccess) return e;                  \
    k_outer_fused<LL, 512, KK><<<(unsigned)blocks, 64 * nw, lds, s>>>(Re, row_ptr, col, sg, n_edges, fhm, flo,  \
                                                                      order, F, n, nrx, rpw, C, H, hdiv,       \
                                                                      n_nodes, accumulate, y);                 \
  } while (0)
  if (nkr != nk) {
    switch (L) {
      case 1: E2F_LAUNCH(1, 5); break;
      case 2: E2F_LAUNCH(2, 14); break;
      case 3: E2F_LAUNCH(3, 30); break;
      case 4: E2F_LAUNCH(4, 30); break;
      default: return hipErrorInvalidValue;
    }
  } else {
    switch (L) {
      case 0: E2F_LAUNCH(0, 1); break;
      case 1: E2F_LAUNCH(1, 4); break;
      case 2: E2F_LAUNCH(2, 9); break;
      case 3: E2F_LAUNCH(3, 16); break;
      case 4: E2F_LAUNCH(4, 25); break;
      default: return hipErrorInvalidValue;
    }
  }
#undef E2F_LAUNCH
  return hipGetLastError();
}

hipError_t launch_recouple(const DevTables& t, const double* R, const float* S, bool shared_s, const int32_t* order,
                           int n, int C, int dh, float* y, hipStream_t s, bool accumulate) {
  const int64_t s_stride = shared_s ? 0 : (int64_t)t.dimT * C;
  if (n == 0) return hipSuccess;
  const int nt = (C + 15) / 16;  // channel tiles; 4 waves
  const int ntw = nt <= 4 ? 1 : (nt <= 8 ? 2 : 4);
  const size_t lds = sizeof(float) * (size_t)rc_rows(t.nk) * rc_qstride(t.nk);
  switch (t.L) {
#define E2F_RC(LL, W)                                                                                       \
  if (ntw == W) {                                                                                           \
    if (hipError_t e = allow_lds(k_recouple<LL, W>, lds); e != hipSuccess) return e;                        \
    k_recouple<LL, W><<<n, 256, lds, s>>>(t, R, S, s_stride, order, C, dh, accumulate, y);                  \
  }
#define E2F_CASE(LL)                                                                                        \
  case LL:                                                                                                  \
    E2F_RC(LL, 1) E2F_RC(LL, 2) E2F_RC(LL, 4)                                                               \
    break;
    E2F_CASE(0) E2F_CASE(1) E2F_CASE(2) E2F_CASE(3) E2F_CASE(4) E2F_CASE(5) E2F_CASE(6)
#undef E2F_CASE
#undef E2F_RC
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_mix(int L, const float* y, const void* W, bool w_bf16, int n, int C, float* out, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int nk = (L + 1) * (L + 1);
  if (C % 16 == 0 && C <= 128) {
    MixGrid g{};
    for (int o = 0; o <= L; ++o) {
      const int64_t wgs = ((int64_t)n * (2 * o + 1) + kMixRowsPerWg - 1) / kMixRowsPerWg;
      if ((int64_t)g.wg_start[o] + wgs > 0x7fffffff) return hipErrorInvalidValue;
      g.wg_start[o + 1] = g.wg_start[o] + (int)wgs;
    }
    const int C16 = C / 16;
    const size_t lds = (size_t)C * (w_bf16 ? (C + 8) * 2 : (C + 4) * 4);
#define E2F_MIX(B_, C16_)                                                                                    \
  if (w_bf16 == B_ && C16 == C16_) {                                                                         \
    if (hipError_t e = allow_lds(k_mix_mfma<B_, C16_>, lds); e != hipSuccess) return e;                      \
    k_mix_mfma<B_, C16_><<<g.wg_start[L + 1], 64 * kMixWaves, lds, s>>>(y, W, n, nk, L, g, out);             \
    return hipGetLastError();                                                                                \
  }
    E2F_MIX(false, 1) E2F_MIX(false, 2) E2F_MIX(false, 3) E2F_MIX(false, 4)
    E2F_MIX(false, 5) E2F_MIX(false, 6) E2F_MIX(false, 7) E2F_MIX(false, 8)
    E2F_MIX(true, 1) E2F_MIX(true, 2) E2F_MIX(true, 3) E2F_MIX(true, 4)
    E2F_MIX(true, 5) E2F_MIX(true, 6) E2F_MIX(true, 7) E2F_MIX(true, 8)
#undef E2F_MIX
    return hipErrorInvalidValue;
  }
  // other channel counts: tiled VALU GEMM per irrep
  for (int o = 0; o <= L; ++o) {
    const int64_t rows = (int64_t)n * (2 * o + 1);
    dim3 grid((unsigned)((rows + 63) / 64), (unsigned)((C + 63) / 64));
    if (w_bf16) k_mix<true><<<grid, 256, 0, s>>>(y, W, n, nk, o, C, out);
    else k_mix<false><<<grid, 256, 0, s>>>(y, W, n, nk, o, C, out);
  }
  return hipGetLastError();
}

hipError_t launch_edge_tp(const DevTables& t, const float* pos, const float* feat, const int64_t* row_ptr,
                          const int32_t* col_idx, const float* alpha, int n, int64_t n_edges, int C, int H, float* y,
                          hipStream_t s, bool y_norm) {
  if (n == 0) return hipSuccess;
  const int threads = C <= 64 ? 64 : 128;
  const size_t lds = sizeof(float) * ((size_t)4 * t.nk * t.nk + (size_t)4 * t.nk);
  switch (t.L) {
#define E2F_CASE(LL)                                                                                        \
  case LL:                                                                                                  \
    if (hipError_t e = allow_lds(k_edge_tp<LL>, lds); e != hipSuccess) return e;                            \
    k_edge_tp<LL><<<n, threads, lds, s>>>(t, pos, feat, row_ptr, col_idx, alpha, C, H, y_norm, n, n_edges, y); \
    break;
    E2F_CASE(0) E2F_CASE(1) E2F_CASE(2) E2F_CASE(3) E2F_CASE(4) E2F_CASE(5) E2F_CASE(6)
#undef E2F_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}


int global_groups(int n, int nk, int C) {
  const int colblocks = (nk * C + 255) / 256;
  return std::max(1, std::min(n, (2048 + colblocks - 1) / colblocks));
}

hipError_t launch_global_moment(const DevTables& t, const double* R, const float* feat, int n, int C, int dh,
                                double* part, double* G64, float* M32, hipStream_t s) {
  const int nk = t.nk, cols = nk * C, G = global_groups(n, nk, C);
  const int64_t W = (int64_t)nk * cols;
  const dim3 grid((unsigned)((cols + 255) / 256), (unsigned)G);
  switch (t.L) {
#define E2F_CASE(LL)                                                                                        \
  case LL:                                                                                                  \
    k_global_G_partial<(LL + 1) * (LL + 1)><<<grid, 256, 0, s>>>(R, feat, n, cols, G, part);                \
    break;
    E2F_CASE(0) E2F_CASE(1) E2F_CASE(2) E2F_CASE(3) E2F_CASE(4) E2F_CASE(5) E2F_CASE(6)
#undef E2F_CASE
    default: return hipErrorInvalidValue;
  }
  k_global_G_finish<<<(unsigned)((W + 255) / 256), 256, 0, s>>>(part, W, G, G64);
  k_global_couple<<<(unsigned)(((int64_t)t.dimT * C + 255) / 256), 256, 0, s>>>(t, G64, C, dh, M32);
  return hipGetLastError();
}

hipError_t launch_alpha_dnorm(const float* pos, const int64_t* row_ptr, const int32_t* col, const float* alpha, int n,
                              int64_t n_edges, int H, int L, int32_t* rows, float* alpha_f, hipStream_t s) {
  if (n_edges == 0) return hipSuccess;
  const int64_t blocks = (n_edges + 255) / 256;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  if (row_ptr) k_edge_rows<<<(n + 255) / 256, 256, 0, s>>>(row_ptr, n, rows);
  k_alpha_dnorm<<<(unsigned)blocks, 256, 0, s>>>(pos, rows, col, alpha, n, n_edges, H, L, alpha_f);
  return hipGetLastError();
}

hipError_t launch_alpha_head_major(const float* alpha, int64_t n_edges, int H, float* alpha_hm, hipStream_t s) {
  if (n_edges == 0) return hipSuccess;
  const int64_t blocks = (n_edges + 255) / 256;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  k_alpha_head_major<<<(unsigned)blocks, 256, 0, s>>>(alpha, n_edges, H, alpha_hm);
  return hipGetLastError();
}

hipError_t launch_iota(int n, int32_t* v, hipStream_t s) {
  if (n == 0) return hipSuccess;
  k_iota<<<(n + 255) / 256, 256, 0, s>>>(n, v);
  return hipGetLastError();
}

bool edge_geom_supported(int C, int H) {
  return C % H == 0 && (C / H) % 4 == 0 && C <= 256;
}

size_t edge_geom_lds(int L, int dh, int qc, int gtot) {
  const size_t nk = (size_t)(L + 1) * (L + 1);
  const size_t zs = (size_t)qc * dh + (((qc * dh) >> 2) & 1 ? 8 : 4);
  return sizeof(float) * (nk * dh + (L <= 4 ? 2 * (size_t)gtot : 0) + nk * zs);
}

hipError_t launch_edge_geom(const DevTables& t, const float* pos, const float* feat, const float* gy,
                            const int64_t* row_ptr, const int32_t* col_idx, const float* alpha, int n, int C, int H,
                            int qc, const int* gmeta, const float* gunit, const int* goc, int gtot, const float* Gt,
                            int64_t n_edges, float* galpha, float* gedge, hipStream_t s) {
  if (n == 0 || (!galpha && !gedge)) return hipSuccess;
  if (!edge_geom_supported(C, H) || qc < 1 || qc > t.nk) return hipErrorInvalidValue;
  const int dh = C / H;
  const size_t lds = edge_geom_lds(t.L, dh, qc, gtot);
  if (lds > 160 * 1024) return hipErrorInvalidValue;
  const int mode = (galpha ? 1 : 0) + (gedge ? 2 : 0);
  int rpw = 4;
  if (const char* v = getenv("E2F_GEOM_RPW")) rpw = std::max(1, atoi(v));
  const int nxr = (n + 7) / 8;
  const unsigned grid = 8u * (unsigned)((nxr + rpw - 1) / rpw);
  const int geom_threads = 256;  // four waves of two edge tiles (the schedule's 128 threads build Z)
  switch (t.L * 8 + mode + (Gt && gedge ? 4 : 0)) {
#define E2F_G(LL, WA_, WP_, GT_)                                                                              \
  case LL * 8 + (WA_ ? 1 : 0) + (WP_ ? 2 : 0) + (GT_ ? 4 : 0):                                                \
    if (hipError_t e = allow_lds(k_edge_geom<LL, 2, WA_, WP_, GT_>, lds); e != hipSuccess) return e;          \
    k_edge_geom<LL, 2, WA_, WP_, GT_><<<grid, geom_threads, lds, s>>>(t, pos, feat, gy, row_ptr, col_idx,      \
                                                                         alpha, n, rpw, C, H, qc, gmeta,     \
                                                                         gunit, goc, gtot, Gt, n_edges,      \
                                                                         galpha, gedge);                     \
    break;
#define E2F_GL(LL)                                                                                            \
  E2F_G(LL, true, false, false) E2F_G(LL, false, true, false) E2F_G(LL, true, true, false)                    \
  E2F_G(LL, false, true, true) E2F_G(LL, true, true, true)
    E2F_GL(0) E2F_GL(1) E2F_GL(2) E2F_GL(3) E2F_GL(4) E2F_GL(5) E2F_GL(6)
#undef E2F_GL
#undef E2F_G
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Gradients of the solid harmonics of every edge, r_e = r_i - r_j:
// Gt[c][be][e] = dR_be/dr_c (c = x, y, z) for be < nk.  Component-major:
// blockIdx.y = be, so a wave evaluates one polynomial (no divergence, its
// table reads uniform) and stores consecutive edges.
__global__ void k_edge_shgrad(DevTables t, const float* __restrict__ pos, const int32_t* __restrict__ rows,
                              const int32_t* __restrict__ col, int64_t n_edges, float* __restrict__ Gt) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int be = blockIdx.y;
  if (e >= n_edges) return;
  const int i = rows[e], j = col[e];
  float gx, gyy, gz;
  sh_poly_grad<float>(t, be, pos[3 * i] - pos[3 * j], pos[3 * i + 1] - pos[3 * j + 1], pos[3 * i + 2] - pos[3 * j + 2],
                      gx, gyy, gz);
  const size_t plane = (size_t)t.nk * n_edges, x = (size_t)be * n_edges + e;
  Gt[x] = gx;
  Gt[plane + x] = gyy;
  Gt[2 * plane + x] = gz;
}

hipError_t launch_edge_shgrad(const DevTables& t, const float* pos, const int32_t* rows, const int32_t* col,
                              int64_t n_edges, float* Gt, hipStream_t s) {
  if (n_edges == 0) return hipSuccess;
  const int64_t blocks = (n_edges + 255) / 256;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  k_edge_shgrad<<<dim3((unsigned)blocks, (unsigned)t.nk), 256, 0, s>>>(t, pos, rows, col, n_edges, Gt);
  return hipGetLastError();
}

hipError_t launch_force_gather(const int64_t* row_ptr, const int64_t* rowT, const int32_t* perm, const float* gedge,
                               int n, float* gpos, hipStream_t s) {
  if (n == 0) return hipSuccess;
  k_force_gather<<<(unsigned)(((int64_t)n * 3 + 255) / 256), 256, 0, s>>>(row_ptr, rowT, perm, gedge, n, gpos);
  return hipGetLastError();
}


size_t transpose_tmp_bytes(int n, int64_t E) {
  size_t a = 0, b = 0;
  hipcub::DeviceRadixSort::SortPairs(nullptr, a, (const int32_t*)nullptr, (int32_t*)nullptr, (const int32_t*)nullptr,
                                     (int32_t*)nullptr, (int)E);
  hipcub::DeviceScan::ExclusiveSum(nullptr, b, (int64_t*)nullptr, (int64_t*)nullptr, n + 1);
  return std::max(a, b);
}

hipError_t launch_transpose_graph(const int64_t* row_ptr, const int32_t* col_idx, const float* alpha, int n,
                                  int64_t E, int H, int32_t* rows, int32_t* iota, int32_t* keys_out, int32_t* perm,
                                  int64_t* cnt, int64_t* rowT_ptr, int32_t* colT, float* alphaT, void* tmp,
                                  size_t tmp_bytes, hipStream_t s) {
  hipError_t e = hipMemsetAsync(cnt, 0, sizeof(int64_t) * (size_t)(n + 1), s);
  if (e != hipSuccess) return e;
  if (E > 0) {
    k_edge_rows<<<(n + 255) / 256, 256, 0, s>>>(row_ptr, n, rows);
    k_sender_counts<<<(unsigned)((E + 255) / 256), 256, 0, s>>>(col_idx, E, n, cnt, iota);
    int bits = 1;
    while ((1LL << bits) < (int64_t)n) ++bits;
    size_t b = tmp_bytes;
    // stable: edges of one sender keep their (ascending receiver) order
    if ((e = hipcub::DeviceRadixSort::SortPairs(tmp, b, col_idx, keys_out, iota, perm, (int)E, 0, bits, s)) !=
        hipSuccess)
      return e;
  }
  size_t b = tmp_bytes;
  if ((e = hipcub::DeviceScan::ExclusiveSum(tmp, b, cnt, rowT_ptr, n + 1, s)) != hipSuccess) return e;
  if (E > 0) k_transpose_gather<<<(unsigned)((E + 255) / 256), 256, 0, s>>>(perm, rows, alpha, E, H, colT, alphaT);
  return hipGetLastError();
}

hipError_t launch_transpose_mix(const void* W, bool bf16, int L, int C, void* WT, hipStream_t s) {
  const int64_t total = (int64_t)(L + 1) * C * C;
  const unsigned grid = (unsigned)((total + 255) / 256);
  if (bf16)
    k_transpose_mix<uint16_t><<<grid, 256, 0, s>>>((const uint16_t*)W, L + 1, C, (uint16_t*)WT);
  else
    k_transpose_mix<float><<<grid, 256, 0, s>>>((const float*)W, L + 1, C, (float*)WT);
  return hipGetLastError();
}

}  // namespace e2f
