// Dense-graph aggregation (Sec. 4.1's dense graphs; Alg. 1 with its attention
// tensor alpha in R^{N x N x H}): per head h the einsum "ijh,jhds->ihds" is a
// dense product S_h = A_h T_h, with A_h [N x N] the attention weights of head
// h (zero diagonal) and T_h [N x W] the head's columns of the j-side node
// products (W = dimT * C/H).  fp32 on v_mfma_f32_16x16x4f32.
//
// Tiling: a workgroup of eight waves owns a 256 x 128 tile of S_h (4 x 2
// waves of 64 x 64, each 4 x 4 MFMA tiles of 16 x 16); K advances 16 at a
// time through double-buffered LDS, the next K slab loaded into registers
// while the current one is multiplied.  A is stored by the alpha kernel with
// rows padded to a multiple of 32 (zeros), so K needs no tail handling.
// Workgroups of one XCD take a contiguous range of (head, row block) tiles
// with every column block, so A's row slabs and T's column slabs in flight
// on an XCD are shared through its L2.  Measured at L = 3, C = 128, H = 8
// (N = 250 .. 4000, whole dense forward): 256 x 128 tiles 0.098 / 0.210 /
// 0.550 / 1.897 / 7.066 ms, against 128 x 128: 0.104 / 0.195 / 0.615 /
// 2.097 / 7.899, 128 x 256: .. / 7.690, 256 x 256: 0.128 / .. / 6.979, and
// 128 x 128 with K slabs of 32: .. / 8.154.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>

#include "e2f_launch.h"

namespace e2f {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

// A[h][i][j] = alpha[i][j][h] (1 if alpha is NULL), 0 for i == j and for the
// padding columns j >= n of rows of lda floats.
__global__ void k_dense_alpha_pad(const float* __restrict__ alpha, int n, int H, int lda, float* __restrict__ A) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // (h, i, j) over padded rows
  const int64_t rowsz = (int64_t)n * lda;
  if (q >= rowsz * H) return;
  const int h = (int)(q / rowsz);
  const int64_t ij = q - (int64_t)h * rowsz;
  const int i = (int)(ij / lda), j = (int)(ij - (int64_t)i * lda);
  A[q] = (j >= n || i == j) ? 0.0f : (alpha ? alpha[((int64_t)i * n + j) * H + h] : 1.0f);
}

// S_h[i][c] = sum_k A_h[i][k] T_h[k][c] for i < n, c < W, k < lda (A is zero
// past n; T rows past n are never read with a nonzero weight, their index is
// clamped).  T_h[k][c] = T[k * ldt + h * W + c], S likewise.  WGM x WGN waves
// of 64 x 64 outputs each; K slabs of BK.
template <int WGM, int WGN, int BK>
__global__ __launch_bounds__(64 * WGM * WGN) void k_dense_gemm(const float* __restrict__ A, int lda, int n,
                                                               const float* __restrict__ T, int64_t ldt, int W,
                                                               float* __restrict__ S, int n_ib, int n_cb, int H,
                                                               int per_xcd) {
  constexpr int BM = 64 * WGM, BN = 64 * WGN, NT = 64 * WGM * WGN;
  // LDS row strides (floats): A [BM][AS] with k contiguous (the MFMA reads of
  // 16 rows x 2 k fall in distinct banks), B [BK][BS] with columns contiguous
  // (16 mod 32: the two k rows of a read fall in different bank halves)
  constexpr int AS = BK + 2, BS = BN + 16;
  constexpr int FA = BM * BK / 4 / NT, FB = BK * BN / 4 / NT;  // float4 loads per thread
  static_assert(FA * NT * 4 == BM * BK && FB * NT * 4 == BK * BN, "tile loads must divide evenly");
  __shared__ __attribute__((aligned(16))) float As[2][BM * AS];
  __shared__ __attribute__((aligned(16))) float Bs[2][BK * BS];
  const int tile = (blockIdx.x % 8) * per_xcd + (int)(blockIdx.x / 8);
  if (tile >= H * n_ib * n_cb) return;  // uniform over the workgroup
  const int cb = tile % n_cb, ib = (tile / n_cb) % n_ib, h = tile / (n_cb * n_ib);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int l16 = lane & 15, k4 = lane >> 4;
  const int wm = (wave / WGN) * 64, wn = (wave % WGN) * 64;
  const float* Ah = A + (int64_t)h * n * lda;
  const float* Th = T + (int64_t)h * W;
  const int nk = lda / BK;
  // float4 f of a slab: A row f / (BK/4) (clamped to n - 1), k 4 (f % (BK/4));
  // B row f / (BN/4) (clamped to n - 1; A is zero there), columns clamped to
  // W - 4 (never stored)
  float4 ra[FA], rb[FB];
  auto load = [&](int kt) {
    const int k0 = kt * BK;
#pragma unroll
    for (int u = 0; u < FA; ++u) {
      const int f = tid + u * NT, r = min(ib * BM + f / (BK / 4), n - 1);
      ra[u] = *(const float4*)(Ah + (int64_t)r * lda + k0 + 4 * (f % (BK / 4)));
    }
#pragma unroll
    for (int u = 0; u < FB; ++u) {
      const int f = tid + u * NT, r = min(k0 + f / (BN / 4), n - 1);
      const int c = min(cb * BN + 4 * (f % (BN / 4)), W - 4);
      rb[u] = *(const float4*)(Th + (int64_t)r * ldt + c);
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int u = 0; u < FA; ++u) {
      const int f = tid + u * NT;
      float* d = As[buf] + (f / (BK / 4)) * AS + 4 * (f % (BK / 4));
      *(float2*)d = make_float2(ra[u].x, ra[u].y);
      *(float2*)(d + 2) = make_float2(ra[u].z, ra[u].w);
    }
#pragma unroll
    for (int u = 0; u < FB; ++u) {
      const int f = tid + u * NT;
      *(float4*)(Bs[buf] + (f / (BN / 4)) * BS + 4 * (f % (BN / 4))) = rb[u];
    }
  };
  v4f acc[4][4];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) acc[mt][nt] = (v4f){0.f, 0.f, 0.f, 0.f};
  load(0);
  store(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load(kt + 1);  // in flight while this slab is multiplied
    const float* as = As[buf];
    const float* bs = Bs[buf];
#pragma unroll
    for (int kk = 0; kk < BK; kk += 4) {
      float a[4], b[4];
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) a[mt] = as[(wm + mt * 16 + l16) * AS + kk + k4];
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) b[nt] = bs[(kk + k4) * BS + wn + nt * 16 + l16];
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
          acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[mt], b[nt], acc[mt][nt], 0, 0, 0);
    }
    if (kt + 1 < nk) store(buf ^ 1);  // the other buffer was last read before the previous barrier
    __syncthreads();
  }
  // acc[mt][nt][v] = S[row wm + 16 mt + 4 k4 + v][col wn + 16 nt + l16]
  float* Sh = S + (int64_t)h * W;
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = ib * BM + wm + mt * 16 + 4 * k4 + v;
      if (row >= n) continue;
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int col = cb * BN + wn + nt * 16 + l16;
        if (col < W) Sh[(int64_t)row * ldt + col] = acc[mt][nt][v];
      }
    }
}

}  // namespace

int dense_lda(int n) { return (n + 31) / 32 * 32; }  // a multiple of the K slab

hipError_t launch_dense_alpha(const float* alpha, int n, int H, float* A, hipStream_t s) {
  const int64_t total = (int64_t)n * dense_lda(n) * H;
  if (total == 0) return hipSuccess;
  if ((total + 255) / 256 > 0x7fffffff) return hipErrorInvalidValue;
  k_dense_alpha_pad<<<(unsigned)((total + 255) / 256), 256, 0, s>>>(alpha, n, H, dense_lda(n), A);
  return hipGetLastError();
}

hipError_t launch_dense_aggregate(const float* A, int n, const float* T, int dimT, int C, int H, float* S,
                                  hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int dh = C / H, W = dimT * dh;
  if (W < 4 || W % 4) return hipErrorInvalidValue;
  // tile shape (waves in M, waves in N, K slab); E2F_DENSE_TILE = "WGM,WGN,BK"
  // selects another of the compiled shapes (tuning)
  static const int shape = [] {
    const char* v = getenv("E2F_DENSE_TILE");
    int a = 4, b = 2, k = 16;
    if (v) sscanf(v, "%d,%d,%d", &a, &b, &k);
    return a * 100 + b * 10 + k / 16;
  }();
  const int wgm = shape / 100, wgn = (shape / 10) % 10;
  const int n_ib = (n + 64 * wgm - 1) / (64 * wgm), n_cb = (W + 64 * wgn - 1) / (64 * wgn);
  const int64_t tiles = (int64_t)H * n_ib * n_cb;
  const int64_t per_xcd = (tiles + 7) / 8;
  if (8 * per_xcd > 0x7fffffff) return hipErrorInvalidValue;
  const int64_t ldt = (int64_t)dimT * C;
  switch (shape) {
#define E2F_DG(M_, N_, K_)                                                                                    \
  case M_ * 100 + N_ * 10 + K_ / 16:                                                                          \
    k_dense_gemm<M_, N_, K_><<<(unsigned)(8 * per_xcd), 64 * M_ * N_, 0, s>>>(A, dense_lda(n), n, T, ldt, W, S, \
                                                                              n_ib, n_cb, H, (int)per_xcd);   \
    break;
    E2F_DG(2, 2, 16) E2F_DG(4, 2, 16) E2F_DG(4, 4, 16)
#undef E2F_DG
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace e2f
