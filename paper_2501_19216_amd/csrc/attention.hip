// Attention weights of the layer's edges (Alg. 1 takes them as input; App. E
// computes them from the scalar features and a radial basis):
//   logit[(i,j)][h] = sum_t q[i][h][t] k[j][h][t] + sum_r w[h][r] exp(-((d - mu_r)/sigma)^2),
//   mu_r = r cutoff / (R - 1), sigma = cutoff / (R - 1), d = |r_i - r_j|,
//   alpha[(i,j)][h] = env(d) * softmax over the row of logit[.][h],
//   env(d) = (cos(pi d / cutoff) + 1) / 2 below the cutoff, 0 from it on.
// One wave per receiver row: lane l takes head l % Hp (Hp = H rounded up to a
// power of two) and every (64/Hp)-th edge, so a wave's accesses of alpha
// [E][H] are contiguous and the per-head max and sum are xor-shuffle
// reductions over the lanes of one head (fixed order: deterministic).  The
// logits are computed once and kept in alpha between the passes.
#include <hip/hip_runtime.h>

#include "e2f_launch.h"

namespace e2f {
namespace {

template <int HP>
__global__ __launch_bounds__(256) void k_attention(const float* __restrict__ pos, const float* __restrict__ q,
                                                   const float* __restrict__ kf, int n, int H, int dk,
                                                   const float* __restrict__ rbf_w, int R, float rc,
                                                   const int64_t* __restrict__ row_ptr,
                                                   const int32_t* __restrict__ col, float* __restrict__ alpha) {
  constexpr int EPI = 64 / HP;  // edges per wave iteration
  const int i = blockIdx.x * 4 + (int)(threadIdx.x >> 6);
  if (i >= n) return;  // uniform over the wave
  const int lane = threadIdx.x & 63;
  const int h = lane % HP, el = lane / HP;
  const bool hv = h < H;
  const int hc = hv ? h : 0;
  const int64_t e0 = row_ptr[i], e1 = row_ptr[i + 1];
  if (e0 == e1) return;
  float w[kAttnMaxRbf];
#pragma unroll
  for (int r = 0; r < kAttnMaxRbf; ++r) w[r] = r < R ? rbf_w[hc * R + r] : 0.0f;
  const float sigma = rc / (float)(R - 1), inv = 1.0f / sigma;
  const float xi = pos[3 * i], yi = pos[3 * i + 1], zi = pos[3 * i + 2];
  const float* qi = q + ((size_t)i * H + hc) * dk;
  // q of this lane's head in registers, as float4 (d_k a multiple of 4, up to 64)
  const bool vec = (dk & 3) == 0 && dk <= 64;
  float4 q4[16];
#pragma unroll
  for (int t = 0; t < 16; ++t)
    q4[t] = (vec && 4 * t < dk) ? ((const float4*)qi)[t] : make_float4(0.f, 0.f, 0.f, 0.f);
  const float kPi = 3.14159265358979f;
  auto logit = [&](int64_t e, float& env) {
    const int j = col[e];
    const float dx = xi - pos[3 * j], dy = yi - pos[3 * j + 1], dz = zi - pos[3 * j + 2];
    const float d = sqrtf(dx * dx + dy * dy + dz * dz);
    const float* kj = kf + ((size_t)j * H + hc) * dk;
    float l = 0.0f;
    if (vec) {
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        if (4 * t < dk) {
          const float4 kv = ((const float4*)kj)[t];
          l += q4[t].x * kv.x + q4[t].y * kv.y + q4[t].z * kv.z + q4[t].w * kv.w;
        }
      }
    } else {
      for (int t = 0; t < dk; ++t) l += qi[t] * kj[t];
    }
#pragma unroll
    for (int r = 0; r < kAttnMaxRbf; ++r) {
      if (r < R) {
        const float z = (d - (float)r * sigma) * inv;
        l += w[r] * expf(-z * z);
      }
    }
    env = d < rc ? 0.5f * (cosf(kPi * d / rc) + 1.0f) : 0.0f;
    return l;
  };
  // pass 1: logits, kept in the output; pass 2: exponentials; pass 3: scale
  float mx = -INFINITY;
  for (int64_t e = e0 + el; e < e1; e += EPI) {
    float env;
    const float l = logit(e, env);
    if (hv) alpha[e * H + h] = l;
    mx = fmaxf(mx, l);
  }
#pragma unroll
  for (int o = 32; o >= HP; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  float den = 0.0f;
  for (int64_t e = e0 + el; e < e1; e += EPI) {
    if (!hv) continue;
    const float ex = expf(alpha[e * H + h] - mx);
    alpha[e * H + h] = ex;
    den += ex;
  }
#pragma unroll
  for (int o = 32; o >= HP; o >>= 1) den += __shfl_xor(den, o);
  const float rden = 1.0f / den;
  for (int64_t e = e0 + el; e < e1; e += EPI) {
    if (!hv) continue;
    const int j = col[e];
    const float dx = xi - pos[3 * j], dy = yi - pos[3 * j + 1], dz = zi - pos[3 * j + 2];
    const float d = sqrtf(dx * dx + dy * dy + dz * dz);
    const float env = d < rc ? 0.5f * (cosf(kPi * d / rc) + 1.0f) : 0.0f;
    alpha[e * H + h] = env * alpha[e * H + h] * rden;
  }
}

}  // namespace

hipError_t launch_attention(const float* pos, const float* q, const float* k, int n, int H, int dk,
                            const float* rbf_w, int R, float rc, const int64_t* row_ptr, const int32_t* col_idx,
                            float* alpha, hipStream_t s) {
  if (n == 0) return hipSuccess;
  int hp = 1;
  while (hp < H) hp <<= 1;
  const unsigned grid = (unsigned)((n + 3) / 4);
  switch (hp) {
#define E2F_ATT(P)                                                                                     \
  case P:                                                                                              \
    k_attention<P><<<grid, 256, 0, s>>>(pos, q, k, n, H, dk, rbf_w, R, rc, row_ptr, col_idx, alpha);   \
    break;
    E2F_ATT(1) E2F_ATT(2) E2F_ATT(4) E2F_ATT(8) E2F_ATT(16) E2F_ATT(32) E2F_ATT(64)
#undef E2F_ATT
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace e2f
