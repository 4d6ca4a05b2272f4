// Clip factors (eq. 2, eq. 7) and the Gaussian noise of eq. 3.
#include "common.hpp"
#include "kernels.hpp"

namespace dpg {

// c_i = min(1, C / ||g_i||), and 1 when the norm is 0 (the limit of the
// expression); computed in double and rounded once.
__global__ void clip_factors_kernel(const float* __restrict__ norm2, int B, float C, float* c) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B) return;
  const double n2 = (double)norm2[i];
  double r = 1.0;
  if (n2 > 0.0) {
    r = (double)C / sqrt(n2);
    if (r > 1.0) r = 1.0;
  }
  c[i] = (float)r;
}

// Philox4x32 with 10 rounds (Salmon, Moraes, Dror, Shaw, SC'11): each round
// multiplies counter words 0 and 2 by the round constants, keeps both halves
// of the 64-bit products and mixes them with words 1 and 3 and the key; the
// key advances by the Weyl increments between rounds.
__device__ __forceinline__ void philox4x32_10(uint32_t (&c)[4], uint32_t k0, uint32_t k1) {
  constexpr uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
  constexpr uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) { k0 += W0; k1 += W1; }
    // Full 64-bit products: one v_mad_u64_u32 each instead of mul_hi + mul_lo.
    const uint64_t p0 = (uint64_t)M0 * c[0], p1 = (uint64_t)M1 * c[2];
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c[1] ^ k0;
    const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c[3] ^ k1;
    c[0] = n0; c[1] = (uint32_t)p1; c[2] = n2; c[3] = (uint32_t)p0;
  }
}

// Four standard normals of Philox block `blk` of one tensor. Uniforms are
// u = (x + 1/2) 2^-32; Box-Muller pairs (u0,u1) and (u2,u3) give
// r cos(2 pi u_odd), r sin(2 pi u_odd) with r = sqrt(-2 ln u_even). In fp32
// the conversion of x is exact below 2^24 (the far tail, small u) and rounds x
// to 24 bits above, which moves ln u by at most 2^-24. The transcendental
// steps run on the hardware units: ln u = ln 2 * V_LOG_F32(u) (base 2),
// V_SQRT_F32, and V_SIN_F32 / V_COS_F32, whose argument is in revolutions,
// so that sin(2 pi u) is V_SIN_F32(u) with no range reduction for u in (0,1).
__device__ __forceinline__ void gauss4(uint64_t blk, uint64_t seed, uint32_t tensor_id,
                                       uint32_t step, float (&z)[4]) {
  uint32_t c[4] = {(uint32_t)blk, (uint32_t)(blk >> 32), tensor_id, step};
  philox4x32_10(c, (uint32_t)seed, (uint32_t)(seed >> 32));
  constexpr float MINUS_2_LN2 = -1.3862943611198906f;
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const float u = ((float)c[2 * p] + 0.5f) * 0x1p-32f;
    const float r = __builtin_amdgcn_sqrtf(MINUS_2_LN2 * __builtin_amdgcn_logf(u));
    const float v = ((float)c[2 * p + 1] + 0.5f) * 0x1p-32f;
    z[2 * p] = r * __builtin_amdgcn_cosf(v);
    z[2 * p + 1] = r * __builtin_amdgcn_sinf(v);
  }
}

// g[j] = (g[j] + sigma*C*z_j) * inv_b, inv_b = 1/B rounded to fp32 (1 when
// there is no division). One thread per Philox block of 4 consecutive
// elements; the gradient is streamed once (non-temporal).
__global__ void add_noise_kernel(float* g, int64_t n, float sigma_c, float inv_b, uint64_t seed,
                                 uint32_t tensor_id, uint32_t step) {
  const int64_t nblk = (n + 3) / 4;
  const bool vec = (((uintptr_t)g) & 15) == 0;
  for (int64_t blk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; blk < nblk;
       blk += (int64_t)gridDim.x * blockDim.x) {
    float z[4];
    gauss4((uint64_t)blk, seed, tensor_id, step, z);
    const int64_t j0 = blk * 4;
    if (vec && j0 + 4 <= n) {
      f32x4 v = __builtin_nontemporal_load((const f32x4*)(g + j0));
#pragma unroll
      for (int q = 0; q < 4; ++q) v[q] = (v[q] + sigma_c * z[q]) * inv_b;
      __builtin_nontemporal_store(v, (f32x4*)(g + j0));
    } else {
      for (int q = 0; q < 4 && j0 + q < n; ++q) g[j0 + q] = (g[j0 + q] + sigma_c * z[q]) * inv_b;
    }
  }
}

hipError_t launch_clip_factors(const float* norm2, int B, float C, float* c, hipStream_t s) {
  if (B == 0) return hipSuccess;
  hipLaunchKernelGGL(clip_factors_kernel, dim3((B + 255) / 256), dim3(256), 0, s, norm2, B, C, c);
  return hipGetLastError();
}

hipError_t launch_add_noise(float* g, int64_t n, float sigma_c, float inv_b, uint64_t seed,
                            uint32_t tensor_id, uint32_t step, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int64_t nblk = (n + 3) / 4;
  int64_t grid = (nblk + 255) / 256;
  if (grid > 8192) grid = 8192;
  hipLaunchKernelGGL(add_noise_kernel, dim3((unsigned)grid), dim3(256), 0, s, g, n, sigma_c,
                     inv_b, seed, tensor_id, step);
  return hipGetLastError();
}

}  // namespace dpg
