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
    const uint32_t hi0 = __umulhi(M0, c[0]), lo0 = M0 * c[0];
    const uint32_t hi1 = __umulhi(M1, c[2]), lo1 = M1 * c[2];
    const uint32_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0; c[1] = lo1; c[2] = n2; c[3] = lo0;
  }
}

// Four standard normals of Philox block `blk` of one tensor. Uniforms are
// u = (x + 1/2) 2^-32; Box-Muller pairs (u0,u1) and (u2,u3) give
// r cos(2 pi u_odd), r sin(2 pi u_odd) with r = sqrt(-2 ln u_even). In fp32
// the conversion of x is exact below 2^24 (the far tail, small u) and rounds x
// to 24 bits above, which moves ln u by at most 2^-24; the angle uses
// sincospi on 2u.
__device__ __forceinline__ void gauss4(uint64_t blk, uint64_t seed, uint32_t tensor_id,
                                       uint32_t step, float (&z)[4]) {
  uint32_t c[4] = {(uint32_t)blk, (uint32_t)(blk >> 32), tensor_id, step};
  philox4x32_10(c, (uint32_t)seed, (uint32_t)(seed >> 32));
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const float u = ((float)c[2 * p] + 0.5f) * 0x1p-32f;
    const float r = sqrtf(-2.f * logf(u));
    const float twice_u = ((float)c[2 * p + 1] + 0.5f) * 0x1p-31f;
    float sn, cs;
    sincospif(twice_u, &sn, &cs);
    z[2 * p] = r * cs;
    z[2 * p + 1] = r * sn;
  }
}

// g[j] = (g[j] + sigma*C*z_j) / B (or without the division). One thread per
// Philox block of 4 consecutive elements.
__global__ void add_noise_kernel(float* g, int64_t n, float sigma_c, int divide, float b_norm,
                                 uint64_t seed, uint32_t tensor_id, uint32_t step) {
  const int64_t nblk = (n + 3) / 4;
  const bool vec = (((uintptr_t)g) & 15) == 0;
  for (int64_t blk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; blk < nblk;
       blk += (int64_t)gridDim.x * blockDim.x) {
    float z[4];
    gauss4((uint64_t)blk, seed, tensor_id, step, z);
    const int64_t j0 = blk * 4;
    if (vec && j0 + 4 <= n) {
      f32x4 v = *(const f32x4*)(g + j0);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float t = v[q] + sigma_c * z[q];
        v[q] = divide ? t / b_norm : t;
      }
      *(f32x4*)(g + j0) = v;
    } else {
      for (int q = 0; q < 4 && j0 + q < n; ++q) {
        const float t = g[j0 + q] + sigma_c * z[q];
        g[j0 + q] = divide ? t / b_norm : t;
      }
    }
  }
}

hipError_t launch_clip_factors(const float* norm2, int B, float C, float* c, hipStream_t s) {
  if (B == 0) return hipSuccess;
  hipLaunchKernelGGL(clip_factors_kernel, dim3((B + 255) / 256), dim3(256), 0, s, norm2, B, C, c);
  return hipGetLastError();
}

hipError_t launch_add_noise(float* g, int64_t n, float sigma_c, int divide, float b_norm,
                            uint64_t seed, uint32_t tensor_id, uint32_t step, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int64_t nblk = (n + 3) / 4;
  int64_t grid = (nblk + 255) / 256;
  if (grid > 8192) grid = 8192;
  hipLaunchKernelGGL(add_noise_kernel, dim3((unsigned)grid), dim3(256), 0, s, g, n, sigma_c,
                     divide, b_norm, seed, tensor_id, step);
  return hipGetLastError();
}

}  // namespace dpg
