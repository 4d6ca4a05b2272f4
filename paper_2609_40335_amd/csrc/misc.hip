// Clip factors (eq. 2, eq. 7) and the Gaussian noise of eq. 3.
#include "common.hpp"
#include "kernels.hpp"

namespace dpg {

// c_i = min(1, C / ||g_i||), and 1 when the norm is 0 (the limit of the
// expression); computed in double and rounded once. A squared norm that is
// not finite (inf, or NaN from an overflowed or corrupt gradient) gives
// c_i = 0: min(1, C/inf) is 0, and a NaN norm is read the same way, so that
// no such example can enter the sum unclipped (the bound of eq. 2). cs
// (optional) receives scale * c_i, also rounded once from double; c may be
// null when only cs is wanted. The squared norm is norm2[i], plus norm2_b[i]
// (in fp32, as an accumulating norm call would add it) when a second part is
// given.
__global__ void clip_factors_kernel(const float* __restrict__ norm2,
                                    const float* __restrict__ norm2_b, int B, float C, float scale,
                                    float* c, float* cs) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B) return;
  const double n2 = (double)(norm2_b ? norm2[i] + norm2_b[i] : norm2[i]);
  double r = 1.0;
  if (!__builtin_isfinite(n2)) {
    r = 0.0;
  } else if (n2 > 0.0) {
    r = (double)C / sqrt(n2);
    if (r > 1.0) r = 1.0;
  }
  if (c) c[i] = (float)r;
  if (cs) cs[i] = (float)(r * (double)scale);
}

// ACC: g[j] = (g[j] + sigma*C*z_j) * inv_b; otherwise g[j] = sigma*C*z_j *
// inv_b without reading g (equal to the accumulating form on zeros). inv_b =
// 1/B rounded to fp32 (1 when there is no division). One thread per Philox
// block of 4 consecutive elements; the gradient is streamed (non-temporal).
template <bool ACC>
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
      f32x4 v = {0.f, 0.f, 0.f, 0.f};
      if (ACC) v = __builtin_nontemporal_load((const f32x4*)(g + j0));
#pragma unroll
      for (int q = 0; q < 4; ++q) v[q] = (v[q] + sigma_c * z[q]) * inv_b;
      __builtin_nontemporal_store(v, (f32x4*)(g + j0));
    } else {
      for (int q = 0; q < 4 && j0 + q < n; ++q)
        g[j0 + q] = ((ACC ? g[j0 + q] : 0.f) + sigma_c * z[q]) * inv_b;
    }
  }
}

hipError_t launch_clip_factors(const float* norm2, const float* norm2_b, int B, float C,
                               float scale, float* c, float* cs, hipStream_t s) {
  if (B == 0) return hipSuccess;
  hipLaunchKernelGGL(clip_factors_kernel, dim3((B + 255) / 256), dim3(256), 0, s, norm2, norm2_b,
                     B, C,
                     scale, c, cs);
  return hipGetLastError();
}

hipError_t launch_add_noise(float* g, int64_t n, float sigma_c, float inv_b, uint64_t seed,
                            uint32_t tensor_id, uint32_t step, bool accumulate, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int64_t nblk = (n + 3) / 4;
  int64_t grid = (nblk + 255) / 256;
  if (grid > 8192) grid = 8192;
  if (accumulate)
    hipLaunchKernelGGL(add_noise_kernel<true>, dim3((unsigned)grid), dim3(256), 0, s, g, n,
                       sigma_c, inv_b, seed, tensor_id, step);
  else
    hipLaunchKernelGGL(add_noise_kernel<false>, dim3((unsigned)grid), dim3(256), 0, s, g, n,
                       sigma_c, inv_b, seed, tensor_id, step);
  return hipGetLastError();
}

}  // namespace dpg
