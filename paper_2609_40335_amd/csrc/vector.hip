// Parameters whose per-example gradients are small enough to materialise:
// vector parameters applied to every token (a linear layer's bias, a
// LayerNorm gain or bias) and the learned position table.
//
// Chain rule: a bias enters every token's output as y_t = ... + b, so its
// per-example gradient is sum_t G[t]; a LayerNorm gain enters as
// y_t = gain * xhat_t + beta, so its gradient is sum_t xhat[t] * G[t] and the
// LayerNorm bias's is sum_t G[t]. The flat per-example norm (eq. 6) adds
// their squared norms. The position table's row t is read by token t of
// every example, so an example's gradient has rows dE[t] (its positions are
// distinct) and squared norm sum_t ||dE[t]||^2.
//
// vec_reduce_kernel streams the token rows once: work item = (parameter,
// example, chunk of 64 lanes x 16 bytes of features); four waves take every
// fourth row each, with two rows' loads in flight per wave; the per-lane
// partial sums meet in LDS. VEC_GRAD writes the example's gradient chunk
// and the chunk's squared norm; a LayerNorm's gain and bias, which share G,
// take one pass (the bias's plain sum rides along as a second output).
// VEC_SQ (the position table) only sums the squared elements, so its items
// also split the example's rows (a scalar partial per row range). Items are numbered example-major, as in the Gram
// kernel, so each XCD's contiguous item range holds whole examples.
//
// vec_sum_kernel and pos_sum_kernel form the clipped sums sum_i c_i g_i of
// the materialised gradients (or of dE for the position table) in a fixed
// order, with the Gaussian mechanism of eq. 3 fused into the store.
#include "common.hpp"
#include "kernels.hpp"

namespace dpg {

constexpr int VR_THREADS = 256;
constexpr int VR_WAVES = VR_THREADS / WAVE;
// Rows in flight per wave: two measured faster than four or eight (fewer
// requests pending at once per CU), with four or eight waves per workgroup.
constexpr int VR_UNROLL = 2;

template <int DT, bool VEC>
__device__ __forceinline__ void widen(const u32x4& v, float (&x)[DT == DT_BF16 ? 8 : 4]) {
  if constexpr (DT == DT_BF16) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      x[2 * q] = __uint_as_float(v[q] << 16);
      x[2 * q + 1] = __uint_as_float(v[q] & 0xFFFF0000u);
    }
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) x[q] = __uint_as_float(v[q]);
  }
}

template <int DT, bool VEC>
__global__ __launch_bounds__(VR_THREADS) void vec_reduce_kernel(VecArgs args) {
  const VecArgs& a = *(const VecArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  (void)args;
  constexpr int EPC = DT == DT_BF16 ? 8 : 4;   // elements per 16-byte chunk
  constexpr int ES = DT == DT_BF16 ? 2 : 4;
  __shared__ float part[VR_WAVES][WAVE * EPC];

  const uint32_t item = xcd_remap(blockIdx.x, gridDim.x);
  const int b = (int)(item / a.per_ex);
  uint32_t rel = item - (uint32_t)b * a.per_ex;
  const int pl = (int)(threadIdx.x & (WAVE - 1));
  const int p = wave_find(rel, pl < a.n_params ? a.P[pl].item_begin : 0u, a.n_params);
  const VecParam& P = a.P[p];
  const int fc = (int)((rel - P.item_begin) / (uint32_t)P.tsplit);
  const int tc = (int)((rel - P.item_begin) - (uint32_t)fc * P.tsplit);
  const int t_end = min(a.T, (tc + 1) * P.trows);
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t col = (int64_t)fc * WAVE * EPC + lane * EPC;

  const uint64_t rows = (uint64_t)a.B * a.T;
  const rsrc_t rg = make_rsrc(P.G, rows * (uint64_t)P.ldg * ES);
  const bool has_x = P.X != nullptr;
  const rsrc_t rx = make_rsrc(has_x ? P.X : P.G, rows * (uint64_t)(has_x ? P.ldx : P.ldg) * ES);
  const uint32_t ldg_b = (uint32_t)(P.ldg * ES), ldx_b = (uint32_t)((has_x ? P.ldx : 0) * ES);
  // Byte offset of (row 0 of example b, this lane's chunk); rows advance by ld.
  const uint32_t g0 = (uint32_t)(((int64_t)b * a.T * P.ldg + col) * ES);
  const uint32_t x0 = (uint32_t)(((int64_t)b * a.T * (has_x ? P.ldx : 0) + col) * ES);

  // acc: sum of x * g (or of g, or of g * g); acc2: the plain sum of g when a
  // LayerNorm's bias shares this entry's G (grad2 set).
  const bool two = P.grad2 != nullptr;
  float acc[EPC], acc2[EPC];
#pragma unroll
  for (int e = 0; e < EPC; ++e) acc[e] = acc2[e] = 0.f;
  const bool live = col < P.d;  // a chunk wholly past d loads nothing
  if (live) {
    for (int t0 = tc * P.trows + w; t0 < t_end; t0 += VR_WAVES * VR_UNROLL) {
      u32x4 gv[VR_UNROLL], xv[VR_UNROLL];
#pragma unroll
      for (int u = 0; u < VR_UNROLL; ++u) {
        const int t = t0 + u * VR_WAVES;
        // Rows past this item's rows and elements past d read as zero.
        const bool in = t < t_end;
        const uint32_t so = in ? (uint32_t)t * ldg_b : 0u;
        gv[u] = in ? buf_chunk<DT, VEC, true, CPOL_STREAM>(rg, g0, so, col, P.d)
                    : u32x4{0u, 0u, 0u, 0u};
        if (has_x && P.mode == VEC_GRAD) {
          const uint32_t sx = in ? (uint32_t)t * ldx_b : 0u;
          xv[u] = in ? buf_chunk<DT, VEC, true, CPOL_STREAM>(rx, x0, sx, col, P.d)
                      : u32x4{0u, 0u, 0u, 0u};
        }
      }
#pragma unroll
      for (int u = 0; u < VR_UNROLL; ++u) {
        float g[EPC];
        widen<DT, VEC>(gv[u], g);
        if (P.mode == VEC_SQ) {
#pragma unroll
          for (int e = 0; e < EPC; ++e) acc[e] += g[e] * g[e];
        } else if (has_x) {
          float x[EPC];
          widen<DT, VEC>(xv[u], x);
#pragma unroll
          for (int e = 0; e < EPC; ++e) acc[e] += x[e] * g[e];
          if (two) {
#pragma unroll
            for (int e = 0; e < EPC; ++e) acc2[e] += g[e];
          }
        } else {
#pragma unroll
          for (int e = 0; e < EPC; ++e) acc[e] += g[e];
        }
      }
    }
  }
  // The four waves' partial sums, added in wave order by wave 0.
  float sq = 0.f;
#pragma unroll
  for (int e = 0; e < EPC; ++e) part[w][lane * EPC + e] = acc[e];
  __syncthreads();
  if (w == 0) {
#pragma unroll
    for (int e = 0; e < EPC; ++e) {
      float v = part[0][lane * EPC + e];
#pragma unroll
      for (int q = 1; q < VR_WAVES; ++q) v += part[q][lane * EPC + e];
      if (P.mode == VEC_SQ) {
        sq += v;
      } else {
        sq += v * v;
        if (col + e < P.d) P.grad[(int64_t)b * P.d + col + e] = v;
      }
    }
  }
  if (two) {
    __syncthreads();  // wave 0 is done reading the first sums
#pragma unroll
    for (int e = 0; e < EPC; ++e) part[w][lane * EPC + e] = acc2[e];
    __syncthreads();
    if (w == 0) {
#pragma unroll
      for (int e = 0; e < EPC; ++e) {
        float v = part[0][lane * EPC + e];
#pragma unroll
        for (int q = 1; q < VR_WAVES; ++q) v += part[q][lane * EPC + e];
        sq += v * v;
        if (col + e < P.d) P.grad2[(int64_t)b * P.d + col + e] = v;
      }
    }
  }
  if (w == 0) {
    sq = wave_sum(sq);
    if (lane == 0) a.ws[(int64_t)b * a.slots + P.slot_begin + fc * P.tsplit + tc] = sq;
  }
}

// One thread per 4 consecutive features of one parameter's clipped sum:
// out[f] = (prior + sum_i c_i grad[i, f] + sigma_c z_f) * inv_b, the sum
// over examples in order. Four consecutive elements of a 1-D tensor starting
// at a multiple of 4 are one Philox block of its noise stream.
__global__ __launch_bounds__(256) void vec_sum_kernel(VecSumArgs a) {
  const uint32_t q = blockIdx.x * 256u + threadIdx.x;
  if (q >= a.n_quads) return;
  int lo = 0, hi = a.n_params - 1;  // the entry whose quads contain q
  while (lo < hi) {
    const int mid = (lo + hi + 1) / 2;
    if (a.P[mid].quad_begin <= q) lo = mid; else hi = mid - 1;
  }
  const VecSumParam& P = a.P[lo];
  const int64_t f = 4 * (int64_t)(q - P.quad_begin);
  // Examples in order; eight examples' loads are issued before their
  // products are added, so the loop is not one memory round trip per example.
  float s[4] = {0.f, 0.f, 0.f, 0.f};
  const bool vec4 = (P.d & 3) == 0 && (((uintptr_t)P.grad) & 15) == 0;
  constexpr int U = 8;
  for (int i0 = 0; i0 < a.B; i0 += U) {
    f32x4 g[U];
    float ci[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + u;
      ci[u] = i < a.B ? a.c[i] : 0.f;
      const float* gp = P.grad + (int64_t)i * P.d + f;
      if (i >= a.B) {
        g[u] = f32x4{0.f, 0.f, 0.f, 0.f};
      } else if (vec4) {
        g[u] = *(const f32x4*)gp;
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) g[u][k] = f + k < P.d ? gp[k] : 0.f;
      }
    }
    // An example with c = 0 (a non-finite norm) is left out, not multiplied
    // by zero: its gradient may hold inf or NaN.
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int k = 0; k < 4; ++k) s[k] += ci[u] != 0.f ? ci[u] * g[u][k] : 0.f;
  }
  float z[4] = {0.f, 0.f, 0.f, 0.f};
  if (a.noise) gauss4((uint64_t)f >> 2, a.seed, P.tensor_id, a.step, z);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (f + k >= P.d) break;
    float v = s[k];
    if (a.noise) v += a.sigma_c * z[k];
    if (P.accumulate) v += P.out[f + k];
    if (a.noise) v *= a.inv_b;
    P.out[f + k] = v;
  }
}

// The position table's clipped sum: one thread per 4 consecutive features of
// one row t: out[t, f] = (prior + [t < T] sum_i c_i dE[i, t, f] + sigma_c z)
// * inv_b, the noise element of (t, f) being t*d + f of the table's stream.
template <int DT>
__global__ __launch_bounds__(256) void pos_sum_kernel(PosSumArgs a) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t qpr = (a.d + 3) / 4;  // quads per row
  if (q >= (int64_t)a.n_pos * qpr) return;
  const int t = (int)(q / qpr);
  const int64_t f = 4 * (q - (int64_t)t * qpr);
  float s[4] = {0.f, 0.f, 0.f, 0.f};
  constexpr int ES = DT == DT_BF16 ? 2 : 4;
  const bool vec4 = f + 4 <= a.d && (a.lde & 3) == 0 && (((uintptr_t)a.E) & (4 * ES - 1)) == 0;
  if (t < a.T) {
    constexpr int U = 8;  // examples whose loads are in flight together
    for (int i0 = 0; i0 < a.B; i0 += U) {
      float e[U][4], ci[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = i0 + u;
        ci[u] = i < a.B ? a.c[i] : 0.f;
        const int64_t at = ((int64_t)i * a.T + t) * a.lde + f;  // element (i, t, f)
        if (i >= a.B) {
#pragma unroll
          for (int k = 0; k < 4; ++k) e[u][k] = 0.f;
        } else if (vec4) {  // the 4 elements in one 8- (bf16) or 16-byte (fp32) load
          if constexpr (DT == DT_BF16) {
            const uint2 w = *(const uint2*)((const uint16_t*)a.E + at);
            e[u][0] = __uint_as_float(w.x << 16); e[u][1] = __uint_as_float(w.x & 0xFFFF0000u);
            e[u][2] = __uint_as_float(w.y << 16); e[u][3] = __uint_as_float(w.y & 0xFFFF0000u);
          } else {
            const f32x4 w = *(const f32x4*)((const float*)a.E + at);
#pragma unroll
            for (int k = 0; k < 4; ++k) e[u][k] = w[k];
          }
        } else {
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            if (f + k < a.d) {
              if constexpr (DT == DT_BF16)
                e[u][k] = bf16_to_f32(((const uint16_t*)a.E)[at + k]);
              else
                e[u][k] = ((const float*)a.E)[at + k];
            } else {
              e[u][k] = 0.f;
            }
          }
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int k = 0; k < 4; ++k) s[k] += ci[u] != 0.f ? ci[u] * e[u][k] : 0.f;  // c = 0: left out
    }
  }
  float* o = a.out + (int64_t)t * a.ldo + f;
  const uint64_t j0 = (uint64_t)t * (uint64_t)a.d + (uint64_t)f;
  float z[4] = {0.f, 0.f, 0.f, 0.f};
  const bool one_block = (j0 & 3) == 0;
  if (a.noise && one_block) gauss4(j0 >> 2, a.seed, a.tensor_id, a.step, z);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (f + k >= a.d) break;
    float v = s[k];
    if (a.noise) {
      float zk = z[k];
      if (!one_block) {  // the row length is not a multiple of 4
        float zz[4];
        const uint64_t j = j0 + k;
        gauss4(j >> 2, a.seed, a.tensor_id, a.step, zz);
        const int r = (int)(j & 3);
        zk = r == 0 ? zz[0] : r == 1 ? zz[1] : r == 2 ? zz[2] : zz[3];
      }
      v += a.sigma_c * zk;
    }
    if (a.accumulate) v += o[k];
    if (a.noise) v *= a.inv_b;
    o[k] = v;
  }
}

hipError_t launch_vec_reduce(const VecArgs& a, int dt, bool vec, hipStream_t s) {
  if (a.n_items == 0) return hipSuccess;
  const dim3 g(a.n_items), blk(VR_THREADS);
  if (dt == DT_BF16) {
    if (vec) hipLaunchKernelGGL((vec_reduce_kernel<DT_BF16, true>), g, blk, 0, s, a);
    else hipLaunchKernelGGL((vec_reduce_kernel<DT_BF16, false>), g, blk, 0, s, a);
  } else {
    if (vec) hipLaunchKernelGGL((vec_reduce_kernel<DT_F32, true>), g, blk, 0, s, a);
    else hipLaunchKernelGGL((vec_reduce_kernel<DT_F32, false>), g, blk, 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_vec_sum(const VecSumArgs& a, hipStream_t s) {
  if (a.n_quads == 0) return hipSuccess;
  hipLaunchKernelGGL(vec_sum_kernel, dim3((a.n_quads + 255) / 256), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_pos_sum(const PosSumArgs& a, int dt, hipStream_t s) {
  const int64_t n = (int64_t)a.n_pos * ((a.d + 3) / 4);
  if (n == 0) return hipSuccess;
  const dim3 g((uint32_t)((n + 255) / 256)), blk(256);
  if (dt == DT_BF16) hipLaunchKernelGGL(pos_sum_kernel<DT_BF16>, g, blk, 0, s, a);
  else hipLaunchKernelGGL(pos_sum_kernel<DT_F32>, g, blk, 0, s, a);
  return hipGetLastError();
}

}  // namespace dpg
