// Ghost norms from T x T Gram matrices on MFMA (gfx950).
//
// For one example i and one linear layer, the squared Frobenius norm of the
// per-example weight gradient A_i^T G_i equals <A_i A_i^T, G_i G_i^T>: expand
// the norm as sum_{t,s} (a_t . a_s)(g_t . g_s). For T = 1 this is the paper's
// outer-product identity (Sec. "Ghost Clipping Mechanism", eq. 4-5); summing
// layers gives eq. 6. The output head is the linear layer d -> V, so its norm is
// the same kernel with G = the logit gradients.
//
// Work item = (layer, example, upper-triangle T-tile pair, chunk of G features).
// A workgroup streams the rows of its two 128-row T-tiles through LDS, first
// over the features of A (Gram P) then over its chunk of G features (Gram Q),
// both accumulated by 32x32 MFMA blocks held in registers, and reduces
// sum w * P o Q in registers. No Gram ever leaves the chip. Splitting the G
// features into chunks is exact because the reduction is linear in Q; P is
// recomputed per chunk. Partials go to a [B, slots] workspace and are summed
// in a fixed order, so results are bitwise reproducible.
//
// The tied cross term <g_in,i, g_out,i> (eq. 11, eq. 13) uses the same tile
// machinery: row v of the input-embedding gradient is the sum of dE_t over the
// tokens with id v, and row v of the output-head gradient is sum_s Gz[s,v] h_s,
// so <g_in, g_out> = sum_{t,s} Gz[s, x_t] <dE_t, h_s>: one T x T product of
// dE and H on MFMA, multiplied element-wise by logit gradients gathered at the
// token ids. No V x d gradient is formed.
#include "common.hpp"
#include "kernels.hpp"

namespace dpg {

constexpr int GR_THREADS = 256;
constexpr int GR_ROWS = 2 * GR_TM;  // LDS rows of one stage (two T-tiles)

enum { PAT_OFF = 0, PAT_D1 = 1, PAT_D2 = 2 };
template <int PAT> struct PatNB;
template <> struct PatNB<PAT_OFF> { static constexpr int NB = 4; };
template <> struct PatNB<PAT_D1> { static constexpr int NB = 3; };
template <> struct PatNB<PAT_D2> { static constexpr int NB = 2; };

// 32x32 blocks a wave owns. Off-diagonal tile pair: wave w takes a 64x64
// quadrant (rows of tile ti are LDS rows 0..127, rows of tile tj are 128..255),
// every block weighted 2 (the pair stands for (ti,tj) and (tj,ti)). Diagonal
// pair: the 10 upper-triangle blocks of the 4x4 block grid, split 3/3/2/2 over
// the waves; diagonal blocks weigh 1, the others 2.
template <int PAT>
__device__ __forceinline__ void block_rows(int w, int (&ra)[4], int (&rb)[4], float (&wt)[4]) {
  if (PAT == PAT_OFF) {
    const int x = (w >> 1) * 64, y = GR_TM + (w & 1) * 64;
    ra[0] = x;      rb[0] = y;      wt[0] = 2.f;
    ra[1] = x;      rb[1] = y + 32; wt[1] = 2.f;
    ra[2] = x + 32; rb[2] = y;      wt[2] = 2.f;
    ra[3] = x + 32; rb[3] = y + 32; wt[3] = 2.f;
  } else if (PAT == PAT_D1) {  // waves 0,1: blocks (x,x) (x,y) (y,y)
    const int x = w * 64, y = x + 32;
    ra[0] = x; rb[0] = x; wt[0] = 1.f;
    ra[1] = x; rb[1] = y; wt[1] = 2.f;
    ra[2] = y; rb[2] = y; wt[2] = 1.f;
    ra[3] = 0; rb[3] = 0; wt[3] = 0.f;
  } else {  // waves 2,3: blocks (x,64) (x,96)
    const int x = (w - 2) * 32;
    ra[0] = x; rb[0] = 64; wt[0] = 2.f;
    ra[1] = x; rb[1] = 96; wt[1] = 2.f;
    ra[2] = 0; rb[2] = 0;  wt[2] = 0.f;
    ra[3] = 0; rb[3] = 0;  wt[3] = 0.f;
  }
}

// One LDS stage (64 bf16 or 32 fp32 features per row) into the NB blocks.
// Lane l supplies row l%32 of each operand and 16-byte chunk 2*ks + l/32, so
// both operands carry the same features in the same MFMA k-slots.
template <int DT, int NB>
__device__ __forceinline__ void stage_mfma(const u32x4* __restrict__ lds, const int (&ra)[4],
                                           const int (&rb)[4], f32x16 (&acc)[4], int lane) {
  const int r32 = lane & 31, half = lane >> 5;
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    const int c = 2 * ks + half;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int row_a = ra[j] + r32, row_b = rb[j] + r32;
      const u32x4 fa = lds[row_a * 8 + swz(row_a, c)];
      const u32x4 fb = lds[row_b * 8 + swz(row_b, c)];
      if constexpr (DT == DT_BF16) {
        acc[j] = mfma32_bf16(fa, fb, acc[j]);
      } else {
#pragma unroll
        for (int m = 0; m < 4; ++m)
          acc[j] = mfma32_f32(__uint_as_float(fa[m]), __uint_as_float(fb[m]), acc[j]);
      }
    }
  }
}

// Streams the rows of one or two T-tiles of a matrix pair through LDS.
// Entry i (0..7) of a thread is LDS row (tid/8) + 32*i, chunk tid%8; entries
// 0..3 are rows of T-tile ti, entries 4..7 rows of T-tile tj. Stage s < nX
// reads features [s*KS, ...) of X up to column x1; later stages read features
// [y0 + (s-nX)*KS, ...) of Y up to column y1.
template <int DT, bool VEC>
struct TileStream {
  static constexpr int EPC = (DT == DT_BF16) ? 8 : 4;
  static constexpr int KS = 8 * EPC;
  static constexpr int ES = (DT == DT_BF16) ? 2 : 4;
  const char* X;
  const char* Y;
  int64_t ldx, ldy;           // row strides in bytes
  int64_t row_i, row_j;       // global row of entry 0 (tile ti) and entry 4 (tile tj)
  int T_end_i, T_end_j;       // entries i with 32*i (+ first row) below these are valid
  int c;                      // this thread's chunk within a row
  int nX;
  int64_t x1, y0, y1;

  // VEC: rows are 16-byte aligned and their stride is a whole number of
  // chunks, so every chunk is one 16-byte load (elements past the valid
  // columns are zeroed in registers). Otherwise elements are loaded one at a
  // time.
  __device__ __forceinline__ void prefetch(int s, u32x4 (&pre)[8], int nent) const {
    const bool inX = s < nX;
    const char* base = inX ? X : Y;
    const int64_t ld = inX ? ldx : ldy;
    const int64_t col = inX ? (int64_t)s * KS + c * EPC : y0 + (int64_t)(s - nX) * KS + c * EPC;
    const int64_t ncol = inX ? x1 : y1;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const bool lo = i < 4;
      const int k = lo ? i : i - 4;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (i < nent && 32 * k < (lo ? T_end_i : T_end_j) && col < ncol) {
        const char* row = base + ((lo ? row_i : row_j) + 32 * k) * ld;
        v = VEC ? load_chunk16_masked<DT>(row, col, ncol) : load_chunk_elems<DT>(row, col, ncol);
      }
      pre[i] = v;
    }
  }
};

__device__ __forceinline__ void store_stage(u32x4* lds, const u32x4 (&pre)[8], int tid, int nent) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    if (i < nent) {
      const int r = (tid >> 3) + 32 * i, c = tid & 7;
      lds[r * 8 + swz(r, c)] = pre[i];
    }
  }
}

template <int DT, bool VEC, int PAT>
__device__ float gram_item(const GramLayer& L, int b, int T, int ti, int tj, int chunk,
                           u32x4* lds) {
  constexpr int NB = PatNB<PAT>::NB;
  using TS = TileStream<DT, VEC>;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int nent = (ti == tj) ? 4 : 8;

  TS ts;
  ts.X = (const char*)L.A;
  ts.Y = (const char*)L.G;
  ts.ldx = L.lda * TS::ES;
  ts.ldy = L.ldg * TS::ES;
  ts.c = tid & 7;
  ts.x1 = L.d_in;
  ts.y0 = (int64_t)L.g0 + (int64_t)chunk * L.kg;
  ts.y1 = ts.y0 + L.kg < L.g1 ? ts.y0 + L.kg : L.g1;
  ts.nX = (L.d_in + TS::KS - 1) / TS::KS;
  const int nY = (int)((ts.y1 - ts.y0 + TS::KS - 1) / TS::KS);
  const int r0 = tid >> 3;
  ts.row_i = (int64_t)b * T + ti * GR_TM + r0;
  ts.row_j = (int64_t)b * T + tj * GR_TM + r0;
  ts.T_end_i = T - (ti * GR_TM + r0);
  ts.T_end_j = T - (tj * GR_TM + r0);

  int ra[4], rb[4];
  float wt[4];
  block_rows<PAT>(w, ra, rb, wt);
  f32x16 accP[4], accQ[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) { accP[j][e] = 0.f; accQ[j][e] = 0.f; }

  // Features of A into P, then this chunk's features of G into Q; the
  // prefetch of stage s+1 is in flight while stage s is multiplied.
  const int n = ts.nX + nY;
  u32x4 pre[8];
  ts.prefetch(0, pre, nent);
  for (int s = 0; s < ts.nX; ++s) {
    __syncthreads();
    store_stage(lds, pre, tid, nent);
    __syncthreads();
    if (s + 1 < n) ts.prefetch(s + 1, pre, nent);
    stage_mfma<DT, NB>(lds, ra, rb, accP, lane);
  }
  for (int s = ts.nX; s < n; ++s) {
    __syncthreads();
    store_stage(lds, pre, tid, nent);
    __syncthreads();
    if (s + 1 < n) ts.prefetch(s + 1, pre, nent);
    stage_mfma<DT, NB>(lds, ra, rb, accQ, lane);
  }
  float part = 0.f;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) s += accP[j][e] * accQ[j][e];
    part += wt[j] * s;
  }
  return part;
}

template <int DT, bool VEC>
__global__ __launch_bounds__(GR_THREADS) void gram_norm_kernel(GramArgs args) {
  // Index the layer table in place in the kernel-argument segment (the only
  // explicit argument sits at offset 0) instead of copying it to the stack.
  const GramArgs& a = *(const GramArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  (void)args;
  __shared__ u32x4 lds[GR_ROWS * 8];
  __shared__ float red[GR_THREADS / WAVE];
  const uint32_t item = xcd_remap(blockIdx.x, gridDim.x);
  int l = 0;
  while (l + 1 < a.n_layers && item >= a.L[l + 1].item_begin) ++l;
  const GramLayer& L = a.L[l];
  uint32_t rel = item - L.item_begin;
  const uint32_t per_b = (uint32_t)a.P * (uint32_t)L.nc;
  const int b = (int)(rel / per_b);
  rel -= (uint32_t)b * per_b;
  const int pair = (int)(rel / (uint32_t)L.nc);
  const int chunk = (int)(rel - (uint32_t)pair * L.nc);
  int ti = 0, rem = pair;
  while (rem >= a.n_t - ti) { rem -= a.n_t - ti; ++ti; }
  const int tj = ti + rem;
  const int w = threadIdx.x >> 6;

  float part;
  if (ti != tj)
    part = gram_item<DT, VEC, PAT_OFF>(L, b, a.T, ti, tj, chunk, lds);
  else if (w < 2)
    part = gram_item<DT, VEC, PAT_D1>(L, b, a.T, ti, tj, chunk, lds);
  else
    part = gram_item<DT, VEC, PAT_D2>(L, b, a.T, ti, tj, chunk, lds);
  part = wave_sum(part);
  if ((threadIdx.x & 63) == 0) red[w] = part;
  __syncthreads();
  if (threadIdx.x == 0)
    a.ws[(int64_t)b * a.slots + L.slot_begin + pair * L.nc + chunk] =
        (red[0] + red[1]) + (red[2] + red[3]);
}

template <int DT, bool VEC>
__global__ __launch_bounds__(GR_THREADS) void tied_cross_kernel(CrossArgs a) {
  __shared__ u32x4 lds[GR_ROWS * 8];
  __shared__ float red[GR_THREADS / WAVE];
  using TS = TileStream<DT, VEC>;
  const uint32_t item = xcd_remap(blockIdx.x, gridDim.x);
  const int b = (int)(item / (uint32_t)a.slots);
  const int pair = (int)(item - (uint32_t)b * a.slots);
  const int ti = pair / a.n_t, tj = pair - ti * a.n_t;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int T = a.T;

  // LDS rows 0..127: dE rows of tile ti; rows 128..255: H rows of tile tj.
  // Both come in the same stage: "X" is dE for entries 0..3 and H for 4..7.
  constexpr int EPC = TS::EPC, KS = TS::KS, ES = TS::ES;
  const int r0 = tid >> 3, c = tid & 7;
  const int64_t row_i = (int64_t)b * T + ti * GR_TM + r0;
  const int64_t row_j = (int64_t)b * T + tj * GR_TM + r0;
  const int end_i = T - (ti * GR_TM + r0), end_j = T - (tj * GR_TM + r0);
  const char* Eb = (const char*)a.E;
  const char* Hb = (const char*)a.H;
  const int64_t lde = a.lde * ES, ldh = a.ldh * ES;
  const int nX = (a.d + KS - 1) / KS;
  int ra[4], rb[4];
  float wt[4];
  block_rows<PAT_OFF>(w, ra, rb, wt);
  f32x16 acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[j][e] = 0.f;

  const int n = nX;
  u32x4 pre[8];
  auto fetch = [&](int s) {
    const int64_t col = (int64_t)s * KS + c * EPC;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      u32x4 v = {0u, 0u, 0u, 0u};
      const bool lo = i < 4;
      const int k = lo ? i : i - 4;
      if (col < a.d && 32 * k < (lo ? end_i : end_j)) {
        const char* row = lo ? Eb + (row_i + 32 * k) * lde : Hb + (row_j + 32 * k) * ldh;
        v = VEC ? load_chunk16_masked<DT>(row, col, a.d) : load_chunk_elems<DT>(row, col, a.d);
      }
      pre[i] = v;
    }
  };
  fetch(0);
  for (int s = 0; s < n; ++s) {
    __syncthreads();
    store_stage(lds, pre, tid, 8);
    __syncthreads();
    if (s + 1 < n) fetch(s + 1);
    stage_mfma<DT, 4>(lds, ra, rb, acc, lane);
  }

  // Block j holds P[t, s] = <dE_t, H_s>: lane l has column s = l%32 and, for
  // accumulator e, row (e/4)*8 + (l/32)*4 + e%4 of the 32x32 MFMA output.
  float part = 0.f;
  const int64_t ldz = a.ldz;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int t0 = ti * GR_TM + ra[j] + (lane >> 5) * 4;
    const int s = tj * GR_TM + (rb[j] - GR_TM) + (lane & 31);
    if (s >= T) continue;
    const int64_t zrow = ((int64_t)b * T + s) * ldz;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int t = t0 + (e >> 2) * 8 + (e & 3);
      if (t < T) {
        const uint32_t v = (uint32_t)a.ids[(int64_t)b * T + t];
        if (v >= (uint32_t)a.V) continue;  // invalid id: contributes nothing
        float g;
        if constexpr (DT == DT_BF16)
          g = bf16_to_f32(((const uint16_t*)a.Gz)[zrow + v]);
        else
          g = ((const float*)a.Gz)[zrow + v];
        part += acc[j][e] * g;
      }
    }
  }
  part = wave_sum(part);
  if (lane == 0) red[w] = part;
  __syncthreads();
  if (tid == 0) a.ws[(int64_t)b * a.slots + pair] = (red[0] + red[1]) + (red[2] + red[3]);
}

// out[b] = (accumulate ? out[b] : 0) + scale * sum_j ws[b, j]; each lane sums
// a fixed stride of slots in double, then a fixed shuffle tree.
__global__ __launch_bounds__(WAVE) void finish_rows_kernel(const float* __restrict__ ws,
                                                           int slots, float* out, int accumulate,
                                                           float scale) {
  const int b = blockIdx.x, lane = threadIdx.x;
  double s = 0.0;
  for (int j = lane; j < slots; j += WAVE) s += (double)ws[(int64_t)b * slots + j];
  s = wave_sum_d(s);
  if (lane == 0) out[b] = (float)((accumulate ? (double)out[b] : 0.0) + (double)scale * s);
}

// `vec` selects the 16-byte load path; the caller sets it only when every
// operand of the launch has 16-byte aligned rows.
hipError_t launch_gram_norm(const GramArgs& a, int dt, bool vec, hipStream_t s) {
  if (a.n_items == 0) return hipSuccess;
  const dim3 g(a.n_items), blk(GR_THREADS);
  if (dt == DT_BF16) {
    if (vec) hipLaunchKernelGGL((gram_norm_kernel<DT_BF16, true>), g, blk, 0, s, a);
    else hipLaunchKernelGGL((gram_norm_kernel<DT_BF16, false>), g, blk, 0, s, a);
  } else {
    if (vec) hipLaunchKernelGGL((gram_norm_kernel<DT_F32, true>), g, blk, 0, s, a);
    else hipLaunchKernelGGL((gram_norm_kernel<DT_F32, false>), g, blk, 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_tied_cross(const CrossArgs& a, int dt, bool vec, hipStream_t s) {
  const uint32_t n = (uint32_t)a.B * (uint32_t)a.slots;
  if (n == 0) return hipSuccess;
  const dim3 g(n), blk(GR_THREADS);
  if (dt == DT_BF16) {
    if (vec) hipLaunchKernelGGL((tied_cross_kernel<DT_BF16, true>), g, blk, 0, s, a);
    else hipLaunchKernelGGL((tied_cross_kernel<DT_BF16, false>), g, blk, 0, s, a);
  } else {
    if (vec) hipLaunchKernelGGL((tied_cross_kernel<DT_F32, true>), g, blk, 0, s, a);
    else hipLaunchKernelGGL((tied_cross_kernel<DT_F32, false>), g, blk, 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_finish_rows(const float* ws, int B, int slots, float* out, int accumulate,
                              float scale, hipStream_t s) {
  if (B == 0) return hipSuccess;
  hipLaunchKernelGGL(finish_rows_kernel, dim3(B), dim3(WAVE), 0, s, ws, slots, out, accumulate,
                     scale);
  return hipGetLastError();
}

}  // namespace dpg
