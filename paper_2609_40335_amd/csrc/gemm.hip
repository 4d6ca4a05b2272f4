// GEMMs whose two operands are both stored token-major: X [K, M] and Y [K, N]
// with the contraction index k (a token of an example) on the rows.
//
// Clipped sum (eq. 3 without the noise; the reweighted second backward of
// Sec. "Ghost Clipping Mechanism"): S = sum_i c_i A_i^T G_i. Stacking the B
// examples' tokens gives one GEMM with K = B*T in which row k of X is scaled
// by c[k / T]. The backward pass is linear in the upstream gradient, so this
// equals the gradient of the loss reweighted by the clip factors.
//
// Direct norm (the materialising alternative, "normal clipping" of Sec.
// "Training Configurations"): ||A_i^T G_i||_F^2 per example, from the same
// GEMM restricted to the example's T rows; each 256x256 output tile is
// squared and summed in registers at the example's last row. A work item of
// the direct-load kernel covers a run of consecutive examples of one tile.
// Optionally each example's tile is also written to a gradient store, from
// which store_sum_kernel forms the clipped sums as weighted sums of the
// stored tiles instead of a second GEMM. The direct form beats the Gram form
// when T + 1 exceeds about R * 2 d_in d_out / (d_in + d_out), R the measured
// ratio of the two kernels' throughputs (about 0.4 to 0.5).
//
// Kernels. dl_gemm_kernel (bf16, 16-byte rows, whole 32-row stages per
// example: the clipped sum and the direct norm) loads rows straight into LDS
// and transposes on the way out of LDS; split_fixup_kernel finishes the tiles
// of its split tail. The general kernel kt_gemm_kernel (fp32, unaligned
// strides, any T) stages through registers:
//
// MFMA wants 8 consecutive k per lane, but both operands are contiguous along
// M/N. Each staging thread loads an 8(k) x 8(m) block with 16-byte buffer
// loads, scales it (X only: exact widening, fp32 multiply,
// v_cvt_pk_bf16_f32 rounding) and transposes it in registers into 8
// k-contiguous chunks written to LDS. Waves 0-3 stage X, waves 4-7 stage Y.
// Tile 256x256, 64 (bf16) or 32 (fp32) k per stage, LDS double-buffered with
// one barrier per stage; each of the 8 waves owns a 128x64 quadrant of 4x2
// 32x32 MFMA blocks, so two waves share every SIMD.
#include "common.hpp"
#include "kernels.hpp"

namespace dpg {

constexpr int GM_THREADS = 512;

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

enum { MODE_SUM = 0, MODE_NORM = 1 };

// Two bf16 held in one dword, each multiplied by s in fp32 and rounded back
// to bf16 (round to nearest even).
__device__ __forceinline__ uint32_t scale_bf16x2(uint32_t w, float s) {
  f32x2 v = {__uint_as_float(w << 16) * s, __uint_as_float(w & 0xFFFF0000u) * s};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

template <int DT>
struct KT {
  static constexpr int RPT = (DT == DT_BF16) ? 8 : 4;  // k rows per thread per stage
  static constexpr int KS = 8 * RPT;                   // k rows per stage
  static constexpr int ES = (DT == DT_BF16) ? 2 : 4;
  static constexpr int EPC = 16 / ES;                  // elements per 16-byte chunk
  static constexpr int CPR = 8 / RPT;                  // chunks per 8-column segment
};

// This thread's block of one operand: rows r0 .. r0+RPT-1 (r0 relative to
// the stage) at columns col .. col+7. voff is this lane's byte offset of
// (r0, col) and soff the wave-uniform byte offset of the stage's first row.
// ROWMASK: rows at or past `rows_left` (counted from the stage start) read
// as zero (they belong to the next example).
template <int DT, bool VEC, bool MASKC, bool ROWMASK>
__device__ __forceinline__ void load_block(rsrc_t r, uint32_t voff, uint32_t soff,
                                           uint32_t ld_bytes, int r0, int64_t rows_left,
                                           int64_t col, int64_t ncol, u32x4 (&raw)[8]) {
  using P = KT<DT>;
#pragma unroll
  for (int j = 0; j < P::RPT; ++j) {
#pragma unroll
    for (int h = 0; h < P::CPR; ++h) {
      u32x4 v = buf_chunk<DT, VEC, MASKC>(r, voff + h * 16, soff + j * ld_bytes,
                                          col + h * P::EPC, ncol);
      if (ROWMASK && r0 + j >= rows_left) v = u32x4{0u, 0u, 0u, 0u};
      raw[j * P::CPR + h] = v;
    }
  }
}

// Scales row j of the block by s[j], transposes it into 8 column chunks of
// RPT consecutive k, and writes them to LDS rows m_row0 .. m_row0+7, chunk kg.
template <int DT, bool SCALE>
__device__ __forceinline__ void store_block_t(u32x4* lds, u32x4 (&raw)[8], const float (&s)[8],
                                              int m_row0, int kg) {
  if constexpr (DT == DT_BF16) {
    if (SCALE) {
#pragma unroll
      for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int p = 0; p < 4; ++p) raw[j][p] = scale_bf16x2(raw[j][p], s[j]);
    }
#pragma unroll
    for (int mm = 0; mm < 8; ++mm) {
      const int p = mm >> 1;
      const uint32_t sel = (mm & 1) ? 0x07060302u : 0x05040100u;
      u32x4 o;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        o[q] = __builtin_amdgcn_perm(raw[2 * q + 1][p], raw[2 * q][p], sel);
      const int r = m_row0 + mm;
      lds[r * 8 + swz(r, kg)] = o;
    }
  } else {
#pragma unroll
    for (int mm = 0; mm < 8; ++mm) {
      const int h = mm >> 2, e = mm & 3;
      u32x4 o;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float v = __uint_as_float(raw[j * 2 + h][e]);
        if (SCALE) v *= s[j];
        o[j] = __float_as_uint(v);
      }
      const int r = m_row0 + mm;
      lds[r * 8 + swz(r, kg)] = o;
    }
  }
}

// One LDS stage into this wave's 4x2 blocks: X rows wm*128 + i*32, Y rows
// wn*64 + j*32. Lane l supplies row l%32 and 16-byte chunk 2*ks + l/32.
template <int DT>
__device__ __forceinline__ void tile_mfma(const u32x4* __restrict__ Xs, const u32x4* __restrict__ Ys,
                                          f32x16 (&acc)[4][2], int wm, int wn, int lane) {
  const int r32 = lane & 31, half = lane >> 5;
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    const int c = 2 * ks + half;
    u32x4 xa[4], yb[2];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int rx = wm * 128 + i * 32 + r32;
      xa[i] = Xs[rx * 8 + swz(rx, c)];
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int ry = wn * 64 + j * 32 + r32;
      yb[j] = Ys[ry * 8 + swz(ry, c)];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        if constexpr (DT == DT_BF16) {
          acc[i][j] = mfma32_bf16(xa[i], yb[j], acc[i][j]);
        } else {
#pragma unroll
          for (int m = 0; m < 4; ++m)
            acc[i][j] = mfma32_f32(__uint_as_float(xa[i][m]), __uint_as_float(yb[j][m]), acc[i][j]);
        }
      }
  }
}

// Tile (mt, nt) of work item rel within a layer: the direction with fewer
// tiles varies fastest, so consecutive items (which run side by side on one
// XCD) share a tile of the operand that has more of them in L2.
__device__ __forceinline__ void tile_of(const GemmLayer& L, uint32_t rel, int& mt, int& nt) {
  if (L.tn <= L.tm) {
    mt = (int)(rel / (uint32_t)L.tn);
    nt = (int)(rel - (uint32_t)mt * L.tn);
  } else {
    nt = (int)(rel / (uint32_t)L.tm);
    mt = (int)(rel - (uint32_t)nt * L.tm);
  }
}

// Writes (or adds) one 256x256 output tile: each wave's 4x2 32x32 blocks at
// rows m0 + wm*128 + i*32, columns n0 + wn*64 + j*32. In a 32x32 block, lane l
// holds column l%32 and, for accumulator e, row (e/4)*8 + (l/32)*4 + e%4.
// Stores bypass L2 residency (the output is written once) so that they do
// not evict operand rows.
//
// With the Gaussian mechanism fused (a.noise): value = (prior + sum +
// sigma_c * z) * inv_b, where z is the standard normal the noise generator
// assigns to the element's row-major index in the output tensor (row length
// M when transposed, N otherwise), i.e. the draw dp_add_noise would add to
// that element. In the transposed layout a lane's 4 accumulators e = 4g..4g+3
// are 4 consecutive elements of one output row starting at a multiple of 4,
// so one Philox block serves them when the row length is a multiple of 4.
__device__ __forceinline__ float noise_at(const GemmArgs& a, uint32_t tid, uint64_t j) {
  float z[4];
  gauss4(j >> 2, a.seed, tid, a.step, z);
  const int q = (int)(j & 3);
  return q == 0 ? z[0] : q == 1 ? z[1] : q == 2 ? z[2] : z[3];
}

__device__ __forceinline__ void store_tile(const GemmArgs& a, const GemmLayer& L, int64_t m0,
                                           int64_t n0, int wm, int wn, int lane,
                                           f32x16 (&acc)[4][2], bool transposed) {
  float* out = L.out;
  const int64_t ldo = L.ldo;
  const bool accum = L.accumulate != 0;
  const bool noise = a.noise != 0;
  const uint32_t tid = L.tensor_id;
  const int mw = (int)m0 + wm * 128 + (lane >> 5) * 4;  // row of e = 0 in block i = 0
  const int nw = (int)n0 + wn * 64 + (lane & 31);         // column in block j = 0
  const bool full = m0 + GM_BM <= L.M && n0 + GM_BN <= L.N;
  if (transposed) {
    // out[n][m]: the 4 accumulators e = 4g..4g+3 are 4 consecutive rows m.
    const bool vec4 = full && (ldo & 3) == 0 && (((uintptr_t)out) & 15) == 0 &&
                      (!noise || (L.M & 3) == 0);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int n = nw + j * 32;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int m = mw + i * 32 + g * 8;
          float* p = out + (int64_t)n * ldo + m;
          if (vec4) {
            f32x4 v = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                       acc[i][j][4 * g + 3]};
            if (accum) v += *(const f32x4*)p;
            if (noise) {
              float z[4];
              gauss4(((uint64_t)n * (uint64_t)L.M + (uint64_t)m) >> 2, a.seed, tid, a.step, z);
#pragma unroll
              for (int r = 0; r < 4; ++r) v[r] = (v[r] + a.sigma_c * z[r]) * a.inv_b;
            }
            __builtin_nontemporal_store(v, (f32x4*)p);
          } else if (n < L.N) {
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (m + r < L.M) {
                float v = (accum ? p[r] : 0.f) + acc[i][j][4 * g + r];
                if (noise)
                  v = (v + a.sigma_c * noise_at(a, tid, (uint64_t)n * (uint64_t)L.M + m + r)) *
                      a.inv_b;
                p[r] = v;
              }
          }
        }
      }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int n = nw + j * 32;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int m = mw + i * 32 + (e >> 2) * 8 + (e & 3);
          float* p = out + (int64_t)m * ldo + n;
          if (full || (m < L.M && n < L.N)) {
            float v = (accum ? *p : 0.f) + acc[i][j][e];
            if (noise)
              v = (v + a.sigma_c * noise_at(a, tid, (uint64_t)m * (uint64_t)L.N + n)) * a.inv_b;
            if (full) __builtin_nontemporal_store(v, p);
            else *p = v;
          }
        }
      }
  }
}

// Row-major store of one tile through LDS, for the non-transposed layout
// (the host orders every launch so that the kernel's rows are the output's
// rows). Each wave copies one 32x32 block at a time into its own 32 x 36
// float slice of LDS (MFMA layout in: lane l writes column l%32 of its 16
// rows), then reads it back as float4s of 4 consecutive columns: lane l takes
// row l/8 + 8*it, columns 4*(l%8) .. +3, so 8 lanes store 128 contiguous bytes
// of a row and every float4 is one Philox block of the output tensor (when
// the row length is a multiple of 4) for the fused Gaussian mechanism.
constexpr int EP_LD = 36;  // floats per LDS row of a block (16-byte aligned rows, fewer conflicts)

__device__ __forceinline__ void store_tile_rows(const GemmArgs& a, const GemmLayer& L, int64_t m0,
                                                int64_t n0, int wm, int wn, int lane,
                                                f32x16 (&acc)[4][2], float* slice) {
  float* out = L.out;
  const int64_t ldo = L.ldo;
  const bool accum = L.accumulate != 0;
  const bool noise = a.noise != 0;
  const uint32_t tid = L.tensor_id;
  const bool full = m0 + GM_BM <= L.M && n0 + GM_BN <= L.N;
  const bool vec = full && (ldo & 3) == 0 && (((uintptr_t)out) & 15) == 0 && (L.N & 3) == 0;
  const int rw = (lane >> 5) * 4;  // row of e = 0 within a block
  const int cw = lane & 31;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
#pragma unroll
      for (int e = 0; e < 16; ++e) slice[(rw + (e >> 2) * 8 + (e & 3)) * EP_LD + cw] = acc[i][j][e];
      const int64_t mb = m0 + wm * 128 + i * 32, nb = n0 + wn * 64 + j * 32;
      // The block's 4 float4s per lane: prior values (when accumulating) are
      // requested first and the noise is drawn while they are in flight.
      const int c4 = 4 * (lane & 7);
      const int64_t n = nb + c4;
      f32x4 v[4], prior[4];
#pragma unroll
      for (int it = 0; it < 4; ++it) {
        const int r = (lane >> 3) + 8 * it;
        v[it] = *(const f32x4*)(slice + r * EP_LD + c4);
      }
      if (vec) {
        if (accum) {
#pragma unroll
          for (int it = 0; it < 4; ++it)
            prior[it] = *(const f32x4*)(out + (mb + (lane >> 3) + 8 * it) * ldo + n);
        }
        if (noise) {
#pragma unroll
          for (int it = 0; it < 4; ++it) {
            const int64_t m = mb + (lane >> 3) + 8 * it;
            float z[4];
            gauss4(((uint64_t)m * (uint64_t)L.N + (uint64_t)n) >> 2, a.seed, tid, a.step, z);
#pragma unroll
            for (int q = 0; q < 4; ++q) v[it][q] += a.sigma_c * z[q];
          }
        }
#pragma unroll
        for (int it = 0; it < 4; ++it) {
          const int64_t m = mb + (lane >> 3) + 8 * it;
          f32x4 x = v[it];
          if (accum) x += prior[it];
          if (noise) x *= a.inv_b;
          __builtin_nontemporal_store(x, (f32x4*)(out + m * ldo + n));
        }
      } else {
#pragma unroll
        for (int it = 0; it < 4; ++it) {
          const int64_t m = mb + (lane >> 3) + 8 * it;
          if (m >= L.M) continue;
          float* p = out + m * ldo + n;
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (n + q < L.N) {
              float x = (accum ? p[q] : 0.f) + v[it][q];
              if (noise)
                x = (x + a.sigma_c * noise_at(a, tid, (uint64_t)m * (uint64_t)L.N + n + q)) *
                    a.inv_b;
              p[q] = x;
            }
        }
      }
    }
}

// A raw 256 x 256 partial tile, row-major, staged through LDS like
// store_tile_rows (8 lanes write 128 contiguous bytes of a row). Plain
// stores, unlike the output's: the fix-up launch right after reads the
// partials back, partly from the caches (its launch 1-2 % shorter at the
// tied head than with the streaming hint).
__device__ __forceinline__ void store_partial(float* dst, int wm, int wn, int lane,
                                              f32x16 (&acc)[4][2], float* slice) {
  const int rw = (lane >> 5) * 4, cw = lane & 31, c4 = 4 * (lane & 7);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
#pragma unroll
      for (int e = 0; e < 16; ++e) slice[(rw + (e >> 2) * 8 + (e & 3)) * EP_LD + cw] = acc[i][j][e];
      const int mb = wm * 128 + i * 32, nb = wn * 64 + j * 32;
#pragma unroll
      for (int it = 0; it < 4; ++it) {
        const int r = (lane >> 3) + 8 * it;
        const f32x4 v = *(const f32x4*)(slice + r * EP_LD + c4);
        *(f32x4*)(dst + (mb + r) * GM_BN + nb + c4) = v;
      }
    }
}

// The split tail tiles: one thread per 4 consecutive elements of a row of
// one tile; the ksplit partials are added in order, then the prior, the
// noise and the division as in store_tile_rows.
__global__ __launch_bounds__(256) void split_fixup_kernel(GemmArgs args) {
  const GemmArgs& a = *(const GemmArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  (void)args;
  constexpr int QPT = GM_BM * GM_BN / 4;            // float4s per tile
  const uint32_t t = blockIdx.x / (QPT / 256);      // split tile
  const int q = (int)(blockIdx.x - t * (QPT / 256)) * 256 + (int)threadIdx.x;
  const uint32_t tile = a.n_full + t;
  const int ln = (int)(threadIdx.x & (WAVE - 1));
  const int l = wave_find(tile, ln < a.n_layers ? a.L[ln].tile_begin : 0u, a.n_layers);
  const GemmLayer& L = a.L[l];
  int mt, nt;
  tile_of(L, tile - L.tile_begin, mt, nt);
  const int r = q / (GM_BN / 4), c4 = (q - r * (GM_BN / 4)) * 4;
  const int64_t m = (int64_t)mt * GM_BM + r, n = (int64_t)nt * GM_BN + c4;
  if (m >= L.M || n >= L.N) return;
  f32x4 v = {0.f, 0.f, 0.f, 0.f};
  const float* src = a.part + (size_t)t * a.ksplit * (GM_BM * GM_BN) + r * GM_BN + c4;
  for (int k = 0; k < a.ksplit; ++k) v += *(const f32x4*)(src + (size_t)k * (GM_BM * GM_BN));
  float* p = L.out + m * L.ldo + n;
  const bool accum = L.accumulate != 0, noise = a.noise != 0;
  const bool vec = n + 4 <= L.N && (L.N & 3) == 0 && (L.ldo & 3) == 0 &&
                   (((uintptr_t)L.out) & 15) == 0;
  if (vec) {
    if (noise) {
      float z[4];
      gauss4(((uint64_t)m * (uint64_t)L.N + (uint64_t)n) >> 2, a.seed, L.tensor_id, a.step, z);
#pragma unroll
      for (int k = 0; k < 4; ++k) v[k] += a.sigma_c * z[k];
    }
    if (accum) v += *(const f32x4*)p;
    if (noise) v *= a.inv_b;
    *(f32x4*)p = v;
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (n + k < L.N) {
        float x = (accum ? p[k] : 0.f) + v[k];
        if (noise)
          x = (x + a.sigma_c * noise_at(a, L.tensor_id, (uint64_t)m * (uint64_t)L.N + n + k)) *
              a.inv_b;
        p[k] = x;
      }
  }
}

// Scaling of the clipped sum: SC_NONE (direct norm), SC_STAGE (rows scaled
// while staged, any T; rows of examples with c = 0 zeroed in both operands),
// SC_ACC (every stage lies inside one example, so the fp32 accumulators are
// rescaled by c_prev / c_next at example boundaries and by the last factor at
// the end; examples with c = 0 are skipped). Either way an example with
// c = 0 contributes nothing, even where its rows hold inf or NaN.
enum { SC_NONE = 0, SC_STAGE = 1, SC_ACC = 2 };

template <int DT, bool VEC, int MODE, int SC>
__global__ __launch_bounds__(GM_THREADS) void kt_gemm_kernel(GemmArgs args) {
  // Index the layer table in place in the kernel-argument segment.
  const GemmArgs& a = *(const GemmArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  (void)args;
  using P = KT<DT>;
  __shared__ u32x4 Xs[2][GM_BM * 8];
  __shared__ u32x4 Ys[2][GM_BN * 8];
  __shared__ float red[GM_THREADS / WAVE];

  const uint32_t item = xcd_remap(blockIdx.x, gridDim.x);
  const int ln = (int)(threadIdx.x & (WAVE - 1));
  const int l = wave_find(item, ln < a.n_layers ? a.L[ln].tile_begin : 0u, a.n_layers);
  const GemmLayer& L = a.L[l];
  uint32_t rel = item - L.tile_begin;
  const uint32_t ntile = (uint32_t)L.tm * (uint32_t)L.tn;
  const int64_t K = (int64_t)a.B * a.T;
  int b = 0;
  int64_t k_begin = 0, k_end = K;
  if (MODE == MODE_NORM) {
    b = (int)(rel / ntile);
    rel -= (uint32_t)b * ntile;
    k_begin = (int64_t)b * a.T;
    k_end = k_begin + a.T;
  }
  int mt, nt;
  tile_of(L, rel, mt, nt);
  const int64_t m0 = (int64_t)mt * GM_BM;
  const int64_t n0 = (int64_t)nt * GM_BN;

  // The wave index goes through readfirstlane so that everything derived
  // from it (staging role, buffer resource) is known to be wave-uniform.
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = w & 1, wn = w >> 1;
  // staging role: waves 0..3 stage X, waves 4..7 stage Y
  const bool stage_x = w < 4;
  const int st = tid & 255, kg = st >> 5, mg = st & 31;
  const uint32_t ld_bytes = (uint32_t)((stage_x ? L.ldx : L.ldy) * P::ES);
  const rsrc_t rsrc = make_rsrc(stage_x ? L.X : L.Y, (uint64_t)K * ld_bytes);
  const int64_t col = (stage_x ? m0 : n0) + mg * 8;
  const int64_t ncol = stage_x ? L.M : L.N;
  const int r0 = kg * P::RPT;                       // this thread's first row in a stage
  const uint32_t voff = (uint32_t)(r0 * ld_bytes + col * P::ES);
  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const int nS = (int)((k_end - k_begin + P::KS - 1) / P::KS);
  const double invT = 1.0 / (double)a.T;
  float sc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) sc[j] = 1.f;
  // Issues the global loads of stage s into r; with SC_STAGE also fetches
  // the clip factors of this thread's rows.
  auto load = [&](int s, u32x4 (&r)[8]) {
    const int64_t ks0 = k_begin + (int64_t)s * P::KS;   // first row of the stage
    // Rows past the matrix read as zero through the buffer bounds; columns
    // past M/N only feed output rows that are never stored, except in the
    // direct norm, whose tile sum must not see them (nor the next example).
    load_block<DT, VEC, MODE == MODE_NORM, MODE == MODE_NORM>(
        rsrc, voff, (uint32_t)(ks0 * ld_bytes), ld_bytes, r0, k_end - ks0, col, ncol, r);
    if (SC == SC_STAGE) {
#pragma unroll
      for (int j = 0; j < P::RPT; ++j) {
        int64_t e = (int64_t)(((double)(ks0 + r0 + j) + 0.5) * invT);
        e = e < a.B ? e : a.B - 1;
        sc[j] = a.c[e];
        // An example with c = 0 (a non-finite norm) is left out of the sum:
        // its rows are zeroed in both operands (0 * inf would be NaN).
        if (sc[j] == 0.f) {
#pragma unroll
          for (int h = 0; h < P::CPR; ++h) r[j * P::CPR + h] = u32x4{0u, 0u, 0u, 0u};
        }
      }
    }
  };
  auto stage = [&](int buf, u32x4 (&r)[8]) {
    if (stage_x)
      store_block_t<DT, SC == SC_STAGE>(Xs[buf], r, sc, mg * 8, kg);
    else
      store_block_t<DT, false>(Ys[buf], r, sc, mg * 8, kg);
  };

  // SC_ACC bookkeeping (wave-uniform): factor of the accumulated examples.
  // The factor of the next example is fetched one example ahead so that no
  // stage waits on it.
  const int spe = (SC == SC_ACC) ? a.T / P::KS : 1;  // stages per example
  float c_acc = 0.f;                                  // 0: nothing accumulated yet
  float c_next = (SC == SC_ACC) ? a.c[0] : 0.f;
  bool skip = false;
  auto compute = [&](int s, int buf) {
    if constexpr (SC == SC_ACC) {
      if (s % spe == 0) {
        const int e = s / spe;
        const float ce = c_next;
        if (e + 1 < a.B) c_next = a.c[e + 1];
        skip = !(ce != 0.f);
        if (!skip) {
          if (c_acc != 0.f) {
            const float f = c_acc / ce;
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
              for (int j = 0; j < 2; ++j) acc[i][j] *= f;
          }
          c_acc = ce;
        }
      }
      if (skip) return;
    }
    tile_mfma<DT>(Xs[buf], Ys[buf], acc, wm, wn, lane);
  };

  if constexpr (SC == SC_ACC) {
    // Two register sets: the loads of stage s+2 are in flight while stage s
    // is multiplied and stage s+1 is transposed into the other LDS buffer.
    // The scheduling fences keep each phase's instructions in place so that
    // the compiler does not hoist loads across phases (which costs registers).
    u32x4 rA[8], rB[8];
    load(0, rA);
    if (nS > 1) load(1, rB);
    stage(0, rA);
    __syncthreads();
    for (int s = 0; s < nS; s += 2) {
      if (s + 2 < nS) load(s + 2, rA);
      __builtin_amdgcn_sched_barrier(0);
      compute(s, 0);
      __builtin_amdgcn_sched_barrier(0);
      if (s + 1 < nS) stage(1, rB);
      __syncthreads();
      if (s + 1 >= nS) break;
      if (s + 3 < nS) load(s + 3, rB);
      __builtin_amdgcn_sched_barrier(0);
      compute(s + 1, 1);
      __builtin_amdgcn_sched_barrier(0);
      if (s + 2 < nS) stage(0, rA);
      __syncthreads();
    }
  } else {
    // One register set (these variants need more registers per stage): the
    // loads of stage s+1 are in flight while stage s is multiplied.
    u32x4 rA[8];
    load(0, rA);
    stage(0, rA);
    __syncthreads();
    for (int s = 0; s < nS; ++s) {
      const int buf = s & 1;
      if (s + 1 < nS) load(s + 1, rA);
      compute(s, buf);
      if (s + 1 < nS) stage(buf ^ 1, rA);
      __syncthreads();
    }
  }
  if constexpr (SC == SC_ACC) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] *= c_acc;
  }

  if constexpr (MODE == MODE_SUM) {
    store_tile(a, L, m0, n0, wm, wn, lane, acc, a.transpose != 0);
  } else {
    float part = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) part += acc[i][j][e] * acc[i][j][e];
    part = wave_sum(part);
    if (lane == 0) red[w] = part;
    __syncthreads();
    if (tid == 0) {
      float t = 0.f;
#pragma unroll
      for (int q = 0; q < GM_THREADS / WAVE; ++q) t += red[q];
      a.ws[(int64_t)b * a.slots + L.slot_begin + rel] = t;
    }
  }
}

// ---------------------------------------------------------------------------
// Direct-load kernel for the bf16 clipped sum and direct norm (16-byte
// aligned rows, T a multiple of 32; B <= 4096 for the clipped sum's factor
// table): no staging through VGPRs at all.
//
// Global rows go straight into LDS through buffer loads that write LDS
// (each lane's 16 bytes land at M0 + 16*lane), so LDS keeps the token-major
// layout: stage row r = token, 256 features = 32 chunks of 16 bytes, chunk c
// stored at physical chunk c ^ dl_sw(r). The MFMA fragments (8 consecutive k
// of one column per lane) come out of LDS through the transposing read
// ds_read_b64_tr_b16, which gathers 4 rows x 4 columns per 16-lane group:
// two such reads give one 32x32x16 operand. With the swizzle the 16 chunks a
// half-wave touches fall in 16 distinct bank groups.
//
// Ring of 4 stages of 32 k (32 KB each: X then Y), worked in ping-pong by
// two groups of four waves, one wave of each group per SIMD: while one group
// issues a stage's 16 MFMAs (at raised wave priority), the other reads the
// next stage's fragments out of LDS, issues its share of a later stage's
// loads and, at an example boundary, rescales its accumulators; a barrier
// swaps the roles. So each SIMD always has one wave feeding its matrix core
// and one wave doing everything else, and the VALU work of the rescale runs
// beside the other group's MFMAs. Group 0 (waves 0-3, the X loaders)
// computes stage s in phase 2s and reads stage s+1 in phase 2s+1; group 1
// (waves 4-7, the Y loaders) reads stage s in phase 2s and computes it in
// phase 2s+1. Stage s's slot is free once phase 2s ends: group 0 refills it
// with stage s+4 in phase 2s+1, and group 1 refills the slot of stage s-1
// with stage s+3 in phase 2s. Every wave waits for its own loads of stage
// s+1 at the end of phase 2s, so the barrier that ends the phase certifies
// that stage s+1 has landed. Every phase issues the same 4 loads per wave
// (stages past the end read zeros through the range check into a slot that
// is never read again), so the wait counts are constants.
//
// The loads are issued from inline assembly: the compiler would otherwise
// treat every later LDS read as possibly aliasing an LDS-writing load and
// drain all of them (vmcnt(0)) before it, serialising the ring. Its wait
// bookkeeping stays sound: untracked loads only make its own waits stricter.
// Clip factors are staged in LDS so that the loop issues no other vector
// memory instruction; each is read one example ahead, so that a rescale never
// waits behind the fragment reads. Scaling is on the fp32 accumulators as in
// SC_ACC. In the direct norm the example boundary instead squares and sums
// each wave's part of the tile (and writes the tile to the gradient store,
// if there is one), then clears the accumulators for the next example.
constexpr int DL_BK = DL_SUM_BK;            // k rows per stage
constexpr int DL_NS = 4;                    // stages in the ring
constexpr int DL_ROWB = GM_BM * 2;          // bytes per LDS row (256 bf16)
constexpr int DL_OPB = DL_BK * DL_ROWB;     // one operand's stage: 16 KB
constexpr int DL_STB = 2 * DL_OPB;          // one stage: X then Y
constexpr int DL_MAXB = DL_SUM_MAXB;        // clip factors held in LDS
constexpr int DL_LOADS = 4;                 // loads per wave per stage
static_assert(GM_BM == GM_BN, "square tiles");
static_assert(DL_STB == (GM_THREADS / WAVE) * DL_LOADS * 1024, "one KB per load");
static_assert(NG_MAX * (GM_THREADS / WAVE) <= DL_MAXB, "direct norm: a part per example and wave fits the factor table");
static_assert((GM_THREADS / WAVE) * 32 * EP_LD * 4 <= DL_NS * DL_STB, "epilogue slices fit the ring");

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(3))) char lds_char_t;
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4_t;

// Physical chunk of chunk c in stage row r is c ^ dl_sw(r). The 4 rows read
// together are r = 4a..4a+3; dl_sw maps them to 0, 6, 12, 10, whose bits 1-2
// and bits 2-3 are both all distinct, so the reads are conflict-free whether
// the LDS serves 16 or 32 lanes of a 64-bit read per cycle.
__device__ __forceinline__ int dl_sw(int r) {
  const int q = r & 3;
  return (q << 2) ^ (q << 1);
}

__device__ __forceinline__ u32x2 lds_read_tr(const lds_char_t* p) {
  return __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)p));
}

// 32x32x16 operand: lane l gets column l%32 at k rows 8*(l/32) .. +7 of the
// 16-row half stage at `off` (two reads of 4 rows each).
__device__ __forceinline__ u32x4 dl_frag(const lds_char_t* base, uint32_t off) {
  const u32x2 lo = lds_read_tr(base + off), hi = lds_read_tr(base + off + 4 * DL_ROWB);
  return u32x4{lo[0], lo[1], hi[0], hi[1]};
}

// s_waitcnt vmcnt(N) leaving the other counters alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// MODE_SUM: the clipped sum over all K = B*T rows. MODE_NORM (the direct
// norm): K restricted to example b's T rows, no factors, and the tile's
// in-range elements squared and summed in registers.
// Gradient store layout (GRAD_STORE): within a tile's 65536 floats, wave w's
// accumulator block (i, j), floats 4q .. 4q+3 of lane l, sit at
// ((w * 8 + i * 2 + j) * 4 + q) * 256 + 4 l: every store and load moves one
// contiguous KB per wave.
__device__ __forceinline__ size_t store_lane_offset(int w, int lane) {
  return (size_t)w * 8 * 4 * 256 + (size_t)lane * 4;
}
__device__ __forceinline__ size_t store_chunk(int i, int j, int q) {
  return (size_t)((i * 2 + j) * 4 + q) * 256;
}

// BIG: some operand of the launch spans 4 GiB or more (see issue()).
template <int MODE, bool BIG>
__global__ __launch_bounds__(GM_THREADS) void dl_gemm_kernel(GemmArgs args) {
  const GemmArgs& a = *(const GemmArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  (void)args;
  __shared__ __attribute__((aligned(1024))) char ring_raw[DL_NS * DL_STB];
  __shared__ float cs[DL_MAXB];
  lds_char_t* ring = (lds_char_t*)(lds_void_t*)ring_raw;

  // Whole tiles come first (spread over the XCDs); the K ranges of the split
  // tail tiles are dispatched last, in round-robin over the XCDs.
  uint32_t item;
  int kc = -1;  // K range of a split tile, or -1
  if (MODE == MODE_NORM || blockIdx.x < a.n_full) {
    item = xcd_remap(blockIdx.x, MODE == MODE_NORM ? gridDim.x : a.n_full);
  } else {
    const uint32_t j = blockIdx.x - a.n_full;
    item = a.n_full + j / (uint32_t)a.ksplit;
    kc = (int)(j - (j / (uint32_t)a.ksplit) * (uint32_t)a.ksplit);
  }
  const int ln = (int)(threadIdx.x & (WAVE - 1));
  const int l = wave_find(item, ln < a.n_layers ? a.L[ln].tile_begin : 0u, a.n_layers);
  const GemmLayer& L = a.L[l];
  uint32_t rel = item - L.tile_begin;
  const int64_t K = (int64_t)a.B * a.T;
  int b = 0;
  int64_t k_begin = 0, k_end = K;
  if (MODE == MODE_SUM && kc >= 0) {
    const int64_t per = (K / DL_BK + a.ksplit - 1) / a.ksplit * DL_BK;  // rows per range
    k_begin = kc * per;
    k_end = k_begin + per < K ? k_begin + per : K;
  }
  int n_ex = 1;  // direct norm: examples b .. b + n_ex - 1 of this item
  if constexpr (MODE == MODE_NORM) {
    const uint32_t ntile = (uint32_t)L.tm * (uint32_t)L.tn;
    const int grp = (int)(rel / ntile);
    rel -= (uint32_t)grp * ntile;
    b = grp * a.eg;
    n_ex = a.B - b < a.eg ? a.B - b : a.eg;
    k_begin = (int64_t)b * a.T;
    k_end = k_begin + (int64_t)n_ex * a.T;
  }
  int mt, nt;
  tile_of(L, rel, mt, nt);
  const int64_t m0 = (int64_t)mt * GM_BM;
  const int64_t n0 = (int64_t)nt * GM_BN;

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = w & 1, wn = w >> 1;

  // Load role: waves 0-3 fill X rows 8w..8w+7 of every stage, waves 4-7 the
  // same rows of Y. Load t writes rows 2t, 2t+1 of that block: lane l takes
  // row l/32 and physical chunk l%32, i.e. logical chunk (l%32) ^ dl_sw(row).
  const bool load_x = w < 4;
  const int wq = w & 3;
  const uint32_t ld_bytes = (uint32_t)((load_x ? L.ldx : L.ldy) * 2);
  const int64_t col0 = load_x ? m0 : n0;
  uint32_t lvo[2];  // lane offsets of loads with t even / odd
#pragma unroll
  for (int par = 0; par < 2; ++par) {
    const int c = (lane & 31) ^ dl_sw(2 * par + (lane >> 5));
    lvo[par] = (uint32_t)((lane >> 5) * ld_bytes + (col0 + 8 * c) * 2);
  }
  const uint32_t lds_role = (uint32_t)(load_x ? 0 : DL_OPB) + (uint32_t)wq * 8 * DL_ROWB;
  const uint64_t gbase = (uint64_t)(load_x ? (const void*)L.X : (const void*)L.Y);
  const uint64_t nrec64 = (uint64_t)K * ld_bytes;
  const uint32_t nrec = nrec64 > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)nrec64;
  const u32x4 desc = {(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)gbase),
                      (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(gbase >> 32)),
                      (uint32_t)__builtin_amdgcn_readfirstlane((int)nrec), (uint32_t)RSRC_WORD3};
  const uint32_t ring_base = (uint32_t)(uintptr_t)ring;
  const int nS = (int)((k_end - k_begin) / DL_BK);
  // Load t (of DL_LOADS) of this wave's share of stage s.
  // An operand of 4 GiB or more does not fit the 32-bit offsets: its
  // descriptor's base moves to each stage's first row instead (the records
  // left from there, none past the last stage). A separate instance, so that
  // launches without such an operand keep the plain loop.
  const bool big = BIG && nrec64 > 0xFFFFFFFFull;
  auto issue = [&](int s, int t) {
    const uint32_t dst = ring_base + (uint32_t)((s % DL_NS) * DL_STB) + lds_role;
    const int64_t row0 = k_begin + (int64_t)s * DL_BK + wq * 8;
    uint32_t sbase;
    u32x4 d = desc;
    if (big) {
      const uint64_t base = gbase + (uint64_t)row0 * ld_bytes;
      const uint64_t rem = s < nS ? (uint64_t)(K - row0) * ld_bytes : 0ull;
      const uint32_t nr = rem > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)rem;
      d = u32x4{(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)base),
                (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(base >> 32)),
                (uint32_t)__builtin_amdgcn_readfirstlane((int)nr), (uint32_t)RSRC_WORD3};
      sbase = 0;
    } else {
      sbase = s < nS ? (uint32_t)(row0 * ld_bytes) : nrec;
    }
    {
      const uint32_t m0v = (uint32_t)__builtin_amdgcn_readfirstlane((int)(dst + t * 1024));
      const uint32_t so = (uint32_t)__builtin_amdgcn_readfirstlane((int)(sbase + 2 * t * ld_bytes));
      // M0 (the LDS destination) is a reserved register that the compiler
      // sets right before each of its own users; this kernel has none. The
      // loads are device-scope (sc1), which measured 0-3 % faster; unlike the
      // Gram's streams they keep the temporal hint, as neighbouring tiles
      // share operand panels through L2 (nt measured slower).
      asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen sc1 lds"
                   :: "s"(m0v), "v"(lvo[t & 1]), "s"(d), "s"(so));
    }
  };

  // Transposing-read lane offsets of this wave's 4 X blocks and 2 Y blocks:
  // within each 16-lane group, lane j addresses row j/4 and columns
  // 4*(j%4) .. +3 of the group's 16 columns.
  const int g = lane >> 4, jl = lane & 15;
  const int rrow = 8 * (g >> 1) + (jl >> 2);
  const int F = dl_sw(jl >> 2);
  uint32_t ox[4], oy[2];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = wm * 128 + i * 32 + 16 * (g & 1) + 4 * (jl & 3);
    ox[i] = (uint32_t)(rrow * DL_ROWB + (((m >> 3) ^ F) << 4) + ((m & 7) << 1));
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int n = wn * 64 + j * 32 + 16 * (g & 1) + 4 * (jl & 3);
    oy[j] = (uint32_t)(DL_OPB + rrow * DL_ROWB + (((n >> 3) ^ F) << 4) + ((n & 7) << 1));
  }

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  if constexpr (MODE == MODE_SUM)
    for (int i = tid; i < a.B; i += GM_THREADS) cs[i] = a.c[i];
  const int spe = a.T / DL_BK;  // stages per example
  // Held in a register: a kernel-argument read inside the loop would be a
  // scalar load whose wait (lgkmcnt) also waits for every LDS read in flight.
  const int nB = __builtin_amdgcn_readfirstlane(a.B);
  // Stage indices below are local to this item's K range, which starts at
  // global stage gs0, inside example e0 (at its start unless this is a split
  // range): the first stage is treated as a boundary, where nothing is yet
  // accumulated.
  const int gs0 = (int)(k_begin / DL_BK);
  const int e0 = gs0 / spe;
  float c_acc = 0.f;            // factor of what is accumulated; 0: nothing yet
  float c_nx = 0.f;             // factor of the example that starts at stage s_nx
  bool skip = false;
  int s_nx = 0, e_nx = e0;      // next example boundary (a local stage) and its example
  // Direct norm: the squared Frobenius norm of this wave's part of the tile
  // for local example le goes to red[le * 8 + w] (the factor table is unused
  // in this mode); the workgroup adds the 8 waves' parts at the end. The
  // columns past M or N were loaded from beyond the rows' valid width and
  // only reach out-of-range elements, which the sum leaves out.
  float* red = cs;
  const bool full = m0 + GM_BM <= L.M && n0 + GM_BN <= L.N;
  int le = 0;
  if constexpr (MODE == MODE_NORM) s_nx = spe;
  auto fin = [&]() __attribute__((always_inline)) {
    float part = 0.f;
    if (full) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int e = 0; e < 16; ++e) part = fmaf(acc[i][j][e], acc[i][j][e], part);
    } else {
      // Rows and columns left in the tile past this lane's first element.
      // Opaque here, so that the compiler does not keep the masks of every
      // accumulator live across the main loop.
      int lim_m = (int)(L.M - m0) - (wm * 128 + (lane >> 5) * 4);
      int lim_n = (int)(L.N - n0) - (wn * 64 + (lane & 31));
      asm volatile("" : "+v"(lim_m), "+v"(lim_n));
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const bool nin = j * 32 < lim_n;
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const float v = acc[i][j][e];
            part += (nin && i * 32 + (e >> 2) * 8 + (e & 3) < lim_m) ? v * v : 0.f;
          }
        }
    }
    part = wave_sum(part);
    if (lane == 0) red[le * (GM_THREADS / WAVE) + w] = part;
    if (a.store) {
      // the example's tile, for a later clipped sum from the store
      float* dst = a.store + ((((size_t)L.slot_begin + rel) * (size_t)a.B + (size_t)(b + le))
                              << 16) + store_lane_offset(w, lane);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const f32x4 v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                             acc[i][j][4 * q + 3]};
            __builtin_nontemporal_store(v, (f32x4*)(dst + store_chunk(i, j, q)));
          }
    }
    ++le;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};
  };
  // Called once per stage, in increasing order, in the memory phase before
  // that stage's MFMAs. Clipped sum: at an example boundary, rescales the
  // accumulators by c_prev / c_next and fetches the factor of the example
  // after. Direct norm: at an example boundary, reduces the finished
  // example's part of the tile and clears the accumulators.
  auto enter = [&](int s) {
    if (MODE == MODE_NORM && s == s_nx) {
      fin();
      s_nx += spe;
    }
    if (MODE == MODE_SUM && s == s_nx) {
      const float ce = c_nx;
      ++e_nx;
      s_nx = e_nx * spe - gs0;
      if (e_nx < nB) c_nx = cs[e_nx];
      skip = !(ce != 0.f);
      if (!skip) {
        if (c_acc != 0.f) {
          const float f = c_acc / ce;
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) acc[i][j] *= f;
        }
        c_acc = ce;
      }
    }
  };
  // rd: both halves (k 0..15 and 16..31) of stage s, 4 X and 2 Y fragments
  // each. rd_issue: the same reads in four groups of three, each group after
  // one of this wave's loads of stage sl. Spreading the loads over the phase
  // keeps the L1's queue of pending requests from filling in one burst (2-4 %
  // faster than issuing all loads first or all reads first).
  auto frag = [&](const lds_char_t* base, int idx) {
    const int h = idx / 6, k = idx % 6;
    return dl_frag(base, (k < 4 ? ox[k] : oy[k - 4]) + h * 16 * DL_ROWB);
  };
  auto rd = [&](int s, u32x4 (&f)[12]) {
    const lds_char_t* base = ring + (s % DL_NS) * DL_STB;
#pragma unroll
    for (int idx = 0; idx < 12; ++idx) f[idx] = frag(base, idx);
  };
  auto rd_issue = [&](int s, int sl, u32x4 (&f)[12]) {
    const lds_char_t* base = ring + (s % DL_NS) * DL_STB;
#pragma unroll
    for (int q = 0; q < DL_LOADS; ++q) {
      issue(sl, q);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int r = 0; r < 3; ++r) f[3 * q + r] = frag(base, 3 * q + r);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  auto compute = [&](const u32x4 (&f)[12]) {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_setprio(1);
    if (!skip) {
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = mfma32_bf16(f[6 * h + i], f[6 * h + 4 + j], acc[i][j]);
    }
    __builtin_amdgcn_s_setprio(0);
    __builtin_amdgcn_sched_barrier(0);
  };
  // Phase boundary; nothing is scheduled across it.
  auto bar = [&]() {
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
  };

  u32x4 fr[12];
  if (w < 4) {
#pragma unroll
    for (int p = 0; p < DL_NS; ++p)
#pragma unroll
      for (int t = 0; t < DL_LOADS; ++t) issue(p, t);
    wait_vmcnt<DL_LOADS * (DL_NS - 1)>();
    bar();  // stage 0 has landed, the factor table is filled
    if constexpr (MODE == MODE_SUM) c_nx = cs[e0];
    rd(0, fr);
    enter(0);
    for (int s = 0; s < nS; ++s) {
      compute(fr);
      wait_vmcnt<DL_LOADS * (DL_NS - 2)>();
      bar();
      rd_issue(s + 1, s + DL_NS, fr);  // past the last stage: reads an unused slot
      if (s + 1 < nS) enter(s + 1);
      bar();
    }
  } else {
#pragma unroll
    for (int p = 0; p < DL_NS - 1; ++p)
#pragma unroll
      for (int t = 0; t < DL_LOADS; ++t) issue(p, t);
    wait_vmcnt<DL_LOADS * (DL_NS - 2)>();
    bar();
    if constexpr (MODE == MODE_SUM) c_nx = cs[e0];
    for (int s = 0; s < nS; ++s) {
      rd_issue(s, s + DL_NS - 1, fr);
      enter(s);
      wait_vmcnt<DL_LOADS * (DL_NS - 2)>();
      bar();
      compute(fr);
      bar();
    }
  }
  // No load may still be writing LDS when the workgroup ends.
  wait_vmcnt<0>();
  if constexpr (MODE == MODE_SUM) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] *= c_acc;
    if (kc >= 0) {
      // A split range: its raw partial tile, for the fixup kernel.
      __syncthreads();
      float* slice = (float*)ring_raw + w * 32 * EP_LD;
      store_partial(a.part + ((size_t)(item - a.n_full) * a.ksplit + kc) * (GM_BM * GM_BN),
                    wm, wn, lane, acc, slice);
    } else if (a.transpose) {
      store_tile(a, L, m0, n0, wm, wn, lane, acc, true);
    } else {
      // The ring is free once every wave is past its last read of it.
      __syncthreads();
      float* slice = (float*)ring_raw + w * 32 * EP_LD;
      store_tile_rows(a, L, m0, n0, wm, wn, lane, acc, slice);
    }
  } else {
    fin();  // the last example
    __syncthreads();
    if (tid < n_ex) {
      float t = 0.f;
#pragma unroll
      for (int q = 0; q < GM_THREADS / WAVE; ++q) t += red[tid * (GM_THREADS / WAVE) + q];
      a.ws[(int64_t)(b + tid) * a.slots + L.slot_begin + rel] = t;
    }
  }
}

// Clipped sum from a gradient store (the materialising form of eq. 3: the
// per-example gradients, already formed by the direct norm, weighted and
// added): one workgroup per output tile, its 8 waves in the register layout
// of dl_gemm_kernel, acc = sum_e c_e tile_e in example order (examples with
// c_e = 0 are left out, as in the GEMM), then the GEMM's own epilogue (prior,
// fused noise, 1/B; row-major, or transposed per layer). HBM-bound: B tiles
// read per output tile.
__global__ __launch_bounds__(GM_THREADS) void store_sum_kernel(GemmArgs args) {
  const GemmArgs& a = *(const GemmArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  (void)args;
  __shared__ __attribute__((aligned(1024))) char stage[(GM_THREADS / WAVE) * 32 * EP_LD * 4];
  const uint32_t item = xcd_remap(blockIdx.x, gridDim.x);
  const int ln = (int)(threadIdx.x & (WAVE - 1));
  const int l = wave_find(item, ln < a.n_layers ? a.L[ln].tile_begin : 0u, a.n_layers);
  const GemmLayer& L = a.L[l];
  const uint32_t rel = item - L.tile_begin;
  int mt, nt;
  tile_of(L, rel, mt, nt);
  const int64_t m0 = (int64_t)mt * GM_BM, n0 = (int64_t)nt * GM_BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = w & 1, wn = w >> 1;
  const float* src = a.store + ((((size_t)L.store_slot + rel) * (size_t)a.B) << 16) +
                     store_lane_offset(w, lane);
  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};
  const int nB = __builtin_amdgcn_readfirstlane(a.B);
  for (int e = 0; e < nB; ++e) {
    const float ce = a.c[e];
    if (!(ce != 0.f)) continue;
    const float* p = src + ((size_t)e << 16);
    // two halves of 16 loads each (i = 0, 1 and i = 2, 3), all in flight
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      f32x4 v[2][2][4];
#pragma unroll
      for (int ii = 0; ii < 2; ++ii)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            v[ii][j][q] = __builtin_nontemporal_load((const f32x4*)(p + store_chunk(2 * hh + ii, j, q)));
#pragma unroll
      for (int ii = 0; ii < 2; ++ii)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              acc[2 * hh + ii][j][4 * q + r] = fmaf(ce, v[ii][j][q][r], acc[2 * hh + ii][j][4 * q + r]);
    }
  }
  if (L.store_transpose) {
    store_tile(a, L, m0, n0, wm, wn, lane, acc, true);
  } else {
    float* slice = (float*)stage + w * 32 * EP_LD;
    store_tile_rows(a, L, m0, n0, wm, wn, lane, acc, slice);
  }
}

hipError_t launch_store_sum(const GemmArgs& a, hipStream_t s) {
  if (a.n_items == 0) return hipSuccess;
  if (!a.store || !a.c) return hipErrorInvalidValue;
  hipLaunchKernelGGL(store_sum_kernel, dim3(a.n_items), dim3(GM_THREADS), 0, s, a);
  return hipGetLastError();
}

template <int DT, bool VEC, int MODE>
static void launch_sc(const GemmArgs& a, int sc, hipStream_t s) {
  const dim3 g(a.n_items), blk(GM_THREADS);
  if constexpr (MODE == MODE_NORM) {
    hipLaunchKernelGGL((kt_gemm_kernel<DT, VEC, MODE, SC_NONE>), g, blk, 0, s, a);
  } else {
    if (sc == SC_ACC)
      hipLaunchKernelGGL((kt_gemm_kernel<DT, VEC, MODE, SC_ACC>), g, blk, 0, s, a);
    else
      hipLaunchKernelGGL((kt_gemm_kernel<DT, VEC, MODE, SC_STAGE>), g, blk, 0, s, a);
  }
}

template <int MODE>
static hipError_t launch_kt(const GemmArgs& a0, int dt, bool vec, int cus, size_t part_bytes,
                            hipStream_t s) {
  if (a0.n_items == 0) return hipSuccess;
  GemmArgs a = a0;
  a.n_full = a.n_items;
  a.n_split = 0;
  a.ksplit = 1;
  // The accumulator form needs every K-stage inside one example.
  const int ks = dt == DT_BF16 ? KT<DT_BF16>::KS : KT<DT_F32>::KS;
  const int sc = MODE == MODE_NORM ? SC_NONE : (a.T % ks == 0 ? SC_ACC : SC_STAGE);
  // Example groups and the gradient store exist only on the direct-load kernel.
  const bool dl = dt == DT_BF16 && vec && a.T % DL_BK == 0;
  if (MODE == MODE_NORM && (a.eg < 1 || a.eg > NG_MAX || ((a.eg > 1 || a.store) && !dl)))
    return hipErrorInvalidValue;
  if (MODE == MODE_SUM && a.store) return hipErrorInvalidValue;
  if (dt == DT_BF16 && vec && a.T % DL_BK == 0 && (MODE == MODE_NORM || a.B <= DL_MAXB)) {
    uint32_t grid = a.n_items;
    if (MODE == MODE_SUM && a.part != nullptr) {
      const TailSplit t = tail_split(a.n_items, (int)((int64_t)a.B * a.T / DL_BK), cus);
      if (t.n_split > 0 && (size_t)t.n_split * t.ks * SPLIT_TILE_BYTES <= part_bytes) {
        a.n_full = t.n_full;
        a.n_split = t.n_split;
        a.ksplit = t.ks;
        grid = t.n_full + t.n_split * (uint32_t)t.ks;
      }
    }
    if (a.big)
      hipLaunchKernelGGL((dl_gemm_kernel<MODE, true>), dim3(grid), dim3(GM_THREADS), 0, s, a);
    else
      hipLaunchKernelGGL((dl_gemm_kernel<MODE, false>), dim3(grid), dim3(GM_THREADS), 0, s, a);
    if (a.n_split > 0) {
      hipLaunchKernelGGL(split_fixup_kernel, dim3(a.n_split * (GM_BM * GM_BN / 4 / 256)),
                         dim3(256), 0, s, a);
    }
    return hipGetLastError();
  }
  if (dt == DT_BF16) {
    if (vec) launch_sc<DT_BF16, true, MODE>(a, sc, s);
    else launch_sc<DT_BF16, false, MODE>(a, sc, s);
  } else {
    if (vec) launch_sc<DT_F32, true, MODE>(a, sc, s);
    else launch_sc<DT_F32, false, MODE>(a, sc, s);
  }
  return hipGetLastError();
}

hipError_t launch_clipped_sum(const GemmArgs& a, int dt, bool vec, int cus, size_t part_bytes,
                              hipStream_t s) {
  return launch_kt<MODE_SUM>(a, dt, vec, cus, part_bytes, s);
}

hipError_t launch_direct_norm(const GemmArgs& a, int dt, bool vec, hipStream_t s) {
  return launch_kt<MODE_NORM>(a, dt, vec, 0, 0, s);
}

}  // namespace dpg
