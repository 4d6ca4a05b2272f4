// Shared device helpers for the gfx950 (CDNA4) kernels of libdpghost.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.hpp"

namespace dpg {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int WAVE = 64;
constexpr int N_XCD = 8;

// The hardware dispatcher hands consecutive workgroup ids to the 8 XCDs in
// turn. Remap so that each XCD walks one contiguous range of logical work
// items: neighbouring items (which share rows of the same example) then run
// on the same XCD and share its L2.
__device__ __forceinline__ uint32_t xcd_remap(uint32_t bid, uint32_t nwg) {
  const uint32_t xcd = bid % N_XCD, local = bid / N_XCD;
  const uint32_t q = nwg / N_XCD, r = nwg % N_XCD;
  return xcd * q + (xcd < r ? xcd : r) + local;
}

// 16-byte chunk c (0..7) of a 128-byte LDS row r lives at physical chunk
// swz(r, c): conflict-free for row-contiguous writes, for column-strided
// writes of 8-row groups, and for 32-row MFMA operand reads.
__device__ __forceinline__ int swz(int r, int c) { return c ^ ((r ^ (r >> 3)) & 7); }

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(((uint32_t)h) << 16);
}

// fp32 -> bf16, round to nearest even (inputs here are finite).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, WAVE);
  return v;
}

// x plus the x of the lane 16 (or 32) lanes away, in every lane, from the
// gfx950 cross-lane swaps (VALU instructions, no LDS permute). permlane16_swap
// of x with itself returns rows (0, 0, 2, 2) of x in one result and rows
// (1, 1, 3, 3) in the other (a row is 16 lanes); permlane32_swap returns the
// low half twice and the high half twice. Both lanes of a pair add the same
// two values in the same order, so they hold the same bits.
__device__ __forceinline__ float xor16_sum(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float xor32_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, WAVE);
  return v;
}

// Entry of a launch's table that work index x falls in: the last of the n
// entries (n <= 64, begins increasing from begin 0) whose begin is <= x. Lane
// j passes entry j's begin; a ballot counts the entries after the first that
// start at or before x. One load per lane instead of a chain of dependent
// scalar loads (one per entry, each a round trip when the scalar cache is
// cold). x must be the same on every lane, and the whole wave active.
__device__ __forceinline__ int wave_find(uint32_t x, uint32_t lane_begin, int n) {
  const int lane = (int)(threadIdx.x & (WAVE - 1));
  const uint64_t m = __ballot(lane >= 1 && lane < n && x >= lane_begin);
  return __builtin_amdgcn_readfirstlane(__popcll(m));
}

// Number of the n keys (n a multiple of 8, 16-byte aligned LDS) below k:
// 16-byte reads, eight keys per step, two steps' reads in flight.
__device__ __forceinline__ int count_below(const uint32_t* keys, int n, uint32_t k) {
  const u32x4* k4 = (const u32x4*)keys;
  int r0 = 0, r1 = 0;
#pragma unroll 4
  for (int j = 0; j < n / 4; j += 2) {
    const u32x4 x = k4[j], y = k4[j + 1];
    r0 += (x[0] < k) + (x[1] < k) + (x[2] < k) + (x[3] < k);
    r1 += (y[0] < k) + (y[1] < k) + (y[2] < k) + (y[3] < k);
  }
  return r0 + r1;
}

// 32x32 output block MFMA step; K per call is 16 (bf16) or 2 (fp32).
__device__ __forceinline__ f32x16 mfma32_bf16(const u32x4& a, const u32x4& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mfma32_f32(float a, float b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// Buffer resources: loads through them need no bounds branches, because the
// hardware returns 0 for any dword at or past num_records bytes.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr int RSRC_WORD3 = 0x00020000;  // raw (untyped) buffer, gfx9 family

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint64_t nbytes) {
  const uint32_t n = nbytes > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)nbytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, RSRC_WORD3);
}
// Cache policy of a load: 0, or CPOL_STREAM (sc1 nt: device scope,
// non-temporal) for data read once, which keeps the streamed lines from
// crowding the caches (measured faster on the kernels that stream every byte
// once; slower where tiles share operands through L2).
constexpr int CPOL_STREAM = 18;

// voff: per-lane byte offset; soff: wave-uniform byte offset (an SGPR).
template <int CPOL = 0>
__device__ __forceinline__ u32x4 buf_load16(rsrc_t r, uint32_t voff, uint32_t soff = 0) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, CPOL));
}
template <int CPOL = 0>
__device__ __forceinline__ uint32_t buf_load4(rsrc_t r, uint32_t voff, uint32_t soff = 0) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, CPOL);
}
template <int CPOL = 0>
__device__ __forceinline__ uint32_t buf_load2(rsrc_t r, uint32_t voff, uint32_t soff = 0) {
  return (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, CPOL);
}

// 16-byte chunk of elements [col, col+EPC) of a row, through a buffer
// resource; the chunk starts at byte voff + soff. VEC: one 16-byte load (the
// row is 16-byte aligned); otherwise one load per element. Elements at or past
// `ncol` are zeroed when MASK is set.
template <int DT, bool VEC, bool MASK, int CPOL = 0>
__device__ __forceinline__ u32x4 buf_chunk(rsrc_t r, uint32_t voff, uint32_t soff, int64_t col,
                                           int64_t ncol) {
  constexpr int ES = (DT == DT_BF16) ? 2 : 4;
  u32x4 v;
  if constexpr (VEC) {
    v = buf_load16<CPOL>(r, voff, soff);
  } else if constexpr (DT == DT_BF16) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      v[q] = buf_load2<CPOL>(r, voff + (2 * q) * ES, soff) |
             (buf_load2<CPOL>(r, voff + (2 * q + 1) * ES, soff) << 16);
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = buf_load4<CPOL>(r, voff + q * ES, soff);
  }
  if constexpr (MASK) {
    const int64_t nv = ncol - col;  // valid elements in the chunk (may be <= 0)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if constexpr (DT == DT_BF16) {
        const int e = 2 * q;
        v[q] = e + 1 < nv ? v[q] : (e < nv ? (v[q] & 0xFFFFu) : 0u);
      } else {
        v[q] = q < nv ? v[q] : 0u;
      }
    }
  }
  return v;
}

// Chunk loaders: 16 bytes = 8 bf16 or 4 fp32 starting at element `col` of a
// row. Elements at or past `ncol` read as zero.
template <int DT>
__device__ __forceinline__ u32x4 load_chunk_elems(const void* row, int64_t col, int64_t ncol) {
  u32x4 r = {0u, 0u, 0u, 0u};
  if constexpr (DT == DT_BF16) {
    const uint16_t* p = (const uint16_t*)row;
    uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (col + e < ncol) w[e >> 1] |= ((uint32_t)p[col + e]) << ((e & 1) * 16);
    }
    r[0] = w[0]; r[1] = w[1]; r[2] = w[2]; r[3] = w[3];
  } else {
    const uint32_t* p = (const uint32_t*)row;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (col + e < ncol) r[e] = p[col + e];
    }
  }
  return r;
}

__device__ __forceinline__ u32x4 load_chunk16(const void* row, int64_t col, int es) {
  return *(const u32x4*)((const char*)row + col * es);
}

// 16-byte chunk at `col` (< ncol) of a 16-byte aligned row whose stride
// covers the whole chunk; elements at or past ncol are zeroed in registers.
template <int DT>
__device__ __forceinline__ u32x4 load_chunk16_masked(const void* row, int64_t col, int64_t ncol) {
  constexpr int EPC = (DT == DT_BF16) ? 8 : 4;
  u32x4 v = load_chunk16(row, col, DT == DT_BF16 ? 2 : 4);
  const int64_t nv = ncol - col;  // valid elements in this chunk, >= 1
  if (nv < EPC) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if constexpr (DT == DT_BF16) {
        const int e = 2 * q;  // elements e, e+1 live in dword q
        v[q] = e + 1 < nv ? v[q] : (e < nv ? (v[q] & 0xFFFFu) : 0u);
      } else {
        v[q] = q < nv ? v[q] : 0u;
      }
    }
  }
  return v;
}

// How a thread's chunk [col, col + EPC) of a row relates to the valid columns.
enum ChunkKind { CHUNK_FULL = 0, CHUNK_PART = 1, CHUNK_NONE = 2 };
template <int DT>
__device__ __forceinline__ int chunk_kind(int64_t col, int64_t ncol) {
  constexpr int EPC = (DT == DT_BF16) ? 8 : 4;
  return col + EPC <= ncol ? CHUNK_FULL : (col < ncol ? CHUNK_PART : CHUNK_NONE);
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

}  // namespace dpg
