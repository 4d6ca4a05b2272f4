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
// For bf16 rows that are 16-byte aligned, dl_gram_kernel loads the rows
// straight into LDS (see there); otherwise a workgroup streams the rows of its two 128-row T-tiles through LDS, first
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
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace dpg {

// Layer, example and item index within (example, layer) of work item `item`.
struct GramItem {
  int l, b;
  uint32_t rel;
};
__device__ __forceinline__ GramItem gram_item(const GramArgs& a, uint32_t item) {
  GramItem g;
  g.b = (int)(item / a.per_ex);
  uint32_t rel = item - (uint32_t)g.b * a.per_ex;
  const int ln = (int)(threadIdx.x & (WAVE - 1));
  const int l = wave_find(rel, ln < a.n_layers ? a.L[ln].item_begin : 0u, a.n_layers);
  g.l = l;
  g.rel = rel - a.L[l].item_begin;
  return g;
}


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
template <int DT, int NB, int NA>
__device__ __forceinline__ void stage_mfma(const u32x4* __restrict__ lds, const int (&ra)[NA],
                                           const int (&rb)[NA], f32x16 (&acc)[NB], int lane) {
  static_assert(NB <= NA, "block list");
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

// A wave's blocks as products of distinct fragments (direct-load kernels,
// bf16): block j multiplies fragment ia(j) (its rows) by fragment ib(j) (its
// columns); the nf fragments are 32-row slices of the stage at row offsets
// rows[0..nf). A fragment that several blocks use (both operands of a
// diagonal block, the blocks of one block row) is read from LDS once per
// k-step, half the reads of one pair per block.
struct FpD1 {   // waves 0, 1 of a diagonal tile: (x,x) (x,y) (y,y); rows {x, y}
  static constexpr int NB = 3, NF = 2;
  static constexpr int ia(int j) { return j < 2 ? 0 : 1; }
  static constexpr int ib(int j) { return j < 1 ? 0 : 1; }
};
struct FpD2 {   // waves 2, 3 of a diagonal tile: (x,64) (x,96); rows {x, 64, 96}
  static constexpr int NB = 2, NF = 3;
  static constexpr int ia(int) { return 0; }
  static constexpr int ib(int j) { return 1 + j; }
};
struct FpOff {  // a 64x64 quadrant of an off-diagonal pair; rows {x, x+32, y, y+32}
  static constexpr int NB = 4, NF = 4;
  static constexpr int ia(int j) { return j >> 1; }
  static constexpr int ib(int j) { return 2 + (j & 1); }
};
// Whole-example Gram (8 waves, block rows 0..7): wave g < 4 takes (g,g)..(g,g+4)
// (rows g..g+4); waves 4..7 the rest of row pairs {g, 7-g}.
struct FpW0 {
  static constexpr int NB = 5, NF = 5;
  static constexpr int ia(int) { return 0; }
  static constexpr int ib(int j) { return j; }
  static constexpr int row(int g, int q) { return 32 * (g + q); }
};
struct FpW4 {   // (0,5) (0,6) (0,7) (7,7)
  static constexpr int NB = 4, NF = 4;
  static constexpr int ia(int j) { return j < 3 ? 0 : 3; }
  static constexpr int ib(int j) { return j < 3 ? 1 + j : 3; }
  static constexpr int row(int, int q) { return q == 0 ? 0 : 32 * (4 + q); }
};
struct FpW5 {   // (1,6) (1,7) (6,6) (6,7)
  static constexpr int NB = 4, NF = 3;
  static constexpr int ia(int j) { return j < 2 ? 0 : 1; }
  static constexpr int ib(int j) { return 1 + (j & 1); }
  static constexpr int row(int, int q) { return q == 0 ? 32 : 32 * (5 + q); }
};
struct FpW6 {   // (2,7) (5,5) (5,6) (5,7)
  static constexpr int NB = 4, NF = 4;
  static constexpr int ia(int j) { return j == 0 ? 0 : 2; }
  static constexpr int ib(int j) { return j == 0 || j == 3 ? 1 : j + 1; }
  static constexpr int row(int, int q) { return q == 0 ? 64 : (q == 1 ? 224 : 32 * (3 + q)); }
};
struct FpW7 {   // (4,4) (4,5) (4,6) (4,7)
  static constexpr int NB = 4, NF = 4;
  static constexpr int ia(int) { return 0; }
  static constexpr int ib(int j) { return j; }
  static constexpr int row(int, int q) { return 32 * (4 + q); }
};

// The whole-example patterns reproduce the block list (entry k of row pair g
// is (g, g+k) for k < 8-g, else (7-g, 7-g + k-(8-g)); wave g takes entries
// 0..4, wave g+4 entries 5..8), checked at compile time.
template <class P>
constexpr bool fp_whole_matches(int w) {
  const int g = w & 3, k0 = (w >> 2) * 5;
  for (int j = 0; j < P::NB; ++j) {
    const int k = k0 + j;
    const int bi = k < 8 - g ? g : 7 - g;
    const int bj = k < 8 - g ? g + k : 7 - g + (k - (8 - g));
    if (P::row(g, P::ia(j)) != 32 * bi || P::row(g, P::ib(j)) != 32 * bj) return false;
  }
  for (int q = 0; q < P::NF; ++q)
    for (int r = 0; r < q; ++r)
      if (P::row(g, q) == P::row(g, r)) return false;
  return true;
}
static_assert(fp_whole_matches<FpW0>(0) && fp_whole_matches<FpW0>(1) &&
                  fp_whole_matches<FpW0>(2) && fp_whole_matches<FpW0>(3) &&
                  fp_whole_matches<FpW4>(4) && fp_whole_matches<FpW5>(5) &&
                  fp_whole_matches<FpW6>(6) && fp_whole_matches<FpW7>(7),
              "fragment patterns of the whole-example Gram");

template <class P>
__device__ __forceinline__ void stage_mfma_fp(const u32x4* __restrict__ lds,
                                              const int (&rows)[P::NF], f32x16 (&acc)[P::NB],
                                              int lane) {
  const int r32 = lane & 31, half = lane >> 5;
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    const int c = 2 * ks + half;
    u32x4 f[P::NF];
#pragma unroll
    for (int q = 0; q < P::NF; ++q) {
      const int row = rows[q] + r32;
      f[q] = lds[row * 8 + swz(row, c)];
    }
#pragma unroll
    for (int j = 0; j < P::NB; ++j) acc[j] = mfma32_bf16(f[P::ia(j)], f[P::ib(j)], acc[j]);
  }
}

// Streams the rows of one or two T-tiles of a matrix pair through LDS.
// Entry i (0..7) of a thread is LDS row (tid/8) + 32*i, chunk tid%8; entries
// 0..3 are rows of T-tile ti, entries 4..7 rows of T-tile tj. Stage s < nX
// reads features [s*KS, ...) of X up to column x1; later stages read features
// [y0 + (s-nX)*KS, ...) of Y up to column y1. The buffer resources span one
// example's T rows, so rows past T read as zero; per-row offsets are
// wave-uniform (SGPR) and only the lane's own (row, chunk) offset is a VGPR.
template <int DT, bool VEC>
struct TileStream {
  static constexpr int EPC = (DT == DT_BF16) ? 8 : 4;
  static constexpr int KS = 8 * EPC;
  static constexpr int ES = (DT == DT_BF16) ? 2 : 4;
  rsrc_t rx, ry;
  uint32_t ldx, ldy;           // row strides in bytes
  uint32_t vxi, vxj, vyi, vyj; // lane offsets of entry 0 / entry 4 in X and Y
  int c;                       // this thread's chunk within a row
  int nX;
  int64_t x1, y0, y1;

  template <int NENT>
  __device__ __forceinline__ void prefetch(int s, u32x4 (&pre)[NENT]) const {
    const bool inX = s < nX;
    const rsrc_t r = inX ? rx : ry;
    const uint32_t ld = inX ? ldx : ldy;
    const int64_t c0 = inX ? (int64_t)s * KS : y0 + (int64_t)(s - nX) * KS;  // stage column
    const int64_t ncol = inX ? x1 : y1;
    const uint32_t vi = inX ? vxi : vyi, vj = inX ? vxj : vyj;
#pragma unroll
    for (int i = 0; i < NENT; ++i) {
      const uint32_t soff = (uint32_t)(c0 * ES) + (uint32_t)(32 * (i & 3)) * ld;
      pre[i] = buf_chunk<DT, VEC, true>(r, i < 4 ? vi : vj, soff, c0 + c * EPC, ncol);
    }
  }
};

template <int NENT>
__device__ __forceinline__ void store_stage(u32x4* lds, const u32x4 (&pre)[NENT], int tid) {
#pragma unroll
  for (int i = 0; i < NENT; ++i) {
    const int r = (tid >> 3) + 32 * i, c = tid & 7;
    lds[r * 8 + swz(r, c)] = pre[i];
  }
}

// LDS of one stage: a diagonal pair streams 128 rows, an off-diagonal 256.
template <int PAT> struct PatRows { static constexpr int ROWS = PAT == PAT_OFF ? 2 * GR_TM : GR_TM; };

template <int DT, bool VEC, int PAT, int PF>
__device__ __forceinline__ float gram_item(const GramLayer& L, int b, int T, int ti, int tj, int chunk,
                           u32x4* lds) {
  constexpr int NB = PatNB<PAT>::NB;
  constexpr int ROWS = PatRows<PAT>::ROWS;
  constexpr int NENT = ROWS / 32;  // 16-byte chunks per thread per stage
  using TS = TileStream<DT, VEC>;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);

  TS ts;
  const uint64_t ex_rows = (uint64_t)b * T;
  ts.ldx = (uint32_t)(L.lda * TS::ES);
  ts.ldy = (uint32_t)(L.ldg * TS::ES);
  ts.rx = make_rsrc((const char*)L.A + ex_rows * ts.ldx, (uint64_t)T * ts.ldx);
  ts.ry = make_rsrc((const char*)L.G + ex_rows * ts.ldy, (uint64_t)T * ts.ldy);
  ts.c = tid & 7;
  ts.x1 = L.d_in;
  ts.y0 = (int64_t)L.g0 + (int64_t)chunk * L.kg;
  ts.y1 = ts.y0 + L.kg < L.g1 ? ts.y0 + L.kg : L.g1;
  ts.nX = ((L.d_in + TS::KS - 1) / TS::KS + 1) & ~1;  // padded to even
  const int nY = (int)((ts.y1 - ts.y0 + TS::KS - 1) / TS::KS);
  const uint32_t r0 = tid >> 3, cb = (tid & 7) * 16;
  ts.vxi = (ti * GR_TM + r0) * ts.ldx + cb;
  ts.vxj = (tj * GR_TM + r0) * ts.ldx + cb;
  ts.vyi = (ti * GR_TM + r0) * ts.ldy + cb;
  ts.vyj = (tj * GR_TM + r0) * ts.ldy + cb;

  int ra[4], rb[4];
  float wt[4];
  block_rows<PAT>(w, ra, rb, wt);
  f32x16 accP[NB], accQ[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) { accP[j][e] = 0.f; accQ[j][e] = 0.f; }

  const int n = ts.nX + nY;
  u32x4* buf0 = lds;
  u32x4* buf1 = lds + ROWS * 8;
  if constexpr (PF == 2) {
    // Two register sets and two LDS buffers: the loads of stage s+2 are in
    // flight while stage s is multiplied and stage s+1 is stored. Even
    // stages use set A and buffer 0. The A phase is padded to an even number
    // of stages (padding stages read masked zeros), so both phases start even
    // and each keeps its own accumulators in its own loop.
    u32x4 pA[NENT], pB[NENT];
    auto phase = [&](int s_begin, int s_end, f32x16 (&acc)[NB]) {
      for (int s = s_begin; s < s_end; s += 2) {
        if (s + 2 < n) ts.template prefetch<NENT>(s + 2, pA);
        stage_mfma<DT, NB>(buf0, ra, rb, acc, lane);
        if (s + 1 < n) store_stage<NENT>(buf1, pB, tid);
        __syncthreads();
        if (s + 1 >= s_end) break;
        if (s + 3 < n) ts.template prefetch<NENT>(s + 3, pB);
        stage_mfma<DT, NB>(buf1, ra, rb, acc, lane);
        if (s + 2 < n) store_stage<NENT>(buf0, pA, tid);
        __syncthreads();
      }
    };
    ts.template prefetch<NENT>(0, pA);
    if (n > 1) ts.template prefetch<NENT>(1, pB);
    store_stage<NENT>(buf0, pA, tid);
    __syncthreads();
    phase(0, ts.nX, accP);
    phase(ts.nX, n, accQ);
  } else {
    // One register set, two LDS buffers: the loads of stage s+1 are in
    // flight while stage s is multiplied.
    u32x4 pA[NENT];
    auto phase = [&](int s_begin, int s_end, f32x16 (&acc)[NB]) {
      for (int s = s_begin; s < s_end; ++s) {
        if (s + 1 < n) ts.template prefetch<NENT>(s + 1, pA);
        stage_mfma<DT, NB>((s & 1) ? buf1 : buf0, ra, rb, acc, lane);
        if (s + 1 < n) store_stage<NENT>((s & 1) ? buf0 : buf1, pA, tid);
        __syncthreads();
      }
    };
    ts.template prefetch<NENT>(0, pA);
    store_stage<NENT>(buf0, pA, tid);
    __syncthreads();
    phase(0, ts.nX, accP);
    phase(ts.nX, n, accQ);
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

// SINGLE: every example fits one T-tile (T <= 128), so only the diagonal
// patterns exist; fewer registers and a 2 x 16 KB LDS footprint let three
// workgroups share a CU.
template <int DT, bool VEC, bool SINGLE>
__global__ __launch_bounds__(GR_THREADS) void gram_norm_kernel(GramArgs args) {
  // Index the layer table in place in the kernel-argument segment (the only
  // explicit argument sits at offset 0) instead of copying it to the stack.
  const GramArgs& a = *(const GramArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  (void)args;
  __shared__ u32x4 lds[2 * (SINGLE ? GR_TM : GR_ROWS) * 8];
  __shared__ float red[GR_THREADS / WAVE];
  const uint32_t item = xcd_remap(blockIdx.x, gridDim.x);
  const GramItem gi = gram_item(a, item);
  const GramLayer& L = a.L[gi.l];
  const int b = gi.b;
  const int pair = (int)(gi.rel / (uint32_t)L.nc);
  const int chunk = (int)(gi.rel - (uint32_t)pair * L.nc);
  int ti = 0, rem = pair;
  while (rem >= a.n_t - ti) { rem -= a.n_t - ti; ++ti; }
  const int tj = ti + rem;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

  float part;
  // Prefetch depth 2 where registers allow (one 128-row tile), else 1.
  if constexpr (SINGLE) {
    if (w < 2)
      part = gram_item<DT, VEC, PAT_D1, 2>(L, b, a.T, ti, tj, chunk, lds);
    else
      part = gram_item<DT, VEC, PAT_D2, 2>(L, b, a.T, ti, tj, chunk, lds);
  } else {
    if (ti != tj)
      part = gram_item<DT, VEC, PAT_OFF, 1>(L, b, a.T, ti, tj, chunk, lds);
    else if (w < 2)
      part = gram_item<DT, VEC, PAT_D1, 1>(L, b, a.T, ti, tj, chunk, lds);
    else
      part = gram_item<DT, VEC, PAT_D2, 1>(L, b, a.T, ti, tj, chunk, lds);
  }
  part = wave_sum(part);
  if ((threadIdx.x & 63) == 0) red[w] = part;
  __syncthreads();
  if (threadIdx.x == 0)
    a.ws[(int64_t)b * a.slots + L.slot_begin + pair * L.nc + chunk] =
        (red[0] + red[1]) + (red[2] + red[3]);
}

// ---------------------------------------------------------------------------
// Direct-load Gram kernel: bf16, 16-byte aligned rows.
// Rows go straight into LDS through LDS-writing buffer loads (lane l's 16
// bytes land at M0 + 16*l), four stages in a ring. A stage holds 64 features
// of the rows of the item's T-tile pair: 128 rows for a diagonal pair, 256
// (tile ti then tile tj) for an off-diagonal one; row r holds its 8 chunks
// with logical chunk c at physical chunk swz(r, c), so the MFMA reads are the
// same as the register-staged kernel's. Rows past T read zero through the
// example's buffer range; chunks wholly past the last feature are pointed
// past the range; a chunk that straddles it is masked in LDS after it lands.
// SINGLE (T <= 128): 16 KB stages, two workgroups per CU; otherwise 32 KB
// stages and one workgroup per CU.
// In single-tile launches the loads carry the non-temporal hint at device
// scope (sc1 nt): each byte is read once (a head's activation rows, re-read
// per logit chunk, still hit L2), and the hint keeps the streamed lines from
// crowding the caches. The T = 128 Gram of a GPT-2 step went from 5.7 to
// 6.4 TB/s with it, the T = 256 one from 4.5 to 4.8 TB/s. Tile-pair launches
// (T > 256) read every T-tile once per pair it belongs to, so their loads keep
// the temporal hint (sc1 only): with nt the T = 1024 Gram took 8-14 % longer.
constexpr int DG_NS = 4;
constexpr int DG_ROWB = 128;                  // 64 bf16 per LDS row

typedef __attribute__((address_space(3))) void lds_void_g;

template <int N>
__device__ __forceinline__ void dg_wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Fused bias gradient. While a G stage (64 features of every example row)
// sits in LDS, NT threads sum its columns: thread t adds features
// 4*(t%16) .. +3 of rows t/16, t/16 + NT/16, ... (8-byte reads); the 4 row
// groups of a wave meet by two cross-lane swaps and each wave leaves 64
// partials in bred. After the next barrier wave 0 adds the waves' partials,
// writes the example's bias row for those features and keeps its square.
template <int ROWS, int NT>
__device__ __forceinline__ void bias_stage(const u32x4* st, float* bred, int tid) {
  const int q = tid & 15, c = q >> 1, h = q & 1;
  const u32x2* st2 = (const u32x2*)st;
  float sm[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < ROWS / (NT / 16); ++i) {
    const int r = (tid >> 4) + i * (NT / 16);
    const u32x2 v = st2[(r * 8 + swz(r, c)) * 2 + h];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      sm[2 * k] += __builtin_bit_cast(float, v[k] << 16);
      sm[2 * k + 1] += __builtin_bit_cast(float, v[k] & 0xFFFF0000u);
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) sm[e] = xor32_sum(xor16_sum(sm[e]));
  const int lane = tid & 63;
  if (lane < 16)
#pragma unroll
    for (int e = 0; e < 4; ++e) bred[(tid >> 6) * 64 + lane * 4 + e] = sm[e];
}

// Wave 0: features c0 .. c0+63 of the bias row `out` (up to c1); returns the
// square of this lane's feature.
template <int NT>
__device__ __forceinline__ float bias_finish(const float* bred, float* out, int64_t c0, int64_t c1,
                                             int tid) {
  if (tid >= 64) return 0.f;
  float v = 0.f;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) v += bred[w * 64 + tid];
  if (c0 + tid >= c1) return 0.f;
  out[c0 + tid] = v;
  return v * v;
}

template <int PAT, bool STREAM>
__device__ __forceinline__ float dg_item(const GramLayer& L, int b, int T, int ti, int tj,
                                         int chunk, u32x4* ring, float* bred) {
  constexpr int NB = PatNB<PAT>::NB;
  constexpr int ROWS = PatRows<PAT>::ROWS;        // 128 or 256
  constexpr int STB = ROWS * DG_ROWB;             // bytes per stage
  constexpr int LOADS = STB / 1024 / (GR_THREADS / WAVE);  // 1 KB loads per wave per stage
  constexpr int WROWS = ROWS / (GR_THREADS / WAVE);        // stage rows per wave
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint64_t ex_rows = (uint64_t)b * T;
  const uint32_t ldx = (uint32_t)(L.lda * 2), ldy = (uint32_t)(L.ldg * 2);
  const uint64_t xb = (uint64_t)L.A + ex_rows * ldx, yb = (uint64_t)L.G + ex_rows * ldy;
  const uint32_t nrx = T * ldx, nry = T * ldy;
  auto desc_of = [](uint64_t base, uint32_t nrec) {
    return u32x4{(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)base),
                 (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(base >> 32)),
                 (uint32_t)__builtin_amdgcn_readfirstlane((int)nrec), (uint32_t)RSRC_WORD3};
  };
  const u32x4 dx = desc_of(xb, nrx), dy = desc_of(yb, nry);
  const int64_t x1 = L.d_in;
  const int64_t y0 = (int64_t)L.g0 + (int64_t)chunk * L.kg;
  const int64_t y1 = y0 + L.kg < L.g1 ? y0 + L.kg : L.g1;
  const int nX = (int)((x1 + 63) / 64);
  const int nY = (int)((y1 - y0 + 63) / 64);
  const int n = nX + nY;
  const uint32_t ring_base = (uint32_t)(uintptr_t)(lds_void_g*)ring;

  // Wave w fills stage rows WROWS*w ..: load t writes rows r = WROWS*w + 8t +
  // l/8 at physical chunk l%8. Stage rows 0..127 are rows of tile ti, rows
  // 128..255 (off-diagonal pairs) rows of tile tj.
  const int lr = lane >> 3;
  const int wr0 = WROWS * w;                               // first stage row of this wave
  const int ex_row0 = (wr0 < GR_TM ? ti : tj) * GR_TM + (wr0 & (GR_TM - 1));
  auto issue = [&](int s) {
    const bool inX = s < nX;
    const u32x4 d = inX ? dx : dy;
    const uint32_t ld = inX ? ldx : ldy, nrec = inX ? nrx : nry;
    const int64_t c0 = inX ? (int64_t)s * 64 : y0 + (int64_t)(s - nX) * 64;
    const int64_t c1 = inX ? x1 : y1;
    const bool live = s < n;
    const uint32_t dst = ring_base + (uint32_t)((s % DG_NS) * STB) + (uint32_t)wr0 * DG_ROWB;
#pragma unroll
    for (int t = 0; t < LOADS; ++t) {
      const int r = wr0 + 8 * t + lr;
      const int c = (lane & 7) ^ ((r ^ (r >> 3)) & 7);
      const int64_t col = c0 + 8 * c;
      const uint32_t voff = (live && col < c1) ? (uint32_t)(lr * ld + col * 2) : nrec;
      const uint32_t m0v = (uint32_t)__builtin_amdgcn_readfirstlane((int)(dst + t * 1024));
      const uint32_t so =
          (uint32_t)__builtin_amdgcn_readfirstlane((int)((uint32_t)(ex_row0 + 8 * t) * ld));
      // Issued from asm so that the compiler does not drain all of them before
      // every LDS read; M0 has no other user in this kernel.
      if constexpr (STREAM)
        asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen sc1 nt lds"
                     :: "s"(m0v), "v"(voff), "s"(d), "s"(so));
      else
        asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen sc1 lds"
                     :: "s"(m0v), "v"(voff), "s"(d), "s"(so));
    }
  };
  // Zero the features at or past c1 inside the chunk that straddles c1.
  auto fix = [&](int s) {
    const bool inX = s < nX;
    const int64_t c0 = inX ? (int64_t)s * 64 : y0 + (int64_t)(s - nX) * 64;
    const int64_t c1 = inX ? x1 : y1;
    const int64_t nv = c1 - c0;  // valid features in this stage
    if (nv >= 64 || (nv & 7) == 0) return;
    if (tid < ROWS) {
      const int cp = (int)(nv >> 3), keep = (int)(nv & 7);
      u32x4* p = ring + (s % DG_NS) * (STB / 16) + tid * 8 + swz(tid, cp);
      u32x4 v = *p;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int e = 2 * q;
        v[q] = e + 1 < keep ? v[q] : (e < keep ? (v[q] & 0xFFFFu) : 0u);
      }
      *p = v;
    }
    __syncthreads();
  };

  int ra[4], rb[4];
  float wt[4];
  block_rows<PAT>(w, ra, rb, wt);
  using FP = std::conditional_t<PAT == PAT_OFF, FpOff,
                                std::conditional_t<PAT == PAT_D1, FpD1, FpD2>>;
  static_assert(FP::NB == NB, "block list");
  int rows[FP::NF];
  if constexpr (PAT == PAT_D1) {
    rows[0] = ra[0]; rows[1] = ra[2];
  } else if constexpr (PAT == PAT_D2) {
    rows[0] = ra[0]; rows[1] = rb[0]; rows[2] = rb[1];
  } else {
    rows[0] = ra[0]; rows[1] = ra[2]; rows[2] = rb[0]; rows[3] = rb[1];
  }
  f32x16 accP[NB], accQ[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) { accP[j][e] = 0.f; accQ[j][e] = 0.f; }

  // The bias applies to single-tile items (T <= 128), whose stages hold all
  // of the example's rows.
  float* const bout =
      (ROWS == GR_TM && T <= GR_TM && L.bias) ? L.bias + (int64_t)b * L.g1 : nullptr;
  float bsq = 0.f;
  auto g_c0 = [&](int s) { return y0 + (int64_t)(s - nX) * 64; };

  // Every iteration issues one stage's loads (past the end they read zeros into
  // a slot nobody reads), so the wait count is a constant.
#pragma unroll
  for (int p = 0; p < DG_NS - 1; ++p) issue(p);
  auto phase = [&](int s_begin, int s_end, f32x16 (&acc)[NB], bool with_bias) {
    for (int s = s_begin; s < s_end; ++s) {
      dg_wait_vmcnt<LOADS * (DG_NS - 2)>();
      __syncthreads();
      fix(s);
      if (with_bias && s > s_begin)
        bsq += bias_finish<GR_THREADS>(bred + ((s - 1) & 1) * GR_THREADS, bout, g_c0(s - 1), y1,
                                       tid);
      issue(s + DG_NS - 1);
      stage_mfma_fp<FP>(ring + (s % DG_NS) * (STB / 16), rows, acc, lane);
      if (with_bias)
        bias_stage<ROWS, GR_THREADS>(ring + (s % DG_NS) * (STB / 16),
                                     bred + (s & 1) * GR_THREADS, tid);
    }
  };
  phase(0, nX, accP, false);
  phase(nX, n, accQ, bout != nullptr);
  if (bout) {
    __syncthreads();
    bsq += bias_finish<GR_THREADS>(bred + ((n - 1) & 1) * GR_THREADS, bout, g_c0(n - 1), y1, tid);
  }
  // No load may still be writing LDS when the workgroup moves on.
  dg_wait_vmcnt<0>();
  float part = bsq;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) s += accP[j][e] * accQ[j][e];
    part += wt[j] * s;
  }
  return part;
}

template <bool SINGLE>
__global__ __launch_bounds__(GR_THREADS, SINGLE ? 2 : 1) void dl_gram_kernel(GramArgs args) {
  const GramArgs& a = *(const GramArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  (void)args;
  __shared__ __attribute__((aligned(1024))) u32x4 ring[DG_NS * (SINGLE ? GR_TM : GR_ROWS) * 8];
  __shared__ float red[GR_THREADS / WAVE];
  __shared__ float bred[SINGLE ? 2 * GR_THREADS : 1];
  const uint32_t item = xcd_remap(blockIdx.x, gridDim.x);
  const GramItem gi = gram_item(a, item);
  const GramLayer& L = a.L[gi.l];
  const int b = gi.b;
  const int pair = (int)(gi.rel / (uint32_t)L.nc);
  const int chunk = (int)(gi.rel - (uint32_t)pair * L.nc);
  int ti = 0, rem = pair;
  while (rem >= a.n_t - ti) { rem -= a.n_t - ti; ++ti; }
  const int tj = ti + rem;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  float part;
  if (!SINGLE && ti != tj)
    part = dg_item<PAT_OFF, false>(L, b, a.T, ti, tj, chunk, ring, bred);
  else if (w < 2)
    part = dg_item<PAT_D1, SINGLE>(L, b, a.T, ti, tj, chunk, ring, bred);
  else
    part = dg_item<PAT_D2, SINGLE>(L, b, a.T, ti, tj, chunk, ring, bred);
  part = wave_sum(part);
  if ((threadIdx.x & 63) == 0) red[w] = part;
  __syncthreads();
  if (threadIdx.x == 0)
    a.ws[(int64_t)b * a.slots + L.slot_begin + pair * L.nc + chunk] =
        (red[0] + red[1]) + (red[2] + red[3]);
}

// Whole-example variant for 128 < T <= 256 (bf16, aligned rows): 8 waves
// reduce all 36 upper 32x32 blocks of the 256 x 256 Gram, so every row is
// read once (pair items would read each T-tile twice). The blocks of row
// pair {g, 7-g} (9 of them) go to waves g (5 blocks) and g+4 (4 blocks), so
// each SIMD carries 9. Stages are 256 rows x 64 features (32 KB), four in a
// ring, one workgroup per CU.
constexpr int DW_NS = 4;
constexpr int DW_THREADS = 512;
constexpr int DW_ROWS = 2 * GR_TM;
constexpr int DW_STB = DW_ROWS * DG_ROWB;
constexpr int DW_LOADS = DW_STB / 1024 / (DW_THREADS / WAVE);
static_assert(DW_LOADS * 8 * (DW_THREADS / WAVE) == DW_ROWS, "rows per load");

template <class P>
__device__ __forceinline__ float dw_item(const GramLayer& L, int b, int T, int chunk, u32x4* ring,
                                         float* bred) {
  constexpr int NB = P::NB;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint64_t ex_rows = (uint64_t)b * T;
  const uint32_t ldx = (uint32_t)(L.lda * 2), ldy = (uint32_t)(L.ldg * 2);
  const uint64_t xb = (uint64_t)L.A + ex_rows * ldx, yb = (uint64_t)L.G + ex_rows * ldy;
  const uint32_t nrx = T * ldx, nry = T * ldy;
  auto desc_of = [](uint64_t base, uint32_t nrec) {
    return u32x4{(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)base),
                 (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(base >> 32)),
                 (uint32_t)__builtin_amdgcn_readfirstlane((int)nrec), (uint32_t)RSRC_WORD3};
  };
  const u32x4 dx = desc_of(xb, nrx), dy = desc_of(yb, nry);
  const int64_t x1 = L.d_in;
  const int64_t y0 = (int64_t)L.g0 + (int64_t)chunk * L.kg;
  const int64_t y1 = y0 + L.kg < L.g1 ? y0 + L.kg : L.g1;
  const int nX = (int)((x1 + 63) / 64);
  const int nY = (int)((y1 - y0 + 63) / 64);
  const int n = nX + nY;
  const uint32_t ring_base = (uint32_t)(uintptr_t)(lds_void_g*)ring;

  // Wave w fills stage rows 32w .. 32w+31 (example rows; past T they read 0).
  const int lr = lane >> 3;
  const int wr0 = 32 * w;
  auto issue = [&](int s) {
    const bool inX = s < nX;
    const u32x4 d = inX ? dx : dy;
    const uint32_t ld = inX ? ldx : ldy, nrec = inX ? nrx : nry;
    const int64_t c0 = inX ? (int64_t)s * 64 : y0 + (int64_t)(s - nX) * 64;
    const int64_t c1 = inX ? x1 : y1;
    const bool live = s < n;
    const uint32_t dst = ring_base + (uint32_t)((s % DW_NS) * DW_STB) + (uint32_t)wr0 * DG_ROWB;
#pragma unroll
    for (int t = 0; t < DW_LOADS; ++t) {
      const int r = wr0 + 8 * t + lr;
      const int c = (lane & 7) ^ ((r ^ (r >> 3)) & 7);
      const int64_t col = c0 + 8 * c;
      const uint32_t voff = (live && col < c1) ? (uint32_t)(lr * ld + col * 2) : nrec;
      const uint32_t m0v = (uint32_t)__builtin_amdgcn_readfirstlane((int)(dst + t * 1024));
      const uint32_t so =
          (uint32_t)__builtin_amdgcn_readfirstlane((int)((uint32_t)(wr0 + 8 * t) * ld));
      // Issued from asm so that the compiler does not drain all of them before
      // every LDS read; M0 has no other user in this kernel.
      asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen sc1 nt lds"
                   :: "s"(m0v), "v"(voff), "s"(d), "s"(so));
    }
  };
  auto fix = [&](int s) {
    const bool inX = s < nX;
    const int64_t c0 = inX ? (int64_t)s * 64 : y0 + (int64_t)(s - nX) * 64;
    const int64_t c1 = inX ? x1 : y1;
    const int64_t nv = c1 - c0;
    if (nv >= 64 || (nv & 7) == 0) return;
    if (tid < DW_ROWS) {
      const int cp = (int)(nv >> 3), keep = (int)(nv & 7);
      u32x4* p = ring + (s % DW_NS) * (DW_STB / 16) + tid * 8 + swz(tid, cp);
      u32x4 v = *p;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int e = 2 * q;
        v[q] = e + 1 < keep ? v[q] : (e < keep ? (v[q] & 0xFFFFu) : 0u);
      }
      *p = v;
    }
    __syncthreads();
  };

  // Block list: entry k of row pair g is (g, g+k) for k < 8-g, else
  // (7-g, 7-g + k-(8-g)); wave g takes entries 0..4, wave g+4 entries 5..8
  // (the patterns FpW0 .. FpW7 list them by fragment).
  const int g = w & 3;
  int rows[P::NF];
#pragma unroll
  for (int q = 0; q < P::NF; ++q) rows[q] = P::row(g, q);
  float wt[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) wt[j] = P::ia(j) == P::ib(j) ? 1.f : 2.f;
  f32x16 accP[NB], accQ[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) { accP[j][e] = 0.f; accQ[j][e] = 0.f; }

  float* const bout = L.bias ? L.bias + (int64_t)b * L.g1 : nullptr;
  float bsq = 0.f;
  auto g_c0 = [&](int s) { return y0 + (int64_t)(s - nX) * 64; };
#pragma unroll
  for (int p = 0; p < DW_NS - 1; ++p) issue(p);
  auto phase = [&](int s_begin, int s_end, f32x16 (&acc)[NB], bool with_bias) {
    for (int s = s_begin; s < s_end; ++s) {
      dg_wait_vmcnt<DW_LOADS * (DW_NS - 2)>();
      __syncthreads();
      fix(s);
      if (with_bias && s > s_begin)
        bsq += bias_finish<DW_THREADS>(bred + ((s - 1) & 1) * DW_THREADS, bout, g_c0(s - 1), y1,
                                       tid);
      issue(s + DW_NS - 1);
      stage_mfma_fp<P>(ring + (s % DW_NS) * (DW_STB / 16), rows, acc, lane);
      if (with_bias)
        bias_stage<DW_ROWS, DW_THREADS>(ring + (s % DW_NS) * (DW_STB / 16),
                                        bred + (s & 1) * DW_THREADS, tid);
    }
  };
  phase(0, nX, accP, false);
  phase(nX, n, accQ, bout != nullptr);
  if (bout) {
    __syncthreads();
    bsq += bias_finish<DW_THREADS>(bred + ((n - 1) & 1) * DW_THREADS, bout, g_c0(n - 1), y1, tid);
  }
  dg_wait_vmcnt<0>();
  float part = bsq;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) s += accP[j][e] * accQ[j][e];
    part += wt[j] * s;
  }
  return part;
}

__global__ __launch_bounds__(DW_THREADS) void dl_gram_whole_kernel(GramArgs args) {
  const GramArgs& a = *(const GramArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  (void)args;
  __shared__ __attribute__((aligned(1024))) u32x4 ring[DW_NS * DW_STB / 16];
  __shared__ float bred[2 * DW_THREADS];
  // The partial sums reuse the ring: every load has landed by then.
  float* red = (float*)ring;
  const uint32_t item = xcd_remap(blockIdx.x, gridDim.x);
  const GramItem gi = gram_item(a, item);
  const GramLayer& L = a.L[gi.l];
  const int b = gi.b;
  const int chunk = (int)gi.rel;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  float part;
  switch (w) {
    case 4: part = dw_item<FpW4>(L, b, a.T, chunk, ring, bred); break;
    case 5: part = dw_item<FpW5>(L, b, a.T, chunk, ring, bred); break;
    case 6: part = dw_item<FpW6>(L, b, a.T, chunk, ring, bred); break;
    case 7: part = dw_item<FpW7>(L, b, a.T, chunk, ring, bred); break;
    default: part = dw_item<FpW0>(L, b, a.T, chunk, ring, bred); break;
  }
  part = wave_sum(part);
  __syncthreads();  // every wave is done reading the ring
  if ((threadIdx.x & 63) == 0) red[w] = part;
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = 0.f;
#pragma unroll
    for (int q = 0; q < DW_THREADS / WAVE; ++q) t += red[q];
    a.ws[(int64_t)b * a.slots + L.slot_begin + chunk] = t;
  }
}

// Direct-load cross term (bf16, aligned rows). Work item = (example b,
// 64-row block qi of dE, 64-row block qj of H), over all d features, so the
// logit gradients are gathered once per product element. A stage holds 64
// features of the 64 dE rows (stage rows 0..63) and the 64 H rows (64..127),
// four stages in a ring, two workgroups per CU; wave w owns the 32x32 block
// (dE rows 32*(w&1), H rows 32*(w>>1)) of the 64x64 product.
constexpr int DC_ROWS = 128;
constexpr int DC_STB = DC_ROWS * DG_ROWB;     // 16 KB
constexpr int DC_LOADS = DC_STB / 1024 / (GR_THREADS / WAVE);

__global__ __launch_bounds__(GR_THREADS, 2) void dl_cross_kernel(CrossArgs a) {
  __shared__ __attribute__((aligned(1024))) u32x4 ring[DG_NS * DC_STB / 16];
  __shared__ float red[GR_THREADS / WAVE];
  const uint32_t item = xcd_remap(blockIdx.x, gridDim.x);
  const int b = (int)(item / (uint32_t)a.slots);
  const int slot = (int)(item - (uint32_t)b * a.slots);
  const int nq = a.n_t;  // 64-row blocks per example in this kernel
  const int qi = slot / nq, qj = slot - qi * nq;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int T = a.T;
  const uint64_t ex_rows = (uint64_t)b * T;
  const uint32_t lde = (uint32_t)(a.lde * 2), ldh = (uint32_t)(a.ldh * 2);
  auto desc_of = [](uint64_t base, uint32_t nrec) {
    return u32x4{(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)base),
                 (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(base >> 32)),
                 (uint32_t)__builtin_amdgcn_readfirstlane((int)nrec), (uint32_t)RSRC_WORD3};
  };
  const bool load_e = w < 2;  // waves 0-1 load dE rows, 2-3 H rows
  const uint32_t ld = load_e ? lde : ldh;
  const uint32_t nrec = (uint32_t)T * ld;
  const u32x4 d = desc_of((uint64_t)(load_e ? a.E : a.H) + ex_rows * ld, nrec);
  const int wr0 = 32 * w;                                   // first stage row of this wave
  const int ex_row0 = (load_e ? qi : qj) * 64 + (wr0 & 63); // its example row
  const int n = (a.d + 63) / 64;
  const uint32_t ring_base = (uint32_t)(uintptr_t)(lds_void_g*)ring;
  const int lr = lane >> 3;
  auto issue = [&](int s) {
    const int64_t c0 = (int64_t)s * 64;
    const bool live = s < n;
    const uint32_t dst = ring_base + (uint32_t)((s % DG_NS) * DC_STB) + (uint32_t)wr0 * DG_ROWB;
#pragma unroll
    for (int t = 0; t < DC_LOADS; ++t) {
      const int r = wr0 + 8 * t + lr;
      const int c = (lane & 7) ^ ((r ^ (r >> 3)) & 7);
      const int64_t col = c0 + 8 * c;
      const uint32_t voff = (live && col < a.d) ? (uint32_t)(lr * ld + col * 2) : nrec;
      const uint32_t m0v = (uint32_t)__builtin_amdgcn_readfirstlane((int)(dst + t * 1024));
      const uint32_t so =
          (uint32_t)__builtin_amdgcn_readfirstlane((int)((uint32_t)(ex_row0 + 8 * t) * ld));
      // Issued from asm so that the compiler does not drain all of them before
      // every LDS read; M0 has no other user in this kernel.
      asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen sc1 nt lds"
                   :: "s"(m0v), "v"(voff), "s"(d), "s"(so));
    }
  };
  auto fix = [&](int s) {
    const int64_t nv = (int64_t)a.d - (int64_t)s * 64;
    if (nv >= 64 || (nv & 7) == 0) return;
    if (tid < DC_ROWS) {
      const int cp = (int)(nv >> 3), keep = (int)(nv & 7);
      u32x4* p = ring + (s % DG_NS) * (DC_STB / 16) + tid * 8 + swz(tid, cp);
      u32x4 v = *p;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int e = 2 * q;
        v[q] = e + 1 < keep ? v[q] : (e < keep ? (v[q] & 0xFFFFu) : 0u);
      }
      *p = v;
    }
    __syncthreads();
  };

  int ra[1] = {32 * (w & 1)}, rb[1] = {64 + 32 * (w >> 1)};
  f32x16 acc[1];
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[0][e] = 0.f;
#pragma unroll
  for (int p = 0; p < DG_NS - 1; ++p) issue(p);
  for (int s = 0; s < n; ++s) {
    dg_wait_vmcnt<DC_LOADS * (DG_NS - 2)>();
    __syncthreads();
    fix(s);
    issue(s + DG_NS - 1);
    stage_mfma<DT_BF16, 1>(ring + (s % DG_NS) * (DC_STB / 16), ra, rb, acc, lane);
  }
  dg_wait_vmcnt<0>();

  // acc holds P[t, s] = <dE_t, H_s>: lane l has s = l%32 of the block and,
  // for accumulator e, t = (e/4)*8 + (l/32)*4 + e%4. Logit gradients are
  // gathered through a range-checked buffer over this example's rows of Gz.
  const uint32_t ldz = (uint32_t)(a.ldz * 2);
  const rsrc_t rZ = make_rsrc((const char*)a.Gz + ex_rows * ldz, (uint64_t)T * ldz);
  const int s_row = qj * 64 + 32 * (w >> 1) + (lane & 31);
  const int t0 = qi * 64 + 32 * (w & 1) + (lane >> 5) * 4;
  float part = 0.f;
  if (s_row < T) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int t = t0 + (e >> 2) * 8 + (e & 3);
      if (t < T) {
        const uint32_t v = (uint32_t)a.ids[ex_rows + t];
        if (v < (uint32_t)a.V)  // an invalid id contributes nothing
          part += acc[0][e] * bf16_to_f32((uint16_t)buf_load2(rZ, (uint32_t)s_row * ldz + v * 2));
      }
    }
  }
  part = wave_sum(part);
  if (lane == 0) red[w] = part;
  __syncthreads();
  if (tid == 0) a.ws[(int64_t)b * a.slots + slot] = (red[0] + red[1]) + (red[2] + red[3]);
}

// Register-direct cross term (bf16, 16-byte aligned rows). Work item =
// (example b, block tb of 32 tokens, block sb of 32 rows of H): the 32 x 32
// block P[s, t] = <h_s, dE_t> on MFMA, each of the 8 waves over an eighth of
// the features with its operands loaded straight into registers (no LDS
// staging: a lane's 8 consecutive features are one 16-byte load), the parts
// added in LDS in a fixed order, then sum P[s, t] Gz[s, x_t]. In the MFMA
// output a lane holds one token t and 16 rows s, so one gather instruction
// reads two rows of Gz at 32 columns x_t (equal ids share an address). Every
// load is issued at the start: the H and dE rows and the ids depend on
// nothing, the gathers only on the ids. (Ranking the tokens by id first, for
// gathers at ascending columns, fetched no fewer bytes and took ~1 us more.)
constexpr int CX_THREADS = 512;
constexpr int CX_NW = CX_THREADS / WAVE;
constexpr int CX_KB = 6;  // 16-feature MFMA steps whose loads a wave issues together
static_assert(16 % CX_NW == 0, "accumulators finished per wave");

__global__ __launch_bounds__(CX_THREADS) void cross_rows_kernel(CrossArgs a) {
  __shared__ float part[CX_NW / 2][16][WAVE];  // 16 KB: leaves room beside a Gram launch
  __shared__ float red[CX_NW];
  const uint32_t item = xcd_remap(blockIdx.x, gridDim.x);
  const int nb = a.n_t;
  const int b = (int)(item / (uint32_t)a.slots);
  const int slot = (int)(item - (uint32_t)b * a.slots);
  const int tb = slot / nb, sb = slot - tb * nb;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int T = a.T;
  const uint32_t V = (uint32_t)a.V;
  const int t_lo = tb * CR_RX_ROWS;
  const int r = lane & 31, h = lane >> 5;
  const uint64_t ex_rows = (uint64_t)b * T;
  const uint32_t lde = (uint32_t)(a.lde * 2), ldh = (uint32_t)(a.ldh * 2);
  const rsrc_t rE = make_rsrc((const char*)a.E + ex_rows * lde, (uint64_t)T * lde);
  const rsrc_t rH = make_rsrc((const char*)a.H + ex_rows * ldh, (uint64_t)T * ldh);
  const rsrc_t rI = make_rsrc(a.ids + ex_rows, (uint64_t)T * 4);
  const int nk = (a.d + 15) / 16;         // 16-feature MFMA steps
  const int kq = (nk + CX_NW - 1) / CX_NW;  // per wave
  const int k0 = min(w * kq, nk), k1 = min(k0 + kq, nk);
  // Rows past the example read zeros through offsets past the range. A lane
  // takes features 16k + 8h .. +7 of its row in both operands; the chunk
  // that straddles d is zeroed on both sides.
  const int s_row = sb * CR_RX_ROWS + r, t_row = t_lo + r;
  const bool t_ok = t_row < T;
  const uint32_t hoff = s_row < T ? (uint32_t)s_row * ldh : (uint32_t)T * ldh;
  const uint32_t eoff = t_ok ? (uint32_t)t_row * lde : (uint32_t)T * lde;
  auto load_op = [&](rsrc_t rs, uint32_t roff, uint32_t end, int k) {
    const int f = k * 16 + 8 * h;
    const bool live = k < k1 && f < a.d;
    return buf_load16(rs, live ? roff + (uint32_t)f * 2 : end);
  };
  // Applied after a batch is issued, and only when d is not a multiple of 8,
  // so that no load waits for the one before it.
  const bool straddle = (a.d & 7) != 0;
  auto mask_op = [&](u32x4& v, int k) {
    const int nv = a.d - (k * 16 + 8 * h);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e2 = 2 * q;
      v[q] &= e2 + 1 < nv ? 0xFFFFFFFFu : (e2 < nv ? 0xFFFFu : 0u);
    }
  };
  // The id of this lane's token first (loads complete in order), then the
  // first batch of H and dE rows.
  const uint32_t id_raw = buf_load4(rI, t_ok ? (uint32_t)t_row * 4 : (uint32_t)T * 4);
  u32x4 fh[CX_KB], fe[CX_KB];
#pragma unroll
  for (int j = 0; j < CX_KB; ++j) {
    fh[j] = load_op(rH, hoff, (uint32_t)T * ldh, k0 + j);
    fe[j] = load_op(rE, eoff, (uint32_t)T * lde, k0 + j);
  }
  __builtin_amdgcn_sched_barrier(0);  // keep the wait for the id after these loads
  // The logit gradients this wave multiplies in the end: wave w finishes
  // accumulators e = EPW*w .. +EPW-1 of the block, row s = sb*32 + 8(e/4) +
  // 4h + e%4, token t_row.
  constexpr int EPW = 16 / CX_NW;
  const uint32_t ldz = (uint32_t)(a.ldz * 2);
  const rsrc_t rZ = make_rsrc((const char*)a.Gz + ex_rows * ldz, (uint64_t)T * ldz);
  const uint32_t v = t_ok ? id_raw : V;
  uint32_t zr[EPW];
#pragma unroll
  for (int i = 0; i < EPW; ++i) {
    const int e = EPW * w + i;
    const int s = sb * CR_RX_ROWS + 8 * (e >> 2) + 4 * h + (e & 3);
    // an invalid id, or a row or token past T, reads zero past the range
    zr[i] = buf_load2(rZ, (v < V && s < T) ? (uint32_t)s * ldz + v * 2 : (uint32_t)T * ldz);
  }
  f32x16 acc;
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.f;
  for (int kb = k0; kb < k1; kb += CX_KB) {
    if (kb != k0) {
#pragma unroll
      for (int j = 0; j < CX_KB; ++j) {
        fh[j] = load_op(rH, hoff, (uint32_t)T * ldh, kb + j);
        fe[j] = load_op(rE, eoff, (uint32_t)T * lde, kb + j);
      }
    }
    if (straddle) {
#pragma unroll
      for (int j = 0; j < CX_KB; ++j) {
        mask_op(fh[j], kb + j);
        mask_op(fe[j], kb + j);
      }
    }
#pragma unroll
    for (int j = 0; j < CX_KB; ++j) acc = mfma32_bf16(fh[j], fe[j], acc);
  }
  // The waves' parts of each accumulator meet in a fixed order in half as
  // much LDS: wave w + CX_NW/2 hands its part to wave w, which adds it; then
  // every wave sums the CX_NW/2 pair sums of its EPW accumulators in order.
  constexpr int NH = CX_NW / 2;
  if (w >= NH) {
#pragma unroll
    for (int e = 0; e < 16; ++e) part[w - NH][e][lane] = acc[e];
  }
  __syncthreads();
  if (w < NH) {
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] += part[w][e][lane];
  }
  __syncthreads();
  if (w < NH) {
#pragma unroll
    for (int e = 0; e < 16; ++e) part[w][e][lane] = acc[e];
  }
  __syncthreads();
  float sum = 0.f;
#pragma unroll
  for (int i = 0; i < EPW; ++i) {
    float pv = part[0][EPW * w + i][lane];
#pragma unroll
    for (int q = 1; q < NH; ++q) pv += part[q][EPW * w + i][lane];
    sum += pv * bf16_to_f32((uint16_t)zr[i]);
  }
  sum = wave_sum(sum);
  if (lane == 0) red[w] = sum;
  __syncthreads();
  if (tid == 0) {
    float t = 0.f;
#pragma unroll
    for (int q = 0; q < CX_NW; ++q) t += red[q];
    a.ws[(int64_t)b * a.slots + slot] = t;
  }
}

// Work item = (example, T-tile pair (ti, tj), chunk of CR_FCHUNK features).
// The reduction is linear in the features, so chunks add up exactly.
template <int DT, bool VEC>
__global__ __launch_bounds__(GR_THREADS) void tied_cross_kernel(CrossArgs a) {
  __shared__ u32x4 lds[GR_ROWS * 8];
  __shared__ float red[GR_THREADS / WAVE];
  using TS = TileStream<DT, VEC>;
  constexpr int EPC = TS::EPC, KS = TS::KS, ES = TS::ES;
  const uint32_t item = xcd_remap(blockIdx.x, gridDim.x);
  const int b = (int)(item / (uint32_t)a.slots);
  const int slot = (int)(item - (uint32_t)b * a.slots);
  const int pair = slot / a.n_fc, fc = slot - pair * a.n_fc;
  const int ti = pair / a.n_t, tj = pair - ti * a.n_t;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int T = a.T;

  // LDS rows 0..127: dE rows of tile ti; rows 128..255: H rows of tile tj,
  // both loaded in the same stage through per-example buffer resources.
  const uint64_t ex_rows = (uint64_t)b * T;
  const uint32_t lde = (uint32_t)(a.lde * ES), ldh = (uint32_t)(a.ldh * ES);
  const rsrc_t rE = make_rsrc((const char*)a.E + ex_rows * lde, (uint64_t)T * lde);
  const rsrc_t rH = make_rsrc((const char*)a.H + ex_rows * ldh, (uint64_t)T * ldh);
  const uint32_t r0 = tid >> 3, c = tid & 7;
  const uint32_t ve = (ti * GR_TM + r0) * lde + c * 16;
  const uint32_t vh = (tj * GR_TM + r0) * ldh + c * 16;
  const int64_t f0 = (int64_t)fc * CR_FCHUNK;
  const int64_t f1 = f0 + CR_FCHUNK < a.d ? f0 + CR_FCHUNK : a.d;
  const int n = (int)((f1 - f0 + KS - 1) / KS);

  int ra[4], rb[4];
  float wt[4];
  block_rows<PAT_OFF>(w, ra, rb, wt);
  f32x16 acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[j][e] = 0.f;

  u32x4 pre[8];
  auto fetch = [&](int s) {
    const int64_t c0 = f0 + (int64_t)s * KS;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const bool lo = i < 4;
      const uint32_t soff = (uint32_t)(c0 * ES) + (uint32_t)(32 * (i & 3)) * (lo ? lde : ldh);
      pre[i] = buf_chunk<DT, VEC, true>(lo ? rE : rH, lo ? ve : vh, soff, c0 + c * EPC, f1);
    }
  };
  fetch(0);
  for (int s = 0; s < n; ++s) {
    __syncthreads();
    store_stage<8>(lds, pre, tid);
    __syncthreads();
    if (s + 1 < n) fetch(s + 1);
    stage_mfma<DT, 4>(lds, ra, rb, acc, lane);
  }

  // Block j holds P[t, s] = <dE_t, H_s> (this feature chunk): lane l has
  // column s = l%32 and, for accumulator e, row (e/4)*8 + (l/32)*4 + e%4 of
  // the 32x32 MFMA output. Logit gradients are gathered through a buffer
  // resource spanning this example's rows of Gz.
  const uint32_t ldz = (uint32_t)(a.ldz * ES);
  const rsrc_t rZ = make_rsrc((const char*)a.Gz + ex_rows * ldz, (uint64_t)T * ldz);
  float part = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int t0 = ti * GR_TM + ra[j] + (lane >> 5) * 4;
    const int s = tj * GR_TM + (rb[j] - GR_TM) + (lane & 31);
    if (s >= T) continue;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int t = t0 + (e >> 2) * 8 + (e & 3);
      if (t < T) {
        const uint32_t v = (uint32_t)a.ids[ex_rows + t];
        if (v >= (uint32_t)a.V) continue;  // invalid id: contributes nothing
        const uint32_t off = (uint32_t)s * ldz + v * ES;
        float g;
        if constexpr (DT == DT_BF16)
          g = bf16_to_f32((uint16_t)buf_load2(rZ, off));
        else
          g = __uint_as_float(buf_load4(rZ, off));
        part += acc[j][e] * g;
      }
    }
  }
  part = wave_sum(part);
  if (lane == 0) red[w] = part;
  __syncthreads();
  if (tid == 0) a.ws[(int64_t)b * a.slots + slot] = (red[0] + red[1]) + (red[2] + red[3]);
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
template <int DT>
static void launch_gram_dt(const GramArgs& a, bool vec, hipStream_t s) {
  const dim3 g(a.n_items), blk(GR_THREADS);
  const bool single = a.n_t == 1;
  if constexpr (DT == DT_BF16) {
    if (vec) {
      if (single) hipLaunchKernelGGL(dl_gram_kernel<true>, g, blk, 0, s, a);
      else if (gram_whole(DT, vec, a.T))
        hipLaunchKernelGGL(dl_gram_whole_kernel, g, dim3(DW_THREADS), 0, s, a);
      else hipLaunchKernelGGL(dl_gram_kernel<false>, g, blk, 0, s, a);
      return;
    }
  }
  if (vec) {
    if (single) hipLaunchKernelGGL((gram_norm_kernel<DT, true, true>), g, blk, 0, s, a);
    else hipLaunchKernelGGL((gram_norm_kernel<DT, true, false>), g, blk, 0, s, a);
  } else {
    if (single) hipLaunchKernelGGL((gram_norm_kernel<DT, false, true>), g, blk, 0, s, a);
    else hipLaunchKernelGGL((gram_norm_kernel<DT, false, false>), g, blk, 0, s, a);
  }
}

hipError_t launch_gram_norm(const GramArgs& a, int dt, bool vec, hipStream_t s) {
  if (a.n_items == 0) return hipSuccess;
  if (dt == DT_BF16)
    launch_gram_dt<DT_BF16>(a, vec, s);
  else
    launch_gram_dt<DT_F32>(a, vec, s);
  return hipGetLastError();
}

hipError_t launch_tied_cross(const CrossArgs& a, int dt, bool vec, hipStream_t s) {
  const uint32_t n = (uint32_t)a.B * (uint32_t)a.slots;
  if (n == 0) return hipSuccess;
  const dim3 g(n), blk(GR_THREADS);
  if (dt == DT_BF16) {
    if (a.kind == CROSS_ROWS) hipLaunchKernelGGL(cross_rows_kernel, g, dim3(CX_THREADS), 0, s, a);
    else if (a.kind == CROSS_DL) hipLaunchKernelGGL(dl_cross_kernel, g, blk, 0, s, a);
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
