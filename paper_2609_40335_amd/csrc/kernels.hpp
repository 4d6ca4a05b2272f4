// Internal launch interface between the C ABI (api.cpp) and the HIP kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dpg {

enum { DT_F32 = 0, DT_BF16 = 1 };  // element type of the float operands

// ----------------------------------------------------------------- Gram norm
constexpr int GR_TM = 128;          // rows of one T-tile
constexpr int GR_MAX_LAYERS = 52;   // layers per launch (kernel arguments stay < 4 KiB)
// bf16 launches with aligned rows and 128 < T <= 256 reduce each example's
// whole 256 x 256 Gram in one work item (one partial slot per chunk) instead
// of one item per T-tile pair.
inline bool gram_whole(int dt, bool vec, int T) {
  return dt == DT_BF16 && vec && T > GR_TM && T <= 2 * GR_TM;
}
// Gram workgroups resident per CU: two for the single-tile direct-load kernel
// (bf16, 16-byte rows, T <= 128), one for the others.
inline int gram_groups_per_cu(int dt, bool vec, int T) {
  return dt == DT_BF16 && vec && T <= GR_TM ? 2 : 1;
}
// Gram launches that can fuse a layer's bias gradient (every example row of
// a stage is in LDS at once).
inline bool gram_fuses_bias(int dt, bool vec, int T) {
  return dt == DT_BF16 && vec && T <= 2 * GR_TM;
}

struct GramLayer {
  const void* A;        // [B*T rows, lda] activations
  const void* G;        // [B*T rows, ldg] output grads
  int64_t lda, ldg;
  int32_t d_in;         // A features
  int32_t g0, g1;       // G feature range of this entry
  int32_t kg;           // G features per chunk
  int32_t nc;           // number of G chunks
  uint32_t item_begin;  // first work item of this layer among an example's items
  int32_t slot_begin;   // first partial slot of this layer in an example's row
  // The layer's bias gradient, fused (bf16, 16-byte rows, T <= 256 only):
  // row b of [B, g1] gets sum_t G[b,t,:], and its squared norm joins the
  // example's partial sums. Null: no bias.
  float* bias;
};

// Work items are numbered example-major: example b owns items
// [b * per_ex, (b + 1) * per_ex), one per (layer, T-tile pair, G chunk), so
// that the contiguous item range each XCD walks holds whole examples (equal
// work per XCD, and an example's G chunks share its A rows in one L2).
struct GramArgs {
  GramLayer L[GR_MAX_LAYERS];
  int32_t n_layers;
  int32_t B, T, n_t, P;   // T-tiles per side, upper-triangle tile pairs
  int32_t slots;          // partial slots per example
  uint32_t per_ex;        // work items per example
  uint32_t n_items;
  float* ws;              // [B, slots]
};

static_assert(sizeof(GramArgs) <= 4096, "kernel arguments must stay within 4 KiB");
hipError_t launch_gram_norm(const GramArgs& a, int dt, bool vec, hipStream_t s);

// Tied cross term: sum_{t,s} Gz[s, ids[t]] <dE_t, H_s>, all T-tile pairs.
constexpr int CR_FCHUNK = 128;  // features per cross-term work item
constexpr int CR_DL_ROWS = 64;  // row block of the direct-load cross kernel
constexpr int CR_RX_ROWS = 32;  // token and row blocks of the register-direct cross kernel
constexpr int CX_ROWS_T = 128;  // longest example given to it (measured: at T = 256 its
                                // 32-row blocks re-read E and H more than dl_cross's 64-row ones)
// Cross-term kernel of a call: the register-staged tied_cross_kernel (fp32 or
// unaligned rows), the register-direct cross_rows_kernel (bf16, aligned rows,
// T <= CX_ROWS_T) or the direct-load dl_cross_kernel (bf16, aligned, longer T).
enum { CROSS_STAGED = 0, CROSS_DL = 1, CROSS_ROWS = 2 };
inline int cross_kind(int dt, bool vec, int T) {
  if (dt != DT_BF16 || !vec) return CROSS_STAGED;
  return T <= CX_ROWS_T ? CROSS_ROWS : CROSS_DL;
}

struct CrossArgs {
  const int32_t* ids;   // [B,T]
  const void* E;        // dE [B*T, lde]
  const void* H;        // [B*T, ldh]
  const void* Gz;       // [B*T, ldz]
  int64_t lde, ldh, ldz;
  int32_t B, T, V, d, n_t;  // n_t: row blocks per example (128, 64 or 32 rows by kernel)
  int32_t n_fc;         // feature chunks (1 for bf16 aligned: all features per item)
  int32_t kind;         // CROSS_STAGED, CROSS_DL or CROSS_ROWS
  int32_t slots;        // n_t * n_t * n_fc
  float* ws;            // [B, slots]
};
hipError_t launch_tied_cross(const CrossArgs& a, int dt, bool vec, hipStream_t s);

// out[b] = (acc ? out[b] : 0) + scale * sum_j ws[b*slots + j], fixed order.
hipError_t launch_finish_rows(const float* ws, int B, int slots, float* out, int accumulate,
                              float scale, hipStream_t s);

// ------------------------------------------------------- K-major GEMM family
constexpr int GM_BM = 256, GM_BN = 256;
constexpr int GM_MAX_LAYERS = 52;   // layers per launch (kernel arguments stay < 4 KiB)

struct GemmLayer {
  const void* X;        // [K rows, ldx]
  const void* Y;        // [K rows, ldy]
  float* out;           // clipped sum: [M, ldo] or transposed [N, ldo]
  union {
    int64_t ldx;          // row stride of X in elements
    int64_t store_slot;   // sum from a gradient store (X, Y unread): first tile slot
  };
  union {
    int64_t ldy;          // row stride of Y in elements
    int64_t store_transpose;  // sum from a gradient store: 1 = output [N, ldo]
  };
  int64_t ldo;          // row stride of out in elements
  int32_t M, N;         // X columns (output rows) and Y columns (output columns)
  uint16_t tm, tn;      // 256-wide tiles along M and N
  uint32_t tile_begin;  // first work item of this entry
  union {
    int32_t slot_begin;   // direct norm: first partial slot in an example's row
    uint32_t tensor_id;   // clipped sum with noise: the tensor's generator id
  };
  int32_t accumulate;   // clipped sum: out += (else out =)
};

struct GemmArgs {
  GemmLayer L[GM_MAX_LAYERS];
  int32_t n_layers;
  int32_t B, T;
  uint32_t n_items;
  int32_t transpose;    // clipped sum: output layout
  const float* c;       // clipped sum: per-example scale [B]
  float* ws;            // direct norm: [B, slots]
  int32_t slots;
  // Gaussian mechanism fused into the clipped sum's store (noise != 0):
  // out = (prior + sum + sigma_c * z) * inv_b, z from Philox (seed, tensor_id,
  // step) at the element's row-major index in the output tensor.
  int32_t noise;
  float sigma_c, inv_b;
  uint32_t step;
  uint64_t seed;
  // Tail split of the clipped sum (direct-load kernel): tiles [0, n_full) are
  // whole work items; each of the n_split tiles after them is ksplit items
  // over consecutive K ranges, whose fp32 partial tiles (256 x 256, row-major)
  // go to part and are added by the fixup kernel. n_full = n_items, ksplit = 1
  // when nothing is split.
  uint32_t n_full, n_split;
  int32_t ksplit;
  float* part;
  int32_t big;          // some operand spans 4 GiB or more (direct-load kernel rebases per stage)
  // Direct norm, direct-load kernel: examples per work item (a tile over eg
  // consecutive examples; items of one layer are group-major). 1 elsewhere.
  int32_t eg;
  // Per-example gradient store: the direct norm (direct-load kernel) also
  // writes each example's fp32 tile there; store_sum_kernel reads it back.
  // Tile slot q of example e is the 65536 floats at ((q * B + e) << 16), in
  // the register order of the 8 waves (GRAD_STORE layout below).
  float* store;
};

static_assert(sizeof(GemmArgs) <= 4096, "kernel arguments must stay within 4 KiB");

// The bf16 direct-load clipped-sum kernel's conditions (16-byte rows, whole
// 32-row stages per example, the factor table in LDS).
constexpr int DL_SUM_BK = 32;
constexpr int DL_SUM_MAXB = 4096;
inline bool dl_sum_applies(int dt, bool vec, int T, int B) {
  return dt == DT_BF16 && vec && T % DL_SUM_BK == 0 && B <= DL_SUM_MAXB;
}

// The last round of a launch of n_tiles equal tiles on `cus` CUs holds
// r = n_tiles mod cus of them (all of them if n_tiles < cus). When r is at most
// half the CUs, each of those tiles is split into ks consecutive K ranges of at
// least 4 stages (ks <= 8, r * ks <= cus), so the round takes about 1/ks of a
// tile's time.
struct TailSplit {
  uint32_t n_full, n_split;
  int32_t ks;
};
inline TailSplit tail_split(uint64_t n_tiles, int k_stages, int cus) {
  TailSplit t{(uint32_t)n_tiles, 0u, 1};
  if (cus <= 0 || n_tiles == 0) return t;
  const uint64_t r = n_tiles % (uint64_t)cus;
  if (r == 0 || 2 * r > (uint64_t)cus) return t;
  int ks = (int)((uint64_t)cus / r);
  ks = ks < 8 ? ks : 8;
  ks = ks < k_stages / 4 ? ks : k_stages / 4;
  if (ks < 2) return t;
  t.n_full = (uint32_t)(n_tiles - r);
  t.n_split = (uint32_t)r;
  t.ks = ks;
  return t;
}
constexpr size_t SPLIT_TILE_BYTES = (size_t)GM_BM * GM_BN * 4;  // one fp32 partial tile

// Direct norm on the direct-load kernel: the number of consecutive examples
// one work item covers. An item streams its examples' K stages without a gap
// and pays the ring's fill and drain once (about NG_OVERHEAD stages), so
// longer items cost less per stage, while fewer, longer items leave more of
// the chip idle in the last round. The choice minimises
// rounds(items) * (eg * stages per example + NG_OVERHEAD) over 1 <= eg <= B
// (eg <= NG_MAX: the item keeps a partial per example and wave in LDS).
constexpr int NG_OVERHEAD = 6;
constexpr int NG_MAX = 512;
inline int norm_group(uint64_t n_tiles, int B, int spe, int cus) {
  if (n_tiles == 0 || B <= 1 || cus <= 0) return 1;
  int best = 1;
  uint64_t best_cost = ~0ull;
  const int top = B < NG_MAX ? B : NG_MAX;
  for (int eg = 1; eg <= top; ++eg) {
    const uint64_t items = n_tiles * (uint64_t)((B + eg - 1) / eg);
    const uint64_t rounds = (items + (uint64_t)cus - 1) / (uint64_t)cus;
    const uint64_t cost = rounds * (uint64_t)(eg * spe + NG_OVERHEAD);
    if (cost < best_cost) { best_cost = cost; best = eg; }
  }
  return best;
}

// Clipped sum: out (+)= sum_i c_i X_i^T Y_i over all B*T rows (K = B*T).
// With a.part set (and room for the split that tail_split gives on `cus` CUs),
// the direct-load kernel splits its last round and a fixup kernel follows.
hipError_t launch_clipped_sum(const GemmArgs& a, int dt, bool vec, int cus, size_t part_bytes,
                              hipStream_t s);
// Direct norm: ws[b, slot] = ||tile of X_b^T Y_b||_F^2 for every output tile.
hipError_t launch_direct_norm(const GemmArgs& a, int dt, bool vec, hipStream_t s);
// Clipped sum from a gradient store: for every tile of every layer,
// out (+)= sum_e c_e * tile_e (then the fused noise and 1/B), one workgroup
// per tile; the layers' store_slot give each layer's first tile slot.
hipError_t launch_store_sum(const GemmArgs& a, hipStream_t s);
constexpr size_t STORE_TILE_FLOATS = (size_t)GM_BM * GM_BN;

// --------------------------------------------------------- embedding / ids
struct EmbedNormArgs {
  const int32_t* ids;   // [B,T]
  const void* E;        // dE [B*T, lde]
  int64_t lde;
  int32_t B, T, V, d;
  int32_t pbits;        // bits for a position in a sort key
  int32_t n_chunks;     // partials per example: feature chunks of 64, or (runs) position ranges
  int32_t runs;         // 1: embed_norm_runs_kernel (rows read EN_VB bytes per lane)
  int32_t gram;         // embed_norm_gram_kernel (bf16, 16-byte rows, T <= EN_G_T): n_chunks
                        // feature chunks; 2 (set at launch): workgroup row 0 ranks the ids
  int32_t* seg_id;      // nullable [B,T]
  int32_t* n_unique;    // nullable [B]
  float* ws;            // [B, n_chunks]
  // T > EN_MAX_T (runs only): each example sorted and ranked by the
  // workspace radix sort (keys [B*T] and their second buffer, digit counts
  // [B, 256, blocks per example], block run counts [B * blocks], run index of
  // every sorted position [B*T], run starts [B, T+1], run counts [B]).
  uint32_t *gkeys, *gkeys2;
  int32_t *ghist, *gruns, *grank, *gseg, *gnseg;
};
hipError_t launch_embed_norm(const EmbedNormArgs& a, int dt, hipStream_t s);

constexpr int EN_MAX_T = 4096;   // tokens per example sorted in LDS (bucketing)
constexpr int EN_CT_T = 256;     // up to this T the norm ranks keys by counting (one per thread)
constexpr int EN_P = 32;         // sorted positions whose runs one workgroup of the norm owns
constexpr int EN_VB = 8;         // bytes per lane load of the run-walking norm
constexpr int EN_BATCH = 32;     // row loads a lane has in flight (EN_P: one batch per range)
constexpr int EN_G_T = 128;      // up to this T (bf16) the norm takes the pairwise (Gram) form
constexpr int EN_GF = 96;        // features per workgroup of the pairwise form
constexpr int ES_MAX_K = 16384;  // tokens per batch sorted in LDS (embedding sum)
constexpr int ES_BLOCK = 32;     // sorted tokens per reduction block
constexpr int GS_KB = 4096;      // keys per block of the workspace radix sort (more than ES_MAX_K keys)

struct EmbedSumArgs {
  const int32_t* ids;   // [K] flattened B*T
  const void* E;        // [K, lde]
  int64_t lde;
  const float* c;       // [B]
  int32_t B, K, T, V, d;
  int32_t pbits;        // bits for a token index in a sort key
  uint32_t* keys;       // workspace [K] sorted keys
  float* head;          // workspace [n_blocks, d] partial of the run a block starts inside
  float* tail;          // workspace [n_blocks, d] partial of the run a block ends inside
  float* out;           // [V, ldo] or transposed [d, ldo]; accumulated into
  int64_t ldo;
  int32_t transpose;
  // Compact form: each run of equal ids gets one row of `rows` (its index is
  // the run's rank among the batch's runs), written once, instead of being
  // added onto out[id]; a later scatter adds the rows onto out.
  int32_t* rank;        // workspace [K] run index of every sorted position
  int32_t* seg;         // workspace [K + 1] first sorted position of every run
  int32_t* n_runs;      // workspace [1] number of runs
  float* rows;          // workspace [K, d] run sums
  // More than ES_MAX_K keys: the workspace radix sort in segments of gs_seg
  // keys (here one: the batch), gs_nbs blocks of GS_KB keys each, gs_blocks
  // in all (keys2: the other key buffer; hist: [segments, 256, gs_nbs]
  // digit counts, then offsets; gs_runs: [gs_blocks] run counts, then bases).
  int32_t gs_blocks, gs_nbs, gs_seg;
  uint32_t* keys2;
  int32_t* hist;
  int32_t* gs_runs;
};
hipError_t launch_embed_sum(const EmbedSumArgs& a, int dt, hipStream_t s);
// The compact form: sort, ranks, run sums into a.rows.
hipError_t launch_embed_rows(const EmbedSumArgs& a, int dt, hipStream_t s);
// out[id of run r] (+)= rows[r] for every run (reads a.keys, a.seg, a.n_runs).
hipError_t launch_embed_scatter(const EmbedSumArgs& a, hipStream_t s);
hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t s);

// ------------------------------------- vector parameters and position table
enum { VEC_GRAD = 0, VEC_SQ = 1 };
constexpr int VR_MAX_PARAMS = 44;   // entries per reduce launch (kernel arguments < 4 KiB)
constexpr int VS_MAX_PARAMS = 64;   // entries per clipped-sum launch
static_assert(GR_MAX_LAYERS <= 64 && GM_MAX_LAYERS <= 64 && VR_MAX_PARAMS <= 64,
              "a wave finds a work item's table entry with one lane per entry");

struct VecParam {
  const void* X;        // [B*T rows, ldx] elementwise factor, or null (a plain sum)
  const void* G;        // [B*T rows, ldg]
  int64_t ldx, ldg;
  int32_t d;            // features
  int32_t mode;         // VEC_GRAD: per-example gradient; VEC_SQ: sum of squares only
  float* grad;          // VEC_GRAD: [B, d] per-example gradients (of X * G, or of G)
  float* grad2;         // VEC_GRAD with X: [B, d] sums of G as well (a LayerNorm bias), or null
  int32_t tsplit;       // row ranges per feature chunk (VEC_SQ; 1 for VEC_GRAD)
  int32_t trows;        // rows per range
  uint32_t item_begin;  // first item of this entry among an example's items
  int32_t slot_begin;   // first partial slot of this entry in an example's row
};

// Items example-major: example b owns [b * per_ex, (b + 1) * per_ex), one per
// (entry, feature chunk of 64 lanes x 16 bytes, row range).
struct VecArgs {
  VecParam P[VR_MAX_PARAMS];
  int32_t n_params;
  int32_t B, T;
  int32_t slots;        // partial slots per example
  uint32_t per_ex;
  uint32_t n_items;
  float* ws;            // [B, slots]
};
static_assert(sizeof(VecArgs) <= 4096, "kernel arguments must stay within 4 KiB");
hipError_t launch_vec_reduce(const VecArgs& a, int dt, bool vec, hipStream_t s);

struct VecSumParam {
  const float* grad;    // [B, d]
  float* out;           // [d]
  int64_t d;
  uint32_t quad_begin;  // first 4-feature group of this entry
  uint32_t tensor_id;
  int32_t accumulate;
};
struct VecSumArgs {
  VecSumParam P[VS_MAX_PARAMS];
  int32_t n_params, B;
  uint32_t n_quads;
  const float* c;       // [B]
  int32_t noise;
  float sigma_c, inv_b;
  uint32_t step;
  uint64_t seed;
};
static_assert(sizeof(VecSumArgs) <= 4096, "kernel arguments must stay within 4 KiB");
hipError_t launch_vec_sum(const VecSumArgs& a, hipStream_t s);

struct PosSumArgs {
  const void* E;        // dE [B*T, lde]
  int64_t lde;
  const float* c;       // [B]
  float* out;           // [n_pos, ldo]
  int64_t ldo;
  int32_t B, T, d, n_pos;
  int32_t accumulate, noise;
  float sigma_c, inv_b;
  uint32_t tensor_id, step;
  uint64_t seed;
};
hipError_t launch_pos_sum(const PosSumArgs& a, int dt, hipStream_t s);

// ----------------------------------------------------------- clip and noise
// c (nullable) = clip factors; cs (nullable) = scale * clip factors; the
// squared norm is norm2 (+ norm2_b when not null).
hipError_t launch_clip_factors(const float* norm2, const float* norm2_b, int B, float C,
                               float scale, float* c, float* cs, hipStream_t s);
// accumulate: g = (g + sigma_c z) inv_b; else g = sigma_c z inv_b (g not read).
hipError_t launch_add_noise(float* g, int64_t n, float sigma_c, float inv_b, uint64_t seed,
                            uint32_t tensor_id, uint32_t step, bool accumulate, hipStream_t s);

}  // namespace dpg
