// C ABI of libdpghost: argument validation, launch planning and dispatch.
// Every argument is checked on the host before any HIP call.
#include "../../include/dpghost.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>
#include <vector>

#include "kernels.hpp"

// Device scratch of dp_ghost_norm_linear_bias_grouped_noalloc (for callers
// that cannot allocate): every device the library runs on holds its own copy
// from the library's load until the process ends. In host code `scratch`
// names a host-side stand-in, never the device memory: host code uses only
// the per-device address hipGetSymbolAddress returns (static_scratch below).
static __device__ __align__(256) unsigned char scratch[DP_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local std::string g_last_error;

dp_status_t fail(dp_status_t s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

dp_status_t hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return DP_OK;
  return fail(DP_EHIP, "%s: %s", what, hipGetErrorString(e));
}

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }
inline bool dtype_ok(dp_dtype_t dt) { return dt == DP_F32 || dt == DP_BF16; }
inline int elems_per_chunk(dp_dtype_t dt) { return dt == DP_BF16 ? 8 : 4; }
inline int stage_features(dp_dtype_t dt) { return dt == DP_BF16 ? 64 : 32; }
inline int kdt(dp_dtype_t dt) { return dt == DP_BF16 ? dpg::DT_BF16 : dpg::DT_F32; }
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline bool vec_ok(const void* p, int64_t ld, dp_dtype_t dt) {
  return aligned16(p) && ld % elems_per_chunk(dt) == 0;
}
inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int bits_for(int64_t n_values) {  // bits to index n_values distinct values
  int b = 0;
  while (b < 63 && (int64_t(1) << b) < n_values) ++b;
  return b;
}
inline size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }
inline int esize(dp_dtype_t dt) { return dt == DP_BF16 ? 2 : 4; }
// Kernels address operands through buffer resources with 32-bit byte offsets.
inline bool span_ok(int64_t rows, int64_t ld, dp_dtype_t dt) {
  return rows * ld * esize(dt) < (int64_t(1) << 32);
}

// ------------------------------------------------------------------ planning
constexpr int KG_SPLIT = 4096;  // G feature ranges longer than this are chunked
constexpr int KG_MIN = 1024;    // narrowest chunk considered

// Compute units of the current device (256 on MI355X), read once per device.
int device_cus() {
  static thread_local int cached_dev = -1, cached_cus = 256;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return cached_cus;
  if (dev != cached_dev) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        cus > 0)
      cached_cus = cus;
    cached_dev = dev;
  }
  return cached_cus;
}

struct GramEntry {
  const void* A;
  const void* G;
  int64_t lda, ldg;
  int d_in, g0, g1, kg, nc;
  int slot_begin;
  bool vec;
  float* bias = nullptr;  // fused bias gradient [B, g1], or null
};

struct GemmEntry {
  const void* X;
  const void* Y;
  int64_t ldx, ldy;
  int M, N, tm, tn;
  int slot_begin;
  float* out;
  int64_t ldo;
  bool vec;
  int acc = 0;             // clipped sum: out += (else out =)
  uint32_t tensor_id = 0;  // clipped sum with noise: generator id of the tensor
};

// The Gaussian mechanism fused into a clipped-sum launch.
struct NoiseCfg {
  bool on = false;
  float sigma_c = 0.f, inv_b = 1.f;
  uint32_t step = 0;
  uint64_t seed = 0;
};

// A layer bias whose gradient the layer's norm launch cannot fuse: reduced
// by the vector kernel instead.
struct BiasEntry {
  const void* G;
  int64_t ldg;
  int d;
  float* grad;
};

struct NormPlan {
  std::vector<GramEntry> gram;
  std::vector<GemmEntry> direct;
  std::vector<BiasEntry> bias_vec;
  int n_t = 0, P = 0;
  int64_t slots = 0;
};

// Gram flops T(T+1)(d_in+d_out) against direct flops 2 T d_in d_out, the
// Gram's weighted by the measured ratio of the two kernels' throughputs near
// the crossover (T = 384 .. 768): ~0.49 for layers whose G is read whole,
// ~0.38 for those whose G is split into feature chunks (an output head).
constexpr double GRAM_VS_DIRECT_THROUGHPUT = 0.49;
constexpr double CHUNKED_GRAM_VS_DIRECT_THROUGHPUT = 0.38;
bool use_direct(const dp_linear_t& L, int T) {
  if (L.algo == DP_NORM_DIRECT) return true;
  if (L.algo == DP_NORM_GRAM) return false;
  const double crossover = 2.0 * (double)L.d_in * L.d_out / ((double)L.d_in + L.d_out);
  const double r = L.d_out > KG_SPLIT ? CHUNKED_GRAM_VS_DIRECT_THROUGHPUT : GRAM_VS_DIRECT_THROUGHPUT;
  return (double)T + 1.0 > r * crossover;
}

// One GEMM entry over the output region [0,M) x [0,N); 16-byte loads when
// both operands have aligned rows whose stride is a whole number of chunks.
void plan_gemm(const void* X, int64_t ldx, int M, const void* Y, int64_t ldy, int N,
               dp_dtype_t dt, float* out, int64_t ldo, std::vector<GemmEntry>& v,
               int64_t* slots, int64_t slot_mult) {
  GemmEntry e{X, Y, ldx, ldy, M, N, (int)ceil_div(M, dpg::GM_BM), (int)ceil_div(N, dpg::GM_BN),
              0, out, ldo, vec_ok(X, ldx, dt) && vec_ok(Y, ldy, dt)};
  if (slots) {
    e.slot_begin = (int)*slots;
    *slots += (int64_t)e.tm * e.tn * slot_mult;
  }
  v.push_back(e);
}

// Work items per (example, G chunk): one per T-tile pair, or one in all when
// the whole-example Gram applies.
int gram_pairs(const NormPlan& p, dp_dtype_t dt, bool vec, int T) {
  return dpg::gram_whole(kdt(dt), vec, T) ? 1 : p.P;
}

// A clipped-sum entry whose kernel rows are the output's rows: X is the
// operand indexing the output's rows (A for [d_in, d_out], G for the
// transposed [d_out, d_in]), so the kernel always stores row-major and the
// caller's layout only decides the operand order.
void plan_sum(const dp_linear_t& L, int transpose_out, dp_dtype_t dt, float* out,
              std::vector<GemmEntry>& v) {
  if (transpose_out)
    plan_gemm(L.G, L.ldg, L.d_out, L.A, L.lda, L.d_in, dt, out, L.d_in, v, nullptr, 0);
  else
    plan_gemm(L.A, L.lda, L.d_in, L.G, L.ldg, L.d_out, dt, out, L.d_out, v, nullptr, 0);
}

// Chunk count of a G range longer than KG_SPLIT features. Chunks are at most
// KG_SPLIT and at least KG_MIN features wide (whole stages); among those
// counts, the one whose launch (this layer's items plus `other` items of the
// same kernel) fills the last round of `slots` concurrent workgroups best,
// the fewest chunks on a tie (each chunk re-reads A).
int pick_chunks(int64_t width, int ks, int64_t items_per_chunk, int64_t other, int64_t slots) {
  const int64_t nc_lo = ceil_div(width, KG_SPLIT);
  const int64_t nc_hi = std::max(nc_lo, ceil_div(width, KG_MIN));
  int64_t best = nc_lo;
  double best_idle = 2.0;
  for (int64_t nc = nc_lo; nc <= nc_hi; ++nc) {
    const int64_t kg = ceil_div(ceil_div(width, nc), ks) * ks;
    const int64_t eff = ceil_div(width, kg);
    const int64_t total = other + items_per_chunk * eff;
    const double idle = (double)(ceil_div(total, slots) * slots - total) / (double)total;
    if (idle < best_idle - 1e-9) { best_idle = idle; best = eff; }
  }
  return (int)best;
}

NormPlan plan_norm(const dp_linear_t* layers, int n, int B, int T, dp_dtype_t dt,
                   float* const* bias = nullptr) {
  NormPlan p;
  p.n_t = (int)ceil_div(T, dpg::GR_TM);
  p.P = p.n_t * (p.n_t + 1) / 2;
  const int ks = stage_features(dt);
  // Items of the unchunked Gram layers, per kernel (16-byte rows or not).
  int64_t plain_items[2] = {0, 0};
  for (int i = 0; i < n; ++i) {
    const dp_linear_t& L = layers[i];
    if (use_direct(L, T) || L.d_out > KG_SPLIT) continue;
    const bool vec = vec_ok(L.A, L.lda, dt) && vec_ok(L.G, L.ldg, dt);
    plain_items[vec] += (int64_t)B * gram_pairs(p, dt, vec, T);
  }
  for (int i = 0; i < n; ++i) {
    const dp_linear_t& L = layers[i];
    float* const bg = bias ? bias[i] : nullptr;
    if (use_direct(L, T)) {
      plan_gemm(L.A, L.lda, L.d_in, L.G, L.ldg, L.d_out, dt, nullptr, 0, p.direct, &p.slots, 1);
      if (bg) p.bias_vec.push_back({L.G, L.ldg, L.d_out, bg});
      continue;
    }
    const bool vec = vec_ok(L.A, L.lda, dt) && vec_ok(L.G, L.ldg, dt);
    int kg = (int)(ceil_div(L.d_out, ks) * ks);
    if (L.d_out > KG_SPLIT) {
      const int64_t per_chunk = (int64_t)B * gram_pairs(p, dt, vec, T);
      const int64_t slots = (int64_t)device_cus() * dpg::gram_groups_per_cu(kdt(dt), vec, T);
      const int nc = pick_chunks(L.d_out, ks, per_chunk, plain_items[vec], slots);
      kg = (int)(ceil_div(ceil_div(L.d_out, nc), ks) * ks);
      plain_items[vec] += per_chunk * ceil_div(L.d_out, kg);
    }
    GramEntry e{L.A, L.G, L.lda, L.ldg, L.d_in, 0, L.d_out, kg, (int)ceil_div(L.d_out, kg),
                (int)p.slots, vec};
    if (bg) {
      if (dpg::gram_fuses_bias(kdt(dt), vec, T))
        e.bias = bg;
      else
        p.bias_vec.push_back({L.G, L.ldg, L.d_out, bg});
    }
    p.slots += (int64_t)gram_pairs(p, dt, e.vec, T) * e.nc;
    p.gram.push_back(e);
  }
  return p;
}

dp_status_t check_layers(const dp_linear_t* layers, int n, int B, int T, dp_dtype_t dt) {
  if (!layers) return fail(DP_EINVAL, "layers is NULL");
  if (n <= 0) return fail(DP_EINVAL, "n_layers must be positive (got %d)", n);
  if (B <= 0 || T <= 0) return fail(DP_EINVAL, "B and T must be positive (got %d, %d)", B, T);
  if (!dtype_ok(dt)) return fail(DP_EINVAL, "unknown dtype %d", (int)dt);
  if (T > 65536) return fail(DP_EUNSUPPORTED, "T = %d exceeds 65536", T);
  for (int i = 0; i < n; ++i) {
    const dp_linear_t& L = layers[i];
    if (!L.A || !L.G) return fail(DP_EINVAL, "layer %d: A or G is NULL", i);
    if (L.d_in <= 0 || L.d_out <= 0)
      return fail(DP_EINVAL, "layer %d: d_in and d_out must be positive", i);
    if (L.lda < L.d_in || L.ldg < L.d_out)
      return fail(DP_EINVAL, "layer %d: row stride smaller than row width", i);
    if (L.algo < DP_NORM_AUTO || L.algo > DP_NORM_DIRECT)
      return fail(DP_EINVAL, "layer %d: unknown algo %d", i, L.algo);
    // Offsets within one example are 32-bit everywhere. Offsets across the
    // batch are 32-bit too except in the direct-load GEMM (bf16, 16-byte rows,
    // whole 32-row stages), which moves its descriptors' base per stage: only
    // layers that take it may span 4 GiB or more.
    if (!span_ok(T, L.lda, dt) || !span_ok(T, L.ldg, dt))
      return fail(DP_EUNSUPPORTED, "layer %d: one example's rows span 4 GiB or more", i);
    const bool dl = dpg::dl_sum_applies(kdt(dt), vec_ok(L.A, L.lda, dt) && vec_ok(L.G, L.ldg, dt),
                                        T, B);
    if (!dl && (!span_ok((int64_t)B * T, L.lda, dt) || !span_ok((int64_t)B * T, L.ldg, dt)))
      return fail(DP_EUNSUPPORTED,
                  "layer %d: an operand spans 4 GiB or more (allowed only for bf16 16-byte rows "
                  "with T a multiple of 32 and B <= 4096)", i);
    if (ceil_div(L.d_in, dpg::GM_BM) > 65535 || ceil_div(L.d_out, dpg::GM_BN) > 65535)
      return fail(DP_EUNSUPPORTED, "layer %d: a width exceeds 65535 tiles of 256", i);
  }
  return DP_OK;
}

// ------------------------------------------------------------------ launches
dp_status_t run_gram(const NormPlan& p, int B, int T, dp_dtype_t dt, float* ws, hipStream_t s) {
  for (int pass = 0; pass < 2; ++pass) {
    const bool vec = pass == 0;
    std::vector<const GramEntry*> sel;
    for (const auto& e : p.gram)
      if (e.vec == vec) sel.push_back(&e);
    // Within an example, the layers with the longest items go first, so that
    // the last items each XCD runs are short ones (a shorter tail).
    std::stable_sort(sel.begin(), sel.end(), [](const GramEntry* x, const GramEntry* y) {
      return x->d_in + x->kg > y->d_in + y->kg;
    });
    for (size_t i0 = 0; i0 < sel.size(); i0 += dpg::GR_MAX_LAYERS) {
      dpg::GramArgs a{};
      a.B = B; a.T = T; a.n_t = p.n_t; a.P = gram_pairs(p, dt, vec, T);
      a.slots = (int32_t)p.slots;
      a.ws = ws;
      uint64_t per_ex = 0;
      const size_t n = std::min(sel.size() - i0, (size_t)dpg::GR_MAX_LAYERS);
      for (size_t j = 0; j < n; ++j) {
        const GramEntry& e = *sel[i0 + j];
        dpg::GramLayer& L = a.L[j];
        L.A = e.A; L.G = e.G; L.lda = e.lda; L.ldg = e.ldg;
        L.d_in = e.d_in; L.g0 = e.g0; L.g1 = e.g1; L.kg = e.kg; L.nc = e.nc;
        L.item_begin = (uint32_t)per_ex;
        L.slot_begin = e.slot_begin;
        L.bias = e.bias;
        per_ex += (uint64_t)a.P * e.nc;
      }
      const uint64_t items = per_ex * (uint64_t)B;
      if (items > 0xFFFFFFFFull) return fail(DP_EUNSUPPORTED, "too many work items (%llu)",
                                             (unsigned long long)items);
      a.n_layers = (int32_t)n;
      a.per_ex = (uint32_t)per_ex;
      a.n_items = (uint32_t)items;
      dp_status_t st = hip_status(dpg::launch_gram_norm(a, kdt(dt), vec, s), "gram_norm launch");
      if (st != DP_OK) return st;
    }
  }
  return DP_OK;
}

// The launches of a GEMM plan: entries with 16-byte rows first, then the
// others, at most GM_MAX_LAYERS per launch.
std::vector<std::pair<bool, std::vector<const GemmEntry*>>> gemm_launches(
    const std::vector<GemmEntry>& entries) {
  std::vector<std::pair<bool, std::vector<const GemmEntry*>>> out;
  for (int pass = 0; pass < 2; ++pass) {
    const bool vec = pass == 0;
    std::vector<const GemmEntry*> sel;
    for (const auto& e : entries)
      if (e.vec == vec) sel.push_back(&e);
    for (size_t i0 = 0; i0 < sel.size(); i0 += dpg::GM_MAX_LAYERS) {
      const size_t n = std::min(sel.size() - i0, (size_t)dpg::GM_MAX_LAYERS);
      out.emplace_back(vec, std::vector<const GemmEntry*>(sel.begin() + i0, sel.begin() + i0 + n));
    }
  }
  return out;
}

// Bytes of partial tiles the split tail of a clipped-sum plan needs (the
// largest over its launches, which run one after another).
size_t sum_split_bytes(const std::vector<GemmEntry>& entries, int B, int T, dp_dtype_t dt) {
  size_t need = 0;
  for (const auto& [vec, sel] : gemm_launches(entries)) {
    if (!dpg::dl_sum_applies(kdt(dt), vec, T, B)) continue;
    uint64_t tiles = 0;
    for (const GemmEntry* e : sel) tiles += (uint64_t)e->tm * e->tn;
    const dpg::TailSplit t = dpg::tail_split(tiles, (int)((int64_t)B * T / dpg::DL_SUM_BK),
                                             device_cus());
    need = std::max(need, (size_t)t.n_split * t.ks * dpg::SPLIT_TILE_BYTES);
  }
  return need;
}

// mode 0: clipped sum (c, out); mode 1: direct norm (ws, slots). A clipped sum
// given `part` (part_bytes) splits the tail of its direct-load launches.
dp_status_t run_gemm(const std::vector<GemmEntry>& entries, int mode, int B, int T, dp_dtype_t dt,
                     const float* c, float* ws, int64_t slots, int transpose, const NoiseCfg& nz,
                     hipStream_t s, float* part = nullptr, size_t part_bytes = 0,
                     float* store = nullptr) {
  for (const auto& [vec, sel] : gemm_launches(entries)) {
    dpg::GemmArgs a{};
    a.B = B; a.T = T; a.c = c; a.ws = ws; a.slots = (int32_t)slots;
    a.transpose = transpose;
    a.store = store;
    a.noise = nz.on ? 1 : 0;
    a.sigma_c = nz.sigma_c; a.inv_b = nz.inv_b; a.step = nz.step; a.seed = nz.seed;
    a.part = part;
    a.eg = 1;
    if (mode == 1 && kdt(dt) == dpg::DT_BF16 && vec && T % dpg::DL_SUM_BK == 0) {
      uint64_t tiles = 0;
      for (const GemmEntry* e : sel) tiles += (uint64_t)e->tm * e->tn;
      a.eg = dpg::norm_group(tiles, B, T / dpg::DL_SUM_BK, device_cus());
    }
    const uint64_t groups = (uint64_t)((B + a.eg - 1) / a.eg);
    uint64_t items = 0;
    for (size_t j = 0; j < sel.size(); ++j) {
      const GemmEntry& e = *sel[j];
      dpg::GemmLayer& L = a.L[j];
      L.X = e.X; L.Y = e.Y; L.ldx = e.ldx; L.ldy = e.ldy;
      L.M = e.M; L.N = e.N;
      L.tm = (uint16_t)e.tm; L.tn = (uint16_t)e.tn;
      if (!span_ok((int64_t)B * T, e.ldx, dt) || !span_ok((int64_t)B * T, e.ldy, dt)) a.big = 1;
      L.tile_begin = (uint32_t)items;
      if (mode == 0) L.tensor_id = e.tensor_id;
      else L.slot_begin = e.slot_begin;
      L.accumulate = e.acc;
      L.out = e.out; L.ldo = e.ldo;
      items += (uint64_t)e.tm * e.tn * (mode == 1 ? groups : 1ull);
    }
    if (items > 0xFFFFFFFFull) return fail(DP_EUNSUPPORTED, "too many work items");
    a.n_layers = (int32_t)sel.size();
    a.n_items = (uint32_t)items;
    hipError_t e = mode == 0 ? dpg::launch_clipped_sum(a, kdt(dt), vec, device_cus(), part_bytes, s)
                             : dpg::launch_direct_norm(a, kdt(dt), vec, s);
    dp_status_t st = hip_status(e, mode == 0 ? "clipped_sum launch" : "direct_norm launch");
    if (st != DP_OK) return st;
  }
  return DP_OK;
}

size_t norm_ws_bytes(const NormPlan& p, int B) { return align_up((size_t)B * p.slots * 4); }

// The device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

dp_status_t static_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(DP_EUNSUPPORTED, "device %d: the static scratch serves devices 0..%d", dev,
                kMaxDevices - 1);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(DP_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return DP_OK;
}

// Embedding-sum workspace layout (bytes): sorted keys, block head/tail partials.
struct EsLayout {
  size_t keys, head, tail, rank, seg, n_runs, rows, keys2, hist, gs_runs, total;
};
// compact: also the ranks, run starts, run count and [K, d] run rows. More
// than ES_MAX_K keys: also the second key buffer, the digit counts and the
// block run counts of the workspace radix sort.
EsLayout es_layout(int64_t K, int d, bool compact = false) {
  EsLayout l{};
  const int64_t nb = ceil_div(K, dpg::ES_BLOCK);
  size_t off = 0;
  l.keys = off; off = align_up(off + (size_t)K * 4);
  l.head = off; off = align_up(off + (size_t)nb * d * 4);
  l.tail = off; off = align_up(off + (size_t)nb * d * 4);
  if (compact) {
    l.rank = off; off = align_up(off + (size_t)K * 4);
    l.seg = off; off = align_up(off + (size_t)(K + 1) * 4);
    l.n_runs = off; off = align_up(off + 4);
    l.rows = off; off = align_up(off + (size_t)K * d * 4);
  }
  if (K > dpg::ES_MAX_K) {
    const int64_t gb = ceil_div(K, dpg::GS_KB);
    l.keys2 = off; off = align_up(off + (size_t)K * 4);
    l.hist = off; off = align_up(off + (size_t)gb * 256 * 4);
    l.gs_runs = off; off = align_up(off + (size_t)gb * 4);
  }
  l.total = off;
  return l;
}


// ------------------------------------------------- vector parameters, positions
struct VecEntry {
  const void* X;
  const void* G;
  int64_t ldx, ldg;
  int d, mode, chunks, slot_begin;
  float* grad;
  bool vec;
  float* grad2 = nullptr;  // fused LayerNorm bias (same G, no X)
  int tsplit = 1, trows = 0;
};

struct VecPlan {
  std::vector<VecEntry> e;
  int64_t slots = 0;
};

int vec_chunk_features(dp_dtype_t dt) { return 64 * elems_per_chunk(dt); }

// Rows per item of a sum-of-squares entry (its partials are scalars, so an
// example's rows may be split into ranges for more parallel work).
constexpr int VEC_SQ_ROWS = 32;

void plan_vec(VecPlan& p, const void* X, int64_t ldx, const void* G, int64_t ldg, int d, int mode,
              float* grad, dp_dtype_t dt, int T, float* grad2 = nullptr) {
  VecEntry e{X, G, ldx, ldg, d, mode, (int)ceil_div(d, vec_chunk_features(dt)), (int)p.slots,
             grad, vec_ok(G, ldg, dt) && (!X || vec_ok(X, ldx, dt))};
  e.grad2 = grad2;
  e.tsplit = mode == dpg::VEC_SQ ? (int)ceil_div(T, VEC_SQ_ROWS) : 1;
  e.trows = mode == dpg::VEC_SQ ? VEC_SQ_ROWS : T;
  p.slots += (int64_t)e.chunks * e.tsplit;
  p.e.push_back(e);
}

// The gradient entries of a grouped call. A LayerNorm's gain (X set) and bias
// (no X, the same G, stride and width) are one entry: one pass over G.
void plan_vec_grads(VecPlan& p, const dp_vector_t* params, int n, float* const* grads,
                    dp_dtype_t dt, int T) {
  std::vector<int> partner(n, -1);
  std::vector<char> claimed(n, 0);
  for (int i = 0; i < n; ++i) {
    const dp_vector_t& v = params[i];
    if (!v.X) continue;
    for (int j = 0; j < n; ++j) {
      const dp_vector_t& u = params[j];
      if (!u.X && !claimed[j] && u.G == v.G && u.ldg == v.ldg && u.d == v.d) {
        partner[i] = j;
        claimed[j] = 1;
        break;
      }
    }
  }
  for (int i = 0; i < n; ++i) {
    if (claimed[i]) continue;
    const dp_vector_t& v = params[i];
    float* g2 = partner[i] >= 0 && grads ? grads[partner[i]] : nullptr;
    float* g = grads ? grads[i] : nullptr;
    plan_vec(p, v.X, v.ldx, v.G, v.ldg, v.d, dpg::VEC_GRAD, g, dt, T, partner[i] >= 0 ? g2 : nullptr);
  }
}

dp_status_t check_vec(const dp_vector_t* params, int n, int B, int T, dp_dtype_t dt) {
  if (!params) return fail(DP_EINVAL, "params is NULL");
  if (n <= 0) return fail(DP_EINVAL, "n must be positive (got %d)", n);
  if (B <= 0 || T <= 0) return fail(DP_EINVAL, "B and T must be positive (got %d, %d)", B, T);
  if (!dtype_ok(dt)) return fail(DP_EINVAL, "unknown dtype %d", (int)dt);
  for (int i = 0; i < n; ++i) {
    const dp_vector_t& v = params[i];
    if (!v.G) return fail(DP_EINVAL, "param %d: G is NULL", i);
    if (v.d <= 0) return fail(DP_EINVAL, "param %d: d must be positive", i);
    if (v.ldg < v.d || (v.X && v.ldx < v.d))
      return fail(DP_EINVAL, "param %d: row stride smaller than d", i);
    if (!span_ok((int64_t)B * T, v.ldg, dt) || (v.X && !span_ok((int64_t)B * T, v.ldx, dt)))
      return fail(DP_EUNSUPPORTED, "param %d: an operand spans 4 GiB or more", i);
  }
  return DP_OK;
}

dp_status_t run_vec(const VecPlan& p, int B, int T, dp_dtype_t dt, float* ws, hipStream_t s) {
  for (int pass = 0; pass < 2; ++pass) {
    const bool vec = pass == 0;
    std::vector<const VecEntry*> sel;
    for (const auto& e : p.e)
      if (e.vec == vec) sel.push_back(&e);
    for (size_t i0 = 0; i0 < sel.size(); i0 += dpg::VR_MAX_PARAMS) {
      dpg::VecArgs a{};
      a.B = B; a.T = T; a.slots = (int32_t)p.slots; a.ws = ws;
      uint64_t per_ex = 0;
      const size_t n = std::min(sel.size() - i0, (size_t)dpg::VR_MAX_PARAMS);
      for (size_t j = 0; j < n; ++j) {
        const VecEntry& e = *sel[i0 + j];
        dpg::VecParam& P = a.P[j];
        P.X = e.X; P.G = e.G; P.ldx = e.ldx; P.ldg = e.ldg; P.d = e.d; P.mode = e.mode;
        P.grad = e.grad; P.grad2 = e.grad2; P.tsplit = e.tsplit; P.trows = e.trows;
        P.item_begin = (uint32_t)per_ex; P.slot_begin = e.slot_begin;
        per_ex += (uint64_t)e.chunks * e.tsplit;
      }
      const uint64_t items = per_ex * (uint64_t)B;
      if (items > 0xFFFFFFFFull) return fail(DP_EUNSUPPORTED, "too many work items");
      a.n_params = (int32_t)n;
      a.per_ex = (uint32_t)per_ex;
      a.n_items = (uint32_t)items;
      dp_status_t st = hip_status(dpg::launch_vec_reduce(a, kdt(dt), vec, s), "vec_reduce launch");
      if (st != DP_OK) return st;
    }
  }
  return DP_OK;
}

dp_status_t check_noise_args(float sigma, float C, int B_norm, uint64_t step) {
  if (!(sigma >= 0.f) || !std::isfinite(sigma)) return fail(DP_EINVAL, "sigma must be >= 0");
  if (!(C > 0.f) || !std::isfinite(C)) return fail(DP_EINVAL, "C must be positive and finite");
  if (B_norm < 0) return fail(DP_EINVAL, "B_norm must be >= 0");
  if (step >> 32) return fail(DP_EINVAL, "step must be < 2^32");
  return DP_OK;
}

}  // namespace

// ======================================================================
extern "C" {

int dp_abi_version(void) { return DP_ABI_VERSION; }

const char* dp_status_string(dp_status_t s) {
  switch (s) {
    case DP_OK: return "ok";
    case DP_EINVAL: return "invalid argument";
    case DP_EUNSUPPORTED: return "unsupported size";
    case DP_EHIP: return "HIP error";
  }
  return "unknown status";
}

const char* dp_last_error(void) { return g_last_error.c_str(); }

size_t dp_ghost_norm_linear_bias_workspace(const dp_linear_t* layers, float* const* bias_grads,
                                           int n_layers, int B, int T, dp_dtype_t dt) {
  if (check_layers(layers, n_layers, B, T, dt) != DP_OK) return 0;
  const NormPlan p = plan_norm(layers, n_layers, B, T, dt, bias_grads);
  VecPlan vp;
  for (const BiasEntry& e : p.bias_vec)
    plan_vec(vp, nullptr, 0, e.G, e.ldg, e.d, dpg::VEC_GRAD, e.grad, dt, T);
  return norm_ws_bytes(p, B) + align_up((size_t)B * vp.slots * 4);
}

size_t dp_ghost_norm_linear_workspace(const dp_linear_t* layers, int n_layers, int B, int T,
                                      dp_dtype_t dt) {
  return dp_ghost_norm_linear_bias_workspace(layers, nullptr, n_layers, B, T, dt);
}

}  // extern "C"

namespace {
// The grouped norm with biases. workspace == NULL with use_static: the
// partials go to this device's static scratch (nothing is allocated).
dp_status_t norm_bias_grouped(const dp_linear_t* layers, float* const* bias_grads, int n_layers,
                              int B, int T, dp_dtype_t dt, float* norm2, int accumulate,
                              void* workspace, size_t workspace_bytes, void* stream,
                              bool use_static) {
  dp_status_t st = check_layers(layers, n_layers, B, T, dt);
  if (st != DP_OK) return st;
  if (!norm2) return fail(DP_EINVAL, "norm2 is NULL");
  const NormPlan p = plan_norm(layers, n_layers, B, T, dt, bias_grads);
  if ((uint64_t)B * p.slots > 0x7FFFFFFFull) return fail(DP_EUNSUPPORTED, "too many partials");
  for (const BiasEntry& e : p.bias_vec)  // the vector kernel's offsets span the batch in 32 bits
    if (!span_ok((int64_t)B * T, e.ldg, dt))
      return fail(DP_EUNSUPPORTED, "a bias whose G spans 4 GiB or more must be fused into the "
                  "Gram launch (bf16, 16-byte rows, T <= 256)");
  VecPlan vp;
  for (const BiasEntry& e : p.bias_vec)
    plan_vec(vp, nullptr, 0, e.G, e.ldg, e.d, dpg::VEC_GRAD, e.grad, dt, T);
  const size_t norm_bytes = norm_ws_bytes(p, B);
  const size_t need = norm_bytes + align_up((size_t)B * vp.slots * 4);
  if (use_static) {
    if (need > (size_t)DP_NOALLOC_SCRATCH_BYTES)
      return fail(DP_EUNSUPPORTED,
                  "this call needs %zu bytes of scratch; the static scratch holds %zu "
                  "(use dp_ghost_norm_linear_bias_grouped with a workspace)",
                  need, (size_t)DP_NOALLOC_SCRATCH_BYTES);
    st = static_scratch(&workspace);
    if (st != DP_OK) return st;
    workspace_bytes = DP_NOALLOC_SCRATCH_BYTES;
  }
  if (!workspace || workspace_bytes < need)
    return fail(DP_EINVAL, "workspace of %zu bytes needed, %zu given", need,
                workspace ? workspace_bytes : (size_t)0);
  hipStream_t s = as_stream(stream);
  float* ws = static_cast<float*>(workspace);
  st = run_gram(p, B, T, dt, ws, s);
  if (st != DP_OK) return st;
  st = run_gemm(p.direct, 1, B, T, dt, nullptr, ws, p.slots, 0, NoiseCfg{}, s);
  if (st != DP_OK) return st;
  float* vws = reinterpret_cast<float*>(static_cast<char*>(workspace) + norm_bytes);
  if (!vp.e.empty()) {
    st = run_vec(vp, B, T, dt, vws, s);
    if (st != DP_OK) return st;
  }
  st = hip_status(dpg::launch_finish_rows(ws, B, (int)p.slots, norm2, accumulate, 1.f, s),
                  "finish launch");
  if (st != DP_OK || vp.e.empty()) return st;
  return hip_status(dpg::launch_finish_rows(vws, B, (int)vp.slots, norm2, 1, 1.f, s),
                    "finish launch");
}
}  // namespace

extern "C" {

dp_status_t dp_ghost_norm_linear_bias_grouped(const dp_linear_t* layers, float* const* bias_grads,
                                              int n_layers, int B, int T, dp_dtype_t dt,
                                              float* norm2, int accumulate, void* workspace,
                                              size_t workspace_bytes, void* stream) {
  return norm_bias_grouped(layers, bias_grads, n_layers, B, T, dt, norm2, accumulate, workspace,
                           workspace_bytes, stream, false);
}

dp_status_t dp_ghost_norm_linear_bias_grouped_noalloc(const dp_linear_t* layers,
                                                      float* const* bias_grads, int n_layers,
                                                      int B, int T, dp_dtype_t dt, float* norm2,
                                                      int accumulate, void* stream) {
  return norm_bias_grouped(layers, bias_grads, n_layers, B, T, dt, norm2, accumulate, nullptr, 0,
                           stream, true);
}

dp_status_t dp_ghost_norm_linear_grouped(const dp_linear_t* layers, int n_layers, int B, int T,
                                         dp_dtype_t dt, float* norm2, int accumulate,
                                         void* workspace, size_t workspace_bytes, void* stream) {
  return dp_ghost_norm_linear_bias_grouped(layers, nullptr, n_layers, B, T, dt, norm2, accumulate,
                                           workspace, workspace_bytes, stream);
}

dp_status_t dp_ghost_norm_linear(const void* A, int64_t lda, const void* G, int64_t ldg, int B,
                                 int T, int d_in, int d_out, dp_dtype_t dt, int algo,
                                 float* norm2, int accumulate, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  dp_linear_t L{A, lda, d_in, G, ldg, d_out, algo};
  return dp_ghost_norm_linear_grouped(&L, 1, B, T, dt, norm2, accumulate, workspace,
                                      workspace_bytes, stream);
}

// Partials per example: one per 64-feature chunk (embed_norm_kernel) or per
// EN_P sorted positions (embed_norm_runs_kernel); the size query cannot know
// which kernel a call takes, so it covers both.
// Past EN_MAX_T tokens an example is sorted through the workspace: keys and
// their second buffer, digit counts, block run counts, run indices, run
// starts and run counts follow the partials.
struct EnLayout {
  size_t gkeys, gkeys2, ghist, gruns, grank, gseg, gnseg, total;
};
EnLayout en_layout(int B, int T, int d) {
  EnLayout l{};
  size_t off = align_up((size_t)B * std::max(ceil_div(d, 64), ceil_div(T, dpg::EN_P)) * 4);
  if (T > dpg::EN_MAX_T) {
    const size_t K = (size_t)B * T, nbs = (size_t)ceil_div(T, dpg::GS_KB);
    l.gkeys = off; off = align_up(off + K * 4);
    l.gkeys2 = off; off = align_up(off + K * 4);
    l.ghist = off; off = align_up(off + (size_t)B * 256 * nbs * 4);
    l.gruns = off; off = align_up(off + (size_t)B * nbs * 4);
    l.grank = off; off = align_up(off + K * 4);
    l.gseg = off; off = align_up(off + (size_t)B * (T + 1) * 4);
    l.gnseg = off; off = align_up(off + (size_t)B * 4);
  }
  l.total = off;
  return l;
}

size_t dp_ghost_norm_embedding_workspace(int B, int T, int d) {
  if (B <= 0 || T <= 0 || d <= 0) return 0;
  return en_layout(B, T, d).total;
}

dp_status_t dp_ghost_norm_embedding(const int32_t* ids, const void* dE, int64_t lde, int B, int T,
                                    int V, int d, dp_dtype_t dt, float* norm2, int accumulate,
                                    int32_t* seg_id, int32_t* n_unique, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  if (!ids || !dE || !norm2) return fail(DP_EINVAL, "ids, dE or norm2 is NULL");
  if (B <= 0 || T <= 0 || V <= 0 || d <= 0)
    return fail(DP_EINVAL, "B, T, V and d must be positive");
  if (lde < d) return fail(DP_EINVAL, "lde (%lld) < d (%d)", (long long)lde, d);
  if (!dtype_ok(dt)) return fail(DP_EINVAL, "unknown dtype %d", (int)dt);
  if ((int64_t)B * T > INT32_MAX) return fail(DP_EUNSUPPORTED, "B*T exceeds 2^31 - 1");
  const int pbits = std::max(1, bits_for(T));
  if (bits_for((int64_t)V + 1) + pbits > 32)  // ids are clamped to V, so V + 1 values
    return fail(DP_EUNSUPPORTED, "V = %d and T = %d do not fit a 32-bit sort key", V, T);
  const size_t need = dp_ghost_norm_embedding_workspace(B, T, d);
  if (!workspace || workspace_bytes < need)
    return fail(DP_EINVAL, "workspace of %zu bytes needed", need);
  dpg::EmbedNormArgs a{};
  a.ids = ids; a.E = dE; a.lde = lde;
  a.B = B; a.T = T; a.V = V; a.d = d;
  a.pbits = pbits;
  // Rows read 8 bytes per lane when they allow it (and an example's rows
  // span less than 4 GiB, for the buffer offsets).
  const int64_t es = esize(dt);
  a.runs = ((uintptr_t)dE % dpg::EN_VB == 0 && (lde * es) % dpg::EN_VB == 0 &&
            (d * es) % dpg::EN_VB == 0 && span_ok(T, lde, dt)) ? 1 : 0;
  a.n_chunks = (int)(a.runs ? ceil_div(T, dpg::EN_P) : ceil_div(d, 64));
  // Short bf16 examples with 16-byte rows (and pieces of 8 features): the
  // pairwise form, one partial per chunk of EN_GF features (fewer than the
  // ceil(d / 64) the workspace holds).
  if (kdt(dt) == dpg::DT_BF16 && T <= dpg::EN_G_T && (uintptr_t)dE % 16 == 0 &&
      (lde * es) % 16 == 0 && d % 8 == 0 && (int64_t)T * lde * es < 0x80000000ll) {
    a.gram = 1;
    a.runs = 0;
    a.n_chunks = (int)ceil_div(d, dpg::EN_GF);
  }
  a.seg_id = seg_id; a.n_unique = n_unique;
  if (T > dpg::EN_MAX_T) {
    if (!a.runs)
      return fail(DP_EUNSUPPORTED, "T = %d exceeds %d for rows that are not whole 8-byte units "
                  "within a 4 GiB span", T, dpg::EN_MAX_T);
    const EnLayout l = en_layout(B, T, d);
    char* w = static_cast<char*>(workspace);
    a.gkeys = reinterpret_cast<uint32_t*>(w + l.gkeys);
    a.gkeys2 = reinterpret_cast<uint32_t*>(w + l.gkeys2);
    a.ghist = reinterpret_cast<int32_t*>(w + l.ghist);
    a.gruns = reinterpret_cast<int32_t*>(w + l.gruns);
    a.grank = reinterpret_cast<int32_t*>(w + l.grank);
    a.gseg = reinterpret_cast<int32_t*>(w + l.gseg);
    a.gnseg = reinterpret_cast<int32_t*>(w + l.gnseg);
  }
  a.ws = static_cast<float*>(workspace);
  hipStream_t s = as_stream(stream);
  dp_status_t st = hip_status(dpg::launch_embed_norm(a, kdt(dt), s), "embed_norm launch");
  if (st != DP_OK) return st;
  return hip_status(dpg::launch_finish_rows(a.ws, B, a.n_chunks, norm2, accumulate, 1.f, s),
                    "finish launch");
}

// Partials per example: (128-row tile pair, 128-feature chunk) for the
// register-staged kernel, (64-row block pair) for the direct-load one,
// (32-token block, 32-row block) for the register-direct one (T <= CX_ROWS_T
// only). The size query cannot know the dtype or alignment of a call, so it
// covers every kernel the call's T allows.
int64_t cross_blocks(int T, int kind) {
  return ceil_div(T, kind == dpg::CROSS_ROWS ? dpg::CR_RX_ROWS
                     : kind == dpg::CROSS_DL ? dpg::CR_DL_ROWS : dpg::GR_TM);
}
int64_t cross_slots(int T, int d, int kind) {
  const int64_t nq = cross_blocks(T, kind);
  return nq * nq * (kind == dpg::CROSS_STAGED ? ceil_div(d, dpg::CR_FCHUNK) : 1);
}

size_t dp_tied_cross_term_workspace(int B, int T, int d) {
  if (B <= 0 || T <= 0 || d <= 0) return 0;
  int64_t m = 0;
  for (int kind : {dpg::CROSS_STAGED, dpg::CROSS_DL, dpg::CROSS_ROWS})
    if (kind != dpg::CROSS_ROWS || T <= dpg::CX_ROWS_T) m = std::max(m, cross_slots(T, d, kind));
  return align_up((size_t)B * m * 4);
}

dp_status_t dp_tied_cross_term(const int32_t* ids, const void* dE, int64_t lde, const void* H,
                               int64_t ldh, const void* Gz, int64_t ldz, int B, int T, int V,
                               int d, dp_dtype_t dt, float scale, float* out, int accumulate,
                               void* workspace, size_t workspace_bytes, void* stream) {
  if (!ids || !dE || !H || !Gz || !out) return fail(DP_EINVAL, "a required pointer is NULL");
  if (B <= 0 || T <= 0 || V <= 0 || d <= 0)
    return fail(DP_EINVAL, "B, T, V and d must be positive");
  if (lde < d || ldh < d || ldz < V) return fail(DP_EINVAL, "row stride smaller than row width");
  if (!dtype_ok(dt)) return fail(DP_EINVAL, "unknown dtype %d", (int)dt);
  if (!std::isfinite(scale)) return fail(DP_EINVAL, "scale must be finite");
  if (T > 65536) return fail(DP_EUNSUPPORTED, "T = %d exceeds 65536", T);
  if (!span_ok(T, lde, dt) || !span_ok(T, ldh, dt) || !span_ok(T, ldz, dt))
    return fail(DP_EUNSUPPORTED, "one example's rows of an operand span 4 GiB or more");
  const size_t need = dp_tied_cross_term_workspace(B, T, d);
  if (!workspace || workspace_bytes < need)
    return fail(DP_EINVAL, "workspace of %zu bytes needed", need);
  dpg::CrossArgs a{};
  a.ids = ids; a.E = dE; a.H = H; a.Gz = Gz;
  a.lde = lde; a.ldh = ldh; a.ldz = ldz;
  a.B = B; a.T = T; a.V = V; a.d = d;
  const bool vec = vec_ok(dE, lde, dt) && vec_ok(H, ldh, dt);
  a.kind = dpg::cross_kind(kdt(dt), vec, T);
  a.n_t = (int)cross_blocks(T, a.kind);
  a.n_fc = a.kind == dpg::CROSS_STAGED ? (int)ceil_div(d, dpg::CR_FCHUNK) : 1;
  a.slots = (int32_t)cross_slots(T, d, a.kind);
  a.ws = static_cast<float*>(workspace);
  hipStream_t s = as_stream(stream);
  dp_status_t st = hip_status(dpg::launch_tied_cross(a, kdt(dt), vec, s), "tied_cross launch");
  if (st != DP_OK) return st;
  return hip_status(dpg::launch_finish_rows(a.ws, B, a.slots, out, accumulate, scale, s),
                    "finish launch");
}

dp_status_t dp_clip_factors(const float* norm2, int B, float C, float* c, void* stream) {
  if (!norm2 || !c) return fail(DP_EINVAL, "norm2 or c is NULL");
  if (B <= 0) return fail(DP_EINVAL, "B must be positive");
  if (!(C > 0.f) || !std::isfinite(C)) return fail(DP_EINVAL, "C must be positive and finite");
  return hip_status(dpg::launch_clip_factors(norm2, nullptr, B, C, 1.f, c, nullptr,
                                            as_stream(stream)),
                    "clip launch");
}

dp_status_t dp_clip_factors_scaled(const float* norm2, int B, float C, float scale, float* c,
                                   float* c_scaled, void* stream) {
  if (!norm2 || !c_scaled) return fail(DP_EINVAL, "norm2 or c_scaled is NULL");
  if (B <= 0) return fail(DP_EINVAL, "B must be positive");
  if (!(C > 0.f) || !std::isfinite(C)) return fail(DP_EINVAL, "C must be positive and finite");
  if (!std::isfinite(scale)) return fail(DP_EINVAL, "scale must be finite");
  return hip_status(dpg::launch_clip_factors(norm2, nullptr, B, C, scale, c, c_scaled,
                                            as_stream(stream)),
                    "clip launch");
}

dp_status_t dp_clip_factors_scaled2(const float* norm2_a, const float* norm2_b, int B, float C,
                                    float scale, float* c, float* c_scaled, void* stream) {
  if (!norm2_a || !norm2_b || !c_scaled)
    return fail(DP_EINVAL, "norm2_a, norm2_b or c_scaled is NULL");
  if (B <= 0) return fail(DP_EINVAL, "B must be positive");
  if (!(C > 0.f) || !std::isfinite(C)) return fail(DP_EINVAL, "C must be positive and finite");
  if (!std::isfinite(scale)) return fail(DP_EINVAL, "scale must be finite");
  return hip_status(dpg::launch_clip_factors(norm2_a, norm2_b, B, C, scale, c, c_scaled,
                                            as_stream(stream)),
                    "clip launch");
}

size_t dp_clipped_grad_sum_workspace(int B, int T, int d_out, int with_ids) {
  if (!with_ids || B <= 0 || T <= 0 || d_out <= 0) return 0;
  return es_layout((int64_t)B * T, d_out).total;
}

dp_status_t dp_clipped_grad_sum_grouped(const dp_linear_t* layers, float* const* outs,
                                        int n_layers, const float* c, int B, int T,
                                        dp_dtype_t dt, int transpose_out, int accumulate,
                                        void* stream) {
  dp_status_t st = check_layers(layers, n_layers, B, T, dt);
  if (st != DP_OK) return st;
  if (!outs || !c) return fail(DP_EINVAL, "outs or c is NULL");
  if ((int64_t)B * T > (int64_t(1) << 40)) return fail(DP_EUNSUPPORTED, "B*T too large");
  std::vector<GemmEntry> entries;
  for (int i = 0; i < n_layers; ++i) {
    if (!outs[i]) return fail(DP_EINVAL, "outs[%d] is NULL", i);
    plan_sum(layers[i], transpose_out, dt, outs[i], entries);
    entries.back().acc = accumulate ? 1 : 0;
  }
  return run_gemm(entries, 0, B, T, dt, c, nullptr, 0, 0, NoiseCfg{}, as_stream(stream));
}

static dp_status_t noised_sum_plan(const dp_linear_t* layers, float* const* outs,
                                   const uint64_t* tensor_ids, const int32_t* accumulate,
                                   int n_layers, int B, int T, dp_dtype_t dt, int transpose_out,
                                   std::vector<GemmEntry>& entries) {
  dp_status_t st = check_layers(layers, n_layers, B, T, dt);
  if (st != DP_OK) return st;
  if ((int64_t)B * T > (int64_t(1) << 40)) return fail(DP_EUNSUPPORTED, "B*T too large");
  for (int i = 0; i < n_layers; ++i) {
    if (outs && !outs[i]) return fail(DP_EINVAL, "outs[%d] is NULL", i);
    if (tensor_ids && tensor_ids[i] >> 32)
      return fail(DP_EINVAL, "tensor_ids[%d] must be < 2^32", i);
    plan_sum(layers[i], transpose_out, dt, outs ? outs[i] : nullptr, entries);
    entries.back().acc = accumulate && accumulate[i] ? 1 : 0;
    entries.back().tensor_id = tensor_ids ? (uint32_t)tensor_ids[i] : 0u;
  }
  return DP_OK;
}

size_t dp_clipped_grad_sum_noised_grouped_workspace(const dp_linear_t* layers, int n_layers,
                                                    int B, int T, dp_dtype_t dt,
                                                    int transpose_out) {
  std::vector<GemmEntry> entries;
  if (noised_sum_plan(layers, nullptr, nullptr, nullptr, n_layers, B, T, dt, transpose_out,
                      entries) != DP_OK)
    return 0;
  return align_up(sum_split_bytes(entries, B, T, dt));
}

dp_status_t dp_clipped_grad_sum_noised_grouped_ws(const dp_linear_t* layers, float* const* outs,
                                                  const uint64_t* tensor_ids,
                                                  const int32_t* accumulate, int n_layers,
                                                  const float* c, int B, int T, dp_dtype_t dt,
                                                  int transpose_out, float sigma, float C,
                                                  int B_norm, uint64_t seed, uint64_t step,
                                                  void* workspace, size_t workspace_bytes,
                                                  void* stream) {
  if (!outs || !c || !tensor_ids) return fail(DP_EINVAL, "outs, c or tensor_ids is NULL");
  std::vector<GemmEntry> entries;
  dp_status_t st = noised_sum_plan(layers, outs, tensor_ids, accumulate, n_layers, B, T, dt,
                                   transpose_out, entries);
  if (st != DP_OK) return st;
  st = check_noise_args(sigma, C, B_norm, step);
  if (st != DP_OK) return st;
  if (workspace_bytes && !workspace) return fail(DP_EINVAL, "workspace is NULL");
  NoiseCfg nz;
  nz.on = true;
  nz.sigma_c = (float)((double)sigma * (double)C);
  nz.inv_b = B_norm > 0 ? (float)(1.0 / (double)B_norm) : 1.f;
  nz.seed = seed;
  nz.step = (uint32_t)step;
  return run_gemm(entries, 0, B, T, dt, c, nullptr, 0, 0, nz, as_stream(stream),
                  static_cast<float*>(workspace), workspace ? workspace_bytes : 0);
}

dp_status_t dp_clipped_grad_sum_noised_grouped(const dp_linear_t* layers, float* const* outs,
                                               const uint64_t* tensor_ids,
                                               const int32_t* accumulate, int n_layers,
                                               const float* c, int B, int T, dp_dtype_t dt,
                                               int transpose_out, float sigma, float C,
                                               int B_norm, uint64_t seed, uint64_t step,
                                               void* stream) {
  return dp_clipped_grad_sum_noised_grouped_ws(layers, outs, tensor_ids, accumulate, n_layers, c,
                                               B, T, dt, transpose_out, sigma, C, B_norm, seed,
                                               step, nullptr, 0, stream);
}

// ------------------------------------------------------- gradient store
// The direct norm's per-example tiles kept in HBM and summed with the clip
// factors afterwards (see the header). Entries are planned in table order,
// X = A, Y = G, so that entry i's slot_begin is its first tile slot.
static dp_status_t store_plan(const dp_linear_t* layers, int n_layers, int B, int T,
                              dp_dtype_t dt, std::vector<GemmEntry>& entries, int64_t* tiles) {
  dp_status_t st = check_layers(layers, n_layers, B, T, dt);
  if (st != DP_OK) return st;
  if (kdt(dt) != dpg::DT_BF16 || T % dpg::DL_SUM_BK != 0)
    return fail(DP_EUNSUPPORTED, "the gradient store needs bf16 and T a multiple of %d",
                dpg::DL_SUM_BK);
  int64_t slots = 0;
  for (int i = 0; i < n_layers; ++i) {
    const dp_linear_t& L = layers[i];
    plan_gemm(L.A, L.lda, L.d_in, L.G, L.ldg, L.d_out, dt, nullptr, 0, entries, &slots, 1);
    if (!entries.back().vec)
      return fail(DP_EUNSUPPORTED, "layer %d: the gradient store needs 16-byte aligned rows", i);
  }
  if ((uint64_t)B * (uint64_t)slots > 0x7FFFFFFFull)
    return fail(DP_EUNSUPPORTED, "too many tiles for the gradient store");
  *tiles = slots;
  return DP_OK;
}

static size_t store_tiles_bytes(int B, int64_t tiles) {
  return (size_t)B * (size_t)tiles * dpg::STORE_TILE_FLOATS * 4;
}

size_t dp_grad_store_bytes(const dp_linear_t* layers, int n_layers, int B, int T,
                           dp_dtype_t dt) {
  std::vector<GemmEntry> entries;
  int64_t tiles = 0;
  if (store_plan(layers, n_layers, B, T, dt, entries, &tiles) != DP_OK) return 0;
  return store_tiles_bytes(B, tiles) + align_up((size_t)B * (size_t)tiles * 4);
}

dp_status_t dp_ghost_norm_linear_store(const dp_linear_t* layers, int n_layers, int B, int T,
                                       dp_dtype_t dt, float* norm2, int accumulate, void* store,
                                       size_t store_bytes, void* stream) {
  std::vector<GemmEntry> entries;
  int64_t tiles = 0;
  dp_status_t st = store_plan(layers, n_layers, B, T, dt, entries, &tiles);
  if (st != DP_OK) return st;
  if (!norm2) return fail(DP_EINVAL, "norm2 is NULL");
  const size_t need = store_tiles_bytes(B, tiles) + align_up((size_t)B * (size_t)tiles * 4);
  if (!store || store_bytes < need)
    return fail(DP_EINVAL, "gradient store of %zu bytes needed, %zu given", need,
                store ? store_bytes : (size_t)0);
  if ((uintptr_t)store % 16)
    return fail(DP_EINVAL, "the gradient store must be 16-byte aligned");
  hipStream_t s = as_stream(stream);
  float* tiles_f = static_cast<float*>(store);
  float* ws = reinterpret_cast<float*>(static_cast<char*>(store) + store_tiles_bytes(B, tiles));
  st = run_gemm(entries, 1, B, T, dt, nullptr, ws, tiles, 0, NoiseCfg{}, s, nullptr, 0, tiles_f);
  if (st != DP_OK) return st;
  return hip_status(dpg::launch_finish_rows(ws, B, (int)tiles, norm2, accumulate, 1.f, s),
                    "finish launch");
}

dp_status_t dp_clipped_grad_sum_noised_store(const dp_linear_t* layers, float* const* outs,
                                             const uint64_t* tensor_ids,
                                             const int32_t* accumulate,
                                             const int32_t* transpose_out, int n_layers,
                                             const float* c, int B, int T, dp_dtype_t dt,
                                             float sigma, float C, int B_norm, uint64_t seed,
                                             uint64_t step, const void* store,
                                             size_t store_bytes, void* stream) {
  if (!outs || !c || !tensor_ids) return fail(DP_EINVAL, "outs, c or tensor_ids is NULL");
  std::vector<GemmEntry> entries;
  int64_t tiles = 0;
  dp_status_t st = store_plan(layers, n_layers, B, T, dt, entries, &tiles);
  if (st != DP_OK) return st;
  st = check_noise_args(sigma, C, B_norm, step);
  if (st != DP_OK) return st;
  if (!store || store_bytes < store_tiles_bytes(B, tiles))
    return fail(DP_EINVAL, "gradient store of %zu bytes needed, %zu given",
                store_tiles_bytes(B, tiles), store ? store_bytes : (size_t)0);
  if ((uintptr_t)store % 16)
    return fail(DP_EINVAL, "the gradient store must be 16-byte aligned");
  for (int i = 0; i < n_layers; ++i) {
    if (!outs[i]) return fail(DP_EINVAL, "outs[%d] is NULL", i);
    if (tensor_ids[i] >> 32) return fail(DP_EINVAL, "tensor_ids[%d] must be < 2^32", i);
    GemmEntry& e = entries[i];
    e.out = outs[i];
    e.ldo = transpose_out && transpose_out[i] ? layers[i].d_in : layers[i].d_out;
    e.acc = accumulate && accumulate[i] ? 1 : 0;
    e.tensor_id = (uint32_t)tensor_ids[i];
  }
  hipStream_t s = as_stream(stream);
  for (size_t i0 = 0; i0 < entries.size(); i0 += dpg::GM_MAX_LAYERS) {
    const size_t n = std::min(entries.size() - i0, (size_t)dpg::GM_MAX_LAYERS);
    dpg::GemmArgs a{};
    a.B = B; a.T = T; a.c = c;
    a.noise = 1;
    a.sigma_c = (float)((double)sigma * (double)C);
    a.inv_b = B_norm > 0 ? (float)(1.0 / (double)B_norm) : 1.f;
    a.seed = seed;
    a.step = (uint32_t)step;
    a.store = static_cast<float*>(const_cast<void*>(store));
    a.eg = 1;
    uint64_t items = 0;
    for (size_t j = 0; j < n; ++j) {
      const GemmEntry& e = entries[i0 + j];
      dpg::GemmLayer& L = a.L[j];
      L.X = nullptr; L.Y = nullptr;
      L.store_slot = e.slot_begin;
      L.store_transpose = transpose_out && transpose_out[i0 + j] ? 1 : 0;
      L.M = e.M; L.N = e.N;
      L.tm = (uint16_t)e.tm; L.tn = (uint16_t)e.tn;
      L.tile_begin = (uint32_t)items;
      L.tensor_id = e.tensor_id;
      L.accumulate = e.acc;
      L.out = e.out; L.ldo = e.ldo;
      items += (uint64_t)e.tm * e.tn;
    }
    if (items > 0xFFFFFFFFull) return fail(DP_EUNSUPPORTED, "too many work items");
    a.n_layers = (int32_t)n;
    a.n_items = (uint32_t)items;
    st = hip_status(dpg::launch_store_sum(a, s), "store_sum launch");
    if (st != DP_OK) return st;
  }
  return DP_OK;
}

// Shared checks and argument set-up of the embedding-form sums.
static dp_status_t embed_sum_args(const int32_t* ids, const void* G, int64_t ldg, const float* c,
                                  int B, int T, int V, int d, bool compact, void* workspace,
                                  size_t workspace_bytes, dpg::EmbedSumArgs& a) {
  if (B <= 0 || T <= 0 || V <= 0 || d <= 0)
    return fail(DP_EINVAL, "B, T, V and d must be positive");
  const int64_t K = (int64_t)B * T;
  if (K > INT32_MAX)
    return fail(DP_EUNSUPPORTED, "B*T = %lld exceeds 2^31 - 1", (long long)K);
  const int pbits = std::max(1, bits_for(K));
  if (bits_for((int64_t)V + 1) + pbits > 32)  // ids are clamped to V, so V + 1 values
    return fail(DP_EUNSUPPORTED, "V and B*T do not fit a 32-bit sort key");
  const EsLayout l = es_layout(K, d, compact);
  if (!workspace || workspace_bytes < l.total)
    return fail(DP_EINVAL, "workspace of %zu bytes needed", l.total);
  char* w = static_cast<char*>(workspace);
  a = dpg::EmbedSumArgs{};
  a.ids = ids; a.E = G; a.lde = ldg; a.c = c;
  a.B = B; a.K = (int32_t)K; a.T = T; a.V = V; a.d = d;
  a.pbits = pbits;
  a.keys = reinterpret_cast<uint32_t*>(w + l.keys);
  a.head = reinterpret_cast<float*>(w + l.head);
  a.tail = reinterpret_cast<float*>(w + l.tail);
  if (compact) {
    a.rank = reinterpret_cast<int32_t*>(w + l.rank);
    a.seg = reinterpret_cast<int32_t*>(w + l.seg);
    a.n_runs = reinterpret_cast<int32_t*>(w + l.n_runs);
    a.rows = reinterpret_cast<float*>(w + l.rows);
  }
  if (K > dpg::ES_MAX_K) {
    a.gs_blocks = a.gs_nbs = (int32_t)ceil_div(K, dpg::GS_KB);
    a.gs_seg = (int32_t)K;
    a.keys2 = reinterpret_cast<uint32_t*>(w + l.keys2);
    a.hist = reinterpret_cast<int32_t*>(w + l.hist);
    a.gs_runs = reinterpret_cast<int32_t*>(w + l.gs_runs);
  }
  return DP_OK;
}

size_t dp_embedding_rows_workspace(int B, int T, int d) {
  if (B <= 0 || T <= 0 || d <= 0) return 0;
  return es_layout((int64_t)B * T, d, true).total;
}

dp_status_t dp_embedding_rows(const void* G, int64_t ldg, const int32_t* ids, const float* c,
                              int B, int T, int V, int d, dp_dtype_t dt, void* workspace,
                              size_t workspace_bytes, void* stream) {
  if (!G || !ids || !c) return fail(DP_EINVAL, "G, ids or c is NULL");
  if (!dtype_ok(dt)) return fail(DP_EINVAL, "unknown dtype %d", (int)dt);
  if (ldg < d) return fail(DP_EINVAL, "ldg < d");
  dpg::EmbedSumArgs a;
  dp_status_t st = embed_sum_args(ids, G, ldg, c, B, T, V, d, true, workspace, workspace_bytes,
                                  a);
  if (st != DP_OK) return st;
  return hip_status(dpg::launch_embed_rows(a, kdt(dt), as_stream(stream)), "embed_rows launch");
}

dp_status_t dp_embedding_rows_add(const void* workspace, size_t workspace_bytes, int B, int T,
                                  int V, int d, int transpose_out, float* out, void* stream) {
  if (!out) return fail(DP_EINVAL, "out is NULL");
  dpg::EmbedSumArgs a;
  dp_status_t st = embed_sum_args(nullptr, nullptr, d, nullptr, B, T, V, d, true,
                                  const_cast<void*>(workspace), workspace_bytes, a);
  if (st != DP_OK) return st;
  a.out = out;
  a.ldo = transpose_out ? V : d;
  a.transpose = transpose_out ? 1 : 0;
  return hip_status(dpg::launch_embed_scatter(a, as_stream(stream)), "embed_scatter launch");
}

dp_status_t dp_clipped_grad_sum(const void* A, int64_t lda, const void* G, int64_t ldg,
                                const int32_t* ids, const float* c, int B, int T, int d_in,
                                int d_out, dp_dtype_t dt, int transpose_out, float* out,
                                int accumulate, void* workspace, size_t workspace_bytes,
                                void* stream) {
  if (!ids) {
    dp_linear_t L{A, lda, d_in, G, ldg, d_out, DP_NORM_AUTO};
    return dp_clipped_grad_sum_grouped(&L, &out, 1, c, B, T, dt, transpose_out, accumulate,
                                       stream);
  }
  // Embedding form: A = onehot(ids), d_in = V.
  if (A) return fail(DP_EINVAL, "pass either A or ids, not both");
  if (!G || !c || !out) return fail(DP_EINVAL, "G, c or out is NULL");
  if (ldg < d_out) return fail(DP_EINVAL, "ldg < d_out");
  if (!dtype_ok(dt)) return fail(DP_EINVAL, "unknown dtype %d", (int)dt);
  dpg::EmbedSumArgs a;
  dp_status_t st = embed_sum_args(ids, G, ldg, c, B, T, d_in, d_out, false, workspace,
                                  workspace_bytes, a);
  if (st != DP_OK) return st;
  hipStream_t s = as_stream(stream);
  if (!accumulate) {
    st = hip_status(dpg::launch_fill_zero(out, (int64_t)d_in * d_out, s), "fill");
    if (st != DP_OK) return st;
  }
  a.out = out;
  a.ldo = transpose_out ? d_in : d_out;
  a.transpose = transpose_out ? 1 : 0;
  return hip_status(dpg::launch_embed_sum(a, kdt(dt), s), "embed_sum launch");
}

static dp_status_t noise_call(float* grad, int64_t n, float sigma, float C, int B_norm,
                              uint64_t seed, uint64_t tensor_id, uint64_t step, bool accumulate,
                              void* stream) {
  if (n < 0) return fail(DP_EINVAL, "n must be >= 0");
  if (n > 0 && !grad) return fail(DP_EINVAL, "grad is NULL");
  if (!(sigma >= 0.f) || !std::isfinite(sigma)) return fail(DP_EINVAL, "sigma must be >= 0");
  if (!(C > 0.f) || !std::isfinite(C)) return fail(DP_EINVAL, "C must be positive and finite");
  if (B_norm < 0) return fail(DP_EINVAL, "B_norm must be >= 0");
  if (tensor_id >> 32 || step >> 32) return fail(DP_EINVAL, "tensor_id and step must be < 2^32");
  const float sigma_c = (float)((double)sigma * (double)C);
  const float inv_b = B_norm > 0 ? (float)(1.0 / (double)B_norm) : 1.f;
  return hip_status(dpg::launch_add_noise(grad, n, sigma_c, inv_b, seed, (uint32_t)tensor_id,
                                          (uint32_t)step, accumulate, as_stream(stream)),
                    "noise launch");
}

dp_status_t dp_add_noise(float* grad, int64_t n, float sigma, float C, int B_norm, uint64_t seed,
                         uint64_t tensor_id, uint64_t step, void* stream) {
  return noise_call(grad, n, sigma, C, B_norm, seed, tensor_id, step, true, stream);
}

dp_status_t dp_noise_fill(float* out, int64_t n, float sigma, float C, int B_norm, uint64_t seed,
                          uint64_t tensor_id, uint64_t step, void* stream) {
  return noise_call(out, n, sigma, C, B_norm, seed, tensor_id, step, false, stream);
}


size_t dp_vector_grads_workspace(const dp_vector_t* params, int n, int B, int T, dp_dtype_t dt) {
  if (check_vec(params, n, B, T, dt) != DP_OK) return 0;
  VecPlan p;
  plan_vec_grads(p, params, n, nullptr, dt, T);
  return align_up((size_t)B * p.slots * 4);
}

dp_status_t dp_vector_grads_grouped(const dp_vector_t* params, int n, int B, int T,
                                    dp_dtype_t dt, float* const* grads, float* norm2,
                                    int accumulate, void* workspace, size_t workspace_bytes,
                                    void* stream) {
  dp_status_t st = check_vec(params, n, B, T, dt);
  if (st != DP_OK) return st;
  if (!grads) return fail(DP_EINVAL, "grads is NULL");
  for (int i = 0; i < n; ++i)
    if (!grads[i]) return fail(DP_EINVAL, "grads[%d] is NULL", i);
  VecPlan p;
  plan_vec_grads(p, params, n, grads, dt, T);
  const size_t need = align_up((size_t)B * p.slots * 4);
  if (!workspace || workspace_bytes < need)
    return fail(DP_EINVAL, "workspace of %zu bytes needed", need);
  float* ws = static_cast<float*>(workspace);
  hipStream_t s = as_stream(stream);
  st = run_vec(p, B, T, dt, ws, s);
  if (st != DP_OK || !norm2) return st;
  return hip_status(dpg::launch_finish_rows(ws, B, (int)p.slots, norm2, accumulate, 1.f, s),
                    "finish launch");
}

dp_status_t dp_vector_clipped_sum_noised_grouped(const float* const* grads, const int32_t* d,
                                                 int n, int B, const float* c,
                                                 float* const* outs, const uint64_t* tensor_ids,
                                                 const int32_t* accumulate, float sigma, float C,
                                                 int B_norm, uint64_t seed, uint64_t step,
                                                 void* stream) {
  if (!grads || !d || !outs || !c || !tensor_ids)
    return fail(DP_EINVAL, "grads, d, outs, c or tensor_ids is NULL");
  if (n <= 0 || B <= 0) return fail(DP_EINVAL, "n and B must be positive");
  dp_status_t st = check_noise_args(sigma, C, B_norm, step);
  if (st != DP_OK) return st;
  for (int i = 0; i < n; ++i) {
    if (!grads[i] || !outs[i]) return fail(DP_EINVAL, "grads[%d] or outs[%d] is NULL", i, i);
    if (d[i] <= 0) return fail(DP_EINVAL, "d[%d] must be positive", i);
    if (tensor_ids[i] >> 32) return fail(DP_EINVAL, "tensor_ids[%d] must be < 2^32", i);
  }
  hipStream_t s = as_stream(stream);
  for (int i0 = 0; i0 < n; i0 += dpg::VS_MAX_PARAMS) {
    dpg::VecSumArgs a{};
    a.B = B; a.c = c; a.noise = 1;
    a.sigma_c = (float)((double)sigma * (double)C);
    a.inv_b = B_norm > 0 ? (float)(1.0 / (double)B_norm) : 1.f;
    a.seed = seed; a.step = (uint32_t)step;
    uint64_t quads = 0;
    const int m = std::min(n - i0, dpg::VS_MAX_PARAMS);
    for (int j = 0; j < m; ++j) {
      dpg::VecSumParam& P = a.P[j];
      P.grad = grads[i0 + j]; P.out = outs[i0 + j]; P.d = d[i0 + j];
      P.quad_begin = (uint32_t)quads;
      P.tensor_id = (uint32_t)tensor_ids[i0 + j];
      P.accumulate = accumulate && accumulate[i0 + j] ? 1 : 0;
      quads += (uint64_t)ceil_div(d[i0 + j], 4);
    }
    if (quads > 0xFFFFFFFFull) return fail(DP_EUNSUPPORTED, "too many features");
    a.n_params = m;
    a.n_quads = (uint32_t)quads;
    st = hip_status(dpg::launch_vec_sum(a, s), "vec_sum launch");
    if (st != DP_OK) return st;
  }
  return DP_OK;
}

size_t dp_ghost_norm_positional_workspace(int B, int T, int d) {
  if (B <= 0 || T <= 0 || d <= 0) return 0;
  // at most 256 features per chunk (fp32): an upper bound for both dtypes
  return align_up((size_t)B * (size_t)ceil_div(d, 256) * (size_t)ceil_div(T, VEC_SQ_ROWS) * 4);
}

dp_status_t dp_ghost_norm_positional(const void* dE, int64_t lde, int B, int T, int d,
                                     dp_dtype_t dt, float* norm2, int accumulate,
                                     void* workspace, size_t workspace_bytes, void* stream) {
  if (!dE || !norm2) return fail(DP_EINVAL, "dE or norm2 is NULL");
  dp_vector_t v{nullptr, 0, dE, lde, d};
  dp_status_t st = check_vec(&v, 1, B, T, dt);
  if (st != DP_OK) return st;
  VecPlan p;
  plan_vec(p, nullptr, 0, dE, lde, d, dpg::VEC_SQ, nullptr, dt, T);
  const size_t need = align_up((size_t)B * p.slots * 4);
  if (!workspace || workspace_bytes < need)
    return fail(DP_EINVAL, "workspace of %zu bytes needed", need);
  float* ws = static_cast<float*>(workspace);
  hipStream_t s = as_stream(stream);
  st = run_vec(p, B, T, dt, ws, s);
  if (st != DP_OK) return st;
  return hip_status(dpg::launch_finish_rows(ws, B, (int)p.slots, norm2, accumulate, 1.f, s),
                    "finish launch");
}

dp_status_t dp_clipped_grad_sum_positional_noised(const void* dE, int64_t lde, const float* c,
                                                  int B, int T, int d, dp_dtype_t dt, float* out,
                                                  int n_pos, int64_t ldo, uint64_t tensor_id,
                                                  int accumulate, float sigma, float C,
                                                  int B_norm, uint64_t seed, uint64_t step,
                                                  void* stream) {
  if (!dE || !c || !out) return fail(DP_EINVAL, "dE, c or out is NULL");
  if (B <= 0 || T <= 0 || d <= 0 || n_pos <= 0)
    return fail(DP_EINVAL, "B, T, d and n_pos must be positive");
  if (T > n_pos) return fail(DP_EINVAL, "T = %d exceeds the table's %d rows", T, n_pos);
  if (lde < d || ldo < d) return fail(DP_EINVAL, "row stride smaller than d");
  if (!dtype_ok(dt)) return fail(DP_EINVAL, "unknown dtype %d", (int)dt);
  if (tensor_id >> 32) return fail(DP_EINVAL, "tensor_id must be < 2^32");
  dp_status_t st = check_noise_args(sigma, C, B_norm, step);
  if (st != DP_OK) return st;
  dpg::PosSumArgs a{};
  a.E = dE; a.lde = lde; a.c = c; a.out = out; a.ldo = ldo;
  a.B = B; a.T = T; a.d = d; a.n_pos = n_pos;
  a.accumulate = accumulate ? 1 : 0; a.noise = 1;
  a.sigma_c = (float)((double)sigma * (double)C);
  a.inv_b = B_norm > 0 ? (float)(1.0 / (double)B_norm) : 1.f;
  a.tensor_id = (uint32_t)tensor_id; a.step = (uint32_t)step; a.seed = seed;
  return hip_status(dpg::launch_pos_sum(a, kdt(dt), as_stream(stream)), "pos_sum launch");
}

}  // extern "C"
