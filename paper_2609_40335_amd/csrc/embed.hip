// Token-id keyed kernels: bucketing, the input-embedding ghost norm and the
// input-embedding part of the clipped sum.
//
// The input embedding looks up row x_t of E for every token (Sec. "Weight
// Tying in Decoder-Only LLMs"), so its per-example gradient has one nonzero
// row per distinct id v: the sum of the output-gradients dE_t of the tokens
// with x_t = v. Its squared norm is sum_v ||sum_{t: x_t = v} dE_t||^2.
//
// Bucketing sorts the packed keys (id << pbits | position) of one example in
// LDS (a stable radix sort on the id bits), marks the first token of each run
// of equal ids, and turns the marks into dense ranks with a wavefront-shuffle
// prefix scan. The norm takes one of two forms. Short bf16 examples (T up
// to 128, 16-byte rows) take the pairwise form of the same quantity, sum over
// token pairs with equal ids of <dE_t, dE_s> (the ghost-norm identity with
// one-hot inputs), on MFMA, beside a workgroup that ranks the ids for the
// buckets. Otherwise each bucket's rows are summed (runs split over
// workgroups, coalesced row reads) and squared. The clipped sum sorts all
// B*T tokens of the batch (radix sort on
// the ids, below) and reduces runs of equal ids in fixed 32-token blocks; a run that crosses a
// block boundary is closed by a fix-up pass that adds the block partials in
// order. Every output row is written by exactly one wave: no atomics, and
// results are bitwise reproducible.
#include "common.hpp"
#include "kernels.hpp"

namespace dpg {

constexpr int EN_THREADS = 256;
static_assert(EN_CT_T <= EN_THREADS, "counting rank: one key per thread");
constexpr int ES_THREADS = 1024;
constexpr int ES_WAVES = 4;  // waves per workgroup of the block and fix-up passes

// Inclusive prefix sum of one value per thread across the workgroup:
// shuffles within each wavefront, then the wave totals through LDS.
__device__ int block_inclusive_scan(int v, int* wave_tot, int tid, int nthreads, int* total) {
  const int lane = tid & 63, w = tid >> 6, nw = nthreads >> 6;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int u = __shfl_up(v, off, 64);
    if (lane >= off) v += u;
  }
  if (lane == 63) wave_tot[w] = v;
  __syncthreads();
  int base = 0, tot = 0;
  for (int i = 0; i < nw; ++i) {
    if (i < w) base += wave_tot[i];
    tot += wave_tot[i];
  }
  __syncthreads();
  *total = tot;
  return v + base;
}

// For n sorted keys: dense rank of every sorted position (rank[p]) and the
// first sorted position of every bucket (seg[r], with seg[n_buckets] = n).
// Returns the number of buckets. Each thread handles a contiguous run.
__device__ int rank_sorted(const uint32_t* keys, int n, int pbits, int32_t* rank, int32_t* seg,
                           int* wave_tot, int tid, int nthreads) {
  const int per = (n + nthreads - 1) / nthreads;
  const int p0 = min(tid * per, n), p1 = min(p0 + per, n);
  int cnt = 0;
  for (int p = p0; p < p1; ++p)
    cnt += (p == 0 || (keys[p] >> pbits) != (keys[p - 1] >> pbits)) ? 1 : 0;
  int total;
  const int incl = block_inclusive_scan(cnt, wave_tot, tid, nthreads, &total);
  int r = incl - cnt;
  for (int p = p0; p < p1; ++p) {
    if (p == 0 || (keys[p] >> pbits) != (keys[p - 1] >> pbits)) seg[r++] = p;
    rank[p] = r - 1;
  }
  if (tid == 0) seg[total] = n;
  __syncthreads();
  return total;
}

// Stable LSD radix sort, 8 bits per pass, of n keys (id << pb | position)
// held in LDS buffer buf0, over the bits of the ids 0..V (ids at or past V
// must already be clamped to V). The keys arrive in position order, so the
// result is the (id, position) order. NW waves; wave w owns a contiguous
// segment of the keys. A pass counts digits per wave (cnt[w][digit]), turns
// the counts into offsets in digit-major, wave-minor order, and scatters each
// wave's keys 64 at a time: lanes with equal digits are found with eight
// ballots and ranked by lane; the group's lowest lane advances the wave's
// running offset. Returns the index of the buffer that holds the result.
// One stable LSD radix pass, 8 bits at bit `sh`, of n keys from LDS buffer
// `in` to `out`. NW waves; wave w owns a contiguous segment of the keys. The
// pass counts digits per wave (cnt[w][digit]), turns the counts into
// offsets in digit-major, wave-minor order, and scatters each wave's keys 64
// at a time: lanes with equal digits are found with eight ballots and ranked
// by lane; the group's lowest lane advances the wave's running offset.
template <int NW>
__device__ void lds_radix_pass(const uint32_t* in, uint32_t* out, int n, int sh, int* cnt,
                               int* wave_tot) {
  static_assert(NW % 4 == 0, "4 (digit, wave) entries per thread");
  constexpr int NT = NW * WAVE;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int seg_len = ((n + NW - 1) / NW + WAVE - 1) / WAVE * WAVE;
  const int s0 = min(w * seg_len, n), s1 = min(s0 + seg_len, n);
  const uint64_t lt = (1ull << lane) - 1ull;
  for (int i = tid; i < NW * 256; i += NT) cnt[i] = 0;
  __syncthreads();
  for (int p = s0 + lane; p < s1; p += WAVE) atomicAdd(&cnt[w * 256 + ((in[p] >> sh) & 255)], 1);
  __syncthreads();
  {
    // thread t holds entries 4t .. 4t+3 of the (digit, wave) order
    const int d = (4 * tid) / NW, w0 = (4 * tid) % NW;
    int v[4], loc = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) { v[q] = cnt[(w0 + q) * 256 + d]; loc += v[q]; }
    int total;
    const int incl = block_inclusive_scan(loc, wave_tot, tid, NT, &total);
    int run = incl - loc;
#pragma unroll
    for (int q = 0; q < 4; ++q) { cnt[(w0 + q) * 256 + d] = run; run += v[q]; }
  }
  __syncthreads();
  for (int base = s0; base < s1; base += WAVE) {
    const int p = base + lane;
    const bool valid = p < s1;
    const uint32_t key = valid ? in[p] : 0u;
    const int dg = (int)((key >> sh) & 255);
    uint64_t m = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const uint64_t mb = __ballot(valid && ((dg >> bit) & 1));
      m &= ((dg >> bit) & 1) ? mb : ~mb;
    }
    const int rank = __popcll(m & lt);
    const int off = valid ? cnt[w * 256 + dg] : 0;
    if (valid) out[off + rank] = key;
    if (valid && rank == 0) cnt[w * 256 + dg] = off + __popcll(m);
  }
  __syncthreads();
}

// Bits of the values 0..V (the ids, clamped to V).
__device__ __forceinline__ int id_bits(uint32_t V) {
  int b = 0;
  while ((1u << b) <= V) ++b;
  return b;
}

// Stable LSD radix sort, 8 bits per pass, of n keys (id << pb | position)
// held in LDS buffer buf0, over the bits of the ids 0..V (ids at or past V
// must already be clamped to V). The keys arrive in position order, so the
// result is the (id, position) order. Returns the index of the buffer that
// holds the result.
template <int NW>
__device__ int lds_radix_sort(uint32_t* buf0, uint32_t* buf1, int n, int pb, uint32_t V, int* cnt,
                              int* wave_tot) {
  const int idbits = id_bits(V);
  int src = 0;
  for (int shift = 0; shift < idbits; shift += 8, src ^= 1)
    lds_radix_pass<NW>(src ? buf1 : buf0, src ? buf0 : buf1, n, pb + shift, cnt, wave_tot);
  return src;
}

template <int DT>
__device__ __forceinline__ float load_elem(const void* base, int64_t idx) {
  if constexpr (DT == DT_BF16)
    return bf16_to_f32(((const uint16_t*)base)[idx]);
  else
    return ((const float*)base)[idx];
}

// ---------------------------------------------------------------------------
// Per-example bucketing and input-embedding norm. Grid (B, ceil(d/64)).
// ---------------------------------------------------------------------------
template <int DT>
__global__ __launch_bounds__(EN_THREADS) void embed_norm_kernel(EmbedNormArgs a) {
  __shared__ uint32_t kbuf[2][EN_MAX_T];
  __shared__ int32_t rank[EN_MAX_T];
  __shared__ int32_t seg[EN_MAX_T + 1];
  __shared__ int cnt[(EN_THREADS / WAVE) * 256];
  __shared__ int wave_tot[EN_THREADS / WAVE];
  __shared__ float red[EN_THREADS / WAVE];
  const int b = blockIdx.x, chunk = blockIdx.y, tid = threadIdx.x;
  const int T = a.T;
  const uint32_t pmask = (1u << a.pbits) - 1u;
  const uint32_t V = (uint32_t)a.V;
  const int32_t* ids = a.ids + (int64_t)b * T;
  for (int p = tid; p < T; p += EN_THREADS) {
    const uint32_t id = (uint32_t)ids[p];
    kbuf[0][p] = ((id < V ? id : V) << a.pbits) | (uint32_t)p;
  }
  __syncthreads();
  const uint32_t* keys =
      kbuf[lds_radix_sort<EN_THREADS / WAVE>(kbuf[0], kbuf[1], T, a.pbits, V, cnt, wave_tot)];
  const int nseg = rank_sorted(keys, T, a.pbits, rank, seg, wave_tot, tid, EN_THREADS);
  if (chunk == 0) {
    if (a.seg_id)
      for (int p = tid; p < T; p += EN_THREADS)
        a.seg_id[(int64_t)b * T + (keys[p] & pmask)] = rank[p];
    if (a.n_unique && tid == 0) a.n_unique[b] = nseg;
  }
  // Bucket sums: wave w walks sorted positions [s_w, e_w) 32 rows at a time
  // (lane = feature), squaring each run of equal ids that closes inside its
  // range. A run that crosses a range boundary leaves partials: hp (the run
  // open at s_w, closing here or, if `through`, passing on) and tp (a run that
  // starts here and stays open at e_w). Wave 0 then chains them in order.
  constexpr int NW = EN_THREADS / WAVE;
  const int lane = tid & 63, w = tid >> 6;
  const int f = chunk * WAVE + lane;
  const bool fok = f < a.d;
  const int fs = fok ? f : a.d - 1;  // a feature index that is always in the row
  const int pb = a.pbits;
  const int64_t row0 = (int64_t)b * T;
  const int per = (T + NW - 1) / NW;
  const int s_w = min(w * per, T), e_w = min(s_w + per, T);
  bool h_open = false, t_open = false, through = false;
  float sq = 0.f, hp = 0.f, tp = 0.f;
  if (s_w < e_w) {
    h_open = s_w > 0 && (keys[s_w - 1] >> pb) == (keys[s_w] >> pb);
    bool in_head = h_open;  // the current run started before s_w
    float acc = 0.f;
    for (int base = s_w; base < e_w; base += 32) {
      const int nb = min(32, e_w - base);
      // Clamped indices keep every address valid, so the 32 loads issue back
      // to back; the values past the range or past d are masked afterwards.
      float ev[32];
#pragma unroll
      for (int j = 0; j < 32; ++j) {
        const int jj = j < nb ? j : nb - 1;
        const float v = load_elem<DT>(a.E, (row0 + (keys[base + jj] & pmask)) * a.lde + fs);
        ev[j] = (j < nb && fok) ? v : 0.f;
      }
#pragma unroll
      for (int j = 0; j < 32; ++j) {
        if (j >= nb) break;
        const int p = base + j;
        acc += ev[j];
        const bool run_end = p + 1 == T || (keys[p + 1] >> pb) != (keys[p] >> pb);
        if (run_end) {
          if (in_head) hp = acc; else sq += acc * acc;
          in_head = false;
          acc = 0.f;
        } else if (p + 1 == e_w) {  // the run stays open past this range
          t_open = true;
          if (in_head) { hp = acc; through = true; } else tp = acc;
        }
      }
    }
  }
  __shared__ float bh[NW][WAVE], bt[NW][WAVE];
  __shared__ int bflag[NW];
  bh[w][lane] = hp;
  bt[w][lane] = tp;
  if (lane == 0) bflag[w] = (h_open ? 1 : 0) | (t_open ? 2 : 0) | (through ? 4 : 0);
  __syncthreads();
  if (w == 0) {
    float carry = 0.f;
    for (int q = 0; q < NW; ++q) {
      const int fl = bflag[q];
      if (fl & 1) {
        carry += bh[q][lane];
        if (!(fl & 4)) { sq += carry * carry; carry = 0.f; }
      }
      if ((fl & 2) && !(fl & 4)) carry = bt[q][lane];
    }
  }
  sq = wave_sum(sq);
  if (lane == 0) red[w] = sq;
  __syncthreads();
  if (tid == 0) a.ws[(int64_t)b * a.n_chunks + chunk] = (red[0] + red[1]) + (red[2] + red[3]);
}

// ---------------------------------------------------------------------------
// Per-example bucketing and input-embedding norm on rows read 8 bytes per
// lane (EN_VB bytes: 4 bf16 or 2 fp32). Grid (B, S): workgroup s of example b
// owns the runs of equal ids that START at sorted positions
// [s*EN_P, (s+1)*EN_P) and walks each of them to its end, so no run is split
// between workgroups and each bucket's squared norm is formed whole. Every
// workgroup sorts the example's keys itself (T <= EN_CT_T: each key's rank is
// counted against all others; longer: the LDS radix sort), which costs less
// than a second launch. Lane q of the workgroup owns features
// [q*VEC, q*VEC + VEC) of every row (nq = d/VEC lanes per row, several
// passes when nq exceeds the workgroup); its loads of up to EN_BATCH
// positions are issued together.
// ---------------------------------------------------------------------------
template <int DT, int MAXT>
__global__ __launch_bounds__(EN_THREADS) void embed_norm_runs_kernel(EmbedNormArgs a) {
  constexpr int VEC = EN_VB / ((DT == DT_BF16) ? 2 : 4);  // elements per lane load
  constexpr int NW = EN_THREADS / WAVE;
  constexpr int LT = MAXT > 0 ? MAXT : 1;  // MAXT = 0: keys, ranks and runs from the workspace
  __shared__ __attribute__((aligned(16))) uint32_t kbuf[(MAXT > EN_CT_T) ? 2 : 1][LT];
  __shared__ int32_t rank_l[LT];
  __shared__ int32_t seg_l[LT + 1];
  __shared__ int cnt[(MAXT > EN_CT_T) ? NW * 256 : 1];
  __shared__ int wave_tot[NW];
  __shared__ float red[NW];
  const int b = blockIdx.x, s = blockIdx.y, tid = threadIdx.x;
  const int T = a.T, pb = a.pbits;
  const uint32_t pmask = (1u << pb) - 1u;
  const uint32_t V = (uint32_t)a.V;
  const int32_t* ids = a.ids + (int64_t)b * T;
  const uint32_t* keys;
  const int32_t* rank = rank_l;
  const int32_t* seg = seg_l;
  int nseg;
  if constexpr (MAXT == 0) {
    // sorted and ranked per example by the workspace radix sort
    keys = a.gkeys + (int64_t)b * T;
    rank = a.grank + (int64_t)b * T;
    seg = a.gseg + (int64_t)b * (T + 1);
    nseg = a.gnseg[b];
  } else if constexpr (MAXT <= EN_CT_T) {
    // Keys are distinct (the position is in the low bits), so a key's rank
    // is the number of smaller keys: T <= EN_THREADS, one key per thread.
    uint32_t k = 0xFFFFFFFFu;
    if (tid < T) {
      const uint32_t id = (uint32_t)ids[tid];
      k = ((id < V ? id : V) << pb) | (uint32_t)tid;
    }
    kbuf[0][tid] = k;  // past T: the largest key, counted by no real key
    __syncthreads();
    const int r = count_below(kbuf[0], (T + 7) & ~7, k);
    __syncthreads();
    if (tid < T) kbuf[0][r] = k;
    __syncthreads();
    keys = kbuf[0];
  } else {
    for (int p = tid; p < T; p += EN_THREADS) {
      const uint32_t id = (uint32_t)ids[p];
      kbuf[0][p] = ((id < V ? id : V) << pb) | (uint32_t)p;
    }
    __syncthreads();
    keys = kbuf[lds_radix_sort<NW>(kbuf[0], kbuf[1], T, pb, V, cnt, wave_tot)];
  }
  if constexpr (MAXT > 0) nseg = rank_sorted(keys, T, pb, rank_l, seg_l, wave_tot, tid, EN_THREADS);
  // Sorted positions [p_lo, p_hi) of this workgroup: bucket ids for them, and
  // the runs that start there.
  const int p_lo = min(s * EN_P, T), p_hi = min(p_lo + EN_P, T);
  if (a.seg_id)
    for (int p = p_lo + tid; p < p_hi; p += EN_THREADS)
      a.seg_id[(int64_t)b * T + (keys[p] & pmask)] = rank[p];
  if (a.n_unique && s == 0 && tid == 0) a.n_unique[b] = nseg;
  // First run start at or after position p (T if none).
  auto run_from = [&](int p) {
    if (p >= T) return T;
    const int r = rank[p];
    return seg[r] == p ? p : seg[r + 1];
  };
  const int q0 = run_from(p_lo), q1 = run_from(p_hi);
  const int nq = a.d / VEC;
  const int64_t row0 = (int64_t)b * T;
  const int esz = (DT == DT_BF16) ? 2 : 4;
  const uint32_t ldb = (uint32_t)(a.lde * esz);
  const rsrc_t rE = make_rsrc((const char*)a.E + row0 * ldb, (uint64_t)T * ldb);
  float sq = 0.f;
  const int lane = tid & 63;
  // Each wave walks the same sorted positions over its own feature lanes (no
  // barrier below). Per batch of EN_BATCH positions, lane j reads position
  // base + j's key and whether a run ends there; the row offsets then go to
  // the loads as wave-uniform offsets (readlane) and the run ends as a ballot
  // mask, so no load or step of the walk waits on an LDS read.
  static_assert(EN_BATCH <= WAVE, "one position per lane");
  for (int q0l = tid - lane; q0l < nq; q0l += EN_THREADS) {
    const int q = q0l + lane;
    const uint32_t coff = (uint32_t)(min(q, nq - 1) * EN_VB);  // lanes past the row repeat its last chunk
    float acc[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] = 0.f;
    for (int base = q0; base < q1; base += EN_BATCH) {
      const int nb = min(EN_BATCH, q1 - base);
      const int pj = base + min(lane, nb - 1);
      const uint32_t myrow = keys[pj] & pmask;
      const bool end_here = lane < nb && (pj + 1 == q1 || rank[pj + 1] != rank[pj]);
      const uint64_t ends = __ballot(end_here);
      uint32_t raw[EN_BATCH][2];
#pragma unroll
      for (int j = 0; j < EN_BATCH; ++j) {
        const uint32_t row = (uint32_t)__builtin_amdgcn_readlane((int)myrow, j);
        const auto v = __builtin_amdgcn_raw_buffer_load_b64(rE, coff, row * ldb, CPOL_STREAM);
        raw[j][0] = v[0];
        raw[j][1] = v[1];
      }
      // predicated, not exited early, so that raw[] stays in registers; the
      // repeated last position past nb is never added
#pragma unroll
      for (int j = 0; j < EN_BATCH; ++j) {
        if (j >= nb) continue;
        if constexpr (DT == DT_BF16) {
          acc[0] += __uint_as_float(raw[j][0] << 16);
          acc[1] += __uint_as_float(raw[j][0] & 0xFFFF0000u);
          acc[2] += __uint_as_float(raw[j][1] << 16);
          acc[3] += __uint_as_float(raw[j][1] & 0xFFFF0000u);
        } else {
          acc[0] += __uint_as_float(raw[j][0]);
          acc[1] += __uint_as_float(raw[j][1]);
        }
        // q1 is a run start, so the walk ends on a run's last position
        if ((ends >> j) & 1ull) {
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            sq += q < nq ? acc[e] * acc[e] : 0.f;
            acc[e] = 0.f;
          }
        }
      }
    }
  }
  sq = wave_sum(sq);
  if ((tid & 63) == 0) red[tid >> 6] = sq;
  __syncthreads();
  if (tid == 0) {
    float t = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) t += red[w];
    a.ws[(int64_t)b * a.n_chunks + s] = t;
  }
}

// Pairwise form of the same norm for short examples (bf16, 16-byte rows,
// T <= EN_G_T): sum_v ||sum_{t: x_t = v} dE_t||^2 = sum_{t,s} [x_t = x_s]
// <dE_t, dE_s>, the ghost-norm identity with one-hot inputs. Nothing waits on
// a sort: the ids and the rows load together, in position order.
// Workgroup (b, c) takes features [c' EN_GF, +EN_GF) of example b, with
// c' = c, or c - 1 when workgroup (b, 0) ranks the ids (dispatched first).
// Wave (i, g) of 8 (row block i of 32 rows, g = 0, 1): the g = 0 waves load
// rows 32i .. 32i+31 straight into MFMA operand fragments (lane l: row l % 32,
// features 16k + 8 (l / 32) .. +7 of step k; the A operand of E_i E_j^T and
// the B operand of E_j E_i^T have this same layout, so every product pairs
// equal features) and stage them in LDS; wave (i, g) multiplies block i with
// the column blocks j = g, g + 2, ...; the pairs (t, s) with equal ids are
// summed. Rows at or past T load as zeros (buffer bounds), features at or past
// d are zeroed.
// Workgroup (b, 0), when buckets are asked for: each token's bucket (the
// rank of its id among the example's distinct ids) from pairwise
// comparisons, and the number of buckets.
constexpr int EG_THREADS = 512;
constexpr int EG_NW = EG_THREADS / WAVE;
constexpr int EG_NB = EN_G_T / 32;        // row blocks
constexpr int EG_JG = EG_NW / EG_NB;      // waves per row block, each over every EG_JG-th column block
constexpr int EG_KS = EN_GF / 16;         // 16-feature steps per workgroup
constexpr int EG_LPT = EG_THREADS / EN_G_T;  // lanes per token when ranking ids
static_assert(EG_NB * EG_JG == EG_NW, "waves split evenly over the row blocks");
static_assert(EG_LPT == 4, "ranking: four lanes per token, quarters met by two shuffles");

__global__ __launch_bounds__(EG_THREADS) void embed_norm_gram_kernel(EmbedNormArgs a) {
  __shared__ u32x4 frag[EG_NB][EG_KS][WAVE];
  __shared__ __attribute__((aligned(16))) uint32_t uid[EN_G_T];
  __shared__ __attribute__((aligned(16))) uint32_t firsts[EN_G_T];
  __shared__ float red[EG_NW];
  __shared__ int cnt[EG_NW];
  const int b = blockIdx.x, c = blockIdx.y, tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int T = a.T;
  const uint32_t V = (uint32_t)a.V;
  const int32_t* ids = a.ids + (int64_t)b * T;
  // Ids clamped to V (one bucket for every id outside [0, V)); positions past
  // T get distinct values above any id, so they pair with nothing.
  const uint32_t u = tid < T ? min((uint32_t)ids[min(tid, T - 1)], V) : 0x80000000u + (uint32_t)tid;

  if (c == 0 && a.gram > 1) {
    // Four lanes per token (t = tid / 4), each comparing against a quarter
    // of the ids; the quarters meet through lane shuffles, which run on
    // every lane (a lane that skipped one would not supply its value).
    if (tid < EN_G_T) uid[tid] = u;
    __syncthreads();
    const int t = tid / EG_LPT, h = tid % EG_LPT;
    constexpr int Q4 = EN_G_T / EG_LPT / 4;  // u32x4 per quarter
    const uint32_t ut = uid[t];
    const u32x4* part_ids = (const u32x4*)uid + h * Q4;
    int dup = 0;  // an earlier position holds the same id
#pragma unroll
    for (int s4 = 0; s4 < Q4; ++s4) {
      const u32x4 v = part_ids[s4];
#pragma unroll
      for (int q = 0; q < 4; ++q) dup |= (h * 4 * Q4 + 4 * s4 + q < t && v[q] == ut) ? 1 : 0;
    }
    dup |= __shfl_xor(dup, 1);
    dup |= __shfl_xor(dup, 2);
    const bool first = dup == 0 && t < T;
    if (h == 0) firsts[t] = first ? 1u : 0u;
    const uint64_t m = __ballot(first && h == 0);
    if (lane == 0) cnt[w] = __popcll(m);
    __syncthreads();
    // bucket: the distinct ids below this one
    const u32x4* part_f = (const u32x4*)firsts + h * Q4;
    int r = 0;
#pragma unroll
    for (int s4 = 0; s4 < Q4; ++s4) {
      const u32x4 v = part_ids[s4], f = part_f[s4];
#pragma unroll
      for (int q = 0; q < 4; ++q) r += (f[q] != 0u && v[q] < ut) ? 1 : 0;
    }
    r += __shfl_xor(r, 1);
    r += __shfl_xor(r, 2);
    if (a.seg_id && h == 0 && t < T) a.seg_id[(int64_t)b * T + t] = r;
    if (a.n_unique && tid == 0) {
      int n = 0;
#pragma unroll
      for (int q = 0; q < EG_NW; ++q) n += cnt[q];
      a.n_unique[b] = n;
    }
    return;
  }
  const int chunk = c - (a.gram > 1 ? 1 : 0);

  const uint32_t ldb = (uint32_t)(a.lde * 2);
  const rsrc_t rE = make_rsrc((const char*)a.E + (int64_t)b * T * ldb, (uint64_t)T * ldb);
  const int nb = (T + 31) / 32;
  const int i = w % EG_NB, g = w / EG_NB;  // row block; column blocks g, g + EG_JG, ...
  u32x4 fa[EG_KS];
  if (g == 0 && i < nb) {
    const uint32_t row = (uint32_t)(32 * i + (lane & 31));
#pragma unroll
    for (int k = 0; k < EG_KS; ++k) {
      const int f = chunk * EN_GF + 16 * k + 8 * (lane >> 5);
      // a feature piece past d reads past the buffer's end, i.e. zeros
      const uint32_t off = f < a.d ? row * ldb + (uint32_t)f * 2 : 0x80000000u;
      fa[k] = buf_load16<CPOL_STREAM>(rE, off);
    }
  }
  if (tid < EN_G_T) uid[tid] = u;
  if (g == 0 && i < nb) {
#pragma unroll
    for (int k = 0; k < EG_KS; ++k) frag[i][k][lane] = fa[k];
  }
  __syncthreads();
  float part = 0.f;
  if (i < nb && g < nb) {
    if (g > 0) {
#pragma unroll
      for (int k = 0; k < EG_KS; ++k) fa[k] = frag[i][k][lane];
    }
    // rows t of this lane's accumulators e: 32 i + (e / 4) 8 + (l / 32) 4 + e % 4
    uint32_t ut[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) ut[e] = uid[32 * i + (e >> 2) * 8 + (lane >> 5) * 4 + (e & 3)];
    for (int j = g; j < nb; j += EG_JG) {
      f32x16 acc = {};
#pragma unroll
      for (int k = 0; k < EG_KS; ++k) acc = mfma32_bf16(fa[k], frag[j][k][lane], acc);
      const uint32_t us = uid[32 * j + (lane & 31)];
#pragma unroll
      for (int e = 0; e < 16; ++e) part += ut[e] == us ? acc[e] : 0.f;
    }
  }
  part = wave_sum(part);
  if (lane == 0) red[w] = part;
  __syncthreads();
  if (tid == 0) {
    float t = 0.f;
#pragma unroll
    for (int q = 0; q < EG_NW; ++q) t += red[q];
    a.ws[(int64_t)b * a.n_chunks + chunk] = t;
  }
}

// ---------------------------------------------------------------------------
// Batch-wide clipped sum of the input embedding:
// out[v, f] (+)= sum over tokens k with ids[k] = v of c[k / T] * E[k, f].
// ---------------------------------------------------------------------------
// Sorts all B*T keys (id << pbits | position) of the batch by id in one
// workgroup (lds_radix_sort); ids at or past V are clamped to V, so they
// sort last and every valid id stays one run.
constexpr int RS_WAVES = ES_THREADS / WAVE;

__global__ __launch_bounds__(ES_THREADS) void embed_sort_kernel(EmbedSumArgs a) {
  __shared__ uint32_t kbuf[2][ES_MAX_K];
  __shared__ int cnt[RS_WAVES * 256];
  __shared__ int wave_tot[ES_THREADS / WAVE];
  const int tid = threadIdx.x, K = a.K, pb = a.pbits;
  const uint32_t V = (uint32_t)a.V;
  for (int p = tid; p < K; p += ES_THREADS) {
    const uint32_t id = (uint32_t)a.ids[p];
    kbuf[0][p] = ((id < V ? id : V) << pb) | (uint32_t)p;
  }
  __syncthreads();
  const int r = lds_radix_sort<RS_WAVES>(kbuf[0], kbuf[1], K, pb, V, cnt, wave_tot);
  for (int p = tid; p < K; p += ES_THREADS) a.keys[p] = kbuf[r][p];
  if (a.rows) {
    // Compact form: ranks and run starts straight to the workspace.
    const int n = rank_sorted(kbuf[r], K, pb, a.rank, a.seg, wave_tot, tid, ES_THREADS);
    if (tid == 0) *a.n_runs = n;
  }
}

// ---------------------------------------------------------------------------
// Sort of more keys than one workgroup's LDS holds: a stable LSD radix sort
// through the workspace, 8 id bits per pass, in segments of gs_seg keys
// sorted independently (the whole batch for the embedding sum, one example
// each for the norm's buckets), GS_KB keys per block, gs_nbs blocks per
// segment. A pass counts each block's digits (hist: per segment, digit-major
// and block-minor), turns the counts into exclusive offsets in that order
// (one workgroup per segment), and scatters: each block sorts its keys by
// the digit in LDS (one stable LDS pass), then writes its j-th key of digit
// d to offset[d][block] + (j - first local index of d) within its segment.
// Blocks and keys within a block keep their order, so the pass is stable
// and the result is the (id, position) order of the single-workgroup sort.
// Pass 0 builds the keys from the ids; the position field of a key is the
// token's index within its segment.
// ---------------------------------------------------------------------------
constexpr int GS_THREADS = 1024;
constexpr int GS_NW = GS_THREADS / WAVE;

struct GsBlock {
  int64_t s0, p0;  // first key of the segment, of the block
  int n, seg, lb;  // keys in the block, segment, block within the segment
};
__device__ __forceinline__ GsBlock gs_block(const EmbedSumArgs& a) {
  GsBlock g;
  g.seg = (int)(blockIdx.x / (uint32_t)a.gs_nbs);
  g.lb = (int)(blockIdx.x - (uint32_t)g.seg * a.gs_nbs);
  g.s0 = (int64_t)g.seg * a.gs_seg;
  g.p0 = g.s0 + (int64_t)g.lb * GS_KB;
  g.n = (int)min((int64_t)GS_KB, g.s0 + a.gs_seg - g.p0);
  return g;
}

__device__ __forceinline__ uint32_t make_key(const EmbedSumArgs& a, const GsBlock& g, int i) {
  const uint32_t id = (uint32_t)a.ids[g.p0 + i];
  return ((id < (uint32_t)a.V ? id : (uint32_t)a.V) << a.pbits) | (uint32_t)(g.p0 + i - g.s0);
}

__global__ __launch_bounds__(GS_THREADS) void gsort_hist_kernel(EmbedSumArgs a, const uint32_t* src,
                                                                 int sh) {
  __shared__ int h[256];
  const GsBlock g = gs_block(a);
  const int tid = threadIdx.x;
  if (tid < 256) h[tid] = 0;
  __syncthreads();
  for (int i = tid; i < g.n; i += GS_THREADS) {
    const uint32_t key = src ? src[g.p0 + i] : make_key(a, g, i);
    atomicAdd(&h[(key >> sh) & 255], 1);  // integer counts: order-free
  }
  __syncthreads();
  if (tid < 256) a.hist[((int64_t)g.seg * 256 + tid) * a.gs_nbs + g.lb] = h[tid];
}

// Exclusive prefix sum, in place, of the n ints of segment blockIdx.x
// (v + blockIdx.x * n), one workgroup each; each thread scans a contiguous
// chunk. total[blockIdx.x] receives the sum when total is not NULL.
__global__ __launch_bounds__(GS_THREADS) void gscan_kernel(int* v, int n, int* total) {
  __shared__ int wave_tot[GS_NW];
  const int tid = threadIdx.x;
  v += (int64_t)blockIdx.x * n;
  const int per = (n + GS_THREADS - 1) / GS_THREADS;
  const int i0 = min(tid * per, n), i1 = min(i0 + per, n);
  int loc = 0;
  for (int i = i0; i < i1; ++i) loc += v[i];
  int tot;
  const int incl = block_inclusive_scan(loc, wave_tot, tid, GS_THREADS, &tot);
  int run = incl - loc;
  for (int i = i0; i < i1; ++i) {
    const int x = v[i];
    v[i] = run;
    run += x;
  }
  if (total && tid == 0) total[blockIdx.x] = tot;
}

__global__ __launch_bounds__(GS_THREADS) void gsort_scatter_kernel(EmbedSumArgs a,
                                                                   const uint32_t* src,
                                                                   uint32_t* dst, int sh) {
  __shared__ uint32_t kin[GS_KB], kout[GS_KB];
  __shared__ int cnt[GS_NW * 256];
  __shared__ int wave_tot[GS_NW];
  __shared__ int lstart[256];
  const GsBlock g = gs_block(a);
  const int tid = threadIdx.x;
  for (int i = tid; i < g.n; i += GS_THREADS) kin[i] = src ? src[g.p0 + i] : make_key(a, g, i);
  if (tid < 256) lstart[tid] = 0;
  __syncthreads();
  lds_radix_pass<GS_NW>(kin, kout, g.n, sh, cnt, wave_tot);
  // first local index of each digit: the count of smaller digits
  for (int i = tid; i < g.n; i += GS_THREADS) atomicAdd(&lstart[(kout[i] >> sh) & 255], 1);
  __syncthreads();
  {
    int c = tid < 256 ? lstart[tid] : 0, tot;
    const int incl = block_inclusive_scan(c, wave_tot, tid, GS_THREADS, &tot);
    __syncthreads();
    if (tid < 256) lstart[tid] = incl - c;
  }
  __syncthreads();
  const int* off = a.hist + (int64_t)g.seg * 256 * a.gs_nbs + g.lb;
  for (int j = tid; j < g.n; j += GS_THREADS) {
    const uint32_t key = kout[j];
    const int d = (int)((key >> sh) & 255);
    dst[g.s0 + off[(int64_t)d * a.gs_nbs] + (j - lstart[d])] = key;
  }
}

// Runs of equal ids in the sorted keys of each segment: heads per block,
// then (after an exclusive scan of each segment's block counts, which also
// gives its run count n_runs[segment]) every sorted position's run index
// within its segment and every run's first position (seg: gs_seg + 1
// entries per segment, the last one gs_seg).
__device__ __forceinline__ bool run_head(const EmbedSumArgs& a, const GsBlock& g, int64_t p) {
  return p == g.s0 || (a.keys[p] >> a.pbits) != (a.keys[p - 1] >> a.pbits);
}

__global__ __launch_bounds__(GS_THREADS) void gruns_count_kernel(EmbedSumArgs a) {
  __shared__ int wave_tot[GS_NW];
  const GsBlock g = gs_block(a);
  const int tid = threadIdx.x;
  int c = 0;
  for (int i = tid; i < g.n; i += GS_THREADS) c += run_head(a, g, g.p0 + i) ? 1 : 0;
  int tot;
  block_inclusive_scan(c, wave_tot, tid, GS_THREADS, &tot);
  if (tid == 0) a.gs_runs[blockIdx.x] = tot;
}

__global__ __launch_bounds__(GS_THREADS) void gruns_write_kernel(EmbedSumArgs a) {
  __shared__ int wave_tot[GS_NW];
  const GsBlock g = gs_block(a);
  const int tid = threadIdx.x;
  const int per = (g.n + GS_THREADS - 1) / GS_THREADS;
  const int i0 = min(tid * per, g.n), i1 = min(i0 + per, g.n);
  int c = 0;
  for (int i = i0; i < i1; ++i) c += run_head(a, g, g.p0 + i) ? 1 : 0;
  int tot;
  const int incl = block_inclusive_scan(c, wave_tot, tid, GS_THREADS, &tot);
  int32_t* seg = a.seg + (int64_t)g.seg * (a.gs_seg + 1);
  int r = a.gs_runs[blockIdx.x] + incl - c;  // runs that start before this thread's first key
  for (int i = i0; i < i1; ++i) {
    const int64_t p = g.p0 + i;
    if (run_head(a, g, p)) seg[r++] = (int32_t)(p - g.s0);
    a.rank[p] = r - 1;
  }
  if (g.lb == a.gs_nbs - 1 && tid == 0) seg[a.n_runs[g.seg]] = a.gs_seg;
}

// Sorted keys into a.keys (and, when `runs`, ranks, run starts and run
// counts) with the workspace radix sort over a.gs_blocks blocks.
static hipError_t launch_gsort(const EmbedSumArgs& a, bool runs, hipStream_t s) {
  int idbits = 0;
  while ((1u << idbits) <= (uint32_t)a.V) ++idbits;
  const int passes = (idbits + 7) / 8;
  const dim3 g(a.gs_blocks), blk(GS_THREADS);
  const int n_seg = a.gs_blocks / a.gs_nbs;
  for (int q = 0; q < passes; ++q) {
    // the last pass writes a.keys
    uint32_t* dst = ((passes - 1 - q) & 1) ? a.keys2 : a.keys;
    const uint32_t* src = q == 0 ? nullptr : (((passes - q) & 1) ? a.keys2 : a.keys);
    const int sh = a.pbits + 8 * q;
    hipLaunchKernelGGL(gsort_hist_kernel, g, blk, 0, s, a, src, sh);
    hipLaunchKernelGGL(gscan_kernel, dim3(n_seg), blk, 0, s, a.hist, 256 * a.gs_nbs,
                       (int*)nullptr);
    hipLaunchKernelGGL(gsort_scatter_kernel, g, blk, 0, s, a, src, dst, sh);
  }
  if (runs) {
    hipLaunchKernelGGL(gruns_count_kernel, g, blk, 0, s, a);
    hipLaunchKernelGGL(gscan_kernel, dim3(n_seg), blk, 0, s, a.gs_runs, a.gs_nbs, a.n_runs);
    hipLaunchKernelGGL(gruns_write_kernel, g, blk, 0, s, a);
  }
  return hipGetLastError();
}

__device__ __forceinline__ void out_add(const EmbedSumArgs& a, uint32_t v, int f, float val) {
  if (v >= (uint32_t)a.V) return;  // invalid id: contributes nothing
  float* o = a.transpose ? a.out + (int64_t)f * a.ldo + v : a.out + (int64_t)v * a.ldo + f;
  *o += val;
}

// A closed run's sum: added onto out[v], or (compact form) written to the
// run's row.
template <bool COMPACT>
__device__ __forceinline__ void run_out(const EmbedSumArgs& a, int rank, uint32_t v, int f,
                                        float val) {
  if constexpr (COMPACT)
    a.rows[(int64_t)rank * a.d + f] = val;
  else
    out_add(a, v, f, val);
}

// One wave per (block of ES_BLOCK sorted tokens, 64-feature chunk). Lanes
// 0..ES_BLOCK-1 first fetch the block's keys and the tokens' clip factors;
// then every lane (one feature) issues the loads of all ES_BLOCK rows back to
// back, and the runs of equal ids are closed in order with the keys broadcast
// from the lanes that hold them.
static_assert(ES_BLOCK <= WAVE, "one key per lane");
template <int DT, bool COMPACT>
__global__ __launch_bounds__(ES_WAVES * WAVE) void embed_block_kernel(EmbedSumArgs a) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n_fc = (a.d + WAVE - 1) / WAVE;
  const int n_blocks = (a.K + ES_BLOCK - 1) / ES_BLOCK;
  const int unit = blockIdx.x * ES_WAVES + w;
  if (unit >= n_blocks * n_fc) return;
  const int q = unit / n_fc, fc = unit - q * n_fc;
  const int f = fc * WAVE + lane;
  const bool fok = f < a.d;
  const int K = a.K, pb = a.pbits;
  const uint32_t pmask = (1u << pb) - 1u;
  const int p0 = q * ES_BLOCK, n = min(ES_BLOCK, K - p0);
  // Keys of this block (lane j < n holds key p0 + j) and their factors.
  const uint32_t mykey = lane < n ? a.keys[p0 + lane] : 0xFFFFFFFFu;
  const float myc = lane < n ? a.c[(int)((mykey & pmask) / (uint32_t)a.T)] : 0.f;
  const int myrank = (COMPACT && lane < n) ? a.rank[p0 + lane] : 0;
  const uint32_t id_before = p0 > 0 ? (a.keys[p0 - 1] >> pb) : 0xFFFFFFFFu;
  const uint32_t id_after = p0 + n < K ? (a.keys[p0 + n] >> pb) : 0xFFFFFFFFu;
  // Every load has a valid address (the last key repeats past the block, the
  // feature is clamped into the row), so all ES_BLOCK loads issue back to back.
  const uint32_t lastkey = (uint32_t)__builtin_amdgcn_readlane((int)mykey, n - 1);
  const int fs = fok ? f : a.d - 1;
  float ev[ES_BLOCK];
#pragma unroll
  for (int j = 0; j < ES_BLOCK; ++j) {
    const uint32_t kj = j < n ? (uint32_t)__builtin_amdgcn_readlane((int)mykey, j) : lastkey;
    const float cj = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, myc), j));
    const float v = load_elem<DT>(a.E, (int64_t)(kj & pmask) * a.lde + fs);
    // A token of an example with c = 0 (a non-finite norm) is left out.
    ev[j] = (j < n && fok && cj != 0.f) ? cj * v : 0.f;
  }
  float acc = 0.f;
  int run_start = 0;
#pragma unroll
  for (int j = 0; j < ES_BLOCK; ++j) {
    if (j >= n) break;
    const uint32_t id = (uint32_t)__builtin_amdgcn_readlane((int)mykey, j) >> pb;
    const uint32_t nid = j + 1 < n ? ((uint32_t)__builtin_amdgcn_readlane((int)mykey, j + 1) >> pb)
                                   : id_after;
    acc += ev[j];
    const bool last = (j + 1 == n) || (nid != id);
    if (last) {
      const bool open_head = run_start == 0 && id_before == id;
      const bool open_tail = j + 1 == n && id_after == id;
      if (fok) {
        if (open_head)
          a.head[(int64_t)q * a.d + f] = acc;
        else if (open_tail)
          a.tail[(int64_t)q * a.d + f] = acc;
        else
          run_out<COMPACT>(a, __builtin_amdgcn_readlane(myrank, j), id, f, acc);
      }
      acc = 0.f;
      run_start = j + 1;
    }
  }
}

// One wave per (block, feature chunk): closes the run that starts in block q
// and continues past it, adding the partials of the blocks it spans in order.
template <bool COMPACT>
__global__ __launch_bounds__(ES_WAVES * WAVE) void embed_fixup_kernel(EmbedSumArgs a) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n_fc = (a.d + WAVE - 1) / WAVE;
  const int n_blocks = (a.K + ES_BLOCK - 1) / ES_BLOCK;
  const int unit = blockIdx.x * ES_WAVES + w;
  if (unit >= n_blocks * n_fc) return;
  const int q = unit / n_fc, fc = unit - q * n_fc;
  const int f = fc * WAVE + lane;
  const int K = a.K, pb = a.pbits;
  const int p0 = q * ES_BLOCK, p1 = min(p0 + ES_BLOCK, K);
  if (p1 >= K) return;
  const uint32_t id = a.keys[p1 - 1] >> pb;
  if ((a.keys[p1] >> pb) != id) return;             // last run ends in this block
  if (p0 > 0 && (a.keys[p0 - 1] >> pb) == id) return;  // it started in an earlier block
  if (f >= a.d) return;
  float acc = a.tail[(int64_t)q * a.d + f];
  for (int qq = q + 1; qq < n_blocks; ++qq) {
    acc += a.head[(int64_t)qq * a.d + f];
    const int e = min(qq * ES_BLOCK + ES_BLOCK, K);
    if (e >= K || (a.keys[e] >> pb) != id) break;   // the run ends in block qq
  }
  run_out<COMPACT>(a, COMPACT ? a.rank[p1 - 1] : 0, id, f, acc);
}

// One thread per 4 consecutive features of one run's row: out[v] (+)= row.
__global__ __launch_bounds__(256) void embed_scatter_kernel(EmbedSumArgs a) {
  const int nq = (a.d + 3) / 4;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int r = (int)(i / nq);
  if (r >= a.K || r >= *a.n_runs) return;
  // The run list comes from the workspace; a position outside it (a
  // workspace dp_embedding_rows has not filled) adds nothing.
  const int p = a.seg[r];
  if (p < 0 || p >= a.K) return;
  const uint32_t v = a.keys[p] >> a.pbits;
  if (v >= (uint32_t)a.V) return;  // invalid ids: contribute nothing
  const int f0 = (int)(i - (int64_t)r * nq) * 4;
  const float* src = a.rows + (int64_t)r * a.d + f0;
  if (!a.transpose && f0 + 4 <= a.d && (a.d & 3) == 0 && (a.ldo & 3) == 0 &&
      (((uintptr_t)a.out) & 15) == 0) {
    f32x4* o = (f32x4*)(a.out + (int64_t)v * a.ldo + f0);
    *o += *(const f32x4*)src;
  } else {
    for (int k = 0; k < 4 && f0 + k < a.d; ++k) out_add(a, v, f0 + k, src[k]);
  }
}

__global__ void fill_zero_kernel(float* p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0.f;
}

hipError_t launch_embed_norm(const EmbedNormArgs& a, int dt, hipStream_t s) {
  if (a.B == 0) return hipSuccess;
  const dim3 g(a.B, a.n_chunks), blk(EN_THREADS);
  if (a.runs && a.T > EN_MAX_T) {
    // each example sorted and ranked through the workspace, then the walk
    EmbedSumArgs sa{};
    sa.ids = a.ids; sa.B = a.B; sa.T = a.T; sa.V = a.V; sa.pbits = a.pbits;
    sa.K = a.B * a.T;
    sa.keys = a.gkeys; sa.keys2 = a.gkeys2; sa.hist = a.ghist; sa.gs_runs = a.gruns;
    sa.rank = a.grank; sa.seg = a.gseg; sa.n_runs = a.gnseg;
    sa.gs_seg = a.T;
    sa.gs_nbs = (a.T + GS_KB - 1) / GS_KB;
    sa.gs_blocks = a.B * sa.gs_nbs;
    const hipError_t e = launch_gsort(sa, true, s);
    if (e != hipSuccess) return e;
    if (dt == DT_BF16) hipLaunchKernelGGL((embed_norm_runs_kernel<DT_BF16, 0>), g, blk, 0, s, a);
    else hipLaunchKernelGGL((embed_norm_runs_kernel<DT_F32, 0>), g, blk, 0, s, a);
    return hipGetLastError();
  }
  if (a.gram) {
    if (dt != DT_BF16 || a.T > EN_G_T) return hipErrorInvalidValue;
    EmbedNormArgs ga = a;
    ga.gram = (a.seg_id || a.n_unique) ? 2 : 1;  // 2: workgroup row 0 ranks the ids
    const dim3 gg(a.B, a.n_chunks + ga.gram - 1);
    hipLaunchKernelGGL(embed_norm_gram_kernel, gg, dim3(EG_THREADS), 0, s, ga);
    return hipGetLastError();
  }
  if (a.runs) {
    if (dt == DT_BF16) {
      if (a.T <= EN_CT_T) hipLaunchKernelGGL((embed_norm_runs_kernel<DT_BF16, EN_CT_T>), g, blk, 0, s, a);
      else hipLaunchKernelGGL((embed_norm_runs_kernel<DT_BF16, EN_MAX_T>), g, blk, 0, s, a);
    } else {
      if (a.T <= EN_CT_T) hipLaunchKernelGGL((embed_norm_runs_kernel<DT_F32, EN_CT_T>), g, blk, 0, s, a);
      else hipLaunchKernelGGL((embed_norm_runs_kernel<DT_F32, EN_MAX_T>), g, blk, 0, s, a);
    }
    return hipGetLastError();
  }
  if (dt == DT_BF16)
    hipLaunchKernelGGL(embed_norm_kernel<DT_BF16>, g, blk, 0, s, a);
  else
    hipLaunchKernelGGL(embed_norm_kernel<DT_F32>, g, blk, 0, s, a);
  return hipGetLastError();
}

// Sorted keys into a.keys (and, for the compact form, ranks, run starts and
// the run count): one workgroup up to ES_MAX_K keys, the radix sort through
// the workspace beyond.
static hipError_t launch_embed_keys(const EmbedSumArgs& a, bool compact, hipStream_t s) {
  if (a.K <= ES_MAX_K) {
    hipLaunchKernelGGL(embed_sort_kernel, dim3(1), dim3(ES_THREADS), 0, s, a);
    return hipGetLastError();
  }
  return launch_gsort(a, compact, s);
}

hipError_t launch_embed_sum(const EmbedSumArgs& a, int dt, hipStream_t s) {
  if (a.K == 0) return hipSuccess;
  hipError_t e = launch_embed_keys(a, false, s);
  if (e != hipSuccess) return e;
  const int n_fc = (a.d + WAVE - 1) / WAVE;
  const int n_blocks = (a.K + ES_BLOCK - 1) / ES_BLOCK;
  const int units = n_blocks * n_fc;
  const dim3 g((units + ES_WAVES - 1) / ES_WAVES), blk(ES_WAVES * WAVE);
  if (dt == DT_BF16)
    hipLaunchKernelGGL((embed_block_kernel<DT_BF16, false>), g, blk, 0, s, a);
  else
    hipLaunchKernelGGL((embed_block_kernel<DT_F32, false>), g, blk, 0, s, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(embed_fixup_kernel<false>, g, blk, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_embed_rows(const EmbedSumArgs& a, int dt, hipStream_t s) {
  if (a.K == 0) return hipSuccess;
  hipError_t e = launch_embed_keys(a, true, s);
  if (e != hipSuccess) return e;
  const int n_fc = (a.d + WAVE - 1) / WAVE;
  const int n_blocks = (a.K + ES_BLOCK - 1) / ES_BLOCK;
  const int units = n_blocks * n_fc;
  const dim3 g((units + ES_WAVES - 1) / ES_WAVES), blk(ES_WAVES * WAVE);
  if (dt == DT_BF16)
    hipLaunchKernelGGL((embed_block_kernel<DT_BF16, true>), g, blk, 0, s, a);
  else
    hipLaunchKernelGGL((embed_block_kernel<DT_F32, true>), g, blk, 0, s, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(embed_fixup_kernel<true>, g, blk, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_embed_scatter(const EmbedSumArgs& a, hipStream_t s) {
  if (a.K == 0) return hipSuccess;
  const int64_t n = (int64_t)a.K * ((a.d + 3) / 4);
  hipLaunchKernelGGL(embed_scatter_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  int64_t nb = (n + 255) / 256;
  if (nb > 65536) nb = 65536;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)nb), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

}  // namespace dpg
