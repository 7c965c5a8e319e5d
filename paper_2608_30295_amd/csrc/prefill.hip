// Prefill-time kernels of CateKV around the score passes (score.h):
// critical-token selection (Algorithm 1, pre-filling stage) -- row-statistics
// merge, BlockMax, top-k -- compaction (Cache(K, V, i_k, L_obs)) and the CV
// head score (Section 3.2, Eq. 1-4) over the observation matrix.
#include "score.h"

#include <algorithm>
#include <mutex>
#include <type_traits>

namespace catekv {

// Exact row statistics (max of s c over the visible columns, log2 units, and
// the sum of exp2(s c - max)) of one query row over one column block, by the
// 16 lanes of a row group; for the blocks whose sum overflowed fp32 in the
// score pass (a score over 2^128 times the offset that pass took from the
// block's first columns).  Plain fp32 dot products: this path is rare.
template <typename T>
__device__ float2 rowstats_exact(const ScoreArgs& a, int sel, int row, int b, int ln) {
  const int h = a.heads[sel];
  const int i = row / a.G, g = row - (row / a.G) * a.G;
  const T* q = reinterpret_cast<const T*>(a.q) + ((size_t)(h * a.G + g) * a.lq + i) * kD;
  const T* kh = reinterpret_cast<const T*>(a.k) + (size_t)h * a.n * kD;
  const int64_t c0 = (int64_t)b * a.cb_tokens, c1 = min(c0 + a.cb_tokens, a.n_keys);
  auto ld = [](const T* p, int d) -> float {
    if constexpr (sizeof(T) == 2) return __uint_as_float((uint32_t)p[d] << 16);
    else return p[d];
  };
  auto score = [&](int64_t col) -> float {   // s c, or -inf where the mask hides the key
    if (a.causal && a.key_off + col > a.q_pos0 + i) return -INFINITY;
    const T* kr = kh + (size_t)(a.key_off + col) * kD;
    float s = 0.f;
    for (int d = 0; d < kD; ++d) s = __builtin_fmaf(ld(q, d), ld(kr, d), s);
    return s * a.c;
  };
  float m = -INFINITY;
  for (int64_t col = c0 + ln; col < c1; col += 16) m = fmaxf(m, score(col));
  m = max16(m);
  if (m == -INFINITY) return make_float2(kMInit, 0.f);
  float l = 0.f;
  for (int64_t col = c0 + ln; col < c1; col += 16) l += fast_exp2(score(col) - m);
  return make_float2(m, sum16(l));
}

// Merge the per-column-block row statistics: offset = m c + log2(l), +inf
// for rows with no visible key and for padding rows.  16 lanes share a row
// and walk its column blocks with independent loads, then reduce over DPP.
// A block whose sum overflowed is recomputed exactly first.
constexpr int kMergeRows = 16;    // rows per 256-thread workgroup
template <typename T>
__global__ __launch_bounds__(256) void rowstats_merge_kernel(ScoreArgs a, int rpad, float* __restrict__ off) {
  const int sel = blockIdx.y;
  const int n_colblk = a.n_colblk, R = a.R;
  const int row = blockIdx.x * kMergeRows + (threadIdx.x >> 4);
  const int ln = threadIdx.x & 15;
  const bool ok = row < R;
  const float2* p = a.rowpart + (size_t)sel * n_colblk * rpad + (ok ? row : 0);
  float M = kMInit, L = 0.f;
  bool bad = false;
  constexpr int UNR = 8;
  for (int b0 = ln; b0 < n_colblk; b0 += 16 * UNR) {
    float2 v[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int b = b0 + 16 * u;
      v[u] = (ok && b < n_colblk) ? p[(size_t)b * rpad] : make_float2(kMInit, 0.f);
      if (!(v[u].y <= 0x1.fffffep127f)) {   // overflowed: merged below
        bad = true;
        v[u] = make_float2(kMInit, 0.f);
      }
    }
    float mb = M;
#pragma unroll
    for (int u = 0; u < UNR; ++u) mb = fmaxf(mb, v[u].x);
    L *= fast_exp2(M - mb);
#pragma unroll
    for (int u = 0; u < UNR; ++u) L += v[u].y * fast_exp2(v[u].x - mb);
    M = mb;
  }
  // any overflowed block of this row: the 16 lanes recompute each of them
  // together, and lane 0 merges the exact statistics
  const uint64_t any = __ballot(bad);
  if ((any >> (threadIdx.x & 48)) & 0xffffull) {
    for (int b = 0; b < n_colblk; ++b) {
      if (p[(size_t)b * rpad].y <= 0x1.fffffep127f) continue;   // the same for the row's 16 lanes
      const float2 e = rowstats_exact<T>(a, sel, row, b, ln);
      if (ln == 0 && e.y > 0.f) {
        const float mb = fmaxf(M, e.x);
        L = L * fast_exp2(M - mb) + e.y * fast_exp2(e.x - mb);
        M = mb;
      }
    }
  }
  const float M16 = max16(M);
  L = sum16(L * fast_exp2(M - M16));
  if (ln == 0 && row < rpad) off[(size_t)sel * rpad + row] = (ok && L > 0.f) ? M16 + __log2f(L) : INFINITY;
}

// ---------------------------------------------------------------------------
// selection: chunk maxima, radix top-k, compaction
// ---------------------------------------------------------------------------

__device__ __forceinline__ uint32_t ord_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// S_c = max of C over chunk c (BlockMax of Algorithm 1).
__global__ void chunk_max_kernel(const float* __restrict__ C, int64_t n_keys, int cs,
                                 int64_t n_chunks, float* __restrict__ S) {
  const int sel = blockIdx.y;
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= n_chunks) return;
  const float* Cs = C + (size_t)sel * n_keys;
  const int64_t e = min((c + 1) * (int64_t)cs, n_keys);
  float mx = -INFINITY;
  for (int64_t j = c * cs; j < e; ++j) mx = fmaxf(mx, Cs[j]);
  S[(size_t)sel * n_chunks + c] = mx;
}

constexpr int kTopkThreads = 1024;

__device__ int block_exclusive_scan(int v, int* s_buf, int* total) {
  // inclusive scan inside each wave (lane shuffles), then the 16 wave totals
  // from LDS: two barriers for the whole workgroup
  constexpr int NW = kTopkThreads / 64;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  int x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  if (lane == 63) s_buf[wave] = x;
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const int sw = s_buf[w];
    before += w < wave ? sw : 0;
    tot += sw;
  }
  *total = tot;
  __syncthreads();                 // s_buf is free for the next scan
  return before + x - v;
}

// Indices of the k largest chunk scores of one head (ties to the lower
// index), written ascending, then -1 padding up to b.
__global__ __launch_bounds__(kTopkThreads) void topk_kernel(const float* __restrict__ S, int64_t n_chunks,
                                                            int k, int b, int32_t* __restrict__ idx_out) {
  __shared__ int s_hist[256];
  __shared__ int s_scan[kTopkThreads];
  __shared__ uint32_t s_prefix;
  __shared__ int s_remaining;
  const int sel = blockIdx.x;
  const float* Ss = S + (size_t)sel * n_chunks;
  const int t = threadIdx.x;

  uint32_t prefix = 0, mask = 0;
  int remaining = k;   // rank (1-based, from the top) still to locate within the prefix
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    if (t < 256) s_hist[t] = 0;
    __syncthreads();
    for (int64_t i = t; i < n_chunks; i += kTopkThreads) {
      const uint32_t key = ord_key(Ss[i]);
      if ((key & mask) == prefix) atomicAdd(&s_hist[(key >> shift) & 255], 1);
    }
    __syncthreads();
    if (t == 0) {
      int cum = 0, bin = 0;
      for (bin = 255; bin > 0; --bin) {
        if (cum + s_hist[bin] >= remaining) break;
        cum += s_hist[bin];
      }
      s_prefix = prefix | ((uint32_t)bin << shift);
      s_remaining = remaining - cum;
    }
    __syncthreads();
    prefix = s_prefix;
    remaining = s_remaining;
    mask |= 255u << shift;
    __syncthreads();
  }
  const uint32_t tau = prefix;   // key of the k-th largest score
  // remaining = how many entries equal to tau are taken (lowest indices first)

  const int64_t per = (n_chunks + kTopkThreads - 1) / kTopkThreads;
  const int64_t lo = min((int64_t)t * per, n_chunks), hi = min(lo + per, n_chunks);
  int n_eq = 0;
  for (int64_t i = lo; i < hi; ++i) n_eq += ord_key(Ss[i]) == tau;
  int tot;
  int eq_before = block_exclusive_scan(n_eq, s_scan, &tot);
  int n_take = 0;
  {
    int eb = eq_before;
    for (int64_t i = lo; i < hi; ++i) {
      const uint32_t key = ord_key(Ss[i]);
      if (key > tau) ++n_take;
      else if (key == tau) { if (eb < remaining) ++n_take; ++eb; }
    }
  }
  int pos = block_exclusive_scan(n_take, s_scan, &tot);
  int32_t* out = idx_out + (size_t)sel * b;
  {
    int eb = eq_before;
    for (int64_t i = lo; i < hi; ++i) {
      const uint32_t key = ord_key(Ss[i]);
      bool take = false;
      if (key > tau) take = true;
      else if (key == tau) { take = eb < remaining; ++eb; }
      if (take && pos < k) out[pos++] = (int32_t)i;
    }
  }
  for (int i = k + t; i < b; i += kTopkThreads) out[i] = -1;
}


// Same selection with the scores held in registers.  Wave w owns the
// contiguous range [w * PER * 64, (w + 1) * PER * 64): its row i is the 64
// consecutive chunks from w * PER * 64 + 64 i, one per lane, so every load
// of the wave is one contiguous 256-byte read and ascending (row, lane) is
// ascending index.  Radix passes over 8-bit digits count into 16 LDS copies
// (lane & 15) of the histogram, double-buffered so the copy for the next
// pass is cleared during this one; wave 0 sums the copies and finds the bin
// of the target rank with a suffix scan, so a pass costs two barriers.  The
// positions of the selected entries come from per-row ballots and one
// exchange of the per-wave counts.
//
// Three uses (MODE): a whole row of scores; one slice of a row (rows are cut
// into PER * kTopkThreads-score slices whose own k best, in ascending order,
// go to a candidate list); a row's candidate list (scores looked up through
// the list, -1 entries never chosen, output mapped back through it).  The k
// best of a row are always among its slices' k best (an entry outranked by k
// entries of its own slice is outranked by k entries of the row; ties go to
// the lower index in both), and the candidate list is ascending, so the two
// stages reproduce the one-stage result.
enum TopkMode { kTopkRow = 0, kTopkSliceMode = 1, kTopkList = 2 };
constexpr int64_t kTopkSlice = 16 * kTopkThreads;   // scores per slice of long rows
constexpr int64_t kTopkSmallSlice = 4 * kTopkThreads;   // scores per slice of short rows

struct TopkArgs {
  const float* S;          // scores [rows][n]
  int64_t n;
  const int32_t* list;     // kTopkList: candidate indices [rows][list_len], -1 = none
  int64_t list_len;
  int k, b;                // select k; kTopkRow / kTopkList write b entries per row (-1 padded)
  int32_t* out;            // kTopkSliceMode: [rows][n_slices][k]; otherwise [rows][b]
};

template <int PER, int MODE>
__global__ __launch_bounds__(kTopkThreads) void topk_wave_kernel(TopkArgs a) {
  constexpr int NW = kTopkThreads / 64;
  constexpr int NCOPY = 16;
  constexpr int RS = 260;                  // words per copy: 256 bins, rows 16-byte aligned
  static_assert(PER <= 32, "validity is a 32-bit mask per lane");
  __shared__ __attribute__((aligned(16))) int s_h[2][NCOPY][RS];
  __shared__ uint32_t s_and[NW], s_or[NW];
  __shared__ int s_gt[NW], s_eq[NW];
  __shared__ uint32_t s_prefix;
  __shared__ int s_remaining;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int row = MODE == kTopkSliceMode ? blockIdx.y : blockIdx.x;
  const float* Ss = a.S + (size_t)row * a.n;
  int64_t start = 0, len = a.n;
  int k = a.k, b = a.b;
  int32_t* out = a.out + (size_t)row * a.b;
  const int32_t* lst = nullptr;
  if (MODE == kTopkSliceMode) {
    constexpr int64_t SL = (int64_t)PER * kTopkThreads;
    start = (int64_t)blockIdx.x * SL;
    len = min(SL, a.n - start);
    k = (int)min((int64_t)a.k, len);
    b = a.k;
    out = a.out + ((size_t)row * gridDim.x + blockIdx.x) * a.k;
  } else if (MODE == kTopkList) {
    len = a.list_len;
    lst = a.list + (size_t)row * a.list_len;
  }
  const int64_t base = (int64_t)wave * PER * 64 + lane;       // entry of row 0; row i adds 64 i
  uint32_t key[PER];
  uint32_t vmask = 0;                                          // bit i: row i holds an entry
  const int64_t rem = len - base;
  const int nv = rem <= 0 ? 0 : (int)min<int64_t>(PER, (rem + 63) / 64);
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    if (MODE == kTopkList) {
      const int32_t j = i < nv ? lst[base + 64 * i] : -1;
      key[i] = j >= 0 ? ord_key(Ss[j]) : 0u;
      vmask |= (j >= 0 ? 1u : 0u) << i;
    } else {
      key[i] = i < nv ? ord_key(Ss[start + base + 64 * i]) : 0u;
      vmask |= (i < nv ? 1u : 0u) << i;
    }
  }
  auto valid = [&](int i) { return (vmask >> i) & 1u; };

  // bits shared by every key: a digit made only of such bits puts all keys in
  // one bin, so its pass is skipped (chunk scores share sign and most exponent bits)
  uint32_t kand = 0xFFFFFFFFu, kor = 0u;
#pragma unroll
  for (int i = 0; i < PER; ++i)
    if (valid(i)) { kand &= key[i]; kor |= key[i]; }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    kand &= (uint32_t)__shfl_xor((int)kand, off);
    kor |= (uint32_t)__shfl_xor((int)kor, off);
  }
  if (lane == 0) { s_and[wave] = kand; s_or[wave] = kor; }
  for (int i = t; i < NCOPY * RS; i += kTopkThreads) (&s_h[0][0][0])[i] = 0;
  __syncthreads();
  kand = 0xFFFFFFFFu;
  kor = 0u;
#pragma unroll
  for (int w = 0; w < NW; ++w) { kand &= s_and[w]; kor |= s_or[w]; }
  const uint32_t varying = kand ^ kor;

  uint32_t prefix = 0, mask = 0;
  int remaining = k;       // rank (from the top) still to locate among keys matching the prefix
  int cur = 0;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    if (((varying >> shift) & 255u) == 0u) {      // the same digit everywhere (uniform branch)
      prefix |= kand & (255u << shift);
      mask |= 255u << shift;
      continue;
    }
    for (int i = t; i < NCOPY * RS; i += kTopkThreads) (&s_h[cur ^ 1][0][0])[i] = 0;
    const int cp = lane & (NCOPY - 1);
#pragma unroll
    for (int i = 0; i < PER; ++i)
      if (valid(i) && (key[i] & mask) == prefix) atomicAdd(&s_h[cur][cp][(key[i] >> shift) & 255u], 1);
    __syncthreads();
    if (wave == 0) {
      // lane l holds bins 4 l .. 4 l + 3; suffix sums over the lanes count the bins above
      int h0 = 0, h1 = 0, h2 = 0, h3 = 0;
#pragma unroll
      for (int c = 0; c < NCOPY; ++c) {
        const int4 v = *reinterpret_cast<const int4*>(&s_h[cur][c][4 * lane]);
        h0 += v.x; h1 += v.y; h2 += v.z; h3 += v.w;
      }
      const int c4 = h0 + h1 + h2 + h3;
      int incl = c4;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_down(incl, off);
        if (lane + off < 64) incl += y;
      }
      const int excl = incl - c4;
      if (excl < remaining && incl >= remaining) {
        const int h[4] = {h0, h1, h2, h3};
        int cum = excl, j = 3;
        for (; j > 0; --j) {
          if (cum + h[j] >= remaining) break;
          cum += h[j];
        }
        s_prefix = prefix | ((uint32_t)(4 * lane + j) << shift);
        s_remaining = remaining - cum;
      }
    }
    __syncthreads();
    prefix = s_prefix;
    remaining = s_remaining;
    mask |= 255u << shift;
    cur ^= 1;
  }
  const uint32_t tau = prefix;   // key of the k-th largest score
  // `remaining` entries equal to tau are taken, lowest indices first

  int n_gt = 0, n_eq = 0;
#pragma unroll
  for (int i = 0; i < PER; ++i)
    if (valid(i)) { n_gt += key[i] > tau; n_eq += key[i] == tau; }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    n_gt += __shfl_xor(n_gt, off);
    n_eq += __shfl_xor(n_eq, off);
  }
  if (lane == 0) { s_gt[wave] = n_gt; s_eq[wave] = n_eq; }
  __syncthreads();
  int pos = 0, eqr = 0;          // entries taken and ties seen in the waves before this one
  for (int w = 0; w < wave; ++w) {
    const int e = s_eq[w];
    pos += s_gt[w] + min(max(remaining - eqr, 0), e);
    eqr += e;
  }
  const uint64_t below = __lanemask_lt();
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const bool v = valid(i);
    const bool gt = v && key[i] > tau, eq = v && key[i] == tau;
    const uint64_t meq = __ballot(eq);
    const bool take = gt || (eq && eqr + __popcll(meq & below) < remaining);
    const uint64_t mt = __ballot(take);
    const int p = pos + __popcll(mt & below);
    if (take && p < k) {
      const int64_t e = base + 64 * i;
      out[p] = MODE == kTopkList ? lst[e] : (int32_t)(start + e);
    }
    pos += __popcll(mt);
    eqr += __popcll(meq);
  }
  for (int i = k + t; i < b; i += kTopkThreads) out[i] = -1;
}

struct CompactArgs {
  const void* k;
  const void* v;
  int64_t n;
  int cs, l_obs, b, b_eff;
  int64_t n_keys, n_chunks;
  const int32_t* idx;     // [n_sel][b]
  void* k_c;
  void* v_c;
  int64_t cap;            // rows per head in k_c / v_c
  int64_t* lens_out;
  int32_t heads[128];
};

// Cache(K, V, i_k, L_obs): rows of the selected chunks (ascending) then the
// last l_obs rows.  One thread moves one 16-byte segment of K and of V.
template <typename T>
__global__ void compact_kernel(CompactArgs a) {
  constexpr int SEG = kD * (int)sizeof(T) / 16;
  const int sel = blockIdx.y;
  const int h = a.heads[sel];
  const int32_t* ix = a.idx + (size_t)sel * a.b;
  const int64_t last = ix[a.b_eff - 1];
  const int64_t tail = a.n_keys - (a.n_chunks - 1) * a.cs;        // size of the last chunk
  const int64_t n_sel_tok = (int64_t)a.b_eff * a.cs - ((last == a.n_chunks - 1) ? (a.cs - tail) : 0);
  const int64_t len = n_sel_tok + a.l_obs;
  if (blockIdx.x == 0 && threadIdx.x == 0) a.lens_out[h] = len;
  const int64_t flat = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t row = flat / SEG;
  const int seg = (int)(flat - row * SEG);
  if (row >= len) return;
  int64_t src;
  if (row < n_sel_tok) {
    int64_t c = ix[row / a.cs];
    c = c < 0 ? 0 : (c >= a.n_chunks ? a.n_chunks - 1 : c);      // defensive clamp
    src = c * a.cs + row % a.cs;
    src = src < a.n_keys ? src : a.n_keys - 1;
  } else {
    src = a.n - a.l_obs + (row - n_sel_tok);
  }
  const size_t so = ((size_t)h * a.n + src) * kD * sizeof(T) + (size_t)seg * 16;
  const size_t dof = ((size_t)sel * a.cap + row) * kD * sizeof(T) + (size_t)seg * 16;
  *reinterpret_cast<uint4*>(reinterpret_cast<char*>(a.k_c) + dof) =
      ld16(reinterpret_cast<const char*>(a.k) + so);
  *reinterpret_cast<uint4*>(reinterpret_cast<char*>(a.v_c) + dof) =
      ld16(reinterpret_cast<const char*>(a.v) + so);
}

// ---------------------------------------------------------------------------
// CV: exact order statistics of the observation matrix, counts, score
// ---------------------------------------------------------------------------

struct CvState {                 // per KV head, in the workspace
  uint32_t prefix;               // radix prefix of the order statistic x_(lo)
  int64_t remaining;             // 0-based rank still to resolve inside the prefix (up to N - 1 >= 2^31)
  uint32_t min_above_key;        // smallest ordered key strictly above x_(lo)
  uint32_t need_scan;            // 1: min_above_key must come from a pass over A
  unsigned long long cnt_lt;     // entries strictly below x_(lo)
  double phi;
  unsigned long long sum_c, sum_c2;
  unsigned long long c0;         // entries in x_(lo)'s top-digit bin (known after the first pass)
  uint32_t n_cand;               // those entries, gathered by the second pass when they fit
};

constexpr int kRadixBins = 2048;   // digits: bits [31:21], [20:10] (11 bits), [9:0] (10 bits)

__device__ __forceinline__ int digit_shift(int pass) { return pass == 0 ? 21 : (pass == 1 ? 10 : 0); }
__device__ __forceinline__ uint32_t digit_mask_above(int pass) {
  return pass == 0 ? 0u : (pass == 1 ? 0xFFE00000u : 0xFFFFFC00u);
}
__device__ __forceinline__ float key_to_float(uint32_t key) {
  return __uint_as_float((key & 0x80000000u) ? (key & 0x7FFFFFFFu) : ~key);
}

__global__ void cv_init_kernel(CvState* st, uint32_t* hist, int64_t N, double k_pct, int hkv) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < 3 * hkv * kRadixBins; i += gridDim.x * blockDim.x)
    hist[i] = 0;
  if (blockIdx.x == 0 && threadIdx.x < hkv) {
    CvState& s = st[threadIdx.x];
    s.prefix = 0;
    s.remaining = (int64_t)floor((double)(N - 1) * k_pct);
    s.min_above_key = 0xFFFFFFFFu;
    s.need_scan = 0;
    s.cnt_lt = 0;
    s.phi = 0.0;
    s.sum_c = 0;
    s.sum_c2 = 0;
    s.c0 = 0;
    s.n_cand = 0;
  }
}

// Histogram of one radix digit over the entries whose higher digits match
// the prefix found so far.  hist: [hkv][kRadixBins] for this pass.  The
// probabilities of A crowd into a few digits, so each wave first counts the
// lanes that share its leading lane's digit with one ballot and one atomic;
// only the other lanes add one by one.  16-byte loads, 4 entries per lane.
__device__ __forceinline__ void hist_add_act(uint32_t* s_h, uint64_t act, bool valid, uint32_t bin) {
  const int lead = __builtin_ctzll(act);
  const uint32_t lb = (uint32_t)__builtin_amdgcn_readlane((int)bin, lead);
  const uint64_t same = __builtin_amdgcn_ballot_w64(valid && bin == lb);
  const int lane = threadIdx.x & 63;
  if (lane == lead) atomicAdd(&s_h[lb], (uint32_t)__builtin_popcountll(same));
  else if (valid && bin != lb) atomicAdd(&s_h[bin], 1u);
}
__device__ __forceinline__ void hist_add(uint32_t* s_h, bool valid, uint32_t bin) {
  const uint64_t act = __builtin_amdgcn_ballot_w64(valid);
  if (act) hist_add_act(s_h, act, valid, bin);
}

// The entries of x_(lo)'s top-digit bin (c0 of them, counted by the first
// pass) are all that the last two digits are resolved over.  When c0 fits the
// candidate buffer (cap keys per head), the second pass also gathers them, so
// the third pass and the search for the next key above x_(lo) read the
// candidates instead of A.  Gathering rides on the histogram's own ballot:
// a wave with no matching lane skips both.
constexpr int kGatherWave = 512;     // candidates a wave stages in LDS before writing them out

__global__ __launch_bounds__(256) void radix_hist_kernel(const float* __restrict__ A, int64_t N, int pass,
                                                         CvState* st, uint32_t* __restrict__ hist,
                                                         uint32_t* __restrict__ cand, uint32_t cap) {
  __shared__ uint32_t s_h[kRadixBins];
  __shared__ uint32_t s_buf[4][kGatherWave];
  __shared__ uint32_t s_wc[4];
  __shared__ uint32_t s_base;
  const int h = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const bool use_cand = st[h].c0 <= (unsigned long long)cap;   // uniform over the launch for head h
  const bool gather = pass == 1 && use_cand;
  for (int i = threadIdx.x; i < kRadixBins; i += blockDim.x) s_h[i] = 0;
  __syncthreads();
  const uint32_t pm = digit_mask_above(pass), pv = st[h].prefix & pm;
  const int shift = digit_shift(pass);
  const uint32_t dmask = pass == 2 ? 0x3FFu : 0x7FFu;
  uint32_t* ch = cand + (size_t)h * cap;
  // a wave-uniform count of the wave's candidates (from the ballots, no
  // atomics in the loop); a wave's stage holds kGatherWave, any beyond go
  // straight to the buffer
  uint32_t wcnt = 0;
  auto visit = [&](bool match, uint32_t key) {
    const uint64_t act = __builtin_amdgcn_ballot_w64(match);
    if (act == 0) return;
    hist_add_act(s_h, act, match, (key >> shift) & dmask);
    if (gather) {
      if (match) {
        const uint32_t off = wcnt + (uint32_t)__builtin_popcountll(act & __lanemask_lt());
        if (off < (uint32_t)kGatherWave) s_buf[wave][off] = key;
        else ch[atomicAdd(&st[h].n_cand, 1u)] = key;
      }
      wcnt += (uint32_t)__builtin_popcountll(act);
    }
  };
  if (pass == 2 && use_cand) {
    const int64_t nc = st[h].n_cand;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nc;
         i += (int64_t)gridDim.x * blockDim.x) {
      const uint32_t key = ch[i];
      hist_add(s_h, (key & pm) == pv, (key >> shift) & dmask);
    }
  } else {
    const float* Ah = A + (size_t)h * N;
    const int64_t n4 = (N & 3) == 0 && ((reinterpret_cast<uintptr_t>(Ah) & 15) == 0) ? N / 4 : 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4;
         i += (int64_t)gridDim.x * blockDim.x) {
      const float4 v = *reinterpret_cast<const float4*>(Ah + 4 * i);
      const float f[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t key = ord_key(f[e]);
        visit((key & pm) == pv, key);
      }
    }
    // entries not covered by the 16-byte loads (N not a multiple of 4, or an unaligned head)
    for (int64_t i = 4 * n4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < N;
         i += (int64_t)gridDim.x * blockDim.x) {
      const uint32_t key = ord_key(Ah[i]);
      visit((key & pm) == pv, key);
    }
  }
  if (gather && lane == 0) s_wc[wave] = min(wcnt, (uint32_t)kGatherWave);
  __syncthreads();
  for (int i = threadIdx.x; i < kRadixBins; i += blockDim.x)
    if (s_h[i]) atomicAdd(&hist[(size_t)h * kRadixBins + i], s_h[i]);
  if (gather) {
    if (threadIdx.x == 0) {
      const uint32_t tot = s_wc[0] + s_wc[1] + s_wc[2] + s_wc[3];
      s_base = tot ? atomicAdd(&st[h].n_cand, tot) : 0u;
    }
    __syncthreads();
    uint32_t dst = s_base;
    for (int w = 0; w < wave; ++w) dst += s_wc[w];
    for (uint32_t i = lane; i < s_wc[wave]; i += 64) ch[dst + i] = s_buf[wave][i];
  }
}

// Pick the digit that holds the target rank: one 256-thread workgroup per
// head, 8 bins per thread, a block scan of the per-thread sums.  The entries
// of lower digits are strictly below x_(lo) and are counted.  After the last
// pass the smallest key above x_(lo) is read off the same histogram when it
// lies in x_(lo)'s bucket; otherwise a pass over A is requested.
constexpr int kPickThreads = 256;
__global__ __launch_bounds__(kPickThreads) void radix_pick_kernel(const uint32_t* __restrict__ hist, int pass,
                                                                  CvState* st, int hkv) {
  constexpr int BPT = kRadixBins / kPickThreads;
  __shared__ int64_t s_tot[kPickThreads / 64];
  __shared__ int s_bin;
  __shared__ int64_t s_cum;
  __shared__ uint32_t s_bcnt;
  __shared__ int s_next;
  const int h = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const uint32_t* hh = hist + (size_t)h * kRadixBins;
  const int nb = pass == 2 ? 1024 : kRadixBins;
  const int64_t rem = st[h].remaining;
  uint32_t c[BPT];
  int64_t mine = 0;
#pragma unroll
  for (int i = 0; i < BPT; ++i) {
    const int bin = t * BPT + i;
    c[i] = bin < nb ? hh[bin] : 0u;
    mine += c[i];
  }
  // exclusive prefix of `mine` over the workgroup
  int64_t x = mine;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int64_t y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  if (lane == 63) s_tot[wave] = x;
  if (t == 0) { s_bin = -1; s_next = 0x7FFFFFFF; }
  __syncthreads();
  int64_t before = x - mine;
#pragma unroll
  for (int w = 0; w < kPickThreads / 64; ++w) before += w < wave ? s_tot[w] : 0;
  if (before <= rem && rem < before + mine) {
    int64_t cum = before;
    int i = 0;
    for (i = 0; i < BPT - 1; ++i) {
      if (cum + c[i] > rem) break;
      cum += c[i];
    }
    s_bin = t * BPT + i;
    s_cum = cum;
    s_bcnt = c[i];
  }
  __syncthreads();
  if (s_bin < 0) {            // rank beyond the counts (not reached with consistent counts): last bin
    if (t == 0) {
      int64_t cum = 0;
      for (int b = 0; b < nb - 1; ++b) cum += hh[b];
      s_bin = nb - 1;
      s_cum = cum;
      s_bcnt = hh[nb - 1];
    }
    __syncthreads();
  }
  const int bin = s_bin;
  if (pass == 2) {
    // first non-empty bin above the chosen one, within x_(lo)'s 22-bit bucket
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
      const int b = t * BPT + i;
      if (b > bin && b < nb && c[i] != 0u) atomicMin(&s_next, b);
    }
  }
  __syncthreads();
  if (t == 0) {
    const uint32_t prefix = st[h].prefix | ((uint32_t)bin << digit_shift(pass));
    st[h].prefix = prefix;
    st[h].remaining = rem - s_cum;
    st[h].cnt_lt += (unsigned long long)s_cum;
    if (pass == 0) st[h].c0 = s_bcnt;
    if (pass == 2) {
      if (s_next != 0x7FFFFFFF) st[h].min_above_key = (prefix & ~0x3FFu) | (uint32_t)s_next;
      else st[h].need_scan = 1;
    }
  }
}

// Smallest ordered key strictly above x_(lo) (needed when x_(lo + 1) differs).
// from_cand: over the gathered candidates (x_(lo)'s top-digit bin), when they
// were gathered; otherwise, and when no candidate lies above x_(lo) (then the
// key sits in a higher top-digit bin), over A.
__global__ __launch_bounds__(256) void radix_min_above_kernel(const float* __restrict__ A, int64_t N, CvState* st,
                                                              const uint32_t* __restrict__ cand, uint32_t cap,
                                                              int from_cand) {
  __shared__ uint32_t s_min;
  const int h = blockIdx.y;
  if (!st[h].need_scan) return;       // found in the last radix histogram
  const bool use_cand = st[h].c0 <= (unsigned long long)cap;
  if (from_cand ? !use_cand : (use_cand && st[h].min_above_key != 0xFFFFFFFFu)) return;
  if (threadIdx.x == 0) s_min = 0xFFFFFFFFu;
  __syncthreads();
  const uint32_t x = st[h].prefix;
  uint32_t mn = 0xFFFFFFFFu;
  if (from_cand) {
    const uint32_t* ch = cand + (size_t)h * cap;
    const int64_t nc = st[h].n_cand;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nc; i += (int64_t)gridDim.x * blockDim.x) {
      const uint32_t key = ch[i];
      if (key > x) mn = min(mn, key);
    }
  } else {
    const float* Ah = A + (size_t)h * N;
    const int64_t n4 = (N & 3) == 0 && ((reinterpret_cast<uintptr_t>(Ah) & 15) == 0) ? N / 4 : 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (int64_t)gridDim.x * blockDim.x) {
      const float4 v = *reinterpret_cast<const float4*>(Ah + 4 * i);
      const uint32_t k4[4] = {ord_key(v.x), ord_key(v.y), ord_key(v.z), ord_key(v.w)};
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (k4[e] > x) mn = min(mn, k4[e]);
    }
    for (int64_t i = 4 * n4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < N;
         i += (int64_t)gridDim.x * blockDim.x) {
      const uint32_t key = ord_key(Ah[i]);
      if (key > x) mn = min(mn, key);
    }
  }
  atomicMin(&s_min, mn);
  __syncthreads();
  if (threadIdx.x == 0 && s_min != 0xFFFFFFFFu) atomicMin(&st[h].min_above_key, s_min);
}

// Phi = alpha * (x_(lo) + frac * (x_(lo+1) - x_(lo))) in fp64 (Eq. 2).
__global__ void cv_threshold_kernel(CvState* st, const uint32_t* __restrict__ hist_last, int64_t N,
                                    double k_pct, double alpha, int hkv) {
  const int h = blockIdx.x * blockDim.x + threadIdx.x;
  if (h >= hkv) return;
  const double pos = (double)(N - 1) * k_pct;
  const int64_t lo = (int64_t)floor(pos);
  const double frac = pos - (double)lo;
  const uint32_t xk = st[h].prefix;
  const unsigned long long eq = hist_last[(size_t)h * kRadixBins + (xk & 0x3FFu)];
  const unsigned long long le = st[h].cnt_lt + eq;        // entries <= x_(lo)
  const double xlo = (double)key_to_float(xk);
  double xhi = xlo;
  if ((int64_t)le < lo + 2 && lo + 1 <= N - 1) xhi = (double)key_to_float(st[h].min_above_key);
  st[h].phi = alpha * (xlo + frac * (xhi - xlo));
}

// C_j = #{i : A[i][j] >= Phi} (Eq. 2-3); exact integer sums of C and C^2.
// A workgroup takes 64 adjacent columns at a time (one per lane, so every
// row read is 256 contiguous bytes, whatever the row stride) and its four
// waves split the rows, each with up to kCountRows loads in flight per lane;
// the four partial counts of a column meet in LDS before C_j is squared.
// The comparison stays in fp64 against Phi.
constexpr int kCountRows = 16;
__global__ __launch_bounds__(256) void cv_count_kernel(const float* __restrict__ A, int lq, int64_t n_keys,
                                                        CvState* st) {
  __shared__ unsigned int s_c[4][64];
  __shared__ unsigned long long s1, s2;
  const int h = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;   // wave = row group
  if (threadIdx.x == 0) { s1 = 0; s2 = 0; }
  __syncthreads();
  const double phi = st[h].phi;
  const float* Ah = A + (size_t)h * lq * n_keys;
  const int rpg = (lq + 3) / 4;
  const int r0 = wave * rpg, r1 = min(lq, r0 + rpg);
  unsigned long long a1 = 0, a2 = 0;
  for (int64_t j0 = (int64_t)blockIdx.x * 64; j0 < n_keys; j0 += (int64_t)gridDim.x * 64) {
    const int64_t j = j0 + lane;
    unsigned int c = 0;
    if (j < n_keys) {
      for (int i0 = r0; i0 < r1; i0 += kCountRows) {
        float v[kCountRows];
#pragma unroll
        for (int u = 0; u < kCountRows; ++u)
          if (i0 + u < r1) v[u] = Ah[(size_t)(i0 + u) * n_keys + j];
#pragma unroll
        for (int u = 0; u < kCountRows; ++u)
          if (i0 + u < r1) c += (double)v[u] >= phi;
      }
    }
    s_c[wave][lane] = c;
    __syncthreads();
    if (wave == 0 && j < n_keys) {
      const unsigned int cj = s_c[0][lane] + s_c[1][lane] + s_c[2][lane] + s_c[3][lane];
      a1 += cj;
      a2 += (unsigned long long)cj * cj;
    }
    __syncthreads();
  }
  if (wave == 0) {              // only wave 0 holds sums
    atomicAdd(&s1, a1);
    atomicAdd(&s2, a2);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    atomicAdd(&st[h].sum_c, s1);
    atomicAdd(&st[h].sum_c2, s2);
  }
}

// Eq. 4: population standard deviation over the mean, from exact integers.
__global__ void cv_final_kernel(const CvState* __restrict__ st, int64_t n_keys, float* cv_out, int hkv) {
  const int h = blockIdx.x * blockDim.x + threadIdx.x;
  if (h >= hkv) return;
  const double N = (double)n_keys;
  const double mu = (double)st[h].sum_c / N;
  if (mu == 0.0) { cv_out[h] = 0.f; return; }
  double var = (double)st[h].sum_c2 / N - mu * mu;
  var = var < 0.0 ? 0.0 : var;
  cv_out[h] = (float)(sqrt(var) / mu);
}

// ---------------------------------------------------------------------------
// host-side launchers
// ---------------------------------------------------------------------------

static inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
// Score workgroups run in a single round: as many as the device holds at once
// (the bf16 residency: two workgroups per compute unit, whose LDS rings fill
// 128 KB of its 160 KB, or one 16-wave workgroup at 512 rows; fp32 beyond 128
// rows runs in two rounds), each over whole 64-column tiles, at least four
// and at most kMaxBlockTokens columns (more rounds beyond).  The count
// depends on the rows but not on the dtype, so workspace sizes do not either.
int64_t score_block_tokens(int64_t n_keys, int n_heads, int rows_pad, int n_cu) {
  const int64_t slots = (int64_t)std::max(1, n_cu) * (score_waves(CATEKV_BF16, rows_pad) > 8 ? 1 : 2);
  const int64_t per_head = std::max<int64_t>(1, slots / std::max(1, n_heads));
  int64_t cb = (std::max<int64_t>(n_keys, 1) + per_head - 1) / per_head;
  cb = (cb + kTileTok - 1) / kTileTok * kTileTok;
  return std::min<int64_t>(std::max<int64_t>(cb, 4 * kTileTok), kMaxBlockTokens);
}

struct SelectLayout {
  size_t rowpart, rowoff, colmass, chunks, topk, total;
};
static SelectLayout select_layout(const SelectGeom& g) {
  SelectLayout L{};
  const int rp = score_rows_pad(g.G * g.l_obs);
  size_t o = 0;
  L.rowpart = o; o += align256((size_t)g.n_sel * g.n_colblk * rp * sizeof(float2));
  L.rowoff = o; o += align256((size_t)g.n_sel * rp * sizeof(float));
  // per-key column mass only when BlockMax cannot be fused into the score pass
  // (cs not dividing the 64-column tile)
  L.colmass = o; o += kTileTok % g.cs == 0 ? 0 : align256((size_t)g.n_sel * g.n_keys * sizeof(float));
  L.chunks = o; o += align256((size_t)g.n_sel * g.n_chunks * sizeof(float));
  L.topk = o; o += align256(topk_workspace_bytes(g.n_sel, g.n_chunks));
  L.total = o;
  return L;
}

size_t select_workspace_bytes(const SelectGeom& g) { return select_layout(g).total; }

// Scratch of catekv_select_critical_noalloc: a file-scope device array, so
// the call allocates nothing.  Every GPU the library runs on holds its own
// copy, at its own address, until the process ends.  In host code the
// array's name is only a host-side stand-in: its device address comes from
// hipGetSymbolAddress, taken once per device with that device current, and
// only that address is handed to kernels.
constexpr size_t kSelectScratchBytes = (size_t)16 << 20;
static __device__ __align__(256) unsigned char scratch[kSelectScratchBytes];

size_t select_scratch_bytes() { return kSelectScratchBytes; }

hipError_t select_scratch(void** ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

hipError_t launch_select(int dtype, const SelectGeom& g, const void* q_obs, const void* k,
                         int32_t* idx_out, void* ws, hipStream_t stream) {
  const SelectLayout L = select_layout(g);
  char* w = reinterpret_cast<char*>(ws);
  const int R = g.G * g.l_obs;
  const int rp = score_rows_pad(R);
  ScoreArgs a{};
  a.q = q_obs; a.k = k; a.hkv = g.hkv; a.lq = g.l_obs; a.G = g.G; a.R = R; a.n = g.n;
  a.key_off = 0; a.n_keys = g.n_keys; a.cb_tokens = g.cb_tokens; a.n_colblk = g.n_colblk;
  a.q_pos0 = g.n - g.l_obs; a.causal = 0; a.c = kLog2e / sqrtf((float)kD);
  for (int i = 0; i < g.n_sel; ++i) a.heads[i] = g.heads[i];
  a.rowpart = reinterpret_cast<float2*>(w + L.rowpart);
  a.rowoff = reinterpret_cast<const float*>(w + L.rowoff);
  a.colmass = reinterpret_cast<float*>(w + L.colmass);
  const dim3 grid(g.n_colblk, g.n_sel);
  hipError_t e = launch_score_rowstats(dtype, g.G, false, rp, grid, stream, a);
  if (e != hipSuccess) return e;
  if (dtype == CATEKV_BF16)
    hipLaunchKernelGGL(rowstats_merge_kernel<uint16_t>, dim3((rp + kMergeRows - 1) / kMergeRows, g.n_sel), dim3(256), 0,
                       stream, a, rp, reinterpret_cast<float*>(w + L.rowoff));
  else
    hipLaunchKernelGGL(rowstats_merge_kernel<float>, dim3((rp + kMergeRows - 1) / kMergeRows, g.n_sel), dim3(256), 0,
                       stream, a, rp, reinterpret_cast<float*>(w + L.rowoff));
  float* S = reinterpret_cast<float*>(w + L.chunks);
  a.chunks = S;
  a.n_chunks = g.n_chunks;
  a.cs_fused = (kTileTok % g.cs == 0) ? g.cs : 0;
  e = launch_score_colmass(dtype, rp, grid, stream, a);
  if (e != hipSuccess) return e;
  if (!a.cs_fused)
    hipLaunchKernelGGL(chunk_max_kernel, dim3((unsigned)((g.n_chunks + 255) / 256), g.n_sel), dim3(256), 0,
                       stream, a.colmass, g.n_keys, g.cs, g.n_chunks, S);
  return launch_topk(S, g.n_sel, g.n_chunks, g.b, idx_out, w + L.topk, stream);
}

size_t topk_workspace_bytes(int n_rows, int64_t n) {
  return n > kTopkSmallSlice ? (size_t)n_rows * 2 * kTopkSlice * sizeof(int32_t) : 0;
}

// k best of each row's candidate list (ascending indices into the row)
static void launch_topk_list(const TopkArgs& a, int n_rows, hipStream_t stream) {
  const int64_t m = a.list_len;
  if (m <= 1 * kTopkThreads)
    hipLaunchKernelGGL((topk_wave_kernel<1, kTopkList>), dim3(n_rows), dim3(kTopkThreads), 0, stream, a);
  else if (m <= 2 * kTopkThreads)
    hipLaunchKernelGGL((topk_wave_kernel<2, kTopkList>), dim3(n_rows), dim3(kTopkThreads), 0, stream, a);
  else if (m <= 4 * kTopkThreads)
    hipLaunchKernelGGL((topk_wave_kernel<4, kTopkList>), dim3(n_rows), dim3(kTopkThreads), 0, stream, a);
  else if (m <= 8 * kTopkThreads)
    hipLaunchKernelGGL((topk_wave_kernel<8, kTopkList>), dim3(n_rows), dim3(kTopkThreads), 0, stream, a);
  else if (m <= 16 * kTopkThreads)
    hipLaunchKernelGGL((topk_wave_kernel<16, kTopkList>), dim3(n_rows), dim3(kTopkThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((topk_wave_kernel<32, kTopkList>), dim3(n_rows), dim3(kTopkThreads), 0, stream, a);
}

hipError_t launch_topk(const float* S, int n_rows, int64_t n, int b, int32_t* idx_out, void* ws,
                       hipStream_t stream) {
  const int k_eff = (int)(b < n ? b : n);
  TopkArgs a{};
  a.S = S; a.n = n; a.k = k_eff; a.b = b; a.out = idx_out;
  const int64_t n_slices = (n + kTopkSlice - 1) / kTopkSlice;
  const int64_t n_small = (n + kTopkSmallSlice - 1) / kTopkSmallSlice;
  // A row of up to 2 kTopkSlice scores fits one workgroup, but a few such rows
  // leave most compute units idle: there 4096-score slices run side by side
  // and a second launch picks among their k best.  Measured: k = 256 of 16384
  // gains ~1.7 us on three rows, k = 1024 loses ~2.7 us, so k is held to at
  // most an eighth of a slice.
  const bool few_short_rows = ws && n > kTopkSmallSlice && n <= 2 * kTopkSlice &&
                              8 * k_eff <= kTopkSmallSlice && (int64_t)n_rows * n_small <= 2048;
  if (few_short_rows) {
    TopkArgs s1 = a;
    s1.out = reinterpret_cast<int32_t*>(ws);
    hipLaunchKernelGGL((topk_wave_kernel<4, kTopkSliceMode>), dim3((unsigned)n_small, n_rows),
                       dim3(kTopkThreads), 0, stream, s1);
    TopkArgs s2 = a;
    s2.list = s1.out;
    s2.list_len = n_small * k_eff;
    launch_topk_list(s2, n_rows, stream);
  } else if (n <= kTopkSlice) {
    hipLaunchKernelGGL((topk_wave_kernel<16, kTopkRow>), dim3(n_rows), dim3(kTopkThreads), 0, stream, a);
  } else if (n <= 2 * kTopkSlice) {
    hipLaunchKernelGGL((topk_wave_kernel<32, kTopkRow>), dim3(n_rows), dim3(kTopkThreads), 0, stream, a);
  } else if (ws && n_slices * k_eff <= 2 * kTopkSlice) {
    // the k best of every slice, then the k best of those candidates
    int32_t* cand = reinterpret_cast<int32_t*>(ws);
    TopkArgs s1 = a;
    s1.out = cand;
    hipLaunchKernelGGL((topk_wave_kernel<16, kTopkSliceMode>), dim3((unsigned)n_slices, n_rows),
                       dim3(kTopkThreads), 0, stream, s1);
    TopkArgs s2 = a;
    s2.list = cand;
    s2.list_len = n_slices * k_eff;
    launch_topk_list(s2, n_rows, stream);
  } else {
    hipLaunchKernelGGL(topk_kernel, dim3(n_rows), dim3(kTopkThreads), 0, stream, S, n, k_eff, b, idx_out);
  }
  return hipGetLastError();
}

hipError_t launch_compact(int dtype, const void* k, const void* v, int hkv, int64_t n, int cs,
                          int l_obs, const int32_t* heads, int n_sel, const int32_t* idx, int b,
                          void* k_c, void* v_c, int64_t* lens_out, hipStream_t stream) {
  (void)hkv;
  CompactArgs a{};
  a.k = k; a.v = v; a.n = n; a.cs = cs; a.l_obs = l_obs; a.b = b;
  a.n_keys = n - l_obs;
  a.n_chunks = (a.n_keys + cs - 1) / cs;
  a.b_eff = (int)(b < a.n_chunks ? b : a.n_chunks);
  a.idx = idx; a.k_c = k_c; a.v_c = v_c;
  a.cap = (int64_t)b * cs + l_obs;
  a.lens_out = lens_out;
  for (int i = 0; i < n_sel; ++i) a.heads[i] = heads[i];
  const int64_t seg = dtype == CATEKV_BF16 ? 16 : 32;
  const int64_t rows = (int64_t)a.b_eff * cs + l_obs;
  const unsigned nblk = (unsigned)((rows * seg + 255) / 256);
  if (dtype == CATEKV_BF16)
    hipLaunchKernelGGL(compact_kernel<uint16_t>, dim3(nblk, n_sel), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(compact_kernel<float>, dim3(nblk, n_sel), dim3(256), 0, stream, a);
  return hipGetLastError();
}

struct ScoreLayout {
  size_t rowpart, rowoff, obs, hist, cand, state, total;
};
// Candidate keys per head: an eighth of the observation matrix (the top-digit
// bin of a high quantile holds far fewer; larger bins take the path over A).
static uint32_t cand_cap(const ScoreGeom& g) {
  const int64_t N = (int64_t)g.lq * g.n_keys;
  return (uint32_t)std::max<int64_t>(4096, (N + 7) / 8);
}
static ScoreLayout score_layout(const ScoreGeom& g) {
  ScoreLayout L{};
  const int rp = score_rows_pad(g.G * g.lq);
  size_t o = 0;
  L.rowpart = o; o += align256((size_t)g.hkv * g.n_colblk * rp * sizeof(float2));
  L.rowoff = o; o += align256((size_t)g.hkv * rp * sizeof(float));
  L.obs = o; o += align256((size_t)g.hkv * g.lq * g.n_keys * sizeof(float));
  L.hist = o; o += align256((size_t)3 * g.hkv * kRadixBins * sizeof(uint32_t));
  L.cand = o; o += align256((size_t)g.hkv * cand_cap(g) * sizeof(uint32_t));
  L.state = o; o += align256((size_t)g.hkv * sizeof(CvState));
  L.total = o;
  return L;
}

size_t score_workspace_bytes(const ScoreGeom& g) { return score_layout(g).total; }

hipError_t launch_score(int dtype, const ScoreGeom& g, const void* q_rows, const void* k,
                        float* cv_out, void* ws, hipStream_t stream) {
  const ScoreLayout L = score_layout(g);
  char* w = reinterpret_cast<char*>(ws);
  const int R = g.G * g.lq;
  const int rp = score_rows_pad(R);
  ScoreArgs a{};
  a.q = q_rows; a.k = k; a.hkv = g.hkv; a.lq = g.lq; a.G = g.G; a.R = R; a.n = g.n;
  a.key_off = g.l_init; a.n_keys = g.n_keys; a.cb_tokens = g.cb_tokens; a.n_colblk = g.n_colblk;
  a.q_pos0 = g.q_pos0; a.causal = g.causal; a.c = kLog2e / sqrtf((float)kD);
  for (int i = 0; i < g.hkv; ++i) a.heads[i] = i;
  a.rowpart = reinterpret_cast<float2*>(w + L.rowpart);
  a.rowoff = reinterpret_cast<const float*>(w + L.rowoff);
  a.obs = reinterpret_cast<float*>(w + L.obs);
  const dim3 grid(g.n_colblk, g.hkv);
  hipError_t e = launch_score_rowstats(dtype, g.G, g.causal, rp, grid, stream, a);
  if (e != hipSuccess) return e;
  if (dtype == CATEKV_BF16)
    hipLaunchKernelGGL(rowstats_merge_kernel<uint16_t>, dim3((rp + kMergeRows - 1) / kMergeRows, g.hkv), dim3(256), 0,
                       stream, a, rp, reinterpret_cast<float*>(w + L.rowoff));
  else
    hipLaunchKernelGGL(rowstats_merge_kernel<float>, dim3((rp + kMergeRows - 1) / kMergeRows, g.hkv), dim3(256), 0,
                       stream, a, rp, reinterpret_cast<float*>(w + L.rowoff));
  e = launch_score_obs(dtype, g.G, g.causal, rp, grid, stream, a);
  if (e != hipSuccess) return e;

  const int64_t N = (int64_t)g.lq * g.n_keys;
  uint32_t* hist = reinterpret_cast<uint32_t*>(w + L.hist);
  CvState* st = reinterpret_cast<CvState*>(w + L.state);
  hipLaunchKernelGGL(cv_init_kernel, dim3(24), dim3(256), 0, stream, st, hist, N, g.k_pct, g.hkv);
  const unsigned hb = (unsigned)std::min<int64_t>(512, (N + 1023) / 1024);
  const unsigned pb = (unsigned)((g.hkv + 63) / 64);
  uint32_t* cand = reinterpret_cast<uint32_t*>(w + L.cand);
  const uint32_t cap = cand_cap(g);
  for (int pass = 0; pass < 3; ++pass) {
    uint32_t* hp = hist + (size_t)pass * g.hkv * kRadixBins;
    hipLaunchKernelGGL(radix_hist_kernel, dim3(hb, g.hkv), dim3(256), 0, stream, a.obs, N, pass, st, hp, cand, cap);
    hipLaunchKernelGGL(radix_pick_kernel, dim3(g.hkv), dim3(kPickThreads), 0, stream, hp, pass, st, g.hkv);
  }
  hipLaunchKernelGGL(radix_min_above_kernel, dim3(hb, g.hkv), dim3(256), 0, stream, a.obs, N, st, cand, cap, 1);
  hipLaunchKernelGGL(radix_min_above_kernel, dim3(hb, g.hkv), dim3(256), 0, stream, a.obs, N, st, cand, cap, 0);
  hipLaunchKernelGGL(cv_threshold_kernel, dim3(pb), dim3(64), 0, stream, st,
                     hist + (size_t)2 * g.hkv * kRadixBins, N, g.k_pct, g.alpha, g.hkv);
  // 64 columns per workgroup and step; few enough workgroups that the two
  // per-head totals are not a hot spot of global atomics
  const unsigned cb = (unsigned)std::min<int64_t>(256, (g.n_keys + 63) / 64);
  hipLaunchKernelGGL(cv_count_kernel, dim3(cb, g.hkv), dim3(256), 0, stream, a.obs, g.lq, g.n_keys, st);
  hipLaunchKernelGGL(cv_final_kernel, dim3(pb), dim3(64), 0, stream, st, g.n_keys, cv_out, g.hkv);
  return hipGetLastError();
}

}  // namespace catekv
