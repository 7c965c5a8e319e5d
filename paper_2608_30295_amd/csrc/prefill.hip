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

constexpr int kMergeRows = 16;    // rows per 256-thread workgroup of the merge

// CV (observation matrix): the sampled entries of A whose query rows are
// the workgroup's kMergeRows rows (G divides kMergeRows, so a query's G rows
// are all here), A = (1/G) sum_g exp2(s c - offset) in plain fp32 dot
// products, one entry per thread at a time with the rows' Q in LDS; the
// sample only has to place the quantile, the bracketing pass classifies A's
// values as the observation pass computes them.
template <typename T, int G>
__device__ void cv_sample_rows(const ScoreArgs& a, int sel, int row0, float my_off) {
  __shared__ float s_q[kMergeRows][kD + 1];   // +1: rows start in different banks
  __shared__ float s_o[kMergeRows];
  const int h = a.heads[sel];
  const int t = threadIdx.x;
  const uint32_t n_keys = (uint32_t)a.n_keys;
  const int64_t N = (int64_t)a.lq * a.n_keys;     // below 2^32 (the entry points check)
  for (int e = t; e < kMergeRows * kD; e += 256) {
    const int rr = e / kD, d = e % kD, r = row0 + rr;
    const int i = r / G, g = r - (r / G) * G;
    const T* q = reinterpret_cast<const T*>(a.q) + ((size_t)(h * G + g) * a.lq + (r < a.R ? i : 0)) * kD;
    float x;
    if constexpr (sizeof(T) == 2) x = __uint_as_float((uint32_t)q[d] << 16);
    else x = q[d];
    s_q[rr][d] = r < a.R ? x : 0.f;
  }
  if ((t & 15) == 0) s_o[t >> 4] = my_off;
  __syncthreads();
  const int q0 = row0 / G, q1 = min(a.lq, (row0 + kMergeRows) / G);   // this workgroup's queries
  if (q0 >= q1) return;
  const int64_t ns = cv_sample_count(N), stride = cv_sample_stride(N);
  const bool all = N < kCvSamples;                                   // sample s is entry s
  const int64_t e0 = (int64_t)q0 * n_keys, e1 = (int64_t)q1 * n_keys;
  // (plain selects: std::min / std::max return references, which the
  // compiler would keep in scratch memory here)
  const int64_t t0 = (e0 - (kCvSampleRun - 1) + stride - 1) / stride;
  const int64_t s0 = all ? e0 : (t0 > 0 ? t0 : 0) * kCvSampleRun;
  const int64_t s1r = all ? e1 : ((e1 - 1) / stride + 1) * kCvSampleRun;
  const int64_t s1 = s1r < ns ? s1r : ns;
  const T* kh = reinterpret_cast<const T*>(a.k) + (size_t)h * a.n * kD;
  const float invG = 1.0f / (float)G;
  for (int64_t s = s0 + t; s < s1; s += 256) {
    const uint32_t ent = (uint32_t)(all ? s : (s / kCvSampleRun) * stride + (s % kCvSampleRun));
    const uint32_t i = ent / n_keys, j = ent - (ent / n_keys) * n_keys;
    if ((int)i < q0 || (int)i >= q1) continue;
    const float* qr = s_q[(i - q0) * G];
    const T* kr = kh + (size_t)(a.key_off + j) * kD;
    float dot[G];
#pragma unroll
    for (int g = 0; g < G; ++g) dot[g] = 0.f;
#pragma unroll 1
    for (int c0 = 0; c0 < kD; c0 += 16) {       // 16 dims: their K values loaded together
      float kv[16];
      if constexpr (sizeof(T) == 2) {
        uint4 w[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) w[u] = *reinterpret_cast<const uint4*>(kr + c0 + 8 * u);
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const uint32_t x[4] = {w[u].x, w[u].y, w[u].z, w[u].w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            kv[8 * u + 2 * e] = bf16_lo(x[e]);
            kv[8 * u + 2 * e + 1] = bf16_hi(x[e]);
          }
        }
      } else {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float4 f = *reinterpret_cast<const float4*>(kr + c0 + 4 * u);
          kv[4 * u] = f.x;
          kv[4 * u + 1] = f.y;
          kv[4 * u + 2] = f.z;
          kv[4 * u + 3] = f.w;
        }
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float* qg = qr + g * (kD + 1) + c0;
#pragma unroll
        for (int d = 0; d < 16; ++d) dot[g] = __builtin_fmaf(qg[d], kv[d], dot[g]);
      }
    }
    const bool vis = !a.causal || a.key_off + (int64_t)j <= a.q_pos0 + (int64_t)i;
    float acc = 0.f;
#pragma unroll
    for (int g = 0; g < G; ++g)
      if (vis) acc += fast_exp2(__builtin_fmaf(dot[g], a.c, -s_o[(i - q0) * G + g]));
    a.cv.samples[(size_t)sel * kCvSamples + s] = acc * invG;
  }
}

// Merge the per-column-block row statistics: offset = m c + log2(l), +inf
// for rows with no visible key and for padding rows.  16 lanes share a row
// and walk its column blocks with independent loads, then reduce over DPP.
// A block whose sum overflowed is recomputed exactly first.
template <typename T>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 4))) void rowstats_merge_kernel(ScoreArgs a, int rpad,
                                                                                               float* __restrict__ off) {
  const int sel = blockIdx.y;
  const int n_colblk = a.n_colblk, R = a.R;
  if (blockIdx.x == 0 && blockIdx.y == 0)
    for (int i = threadIdx.x; i < a.n_zero; i += blockDim.x) a.zero_u32[i] = 0;
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
  const float o = (ok && L > 0.f) ? M16 + __log2f(L) : INFINITY;
  if (ln == 0 && row < rpad) off[(size_t)sel * rpad + row] = o;
  if (a.cv.samples) {
    const int r0 = blockIdx.x * kMergeRows;
    if (a.G == 1) cv_sample_rows<T, 1>(a, sel, r0, o);
    else if (a.G == 2) cv_sample_rows<T, 2>(a, sel, r0, o);
    else if (a.G == 4) cv_sample_rows<T, 4>(a, sel, r0, o);
    else cv_sample_rows<T, 8>(a, sel, r0, o);
  }
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
// ascending index.  Radix passes over 8-bit digits, from the highest bit in
// which the keys differ, count into 16 LDS copies (lane & 15) of the
// histogram, double-buffered so the copy for the next pass is cleared during
// this one; wave 0 sums the copies and finds the bin of the target rank with a
// suffix scan (DPP steps), so a pass costs two barriers.  Once the target bin
// holds at most 64 keys, they are listed and one wave ranks them, in place of
// the remaining passes.  The positions of the selected entries come from
// per-row ballots and one exchange of the per-wave counts.
//
// Three uses (MODE): a whole row of scores; one slice of a row (rows are cut
// into PER * kTopkThreads-score slices whose own k best, in ascending order,
// go to a candidate list with their keys); a row's candidate list (keys read
// from the list, -1 entries never chosen, the candidates' indices out).  The k
// best of a row are always among its slices' k best (an entry outranked by k
// entries of its own slice is outranked by k entries of the row; ties go to
// the lower index in both), and the candidate list is ascending, so the two
// stages reproduce the one-stage result.
enum TopkMode { kTopkRow = 0, kTopkSliceMode = 1, kTopkList = 2 };
constexpr int64_t kTopkSlice = 16 * kTopkThreads;   // scores per slice of long rows
constexpr int64_t kTopkSmallSlice = 4 * kTopkThreads;   // scores per slice of short rows

// A candidate: the score's ordered key (low word) and its index (high word,
// -1 for none).  The two stages run in one launch (topk_fused_kernel): a
// slice writes its candidates with device-scope atomics and the list stage
// reads them with device-scope atomic loads, so a workgroup on another XCD
// sees them, and the list stage needs no second look at the scores.
typedef unsigned long long TopkCand;

struct TopkArgs {
  const float* S;          // scores [rows][n]
  int64_t n;
  const TopkCand* list;    // kTopkList: candidates [rows][list_len]
  int64_t list_len;
  int k, b;                // select k; kTopkRow / kTopkList write b entries per row (-1 padded)
  int32_t* out;            // kTopkRow / kTopkList: [rows][b]
  TopkCand* cand;          // kTopkSliceMode: [rows][n_slices][k]
};

// Wave-wide AND / OR of a word (every lane gets it): DPP steps inside each
// row of 16 lanes, then the gfx950 row swaps; no LDS traffic.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, false);
}
__device__ __forceinline__ uint32_t wave_and(uint32_t x) {
  x &= dpp_u32<kDppXor1>(x);
  x &= dpp_u32<kDppXor2>(x);
  x &= dpp_u32<kDppHalfMirror>(x);
  x &= dpp_u32<kDppMirror>(x);
  const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  x = r[0] & r[1];
  const auto r2 = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return r2[0] & r2[1];
}
__device__ __forceinline__ uint32_t wave_or(uint32_t x) {
  x |= dpp_u32<kDppXor1>(x);
  x |= dpp_u32<kDppXor2>(x);
  x |= dpp_u32<kDppHalfMirror>(x);
  x |= dpp_u32<kDppMirror>(x);
  const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  x = r[0] | r[1];
  const auto r2 = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return r2[0] | r2[1];
}
// Inclusive suffix sums over the 64 lanes (lane l gets the sum over lanes
// l..63): row_shl steps (lane l reads lane l + s of its row, 0 past the row's
// end), then the totals of the rows above by readlane.
__device__ __forceinline__ int wave_suffix_sum(int x) {
  x += (int)dpp_u32<0x101>((uint32_t)x);
  x += (int)dpp_u32<0x102>((uint32_t)x);
  x += (int)dpp_u32<0x104>((uint32_t)x);
  x += (int)dpp_u32<0x108>((uint32_t)x);
  const int r1 = __builtin_amdgcn_readlane(x, 16), r2 = __builtin_amdgcn_readlane(x, 32),
            r3 = __builtin_amdgcn_readlane(x, 48);
  const int row = (int)(threadIdx.x & 63) >> 4;
  return x + (row < 1 ? r1 : 0) + (row < 2 ? r2 : 0) + (row < 3 ? r3 : 0);
}

template <int PER, int MODE>
__device__ __forceinline__ void topk_body(const TopkArgs& a, int row, int slice, int n_slices) {
  constexpr int NW = kTopkThreads / 64;
  constexpr int NCOPY = 16;
  constexpr int RS = 260;                  // words per copy: 256 bins, rows 16-byte aligned
  constexpr int kSmallBin = 64;            // a target bin this small is ranked by one wave
  static_assert(PER <= 32, "validity is a 32-bit mask per lane");
  __shared__ __attribute__((aligned(16))) int s_h[2][NCOPY][RS];
  __shared__ uint32_t s_and[NW], s_or[NW];
  __shared__ int s_gt[NW], s_eq[NW];
  __shared__ uint32_t s_prefix;
  __shared__ int s_remaining, s_small, s_nlist;
  __shared__ uint32_t s_list[kSmallBin];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const float* Ss = a.S + (size_t)row * a.n;
  int64_t start = 0, len = a.n;
  int k = a.k, b = a.b;
  int32_t* out = a.out + (size_t)row * a.b;
  TopkCand* cout = nullptr;
  const TopkCand* lst = nullptr;
  if (MODE == kTopkSliceMode) {
    constexpr int64_t SL = (int64_t)PER * kTopkThreads;
    start = (int64_t)slice * SL;
    len = min(SL, a.n - start);
    k = (int)min((int64_t)a.k, len);
    b = a.k;
    cout = a.cand + ((size_t)row * n_slices + slice) * a.k;
  } else if (MODE == kTopkList) {
    len = a.list_len;
    lst = a.list + (size_t)row * a.list_len;
  }
  const int64_t base = (int64_t)wave * PER * 64 + lane;       // entry of row 0; row i adds 64 i
  // kTopkList keeps the candidates' indices in registers up to 8 per lane
  // and reads longer lists' indices again when writing (registers: at most
  // 128 per lane at 1024 threads)
  constexpr bool KEEP = PER <= 8;
  uint32_t key[PER];
  int32_t idx[KEEP ? PER : 1];
  uint32_t vmask = 0;                                          // bit i: row i holds an entry
  // every load is issued (entries past the end re-read the last one, len >= 1
  // in every mode), so none waits behind a branch
  const int64_t last = len - 1;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int64_t e = base + 64 * i;
    const bool in = e < len;
    const int64_t ec = in ? e : last;
    if (MODE == kTopkList) {
      const TopkCand c = __hip_atomic_load(&lst[ec], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const int32_t j = in ? (int32_t)(c >> 32) : -1;
      if (KEEP) idx[KEEP ? i : 0] = j;
      key[i] = j >= 0 ? (uint32_t)c : 0u;
      vmask |= (j >= 0 ? 1u : 0u) << i;
    } else {
      const uint32_t kk = ord_key(Ss[start + ec]);
      key[i] = in ? kk : 0u;
      vmask |= (in ? 1u : 0u) << i;
    }
  }
  auto valid = [&](int i) { return (vmask >> i) & 1u; };

  // bits shared by every key need no pass: the digits start at the highest
  // bit that differs between keys (chunk scores share sign and most exponent
  // bits), and a digit made only of shared bits is skipped
  uint32_t kand = 0xFFFFFFFFu, kor = 0u;
#pragma unroll
  for (int i = 0; i < PER; ++i)
    if (valid(i)) { kand &= key[i]; kor |= key[i]; }
  kand = wave_and(kand);
  kor = wave_or(kor);
  if (lane == 0) { s_and[wave] = kand; s_or[wave] = kor; }
  for (int i = t; i < NCOPY * RS; i += kTopkThreads) (&s_h[0][0][0])[i] = 0;
  if (t == 0) { s_small = 0; s_nlist = 0; }
  __syncthreads();
  kand = 0xFFFFFFFFu;
  kor = 0u;
#pragma unroll
  for (int w = 0; w < NW; ++w) { kand &= s_and[w]; kor |= s_or[w]; }
  const uint32_t varying = __builtin_amdgcn_readfirstlane(kand ^ kor);
  kand = __builtin_amdgcn_readfirstlane(kand);
  const int hb = varying ? 31 - __builtin_clz(varying) : -1;

  // the bits above hb are every key's: the prefix starts with them
  const uint32_t low = varying ? (2u << hb) - 1u : 0u;
  uint32_t prefix = kand & ~low, mask = ~low;
  int remaining = k;       // rank (from the top) still to locate among keys matching the prefix
  int cur = 0;
  bool small = false;
  for (int top = hb; top >= 0; top -= 8) {
    // the last digit may reach below bit 0: it then starts at bit 0 and its
    // upper bits, already fixed by the prefix, are the same for every key counted
    const int shift = top >= 7 ? top - 7 : 0;
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
      const int incl = wave_suffix_sum(c4);
      const int excl = incl - c4;
      if (excl < remaining && incl >= remaining) {
        // the bin among the lane's four (highest first) where the rank falls;
        // cum counts the keys in the bins above it
        int cum = excl, j, hj;
        if (cum + h3 >= remaining) { j = 3; hj = h3; }
        else if ((cum += h3) + h2 >= remaining) { j = 2; hj = h2; }
        else if ((cum += h2) + h1 >= remaining) { j = 1; hj = h1; }
        else { cum += h1; j = 0; hj = h0; }
        s_prefix = prefix | ((uint32_t)(4 * lane + j) << shift);
        s_remaining = remaining - cum;
        s_small = top >= 8 && hj <= kSmallBin;   // more passes to go, few keys left in the bin
      }
    }
    __syncthreads();
    prefix = s_prefix;
    remaining = s_remaining;
    mask |= 255u << shift;
    cur ^= 1;
    small = s_small;
    if (small) break;
  }
  if (small) {
    // the keys matching the prefix (at most kSmallBin) go to a list, and one
    // wave finds the key of rank `remaining` among them by counting, for
    // each, the keys above and at it
#pragma unroll
    for (int i = 0; i < PER; ++i)
      if (valid(i) && (key[i] & mask) == prefix) {
        const int p = atomicAdd(&s_nlist, 1);
        if (p < kSmallBin) s_list[p] = key[i];
      }
    __syncthreads();
    if (wave == 0) {
      const int m = min(s_nlist, kSmallBin);
      const uint32_t mine = lane < m ? s_list[lane] : 0u;
      int gt = 0, ge = 0;
      for (int j = 0; j < m; ++j) {
        const uint32_t kj = (uint32_t)__builtin_amdgcn_readlane((int)mine, j);
        gt += kj > mine;
        ge += kj >= mine;
      }
      if (lane < m && gt < remaining && remaining <= ge) {   // lanes holding that key write alike
        s_prefix = mine;
        s_remaining = remaining - gt;
      }
    }
    __syncthreads();
    prefix = s_prefix;
    remaining = s_remaining;
  }
  const uint32_t tau = prefix;   // key of the k-th largest score
  // `remaining` entries equal to tau are taken, lowest indices first

  int n_gt = 0, n_eq = 0;        // the wave's counts, from ballots (wave-uniform)
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const bool v = valid(i);
    n_gt += __popcll(__ballot(v && key[i] > tau));
    n_eq += __popcll(__ballot(v && key[i] == tau));
  }
  if (lane == 0) { s_gt[wave] = n_gt; s_eq[wave] = n_eq; }
  __syncthreads();
  int pos = 0, eqr = 0;          // entries taken and ties seen in the waves before this one
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    if (w < wave) {
      const int e = s_eq[w];
      pos += s_gt[w] + min(max(remaining - eqr, 0), e);
      eqr += e;
    }
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
      if (MODE == kTopkList)
        out[p] = KEEP ? idx[KEEP ? i : 0]
                      : (int32_t)(__hip_atomic_load(&lst[e], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >> 32);
      else if (MODE == kTopkSliceMode)
        atomicExch(&cout[p], ((TopkCand)(uint32_t)(start + e) << 32) | key[i]);
      else out[p] = (int32_t)(start + e);
    }
    pos += __popcll(mt);
    eqr += __popcll(meq);
  }
  for (int i = k + t; i < b; i += kTopkThreads) {
    if (MODE == kTopkSliceMode) atomicExch(&cout[i], 0xFFFFFFFF00000000ull);
    else out[i] = -1;
  }
}

// one row per workgroup
template <int PER>
__global__ __launch_bounds__(kTopkThreads) void topk_wave_kernel(TopkArgs a) {
  topk_body<PER, kTopkRow>(a, blockIdx.x, 0, 1);
}

// Both stages in one launch, grid (slices, rows): every workgroup selects its
// slice's k best; the last of a row to finish (arrive[row] counts them, zero
// on entry and reset on exit) selects the row's k best among the candidates.
// A workgroup arrives once its candidate stores have completed (device-scope
// atomics, waited for), so no cache write-back is needed.
template <int PER1, int PER2>
__global__ __launch_bounds__(kTopkThreads) void topk_fused_kernel(TopkArgs s1, TopkArgs s2, uint32_t* arrive) {
  __shared__ int s_last;
  const int row = blockIdx.y;
  topk_body<PER1, kTopkSliceMode>(s1, row, blockIdx.x, gridDim.x);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) s_last = atomicAdd(&arrive[row], 1u) == gridDim.x - 1;
  __syncthreads();
  if (!s_last) return;
  topk_body<PER2, kTopkList>(s2, row, 0, 1);
  if (threadIdx.x == 0) arrive[row] = 0;
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
  const int64_t flat = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t row = flat / SEG;
  const int seg = (int)(flat - row * SEG);
  // the row's chunk index is read alongside the last one (window rows read
  // the last one twice), so both loads take one round trip
  const int64_t last = ix[a.b_eff - 1];
  int64_t c = ix[min(row / a.cs, (int64_t)a.b_eff - 1)];
  const int64_t tail = a.n_keys - (a.n_chunks - 1) * a.cs;        // size of the last chunk
  const int64_t n_sel_tok = (int64_t)a.b_eff * a.cs - ((last == a.n_chunks - 1) ? (a.cs - tail) : 0);
  const int64_t len = n_sel_tok + a.l_obs;
  if (blockIdx.x == 0 && threadIdx.x == 0) a.lens_out[h] = len;
  if (row >= len) return;
  int64_t src;
  if (row < n_sel_tok) {
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
  a.zero_u32 = reinterpret_cast<uint32_t*>(w + L.topk);   // the top-k's arrival counters
  a.n_zero = g.n_sel;
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

// ws: n_rows arrival counters (zero on entry: the caller's previous kernel
// clears them; left zero), then the candidate lists of two-stage rows.
size_t topk_counter_bytes(int n_rows) { return align256((size_t)n_rows * sizeof(uint32_t)); }
size_t topk_workspace_bytes(int n_rows, int64_t n) {
  return topk_counter_bytes(n_rows) + (n > kTopkSmallSlice ? (size_t)n_rows * 2 * kTopkSlice * sizeof(TopkCand) : 0);
}

// both stages in one launch; PER2 from the candidate list's length
template <int PER1>
static void launch_topk_fused(const TopkArgs& s1, const TopkArgs& s2, unsigned n_slices, int n_rows,
                              uint32_t* arrive, hipStream_t stream) {
  const int64_t m = s2.list_len;
  const dim3 grid(n_slices, n_rows), block(kTopkThreads);
  if (m <= 1 * kTopkThreads) hipLaunchKernelGGL((topk_fused_kernel<PER1, 1>), grid, block, 0, stream, s1, s2, arrive);
  else if (m <= 2 * kTopkThreads) hipLaunchKernelGGL((topk_fused_kernel<PER1, 2>), grid, block, 0, stream, s1, s2, arrive);
  else if (m <= 4 * kTopkThreads) hipLaunchKernelGGL((topk_fused_kernel<PER1, 4>), grid, block, 0, stream, s1, s2, arrive);
  else if (m <= 8 * kTopkThreads) hipLaunchKernelGGL((topk_fused_kernel<PER1, 8>), grid, block, 0, stream, s1, s2, arrive);
  else if (m <= 16 * kTopkThreads) hipLaunchKernelGGL((topk_fused_kernel<PER1, 16>), grid, block, 0, stream, s1, s2, arrive);
  else hipLaunchKernelGGL((topk_fused_kernel<PER1, 32>), grid, block, 0, stream, s1, s2, arrive);
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
  uint32_t* arrive = reinterpret_cast<uint32_t*>(ws);
  TopkCand* cand = ws ? reinterpret_cast<TopkCand*>(reinterpret_cast<char*>(ws) + topk_counter_bytes(n_rows)) : nullptr;
  if (few_short_rows) {
    TopkArgs s1 = a;
    s1.cand = cand;
    TopkArgs s2 = a;
    s2.list = cand;
    s2.list_len = n_small * k_eff;
    launch_topk_fused<4>(s1, s2, (unsigned)n_small, n_rows, arrive, stream);
  } else if (n <= kTopkSlice) {
    hipLaunchKernelGGL((topk_wave_kernel<16>), dim3(n_rows), dim3(kTopkThreads), 0, stream, a);
  } else if (n <= 2 * kTopkSlice) {
    hipLaunchKernelGGL((topk_wave_kernel<32>), dim3(n_rows), dim3(kTopkThreads), 0, stream, a);
  } else if (ws && n_slices * k_eff <= 2 * kTopkSlice) {
    // the k best of every slice, then the k best of those candidates
    TopkArgs s1 = a;
    s1.cand = cand;
    TopkArgs s2 = a;
    s2.list = cand;
    s2.list_len = n_slices * k_eff;
    launch_topk_fused<16>(s1, s2, (unsigned)n_slices, n_rows, arrive, stream);
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
  size_t rowpart, rowoff, obs, cv, total;
};
static ScoreLayout score_layout(const ScoreGeom& g) {
  ScoreLayout L{};
  const int rp = score_rows_pad(g.G * g.lq);
  size_t o = 0;
  L.rowpart = o; o += align256((size_t)g.hkv * g.n_colblk * rp * sizeof(float2));
  L.rowoff = o; o += align256((size_t)g.hkv * rp * sizeof(float));
  L.obs = o; o += align256((size_t)g.hkv * g.lq * g.n_keys * sizeof(float));
  L.cv = o; o += align256(cv_workspace_bytes(g.hkv, g.lq, g.n_keys, g.n_colblk));
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
  a.cv = cv_link(w + L.cv, g.hkv, g.lq, g.n_keys, g.n_colblk, kCvMaxSub);
  const dim3 grid(g.n_colblk, g.hkv);
  hipError_t e = launch_score_rowstats(dtype, g.G, g.causal, rp, grid, stream, a);
  if (e != hipSuccess) return e;
  if (dtype == CATEKV_BF16)
    hipLaunchKernelGGL(rowstats_merge_kernel<uint16_t>, dim3((rp + kMergeRows - 1) / kMergeRows, g.hkv), dim3(256), 0,
                       stream, a, rp, reinterpret_cast<float*>(w + L.rowoff));
  else
    hipLaunchKernelGGL(rowstats_merge_kernel<float>, dim3((rp + kMergeRows - 1) / kMergeRows, g.hkv), dim3(256), 0,
                       stream, a, rp, reinterpret_cast<float*>(w + L.rowoff));
  // the merge also took the sampled entries of A; the bracket from them,
  // the bracketing pass, A itself only for the heads the bracket missed
  e = launch_cv_sample(a, g.k_pct, g.alpha, stream);
  if (e != hipSuccess) return e;
  e = launch_score_obs_bracket(dtype, g.G, g.causal, rp, grid, stream, a);
  if (e != hipSuccess) return e;
  a.cv_gate = 1;
  e = launch_score_obs(dtype, g.G, g.causal, rp, grid, stream, a);
  if (e != hipSuccess) return e;
  return launch_cv_finish(a, g.k_pct, g.alpha, cv_out, stream);
}

}  // namespace catekv
