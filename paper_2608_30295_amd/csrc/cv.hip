// CV head score (Section 3.2, Eq. 2-4) over the observation matrix A of each
// KV head (Eq. 1; [lq][n_keys] fp32, row-major, written by the score pass):
// Phi = alpha times the k-th percentile of A's N = lq n_keys entries (linear
// interpolation between the order statistics x_(lo) and x_(lo+1),
// lo = floor((N - 1) k)), C_j = #{i : A[i][j] >= Phi}, and the score is the
// population standard deviation of C over its mean.
//
// Bracket route: a sample of A gives a key range [k_lo, k_hi] expected to
// hold ranks lo and lo + 1, and with it a bound t_lo <= Phi.  The
// observation pass writes out the few entries at or above the lower of the
// two bounds with their columns (every entry at or above Phi is among
// them); x_(lo), x_(lo+1) and Phi are resolved over those inside the key
// range, and C_j is the count of column j's gathered values at or above Phi.
// Radix route: when the sample's range misses a rank, or the gathered
// entries overflow their buffer (heavy ties), exact radix passes over A
// take over for that head.
#include "score.h"

#include <algorithm>
#include <cmath>

namespace catekv {
namespace {

constexpr int kBins = kCvBins;
constexpr uint32_t kNone = kCvNone;
__device__ __forceinline__ uint32_t ord_key(float f) { return cv_key(f); }
__device__ __forceinline__ float key_to_float(uint32_t key) { return cv_key_float(key); }
__device__ __forceinline__ bool bracket_route(const CvState& S, int64_t N) { return cv_bracket_route(S, N); }

__device__ __forceinline__ uint32_t mbcnt(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}


// For a histogram hh[0, nb) (LDS or global) and 0-based ranks r0, r1 below
// its total: the bins holding them (s_bin[0], s_bin[1]), their positions
// inside those bins (s_pos[0], s_pos[1]) and the first non-empty bin above
// s_bin[0] (s_bin[2], kNone if none).  A 64-bit block prefix over NT
// threads, kBins / NT bins each.  Called by the whole workgroup.
template <int NT>
__device__ void locate_ranks(const uint32_t* hh, int nb, int64_t r0, int64_t r1, int64_t* s_tot, uint32_t* s_bin,
                             int64_t* s_pos) {
  constexpr int BPT = kBins / NT;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  __syncthreads();                 // earlier readers of s_bin / s_pos are done
  uint32_t c[BPT];
  uint32_t mine = 0;               // a head's counts stay below 2^32 (N < 2^32)
#pragma unroll
  for (int i = 0; i < BPT; ++i) {
    const int b = t * BPT + i;
    c[i] = b < nb ? hh[b] : 0u;
    mine += c[i];
  }
  uint32_t x = mine;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  if (lane == 63) s_tot[wave] = x;
  if (t == 0) {
    s_bin[0] = s_bin[1] = (uint32_t)(nb - 1);
    s_bin[2] = kNone;
    s_pos[0] = s_pos[1] = 0;
  }
  __syncthreads();
  int64_t before = (int64_t)(x - mine);
  for (int w = 0; w < wave; ++w) before += s_tot[w];
#pragma unroll
  for (int i = 0; i < BPT; ++i) {
    const int64_t b0 = before, b1 = before + c[i];   // ranks [b0, b1) fall in this bin
    if (b0 <= r0 && r0 < b1) { s_bin[0] = t * BPT + i; s_pos[0] = r0 - b0; }
    if (b0 <= r1 && r1 < b1) { s_bin[1] = t * BPT + i; s_pos[1] = r1 - b0; }
    before = b1;
  }
  __syncthreads();
  const uint32_t b = s_bin[0];
  uint32_t nxt = kNone;
#pragma unroll
  for (int i = 0; i < BPT; ++i)
    if ((uint32_t)(t * BPT + i) > b && c[i] != 0u) nxt = min(nxt, (uint32_t)(t * BPT + i));
  for (int off = 32; off > 0; off >>= 1) nxt = min(nxt, (uint32_t)__shfl_xor((int)nxt, off));
  if (lane == 0 && nxt != kNone) atomicMin(&s_bin[2], nxt);
  __syncthreads();
}

// Sum over a workgroup of 256 threads (4 waves); s holds 4 partials.
__device__ __forceinline__ unsigned long long block_sum256(unsigned long long v, unsigned long long* s) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) s[threadIdx.x >> 6] = v;
  __syncthreads();
  return s[0] + s[1] + s[2] + s[3];
}

// Eq. 4 from exact integer sums: sqrt(E[C^2] - E[C]^2) / E[C].
__device__ __forceinline__ float cv_value(unsigned long long s1, unsigned long long s2, int64_t n_keys) {
  const double N = (double)n_keys;
  const double mu = (double)s1 / N;
  if (mu == 0.0) return 0.f;
  double var = (double)s2 / N - mu * mu;
  var = var < 0.0 ? 0.0 : var;
  return (float)(sqrt(var) / mu);
}

// Called by thread 0 of every workgroup of the launch that ends head h, after
// its own additions to *sum_c and *sum_c2: the last to arrive writes the
// score.  Nothing waits; the sums are read with atomics, after a fence.
__device__ void arrive_and_finish(CvState& S, unsigned long long* sum_c, unsigned long long* sum_c2, int64_t n_keys,
                                  float* cv_out, int h) {
  __threadfence();
  const uint32_t done = atomicAdd(&S.arrive_f, 1u);
  if (done == gridDim.x - 1) {
    __threadfence();
    const unsigned long long s1 = atomicAdd(sum_c, 0ull), s2 = atomicAdd(sum_c2, 0ull);
    cv_out[h] = cv_value(s1, s2, n_keys);
  }
}

// Phi = alpha (x_lo + frac (x_hi - x_lo)) in fp64 (Eq. 2 with the
// interpolated percentile).
__device__ __forceinline__ double phi_of(double xlo, double xhi, int64_t N, double k_pct, double alpha, int64_t lo) {
  const double pos = (double)(N - 1) * k_pct;
  const double frac = pos - (double)lo;
  return alpha * (xlo + frac * (xhi - xlo));
}

// ---------------------------------------------------------------------------
// 1. Sample: state, and the bracket from the sampled entries of A
// ---------------------------------------------------------------------------

// The sample's first two radix digits give the 22-bit key prefixes holding
// sample ranks lo s / N -+ (8 sigma + 32), sigma the binomial spread of a
// sample rank; the bracket is every key with a prefix in that range.  As
// x_(lo) >= the bracket's bottom f_lo, Phi >= alpha f_lo: t_lo is that bound
// less 2^-40 relative (far beyond the rounding of the fp64 interpolation),
// rounded down to a float.
constexpr int kSampleThreads = 1024;
constexpr int kSamplePer = kCvSamples / kSampleThreads;

__global__ __launch_bounds__(kSampleThreads) void cv_sample_kernel(const float* __restrict__ samples, int64_t N,
                                                                   double k_pct, double alpha, CvState* st,
                                                                   uint32_t* __restrict__ hist, int hkv) {
  __shared__ uint32_t s_h[kBins];
  __shared__ uint32_t s_h2[2][kBins];
  __shared__ int64_t s_tot[kSampleThreads / 64];
  __shared__ uint32_t s_bin[3];
  __shared__ int64_t s_pos[2];
  const int h = blockIdx.x;
  const int t = threadIdx.x;
  for (int p = 0; p < 4; ++p)
    for (int i = t; i < kBins; i += kSampleThreads) hist[((size_t)p * hkv + h) * kBins + i] = 0;
  for (int i = t; i < kBins; i += kSampleThreads) s_h[i] = 0;
  for (int i = t; i < 2 * kBins; i += kSampleThreads) s_h2[i / kBins][i % kBins] = 0;
  const int64_t rank = (int64_t)floor((double)(N - 1) * k_pct);
  __syncthreads();
  const int64_t ns = cv_sample_count(N);
  const float* sh = samples + (size_t)h * kCvSamples;
  float v[kSamplePer];
#pragma unroll
  for (int u = 0; u < kSamplePer; ++u) v[u] = sh[std::min<int64_t>((int64_t)t * kSamplePer + u, ns - 1)];
#pragma unroll
  for (int u = 0; u < kSamplePer; ++u) hist_add(s_h, (int64_t)t * kSamplePer + u < ns, ord_key(v[u]) >> 21);
  const double rs = (double)rank * (double)ns / (double)N;
  const double pq = (double)rank / (double)N;
  const double m = 8.0 * sqrt((double)ns * pq * (1.0 - pq)) + 32.0;
  const int64_t lo_s = (int64_t)fmax(0.0, floor(rs - m)), hi_s = (int64_t)fmin((double)(ns - 1), ceil(rs + m));
  locate_ranks<kSampleThreads>(s_h, kBins, lo_s, hi_s, s_tot, s_bin, s_pos);
  const uint32_t bl = s_bin[0], bh = s_bin[1];
  const int64_t rl = s_pos[0], rh = s_pos[1];
#pragma unroll
  for (int u = 0; u < kSamplePer; ++u) {
    const bool ok = (int64_t)t * kSamplePer + u < ns;
    const uint32_t key = ord_key(v[u]);
    if (ok && (key >> 21) == bl) atomicAdd(&s_h2[0][(key >> 10) & 0x7FF], 1u);
    if (ok && (key >> 21) == bh) atomicAdd(&s_h2[1][(key >> 10) & 0x7FF], 1u);
  }
  locate_ranks<kSampleThreads>(s_h2[0], kBins, rl, rl, s_tot, s_bin, s_pos);
  const uint32_t d_lo = s_bin[0];
  locate_ranks<kSampleThreads>(s_h2[1], kBins, rh, rh, s_tot, s_bin, s_pos);
  const uint32_t d_hi = s_bin[0];
  if (t == 0) {
    CvState& s = st[h];
    const uint32_t p_lo = (bl << 11) | d_lo, p_hi = (bh << 11) | d_hi;
    const uint32_t k_lo = p_lo << 10;
    const uint32_t k_hi = p_hi == 0x3FFFFFu ? 0xFFFFFFFFu : ((p_hi + 1) << 10) - 1;
    const float f_lo = key_to_float(k_lo);
    const double dl = alpha * (double)f_lo - fabs(alpha * (double)f_lo) * 0x1p-40;
    float tl = (float)dl;
    if ((double)tl > dl) tl = nextafterf(tl, -INFINITY);
    const uint32_t span = k_hi - k_lo;
    const int bits = span ? 32 - __clz((int)span) : 0;
    s.rank = rank;
    s.k_lo = k_lo;
    s.k_hi = k_hi;
    s.t_lo = tl;
    s.shift1 = bits > 11 ? bits - 11 : 0;
    s.phi_over = 0;
    s.n_cand = 0;
    s.ge_lo = 0;
    s.sum_c = 0;
    s.sum_c2 = 0;
    s.phi = 0.0;
    s.min2 = kNone;
    s.n_list = 0;
    s.arrive_r = 0;
    s.arrive_f = 0;
    s.fb_min = kNone;
    s.fb_prefix[0] = s.fb_prefix[1] = 0;
    s.fb_rem[0] = s.fb_rem[1] = 0;
    s.fb_lt[0] = s.fb_lt[1] = 0;
    s.fb_sum_c = 0;
    s.fb_sum_c2 = 0;
  }
}

// ---------------------------------------------------------------------------
// 2. The bracketing pass is the observation-matrix pass (score.h,
//    kObsBracket): the entries at or above min(bracket bottom, t_lo) as
//    (value, column), in one buffer per wave of each column block; at its
//    end each workgroup counts its pairs into the head's totals (bracket
//    entries by first digit, entries at or above the bracket's bottom).
// ---------------------------------------------------------------------------

constexpr int kCountRows = 16;    // rows per lane loaded together by the radix route's column walk

// The radix route's column walk: ~1024 workgroups over all heads.
int64_t col_blocks(int64_t n_keys, int hkv) {
  const int64_t blocks = (n_keys + 63) / 64;
  const int64_t want = std::max<int64_t>(128, 1024 / std::max(1, hkv));
  return std::max<int64_t>(1, std::min(blocks, want));
}

__device__ __forceinline__ void hist_over_A(const float* __restrict__ Ah, int64_t N, uint32_t* s_h, uint32_t mask,
                                            uint32_t want, int shift, uint32_t dmask, uint32_t above, uint32_t* mn) {
  const int64_t n4 = (N & 3) == 0 && ((reinterpret_cast<uintptr_t>(Ah) & 15) == 0) ? N / 4 : 0;
  const int64_t step = (int64_t)gridDim.x * blockDim.x;
  auto visit = [&](float f) {
    const uint32_t key = ord_key(f);
    hist_add(s_h, (key & mask) == want, (key >> shift) & dmask);
    if ((key & mask) > above) *mn = min(*mn, key);
  };
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += step) {
    const float4 v = *reinterpret_cast<const float4*>(Ah + 4 * i);
    visit(v.x);
    visit(v.y);
    visit(v.z);
    visit(v.w);
  }
  for (int64_t i = 4 * n4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < N; i += step) visit(Ah[i]);
}

__device__ __forceinline__ void flush_hist(const uint32_t* s_h, uint32_t* __restrict__ g) {
  for (int i = threadIdx.x; i < kBins; i += blockDim.x)
    if (s_h[i]) atomicAdd(&g[i], s_h[i]);
}

// nb (<= 64) consecutive pair buffers starting at buffer `first`, seen as
// one index space: s_pre[w] = pairs before buffer w (filled by the first
// wave, all fills loaded at once); returns the total.  Item k lies in the
// last buffer w with s_pre[w] <= k.
__device__ uint32_t buffer_prefix(const uint32_t* __restrict__ pfill, size_t first, int nb, uint32_t* s_pre) {
  const int t = threadIdx.x;
  if (t < 64) {
    const uint32_t f = t < nb ? pfill[first + t] : 0u;
    uint32_t x = f;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const uint32_t y = __shfl_up(x, off);
      if (t >= off) x += y;
    }
    if (t < nb) s_pre[t] = x - f;
    if (t == nb - 1) s_pre[nb] = x;
  }
  __syncthreads();
  return s_pre[nb];
}
__device__ __forceinline__ const uint2* buffer_item(const uint2* __restrict__ pairs, size_t first, int nb,
                                                    uint32_t capw, const uint32_t* s_pre, uint32_t k) {
  int w = 0;
  while (w + 1 < nb && s_pre[w + 1] <= k) ++w;
  return pairs + (first + w) * capw + (k - s_pre[w]);
}

// ---------------------------------------------------------------------------
// 3. Bracket route: workgroup x takes the pairs of column-walk workgroups
//    [kRegions x, kRegions (x + 1)) and lists the bracket entries in
//    x_(lo)'s first-digit bin; it also keeps the smallest bracket entry above
//    that bin.  The last workgroup of a head to finish takes x_(lo), x_(lo+1)
//    and Phi.  Radix route: histogram of the top key digit over A.
// ---------------------------------------------------------------------------

constexpr int kListCap = kCvListCap;
constexpr int kRegions = 8;        // pair buffers per listing workgroup
constexpr int kShortList = 1024;   // lists resolved by counting ranks
constexpr int kListStage = 2048;   // entries staged before a reservation (a round adds <= 1024)

// Offsets key - k_lo of one workgroup's gathered pairs, 4 per thread and
// round (the same trip count on every lane); f(inside the bracket, offset).
template <typename F>
__device__ __forceinline__ void for_pairs(const uint2* __restrict__ ph, uint32_t fill, uint32_t k_lo, uint32_t span,
                                          F&& f) {
  for (uint32_t i0 = 0; i0 < fill; i0 += 4 * 256) {
    uint32_t o[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {   // every load issued (clamped), then used
      const uint32_t i = i0 + u * 256 + threadIdx.x;
      const uint32_t x = ph[min(i, fill - 1)].x;
      o[u] = i < fill ? (x | 0x80000000u) - k_lo : kNone;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) f(o[u] <= span, o[u]);
  }
}

// x_(lo) and the key after it, by the last listing workgroup of a head: its
// offset key - k_lo is b1's bin (first digit) followed by the rank-rem entry
// of the list.  A short list is resolved by counting each entry's rank (LDS
// broadcasts), a longer one by its remaining digits, 11 bits at a time (over
// every workgroup's pairs again if the list overflowed).  The list, its
// count and min2 are read with atomic loads.  Returns (in thread 0) Phi.
__device__ double resolve_phi(CvState& S, const uint32_t* __restrict__ hist0, const uint32_t* __restrict__ lh,
                              const uint2* __restrict__ pairs, const uint32_t* __restrict__ pfill, uint32_t capw,
                              int cb, int h, int64_t N, double k_pct, double alpha, uint32_t b1, uint32_t next1,
                              int64_t rem, unsigned long long lt, uint32_t* s_h, int64_t* s_tot, uint32_t* s_bin,
                              int64_t* s_pos, uint32_t* s_x) {
  const int t = threadIdx.x, lane = t & 63;
  const int64_t lo = S.rank;
  const uint32_t k_lo = S.k_lo, span = S.k_hi - S.k_lo;
  const int sh1 = S.shift1;
  uint32_t P = b1, eq = 0, next = next1;
  if (sh1 == 0) {
    eq = hist0[(size_t)h * kBins + b1];
  } else {
    const uint32_t nl = __hip_atomic_load(&S.n_list, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t min2 = __hip_atomic_load(&S.min2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (nl <= (uint32_t)kShortList) {
      uint32_t* s_l = s_h;
      __syncthreads();
      for (uint32_t i = t; i < nl; i += 256) s_l[i] = __hip_atomic_load(&lh[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (t == 0) {
        s_x[0] = kNone;
        s_x[3] = kNone;
      }
      __syncthreads();
      for (uint32_t i = t; i < nl; i += 256) {
        const uint32_t e = s_l[i];
        uint32_t n_lt = 0, n_eq = 0;
        for (uint32_t m = 0; m < nl; ++m) {
          const uint32_t f = s_l[m];
          n_lt += f < e;
          n_eq += f == e;
        }
        if ((int64_t)n_lt <= rem && rem < (int64_t)(n_lt + n_eq)) {   // every entry of the run writes the same
          s_x[0] = e;
          s_x[1] = n_lt;
          s_x[2] = n_eq;
        }
      }
      __syncthreads();
      const uint32_t x = s_x[0];
      uint32_t mn = kNone;
      for (uint32_t i = t; i < nl; i += 256)
        if (s_l[i] > x) mn = min(mn, s_l[i]);
      for (int off = 32; off > 0; off >>= 1) mn = min(mn, (uint32_t)__shfl_xor((int)mn, off));
      if (lane == 0 && mn != kNone) atomicMin(&s_x[3], mn);
      __syncthreads();
      P = x;
      lt += s_x[1];
      eq = s_x[2];
      next = min(s_x[3], min2);
    } else {
      const bool from_list = nl <= (uint32_t)kListCap;
      int bits = sh1;
      while (bits > 0) {
        const int d = bits > 11 ? 11 : bits;
        const int nsh = bits - d;
        const uint32_t dmask = (1u << d) - 1u;
        const bool last = nsh == 0;
        __syncthreads();
        for (int i = t; i < kBins; i += 256) s_h[i] = 0;
        if (t == 0) s_x[3] = kNone;
        __syncthreads();
        uint32_t mn = kNone;
        auto visit = [&](bool ok, uint32_t o) {
          const uint32_t hi = o >> bits;
          hist_add(s_h, ok && hi == P, (o >> nsh) & dmask);
          if (last && ok && hi > P) mn = min(mn, o);
        };
        if (from_list) {
          for (uint32_t k0 = 0; k0 < nl; k0 += 4 * 256) {
            uint32_t o[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const uint32_t x =
                  __hip_atomic_load(&lh[min(k0 + u * 256 + t, nl - 1)], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              o[u] = k0 + u * 256 + t < nl ? x : kNone;
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) visit(o[u] != kNone, o[u]);
          }
        } else {
          for (int r = 0; r < cb; ++r) {
            const size_t wr = (size_t)h * cb + r;
            for_pairs(pairs + wr * capw, pfill[wr], k_lo, span, visit);
          }
        }
        for (int off = 32; off > 0; off >>= 1) mn = min(mn, (uint32_t)__shfl_xor((int)mn, off));
        if (lane == 0 && mn != kNone) atomicMin(&s_x[3], mn);
        locate_ranks<256>(s_h, 1 << d, rem, rem, s_tot, s_bin, s_pos);
        const uint32_t b = s_bin[0];
        lt += (unsigned long long)(rem - s_pos[0]);
        rem = s_pos[0];
        P = (P << d) | b;
        if (last) {
          eq = s_h[b];
          next = s_bin[2] != kNone ? ((P & ~dmask) | s_bin[2]) : min(s_x[3], min2);
        }
        bits = nsh;
      }
    }
  }
  const double xlo = (double)key_to_float(k_lo + P);
  double xhi = xlo;
  if ((int64_t)(lt + eq) < lo + 2 && lo + 1 <= N - 1 && next != kNone) xhi = (double)key_to_float(k_lo + next);
  return phi_of(xlo, xhi, N, k_pct, alpha, lo);
}

__global__ __launch_bounds__(256) void cv_list_kernel(const float* __restrict__ A, int64_t N, CvState* st,
                                                      const uint32_t* __restrict__ hist0, uint32_t* __restrict__ hist1,
                                                      const uint2* __restrict__ pairs,
                                                      const uint32_t* __restrict__ pfill, uint32_t capw, int cb,
                                                      uint32_t* __restrict__ list, double k_pct, double alpha) {
  __shared__ uint32_t s_h[kBins];
  __shared__ int64_t s_tot[4];
  __shared__ uint32_t s_bin[3];
  __shared__ int64_t s_pos[2];
  __shared__ uint32_t s_min;
  __shared__ uint32_t s_stage[kListStage];
  __shared__ uint32_t s_nl, s_lbase;
  __shared__ uint32_t s_x[4];
  __shared__ int s_last;
  __shared__ uint32_t s_pre[kRegions + 1];
  const int h = blockIdx.y;
  const int t = threadIdx.x, lane = t & 63;
  CvState& S = st[h];
  if (!bracket_route(S, N)) {
    for (int i = t; i < kBins; i += 256) s_h[i] = 0;
    __syncthreads();
    uint32_t mn = kNone;
    hist_over_A(A + (size_t)h * N, N, s_h, 0u, 0u, 21, 0x7FFu, kNone, &mn);
    __syncthreads();
    flush_hist(s_h, hist1 + (size_t)h * kBins);
    return;
  }
  const int sh1 = S.shift1;
  const int nwg = sh1 == 0 ? 1 : (cb + kRegions - 1) / kRegions;
  if ((int)blockIdx.x >= nwg) return;
  const uint32_t k_lo = S.k_lo, span = S.k_hi - S.k_lo;
  const unsigned long long below = cv_below(S, N);
  const int64_t rem0 = S.rank - (int64_t)below;
  locate_ranks<256>(hist0 + (size_t)h * kBins, kBins, rem0, rem0, s_tot, s_bin, s_pos);
  const uint32_t b1 = s_bin[0], next1 = s_bin[2];
  const int64_t rem1 = s_pos[0];
  uint32_t* lh = list + (size_t)h * kListCap;
  if (sh1 > 0) {
    if (t == 0) {
      s_nl = 0;
      s_min = kNone;
    }
    __syncthreads();
    uint32_t mn = kNone;
    auto out = [&]() {             // the staged entries to the list, one reservation
      const uint32_t nst = s_nl;
      if (nst) {
        if (t == 0) s_lbase = atomicAdd(&S.n_list, nst);
        __syncthreads();
        // atomic writes: each entry is at the coherence point when it returns
        for (uint32_t i = t; i < nst; i += 256)
          if (s_lbase + i < (uint32_t)kListCap) atomicExch(&lh[s_lbase + i], s_stage[i]);
      }
      __syncthreads();
      if (t == 0) s_nl = 0;
      __syncthreads();
    };
    const int r0 = blockIdx.x * kRegions, nb = min(cb, r0 + kRegions) - r0;
    const size_t first = (size_t)h * cb + r0;
    const uint32_t total = buffer_prefix(pfill, first, nb, s_pre);
    for (uint32_t i0 = 0; i0 < total; i0 += 4 * 256) {   // the same trip count on every lane
      uint32_t o[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {   // every load issued (clamped), then used
        const uint32_t i = i0 + u * 256 + t;
        const uint32_t x = buffer_item(pairs, first, nb, capw, s_pre, min(i, total - 1))->x;
        o[u] = i < total ? (x | 0x80000000u) - k_lo : kNone;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const bool ok = o[u] <= span;
        const bool in = ok && (o[u] >> sh1) == b1;
        if (ok && (o[u] >> sh1) > b1) mn = min(mn, o[u]);
        const uint64_t bal = __builtin_amdgcn_ballot_w64(in);
        if (bal) {
          uint32_t base = 0;
          if (lane == 0) base = atomicAdd(&s_nl, (uint32_t)__builtin_popcountll(bal));
          base = __shfl(base, 0) + mbcnt(bal);
          if (in) s_stage[base] = o[u];
        }
      }
      __syncthreads();
      if (s_nl > (uint32_t)(kListStage - 4 * 256)) out();   // room for the next round
    }
    out();
    for (int off = 32; off > 0; off >>= 1) mn = min(mn, (uint32_t)__shfl_xor((int)mn, off));
    if (lane == 0 && mn != kNone) atomicMin(&s_min, mn);
    __syncthreads();
    if (t == 0 && s_min != kNone) atomicMin(&S.min2, s_min);
  }
  // arrival once this workgroup's list entries, minimum and count have all
  // completed (device-scope atomics, waited for); the last one takes Phi
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (t == 0) s_last = atomicAdd(&S.arrive_r, 1u) == (uint32_t)nwg - 1;
  __syncthreads();
  if (!s_last) return;
  const double phi = resolve_phi(S, hist0, lh, pairs, pfill, capw, cb, h, N, k_pct, alpha, b1, next1, rem1,
                                 below + (unsigned long long)(rem0 - rem1), s_h, s_tot, s_bin, s_pos, s_x);
  if (t == 0) S.phi = phi;
}

// ---------------------------------------------------------------------------
// 4. Bracket route: each column block counts its gathered values at or
//    above Phi per column (LDS counters): C_j, and the sums of C_j and
//    C_j^2.  Radix route: the second key digit over A.
// ---------------------------------------------------------------------------

constexpr int kColWin = 8192;      // columns counted in LDS at a time

__global__ __launch_bounds__(256) void cv_columns_kernel(const float* __restrict__ A, int64_t N, CvState* st,
                                                         const uint32_t* __restrict__ hist1,
                                                         uint32_t* __restrict__ hist2, const uint2* __restrict__ pairs,
                                                         const uint32_t* __restrict__ pfill, uint32_t capw, int nsub,
                                                         int n_colblk, int64_t cb_tokens,
                                                         int64_t n_keys) {
  __shared__ uint32_t s_e[kColWin];
  __shared__ uint32_t s_pre[kCvMaxSub + 1];
  __shared__ int64_t s_tot[4];
  __shared__ uint32_t s_bin[3];
  __shared__ int64_t s_pos[2];
  __shared__ unsigned long long s_red[4];
  const int h = blockIdx.y;
  const int t = threadIdx.x;
  CvState& S = st[h];
  if (!bracket_route(S, N)) {
    const int64_t rank = S.rank;
    locate_ranks<256>(hist1 + (size_t)h * kBins, kBins, rank, rank, s_tot, s_bin, s_pos);
    const uint32_t b0 = s_bin[0];
    if (blockIdx.x == 0 && t == 0) {
      S.fb_prefix[0] = b0 << 21;
      S.fb_rem[0] = s_pos[0];
      S.fb_lt[0] = (unsigned long long)(rank - s_pos[0]);
    }
    uint32_t* s_h = s_e;
    for (int i = t; i < kBins; i += 256) s_h[i] = 0;
    __syncthreads();
    uint32_t mn = kNone;
    hist_over_A(A + (size_t)h * N, N, s_h, 0xFFE00000u, b0 << 21, 10, 0x7FFu, kNone, &mn);
    __syncthreads();
    flush_hist(s_h, hist2 + (size_t)h * kBins);
    return;
  }
  // C_j of column block b's columns: its gathered values at or above Phi
  // (every entry there is one), counted per column in LDS, kColWin columns
  // at a time
  const double phi = S.phi;
  const int b = blockIdx.x;
  const int64_t c0 = (int64_t)b * cb_tokens, c1 = c0 + cb_tokens < n_keys ? c0 + cb_tokens : n_keys;
  const size_t first = ((size_t)h * n_colblk + b) * nsub;
  const uint32_t total = buffer_prefix(pfill, first, nsub, s_pre);
  unsigned long long a1 = 0, a2 = 0;
  for (int64_t w0 = c0; w0 < c1; w0 += kColWin) {
    const int nw = (int)std::min<int64_t>(kColWin, c1 - w0);
    __syncthreads();
    for (int i = t; i < nw; i += 256) s_e[i] = 0;
    __syncthreads();
    for (uint32_t i0 = 0; i0 < total; i0 += 4 * 256) {
      uint2 e[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)   // every load issued (clamped), then used
        e[u] = *buffer_item(pairs, first, nsub, capw, s_pre, min(i0 + u * 256 + t, total - 1));
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float x = __uint_as_float(e[u].x);
        const int64_t rel = (int64_t)e[u].y - w0;
        if (i0 + u * 256 + t < total && rel >= 0 && rel < nw && (double)x >= phi) atomicAdd(&s_e[rel], 1u);
      }
    }
    __syncthreads();
    for (int l = t; l < nw; l += 256) {
      const unsigned long long c = s_e[l];
      a1 += c;
      a2 += c * c;
    }
  }
  const unsigned long long t1 = block_sum256(a1, s_red);
  const unsigned long long t2 = block_sum256(a2, s_red);
  if (t == 0 && t1) {
    atomicAdd(&S.sum_c, t1);
    atomicAdd(&S.sum_c2, t2);
  }
}

// ---------------------------------------------------------------------------
// 5-6. Radix route: the last key digit over A (and the smallest key above
//      x_(lo)'s 22-bit bucket), then Phi, C_j over A and the score.  The
//      bracket route's score is written by the first of the two.
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void cv_digit2_kernel(const float* __restrict__ A, int64_t N, CvState* st,
                                                        const uint32_t* __restrict__ hist2,
                                                        uint32_t* __restrict__ hist3, int64_t n_keys,
                                                        float* __restrict__ cv_out) {
  __shared__ uint32_t s_h[kBins];
  __shared__ int64_t s_tot[4];
  __shared__ uint32_t s_bin[3];
  __shared__ int64_t s_pos[2];
  __shared__ uint32_t s_min;
  const int h = blockIdx.y;
  CvState& S = st[h];
  if (bracket_route(S, N)) {  // the bracket route's score, from the previous launch's sums
    if (blockIdx.x == 0 && threadIdx.x == 0) cv_out[h] = cv_value(S.sum_c, S.sum_c2, n_keys);
    return;
  }
  const int64_t rem0 = S.fb_rem[0];
  locate_ranks<256>(hist2 + (size_t)h * kBins, kBins, rem0, rem0, s_tot, s_bin, s_pos);
  const uint32_t prefix = S.fb_prefix[0] | (s_bin[0] << 10);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    S.fb_prefix[1] = prefix;
    S.fb_rem[1] = s_pos[0];
    S.fb_lt[1] = S.fb_lt[0] + (unsigned long long)(rem0 - s_pos[0]);
  }
  for (int i = threadIdx.x; i < kBins; i += 256) s_h[i] = 0;
  if (threadIdx.x == 0) s_min = kNone;
  __syncthreads();
  uint32_t mn = kNone;
  hist_over_A(A + (size_t)h * N, N, s_h, 0xFFFFFC00u, prefix, 0, 0x3FFu, prefix, &mn);
  for (int off = 32; off > 0; off >>= 1) mn = min(mn, (uint32_t)__shfl_xor((int)mn, off));
  if ((threadIdx.x & 63) == 0 && mn != kNone) atomicMin(&s_min, mn);
  __syncthreads();
  flush_hist(s_h, hist3 + (size_t)h * kBins);
  if (threadIdx.x == 0 && s_min != kNone) atomicMin(&S.fb_min, s_min);
}

__global__ __launch_bounds__(256) void cv_count_kernel(const float* __restrict__ A, int lq, int64_t n_keys,
                                                       CvState* st, const uint32_t* __restrict__ hist3, double k_pct,
                                                       double alpha, float* __restrict__ cv_out) {
  __shared__ int64_t s_tot[4];
  __shared__ uint32_t s_bin[3];
  __shared__ int64_t s_pos[2];
  __shared__ unsigned int s_c[4][64];
  __shared__ unsigned long long s_red[4];
  const int h = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  CvState& S = st[h];
  const int64_t N = (int64_t)lq * n_keys;
  if (bracket_route(S, N)) return;
  const int64_t lo = S.rank, rem1 = S.fb_rem[1];
  const uint32_t* hh = hist3 + (size_t)h * kBins;
  locate_ranks<256>(hh, 1024, rem1, rem1, s_tot, s_bin, s_pos);
  const uint32_t prefix = S.fb_prefix[1];
  const uint32_t xk = prefix | s_bin[0];
  const unsigned long long le = S.fb_lt[1] + (unsigned long long)(rem1 - s_pos[0]) + hh[s_bin[0]];
  const uint32_t above = s_bin[2] != kNone ? (prefix | s_bin[2]) : S.fb_min;
  const double xlo = (double)key_to_float(xk);
  double xhi = xlo;
  if ((int64_t)le < lo + 2 && lo + 1 <= N - 1 && above != kNone) xhi = (double)key_to_float(above);
  const double phi = phi_of(xlo, xhi, N, k_pct, alpha, lo);
  if (blockIdx.x == 0 && threadIdx.x == 0) S.phi = phi;
  const float* Ah = A + (size_t)h * lq * n_keys;
  const int rpg = (lq + 3) / 4;
  const int r0 = min(lq, wave * rpg), r1 = min(lq, r0 + rpg);
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
  const unsigned long long t1 = block_sum256(a1, s_red);
  const unsigned long long t2 = block_sum256(a2, s_red);
  if (threadIdx.x == 0) {
    if (t1) {
      atomicAdd(&S.fb_sum_c, t1);
      atomicAdd(&S.fb_sum_c2, t2);
    }
    arrive_and_finish(S, &S.fb_sum_c, &S.fb_sum_c2, n_keys, cv_out, h);
  }
}

// Gathered pairs: a sixteenth of A per head, split evenly over the waves of
// the column blocks (the union of bracket and Phi's range holds about 1-2%
// of A at the sample's margins; a wave's overflow sends the head the radix
// route).
uint32_t pair_cap(int64_t N, int64_t nbuf) {
  const int64_t c = std::max<int64_t>(64, ((N + 15) / 16 + nbuf - 1) / nbuf);
  return (uint32_t)((c + 3) & ~(int64_t)3);
}

struct CvLayout {
  size_t hist, list, samples, pairs, pfill, state, total;
};
size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }
CvLayout cv_layout(int hkv, int lq, int64_t n_keys, int n_colblk) {
  const int64_t N = (int64_t)lq * n_keys;
  const int64_t nbuf = (int64_t)n_colblk * kCvMaxSub;
  CvLayout L{};
  size_t o = 0;
  L.hist = o; o += al256((size_t)4 * hkv * kBins * sizeof(uint32_t));
  L.list = o; o += al256((size_t)hkv * kListCap * sizeof(uint32_t));
  L.samples = o; o += al256((size_t)hkv * kCvSamples * sizeof(float));
  L.pairs = o; o += al256((size_t)hkv * nbuf * pair_cap(N, nbuf) * sizeof(uint2));
  L.pfill = o; o += al256((size_t)hkv * nbuf * sizeof(uint32_t));
  L.state = o; o += al256((size_t)hkv * sizeof(CvState));
  L.total = o;
  return L;
}

}  // namespace

size_t cv_workspace_bytes(int hkv, int lq, int64_t n_keys, int n_colblk) {
  return cv_layout(hkv, lq, n_keys, n_colblk).total;
}

CvLink cv_link(void* ws, int hkv, int lq, int64_t n_keys, int n_colblk, int nsub) {
  const CvLayout L = cv_layout(hkv, lq, n_keys, n_colblk);
  char* w = reinterpret_cast<char*>(ws);
  CvLink c{};
  c.st = reinterpret_cast<CvState*>(w + L.state);
  c.samples = reinterpret_cast<float*>(w + L.samples);
  c.hist = reinterpret_cast<uint32_t*>(w + L.hist);
  c.hist0 = c.hist;
  c.list = reinterpret_cast<uint32_t*>(w + L.list);
  c.pairs = reinterpret_cast<uint2*>(w + L.pairs);
  c.pfill = reinterpret_cast<uint32_t*>(w + L.pfill);
  c.capw = pair_cap((int64_t)lq * n_keys, (int64_t)n_colblk * kCvMaxSub);
  c.nsub = nsub;
  return c;
}

hipError_t launch_cv_sample(const ScoreArgs& a, double k_pct, double alpha, hipStream_t stream) {
  const int64_t N = (int64_t)a.lq * a.n_keys;
  hipLaunchKernelGGL(cv_sample_kernel, dim3(a.hkv), dim3(kSampleThreads), 0, stream, a.cv.samples, N, k_pct, alpha,
                     a.cv.st, a.cv.hist, a.hkv);
  return hipGetLastError();
}

hipError_t launch_cv_finish(const ScoreArgs& a, double k_pct, double alpha, float* cv_out, hipStream_t stream) {
  const int hkv = a.hkv, lq = a.lq;
  const int64_t n_keys = a.n_keys, N = (int64_t)lq * n_keys;
  const CvLink& c = a.cv;
  const size_t hs = (size_t)hkv * kBins;
  uint32_t* hist = c.hist;
  const float* A = a.obs;
  const int nbuf = a.n_colblk * c.nsub;
  // radix-route passes over A: 128 workgroups per head (launches that only
  // return on the bracket route stay short)
  const unsigned hb = (unsigned)std::max<int64_t>(1, std::min<int64_t>(128, (N + 1023) / 1024));
  const unsigned lw = (unsigned)std::max<int64_t>(hb, (nbuf + kRegions - 1) / kRegions);
  const dim3 walk((unsigned)col_blocks(n_keys, hkv), hkv), flat(hb, hkv);
  hipLaunchKernelGGL(cv_list_kernel, dim3(lw, hkv), dim3(256), 0, stream, A, N, c.st, hist, hist + hs, c.pairs,
                     c.pfill, c.capw, nbuf, c.list, k_pct, alpha);
  hipLaunchKernelGGL(cv_columns_kernel, dim3((unsigned)a.n_colblk, hkv), dim3(256), 0, stream, A, N, c.st, hist + hs,
                     hist + 2 * hs, c.pairs, c.pfill, c.capw, c.nsub, a.n_colblk, a.cb_tokens, n_keys);
  hipLaunchKernelGGL(cv_digit2_kernel, flat, dim3(256), 0, stream, A, N, c.st, hist + 2 * hs, hist + 3 * hs, n_keys,
                     cv_out);
  hipLaunchKernelGGL(cv_count_kernel, walk, dim3(256), 0, stream, A, lq, n_keys, c.st, hist + 3 * hs, k_pct, alpha,
                     cv_out);
  return hipGetLastError();
}

}  // namespace catekv
