// Per-head state of the CV score (Section 3.2, Eq. 2-4) shared by the
// kernels of csrc/cv.hip and the observation-matrix passes of score.h, and
// the workspace regions they exchange.  Device code only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace catekv {

constexpr int kCvBins = 2048;                 // radix and first-digit histograms
constexpr uint32_t kCvNone = 0xFFFFFFFFu;
constexpr int kCvListCap = 65536;             // entries of x_(lo)'s first-digit bin listed, at most
constexpr int kCvMaxSub = 16;                 // waves per score workgroup, at most

// The sample of A that brackets the quantile: 1024 runs of 8 consecutive
// entries spread evenly over the N entries (all of them when N <= 8192).
// Sample s = 8 t + u is entry t * stride + u in row-major order.
constexpr int kCvSampleRuns = 1024, kCvSampleRun = 8, kCvSamples = kCvSampleRuns * kCvSampleRun;
__host__ __device__ inline int64_t cv_sample_count(int64_t N) { return N < kCvSamples ? N : kCvSamples; }
__host__ __device__ inline int64_t cv_sample_stride(int64_t N) {
  return N < kCvSamples ? kCvSampleRun : (N / kCvSampleRuns) & ~(int64_t)(kCvSampleRun - 1);
}

// Ordered integer key of a float: key order is float order (-0 < +0).
__device__ __forceinline__ uint32_t cv_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float cv_key_float(uint32_t key) {
  return __uint_as_float((key & 0x80000000u) ? (key & 0x7FFFFFFFu) : ~key);
}

// LDS histogram update by a wave: the lanes that share the leading active
// lane's bin add with one atomic, the rest one by one.  act = ballot(valid).
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

struct CvState {                   // per KV head, in the workspace
  int64_t rank;                    // lo = floor((N - 1) k), 0-based
  uint32_t k_lo, k_hi;             // the bracket: ordered keys [k_lo, k_hi]
  float t_lo;                      // Phi >= t_lo (a float)
  int shift1;                      // (key - k_lo) >> shift1: first digit over the bracket
  uint32_t phi_over;               // a wave's gathered pairs overflowed its buffer
  unsigned long long n_cand;       // entries inside the bracket (from the pairs)
  unsigned long long ge_lo;        // entries at or above the bracket's bottom (all are pairs)
  unsigned long long sum_c, sum_c2;  // bracket route: sums of C_j and C_j^2 (from the pairs)
  double phi;
  uint32_t min2;                   // bracket route: smallest key offset above x_(lo)'s first-digit bin
  uint32_t n_list;                 // bracket route: entries of x_(lo)'s first-digit bin
  uint32_t arrive_r;               // bracket route: listing workgroups done
  uint32_t arrive_f;               // radix route: workgroups done in the launch that ends the head
  uint32_t fb_min;                 // radix route: smallest key above x_(lo)'s 22-bit bucket
  uint32_t fb_prefix[2];           // radix route: key prefix after the first and second digit
  int64_t fb_rem[2];               //   rank left inside that prefix
  unsigned long long fb_lt[2];     //   entries below that prefix
  unsigned long long fb_sum_c, fb_sum_c2;
};

// The first float above the bracket's keys.
__device__ __forceinline__ float cv_bracket_top(uint32_t k_hi) {
  const float f = k_hi == kCvNone ? INFINITY : cv_key_float(k_hi + 1);
  return f != f ? INFINITY : f;
}

// Entries below the bracket: N less those at or above its bottom, which are
// all among the pairs (valid for a head whose pairs all fit their buffers).
__device__ __forceinline__ unsigned long long cv_below(const CvState& S, int64_t N) {
  return (unsigned long long)N - S.ge_lo;
}

// The head takes the bracket route when every gathered pair fit its buffer
// and the bracket holds ranks lo and lo + 1 (lo only, when lo = N - 1).
// Decided alike by every launch after the pair count.
__device__ __forceinline__ bool cv_bracket_route(const CvState& S, int64_t N) {
  if (S.phi_over) return false;
  const int64_t lo = S.rank;
  const unsigned long long top = (unsigned long long)(lo + 1 <= N - 1 ? lo + 1 : lo);
  const unsigned long long below = cv_below(S, N);
  return below <= (unsigned long long)lo && top < below + S.n_cand;
}

// What the observation-matrix pass exchanges with the CV kernels.  Pairs
// (value bits, key column) of the entries at or above the lower of the
// bracket's bottom and t_lo go to wave w of column block b's own buffer,
// pairs + ((h * n_colblk + b) * nsub + w) * capw, its fill to
// pfill[(h * n_colblk + b) * nsub + w].
struct CvLink {
  CvState* st;                     // [hkv]
  float* samples;                  // [hkv][kCvSamples] sampled entries of A (from the row-statistics merge)
  uint32_t* hist0;                 // [hkv][kCvBins] first digit of key - k_lo of the bracket entries
  uint2* pairs;
  uint32_t* pfill;
  uint32_t capw;                   // pairs per wave buffer
  int nsub;                        // waves per column block (buffers per block)
  uint32_t* hist;                  // [4][hkv][kCvBins]: hist0, then the radix route's three digits
  uint32_t* list;                  // [hkv][kCvListCap] bracket entries of x_(lo)'s first-digit bin
};

}  // namespace catekv
