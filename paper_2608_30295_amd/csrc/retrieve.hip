// Query-aware retrieval in adaptive heads: the "all or query-aware"
// Retrieval(q, cache_k, cache_v) of Algorithm 1's decoding stage, with the
// page-based retrieval (Quest) that Section 4 integrates into the adaptive
// heads.  Pages are the cs-row chunks of a head's cache.
//
//   page bounds (once per cache):  kmin[p][j] = min over the page's rows of
//                                  K[t][j], kmax likewise
//   page score (every step):       max over the group's query heads g of
//                                  sum_j max(q_g[j] kmin[p][j], q_g[j] kmax[p][j]),
//                                  an upper bound of q_g . k over the page
//
// The pages with the largest scores go through the top-k of the selection
// path; compaction with a zero window then gathers their rows for decoding.
// Both kernels stream their inputs once (HBM-bound): 16-byte segments, one
// per lane, with the lanes of a row adjacent.
#include "common.h"
#include "internal.h"

#include <algorithm>

namespace catekv {

struct PageBoundsArgs {
  const void* k;          // [hkv][n][d]
  int64_t n;
  int cs;
  int64_t n_pages;
  int32_t heads[128];     // KV head per blockIdx.y
  void* kmin;             // [n_sel][n_pages][d]
  void* kmax;
};

struct PageScoreArgs {
  const void* q;          // [hq][d] of one sequence
  const void* kmin;       // [n_sel][n_pages][d]
  const void* kmax;
  int64_t n_pages;
  int32_t heads[128];
  float* scores;          // [n_sel][n_pages]
  uint32_t* zero_u32;     // cleared here for the top-k launch that follows, n_zero words
  int n_zero;
};

// 16 bytes as fp32 values (8 bf16 or 4 fp32) and back; bf16 <-> fp32 is exact
// in both directions for values that came from bf16.
template <typename T> struct Seg16;
template <> struct Seg16<uint16_t> {
  static constexpr int E = 8;
  __device__ static __forceinline__ void unpack(uint4 w, float* f) {
    const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) { f[2 * i] = bf16_lo(u[i]); f[2 * i + 1] = bf16_hi(u[i]); }
  }
  __device__ static __forceinline__ uint4 pack(const float* f) {
    uint32_t u[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) u[i] = (__float_as_uint(f[2 * i]) >> 16) | (__float_as_uint(f[2 * i + 1]) & 0xffff0000u);
    return make_uint4(u[0], u[1], u[2], u[3]);
  }
};
template <> struct Seg16<float> {
  static constexpr int E = 4;
  __device__ static __forceinline__ void unpack(uint4 w, float* f) {
    f[0] = __uint_as_float(w.x); f[1] = __uint_as_float(w.y); f[2] = __uint_as_float(w.z); f[3] = __uint_as_float(w.w);
  }
  __device__ static __forceinline__ uint4 pack(const float* f) {
    return make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]), __float_as_uint(f[3]));
  }
};

// One thread per (page, 16-byte segment); the segments of a row are adjacent
// threads, so each of the page's rows is read as one contiguous row.
template <typename T>
__global__ __launch_bounds__(256) void page_bounds_kernel(PageBoundsArgs a) {
  using S = Seg16<T>;
  constexpr int SEG = kD * (int)sizeof(T) / 16;
  constexpr size_t ROW = (size_t)kD * sizeof(T);
  const int sel = blockIdx.y;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t page = gid / SEG;
  const int seg = (int)(gid - page * SEG);
  if (page >= a.n_pages) return;
  const char* kh = reinterpret_cast<const char*>(a.k) + (size_t)a.heads[sel] * a.n * ROW + seg * 16;
  const int64_t r0 = page * a.cs;
  const int64_t r1 = min(r0 + (int64_t)a.cs, a.n);
  float mn[S::E], mx[S::E];
  S::unpack(ldg16(kh + (size_t)r0 * ROW), mn);
#pragma unroll
  for (int e = 0; e < S::E; ++e) mx[e] = mn[e];
  for (int64_t r = r0 + 1; r < r1; ++r) {
    float f[S::E];
    S::unpack(ldg16(kh + (size_t)r * ROW), f);
#pragma unroll
    for (int e = 0; e < S::E; ++e) { mn[e] = fminf(mn[e], f[e]); mx[e] = fmaxf(mx[e], f[e]); }
  }
  const size_t o = ((size_t)sel * a.n_pages + page) * ROW + seg * 16;
  *reinterpret_cast<uint4*>(reinterpret_cast<char*>(a.kmin) + o) = S::pack(mn);
  *reinterpret_cast<uint4*>(reinterpret_cast<char*>(a.kmax) + o) = S::pack(mx);
}

// SEG lanes per page (16 for bf16, 32 for fp32), 64 / SEG pages per wave per
// iteration; every lane holds its dims of the group's G query rows.
template <typename T, int G>
__global__ __launch_bounds__(256) void page_score_kernel(PageScoreArgs a) {
  using S = Seg16<T>;
  constexpr int SEG = kD * (int)sizeof(T) / 16;
  constexpr int PPW = 64 / SEG;
  constexpr size_t ROW = (size_t)kD * sizeof(T);
  const int sel = blockIdx.y;
  const int h = a.heads[sel];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int seg = lane % SEG, sub = lane / SEG;
  if (blockIdx.x == 0 && blockIdx.y == 0)
    for (int i = threadIdx.x; i < a.n_zero; i += blockDim.x) a.zero_u32[i] = 0;
  float qv[G][S::E];
#pragma unroll
  for (int g = 0; g < G; ++g)
    S::unpack(ldg16(reinterpret_cast<const char*>(a.q) + (size_t)(h * G + g) * ROW + seg * 16), qv[g]);
  const char* mnb = reinterpret_cast<const char*>(a.kmin) + (size_t)sel * a.n_pages * ROW + seg * 16;
  const char* mxb = reinterpret_cast<const char*>(a.kmax) + (size_t)sel * a.n_pages * ROW + seg * 16;
  const int64_t stride = (int64_t)gridDim.x * (blockDim.x / 64) * PPW;
  for (int64_t p0 = ((int64_t)blockIdx.x * (blockDim.x / 64) + wave) * PPW; p0 < a.n_pages; p0 += stride) {
    const int64_t page = p0 + sub;
    const bool ok = page < a.n_pages;
    float mn[S::E], mx[S::E];
    S::unpack(ldg16(mnb + (size_t)(ok ? page : 0) * ROW), mn);
    S::unpack(ldg16(mxb + (size_t)(ok ? page : 0) * ROW), mx);
    float best = -INFINITY;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < S::E; ++e) s += fmaxf(qv[g][e] * mn[e], qv[g][e] * mx[e]);
      s = sum16(s);
      if (SEG == 32) s = add_xor16(s);
      best = fmaxf(best, s);
    }
    if (seg == 0 && ok) a.scores[(size_t)sel * a.n_pages + page] = best;
  }
}

hipError_t launch_page_bounds(int dtype, const void* k, int64_t n, int cs, const int32_t* heads, int n_sel,
                              void* kmin, void* kmax, hipStream_t stream) {
  PageBoundsArgs a{};
  a.k = k; a.n = n; a.cs = cs;
  a.n_pages = (n + cs - 1) / cs;
  for (int i = 0; i < n_sel; ++i) a.heads[i] = heads[i];
  a.kmin = kmin; a.kmax = kmax;
  const int seg = dtype == CATEKV_BF16 ? 16 : 32;
  const unsigned nblk = (unsigned)((a.n_pages * seg + 255) / 256);
  if (dtype == CATEKV_BF16)
    hipLaunchKernelGGL(page_bounds_kernel<uint16_t>, dim3(nblk, n_sel), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(page_bounds_kernel<float>, dim3(nblk, n_sel), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_page_scores(int dtype, int G, const void* q, const void* kmin, const void* kmax,
                              int64_t n_pages, const int32_t* heads, int n_sel, float* scores,
                              uint32_t* zero_u32, int n_zero, hipStream_t stream) {
  PageScoreArgs a{};
  a.q = q; a.kmin = kmin; a.kmax = kmax; a.n_pages = n_pages; a.scores = scores;
  a.zero_u32 = zero_u32; a.n_zero = n_zero;
  for (int i = 0; i < n_sel; ++i) a.heads[i] = heads[i];
  const int ppb = 4 * (dtype == CATEKV_BF16 ? 4 : 2);      // pages per workgroup per iteration
  const unsigned nblk = (unsigned)std::min<int64_t>((n_pages + ppb - 1) / ppb, 1024);
#define CATEKV_PS(T, GG) \
  if (G == GG) { hipLaunchKernelGGL((page_score_kernel<T, GG>), dim3(nblk, n_sel), dim3(256), 0, stream, a); \
                 return hipGetLastError(); }
  if (dtype == CATEKV_BF16) {
    CATEKV_PS(uint16_t, 1) CATEKV_PS(uint16_t, 2) CATEKV_PS(uint16_t, 4) CATEKV_PS(uint16_t, 8)
  } else {
    CATEKV_PS(float, 1) CATEKV_PS(float, 2) CATEKV_PS(float, 4) CATEKV_PS(float, 8)
  }
#undef CATEKV_PS
  return hipErrorInvalidValue;
}

}  // namespace catekv
