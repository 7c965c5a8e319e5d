// Hybrid-KV GQA decode attention (CateKV, Algorithm 1, decoding stage).
//
// Every (sequence, KV head) view -- a full cache for adaptive heads, a
// compact cache for consistent heads -- is cut into split-KV work items by
// the host plan.  One workgroup handles one item for all G query heads of
// the group, so each K/V row is read from HBM exactly once per step.
//
// Streaming kernel: 8 lanes share one token row (each lane owns 16 of the 128
// dims, fetched as 16-byte loads), so one wave covers 8 tokens per load
// instruction.  Loads run NS stages ahead of use in a register ring.  q.k
// partial sums are reduced over the 8 lanes with DPP; each group of 8 lanes
// keeps its own online-softmax state (running max m, sum l, unnormalised o),
// merged across groups and waves at the end.  An item that covers its whole
// view writes the normalised output directly; otherwise it writes a partial
// (o, m, l) that the combine kernel merges with the view's other partials
// (log-sum-exp weighting).  No cross-workgroup synchronisation is needed.
#include "common.h"
#include "internal.h"

namespace catekv {

template <typename T> struct Store;
template <> struct Store<uint16_t> { static constexpr int kNV = 8; };  // bf16 per 16 B
template <> struct Store<float> { static constexpr int kNV = 4; };     // fp32 per 16 B

// Lane j (0..7) of a token group owns, for piece p < NP, the NV elements
// starting at (p * 8 + j) * NV.  NP * NV = 16 dims per lane.
template <typename T>
struct Row {
  static constexpr int NV = Store<T>::kNV;
  static constexpr int NP = 16 / NV;
  uint4 w[NP];
};

template <typename T>
__device__ __forceinline__ void load_row(Row<T>& r, const T* row, int j) {
#pragma unroll
  for (int p = 0; p < Row<T>::NP; ++p) r.w[p] = ldg16(row + (p * 8 + j) * Row<T>::NV);
}

// 16 fp32 values of the row owned by this lane.
template <typename T>
__device__ __forceinline__ void row_to_f32(const Row<T>& r, float (&f)[16]);

template <>
__device__ __forceinline__ void row_to_f32<uint16_t>(const Row<uint16_t>& r, float (&f)[16]) {
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const uint32_t w[4] = {r.w[p].x, r.w[p].y, r.w[p].z, r.w[p].w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[p * 8 + 2 * i] = bf16_lo(w[i]);
      f[p * 8 + 2 * i + 1] = bf16_hi(w[i]);
    }
  }
}

template <>
__device__ __forceinline__ void row_to_f32<float>(const Row<float>& r, float (&f)[16]) {
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    f[p * 4 + 0] = __uint_as_float(r.w[p].x);
    f[p * 4 + 1] = __uint_as_float(r.w[p].y);
    f[p * 4 + 2] = __uint_as_float(r.w[p].z);
    f[p * 4 + 3] = __uint_as_float(r.w[p].w);
  }
}

// The query of one head restricted to the lane's 16 dims.
template <typename T> struct QFrag;

template <> struct QFrag<uint16_t> {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  bf16x2 w[8];
  __device__ __forceinline__ void load(const uint16_t* q, int j) {
    Row<uint16_t> r;
    load_row(r, q, j);
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      w[p * 4 + 0] = __builtin_bit_cast(bf16x2, r.w[p].x);
      w[p * 4 + 1] = __builtin_bit_cast(bf16x2, r.w[p].y);
      w[p * 4 + 2] = __builtin_bit_cast(bf16x2, r.w[p].z);
      w[p * 4 + 3] = __builtin_bit_cast(bf16x2, r.w[p].w);
    }
  }
  // partial q.k over the lane's dims: bf16 pair products accumulated in fp32
  __device__ __forceinline__ float dot(const Row<uint16_t>& k) const {
    float acc = 0.f;
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, k.w[p].x), w[p * 4 + 0], acc, false);
      acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, k.w[p].y), w[p * 4 + 1], acc, false);
      acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, k.w[p].z), w[p * 4 + 2], acc, false);
      acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, k.w[p].w), w[p * 4 + 3], acc, false);
    }
    return acc;
  }
};

template <> struct QFrag<float> {
  float w[16];
  __device__ __forceinline__ void load(const float* q, int j) {
    Row<float> r;
    load_row(r, q, j);
    row_to_f32(r, w);
  }
  __device__ __forceinline__ float dot(const Row<float>& k) const {
    float f[16];
    row_to_f32(k, f);
    float acc = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) acc = __builtin_fmaf(w[e], f[e], acc);
    return acc;
  }
};

// dim index of element e (0..15) of lane j
template <typename T>
__device__ __forceinline__ int dim_of(int j, int e) {
  constexpr int NV = Store<T>::kNV;
  return ((e / NV) * 8 + j) * NV + (e % NV);
}

template <typename T, int G, int WAVES, int NS>
__global__ __launch_bounds__(WAVES * 64) void decode_split_kernel(DecodeArgs a) {
  constexpr int SF = G * kD + 2 * G;            // floats per partial slot
  constexpr int NT = WAVES * 64;
  constexpr int TPW = 8;                        // tokens per wave per stage
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int j = lane & 7;                       // lane within the token group
  const int gi = lane >> 3;                     // token group within the wave

  const DecodeItem it = a.items[blockIdx.x];
  const int bh = it.bh;
  const int hkv = a.hkv;
  const int b = bh / hkv, h = bh - b * hkv;
  const catekv_kv_ptrs view = a.kv[bh];
  int64_t len = a.lens[bh];
  const ViewInfo vi = a.views[bh];
  len = len < 0 ? 0 : len;
  const int t0 = it.t0;
  const int t_end = (int)((int64_t)it.t1 < len ? (int64_t)it.t1 : len);
  const T* kbase = reinterpret_cast<const T*>(view.k);
  const T* vbase = reinterpret_cast<const T*>(view.v);
  const float scale = a.scale;
  const float c = scale * kLog2e;               // raw dot -> log2 units

  QFrag<T> qf[G];
  const int hq = hkv * G;
  const T* qb = reinterpret_cast<const T*>(a.q);
#pragma unroll
  for (int g = 0; g < G; ++g) qf[g].load(qb + ((size_t)b * hq + (size_t)h * G + g) * kD, j);

  float m[G], l[G], o[G][16];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -INFINITY;
    l[g] = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) o[g][e] = 0.f;
  }

  // stage s of wave w covers tokens t0 + (s * WAVES + w) * 8 + [0, 8)
  const int ntok = t_end > t0 ? t_end - t0 : 0;
  const int n_st = (ntok + TPW * WAVES - 1) / (TPW * WAVES);
  const float thr = 8.0f / c;                   // raw-unit slack before the running max is refreshed

  Row<T> kb[NS], vb[NS];
  auto issue = [&](int buf, int st) {
    int tok = t0 + (st * WAVES + wave) * TPW + gi;
    tok = tok < t_end ? tok : t0;               // rows past the end re-read a valid row
    load_row(kb[buf], kbase + (size_t)tok * kD, j);
    load_row(vb[buf], vbase + (size_t)tok * kD, j);
  };
  auto consume = [&](int buf, int st) {
    const int tok = t0 + (st * WAVES + wave) * TPW + gi;
    const bool valid = tok < t_end;
    float s[G];
    bool need = false;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float x = sum8(qf[g].dot(kb[buf]));
      s[g] = valid ? x : -INFINITY;
      need |= s[g] > m[g] + thr;
    }
    if (__builtin_amdgcn_ballot_w64(need)) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float nm = fmaxf(m[g], s[g]);
        if (nm > m[g]) {
          const float corr = m[g] == -INFINITY ? 0.f : fast_exp2((m[g] - nm) * c);
          l[g] *= corr;
#pragma unroll
          for (int e = 0; e < 16; ++e) o[g][e] *= corr;
          m[g] = nm;
        }
      }
    }
    float vf[16];
    row_to_f32(vb[buf], vf);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float p = valid ? fast_exp2(__builtin_fmaf(s[g], c, -m[g] * c)) : 0.f;
      l[g] += p;
#pragma unroll
      for (int e = 0; e < 16; ++e) o[g][e] = __builtin_fmaf(p, vf[e], o[g][e]);
    }
  };

  if (n_st > 0) {
#pragma unroll
    for (int s = 0; s < NS - 1; ++s)
      if (s < n_st) issue(s, s);
    for (int base = 0; base < n_st; base += NS) {
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const int st = base + s;
        if (st < n_st) {
          if (st + NS - 1 < n_st) issue((s + NS - 1) % NS, st + NS - 1);
          consume(s, st);
        }
      }
    }
  }

  // ---- merge the 8 token groups of the wave (lanes l, l^8, l^16, l^32) ----
#pragma unroll
  for (int g = 0; g < G; ++g) {
    float M = m[g];
    M = fmaxf(M, shfl_xor(M, 8));
    M = fmaxf(M, shfl_xor(M, 16));
    M = fmaxf(M, shfl_xor(M, 32));
    const float corr = m[g] == -INFINITY ? 0.f : fast_exp2((m[g] - M) * c);
    float lg = l[g] * corr;
    lg += shfl_xor(lg, 8);
    lg += shfl_xor(lg, 16);
    lg += shfl_xor(lg, 32);
    l[g] = lg;
    m[g] = M;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      float x = o[g][e] * corr;
      x += shfl_xor(x, 8);
      x += shfl_xor(x, 16);
      x += shfl_xor(x, 32);
      o[g][e] = x;
    }
  }

  // ---- merge the waves through LDS -----------------------------------------
  __shared__ float s_o[WAVES][G][kD];
  __shared__ float s_m[WAVES][G], s_l[WAVES][G];
  if (gi == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
#pragma unroll
      for (int e = 0; e < 16; ++e) s_o[wave][g][dim_of<T>(j, e)] = o[g][e];
      if (j == 0) {
        s_m[wave][g] = m[g];
        s_l[wave][g] = l[g];
      }
    }
  }
  __syncthreads();

  const size_t row0 = (size_t)b * hq + (size_t)h * G;
  float* slot = a.slots + (size_t)(vi.first_slot + it.part) * SF;
  for (int t = threadIdx.x; t < G * kD; t += NT) {
    const int g = t / kD, e = t - g * kD;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) M = fmaxf(M, s_m[w][g]);
    float L = 0.f, Ov = 0.f;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) {
      const float cw = s_m[w][g] == -INFINITY ? 0.f : fast_exp2((s_m[w][g] - M) * c);
      L += s_l[w][g] * cw;
      Ov += s_o[w][g][e] * cw;
    }
    const float Mn = M * scale;                 // natural-log units of the scaled score
    if (vi.n_parts == 1) {
      a.out[(row0 + g) * kD + e] = L > 0.f ? Ov / L : 0.f;
      if (a.lse && e == 0) a.lse[row0 + g] = L > 0.f ? Mn + logf(L) : -INFINITY;
    } else {
      slot[g * kD + e] = Ov;
      if (e == 0) {
        slot[G * kD + g] = L > 0.f ? Mn : -INFINITY;
        slot[G * kD + G + g] = L;
      }
    }
  }
}

// Merges the partials of every view cut into more than one item.  One
// workgroup per (view, query head of the group): all (m, l) pairs go to LDS,
// then 8 lanes of parts x 128 dims accumulate the weighted o.
constexpr int kCombineThreads = 1024;
constexpr int kCombineLanes = kCombineThreads / kD;   // parts handled in parallel per dim
constexpr int kCombineMaxParts = 4096;

template <int G>
__global__ __launch_bounds__(kCombineThreads) void decode_combine_kernel(DecodeArgs a) {
  constexpr int SF = G * kD + 2 * G;
  const int bh = blockIdx.x / G, g = blockIdx.x - (blockIdx.x / G) * G;
  const ViewInfo vi = a.views[bh];
  const int P = vi.n_parts;
  if (P <= 1) return;
  __shared__ float s_w[kCombineMaxParts];
  __shared__ float s_red[kCombineThreads / 64];
  __shared__ float s_acc[kCombineLanes][kD];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const float* base = a.slots + (size_t)vi.first_slot * SF;

  // global max of the parts' m
  float M = -INFINITY;
  for (int s = t; s < P; s += kCombineThreads) {
    const float ms = base[(size_t)s * SF + G * kD + g];
    s_w[s] = ms;
    M = fmaxf(M, ms);
  }
  for (int off = 32; off > 0; off >>= 1) M = fmaxf(M, shfl_xor(M, off));
  if (lane == 0) s_red[wave] = M;
  __syncthreads();
  M = s_red[0];
#pragma unroll
  for (int w = 1; w < kCombineThreads / 64; ++w) M = fmaxf(M, s_red[w]);
  __syncthreads();
  // weights w_s = exp(m_s - M) and L = sum w_s l_s
  float L = 0.f;
  for (int s = t; s < P; s += kCombineThreads) {
    const float ms = s_w[s];
    const float w = ms == -INFINITY ? 0.f : fast_exp2((ms - M) * kLog2e);
    s_w[s] = w;
    L += w * base[(size_t)s * SF + G * kD + G + g];
  }
  for (int off = 32; off > 0; off >>= 1) L += shfl_xor(L, off);
  if (lane == 0) s_red[wave] = L;
  __syncthreads();
  L = 0.f;
#pragma unroll
  for (int w = 0; w < kCombineThreads / 64; ++w) L += s_red[w];

  // o = sum_s w_s o_s
  const int e = t % kD, pl = t / kD;
  float acc = 0.f;
  constexpr int UNR = 8;
  for (int s0 = pl; s0 < P; s0 += kCombineLanes * UNR) {
    float v[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int s = s0 + u * kCombineLanes;
      v[u] = s < P ? base[(size_t)s * SF + g * kD + e] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int s = s0 + u * kCombineLanes;
      acc += s < P ? s_w[s] * v[u] : 0.f;
    }
  }
  s_acc[pl][e] = acc;
  __syncthreads();
  if (t < kD) {
    float o = 0.f;
#pragma unroll
    for (int p = 0; p < kCombineLanes; ++p) o += s_acc[p][t];
    const int hkv = a.hkv, b = bh / hkv, h = bh - b * hkv;
    const size_t row = (size_t)b * hkv * G + (size_t)h * G + g;
    a.out[row * kD + t] = L > 0.f ? o / L : 0.f;
    if (a.lse && t == 0) a.lse[row] = L > 0.f ? M + logf(L) : -INFINITY;
  }
}

template <typename T, int G>
static hipError_t launch_t(const DecodeArgs& a, bool combine, hipStream_t stream) {
  constexpr int WAVES = 4, NS = 4;
  hipLaunchKernelGGL((decode_split_kernel<T, G, WAVES, NS>), dim3(a.n_items), dim3(WAVES * 64), 0, stream, a);
  if (combine)
    hipLaunchKernelGGL((decode_combine_kernel<G>), dim3(a.n_views * G), dim3(kCombineThreads), 0, stream, a);
  return hipGetLastError();
}

int decode_max_parts() { return kCombineMaxParts; }

hipError_t launch_decode(int dtype, int G, const DecodeArgs& a, bool combine, hipStream_t stream) {
#define CATEKV_DEC(T, GG) \
  if (G == GG) return launch_t<T, GG>(a, combine, stream);
  if (dtype == CATEKV_BF16) {
    CATEKV_DEC(uint16_t, 1) CATEKV_DEC(uint16_t, 2) CATEKV_DEC(uint16_t, 4) CATEKV_DEC(uint16_t, 8)
  } else {
    CATEKV_DEC(float, 1) CATEKV_DEC(float, 2) CATEKV_DEC(float, 4) CATEKV_DEC(float, 8)
  }
#undef CATEKV_DEC
  return hipErrorInvalidValue;
}

}  // namespace catekv
