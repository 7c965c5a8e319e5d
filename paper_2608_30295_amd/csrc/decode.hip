// Hybrid-KV GQA decode attention (CateKV, Algorithm 1, decoding stage).
//
// Every (sequence, KV head) view -- a full cache for adaptive heads, a
// compact cache for consistent heads -- is cut into split-KV work items by
// the host plan.  One workgroup handles one item for all G query heads of
// the group, so each K/V row is read from HBM exactly once per step.
//
// Layout inside a wave: 8 lanes share one token row (each lane owns 16 of the
// 128 dims, fetched as 16-byte loads), so a wave covers 8 tokens per load
// instruction.  q.k partial sums are reduced over the 8 lanes with DPP.  Each
// group of 8 lanes keeps its own online-softmax state (running max m, sum l,
// unnormalised o); the states are merged across groups and waves at the end,
// and across items by the last-arriving workgroup of the view (atomic
// counter), which writes the normalised output and its log-sum-exp.
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
  for (int p = 0; p < Row<T>::NP; ++p) r.w[p] = ld16(row + (p * 8 + j) * Row<T>::NV);
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

// Merge `cnt` partial slots (stride SF floats) for output element (g, e):
// returns the merged unnormalised o, the sum l and the max m (natural-log units).
template <int G>
__device__ __forceinline__ void merge_slots(const float* src, int cnt, int g, int e, float& M,
                                            float& L, float& Ov) {
  constexpr int SF = G * kD + 2 * G;
  M = -INFINITY;
  for (int s = 0; s < cnt; ++s) M = fmaxf(M, src[s * SF + G * kD + g]);
  L = 0.f;
  Ov = 0.f;
  for (int s = 0; s < cnt; ++s) {
    const float ms = src[s * SF + G * kD + g];
    const float cw = ms == -INFINITY ? 0.f : fast_exp2((ms - M) * kLog2e);
    L += src[s * SF + G * kD + G + g] * cw;
    Ov += src[s * SF + g * kD + e] * cw;
  }
}

template <int G>
__device__ __forceinline__ void emit(float* out, float* lse, size_t row, int e, float M, float L, float Ov) {
  out[row * kD + e] = L > 0.f ? Ov / L : 0.f;
  if (lse && e == 0) lse[row] = L > 0.f ? M + logf(L) : -INFINITY;
}

template <int G>
__device__ __forceinline__ void put_slot(float* slot, int g, int e, float M, float L, float Ov) {
  slot[g * kD + e] = Ov;
  if (e == 0) {
    slot[G * kD + g] = L > 0.f ? M : -INFINITY;
    slot[G * kD + G + g] = L;
  }
}

template <typename T, int G, int WAVES, int U>
__global__ __launch_bounds__(WAVES * 64) void decode_kernel(DecodeArgs a) {
  constexpr int TOK_IT = 8 * U;                 // tokens per wave iteration
  constexpr int SF = G * kD + 2 * G;            // floats per partial slot
  constexpr int NT = WAVES * 64;
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

  const int ntok = t_end > t0 ? t_end - t0 : 0;
  const int n_it = (ntok + TOK_IT * WAVES - 1) / (TOK_IT * WAVES);
  // raw-unit slack before the running max is refreshed (2^8 headroom in p)
  const float thr = 8.0f / c;

  Row<T> kb[2][U], vb[2][U];
  auto issue = [&](int buf, int iter) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      int tok = t0 + (iter * WAVES + wave) * TOK_IT + u * 8 + gi;
      tok = tok < t_end ? tok : t0;               // masked rows re-read a valid row
      load_row(kb[buf][u], kbase + (size_t)tok * kD, j);
      load_row(vb[buf][u], vbase + (size_t)tok * kD, j);
    }
  };
  auto consume = [&](int buf, int iter) {
    float s[U][G];
    bool valid[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int tok = t0 + (iter * WAVES + wave) * TOK_IT + u * 8 + gi;
      valid[u] = tok < t_end;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float x = sum8(qf[g].dot(kb[buf][u]));
        s[u][g] = valid[u] ? x : -INFINITY;
      }
    }
    bool need = false;
    float mt[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      mt[g] = s[0][g];
#pragma unroll
      for (int u = 1; u < U; ++u) mt[g] = fmaxf(mt[g], s[u][g]);
      need |= mt[g] > m[g] + thr;
    }
    if (__builtin_amdgcn_ballot_w64(need)) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float nm = fmaxf(m[g], mt[g]);
        if (nm > m[g]) {
          const float corr = m[g] == -INFINITY ? 0.f : fast_exp2((m[g] - nm) * c);
          l[g] *= corr;
#pragma unroll
          for (int e = 0; e < 16; ++e) o[g][e] *= corr;
          m[g] = nm;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float vf[16];
      row_to_f32(vb[buf][u], vf);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float p = valid[u] ? fast_exp2(__builtin_fmaf(s[u][g], c, -m[g] * c)) : 0.f;
        l[g] += p;
#pragma unroll
        for (int e = 0; e < 16; ++e) o[g][e] = __builtin_fmaf(p, vf[e], o[g][e]);
      }
    }
  };

  if (n_it > 0) {
    issue(0, 0);
    for (int iter = 0; iter < n_it; iter += 2) {
      if (iter + 1 < n_it) issue(1, iter + 1);
      consume(0, iter);
      if (iter + 1 < n_it) {
        if (iter + 2 < n_it) issue(0, iter + 2);
        consume(1, iter + 1);
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
  __shared__ int s_flag;
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

  const ViewInfo vi = a.views[bh];
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
    if (vi.n_parts == 1) emit<G>(a.out, a.lse, row0 + g, e, Mn, L, Ov);
    else put_slot<G>(slot, g, e, Mn, L, Ov);
  }
  if (vi.n_parts == 1) return;

  // ---- level 1: the last item of a merge group merges the group -----------
  const int grp = it.part / kMergeGroup;
  const int g_first = grp * kMergeGroup;
  const int g_cnt = min(kMergeGroup, vi.n_parts - g_first);
  const bool single_group = vi.n_groups == 1;
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    int* ctr = single_group ? &a.counters[bh] : &a.counters[a.n_views + vi.gcounter + grp];
    s_flag = atomicAdd(ctr, 1) == g_cnt - 1;
    if (s_flag) *ctr = 0;                       // every member has arrived: reset for the next step
  }
  __syncthreads();
  if (!s_flag) return;
  __threadfence();
  const float* gsrc = a.slots + (size_t)(vi.first_slot + g_first) * SF;
  float* gdst = single_group ? nullptr : a.gslots + (size_t)(vi.first_gslot + grp) * SF;
  for (int t = threadIdx.x; t < G * kD; t += NT) {
    const int g = t / kD, e = t - g * kD;
    float M, L, Ov;
    merge_slots<G>(gsrc, g_cnt, g, e, M, L, Ov);
    if (single_group) emit<G>(a.out, a.lse, row0 + g, e, M, L, Ov);
    else put_slot<G>(gdst, g, e, M, L, Ov);
  }
  if (single_group) return;

  // ---- level 2: the last group of the view merges the group results -------
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    int* ctr = &a.counters[bh];
    s_flag = atomicAdd(ctr, 1) == vi.n_groups - 1;
    if (s_flag) *ctr = 0;
  }
  __syncthreads();
  if (!s_flag) return;
  __threadfence();
  const float* vsrc = a.gslots + (size_t)vi.first_gslot * SF;
  for (int t = threadIdx.x; t < G * kD; t += NT) {
    const int g = t / kD, e = t - g * kD;
    float M, L, Ov;
    merge_slots<G>(vsrc, vi.n_groups, g, e, M, L, Ov);
    emit<G>(a.out, a.lse, row0 + g, e, M, L, Ov);
  }
}

template <typename T, int G>
static hipError_t launch_t(const DecodeArgs& a, hipStream_t stream) {
  constexpr int WAVES = 4, U = 2;
  hipLaunchKernelGGL((decode_kernel<T, G, WAVES, U>), dim3(a.n_items), dim3(WAVES * 64), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_decode(int dtype, int G, const DecodeArgs& a, hipStream_t stream) {
#define CATEKV_DEC(T, GG) \
  if (G == GG) return launch_t<T, GG>(a, stream);
  if (dtype == CATEKV_BF16) {
    CATEKV_DEC(uint16_t, 1) CATEKV_DEC(uint16_t, 2) CATEKV_DEC(uint16_t, 4) CATEKV_DEC(uint16_t, 8)
  } else {
    CATEKV_DEC(float, 1) CATEKV_DEC(float, 2) CATEKV_DEC(float, 4) CATEKV_DEC(float, 8)
  }
#undef CATEKV_DEC
  return hipErrorInvalidValue;
}

}  // namespace catekv
