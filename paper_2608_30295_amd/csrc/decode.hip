// Hybrid-KV GQA decode attention (CateKV, Algorithm 1, decoding stage).
//
// Every (sequence, KV head) view -- a full cache for adaptive heads, a
// compact cache for consistent heads -- is a run of tokens.  The host plan
// lays all views end to end and cuts the run into equal shares, one per
// persistent workgroup (stream-K), so long adaptive views and short
// consistent views balance across CUs.  A workgroup streams the 1-3
// segments of its share for all G query heads of the group, so each K/V row
// is read from HBM exactly once per step.
//
// Streaming: 8 lanes share one token row (each lane owns 16 of the 128 dims,
// fetched as 16-byte global loads), so one wave covers 8 tokens per load
// instruction; loads run NS stages ahead of use in a register ring.  q.k
// partial sums are reduced over the 8 lanes with DPP; each group of 8 lanes
// keeps its own online-softmax state (running max m, sum l, unnormalised o),
// merged across groups and waves at the end of a segment.  A segment that
// covers its whole view writes the normalised output and log-sum-exp;
// otherwise it writes a partial (o, m, l), and the combine kernel merges the
// partials of each such view (log-sum-exp weighting) right after.
#include "common.h"
#include "internal.h"

#include <type_traits>

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

// ---- partials ----------------------------------------------------------------
// A segment that does not cover its whole view stores (o, m, l) in its slot
// with plain stores; the combine kernel, launched right after on the same
// stream, sees them complete at the kernel boundary.
template <int G>
__device__ __forceinline__ void put_slot(float* slot, int g, int e, float M, float L, float Ov) {
  slot[g * kD + e] = Ov;
  if (e == 0) {
    slot[G * kD + g] = L > 0.f ? M : -INFINITY;
    slot[G * kD + G + g] = L;
  }
}

__device__ __forceinline__ void emit(float* out, float* lse, size_t row, int e, float M, float L, float Ov) {
  out[row * kD + e] = L > 0.f ? Ov / L : 0.f;
  if (lse && e == 0) lse[row] = L > 0.f ? M + logf(L) : -INFINITY;
}

// Persistent stream-K worker: workgroup w streams segments
// [worker_seg[w], worker_seg[w + 1]) of the plan, each a token range of one view.
template <typename T, int G, int WAVES, int NS>
__global__ __launch_bounds__(WAVES * 64) void decode_stream_kernel(DecodeArgs a) {
  constexpr int SF = G * kD + 2 * G;            // floats per partial slot
  constexpr int NT = WAVES * 64;
  constexpr int TPW = 8;                        // tokens per wave per stage
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int j = lane & 7;                       // lane within the token group
  const int gi = lane >> 3;                     // token group within the wave
  const int hkv = a.hkv, hq = hkv * G;
  const float scale = a.scale;
  const float c = scale * kLog2e;               // raw dot -> log2 units
  const float thr = 8.0f / c;                   // raw-unit slack before the running max is refreshed

  __shared__ float s_o[WAVES][G][kD];
  __shared__ float s_m[WAVES][G], s_l[WAVES][G];

  const int seg_lo = a.worker_seg[blockIdx.x], seg_hi = a.worker_seg[blockIdx.x + 1];
  for (int sg = seg_lo; sg < seg_hi; ++sg) {
    const DecodeItem it = a.items[sg];
    const int bh = it.bh;
    const int b = bh / hkv, h = bh - b * hkv;
    const catekv_kv_ptrs view = a.kv[bh];
    int64_t len = a.lens[bh];
    const ViewInfo vi = a.views[bh];
    len = len < 0 ? 0 : len;
    const int t0 = it.t0;
    const int t_end = (int)((int64_t)it.t1 < len ? (int64_t)it.t1 : len);
    const T* kbase = reinterpret_cast<const T*>(view.k);
    const T* vbase = reinterpret_cast<const T*>(view.v);

    QFrag<T> qf[G];
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

    Row<T> kb[NS], vb[NS];
    auto issue = [&](int buf, int st) {
      int tok = t0 + (st * WAVES + wave) * TPW + gi;
      tok = tok < t_end ? tok : t0;             // rows past the end re-read a valid row
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

    // Loads are issued unconditionally (stages past the end re-read row t0,
    // which is cached) so that every wait in the ring is a static count and
    // the NS - 1 stages ahead stay in flight.
    if (n_st > 0) {
      const int n_pad = (n_st + NS - 1) / NS * NS;
#pragma unroll
      for (int s = 0; s < NS - 1; ++s) issue(s, s);
      for (int base = 0; base < n_pad; base += NS) {
#pragma unroll
        for (int s = 0; s < NS; ++s) {
          issue((s + NS - 1) % NS, base + s + NS - 1);
          consume(s, base + s);
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

    // ---- merge the waves through LDS ---------------------------------------
    __syncthreads();                            // LDS of the previous segment is free
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
      const float Mn = M * scale;               // natural-log units of the scaled score
      if (vi.n_parts == 1) emit(a.out, a.lse, row0 + g, e, Mn, L, Ov);
      else put_slot<G>(slot, g, e, Mn, L, Ov);
    }
  }
}

// ---- bf16 storage: the contraction runs on MFMA -----------------------------
// Per wave and stage, a tile of 16 tokens:
//  * S^T = K Q^T with v_mfma_f32_16x16x32_bf16: A = the K tile (lane l holds
//    token l % 16, dims [32 ks + 8 (l / 16), +8) for k-step ks), B = Q^T with
//    the G heads as columns (zero columns past G).  The result puts the score
//    of token 4 k + r and head j in lane j + 16 k, register r.
//  * Those lanes and registers are exactly the A operand of
//    v_mfma_f32_16x16x4_f32 for the token group {4 k + r : k < 4} (A[head][k]),
//    so P = exp(S - m) needs no data movement.  B is V in its natural row
//    layout: lane l holds token 4 (l / 16) + r, dims [8 (l % 16), +8), and
//    register e of that row feeds the product for dims 8 n + e.
//  * O accumulates in 8 tiles (one per e): head i, dim 8 n + e sits in lane
//    n + 16 (i / 4), register i % 4.
// The running max of a head is kept equal across the four lanes that hold
// its tokens, so every product that accumulates into O uses the same scale.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
constexpr float kDecodeMFloor = -1e30f;

template <int G, int WAVES, int NS>
__global__ __launch_bounds__(WAVES * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
void decode_stream_mfma_kernel(DecodeArgs a) {
  static_assert(G <= 16, "heads of a group must fit the 16 MFMA columns");
  constexpr int SF = G * kD + 2 * G;
  constexpr int NT = WAVES * 64;
  constexpr int TPW = 16;                       // tokens per wave per stage
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int n16 = lane & 15, k4 = lane >> 4;
  const int hkv = a.hkv, hq = hkv * G;
  const float scale = a.scale;
  const float c = scale * kLog2e;
  const float thr = 8.0f / c;
  const bool head_lane = n16 < G;               // lanes whose column is a real head

  __shared__ float s_o[WAVES][G][kD];
  __shared__ float s_m[WAVES][G], s_l[WAVES][G];

  const int seg_lo = a.worker_seg[blockIdx.x], seg_hi = a.worker_seg[blockIdx.x + 1];
  for (int sg = seg_lo; sg < seg_hi; ++sg) {
    const DecodeItem it = a.items[sg];
    const int bh = it.bh;
    const int b = bh / hkv, h = bh - b * hkv;
    const catekv_kv_ptrs view = a.kv[bh];
    int64_t len = a.lens[bh];
    const ViewInfo vi = a.views[bh];
    len = len < 0 ? 0 : len;
    const int t0 = it.t0;
    const int t_end = (int)((int64_t)it.t1 < len ? (int64_t)it.t1 : len);
    const char* kbase = reinterpret_cast<const char*>(view.k);
    const char* vbase = reinterpret_cast<const char*>(view.v);

    // B operand of S^T: head n16's dims [32 ks + 8 k4, +8)
    uint4 qb[4];
    {
      const char* qrow = reinterpret_cast<const char*>(a.q) +
                         ((size_t)b * hq + (size_t)h * G + (head_lane ? n16 : 0)) * kD * 2;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const uint4 v = ldg16(qrow + ks * 64 + k4 * 16);
        qb[ks] = head_lane ? v : make_uint4(0, 0, 0, 0);
      }
    }

    f32x4_t O[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) O[e] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    // a finite floor keeps exp2(s c - m c) = 0 for masked tokens (s = -inf) even
    // before the first valid token; +inf makes p = 0 on padding columns
    float m = head_lane ? kDecodeMFloor : INFINITY;
    float l = 0.f;

    const int ntok = t_end > t0 ? t_end - t0 : 0;
    const int n_units = (ntok + TPW - 1) / TPW;   // 16-token units of the segment

    // wave w takes units w, w + WAVES, w + 2 WAVES, ... (unit numbers ride
    // along the prefetch ring)
    int st_ctr = 0;
    auto grab = [&]() -> int { return (st_ctr++) * WAVES + wave; };
    int unit[NS];

    uint4 kb[NS][4], vb[NS][4];
    auto issue = [&](int buf, int un) {
      const int tile = t0 + un * TPW;
      int tk = tile + n16;
      tk = tk < t_end ? tk : t0;                  // rows past the end re-read row t0
      const char* kr = kbase + (size_t)tk * (kD * 2) + k4 * 16;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) kb[buf][ks] = ldg16(kr + ks * 64);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        int tv = tile + 4 * k4 + r;
        tv = tv < t_end ? tv : t0;
        vb[buf][r] = ldg16(vbase + (size_t)tv * (kD * 2) + n16 * 16);
      }
    };
    auto consume = [&](int buf, int un) {
      const int tile = t0 + un * TPW;
      f32x4_t S = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        S = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kb[buf][ks]),
                                                    __builtin_bit_cast(bf16x8_t, qb[ks]), S, 0, 0, 0);
      float sv[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) sv[r] = tile + 4 * k4 + r < t_end ? S[r] : -INFINITY;
      float mx = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
      mx = fmaxf(mx, shfl_xor(mx, 16));
      mx = fmaxf(mx, shfl_xor(mx, 32));
      const bool need = head_lane && mx > m + thr;
      if (__builtin_amdgcn_ballot_w64(need)) {
        // refresh the running max of every head that needs it; rescale l and O
        float corr = 1.f;
        if (head_lane && mx > m) {
          corr = fast_exp2((m - mx) * c);       // 0 while m is still the floor
          m = mx;
        }
        l *= corr;
        // O register r of lane L belongs to head 4 (L / 16) + r: fetch that head's corr
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int src = (4 * k4 + r) & 15;
          const float cr = __int_as_float(__builtin_amdgcn_ds_bpermute(src << 2, __float_as_int(corr)));
#pragma unroll
          for (int e = 0; e < 8; ++e) O[e][r] *= cr;
        }
      }
      const float mc = m * c;
      f32x4_t P;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        P[r] = fast_exp2(__builtin_fmaf(sv[r], c, -mc));
        l += P[r];
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const uint32_t w[4] = {vb[buf][r].x, vb[buf][r].y, vb[buf][r].z, vb[buf][r].w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          O[2 * i] = __builtin_amdgcn_mfma_f32_16x16x4f32(P[r], bf16_lo(w[i]), O[2 * i], 0, 0, 0);
          O[2 * i + 1] = __builtin_amdgcn_mfma_f32_16x16x4f32(P[r], bf16_hi(w[i]), O[2 * i + 1], 0, 0, 0);
        }
      }
    };

    if (n_units > 0) {
      // units past the end re-read row t0 (cached) and contribute nothing
#pragma unroll
      for (int s = 0; s < NS - 1; ++s) {
        unit[s] = grab();
        issue(s, unit[s]);
      }
      bool more = true;
      while (more) {
#pragma unroll
        for (int s = 0; s < NS; ++s) {
          const int nb = (s + NS - 1) % NS;
          unit[nb] = grab();
          issue(nb, unit[nb]);
          if (unit[s] < n_units) consume(s, unit[s]);
          else more = false;
        }
      }
    }

    // l of a head is spread over its four lanes (one per token quarter)
    l += shfl_xor(l, 16);
    l += shfl_xor(l, 32);

    __syncthreads();                            // LDS of the previous segment is free
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int head = 4 * k4 + r;
      if (head < G) {
#pragma unroll
        for (int e = 0; e < 8; ++e) s_o[wave][head][8 * n16 + e] = O[e][r];
      }
    }
    if (lane < G) {
      s_m[wave][lane] = m;
      s_l[wave][lane] = l;
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
      const float Mn = M * scale;
      if (vi.n_parts == 1) emit(a.out, a.lse, row0 + g, e, Mn, L, Ov);
      else put_slot<G>(slot, g, e, Mn, L, Ov);
    }
  }
}

// ---- bf16 storage, one 8-wave workgroup per compute unit ---------------------
// The same contraction layout as above, with three changes:
//  * All segments of the worker are described once, at the start, in an LDS
//    table (view pointers, token range, output row or partial slot, and the
//    group's query rows), so no descriptor load sits between two tiles.
//  * Each wave's tiles (tile u of a segment goes to wave u % 8) form one
//    continuous stream across the worker's segments: the load of the next tile
//    is issued before the current one is used even when the next tile belongs
//    to the next segment.
//  * At the end of a segment the eight waves merge their (m, l, O) through LDS
//    after a barrier that waits only for LDS operations, so the loads already
//    in flight keep streaming; a wave with no tile in a segment contributes an
//    empty state.  The LDS merge area is double-buffered by segment parity.
// P V runs on v_mfma_f32_16x16x16_bf16 with P split into a bf16 high part and
// a bf16 remainder (P = hi + lo up to 2^-18 relative; the bf16 products are
// exact in the fp32 accumulator).  The score tile's lanes and registers are
// already that instruction's A operand (head = lane % 16, token 4 (lane / 16)
// + i); the B operand of product e takes dim 8 (lane % 16) + e of the four
// token rows a lane loaded, so O keeps the layout of the fp32 path.
constexpr int kV2Waves = 8;
constexpr int kV2MaxSeg = kDecodeV2MaxSeg;   // segments per worker held in the LDS table

struct V2Seg {
  const char* k;
  const char* v;
  int32_t t0, t_end, n_units, row0, slot;
};

// Views whose K/V pointers and lengths every workgroup reads into LDS at the
// start, side by side with its own segment list (larger batches read them
// per segment, one load later).
constexpr int kV2PreViews = 256;

typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// bf16 pair (RNE) of two fp32 values, as one 32-bit word (x in the low half)
__device__ __forceinline__ uint32_t pack_bf16(float x, float y) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{x, y}), bf16x2_t));
}

template <int G>
__global__ __launch_bounds__(kV2Waves * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
void decode_stream_v2_kernel(DecodeArgs a) {
  static_assert(G <= 16, "heads of a group must fit the 16 MFMA columns");
  constexpr int WAVES = kV2Waves;
  constexpr int NT = WAVES * 64;
  constexpr int SF = G * kD + 2 * G;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int n16 = lane & 15, k4 = lane >> 4;
  const int hkv = a.hkv, hq = hkv * G;
  const float scale = a.scale;
  const float c = scale * kLog2e;
  const float thr = 8.0f / c;
  const bool head_lane = n16 < G;

  __shared__ V2Seg s_seg[kV2MaxSeg];
  __shared__ uint4 s_q[kV2MaxSeg][G][16];       // per segment: G query rows of 16 x 16 bytes
  __shared__ float s_o[2][WAVES][G][kD];
  __shared__ float s_ml[2][WAVES][2][G];
  __shared__ catekv_kv_ptrs s_kv[kV2PreViews];
  __shared__ int64_t s_len[kV2PreViews];

  // Start-up: the segment list with the worker's segment count and (small
  // batches) every view's pointers and length are independent loads, all
  // issued before the first wait; the query rows follow one load later.
  const int nv = a.n_views;
  const bool pre = nv <= kV2PreViews;
  const V2Item it = a.v2items[(size_t)blockIdx.x * kV2MaxSeg +
                              ((int)threadIdx.x < kV2MaxSeg ? (int)threadIdx.x : kV2MaxSeg - 1)];
  if (pre) {
    const int tv = (int)threadIdx.x < nv ? (int)threadIdx.x : nv - 1;
    const catekv_kv_ptrs pv = a.kv[tv];
    const int64_t pl = a.lens[tv];
    if ((int)threadIdx.x < nv) {
      s_kv[threadIdx.x] = pv;
      s_len[threadIdx.x] = pl;
    }
  }
  __syncthreads();
  // every entry carries the segment count, which the plan keeps in [1, kV2MaxSeg]
  const int nseg = __builtin_amdgcn_readfirstlane((uint32_t)it.bh_n >> 24);
  if ((int)threadIdx.x < nseg) {
    const int bh = it.bh_n & 0xFFFFFF;
    const catekv_kv_ptrs view = pre ? s_kv[bh] : a.kv[bh];
    int64_t len = pre ? s_len[bh] : a.lens[bh];
    len = len < 0 ? 0 : len;
    const int t_end = (int)((int64_t)it.t1 < len ? (int64_t)it.t1 : len);
    const int b = bh / hkv, h = bh - b * hkv;
    V2Seg sg;
    sg.k = reinterpret_cast<const char*>(view.k);
    sg.v = reinterpret_cast<const char*>(view.v);
    sg.t0 = it.t0;
    sg.t_end = t_end;
    sg.n_units = t_end > it.t0 ? (t_end - it.t0 + 15) / 16 : 0;
    sg.row0 = b * hq + h * G;
    sg.slot = it.slot;
    s_seg[threadIdx.x] = sg;
  }
  __syncthreads();

  // ---- this wave's tile stream ----------------------------------------------
  int is = 0, iu = wave;                          // issue cursor: segment, tile of the segment
  auto skip = [&]() {
    while (is < nseg && iu >= s_seg[is].n_units) {
      ++is;
      iu = wave;
    }
  };
  skip();

  uint4 kb[2][4], vb[2][4];
  int meta_seg[2], meta_tile[2];                 // segment and first token of the tile in each buffer
  int lseg = 0, ltile = 0;                       // the last tile issued for real
  // Loads of one tile (called only while the stream has tiles; past its end
  // the last real tile would be read again and the buffer marked empty).
  // Rows past a segment's end re-read its first row, so every address lies
  // inside a segment's rows.
  auto issue = [&](int buf) {
    if (is < nseg) {
      lseg = is;
      ltile = s_seg[is].t0 + iu * 16;
      meta_seg[buf] = is;
      meta_tile[buf] = ltile;
      iu += WAVES;
      skip();
    } else {
      meta_seg[buf] = -1;
    }
    const V2Seg& sg = s_seg[lseg];
    int tk = ltile + n16;
    tk = tk < sg.t_end ? tk : sg.t0;
    const char* kr = sg.k + (size_t)tk * (kD * 2) + k4 * 16;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) kb[buf][ks] = ldg16(kr + ks * 64);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      int tv = ltile + 4 * k4 + r;
      tv = tv < sg.t_end ? tv : sg.t0;
      vb[buf][r] = ldg16(sg.v + (size_t)tv * (kD * 2) + n16 * 16);
    }
  };

  // running state of the segment whose tiles this wave is consuming
  f32x4_t O[8];
  float m, l;
  int st_seg = -1;
  auto reset_state = [&]() {
#pragma unroll
    for (int e = 0; e < 8; ++e) O[e] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    m = head_lane ? kDecodeMFloor : INFINITY;
    l = 0.f;
  };
  reset_state();
  uint4 qb[4];
  int q_seg = -1;

  // merge of segment s: every wave writes its state (or an empty one), then the
  // workgroup reduces the eight states and writes the output or the partial
  int merged = 0;
  auto merge = [&](int s) {
    const int buf = s & 1;
    const bool mine = st_seg == s;
    float lt = mine ? l : 0.f;
    lt += shfl_xor(lt, 16);
    lt += shfl_xor(lt, 32);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int head = 4 * k4 + r;
      if (head < G) {
#pragma unroll
        for (int e = 0; e < 8; ++e) s_o[buf][wave][head][8 * n16 + e] = mine ? O[e][r] : 0.f;
      }
    }
    if (lane < G) {
      s_ml[buf][wave][0][lane] = mine ? m : kDecodeMFloor;
      s_ml[buf][wave][1][lane] = lt;
    }
    if (mine) {
      reset_state();
      st_seg = -1;
    }
    barrier_lds_only();
    const V2Seg& sg = s_seg[s];
    for (int t = threadIdx.x; t < G * kD; t += NT) {
      const int g = t / kD, e = t - g * kD;
      float M = kDecodeMFloor;
#pragma unroll
      for (int w = 0; w < WAVES; ++w) M = fmaxf(M, s_ml[buf][w][0][g]);
      float L = 0.f, Ov = 0.f;
#pragma unroll
      for (int w = 0; w < WAVES; ++w) {
        const float cw = fast_exp2((s_ml[buf][w][0][g] - M) * c);
        L += s_ml[buf][w][1][g] * cw;
        Ov += s_o[buf][w][g][e] * cw;
      }
      const float Mn = M * scale;                 // natural-log units of the scaled score
      if (sg.slot < 0) emit(a.out, a.lse, (size_t)sg.row0 + g, e, Mn, L, Ov);
      else put_slot<G>(a.slots + (size_t)sg.slot * SF, g, e, Mn, L, Ov);
    }
  };

  auto consume = [&](int buf) {
    const int s = meta_seg[buf];
    while (merged < s) merge(merged++);
    if (q_seg != s) {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) qb[ks] = head_lane ? s_q[s][head_lane ? n16 : 0][4 * ks + k4] : make_uint4(0, 0, 0, 0);
      q_seg = s;
    }
    st_seg = s;
    const int tile = meta_tile[buf];
    const int t_end = s_seg[s].t_end;
    f32x4_t S = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      S = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kb[buf][ks]),
                                                  __builtin_bit_cast(bf16x8_t, qb[ks]), S, 0, 0, 0);
    float sv[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) sv[r] = tile + 4 * k4 + r < t_end ? S[r] : -INFINITY;
    float mx = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
    mx = fmaxf(mx, shfl_xor(mx, 16));
    mx = fmaxf(mx, shfl_xor(mx, 32));
    const bool need = head_lane && mx > m + thr;
    if (__builtin_amdgcn_ballot_w64(need)) {
      float corr = 1.f;
      if (head_lane && mx > m) {
        corr = fast_exp2((m - mx) * c);           // 0 while m is still the floor
        m = mx;
      }
      l *= corr;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int src = (4 * k4 + r) & 15;
        const float cr = __int_as_float(__builtin_amdgcn_ds_bpermute(src << 2, __float_as_int(corr)));
#pragma unroll
        for (int e = 0; e < 8; ++e) O[e][r] *= cr;
      }
    }
    const float mc = m * c;
    float P[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      P[r] = fast_exp2(__builtin_fmaf(sv[r], c, -mc));
      l += P[r];
    }
    // P = hi + lo, both bf16
    const uint32_t h01 = pack_bf16(P[0], P[1]), h23 = pack_bf16(P[2], P[3]);
    const uint32_t l01 = pack_bf16(P[0] - __uint_as_float(h01 << 16), P[1] - __uint_as_float(h01 & 0xffff0000u));
    const uint32_t l23 = pack_bf16(P[2] - __uint_as_float(h23 << 16), P[3] - __uint_as_float(h23 & 0xffff0000u));
    const s16x4_t A_hi = __builtin_bit_cast(s16x4_t, make_uint2(h01, h23));
    const s16x4_t A_lo = __builtin_bit_cast(s16x4_t, make_uint2(l01, l23));
    const uint32_t w0[4] = {vb[buf][0].x, vb[buf][0].y, vb[buf][0].z, vb[buf][0].w};
    const uint32_t w1[4] = {vb[buf][1].x, vb[buf][1].y, vb[buf][1].z, vb[buf][1].w};
    const uint32_t w2[4] = {vb[buf][2].x, vb[buf][2].y, vb[buf][2].z, vb[buf][2].w};
    const uint32_t w3[4] = {vb[buf][3].x, vb[buf][3].y, vb[buf][3].z, vb[buf][3].w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      // dims 8 n16 + 2 i (low halves) and 8 n16 + 2 i + 1 (high halves) of the four token rows
      const uint2 be = make_uint2((w0[i] & 0xffffu) | (w1[i] << 16), (w2[i] & 0xffffu) | (w3[i] << 16));
      const uint2 bo = make_uint2((w0[i] >> 16) | (w1[i] & 0xffff0000u), (w2[i] >> 16) | (w3[i] & 0xffff0000u));
      const s16x4_t Be = __builtin_bit_cast(s16x4_t, be), Bo = __builtin_bit_cast(s16x4_t, bo);
      O[2 * i] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(A_hi, Be, O[2 * i], 0, 0, 0);
      O[2 * i] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(A_lo, Be, O[2 * i], 0, 0, 0);
      O[2 * i + 1] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(A_hi, Bo, O[2 * i + 1], 0, 0, 0);
      O[2 * i + 1] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(A_lo, Bo, O[2 * i + 1], 0, 0, 0);
    }
  };

  // the query rows of every segment to LDS (clamped: every thread loads and
  // stores; a clamped thread writes the last piece again, the same value)
  constexpr int QP = (kV2MaxSeg * G * 16 + NT - 1) / NT;
  const int nq = nseg * G * 16;                  // > 0: a worker has at least one segment
  {
    uint4 qv[QP];
#pragma unroll
    for (int p = 0; p < QP; ++p) {
      int t = threadIdx.x + p * NT;
      t = t < nq ? t : nq - 1;
      const int sgi = t / (G * 16), r = t - sgi * (G * 16);
      qv[p] = ldg16(reinterpret_cast<const char*>(a.q) + ((size_t)s_seg[sgi].row0 + (r >> 4)) * (kD * 2) +
                    (r & 15) * 16);
    }
#pragma unroll
    for (int p = 0; p < QP; ++p) {
      int t = threadIdx.x + p * NT;
      t = t < nq ? t : nq - 1;
      const int sgi = t / (G * 16), r = t - sgi * (G * 16);
      s_q[sgi][r >> 4][r & 15] = qv[p];
    }
  }
  __syncthreads();

  // This wave's tiles (tile u of a segment for u = wave, wave + 8, ...) are
  // counted first, so that every issue loads a real tile: no load is still
  // in flight when the stream ends.  Buffer 0 holds tile i on entry to the
  // loop, whose body keeps one tile in flight while it consumes another.
  int n_my = 0;
  for (int s2 = 0; s2 < nseg; ++s2) {
    const int u = s_seg[s2].n_units;
    n_my += u > wave ? (u - wave + WAVES - 1) / WAVES : 0;
  }
  if (n_my > 0) {
    issue(0);
    int i = 0;
    while (i + 2 < n_my) {     // tiles i, i + 1 and i + 2 exist
      issue(1);
      consume(0);
      issue(0);
      consume(1);
      i += 2;
    }
    if (i + 1 < n_my) {
      issue(1);
      consume(0);
      consume(1);
    } else {
      consume(0);
    }
  }
  while (merged < nseg) merge(merged++);
}

// Merges the partials of every view covered by more than one segment: one
// workgroup per (view, query head).  Thread (part lane pl, dim quad dq) loads
// the float4 o of parts pl, pl + 8, ... together with their (m, l) in one
// round of independent loads; the max and the weights are reduced in LDS.
constexpr int kCombineThreads = 512;
constexpr int kCombineLanes = kCombineThreads / 32;    // parts handled side by side
constexpr int kCombineBatch = 16;                      // parts per thread per round

template <int G>
__global__ __launch_bounds__(kCombineThreads) void decode_combine_kernel(DecodeArgs a) {
  constexpr int SF = G * kD + 2 * G;
  const int bh = blockIdx.x / G, g = blockIdx.x - (blockIdx.x / G) * G;
  const ViewInfo vi = a.views[bh];
  const int P = vi.n_parts;
  if (P <= 1) return;
  __shared__ float s_red[kCombineThreads / 64];
  __shared__ float4 s_acc[kCombineLanes][32];
  __shared__ float s_l[kCombineLanes][32];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int pl = t >> 5, dq = t & 31;
  const float* base = a.slots + (size_t)vi.first_slot * SF;

  float M = -INFINITY, L = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s0 = pl; s0 < P; s0 += kCombineLanes * kCombineBatch) {
    float ms[kCombineBatch], ls[kCombineBatch];
    float4 os[kCombineBatch];
#pragma unroll
    for (int u = 0; u < kCombineBatch; ++u) {
      const int s = s0 + u * kCombineLanes;
      if (s < P) {
        const float* sl = base + (size_t)s * SF;
        ms[u] = sl[G * kD + g];
        ls[u] = sl[G * kD + G + g];
        os[u] = *reinterpret_cast<const float4*>(sl + g * kD + 4 * dq);
      } else {
        ms[u] = -INFINITY;
        ls[u] = 0.f;
        os[u] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
    float mb = M;
#pragma unroll
    for (int u = 0; u < kCombineBatch; ++u) mb = fmaxf(mb, ms[u]);
    const float ca = M == -INFINITY ? 0.f : fast_exp2((M - mb) * kLog2e);
    L *= ca;
    acc.x *= ca; acc.y *= ca; acc.z *= ca; acc.w *= ca;
#pragma unroll
    for (int u = 0; u < kCombineBatch; ++u) {
      const float w = ms[u] == -INFINITY ? 0.f : fast_exp2((ms[u] - mb) * kLog2e);
      L += w * ls[u];
      acc.x += w * os[u].x; acc.y += w * os[u].y; acc.z += w * os[u].z; acc.w += w * os[u].w;
    }
    M = mb;
  }
  // global max over the part lanes, then rescale each lane's sums to it
  float Mx = M;
  for (int off = 32; off > 0; off >>= 1) Mx = fmaxf(Mx, shfl_xor(Mx, off));
  if (lane == 0) s_red[wave] = Mx;
  __syncthreads();
  Mx = s_red[0];
#pragma unroll
  for (int w = 1; w < kCombineThreads / 64; ++w) Mx = fmaxf(Mx, s_red[w]);
  const float cs = M == -INFINITY ? 0.f : fast_exp2((M - Mx) * kLog2e);
  s_acc[pl][dq] = make_float4(acc.x * cs, acc.y * cs, acc.z * cs, acc.w * cs);
  s_l[pl][dq] = L * cs;
  __syncthreads();
  if (t < 32) {
    float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
    float Lt = 0.f;
#pragma unroll
    for (int p = 0; p < kCombineLanes; ++p) {
      o.x += s_acc[p][t].x; o.y += s_acc[p][t].y; o.z += s_acc[p][t].z; o.w += s_acc[p][t].w;
      Lt += s_l[p][t];
    }
    const int hkv = a.hkv, b = bh / hkv, h = bh - b * hkv;
    const size_t row = (size_t)b * hkv * G + (size_t)h * G + g;
    const float inv = Lt > 0.f ? 1.f / Lt : 0.f;
    *reinterpret_cast<float4*>(a.out + row * kD + 4 * t) = make_float4(o.x * inv, o.y * inv, o.z * inv, o.w * inv);
    if (a.lse && t == 0) a.lse[row] = Lt > 0.f ? Mx + logf(Lt) : -INFINITY;
  }
}

template <typename T, int G>
static hipError_t launch_t(const DecodeArgs& a, hipStream_t stream) {
  if constexpr (std::is_same<T, uint16_t>::value) {
    if (a.variant == kDecodeStreamV2)
      hipLaunchKernelGGL((decode_stream_v2_kernel<G>), dim3(a.n_workers), dim3(kV2Waves * 64), 0, stream, a);
    else
      hipLaunchKernelGGL((decode_stream_mfma_kernel<G, kDecodeWaves, kDecodeStagesMfma>), dim3(a.n_workers),
                         dim3(kDecodeWaves * 64), 0, stream, a);
  } else
    hipLaunchKernelGGL((decode_stream_kernel<T, G, kDecodeWaves, kDecodeStages>), dim3(a.n_workers),
                       dim3(kDecodeWaves * 64), 0, stream, a);
  if (a.n_multi > 0)
    hipLaunchKernelGGL((decode_combine_kernel<G>), dim3(a.n_views * G), dim3(kCombineThreads), 0, stream, a);
  return hipGetLastError();
}

template <typename T, int G>
static int occupancy_t() {
  int n = 0;
  hipError_t e;
  if constexpr (std::is_same<T, uint16_t>::value)
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, decode_stream_mfma_kernel<G, kDecodeWaves, kDecodeStagesMfma>,
                                                     kDecodeWaves * 64, 0);
  else
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, decode_stream_kernel<T, G, kDecodeWaves, kDecodeStages>,
                                                     kDecodeWaves * 64, 0);
  if (e != hipSuccess) return 1;
  return n < 1 ? 1 : n;
}

int decode_blocks_per_cu(int dtype, int G) {
#define CATEKV_OCC(T, GG) \
  if (G == GG) return occupancy_t<T, GG>();
  if (dtype == CATEKV_BF16) {
    CATEKV_OCC(uint16_t, 1) CATEKV_OCC(uint16_t, 2) CATEKV_OCC(uint16_t, 4) CATEKV_OCC(uint16_t, 8)
  } else {
    CATEKV_OCC(float, 1) CATEKV_OCC(float, 2) CATEKV_OCC(float, 4) CATEKV_OCC(float, 8)
  }
#undef CATEKV_OCC
  return 1;
}

// Appends the newest token of every view: one 64-thread workgroup per view,
// one 16-byte piece of the K row or of the V row per thread.  The length is
// bumped only after every thread has read it.
template <typename T>
__global__ __launch_bounds__(64) void append_kv_kernel(AppendArgs a) {
  constexpr int kPieces = kD * (int)sizeof(T) / 16;   // 16-byte pieces per row
  static_assert(2 * kPieces <= 64, "one thread per piece of the K and V rows");
  const int bh = blockIdx.x;
  const int64_t L = a.lens[bh];
  if (L < 0 || L >= a.capacity[bh]) {
    if (threadIdx.x == 0 && a.overflow) *a.overflow = 1;
    return;
  }
  const int t = threadIdx.x;
  const size_t row = (size_t)kD * sizeof(T);
  const catekv_kv_ptrs p = a.kv[bh];
  if (t < 2 * kPieces) {
    const bool is_k = t < kPieces;
    const int piece = is_k ? t : t - kPieces;
    const char* src = reinterpret_cast<const char*>(is_k ? a.k_new : a.v_new) + (size_t)bh * row + piece * 16;
    char* dst = reinterpret_cast<char*>(const_cast<void*>(is_k ? p.k : p.v)) + (size_t)L * row + piece * 16;
    *reinterpret_cast<uint4*>(dst) = ldg16(src);
  }
  __syncthreads();
  if (t == 0) a.lens[bh] = L + 1;
}

hipError_t launch_append(int dtype, const AppendArgs& a, hipStream_t stream) {
  if (a.n_views <= 0) return hipSuccess;
  if (dtype == CATEKV_BF16)
    hipLaunchKernelGGL(append_kv_kernel<uint16_t>, dim3(a.n_views), dim3(64), 0, stream, a);
  else
    hipLaunchKernelGGL(append_kv_kernel<float>, dim3(a.n_views), dim3(64), 0, stream, a);
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
