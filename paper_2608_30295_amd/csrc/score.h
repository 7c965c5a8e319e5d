// Score passes of the prefill kernels (Algorithm 1, pre-filling stage, and
// the observation matrix of Section 3.2): the softmax rows of the G * L query
// rows of one KV head over a long key range, tile by tile with MFMA, never
// storing the score block:
//   pass 1  per row: maximum m and sum l of exp(s - m)   (row statistics)
//   merge   per row: offset = m * log2(e) / sqrt(d) + log2(l)
//   pass 2  p = exp2(s * log2(e) / sqrt(d) - offset), then either the column
//           mass C_j = (1/G) sum_rows p (selection) or the group-mean
//           observation matrix A[i][j] (CV).
// Workgroup = 4 waves sharing one 64-token K tile staged in LDS; wave w owns
// rows [w * MT * 16, (w + 1) * MT * 16) with their Q fragments in registers.
// Each pass is instantiated in a source file of its own (score_*.hip).
#pragma once

#include "common.h"
#include "cv_state.h"
#include "internal.h"

#include <type_traits>

namespace catekv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kTileTok = 64;     // tokens per LDS tile (4 MFMA column tiles)
constexpr float kMInit = -1e30f; // finite "minus infinity" for running maxima

// MFMA fragment traits.  In k-group kg a lane holds 16 bytes of its row:
// byte offset kg * 64 + (lane / 16) * 16, i.e. 16-byte segment kg * 4 + lane / 16.
// The contraction runs over the head dimension, so any dim permutation that is
// the same for Q and K gives the same dot products.
template <typename T> struct Frag;
template <> struct Frag<uint16_t> {
  static constexpr int KG = 4;   // 4 x (16 x 16 x 32) per 128 dims
  static constexpr int SEG = 16; // 16-byte segments per row
  __device__ static __forceinline__ floatx4 mma(uint4 a, uint4 b, floatx4 acc) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
  }
};
template <> struct Frag<float> {
  static constexpr int KG = 8;   // 8 x 4 x (16 x 16 x 4) per 128 dims
  static constexpr int SEG = 32;
  __device__ static __forceinline__ floatx4 mma(uint4 a, uint4 b, floatx4 acc) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
    return acc;
  }
};

// XOR-swizzled slot of (token, segment) in the LDS tile: 16 consecutive
// tokens reading the same segment hit 16 distinct bank groups.
template <typename T>
__device__ __forceinline__ int tile_slot(int tok, int seg) {
  return tok * Frag<T>::SEG + (seg ^ (tok & 15));
}

// Output-tile shape of the score block: 16 x 16 tiles
// (v_mfma_f32_16x16x32_bf16 / 4 x v_mfma_f32_16x16x4f32).  At k-step ks a
// lane's A (Q) and B (K) fragments are 16 bytes of tile row / column
// frag_rc(lane): 16-byte segment seg(ks, lane) of that row of Q or K (the
// same segment for both, so every dot product covers all 128 dims).
// Accumulator register r of a lane holds the score of tile row row(lane, r)
// and tile column col(lane).
template <typename T> struct Shape {
  using Acc = floatx4;
  static constexpr int TR = 16, TC = 16, NR = 4, KS = Frag<T>::KG;
  static constexpr int kPair8 = 16;   // lanes l and l ^ 16 hold the two halves of an aligned group of 8 rows
  __device__ static __forceinline__ int frag_rc(int lane) { return lane & 15; }
  __device__ static __forceinline__ int seg(int ks, int lane) { return ks * 4 + (lane >> 4); }
  __device__ static __forceinline__ int row(int lane, int r) { return 4 * (lane >> 4) + r; }
  __device__ static __forceinline__ int col(int lane) { return lane & 15; }
  __device__ static __forceinline__ Acc zero() { return Acc{0.f, 0.f, 0.f, 0.f}; }
  __device__ static __forceinline__ Acc mma(uint4 a, uint4 b, Acc c) { return Frag<T>::mma(a, b, c); }
  // over the lanes holding one row (its 16 columns) / one column (its 16 rows)
  __device__ static __forceinline__ float row_max(float x) { return max16(x); }
  __device__ static __forceinline__ float row_sum(float x) { return sum16(x); }
  __device__ static __forceinline__ float col_sum(float x) { return add_xor32(add_xor16(x)); }
};
enum ScoreMode { kRowStats = 0, kColMass = 1, kObsMatrix = 2, kObsBracket = 3 };
enum RowStatsVar { kRsSum = 0, kRsMax = 1 };

struct ScoreArgs {
  const void* q;          // [hq][lq][d]
  const void* k;          // [hkv][n][d]
  int hkv, lq, G, R;      // R = G * lq rows per KV head
  int64_t n;
  int64_t key_off;        // absolute position of key column 0
  int64_t n_keys;         // key columns
  int64_t cb_tokens;      // key columns per workgroup
  int n_colblk;
  int64_t q_pos0;         // absolute position of query row i = 0 (causal mask)
  int causal;             // the causal mask applies (the score kernels take it as a template argument)
  float c;                // log2(e) / sqrt(d)
  int32_t heads[128];     // KV head per blockIdx.y
  float2* rowpart;        // kRowStats out: [n_sel][n_colblk][R_pad] (max * c, sum)
  const float* rowoff;    // kColMass / kObsMatrix in: [n_sel][R_pad]
  float* colmass;         // kColMass out: [n_sel][n_keys] (when cs_fused == 0)
  float* chunks;          // kColMass out: [n_sel][n_chunks] chunk maxima (when cs_fused > 0)
  int cs_fused;           // chunk size when it divides the 64-column tile, else 0
  int64_t n_chunks;
  float* obs;             // kObsMatrix out: [n_sel][lq][n_keys]
  // kObsBracket: A's values at or above the CV bracket's lower end written
  // out with their columns instead of every value stored; kObsMatrix with
  // cv_gate set skips the heads whose bracket took them (only the radix
  // route reads A)
  CvLink cv;
  int cv_gate;
  uint32_t* zero_u32;     // cleared by the row-statistics merge (a later launch's counters), n_zero words
  int n_zero;
};

template <typename T, int W, int MT, int MODE, int G, bool CAUSAL>
__device__ __forceinline__ void score_body(const ScoreArgs& a) {
  using S = Shape<T>;
  using Acc = typename S::Acc;
  constexpr int SEG = Frag<T>::SEG, KS = S::KS, TR = S::TR, TC = S::TC, NR = S::NR;
  constexpr int NCT = 32 / TC;            // column tiles per half tile (32 columns)
  // G = 0: the group size is taken at run time (a.G); only the passes whose
  // arithmetic never splits a group's rows (row statistics without a causal
  // mask, column mass) are built that way
  constexpr bool OBSB = MODE == kObsBracket;
  static_assert(G > 0 || (!CAUSAL && MODE != kObsMatrix && !OBSB), "G must be fixed for masks and the group mean");
  const int GR = G > 0 ? G : a.G;
  constexpr int RPAD = W * MT * TR;
  constexpr int NSTAGE = kTileTok * SEG / (W * 64);   // 16-byte loads per thread per tile
  constexpr int NRING = sizeof(T) == 2 ? 4 : 2;               // LDS stages (16 KB bf16, 32 KB fp32 each)
  // s_waitcnt immediate: vmcnt <= NSTAGE * (NRING - 2), expcnt not waited on;
  // lgkmcnt(0) in column-mass mode, whose column partials in LDS the barrier publishes
  constexpr int VM = NSTAGE * (NRING - 2);
  constexpr int LGKM = MODE == kColMass ? 0 : 0xF;
  constexpr int kWaitRing = (VM & 0xF) | ((VM >> 4) << 14) | (0x7 << 4) | (LGKM << 8);
  // one LDS array per ring stage: stages chosen at compile time do not alias,
  // so the compiler adds no waits of its own between the loads and the reads
  __shared__ uint4 s_r0[kTileTok * SEG], s_r1[kTileTok * SEG], s_r2[kTileTok * SEG], s_r3[kTileTok * SEG];
  __shared__ float s_col[2][W][kTileTok];   // per-wave column partials, by tile parity

  // the wave index is uniform: kept in a scalar register, LDS stage addresses
  // (M0 of the global-to-LDS loads) are formed on the scalar unit
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int sel = blockIdx.y, cb = blockIdx.x;
  const int h = a.heads[sel];
  const int64_t col0 = (int64_t)cb * a.cb_tokens;                   // first key column
  const int64_t col_end = min(col0 + a.cb_tokens, a.n_keys);
  const int n_tiles = (int)((col_end - col0 + kTileTok - 1) / kTileTok);
  if (MODE == kObsMatrix && a.cv_gate && cv_bracket_route(a.cv.st[sel], (int64_t)a.lq * a.n_keys)) return;
  const T* kh = reinterpret_cast<const T*>(a.k) + (size_t)h * a.n * kD;
  const T* qb = reinterpret_cast<const T*>(a.q);

  // Q fragments: the wave's row tile mt, tile row frag_rc(lane), segment seg(ks, lane)
  uint4 qf[MT][KS];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int row = (wave * MT + mt) * TR + S::frag_rc(lane);
    const bool ok = row < a.R;
    const int i = row / GR, g = row - (row / GR) * GR;
    const T* qrow = qb + ((size_t)(h * GR + g) * a.lq + (ok ? i : 0)) * kD;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      uint4 v = ld16(reinterpret_cast<const char*>(qrow) + S::seg(ks, lane) * 16);
      qf[mt][ks] = ok ? v : make_uint4(0, 0, 0, 0);
    }
  }
  // the row of this lane's accumulator register r in row tile mt
  auto row_of = [&](int mt, int r) { return (wave * MT + mt) * TR + S::row(lane, r); };

  float st_mc[MT][NR], st_l[MT][NR];   // kRowStats: row offset (log2 units), sum
  float off[MT][NR];                   // kColMass / kObsMatrix
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      st_mc[mt][r] = kMInit;
      st_l[mt][r] = 0.f;
      off[mt][r] = 0.f;
      if (MODE != kRowStats) off[mt][r] = a.rowoff[(size_t)sel * RPAD + row_of(mt, r)];
    }

  // kObsBracket: the entries at or above u_lo (the lower of the bracket's
  // bottom and Phi's range's) go to this wave's pair buffer (fill:
  // wave-uniform); they are all the entries at or above Phi
  uint32_t wfill = 0;
  float bu_lo = 0.f;
  uint2* wpairs = nullptr;
  if (OBSB) {
    const CvState& B = a.cv.st[sel];
    bu_lo = fminf(cv_key_float(B.k_lo), B.t_lo);
    wpairs = a.cv.pairs + (((size_t)sel * a.n_colblk + cb) * a.cv.nsub + wave) * a.cv.capw;
  }
  // one A value of this lane (key column col; ok: a real entry)
  auto classify = [&](float v, bool ok, uint32_t col) {
    const bool in_u = ok && v >= bu_lo;
    const uint64_t bal = __builtin_amdgcn_ballot_w64(in_u);
    if (bal) {
      const uint32_t at = wfill + (uint32_t)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                                                      __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
      if (in_u && at < a.cv.capw) wpairs[at] = make_uint2(__float_as_uint(v), col);
      wfill += (uint32_t)__builtin_popcountll(bal);
    }
  };

  // K tiles arrive through a ring of NRING LDS stages filled by direct
  // global-to-LDS loads (no staging registers).  Thread x's load i lands in
  // slot i * 64 W + x; the slot's (token, position) picks which 16-byte
  // segment of which row it fetches, so the ring holds the XOR-swizzled
  // layout that tile_slot() reads.
  const int full_tiles = (int)((col_end - col0) / kTileTok);   // tiles with no column past the end
  const char* kbase = reinterpret_cast<const char*>(kh + (size_t)(a.key_off + col0) * kD);
  // byte offset of each of this thread's loads inside a tile (unsigned: the
  // loads take a scalar base plus a 32-bit vector offset)
  uint32_t src_off[NSTAGE];
#pragma unroll
  for (int i = 0; i < NSTAGE; ++i) {
    const int slot = i * W * 64 + threadIdx.x;
    const int tok = slot / SEG, pos = slot - (slot / SEG) * SEG;
    src_off[i] = (uint32_t)(tok * (kD * (int)sizeof(T)) + (pos ^ (tok & 15)) * 16);
  }
  // block-relative 32-bit offsets: a block spans at most kMaxBlockTokens
  // columns, under 2 GiB of K rows
  constexpr uint32_t ROWB = kD * sizeof(T);                  // bytes per K row (a power of two)
  const int n_cols = (int)(col_end - col0);
  // branch-free: a row past the end (or in a tile past the last) re-reads
  // row 0 of the block
  auto issue = [&](uint4* stage, int tile) {
#pragma unroll
    for (int i = 0; i < NSTAGE; ++i) {
      const int col = tile * kTileTok + (int)(src_off[i] / ROWB);
      const uint32_t o = col < n_cols ? (uint32_t)tile * (kTileTok * ROWB) + src_off[i] : (src_off[i] & (ROWB - 1));
      __builtin_amdgcn_global_load_lds(kbase + o, (lds_void*)&stage[i * W * 64 + wave * 64], 16, 0, 0);
    }
  };
  auto ring = [&](int k) -> uint4* { return k == 0 ? s_r0 : k == 1 ? s_r1 : k == 2 ? s_r2 : s_r3; };

  // Column mass of tile t: the four waves' partials are summed by one wave
  // (t mod 4) during tile t + 1, after the barrier that published them, so no
  // wave waits for this step and no barrier of its own is needed.  With cs
  // dividing 64 a chunk never straddles a tile and BlockMax is taken here.
  auto finish_cols = [&](int t) {
    const int p = t & 1;
    const int64_t col = col0 + (int64_t)t * kTileTok + lane;
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < W; ++w) v += s_col[p][w][lane];
    v *= 1.0f / (float)GR;
    if (a.cs_fused > 0) {
      const float mx = max_in_group(col < col_end ? v : -INFINITY, a.cs_fused);
      if ((lane & (a.cs_fused - 1)) == 0 && col < col_end)
        a.chunks[(size_t)sel * a.n_chunks + col / a.cs_fused] = mx;
    } else if (col < col_end) {
      a.colmass[(size_t)sel * a.n_keys + col] = v;
    }
  };
  // keys at or past column col_end, and (causal) keys past a row's position,
  // score -inf.  Columns count from col0; a row at query index i sees
  // columns up to lim_rel + i (lim_rel clamped: every column of a block lies
  // within 2^30 of its start).
  const int lim_rel = (int)max((int64_t)-(1 << 30), min((int64_t)(1 << 30), a.q_pos0 - a.key_off - col0));
  auto mask_acc = [&](Acc& x, int col_rel, int mt) {
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      const int row = row_of(mt, r);
      bool ok = col_rel < n_cols;
      if (CAUSAL) ok = ok && (col_rel - row / G <= lim_rel);
      x[r] = ok ? x[r] : -INFINITY;
    }
  };

  // One tile: the whole 64-column score block of this wave first (MFMA), then
  // the softmax arithmetic on it (VALU); without branches inside, the
  // scheduler overlaps the two.  Masks are needed only on a ragged last tile
  // or where keys can lie past a row's position.  In row-statistics mode VAR
  // picks what a tile adds to the row state: kRsSum the terms exp2(s c - m)
  // against the lane's offset m = st_mc, kRsMax the maximum s c itself.
  auto do_tile = [&](const uint4* cur, int tile, auto var_tag, auto mask_tag, bool first_half_only = false) {
    constexpr int VAR = decltype(var_tag)::value;
    const int64_t tcol0 = col0 + (int64_t)tile * kTileTok;
    float cmass[kTileTok / TC];
#pragma unroll
    for (int t = 0; t < kTileTok / TC; ++t) cmass[t] = -0.f;   // -0 + x folds to x
    // the MFMA work of one half tile (32 columns: NCT column tiles); k-step
    // outer, row tile inner: a B fragment is live for MT MFMAs, and the MT
    // accumulator chains interleave
    auto mfma_half = [&](int hh, Acc (&acc)[NCT][MT]) {
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const uint4 bf = cur[tile_slot<T>(hh * 32 + ct * TC + S::frag_rc(lane), S::seg(ks, lane))];
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) acc[ct][mt] = S::mma(qf[mt][ks], bf, ks == 0 ? S::zero() : acc[ct][mt]);
        }
      }
    };
    // the softmax arithmetic of one half tile
    auto valu_half = [&](int hh, Acc (&acc)[NCT][MT], auto mask_tag) {
      constexpr bool MASK = decltype(mask_tag)::value;
      if (MASK) {
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) mask_acc(acc[ct][mt], tile * kTileTok + hh * 32 + ct * TC + S::col(lane), mt);
      }
      if (MODE == kRowStats && VAR == kRsSum) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int r = 0; r < NR; ++r) {
            float t = fast_exp2(__builtin_fmaf(acc[0][mt][r], a.c, -st_mc[mt][r]));
#pragma unroll
            for (int ct = 1; ct < NCT; ++ct) t += fast_exp2(__builtin_fmaf(acc[ct][mt][r], a.c, -st_mc[mt][r]));
            st_l[mt][r] += t;
          }
      } else if (MODE == kRowStats) {
        // c > 0, so the maximum of s c is c times the maximum of s; masked
        // scores (-inf) leave the state alone
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int r = 0; r < NR; ++r) {
            float m = acc[0][mt][r];
#pragma unroll
            for (int ct = 1; ct < NCT; ++ct) m = fmaxf(m, acc[ct][mt][r]);
            st_mc[mt][r] = fmaxf(st_mc[mt][r], m * a.c);
          }
      } else if (MODE == kColMass) {
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < NR; ++r)
              cmass[hh * NCT + ct] += fast_exp2(__builtin_fmaf(acc[ct][mt][r], a.c, -off[mt][r]));
      } else {  // kObsMatrix / kObsBracket: group mean over the G rows of each query i
        const float invG = 1.0f / (float)G;
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
          const int64_t col = tcol0 + hh * 32 + ct * TC + S::col(lane);
          const uint32_t col32 = (uint32_t)tcol0 + (uint32_t)(hh * 32 + ct * TC + S::col(lane));   // key columns < 2^32
          const bool colok = !MASK || col < col_end;
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            float p[NR];
#pragma unroll
            for (int r = 0; r < NR; ++r) p[r] = fast_exp2(__builtin_fmaf(acc[ct][mt][r], a.c, -off[mt][r]));
            if (G == 1 || G == 2 || G == 4) {
              // the lane's NR registers hold NR consecutive rows from a multiple of 4:
              // queries i0 .. i0 + NR / G - 1, one store base for all of them
              const int i0 = row_of(mt, 0) / G;
              float* ob = OBSB ? nullptr : a.obs + ((size_t)sel * a.lq + i0) * a.n_keys + col;
#pragma unroll
              for (int r0 = 0; r0 < NR; r0 += G) {
                float v = p[r0];
#pragma unroll
                for (int r = 1; r < G; ++r) v += p[r0 + r];
                const bool ok = i0 + r0 / G < a.lq && colok;
                if (OBSB) classify(v * invG, ok, col32);
                else if (ok) ob[(size_t)(r0 / G) * a.n_keys] = v * invG;
              }
            } else {  // G == 8: lanes l and l ^ kPair8 hold the two halves of each group of 8 rows
#pragma unroll
              for (int b4 = 0; b4 < NR; b4 += 4) {
                const float q4 = p[b4] + p[b4 + 1] + p[b4 + 2] + p[b4 + 3];
                const float v = S::kPair8 == 16 ? add_xor16(q4) : add_xor32(q4);
                const int i = row_of(mt, b4) / 8;
                const bool ok = (lane & S::kPair8) == 0 && i < a.lq && colok;
                if (OBSB) classify(v * invG, ok, col32);
                else if (ok) a.obs[((size_t)sel * a.lq + i) * a.n_keys + col] = v * invG;
              }
            }
          }
        }
      }
    };
    // one half's accumulators live at a time: the second half's MFMAs stay
    // after the first half's softmax work
    Acc acc0[NCT][MT], acc1[NCT][MT];
    mfma_half(0, acc0);
    valu_half(0, acc0, mask_tag);
    if (first_half_only) return;
    __builtin_amdgcn_sched_barrier(0);
    mfma_half(1, acc1);
    valu_half(1, acc1, mask_tag);

    if (MODE == kColMass) {
      // sum over the lanes holding each column; each wave leaves its partial in LDS
#pragma unroll
      for (int t = 0; t < kTileTok / TC; ++t) {
        const float v = S::col_sum(cmass[t]);
        if (lane < TC) s_col[tile & 1][wave][t * TC + lane] = v;
      }
    }
  };

  // One step of the ring: wait for tile `tile` (stage S), publish it to the
  // workgroup, refill the stage the previous step freed, run the tile.
  // Vector memory operations retire in order, so the tile's loads are done
  // once at most NRING - 2 later groups are outstanding; the barrier makes
  // every wave's part of the tile visible and frees the stage the issue
  // overwrites.
  auto step = [&](int S, int tile, auto&& body) {
    compiler_fence();
    __builtin_amdgcn_s_waitcnt(kWaitRing);
    __builtin_amdgcn_s_barrier();
    compiler_fence();
    issue(ring((S + NRING - 1) % NRING), tile + NRING - 1);
    if (MODE == kColMass && tile > 0 && wave == ((tile - 1) & (W - 1))) finish_cols(tile - 1);
    body(ring(S), tile);
  };
  auto prime = [&]() {
#pragma unroll
    for (int t = 0; t < NRING - 1; ++t) issue(ring(t), t);
  };
  // Tiles [0, n_plain) need no mask: every column lies before col_end and
  // (causal) at or before the position of every row.  The rest -- a ragged
  // last tile, the diagonal of a causal block -- come after them.
  int n_plain = full_tiles;
  if (CAUSAL) {
    const int64_t lim = a.q_pos0 - a.key_off - col0 + 1;   // columns [0, lim) are visible to every row
    n_plain = (int)min((int64_t)n_plain, lim <= 0 ? (int64_t)0 : lim / kTileTok);
  }
  using Plain = std::false_type;
  using Masked = std::true_type;
  // tiles [S0, n_tiles): the plain ones in whole turns of the ring with the
  // stage known at compile time (S0 is 0 or 1; no branch inside a turn, so a
  // tile's MFMA and VALU work share one basic block), the rest of the plain
  // ones, then the masked ones
  auto run = [&](auto s0_tag, auto var_tag) {
    constexpr int S0 = decltype(s0_tag)::value;
    int tile = S0;
    for (; tile + NRING <= n_plain; tile += NRING) {
#pragma unroll
      for (int u = 0; u < NRING; ++u)
        step((S0 + u) % NRING, tile + u, [&](const uint4* cur, int t) { do_tile(cur, t, var_tag, Plain{}); });
    }
    for (; tile < n_plain; ++tile)
      step(tile % NRING, tile, [&](const uint4* cur, int t) { do_tile(cur, t, var_tag, Plain{}); });
    for (; tile < n_tiles; ++tile)
      step(tile % NRING, tile, [&](const uint4* cur, int t) { do_tile(cur, t, var_tag, Masked{}); });
  };
  using RsSum = std::integral_constant<int, kRsSum>;
  using RsMax = std::integral_constant<int, kRsMax>;

  prime();
  if (MODE == kRowStats) {
    // Each row's offset is its maximum over the first 32 columns of the block
    // (log2 units; kMInit for a row that sees no key there -- it then sees
    // none in the whole block, as a row's visible keys form a prefix of the
    // key range).  Later tiles add their terms against that offset with no
    // running maximum: terms up to 2^128 stay finite in fp32.  A sum that
    // overflows anyway is written as it is (inf); the merge recomputes that
    // block's statistics exactly.
    if (n_tiles > 0) {
      auto first = [&](auto mask_tag) {
        step(0, 0, [&](const uint4* cur, int t) {
          do_tile(cur, t, RsMax{}, mask_tag, true);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < NR; ++r) st_mc[mt][r] = S::row_max(st_mc[mt][r]);
          do_tile(cur, t, RsSum{}, mask_tag);
        });
      };
      if (n_plain > 0) first(Plain{});
      else first(Masked{});
      run(std::integral_constant<int, 1>{}, RsSum{});
    }
  } else {
    run(std::integral_constant<int, 0>{}, RsSum{});
  }

  if (MODE == kColMass) {
    barrier_lds_only();
    if (n_tiles > 0 && wave == ((n_tiles - 1) & (W - 1))) finish_cols(n_tiles - 1);
  }

  // the ring's trailing loads must land before the workgroup's LDS is released
  __builtin_amdgcn_s_waitcnt(0);
  compiler_fence();

  if (OBSB) {                      // the waves' pair fills
    if (lane == 0) {
      a.cv.pfill[((size_t)sel * a.n_colblk + cb) * a.cv.nsub + wave] = min(wfill, a.cv.capw);
      if (wfill > a.cv.capw) atomicOr(&a.cv.st[sel].phi_over, 1u);
    }
    if (threadIdx.x >= W && threadIdx.x < a.cv.nsub)   // buffers of waves this shape does not have
      a.cv.pfill[((size_t)sel * a.n_colblk + cb) * a.cv.nsub + threadIdx.x] = 0;
    // Each wave reads its own pairs back (its stores have completed: the
    // wait above): the bracket entries are counted and histogrammed by
    // their first digit (key - k_lo) >> shift1, and the pairs at or above
    // the bracket's bottom counted; the block's counts and histogram go to
    // the head's totals with one atomic each.
    __shared__ uint32_t s_ph[OBSB ? kCvBins : 1];
    __shared__ uint32_t s_pc[OBSB ? 2 * W : 1];
    for (int i = threadIdx.x; i < kCvBins; i += W * 64) s_ph[i] = 0;
    __syncthreads();
    const CvState& B = a.cv.st[sel];
    const uint32_t k_lo = B.k_lo, span = B.k_hi - B.k_lo;
    const int sh1 = B.shift1;
    const float f_lo = cv_key_float(k_lo);
    const uint32_t fill = min(wfill, a.cv.capw);
    uint32_t n_in = 0, n_lo = 0;
    for (uint32_t i0 = 0; i0 < fill; i0 += 4 * 64) {   // the same trip count on every lane
      uint32_t x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {     // every load issued (clamped), then used
        const uint32_t i = i0 + u * 64 + lane;
        x[u] = wpairs[i < fill ? i : fill - 1].x;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const bool ok = i0 + u * 64 + lane < fill;
        const uint32_t o = (x[u] | 0x80000000u) - k_lo;
        const bool in = ok && o <= span;
        n_in += in;
        n_lo += ok && __uint_as_float(x[u]) >= f_lo;
        hist_add(s_ph, in, o >> sh1);
      }
    }
    for (int off = 32; off > 0; off >>= 1) {
      n_in += __shfl_xor(n_in, off);
      n_lo += __shfl_xor(n_lo, off);
    }
    if (lane == 0) {
      s_pc[wave] = n_in;
      s_pc[W + wave] = n_lo;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      unsigned long long c_in = 0, c_lo = 0;
#pragma unroll
      for (int w = 0; w < W; ++w) {
        c_in += s_pc[w];
        c_lo += s_pc[W + w];
      }
      if (c_in) atomicAdd(&a.cv.st[sel].n_cand, c_in);
      if (c_lo) atomicAdd(&a.cv.st[sel].ge_lo, c_lo);
    }
    uint32_t* h0 = a.cv.hist0 + (size_t)sel * kCvBins;
    for (int i = threadIdx.x; i < kCvBins; i += W * 64)
      if (s_ph[i]) atomicAdd(&h0[i], s_ph[i]);
  }

  if (MODE == kRowStats) {
    // merge the lanes that share each row (maxima in log2 units)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < NR; ++r) {
        const float m = st_mc[mt][r];
        const float M = S::row_max(m);
        const float lsum = S::row_sum(st_l[mt][r] * fast_exp2(m - M));
        if (S::col(lane) == 0)
          a.rowpart[((size_t)sel * a.n_colblk + cb) * RPAD + row_of(mt, r)] = make_float2(M, lsum);
      }
  }
}

// Workgroup shapes, W waves of MT 16-row tiles (W * MT * 16 = rows), WPE
// waves per SIMD (registers: 512 / WPE per wave).  The LDS ring (64 KB)
// allows two workgroups per compute unit.  bf16 runs four waves per SIMD from
// 128 rows on: 8-wave workgroups of one or two row tiles per wave, two per
// CU; 512 rows in one 16-wave workgroup per CU.  Measured at 256 rows (5
// heads, 128K keys): pass times 53 / 57 us against 58 / 61 us for 4 waves of
// 4 row tiles at two waves per SIMD.  fp32 fragments are twice as wide and
// keep two waves per SIMD.  The block count (score_block_tokens) follows
// the bf16 residency; the other shapes run in more rounds.
template <typename T, int W, int MT, int MODE, int G, bool CAUSAL, int WPE>
__global__ __launch_bounds__(W * 64) __attribute__((amdgpu_waves_per_eu(WPE)))
void score_kernel(ScoreArgs a) {
  score_body<T, W, MT, MODE, G, CAUSAL>(a);
}

template <typename T, int MODE, int G, bool CAUSAL>
inline hipError_t launch_score_mt(int rows_pad, dim3 grid, hipStream_t s, const ScoreArgs& a) {
  constexpr bool F32 = std::is_same<T, float>::value;
  // one query per row (G = 1) stores every row of the observation matrix on
  // its own: those passes keep two waves per SIMD
  constexpr bool NARROW = (MODE == kObsMatrix || MODE == kObsBracket) && G == 1;
#define CATEKV_SK(WW, MM, PP) \
  hipLaunchKernelGGL((score_kernel<T, WW, MM, MODE, G, CAUSAL, PP>), grid, dim3((WW) * 64), 0, s, a)
  if constexpr (F32) {
    if (rows_pad == 64) CATEKV_SK(4, 1, 2);
    else if (rows_pad == 128) CATEKV_SK(4, 2, 2);
    else if (rows_pad == 256) CATEKV_SK(8, 2, 2);
    else if (rows_pad == 512) CATEKV_SK(8, 4, 2);
    else return hipErrorInvalidValue;
  } else if constexpr (NARROW) {
    if (rows_pad == 64) CATEKV_SK(4, 1, 2);
    else if (rows_pad == 128) CATEKV_SK(8, 1, 4);
    else if (rows_pad == 256) CATEKV_SK(8, 2, 2);
    else if (rows_pad == 512) CATEKV_SK(8, 4, 2);
    else return hipErrorInvalidValue;
  } else {
    if (rows_pad == 64) CATEKV_SK(4, 1, 2);
    else if (rows_pad == 128) CATEKV_SK(8, 1, 4);
    else if (rows_pad == 256) CATEKV_SK(8, 2, 4);
    else if (rows_pad == 512) CATEKV_SK(16, 2, 4);
    else return hipErrorInvalidValue;
  }
#undef CATEKV_SK
  return hipGetLastError();
}

// Launch one score pass over grid (column blocks, heads) for rows_pad query
// rows (64, 128, 256 or 512; see score_waves).
hipError_t launch_score_rowstats(int dtype, int G, bool causal, int rows_pad, dim3 grid, hipStream_t s,
                                 const ScoreArgs& a);
hipError_t launch_score_colmass(int dtype, int rows_pad, dim3 grid, hipStream_t s, const ScoreArgs& a);
hipError_t launch_score_obs(int dtype, int G, bool causal, int rows_pad, dim3 grid, hipStream_t s,
                            const ScoreArgs& a);
hipError_t launch_score_obs_bracket(int dtype, int G, bool causal, int rows_pad, dim3 grid, hipStream_t s,
                                    const ScoreArgs& a);

// The CV score's own kernels (cv.hip) around the observation-matrix passes:
// the workspace they share, the bracket from the merge's samples, and after
// the bracketing pass the order statistic, the column counts and the score.
size_t cv_workspace_bytes(int hkv, int lq, int64_t n_keys, int n_colblk);
CvLink cv_link(void* ws, int hkv, int lq, int64_t n_keys, int n_colblk, int nsub);
hipError_t launch_cv_sample(const ScoreArgs& a, double k_pct, double alpha, hipStream_t s);
hipError_t launch_cv_finish(const ScoreArgs& a, double k_pct, double alpha, float* cv_out, hipStream_t s);

}  // namespace catekv
