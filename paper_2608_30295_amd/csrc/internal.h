// Internal interface between the host C ABI (api.cpp) and the kernel
// launchers (*.hip).  Plain C++: no HIP types beyond hipStream_t.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

#include "catekv.h"

namespace catekv {

constexpr int kD = 128;   // supported head dimension

// One split-KV work item of the decode plan: tokens [t0, t1) of the view
// bh = b * hkv + h; `part` is its index among the view's items.
struct DecodeItem {
  int32_t bh;
  int32_t part;
  int32_t t0;
  int32_t t1;
};

constexpr int kDecodeWaves = 4;    // waves per decode workgroup
constexpr int kDecodeStages = 4;   // register prefetch depth (fp32 path)
constexpr int kDecodeStagesMfma = 2;   // register prefetch depth (bf16 MFMA path, 16-token stages)
constexpr int kDecodeQuantum = 64; // tokens per workgroup load stage (16 per wave)

// Decode kernels a plan is cut for.
constexpr int kDecodeStreamK4 = 1;   // 4-wave workgroups, as many as the device holds (any segment count)
constexpr int kDecodeStreamV2 = 2;   // one 8-wave workgroup per compute unit (bf16), <= kDecodeV2MaxSeg
                                     // segments per workgroup
constexpr int kDecodeV2MaxSeg = 16;

// A segment of a one-workgroup-per-CU plan (kDecodeStreamV2) as the stream
// kernel reads it: the plan also writes them worker-major, kDecodeV2MaxSeg
// entries per worker, so that a workgroup finds its segments with one load.
struct V2Item {
  int32_t bh_n;           // view bh (low 24 bits) and the worker's segment count (high 8 bits)
  int32_t t0;
  int32_t t1;
  int32_t slot;           // partial slot, or -1 when the segment covers its whole view
};

// Per view: where its partial slots live and how many segments cover it.
struct ViewInfo {
  int32_t first_slot;     // slot of part 0
  int32_t n_parts;        // segments covering the view
};

// Floats per decode partial slot for a group of G query heads: o[G][128],
// m[G], l[G].
inline size_t decode_slot_floats(int G) { return (size_t)G * 128 + 2 * (size_t)G; }

struct DecodeArgs {
  const void* q;
  const catekv_kv_ptrs* kv;
  const int64_t* lens;
  const DecodeItem* items;      // segments, grouped by worker
  const int32_t* worker_seg;    // [n_workers + 1] first segment of each worker
  const V2Item* v2items;        // kDecodeStreamV2: [n_workers][kDecodeV2MaxSeg]
  const ViewInfo* views;
  float* slots;                 // partial slots
  int n_workers, n_views, n_multi, hkv;
  int variant;                  // kDecodeStreamK4 or kDecodeStreamV2
  float scale;
  float* out;
  float* lse;
};

// Decode workgroups one CU holds at once (occupancy of the stream kernel).
int decode_blocks_per_cu(int dtype, int G);
hipError_t launch_decode(int dtype, int G, const DecodeArgs& a, hipStream_t stream);

// ---- decode-time KV append ------------------------------------------------
struct AppendArgs {
  const catekv_kv_ptrs* kv;
  const int64_t* capacity;
  int64_t* lens;
  const void* k_new;
  const void* v_new;
  int32_t* overflow;        // may be null
  int n_views;
};
hipError_t launch_append(int dtype, const AppendArgs& a, hipStream_t stream);

// ---- critical-token selection ------------------------------------------
struct SelectGeom {
  int hq, hkv, G, l_obs, cs, n_sel, b;
  int64_t n, n_keys;       // n_keys = n - l_obs
  int64_t n_chunks;
  int64_t cb_tokens;       // key columns per score workgroup
  int n_colblk;            // column blocks of the score passes
  int heads[128];
};

// Query rows of the score passes, padded to a whole number of 16-row tiles
// per wave: 64, 128, 256 or 512.
inline int score_rows_pad(int rows) {
  const int mt = (rows + 63) / 64;
  return (mt <= 1 ? 1 : mt <= 2 ? 2 : mt <= 4 ? 4 : 8) * 64;
}
// Waves per score workgroup.  bf16: 4 up to 64 rows, 8 up to 256, 16 for
// 512 (four waves per SIMD from 128 rows on); fp32: 4 up to 128 rows, else 8.
inline int score_waves(int dtype, int rows_pad) {
  if (dtype == CATEKV_F32) return rows_pad > 128 ? 8 : 4;
  return rows_pad <= 64 ? 4 : rows_pad <= 256 ? 8 : 16;
}
// Key columns per score workgroup for n_keys columns of n_heads KV heads and
// rows_pad query rows on a device of n_cu compute units; at most
// kMaxBlockTokens (the kernels address a block's K rows with 32-bit offsets).
constexpr int64_t kMaxBlockTokens = (int64_t)1 << 22;
int64_t score_block_tokens(int64_t n_keys, int n_heads, int rows_pad, int n_cu);
size_t select_workspace_bytes(const SelectGeom& g);
// The file-scope scratch of the allocation-free selection: its size, and its
// device address on the current device.
size_t select_scratch_bytes();
hipError_t select_scratch(void** ptr);
hipError_t launch_select(int dtype, const SelectGeom& g, const void* q_obs, const void* k,
                         int32_t* idx_out, void* ws, hipStream_t stream);
hipError_t launch_compact(int dtype, const void* k, const void* v, int hkv, int64_t n, int cs,
                          int l_obs, const int32_t* heads, int n_sel, const int32_t* idx, int b,
                          void* k_c, void* v_c, int64_t* lens_out, hipStream_t stream);

// Indices of the min(b, n) largest of each row of S [n_rows][n] (ties to the
// lower index), ascending, -1 padded to b.  ws: topk_workspace_bytes() bytes
// (rows longer than 4096 scores are reduced slice by slice through it); its
// first n_rows 32-bit words must be zero on entry (an earlier launch of the
// same call clears them) and are left zero.
size_t topk_workspace_bytes(int n_rows, int64_t n);
hipError_t launch_topk(const float* S, int n_rows, int64_t n, int b, int32_t* idx_out, void* ws,
                       hipStream_t stream);

// ---- query-aware retrieval in adaptive heads (page bounds and scores) -----
hipError_t launch_page_bounds(int dtype, const void* k, int64_t n, int cs, const int32_t* heads, int n_sel,
                              void* kmin, void* kmax, hipStream_t stream);
hipError_t launch_page_scores(int dtype, int G, const void* q, const void* kmin, const void* kmax,
                              int64_t n_pages, const int32_t* heads, int n_sel, float* scores,
                              uint32_t* zero_u32, int n_zero, hipStream_t stream);

// ---- CV head scoring -----------------------------------------------------
struct ScoreGeom {
  int hq, hkv, G, lq;
  int64_t n, l_init, l_rec, n_keys;   // n_keys = n - l_init - l_rec
  int64_t q_pos0;
  int causal;
  double k_pct, alpha;
  int64_t cb_tokens;
  int n_colblk;
};

size_t score_workspace_bytes(const ScoreGeom& g);

hipError_t launch_score(int dtype, const ScoreGeom& g, const void* q_rows, const void* k,
                        float* cv_out, void* ws, hipStream_t stream);

}  // namespace catekv
