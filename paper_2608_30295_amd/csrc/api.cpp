// Host side of the CateKV C ABI: argument validation, workspace layout, the
// decode work list and head classification.  Every argument is checked
// before anything is enqueued; kernel launches live in the .hip files.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <numeric>
#include <string>
#include <vector>

#include "catekv.h"
#include "internal.h"

namespace {

thread_local std::string g_err;
constexpr uint64_t kPlanMagic = 0x43617465504c414eull;   // "CatePLAN"
constexpr int kMaxHeads = 128;
constexpr int kMaxRows = 512;                           // G * L rows per KV head in the score passes

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return CATEKV_OK;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(CATEKV_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool valid_dtype(int dt) { return dt == CATEKV_F32 || dt == CATEKV_BF16; }

int check_heads(int hq, int hkv, int d) {
  if (d != catekv::kD) return fail(CATEKV_ERR_UNSUPPORTED, "head dimension %d unsupported (only 128)", d);
  if (hkv < 1 || hq < 1) return fail(CATEKV_ERR_INVALID_ARG, "hq=%d hkv=%d must be positive", hq, hkv);
  if (hkv > kMaxHeads) return fail(CATEKV_ERR_UNSUPPORTED, "hkv=%d above %d", hkv, kMaxHeads);
  if (hq % hkv) return fail(CATEKV_ERR_INVALID_ARG, "hq=%d is not a multiple of hkv=%d", hq, hkv);
  const int G = hq / hkv;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return fail(CATEKV_ERR_UNSUPPORTED, "group size hq/hkv=%d unsupported (1, 2, 4 or 8)", G);
  return CATEKV_OK;
}

int check_ws(const void* ws, size_t ws_bytes, size_t need) {
  if (need == 0) return CATEKV_OK;
  if (!ws) return fail(CATEKV_ERR_WORKSPACE, "workspace pointer is null (need %zu bytes)", need);
  if (reinterpret_cast<uintptr_t>(ws) % 256) return fail(CATEKV_ERR_WORKSPACE, "workspace not 256-byte aligned");
  if (ws_bytes < need) return fail(CATEKV_ERR_WORKSPACE, "workspace %zu bytes, need %zu", ws_bytes, need);
  return CATEKV_OK;
}

// Linearly interpolated quantile of x (copied, sorted ascending).
double quantile_linear(std::vector<double> x, double p) {
  std::sort(x.begin(), x.end());
  const double h = (double)(x.size() - 1) * p;
  const size_t lo = (size_t)std::floor(h);
  const size_t hi = std::min(lo + 1, x.size() - 1);
  return x[lo] + (h - (double)lo) * (x[hi] - x[lo]);
}

// ---- decode plan: stream-K shares of the concatenated views ---------------

struct Segment {
  int view, worker;
  int64_t t0, t1;
};

struct PlanLayout {
  int n_workers = 0, n_segments = 0, n_slots = 0, n_multi = 0;
  size_t segs_off = 0, workers_off = 0, views_off = 0, slots_off = 0, total = 0;
  std::vector<Segment> segs;   // grouped by worker
};

size_t a256(size_t x) { return (x + 255) & ~(size_t)255; }

// The worker-major segment table sits right after the segment list.
size_t v2_items_off(size_t segs_off, int n_segments) {
  return segs_off + a256((size_t)n_segments * sizeof(catekv::DecodeItem));
}

int device_cus() {
  int dev = 0, n_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n_cu < 1)
    n_cu = 256;
  return n_cu;
}

// Workgroups of a 4-wave plan: as many as the device holds at once, or one
// per compute unit when the step is small (fewer than kFewTokens rows in all
// views; 128 MB of bf16 K and V): a step that short is dominated by its fixed
// costs (start-up chain, partials, merge), which one workgroup per CU halves,
// while a longer step streams slightly faster with two.
constexpr int64_t kFewTokens = 1 << 18;
int device_workers(int G, const int64_t* max_len, int n_views) {
  const int n_cu = device_cus();
  int64_t total = 0;
  for (int v = 0; v < n_views; ++v) total += max_len[v];
  return total < kFewTokens ? n_cu : n_cu * catekv::decode_blocks_per_cu(CATEKV_BF16, G);
}

// Cuts the views (in index order, laid end to end in units of
// kDecodeQuantum tokens) into n_workers near-equal shares.
PlanLayout plan_layout(const int64_t* max_len, int n_views, int G, int split, int workers_hint) {
  PlanLayout P;
  const int64_t Q = catekv::kDecodeQuantum;
  std::vector<int64_t> units(n_views);
  int64_t U = 0;
  for (int v = 0; v < n_views; ++v) {
    units[v] = (max_len[v] + Q - 1) / Q;
    U += units[v];
  }
  int64_t W = split > 0 ? (U * Q + split - 1) / split : workers_hint;
  W = std::max<int64_t>(1, std::min<int64_t>(W, std::max<int64_t>(U, 1)));
  P.n_workers = (int)W;
  int v = 0;
  int64_t off = 0;   // units consumed of view v
  for (int64_t w = 0; w < W; ++w) {
    int64_t need = (w + 1) * U / W - w * U / W;
    while (need > 0 && v < n_views) {
      if (units[v] == 0) { ++v; off = 0; continue; }
      const int64_t take = std::min(need, units[v] - off);
      P.segs.push_back({v, (int)w, off * Q, std::min(max_len[v], (off + take) * Q)});
      need -= take;
      off += take;
      if (off == units[v]) { ++v; off = 0; }
    }
  }
  // empty views still produce an output (zeros and -inf): one empty segment each
  for (int e = 0; e < n_views; ++e)
    if (units[e] == 0) P.segs.push_back({e, (int)(e % W), 0, 0});
  std::stable_sort(P.segs.begin(), P.segs.end(), [](const Segment& x, const Segment& y) { return x.worker < y.worker; });
  P.n_segments = (int)P.segs.size();
  std::vector<int> parts(n_views, 0);
  for (const Segment& s : P.segs) parts[s.view]++;
  for (int i = 0; i < n_views; ++i) {
    P.n_slots += parts[i];
    P.n_multi += parts[i] > 1;
  }
  const size_t sf = catekv::decode_slot_floats(G) * sizeof(float);
  size_t o = 0;
  P.segs_off = o; o += a256((size_t)P.n_segments * sizeof(catekv::DecodeItem));
  o += a256((size_t)P.n_workers * catekv::kDecodeV2MaxSeg * sizeof(catekv::V2Item));   // v2_items_off()
  P.workers_off = o; o += a256((size_t)(P.n_workers + 1) * sizeof(int32_t));
  P.views_off = o; o += a256((size_t)n_views * sizeof(catekv::ViewInfo));
  P.slots_off = o; o += a256((size_t)std::max(P.n_slots, 1) * sf);
  P.total = o;
  return P;
}

// The decode layout of a plan: one 8-wave workgroup per compute unit, whose
// LDS table holds up to kDecodeV2MaxSeg segments per workgroup; when some
// workgroup's share would cross more views than that (many tiny or empty
// views), the 4-wave layout, which reads segment descriptors as it goes.
PlanLayout choose_plan(const int64_t* max_len, int n_views, int G, int split, int* variant) {
  PlanLayout P = plan_layout(max_len, n_views, G, split, device_cus());
  std::vector<int> per_worker(P.n_workers, 0);
  int most = 0;
  for (const Segment& sg : P.segs) most = std::max(most, ++per_worker[sg.worker]);
  const int least = *std::min_element(per_worker.begin(), per_worker.end());   // the stream kernel assumes >= 1
  if (most <= catekv::kDecodeV2MaxSeg && least >= 1 && n_views < (1 << 24)) {   // view ids fit 24 bits
    *variant = catekv::kDecodeStreamV2;
    return P;
  }
  *variant = catekv::kDecodeStreamK4;
  return plan_layout(max_len, n_views, G, split, device_workers(G, max_len, n_views));
}

int check_lengths(const int64_t* max_len, int n) {
  for (int i = 0; i < n; ++i) {
    if (max_len[i] < 0) return fail(CATEKV_ERR_INVALID_ARG, "max_len[%d] = %lld is negative", i, (long long)max_len[i]);
    if (max_len[i] > INT32_MAX)
      return fail(CATEKV_ERR_UNSUPPORTED, "max_len[%d] = %lld above 2^31 - 1", i, (long long)max_len[i]);
  }
  return CATEKV_OK;
}

int check_head_list(int hkv, const int32_t* heads, int n_sel) {
  if (n_sel < 1 || n_sel > hkv) return fail(CATEKV_ERR_INVALID_ARG, "n_sel=%d outside [1, hkv=%d]", n_sel, hkv);
  if (!heads) return fail(CATEKV_ERR_INVALID_ARG, "sel_heads_host is null");
  std::vector<char> seen(hkv, 0);
  for (int i = 0; i < n_sel; ++i) {
    if (heads[i] < 0 || heads[i] >= hkv) return fail(CATEKV_ERR_INVALID_ARG, "sel_heads_host[%d]=%d out of range", i, heads[i]);
    if (seen[heads[i]]) return fail(CATEKV_ERR_INVALID_ARG, "KV head %d selected twice", heads[i]);
    seen[heads[i]] = 1;
  }
  return CATEKV_OK;
}

// Checks shared by selection and compaction (window, chunking, budget, heads).
int check_window(int hkv, int l_obs, int64_t n, int cs, const int32_t* heads, int n_sel, int b, int min_l_obs = 1) {
  if (l_obs < min_l_obs) return fail(CATEKV_ERR_INVALID_ARG, "l_obs=%d must be >= %d", l_obs, min_l_obs);
  if ((int64_t)l_obs >= n) return fail(CATEKV_ERR_INVALID_ARG, "l_obs=%d must be below n=%lld", l_obs, (long long)n);
  if (n > INT32_MAX) return fail(CATEKV_ERR_UNSUPPORTED, "n=%lld above 2^31 - 1", (long long)n);
  if (cs < 1) return fail(CATEKV_ERR_INVALID_ARG, "chunk size %d must be >= 1", cs);
  if (b < 1) return fail(CATEKV_ERR_INVALID_ARG, "chunk budget %d must be >= 1", b);
  if ((int64_t)b * cs + l_obs > INT32_MAX) return fail(CATEKV_ERR_UNSUPPORTED, "compact capacity above 2^31 - 1");
  return check_head_list(hkv, heads, n_sel);
}

int check_selection(int hq, int hkv, int l_obs, int64_t n, int d, int cs, const int32_t* heads,
                    int n_sel, int b) {
  int rc = check_heads(hq, hkv, d);
  if (rc) return rc;
  rc = check_window(hkv, l_obs, n, cs, heads, n_sel, b);
  if (rc) return rc;
  if ((hq / hkv) * l_obs > kMaxRows)
    return fail(CATEKV_ERR_UNSUPPORTED, "G * l_obs = %d rows above %d", (hq / hkv) * l_obs, kMaxRows);
  return CATEKV_OK;
}

catekv::SelectGeom select_geom(int hq, int hkv, int l_obs, int64_t n, int cs, const int32_t* heads,
                               int n_sel, int b) {
  catekv::SelectGeom g{};
  g.hq = hq; g.hkv = hkv; g.G = hq / hkv; g.l_obs = l_obs; g.cs = cs; g.n_sel = n_sel; g.b = b;
  g.n = n;
  g.n_keys = n - l_obs;
  g.n_chunks = (g.n_keys + cs - 1) / cs;
  g.cb_tokens = catekv::score_block_tokens(g.n_keys, n_sel, catekv::score_rows_pad(g.G * l_obs), device_cus());
  g.n_colblk = (int)((std::max<int64_t>(g.n_keys, 1) + g.cb_tokens - 1) / g.cb_tokens);
  for (int i = 0; i < n_sel && heads; ++i) g.heads[i] = heads[i];
  return g;
}

catekv::ScoreGeom score_geom(int hq, int hkv, int lq, int64_t n, int64_t l_init, int64_t l_rec) {
  catekv::ScoreGeom g{};
  g.hq = hq; g.hkv = hkv; g.G = hkv > 0 ? hq / hkv : 1; g.lq = lq; g.n = n;
  g.l_init = l_init; g.l_rec = l_rec;
  g.n_keys = n - l_init - l_rec;
  g.cb_tokens = catekv::score_block_tokens(g.n_keys, hkv, catekv::score_rows_pad(g.G * lq), device_cus());
  g.n_colblk = (int)((std::max<int64_t>(g.n_keys, 1) + g.cb_tokens - 1) / g.cb_tokens);
  return g;
}

}  // namespace

extern "C" {

const char* catekv_last_error(void) { return g_err.c_str(); }

const char* catekv_version(void) { return "catekv-mi355x 0.1 (gfx950)"; }

size_t catekv_score_heads_workspace(int hq, int hkv, int lq, int64_t n, int64_t l_init, int64_t l_rec) {
  if (hkv < 1 || hq < 1 || lq < 1 || n - l_init - l_rec < 1) return 0;
  return catekv::score_workspace_bytes(score_geom(hq, hkv, lq, n, l_init, l_rec));
}

int catekv_score_heads(int dtype, const void* q_rows, int64_t q_pos0, const void* k, int hq, int hkv,
                       int lq, int64_t n, int d, int64_t l_init, int64_t l_rec, double k_pct,
                       double alpha, int causal, float* cv_out, void* ws, size_t ws_bytes,
                       void* stream) {
  if (!valid_dtype(dtype)) return fail(CATEKV_ERR_UNSUPPORTED, "dtype %d unsupported", dtype);
  if (!q_rows || !k || !cv_out) return fail(CATEKV_ERR_INVALID_ARG, "null tensor pointer");
  int rc = check_heads(hq, hkv, d);
  if (rc) return rc;
  if (lq < 1) return fail(CATEKV_ERR_INVALID_ARG, "lq=%d must be >= 1", lq);
  if (l_init < 0 || l_rec < 0) return fail(CATEKV_ERR_INVALID_ARG, "l_init and l_rec must be >= 0");
  if (l_init + l_rec >= n) return fail(CATEKV_ERR_INVALID_ARG, "l_init + l_rec = %lld leaves no key of n=%lld",
                                       (long long)(l_init + l_rec), (long long)n);
  if (n > INT32_MAX) return fail(CATEKV_ERR_UNSUPPORTED, "n=%lld above 2^31 - 1", (long long)n);
  if (!(k_pct >= 0.0 && k_pct <= 1.0)) return fail(CATEKV_ERR_INVALID_ARG, "k_pct=%g outside [0, 1]", k_pct);
  if (!(alpha > 0.0) || !std::isfinite(alpha)) return fail(CATEKV_ERR_INVALID_ARG, "alpha=%g must be > 0", alpha);
  if (causal && q_pos0 < l_init)
    return fail(CATEKV_ERR_INVALID_ARG, "q_pos0=%lld < l_init=%lld leaves a row with no visible key",
                (long long)q_pos0, (long long)l_init);
  if ((hq / hkv) * lq > kMaxRows)
    return fail(CATEKV_ERR_UNSUPPORTED, "G * lq = %d rows above %d", (hq / hkv) * lq, kMaxRows);
  if ((int64_t)lq * (n - l_init - l_rec) > (int64_t)INT32_MAX * 2)
    return fail(CATEKV_ERR_UNSUPPORTED, "observation matrix too large");
  catekv::ScoreGeom g = score_geom(hq, hkv, lq, n, l_init, l_rec);
  g.q_pos0 = q_pos0;
  g.causal = causal ? 1 : 0;
  g.k_pct = k_pct;
  g.alpha = alpha;
  rc = check_ws(ws, ws_bytes, catekv::score_workspace_bytes(g));
  if (rc) return rc;
  hipError_t e = catekv::launch_score(dtype, g, q_rows, k, cv_out, ws, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "score_heads launch");
  return ok();
}

int catekv_adaptive_budget(int64_t n, int l_obs, int cs, double eta, int64_t* b_out) {
  if (!b_out) return fail(CATEKV_ERR_INVALID_ARG, "b_out is null");
  if (l_obs < 0 || (int64_t)l_obs >= n) return fail(CATEKV_ERR_INVALID_ARG, "l_obs=%d outside [0, n=%lld)", l_obs, (long long)n);
  if (cs < 1) return fail(CATEKV_ERR_INVALID_ARG, "chunk size %d must be >= 1", cs);
  if (!(eta >= 0.0 && eta <= 1.0)) return fail(CATEKV_ERR_INVALID_ARG, "eta=%g outside [0, 1]", eta);
  const int64_t nc = (n - l_obs + cs - 1) / cs;
  // eta is the decimal ratio the caller means: a product within 1e-9
  // (relative) of an integer is that integer, so the binary representation
  // of, e.g., 0.1 or 0.3 neither adds nor drops a chunk
  const double p = eta * (double)nc;
  const double r = std::nearbyint(p);
  const int64_t b = std::fabs(p - r) <= 1e-9 * std::max(1.0, p) ? (int64_t)r : (int64_t)std::ceil(p);
  *b_out = std::min<int64_t>(std::max<int64_t>(b, 0), nc);
  return ok();
}

int catekv_classify_heads(const float* cv_host, int S, int H, double r, uint8_t* is_consistent_host) {
  if (!cv_host || !is_consistent_host) return fail(CATEKV_ERR_INVALID_ARG, "null pointer");
  if (S < 1 || H < 1) return fail(CATEKV_ERR_INVALID_ARG, "S=%d H=%d must be >= 1", S, H);
  if (!(r >= 0.0 && r < 1.0)) return fail(CATEKV_ERR_INVALID_ARG, "r=%g outside [0, 1)", r);
  std::vector<double> freq(H, 0.0), mean(H, 0.0);
  for (int s = 0; s < S; ++s) {
    std::vector<double> row(cv_host + (size_t)s * H, cv_host + (size_t)(s + 1) * H);
    const double gamma = quantile_linear(row, r);
    for (int h = 0; h < H; ++h) {
      if (row[h] > gamma) freq[h] += 1.0;
      mean[h] += row[h];
    }
  }
  std::vector<int> order(H);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) {
    if (freq[a] != freq[b]) return freq[a] > freq[b];
    if (mean[a] != mean[b]) return mean[a] > mean[b];
    return a < b;
  });
  const int n_cons = H - 1 - (int)std::floor((double)(H - 1) * r);
  for (int h = 0; h < H; ++h) is_consistent_host[h] = 0;
  for (int i = 0; i < n_cons; ++i) is_consistent_host[order[i]] = 1;
  return ok();
}

size_t catekv_select_workspace(int hq, int hkv, int l_obs, int64_t n, int cs, int n_sel) {
  if (hkv < 1 || hq < 1 || l_obs < 1 || (int64_t)l_obs >= n || cs < 1 || n_sel < 1) return 0;
  return catekv::select_workspace_bytes(select_geom(hq, hkv, l_obs, n, cs, nullptr, n_sel, 1));
}

int catekv_select_critical(int dtype, const void* q_obs, const void* k, int hq, int hkv, int l_obs,
                           int64_t n, int d, int cs, const int32_t* sel_heads_host, int n_sel, int b,
                           int32_t* idx_out, void* ws, size_t ws_bytes, void* stream) {
  if (!valid_dtype(dtype)) return fail(CATEKV_ERR_UNSUPPORTED, "dtype %d unsupported", dtype);
  if (!q_obs || !k || !idx_out) return fail(CATEKV_ERR_INVALID_ARG, "null tensor pointer");
  int rc = check_selection(hq, hkv, l_obs, n, d, cs, sel_heads_host, n_sel, b);
  if (rc) return rc;
  const catekv::SelectGeom g = select_geom(hq, hkv, l_obs, n, cs, sel_heads_host, n_sel, b);
  rc = check_ws(ws, ws_bytes, catekv::select_workspace_bytes(g));
  if (rc) return rc;
  hipError_t e = catekv::launch_select(dtype, g, q_obs, k, idx_out, ws, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "select_critical launch");
  return ok();
}

int catekv_select_critical_noalloc(int dtype, const void* q_obs, const void* k, int hq, int hkv, int l_obs,
                                   int64_t n, int d, int cs, const int32_t* sel_heads_host, int n_sel, int b,
                                   int32_t* idx_out, void* stream) {
  if (!valid_dtype(dtype)) return fail(CATEKV_ERR_UNSUPPORTED, "dtype %d unsupported", dtype);
  if (!q_obs || !k || !idx_out) return fail(CATEKV_ERR_INVALID_ARG, "null tensor pointer");
  int rc = check_selection(hq, hkv, l_obs, n, d, cs, sel_heads_host, n_sel, b);
  if (rc) return rc;
  const catekv::SelectGeom g = select_geom(hq, hkv, l_obs, n, cs, sel_heads_host, n_sel, b);
  const size_t need = catekv::select_workspace_bytes(g), have = catekv::select_scratch_bytes();
  if (need > have)
    return fail(CATEKV_ERR_UNSUPPORTED,
                "this selection needs %zu bytes of scratch; the allocation-free call holds %zu "
                "(use catekv_select_critical with a workspace)", need, have);
  void* ws = nullptr;
  hipError_t e = catekv::select_scratch(&ws);
  if (e != hipSuccess) return hip_fail(e, "select_critical_noalloc scratch address");
  e = catekv::launch_select(dtype, g, q_obs, k, idx_out, ws, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "select_critical_noalloc launch");
  return ok();
}

int catekv_compact_kv(int dtype, const void* k, const void* v, int hkv, int64_t n, int d, int cs,
                      int l_obs, const int32_t* sel_heads_host, int n_sel, const int32_t* idx, int b,
                      void* k_c, void* v_c, int64_t* lens_out, void* stream) {
  if (!valid_dtype(dtype)) return fail(CATEKV_ERR_UNSUPPORTED, "dtype %d unsupported", dtype);
  if (!k || !v || !idx || !k_c || !v_c || !lens_out) return fail(CATEKV_ERR_INVALID_ARG, "null tensor pointer");
  int rc = check_heads(hkv, hkv, d);
  if (rc) return rc;
  rc = check_window(hkv, l_obs, n, cs, sel_heads_host, n_sel, b, 0);
  if (rc) return rc;
  hipError_t e = catekv::launch_compact(dtype, k, v, hkv, n, cs, l_obs, sel_heads_host, n_sel, idx, b, k_c,
                                        v_c, lens_out, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "compact_kv launch");
  return ok();
}

size_t catekv_decode_workspace(const int64_t* max_len_host, int batch, int hq, int hkv, int split_tokens) {
  if (!max_len_host || batch < 1 || hkv < 1 || hq < 1 || hq % hkv) return 0;
  const int nv = batch * hkv;
  for (int i = 0; i < nv; ++i)
    if (max_len_host[i] < 0 || max_len_host[i] > INT32_MAX) return 0;
  int variant = 0;
  return choose_plan(max_len_host, nv, hq / hkv, split_tokens, &variant).total;
}

int catekv_decode_plan(const int64_t* max_len_host, int batch, int hq, int hkv, int split_tokens,
                       catekv_decode_plan_t* plan, void* ws, size_t ws_bytes, void* stream) {
  if (!max_len_host || !plan) return fail(CATEKV_ERR_INVALID_ARG, "null pointer");
  if (batch < 1) return fail(CATEKV_ERR_INVALID_ARG, "batch=%d must be >= 1", batch);
  int rc = check_heads(hq, hkv, catekv::kD);
  if (rc) return rc;
  const int nv = batch * hkv;
  rc = check_lengths(max_len_host, nv);
  if (rc) return rc;
  if (!ws) return fail(CATEKV_ERR_WORKSPACE, "workspace pointer is null");
  const int G = hq / hkv;
  int variant = 0;
  const PlanLayout P = choose_plan(max_len_host, nv, G, split_tokens, &variant);
  rc = check_ws(ws, ws_bytes, P.total);
  if (rc) return rc;

  std::vector<catekv::DecodeItem> segs(P.n_segments);
  std::vector<int32_t> wseg(P.n_workers + 1, 0);
  std::vector<catekv::ViewInfo> views(nv);
  std::vector<int> parts(nv, 0);
  for (const Segment& s : P.segs) parts[s.view]++;
  int slot = 0;
  int64_t total = 0;
  for (int v = 0; v < nv; ++v) {
    total += max_len_host[v];
    views[v].first_slot = slot;
    views[v].n_parts = parts[v];
    slot += parts[v];
  }
  std::vector<int> next_part(nv, 0);
  for (int i = 0; i < P.n_segments; ++i) {
    const Segment& s = P.segs[i];
    segs[i] = {s.view, next_part[s.view]++, (int32_t)s.t0, (int32_t)s.t1};
    wseg[s.worker + 1] = i + 1;
  }
  for (int w = 1; w <= P.n_workers; ++w) wseg[w] = std::max(wseg[w], wseg[w - 1]);
  std::vector<catekv::V2Item> v2((size_t)P.n_workers * catekv::kDecodeV2MaxSeg, catekv::V2Item{0, 0, 0, -1});
  if (variant == catekv::kDecodeStreamV2) {
    // every entry of a worker, padding included, carries the worker's segment count
    for (int w = 0; w < P.n_workers; ++w) {
      const int ns = wseg[w + 1] - wseg[w];   // in [1, kDecodeV2MaxSeg] for this variant
      for (int j = 0; j < catekv::kDecodeV2MaxSeg; ++j) {
        catekv::V2Item& e = v2[(size_t)w * catekv::kDecodeV2MaxSeg + j];
        if (j < ns) {
          const catekv::DecodeItem& it = segs[wseg[w] + j];
          const catekv::ViewInfo& vi = views[it.bh];
          e = catekv::V2Item{it.bh, it.t0, it.t1, vi.n_parts > 1 ? vi.first_slot + it.part : -1};
        }
        e.bh_n |= ns << 24;
      }
    }
  }

  std::vector<unsigned char> host(P.slots_off, 0);
  std::memcpy(host.data() + P.segs_off, segs.data(), segs.size() * sizeof(catekv::DecodeItem));
  std::memcpy(host.data() + P.workers_off, wseg.data(), wseg.size() * sizeof(int32_t));
  std::memcpy(host.data() + P.views_off, views.data(), views.size() * sizeof(catekv::ViewInfo));
  std::memcpy(host.data() + v2_items_off(P.segs_off, P.n_segments), v2.data(), v2.size() * sizeof(catekv::V2Item));
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = hipMemcpyAsync(ws, host.data(), host.size(), hipMemcpyHostToDevice, s);
  if (e != hipSuccess) return hip_fail(e, "decode_plan upload");
  e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "decode_plan synchronize");

  std::memset(plan, 0, sizeof *plan);
  plan->magic = kPlanMagic;
  plan->batch = batch;
  plan->hq = hq;
  plan->hkv = hkv;
  plan->split_tokens = split_tokens;
  plan->n_workers = P.n_workers;
  plan->n_segments = P.n_segments;
  plan->n_slots = P.n_slots;
  plan->n_multi = P.n_multi;
  plan->variant = variant;
  plan->segs_off = P.segs_off;
  plan->workers_off = P.workers_off;
  plan->views_off = P.views_off;
  plan->slots_off = P.slots_off;
  plan->ws_bytes = P.total;
  plan->max_len_total = total;
  return ok();
}

int catekv_decode_attn(int dtype, const catekv_decode_plan_t* plan, const void* q, const catekv_kv_ptrs* kv,
                       const int64_t* lens, int batch, int hq, int hkv, int d, float scale, float* out,
                       float* lse, void* ws, size_t ws_bytes, void* stream) {
  if (!valid_dtype(dtype)) return fail(CATEKV_ERR_UNSUPPORTED, "dtype %d unsupported", dtype);
  if (!plan || plan->magic != kPlanMagic) return fail(CATEKV_ERR_INVALID_ARG, "plan missing or not built by catekv_decode_plan");
  if (!q || !kv || !lens || !out) return fail(CATEKV_ERR_INVALID_ARG, "null tensor pointer");
  int rc = check_heads(hq, hkv, d);
  if (rc) return rc;
  if (plan->batch != batch || plan->hq != hq || plan->hkv != hkv)
    return fail(CATEKV_ERR_INVALID_ARG, "shapes (batch=%d hq=%d hkv=%d) differ from the plan (%d, %d, %d)", batch, hq,
                hkv, plan->batch, plan->hq, plan->hkv);
  if (!(scale > 0.f) || !std::isfinite(scale))
    return fail(CATEKV_ERR_INVALID_ARG, "scale=%g must be positive and finite", (double)scale);
  rc = check_ws(ws, ws_bytes, plan->ws_bytes);
  if (rc) return rc;
  char* w = reinterpret_cast<char*>(ws);
  catekv::DecodeArgs a{};
  a.q = q;
  a.kv = kv;
  a.lens = lens;
  a.items = reinterpret_cast<const catekv::DecodeItem*>(w + plan->segs_off);
  a.worker_seg = reinterpret_cast<const int32_t*>(w + plan->workers_off);
  a.v2items = reinterpret_cast<const catekv::V2Item*>(w + v2_items_off(plan->segs_off, plan->n_segments));
  a.views = reinterpret_cast<const catekv::ViewInfo*>(w + plan->views_off);
  a.slots = reinterpret_cast<float*>(w + plan->slots_off);
  a.n_workers = plan->n_workers;
  a.n_multi = plan->n_multi;
  a.n_views = batch * hkv;
  a.hkv = hkv;
  a.variant = plan->variant;
  a.scale = scale;
  a.out = out;
  a.lse = lse;
  hipError_t e = catekv::launch_decode(dtype, hq / hkv, a, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "decode_attn launch");
  return ok();
}

int catekv_page_bounds(int dtype, const void* k, int hkv, int64_t n, int d, int cs, const int32_t* heads_host,
                       int n_sel, void* kmin, void* kmax, void* stream) {
  if (!valid_dtype(dtype)) return fail(CATEKV_ERR_UNSUPPORTED, "dtype %d unsupported", dtype);
  if (!k || !kmin || !kmax) return fail(CATEKV_ERR_INVALID_ARG, "null tensor pointer");
  int rc = check_heads(hkv, hkv, d);
  if (rc) return rc;
  if (n < 1) return fail(CATEKV_ERR_INVALID_ARG, "n=%lld must be >= 1", (long long)n);
  if (n > INT32_MAX) return fail(CATEKV_ERR_UNSUPPORTED, "n=%lld above 2^31 - 1", (long long)n);
  if (cs < 1) return fail(CATEKV_ERR_INVALID_ARG, "chunk size %d must be >= 1", cs);
  rc = check_head_list(hkv, heads_host, n_sel);
  if (rc) return rc;
  hipError_t e = catekv::launch_page_bounds(dtype, k, n, cs, heads_host, n_sel, kmin, kmax,
                                            reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "page_bounds launch");
  return ok();
}

size_t catekv_retrieve_workspace(int n_sel, int64_t n_pages) {
  if (n_sel < 1 || n_pages < 1) return 0;
  return a256((size_t)n_sel * (size_t)n_pages * sizeof(float)) + a256(catekv::topk_workspace_bytes(n_sel, n_pages));
}

int catekv_retrieve_pages(int dtype, const void* q, const void* kmin, const void* kmax, int hq, int hkv,
                          int64_t n_pages, int d, const int32_t* heads_host, int n_sel, int n_keep,
                          int32_t* idx_out, void* ws, size_t ws_bytes, void* stream) {
  if (!valid_dtype(dtype)) return fail(CATEKV_ERR_UNSUPPORTED, "dtype %d unsupported", dtype);
  if (!q || !kmin || !kmax || !idx_out) return fail(CATEKV_ERR_INVALID_ARG, "null tensor pointer");
  int rc = check_heads(hq, hkv, d);
  if (rc) return rc;
  if (n_pages < 1) return fail(CATEKV_ERR_INVALID_ARG, "n_pages=%lld must be >= 1", (long long)n_pages);
  if (n_pages > INT32_MAX) return fail(CATEKV_ERR_UNSUPPORTED, "n_pages above 2^31 - 1");
  if (n_keep < 1) return fail(CATEKV_ERR_INVALID_ARG, "n_keep=%d must be >= 1", n_keep);
  rc = check_head_list(hkv, heads_host, n_sel);
  if (rc) return rc;
  rc = check_ws(ws, ws_bytes, catekv_retrieve_workspace(n_sel, n_pages));
  if (rc) return rc;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  float* scores = reinterpret_cast<float*>(ws);
  char* topk_ws = reinterpret_cast<char*>(ws) + a256((size_t)n_sel * (size_t)n_pages * sizeof(float));
  // the page-score launch clears the top-k's arrival counters (its first n_sel words)
  hipError_t e = catekv::launch_page_scores(dtype, hq / hkv, q, kmin, kmax, n_pages, heads_host, n_sel, scores,
                                            reinterpret_cast<uint32_t*>(topk_ws), n_sel, s);
  if (e == hipSuccess) e = catekv::launch_topk(scores, n_sel, n_pages, n_keep, idx_out, topk_ws, s);
  if (e != hipSuccess) return hip_fail(e, "retrieve_pages launch");
  return ok();
}

int catekv_append_kv(int dtype, const catekv_kv_ptrs* kv, const int64_t* capacity, int64_t* lens,
                     const void* k_new, const void* v_new, int batch, int hkv, int d, int32_t* overflow,
                     void* stream) {
  if (!valid_dtype(dtype)) return fail(CATEKV_ERR_UNSUPPORTED, "dtype %d unsupported", dtype);
  if (!kv || !capacity || !lens || !k_new || !v_new) return fail(CATEKV_ERR_INVALID_ARG, "null tensor pointer");
  if (batch < 1 || hkv < 1) return fail(CATEKV_ERR_INVALID_ARG, "batch=%d hkv=%d must be >= 1", batch, hkv);
  if (d != catekv::kD) return fail(CATEKV_ERR_INVALID_ARG, "d=%d unsupported (d must be %d)", d, catekv::kD);
  if ((int64_t)batch * hkv > (int64_t)INT32_MAX) return fail(CATEKV_ERR_INVALID_ARG, "batch * hkv too large");
  catekv::AppendArgs a{};
  a.kv = kv;
  a.capacity = capacity;
  a.lens = lens;
  a.k_new = k_new;
  a.v_new = v_new;
  a.overflow = overflow;
  a.n_views = batch * hkv;
  hipError_t e = catekv::launch_append(dtype, a, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "append_kv launch");
  return ok();
}

}  // extern "C"
