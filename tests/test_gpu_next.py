"""GPU parity of the extensions around the core path: the decode-time KV
append of a generation loop, adaptive retention below 1 and query-aware
retrieval in the adaptive heads, each against the oracle."""
import math
import sys

import numpy as np
import pytest
import torch

import oracle as O
import paper_2608_30295_amd as ck
import synth
from gpu_util import DEV, assert_rows_close, f64, to_dev, to_host_storage

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _storage(x, dtype):
    return synth.f32_to_bf16_bits(x) if dtype == "bf16" else x.astype(np.float32)


# ------------------------------------------------------------ KV append

@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_append_then_decode_growing_cache(dtype):
    """A generation loop: every step appends one token to every view (compact
    or full alike) and decodes over the grown caches with one plan built at
    capacity; a view that reaches capacity stops growing and raises the
    overflow flag."""
    rng = np.random.default_rng(21)
    B, hq, hkv, d, steps = 2, 8, 2, 128, 20
    lens0 = np.array([100, 2500, 0, 37], dtype=np.int64)
    cap = lens0 + np.array([24, 24, 24, 5])
    say(f"append/decode {dtype}: lens {lens0.tolist()} capacity {cap.tolist()}")
    host_k, host_v, dev_k, dev_v = [], [], [], []
    for L, C in zip(lens0, cap):
        k = _storage(rng.standard_normal((C, d), dtype=np.float32), dtype)
        v = _storage(rng.standard_normal((C, d), dtype=np.float32), dtype)
        host_k.append(k[:L].copy())
        host_v.append(v[:L].copy())
        dev_k.append(to_dev(k))          # rows past L hold stale data the decode must never read
        dev_v.append(to_dev(v))
    table = ck.kv_table([(k.data_ptr(), v.data_ptr()) for k, v in zip(dev_k, dev_v)], DEV)
    capacity = torch.from_numpy(cap).to(DEV)
    lens = torch.from_numpy(lens0.copy()).to(DEV)
    overflow = torch.zeros(1, dtype=torch.int32, device=DEV)
    plan = ck.decode_plan(cap.reshape(B, hkv), hq, hkv, DEV, split_tokens=256)
    for t in range(steps):
        k_new = _storage(rng.standard_normal((B, hkv, d), dtype=np.float32), dtype)
        v_new = _storage(rng.standard_normal((B, hkv, d), dtype=np.float32), dtype)
        ck.append_kv(table, capacity, lens, to_dev(k_new), to_dev(v_new), overflow)
        for i in range(B * hkv):
            host_k[i], host_v[i], _ = O.append_token(host_k[i], host_v[i], k_new.reshape(-1, d)[i],
                                                     v_new.reshape(-1, d)[i], int(cap[i]))
        q = _storage(rng.standard_normal((B, hq, d), dtype=np.float32), dtype)
        out, lse = ck.decode_attn(plan, to_dev(q), table, lens.view(B, hkv))
        torch.cuda.synchronize()
        assert lens.cpu().numpy().tolist() == [h.shape[0] for h in host_k]
        out, lse = out.cpu().numpy(), lse.cpu().numpy()
        for b in range(B):
            views = [(f64(host_k[b * hkv + h]), f64(host_v[b * hkv + h])) for h in range(hkv)]
            o_ref, l_ref = O.decode_gqa(f64(q)[b], views)
            assert_rows_close(out[b], o_ref, dtype, f"step {t} b={b}")
            np.testing.assert_allclose(lse[b], l_ref, atol=1e-4, rtol=0)
    assert int(overflow.item()) == 1
    assert lens.cpu().numpy().tolist() == (lens0 + np.minimum(steps, cap - lens0)).tolist()
    for i in range(B * hkv):
        L = host_k[i].shape[0]
        assert np.array_equal(to_host_storage(dev_k[i])[:L], host_k[i])
        assert np.array_equal(to_host_storage(dev_v[i])[:L], host_v[i])


def test_append_without_overflow_leaves_flag_clear():
    rng = np.random.default_rng(22)
    k = torch.zeros(3, 128, dtype=torch.bfloat16, device=DEV)
    v = torch.zeros(3, 128, dtype=torch.bfloat16, device=DEV)
    table = ck.kv_table([(k.data_ptr(), v.data_ptr())], DEV)
    cap = torch.tensor([3], dtype=torch.int64, device=DEV)
    lens = torch.tensor([1], dtype=torch.int64, device=DEV)
    flag = torch.zeros(1, dtype=torch.int32, device=DEV)
    row = synth.f32_to_bf16_bits(rng.standard_normal((1, 1, 128), dtype=np.float32))
    ck.append_kv(table, cap, lens, to_dev(row), to_dev(row), flag)
    ck.append_kv(table, cap, lens, to_dev(row), to_dev(row), flag)
    torch.cuda.synchronize()
    assert int(lens.item()) == 3 and int(flag.item()) == 0
    ck.append_kv(table, cap, lens, to_dev(row), to_dev(row), None)     # full: unchanged, no flag to set
    torch.cuda.synchronize()
    assert int(lens.item()) == 3
    assert np.array_equal(to_host_storage(k)[1], row[0, 0]) and np.array_equal(to_host_storage(k)[2], row[0, 0])


# --------------------------------------------- adaptive retention below 1

@pytest.mark.parametrize("eta", [0.5, 0.3, 0.05])
def test_retention_below_one(eta):
    """Adaptive heads keep ceil(eta * chunks) chunks (argtopk(C_chunk, n eta)
    of Algorithm 1) through the same selection and compaction kernels;
    decoding then runs over compact views for every head."""
    wl = synth.WORKLOADS["ctx32k_bf16"].scaled(n=20000 + 64 + 5)
    seq = synth.make_sequence(wl)
    n, G = seq.n, wl.group
    adaptive, consistent = [0, 3, 6], [1, 2, 4, 5, 7]
    ba = ck.adaptive_budget(n, wl.l_obs, wl.cs, eta)
    say(f"retention eta={eta}: {ba} of {-(-(n - wl.l_obs) // wl.cs)} chunks per adaptive head")
    q_obs, k, v = to_dev(seq.q_obs), to_dev(seq.k), to_dev(seq.v)
    lens = torch.full((wl.hkv,), n, dtype=torch.int64, device=DEV)
    idx_c = ck.select_critical(q_obs, k, consistent, wl.cs, wl.chunk_budget)
    kc, vc = ck.compact_kv(k, v, consistent, idx_c, wl.cs, wl.l_obs, lens)
    idx_a = ck.select_critical(q_obs, k, adaptive, wl.cs, ba)
    ka, va = ck.compact_kv(k, v, adaptive, idx_a, wl.cs, wl.l_obs, lens)
    torch.cuda.synchronize()
    idx_a_h, idx_c_h = idx_a.cpu().numpy(), idx_c.cpu().numpy()
    qf, scale = f64(seq.q_obs), 1 / math.sqrt(128)
    from gpu_util import check_topk
    for s, h in enumerate(adaptive):
        sc = O.chunk_scores(qf[h * G:(h + 1) * G], f64(seq.k[h:h + 1]), 0, G, wl.l_obs, wl.cs, scale)
        check_topk(idx_a_h[s], sc, ba)
    ka_h, va_h = to_host_storage(ka), to_host_storage(va)
    lens_h = lens.cpu().numpy()
    rows = {}
    for heads_, idx_h, kk, vv in ((adaptive, idx_a_h, ka_h, va_h), (consistent, idx_c_h, None, None)):
        for s, h in enumerate(heads_):
            sel = idx_h[s][idx_h[s] >= 0]
            rows[h] = O.compact_rows(n, wl.l_obs, wl.cs, sel)
            assert lens_h[h] == rows[h].size
            if kk is not None:
                assert np.array_equal(kk[s][:rows[h].size], seq.k[h][rows[h]])
                assert np.array_equal(vv[s][:rows[h].size], seq.v[h][rows[h]])
    pairs, maxlen = [], []
    for h in range(wl.hkv):
        kt, vt = (ka[adaptive.index(h)], va[adaptive.index(h)]) if h in adaptive else \
            (kc[consistent.index(h)], vc[consistent.index(h)])
        pairs.append((kt.data_ptr(), vt.data_ptr()))
        maxlen.append(kt.shape[0])
    plan = ck.decode_plan(np.array([maxlen]), wl.hq, wl.hkv, DEV)
    q_st = synth.decode_queries(wl, 3)
    out, lse = ck.decode_attn(plan, to_dev(q_st), ck.kv_table(pairs, DEV), lens.view(1, -1))
    torch.cuda.synchronize()
    views = [(f64(seq.k[h][rows[h]]), f64(seq.v[h][rows[h]])) for h in range(wl.hkv)]
    o_ref, l_ref = O.decode_gqa(f64(q_st)[0], views)
    assert_rows_close(out.cpu().numpy()[0], o_ref, "bf16", f"eta={eta}")
    np.testing.assert_allclose(lse.cpu().numpy()[0], l_ref, atol=1e-4, rtol=0)


# ------------------------------------- query-aware retrieval (adaptive heads)

@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_page_bounds(dtype):
    rng = np.random.default_rng(31)
    k = _storage(rng.standard_normal((3, 1003, 128), dtype=np.float32), dtype)   # ragged last page
    say(f"page bounds {dtype}")
    kmin, kmax = ck.page_bounds(to_dev(k), [2, 0], 8)
    torch.cuda.synchronize()
    got_min, got_max = f64(to_host_storage(kmin)), f64(to_host_storage(kmax))
    for s, h in enumerate([2, 0]):
        mn, mx = O.page_bounds(f64(k[h]), 8)
        assert np.array_equal(got_min[s], mn) and np.array_equal(got_max[s], mx)


@pytest.mark.parametrize("dtype,n_keep", [("bf16", 64), ("f32", 64), ("bf16", 3000)])
def test_retrieve_gather_decode(dtype, n_keep):
    """One decode step with query-aware retrieval in the adaptive heads: page
    scores and top pages against the oracle, the gathered rows bitwise, and
    attention over them."""
    name = "ctx32k_bf16" if dtype == "bf16" else "ctx4k_f32"
    wl = synth.WORKLOADS[name].scaled(n=20000 + 3 if dtype == "bf16" else 4096)
    seq = synth.make_sequence(wl)
    n, G, cs = seq.n, wl.group, wl.cs
    adaptive = [0, 3, 6] if wl.hkv == 8 else [0, 2]
    n_pages = -(-n // cs)
    say(f"retrieve {dtype}: n={n} pages={n_pages} keep={n_keep} heads={adaptive}")
    k, v = to_dev(seq.k), to_dev(seq.v)
    kmin, kmax = ck.page_bounds(k, adaptive, cs)
    q_st = synth.decode_queries(wl, 5)
    idx = ck.retrieve_pages(to_dev(q_st)[0], kmin, kmax, adaptive, wl.hkv, n_keep)
    lens = torch.full((wl.hkv,), n, dtype=torch.int64, device=DEV)
    kg, vg = ck.compact_kv(k, v, adaptive, idx, cs, 0, lens)
    torch.cuda.synchronize()
    idx_h, lens_h = idx.cpu().numpy(), lens.cpu().numpy()
    kg_h, vg_h = to_host_storage(kg), to_host_storage(vg)
    qf = f64(q_st)[0]
    from gpu_util import check_topk
    rows = {}
    for s, h in enumerate(adaptive):
        mn, mx = O.page_bounds(f64(seq.k[h]), cs)
        sc = O.page_scores(qf[h * G:(h + 1) * G], mn, mx)
        swaps = check_topk(idx_h[s], sc, n_keep)
        sel = idx_h[s][idx_h[s] >= 0]
        rows[h] = O.chunk_rows(n, cs, sel)
        assert lens_h[h] == rows[h].size
        assert np.array_equal(kg_h[s][:rows[h].size], seq.k[h][rows[h]])
        assert np.array_equal(vg_h[s][:rows[h].size], seq.v[h][rows[h]])
        say(f"  head {h}: {sel.size} pages, {swaps} swaps inside the band")
    pairs, maxlen = [], []
    for h in range(wl.hkv):
        kt, vt = (kg[adaptive.index(h)], vg[adaptive.index(h)]) if h in adaptive else (k[h], v[h])
        pairs.append((kt.data_ptr(), vt.data_ptr()))
        maxlen.append(kt.shape[0])
    plan = ck.decode_plan(np.array([maxlen]), wl.hq, wl.hkv, DEV)
    out, lse = ck.decode_attn(plan, to_dev(q_st), ck.kv_table(pairs, DEV), lens.view(1, -1))
    torch.cuda.synchronize()
    views = [(f64(seq.k[h][rows[h]]), f64(seq.v[h][rows[h]])) if h in adaptive else (f64(seq.k[h]), f64(seq.v[h]))
             for h in range(wl.hkv)]
    o_ref, l_ref = O.decode_gqa(qf, views)
    assert_rows_close(out.cpu().numpy()[0], o_ref, dtype, "retrieval decode")
    np.testing.assert_allclose(lse.cpu().numpy()[0], l_ref, atol=1e-4, rtol=0)


def test_retrieve_more_pages_than_exist():
    rng = np.random.default_rng(33)
    k = to_dev(synth.f32_to_bf16_bits(rng.standard_normal((1, 50, 128), dtype=np.float32)))
    q = to_dev(synth.f32_to_bf16_bits(rng.standard_normal((4, 128), dtype=np.float32)))
    kmin, kmax = ck.page_bounds(k, [0], 8)
    idx = ck.retrieve_pages(q, kmin, kmax, [0], 1, 10).cpu().numpy()
    assert idx[0].tolist() == list(range(7)) + [-1, -1, -1]


@pytest.mark.parametrize("n_pages,n_keep", [(9000, 700), (20000, 700), (40000, 700), (40000, 15000),
                                            (4097, 300), (12289, 1), (16384, 256), (32768, 512)])
def test_retrieve_exact_ties_lowest_pages_first(n_pages, n_keep):
    """Pages repeat 37 random patterns, so page scores tie exactly in groups
    and the k-th score falls inside a group: the chosen pages must be the
    oracle's (ties to the lower page) on every path of the top-k: one
    workgroup per row up to 16384 and up to 32768 scores, slices then
    candidates beyond that, and the global-memory kernel when the slices'
    candidates would not fit; for short rows with k <= 512, 4096-score
    slices then candidates (a one-score last slice at 4097, k = 1, k = 512)."""
    rng = np.random.default_rng(40 + n_pages + n_keep)
    cs, G = 8, 4
    pat = synth.f32_to_bf16_bits(rng.standard_normal((37, cs, 128), dtype=np.float32))
    kk = pat[np.arange(n_pages) % 37].reshape(1, n_pages * cs, 128)
    q_st = synth.f32_to_bf16_bits(rng.standard_normal((G, 128), dtype=np.float32))
    say(f"retrieve ties: pages={n_pages} keep={n_keep}")
    kmin, kmax = ck.page_bounds(to_dev(kk), [0], cs)
    idx = ck.retrieve_pages(to_dev(q_st), kmin, kmax, [0], 1, n_keep).cpu().numpy()[0]
    mn, mx = O.page_bounds(f64(kk[0]), cs)
    sc = O.page_scores(f64(q_st), mn, mx)
    want = O.argtopk_ascending(sc, n_keep)
    kth = np.sort(sc)[::-1][n_keep - 1]
    assert (sc == kth).sum() > 1 and (sc > kth).sum() < n_keep   # the k-th lies inside a tie group
    assert idx.tolist() == want.tolist()


@pytest.mark.parametrize("n_pages,n_keep", [(70000, 3000), (100000, 3000)])
def test_retrieve_exact_ties_long_candidate_lists(n_pages, n_keep):
    """Slices then candidates with 15000 and 21000 candidates per row (the
    list stage reads the candidates' indices again when writing); the pages
    repeat 37 patterns, so the oracle scores the patterns and tiles them."""
    rng = np.random.default_rng(90 + n_pages + n_keep)
    cs, G = 8, 4
    pat = synth.f32_to_bf16_bits(rng.standard_normal((37, cs, 128), dtype=np.float32))
    kk = pat[np.arange(n_pages) % 37].reshape(1, n_pages * cs, 128)
    q_st = synth.f32_to_bf16_bits(rng.standard_normal((G, 128), dtype=np.float32))
    say(f"retrieve long lists: pages={n_pages} keep={n_keep}")
    kmin, kmax = ck.page_bounds(to_dev(kk), [0], cs)
    idx = ck.retrieve_pages(to_dev(q_st), kmin, kmax, [0], 1, n_keep).cpu().numpy()[0]
    mn, mx = O.page_bounds(f64(pat.reshape(37 * cs, 128)), cs)
    sc = O.page_scores(f64(q_st), mn, mx)[np.arange(n_pages) % 37]
    want = O.argtopk_ascending(sc, n_keep)
    kth = np.sort(sc)[::-1][n_keep - 1]
    assert (sc == kth).sum() > 1 and (sc > kth).sum() < n_keep
    assert idx.tolist() == want.tolist()


@pytest.mark.parametrize("n_pages,n_keep", [(16384, 256), (3000, 700), (30000, 1000)])
def test_retrieve_small_tie_group_at_kth(n_pages, n_keep):
    """Distinct pages except 21 equal ones that hold the k-th score: the
    top-k's last bin is small, so its keys are ranked by one wave instead of
    more radix passes, and the tie must still go to the lower pages (row
    paths at 3000 and 30000 pages, slices then candidates at 16384)."""
    rng = np.random.default_rng(500 + n_pages + n_keep)
    cs, G = 8, 4
    kk = synth.f32_to_bf16_bits(rng.standard_normal((n_pages, cs, 128), dtype=np.float32))
    q_st = synth.f32_to_bf16_bits(rng.standard_normal((G, 128), dtype=np.float32))

    def scores(pages):
        mn, mx = O.page_bounds(f64(pages.reshape(n_pages * cs, 128)), cs)
        return O.page_scores(f64(q_st), mn, mx)

    kth_page = np.argsort(-scores(kk), kind="stable")[n_keep - 1]
    dup = rng.choice(np.setdiff1d(np.arange(n_pages), [kth_page]), 20, replace=False)
    kk[dup] = kk[kth_page]
    sc = scores(kk)
    kth = np.sort(sc)[::-1][n_keep - 1]
    assert (sc == kth).sum() == 21 and (sc > kth).sum() < n_keep
    say(f"retrieve small tie group: pages={n_pages} keep={n_keep}")
    kmin, kmax = ck.page_bounds(to_dev(kk.reshape(1, n_pages * cs, 128)), [0], cs)
    idx = ck.retrieve_pages(to_dev(q_st), kmin, kmax, [0], 1, n_keep).cpu().numpy()[0]
    assert idx.tolist() == O.argtopk_ascending(sc, n_keep).tolist()


@pytest.mark.parametrize("n_pages,n_keep", [(3000, 700), (16384, 256), (30000, 1000), (40000, 700)])
def test_retrieve_all_pages_equal(n_pages, n_keep):
    """Every page the same: all scores tie, no key bit differs, so the
    top-k runs no radix pass and must return the first n_keep pages (one
    workgroup per row, 4096-score slices, 16384-score slices)."""
    rng = np.random.default_rng(600 + n_pages)
    cs, G = 8, 4
    page = synth.f32_to_bf16_bits(rng.standard_normal((1, cs, 128), dtype=np.float32))
    kk = np.repeat(page, n_pages, axis=0).reshape(1, n_pages * cs, 128)
    q_st = synth.f32_to_bf16_bits(rng.standard_normal((G, 128), dtype=np.float32))
    say(f"retrieve equal pages: pages={n_pages} keep={n_keep}")
    kmin, kmax = ck.page_bounds(to_dev(kk), [0], cs)
    idx = ck.retrieve_pages(to_dev(q_st), kmin, kmax, [0], 1, n_keep).cpu().numpy()[0]
    mn, mx = O.page_bounds(f64(page[0]), cs)
    sc = np.repeat(O.page_scores(f64(q_st), mn, mx), n_pages)
    assert idx.tolist() == O.argtopk_ascending(sc, n_keep).tolist() == list(range(n_keep))


# ---------------------------------------------------- attention recall

def test_recall_of_gpu_selection_and_retrieval_matches_oracle():
    """The recall diagnostic on the GPU's own choices: the consistent
    pattern from select_critical and the pages from retrieve_pages keep the
    same attention mass as the oracle's choices."""
    wl = synth.WORKLOADS["ctx4k_f32"]
    seq = synth.make_sequence(wl)
    n, G, cs, l_obs, b = seq.n, wl.group, wl.cs, wl.l_obs, wl.chunk_budget
    scale = 1 / math.sqrt(128)
    qf, kf = f64(seq.q_obs), f64(seq.k)
    k = to_dev(seq.k)
    idx_g = ck.select_critical(to_dev(seq.q_obs), k, list(range(wl.hkv)), cs, b).cpu().numpy()
    idx_o = O.select_critical(qf, kf, range(wl.hkv), cs, b)
    kmin, kmax = ck.page_bounds(k, list(range(wl.hkv)), cs)
    q_st = synth.decode_queries(wl, 2)[0]
    pages_g = ck.retrieve_pages(to_dev(q_st), kmin, kmax, list(range(wl.hkv)), wl.hkv, (b * cs + l_obs) // cs)
    pages_g = pages_g.cpu().numpy()
    qd = f64(q_st)
    worst = 0.0
    for h in range(wl.hkv):
        rows_g = O.compact_rows(n, l_obs, cs, idx_g[h][idx_g[h] >= 0])
        rows_o = O.compact_rows(n, l_obs, cs, idx_o[h])
        mn, mx = O.page_bounds(kf[h], cs)
        p_o = O.argtopk_ascending(O.page_scores(qd[h * G:(h + 1) * G], mn, mx), (b * cs + l_obs) // cs)
        for g in range(h * G, (h + 1) * G):
            a = O.attention_recall(qd[g], kf[h], rows_g, scale) - O.attention_recall(qd[g], kf[h], rows_o, scale)
            c = O.attention_recall(qd[g], kf[h], O.chunk_rows(n, cs, pages_g[h]), scale) - \
                O.attention_recall(qd[g], kf[h], O.chunk_rows(n, cs, p_o), scale)
            worst = max(worst, abs(a), abs(c))
    say(f"largest recall difference GPU vs oracle choices: {worst:.2e}")
    assert worst < 1e-6
