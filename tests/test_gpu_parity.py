"""GPU parity: every C-ABI call against the CPU oracle on the same seeded
inputs (small and ragged sizes here; full sizes in test_gpu_fullsize.py)."""
import math
import sys

import numpy as np
import pytest
import torch

import oracle as O
import paper_2608_30295_amd as ck
import synth
from gpu_util import DEV, assert_rows_close, check_topk, f64, to_dev, to_host_storage

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _views(rng, lens, dtype, heavy=True):
    """Independent K/V buffers per view (storage arrays)."""
    out = []
    for L in lens:
        k = rng.standard_normal((max(L, 1), 128), dtype=np.float32)
        v = rng.standard_normal((max(L, 1), 128), dtype=np.float32)
        if heavy and L > 10:
            hot = rng.choice(L, size=max(1, L // 100), replace=False)
            k[hot] *= 3
        if dtype == "bf16":
            k, v = synth.f32_to_bf16_bits(k), synth.f32_to_bf16_bits(v)
        out.append((k, v))
    return out


def run_decode(views, B, hq, hkv, dtype, q_st, split=0, lens_dev=None, max_len=None):
    kd = [(to_dev(k), to_dev(v)) for k, v in views]
    table = ck.kv_table([(k.data_ptr(), v.data_ptr()) for k, v in kd], DEV)
    lens = np.array([0 if L is None else L for L in (max_len if max_len is not None else
                                                     [kv[0].shape[0] for kv in views])], dtype=np.int64)
    plan = ck.decode_plan(lens, hq, hkv, DEV, split_tokens=split)
    if lens_dev is None:
        lens_dev = torch.from_numpy(lens).to(DEV)
    q = to_dev(q_st)
    out, lse = ck.decode_attn(plan, q, table, lens_dev)
    torch.cuda.synchronize()
    return out.cpu().numpy(), lse.cpu().numpy(), kd, plan


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_decode_ragged_views(dtype):
    rng = np.random.default_rng(11)
    B, hq, hkv = 2, 8, 2
    lens = [37, 40000, 1, 2113]
    views = _views(rng, lens, dtype)
    q = rng.standard_normal((B, hq, 128), dtype=np.float32)
    q_st = synth.f32_to_bf16_bits(q) if dtype == "bf16" else q
    say(f"decode ragged {dtype} lens={lens}")
    out, lse, _, plan = run_decode(views, B, hq, hkv, dtype, q_st, split=256)
    assert plan.plan.n_multi > 0            # views merged from several partials
    qq = f64(q_st)
    for b in range(B):
        vv = [(f64(views[b * hkv + h][0])[:lens[b * hkv + h]], f64(views[b * hkv + h][1])[:lens[b * hkv + h]])
              for h in range(hkv)]
        o_ref, l_ref = O.decode_gqa(qq[b], vv)
        assert_rows_close(out[b], o_ref, dtype, f"b={b}")
        np.testing.assert_allclose(lse[b], l_ref, atol=1e-4, rtol=0)


def test_decode_more_views_than_preloaded():
    """320 views (40 sequences x 8 KV heads) on the one-workgroup-per-CU
    layout: beyond 256 views the stream kernel reads each segment's view
    pointers and length itself instead of from the table every workgroup
    preloads."""
    rng = np.random.default_rng(17)
    B, hq, hkv = 40, 16, 8
    lens = rng.integers(300, 700, size=B * hkv).tolist()
    views = _views(rng, lens, "bf16")
    q_st = synth.f32_to_bf16_bits(rng.standard_normal((B, hq, 128), dtype=np.float32))
    say(f"decode {B * hkv} views")
    out, lse, _, plan = run_decode(views, B, hq, hkv, "bf16", q_st)
    assert plan.plan.variant == 2 and plan.plan.n_multi > 0
    qq = f64(q_st)
    for b in range(B):
        vv = [(f64(views[b * hkv + h][0]), f64(views[b * hkv + h][1])) for h in range(hkv)]
        o_ref, l_ref = O.decode_gqa(qq[b], vv)
        assert_rows_close(out[b], o_ref, "bf16", f"b={b}")
        np.testing.assert_allclose(lse[b], l_ref, atol=1e-4, rtol=0)


def test_decode_empty_and_single_token_views():
    rng = np.random.default_rng(12)
    B, hq, hkv = 1, 4, 4
    lens = [0, 1, 2, 300]
    views = _views(rng, lens, "bf16")
    q_st = synth.f32_to_bf16_bits(rng.standard_normal((B, hq, 128), dtype=np.float32))
    say("decode empty/single views")
    out, lse, _, _ = run_decode(views, B, hq, hkv, "bf16", q_st, max_len=lens)
    assert (out[0, 0] == 0).all() and lse[0, 0] == -np.inf
    np.testing.assert_allclose(out[0, 1], f64(views[1][1])[0], atol=1e-6)
    for h in (2, 3):
        o_ref, l_ref, _ = O.attention_decode(f64(q_st)[0, h], f64(views[h][0])[:lens[h]], f64(views[h][1])[:lens[h]],
                                             1 / math.sqrt(128))
        assert_rows_close(out[0, h][None], o_ref[None], "bf16")


def test_decode_device_length_below_plan():
    # the plan holds upper bounds; the actual length is read on the device
    rng = np.random.default_rng(13)
    B, hq, hkv = 1, 8, 2
    cap = [3000, 1200]
    actual = [2111, 1200]
    views = _views(rng, cap, "bf16")
    q_st = synth.f32_to_bf16_bits(rng.standard_normal((B, hq, 128), dtype=np.float32))
    say("decode device lengths below plan")
    lens_dev = torch.tensor(actual, dtype=torch.int64, device=DEV)
    out, lse, _, _ = run_decode(views, B, hq, hkv, "bf16", q_st, split=512, lens_dev=lens_dev, max_len=cap)
    vv = [(f64(views[h][0])[:actual[h]], f64(views[h][1])[:actual[h]]) for h in range(hkv)]
    o_ref, l_ref = O.decode_gqa(f64(q_st)[0], vv)
    assert_rows_close(out[0], o_ref, "bf16")


def test_decode_device_length_above_plan_and_negative():
    # L = min(lens, planned max_len): a device length above the plan is
    # clamped to it, a negative one reads as an empty view
    rng = np.random.default_rng(16)
    B, hq, hkv = 1, 12, 3
    held = [5000, 700, 300]               # rows each view holds
    plan_len = [1000, 700, 300]
    actual = [5000, 650, -3]
    views = _views(rng, held, "bf16")
    q_st = synth.f32_to_bf16_bits(rng.standard_normal((B, hq, 128), dtype=np.float32))
    say("decode device lengths above the plan and negative")
    lens_dev = torch.tensor(actual, dtype=torch.int64, device=DEV)
    out, lse, _, _ = run_decode(views, B, hq, hkv, "bf16", q_st, split=256, lens_dev=lens_dev, max_len=plan_len)
    used = [1000, 650]
    vv = [(f64(views[h][0])[:used[h]], f64(views[h][1])[:used[h]]) for h in range(2)]
    o_ref, l_ref = O.decode_gqa(f64(q_st)[0][:8], vv)
    assert_rows_close(out[0][:8], o_ref, "bf16")
    np.testing.assert_allclose(lse[0][:8], l_ref, atol=1e-4, rtol=0)
    assert (out[0][8:] == 0).all() and (lse[0][8:] == -np.inf).all()


@pytest.mark.parametrize("G", [1, 2, 4, 8])
def test_decode_group_sizes(G):
    rng = np.random.default_rng(20 + G)
    hkv = 2
    hq = G * hkv
    lens = [777, 3001]
    views = _views(rng, lens, "bf16")
    q_st = synth.f32_to_bf16_bits(rng.standard_normal((1, hq, 128), dtype=np.float32))
    say(f"decode G={G}")
    out, lse, _, _ = run_decode(views, 1, hq, hkv, "bf16", q_st, split=256)
    vv = [(f64(k), f64(v)) for k, v in views]
    o_ref, l_ref = O.decode_gqa(f64(q_st)[0], vv)
    assert_rows_close(out[0], o_ref, "bf16")
    np.testing.assert_allclose(lse[0], l_ref, atol=1e-4, rtol=0)


def test_decode_repeated_steps_reuse_plan():
    # counters are reset by the kernel itself: several steps on one plan agree
    rng = np.random.default_rng(14)
    lens = [9000, 500]
    views = _views(rng, lens, "bf16")
    q_st = synth.f32_to_bf16_bits(rng.standard_normal((1, 8, 128), dtype=np.float32))
    say("decode repeated steps")
    kd = [(to_dev(k), to_dev(v)) for k, v in views]
    table = ck.kv_table([(k.data_ptr(), v.data_ptr()) for k, v in kd], DEV)
    plan = ck.decode_plan(np.array(lens), 8, 2, DEV, split_tokens=256)
    lens_dev = torch.tensor(lens, dtype=torch.int64, device=DEV)
    q = to_dev(q_st)
    outs = []
    for _ in range(4):
        o, _ = ck.decode_attn(plan, q, table, lens_dev)
        outs.append(o.clone())
    torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(o, outs[0])
    o_ref, _ = O.decode_gqa(f64(q_st)[0], [(f64(k), f64(v)) for k, v in views])
    assert_rows_close(outs[0].cpu().numpy()[0], o_ref, "bf16")


@pytest.mark.parametrize("G", [4, 8])
def test_decode_steps_alternating_inputs_and_graph_replays(G):
    # consecutive steps with other queries and caches on one plan and
    # workspace must each match the oracle (no partial of an earlier step
    # leaks into a later merge), and graph replays must reproduce the eager
    # steps bit for bit
    rng = np.random.default_rng(15 + G)
    B, hkv = 2, 2
    hq = G * hkv
    lens = [9000, 500, 30000, 64]
    sets = [_views(rng, lens, "bf16"), _views(rng, lens, "bf16")]
    qs = [synth.f32_to_bf16_bits(rng.standard_normal((B, hq, 128), dtype=np.float32)) for _ in range(3)]
    say(f"decode alternating steps G={G}")
    kds = [[(to_dev(k), to_dev(v)) for k, v in vs] for vs in sets]
    tables = [ck.kv_table([(k.data_ptr(), v.data_ptr()) for k, v in kd], DEV) for kd in kds]
    plan = ck.decode_plan(np.array(lens), hq, hkv, DEV, split_tokens=256)
    assert plan.plan.n_multi == 3
    lens_dev = torch.tensor(lens, dtype=torch.int64, device=DEV)
    qd = [to_dev(q) for q in qs]
    steps = [(0, 0), (1, 1), (2, 0), (0, 1), (1, 0)]
    outs = [torch.empty((B, hq, 128), dtype=torch.float32, device=DEV) for _ in steps]
    lses = [torch.empty((B, hq), dtype=torch.float32, device=DEV) for _ in steps]
    for i, (qi, si) in enumerate(steps):
        ck.decode_attn(plan, qd[qi], tables[si], lens_dev, out=outs[i], lse=lses[i])
    torch.cuda.synchronize()
    eager = [(o.clone(), l.clone()) for o, l in zip(outs, lses)]
    for i, (qi, si) in enumerate(steps):
        qq = f64(qs[qi])
        for b in range(B):
            vv = [(f64(sets[si][b * hkv + h][0]), f64(sets[si][b * hkv + h][1])) for h in range(hkv)]
            o_ref, l_ref = O.decode_gqa(qq[b], vv)
            assert_rows_close(eager[i][0].cpu().numpy()[b], o_ref, "bf16", f"step {i} b={b}")
            np.testing.assert_allclose(eager[i][1].cpu().numpy()[b], l_ref, atol=1e-4, rtol=0)
    s2 = torch.cuda.Stream(device=DEV)
    s2.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s2):
        g.capture_begin()
        for i, (qi, si) in enumerate(steps):
            ck.decode_attn(plan, qd[qi], tables[si], lens_dev, out=outs[i], lse=lses[i])
        g.capture_end()
    torch.cuda.current_stream().wait_stream(s2)
    for rep in range(3):
        for o in outs:
            o.fill_(7.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i in range(len(steps)):
            assert torch.equal(outs[i], eager[i][0]), f"replay {rep} step {i}"
            assert torch.equal(lses[i], eager[i][1]), f"replay {rep} step {i}"
        # eager work between replays on the same plan
        ck.decode_attn(plan, qd[2], tables[1], lens_dev)
        torch.cuda.synchronize()


# ---------------------------------------------------------------- selection

def _small(name, **kw):
    return synth.WORKLOADS[name].scaled(**kw)


SEL_CASES = [
    ("ctx4k_f32", dict()),                                    # the full 4K fp32 workload
    ("ctx32k_bf16", dict(n=5000 + 64 + 3)),                   # ragged last tile and chunk
    ("ctx32k_bf16", dict(n=64 + 40)),                         # shorter than one tile
    ("ctx128k_bf16", dict(n=9000, hq=16, hkv=2)),            # G = 8 rows of 512
    ("ctx32k_bf16", dict(n=64 + 8 * 17000 + 3, hq=8, hkv=2)), # over 16384 chunk scores per head
    ("ctx32k_bf16", dict(n=16 + 8 * 40000 + 5, hq=4, hkv=2, l_obs=16)),   # over 32768: slices, then candidates
    ("ctx32k_bf16", dict(n=64 + 8 * 4097, hq=8, hkv=2, budget=4096)),    # 4096-score slices, one-score last slice, k = 512
    ("ctx32k_bf16", dict(n=64 + 8 * 9000 + 5, hq=8, hkv=2, budget=8)),   # 4096-score slices, k = 1
    ("ctx32k_bf16", dict(n=6000 + 11, hq=4, hkv=4)),          # one query head per KV head (64 rows)
    ("ctx32k_bf16", dict(n=6000 + 29, hq=8, hkv=4, l_obs=32)), # G = 2 at 32 window rows (64 rows)
    ("ctx32k_bf16", dict(n=7000 + 3, l_obs=37)),              # 148 rows, padded to 256
]


@pytest.mark.parametrize("hq", [8, 16])
def test_select_score_spikes_move_the_row_maximum(hq):
    """Five keys along each group's mean query direction, scaled so that
    most rows score them 60-900 nats above the other keys, sit after the
    rows' first tiles.  The first spike's terms stay inside fp32's range
    against the offset the first tile fixed; the others overflow it and send
    their column blocks through the exact-maximum sweep.  Either way the
    selection matches the oracle's, for 256 rows (G = 4) and for 512 rows
    (G = 8, eight-wave workgroups)."""
    wl = _small("ctx32k_bf16", n=9000 + 37, hq=hq, hkv=2)
    seq = synth.make_sequence(wl)
    G, d = wl.group, 128
    k32 = synth.bf16_bits_to_f32(seq.k)
    q32 = synth.bf16_bits_to_f32(seq.q_obs)
    spikes = [2503, 6001, 6002, 7500, 8801]
    for h in range(wl.hkv):
        u = q32[h * G:(h + 1) * G].reshape(-1, d).astype(np.float64).mean(axis=0)
        u /= np.linalg.norm(u)
        for j, p in enumerate(spikes):
            k32[h, p] = (60.0 * (1 + j) * math.sqrt(d) * u).astype(np.float32)
    kb = synth.f32_to_bf16_bits(k32)
    heads = [1, 0]
    b = wl.chunk_budget
    say(f"select with score spikes n={seq.n} b={b} spikes={spikes}")
    idx = ck.select_critical(to_dev(seq.q_obs), to_dev(kb), heads, wl.cs, b).cpu().numpy()
    qf, kf = f64(seq.q_obs), f64(kb)
    for s_, h in enumerate(heads):
        sc = O.chunk_scores(qf, kf, h, G, wl.l_obs, wl.cs, 1 / math.sqrt(d))
        assert int(np.argmax(sc)) == spikes[-1] // wl.cs   # the largest spike's chunk leads
        check_topk(idx[s_], sc, b)


@pytest.mark.parametrize("name,kw", SEL_CASES)
def test_select_and_compact(name, kw):
    wl = _small(name, **kw)
    seq = synth.make_sequence(wl)
    heads = list(range(wl.hkv))[::-1][: max(1, wl.hkv // 2 + 1)]
    say(f"select {wl.name} n={seq.n} hq={wl.hq} hkv={wl.hkv} heads={heads} b={wl.chunk_budget}")
    q_obs, k, v = to_dev(seq.q_obs), to_dev(seq.k), to_dev(seq.v)
    idx = ck.select_critical(q_obs, k, heads, wl.cs, wl.chunk_budget)
    torch.cuda.synchronize()
    idx = idx.cpu().numpy()
    qf, kf = f64(seq.q_obs), f64(seq.k)
    scale = 1 / math.sqrt(128)
    for s, h in enumerate(heads):
        sc = O.chunk_scores(qf, kf, h, wl.group, wl.l_obs, wl.cs, scale)
        swaps = check_topk(idx[s], sc, wl.chunk_budget)
        say(f"  head {h}: swaps inside the 1e-5 band: {swaps}")
    # compaction, staged on the GPU's own indices: bitwise
    lens = torch.full((wl.hkv,), -7, dtype=torch.int64, device=DEV)
    idx_d = torch.from_numpy(idx).to(DEV)
    k_c, v_c = ck.compact_kv(k, v, heads, idx_d, wl.cs, wl.l_obs, lens)
    torch.cuda.synchronize()
    lens = lens.cpu().numpy()
    kc_h, vc_h = to_host_storage(k_c), to_host_storage(v_c)
    for s, h in enumerate(heads):
        sel = idx[s][idx[s] >= 0]
        rows = O.compact_rows(seq.n, wl.l_obs, wl.cs, sel)
        assert lens[h] == rows.size
        assert np.array_equal(kc_h[s][:rows.size], seq.k[h][rows])
        assert np.array_equal(vc_h[s][:rows.size], seq.v[h][rows])
    for h in range(wl.hkv):
        if h not in heads:
            assert lens[h] == -7


def test_select_budget_above_chunk_count_and_zero_keys():
    wl = _small("ctx32k_bf16", n=64 + 8 * 20 + 5, hq=8, hkv=2)
    seq = synth.make_sequence(wl)
    k0 = np.zeros_like(seq.k)
    say("select with zero keys and a budget above the chunk count")
    idx = ck.select_critical(to_dev(seq.q_obs), to_dev(k0), [0, 1], wl.cs, 40).cpu().numpy()
    nc = -(-(seq.n - 64) // 8)
    for s in range(2):
        assert idx[s][:nc].tolist() == list(range(nc))
        assert (idx[s][nc:] == -1).all()
    idx = ck.select_critical(to_dev(seq.q_obs), to_dev(k0), [1], wl.cs, 5).cpu().numpy()
    assert idx[0].tolist() == [0, 1, 2, 3, 4]


def test_full_budget_pipeline_equals_full_attention():
    # budget >= chunk count: the compact cache is the full cache, and decoding
    # over it reproduces full attention
    wl = _small("ctx32k_bf16", n=2048 + 64 + 5, hq=8, hkv=2)
    seq = synth.make_sequence(wl)
    say("full-budget pipeline")
    k, v = to_dev(seq.k), to_dev(seq.v)
    nc = -(-(seq.n - 64) // 8)
    idx = ck.select_critical(to_dev(seq.q_obs), k, [0, 1], 8, nc + 3)
    lens = torch.zeros(2, dtype=torch.int64, device=DEV)
    k_c, v_c = ck.compact_kv(k, v, [0, 1], idx, 8, 64, lens)
    torch.cuda.synchronize()
    assert lens.cpu().tolist() == [seq.n, seq.n]
    assert torch.equal(k_c[:, :seq.n].view(torch.int16), k.view(torch.int16))
    q_st = synth.decode_queries(wl, 0)
    table = ck.kv_table([(k_c[h].data_ptr(), v_c[h].data_ptr()) for h in range(2)], DEV)
    plan = ck.decode_plan(np.array([k_c.shape[1]] * 2), 8, 2, DEV)
    out, _ = ck.decode_attn(plan, to_dev(q_st), table, lens)
    o_ref, _ = O.decode_gqa(f64(q_st)[0], [(f64(seq.k[h]), f64(seq.v[h])) for h in range(2)])
    assert_rows_close(out.cpu().numpy()[0], o_ref, "bf16")


# ---------------------------------------------------------------- CV score

CV_CASES = [
    ("ctx4k_f32", dict(), True),
    ("ctx32k_bf16", dict(n=6000), True),
    ("ctx1m_bf16", dict(n=7000), True),          # decode-time calibration rows (mask is a no-op)
    ("ctx32k_bf16", dict(n=3000, hq=16, hkv=2), False),
    ("ctx32k_bf16", dict(n=5000, hq=4, hkv=4), True),      # one query head per KV head
    ("ctx32k_bf16", dict(n=4000, hq=8, hkv=4), False),     # two
    ("ctx32k_bf16", dict(n=4500, l_obs=37), True),         # 148 rows: padding rows in every pass
]


@pytest.mark.parametrize("name,kw,causal", CV_CASES)
def test_score_heads(name, kw, causal):
    wl = _small(name, **kw)
    seq = synth.make_sequence(wl)
    say(f"score_heads {wl.name} n={seq.n} rows={seq.q_cv.shape[1]} causal={causal}")
    cv = ck.score_heads(to_dev(seq.q_cv), to_dev(seq.k), q_pos0=seq.q_cv_pos0, l_init=wl.l_init,
                        l_rec=wl.l_rec, k_pct=wl.k_pct, alpha=wl.alpha, causal=causal)
    torch.cuda.synchronize()
    cv = cv.cpu().numpy().astype(np.float64)
    ref = O.score_heads(f64(seq.q_cv), seq.q_cv_pos0, f64(seq.k), wl.l_init, wl.l_rec, wl.k_pct, wl.alpha,
                        causal=causal)
    say("  gpu", np.round(cv, 6), "\n  ref", np.round(ref, 6))
    np.testing.assert_allclose(cv, ref, rtol=1e-4, atol=1e-6)


def test_score_heads_rows_mid_sequence_causal():
    """Observation rows in the middle of the sequence: under the causal mask
    each row sees a prefix of the keys, whole column blocks past the rows are
    invisible to all of them, and the blocks across the diagonal are partly
    visible."""
    wl = _small("ctx32k_bf16", n=6000)
    seq = synth.make_sequence(wl)
    q_pos0 = 2500
    say(f"score_heads rows at {q_pos0}.. of n={seq.n}, causal")
    cv = ck.score_heads(to_dev(seq.q_cv), to_dev(seq.k), q_pos0=q_pos0, l_init=wl.l_init,
                        l_rec=wl.l_rec, k_pct=wl.k_pct, alpha=wl.alpha, causal=True)
    torch.cuda.synchronize()
    cv = cv.cpu().numpy().astype(np.float64)
    ref = O.score_heads(f64(seq.q_cv), q_pos0, f64(seq.k), wl.l_init, wl.l_rec, wl.k_pct, wl.alpha,
                        causal=True)
    say("  gpu", np.round(cv, 6), "\n  ref", np.round(ref, 6))
    np.testing.assert_allclose(cv, ref, rtol=1e-4, atol=1e-6)


def test_score_heads_crowded_and_spread_quantile_bins():
    # head 0 has zero keys: every entry of its observation matrix is equal, so
    # the quantile's top-digit bin holds all of them (more than the candidate
    # buffer: the passes run over A); head 1 is spread (candidates gathered)
    wl = _small("ctx32k_bf16", n=3000, hq=8, hkv=2)
    seq = synth.make_sequence(wl)
    k = seq.k.copy()
    k[0] = 0
    say("score_heads with a crowded and a spread head")
    cv = ck.score_heads(to_dev(seq.q_cv), to_dev(k), q_pos0=seq.q_cv_pos0, l_init=wl.l_init,
                        l_rec=wl.l_rec, k_pct=wl.k_pct, alpha=wl.alpha, causal=False)
    torch.cuda.synchronize()
    cv = cv.cpu().numpy().astype(np.float64)
    ref = O.score_heads(f64(seq.q_cv), seq.q_cv_pos0, f64(k), wl.l_init, wl.l_rec, wl.k_pct, wl.alpha,
                        causal=False)
    say("  gpu", np.round(cv, 6), "\n  ref", np.round(ref, 6))
    assert ref[0] == 0.0
    np.testing.assert_allclose(cv, ref, rtol=1e-4, atol=1e-6)


@pytest.mark.parametrize("k_pct,alpha", [(0.984, 0.8), (0.99, 1.0), (0.996, 0.8)])
def test_score_heads_paper_percentiles(k_pct, alpha):
    """The percentile thresholds and scaling factors of the paper's settings
    (Section 5): Phi = alpha * Quantile_k below the quantile itself when
    alpha < 1, so Phi's range and the bracket are apart."""
    wl = _small("ctx32k_bf16", n=6000)
    seq = synth.make_sequence(wl)
    say(f"score_heads k={k_pct} alpha={alpha}")
    cv = ck.score_heads(to_dev(seq.q_cv), to_dev(seq.k), q_pos0=seq.q_cv_pos0, l_init=wl.l_init,
                        l_rec=wl.l_rec, k_pct=k_pct, alpha=alpha)
    torch.cuda.synchronize()
    cv = cv.cpu().numpy().astype(np.float64)
    ref = O.score_heads(f64(seq.q_cv), seq.q_cv_pos0, f64(seq.k), wl.l_init, wl.l_rec, k_pct, alpha)
    say("  gpu", np.round(cv, 6), "\n  ref", np.round(ref, 6))
    np.testing.assert_allclose(cv, ref, rtol=1e-4, atol=1e-6)


@pytest.mark.parametrize("n,m,k_pct", [(20000, 40, 0.999), (60000, 1040, 0.99)])
def test_score_heads_tied_top_columns(n, m, k_pct):
    """Closed form with a tie at the quantile: identical query rows, m key
    columns (spread evenly) with one equal, larger score and the others
    small and spread out.  Rank lo lands among the lq * m tied entries, so Phi is their
    value, C is lq on the m columns and 0 elsewhere, cv = sqrt((n - m) / m).
    The tied bin holds 2560 entries (a list resolved digit by digit) or
    66560 (more than the list takes: resolved over every gathered entry)."""
    lq, G = 64, 4
    rng = np.random.default_rng(7)
    k = np.zeros((1, n, 128), dtype=np.float32)
    k[0, :, 1:] = 0.1 * rng.standard_normal((n, 127), dtype=np.float32)
    cols = np.linspace(0, n - 1, m).astype(np.int64)
    k[0, cols, :] = 0.0
    k[0, cols, 0] = 8.0                      # exact in bf16: score 8 / sqrt(128) against q = e_0
    q = np.zeros((G, lq, 128), dtype=np.float32)
    q[:, :, 0] = 1.0
    q[:, :, 1:] = 0.5 * rng.standard_normal(127, dtype=np.float32)   # the other columns' scores spread out
    kb, qb = synth.f32_to_bf16_bits(k), synth.f32_to_bf16_bits(q)
    say(f"tied top columns n={n} m={m} k={k_pct} (tie of {lq * m} entries)")
    cv = ck.score_heads(to_dev(qb), to_dev(kb), q_pos0=n, l_init=0, l_rec=0, k_pct=k_pct, alpha=1.0, causal=False)
    torch.cuda.synchronize()
    want = math.sqrt((n - m) / m)
    got = float(cv.cpu()[0])
    say(f"  gpu {got:.6f} closed form {want:.6f}")
    assert abs(got - want) <= 1e-5 * want


def test_score_heads_toy_through_abi():
    # the hand-worked 2 x 4 toy (cv = sqrt(3)) driven through the GPU path
    A = np.array([[0.7, 0.1, 0.1, 0.1], [0.6, 0.2, 0.1, 0.1]])
    q = np.zeros((1, 2, 128), dtype=np.float32)
    q[0, 0, 0] = q[0, 1, 1] = 1.0
    k = np.zeros((1, 4, 128), dtype=np.float32)
    k[0, :, 0] = np.log(A[0]) * math.sqrt(128)
    k[0, :, 1] = np.log(A[1]) * math.sqrt(128)
    say("score_heads toy")
    cv = ck.score_heads(to_dev(q), to_dev(k), q_pos0=10, l_init=0, l_rec=0, k_pct=0.75, alpha=1.0)
    assert abs(float(cv.cpu()[0]) - math.sqrt(3)) < 1e-5


# ----------------------------------------------------- whole pipeline (4K)

def test_pipeline_ctx4k_f32():
    """CV score -> Eq. 5 -> select -> compact -> one decode step on the 4K fp32
    workload, against the oracle running the same steps."""
    wl = synth.WORKLOADS["ctx4k_f32"]
    seq = synth.make_sequence(wl)
    say("pipeline ctx4k_f32")
    k, v = to_dev(seq.k), to_dev(seq.v)
    cv = ck.score_heads(to_dev(seq.q_cv), k, q_pos0=seq.q_cv_pos0, l_init=wl.l_init, l_rec=wl.l_rec,
                        k_pct=wl.k_pct, alpha=wl.alpha).cpu().numpy()
    cv_ref = O.score_heads(f64(seq.q_cv), seq.q_cv_pos0, f64(seq.k), wl.l_init, wl.l_rec, wl.k_pct, wl.alpha)
    np.testing.assert_allclose(cv, cv_ref, rtol=1e-4)
    cons = ck.classify_heads(cv[None], wl.r)
    cons_ref = O.static_head_types(cv_ref[None], wl.r)
    assert cons.tolist() == cons_ref.tolist()
    heads = [h for h in range(wl.hkv) if cons[h]]
    assert len(heads) == 4
    idx = ck.select_critical(to_dev(seq.q_obs), k, heads, wl.cs, wl.chunk_budget)
    idx_h = idx.cpu().numpy()
    for s, h in enumerate(heads):
        sc = O.chunk_scores(f64(seq.q_obs), f64(seq.k), h, wl.group, wl.l_obs, wl.cs, 1 / math.sqrt(128))
        check_topk(idx_h[s], sc, wl.chunk_budget)
    # downstream stages are compared on the GPU's own selection
    idx_ref = [row[row >= 0] for row in idx_h]
    lens = torch.tensor([seq.n] * wl.hkv, dtype=torch.int64, device=DEV)
    k_c, v_c = ck.compact_kv(k, v, heads, idx, wl.cs, wl.l_obs, lens)
    pairs, maxlen = [], []
    for h in range(wl.hkv):
        if h in heads:
            s = heads.index(h)
            pairs.append((k_c[s].data_ptr(), v_c[s].data_ptr()))
            maxlen.append(k_c.shape[1])
        else:
            pairs.append((k[h].data_ptr(), v[h].data_ptr()))
            maxlen.append(seq.n)
    plan = ck.decode_plan(np.array(maxlen), wl.hq, wl.hkv, DEV)
    q_st = synth.decode_queries(wl, 0)
    out, lse = ck.decode_attn(plan, to_dev(q_st), ck.kv_table(pairs, DEV), lens)
    kc_ref, vc_ref = O.compact_kv(f64(seq.k), f64(seq.v), heads, idx_ref, wl.cs, wl.l_obs)
    views = [(kc_ref[heads.index(h)], vc_ref[heads.index(h)]) if h in heads else (f64(seq.k[h]), f64(seq.v[h]))
             for h in range(wl.hkv)]
    o_ref, l_ref = O.decode_gqa(f64(q_st)[0], views)
    assert_rows_close(out.cpu().numpy()[0], o_ref, "f32")
    np.testing.assert_allclose(lse.cpu().numpy()[0], l_ref, atol=1e-5)
