"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times (default decode plan with one stream-K worker per resident
slot, default score geometry), on the outputs the oracle can compute one by
one: every CV score and chunk selection of sampled heads, bitwise compaction,
and decode outputs of sampled query heads.

Each sequence runs the whole prefill-side path on the GPU: CV score (Eq. 1-4),
Eq. 5 on the scores, selection (Algorithm 1) and compaction; decode then reads
compact views for the consistent heads and the original cache for the rest.
The decode oracle is given views built from the original K/V and the GPU's own
chunk indices, so a compaction error also shows up there."""
import math
import sys
import time

import numpy as np
import pytest
import torch

import oracle as O
import paper_2608_30295_amd as ck
import synth
from gpu_util import DEV, assert_rows_close, check_topk, f64, to_dev, to_host_storage

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

SCALE = 1.0 / math.sqrt(128)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


class Prefilled:
    """One sequence after the GPU's prefill-side path."""

    def __init__(self, wl, b=0):
        t0 = time.time()
        self.wl = wl
        self.seq = synth.make_sequence(wl, b)
        seq = self.seq
        say(f"  [{wl.name} b={b}] n={seq.n} generated in {time.time() - t0:.1f}s")
        self.k, self.v = to_dev(seq.k), to_dev(seq.v)
        cv = ck.score_heads(to_dev(seq.q_cv), self.k, q_pos0=seq.q_cv_pos0, l_init=wl.l_init,
                            l_rec=wl.l_rec, k_pct=wl.k_pct, alpha=wl.alpha)
        self.cv = cv.cpu().numpy().astype(np.float64)
        cons = ck.classify_heads(self.cv[None].astype(np.float32), wl.r)
        self.heads = [h for h in range(wl.hkv) if cons[h]]
        idx = ck.select_critical(to_dev(seq.q_obs), self.k, self.heads, wl.cs, wl.chunk_budget)
        self.lens = torch.full((wl.hkv,), seq.n, dtype=torch.int64, device=DEV)
        self.k_c, self.v_c = ck.compact_kv(self.k, self.v, self.heads, idx, wl.cs, wl.l_obs, self.lens)
        torch.cuda.synchronize()
        self.idx = idx.cpu().numpy()

    def view_pairs(self):
        pairs, maxlen = [], []
        for h in range(self.wl.hkv):
            if h in self.heads:
                s = self.heads.index(h)
                pairs.append((self.k_c[s].data_ptr(), self.v_c[s].data_ptr()))
                maxlen.append(self.k_c.shape[1])
            else:
                pairs.append((self.k[h].data_ptr(), self.v[h].data_ptr()))
                maxlen.append(self.seq.n)
        return pairs, maxlen

    def oracle_view(self, h):
        """(K, V) in fp64 of KV head h's decode view, from the original cache."""
        seq = self.seq
        if h in self.heads:
            sel = self.idx[self.heads.index(h)]
            rows = O.compact_rows(seq.n, self.wl.l_obs, self.wl.cs, sel[sel >= 0])
            return f64(seq.k[h][rows]), f64(seq.v[h][rows])
        return f64(seq.k[h]), f64(seq.v[h])


def check_selection(p: Prefilled, heads):
    qf = f64(p.seq.q_obs)
    G = p.wl.group
    for h in heads:
        t0 = time.time()
        # one head at a time: the oracle sees that head's group and keys only
        sc = O.chunk_scores(qf[h * G:(h + 1) * G], f64(p.seq.k[h:h + 1]), 0, G, p.wl.l_obs, p.wl.cs, SCALE)
        swaps = check_topk(p.idx[p.heads.index(h)], sc, p.wl.chunk_budget)
        say(f"  select head {h}: ok, {swaps} swaps inside the 1e-5 band ({time.time() - t0:.1f}s)")


def check_compaction(p: Prefilled):
    kc, vc = to_host_storage(p.k_c), to_host_storage(p.v_c)
    lens = p.lens.cpu().numpy()
    for s, h in enumerate(p.heads):
        sel = p.idx[s][p.idx[s] >= 0]
        rows = O.compact_rows(p.seq.n, p.wl.l_obs, p.wl.cs, sel)
        assert lens[h] == rows.size
        assert np.array_equal(kc[s][:rows.size], p.seq.k[h][rows])
        assert np.array_equal(vc[s][:rows.size], p.seq.v[h][rows])
    for h in range(p.wl.hkv):
        if h not in p.heads:
            assert lens[h] == p.seq.n


def decode_batch(prefilled, wl, step):
    pairs, maxlen, lens = [], [], []
    for p in prefilled:
        pr, ml = p.view_pairs()
        pairs += pr
        maxlen += ml
        lens.append(p.lens)
    table = ck.kv_table(pairs, DEV)
    plan = ck.decode_plan(np.array(maxlen, dtype=np.int64).reshape(len(prefilled), wl.hkv), wl.hq, wl.hkv, DEV)
    q_st = synth.decode_queries(wl, step)
    out, lse = ck.decode_attn(plan, to_dev(q_st), table, torch.stack(lens))
    torch.cuda.synchronize()
    return q_st, out.cpu().numpy(), lse.cpu().numpy(), plan


def check_decode(p: Prefilled, q_st_b, out_b, lse_b, qheads):
    G = p.wl.group
    qf = f64(q_st_b)
    for g in qheads:
        kh, vh = p.oracle_view(g // G)
        o_ref, l_ref, _ = O.attention_decode(qf[g], kh, vh, SCALE)
        assert_rows_close(out_b[g][None], o_ref[None], p.wl.dtype, f"q-head {g}")
        assert abs(float(lse_b[g]) - l_ref) < 1e-4, (g, lse_b[g], l_ref)


# ------------------------------------------------------------ 128K, batch 1

@pytest.fixture(scope="module")
def p128k():
    say("prefill ctx128k_bf16 at full size")
    return Prefilled(synth.WORKLOADS["ctx128k_bf16"])


def test_ctx128k_cv_and_classification(p128k):
    p, wl = p128k, p128k.wl
    t0 = time.time()
    ref = O.score_heads(f64(p.seq.q_cv), p.seq.q_cv_pos0, f64(p.seq.k), wl.l_init, wl.l_rec, wl.k_pct, wl.alpha)
    say(f"  cv gpu {np.round(p.cv, 5).tolist()}\n  cv ref {np.round(ref, 5).tolist()} ({time.time() - t0:.1f}s)")
    np.testing.assert_allclose(p.cv, ref, rtol=1e-4, atol=1e-6)
    assert O.static_head_types(ref[None], wl.r).nonzero()[0].tolist() == p.heads
    assert len(p.heads) == 5


def test_ctx128k_selection_and_compaction(p128k):
    check_selection(p128k, p128k.heads)
    check_compaction(p128k)


def test_ctx128k_decode_all_heads(p128k):
    wl = p128k.wl
    for step in (0, 1):
        q_st, out, lse, plan = decode_batch([p128k], wl, step)
        say(f"  decode step {step}: {plan.plan.n_workers} workers, {plan.plan.n_segments} segments")
        check_decode(p128k, q_st[0], out[0], lse[0], range(wl.hq))


# ------------------------------------------------------ 16 ragged sequences

@pytest.mark.timeout(600)
def test_batch16_ragged_decode():
    wl = synth.WORKLOADS["batch16_ragged_bf16"]
    say(f"prefill batch16_ragged_bf16: lengths {synth.sequence_lengths(wl)}")
    ps = [Prefilled(wl, b) for b in range(wl.batch)]
    q_st, out, lse, plan = decode_batch(ps, wl, 0)
    say(f"  decode: {plan.plan.n_workers} workers, {plan.plan.n_segments} segments, {plan.plan.n_multi} split views")
    for b, p in enumerate(ps):
        cons_g = p.heads[0] * wl.group + (b % wl.group)
        adap = [h for h in range(wl.hkv) if h not in p.heads]
        qheads = [cons_g] + ([adap[b % len(adap)] * wl.group + 1] if adap else [])
        check_decode(p, q_st[b], out[b], lse[b], qheads)
    # the selection of one sequence against the oracle
    check_selection(ps[3], ps[3].heads[:1])
    check_compaction(ps[3])


# ------------------------------------------------------------- 1M, batch 1

@pytest.mark.timeout(900)
def test_ctx1m_sampled():
    wl = synth.WORKLOADS["ctx1m_bf16"]
    say("prefill ctx1m_bf16 at full size")
    p = Prefilled(wl)
    assert len(p.heads) == 6
    # CV of two heads from the 32 calibration decode queries
    qcv = f64(p.seq.q_cv)
    for h in (p.heads[0], [x for x in range(wl.hkv) if x not in p.heads][0]):
        t0 = time.time()
        G = wl.group
        ref = O.score_heads(qcv[h * G:(h + 1) * G], p.seq.q_cv_pos0, f64(p.seq.k[h:h + 1]), wl.l_init,
                            wl.l_rec, wl.k_pct, wl.alpha)
        say(f"  cv head {h}: gpu {p.cv[h]:.6f} ref {ref[0]:.6f} ({time.time() - t0:.1f}s)")
        assert abs(p.cv[h] - ref[0]) <= 1e-4 * abs(ref[0]) + 1e-6
    check_selection(p, p.heads[:1])
    check_compaction(p)
    q_st, out, lse, plan = decode_batch([p], wl, 0)
    adap = [h for h in range(wl.hkv) if h not in p.heads][0]
    check_decode(p, q_st[0], out[0], lse[0], [p.heads[0] * wl.group, adap * wl.group + 2])


def test_cv_quantile_rank_beyond_two_to_the_31():
    """Eq. 2 over an observation matrix of more than 2^31 entries: the rank of
    the k-th percentile element, floor((N - 1) k), no longer fits 32 bits.
    Closed form: one query row pattern (q = e_0) against zero keys except m
    planted keys with one equal, larger score; every row puts the same mass
    on the planted columns, the quantile lands among those entries, so C is
    L_q on the m planted columns and 0 elsewhere and cv = sqrt((n'' - m) / m)."""
    lq, n, m = 64, 33_600_000, 16_800
    N = lq * n
    assert N > 2 ** 31
    k_pct = 0.9999                     # (N - 1) k lies among the lq * m planted entries
    assert (N - 1) * k_pct >= N - lq * m
    say(f"CV over {N} observation entries (rank {int((N - 1) * k_pct)})")
    k = torch.zeros((1, n, 128), dtype=torch.bfloat16, device=DEV)
    cols = torch.from_numpy(np.random.default_rng(5).choice(n, size=m, replace=False)).to(DEV)
    k[0, cols, 0] = 45.25              # exact in bf16: score 45.25 / sqrt(128) against q = e_0
    q = torch.zeros((1, lq, 128), dtype=torch.bfloat16, device=DEV)
    q[0, :, 0] = 1.0
    cv = ck.score_heads(q, k, q_pos0=n, l_init=0, l_rec=0, k_pct=k_pct, alpha=1.0, causal=False)
    torch.cuda.synchronize()
    want = math.sqrt((n - m) / m)
    got = float(cv.cpu()[0])
    del k
    torch.cuda.empty_cache()
    assert abs(got - want) <= 1e-4 * want, (got, want)
