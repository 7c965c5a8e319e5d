"""Attention-recall diagnostic (Figure 4 and its discussion): per query head,
the share of the full attention mass of decode queries that each pattern
keeps under one sparse budget -- consistent (Algorithm 1's prefill selection
plus the window), streaming (initial plus most recent rows), query-aware
pages (Quest bound, pages of cs rows) and the per-query top-k upper bound.

Inputs are synthetic: the 4K fp32 workload, whose keys carry planted
directions along each group's mean window query; decode queries are window
queries of the same head plus Gaussian noise (decode queries that resemble
the observation window, the situation the consistent pattern relies on).
The recall values describe these inputs only, not the paper's models.

Checks that hold for any inputs: recall lies in [0, 1] and the top-k pattern
is an upper bound of every pattern with the same number of rows.  Checks of
this recipe: the consistent pattern recalls more than the streaming pattern
on average."""
import math

import numpy as np

import oracle as O
import synth


def recall_table(n_queries=8, noise=0.5, seed=7):
    wl = synth.WORKLOADS["ctx4k_f32"]
    seq = synth.make_sequence(wl)
    n, G, cs, l_obs = seq.n, wl.group, wl.cs, wl.l_obs
    scale = 1 / math.sqrt(wl.d)
    qf, kf = synth.storage_to_f64(seq.q_obs), synth.storage_to_f64(seq.k)
    b = wl.chunk_budget
    budget_rows = b * cs + l_obs                       # the consistent heads' compact length
    idx = O.select_critical(qf, kf, range(wl.hkv), cs, b)
    r = np.random.default_rng(seed)
    table = {p: np.zeros(wl.hq) for p in ("consistent", "streaming", "quest", "topk")}
    for h in range(wl.hkv):
        keep_c = O.compact_rows(n, l_obs, cs, idx[h])
        keep_s = O.streaming_keep(n, budget_rows, 4)
        kmin, kmax = O.page_bounds(kf[h], cs)
        for g in range(h * G, (h + 1) * G):
            rows = r.integers(0, l_obs, size=n_queries)
            qs = qf[g, rows] + noise * r.standard_normal((n_queries, wl.d))
            for q in qs:
                pages = O.argtopk_ascending(O.page_scores(q[None], kmin, kmax), budget_rows // cs)
                keep_q = O.chunk_rows(n, cs, pages)
                keep_t = O.topk_keep(q, kf[h], budget_rows, scale)
                rec = {"consistent": O.attention_recall(q, kf[h], keep_c, scale),
                       "streaming": O.attention_recall(q, kf[h], keep_s, scale),
                       "quest": O.attention_recall(q, kf[h], keep_q, scale),
                       "topk": O.attention_recall(q, kf[h], keep_t, scale)}
                for p, v in rec.items():
                    assert -1e-12 <= v <= 1 + 1e-12
                sizes = {"consistent": keep_c.size, "streaming": keep_s.size, "quest": keep_q.size}
                for p, sz in sizes.items():
                    # the top-k pattern with as many rows is an upper bound
                    ub = O.attention_recall(q, kf[h], O.topk_keep(q, kf[h], sz, scale), scale)
                    assert rec[p] <= ub + 1e-12
                for p, v in rec.items():
                    table[p][g] += v / n_queries
    return table


def test_attention_recall_patterns():
    t = recall_table()
    print("\nmean attention recall per query head (budget 288 rows of 4096):")
    for p, v in t.items():
        print(f"  {p:10s} mean {v.mean():.3f}  min {v.min():.3f}  max {v.max():.3f}")
    assert (t["topk"] >= t["consistent"] - 1e-12).all()
    assert t["consistent"].mean() > t["streaming"].mean()
