"""Seeded random configurations through the C ABI against the oracle:
decode over random batches, group sizes, view lengths (including empty and
one-row views) and splits; selection over random context lengths, chunk
sizes and budgets; page retrieval with random tie groups.  Each case prints
its parameters before it runs."""
import math
import sys

import numpy as np
import pytest
import torch

import oracle as O
import paper_2608_30295_amd as ck
import synth
from gpu_util import DEV, assert_rows_close, check_topk, f64, to_dev

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _bf16(rng, shape, scale=1.0):
    return synth.f32_to_bf16_bits(scale * rng.standard_normal(shape, dtype=np.float32))


@pytest.mark.parametrize("seed", range(6))
def test_decode_random(seed):
    rng = np.random.default_rng(500 + seed)
    G = int(rng.choice([1, 2, 4, 8]))
    hkv = int(rng.integers(1, 5))
    B = int(rng.integers(1, 4))
    hq = G * hkv
    lens = [int(x) for x in rng.choice([0, 1, 7, 64, 65, 300, 2112, 5000, 20000], size=B * hkv)]
    split = int(rng.choice([0, 64, 192, 1024]))
    say(f"decode seed={seed} B={B} hkv={hkv} G={G} lens={lens} split={split}")
    views = [(_bf16(rng, (max(L, 1), 128)), _bf16(rng, (max(L, 1), 128))) for L in lens]
    kd = [(to_dev(k), to_dev(v)) for k, v in views]
    table = ck.kv_table([(k.data_ptr(), v.data_ptr()) for k, v in kd], DEV)
    plan = ck.decode_plan(np.array(lens, dtype=np.int64).reshape(B, hkv), hq, hkv, DEV, split_tokens=split)
    q = _bf16(rng, (B, hq, 128))
    out, lse = ck.decode_attn(plan, to_dev(q), table, torch.tensor(lens, dtype=torch.int64, device=DEV).view(B, hkv))
    torch.cuda.synchronize()
    out, lse = out.cpu().numpy(), lse.cpu().numpy()
    for b in range(B):
        for h in range(hkv):
            L = lens[b * hkv + h]
            for g in range(h * G, (h + 1) * G):
                if L == 0:
                    assert (out[b, g] == 0).all() and lse[b, g] == -np.inf
                    continue
                k, v = views[b * hkv + h]
                o_ref, l_ref, _ = O.attention_decode(f64(q)[b, g], f64(k)[:L], f64(v)[:L], 1 / math.sqrt(128))
                assert_rows_close(out[b, g][None], o_ref[None], "bf16", f"b={b} g={g} L={L}")
                assert abs(lse[b, g] - l_ref) <= 1e-4


@pytest.mark.parametrize("seed", range(4))
def test_select_random(seed):
    rng = np.random.default_rng(600 + seed)
    cs = int(rng.choice([4, 8, 12, 16, 24, 32]))   # 12 and 24 do not divide the 64-column tile
    l_obs = int(rng.choice([16, 32, 64]))
    n = int(rng.integers(l_obs + 1, 9000))
    hkv, G = 2, int(rng.choice([2, 4]))
    wl = synth.WORKLOADS["ctx32k_bf16"].scaled(n=n, hq=G * hkv, hkv=hkv, l_obs=l_obs, cs=cs)
    seq = synth.make_sequence(wl)
    n_chunks = -(-(n - l_obs) // cs)
    b = int(rng.integers(1, n_chunks + 3))
    heads = [int(h) for h in rng.permutation(hkv)[:int(rng.integers(1, hkv + 1))]]
    say(f"select seed={seed} n={n} cs={cs} l_obs={l_obs} G={G} b={b} chunks={n_chunks} heads={heads}")
    idx = ck.select_critical(to_dev(seq.q_obs), to_dev(seq.k), heads, cs, b).cpu().numpy()
    qf, kf = f64(seq.q_obs), f64(seq.k)
    for s, h in enumerate(heads):
        sc = O.chunk_scores(qf, kf, h, G, l_obs, cs, 1 / math.sqrt(128))
        check_topk(idx[s], sc, b)


@pytest.mark.parametrize("seed", range(4))
def test_retrieve_random_ties(seed):
    rng = np.random.default_rng(700 + seed)
    cs = int(rng.choice([4, 8, 16]))
    n_pat = int(rng.integers(1, 50))
    n_pages = int(rng.integers(1, 30000))
    n_keep = int(rng.integers(1, 2 * n_pages + 2))
    G = int(rng.choice([1, 2, 4, 8]))
    say(f"retrieve seed={seed} cs={cs} patterns={n_pat} pages={n_pages} keep={n_keep} G={G}")
    pat = _bf16(rng, (n_pat, cs, 128))
    kk = pat[rng.integers(0, n_pat, size=n_pages)].reshape(1, n_pages * cs, 128)
    q = _bf16(rng, (G, 128))
    kmin, kmax = ck.page_bounds(to_dev(kk), [0], cs)
    idx = ck.retrieve_pages(to_dev(q), kmin, kmax, [0], 1, n_keep).cpu().numpy()[0]
    mn, mx = O.page_bounds(f64(kk[0]), cs)
    sc = O.page_scores(f64(q), mn, mx)
    want = O.argtopk_ascending(sc, min(n_keep, n_pages)).tolist()
    want += [-1] * (n_keep - len(want))
    assert idx.tolist() == want
