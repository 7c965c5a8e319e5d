"""Pins for the CPU oracle: facts fixed by the paper's definitions and by
mathematics, checked without re-typing the oracle's formulas.

Each group names the passage it pins (CateKV: Algorithm 1, Section 3.2
Eq. 1-5).  A plausible slip in the oracle -- a dropped 1/sqrt(d), a softmax
over the wrong axis, a transposed operand, a wrong tie rule, an off-by-one in
the chunking or the quantile -- fails at least one of them.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rng(seed):
    return np.random.default_rng(seed)


# --------------------------------------------------------------------------
# decoding-stage Attention(q, k, v) (Algorithm 1)
# --------------------------------------------------------------------------

class TestDecodeAttention:
    def test_weights_sum_to_one(self):
        r = rng(1)
        q, k, v = r.normal(size=128), r.normal(size=(300, 128)), r.normal(size=(300, 128))
        _, _, w = O.attention_decode(q, k, v, 1 / math.sqrt(128))
        assert abs(w.sum() - 1) < 1e-12 and (w > 0).all()

    def test_single_token_returns_its_value(self):
        r = rng(2)
        q, k, v = r.normal(size=128), r.normal(size=(1, 128)), r.normal(size=(1, 128))
        o, lse, _ = O.attention_decode(q, k, v, 0.1)
        np.testing.assert_array_equal(o, v[0])
        assert abs(lse - 0.1 * float(q @ k[0])) < 1e-12

    def test_equal_keys_average_values(self):
        r = rng(3)
        q, v = r.normal(size=128), r.normal(size=(37, 128))
        k = np.tile(r.normal(size=128), (37, 1))
        o, lse, _ = O.attention_decode(q, k, v, 0.3)
        np.testing.assert_allclose(o, v.mean(axis=0), rtol=0, atol=1e-13)
        assert abs(lse - (0.3 * float(q @ k[0]) + math.log(37))) < 1e-12

    def test_permutation_invariance(self):
        r = rng(4)
        q, k, v = r.normal(size=128), r.normal(size=(200, 128)), r.normal(size=(200, 128))
        p = r.permutation(200)
        o1, l1, _ = O.attention_decode(q, k, v, 0.09)
        o2, l2, _ = O.attention_decode(q, k[p], v[p], 0.09)
        np.testing.assert_allclose(o1, o2, atol=1e-13)
        assert abs(l1 - l2) < 1e-12

    def test_matches_library_sdpa_fp64(self):
        r = rng(5)
        Hq, Hkv, d, L = 8, 2, 128, 500
        q = r.normal(size=(Hq, d))
        k = r.normal(size=(Hkv, L, d)) * 1.5
        v = r.normal(size=(Hkv, L, d))
        out, _ = O.decode_gqa(q, [(k[h], v[h]) for h in range(Hkv)])
        G = Hq // Hkv
        kt = torch.from_numpy(np.repeat(k, G, axis=0))[None]
        vt = torch.from_numpy(np.repeat(v, G, axis=0))[None]
        qt = torch.from_numpy(q)[None, :, None, :]
        ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt)[0, :, 0].numpy()
        np.testing.assert_allclose(out, ref, atol=1e-12, rtol=0)

    def test_split_and_logsumexp_merge(self):
        # attention over a union of two key sets equals the lse-weighted merge
        r = rng(6)
        q, k, v = r.normal(size=128), r.normal(size=(301, 128)), r.normal(size=(301, 128))
        o, lse, _ = O.attention_decode(q, k, v, 0.088)
        oa, la, _ = O.attention_decode(q, k[:120], v[:120], 0.088)
        ob, lb, _ = O.attention_decode(q, k[120:], v[120:], 0.088)
        M = max(la, lb)
        wa, wb = math.exp(la - M), math.exp(lb - M)
        np.testing.assert_allclose((wa * oa + wb * ob) / (wa + wb), o, atol=1e-13)
        assert abs(M + math.log(wa + wb) - lse) < 1e-12

    def test_empty_view(self):
        o, lse, _ = O.attention_decode(np.ones(4), np.zeros((0, 4)), np.zeros((0, 4)), 1.0)
        assert (o == 0).all() and lse == -math.inf

    def test_gqa_head_mapping_is_contiguous(self):
        # query head g reads KV head g // G: give each KV head a constant value row
        r = rng(7)
        Hq, Hkv, d = 8, 4, 16
        views = [(r.normal(size=(5, d)), np.full((5, d), float(h))) for h in range(Hkv)]
        out, _ = O.decode_gqa(r.normal(size=(Hq, d)), views)
        np.testing.assert_allclose(out[:, 0], [0, 0, 1, 1, 2, 2, 3, 3], atol=1e-14)


# --------------------------------------------------------------------------
# pre-filling stage: window scores, BlockMax, argtopk, Cache (Algorithm 1)
# --------------------------------------------------------------------------

class TestSelection:
    def test_two_key_worked_example(self):
        # s1 - s2 = ln 3 after the 1/sqrt(d) scale => softmax = (3/4, 1/4)
        d = 16
        q = np.zeros((1, 1, d)); q[0, 0, 0] = 1.0
        k = np.zeros((2, d)); k[0, 0] = math.log(3.0) * math.sqrt(d)
        A = O.selection_observation_matrix(q, k, 1 / math.sqrt(d))
        np.testing.assert_allclose(A, [[0.75, 0.25]], atol=1e-15)

    def test_column_mass_sums_to_window_length(self):
        r = rng(10)
        G, L, n, d = 4, 16, 333, 32
        A = O.selection_observation_matrix(r.normal(size=(G, L, d)), r.normal(size=(n, d)), 0.2)
        assert A.shape == (L, n)
        np.testing.assert_allclose(A.sum(axis=1), np.ones(L), atol=1e-13)
        assert abs(A.sum(axis=0).sum() - L) < 1e-11

    def test_key_shift_invariance(self):
        # adding one vector to every key shifts each row's scores by a constant
        r = rng(11)
        q, k = r.normal(size=(2, 8, 32)), r.normal(size=(100, 32))
        c = r.normal(size=32) * 3
        A1 = O.selection_observation_matrix(q, k, 0.17)
        A2 = O.selection_observation_matrix(q, k + c, 0.17)
        np.testing.assert_allclose(A1, A2, atol=1e-13)

    def test_group_mean_of_identical_heads(self):
        r = rng(12)
        q1, k = r.normal(size=(1, 8, 32)), r.normal(size=(90, 32))
        A1 = O.selection_observation_matrix(q1, k, 0.2)
        A4 = O.selection_observation_matrix(np.repeat(q1, 4, axis=0), k, 0.2)
        np.testing.assert_allclose(A1, A4, atol=1e-15)

    def test_group_mean_is_mean_of_head_matrices(self):
        r = rng(13)
        q, k = r.normal(size=(2, 4, 16)), r.normal(size=(40, 16))
        A = O.selection_observation_matrix(q, k, 0.25)
        Aa = O.selection_observation_matrix(q[:1], k, 0.25)
        Ab = O.selection_observation_matrix(q[1:], k, 0.25)
        np.testing.assert_allclose(A, (Aa + Ab) / 2, atol=1e-15)

    def test_chunk_scores_with_unit_chunks_sum_to_window_length(self):
        # Algorithm 1 normalises each window row over exactly K[:-L_obs]: with
        # cs = 1, BlockMax is the identity and the column masses of the L_obs
        # row-stochastic rows add up to L_obs.  A softmax over any wider key
        # range (the whole row, or one window key more) leaves less.
        r = rng(19)
        Hq, Hkv, L, n, d = 8, 2, 12, 150, 32
        q, k = r.normal(size=(Hq, L, d)), r.normal(size=(Hkv, n, d))
        for h in range(Hkv):
            C = O.chunk_scores(q, k, h, Hq // Hkv, L, 1, 1 / math.sqrt(d))
            assert C.shape == (n - L,)
            assert abs(C.sum() - L) < 1e-11

    @pytest.mark.parametrize("L", [1, 3])
    def test_chunk_scores_exclude_the_window_keys(self, L):
        # Two prefix keys whose scores differ by ln 3 and L window keys with a
        # far larger score.  Restricted to K[:-L_obs], every window row puts
        # 3/4 and 1/4 on the two prefix keys, so C = (3/4 L, 1/4 L); were the
        # window keys inside the softmax they would take almost all the mass.
        d = 16
        q = np.zeros((1, L, d)); q[0, :, 0] = 1.0
        k = np.zeros((1, 2 + L, d))
        k[0, 0, 0] = math.log(3.0) * math.sqrt(d)
        k[0, 2:, 0] = 40.0 * math.sqrt(d)
        C = O.chunk_scores(q, k, 0, 1, L, 1, 1 / math.sqrt(d))
        np.testing.assert_allclose(C, [0.75 * L, 0.25 * L], rtol=0, atol=1e-14)
        # one chunk over both keys: BlockMax keeps the larger mass
        C2 = O.chunk_scores(q, k, 0, 1, L, 2, 1 / math.sqrt(d))
        np.testing.assert_allclose(C2, [0.75 * L], rtol=0, atol=1e-14)

    def test_block_max_worked_example(self):
        np.testing.assert_array_equal(O.block_max(np.array([1., 5., 2., 3., 4.]), 2), [5, 3, 4])
        np.testing.assert_array_equal(O.block_max(np.array([1., 5., 2.]), 8), [5])

    @pytest.mark.parametrize("seed", range(20))
    def test_topk_brute_force(self, seed):
        r = rng(100 + seed)
        nc = int(r.integers(1, 9))
        sc = r.integers(0, 4, size=nc).astype(np.float64)   # many ties
        b = int(r.integers(1, nc + 2))
        got = O.argtopk_ascending(sc, b)
        # exhaustive: the unique b-subset in which every kept chunk beats every
        # dropped one under (score desc, index asc)
        want = None
        for S in itertools.combinations(range(nc), min(b, nc)):
            rest = [j for j in range(nc) if j not in S]
            if all(sc[i] > sc[j] or (sc[i] == sc[j] and i < j) for i in S for j in rest):
                assert want is None
                want = list(S)
        assert list(got) == want

    def test_zero_keys_select_first_chunks(self):
        r = rng(14)
        Hq, Hkv, L, n, d = 8, 2, 8, 8 * 10 + 8 + 5, 16
        k = np.zeros((Hkv, n, d))
        idx = O.select_critical(r.normal(size=(Hq, L, d)), k, [0, 1], cs=8, b=4)
        for ih in idx:
            np.testing.assert_array_equal(ih, [0, 1, 2, 3])

    def test_planted_keys_are_recalled(self):
        r = rng(15)
        Hq, Hkv, L, n, d, cs = 8, 2, 8, 1024, 64, 8
        q = r.normal(size=(Hq, L, d))
        k = r.normal(size=(Hkv, n, d))
        planted = {}
        for h in range(Hkv):
            u = q[h * 4:(h + 1) * 4].reshape(-1, d).mean(axis=0)
            u /= np.linalg.norm(u)
            pos = np.sort(r.choice(n - L, size=6, replace=False))
            k[h, pos] = 12 * math.sqrt(d) * u
            planted[h] = set(pos // cs)
        idx = O.select_critical(q, k, [0, 1], cs=cs, b=len(planted[0]) + 2)
        for h, ih in enumerate(idx):
            assert planted[h] <= set(ih.tolist())

    def test_partial_last_chunk_and_clamped_budget(self):
        # n' = 21 tokens, cs = 8: chunks [0,8), [8,16), [16,21)
        rows = O.compact_rows(n=21 + 3, l_obs=3, cs=8, idx=np.array([0, 2]))
        np.testing.assert_array_equal(rows, list(range(0, 8)) + list(range(16, 21)) + [21, 22, 23])
        r = rng(16)
        idx = O.select_critical(r.normal(size=(4, 3, 16)), r.normal(size=(1, 24, 16)), [0], 8, 99)
        np.testing.assert_array_equal(idx[0], [0, 1, 2])

    def test_full_budget_reproduces_full_attention_exactly(self):
        r = rng(17)
        Hq, Hkv, L, n, d, cs = 8, 2, 16, 8 * 37 + 16 + 3, 32, 8
        q_obs, k, v = r.normal(size=(Hq, L, d)), r.normal(size=(Hkv, n, d)), r.normal(size=(Hkv, n, d))
        nch = -(-(n - L) // cs)
        idx = O.select_critical(q_obs, k, [0, 1], cs, nch + 5)
        kc, vc = O.compact_kv(k, v, [0, 1], idx, cs, L)
        for h in range(Hkv):
            np.testing.assert_array_equal(kc[h], k[h])
            np.testing.assert_array_equal(vc[h], v[h])
        q = r.normal(size=(Hq, d))
        full, _ = O.decode_gqa(q, [(k[h], v[h]) for h in range(Hkv)])
        comp, _ = O.decode_gqa(q, list(zip(kc, vc)))
        np.testing.assert_array_equal(full, comp)

    def test_compact_then_decode_equals_masked_twin(self):
        r = rng(18)
        Hq, Hkv, L, n, d, cs = 8, 2, 16, 500, 32, 8
        q_obs, k, v = r.normal(size=(Hq, L, d)), r.normal(size=(Hkv, n, d)), r.normal(size=(Hkv, n, d))
        idx = O.select_critical(q_obs, k, [0, 1], cs, 11)
        kc, vc = O.compact_kv(k, v, [0, 1], idx, cs, L)
        q = r.normal(size=(Hq, d))
        comp, _ = O.decode_gqa(q, list(zip(kc, vc)))
        for g in range(Hq):
            h = g // 4
            keep = np.zeros(n, dtype=bool)
            keep[O.compact_rows(n, L, cs, idx[h])] = True
            twin = O.masked_attention_decode(q[g], k[h], v[h], keep, 1 / math.sqrt(d))
            np.testing.assert_allclose(comp[g], twin, atol=1e-13)


# --------------------------------------------------------------------------
# CV scoring: Eq. 1-4
# --------------------------------------------------------------------------

class TestCV:
    def test_hand_worked_toy(self):
        g = json.load(open(os.path.join(GOLDEN, "cv_toy.json")))
        A = np.array(g["A"])
        cv, C, phi = O.cv_from_observation(A, g["k"], g["alpha"])
        assert abs(phi - g["phi_linear_quantile"]) < 1e-15
        assert C.tolist() == g["C_linear_quantile"]
        assert abs(cv - g["cv_linear_quantile"]) < 1e-12

    def test_toy_through_the_attention_path(self):
        # q_i = e_i and k_j = sqrt(d) (log a_1j, log a_2j, 0, ...) give scores
        # log a_ij, so the softmax rows equal the toy rows.
        g = json.load(open(os.path.join(GOLDEN, "cv_toy.json")))
        A = np.array(g["A"])
        d = 128
        q = np.zeros((1, 2, d)); q[0, 0, 0] = q[0, 1, 1] = 1.0
        k = np.zeros((1, 4, d)); k[0, :, 0] = np.log(A[0]) * math.sqrt(d); k[0, :, 1] = np.log(A[1]) * math.sqrt(d)
        cv = O.score_heads(q, 10, k, 0, 0, g["k"], g["alpha"], causal=True)
        assert abs(cv[0] - math.sqrt(3)) < 1e-12
        # four identical query heads sharing the KV head: same score
        cv4 = O.score_heads(np.repeat(q, 4, axis=0), 10, k, 0, 0, g["k"], g["alpha"])
        assert abs(cv4[0] - math.sqrt(3)) < 1e-12

    @pytest.mark.parametrize("N,m,L", [(1000, 10, 8), (4096, 40, 16), (777, 7, 3)])
    def test_closed_form_planted_columns(self, N, m, L):
        # m columns hold all the mass of every row: C = L on those columns and 0
        # elsewhere, so cv = sqrt((N - m) / m)
        A = np.zeros((L, N))
        cols = rng(N).choice(N, size=m, replace=False)
        A[:, cols] = 1.0 / m
        cv, C, _ = O.cv_from_observation(A, 0.999, 1.0)
        assert sorted(np.nonzero(C)[0].tolist()) == sorted(cols.tolist())
        assert abs(cv - math.sqrt((N - m) / m)) < 1e-12

    def test_constant_counts_give_zero(self):
        A = np.full((5, 40), 1 / 40)
        assert O.cv_from_observation(A, 0.9, 1.0)[0] == 0.0

    def test_zero_mean_gives_zero(self):
        A = np.full((3, 10), 0.1)
        assert O.cv_from_observation(A, 0.5, 2.0)[0] == 0.0

    def test_scale_invariance_of_binarisation(self):
        r = rng(20)
        A = r.random((8, 300))
        c1, C1, _ = O.cv_from_observation(A, 0.97, 0.9)
        c2, C2, _ = O.cv_from_observation(A * 4.0, 0.97, 0.9)
        assert c1 == c2 and (C1 == C2).all()

    def test_rows_are_softmax_restricted_to_key_range(self):
        r = rng(21)
        G, Lq, n, d = 2, 6, 50, 16
        q, k = r.normal(size=(G, Lq, d)), r.normal(size=(n, d))
        A = O.cv_observation_matrix(q, k, q_pos0=n - Lq, l_init=3, l_rec=4, scale=0.25, causal=True)
        assert A.shape == (Lq, n - 7)
        np.testing.assert_allclose(A.sum(axis=1), np.ones(Lq), atol=1e-13)
        # row i sits at absolute position n - Lq + i: keys beyond it carry no weight
        for i in range(Lq):
            pos = n - Lq + i
            assert (A[i, pos - 3 + 1:] == 0).all()
            assert (A[i, :pos - 3 + 1] > 0).all()

    def test_causal_mask_is_a_noop_for_decode_rows(self):
        r = rng(22)
        q, k = r.normal(size=(2, 4, 16)), r.normal(size=(60, 16))
        A1 = O.cv_observation_matrix(q, k, 60, 5, 2, 0.25, causal=True)
        A2 = O.cv_observation_matrix(q, k, 60, 5, 2, 0.25, causal=False)
        np.testing.assert_array_equal(A1, A2)

    def test_excluded_tokens_do_not_matter(self):
        # changing keys outside [l_init, n - l_rec) leaves the score unchanged
        r = rng(23)
        q, k = r.normal(size=(4, 8, 16)), r.normal(size=(1, 80, 16))
        a = O.score_heads(q, 80, k, 6, 9, 0.9, 1.0)
        k2 = k.copy(); k2[0, :6] = 50.0; k2[0, -9:] = -50.0
        b = O.score_heads(q, 80, k2, 6, 9, 0.9, 1.0)
        assert a[0] == b[0]

    def test_concentrated_head_scores_higher(self):
        # a head whose rows agree on a few keys scores above a diffuse head
        r = rng(24)
        d, n, L = 32, 400, 16
        k = r.normal(size=(2, n, d))
        u = r.normal(size=d); u /= np.linalg.norm(u)
        hot = r.choice(n - 20, size=5, replace=False) + 10
        k[0, hot] = 8 * math.sqrt(d) * u
        q = r.normal(size=(2, L, d)) * 0.3
        q[0] += u
        cv = O.score_heads(q, n, k, 4, 4, 0.99, 1.0)
        assert cv[0] > cv[1]


# --------------------------------------------------------------------------
# quantile and Eq. 5 / static identification
# --------------------------------------------------------------------------

class TestQuantileAndClassify:
    @pytest.mark.parametrize("p", [0.0, 0.25, 0.4, 0.5, 0.9, 0.996, 1.0])
    def test_quantile_matches_library(self, p):
        x = rng(30).normal(size=(7, 13))
        assert abs(O.quantile_type7(x, p) - float(np.quantile(x, p, method="linear"))) < 1e-14

    def test_quantile_hand_values(self):
        assert O.quantile_type7(np.array([4., 1., 3., 2.]), 0.5) == 2.5
        assert O.quantile_type7(np.array([5.]), 0.3) == 5.0

    @pytest.mark.parametrize("r,n_cons", [(0.25, 6), (0.4, 5), (0.5, 4)])
    def test_eq5_counts_for_eight_heads(self, r, n_cons):
        s = rng(31).permutation(np.arange(8) * 0.1 + 0.05)
        c = O.classify_sample(s, r)
        assert c.sum() == n_cons
        assert set(np.argsort(s)[-n_cons:]) == set(np.nonzero(c)[0])

    def test_eq5_tie_at_threshold_is_adaptive(self):
        # r = 0.5: Gamma interpolates between the 4th and 5th smallest scores,
        # both 4, so Gamma = 4 and neither head equal to it is strictly above
        s = np.array([1., 2., 3., 4., 4., 5., 6., 7.])
        c = O.classify_sample(s, 0.5)
        assert c.tolist() == [False, False, False, False, False, True, True, True]

    def test_static_identification(self):
        # head 0 is consistent in 2 of 3 samples, head 3 in all, others vary
        sc = np.array([[9., 1., 2., 8.],
                       [9., 3., 1., 8.],
                       [0., 5., 4., 9.]])
        st = O.static_head_types(sc, 0.5)
        # r = 0.5 with H = 4: Eq. 5 keeps 2 heads per sample
        assert st.tolist() == [True, False, False, True]
        assert O.static_head_types(sc[:1], 0.5).tolist() == O.classify_sample(sc[0], 0.5).tolist()

    @pytest.mark.parametrize("r,n_cons", [(0.25, 6), (0.3, 5), (0.4, 5), (0.5, 4)])
    def test_static_set_size_equals_one_sample_of_distinct_scores(self, r, n_cons):
        # eight heads, distinct scores: Eq. 5 keeps the heads strictly above the
        # linear r-quantile; the static set over several samples keeps as many
        sc = np.stack([rng(32 + s).permutation(np.arange(8) * 0.1 + 0.05) for s in range(5)])
        assert O.classify_sample(sc[0], r).sum() == n_cons
        assert O.static_head_types(sc, r).sum() == n_cons


class TestAroundDecoding:
    """Generation-loop append, retention below 1, query-aware retrieval and
    attention recall."""

    def test_append_reproduces_the_longer_sequence(self):
        r = rng(40)
        n, T, d = 50, 7, 16
        K, V = r.normal(size=(n + T, d)), r.normal(size=(n + T, d))
        k, v = K[:n], V[:n]
        for t in range(T):
            k, v, ok = O.append_token(k, v, K[n + t], V[n + t], capacity=n + T)
            assert ok
        assert np.array_equal(k, K) and np.array_equal(v, V)
        # decoding the grown view is attention over the whole sequence (library SDPA)
        q = r.normal(size=d)
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q)[None, None, None], torch.from_numpy(K)[None, None],
            torch.from_numpy(V)[None, None], scale=0.25)[0, 0, 0].numpy()
        np.testing.assert_allclose(O.attention_decode(q, k, v, 0.25)[0], ref, atol=1e-12)

    def test_append_stops_at_capacity(self):
        k, v = np.zeros((3, 4)), np.zeros((3, 4))
        k2, v2, ok = O.append_token(k, v, np.ones(4), np.ones(4), capacity=3)
        assert not ok and k2.shape[0] == 3

    def test_adaptive_budget_hand_values(self):
        # n - l_obs = 90 keys -> 12 chunks of 8 (the last one partial)
        assert [O.adaptive_budget(100, 10, 8, e) for e in (1.0, 0.5, 0.3, 0.25, 0.0)] == [12, 6, 4, 3, 0]

    def test_retention_one_keeps_the_whole_cache(self):
        r = rng(41)
        n, l_obs, cs = 61, 5, 8
        q, k = r.normal(size=(2, l_obs, 16)), r.normal(size=(1, n, 16))
        b = O.adaptive_budget(n, l_obs, cs, 1.0)
        idx = O.select_critical(q, k, [0], cs, b)[0]
        assert np.array_equal(O.compact_rows(n, l_obs, cs, idx), np.arange(n))

    def test_page_bounds_match_library_reduction(self):
        r = rng(42)
        k = r.normal(size=(37, 5))
        kmin, kmax = O.page_bounds(k, 8)
        starts = np.arange(0, 37, 8)
        np.testing.assert_array_equal(kmin, np.minimum.reduceat(k, starts, axis=0))
        np.testing.assert_array_equal(kmax, np.maximum.reduceat(k, starts, axis=0))

    @pytest.mark.parametrize("seed", [0, 1, 2])
    def test_page_score_bounds_every_token(self, seed):
        r = rng(43 + seed)
        k, qg = r.normal(size=(45, 12)), r.normal(size=(4, 12))
        kmin, kmax = O.page_bounds(k, 8)
        sc = O.page_scores(qg, kmin, kmax)
        for c in range(sc.shape[0]):
            rows = k[c * 8:(c + 1) * 8]
            assert sc[c] >= (qg @ rows.T).max() - 1e-12

    def test_page_score_is_tight_for_single_rows_and_repeated_rows(self):
        r = rng(46)
        k, qg = r.normal(size=(9, 6)), r.normal(size=(2, 6))
        kmin, kmax = O.page_bounds(k, 1)
        np.testing.assert_allclose(O.page_scores(qg, kmin, kmax), (qg @ k.T).max(axis=0), atol=1e-12)
        rep = np.repeat(k[:2], 4, axis=0)            # two pages of four identical rows
        kmin, kmax = O.page_bounds(rep, 4)
        np.testing.assert_allclose(O.page_scores(qg, kmin, kmax), (qg @ k[:2].T).max(axis=0), atol=1e-12)

    def test_page_score_one_dimension_is_the_exact_maximum(self):
        r = rng(47)
        k, q = r.normal(size=(20, 1)), r.normal(size=(1, 1))
        kmin, kmax = O.page_bounds(k, 5)
        np.testing.assert_allclose(O.page_scores(q, kmin, kmax), (q @ k.T).reshape(4, 5).max(axis=1), atol=1e-12)

    def test_retrieval_with_single_row_pages_is_token_topk(self):
        r = rng(48)
        k, qg = r.normal(size=(30, 8)), r.normal(size=(3, 8))
        got = O.retrieve_pages(qg, k, 1, 7)
        best = (qg @ k.T).max(axis=0)
        assert set(got.tolist()) == set(np.argsort(-best)[:7].tolist())
        assert (np.diff(got) > 0).all()

    def test_recall_extremes_and_topk_optimality(self):
        r = rng(49)
        k, q = r.normal(size=(8, 4)), r.normal(size=4)
        assert abs(O.attention_recall(q, k, np.arange(8), 0.5) - 1.0) < 1e-12
        assert O.attention_recall(q, k, np.zeros(0, dtype=np.int64), 0.5) == 0.0
        best = max(O.attention_recall(q, k, np.array(c), 0.5) for c in itertools.combinations(range(8), 3))
        assert abs(O.attention_recall(q, k, O.topk_keep(q, k, 3, 0.5), 0.5) - best) < 1e-12

    def test_streaming_and_chunk_rows(self):
        assert O.streaming_keep(10, 4, 1).tolist() == [0, 7, 8, 9]
        assert O.streaming_keep(5, 9, 2).tolist() == [0, 1, 2, 3, 4]
        assert O.chunk_rows(20, 8, np.array([2, 0])).tolist() == list(range(8)) + [16, 17, 18, 19]
