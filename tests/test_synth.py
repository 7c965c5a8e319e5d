"""The seeded input generator: determinism, bf16 rounding and workload recipes."""
import numpy as np
import pytest
import torch

import synth


def test_bf16_rounding_matches_library_round_to_nearest_even():
    r = np.random.default_rng(0)
    x = np.concatenate([
        r.normal(size=20000).astype(np.float32) * np.float32(7.0),
        np.array([0.0, -0.0, 1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 3.0e38, -3.4e38,
                  1e-40, np.inf, -np.inf], dtype=np.float32)])
    ours = synth.f32_to_bf16_bits(x)
    lib = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, lib)
    # hand cases: a tie rounds to even, just above a tie rounds up
    assert synth.f32_to_bf16_bits(np.float32([1.0 + 2 ** -8]))[0] == 0x3F80
    assert synth.f32_to_bf16_bits(np.float32([1.0 + 3 * 2 ** -8]))[0] == 0x3F82


def test_widening_is_exact():
    bits = np.arange(0, 65536, 97, dtype=np.uint16)
    f = synth.bf16_bits_to_f32(bits)
    fin = np.isfinite(f)
    np.testing.assert_array_equal(synth.f32_to_bf16_bits(f[fin]), bits[fin])


def small(name, **kw):
    return synth.WORKLOADS[name].scaled(**kw)


def test_same_seed_same_bytes_and_order_independence():
    wl = small("ctx32k_bf16", n=700, hkv=2, hq=8)
    a = synth.make_sequence(wl)
    _ = synth.decode_queries(wl, 3)          # draw something else in between
    b = synth.make_sequence(wl)
    for x, y in [(a.k, b.k), (a.v, b.v), (a.q_obs, b.q_obs)]:
        assert x.tobytes() == y.tobytes()
    assert synth.decode_queries(wl, 5).tobytes() == synth.decode_queries(wl, 5).tobytes()
    assert synth.decode_queries(wl, 5).tobytes() != synth.decode_queries(wl, 6).tobytes()
    c = synth.make_sequence(wl.scaled(seed=wl.seed + 1))
    assert c.k.tobytes() != a.k.tobytes()


def test_heavy_hitter_recipe():
    wl = small("ctx32k_bf16", n=4000, hkv=2, hq=8)
    s = synth.make_sequence(wl)
    assert s.k.dtype == np.uint16 and s.k.shape == (2, 4000, 128)
    k = synth.storage_to_f64(s.k)
    for h in range(2):
        assert len(s.planted[h]) == 40
        norms = np.linalg.norm(k[h], axis=1)
        # scaled rows have ~3x the norm of the others
        assert norms[s.planted[h]].mean() > 2.5 * np.delete(norms, s.planted[h]).mean()


def test_direction_recipe():
    wl = synth.WORKLOADS["ctx4k_f32"].scaled(n=600, hkv=2, hq=8)
    s = synth.make_sequence(wl)
    assert s.k.dtype == np.float32
    q = s.q_obs.astype(np.float64)
    for h in range(2):
        u = q[h * 4:(h + 1) * 4].reshape(-1, 128).mean(axis=0)
        u /= np.linalg.norm(u)
        proj = s.k[h].astype(np.float64) @ u
        assert (proj[s.planted[h]] > 30).all()
        assert np.abs(np.delete(proj, s.planted[h])).max() < 6
        assert s.planted[h].max() < 600 - wl.l_obs


def test_ragged_lengths_and_calibration_rows():
    wl = synth.WORKLOADS["batch16_ragged_bf16"]
    lens = synth.sequence_lengths(wl)
    assert len(lens) == 16 and min(lens) >= 16384 and max(lens) <= 65536
    assert lens == synth.sequence_lengths(wl)
    wl5 = synth.WORKLOADS["ctx1m_bf16"].scaled(n=2000, hkv=1, hq=4)
    s = synth.make_sequence(wl5)
    assert s.q_cv.shape == (4, 32, 128) and s.q_cv_pos0 == 2000
    assert s.q_obs.shape == (4, 64, 128)


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_workload_knobs_are_consistent(name):
    wl = synth.WORKLOADS[name]
    assert wl.hq % wl.hkv == 0 and wl.budget % wl.cs == 0
    assert wl.l_init == wl.budget // 32 and wl.l_rec == wl.budget // 128
