"""Pins of the oracle's Philox generator, noise transforms and parameter init."""
import math
import os

import numpy as np
import pytest
from scipy import stats

from oracle import noise, params, philox

GOLD = os.path.join(os.path.dirname(__file__), "golden", "philox_kat.txt")


def _kat():
    rows = []
    for line in open(GOLD):
        if line.startswith("#") or not line.strip():
            continue
        v = [int(t, 16) for t in line.split()]
        rows.append((v[:4], v[4:6], v[6:10]))
    return rows


@pytest.mark.parametrize("ctr,key,want", _kat())
def test_philox_known_answers_scalar(ctr, key, want):
    assert list(philox.philox_scalar(ctr, key)) == want


@pytest.mark.parametrize("ctr,key,want", _kat())
def test_philox_known_answers_vector(ctr, key, want):
    out = philox.philox(*[np.array([c]) for c in ctr], *[np.array([k]) for k in key])
    assert [int(o[0]) for o in out] == want


def test_philox_vector_matches_scalar_random():
    r = np.random.default_rng(0)
    c = r.integers(0, 2 ** 32, size=(6, 200), dtype=np.uint64)
    out = philox.philox(*c)
    for i in range(200):
        s = philox.philox_scalar(c[:4, i], c[4:, i])
        assert tuple(int(o[i]) for o in out) == s


def test_counter_words_layout():
    seed = 0x1234567890ABCDEF
    k = (seed & 0xFFFFFFFF, seed >> 32)
    w = philox.counter_words(seed, philox.STREAM_CLASS, 7, 11, np.arange(10))
    for j in range(10):
        blk = philox.philox_scalar((j >> 2, 11, 7, philox.STREAM_CLASS), k)
        assert int(w[j]) == blk[j & 3]


def test_uniform_exact_endpoints():
    assert noise.uniform(0) == 2.0 ** -33
    assert noise.uniform(2 ** 32 - 1) == 1.0 - 2.0 ** -33
    assert noise.complement(2 ** 32 - 1) == 2.0 ** -33


def test_exponential_relative_accuracy_near_one():
    # u = 1 - 2^-33 -> E = -log(1 - 2^-33) = 2^-33 + 2^-67 + ...
    c = 2.0 ** -33
    e = noise.exponential(np.array([2 ** 32 - 1], dtype=np.uint32))[0]
    assert abs(e / (c + c * c / 2) - 1.0) < 1e-15
    # u = 2^-33 -> E = 33 log 2
    e0 = noise.exponential(np.array([0], dtype=np.uint32))[0]
    assert abs(e0 - 33 * math.log(2.0)) < 1e-13


def _words(n, stream=5):
    return philox.counter_words(99, stream, 0, 0, np.arange(n))


def test_uniform_ks():
    assert stats.kstest(noise.uniform(_words(20000)), "uniform").pvalue > 1e-3


def test_exponential_ks():
    assert stats.kstest(noise.exponential(_words(20000)), "expon").pvalue > 1e-3


def test_gumbel_ks():
    assert stats.kstest(noise.gumbel(_words(20000)), "gumbel_r").pvalue > 1e-3


def test_normal_icdf_ks_monotone_symmetric():
    w = _words(20000)
    assert stats.kstest(noise.normal_icdf(w), "norm").pvalue > 1e-3
    ws = np.sort(w)
    assert np.all(np.diff(noise.normal_icdf(ws)) >= 0)
    assert np.allclose(noise.normal_icdf(ws), -noise.normal_icdf(np.uint32(2 ** 32 - 1) - ws), atol=1e-12)


def test_box_muller_ks():
    w = philox.philox(np.arange(10000), 0, 0, 0, 1, 2)
    z = np.concatenate([noise.box_muller(w[0], w[1], False), noise.box_muller(w[0], w[1], True)])
    assert stats.kstest(z, "norm").pvalue > 1e-3


def test_round_bf16_ties_and_fp32_agreement():
    assert params.round_bf16(1.0 + 2.0 ** -8) == 1.0
    assert params.round_bf16(1.0 + 3 * 2.0 ** -8) == 1.0 + 2.0 ** -6
    assert params.round_bf16(-(1.0 + 3 * 2.0 ** -8)) == -(1.0 + 2.0 ** -6)
    assert params.round_bf16(1.0 + 2.0 ** -8 + 2.0 ** -40) == 1.0 + 2.0 ** -7
    # for fp32 inputs, direct rounding equals the classic fp32 -> bf16 bit rounding
    f = (np.random.default_rng(1).standard_normal(5000) * 0.02).astype(np.float32)
    b = f.view(np.uint32).astype(np.uint64)
    b = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    ref = b.astype(np.uint32).view(np.float32).astype(np.float64)
    assert np.array_equal(params.round_bf16(f.astype(np.float64)), ref)


def test_param_elements_from_scalar_philox():
    cfg = dict(n_layers=1, d_model=8, n_heads=2, d_mlp=16, vocab=5, prior="mask",
               dtype="fp32", max_len=4)
    P = params.init_params(cfg, seed=77)
    sp = params.specs(cfg)
    for tid, (name, shape, kind) in enumerate(sp):
        flat = P[name].reshape(-1)
        for e in (0, 1, flat.size - 1):
            w = philox.philox_scalar((e >> 1, 0, tid, philox.STREAM_PARAM), (77, 0))
            u1, u2 = (w[0] + 0.5) * 2.0 ** -32, (w[1] + 0.5) * 2.0 ** -32
            r = math.sqrt(-2.0 * math.log(u1))
            z = r * (math.sin(2 * math.pi * u2) if e & 1 else math.cos(2 * math.pi * u2))
            v = 0.02 * z if kind == "w" else 1.0 + 0.02 * z
            assert flat[e] == float(np.float32(v))
    assert P["tok_emb"].shape == (6, 8) and P["w_out"].shape == (5, 8)
    assert len(sp) == 2 + 12 + 3


def test_param_statistics():
    cfg = dict(n_layers=1, d_model=64, n_heads=2, d_mlp=256, vocab=32, prior="mask",
               dtype="bf16", max_len=32)
    P = params.init_params(cfg, seed=5)
    w = P["l0.w_1"].reshape(-1)
    assert abs(w.std() - 0.02) < 0.002 and abs(w.mean()) < 0.002
    g = P["l0.ln1_g"]
    assert abs(g.mean() - 1.0) < 0.02
    assert np.array_equal(params.round_bf16(w), w)
