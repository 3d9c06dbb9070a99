"""Pins of the oracle denoiser forward pass (the paper fixes no values for it)."""
import numpy as np

from oracle import forward, forward_loops, params

CFG = dict(n_layers=2, d_model=16, n_heads=2, d_mlp=40, vocab=11, prior="mask",
           dtype="fp32", max_len=7, time_cond=True, norm_eps=1e-5)


def _P(cfg=CFG, seed=3, scale=None):
    P = params.init_params(cfg, seed)
    if scale:   # larger weights make every term matter numerically
        P = {k: (v * scale if not k.endswith("_g") else v) for k, v in P.items()}
    return P


def _z(B=2, L=7, V=11, seed=0):
    return np.random.default_rng(seed).integers(0, V + 1, size=(B, L))


def test_vectorised_equals_scalar_loops():
    P = _P(scale=20.0)
    z = _z()
    for at in (0.0, 0.37, 1.0):
        a = forward.forward(CFG, P, z, at)
        b = np.array(forward_loops.forward_loops(CFG, P, z, at))
        assert a.shape == (2, 7, 11)
        assert np.abs(a - b).max() < 1e-10 * max(1.0, np.abs(a).max())


def test_time_embedding_values():
    e = forward.time_embedding(1.0, 8)
    assert np.array_equal(e, np.array([0, 0, 0, 0, 1, 1, 1, 1], float))
    e = forward.time_embedding(0.5, 4)      # tau = 500, w = (1, 0.01)
    assert np.allclose(e, [np.sin(500.0), np.sin(5.0), np.cos(500.0), np.cos(5.0)], atol=1e-15)


def test_layer_norm_moments():
    x = np.random.default_rng(1).standard_normal((5, 64)) * 3 + 2
    y = forward.layer_norm(x, np.ones(64), np.zeros(64), 0.0)
    assert np.allclose(y.mean(-1), 0, atol=1e-12) and np.allclose(y.var(-1), 1, atol=1e-12)


def test_permutation_equivariance_without_positions():
    P = _P(scale=10.0)
    P["pos_emb"] = np.zeros_like(P["pos_emb"])
    z = _z(B=1)
    perm = np.random.default_rng(2).permutation(7)
    a = forward.forward(CFG, P, z, 0.3)
    b = forward.forward(CFG, P, z[:, perm], 0.3)
    assert np.allclose(a[:, perm], b, atol=1e-12)


def test_attention_is_not_causal():
    P = _P(scale=10.0)
    z = _z(B=1)
    z2 = z.copy()
    z2[0, -1] = (z2[0, -1] + 1) % 12
    a = forward.forward(CFG, P, z, 0.3)
    b = forward.forward(CFG, P, z2, 0.3)
    assert np.abs(a[0, 0] - b[0, 0]).max() > 1e-6


def test_time_conditioning_changes_output():
    P = _P(scale=10.0)
    z = _z(B=1)
    assert np.abs(forward.forward(CFG, P, z, 0.1) - forward.forward(CFG, P, z, 0.9)).max() > 1e-6
    cfg = dict(CFG, time_cond=False)
    assert np.array_equal(forward.forward(cfg, P, z, 0.1), forward.forward(cfg, P, z, 0.9))


def test_x_theta_is_softmax():
    l = np.random.default_rng(3).standard_normal((4, 9)) * 5
    x = forward.x_theta(l)
    assert np.allclose(x.sum(-1), 1) and np.allclose(np.log(x[:, 1] / x[:, 0]), l[:, 1] - l[:, 0])
