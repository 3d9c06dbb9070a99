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


def test_rms_norm_unit_mean_square_and_scale_invariance():
    """With unit gain and eps = 0 every output row has mean square 1, and scaling a row by a > 0
    leaves it unchanged (the defining properties of RMS normalisation)."""
    x = np.random.default_rng(2).standard_normal((5, 64)) * 3 + 2
    y = forward.rms_norm(x, np.ones(64), 0.0)
    assert np.allclose((y ** 2).mean(-1), 1, atol=1e-12)
    assert np.allclose(forward.rms_norm(7.5 * x, np.ones(64), 0.0), y, atol=1e-12)
    # the mean is not removed: a row's sign pattern and the ratios of its entries survive
    assert np.allclose(y / y[:, :1], x / x[:, :1], atol=1e-10)


def test_rms_norm_closed_form_on_constant_rows():
    g = np.linspace(0.5, 2.0, 8)
    for c, eps in ((3.0, 0.0), (-0.25, 1e-2), (1e-3, 1e-5)):
        y = forward.rms_norm(np.full((1, 8), c), g, eps)
        assert np.allclose(y[0], c / np.sqrt(c * c + eps) * g, rtol=1e-14, atol=0)


def test_rms_norm_equals_layer_norm_on_centred_rows():
    """On rows of mean zero the mean square is the biased variance, so RMSNorm and LayerNorm with a
    zero shift coincide (for any eps)."""
    rng = np.random.default_rng(4)
    x = rng.standard_normal((6, 32)) * 2.5
    x -= x.mean(-1, keepdims=True)
    g = rng.uniform(0.5, 1.5, 32)
    for eps in (0.0, 1e-5, 0.3):
        assert np.allclose(forward.rms_norm(x, g, eps), forward.layer_norm(x, g, np.zeros(32), eps),
                           atol=1e-13)


def test_rms_norm_equals_library():
    torch = __import__("pytest").importorskip("torch")
    rng = np.random.default_rng(5)
    x, g = rng.standard_normal((4, 48)) * 3 + 1, rng.uniform(0.5, 1.5, 48)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (48,), torch.from_numpy(g), eps=1e-5).numpy()
    assert np.allclose(forward.rms_norm(x, g, 1e-5), ref, rtol=1e-13, atol=1e-13)


def test_rms_forward_vectorised_equals_scalar_loops():
    cfg = dict(CFG, norm="rms")
    P = _P(cfg, scale=20.0)
    z = _z()
    a = forward.forward(cfg, P, z, 0.37)
    b = np.array(forward_loops.forward_loops(cfg, P, z, 0.37))
    assert np.abs(a - b).max() < 1e-10 * max(1.0, np.abs(a).max())
    # and the shift vectors are not read: changing them changes nothing
    P2 = {k: (v + 1.0 if k.endswith("_b") and "ln" in k else v) for k, v in P.items()}
    assert np.array_equal(forward.forward(cfg, P2, z, 0.37), a)
    # while under LayerNorm the same change moves the logits
    assert np.abs(forward.forward(CFG, P2, z, 0.37) - forward.forward(CFG, P, z, 0.37)).max() > 1e-3


def test_unknown_norm_is_refused():
    import pytest
    with pytest.raises(ValueError):
        forward.forward(dict(CFG, norm="group"), _P(), _z(), 0.5)


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
