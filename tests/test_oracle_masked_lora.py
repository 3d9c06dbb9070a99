"""Pins of the attention patterns and the gated-LoRA forward pass of the oracle.

Patterns (Sec. 3.1 causal AR pathway, Sec. 3.2 block diffusion over [x, z_1],
Sec. 4.1 drafting) are pinned by closed-form pair counts, reductions between
patterns, and by the reach of a perturbation through the whole network.  The
gated adapters (Sec. 3.2, Sec. 4.1; W + (alpha/r) B A of App. "Varying LoRA
alpha / r") are pinned by the merged-weight identity, by gates-off == base
model, by the scalar-loop forward and by the teacher property of Sec. 3.2.
"""
import numpy as np
import pytest

from oracle import forward, forward_loops, masks, params

CFG = dict(n_layers=2, d_model=16, n_heads=2, d_mlp=40, vocab=11, prior="mask",
           dtype="fp32", max_len=12, time_cond=True, norm_eps=1e-5)
LCFG = dict(CFG, lora_rank=4, lora_alpha=8.0)


def _P(cfg, seed=3, scale=10.0):
    P = params.init_params(cfg, seed)
    return {k: (v * scale if not k.endswith("_g") else v) for k, v in P.items()}


def _z(B, L, V=11, seed=0):
    return np.random.default_rng(seed).integers(0, V + 1, size=(B, L))


# ---------------------------------------------------------------- patterns

@pytest.mark.parametrize("L", [1, 5, 12])
def test_pattern_counts(L):
    assert masks.bidirectional(L).sum() == L * L
    assert masks.causal(L).sum() == L * (L + 1) // 2
    for bs in (1, 2, 3, 5):
        full, rem = divmod(L, bs)
        sizes = [bs] * full + ([rem] if rem else [])
        before = np.concatenate([[0], np.cumsum(sizes)])[:-1]
        want = sum(s * (b + s) for s, b in zip(sizes, before))
        assert masks.block_causal(L, bs).sum() == want


@pytest.mark.parametrize("N,bs", [(1, 1), (1, 4), (3, 2), (2, 5)])
def test_draft_training_counts_and_blocks(N, bs):
    v = masks.draft_training(N, bs)
    n = N * bs
    assert v.shape == (2 * n, 2 * n)
    assert v[:n, :n].sum() == n * (n + 1) // 2 and not v[:n, n:].any()
    for b in range(N):
        rows = slice(n + b * bs, n + (b + 1) * bs)
        assert v[rows, :b * bs].all() and not v[rows, b * bs:n].any()
        assert np.array_equal(v[rows, n + b * bs:n + (b + 1) * bs], np.tril(np.ones((bs, bs), bool)))
        others = np.ones(n, bool)
        others[b * bs:(b + 1) * bs] = False
        assert not v[rows, n:][:, others].any()
    assert v.diagonal().all()


def test_pattern_reductions():
    assert np.array_equal(masks.block_causal(9, 1), masks.causal(9))
    assert np.array_equal(masks.block_causal(9, 9), masks.bidirectional(9))
    assert np.array_equal(masks.block_causal(9, 20), masks.bidirectional(9))
    # a single block: z_1 sees no clean block and is causal within itself, like x
    v = masks.draft_training(1, 6)
    assert np.array_equal(v[6:, 6:], masks.causal(6)) and not v[6:, :6].any()


# ---------------------------------------------------------------- forward under patterns

def _patterns(L):
    return {"causal": masks.causal(L), "block3": masks.block_causal(L, 3),
            "block5": masks.block_causal(L, 5), "train": masks.draft_training(L // 6, 3)}


@pytest.mark.parametrize("name", ["causal", "block3", "block5", "train"])
def test_masked_forward_equals_scalar_loops(name):
    L = 12
    vis = _patterns(L)[name]
    P = _P(CFG)
    z = _z(2, L)
    a = forward.forward(CFG, P, z, 0.4, vis)
    b = np.array(forward_loops.forward_loops(CFG, P, z, 0.4, vis.tolist()))
    assert np.abs(a - b).max() < 1e-10 * max(1.0, np.abs(a).max())


def test_bidirectional_pattern_equals_unmasked():
    P = _P(CFG)
    z = _z(2, 9)
    assert np.array_equal(forward.forward(CFG, P, z, 0.3, masks.bidirectional(9)),
                          forward.forward(CFG, P, z, 0.3))


@pytest.mark.parametrize("name", ["causal", "block3", "block5", "train"])
def test_perturbation_reaches_exactly_the_positions_that_see_it(name):
    """Under a pattern, position p influences position i iff i reaches p through visible keys.

    For the patterns here visibility is transitive (every visible key's own visible set is a
    subset of the query's, up to the query itself), so i depends on p iff vis[i, p]."""
    L = 12
    vis = _patterns(L)[name]
    P = _P(CFG)
    z = _z(1, L, seed=4)
    base = forward.forward(CFG, P, z, 0.3, vis)
    for p in range(L):
        z2 = z.copy()
        z2[0, p] = (z2[0, p] + 5) % 12
        out = forward.forward(CFG, P, z2, 0.3, vis)
        changed = np.abs(out - base).max(axis=-1)[0] > 1e-9
        unchanged_exact = np.array_equal(out[0, ~vis[:, p]], base[0, ~vis[:, p]])
        assert unchanged_exact, (name, p)
        assert np.array_equal(changed, vis[:, p]), (name, p, changed.astype(int), vis[:, p].astype(int))


# ---------------------------------------------------------------- gated adapters

def test_lora_param_storage_roundtrip():
    P = params.init_params(LCFG, 9)
    r = LCFG["lora_rank"]
    assert P["l0.w_qkv"].shape == (48, 16) and P["l0.lora_b_qkv"].shape == (48, r)
    assert P["l1.lora_a_2"].shape == (r, 40) and P["l1.lora_b_2"].shape == (16, r)
    st = params.storage_tensors(LCFG, P)
    sp = params.specs(LCFG)
    assert len(st) == len(sp) == 2 + 12 * 2 + 3 + 4 * 2
    for a, (name, shape, _) in zip(st, sp):
        assert a.shape == tuple(shape), name
    # the base tensors of a LoRA config are the leading columns of the stored rows
    assert np.array_equal(st[4][:, :16], P["l0.w_qkv"]) and np.array_equal(st[4][:, 16:], P["l0.lora_b_qkv"])


def _merged(cfg, P):
    """Base-model parameters with each W replaced by W + (alpha/r) B A."""
    s = cfg["lora_alpha"] / cfg["lora_rank"]
    Q = {k: v for k, v in P.items() if "lora_" not in k}
    for l in range(cfg["n_layers"]):
        for p in params.PROJ:
            Q[f"l{l}.w_{p}"] = P[f"l{l}.w_{p}"] + s * P[f"l{l}.lora_b_{p}"] @ P[f"l{l}.lora_a_{p}"]
    return Q


def test_all_gates_on_equals_merged_weights():
    P = _P(LCFG, scale=5.0)
    z = _z(2, 8)
    base_cfg = dict(LCFG, lora_rank=0)
    a = forward.forward(LCFG, P, z, 0.6)
    b = forward.forward(base_cfg, _merged(LCFG, P), z, 0.6)
    assert np.abs(a - b).max() < 1e-10 * max(1.0, np.abs(a).max())
    lora_only = forward.forward(base_cfg, {k: v for k, v in P.items() if "lora_" not in k}, z, 0.6)
    assert np.abs(a - lora_only).max() > 1e-2   # the adapters matter at this scale


def test_all_gates_off_equals_base_model():
    P = _P(LCFG, scale=5.0)
    z = _z(2, 8)
    vis = masks.causal(8)
    a = forward.forward(LCFG, P, z, 0.6, vis, gate=np.zeros(8))
    b = forward.forward(dict(LCFG, lora_rank=0), {k: v for k, v in P.items() if "lora_" not in k}, z, 0.6, vis)
    assert np.array_equal(a, b)


@pytest.mark.parametrize("pattern", [None, "causal", "train"])
def test_gated_lora_equals_scalar_loops(pattern):
    L = 12
    vis = None if pattern is None else _patterns(L)[pattern]
    gate = (np.arange(L) % 3 != 1).astype(float)
    P = _P(LCFG, scale=5.0)
    z = _z(2, L, seed=7)
    a = forward.forward(LCFG, P, z, 0.25, vis, gate)
    b = np.array(forward_loops.forward_loops(LCFG, P, z, 0.25, None if vis is None else vis.tolist(),
                                             gate.tolist()))
    assert np.abs(a - b).max() < 1e-10 * max(1.0, np.abs(a).max())


def test_teacher_logits_from_one_pass_over_x_and_z():
    """Sec. 3.2: in one pass over [x, z_1] with the block-causal pattern and adapters on z_1 only,
    the logits at x are the base model's causal logits on x alone."""
    N, bs = 2, 3
    n = N * bs
    P = _P(LCFG, scale=5.0)
    x = _z(2, n, V=10, seed=11)
    z1 = np.full((2, n), 11)                          # the all-mask z_1
    seq = np.concatenate([x, z1], axis=1)
    gate = np.concatenate([np.zeros(n), np.ones(n)])
    out = forward.forward(LCFG, P, seq, 1.0, masks.draft_training(N, bs), gate)
    base = forward.forward(dict(LCFG, lora_rank=0), {k: v for k, v in P.items() if "lora_" not in k},
                           x, 1.0, masks.causal(n))
    assert np.abs(out[:, :n] - base).max() < 1e-12 * max(1.0, np.abs(base).max())
    # and the z_1 logits do use the adapters
    out_off = forward.forward(LCFG, P, seq, 1.0, masks.draft_training(N, bs), np.zeros(2 * n))
    assert np.abs(out[:, n:] - out_off[:, n:]).max() > 1e-3
