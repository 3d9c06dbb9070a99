"""The C ABI: exported symbols, layouts and host-side validation (no GPU needed).

Validation failures must return their status before any launch, so they can be
exercised here with dummy non-null pointers that are never dereferenced.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import workloads
from oracle import params as oparams, sampler as osampler
from paper_2609_04010_amd import _lib as dd

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "dd.h")
FAKE = ctypes.c_void_p(0x10000)  # never dereferenced: every call below fails validation first


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dd_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    L = dd.lib()
    names = _declared()
    assert len(names) >= 20
    for n in names:
        assert hasattr(L, n), n
    assert sorted(dd.EXPORTED) == names


@pytest.mark.parametrize("c", [1, 2, 5])
def test_param_layout_matches_oracle_tensor_list(c):
    cfg = workloads.model_cfg(c)
    specs = oparams.specs(cfg)
    assert dd.param_count(cfg) == len(specs)
    es = 2 if cfg["dtype"] == "bf16" else 4
    end = 0
    for tid, (name, shape, _) in enumerate(specs):
        off, r, cc = dd.param_tensor(cfg, tid)
        n = int(np.prod(shape))
        assert r * cc == n and (r == shape[0] if len(shape) == 2 else r == 1), name
        assert off % 256 == 0 and off >= end
        end = off + n * es
    assert dd.param_bytes(cfg) >= end


def test_sizes_and_noise_width():
    cfg = workloads.model_cfg(2)
    assert dd.logits_ld(50257) == 50304 and dd.logits_ld(32) == 64
    for prior in ("mask", "uniform"):
        for V in (1, 32, 256, 257, 50257):
            assert dd.noise_width(prior, V) == osampler.noise_width(prior, V)
    w1, w2 = dd.workspace_bytes(cfg, 1, 128), dd.workspace_bytes(cfg, 2, 128)
    assert 0 < w1 < w2 < dd.loop_workspace_bytes(cfg, 2, 128)
    assert dd.workspace_bytes(cfg, 0, 128) == 0


def _post(**kw):
    a = dict(prior=0, logits=FAKE, dtype=0, ld=64, rows=4, V=32, mask_id=None, z_t=FAKE, at=0.2, as_=0.5,
             noise=None, seed=0, step=1, row0=0, z_s=FAKE, row_lse=None, probs=None, err=None)
    a.update(kw)
    mid = a["mask_id"] if a["mask_id"] is not None else (a["V"] if a["prior"] == 0 else -1)
    return dd.lib().dd_posterior_sample(a["prior"], a["logits"], a["dtype"], a["ld"], a["rows"],
                                        a["V"], mid, a["z_t"], a["at"], a["as_"], a["noise"], a["seed"],
                                        a["step"], a["row0"], a["z_s"], a["row_lse"], a["probs"], a["err"],
                                        None)


@pytest.mark.parametrize("kw,status", [
    (dict(prior=7), 1), (dict(dtype=9), 3), (dict(V=0), 1), (dict(rows=-1), 1),
    (dict(ld=31), 2), (dict(ld=36), 2), (dict(at=0.5, as_=0.5), 1), (dict(at=0.6, as_=0.5), 1),
    (dict(at=-0.1), 1), (dict(as_=1.5), 1), (dict(logits=None), 1), (dict(z_s=None), 1),
    (dict(mask_id=31), 6), (dict(mask_id=-1), 6), (dict(prior=1, mask_id=32), 6), (dict(prior=1, mask_id=0), 6),
])
def test_posterior_validation(kw, status):
    assert _post(**kw) == status


def test_posterior_mask_id_message():
    """A mask id that does not fit the prior is refused with a reason naming the expected id."""
    assert _post(mask_id=5) == 6
    msg = dd.lib().dd_last_error()
    assert b"mask_id 5" in msg and b"32" in msg


def test_posterior_zero_rows_is_a_noop():
    assert _post(rows=0, logits=None, z_t=None, z_s=None) == 0


def _cfg_struct(**over):
    cfg = workloads.model_cfg(2)
    cfg.update(over)
    return dd.make_config(cfg)


def _fwd(cfg, B=1, L=16, at=0.5, ld=50304, ws_bytes=1 << 40):
    return dd.lib().dd_denoise_forward(ctypes.byref(cfg), FAKE, FAKE, B, L, at, FAKE, ld, FAKE,
                                       ws_bytes, None)


def test_forward_validation():
    assert _fwd(_cfg_struct(), L=2048) == 2            # L > max_len
    assert _fwd(_cfg_struct(mask_id=0)) == 6           # the masked prior's mask is id V
    assert _fwd(_cfg_struct(prior="uniform", mask_id=50257)) == 6   # the uniform prior has none
    assert _fwd(_cfg_struct(), B=0) == 1
    assert _fwd(_cfg_struct(), at=1.5) == 1
    assert _fwd(_cfg_struct(), ld=50257) == 2          # not a multiple of 8
    assert _fwd(_cfg_struct(), ld=50000) == 2          # < V
    assert _fwd(_cfg_struct(), ws_bytes=10) == 4
    assert _fwd(_cfg_struct(n_heads=24)) == 6          # bf16 attention needs dh = 64
    assert _fwd(_cfg_struct(d_model=100, n_heads=4)) in (1, 6)
    bad = _cfg_struct()
    bad.prior = 5
    assert _fwd(bad) == 1
    bad = _cfg_struct()
    bad.dtype = 3
    assert _fwd(bad) == 1
    bad = _cfg_struct()
    bad.norm = 2
    assert _fwd(bad) == 1
    assert dd.lib().dd_last_error() == b"unknown norm 2"
    assert dd.make_config(dict(workloads.model_cfg(2), norm="rms")).norm == dd.DD_NORM_RMS
    assert dd.make_config(workloads.model_cfg(2)).norm == dd.DD_NORM_LAYER
    with pytest.raises(ValueError):
        dd.make_config(dict(workloads.model_cfg(2), norm="group"))


def test_config_errors_keep_their_message():
    """A configuration refused by the shared check keeps the check's own message (it is not
    formatted into itself)."""
    L = dd.lib()
    bad = _cfg_struct(d_model=770)
    assert _fwd(bad) == 1
    assert L.dd_last_error() == b"d_model must be even and divisible by n_heads"
    bad = _cfg_struct(lora_rank=12)
    assert L.dd_init_params(ctypes.byref(bad), FAKE, 1 << 40, 0, None, None) == 1
    assert L.dd_last_error() == b"lora_rank must be a non-negative multiple of 8 (got 12)"
    bad = _cfg_struct(n_heads=24)
    assert _fwd(bad) == 6
    assert L.dd_last_error().startswith(b"head dim 32 unsupported")
    assert L.dd_param_bytes(ctypes.byref(_cfg_struct(mask_id=7))) == 0


def test_loop_validation():
    cfg = _cfg_struct()
    al = (ctypes.c_double * 3)(1.0, 0.5, 0.5)         # not strictly decreasing
    assert dd.lib().dd_sample_loop(ctypes.byref(cfg), FAKE, 1, 16, 2, al, FAKE, None, 0, None, FAKE,
                                   1 << 40, None) == 1
    al = (ctypes.c_double * 3)(1.0, 0.5, 0.0)
    assert dd.lib().dd_sample_loop(ctypes.byref(cfg), FAKE, 1, 16, 2, al, FAKE, None, 0, None, FAKE,
                                   10, None) == 4
    assert dd.lib().dd_sample_loop(ctypes.byref(cfg), FAKE, 1, 16, 0, al, FAKE, None, 0, None, FAKE,
                                   1 << 40, None) == 1
    # unknown loop flags
    psi = lambda c, flags, words=None: dd.lib().dd_psi_sample_loop(ctypes.byref(c), FAKE, 1, 16, 2, al, None, flags,
                                                                   FAKE, words, 0, None, FAKE, 1 << 40, None)
    assert psi(cfg, 4) == 1
    assert b"flags" in dd.lib().dd_last_error()
    # the store-free draw: not with the posterior pass, the uniform prior, fp32 or explicit noise
    assert psi(cfg, dd.DD_LOOP_STORE_FREE | dd.DD_LOOP_POSTERIOR_PASS) == 1
    assert psi(_cfg_struct(prior="uniform", mask_id=-1), dd.DD_LOOP_STORE_FREE) == 6
    assert dd.lib().dd_last_error().startswith(b"DD_LOOP_STORE_FREE needs the masked prior")
    assert psi(dd.make_config(workloads.model_cfg(1)), dd.DD_LOOP_STORE_FREE) == 6
    assert psi(cfg, dd.DD_LOOP_STORE_FREE, words=FAKE) == 6
    assert dd.lib().dd_last_error() == b"DD_LOOP_STORE_FREE draws Philox noise only"


def test_loop_workspace_layout():
    """The inspection regions lie inside the loop workspace, aligned and without overlap."""
    for c, B, L in ((1, 4, 32), (2, 2, 128), (3, 1, 64)):
        cfg = workloads.model_cfg(c)
        lay = dd.loop_workspace_layout(cfg, B, L)
        M, V = B * L, cfg["vocab"]
        es = 2 if cfg["dtype"] == "bf16" else 4
        regions = sorted([(lay["err"], 4), (lay["logits"], M * lay["logits_ld"] * es), (lay["rows"], 4 * M),
                          (lay["count"], 4), (lay["glse"], 4 * M * lay["glse_ld"]), (lay["row_lse"], 4 * M)])
        assert lay["logits_ld"] == dd.logits_ld(V) and lay["glse_ld"] >= (V + 255) // 256
        assert lay["logits"] >= dd.workspace_bytes(cfg, B, L)
        for (o1, n1), (o2, _) in zip(regions, regions[1:]):
            assert o1 % 256 == 0 and o1 + n1 <= o2
        assert regions[-1][0] + regions[-1][1] <= dd.loop_workspace_bytes(cfg, B, L)
        # the store-free candidates live in the logits region and fit there
        assert lay["cand"] == lay["logits"] and 4 * M * lay["glse_ld"] <= M * lay["logits_ld"] * es
    with pytest.raises(dd.DDError):
        dd.loop_workspace_layout(workloads.model_cfg(2), 0, 16)


def test_latent_and_init_validation():
    L = dd.lib()
    assert L.dd_gaussian_latent_argmax(FAKE, 4, 0, 0.0, 1.0, 0, 0, 0, FAKE, None, None) == 1
    assert L.dd_gaussian_latent_argmax(FAKE, 4, 8, 0.0, 0.0, 0, 0, 0, FAKE, None, None) == 1
    assert L.dd_gaussian_latent_argmax(None, 0, 8, 0.0, 1.0, 0, 0, 0, None, None, None) == 0
    cfg = _cfg_struct()
    assert L.dd_init_params(ctypes.byref(cfg), FAKE, 100, 0, None, None) == 4
    assert L.dd_init_params(ctypes.byref(cfg), None, 1 << 40, 0, None, None) == 1


def test_status_strings_and_last_error():
    L = dd.lib()
    assert L.dd_status_str(0) == b"ok" and L.dd_status_str(4) == b"buffer too small"
    _post(ld=31)
    assert b"ld" in L.dd_last_error()


def test_pack_params_rejects_non_bf16_values():
    cfg = workloads.model_cfg(1, dtype="bf16", n_layers=1)
    specs = oparams.specs(cfg)
    P = workloads.host_params(cfg, 3, specs)
    blob = dd.pack_params(cfg, [P[n] for n, _, _ in specs])
    assert blob.size == dd.param_bytes(cfg)
    bad = [P[n] for n, _, _ in specs]
    bad[0] = bad[0] + 1e-5
    with pytest.raises(ValueError):
        dd.pack_params(cfg, bad)


def test_psi_entry_points_validate_kappa():
    """kappa outside [0, 1] is rejected before anything reaches the GPU."""
    L = dd.lib()
    for kappa, status in ((-0.1, 1), (1.5, 1), (float("nan"), 1)):
        assert L.dd_psi_posterior_sample(0, FAKE, 0, 64, 4, 32, 32, FAKE, 0.2, 0.5, kappa, None, 0, 1, 0, FAKE,
                                         None, None, None, None) == status
    assert L.dd_psi_posterior_sample(0, None, 0, 64, 0, 32, 32, None, 0.2, 0.5, 0.5, None, 0, 1, 0, None,
                                     None, None, None, None) == 0      # zero rows: nothing to do
    cfg = _cfg_struct()
    al = (ctypes.c_double * 3)(1.0, 0.5, 0.0)
    bad = (ctypes.c_double * 3)(1.0, 0.5, 2.0)
    assert L.dd_psi_sample_loop(ctypes.byref(cfg), FAKE, 1, 16, 2, al, bad, 0, FAKE, None, 0, None, FAKE,
                                1 << 40, None) == 1


def test_spec_verify_validation_and_sizes():
    from oracle import verify as overify
    L = dd.lib()
    args = lambda **k: dict(dict(p=FAKE, q=FAKE, dt=0, ld=64, S=4, B=3, V=32, draft=FAKE, noise=None, seed=0,
                                 step=0, row0=0, n=FAKE, z=FAKE, ws=FAKE, wsb=1 << 20, err=None), **k)

    def call(**k):
        a = args(**k)
        return L.dd_spec_verify(a["p"], a["q"], a["dt"], a["ld"], a["S"], a["B"], a["V"], a["draft"], a["noise"],
                                a["seed"], a["step"], a["row0"], a["n"], a["z"], a["ws"], a["wsb"], a["err"], None)
    assert call(dt=7) == 3
    assert call(B=0) == 1
    assert call(ld=30) == 2 and call(ld=36) == 2
    assert call(wsb=8) == 4
    assert call(q=None) == 1                       # B > 1 needs draft logits
    assert call(S=0, p=None, n=None, z=None, ws=None) == 0
    assert dd.spec_verify_workspace_bytes(4, 3) == 256 and dd.spec_verify_workspace_bytes(100, 8) == 6144
    # the allocation-free form validates the same way and refuses more rows than its array holds
    nv = lambda **k: (lambda a: L.dd_spec_verify_noalloc(a["p"], a["q"], a["dt"], a["ld"], a["S"], a["B"], a["V"],
                                                         a["draft"], a["noise"], a["seed"], a["step"], a["row0"],
                                                         a["n"], a["z"], a["err"], None))(args(**k))
    assert nv(dt=7) == 3 and nv(B=0) == 1 and nv(ld=30) == 2 and nv(q=None) == 1
    assert nv(S=0, p=None, n=None, z=None) == 0
    assert nv(S=dd.SPEC_VERIFY_NOALLOC_ROWS // 5 + 1) == 4         # S (2B - 1) = 5 S rows
    assert b"exceed" in L.dd_last_error()
    for B, V in ((1, 32), (4, 300), (16, 50257)):
        assert dd.spec_verify_noise_width(B, V) == overify.noise_width(B, V)


@pytest.mark.parametrize("pattern,L,block", [("bidirectional", 7, 0), ("causal", 9, 0), ("block_causal", 10, 3),
                                             ("block_causal", 8, 8), ("draft_train", 12, 3),
                                             ("draft_train", 2, 1), ("draft_train", 16, 8)])
def test_attn_mask_build_matches_oracle_patterns(pattern, L, block):
    """The library's (pre, lo, hi) form, expanded, is the oracle's visibility matrix, bit for bit."""
    from oracle import masks
    m = dd.attn_mask_build(pattern, L, block)
    pre, lo, hi = m[0][:, None], m[1][:, None], m[2][:, None]
    j = np.arange(L)[None, :]
    vis = (j < pre) | ((j >= lo) & (j < hi))
    want = {"bidirectional": lambda: masks.bidirectional(L), "causal": lambda: masks.causal(L),
            "block_causal": lambda: masks.block_causal(L, block),
            "draft_train": lambda: masks.draft_training(L // 2 // block, block)}[pattern]()
    assert np.array_equal(vis, want)
    assert ((0 <= m[0]) & (m[0] <= L) & (0 <= m[1]) & (m[1] <= m[2]) & (m[2] <= L)).all()


def test_attn_mask_build_validation():
    L = dd.lib()
    out = (ctypes.c_int32 * 64)()
    assert L.dd_attn_mask_build(1, 8, 0, None) == 1
    assert L.dd_attn_mask_build(9, 8, 0, out) == 1
    assert L.dd_attn_mask_build(1, 0, 0, out) == 1
    assert L.dd_attn_mask_build(2, 8, 0, out) == 1
    assert L.dd_attn_mask_build(3, 9, 1, out) == 2      # L odd
    assert L.dd_attn_mask_build(3, 12, 4, out) == 2     # L/2 = 6 not a multiple of 4
    assert L.dd_attn_mask_build(3, 12, 3, out) == 0


def _lora_cfg(**over):
    return {**workloads.model_cfg(1, n_layers=2), "lora_rank": 16, "lora_alpha": 32.0, **over}


def test_lora_param_layout_matches_oracle_storage():
    cfg = _lora_cfg()
    specs = oparams.specs(cfg)
    assert dd.param_count(cfg) == len(specs) == 2 + 12 * 2 + 3 + 4 * 2
    es = 2 if cfg["dtype"] == "bf16" else 4
    end = 0
    for tid, (name, shape, _) in enumerate(specs):
        off, r, cc = dd.param_tensor(cfg, tid)
        assert (r, cc) == (tuple(shape) if len(shape) == 2 else (1, shape[0])), name
        assert off % 256 == 0 and off >= end
        end = off + int(np.prod(shape)) * es
    assert dd.param_bytes(cfg) >= end
    P = oparams.init_params(cfg, 4)
    blob = dd.pack_params(cfg, oparams.storage_tensors(cfg, P))
    assert blob.size == dd.param_bytes(cfg)


def test_lora_workspace_and_validation():
    base = workloads.model_cfg(1, n_layers=2)
    cfg = _lora_cfg()
    B, Lq = 2, 64
    d, F, r = cfg["d_model"], cfg["d_mlp"], cfg["lora_rank"]
    grow = dd.workspace_bytes(cfg, B, Lq) - dd.workspace_bytes(base, B, Lq)
    es = 2 if cfg["dtype"] == "bf16" else 4
    assert 3 * B * Lq * r * es <= grow <= 3 * B * Lq * r * es + 3 * 256
    L = dd.lib()
    for bad in (dict(lora_rank=12), dict(lora_rank=-8), dict(lora_alpha=0.0), dict(lora_alpha=float("inf"))):
        c = dd.make_config(_lora_cfg(**bad))
        assert L.dd_param_count(ctypes.byref(c)) == 0
        assert L.dd_denoise_forward_ex(ctypes.byref(c), FAKE, FAKE, 1, 8, 0.5, None, None, FAKE, 64, FAKE,
                                       1 << 30, None) == 1
    # a gate for a model without adapters is an argument error, found before any launch
    c = dd.make_config(base)
    assert L.dd_denoise_forward_ex(ctypes.byref(c), FAKE, FAKE, 1, 8, 0.5, None, FAKE, FAKE, 64, FAKE,
                                   1 << 30, None) == 1
    assert b"adapters" in L.dd_last_error()
    c = dd.make_config(cfg)
    assert L.dd_denoise_forward_ex(ctypes.byref(c), FAKE, FAKE, 1, 8, 0.5, None, FAKE, FAKE, 64, FAKE,
                                   16, None) == 4
