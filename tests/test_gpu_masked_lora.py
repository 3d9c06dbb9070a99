"""GPU parity of the denoiser under attention patterns and with gated LoRA adapters, through
dd_denoise_forward_ex, against the float64 oracle on the same seeded inputs.

Patterns: causal (AR pathway, drafting pass), block-causal, the [x, z_1] block-diffusion pattern;
lengths that span several 128-query workgroups and 64-key tiles with a ragged tail, block sizes
aligned and not aligned to the tiles.  Adapters: the paper's rank 128 / alpha 256 on the bf16
GPT-2-small shape, a rank whose K = in + r misses the 128 multiple (fallback GEMM), the fp32 build,
mixed per-position gates, and the teacher property of the [x, z_1] pass.
"""
import numpy as np
import pytest

import workloads
from oracle import forward as oforward, masks as omasks, params as oparams
from paper_2609_04010_amd import _lib as dd
from tests.gpu_util import dev_i32, say, torch_or_skip

pytestmark = pytest.mark.gpu

LOGIT_TOL = {"bf16": 5e-2, "fp32": 1e-4}


def _vis(pattern, L, block):
    return {"bidirectional": lambda: omasks.bidirectional(L), "causal": lambda: omasks.causal(L),
            "block_causal": lambda: omasks.block_causal(L, block),
            "draft_train": lambda: omasks.draft_training(L // 2 // block, block)}[pattern]()


def _params(torch, cfg, seed, src):
    if src == "seeded":
        buf = torch.zeros(dd.param_bytes(cfg), dtype=torch.uint8, device="cuda")
        dd.init_params(cfg, buf, seed=seed)
        return oparams.init_params(cfg, seed), buf
    P = oparams.split_storage(cfg, workloads.host_params(cfg, seed, oparams.specs(cfg)))
    blob = dd.pack_params(cfg, oparams.storage_tensors(cfg, P))
    buf = torch.zeros(blob.size, dtype=torch.uint8, device="cuda")
    dd.init_params(cfg, buf, host_blob=blob)
    return P, buf


def _forward_ex(torch, cfg, buf, z, at, mask=None, gate=None):
    B, L = z.shape
    V = cfg["vocab"]
    ld = int(dd.logits_ld(V))
    tdt = torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32
    logits = torch.zeros((B * L, ld), dtype=tdt, device="cuda")
    ws = torch.zeros(dd.workspace_bytes(cfg, B, L), dtype=torch.uint8, device="cuda")
    dmask = dev_i32(torch, np.asarray(mask).reshape(-1)) if mask is not None else None
    dgate = dev_i32(torch, gate) if gate is not None else None
    dd.denoise_forward_ex(cfg, buf, dev_i32(torch, z), B, L, at, logits, ld, ws, attn_mask=dmask, lora_gate=dgate)
    err = dd.read_device_error(ws[:4].view(torch.int32))
    return logits[:, :V].float().cpu().numpy().astype(np.float64).reshape(B, L, V), err


def _tokens(cfg, c, B, L, mf=0.5):
    V = cfg["vocab"]
    if cfg["prior"] == "mask":
        return workloads.masked_state(workloads.seeds(c)["data"], B, L, V, mf)
    return workloads.uniform_state(workloads.seeds(c)["data"], B, L, V)


MASK_CASES = [
    # workload, overrides, B, L, pattern, block, alpha_t
    (1, {}, 3, 32, "causal", 0, 0.5),
    (1, {"max_len": 64}, 2, 60, "draft_train", 5, 0.3),
    (2, {"n_layers": 2}, 2, 300, "causal", 0, 0.5),
    (2, {"n_layers": 2}, 2, 300, "block_causal", 100, 0.4),
    (2, {"n_layers": 2}, 2, 256, "block_causal", 64, 0.6),
    (2, {"n_layers": 2}, 2, 320, "draft_train", 16, 1.0),
    (2, {"n_layers": 2}, 1, 264, "draft_train", 33, 0.8),
    (2, {"n_layers": 2}, 2, 200, "bidirectional", 0, 0.5),
]


@pytest.mark.parametrize("case", MASK_CASES, ids=lambda c: f"w{c[0]}-L{c[3]}-{c[4]}{c[5] or ''}")
def test_masked_forward_parity(case):
    torch = torch_or_skip()
    c, over, B, L, pattern, block, at = case
    say("masked forward", case)
    cfg = workloads.model_cfg(c, **over)
    P, buf = _params(torch, cfg, workloads.seeds(c)["param"], "seeded" if c == 1 else "host")
    z = _tokens(cfg, c, B, L)
    mask = dd.attn_mask_build(pattern, L, block)
    got, err = _forward_ex(torch, cfg, buf, z, at, mask)
    assert err == 0
    ref = oforward.forward(cfg, P, z, at, _vis(pattern, L, block))
    e = float(np.abs(got - ref).max())
    say(f"max |dlogit| = {e:.3e} (logit std {ref.std():.3f})")
    assert e <= LOGIT_TOL[cfg["dtype"]]


def test_full_pattern_equals_unmasked_kernel():
    """The pattern kernel with every key visible reproduces the unmasked kernel."""
    torch = torch_or_skip()
    cfg = workloads.model_cfg(2, n_layers=2)
    P, buf = _params(torch, cfg, 5, "host")
    z = _tokens(cfg, 2, 2, 200)
    a, _ = _forward_ex(torch, cfg, buf, z, 0.5)
    b, err = _forward_ex(torch, cfg, buf, z, 0.5, dd.attn_mask_build("bidirectional", 200))
    d = float(np.abs(a - b).max())
    say(f"full pattern vs unmasked: max diff {d:.3e}, identical {np.array_equal(a, b)}")
    assert err == 0 and d <= 1e-3


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_invalid_pattern_entry_is_reported_and_sees_every_key(dtype):
    torch = torch_or_skip()
    over = {"n_layers": 2} if dtype == "bf16" else {}
    c = 2 if dtype == "bf16" else 1
    cfg = workloads.model_cfg(c, **over)
    P, buf = _params(torch, cfg, 7, "host" if dtype == "bf16" else "seeded")
    L = 96 if dtype == "bf16" else 32
    z = _tokens(cfg, c, 1, L)
    mask = dd.attn_mask_build("causal", L)
    mask[0, 5] = L + 3                    # pre > L
    mask[1, 9], mask[2, 9] = 4, 2         # lo > hi
    got, err = _forward_ex(torch, cfg, buf, z, 0.5, mask)
    assert err == dd.DD_DEVERR_MASK
    vis = omasks.causal(L)
    vis[5, :] = True
    vis[9, :] = True
    ref = oforward.forward(cfg, P, z, 0.5, vis)
    e = float(np.abs(got - ref).max())
    say(f"invalid entries: max |dlogit| = {e:.3e}")
    assert e <= LOGIT_TOL[dtype]


# ---------------------------------------------------------------- gated adapters

LORA_CASES = [
    # workload, overrides (rank, alpha, ...), B, L, pattern, block, gate kind, params source
    (1, {"lora_rank": 8, "lora_alpha": 16.0}, 4, 32, "causal", 0, "mixed", "seeded"),
    (1, {"lora_rank": 16, "lora_alpha": 32.0}, 2, 32, None, 0, None, "seeded"),
    (2, {"n_layers": 2, "lora_rank": 128, "lora_alpha": 256.0}, 2, 192, "draft_train", 8, "noisy", "seeded"),
    (2, {"n_layers": 2, "lora_rank": 128, "lora_alpha": 256.0}, 2, 300, None, 0, None, "host"),
    (2, {"n_layers": 2, "lora_rank": 16, "lora_alpha": 64.0}, 2, 200, "causal", 0, "mixed", "host"),
]


def _gate(kind, L):
    if kind is None:
        return None
    if kind == "noisy":              # adapters on the second half ([x, z_1]: z_1 only)
        return (np.arange(L) >= L // 2).astype(np.int32)
    return (np.arange(L) % 3 != 1).astype(np.int32)


@pytest.mark.parametrize("case", LORA_CASES, ids=lambda c: f"w{c[0]}-r{c[1]['lora_rank']}-L{c[3]}-{c[4]}-{c[6]}")
def test_gated_lora_forward_parity(case):
    torch = torch_or_skip()
    c, over, B, L, pattern, block, gk, src = case
    say("gated lora forward", case)
    cfg = workloads.model_cfg(c, **over)
    P, buf = _params(torch, cfg, workloads.seeds(c)["param"] + 17, src)
    z = _tokens(cfg, c, B, L)
    mask = dd.attn_mask_build(pattern, L, block) if pattern else None
    gate = _gate(gk, L)
    got, err = _forward_ex(torch, cfg, buf, z, 0.5, mask, gate)
    assert err == 0
    ref = oforward.forward(cfg, P, z, 0.5, _vis(pattern, L, block) if pattern else None,
                           None if gate is None else gate.astype(np.float64))
    base_cfg = dict(cfg, lora_rank=0)
    base = oforward.forward(base_cfg, {k: v for k, v in P.items() if "lora_" not in k}, z, 0.5,
                            _vis(pattern, L, block) if pattern else None)
    e = float(np.abs(got - ref).max())
    say(f"max |dlogit| = {e:.3e}; adapter effect max {np.abs(ref - base).max():.3e} (logit std {ref.std():.3f})")
    assert np.abs(ref - base).max() > 5 * LOGIT_TOL[cfg["dtype"]]   # the adapters matter here
    assert e <= LOGIT_TOL[cfg["dtype"]]


def _bf16_ulp(v):
    """Spacing of bf16 values at |v| (8 significant bits)."""
    e = np.floor(np.log2(np.maximum(np.abs(v), 2.0 ** -126)))
    return 2.0 ** (e - 7)


@pytest.mark.parametrize("tile", [None, "0"])
def test_teacher_logits_in_one_pass_match_base_model_on_gpu(tile, monkeypatch):
    """Sec. 3.2 on the GPU: [x, z_1] with adapters on z_1 only gives, at x, the base model's causal
    logits of x alone (run by the same library on a base-layout copy of the weights).

    Every layer computes the x rows identically in the two calls: the adapter columns of those rows
    are exact zeros (gate off), the K loops of the body GEMMs run in the same order wherever a row
    sits, and each 32-query wavefront of the attention holds the same x queries and visits the same
    key tiles (keys a query cannot see contribute exact zeros in both).  The one difference is the
    vocabulary projection, which starts the K loop of M-tile tm, N-tile tn at K-slice
    ((tm mod 8) + 2 tn) mod nk to spread L2 requests: sequence 1's x rows sit in M-tiles 0 and 1 of
    the [x, z_1] call but all in M-tile 0 of the call on x alone, so their fp32 sums are taken in
    another order and a logit can round to the neighbouring bf16 value.  Hence: at most one bf16
    ulp of the logit with the default tiles (2^-6 = 1.6e-2 for |logit| in [2, 4)), and bit-identical
    logits with the register-staged 128 x 128 tile (DD_GEMM_TILE=0), whose K loop always starts at
    slice 0."""
    torch = torch_or_skip()
    if tile is None:
        monkeypatch.delenv("DD_GEMM_TILE", raising=False)
    else:
        monkeypatch.setenv("DD_GEMM_TILE", tile)
    over = {"n_layers": 2, "lora_rank": 128, "lora_alpha": 256.0}
    cfg = workloads.model_cfg(2, **over)
    P, buf = _params(torch, cfg, 31, "host")
    n, bs = 96, 8
    x = workloads.clean_tokens(41, 2, n, cfg["vocab"])
    seq = np.concatenate([x, np.full((2, n), cfg["vocab"])], axis=1)
    gate = (np.arange(2 * n) >= n).astype(np.int32)
    got, err = _forward_ex(torch, cfg, buf, seq, 1.0, dd.attn_mask_build("draft_train", 2 * n, bs), gate)
    assert err == 0
    base_cfg = dict(cfg, lora_rank=0)
    Pb = {k: v for k, v in P.items() if "lora_" not in k}
    blob = dd.pack_params(base_cfg, oparams.storage_tensors(base_cfg, Pb))
    bbuf = torch.zeros(blob.size, dtype=torch.uint8, device="cuda")
    dd.init_params(base_cfg, bbuf, host_blob=blob)
    teach, err2 = _forward_ex(torch, base_cfg, bbuf, x, 1.0, dd.attn_mask_build("causal", n))
    assert err2 == 0
    diff = np.abs(got[:, :n] - teach)
    nd = int((diff > 0).sum())
    rows = np.nonzero(diff.max(axis=2) > 0)
    say(f"tile {tile}: teacher logits max diff {diff.max():.3e}, {nd} of {diff.size} differ, in rows "
        f"{sorted(set(zip(rows[0].tolist(), rows[1].tolist())))[:3]} .. (sequence, position)")
    if tile is None:
        # rows whose vocabulary M-tile is the same in both calls: sequence 0, and positions 0..63 of
        # sequence 1 (rows 192..255 of the [x, z_1] call, 96..159 of the call on x alone)
        assert (diff[0] == 0).all() and (diff[1, :64] == 0).all()
        # positions 64..95 of sequence 1 (rows 256..287: M-tile 1, against M-tile 0): the same fp32
        # products summed in another order, rounded to bf16.  Bound: one bf16 ulp of the larger value
        # plus the fp32 summation error of a 768-term dot product (about 1e-6 here; it dominates only
        # for logits near zero, where the terms cancel)
        ulp = np.maximum(_bf16_ulp(teach[1, 64:]), _bf16_ulp(got[1, 64:n]))
        assert np.all(diff[1, 64:] <= ulp + 4e-6)
    else:
        assert nd == 0


def test_sample_loop_with_adapters_matches_oracle():
    """The T-step loop on a model with adapters (all gates on), fp32 workload 1, explicit noise,
    free running on both sides."""
    from oracle import loop as oloop, sampler as osampler, schedule as osched
    from tests.gpu_util import compare_ids, dev_words
    torch = torch_or_skip()
    cfg = workloads.model_cfg(1, lora_rank=8, lora_alpha=16.0)
    w, s = workloads.WORKLOADS[1], workloads.seeds(1)
    B, L, V, T = w["B"], w["L"], w["vocab"], w["T"]
    P, buf = _params(torch, cfg, s["param"], "seeded")
    words = workloads.noise_words(s["noise"], (T, B * L, osampler.noise_width("mask", V)))
    z1 = workloads.all_mask(B, L, V)
    al = osched.alphas(T)
    z = dev_i32(torch, z1)
    trace = torch.zeros(((T + 1) * B * L,), dtype=torch.int32, device="cuda")
    ws = torch.zeros(dd.loop_workspace_bytes(cfg, B, L), dtype=torch.uint8, device="cuda")
    dd.sample_loop(cfg, buf, B, L, T, al, z, ws, noise_words=dev_words(torch, words), z_trace=trace)
    assert dd.read_device_error(ws[:4].view(torch.int32)) == 0
    trace = trace.cpu().numpy().reshape(T + 1, B, L)
    _, rtrace, gaps = oloop.sample_loop(cfg, P, z1, T, al, noise_words=words)
    say(f"adapter loop: trace agreement {np.mean(trace == rtrace):.6f}")
    for k in range(T):
        compare_ids(trace[k + 1].reshape(-1), rtrace[k + 1].reshape(-1), gaps[k], f"step {T - k}")


@pytest.mark.parametrize("c", [1, 2])
def test_forward_ex_without_pattern_or_gate_equals_forward(c):
    """dd_denoise_forward_ex(NULL, NULL) is dd_denoise_forward, bit for bit, with and without adapters."""
    torch = torch_or_skip()
    over = {"n_layers": 2} if c == 2 else {}
    for extra in ({}, {"lora_rank": 16, "lora_alpha": 32.0}):
        cfg = workloads.model_cfg(c, **over, **extra)
        _, buf = _params(torch, cfg, 3, "seeded")
        B, L = 2, (32 if c == 1 else 64)
        z = _tokens(cfg, c, B, L)
        V = cfg["vocab"]
        ld = int(dd.logits_ld(V))
        tdt = torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32
        outs = []
        for ex in (False, True):
            logits = torch.zeros((B * L, ld), dtype=tdt, device="cuda")
            ws = torch.zeros(dd.workspace_bytes(cfg, B, L), dtype=torch.uint8, device="cuda")
            if ex:
                dd.denoise_forward_ex(cfg, buf, dev_i32(torch, z), B, L, 0.5, logits, ld, ws)
            else:
                dd.denoise_forward(cfg, buf, dev_i32(torch, z), B, L, 0.5, logits, ld, ws)
            outs.append(logits.float().cpu().numpy())
        say(f"workload {c} {extra}: identical {np.array_equal(outs[0], outs[1])}")
        assert np.array_equal(outs[0], outs[1])
