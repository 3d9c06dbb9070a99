"""The launch profiler (dd_profile_*): every kernel of a forward pass is recorded once, in its
class, with a positive duration taken from the dispatch itself, and the recorded kernels fit in
the wall time of the calls; a class mask records that class only; the trace copy of the loop
(a memory copy, not a kernel) is recorded around the copy."""
import time

import numpy as np
import pytest

import workloads
from paper_2609_04010_amd import _lib as dd
from tests.gpu_util import say, torch_or_skip

pytestmark = pytest.mark.gpu


def _setup(torch, n_layers=2, B=2, L=256):
    cfg = workloads.model_cfg(2, n_layers=n_layers)
    params = torch.zeros(dd.param_bytes(cfg), dtype=torch.uint8, device="cuda")
    dd.init_params(cfg, params, seed=3)
    V = cfg["vocab"]
    ld = int(dd.logits_ld(V))
    logits = torch.empty((B * L, ld), dtype=torch.bfloat16, device="cuda")
    ws = torch.zeros(dd.workspace_bytes(cfg, B, L), dtype=torch.uint8, device="cuda")
    z = torch.from_numpy(workloads.masked_state(5, B, L, V, 0.5).reshape(-1)).cuda()
    run = lambda: dd.denoise_forward(cfg, params, z, B, L, 0.5, logits, ld, ws)
    return cfg, run


def test_profiler_records_each_kernel_of_a_forward_once():
    torch = torch_or_skip()
    cfg, run = _setup(torch)
    nl = cfg["n_layers"]
    run()
    torch.cuda.synchronize()
    reps = 3
    dd.profile_begin(reps * (8 * nl + 8))
    t0 = time.perf_counter()
    for _ in range(reps):
        run()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3
    dd.profile_end()
    prof = dd.profile_read()
    say("profile", {k: (n, round(ms, 4)) for k, (n, ms) in prof.items()}, "wall ms", round(wall, 3))
    want = {"time_embedding": 1, "embed_layernorm": 1, "gemm_qkv": nl, "attention": nl,
            "gemm_attn_out": nl, "gemm_mlp_up": nl, "gemm_mlp_down": nl, "layernorm": 2 * nl,
            "gemm_vocab": 1}
    for k, n in want.items():
        assert prof[k][0] == reps * n, (k, prof[k])
        assert prof[k][1] > 0.0
    assert sum(ms for _, ms in prof.values()) <= wall
    # a class mask: that class only
    dd.profile_begin(64, classes=["attention"])
    run()
    torch.cuda.synchronize()
    dd.profile_end()
    prof = dd.profile_read()
    assert prof["attention"][0] == nl and all(n == 0 for k, (n, _) in prof.items() if k != "attention")


def test_profiler_records_the_loop_trace_copies():
    torch = torch_or_skip()
    cfg = workloads.model_cfg(2, n_layers=1)
    V = cfg["vocab"]
    B, L, T = 1, 128, 3
    params = torch.zeros(dd.param_bytes(cfg), dtype=torch.uint8, device="cuda")
    dd.init_params(cfg, params, seed=3)
    ws = torch.zeros(dd.loop_workspace_bytes(cfg, B, L), dtype=torch.uint8, device="cuda")
    z = torch.full((B * L,), V, dtype=torch.int32, device="cuda")
    tr = torch.zeros(((T + 1) * B * L,), dtype=torch.int32, device="cuda")
    dd.profile_begin(T * 20 + 8)
    dd.sample_loop(cfg, params, B, L, T, 1.0 - np.arange(T + 1) / T, z, ws, noise_seed=1, z_trace=tr)
    torch.cuda.synchronize()
    dd.profile_end()
    prof = dd.profile_read()
    say("loop profile", {k: n for k, (n, _) in prof.items()})
    assert prof["copy"][0] == T + 1 and prof["copy"][1] > 0.0
    assert prof["posterior_sample"][0] == T and prof["gemm_vocab"][0] == T
