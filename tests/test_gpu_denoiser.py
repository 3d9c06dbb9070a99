"""GPU parity of the denoiser forward pass and the T-step loop, through the C ABI,
against the float64 oracle on the same seeded inputs."""
import numpy as np
import pytest

import workloads
from oracle import forward as oforward, latent as olatent, loop as oloop, params as oparams, \
    sampler as osampler, schedule as osched
from paper_2609_04010_amd import _lib as dd
from tests.gpu_util import compare_ids, dev_i32, dev_words, say, torch_or_skip

pytestmark = pytest.mark.gpu

LOGIT_TOL = {"bf16": 5e-2, "fp32": 1e-4}


def _params_host(torch, cfg, seed):
    """Host-generated parameters (workloads) uploaded through the host-blob path."""
    specs = oparams.specs(cfg)
    P = workloads.host_params(cfg, seed, specs)
    blob = dd.pack_params(cfg, [P[n] for n, _, _ in specs])
    buf = torch.zeros(blob.size, dtype=torch.uint8, device="cuda")
    dd.init_params(cfg, buf, host_blob=blob)
    return P, buf


def _params_seeded(torch, cfg, seed):
    """In-kernel initialisation on the GPU; the oracle regenerates the same values itself."""
    buf = torch.zeros(dd.param_bytes(cfg), dtype=torch.uint8, device="cuda")
    dd.init_params(cfg, buf, seed=seed)
    return oparams.init_params(cfg, seed), buf


def _forward_gpu(torch, cfg, buf, z, at):
    B, L = z.shape
    V = cfg["vocab"]
    ld = int(dd.logits_ld(V))
    tdt = torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32
    logits = torch.zeros((B * L, ld), dtype=tdt, device="cuda")
    ws = torch.zeros(dd.workspace_bytes(cfg, B, L), dtype=torch.uint8, device="cuda")
    dd.denoise_forward(cfg, buf, dev_i32(torch, z), B, L, at, logits, ld, ws)
    err = dd.read_device_error(ws[:4].view(torch.int32))
    assert err == 0
    return logits[:, :V].float().cpu().numpy().astype(np.float64).reshape(B, L, V)


FWD_CASES = [
    # workload, overrides, B, L, alpha_t, mask fraction, params source
    (1, {}, 4, 32, 0.0, 1.0, "seeded"),
    (1, {}, 4, 32, 0.625, 0.375, "seeded"),
    (1, {}, 3, 29, 0.9, 0.1, "host"),
    (2, {}, 2, 200, 0.5, 0.5, "host"),
    (2, {}, 1, 1024, 0.25, 0.75, "host"),
    (3, {}, 2, 130, 0.4, 0.0, "host"),
    (5, {"max_len": 4096}, 1, 300, 0.7, 0.3, "host"),
    # RMSNorm: fp32 (row-per-wavefront kernels), bf16 at d 64 (the same kernels in bf16) and bf16
    # at d 768 / 1024 (the four-features-per-lane kernels)
    (1, {"norm": "rms"}, 4, 32, 0.625, 0.375, "seeded"),
    (1, {"norm": "rms", "dtype": "bf16", "n_heads": 1, "max_len": 96}, 2, 70, 0.5, 0.5, "host"),
    (2, {"norm": "rms", "n_layers": 3}, 2, 200, 0.5, 0.5, "host"),
    (5, {"norm": "rms", "n_layers": 2, "max_len": 4096}, 1, 300, 0.7, 0.3, "host"),
    # the residual projections' operand ring over two tiles per workgroup (33 x 990 rows: 512 tiles
    # of 256 x 192 for 256 CUs, the last M-tile ragged) and with two K-tiles (d_mlp 128)
    (2, {"n_layers": 1, "d_mlp": 128, "vocab": 300}, 33, 990, 0.5, 0.5, "host"),
]


def _fwd_id(c):
    return f"w{c[0]}-B{c[2]}-L{c[3]}-a{c[4]}" + ("-" + "-".join(f"{k}{v}" for k, v in c[1].items()) if c[1] else "")


@pytest.mark.parametrize("case", FWD_CASES, ids=_fwd_id)
def test_denoise_forward_parity(case):
    torch = torch_or_skip()
    c, over, B, L, at, mf, src = case
    say("forward", case)
    cfg = workloads.model_cfg(c, **over)
    seed = workloads.seeds(c)["param"]
    P, buf = (_params_seeded if src == "seeded" else _params_host)(torch, cfg, seed)
    V = cfg["vocab"]
    if cfg["prior"] == "mask":
        z = workloads.masked_state(workloads.seeds(c)["data"], B, L, V, mf)
    else:
        z = workloads.uniform_state(workloads.seeds(c)["data"], B, L, V)
    got = _forward_gpu(torch, cfg, buf, z, at)
    ref = oforward.forward(cfg, P, z, at)
    err = float(np.abs(got - ref).max())
    say(f"max |dlogit| = {err:.3e} (logit std {ref.std():.3f})")
    assert err <= LOGIT_TOL[cfg["dtype"]]


def _far_first_tile_params(cfg, seed, f1=3, f2=17, c=72.0):
    """Host parameters of a one-head model in which every query scores keys 0..63 far below the
    others.  Features f1 and f2 (< d / 2, where the time embedding at alpha_t = 1 is 0) are equal in
    every token embedding, in the LayerNorm gain and bias, and in the position embedding past 63,
    so after LN1 they are equal there; positions 0..63 put +64 and -64 on them.  Key component 0 is
    x[f2] - x[f1] (zero past 63, about -11.3 before) and query component 0 carries a bias c."""
    specs = oparams.specs(cfg)
    P = workloads.host_params(cfg, seed, specs)
    P["tok_emb"][:, f2] = P["tok_emb"][:, f1]
    P["l0.ln1_g"][f2] = P["l0.ln1_g"][f1]
    P["l0.ln1_b"][f2] = P["l0.ln1_b"][f1]
    pos = P["pos_emb"]
    pos[:, f2] = pos[:, f1]
    pos[:64, f1], pos[:64, f2] = 64.0, -64.0
    d = cfg["d_model"]
    wk = P["l0.w_qkv"][d]                 # key component 0
    wk[:] = 0.0
    wk[f1], wk[f2] = -1.0, 1.0
    P["l0.b_qkv"][d] = 0.0
    P["l0.b_qkv"][0] = c                  # query component 0
    return P, specs


@pytest.mark.parametrize("L", [200, 1024])
def test_attention_raises_its_reference_after_the_first_tile(L):
    """Keys 0..63 score about 150 (base 2) below the rest for every query, so the exponent reference
    set by the first key tile is exceeded by more than 2^64 in the second: the attention kernel takes
    its recompute-and-raise path there and the fast path afterwards.  The gap is past 128, so
    exponentials taken against the first tile's reference would overflow fp32.  The forward pass
    matches the oracle to the logit bar (L 200: ragged last tile)."""
    torch = torch_or_skip()
    cfg = workloads.model_cfg(2, n_layers=1, d_model=64, n_heads=1, d_mlp=256, vocab=1000)
    P, specs = _far_first_tile_params(cfg, seed=23)
    B, V = 2, cfg["vocab"]
    z = workloads.masked_state(5, B, L, V, 0.5)
    # the precondition, from the oracle's own pieces: scores (base 2) of keys past 63 exceed those
    # of keys 0..63 by more than 128 for every query
    h = P["tok_emb"][z] + P["pos_emb"][:L][None] + oforward.time_embedding(1.0, 64)[None, None]
    x = oforward.layer_norm(h, P["l0.ln1_g"], P["l0.ln1_b"], cfg["norm_eps"])
    qkv = x @ P["l0.w_qkv"].T + P["l0.b_qkv"]
    q, k = qkv[..., :64], qkv[..., 64:128]
    s2 = np.einsum("bid,bjd->bij", q, k) / 8.0 * np.log2(np.e)
    gap = s2[:, :, 64:128].max(axis=2) - s2[:, :, :64].max(axis=2)
    say(f"L {L}: smallest gap between the second and the first key tile {gap.min():.1f}")
    assert gap.min() > 128 + 5
    blob = dd.pack_params(cfg, [P[n] for n, _, _ in specs])
    buf = torch.zeros(blob.size, dtype=torch.uint8, device="cuda")
    dd.init_params(cfg, buf, host_blob=blob)
    got = _forward_gpu(torch, cfg, buf, z, 1.0)
    ref = oforward.forward(cfg, P, z, 1.0)
    err = float(np.abs(got - ref).max())
    say(f"max |dlogit| = {err:.3e} (logit std {ref.std():.3f})")
    assert err <= LOGIT_TOL["bf16"]


def test_forward_out_of_range_token_sets_error_word():
    torch = torch_or_skip()
    cfg = workloads.model_cfg(1)
    _, buf = _params_seeded(torch, cfg, 3)
    z = workloads.all_mask(1, 8, cfg["vocab"])
    z[0, 3] = 999
    ld = int(dd.logits_ld(cfg["vocab"]))
    logits = torch.zeros((8, ld), dtype=torch.float32, device="cuda")
    ws = torch.zeros(dd.workspace_bytes(cfg, 1, 8), dtype=torch.uint8, device="cuda")
    dd.denoise_forward(cfg, buf, dev_i32(torch, z), 1, 8, 0.5, logits, ld, ws)
    assert dd.read_device_error(ws[:4].view(torch.int32)) == dd.DD_DEVERR_TOKEN
    dd.workspace_reset(ws)
    assert dd.read_device_error(ws[:4].view(torch.int32)) == 0


def _loop_gpu(torch, cfg, buf, z1, T, alphas, words=None, seed=0, kappas=None, posterior_pass=False):
    B, L = z1.shape
    z = dev_i32(torch, z1)
    trace = torch.zeros(((T + 1) * B * L,), dtype=torch.int32, device="cuda")
    ws = torch.zeros(dd.loop_workspace_bytes(cfg, B, L), dtype=torch.uint8, device="cuda")
    dd.sample_loop(cfg, buf, B, L, T, alphas, z, ws,
                   noise_words=dev_words(torch, words) if words is not None else None,
                   noise_seed=seed, z_trace=trace, kappas=kappas, posterior_pass=posterior_pass)
    assert dd.read_device_error(ws[:4].view(torch.int32)) == 0
    return z.cpu().numpy().reshape(B, L), trace.cpu().numpy().reshape(T + 1, B, L)


@pytest.mark.parametrize("norm", ["layer", "rms"])
def test_loop_config1_free_running_matches_oracle(norm):
    """fp32 workload 1: the whole 8-step loop on explicit noise, free running on both sides (with
    LayerNorm, the workload's choice, and with RMSNorm)."""
    torch = torch_or_skip()
    cfg = workloads.model_cfg(1, norm=norm)
    w, s = workloads.WORKLOADS[1], workloads.seeds(1)
    B, L, V, T = w["B"], w["L"], w["vocab"], w["T"]
    P, buf = _params_seeded(torch, cfg, s["param"])
    words = workloads.noise_words(s["noise"], (T, B * L, osampler.noise_width("mask", V)))
    z1 = workloads.all_mask(B, L, V)
    al = osched.alphas(T)
    z0, trace = _loop_gpu(torch, cfg, buf, z1, T, al, words=words)
    rz0, rtrace, gaps = oloop.sample_loop(cfg, P, z1, T, al, noise_words=words)
    say(f"loop: min gap {np.min(gaps):.3e}; trace agreement {np.mean(trace == rtrace):.6f}")
    for k in range(T):
        compare_ids(trace[k + 1].reshape(-1), rtrace[k + 1].reshape(-1), gaps[k], f"step {T - k}")
    assert np.array_equal(z0, rz0)


@pytest.mark.parametrize("c,B,L,T", [(2, 2, 128, 8), (4, 2, 96, 8)])
def test_loop_bookkeeping_masked(c, B, L, T):
    torch = torch_or_skip()
    say("loop bookkeeping", c, B, L, T)
    cfg = workloads.model_cfg(c)
    V = cfg["vocab"]
    _, buf = _params_seeded(torch, cfg, workloads.seeds(c)["param"])
    z1 = workloads.all_mask(B, L, V)
    z0, trace = _loop_gpu(torch, cfg, buf, z1, T, osched.alphas(T), seed=workloads.seeds(c)["noise"])
    masked = (trace == V).sum(axis=(1, 2))
    say("masked per step", masked.tolist())
    assert masked[0] == B * L and masked[-1] == 0 and np.all(np.diff(masked) <= 0)
    for k in range(1, T + 1):
        was = trace[k - 1] != V
        assert np.array_equal(trace[k][was], trace[k - 1][was])
    assert np.all((z0 >= 0) & (z0 < V))
    z0b, _ = _loop_gpu(torch, cfg, buf, z1, T, osched.alphas(T), seed=workloads.seeds(c)["noise"])
    assert np.array_equal(z0, z0b)                                   # deterministic


@pytest.mark.parametrize("noise", ["words", "philox"])
def test_loop_uniform_reduced_config3_free_running_matches_oracle(noise):
    """The uniform-prior loop (App. A.2) from a Gaussian-latent start (App. A.5) in fp32 on a reduced
    workload-3 model (2 layers, d 64, V 1000 in four groups, the last one ragged): every step's
    state against the oracle's free-running loop on the same noise (explicit words or Philox), ids
    by the gap rule, and z_0 identical."""
    torch = torch_or_skip()
    cfg = workloads.model_cfg(3, dtype="fp32", n_layers=2, d_model=64, n_heads=2, d_mlp=256,
                              vocab=1000, max_len=64)
    s = workloads.seeds(3)
    B, L, V, T = 2, 48, cfg["vocab"], 6
    say("uniform loop, reduced workload 3", B, L, V, T, noise)
    P, buf = _params_seeded(torch, cfg, s["param"])
    x = workloads.clean_tokens(s["data"], B, L, V)
    z1d = torch.empty(B * L, dtype=torch.int32, device="cuda")
    dd.gaussian_latent_argmax(dev_i32(torch, x), B * L, V, 0.0, 1.0, seed=s["noise"], step=0, z_out=z1d)
    z1 = z1d.cpu().numpy().reshape(B, L)
    assert np.array_equal(z1.reshape(-1), olatent.latent_argmax(x.reshape(-1), V, 0.0, 1.0, s["noise"], 0))
    al = osched.alphas(T)
    if noise == "words":
        words = workloads.noise_words(s["noise"] + 2, (T, B * L, osampler.noise_width("uniform", V)))
        z0, trace = _loop_gpu(torch, cfg, buf, z1, T, al, words=words)
        rz0, rtrace, gaps = oloop.sample_loop(cfg, P, z1, T, al, noise_words=words)
    else:
        z0, trace = _loop_gpu(torch, cfg, buf, z1, T, al, seed=s["noise"])
        rz0, rtrace, gaps = oloop.sample_loop(cfg, P, z1, T, al, noise_seed=s["noise"])
    changed = float(np.mean(trace[-1] != trace[0]))
    say(f"uniform loop: min gap {np.min(gaps):.3e}; agreement {np.mean(trace == rtrace):.6f}; "
        f"changed since z_1 {changed:.3f}")
    for k in range(T):
        compare_ids(trace[k + 1].reshape(-1), rtrace[k + 1].reshape(-1), gaps[k], f"step {T - k}")
    assert np.array_equal(z0, rz0)
    assert changed > 0.5


def test_loop_uniform_prior_runs_in_range():
    torch = torch_or_skip()
    cfg = workloads.model_cfg(3)
    V = cfg["vocab"]
    B, L, T = 2, 64, 4
    _, buf = _params_seeded(torch, cfg, workloads.seeds(3)["param"])
    x = workloads.clean_tokens(workloads.seeds(3)["data"], B, L, V)
    z1d = torch.empty(B * L, dtype=torch.int32, device="cuda")
    dd.gaussian_latent_argmax(dev_i32(torch, x), B * L, V, 0.0, 1.0, seed=9, step=0, z_out=z1d)
    z1 = z1d.cpu().numpy().reshape(B, L)
    z0, trace = _loop_gpu(torch, cfg, buf, z1, T, osched.alphas(T), seed=5)
    assert np.all((trace >= 0) & (trace < V))
    assert np.mean(trace[-1] != trace[0]) > 0.5          # the uniform prior keeps revising tokens


@pytest.mark.parametrize("tile", ["0", "1", "2", "3", "4", "5", "6", "7", "8", "9", "10"])
def test_forward_parity_every_gemm_tile(tile, monkeypatch):
    """Each GEMM tile variant (64/128/256 rows x 32/128/192/256 columns, 1, 4 or 8 wavefronts) on
    ragged M and N."""
    torch = torch_or_skip()
    monkeypatch.setenv("DD_GEMM_TILE", tile)
    say("gemm tile", tile)
    cfg = workloads.model_cfg(2, n_layers=2)
    P, buf = _params_host(torch, cfg, 7)
    z = workloads.masked_state(8, 3, 190, cfg["vocab"], 0.5)
    got = _forward_gpu(torch, cfg, buf, z, 0.5)
    ref = oforward.forward(cfg, P, z, 0.5)
    err = float(np.abs(got - ref).max())
    say(f"tile {tile}: max |dlogit| = {err:.3e}")
    assert err <= LOGIT_TOL["bf16"]


def _mixed_start(B, L, V, seed):
    """Sequence 0 fully decoded (no listed row), sequence 1 masked at a random third of its
    positions, the others all masked."""
    rng = np.random.default_rng(seed)
    z1 = rng.integers(0, V, size=(B, L)).astype(np.int32)
    if B > 1:
        z1[1, rng.random(L) < 1 / 3] = V
    z1[2:] = V
    return z1


@pytest.mark.parametrize("c,over,B,L,T,start", [
    (2, dict(n_layers=2), 2, 300, 6, "all_mask"),
    (5, dict(n_layers=1), 1, 520, 4, "all_mask"),
    (2, dict(n_layers=1, vocab=1000), 3, 200, 4, "mixed"),   # a sequence with no listed row
    (2, dict(n_layers=1, vocab=1000), 3, 203, 4, "mixed"),   # sequence starts inside a 4-row group
    (2, dict(n_layers=1, vocab=300), 6, 3, 3, "mixed"),      # several starts in one 4-row group
])
def test_compacted_loop_equals_full_path_loop(c, over, B, L, T, start):
    """dd_sample_loop (vocabulary projection and draw on the still-masked rows only, and the last
    layer from its attention queries on as well) must give the same trajectory as
    dd_denoise_forward + dd_posterior_sample applied to every row.  (The loop's group
    log-sum-exps come from the projection's epilogue, the entry point's from its own pass:
    summation order only, which no draw at these seeds is close enough to feel.)"""
    torch = torch_or_skip()
    say("compacted loop", c, over, B, L, T, start)
    cfg = workloads.model_cfg(c, **over)
    V = cfg["vocab"]
    _, buf = _params_seeded(torch, cfg, 41)
    z1 = workloads.all_mask(B, L, V) if start == "all_mask" else _mixed_start(B, L, V, 7)
    al = osched.alphas(T)
    _, trace = _loop_gpu(torch, cfg, buf, z1, T, al, seed=77)
    M = B * L
    ld = int(dd.logits_ld(V))
    logits = torch.zeros((M, ld), dtype=torch.bfloat16, device="cuda")
    ws = torch.zeros(dd.workspace_bytes(cfg, B, L), dtype=torch.uint8, device="cuda")
    z = dev_i32(torch, z1)
    for k in range(T, 0, -1):
        dd.denoise_forward(cfg, buf, z, B, L, al[k], logits, ld, ws)
        dd.posterior_sample("mask", logits, "bf16", ld, M, V, z, al[k], al[k - 1], z, seed=77, step=k)
        got = z.cpu().numpy().reshape(B, L)
        assert np.array_equal(got, trace[T - k + 1]), f"step {k}"
    say("masked per step", [(t == V).sum() for t in trace])


@pytest.mark.parametrize("c,over,B,L,T", [
    (2, dict(n_layers=2), 2, 300, 6),                 # 197 groups, the last one 81 classes wide
    (2, dict(n_layers=1, vocab=1000), 3, 200, 6),     # 4 groups, the last one 232 wide
    (2, dict(n_layers=1, vocab=300), 2, 256, 5),      # 2 groups, the last one 44 wide
    (2, dict(n_layers=1, vocab=512), 2, 128, 4),      # 2 whole groups, no ragged one
    (2, dict(n_layers=1, vocab=100), 2, 128, 4),      # a single group narrower than the tile
    (3, dict(n_layers=2), 2, 300, 4),                 # uniform prior: every row, no compaction
])
def test_loop_group_lse_epilogue_equals_posterior_pass(c, over, B, L, T):
    """The loop draws from the per-group log-sum-exps that the vocabulary projection's epilogue
    computes from the logits it stores; the same loop with DD_LOOP_POSTERIOR_PASS draws from the
    posterior kernel's own pass over those logits (the path the posterior parity tests cover).  The
    two differ only in the summation order inside each group's log-sum-exp, which can decide a draw
    only when two level-1 scores are within a few ulps; with these seeds the trajectories agree."""
    torch = torch_or_skip()
    say("group lse loop", c, over, B, L, T)
    cfg = workloads.model_cfg(c, **over)
    V = cfg["vocab"]
    _, buf = _params_seeded(torch, cfg, 45)
    if cfg["prior"] == "mask":
        z1 = workloads.all_mask(B, L, V)
    else:
        z1 = np.random.default_rng(6).integers(0, V, size=(B, L)).astype(np.int32)
    al = osched.alphas(T)
    _, fused = _loop_gpu(torch, cfg, buf, z1, T, al, seed=91)
    _, passed = _loop_gpu(torch, cfg, buf, z1, T, al, seed=91, posterior_pass=True)
    last = (V - 1) // 256 * 256
    drawn_last = int(sum(((t >= last) & (t < V)).sum() for t in fused[1:]))
    say(f"agreement {np.mean(fused == passed):.6f}; draws in the last (ragged) group {drawn_last}")
    for k in range(1, T + 1):
        assert np.array_equal(fused[k], passed[k]), f"step {T - k + 1}"
    assert np.mean(fused[-1] != fused[0]) > 0.3       # the loop did draw


def test_loop_from_a_decoded_state_leaves_it_unchanged():
    """Masked prior, no mask token in z_1: every step's compacted list is empty, so the gathered
    vocabulary projection and the grouped draw launch with no rows, and z stays as it was."""
    torch = torch_or_skip()
    cfg = workloads.model_cfg(2, n_layers=1)
    V = cfg["vocab"]
    B, L, T = 2, 128, 4
    say("loop from a decoded state", B, L, T)
    _, buf = _params_seeded(torch, cfg, 49)
    z1 = np.random.default_rng(8).integers(0, V, size=(B, L)).astype(np.int32)
    z0, trace = _loop_gpu(torch, cfg, buf, z1, T, osched.alphas(T), seed=95)
    assert np.array_equal(z0, z1)
    assert all(np.array_equal(t, z1) for t in trace)


def test_bf16_loop_without_compaction_equals_full_path():
    """bf16 with d_model % 128 != 0 (d = 64): no row compaction and no group log-sum-exp epilogue, so
    the loop runs the vocabulary projection on every row and the posterior's own pass; it must give
    exactly the trajectory of dd_denoise_forward + dd_posterior_sample on every row."""
    torch = torch_or_skip()
    cfg = workloads.model_cfg(2, n_layers=2, d_model=64, n_heads=1, d_mlp=256, vocab=1000)
    V = cfg["vocab"]
    B, L, T = 2, 100, 5
    say("bf16 loop without compaction", B, L, T)
    _, buf = _params_seeded(torch, cfg, 47)
    z1 = workloads.all_mask(B, L, V)
    al = osched.alphas(T)
    _, trace = _loop_gpu(torch, cfg, buf, z1, T, al, seed=93)
    M = B * L
    ld = int(dd.logits_ld(V))
    logits = torch.zeros((M, ld), dtype=torch.bfloat16, device="cuda")
    ws = torch.zeros(dd.workspace_bytes(cfg, B, L), dtype=torch.uint8, device="cuda")
    z = dev_i32(torch, z1)
    for k in range(T, 0, -1):
        dd.denoise_forward(cfg, buf, z, B, L, al[k], logits, ld, ws)
        dd.posterior_sample("mask", logits, "bf16", ld, M, V, z, al[k], al[k - 1], z, seed=93, step=k)
        assert np.array_equal(z.cpu().numpy().reshape(B, L), trace[T - k + 1]), f"step {k}"
    assert (trace[-1] != V).all() and (np.diff([(t == V).sum() for t in trace]) <= 0).all()


# ---------------------------------------------------------------- Psi sampler loop (kappa < 1)

def test_psi_loop_config1_free_running_matches_oracle():
    """fp32 workload 1 with kappa = 0.5 at every step (App. A.4): decoded tokens can be remasked;
    the whole loop on explicit noise, free running on both sides."""
    torch = torch_or_skip()
    cfg = workloads.model_cfg(1)
    w, s = workloads.WORKLOADS[1], workloads.seeds(1)
    B, L, V, T = w["B"], w["L"], w["vocab"], w["T"]
    P, buf = _params_seeded(torch, cfg, s["param"])
    words = workloads.noise_words(s["noise"] + 1, (T, B * L, osampler.noise_width("mask", V)))
    z1 = workloads.all_mask(B, L, V)
    al = osched.alphas(T)
    kap = np.full(T + 1, 0.5)
    z0, trace = _loop_gpu(torch, cfg, buf, z1, T, al, words=words, kappas=kap)
    rz0, rtrace, gaps = oloop.sample_loop(cfg, P, z1, T, al, noise_words=words, kappas=kap)
    remasked = sum(int(((a != V) & (b == V)).sum()) for a, b in zip(trace[:-1], trace[1:]))
    say(f"psi loop: min gap {np.min(gaps):.3e}; remasked {remasked}; agreement {np.mean(trace == rtrace):.6f}")
    for k in range(T):
        compare_ids(trace[k + 1].reshape(-1), rtrace[k + 1].reshape(-1), gaps[k], f"step {T - k}")
    assert np.array_equal(z0, rz0)
    assert remasked > 0 and (z0 != V).all()


@pytest.mark.parametrize("kappa", [0.0, 0.4])
def test_psi_compacted_loop_equals_full_path_loop(kappa):
    """dd_psi_sample_loop (keep/remask of decoded rows, then the vocabulary projection and draw on
    the still-masked rows) must give the same trajectory as dd_denoise_forward +
    dd_psi_posterior_sample on every row."""
    torch = torch_or_skip()
    say("psi compacted loop", kappa)
    cfg = workloads.model_cfg(2, n_layers=2)
    V = cfg["vocab"]
    B, L, T = 2, 300, 6
    _, buf = _params_seeded(torch, cfg, 43)
    z1 = workloads.all_mask(B, L, V)
    al = osched.alphas(T)
    kap = np.full(T + 1, kappa)
    _, trace = _loop_gpu(torch, cfg, buf, z1, T, al, seed=78, kappas=kap)
    M = B * L
    ld = int(dd.logits_ld(V))
    logits = torch.zeros((M, ld), dtype=torch.bfloat16, device="cuda")
    ws = torch.zeros(dd.workspace_bytes(cfg, B, L), dtype=torch.uint8, device="cuda")
    z = dev_i32(torch, z1)
    for k in range(T, 0, -1):
        dd.denoise_forward(cfg, buf, z, B, L, al[k], logits, ld, ws)
        dd.psi_posterior_sample("mask", logits, "bf16", ld, M, V, z, al[k], al[k - 1], kappa, z, seed=78, step=k)
        got = z.cpu().numpy().reshape(B, L)
        assert np.array_equal(got, trace[T - k + 1]), f"step {k}"
    remasked = sum(int(((a != V) & (b == V)).sum()) for a, b in zip(trace[:-1], trace[1:]))
    say("masked per step", [(t == V).sum() for t in trace], "remasked", remasked)
    assert remasked > 0 and (trace[-1] != V).all()
