"""Stage-isolated parity at the launch shapes the benchmark times (every workload but the tiny one).

Each reverse step runs as a one-step dd_sample_loop on the whole batch (the same code as every
step of a T-step loop; its noise counters therefore carry step 1).  After the step the loop
workspace still holds what the step computed (dd_loop_workspace_layout): the vocabulary projection
of the rows the step drew, their per-group log-sum-exps and the row log-sum-exp the draw used.  One
sequence is then checked against the float64 oracle, one stage at a time:

  1. logits    the oracle's forward pass on the same state and the same (device-held) weights;
               max |dlogit| <= 5e-2 (bf16), over every drawn row of the sequence and all V columns;
  2. draw      the oracle's posterior and two-level Gumbel-max draw on the GPU's own logits (upcast
               exactly) with the same noise counters: ids equal wherever both of the oracle's
               top-two gaps exceed 1e-3, and on >= 99.9 % of rows;
  3. probs     the posterior the draw's fp32 row log-sum-exp implies, p(exp(l - row_lse)), against
               the oracle's on the same logits: max |dp| <= 1e-3; and the group masses
               exp(glse_g - row_lse) of the vocabulary epilogue against the oracle's group sums;
  4. carry     rows unmasked before the step keep their token (whole batch, bit for bit).

Stage 1 compares two forward passes; stages 2-3 never compare a GPU draw with an oracle draw made
from the oracle's own logits (their difference, up to the logit bar, is far above the 1e-3 gap).
Workload 4 checks sequence 127 of 128, whose logit rows start past 2^31 elements of the logit
matrix; workload 5 runs the 24-layer d 1024 model at L 4096 (its float64 forward pass takes about a
minute on the host, and prints its progress per layer).
"""
import time

import numpy as np
import pytest

import workloads
from oracle import forward as oforward, latent as olatent, params as oparams, posterior as oposterior, \
    sampler as osampler
from paper_2609_04010_amd import _lib as dd
from tests.gpu_util import PROB_TOL, compare_ids, dev_i32, say, torch_or_skip

# the float64 forward pass of the largest workload takes minutes on the host
pytestmark = [pytest.mark.gpu, pytest.mark.timeout(1200)]

LOGIT_TOL = 5e-2

# workload, the sequence checked, number of reverse steps, steps whose logits the oracle recomputes
FULL_CASES = [(2, 11, 2, 2), (3, 5, 2, 2), (4, 127, 2, 2), (5, 7, 2, 2)]


def _host_params(torch, cfg, seed):
    specs = oparams.specs(cfg)
    P = workloads.host_params(cfg, seed, specs)
    blob = dd.pack_params(cfg, [P[n] for n, _, _ in specs])
    buf = torch.zeros(blob.size, dtype=torch.uint8, device="cuda")
    dd.init_params(cfg, buf, host_blob=blob)
    return P, buf


def _ws_i32(torch, ws, off, n):
    return ws[off:off + 4 * n].view(torch.int32).cpu().numpy()


def _ws_f32(torch, ws, off, n, first=0):
    """fp32 elements first .. first + n of the array at byte offset off of the workspace."""
    a = off + 4 * first
    return ws[a:a + 4 * n].view(torch.float32).cpu().numpy()


def _ws_logits(torch, ws, lay, j0, j1, V):
    """Logits rows j0 .. j1 (bf16) of the loop workspace as float64 [j1 - j0, V]."""
    ld = lay["logits_ld"]
    a = lay["logits"] + 2 * j0 * ld
    t = ws[a:a + 2 * (j1 - j0) * ld].view(torch.bfloat16).view(j1 - j0, ld)[:, :V]
    return t.float().cpu().numpy().astype(np.float64)


def _group_lse(l, V):
    """float64 log-sum-exp of each group of 256 classes of every row of l."""
    ng = (V + 255) // 256
    out = np.empty((l.shape[0], ng))
    for g in range(ng):
        s = l[:, 256 * g:min(V, 256 * (g + 1))]
        m = s.max(axis=1, keepdims=True)
        out[:, g] = m[:, 0] + np.log(np.exp(s - m).sum(axis=1))
    return out


@pytest.mark.parametrize("case", FULL_CASES, ids=lambda c: f"w{c[0]}-seq{c[1]}")
def test_full_size_step_parity_stage_isolated(case):
    torch = torch_or_skip()
    c, b, nsteps, nfwd = case
    w, s = workloads.WORKLOADS[c], workloads.seeds(c)
    cfg = workloads.model_cfg(c)
    B, L, V, T, prior = w["B"], w["L"], w["vocab"], w["T"], w["prior"]
    M = B * L
    say(f"full-size step parity: workload {c} ({w['name']}), B {B} x L {L}, sequence {b}, {nsteps} steps")
    t0 = time.time()
    P, buf = _host_params(torch, cfg, s["param"])
    say(f"  parameters ready ({time.time() - t0:.0f} s)")
    ws = torch.zeros(dd.loop_workspace_bytes(cfg, B, L), dtype=torch.uint8, device="cuda")
    lay = dd.loop_workspace_layout(cfg, B, L)
    r0 = b * L
    seq = np.arange(r0, r0 + L)
    if prior == "mask":
        z = torch.full((M,), V, dtype=torch.int32, device="cuda")
    else:   # z_1 = Gaussian-latent argmax of clean tokens at alpha_tilde = 0 (App. A.5)
        x = workloads.clean_tokens(s["data"], B, L, V).reshape(-1)
        z = torch.empty(M, dtype=torch.int32, device="cuda")
        dd.gaussian_latent_argmax(dev_i32(torch, x), M, V, 0.0, 1.0, seed=s["noise"], step=0, z_out=z)
        ref_z1 = olatent.latent_argmax(x[seq], V, 0.0, 1.0, s["noise"], 0, rows=seq)
        assert np.array_equal(z.cpu().numpy()[seq], ref_z1), "Gaussian-latent start differs"
        say("  Gaussian-latent start of the sequence equals the oracle's")
    alphas = 1.0 - np.arange(T + 1) / T
    for i in range(nsteps):
        k = T - i
        at, as_ = alphas[k], alphas[k - 1]
        before = z.cpu().numpy()
        dd.sample_loop(cfg, buf, B, L, 1, np.array([as_, at]), z, ws, noise_seed=s["noise"])
        assert dd.read_device_error(ws[:4].view(torch.int32)) == 0
        after = z.cpu().numpy()
        count = int(_ws_i32(torch, ws, lay["count"], 1)[0])
        if count >= 0:   # compacted: logits row j belongs to token row rows[j]
            rows = _ws_i32(torch, ws, lay["rows"], count)
            js = np.nonzero((rows >= r0) & (rows < r0 + L))[0]
            # listed: the masked rows that stage 0 of the draw unmasks (the rest stay masked)
            assert np.array_equal(rows[js], seq[(before[seq] == V) & (after[seq] != V)])
            if js.size == 0:
                say(f"  step {k}/{T}: no row of the sequence unmasks")
                continue
            assert np.array_equal(js, np.arange(js[0], js[-1] + 1))
            j0, j1, tok = int(js[0]), int(js[-1]) + 1, rows[js]
        else:
            j0, j1, tok = r0, r0 + L, seq
        first = j0 * lay["logits_ld"]
        say(f"  step {k}/{T} (alpha_t {at:.6f}, alpha_s {as_:.6f}): {tok.size} rows of the sequence drawn; "
            f"their logits start at element {first}" + (" (past 2^31)" if first >= 2 ** 31 else ""))
        G = _ws_logits(torch, ws, lay, j0, j1, V)
        # stage 4: carry-over (masked prior), whole batch
        if prior == "mask":
            was = before != V
            assert np.array_equal(after[was], before[was]), "an unmasked token changed"
            assert (after == V).sum() <= (before == V).sum()
        # stage 1: logits against the oracle's forward pass on the same state
        if i < nfwd:
            t1 = time.time()
            ref = oforward.forward(cfg, P, before[seq][None], at,
                                   on_layer=lambda l: say(f"    oracle layer {l + 1}/{cfg['n_layers']} "
                                                          f"({time.time() - t1:.0f} s)")
                                   if L >= 4096 else None).reshape(L, V)
            dl = float(np.abs(G - ref[tok - r0]).max())
            say(f"  logits: max |dlogit| = {dl:.3e} over {tok.size} x {V} (logit std {ref.std():.3f}; "
                f"oracle {time.time() - t1:.0f} s)")
            assert dl <= LOGIT_TOL
        # stage 2: the oracle's draw on the GPU's logits, same noise counters (step 1 of a one-step loop)
        zs, gaps, probs = osampler.posterior_sample(prior, G, before[tok], at, as_,
                                                    osampler.PhiloxNoise(s["noise"], 1), rows=tok,
                                                    return_probs=True)
        compare_ids(after[tok], zs, gaps, f"  ids, step {k}")
        # stage 3: the probabilities the draw's fp32 row log-sum-exp implies, and the group masses
        rl = _ws_f32(torch, ws, lay["row_lse"], M)[tok].astype(np.float64)
        lse = G.max(axis=1) + np.log(np.exp(G - G.max(axis=1, keepdims=True)).sum(axis=1))
        dp = 0.0
        for q in range(tok.size):
            pg = oposterior.posterior(prior, np.exp(G[q] - rl[q]), int(before[tok[q]]), at, as_)
            dp = max(dp, float(np.abs(pg - probs[q]).max()))
        ng = (V + 255) // 256
        gl = _ws_f32(torch, ws, lay["glse"], (j1 - j0) * lay["glse_ld"], j0 * lay["glse_ld"])
        gl = gl.reshape(j1 - j0, lay["glse_ld"])[:, :ng].astype(np.float64)
        rgl = _group_lse(G, V)
        dmass = float(np.abs(np.exp(gl - rl[:, None]) - np.exp(rgl - lse[:, None])).max())
        say(f"  probabilities: max |dp| = {dp:.3e}, max |d row lse| = {np.abs(rl - lse).max():.3e}, "
            f"max |d group lse| = {np.abs(gl - rgl).max():.3e}, max |d group mass| = {dmass:.3e}")
        assert dp <= PROB_TOL and dmass <= PROB_TOL
