"""The store-free draw (DD_LOOP_STORE_FREE): the vocabulary projection writes no logits, only each
row's per-group log-sum-exps and per-group inverse-CDF candidates, and the draw takes level 1 from
the former and level 2 from the candidate of the chosen group.

Stage-isolated like the full-size tests: one reverse step runs twice from the same state, first in
the default mode (which leaves the step's logits in the workspace), then store-free.  The forward
pass is the same in both, so the default run's logits are the ones the store-free epilogue saw.
Checked against the oracle on those logits, with the same Philox counters (step 1 of a one-step
loop): every group's candidate of the drawn rows (oracle.sampler.group_candidates; exact where the
uniform's target lies more than 1e-4 of the group's mass from a class boundary), the group
log-sum-exps (bit-identical to the default mode's), and the ids (oracle.sampler.posterior_sample /
psi_sample with the inverse-CDF level 2, gap rule); carry-over bit-exact.
"""
import numpy as np
import pytest

import workloads
from oracle import params as oparams, sampler as osampler
from paper_2609_04010_amd import _lib as dd
from tests.gpu_util import compare_ids, say, torch_or_skip

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]

CAND_GAP = 1e-4


def _params(torch, cfg, seed):
    specs = oparams.specs(cfg)
    P = workloads.host_params(cfg, seed, specs)
    blob = dd.pack_params(cfg, [P[n] for n, _, _ in specs])
    buf = torch.zeros(blob.size, dtype=torch.uint8, device="cuda")
    dd.init_params(cfg, buf, host_blob=blob)
    return buf


def _ws(torch, ws, off, n, dt):
    return ws[off:off + 4 * n].view(dt).cpu().numpy()


def _one_step(torch, cfg, buf, B, L, z0, at, as_, seed, kappa, store_free, check_rows=None):
    """One reverse step (a one-step loop) from state z0; returns (z after, count, rows, logits or
    None, glse [count, ngroups], cand [count, ngroups] or None)."""
    V = cfg["vocab"]
    M = B * L
    lay = dd.loop_workspace_layout(cfg, B, L)
    ws = torch.zeros(dd.loop_workspace_bytes(cfg, B, L), dtype=torch.uint8, device="cuda")
    z = torch.from_numpy(z0.astype(np.int32)).cuda()
    kap = None if kappa is None else np.array([1.0, kappa])
    dd.sample_loop(cfg, buf, B, L, 1, np.array([as_, at]), z, ws, noise_seed=seed, kappas=kap,
                   store_free=store_free)
    assert dd.read_device_error(ws[:4].view(torch.int32)) == 0
    count = int(_ws(torch, ws, lay["count"], 1, torch.int32)[0])
    rows = _ws(torch, ws, lay["rows"], count, torch.int32)
    ng, gld = (V + 255) // 256, lay["glse_ld"]
    glse = _ws(torch, ws, lay["glse"], count * gld, torch.float32).reshape(count, gld)[:, :ng]
    logits = cand = None
    if store_free:
        cand = _ws(torch, ws, lay["cand"], count * gld, torch.int32).reshape(count, gld)[:, :ng]
    else:
        ld = lay["logits_ld"]
        a = lay["logits"]
        logits = ws[a:a + 2 * count * ld].view(torch.bfloat16).view(count, ld)[:, :V].float().cpu().numpy()
    return z.cpu().numpy(), count, rows, logits, glse, cand


def _check(torch, cfg, B, L, frac, at, as_, kappa, seed, cand_rows=None, ids_last_seq=False):
    V = cfg["vocab"]
    buf = _params(torch, cfg, seed)
    z0 = workloads.masked_state(seed + 1, B, L, V, frac).reshape(-1)
    noise = seed + 2
    za, ca, ra, G, ga, _ = _one_step(torch, cfg, buf, B, L, z0, at, as_, noise, kappa, False)
    zb, cb, rb, _, gb, cand = _one_step(torch, cfg, buf, B, L, z0, at, as_, noise, kappa, True)
    assert ca == cb and np.array_equal(ra, rb)
    assert np.array_equal(ga, gb), "group log-sum-exps differ between the modes"
    say(f"  {cb} rows drawn of {B * L}; V {V}; kappa {kappa}")
    G = G.astype(np.float64)
    nz = osampler.PhiloxNoise(noise, 1)
    # every group's candidate (on a subset of rows at the largest sizes)
    sel = np.arange(cb) if cand_rows is None else np.linspace(0, cb - 1, min(cand_rows, cb)).astype(int)
    mism = clear = 0
    for j in sel:
        ref, gaps = osampler.group_candidates(G[j], int(rb[j]), nz, V)
        ok = gaps > CAND_GAP
        clear += int(ok.sum())
        bad = np.nonzero(ok & (cand[j] != ref))[0]
        assert bad.size == 0, f"row {j} (token {rb[j]}): candidates {cand[j][bad]} vs {ref[bad]} in groups {bad}"
        mism += int((cand[j] != ref).sum())
    say(f"  candidates: {sel.size} rows x {cand.shape[1]} groups, {clear} clear, {mism} differ (all near a boundary)")
    # the ids: the oracle's inverse-CDF two-level draw on the same logits and counters (with
    # ids_last_seq on the logits rows of the last sequence only: the end of the list)
    js = np.nonzero(rb >= (B - 1) * L)[0] if ids_last_seq else np.arange(cb)
    tok = rb[js]
    if kappa is None:
        zs, gaps = osampler.posterior_sample("mask", G[js], z0[tok], at, as_, nz, rows=tok, level2="cdf")
    else:
        zs, gaps = osampler.psi_sample("mask", G[js], z0[tok], at, as_, kappa, nz, rows=tok, level2="cdf")
    compare_ids(zb[tok], zs, gaps, "  store-free ids")
    tok = rb
    # rows not in the list: carried over (kappa None) or kept / remasked exactly as the default mode
    rest = np.setdiff1d(np.arange(B * L), tok)
    if kappa is None:
        assert np.array_equal(zb[rest], z0[rest])
    else:
        assert np.array_equal(zb[rest], za[rest])
    # level 1 is shared (same group log-sum-exps, same words): the store-free id lies in the group
    # the default mode's id lies in
    grp = lambda z: np.where(z == V, -1, z // 256)
    assert np.array_equal(grp(zb[tok]), grp(za[tok]))


CASES = [
    # workload, overrides, B, L, masked fraction, alpha_t, alpha_s, kappa
    (2, dict(n_layers=2), 2, 300, 0.7, 0.5, 0.6, None),
    (2, dict(n_layers=1, vocab=1000), 3, 200, 1.0, 0.0, 0.1, None),
    (2, dict(n_layers=1, vocab=512), 2, 130, 0.5, 0.3, 0.45, None),
    (2, dict(n_layers=1, vocab=700), 2, 256, 0.6, 0.4, 0.55, 0.5),
    (5, dict(n_layers=1, max_len=4096), 1, 520, 0.8, 0.6, 0.7, None),
    # one ragged group only (V < 256), and a last group of a single class
    (2, dict(n_layers=1, vocab=100), 2, 96, 1.0, 0.0, 0.25, None),
    (2, dict(n_layers=1, vocab=257), 2, 96, 0.9, 0.2, 0.5, 0.3),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"w{c[0]}-V{c[1].get('vocab', 'full')}-B{c[2]}-L{c[3]}-k{c[7]}")
def test_store_free_step_matches_oracle(case):
    torch = torch_or_skip()
    c, over, B, L, frac, at, as_, kappa = case
    cfg = workloads.model_cfg(c, **over)
    say("store-free step", case)
    _check(torch, cfg, B, L, frac, at, as_, kappa, workloads.seeds(c)["param"] + 7)


def test_store_free_step_full_size_workload2():
    """The benchmark's launch shape (B 16 x L 1024, 12 layers, V 50257), the first reverse step of its
    schedule (every row masked); candidates checked on 512 of the rows."""
    torch = torch_or_skip()
    cfg = workloads.model_cfg(2)
    w = workloads.WORKLOADS[2]
    T = w["T"]
    say("store-free step, workload 2 full size")
    _check(torch, cfg, w["B"], w["L"], 1.0, 0.0, 1.0 / T, None, workloads.seeds(2)["param"], cand_rows=512)


def test_store_free_step_full_size_workload4():
    """B 128 x L 1024 (131072 rows, the largest batch): a mid-schedule step from a state with a
    quarter of the rows masked; ids checked on the last sequence's rows (the end of the compacted
    list), candidates on 256 rows spread over the list."""
    torch = torch_or_skip()
    cfg = workloads.model_cfg(4)
    w = workloads.WORKLOADS[4]
    B, L = w["B"], w["L"]
    say("store-free step, workload 4 full size")
    seed = workloads.seeds(4)["param"]
    _check(torch, cfg, B, L, 0.25, 0.7, 0.75, None, seed, cand_rows=256, ids_last_seq=True)


def test_store_free_loop_bookkeeping_and_determinism():
    torch = torch_or_skip()
    cfg = workloads.model_cfg(2, n_layers=2)
    V = cfg["vocab"]
    B, L, T = 2, 192, 8
    buf = _params(torch, cfg, 4)
    M = B * L
    def run():
        z = torch.full((M,), V, dtype=torch.int32, device="cuda")
        tr = torch.zeros(((T + 1) * M,), dtype=torch.int32, device="cuda")
        ws = torch.zeros(dd.loop_workspace_bytes(cfg, B, L), dtype=torch.uint8, device="cuda")
        dd.sample_loop(cfg, buf, B, L, T, 1.0 - np.arange(T + 1) / T, z, ws, noise_seed=5, z_trace=tr,
                       store_free=True)
        assert dd.read_device_error(ws[:4].view(torch.int32)) == 0
        return tr.cpu().numpy().reshape(T + 1, M)
    trace = run()
    masked = (trace == V).sum(axis=1)
    say("masked per step", masked.tolist())
    assert masked[0] == M and masked[-1] == 0 and np.all(np.diff(masked) <= 0)
    for k in range(1, T + 1):
        was = trace[k - 1] != V
        assert np.array_equal(trace[k][was], trace[k - 1][was])
    assert np.all((trace[-1] >= 0) & (trace[-1] < V))
    assert np.array_equal(run(), trace)
