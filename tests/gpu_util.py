"""Helpers shared by the GPU parity tests (not a test module)."""
import sys

import numpy as np
import pytest

GAP = 1e-3          # ids must agree wherever the oracle's top-two perturbed scores differ by more
MIN_AGREE = 0.999   # and on at least this fraction of rows overall
PROB_TOL = 1e-3     # posterior probabilities, absolute


def torch_or_skip():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev_i32(torch, a):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.int32))).cuda()


def dev_words(torch, w):
    """uint32 noise words as an int32 device tensor holding the same bits."""
    return torch.from_numpy(np.ascontiguousarray(np.asarray(w, dtype=np.uint32)).view(np.int32)).cuda()


def round_to_dtype(x, dtype):
    """float64 values rounded (nearest even) to bf16 or fp32, returned as float64."""
    import torch
    t = torch.from_numpy(np.asarray(x, dtype=np.float32))
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
    return t.to(torch.float64).numpy()


def logits_dev(torch, vals, dtype, ld):
    R, V = vals.shape
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    out = torch.zeros((R, ld), dtype=tdt)
    out[:, :V] = torch.from_numpy(np.asarray(vals, dtype=np.float32)).to(tdt)
    return out.cuda()


def compare_ids(gpu, ref, gaps, what):
    """Gap rule: exact where min(level gaps) > GAP, and >= MIN_AGREE agreement overall."""
    gpu, ref = np.asarray(gpu), np.asarray(ref)
    g = np.min(gaps, axis=1) if gaps.ndim == 2 else gaps
    clear = g > GAP
    bad = np.nonzero(clear & (gpu != ref))[0]
    agree = float(np.mean(gpu == ref))
    say(f"{what}: rows={gpu.size} agree={agree:.6f} clear={int(clear.sum())} clear_mismatch={bad.size}")
    assert bad.size == 0, f"{what}: ids differ on clear rows {bad[:10]} gpu={gpu[bad[:10]]} ref={ref[bad[:10]]}"
    assert agree >= MIN_AGREE, f"{what}: agreement {agree}"
