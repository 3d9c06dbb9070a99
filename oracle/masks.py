"""Attention visibility patterns of the denoiser (test infrastructure only).

A pattern is a boolean matrix vis[i, j]: query position i may attend to key
position j.  Each builder writes the pattern's definition out element by
element.

  bidirectional  every query sees every key (the denoiser of Background,
                 Discrete Diffusion Language Models).
  causal         key j is visible to query i iff j <= i.  This is the mask of
                 the AR pathway (Sec. 3.1, eq. (denoise-ar)) and of the
                 drafting pass: the block [clean, z_t] of Sec. 4.1 attends
                 causally within itself and to the whole cached context, so
                 one pass over the concatenated sequence is causal
                 throughout.
  block_causal   blocks of `bs` consecutive positions; query i sees key j iff
                 block(j) <= block(i).  This is attention that is
                 bidirectional within a draft block and causal across blocks
                 (the draft-block attention of the baselines in Sec. 5.1).
  draft_training the sequence [x, z_1] of Sec. 3.2 (Block Diffusion): x and z_1
                 each have N blocks of bs tokens.  Attention is causal within
                 x and within each noisy block z_1^(b), and every token of
                 z_1^(b) also sees all clean blocks x^(<b).  x never sees z_1.

Pinned by counting the visible pairs against closed forms, by the special
cases (N = 1 and bs = 1 reductions) and by the causal-invariance tests of the
forward pass (a perturbation never reaches a position that cannot see it).
"""
import numpy as np


def bidirectional(L):
    return np.ones((L, L), dtype=bool)


def causal(L):
    vis = np.zeros((L, L), dtype=bool)
    for i in range(L):
        for j in range(L):
            vis[i, j] = j <= i
    return vis


def block_causal(L, bs):
    vis = np.zeros((L, L), dtype=bool)
    for i in range(L):
        for j in range(L):
            vis[i, j] = (j // bs) <= (i // bs)
    return vis


def draft_training(n_blocks, bs):
    """Pattern over [x, z_1], both of length n_blocks * bs (total 2 n_blocks bs)."""
    n = n_blocks * bs
    L = 2 * n
    vis = np.zeros((L, L), dtype=bool)
    for i in range(L):
        for j in range(L):
            if i < n:                        # clean position: causal within x only
                vis[i, j] = j < n and j <= i
            else:                            # noisy position i = n + b bs + l
                b, l = divmod(i - n, bs)
                if j < n:                    # clean keys: all of x^(<b)
                    vis[i, j] = j < b * bs
                else:                        # noisy keys: causal within z_1^(b)
                    bj, lj = divmod(j - n, bs)
                    vis[i, j] = bj == b and lj <= l
    return vis
