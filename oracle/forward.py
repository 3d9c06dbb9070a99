"""The bidirectional transformer denoiser x_theta(z_t, t) in float64
(test infrastructure only).

The paper (Background, Discrete Diffusion Language Models) defines the
denoiser only as a map from (z_t, t) to per-position distributions over the
vocabulary; its own model is a causal AR transformer (Sec. 3, Diffusion-
augmented LLMs) which this path does not use.  The workloads fix a pre-LN,
GPT-2-shaped, non-causal transformer.  This build's reading:

  h   = tok_emb[z_t] + pos_emb[l] + temb(alpha_t)
  temb_j = sin(tau w_j) (j < d/2), cos(tau w_{j-d/2}) (j >= d/2),
           w_i = 10000 ** (-i / (d/2)), tau = 1000 (1 - alpha_t)
  per layer:  a = LN1(h); [q|k|v] = a W_qkv^T + b_qkv
              h += softmax(q k^T / sqrt(dh)) v  W_o^T + b_o   (no mask, per head)
              a = LN2(h); h += gelu_tanh(a W_1^T + b_1) W_2^T + b_2
  logits = LN_f(h) W_out^T                        (V columns, no bias)

LayerNorm uses the biased variance and eps = cfg['norm_eps'].  x_theta is the
softmax of the logits over the V real tokens (the mask class gets zero mass,
App. A.1: clean data contains no mask token).

Parity unpinned by the paper (the architecture is a convention): pinned by a
second, independent scalar-loop implementation (forward_loops), by LayerNorm
moments, by permutation equivariance with zero position embeddings and by
non-causality.
"""
import numpy as np


def time_embedding(alpha_t, d):
    half = d // 2
    tau = 1000.0 * (1.0 - float(alpha_t))
    w = 10000.0 ** (-np.arange(half, dtype=np.float64) / half)
    return np.concatenate([np.sin(tau * w), np.cos(tau * w)])


def layer_norm(x, g, b, eps):
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def gelu_tanh(x):
    return 0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (x + 0.044715 * x ** 3)))


def attention(q, k, v):
    """Non-causal softmax attention for one head: q, k, v are [L, dh]."""
    s = q @ k.T / np.sqrt(q.shape[-1])
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p /= p.sum(axis=-1, keepdims=True)
    return p @ v


def forward_hidden(cfg, P, z, alpha_t):
    """Final-LN activations [B, L, d] for token ids z [B, L]."""
    z = np.asarray(z)
    B, L = z.shape
    d, H = cfg["d_model"], cfg["n_heads"]
    dh = d // H
    eps = cfg["norm_eps"]
    h = P["tok_emb"][z] + P["pos_emb"][:L][None]
    if cfg.get("time_cond", True):
        h = h + time_embedding(alpha_t, d)[None, None]
    for l in range(cfg["n_layers"]):
        p = lambda n: P[f"l{l}.{n}"]
        a = layer_norm(h, p("ln1_g"), p("ln1_b"), eps)
        qkv = a @ p("w_qkv").T + p("b_qkv")
        q, k, v = qkv[..., :d], qkv[..., d:2 * d], qkv[..., 2 * d:]
        o = np.empty_like(q)
        for b in range(B):
            for hh in range(H):
                cs = slice(hh * dh, (hh + 1) * dh)
                o[b, :, cs] = attention(q[b, :, cs], k[b, :, cs], v[b, :, cs])
        h = h + o @ p("w_o").T + p("b_o")
        a = layer_norm(h, p("ln2_g"), p("ln2_b"), eps)
        h = h + gelu_tanh(a @ p("w_1").T + p("b_1")) @ p("w_2").T + p("b_2")
    return layer_norm(h, P["lnf_g"], P["lnf_b"], eps)


def forward(cfg, P, z, alpha_t):
    """Logits [B, L, V] (float64) of the denoiser at noise level alpha_t."""
    return forward_hidden(cfg, P, z, alpha_t) @ P["w_out"].T


def x_theta(logits):
    """Per-position probabilities over the V real tokens (softmax of the logits)."""
    m = logits.max(axis=-1, keepdims=True)
    e = np.exp(logits - m)
    return e / e.sum(axis=-1, keepdims=True)
