"""The bidirectional transformer denoiser x_theta(z_t, t) in float64
(test infrastructure only).

The paper (Background, Discrete Diffusion Language Models) defines the
denoiser only as a map from (z_t, t) to per-position distributions over the
vocabulary; its own model is a causal AR transformer (Sec. 3, Diffusion-
augmented LLMs) which this path does not use.  The workloads fix a pre-LN,
GPT-2-shaped, non-causal transformer.  Reading adopted here:

  h   = tok_emb[z_t] + pos_emb[l] + temb(alpha_t)
  temb_j = sin(tau w_j) (j < d/2), cos(tau w_{j-d/2}) (j >= d/2),
           w_i = 10000 ** (-i / (d/2)), tau = 1000 (1 - alpha_t)
  per layer:  a = LN1(h); [q|k|v] = a W_qkv^T + b_qkv
              h += softmax(q k^T / sqrt(dh)) v  W_o^T + b_o   (per head)
              a = LN2(h); h += gelu_tanh(a W_1^T + b_1) W_2^T + b_2
  logits = LN_f(h) W_out^T                        (V columns, no bias)

LN is cfg['norm']: "layer" (the default) is LayerNorm with the biased variance,
(x - mean) / sqrt(var + eps) g + b; "rms" is RMSNorm, x / sqrt(mean(x^2) + eps) g,
over the whole row with no shift (the paper's own model, Sec. 5.1, names a
grouped RMSNorm without giving the groups; the reading here is one group, the
row), eps = cfg['norm_eps'] in both.  x_theta is the
softmax of the logits over the V real tokens (the mask class gets zero mass,
App. A.1: clean data contains no mask token).

Two extensions toward the paper's drafting pathway (Sec. 3.1 - 3.2, Sec. 4.1):
  vis   [L, L] boolean attention pattern (oracle.masks): query i attends only
        to keys j with vis[i, j]; the softmax runs over those keys alone.
        None is the bidirectional pattern.
  gated LoRA (cfg['lora_rank'] = r > 0): each projection y = a W^T + b becomes
        y = a W^T + b + g_l (alpha/r) (a A^T) B^T
        at sequence position l, with g_l in {0, 1} the per-position adapter
        gate (Sec. 3.2 and Sec. 4.1: adapters off at clean positions, on at
        noisy ones); gate None switches them on everywhere.  With g_l = 1 this
        is the merged weight W + (alpha/r) B A of App. "Varying LoRA alpha / r".

The paper does not fix this architecture, so its pins come from elsewhere: a
library implementation of the same pre-LN layer (torch.nn.TransformerEncoderLayer
with norm_first and tanh GELU, in float64, with and without an attention
pattern), a second, independent scalar-loop implementation (forward_loops),
LayerNorm moments, permutation equivariance with zero position embeddings and
non-causality.  The extensions are pinned by forward_loops under every
pattern and gate, by the reach of a perturbation under each pattern (it
changes exactly the positions that can see it), by the merged-weight identity
(all gates on == base weights W + (alpha/r) B A) and by the teacher property
of Sec. 3.2 (under the [x, z_1] pattern with adapters on z_1 only, the logits
at x equal the base model's causal logits on x alone).
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


def rms_norm(x, g, eps):
    ms = (x ** 2).mean(axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def normalise(cfg, x, g, b):
    """The normalisation cfg['norm'] selects ("layer" or "rms"; the shift b is unused by RMSNorm)."""
    norm = cfg.get("norm", "layer")
    if norm == "rms":
        return rms_norm(x, g, cfg["norm_eps"])
    if norm != "layer":
        raise ValueError(f"unknown norm {norm!r}")
    return layer_norm(x, g, b, cfg["norm_eps"])


def gelu_tanh(x):
    return 0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (x + 0.044715 * x ** 3)))


def attention(q, k, v, vis=None):
    """Softmax attention for one head: q, k, v are [L, dh]; vis [L, L] or None (all visible)."""
    s = q @ k.T / np.sqrt(q.shape[-1])
    if vis is not None:
        s = np.where(vis, s, -np.inf)
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p /= p.sum(axis=-1, keepdims=True)
    return p @ v


def projection(cfg, P, l, name, a, gate):
    """a W^T + b of projection `name` (qkv, o, 1, 2) of layer l, plus the gated adapter term."""
    y = a @ P[f"l{l}.w_{name}"].T + P[f"l{l}.b_{name}"]
    r = int(cfg.get("lora_rank", 0) or 0)
    if r:
        scale = float(cfg["lora_alpha"]) / r
        u = a @ P[f"l{l}.lora_a_{name}"].T
        y = y + (gate[None, :, None] * scale) * (u @ P[f"l{l}.lora_b_{name}"].T)
    return y


def forward_hidden(cfg, P, z, alpha_t, vis=None, gate=None, on_layer=None):
    """Final-LN activations [B, L, d] for token ids z [B, L].  on_layer: optional callable that is
    given the index of each layer once it is done (progress reporting of long runs only)."""
    z = np.asarray(z)
    B, L = z.shape
    d, H = cfg["d_model"], cfg["n_heads"]
    dh = d // H
    g = np.ones(L) if gate is None else np.asarray(gate, dtype=np.float64)
    h = P["tok_emb"][z] + P["pos_emb"][:L][None]
    if cfg.get("time_cond", True):
        h = h + time_embedding(alpha_t, d)[None, None]
    for l in range(cfg["n_layers"]):
        p = lambda n: P[f"l{l}.{n}"]
        a = normalise(cfg, h, p("ln1_g"), p("ln1_b"))
        qkv = projection(cfg, P, l, "qkv", a, g)
        q, k, v = qkv[..., :d], qkv[..., d:2 * d], qkv[..., 2 * d:]
        o = np.empty_like(q)
        for b in range(B):
            for hh in range(H):
                cs = slice(hh * dh, (hh + 1) * dh)
                o[b, :, cs] = attention(q[b, :, cs], k[b, :, cs], v[b, :, cs], vis)
        h = h + projection(cfg, P, l, "o", o, g)
        a = normalise(cfg, h, p("ln2_g"), p("ln2_b"))
        h = h + projection(cfg, P, l, "2", gelu_tanh(projection(cfg, P, l, "1", a, g)), g)
        if on_layer is not None:
            on_layer(l)
    return normalise(cfg, h, P["lnf_g"], P["lnf_b"])


def forward(cfg, P, z, alpha_t, vis=None, gate=None, on_layer=None):
    """Logits [B, L, V] (float64) of the denoiser at noise level alpha_t."""
    return forward_hidden(cfg, P, z, alpha_t, vis, gate, on_layer) @ P["w_out"].T


def x_theta(logits):
    """Per-position probabilities over the V real tokens (softmax of the logits)."""
    m = logits.max(axis=-1, keepdims=True)
    e = np.exp(logits - m)
    return e / e.sum(axis=-1, keepdims=True)
