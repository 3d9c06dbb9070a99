"""The oracle's denoiser against a library implementation of the same architecture.

A pre-LN transformer layer (LayerNorm -> multi-head self-attention -> residual, LayerNorm -> MLP with
tanh GELU -> residual) is what torch.nn.TransformerEncoderLayer computes with norm_first=True, so
the oracle's forward pass (embeddings + time embedding, the layers, the final LayerNorm and the
vocabulary projection) must agree with a stack of those layers loaded with the same parameters, in
float64 on the CPU, with and without an attention pattern.  The library's attention, LayerNorm and
linear layers are independent of the oracle's code.  Under norm = "rms" the layer's two LayerNorm
modules are replaced by torch.nn.RMSNorm modules (a library RMSNorm with the same gain) and the final
normalisation is torch's rms_norm.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
import torch.nn.functional as F  # noqa: E402

from oracle import forward, masks, params  # noqa: E402

CFG = dict(n_layers=2, d_model=16, n_heads=2, d_mlp=40, vocab=11, prior="mask", dtype="fp32",
           max_len=12, time_cond=True, norm_eps=1e-5)


def _library_logits(cfg, P, z, alpha_t, vis=None):
    d, H, Fm, eps = cfg["d_model"], cfg["n_heads"], cfg["d_mlp"], cfg["norm_eps"]
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))
    z = np.asarray(z)
    B, L = z.shape
    # token + position embedding and the sinusoidal time embedding of tau = 1000 (1 - alpha_t)
    half = d // 2
    tau = 1000.0 * (1.0 - alpha_t)
    w = 10000.0 ** (-np.arange(half) / half)
    temb = np.concatenate([np.sin(tau * w), np.cos(tau * w)])
    x = t(P["tok_emb"][z] + P["pos_emb"][:L][None] + temb[None, None])
    mask = None if vis is None else ~t(vis).bool()          # True: the key may not be attended
    rms = cfg.get("norm", "layer") == "rms"
    for l in range(cfg["n_layers"]):
        layer = torch.nn.TransformerEncoderLayer(d, H, dim_feedforward=Fm, dropout=0.0,
                                                 activation=lambda a: F.gelu(a, approximate="tanh"),
                                                 layer_norm_eps=eps, batch_first=True, norm_first=True,
                                                 dtype=torch.float64)
        if rms:
            layer.norm1 = torch.nn.RMSNorm(d, eps=eps, dtype=torch.float64)
            layer.norm2 = torch.nn.RMSNorm(d, eps=eps, dtype=torch.float64)
        p = lambda n: t(P[f"l{l}.{n}"])
        with torch.no_grad():
            layer.self_attn.in_proj_weight.copy_(p("w_qkv"))
            layer.self_attn.in_proj_bias.copy_(p("b_qkv"))
            layer.self_attn.out_proj.weight.copy_(p("w_o"))
            layer.self_attn.out_proj.bias.copy_(p("b_o"))
            layer.linear1.weight.copy_(p("w_1"))
            layer.linear1.bias.copy_(p("b_1"))
            layer.linear2.weight.copy_(p("w_2"))
            layer.linear2.bias.copy_(p("b_2"))
            layer.norm1.weight.copy_(p("ln1_g"))
            layer.norm2.weight.copy_(p("ln2_g"))
            if not rms:
                layer.norm1.bias.copy_(p("ln1_b"))
                layer.norm2.bias.copy_(p("ln2_b"))
        layer.eval()
        with torch.no_grad():
            x = layer(x, src_mask=mask)
    if rms:
        x = F.rms_norm(x, (d,), t(P["lnf_g"]), eps)
    else:
        x = F.layer_norm(x, (d,), t(P["lnf_g"]), t(P["lnf_b"]), eps)
    return (x @ t(P["w_out"]).T).numpy()


def _params(seed=3, scale=4.0, cfg=CFG):
    P = params.init_params(cfg, seed)
    return {k: (v * scale if not k.endswith("_g") else v) for k, v in P.items()}


@pytest.mark.parametrize("norm", ["layer", "rms"])
@pytest.mark.parametrize("alpha_t", [1.0, 0.37, 0.0])
def test_forward_equals_library_transformer(alpha_t, norm):
    cfg = dict(CFG, norm=norm)
    P = _params(cfg=cfg)
    z = np.random.default_rng(5).integers(0, CFG["vocab"] + 1, size=(3, 12))
    ours = forward.forward(cfg, P, z, alpha_t)
    lib = _library_logits(cfg, P, z, alpha_t)
    assert np.abs(ours - lib).max() < 1e-10 * max(1.0, np.abs(lib).max())


@pytest.mark.parametrize("name", ["causal", "block", "draft"])
def test_masked_forward_equals_library_transformer(name):
    L = 12
    vis = {"causal": masks.causal(L), "block": masks.block_causal(L, 5), "draft": masks.draft_training(2, 3)}[name]
    P = _params(seed=9)
    z = np.random.default_rng(6).integers(0, CFG["vocab"] + 1, size=(2, L))
    ours = forward.forward(CFG, P, z, 0.5, vis)
    lib = _library_logits(CFG, P, z, 0.5, vis)
    assert np.abs(ours - lib).max() < 1e-10 * max(1.0, np.abs(lib).max())
