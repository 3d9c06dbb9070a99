"""A second, independently written denoiser forward pass using scalar loops
and the `math` module only (test infrastructure only; small shapes only).

It restates the same architecture as `forward` token by token and feature by
feature, without numpy linear algebra, so that a transposed operand, a wrong
head slice, a missing bias or a wrong normalisation in either implementation
shows up as a disagreement.  Used only as a pin of `forward`.
"""
import math


def _ln(vec, g, b, eps):
    n = len(vec)
    mu = sum(vec) / n
    var = sum((x - mu) * (x - mu) for x in vec) / n
    inv = 1.0 / math.sqrt(var + eps)
    return [(vec[i] - mu) * inv * g[i] + b[i] for i in range(n)]


def _rms(vec, g, eps):
    n = len(vec)
    ms = sum(x * x for x in vec) / n
    inv = 1.0 / math.sqrt(ms + eps)
    return [vec[i] * inv * g[i] for i in range(n)]


def _linear(vec, W, bias):
    """W is a nested list [out][in]; returns W vec + bias."""
    out = []
    for o in range(len(W)):
        row = W[o]
        acc = 0.0
        for i in range(len(vec)):
            acc += row[i] * vec[i]
        out.append(acc + (bias[o] if bias is not None else 0.0))
    return out


def _gelu(x):
    c = math.sqrt(2.0 / math.pi)
    return 0.5 * x * (1.0 + math.tanh(c * (x + 0.044715 * x * x * x)))


def forward_loops(cfg, P, z, alpha_t, vis=None, gate=None):
    """Logits as nested lists [B][L][V]; P values may be numpy arrays.

    vis[i][j] false hides key j from query i (None: all visible); gate[l] in
    {0, 1} switches the adapters of position l (None: all on)."""
    tl = lambda a: a.tolist()
    d, H, V = cfg["d_model"], cfg["n_heads"], cfg["vocab"]
    r = int(cfg.get("lora_rank", 0) or 0)
    scale = float(cfg["lora_alpha"]) / r if r else 0.0
    dh = d // H
    eps = cfg["norm_eps"]
    rms = cfg.get("norm", "layer") == "rms"
    norm = (lambda vec, g, b: _rms(vec, g, eps)) if rms else (lambda vec, g, b: _ln(vec, g, b, eps))
    tok, pos = tl(P["tok_emb"]), tl(P["pos_emb"])
    half = d // 2
    tau = 1000.0 * (1.0 - alpha_t)
    temb = [0.0] * d
    if cfg.get("time_cond", True):
        for j in range(d):
            i = j if j < half else j - half
            ang = tau * math.pow(10000.0, -i / half)
            temb[j] = math.sin(ang) if j < half else math.cos(ang)
    out = []
    for seq in z:
        L = len(seq)
        hs = [[tok[int(seq[l])][j] + pos[l][j] + temb[j] for j in range(d)] for l in range(L)]
        for layer in range(cfg["n_layers"]):
            g = lambda n: tl(P[f"l{layer}.{n}"])
            ln1g, ln1b, ln2g, ln2b = g("ln1_g"), g("ln1_b"), g("ln2_g"), g("ln2_b")
            proj = {}
            for p in ("qkv", "o", "1", "2"):
                ad = (g(f"lora_a_{p}"), g(f"lora_b_{p}")) if r else None
                proj[p] = (g(f"w_{p}"), g(f"b_{p}"), ad)

            def lin(p, vec, l):
                W, bias, ad = proj[p]
                y = _linear(vec, W, bias)
                if ad is not None and (gate is None or gate[l]):
                    t = _linear(_linear(vec, ad[0], None), ad[1], None)
                    y = [y[o] + scale * t[o] for o in range(len(y))]
                return y

            qkv = [lin("qkv", norm(hs[l], ln1g, ln1b), l) for l in range(L)]
            att = [[0.0] * d for _ in range(L)]
            for hh in range(H):
                off = hh * dh
                for i in range(L):
                    keys = [j for j in range(L) if vis is None or vis[i][j]]
                    scores = []
                    for j in keys:
                        s = 0.0
                        for c in range(dh):
                            s += qkv[i][off + c] * qkv[j][d + off + c]
                        scores.append(s / math.sqrt(dh))
                    mx = max(scores)
                    ws = [math.exp(s - mx) for s in scores]
                    tot = sum(ws)
                    for c in range(dh):
                        acc = 0.0
                        for wj, j in zip(ws, keys):
                            acc += wj * qkv[j][2 * d + off + c]
                        att[i][off + c] = acc / tot
            for l in range(L):
                o = lin("o", att[l], l)
                hs[l] = [hs[l][j] + o[j] for j in range(d)]
                u = [_gelu(x) for x in lin("1", norm(hs[l], ln2g, ln2b), l)]
                m = lin("2", u, l)
                hs[l] = [hs[l][j] + m[j] for j in range(d)]
        lnfg, lnfb, wout = tl(P["lnf_g"]), tl(P["lnf_b"]), tl(P["w_out"])
        out.append([_linear(norm(hs[l], lnfg, lnfb), wout, None) for l in range(L)])
    return out
