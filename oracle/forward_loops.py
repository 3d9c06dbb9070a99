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


def forward_loops(cfg, P, z, alpha_t):
    """Logits as nested lists [B][L][V]; P values may be numpy arrays."""
    tl = lambda a: a.tolist()
    d, H, V = cfg["d_model"], cfg["n_heads"], cfg["vocab"]
    dh = d // H
    eps = cfg["norm_eps"]
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
            ln1g, ln1b, wqkv, bqkv = g("ln1_g"), g("ln1_b"), g("w_qkv"), g("b_qkv")
            wo, bo, ln2g, ln2b = g("w_o"), g("b_o"), g("ln2_g"), g("ln2_b")
            w1, b1, w2, b2 = g("w_1"), g("b_1"), g("w_2"), g("b_2")
            qkv = [_linear(_ln(hs[l], ln1g, ln1b, eps), wqkv, bqkv) for l in range(L)]
            att = [[0.0] * d for _ in range(L)]
            for hh in range(H):
                off = hh * dh
                for i in range(L):
                    scores = []
                    for j in range(L):
                        s = 0.0
                        for c in range(dh):
                            s += qkv[i][off + c] * qkv[j][d + off + c]
                        scores.append(s / math.sqrt(dh))
                    mx = max(scores)
                    ws = [math.exp(s - mx) for s in scores]
                    tot = sum(ws)
                    for c in range(dh):
                        acc = 0.0
                        for j in range(L):
                            acc += ws[j] * qkv[j][2 * d + off + c]
                        att[i][off + c] = acc / tot
            for l in range(L):
                o = _linear(att[l], wo, bo)
                hs[l] = [hs[l][j] + o[j] for j in range(d)]
                u = [_gelu(x) for x in _linear(_ln(hs[l], ln2g, ln2b, eps), w1, b1)]
                m = _linear(u, w2, b2)
                hs[l] = [hs[l][j] + m[j] for j in range(d)]
        lnfg, lnfb, wout = tl(P["lnf_g"]), tl(P["lnf_b"]), tl(P["w_out"])
        out.append([_linear(_ln(hs[l], lnfg, lnfb, eps), wout, None) for l in range(L)])
    return out
