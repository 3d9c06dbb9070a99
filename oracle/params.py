"""Denoiser parameters: the ordered tensor list and seeded initialisation
(test infrastructure only).

The paper's denoiser for this path is not specified beyond "a denoising model
x_theta" (Background, Discrete Diffusion Language Models); the workloads name a
pre-LayerNorm GPT-2-shaped bidirectional transformer.  Tensor order (the id of
each tensor is its index in this list), every matrix stored [out][in]:

  0  tok_emb [n_tok, d]      n_tok = V + 1 (mask prior, mask id V) or V
  1  pos_emb [max_len, d]
  per layer l, ids 2 + 12 l + (0..11):
     ln1_g [d], ln1_b [d], w_qkv [3d, d], b_qkv [3d], w_o [d, d], b_o [d],
     ln2_g [d], ln2_b [d], w_1 [F, d], b_1 [F], w_2 [d, F], b_2 [d]
  then lnf_g [d], lnf_b [d], w_out [V, d]

Adapters (cfg['lora_rank'] = r > 0, Sec. 3.1: every projection of a layer has
a LoRA adapter W + (alpha/r) B A, App. "Varying LoRA alpha / r"): the
projection tensors w_qkv, w_o, w_1, w_2 are stored [out, in + r] with row o
holding W[o, :] followed by B[o, :] (B [out, r]); the A matrices [r, in] follow
w_out, per layer l at ids 2 + 12 L + 3 + 4 l + (0..3) for qkv, o, 1, 2
(L = n_layers).  `init_params` splits each stored row into P['l.w_*'] and
P['l.lora_b_*']; `storage_tensors` joins them again in id order.

Initialisation (the reading adopted here of "weights ~ N(0, 0.02)"): element e of
tensor `id` takes the Box-Muller normal of Philox block
(e >> 1 low, e >> 1 high, id, STREAM_PARAM) under key `seed`, using words 0
and 1 (cosine branch for even e, sine for odd e).  Matrices, embeddings,
biases and LayerNorm shifts are 0.02 z; LayerNorm gains are 1 + 0.02 z.  The
float64 value is rounded to nearest-even bf16 (direct from float64) or fp32.

Pinned: the normal transform by KS tests; element placement by a scalar
re-derivation of single elements from `philox_scalar`.
"""
import numpy as np

from . import philox as _ph
from . import noise as _nz


def n_tok(cfg):
    return cfg["vocab"] + 1 if cfg["prior"] == "mask" else cfg["vocab"]


PROJ = ("qkv", "o", "1", "2")


def lora_rank(cfg):
    return int(cfg.get("lora_rank", 0) or 0)


def proj_shape(cfg, name):
    """(out, in) of projection `name` in PROJ."""
    d, F = cfg["d_model"], cfg["d_mlp"]
    return {"qkv": (3 * d, d), "o": (d, d), "1": (F, d), "2": (d, F)}[name]


def specs(cfg):
    """List of (name, stored shape, kind) in id order; kind is 'w' or 'gain'.

    With adapters the projections are listed with their stored shape
    [out, in + r] (W and B side by side) under the name of W."""
    d, F, V = cfg["d_model"], cfg["d_mlp"], cfg["vocab"]
    r = lora_rank(cfg)
    out = [("tok_emb", (n_tok(cfg), d), "w"), ("pos_emb", (cfg["max_len"], d), "w")]
    for l in range(cfg["n_layers"]):
        wq, wo, w1, w2 = ((o, i + r) for o, i in (proj_shape(cfg, p) for p in PROJ))
        out += [
            (f"l{l}.ln1_g", (d,), "gain"), (f"l{l}.ln1_b", (d,), "w"),
            (f"l{l}.w_qkv", wq, "w"), (f"l{l}.b_qkv", (3 * d,), "w"),
            (f"l{l}.w_o", wo, "w"), (f"l{l}.b_o", (d,), "w"),
            (f"l{l}.ln2_g", (d,), "gain"), (f"l{l}.ln2_b", (d,), "w"),
            (f"l{l}.w_1", w1, "w"), (f"l{l}.b_1", (F,), "w"),
            (f"l{l}.w_2", w2, "w"), (f"l{l}.b_2", (d,), "w"),
        ]
    out += [("lnf_g", (d,), "gain"), ("lnf_b", (d,), "w"), ("w_out", (V, d), "w")]
    if r:
        for l in range(cfg["n_layers"]):
            out += [(f"l{l}.lora_a_{p}", (r, proj_shape(cfg, p)[1]), "w") for p in PROJ]
    return out


def split_storage(cfg, P):
    """Split stored [W | B] projections into P['l.w_*'] and P['l.lora_b_*'] (in place)."""
    if not lora_rank(cfg):
        return P
    for l in range(cfg["n_layers"]):
        for p in PROJ:
            k = f"l{l}.w_{p}"
            m = proj_shape(cfg, p)[1]
            if P[k].shape[1] == m:
                continue
            P[f"l{l}.lora_b_{p}"] = P[k][:, m:].copy()
            P[k] = P[k][:, :m].copy()
    return P


def storage_tensors(cfg, P):
    """The tensors of P in id order and stored shape (the inverse of split_storage)."""
    out = []
    for name, shape, _ in specs(cfg):
        a = P[name]
        if a.shape != tuple(shape) and len(shape) == 2:
            l, p = name.split(".w_")
            a = np.concatenate([a, P[f"{l}.lora_b_{p}"]], axis=1)
        out.append(a)
    return out


def round_bf16(x):
    """Round float64 values to the nearest bfloat16 (ties to even), returned as float64.

    bfloat16 keeps 8 significant bits; for normal numbers this is
    frexp-scaling the significand to [2**7, 2**8) and rounding half to even.
    """
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                 # x = m * 2**e, 0.5 <= |m| < 1
    r = np.rint(m * 256.0)             # numpy rint rounds half to even
    return np.ldexp(r, e - 8)


def round_to(x, dtype):
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "fp32":
        return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)
    raise ValueError(dtype)


def normals(seed, tensor_id, count, start=0):
    """Standard normals for elements start .. start+count-1 of one tensor (float64)."""
    return normals_at(seed, tensor_id, np.arange(start, start + count, dtype=np.uint64))


def normals_at(seed, tensor_id, idx):
    """Standard normals for the given flat element indices of one tensor (float64)."""
    e = np.asarray(idx, dtype=np.uint64)
    pair = e >> np.uint64(1)
    k0, k1 = _ph.key_of(seed)
    w0, w1, _, _ = _ph.philox(pair & np.uint64(0xFFFFFFFF), pair >> np.uint64(32),
                              np.uint64(tensor_id), np.uint64(_ph.STREAM_PARAM), k0, k1)
    return _nz.box_muller(w0, w1, (e & np.uint64(1)).astype(bool))


def values_at(cfg, seed, tensor_id, idx):
    """Initial values of selected elements of one tensor, rounded like init_params."""
    kind = specs(cfg)[tensor_id][2]
    z = normals_at(seed, tensor_id, idx)
    return round_to(0.02 * z if kind == "w" else 1.0 + 0.02 * z, cfg["dtype"])


def init_params(cfg, seed):
    """All tensors as float64 arrays holding exactly representable values of cfg['dtype']."""
    P = {}
    for tid, (name, shape, kind) in enumerate(specs(cfg)):
        z = normals(seed, tid, int(np.prod(shape))).reshape(shape)
        v = 0.02 * z if kind == "w" else 1.0 + 0.02 * z
        P[name] = round_to(v, cfg["dtype"])
    return split_storage(cfg, P)
