"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module holds shapes and seeded random inputs only (numpy's PCG64 via
default_rng): token ids, masked states, synthetic logits, explicit noise
words and host parameter tensors.  It contains none of the method's
arithmetic; it is imported by both sides of every parity check and by
neither implementation.

Workload recipe (the paper's own workloads need its datasets and trained
weights, which are absent; its throughput test feeds uniformly random input
tokens, so token ids here are i.i.d. uniform over the V real tokens):

  1 tiny-mask-fp32      2 layers, d 64, 2 heads, MLP 256, V 32 + mask, L 32,
                        B 4, fp32, T 8, all-mask start, explicit noise words
  2 gpt2s-mask          12 layers, d 768, 12 heads, MLP 3072, V 50257 + mask,
                        L 1024, B 16, bf16, T 128, all-mask start, Philox noise
  3 gpt2s-uniform       as 2 with the uniform prior (K = V), T 64, start
                        z_1 = Gaussian-latent argmax at alpha_tilde = 0
  4 gpt2s-mask-b128     as 2 with B 128, T 8
  5 l24d1024-mask       24 layers, d 1024, 16 heads, MLP 4096, L 4096, B 8, T 256

Seeds for workload c: params 1000 + c, data 2000 + c, noise 3000 + c.
"""
import numpy as np

WORKLOADS = {
    1: dict(name="tiny-mask-fp32", n_layers=2, d_model=64, n_heads=2, d_mlp=256, vocab=32,
            prior="mask", B=4, L=32, T=8, dtype="fp32", noise="explicit"),
    2: dict(name="gpt2s-mask-bf16", n_layers=12, d_model=768, n_heads=12, d_mlp=3072, vocab=50257,
            prior="mask", B=16, L=1024, T=128, dtype="bf16", noise="philox"),
    3: dict(name="gpt2s-uniform-bf16", n_layers=12, d_model=768, n_heads=12, d_mlp=3072, vocab=50257,
            prior="uniform", B=16, L=1024, T=64, dtype="bf16", noise="philox"),
    4: dict(name="gpt2s-mask-b128-bf16", n_layers=12, d_model=768, n_heads=12, d_mlp=3072, vocab=50257,
            prior="mask", B=128, L=1024, T=8, dtype="bf16", noise="philox"),
    5: dict(name="l24d1024-mask-bf16", n_layers=24, d_model=1024, n_heads=16, d_mlp=4096, vocab=50257,
            prior="mask", B=8, L=4096, T=256, dtype="bf16", noise="philox"),
}


def model_cfg(c, **over):
    """Architecture dictionary for workload c (keys the oracle and binding read)."""
    w = dict(WORKLOADS[c])
    cfg = dict(n_layers=w["n_layers"], d_model=w["d_model"], n_heads=w["n_heads"],
               d_mlp=w["d_mlp"], vocab=w["vocab"], prior=w["prior"], dtype=w["dtype"],
               max_len=w["L"], time_cond=True, norm_eps=1e-5)
    cfg.update(over)
    return cfg


def seeds(c):
    return dict(param=1000 + c, data=2000 + c, noise=3000 + c)


def rng(seed):
    return np.random.default_rng(seed)


def clean_tokens(seed, B, L, V):
    """i.i.d. uniform token ids in [0, V)."""
    return rng(seed).integers(0, V, size=(B, L), dtype=np.int64).astype(np.int32)


def masked_state(seed, B, L, V, mask_frac):
    """Uniform clean tokens with each position replaced by the mask id V w.p. mask_frac."""
    r = rng(seed)
    x = r.integers(0, V, size=(B, L), dtype=np.int64)
    m = r.random((B, L)) < mask_frac
    return np.where(m, V, x).astype(np.int32)


def all_mask(B, L, V):
    return np.full((B, L), V, dtype=np.int32)


def uniform_state(seed, B, L, V):
    return clean_tokens(seed, B, L, V)


def synthetic_logits(seed, R, V, scale=2.0, spike_frac=0.0, spike=12.0):
    """Logits [R, V] ~ scale * N(0, 1); optionally a few large spikes per row so that
    posteriors are peaked as well as flat."""
    r = rng(seed)
    l = scale * r.standard_normal((R, V))
    if spike_frac > 0:
        hit = r.random((R, V)) < spike_frac
        l = np.where(hit, l + spike, l)
    return l


def noise_words(seed, shape):
    """Explicit uniform noise as raw 32-bit words."""
    return rng(seed).integers(0, 2 ** 32, size=shape, dtype=np.uint64).astype(np.uint32)


def host_params(cfg, seed, specs):
    """Host parameter tensors ~ N(0, 0.02) (gains 1 + N(0, 0.02)) rounded to cfg['dtype'].

    `specs` is the (name, shape, kind) list; rounding uses numpy's float32 cast
    (round to nearest even) and, for bf16, a second round-to-nearest-even of
    the float32 bit pattern to 8 significant bits.
    """
    r = rng(seed)
    out = {}
    for name, shape, kind in specs:
        v = 0.02 * r.standard_normal(shape)
        if kind == "gain":
            v = v + 1.0
        f = v.astype(np.float32)
        if cfg["dtype"] == "bf16":
            b = f.view(np.uint32).astype(np.uint64)
            b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16 << 16
            f = b.astype(np.uint32).view(np.float32)
        out[name] = f.astype(np.float64)
    return out
