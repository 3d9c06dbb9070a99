"""ctypes binding of libdd.so (include/dd.h).

Argument marshalling only: every step of the reverse step runs in the HIP
library.  Device buffers are torch tensors (data_ptr + the current HIP stream);
each wrapper checks that the tensors it hands over are contiguous, on the GPU and
large enough for the sizes it passes, so the library never reads or writes
outside an allocation.  The library must have been built in-tree
(python -m paper_2609_04010_amd.build); nothing falls back to another
implementation when it is missing.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdd.so")

DD_BF16, DD_FP32 = 0, 1
DD_PRIOR_MASK, DD_PRIOR_UNIFORM = 0, 1
DD_NORM_LAYER, DD_NORM_RMS = 0, 1
DD_GUMBEL_GROUP = 256
DD_DEVERR_TOKEN = 1
DD_DEVERR_MASK = 2
DD_DEVERR_LOGITS = 4
DD_LOOP_POSTERIOR_PASS = 1
DD_LOOP_STORE_FREE = 2
ATTN_PATTERNS = {"bidirectional": 0, "causal": 1, "block_causal": 2, "draft_train": 3}
STATUS = {0: "DD_OK", 1: "DD_E_ARG", 2: "DD_E_SHAPE", 3: "DD_E_DTYPE", 4: "DD_E_WORKSPACE",
          5: "DD_E_HIP", 6: "DD_E_UNSUPPORTED", 7: "DD_E_DEVICE"}

EXPORTED = [
    "dd_param_count", "dd_param_tensor", "dd_param_bytes", "dd_workspace_bytes",
    "dd_loop_workspace_bytes", "dd_loop_workspace_layout", "dd_logits_ld", "dd_noise_width",
    "dd_status_str", "dd_last_error",
    "dd_workspace_reset", "dd_read_device_error", "dd_init_params", "dd_denoise_forward",
    "dd_attn_mask_build", "dd_denoise_forward_ex",
    "dd_posterior_sample", "dd_psi_posterior_sample", "dd_sample_loop", "dd_psi_sample_loop",
    "dd_gaussian_latent_argmax", "dd_spec_verify_workspace_bytes", "dd_spec_verify_noise_width",
    "dd_spec_verify", "dd_spec_verify_noalloc", "dd_profile_begin",
    "dd_profile_end", "dd_profile_num_classes", "dd_profile_read",
]


class DDConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("d_mlp", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("mask_id", ctypes.c_int32), ("max_len", ctypes.c_int32),
                ("prior", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("time_cond", ctypes.c_int32), ("norm", ctypes.c_int32), ("norm_eps", ctypes.c_float),
                ("lora_rank", ctypes.c_int32), ("lora_alpha", ctypes.c_float)]


class DDLoopWsLayout(ctypes.Structure):
    _fields_ = [("err", ctypes.c_size_t), ("logits", ctypes.c_size_t), ("rows", ctypes.c_size_t),
                ("count", ctypes.c_size_t), ("glse", ctypes.c_size_t), ("cand", ctypes.c_size_t),
                ("row_lse", ctypes.c_size_t),
                ("logits_ld", ctypes.c_int64), ("glse_ld", ctypes.c_int64)]


class DDError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2609_04010_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        c = ctypes
        P = c.c_void_p
        cfgp = c.POINTER(DDConfig)
        sig = {
            "dd_param_count": (c.c_int32, [cfgp]),
            "dd_param_tensor": (c.c_int32, [cfgp, c.c_int32, c.POINTER(c.c_size_t),
                                            c.POINTER(c.c_int64), c.POINTER(c.c_int64)]),
            "dd_param_bytes": (c.c_size_t, [cfgp]),
            "dd_workspace_bytes": (c.c_size_t, [cfgp, c.c_int32, c.c_int32]),
            "dd_loop_workspace_bytes": (c.c_size_t, [cfgp, c.c_int32, c.c_int32]),
            "dd_loop_workspace_layout": (c.c_int32, [cfgp, c.c_int32, c.c_int32, c.POINTER(DDLoopWsLayout)]),
            "dd_logits_ld": (c.c_int64, [c.c_int32]),
            "dd_noise_width": (c.c_int32, [c.c_int32, c.c_int32]),
            "dd_status_str": (c.c_char_p, [c.c_int32]),
            "dd_last_error": (c.c_char_p, []),
            "dd_workspace_reset": (c.c_int32, [P, P]),
            "dd_read_device_error": (c.c_int32, [P, c.POINTER(c.c_int32), P]),
            "dd_init_params": (c.c_int32, [cfgp, P, c.c_size_t, c.c_uint64, P, P]),
            "dd_denoise_forward": (c.c_int32, [cfgp, P, P, c.c_int32, c.c_int32, c.c_double, P,
                                               c.c_int64, P, c.c_size_t, P]),
            "dd_attn_mask_build": (c.c_int32, [c.c_int32, c.c_int32, c.c_int32, c.POINTER(c.c_int32)]),
            "dd_denoise_forward_ex": (c.c_int32, [cfgp, P, P, c.c_int32, c.c_int32, c.c_double, P, P,
                                                  P, c.c_int64, P, c.c_size_t, P]),
            "dd_posterior_sample": (c.c_int32, [c.c_int32, P, c.c_int32, c.c_int64, c.c_int32,
                                                c.c_int32, c.c_int32, P, c.c_double, c.c_double, P,
                                                c.c_uint64, c.c_uint32, c.c_uint32, P, P, P, P, P]),
            "dd_psi_posterior_sample": (c.c_int32, [c.c_int32, P, c.c_int32, c.c_int64, c.c_int32,
                                                    c.c_int32, c.c_int32, P, c.c_double, c.c_double,
                                                    c.c_double, P, c.c_uint64, c.c_uint32, c.c_uint32,
                                                    P, P, P, P, P]),
            "dd_sample_loop": (c.c_int32, [cfgp, P, c.c_int32, c.c_int32, c.c_int32,
                                           c.POINTER(c.c_double), P, P, c.c_uint64, P, P,
                                           c.c_size_t, P]),
            "dd_psi_sample_loop": (c.c_int32, [cfgp, P, c.c_int32, c.c_int32, c.c_int32,
                                               c.POINTER(c.c_double), c.POINTER(c.c_double), c.c_uint32,
                                               P, P, c.c_uint64, P, P, c.c_size_t, P]),
            "dd_gaussian_latent_argmax": (c.c_int32, [P, c.c_int32, c.c_int32, c.c_double,
                                                      c.c_double, c.c_uint64, c.c_uint32,
                                                      c.c_uint32, P, P, P]),
            "dd_spec_verify_workspace_bytes": (c.c_size_t, [c.c_int32, c.c_int32]),
            "dd_spec_verify_noise_width": (c.c_int32, [c.c_int32, c.c_int32]),
            "dd_spec_verify": (c.c_int32, [P, P, c.c_int32, c.c_int64, c.c_int32, c.c_int32, c.c_int32, P,
                                           P, c.c_uint64, c.c_uint32, c.c_uint32, P, P, P, c.c_size_t, P,
                                           P]),
            "dd_spec_verify_noalloc": (c.c_int32, [P, P, c.c_int32, c.c_int64, c.c_int32, c.c_int32, c.c_int32,
                                                   P, P, c.c_uint64, c.c_uint32, c.c_uint32, P, P, P, P]),
            "dd_profile_begin": (c.c_int32, [c.c_int32, c.c_uint32]),
            "dd_profile_end": (c.c_int32, []),
            "dd_profile_num_classes": (c.c_int32, []),
            "dd_profile_read": (c.c_int32, [c.c_int32, c.POINTER(c.c_char_p),
                                            c.POINTER(c.c_int64), c.POINTER(c.c_double)]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(st):
    if st != 0:
        raise DDError(st, lib().dd_last_error().decode())


def default_mask_id(prior, V):
    """The mask id a prior takes: V (the K-th category) for the masked prior, -1 for the uniform."""
    return int(V) if prior == "mask" else -1


def make_config(cfg):
    """DDConfig from the architecture dictionary used by the workloads and the oracle."""
    mid = cfg.get("mask_id", default_mask_id(cfg["prior"], cfg["vocab"]))
    return DDConfig(int(cfg["n_layers"]), int(cfg["d_model"]), int(cfg["n_heads"]),
                    int(cfg["d_mlp"]), int(cfg["vocab"]), int(mid), int(cfg["max_len"]),
                    DD_PRIOR_MASK if cfg["prior"] == "mask" else DD_PRIOR_UNIFORM,
                    DD_BF16 if cfg["dtype"] == "bf16" else DD_FP32,
                    1 if cfg.get("time_cond", True) else 0, norm_code(cfg.get("norm", "layer")),
                    float(cfg.get("norm_eps", 1e-5)),
                    int(cfg.get("lora_rank", 0) or 0), float(cfg.get("lora_alpha", 0.0) or 0.0))


def norm_code(norm):
    """dd_norm of a normalisation name: "layer" (LayerNorm) or "rms" (RMSNorm)."""
    if norm not in ("layer", "rms"):
        raise ValueError(f"unknown norm {norm!r}")
    return DD_NORM_RMS if norm == "rms" else DD_NORM_LAYER


def prior_code(prior):
    return DD_PRIOR_MASK if prior == "mask" else DD_PRIOR_UNIFORM


def dtype_code(dtype):
    return DD_BF16 if dtype == "bf16" else DD_FP32


# ---------------------------------------------------------------- host-only queries

def param_count(cfg):
    return lib().dd_param_count(ctypes.byref(make_config(cfg)))


def param_tensor(cfg, tid):
    off, r, c = ctypes.c_size_t(), ctypes.c_int64(), ctypes.c_int64()
    _check(lib().dd_param_tensor(ctypes.byref(make_config(cfg)), tid, ctypes.byref(off),
                                 ctypes.byref(r), ctypes.byref(c)))
    return off.value, r.value, c.value


def param_bytes(cfg):
    return lib().dd_param_bytes(ctypes.byref(make_config(cfg)))


def workspace_bytes(cfg, B, L):
    return lib().dd_workspace_bytes(ctypes.byref(make_config(cfg)), B, L)


def loop_workspace_bytes(cfg, B, L):
    return lib().dd_loop_workspace_bytes(ctypes.byref(make_config(cfg)), B, L)


def loop_workspace_layout(cfg, B, L):
    """dict of the loop workspace regions (byte offsets, row strides) of dd_loop_workspace_layout."""
    out = DDLoopWsLayout()
    _check(lib().dd_loop_workspace_layout(ctypes.byref(make_config(cfg)), int(B), int(L), ctypes.byref(out)))
    return {n: getattr(out, n) for n, _ in DDLoopWsLayout._fields_}


def logits_ld(V):
    return lib().dd_logits_ld(V)


def noise_width(prior, V):
    return lib().dd_noise_width(prior_code(prior), V)


def pack_params(cfg, tensors_by_id):
    """Host blob in the library's parameter layout from a list of float arrays (id order)."""
    nbytes = param_bytes(cfg)
    blob = np.zeros(nbytes, dtype=np.uint8)
    for tid, arr in enumerate(tensors_by_id):
        off, r, c = param_tensor(cfg, tid)
        a = np.asarray(arr, dtype=np.float64).reshape(-1)
        assert a.size == r * c, (tid, a.shape, r, c)
        f = a.astype(np.float32)
        if cfg["dtype"] == "bf16":
            u = f.view(np.uint32)
            if not np.array_equal(u & 0xFFFF, np.zeros_like(u)):
                raise ValueError(f"tensor {tid} is not exactly representable in bf16")
            raw = (u >> 16).astype(np.uint16).view(np.uint8)
        else:
            raw = f.view(np.uint8)
        blob[off:off + raw.size] = raw
    return blob


# ---------------------------------------------------------------- device calls

def _torch():
    import torch
    return torch


def _stream():
    return ctypes.c_void_p(_torch().cuda.current_stream().cuda_stream)


def _ptr(t, nbytes, name, dtype=None):
    """Device pointer of a contiguous GPU tensor holding at least `nbytes` bytes."""
    if t is None:
        return None
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must have dtype {dtype}, got {t.dtype}")
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{name} holds {have} bytes, needs {nbytes}")
    return ctypes.c_void_p(t.data_ptr())


def init_params(cfg, params, seed=0, host_blob=None):
    need = param_bytes(cfg)
    src = None
    if host_blob is not None:
        host_blob = np.ascontiguousarray(host_blob, dtype=np.uint8)
        if host_blob.size < need:
            raise ValueError("host blob too small")
        src = host_blob.ctypes.data_as(ctypes.c_void_p)
    _check(lib().dd_init_params(ctypes.byref(make_config(cfg)), _ptr(params, need, "params"),
                                params.numel() * params.element_size(), int(seed), src, _stream()))
    if host_blob is not None:
        _torch().cuda.current_stream().synchronize()   # the host blob must outlive the copy


def denoise_forward(cfg, params, z_t, B, L, alpha_t, logits, ld, ws):
    torch = _torch()
    es = 2 if cfg["dtype"] == "bf16" else 4
    M = B * L
    _check(lib().dd_denoise_forward(
        ctypes.byref(make_config(cfg)), _ptr(params, param_bytes(cfg), "params"),
        _ptr(z_t, 4 * M, "z_t", torch.int32), B, L, float(alpha_t),
        _ptr(logits, es * M * ld, "logits"), int(ld),
        _ptr(ws, workspace_bytes(cfg, B, L), "ws"), ws.numel() * ws.element_size(), _stream()))


def attn_mask_build(pattern, L, block=0):
    """Host int32 array [3, L] (pre, lo, hi) of a named pattern (see ATTN_PATTERNS)."""
    out = np.zeros(3 * L, dtype=np.int32)
    code = ATTN_PATTERNS[pattern] if isinstance(pattern, str) else int(pattern)
    _check(lib().dd_attn_mask_build(code, int(L), int(block),
                                    out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))))
    return out.reshape(3, L)


def denoise_forward_ex(cfg, params, z_t, B, L, alpha_t, logits, ld, ws, attn_mask=None, lora_gate=None):
    """dd_denoise_forward_ex; attn_mask is a device int32 tensor of 3 L entries, lora_gate of L."""
    torch = _torch()
    es = 2 if cfg["dtype"] == "bf16" else 4
    M = B * L
    _check(lib().dd_denoise_forward_ex(
        ctypes.byref(make_config(cfg)), _ptr(params, param_bytes(cfg), "params"),
        _ptr(z_t, 4 * M, "z_t", torch.int32), B, L, float(alpha_t),
        _ptr(attn_mask, 12 * L, "attn_mask", torch.int32) if attn_mask is not None else None,
        _ptr(lora_gate, 4 * L, "lora_gate", torch.int32) if lora_gate is not None else None,
        _ptr(logits, es * M * ld, "logits"), int(ld),
        _ptr(ws, workspace_bytes(cfg, B, L), "ws"), ws.numel() * ws.element_size(), _stream()))


def _posterior_args(prior, logits, logits_dtype, ld, rows, V, z_t, noise_words, z_s, row_lse, probs,
                    dev_err):
    torch = _torch()
    es = 2 if logits_dtype == "bf16" else 4
    K = V + 1 if prior == "mask" else V
    nu = noise_width(prior, V)
    lg = _ptr(logits, es * rows * ld, "logits") if rows > 0 else None
    return (lg, _ptr(z_t, 4 * rows, "z_t", torch.int32),
            _ptr(noise_words, 4 * rows * nu, "noise_words", torch.int32) if noise_words is not None else None,
            _ptr(z_s, 4 * rows, "z_s", torch.int32),
            _ptr(row_lse, 4 * rows, "row_lse", torch.float32) if row_lse is not None else None,
            _ptr(probs, 4 * rows * K, "probs", torch.float32) if probs is not None else None,
            _ptr(dev_err, 4, "dev_err", torch.int32) if dev_err is not None else None)


def posterior_sample(prior, logits, logits_dtype, ld, rows, V, z_t, alpha_t, alpha_s, z_s,
                     noise_words=None, seed=0, step=0, row0=0, probs=None, dev_err=None, row_lse=None,
                     mask_id=None):
    """dd_posterior_sample; mask_id defaults to the prior's (V for "mask", -1 for "uniform")."""
    lg, zt, nw, zs, rl, pr, er = _posterior_args(prior, logits, logits_dtype, ld, rows, V, z_t, noise_words,
                                                 z_s, row_lse, probs, dev_err)
    mid = default_mask_id(prior, V) if mask_id is None else int(mask_id)
    _check(lib().dd_posterior_sample(
        prior_code(prior), lg, dtype_code(logits_dtype), int(ld), int(rows), int(V), mid, zt, float(alpha_t),
        float(alpha_s), nw, int(seed) & 0xFFFFFFFFFFFFFFFF, int(step), int(row0), zs, rl, pr, er, _stream()))


def psi_posterior_sample(prior, logits, logits_dtype, ld, rows, V, z_t, alpha_t, alpha_s, kappa, z_s,
                         noise_words=None, seed=0, step=0, row0=0, probs=None, dev_err=None, row_lse=None,
                         mask_id=None):
    lg, zt, nw, zs, rl, pr, er = _posterior_args(prior, logits, logits_dtype, ld, rows, V, z_t, noise_words,
                                                 z_s, row_lse, probs, dev_err)
    mid = default_mask_id(prior, V) if mask_id is None else int(mask_id)
    _check(lib().dd_psi_posterior_sample(
        prior_code(prior), lg, dtype_code(logits_dtype), int(ld), int(rows), int(V), mid, zt, float(alpha_t),
        float(alpha_s), float(kappa), nw, int(seed) & 0xFFFFFFFFFFFFFFFF, int(step), int(row0), zs, rl, pr, er,
        _stream()))


def sample_loop(cfg, params, B, L, T, alphas, z, ws, noise_words=None, noise_seed=0, z_trace=None,
                kappas=None, posterior_pass=False, store_free=False):
    """dd_sample_loop, or dd_psi_sample_loop when kappas (T + 1 values) is given or a flag is set:
    posterior_pass (DD_LOOP_POSTERIOR_PASS), store_free (DD_LOOP_STORE_FREE)."""
    torch = _torch()
    M = B * L
    a = np.ascontiguousarray(alphas, dtype=np.float64)
    if a.shape != (T + 1,):
        raise ValueError("alphas must hold T + 1 values")
    nu = noise_width(cfg["prior"], cfg["vocab"])
    dp = ctypes.POINTER(ctypes.c_double)
    head = (ctypes.byref(make_config(cfg)), _ptr(params, param_bytes(cfg), "params"), B, L, T, a.ctypes.data_as(dp))
    tail = (_ptr(z, 4 * M, "z", torch.int32),
            _ptr(noise_words, 4 * T * M * nu, "noise_words", torch.int32) if noise_words is not None else None,
            int(noise_seed) & 0xFFFFFFFFFFFFFFFF,
            _ptr(z_trace, 4 * (T + 1) * M, "z_trace", torch.int32) if z_trace is not None else None,
            _ptr(ws, loop_workspace_bytes(cfg, B, L), "ws"), ws.numel() * ws.element_size(), _stream())
    if kappas is None and not posterior_pass and not store_free:
        _check(lib().dd_sample_loop(*head, *tail))
    else:
        k = None
        if kappas is not None:
            k = np.ascontiguousarray(kappas, dtype=np.float64)
            if k.shape != (T + 1,):
                raise ValueError("kappas must hold T + 1 values")
        flags = (DD_LOOP_POSTERIOR_PASS if posterior_pass else 0) | (DD_LOOP_STORE_FREE if store_free else 0)
        _check(lib().dd_psi_sample_loop(*head, k.ctypes.data_as(dp) if k is not None else None, flags, *tail))


def spec_verify_workspace_bytes(S, B):
    return int(lib().dd_spec_verify_workspace_bytes(int(S), int(B)))


def spec_verify_noise_width(B, V):
    return int(lib().dd_spec_verify_noise_width(int(B), int(V)))


def spec_verify(p_logits, q_logits, logits_dtype, ld, S, B, V, draft, n_out, z_out, ws, noise_words=None,
                seed=0, step=0, row0=0, dev_err=None):
    torch = _torch()
    es = 2 if logits_dtype == "bf16" else 4
    nu = spec_verify_noise_width(B, V)
    _check(lib().dd_spec_verify(
        _ptr(p_logits, es * S * B * ld, "p_logits"),
        _ptr(q_logits, es * S * (B - 1) * ld, "q_logits") if B > 1 else None, dtype_code(logits_dtype),
        int(ld), int(S), int(B), int(V),
        _ptr(draft, 4 * S * (B - 1), "draft", torch.int32) if B > 1 else None,
        _ptr(noise_words, 4 * S * nu, "noise_words", torch.int32) if noise_words is not None else None,
        int(seed) & 0xFFFFFFFFFFFFFFFF, int(step), int(row0), _ptr(n_out, 4 * S, "n_out", torch.int32),
        _ptr(z_out, 4 * S, "z_out", torch.int32), _ptr(ws, spec_verify_workspace_bytes(S, B), "ws"),
        ws.numel() * ws.element_size(), _ptr(dev_err, 4, "dev_err", torch.int32) if dev_err is not None else None,
        _stream()))


SPEC_VERIFY_NOALLOC_ROWS = 1 << 18


def spec_verify_noalloc(p_logits, q_logits, logits_dtype, ld, S, B, V, draft, n_out, z_out, noise_words=None,
                        seed=0, step=0, row0=0, dev_err=None):
    """dd_spec_verify_noalloc: dd_spec_verify without a workspace (library-held device array)."""
    torch = _torch()
    es = 2 if logits_dtype == "bf16" else 4
    nu = spec_verify_noise_width(B, V)
    _check(lib().dd_spec_verify_noalloc(
        _ptr(p_logits, es * S * B * ld, "p_logits"),
        _ptr(q_logits, es * S * (B - 1) * ld, "q_logits") if B > 1 else None, dtype_code(logits_dtype),
        int(ld), int(S), int(B), int(V),
        _ptr(draft, 4 * S * (B - 1), "draft", torch.int32) if B > 1 else None,
        _ptr(noise_words, 4 * S * nu, "noise_words", torch.int32) if noise_words is not None else None,
        int(seed) & 0xFFFFFFFFFFFFFFFF, int(step), int(row0), _ptr(n_out, 4 * S, "n_out", torch.int32),
        _ptr(z_out, 4 * S, "z_out", torch.int32),
        _ptr(dev_err, 4, "dev_err", torch.int32) if dev_err is not None else None, _stream()))


def gaussian_latent_argmax(x, rows, V, alpha_tilde, sigma, seed, step, z_out, row0=0, dev_err=None):
    torch = _torch()
    _check(lib().dd_gaussian_latent_argmax(
        _ptr(x, 4 * rows, "x", torch.int32), int(rows), int(V), float(alpha_tilde), float(sigma),
        int(seed) & 0xFFFFFFFFFFFFFFFF, int(step), int(row0), _ptr(z_out, 4 * rows, "z_out", torch.int32),
        _ptr(dev_err, 4, "dev_err", torch.int32) if dev_err is not None else None, _stream()))


def workspace_reset(ws):
    _check(lib().dd_workspace_reset(_ptr(ws, 4, "ws"), _stream()))


def read_device_error(err):
    code = ctypes.c_int32(0)
    st = lib().dd_read_device_error(_ptr(err, 4, "err"), ctypes.byref(code), _stream())
    if st not in (0, 7):
        _check(st)
    return code.value


PROFILE_CLASSES = ["time_embedding", "embed_layernorm", "layernorm", "gemm_qkv", "attention",
                   "gemm_attn_out", "gemm_mlp_up", "gemm_mlp_down", "gemm_vocab",
                   "posterior_sample", "gaussian_latent", "init_params", "copy", "compact_masked",
                   "gemm_lora_down"]


def profile_begin(max_launches, classes=None):
    """Start event timing; `classes` is a list of class names (None: every class)."""
    mask = 0
    for name in classes or []:
        mask |= 1 << PROFILE_CLASSES.index(name)
    _check(lib().dd_profile_begin(int(max_launches), mask))


def profile_end():
    _check(lib().dd_profile_end())


def profile_read():
    """{class name: (launches, total ms)} for every class with at least one launch."""
    out = {}
    for c in range(lib().dd_profile_num_classes()):
        name, n, ms = ctypes.c_char_p(), ctypes.c_int64(), ctypes.c_double()
        _check(lib().dd_profile_read(c, ctypes.byref(name), ctypes.byref(n), ctypes.byref(ms)))
        if n.value:
            out[name.value.decode()] = (n.value, ms.value)
    return out
