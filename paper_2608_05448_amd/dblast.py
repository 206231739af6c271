"""Python binding of libdblast.so: the C ABI of include/dblast.h, with the same names.

Argument marshalling only: tensors are checked for device, dtype, layout and shape, their
device pointers and the current HIP stream are passed to the library, and a workspace tensor
is allocated when the call needs one. Every step of the computation runs in the library's
kernels. There is no fallback: if the library is not built or no GPU is visible, calls raise.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdblast.so")

DBL_OK, DBL_EINVAL, DBL_ESHAPE, DBL_EDTYPE, DBL_EWORKSPACE, DBL_EHIP = range(6)
DBL_F32, DBL_BF16 = 0, 1
(DBL_OP_HEAD, DBL_OP_SAMPLE, DBL_OP_VERIFY, DBL_OP_EXPECTED_LEN, DBL_OP_SAMPLE_GREEDY,
 DBL_OP_VERIFY_GREEDY, DBL_OP_EXPECTED_LEN_GREEDY, DBL_OP_TARGET) = range(8)
VTILE = 128


class Shape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int64), ("K", ctypes.c_int64), ("R", ctypes.c_int64),
                ("d", ctypes.c_int64), ("V", ctypes.c_int64)]


class DblastError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


_lib = None
_P = ctypes.c_void_p
_F = ctypes.c_float
_I64 = ctypes.c_int64
_U64 = ctypes.c_uint64
_SZ = ctypes.c_size_t

_SIGS = {
    "dbl_vtile": (ctypes.c_int, []),
    "dbl_ntiles": (_I64, [_I64]),
    "dbl_workspace_bytes": (_SZ, [ctypes.c_int, Shape]),
    "dbl_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "dbl_last_error": (ctypes.c_char_p, []),
    "dbl_head_logprobs": (ctypes.c_int, [Shape, ctypes.c_int, _P, _P, _P, _P, _P, _P, _P, _SZ,
                                         _P]),
    "dbl_sample_block": (ctypes.c_int, [Shape, _P, _P, _P, _P, _F, _U64, _U64, _I64, _P, _P, _P,
                                        _SZ, _P]),
    "dbl_verify_block": (ctypes.c_int, [Shape, _P, _P, _P, _P, _F, _P, _P, _I64, _U64, _U64, _I64,
                                        _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "dbl_verify_block_static": (ctypes.c_int, [Shape, _P, _P, _P, _P, _F, _P, _P, _I64, _U64,
                                               _U64, _I64, _P, _P, _P, _P, _P, _P]),
    "dbl_expected_len": (ctypes.c_int, [Shape, _P, _P, _P, _P, _F, _P, _P, _P, _P, _P, _SZ, _P]),
    "dbl_sample_greedy": (ctypes.c_int, [Shape, _P, _P, _F, _U64, _U64, _I64, _P, _P, _P]),
    "dbl_verify_greedy": (ctypes.c_int, [Shape, _P, _P, _F, _P, _P, _I64, _U64, _U64, _I64, _P,
                                         _P, _P, _P, _P, _P, _SZ, _P]),
    "dbl_expected_len_greedy": (ctypes.c_int, [Shape, _P, _P, _F, _P, _P, _P, _P, _P, _SZ, _P]),
    "dbl_acceptance_objective": (ctypes.c_int, [Shape, _P, _P, _P, _P, _F, _P, _P, _F, _P, _P,
                                                _P, _P, _P, _P]),
    "dbl_expand_branches": (ctypes.c_int, [Shape, _P, _P, _P, _P, _P]),
    "dbl_prior_head": (ctypes.c_int, [Shape, _P, _P, _P, _P, _P]),
    "dbl_target_logprobs": (ctypes.c_int, [_I64, _I64, _P, _F, _I64, _F, _P, _P, _SZ, _P]),
    "dbl_early_determinism": (ctypes.c_int, [_I64, _I64, _I64, _P, _P, _P, _P, _P]),
    "dbl_stream_read_probe": (ctypes.c_int, [_P, _I64, _P, _I64, _P]),
}
EXPORTED = tuple(_SIGS)


def load(path: str = LIB_PATH):
    """Load libdblast.so (once). Raises if it is missing: there is no other implementation."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run `python -m paper_2608_05448_amd.build` "
                           "(the DBLast path has no CPU or PyTorch fallback)")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int):
    if status != DBL_OK:
        lib = load()
        raise DblastError(status, lib.dbl_last_error().decode() or
                          lib.dbl_status_string(status).decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _need(t, name, dtype, shape=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def ntiles(V: int) -> int:
    return (V + VTILE - 1) // VTILE


def dbl_workspace_bytes(op: int, B: int, K: int, R: int, d: int, V: int) -> int:
    return int(load().dbl_workspace_bytes(op, Shape(B, K, R, d, V)))


def _workspace(op, shape, device, ws=None):
    n = int(load().dbl_workspace_bytes(op, shape))
    if n == 0:
        return None, 0
    if ws is not None:
        if ws.numel() * ws.element_size() < n:
            raise ValueError(f"workspace needs {n} bytes")
        return ws, ws.numel() * ws.element_size()
    return torch.empty(n, dtype=torch.uint8, device=device), n


def dbl_head_logprobs(h, w, tls=None, lmass=None, lse=None, argmax=None, ws=None):
    """Branch log-probabilities for h [B, K, R, d] and w [V, d] (bf16 or fp32).

    Returns (tls [B, K, R, V], lmass [B, K, R, nT], lse [B, K, R]) fp32 on the device; with
    ``argmax`` (True, or an int32 [B, K, R] tensor to fill) also the per-row argmax (the greedy
    branch tokens) as a fourth element.
    """
    if h.dtype not in (torch.bfloat16, torch.float32):
        raise TypeError("h must be bfloat16 or float32")
    B, K, R, d = h.shape
    V = w.shape[0]
    _need(h, "h", h.dtype)
    _need(w, "w", h.dtype, (V, d))
    dev = h.device
    nT = ntiles(V)
    tls = torch.empty((B, K, R, V), dtype=torch.float32, device=dev) if tls is None else tls
    lmass = torch.empty((B, K, R, nT), dtype=torch.float32, device=dev) if lmass is None else lmass
    lse = torch.empty((B, K, R), dtype=torch.float32, device=dev) if lse is None else lse
    _need(tls, "tls", torch.float32, (B, K, R, V))
    _need(lmass, "lmass", torch.float32, (B, K, R, nT))
    _need(lse, "lse", torch.float32, (B, K, R))
    shape = Shape(B, K, R, d, V)
    want_arg = argmax is not None and argmax is not False
    if want_arg:
        if argmax is True:
            argmax = torch.empty((B, K, R), dtype=torch.int32, device=dev)
        _need(argmax, "argmax", torch.int32, (B, K, R))
        ws, nws = _workspace(DBL_OP_HEAD, shape, dev, ws)
    else:
        argmax, ws, nws = None, None, 0
    dt = DBL_BF16 if h.dtype == torch.bfloat16 else DBL_F32
    _check(load().dbl_head_logprobs(shape, dt, _ptr(h), _ptr(w), _ptr(tls), _ptr(lmass),
                                    _ptr(lse), _ptr(argmax), _ptr(ws), nws, _stream(dev)))
    return (tls, lmass, lse, argmax) if want_arg else (tls, lmass, lse)


def _block_shape(tls, lmass, lse, prior_logits):
    B, K, R, V = tls.shape
    _need(tls, "tls", torch.float32)
    _need(lmass, "lmass", torch.float32, (B, K, R, ntiles(V)))
    _need(lse, "lse", torch.float32, (B, K, R))
    _need(prior_logits, "prior_logits", torch.float32, (B, R))
    return Shape(B, K, R, 0, V)


def dbl_sample_block(tls, lmass, lse, prior_logits, z_temp=1.0, seed=0, step=0, seq_offset=0,
                     z_out=None, x_out=None, ws=None):
    """Draw one block per sequence: returns (z [B] int32, x [B, K] int32)."""
    shape = _block_shape(tls, lmass, lse, prior_logits)
    dev = tls.device
    z_out = torch.empty(shape.B, dtype=torch.int32, device=dev) if z_out is None else z_out
    x_out = torch.empty((shape.B, shape.K), dtype=torch.int32, device=dev) if x_out is None else x_out
    _need(z_out, "z_out", torch.int32, (shape.B,))
    _need(x_out, "x_out", torch.int32, (shape.B, shape.K))
    ws, nws = _workspace(DBL_OP_SAMPLE, shape, dev, ws)
    _check(load().dbl_sample_block(shape, _ptr(tls), _ptr(lmass), _ptr(lse), _ptr(prior_logits),
                                   float(z_temp), int(seed), int(step), int(seq_offset),
                                   _ptr(z_out), _ptr(x_out), _ptr(ws), nws, _stream(dev)))
    return z_out, x_out


def dbl_verify_block(tls, lmass, lse, prior_logits, x, logp, z_temp=1.0, seed=0, step=0,
                     seq_offset=0, want_beta=True, want_al=True, want_exp_len=True, out=None,
                     ws=None):
    """Verify drafted blocks x [B, K] against target log-probs logp [B, Kp, V].

    Returns a dict with n_accept [B], next_token [B] and, as requested, accept_mass [B, K],
    al_expected [B], exp_len [B].
    """
    shape = _block_shape(tls, lmass, lse, prior_logits)
    dev = tls.device
    B, K, V = shape.B, shape.K, shape.V
    _need(x, "x", torch.int32, (B, K))
    if logp.dim() != 3 or logp.shape[0] != B or logp.shape[2] != V:
        raise ValueError("logp must be [B, Kp, V]")
    _need(logp, "logp", torch.float32)
    Kp = logp.shape[1]
    o = {} if out is None else dict(out)
    o.setdefault("n_accept", torch.empty(B, dtype=torch.int32, device=dev))
    o.setdefault("next_token", torch.empty(B, dtype=torch.int32, device=dev))
    if want_beta:
        o.setdefault("accept_mass", torch.empty((B, K), dtype=torch.float32, device=dev))
    if want_al:
        o.setdefault("al_expected", torch.empty(B, dtype=torch.float32, device=dev))
    if want_exp_len:
        o.setdefault("exp_len", torch.empty(B, dtype=torch.float32, device=dev))
    ws, nws = _workspace(DBL_OP_VERIFY, shape, dev, ws)
    _check(load().dbl_verify_block(shape, _ptr(tls), _ptr(lmass), _ptr(lse), _ptr(prior_logits),
                                   float(z_temp), _ptr(x), _ptr(logp), int(Kp), int(seed),
                                   int(step), int(seq_offset), _ptr(o["n_accept"]),
                                   _ptr(o["next_token"]), _ptr(o.get("accept_mass")),
                                   _ptr(o.get("al_expected")), _ptr(o.get("exp_len")), _ptr(ws),
                                   nws, _stream(dev)))
    return o


def dbl_verify_block_static(tls, lmass, lse, prior_logits, x, logp, z_temp=1.0, seed=0, step=0,
                            seq_offset=0, want_beta=True, want_al=True, want_exp_len=True,
                            out=None):
    """``dbl_verify_block`` without a workspace: the library's fixed per-GPU scratch is used
    (shapes needing more than 8 MiB of it are rejected). Calls that overlap on one GPU race."""
    shape = _block_shape(tls, lmass, lse, prior_logits)
    dev = tls.device
    B, K, V = shape.B, shape.K, shape.V
    _need(x, "x", torch.int32, (B, K))
    if logp.dim() != 3 or logp.shape[0] != B or logp.shape[2] != V:
        raise ValueError("logp must be [B, Kp, V]")
    _need(logp, "logp", torch.float32)
    Kp = logp.shape[1]
    o = {} if out is None else dict(out)
    o.setdefault("n_accept", torch.empty(B, dtype=torch.int32, device=dev))
    o.setdefault("next_token", torch.empty(B, dtype=torch.int32, device=dev))
    if want_beta:
        o.setdefault("accept_mass", torch.empty((B, K), dtype=torch.float32, device=dev))
    if want_al:
        o.setdefault("al_expected", torch.empty(B, dtype=torch.float32, device=dev))
    if want_exp_len:
        o.setdefault("exp_len", torch.empty(B, dtype=torch.float32, device=dev))
    _check(load().dbl_verify_block_static(shape, _ptr(tls), _ptr(lmass), _ptr(lse),
                                          _ptr(prior_logits), float(z_temp), _ptr(x), _ptr(logp),
                                          int(Kp), int(seed), int(step), int(seq_offset),
                                          _ptr(o["n_accept"]), _ptr(o["next_token"]),
                                          _ptr(o.get("accept_mass")), _ptr(o.get("al_expected")),
                                          _ptr(o.get("exp_len")), _stream(dev)))
    return o


def dbl_expected_len(tls, lmass, lse, prior_logits, x, logp, z_temp=1.0, want_beta=True,
                     beta=None, exp_len=None, ws=None):
    """Acceptance masses and expected accepted length along trajectories x [B, K]."""
    shape = _block_shape(tls, lmass, lse, prior_logits)
    dev = tls.device
    B, K, V = shape.B, shape.K, shape.V
    _need(x, "x", torch.int32, (B, K))
    _need(logp, "logp", torch.float32, (B, K, V))
    if want_beta and beta is None:
        beta = torch.empty((B, K), dtype=torch.float32, device=dev)
    exp_len = torch.empty(B, dtype=torch.float32, device=dev) if exp_len is None else exp_len
    ws, nws = _workspace(DBL_OP_EXPECTED_LEN, shape, dev, ws)
    _check(load().dbl_expected_len(shape, _ptr(tls), _ptr(lmass), _ptr(lse), _ptr(prior_logits),
                                   float(z_temp), _ptr(x), _ptr(logp), _ptr(beta), _ptr(exp_len),
                                   _ptr(ws), nws, _stream(dev)))
    return beta, exp_len


def _greedy_shape(x_hat, prior_logits, V):
    B, K, R = x_hat.shape
    _need(x_hat, "x_hat", torch.int32)
    _need(prior_logits, "prior_logits", torch.float32, (B, R))
    return Shape(B, K, R, 0, int(V))


def dbl_sample_greedy(x_hat, prior_logits, z_temp=1.0, seed=0, step=0, seq_offset=0, V=1,
                      z_out=None, x_out=None):
    """Greedy-branch draw from branch tokens x_hat [B, K, R]: returns (z [B], x [B, K]) int32.
    ``V`` is only used for shape validation (the draw reads no vocabulary row)."""
    shape = _greedy_shape(x_hat, prior_logits, V)
    dev = x_hat.device
    z_out = torch.empty(shape.B, dtype=torch.int32, device=dev) if z_out is None else z_out
    x_out = torch.empty((shape.B, shape.K), dtype=torch.int32, device=dev) if x_out is None else x_out
    _need(z_out, "z_out", torch.int32, (shape.B,))
    _need(x_out, "x_out", torch.int32, (shape.B, shape.K))
    _check(load().dbl_sample_greedy(shape, _ptr(x_hat), _ptr(prior_logits), float(z_temp),
                                    int(seed), int(step), int(seq_offset), _ptr(z_out),
                                    _ptr(x_out), _stream(dev)))
    return z_out, x_out


def dbl_verify_greedy(x_hat, prior_logits, x, logp, z_temp=1.0, seed=0, step=0, seq_offset=0,
                      want_beta=True, want_al=True, want_exp_len=True, out=None, ws=None):
    """Verify drafted blocks x [B, K] against logp [B, Kp, V] with the greedy-branch conditional
    of branch tokens x_hat [B, K, R]; returns the same dict as ``dbl_verify_block``."""
    if logp.dim() != 3:
        raise ValueError("logp must be [B, Kp, V]")
    shape = _greedy_shape(x_hat, prior_logits, logp.shape[2])
    dev = x_hat.device
    B, K = shape.B, shape.K
    _need(x, "x", torch.int32, (B, K))
    if logp.shape[0] != B:
        raise ValueError("logp must be [B, Kp, V]")
    _need(logp, "logp", torch.float32)
    Kp = logp.shape[1]
    o = {} if out is None else dict(out)
    o.setdefault("n_accept", torch.empty(B, dtype=torch.int32, device=dev))
    o.setdefault("next_token", torch.empty(B, dtype=torch.int32, device=dev))
    if want_beta:
        o.setdefault("accept_mass", torch.empty((B, K), dtype=torch.float32, device=dev))
    if want_al:
        o.setdefault("al_expected", torch.empty(B, dtype=torch.float32, device=dev))
    if want_exp_len:
        o.setdefault("exp_len", torch.empty(B, dtype=torch.float32, device=dev))
    ws, nws = _workspace(DBL_OP_VERIFY_GREEDY, shape, dev, ws)
    _check(load().dbl_verify_greedy(shape, _ptr(x_hat), _ptr(prior_logits), float(z_temp),
                                    _ptr(x), _ptr(logp), int(Kp), int(seed), int(step),
                                    int(seq_offset), _ptr(o["n_accept"]), _ptr(o["next_token"]),
                                    _ptr(o.get("accept_mass")), _ptr(o.get("al_expected")),
                                    _ptr(o.get("exp_len")), _ptr(ws), nws, _stream(dev)))
    return o


def dbl_expected_len_greedy(x_hat, prior_logits, x, logp, z_temp=1.0, want_beta=True, beta=None,
                            exp_len=None, ws=None):
    """Acceptance masses and expected accepted length along trajectories x [B, K] under the
    greedy-branch conditional of x_hat [B, K, R]."""
    shape = _greedy_shape(x_hat, prior_logits, logp.shape[-1])
    dev = x_hat.device
    B, K, V = shape.B, shape.K, shape.V
    _need(x, "x", torch.int32, (B, K))
    _need(logp, "logp", torch.float32, (B, K, V))
    if want_beta and beta is None:
        beta = torch.empty((B, K), dtype=torch.float32, device=dev)
    exp_len = torch.empty(B, dtype=torch.float32, device=dev) if exp_len is None else exp_len
    ws, nws = _workspace(DBL_OP_EXPECTED_LEN_GREEDY, shape, dev, ws)
    _check(load().dbl_expected_len_greedy(shape, _ptr(x_hat), _ptr(prior_logits), float(z_temp),
                                          _ptr(x), _ptr(logp), _ptr(beta), _ptr(exp_len),
                                          _ptr(ws), nws, _stream(dev)))
    return beta, exp_len


def dbl_acceptance_objective(tls, lmass, lse, prior_logits, x, logp, z_temp=1.0, tau=0.1,
                             want_terms=True, out=None):
    """Training-surrogate forward along target trajectories x [B, K] with target log-probs
    logp [B, K, V]: returns a dict with ell_tau [B] int32, J [B], nll [B] and, with
    ``want_terms``, log_r [B, K] and S [B, K] (fp32)."""
    shape = _block_shape(tls, lmass, lse, prior_logits)
    dev = tls.device
    B, K, V = shape.B, shape.K, shape.V
    _need(x, "x", torch.int32, (B, K))
    _need(logp, "logp", torch.float32, (B, K, V))
    o = {} if out is None else dict(out)
    o.setdefault("ell_tau", torch.empty(B, dtype=torch.int32, device=dev))
    o.setdefault("J", torch.empty(B, dtype=torch.float32, device=dev))
    o.setdefault("nll", torch.empty(B, dtype=torch.float32, device=dev))
    if want_terms:
        o.setdefault("log_r", torch.empty((B, K), dtype=torch.float32, device=dev))
        o.setdefault("S", torch.empty((B, K), dtype=torch.float32, device=dev))
    _check(load().dbl_acceptance_objective(shape, _ptr(tls), _ptr(lmass), _ptr(lse),
                                           _ptr(prior_logits), float(z_temp), _ptr(x),
                                           _ptr(logp), float(tau), _ptr(o.get("log_r")),
                                           _ptr(o.get("S")), _ptr(o["ell_tau"]), _ptr(o["J"]),
                                           _ptr(o["nll"]), _stream(dev)))
    return o


def dbl_expand_branches(h, W, c, R, out=None):
    """Branch states h_{k,z} = h_k + W_z h_k + c_z: h [B, K, d] bf16, W [R*d, d], c [R*d] bf16.
    Returns [B, K, R, d] bf16 (the head's input)."""
    B, K, d = h.shape
    _need(h, "h", torch.bfloat16)
    _need(W, "W", torch.bfloat16, (R * d, d))
    _need(c, "c", torch.bfloat16, (R * d,))
    dev = h.device
    out = torch.empty((B, K, R, d), dtype=torch.bfloat16, device=dev) if out is None else out
    _need(out, "out", torch.bfloat16, (B, K, R, d))
    _check(load().dbl_expand_branches(Shape(B, K, R, d, 1), _ptr(h), _ptr(W), _ptr(c), _ptr(out),
                                      _stream(dev)))
    return out


def dbl_prior_head(h_anchor, U, e, out=None):
    """Category logits l = U h_anchor + e: h_anchor [B, d], U [R, d], e [R] bf16 -> [B, R] fp32."""
    B, d = h_anchor.shape
    R = U.shape[0]
    _need(h_anchor, "h_anchor", torch.bfloat16)
    _need(U, "U", torch.bfloat16, (R, d))
    _need(e, "e", torch.bfloat16, (R,))
    dev = h_anchor.device
    out = torch.empty((B, R), dtype=torch.float32, device=dev) if out is None else out
    _need(out, "out", torch.float32, (B, R))
    _check(load().dbl_prior_head(Shape(B, 1, R, d, 1), _ptr(h_anchor), _ptr(U), _ptr(e),
                                 _ptr(out), _stream(dev)))
    return out


def dbl_target_logprobs(logits, temperature=1.0, top_k=0, top_p=1.0, out=None, ws=None,
                        split=True):
    """Target sampling log-probabilities for logits [..., V] fp32 (temperature, top-k, top-p).
    ``out`` must not overlap ``logits``. With ``split`` (default) a workspace (``ws`` or a new
    one) lets rows be split over several workgroups; the result is the same either way."""
    _need(logits, "logits", torch.float32)
    V = logits.shape[-1]
    N = logits.numel() // V
    out = torch.empty_like(logits) if out is None else out
    _need(out, "out", torch.float32, tuple(logits.shape))
    if split:
        ws, nws = _workspace(DBL_OP_TARGET, Shape(N, 1, 1, 0, V), logits.device, ws)
    else:
        ws, nws = None, 0
    _check(load().dbl_target_logprobs(N, V, _ptr(logits), float(temperature), int(top_k),
                                      float(top_p), _ptr(out), _ptr(ws), nws,
                                      _stream(logits.device)))
    return out


def dbl_early_determinism(x, logp):
    """Early-determinism estimate from sampled target blocks x [M, b] and their target
    log-probs logp [M, b, V]: returns (terms [M], mean [] ) fp32 tensors."""
    M, b = x.shape
    _need(x, "x", torch.int32)
    _need(logp, "logp", torch.float32, (M, b, logp.shape[-1]))
    dev = x.device
    terms = torch.empty(M, dtype=torch.float32, device=dev)
    mean = torch.empty((), dtype=torch.float32, device=dev)
    _check(load().dbl_early_determinism(M, b, logp.shape[-1], _ptr(x), _ptr(logp), _ptr(terms),
                                        _ptr(mean), _stream(dev)))
    return terms, mean


def dbl_stream_read_probe(buf, partials):
    """Diagnostic: read every 16-byte word of ``buf`` once (one workgroup per element of
    ``partials``, fp32 [n]); each writes the sum of the values it read. Returns ``partials``."""
    _need(buf, "buf", buf.dtype)
    _need(partials, "partials", torch.float32)
    nbytes = buf.numel() * buf.element_size()
    _check(load().dbl_stream_read_probe(_ptr(buf), nbytes, _ptr(partials), partials.numel(),
                                        _stream(buf.device)))
    return partials
