"""Python wrapper of the fp64 CPU oracle for the gated delta rule.

TEST INFRASTRUCTURE ONLY.  This is the correctness reference the HIP path is
checked against.  Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` may import it; the product package never does and
shares no code with it.

The arithmetic lives in ``gdn_oracle.c`` (the token-by-token recurrence of the
paper's Sec. 3.1, Eq. "gated_delta_rule", in its rank-one online-regression
form, and the hand-derived vector-Jacobian product).  This module only
marshals arrays: every input is upcast exactly to float64 (bf16 and fp32 are
exactly representable), and dense ``[B, T, H, d]`` inputs are treated as B
packed sequences of length T.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gdn_oracle.c")
_LIB = os.path.join(_HERE, "libgdn_oracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc into ``oracle/libgdn_oracle.so``."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-fPIC", "-shared",
                               "-pthread", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i = ctypes.c_int
        lib.gdn_oracle_fwd.argtypes = [i, P, i, i, i, P, P, P, P, P, P, P, P, i]
        lib.gdn_oracle_fwd.restype = i
        lib.gdn_oracle_bwd.argtypes = [i, P, i, i, i, P, P, P, P, P, P, P, P,
                                       P, P, P, P, P, P, P, P, i, i]
        lib.gdn_oracle_bwd.restype = i
        _lib = lib
    return _lib


def _f64(x):
    if x is None:
        return None
    try:  # torch tensors (bf16 has no numpy dtype)
        import torch
        if isinstance(x, torch.Tensor):
            return np.ascontiguousarray(x.detach().to("cpu", torch.float64).numpy())
    except ImportError:  # pragma: no cover
        pass
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def default_threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def _packed(q, k, v, beta, log_alpha, cu_seqlens):
    """Return (cu int64[N+1], arrays flattened to [Ttot, H, ...], dense shape or None)."""
    q, k, v, beta, log_alpha = map(_f64, (q, k, v, beta, log_alpha))
    if cu_seqlens is None:
        if q.ndim != 4:
            raise ValueError("dense inputs must be [B, T, H, d]")
        B, T, H, _ = q.shape
        cu = np.arange(B + 1, dtype=np.int64) * T
        dense = (B, T)
        q = q.reshape(B * T, H, -1)
        k = k.reshape(B * T, H, -1)
        v = v.reshape(B * T, H, -1)
        beta = beta.reshape(B * T, H)
        log_alpha = log_alpha.reshape(B * T, H)
    else:
        cu = np.ascontiguousarray(np.asarray(_f64(cu_seqlens), dtype=np.int64))
        dense = None
        if q.ndim == 4:  # [1, Ttot, H, d]
            q, k, v = q[0], k[0], v[0]
            beta, log_alpha = beta[0], log_alpha[0]
        q, k, v, beta, log_alpha = map(np.ascontiguousarray, (q, k, v, beta, log_alpha))
    return cu, q, k, v, beta, log_alpha, dense


def fwd(q, k, v, beta, log_alpha, h0=None, cu_seqlens=None, nthreads=None):
    """Token-recurrence forward in fp64.  Returns (o, ht) as float64 arrays.

    Dense: q,k [B,T,H,dk], v [B,T,H,dv], beta/log_alpha [B,T,H], h0 [B,H,dk,dv].
    Packed: same with a leading 1 (or no batch dim) and cu_seqlens [N+1].
    """
    cu, q, k, v, beta, log_alpha, dense = _packed(q, k, v, beta, log_alpha, cu_seqlens)
    N = cu.shape[0] - 1
    Ttot, H, dk = q.shape
    dv = v.shape[-1]
    h0 = _f64(h0)
    o = np.zeros((Ttot, H, dv))
    ht = np.zeros((N, H, dk, dv))
    rc = _load().gdn_oracle_fwd(N, _ptr(cu), H, dk, dv, _ptr(q), _ptr(k), _ptr(v), _ptr(beta),
                                _ptr(log_alpha), _ptr(h0), _ptr(o), _ptr(ht),
                                nthreads or default_threads())
    if rc:
        raise RuntimeError("oracle forward failed (%d)" % rc)
    if dense:
        o = o.reshape(dense[0], dense[1], H, dv)
    return o, ht


def bwd(q, k, v, beta, log_alpha, dO, h0=None, dht=None, cu_seqlens=None, nthreads=None,
        seg=64):
    """Token-recurrence VJP in fp64.

    Returns a dict with o, ht (the forward, recomputed) and dq, dk, dv, dbeta,
    dlog_alpha, dh0, shaped like their inputs.
    """
    cu, q, k, v, beta, log_alpha, dense = _packed(q, k, v, beta, log_alpha, cu_seqlens)
    N = cu.shape[0] - 1
    Ttot, H, dk = q.shape
    dv = v.shape[-1]
    dO = _f64(dO).reshape(Ttot, H, dv)
    h0, dht = _f64(h0), _f64(dht)
    out = dict(o=np.zeros((Ttot, H, dv)), ht=np.zeros((N, H, dk, dv)),
               dq=np.zeros((Ttot, H, dk)), dk=np.zeros((Ttot, H, dk)),
               dv=np.zeros((Ttot, H, dv)), dbeta=np.zeros((Ttot, H)),
               dlog_alpha=np.zeros((Ttot, H)), dh0=np.zeros((N, H, dk, dv)))
    rc = _load().gdn_oracle_bwd(
        N, _ptr(cu), H, dk, dv, _ptr(q), _ptr(k), _ptr(v), _ptr(beta), _ptr(log_alpha),
        _ptr(h0), _ptr(dO), _ptr(dht), _ptr(out["o"]), _ptr(out["ht"]), _ptr(out["dq"]),
        _ptr(out["dk"]), _ptr(out["dv"]), _ptr(out["dbeta"]), _ptr(out["dlog_alpha"]),
        _ptr(out["dh0"]), seg, nthreads or default_threads())
    if rc:
        raise RuntimeError("oracle backward failed (%d)" % rc)
    if dense:
        B, T = dense
        for name in ("o", "dq", "dk", "dv"):
            out[name] = out[name].reshape(B, T, H, -1)
        for name in ("dbeta", "dlog_alpha"):
            out[name] = out[name].reshape(B, T, H)
    return out
