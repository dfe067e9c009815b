"""Thin ctypes binding of libgdn (include/gdn.h).

Argument marshalling only: every step of the computation runs in the HIP
kernels of ``libgdn.so``.  PyTorch provides device memory and the current
stream.  There is no fallback: if the library is missing, loading fails.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgdn.so")

GDN_F32, GDN_BF16 = 0, 1
STATUS = {0: "GDN_OK", 1: "GDN_ERR_NULL", 2: "GDN_ERR_SHAPE", 3: "GDN_ERR_UNSUPPORTED",
          4: "GDN_ERR_CU_SEQLENS", 5: "GDN_ERR_WORKSPACE", 6: "GDN_ERR_HIP", 7: "GDN_ERR_ALIGN",
          8: "GDN_ERR_SAVED", 9: "GDN_ERR_VALUE"}
EXPORTS = ("gdn_chunk_fwd", "gdn_chunk_bwd", "gdn_chunk_fwd_workspace_size",
           "gdn_chunk_bwd_workspace_size", "gdn_chunk_fwd_timed", "gdn_chunk_bwd_timed",
           "gdn_chunk_saved_size", "gdn_chunk_fwd_save_workspace_size",
           "gdn_chunk_bwd_saved_workspace_size", "gdn_chunk_fwd_save", "gdn_chunk_bwd_saved",
           "gdn_chunk_fwd_save_timed", "gdn_chunk_bwd_saved_timed", "gdn_recurrent_fwd",
           "gdn_recurrent_fwd_timed", "gdn_conv_silu_workspace_size", "gdn_conv_silu_fwd",
           "gdn_conv_silu_bwd", "gdn_norm_gate_workspace_size", "gdn_norm_gate_fwd",
           "gdn_norm_gate_bwd", "gdn_status_string", "gdn_chunk_fwd_noalloc",
           "gdn_block_fwd", "gdn_block_fwd_save", "gdn_block_bwd_saved",
           "gdn_block_bwd_saved_workspace_size", "gdn_block_fwd_timed",
           "gdn_block_fwd_save_timed", "gdn_block_bwd_saved_timed", "gdn_debug_audit",
           "gdn_debug_audit_field", "gdn_debug_block_bwd")
# bytes of the library's static workspace behind gdn_chunk_fwd_noalloc
NOALLOC_SCRATCH_BYTES = 64 << 20


class Problem(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("T", ctypes.c_int32), ("H", ctypes.c_int32),
                ("dk", ctypes.c_int32), ("dv", ctypes.c_int32), ("num_seqs", ctypes.c_int32),
                ("cu_seqlens", ctypes.c_void_p), ("cu_seqlens_host", ctypes.c_void_p),
                ("dtype", ctypes.c_int)]


class BlockPrologue(ctypes.Structure):
    _fields_ = [("width", ctypes.c_int32), ("eps", ctypes.c_float),
                ("xq", ctypes.c_void_p), ("xk", ctypes.c_void_p), ("xv", ctypes.c_void_p),
                ("wq", ctypes.c_void_p), ("wk", ctypes.c_void_p), ("wv", ctypes.c_void_p)]


class Timing(ctypes.Structure):
    _fields_ = [("events", ctypes.POINTER(ctypes.c_void_p)), ("capacity", ctypes.c_int32),
                ("launched", ctypes.c_int32), ("names", ctypes.c_char_p * 8)]


class LaunchTimer:
    """Caller-owned HIP events for the *_timed entry points (2 per launch)."""

    def __init__(self, max_launches: int = 8):
        self._hip = ctypes.CDLL("libamdhip64.so")
        self._hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self._hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float),
                                                  ctypes.c_void_p, ctypes.c_void_p]
        self._hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        n = 2 * max_launches
        self.events = (ctypes.c_void_p * n)()
        for i in range(n):
            ev = ctypes.c_void_p()
            if self._hip.hipEventCreate(ctypes.byref(ev)) != 0:
                raise RuntimeError("hipEventCreate failed")
            self.events[i] = ev.value
        self.timing = Timing(ctypes.cast(self.events, ctypes.POINTER(ctypes.c_void_p)), n, 0)

    def durations_ms(self):
        """{kernel name: ms} of the last timed call (stream must have passed it)."""
        out = {}
        for i in range(min(self.timing.launched, len(self.events) // 2)):
            ms = ctypes.c_float()
            if self._hip.hipEventElapsedTime(ctypes.byref(ms), self.events[2 * i],
                                             self.events[2 * i + 1]) != 0:
                raise RuntimeError("hipEventElapsedTime failed")
            out[self.timing.names[i].decode()] = ms.value
        return out

    def close(self):
        for e in self.events:
            if e:
                self._hip.hipEventDestroy(e)
        self.events = (ctypes.c_void_p * 0)()


class GdnError(RuntimeError):
    def __init__(self, code: int):
        super().__init__(STATUS.get(code, "status %d" % code))
        self.code = code


_lib = None


def load_library():
    """Load libgdn.so (built by ``paper_2412_06464_amd.build``); raise if absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libgdn.so is not built (%s); run "
                               "`python -m paper_2412_06464_amd.build`" % LIB_PATH)
        lib = ctypes.CDLL(LIB_PATH)
        P, S = ctypes.c_void_p, ctypes.c_size_t
        pp = ctypes.POINTER(Problem)
        lib.gdn_chunk_fwd_workspace_size.argtypes = [pp]
        lib.gdn_chunk_fwd_workspace_size.restype = S
        lib.gdn_chunk_bwd_workspace_size.argtypes = [pp]
        lib.gdn_chunk_bwd_workspace_size.restype = S
        lib.gdn_chunk_fwd.argtypes = [pp] + [P] * 8 + [P, S, P]
        lib.gdn_chunk_fwd.restype = ctypes.c_int
        lib.gdn_chunk_fwd_noalloc.argtypes = [pp] + [P] * 8 + [P]
        lib.gdn_chunk_fwd_noalloc.restype = ctypes.c_int
        lib.gdn_chunk_bwd.argtypes = [pp] + [P] * 14 + [P, S, P]
        lib.gdn_chunk_bwd.restype = ctypes.c_int
        pt = ctypes.POINTER(Timing)
        lib.gdn_chunk_fwd_timed.argtypes = [pp] + [P] * 8 + [P, S, P, pt]
        lib.gdn_chunk_fwd_timed.restype = ctypes.c_int
        lib.gdn_chunk_bwd_timed.argtypes = [pp] + [P] * 14 + [P, S, P, pt]
        lib.gdn_chunk_bwd_timed.restype = ctypes.c_int
        for name in ("gdn_chunk_saved_size", "gdn_chunk_fwd_save_workspace_size",
                     "gdn_chunk_bwd_saved_workspace_size"):
            getattr(lib, name).argtypes = [pp]
            getattr(lib, name).restype = S
        lib.gdn_chunk_fwd_save.argtypes = [pp] + [P] * 8 + [P, S, P, S, P]
        lib.gdn_chunk_fwd_save.restype = ctypes.c_int
        lib.gdn_chunk_fwd_save_timed.argtypes = [pp] + [P] * 8 + [P, S, P, S, P, pt]
        lib.gdn_chunk_fwd_save_timed.restype = ctypes.c_int
        lib.gdn_chunk_bwd_saved.argtypes = [pp] + [P] * 7 + [S] + [P] * 6 + [P, S, P]
        lib.gdn_chunk_bwd_saved.restype = ctypes.c_int
        lib.gdn_chunk_bwd_saved_timed.argtypes = [pp] + [P] * 7 + [S] + [P] * 6 + [P, S, P, pt]
        lib.gdn_chunk_bwd_saved_timed.restype = ctypes.c_int
        lib.gdn_recurrent_fwd.argtypes = [pp] + [P] * 8 + [P]
        lib.gdn_recurrent_fwd.restype = ctypes.c_int
        lib.gdn_recurrent_fwd_timed.argtypes = [pp] + [P] * 8 + [P, pt]
        lib.gdn_recurrent_fwd_timed.restype = ctypes.c_int
        I, F = ctypes.c_int, ctypes.c_float
        lib.gdn_conv_silu_workspace_size.argtypes = [pp, I, I]
        lib.gdn_conv_silu_workspace_size.restype = S
        lib.gdn_conv_silu_fwd.argtypes = [pp, I, I, I, F, P, P, P, P, S, P]
        lib.gdn_conv_silu_fwd.restype = ctypes.c_int
        lib.gdn_conv_silu_bwd.argtypes = [pp, I, I, I, F, P, P, P, P, P, P, S, P]
        lib.gdn_conv_silu_bwd.restype = ctypes.c_int
        lib.gdn_norm_gate_workspace_size.argtypes = [pp]
        lib.gdn_norm_gate_workspace_size.restype = S
        lib.gdn_norm_gate_fwd.argtypes = [pp, F, P, P, P, P, P]
        lib.gdn_norm_gate_fwd.restype = ctypes.c_int
        lib.gdn_norm_gate_bwd.argtypes = [pp, F, P, P, P, P, P, P, P, P, S, P]
        lib.gdn_norm_gate_bwd.restype = ctypes.c_int
        pb = ctypes.POINTER(BlockPrologue)
        lib.gdn_block_fwd.argtypes = [pp, pb] + [P] * 8 + [P, S, P]
        lib.gdn_block_fwd.restype = ctypes.c_int
        lib.gdn_block_fwd_timed.argtypes = [pp, pb] + [P] * 8 + [P, S, P, pt]
        lib.gdn_block_fwd_timed.restype = ctypes.c_int
        lib.gdn_block_fwd_save.argtypes = [pp, pb] + [P] * 8 + [P, S, P, S, P]
        lib.gdn_block_fwd_save.restype = ctypes.c_int
        lib.gdn_block_fwd_save_timed.argtypes = [pp, pb] + [P] * 8 + [P, S, P, S, P, pt]
        lib.gdn_block_fwd_save_timed.restype = ctypes.c_int
        lib.gdn_block_bwd_saved_workspace_size.argtypes = [pp, I]
        lib.gdn_block_bwd_saved_workspace_size.restype = S
        lib.gdn_block_bwd_saved.argtypes = [pp, pb] + [P] * 7 + [S] + [P] * 9 + [P, S, P]
        lib.gdn_block_bwd_saved.restype = ctypes.c_int
        lib.gdn_block_bwd_saved_timed.argtypes = [pp, pb] + [P] * 7 + [S] + [P] * 9 + [P, S, P,
                                                                                     pt]
        lib.gdn_block_bwd_saved_timed.restype = ctypes.c_int
        lib.gdn_debug_audit.argtypes = [ctypes.c_int32, ctypes.c_uint64]
        lib.gdn_debug_audit.restype = ctypes.c_int32
        lib.gdn_debug_audit_field.argtypes = [ctypes.c_int32]
        lib.gdn_debug_audit_field.restype = ctypes.c_char_p
        lib.gdn_debug_block_bwd.argtypes = [ctypes.c_int32]
        lib.gdn_debug_block_bwd.restype = ctypes.c_int32
        lib.gdn_status_string.argtypes = [ctypes.c_int]
        lib.gdn_status_string.restype = ctypes.c_char_p
        _lib = lib
    return _lib


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _cu_pair(cu_seqlens, cu_seqlens_host, device, keep):
    """Device and host int32 copies of packed sequence boundaries.

    The kernels read the device copy as contiguous int32 on the device of the
    data; an int64 tensor (what ``torch.tensor`` and ``cumsum`` give) is
    converted here, and the converted copy is kept alive in ``keep`` until the
    call returns.  Without a host copy it is read back from the device (a
    synchronisation)."""
    if not isinstance(cu_seqlens, torch.Tensor) or cu_seqlens.dim() != 1:
        raise TypeError("cu_seqlens must be a 1-d tensor")
    if cu_seqlens.device != device:
        raise ValueError("cu_seqlens is on %s, the data on %s" % (cu_seqlens.device, device))
    if cu_seqlens.dtype not in (torch.int32, torch.int64):
        raise TypeError("cu_seqlens must be int32 (or int64, converted)")
    dev = cu_seqlens
    if dev.dtype != torch.int32 or not dev.is_contiguous():
        dev = dev.to(torch.int32).contiguous()
        keep.append(dev)
    if cu_seqlens_host is None:
        cu_seqlens_host = dev.to("cpu")
    if not isinstance(cu_seqlens_host, torch.Tensor) or cu_seqlens_host.device.type != "cpu":
        raise TypeError("cu_seqlens_host must be a CPU tensor")
    host = cu_seqlens_host.to(torch.int32).contiguous()
    if host.numel() != dev.numel():
        raise ValueError("cu_seqlens (%d values) and cu_seqlens_host (%d values) differ"
                         % (dev.numel(), host.numel()))
    keep.append(host)
    return dev, host


def make_problem(q: torch.Tensor, v: torch.Tensor, cu_seqlens=None, cu_seqlens_host=None):
    """Build the gdn_problem for q [B,T,H,dk], v [B,T,H,dv].  Returns (problem, keepalive)."""
    if q.dim() != 4 or v.dim() != 4 or q.shape[:3] != v.shape[:3]:
        raise ValueError("q must be [B,T,H,dk] and v [B,T,H,dv] over the same B, T, H")
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    dt = {torch.float32: GDN_F32, torch.bfloat16: GDN_BF16}.get(q.dtype)
    if dt is None:
        raise TypeError("q must be float32 or bfloat16")
    keep = []
    p = Problem(B, T, H, dk, dv, 0, None, None, dt)
    if cu_seqlens is not None:
        dev, host = _cu_pair(cu_seqlens, cu_seqlens_host, q.device, keep)
        p.num_seqs = host.numel() - 1
        p.cu_seqlens = dev.data_ptr()
        p.cu_seqlens_host = host.data_ptr()
    return p, keep


def _check_tensors(q, rows=(), gates=(), states=(), nstate=None):
    """Argument checks before a call: every tensor on q's device and
    contiguous; ``rows`` [B,T,H,*] in q's dtype; ``gates`` [B,T,H] float32;
    ``states`` [Nseq,H,dk,dv] float32.  None entries are skipped."""
    B, T, H, dk = q.shape
    named = (("q", q),) + tuple(rows) + tuple(gates) + tuple((n, t) for n, t, _ in states)
    for name, t in named:
        if t is None:
            continue
        if not isinstance(t, torch.Tensor):
            raise TypeError("%s must be a tensor" % name)
        if t.device != q.device:
            raise ValueError("%s is on %s, q on %s" % (name, t.device, q.device))
        if not t.is_contiguous():
            raise ValueError("%s must be contiguous" % name)
    for name, t in rows:
        if t is not None and (t.dtype != q.dtype or t.dim() != 4 or t.shape[:3] != q.shape[:3]):
            raise ValueError("%s must be [B,T,H,*] in q's dtype %s" % (name, q.dtype))
    for name, t in gates:
        if t is not None and (t.dtype != torch.float32 or tuple(t.shape) != (B, T, H)):
            raise ValueError("%s must be float32 [B,T,H]" % name)
    for name, t, d2 in states:
        if t is not None and (t.dtype != torch.float32 or tuple(t.shape) != (nstate, H, dk, d2)):
            raise ValueError("%s must be float32 [%d,%d,%d,%d]" % (name, nstate, H, dk, d2))


def gdn_chunk_fwd_workspace_size(p: Problem) -> int:
    return int(load_library().gdn_chunk_fwd_workspace_size(ctypes.byref(p)))


def gdn_chunk_bwd_workspace_size(p: Problem) -> int:
    return int(load_library().gdn_chunk_bwd_workspace_size(ctypes.byref(p)))


def gdn_chunk_saved_size(p: Problem) -> int:
    return int(load_library().gdn_chunk_saved_size(ctypes.byref(p)))


def gdn_chunk_fwd_save_workspace_size(p: Problem) -> int:
    return int(load_library().gdn_chunk_fwd_save_workspace_size(ctypes.byref(p)))


def gdn_chunk_bwd_saved_workspace_size(p: Problem) -> int:
    return int(load_library().gdn_chunk_bwd_saved_workspace_size(ctypes.byref(p)))


def gdn_status_string(code: int) -> str:
    return load_library().gdn_status_string(code).decode()


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _check(code: int):
    if code != 0:
        raise GdnError(code)


def _nstate(q, cu_seqlens):
    return q.shape[0] if cu_seqlens is None else cu_seqlens.numel() - 1


def gdn_chunk_fwd(q, k, v, beta, log_alpha, h0=None, cu_seqlens=None, cu_seqlens_host=None,
                  output_final_state=True, o=None, ht=None, workspace=None, timer=None):
    """Forward of the chunkwise gated delta rule on the current stream.

    q, k [B,T,H,dk] and v [B,T,H,dv] (fp32 or bf16, same dtype), beta and
    log_alpha [B,T,H] fp32 (log_alpha None: alpha == 1, the ungated rule),
    h0 [Nseq,H,dk,dv] fp32 or None; packed input
    passes cu_seqlens (int32 [N+1], device) with B == 1.  Returns (o, ht).
    ``timer`` (a LaunchTimer) routes the call through gdn_chunk_fwd_timed.
    """
    lib = load_library()
    p, keep = make_problem(q, v, cu_seqlens, cu_seqlens_host)
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    if o is None:
        o = torch.empty((B, T, H, dv), dtype=q.dtype, device=q.device)
    if ht is None and output_final_state:
        ht = torch.empty((_nstate(q, cu_seqlens), H, dk, dv), dtype=torch.float32,
                         device=q.device)
    _check_tensors(q, rows=(("k", k), ("v", v), ("o", o)), gates=(("beta", beta),
                   ("log_alpha", log_alpha)), states=(("h0", h0, dv), ("ht", ht, dv)),
                   nstate=_nstate(q, cu_seqlens))
    if k.shape != q.shape or o.shape != v.shape:
        raise ValueError("k must match q, and o must match v")
    need = lib.gdn_chunk_fwd_workspace_size(ctypes.byref(p))
    if need == 0:
        _check(lib.gdn_chunk_fwd(ctypes.byref(p), *[None] * 8, None, 0, None))
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    args = (ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(beta), _ptr(log_alpha), _ptr(h0),
            _ptr(o), _ptr(ht), _ptr(workspace), workspace.numel(), _stream(q.device))
    if timer is None:
        _check(lib.gdn_chunk_fwd(*args))
    else:
        _check(lib.gdn_chunk_fwd_timed(*args, ctypes.byref(timer.timing)))
    del keep
    return o, ht


def gdn_chunk_fwd_noalloc(q, k, v, beta, log_alpha, h0=None, cu_seqlens=None,
                          cu_seqlens_host=None, o=None, ht=None):
    """gdn_chunk_fwd on the library's static workspace (no allocation in the
    library; pass ``o`` and ``ht`` to allocate nothing here either).  Raises
    GdnError(GDN_ERR_WORKSPACE) for problems whose workspace exceeds
    NOALLOC_SCRATCH_BYTES.  Calls on one GPU must not overlap in time."""
    lib = load_library()
    p, keep = make_problem(q, v, cu_seqlens, cu_seqlens_host)
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    if o is None:
        o = torch.empty((B, T, H, dv), dtype=q.dtype, device=q.device)
    _check_tensors(q, rows=(("k", k), ("v", v), ("o", o)), gates=(("beta", beta),
                   ("log_alpha", log_alpha)), states=(("h0", h0, dv), ("ht", ht, dv)),
                   nstate=_nstate(q, cu_seqlens))
    if k.shape != q.shape or o.shape != v.shape:
        raise ValueError("k must match q, and o must match v")
    _check(lib.gdn_chunk_fwd_noalloc(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(beta),
                                     _ptr(log_alpha), _ptr(h0), _ptr(o), _ptr(ht),
                                     _stream(q.device)))
    del keep
    return o, ht


def gdn_chunk_bwd(q, k, v, beta, log_alpha, dO, h0=None, dht=None, cu_seqlens=None,
                  cu_seqlens_host=None, need_dh0=True, need_dlog_alpha=True, workspace=None,
                  out=None, timer=None):
    """Backward (stateless): returns dict dq, dk, dv, dbeta, dlog_alpha, dh0.
    ``log_alpha`` None means alpha == 1; ``need_dlog_alpha`` False skips the
    gate gradient (dlog_alpha None).  ``timer`` (a LaunchTimer) routes the
    call through gdn_chunk_bwd_timed."""
    lib = load_library()
    p, keep = make_problem(q, v, cu_seqlens, cu_seqlens_host)
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    if out is None:
        out = dict(dq=torch.empty_like(q), dk=torch.empty_like(k), dv=torch.empty_like(v),
                   dbeta=torch.empty_like(beta),
                   dlog_alpha=torch.empty_like(beta) if need_dlog_alpha else None,
                   dh0=torch.empty((_nstate(q, cu_seqlens), H, dk, dv), dtype=torch.float32,
                                   device=q.device) if need_dh0 else None)
    _check_tensors(q, rows=(("k", k), ("v", v), ("dO", dO), ("dq", out["dq"]), ("dk", out["dk"]),
                            ("dv", out["dv"])),
                   gates=(("beta", beta), ("log_alpha", log_alpha), ("dbeta", out["dbeta"]),
                          ("dlog_alpha", out["dlog_alpha"])),
                   states=(("h0", h0, dv), ("dht", dht, dv), ("dh0", out["dh0"], dv)),
                   nstate=_nstate(q, cu_seqlens))
    if k.shape != q.shape or dO.shape != v.shape:
        raise ValueError("k must match q, and dO must match v")
    need = lib.gdn_chunk_bwd_workspace_size(ctypes.byref(p))
    if need == 0:
        _check(lib.gdn_chunk_bwd(ctypes.byref(p), *[None] * 14, None, 0, None))
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    args = (ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(beta), _ptr(log_alpha), _ptr(h0),
            _ptr(dO), _ptr(dht), _ptr(out["dq"]), _ptr(out["dk"]), _ptr(out["dv"]),
            _ptr(out["dbeta"]), _ptr(out["dlog_alpha"]), _ptr(out["dh0"]), _ptr(workspace),
            workspace.numel(), _stream(q.device))
    if timer is None:
        _check(lib.gdn_chunk_bwd(*args))
    else:
        _check(lib.gdn_chunk_bwd_timed(*args, ctypes.byref(timer.timing)))
    del keep
    return out


def gdn_chunk_fwd_save(q, k, v, beta, log_alpha, h0=None, cu_seqlens=None, cu_seqlens_host=None,
                       output_final_state=True, o=None, ht=None, saved=None, workspace=None,
                       timer=None):
    """Forward that also fills the buffer the saved backward reads.

    Same arguments and outputs as gdn_chunk_fwd; returns (o, ht, saved), where
    ``saved`` is a uint8 device tensor of gdn_chunk_saved_size bytes (pass one
    in to reuse it).  ``timer`` routes the call through gdn_chunk_fwd_save_timed.
    """
    lib = load_library()
    p, keep = make_problem(q, v, cu_seqlens, cu_seqlens_host)
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    if o is None:
        o = torch.empty((B, T, H, dv), dtype=q.dtype, device=q.device)
    if ht is None and output_final_state:
        ht = torch.empty((_nstate(q, cu_seqlens), H, dk, dv), dtype=torch.float32,
                         device=q.device)
    _check_tensors(q, rows=(("k", k), ("v", v), ("o", o)), gates=(("beta", beta),
                   ("log_alpha", log_alpha)), states=(("h0", h0, dv), ("ht", ht, dv)),
                   nstate=_nstate(q, cu_seqlens))
    if k.shape != q.shape or o.shape != v.shape:
        raise ValueError("k must match q, and o must match v")
    need = lib.gdn_chunk_fwd_save_workspace_size(ctypes.byref(p))
    if need == 0:
        _check(lib.gdn_chunk_fwd_save(ctypes.byref(p), *[None] * 8, None, 0, None, 0, None))
    nsave = lib.gdn_chunk_saved_size(ctypes.byref(p))
    if saved is None or saved.numel() < nsave:
        saved = torch.empty(nsave, dtype=torch.uint8, device=q.device)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    args = (ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(beta), _ptr(log_alpha), _ptr(h0),
            _ptr(o), _ptr(ht), _ptr(saved), saved.numel(), _ptr(workspace), workspace.numel(),
            _stream(q.device))
    if timer is None:
        _check(lib.gdn_chunk_fwd_save(*args))
    else:
        _check(lib.gdn_chunk_fwd_save_timed(*args, ctypes.byref(timer.timing)))
    del keep
    return o, ht, saved


def gdn_chunk_bwd_saved(q, k, v, beta, dO, saved, dht=None, cu_seqlens=None,
                        cu_seqlens_host=None, need_dh0=True, need_dlog_alpha=True,
                        workspace=None, out=None, timer=None):
    """Backward from gdn_chunk_fwd_save's buffer: dict dq, dk, dv, dbeta, dlog_alpha, dh0.

    ``q``, ``k``, ``v`` and ``beta`` are the tensors the saving forward read;
    the gates and h0 enter through ``saved``.  ``need_dlog_alpha`` False
    skips the gate gradient.  ``timer`` routes the call through
    gdn_chunk_bwd_saved_timed.
    """
    lib = load_library()
    p, keep = make_problem(q, v, cu_seqlens, cu_seqlens_host)
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    if out is None:
        out = dict(dq=torch.empty_like(q), dk=torch.empty_like(q), dv=torch.empty_like(v),
                   dbeta=torch.empty_like(beta),
                   dlog_alpha=torch.empty_like(beta) if need_dlog_alpha else None,
                   dh0=torch.empty((_nstate(q, cu_seqlens), H, dk, dv), dtype=torch.float32,
                                   device=q.device) if need_dh0 else None)
    _check_tensors(q, rows=(("k", k), ("v", v), ("dO", dO), ("dq", out["dq"]), ("dk", out["dk"]),
                            ("dv", out["dv"])),
                   gates=(("beta", beta), ("dbeta", out["dbeta"]),
                          ("dlog_alpha", out["dlog_alpha"])),
                   states=(("dht", dht, dv), ("dh0", out["dh0"], dv)),
                   nstate=_nstate(q, cu_seqlens))
    if k.shape != q.shape or dO.shape != v.shape:
        raise ValueError("k must match q, and dO must match v")
    if saved.device != q.device or saved.dtype != torch.uint8 or not saved.is_contiguous():
        raise ValueError("saved must be a contiguous uint8 tensor on q's device")
    need = lib.gdn_chunk_bwd_saved_workspace_size(ctypes.byref(p))
    if need == 0:
        _check(lib.gdn_chunk_bwd_saved(ctypes.byref(p), *[None] * 7, 0, *[None] * 6, None, 0,
                                       None))
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    args = (ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(beta), _ptr(dO), _ptr(dht),
            _ptr(saved),
            saved.numel(), _ptr(out["dq"]), _ptr(out["dk"]), _ptr(out["dv"]), _ptr(out["dbeta"]),
            _ptr(out["dlog_alpha"]), _ptr(out["dh0"]), _ptr(workspace), workspace.numel(),
            _stream(q.device))
    if timer is None:
        _check(lib.gdn_chunk_bwd_saved(*args))
    else:
        _check(lib.gdn_chunk_bwd_saved_timed(*args, ctypes.byref(timer.timing)))
    del keep
    return out


def gdn_recurrent_fwd(q, k, v, beta, log_alpha, h0=None, cu_seqlens=None, cu_seqlens_host=None,
                      output_final_state=True, o=None, ht=None, timer=None):
    """Token-by-token forward (inference; T = 1 is one decode step).

    Same arguments and results as gdn_chunk_fwd, without a workspace.  Pass
    ``ht=h0`` to update the state in place.  ``timer`` routes the call
    through gdn_recurrent_fwd_timed.
    """
    lib = load_library()
    p, keep = make_problem(q, v, cu_seqlens, cu_seqlens_host)
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    if o is None:
        o = torch.empty((B, T, H, dv), dtype=q.dtype, device=q.device)
    if ht is None and output_final_state:
        ht = torch.empty((_nstate(q, cu_seqlens), H, dk, dv), dtype=torch.float32,
                         device=q.device)
    _check_tensors(q, rows=(("k", k), ("v", v), ("o", o)), gates=(("beta", beta),
                   ("log_alpha", log_alpha)), states=(("h0", h0, dv), ("ht", ht, dv)),
                   nstate=_nstate(q, cu_seqlens))
    if k.shape != q.shape or o.shape != v.shape:
        raise ValueError("k must match q, and o must match v")
    args = (ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(beta), _ptr(log_alpha), _ptr(h0),
            _ptr(o), _ptr(ht), _stream(q.device))
    if timer is None:
        _check(lib.gdn_recurrent_fwd(*args))
    else:
        _check(lib.gdn_recurrent_fwd_timed(*args, ctypes.byref(timer.timing)))
    del keep
    return o, ht


# ------------------------------------------------------------------ block prologue / epilogue

# the (dk, dv) pair of a supported rule problem that has a given head dim
_PAIR = {64: (64, 64), 128: (128, 128), 256: (256, 512), 512: (256, 512)}


def block_problem(x: torch.Tensor, cu_seqlens=None, cu_seqlens_host=None):
    """gdn_problem for a [B, T, H, d] tensor of the block (d is its dk or dv)."""
    B, T, H, d = x.shape
    if d not in _PAIR:
        raise ValueError("unsupported head dim %d" % d)
    dk, dv = _PAIR[d]
    q = torch.empty((B, T, H, dk), dtype=x.dtype, device="meta")
    v = torch.empty((B, T, H, dv), dtype=x.dtype, device="meta")
    return make_problem_meta(q, v, cu_seqlens, cu_seqlens_host)


def make_problem_meta(q, v, cu_seqlens=None, cu_seqlens_host=None):
    """make_problem for shape-only tensors (no data pointer needed)."""
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    dt = {torch.float32: GDN_F32, torch.bfloat16: GDN_BF16}.get(q.dtype)
    if dt is None:
        raise TypeError("dtype must be float32 or bfloat16")
    keep = []
    p = Problem(B, T, H, dk, dv, 0, None, None, dt)
    if cu_seqlens is not None:
        dev, host = _cu_pair(cu_seqlens, cu_seqlens_host, cu_seqlens.device, keep)
        p.num_seqs = host.numel() - 1
        p.cu_seqlens = dev.data_ptr()
        p.cu_seqlens_host = host.data_ptr()
    return p, keep


def gdn_conv_silu_fwd(x, w, l2norm=True, eps=1e-6, cu_seqlens=None, cu_seqlens_host=None, y=None,
                      workspace=None):
    """Short causal convolution + SiLU (+ L2 per row) of x [B, T, H, d]; w fp32 [H * d, W]."""
    lib = load_library()
    p, keep = block_problem(x, cu_seqlens, cu_seqlens_host)
    d, W = x.shape[-1], w.shape[1]
    if y is None:
        y = torch.empty_like(x)
    need = lib.gdn_conv_silu_workspace_size(ctypes.byref(p), d, W)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    _check(lib.gdn_conv_silu_fwd(ctypes.byref(p), d, W, int(l2norm), eps, _ptr(x), _ptr(w),
                                 _ptr(y), _ptr(workspace), workspace.numel(), _stream(x.device)))
    del keep
    return y


def gdn_conv_silu_bwd(x, w, dy, l2norm=True, eps=1e-6, cu_seqlens=None, cu_seqlens_host=None,
                      dx=None, dw=None, workspace=None):
    """Backward of gdn_conv_silu_fwd: returns (dx, dw)."""
    lib = load_library()
    p, keep = block_problem(x, cu_seqlens, cu_seqlens_host)
    d, W = x.shape[-1], w.shape[1]
    if dx is None:
        dx = torch.empty_like(x)
    if dw is None:
        dw = torch.empty_like(w)
    need = lib.gdn_conv_silu_workspace_size(ctypes.byref(p), d, W)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    _check(lib.gdn_conv_silu_bwd(ctypes.byref(p), d, W, int(l2norm), eps, _ptr(x), _ptr(w),
                                 _ptr(dy), _ptr(dx), _ptr(dw), _ptr(workspace),
                                 workspace.numel(), _stream(x.device)))
    del keep
    return dx, dw


def gdn_norm_gate_fwd(o, g, w, eps=1e-5, y=None):
    """RMS normalisation of o [B, T, H, dv] per (token, head), times w [dv], times silu(g)."""
    lib = load_library()
    p, keep = block_problem(o)
    if y is None:
        y = torch.empty_like(o)
    _check(lib.gdn_norm_gate_fwd(ctypes.byref(p), eps, _ptr(o), _ptr(g), _ptr(w), _ptr(y),
                                 _stream(o.device)))
    del keep
    return y


def gdn_norm_gate_bwd(o, g, w, dy, eps=1e-5, dout=None, dg=None, dw=None, workspace=None):
    """Backward of gdn_norm_gate_fwd: returns (dout, dg, dw)."""
    lib = load_library()
    p, keep = block_problem(o)
    if dout is None:
        dout = torch.empty_like(o)
    if dg is None:
        dg = torch.empty_like(g)
    if dw is None:
        dw = torch.empty_like(w)
    need = lib.gdn_norm_gate_workspace_size(ctypes.byref(p))
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=o.device)
    _check(lib.gdn_norm_gate_bwd(ctypes.byref(p), eps, _ptr(o), _ptr(g), _ptr(w), _ptr(dy),
                                 _ptr(dout), _ptr(dg), _ptr(dw), _ptr(workspace),
                                 workspace.numel(), _stream(o.device)))
    del keep
    return dout, dg, dw


# ------------------------------------------------------------ fused block


def _prologue(xq, xk, xv, wq, wk, wv, eps):
    """BlockPrologue for the projections and fp32 weights [H * d, W]."""
    B, T, H, dk = xq.shape
    dv = xv.shape[-1]
    W = wq.shape[1] if wq.dim() == 2 else -1
    _check_tensors(xq, rows=(("xk", xk), ("xv", xv)))
    if xk.shape != xq.shape:
        raise ValueError("xk must match xq")
    for name, w, d in (("wq", wq, dk), ("wk", wk, dk), ("wv", wv, dv)):
        if (not isinstance(w, torch.Tensor) or w.device != xq.device or w.dtype != torch.float32
                or not w.is_contiguous() or tuple(w.shape) != (H * d, W)):
            raise ValueError("%s must be contiguous float32 [%d, width] on %s"
                             % (name, H * d, xq.device))
    return BlockPrologue(W, eps, xq.data_ptr(), xk.data_ptr(), xv.data_ptr(), wq.data_ptr(),
                         wk.data_ptr(), wv.data_ptr())


def gdn_block_fwd(xq, xk, xv, wq, wk, wv, beta, log_alpha, h0=None, eps=1e-6, cu_seqlens=None,
                  cu_seqlens_host=None, output_final_state=True, want_qkv=False, save=False,
                  o=None, ht=None, q=None, k=None, v=None, saved=None, workspace=None,
                  timer=None):
    """Fused block forward: the prologue (short convolution, SiLU, L2 of q
    and k) inside the chunked rule's kernels.  Returns a dict with o, ht, the
    rule's q, k, v (with ``want_qkv``, and always with ``save``), and saved
    (with ``save``: gdn_block_fwd_save, for gdn_block_bwd_saved).  Output
    tensors passed in (o, ht, q, k, v, saved) are written in place."""
    lib = load_library()
    p, keep = make_problem(xq, xv, cu_seqlens, cu_seqlens_host)
    pro = _prologue(xq, xk, xv, wq, wk, wv, eps)
    B, T, H, dk = xq.shape
    dv = xv.shape[-1]
    ns = _nstate(xq, cu_seqlens)
    if o is None:
        o = torch.empty((B, T, H, dv), dtype=xq.dtype, device=xq.device)
    if ht is None and output_final_state:
        ht = torch.empty((ns, H, dk, dv), dtype=torch.float32, device=xq.device)
    want_qkv = want_qkv or save
    if q is None and want_qkv:
        q = torch.empty_like(xq)
    if k is None and want_qkv:
        k = torch.empty_like(xk)
    if v is None and want_qkv:
        v = torch.empty_like(xv)
    _check_tensors(xq, rows=(("o", o), ("q", q), ("k", k), ("v", v)),
                   gates=(("beta", beta), ("log_alpha", log_alpha)),
                   states=(("h0", h0, dv), ("ht", ht, dv)), nstate=ns)
    if o.shape != xv.shape or (v is not None and v.shape != xv.shape) or any(
            t is not None and t.shape != xq.shape for t in (q, k)):
        raise ValueError("o and v must match xv, q and k must match xq")
    need = (lib.gdn_chunk_fwd_save_workspace_size if save
            else lib.gdn_chunk_fwd_workspace_size)(ctypes.byref(p))
    if need == 0:  # the problem is invalid: let the library name the error
        _check(lib.gdn_block_fwd(ctypes.byref(p), ctypes.byref(pro), *[None] * 8, None, 0, None))
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=xq.device)
    head = (ctypes.byref(p), ctypes.byref(pro), _ptr(beta), _ptr(log_alpha), _ptr(h0), _ptr(o),
            _ptr(ht), _ptr(q), _ptr(k), _ptr(v))
    tail = (_ptr(workspace), workspace.numel(), _stream(xq.device))
    if save:
        nsave = lib.gdn_chunk_saved_size(ctypes.byref(p))
        if saved is None or saved.numel() < nsave:
            saved = torch.empty(nsave, dtype=torch.uint8, device=xq.device)
        args = head + (_ptr(saved), saved.numel()) + tail
        if timer is None:
            _check(lib.gdn_block_fwd_save(*args))
        else:
            _check(lib.gdn_block_fwd_save_timed(*args, ctypes.byref(timer.timing)))
    else:
        args = head + tail
        if timer is None:
            _check(lib.gdn_block_fwd(*args))
        else:
            _check(lib.gdn_block_fwd_timed(*args, ctypes.byref(timer.timing)))
    del keep
    return dict(o=o, ht=ht, q=q, k=k, v=v, saved=saved if save else None)


def gdn_block_bwd_saved(xq, xk, xv, wq, wk, wv, q, k, v, beta, dO, saved, dht=None, eps=1e-6,
                        cu_seqlens=None, cu_seqlens_host=None, need_dh0=True,
                        need_dlog_alpha=True, workspace=None, out=None, timer=None):
    """Fused block backward from gdn_block_fwd(save=True): dict dxq, dxk,
    dxv, dwq, dwk, dwv, dbeta, dlog_alpha, dh0.  ``q``, ``k``, ``v`` are the
    rule's inputs the saving forward returned."""
    lib = load_library()
    p, keep = make_problem(xq, xv, cu_seqlens, cu_seqlens_host)
    pro = _prologue(xq, xk, xv, wq, wk, wv, eps)
    B, T, H, dk = xq.shape
    dv = xv.shape[-1]
    ns = _nstate(xq, cu_seqlens)
    if out is None:
        out = dict(dxq=torch.empty_like(xq), dxk=torch.empty_like(xk), dxv=torch.empty_like(xv),
                   dwq=torch.empty_like(wq), dwk=torch.empty_like(wk), dwv=torch.empty_like(wv),
                   dbeta=torch.empty_like(beta),
                   dlog_alpha=torch.empty_like(beta) if need_dlog_alpha else None,
                   dh0=torch.empty((ns, H, dk, dv), dtype=torch.float32,
                                   device=xq.device) if need_dh0 else None)
    _check_tensors(xq, rows=(("q", q), ("k", k), ("v", v), ("dO", dO), ("dxq", out["dxq"]),
                             ("dxk", out["dxk"]), ("dxv", out["dxv"])),
                   gates=(("beta", beta), ("dbeta", out["dbeta"]),
                          ("dlog_alpha", out["dlog_alpha"])),
                   states=(("dht", dht, dv), ("dh0", out["dh0"], dv)), nstate=ns)
    if v.shape != xv.shape or dO.shape != xv.shape or q.shape != xq.shape or k.shape != xq.shape:
        raise ValueError("q and k must match xq, v and dO xv")
    for name in ("dwq", "dwk", "dwv"):
        w = {"dwq": wq, "dwk": wk, "dwv": wv}[name]
        t = out[name]
        if t.dtype != torch.float32 or t.shape != w.shape or not t.is_contiguous() \
                or t.device != xq.device:
            raise ValueError("%s must be contiguous float32 shaped as its weight" % name)
    if saved.device != xq.device or saved.dtype != torch.uint8 or not saved.is_contiguous():
        raise ValueError("saved must be a contiguous uint8 tensor on xq's device")
    need = lib.gdn_block_bwd_saved_workspace_size(ctypes.byref(p), pro.width)
    if need == 0:
        _check(lib.gdn_block_bwd_saved(ctypes.byref(p), ctypes.byref(pro), *[None] * 7, 0,
                                       *[None] * 9, None, 0, None))
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=xq.device)
    args = (ctypes.byref(p), ctypes.byref(pro), _ptr(q), _ptr(k), _ptr(v), _ptr(beta), _ptr(dO),
            _ptr(dht),
            _ptr(saved), saved.numel(), _ptr(out["dxq"]), _ptr(out["dxk"]), _ptr(out["dxv"]),
            _ptr(out["dwq"]), _ptr(out["dwk"]), _ptr(out["dwv"]), _ptr(out["dbeta"]),
            _ptr(out["dlog_alpha"]), _ptr(out["dh0"]), _ptr(workspace), workspace.numel(),
            _stream(xq.device))
    if timer is None:
        _check(lib.gdn_block_bwd_saved(*args))
    else:
        _check(lib.gdn_block_bwd_saved_timed(*args, ctypes.byref(timer.timing)))
    del keep
    return out
