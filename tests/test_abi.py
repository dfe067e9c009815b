"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, sizes workspaces, and rejects bad arguments on the host
before any launch."""
import ctypes
import os
import re

import pytest

from paper_2412_06464_amd import gdn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gdn.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(gdn.LIB_PATH):
        from paper_2412_06464_amd import build
        build.build()
    return gdn.load_library()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(
        r"^\s*(?:const\s+)?[a-z_][a-z_0-9]*\s*\*?\s*(gdn_[a-z_0-9]+)\s*\(", text, re.M)))


def test_header_declares_expected_entry_points():
    assert declared_functions() == sorted(gdn.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def problem(B=2, T=100, H=3, dk=64, dv=64, dtype=gdn.GDN_BF16, cu=None):
    p = gdn.Problem(B, T, H, dk, dv, 0, None, None, dtype)
    keep = None
    if cu is not None:
        arr = (ctypes.c_int32 * len(cu))(*cu)
        keep = arr
        p.num_seqs = len(cu) - 1
        p.cu_seqlens = 0x1000  # a device address is never dereferenced on the host
        p.cu_seqlens_host = ctypes.addressof(arr)
    return p, keep


def test_status_strings(lib):
    for code, name in gdn.STATUS.items():
        assert gdn.gdn_status_string(code).startswith(name)


def test_workspace_sizes(lib):
    p, _ = problem()
    f = gdn.gdn_chunk_fwd_workspace_size(p)
    b = gdn.gdn_chunk_bwd_workspace_size(p)
    NCH = 2 * 2 * 3  # two sequences of 100 tokens -> 2 chunks each, 3 heads
    e = 2
    # forward: W~, Kbar^T (64 x dk), U~ (64 x dv), P (64 x 64) per chunk-head
    assert f >= NCH * (2 * 64 * 64 * e + 64 * 64 * e + 64 * 64 * e)
    # backward adds entry states and exit-state gradients (dk x dv), V' and dX
    # (64 x dv), and P^T, strictLower(Gamma K K^T)^T (64 x 64)
    assert b - f >= NCH * (2 * 64 * 64 * e + 2 * 64 * 64 * e + 2 * 64 * 64 * e)
    bad, _ = problem(dk=96)
    assert gdn.gdn_chunk_fwd_workspace_size(bad) == 0


@pytest.mark.parametrize("kw,code", [
    (dict(dk=96), 3), (dict(dk=128, dv=64), 3), (dict(dtype=gdn.GDN_F32, dk=256, dv=256), 3),
    (dict(B=0), 2), (dict(T=0), 2), (dict(H=0), 2), (dict(dtype=7), 3),
])
def test_bad_problem_rejected_before_launch(lib, kw, code):
    p, _ = problem(**kw)
    fake = ctypes.c_void_p(0x10000)
    rc = lib.gdn_chunk_fwd(ctypes.byref(p), fake, fake, fake, fake, fake, None, fake, None,
                           fake, 1 << 40, None)
    assert rc == code
    rc = lib.gdn_chunk_bwd(ctypes.byref(p), *([fake] * 5), None, fake, None, *([fake] * 5),
                           None, fake, 1 << 40, None)
    assert rc == code


@pytest.mark.parametrize("cu,code", [
    ([0, 50, 40, 100], 4),   # decreasing
    ([0, 50, 99], 4),        # does not end at T
    ([1, 50, 100], 4),       # does not start at 0
])
def test_bad_cu_seqlens(lib, cu, code):
    p, keep = problem(B=1, cu=cu)
    fake = ctypes.c_void_p(0x10000)
    rc = lib.gdn_chunk_fwd(ctypes.byref(p), fake, fake, fake, fake, fake, None, fake, None,
                           fake, 1 << 40, None)
    assert rc == code
    del keep


def test_packed_needs_batch_one_and_host_copy(lib):
    p, keep = problem(B=2, cu=[0, 100])
    fake = ctypes.c_void_p(0x10000)
    assert lib.gdn_chunk_fwd(ctypes.byref(p), fake, fake, fake, fake, fake, None, fake, None,
                             fake, 1 << 40, None) == 2
    p, keep = problem(B=1, T=100, cu=[0, 100])
    p.cu_seqlens_host = None
    assert lib.gdn_chunk_fwd(ctypes.byref(p), fake, fake, fake, fake, fake, None, fake, None,
                             fake, 1 << 40, None) == 4


def test_null_misaligned_and_small_workspace(lib):
    p, _ = problem()
    fake = ctypes.c_void_p(0x10000)
    odd = ctypes.c_void_p(0x10008)
    args = [fake] * 5 + [None, fake, None]
    assert lib.gdn_chunk_fwd(ctypes.byref(p), None, *args[1:], fake, 1 << 40, None) == 1
    assert lib.gdn_chunk_fwd(ctypes.byref(p), odd, *args[1:], fake, 1 << 40, None) == 7
    need = gdn.gdn_chunk_fwd_workspace_size(p)
    assert lib.gdn_chunk_fwd(ctypes.byref(p), *args, fake, need - 1, None) == 5
    assert lib.gdn_chunk_fwd(ctypes.byref(p), *args, None, need, None) == 5
    bargs = [fake] * 5 + [None, fake, None] + [fake] * 5 + [None]
    needb = gdn.gdn_chunk_bwd_workspace_size(p)
    assert lib.gdn_chunk_bwd(ctypes.byref(p), *bargs, fake, needb - 1, None) == 5
    bargs[6] = None  # dO
    assert lib.gdn_chunk_bwd(ctypes.byref(p), *bargs, fake, needb, None) == 1


def test_saved_path_sizes(lib):
    p, _ = problem()
    NCH = 2 * 2 * 3
    e = 2
    s = gdn.gdn_chunk_saved_size(p)
    fw = gdn.gdn_chunk_fwd_save_workspace_size(p)
    bw = gdn.gdn_chunk_bwd_saved_workspace_size(p)
    # saved: entry states (dk x dv) and V' (64 x dv) per chunk-head, the
    # gates' cumulative sums, P and strictLower(Gamma K K^T) in fp32
    assert s >= NCH * (64 * 64 * e + 64 * 64 * e + 64 * 4 + 2 * 64 * 64 * 4)
    # the stateless backward holds everything the saved path splits up
    assert gdn.gdn_chunk_bwd_workspace_size(p) >= s + bw
    assert fw >= NCH * (3 * 64 * 64 * e)  # at least W~, Kbar^T, U~
    bad, _ = problem(dk=96)
    for f in (gdn.gdn_chunk_saved_size, gdn.gdn_chunk_fwd_save_workspace_size,
              gdn.gdn_chunk_bwd_saved_workspace_size):
        assert f(bad) == 0


def test_saved_path_rejects_bad_arguments(lib):
    p, _ = problem()
    fake = ctypes.c_void_p(0x10000)
    odd = ctypes.c_void_p(0x10008)
    ns = gdn.gdn_chunk_saved_size(p)
    fw = gdn.gdn_chunk_fwd_save_workspace_size(p)
    bw = gdn.gdn_chunk_bwd_saved_workspace_size(p)
    fargs = [fake] * 5 + [None, fake, None]
    assert lib.gdn_chunk_fwd_save(ctypes.byref(p), *fargs, fake, ns - 1, fake, fw, None) == 8
    assert lib.gdn_chunk_fwd_save(ctypes.byref(p), *fargs, None, ns, fake, fw, None) == 8
    assert lib.gdn_chunk_fwd_save(ctypes.byref(p), *fargs, fake, ns, fake, fw - 1, None) == 5
    assert lib.gdn_chunk_fwd_save(ctypes.byref(p), *fargs, odd, ns, fake, fw, None) == 7
    assert lib.gdn_chunk_fwd_save(ctypes.byref(p), None, *fargs[1:], fake, ns, fake, fw,
                                  None) == 1
    # q, k, v, beta, dO, dht, saved, saved_bytes, dq, dk, dv, dbeta, dlog_alpha, dh0
    bargs = [fake, fake, fake, fake, fake, None, fake, ns, fake, fake, fake, fake, fake, None]
    assert lib.gdn_chunk_bwd_saved(ctypes.byref(p), *bargs, fake, bw - 1, None) == 5
    bargs[7] = ns - 1
    assert lib.gdn_chunk_bwd_saved(ctypes.byref(p), *bargs, fake, bw, None) == 8
    bargs[7] = ns
    for i in (0, 1, 4):  # q, k, dO
        nulled = list(bargs)
        nulled[i] = None
        assert lib.gdn_chunk_bwd_saved(ctypes.byref(p), *nulled, fake, bw, None) == 1
    bargs[4] = None
    bad, _ = problem(dk=96)
    assert lib.gdn_chunk_bwd_saved(ctypes.byref(bad), *bargs, fake, bw, None) == 3


def test_null_gates_are_accepted(lib):
    """log_alpha NULL (alpha == 1) and dlog_alpha NULL are valid: the calls
    get as far as the workspace check."""
    p, _ = problem()
    fake = ctypes.c_void_p(0x10000)
    need = gdn.gdn_chunk_fwd_workspace_size(p)
    assert lib.gdn_chunk_fwd(ctypes.byref(p), fake, fake, fake, fake, None, None, fake, None,
                             fake, need - 1, None) == 5
    needb = gdn.gdn_chunk_bwd_workspace_size(p)
    bargs = [fake] * 4 + [None, None, fake, None] + [fake] * 4 + [None, None]
    assert lib.gdn_chunk_bwd(ctypes.byref(p), *bargs, fake, needb - 1, None) == 5


def test_recurrent_rejects_bad_arguments(lib):
    p, _ = problem()
    fake = ctypes.c_void_p(0x10000)
    odd = ctypes.c_void_p(0x10008)
    args = [fake] * 5 + [None, fake, None]
    assert lib.gdn_recurrent_fwd(ctypes.byref(p), None, *args[1:], None) == 1
    assert lib.gdn_recurrent_fwd(ctypes.byref(p), odd, *args[1:], None) == 7
    bad, _ = problem(dk=96)
    assert lib.gdn_recurrent_fwd(ctypes.byref(bad), *args, None) == 3
    badcu, keep = problem(B=1, cu=[0, 60, 50, 100])
    assert lib.gdn_recurrent_fwd(ctypes.byref(badcu), *args, None) == 4


def test_block_ops_reject_bad_arguments(lib):
    p, _ = problem(dk=256, dv=512)
    fake = ctypes.c_void_p(0x10000)
    odd = ctypes.c_void_p(0x10008)
    need = lib.gdn_conv_silu_workspace_size(ctypes.byref(p), 256, 4)
    assert need > 0
    assert lib.gdn_conv_silu_workspace_size(ctypes.byref(p), 128, 4) == 0  # not dk or dv
    f = lambda dim, W, eps, x, y, n: lib.gdn_conv_silu_fwd(ctypes.byref(p), dim, W, 1, eps, x,
                                                           fake, y, fake, n, None)
    assert f(256, 5, 1e-6, fake, fake, need) == 9
    assert f(256, 0, 1e-6, fake, fake, need) == 9
    assert f(256, 4, -1.0, fake, fake, need) == 9
    assert f(128, 4, 1e-6, fake, fake, need) == 3
    assert f(256, 4, 1e-6, None, fake, need) == 1
    assert f(256, 4, 1e-6, fake, None, need) == 1
    assert f(256, 4, 1e-6, odd, fake, need) == 7
    assert f(256, 4, 1e-6, fake, fake, need - 1) == 5
    assert lib.gdn_conv_silu_bwd(ctypes.byref(p), 512, 4, 0, 1e-6, fake, fake, fake, fake, None,
                                 fake, need, None) == 1
    nw = lib.gdn_norm_gate_workspace_size(ctypes.byref(p))
    assert nw >= 200 // 64 * 512 * 4  # one partial dv-vector per 64 rows
    assert lib.gdn_norm_gate_fwd(ctypes.byref(p), -1.0, fake, fake, fake, fake, None) == 9
    assert lib.gdn_norm_gate_fwd(ctypes.byref(p), 1e-5, fake, None, fake, fake, None) == 1
    assert lib.gdn_norm_gate_bwd(ctypes.byref(p), 1e-5, fake, fake, fake, fake, fake, fake, fake,
                                 fake, nw - 1, None) == 5


def test_binding_converts_int64_cu_seqlens():
    """torch.tensor and cumsum give int64; the kernels read int32.  The binding
    hands the library an int32 copy (kept alive for the call) and checks that
    the host and device copies describe the same number of sequences."""
    import torch
    q = torch.zeros((1, 10, 2, 64), dtype=torch.bfloat16)
    v = torch.zeros((1, 10, 2, 64), dtype=torch.bfloat16)
    cu = torch.tensor([0, 3, 3, 10])  # int64
    p, keep = gdn.make_problem(q, v, cu)
    assert p.num_seqs == 3
    dev = ctypes.cast(p.cu_seqlens, ctypes.POINTER(ctypes.c_int32))
    host = ctypes.cast(p.cu_seqlens_host, ctypes.POINTER(ctypes.c_int32))
    assert [dev[i] for i in range(4)] == [0, 3, 3, 10]
    assert [host[i] for i in range(4)] == [0, 3, 3, 10]
    assert any(t.data_ptr() == p.cu_seqlens for t in keep)
    with pytest.raises(ValueError):
        gdn.make_problem(q, v, cu, torch.tensor([0, 10], dtype=torch.int32))
    with pytest.raises(TypeError):
        gdn.make_problem(q, v, cu.to(torch.float32))


def test_binding_rejects_mismatched_tensors():
    import torch
    q = torch.zeros((1, 10, 2, 64), dtype=torch.bfloat16)
    good = dict(rows=(("k", q.clone()),), gates=(("beta", torch.zeros(1, 10, 2)),),
                states=(("h0", torch.zeros(1, 2, 64, 64), 64),), nstate=1)
    gdn._check_tensors(q, **good)
    bad_cases = [
        dict(good, rows=(("k", q.to(torch.float32)),)),                  # dtype
        dict(good, rows=(("k", q.transpose(1, 2).contiguous().transpose(1, 2)),)),  # strides
        dict(good, gates=(("beta", torch.zeros(1, 10, 2, dtype=torch.float64)),)),
        dict(good, gates=(("beta", torch.zeros(1, 10, 3)),)),           # shape
        dict(good, states=(("h0", torch.zeros(2, 2, 64, 64), 64),)),    # sequences
        dict(good, states=(("h0", torch.zeros(1, 2, 64, 64).to(torch.bfloat16), 64),)),
    ]
    for kw in bad_cases:
        with pytest.raises(ValueError):
            gdn._check_tensors(q, **kw)


def test_noalloc_forward_checks_before_any_hip_call(lib):
    """The no-allocation forward rejects bad arguments and problems whose
    workspace exceeds the static array with a status, before it touches the
    GPU (this runs on a host without one)."""
    assert gdn.NOALLOC_SCRATCH_BYTES == 64 << 20
    fake = ctypes.c_void_p(0x10000)
    # 8 x 4096 tokens x 6 heads at 256/512: 3072 chunk-heads, ~517 MB of workspace
    big, _ = problem(B=8, T=4096, H=6, dk=256, dv=512)
    assert gdn.gdn_chunk_fwd_workspace_size(big) > gdn.NOALLOC_SCRATCH_BYTES
    rc = lib.gdn_chunk_fwd_noalloc(ctypes.byref(big), fake, fake, fake, fake, fake, None, fake,
                                   None, None)
    assert rc == 5  # GDN_ERR_WORKSPACE
    small, _ = problem(B=1, T=64, H=1)
    assert gdn.gdn_chunk_fwd_workspace_size(small) <= gdn.NOALLOC_SCRATCH_BYTES
    rc = lib.gdn_chunk_fwd_noalloc(ctypes.byref(small), None, fake, fake, fake, fake, None, fake,
                                   None, None)
    assert rc == 1  # GDN_ERR_NULL
    bad, _ = problem(dk=96)
    rc = lib.gdn_chunk_fwd_noalloc(ctypes.byref(bad), fake, fake, fake, fake, fake, None, fake,
                                   None, None)
    assert rc == 3  # GDN_ERR_UNSUPPORTED


def test_fused_block_checks_before_any_launch(lib):
    """The fused block's entry points check the prologue description, the
    pointers and the workspace on the host, and return a status before any
    launch (this runs on a host without a GPU)."""
    fake = ctypes.c_void_p(0x10000)
    odd = 0x10008
    p, _ = problem(dk=256, dv=512)
    ws = gdn.gdn_chunk_fwd_workspace_size(p)

    def pro(width=4, eps=1e-6, **kw):
        ptrs = dict(xq=0x10000, xk=0x10000, xv=0x10000, wq=0x10000, wk=0x10000, wv=0x10000)
        ptrs.update(kw)
        return gdn.BlockPrologue(width, eps, *[ptrs[n] for n in ("xq", "xk", "xv", "wq", "wk",
                                                                 "wv")])

    def fwd(pr, prob=p, o=fake, n=ws):
        return lib.gdn_block_fwd(ctypes.byref(prob), None if pr is None else ctypes.byref(pr),
                                 fake, fake, None, o, None, None, None, None, fake, n, None)

    assert fwd(None) == 1                      # GDN_ERR_NULL
    assert fwd(pro(width=0)) == 9              # GDN_ERR_VALUE
    assert fwd(pro(width=5)) == 9
    assert fwd(pro(eps=-1.0)) == 9
    assert fwd(pro(eps=float("inf"))) == 9
    assert fwd(pro(xk=None)) == 1
    assert fwd(pro(wv=None)) == 1
    assert fwd(pro(xv=odd)) == 7               # GDN_ERR_ALIGN
    assert fwd(pro(), o=None) == 1
    assert fwd(pro(), n=ws - 1) == 5           # GDN_ERR_WORKSPACE
    f32, _ = problem(dk=64, dv=64, dtype=gdn.GDN_F32)
    assert fwd(pro(), prob=f32, n=1 << 30) == 3  # GDN_ERR_UNSUPPORTED: bf16 only
    # the saving forward needs the rule's v and a large enough saved buffer
    nsave = gdn.gdn_chunk_saved_size(p)
    wss = gdn.gdn_chunk_fwd_save_workspace_size(p)
    fs = lambda k, n: lib.gdn_block_fwd_save(ctypes.byref(p), ctypes.byref(pro()), fake, fake,
                                             None, fake, None, fake, k, fake, fake, n, fake, wss,
                                             None)
    assert fs(None, nsave) == 1                # the rule's q, k, v are required here
    assert fs(fake, nsave - 1) == 8            # GDN_ERR_SAVED
    # backward: workspace of the rule's backward plus the prologue's buffers
    wb = lib.gdn_block_bwd_saved_workspace_size(ctypes.byref(p), 4)
    assert wb > gdn.gdn_chunk_bwd_saved_workspace_size(p)
    assert lib.gdn_block_bwd_saved_workspace_size(ctypes.byref(p), 5) == 0
    assert lib.gdn_block_bwd_saved_workspace_size(ctypes.byref(p), 1) < wb

    def bwd(pr, n=wb, dxv=fake, q=fake):
        return lib.gdn_block_bwd_saved(ctypes.byref(p), ctypes.byref(pr), q, fake, fake, fake,
                                       fake, None, fake, nsave, fake, fake, dxv, fake, fake, fake,
                                       fake, None, None, fake, n, None)

    assert bwd(pro(), dxv=None) == 1
    assert bwd(pro(), q=None) == 1
    assert bwd(pro(width=7)) == 9
    assert bwd(pro(), n=wb - 1) == 5


# What every launch sequence dereferences, written from the kernels' reads
# and writes: the prep's operands (W~, Kbar^T, U~ and the forward's P and
# e^g Q), what a saving forward keeps (gates, the backward's operands, chunk
# states, V'), the backward's own intermediates (dS, dX, gate partial sums).
_SAVED = {"g", "Kf", "PTf", "TTf", "nWT", "QgT", "Ak", "Sc", "Vp"}
_FWD = {"q", "k", "v", "beta", "o", "g", "Wf", "KbT", "Uc", "Pf", "Qf"}
_BWD_SAVED = {"q", "k", "v", "beta", "dO", "dq", "dk", "dv", "dbeta", "dSc", "dXb",
              "gpart"} | _SAVED
_BLOCK_FWD = {"xq", "xk", "xv", "cwq", "cwk", "cwv", "beta", "o", "g", "Wf", "KbT", "Uc", "Pf",
              "Qf"}
AUDIT_EXPECT = {
    0: _FWD,
    1: _BWD_SAVED | {"Wf", "KbT", "Uc"},
    2: _FWD | _SAVED,
    3: _BWD_SAVED,
    4: {"q", "k", "v", "beta", "o"},
    5: _BLOCK_FWD,
    6: _BLOCK_FWD | _SAVED | {"yq", "yk", "yv"},
    7: _BWD_SAVED | {"xq", "xk", "cwq", "cwk", "info", "seq_chunk0", "bhead", "btail", "bpart",
                     "btmp", "dwq", "dwk"},
}


def test_launch_sequences_audit_their_pointers(lib):
    """Each launch sequence refuses a description that lacks a pointer its
    kernels dereference, and only those: every required field, removed alone,
    is reported; every other field may be missing.  Packed input adds the
    chunk table (the token-by-token form reads the boundaries directly)."""
    names = []
    while lib.gdn_debug_audit_field(len(names)) is not None:
        names.append(lib.gdn_debug_audit_field(len(names)).decode())
    idx = {n: i for i, n in enumerate(names)}
    everything = (1 << len(names)) - 1
    assert lib.gdn_debug_audit(8, everything) == -2
    for seq, need in AUDIT_EXPECT.items():
        assert need <= set(names), need - set(names)
        base = everything & ~(1 << idx["log_alpha"]) & ~(1 << idx["cu"])  # ungated, dense
        assert lib.gdn_debug_audit(seq, base) == -1, seq
        for n in names:
            if n in ("log_alpha", "cu"):
                continue
            got = lib.gdn_debug_audit(seq, base & ~(1 << idx[n]))
            assert got == (idx[n] if n in need else -1), (seq, n, got)
        table = {"info", "seq_chunk0"} if seq != 4 else set()
        packed = base | (1 << idx["cu"])
        for n in ("info", "seq_chunk0"):
            got = lib.gdn_debug_audit(seq, packed & ~(1 << idx[n]))
            assert got == (idx[n] if (n in table or n in need) else -1), (seq, n, got)
