"""The C ABI on the CPU: the library loads, exports every symbol the header declares, and
rejects bad arguments before any HIP call (so these run without a GPU). The same tests run a
second time, in a child process, against a build of the library with AddressSanitizer and
UndefinedBehaviorSanitizer on its host code."""
import ctypes
import math
import os
import re
import subprocess
import sys

import pytest

from paper_2105_08810_amd import snn

# set in the child process of test_validation_under_sanitizers: the sanitized library
SAN_LIB = os.environ.get("SNN_ABI_SANITIZED_LIB")

NAN = float("nan")
INF = math.inf
FAKE = 0x1000  # never dereferenced: every call below must fail validation first


@pytest.fixture(scope="module")
def lib():
    if SAN_LIB:
        l = ctypes.CDLL(SAN_LIB)
        for name, (res, args) in snn._SIGNATURES.items():
            getattr(l, name).restype = res
            getattr(l, name).argtypes = args
        return l
    if not os.path.exists(snn.LIB_PATH):
        from paper_2105_08810_amd import build
        build.build(verbose=False)
    return snn.lib()


def test_exports_every_declared_symbol(lib):
    with open(snn.HEADER) as f:
        text = f.read()
    declared = set(re.findall(r"\b(snn_[a-z_]+)\s*\(", text))
    assert {"snn_lif_forward", "snn_active_compact", "snn_sparse_backward", "snn_dense_backward_ref"} <= declared
    raw = ctypes.CDLL(SAN_LIB or snn.LIB_PATH)
    for name in sorted(declared):
        assert hasattr(raw, name), name
    assert declared == set(snn._SIGNATURES), "binding and header disagree"


def test_status_strings(lib):
    assert snn.status_string(0) == "SNN_OK"
    assert snn.status_string(-1) == "SNN_ERR_INVALID_ARG"
    assert snn.status_string(-2) == "SNN_ERR_UNSUPPORTED"
    assert snn.status_string(-3) == "SNN_ERR_HIP"
    assert snn.status_string(12345) == "SNN_UNKNOWN_STATUS"


def _fwd(lib, **kw):
    a = dict(s_in=FAKE, W=FAKE, T=10, B=4, N_in=32, N_out=16, alpha=0.9, theta=1.0, V=FAKE, s_out=FAKE,
             trace=FAKE, stream=None)
    a.update(kw)
    return lib.snn_lif_forward(a["s_in"], a["W"], a["T"], a["B"], a["N_in"], a["N_out"], a["alpha"], a["theta"],
                               a["V"], a["s_out"], a["trace"], a["stream"])


@pytest.mark.parametrize("kw", [dict(s_in=None), dict(W=None), dict(V=None), dict(s_out=None), dict(T=0),
                                dict(B=-1), dict(N_in=0), dict(N_out=0), dict(alpha=0.0), dict(alpha=1.5),
                                dict(alpha=NAN), dict(theta=NAN), dict(T=70000, B=70000)])
def test_forward_rejects(lib, kw):
    assert _fwd(lib, **kw) == snn.SNN_ERR_INVALID_ARG


def test_forward_unsupported_width(lib):
    assert _fwd(lib, N_out=5000) == snn.SNN_ERR_UNSUPPORTED


def _cmp(lib, **kw):
    a = dict(V=FAKE, T=10, B=4, N=16, theta=1.0, b_th=0.2, beta=100.0, row_ptr=FAKE, col_idx=FAKE, g=FAKE, cap=100,
             nnz=FAKE, ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    return lib.snn_active_compact(a["V"], a["T"], a["B"], a["N"], a["theta"], a["b_th"], a["beta"], a["row_ptr"],
                                  a["col_idx"], a["g"], a["cap"], a["nnz"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw", [dict(V=None), dict(row_ptr=None), dict(nnz=None), dict(ws=None), dict(N=0),
                                dict(b_th=-0.1), dict(b_th=NAN), dict(theta=NAN), dict(beta=NAN), dict(beta=-1.0),
                                dict(cap=-1), dict(col_idx=None), dict(ws_bytes=8)])
def test_compact_rejects(lib, kw):
    assert _cmp(lib, **kw) == snn.SNN_ERR_INVALID_ARG


def test_workspace_queries(lib):
    assert lib.snn_active_compact_workspace(10, 4, 16) > 0
    assert lib.snn_active_compact_workspace(0, 4, 16) == 0
    assert lib.snn_sparse_backward_workspace(500, 256, 1024, 1024, 10 ** 6) > 0
    assert lib.snn_sparse_backward_workspace(10, 4, 0, 16, 10) == 0
    assert lib.snn_sparse_backward_workspace(10, 4, 8, 16, -1) == 0
    # the slab-major entry copy grows with the entry capacity (layers of more than 300 outputs, or
    # of more than 1024 inputs, that do not take the matrix cores); layers of 33..300 outputs and
    # at most 1024 inputs read the CSR directly and narrow layers use a dense G of T*B*N_out,
    # whatever the capacity
    assert (lib.snn_sparse_backward_workspace(10, 4, 8, 2048, 10 ** 5)
            > lib.snn_sparse_backward_workspace(10, 4, 8, 2048, 10))
    assert (lib.snn_sparse_backward_workspace(10, 4, 8, 64, 10 ** 5)
            == lib.snn_sparse_backward_workspace(10, 4, 8, 64, 10) > 0)
    assert (lib.snn_sparse_backward_workspace(10, 4, 8, 16, 10 ** 5)
            == lib.snn_sparse_backward_workspace(10, 4, 8, 16, 10) >= 2 * 10 * 4 * 16 * 4)
    assert lib.snn_dense_backward_workspace(500, 256, 1024, 1024) >= 2 * 500 * 256 * 1024 * 4
    assert lib.snn_readout_ce_workspace(10, 4, 3, 0) > 0
    assert lib.snn_readout_ce_workspace(10, 4, 3, 2) == 0
    # deterministic: the same dimensions always give the same size
    assert (lib.snn_sparse_backward_workspace(100, 256, 784, 200, 5000)
            == lib.snn_sparse_backward_workspace(100, 256, 784, 200, 5000))


def _sb(lib, **kw):
    a = dict(W=FAKE, tr=FAKE, T=10, B=4, N_in=32, N_out=16, alpha=0.9, orp=FAKE, oci=FAKE, og=FAKE, oeps=FAKE,
             ocap=10, irp=FAKE, ici=FAKE, icap=10, eps_in=FAKE, dW=FAKE, ws=FAKE, ws_bytes=1 << 40)
    a.update(kw)
    return lib.snn_sparse_backward(a["W"], a["tr"], a["T"], a["B"], a["N_in"], a["N_out"], a["alpha"], a["orp"],
                                   a["oci"], a["og"], a["oeps"], a["ocap"], a["irp"], a["ici"], a["icap"],
                                   a["eps_in"], a["dW"], a["ws"], a["ws_bytes"], None, None)


@pytest.mark.parametrize("kw", [dict(W=None), dict(tr=None), dict(orp=None), dict(dW=None), dict(oci=None),
                                dict(oeps=None), dict(alpha=2.0), dict(ocap=-1), dict(icap=-5), dict(ws_bytes=16),
                                dict(irp=None), dict(eps_in=None), dict(T=0), dict(N_out=-3)])
def test_sparse_backward_rejects(lib, kw):
    assert _sb(lib, **kw) == snn.SNN_ERR_INVALID_ARG


def test_sparse_backward_unsupported_width(lib):
    assert _sb(lib, N_out=5000) == snn.SNN_ERR_UNSUPPORTED


def _db(lib, **kw):
    a = dict(W=FAKE, tr=FAKE, V=FAKE, eps=FAKE, T=10, B=4, N_in=32, N_out=16, alpha=0.9, theta=1.0, b_th=0.2,
             beta=100.0, gi=FAKE, dW=FAKE, ws=FAKE, ws_bytes=1 << 40)
    a.update(kw)
    return lib.snn_dense_backward_ref(a["W"], a["tr"], a["V"], a["eps"], a["T"], a["B"], a["N_in"], a["N_out"],
                                      a["alpha"], a["theta"], a["b_th"], a["beta"], a["gi"], a["dW"], a["ws"],
                                      a["ws_bytes"], None)


@pytest.mark.parametrize("kw", [dict(W=None), dict(eps=None), dict(dW=None), dict(V=None), dict(b_th=-1.0),
                                dict(beta=NAN), dict(theta=NAN), dict(alpha=-0.5), dict(ws_bytes=4), dict(B=0)])
def test_dense_backward_rejects(lib, kw):
    assert _db(lib, **kw) == snn.SNN_ERR_INVALID_ARG


@pytest.mark.parametrize("kw", [dict(mode=2), dict(V=None), dict(labels=None), dict(C=0), dict(ws_bytes=1)])
def test_readout_rejects(lib, kw):
    a = dict(V=FAKE, labels=FAKE, T=10, B=4, C=3, mode=0, rp=FAKE, ci=FAKE, eps=FAKE, loss=FAKE, dense=None,
             ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    st = lib.snn_readout_ce(a["V"], a["labels"], a["T"], a["B"], a["C"], a["mode"], a["rp"], a["ci"], a["eps"],
                            a["loss"], a["dense"], a["ws"], a["ws_bytes"], None)
    assert st == snn.SNN_ERR_INVALID_ARG


def _sdw(lib, **kw):
    a = dict(tr=FAKE, T=10, B=4, N_in=32, N_out=16, orp=FAKE, oci=FAKE, og=FAKE, oeps=FAKE, ocap=10, dW=FAKE, ws=FAKE,
             ws_bytes=1 << 40)
    a.update(kw)
    return lib.snn_sparse_dw(a["tr"], a["T"], a["B"], a["N_in"], a["N_out"], a["orp"], a["oci"], a["og"], a["oeps"],
                             a["ocap"], a["dW"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw", [dict(tr=None), dict(dW=None), dict(orp=None), dict(oci=None), dict(oeps=None),
                                dict(ocap=-1), dict(ws=None), dict(ws_bytes=8), dict(T=0), dict(N_in=-2)])
def test_sparse_dw_rejects(lib, kw):
    assert _sdw(lib, **kw) == snn.SNN_ERR_INVALID_ARG


def test_sparse_dw_unsupported_width(lib):
    assert _sdw(lib, N_out=5000) == snn.SNN_ERR_UNSUPPORTED


def _sds(lib, **kw):
    a = dict(s=FAKE, ck=FAKE, K=8, alpha=0.9, T=10, B=4, N_in=32, N_out=16, orp=FAKE, oci=FAKE, og=FAKE, oeps=FAKE,
             ocap=10, dW=FAKE, ws=FAKE, ws_bytes=1 << 40)
    a.update(kw)
    return lib.snn_sparse_dw_spikes(a["s"], a["ck"], a["K"], a["alpha"], a["T"], a["B"], a["N_in"], a["N_out"],
                                    a["orp"], a["oci"], a["og"], a["oeps"], a["ocap"], a["dW"], a["ws"], a["ws_bytes"],
                                    None)


@pytest.mark.parametrize("kw", [dict(s=None), dict(ck=None), dict(K=0), dict(alpha=1.5), dict(alpha=NAN),
                                dict(dW=None), dict(orp=None), dict(oeps=None), dict(ocap=-1), dict(ws=None),
                                dict(ws_bytes=8), dict(T=0)])
def test_sparse_dw_spikes_rejects(lib, kw):
    assert _sds(lib, **kw) == snn.SNN_ERR_INVALID_ARG


def test_sparse_dw_spikes_unsupported_width_and_sizes(lib):
    assert _sds(lib, N_out=5000) == snn.SNN_ERR_UNSUPPORTED
    assert lib.snn_trace_checkpoint_count(500, 32) == 16
    assert lib.snn_trace_checkpoint_count(17, 1) == 17
    assert lib.snn_trace_checkpoint_count(0, 4) == 0 and lib.snn_trace_checkpoint_count(10, 0) == 0
    assert lib.snn_sparse_dw_spikes_workspace(500, 256, 1024, 1024, 10 ** 6, 32) > 0
    assert lib.snn_sparse_dw_spikes_workspace(500, 256, 1024, 1024, 10 ** 6, 0) == 0
    for kw in (dict(s=None), dict(ck=None), dict(K=0), dict(alpha=0.0), dict(B=0)):
        a = dict(s=FAKE, T=10, B=4, N_in=32, alpha=0.9, K=4, ck=FAKE)
        a.update(kw)
        assert lib.snn_trace_checkpoints(a["s"], a["T"], a["B"], a["N_in"], a["alpha"], a["K"], a["ck"],
                                         None) == snn.SNN_ERR_INVALID_ARG


@pytest.mark.parametrize("kw", [dict(orp=None), dict(oci=None), dict(ocap=-1), dict(ws=None), dict(ws_bytes=8),
                                dict(T=0), dict(N_in=-2)])
def test_sparse_dw_layout_rejects(lib, kw):
    a = dict(T=10, B=4, N_in=32, N_out=16, orp=FAKE, oci=FAKE, ocap=10, ws=FAKE, ws_bytes=1 << 40)
    a.update(kw)
    assert lib.snn_sparse_dw_layout(a["T"], a["B"], a["N_in"], a["N_out"], a["orp"], a["oci"], a["ocap"], a["ws"],
                                    a["ws_bytes"], None) == snn.SNN_ERR_INVALID_ARG


@pytest.mark.parametrize("kw", [dict(tr=None), dict(dW=None), dict(orp=None), dict(oeps=None), dict(ws_bytes=8)])
def test_sparse_dw_prepared_rejects(lib, kw):
    a = dict(tr=FAKE, T=10, B=4, N_in=32, N_out=16, orp=FAKE, oci=FAKE, og=FAKE, oeps=FAKE, ocap=10, dW=FAKE,
             ws=FAKE, ws_bytes=1 << 40)
    a.update(kw)
    assert lib.snn_sparse_dw_prepared(a["tr"], a["T"], a["B"], a["N_in"], a["N_out"], a["orp"], a["oci"], a["og"],
                                      a["oeps"], a["ocap"], a["dW"], a["ws"], a["ws_bytes"],
                                      None) == snn.SNN_ERR_INVALID_ARG


def _sgi(lib, **kw):
    a = dict(W=FAKE, T=10, B=4, N_in=32, N_out=16, alpha=0.9, orp=FAKE, oci=FAKE, og=FAKE, oeps=FAKE, ocap=10,
             irp=FAKE, ici=FAKE, icap=10, eps_in=FAKE, share=1, ws=FAKE, ws_bytes=1 << 40)
    a.update(kw)
    return lib.snn_sparse_grad_in(a["W"], a["T"], a["B"], a["N_in"], a["N_out"], a["alpha"], a["orp"], a["oci"],
                                  a["og"], a["oeps"], a["ocap"], a["irp"], a["ici"], a["icap"], a["eps_in"],
                                  a["share"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw", [dict(W=None), dict(alpha=0.0), dict(alpha=NAN), dict(orp=None), dict(oeps=None),
                                dict(irp=None), dict(ici=None), dict(eps_in=None), dict(icap=-1), dict(ws=None),
                                dict(ws_bytes=4), dict(B=0)])
def test_sparse_grad_in_rejects(lib, kw):
    assert _sgi(lib, **kw) == snn.SNN_ERR_INVALID_ARG


def test_split_workspaces(lib):
    dw = lib.snn_sparse_dw_workspace(500, 256, 1024, 1024, 10 ** 6)
    gi = lib.snn_sparse_grad_in_workspace(500, 256, 1024)
    assert dw > 0 and gi > 0
    assert lib.snn_sparse_backward_workspace(500, 256, 1024, 1024, 10 ** 6) >= dw + gi
    assert lib.snn_sparse_grad_in_workspace(0, 256, 1024) == 0


def test_fused_forward_rejects(lib):
    f = lambda **kw: lib.snn_lif_forward_active(  # noqa: E731
        kw.get("s", FAKE), FAKE, 10, 4, 32, 16, 0.9, 1.0, kw.get("b", 0.2), FAKE, FAKE, FAKE, kw.get("bits", FAKE),
        None)
    assert f(bits=None) == snn.SNN_ERR_INVALID_ARG
    assert f(b=NAN) == snn.SNN_ERR_INVALID_ARG
    assert f(b=-0.5) == snn.SNN_ERR_INVALID_ARG
    assert f(s=None) == snn.SNN_ERR_INVALID_ARG
    assert lib.snn_active_bits_words(10, 4, 16) == 10  # ceil(4 * 16 / 64) words per step
    assert lib.snn_active_bits_words(3, 5, 100) == 3 * 8
    assert lib.snn_active_bits_words(0, 5, 100) == 0


def test_forward_traces_rejects(lib):
    f = lambda **kw: lib.snn_lif_forward_traces(  # noqa: E731
        kw.get("s", FAKE), FAKE, 10, 4, 32, 16, 0.9, 1.0, kw.get("b", 0.2), FAKE, FAKE, FAKE, kw.get("to", FAKE),
        kw.get("an", 0.9), kw.get("bits", FAKE), None)
    for an in (0.0, -0.5, 1.5, NAN):  # the output trace's leak must lie in (0, 1]
        assert f(an=an) == snn.SNN_ERR_INVALID_ARG
    assert f(b=NAN) == snn.SNN_ERR_INVALID_ARG
    assert f(b=-0.5) == snn.SNN_ERR_INVALID_ARG
    assert f(s=None) == snn.SNN_ERR_INVALID_ARG
    assert f(s=None, to=None, bits=None, an=NAN, b=NAN) == snn.SNN_ERR_INVALID_ARG


def _cb(lib, **kw):
    a = dict(bits=FAKE, V=FAKE, T=10, B=4, N=16, theta=1.0, beta=100.0, rp=FAKE, ci=FAKE, g=FAKE, cap=100, nnz=FAKE,
             ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    return lib.snn_active_compact_bits(a["bits"], a["V"], a["T"], a["B"], a["N"], a["theta"], a["beta"], a["rp"],
                                       a["ci"], a["g"], a["cap"], a["nnz"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw", [dict(bits=None), dict(rp=None), dict(nnz=None), dict(ws=None), dict(ws_bytes=4),
                                dict(cap=-1), dict(ci=None), dict(V=None), dict(beta=NAN), dict(N=0)])
def test_compact_bits_rejects(lib, kw):
    assert _cb(lib, **kw) == snn.SNN_ERR_INVALID_ARG


def test_compact_bits_v_optional_without_g(lib):
    # V may be NULL when no g is asked for: validation passes that point and fails on the
    # (deliberately) missing workspace instead
    assert _cb(lib, V=None, g=None, ws=None) == snn.SNN_ERR_INVALID_ARG
    assert lib.snn_active_compact_bits_workspace(10, 4, 16) > 0


def _cbn(lib, **kw):
    a = dict(bits=FAKE, V=FAKE, T=10, B=4, N=16, theta=1.0, beta=100.0, rp=FAKE, ci=FAKE, g=FAKE, cap=100, nnz=FAKE)
    a.update(kw)
    return lib.snn_active_compact_bits_noalloc(a["bits"], a["V"], a["T"], a["B"], a["N"], a["theta"], a["beta"],
                                               a["rp"], a["ci"], a["g"], a["cap"], a["nnz"], None)


@pytest.mark.parametrize("kw", [dict(bits=None), dict(rp=None), dict(nnz=None), dict(cap=-1), dict(ci=None),
                                dict(V=None), dict(beta=NAN), dict(theta=NAN), dict(N=0), dict(T=-1)])
def test_compact_bits_noalloc_rejects(lib, kw):
    assert _cbn(lib, **kw) == snn.SNN_ERR_INVALID_ARG


def test_compact_bits_noalloc_size_limit(lib):
    # the library's device array holds 8 MiB: the row counts and scan temporaries of at most
    # about 2e6 rows; larger inputs are refused before any HIP call
    limit = 8 << 20
    assert lib.snn_active_compact_bits_workspace(2000, 1000, 64) <= limit
    assert lib.snn_active_compact_bits_workspace(3000, 1000, 64) > limit
    assert _cbn(lib, T=3000, B=1000, N=64) == snn.SNN_ERR_UNSUPPORTED
    assert _cbn(lib, T=100000, B=100000, N=64) == snn.SNN_ERR_INVALID_ARG  # T*B past int32, as for the other form


def _reg(lib, **kw):
    a = dict(S=FAKE, T=10, B=4, N=16, ll=100.0, nl=0.001, lu=0.06, nu=1.0, zeta=FAKE, coef=FAKE, pen=FAKE, ws=FAKE,
             ws_bytes=1 << 30)
    a.update(kw)
    return lib.snn_activity_reg(a["S"], a["T"], a["B"], a["N"], a["ll"], a["nl"], a["lu"], a["nu"], a["zeta"],
                                a["coef"], a["pen"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw", [dict(S=None), dict(coef=None), dict(ws=None), dict(ws_bytes=16), dict(T=0),
                                dict(N=-1), dict(ll=-1.0), dict(lu=NAN), dict(ll=INF), dict(nl=NAN), dict(nu=INF),
                                dict(T=70000, B=70000)])
def test_activity_reg_rejects(lib, kw):
    assert _reg(lib, **kw) == snn.SNN_ERR_INVALID_ARG


def test_activity_reg_workspace(lib):
    # 2048 target blocks over 65536 quads of 256 threads: 8 chunks of 63 steps at T=500, B=256, N=1024
    assert lib.snn_activity_reg_workspace(500, 256, 1024) >= 8 * 256 * 1024 * 4 + 256 * 8
    assert lib.snn_activity_reg_workspace(0, 4, 16) == 0
    assert lib.snn_activity_reg_workspace(20, 4, 32) >= 20 * 4 * 32 * 4


@pytest.mark.parametrize("kw", [dict(coef=None), dict(eps=None), dict(T=0), dict(B=-1),
                                dict(rp=FAKE, ci=None), dict(rp=FAKE, cap=-1)])
def test_activity_reg_grad_rejects(lib, kw):
    a = dict(coef=FAKE, T=10, B=4, N=16, rp=None, ci=FAKE, cap=10, eps=FAKE)
    a.update(kw)
    assert lib.snn_activity_reg_grad(a["coef"], a["T"], a["B"], a["N"], a["rp"], a["ci"], a["cap"], a["eps"],
                                     None) == snn.SNN_ERR_INVALID_ARG


@pytest.mark.parametrize("kw", [dict(W=None), dict(g=None), dict(m=None), dict(v=None), dict(n=0), dict(step=0),
                                dict(lr=-1e-3), dict(lr=NAN), dict(b1=1.0), dict(b2=-0.1), dict(b2=NAN),
                                dict(eps=0.0), dict(eps=INF)])
def test_adam_rejects(lib, kw):
    a = dict(W=FAKE, g=FAKE, m=FAKE, v=FAKE, n=100, lr=1e-3, b1=0.9, b2=0.999, eps=1e-8, step=1)
    a.update(kw)
    assert lib.snn_adam_step(a["W"], a["g"], a["m"], a["v"], a["n"], a["lr"], a["b1"], a["b2"], a["eps"], a["step"],
                             None) == snn.SNN_ERR_INVALID_ARG


def test_conv_entry_points_reject(lib):
    E = snn.SNN_ERR_INVALID_ARG
    f = lambda **kw: lib.snn_conv_lif_forward(  # noqa: E731
        kw.get("x", FAKE), kw.get("w", FAKE), kw.get("T", 10), 4, kw.get("H", 8), 8, 1, kw.get("F", 64),
        kw.get("a", 0.9), kw.get("th", 1.0), kw.get("b", 0.2), kw.get("V", FAKE), FAKE, FAKE, kw.get("bits", FAKE), None)
    for kw in (dict(x=None), dict(w=None), dict(V=None), dict(T=0), dict(F=0), dict(a=0.0), dict(a=NAN),
               dict(th=NAN), dict(b=NAN), dict(b=-1.0), dict(H=70000, T=70000)):
        assert f(**kw) == E, kw
    assert lib.snn_maxpool_spikes(None, 10, 4, 8, 8, 64, FAKE, FAKE, None) == E
    assert lib.snn_maxpool_spikes(FAKE, 10, 4, 7, 8, 64, FAKE, FAKE, None) == E  # odd height
    assert lib.snn_maxpool_spikes(FAKE, 10, 4, 8, 8, 64, FAKE, None, None) == E
    assert lib.snn_pool_route_bits(FAKE, FAKE, 10, 4, 8, 9, 64, FAKE, None) == E  # odd width
    assert lib.snn_pool_route_bits(None, FAKE, 10, 4, 8, 8, 64, FAKE, None) == E
    assert lib.snn_pool_scatter_eps(10, 4, 8, 8, 64, FAKE, FAKE, -1, FAKE, FAKE, FAKE, FAKE, 5, FAKE, None) == E
    assert lib.snn_pool_scatter_eps(10, 4, 8, 8, 64, FAKE, None, 5, FAKE, FAKE, FAKE, FAKE, 5, FAKE, None) == E
    assert lib.snn_pool_scatter_eps(10, 4, 8, 8, 64, FAKE, FAKE, 5, FAKE, FAKE, FAKE, FAKE, 5, None, None) == E
    assert lib.snn_pool_scatter_eps_dense(FAKE, None, 10, 4, 8, 8, 64, FAKE, None) == E
    ws = lib.snn_conv_sparse_dw_workspace(10, 4, 8, 8, 1, 64)
    assert ws >= 9 * 64 * 8 and lib.snn_conv_sparse_dw_workspace(10, 4, 7, 8, 1, 64) == 0
    assert lib.snn_conv_sparse_dw(FAKE, 10, 4, 8, 8, 1, 64, FAKE, FAKE, FAKE, FAKE, 100, FAKE, FAKE, 8, None) == E
    assert lib.snn_conv_sparse_dw(FAKE, 10, 4, 8, 8, 1, 64, FAKE, None, FAKE, FAKE, 100, FAKE, FAKE, ws, None) == E
    assert lib.snn_conv_sparse_dw(FAKE, 10, 4, 8, 8, 64, 64, FAKE, FAKE, FAKE, FAKE, 100, FAKE, FAKE, 1 << 40,
                                  None) == snn.SNN_ERR_UNSUPPORTED
    pooled = lambda **kw: lib.snn_conv_sparse_dw_pooled(  # noqa: E731
        FAKE, kw.get("v", FAKE), kw.get("arg", FAKE), 10, 4, kw.get("H", 8), 8, kw.get("C", 1), 64,
        kw.get("theta", 1.0), kw.get("b_th", 0.2), kw.get("beta", 100.0), FAKE, kw.get("col", FAKE), FAKE,
        kw.get("cap", 100), FAKE, FAKE, kw.get("ws", ws), None)
    for kw in ({"v": None}, {"arg": None}, {"col": None}, {"cap": -1}, {"H": 7}, {"theta": math.nan},
               {"b_th": -1.0}, {"b_th": math.nan}, {"beta": -1.0}, {"ws": 8}):
        assert pooled(**kw) == E, kw
    assert pooled(C=64, ws=1 << 40) == snn.SNN_ERR_UNSUPPORTED
    wd = lib.snn_conv_dense_dw_workspace(10, 4, 8, 8, 1, 64)
    assert wd > 0 and lib.snn_conv_dense_dw_workspace(10, 4, 7, 8, 1, 64) == 0
    assert lib.snn_conv_dense_dw(FAKE, FAKE, FAKE, 10, 4, 8, 8, 1, 64, 1.0, NAN, 100.0, FAKE, FAKE, wd, None) == E
    assert lib.snn_conv_dense_dw(FAKE, None, FAKE, 10, 4, 8, 8, 1, 64, 1.0, 0.2, 100.0, FAKE, FAKE, wd, None) == E
    assert lib.snn_conv_dense_dw(FAKE, FAKE, FAKE, 10, 4, 8, 8, 4096, 512, 1.0, 0.2, 100.0, FAKE, FAKE, 1 << 40,
                                 None) == snn.SNN_ERR_UNSUPPORTED


@pytest.mark.skipif(SAN_LIB is not None, reason="runs in the parent process only")
def test_validation_under_sanitizers():
    """Every test above, in a child process, against libsnn_san.so (host code built with
    -fsanitize=address,undefined, no recovery): any out-of-bounds access, overflow or other
    undefined behaviour in the argument checks, workspace queries or plans ends the child."""
    from paper_2105_08810_amd import build
    path = build.build_sanitized()
    env = dict(os.environ)
    env.update(SNN_ABI_SANITIZED_LIB=path, LD_PRELOAD=build.asan_runtime(),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", __file__],
                       capture_output=True, text=True, env=env, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert " passed" in out
