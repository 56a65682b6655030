"""The C ABI without a GPU: the library loads, exports every function that
include/llep.h declares, sizes its buffers, and rejects bad arguments on the
host before anything is enqueued."""

import ctypes
import os
import re

import pytest

from conftest import ROOT

B = pytest.importorskip("paper_2601_17111_amd.binding")

HEADER = os.path.join(ROOT, "include", "llep.h")


def _lib():
    if not os.path.exists(B.LIB_PATH):
        pytest.skip("libllep.so not built")
    return B.lib()


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(llep_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_function():
    L = _lib()
    names = _declared()
    assert {"llep_plan", "llep_permute", "llep_grouped_ffn", "llep_combine"} <= set(names)
    for n in names:
        assert hasattr(L, n), f"{n} declared in llep.h but not exported"
    assert set(B.EXPORTED) == set(names)


def test_struct_layouts():
    assert ctypes.sizeof(B.llep_plan_params) == 48
    assert ctypes.sizeof(B.llep_plan_info) == 32
    assert ctypes.sizeof(B.llep_plan_buffers) == 10 * ctypes.sizeof(ctypes.c_void_p)
    assert B.llep_plan_params.capacity.offset == 24
    assert B.llep_plan_params.lam.offset == 32
    assert B.llep_plan_params.mode.offset == 40


def _params(**kw):
    d = dict(T=256, K=2, E=8, P=4, capacity=160)
    d.update(kw)
    return B.make_params(**d)


def test_size_queries():
    _lib()
    p = _params()
    assert B.llep_plan_max_chunks(p) == 2 * 8 + 4
    tiles = -(-256 * 2 // 1024)  # pairs are ranked in tiles of 1024
    # per tile: E counts (then bases), a bad-id flag, E counts per 256-pair slice
    assert B.llep_plan_rank_base_elems(p) == tiles * 8 + tiles + tiles * 4 * 8
    p = _params(T=65536, K=8, E=128, P=8, capacity=72090)
    assert B.llep_plan_rank_base_elems(p) == 512 * 128 + 512 + 512 * 4 * 128
    ws = B.llep_grouped_ffn_workspace_bytes(p, 768, B.LLEP_BF16)
    assert ws >= 65536 * 8 * 768 * 2
    L = B.lib()
    assert L.llep_packed_gate_up_bytes(4, 128, 64, B.LLEP_BF16) == 4 * 128 * 128 * 2
    assert L.llep_packed_down_bytes(4, 128, 64, B.LLEP_F32) == 4 * 128 * 64 * 4
    assert L.llep_packed_down_bytes(4, 128, 64, 7) == 0


@pytest.mark.parametrize("bad", [
    dict(T=-1), dict(K=0), dict(E=0), dict(E=1024, P=8), dict(P=0), dict(P=65, E=130),
    dict(E=10, P=4), dict(capacity=0), dict(T=2**31, K=1), dict(T=2**30, K=2),
])
def test_bad_params_rejected(bad):
    L = _lib()
    p = _params(**bad)
    assert L.llep_plan_max_chunks(ctypes.byref(p)) == -1
    bufs = B.llep_plan_buffers(*([8] * 10))  # never dereferenced on the host
    rc = L.llep_plan(ctypes.byref(p), ctypes.c_void_p(16), ctypes.byref(bufs), None)
    assert rc == B.LLEP_E_ARG
    assert B.last_error() != ""


def test_bad_mode_and_reserved():
    L = _lib()
    bufs = B.llep_plan_buffers(*([8] * 10))
    p = _params()
    p.mode = 5
    assert L.llep_plan(ctypes.byref(p), ctypes.c_void_p(16), ctypes.byref(bufs), None) == B.LLEP_E_ARG
    p = _params()
    p.reserved = 1
    assert L.llep_plan(ctypes.byref(p), ctypes.c_void_p(16), ctypes.byref(bufs), None) == B.LLEP_E_ARG


def test_null_pointers_rejected():
    L = _lib()
    p = _params()
    good = [16 * (i + 1) for i in range(10)]
    for i in range(10):
        ptrs = list(good)
        ptrs[i] = None
        bufs = B.llep_plan_buffers(*ptrs)
        assert L.llep_plan(ctypes.byref(p), ctypes.c_void_p(16), ctypes.byref(bufs), None) == B.LLEP_E_ARG
    bufs = B.llep_plan_buffers(*good)
    assert L.llep_plan(ctypes.byref(p), None, ctypes.byref(bufs), None) == B.LLEP_E_ARG
    assert L.llep_plan(None, ctypes.c_void_p(16), ctypes.byref(bufs), None) == B.LLEP_E_ARG


def test_permute_combine_argument_checks():
    L = _lib()
    p = _params()
    bufs = B.llep_plan_buffers(*[16 * (i + 1) for i in range(10)])
    a = ctypes.c_void_p(4096)
    # D not a whole number of 16-byte vectors
    rc = L.llep_permute(ctypes.byref(p), ctypes.byref(bufs), a, a, a, 12, B.LLEP_BF16, a, a, a, a, None)
    assert rc == B.LLEP_E_ARG
    # unknown dtype
    rc = L.llep_permute(ctypes.byref(p), ctypes.byref(bufs), a, a, a, 64, 9, a, a, a, a, None)
    assert rc == B.LLEP_E_DTYPE
    # misaligned x
    rc = L.llep_permute(ctypes.byref(p), ctypes.byref(bufs), a, a, ctypes.c_void_p(4100), 64,
                        B.LLEP_F32, a, a, a, a, None)
    assert rc == B.LLEP_E_ARG
    rc = L.llep_combine(ctypes.byref(p), a, a, a, 64, B.LLEP_BF16, None, None)
    assert rc == B.LLEP_E_ARG
    rc = L.llep_combine(ctypes.byref(p), a, a, a, 60, B.LLEP_BF16, a, None)
    assert rc == B.LLEP_E_ARG


def test_ffn_argument_checks():
    L = _lib()
    p = _params()
    bufs = B.llep_plan_buffers(*[16 * (i + 1) for i in range(10)])
    a = ctypes.c_void_p(4096)
    ws_need = B.llep_grouped_ffn_workspace_bytes(p, 128, B.LLEP_F32)
    ws = ctypes.c_void_p(1 << 20)
    ok_args = lambda **kw: dict(dict(device=0, D=64, F=128, dtype=B.LLEP_F32, ws=ws, nbytes=ws_need), **kw)

    def call(device, D, F, dtype, ws, nbytes):
        return L.llep_grouped_ffn(ctypes.byref(p), ctypes.byref(bufs), device, a, a, a, D, F,
                                  dtype, a, ws, nbytes, None)
    assert call(**ok_args(D=96)) == B.LLEP_E_ARG          # D % 64
    assert call(**ok_args(F=100)) == B.LLEP_E_ARG         # F % 64
    assert call(**ok_args(D=B.LLEP_MAX_FFN_DIM + 64)) == B.LLEP_E_ARG
    assert call(**ok_args(F=B.LLEP_MAX_FFN_DIM + 64)) == B.LLEP_E_ARG
    assert call(**ok_args(device=4)) == B.LLEP_E_ARG      # device >= P
    assert call(**ok_args(device=-2)) == B.LLEP_E_ARG
    assert call(**ok_args(dtype=3)) == B.LLEP_E_DTYPE
    assert call(**ok_args(nbytes=ws_need - 1)) == B.LLEP_E_WORKSPACE
    assert call(**ok_args(ws=None)) == B.LLEP_E_WORKSPACE
    assert call(**ok_args(ws=ctypes.c_void_p((1 << 20) + 128))) == B.LLEP_E_WORKSPACE

    def train(gate_up, **kw):
        k = ok_args(**kw)
        return L.llep_grouped_ffn_train(ctypes.byref(p), ctypes.byref(bufs), k["device"], a, a, a,
                                        k["D"], k["F"], k["dtype"], a, gate_up, k["ws"],
                                        k["nbytes"], None)
    assert train(None) == B.LLEP_E_ARG                    # gate_up required
    assert train(ctypes.c_void_p(4104)) == B.LLEP_E_ARG   # misaligned
    assert train(a, D=96) == B.LLEP_E_ARG
    assert train(a, nbytes=ws_need - 1) == B.LLEP_E_WORKSPACE
    # pack
    assert L.llep_pack_weights(4, 64, 96, B.LLEP_BF16, a, a, a, a, a, None) == B.LLEP_E_ARG
    assert L.llep_pack_weights(0, 64, 64, B.LLEP_BF16, a, a, a, a, a, None) == B.LLEP_E_ARG
    assert L.llep_pack_weights(4, 64, 64, B.LLEP_BF16, a, None, a, a, a, None) == B.LLEP_E_ARG


def test_backward_argument_checks():
    L = _lib()
    p = _params()
    bufs = B.llep_plan_buffers(*[16 * (i + 1) for i in range(10)])
    a = ctypes.c_void_p(4096)
    bf = B.LLEP_BF16
    # combine backward: dtype, nulls, alignment, D % 8
    assert L.llep_combine_backward(ctypes.byref(p), a, a, a, a, 64, 5, a, a,
                                   None) == B.LLEP_E_DTYPE
    assert L.llep_combine_backward(ctypes.byref(p), a, a, None, a, 64, bf, a, a,
                                   None) == B.LLEP_E_ARG
    assert L.llep_combine_backward(ctypes.byref(p), a, a, a, ctypes.c_void_p(4104), 64, bf, a, a,
                                   None) == B.LLEP_E_ARG
    assert L.llep_combine_backward(ctypes.byref(p), a, a, a, a, 60, bf, a, a, None) == B.LLEP_E_ARG
    # the forward combine accepts null gates (all ones) but not a null output
    assert L.llep_combine(ctypes.byref(p), a, a, None, 64, bf, None, None) == B.LLEP_E_ARG
    # backward packing
    assert L.llep_pack_weights_backward(4, 64, 64, 5, a, a, a, a, a, None) == B.LLEP_E_DTYPE
    assert L.llep_pack_weights_backward(4, 64, 96, bf, a, a, a, a, a, None) == B.LLEP_E_ARG
    assert L.llep_pack_weights_backward(4, 64, 64, bf, a, a, a, None, a, None) == B.LLEP_E_ARG
    # grouped FFN backward
    assert B.llep_grouped_ffn_backward_workspace_bytes(p, 64, 128, 5) == 0
    assert B.llep_grouped_ffn_backward_workspace_bytes(p, 64, 128, B.LLEP_F32) > 0
    need = B.llep_grouped_ffn_backward_workspace_bytes(p, 64, 128, bf)
    # at least the recomputed gate/up values, their gradients and the activation
    assert need >= p.T * p.K * 128 * 2 * 5
    ws = ctypes.c_void_p(1 << 24)
    ok = dict(device=0, D=64, F=128, dtype=bf, ws=ws, nbytes=need, dw=a)

    def call(device, D, F, dtype, ws, nbytes, dw, gate_up=None):
        return L.llep_grouped_ffn_backward(ctypes.byref(p), ctypes.byref(bufs), device, a, a, a, a,
                                           a, gate_up, D, F, dtype, a, dw, a, a, ws, nbytes, None)
    assert call(**dict(ok, dtype=5)) == B.LLEP_E_DTYPE
    assert call(**dict(ok, D=96)) == B.LLEP_E_ARG
    assert call(**dict(ok, device=4)) == B.LLEP_E_ARG
    assert call(**dict(ok, dw=None)) == B.LLEP_E_ARG
    assert call(**dict(ok, dw=ctypes.c_void_p(4100))) == B.LLEP_E_ARG
    assert call(**dict(ok, nbytes=need - 1)) == B.LLEP_E_WORKSPACE
    assert call(**dict(ok, ws=ctypes.c_void_p((1 << 24) + 64))) == B.LLEP_E_WORKSPACE
    assert call(**dict(ok, gate_up=ctypes.c_void_p(4104))) == B.LLEP_E_ARG
    # more pairs than the backward's 32-bit operand offsets reach
    big = B.make_params(1 << 20, 8, 8, 4, (1 << 23) // 4)
    nb = B.llep_grouped_ffn_backward_workspace_bytes(big, 64, 128, bf)
    assert L.llep_grouped_ffn_backward(ctypes.byref(big), ctypes.byref(bufs), 0, a, a, a, a, a,
                                       None, 64, 128, bf, a, a, a, a, ws, nb, None) == B.LLEP_E_ARG
    assert "too large" in B.last_error()


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(B, "_lib", None)
    monkeypatch.setattr(B, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="missing"):
        B.lib()
