"""C-ABI checks that need no GPU: every declared symbol is exported, and every
argument error is reported before any HIP call."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lrqat.h")

lrqat = pytest.importorskip("paper_2406_06385_amd.lrqat")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lrqat_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(lrqat.LIB_PATH):
        pytest.skip("liblrqat.so not built")
    return lrqat._lib()


def test_every_declared_symbol_is_exported(lib):
    names = _declared_functions()
    assert len(names) >= 11
    out = subprocess.run(["nm", "-D", "--defined-only", lrqat.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (lrqat_\w+)", out))
    assert set(names) <= exported, set(names) - exported
    for n in names:
        assert hasattr(lib, n)


def _layer(**kw):
    base = dict(out_features=64, in_features=128, rank=8, alpha=8.0, bits=4, phi_format="q8",
                group_size=0, act_bits=0, act_dtype="bf16")
    base.update(kw)
    return lrqat.LayerSpec(**base).c_struct()


FAKE = 1 << 20          # a 256-byte aligned dummy device address, never dereferenced
BAD_ALIGN = FAKE + 2


def _fwd(lib, L, T=16, X=FAKE, ws_bytes=1 << 30, Y=FAKE, z=None):
    P = ctypes.c_void_p
    return lib.lrqat_forward(ctypes.byref(L), T, P(X), P(FAKE), P(FAKE), P(z) if z else None, P(FAKE), P(FAKE),
                             P(Y), P(FAKE), ws_bytes, None)


def _bwd(lib, L, T=16, ds=None, accumulate=0, dX=FAKE, ws_bytes=1 << 30, z=None):
    P = ctypes.c_void_p
    return lib.lrqat_backward(ctypes.byref(L), T, P(FAKE), P(FAKE), P(FAKE), P(z) if z else None, P(FAKE), P(FAKE),
                              P(FAKE), P(dX), P(FAKE), P(FAKE), P(ds) if ds else None, accumulate, P(FAKE), ws_bytes,
                              None)


def _bwd_static(lib, L, T=16):
    P = ctypes.c_void_p
    return lib.lrqat_backward_static(ctypes.byref(L), T, P(FAKE), P(FAKE), P(FAKE), None, P(FAKE), P(FAKE),
                                     P(FAKE), P(FAKE), P(FAKE), P(FAKE), None, 0, None)


@pytest.mark.parametrize("kw,status", [
    (dict(bits=8), lrqat.LRQAT_EINVAL),
    (dict(bits=1), lrqat.LRQAT_EINVAL),
    (dict(bits=5), lrqat.LRQAT_OK),
    (dict(bits=7), lrqat.LRQAT_OK),
    (dict(bits=5, phi_format="int_packed2"), lrqat.LRQAT_EINVAL),
    (dict(in_features=127, phi_format="int_packed2"), lrqat.LRQAT_EINVAL),
    (dict(group_size=48), lrqat.LRQAT_EINVAL),
    (dict(group_size=64, in_features=192), lrqat.LRQAT_OK),
    (dict(group_size=16, in_features=128), lrqat.LRQAT_EUNSUPPORTED),
    (dict(rank=0), lrqat.LRQAT_EINVAL),
    (dict(rank=257), lrqat.LRQAT_EINVAL),
    (dict(out_features=0), lrqat.LRQAT_EINVAL),
    (dict(alpha=float("inf")), lrqat.LRQAT_EINVAL),
    (dict(act_bits=4), lrqat.LRQAT_EINVAL),
    (dict(act_bits=8, act_dtype="fp32"), lrqat.LRQAT_EUNSUPPORTED),
])
def test_layer_validation(lib, kw, status):
    L = _layer(**kw)
    if status == lrqat.LRQAT_OK:
        assert lib.lrqat_forward_workspace_size(ctypes.byref(L), 16) > 0
        return
    assert lib.lrqat_forward_workspace_size(ctypes.byref(L), 16) == 0
    assert _fwd(lib, L) == status
    assert _bwd(lib, L) == status
    assert lib.lrqat_last_error().decode() != ""


def test_pointer_and_workspace_errors(lib):
    L = _layer()
    assert _fwd(lib, L, X=0) == lrqat.LRQAT_EINVAL
    assert b"X is NULL" in lib.lrqat_last_error()
    assert _fwd(lib, L, X=BAD_ALIGN) == lrqat.LRQAT_EINVAL
    assert _fwd(lib, L, Y=BAD_ALIGN) == lrqat.LRQAT_EINVAL
    need = lib.lrqat_forward_workspace_size(ctypes.byref(L), 16)
    assert _fwd(lib, L, ws_bytes=need - 1) == lrqat.LRQAT_EWORKSPACE
    assert _fwd(lib, L, T=-1) == lrqat.LRQAT_EINVAL
    assert _fwd(lib, L, T=0) == lrqat.LRQAT_OK          # no-op, launches nothing
    assert _bwd(lib, L, ds=BAD_ALIGN) == lrqat.LRQAT_EINVAL
    assert _fwd(lib, L, z=BAD_ALIGN) == lrqat.LRQAT_EINVAL
    assert _bwd(lib, L, accumulate=2) == lrqat.LRQAT_EINVAL
    assert _bwd(lib, L, dX=BAD_ALIGN) == lrqat.LRQAT_EINVAL
    needb = lib.lrqat_backward_workspace_size(ctypes.byref(L), 16)
    assert _bwd(lib, L, ws_bytes=needb - 1) == lrqat.LRQAT_EWORKSPACE
    P = ctypes.c_void_p
    assert lib.lrqat_merge_to_int4(ctypes.byref(_layer(in_features=127)), P(FAKE), P(FAKE), P(FAKE), P(FAKE),
                                   None) == lrqat.LRQAT_EINVAL
    assert lib.lrqat_merge_to_int4(ctypes.byref(L), P(FAKE), P(FAKE), P(FAKE), P(0), None) == lrqat.LRQAT_EINVAL
    assert lib.lrqat_init_from_weights(ctypes.byref(L), P(0), P(FAKE), None, P(FAKE), None) == lrqat.LRQAT_EINVAL
    assert lib.lrqat_init_from_weights(ctypes.byref(L), P(FAKE), P(FAKE), P(BAD_ALIGN), P(FAKE),
                                       None) == lrqat.LRQAT_EINVAL
    # inference on merged weights: int4 only, argument checks before any launch
    assert lib.lrqat_infer_forward(ctypes.byref(_layer(bits=5)), 16, P(FAKE), P(FAKE), P(FAKE), None, P(FAKE),
                                   P(FAKE), 1 << 30, None) == lrqat.LRQAT_EINVAL
    assert lib.lrqat_infer_forward(ctypes.byref(L), 16, P(0), P(FAKE), P(FAKE), None, P(FAKE), P(FAKE), 1 << 30,
                                   None) == lrqat.LRQAT_EINVAL
    La = _layer(act_bits=8)  # W4A8 needs workspace for the activation codes
    assert lib.lrqat_infer_forward(ctypes.byref(La), 16, P(FAKE), P(FAKE), P(FAKE), None, P(FAKE), P(FAKE), 0,
                                   None) == lrqat.LRQAT_EWORKSPACE
    assert lib.lrqat_infer_workspace_size(ctypes.byref(L), 16) >= 256
    assert lib.lrqat_forward(None, 16, P(FAKE), P(FAKE), P(FAKE), None, P(FAKE), P(FAKE), P(FAKE), P(FAKE),
                             1 << 30, None) == lrqat.LRQAT_EINVAL


def test_static_backward_rejects_layers_beyond_its_array(lib):
    """The no-allocation backward refuses, before any HIP call, a layer whose
    scratch would not fit the library's device array."""
    cap = lib.lrqat_backward_static_capacity()
    assert cap == 64 << 20
    big = _layer(out_features=14336, in_features=4096, rank=32)
    assert lib.lrqat_backward_workspace_size(ctypes.byref(big), 8192) > cap
    assert _bwd_static(lib, big, T=8192) == lrqat.LRQAT_EWORKSPACE
    assert b"lrqat_backward_static" in lib.lrqat_last_error()
    assert _bwd_static(lib, _layer(bits=1)) == lrqat.LRQAT_EINVAL


def test_workspace_sizes_grow_with_tokens_and_backward(lib):
    for kw in (dict(), dict(act_bits=8, phi_format="int_packed2"), dict(act_dtype="fp32")):
        L = _layer(**kw)
        f1 = lib.lrqat_forward_workspace_size(ctypes.byref(L), 1)
        b1 = lib.lrqat_backward_workspace_size(ctypes.byref(L), 1)
        assert 0 < f1 <= b1
        assert f1 % 256 == 0 and b1 % 256 == 0
        f2 = lib.lrqat_forward_workspace_size(ctypes.byref(L), 4096)
        assert f2 >= f1
        assert (f2 > f1) == (kw.get("act_bits", 0) == 8)


def test_status_strings(lib):
    for code, name in enumerate(["LRQAT_OK", "LRQAT_EINVAL", "LRQAT_EUNSUPPORTED", "LRQAT_EWORKSPACE", "LRQAT_EHIP"]):
        assert lib.lrqat_status_string(code).decode() == name
