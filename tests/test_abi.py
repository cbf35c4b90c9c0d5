"""The C-ABI library loads without a GPU, exports every entry point that
include/sa.h declares, and rejects invalid arguments with the documented
status before any HIP call (so these run on a machine with no GPU)."""

import ctypes
import os
import re

import pytest

from paper_2302_13451_amd import binding as bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = ctypes.c_void_p(0x10000)   # never dereferenced: every call below fails validation
FAKE_ODD = ctypes.c_void_p(0x10008)


def declared_functions():
    with open(os.path.join(ROOT, "include", "sa.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    return bd.load_library()


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("sa_forward", "sa_backward", "llsa_forward", "llsa_paper_forward", "llsa_backward",
              "llsa_paper_backward", "sa_stream_step", "llsa_stream_step",
              "sa_last_error", "sa_abi_version"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert lib.sa_abi_version() == 1


def fwd(lib, q=FAKE, k=FAKE, v=FAKE, out=FAKE, lse=None, B=2, T=8, H=2, d=64, Lb=2, La=1,
        lengths=None, dtype=bd.SA_BF16):
    return lib.sa_forward(q, k, v, out, lse, B, T, H, d, Lb, La, lengths, dtype, None)


def test_forward_validation(lib):
    assert fwd(lib, B=0) == bd.SA_OK          # empty batch: no-op, no HIP call
    assert fwd(lib, T=0, q=None) == bd.SA_OK
    assert fwd(lib, B=-1) == bd.SA_ERR_INVALID
    assert fwd(lib, Lb=-1) == bd.SA_ERR_INVALID
    assert fwd(lib, La=-3) == bd.SA_ERR_INVALID
    assert fwd(lib, d=48) == bd.SA_ERR_UNSUPPORTED
    assert fwd(lib, d=128) == bd.SA_ERR_UNSUPPORTED
    assert fwd(lib, dtype=7) == bd.SA_ERR_UNSUPPORTED
    assert fwd(lib, q=None) == bd.SA_ERR_NULL
    assert "NULL" in lib.sa_last_error().decode()
    assert fwd(lib, out=None) == bd.SA_ERR_NULL
    assert fwd(lib, k=FAKE_ODD) == bd.SA_ERR_INVALID
    assert fwd(lib, lengths=ctypes.c_void_p(0x10002)) == bd.SA_ERR_INVALID
    assert fwd(lib, B=1 << 16, T=1 << 12, H=1 << 4) == bd.SA_ERR_INVALID   # B*T*H >= 2^31
    assert fwd(lib, T=(1 << 30) + 1, B=1, H=1) == bd.SA_ERR_INVALID


def test_backward_validation(lib):
    def bwd(lse=FAKE, dq=FAKE, B=2, d=64, dtype=bd.SA_BF16):
        return lib.sa_backward(FAKE, FAKE, FAKE, FAKE, lse, FAKE, dq, FAKE, FAKE, B, 8, 2, d, 2, 1,
                               None, dtype, None)
    assert bwd(B=0) == bd.SA_OK
    assert bwd(lse=None) == bd.SA_ERR_NULL
    assert bwd(dq=None) == bd.SA_ERR_NULL
    assert bwd(d=16) == bd.SA_ERR_UNSUPPORTED
    assert bwd(dq=FAKE_ODD) == bd.SA_ERR_INVALID


def test_llsa_validation(lib):
    def ll(q=FAKE, B=2, Lb=2, La=1, d=32):
        return lib.llsa_forward(q, FAKE, FAKE, FAKE, None, B, 8, 2, d, Lb, La, None, bd.SA_F32,
                                None)
    assert ll(B=0) == bd.SA_OK
    assert ll(q=None) == bd.SA_ERR_NULL
    assert ll(La=-1) == bd.SA_ERR_INVALID
    assert ll(d=100) == bd.SA_ERR_UNSUPPORTED


def test_llsa_backward_validation(lib):
    def lb(lse=FAKE, dv=FAKE, B=2, Lb=2, La=1, d=64, dtype=bd.SA_BF16):
        return lib.llsa_backward(FAKE, FAKE, FAKE, FAKE, lse, FAKE, FAKE, FAKE, dv, B, 8, 2, d,
                                 Lb, La, None, dtype, None)
    assert lb(B=0) == bd.SA_OK
    assert lb(lse=None) == bd.SA_ERR_NULL
    assert lb(dv=None) == bd.SA_ERR_NULL
    assert lb(dv=FAKE_ODD) == bd.SA_ERR_INVALID
    assert lb(La=-1) == bd.SA_ERR_INVALID
    assert lb(d=16) == bd.SA_ERR_UNSUPPORTED
    assert lb(dtype=7) == bd.SA_ERR_UNSUPPORTED
    # float32 and every window are supported: those calls reach a launch, so
    # they are exercised by the GPU tests, not here


def test_llsa_paper_forward_validation(lib):
    def lp(lse=FAKE, out=FAKE, B=2, Lb=2, La=3, d=64, dtype=bd.SA_BF16):
        return lib.llsa_paper_forward(FAKE, FAKE, FAKE, out, lse, B, 8, 2, d, Lb, La, None, dtype,
                                      None)
    assert lp(B=0) == bd.SA_OK
    assert lp(lse=None) == bd.SA_ERR_NULL
    assert lp(out=None) == bd.SA_ERR_NULL
    assert lp(out=FAKE_ODD) == bd.SA_ERR_INVALID
    assert lp(La=-1) == bd.SA_ERR_INVALID
    assert lp(La=65) == bd.SA_ERR_INVALID                      # above SA_LLSA_PAPER_MAX_LA
    assert "exceeds 64" in lib.sa_last_error().decode()
    assert lp(d=16) == bd.SA_ERR_UNSUPPORTED
    assert lp(dtype=7) == bd.SA_ERR_UNSUPPORTED


def test_llsa_paper_backward_validation(lib):
    def lb(lse=FAKE, dv=FAKE, B=2, Lb=2, La=1, d=64, dtype=bd.SA_BF16, T=8):
        return lib.llsa_paper_backward(FAKE, FAKE, FAKE, FAKE, lse, FAKE, FAKE, FAKE, dv, B, T, 2,
                                       d, Lb, La, None, dtype, None)
    assert lb(B=0) == bd.SA_OK
    assert lb(lse=None) == bd.SA_ERR_NULL
    assert lb(dv=None) == bd.SA_ERR_NULL
    assert lb(dv=FAKE_ODD) == bd.SA_ERR_INVALID
    assert lb(La=65) == bd.SA_ERR_INVALID
    assert lb(d=16) == bd.SA_ERR_UNSUPPORTED
    assert lb(dtype=7) == bd.SA_ERR_UNSUPPORTED


def test_stream_validation(lib):
    def st(R=11, S=4, Lb=8, La=2, step=FAKE, q=FAKE, d=64):
        return lib.sa_stream_step(q, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, R, step, None, S, 2, d,
                                  Lb, La, None, bd.SA_BF16, None)
    assert st(R=10) == bd.SA_ERR_INVALID        # ring smaller than Lb + La + 1
    assert "smaller than the window" in bd.load_library().sa_last_error().decode()
    assert st(Lb=1000, La=100, R=2000) == bd.SA_ERR_INVALID   # window above the maximum
    assert st(S=0) == bd.SA_OK
    assert st(step=None) == bd.SA_ERR_NULL
    assert st(step=ctypes.c_void_p(0x10002)) == bd.SA_ERR_INVALID
    assert st(q=None) == bd.SA_ERR_NULL
    assert st(S=-1) == bd.SA_ERR_INVALID
    assert st(d=16) == bd.SA_ERR_UNSUPPORTED


def test_llsa_stream_validation(lib):
    def st(R=11, S=4, Lb=8, La=2, step=FAKE, kl=FAKE, d=64):
        return lib.llsa_stream_step(FAKE, FAKE, FAKE, FAKE, kl, FAKE, FAKE, FAKE, FAKE, FAKE,
                                    FAKE, FAKE, R, step, None, None, S, 2, d, Lb, La, None,
                                    bd.SA_BF16, None)
    assert st(R=10) == bd.SA_ERR_INVALID        # ring smaller than Lb + La + 1
    assert "smaller than the window" in lib.sa_last_error().decode()
    assert st(Lb=1000, La=100, R=2000) == bd.SA_ERR_INVALID
    assert st(S=0) == bd.SA_OK
    assert st(step=None) == bd.SA_ERR_NULL
    assert st(kl=None) == bd.SA_ERR_NULL
    assert st(kl=FAKE_ODD) == bd.SA_ERR_INVALID
    assert st(S=-1) == bd.SA_ERR_INVALID
    assert st(d=16) == bd.SA_ERR_UNSUPPORTED


def test_binding_fails_loudly_without_the_library(monkeypatch, tmp_path):
    monkeypatch.setattr(bd, "_lib", None)
    monkeypatch.setattr(bd, "_LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(bd.SAError):
        bd.load_library()


def test_copy_reference_validation(lib):
    cp = lib.sa_copy_reference
    assert cp(FAKE, ctypes.c_void_p(0x20000), 0, 0, None) == bd.SA_OK
    assert cp(FAKE, ctypes.c_void_p(0x20000), 24, 0, None) == bd.SA_ERR_INVALID    # not 16-byte pieces
    assert cp(FAKE, ctypes.c_void_p(0x20000), -16, 0, None) == bd.SA_ERR_INVALID
    assert cp(FAKE, ctypes.c_void_p(0x20000), 64, 2, None) == bd.SA_ERR_INVALID    # no mode 2
    assert cp(None, ctypes.c_void_p(0x20000), 64, 0, None) == bd.SA_ERR_NULL
    assert cp(FAKE_ODD, ctypes.c_void_p(0x20000), 64, 1, None) == bd.SA_ERR_INVALID
    assert cp(FAKE, ctypes.c_void_p(0x10010), 64, 0, None) == bd.SA_ERR_INVALID   # overlap
