"""The C-ABI library loads and exports every entry point include/gift.h
declares (no GPU: only calls that touch no device)."""
import os
import re
import subprocess
import sys

import pytest

from paper_2608_25431_amd import gift

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = set()
    for h in os.listdir(os.path.join(ROOT, "include")):
        if h.endswith(".h"):
            src = open(os.path.join(ROOT, "include", h)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names |= set(re.findall(r"\b(gift_[a-z_]+)\s*\(", src))
    return names


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(gift.LIB_PATH):
        from paper_2608_25431_amd import build
        build.build()
    return gift.lib()


def test_header_declares_the_documented_api():
    assert declared_functions() == set(gift.EXPORTS)


def test_every_declared_symbol_is_exported(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", gift.LIB_PATH], capture_output=True, text=True).stdout
    exported = {l.split()[-1] for l in out.splitlines() if l.strip()}
    for name in declared_functions():
        assert name in exported, name
        assert hasattr(lib, name)


def test_status_strings(lib):
    for s in range(-9, 1):
        assert gift.status_string(s)
    assert gift.status_string(-100) == "unknown status"
    assert gift.last_error() == ""


def test_binding_fails_loudly_without_the_library(tmp_path, monkeypatch):
    monkeypatch.setattr(gift, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(gift, "_lib", None)
    with pytest.raises(ImportError):
        gift.lib()


def test_null_key_table_is_rejected_on_the_host(lib):
    import ctypes
    t = gift._Tensor(None, 0, 16)
    tab = gift._SegTable(None, 0, None, None)
    assert lib.gift_seal(ctypes.byref(t), ctypes.byref(tab), None, None, None, None, None) == gift.E_INVALID
    assert lib.gift_key_table_create(None, 1, None, ctypes.byref(ctypes.c_void_p())) == gift.E_INVALID
    assert lib.gift_key_table_destroy(None) == gift.OK
    assert lib.gift_key_table_users(None) == 0


def test_loads_beside_torchs_hip_runtime(lib):
    # torch ships its own libamdhip64, which a process that imports torch first
    # has loaded: the library may only use entry points that runtime exports
    code = ("import sys, ctypes, torch; sys.path.insert(0, %r); "
            "from paper_2608_25431_amd import gift; ctypes.CDLL(gift.LIB_PATH)" % ROOT)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
