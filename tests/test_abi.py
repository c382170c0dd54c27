"""The C-ABI library loads and exports every entry point include/gift.h
declares (no GPU: only calls that touch no device)."""
import os
import re
import subprocess
import sys

import numpy as np
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


def test_binding_rejects_host_and_short_device_buffers():
    # checked before the library is called, so no GPU is needed: a host buffer
    # or a short one would otherwise reach the kernels as a device address
    torch = pytest.importorskip("torch")
    import types
    kt = types.SimpleNamespace(handle=None, n_users=1)
    nb = np.zeros(12, np.uint8)
    cpu = torch.zeros(64, dtype=torch.uint8)
    with pytest.raises(ValueError, match="on the GPU"):
        gift.seal(cpu, 1, 64, [(0, 1, 0, 0)], kt, nb, cpu, cpu)
    with pytest.raises(ValueError, match="host memory"):
        gift.seal(np.zeros(64, np.uint8), 1, 64, [(0, 1, 0, 0)], kt, nb, 0, 0)


class _FakeCuda:
    """Stands in for a CUDA tensor of n bytes at a fake address."""

    is_cuda = True

    def __init__(self, n, contiguous=True):
        self.n, self.contiguous = n, contiguous

    def data_ptr(self):
        return 1 << 40

    def is_contiguous(self):
        return self.contiguous

    def numel(self):
        return self.n

    def element_size(self):
        return 1


def test_binding_checks_device_buffer_sizes():
    import types
    kt = types.SimpleNamespace(handle=None, n_users=1)
    nb = np.zeros(12, np.uint8)
    segs = [(0, 1, 0, 0), (1, 1, 0, 1)]
    ok = _FakeCuda(128)
    with pytest.raises(ValueError, match="tags: 16 bytes, the call needs 32"):
        gift.seal(ok, 2, 64, segs, kt, nb, ok, _FakeCuda(16))
    with pytest.raises(ValueError, match="out: 100 bytes"):
        gift.seal(ok, 2, 64, segs, kt, nb, _FakeCuda(100), ok)
    with pytest.raises(ValueError, match="verdicts: 4 bytes"):
        gift.open(ok, 2, 64, segs, kt, nb, ok, ok, _FakeCuda(4))
    with pytest.raises(ValueError, match="row_labels: 4 bytes"):
        gift.seal(ok, 2, 64, segs, kt, nb, ok, ok, row_labels=_FakeCuda(4))
    with pytest.raises(ValueError, match="contiguous"):
        gift.seal(ok, 2, 64, segs, kt, nb, _FakeCuda(128, contiguous=False), ok)
    with pytest.raises(ValueError, match="nonces: 8 bytes"):
        gift.token_encrypt(segs, _FakeCuda(16), _FakeCuda(8), 2, kt, 0, _FakeCuda(32))


def test_lds_probe_library_exports_its_entry_point(lib):
    """The benchmark's LDS-rate probes live in a library of their own, which
    exports one C entry point and nothing of the hot path."""
    from paper_2608_25431_amd import build
    assert os.path.exists(build.PROBE_LIB)
    out = subprocess.run(["nm", "-D", "--defined-only", build.PROBE_LIB], capture_output=True, text=True).stdout
    exported = {l.split()[-1] for l in out.splitlines() if l.strip()}
    assert "gift_probe_lds" in exported
    assert not (exported & declared_functions())
