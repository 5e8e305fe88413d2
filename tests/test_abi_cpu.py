"""Host-side checks of the C ABI library that need no GPU."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pictura.h")
LIB = os.path.join(ROOT, "paper_2607_26005_amd", "libpictura.so")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pictura_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_2607_26005_amd import build
        build.build()
    return ctypes.CDLL(LIB)


def test_every_declared_symbol_is_exported(lib):
    names = _declared()
    assert "pictura_render_views" in names and "pictura_scene_upload" in names and "pictura_bin_scene" in names
    for n in names:
        assert hasattr(lib, n), n


def test_binding_names_match_header(lib):
    from paper_2607_26005_amd import pictura
    assert sorted(pictura.EXPORTED) == _declared()


def test_create_without_device_is_edevice(lib):
    import torch
    if torch.cuda.device_count() > 0:
        pytest.skip("a HIP device is present")
    h = ctypes.c_void_p()
    lib.pictura_create.argtypes = [ctypes.c_int32, ctypes.POINTER(ctypes.c_void_p)]
    assert lib.pictura_create(0, ctypes.byref(h)) == -3
    assert h.value is None
