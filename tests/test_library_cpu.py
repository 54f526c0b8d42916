"""Host-side checks of the C-ABI library that need no GPU: it loads, it exports
every entry point include/lst.h declares, and argument errors detected on the
host are reported without touching a device."""
import ctypes
import os
import re

import pytest

import paper_1412_7091_amd as lst

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(REPO, "include", "lst.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lst_[a-z_A-Z]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(lst.LIB_PATH):
        pytest.fail("liblst.so is not built (run __graft_entry__.build())")
    return lst.load_library()


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert "lst_step" in names and "lst_init" in names
    for n in names:
        assert hasattr(lib, n), f"{n} declared in include/lst.h but not exported"
    assert set(names) == set(lst.EXPORTED)


def test_strerror(lib):
    assert lst.lst_strerror(lst.LST_OK) == "ok"
    assert "index" in lst.lst_strerror(lst.LST_EINDEX)
    assert lst.lst_strerror(12345) == "unknown status"


def test_null_state_and_bad_config_rejected_on_host(lib):
    assert lib.lst_step(None, 1, 1, None, None, None, 0.1, None, None) == lst.LST_EINVAL
    assert lib.lst_naive_step(None, 1, 1, None, None, None, 0.1, None, None) == lst.LST_EINVAL
    assert lib.lst_sync(None) == lst.LST_EINVAL
    assert lib.lst_materialize_W(None, None) == lst.LST_EINVAL
    lib.lst_free(None)
    h = ctypes.c_void_p()
    fake_dev = ctypes.c_void_p(16)  # never dereferenced: the config is rejected first
    for cfg in (lst.lst_config(7, 1e-3, 4, 4, 0.0),         # unknown loss
                lst.lst_config(0, 1e-3, 0, 4, 0.0),         # m_max < 1
                lst.lst_config(0, 1e-3, 4, 2000, 0.0),      # K_max > 1024
                lst.lst_config(0, 1e-3, 512, 64, 0.0),      # m_max * K_max > 16384
                lst.lst_config(1, 0.0, 4, 1, 0.0),          # spherical needs eps > 0
                lst.lst_config(0, 1e-3, 4, 4, -1.0)):       # cond_max < 0
        assert lib.lst_init(ctypes.byref(h), 10, 4, fake_dev, None, ctypes.byref(cfg), None) \
            == lst.LST_EINVAL
    cfg = lst.lst_config(0, 1e-3, 4, 4, 0.0)
    assert lib.lst_init(ctypes.byref(h), 0, 4, fake_dev, None, ctypes.byref(cfg), None) == lst.LST_EINVAL
    assert lib.lst_init(ctypes.byref(h), 10, 0, fake_dev, None, ctypes.byref(cfg), None) == lst.LST_EINVAL
    assert lib.lst_init(ctypes.byref(h), 10, 4, None, None, ctypes.byref(cfg), None) == lst.LST_EINVAL
    assert h.value is None


def test_stabilize_arguments_rejected_on_host(lib):
    good = lst.lst_stab_config(1e-3, 100.0, 7, 2, 1)
    assert lib.lst_stabilize(None, ctypes.byref(good), None) == lst.LST_EINVAL
    assert lib.lst_set_stabilize(None, 1, ctypes.byref(good)) == lst.LST_EINVAL


def test_input_layer_arguments_rejected_on_host(lib):
    h = ctypes.c_void_p()
    fake_dev = ctypes.c_void_p(16)  # never dereferenced
    assert lib.lst_input_init(ctypes.byref(h), 0, 4, fake_dev, None) == lst.LST_EINVAL
    assert lib.lst_input_init(ctypes.byref(h), 10, 0, fake_dev, None) == lst.LST_EINVAL
    assert lib.lst_input_init(ctypes.byref(h), 10, 4, None, None) == lst.LST_EINVAL
    assert lib.lst_input_forward(None, 1, 1, fake_dev, fake_dev, fake_dev) == lst.LST_EINVAL
    assert lib.lst_input_update(None, 1, 1, fake_dev, fake_dev, fake_dev, 0.1) == lst.LST_EINVAL
    assert lib.lst_input_sync(None) == lst.LST_EINVAL
    lib.lst_input_free(None)
