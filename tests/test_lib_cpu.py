"""Host-side checks of the C ABI that need no GPU: the library loads and
exports every entry point the public headers declare, and the binding's
marshalling table covers them."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2607_17299_amd", "libwar.so")


def _declared():
    names = set()
    for h in ("war.h", "war_debug.h"):
        text = open(os.path.join(ROOT, "include", h)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(war_[a-z0-9_]+)\s*\(", text))
    return names


@pytest.mark.skipif(not os.path.exists(LIB), reason="libwar.so not built")
def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(LIB)
    declared = _declared()
    assert {"war_verify_step", "war_kv_commit", "war_prefill_append", "war_kv_alloc",
            "war_kv_free"} <= declared
    for name in sorted(declared):
        assert hasattr(lib, name), name


@pytest.mark.skipif(not os.path.exists(LIB), reason="libwar.so not built")
def test_binding_covers_every_declared_symbol():
    from paper_2607_17299_amd import war
    assert _declared() == set(war.EXPORTS)
    war.load_library()


@pytest.mark.skipif(not os.path.exists(LIB), reason="libwar.so not built")
def test_config_validation_without_gpu():
    # argument checks run before any device call
    from paper_2607_17299_amd import synth, war
    lib = war.load_library()
    bad = war.config_struct(synth.TINY, 64)
    bad.head_dim = 96
    h = ctypes.c_void_p()
    arr = (ctypes.c_void_p * 17)()
    assert lib.war_model_create(ctypes.byref(bad), arr, 17, ctypes.byref(h)) == -4
    ok = war.config_struct(synth.TINY, 64)
    assert lib.war_weight_count(ctypes.byref(ok)) == 3 + 7 * synth.TINY.n_layers
    assert lib.war_model_create(ctypes.byref(ok), arr, 5, ctypes.byref(h)) == -1
    assert b"weight" in lib.war_last_error()
