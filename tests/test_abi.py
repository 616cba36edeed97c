"""CPU checks of the C-ABI library: it loads, exports every symbol that
include/polyglot.h declares, and rejects bad arguments before touching the GPU
(host-side validation; no compute call is made here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "polyglot.h")


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(polyglot_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    import paper_1404_1521_amd as pg
    if not os.path.exists(pg.LIB_PATH):
        pytest.fail("libpolyglot.so is not built (run __graft_entry__.build())")
    return pg.load_library()


def test_header_declares_the_binding_exports():
    import paper_1404_1521_amd as pg
    assert declared_symbols() == sorted(pg.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_symbols():
        assert hasattr(lib, name), name


def test_header_compiles_as_c():
    import subprocess
    import tempfile
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "t.c")
        with open(src, "w") as f:
            f.write('#include "polyglot.h"\nint main(void){polyglot_config c={0};(void)c;return 0;}\n')
        r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I",
                            os.path.join(ROOT, "include"), "-c", src, "-o",
                            os.path.join(d, "t.o")], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr


def _cfg(**kw):
    import paper_1404_1521_amd as pg
    base = dict(V=1000, d=16, win=5, H=8, max_batch=32, scatter_mode=0, max_scatter=0,
                max_rows=0)
    base.update(kw)
    return pg.Config(**base)


@pytest.mark.parametrize("kw", [
    dict(d=24), dict(d=0), dict(d=272), dict(win=4), dict(win=0), dict(win=33), dict(H=0),
    dict(H=65), dict(V=0), dict(win=9, d=64), dict(scatter_mode=2), dict(max_scatter=-1),
    dict(max_scatter=10, max_rows=0),
    # W1 (64 x 388 floats) and the tile buffers exceed one workgroup's 160 KiB of LDS
    dict(H=48, d=128, win=3),
    # hidden layers above 64 units: multiples of 64 up to 256, d a multiple of 64
    dict(H=96, d=64), dict(H=128, d=80), dict(H=320, d=64),
])
def test_init_rejects_bad_config_before_any_device_call(lib, kw):
    import paper_1404_1521_amd as pg
    h = ctypes.c_void_p(123)
    rc = lib.polyglot_init(ctypes.byref(_cfg(**kw)), None, ctypes.byref(h))
    assert rc == pg.EINVAL
    assert h.value is None


def test_init_rejects_bad_batch(lib):
    import paper_1404_1521_amd as pg
    h = ctypes.c_void_p()
    assert lib.polyglot_init(ctypes.byref(_cfg(max_batch=0)), None, ctypes.byref(h)) == pg.EBATCH


def test_null_context_is_rejected(lib):
    import paper_1404_1521_amd as pg
    assert lib.polyglot_init(None, None, None) == pg.ENULL
    assert lib.polyglot_destroy(None) == pg.ENULL
    assert lib.polyglot_status(None) == pg.ENULL
    assert lib.polyglot_train_step(None, *([None] * 7), 1, ctypes.c_float(0.1), None) == pg.ENULL
    assert lib.polyglot_train_steps(None, *([None] * 7), 1, 1, ctypes.c_float(0.1),
                                    None) == pg.ENULL
    loss = ctypes.c_float(7.0)
    assert lib.polyglot_train_step_sync(None, *([None] * 7), 1, ctypes.c_float(0.1),
                                        ctypes.byref(loss)) == pg.ENULL
    assert lib.polyglot_train_step_sync(None, *([None] * 7), 1, ctypes.c_float(0.1),
                                        None) == pg.ENULL
    assert loss.value == 7.0
    assert lib.polyglot_score(None, *([None] * 6), 1, None) == pg.ENULL
    assert lib.polyglot_gather(None, None, None, None, 1, None, None) == pg.ENULL
    assert lib.polyglot_scatter_add(None, None, 1, 4, None, None, 1, ctypes.c_float(1.0),
                                    0) == pg.ENULL
    assert lib.polyglot_touched_rows(None, None, 0, None) == pg.ENULL
    assert lib.polyglot_last_error(None) == b""


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    import paper_1404_1521_amd as pg
    monkeypatch.setattr(pg, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(pg, "_lib", None)
    with pytest.raises(RuntimeError, match="not built"):
        pg.load_library()
