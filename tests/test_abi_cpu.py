"""The C ABI loads and exports every symbol include/stage.h declares, and the
argument checks that run before any device work return the documented codes
(CPU only: no compute call is made)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2608_19147_amd as pkg
from paper_2608_19147_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2608_19147_amd import build

        build.build()
    return _lib.load()


def header_functions():
    src = open(os.path.join(ROOT, "include", "stage.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"^(?:const\s+)?\w+\s*\*?\s+(\w+)\s*\(", src, flags=re.M)
    return sorted(set(names))


def test_header_matches_binding():
    assert header_functions() == sorted(_lib.EXPORTS)


def test_every_symbol_exported(lib):
    for name in header_functions():
        assert hasattr(lib, name), name


def _cfg(**kw):
    base = dict(n_layers=1, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn=688, group_size=128,
                rms_eps=1e-5, act_dtype=_lib.DTYPE_F16, kv_dtype=_lib.DTYPE_F16, rope_theta=500000.0,
                max_positions=128, rope_cos_sin=None)
    base.update(kw)
    return _lib.StageConfig(**base)


def _create(lib, cfg, layers=None):
    h = ctypes.c_void_p()
    if layers is None:
        layers = (_lib.LayerWeights * max(1, cfg.n_layers))()
    return lib.stage_create(ctypes.byref(cfg), layers, 0, None, ctypes.byref(h)), h


@pytest.mark.parametrize("kw,code", [
    (dict(head_dim=96), -7),
    (dict(n_kv_heads=3), -1),
    (dict(group_size=100), -7),
    (dict(act_dtype=7), -1),
    (dict(n_layers=0), -1),
    (dict(rms_eps=0.0), -1),
    (dict(hidden=252), -7),
])
def test_config_rejected(lib, kw, code):
    rc, h = _create(lib, _cfg(**kw))
    assert rc == code
    assert h.value is None
    assert lib.stage_last_error()


def test_null_arguments(lib):
    h = ctypes.c_void_p()
    assert lib.stage_create(None, None, 0, None, ctypes.byref(h)) == -1
    assert b"NULL" in lib.stage_last_error()
    assert lib.stage_forward(None, None, 0, None, None, None) == -1
    assert lib.kv_truncate(None, 0) == -1
    assert lib.kv_state_alloc(None, 1, 1, ctypes.byref(h)) == -1
    assert lib.stage_destroy(None) == -1
    assert lib.stage_weight_bytes(None) == -1


def test_matrix_shape_checked_before_device_work(lib):
    """A layer whose wq has the wrong N is rejected with STAGE_E_SHAPE."""
    cfg = _cfg()
    layers = (_lib.LayerWeights * 1)()
    bufs = []
    dims = {"wq": (256, 256), "wk": (128, 256), "wv": (128, 256), "wo": (256, 256),
            "wg": (688, 256), "wu": (688, 256), "wd": (256, 688)}
    for name, (n, k) in dims.items():
        q = np.zeros((n, k // 2), np.uint8)
        s = np.zeros((n, (k + 127) // 128), np.uint16)
        bufs += [q, s]
        setattr(layers[0], name, _lib.QuantMatrix(q=q.ctypes.data, scales=s.ctypes.data, n=n, k=k))
    g = np.ones(256, np.uint16)
    layers[0].attn_norm = g.ctypes.data
    layers[0].ffn_norm = g.ctypes.data
    layers[0].wq.n = 255
    rc, _ = _create(lib, cfg, layers)
    assert rc == -2 and b"wq" in lib.stage_last_error()


def test_package_exports():
    assert set(pkg.EXPORTS) == set(header_functions())
