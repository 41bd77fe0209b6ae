"""C ABI checks that need no GPU: the library loads, exports every function
include/rv.h declares, and host-side validation that happens before any
handle exists reports the documented codes."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "rv.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rv_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol(rv):
    lib = ctypes.CDLL(rv.LIB_PATH)
    names = declared_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(rv.EXPORTED) == names


def test_status_strings(rv):
    assert rv.rv_status_str(0) == "ok"
    assert "range" in rv.rv_status_str(-2)
    assert rv.rv_status_str(-99) == "unknown status"


@pytest.mark.parametrize("field,value,msg", [
    ("head_dim", 96, "head_dim"), ("d_model", 100, "multiples of 128"), ("n_kv_heads", 3, "multiple of n_kv_heads"),
    ("vocab", 1001, "vocab"), ("dtype", 7, "dtype"), ("rms_eps", 0.0, "rms_eps"), ("n_layers", 0, "positive"),
])
def test_config_validation(rv, field, value, msg):
    import workload
    cfg = rv.make_config(workload.TINY)
    setattr(cfg, field, value)
    with pytest.raises(rv.RVError) as e:
        rv.rv_model_bytes(cfg)
    assert e.value.name == "RV_E_ARG" and msg in str(e.value)


def test_model_bytes_match_shape(rv):
    import workload
    s = workload.LLAMA8B
    n = rv.rv_model_bytes(rv.make_config(s))
    params = (2 * s.vocab * s.d_model + s.n_layers * (
        s.d_model * (s.n_heads + 2 * s.n_kv_heads) * s.head_dim + s.d_model * s.n_heads * s.head_dim
        + 3 * s.d_model * s.ffn_dim))
    gains = (2 * s.n_layers + 1) * s.d_model * 4  # fp32 RMSNorm gains
    assert params * 2 + gains <= n < params * 2 + gains + 256 * 300


def test_null_arguments_rejected_without_device(rv):
    import workload
    cfg = rv.make_config(workload.TINY)
    h = ctypes.c_void_p()
    st = rv._lib.rv_init_weights(ctypes.byref(cfg), 0, None, 0, None, ctypes.byref(h))
    assert st == -1 and "NULL" in rv.rv_last_error()
    n = ctypes.c_size_t()
    assert rv._lib.rv_cache_bytes(None, 1, 16, 16, 4, ctypes.byref(n)) == -1
    assert rv._lib.rv_verify(None, None, None, 0, None, 0, None, None, None, None) == -1
    assert rv._lib.rv_prefill_cache(None, None, 1, None, None) == -1
