"""Host-side checks of the C ABI that need no GPU: symbols, schedule tables, AAL, validation."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle as O
import uad_workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def uad():
    import paper_2609_37772_amd as U
    if not os.path.exists(U.LIB_PATH):
        pytest.fail("libuad.so is not built (run python -m paper_2609_37772_amd.build)")
    U.load_library()
    return U


def declared_symbols():
    src = open(os.path.join(ROOT, "include", "uad.h")).read()
    return sorted(set(re.findall(r"\b(uad_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol(uad):
    lib = ctypes.CDLL(uad.LIB_PATH)
    decl = declared_symbols()
    assert len(decl) >= 13
    for name in decl:
        assert hasattr(lib, name), f"libuad.so does not export {name}"
    assert sorted(decl) == sorted(uad.EXPORTED_SYMBOLS)


@pytest.mark.parametrize("wl", W.WORKLOAD_ORDER)
def test_schedule_builder_matches_oracle_bit_exact(uad, wl):
    bud = W.make_budgets(W.get_workload(wl))
    n, t, dt, mask = uad.uad_build_schedule(bud)
    n2, t2, dt2, mask2 = O.build_schedule(bud)
    assert n == n2
    assert t.tobytes() == t2.tobytes()
    assert dt.tobytes() == dt2.tobytes()
    assert mask.tobytes() == mask2.tobytes()


def test_schedule_builder_edge_cases(uad):
    n, t, dt, mask = uad.uad_build_schedule(np.array([[1]]))
    assert n == 1 and t[0, 0, 0] == 1.0 and dt[0, 0, 0] == -1.0 and mask[0, 0, 0] == 0
    bud = np.array([[64, 1, 3]])
    n, t, dt, mask = uad.uad_build_schedule(bud, max_steps=64)
    n2, t2, dt2, mask2 = O.build_schedule(bud)
    assert n == 64 and t.tobytes() == t2.tobytes() and mask.tobytes() == mask2.tobytes()
    for bad in (np.array([[0, 2]]), np.array([[65]]), np.array([[-3]])):
        with pytest.raises(uad.UadError):
            uad.uad_build_schedule(bad, max_steps=64)


def test_aal_matches_oracle_controller(uad):
    rng = np.random.default_rng(0)
    for _ in range(100):
        rel = np.sort(rng.uniform(0, 50, 10))
        tact = float(rng.uniform(0, 20))
        assert abs(uad.uad_aal(rel, tact) - O.aal_controller(rel, tact)) < 1e-12
    with pytest.raises(uad.UadError):
        uad.uad_aal(np.zeros(0), 1.0)


def _cfg(uad, **kw):
    base = dict(n_layers=1, d_model=64, n_heads=2, n_kv_heads=1, head_dim=64, d_ff=128, action_dim=4,
                max_batch=1, max_chunk=8, max_prefix=8, rms_eps=1e-6, flags=0)
    base.update(kw)
    return uad._binding.uad_model_config(**base)


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 96, 7), ("d_model", 48, 7), ("n_kv_heads", 3, 7), ("action_dim", 65, 7),
    ("n_layers", 0, 1), ("max_batch", 0, 1), ("flags", 2, 1), ("flags", -1, 1),
])
def test_create_validates_before_device_work(uad, field, value, status):
    lib = uad.load_library()
    cfg = _cfg(uad, **{field: value})
    out = ctypes.c_void_p(1234)
    st = lib.uad_create(ctypes.byref(cfg), 0, None, ctypes.byref(out))
    assert st == status
    assert out.value is None
    assert len(uad.uad_last_error(None)) > 0


def test_null_context_is_rejected(uad):
    lib = uad.load_library()
    assert lib.uad_synchronize(None) == 1
    assert lib.uad_denoise_step(None, None, None, None, None, None, 1, 1) == 1
    assert lib.uad_load_weights(None, None, 0) == 1
