"""Mutation check of the oracle's pins (CPU).

Each mutant plants one plausible mistake in a copy of the oracle's source (a
dropped term, a wrong sign, index or step size, a swapped operand) and runs
every pin of ``tests/test_oracle_pins.py`` against that copy; at least one pin
must fail.  A mutant that passes every pin names a part of the oracle that
nothing outside the oracle fixes.
"""
import inspect
import os
import sys
import types

import pytest

from tests import test_oracle_pins as pins

ORACLE_SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "uad_oracle.py")

# (name, original text, planted mistake); the first occurrence of the original is replaced.
MUTANTS = [
    ("RMSNorm eps dropped", "np.sqrt(ms + h.dtype.type(eps))", "np.sqrt(ms)"),
    ("GQA head index", "g = (j * Hkv) // Hq", "g = j % Hkv"),
    ("sin / cos swapped", "[np.sin(a64), np.cos(a64)]", "[np.cos(a64), np.sin(a64)]"),
    ("GELU cubic term dropped", "(z + a * z * z * z)", "(z)"),
    ("attention residual dropped", 'h = h + o @ W[p + "wo"].T', 'h = o @ W[p + "wo"].T'),
    ("softmax scale dropped", "s = (q[:, j, :] @ k[:, g, :].T) * scale", "s = q[:, j, :] @ k[:, g, :].T"),
    ("action / time concat order", "np.concatenate([a, e], axis=-1)", "np.concatenate([e, a], axis=-1)"),
    ("MLP norm takes the attention gain", 'n2 = rms_norm(h, W[p + "mlp_norm"]', 'n2 = rms_norm(h, W[p + "attn_norm"]'),
    ("prefix keys and values dropped (input-conditioned expert)",
     "k_all = np.concatenate([m.prefix_k[env][l], k], axis=0)\n        v_all = np.concatenate([m.prefix_v[env][l], v], axis=0)",
     "k_all = k\n        v_all = v"),
    ("TR sum scaled by 1/K", "x0[:, :U] + (-(one / np.float32(Nstar))) * vsum", "x0[:, :U] + (-(one / np.float32(K))) * vsum"),
    ("urgent tokens step by 1/N*", "dt = -(one / budgets.astype(np.float32))\n        v = vf(x, t)",
     "dt = np.full(budgets.shape, -(one / np.float32(Nstar)), np.float32)\n        v = vf(x, t)"),
    ("TR sum starts at the second velocity", "vsum = v[:, :U].copy() if vsum is None else vsum + v[:, :U]",
     "vsum = np.zeros_like(v[:, :U]) if vsum is None else vsum + v[:, :U]"),
    ("ghost flow time one step late", "tk = np.float32(Nstar - k) / np.float32(Nstar)\n        t = np.full((B, H), tk",
     "tk = np.float32(Nstar - k - 1) / np.float32(Nstar)\n        t = np.full((B, H), tk"),
    ("schedule time offset", "t[k] = (N - np.minimum(k, N))", "t[k] = (N - np.minimum(k + 1, N))"),
    ("mask one step late", "mask[k] = (k >= N).astype(np.uint8)", "mask[k] = (k > N).astype(np.uint8)"),
    ("released before the last update", "released[now] = x[now]", "released[now] = x_in[now]"),
    ("frozen token updated as x + 0 v", "return np.where(frozen[..., None], x, upd)", "return upd"),
    ("GAC divisor", "shift = E / tail.dtype.type(n)", "shift = E / tail.dtype.type(n + 1)"),
    ("GAC error sign", "E = np.sum(ghosts - released, axis=1)", "E = np.sum(released - ghosts, axis=1)"),
    ("controller wait", "wait += r - clock", "wait += r"),
    ("vanilla step sign", "dtk = -(np.float32(1) / np.float32(N))", "dtk = np.float32(1) / np.float32(N)"),
    ("adaptive norm scale without 1 +", "return r * (h.dtype.type(1) + scale) + shift", "return r * scale + shift"),
    ("adaptive norm gate dropped", 'h = h + ga * (g @ W[p + "w_down"].T)', 'h = h + (g @ W[p + "w_down"].T)'),
    ("GeGLU gate and up swapped", 'g = gelu_tanh(n2 @ W[p + "w_gate"].T) * (n2 @ W[p + "w_up"].T)',
     'g = gelu_tanh(n2 @ W[p + "w_up"].T) * (n2 @ W[p + "w_gate"].T)'),
    ("chunk keys and values dropped",
     "k_all = np.concatenate([m.prefix_k[env][l], k], axis=0)\n        v_all = np.concatenate([m.prefix_v[env][l], v], axis=0)",
     "k_all = m.prefix_k[env][l]\n        v_all = m.prefix_v[env][l]"),
    ("time MLP SiLU dropped", 'z = silu(u @ W["time_mlp_in.w"].T + W["time_mlp_in.b"])',
     'z = u @ W["time_mlp_in.w"].T + W["time_mlp_in.b"]'),
    ("time frequencies without the 1000 factor", "(1000.0 * np.power(10000.0, -j / (d // 2)))",
     "(np.power(10000.0, -j / (d // 2)))"),
    ("adaptive norm shift dropped", "return r * (h.dtype.type(1) + scale) + shift", "return r * (h.dtype.type(1) + scale)"),
    ("GAC dimension mask ignored", "shift = np.where(np.asarray(dim_mask, bool)[None, :], shift, 0)", "shift = shift"),
    ("adaptive conditioning outer SiLU dropped",
     'c = silu(silu(e @ W["time_mlp_in.w"].T + W["time_mlp_in.b"]) @ W["time_mlp_out.w"].T + W["time_mlp_out.b"])',
     'c = silu(e @ W["time_mlp_in.w"].T + W["time_mlp_in.b"]) @ W["time_mlp_out.w"].T + W["time_mlp_out.b"]'),
    ("final norm takes a layer's gain", 'nf = rms_norm(h, W["final_norm"], m.rms_eps)',
     'nf = rms_norm(h, W["layers.0.mlp_norm"], m.rms_eps)'),
]


def _load_mutant(old: str, new: str) -> types.ModuleType:
    src = open(ORACLE_SRC).read()
    assert old in src, f"mutation site absent: {old!r}"
    name = "oracle_mutant"
    mod = types.ModuleType(name)
    mod.__file__ = ORACLE_SRC
    sys.modules[name] = mod  # dataclasses look their module up while the class is built
    try:
        exec(compile(src.replace(old, new, 1), ORACLE_SRC + " (mutant)", "exec"), mod.__dict__)
    finally:
        del sys.modules[name]
    return mod


def _pin_cases():
    """Every pin test of test_oracle_pins with each of its parameter sets."""
    cases = []
    for name, fn in sorted(vars(pins).items()):
        if not name.startswith("test_") or not callable(fn):
            continue
        params = [{}]
        for mark in getattr(fn, "pytestmark", []):
            if mark.name != "parametrize":
                continue
            argnames, values = mark.args[0], mark.args[1]
            names = [a.strip() for a in argnames.split(",")] if isinstance(argnames, str) else list(argnames)
            expanded = []
            for p in params:
                for v in values:
                    v = v if len(names) > 1 else (v,)
                    expanded.append({**p, **dict(zip(names, v))})
            params = expanded
        assert set(inspect.signature(fn).parameters) <= set(params[0]), f"{name} needs fixtures"
        cases.extend((name, fn, p) for p in params)
    return cases


def test_unmodified_source_passes_every_pin(monkeypatch):
    """The mutant loader itself changes nothing: the oracle's own source, loaded the same way, passes."""
    src_mod = _load_mutant("def silu(", "def silu(")
    monkeypatch.setattr(pins, "O", src_mod)
    for name, fn, kw in _pin_cases():
        fn(**kw)


@pytest.mark.parametrize("label,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_fails_a_pin(monkeypatch, label, old, new):
    mut = _load_mutant(old, new)
    monkeypatch.setattr(pins, "O", mut)
    for name, fn, kw in _pin_cases():
        try:
            fn(**kw)
        except Exception as e:
            print(f"mutant '{label}' fails {name}{kw or ''}: {type(e).__name__}")
            return
    pytest.fail(f"mutant '{label}' passes every oracle pin")
