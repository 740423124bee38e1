"""Seeded synthetic workloads for the UAD action-expert hot path.

This module is shared by the CPU oracle, the tests and the benchmark.  It holds
*only* workload definitions and seeded random draws (model shapes, random-init
weights, cached prefix K/V, initial noise and per-token step budgets); none of
the method's arithmetic (no schedule tables, no embeddings, no network) lives
here.

The paper evaluates trained SmolVLA / pi0.5 experts on LIBERO-Plus, Meta-World+
and a real robot; those weights and benchmarks are not available, so these
random-init workloads stand in for them with the paper's chunk structure
(chunk H=50, executed prefix S=10, per-token budgets; Sec. 4.2, App. C.1) and
the action-expert shapes listed below.

Random streams: every named tensor draws from its own PCG64 stream seeded with
``SeedSequence([seed, crc32(name)])`` so that any tensor can be regenerated in
isolation (e.g. one environment of a batch).
"""
from __future__ import annotations

import dataclasses
import zlib
from typing import Dict, Iterator, List, Optional, Tuple

import numpy as np

__all__ = [
    "ModelShape", "Workload", "WORKLOADS", "get_workload", "weight_specs",
    "draw", "round_to_bf16", "bf16_bits", "make_weights", "make_prefix",
    "make_noise", "make_budgets", "weight_param_count",
]


@dataclasses.dataclass(frozen=True)
class ModelShape:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    action_dim: int
    rms_eps: float = 1e-6
    # "input": time embedding concatenated to the action token before the time
    # MLP; "adarms": time MLP output modulates every RMSNorm (scale, shift) and
    # gates every residual branch (App. C.1, the pi0.5-style variant)
    conditioning: str = "input"


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    shape: ModelShape
    batch: int
    chunk: int          # H, actions per chunk
    prefix: int         # P, cached vision-language prefix tokens per layer
    budget_kind: str    # "uniform" | "groups" | "random" | "linear"
    budget_arg: tuple
    bf16: bool          # canonical weights / prefix rounded once to bf16
    seed: int = 0
    executed: int = 10  # S, executed prefix of the chunk (App. C.1)


# Shapes of the five synthetic workloads (sizes in tokens, dims in elements).
WORKLOADS: Dict[str, Workload] = {
    # 2 layers, width 256, 4 heads x 64 (MHA), GeGLU 1024, prefix 64, H=16, Da=7,
    # 10 uniform steps, fp32 weights.
    "tiny": Workload("tiny", ModelShape(2, 256, 4, 4, 64, 1024, 7), 1, 16, 64,
                     "uniform", (10,), bf16=False),
    # pi0-scale expert at batch 1: 18 layers, width 1024, 8 q heads / 1 kv head
    # of 256, GeGLU 4096, prefix 816, H=50, Da=32, 10 uniform steps.
    "pi0_b1": Workload("pi0_b1", ModelShape(18, 1024, 8, 1, 256, 4096, 32), 1, 50, 816,
                       "uniform", (10,), bf16=True),
    # same model, UAD budgets: actions 0-4 get 4 steps, 5-24 get 7, 25-49 get 10.
    "pi0_b1_uad": Workload("pi0_b1_uad", ModelShape(18, 1024, 8, 1, 256, 4096, 32), 1, 50, 816,
                           "groups", ((5, 4), (20, 7), (25, 10)), bf16=True),
    # 64 independent environments, per-environment random UAD schedule.
    "pi0_fleet_b64": Workload("pi0_fleet_b64", ModelShape(18, 1024, 8, 1, 256, 4096, 32), 64, 50, 816,
                              "random", (3, 10), bf16=True),
    # 24 layers, width 1536, 12 q heads / 2 kv heads of 128, GeGLU 6144, prefix 1024,
    # H=128, batch 16, budgets rising linearly 3 -> 12 across the chunk.
    "large_b16": Workload("large_b16", ModelShape(24, 1536, 12, 2, 128, 6144, 32), 16, 128, 1024,
                          "linear", (3, 12), bf16=True),
}

# Adaptive-norm time conditioning (the pi0.5-style expert of App. C.1): the
# tiny and pi0-scale models with modulated norms instead of input conditioning.
WORKLOADS["tiny_adarms"] = Workload("tiny_adarms", ModelShape(2, 256, 4, 4, 64, 1024, 7, conditioning="adarms"),
                                    1, 16, 64, "uniform", (10,), bf16=False)
WORKLOADS["pi05_b1_adarms"] = Workload("pi05_b1_adarms",
                                       ModelShape(18, 1024, 8, 1, 256, 4096, 32, conditioning="adarms"),
                                       1, 50, 816, "uniform", (10,), bf16=True)

WORKLOAD_ORDER = ["tiny", "pi0_b1", "pi0_b1_uad", "pi0_fleet_b64", "large_b16"]
ADARMS_WORKLOADS = ["tiny_adarms", "pi05_b1_adarms"]


def get_workload(name: str, **overrides) -> Workload:
    """Return a named workload, optionally with fields replaced (e.g. batch)."""
    w = WORKLOADS[name]
    return dataclasses.replace(w, **overrides) if overrides else w


# ----------------------------------------------------------------------------
# Tensor naming (PyTorch Linear layout: weight [out, in], row-major)
# ----------------------------------------------------------------------------
def weight_specs(s: ModelShape) -> List[Tuple[str, Tuple[int, ...], str]]:
    """(name, shape, init) for every named weight; init in {"w", "gain", "bias"}."""
    d, hq, hkv, hd, f, da = s.d_model, s.n_heads, s.n_kv_heads, s.head_dim, s.d_ff, s.action_dim
    ada = s.conditioning == "adarms"
    out = [
        ("action_in.w", (d, da), "w"), ("action_in.b", (d,), "bias"),
        ("time_mlp_in.w", (d, d if ada else 2 * d), "w"), ("time_mlp_in.b", (d,), "bias"),
        ("time_mlp_out.w", (d, d), "w"), ("time_mlp_out.b", (d,), "bias"),
    ]
    for l in range(s.n_layers):
        p = f"layers.{l}."
        out += [(p + "attn_mod.w", (3 * d, d), "w"), (p + "attn_mod.b", (3 * d,), "bias")] if ada else \
               [(p + "attn_norm", (d,), "gain")]
        out += [
            (p + "wq", (hq * hd, d), "w"), (p + "wk", (hkv * hd, d), "w"),
            (p + "wv", (hkv * hd, d), "w"), (p + "wo", (d, hq * hd), "w"),
        ]
        out += [(p + "mlp_mod.w", (3 * d, d), "w"), (p + "mlp_mod.b", (3 * d,), "bias")] if ada else \
               [(p + "mlp_norm", (d,), "gain")]
        out += [
            (p + "w_gate", (f, d), "w"), (p + "w_up", (f, d), "w"),
            (p + "w_down", (d, f), "w"),
        ]
    out += [("final_mod.w", (2 * d, d), "w"), ("final_mod.b", (2 * d,), "bias")] if ada else \
           [("final_norm", (d,), "gain")]
    out += [("action_out.w", (da, d), "w"), ("action_out.b", (da,), "bias")]
    return out


def weight_param_count(s: ModelShape) -> int:
    return int(sum(int(np.prod(shp)) for _, shp, _ in weight_specs(s)))


# ----------------------------------------------------------------------------
# Seeded draws
# ----------------------------------------------------------------------------
def _rng(seed: int, name: str) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, zlib.crc32(name.encode())])))


def draw(seed: int, name: str, shape, scale: float = 1.0, offset: float = 0.0) -> np.ndarray:
    """fp32 standard-normal draw from the named stream, times scale, plus offset."""
    z = _rng(seed, name).standard_normal(size=shape, dtype=np.float32)
    if scale != 1.0:
        z *= np.float32(scale)
    if offset != 0.0:
        z += np.float32(offset)
    return z


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); returned as fp32.

    The canonical inputs of the bf16 workloads are these values: the oracle
    holds them as fp32 and the device receives the identical bf16 bits.
    """
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = (u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Upper 16 bits of fp32 values that are already bf16-representable."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    if np.any(u & np.uint32(0xFFFF)):
        raise ValueError("bf16_bits: values are not bf16-representable; round first")
    return (u >> np.uint32(16)).astype(np.uint16)


def make_weights(w: Workload) -> Dict[str, np.ndarray]:
    """Random-init weights: N(0, 0.02) matrices and biases, norm gains 1 + 0.02 z."""
    out = {}
    for name, shp, kind in weight_specs(w.shape):
        if kind == "gain":
            a = draw(w.seed, name, shp, 0.02, 1.0)
        else:
            a = draw(w.seed, name, shp, 0.02)
        out[name] = round_to_bf16(a) if w.bf16 else a
    return out


def make_prefix(w: Workload, b: int) -> Tuple[np.ndarray, np.ndarray]:
    """Cached prefix K and V of environment b: each fp32 [L][P][Hkv][hd], N(0,1)."""
    s = w.shape
    ks, vs = [], []
    for l in range(s.n_layers):
        k = draw(w.seed, f"prefix.{b}.{l}.k", (w.prefix, s.n_kv_heads, s.head_dim))
        v = draw(w.seed, f"prefix.{b}.{l}.v", (w.prefix, s.n_kv_heads, s.head_dim))
        ks.append(round_to_bf16(k) if w.bf16 else k)
        vs.append(round_to_bf16(v) if w.bf16 else v)
    return np.stack(ks), np.stack(vs)


def make_noise(w: Workload, b: int) -> np.ndarray:
    """Initial noise x_0 of environment b: fp32 [H][Da], N(0,1) (Sec. 3)."""
    return draw(w.seed, f"noise.{b}", (w.chunk, w.shape.action_dim))


def _budgets_env(w: Workload, b: int) -> np.ndarray:
    H = w.chunk
    if w.budget_kind == "uniform":
        return np.full(H, w.budget_arg[0], np.int32)
    if w.budget_kind == "groups":
        parts = [np.full(n, nb, np.int32) for n, nb in w.budget_arg]
        out = np.concatenate(parts)
        assert out.shape[0] == H
        return out
    if w.budget_kind == "random":
        # urgent prefix length U ~ U{3..10}; tail budget N* ~ U{4..10};
        # urgent budget K ~ U{3..N*-1}; budgets stay within 3..10.
        lo, hi = w.budget_arg
        g = _rng(w.seed, f"sched.{b}")
        U = int(g.integers(lo, hi + 1))
        nstar = int(g.integers(lo + 1, hi + 1))
        K = int(g.integers(lo, nstar))
        out = np.full(H, nstar, np.int32)
        out[:U] = K
        return out
    if w.budget_kind == "linear":
        lo, hi = w.budget_arg
        i = np.arange(H, dtype=np.int64)
        # integer round-half-up of lo + (hi-lo) * i / (H-1)
        num = (hi - lo) * i * 2 + (H - 1)
        return (lo + num // (2 * (H - 1))).astype(np.int32)
    raise ValueError(w.budget_kind)


def make_budgets(w: Workload) -> np.ndarray:
    """Per-token integer step budgets N_i, int32 [B][H]."""
    return np.stack([_budgets_env(w, b) for b in range(w.batch)])


def iter_envs(w: Workload) -> Iterator[int]:
    return iter(range(w.batch))
