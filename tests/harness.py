"""Shared set-up for GPU tests: seeded inputs -> oracle model + libuad expert."""
from __future__ import annotations

import dataclasses
import sys
from typing import Dict, List, Optional

import numpy as np

import oracle as O
import uad_workloads as W


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


@dataclasses.dataclass
class Case:
    wl: W.Workload
    weights: Dict[str, np.ndarray]
    noise: np.ndarray           # [B][H][Da]
    budgets: np.ndarray         # [B][H]
    prefix: List[tuple]         # per env (k, v) [L][P][Hkv][hd] fp32
    expert: object = None

    def oracle_model(self, envs: Optional[List[int]] = None, dtype=np.float32) -> O.Model:
        envs = list(range(self.wl.batch)) if envs is None else envs
        return O.build_model(self.wl.shape, self.weights, [self.prefix[b][0] for b in envs],
                             [self.prefix[b][1] for b in envs], dtype=dtype)


def prefix_stack_bf16(case: Case) -> tuple:
    """[L][B][P][Hkv][hd] arrays for uad_set_prefix_kv (bf16 bits when the workload is bf16)."""
    s, B, P = case.wl.shape, case.wl.batch, case.wl.prefix
    dt = np.uint16 if case.wl.bf16 else np.float32
    K = np.empty((s.n_layers, B, P, s.n_kv_heads, s.head_dim), dt)
    V = np.empty_like(K)
    for b in range(B):
        k, v = case.prefix[b]
        K[:, b] = W.bf16_bits(k) if case.wl.bf16 else k
        V[:, b] = W.bf16_bits(v) if case.wl.bf16 else v
    return K, V


def make_case(name: str, with_expert: bool = True, **overrides) -> Case:
    wl = W.get_workload(name, **overrides)
    log(f"[setup] {name} B={wl.batch} H={wl.chunk} P={wl.prefix} L={wl.shape.n_layers} d={wl.shape.d_model}")
    weights = W.make_weights(wl)
    noise = np.stack([W.make_noise(wl, b) for b in range(wl.batch)])
    budgets = W.make_budgets(wl)
    prefix = [W.make_prefix(wl, b) for b in range(wl.batch)]
    case = Case(wl, weights, noise, budgets, prefix)
    if with_expert:
        import paper_2609_37772_amd as U
        ex = U.ActionExpert(wl.shape, wl.batch, wl.chunk, wl.prefix)
        ex.load_weights(weights)
        K, V = prefix_stack_bf16(case)
        ex.set_prefix_kv(K, V, wl.batch, wl.prefix)
        case.expert = ex
    return case


def rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    """Normwise max relative error: max|got - ref| / max|ref|."""
    return float(np.max(np.abs(got - ref)) / max(np.max(np.abs(ref)), 1e-30))
