"""Convenience wrapper owning one libuad context (marshalling only)."""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np
import torch

from . import _binding as B


class ActionExpert:
    """One UAD action expert on one GPU: weights, prefix K/V and workspace live in libuad."""

    def __init__(self, shape, max_batch: int, max_chunk: int, max_prefix: int, device: int = 0,
                 stream: Optional[torch.cuda.Stream] = None):
        self.shape = shape
        self.device = device
        self.max_batch, self.max_chunk, self.max_prefix = max_batch, max_chunk, max_prefix
        self.ctx = B.uad_create(shape, max_batch, max_chunk, max_prefix, device, stream)

    def close(self):
        if getattr(self, "ctx", None):
            B.uad_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def load_weights(self, weights: Dict[str, object]) -> None:
        B.uad_load_weights(self.ctx, weights)

    def set_prefix_kv(self, k, v, batch: int, prefix_len: int) -> None:
        B.uad_set_prefix_kv(self.ctx, k, v, batch, prefix_len)

    def step(self, x, t, dt, mask, v_out=None) -> None:
        B.uad_denoise_step(self.ctx, x, t, dt, mask, v_out)

    def schedule(self, x, t_sched, dt_sched, mask_sched, released=None, release_step=None, step_ticks=None):
        B.uad_denoise_schedule(self.ctx, x, t_sched, dt_sched, mask_sched, released, release_step, step_ticks)

    def schedule_budgets(self, x, budgets, released=None, release_step=None, step_ticks=None):
        """A schedule from host budgets, finished environments skipped (uad_denoise_budgets)."""
        B.uad_denoise_budgets(self.ctx, x, budgets, released, release_step, step_ticks)

    def release(self, x, U: int, K: int, Nstar: int, S: int, reconcile: bool = True, urgent=None,
                executed=None, gac_mask=None, urgent_host=None, release_event=None, step_ticks=None):
        """Urgency-aware release (UAER, or TR + ghosts, GAC when ``executed`` is given).

        Allocates ``urgent`` [B][U][Da] on the device when not given and returns it.
        """
        B_, H_, Da = x.shape
        if urgent is None:
            urgent = torch.empty((B_, U, Da), dtype=torch.float32, device=x.device)
        mode = B.UAD_RELEASE_TR if reconcile else B.UAD_RELEASE_UAER
        B.uad_denoise_release(self.ctx, x, U, K, Nstar, S, mode, urgent, executed, gac_mask, urgent_host,
                              release_event, step_ticks)
        return urgent

    def debug_velocity_field(self, enable: bool, alpha: float = 0.0, beta: float = 0.0) -> None:
        B.uad_debug_velocity_field(self.ctx, enable, alpha, beta)

    def synchronize(self) -> None:
        B.uad_synchronize(self.ctx)

    def tick_rate_hz(self) -> float:
        return B.uad_tick_rate_hz(self.ctx)

    def schedule_tables(self, budgets: np.ndarray, device=None):
        """Build the per-step tables with the library's host builder and copy them to the device."""
        n, t, dt, mask = B.uad_build_schedule(budgets)
        dev = device if device is not None else torch.device("cuda", self.device)
        return (n, torch.from_numpy(t).to(dev), torch.from_numpy(dt).to(dev), torch.from_numpy(mask).to(dev))
