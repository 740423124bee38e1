"""The step entry point that allocates nothing (uad_denoise_step_static), called
through the C ABI, against uad_denoise_step on the same inputs: two calls in a
row, the second with a smaller batch and chunk, both with split-KV partials in
the static scratch array (a 1722-key prefix splits the keys 15 ways)."""
import ctypes

import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_37772_amd as U
from tests.harness import log, make_case, prefix_stack_bf16, rel_err

pytestmark = pytest.mark.gpu


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def test_static_step_matches_step(gpu):
    c = make_case("tiny", with_expert=False, batch=2, chunk=71, prefix=1722)
    ex = U.ActionExpert(c.wl.shape, 2, 71, 1722)
    lib = U.load_library()
    try:
        ex.load_weights(c.weights)
        K, V = prefix_stack_bf16(c)
        ex.set_prefix_kv(K, V, 2, 1722)
        n, t, dt, mask = O.build_schedule(c.budgets)
        v_ref = O.velocity(c.oracle_model(), c.noise, t[1])
        for B, H in ((2, 71), (1, 40)):  # the second call is smaller
            x0 = np.ascontiguousarray(c.noise[:B, :H])
            ins = [dev(t[1][:B, :H]), dev(dt[1][:B, :H]), dev(mask[1][:B, :H])]
            outs = {}
            for fn in ("uad_denoise_step", "uad_denoise_step_static"):
                x = dev(x0)
                v = torch.empty_like(x)
                ptrs = [ctypes.c_void_p(a.data_ptr()) for a in (x, *ins, v)]
                st = getattr(lib, fn)(ex.ctx, *ptrs, B, H)
                assert st == 0, U.uad_last_error(ex.ctx)
                ex.synchronize()
                outs[fn] = (x.cpu().numpy(), v.cpu().numpy())
            xa, va = outs["uad_denoise_step"]
            xb, vb = outs["uad_denoise_step_static"]
            assert xa.tobytes() == xb.tobytes() and va.tobytes() == vb.tobytes()
            if H == 71:  # the full chunk also against the oracle
                for b in range(B):
                    e = rel_err(vb[b], v_ref[b])
                    log(f"[static step B={B} H={H}] env {b}: velocity rel err {e:.2e}")
                    assert e <= 2e-2
            log(f"[static step B={B} H={H}] bit-identical to uad_denoise_step")
    finally:
        ex.close()
