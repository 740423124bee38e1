"""GPU parity of the adaptive-norm-conditioned expert (App. C.1, the
pi0.5-style variant: the per-token time modulates every RMSNorm and gates
every residual branch) against the oracle, through the C ABI.

Bars as for the input-conditioned expert: per-step velocities within a
normwise max relative error of 2e-2 (teacher-forced), final and released
actions within 1e-2 absolute (free-running schedule), release steps
bit-exact; the release path (TR, K = 1) reproduces the uniform schedule bit
for bit on this model too.
"""
import numpy as np
import pytest
import torch

import oracle as O
from tests.harness import log, make_case, rel_err

pytestmark = pytest.mark.gpu

VEL_RTOL = 2e-2
ACT_ATOL = 1e-2
_cases = {}


def case(name, **kw):
    key = (name, tuple(sorted(kw.items())))
    if key not in _cases:
        _cases[key] = make_case(name, **kw)
    return _cases[key]


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("name,steps", [("tiny_adarms", None), ("pi05_b1_adarms", [0, 4, 9])])
def test_adarms_teacher_forced_velocity(gpu, name, steps):
    c = case(name)
    r = O.denoise_schedule(c.oracle_model(), c.noise, c.budgets, keep_history=True)
    for k in (range(r["n_steps"]) if steps is None else steps):
        x_in, v_ref = r["history"][k]
        xg = dev(x_in.astype(np.float32))
        vg = torch.empty_like(xg)
        c.expert.step(xg, dev(r["t"][k].astype(np.float32)), dev(r["dt"][k].astype(np.float32)),
                      dev(r["mask"][k].astype(np.uint8)), vg)
        torch.cuda.synchronize()
        e = rel_err(vg.cpu().numpy()[0], v_ref[0])
        log(f"[{name}] step {k}: velocity rel err {e:.2e}")
        assert e <= VEL_RTOL


@pytest.mark.parametrize("name", ["tiny_adarms", "pi05_b1_adarms"])
def test_adarms_free_running_uad_schedule(gpu, name):
    """Budgets 4 / 7 / 10 over the chunk: per-token flow times reach the norms."""
    c = case(name)
    H = c.wl.chunk
    bud = np.full((1, H), 10, np.int32)
    bud[0, : H // 10] = 4
    bud[0, H // 10: H // 2] = 7
    r = O.denoise_schedule(c.oracle_model(), c.noise, bud)
    n, tg, dtg, mg = c.expert.schedule_tables(bud)
    x = dev(c.noise.astype(np.float32))
    rel = torch.zeros_like(x)
    rst = torch.full(bud.shape, -1, dtype=torch.int32, device="cuda")
    c.expert.schedule(x, tg, dtg, mg, rel, rst)
    torch.cuda.synchronize()
    ex, er = np.abs(x.cpu().numpy() - r["x"]).max(), np.abs(rel.cpu().numpy() - r["released"]).max()
    log(f"[{name}] final max abs err {ex:.2e}, released {er:.2e}")
    assert ex <= ACT_ATOL and er <= ACT_ATOL
    np.testing.assert_array_equal(rst.cpu().numpy(), r["release_step"])


def test_adarms_tr_k1_bit_exact(gpu):
    c = case("tiny_adarms")
    x = dev(c.noise.astype(np.float32))
    c.expert.release(x, 5, 1, 7, 10)
    n, tg, dtg, mg = c.expert.schedule_tables(np.full((1, c.wl.chunk), 7, np.int32))
    xv = dev(c.noise.astype(np.float32))
    c.expert.schedule(xv, tg, dtg, mg)
    torch.cuda.synchronize()
    assert torch.equal(x, xv)


def test_adarms_time_changes_velocity(gpu):
    """Time must reach the output through the modulations: same x, different t."""
    c = case("tiny_adarms")
    H, Da = c.wl.chunk, c.wl.shape.action_dim
    vs = []
    for tv in (1.0, 0.3):
        xg = dev(c.noise.astype(np.float32))
        vg = torch.empty_like(xg)
        c.expert.step(xg, torch.full((1, H), tv, device="cuda"), torch.zeros((1, H), device="cuda"),
                      torch.zeros((1, H), dtype=torch.uint8, device="cuda"), vg)
        vs.append(vg.cpu().numpy())
    assert np.abs(vs[0] - vs[1]).max() > 1e-3


@pytest.mark.parametrize("batch", [8, 24])
def test_adarms_batched_sampled_envs(gpu, batch):
    """8 / 24 environments, M = 400 / 1200 rows: the batched projection kernel
    serves the time MLP, the modulation GEMM and the gated residual epilogues
    (at 1200 rows the embedding kernel also takes 16 tokens per workgroup).
    Sampled environments against the oracle run alone: one teacher-forced
    step, then the free-running UAD schedule."""
    c = case("pi05_b1_adarms", batch=batch)
    B, H = c.budgets.shape
    bud = np.full((B, H), 10, np.int32)
    bud[:, : H // 10] = 4
    bud[:, H // 10: H // 2] = 7
    n, t, dt, mask = O.build_schedule(bud)
    xg = dev(c.noise.astype(np.float32))
    vg = torch.empty_like(xg)
    c.expert.step(xg, dev(t[0].astype(np.float32)), dev(dt[0].astype(np.float32)), dev(mask[0].astype(np.uint8)), vg)
    torch.cuda.synchronize()
    v = vg.cpu().numpy()
    nt, tg, dtg, mg = c.expert.schedule_tables(bud)
    x = dev(c.noise.astype(np.float32))
    rel = torch.zeros_like(x)
    rst = torch.full(bud.shape, -1, dtype=torch.int32, device="cuda")
    c.expert.schedule(x, tg, dtg, mg, rel, rst)
    torch.cuda.synchronize()
    rel = rel.cpu().numpy()
    for b in (0, B - 1):
        mb = c.oracle_model([b])
        e = rel_err(v[b], O.velocity(mb, c.noise[b:b + 1], t[0][b:b + 1])[0])
        r = O.denoise_schedule(mb, c.noise[b:b + 1], bud[b:b + 1])
        ea = float(np.abs(rel[b] - r["released"][0]).max())
        log(f"[pi05 B={batch}] env {b}: step-0 velocity rel err {e:.2e}, released abs err {ea:.2e}")
        assert e <= VEL_RTOL and ea <= ACT_ATOL
    np.testing.assert_array_equal(rst.cpu().numpy(), O.release_steps(bud))


@pytest.mark.parametrize("top", [64, 2])
def test_adarms_schedule_level_conditioning_step_counts(gpu, top):
    """The schedule computes the conditioning of all its steps at once: a
    64-step schedule (a budget of 64, the largest the builder takes, on every
    third token) and a 2-step one on the same context, which grow and reuse the
    schedule-level buffers; both against the oracle, and a single joint step
    afterwards still matches it."""
    c = case("tiny_adarms")
    H = c.wl.chunk
    bud = np.full((1, H), top, np.int32)
    bud[0, 1::3] = 1
    r = O.denoise_schedule(c.oracle_model(), c.noise, bud)
    n, tg, dtg, mg = c.expert.schedule_tables(bud)
    assert n == top
    x = dev(c.noise.astype(np.float32))
    rel = torch.zeros_like(x)
    rst = torch.full(bud.shape, -1, dtype=torch.int32, device="cuda")
    c.expert.schedule(x, tg, dtg, mg, rel, rst)
    torch.cuda.synchronize()
    ex, er = np.abs(x.cpu().numpy() - r["x"]).max(), np.abs(rel.cpu().numpy() - r["released"]).max()
    log(f"[tiny_adarms {top} steps] final max abs err {ex:.2e}, released {er:.2e}")
    assert ex <= ACT_ATOL and er <= ACT_ATOL
    np.testing.assert_array_equal(rst.cpu().numpy(), r["release_step"])
    # one teacher-forced joint step at mid-schedule flow times
    t = np.linspace(0.9, 0.1, H, dtype=np.float32)[None]
    xg = dev(c.noise.astype(np.float32))
    vg = torch.empty_like(xg)
    c.expert.step(xg, dev(t), dev(np.zeros_like(t)), dev(np.zeros(t.shape, np.uint8)), vg)
    torch.cuda.synchronize()
    e = rel_err(vg.cpu().numpy(), O.velocity(c.oracle_model(), c.noise, t))
    log(f"[tiny_adarms] single step after the schedule: velocity rel err {e:.2e}")
    assert e <= VEL_RTOL


@pytest.mark.parametrize("pattern", ["16_times", "50_times"])
def test_adarms_many_flow_times_one_step(gpu, pattern):
    """A joint step of the pi0.5-scale adaptive-norm expert after a schedule
    (schedule-level conditioning in place) whose 50 tokens take 16 flow times
    in an irregular order, or 50 distinct ones: every token's norms get their
    own modulations; against the oracle."""
    c = case("pi05_b1_adarms")
    H = c.wl.chunk
    n, tg, dtg, mg = c.expert.schedule_tables(np.full((1, H), 10, np.int32))
    xs = dev(c.noise.astype(np.float32))
    c.expert.schedule(xs, tg, dtg, mg)
    if pattern == "16_times":
        t = (((np.arange(H) * 7) % 16 + 1) / np.float32(17)).astype(np.float32)[None]
        assert len(np.unique(t)) == 16
    else:
        t = np.linspace(0.95, 0.05, H, dtype=np.float32)[None]
        assert len(np.unique(t)) == H
    xg = dev(c.noise.astype(np.float32))
    vg = torch.empty_like(xg)
    c.expert.step(xg, dev(t), dev(np.zeros_like(t)), dev(np.zeros(t.shape, np.uint8)), vg)
    torch.cuda.synchronize()
    e = rel_err(vg.cpu().numpy(), O.velocity(c.oracle_model(), c.noise, t))
    log(f"[pi05_b1_adarms {pattern}] velocity rel err {e:.2e}")
    assert e <= VEL_RTOL
