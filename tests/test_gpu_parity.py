"""GPU parity of the libuad hot path against the CPU oracle, through the C ABI.

Bars: per-step velocities within a normwise max relative error of 2e-2
(teacher-forced: the GPU step gets the oracle's state, times and mask), final
and released actions within 1e-2 absolute (free-running schedule), schedule
tables, masks and release steps bit-exact, frozen tokens bit-identical.
"""
import numpy as np
import pytest
import torch

import oracle as O
import uad_workloads as W
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


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t if dtype is None else t.to(dtype)


def gpu_velocity(c, x, t, dt, mask):
    """One GPU step on given inputs; returns (x_after, v)."""
    xg = dev(x.astype(np.float32))
    vg = torch.empty_like(xg)
    c.expert.step(xg, dev(t.astype(np.float32)), dev(dt.astype(np.float32)), dev(mask.astype(np.uint8)), vg)
    torch.cuda.synchronize()
    return xg.cpu().numpy(), vg.cpu().numpy()


def run_schedule_gpu(c, x0, budgets):
    n, tg, dtg, mg = c.expert.schedule_tables(budgets)
    xg = dev(x0.astype(np.float32))
    rel = torch.zeros_like(xg)
    rst = torch.full(budgets.shape, -1, dtype=torch.int32, device="cuda")
    c.expert.schedule(xg, tg, dtg, mg, rel, rst)
    torch.cuda.synchronize()
    return xg.cpu().numpy(), rel.cpu().numpy(), rst.cpu().numpy()


# ----------------------------------------------------------------------------
# Teacher-forced velocities + free-running schedules, per workload
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("name,steps", [("tiny", None), ("pi0_b1", [0, 5, 9]), ("pi0_b1_uad", [0, 4, 8])])
def test_teacher_forced_velocity(gpu, name, steps):
    c = case(name)
    m = c.oracle_model()
    r = O.denoise_schedule(m, c.noise, c.budgets, keep_history=True)
    ks = range(r["n_steps"]) if steps is None else steps
    for k in ks:
        x_in, v_ref = r["history"][k]
        _, v = gpu_velocity(c, x_in, r["t"][k], r["dt"][k], r["mask"][k])
        for b in range(c.wl.batch):
            e = rel_err(v[b], v_ref[b])
            log(f"[{name}] step {k} env {b}: velocity rel err {e:.2e}")
            assert e <= VEL_RTOL


@pytest.mark.parametrize("name", ["tiny", "pi0_b1", "pi0_b1_uad"])
def test_free_running_schedule(gpu, name):
    c = case(name)
    r = O.denoise_schedule(c.oracle_model(), c.noise, c.budgets)
    x, rel, rst = run_schedule_gpu(c, c.noise, c.budgets)
    err_x = float(np.max(np.abs(x - r["x"])))
    err_rel = float(np.max(np.abs(rel - r["released"])))
    log(f"[{name}] final max abs err {err_x:.2e}, released {err_rel:.2e}")
    assert err_x <= ACT_ATOL and err_rel <= ACT_ATOL
    np.testing.assert_array_equal(rst, r["release_step"])
    # released actions of a token equal its final state (frozen afterwards)
    assert rel.tobytes() == x.tobytes()


def _steps_to_force(n):
    """First, middle and last step of an n-step schedule."""
    return sorted({0, n // 2, n - 1})


_oracle_runs = {}


def oracle_schedule(c, tag):
    """The oracle's schedule of every environment of case c (with history), computed once per case."""
    if tag not in _oracle_runs:
        log(f"[{tag}] oracle schedule of {c.wl.batch} environments")
        _oracle_runs[tag] = O.denoise_schedule(c.oracle_model(), c.noise, c.budgets, keep_history=True)
    return _oracle_runs[tag]


def run_budgets_gpu(c, x0, budgets):
    xg = dev(x0.astype(np.float32))
    rel = torch.zeros_like(xg)
    rst = torch.full(budgets.shape, -1, dtype=torch.int32, device="cuda")
    c.expert.schedule_budgets(xg, budgets, rel, rst)
    c.expert.synchronize()
    return xg.cpu().numpy(), rel.cpu().numpy(), rst.cpu().numpy()


def _every_env_against_oracle(c, tag):
    """Every environment of a batched workload against the oracle: per-step
    velocities teacher-forced at the first, a middle and the last step (the
    GPU step gets the oracle's states of ALL environments), then the
    free-running schedule's released actions, final states and release steps."""
    B = c.wl.batch
    r = oracle_schedule(c, tag)
    worst_v = 0.0
    for k in _steps_to_force(r["n_steps"]):
        x_in, v_ref = r["history"][k]
        _, v = gpu_velocity(c, x_in, r["t"][k], r["dt"][k], r["mask"][k])
        errs = [rel_err(v[b], v_ref[b]) for b in range(B)]
        worst_v = max(worst_v, max(errs))
        log(f"[{tag}] step {k}: velocity rel err max {max(errs):.2e} (env {int(np.argmax(errs))}) over {B} envs")
        assert max(errs) <= VEL_RTOL
    x, rel, rst = run_schedule_gpu(c, c.noise, c.budgets)
    err_rel = np.max(np.abs(rel - r["released"]), axis=(1, 2))
    err_x = np.max(np.abs(x - r["x"]), axis=(1, 2))
    log(f"[{tag}] free-running: released max abs err {err_rel.max():.2e} (env {int(np.argmax(err_rel))}), "
        f"final {err_x.max():.2e} over {B} envs")
    assert err_rel.max() <= ACT_ATOL and err_x.max() <= ACT_ATOL
    np.testing.assert_array_equal(rst, r["release_step"])
    np.testing.assert_array_equal(rst, O.release_steps(c.budgets))
    assert rel.tobytes() == x.tobytes()  # a token's released action is its final, frozen state


@pytest.mark.timeout(900)
def test_fleet_every_env(gpu):
    """64 environments (3,200 token rows), per-environment random budgets."""
    _every_env_against_oracle(case("pi0_fleet_b64"), "fleet")


@pytest.mark.timeout(900)
def test_large_every_env(gpu):
    """24 layers, width 1536, GQA 12/2, H=128, 16 environments, linear budgets 3..12."""
    _every_env_against_oracle(case("large_b16"), "large")


@pytest.mark.timeout(900)
def test_fleet_budgets_finished_environments_skipped(gpu):
    """uad_denoise_budgets on the fleet (per-environment budgets 3..10): steps
    after an environment's last release skip it; every environment's released
    actions, final states and release steps against the oracle, and against
    the uncompacted schedule on the same tables."""
    c = case("pi0_fleet_b64")
    r = oracle_schedule(c, "fleet")
    x, rel, rst = run_budgets_gpu(c, c.noise, c.budgets)
    xs, rels, rsts = run_schedule_gpu(c, c.noise, c.budgets)
    err_rel = float(np.max(np.abs(rel - r["released"])))
    err_x = float(np.max(np.abs(x - r["x"])))
    err_vs = float(np.max(np.abs(rel - rels)))
    active = [int(np.sum(c.budgets.max(axis=1) > k)) for k in range(r["n_steps"])]
    log(f"[fleet budgets] environments per step {active}; released max abs err {err_rel:.2e}, "
        f"final {err_x:.2e}; vs uncompacted schedule {err_vs:.2e}")
    assert err_rel <= ACT_ATOL and err_x <= ACT_ATOL and err_vs <= ACT_ATOL
    np.testing.assert_array_equal(rst, r["release_step"])
    np.testing.assert_array_equal(rst, rsts)
    assert rel.tobytes() == x.tobytes()


def test_budgets_non_contiguous_finished_environments(gpu):
    """Four environments finishing at steps 3, 1, 5 and 2 (largest budgets), so
    the environments still running are not a prefix of the batch: against the
    oracle, and under the linear field v = alpha x + beta bit for bit against
    the uncompacted schedule and within 2e-6 of the closed form."""
    c = case("tiny", batch=4)
    H = c.wl.chunk
    bud = np.stack([np.full(H, 3), np.full(H, 1), np.array([1 + (i % 5) for i in range(H)]),
                    np.array([1 + (i % 2) for i in range(H)])]).astype(np.int32)
    r = O.denoise_schedule(c.oracle_model(), c.noise, bud)
    x, rel, rst = run_budgets_gpu(c, c.noise, bud)
    e = float(np.max(np.abs(rel - r["released"])))
    log(f"[budgets, 4 environments] released max abs err {e:.2e}")
    assert e <= ACT_ATOL and float(np.max(np.abs(x - r["x"]))) <= ACT_ATOL
    np.testing.assert_array_equal(rst, r["release_step"])
    alpha, beta = 0.35, -0.2
    c.expert.debug_velocity_field(True, alpha, beta)
    try:
        xb, relb, rstb = run_budgets_gpu(c, c.noise, bud)
        xs, rels, rsts = run_schedule_gpu(c, c.noise, bud)
    finally:
        c.expert.debug_velocity_field(False)
    assert relb.tobytes() == rels.tobytes() and xb.tobytes() == xs.tobytes()
    np.testing.assert_array_equal(rstb, rsts)
    N = bud.astype(np.float64)[..., None]
    g = (1.0 + alpha * (-1.0 / N)) ** N
    ref = g * c.noise + beta * (g - 1.0) / alpha
    np.testing.assert_allclose(relb, ref, rtol=2e-6, atol=2e-6)


def test_frozen_tokens_bit_identical_batched(gpu):
    """Frozen tokens stay bit-identical through the batched final projection
    (16 tokens per workgroup on MFMA, used from 1,024 token rows on when the
    width is a multiple of 512: here 64 environments x 50 tokens, width 1024),
    a -0.0 among them."""
    c = case("pi0_fleet_b64")
    n, tg, dtg, mg = c.expert.schedule_tables(c.budgets)
    x0 = c.noise.astype(np.float32).copy()
    x0[:, 0, 0] = -0.0
    xg = dev(x0)
    snaps = []
    for k in range(n):
        c.expert.step(xg, tg[k], dtg[k], mg[k])
        torch.cuda.synchronize()
        snaps.append(xg.cpu().numpy().copy())
    B, H = c.budgets.shape
    checked = 0
    for b in range(B):
        for i in range(H):
            N = int(c.budgets[b, i])
            for k in range(N, n):
                assert snaps[k][b, i].tobytes() == snaps[N - 1][b, i].tobytes(), (b, i, k)
                checked += 1
    log(f"[fleet] {checked} frozen (token, step) pairs bit-identical")
    assert checked > 0


@pytest.mark.parametrize("batch", [41, 48, 49, 60])
def test_fleet_ragged_row_panels(gpu, batch):
    """Fleet model at 2050 / 2400 / 2450 / 3000 token rows, not a multiple of
    the batched kernels' 128-row panels: the k-halves projections (2400 rows),
    the residual LDS ring (3000 rows) and the 128 x 256 gate/up ring end on a
    partial panel; gate/up runs on 144-row tiles at 2050 rows (15 panels, the
    last 34 rows) and on 160-row tiles at 2400 and 2450 rows (the last panel
    of 2450 holds 50 rows); the last environment's rows lie in the partial
    panel."""
    c = make_case("pi0_fleet_b64", batch=batch)
    n, t, dt, mask = O.build_schedule(c.budgets)
    _, v = gpu_velocity(c, c.noise, t[0], dt[0], mask[0])
    for b in (0, batch - 1):
        mb = c.oracle_model([b])
        v_ref = O.velocity(mb, c.noise[b:b + 1], t[0][b:b + 1])[0]
        e = rel_err(v[b], v_ref)
        log(f"[fleet B={batch}] env {b}: step-0 velocity rel err {e:.2e}")
        assert e <= VEL_RTOL
    c.expert.close()


@pytest.mark.parametrize("batch", [6, 12, 17])
def test_fleet_small_batches_with_weight_read_ahead(gpu, batch):
    """A few environments of the fleet model, where the attention's key splits
    are chosen to leave CUs to the weight read-ahead (6, 12 and 17
    environments: 5, 2 and 1 splits of the 28 key blocks) and the read-ahead
    workgroups run in the attention and merge launches: the first and last
    environment's step-0 velocities against the oracle run alone."""
    c = make_case("pi0_fleet_b64", batch=batch)
    n, t, dt, mask = O.build_schedule(c.budgets)
    _, v = gpu_velocity(c, c.noise, t[0], dt[0], mask[0])
    for b in (0, batch - 1):
        mb = c.oracle_model([b])
        v_ref = O.velocity(mb, c.noise[b:b + 1], t[0][b:b + 1])[0]
        e = rel_err(v[b], v_ref)
        log(f"[fleet B={batch}] env {b}: step-0 velocity rel err {e:.2e}")
        assert e <= VEL_RTOL
    c.expert.close()


# ----------------------------------------------------------------------------
# Invariants of the method on the GPU path
# ----------------------------------------------------------------------------
def test_uniform_schedule_equals_repeated_vanilla_steps_bit_exact(gpu):
    c = case("tiny")
    N = 10
    x, _, _ = run_schedule_gpu(c, c.noise, np.full_like(c.budgets, N))
    xg = dev(c.noise.astype(np.float32))
    B, H = c.budgets.shape
    for k in range(N):
        tk = np.full((B, H), np.float32(N - k) / np.float32(N), np.float32)
        dtk = np.full((B, H), -(np.float32(1) / np.float32(N)), np.float32)
        c.expert.step(xg, dev(tk), dev(dtk), dev(np.zeros((B, H), np.uint8)))
    torch.cuda.synchronize()
    assert xg.cpu().numpy().tobytes() == x.tobytes()


def test_frozen_tokens_bit_identical_on_gpu(gpu):
    c = case("pi0_b1_uad")
    n, tg, dtg, mg = c.expert.schedule_tables(c.budgets)
    x0 = c.noise.astype(np.float32).copy()
    x0[0, 0, 0] = -0.0
    xg = dev(x0)
    snaps = []
    for k in range(n):
        c.expert.step(xg, tg[k], dtg[k], mg[k])
        torch.cuda.synchronize()
        snaps.append(xg.cpu().numpy().copy())
    for i, N in enumerate(c.budgets[0]):
        for k in range(N, n):
            assert snaps[k][0, i].tobytes() == snaps[N - 1][0, i].tobytes()


def test_nan_velocity_never_reaches_frozen_tokens(gpu):
    c = case("tiny")
    B, H, Da = c.noise.shape
    x0 = c.noise.astype(np.float32).copy()
    x0[0, 1, :] = -0.0
    mask = np.zeros((B, H), np.uint8)
    mask[0, :4] = 1
    dt = np.full((B, H), -0.1, np.float32)
    dt[0, 4:6] = 0.0
    c.expert.debug_velocity_field(True, 0.0, float("nan"))
    try:
        x1, v = gpu_velocity(c, x0, np.ones((B, H), np.float32), dt, mask)
    finally:
        c.expert.debug_velocity_field(False)
    assert x1[0, :6].tobytes() == x0[0, :6].tobytes()
    assert np.all(np.isnan(x1[0, 6:])) and np.all(np.isnan(v))


@pytest.mark.parametrize("alpha,beta", [(0.0, 0.7), (0.35, -0.2), (-1.3, 0.5)])
def test_linear_field_closed_form_on_gpu(gpu, alpha, beta):
    c = case("pi0_b1_uad")
    c.expert.debug_velocity_field(True, alpha, beta)
    try:
        x, rel, rst = run_schedule_gpu(c, c.noise, c.budgets)
    finally:
        c.expert.debug_velocity_field(False)
    N = c.budgets.astype(np.float64)[..., None]
    dtv = -1.0 / N
    g = (1.0 + alpha * dtv) ** N
    ref = g * c.noise + (beta * (g - 1.0) / alpha if alpha != 0 else beta * N * dtv)
    np.testing.assert_allclose(rel, ref, rtol=2e-6, atol=2e-6)
    np.testing.assert_array_equal(rst, O.release_steps(c.budgets))


def test_run_to_run_determinism(gpu):
    c = case("pi0_b1_uad")
    a = run_schedule_gpu(c, c.noise, c.budgets)
    b = run_schedule_gpu(c, c.noise, c.budgets)
    for u, w in zip(a, b):
        assert u.tobytes() == w.tobytes()


# ----------------------------------------------------------------------------
# Edge cases: ragged chunks, no prefix, single token, batch subsets
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("H,P", [(1, 64), (37, 0), (16, 1), (45, 97)])
def test_ragged_chunk_and_prefix(gpu, H, P):
    c = case("tiny", chunk=H, prefix=P, batch=2)
    m = c.oracle_model()
    n, t, dt, mask = O.build_schedule(np.array([[3] * H, [1 + (i % 4) for i in range(H)]]))
    x_in = c.noise
    v_ref = O.velocity(m, x_in, t[1])
    _, v = gpu_velocity(c, x_in, t[1], dt[1], mask[1])
    for b in range(2):
        e = rel_err(v[b], v_ref[b])
        log(f"[ragged H={H} P={P}] env {b}: velocity rel err {e:.2e}")
        assert e <= VEL_RTOL


def test_batch_subset_matches_full_batch(gpu):
    """A call with fewer environments than the prefix holds uses the first ones."""
    c = case("tiny", batch=3)
    n, t, dt, mask = O.build_schedule(c.budgets)
    _, v3 = gpu_velocity(c, c.noise, t[2], dt[2], mask[2])
    _, v1 = gpu_velocity(c, c.noise[:1], t[2][:1], dt[2][:1], mask[2][:1])
    assert rel_err(v1[0], v3[0]) <= 1e-3


@pytest.mark.gpu
def test_weight_beyond_fp16_range_is_rejected(gpu):
    """Projection weights are held as fp16 (exact for bf16 magnitudes in
    [2^-14, 65504]); a weight outside that range must be refused, not
    silently turned into inf."""
    import paper_2609_37772_amd as U
    case = make_case("tiny", with_expert=False)
    ex = U.ActionExpert(case.wl.shape, 1, case.wl.chunk, case.wl.prefix)
    try:
        bad = dict(case.weights)
        w = bad["layers.0.w_up"].copy()
        w[3, 5] = 1.0e5
        bad["layers.0.w_up"] = w
        with pytest.raises(U.UadError) as ei:
            ex.load_weights(bad)
        assert "fp16" in str(ei.value)
        ex.load_weights(case.weights)  # the same context accepts in-range weights afterwards
    finally:
        ex.close()
