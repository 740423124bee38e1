"""GPU edge cases through the C ABI: argument errors of a step and a schedule
(empty and oversized shapes, missing state), the shortest and longest
schedules (every budget 1; a budget of 64, the largest the schedule builder
takes), and a mid-size batch (8 environments, 400 rows) where the attention
splits its keys over a few long streamed splits and the projections mix the
small-M and the batched kernels.

Bars as for the other parity tests: velocities within a normwise max
relative error of 2e-2, released actions within 1e-2 absolute, release steps
bit-exact.
"""
import ctypes

import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_37772_amd as U
from tests.harness import log, make_case, prefix_stack_bf16, rel_err

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


def schedule_gpu(c, budgets):
    n, tg, dtg, mg = c.expert.schedule_tables(budgets)
    x = dev(c.noise.astype(np.float32))
    rel = torch.zeros_like(x)
    rst = torch.full(budgets.shape, -1, dtype=torch.int32, device="cuda")
    c.expert.schedule(x, tg, dtg, mg, rel, rst)
    torch.cuda.synchronize()
    return n, x.cpu().numpy(), rel.cpu().numpy(), rst.cpu().numpy()


def test_step_and_schedule_argument_errors(gpu):
    """Zero or oversized batch / chunk, null pointers, zero steps: rejected
    before any device work, with the status the header documents."""
    c = case("tiny")
    lib = U.load_library()
    B, H, Da = c.noise.shape
    x = dev(c.noise.astype(np.float32))
    t = torch.ones((B, H), device="cuda")
    dt = torch.zeros((B, H), device="cuda")
    m = torch.zeros((B, H), dtype=torch.uint8, device="cuda")
    p = [ctypes.c_void_p(v.data_ptr()) for v in (x, t, dt, m)]
    ctx = c.expert.ctx
    for bb, hh, want in [(0, H, 1), (B, 0, 1), (-1, H, 1), (B + 1, H, 2), (B, H + 1000, 2)]:
        assert lib.uad_denoise_step(ctx, *p, None, bb, hh) == want
        assert lib.uad_denoise_schedule(ctx, *p, 1, bb, hh, None, None, None) == want
    assert lib.uad_denoise_step(ctx, None, *p[1:], None, B, H) == 1
    assert lib.uad_denoise_schedule(ctx, *p, 0, B, H, None, None, None) == 1
    assert "n_steps" in U.uad_last_error(ctx)
    # a context without weights or prefix: UAD_E_STATE
    fresh = U.ActionExpert(c.wl.shape, B, H, c.wl.prefix)
    try:
        assert lib.uad_denoise_step(fresh.ctx, *p, None, B, H) == 3
        assert "weights" in U.uad_last_error(fresh.ctx)
    finally:
        fresh.close()
    # the valid call still works afterwards
    c.expert.step(x, t, dt, m)
    torch.cuda.synchronize()
    assert torch.equal(x.cpu(), torch.from_numpy(c.noise.astype(np.float32)))  # dt = 0: unchanged


@pytest.mark.parametrize("kind", ["all_ones", "max_budget"])
def test_shortest_and_longest_schedules(gpu, kind):
    c = case("tiny")
    B, H = c.budgets.shape
    if kind == "all_ones":
        bud = np.ones((B, H), np.int32)
    else:
        bud = np.full((B, H), 10, np.int32)
        bud[0, ::3] = 64
        bud[0, 1] = 1
    r = O.denoise_schedule(c.oracle_model(), c.noise, bud)
    n, x, rel, rst = schedule_gpu(c, bud)
    assert n == int(bud.max())
    ex, er = float(np.abs(x - r["x"]).max()), float(np.abs(rel - r["released"]).max())
    log(f"[tiny {kind}] {n} steps: final max abs err {ex:.2e}, released {er:.2e}")
    assert ex <= ACT_ATOL and er <= ACT_ATOL
    np.testing.assert_array_equal(rst, r["release_step"])


def test_mid_batch_sampled_envs(gpu):
    """8 environments of the pi0-scale model (400 rows): streamed split-KV
    attention with a merge, mixed projection kernels; sampled environments
    against the oracle run alone."""
    c = case("pi0_fleet_b64", batch=8)
    B, H = c.budgets.shape
    n, t, dt, mask = O.build_schedule(c.budgets)
    xg = dev(c.noise.astype(np.float32))
    vg = torch.empty_like(xg)
    c.expert.step(xg, dev(t[0].astype(np.float32)), dev(dt[0].astype(np.float32)), dev(mask[0].astype(np.uint8)), vg)
    torch.cuda.synchronize()
    v = vg.cpu().numpy()
    _, x, rel, rst = schedule_gpu(c, c.budgets)
    for b in (0, B - 1):
        mb = c.oracle_model([b])
        e = rel_err(v[b], O.velocity(mb, c.noise[b:b + 1], t[0][b:b + 1])[0])
        r = O.denoise_schedule(mb, c.noise[b:b + 1], c.budgets[b:b + 1])
        ea = float(np.abs(rel[b] - r["released"][0]).max())
        log(f"[pi0 B=8] env {b}: step-0 velocity rel err {e:.2e}, released abs err {ea:.2e}")
        assert e <= VEL_RTOL and ea <= ACT_ATOL
    np.testing.assert_array_equal(rst, O.release_steps(c.budgets))


def test_tall_query_blocks_sampled_envs(gpu):
    """40 environments of the small model with a 128-token chunk and a 256-token
    prefix (12 key blocks, no split-KV): the attention runs 8-wave workgroups
    of 128 query rows, one per (environment, KV head); the other row-block
    sizes are covered by the fleet (7 waves) and the large expert (6).
    Sampled environments against the oracle run alone."""
    c = case("tiny", batch=40, chunk=128, prefix=256)
    B, H = c.budgets.shape
    n, t, dt, mask = O.build_schedule(c.budgets)
    xg = dev(c.noise.astype(np.float32))
    vg = torch.empty_like(xg)
    c.expert.step(xg, dev(t[0].astype(np.float32)), dev(dt[0].astype(np.float32)), dev(mask[0].astype(np.uint8)), vg)
    torch.cuda.synchronize()
    v = vg.cpu().numpy()
    _, x, rel, rst = schedule_gpu(c, c.budgets)
    for b in (0, 23, B - 1):
        mb = c.oracle_model([b])
        e = rel_err(v[b], O.velocity(mb, c.noise[b:b + 1], t[0][b:b + 1])[0])
        r = O.denoise_schedule(mb, c.noise[b:b + 1], c.budgets[b:b + 1])
        ea = float(np.abs(rel[b] - r["released"][0]).max())
        log(f"[tiny B=40 H=128] env {b}: step-0 velocity rel err {e:.2e}, released abs err {ea:.2e}")
        assert e <= VEL_RTOL and ea <= ACT_ATOL
    np.testing.assert_array_equal(rst, O.release_steps(c.budgets))


@pytest.mark.parametrize("name,kw,envs", [
    # head dim 64: 128 + 211 = 339 keys, 11 key blocks, the last holding 19
    ("tiny", dict(batch=40, chunk=128, prefix=211), (0, 39)),
    # head dim 128: 128 + 980 = 1108 keys, 35 key blocks, the last holding 20
    ("large_b16", dict(prefix=980), (0, 15)),
], ids=["hd64", "hd128"])
def test_tall_query_blocks_odd_ragged_keys(gpu, name, kw, envs):
    """Tall attention workgroups (no split-KV) stage two key blocks at a time at
    head dims 64 and 128; an odd block count leaves a last stage of one block,
    and a ragged key count a partly masked last block.  Step-0 velocities of
    sampled environments, and the first one's released actions, against the
    oracle run alone; release steps bit-exact."""
    c = case(name, **kw)
    B, H = c.budgets.shape
    assert (c.wl.prefix + c.wl.chunk) % 32 and ((c.wl.prefix + c.wl.chunk + 31) // 32) % 2 == 1
    n, t, dt, mask = O.build_schedule(c.budgets)
    xg = dev(c.noise.astype(np.float32))
    vg = torch.empty_like(xg)
    c.expert.step(xg, dev(t[0].astype(np.float32)), dev(dt[0].astype(np.float32)), dev(mask[0].astype(np.uint8)), vg)
    torch.cuda.synchronize()
    v = vg.cpu().numpy()
    _, x, rel, rst = schedule_gpu(c, c.budgets)
    for i, b in enumerate(envs):
        mb = c.oracle_model([b])
        e = rel_err(v[b], O.velocity(mb, c.noise[b:b + 1], t[0][b:b + 1])[0])
        log(f"[{name} P={c.wl.prefix} H={H}] env {b}: step-0 velocity rel err {e:.2e}")
        assert e <= VEL_RTOL
        if i == 0:
            r = O.denoise_schedule(mb, c.noise[b:b + 1], c.budgets[b:b + 1])
            ea = float(np.abs(rel[b] - r["released"][0]).max())
            log(f"[{name} P={c.wl.prefix} H={H}] env {b}: released abs err {ea:.2e}")
            assert ea <= ACT_ATOL
    np.testing.assert_array_equal(rst, O.release_steps(c.budgets))


def test_fp16_operand_overflow_raises_range_status(gpu):
    """An activation beyond the fp16 range (the fp32 action input projection
    scaled by 1e7, so that |W_in x| is far above 65504 in the time MLP's fp16
    operand) raises UAD_E_RANGE at the next synchronisation instead of passing
    as inf; the report clears the status, and in-range weights run clean."""
    c = make_case("tiny", with_expert=False)
    ex = U.ActionExpert(c.wl.shape, 1, c.wl.chunk, c.wl.prefix)
    try:
        K, V = prefix_stack_bf16(c)
        ex.set_prefix_kv(K, V, 1, c.wl.prefix)
        big = dict(c.weights)
        big["action_in.w"] = (c.weights["action_in.w"] * np.float32(1e7)).astype(np.float32)
        ex.load_weights(big)
        n, t, dt, mask = O.build_schedule(c.budgets)
        x = dev(c.noise.astype(np.float32))
        ex.step(x, dev(t[0]), dev(dt[0]), dev(mask[0]))
        with pytest.raises(U.UadError) as ei:
            ex.synchronize()
        assert ei.value.status == 8 and "65504" in str(ei.value)
        ex.synchronize()  # reported once, then cleared
        ex.load_weights(c.weights)
        x = dev(c.noise.astype(np.float32))
        v = torch.empty_like(x)
        ex.step(x, dev(t[0]), dev(dt[0]), dev(mask[0]), v)
        ex.synchronize()
        assert torch.isfinite(v).all()
    finally:
        ex.close()


def test_split_partials_sized_for_every_prefix(gpu):
    """A context for prefixes up to 2048 keys, called with 2 environments, a
    71-action chunk and a 1722-key prefix: that call splits the keys 15 ways,
    more than the longest prefix does (14), since the split count is not
    monotone in the prefix length.  The workspace is sized over every prefix
    length, and the step matches the oracle."""
    c = make_case("tiny", with_expert=False, batch=2, chunk=71, prefix=1722)
    ex = U.ActionExpert(c.wl.shape, 2, 128, 2048)
    try:
        ex.load_weights(c.weights)
        K, V = prefix_stack_bf16(c)
        ex.set_prefix_kv(K, V, 2, 1722)
        n, t, dt, mask = O.build_schedule(c.budgets)
        v_ref = O.velocity(c.oracle_model(), c.noise, t[0])
        x = dev(c.noise.astype(np.float32))
        v = torch.empty_like(x)
        ex.step(x, dev(t[0]), dev(dt[0]), dev(mask[0]), v)
        ex.synchronize()
        v = v.cpu().numpy()
        for b in range(2):
            e = rel_err(v[b], v_ref[b])
            log(f"[P=1722 of 2048, H=71, B=2] env {b}: velocity rel err {e:.2e}")
            assert e <= VEL_RTOL
    finally:
        ex.close()


def _random_shapes(seed, n):
    """n seeded (batch, chunk, prefix) triples of the small model: 1..24 environments,
    1..128 actions, 0..700 prefix tokens (crossing the split-KV, tall-workgroup and
    ragged-block boundaries of the attention and the small-M / batched projections)."""
    rs = np.random.RandomState(seed)
    return [(int(rs.randint(1, 25)), int(rs.randint(1, 129)), int(rs.randint(0, 701))) for _ in range(n)]


@pytest.mark.parametrize("B,H,P", _random_shapes(20261202, 8))
def test_random_shapes_every_env(gpu, B, H, P):
    """Seeded random shapes of the small model, every environment against the
    oracle: step-0 velocities, then a whole schedule's released actions, final
    states and release steps."""
    c = make_case("tiny", batch=B, chunk=H, prefix=P)
    try:
        m = c.oracle_model()
        n, t, dt, mask = O.build_schedule(c.budgets)
        xg = dev(c.noise.astype(np.float32))
        vg = torch.empty_like(xg)
        c.expert.step(xg, dev(t[0].astype(np.float32)), dev(dt[0].astype(np.float32)),
                      dev(mask[0].astype(np.uint8)), vg)
        torch.cuda.synchronize()
        v_ref = O.velocity(m, c.noise, t[0])
        ev = max(rel_err(vg.cpu().numpy()[b], v_ref[b]) for b in range(B))
        r = O.denoise_schedule(m, c.noise, c.budgets)
        _, x, rel, rst = schedule_gpu(c, c.budgets)
        ea = float(np.abs(rel - r["released"]).max())
        ex = float(np.abs(x - r["x"]).max())
        log(f"[tiny B={B} H={H} P={P}] worst step-0 velocity rel err {ev:.2e}, released {ea:.2e}, final {ex:.2e}")
        assert ev <= VEL_RTOL and ea <= ACT_ATOL and ex <= ACT_ATOL
        np.testing.assert_array_equal(rst, r["release_step"])
    finally:
        c.expert.close()


@pytest.mark.parametrize("Da", [7, 20])
def test_batched_final_projection_ragged_rows_and_outputs(gpu, Da):
    """The batched final projection (fp32 MFMA from 1024 tokens when the width is a
    multiple of 512): 21 environments x 50 actions = 1050 token rows (the last
    16-row tile holds 10), Da = 7 (one partial output tile) or 20 (a full and a
    partial one), width 512, every environment against the oracle: step-0
    velocities, then a whole schedule's released actions, final states and
    release steps."""
    import uad_workloads as W
    shape = W.ModelShape(2, 512, 4, 4, 64, 1024, Da)
    c = make_case("tiny", batch=21, chunk=50, prefix=40, shape=shape)
    try:
        m = c.oracle_model()
        n, t, dt, mask = O.build_schedule(c.budgets)
        xg = dev(c.noise.astype(np.float32))
        vg = torch.empty_like(xg)
        c.expert.step(xg, dev(t[0].astype(np.float32)), dev(dt[0].astype(np.float32)),
                      dev(mask[0].astype(np.uint8)), vg)
        torch.cuda.synchronize()
        v_ref = O.velocity(m, c.noise, t[0])
        ev = max(rel_err(vg.cpu().numpy()[b], v_ref[b]) for b in range(c.wl.batch))
        r = O.denoise_schedule(m, c.noise, c.budgets)
        _, x, rel, rst = schedule_gpu(c, c.budgets)
        ea = float(np.abs(rel - r["released"]).max())
        ex = float(np.abs(x - r["x"]).max())
        log(f"[final rows 1050, Da={Da}, d=512] worst step-0 velocity rel err {ev:.2e}, released {ea:.2e}, "
            f"final {ex:.2e}")
        assert ev <= VEL_RTOL and ea <= ACT_ATOL and ex <= ACT_ATOL
        np.testing.assert_array_equal(rst, r["release_step"])
    finally:
        c.expert.close()


@pytest.mark.parametrize("width,B,H", [(1024, 32, 50), (1024, 22, 50), (1536, 8, 128), (1536, 8, 125),
                                       (1024, 64, 50), (1536, 16, 128)],
                         ids=["w1024_1600rows", "w1024_1100rows_3way", "w1536_1024rows", "w1536_1000rows",
                              "w1024_3200rows_down", "w1536_2048rows_down"])
def test_split_k_residual_projections(gpu, width, B, H):
    """Residual projections split over K (tiles filling at most half the CUs:
    1600 rows x 1024 columns = 104 tiles of 128 x 128, two ways; 1100 rows =
    72 tiles, down (K = 4096) three ways over uneven k-ranges of 42 and 43
    blocks; 1024 and 1000 rows x 1536 = 128 tiles of 128 x 96, two ways; the
    1600-, 1100- and 1000-row cases end in a ragged row panel), and only down
    (K >= 4096), two ways, where the tiles fill more than half the CUs (3200
    rows x 1024 = 200 tiles, 2048 rows x 1536 = 256 tiles of 96 columns),
    2 layers of the pi0-scale and large experts' widths:
    step-0 velocities of every environment against the oracle, the same step
    24 times more bit for bit (the partials are added in split order whatever
    the arrival order), then a whole schedule's released actions and final
    states."""
    _two_layer_case(width, B, H, "split-K")


@pytest.mark.parametrize("B,rows", [(11, 144), (12, 160)], ids=["1408rows_144", "1536rows_160"])
def test_gate_up_taller_tiles_long_k(gpu, B, rows):
    """Gate/up of the 1536-wide expert (K = 1536) on taller tiles: 11
    environments x 128 tokens = 1408 rows make 528 tiles of 128 x 256 for 512
    co-resident workgroups but 480 of 144 x 256 (3-stage ring, the last panel
    112 rows); 12 environments (1536 rows, 576 tiles) 480 of 160 x 256
    (2-stage ring, the last panel 96 rows); 2 layers, the same checks as the
    split-K cases (down splits two ways here too)."""
    _two_layer_case(1536, B, 128, f"gate/up {rows}-row tiles")


def _two_layer_case(width, B, H, label):
    import uad_workloads as W
    shape = (W.ModelShape(2, 1024, 8, 1, 256, 4096, 32) if width == 1024
             else W.ModelShape(2, 1536, 12, 2, 128, 6144, 32))
    c = make_case("pi0_fleet_b64", batch=B, chunk=H, prefix=64, shape=shape)
    try:
        m = c.oracle_model()
        n, t, dt, mask = O.build_schedule(c.budgets)
        xg = dev(c.noise.astype(np.float32))
        args = (dev(t[0].astype(np.float32)), dev(dt[0].astype(np.float32)), dev(mask[0].astype(np.uint8)))
        v1, v2 = torch.empty_like(xg), torch.empty_like(xg)
        c.expert.step(xg.clone(), *args, v1)
        repeats_equal = True
        for _ in range(24):  # the partials' arrival order varies from call to call; the sums must not
            c.expert.step(xg.clone(), *args, v2)
            repeats_equal &= bool(torch.equal(v1, v2))
        torch.cuda.synchronize()
        v_ref = O.velocity(m, c.noise, t[0])
        ev = max(rel_err(v1.cpu().numpy()[b], v_ref[b]) for b in range(B))
        r = O.denoise_schedule(m, c.noise, c.budgets)
        _, x, rel, rst = schedule_gpu(c, c.budgets)
        ea = float(np.abs(rel - r["released"]).max())
        ex = float(np.abs(x - r["x"]).max())
        log(f"[{label} width {width}, {B * H} rows] worst step-0 velocity rel err {ev:.2e}, released {ea:.2e}, "
            f"final {ex:.2e}")
        assert repeats_equal
        assert ev <= VEL_RTOL and ea <= ACT_ATOL and ex <= ACT_ATOL
        np.testing.assert_array_equal(rst, r["release_step"])
    finally:
        c.expert.close()

