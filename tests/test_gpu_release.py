"""GPU urgency-aware release (UAER, Trajectory Reconciliation + ghosts, Ghost
Action Correction, asynchronous host release) through the C ABI.

Bars: against the oracle's uad_tr_gac, released urgent actions, final states
(ghosts and tail) and GAC-corrected executed actions within 1e-2 absolute;
with K = 1 the TR tail and ghosts equal the GPU's own uniform N*-step
schedule bit for bit (Sec. 4.3, exact recovery); the release path performs
exactly N* joint evaluations.
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_37772_amd as U
from tests.harness import log, make_case

pytestmark = pytest.mark.gpu

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


def gpu_release(c, U_, K, Ns, S, reconcile=True, with_gac=True, gac_mask=None):
    x = dev(c.noise.astype(np.float32))
    B, H, Da = x.shape
    urgent = torch.full((B, U_, Da), float("nan"), device="cuda")
    executed = torch.full((B, S, Da), float("nan"), device="cuda") if with_gac else None
    gm = dev(gac_mask.astype(np.uint8)) if gac_mask is not None else None
    c.expert.release(x, U_, K, Ns, S, reconcile=reconcile, urgent=urgent, executed=executed, gac_mask=gm)
    torch.cuda.synchronize()
    return (x.cpu().numpy(), urgent.cpu().numpy(), None if executed is None else executed.cpu().numpy())


def gpu_uniform(c, Ns):
    n, tg, dtg, mg = c.expert.schedule_tables(np.full(c.budgets.shape, Ns, np.int32))
    x = dev(c.noise.astype(np.float32))
    c.expert.schedule(x, tg, dtg, mg)
    torch.cuda.synchronize()
    return x.cpu().numpy()


@pytest.mark.parametrize("name,U_,Ns,S", [("tiny", 5, 7, 10), ("pi0_b1", 5, 7, 10), ("pi0_b1", 2, 2, 10)])
def test_tr_k1_recovers_uniform_schedule_bit_exact(gpu, name, U_, Ns, S):
    """K = 1: the first joint evaluation equals vanilla's, so the reconciled
    urgent states equal vanilla's x_1 and the whole chunk then follows the
    uniform schedule: tail and ghosts bit-identical to it (Sec. 4.3)."""
    c = case(name)
    if S > c.wl.chunk:
        pytest.skip("chunk shorter than S")
    log(f"[{name}] TR K=1 U={U_} N*={Ns} S={S} vs uniform {Ns}-step schedule")
    x_tr, urgent, _ = gpu_release(c, U_, 1, Ns, S, with_gac=False)
    x_v = gpu_uniform(c, Ns)
    assert np.array_equal(x_tr, x_v), f"max diff {np.abs(x_tr - x_v).max()}"
    # released urgent actions = one Euler step of size 1 from the same velocity
    m = c.oracle_model()
    ref = O.uad_tr_gac(m, c.noise, U_, 1, Ns, S)
    err = np.abs(urgent - ref["released_urgent"]).max()
    log(f"[{name}] urgent max abs err {err:.2e}")
    assert err <= ACT_ATOL


@pytest.mark.parametrize("name,U_,K,Ns,S", [("tiny", 5, 3, 7, 10), ("pi0_b1", 5, 3, 7, 10), ("pi0_b1", 3, 2, 10, 10)])
def test_tr_gac_matches_oracle(gpu, name, U_, K, Ns, S):
    c = case(name)
    log(f"[{name}] TR + GAC U={U_} K={K} N*={Ns} S={S}")
    x, urgent, executed = gpu_release(c, U_, K, Ns, S)
    ref = O.uad_tr_gac(c.oracle_model(), c.noise, U_, K, Ns, S)
    e_u = np.abs(urgent - ref["released_urgent"]).max()
    e_f = np.abs(x - ref["final"]).max()
    e_x = np.abs(executed - ref["executed"]).max()
    log(f"[{name}] urgent {e_u:.2e} final {e_f:.2e} executed {e_x:.2e}")
    assert e_u <= ACT_ATOL and e_f <= ACT_ATOL and e_x <= ACT_ATOL
    # executed = released urgent actions unchanged, then tail + E/(S-U) (Eqs. 8-9)
    assert np.array_equal(executed[:, :U_], urgent)
    E = np.zeros(urgent.shape[::2], np.float32)
    for i in range(U_):
        E = E + (x[:, i] - urgent[:, i])
    np.testing.assert_allclose(executed[:, U_:S], x[:, U_:S] + (E / np.float32(S - U_))[:, None, :],
                               rtol=0, atol=1e-6)


@pytest.mark.parametrize("name", ["tiny", "pi0_b1"])
def test_plain_early_release_matches_oracle(gpu, name):
    """UAER without reconciliation: urgent tokens frozen at x_K, still context."""
    c = case(name)
    U_, K, Ns, S = 5, 2, 7, 10
    x, urgent, _ = gpu_release(c, U_, K, Ns, S, reconcile=False, with_gac=False)
    ref = O.uad_tr_gac(c.oracle_model(), c.noise, U_, K, Ns, S, reconcile=False)
    assert np.array_equal(x[:, :U_], urgent), "frozen urgent states must stay bit-identical to the release"
    e_u = np.abs(urgent - ref["released_urgent"]).max()
    e_f = np.abs(x - ref["final"]).max()
    log(f"[{name}] UAER urgent {e_u:.2e} final {e_f:.2e}")
    assert e_u <= ACT_ATOL and e_f <= ACT_ATOL


def test_gac_dimension_mask(gpu):
    """Masked dimensions (e.g. a gripper) keep the denoised tail unchanged."""
    c = case("tiny")
    Da = c.wl.shape.action_dim
    mask = (np.arange(Da) % 3 != 2).astype(np.uint8)
    x, urgent, executed = gpu_release(c, 4, 1, 5, 10, gac_mask=mask)
    keep = mask == 0
    assert np.array_equal(executed[:, 4:10][..., keep], x[:, 4:10][..., keep])
    assert not np.array_equal(executed[:, 4:10][..., ~keep], x[:, 4:10][..., ~keep])


def test_async_release_to_pinned_host(gpu):
    """The urgent actions reach pinned host memory on the release stream and the
    release event fires; values equal the device copy bit for bit."""
    c = case("pi0_b1")
    B, H, Da = c.noise.shape
    x = dev(c.noise.astype(np.float32))
    urgent = torch.empty((B, 5, Da), device="cuda")
    host = torch.full((B, 5, Da), float("nan")).pin_memory()
    ev = torch.cuda.Event()
    ticks = torch.zeros(8, dtype=torch.uint64).pin_memory()
    c.expert.release(x, 5, 1, 7, 10, urgent=urgent, urgent_host=host, release_event=ev, step_ticks=ticks)
    ev.synchronize()
    got = host.clone()
    torch.cuda.synchronize()
    assert torch.equal(got, urgent.cpu())
    tk = ticks.numpy().astype(np.int64)
    assert np.all(np.diff(tk) > 0), "step ticks must increase"


def test_release_to_pageable_host_through_c_abi(gpu):
    """Host memory that is not page-locked (a NumPy array) takes the copy on
    the release stream instead of the release kernel's direct stores: the
    values still equal the device copy bit for bit, and the pinned path on
    the same context still works afterwards."""
    import ctypes
    c = case("tiny")
    B, H, Da = c.noise.shape
    U_, K, Ns, S = 4, 2, 5, 10
    lib = U.load_library()
    x = dev(c.noise.astype(np.float32))
    urgent = torch.empty((B, U_, Da), device="cuda")
    host = np.full((B, U_, Da), np.nan, np.float32)
    vp = ctypes.c_void_p
    st = lib.uad_denoise_release(c.expert.ctx, vp(x.data_ptr()), B, H, U_, K, Ns, S, U.UAD_RELEASE_TR,
                                 vp(urgent.data_ptr()), None, None, vp(host.ctypes.data), None, None)
    assert st == 0
    torch.cuda.synchronize()  # the release stream's copy included
    assert np.array_equal(host, urgent.cpu().numpy())
    pinned = torch.full((B, U_, Da), float("nan")).pin_memory()
    ev = torch.cuda.Event()
    x2 = dev(c.noise.astype(np.float32))
    c.expert.release(x2, U_, K, Ns, S, urgent=urgent, urgent_host=pinned, release_event=ev)
    ev.synchronize()
    got = pinned.clone()
    torch.cuda.synchronize()
    assert torch.equal(got, urgent.cpu())
    assert np.array_equal(host, got.numpy())  # same inputs, same release


def test_release_costs_exactly_nstar_evaluations(gpu):
    """TR needs no extra F_theta evaluations (Sec. 4.3): N* joint steps in total."""
    c = case("tiny")
    U.uad_profile_enable(c.expert.ctx, True)
    try:
        gpu_release(c, 5, 3, 7, 10)
        prof = U.uad_profile_read(c.expert.ctx)
    finally:
        U.uad_profile_enable(c.expert.ctx, False)
    assert prof["final_euler"][1] == 7
    assert prof["temb"][1] == 7


@pytest.mark.parametrize("U_,K,Ns,S,reconcile,gac", [
    (0, 1, 7, 10, True, False), (5, 0, 7, 10, True, False), (5, 7, 7, 10, True, False),
    (10, 1, 7, 10, True, False), (5, 1, 65, 10, True, False), (5, 1, 7, 10, False, True)])
def test_release_argument_errors(gpu, U_, K, Ns, S, reconcile, gac):
    c = case("tiny")
    x = dev(c.noise.astype(np.float32))
    B, H, Da = x.shape
    urgent = torch.empty((B, max(U_, 1), Da), device="cuda")
    executed = torch.empty((B, S, Da), device="cuda") if gac else None
    mode = U.UAD_RELEASE_TR if reconcile else U.UAD_RELEASE_UAER
    with pytest.raises(U.UadError) as ei:
        U.uad_denoise_release(c.expert.ctx, x, U_, K, Ns, S, mode, urgent if U_ >= 1 else urgent[:, :0],
                              executed)
    assert ei.value.status == 1  # UAD_E_INVALID
