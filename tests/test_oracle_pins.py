"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test checks one function against brute force on tiny inputs, a closed
form, a library routine (torch CPU / scipy) or an invariant the paper states,
chosen so that a dropped term, a wrong sign or index, or a transposed operand
fails at least one of them.
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
import uad_workloads as W
from tests import bruteforce

TINY = W.ModelShape(n_layers=2, d_model=8, n_heads=2, n_kv_heads=1, head_dim=4, d_ff=12, action_dim=3)


def tiny_model(shape=TINY, P=3, B=1, seed=7, dtype=np.float64, scale=0.5):
    """A tiny model with non-square, non-symmetric weights (larger scale so every term matters)."""
    wl = W.Workload("t", shape, B, 2, P, "uniform", (3,), bf16=False, seed=seed)
    weights = {}
    for name, shp, kind in W.weight_specs(shape):
        z = W.draw(seed, name, shp, scale)
        weights[name] = z + 1.0 if kind == "gain" else z
    pk, pv = zip(*[W.make_prefix(wl, b) for b in range(B)])
    return O.build_model(shape, weights, pk, pv, dtype=dtype), weights, pk, pv


# ----------------------------------------------------------------------------
# Components against library routines / closed forms / brute force
# ----------------------------------------------------------------------------
def test_attention_matches_scalar_bruteforce_float64():
    rng = np.random.default_rng(1)
    T, S, Hq, Hkv, hd = 2, 5, 2, 1, 4
    q = rng.standard_normal((T, Hq, hd))
    k = rng.standard_normal((S, Hkv, hd))
    v = rng.standard_normal((S, Hkv, hd))
    o = O.attention(q, k, v)
    for i in range(T):
        for j in range(Hq):
            sc = [sum(q[i, j, c] * k[s, 0, c] for c in range(hd)) / math.sqrt(hd) for s in range(S)]
            ex = [math.exp(x) for x in sc]          # unshifted: shift-invariance is part of the check
            den = sum(ex)
            for c in range(hd):
                ref = sum(ex[s] * v[s, 0, c] for s in range(S)) / den
                assert abs(o[i, j, c] - ref) < 1e-12


def test_attention_gqa_equals_explicit_replication_and_torch_sdpa():
    rng = np.random.default_rng(2)
    T, S, Hq, Hkv, hd = 5, 9, 6, 2, 8
    q = rng.standard_normal((T, Hq, hd))
    k = rng.standard_normal((S, Hkv, hd))
    v = rng.standard_normal((S, Hkv, hd))
    o = O.attention(q, k, v)
    # query head j reads kv head floor(j*Hkv/Hq): heads 0-2 -> 0, 3-5 -> 1
    krep = np.repeat(k, Hq // Hkv, axis=1)
    vrep = np.repeat(v, Hq // Hkv, axis=1)
    np.testing.assert_allclose(O.attention(q, krep, vrep), o, rtol=0, atol=1e-13)
    tq = torch.from_numpy(q).permute(1, 0, 2)[None]
    tk = torch.from_numpy(krep).permute(1, 0, 2)[None]
    tv = torch.from_numpy(vrep).permute(1, 0, 2)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv)[0].permute(1, 0, 2).numpy()
    np.testing.assert_allclose(o, ref, rtol=0, atol=1e-12)


def test_attention_identical_keys_gives_mean_of_values():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((4, 2, 8))
    k = np.repeat(rng.standard_normal((1, 1, 8)), 7, axis=0)
    v = rng.standard_normal((7, 1, 8))
    o = O.attention(q, k, v)
    np.testing.assert_allclose(o, np.broadcast_to(v.mean(axis=0)[None], o.shape), atol=1e-13)


def test_rms_norm_constant_vector_and_torch():
    for c in (3.0, -0.25, 1e-4):
        h = np.full((1, 16), c)
        g = np.linspace(0.5, 1.5, 16)
        out = O.rms_norm(h, g, 1e-6)
        np.testing.assert_allclose(out[0], c / math.sqrt(c * c + 1e-6) * g, rtol=1e-14)
    rng = np.random.default_rng(4)
    h = rng.standard_normal((5, 32))
    g = rng.standard_normal(32)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(h), (32,), torch.from_numpy(g), eps=1e-6).numpy()
    np.testing.assert_allclose(O.rms_norm(h, g, 1e-6), ref, rtol=1e-13)
    # scale invariance (eps aside)
    np.testing.assert_allclose(O.rms_norm(7.0 * h, g, 0.0), O.rms_norm(h, g, 0.0), rtol=1e-13)


def test_gelu_tanh_special_values_and_library():
    z = np.linspace(-6, 6, 1001)
    gz = O.gelu_tanh(z)
    assert O.gelu_tanh(np.array([0.0]))[0] == 0.0
    # odd-part identity of the tanh form: gelu(z) - gelu(-z) = z exactly in reals
    np.testing.assert_allclose(gz - O.gelu_tanh(-z), z, atol=1e-14)
    ref = torch.nn.functional.gelu(torch.from_numpy(z), approximate="tanh").numpy()
    np.testing.assert_allclose(gz, ref, atol=1e-14)
    # close to the exact erf GELU (the tanh form is an approximation of it)
    from scipy.special import erf
    exact = 0.5 * z * (1 + erf(z / math.sqrt(2)))
    assert np.max(np.abs(gz - exact)) < 1e-3


def test_silu_identity_and_library():
    z = np.linspace(-8, 8, 513)
    np.testing.assert_allclose(O.silu(z) - O.silu(-z), z, atol=1e-13)
    np.testing.assert_allclose(O.silu(z), torch.nn.functional.silu(torch.from_numpy(z)).numpy(), atol=1e-14)


def test_time_embedding_special_values():
    d = 16
    e0 = O.time_embedding(np.zeros(3), d)
    np.testing.assert_array_equal(e0[:, : d // 2], 0.0)
    np.testing.assert_array_equal(e0[:, d // 2:], 1.0)
    t = np.array([0.1, 0.37, 1.0])
    e = O.time_embedding(t, d)
    np.testing.assert_allclose(e[:, : d // 2] ** 2 + e[:, d // 2:] ** 2, 1.0, atol=1e-14)
    # first frequency is 1000, frequencies fall geometrically by 10000^(1/(d/2))
    np.testing.assert_allclose(e[:, 0], np.sin(1000.0 * t), atol=1e-12)
    w = O.time_frequencies(d, np.float64)
    np.testing.assert_allclose(w[1:] / w[:-1], 10000.0 ** (-1.0 / (d // 2)), rtol=1e-14)


def test_full_forward_matches_scalar_bruteforce():
    m, weights, pk, pv = tiny_model()
    rng = np.random.default_rng(5)
    x = rng.standard_normal((2, TINY.action_dim))
    t = np.array([0.9, 0.25])
    got = O.action_expert(m, 0, x, t)
    Wl = {k: v.tolist() for k, v in weights.items()}
    ref = bruteforce.forward_env(Wl, TINY, pk[0].tolist(), pv[0].tolist(), x.tolist(), t.tolist())
    np.testing.assert_allclose(got, np.array(ref), rtol=0, atol=1e-11)


def test_forward_bruteforce_mha_and_wider_gqa():
    shape = W.ModelShape(n_layers=1, d_model=12, n_heads=3, n_kv_heads=3, head_dim=2, d_ff=5, action_dim=2)
    m, weights, pk, pv = tiny_model(shape, P=2, seed=11)
    x = np.random.default_rng(6).standard_normal((2, 2))
    t = np.array([0.5, 0.0])
    ref = bruteforce.forward_env({k: v.tolist() for k, v in weights.items()}, shape,
                                 pk[0].tolist(), pv[0].tolist(), x.tolist(), t.tolist())
    np.testing.assert_allclose(O.action_expert(m, 0, x, t), np.array(ref), atol=1e-11)


def test_permutation_equivariance_without_positions():
    m, *_ = tiny_model()
    rng = np.random.default_rng(8)
    x = rng.standard_normal((5, TINY.action_dim))
    t = rng.uniform(0, 1, 5)
    perm = np.array([3, 0, 4, 1, 2])
    v = O.action_expert(m, 0, x, t)
    vp = O.action_expert(m, 0, x[perm], t[perm])
    np.testing.assert_allclose(vp, v[perm], atol=1e-12)


def test_zero_output_weight_gives_bias():
    m, *_ = tiny_model()
    m.weights["action_out.w"] = np.zeros_like(m.weights["action_out.w"])
    v = O.action_expert(m, 0, np.ones((2, 3)), np.array([0.3, 0.7]))
    np.testing.assert_array_equal(v, np.broadcast_to(m.weights["action_out.b"], v.shape))


def test_batch_envs_are_independent():
    m, *_ = tiny_model(B=3)
    rng = np.random.default_rng(9)
    x = rng.standard_normal((3, 4, 3))
    t = rng.uniform(0, 1, (3, 4))
    vb = O.velocity(m, x, t)
    for b in range(3):
        np.testing.assert_array_equal(vb[b], O.action_expert(m, b, x[b], t[b]))
    # envs really differ (own prefix), so independence is not vacuous
    assert np.max(np.abs(O.action_expert(m, 0, x[1], t[1]) - vb[1])) > 1e-6


# ----------------------------------------------------------------------------
# Schedule, integrator and the paper's invariants
# ----------------------------------------------------------------------------
def test_schedule_tables_closed_form_groups():
    """Budgets 4/7/10 over tokens 0-4/5-24/25-49 (Eqs. 4-5): exact integer/fraction structure."""
    bud = W.make_budgets(W.get_workload("pi0_b1_uad"))
    n, t, dt, mask = O.build_schedule(bud)
    assert n == 10 and t.shape == (10, 1, 50)
    for k in range(10):
        for i in range(50):
            N = 4 if i < 5 else (7 if i < 25 else 10)
            assert mask[k, 0, i] == (1 if k >= N else 0)
            assert t[k, 0, i] == np.float32(max(N - k, 0)) / np.float32(N)
            assert dt[k, 0, i] == (np.float32(-1.0) / np.float32(N) if k < N else 0.0)
    assert np.all(t[0] == 1.0)
    np.testing.assert_array_equal(O.release_steps(bud)[0, [0, 4, 5, 24, 25, 49]], [3, 3, 6, 6, 9, 9])


def test_schedule_from_golden_fixture():
    """Hand-derived rows for the 4/7/10 UAD schedule, tests/golden/schedule_uad_4_7_10.txt."""
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "schedule_uad_4_7_10.txt")
    bud = W.make_budgets(W.get_workload("pi0_b1_uad"))
    n, t, dt, mask = O.build_schedule(bud)
    rows = [ln.split() for ln in open(path) if ln.strip() and not ln.startswith("#")]
    assert len(rows) == 30
    for step, tok, tn, td, dn, dd, mk in rows:
        k, i = int(step), int(tok)
        assert t[k, 0, i] == np.float32(int(tn)) / np.float32(int(td))
        assert dt[k, 0, i] == (np.float32(int(dn)) / np.float32(int(dd)) if int(dd) else 0.0)
        assert mask[k, 0, i] == int(mk)


def test_linear_budgets_counts():
    bud = W.make_budgets(W.get_workload("large_b16"))[0]
    assert bud[0] == 3 and bud[-1] == 12 and np.all(np.diff(bud) >= 0)
    counts = [int(np.sum(bud == n)) for n in range(3, 13)]
    assert counts == [8, 14, 14, 14, 14, 14, 14, 14, 14, 8]


def test_random_budgets_within_range():
    bud = W.make_budgets(W.get_workload("pi0_fleet_b64"))
    assert bud.shape == (64, 50) and bud.min() >= 3 and bud.max() <= 10
    for b in range(64):
        vals = np.unique(bud[b])
        assert len(vals) == 2 and vals[0] < vals[1]
        U = int(np.sum(bud[b] == vals[0]))
        assert 3 <= U <= 10 and np.all(bud[b, :U] == vals[0])


def test_uniform_schedule_reproduces_vanilla_bit_exact():
    m, *_ = tiny_model(dtype=np.float32, B=2)
    x0 = np.random.default_rng(10).standard_normal((2, 4, 3)).astype(np.float32)
    for N in (1, 2, 3, 5):
        r = O.denoise_schedule(m, x0, np.full((2, 4), N))
        van = O.vanilla_denoise(m, x0, N)
        assert r["x"].tobytes() == van.tobytes()
        assert r["released"].tobytes() == van.tobytes()


def test_frozen_tokens_bit_identical_with_nan_and_negzero():
    x = np.array([[[-0.0, 1.5], [2.0, -3.0], [0.5, 0.25]]], np.float32)
    v = np.array([[[np.nan, np.inf], [1.0, 1.0], [-np.inf, 0.0]]], np.float32)
    dt = np.array([[-0.5, -0.5, 0.0]], np.float32)
    mask = np.array([[1, 0, 0]], np.uint8)
    out = O.euler_update(x, v, dt, mask)
    assert out[0, 0].tobytes() == x[0, 0].tobytes()     # masked: copied even with NaN/Inf v
    assert out[0, 2].tobytes() == x[0, 2].tobytes()     # dt == 0: copied
    np.testing.assert_array_equal(out[0, 1], [1.5, -3.5])
    assert np.signbit(out[0, 0, 0])


def test_frozen_tokens_stay_fixed_through_schedule():
    m, *_ = tiny_model(dtype=np.float32)
    x0 = np.random.default_rng(11).standard_normal((1, 4, 3)).astype(np.float32)
    bud = np.array([[1, 2, 4, 4]])
    r = O.denoise_schedule(m, x0, bud, keep_history=True)
    for i, N in enumerate(bud[0]):
        for k in range(N, r["n_steps"]):
            xin = r["history"][k][0]
            assert xin[0, i].tobytes() == r["released"][0, i].tobytes()
        assert r["x"][0, i].tobytes() == r["released"][0, i].tobytes()


@pytest.mark.parametrize("alpha,beta", [(0.0, 0.7), (0.35, -0.2), (-1.3, 0.5)])
def test_linear_velocity_field_closed_form(alpha, beta):
    """v = alpha x + beta: after N_i steps of dt_i = -1/N_i the state has a closed form."""
    x0 = np.random.default_rng(12).standard_normal((2, 6, 3)).astype(np.float32)
    bud = np.array([[1, 2, 3, 5, 7, 10], [10, 9, 4, 4, 2, 1]])
    fn = lambda x, t: (np.float32(alpha) * x + np.float32(beta)).astype(np.float32)
    r = O.denoise_schedule(None, x0, bud, velocity_fn=fn)
    N = bud.astype(np.float64)[..., None]
    dt = -1.0 / N
    g = (1.0 + alpha * dt) ** N
    ref = g * x0 + (beta * (g - 1.0) / alpha if alpha != 0 else beta * N * dt)
    np.testing.assert_allclose(r["released"], ref, rtol=2e-6, atol=2e-6)
    np.testing.assert_allclose(r["x"], ref, rtol=2e-6, atol=2e-6)


# ----------------------------------------------------------------------------
# Trajectory Reconciliation / GAC / latency model
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("Nstar,U", [(2, 2), (3, 3), (7, 5)])
def test_tr_exact_recovery_at_k1(Nstar, U):
    """K = 1: ghosts and tail follow the vanilla trajectory bit-for-bit (Sec. 4.3)."""
    m, *_ = tiny_model(dtype=np.float32, B=1)
    H = 10
    x0 = np.random.default_rng(13).standard_normal((1, H, 3)).astype(np.float32)
    r = O.uad_tr_gac(m, x0, U=U, K=1, Nstar=Nstar, S=H)
    van = O.vanilla_denoise(m, x0, Nstar)
    assert r["final"].tobytes() == van.tobytes()
    assert r["ghosts"].tobytes() == van[:, :U].tobytes()
    # plain UAER (no reconciliation) does perturb the tail
    r0 = O.uad_tr_gac(m, x0, U=U, K=1, Nstar=Nstar, S=H, reconcile=False)
    assert np.max(np.abs(r0["final"][:, U:] - van[:, U:])) > 1e-6


def test_tr_reduces_tail_error_for_k_gt_1():
    m, *_ = tiny_model(dtype=np.float64, B=1)
    x0 = np.random.default_rng(14).standard_normal((1, 10, 3))
    van = O.vanilla_denoise(m, x0, 6)
    tr = O.uad_tr_gac(m, x0, U=4, K=2, Nstar=6, S=10)
    naive = O.uad_tr_gac(m, x0, U=4, K=2, Nstar=6, S=10, reconcile=False)
    e_tr = np.linalg.norm(tr["final"][:, 4:] - van[:, 4:])
    e_naive = np.linalg.norm(naive["final"][:, 4:] - van[:, 4:])
    assert e_tr < e_naive


@pytest.mark.parametrize("K,Nstar,U", [(2, 6, 4), (3, 7, 5), (2, 3, 1)])
def test_early_release_equals_per_token_schedule(K, Nstar, U):
    """Sec. 4.2 Eq. 5: the urgent actions released after K steps of 1/K are
    those of the per-token schedule with budgets K (urgent) and N* (tail),
    built by the separately pinned table builder, bit for bit; without
    reconciliation (plain UAER) the whole final state is that schedule's."""
    m, *_ = tiny_model(dtype=np.float32, B=2)
    H = 8
    x0 = np.random.default_rng(31).standard_normal((2, H, 3)).astype(np.float32)
    bud = np.full((2, H), Nstar)
    bud[:, :U] = K
    sch = O.denoise_schedule(m, x0, bud)
    for reconcile in (True, False):
        r = O.uad_tr_gac(m, x0, U=U, K=K, Nstar=Nstar, S=H, reconcile=reconcile)
        assert r["released_urgent"].tobytes() == sch["released"][:, :U].tobytes()
    r0 = O.uad_tr_gac(m, x0, U=U, K=K, Nstar=Nstar, S=H, reconcile=False)
    assert r0["final"].tobytes() == sch["x"].tobytes()
    assert r0["ghosts"] is None


def _linear_flow(x, alpha, beta, dt, n):
    """n Euler steps of size dt under v = alpha x + beta, closed form (float64)."""
    g = (1.0 + alpha * dt) ** n
    return g * x + (beta * (g - 1.0) / alpha if alpha != 0 else beta * n * dt)


@pytest.mark.parametrize("K,Nstar", [(2, 5), (3, 7)])
@pytest.mark.parametrize("alpha,beta", [(0.0, 0.6), (0.4, -0.3), (-1.1, 0.5)])
def test_tr_linear_field_closed_form(K, Nstar, alpha, beta):
    """Sec. 4.2 Eq. 5, Sec. 4.3 Eqs. 6-7, Sec. 4.4 Eqs. 8-9 under v = alpha x + beta.

    Urgent tokens take K steps of dt_u = -1/K: a = g^K x_0 + beta (g^K - 1)/alpha
    with g = 1 + alpha dt_u.  Their velocities are v_k = g^(k-1) (alpha x_0 + beta),
    so TR gives x'_K = x_0 + dt* (alpha x_0 + beta) sum_{j<K} g^j, dt* = -1/N*;
    the ghosts then take N* - K steps of dt*, the tail N* steps of dt*, and
    GAC adds E / (S - U) with E = sum_i (ghost_i - a_i)."""
    B, H, U, Da = 2, 9, 4, 3
    x0 = np.random.default_rng(32).standard_normal((B, H, Da)).astype(np.float32)
    fn = lambda x, t: (np.float32(alpha) * x + np.float32(beta)).astype(np.float32)
    r = O.uad_tr_gac(None, x0, U=U, K=K, Nstar=Nstar, S=H, velocity_fn=fn)
    x = x0.astype(np.float64)
    du, ds = -1.0 / K, -1.0 / Nstar
    a_ref = _linear_flow(x[:, :U], alpha, beta, du, K)
    g = 1.0 + alpha * du
    vsum = (alpha * x[:, :U] + beta) * sum(g ** j for j in range(K))
    ghosts = _linear_flow(x[:, :U] + ds * vsum, alpha, beta, ds, Nstar - K)
    tail = _linear_flow(x[:, U:], alpha, beta, ds, Nstar)
    tol = dict(rtol=4e-6, atol=4e-6)
    np.testing.assert_allclose(r["released_urgent"], a_ref, **tol)
    np.testing.assert_allclose(r["ghosts"], ghosts, **tol)
    np.testing.assert_allclose(r["final"][:, :U], ghosts, **tol)
    np.testing.assert_allclose(r["final"][:, U:], tail, **tol)
    E = np.sum(ghosts - a_ref, axis=1)
    np.testing.assert_allclose(r["E"], E, rtol=2e-5, atol=2e-5)
    np.testing.assert_allclose(r["executed"][:, :U], a_ref, **tol)
    np.testing.assert_allclose(r["executed"][:, U:], tail + E[:, None, :] / (H - U), rtol=2e-5, atol=2e-5)


def test_gac_closed_form():
    rng = np.random.default_rng(15)
    B, U, S, Da = 2, 3, 10, 4
    rel = rng.standard_normal((B, U, Da))
    gh = rng.standard_normal((B, U, Da))
    tail = rng.standard_normal((B, S - U, Da))
    E, cor = O.gac_correct(rel, gh, tail)
    # the executed tail absorbs exactly E in total
    np.testing.assert_allclose(np.sum(cor - tail, axis=1), E, atol=1e-13)
    np.testing.assert_allclose(E, np.sum(gh, 1) - np.sum(rel, 1), atol=1e-13)
    # masked dimension (e.g. gripper) is untouched
    dm = np.array([1, 1, 1, 0])
    _, cor2 = O.gac_correct(rel, gh, tail, dm)
    np.testing.assert_array_equal(cor2[..., 3], tail[..., 3])


def test_aal_controller_reproduces_latency_model():
    rng = np.random.default_rng(16)
    for _ in range(200):
        S = 10
        U = int(rng.integers(1, S))
        Nstar = int(rng.integers(2, 11))
        K = int(rng.integers(1, Nstar))
        T_D, T_act, T_vlm = rng.uniform(1, 30), rng.uniform(1, 60), rng.uniform(0, 50)
        rel = [T_vlm + K * T_D] * U + [T_vlm + Nstar * T_D] * (S - U)
        assert abs(O.aal_controller(rel, T_act) - O.latency_uaer(T_vlm, T_D, Nstar, K, U, T_act, S)) < 1e-9
        van = [T_vlm + Nstar * T_D] * S
        assert abs(O.aal_controller(van, T_act) - O.latency_vanilla(T_vlm, T_D, Nstar, S)) < 1e-9


# ----------------------------------------------------------------------------
# Adaptive-norm time conditioning (App. C.1, reading 9)
# ----------------------------------------------------------------------------
TINY_ADA = W.ModelShape(n_layers=2, d_model=8, n_heads=2, n_kv_heads=1, head_dim=4, d_ff=12, action_dim=3,
                        conditioning="adarms")


def test_adarms_forward_matches_scalar_bruteforce():
    for shape, seed in ((TINY_ADA, 21), (W.ModelShape(1, 12, 3, 3, 2, 5, 2, conditioning="adarms"), 22)):
        m, weights, pk, pv = tiny_model(shape, P=3, seed=seed)
        x = np.random.default_rng(seed).standard_normal((3, shape.action_dim))
        t = np.array([1.0, 0.4, 0.0])
        ref = bruteforce.forward_env_adarms({k: v.tolist() for k, v in weights.items()}, shape,
                                            pk[0].tolist(), pv[0].tolist(), x.tolist(), t.tolist())
        np.testing.assert_allclose(O.action_expert(m, 0, x, t), np.array(ref), rtol=0, atol=1e-11)


def test_ada_rms_norm_special_cases():
    rng = np.random.default_rng(3)
    h = rng.standard_normal((4, 8))
    z = np.zeros_like(h)
    # no modulation = RMSNorm with unit gain; scale s = RMSNorm with gain 1 + s (per token)
    np.testing.assert_allclose(O.ada_rms_norm(h, z, z, 1e-6), O.rms_norm(h, np.ones(8), 1e-6), atol=1e-15)
    s = rng.standard_normal(8)
    np.testing.assert_allclose(O.ada_rms_norm(h, np.broadcast_to(s, h.shape), z, 1e-6),
                               O.rms_norm(h, 1 + s, 1e-6), atol=1e-14)
    # constant vector c*1 normalises to sign(c) (up to eps), then (1 + a) * sign(c) + b
    c = np.full((1, 8), -2.5)
    a, b = rng.standard_normal((1, 8)), rng.standard_normal((1, 8))
    np.testing.assert_allclose(O.ada_rms_norm(c, a, b, 0.0), -(1 + a) + b, atol=1e-14)
    # torch's functional rms_norm as a library reference for the normalisation
    ref = torch.nn.functional.rms_norm(torch.from_numpy(h), (8,), eps=1e-6).numpy() * (1 + a) + b
    np.testing.assert_allclose(O.ada_rms_norm(h, np.broadcast_to(a, h.shape), np.broadcast_to(b, h.shape), 1e-6),
                               ref, atol=1e-14)


def test_adarms_time_enters_only_through_modulation():
    """With every modulation matrix zero, v no longer depends on t; with them, it does."""
    m, *_ = tiny_model(TINY_ADA, seed=23)
    x = np.random.default_rng(4).standard_normal((2, 3))
    t1, t2 = np.array([0.9, 0.1]), np.array([0.3, 0.6])
    assert not np.allclose(O.action_expert(m, 0, x, t1), O.action_expert(m, 0, x, t2))
    for k in list(m.weights):
        if k.endswith("_mod.w"):
            m.weights[k] = np.zeros_like(m.weights[k])
    np.testing.assert_array_equal(O.action_expert(m, 0, x, t1), O.action_expert(m, 0, x, t2))


def test_adarms_zero_gates_closed_form():
    """gamma = 0 on every branch: the layers do nothing and
    v = (RMS(h_0) (1 + a_f) + b_f) W_out^T + b_out with h_0 = W_in x + b_in."""
    m, *_ = tiny_model(TINY_ADA, seed=24)
    d = TINY_ADA.d_model
    for l in range(TINY_ADA.n_layers):
        for s in ("attn_mod", "mlp_mod"):
            m.weights[f"layers.{l}.{s}.w"][2 * d:] = 0
            m.weights[f"layers.{l}.{s}.b"][2 * d:] = 0
    x = np.random.default_rng(5).standard_normal((2, 3))
    t = np.array([0.8, 0.2])
    Wt = m.weights
    e = O.time_embedding(t, d)
    c = O.silu(O.silu(e @ Wt["time_mlp_in.w"].T + Wt["time_mlp_in.b"]) @ Wt["time_mlp_out.w"].T + Wt["time_mlp_out.b"])
    h0 = x @ Wt["action_in.w"].T + Wt["action_in.b"]
    mf = c @ Wt["final_mod.w"].T + Wt["final_mod.b"]
    r = h0 / np.sqrt((h0 ** 2).mean(-1, keepdims=True) + 1e-6)
    ref = (r * (1 + mf[:, :d]) + mf[:, d:]) @ Wt["action_out.w"].T + Wt["action_out.b"]
    np.testing.assert_allclose(O.action_expert(m, 0, x, t), ref, atol=1e-12)
