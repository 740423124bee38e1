"""Plain, slow, obviously-correct CPU oracle of Urgency-Aware Denoising (UAD).

TEST INFRASTRUCTURE ONLY: used by ``tests/``, the smoke check and the CPU
baseline of the benchmark; never by the product path.  It shares no code with
the HIP library and does not import it.  Inputs come from ``uad_workloads``
(seeded draws only).

What it computes, in the paper's order and notation:

* The flow-matching velocity ``v_k <- F_theta(x_{k-1}, o, L)`` of the action
  expert over the whole chunk in ONE joint evaluation (Sec. 3, Eq. 1), with a
  separate flow time per action token (App. C.1, "Per-Action Time
  Conditioning").  The context (o, L) is represented by the cached prefix K/V of
  each layer; the expert's architecture is not given by the paper, so the
  readings listed below fix it.
* The uniform Euler update (Sec. 3, Eq. 2) and the urgency-aware per-token
  update with budgets N_i (Sec. 4.2, Eqs. 3-5), releasing a^i = x^i after its
  last step.
* Trajectory Reconciliation (Sec. 4.3, Eqs. 6-7), ghost actions (Sec. 4.3) and
  Ghost Action Correction on additive dimensions (Sec. 4.4, Eqs. 8-9).
* The latency model of App. B (Eqs. latency_vanilla / latency_uaer) and an
  availability-latency controller that replays release times against the
  per-action execution budget T_act (App. C.3).

Readings where the paper is silent (each is also listed in the design notes):

1. Time runs from t=1 (noise) to t=0; the per-token step is dt_i = -(1/N_i),
   x <- x + dt*v.  This is the paper's x_k = x_{k-1} + v_k/N_i with the
   velocity sign flipped; the integrator is sign-agnostic since t and dt are
   inputs.
2. t_i at step k (0-based) is (N_i - min(k, N_i)) / N_i, divided in fp32 from
   integers, not accumulated.
3. Time embedding: e_j = sin(w_j t), e_{j+d/2} = cos(w_j t) with
   w_j = 1000 * 10000^(-j/(d/2)); the action token is conditioned before the
   action MLP: h = W2 SiLU(W1 [W_in x + b_in ; e(t)] + b1) + b2.
4. Released tokens stay in the sequence (x frozen, t = 0) and keep serving as
   keys/values for the other tokens.
5. Every chunk token attends to all P prefix tokens and all H chunk tokens
   (no mask, no positional encoding), softmax scale 1/sqrt(head_dim);
   query head j reads KV head floor(j * Hkv / Hq).
6. Pre-norm residual blocks with RMSNorm (eps 1e-6, learned gain), bias-free
   projections, GeGLU MLP with the tanh form of GELU.
7. A frozen token (mask = 1, or dt = 0) is copied, never updated with
   x + 0*v, so it stays bit-identical whatever v holds.
8. Ghost tokens after reconciliation run at t = (N* - k)/N*, dt = -(1/N*),
   and the reconciliation sum accumulates the cached velocities in step order.
9. Adaptive-norm conditioning (the pi0.5-style expert, App. C.1; the paper
   names the mechanism but gives no formula): c = SiLU(W_t2 SiLU(W_t1 e(t) +
   b_t1) + b_t2) per token; the action token is h_0 = W_in x + b_in; every
   norm site s (attention and MLP of each layer) takes (alpha, beta, gamma) =
   W_s c + b_s and computes n = RMS(h) * (1 + alpha) + beta (no separate
   gain), the branch output enters the residual as h += gamma * branch; the
   final norm takes (alpha_f, beta_f) = W_f c + b_f.

Precision: fp32 throughout (the numpy matmuls are BLAS sgemm), or float64 when
a model is built with ``dtype=np.float64``.  The time-embedding arguments are
formed in the working precision and sin/cos are evaluated in float64.
"""
from __future__ import annotations

import dataclasses
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "Model", "build_model", "rms_norm", "ada_rms_norm", "silu", "gelu_tanh", "time_embedding",
    "time_frequencies", "attention", "action_expert", "velocity", "euler_update",
    "build_schedule", "denoise_step", "denoise_schedule", "vanilla_denoise",
    "release_steps", "uad_tr_gac", "gac_correct", "aal_controller",
    "latency_vanilla", "latency_uaer",
]


# ----------------------------------------------------------------------------
# Model container
# ----------------------------------------------------------------------------
@dataclasses.dataclass
class Model:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    action_dim: int
    rms_eps: float
    weights: Dict[str, np.ndarray]
    prefix_k: List[np.ndarray]   # per env: [L][P][Hkv][hd]
    prefix_v: List[np.ndarray]
    dtype: type = np.float32
    conditioning: str = "input"  # "input" (reading 3) or "adarms" (reading 9)


def build_model(shape, weights: Dict[str, np.ndarray], prefix_k: Sequence[np.ndarray],
                prefix_v: Sequence[np.ndarray], dtype=np.float32) -> Model:
    dt = np.dtype(dtype).type
    return Model(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads,
                 shape.head_dim, shape.d_ff, shape.action_dim, shape.rms_eps,
                 {k: np.asarray(v, dt) for k, v in weights.items()},
                 [np.asarray(k, dt) for k in prefix_k], [np.asarray(v, dt) for v in prefix_v], dt,
                 getattr(shape, "conditioning", "input"))


# ----------------------------------------------------------------------------
# Elementwise pieces (reading 6 / reading 3)
# ----------------------------------------------------------------------------
def rms_norm(h: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm over the last axis: h / sqrt(mean(h^2) + eps) * gain."""
    ms = np.mean(h * h, axis=-1, keepdims=True)
    return h / np.sqrt(ms + h.dtype.type(eps)) * gain


def ada_rms_norm(h: np.ndarray, scale: np.ndarray, shift: np.ndarray, eps: float) -> np.ndarray:
    """Adaptive RMSNorm (reading 9): h / sqrt(mean(h^2) + eps) * (1 + scale) + shift."""
    r = h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + h.dtype.type(eps))
    return r * (h.dtype.type(1) + scale) + shift


def silu(z: np.ndarray) -> np.ndarray:
    return z / (z.dtype.type(1) + np.exp(-z))


def gelu_tanh(z: np.ndarray) -> np.ndarray:
    """GELU, tanh form: z/2 * (1 + tanh(sqrt(2/pi) * (z + 0.044715 z^3)))."""
    c = z.dtype.type(np.sqrt(2.0 / np.pi))
    a = z.dtype.type(0.044715)
    half = z.dtype.type(0.5)
    return half * z * (z.dtype.type(1) + np.tanh(c * (z + a * z * z * z)))


def time_frequencies(d: int, dtype=np.float32) -> np.ndarray:
    """w_j = 1000 * 10000^(-j/(d/2)), j < d/2 (reading 3), rounded to dtype."""
    j = np.arange(d // 2, dtype=np.float64)
    return (1000.0 * np.power(10000.0, -j / (d // 2))).astype(dtype)


def time_embedding(t: np.ndarray, d: int) -> np.ndarray:
    """Per-token sinusoidal embedding [.., d]: first half sin(w t), second half cos(w t)."""
    dt = t.dtype.type
    w = time_frequencies(d, dt)
    arg = (t[..., None] * w).astype(dt)           # argument in working precision
    a64 = arg.astype(np.float64)
    return np.concatenate([np.sin(a64), np.cos(a64)], axis=-1).astype(dt)


# ----------------------------------------------------------------------------
# Attention (reading 5): joint attention of chunk queries over [prefix ; chunk]
# ----------------------------------------------------------------------------
def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """q [T, Hq, hd], k/v [S, Hkv, hd] -> o [T, Hq, hd]; max-subtracted softmax."""
    T, Hq, hd = q.shape
    Hkv = k.shape[1]
    one = q.dtype.type(1)
    scale = one / np.sqrt(q.dtype.type(hd))
    o = np.empty_like(q)
    for j in range(Hq):
        g = (j * Hkv) // Hq
        s = (q[:, j, :] @ k[:, g, :].T) * scale
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        o[:, j, :] = p @ v[:, g, :]
    return o


# ----------------------------------------------------------------------------
# The action expert F_theta (Sec. 3 Eq. 1; App. C.1)
# ----------------------------------------------------------------------------
def action_expert(m: Model, env: int, x: np.ndarray, t: np.ndarray) -> np.ndarray:
    """One joint evaluation over the chunk of one environment.

    x [H, Da] noisy actions, t [H] per-token flow time -> velocity [H, Da].
    """
    if m.conditioning == "adarms":
        return _action_expert_adarms(m, env, x, t)
    W, dt = m.weights, m.dtype
    x = np.asarray(x, dt)
    t = np.asarray(t, dt)
    H = x.shape[0]
    # per-token time conditioning before the action MLP (App. C.1, reading 3)
    a = x @ W["action_in.w"].T + W["action_in.b"]
    e = time_embedding(t, m.d_model)
    u = np.concatenate([a, e], axis=-1)
    z = silu(u @ W["time_mlp_in.w"].T + W["time_mlp_in.b"])
    h = z @ W["time_mlp_out.w"].T + W["time_mlp_out.b"]
    for l in range(m.n_layers):
        p = f"layers.{l}."
        n = rms_norm(h, W[p + "attn_norm"], m.rms_eps)
        q = (n @ W[p + "wq"].T).reshape(H, m.n_heads, m.head_dim)
        k = (n @ W[p + "wk"].T).reshape(H, m.n_kv_heads, m.head_dim)
        v = (n @ W[p + "wv"].T).reshape(H, m.n_kv_heads, m.head_dim)
        k_all = np.concatenate([m.prefix_k[env][l], k], axis=0)
        v_all = np.concatenate([m.prefix_v[env][l], v], axis=0)
        o = attention(q, k_all, v_all).reshape(H, m.n_heads * m.head_dim)
        h = h + o @ W[p + "wo"].T
        n2 = rms_norm(h, W[p + "mlp_norm"], m.rms_eps)
        g = gelu_tanh(n2 @ W[p + "w_gate"].T) * (n2 @ W[p + "w_up"].T)
        h = h + g @ W[p + "w_down"].T
    nf = rms_norm(h, W["final_norm"], m.rms_eps)
    return nf @ W["action_out.w"].T + W["action_out.b"]


def _action_expert_adarms(m: Model, env: int, x: np.ndarray, t: np.ndarray) -> np.ndarray:
    """The expert with adaptive-norm time conditioning (App. C.1, reading 9)."""
    W, dt = m.weights, m.dtype
    x = np.asarray(x, dt)
    t = np.asarray(t, dt)
    H, d = x.shape[0], m.d_model
    e = time_embedding(t, d)
    c = silu(silu(e @ W["time_mlp_in.w"].T + W["time_mlp_in.b"]) @ W["time_mlp_out.w"].T + W["time_mlp_out.b"])
    h = x @ W["action_in.w"].T + W["action_in.b"]
    for l in range(m.n_layers):
        p = f"layers.{l}."
        ma = c @ W[p + "attn_mod.w"].T + W[p + "attn_mod.b"]
        al, be, ga = ma[:, :d], ma[:, d:2 * d], ma[:, 2 * d:]
        n = ada_rms_norm(h, al, be, m.rms_eps)
        q = (n @ W[p + "wq"].T).reshape(H, m.n_heads, m.head_dim)
        k = (n @ W[p + "wk"].T).reshape(H, m.n_kv_heads, m.head_dim)
        v = (n @ W[p + "wv"].T).reshape(H, m.n_kv_heads, m.head_dim)
        k_all = np.concatenate([m.prefix_k[env][l], k], axis=0)
        v_all = np.concatenate([m.prefix_v[env][l], v], axis=0)
        o = attention(q, k_all, v_all).reshape(H, m.n_heads * m.head_dim)
        h = h + ga * (o @ W[p + "wo"].T)
        mm = c @ W[p + "mlp_mod.w"].T + W[p + "mlp_mod.b"]
        al, be, ga = mm[:, :d], mm[:, d:2 * d], mm[:, 2 * d:]
        n2 = ada_rms_norm(h, al, be, m.rms_eps)
        g = gelu_tanh(n2 @ W[p + "w_gate"].T) * (n2 @ W[p + "w_up"].T)
        h = h + ga * (g @ W[p + "w_down"].T)
    mf = c @ W["final_mod.w"].T + W["final_mod.b"]
    nf = ada_rms_norm(h, mf[:, :d], mf[:, d:], m.rms_eps)
    return nf @ W["action_out.w"].T + W["action_out.b"]


VelocityFn = Callable[[np.ndarray, np.ndarray], np.ndarray]


def velocity(m: Model, x: np.ndarray, t: np.ndarray) -> np.ndarray:
    """Batched F_theta: x [B, H, Da], t [B, H] -> v [B, H, Da]; envs are independent."""
    return np.stack([action_expert(m, b, x[b], t[b]) for b in range(x.shape[0])])


# ----------------------------------------------------------------------------
# Integrator and schedule (Sec. 3 Eq. 2; Sec. 4.2 Eqs. 4-5)
# ----------------------------------------------------------------------------
def euler_update(x: np.ndarray, v: np.ndarray, dt: np.ndarray, mask: np.ndarray) -> np.ndarray:
    """Per-token Euler step x_i <- x_i + dt_i v_i; frozen tokens are copied (reading 7)."""
    frozen = (np.asarray(mask) != 0) | (dt == 0)
    with np.errstate(invalid="ignore", over="ignore"):
        upd = x + dt[..., None] * v
    return np.where(frozen[..., None], x, upd)


def build_schedule(budgets: np.ndarray) -> Tuple[int, np.ndarray, np.ndarray, np.ndarray]:
    """Per-step tables from integer budgets N_i (Eq. 4): (n_steps, t, dt, mask).

    t[k] = (N - min(k, N)) / N, dt[k] = -(1/N) while k < N else 0,
    mask[k] = 1 once k >= N (token released and frozen).  Shapes [n_steps][B][H].
    """
    N = np.asarray(budgets, np.int64)
    if N.size == 0 or N.min() < 1:
        raise ValueError("budgets must be >= 1")
    n_steps = int(N.max())
    Nf = N.astype(np.float32)
    t = np.empty((n_steps,) + N.shape, np.float32)
    dt = np.empty_like(t)
    mask = np.empty((n_steps,) + N.shape, np.uint8)
    for k in range(n_steps):
        t[k] = (N - np.minimum(k, N)).astype(np.float32) / Nf
        dt[k] = np.where(k < N, -(np.float32(1) / Nf), np.float32(0))
        mask[k] = (k >= N).astype(np.uint8)
    return n_steps, t, dt, mask


def release_steps(budgets: np.ndarray) -> np.ndarray:
    """0-based step after which token i is released: N_i - 1 (Eq. 5 text)."""
    return np.asarray(budgets, np.int32) - 1


def denoise_step(m: Model, x, t, dt, mask, velocity_fn: Optional[VelocityFn] = None):
    """One joint F_theta evaluation over all tokens (frozen ones included) + masked Euler."""
    v = velocity(m, x, t) if velocity_fn is None else velocity_fn(x, t)
    return euler_update(x, v, dt, mask), v


def denoise_schedule(m: Optional[Model], x0: np.ndarray, budgets: np.ndarray,
                     velocity_fn: Optional[VelocityFn] = None, keep_history: bool = False):
    """UAER with per-token budgets N_i (Sec. 4.2).

    Returns a dict with the final state, the released actions a^i = x^i after
    token i's last step, the release step of each token and, optionally, the
    per-step inputs and velocities (for teacher-forced comparisons).
    """
    n_steps, t, dt, mask = build_schedule(budgets)
    x = np.array(x0, dtype=(m.dtype if m is not None else np.float32))
    rel = release_steps(budgets)
    released = np.zeros_like(x)
    hist = []
    for k in range(n_steps):
        x_in = x
        x, v = denoise_step(m, x, t[k], dt[k], mask[k], velocity_fn)
        if keep_history:
            hist.append((x_in, v))
        now = rel == k
        released[now] = x[now]
    out = {"x": x, "released": released, "release_step": rel, "n_steps": n_steps,
           "t": t, "dt": dt, "mask": mask}
    if keep_history:
        out["history"] = hist
    return out


def vanilla_denoise(m: Optional[Model], x0: np.ndarray, N: int,
                    velocity_fn: Optional[VelocityFn] = None) -> np.ndarray:
    """Uniform Euler over N steps with one scalar flow time shared by all tokens (Eq. 2)."""
    x = np.array(x0, dtype=(m.dtype if m is not None else np.float32))
    B, H = x.shape[:2]
    for k in range(N):
        tk = np.float32(N - k) / np.float32(N)
        dtk = -(np.float32(1) / np.float32(N))
        tvec = np.full((B, H), tk, np.float32)
        v = velocity(m, x, tvec) if velocity_fn is None else velocity_fn(x, tvec)
        x = x + dtk * v
    return x


# ----------------------------------------------------------------------------
# Trajectory Reconciliation and Ghost Action Correction (Sec. 4.3, 4.4)
# ----------------------------------------------------------------------------
def uad_tr_gac(m: Optional[Model], x0: np.ndarray, U: int, K: int, Nstar: int, S: int,
               velocity_fn: Optional[VelocityFn] = None, reconcile: bool = True):
    """UAER + TR (+ ghosts) on a chunk, with GAC applied to the executed tail.

    Steps 1..K: urgent tokens (i < U) use budget K, tail tokens budget N*.
    After step K the urgent a^i = x_K^i are released; with ``reconcile`` their
    internal states are replaced by x'_K = x_0 + dt* * sum_{k<=K} v_k
    (dt* = -(1/N*), Eq. 6) and continue as ghosts with the tail's time and
    step for k > K (Eq. 7).  Without ``reconcile`` (plain UAER) the released
    tokens stay frozen.  Returns released urgent actions, ghost actions,
    tail states, error vector E (Eq. 8) and GAC-corrected executed actions (Eq. 9).
    """
    if not (1 <= K < Nstar) or not (1 <= U < S):
        raise ValueError("need 1 <= K < N* and 1 <= U < S")
    dtyp = m.dtype if m is not None else np.float32
    x = np.array(x0, dtype=dtyp)
    B, H, Da = x.shape
    one = np.float32(1)
    vf = (lambda xx, tt: velocity(m, xx, tt)) if velocity_fn is None else velocity_fn
    budgets = np.full((B, H), Nstar, np.int64)
    budgets[:, :U] = K
    vsum = None
    for k in range(K):
        t = (budgets - k).astype(np.float32) / budgets.astype(np.float32)
        dt = -(one / budgets.astype(np.float32))
        v = vf(x, t)
        vsum = v[:, :U].copy() if vsum is None else vsum + v[:, :U]
        x = x + dt[..., None] * v
    a_urgent = x[:, :U].copy()
    if reconcile:
        x[:, :U] = x0[:, :U] + (-(one / np.float32(Nstar))) * vsum
    frozen = np.zeros((B, H), bool)
    if not reconcile:
        frozen[:, :U] = True
    for k in range(K, Nstar):
        tk = np.float32(Nstar - k) / np.float32(Nstar)
        t = np.full((B, H), tk, np.float32)
        if not reconcile:
            t[:, :U] = 0
        v = vf(x, t)
        dt = np.full((B, H), -(one / np.float32(Nstar)), np.float32)
        x = euler_update(x, v, dt, frozen.astype(np.uint8))
    ghosts = x[:, :U].copy() if reconcile else None
    out = {"released_urgent": a_urgent, "final": x, "ghosts": ghosts}
    if reconcile:
        E, corrected = gac_correct(a_urgent, ghosts, x[:, U:S])
        out["E"] = E
        out["executed"] = np.concatenate([a_urgent, corrected], axis=1)
    return out


def gac_correct(released: np.ndarray, ghosts: np.ndarray, tail: np.ndarray,
                dim_mask: Optional[np.ndarray] = None):
    """GAC on additive dimensions.

    E = sum_{i<U} (a'^i - a^i)  (Eq. 8);  a^i = x^i_{N*} + E/(S-U), i = U..S-1  (Eq. 9).
    ``tail`` holds x^i_{N*} for i = U..S-1 ([B, S-U, Da]); ``dim_mask`` (Da,)
    selects the dimensions that are corrected (others, e.g. a gripper, untouched).
    """
    E = np.sum(ghosts - released, axis=1)
    n = tail.shape[1]
    shift = E / tail.dtype.type(n)
    if dim_mask is not None:
        shift = np.where(np.asarray(dim_mask, bool)[None, :], shift, 0)
    return E, tail + shift[:, None, :]


# ----------------------------------------------------------------------------
# Availability latency (App. B; App. C.3)
# ----------------------------------------------------------------------------
def latency_vanilla(T_vlm: float, T_D: float, Nstar: int, S: int) -> float:
    """Average action-availability latency of vanilla inference (Eq. latency_vanilla)."""
    return (T_vlm + Nstar * T_D) / S


def latency_uaer(T_vlm: float, T_D: float, Nstar: int, K: int, U: int, T_act: float, S: int) -> float:
    """Average action-availability latency of UAER (Eq. latency_uaer)."""
    return (T_vlm + K * T_D + max((Nstar - K) * T_D - U * T_act, 0.0)) / S


def aal_controller(release_times: Sequence[float], T_act: float) -> float:
    """Replay a controller that executes actions in order, each for T_act.

    Action j can start once it is released (release_times[j], measured from the
    request) and the previous action finished; the wait before each start is
    the exposed latency.  Returns the total wait divided by the number of
    executed actions (AAL, App. C.3).
    """
    clock = 0.0
    wait = 0.0
    for r in release_times:
        if r > clock:
            wait += r - clock
            clock = r
        clock += T_act
    return wait / len(release_times)
