"""Scalar, loop-by-loop float64 reference of one joint action-expert evaluation.

Used only to pin the oracle on tiny shapes.  Written independently of the
oracle: plain Python lists and the ``math`` module, no numpy array algebra,
every sum spelled out as a loop over the definition.
"""
import math


def _matvec(W, x):
    # W: list of rows [out][in]; y_o = sum_i W[o][i] x_i
    return [sum(W[o][i] * x[i] for i in range(len(x))) for o in range(len(W))]


def _rms(h, g, eps):
    ms = sum(v * v for v in h) / len(h)
    r = 1.0 / math.sqrt(ms + eps)
    return [h[i] * r * g[i] for i in range(len(h))]


def _gelu(z):
    return 0.5 * z * (1.0 + math.tanh(math.sqrt(2.0 / math.pi) * (z + 0.044715 * z ** 3)))


def _silu(z):
    return z / (1.0 + math.exp(-z))


def _temb(t, d):
    half = d // 2
    freqs = [1000.0 * 10000.0 ** (-j / half) for j in range(half)]
    return [math.sin(f * t) for f in freqs] + [math.cos(f * t) for f in freqs]


def forward_env(W, shape, pk, pv, x, t):
    """W: dict name -> nested lists; pk/pv: [L][P][Hkv][hd]; x: [H][Da]; t: [H]."""
    L, d, Hq, Hkv, hd = shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim
    eps = shape.rms_eps
    H = len(x)
    hs = []
    for i in range(H):
        a = [v + b for v, b in zip(_matvec(W["action_in.w"], x[i]), W["action_in.b"])]
        u = a + _temb(t[i], d)
        z = [_silu(v + b) for v, b in zip(_matvec(W["time_mlp_in.w"], u), W["time_mlp_in.b"])]
        hs.append([v + b for v, b in zip(_matvec(W["time_mlp_out.w"], z), W["time_mlp_out.b"])])
    for l in range(L):
        p = f"layers.{l}."
        ns = [_rms(hs[i], W[p + "attn_norm"], eps) for i in range(H)]
        qs = [_matvec(W[p + "wq"], n) for n in ns]
        ks = [_matvec(W[p + "wk"], n) for n in ns]
        vs = [_matvec(W[p + "wv"], n) for n in ns]
        P = len(pk[l])
        new_h = []
        for i in range(H):
            o = []
            for j in range(Hq):
                g = (j * Hkv) // Hq
                keys = [pk[l][s][g] for s in range(P)] + [ks[s][g * hd:(g + 1) * hd] for s in range(H)]
                vals = [pv[l][s][g] for s in range(P)] + [vs[s][g * hd:(g + 1) * hd] for s in range(H)]
                qj = qs[i][j * hd:(j + 1) * hd]
                sc = [sum(qj[c] * kk[c] for c in range(hd)) / math.sqrt(hd) for kk in keys]
                mx = max(sc)
                ex = [math.exp(s - mx) for s in sc]
                den = sum(ex)
                for c in range(hd):
                    o.append(sum(ex[s] * vals[s][c] for s in range(len(keys))) / den)
            ao = _matvec(W[p + "wo"], o)
            new_h.append([hs[i][c] + ao[c] for c in range(d)])
        hs = new_h
        for i in range(H):
            n2 = _rms(hs[i], W[p + "mlp_norm"], eps)
            gate = _matvec(W[p + "w_gate"], n2)
            up = _matvec(W[p + "w_up"], n2)
            gg = [_gelu(gate[c]) * up[c] for c in range(len(gate))]
            dn = _matvec(W[p + "w_down"], gg)
            hs[i] = [hs[i][c] + dn[c] for c in range(d)]
    out = []
    for i in range(H):
        nf = _rms(hs[i], W["final_norm"], eps)
        out.append([v + b for v, b in zip(_matvec(W["action_out.w"], nf), W["action_out.b"])])
    return out


def _adarms(h, scale, shift, eps):
    # h / rms(h) * (1 + scale_c) + shift_c, every term spelled out
    ms = sum(v * v for v in h) / len(h)
    r = 1.0 / math.sqrt(ms + eps)
    return [h[c] * r * (1.0 + scale[c]) + shift[c] for c in range(len(h))]


def forward_env_adarms(W, shape, pk, pv, x, t):
    """The adaptive-norm-conditioned expert, token by token (same arguments as forward_env)."""
    L, d, Hq, Hkv, hd = shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim
    eps = shape.rms_eps
    H = len(x)
    cs, hs = [], []
    for i in range(H):
        e = _temb(t[i], d)
        z = [_silu(v + b) for v, b in zip(_matvec(W["time_mlp_in.w"], e), W["time_mlp_in.b"])]
        cs.append([_silu(v + b) for v, b in zip(_matvec(W["time_mlp_out.w"], z), W["time_mlp_out.b"])])
        hs.append([v + b for v, b in zip(_matvec(W["action_in.w"], x[i]), W["action_in.b"])])

    def mod(name, i):
        return [v + b for v, b in zip(_matvec(W[name + ".w"], cs[i]), W[name + ".b"])]

    for l in range(L):
        p = f"layers.{l}."
        ns = []
        gates = []
        for i in range(H):
            m = mod(p + "attn_mod", i)
            ns.append(_adarms(hs[i], m[:d], m[d:2 * d], eps))
            gates.append(m[2 * d:])
        qs = [_matvec(W[p + "wq"], n) for n in ns]
        ks = [_matvec(W[p + "wk"], n) for n in ns]
        vs = [_matvec(W[p + "wv"], n) for n in ns]
        P = len(pk[l])
        new_h = []
        for i in range(H):
            o = []
            for j in range(Hq):
                g = (j * Hkv) // Hq
                keys = [pk[l][s][g] for s in range(P)] + [ks[s][g * hd:(g + 1) * hd] for s in range(H)]
                vals = [pv[l][s][g] for s in range(P)] + [vs[s][g * hd:(g + 1) * hd] for s in range(H)]
                qj = qs[i][j * hd:(j + 1) * hd]
                sc = [sum(qj[c] * kk[c] for c in range(hd)) / math.sqrt(hd) for kk in keys]
                mx = max(sc)
                ex = [math.exp(s - mx) for s in sc]
                den = sum(ex)
                for c in range(hd):
                    o.append(sum(ex[s] * vals[s][c] for s in range(len(keys))) / den)
            ao = _matvec(W[p + "wo"], o)
            new_h.append([hs[i][c] + gates[i][c] * ao[c] for c in range(d)])
        hs = new_h
        for i in range(H):
            m = mod(p + "mlp_mod", i)
            n2 = _adarms(hs[i], m[:d], m[d:2 * d], eps)
            gate = _matvec(W[p + "w_gate"], n2)
            up = _matvec(W[p + "w_up"], n2)
            gg = [_gelu(gate[c]) * up[c] for c in range(len(gate))]
            dn = _matvec(W[p + "w_down"], gg)
            hs[i] = [hs[i][c] + m[2 * d + c] * dn[c] for c in range(d)]
    out = []
    for i in range(H):
        m = mod("final_mod", i)
        nf = _adarms(hs[i], m[:d], m[d:], eps)
        out.append([v + b for v, b in zip(_matvec(W["action_out.w"], nf), W["action_out.b"])])
    return out
