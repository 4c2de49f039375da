"""Scalar-loop evaluation of one action-expert forward, for tiny shapes only.

An independent second reading of the same definitions (Eq. 1, Eq. 2, the
conditioning MLP of Appendix B.3, rotate-half RoPE, gated GELU), written with
plain Python floats and ``math`` so that a vectorisation mistake in the oracle
(a transposed operand, a wrong axis, a wrong split of the packed weights) shows
up as a mismatch.  It shares no code with ``oracle/``.
"""
import math


def _matvec(W, x):
    # W: list of rows (output features), x: list
    return [sum(W[o][i] * x[i] for i in range(len(x))) for o in range(len(W))]


def _rot(vec, p, theta):
    d = len(vec)
    h = d // 2
    out = [0.0] * d
    for i in range(h):
        ang = p * theta ** (-2.0 * i / d)
        c, s = math.cos(ang), math.sin(ang)
        out[i] = vec[i] * c - vec[i + h] * s
        out[i + h] = vec[i + h] * c + vec[i] * s
    return out


def _norm_mod(row, scale, shift, eps):
    ms = sum(v * v for v in row) / len(row)
    r = math.sqrt(ms + eps)
    return [row[i] / r * (1.0 + scale[i]) + shift[i] for i in range(len(row))]


def _tolist(a):
    return a.tolist() if hasattr(a, "tolist") else a


def velocity_loops(cfg, weights, state, x, tau, ctx_k, ctx_v, dyn_pos):
    """v(x, tau) for one env with explicit loops.

    ctx_k / ctx_v: context keys / values already with RoPE on K, lists of
    [Hkv][dh] per context row.  Returns a list of H rows of d_a floats.
    """
    D, L, Fm = cfg.width, cfg.n_layers, cfg.mlp_dim
    Hq, Hkv, dh = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    H = cfg.action_horizon
    T = H + 1
    W = {k: _tolist(v) for k, v in weights.items()}
    state = _tolist(state)
    x = _tolist(x)

    # condition vector: sinusoidal time embedding then the state
    half = D // 2
    temb_s, temb_c = [], []
    for i in range(half):
        frac = i / (half - 1)
        period = cfg.temb_min_period * (cfg.temb_max_period / cfg.temb_min_period) ** frac
        a = 2.0 * math.pi * tau / period
        temb_s.append(math.sin(a))
        temb_c.append(math.cos(a))
    cond = temb_s + temb_c + list(state)

    mods = []
    for s in range(2 * L + 1):
        hid = _matvec(W["w_mod1"][s], cond)
        hid = [v / (1.0 + math.exp(-v)) for v in hid]
        m = _matvec(W["w_mod2"][s], hid)
        sc, sh, g = m[:D], m[D:2 * D], m[2 * D:]
        if cfg.mod_mode == "scale_only":
            sh, g = [0.0] * D, [1.0] * D
        mods.append((sc, sh, g))

    h = [[v * cfg.embed_scale for v in _matvec(W["w_state"], state)]]
    for i in range(H):
        h.append([v * cfg.embed_scale for v in _matvec(W["w_ain"], x[i])])

    for l in range(L):
        n_ctx = len(ctx_k[l])
        sc, sh, g = mods[2 * l]
        qs, ks, vs = [], [], []
        for t in range(T):
            y = _norm_mod(h[t], sc, sh, cfg.rms_eps)
            row = _matvec(W["w_qkv"][l], y)
            q_heads = [_rot(row[j * dh:(j + 1) * dh], dyn_pos[t], cfg.rope_theta) for j in range(Hq)]
            k_heads = [_rot(row[(Hq + j) * dh:(Hq + j + 1) * dh], dyn_pos[t], cfg.rope_theta)
                       for j in range(Hkv)]
            v_heads = [row[(Hq + Hkv + j) * dh:(Hq + Hkv + j + 1) * dh] for j in range(Hkv)]
            qs.append(q_heads)
            ks.append(k_heads)
            vs.append(v_heads)
        keys = [list(r) for r in ctx_k[l]] + ks
        vals = [list(r) for r in ctx_v[l]] + vs
        new_h = []
        for t in range(T):
            o_row = []
            for j in range(Hq):
                kvh = j // (Hq // Hkv)
                # visible keys: all context rows; among dynamic rows the state
                # token sees itself only, action tokens see every dynamic row
                vis = list(range(n_ctx)) + ([n_ctx] if t == 0 else list(range(n_ctx, n_ctx + T)))
                sc_list = []
                for key in vis:
                    dot = 0.0
                    for e in range(dh):
                        dot += qs[t][j][e] * keys[key][kvh][e]
                    sc_list.append(dot / math.sqrt(dh))
                mx = max(sc_list)
                ex = [math.exp(s_ - mx) for s_ in sc_list]
                tot = sum(ex)
                for e in range(dh):
                    acc = 0.0
                    for idx, key in enumerate(vis):
                        acc += ex[idx] / tot * vals[key][kvh][e]
                    o_row.append(acc)
            proj = _matvec(W["w_o"][l], o_row)
            new_h.append([h[t][i] + g[i] * proj[i] for i in range(D)])
        h = new_h
        sc2, sh2, g2 = mods[2 * l + 1]
        new_h = []
        for t in range(T):
            y = _norm_mod(h[t], sc2, sh2, cfg.rms_eps)
            u = _matvec(W["w_gu"][l], y)
            z = []
            for i in range(Fm):
                a = u[i]
                ga = 0.5 * a * (1.0 + math.tanh(math.sqrt(2.0 / math.pi) * (a + 0.044715 * a * a * a)))
                z.append(ga * u[Fm + i])
            down = _matvec(W["w_down"][l], z)
            new_h.append([h[t][i] + g2[i] * down[i] for i in range(D)])
        h = new_h
    scf, shf, _ = mods[2 * L]
    out = []
    for t in range(1, T):
        y = _norm_mod(h[t], scf, shf, cfg.rms_eps)
        out.append(_matvec(W["w_aout"], y))
    return out


def context_loops(cfg, weights, static_k, static_v, frames, window, env, static_pos, frame_pos):
    """Cached K/V of every layer rebuilt from the raw sources with loops.

    static_k / static_v: [B][L][Ls][Hkv*dh] pre-RoPE prefix; frames: frame
    index -> per-env frame ([B][F][frame_dim] embeddings, or [B][L][2][F][Hkv*dh]
    pre-RoPE K then V); window: the frame indices in the window, oldest first.
    static_pos: the Ls prefix positions; frame_pos[f]: the F positions of frame f.
    On the embedding path the frame projection w_kv[l] holds the Hkv*dh K rows
    first and then the Hkv*dh V rows (the packed layout the C header documents).
    RoPE goes on K only.  Returns per-layer lists of context rows, each row a
    list of Hkv heads of dh floats: (keys, values).
    """
    Hkv, dh, L = cfg.n_kv_heads, cfg.head_dim, cfg.n_layers
    sk = _tolist(static_k)[env]
    sv = _tolist(static_v)[env]
    keys, vals = [], []
    for l in range(L):
        kl, vl = [], []
        for r in range(cfg.static_len):
            kl.append([_rot(sk[l][r][j * dh:(j + 1) * dh], static_pos[r], cfg.rope_theta) for j in range(Hkv)])
            vl.append([list(sv[l][r][j * dh:(j + 1) * dh]) for j in range(Hkv)])
        for f in window:
            fr = _tolist(frames[f])[env]
            for t in range(cfg.frame_tokens):
                if cfg.frame_dim > 0:
                    wkv = _tolist(weights["w_kv"])[l]
                    e = fr[t]
                    krow = [sum(wkv[o][i] * e[i] for i in range(cfg.frame_dim)) for o in range(Hkv * dh)]
                    vrow = [sum(wkv[Hkv * dh + o][i] * e[i] for i in range(cfg.frame_dim)) for o in range(Hkv * dh)]
                else:
                    krow = list(fr[l][0][t])
                    vrow = list(fr[l][1][t])
                kl.append([_rot(krow[j * dh:(j + 1) * dh], frame_pos[f][t], cfg.rope_theta) for j in range(Hkv)])
                vl.append([vrow[j * dh:(j + 1) * dh] for j in range(Hkv)])
        keys.append(kl)
        vals.append(vl)
    return keys, vals


def euler_loops(vel, x0, taus):
    """x_{k+1} = x_k + (tau_{k+1} - tau_k) v(x_k, tau_k) on lists of rows."""
    x = [list(r) for r in _tolist(x0)]
    for k in range(len(taus) - 1):
        v = vel(x, float(taus[k]))
        dt = float(taus[k + 1]) - float(taus[k])
        x = [[x[i][j] + dt * v[i][j] for j in range(len(x[i]))] for i in range(len(x))]
    return x
