"""Scalar-loop float64 forward pass, written independently of the oracle, for tiny shapes.

Plain Python lists and the ``math`` module only: every sum is an explicit loop, so
this shares no vectorised helper with the oracle it is used to pin.  Same model
family (pre-norm decoder, RMSNorm, half-split rotary embedding, grouped-query
attention with contiguous query-head groups, SwiGLU MLP).
"""
import math


def _mat(w):
    return [list(map(float, row)) for row in w]


def _rms(x, g, eps):
    ms = 0.0
    for v in x:
        ms += v * v
    ms /= len(x)
    r = 1.0 / math.sqrt(ms + eps)
    return [x[c] * r * float(g[c]) for c in range(len(x))]


def _matvec(w, x):
    out = []
    for row in w:
        s = 0.0
        for c in range(len(x)):
            s += row[c] * x[c]
        out.append(s)
    return out


def _rotate(vec, pos, base):
    hd = len(vec)
    half = hd // 2
    out = list(vec)
    for i in range(half):
        theta = base ** (-(2.0 * i) / hd)
        a = pos * theta
        c, s = math.cos(a), math.sin(a)
        out[i] = vec[i] * c - vec[i + half] * s
        out[i + half] = vec[i + half] * c + vec[i] * s
    return out


def forward(cfg, weights, ids):
    """Final-normed hidden rows, list of n lists of d floats."""
    d, nq, nkv, hd = cfg.d_model, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    per_group = nq // nkv
    E = weights["tok_emb"]
    x = [list(map(float, E[t])) for t in ids]
    n = len(ids)
    for layer in weights["layers"]:
        wqkv = _mat(layer["w_qkv"])
        wo, wg, wu, wd = (_mat(layer[k]) for k in ("w_o", "w_gate", "w_up", "w_down"))
        qs, ks, vs = [], [], []
        for i in range(n):
            a = _rms(x[i], layer["attn_norm"], cfg.rms_eps)
            y = _matvec(wqkv, a)
            q = [_rotate(y[h * hd:(h + 1) * hd], i, cfg.rope_base) for h in range(nq)]
            koff = nq * hd
            voff = koff + nkv * hd
            k = [_rotate(y[koff + g * hd:koff + (g + 1) * hd], i, cfg.rope_base) for g in range(nkv)]
            v = [y[voff + g * hd:voff + (g + 1) * hd] for g in range(nkv)]
            qs.append(q)
            ks.append(k)
            vs.append(v)
        new_x = []
        for i in range(n):
            o = []
            for h in range(nq):
                g = h // per_group
                scores = []
                for j in range(i + 1):
                    s = 0.0
                    for e in range(hd):
                        s += qs[i][h][e] * ks[j][g][e]
                    scores.append(s / math.sqrt(hd))
                m = max(scores)
                ex = [math.exp(s - m) for s in scores]
                z = sum(ex)
                for e in range(hd):
                    acc = 0.0
                    for j in range(i + 1):
                        acc += ex[j] / z * vs[j][g][e]
                    o.append(acc)
            proj = _matvec(wo, o)
            xi = [x[i][c] + proj[c] for c in range(d)]
            b = _rms(xi, layer["mlp_norm"], cfg.rms_eps)
            gate = _matvec(wg, b)
            up = _matvec(wu, b)
            hmid = [gate[f] / (1.0 + math.exp(-gate[f])) * up[f] for f in range(len(gate))]
            down = _matvec(wd, hmid)
            new_x.append([xi[c] + down[c] for c in range(d)])
        x = new_x
    return [_rms(x[i], weights["final_norm"], cfg.rms_eps) for i in range(n)]


def logits(weights, h):
    return _matvec(_mat(weights["lm_head"]), h)
