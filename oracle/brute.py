"""Scalar-loop brute force of the same decoder layer, for tiny shapes only.

Written independently of ``layer.py`` (plain Python floats and loops, the
``math`` module, no numpy arithmetic), so that a slip in the vectorised
oracle (a transposed operand, a wrong head-to-KV-head index, a wrong RoPE
pair or sign, a dropped residual) shows up as a mismatch. Same readings as
``layer.py``; see its docstring for the layer and the paper sections.
"""
import math


def _vec(a):
    return [float(v) for v in a]


def _mat(a):
    return [[float(v) for v in row] for row in a]


def brute_layer(w, n_q, n_kv, d, eps, base, X, k_cache, v_cache, pos0,
                peer_attn=None, peer_ffn=None, window=0):
    """Full layer over T tokens; inputs are nested sequences or arrays.
    ``window`` > 0: token at position p attends to positions p - window + 1
    .. p only (sliding window).

    Returns dict of python lists: p_attn, h, p_ffn, y ([T][H]).
    """
    X = _mat(X)
    T, H = len(X), len(X[0])
    g1, g2 = _vec(w.g_attn), _vec(w.g_ffn)
    wq, wk, wv, wo = _mat(w.wq), _mat(w.wk), _mat(w.wv), _mat(w.wo)
    wg, wu, wd = _mat(w.wg), _mat(w.wu), _mat(w.wd)
    F = len(wg)
    group = (n_q // n_kv) if n_kv else 1

    # key/value lists per KV head, starting with the cached positions
    keys = [[_vec(k_cache[g][p]) for p in range(pos0)] for g in range(n_kv)]
    vals = [[_vec(v_cache[g][p]) for p in range(pos0)] for g in range(n_kv)]

    def rms(vec, gain):
        s = 0.0
        for a in vec:
            s += a * a
        r = 1.0 / math.sqrt(s / len(vec) + eps)
        return [vec[i] * r * gain[i] for i in range(len(vec))]

    def matvec(M, vec):
        out = []
        for row in M:
            acc = 0.0
            for a, b in zip(row, vec):
                acc += a * b
            out.append(acc)
        return out

    def rotate(head, p):
        out = list(head)
        for i in range(d // 2):
            ang = p * base ** (-(2.0 * i) / d)
            c, s = math.cos(ang), math.sin(ang)
            a, b = head[2 * i], head[2 * i + 1]
            out[2 * i] = a * c - b * s
            out[2 * i + 1] = a * s + b * c
        return out

    res = {"p_attn": [], "h": [], "p_ffn": [], "y": []}
    # Keys/values of the whole chunk are appended before any token attends;
    # causality limits token t to positions <= pos0 + t.
    per_tok = []
    for t in range(T):
        p = pos0 + t
        u = rms(X[t], g1)
        qf, kf, vf = matvec(wq, u), matvec(wk, u), matvec(wv, u)
        qs = [rotate(qf[j * d:(j + 1) * d], p) for j in range(n_q)]
        for g in range(n_kv):
            keys[g].append(rotate(kf[g * d:(g + 1) * d], p))
            vals[g].append(vf[g * d:(g + 1) * d])
        per_tok.append(qs)
    for t in range(T):
        p = pos0 + t
        cat = []
        for j in range(n_q):
            g = j // group
            first = max(0, p - window + 1) if window > 0 else 0
            span = list(range(first, p + 1))
            scores = []
            for pp in span:
                acc = 0.0
                for i in range(d):
                    acc += per_tok[t][j][i] * keys[g][pp][i]
                scores.append(acc / math.sqrt(d))
            mx = max(scores)
            ex = [math.exp(s - mx) for s in scores]
            tot = sum(ex)
            o = [0.0] * d
            for n, pp in enumerate(span):
                wgt = ex[n] / tot
                for i in range(d):
                    o[i] += wgt * vals[g][pp][i]
            cat.extend(o)
        pa = matvec(wo, cat)
        pe = [0.0] * H if peer_attn is None else _vec(peer_attn[t])
        h = [X[t][i] + pa[i] + pe[i] for i in range(H)]
        wn = rms(h, g2)
        gate, up = matvec(wg, wn), matvec(wu, wn)
        m = [gate[c] / (1.0 + math.exp(-gate[c])) * up[c] for c in range(F)]
        pf = matvec(wd, m)
        pe2 = [0.0] * H if peer_ffn is None else _vec(peer_ffn[t])
        y = [h[i] + pf[i] + pe2[i] for i in range(H)]
        res["p_attn"].append(pa)
        res["h"].append(h)
        res["p_ffn"].append(pf)
        res["y"].append(y)
    return res
