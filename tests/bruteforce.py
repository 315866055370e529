"""Brute-force float64 decoder in pure Python loops (math.fsum), for tiny
shapes only. Written independently of ``oracle/llama.py`` to pin it: every
sum is an explicit loop, every index is spelled out, and nothing is shared
with the oracle except the weight source.
"""
from __future__ import annotations

import math


def _vec(a):
    return [float(t) for t in a]


def _mat(a):
    return [[float(t) for t in row] for row in a]


def _matvec(w, x):
    return [math.fsum(w[j][i] * x[i] for i in range(len(x))) for j in range(len(w))]


def _rmsnorm(x, g, eps):
    ms = math.fsum(t * t for t in x) / len(x)
    r = 1.0 / math.sqrt(ms + eps)
    return [x[i] * r * g[i] for i in range(len(x))]


def _rope(vec, pos, d, base):
    """Rotate one head vector: element i pairs with i + d/2."""
    half = d // 2
    out = list(vec)
    for i in range(half):
        theta = pos * base ** (-2.0 * i / d)
        c, s = math.cos(theta), math.sin(theta)
        a, b = vec[i], vec[i + half]
        out[i] = a * c - b * s
        out[i + half] = b * c + a * s
    return out


def _silu(z):
    return z / (1.0 + math.exp(-z))


class BruteDecoder:
    def __init__(self, cfg, weights):
        self.cfg = cfg
        L = cfg.n_layers
        self.E = _mat(weights(-1, "embed"))
        self.head = _mat(weights(-1, "lm_head"))
        self.gf = _vec(weights(-1, "final_norm"))
        self.layers = []
        for l in range(L):
            self.layers.append({k: (_mat(weights(l, k)) if k.startswith("w")
                                    else _vec(weights(l, k)))
                                for k in ("attn_norm", "wq", "wk", "wv", "wo",
                                          "ffn_norm", "wgate", "wup", "wdown")})

    def hidden_after(self, layer_begin, layer_end, xs):
        """Run layers [begin, end) on a whole sequence of hidden vectors xs
        (positions 0..n-1). Returns the hidden vectors after layer end-1."""
        cfg = self.cfg
        d, nh, nkv = cfg.head_dim, cfg.n_heads, cfg.n_kv_heads
        rep = nh // nkv
        xs = [list(x) for x in xs]
        n = len(xs)
        for l in range(layer_begin, layer_end):
            W = self.layers[l]
            qs, ks, vs = [], [], []
            for t in range(n):
                u = _rmsnorm(xs[t], W["attn_norm"], cfg.rms_eps)
                q, k, v = _matvec(W["wq"], u), _matvec(W["wk"], u), _matvec(W["wv"], u)
                qs.append([_rope(q[h * d:(h + 1) * d], t, d, cfg.rope_base) for h in range(nh)])
                ks.append([_rope(k[h * d:(h + 1) * d], t, d, cfg.rope_base) for h in range(nkv)])
                vs.append([v[h * d:(h + 1) * d] for h in range(nkv)])
            for t in range(n):
                o = []
                for h in range(nh):
                    kh = h // rep
                    sc = [math.fsum(qs[t][h][i] * ks[j][kh][i] for i in range(d)) / math.sqrt(d)
                          for j in range(t + 1)]
                    mx = max(sc)
                    e = [math.exp(s - mx) for s in sc]
                    z = math.fsum(e)
                    o.extend(math.fsum(e[j] / z * vs[j][kh][i] for j in range(t + 1))
                             for i in range(d))
                ao = _matvec(W["wo"], o)
                xs[t] = [xs[t][i] + ao[i] for i in range(cfg.hidden)]
            for t in range(n):
                u = _rmsnorm(xs[t], W["ffn_norm"], cfg.rms_eps)
                g, up = _matvec(W["wgate"], u), _matvec(W["wup"], u)
                a = [_silu(g[i]) * up[i] for i in range(cfg.ffn)]
                dn = _matvec(W["wdown"], a)
                xs[t] = [xs[t][i] + dn[i] for i in range(cfg.hidden)]
        return xs

    def logits(self, tokens):
        """All-position logits of the whole model on one sequence."""
        xs = [list(self.E[t]) for t in tokens]
        xs = self.hidden_after(0, self.cfg.n_layers, xs)
        return [_matvec(self.head, _rmsnorm(x, self.gf, self.cfg.rms_eps)) for x in xs]
