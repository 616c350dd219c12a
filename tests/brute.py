"""Scalar brute force of the decoder layer and head, for tiny shapes only.

Written independently of ``oracle/`` with explicit Python loops over float
(IEEE double) scalars, so that a mistake in the vectorised oracle (a dropped
term, a transposed operand, a wrong head group or rotation pair) shows up as a
disagreement.  It follows the same textbook definition: pre-norm RMSNorm,
grouped-query attention with rotate-half RoPE, SwiGLU MLP, greedy head.
"""
import math


def widen(bits):
    """bf16 bit patterns (nested lists or numpy uint16) to nested lists of float."""
    import struct

    def one(b):
        return struct.unpack("<f", struct.pack("<I", int(b) << 16))[0]

    if hasattr(bits, "tolist"):
        bits = bits.tolist()
    if isinstance(bits, list):
        return [widen(b) for b in bits]
    return one(bits)


def norm_vec(x, g, eps):
    s = 0.0
    for xi in x:
        s += xi * xi
    r = 1.0 / math.sqrt(s / len(x) + eps)
    return [x[i] * r * g[i] for i in range(len(x))]


def matvec(W, x):
    out = []
    for row in W:
        acc = 0.0
        for j in range(len(x)):
            acc += row[j] * x[j]
        out.append(acc)
    return out


def rotate(vec, p, theta):
    hd = len(vec)
    half = hd // 2
    out = list(vec)
    for i in range(half):
        ang = p * theta ** (-(2.0 * i) / hd)
        c, s = math.cos(ang), math.sin(ang)
        a, b = vec[i], vec[i + half]
        out[i] = a * c - b * s
        out[i + half] = b * c + a * s
    return out


class BruteStage:
    """Layers ``lo..hi-1`` with weights W[l][name] as nested float lists."""

    def __init__(self, shape, lo, hi, W, head=None):
        self.s, self.lo, self.hi, self.W, self.head = shape, lo, hi, W, head
        self.K = {}  # (layer, user) -> list over positions of [kv_head][hd]
        self.V = {}

    def layer(self, l, rows, users, positions):
        s = self.s
        nq, nkv, hd = s.n_q_heads, s.n_kv_heads, s.head_dim
        w = self.W[l]
        qs = []
        for n, x in enumerate(rows):
            xn = norm_vec(x, w["attn_norm"], s.rms_eps)
            q = matvec(w["wq"], xn)
            k = matvec(w["wk"], xn)
            v = matvec(w["wv"], xn)
            p = positions[n]
            qh = [rotate(q[h * hd:(h + 1) * hd], p, s.rope_theta) for h in range(nq)]
            kh = [rotate(k[g * hd:(g + 1) * hd], p, s.rope_theta) for g in range(nkv)]
            vh = [v[g * hd:(g + 1) * hd] for g in range(nkv)]
            Kc = self.K.setdefault((l, users[n]), [])
            Vc = self.V.setdefault((l, users[n]), [])
            while len(Kc) <= p:
                Kc.append(None)
                Vc.append(None)
            Kc[p], Vc[p] = kh, vh
            qs.append(qh)
        outs = []
        for n, x in enumerate(rows):
            p = positions[n]
            Kc, Vc = self.K[(l, users[n])], self.V[(l, users[n])]
            att = []
            per_group = nq // nkv
            for h in range(nq):
                g = h // per_group
                scores = []
                for t in range(p + 1):
                    d = 0.0
                    for i in range(hd):
                        d += qs[n][h][i] * Kc[t][g][i]
                    scores.append(d / math.sqrt(hd))
                m = max(scores)
                ex = [math.exp(sc - m) for sc in scores]
                tot = sum(ex)
                for i in range(hd):
                    acc = 0.0
                    for t in range(p + 1):
                        acc += ex[t] / tot * Vc[t][g][i]
                    att.append(acc)
            o = matvec(w["wo"], att)
            x1 = [x[i] + o[i] for i in range(len(x))]
            z = norm_vec(x1, w["mlp_norm"], s.rms_eps)
            gt = matvec(w["wg"], z)
            up = matvec(w["wu"], z)
            a = [gt[j] / (1.0 + math.exp(-gt[j])) * up[j] for j in range(len(gt))]
            d = matvec(w["wd"], a)
            outs.append([x1[i] + d[i] for i in range(len(x1))])
        return outs

    def forward(self, rows, users, positions):
        for l in range(self.lo, self.hi):
            rows = self.layer(l, rows, users, positions)
        return rows

    def embed(self, toks):
        return [list(self.head["embed"][t]) for t in toks]

    def logits(self, rows):
        out = []
        for x in rows:
            xn = norm_vec(x, self.head["final_norm"], self.s.rms_eps)
            out.append(matvec(self.head["lm_head"], xn))
        return out
