"""Pure-Python brute force for tiny draft-attention cases (a pin for the oracle, not the oracle).

Written independently of ``oracle/``: its own bf16 decode (``struct``), its own
page walk, RoPE in complex form (the pair (x_m, x_{m+D/2}) is the complex number
x_m + i x_{m+D/2} multiplied by e^{i p theta_m}), explicit loops and
``math.fsum``.  Only for shapes with a handful of keys and head_dim <= 8.
"""
import cmath
import math
import struct


def _val(x, dtype):
    if dtype == "bf16":
        return struct.unpack("<f", struct.pack("<I", (int(x) & 0xFFFF) << 16))[0]
    return float(x)


def _vec(a, dtype):
    return [_val(v, dtype) for v in list(a)]


def _rot(vec, pos, theta):
    D = len(vec)
    h = D // 2
    out = [0.0] * D
    for m in range(h):
        z = complex(vec[m], vec[m + h]) * cmath.exp(1j * pos * theta ** (-2.0 * m / D))
        out[m], out[m + h] = z.real, z.imag
    return out


def _attend(qv, keys, vals, scale):
    z = [scale * math.fsum(a * b for a, b in zip(qv, k)) for k in keys]
    mx = max(z)
    e = [math.exp(v - mx) for v in z]
    tot = math.fsum(e)
    D = len(vals[0])
    return [math.fsum(e[i] * vals[i][d] for i in range(len(vals))) / tot for d in range(D)]


def _prefix(pages, table_row, T, P, g, dtype):
    ks = []
    for t in range(T):
        page = int(table_row[t // P])
        ks.append(_vec(pages[page][g][t % P], dtype))
    return ks


def _ancestors(parents, i):
    out = []
    while i != -1:
        out.append(i)
        i = int(parents[i])
    return out


def brute_step(case):
    c = case
    B, n, Hq, D = c.q.shape
    Hkv = c.num_kv_heads
    G = Hq // Hkv
    out = [[[None] * Hq for _ in range(n)] for _ in range(B)]
    pb = getattr(c, "pos_base", None)
    for b in range(B):
        T = int(c.ctx_lens[b])
        base = T if pb is None else int(pb[b])
        s0 = int(c.step_offsets[b])
        for j in range(n):
            for h in range(Hq):
                g = h // G
                keys = _prefix(c.k_pages, c.page_table[b], T, c.page_size, g, c.dtype)
                vals = _prefix(c.v_pages, c.page_table[b], T, c.page_size, g, c.dtype)
                for s in range(s0 + j + 1):
                    keys.append(_rot(_vec(c.draft_k[b][s][g], c.dtype), base + s, c.rope_theta))
                    vals.append(_vec(c.draft_v[b][s][g], c.dtype))
                qv = _rot(_vec(c.q[b][j][h], c.dtype), base + s0 + j, c.rope_theta)
                out[b][j][h] = _attend(qv, keys, vals, c.scale)
    return out


def brute_tree(case):
    c = case
    B, nq, Hq, D = c.q.shape
    Hkv = c.num_kv_heads
    G = Hq // Hkv
    pb = getattr(c, "pos_base", None)
    qn = getattr(c, "query_nodes", None)
    out = [[[None] * Hq for _ in range(nq)] for _ in range(B)]
    for b in range(B):
        T = int(c.ctx_lens[b])
        base = T if pb is None else int(pb[b])
        par = [int(p) for p in c.parents[b]]
        for row in range(nq):
            i = row if qn is None else int(qn[b][row])
            anc = _ancestors(par, i)
            for h in range(Hq):
                g = h // G
                keys = _prefix(c.k_pages, c.page_table[b], T, c.page_size, g, c.dtype)
                vals = _prefix(c.v_pages, c.page_table[b], T, c.page_size, g, c.dtype)
                for s in sorted(anc):
                    ds = len(_ancestors(par, s)) - 1
                    keys.append(_rot(_vec(c.draft_k[b][s][g], c.dtype), base + ds, c.rope_theta))
                    vals.append(_vec(c.draft_v[b][s][g], c.dtype))
                qv = _rot(_vec(c.q[b][row][h], c.dtype), base + len(anc) - 1, c.rope_theta)
                out[b][row][h] = _attend(qv, keys, vals, c.scale)
    return out
