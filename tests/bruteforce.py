"""Pure-Python scalar reference for tiny problems (pin P1 of the oracle).

Written independently of ``oracle/``: rank ownership is taken from the list of
chunks a rank holds (chunks r and 2C-1-r of every sequence), the key set and
the mask are enumerated with explicit loops, the softmax uses ``math.exp`` with
an explicit running maximum, and the backward uses the textbook softmax
Jacobian sum_k P_ik dP_ik instead of <dO, O>.
"""

import math


def rank_positions(L, C, r):
    c = L // (2 * C)
    return list(range(r * c, (r + 1) * c)) + list(range((2 * C - 1 - r) * c, (2 * C - r) * c))


def queries(prob, r):
    """List of query records: (kind, seq, P, group, idx, global row)."""
    out = []
    cu = [int(x) for x in prob.cu_seqlens]
    C = prob.cp_size
    for s in range(len(cu) - 1):
        L = cu[s + 1] - cu[s]
        owned = set(rank_positions(L, C, r))
        if prob.has_main[s]:
            for p in sorted(owned):
                out.append(("m", s, p, -1, -1, cu[s] + p))
        for g in range(len(prob.g_seq)):
            if int(prob.g_seq[g]) == s and int(prob.g_anchor[g]) in owned:
                for i in range(int(prob.g_len[g])):
                    out.append(("b", s, int(prob.g_anchor[g]), g, i, int(prob.g_row0[g]) + i))
    return out


def keys_of(prob, q):
    """Allowed keys of query record q: list of ("m"|"b", global row)."""
    kind, s, P, g, i, _ = q
    base = int(prob.cu_seqlens[s])
    ks = [("m", base + j) for j in range(P + 1)]
    if kind == "b":
        n = int(prob.g_len[g])
        if int(prob.g_kind[g]) == 0:   # chain: members 0..i
            members = range(i + 1)
        else:                          # block: all members
            members = range(n)
        ks += [("b", int(prob.g_row0[g]) + j) for j in members]
    return ks


def _dot(a, b):
    return sum(x * y for x, y in zip(a, b))


def forward_backward(prob, T, dO=None, r=None):
    """T: dict of nested lists qm,km,vm,qb,kb,vb ([row][head][dim]).
    dO: dict with keys ("m"|"b", global row) -> [head][dim].
    Returns dicts keyed like dO: O, LSE (per head), and gradients."""
    r = prob.cp_rank if r is None else r
    Hq, Hkv, d = prob.hq, prob.hkv, prob.head_dim
    G = Hq // Hkv
    O, LSE = {}, {}
    grads = {}

    def addg(key, h, vec, name):
        buf = grads.setdefault((name,) + key, [[0.0] * d for _ in range(Hkv if name in ("dk", "dv") else Hq)])
        for t in range(d):
            buf[h][t] += vec[t]

    for q in queries(prob, r):
        key = (q[0], q[5])
        qt = T["qm"] if q[0] == "m" else T["qb"]
        ks = keys_of(prob, q)
        O[key] = []
        LSE[key] = []
        for h in range(Hq):
            kvh = h // G
            qv = qt[q[5]][h]
            kv = [(T["km"] if kk == "m" else T["kb"])[row][kvh] for kk, row in ks]
            vv = [(T["vm"] if kk == "m" else T["vb"])[row][kvh] for kk, row in ks]
            s = [prob.scale * _dot(qv, k) for k in kv]
            m = -math.inf
            for x in s:
                if x > m:
                    m = x
            e = [math.exp(x - m) for x in s]
            z = sum(e)
            p = [x / z for x in e]
            o = [sum(p[j] * vv[j][t] for j in range(len(vv))) for t in range(d)]
            O[key].append(o)
            LSE[key].append(m + math.log(z))
            if dO is None:
                continue
            g = dO[key][h]
            dp = [_dot(g, v) for v in vv]
            pdp = sum(p[j] * dp[j] for j in range(len(p)))
            ds = [p[j] * (dp[j] - pdp) for j in range(len(p))]
            dq = [prob.scale * sum(ds[j] * kv[j][t] for j in range(len(kv))) for t in range(d)]
            addg(key, h, dq, "dq")
            for j, (kk, row) in enumerate(ks):
                addg((kk, row), kvh, [prob.scale * ds[j] * qv[t] for t in range(d)], "dk")
                addg((kk, row), kvh, [p[j] * g[t] for t in range(d)], "dv")
    return O, LSE, grads
