"""Pure-Python brute force of the MoE layer, used to pin the oracle on tiny inputs.

It is a different algorithm from the oracle on purpose:

* top-k is chosen by enumerating every k-subset of experts and keeping the
  unique one whose members all rank ahead of every non-member (larger logit,
  or an equal logit and a lower index);
* every expert's FFN is evaluated densely for every token, and the output is
  the full sum over experts of G[t,e] * FFN_e(x_t) with G zero outside the
  chosen subset;
* the slot order of the chosen experts is found by sorting on (-logit, index).

Inputs are Python lists of floats (already widened from bf16).  Only for
T, d, ffn, E of a few units: plain loops, no numpy.
"""

from __future__ import annotations

import itertools
import math


def ahead(la, a, lb, b):
    return la > lb or (la == lb and a < b)


def topk_subset(logits, k):
    """The unique k-subset whose members all rank ahead of all non-members."""
    E = len(logits)
    found = []
    for sub in itertools.combinations(range(E), k):
        rest = [e for e in range(E) if e not in sub]
        if all(ahead(logits[i], i, logits[o], o) for i in sub for o in rest):
            found.append(sub)
    assert len(found) == 1, f"expected one top-k subset, got {found}"
    return found[0]


def route(logits_row, k):
    sub = topk_subset(logits_row, k)
    order = sorted(sub, key=lambda e: (-logits_row[e], e))
    top = logits_row[order[0]]
    ex = [math.exp(logits_row[e] - top) for e in order]
    s = sum(ex)
    return order, [v / s for v in ex]


def matvec(W, v):
    return [sum(W[r][i] * v[i] for i in range(len(v))) for r in range(len(W))]


def silu(z):
    return z / (1.0 + math.exp(-z))


def expert_ffn(W1e, W3e, W2e, x):
    u = matvec(W1e, x)
    v = matvec(W3e, x)
    h = [silu(a) * b for a, b in zip(u, v)]
    return matvec(W2e, h)


def moe_layer(x, wr, w1, w3, w2, k, bias=None):
    """x: [T][d]; wr: [E][d]; w1,w3: [E][ffn][d]; w2: [E][d][ffn].

    Returns (out [T][d], ids [T][k], gates [T][k], logits [T][E])."""
    E = len(wr)
    d = len(x[0]) if x else 0
    outs, ids, gates, logits = [], [], [], []
    for xt in x:
        lg = [sum(xt[i] * wr[e][i] for i in range(d)) + (bias[e] if bias is not None else 0.0)
              for e in range(E)]
        order, g = route(lg, k)
        G = [0.0] * E
        for e, gv in zip(order, g):
            G[e] = gv
        # dense: every expert evaluated, weighted by G (zero outside the top-k)
        acc = [0.0] * d
        for e in range(E):
            ye = expert_ffn(w1[e], w3[e], w2[e], xt)
            for i in range(d):
                acc[i] += G[e] * ye[i]
        outs.append(acc)
        ids.append(list(order))
        gates.append(g)
        logits.append(lg)
    return outs, ids, gates, logits


def dispatch(ids, E):
    """counts, offsets, perm recounted by brute force."""
    flat = [e for row in ids for e in row]
    counts = [flat.count(e) for e in range(E)]
    offsets = [0]
    for c in counts:
        offsets.append(offsets[-1] + c)
    perm = sorted(range(len(flat)), key=lambda a: (flat[a], a))
    return counts, offsets, perm
