"""50-digit ``decimal`` evaluation of attention, used to pin the fp64 oracle.

Independent of ``oracle/``: pure Python loops over Decimal numbers, written
from the definition of softmax attention (scores, log-sum-exp, weighted sum).
"""
from decimal import Decimal, getcontext

getcontext().prec = 50


def _d(x):
    return Decimal(float(x))  # exact: every float64 is a finite decimal


def attend_decimal(q, k, v, scale):
    """q [Lq][d], k/v [Lk][d] nested lists of floats -> (O, LSE) as Decimals."""
    sc = _d(scale)
    out, lses = [], []
    for qi in q:
        s = [sc * sum(_d(a) * _d(b) for a, b in zip(qi, kj)) for kj in k]
        m = max(s)
        tot = sum((x - m).exp() for x in s)
        lse = m + tot.ln()
        p = [(x - lse).exp() for x in s]
        out.append([sum(pj * _d(vj[c]) for pj, vj in zip(p, v)) for c in range(len(v[0]))])
        lses.append(lse)
    return out, lses
