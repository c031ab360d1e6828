"""50-digit decimal brute force of verification attention (tiny inputs).

Test infrastructure only.  Writes Eq. 12 of Sec. 4.2 out element by element:
an explicit visibility matrix (all history, candidates j <= i), scores
s_t = sigma * sum_c q_c k_{t,c} with sigma = 1/sqrt(d), weights e^{s_t - m}
with m the maximum visible score, and O = sum_t w_t v_t / sum_t w_t.

bfloat16 inputs are dyadic rationals, so ``Decimal(float)`` is exact and the
only rounding is the 50-digit context.  Shares no code with the fp64 oracle
beyond the two readings (GQA group, candidate causality), which it restates.
"""
from __future__ import annotations

from decimal import Decimal, getcontext
from typing import List, Sequence, Tuple


def verify_attention_decimal(q, k_hist, v_hist, k_cand, v_cand) -> Tuple[List, List]:
    """Returns (O, LSE) as nested lists of Decimal: O[row][h][c], LSE[row][h]
    with rows packed in request order."""
    getcontext().prec = 50
    O_all, L_all = [], []
    for b in range(len(q)):
        qb, kh, vh, kc, vc = q[b], k_hist[b], v_hist[b], k_cand[b], v_cand[b]
        n, Hq, d = len(qb), len(qb[0]), len(qb[0][0])
        C = len(kh)
        Hkv = len(kc[0])
        G = Hq // Hkv
        sigma = Decimal(1) / Decimal(d).sqrt()
        for i in range(n):
            orow, lrow = [], []
            for h in range(Hq):
                g = h // G
                keys, vals = [], []
                for t in range(C):                      # committed history
                    keys.append(kh[t][g])
                    vals.append(vh[t][g])
                for j in range(n):                      # candidates j <= i
                    if j <= i:
                        keys.append(kc[j][g])
                        vals.append(vc[j][g])
                qv = [Decimal(float(x)) for x in qb[i][h]]
                scores = []
                for kv in keys:
                    acc = Decimal(0)
                    for c in range(d):
                        acc += qv[c] * Decimal(float(kv[c]))
                    scores.append(sigma * acc)
                m = max(scores)
                w = [(s - m).exp() for s in scores]
                l = sum(w, Decimal(0))
                out = []
                for c in range(d):
                    num = Decimal(0)
                    for t, vv in enumerate(vals):
                        num += w[t] * Decimal(float(vv[c]))
                    out.append(num / l)
                orow.append(out)
                lrow.append(m + l.ln())
            O_all.append(orow)
            L_all.append(lrow)
    return O_all, L_all
