"""Scalar-loop attention forward and backward for tiny inputs (oracle; test only).

The same definition as oracle/attention.py (see its docstring for the paper
passages), written element by element with Python floats and math.exp, with no
numpy matrix products, so that a slip in one of the two implementations shows
up as a disagreement.  The backward loops follow the chain rule of
L = sum(O * dO) through O_i = sum_j P_ij v_j and the row softmax, element by
element.  Only for B, S, H, d of a few units.  S is the query length; the
key/value length S_k defaults to S (cross-attention when it differs).
"""
import math


def _get(x, b, s, h, d, i):
    return float(x[b][s][h * d + i])


def fwd(q, k, v, B, S, Hq, Hkv, d, scale, causal=False, kv_len=None, S_k=None):
    """Returns O as nested lists [B][S][Hq*d], LSE [B][Hq][S], P [B][Hq][S][S_k]."""
    G = Hq // Hkv
    S_k = S if S_k is None else S_k
    O = [[[0.0] * (Hq * d) for _ in range(S)] for _ in range(B)]
    LSE = [[[0.0] * S for _ in range(Hq)] for _ in range(B)]
    P = [[[[0.0] * S_k for _ in range(S)] for _ in range(Hq)] for _ in range(B)]
    for b in range(B):
        for h in range(Hq):
            g = h // G
            for i in range(S):
                scores = []
                for j in range(S_k):
                    ok = True
                    if causal and j > i:
                        ok = False
                    if kv_len is not None and j >= int(kv_len[b]):
                        ok = False
                    if ok:
                        dot = 0.0
                        for t in range(d):
                            dot += _get(q, b, i, h, d, t) * _get(k, b, j, g, d, t)
                        scores.append((j, scale * dot))
                if not scores:
                    LSE[b][h][i] = -math.inf
                    continue
                mx = max(sv for _, sv in scores)
                tot = sum(math.exp(sv - mx) for _, sv in scores)
                LSE[b][h][i] = mx + math.log(tot)
                for j, sv in scores:
                    P[b][h][i][j] = math.exp(sv - mx) / tot
                for t in range(d):
                    acc = 0.0
                    for j, _ in scores:
                        acc += P[b][h][i][j] * _get(v, b, j, g, d, t)
                    O[b][i][h * d + t] = acc
    return O, LSE, P


def bwd(q, k, v, do, B, S, Hq, Hkv, d, scale, causal=False, kv_len=None, S_k=None):
    """Returns dQ [B][S][Hq*d], dK, dV [B][S_k][Hkv*d] as nested lists."""
    G = Hq // Hkv
    S_k = S if S_k is None else S_k
    O, _, P = fwd(q, k, v, B, S, Hq, Hkv, d, scale, causal, kv_len, S_k)
    dQ = [[[0.0] * (Hq * d) for _ in range(S)] for _ in range(B)]
    dK = [[[0.0] * (Hkv * d) for _ in range(S_k)] for _ in range(B)]
    dV = [[[0.0] * (Hkv * d) for _ in range(S_k)] for _ in range(B)]
    for b in range(B):
        for h in range(Hq):
            g = h // G
            for i in range(S):
                # dL/dP_ij = dO_i . v_j ; softmax Jacobian: dS_ij = P_ij (dP_ij - sum_l P_il dP_il)
                dP = [0.0] * S_k
                for j in range(S_k):
                    acc = 0.0
                    for t in range(d):
                        acc += _get(do, b, i, h, d, t) * _get(v, b, j, g, d, t)
                    dP[j] = acc
                expect = sum(P[b][h][i][j] * dP[j] for j in range(S_k))
                for j in range(S_k):
                    pij = P[b][h][i][j]
                    if pij == 0.0:
                        continue
                    ds = pij * (dP[j] - expect)
                    for t in range(d):
                        dQ[b][i][h * d + t] += scale * ds * _get(k, b, j, g, d, t)
                        dK[b][j][g * d + t] += scale * ds * _get(q, b, i, h, d, t)
                        dV[b][j][g * d + t] += pij * _get(do, b, i, h, d, t)
    return dQ, dK, dV
