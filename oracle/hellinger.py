"""Topic-model comparison by Hellinger distance (fp64 numpy oracle).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: never imported by the
product library, and sharing no code with it.

The thesis compares two topic models (its GPU samplers against the original
serial SPDP) by the Hellinger distance between every pair of their topics,
with the second model's topics re-ordered to line up with the first's
(chapter "Experiments", subsection "Hellinger Distance").  It cites the
distance without writing it out; this module uses the textbook definition
for discrete distributions p, q over the same outcomes,

    H(p, q) = sqrt( 1/2 * sum_v (sqrt(p_v) - sqrt(q_v))^2 )   in [0, 1],

and takes the reordering of topics as the one-to-one matching of topics of least
total distance (a linear assignment problem, solved here by scipy's library
routine).
"""
from __future__ import annotations

import numpy as np
from scipy.optimize import linear_sum_assignment


def hellinger(P: np.ndarray, Q: np.ndarray) -> np.ndarray:
    """H[i, j] = Hellinger distance between row i of P [kp, V] and row j of
    Q [kq, V]; each row is a distribution over the same V outcomes."""
    P = np.asarray(P, dtype=np.float64)
    Q = np.asarray(Q, dtype=np.float64)
    if P.ndim != 2 or Q.ndim != 2 or P.shape[1] != Q.shape[1]:
        raise ValueError("P and Q must be [kp, V] and [kq, V]")
    sp, sq = np.sqrt(P), np.sqrt(Q)
    H = np.empty((P.shape[0], Q.shape[0]))
    for i in range(P.shape[0]):
        d = sp[i][None, :] - sq
        H[i] = np.sqrt(0.5 * (d * d).sum(axis=1))
    return H


def align_topics(H: np.ndarray):
    """Match every row of H [kp, kq] (kp <= kq) to its own column so that the
    summed distance is least.  Returns (match [kp] int64: column of row i,
    total distance)."""
    H = np.asarray(H, dtype=np.float64)
    if H.shape[0] > H.shape[1]:
        raise ValueError("align_topics needs kp <= kq")
    rows, cols = linear_sum_assignment(H)
    match = np.empty(H.shape[0], dtype=np.int64)
    match[rows] = cols
    return match, float(H[rows, cols].sum())
