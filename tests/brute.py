"""Brute-force probabilities of tiny SPDP corpora from the generative process.

Independent of the oracle's closed-form joint: p(W, Z) is computed here by
summing, over every seating arrangement of every restaurant, the sequential
Chinese-restaurant probabilities of the process definition (thesis, PDP
section: a new table w.p. (b + a J)/(b + N) with a dish from the base, else an
existing table of size n_j w.p. (n_j - a)/(b + N)), with the shadow base
phi0_k ~ Dirichlet(gamma) integrated out as a Polya urn over the dishes of the
tables of topic k in all groups, and theta_d ~ Dirichlet(alpha) integrated out
as a Polya urn over the topics of each document.  Pure Python, tiny inputs only.
"""
from __future__ import annotations

import itertools
import math


def _seatings(words_in_rest):
    """All table assignments (restricted growth strings) where tables share a dish."""
    n = len(words_in_rest)
    out = []

    def rec(i, assign, dishes):
        if i == n:
            out.append(tuple(assign))
            return
        w = words_in_rest[i]
        for tb, dish in enumerate(dishes):
            if dish == w:
                assign.append(tb)
                rec(i + 1, assign, dishes)
                assign.pop()
        assign.append(len(dishes))
        dishes.append(w)
        rec(i + 1, assign, dishes)
        dishes.pop()
        assign.pop()

    rec(0, [], [])
    return out


def log_p_Z(doc_off, z, K, alpha):
    lp = 0.0
    for d in range(len(doc_off) - 1):
        c = [0] * K
        for l, i in enumerate(range(doc_off[d], doc_off[d + 1])):
            lp += math.log((alpha + c[z[i]]) / (K * alpha + l))
            c[z[i]] += 1
    return lp


def p_W_given_Z(words, doc_off, doc_group, z, G, K, V, a, b, gamma):
    """Sum over all joint seatings of the sequential CRP + Polya-urn probabilities."""
    rest = {}
    for d in range(len(doc_off) - 1):
        g = doc_group[d]
        for i in range(doc_off[d], doc_off[d + 1]):
            rest.setdefault((g, z[i]), []).append(i)
    keys = sorted(rest)
    per_rest = [_seatings([words[i] for i in rest[key]]) for key in keys]
    total = 0.0
    for combo in itertools.product(*per_rest):
        p = 1.0
        B = {}
        Bk = [0] * K
        for key, seat in zip(keys, combo):
            k = key[1]
            sizes = []
            for c_idx, (i, tb) in enumerate(zip(rest[key], seat)):
                w = words[i]
                if tb == len(sizes):
                    p *= (b + a * len(sizes)) / (b + c_idx)
                    p *= (gamma + B.get((k, w), 0)) / (V * gamma + Bk[k])
                    B[(k, w)] = B.get((k, w), 0) + 1
                    Bk[k] += 1
                    sizes.append(1)
                else:
                    p *= (sizes[tb] - a) / (b + c_idx)
                    sizes[tb] += 1
        total += p
    return total


def log_p_WZ(words, doc_off, doc_group, z, G, K, V, alpha, a, b, gamma):
    return log_p_Z(doc_off, z, K, alpha) + math.log(
        p_W_given_Z(words, doc_off, doc_group, z, G, K, V, a, b, gamma))


def p_W_given_Z_assoc(words, doc_off, doc_group, z, G, K, V, a, b, gamma, assoc):
    """p(W | Z) of the model with word associations, by the same enumeration:
    a new table of group g first draws its source v from the Polya urn of its
    topic's shadow base (counts kept per source), then serves word w with
    probability p_{g,w,v} (column v of P^g); every source choice of every
    table is summed over.  `assoc[(g, w)]` maps source v -> p_{g,w,v}."""
    rest = {}
    for d in range(len(doc_off) - 1):
        g = doc_group[d]
        for i in range(doc_off[d], doc_off[d + 1]):
            rest.setdefault((g, z[i]), []).append(i)
    keys = sorted(rest)
    per_rest = [_seatings([words[i] for i in rest[key]]) for key in keys]
    total = 0.0
    for combo in itertools.product(*per_rest):
        p_seat = 1.0
        tables = []  # (g, k, w) of every new table, in order
        for key, seat in zip(keys, combo):
            g, k = key
            sizes = []
            for c_idx, (i, tb) in enumerate(zip(rest[key], seat)):
                if tb == len(sizes):
                    p_seat *= (b + a * len(sizes)) / (b + c_idx)
                    tables.append((g, k, words[i]))
                    sizes.append(1)
                else:
                    p_seat *= (sizes[tb] - a) / (b + c_idx)
                    sizes[tb] += 1
        choices = [sorted(assoc[(g, w)].items()) for g, _, w in tables]
        for pick in itertools.product(*choices):
            p = p_seat
            B = {}
            Bk = [0] * K
            for (g, k, w), (v, pv) in zip(tables, pick):
                p *= (gamma + B.get((k, v), 0)) / (V * gamma + Bk[k]) * pv
                B[(k, v)] = B.get((k, v), 0) + 1
                Bk[k] += 1
            total += p
    return total
