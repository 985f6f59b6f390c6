"""Brute-force and exact-rational restatements used to pin the oracle.

These are deliberately written differently from the oracle (pure Python
loops, ``fractions.Fraction``, direct evaluation of the defining formulas)
so that a mistake in one is unlikely to be repeated in the other.
"""
from __future__ import annotations

import struct
from fractions import Fraction


def bf16_bits_to_fraction(bits: int) -> Fraction:
    """Exact value of a bf16 bit pattern (finite values only)."""
    sign = -1 if bits & 0x8000 else 1
    exp = (bits >> 7) & 0xFF
    man = bits & 0x7F
    if exp == 0xFF:
        raise ValueError("non-finite")
    if exp == 0:
        return sign * Fraction(man, 1 << 7) * Fraction(1, 1 << 126)
    return sign * (1 + Fraction(man, 1 << 7)) * (Fraction(2) ** (exp - 127))


def f32_to_fraction(x: float) -> Fraction:
    return Fraction(struct.unpack("<f", struct.pack("<f", x))[0])


def bf16_round_exact(x: float) -> int:
    """Nearest bf16 to an fp32 value by exhaustive comparison of neighbours.

    Looks at the two bf16 patterns that bracket x (truncation and the next
    one up in magnitude) and picks the nearer; on an exact tie, the one with
    an even last bit.
    """
    v = f32_to_fraction(x)
    u = struct.unpack("<I", struct.pack("<f", x))[0]
    lo = u >> 16
    hi = lo + 1
    a, b = bf16_bits_to_fraction(lo), bf16_bits_to_fraction(hi)
    da, db = abs(v - a), abs(b - v)
    if da < db:
        return lo
    if db < da:
        return hi
    return lo if lo % 2 == 0 else hi


def dot_exact(qbits, hbits) -> Fraction:
    return sum((bf16_bits_to_fraction(int(a)) * bf16_bits_to_fraction(int(b))
                for a, b in zip(qbits, hbits)), Fraction(0))


def topk_sorted(scores, k):
    """Sort every index by (score desc, index asc) and keep the first k."""
    order = sorted(range(len(scores)), key=lambda n: (-scores[n], n))
    return order[:k]


def bin_linear(L, edges):
    """Scan the edges: largest b in [0, B-1] with edges[b] <= L, else 0."""
    B = len(edges) - 1
    best = 0
    for b in range(B):
        if edges[b] <= L:
            best = b
    return best


def histogram_exact(ids, sims, lengths, edges, tau, uniform=False):
    """One request's counts and masses with Fractions (sims given as floats);
    uniform=True weighs every neighbour at or above tau by 1 instead of s."""
    B = len(edges) - 1
    counts = [0] * B
    wsum = [Fraction(0)] * B
    valid = [(i, Fraction(s)) for i, s in zip(ids, sims) if i >= 0]
    t = Fraction(tau)
    for i, s in valid:
        b = bin_linear(lengths[i], edges)
        counts[b] += 1
        if s >= t:
            wsum[b] += 1 if uniform else s
    W = sum(wsum, Fraction(0))
    m = len(valid)
    if W > 0:
        mass = [w / W for w in wsum]
    else:
        mass = [Fraction(c, m) for c in counts]
    return counts, mass


def gittins_by_delta(p, x, extra_points=()):
    """inf over Delta of E[min(X, Delta)] / P(X <= Delta), evaluated directly.

    ``p`` and ``x`` are sequences of Fractions (any order, any scale). The
    ratio is evaluated at every support point, at midpoints between
    consecutive distinct support points, just above the largest one, and at
    any ``extra_points``; points with P(X <= Delta) = 0 are skipped. Returns
    (minimum over all evaluated Delta, list of (Delta, ratio)).
    """
    pts = sorted(set(x))
    deltas = list(pts)
    deltas += [(a + b) / 2 for a, b in zip(pts, pts[1:])]
    if pts:
        deltas.append(pts[-1] + 1)
    deltas += list(extra_points)
    evals = []
    for D in deltas:
        if D <= 0:
            continue
        spend = sum((pi * min(xi, D) for pi, xi in zip(p, x)), Fraction(0))
        done = sum((pi for pi, xi in zip(p, x) if xi <= D), Fraction(0))
        if done > 0:
            evals.append((D, spend / done))
    if not evals:
        return None, evals
    return min(r for _, r in evals), evals


def stable_order(keys):
    return sorted(range(len(keys)), key=lambda i: (keys[i], i))


def gittins_attained_by_delta(p, x, a, extra_points=()):
    """inf over Delta > 0 of E[min(X - a, Delta); X > a] / P(a < X <= a + Delta).

    Evaluated directly at Delta = (support point - a) for every support point
    above a, at midpoints between those, just above the largest, and at any
    ``extra_points``; Deltas with P(a < X <= a + Delta) = 0 are skipped.
    Returns the minimum, or None when no mass lies above a.
    """
    above = sorted(set(xi - a for xi in x if xi > a))
    deltas = list(above) + [(u + v) / 2 for u, v in zip(above, above[1:])]
    if above:
        deltas.append(above[-1] + 1)
    deltas += [d for d in extra_points if d > 0]
    best = None
    for D in deltas:
        spend = sum((pi * min(xi - a, D) for pi, xi in zip(p, x) if xi > a), Fraction(0))
        done = sum((pi for pi, xi in zip(p, x) if a < xi <= a + D), Fraction(0))
        if done > 0:
            r = spend / done
            best = r if best is None or r < best else best
    return best
