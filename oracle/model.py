"""Closed-form completion times and lower bounds, in exact rationals.

TEST INFRASTRUCTURE ONLY (see the package docstring).

All times are in the paper's bandwidth-bound unit, the time a healthy NIC
needs for one element; a NIC slowed by a factor l needs l of these units;
latency and launch costs are excluded (Sec. 3, problem setting).  Bandwidths
are turned into slowdowns as l_i = max(b) / b_i, so ``Fraction`` keeps every
value exact for the binary fractions used by the workloads.
"""
from __future__ import annotations

from fractions import Fraction as F


def slowdowns(bandwidths):
    """(l_1 >= ... >= l_m, p): the stragglers' slowdowns sorted descending."""
    b = [F(x) for x in bandwidths]
    if any(x <= 0 for x in b):
        raise ValueError("bandwidths must be > 0")
    bmax = max(b)
    ells = sorted((bmax / x for x in b if x < bmax), reverse=True)
    return ells, len(b)


def t0(p, n):
    """Fault-free optimum with one GPU per server: 2(p-1)n/p (Sec. 3)."""
    return F(2 * (p - 1), p) * n


def optcc_single(p, ell, n, k):
    """One straggler (Sec. 4.3 time analysis, App. C):
    l >= 2: T = l n (k+1)/k;  l < 2: T = 2(p-1) l n / ((p-2) l + 2) * (k+l-1)/k."""
    ell = F(ell)
    if ell >= 2:
        return ell * n * F(k + 1, k)
    return F(2 * (p - 1)) * ell * n / ((p - 2) * ell + 2) * (k + ell - 1) / k


def optcc_multi(p, ells, n, k):
    """m >= 2 stragglers (App. D time analysis): s = n/(k(p-m)),
    T_body = max{2(p-1)s, (l_1(p-m) + 2(m-1))s}, T = (k+4) T_body."""
    m = len(ells)
    s = F(n) / (k * (p - m))
    body = max(2 * (p - 1) * s, (ells[0] * (p - m) + 2 * (m - 1)) * s)
    return (k + 4) * body


def optcc_time(bandwidths, n, k):
    """Completion time of the OptCC schedule for this bandwidth profile."""
    ells, p = slowdowns(bandwidths)
    if not ells:
        return t0(p, n)  # no straggler: the ring schedule, exactly T0
    if len(ells) == 1:
        return optcc_single(p, ells[0], n, k)
    return optcc_multi(p, ells, n, k)


def lb_weak_single(p, ell, n):
    """Theorem 1: T >= max{2l(p-1)/(l(p-1)+1), l} n."""
    ell = F(ell)
    return max(2 * ell * (p - 1) / (ell * (p - 1) + 1), ell) * n


def lb_tight_single(p, ell, n):
    """Tight single-straggler bound (App. B.1): T >= max{2l(p-1)/(l(p-2)+2), l} n."""
    ell = F(ell)
    return max(2 * ell * (p - 1) / (ell * (p - 2) + 2), ell) * n


def lb_multi(p, ells, n):
    """Theorem 2: T >= max{2(p-1)/(p-m+sum 1/l_i), l_1} n."""
    m = len(ells)
    y0 = F(2 * (p - 1)) / (p - m + sum(F(1) / e for e in ells))
    return max(y0, max(ells)) * n


def lower_bound(bandwidths, n):
    """Best known lower bound: T0 without stragglers, the tight bound for one
    straggler, Theorem 2 for several (App. A, best lower bounds table)."""
    ells, p = slowdowns(bandwidths)
    if not ells:
        return t0(p, n)
    if len(ells) == 1:
        return lb_tight_single(p, ells[0], n)
    return lb_multi(p, ells, n)


def degraded_ring(bandwidths, n):
    """A plain ring runs at the slowest NIC: l_max T0 (context figure)."""
    ells, p = slowdowns(bandwidths)
    return (ells[0] if ells else F(1)) * t0(p, n)


def bubble_split(p, ell, n, k):
    """Section size s' and P2P chunk D per segment for l < 2 (App. C):
    s' = n l / (k((p-2)l+2)), D = (2-l) s' / l."""
    ell = F(ell)
    sp = F(n) * ell / (k * ((p - 2) * ell + 2))
    return sp, (2 - ell) * sp / ell


def straggler_volume_optimum(p, ell, n):
    """z* n with z* = 2(p-1)/(l(p-2)+2): the straggler send/receive volume at
    the minimiser of the tight bound's min-max problem (App. B.1)."""
    return F(2 * (p - 1)) / (F(ell) * (p - 2) + 2) * n


# ------------------------------------------------ several GPUs per server
def t0_servers(p, g, n):
    """Fault-free optimum with g GPUs per server: 2(p-1)n/(gp) (Sec. 3)."""
    return F(2 * (p - 1), g * p) * n


def optcc_servers(q, g, ell, n, k):
    """App. E time analysis (single straggler server, no bubble filling):
    T <= l n (k+5.5)/(g k) for l >= 2, 2 n (k+5.5)/(g k) for l < 2."""
    ell = F(ell)
    body = ell if ell >= 2 else F(2)
    return body * n * (k + F(11, 2)) / (g * k)


def lb_servers_weak(q, g, ell, n):
    """Theorem 3: T >= (n/g) max{2l(q-1)/(1+l(q-1)), l} (App. B.3 form)."""
    ell = F(ell)
    return F(n, g) * max(2 * ell * (q - 1) / (1 + ell * (q - 1)), ell)


def lb_servers_tight(q, g, ell, n):
    """Tight multi-GPU bound (App. B.3): T >= (n/g) max{2l(q-1)/(l(q-2)+2), l}."""
    ell = F(ell)
    return F(n, g) * max(2 * ell * (q - 1) / (ell * (q - 2) + 2), ell)
