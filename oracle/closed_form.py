"""The final value of every coordinate, written directly from the stated
conventions, without the oracle's step list.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The step-by-step executor (``oracle.run``) applies the schedule it builds;
this module derives, for each coordinate, the expression the schedule must
evaluate from the paper's stages and the readings listed below, and evaluates it
with the same rounding rule.  The two agreeing bit for bit checks that the
step list implements the readings.

Readings used (paper: "Don't Let a Few Network Failures Slow the Entire
AllReduce"):
* stragglers are the ranks slower than the fastest, sorted by slowdown
  l = max(b)/b descending, ties to the lower rank; the healthy ranks form the
  ring in ascending order (Sec. 4.1 Stage 1);
* split: quanta of 64 elements; segment g owns quanta
  [floor(g NQ / k), floor((g+1) NQ / k)); with one straggler and l < 2 the
  segment ends with a point-to-point chunk of floor(x + 1/2) quanta,
  x = Lq (2 - l) / ((p - 2) l + 2) (App. C, D = (2 - l) s' / l); the other
  quanta are split over the healthy ranks' sections, the first ones one
  quantum larger; element ranges are clipped at N;
* section j's Stage-1 chain starts at R[j] and adds R[j+1], ..., R[j+P'-1]
  one hop at a time (Sec. 4.1);
* one straggler: segments g with g mod 4 in {0, 2} (patterns A, C) use
  ordering 1 (the straggler adds its value to the chain's result), the
  others ordering 2 (the straggler's value joins at the chain start);
* several stragglers (App. D): g mod 4 in {0, 1} (patterns B, D) fold all
  stragglers' values into the chain start, in one step; g mod 4 in {2, 3}
  (A', C') fold all but the worst there, and the worst adds its value to the
  chain's result;
* bubble filling (Sec. 4.2, App. C): the straggler sums its own chunk and
  R[0], ..., R[P'-1] in that order, rounding once;
* several GPUs per server (App. E): ranks server-major; g parts of whole
  quanta, part i led by local GPU i; a collect runs the local ring from
  position g-1 down to the leader, each GPU adding its value; segment c of a
  part uses type 1 (c mod 4 in {0, 2}: chain over the healthy leaders, then
  the straggler server's leader and the rest of its ring add their values in
  ring order) or type 2 (the straggler server's collected sum joins the
  chain start);
* rounding: every step narrows its fp32 sum once (round to nearest even for
  bf16 and fp16, exact for fp32); a step with several sources accumulates in
  fp32 first.
"""
from __future__ import annotations

import numpy as np

Q = 64


def _to_f32(dtype, a):
    import oracle
    if dtype == "f32":
        return a.astype(np.float32)
    if dtype == "bf16":
        return oracle.bf16_to_f64(a).astype(np.float32)
    if dtype == "f16":
        return oracle.f16_to_f64(a).astype(np.float32)
    raise ValueError("floating-point types only: integer sums do not depend on the order")


def _narrow(dtype, f):
    import oracle
    if dtype == "f32":
        return f.astype(np.float32)
    if dtype == "bf16":
        return oracle.bf16_round(f)
    return oracle.f16_round(f)


def _step(dtype, a, b):
    """One single-source step: narrow(widen(a) + widen(b))."""
    return _narrow(dtype, _to_f32(dtype, a) + _to_f32(dtype, b))


def _multi(dtype, first, rest):
    """One multi-source step: fp32 sum of first, then rest in order, narrowed once."""
    acc = _to_f32(dtype, first)
    for r in rest:
        acc = acc + _to_f32(dtype, r)
    return _narrow(dtype, acc)


def _ranks(bandwidths):
    bmax = max(bandwidths)
    ell = [bmax / b for b in bandwidths]
    strag = sorted((r for r in range(len(bandwidths)) if bandwidths[r] < bmax),
                   key=lambda r: (-ell[r], r))
    ring = [r for r in range(len(bandwidths)) if r not in strag]
    return ring, strag, ell


def _sections(q0, q1, parts, n):
    """Element ranges of `parts` sections over quanta [q0, q1), the first ones
    one quantum larger, clipped at n."""
    base, rem = divmod(q1 - q0, parts)
    out, q = [], q0
    for j in range(parts):
        sz = base + (1 if j < rem else 0)
        out.append((min(q * Q, n), min((q + sz) * Q, n)))
        q += sz
    return out


def final_values(dtype, x, bandwidths, k):
    """Every coordinate's final value for one GPU per server; x is [p, N]."""
    p, n = x.shape
    ring, strag, ell = _ranks(bandwidths)
    pp, m = len(ring), len(strag)
    nq = -(-n // Q)
    out = np.empty(n, dtype=x.dtype)
    for g in range(k):
        q0, q1 = g * nq // k, (g + 1) * nq // k
        lq = q1 - q0
        dq = 0
        if m == 1 and ell[strag[0]] < 2:
            el = ell[strag[0]]
            xq = (lq * (2 - el)) / ((p - 2) * el + 2)
            dq = min(max(int(np.floor(xq + 0.5)), 0), lq)
        for j, (a, b) in enumerate(_sections(q0, q1 - dq, pp, n)):
            if a >= b:
                continue
            chain = [ring[(j + t) % pp] for t in range(pp)]
            col = x[:, a:b]
            if m == 0:
                v = col[chain[0]]
            elif m == 1:
                v = col[chain[0]] if g % 4 in (0, 2) else _step(dtype, col[chain[0]], col[strag[0]])
            elif g % 4 in (0, 1):  # B, D
                v = _multi(dtype, col[chain[0]], [col[s] for s in strag])
            else:  # A', C': all but the worst straggler at the chain start
                v = _multi(dtype, col[chain[0]], [col[s] for s in strag[1:]])
            for r in chain[1:]:
                v = _step(dtype, col[r], v)
            if (m == 1 and g % 4 in (0, 2)) or (m >= 2 and g % 4 in (2, 3)):
                v = _step(dtype, col[strag[0]], v)
            out[a:b] = v
        if dq:
            a, b = min((q1 - dq) * Q, n), min(q1 * Q, n)
            if a < b:
                col = x[:, a:b]
                out[a:b] = _multi(dtype, col[strag[0]], [col[r] for r in ring])
    return out


def final_values_servers(dtype, x, q, gpus, server_bandwidths, k):
    """Every coordinate's final value for q servers of `gpus` GPUs each."""
    p, n = x.shape
    ring, strag, _ = _ranks(server_bandwidths)
    assert len(strag) == 1 and p == q * gpus
    s = strag[0]
    pp = len(ring)
    nq = -(-n // Q)
    out = np.empty(n, dtype=x.dtype)

    def collect(col, server, part):
        """The leader's sum: from local position g-1 down to 0."""
        pos = [server * gpus + (part + d) % gpus for d in range(gpus)]
        acc = col[pos[-1]]
        for r in reversed(pos[:-1]):
            acc = _step(dtype, col[r], acc)
        return acc

    for part in range(gpus):
        pq0, pq1 = part * nq // gpus, (part + 1) * nq // gpus
        plen = pq1 - pq0
        for c in range(k):
            q0, q1 = pq0 + c * plen // k, pq0 + (c + 1) * plen // k
            for j, (a, b) in enumerate(_sections(q0, q1, pp, n)):
                if a >= b:
                    continue
                col = x[:, a:b]
                chain = [ring[(j + t) % pp] for t in range(pp)]
                v = collect(col, chain[0], part)
                if c % 4 not in (0, 2):  # type 2: the straggler server's sum first
                    v = _step(dtype, collect(col, s, part), v)
                for h in chain[1:]:
                    v = _step(dtype, collect(col, h, part), v)
                if c % 4 in (0, 2):  # type 1: the straggler's ring, leader first
                    for d in range(gpus):
                        v = _step(dtype, col[s * gpus + (part + d) % gpus], v)
                out[a:b] = v
    return out
