"""The time model pinned to values the paper's formulas fix (CPU only).

`tests/golden/model_values.json` holds completion times, body counts and
lower bounds evaluated by hand from the printed formulas at finite k: the
five headline workloads, the two examples of Sec. 4.2, a straggler-bound
case of App. D, and three server shapes of App. E.  The oracle's exact
rationals (`oracle/model.py`) must equal every one of them; so must the
library's fp64 model calls, to rounding.  Because the values are taken at
finite k, the body counts k+1 (Sec. 4.3), k+l-1 (App. C), k+4 (App. D) and
k+5.5 (App. E) are each pinned, not only their limits.
"""
import json
import os
from fractions import Fraction as F

import pytest

from oracle import model

GOLD = os.path.join(os.path.dirname(__file__), "golden", "model_values.json")


def golden():
    return json.load(open(GOLD))


def _bw_from_ells(p, ells):
    """Bandwidths 1/l for the stragglers (ranks p-m..p-1), 1 for the rest."""
    b = [F(1)] * p
    for i, e in enumerate(ells):
        b[p - len(ells) + i] = 1 / F(e)
    return b


def model_failures(mod):
    """Every golden value the model module `mod` does not reproduce exactly."""
    g = golden()
    bad = []

    def chk(name, what, got, want):
        if got != F(want):
            bad.append(f"{name}: {what} = {got}, golden {want}")

    for e in g["single"]:
        p, k, ell = e["p"], e["k"], F(e["ells"][0])
        bw = _bw_from_ells(p, e["ells"])
        chk(e["name"], "optcc_single", mod.optcc_single(p, ell, 1, k), e["optcc"])
        chk(e["name"], "optcc_time", mod.optcc_time(bw, 1, k), e["optcc"])
        chk(e["name"], "bodies x body", F(e["bodies"]) * F(e["body"]), e["optcc"])
        chk(e["name"], "t0", mod.t0(p, 1), e["t0"])
        chk(e["name"], "lower_bound", mod.lower_bound(bw, 1), e["lb_best"])
        chk(e["name"], "lb_tight_single", mod.lb_tight_single(p, ell, 1), e["lb_best"])
        chk(e["name"], "lb_weak_single", mod.lb_weak_single(p, ell, 1), e["lb_weak"])
        chk(e["name"], "degraded_ring", mod.degraded_ring(bw, 1), e["degraded_ring"])
        if "s_prime" in e:
            sp, d = mod.bubble_split(p, ell, 1, k)
            chk(e["name"], "s'", sp, e["s_prime"])
            chk(e["name"], "D", d, e["p2p_chunk"])
    for e in g["multi"]:
        p, k = e["p"], e["k"]
        ells = [F(x) for x in e["ells"]]
        bw = _bw_from_ells(p, e["ells"])
        chk(e["name"], "optcc_multi", mod.optcc_multi(p, ells, 1, k), e["optcc"])
        chk(e["name"], "optcc_time", mod.optcc_time(bw, 1, k), e["optcc"])
        chk(e["name"], "bodies x body", F(e["bodies"]) * F(e["body"]), e["optcc"])
        chk(e["name"], "t0", mod.t0(p, 1), e["t0"])
        chk(e["name"], "lower_bound", mod.lower_bound(bw, 1), e["lb_best"])
        chk(e["name"], "lb_multi", mod.lb_multi(p, ells, 1), e["lb_best"])
        chk(e["name"], "degraded_ring", mod.degraded_ring(bw, 1), e["degraded_ring"])
    for e in g["servers"]:
        q, gg, k, ell = e["q"], e["g"], e["k"], F(e["ell"])
        chk(e["name"], "optcc_servers", mod.optcc_servers(q, gg, ell, 1, k), e["optcc"])
        chk(e["name"], "bodies x body", F(e["bodies"]) * F(e["body"]), e["optcc"])
        chk(e["name"], "t0_servers", mod.t0_servers(q * gg, gg, 1), e["t0"])
        chk(e["name"], "lb_servers_tight", mod.lb_servers_tight(q, gg, ell, 1), e["lb_tight"])
        chk(e["name"], "lb_servers_weak", mod.lb_servers_weak(q, gg, ell, 1), e["lb_weak"])
    return bad


def test_oracle_model_equals_golden():
    assert model_failures(model) == []


def test_golden_body_counts():
    """The body counts themselves: k+1 (l >= 2), k+l-1 (l < 2), k+4 (m >= 2),
    k+11/2 (several GPUs per server)."""
    g = golden()
    for e in g["single"]:
        ell, k = F(e["ells"][0]), e["k"]
        assert F(e["bodies"]) == (k + 1 if ell >= 2 else k + ell - 1), e["name"]
    for e in g["multi"]:
        assert F(e["bodies"]) == e["k"] + 4, e["name"]
    for e in g["servers"]:
        assert F(e["bodies"]) == e["k"] + F(11, 2), e["name"]


@pytest.fixture(scope="module")
def o():
    from paper_2606_01680_amd import optcc
    return optcc


def _close(a, b):
    return abs(a - float(b)) <= 1e-12 * max(1.0, abs(float(b)))


def test_library_model_equals_golden(o):
    """The library's fp64 model calls (row a9) reproduce the same values; its
    plans need whole sections, so N is a multiple of every denominator."""
    g = golden()
    n = 1 << 22
    for e in g["single"] + g["multi"]:
        p, k = e["p"], e["k"]
        bw = [float(x) for x in _bw_from_ells(p, e["ells"])]
        plan = o.optcc_plan(p, bw, n, k)
        assert _close(o.optcc_model_time(plan) / n, F(e["optcc"])), e["name"]
        assert _close(o.optcc_lower_bound(p, bw, n) / n, F(e["lb_best"])), e["name"]
    for e in g["servers"]:
        q, gg, k = e["q"], e["g"], e["k"]
        bw = [1.0] * q
        bw[-1] = float(1 / F(e["ell"]))
        plan = o.optcc_plan_servers(q, gg, bw, n, k)
        assert _close(o.optcc_model_time(plan) / n, F(e["optcc"])), e["name"]
        assert _close(o.optcc_lower_bound_servers(q, gg, bw, n) / n, F(e["lb_tight"])), e["name"]
