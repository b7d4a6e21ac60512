"""The oracle's pins catch plausible mistakes (CPU only).

Each case plants one mistake in a copy of the oracle's C source (a wrong
holder index, Stage 2 as a copy, a dropped straggler fold, an allgather one
hop short, a point-to-point star missing a rank, the bubble-filling split
rounded the wrong way), builds it with the same flags, and checks that the
properties the paper fixes reject it: every rank ends with the exact int32
sum (Sec. 3), and the bubble-filling split of the Sec. 4.2 / App. C example
(golden fixture) with App. C's D rounded to the nearest whole quantum at
other lengths.  The unmodified copy passes the same checks, so the checks
are not failing for some other reason.  A second set plants mistakes in
the order of the additions, which exact sums cannot see, and requires the
bit-for-bit comparison with the closed form of the readings to reject them.
"""
import json
import os
import subprocess
from fractions import Fraction as F

import numpy as np
import pytest

import oracle
from oracle import model

GOLD = os.path.join(os.path.dirname(__file__), "golden")

# (name, text in the oracle's source, replacement)
MUTATIONS = [
    ("holder index",
     "int holder = ring_at(s, j, pp - 1);", "int holder = ring_at(s, j, pp - 2);"),
    ("Stage 2 as a copy",
     "rc |= push_step(s, 2, g, j, ORC_REDUCE, fin, one, 1, off, len);",
     "rc |= push_step(s, 2, g, j, ORC_COPY, fin, one, 1, off, len);"),
    ("straggler fold dropped",
     "if (npre > 0) rc |= push_step(s, 0,", "if (0) rc |= push_step(s, 0,"),
    ("allgather one hop short",
     "for (int t = 0; t <= pp - 2; ++t) {\n    one[0] = ring_at(s, j, t - 1);",
     "for (int t = 0; t <= pp - 3; ++t) {\n    one[0] = ring_at(s, j, t - 1);"),
    ("P2P star misses a rank",
     "push_step(s, 2, g, -1, ORC_REDUCE, st, s->ring, s->pp, off, len);",
     "push_step(s, 2, g, -1, ORC_REDUCE, st, s->ring, s->pp - 1, off, len);"),
    ("bubble split rounded down",
     "dq = (int64_t)floor(x + 0.5);", "dq = (int64_t)floor(x);"),
]

PROFILES = [(5, {0: 0.5}), (8, {7: 0.875}), (6, {0: 0.5, 5: 0.75}), (9, {0: 0.875, 3: 0.75, 8: 0.5})]


def _bw(p, slow):
    b = [1.0] * p
    for r, v in slow.items():
        b[r] = v
    return b


def _int32_sums_hold():
    """Sec. 3: every rank ends with the elementwise sum (int32 wraps exactly)."""
    for p, slow in PROFILES:
        for n, k in [(1000, 4), (64 * 41 + 7, 8)]:
            rng = np.random.default_rng(11 * p + n)
            x = rng.integers(-(2**31), 2**31, size=(p, n), dtype=np.int64).astype(np.int32)
            want = (x.astype(np.int64).sum(0) + 2**31) % 2**32 - 2**31
            y = oracle.run(oracle.Schedule(p, _bw(p, slow), n, k), "i32", x.copy())
            if not (y.astype(np.int64) == want[None, :]).all():
                return False
    return True


def _bubble_example_holds():
    """Sec. 4.2 / App. C at p = 5, l = 1.5, k = 4: P2P chunks of D = n/52 and
    sections of s' = 3n/52 when n is 52 quanta."""
    g = json.load(open(os.path.join(GOLD, "bubble_example_p5_l1.5.json")))
    p, k, ell = g["p"], g["k"], F(g["ell"])
    sp, d = model.bubble_split(p, ell, 1, k)
    n = 52 * 64
    s = oracle.Schedule(p, g["bandwidths"], n, k)
    for seg in range(k):
        if s.p2p_len[seg] != d * n:
            return False
        secs = {st["sec"]: st["len"] for st in s.steps() if st["seg"] == seg and st["sec"] >= 0}
        if set(secs.values()) != {sp * n}:
            return False
    # at other lengths each P2P chunk is App. C's D in whole quanta, rounded
    # to the nearest (within half a quantum of the real value)
    for p, b, k, lq in [(5, 2 / 3, 4, 11), (8, 0.875, 4, 10), (16, 0.75, 8, 23)]:
        bw = [1.0] * (p - 1) + [b]
        ell = 1 / F(b).limit_denominator(10**6)
        _, d = model.bubble_split(p, ell, 1, k)
        s = oracle.Schedule(p, bw, 64 * k * lq, k)
        for seg in range(k):
            if abs(F(s.p2p_len[seg], 64) - d * k * lq) > F(1, 2):
                return False
    return True


def _build(tmp_path, name, src):
    c = tmp_path / f"{name}.c"
    so = tmp_path / f"lib{name}.so"
    c.write_text(src)
    subprocess.run(["gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math", "-shared",
                    "-fPIC", "-o", str(so), str(c), "-lm"], check=True)
    return str(so)


def _checks_with(monkeypatch, so):
    monkeypatch.setattr(oracle, "_LIB", so)
    monkeypatch.setattr(oracle, "_lib", None)
    try:
        return _int32_sums_hold() and _bubble_example_holds()
    except oracle.OracleError:
        return False


@pytest.fixture(scope="module")
def source():
    return open(oracle._SRC).read()


def test_unmodified_copy_passes(tmp_path, monkeypatch, source):
    assert _checks_with(monkeypatch, _build(tmp_path, "control", source))


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_is_caught(tmp_path, monkeypatch, source, name, old, new):
    assert source.count(old) == 1, f"mutation site of {name!r} not found once"
    so = _build(tmp_path, "m" + str(abs(hash(name)) % 10**8), source.replace(old, new))
    assert not _checks_with(monkeypatch, so), f"{name}: not caught"


# ------------------------------------------------------- order of additions
# Planted mistakes that keep every sum exact in int32 but add in another
# order or round elsewhere: the exact sums cannot see them, the bit-for-bit
# comparison with the closed form of the readings (oracle/closed_form.py,
# tests/test_oracle_closed_form.py) must.
ASSOCIATION_MUTATIONS = [
    ("fp32 sources summed from the last",
     "float acc = b[st->dst][c];\n    for (int i = 0; i < st->nsrc; ++i) acc = acc + b[srcs[i]][c];",
     "float acc = b[st->dst][c];\n    for (int i = st->nsrc - 1; i >= 0; --i) acc = acc + b[srcs[i]][c];"),
    ("stragglers folded best first",
     "for (int i = 0; i < m; ++i) pre[npre++] = s->strag[i];",
     "for (int i = m - 1; i >= 0; --i) pre[npre++] = s->strag[i];"),
    ("bf16 rounded after every source",
     "for (int i = 0; i < st->nsrc; ++i) acc = acc + bf16_widen(b[srcs[i]][c]);",
     "for (int i = 0; i < st->nsrc; ++i) acc = bf16_widen(bf16_narrow(acc + bf16_widen(b[srcs[i]][c])));"),
    ("local ring the other way round",
     "return sv * s->g + (part + d) % s->g;",
     "return sv * s->g + (part + s->g - d) % s->g;"),
]

# ring; one straggler with l >= 2 and with l < 2 (P2P chunks); two and three
# stragglers; servers of 3 and 4 GPUs
ORDER_PROFILES = [(6, [1.0] * 6, 4), (5, [0.5, 1, 1, 1, 1], 8), (8, [1.0] * 7 + [0.875], 8),
                  (6, [0.5, 1, 1, 1, 1, 0.75], 8), (9, [0.875, 1, 1, 0.75, 1, 1, 1, 1, 0.5], 8)]
ORDER_SERVERS = [(4, 3, [1, 1, 0.5, 1], 24), (3, 4, [1, 0.25, 1], 24)]


def _closed_form_failures():
    """Profiles whose fp32 or bf16 results differ from the closed form."""
    from oracle import closed_form as cf
    bad = []
    for dtype in ("f32", "bf16"):
        for p, bw, k in ORDER_PROFILES:
            n = 64 * 3 * k * p + 17
            x = np.random.default_rng(p + k).standard_normal((p, n)).astype(np.float32)
            x = x if dtype == "f32" else oracle.bf16_round(x)
            got = oracle.run(oracle.Schedule(p, bw, n, k), dtype, x.copy())
            if not np.array_equal(got[0].view(np.uint8), cf.final_values(dtype, x, bw, k).view(np.uint8)):
                bad.append((dtype, p, bw))
        for q, g, bw, k in ORDER_SERVERS:
            n = 64 * 2 * k * g + 33
            x = np.random.default_rng(q * g).standard_normal((q * g, n)).astype(np.float32)
            x = x if dtype == "f32" else oracle.bf16_round(x)
            got = oracle.run(oracle.Schedule.servers(q, g, bw, n, k), dtype, x.copy())
            want = cf.final_values_servers(dtype, x, q, g, bw, k)
            if not np.array_equal(got[0].view(np.uint8), want.view(np.uint8)):
                bad.append((dtype, q, g, bw))
    return bad


def _order_checks_with(monkeypatch, so):
    """(exact int32 sums hold, closed-form failures) for the library `so`."""
    monkeypatch.setattr(oracle, "_LIB", so)
    monkeypatch.setattr(oracle, "_lib", None)
    return _int32_sums_hold(), _closed_form_failures()


def test_unmodified_copy_passes_the_order_pins(tmp_path, monkeypatch, source):
    ints, bad = _order_checks_with(monkeypatch, _build(tmp_path, "control_order", source))
    assert ints and bad == []


@pytest.mark.parametrize("name,old,new", ASSOCIATION_MUTATIONS,
                         ids=[m[0] for m in ASSOCIATION_MUTATIONS])
def test_planted_order_mistake_is_caught(tmp_path, monkeypatch, source, name, old, new):
    assert source.count(old) == 1, f"mutation site of {name!r} not found once"
    so = _build(tmp_path, "o" + str(abs(hash(name)) % 10**8), source.replace(old, new))
    ints, bad = _order_checks_with(monkeypatch, so)
    assert ints, f"{name}: the exact int32 sums should not see this mistake"
    assert bad, f"{name}: not caught"


# ---------------------------------------------------------------- time model
# Planted mistakes in a copy of oracle/model.py: each body count off by a
# fraction of a body, and the l < 2 branch without its head/tail term.  The
# hand-evaluated golden values at finite k (tests/golden/model_values.json)
# must reject every one.
MODEL_MUTATIONS = [
    ("App. D body count k+3", "return (k + 4) * body", "return (k + 3) * body"),
    ("App. E body count k+5", "(k + F(11, 2))", "(k + 5)"),
    ("Sec. 4.3 body count k", "ell * n * F(k + 1, k)", "ell * n"),
    ("App. C head/tail dropped", "* (k + ell - 1) / k", "* k / k"),
    ("App. D extra sections dropped", "(ells[0] * (p - m) + 2 * (m - 1)) * s",
     "(ells[0] * (p - m)) * s"),
]


def _model_copy(tmp_path, name, text):
    import importlib.util
    path = tmp_path / f"model_{name}.py"
    path.write_text(text)
    spec = importlib.util.spec_from_file_location(f"model_{name}", str(path))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_unmodified_model_copy_passes(tmp_path):
    from test_model_golden import model_failures
    text = open(model.__file__).read()
    assert model_failures(_model_copy(tmp_path, "control", text)) == []


@pytest.mark.parametrize("name,old,new", MODEL_MUTATIONS, ids=[m[0] for m in MODEL_MUTATIONS])
def test_planted_model_mistake_is_caught(tmp_path, name, old, new):
    from test_model_golden import model_failures
    text = open(model.__file__).read()
    assert text.count(old) == 1, f"mutation site of {name!r} not found once"
    mod = _model_copy(tmp_path, "m" + str(abs(hash(name)) % 10**8), text.replace(old, new))
    assert model_failures(mod), f"{name}: not caught"
