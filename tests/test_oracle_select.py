"""Pins of the oracle's correction rules (Sec. 3.3 "Verification as Auto Correction")
and of its counter-based uniform generator.

The accept/reject rule is pinned by the speculative-sampling identity: when the
draft is drawn from q, accepting with probability min(p/q, 1) and otherwise
drawing from [p - q]_+ yields exactly p.  The identity is checked by sweeping
the uniforms over a regular grid, so every branch of the oracle's own code is
exercised; a wrong ratio, a dropped max(0, .), a swapped p/q or an off-by-one
in the inverse CDF breaks it.
"""
import os

import numpy as np
import pytest

from oracle import select as R

GOLD = os.path.join(os.path.dirname(__file__), "golden", "splitmix64.txt")


def _published():
    out, seed = {}, None
    for line in open(GOLD):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        if line.startswith("seed"):
            seed = int(line.split()[1])
            out[seed] = []
        else:
            out[seed].append(int(line, 0))
    return out


def test_splitmix64_published_values():
    for seed, vals in _published().items():
        assert R.splitmix64_stream(seed, len(vals)) == vals


def test_uniform_is_stream_output():
    # u at counter c is output c+1 of the seeded stream, top 24 bits
    for seed in (0, 3, 1234567):
        for (b, pos, rnd, st) in [(0, 0, 0, 0), (0, 0, 0, 1), (1, 5, 2, 0), (3, 100, 0, 2)]:
            c = R.counter(b, pos, rnd, st)
            if c > 5000:
                continue
            z = R.splitmix64_stream(seed, c + 1)[-1]
            assert R.uniform(seed, b, pos, rnd, st) == (z >> 40) / float(1 << 24)


def test_uniform_counters_distinct_and_uniform():
    us = np.array([R.uniform(3, b, pos, r, s) for b in range(2) for pos in range(40) for r in range(5) for s in range(2)])
    assert len(np.unique(us)) == len(us)
    assert abs(us.mean() - 0.5) < 0.05
    assert np.all((us >= 0) & (us < 1))


def test_argmax_ties_lowest_id():
    assert R.argmax_lowest(np.array([0.0, 2.0, 1.0, 2.0])) == 1
    assert R.argmax_lowest(np.array([5.0, 5.0])) == 0


def test_warp_closed_forms():
    L = np.log(np.array([1.0, 2.0, 4.0]))
    assert np.allclose(R.warp(L), [1 / 7, 2 / 7, 4 / 7], rtol=0, atol=1e-15)
    # temperature 2: weights sqrt(1), sqrt(2), sqrt(4)
    w = np.array([1.0, np.sqrt(2.0), 2.0])
    assert np.allclose(R.warp(L, temperature=2.0), w / w.sum(), rtol=0, atol=1e-15)
    # top-2 keeps the two largest
    assert np.allclose(R.warp(L, top_k=2), [0, 1 / 3, 2 / 3], rtol=0, atol=1e-15)
    # boundary ties keep the lowest ids
    assert np.allclose(R.warp(np.array([1.0, 1.0, 1.0, 0.0]), top_k=2), [0.5, 0.5, 0, 0])
    assert np.allclose(R.warp(np.array([0.0, 1.0, 1.0, 1.0]), top_k=2), [0, 0.5, 0.5, 0])
    # top_k >= V is no truncation
    assert np.allclose(R.warp(L, top_k=3), R.warp(L))


def test_invcdf_boundaries():
    w = np.array([0.25, 0.25, 0.5])
    assert R.invcdf(w, 0.0) == 0
    assert R.invcdf(w, 0.2499) == 0
    assert R.invcdf(w, 0.25) == 1     # strict '>' at the boundary
    assert R.invcdf(w, 0.5) == 2
    assert R.invcdf(w, 0.999999) == 2
    z = np.array([0.0, 3.0, 0.0, 0.0])
    for u in (0.0, 0.5, 0.9999999):
        assert R.invcdf(z, u) == 1      # zero-weight ids are never drawn
    assert R.invcdf(np.array([0.2, 0.8, 0.0]), 0.9999999999) == 1


GRID = 1 << 13
UG = (np.arange(GRID) + 0.5) / GRID  # cell centres of a regular grid on [0, 1)


def _rule_distribution(rule, L, t, ref, T=1.0, top_k=0):
    """Exact output distribution of select_position at one position, from the
    uniform grid: u0 sweeps the accept test (u1 fixed), u1 sweeps the draw of a
    rejected or sampled position (u0 = 1 - tiny, so a rejection happens
    whenever alpha < 1)."""
    V = L.shape[0]
    dist = np.zeros(V)
    if rule == R.RULE_SAMPLE:
        for u1 in UG:
            a, _, _ = R.select_position(rule, L, t, ref, 0.0, u1, T, top_k)
            dist[a] += 1.0 / GRID
        return dist
    acc = 0
    for u0 in UG:
        a, ok, _ = R.select_position(rule, L, t, ref, u0, 0.5, T, top_k)
        acc += ok
    p_acc = acc / GRID
    dist[t] += p_acc
    if p_acc < 1.0:
        for u1 in UG:
            a, ok, repl = R.select_position(rule, L, t, ref, 1.0 - 1e-12, u1, T, top_k)
            assert not ok and repl
            dist[a] += (1.0 - p_acc) / GRID
    return dist


def test_accept_probability_closed_form():
    p = np.array([0.2, 0.3, 0.5])
    q = np.array([0.5, 0.3, 0.2])
    assert R.accept_prob(p, q, 0) == pytest.approx(0.4)
    assert R.accept_prob(p, q, 2) == 1.0
    assert R.accept_prob(p, np.array([0.0, 0.5, 0.5]), 0) == 1.0
    assert R.accept_prob(np.array([0.0, 1.0]), np.array([0.0, 1.0]), 0) == 0.0
    r = R.residual(p, q)
    assert np.allclose(r, [0.0, 0.0, 0.3])


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_speculative_sampling_identity(seed):
    rng = np.random.default_rng(seed)
    V = 5
    Lp = rng.normal(size=V) * 1.5
    Lq = rng.normal(size=V) * 1.5
    p, q = R.warp(Lp), R.warp(Lq)
    out = np.zeros(V)
    for t in range(V):
        out += q[t] * _rule_distribution(R.RULE_ACCEPT_REJECT, Lp, t, Lq)
    assert np.abs(out - p).max() < 4.0 / GRID


def test_point_mass_draft_gives_p():
    # a deterministic draft t with q = point mass: output ~ p for every t
    L = np.array([0.3, -1.0, 1.2, 0.1])
    p = R.warp(L)
    for t in range(4):
        d = _rule_distribution(R.RULE_ACCEPT_REJECT, L, t, None)
        assert np.abs(d - p).max() < 4.0 / GRID


def test_identity_with_temperature_and_topk():
    rng = np.random.default_rng(7)
    V, T, k = 6, 0.7, 4
    Lp, Lq = rng.normal(size=V), rng.normal(size=V)
    p, q = R.warp(Lp, T, k), R.warp(Lq, T, k)
    out = np.zeros(V)
    for t in range(V):
        if q[t] > 0:
            out += q[t] * _rule_distribution(R.RULE_ACCEPT_REJECT, Lp, t, Lq, T, k)
    assert np.abs(out - p).max() < 4.0 / GRID
    assert np.all(out[p == 0] == 0)


def test_sampling_rule_distribution():
    L = np.array([1.0, 0.0, 2.0, -0.5])
    d = _rule_distribution(R.RULE_SAMPLE, L, 0, None)
    assert np.abs(d - R.warp(L)).max() < 2.0 / GRID


def test_equal_reference_always_accepts():
    L = np.array([0.5, 1.5, -2.0])
    for t in range(3):
        for u0 in (0.0, 0.5, 0.999):
            a, ok, repl = R.select_position(R.RULE_ACCEPT_REJECT, L, t, L.copy(), u0, 0.3)
            assert ok and a == t and not repl


def test_greedy_rule():
    L = np.array([0.1, 0.9, 0.9, -3.0])
    assert R.select_position(R.RULE_GREEDY, L, 1, None, 0.5, 0.5) == (1, True, False)
    assert R.select_position(R.RULE_GREEDY, L, 3, None, 0.5, 0.5) == (1, False, False)


def test_first_token_sampling():
    L = np.array([0.0, 5.0, 1.0])
    assert R.sample_first(R.RULE_GREEDY, L, 0.9) == 1
    assert R.sample_first(R.RULE_SAMPLE, L, 0.0) == 0
    assert R.sample_first(R.RULE_ACCEPT_REJECT, L, 0.9999) == 2


def test_accept_is_strict_on_the_uniform_grid():
    """Keep the draft with probability alpha exactly: over the 2^24-point grid
    of uniforms, u < alpha holds for ceil(alpha * 2^24) of them, so a draft the
    backbone gives zero probability (alpha = 0) is never kept, even at u = 0,
    and one it gives at least q's mass (alpha = 1) always is."""
    L = np.array([2.0, 1.0, -1.0, 0.5])
    # t = 2 lies outside the top 2 codes: p(t) = 0 against a point-mass draft
    a, ok, repl = R.select_position(R.RULE_ACCEPT_REJECT, L, 2, None, 0.0, 0.25, 1.0, 2)
    assert not ok and repl and a != 2
    # q equal to p: alpha = 1 at the largest grid value
    a, ok, repl = R.select_position(R.RULE_ACCEPT_REJECT, L, 0, L.copy(), 1.0 - 2.0 ** -24, 0.25)
    assert ok and a == 0 and not repl


def test_counter_fields_do_not_overlap():
    """The counter packs (sequence, position, round, stream) into disjoint bit
    fields over their whole stated ranges: changing any one field at its
    lowest or highest value gives a different counter from changing any other."""
    hi = {"b": (1 << 20) - 1, "pos": (1 << 24) - 1, "rnd": (1 << 16) - 1, "stream": 15}
    seen = {}
    for f, top in hi.items():
        for v in (1, top, 1 << (top.bit_length() - 1)):
            args = {"b": 0, "pos": 0, "rnd": 0, "stream": 0}
            args[f] = v
            c = R.counter(**args)
            assert c not in seen, (f, v, seen.get(c))
            seen[c] = (f, v)
    # every field set to its highest value fills exactly 64 bits
    assert R.counter(**hi) == (1 << 64) - 1
