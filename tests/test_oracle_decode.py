"""Pins of the oracle's verify / commit / decode logic (Sec. 3.3 "Verification as
Auto Correction"; Eq. 1 for the sequential reference).

* Strict truncation at the first mismatch is exact speculative decoding: it
  must reproduce greedy AR decoding token for token whatever the drafts are.
* Greedy correction rounds are Jacobi iterations: after j rounds the first j
  block positions equal greedy AR, so r >= K rounds per block reproduce AR.
* Drafts equal to the backbone's own argmax are all accepted in round one.
* Brute force: on a 4x4 grid with a 2-code image vocabulary, every possible
  draft row gives verify logits equal to independent full forwards of the
  corresponding sequences.
"""
import itertools

import numpy as np
import pytest

import synth
from oracle import decode as Dc
from oracle import model as M
from oracle import schedule as S
from oracle import select as R
from tests import oracle_util as U


def _setup(shape=U.TINY_GQA, seed=0):
    buf = U.packed(shape, seed=seed)
    return U.model(shape, buf)


@pytest.mark.parametrize("shape", [U.TINY_GQA, U.TINY_BF16], ids=["f32", "bf16"])
@pytest.mark.parametrize("p", [0.0, 0.5, 1.0])
def test_truncation_reproduces_greedy_ar(shape, p):
    mod = _setup(shape)
    pre = synth.prompt(shape, 2, 6)
    ar = Dc.ar_decode(mod, pre, 20)
    drafts = synth.plant(ar, p, shape.v_img)
    for K in (2, 5):
        out, passes = Dc.decode_truncate(mod, pre, drafts, K)
        assert np.array_equal(out, ar)
        if p == 1.0:
            # every draft accepted: a block of K settles K tokens (K-1 drafts plus
            # the bonus token); ceil((N - 1) / K) verify passes + prefill per sequence
            assert passes == 2 * (1 + int(np.ceil(19 / K)))


@pytest.mark.parametrize("shape", [U.TINY_GQA, U.TINY_BF16], ids=["f32", "bf16"])
def test_jacobi_rounds_reproduce_greedy_ar(shape):
    mod = _setup(shape)
    H = W = 5
    pre = synth.prompt(shape, 2, 6)
    ar = Dc.ar_decode(mod, pre, H * W).reshape(2, H, W)
    drafts = synth.plant(ar, 0.3, shape.v_img)
    out, st = Dc.decode_image(mod, pre, H, W, drafts, rule=R.RULE_GREEDY, k_h=5, h_rounds=6, b=W)
    assert np.array_equal(out, ar)
    assert st["passes"] == S.n_passes(S.plan(H, W, k_h=5, h_rounds=6, b=W))


def test_jacobi_prefix_property():
    """After j greedy rounds on a block, its first j positions equal greedy AR."""
    mod = _setup()
    pre = synth.prompt(U.TINY_GQA, 1, 5)
    ar = Dc.ar_decode(mod, pre, 9)
    s = Dc.prefill(mod, pre, 5 + 9)
    blk = synth.random_codes(U.TINY_GQA, (1, 9))
    for j in range(1, 10):
        blk, _, _, _ = Dc.verify_round(s, blk, 0, R.RULE_GREEDY, j)
        assert np.array_equal(blk[0, :j], ar[0, :j])
        assert int(s.f[0]) == 5


def test_planted_argmax_drafts_all_accepted():
    """Drafts built left to right from the backbone's own argmax are all
    accepted by a greedy round (the planted-acceptance recipe at p = 1)."""
    mod = _setup()
    pre = synth.prompt(U.TINY_GQA, 1, 5)
    s = Dc.prefill(mod, pre, 5 + 8)
    ar = Dc.ar_decode(mod, pre, 8)
    new, acc, cnt, _ = Dc.verify_round(s, ar, 0, R.RULE_GREEDY, 0)
    assert acc.all() and cnt[0] == 8 and np.array_equal(new, ar)


def test_verify_keeps_frontier_commit_advances():
    mod = _setup()
    pre = synth.prompt(U.TINY_GQA, 2, 4)
    s = Dc.prefill(mod, pre, 4 + 10)
    assert list(s.f) == [4, 4]
    blk = synth.random_codes(U.TINY_GQA, (2, 6))
    Dc.verify_round(s, blk, 0, R.RULE_GREEDY, 0)
    assert list(s.f) == [4, 4]
    logits, _ = Dc.commit(s, blk)
    assert list(s.f) == [10, 10]
    assert np.array_equal(s.carry, logits[:, -1])
    # the carry equals a fresh forward's prediction at the last committed position
    full = np.concatenate([pre, blk + U.TINY_GQA.img_lo], axis=1)
    lf, hf = M.forward_nocache(mod, full)
    assert np.allclose(s.carry, lf[:, -1], rtol=0, atol=1e-12)
    # and the carried state is that position's pre-norm state (the one that scored the carry)
    assert np.allclose(s.h_carry, hf[:, -1], rtol=0, atol=1e-12)


def test_verify_uniforms_at_absolute_positions():
    """Rule (B) at block position k of sequence b takes the sampling uniform of
    the counter (b, f + k, round, stream 1): the raster position, not the
    block offset, so that blocks starting elsewhere draw other numbers."""
    mod = _setup()
    pre = synth.prompt(U.TINY_GQA, 2, 4)
    s = Dc.prefill(mod, pre, 4 + 12)
    blk0 = synth.random_codes(U.TINY_GQA, (2, 4))
    Dc.commit(s, blk0)
    blk = synth.random_codes(U.TINY_GQA, (2, 5))
    seed, rnd = 11, 3
    carry = s.carry.copy()
    new, _, _, logits = Dc.verify_round(s, blk, 0, R.RULE_SAMPLE, rnd, seed)
    for b in range(2):
        for k in range(5):
            L = carry[b] if k == 0 else logits[b, k - 1]
            u1 = R.uniform(seed, b, 8 + k, rnd, 1)
            assert new[b, k] == R.invcdf(R.warp(L), u1), (b, k)
    # rule (C) against a point-mass draft keeps t exactly when the accept
    # uniform of stream 0 at (b, f + k, round) lies below p(t); the drafts are
    # the greedy continuation and the temperatures low, so p(t) spreads over
    # (0, 1) and both outcomes occur
    ar = Dc.ar_decode(mod, np.concatenate([pre, blk0 + U.TINY_GQA.img_lo], axis=1), 5)
    seen = set()
    for T in (0.005, 0.01, 0.02, 0.05):
        s2 = Dc.prefill(mod, pre, 4 + 12)
        Dc.commit(s2, blk0)
        carry = s2.carry.copy()
        _, acc, _, logits = Dc.verify_round(s2, ar, 0, R.RULE_ACCEPT_REJECT, rnd, seed, T)
        for b in range(2):
            for k in range(5):
                L = carry[b] if k == 0 else logits[b, k - 1]
                u0 = R.uniform(seed, b, 8 + k, rnd, 0)
                assert acc[b, k] == (u0 < R.warp(L, T)[ar[b, k]]), (T, b, k)
                seen.add(bool(acc[b, k]))
    assert seen == {True, False}


def test_first_token_uses_stream_two():
    """The first image token (no draft) is a plain sample of the prefill's
    last logits with the uniform of counter (b, P, round 0, stream 2)."""
    mod = _setup()
    P = 4
    pre = synth.prompt(U.TINY_GQA, 2, P)
    carry = Dc.prefill(mod, pre, P + 9).carry
    drafts = synth.random_codes(U.TINY_GQA, (2, 3, 3))
    seed = 5
    out, _ = Dc.decode_image(mod, pre, 3, 3, drafts, rule=R.RULE_SAMPLE, seed=seed)
    for b in range(2):
        assert out[b, 0, 0] == R.invcdf(R.warp(carry[b]), R.uniform(seed, b, P, 0, 2))


def test_rule_c_same_reference_accepts_everything():
    """When the reference logits equal the scoring logits, alpha = 1 everywhere."""
    mod = _setup()
    pre = synth.prompt(U.TINY_GQA, 1, 5)
    s = Dc.prefill(mod, pre, 5 + 6)
    blk = synth.random_codes(U.TINY_GQA, (1, 6))
    logits, _ = M.forward(mod, s.cache.copy(), blk + U.TINY_GQA.img_lo, s.f)
    ref = [[s.carry[0]] + [logits[0, k - 1] for k in range(1, 6)]]
    new, acc, cnt, _ = Dc.verify_round(s, blk, 0, R.RULE_ACCEPT_REJECT, 0, seed=3, ref=ref)
    assert acc.all() and np.array_equal(new, blk)


def test_rule_c_rejection_replaces_reference():
    mod = _setup()
    pre = synth.prompt(U.TINY_GQA, 1, 5)
    s = Dc.prefill(mod, pre, 5 + 6)
    blk = synth.random_codes(U.TINY_GQA, (1, 6))
    ref = [[None] * 6]
    new, acc, cnt, logits = Dc.verify_round(s, blk, 0, R.RULE_ACCEPT_REJECT, 0, seed=3, ref=ref)
    for k in range(6):
        if acc[0, k]:
            assert ref[0][k] is None and new[0, k] == blk[0, k]
        else:
            want = s.carry[0] if k == 0 else logits[0, k - 1]
            assert np.array_equal(ref[0][k], want)
    assert cnt[0] == acc.sum()


def test_bruteforce_4x4_verify_equals_full_forwards():
    """4x4 grid, 2 image codes: for every draft of row 1 (2^4), each verify logit
    equals the last logit of an independent full forward of that sequence."""
    shape = synth.ModelShape(1, 16, 2, 1, 8, 24, 6, 2, "f32")
    mod = _setup(shape)
    pre = synth.prompt(shape, 1, 3)
    row0 = np.array([[1, 0, 1, 1]])
    s = Dc.prefill(mod, pre, 3 + 16)
    Dc.commit(s, row0)
    base = np.concatenate([pre, row0 + shape.img_lo], axis=1)
    for draft in itertools.product(range(2), repeat=4):
        d = np.array([draft])
        c = s.cache.copy()
        lv, _ = M.forward(mod, c, d + shape.img_lo, s.f)
        for k in range(4):
            seq = np.concatenate([base, d[:, :k + 1] + shape.img_lo], axis=1)
            lf, _ = M.forward_nocache(mod, seq)
            assert np.allclose(lv[0, k], lf[0, -1], rtol=0, atol=1e-12)


def test_decode_image_rule_c_runs_and_counts():
    mod = _setup()
    H, W = 4, 6
    pre = synth.prompt(U.TINY_GQA, 2, 5)
    drafts = synth.random_codes(U.TINY_GQA, (2, H, W))
    out, st = Dc.decode_image(mod, pre, H, W, drafts, rule=R.RULE_ACCEPT_REJECT, seed=3, top_k=10, b=2)
    assert out.shape == (2, H, W)
    assert st["passes"] == S.n_passes(S.plan(H, W, b=2))
    assert 0 <= st["accepted"] <= st["proposed"]
    # deterministic in the seed
    out2, st2 = Dc.decode_image(mod, pre, H, W, drafts, rule=R.RULE_ACCEPT_REJECT, seed=3, top_k=10, b=2)
    assert np.array_equal(out, out2) and st == st2
    # another sampling seed gives another image
    out3, _ = Dc.decode_image(mod, pre, H, W, drafts, rule=R.RULE_ACCEPT_REJECT, seed=4, top_k=10, b=2)
    assert not np.array_equal(out, out3)
