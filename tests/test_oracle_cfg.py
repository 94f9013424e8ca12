"""Pins of the oracle's classifier-free guidance (the backbones decode with it:
Table "app_config" CFG weights; the logit mix of Ho & Salimans).

Every pin compares a guided session with unguided sessions of the same
streams, which share none of the guidance code: weight 1 must decode exactly
like the conditional prompts alone and weight 0 like the unconditional ones,
equal prompts must make the weight irrelevant, the guided logits of a verify
pass and of the carry must be the affine combination of the two streams' own
logits, each image must pair with its own twin, and the commit must return
the conditional stream's hidden states.
"""
import numpy as np
import pytest

from oracle import decode as Dc
from oracle import model as M
from oracle import schedule as S
from oracle import select as R
from tests import oracle_util as U

SHAPE = U.TINY_GQA  # fp32, d = 32, GQA 4/2, text ids [0, 8), 32 image codes
H = W = 4


def _model():
    return U.model(SHAPE, U.packed(SHAPE))


def _prompts(Bi, P, seed):
    rng = np.random.default_rng(seed)
    return rng.integers(0, SHAPE.img_lo, size=(Bi, P))


def _drafts(Bi, seed=9):
    return np.random.default_rng(seed).integers(0, SHAPE.v_img, size=(Bi, H, W))


def _decode(model, prefix, drafts, rule, guide=None, trace=None):
    return Dc.decode_image(model, prefix, H, W, drafts, rule=rule, seed=3, k_h=2, b=2, trace=trace, guide=guide)


@pytest.mark.parametrize("rule", [R.RULE_GREEDY, R.RULE_SAMPLE, R.RULE_ACCEPT_REJECT])
def test_weight_one_is_the_conditional_decode(rule):
    model = _model()
    pc, pu = _prompts(2, 5, 1), _prompts(2, 5, 2)
    dr = _drafts(2)
    tg, tr_g = [], []
    got, st_g = _decode(model, np.concatenate([pc, pu]), dr, rule, guide=1.0, trace=tr_g)
    want, st_w = _decode(model, pc, dr, rule, trace=tg)
    assert np.array_equal(got, want)
    assert st_g == st_w
    for a, b in zip(tr_g, tg):
        assert np.allclose(a[3], b[3], rtol=1e-12, atol=1e-12)  # guided logits = conditional logits


@pytest.mark.parametrize("rule", [R.RULE_GREEDY, R.RULE_ACCEPT_REJECT])
def test_weight_zero_is_the_unconditional_decode(rule):
    model = _model()
    pc, pu = _prompts(2, 5, 1), _prompts(2, 5, 2)
    dr = _drafts(2)
    got, st_g = _decode(model, np.concatenate([pc, pu]), dr, rule, guide=0.0)
    want, st_w = _decode(model, pu, dr, rule)
    assert np.array_equal(got, want)
    assert st_g == st_w


def test_equal_prompts_make_the_weight_irrelevant():
    model = _model()
    pc = _prompts(2, 6, 4)
    dr = _drafts(2)
    want, _ = _decode(model, pc, dr, R.RULE_SAMPLE)
    for w in (3.0, 5.0):
        got, _ = _decode(model, np.concatenate([pc, pc]), dr, R.RULE_SAMPLE, guide=w)
        assert np.array_equal(got, want)


def test_guided_logits_are_affine_in_the_weight():
    """A guided verify pass and its carry against two unguided sessions fed the same
    blocks: l = l_u + w (l_c - l_u) with the streams' own logits."""
    model = _model()
    pc, pu = _prompts(2, 5, 1), _prompts(2, 5, 2)
    w = 3.0
    g = Dc.prefill(model, np.concatenate([pc, pu]), 40, guide=w)
    c = Dc.prefill(model, pc, 40)
    u = Dc.prefill(model, pu, 40)
    for b in range(2):
        assert np.allclose(Dc.carry_of(g, b), w * c.carry[b] - (w - 1) * u.carry[b], rtol=1e-12, atol=1e-12)
    rng = np.random.default_rng(7)
    blk = rng.integers(0, SHAPE.v_img, size=(2, 6))
    _, _, _, lg = Dc.verify_round(g, blk, 0, R.RULE_GREEDY, 0)
    lc, _ = M.forward(model, c.cache, blk + SHAPE.img_lo, c.f)
    lu, _ = M.forward(model, u.cache, blk + SHAPE.img_lo, u.f)
    assert np.allclose(lg, w * lc - (w - 1) * lu, rtol=1e-11, atol=1e-11)
    # greedy corrections follow the guided scores, not the conditional ones
    new, _, _, _ = Dc.verify_round(g, blk, 0, R.RULE_GREEDY, 1)
    for b in range(2):
        assert new[b, 0] == R.argmax_lowest(w * c.carry[b] - (w - 1) * u.carry[b])
        for k in range(1, 6):
            assert new[b, k] == R.argmax_lowest(w * lc[b, k - 1] - (w - 1) * lu[b, k - 1])
    # the commit advances both streams and returns the conditional stream's states
    lg_c, hp = Dc.commit(g, new)
    lc2, hc = M.forward(model, c.cache, new + SHAPE.img_lo, c.f)
    lu2, _ = M.forward(model, u.cache, new + SHAPE.img_lo, u.f)
    assert np.allclose(hp, hc, rtol=1e-12, atol=1e-12)
    assert np.allclose(lg_c, w * lc2 - (w - 1) * lu2, rtol=1e-11, atol=1e-11)
    assert list(g.f) == [5 + 6] * 4


def test_images_pair_with_their_own_twins():
    """Greedy (no uniforms): an image decoded in a guided batch of two equals the
    same image decoded alone with its own prompt pair."""
    model = _model()
    pc, pu = _prompts(2, 5, 11), _prompts(2, 5, 12)
    dr = _drafts(2, seed=13)
    both, st = _decode(model, np.concatenate([pc, pu]), dr, R.RULE_GREEDY, guide=4.0)
    for b in range(2):
        one, _ = _decode(model, np.stack([pc[b], pu[b]]), dr[b:b + 1], R.RULE_GREEDY, guide=4.0)
        assert np.array_equal(both[b], one[0])
    ops = S.plan(H, W, k_h=2, h_rounds=1, k_v=1, b=2, i=0)
    assert st["passes"] == S.n_passes(ops)
    # guidance changes the image (the weight matters when the prompts differ)
    plain, _ = _decode(model, pc, dr, R.RULE_GREEDY)
    assert not np.array_equal(both, plain)
