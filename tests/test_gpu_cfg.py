"""Classifier-free guidance on the GPU against the oracle's guided sessions:
paired conditional / unconditional streams, guided logits l_u + w (l_c - l_u)
for every decision and the carry (Table "app_config" weights; w = 5 here).

Tiny fp32 decoder (2 layers, d=256, 1024 codes): verify rounds and commits
under rules A, B and C through ssd_verify_step, and whole images through
ssd_decode_image, decisions bit-exact.  2-layer decoder of the 1B widths
(bf16): a 24-token row under rules A and C.  Guided logits carry the streams'
errors times |w| + |1 - w| (9 at w = 5), so their tolerance is scaled by it.
"""
import dataclasses

import numpy as np
import pytest

import paper_2606_20543_amd as ssd
import synth
from oracle import decode as Dc
from oracle import schedule as S
from oracle import select as R
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

TINY = synth.TINY
P, H, W = 16, 8, 8
WEIGHT = 5.0


@pytest.fixture(scope="module")
def tiny():
    p = G.Pair(TINY, gain_std=0.1)
    yield p
    p.close()


def _prompts(shape, Bi, P_):
    """Conditional prompts over their unconditional twins (another seed)."""
    return np.concatenate([synth.prompt(shape, Bi, P_), synth.prompt(shape, Bi, P_, seed=7)])


def _sched(rule, top_k=0, b=2, cfg=1, weight=WEIGHT):
    s = ssd.ssd_schedule()
    s.grid_h, s.grid_w, s.k_h, s.h_rounds, s.k_v, s.b_rounds, s.i_rounds = H, W, 5, 1, 1, b, 0
    s.rule, s.top_k, s.temperature, s.seed = rule, top_k, 1.0, 3
    s.cfg, s.cfg_weight = cfg, weight
    return s


def _rounds(shape, pair, Bi, P_, blocks, rule, top_k=0):
    """Guided verify rounds (with explicit rule-C references) and commits, step by step."""
    pre = _prompts(shape, Bi, P_)
    sess = ssd.ssd_prefill(pair.model, 2 * Bi, P_, pre, P_ + 200, 32)
    ssd.ssd_session_set_cfg(sess, WEIGHT)
    os_ = Dc.prefill(pair.om, pre, P_ + 200, guide=WEIGHT)
    stats = {}
    rng = np.random.default_rng(21)
    rnd = 0
    try:
        for K, rounds in blocks:
            blk = rng.integers(0, shape.v_img, size=(Bi, K)).astype(np.int64)
            print(f"guided block K={K}, {rounds} rounds, rule {rule}", flush=True)
            for _ in range(rounds):
                ref = None
                if rule == R.RULE_ACCEPT_REJECT:
                    ref = (2.0 * rng.standard_normal((Bi, K, shape.v_img))).astype(np.float32)
                blk, _ = G.check_round(shape, sess, os_, blk, 0, rule, rnd, top_k, ref, stats)
                rnd += 1
            G.check_commit(shape, sess, os_, blk, stats, want_h=True)
        print("stats", stats, flush=True)
        assert stats["flips"] <= 0.02 * stats["positions"] + 1
        return stats
    finally:
        ssd.ssd_free_session(sess)


@pytest.mark.parametrize("rule,top_k", [(R.RULE_GREEDY, 0), (R.RULE_SAMPLE, 50), (R.RULE_ACCEPT_REJECT, 100)])
def test_guided_rounds_tiny(tiny, rule, top_k):
    stats = _rounds(TINY, tiny, 2, P, ((6, 1), (8, 2), (16, 2)), rule, top_k)
    if TINY.dtype == "f32":
        assert stats["flips"] == 0


@pytest.mark.parametrize("rule,top_k", [(R.RULE_GREEDY, 0), (R.RULE_ACCEPT_REJECT, 100)])
def test_guided_decode_image_tiny(tiny, rule, top_k):
    Bi = 2
    pre = _prompts(TINY, Bi, P)
    drafts = synth.random_codes(TINY, (Bi, H, W))
    out = np.zeros((Bi, H, W), np.int32)
    st = ssd.ssd_decode_image(tiny.model, _sched(rule, top_k), Bi, P, pre, (drafts + TINY.img_lo).astype(np.int32),
                              out)
    otok, ost = Dc.decode_image(tiny.om, pre, H, W, drafts, rule=rule, seed=3, top_k=top_k, b=2, guide=WEIGHT)
    assert np.array_equal(out - TINY.img_lo, otok)
    ops = S.plan(H, W, b=2)
    assert ost["passes"] == S.n_passes(ops) and st.passes == G.executed_passes(ops)
    assert st.accepted == ost["accepted"] and st.proposed == ost["proposed"]
    # the same images unguided differ (the weight matters for distinct prompts)
    out0 = np.zeros_like(out)
    ssd.ssd_decode_image(tiny.model, _sched(rule, top_k, cfg=0), Bi, P, pre[:Bi].copy(),
                         (drafts + TINY.img_lo).astype(np.int32), out0)
    assert not np.array_equal(out0, out)


def test_equal_prompts_make_the_weight_irrelevant(tiny):
    """Identical streams give l_c == l_u exactly, so any weight decodes the same image."""
    Bi = 2
    pc = synth.prompt(TINY, Bi, P)
    pre = np.concatenate([pc, pc])
    drafts = (synth.random_codes(TINY, (Bi, H, W)) + TINY.img_lo).astype(np.int32)
    outs = []
    for w in (5.0, 1.5):
        out = np.zeros((Bi, H, W), np.int32)
        ssd.ssd_decode_image(tiny.model, _sched(R.RULE_SAMPLE, 50, weight=w), Bi, P, pre, drafts, out)
        outs.append(out)
    assert np.array_equal(outs[0], outs[1])


def test_guidance_argument_errors(tiny):
    sess = ssd.ssd_prefill(tiny.model, 3, P, synth.prompt(TINY, 3, P), P + 32, 8)
    try:
        with pytest.raises(ssd.SSDError) as e:
            ssd.ssd_session_set_cfg(sess, WEIGHT)
        assert e.value.status == ssd.SSD_E_INVAL
    finally:
        ssd.ssd_free_session(sess)
    sess = ssd.ssd_prefill(tiny.model, 2, P, _prompts(TINY, 1, P), P + 32, 8)
    try:
        ssd.ssd_session_set_cfg(sess, WEIGHT)
        with pytest.raises(ssd.SSDError) as e:
            ssd.ssd_session_set_cfg(sess, float("nan"))
        assert e.value.status == ssd.SSD_E_INVAL
        tok = np.full((1, 4), TINY.img_lo, np.int32)
        with pytest.raises(ssd.SSDError) as e:
            ssd.ssd_verify_step(sess, 4, tok, G.vparams(truncate=1))
        assert e.value.status == ssd.SSD_E_INVAL
    finally:
        ssd.ssd_free_session(sess)


BF16 = dataclasses.replace(synth.M1B, n_layers=2)


@pytest.fixture(scope="module")
def wide():
    print("building 2-layer 1B-width model", flush=True)
    p = G.Pair(BF16)
    yield p
    p.close()


@pytest.mark.parametrize("rule,top_k", [(R.RULE_GREEDY, 0), (R.RULE_ACCEPT_REJECT, 2000)])
def test_guided_rounds_bf16(wide, rule, top_k):
    stats = _rounds(BF16, wide, 1, 40, ((24, 2), (5, 1)), rule, top_k)
    print("bf16 guided max logit error", stats["max_logit_err"], flush=True)
