"""GPU parity on the tiny fp32 decoder (2 layers, d=256, 4x64 heads, MLP 688,
1024 image codes, 16-token prompt, 8x8 grid): the HIP path through the C ABI
against the oracle, logits within 1e-5 and every decision bit-exact."""
import numpy as np
import pytest

import paper_2606_20543_amd as ssd
import synth
from oracle import decode as Dc
from oracle import schedule as S
from oracle import select as R
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

SHAPE = synth.TINY
P, H, W = 16, 8, 8


@pytest.fixture(scope="module")
def pair():
    p = G.Pair(SHAPE, gain_std=0.1)
    yield p
    p.close()


def _sched(rule, b=2, top_k=0, seed=3, k_h=5, h_rounds=1, k_v=1, i=0):
    s = ssd.ssd_schedule()
    s.grid_h, s.grid_w, s.k_h, s.h_rounds, s.k_v, s.b_rounds, s.i_rounds = H, W, k_h, h_rounds, k_v, b, i
    s.rule, s.top_k, s.temperature, s.seed = rule, top_k, 1.0, seed
    return s


def test_prefill_carry(pair):
    pre = synth.prompt(SHAPE, 2, P)
    sess = ssd.ssd_prefill(pair.model, 2, P, pre, P + H * W, 16)
    try:
        carry = np.zeros((2, SHAPE.v_img), np.float32)
        ssd.ssd_get_carry(sess, carry)
        os_ = Dc.prefill(pair.om, pre, P + H * W)
        assert np.abs(carry - os_.carry).max() < G.TOL["f32"]
    finally:
        ssd.ssd_free_session(sess)


@pytest.mark.parametrize("rule,top_k", [(R.RULE_GREEDY, 0), (R.RULE_SAMPLE, 50), (R.RULE_ACCEPT_REJECT, 0),
                                        (R.RULE_ACCEPT_REJECT, 100)])
def test_verify_rounds_step_by_step(pair, rule, top_k):
    """Every op of the image plan through ssd_verify_step, side by side with the
    oracle: logits, tokens, accept flags, counts and frontiers."""
    B = 2
    pre = synth.prompt(SHAPE, B, P)
    ar = Dc.ar_decode(pair.om, pre, H * W)
    drafts = synth.plant(ar, 0.6, SHAPE.v_img).reshape(B, H * W)
    sess = ssd.ssd_prefill(pair.model, B, P, pre, P + H * W, 16)
    os_ = Dc.prefill(pair.om, pre, P + H * W)
    work = drafts.copy()
    refs = [dict() for _ in range(B)]
    try:
        for op in S.plan(H, W, b=2):
            if op[0] == "first":
                carry = np.zeros((B, SHAPE.v_img), np.float32)
                ssd.ssd_get_carry(sess, carry)
                for b in range(B):
                    work[b, 0] = R.sample_first(rule, os_.carry[b], R.uniform(3, b, P, 0, 2), 1.0, top_k)
                    assert work[b, 0] == R.sample_first(rule, carry[b].astype(np.float64),
                                                        R.uniform(3, b, P, 0, 2), 1.0, top_k)
            elif op[0] == "verify":
                _, start, K, nf, rnd = op
                blk = work[:, start:start + K]
                prm = G.vparams(rule, top_k=top_k, rnd=rnd, n_fixed=nf)
                f_before = os_.f.copy()
                carry = np.zeros((B, SHAPE.v_img), np.float32)
                ssd.ssd_get_carry(sess, carry)
                out = G.gpu_verify(sess, SHAPE, blk + SHAPE.img_lo, prm)
                ref = None
                if rule == R.RULE_ACCEPT_REJECT:
                    ref = [[refs[b].get(start + k) for k in range(K)] for b in range(B)]
                gnew, gacc, gcnt, _ = G.oracle_rule_on(out["logits"], carry, blk, nf, rule, rnd, 3, f_before,
                                                       1.0, top_k, ref)
                onew, oacc, ocnt, ologits = Dc.verify_round(os_, blk, nf, rule, rnd, 3, 1.0, top_k, ref)
                assert np.abs(out["logits"] - ologits).max() < G.TOL["f32"]
                # decision arithmetic parity on the GPU's own logits
                assert np.array_equal(out["tokens"] - SHAPE.img_lo, gnew)
                assert np.array_equal(out["accept"][:, nf:], gacc[:, nf:])
                assert np.array_equal(out["count"], gcnt)
                # end to end: no ambiguity at fp32
                assert np.array_equal(onew, gnew) and np.array_equal(oacc, gacc)
                assert list(out["frontier"]) == list(os_.f)
                if ref is not None:
                    for b in range(B):
                        for k in range(K):
                            refs[b][start + k] = ref[b][k]
                work[:, start:start + K] = onew
            elif op[0] == "commit":
                _, start, K = op
                blk = work[:, start:start + K]
                out = G.gpu_verify(sess, SHAPE, blk + SHAPE.img_lo, G.vparams(commit=1), want_h=True)
                ol, oh = Dc.commit(os_, blk)
                assert np.abs(out["logits"] - ol).max() < G.TOL["f32"]
                assert np.abs(out["h_pre"] - oh).max() < G.TOL["f32"] * 10
                assert list(out["frontier"]) == list(os_.f)
                for b in range(B):
                    for k in range(K):
                        refs[b].pop(start + k, None)
    finally:
        ssd.ssd_free_session(sess)


@pytest.mark.parametrize("rule,top_k,b", [(R.RULE_GREEDY, 0, 2), (R.RULE_ACCEPT_REJECT, 100, 2),
                                          (R.RULE_SAMPLE, 0, 1), (R.RULE_GREEDY, 0, 0)])
def test_decode_image_matches_oracle(pair, rule, top_k, b):
    B = 2
    pre = synth.prompt(SHAPE, B, P)
    ar = Dc.ar_decode(pair.om, pre, H * W).reshape(B, H, W)
    drafts = synth.plant(ar, 0.6, SHAPE.v_img)
    out = np.zeros((B, H, W), np.int32)
    st = ssd.ssd_decode_image(pair.model, _sched(rule, b=b, top_k=top_k), B, P, pre, (drafts + SHAPE.img_lo).astype(np.int32), out)
    otok, ost = Dc.decode_image(pair.om, pre, H, W, drafts, rule=rule, seed=3, top_k=top_k, b=b)
    assert np.array_equal(out - SHAPE.img_lo, otok)
    ops = S.plan(H, W, b=b)
    assert ost["passes"] == S.n_passes(ops) and st.passes == G.executed_passes(ops)
    assert st.accepted == ost["accepted"] and st.proposed == ost["proposed"]


def test_decode_image_staged_multirow(pair):
    B = 1
    pre = synth.prompt(SHAPE, B, P)
    drafts = synth.random_codes(SHAPE, (B, H, W))
    out = np.zeros((B, H, W), np.int32)
    st = ssd.ssd_decode_image(pair.model, _sched(R.RULE_GREEDY, b=3, k_v=3, i=2), B, P, pre,
                              (drafts + SHAPE.img_lo).astype(np.int32), out)
    otok, ost = Dc.decode_image(pair.om, pre, H, W, drafts, rule=R.RULE_GREEDY, b=3, k_v=3, i=2)
    assert np.array_equal(out - SHAPE.img_lo, otok)
    assert st.passes == G.executed_passes(S.plan(H, W, b=3, k_v=3, i=2))


def test_jacobi_greedy_reproduces_ar(pair):
    """r >= K greedy rounds per block reproduce greedy AR (GPU alone)."""
    B = 1
    pre = synth.prompt(SHAPE, B, P)
    ar = Dc.ar_decode(pair.om, pre, H * W).reshape(B, H, W)
    drafts = synth.random_codes(SHAPE, (B, H, W))
    out = np.zeros((B, H, W), np.int32)
    ssd.ssd_decode_image(pair.model, _sched(R.RULE_GREEDY, b=W, h_rounds=6), B, P, pre,
                         (drafts + SHAPE.img_lo).astype(np.int32), out)
    assert np.array_equal(out - SHAPE.img_lo, ar)


def test_truncate_mode_reproduces_ar(pair):
    """Strict greedy verification through the ABI: blocks start at the frontier
    with the carry's argmax as first token; result equals greedy AR."""
    B, N, K = 2, 40, 6
    pre = synth.prompt(SHAPE, B, P)
    ar = Dc.ar_decode(pair.om, pre, N)
    drafts = synth.plant(ar, 0.7, SHAPE.v_img)
    sess = ssd.ssd_prefill(pair.model, B, P, pre, P + 2 * N + 2 * K, K)
    try:
        done = np.zeros(B, int)
        out = np.full((B, N), -1)
        carry = np.zeros((B, SHAPE.v_img), np.float32)
        for _ in range(N + 1):
            if (done >= N).all():
                break
            ssd.ssd_get_carry(sess, carry)
            blk = np.zeros((B, K), np.int64)
            for b in range(B):
                d = min(done[b], N - 1)
                blk[b, 0] = int(np.argmax(carry[b]))
                for k in range(1, K):
                    blk[b, k] = drafts[b, min(d + k, N - 1)]
            res = G.gpu_verify(sess, SHAPE, blk + SHAPE.img_lo, G.vparams(truncate=1))
            for b in range(B):
                adv = int(res["frontier"][b]) - P - done[b]
                assert adv >= 1
                for k in range(adv):
                    if done[b] + k < N:
                        out[b, done[b] + k] = blk[b, k]
                done[b] += adv
        assert np.array_equal(out, ar)
    finally:
        ssd.ssd_free_session(sess)
