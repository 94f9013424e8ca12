"""Failure paths of the C ABI on a real session (the contract of include/ssd.h:
validation happens before any launch and a refused call leaves the session
unchanged; a device failure poisons the object, and every later call on it is
refused with SSD_E_STATE).

* SSD_E_CAPACITY: a block running past max_ctx;
* SSD_E_INVAL: a block token outside the image codes, a block longer than the
  session's max_block, guidance on an odd batch;
* SSD_E_OOM: a session whose KV cache cannot be allocated (absurd max_ctx and
  batch); the model stays usable;
* SSD_E_DEVICE then SSD_E_STATE: the single-launch forward pass with its
  dependency waits bounded to zero polls (set from the host at model creation),
  so a wait gives up, the grid drains through the abandon path and the host
  reports the failure at its synchronization -- every kernel exits normally.
After each refused call the frontier and the carry are bit-identical to before
and the next valid call gives the same result as on an untouched twin session.
"""
import dataclasses
import os

import numpy as np
import pytest

import paper_2606_20543_amd as ssd
import synth
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

SHAPE = dataclasses.replace(synth.M1B, n_layers=2)
P = 16


@pytest.fixture(scope="module")
def pair():
    print("errors: 2-layer 1B-width model", flush=True)
    p = G.Pair(SHAPE, oracle=False)
    yield p
    p.close()


def _state(sess, B):
    carry = np.zeros((B, SHAPE.v_img), np.float32)
    ssd.ssd_get_carry(sess, carry)
    tok = np.full((B, 1), SHAPE.img_lo, np.int32)
    fr = np.zeros(B, np.int32)
    lg = np.zeros((B, 1, SHAPE.v_img), np.float32)
    ssd.ssd_verify_step(sess, 1, tok, G.vparams(), frontier=fr, logits_out=lg)  # frontier unchanged by a round
    return carry, fr, lg


def _expect(status, fn, *a, **k):
    with pytest.raises(ssd.SSDError) as e:
        fn(*a, **k)
    assert e.value.status == status, (e.value.status, ssd.ssd_last_error())
    return ssd.ssd_last_error()


def test_refused_calls_leave_the_session_unchanged(pair):
    B, K = 2, 6
    pre = synth.prompt(SHAPE, B, P)
    max_ctx = P + 10
    sess = ssd.ssd_prefill(pair.model, B, P, pre, max_ctx, 8)
    twin = ssd.ssd_prefill(pair.model, B, P, pre, max_ctx, 8)
    try:
        blk = (synth.random_codes(SHAPE, (B, K), stream=3) + SHAPE.img_lo).astype(np.int32)
        for s_ in (sess, twin):
            ssd.ssd_verify_step(s_, K, blk.copy(), G.vparams(commit=1))  # f = P + 6
        before = _state(sess, B)
        # past max_ctx: [P+6, P+12) > P+10
        big = (synth.random_codes(SHAPE, (B, 6), stream=4) + SHAPE.img_lo).astype(np.int32)
        msg = _expect(ssd.SSD_E_CAPACITY, ssd.ssd_verify_step, sess, 6, big.copy(), G.vparams())
        assert "max_ctx" in msg
        _expect(ssd.SSD_E_CAPACITY, ssd.ssd_verify_step, sess, 6, big.copy(), G.vparams(commit=1))
        # a token outside the image codes, a block longer than max_block, a bad rule
        bad = big[:, :2].copy()
        bad[1, 1] = SHAPE.img_lo - 1
        _expect(ssd.SSD_E_INVAL, ssd.ssd_verify_step, sess, 2, bad, G.vparams())
        _expect(ssd.SSD_E_INVAL, ssd.ssd_verify_step, sess, 9, np.zeros((B, 9), np.int32) + SHAPE.img_lo,
                G.vparams())
        _expect(ssd.SSD_E_INVAL, ssd.ssd_verify_step, sess, 2, big[:, :2].copy(), G.vparams(rule=7))
        after = _state(sess, B)
        for a, b in zip(before, after):
            assert np.array_equal(a, b)
        assert list(after[1]) == [P + K] * B
        # the next valid call equals the twin's
        nxt = big[:, :4].copy()
        out_s = G.gpu_verify(sess, SHAPE, nxt.copy(), G.vparams(rnd=1))
        _state(twin, B)
        out_t = G.gpu_verify(twin, SHAPE, nxt.copy(), G.vparams(rnd=1))
        assert np.array_equal(out_s["tokens"], out_t["tokens"])
        assert np.array_equal(out_s["logits"], out_t["logits"])
    finally:
        ssd.ssd_free_session(sess)
        ssd.ssd_free_session(twin)


def test_guidance_needs_an_even_batch(pair):
    pre = synth.prompt(SHAPE, 3, P)
    sess = ssd.ssd_prefill(pair.model, 3, P, pre, P + 8, 4)
    try:
        _expect(ssd.SSD_E_INVAL, ssd.ssd_session_set_cfg, sess, 5.0)
        carry, fr, _ = _state(sess, 3)
        assert list(fr) == [P] * 3
    finally:
        ssd.ssd_free_session(sess)


def test_out_of_memory_session_is_refused(pair):
    # a KV cache of 8192 sequences x 4096 positions x 16 KiB (2 layers of 16 KV heads
    # of 128, K and V in bf16): 512 GiB, beyond the GPU's 288 GB
    B = 8192
    pre = np.zeros((B, 1), np.int32)
    msg = _expect(ssd.SSD_E_OOM, ssd.ssd_prefill, pair.model, B, 1, pre, 4096, 1)
    assert "allocation" in msg
    # the model is still usable
    p2 = synth.prompt(SHAPE, 1, P)
    sess = ssd.ssd_prefill(pair.model, 1, P, p2, P + 4, 4)
    ssd.ssd_free_session(sess)


def test_abandoned_wait_poisons_the_session():
    saved = {k: os.environ.get(k) for k in ("SSD_FORWARD", "SSD_FWD_SPIN_LIMIT")}
    os.environ["SSD_FORWARD"] = "persistent"
    os.environ["SSD_FWD_SPIN_LIMIT"] = "0"
    try:
        print("errors: persistent pass with zero-poll waits", flush=True)
        p = G.Pair(SHAPE, oracle=False)
    finally:
        for k, v in saved.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
    try:
        # the prefix pass (48 rows) runs per kernel; blocks of at most 32 rows take the single launch
        B, P2 = 2, 24
        pre = synth.prompt(SHAPE, B, P2)
        sess = ssd.ssd_prefill(p.model, B, P2, pre, P2 + 16, 8)
        try:
            blk = (synth.random_codes(SHAPE, (B, 8), stream=5) + SHAPE.img_lo).astype(np.int32)
            msg = _expect(ssd.SSD_E_DEVICE, ssd.ssd_verify_step, sess, 8, blk.copy(), G.vparams(),
                          frontier=np.zeros(B, np.int32))
            assert "abandoned" in msg
            _expect(ssd.SSD_E_STATE, ssd.ssd_verify_step, sess, 8, blk.copy(), G.vparams())
            _expect(ssd.SSD_E_STATE, ssd.ssd_verify_step, sess, 2, blk[:, :2].copy(), G.vparams(commit=1))
        finally:
            ssd.ssd_free_session(sess)
    finally:
        p.close()
