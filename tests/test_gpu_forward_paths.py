"""Both forward-pass paths of bf16 models against the oracle: the single
cooperative launch that runs the whole backbone for blocks of up to 32 tokens,
and the one-launch-per-projection path (SSD_FORWARD at model creation picks
one), on a 2-layer decoder of the 1B widths (d=2048, 16x128 heads, MLP 5632,
16384 image codes).  Two sequences; blocks of 1, 9, 16 and 8 tokens (2 to 32 rows: one and
two 16-token tiles); verify rounds and commits, the commits both with logits
for every row and with the last row only (the image decoder's commit)."""
import dataclasses
import os

import numpy as np
import pytest

import paper_2606_20543_amd as ssd
import synth
from oracle import decode as Dc
from oracle import select as R
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

SHAPE = dataclasses.replace(synth.M1B, n_layers=2)
TOL = G.TOL["bf16"]


@pytest.fixture(scope="module", params=["persistent", "kernels"])
def pair(request):
    old = os.environ.get("SSD_FORWARD")
    os.environ["SSD_FORWARD"] = request.param
    try:
        print(f"building 2-layer 1B-width model ({request.param} forward)", flush=True)
        p = G.Pair(SHAPE)
    finally:
        if old is None:
            os.environ.pop("SSD_FORWARD", None)
        else:
            os.environ["SSD_FORWARD"] = old
    p.path = request.param
    yield p
    p.close()


def _commit_last_row(sess, os_, blk, stats):
    """Commit without a logits output: the library computes the last row of
    each sequence only; its carry must match the oracle's."""
    B, K = blk.shape
    tok = np.ascontiguousarray((blk + SHAPE.img_lo).astype(np.int32))
    fr = np.zeros(B, np.int32)
    ssd.ssd_verify_step(sess, K, tok, G.vparams(commit=1), frontier=fr)
    Dc.commit(os_, blk)
    carry = np.zeros((B, SHAPE.v_img), np.float32)
    ssd.ssd_get_carry(sess, carry)
    err = float(np.abs(carry - os_.carry).max())
    stats["max_logit_err"] = max(stats.get("max_logit_err", 0.0), err)
    assert err < TOL, f"carry error {err}"
    assert list(fr) == list(os_.f)


def test_forward_paths(pair):
    B, P = 2, 40
    pre = synth.prompt(SHAPE, B, P)
    sess = ssd.ssd_prefill(pair.model, B, P, pre, P + 200, 16)
    os_ = Dc.prefill(pair.om, pre, P + 200)
    stats = {}
    rng = np.random.default_rng(11)
    ssd.ssd_profile_read(pair.model, reset=True)
    ssd.ssd_profile(pair.model, 1)
    try:
        rnd = 0
        for K, rounds, commit_rows in ((1, 1, "all"), (9, 2, "all"), (16, 1, "last"), (8, 1, "last")):
            blk = rng.integers(0, SHAPE.v_img, size=(B, K)).astype(np.int64)
            print(f"{pair.path}: block K={K} ({B * K} rows)", flush=True)
            for _ in range(rounds):
                blk, _ = G.check_round(SHAPE, sess, os_, blk, 0, R.RULE_GREEDY, rnd, 0, None, stats)
                rnd += 1
            if commit_rows == "all":
                G.check_commit(SHAPE, sess, os_, blk, stats, want_h=True)
            else:
                _commit_last_row(sess, os_, blk, stats)
        ssd.ssd_profile(pair.model, 0)
        prof = ssd.ssd_profile_read(pair.model, reset=True)
        print(pair.path, "stats", stats, {k: v[1] for k, v in prof.items()}, flush=True)
        if pair.path == "persistent":
            # every pass of this session has at most 32 rows: all of them ran as one launch
            assert prof["forward"][1] == 9 and prof["qkv"][1] == 0 and prof["attention"][1] == 0
        else:
            assert prof["forward"][1] == 0 and prof["qkv"][1] > 0
        assert stats["flips"] <= 0.02 * stats["positions"] + 1
    finally:
        ssd.ssd_profile(pair.model, 0)
        ssd.ssd_free_session(sess)
