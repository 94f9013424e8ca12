"""Pins of planted drafts, the measurement input that fixes the acceptance rate
(the paper measures with trained heads, which are not available; Sec. 3.3
"Verification as Auto Correction" defines what a verify round accepts).

A planted draft is the backbone's own greedy argmax for its position given
everything chosen or drafted before it, kept with a coin flip, else replaced by
another code.  Under rule (A):

* the first verify round of a position accepts it exactly when its coin kept
  it (the verify pass sees the same context the draft was planted against);
* strict verification accepts, per pass, exactly the leading run of kept
  coins after the pending token, so its accepted and tested counts are a
  function of the coins alone, and its output is greedy AR decoding.

Planting against the wrong context (the committed tokens only, or shifted by
one position) or a replacement equal to the argmax breaks these counts.
"""
import numpy as np
import pytest

import synth
from oracle import decode as Dc
from oracle import schedule as S
from oracle import select as R
from tests import oracle_util as U


def _coins(shape, B, n, p, seed=5):
    keep = synth.uniform(seed, 0, B * n) < p
    repl = synth.randint(seed, 1, 0, shape.v_img - 1, B * n).astype(np.int64)
    return keep.reshape(B, n), repl.reshape(B, n)


@pytest.mark.parametrize("shape", [U.TINY_GQA, U.TINY_BF16], ids=["f32", "bf16"])
@pytest.mark.parametrize("p", [0.3, 0.8])
def test_first_round_accepts_exactly_the_kept_drafts(shape, p):
    mod = U.model(shape, U.packed(shape))
    B, H, W = 2, 4, 5
    pre = synth.prompt(shape, B, 6)
    keep, repl = _coins(shape, B, H * W, p)
    tr = []
    out, st = Dc.decode_image(mod, pre, H, W, repl.reshape(B, H, W), rule=R.RULE_GREEDY, k_h=3, b=2,
                              plant=(keep.reshape(B, H, W), repl.reshape(B, H, W)), trace=tr)
    # every image position but the first is drafted once and first verified once
    assert st["proposed_first"] == B * (H * W - 1)
    assert st["accepted_first"] == int(keep[:, 1:].sum())
    # the pass count is the schedule's, planting adds no pass
    assert st["passes"] == S.n_passes(S.plan(H, W, k_h=3, b=2))
    # the planted table as plain drafts reproduces the decode
    out2, st2 = Dc.decode_image(mod, pre, H, W, st["planted"], rule=R.RULE_GREEDY, k_h=3, b=2)
    assert np.array_equal(out, out2)
    assert st2["accepted"] == st["accepted"] and st2["accepted_first"] == st["accepted_first"]


def test_planted_replacements_differ_from_the_argmax():
    shape = U.TINY_GQA
    mod = U.model(shape, U.packed(shape))
    pre = synth.prompt(shape, 1, 6)
    for r in range(shape.v_img - 1):
        t, a = Dc.planted_draft(mod, pre[0], [3, 1], False, r)
        assert t != a and t == r + (r >= a)
        t, a2 = Dc.planted_draft(mod, pre[0], [3, 1], True, r)
        assert t == a == a2


def _strict_counts(keep, N, K):
    """Accepted and tested drafts of strict verification when draft x is
    accepted exactly when its coin is kept: runs of kept coins, pass by pass."""
    acc = tested = passes = 0
    done = 0
    while done < N - 1:
        k_blk = min(K, N - done)
        n = 0
        while n < k_blk - 1 and keep[done + 1 + n]:
            n += 1
        acc += n
        tested += n + (1 if n < k_blk - 1 else 0)
        done += 1 + n
        passes += 1
    return acc, tested, passes


@pytest.mark.parametrize("shape", [U.TINY_GQA, U.TINY_BF16], ids=["f32", "bf16"])
@pytest.mark.parametrize("p,K", [(0.3, 4), (0.7, 6), (0.95, 3)])
def test_strict_decode_with_planted_drafts(shape, p, K):
    mod = U.model(shape, U.packed(shape))
    B, N = 2, 18
    pre = synth.prompt(shape, B, 6)
    keep, repl = _coins(shape, B, N, p, seed=9)
    st = {}
    out, passes = Dc.decode_truncate(mod, pre, repl, K, plant=(keep, repl), stats=st)
    assert np.array_equal(out, Dc.ar_decode(mod, pre, N))
    want = [_strict_counts(keep[b], N, K) for b in range(B)]
    assert st["accepted"] == sum(w[0] for w in want)
    assert st["proposed"] == sum(w[1] for w in want)
    assert passes == sum(w[2] + 1 for w in want)  # + prefill
    # the planted table as plain drafts gives the same passes and counts
    st2 = {}
    out2, passes2 = Dc.decode_truncate(mod, pre, st["planted"], K, stats=st2)
    assert np.array_equal(out2, out) and passes2 == passes
    assert (st2["accepted"], st2["proposed"]) == (st["accepted"], st["proposed"])
