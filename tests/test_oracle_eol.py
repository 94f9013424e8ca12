"""Pins of the end-of-line layout (the Lumina-mGPT and Emu3 backbones end every
image row with one end-of-line token: their AR reference step counts are
2,352 = 48 x 49 and 8,190 = 90 x 91 in the configuration-sweep and Pareto
tables, against 576 = 24 x 24 for Janus-Pro).

The layout is pinned against an independent token-by-token AR decoder that
forces the token after every W image tokens: greedy verification with enough
rounds per block reproduces it exactly, and drafts equal to it are all
accepted; the end-of-line positions are never verified or counted; the pass
count of the SSD schedule does not change (the printed SSD step counts of the
two backbones hold with the layout)."""
import numpy as np
import pytest

import synth
from oracle import decode as Dc
from oracle import schedule as S
from oracle import select as R
from tests import oracle_util as U

SHAPE = U.TINY_GQA  # text ids [0, 8): the end-of-line token is a text id
EOL = 5


def _model():
    return U.model(SHAPE, U.packed(SHAPE))


def test_ar_steps_follow_the_printed_counts():
    model = _model()
    pre = synth.prompt(SHAPE, 2, 4)
    for H, W in ((3, 4), (2, 5)):
        _, passes = Dc.ar_decode_eol(model, pre, H, W, EOL)
        assert passes == H * (W + 1)
    # the printed AR references: one step per image token and per row end
    assert 48 * (48 + 1) == 2352 and 90 * (90 + 1) == 8190 and 24 * 24 == 576


@pytest.mark.parametrize("k_v,b,i", [(1, 7, 0), (2, 14, 7)])
def test_jacobi_rounds_with_eol_reproduce_greedy_ar(k_v, b, i):
    """A block of K positions settles after K greedy rounds (Jacobi), so rounds
    >= the block length reproduce greedy AR with the forced end-of-line tokens."""
    model = _model()
    H, W = 4, 5
    pre = synth.prompt(SHAPE, 2, 4)
    ar, _ = Dc.ar_decode_eol(model, pre, H, W, EOL)
    drafts = synth.plant(ar, 0.3, SHAPE.v_img)
    out, st = Dc.decode_image(model, pre, H, W, drafts, rule=R.RULE_GREEDY, k_h=5, h_rounds=7, k_v=k_v, b=b, i=i,
                              eol_id=EOL)
    assert np.array_equal(out, ar)
    assert st["passes"] == S.n_passes(S.plan(H, W, k_h=5, h_rounds=7, k_v=k_v, b=b, i=i, eol=True))


def test_ar_drafts_are_all_accepted_and_row_ends_are_not_counted():
    model = _model()
    H, W = 3, 6
    pre = synth.prompt(SHAPE, 2, 4)
    ar, _ = Dc.ar_decode_eol(model, pre, H, W, EOL)
    out, st = Dc.decode_image(model, pre, H, W, ar, rule=R.RULE_GREEDY, k_h=3, b=2, eol_id=EOL)
    assert np.array_equal(out, ar)
    assert st["accepted"] == st["proposed"]
    # image positions verified: row 0 runs once each (minus the fixed first token), rows 1.. twice
    assert st["proposed"] == 2 * ((W - 1) + 2 * (H - 1) * W)


def test_row_end_token_is_in_the_sequence():
    """The decode depends on which token ends the rows (it is really fed)."""
    model = _model()
    pre = synth.prompt(SHAPE, 1, 4)
    a, _ = Dc.ar_decode_eol(model, pre, 3, 4, 5)
    c, _ = Dc.ar_decode_eol(model, pre, 3, 4, 6)
    assert not np.array_equal(a, c)
    drafts = synth.random_codes(SHAPE, (1, 3, 4))
    x, _ = Dc.decode_image(model, pre, 3, 4, drafts, rule=R.RULE_GREEDY, b=2, eol_id=5)
    y, _ = Dc.decode_image(model, pre, 3, 4, drafts, rule=R.RULE_GREEDY, b=2, eol_id=6)
    assert not np.array_equal(x, y)


@pytest.mark.parametrize("H,k_v,b,i,steps", [(48, 2, 5, 4, 280), (90, 1, 5, 0, 571), (48, 3, 5, 4, 272)])
def test_printed_ssd_steps_hold_with_the_layout(H, k_v, b, i, steps):
    """Table "app_pareto" / "abl_nvert": the EOL backbones' SSD step counts."""
    assert S.n_passes(S.plan(H, H, k_h=5, k_v=k_v, b=b, i=i, eol=True)) == steps
    assert S.n_passes(S.plan(H, H, k_h=5, k_v=k_v, b=b, i=i, eol=False)) == steps
