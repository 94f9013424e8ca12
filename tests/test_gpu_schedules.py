"""Degenerate grids and schedules of the image decode on the GPU against the
oracle (tiny fp32 decoder, decisions bit-exact): a single row (no vertical
stage), a single column (no horizontal runs), runs longer than the row, a
vertical group taller than the rest of the image, no verification rounds in
the horizontal stage, one-token runs, and head-drafted decodes where one head
family is never used."""
import numpy as np
import pytest

import paper_2606_20543_amd as ssd
import synth
from oracle import decode as Dc
from oracle import draft as Dr
from oracle import schedule as S
from oracle import select as R
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

SHAPE = synth.TINY
P = 16


@pytest.fixture(scope="module")
def pair():
    p = G.Pair(SHAPE, gain_std=0.1)
    yield p
    p.close()


def _sched(H, W, k_h, h_rounds, k_v, b, i, rule, top_k):
    s = ssd.ssd_schedule()
    s.grid_h, s.grid_w, s.k_h, s.h_rounds, s.k_v, s.b_rounds, s.i_rounds = H, W, k_h, h_rounds, k_v, b, i
    s.rule, s.top_k, s.temperature, s.seed = rule, top_k, 1.0, 3
    return s


CASES = [  # H, W, k_h, h_rounds, k_v, b, i, rule, top_k
    (1, 8, 5, 1, 1, 2, 0, R.RULE_ACCEPT_REJECT, 0),   # one row: horizontal stage only
    (6, 1, 5, 1, 1, 2, 0, R.RULE_GREEDY, 0),          # one column: no horizontal run
    (5, 4, 9, 1, 1, 2, 0, R.RULE_SAMPLE, 40),         # a run longer than the row
    (4, 5, 2, 1, 6, 2, 1, R.RULE_ACCEPT_REJECT, 50),  # a group taller than the remaining rows
    (3, 6, 3, 0, 1, 1, 0, R.RULE_GREEDY, 0),          # horizontal runs committed unverified
    (2, 2, 1, 2, 1, 3, 0, R.RULE_SAMPLE, 0),          # one-token runs, 2x2 grid
]


@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}x{c[1]}-kh{c[2]}-hr{c[3]}-kv{c[4]}-b{c[5]}-i{c[6]}" for c in CASES])
def test_degenerate_schedule_matches_oracle(pair, case):
    H, W, k_h, h_rounds, k_v, b, i, rule, top_k = case
    B = 2
    pre = synth.prompt(SHAPE, B, P)
    drafts = synth.random_codes(SHAPE, (B, H, W), stream=21)
    out = np.zeros((B, H, W), np.int32)
    print(f"schedule {case}", flush=True)
    st = ssd.ssd_decode_image(pair.model, _sched(*case), B, P, pre, (drafts + SHAPE.img_lo).astype(np.int32), out)
    otok, ost = Dc.decode_image(pair.om, pre, H, W, drafts, rule=rule, seed=3, top_k=top_k, k_h=k_h,
                                h_rounds=h_rounds, k_v=k_v, b=b, i=i)
    assert np.array_equal(out - SHAPE.img_lo, otok)
    ops = S.plan(H, W, k_h=k_h, h_rounds=h_rounds, k_v=k_v, b=b, i=i)
    assert ost["passes"] == S.n_passes(ops) and st.passes == G.executed_passes(ops)
    assert st.accepted == ost["accepted"] and st.proposed == ost["proposed"]


@pytest.mark.parametrize("H,W", [(1, 6), (5, 1)])
def test_heads_decode_with_one_head_family(pair, H, W):
    """A single row needs no vertical head, a single column no horizontal head."""
    mi, d = 256, SHAPE.d_model
    k_h = min(3, W - 1)
    n = k_h + (1 if H > 1 else 0)
    ws = [synth.draft_head_weights(d, mi, seed=30 + j, std=0.05, gain_std=0.1, dtype="f32") for j in range(n)]
    heads = [ssd.ssd_draft_head_init(pair.model, mi, w, 2 * W) for w in ws]
    try:
        B = 2
        pre = synth.prompt(SHAPE, B, P)
        out = np.zeros((B, H, W), np.int32)
        sc = _sched(H, W, max(k_h, 1), 1, 1, 2, 0, R.RULE_ACCEPT_REJECT, 0)
        st = ssd.ssd_decode_image_heads(pair.model, sc, B, P, pre, heads[:k_h], heads[k_h:], out)
        ora = [Dr.Head(d, mi, w) for w in ws]
        otok, ost = Dc.decode_image(pair.om, pre, H, W, None, rule=R.RULE_ACCEPT_REJECT, seed=3, k_h=max(k_h, 1),
                                    b=2, heads=(ora[:k_h], ora[k_h:]))
        assert np.array_equal(out - SHAPE.img_lo, otok)
        ops = S.plan(H, W, k_h=max(k_h, 1), b=2)
        assert st.passes == G.executed_passes(ops, heads=True) and st.accepted == ost["accepted"]
    finally:
        for h in heads:
            ssd.ssd_free_draft_head(h)


FUSE_CASES = [  # rule, top_k, k_v, b, i, cfg, eol
    (R.RULE_GREEDY, 0, 1, 2, 0, 0, 0),
    (R.RULE_ACCEPT_REJECT, 100, 2, 2, 1, 0, 0),
    (R.RULE_SAMPLE, 40, 1, 1, 0, 1, 0),
    (R.RULE_ACCEPT_REJECT, 0, 1, 2, 0, 0, 1),
]


@pytest.mark.parametrize("case", FUSE_CASES, ids=[f"rule{c[0]}-kv{c[2]}-cfg{c[5]}-eol{c[6]}" for c in FUSE_CASES])
def test_fused_commits_decide_like_separate_passes(pair, case):
    """A commit run inside the next verify round's pass decides exactly what the
    separate passes decide (fp32: bit for bit), with fewer passes."""
    rule, top_k, k_v, b, i, cfg, eol = case
    H, W, B = 6, 7, 2
    pre = synth.prompt(SHAPE, B, P)
    if cfg:
        pre = np.concatenate([pre, synth.prompt(SHAPE, B, P, seed=7)])
    drafts = (synth.random_codes(SHAPE, (B, H, W), stream=41) + SHAPE.img_lo).astype(np.int32)
    q = None
    if rule == R.RULE_ACCEPT_REJECT:
        q = synth.normal(synth.SEED_DRAFTS, 42, B * H * W * SHAPE.v_img, std=1.5).astype(np.float32)
        q = q.reshape(B, H, W, SHAPE.v_img)
    outs, stats = [], []
    for separate in (0, 1):
        sc = _sched(H, W, 5, 1, k_v, b, i, rule, top_k)
        sc.cfg, sc.cfg_weight, sc.eol, sc.eol_id, sc.separate_commit = cfg, 3.0, eol, 3, separate
        out = np.zeros((B, H, W), np.int32)
        stats.append(ssd.ssd_decode_image(pair.model, sc, B, P, pre, drafts, out, draft_logits=q))
        outs.append(out)
    assert np.array_equal(outs[0], outs[1])
    assert stats[0].accepted == stats[1].accepted and stats[0].proposed == stats[1].proposed
    ops = S.plan(H, W, k_h=5, k_v=k_v, b=b, i=i, eol=bool(eol))
    assert stats[1].passes == S.n_passes(ops)
    assert stats[0].passes == G.executed_passes(ops) < stats[1].passes
