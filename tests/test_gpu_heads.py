"""Images drafted by spatial heads on the GPU (ssd_decode_image_heads) against
the oracle's head-drafted decode (Sec. 3.3: horizontal heads draft the rest of
the row from the last chosen token, vertical heads whole rows from the row
above; heads on [h; e] of the source token, h the state that scored it).

Tiny fp32 decoder (2 layers, d=256, 1024 codes, 16-token prompt, 8x8 grid)
with seeded fp32 heads (m = 256): the head alone (logits within 1e-5, drafts
exact), then whole images under rules A, B and C, joint and staged multi-row
schedules and guidance, tokens and counts bit-exact.  2-layer decoder of the 1B
widths (bf16): the same driver end to end (valid codes, pass count, repeatable).
"""
import dataclasses

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

TINY = synth.TINY
P, H, W = 16, 8, 8
MI = 256


def _sched(rule, top_k=0, k_h=5, k_v=1, b=2, i=0, cfg=0, weight=0.0):
    s = ssd.ssd_schedule()
    s.grid_h, s.grid_w, s.k_h, s.h_rounds, s.k_v, s.b_rounds, s.i_rounds = H, W, k_h, 1, k_v, b, i
    s.rule, s.top_k, s.temperature, s.seed = rule, top_k, 1.0, 3
    s.cfg, s.cfg_weight = cfg, weight
    return s


class Heads:
    """k_h horizontal and k_v vertical heads, on the GPU and in the oracle, from
    seeded weights (seed = head index, horizontal first)."""

    def __init__(self, pair, k_h, k_v, max_rows, dtype, std=0.05):
        self.shape = pair.shape
        d = pair.shape.d_model
        self.gpu, self.ora = [], []
        for j in range(k_h + k_v):
            w = synth.draft_head_weights(d, MI, seed=10 + j, std=std, gain_std=0.1, dtype=dtype)
            self.gpu.append(ssd.ssd_draft_head_init(pair.model, MI, w, max_rows))
            self.ora.append(Dr.Head(d, MI, w))
        self.k_h = k_h

    def lists(self, side):
        return (self.gpu if side == "gpu" else self.ora)[:self.k_h], (self.gpu if side == "gpu" else self.ora)[self.k_h:]

    def close(self):
        for h in self.gpu:
            ssd.ssd_free_draft_head(h)
        self.gpu = []


@pytest.fixture(scope="module")
def tiny():
    p = G.Pair(TINY, gain_std=0.1)
    hs = Heads(p, 5, 2, 2 * W, "f32")
    yield p, hs
    hs.close()
    p.close()


def test_fp32_head_matches_oracle(tiny):
    pair, hs = tiny
    R_ = 12
    h = synth.hidden_states(R_, TINY.d_model)
    tok = synth.randint(synth.SEED_HEADS, 5, 0, TINY.vocab, R_).astype(np.int32)
    for j in (0, 6):
        dr = np.zeros(R_, np.int32)
        lg = np.zeros((R_, TINY.v_img), np.float32)
        ssd.ssd_draft_head_run(hs.gpu[j], R_, h, tok, dr, lg)
        oidx, olg = Dr.draft(pair.om, hs.ora[j], h.astype(np.float64), tok)
        assert np.abs(lg - olg).max() < G.TOL["f32"]
        assert np.array_equal(dr - TINY.img_lo, oidx)


@pytest.mark.parametrize("rule,top_k,k_v,b,i", [(R.RULE_GREEDY, 0, 1, 2, 0), (R.RULE_SAMPLE, 50, 1, 2, 0),
                                                 (R.RULE_ACCEPT_REJECT, 100, 1, 2, 0),
                                                 (R.RULE_ACCEPT_REJECT, 0, 2, 2, 1)])
def test_heads_decode_matches_oracle(tiny, rule, top_k, k_v, b, i):
    pair, hs = tiny
    B = 2
    pre = synth.prompt(TINY, B, P)
    out = np.zeros((B, H, W), np.int32)
    gh, gv = hs.lists("gpu")
    print(f"heads decode rule {rule} top_k {top_k} k_v {k_v} b {b} i {i}", flush=True)
    st = ssd.ssd_decode_image_heads(pair.model, _sched(rule, top_k, k_v=k_v, b=b, i=i), B, P, pre, gh, gv[:k_v], out)
    oh, ov = hs.lists("oracle")
    otok, ost = Dc.decode_image(pair.om, pre, H, W, None, rule=rule, seed=3, top_k=top_k, k_v=k_v, b=b, i=i,
                                heads=(oh, ov[:k_v]))
    assert np.array_equal(out - TINY.img_lo, otok)
    ops = S.plan(H, W, k_v=k_v, b=b, i=i)
    assert ost["passes"] == S.n_passes(ops) and st.passes == G.executed_passes(ops, heads=True)
    assert st.accepted == ost["accepted"] and st.proposed == ost["proposed"]


def test_guided_heads_decode_matches_oracle(tiny):
    pair, hs = tiny
    pre = np.concatenate([synth.prompt(TINY, 1, P), synth.prompt(TINY, 1, P, seed=7)])
    out = np.zeros((1, H, W), np.int32)
    gh, gv = hs.lists("gpu")
    st = ssd.ssd_decode_image_heads(pair.model, _sched(R.RULE_ACCEPT_REJECT, 100, cfg=1, weight=4.0), 1, P, pre,
                                    gh, gv[:1], out)
    oh, ov = hs.lists("oracle")
    otok, ost = Dc.decode_image(pair.om, pre, H, W, None, rule=R.RULE_ACCEPT_REJECT, seed=3, top_k=100,
                                heads=(oh, ov[:1]), guide=4.0)
    assert np.array_equal(out - TINY.img_lo, otok)
    assert st.accepted == ost["accepted"]


def test_heads_decode_with_row_ends_matches_oracle(tiny):
    """The end-of-line layout under head drafting: a row end's state scores the
    next row's first token, drafts land at sequence positions."""
    pair, hs = tiny
    B = 2
    pre = synth.prompt(TINY, B, P)
    out = np.zeros((B, H, W), np.int32)
    sc = _sched(R.RULE_ACCEPT_REJECT, 100, k_v=2, b=2, i=1)
    sc.eol, sc.eol_id = 1, 3
    gh, gv = hs.lists("gpu")
    st = ssd.ssd_decode_image_heads(pair.model, sc, B, P, pre, gh, gv, out)
    oh, ov = hs.lists("oracle")
    otok, ost = Dc.decode_image(pair.om, pre, H, W, None, rule=R.RULE_ACCEPT_REJECT, seed=3, top_k=100, k_v=2, b=2,
                                i=1, heads=(oh, ov), eol_id=3)
    assert np.array_equal(out - TINY.img_lo, otok)
    assert st.passes == G.executed_passes(S.plan(H, W, k_v=2, b=2, i=1, eol=True), heads=True)
    assert st.accepted == ost["accepted"] and st.proposed == ost["proposed"]


def test_heads_argument_errors(tiny):
    pair, hs = tiny
    pre = synth.prompt(TINY, 1, P)
    out = np.zeros((1, H, W), np.int32)
    gh, gv = hs.lists("gpu")
    with pytest.raises(ssd.SSDError) as e:  # five-token runs need five horizontal heads
        ssd.ssd_decode_image_heads(pair.model, _sched(R.RULE_GREEDY), 1, P, pre, gh[:3], gv[:1], out)
    assert e.value.status == ssd.SSD_E_INVAL
    with pytest.raises(ssd.SSDError) as e:  # no vertical head
        ssd.ssd_decode_image_heads(pair.model, _sched(R.RULE_GREEDY), 1, P, pre, gh, [], out)
    assert e.value.status == ssd.SSD_E_INVAL
    small = ssd.ssd_draft_head_init(pair.model, MI, synth.draft_head_weights(TINY.d_model, MI, dtype="f32"), W - 1)
    try:
        with pytest.raises(ssd.SSDError) as e:  # a vertical head drafts W rows per call
            ssd.ssd_decode_image_heads(pair.model, _sched(R.RULE_GREEDY), 1, P, pre, gh, [small], out)
        assert e.value.status == ssd.SSD_E_INVAL
    finally:
        ssd.ssd_free_draft_head(small)


BF16 = dataclasses.replace(synth.M1B, n_layers=2)


def test_heads_decode_bf16_runs_and_repeats():
    pair = G.Pair(BF16, oracle=False)
    hs = Heads(pair, 5, 1, 2 * W, "bf16", std=0.02)
    try:
        B = 2
        pre = synth.prompt(BF16, B, P)
        gh, gv = hs.lists("gpu")
        outs = []
        for _ in range(2):
            out = np.zeros((B, H, W), np.int32)
            st = ssd.ssd_decode_image_heads(pair.model, _sched(R.RULE_ACCEPT_REJECT, 2000), B, P, pre, gh, gv, out)
            outs.append(out)
        assert np.array_equal(outs[0], outs[1])
        assert ((outs[0] >= BF16.img_lo) & (outs[0] < BF16.img_hi)).all()
        assert st.passes == G.executed_passes(S.plan(H, W, b=2), heads=True)
    finally:
        hs.close()
        pair.close()
