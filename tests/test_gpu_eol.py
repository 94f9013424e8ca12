"""The end-of-line layout on the GPU against the oracle (tiny fp32 decoder, 16-token
prompt, 6x7 grid, decisions bit-exact): every image row closed by one fixed token
that rides along with the block completing its row and is never verified
(the row layout of the Lumina-mGPT and Emu3 backbones)."""
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
P, H, W = 16, 6, 7
EOL = 3  # this vocabulary is all image codes; any id serves as the row end


@pytest.fixture(scope="module")
def pair():
    p = G.Pair(SHAPE, gain_std=0.1)
    yield p
    p.close()


def _sched(rule, top_k=0, k_h=5, h_rounds=1, k_v=1, b=2, i=0, cfg=0, weight=0.0):
    s = ssd.ssd_schedule()
    s.grid_h, s.grid_w, s.k_h, s.h_rounds, s.k_v, s.b_rounds, s.i_rounds = H, W, k_h, h_rounds, k_v, b, i
    s.rule, s.top_k, s.temperature, s.seed = rule, top_k, 1.0, 3
    s.cfg, s.cfg_weight, s.eol, s.eol_id = cfg, weight, 1, EOL
    return s


@pytest.mark.parametrize("rule,top_k,k_v,b,i", [(R.RULE_GREEDY, 0, 1, 2, 0), (R.RULE_SAMPLE, 60, 1, 1, 0),
                                                 (R.RULE_ACCEPT_REJECT, 100, 2, 2, 1)])
def test_eol_decode_matches_oracle(pair, rule, top_k, k_v, b, i):
    B = 2
    pre = synth.prompt(SHAPE, B, P)
    drafts = synth.random_codes(SHAPE, (B, H, W), stream=31)
    q = None
    if rule == R.RULE_ACCEPT_REJECT:
        q = synth.normal(synth.SEED_DRAFTS, 32, B * H * W * SHAPE.v_img, std=1.5).reshape(B, H, W, SHAPE.v_img)
        drafts = q.argmax(axis=-1).astype(np.int64)
    out = np.zeros((B, H, W), np.int32)
    print(f"eol decode rule {rule} k_v {k_v}", flush=True)
    st = ssd.ssd_decode_image(pair.model, _sched(rule, top_k, k_v=k_v, b=b, i=i), B, P, pre,
                              (drafts + SHAPE.img_lo).astype(np.int32), out,
                              draft_logits=None if q is None else np.ascontiguousarray(q, np.float32))
    otok, ost = Dc.decode_image(pair.om, pre, H, W, drafts, rule=rule, seed=3, top_k=top_k, k_v=k_v, b=b, i=i,
                                q_table=q, eol_id=EOL)
    assert np.array_equal(out - SHAPE.img_lo, otok)
    ops = S.plan(H, W, k_v=k_v, b=b, i=i, eol=True)
    assert ost["passes"] == S.n_passes(ops) and st.passes == G.executed_passes(ops)
    assert st.accepted == ost["accepted"] and st.proposed == ost["proposed"]


def test_eol_jacobi_rounds_reproduce_ar(pair):
    """Enough greedy rounds per block give the greedy AR image with forced row ends."""
    B = 1
    pre = synth.prompt(SHAPE, B, P)
    ar, _ = Dc.ar_decode_eol(pair.om, pre, H, W, EOL)
    drafts = synth.random_codes(SHAPE, (B, H, W), stream=33)
    out = np.zeros((B, H, W), np.int32)
    ssd.ssd_decode_image(pair.model, _sched(R.RULE_GREEDY, h_rounds=7, b=W + 1), B, P, pre,
                         (drafts + SHAPE.img_lo).astype(np.int32), out)
    assert np.array_equal(out - SHAPE.img_lo, ar)


def test_eol_guided_decode_matches_oracle(pair):
    pre = np.concatenate([synth.prompt(SHAPE, 1, P), synth.prompt(SHAPE, 1, P, seed=7)])
    drafts = synth.random_codes(SHAPE, (1, H, W), stream=34)
    out = np.zeros((1, H, W), np.int32)
    st = ssd.ssd_decode_image(pair.model, _sched(R.RULE_SAMPLE, 50, cfg=1, weight=3.0), 1, P, pre,
                              (drafts + SHAPE.img_lo).astype(np.int32), out)
    otok, ost = Dc.decode_image(pair.om, pre, H, W, drafts, rule=R.RULE_SAMPLE, seed=3, top_k=50, guide=3.0,
                                eol_id=EOL)
    assert np.array_equal(out - SHAPE.img_lo, otok)
    assert st.passes == G.executed_passes(S.plan(H, W, b=2, eol=True)) and st.accepted == ost["accepted"]


def test_eol_argument_errors(pair):
    pre = synth.prompt(SHAPE, 1, P)
    drafts = (synth.random_codes(SHAPE, (1, H, W)) + SHAPE.img_lo).astype(np.int32)
    out = np.zeros((1, H, W), np.int32)
    sc = _sched(R.RULE_GREEDY)
    sc.eol_id = SHAPE.vocab
    with pytest.raises(ssd.SSDError) as e:
        ssd.ssd_decode_image(pair.model, sc, 1, P, pre, drafts, out)
    assert e.value.status == ssd.SSD_E_INVAL
    sc = _sched(R.RULE_GREEDY)
    sc.eol = 2
    with pytest.raises(ssd.SSDError) as e:
        ssd.ssd_decode_image(pair.model, sc, 1, P, pre, drafts, out)
    assert e.value.status == ssd.SSD_E_INVAL
