"""Pins of the oracle's head-drafted image decode (Sec. 3.3: horizontal heads
draft the rest of the row from the last chosen token, vertical heads draft whole
rows from the completed row above; Eq. 2 heads on [h; e] of the source token,
h the pre-norm state that scored it).

Each pin ties the driver to something outside it: zero heads must decode like a
planted table of zeros with uniform draft distributions; heads that copy a
permutation of the source token's embedding must draft a function of that token
alone (recomputed from the backbone's tensors, a different permutation per head,
so offsets and directions are pinned); heads that copy the state must draft the
argmax of the state that scored the source token, taken from a full no-cache
forward over the final prompt and image.
"""
import numpy as np
import pytest

from oracle import decode as Dc
from oracle import draft as Dr
from oracle import model as M
from oracle import schedule as S
from oracle import select as R
from tests import oracle_util as U

SHAPE = U.TINY_GQA  # fp32 backbone, d = 32, 32 image codes
H, W, P = 5, 6, 4
D, MI = SHAPE.d_model, 64


def _model():
    return U.model(SHAPE, U.packed(SHAPE))


def _head(w0=None, w2=None, scale=0.3, seed=0):
    rng = np.random.default_rng(seed)
    parts = {"w0": rng.normal(0, scale, (D, 2 * D)), "g": 1 + 0.1 * rng.normal(size=D),
             "w1": rng.normal(0, scale, (MI, D)), "w3": rng.normal(0, scale, (MI, D)),
             "w2": rng.normal(0, scale, (D, MI))}
    if w0 is not None:
        parts["w0"] = w0
    if w2 is not None:
        parts["w2"] = w2
    buf = np.concatenate([np.asarray(parts[n], np.float32).reshape(-1) for n, _ in Dr.head_layout(D, MI)])
    return Dr.Head(D, MI, buf)


def _heads(k_h, k_v, make):
    return [make("h", j) for j in range(k_h)], [make("v", j) for j in range(k_v)]


def _drafts(trace):
    return [t for t in trace if t[0][0].startswith("draft")]


def _prefix(B):
    return np.random.default_rng(3).integers(0, SHAPE.img_lo, size=(B, P))


@pytest.mark.parametrize("rule,top_k", [(R.RULE_GREEDY, 0), (R.RULE_SAMPLE, 0), (R.RULE_ACCEPT_REJECT, 0),
                                        (R.RULE_ACCEPT_REJECT, 7)])
def test_zero_heads_are_planted_zeros_with_uniform_q(rule, top_k):
    model = _model()
    zero = _head(w0=np.zeros((D, 2 * D)), w2=np.zeros((D, MI)))
    hh = ([zero] * 3, [zero] * 2)
    kw = dict(rule=rule, seed=5, top_k=top_k, k_h=3, k_v=2, b=2, i=1)
    got, st = Dc.decode_image(model, _prefix(2), H, W, None, heads=hh, **kw)
    q = np.zeros((2, H, W, SHAPE.img_hi - SHAPE.img_lo)) if rule == R.RULE_ACCEPT_REJECT else None
    want, st2 = Dc.decode_image(model, _prefix(2), H, W, np.zeros((2, H, W), np.int64), q_table=q, **kw)
    assert np.array_equal(got, want) and st == st2
    assert st["passes"] == S.n_passes(S.plan(H, W, k_h=3, k_v=2, b=2, i=1))


def _perm(kind, j):
    p = np.random.default_rng(100 + 10 * (kind == "v") + j).permutation(D)
    return np.eye(D)[p]


@pytest.mark.parametrize("eol", [None, 5])
def test_embedding_heads_draft_from_their_source_tokens(eol):
    model = _model()
    hh = _heads(3, 2, lambda kind, j: _head(w0=np.concatenate([np.zeros((D, D)), _perm(kind, j)], axis=1),
                                            w2=np.zeros((D, MI)), seed=j))
    trace = []
    img, _ = Dc.decode_image(model, _prefix(2), H, W, None, rule=R.RULE_GREEDY, k_h=3, k_v=2, b=1, i=1,
                             heads=hh, trace=trace, eol_id=eol)
    flat = img.reshape(2, -1)
    lm = model.lm_img
    n_ops = {"draft_h": 0, "draft_v": 0}
    for op, j, srcs, dsts, drafted in _drafts(trace):
        n_ops[op[0]] += 1
        perm = _perm("h" if op[0] == "draft_h" else "v", j - 1)
        e = model.tok_emb[flat[:, srcs] + SHAPE.img_lo]            # (B, n, d) embeddings of the source tokens
        z = (model.final_norm * (e @ perm.T)) @ lm.T                 # positive 1/rms does not move the argmax
        want = z.argmax(axis=-1)
        assert np.array_equal(drafted.reshape(want.shape), want)
        step = 1 if op[0] == "draft_h" else W
        assert np.array_equal(dsts.reshape(-1), (srcs + j * step).reshape(-1))
    ops = S.plan(H, W, k_h=3, k_v=2, b=1, i=1)
    assert n_ops["draft_h"] == sum(o[2] for o in ops if o[0] == "draft_h")
    assert n_ops["draft_v"] == sum(o[2] for o in ops if o[0] == "draft_v")


@pytest.mark.parametrize("eol", [None, 5])
def test_state_heads_draft_the_argmax_that_scored_the_source(eol):
    model = _model()
    eye = np.concatenate([np.eye(D), np.zeros((D, D))], axis=1)
    hh = _heads(2, 1, lambda kind, j: _head(w0=eye, w2=np.zeros((D, MI)), seed=j))
    trace = []
    pre = _prefix(2)
    img, _ = Dc.decode_image(model, pre, H, W, None, rule=R.RULE_SAMPLE, seed=9, k_h=2, k_v=1, b=2,
                             heads=hh, trace=trace, eol_id=eol)
    # full forward over the final sequence without a cache (rows closed by the
    # end-of-line token when there is one): the state at the sequence position
    # before image token p scored it
    rows = img + SHAPE.img_lo
    if eol is not None:
        rows = np.concatenate([rows, np.full((2, H, 1), eol)], axis=2)
    seq = np.concatenate([pre, rows.reshape(2, -1)], axis=1)
    logits, _ = M.forward(model, M.Cache(model.cfg, 2, seq.shape[1]), seq, np.zeros(2, np.int64))
    RW = W + (eol is not None)
    for op, j, srcs, dsts, drafted in _drafts(trace):
        spos = (srcs // W) * RW + srcs % W
        want = logits[:, P + spos - 1].argmax(axis=-1)
        assert np.array_equal(drafted.reshape(want.shape), want)


def test_heads_decode_under_guidance_uses_the_conditional_states():
    model = _model()
    hh = _heads(3, 1, lambda kind, j: _head(seed=10 * (kind == "v") + j))
    both = np.concatenate([_prefix(1), np.zeros((1, P), np.int64)])
    trace = []
    img, st = Dc.decode_image(model, both, H, W, None, rule=R.RULE_ACCEPT_REJECT, seed=2, k_h=3, b=2,
                              heads=hh, guide=3.0, trace=trace)
    assert img.shape == (1, H, W) and st["passes"] == S.n_passes(S.plan(H, W, k_h=3, b=2))
    # the first run is drafted from the prefill's last conditional state and the first token
    g = Dc.prefill(model, both, P + H * W, guide=3.0)
    op, j, srcs, dsts, drafted = _drafts(trace)[0]
    idx, _ = Dr.draft(model, hh[0][0], g.h_carry[:1], img.reshape(1, -1)[:, 0] + SHAPE.img_lo)
    assert op[0] == "draft_h" and j == 1 and drafted.reshape(-1)[0] == idx[0]
