"""GPU parity of the spatial draft head (Sec. 3.3, Eq. 2) against the oracle:
a head of the 1B widths (d = 2048, m = 2d = 4096) on a 2-layer 1B-width bf16
decoder (the head uses the backbone's embedding, final norm and output layer
only), synthetic pre-norm states and random tokens, for a full 24-token row,
a ragged 5-row call and a 40-row call (the multi-tile GEMM path); logits within
the bf16 tolerance, drafts exact on the GPU's own logits (lowest id among
maxima) and equal to the oracle's except where its top-2 gap is within the
logit error."""
import dataclasses

import numpy as np
import pytest

import paper_2606_20543_amd as ssd
import synth
from oracle import draft as Dr
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

SHAPE = dataclasses.replace(synth.M1B, n_layers=2)
TOL = G.TOL["bf16"]
MI = 2 * SHAPE.d_model


@pytest.fixture(scope="module")
def setup():
    print("building 2-layer 1B-width model and a draft head", flush=True)
    p = G.Pair(SHAPE)
    bits = synth.draft_head_weights(SHAPE.d_model, MI, gain_std=0.1)
    assert ssd.ssd_draft_head_numel(p.model, MI) == bits.shape[0] == Dr.head_numel(SHAPE.d_model, MI)
    head = ssd.ssd_draft_head_init(p.model, MI, bits, 64)
    oh = Dr.Head(SHAPE.d_model, MI, bits)
    yield p, head, oh
    ssd.ssd_free_draft_head(head)
    p.close()


@pytest.mark.parametrize("R", [24, 5, 40])
def test_draft_head_rows(setup, R):
    p, head, oh = setup
    d = SHAPE.d_model
    h = synth.hidden_states(R, d, stream=100 + R)
    tok = synth.randint(synth.SEED_HEADS, 200 + R, 0, SHAPE.vocab, R).astype(np.int32)
    drafts = np.zeros(R, np.int32)
    logits = np.zeros((R, SHAPE.v_img), np.float32)
    print(f"draft head: R={R}", flush=True)
    ssd.ssd_draft_head_run(head, R, h, tok, drafts, logits)
    o_idx, o_logits = Dr.draft(p.om, oh, h.astype(np.float64), tok)
    err = float(np.abs(logits - o_logits).max())
    print(f"R={R} max logit error {err:.2e}", flush=True)
    assert err < TOL
    # decisions: the GPU's argmax of its own logits (lowest id among maxima)
    assert np.array_equal(drafts - SHAPE.img_lo, logits.argmax(axis=1))
    for r in np.nonzero(drafts - SHAPE.img_lo != o_idx)[0]:
        assert G.greedy_gap(o_logits[r]) < 2 * err, f"row {r}: draft differs beyond the logit error"


def test_draft_head_device_pointers(setup):
    """Device inputs and outputs (no synchronization inside the call) give the same drafts."""
    p, head, oh = setup
    d, R = SHAPE.d_model, 24
    h = synth.hidden_states(R, d, stream=7)
    tok = synth.randint(synth.SEED_HEADS, 8, SHAPE.img_lo, SHAPE.img_hi, R).astype(np.int32)
    dh, dt, dd = G.DeviceArray(h), G.DeviceArray(tok), G.DeviceArray(np.zeros(R, np.int32))
    try:
        ssd.ssd_draft_head_run(head, R, dh.ptr, dt.ptr, dd.ptr)
        host = np.zeros(R, np.int32)
        ssd.ssd_draft_head_run(head, R, h, tok, host)
        assert np.array_equal(dd.numpy(), host)
    finally:
        for a in (dh, dt, dd):
            a.free()
