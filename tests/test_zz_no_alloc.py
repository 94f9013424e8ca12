"""The allocation-free draft-head run (ssd_draft_head_run_noalloc, workspace in
the library's static device array) against the ordinary run of the same head
(ssd_draft_head_run, the head's own workspace): the same kernels on the same
plans, so drafts and logits must be identical, on two calls in a row, the
second with fewer rows (the array keeps the first call's contents).  Sizes
beyond the static workspace and host arrays are refused before any launch."""
import ctypes
import dataclasses

import numpy as np
import pytest

import paper_2606_20543_amd as ssd
import synth
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

SHAPE = dataclasses.replace(synth.M1B, n_layers=2)
MI = 2 * SHAPE.d_model
MAX_ROWS = 512


@pytest.fixture(scope="module")
def head():
    print("no-alloc: 2-layer 1B-width model and a draft head", flush=True)
    p = G.Pair(SHAPE, oracle=False)
    h = ssd.ssd_draft_head_init(p.model, MI, synth.draft_head_weights(SHAPE.d_model, MI, gain_std=0.1), MAX_ROWS)
    yield h
    ssd.ssd_free_draft_head(h)
    p.close()


def _run(head, R, stream, noalloc):
    d = SHAPE.d_model
    h = synth.hidden_states(R, d, stream=stream)
    tok = synth.randint(synth.SEED_HEADS, stream + 1, 0, SHAPE.vocab, R).astype(np.int32)
    arrs = [G.DeviceArray(h), G.DeviceArray(tok), G.DeviceArray(np.zeros(R, np.int32)),
            G.DeviceArray(np.zeros((R, SHAPE.v_img), np.float32))]
    try:
        fn = ssd.ssd_draft_head_run_noalloc if noalloc else ssd.ssd_draft_head_run
        fn(head, R, arrs[0].ptr, arrs[1].ptr, arrs[2].ptr, arrs[3].ptr)
        return arrs[2].numpy(), arrs[3].numpy()
    finally:
        for a in arrs:
            a.free()


def test_noalloc_equals_ordinary_run_twice(head):
    for R, stream in ((40, 300), (7, 310)):  # the second call smaller than the first
        print(f"no-alloc: R={R}", flush=True)
        want_d, want_l = _run(head, R, stream, noalloc=False)
        got_d, got_l = _run(head, R, stream, noalloc=True)
        assert np.array_equal(got_d, want_d)
        assert np.array_equal(got_l, want_l)
        assert np.array_equal(got_d - SHAPE.img_lo, want_l.argmax(axis=1))


def test_noalloc_refuses_what_it_cannot_hold(head):
    L = ssd.lib()
    d = SHAPE.d_model
    R = MAX_ROWS  # inside max_rows, beyond the static workspace
    arrs = [G.DeviceArray(np.zeros((R, d), np.float32)), G.DeviceArray(np.zeros(R, np.int32)),
            G.DeviceArray(np.zeros(R, np.int32))]
    try:
        st = L.ssd_draft_head_run_noalloc(ctypes.c_void_p(head), R, ctypes.c_void_p(arrs[0].ptr),
                                          ctypes.c_void_p(arrs[1].ptr), ctypes.c_void_p(arrs[2].ptr), None)
        assert st == ssd.SSD_E_INVAL and "static workspace" in ssd.ssd_last_error()
        host = np.zeros(8, np.int32)
        st = L.ssd_draft_head_run_noalloc(ctypes.c_void_p(head), 8, ctypes.c_void_p(arrs[0].ptr),
                                          ctypes.c_void_p(arrs[1].ptr), host.ctypes.data_as(ctypes.c_void_p), None)
        assert st == ssd.SSD_E_INVAL and "device arrays" in ssd.ssd_last_error()
    finally:
        for a in arrs:
            a.free()
    # the head still works after the refusals
    d1, _ = _run(head, 5, 320, noalloc=True)
    d2, _ = _run(head, 5, 320, noalloc=False)
    assert np.array_equal(d1, d2)
