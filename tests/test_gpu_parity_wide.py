"""GPU parity at the widths of the 7B-class and 8B-class (GQA) decoders and at
the longest contexts of the 1B 32x32 and 8B 64x64 workloads.

Depth is cut to two layers.  The layer count changes no kernel shape or launch
configuration: every GEMM, attention and selection launch below is the one the
full-depth model makes for that block size, batch and context, while the oracle
stays within seconds.  Cases:

  7B width (d 4096, 32x128 heads, MLP 11008, vocab 65536 of which 8192 image
      codes): batch 1, 128-token prompt, one 32-token row block, rule (A),
      2 rounds + commit (M = 32)
  8B width (32 query / 8 KV heads, MLP 14336, 32768 image codes): batch 8,
      256-token prompt, one 64-token row block, rule (A), 1 round + commit
      (M = 512: the large-token-tile GEMM path, 4 query heads per KV head)
  1B width, batch 4, a 32-token block at context 1056..1088 (the last row of
      the 32x32 image), top-k 2000, rule (C) with draft distributions q
      (split-KV attention with a cross-chunk merge)
  8B width, batch 1, a 64-token block at context 4288..4352 (the last row of
      the 64x64 image), rule (A)
  8B width, batch 8, a 64-token block at context 4288..4352 for every
      sequence (the shape the bench's attention_at_scale and gemm_at_scale time:
      512-row tiled GEMMs, 4 query heads per KV head over 4352 keys); the oracle
      recomputes two of the eight sequences (sequences are independent), the
      rule on the GPU's own logits is checked for all eight
  7B width, batch 1, a 32-token block at context 1120..1152 (the last row of
      the 32x32 workload), 2 rounds + commit
  8B width, batch 8, 256-token prompt, one 128-token block (M = 1024: the
      passes that carry a commit; gate/up as whole tiles plus a K-split tail)
  8B width, batch 8, 40-token blocks (M = 320: blocks not aligned to the
      16-row groups of the tiled epilogues, a half-full last row tile)
  8B width, batch 2, a 40-token block at context 600..640: 160 query rows per
      (sequence, KV head), so the query-split attention runs one full 128-row
      group and one of 32 rows whose other 96 are padding
  1B width, batch 4, 64-token prompt and a 256-token block (M = 1024: gate/up
      as whole tiles plus a K-split tail of its own shape)
  1B width, batch 4, 64-token prompt and a 64-token block (M = 256, prefill
      and verify): tiled GEMMs whose K range is split over workgroups to
      fill the CUs (O and down projections in 4 splits, QKV in 2), rule (A),
      2 rounds + commit; the same block and a 24-token one with the XCD-local
      reductions switched off (device-scope fences)
"""
import dataclasses

import numpy as np
import pytest

import paper_2606_20543_amd as ssd
import synth
from oracle import decode as Dc
from oracle import select as R
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

W7 = dataclasses.replace(synth.M7B, n_layers=2)
W8 = dataclasses.replace(synth.M8B, n_layers=2)
W1 = dataclasses.replace(synth.M1B, n_layers=2)


def _pair(shape, name):
    print(f"building {name} (GPU + oracle)", flush=True)
    return G.Pair(shape)


@pytest.fixture(scope="module")
def pair7():
    p = _pair(W7, "7B-width 2-layer model")
    yield p
    p.close()


@pytest.fixture(scope="module")
def pair8():
    p = _pair(W8, "8B-width GQA 2-layer model")
    yield p
    p.close()


@pytest.fixture(scope="module")
def pair1():
    p = _pair(W1, "1B-width 2-layer model")
    yield p
    p.close()


def _greedy_block(pair, shape, B, P, K, rounds, keep, seed_stream):
    """Prompt, then one K-token block with drafts planted from the oracle's
    greedy continuation (keep probability `keep`), `rounds` greedy rounds and
    a commit, checked round by round."""
    pre = synth.prompt(shape, B, P)
    os_ = Dc.prefill(pair.om, pre, P + K)
    print(f"oracle greedy continuation of {K} tokens", flush=True)
    ar = Dc.ar_decode(pair.om, pre, K)
    drafts = synth.plant(ar, keep, shape.v_img, stream=seed_stream)
    sess = ssd.ssd_prefill(pair.model, B, P, pre, P + K, K)
    stats = {}
    try:
        blk = drafts.copy()
        for rnd in range(rounds):
            blk, _ = G.check_round(shape, sess, os_, blk, 0, R.RULE_GREEDY, rnd, 0, None, stats)
        G.check_commit(shape, sess, os_, blk, stats, want_h=True)
        print("parity stats", stats, flush=True)
        assert stats["flips"] <= 0.02 * stats["positions"] + 1
        assert stats["flips"] <= G.flips_expected_bound(stats["flips_expected"])
    finally:
        ssd.ssd_free_session(sess)


def test_7b_width_row_block(pair7):
    _greedy_block(pair7, W7, B=1, P=128, K=32, rounds=2, keep=0.6, seed_stream=11)


def test_8b_width_gqa_batch8(pair8):
    """512 rows, the 64x64 workload's verify passes: QKV as 128 x 192 tiles in
    two K splits, gate/up as 256 whole tiles of 128 x 256 and then the last
    48 feature blocks as 256 tiles of 128 x 192, down K-split in four."""
    _greedy_block(pair8, W8, B=8, P=256, K=64, rounds=1, keep=0.6, seed_stream=12)


def test_8b_width_batch8_block128(pair8):
    """1024 rows per pass, the size of the 64x64 workload's passes that carry a
    commit: QKV on 256 whole tiles of 128 x 192, O and down K-split in two, gate/up as 768
    whole tiles in three full rounds and the last 16 feature blocks K-split in
    a second launch, the output layer on 1024 tiles."""
    _greedy_block(pair8, W8, B=8, P=256, K=128, rounds=1, keep=0.6, seed_stream=22)


def test_8b_width_batch7_block64(pair8):
    """448 rows: gate/up's second launch of 128 x 192 tiles over a last
    row tile of 64 rows, and QKV's 128 x 192 tiles in two K splits over it."""
    _greedy_block(pair8, W8, B=7, P=256, K=64, rounds=1, keep=0.6, seed_stream=26)


def test_8b_width_batch8_block40(pair8):
    """320 rows of 40-token blocks: the eight-wave tiles' query and residual
    epilogues where a block starts mid-way through a 16-row group and the
    last 128-row tile is half full (its second row half has no rows)."""
    _greedy_block(pair8, W8, B=8, P=256, K=40, rounds=1, keep=0.6, seed_stream=24)


def test_8b_width_batch8_single_token(pair8):
    """Eight rows of one token each, the passes of greedy AR decoding and of
    the planting run: the weight-streaming GEMMs at the 8B widths and the
    one-query-per-sequence attention under GQA 4."""
    _greedy_block(pair8, W8, B=8, P=600, K=1, rounds=1, keep=0.6, seed_stream=27)


def test_7b_width_single_token(pair7):
    """One token at the 7B widths: the AR step of the strict decode's baseline."""
    _greedy_block(pair7, W7, B=1, P=300, K=1, rounds=1, keep=0.6, seed_stream=28)


def test_8b_width_context_4352(pair8):
    """The 64x64 workload's last row: keys 0..4351 in the split-KV attention."""
    B, P, K = 1, 4288, 64
    pre = synth.prompt(W8, B, P)
    print("oracle prefill of 4288 tokens", flush=True)
    os_ = Dc.prefill(pair8.om, pre, P + K)
    drafts = synth.random_codes(W8, (B, K), stream=13)
    sess = ssd.ssd_prefill(pair8.model, B, P, pre, P + K, K)
    stats = {}
    try:
        blk, _ = G.check_round(W8, sess, os_, drafts, 0, R.RULE_GREEDY, 0, 0, None, stats)
        G.check_commit(W8, sess, os_, blk, stats)
        print("parity stats", stats, flush=True)
        assert stats["flips"] <= 0.02 * stats["positions"] + 1
    finally:
        ssd.ssd_free_session(sess)


def test_8b_width_batch8_context_4352(pair8):
    """Every sequence of the batch verifies its last 64-token row over 4288 cached
    positions; sequences 0 and 7 are recomputed by the oracle."""
    B, P, K = 8, 4288, 64
    pre = synth.prompt(W8, B, P)
    drafts = synth.random_codes(W8, (B, K), stream=18)
    sess = ssd.ssd_prefill(pair8.model, B, P, pre, P + K, K)
    stats = {}
    try:
        carry = np.zeros((B, W8.v_img), np.float32)
        ssd.ssd_get_carry(sess, carry)
        out = G.gpu_verify(sess, W8, drafts + W8.img_lo, G.vparams())
        gnew, gacc, gcnt, _ = G.oracle_rule_on(out["logits"], carry, drafts, 0, R.RULE_GREEDY, 0, 3, [P] * B)
        assert np.array_equal(out["tokens"] - W8.img_lo, gnew)
        assert np.array_equal(out["accept"], gacc) and np.array_equal(out["count"], gcnt)
        com = G.gpu_verify(sess, W8, gnew + W8.img_lo, G.vparams(commit=1), want_h=True)
        assert list(com["frontier"]) == [P + K] * B
        for b in (0, 7):
            print(f"oracle prefill of 4288 tokens, sequence {b}", flush=True)
            os_ = Dc.prefill(pair8.om, pre[b:b + 1], P + K)
            cerr = float(np.abs(carry[b] - os_.carry[0]).max())
            onew, oacc, _, ol = Dc.verify_round(os_, drafts[b:b + 1], 0, R.RULE_GREEDY, 0, 3)
            err = float(np.abs(out["logits"][b] - ol[0]).max())
            stats["max_logit_err"] = max(stats.get("max_logit_err", 0.0), err, cerr)
            assert err < G.TOL["bf16"] and cerr < G.TOL["bf16"], (b, err, cerr)
            flips = 0
            for k in np.nonzero(onew[0] != gnew[b])[0]:
                Lo = os_.carry[0] if k == 0 else ol[0, k - 1]
                assert G.greedy_gap(Lo) < 2 * G.TOL["bf16"], f"sequence {b}, position {k}"
                flips += 1
            stats["flips"] = stats.get("flips", 0) + flips
            cl, ch = Dc.commit(os_, gnew[b:b + 1])
            err = float(np.abs(com["logits"][b] - cl[0]).max())
            stats["max_logit_err"] = max(stats["max_logit_err"], err)
            assert err < G.TOL["bf16"]
            G.check_h_pre(W8, com["h_pre"][b:b + 1], ch, stats)
        print("parity stats", stats, flush=True)
        assert stats["flips"] <= 0.02 * 2 * K + 1
    finally:
        ssd.ssd_free_session(sess)


def test_8b_width_ragged_query_split(pair8):
    """The query-split attention with a partial query group (rows past K*g masked
    and never stored) and short key chunks."""
    _greedy_block(pair8, W8, B=2, P=600, K=40, rounds=1, keep=0.6, seed_stream=21)


def test_7b_width_batch4_block64(pair7):
    """256 rows at the 7B widths: QKV (12288 features) as 64 x 2 tiles of
    128 x 192 in two K splits instead of 48 x 2 of 128 x 256."""
    _greedy_block(pair7, W7, B=4, P=128, K=64, rounds=1, keep=0.6, seed_stream=25)


def test_7b_width_context_1152(pair7):
    """The 32x32 workload's last row: a 32-token block over 1120 cached positions."""
    _greedy_block(pair7, W7, B=1, P=1120, K=32, rounds=2, keep=0.6, seed_stream=19)


def test_1b_width_b4_context_1088_rule_c(pair1):
    pair = pair1
    B, P, K, top_k = 4, 1056, 32, 2000
    pre = synth.prompt(W1, B, P)
    print("oracle prefill of 4 x 1056 tokens", flush=True)
    os_ = Dc.prefill(pair.om, pre, P + K)
    q = synth.normal(synth.SEED_DRAFTS, 14, B * K * W1.v_img, std=1.5).reshape(B, K, W1.v_img)
    drafts = q.argmax(axis=2).astype(np.int64)
    sess = ssd.ssd_prefill(pair.model, B, P, pre, P + K, K)
    stats = {}
    try:
        blk, _ = G.check_round(W1, sess, os_, drafts, 0, R.RULE_ACCEPT_REJECT, 0, top_k, q, stats)
        G.check_commit(W1, sess, os_, blk, stats, want_h=True)
        print("parity stats", stats, flush=True)
        assert stats["flips"] <= G.flips_expected_bound(stats["flips_expected"]), stats
    finally:
        ssd.ssd_free_session(sess)


def test_1b_width_b4_block64_split_tiles(pair1):
    _greedy_block(pair1, W1, B=4, P=64, K=64, rounds=2, keep=0.6, seed_stream=15)


def test_1b_width_b4_block256(pair1):
    """1024 rows at the 1B widths: gate/up as 256 whole tiles and a K-split
    second launch of the other 12 feature blocks (a different split than at the
    8B widths), the output layer on 512 tiles."""
    _greedy_block(pair1, W1, B=4, P=64, K=256, rounds=1, keep=0.6, seed_stream=23)


def test_1b_width_fenced_reductions(monkeypatch):
    """The same 256-row block, and a 24-token one, on a model created with the
    XCD-local workgroup mapping switched off (SSD_NO_XCD_LOCAL=1): every
    split-K and key-chunk reduction then publishes its partials through
    device-scope fences instead of one XCD's L2."""
    monkeypatch.setenv("SSD_NO_XCD_LOCAL", "1")
    pair = _pair(W1, "1B-width 2-layer model, fenced reductions")
    monkeypatch.delenv("SSD_NO_XCD_LOCAL")
    try:
        _greedy_block(pair, W1, B=4, P=64, K=64, rounds=1, keep=0.6, seed_stream=16)
        _greedy_block(pair, W1, B=1, P=64, K=24, rounds=2, keep=0.6, seed_stream=17)
    finally:
        pair.close()
