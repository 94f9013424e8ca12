"""Pins of the oracle's spatial draft head (Sec. 3.3 "Draft Prediction in
Latent Space", Eq. 2) and its draft decode through the backbone's output layer.

Each pin ties the oracle to something other than itself: the parameter count
the paper prints, the backbone oracle's own output layer (an identity head
must reproduce the logits of the forward pass that produced h), the residual
and normalization structure of Eq. 2 (exact scale identities), and the
lowest-id tie rule of the argmax.
"""
import numpy as np

import synth
from oracle import draft as Dr
from oracle import model as M
from tests import oracle_util as U

SHAPE = U.TINY_BF16  # d = 32, vocabulary 40 (32 image codes)
ONE = np.uint16(0x3F80)  # bf16 bits of 1.0


def _head_bits(d, m, **edits):
    """Random head weights (bf16 bits) with named tensors replaced."""
    buf = synth.draft_head_weights(d, m, std=0.2, gain_std=0.1)
    off = 0
    for name, shape in Dr.head_layout(d, m):
        n = int(np.prod(shape))
        if name in edits:
            buf[off:off + n] = np.asarray(edits[name], dtype=np.uint16).reshape(-1)
        off += n
    return buf


def _eye_bits(rows, cols, col0):
    """bf16 bits of [rows x cols] with ones at (i, col0 + i)."""
    a = np.zeros((rows, cols), dtype=np.uint16)
    a[np.arange(rows), col0 + np.arange(rows)] = ONE
    return a


def test_parameter_count_matches_the_paper():
    # Table "app_config": 134.2 M parameters per head at d = 4096 (all three backbones' heads);
    # W0 (d x 2d) + gain + W1, W3 (m x d) + W2 (d x m) gives that count with m = 2d
    n = Dr.head_numel(4096, 8192)
    assert round(n / 1e6, 1) == 134.2
    assert synth.draft_head_weights(32, 64).shape[0] == Dr.head_numel(32, 64)


def test_identity_head_reproduces_the_backbones_logits():
    """W0 = [I | 0], W2 = 0: h_hat = h, so the draft logits are the forward pass's own
    logits for the positions whose pre-norm states were fed in (concatenation order, W0
    orientation, the final norm's gain and 1/rms, the image rows of the LM head)."""
    buf = U.packed(SHAPE)
    model = U.model(SHAPE, buf)
    d = SHAPE.d_model
    rng = np.random.default_rng(5)
    B, K = 2, 5
    tokens = rng.integers(SHAPE.img_lo, SHAPE.img_hi, size=(B, K))
    cache = M.Cache(model.cfg, B, 16)
    logits, h_pre = M.forward(model, cache, tokens, np.array([0, 3]))
    m = 48
    hb = Dr.Head(d, m, _head_bits(d, m, w0=_eye_bits(d, 2 * d, 0), w2=np.zeros((d, m))))
    idx, lg = Dr.draft(model, hb, h_pre.reshape(B * K, d), tokens.reshape(-1))
    assert np.allclose(lg, logits.reshape(B * K, -1), rtol=1e-12, atol=1e-12)
    assert np.array_equal(idx, logits.reshape(B * K, -1).argmax(axis=1))


def test_embedding_half_of_the_input():
    """W0 = [0 | I], W2 = 0: h_hat = e, the token's embedding row, which is also the
    pre-norm state of a backbone whose residual branches are zero (wo = w2 = 0)."""
    buf = U.packed(SHAPE)
    t = U.tensors(SHAPE, buf)
    for l in range(SHAPE.n_layers):
        t[("wo", l)][...] = 0
        t[("w2", l)][...] = 0
    model = U.model(SHAPE, buf)
    d, m = SHAPE.d_model, 16
    tokens = np.array([[33, 8, 39]])
    cache = M.Cache(model.cfg, 1, 8)
    logits, h_pre = M.forward(model, cache, tokens, np.array([0]))
    hb = Dr.Head(d, m, _head_bits(d, m, w0=_eye_bits(d, 2 * d, d), w2=np.zeros((d, m))))
    junk = np.random.default_rng(1).normal(size=(3, d))  # h is ignored by this head
    _, lg = Dr.draft(model, hb, junk, tokens.reshape(-1))
    assert np.allclose(lg, logits.reshape(3, -1), rtol=1e-12, atol=1e-12)


def test_gate_zero_removes_the_mlp_branch():
    """W1 = 0: silu(0) = 0, so h_hat no longer depends on W2, W3 or the gain."""
    d, m = 32, 40
    rng = np.random.default_rng(2)
    h, e = rng.normal(size=(4, d)), rng.normal(size=(4, d))
    bits = _head_bits(d, m, w1=np.zeros((m, d)))
    a, b = Dr.Head(d, m, bits), Dr.Head(d, m, bits)
    b.g, b.w3, b.w2 = rng.normal(size=d), rng.normal(size=(m, d)), rng.normal(size=(d, m))
    assert np.array_equal(Dr.f_phi(a, h, e, 1e-5), Dr.f_phi(b, h, e, 1e-5))
    # with W1 != 0 the branch is live: changing W2 changes h_hat
    c = Dr.Head(d, m, _head_bits(d, m))
    c2 = Dr.Head(d, m, _head_bits(d, m))
    c2.w2 = rng.normal(size=(d, m))
    assert not np.allclose(Dr.f_phi(c, h, e, 1e-5), Dr.f_phi(c2, h, e, 1e-5))


def test_norm_sits_on_the_branch_input():
    """With eps = 0 the RMSNorm makes the SwiGLU branch invariant to scaling z, so
    h_hat(lam z) - h_hat(z) = (lam - 1) W0 z, and W0 z is the head with W2 = 0."""
    d, m = 32, 64
    full = Dr.Head(d, m, _head_bits(d, m))
    lin = Dr.Head(d, m, _head_bits(d, m, w2=np.zeros((d, m))))
    rng = np.random.default_rng(4)
    h, e = rng.normal(size=(6, d)), rng.normal(size=(6, d))
    for lam in (0.5, 3.0):
        lhs = Dr.f_phi(full, lam * h, lam * e, 0.0) - Dr.f_phi(full, h, e, 0.0)
        rhs = (lam - 1.0) * Dr.f_phi(lin, h, e, 0.0)
        assert np.allclose(lhs, rhs, rtol=1e-11, atol=1e-11)
    # and the branch is really there: with W2 != 0 the head is not linear in z
    assert not np.allclose(Dr.f_phi(full, 2 * h, 2 * e, 0.0), 2 * Dr.f_phi(full, h, e, 0.0))


def test_rows_are_independent():
    buf = U.packed(SHAPE)
    model = U.model(SHAPE, buf)
    d, m = SHAPE.d_model, 48
    hb = Dr.Head(d, m, _head_bits(d, m))
    rng = np.random.default_rng(6)
    h = rng.normal(size=(7, d))
    tok = rng.integers(0, SHAPE.vocab, size=7)
    idx, lg = Dr.draft(model, hb, h, tok)
    for r in range(7):
        i1, l1 = Dr.draft(model, hb, h[r:r + 1], tok[r:r + 1])
        assert i1[0] == idx[r] and np.allclose(l1[0], lg[r], rtol=1e-13, atol=1e-13)


def test_argmax_ties_go_to_the_lowest_code():
    buf = U.packed(SHAPE)
    t = U.tensors(SHAPE, buf)
    lm = t[("lm_head", -1)]
    lm[SHAPE.img_lo:SHAPE.img_hi] = lm[SHAPE.img_lo]  # every image code scores alike
    model = U.model(SHAPE, buf)
    d, m = SHAPE.d_model, 48
    hb = Dr.Head(d, m, _head_bits(d, m))
    rng = np.random.default_rng(7)
    idx, lg = Dr.draft(model, hb, rng.normal(size=(5, d)), rng.integers(0, SHAPE.vocab, size=5))
    assert np.all(lg == lg[:, :1])
    assert np.all(idx == 0)


def test_head_norm_epsilon_closed_form():
    """The head's RMSNorm adds the backbone's epsilon inside the root: with
    W0 = [I | 0], gain 1 and W1 = W3 = W2 = I, an input state of constant
    entries c with c^2 = eps normalizes to 1/sqrt(2) in every entry, so
    h_hat = c + silu(1/sqrt(2)) / sqrt(2)."""
    d = m = 8
    eps = 1e-5
    eye = _eye_bits(d, d, 0)
    head = Dr.Head(d, m, _head_bits(d, m, w0=_eye_bits(d, 2 * d, 0), g=np.full(d, ONE), w1=eye, w3=eye, w2=eye))
    c = np.sqrt(eps)
    h = np.full((1, d), c)
    e = np.random.default_rng(0).normal(size=(1, d))
    n = 1.0 / np.sqrt(2.0)
    want = c + n * n / (1.0 + np.exp(-n))
    assert np.allclose(Dr.f_phi(head, h, e, eps), want, rtol=1e-13, atol=0)
