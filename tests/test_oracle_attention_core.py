"""Pins of the oracle's attention core: rotary embedding on queries and keys at
their raster positions, the rotary base, the 1/sqrt(D) score scale and the
softmax (Sec. 3.1 Eq. 1: the frozen backbone scores every raster position;
Sec. 3.3 "Verification as Auto Correction": a drafted block passes through that
same backbone, each position attending to the cache and the block up to itself).

Two independent routes fix these parts:

* a closed form.  One head with D = 8 whose raw query and key are fixed
  combinations of the rotary basis vectors.  Rotating both by their positions
  makes the score of query i against key j a trigonometric function of i - j
  alone, a*b*cos((i-j) w) + a*b'*sin((i-j) w) + ..., with w the pair's rotary
  frequency theta^(-2j/D).  The expected attention weights follow from that
  identity and a softmax, not from rotating vectors.
* a textbook block written against torch (CPU, float64): rotary embedding as
  multiplication of the (x_j, x_{j+D/2}) pairs by unit complex numbers, and
  torch's own scaled_dot_product_attention (default scale 1/sqrt(D), grouped
  KV heads by its enable_gqa option) for the attention.

Mistakes each of these catches: no rotation of q or of k, q and k rotated at
different positions, a different rotary base, a rotation in the wrong
direction, scores divided by D or not scaled, a sharpened or flattened softmax.
"""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import model as M
from tests import oracle_util as U

THETA = 10000.0


def _one_head_model(D=8, vocab=12, theta_used=THETA):
    """One layer, one head, d = D; attention gain 1, Wv = Wo = I, MLP off.
    h_pre = x + o, so the attention output is observable exactly."""
    shape = synth.ModelShape(1, D, 1, 1, D, 4, vocab, vocab, "f32")
    buf = U.packed(shape, seed=3, std=0.3, gain_std=0.0)
    T = U.tensors(shape, buf)
    T[("attn_norm", 0)][:] = 1.0
    T[("wv", 0)][:] = np.eye(D, dtype=np.float32)
    T[("wo", 0)][:] = np.eye(D, dtype=np.float32)
    T[("w2", 0)][:] = 0
    return shape, buf, T


def _rotary_freqs(D, theta):
    # pair j (dims j and j + D/2) turns by theta^(-2j/D) radians per position
    return np.array([theta ** (-2.0 * j / D) for j in range(D // 2)])


def _closed_form_attention(x, rinv, qa, kb, D, theta, positions):
    """Expected h_pre for the one-head model.

    x     -- (n, D) token embeddings, rinv -- (n,) 1/rms of each row
    qa    -- raw query direction: dict {dim: coefficient}, applied as q = rinv * x[0] * qa
    kb    -- raw key direction, same convention
    The raw query of token i is rinv_i * x_i[0] * sum_c qa[c] e_c (Wq has
    column 0 only); after rotation by position angle the inner product of a
    rotated e_c (query at i) and a rotated e_e (key at j) is
      same pair, c = e:                 cos(dt)
      c = j, e = j + D/2 (partner):    +sin(dt)   with dt = (i - j) w_j
      c = j + D/2, e = j:              -sin(dt)
    and 0 across different pairs."""
    half = D // 2
    w = _rotary_freqs(D, theta)
    n = x.shape[0]
    out = np.zeros_like(x)
    v = x * rinv[:, None]  # Wv = I, gain 1
    for i in range(n):
        s = np.empty(i + 1)
        for j in range(i + 1):
            tot = 0.0
            for c, a in qa.items():
                for e, b in kb.items():
                    if c % half != e % half:
                        continue
                    dt = (positions[i] - positions[j]) * w[c % half]
                    if c == e:
                        val = math.cos(dt)
                    elif c < half:      # query on the first half, key on its partner
                        val = math.sin(dt)
                    else:               # query on the second half, key on its partner
                        val = -math.sin(dt)
                    tot += a * b * val
            s[j] = tot * (rinv[i] * x[i, 0]) * (rinv[j] * x[j, 0]) / math.sqrt(D)
        p = np.exp(s - s.max())
        p /= p.sum()
        out[i] = x[i] + p @ v[: i + 1]
    return out


def _set_direction(W, coeffs):
    """Wq or Wk with column 0 only; returns the coefficients as stored (float32)."""
    W[:] = 0
    for dim, c in coeffs.items():
        W[dim, 0] = c
    return {dim: float(W[dim, 0]) for dim in coeffs}


@pytest.mark.parametrize("case", ["pair0", "pair1-sine", "mixed"])
def test_rotary_attention_closed_form(case):
    D = 8
    shape, buf, T = _one_head_model(D)
    qa, kb = {
        # pair 0 turns 1 rad per position: cosine of the distance
        "pair0": ({0: 2.0}, {0: 1.5}),
        # query on dim 1, key on its partner dim 5 (pair 1, 0.1 rad per position):
        # the score is an odd function of i - j, so the rotation's direction matters
        "pair1-sine": ({1: 3.0}, {5: 2.5}),
        # both pairs at once: the frequencies of pairs 0 and 1 both enter
        "mixed": ({0: 1.0, 1: 2.0, 4: -0.7}, {0: 1.2, 5: -1.8, 1: 0.9}),
    }[case]
    qa = _set_direction(T[("wq", 0)], qa)
    kb = _set_direction(T[("wk", 0)], kb)
    toks = np.array([[3, 7, 1, 9, 4, 11, 2]])
    x = T[("tok_emb", -1)][toks[0]].astype(np.float64)
    # keep x[:,0] away from zero so every score is far from flat
    x[:, 0] = np.where(np.abs(x[:, 0]) < 0.2, 0.5, x[:, 0])
    T[("tok_emb", -1)][toks[0], 0] = x[:, 0].astype(np.float32)
    x = T[("tok_emb", -1)][toks[0]].astype(np.float64)
    rinv = 1.0 / np.sqrt(np.mean(x * x, axis=1) + 1e-5)
    want = _closed_form_attention(x, rinv, qa, kb, D, THETA, np.arange(toks.shape[1]))
    _, h = M.forward_nocache(U.model(shape, buf), toks)
    assert np.allclose(h[0], want, rtol=0, atol=1e-12)
    # the attention is far from uniform, so a wrong scale would show
    flat = _closed_form_attention(x, rinv, {}, {}, D, THETA, np.arange(toks.shape[1]))
    assert np.abs(want - flat).max() > 0.05


def test_rotary_attention_closed_form_in_a_later_block():
    """The same closed form for a block at absolute positions 5..8 over a cached
    prefix 0..4: queries and keys of the block and keys of the cache are rotated
    at their own raster positions."""
    D = 8
    shape, buf, T = _one_head_model(D)
    qa, kb = {0: 1.0, 1: 2.0}, {4: 1.1, 1: 1.3}
    qa = _set_direction(T[("wq", 0)], qa)
    kb = _set_direction(T[("wk", 0)], kb)
    toks = np.array([[3, 7, 1, 9, 4, 11, 2, 6, 10]])
    T[("tok_emb", -1)][:, 0] = np.where(np.abs(T[("tok_emb", -1)][:, 0]) < 0.2, 0.6,
                                       T[("tok_emb", -1)][:, 0])
    mod = U.model(shape, buf)
    c = M.Cache(mod.cfg, 1, 9)
    M.forward(mod, c, toks[:, :5], [0])
    _, h = M.forward(mod, c, toks[:, 5:], [5])
    x = T[("tok_emb", -1)][toks[0]].astype(np.float64)
    rinv = 1.0 / np.sqrt(np.mean(x * x, axis=1) + 1e-5)
    want = _closed_form_attention(x, rinv, qa, kb, D, THETA, np.arange(9))
    assert np.allclose(h[0], want[5:], rtol=0, atol=1e-12)


def test_two_key_softmax_is_logistic():
    """Two tokens, raw query a e0 and raw key b e0 (pair 0, 1 rad per position):
    the second query's scores differ by a b r1 x1 (r1 x1 - r0 x0 cos 1) / sqrt(D)
    between key 1 and key 0, and its weight on key 1 is the logistic function of
    that difference."""
    D = 8
    shape, buf, T = _one_head_model(D)
    a, b = 0.8, 0.6
    a = _set_direction(T[("wq", 0)], {0: a})[0]
    b = _set_direction(T[("wk", 0)], {0: b})[0]
    toks = np.array([[4, 9]])
    T[("tok_emb", -1)][4, 0] = 0.9
    T[("tok_emb", -1)][9, 0] = -0.8
    x = T[("tok_emb", -1)][toks[0]].astype(np.float64)
    r = 1.0 / np.sqrt(np.mean(x * x, axis=1) + 1e-5)
    q1 = a * r[1] * x[1, 0]
    s11 = q1 * b * r[1] * x[1, 0] / math.sqrt(D)
    s10 = q1 * b * r[0] * x[0, 0] * math.cos(1.0) / math.sqrt(D)
    w1 = 1.0 / (1.0 + math.exp(-(s11 - s10)))
    v = x * r[:, None]
    want = x[1] + (1 - w1) * v[0] + w1 * v[1]
    _, h = M.forward_nocache(U.model(shape, buf), toks)
    assert np.allclose(h[0, 1], want, rtol=0, atol=1e-12)
    assert 0.05 < w1 < 0.95 and abs(w1 - 0.5) > 0.1


# ---------------------------------------------------------------------------
# textbook block in torch (float64, CPU)


def _rotate_complex(x, pos, D, theta):
    """x (..., n, H, D) rotated at positions pos (n,): the pairs (x_j, x_{j+D/2})
    taken as complex numbers and multiplied by exp(i * pos * theta^(-2j/D))."""
    half = D // 2
    freqs = theta ** (-torch.arange(half, dtype=torch.float64) * 2.0 / D)
    ang = pos.to(torch.float64)[:, None] * freqs[None, :]  # (n, half)
    rot = torch.polar(torch.ones_like(ang), ang)[:, None, :]  # (n, 1, half)
    z = torch.complex(x[..., :half], x[..., half:]) * rot
    return torch.cat([z.real, z.imag], dim=-1)


def _rms_norm(x, g, eps=1e-5):
    return x * torch.rsqrt((x * x).mean(-1, keepdim=True) + eps) * g


def _torch_forward(shape, buf, tokens, round_kv):
    T = {k: torch.from_numpy(np.asarray(
        M.bf16_bits_to_f64(v) if shape.dtype == "bf16" else v, dtype=np.float64).copy())
        for k, v in U.tensors(shape, buf).items()}
    Hq, Hkv, D = shape.n_heads, shape.n_kv_heads, shape.head_dim
    tok = torch.from_numpy(np.asarray(tokens))
    n = tok.shape[1]
    pos = torch.arange(n)
    x = T[("tok_emb", -1)][tok]  # (1, n, d)
    for l in range(shape.n_layers):
        h = _rms_norm(x, T[("attn_norm", l)])
        q = (h @ T[("wq", l)].T).view(1, n, Hq, D)
        k = (h @ T[("wk", l)].T).view(1, n, Hkv, D)
        v = (h @ T[("wv", l)].T).view(1, n, Hkv, D)
        q = _rotate_complex(q, pos, D, THETA)
        k = _rotate_complex(k, pos, D, THETA)
        if round_kv:
            k = k.float().bfloat16().double()
            v = v.float().bfloat16().double()
        o = torch.nn.functional.scaled_dot_product_attention(
            q.transpose(1, 2), k.transpose(1, 2), v.transpose(1, 2), is_causal=True,
            enable_gqa=(Hq != Hkv))
        x = x + o.transpose(1, 2).reshape(1, n, Hq * D) @ T[("wo", l)].T
        h = _rms_norm(x, T[("mlp_norm", l)])
        x = x + (torch.nn.functional.silu(h @ T[("w1", l)].T) * (h @ T[("w3", l)].T)) @ T[("w2", l)].T
    logits = _rms_norm(x, T[("final_norm", -1)]) @ T[("lm_head", -1)][shape.img_lo:].T
    return logits.numpy(), x.numpy()


@pytest.mark.parametrize("shape", [U.TINY_GQA, U.TINY_BF16,
                                   synth.ModelShape(2, 64, 2, 2, 32, 96, 50, 40, "f32")],
                         ids=["gqa-f32", "gqa-bf16", "mha-D32"])
def test_forward_equals_textbook_block(shape):
    buf = U.packed(shape, seed=7, std=0.25, gain_std=0.1)
    rng = np.random.default_rng(11)
    toks = rng.integers(0, shape.vocab, size=(1, 14))
    l_or, h_or = M.forward_nocache(U.model(shape, buf), toks)
    l_t, h_t = _torch_forward(shape, buf, toks, round_kv=(shape.dtype == "bf16"))
    tol = 1e-10 if shape.dtype == "f32" else 1e-6
    assert np.allclose(h_or[0], h_t[0], rtol=0, atol=tol)
    assert np.allclose(l_or[0], l_t[0], rtol=0, atol=tol)
    assert np.abs(l_t).max() > 0.1


def test_textbook_block_sees_rotation_and_scale():
    """The torch block itself reacts to the parts pinned above (so agreement
    with it is informative): other theta or no rotation changes its output."""
    shape = U.TINY_GQA
    buf = U.packed(shape, seed=7, std=0.25, gain_std=0.1)
    toks = np.random.default_rng(11).integers(0, shape.vocab, size=(1, 14))
    l_ref, _ = _torch_forward(shape, buf, toks, round_kv=False)
    global THETA
    saved = THETA
    try:
        THETA = 10.0 * saved
        l_other, _ = _torch_forward(shape, buf, toks, round_kv=False)
    finally:
        THETA = saved
    assert np.abs(l_ref - l_other).max() > 1e-3
