"""Pins of the oracle's backbone forward pass (Sec. 3.1 Eq. 1; Sec. 3.3).

Closed forms for special weight settings, exact invariants of causal
attention with a KV cache, and equivalences that any correct implementation
satisfies.  Each is chosen so that a plausible slip -- a transposed weight, a
mask that is off by one, a wrong KV-head mapping, rotary pairs or frequencies
mixed up, a missing gain or 1/rms -- fails at least one of them.
"""
import math

import numpy as np
import pytest

import synth
from oracle import model as M
from tests import oracle_util as U

F32 = U.TINY_GQA


def _fresh(shape=F32, **kw):
    buf = U.packed(shape, **kw)
    return buf, U.tensors(shape, buf)


def test_layout_size_matches_generator():
    for shp in (F32, synth.TINY, synth.M1B):
        assert sum(int(np.prod(s)) for _, _, s in M.layout(U.config_of(shp))) == synth.n_params(shp)


def test_rope_closed_form():
    # D = 4, theta = 1e4: frequencies 1 and 1e-2; rotate-half pairs (0,2), (1,3)
    inv = 10000.0 ** (-(2.0 * np.arange(2)) / 4)
    assert np.allclose(inv, [1.0, 0.01])
    for p in (0, 1, 7, 300):
        e0 = M.rope(np.array([1.0, 0, 0, 0]).reshape(1, 1, 1, 4), np.array([[p]]), inv).ravel()
        assert np.allclose(e0, [math.cos(p), 0, math.sin(p), 0], atol=1e-15)
        e1 = M.rope(np.array([0, 1.0, 0, 0]).reshape(1, 1, 1, 4), np.array([[p]]), inv).ravel()
        assert np.allclose(e1, [0, math.cos(0.01 * p), 0, math.sin(0.01 * p)], atol=1e-15)
        e2 = M.rope(np.array([0, 0, 1.0, 0]).reshape(1, 1, 1, 4), np.array([[p]]), inv).ravel()
        assert np.allclose(e2, [-math.sin(p), 0, math.cos(p), 0], atol=1e-15)


def test_rope_relative_position():
    rng = np.random.default_rng(0)
    D = 16
    inv = 10000.0 ** (-(2.0 * np.arange(D // 2)) / D)
    q = rng.normal(size=(1, 1, 1, D))
    k = rng.normal(size=(1, 1, 1, D))
    for m, n, c in [(5, 2, 11), (100, 37, 1000), (3, 3, 4)]:
        s1 = (M.rope(q, np.array([[m]]), inv) * M.rope(k, np.array([[n]]), inv)).sum()
        s2 = (M.rope(q, np.array([[m + c]]), inv) * M.rope(k, np.array([[n + c]]), inv)).sum()
        assert abs(s1 - s2) < 1e-10
        # rotation preserves the norm
        assert abs(np.linalg.norm(M.rope(q, np.array([[m]]), inv)) - np.linalg.norm(q)) < 1e-12


def test_final_norm_and_head_one_hot_closed_form():
    """Residual branches off (Wo = W2 = 0): h_pre = E[t].  With E[t] = s * e_j the
    RMSNorm gives sqrt(d) * e_j (up to eps), so logit v = g_f[j] sqrt(d) Wlm[v, j]."""
    buf, T = _fresh()
    for l in range(F32.n_layers):
        T[("wo", l)][:] = 0
        T[("w2", l)][:] = 0
    tok, j, s = F32.img_lo + 3, 5, float(np.float32(0.7))
    T[("tok_emb", -1)][tok] = 0
    T[("tok_emb", -1)][tok, j] = s
    mod = U.model(F32, buf)
    logits, h = M.forward_nocache(mod, np.array([[tok]]))
    d = F32.d_model
    assert np.allclose(h[0, 0], T[("tok_emb", -1)][tok].astype(np.float64), atol=0)
    scale = s / math.sqrt(s * s / d + 1e-5)
    want = float(T[("final_norm", -1)][j]) * scale * T[("lm_head", -1)][F32.img_lo:, j].astype(np.float64)
    assert np.allclose(logits[0, 0], want, rtol=1e-12, atol=1e-14)
    assert logits.shape == (1, 1, F32.v_img)


def test_single_key_attention_is_value():
    """One token, one layer: softmax over one key is 1, so the attention output
    of head h is the value of KV head h // g; with Wo = I and the MLP off,
    h_pre = x + concat_h v_{h//g}."""
    shape = synth.ModelShape(1, 32, 4, 2, 8, 48, 40, 32, "f32")
    buf, T = _fresh(shape)
    T[("wo", 0)][:] = np.eye(32, dtype=np.float32)
    T[("w2", 0)][:] = 0
    mod = U.model(shape, buf)
    tok = 11
    _, h = M.forward_nocache(mod, np.array([[tok]]))
    x = T[("tok_emb", -1)][tok].astype(np.float64)
    rinv = 1.0 / math.sqrt(np.mean(x * x) + 1e-5)
    v = (T[("wv", 0)].astype(np.float64) @ (T[("attn_norm", 0)] * x)) * rinv  # (Hkv*D,)
    v = v.reshape(2, 8)
    want = x + np.concatenate([v[0], v[0], v[1], v[1]])
    assert np.allclose(h[0, 0], want, rtol=1e-12, atol=1e-13)


def test_uniform_attention_is_causal_mean():
    """Wq = 0 makes every score 0: query k averages the values of positions 0..k
    exactly (mask extent and cache slots); Wo = I, MLP off, one layer."""
    shape = synth.ModelShape(1, 32, 4, 4, 8, 48, 40, 32, "f32")
    buf, T = _fresh(shape)
    T[("wq", 0)][:] = 0
    T[("wo", 0)][:] = np.eye(32, dtype=np.float32)
    T[("w2", 0)][:] = 0
    mod = U.model(shape, buf)
    toks = np.array([[3, 17, 25, 9, 30, 1]])
    _, h = M.forward_nocache(mod, toks)
    x = T[("tok_emb", -1)][toks[0]].astype(np.float64)  # (n, d)
    rinv = 1.0 / np.sqrt(np.mean(x * x, axis=1) + 1e-5)
    v = ((T[("attn_norm", 0)] * x) @ T[("wv", 0)].astype(np.float64).T) * rinv[:, None]
    for k in range(toks.shape[1]):
        assert np.allclose(h[0, k], x[k] + v[:k + 1].mean(axis=0), rtol=1e-12, atol=1e-13)


def test_swiglu_one_hot_closed_form():
    """Attention off, x = s e_0, W1 = a E00, W3 = c E00, W2 = E00, gains 1:
    h_pre[0] = s + silu(a sqrt(d)') * c sqrt(d)' with sqrt(d)' = s / rms(x);
    sigmoid(ln 3) = 3/4 picks a = ln 3 / sqrt(d)'."""
    shape = synth.ModelShape(1, 16, 2, 2, 8, 8, 20, 16, "f32")
    buf, T = _fresh(shape, gain_std=0.0)
    T[("wo", 0)][:] = 0
    for n in ("w1", "w3", "w2"):
        T[(n, 0)][:] = 0
    s = 0.5
    nrm = s / math.sqrt(s * s / 16 + 1e-5)
    a = math.log(3.0) / nrm
    c = 0.25
    T[("w1", 0)][0, 0] = a
    T[("w3", 0)][0, 0] = c
    T[("w2", 0)][0, 0] = 1.0
    tok = 2
    T[("tok_emb", -1)][tok] = 0
    T[("tok_emb", -1)][tok, 0] = s
    mod = U.model(shape, buf)
    _, h = M.forward_nocache(mod, np.array([[tok]]))
    a32, c32 = float(np.float32(a)), float(np.float32(c))
    z = a32 * nrm
    want0 = s + (z / (1 + math.exp(-z))) * c32 * nrm
    assert abs(float(np.float32(a)) * nrm - math.log(3.0)) < 1e-6
    assert abs(h[0, 0, 0] - want0) < 1e-12
    assert np.all(h[0, 0, 1:] == 0)


def test_causality():
    buf, _ = _fresh()
    mod = U.model(F32, buf)
    rng = np.random.default_rng(1)
    toks = rng.integers(0, F32.vocab, size=(1, 12))
    l1, h1 = M.forward_nocache(mod, toks)
    toks2 = toks.copy()
    toks2[0, 7] = (toks2[0, 7] + 5) % F32.vocab
    l2, h2 = M.forward_nocache(mod, toks2)
    assert np.array_equal(l1[:, :7], l2[:, :7]) and np.array_equal(h1[:, :7], h2[:, :7])
    assert not np.allclose(l1[:, 7:], l2[:, 7:])


@pytest.mark.parametrize("shape", [F32, U.TINY_BF16], ids=["f32", "bf16"])
def test_block_equals_token_by_token(shape):
    buf, _ = _fresh(shape)
    mod = U.model(shape, buf)
    rng = np.random.default_rng(2)
    B, P, K = 2, 5, 7
    pre = rng.integers(0, shape.vocab, size=(B, P))
    blk = rng.integers(shape.img_lo, shape.vocab, size=(B, K))
    c1 = M.Cache(mod.cfg, B, P + K)
    M.forward(mod, c1, pre, np.zeros(B, int))
    c2 = c1.copy()
    lb, hb = M.forward(mod, c1, blk, np.full(B, P))
    for k in range(K):
        lk, hk = M.forward(mod, c2, blk[:, k:k + 1], np.full(B, P + k))
        tol = 1e-12 if shape.dtype == "f32" else 1e-9
        assert np.allclose(lk[:, 0], lb[:, k], rtol=0, atol=tol)
        assert np.allclose(hk[:, 0], hb[:, k], rtol=0, atol=tol)
    assert np.allclose(c1.k, c2.k, atol=1e-12) and np.allclose(c1.v, c2.v, atol=1e-12)


def test_cache_equals_recompute():
    buf, _ = _fresh()
    mod = U.model(F32, buf)
    rng = np.random.default_rng(3)
    seq = rng.integers(0, F32.vocab, size=(2, 15))
    lfull, hfull = M.forward_nocache(mod, seq)
    c = M.Cache(mod.cfg, 2, 15)
    M.forward(mod, c, seq[:, :6], np.zeros(2, int))
    l2, _ = M.forward(mod, c, seq[:, 6:10], np.full(2, 6))
    l3, h3 = M.forward(mod, c, seq[:, 10:], np.full(2, 10))
    assert np.allclose(l2, lfull[:, 6:10], rtol=0, atol=1e-12)
    assert np.allclose(l3, lfull[:, 10:], rtol=0, atol=1e-12)
    assert np.allclose(h3, hfull[:, 10:], rtol=0, atol=1e-12)


def test_provisional_block_overwrite():
    """Re-running a block at the same frontier replaces its KV slots: the result
    equals a fresh run on the second block."""
    buf, _ = _fresh()
    mod = U.model(F32, buf)
    rng = np.random.default_rng(4)
    pre = rng.integers(0, F32.vocab, size=(1, 4))
    b1 = rng.integers(F32.img_lo, F32.vocab, size=(1, 5))
    b2 = rng.integers(F32.img_lo, F32.vocab, size=(1, 5))
    c = M.Cache(mod.cfg, 1, 9)
    M.forward(mod, c, pre, [0])
    c0 = c.copy()
    M.forward(mod, c, b1, [4])
    la, _ = M.forward(mod, c, b2, [4])
    lb, _ = M.forward(mod, c0, b2, [4])
    assert np.array_equal(la, lb)


def test_gqa_equals_mha_with_shared_kv():
    shape = F32
    buf, T = _fresh(shape)
    mha = synth.ModelShape(shape.n_layers, shape.d_model, 4, 4, 8, shape.d_ff, shape.vocab, shape.v_img, "f32")
    buf2 = synth.weights(mha, seed=9)
    T2 = U.tensors(mha, buf2)
    for key, arr in T.items():
        name, l = key
        if name in ("wk", "wv"):
            # query head h reads KV head h // 2: duplicate each KV head's rows
            a = arr.reshape(2, 8, -1)
            T2[key][:] = np.repeat(a, 2, axis=0).reshape(32, -1)
        else:
            T2[key][:] = arr
    rng = np.random.default_rng(5)
    seq = rng.integers(0, shape.vocab, size=(1, 9))
    la, ha = M.forward_nocache(U.model(shape, buf), seq)
    lb, hb = M.forward_nocache(U.model(mha, buf2), seq)
    assert np.allclose(la, lb, rtol=0, atol=1e-12) and np.allclose(ha, hb, rtol=0, atol=1e-12)


def test_batch_rows_independent():
    buf, _ = _fresh()
    mod = U.model(F32, buf)
    rng = np.random.default_rng(6)
    seq = rng.integers(0, F32.vocab, size=(3, 8))
    l, h = M.forward_nocache(mod, seq)
    for b in range(3):
        lb, hb = M.forward_nocache(mod, seq[b:b + 1])
        assert np.allclose(lb[0], l[b], rtol=0, atol=1e-12)


def test_bf16_rounding_points():
    buf, _ = _fresh(U.TINY_BF16)
    mod = U.model(U.TINY_BF16, buf)
    seq = np.array([[1, 5, 9, 33, 39]])
    c = M.Cache(mod.cfg, 1, 5)
    l, h = M.forward(mod, c, seq, [0])
    # the cache holds bf16 values only
    assert np.array_equal(M.bf16_round(c.k), c.k) and np.array_equal(M.bf16_round(c.v), c.v)
    # same bf16-valued weights in an fp32 model: close but not identical
    f32shape = synth.ModelShape(2, 32, 4, 2, 8, 48, 40, 32, "f32")
    buf32 = M.bf16_bits_to_f64(buf).astype(np.float32)
    l32, _ = M.forward_nocache(U.model(f32shape, buf32), seq)
    assert not np.array_equal(l, l32)
    assert np.abs(l - l32).max() < 0.05 * np.abs(l32).max()


def test_bf16_round_ties_to_even():
    one = 1.0
    ulp = 2.0 ** -7
    assert M.bf16_round(np.array([one + ulp / 2]))[0] == one          # tie -> even
    assert M.bf16_round(np.array([one + 1.5 * ulp]))[0] == one + 2 * ulp
    assert M.bf16_round(np.array([one + 0.51 * ulp]))[0] == one + ulp
    assert M.bf16_round(np.array([-3.0]))[0] == -3.0


def test_batch_rows_at_different_frontiers():
    """Rows of one batched block at different positions: each row's queries and
    keys are rotated at its own positions and see its own context only, so
    each row's logits and states equal a no-cache recompute of that row's own
    sequence (here row 1's block overwrites the last two slots of its prefix)."""
    buf, _ = _fresh()
    mod = U.model(F32, buf)
    rng = np.random.default_rng(9)
    pre = rng.integers(0, F32.vocab, size=(2, 4))
    blk = rng.integers(0, F32.vocab, size=(2, 3))
    c = M.Cache(mod.cfg, 2, 8)
    M.forward(mod, c, pre, np.array([0, 0]))
    starts = np.array([4, 2])
    l, h = M.forward(mod, c, blk, starts)
    for b in range(2):
        seq = np.concatenate([pre[b, :starts[b]], blk[b]])[None, :]
        lf, hf = M.forward_nocache(mod, seq)
        assert np.allclose(l[b], lf[0, -3:], rtol=0, atol=1e-12), b
        assert np.allclose(h[b], hf[0, -3:], rtol=0, atol=1e-12), b
