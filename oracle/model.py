"""Backbone forward pass with a KV cache (oracle, test infrastructure).

Paper: Sec. 3.1, Eq. 1 -- a decoder-only transformer predicts raster-ordered
image tokens t_i ~ p(t_i | c, t_1..t_{i-1}) after a text prefix c.  Sec. 3.3
("Verification as Auto Correction") passes a whole drafted block through the
same frozen, unmodified backbone in one forward pass; position k of the block
sees the committed cache and the block tokens up to itself.  Sec. 3.3
("Draft Prediction in Latent Space") names the pieces used here: RMSNorm, the
last layer's pre-norm hidden state h_pre, and the GenHead output layer; the
SwiGLU form W2(silu(W1 z) * W3 z) is the one Eq. 2 writes out.

The paper does not print the backbone's equations; this is the standard
LLaMA-style block its backbones share (these readings fill in what it leaves open):
pre-RMSNorm (eps 1e-5), rotary embedding on raster positions (rotate-half
pairing, theta 1e4), causal softmax attention with 1/sqrt(D) scaling and
grouped KV heads (query head h uses KV head h // (Hq/Hkv)), SwiGLU MLP, no
biases, untied embedding and output layer, logits restricted to the image-code
range [img_lo, img_hi).

Precision contract (bf16 models; an fp32 model rounds nowhere).  The paper
fixes no arithmetic precision; its memory figures imply bf16 weights.  Here
the stored state is bf16 and the transient activations are not rounded:
  * weights and the KV cache hold bf16 values: k is rounded after the rotary
    embedding, v after its projection (rho = round-to-nearest-even to bf16);
  * RMSNorm is the plain definition n = g * x / sqrt(mean(x^2) + eps), and a
    linear layer after it is n @ W^T (a kernel may apply the per-row 1/rms
    after the product instead; the two agree up to rounding);
  * everything else (residual stream, q, attention weights and output, the
    SwiGLU product, logits) stays unrounded float64.
Rounding activations to bf16 as well would make the comparison meaningless
for deep random-init models: each rounding is a discontinuity, and a 1e-7
relative change of the input then moves the 24-layer model's logits by
~3e-2, while with bf16 state only it moves them by ~5e-4.

Pins: tests/test_oracle_model.py -- closed-form special cases (single key,
zero residual branches, rotary rotation), causality, batched block == one
token at a time, cached == uncached recompute, relative-position property of
the rotation, GQA == MHA with duplicated KV heads, batch-row independence;
tests/test_oracle_attention_core.py -- attention weights of a one-head model
in closed form (scores a trigonometric function of the query-key distance:
rotation of q and k at their raster positions, the rotary base, 1/sqrt(D),
the softmax), in the first block and in a later block over a cache, and the
whole forward pass against a textbook block written with torch's own
attention routine and complex-number rotation.

This module is test infrastructure: only the tests, the smoke check and the
benchmark's CPU baseline use it.
"""

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Config:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    img_lo: int
    img_hi: int
    dtype: str  # "f32" or "bf16"
    rms_eps: float = 1e-5
    rope_theta: float = 10000.0

    @property
    def v_img(self):
        return self.img_hi - self.img_lo


def layout(cfg):
    """(name, layer, shape) of every tensor of the packed weight buffer, in order."""
    d, D, m = cfg.d_model, cfg.head_dim, cfg.d_ff
    out = [("tok_emb", -1, (cfg.vocab, d))]
    for l in range(cfg.n_layers):
        out += [
            ("attn_norm", l, (d,)),
            ("wq", l, (cfg.n_heads * D, d)),
            ("wk", l, (cfg.n_kv_heads * D, d)),
            ("wv", l, (cfg.n_kv_heads * D, d)),
            ("wo", l, (d, cfg.n_heads * D)),
            ("mlp_norm", l, (d,)),
            ("w1", l, (m, d)),
            ("w3", l, (m, d)),
            ("w2", l, (d, m)),
        ]
    out += [("final_norm", -1, (d,)), ("lm_head", -1, (cfg.vocab, d))]
    return out


def bf16_round(x):
    """Round float64 values to the nearest bf16 (via float32, ties to even)."""
    a = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    a = (a + 0x7FFF + ((a >> 16) & 1)) & 0xFFFF0000
    return a.astype(np.uint32).view(np.float32).astype(np.float64)


def bf16_bits_to_f64(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


class Model:
    """Weights unpacked from the packed buffer into float64 arrays."""

    def __init__(self, cfg, packed):
        self.cfg = cfg
        if cfg.dtype == "bf16":
            assert packed.dtype == np.uint16
            conv = bf16_bits_to_f64
            self.rho = bf16_round
        elif cfg.dtype == "f32":
            assert packed.dtype == np.float32
            conv = lambda a: np.asarray(a, dtype=np.float64)  # noqa: E731
            self.rho = lambda a: a  # noqa: E731
        else:
            raise ValueError(cfg.dtype)
        off = 0
        self.layers = [dict() for _ in range(cfg.n_layers)]
        for name, l, shape in layout(cfg):
            n = int(np.prod(shape))
            t = conv(packed[off:off + n]).reshape(shape)
            off += n
            if l >= 0:
                self.layers[l][name] = t
            else:
                setattr(self, name, t)
        assert off == packed.shape[0], "packed buffer size does not match the config"
        self.lm_img = self.lm_head[cfg.img_lo:cfg.img_hi]
        half = cfg.head_dim // 2
        self.inv_freq = cfg.rope_theta ** (-(2.0 * np.arange(half)) / cfg.head_dim)


class Cache:
    """KV cache [L][B][Hkv][Lmax][D] in float64 (holding bf16 values for bf16 models)."""

    def __init__(self, cfg, B, max_ctx):
        shape = (cfg.n_layers, B, cfg.n_kv_heads, max_ctx, cfg.head_dim)
        self.k = np.zeros(shape)
        self.v = np.zeros(shape)
        self.max_ctx = max_ctx

    def copy(self):
        c = Cache.__new__(Cache)
        c.k, c.v, c.max_ctx = self.k.copy(), self.v.copy(), self.max_ctx
        return c


def rms_inv(x, eps):
    return 1.0 / np.sqrt(np.mean(x * x, axis=-1) + eps)


def rms_norm(x, g, eps):
    """RMSNorm over the last axis: g * x / sqrt(mean(x^2) + eps)."""
    return g * x * rms_inv(x, eps)[..., None]


def rope(x, pos, inv_freq):
    """Rotate-half rotary embedding. x: (B, K, H, D); pos: (B, K) absolute positions."""
    half = x.shape[-1] // 2
    ang = pos[:, :, None].astype(np.float64) * inv_freq[None, None, :]  # (B, K, half)
    c = np.cos(ang)[:, :, None, :]
    s = np.sin(ang)[:, :, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(x):
    return x / (1.0 + np.exp(-x))


def forward(model, cache, tokens, start):
    """Forward a block of tokens through the backbone.

    tokens -- int array (B, K) of vocabulary ids
    start  -- int array (B,) first absolute position of each row's block; the
              block occupies cache slots [start, start + K) and attends to
              slots [0, start + k] (causal over raster positions)
    Writes the block's k/v into the cache (slots [start, start+K)).
    Returns (logits (B, K, V_img), h_pre (B, K, d)) in float64.
    """
    cfg, rho = model.cfg, model.rho
    tokens = np.asarray(tokens)
    start = np.asarray(start, dtype=np.int64)
    B, K = tokens.shape
    Hq, Hkv, D = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    g = Hq // Hkv
    pos = start[:, None] + np.arange(K)[None, :]  # (B, K)
    assert int(pos.max()) < cache.max_ctx
    x = model.tok_emb[tokens]  # (B, K, d)
    for l, W in enumerate(model.layers):
        # attention block
        n1 = rms_norm(x, W["attn_norm"], cfg.rms_eps)
        q = (n1 @ W["wq"].T).reshape(B, K, Hq, D)
        k = (n1 @ W["wk"].T).reshape(B, K, Hkv, D)
        v = (n1 @ W["wv"].T).reshape(B, K, Hkv, D)
        q = rope(q, pos, model.inv_freq)
        k = rho(rope(k, pos, model.inv_freq))
        v = rho(v)
        o = np.zeros((B, K, Hq, D))
        for b in range(B):
            s0 = int(start[b])
            cache.k[l, b, :, s0:s0 + K, :] = k[b].transpose(1, 0, 2)
            cache.v[l, b, :, s0:s0 + K, :] = v[b].transpose(1, 0, 2)
            n = s0 + K
            keys = cache.k[l, b, :, :n, :]  # (Hkv, n, D)
            vals = cache.v[l, b, :, :n, :]
            visible = np.arange(n)[None, :] <= pos[b][:, None]  # (K, n)
            for h in range(Hq):
                kv = h // g
                s = (q[b, :, h, :] @ keys[kv].T) / np.sqrt(D)  # (K, n)
                s = np.where(visible, s, -np.inf)
                s = s - s.max(axis=1, keepdims=True)
                p = np.exp(s)
                p /= p.sum(axis=1, keepdims=True)
                o[b, :, h, :] = p @ vals[kv]
        o = o.reshape(B, K, Hq * D)
        x = x + o @ W["wo"].T
        # MLP block
        n2 = rms_norm(x, W["mlp_norm"], cfg.rms_eps)
        hdn = silu(n2 @ W["w1"].T) * (n2 @ W["w3"].T)
        x = x + hdn @ W["w2"].T
    h_pre = x
    logits = rms_norm(x, model.final_norm, cfg.rms_eps) @ model.lm_img.T
    return logits, h_pre


def forward_nocache(model, tokens):
    """Whole-sequence forward from position 0 without a persistent cache
    (fresh cache sized to the sequence).  Used by the cache-consistency pin."""
    tokens = np.asarray(tokens)
    B, n = tokens.shape
    c = Cache(model.cfg, B, n)
    return forward(model, c, tokens, np.zeros(B, dtype=np.int64))
