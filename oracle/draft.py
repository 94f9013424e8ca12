"""Spatial draft head f_phi (oracle, test infrastructure only).

Paper: Sec. 3.3, "Draft Prediction in Latent Space", Eq. 2.  A head predicts
the last layer's pre-norm hidden state at a spatial offset from the hidden
state h of a decoded position and the embedding e of its token:

    z     = [h; e]                                  (2d)
    u     = W0 z                                    (W0: d x 2d)
    h_hat = u + SwiGLU(RMSNorm(u)),  SwiGLU(v) = W2 (silu(W1 v) * W3 v)
                                                    (W1, W3: m x d, W2: d x m)

and the draft token is the argmax of the backbone's own output layer on the
predicted state, GenHead(RMSNorm(h_hat)) -- the backbone's final norm and LM
head, restricted to the image codes as everywhere here.

Readings where the paper leaves details open: the head's RMSNorm has a gain vector g of its
own (the paper does not name the norm's parameters; the backbone's norms carry
gains) and the backbone's epsilon; m is a free size (the paper's 134.2 M
parameters per head at d = 4096 give m = 2d); the draft distribution a rule-(C)
verification needs is the softmax of the same logits (t_hat = argmax q).
Precision contract as the backbone's (oracle/model.py): bf16 weights, float64
activations, the per-row 1/rms(u) applied after the products with g * u.

Pins: tests/test_oracle_draft.py.
"""

import numpy as np

from oracle import model as M


def head_layout(d, m):
    """(name, shape) of the packed head weights, in order."""
    return [("w0", (d, 2 * d)), ("g", (d,)), ("w1", (m, d)), ("w3", (m, d)), ("w2", (d, m))]


def head_numel(d, m):
    return int(sum(np.prod(s) for _, s in head_layout(d, m)))


class Head:
    """A draft head's weights unpacked to float64 (bf16 bits or float32 in, like the
    backbone's)."""

    def __init__(self, d, m, packed):
        assert packed.dtype in (np.uint16, np.float32) and packed.shape[0] == head_numel(d, m)
        off = 0
        for name, shape in head_layout(d, m):
            n = int(np.prod(shape))
            part = packed[off:off + n]
            v = M.bf16_bits_to_f64(part) if packed.dtype == np.uint16 else part.astype(np.float64)
            setattr(self, name, v.reshape(shape))
            off += n
        self.d, self.m = d, m


def f_phi(head, h, e, eps):
    """Eq. 2 on rows: h, e (R, d) -> predicted hidden states h_hat (R, d)."""
    z = np.concatenate([h, e], axis=-1)
    u = z @ head.w0.T
    n = M.rms_norm(u, head.g, eps)
    return u + (M.silu(n @ head.w1.T) * (n @ head.w3.T)) @ head.w2.T


def argmax_lowest(x):
    """Index of the row maximum, the lowest index among ties (rows of a 2-D array)."""
    return np.argmax(x, axis=-1)  # numpy returns the first maximal index


def draft(model, head, h, tokens):
    """Draft tokens for rows (h (R, d) pre-norm states, tokens (R,) vocabulary ids of
    the same positions): (image-code indices (R,), logits (R, V_img))."""
    e = model.tok_emb[np.asarray(tokens, dtype=np.int64)]
    hh = f_phi(head, np.asarray(h, dtype=np.float64), e, model.cfg.rms_eps)
    logits = M.rms_norm(hh, model.final_norm, model.cfg.rms_eps) @ model.lm_img.T
    return argmax_lowest(logits), logits
