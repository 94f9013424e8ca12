"""Helpers for the oracle pins: tiny configurations and packed-weight editing."""
import numpy as np

import synth
from oracle import model as M


def config_of(shape):
    return M.Config(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim,
                    shape.d_ff, shape.vocab, shape.img_lo, shape.img_hi, shape.dtype)


# text + image vocabulary, grouped-query attention, fp32 (no rounding points)
TINY_GQA = synth.ModelShape(2, 32, 4, 2, 8, 48, 40, 32, "f32")
TINY_BF16 = synth.ModelShape(2, 32, 4, 2, 8, 48, 40, 32, "bf16")


def packed(shape, seed=0, std=0.2, gain_std=0.1):
    return synth.weights(shape, seed=seed, std=std, gain_std=gain_std)


def tensors(shape, buf):
    """Dict (name, layer) -> view into the packed buffer."""
    out = {}
    off = 0
    layer = -1
    names = synth.tensor_shapes(shape)
    for name, shp in names:
        n = int(np.prod(shp))
        if name == "attn_norm":
            layer += 1
        key = (name, layer if name not in ("tok_emb", "final_norm", "lm_head") else -1)
        out[key] = buf[off:off + n].reshape(shp)
        off += n
    return out


def model(shape, buf):
    return M.Model(config_of(shape), buf)
