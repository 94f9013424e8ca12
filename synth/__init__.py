"""Seeded synthetic inputs shared by the CPU oracle and the GPU path.

This module only draws random numbers and lays them out in the boundary's
input formats (the packed weight buffer, prompt ids, draft tables).  It holds
none of the decoding method's arithmetic.

The five workloads are decoder-only image-token transformers shaped like the
paper's backbones (Sec. 4 "Models": 24x24, 48x48 and 90x90 token grids;
Appendix "Generalization of the Drafting Heads": codebooks of 16384, 8192 and
32768 codes) with random N(0, 0.02) weights -- the paper's trained weights and
prompt datasets are not available, so seeded synthetic inputs of the same
shapes stand in for them.

Recipe (seeds are fixed per purpose):
  weights        seed 0: every matrix N(0, 0.02) rounded to the model dtype,
                 norm gains 1 (or 1 + 0.1 N(0,1) for gain-sensitive tests)
  prompt         seed 1: uniform ids in the text range [0, img_lo) when the
                 vocabulary has one, else over the whole vocabulary
  planted drafts seed 2: Bernoulli(p) keep / uniform replacement code
  sampling       seed 3: the method's own counter-based uniforms
"""

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gen.c")
_LIB = os.path.join(_HERE, "libsynth.so")
_lib = None

SEED_WEIGHTS, SEED_PROMPT, SEED_DRAFTS, SEED_SAMPLING = 0, 1, 2, 3


def build():
    """Compile the generator (plain C, OpenMP)."""
    tmp = _LIB + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", _SRC, "-o", tmp, "-lm"])
    os.replace(tmp, _LIB)


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        u64, i64, i32, dbl, vp = ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32, ctypes.c_double, ctypes.c_void_p
        L.synth_u64.argtypes = [u64, u64, u64, i64, vp]
        L.synth_normal_f32.argtypes = [u64, u64, dbl, dbl, i64, vp]
        L.synth_normal_bf16.argtypes = [u64, u64, dbl, dbl, i64, vp]
        L.synth_randint.argtypes = [u64, u64, i32, i32, i64, vp]
        L.synth_uniform.argtypes = [u64, u64, i64, vp]
        for f in (L.synth_u64, L.synth_normal_f32, L.synth_normal_bf16, L.synth_randint, L.synth_uniform):
            f.restype = None
        _lib = L
    return _lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def u64(seed, stream, n, i0=0):
    out = np.empty(n, dtype=np.uint64)
    lib().synth_u64(seed, stream, i0, n, _ptr(out))
    return out


def normal(seed, stream, n, mean=0.0, std=1.0):
    out = np.empty(n, dtype=np.float32)
    lib().synth_normal_f32(seed, stream, mean, std, n, _ptr(out))
    return out


def randint(seed, stream, lo, hi, n):
    out = np.empty(n, dtype=np.int32)
    lib().synth_randint(seed, stream, lo, hi, n, _ptr(out))
    return out


def uniform(seed, stream, n):
    out = np.empty(n, dtype=np.float64)
    lib().synth_uniform(seed, stream, n, _ptr(out))
    return out


@dataclass(frozen=True)
class ModelShape:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    v_img: int
    dtype: str  # "f32" | "bf16"

    @property
    def img_lo(self):
        return self.vocab - self.v_img

    @property
    def img_hi(self):
        return self.vocab


def tensor_shapes(m):
    """(name, shape) of the packed weight buffer, in the boundary's documented order."""
    d, D, f = m.d_model, m.head_dim, m.d_ff
    out = [("tok_emb", (m.vocab, d))]
    for _ in range(m.n_layers):
        out += [("attn_norm", (d,)), ("wq", (m.n_heads * D, d)), ("wk", (m.n_kv_heads * D, d)),
                ("wv", (m.n_kv_heads * D, d)), ("wo", (d, m.n_heads * D)), ("mlp_norm", (d,)),
                ("w1", (f, d)), ("w3", (f, d)), ("w2", (d, f))]
    out += [("final_norm", (d,)), ("lm_head", (m.vocab, d))]
    return out


def n_params(m):
    return sum(int(np.prod(s)) for _, s in tensor_shapes(m))


def weights(m, seed=SEED_WEIGHTS, std=0.02, gain_std=0.0):
    """Packed weight buffer: uint16 bf16 bits for bf16 models, float32 otherwise.
    Tensor j of the layout uses generator stream j, so every tensor is
    independent of the others' sizes."""
    total = n_params(m)
    if m.dtype == "bf16":
        buf = np.empty(total, dtype=np.uint16)
        fn = lib().synth_normal_bf16
    elif m.dtype == "f32":
        buf = np.empty(total, dtype=np.float32)
        fn = lib().synth_normal_f32
    else:
        raise ValueError(m.dtype)
    off = 0
    base = buf.ctypes.data
    for j, (name, shape) in enumerate(tensor_shapes(m)):
        n = int(np.prod(shape))
        if name.endswith("norm"):
            mean, sd = 1.0, gain_std
        else:
            mean, sd = 0.0, std
        fn(seed, j, mean, sd, n, ctypes.c_void_p(base + off * buf.itemsize))
        off += n
    return buf


SEED_HEADS = 4


def draft_head_weights(d, m, seed=SEED_HEADS, std=0.02, gain_std=0.0, dtype="bf16"):
    """Packed weights of one spatial draft head: W0 [d][2d], gain [d], W1 [m][d],
    W3 [m][d], W2 [d][m] (tensor j on generator stream j; gains around 1), as
    bf16 bits (uint16) or float32."""
    shapes = [("w0", (d, 2 * d)), ("g", (d,)), ("w1", (m, d)), ("w3", (m, d)), ("w2", (d, m))]
    total = int(sum(np.prod(s) for _, s in shapes))
    if dtype == "bf16":
        buf, fn = np.empty(total, dtype=np.uint16), lib().synth_normal_bf16
    elif dtype == "f32":
        buf, fn = np.empty(total, dtype=np.float32), lib().synth_normal_f32
    else:
        raise ValueError(dtype)
    off = 0
    base = buf.ctypes.data
    for j, (name, shape) in enumerate(shapes):
        n = int(np.prod(shape))
        mean, sd = (1.0, gain_std) if name == "g" else (0.0, std)
        fn(seed, j, mean, sd, n, ctypes.c_void_p(base + off * buf.itemsize))
        off += n
    return buf


def hidden_states(R, d, seed=SEED_HEADS, stream=100, std=1.0):
    """Synthetic pre-norm hidden states [R][d] (float32), N(0, std)."""
    return normal(seed, stream, R * d, std=std).astype(np.float32).reshape(R, d)


def prompt(m, B, P, seed=SEED_PROMPT):
    lo, hi = (0, m.img_lo) if m.img_lo > 0 else (0, m.vocab)
    return randint(seed, 0, lo, hi, B * P).reshape(B, P)


def random_codes(m, shape, seed=SEED_DRAFTS, stream=0):
    n = int(np.prod(shape))
    return randint(seed, stream, 0, m.v_img, n).reshape(shape)


def plant(target, p, v_img, seed=SEED_DRAFTS, stream=1):
    """Planted drafts: keep each target code with probability p, otherwise
    replace it with a uniformly drawn *different* code."""
    target = np.asarray(target, dtype=np.int64)
    n = target.size
    keep = uniform(seed, stream, n) < p
    repl = randint(seed, stream + 1, 0, v_img - 1, n).astype(np.int64)
    flat = target.reshape(-1)
    repl = repl + (repl >= flat)  # skip the target itself
    return np.where(keep, flat, repl).reshape(target.shape)


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    batch: int
    prefix: int
    grid: int
    rule: int  # 0 greedy, 1 sample, 2 accept-reject
    rounds: int
    top_k: int = 0
    temperature: float = 1.0
    accept_p: tuple = (0.6,)
    notes: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def max_ctx(self):
        return self.prefix + self.grid * self.grid


TINY = ModelShape(2, 256, 4, 4, 64, 688, 1024, 1024, "f32")
M1B = ModelShape(24, 2048, 16, 16, 128, 5632, 16384, 16384, "bf16")
M7B = ModelShape(32, 4096, 32, 32, 128, 11008, 65536, 8192, "bf16")
M8B = ModelShape(32, 4096, 32, 8, 128, 14336, 65536, 32768, "bf16")

WORKLOADS = {
    "tiny-f32-8x8": Workload("tiny-f32-8x8", TINY, 1, 16, 8, 0, 2),
    "1b-24x24": Workload("1b-24x24", M1B, 1, 64, 24, 0, 2),
    "1b-32x32-b4-ar": Workload("1b-32x32-b4-ar", M1B, 4, 64, 32, 2, 2, top_k=2000),
    "7b-32x32": Workload("7b-32x32", M7B, 1, 128, 32, 0, 2, accept_p=(0.3, 0.6, 0.9)),
    "8b-64x64-b8": Workload("8b-64x64-b8", M8B, 8, 256, 64, 0, 5),
}
