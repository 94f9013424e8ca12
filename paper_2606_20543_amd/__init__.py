"""Python binding of libssd.so, the MI355X verify-step library of Spatially
Speculative Decoding.  Argument marshalling only: every step of the verify
path runs in the library's HIP kernels.  The C ABI is declared (and
documented) in include/ssd.h; the functions here carry the same names.

Array arguments may be numpy arrays (host memory), torch tensors (device or
host memory) or raw integer addresses.  There is no CPU fallback: if the
library is not built, importing works but every call raises.
"""
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libssd.so")

SSD_OK, SSD_E_INVAL, SSD_E_STATE, SSD_E_CAPACITY, SSD_E_OOM, SSD_E_DEVICE = 0, -1, -2, -3, -4, -5
SSD_F32, SSD_BF16 = 0, 1
SSD_GREEDY, SSD_SAMPLE, SSD_ACCEPT_REJECT = 0, 1, 2

EXPORTED = [
    "ssd_init_model", "ssd_weights_numel", "ssd_free_model", "ssd_prefill", "ssd_free_session",
    "ssd_verify_step", "ssd_get_carry", "ssd_session_set_cfg", "ssd_decode_image", "ssd_profile", "ssd_profile_read", "ssd_last_error",
    "ssd_draft_head_numel", "ssd_draft_head_init", "ssd_draft_head_run", "ssd_free_draft_head",
    "ssd_decode_image_heads", "ssd_plant_image", "ssd_draft_head_run_noalloc",
]


class SSDError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"ssd status {status}: {message}")
        self.status = status


class ssd_model_config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("d_ff", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("img_lo", ctypes.c_int32), ("img_hi", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("rms_eps", ctypes.c_float), ("rope_theta", ctypes.c_float)]


class ssd_verify_params(ctypes.Structure):
    _fields_ = [("rule", ctypes.c_int32), ("top_k", ctypes.c_int32), ("temperature", ctypes.c_double),
                ("seed", ctypes.c_uint64), ("round", ctypes.c_uint32), ("n_fixed", ctypes.c_int32),
                ("commit", ctypes.c_int32), ("truncate", ctypes.c_int32)]


class ssd_schedule(ctypes.Structure):
    _fields_ = [("grid_h", ctypes.c_int32), ("grid_w", ctypes.c_int32), ("k_h", ctypes.c_int32),
                ("h_rounds", ctypes.c_int32), ("k_v", ctypes.c_int32), ("b_rounds", ctypes.c_int32),
                ("i_rounds", ctypes.c_int32), ("rule", ctypes.c_int32), ("top_k", ctypes.c_int32),
                ("temperature", ctypes.c_double), ("seed", ctypes.c_uint64), ("cfg", ctypes.c_int32),
                ("cfg_weight", ctypes.c_float), ("eol", ctypes.c_int32), ("eol_id", ctypes.c_int32),
                ("separate_commit", ctypes.c_int32), ("truncate", ctypes.c_int32), ("trunc_block", ctypes.c_int32)]


class ssd_stats(ctypes.Structure):
    _fields_ = [("passes", ctypes.c_int64), ("verify_rounds", ctypes.c_int64), ("accepted", ctypes.c_int64),
                ("proposed", ctypes.c_int64), ("accepted_round", ctypes.c_int64 * 8),
                ("proposed_round", ctypes.c_int64 * 8), ("wall_ns", ctypes.c_int64)]


_lib = None


def lib():
    """Load libssd.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: run __graft_entry__.build() (no CPU fallback exists)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        L.ssd_init_model.argtypes = [ctypes.POINTER(ssd_model_config), vp, vp, ctypes.POINTER(vp)]
        L.ssd_weights_numel.argtypes = [ctypes.POINTER(ssd_model_config)]
        L.ssd_weights_numel.restype = i64
        L.ssd_free_model.argtypes = [vp]
        L.ssd_free_model.restype = None
        L.ssd_prefill.argtypes = [vp, i32, i32, vp, i32, i32, vp, ctypes.POINTER(vp)]
        L.ssd_free_session.argtypes = [vp]
        L.ssd_free_session.restype = None
        L.ssd_verify_step.argtypes = [vp, i32, vp, vp, ctypes.POINTER(ssd_verify_params), vp, vp, vp, vp, vp]
        L.ssd_get_carry.argtypes = [vp, vp]
        L.ssd_session_set_cfg.argtypes = [vp, ctypes.c_float]
        L.ssd_decode_image.argtypes = [vp, ctypes.POINTER(ssd_schedule), i32, i32, vp, vp, vp, vp,
                                       ctypes.POINTER(ssd_stats), vp]
        L.ssd_profile.argtypes = [vp, i32]
        L.ssd_profile_read.argtypes = [vp, vp, vp, vp, vp, i32]
        L.ssd_draft_head_numel.argtypes = [vp, i32]
        L.ssd_draft_head_numel.restype = i64
        L.ssd_draft_head_init.argtypes = [vp, i32, vp, i32, ctypes.POINTER(vp)]
        L.ssd_draft_head_run.argtypes = [vp, i32, vp, vp, vp, vp]
        L.ssd_draft_head_run_noalloc.argtypes = [vp, i32, vp, vp, vp, vp]
        L.ssd_free_draft_head.argtypes = [vp]
        L.ssd_plant_image.argtypes = [vp, ctypes.POINTER(ssd_schedule), i32, i32, vp, vp, vp, vp, vp,
                                      ctypes.POINTER(ssd_stats), vp]
        L.ssd_decode_image_heads.argtypes = [vp, ctypes.POINTER(ssd_schedule), i32, i32, vp, ctypes.POINTER(vp), i32,
                                             ctypes.POINTER(vp), i32, vp, ctypes.POINTER(ssd_stats), vp]
        L.ssd_free_draft_head.restype = None
        L.ssd_last_error.argtypes = []
        L.ssd_last_error.restype = ctypes.c_char_p
        for name in ("ssd_init_model", "ssd_prefill", "ssd_verify_step", "ssd_get_carry", "ssd_session_set_cfg",
                     "ssd_decode_image", "ssd_profile", "ssd_profile_read", "ssd_draft_head_init", "ssd_draft_head_run",
                     "ssd_decode_image_heads", "ssd_plant_image", "ssd_draft_head_run_noalloc"):
            getattr(L, name).restype = i32
        _lib = L
    return _lib


def _ptr(x):
    """Address of an array-like: None, int, numpy array or torch tensor."""
    if x is None:
        return None
    if isinstance(x, int):
        return ctypes.c_void_p(x)
    if hasattr(x, "data_ptr"):
        assert x.is_contiguous(), "tensors passed to libssd must be contiguous"
        return ctypes.c_void_p(x.data_ptr())
    if hasattr(x, "ctypes"):
        assert x.flags["C_CONTIGUOUS"], "arrays passed to libssd must be C-contiguous"
        return ctypes.c_void_p(x.ctypes.data)
    raise TypeError(f"cannot take the address of {type(x)}")


def _check(status):
    if status != SSD_OK:
        raise SSDError(status, lib().ssd_last_error().decode())


def ssd_last_error():
    return lib().ssd_last_error().decode()


def ssd_weights_numel(cfg):
    return int(lib().ssd_weights_numel(ctypes.byref(cfg)))


def ssd_init_model(cfg, weights, stream=None):
    out = ctypes.c_void_p()
    _check(lib().ssd_init_model(ctypes.byref(cfg), _ptr(weights), _ptr(stream), ctypes.byref(out)))
    return out.value


def ssd_free_model(model):
    lib().ssd_free_model(ctypes.c_void_p(model))


def ssd_prefill(model, B, P, prefix, max_ctx, max_block, stream=None):
    out = ctypes.c_void_p()
    _check(lib().ssd_prefill(ctypes.c_void_p(model), B, P, _ptr(prefix), max_ctx, max_block, _ptr(stream),
                             ctypes.byref(out)))
    return out.value


def ssd_free_session(sess):
    lib().ssd_free_session(ctypes.c_void_p(sess))


def ssd_verify_step(sess, K, tokens, params, ref_logits=None, accept_mask=None, accept_count=None, frontier=None,
                    logits_out=None, h_pre_out=None):
    _check(lib().ssd_verify_step(ctypes.c_void_p(sess), K, _ptr(tokens), _ptr(ref_logits), ctypes.byref(params),
                                 _ptr(accept_mask), _ptr(accept_count), _ptr(frontier), _ptr(logits_out),
                                 _ptr(h_pre_out)))


def ssd_get_carry(sess, carry_out):
    _check(lib().ssd_get_carry(ctypes.c_void_p(sess), _ptr(carry_out)))


def ssd_session_set_cfg(sess, weight):
    _check(lib().ssd_session_set_cfg(ctypes.c_void_p(sess), float(weight)))


def ssd_decode_image(model, sched, B, P, prefix, drafts, out_tokens, draft_logits=None, stream=None):
    st = ssd_stats()
    _check(lib().ssd_decode_image(ctypes.c_void_p(model), ctypes.byref(sched), B, P, _ptr(prefix), _ptr(drafts),
                                  _ptr(draft_logits), _ptr(out_tokens), ctypes.byref(st), _ptr(stream)))
    return st


def ssd_plant_image(model, sched, B, P, prefix, keep, repl, drafts_out, out_tokens, stream=None):
    """keep [B][H][W] uint8, repl [B][H][W] int32 image-code indices; fills drafts_out and out_tokens."""
    st = ssd_stats()
    _check(lib().ssd_plant_image(ctypes.c_void_p(model), ctypes.byref(sched), B, P, _ptr(prefix), _ptr(keep),
                                 _ptr(repl), _ptr(drafts_out), _ptr(out_tokens), ctypes.byref(st), _ptr(stream)))
    return st


def ssd_draft_head_numel(model, m):
    return int(lib().ssd_draft_head_numel(ctypes.c_void_p(model), m))


def ssd_draft_head_init(model, m, weights, max_rows):
    out = ctypes.c_void_p()
    _check(lib().ssd_draft_head_init(ctypes.c_void_p(model), m, _ptr(weights), max_rows, ctypes.byref(out)))
    return out.value


def ssd_draft_head_run(head, R, h, tokens, drafts, logits_out=None):
    _check(lib().ssd_draft_head_run(ctypes.c_void_p(head), R, _ptr(h), _ptr(tokens), _ptr(drafts),
                                    _ptr(logits_out)))


def ssd_draft_head_run_noalloc(head, R, h, tokens, drafts, logits_out=None):
    """Device arrays only; the workspace comes from the library's static array."""
    _check(lib().ssd_draft_head_run_noalloc(ctypes.c_void_p(head), R, _ptr(h), _ptr(tokens), _ptr(drafts),
                                            _ptr(logits_out)))


def ssd_free_draft_head(head):
    lib().ssd_free_draft_head(ctypes.c_void_p(head))


def ssd_decode_image_heads(model, sched, B, P, prefix, h_heads, v_heads, out_tokens, stream=None):
    """h_heads / v_heads: sequences of head handles (horizontal offsets +1.., vertical rows +1..)."""
    hh = (ctypes.c_void_p * max(len(h_heads), 1))(*h_heads)
    vh = (ctypes.c_void_p * max(len(v_heads), 1))(*v_heads)
    st = ssd_stats()
    _check(lib().ssd_decode_image_heads(ctypes.c_void_p(model), ctypes.byref(sched), B, P, _ptr(prefix), hh,
                                        len(h_heads), vh, len(v_heads), _ptr(out_tokens), ctypes.byref(st),
                                        _ptr(stream)))
    return st


def ssd_profile(model, enable):
    _check(lib().ssd_profile(ctypes.c_void_p(model), int(enable)))


PROFILE_CLASSES = ("qkv", "o_proj", "gate_up", "down", "lm_head", "attention", "forward", "tiled_gemm")


def ssd_profile_read(model, reset=False):
    """{class: (ms, launches, bytes, flops)} for the eight launch classes."""
    import numpy as np
    k = len(PROFILE_CLASSES)
    ms = np.zeros(k, np.float64)
    n = np.zeros(k, np.int64)
    by = np.zeros(k, np.float64)
    fl = np.zeros(k, np.float64)
    _check(lib().ssd_profile_read(ctypes.c_void_p(model), _ptr(ms), _ptr(n), _ptr(by), _ptr(fl), int(reset)))
    return {c: (float(ms[i]), int(n[i]), float(by[i]), float(fl[i])) for i, c in enumerate(PROFILE_CLASSES)}
