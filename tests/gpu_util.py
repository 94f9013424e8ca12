"""Helpers for GPU parity tests: build a model on the GPU through the C ABI and
run the oracle beside it on the same seeded inputs.

Parity protocol (decisions under bf16 logits):
  1. logits: GPU vs oracle within the dtype's tolerance (2e-2 bf16, 1e-5 fp32);
  2. decisions: the oracle's rule applied to the GPU's own logits (and the
     same counter-based uniforms) reproduces the GPU's tokens, accept flags
     and counts exactly;
  3. end to end: where the oracle's rule on the oracle's logits disagrees with
     the GPU, the disagreement must be one that the logit tolerance allows (a
     greedy top-2 gap within twice the tolerance); both sides then continue
     from the GPU's tokens (re-sync).
"""
import numpy as np

import paper_2606_20543_amd as ssd
import synth
from oracle import decode as Dc
from oracle import model as M
from oracle import schedule as S
from oracle import select as R

TOL = {"f32": 1e-5, "bf16": 2e-2}


def executed_passes(ops, heads=False, separate=False):
    """Backbone passes the library runs for a plan: a commit followed by a verify
    round of the adjacent block (no head drafting in between, no fixed first
    position) shares that round's pass unless commits are kept separate."""
    n = S.n_passes(ops)
    if separate:
        return n
    fused = 0
    for i, o in enumerate(ops):
        if o[0] != "commit":
            continue
        j = i + 1
        while j < len(ops) and ops[j][0] in ("draft_h", "draft_v") and not heads:
            j += 1
        if j < len(ops) and ops[j][0] == "verify" and ops[j][3] == 0 and ops[j][1] == o[1] + o[2]:
            fused += 1
    return n - fused


def tol_of(shape, os_):
    """Logit tolerance of a session: guided logits l_u + w (l_c - l_u) carry the
    streams' errors times |w| + |1 - w|."""
    w = getattr(os_, "guide", None)
    return TOL[shape.dtype] * (1.0 if w is None else max(1.0, abs(w) + abs(1.0 - w)))


def oracle_carry(os_, B):
    """The oracle session's scores of position f per image (guided under CFG)."""
    return np.stack([Dc.carry_of(os_, b) for b in range(B)])


class DeviceArray:
    """Device memory from the HIP runtime the library itself links (not torch's, which
    ships its own runtime), for calls with device pointers."""

    _hip = None

    @classmethod
    def hip(cls):
        import ctypes
        if cls._hip is None:
            ssd.lib()  # the library's runtime is then already loaded under this name
            h = ctypes.CDLL("libamdhip64.so.7")
            h.hipMalloc.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t]
            h.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
            h.hipFree.argtypes = [ctypes.c_void_p]
            h.hipDeviceSynchronize.argtypes = []
            cls._hip = h
        return cls._hip

    def __init__(self, host):
        import ctypes
        self.shape, self.dtype = host.shape, host.dtype
        self.nbytes = host.nbytes
        p = ctypes.c_void_p()
        assert self.hip().hipMalloc(ctypes.byref(p), self.nbytes) == 0
        self.ptr = p.value
        assert self.hip().hipMemcpy(self.ptr, host.ctypes.data, self.nbytes, 1) == 0  # host to device

    def numpy(self):
        out = np.empty(self.shape, self.dtype)
        assert self.hip().hipDeviceSynchronize() == 0
        assert self.hip().hipMemcpy(out.ctypes.data, self.ptr, self.nbytes, 2) == 0  # device to host
        return out

    def free(self):
        if self.ptr:
            self.hip().hipFree(self.ptr)
            self.ptr = None


def cfg_of(shape):
    c = ssd.ssd_model_config()
    c.n_layers, c.d_model, c.n_heads, c.n_kv_heads = shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads
    c.head_dim, c.d_ff, c.vocab = shape.head_dim, shape.d_ff, shape.vocab
    c.img_lo, c.img_hi = shape.img_lo, shape.img_hi
    c.dtype = ssd.SSD_BF16 if shape.dtype == "bf16" else ssd.SSD_F32
    c.rms_eps, c.rope_theta = 1e-5, 10000.0
    return c


def oracle_cfg(shape):
    return M.Config(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim, shape.d_ff,
                    shape.vocab, shape.img_lo, shape.img_hi, shape.dtype)


class Pair:
    """A model loaded on the GPU and in the oracle from the same packed weights."""

    def __init__(self, shape, seed=0, gain_std=0.0, oracle=True):
        self.shape = shape
        self.w = synth.weights(shape, seed=seed, gain_std=gain_std)
        self.cfg = cfg_of(shape)
        assert ssd.ssd_weights_numel(self.cfg) == self.w.size
        self.model = ssd.ssd_init_model(self.cfg, self.w)
        self.om = M.Model(oracle_cfg(shape), self.w) if oracle else None

    def close(self):
        if self.model:
            ssd.ssd_free_model(self.model)
            self.model = None


def vparams(rule=R.RULE_GREEDY, top_k=0, T=1.0, seed=3, rnd=0, n_fixed=0, commit=0, truncate=0):
    p = ssd.ssd_verify_params()
    p.rule, p.top_k, p.temperature, p.seed = rule, top_k, T, seed
    p.round, p.n_fixed, p.commit, p.truncate = rnd, n_fixed, commit, truncate
    return p


def gpu_verify(sess, shape, block_abs, prm, ref=None, want_h=False):
    """One ssd_verify_step with host buffers; returns dict of outputs."""
    B, K = block_abs.shape
    tok = np.ascontiguousarray(block_abs.astype(np.int32))
    acc = np.zeros((B, K), np.uint8)
    cnt = np.zeros(B, np.int32)
    fr = np.zeros(B, np.int32)
    lg = np.zeros((B, K, shape.v_img), np.float32)
    hp = np.zeros((B, K, shape.d_model), np.float32) if want_h else None
    ssd.ssd_verify_step(sess, K, tok, prm, ref_logits=ref, accept_mask=acc, accept_count=cnt, frontier=fr,
                        logits_out=lg, h_pre_out=hp)
    return {"tokens": tok, "accept": acc.astype(bool), "count": cnt, "frontier": fr, "logits": lg, "h_pre": hp}


def oracle_rule_on(logits_gpu, carry_gpu, block_codes, n_fixed, rule, rnd, seed, f, T=1.0, top_k=0, refs=None):
    """Apply the oracle's rule to given (GPU) logits; returns (codes, accept, count, refs_after)."""
    B, K = block_codes.shape
    new = block_codes.copy()
    acc = np.zeros((B, K), bool)
    refs_after = None if refs is None else [list(r) for r in refs]
    for b in range(B):
        for k in range(n_fixed, K):
            L = carry_gpu[b] if k == 0 else logits_gpu[b, k - 1]
            L = L.astype(np.float64)
            pos = int(f[b]) + k
            u0 = R.uniform(seed, b, pos, rnd, 0)
            u1 = R.uniform(seed, b, pos, rnd, 1)
            rk = None if refs is None else refs[b][k]
            t, a, repl = R.select_position(rule, L, int(block_codes[b, k]), rk, u0, u1, T, top_k)
            new[b, k] = t
            acc[b, k] = a
            if repl and refs_after is not None:
                refs_after[b][k] = L
    return new, acc, acc[:, n_fixed:].sum(axis=1), refs_after


def greedy_gap(L):
    s = np.sort(np.asarray(L, np.float64))
    return s[-1] - s[-2]


def flip_within_tolerance(rule, L_oracle, ref_oracle, t, u0, u1, new_gpu, acc_gpu, delta, T=1.0, top_k=0):
    """Whether a GPU decision that differs from the oracle's is one the logit
    error `delta` (max |GPU - oracle| on the rows involved) can cause.

    A logit error of at most delta changes every warped probability by a
    factor within exp(+-2 delta), so: alpha by a factor within exp(+-4 delta);
    the cumulative residual (or p) mass at any code by at most
    2 (exp(2 delta) - 1) per distribution involved.  The GPU's outcome is
    accepted when the oracle's own numbers put the uniform inside that band.
    """
    if rule == R.RULE_GREEDY:
        return greedy_gap(L_oracle) < 2 * delta
    p = R.warp(L_oracle, T, top_k)
    if rule == R.RULE_SAMPLE:
        w, eps_a, accept_ok = p, 2 * (np.exp(2 * delta) - 1), None
    else:
        q = R.point_mass(p.shape[0], t) if ref_oracle is None else R.warp(ref_oracle, T, top_k)
        alpha = R.accept_prob(p, q, t)
        band = alpha * (np.exp(4 * delta) - 1) + 1e-12
        if acc_gpu:
            return new_gpu == t and u0 < alpha + band
        if u0 < alpha - band:
            return False
        w, eps_a = R.residual(p, q), 4 * (np.exp(2 * delta) - 1)
    c = np.cumsum(w)
    target = u1 * c[-1]
    lo = c[new_gpu - 1] if new_gpu > 0 else 0.0
    hi = c[new_gpu]
    return lo - eps_a <= target <= hi + eps_a


def _interval_overlap(w1, w2):
    """Probability that inverse-CDF sampling of the weights w1 and w2 with one
    shared uniform u picks the same code: the total length of the overlaps of
    code v's intervals [C(v-1), C(v)) / Z under the two distributions."""
    c1 = np.concatenate([[0.0], np.cumsum(w1)])
    c2 = np.concatenate([[0.0], np.cumsum(w2)])
    if c1[-1] <= 0 or c2[-1] <= 0:
        return 1.0
    c1, c2 = c1 / c1[-1], c2 / c2[-1]
    lo = np.maximum(c1[:-1], c2[:-1])
    hi = np.minimum(c1[1:], c2[1:])
    return float(np.clip(hi - lo, 0.0, None).sum())


def flip_probability(rule, L_oracle, L_gpu, ref, t, T=1.0, top_k=0):
    """Probability over the position's uniforms (u0 for the accept test, u1 for
    the sample, independent) that the rule decides differently on the two
    logit rows: the expected flip count of the parity protocol's end-to-end
    step, from the logit errors actually realized."""
    if rule == R.RULE_GREEDY:
        return float(R.argmax_lowest(L_oracle) != R.argmax_lowest(L_gpu))
    po, pg = R.warp(L_oracle, T, top_k), R.warp(L_gpu, T, top_k)
    if rule == R.RULE_SAMPLE:
        return 1.0 - _interval_overlap(po, pg)
    if ref is None:
        qo = qg = R.point_mass(po.shape[0], t)
    else:
        qo = qg = R.warp(ref, T, top_k)
    ao, ag = R.accept_prob(po, qo, t), R.accept_prob(pg, qg, t)
    both_reject = 1.0 - max(ao, ag)
    return abs(ao - ag) + both_reject * (1.0 - _interval_overlap(R.residual(po, qo), R.residual(pg, qg)))


def flips_expected_bound(expected):
    """Upper bound for an observed flip count given its expectation (a sum of
    independent Bernoulli trials): mean + 4 standard deviations + 2."""
    return expected + 4.0 * np.sqrt(max(expected, 0.0)) + 2.0


def check_round(shape, sess, os_, blk, nf, rule, rnd, top_k, ref, stats):
    """One verify round on the GPU and in the oracle from the same state, under
    the parity protocol above; the oracle session os_ advances with it.  Returns
    (the GPU's new block codes, the GPU outputs)."""
    tol = tol_of(shape, os_)
    B, K = blk.shape
    carry = np.zeros((B, shape.v_img), np.float32)
    ssd.ssd_get_carry(sess, carry)
    f_before = os_.f[:B].copy()
    ocarry = oracle_carry(os_, B)
    cerr = float(np.abs(carry - ocarry).max())
    stats["max_logit_err"] = max(stats.get("max_logit_err", 0.0), cerr)
    assert cerr < tol, f"carry error {cerr}"
    out = gpu_verify(sess, shape, blk + shape.img_lo, vparams(rule, top_k=top_k, rnd=rnd, n_fixed=nf),
                     ref=None if ref is None else np.ascontiguousarray(ref, np.float32))
    refs = None
    if ref is not None:
        refs = [[ref[b, k].astype(np.float64) for k in range(K)] for b in range(B)]
    gnew, gacc, gcnt, _ = oracle_rule_on(out["logits"], carry, blk, nf, rule, rnd, 3, f_before, 1.0, top_k, refs)
    onew, oacc, _, ologits = Dc.verify_round(os_, blk, nf, rule, rnd, 3, 1.0, top_k,
                                             None if refs is None else [list(r) for r in refs])
    err = float(np.abs(out["logits"] - ologits).max())
    stats["max_logit_err"] = max(stats["max_logit_err"], err)
    assert err < tol, f"logit error {err}"
    assert np.array_equal(out["tokens"] - shape.img_lo, gnew)
    assert np.array_equal(out["accept"][:, nf:], gacc[:, nf:])
    assert np.array_equal(out["count"], gcnt)
    assert list(out["frontier"]) == list(f_before)
    diff = np.argwhere((onew != gnew) | (oacc != gacc))
    stats["flips"] = stats.get("flips", 0) + len(diff)
    stats["positions"] = stats.get("positions", 0) + B * (K - nf)
    exp = 0.0
    for b in range(B):
        for k in range(nf, K):
            Lo = ocarry[b] if k == 0 else ologits[b, k - 1]
            Lg = carry[b] if k == 0 else out["logits"][b, k - 1]
            exp += flip_probability(rule, Lo, Lg, None if refs is None else refs[b][k], int(blk[b, k]), 1.0, top_k)
    stats["flips_expected"] = stats.get("flips_expected", 0.0) + exp
    for b, k in diff:
        Lo = ocarry[b] if k == 0 else ologits[b, k - 1]
        Lg = carry[b] if k == 0 else out["logits"][b, k - 1]
        delta = float(np.abs(Lg - Lo).max())
        pos = int(f_before[b]) + int(k)
        ok = flip_within_tolerance(rule, Lo, None if refs is None else refs[b][k], int(blk[b, k]),
                                   R.uniform(3, b, pos, rnd, 0), R.uniform(3, b, pos, rnd, 1),
                                   int(gnew[b, k]), bool(gacc[b, k]), delta, 1.0, top_k)
        assert ok, f"decision at (b={b}, k={k}) differs beyond what logit error {delta:.2e} allows"
    return gnew, out


# h_pre (the last layer's pre-norm state, the draft heads' input) elementwise,
# relative to its row's root mean square.  The output layer sees h / rms(h): an
# error of e * rms(h) on every element of a row moves a logit by about
# e * sqrt(d) * 0.02 (a sum of d terms of random sign against N(0, 0.02)
# weights), i.e. by e to 1.3 e at d = 2048..4096.  The bf16 bound is half of the
# 2e-2 logit tolerance (measured: 2.3e-3 on the 24-layer 1B model); fp32 models:
# the fp32 accumulation error.
H_RTOL = {"f32": 1e-5, "bf16": 1e-2}


def check_h_pre(shape, h_gpu, h_oracle, stats):
    rms = np.sqrt(np.mean(np.asarray(h_oracle, np.float64) ** 2, axis=-1, keepdims=True))
    rel = np.abs(np.asarray(h_gpu, np.float64) - h_oracle) / rms
    stats["max_h_rel_err"] = max(stats.get("max_h_rel_err", 0.0), float(rel.max()))
    assert rel.max() < H_RTOL[shape.dtype], f"h_pre error {rel.max():.2e} of the row rms"


def check_commit(shape, sess, os_, blk, stats, want_h=False):
    """Commit pass on both sides: logits within tolerance, same frontier; h_pre
    elementwise within H_RTOL of its row's rms."""
    tol = tol_of(shape, os_)
    out = gpu_verify(sess, shape, blk + shape.img_lo, vparams(commit=1), want_h=want_h)
    ol, oh = Dc.commit(os_, blk)
    err = float(np.abs(out["logits"] - ol).max())
    stats["max_logit_err"] = max(stats.get("max_logit_err", 0.0), err)
    assert err < tol, f"commit logit error {err}"
    if want_h:
        check_h_pre(shape, out["h_pre"], oh, stats)
    assert list(out["frontier"]) == list(os_.f[:blk.shape[0]])
    return out
