"""Verify rounds, commit, strict truncation, AR decoding and the image driver
(oracle, test infrastructure).

Paper: Sec. 3.3 "Verification as Auto Correction".  A drafted block goes
through the backbone in one pass; every drafted position is corrected
independently by rule (A), (B) or (C) (see ``oracle.select``); the procedure
repeats for a fixed number of rounds, rejected positions take the previous
round's backbone distribution as their reference; after the last round one
more forward pass commits the corrected block and updates the KV cache.
Strict verification that truncates at the first mismatch is the standard
speculative scheme the paper contrasts with; it is kept here as a mode because
it is exact (it reproduces greedy AR decoding), which pins the forward pass.

Scoring alignment (reading): block position k is scored by the backbone's
prediction for position f+k, i.e. the logits output at block position k-1;
position 0 is scored by the carry -- the last logits of the previous commit
(or of the prefill).  A block may start with one fixed position (n_fixed = 1):
a token already chosen but not yet in the cache, which is not verified.

Classifier-free guidance (the paper's backbones decode with it, Table
"app_config": weights 5.0, 4.0, 3.0; the mix is Ho & Salimans' for logits): a
guided session pairs B = 2*Bi sequences -- image b's conditional stream is
sequence b, its unconditional stream sequence Bi + b (a null prompt of the
same length).  Both streams get the image's block, and every decision scores
with the guided logits l_u + w (l_c - l_u), the carry included.

Pins: tests/test_oracle_decode.py -- truncation decoding and Jacobi-style
greedy rounds (r >= K) both reproduce greedy AR decoding (Eq. 1 with argmax)
token for token; the verify pass leaves the frontier unchanged and the commit
pass advances it by K; the pass count of a decoded image equals the plan's.
tests/test_oracle_cfg.py -- guidance against unguided sessions of the same
streams (w = 1 and w = 0 give the conditional and unconditional decodes, equal
prompts make w irrelevant, the guided logits are affine in w with the two
streams' own logits, images pair with their own twins).
"""

import numpy as np

from . import draft as Dr
from . import model as M
from . import schedule as S
from . import select as R


class Session:
    def __init__(self, model, B, P, max_ctx):
        self.model = model
        self.cfg = model.cfg
        self.B, self.P = B, P
        self.cache = M.Cache(model.cfg, B, max_ctx)
        self.f = np.zeros(B, dtype=np.int64)
        self.carry = None  # (B, V_img) float64
        self.h_carry = None  # (B, d) pre-norm state of the last cached position (it scored the carry)
        self.passes = 0
        self.guide = None  # CFG weight w, or None (unguided)
        self.n_img = B     # images decoded: B, or B / 2 under guidance


def mix(l_c, l_u, w):
    """Guided logits of a conditional / unconditional pair (CFG)."""
    return l_u + w * (l_c - l_u)


def set_guidance(sess, w):
    """Pair the session's sequences for classifier-free guidance with weight w."""
    assert sess.B % 2 == 0
    sess.guide = float(w)
    sess.n_img = sess.B // 2


def carry_of(sess, b):
    """Logits that score image b's position f (guided under CFG)."""
    if sess.guide is None:
        return sess.carry[b]
    return mix(sess.carry[b], sess.carry[b + sess.n_img], sess.guide)


def guided(sess, logits):
    """Per-image logits (n_img, K, V_img) of a pass over every stream."""
    if sess.guide is None:
        return logits
    return mix(logits[:sess.n_img], logits[sess.n_img:], sess.guide)


def streams(sess, block):
    """Block tokens of every sequence: under guidance both streams of an image get its block."""
    return block if sess.guide is None else np.concatenate([block, block], axis=0)


def prefill(model, prefix, max_ctx, guide=None):
    """Forward the text prefix (B, P) from position 0; the carry is the last
    position's logits (they score the first image token).  With a guidance
    weight, prefix stacks the Bi conditional prompts over their Bi
    unconditional twins."""
    prefix = np.asarray(prefix)
    B, P = prefix.shape
    s = Session(model, B, P, max_ctx)
    logits, h_pre = M.forward(model, s.cache, prefix, s.f)
    s.f[:] = P
    s.carry = logits[:, P - 1, :].copy()
    s.h_carry = h_pre[:, P - 1, :].copy()
    s.passes = 1
    if guide is not None:
        set_guidance(s, guide)
    return s


def scoring_logits(sess, logits, b, k):
    """Logits that score block position k of image b (logits: the pass's, every stream)."""
    if k == 0:
        return carry_of(sess, b)
    if sess.guide is None:
        return logits[b, k - 1]
    return mix(logits[b, k - 1], logits[b + sess.n_img, k - 1], sess.guide)


def block_tokens(sess, block, eol=None):
    """Vocabulary ids of a block of image codes at the frontier, and the block
    offsets holding an end-of-line token (eol = (id, period, base): sequence
    position p is one when (p - base) % period == period - 1; the codes there
    are placeholders)."""
    toks = np.asarray(block, dtype=np.int64) + sess.cfg.img_lo
    fixed = np.zeros(toks.shape, dtype=bool)
    if eol is not None:
        eid, period, base = eol
        pos = sess.f[:toks.shape[0], None] + np.arange(toks.shape[1])[None, :]
        fixed = (pos - base) % period == period - 1
        toks = np.where(fixed, eid, toks)
    return toks, fixed


def verify_round(sess, block, n_fixed, rule, rnd, seed=0, temperature=1.0, top_k=0, ref=None, eol=None):
    """One verify-and-correct round.

    block -- (B, K) image-code indices (0-based within the image range), one
             row per image (B = n_img)
    ref   -- list over b of lists over k of reference logits (None = point mass);
             updated in place for rule (C) rejections
    Returns (new_block, accept (B,K) bool, count (B,), logits (B,K,V_img)),
    the logits guided under CFG.
    The frontier does not move; the block's KV slots are overwritten.
    """
    block = np.asarray(block, dtype=np.int64)
    B, K = block.shape
    assert B == sess.n_img
    toks, fixed = block_tokens(sess, block, eol)
    logits, _ = M.forward(sess.model, sess.cache, streams(sess, toks), sess.f)
    sess.passes += 1
    new = block.copy()
    acc = np.zeros((B, K), dtype=bool)
    for b in range(B):
        for k in range(n_fixed, K):
            if fixed[b, k]:  # end-of-line positions are not verified
                continue
            pos = int(sess.f[b]) + k
            u0 = R.uniform(seed, b, pos, rnd, 0)
            u1 = R.uniform(seed, b, pos, rnd, 1)
            L = scoring_logits(sess, logits, b, k)
            rk = None if ref is None else ref[b][k]
            t, a, replaced = R.select_position(rule, L, int(block[b, k]), rk, u0, u1, temperature, top_k)
            new[b, k] = t
            acc[b, k] = a
            if replaced and ref is not None:
                ref[b][k] = np.array(L, dtype=np.float64)
    return new, acc, acc[:, n_fixed:].sum(axis=1), guided(sess, logits)


def commit(sess, block, eol=None):
    """Commit pass: forward the final block, keep its KV, advance the frontier
    by K and take the last position's logits as the new carry (per stream).
    Returns the per-image (guided) logits and the conditional stream's h_pre."""
    block = np.asarray(block, dtype=np.int64)
    K = block.shape[1]
    assert block.shape[0] == sess.n_img
    toks, _ = block_tokens(sess, block, eol)
    logits, h_pre = M.forward(sess.model, sess.cache, streams(sess, toks), sess.f)
    sess.passes += 1
    sess.f += K
    sess.carry = logits[:, K - 1, :].copy()
    sess.h_carry = h_pre[:, K - 1, :].copy()
    return guided(sess, logits), h_pre[:sess.n_img]


def truncate_step(sess, block, n_fixed):
    """Strict greedy verification (single sequence or uniform frontier per row):
    accept the leading run of drafts equal to the argmax, then take the argmax
    at the first mismatch (or after the block) as the pending token.
    Returns (n_accepted (B,), pending (B,)).  The frontier advances by
    n_fixed + n_accepted; the KV of those positions is already final."""
    cfg = sess.cfg
    assert sess.guide is None, "strict truncation is not defined here for guided sessions"
    block = np.asarray(block, dtype=np.int64)
    B, K = block.shape
    logits, _ = M.forward(sess.model, sess.cache, block + cfg.img_lo, sess.f)
    sess.passes += 1
    n_acc = np.zeros(B, dtype=np.int64)
    pending = np.zeros(B, dtype=np.int64)
    for b in range(B):
        n = 0
        k = n_fixed
        while k < K:
            a = R.argmax_lowest(scoring_logits(sess, logits, b, k))
            if a != block[b, k]:
                break
            n += 1
            k += 1
        # k is the first unaccepted block position (or K)
        pending[b] = R.argmax_lowest(logits[b, k - 1]) if k >= 1 else R.argmax_lowest(sess.carry[b])
        n_acc[b] = n
        sess.f[b] += n_fixed + n
    return n_acc, pending


def ar_decode(model, prefix, n_tokens):
    """Greedy autoregressive decoding (Eq. 1 with argmax): one forward pass per
    image token.  Returns (B, n_tokens) image-code indices."""
    prefix = np.asarray(prefix)
    B, P = prefix.shape
    s = prefill(model, prefix, P + n_tokens)
    out = np.zeros((B, n_tokens), dtype=np.int64)
    for j in range(n_tokens):
        for b in range(B):
            out[b, j] = R.argmax_lowest(s.carry[b])
        if j + 1 < n_tokens:
            commit(s, out[:, j:j + 1])
    return out


def ar_decode_eol(model, prefix, H, W, eol_id):
    """Greedy AR decoding of an image whose rows each end with the end-of-line
    token eol_id (forced, one pass like any other token).  Returns (image
    codes (B, H, W), passes): the passes are H (W + 1), one per generated token,
    the prefill producing the first."""
    prefix = np.asarray(prefix)
    B, P = prefix.shape
    s = prefill(model, prefix, P + H * (W + 1))
    img = np.zeros((B, H, W), dtype=np.int64)
    n = H * (W + 1)
    for p in range(n):
        y, x = divmod(p, W + 1)
        if x < W:
            img[:, y, x] = [R.argmax_lowest(s.carry[b]) for b in range(B)]
            tok = img[:, y, x:x + 1] + model.cfg.img_lo
        else:
            tok = np.full((B, 1), eol_id, dtype=np.int64)
        if p + 1 < n:
            logits, _ = M.forward(model, s.cache, tok, s.f)
            s.passes += 1
            s.f += 1
            s.carry = logits[:, 0, :].copy()
    return img, s.passes


def decode_truncate(model, prefix, drafts, K, plant=None, stats=None):
    """Exact greedy speculative decoding of len(drafts[b]) image tokens per
    sequence with blocks of K positions ([pending, K-1 drafts]); sequences are
    decoded one at a time.  Returns (tokens (B, N), passes).

    plant -- optional (keep (B, N) bool, repl (B, N) codes): before each pass the
             drafts it tests are planted left to right (planted_draft) against
             the committed tokens and the drafts before them, stopping after the
             first replaced one; `drafts` is then overwritten with the planted
             table.  stats (a dict) receives accepted / proposed (drafts tested:
             the accepted run and the first mismatch of each pass)."""
    prefix = np.asarray(prefix)
    drafts = np.array(drafts, dtype=np.int64)
    B, N = drafts.shape
    P = prefix.shape[1]
    out = np.zeros((B, N), dtype=np.int64)
    passes = 0
    acc_tot = prop_tot = 0
    for b in range(B):
        s = prefill(model, prefix[b:b + 1], P + N + K)
        pending = R.argmax_lowest(s.carry[0])
        done = 0  # tokens final (in cache)
        while True:
            out[b, done] = pending
            if done + 1 == N:
                break
            k_blk = min(K, N - done)
            if plant is not None:
                before = list(out[b, :done + 1])
                for x in range(done + 1, done + k_blk):
                    t, _ = planted_draft(model, prefix[b], before, plant[0][b][x], plant[1][b][x])
                    drafts[b, x] = t
                    before.append(t)
                    if not plant[0][b][x]:
                        break
            blk = np.concatenate([[pending], drafts[b, done + 1:done + k_blk]])[None, :]
            n_acc, pend = truncate_step(s, blk, 1)
            n = int(n_acc[0])
            acc_tot += n
            prop_tot += n + (1 if n < k_blk - 1 else 0)
            out[b, done + 1:done + 1 + n] = blk[0, 1:1 + n]
            done += 1 + n
            pending = int(pend[0])
            if done >= N:
                break
        passes += s.passes
    if stats is not None:
        stats.update(accepted=acc_tot, proposed=prop_tot, planted=drafts)
    return out, passes


def planted_draft(model, prefix_row, before, keep, repl):
    """One planted draft (a measurement input, not the method): a = the greedy
    argmax of the backbone's logits for the next position given the prompt and
    the image tokens `before` (everything chosen or drafted ahead of it), from a
    plain no-cache forward pass; the draft is a if keep, else the code
    repl + (repl >= a) (repl uniform over [0, V_img - 1) gives a uniform other
    code).  Returns (draft, a) as image-code indices."""
    toks = np.concatenate([np.asarray(prefix_row, dtype=np.int64),
                           np.asarray(before, dtype=np.int64) + model.cfg.img_lo])[None, :]
    logits, _ = M.forward_nocache(model, toks)
    a = R.argmax_lowest(logits[0, -1])
    return (a if keep else int(repl) + (int(repl) >= a)), a


def decode_image(model, prefix, H, W, drafts, rule=R.RULE_GREEDY, seed=0, temperature=1.0, top_k=0,
                 k_h=5, h_rounds=1, k_v=1, b=2, i=0, q_table=None, trace=None, guide=None, heads=None,
                 eol_id=None, plant=None):
    """Decode one image per sequence under the SSD schedule, with planted drafts
    or drafted by spatial heads (Sec. 3.3).

    prefix  -- (B, P) prompts; with a guidance weight `guide`, (2B, P): the B
               conditional prompts over their unconditional twins
    drafts  -- (B, H, W) image-code indices used as the draft of every position
               (ignored when heads are given)
    heads   -- optional (horizontal, vertical): lists of oracle.draft.Head, the
               horizontal head for offset +j at index j-1 (k_h of them) and the
               vertical head for +j rows at index j-1 (k_v).  Head inputs are
               [h; e] of a chosen token: h the pre-norm state that scored it (the
               state of the raster position before it, conditional stream under
               guidance), e its embedding; the drafts are the argmax of the
               backbone's output layer on the predicted states, and under rule C
               their softmax is the draft distribution q of the first round.
    eol_id  -- optional end-of-line token id: every image row is followed by it
               in the sequence (fixed, never verified); with heads, the row end's
               state scores the next row's first token
    q_table -- optional (B, H, W, V_img) draft logits (rule C reference for the
               first round of each position); None = point masses at the drafts
    trace   -- optional list collecting (op, accept, count, logits) per verify
    plant   -- optional (keep (B, H, W) bool, repl (B, H, W) codes): drafts are
               planted at each draft op, left to right (planted_draft), against
               the tokens chosen so far; stats["planted"] then holds the table
               (B, H, W) of planted drafts
    Returns (tokens (B, H, W), stats dict).
    """
    cfg = model.cfg
    prefix = np.asarray(prefix)
    B, P = prefix.shape
    if guide is not None:
        B //= 2
    N = H * W
    eol = eol_id is not None
    RW = W + 1 if eol else W
    NS = H * RW  # sequence positions of the image
    ev = (eol_id, RW, P) if eol else None
    ops = S.plan(H, W, k_h=k_h, h_rounds=h_rounds, k_v=k_v, b=b, i=i, eol=eol)
    sess = None
    if heads is None:
        work = np.zeros((B, H, RW), dtype=np.int64)
        work[:, :, :W] = np.asarray(drafts, dtype=np.int64).reshape(B, H, W)
        work = work.reshape(B, NS)
        if eol and q_table is not None:
            qs = np.zeros((B, H, RW, q_table.shape[-1]))
            qs[:, :, :W] = np.asarray(q_table).reshape(B, H, W, -1)
            q_table = qs.reshape(B, NS, -1)
    else:
        work = np.zeros((B, NS), dtype=np.int64)
        hs = np.zeros((B, N, cfg.d_model))  # hs[:, p]: the state that scored image token p
        q_table = np.zeros((B, NS, cfg.img_hi - cfg.img_lo)) if rule == R.RULE_ACCEPT_REJECT else None

    def seq_of(p):  # sequence position (after the prompt) of image index p
        return (np.asarray(p) // W) * RW + np.asarray(p) % W
    refs = [dict() for _ in range(B)]  # image index -> reference logits
    stats = {"accepted": 0, "proposed": 0, "verify_rounds": 0, "accepted_first": 0, "proposed_first": 0}
    if plant is not None:
        assert heads is None and not eol and guide is None
        keep = np.asarray(plant[0]).reshape(B, N).astype(bool)
        repl = np.asarray(plant[1]).reshape(B, N)
        stats["planted"] = repl.copy()
    fresh = set()  # image indexes drafted and not yet verified
    for op in ops:
        if op[0] == "prefill":
            sess = prefill(model, prefix, P + NS, guide)
            if heads is not None:
                hs[:, 0] = sess.h_carry[:B]
        elif op[0] in ("draft_h", "draft_v"):
            if op[0] == "draft_h":
                new_idx = [op[1] + j for j in range(1, op[2] + 1)]
            else:
                new_idx = [x for r in range(op[1] + 1, op[1] + op[2] + 1) for x in range(r * W, (r + 1) * W)]
            fresh.update(new_idx)
            if plant is not None:
                for x in new_idx:  # left to right: each draft sees the ones before it
                    for bb in range(B):
                        t, _ = planted_draft(model, prefix[bb], work[bb, :x], keep[bb, x], repl[bb, x])
                        work[bb, x] = t
                        stats["planted"][bb, x] = t
                continue
            if heads is None:
                continue
            if op[0] == "draft_h":
                _, src, n = op
                srcs = np.array([src])
                dst = [src + j for j in range(1, n + 1)]
                lst = heads[0]
            else:
                _, y0, m = op
                srcs = y0 * W + np.arange(W)
                dst = [srcs + j * W for j in range(1, m + 1)]
                lst = heads[1]
            for j, d_idx in enumerate(dst):
                idx, lg = Dr.draft(model, lst[j], hs[:, srcs].reshape(-1, cfg.d_model),
                                   (work[:, seq_of(srcs)] + cfg.img_lo).reshape(-1))
                dq = seq_of(d_idx)
                work[:, dq] = idx.reshape(B, -1) if np.ndim(d_idx) else idx
                if q_table is not None:
                    q_table[:, dq] = lg.reshape(B, -1, lg.shape[-1]) if np.ndim(d_idx) else lg
                if trace is not None:
                    trace.append((op, j + 1, srcs.copy(), np.atleast_1d(d_idx).copy(), work[:, dq].copy()))
        elif op[0] == "first":
            for bb in range(B):
                u1 = R.uniform(seed, bb, P, 0, 2)
                work[bb, 0] = R.sample_first(rule, carry_of(sess, bb), u1, temperature, top_k)
        elif op[0] == "verify":
            _, start, K, nf, rnd = op
            assert int(sess.f[0]) == P + start
            ref = None
            if rule == R.RULE_ACCEPT_REJECT:
                ref = []
                for bb in range(B):
                    row = []
                    for k in range(K):
                        idx = start + k
                        if idx not in refs[bb]:
                            refs[bb][idx] = None if q_table is None else \
                                np.asarray(q_table[bb].reshape(NS, -1)[idx], np.float64)
                        row.append(refs[bb][idx])
                    ref.append(row)
            blk = work[:, start:start + K]
            new, acc, cnt, logits = verify_round(sess, blk, nf, rule, rnd, seed, temperature, top_k, ref, ev)
            if ref is not None:
                for bb in range(B):
                    for k in range(K):
                        refs[bb][start + k] = ref[bb][k]
            work[:, start:start + K] = new
            stats["accepted"] += int(cnt.sum())
            n_eol = sum(1 for k in range(K) if eol and (start + k) % RW == W)
            stats["proposed"] += B * (K - nf - n_eol)
            stats["verify_rounds"] += 1
            # first round of freshly drafted positions (image indexes; eol off here)
            first = [k for k in range(nf, K) if (start + k) in fresh]
            if first and not eol:
                stats["accepted_first"] += int(acc[:, first].sum())
                stats["proposed_first"] += B * len(first)
                fresh.difference_update(start + k for k in first)
            if trace is not None:
                trace.append((op, acc, cnt, logits, new))
        elif op[0] == "commit":
            _, start, K = op
            assert int(sess.f[0]) == P + start
            _, hp = commit(sess, work[:, start:start + K], ev)
            if heads is not None:
                # the state of block offset k scores sequence position start + k + 1:
                # kept when that is an image position (a row end's state scores the next row)
                for k in range(K):
                    q1 = start + k + 1
                    if q1 < NS and q1 % RW != W:
                        hs[:, (q1 // RW) * W + q1 % RW] = hp[:, k]
            for bb in range(B):
                for k in range(K):
                    refs[bb].pop(start + k, None)
    stats["passes"] = sess.passes
    if plant is not None:
        stats["planted"] = stats["planted"].reshape(B, H, W)
    assert sess.passes == S.n_passes(ops)
    return work.reshape(B, H, RW)[:, :, :W], stats
