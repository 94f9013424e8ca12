"""Per-position correction rules of the verify step (oracle, test infrastructure).

Paper: Sec. 3.3, paragraph "Verification as Auto Correction".  Every drafted
position k has a draft token t_k (the argmax of its draft distribution q_k)
and, after the verification forward pass, a backbone distribution p_k.  One of
three rules picks the final token, independently for every position:

  (A) greedy      -- argmax_v p_k(v)
  (B) sampling    -- a sample from p_k
  (C) accept/reject (the paper's default) -- keep t_k with probability
      alpha = min(p_k(t_k) / q_k(t_k), 1); otherwise draw from the residual
      [p_k - q_k]_+ / sum_v [p_k - q_k]_+.

The same paragraph's next part fixes the multi-round bookkeeping: a rejected
position takes the previous round's backbone distribution as its new reference
q; an accepted one keeps its reference.

Readings (the paper is silent on these):
  * temperature T and top-k truncation ("warp") are applied identically to p
    and q; the top-k set is ordered by (value descending, id ascending);
  * the draft distribution of a planted draft is a point mass at the draft;
  * q(t) = 0 with p(t) > 0 gives alpha = 1; p(t) = q(t) = 0 gives alpha = 0;
  * a zero-mass residual (only possible through rounding) keeps the token;
  * argmax ties go to the lowest id.

Randomness: u = 24-bit uniform from SplitMix64 (Steele, Lea & Flood,
OOPSLA 2014) at the counter c = (b<<44) | (pos<<20) | (round<<4) | stream:
u = (mix(seed + (c + 1) * 0x9E3779B97F4A7C15) >> 40) * 2**-24, where mix is the
SplitMix64 output function.  stream 0 drives the accept test, stream 1 the
(residual) sample.  Pinned by the generator's published output values.

All probabilities are float64.  Pins: tests/test_oracle_select.py (closed forms,
the speculative-sampling identity by exhaustive enumeration of the 2^24
uniform grid, published SplitMix64 values).
"""

import numpy as np

GOLDEN = 0x9E3779B97F4A7C15
MASK64 = (1 << 64) - 1

RULE_GREEDY = 0
RULE_SAMPLE = 1
RULE_ACCEPT_REJECT = 2


def splitmix64_mix(z):
    """SplitMix64 output function (Steele, Lea & Flood 2014), on Python ints."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def splitmix64_stream(seed, n):
    """First n outputs of the SplitMix64 generator seeded with ``seed``."""
    out = []
    s = seed & MASK64
    for _ in range(n):
        s = (s + GOLDEN) & MASK64
        out.append(splitmix64_mix(s))
    return out


def counter(b, pos, rnd, stream):
    b, pos, rnd, stream = int(b), int(pos), int(rnd), int(stream)  # Python ints: no 64-bit overflow
    assert 0 <= b < (1 << 20) and 0 <= pos < (1 << 24)
    assert 0 <= rnd < (1 << 16) and 0 <= stream < 16
    return (b << 44) | (pos << 20) | (rnd << 4) | stream


def uniform(seed, b, pos, rnd, stream):
    """Counter-based 24-bit uniform in [0, 1): output number c+1 of the SplitMix64
    stream seeded with ``seed``."""
    c = counter(b, pos, rnd, stream)
    z = splitmix64_mix((seed + (c + 1) * GOLDEN) & MASK64)
    return (z >> 40) * (1.0 / (1 << 24))


def topk_mask(z, top_k):
    """Boolean mask of the top_k entries of z, ordered by (value desc, id asc).
    top_k <= 0 or >= len(z) keeps everything."""
    V = z.shape[0]
    if top_k <= 0 or top_k >= V:
        return np.ones(V, dtype=bool)
    order = np.lexsort((np.arange(V), -z))  # last key is primary
    mask = np.zeros(V, dtype=bool)
    mask[order[:top_k]] = True
    return mask


def warp(logits, temperature=1.0, top_k=0):
    """Normalised distribution softmax(top_k(logits / T)) in float64."""
    z = np.asarray(logits, dtype=np.float64) / float(temperature)
    keep = topk_mask(z, top_k)
    m = z[keep].max()
    w = np.where(keep, np.exp(z - m), 0.0)
    return w / w.sum()


def invcdf(w, u):
    """Smallest id v (ascending) with cumsum(w)[v] > u * sum(w); sequential
    float64 sums.  Falls back to the last id of positive weight."""
    w = np.asarray(w, dtype=np.float64)
    c = np.cumsum(w)
    target = u * c[-1]
    idx = int(np.searchsorted(c, target, side="right"))
    if idx >= w.shape[0]:
        idx = int(np.nonzero(w > 0)[0][-1])
    return idx


def argmax_lowest(logits):
    """argmax with ties to the lowest id (numpy's argmax returns the first)."""
    return int(np.argmax(np.asarray(logits)))


def accept_prob(p, q, t):
    """alpha = min(p(t)/q(t), 1) with the zero-q reading above."""
    pt, qt = float(p[t]), float(q[t])
    if qt > 0.0:
        return min(pt / qt, 1.0)
    return 1.0 if pt > 0.0 else 0.0


def residual(p, q):
    """Unnormalised residual [p - q]_+ (the paper's tilde p_k times its sum)."""
    return np.maximum(np.asarray(p, np.float64) - np.asarray(q, np.float64), 0.0)


def point_mass(V, t):
    q = np.zeros(V, dtype=np.float64)
    q[t] = 1.0
    return q


def select_position(rule, L, t, ref, u0, u1, temperature=1.0, top_k=0):
    """Apply one rule at one position.

    L    -- scoring logits (V_img,) for this position (the backbone's p_k, before warp)
    t    -- current token (image-code index, 0-based)
    ref  -- reference logits (V_img,) or None for a point mass at t (rule C only)
    u0, u1 -- the accept-test and sampling uniforms
    Returns (new_token, accepted, ref_replaced) where ref_replaced says the
    reference distribution becomes this round's p (rule C rejection).
    """
    if rule == RULE_GREEDY:
        a = argmax_lowest(L)
        return a, a == t, False
    p = warp(L, temperature, top_k)
    if rule == RULE_SAMPLE:
        a = invcdf(p, u1)
        return a, a == t, False
    if rule != RULE_ACCEPT_REJECT:
        raise ValueError("unknown rule")
    q = point_mass(p.shape[0], t) if ref is None else warp(ref, temperature, top_k)
    alpha = accept_prob(p, q, t)
    if u0 < alpha:
        return t, True, False
    r = residual(p, q)
    if not r.sum() > 0.0:
        return t, True, False
    return invcdf(r, u1), False, True


def sample_first(rule, L, u1, temperature=1.0, top_k=0):
    """The first image token comes from the prefill's last logits with no draft:
    argmax for rule (A), otherwise a plain sample of warp(L)."""
    if rule == RULE_GREEDY:
        return argmax_lowest(L)
    return invcdf(warp(L, temperature, top_k), u1)
