"""Pass plan of one image under the SSD schedule (oracle, test infrastructure).

Paper: Sec. 3.3 (horizontal heads finish the current row, then k_v vertical
heads draft whole rows); Sec. 4 "SSD Configuration" (5 horizontal tokens with
one verification round; k_v rows per vertical iteration; staged verification
with b base rounds on all rows of the group and i incremental rounds on the
trailing rows); Appendix "Multi-Row Anticipation Ablations" (joint = all rounds
on all rows; staged = commit the leading row before refining the trailing one);
Sec. 3.3 "Verification as Auto Correction" (a fixed number of rounds, then one
commit pass).

Readings:
  * pass 1 is the prefix prefill; its last logits give the first image token
    with no draft;
  * the remaining W-1 tokens of row 0 go in blocks of k_h; the first block also
    carries the already-chosen first token as a fixed (unverified) position;
  * vertical rows go in groups of up to k_v rows; after the b joint rounds the
    leading row is committed, then every later row of the group gets i rounds
    on the still-uncommitted rows of the group followed by its own commit;
  * joint verification (all rounds on the whole group) is the staged plan
    with i = 0: the group's rows are committed one after another;
  * the verify round index that feeds the random counter increases over the
    whole image, so no (position, round) pair repeats;
  * end-of-line layout (the Lumina-mGPT and Emu3 backbones: their AR step
    counts are H (W + 1), Appendix tables of the configuration sweeps): each
    image row is followed by one fixed end-of-line token, so row y occupies
    sequence positions y (W + 1) .. y (W + 1) + W; the end-of-line token rides
    along with the block that completes its row (the last horizontal run, each
    row of a vertical group) and is never verified, so the pass count is the
    same as without it;
  * drafting happens where the paper puts it: before each horizontal run the
    horizontal heads draft the run from the last token already chosen (after
    the prefill: the first token), and at the start of each vertical group the
    vertical heads draft the group's rows from the completed row above.
    Drafting is not a backbone pass.

Pin: tests/test_schedule.py -- the pass count equals all 31 step counts printed
in the paper's tables (verification rounds, vertical lookahead, Pareto sweep,
configuration sweeps for the three backbones, joint-vs-staged ablation).
"""


def plan(H, W, k_h=5, h_rounds=1, k_v=1, b=2, i=0, eol=False):
    """List of ops for one image.  Block coordinates are image indices
    (row-major, 0 = top-left); with eol, verify/commit coordinates are sequence
    positions after the prompt (row y starts at y (W + 1)) and blocks that end a
    row include its end-of-line position (draft ops stay in image indices).  Ops:
      ("prefill",)
      ("first",)                                -- pick image token 0 from the carry
      ("verify", start, K, n_fixed, round)      -- one verify-and-correct round
      ("commit", start, K)                      -- commit pass over [start, start+K)
      ("draft_h", src, n)                       -- horizontal heads 1..n draft src+1..src+n
      ("draft_v", y0, m)                        -- vertical heads 1..m draft rows y0+1..y0+m
                                                   from row y0
    """
    ops = [("prefill",), ("first",)]
    rnd = 0
    RW = W + 1 if eol else W  # sequence positions per row
    tail = 1 if eol else 0    # end-of-line position closing a row

    def verify(start, K, nf, count):
        nonlocal rnd
        for _ in range(count):
            ops.append(("verify", start, K, nf, rnd))
            rnd += 1

    # horizontal stage on row 0
    s = 1
    first = True
    while s < W:
        e = min(s + k_h, W)
        t = tail if e == W else 0
        if first:
            ops.append(("draft_h", 0, e - 1))
            verify(0, e + t, 1, h_rounds)
            ops.append(("commit", 0, e + t))
            first = False
        else:
            ops.append(("draft_h", s - 1, e - s))
            verify(s, e - s + t, 0, h_rounds)
            ops.append(("commit", s, e - s + t))
        s = e
    if W == 1:  # degenerate one-column grid: commit the first token alone
        ops.append(("commit", 0, 1 + tail))
    # vertical stage, groups of up to k_v rows
    y = 1
    while y < H:
        m = min(k_v, H - y)
        ops.append(("draft_v", y - 1, m))
        verify(y * RW, m * RW, 0, b)
        ops.append(("commit", y * RW, RW))
        for j in range(1, m):
            verify((y + j) * RW, (m - j) * RW, 0, i)
            ops.append(("commit", (y + j) * RW, RW))
        y += m
    return ops


def n_passes(ops):
    """Backbone forward passes of a plan (prefill + verify rounds + commits)."""
    return sum(1 for o in ops if o[0] in ("prefill", "verify", "commit"))
