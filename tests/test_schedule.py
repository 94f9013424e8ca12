"""Pass plan of an image vs the step counts printed in the paper's tables."""
import os

import pytest

from oracle import schedule as S

GOLD = os.path.join(os.path.dirname(__file__), "golden", "step_counts.txt")


def _rows():
    out = []
    for line in open(GOLD):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        t, bb, side, kv, b, i, steps = line.split()
        out.append((t, bb, int(side), int(kv), int(b), int(i), int(steps)))
    return out


ROWS = _rows()


def test_fixture_size():
    assert len(ROWS) == 75


@pytest.mark.parametrize("row", ROWS, ids=lambda r: f"{r[0]}-{r[1]}-v{r[3]}b{r[4]}i{r[5]}")
def test_pass_count_matches_paper(row):
    _, _, side, kv, b, i, steps = row
    ops = S.plan(side, side, k_h=5, h_rounds=1, k_v=kv, b=b, i=i)
    assert S.n_passes(ops) == steps


def test_plan_covers_every_position_once():
    for (H, W, kv, b, i) in [(24, 24, 1, 2, 0), (48, 48, 2, 5, 4), (7, 3, 3, 1, 1), (5, 1, 1, 2, 0), (1, 9, 1, 1, 0)]:
        ops = S.plan(H, W, k_v=kv, b=b, i=i)
        committed = []
        for o in ops:
            if o[0] == "commit":
                committed += list(range(o[1], o[1] + o[2]))
        assert committed == list(range(H * W))


def test_rounds_strictly_increase():
    ops = S.plan(48, 48, k_v=2, b=5, i=4)
    rnds = [o[4] for o in ops if o[0] == "verify"]
    assert rnds == list(range(len(rnds)))


def test_staged_plan_worked_example():
    """A 4 x 2 grid with groups of three rows, b = 2 joint rounds and i = 1
    incremental round (Sec. 4 "SSD Configuration"; Appendix "Multi-Row
    Anticipation Ablations"), written out by hand: row 0's last token as one
    horizontal run behind the fixed first token, then the b rounds over all
    three rows of the group, the leading row committed, one round over the
    two rows still open, the next row committed, one round over the last."""
    assert S.plan(4, 2, k_h=5, h_rounds=1, k_v=3, b=2, i=1) == [
        ("prefill",), ("first",),
        ("draft_h", 0, 1), ("verify", 0, 2, 1, 0), ("commit", 0, 2),
        ("draft_v", 0, 3), ("verify", 2, 6, 0, 1), ("verify", 2, 6, 0, 2), ("commit", 2, 2),
        ("verify", 4, 4, 0, 3), ("commit", 4, 2),
        ("verify", 6, 2, 0, 4), ("commit", 6, 2),
    ]
