"""Host-side invariants of the bf16 GEMM launch plans (no GPU: the planner is
host code inside libssd.so, called here through its C++ symbols).

Every plan must tile its problem exactly (feature blocks x block width = N,
splits x chunks x chunk width = K), give the tiled kernel's pipeline a stage
count it runs (a multiple of the depth for depths 2 and 4, at least two
stages for depth 3), and fit the workspaces that sessions
and draft heads size once, at creation, by planning a fixed set of row
counts: a plan for any row count must need no more split-K partials,
arrival counters or per-row x^2 parts than the largest of that set, or a
launch would write past its buffer.  Shapes: the projections of the 1B, 7B
and 8B backbones and of a draft head (m = 2d), row counts 1..4352.
"""
import ctypes

import pytest

import paper_2606_20543_amd as ssd
import synth


class GemmPlan(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in ("MT", "NT", "KCB", "WV", "S", "n_fb", "kchunks", "bn", "xcd", "tile",
                                            "m_tiles", "depth", "tail_fb", "tail_S", "tail_nt")]


TILE_ROWS, TILE_KT = 128, 64
RMS_MAX_PARTS = 128


@pytest.fixture(scope="module")
def planner():
    L = ssd.lib()
    plan = getattr(L, "_ZN3ssd14gemm_plan_bf16Eiiii")
    plan.argtypes = [ctypes.c_int] * 4
    plan.restype = GemmPlan
    parts = getattr(L, "_ZN3ssd20gemm_partials_floatsERKNS_8GemmPlanEi")
    parts.argtypes = [ctypes.POINTER(GemmPlan), ctypes.c_int]
    parts.restype = ctypes.c_size_t
    return lambda M, N, K, xcd=8: plan(M, N, K, xcd), lambda p, M: parts(ctypes.byref(p), M)


def counters(p):
    """Arrival counters a plan uses (split-K reductions)."""
    if p.tile and p.tail_fb:
        return 0 if p.tail_nt else (p.n_fb - p.tail_fb) * p.m_tiles
    if p.tile:
        return p.n_fb * p.m_tiles if p.S > 1 else 0
    return p.n_fb


def row_classes():
    """The row counts workspaces are sized over (the planner's classes: up to
    16, 32 and 64 rows, 65..128, then each count of 128-row tiles to 256)."""
    return [1, 16, 17, 32, 33, 64, 65, 128] + [128 * t for t in range(2, 257)]


def shapes(m):
    d, D = m.d_model, m.head_dim
    mi = 2 * d
    return [((m.n_heads + 2 * m.n_kv_heads) * D, d), (d, m.n_heads * D), (2 * m.d_ff, d), (d, m.d_ff),
            (m.v_img, d), (d, 2 * d), (2 * mi, d), (d, mi)]


ROWS = sorted(set(list(range(1, 300)) + list(range(300, 4353, 37)) + [512, 1024, 2048, 4224, 4288, 4352]))


@pytest.mark.parametrize("model", [synth.M1B, synth.M7B, synth.M8B], ids=["1b", "7b", "8b"])
def test_plans_tile_their_problem(planner, model):
    plan, _ = planner
    for N, K in shapes(model):
        for M in ROWS:
            p = plan(M, N, K)
            where = f"M={M} N={N} K={K}"
            assert p.S >= 1 and p.n_fb >= 1, where
            if p.tile == 3:
                # 128 x 256 (or 128 x 192) tiles of eight waves: K split within 256 workgroups, >= 32 stages each
                assert M > 64, where
                assert p.NT in (3, 4) and p.bn == 64 * p.NT and p.n_fb * p.bn == N and p.WV == 8, where
                assert p.m_tiles == (M + TILE_ROWS - 1) // TILE_ROWS, where
                assert p.kchunks * p.S * TILE_KT == K and p.kchunks >= 32, where
                assert p.S == 1 or p.n_fb * p.m_tiles * p.S <= 256, where
                if p.NT == 3:
                    # only where the 256-feature grid would leave CUs idle, and never on a residual projection
                    assert N > K and p.n_fb * p.m_tiles * p.S <= 256 and not p.tail_fb, where
                    assert (N // 256) * p.m_tiles * p.S < p.n_fb * p.m_tiles * p.S, where
                if p.tail_fb:
                    # whole rounds of 256 tiles, then the remaining feature blocks K-split within one more,
                    # or as 128 x 192 tiles in one more
                    assert p.S == 1 and p.NT == 4 and 0 < p.tail_fb < p.n_fb, where
                    assert (p.tail_fb * p.m_tiles) % 256 == 0, where
                    r = (p.n_fb - p.tail_fb) * p.m_tiles
                    assert 0 < r < 256, where
                    if p.tail_nt:
                        fr = (p.n_fb - p.tail_fb) * 256
                        assert p.tail_nt == 3 and p.tail_S == 1 and N > K and fr % 192 == 0, where
                        assert r < (fr // 192) * p.m_tiles <= 256, where
                    else:
                        assert r * p.tail_S <= 256 and p.tail_S > 1, where
                        assert (K // TILE_KT) % p.tail_S == 0 and K // TILE_KT // p.tail_S >= 16, where
                else:
                    assert p.tail_S == 1 and p.tail_nt == 0, where
            elif p.tile:
                assert M > 64, where
                assert p.NT in (2, 4) and p.bn == 32 * p.NT and p.n_fb * p.bn == N, where
                assert p.m_tiles == (M + TILE_ROWS - 1) // TILE_ROWS, where
                assert p.kchunks * p.S * TILE_KT == K, where
                # depth 3 (128-feature tiles): any count of at least two stages;
                # depths 2 and 4 run whole groups of stages per trip
                if p.depth == 3:
                    assert p.NT == 4 and p.kchunks >= 2, where
                else:
                    assert p.depth in (2, 4) and p.kchunks % p.depth == 0, where
                if p.S > 1:
                    assert p.n_fb * p.m_tiles * p.S < 512, where  # splits stop once the grid fills the CUs
            else:
                assert p.n_fb * p.bn >= N > (p.n_fb - 1) * p.bn, where
                assert p.KCB * p.kchunks * p.S * 32 == K, where
            if N == model.d_model:
                # consumers read at most this many per-row x^2 parts
                assert p.n_fb <= (N + 63) // 64 <= RMS_MAX_PARTS, where


@pytest.mark.parametrize("model", [synth.M1B, synth.M7B, synth.M8B], ids=["1b", "7b", "8b"])
def test_workspace_classes_bound_every_row_count(planner, model):
    plan, partials = planner
    for N, K in shapes(model):
        cap_part = max(partials(plan(Mc, N, K, 0), Mc) for Mc in row_classes())
        cap_cnt = max(counters(plan(Mc, N, K, 0)) for Mc in row_classes())
        for M in ROWS:
            for xcd in (0, 8):
                p = plan(M, N, K, xcd)
                assert partials(p, M) <= cap_part, f"M={M} N={N} K={K}: split-K partials beyond the workspace"
                assert counters(p) <= cap_cnt, f"M={M} N={N} K={K}: arrival counters beyond the workspace"


def test_tiled_plan_choices(planner):
    """The measured choices: 128 x 256 eight-wave tiles where each workgroup
    keeps at least 32 stages after the K split (at most 256 workgroups), else
    128-feature tiles (three weight stages) where they make at least 160
    workgroups, 64-feature tiles with four pipeline stages otherwise, K split
    until the grid reaches 256 workgroups; 128 x 192 eight-wave tiles where
    the 256-feature grid leaves CUs idle; streaming launches up to 64 rows."""
    plan, _ = planner
    m = synth.M8B
    gu = plan(512, 2 * m.d_ff, m.d_model)  # 112 x 4 = 448 tiles of 128 x 256: 256, then 192 as 256 of 128 x 192
    assert (gu.tile, gu.bn, gu.S, gu.tail_fb, gu.tail_nt, gu.tail_S) == (3, 256, 1, 64, 3, 1)
    lm = plan(512, m.v_img, m.d_model)  # 128 x 4 = 512
    assert (lm.tile, lm.S) == (3, 1)
    dn = plan(512, m.d_model, m.d_ff)  # 16 x 4 tiles, 224 stages in 4 splits of 56
    assert (dn.tile, dn.S, dn.kchunks) == (3, 4, 56)
    nq = (m.n_heads + 2 * m.n_kv_heads) * m.head_dim
    qkv = plan(512, nq, m.d_model)  # 32 x 4 tiles of 128 x 192 in 2 splits of 32 stages (24 x 4 x 2 of 256: 192 CUs)
    assert (qkv.tile, qkv.NT, qkv.bn, qkv.S, qkv.kchunks) == (3, 3, 192, 2, 32)
    qkv1k = plan(1024, nq, m.d_model)  # 32 x 8 tiles of 128 x 192, no split
    assert (qkv1k.tile, qkv1k.NT, qkv1k.S) == (3, 3, 1)
    o = plan(512, m.d_model, m.n_heads * m.head_dim)  # 16 x 4 x 4 splits would leave 16 stages: 128 x 128
    assert (o.tile, o.NT, o.S, o.depth) == (1, 2, 1, 4)
    gu1k = plan(1024, 2 * m.d_ff, m.d_model)  # 896 tiles: 768 in three full rounds, 128 in two splits of 32
    assert (gu1k.tile, gu1k.S, gu1k.tail_fb, gu1k.tail_S, gu1k.tail_nt) == (3, 1, 96, 2, 0)
    assert lm.tail_fb == 0 and (lm.NT, dn.NT) == (4, 4)  # two whole rounds; a residual projection
    o1 = plan(256, synth.M1B.d_model, synth.M1B.d_model)  # 32 x 2 tiles of 64 features: 4 splits
    assert (o1.tile, o1.NT, o1.S) == (1, 2, 4)
    for M in (1, 24, 48, 64):
        assert plan(M, 2 * synth.M1B.d_ff, synth.M1B.d_model).tile == 0
