"""Host-side cache-load planner (mask_plan_copies): the copies a cached block's
load issues for one request (Sec. 4.2, Fig. 8: only the unmasked image tokens'
cached rows are loaded). Host-only, no GPU."""
import math

import numpy as np
import pytest

from paper_2505_20600_amd import maskstep as MS
from paper_2505_20600_amd import workloads as W


def _merged_runs(m, gap):
    """Unmasked runs in token order, merged across masked gaps of <= gap rows."""
    out, n, N = [], 0, len(m)
    while n < N:
        while n < N and m[n]:
            n += 1
        if n >= N:
            break
        n0 = n
        while n < N and not m[n]:
            n += 1
        if out and n0 - (out[-1][0] + out[-1][1]) <= gap:
            out[-1] = (out[-1][0], n - out[-1][0], 1)
        else:
            out.append((n0, n - n0, 1))
    return out


def _cost(plan, C):
    return sum(C + w * h for _, w, h in plan)


def _check_plan(plan, m, P):
    """Every copy in bounds, strided copies narrower than a grid row, copies
    disjoint, every unmasked row covered; returns the rows moved."""
    N = len(m)
    hits = np.zeros(N, np.int32)
    for n0, w, h in plan:
        assert w >= 1 and h >= 1 and n0 >= 0
        assert h == 1 or w < P
        assert n0 + (h - 1) * P + w <= N
        for i in range(h):
            hits[n0 + i * P:n0 + i * P + w] += 1
    assert hits.max(initial=0) <= 1, "copies overlap"
    assert (hits[m == 0] == 1).all(), "an unmasked row is not loaded"
    return int(hits.sum())


def _masks():
    g = np.random.default_rng(11)
    out = {"empty": np.zeros((16, 24), np.uint8), "full": np.ones((16, 24), np.uint8)}
    rect = np.zeros((64, 64), np.uint8)
    rect[10:30, 20:50] = 1
    out["rect"] = rect
    two = np.zeros((64, 64), np.uint8)
    two[5:25, 4:20] = 1
    two[12:40, 36:60] = 1
    out["two_rects_side_by_side"] = two
    out["scatter"] = (g.random((32, 40)) < 0.3).astype(np.uint8)
    stripes = np.zeros((32, 32), np.uint8)
    stripes[:, ::3] = 1
    out["column_stripes"] = stripes
    out["last_row"] = np.zeros((8, 8), np.uint8)
    out["last_row"][7] = 1
    for i, r in enumerate((0.05, 0.2, 0.45, 0.8)):
        out[f"blob{r}"] = W.blob_mask(64, 64, r, W.rng(9, 3, i)).reshape(64, 64)
        out[f"ellipse{r}"] = W.ellipse_mask(48, 80, r, W.rng(9, 4, i)).reshape(48, 80)
    return out


MASKS = _masks()


@pytest.mark.parametrize("C", [0.0, 1.0, 6.5, 42.7, 113.8, 1e4])
@pytest.mark.parametrize("name", sorted(MASKS))
def test_plan_covers_every_unmasked_row_and_beats_merged_runs(name, C):
    mask = MASKS[name]
    H, P = mask.shape
    m = mask.reshape(-1)
    plan = MS.mask_plan_copies(m, H, P, C)
    moved = _check_plan(plan, m, P)
    assert moved >= int((m == 0).sum())
    assert _cost(plan, C) <= _cost(_merged_runs(m, math.floor(min(C, m.size))), C) + 1e-9
    if C == 0.0:
        assert moved == int((m == 0).sum())   # commands free: exactly the unmasked rows


def test_degenerate_masks():
    assert MS.mask_plan_copies(np.zeros(96, np.uint8), 8, 12, 42.7) == [(0, 96, 1)]
    assert MS.mask_plan_copies(np.ones(96, np.uint8), 8, 12, 42.7) == []
    one = np.zeros(96, np.uint8)
    one[0] = 1
    assert MS.mask_plan_copies(one, 8, 12, 42.7) == [(1, 95, 1)]


def test_rectangle_hole_is_skipped_by_one_strided_copy():
    """A 20-row x 30-column masked rectangle on a 64 x 64 grid: the rows above
    and the left part of its first row, one strided copy from each row's right
    part to the next row's left part, then the rest: no masked row moved."""
    m = MASKS["rect"].reshape(-1)
    plan = MS.mask_plan_copies(m, 64, 64, 42.7)
    assert plan == [(0, 10 * 64 + 20, 1), (10 * 64 + 50, 34, 19), (29 * 64 + 50, 4096 - (29 * 64 + 50), 1)]
    assert _check_plan(plan, m, 64) == int((m == 0).sum())


def test_workload_masks_load_fewer_bytes_than_merged_runs():
    """On the 19-block d=3072 workload's blob masks (12 KiB K/V rows, a command
    worth 512 KiB) the plan is at least 4% cheaper under the cost model and
    moves at most 1.2x the unmasked rows (merged runs: ~1.3x)."""
    shape = W.CONFIGS["c5"]
    C = 512 * 1024 / (2 * shape.d_model * 2)
    plan_cost = runs_cost = moved = unmasked = 0.0
    for ms in range(4):
        for m in W.workload_mask("c5", shape, ms):
            plan = MS.mask_plan_copies(m, shape.grid_h, shape.grid_w, C)
            moved += _check_plan(plan, m, shape.grid_w)
            unmasked += int((m == 0).sum())
            plan_cost += _cost(plan, C)
            runs_cost += _cost(_merged_runs(m, math.floor(C)), C)
    assert plan_cost <= 0.96 * runs_cost
    assert moved <= 1.2 * unmasked


def test_plan_copies_validates_arguments():
    import ctypes as C
    m = np.zeros(64, np.uint8)
    n = C.c_int32()
    assert MS.load().mask_plan_copies(m.ctypes.data, 0, 64, 1.0, None, 0, C.byref(n)) == MS.MS_ESHAPE
    assert MS.load().mask_plan_copies(m.ctypes.data, 2048, 1024, 1.0, None, 0, C.byref(n)) == MS.MS_ESHAPE
    for bad in (-1.0, float("nan"), float("inf")):
        with pytest.raises(MS.MaskStepError) as e:
            MS.mask_plan_copies(m, 8, 8, bad)
        assert e.value.status == MS.MS_EINVAL
    two = np.zeros(64, np.uint8)
    two[30] = 1
    out = (C.c_int32 * 3)()
    st = MS.load().mask_plan_copies(two.ctypes.data, 8, 8, 0.0, out, 1, C.byref(n))
    assert st == MS.MS_ESHAPE and n.value == 2   # two copies, room for one
    assert MS.load().mask_plan_copies(None, 8, 8, 0.0, out, 1, C.byref(n)) == MS.MS_EINVAL


@pytest.mark.parametrize("H,P,kind", [(65536, 16, "column"), (1 << 20, 1, "runs"), (1024, 1024, "checker")])
def test_planner_time_stays_bounded_on_tall_and_busy_grids(H, P, kind):
    """The band search and the hole-dropping pass are bounded, so the planner's
    host time stays linear in the tokens (these took seconds to minutes with an
    unbounded band search)."""
    import time
    m = np.zeros((H, P), np.uint8)
    if kind == "column":
        m[:, 4:8] = 1
    elif kind == "runs":
        m[(np.arange(H) // 50) % 2 == 0] = 1
    else:
        m[::2, ::2] = 1
        m[1::2, 1::2] = 1
    t = time.perf_counter()
    plan = MS.mask_plan_copies(m.reshape(-1), H, P, 42.7)
    assert time.perf_counter() - t < 3.0
    _check_plan(plan, m.reshape(-1), P)
    if kind == "column":
        assert plan == [(0, 4, 1), (8, 12, H - 1), ((H - 1) * P + 8, 8, 1)]
