"""A host model of the decode kernels' work partition (the flat granule space,
the weighted split into per-wave ranges, the piece resolver, and the merge
plan's slots), checked for the invariants the kernels rely on:

* every real granule of every sequence is covered by exactly one piece;
* no piece is empty or reaches past its sequence's granules;
* the merge plan names exactly the slots the pieces are written to;
* some ranges may hold virtual granules only (those waves do no work).

It restates the arithmetic of `build_tables`, `Split`, `next_piece` and
`write_plan` (kva_kernels.hip) in Python, so a change to the partition can be
checked here on the CPU before it runs on the GPU."""
import numpy as np
import pytest

import workloads as W


def _simulate(lens, vgran, waves_per_head, wa=28, wb=25, weighted=True):
    L = np.asarray(lens, dtype=np.int64)
    B = len(L)
    n = (L + 15) // 16
    n_aug = np.where(n > 0, n + vgran, 0)
    pre = np.concatenate([[0], np.cumsum(n_aug)])
    gtot = int(pre[-1])
    if gtot == 0:
        return 0, 0
    wh = min(waves_per_head, (gtot + 1) // 2)
    if not weighted:
        wa = wb = 1

    def wsum(i):
        return ((i + 1) >> 1) * wa + (i >> 1) * wb

    if gtot * min(wa, wb) < wsum(wh):
        wa = wb = 1
    x = [gtot * wsum(i) // wsum(wh) for i in range(wh + 1)]

    def range_of(y):
        v = ((y + 1) * wsum(wh) - 1) // gtot
        k = v // (wa + wb)
        i = 2 * k + (1 if v - k * (wa + wb) >= wa else 0)
        return min(i, wh - 1)

    covered = [np.zeros(int(n[b]), dtype=int) for b in range(B)]
    slots, idle = set(), 0
    for i in range(wh):
        ru, ru1 = x[i], x[i + 1]
        rb = min(max(int(np.searchsorted(pre, ru, side="right")) - 1, 0), B - 1)
        pieces = 0
        while True:
            done = False
            while True:
                if ru >= ru1:
                    done = True
                    break
                st, en = int(pre[rb]), int(pre[rb + 1])
                while en <= ru and rb + 1 < B:
                    rb += 1
                    st, en = en, int(pre[rb + 1])
                st += vgran if en > st else 0       # the sequence's virtual granules
                if ru >= st:
                    break
                ru = min(st, ru1)
            if done:
                break
            cnt = (int(L[rb]) + 15) // 16
            lo = cnt - (en - st)
            pe = min(ru1, en)
            g0, g1 = ru - st + lo, pe - st + lo
            assert 0 <= g0 < g1 <= cnt
            covered[rb][g0:g1] += 1
            slots.add(i + rb)
            pieces += 1
            ru = pe
        idle += pieces == 0
    for b in range(B):
        assert (covered[b] == 1).all(), b
    plan = set()
    for b in range(B):
        en = int(pre[b + 1])
        st = int(pre[b]) + (vgran if en > pre[b] else 0)
        if en > st:
            for r in range(range_of(st), range_of(en - 1) + 1):
                plan.add(r + b)
    assert plan == slots
    return wh, idle


_LENGTHS = None


def _lengths():
    global _LENGTHS
    if _LENGTHS is not None:
        return _LENGTHS
    rng = np.random.default_rng(514)
    mixed = rng.integers(0, 2500, size=41)
    mixed[[3, 17]] = 0
    mixed[9] = 1
    _LENGTHS = {
        "short_and_long": [1, 7, 16, 17, 300, 1025, 3000],
        "mixed_with_empty": list(mixed),
        "config3": list(W.config_lengths(3)),
        "config4": list(W.config_lengths(4)),
        "single_token": [1],
        "ragged": [1, 2, 15, 16, 17, 31, 33, 64, 100, 255, 256, 257, 1000, 1023, 2049, 4097],
        "all_empty_but_one": [0, 0, 5, 0],
    }
    return _LENGTHS


@pytest.mark.parametrize("name", list(_lengths()))
@pytest.mark.parametrize("vgran", [0, 1, 2, 7, 64])
def test_partition_covers_every_granule_once(name, vgran):
    lens = _lengths()[name]
    for waves in (128, 256, 512):
        for weighted in (True, False):
            _simulate(lens, vgran, waves, weighted=weighted)


def test_virtual_granules_can_leave_ranges_without_work():
    """With virtual granules a range may hold none of a sequence's real
    granules: the kernel must return such a wave before its first load."""
    _, idle0 = _simulate([1, 7, 16, 17, 300, 1025, 3000], 0, 512)
    _, idle2 = _simulate([1, 7, 16, 17, 300, 1025, 3000], 2, 512)
    assert idle0 == 0 and idle2 > 0
