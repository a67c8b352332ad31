"""CPU model of the streaming copy's work split (the index arithmetic of
copy_kernel, restated): the buffer of n16 16-byte words is cut into one slice
per XCD in proportion to the copy's CUs there, and the workgroups of one
residue class of block indices (the ones the hardware deals to one XCD)
stride over that slice.  Checked before any device run, for every dispatch
rotation (which XCD the dealing starts on): every word is copied exactly once
per pass and no index leaves [0, n16).
"""
import numpy as np
import pytest

THREADS, UNROLL = 256, 4


def copy_grid(cus):
    return len(cus) * max(1, 8 * max(cus))


def model_counts(n16: int, cus, grid: int, rotation: int) -> np.ndarray:
    """How often each word is written in one pass, if block b runs on XCD
    (b mod n + rotation) mod n; raises if an index leaves the buffer."""
    n_x = len(cus)
    total = sum(cus)
    counts = np.zeros(n16, dtype=np.int64)
    block = UNROLL * THREADS
    for b in range(grid):
        x = (b % n_x + rotation) % n_x
        if cus[x] <= 0 or total == 0:
            continue
        before = sum(cus[:x])
        lo = n16 * before // total
        hi = n16 * (before + cus[x]) // total
        cls = b % n_x
        members = (grid - cls + n_x - 1) // n_x
        first = lo + (b // n_x) * block
        stride = members * block
        for i0 in range(first, hi, stride):
            # lanes t = 0..255, words i0 + t + j * 256, kept while < hi
            idx = i0 + np.arange(THREADS)[None, :] + THREADS * np.arange(UNROLL)[:, None]
            idx = idx[idx < hi]
            assert idx.size == 0 or (idx.min() >= 0 and idx.max() < n16)
            np.add.at(counts, idx, 1)
    return counts


CASES = [
    (64 * 1024 * 1024 // 16 // 64, [32] * 8),            # 1 MiB, the whole chip
    (12345, [32] * 8),                                  # ragged, smaller than one round
    (100003, [0, 0, 0, 0, 31, 31, 31, 31]),             # one die's XCDs (XCD filter)
    (77777, [17, 9, 23, 16, 12, 20, 15, 16]),           # a random 128-CU complement
    (1 << 16, [3, 0, 0, 0, 0, 0, 0, 1]),                # very uneven
    (1, [32] * 8),                                      # a single word
]


@pytest.mark.parametrize("n16,cus", CASES)
def test_every_word_once_per_pass_for_every_rotation(n16, cus):
    grid = copy_grid(cus)
    for rot in range(len(cus)):
        c = model_counts(n16, cus, grid, rot)
        assert (c == 1).all(), (rot, int((c == 0).sum()), int((c > 1).sum()))


def test_explicit_small_grids_cover_the_buffer():
    # a grid that is not a multiple of the XCD count (fewer members in the last classes)
    cus = [32] * 8
    for grid in (1, 7, 9, 61):
        for rot in (0, 3):
            c = model_counts(5000, cus, grid, rot)
            # classes without a workgroup leave their slice uncopied; the rest once
            classes = {b % 8 for b in range(grid)}
            x_with = {(k + rot) % 8 for k in classes}
            for x in range(8):
                lo, hi = 5000 * x // 8, 5000 * (x + 1) // 8
                want = 1 if x in x_with else 0
                assert (c[lo:hi] == want).all(), (grid, rot, x)
