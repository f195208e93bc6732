"""The update's chunk-ownership rule, modelled on the CPU.

The fused update cuts the sorted look-ups into chunks of C and hands every
segment (the look-ups of one row) to exactly one wavefront:
  * a segment inside one chunk is summed and applied by that chunk;
  * with 64-lane rows, a segment that begins in a chunk, crosses its end and
    ends within the next chunk's first `win` look-ups is walked to its end by
    the chunk where it begins, and the next chunk starts after it;
  * any other crossing segment is parked as partial sums (slot 2c for a
    chunk's first segment, 2c+1 for its last), groups of 16 chunks that one
    segment fills are pre-summed, and the chunk where the segment begins adds
    the partials in chunk order and applies the row.
This model restates those decisions (which keys each side looks at, which
slot it writes, which chunk the fix-up takes) and checks, on random segment
lengths around the chunk and window lengths, that every segment is applied
exactly once with all its look-ups in increasing order.  It checks the rule,
not the kernels; the GPU parity tests check the kernels.
"""
import numpy as np
import pytest

NOKEY = -1
GROUP = 16  # chunks per pre-summed group


def applied_segments(keys, C, U, win, fix_win=None):
    """Segments as the update applies them: {key: [positions summed]}.
    win = 0: no walking past a chunk end (rows of fewer than 64 lanes).
    fix_win: the window the fix-up assumes (the update's own by default)."""
    fix_win = win if fix_win is None else fix_win
    NS = len(keys)
    key = lambda i: int(keys[i]) if 0 <= i < NS else NOKEY
    nch = (NS + C - 1) // C
    carry, out = {}, {}

    def apply(k, pos):
        assert k not in out, f"row {k} applied twice"
        out[k] = pos

    for c in range(nch):
        lo, hi0 = c * C, min(c * C + C, NS)
        kprev, knext0, klast = key(lo - 1), key(hi0), key(hi0 - 1)
        hi, knext = hi0, knext0
        first_open, is_first, s0 = kprev == key(lo), True, lo
        if win:
            kpp = key(lo - C - 1) if lo > C else NOKEY
            if knext0 == klast and kprev != klast:
                past = [r for r in range(win) if hi0 + r >= NS or key(hi0 + r) != klast]
                if past:
                    hi = hi0 + past[0]
                    knext = key(hi)
            if first_open and kpp != kprev:
                lead = [r for r in range(win) if lo + r >= hi0 or key(lo + r) != kprev]
                if lead:
                    s0 = lo + lead[0]
                    if s0 >= hi0:
                        continue
                    first_open, is_first = False, False
        cur, acc = key(s0), []
        for s in range(s0, hi):
            if key(s) != cur:
                if is_first and first_open:
                    carry[2 * c] = acc
                else:
                    apply(cur, acc)
                cur, acc, is_first = key(s), [], False
            acc = acc + [s]
        last_open = knext == cur
        if is_first and (first_open or last_open):
            carry[2 * c] = acc
        elif not is_first and last_open:
            carry[2 * c + 1] = acc
        else:
            apply(cur, acc)

    ngroups = (nch + GROUP - 1) // GROUP
    gsum = {}
    for g in range(ngroups):
        c0 = g * GROUP
        if c0 > 0 and c0 + GROUP <= nch and (c0 + GROUP) * C < NS and key(c0 * C - 1) == key((c0 + GROUP) * C):
            gsum[g] = sum((carry[2 * (c0 + u)] for u in range(GROUP)), [])

    for c in range(nch):
        lo, hi = c * C, c * C + C
        if hi >= NS:
            continue
        kl = key(hi - 1)
        need = key(hi) == kl and key(lo - 1) != kl
        if fix_win:
            need = need and hi + fix_win - 1 < NS and key(hi + fix_win - 1) == kl
        if not need:
            continue
        acc = list(carry[2 * c + 1 if key(lo) != kl else 2 * c])
        c2 = c + 1
        while True:
            g, off = divmod(c2, GROUP)
            if off == 0 and g in gsum:
                acc += gsum[g]
                c2 += GROUP
                continue
            acc += carry[2 * c2]
            if not ((c2 + 1) * C < NS and key((c2 + 1) * C) == kl):
                break
            c2 += 1
        apply(kl, acc)
    return out


def check(lengths, C, U, win):
    keys = np.repeat(np.arange(len(lengths), dtype=np.int64) * 3 + 1, lengths)
    got = applied_segments(keys, C, U, win)
    starts = np.r_[0, np.cumsum(lengths)]
    assert sorted(got) == [int(k) for k in np.unique(keys)]
    for i, k in enumerate(np.arange(len(lengths)) * 3 + 1):
        assert got[int(k)] == list(range(starts[i], starts[i + 1])), f"segment {i} summed wrongly"


@pytest.mark.parametrize("seed", range(4))
def test_every_segment_applied_once(seed):
    rng = np.random.default_rng(seed)
    for trial in range(150):
        win = int(rng.choice([0, 64]))
        C = int(rng.choice([128, 256])) if win else int(rng.choice([8, 32, 128]))
        kinds = np.array([1, 2, 3, win - 1, win, win + 1, C - 1, C, C + 1, 2 * C - 1, 2 * C,
                          2 * C + 1, GROUP * C, GROUP * C + 1, 20 * C + 3])
        kinds = kinds[kinds > 0]
        L = rng.choice(kinds, int(rng.integers(1, 60)))
        if trial % 3 == 0:
            L = rng.integers(1, 3 * C, int(rng.integers(1, 60)))
        check(L, C, 8, win)


@pytest.mark.parametrize("fix_win", [63, 65, 0])
def test_model_catches_a_wrong_window(fix_win):
    """The check is not vacuous: with chunks of 128 and a window of 64, a
    segment crossing the first boundary and ending 63 or 64 look-ups past it
    is applied twice, or never, by a fix-up that assumes another window."""
    for tail in (63, 64):
        lengths = np.array([100, 28 + tail, 300, 5])
        check(lengths, 128, 8, 64)
    # (a missing partial sum shows as a KeyError, a second application or a
    # row never applied as an AssertionError)
    with pytest.raises((AssertionError, KeyError)):
        for tail in (63, 64):
            lengths = np.array([100, 28 + tail, 300, 5])
            keys = np.repeat(np.arange(lengths.size, dtype=np.int64) * 3 + 1, lengths)
            got = applied_segments(keys, 128, 8, 64, fix_win=fix_win)
            assert sorted(got) == [int(k) for k in np.unique(keys)]
