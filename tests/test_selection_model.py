"""Hazard checks of the selection kernels on a host model of their barrier
phases (tests/selection_model.py): threads run in a random order between
barriers and every LDS access is logged.  Over seeded launches at the
shapes that matter (one chunk of 8 or 16 keys per thread, several first-
level chunks with the group-maxima bound, survivor levels, a final level by
rank and by bitonic network, streaming rounds over device-side counts) and
with ties, NaN, +-0, infinities and padding, no phase may hold a
cross-thread read/write conflict, no word may be read before this launch
wrote it, every radix pass must have exactly one lane writing the digit
record, and the rows must equal a plain sort's.  The detector itself is
checked by planting two hazards: a missing barrier and a radix pass whose
digit record nobody writes.  The score-word statistics of first-level
chunks are checked against the direct ones on every launch."""
import numpy as np
import pytest

import selection_model as sm


def plain_topk(scores, k):
    keys = sm.pack_keys(scores, np.arange(len(scores)))
    top = sorted(keys, reverse=True)[:k]
    return [sm.key_row(x) for x in top] + [-1] * (k - len(top))


def make_scores(rng, n, kind):
    s = rng.normal(0.0, 1.0, n).astype(np.float32)
    if kind == "ties":
        s = (np.round(s * 8) / 8).astype(np.float32)
    elif kind == "specials":
        pick = rng.integers(0, 10, n)
        s[pick == 0] = np.nan
        s[pick == 1] = np.inf
        s[pick == 2] = -np.inf
        s[pick == 3] = -0.0
        s[pick == 4] = 0.0
    elif kind == "one-value":
        s[:] = 0.25
    elif kind == "mostly-nan":
        s[rng.random(n) < 0.97] = np.nan
    return s


CASES = [
    # n, k, kind: one block (8, 16 and 32 keys per thread), the first level with
    # the bound (groups of 64 .. 1 lanes, and none for k > 512), survivor
    # levels, rank (k <= 256) and bitonic (k > 256) finals
    (40, 40, "normal"),
    (4096, 64, "ties"),
    (4097, 100, "specials"),
    (8192, 1, "one-value"),
    (8193, 64, "normal"),
    (12000, 64, "specials"),
    (16384, 1024, "ties"),
    (3 * 8192 + 777, 8, "ties"),
    (3 * 8192 + 777, 300, "specials"),
    (3 * 8192 + 777, 1024, "mostly-nan"),
    (5 * 8192 - 3, 600, "normal"),
    (9 * 8192 + 5, 1024, "ties"),
]


@pytest.mark.parametrize("n,k,kind", CASES, ids=[f"{n}-{k}-{kind}" for n, k, kind in CASES])
def test_select_kernel_phases_are_race_free(n, k, kind):
    rng = np.random.default_rng(n * 31 + k)
    for seed in range(2):
        s = make_scores(rng, n, kind)
        got = sm.select_launch(s, k, np.random.default_rng(seed))   # raises Hazard on a race
        assert got == plain_topk(s, k)


@pytest.mark.parametrize("count,cap,k", [(37, 5000, 64), (3000, 5000, 64), (6000, 9000, 256),
                                         (20000, 20000, 1024), (9000, 17000, 300)])
def test_stream_kernel_rounds_are_race_free(count, cap, k):
    rng = np.random.default_rng(count + k)
    s = make_scores(rng, cap, "specials")
    keys = sm.pack_keys(s, np.arange(cap))
    # a candidate buffer: the first `count` entries are live, with padding
    # keys sprinkled among them
    for i in rng.choice(count, count // 50, replace=False):
        keys[i] = 0
    got = sm.stream_launch(keys, count, k, np.random.default_rng(1))
    live = [x for x in keys[:count] if x != 0]
    want = [sm.key_row(x) for x in sorted(live, reverse=True)[:k]]
    want += [-1] * (k - len(want))
    assert got == want


@pytest.mark.parametrize("start,length", [(0, 1), (5, 2), (7, 2), (1023, 3), (4096, 4096),
                                          ((1 << 20) - 5, 8192), ((1 << 31) - 8195, 8192),
                                          ((1 << 31) - 1, 1), (12345, 777)])
def test_score_chunk_statistics_match_the_direct_ones(start, length):
    """The row words' AND / OR of a first-level chunk come from the ends of
    its row range (score_stats asserts them equal to the direct statistics
    of the real keys); chunks that start anywhere, cross carries into high
    bits or hold one or two rows select exactly."""
    rng = np.random.default_rng(start + length)
    s = make_scores(rng, length, "ties")
    keys = sm.pack_keys(s, np.arange(start, start + length))
    per = 16 if length > 4096 else 8
    for k in (1, 8, min(length, 1024)):
        kk = min(k, length)
        out, _ = sm.select_block(keys, kk, 512, per, bound=True, final=True,
                                 rng=np.random.default_rng(k), score_start=start)
        assert out == sorted(keys, reverse=True)[:kk]


def test_detector_flags_a_missing_barrier(monkeypatch):
    """The rank counts' zeroing and their atomic updates in one phase: the
    zeroing thread and the updating threads conflict."""
    real_final = sm.final_output

    def no_barrier_after_zeroing(B, nt, k, rank_max=256):
        orig = B.sync
        calls = {"n": 0}

        def sync():
            calls["n"] += 1
            if calls["n"] != 2:            # drop the barrier after the zeroing
                orig()
        B.sync = sync
        try:
            return real_final(B, nt, k, rank_max)
        finally:
            B.sync = orig
    monkeypatch.setattr(sm, "final_output", no_barrier_after_zeroing)
    s = make_scores(np.random.default_rng(3), 5000, "normal")
    with pytest.raises(sm.Hazard):
        sm.select_launch(s, 64, np.random.default_rng(0))


def test_detector_flags_an_unwritten_digit_record():
    """A pass asked for more keys than match its prefix: no lane writes the
    digit record, and its readers would see stale words."""
    B = sm.Block(512, np.random.default_rng(0))
    for name, n in (("hist", 8 * 256), ("tot", 256), ("info", 4)):
        B.alloc(name, n)
    key = [[(1 << 63) | (t * 16 + e) for e in range(16)] for t in range(512)]
    cs = (8192, (1 << 63), (1 << 63) | 8191, 0, 0)
    with pytest.raises(sm.Hazard):
        sm.radix_select(B, key, 9000, cs, False)
