"""A host model of the selection kernels' barrier phases, for hazard checks.

It executes the block-level algorithm of `select_kernel` (chunk statistics,
radix select, ballot compaction, final ordering by rank or bitonic network)
and `select_stream_kernel`'s rounds, phase by phase: between two barriers the
threads of the block run in a random order, and every shared-memory (LDS)
access is logged with its phase, thread, array and word.  Wave-wide
operations (ballot, cross-lane shuffles, DPP) read registers only and are
evaluated per wave with every lane present, as on the device.

After a launch the log is checked for
  * cross-thread conflicts inside one phase: a word written (or atomically
    updated) by one thread and read or written by another between the same
    two barriers (atomic updates among themselves are fine);
  * stale reads: a word read before anything in this launch wrote it (LDS is
    not cleared between blocks, so such a read sees an earlier block's data);
  * radix passes in which no lane writes the digit record (`s_info`), whose
    readers would then see the previous pass's (or block's) values.

This is a test instrument that mirrors the kernel, not the oracle: its
results are checked against a plain sort, never used as a parity reference.
"""
from __future__ import annotations

import numpy as np

M64 = (1 << 64) - 1


class Hazard(AssertionError):
    pass


class Block:
    """Shared memory of one workgroup plus the access log of the launch."""

    def __init__(self, threads: int, rng: np.random.Generator, poison: int = 0xDEADBEEF):
        self.T = threads
        self.W = threads // 64
        self.rng = rng
        self.phase = 0
        self.lds = {}
        self.written = {}
        self.log = []          # (phase, tid, array, index, kind)
        self.stale = []
        self.poison = poison

    def alloc(self, name: str, n: int):
        # LDS holds whatever the previous block left: poison it
        self.lds[name] = [self.poison] * n
        self.written[name] = [False] * n

    def order(self):
        return [int(t) for t in self.rng.permutation(self.T)]

    def sync(self):
        self.phase += 1

    def rd(self, tid, name, i):
        self.log.append((self.phase, int(tid), name, int(i), "r"))
        if not self.written[name][i]:
            self.stale.append((self.phase, int(tid), name, int(i)))
        return self.lds[name][i]

    def wr(self, tid, name, i, v):
        self.log.append((self.phase, int(tid), name, int(i), "w"))
        self.written[name][i] = True
        self.lds[name][i] = v

    def atomic_add(self, tid, name, i, v):
        self.log.append((self.phase, int(tid), name, int(i), "a"))
        if not self.written[name][i]:
            self.stale.append((self.phase, int(tid), name, int(i)))
        self.lds[name][i] = self.lds[name][i] + v

    def check(self):
        """Raise Hazard on any conflict or stale read of this launch."""
        if self.stale:
            raise Hazard(f"stale LDS reads (phase, thread, array, word): {self.stale[:5]}")
        by_word = {}
        for ph, tid, name, i, kind in self.log:
            by_word.setdefault((ph, name, i), []).append((tid, kind))
        for (ph, name, i), acc in by_word.items():
            writers = {t for t, k in acc if k == "w"}
            atomics = {t for t, k in acc if k == "a"}
            readers = {t for t, k in acc if k == "r"}
            if len(writers) > 1:
                raise Hazard(f"phase {ph}: {name}[{i}] written by threads {sorted(writers)[:4]}")
            if writers and atomics:
                raise Hazard(f"phase {ph}: {name}[{i}] written and atomically updated")
            for w in writers | atomics:
                others = readers - {w}
                if others:
                    raise Hazard(f"phase {ph}: {name}[{i}] written by thread {w}, read by "
                                 f"{sorted(others)[:4]}")


# ------------------------------------------------------------ key helpers

def score_key(s: np.ndarray) -> np.ndarray:
    """Order-preserving uint32 of fp32 scores: NaN -> 0, -0 -> +0."""
    s = np.asarray(s, dtype=np.float32) + np.float32(0.0)
    u = s.view(np.uint32).astype(np.uint64)
    k = np.where(u & 0x80000000, (~u) & 0xFFFFFFFF, u | 0x80000000)
    return np.where(np.isnan(s), 0, k).astype(np.uint64)


def pack_keys(scores: np.ndarray, rows: np.ndarray) -> list:
    sk = score_key(scores)
    return [int((int(a) << 32) | (0xFFFFFFFF - int(r))) for a, r in zip(sk, rows)]


def key_row(k: int) -> int:
    return 0xFFFFFFFF - (k & 0xFFFFFFFF)


def clz32(x: int) -> int:
    return 32 - x.bit_length()


def clz64(x: int) -> int:
    return 64 - x.bit_length()


# --------------------------------------------------------- wave operations

def wave_lanes(T):
    return [list(range(w * 64, w * 64 + 64)) for w in range(T // 64)]


def dpp_max_ladder(vals, g):
    """Group maxima over g consecutive lanes (g a power of two <= 64, or 0)
    and the wave maximum, as the DPP/shuffle ladder forms them."""
    v = list(vals)
    gm = list(vals) if g == 1 else [0] * 64
    size = 1
    while size < 64:
        size *= 2
        v = [max(v[l], v[l ^ (size // 2)]) for l in range(64)]
        if g == size:
            gm = list(v)
    return v, gm


# -------------------------------------------------------------- the phases

def chunk_stats(B: Block, key, kk: int, bound: bool):
    """Per wave: real-key count, AND / OR of real keys, with bound the group
    maxima ladder; lane 0 of each wave writes; barrier; all threads read."""
    T, P = B.T, len(key[0])
    per_wave = []
    for lanes in wave_lanes(T):
        nz = sum(1 for t in lanes for e in range(P) if key[t][e] != 0)
        a, o = M64, 0
        mx = []
        for t in lanes:
            for e in range(P):
                if key[t][e] != 0:
                    a &= key[t][e]
                    o |= key[t][e]
            mx.append(max((key[t][e] >> 32) for e in range(P)))
        lo = hi = 0
        if bound:
            gq = T // (kk if kk > 0 else 1)
            g = 64 if gq >= 64 else ((1 << (31 - clz32(gq))) if gq > 0 else 0)
            v, gm = dpp_max_ladder(mx, g)
            hi = v[0]
            lo = min(gm)
        per_wave.append((nz, a, o, lo, hi))
    for t in B.order():
        if t % 64 == 0:
            w = t // 64
            nz, a, o, lo, hi = per_wave[w]
            B.wr(t, "nzw", w, nz)
            B.wr(t, "andw", w, a)
            B.wr(t, "orw", w, o)
            if bound:
                B.wr(t, "loww", w, lo)
                B.wr(t, "highw", w, hi)
    B.sync()
    res = None
    for t in B.order():
        r = [0, M64, 0, 0xFFFFFFFF, 0]
        for w in range(B.W):
            r[0] += B.rd(t, "nzw", w)
            r[1] &= B.rd(t, "andw", w)
            r[2] |= B.rd(t, "orw", w)
            if bound:
                r[3] = min(r[3], B.rd(t, "loww", w))
                r[4] = max(r[4], B.rd(t, "highw", w))
        if not bound:
            r[3] = r[4] = 0
        assert res is None or res == r, "threads disagree on the chunk statistics"
        res = r
    return res


def score_stats(B: Block, key, kk: int, start: int, n_real: int):
    """chunk_stats with the bound for a chunk of raw scores (rows start ..
    start + n_real - 1): AND / OR over the score words, where a slot past
    the chunk holds a copy of the last real slot's; the row words' AND / OR
    from the two ends of the row range.  Checked against the direct
    statistics of the real keys."""
    T, P = B.T, len(key[0])
    last_word = key[(n_real - 1) % T][(n_real - 1) // T] >> 32
    per_wave = []
    for lanes in wave_lanes(T):
        a, o = 0xFFFFFFFF, 0
        mx = []
        for t in lanes:
            for e in range(P):
                w = (key[t][e] >> 32) if t + e * T < n_real else last_word
                a &= w
                o |= w
            mx.append(max((key[t][e] >> 32) for e in range(P)))
        gq = T // (kk if kk > 0 else 1)
        g = 64 if gq >= 64 else ((1 << (31 - clz32(gq))) if gq > 0 else 0)
        v, gm = dpp_max_ladder(mx, g)
        per_wave.append((0, a << 32, o << 32, min(gm), v[0]))
    for t in B.order():
        if t % 64 == 0:
            w = t // 64
            nz, a, o, lo, hi = per_wave[w]
            B.wr(t, "nzw", w, nz)
            B.wr(t, "andw", w, a)
            B.wr(t, "orw", w, o)
            B.wr(t, "loww", w, lo)
            B.wr(t, "highw", w, hi)
    B.sync()
    res = None
    for t in B.order():
        r = [0, M64, 0, 0xFFFFFFFF, 0]
        for w in range(B.W):
            r[0] += B.rd(t, "nzw", w)
            r[1] &= B.rd(t, "andw", w)
            r[2] |= B.rd(t, "orw", w)
            r[3] = min(r[3], B.rd(t, "loww", w))
            r[4] = max(r[4], B.rd(t, "highw", w))
        first = 0xFFFFFFFF - start
        x = first ^ (0xFFFFFFFF - (start + n_real - 1))
        below = (0xFFFFFFFF >> clz32(x)) if x else 0
        r[0] = n_real
        r[1] |= first & ~below & 0xFFFFFFFF
        r[2] |= first | below
        assert res is None or res == r, "threads disagree on the chunk statistics"
        res = r
    real = [key[t][e] for t in range(T) for e in range(P) if t + e * T < n_real]
    a = o = None
    for x in real:
        a = x if a is None else a & x
        o = x if o is None else o | x
    assert all(x != 0 for x in real) and (res[0], res[1], res[2]) == (len(real), a, o), \
        "score-word statistics differ from the direct ones"
    return res


def radix_select(B: Block, key, need: int, cs, bound: bool):
    T, P, W = B.T, len(key[0]), B.W
    nz, all_and, any_or, low32, high32 = cs
    diff = all_and ^ any_or
    if diff == 0:
        return all_and, M64
    hb = 63 - clz64(diff)
    if bound:
        span = low32 ^ high32
        hs = (63 - clz32(span)) if span else 31
        hb = min(hs, hb)
    mask = (~(((2 << hb) & M64) - 1)) & M64
    prefix = ((((high32 << 32) | (all_and & 0xFFFFFFFF)) if bound else all_and) & mask)
    for t in B.order():
        for b in range(t, W * 256, T):
            B.wr(t, "hist", b, 0)
    B.sync()
    hi = hb
    while hi >= 0:
        lo = hi - 7 if hi >= 7 else 0
        dmask = (1 << (hi - lo + 1)) - 1
        for t in B.order():
            my = (t // 64) * 256
            for e in range(P):
                if (key[t][e] & mask) == prefix:
                    B.atomic_add(t, "hist", my + ((key[t][e] >> lo) & dmask), 1)
        B.sync()
        # wave 0: each lane totals its four digits over the waves'
        # histograms (clearing them), then suffix sums over lanes (registers)
        local = {}
        for t in B.order():
            if t < 64:
                h = []
                for j in range(4):
                    tot = 0
                    for w in range(W):
                        tot += B.rd(t, "hist", w * 256 + 4 * t + j)
                        B.wr(t, "hist", w * 256 + 4 * t + j, 0)
                    h.append(tot)
                local[t] = h
        incl = [sum(sum(local[m]) for m in range(l, 64)) for l in range(64)]
        writers = 0
        for t in B.order():
            if t < 64:
                h = local[t]
                above = incl[t] - sum(h)
                if above < need <= incl[t]:
                    for j in (3, 2, 1, 0):
                        if above + h[j] >= need:
                            B.wr(t, "info", 0, 4 * t + j)
                            B.wr(t, "info", 1, above)
                            B.wr(t, "info", 2, h[j])
                            writers += 1
                            break
                        above += h[j]
        if writers != 1:
            raise Hazard(f"{writers} lanes wrote the digit record in the pass at bit {hi}")
        B.sync()
        got = None
        for t in B.order():
            vals = (B.rd(t, "info", 0), B.rd(t, "info", 1), B.rd(t, "info", 2))
            assert got is None or got == vals
            got = vals
        digit, above, in_bucket = got
        need -= above
        prefix |= digit << lo
        mask |= dmask << lo
        if in_bucket == need:
            break
        hi -= 8
    B.sync()
    return prefix, mask


def compact_taken(B: Block, key, tmask: int, tpre: int, dst, cap: int):
    """Keys with (key & tmask) >= tpre to dst[0 .. min(taken, cap)) by
    ballot prefix sums; dst: ("lds", name) or a Python list (global
    memory)."""
    T, P = B.T, len(key[0])
    tk = [[(key[t][e] & tmask) >= tpre for e in range(P)] for t in range(T)]
    for t in B.order():
        if t % 64 == 0:
            w = t // 64
            B.wr(t, "wc", w, sum(tk[u][e] for u in range(w * 64, w * 64 + 64) for e in range(P)))
    B.sync()
    total = None
    for t in B.order():
        w, lane = t // 64, t % 64
        base = tot = 0
        for v in range(B.W):
            c = B.rd(t, "wc", v)
            base += c if v < w else 0
            tot += c
        total = tot
        for e in range(P):
            m = [tk[u][e] for u in range(w * 64, w * 64 + 64)]
            pos = base + sum(m[:lane])
            if tk[t][e] and pos < cap:
                if isinstance(dst, tuple):
                    B.wr(t, dst[1], pos, key[t][e])
                else:
                    dst[pos] = key[t][e]
            base += sum(m)
    return total


def final_output(B: Block, nt: int, k: int, rank_max: int = 256):
    T = B.T
    p = 1
    while p < nt:
        p <<= 1
    B.sync()
    if p <= rank_max:
        for t in B.order():
            for i in range(t, nt, T):
                B.wr(t, "rank", i, 0)
        B.sync()
        g = T // p
        kis = {}
        for t in B.order():
            i, part = t // g, t % g
            ki = B.rd(t, "sel", i) if i < nt else 0
            kis[t] = ki
            if i < nt:
                c = 0
                for j in range(part, nt, g):
                    kj = B.rd(t, "sel", j)
                    c += (kj > ki) | ((kj == ki) & (j < i))
                if c:
                    B.atomic_add(t, "rank", i, c)
        B.sync()
        for t in B.order():
            i, part = t // g, t % g
            if i < nt and part == 0:
                B.wr(t, "sorted", B.rd(t, "rank", i), kis[t])
            for r in range(nt + t, k, T):
                B.wr(t, "sorted", r, 0)
        src = "sorted"
    else:
        for t in B.order():
            for r in range(nt + t, max(p, k), T):
                B.wr(t, "sel", r, 0)
        B.sync()
        size = 2
        while size <= p:
            stride = size >> 1
            while stride > 0:
                for t in B.order():
                    for i in range(t, p >> 1, T):
                        pos = 2 * i - (i & (stride - 1))
                        partner = pos + stride
                        desc = (pos & size) == 0
                        a, b = B.rd(t, "sel", pos), B.rd(t, "sel", partner)
                        if (a < b) == desc:
                            B.wr(t, "sel", pos, b)
                            B.wr(t, "sel", partner, a)
                B.sync()
                stride >>= 1
            size <<= 1
        src = "sel"
    B.sync()
    out = [None] * k
    for t in B.order():
        for r in range(t, k, T):
            out[r] = B.rd(t, src, r)
    return out


def select_block(keys_in: list, k: int, threads: int, per: int, bound: bool, final: bool,
                 rng: np.random.Generator, score_start=None):
    """One block of select_kernel over one chunk (a list of packed keys, at
    most threads * per; missing slots are padding).  score_start: the chunk
    holds raw scores of rows score_start .. (the score-word statistics).
    Returns (out, block): the kk survivor keys (padded with 0) or, when
    final, the k output keys in order."""
    T, P = threads, per
    CH = T * P
    assert len(keys_in) <= CH
    B = Block(T, rng)
    for name, n in (("nzw", B.W), ("andw", B.W), ("orw", B.W), ("loww", B.W), ("highw", B.W),
                    ("hist", B.W * 256), ("tot", 256), ("info", 4), ("wc", B.W),
                    ("sel", 1024), ("sorted", 1024), ("rank", 256)):
        B.alloc(name, n)
    key = [[keys_in[t + e * T] if t + e * T < len(keys_in) else 0 for e in range(P)]
           for t in range(T)]
    kk = min(k, CH)
    if score_start is not None:
        cs = score_stats(B, key, kk, score_start, len(keys_in))
    else:
        cs = chunk_stats(B, key, kk, bound)
    allk = cs[0] <= kk
    prefix, mask = 1, M64                  # every real key
    if not allk:
        prefix, mask = radix_select(B, key, kk, cs, bound)
    if not final:
        out = [None] * kk
        tot = compact_taken(B, key, mask, prefix, out, kk)
        nt = min(tot, kk)
        for i in range(nt, kk):
            out[i] = 0
        B.check()
        return out, B
    tot = compact_taken(B, key, mask, prefix, ("lds", "sel"), kk)
    nt = min(tot, kk)
    out = final_output(B, nt, k)
    B.check()
    return out, B


def select_launch(scores: np.ndarray, k: int, rng: np.random.Generator, per: int = 16,
                  threads: int = 512):
    """All levels of launch_topk_gather for one query's scores: up to two
    chunks one final block (with the group-maxima bound); more, the first
    level from scores (with the bound), survivor levels, the final level.
    Returns the ordered top-k rows (-1 for padding)."""
    n = len(scores)
    CH = threads * per
    keys = pack_keys(scores, np.arange(n))
    kk = min(k, 8192)
    chunks = -(-n // 8192)
    if chunks <= 2:
        p = 8 if n <= threads * 8 else (per if chunks == 1 else 2 * per)
        out, _ = select_block(keys, k, threads, p, bound=True, final=True, rng=rng,
                              score_start=0)
        return [(-1 if x == 0 else key_row(x)) for x in out]
    level = []
    for c in range(chunks):
        o, _ = select_block(keys[c * 8192:(c + 1) * 8192], k, threads, 16, bound=True,
                            final=False, rng=rng, score_start=c * 8192)
        level += o
    while -(-len(level) // 8192) > 1:
        nxt = []
        for c in range(-(-len(level) // 8192)):
            o, _ = select_block(level[c * 8192:(c + 1) * 8192], k, threads, 16, bound=False,
                                final=False, rng=rng)
            nxt += o
        level = nxt
    p = 8 if len(level) <= threads * 8 else 16
    out, _ = select_block(level, k, threads, p, bound=False, final=True, rng=rng)
    return [(-1 if x == 0 else key_row(x)) for x in out]


def stream_launch(keys_in: list, count: int, k: int, rng: np.random.Generator,
                  threads: int = 1024):
    """select_stream_kernel for one query: rounds over the first `count`
    keys of the buffer, then the final ordering."""
    T = threads
    B = Block(T, rng)
    for name, n in (("nzw", B.W), ("andw", B.W), ("orw", B.W), ("hist", B.W * 256),
                    ("tot", 256), ("info", 4), ("wc", B.W), ("sel", 1024), ("sorted", 1024),
                    ("rank", 256)):
        B.alloc(name, n)
    P = 4 if count <= T * 4 else (8 if count <= T * 8 else 16)
    R = T * P
    kk = k
    nt = 0
    pos = 0
    while True:
        take = min(R - nt, count - pos)
        key = [[0] * P for _ in range(T)]
        for t in B.order():
            for e in range(P):
                i = t + e * T
                j = pos + (i - nt)
                jc = 0 if j < 0 else (j if j < len(keys_in) else len(keys_in) - 1)
                v = keys_in[jc]
                if i < nt:
                    v = B.rd(t, "sel", i)
                elif i - nt >= take:
                    v = 0
                key[t][e] = v
        B.sync()
        cs = chunk_stats(B, key, kk, False)
        allk = cs[0] <= kk
        prefix, mask = 1, M64              # every real key
        if not allk:
            prefix, mask = radix_select(B, key, kk, cs, False)
        tot = compact_taken(B, key, mask, prefix, ("lds", "sel"), kk)
        nt = min(tot, kk)
        pos += take
        B.sync()
        if pos >= count:
            break
    out = final_output(B, nt, k)
    B.check()
    return [(-1 if x == 0 else key_row(x)) for x in out]
