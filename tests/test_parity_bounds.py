"""The retrieval error bounds used by the GPU parity tests (tests/parity.py,
ScoreBound) checked on the CPU against binary32 emulations of each path's
arithmetic: the single-query scan's per-lane FMA chains and 64-lane tree, the
matrix-core scan's hi/lo split of an fp32 query with one fp32 accumulation
per 32-dimension step, and fp32 inverse norms for cosine.  Every emulated
score must lie within its bound of the exact (oracle) score, and the bound
must stay ~1e-5 relative: tight enough that a real scan error of 1e-4 would
not be excused."""
import numpy as np
import pytest

import oracle
from parity import ScoreBound, decode_rows

f32 = np.float32


def to_bits(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round-to-nearest-even to f16/bf16, as raw bits."""
    if dtype == "f16":
        return x.astype(np.float16).view(np.uint16)
    u = x.astype(np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    return r


def make_rows(rng, n, d, dtype):
    cent = rng.normal(0.0, 1.0, (8, d))
    x = cent[rng.integers(0, 8, n)] + rng.normal(0.0, 0.3, (n, d))
    x[:, rng.permutation(d)[:4]] *= 20.0
    return to_bits(x, dtype)


def pairwise_f32(v):
    """Sum the last axis in a binary tree, rounding to binary32 at each add."""
    v = v.astype(f32)
    while v.shape[-1] > 1:
        if v.shape[-1] % 2:
            v = np.concatenate([v, np.zeros(v.shape[:-1] + (1,), f32)], axis=-1)
        v = (v[..., 0::2] + v[..., 1::2]).astype(f32)
    return v[..., 0]


def gemv_emulate(k, q):
    """Per lane l: elements 512c + 8l + j; two FMA chains (even / odd j),
    chains added, then a 64-lane tree.  FMA = exact product + one rounding."""
    n, d = k.shape
    nc = -(-d // 512)
    kp = np.zeros((n, nc * 512))
    kp[:, :d] = k
    qp = np.zeros(nc * 512)
    qp[:d] = q
    kp = kp.reshape(n, nc, 64, 8)
    qp = qp.reshape(nc, 64, 8)
    a0 = np.zeros((n, 64), f32)
    a1 = np.zeros((n, 64), f32)
    for c in range(nc):
        for w in range(4):
            a0 = (a0.astype(np.float64) + kp[:, c, :, 2 * w] * qp[c, :, 2 * w]).astype(f32)
            a1 = (a1.astype(np.float64) + kp[:, c, :, 2 * w + 1] * qp[c, :, 2 * w + 1]).astype(f32)
    return pairwise_f32((a0 + a1).astype(f32))


def mfma_emulate(k, q, kdt, split=True):
    """hi = RN(q), lo = RN(q - hi) in the key type; per 32-dimension step the
    32 exact products are summed and rounded once, then added to the fp32
    accumulator (hi step, then lo step)."""
    n, d = k.shape
    hi = decode_rows(to_bits(q, kdt), kdt)
    lo = decode_rows(to_bits(q - hi, kdt), kdt) if split else np.zeros(d)
    acc = np.zeros(n, f32)
    for s0 in range(0, d, 32):
        sl = slice(s0, min(d, s0 + 32))
        for part in ((hi, lo) if split else (hi,)):
            t = (k[:, sl] * part[sl]).sum(axis=1).astype(f32)
            acc = (acc + t).astype(f32)
    return acc


def cosine_scale(k, q, dot):
    inv_k = (f32(1.0) / np.sqrt(pairwise_f32(k * k))).astype(f32)
    inv_q = (f32(1.0) / np.sqrt(pairwise_f32((q * q)[None, :])[0])).astype(f32)
    return ((dot * inv_k).astype(f32) * inv_q).astype(f32)


@pytest.mark.parametrize("d,kdt", [(1000, "f16"), (4096, "bf16"), (8192, "bf16"),
                                   (5120, "f16")])
@pytest.mark.parametrize("path", ["gemv", "mfma"])
@pytest.mark.parametrize("metric", ["cosine", "ip"])
def test_bound_covers_emulated_path(d, kdt, path, metric):
    rng = np.random.default_rng(d + len(kdt) + len(path) + len(metric))
    n = 200
    kb = make_rows(rng, n, d, kdt)
    k = decode_rows(kb, kdt)
    q = (k[3] + rng.normal(0.0, 0.05, d)).astype(f32).astype(np.float64)
    exact = oracle.scores(kb, kdt, q.astype(np.float32)[None, :], "f32", metric=metric)[0]
    dot = gemv_emulate(k, q) if path == "gemv" else mfma_emulate(k, q, kdt)
    got = cosine_scale(k, q, dot) if metric == "cosine" else dot
    b = ScoreBound(kb, kdt, q, metric, path)(np.arange(n))
    err = np.abs(got.astype(np.float64) - exact)
    assert (err <= b).all(), f"row {np.argmax(err > b)}: error {err.max():.3g} beyond bound"
    # tight: for the rows that compete for the top (similar rows), ~1e-5
    top = np.argsort(-exact)[:20]
    rel = b[top] / np.abs(exact[top])
    assert rel.max() < (1.2e-4 if path == "mfma" else 4e-5), rel.max()


def test_bound_rejects_a_real_error():
    """A scan that loses the lo half of the query (bf16 query precision) has
    errors of ~1e-4 relative on the top rows: the bound must not excuse it."""
    rng = np.random.default_rng(7)
    d, kdt, n = 4096, "bf16", 200
    kb = make_rows(rng, n, d, kdt)
    k = decode_rows(kb, kdt)
    q = (k[5] + rng.normal(0.0, 0.05, d)).astype(f32).astype(np.float64)
    exact = oracle.scores(kb, kdt, q.astype(np.float32)[None, :], "f32", metric="cosine")[0]
    got = cosine_scale(k, q, mfma_emulate(k, q, kdt, split=False))
    b = ScoreBound(kb, kdt, q, "cosine", "mfma")(np.arange(n))
    assert (np.abs(got - exact) > b).any()


# The batched search over large stores ranks by a fp32 rescore of a band
# chosen with hi-only matrix-core scores; query_split_kernel's margin
# (restated below; inner product through the store's largest key norm) must
# bound |hi-only score - rescore| twice over, also for rows built to make the
# hi half's error as large as Cauchy-Schwarz allows.

def rescore_emulate(k, q):
    """rescore_kernel's sum: lane l takes the 8-element units l, l + 64, ...;
    units l + 128 i go to chain 0 and l + 64 + 128 i to chain 1 (element
    order inside a unit, one FMA each), chains added, 64-lane butterfly."""
    n, d = k.shape
    nu = d // 8
    nup = -(-nu // 128) * 128
    kp = np.zeros((n, nup * 8))
    kp[:, :d] = k
    qp = np.zeros(nup * 8)
    qp[:d] = q
    kp = kp.reshape(n, nup // 128, 2, 64, 8)      # [row, i, chain, lane, element]
    qp = qp.reshape(nup // 128, 2, 64, 8)
    acc = np.zeros((n, 2, 64), f32)
    for i in range(nup // 128):
        for e in range(8):
            acc = (acc.astype(np.float64) + kp[:, i, :, :, e] * qp[i, :, :, e]).astype(f32)
    a = (acc[:, 0] + acc[:, 1]).astype(f32)
    for off in (32, 16, 8, 4, 2, 1):                # butterfly: lane l adds lane l ^ off
        a = (a + a[:, np.arange(64) ^ off]).astype(f32)
    return a[:, 0]


def kernel_margin(q, kdt, d, kmax=None):
    """Cosine (kmax None), or inner product with the store's largest key norm."""
    hi = decode_rows(to_bits(q, kdt), kdt)
    ll = f32(((q - hi) ** 2).sum())
    ss = f32((q * q).sum())
    inv_q = f32(1.0) / np.sqrt(ss)
    depth = (-(-d // 32) + 8) + (d // 128 + 8) + 2 * (d // 64 + 16) + 4
    rnd = depth * 2.0 ** -24
    if kmax is None:
        return 2.0 * (1.01 * float(np.sqrt(ll)) * float(inv_q) + 2.0 * 1.01 * rnd)
    return 2.0 * (1.01 * float(np.sqrt(ll)) + 2.0 * 1.01 * rnd * float(np.sqrt(ss))) * (
        1.001 * float(f32(kmax)))


@pytest.mark.parametrize("metric", ["cosine", "ip"])
@pytest.mark.parametrize("d,kdt", [(128, "bf16"), (1000, "f16"), (4096, "bf16"),
                                   (5120, "f16"), (8192, "bf16")])
def test_batched_margin_bounds_hi_only_against_rescore(d, kdt, metric):
    rng = np.random.default_rng(d * 3 + len(kdt))
    kb = make_rows(rng, 120, d, kdt)
    k = decode_rows(kb, kdt)
    q = (k[7] + rng.normal(0.0, 0.05, d)).astype(f32).astype(np.float64)
    lo = q - decode_rows(to_bits(q, kdt), kdt)
    qn, lon = np.linalg.norm(q), np.linalg.norm(lo)
    # rows along q with the hi half's error direction mixed in, and rows along
    # that direction alone: |sum (q - hi) k| / (|q| |k|) reaches |q - hi| / |q|
    adv = [q + a * lo / lon * qn for a in (0.003, 0.03, 0.3, 1.0)]
    adv += [lo / lon * s for s in (1.0, 1e3)]
    adv += [np.sign(lo) * np.abs(k[j]) for j in range(4)]
    kb = np.concatenate([kb, to_bits(np.array(adv), kdt)])
    k = decode_rows(kb, kdt)
    a = mfma_emulate(k, q, kdt, split=False)
    r = rescore_emulate(k, q)
    if metric == "cosine":
        a, r = cosine_scale(k, q, a), cosine_scale(k, q, r)
        m = kernel_margin(q, kdt, d)
    else:
        # the index's largest key norm: fp32 sums of squares, rounded sqrt
        m = kernel_margin(q, kdt, d, kmax=np.sqrt(pairwise_f32(k * k)).astype(f32).max())
    a, r = a.astype(np.float64), r.astype(np.float64)
    gap = np.abs(a - r)
    assert (gap <= m / 2).all(), f"row {np.argmax(gap > m / 2)}: |A - R| {gap.max():.3g} > {m / 2:.3g}"
    # the adversarial rows use a large part of the allowance: the margin is
    # not loose by orders of magnitude (a band that holds the whole store)
    assert gap[-len(adv):].max() > 0.25 * (m / 2), (gap[-len(adv):].max(), m)
    # and the rescore is the single-query scan's accuracy
    exact = oracle.scores(kb, kdt, q.astype(np.float32)[None, :], "f32", metric=metric)[0]
    b = ScoreBound(kb, kdt, q, metric, "gemv")(np.arange(k.shape[0]))
    assert (np.abs(r - exact) <= b).all()
