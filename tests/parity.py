"""Parity rules between the HIP path and the oracle (shared by the GPU tests).

Retrieval.  Each path's scores carry a rounding error that its arithmetic
bounds (ScoreBound: fp32 accumulation over the kernel's summation tree, the
hi/lo split of an fp32 query on the matrix cores, the fp32 norms of cosine).
The ordered top-k ids must equal the oracle's, except that the entry at a
rank may differ from the oracle's where the two rows' oracle scores lie
within the sum of their bounds (an exact-arithmetic near tie); at the k/k+1
boundary an id may differ only within the same allowance of the oracle's
k-th score.  Every returned score must lie within its bound of the oracle's.
The bounds are ~1e-5 relative, far inside the 1e-3 the method's contract
allows; callers without a bound (approximate and projected paths) keep the
1e-3 rule.  Drafts must match exactly for every id.
Verification: ranks, exact-match and top-k bits exactly; gate scores within
GATE_ABS; the entropy bit and the accepted length exactly unless a gate score
lies within GATE_ABS of gamma.
"""
import math

import numpy as np
import torch

import oracle

REL_TIE = 1e-3
REL_SCORE = 1e-3
GATE_ABS = 1e-4
U32 = 2.0 ** -24        # binary32 unit roundoff
SAFETY = 2.0            # over the first-order bounds below


def host_bits(t: torch.Tensor) -> np.ndarray:
    """Raw uint16 bit patterns (f16/bf16) or float32 array of a device tensor."""
    t = t.detach().cpu().contiguous()
    if t.dtype in (torch.float16, torch.bfloat16):
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def dt_name(t: torch.Tensor) -> str:
    return {torch.float32: "f32", torch.float16: "f16", torch.bfloat16: "bf16"}[t.dtype]


def decode_rows(bits: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of raw f16/bf16 bit patterns (or f32 values)."""
    bits = np.ascontiguousarray(bits)
    if dtype == "bf16":
        return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    if dtype == "f16":
        return bits.view(np.float16).astype(np.float64)
    return bits.astype(np.float64)


class ScoreBound:
    """Bound on |GPU score - exact score| for the rows of one query.

    The exact score is s = scale * sum_t q_t K_t (scale = 1/(|q| |K|) for
    cosine, 1 for inner product).  With A = scale * sum_t |q_t K_t|:

      |error| <= SAFETY * ((acc * u + split) * A + norm * u * |s|) + tiny

    where u = 2^-24 and, per path,
      gemv:  each lane runs two fp32 FMA chains of d/128 products, the chains
             are added and the wave sums 64 partials in a 6-level tree:
             acc = d/128 + 8;
      mfma:  the matrix core adds 32 exact products per instruction into an
             fp32 accumulator (taken as a 6-level adder tree), one chain of
             ceil(d/32) instructions per query half: acc = halves*ceil(d/32)+8;
             an fp32 query split into hi + lo in the key type leaves
             |q - hi - lo| <= 2^-16 |q| (bf16) or 2^-22 |q| (f16), and for
             f16 a subnormal lo adds at most 2^-25 per element (tiny);
      short: d <= 64 products in any fp32 order: acc = d + 8.
    Cosine scales by fp32 inverse norms, each a blocked fp32 sum of squares,
    a square root and a reciprocal: norm = d/64 + 16 (zero for inner product).
    """

    def __init__(self, keys_bits, key_dtype: str, q_row, metric: str, path: str,
                 q_in_key_type: bool = False):
        self.keys = keys_bits                    # n x ld raw bits (array-like over rows)
        self.kdt = key_dtype
        self.q = np.asarray(q_row, dtype=np.float64)
        self.d = self.q.shape[0]
        self.cos = metric == "cosine"
        d = self.d
        if path == "gemv":
            acc, split = d / 128 + 8, 0.0
        elif path == "mfma":
            halves = 1 if q_in_key_type else 2
            acc = halves * math.ceil(d / 32) + 8
            split = 0.0 if q_in_key_type else (2.0 ** -16 if key_dtype == "bf16" else 2.0 ** -22)
        elif path == "short":
            acc, split = d + 8, 0.0
        else:
            raise ValueError(path)
        self.coef_a = SAFETY * (acc * U32 + split)
        self.coef_s = SAFETY * (d / 64 + 16) * U32 if self.cos else 0.0
        self.f16_split = key_dtype == "f16" and split > 0
        self.qn = float(np.sqrt((self.q * self.q).sum()))
        self.cache = {}

    def __call__(self, rows) -> np.ndarray:
        rows = np.asarray(rows, dtype=np.int64).ravel()
        need = sorted(set(rows.tolist()) - set(self.cache))
        if need:
            kb = np.asarray(self.keys[need])[:, :self.d]
            k = decode_rows(kb, self.kdt)
            s = k @ self.q
            a = np.abs(k) @ np.abs(self.q)
            l1 = np.abs(k).sum(axis=1)
            if self.cos:
                kn = np.sqrt((k * k).sum(axis=1))
                scale = np.where((kn > 0) & (self.qn > 0), 1.0 / np.maximum(kn * self.qn, 1e-300),
                                 0.0)
            else:
                scale = np.ones(len(need))
            b = self.coef_a * a * scale + self.coef_s * np.abs(s * scale) + 1e-30
            if self.f16_split:
                b = b + SAFETY * 2.0 ** -25 * l1 * scale
            for i, r in enumerate(need):
                self.cache[r] = float(b[i])
        return np.array([self.cache[int(r)] for r in rows])


# Stores of more than this many rows are searched in batches through a
# sampled threshold; for long keys the returned scores are then fp32
# rescores of the band around the k-th (the single-query scan's arithmetic).
BATCH_DIRECT_MAX = 131072


def retrieval_path(n_queries: int, d: int, n: int = 0, metric: str = "cosine") -> str:
    """The arithmetic of the scores sense_retrieve returns for a static index:
    single queries from the vector ALUs (the short-row scan for d <= 64),
    batches of two or more from the matrix cores, except batches of long keys
    over more than BATCH_DIRECT_MAX rows, whose returned scores are fp32
    rescores (the single-query scan's sum order).  (metric: either; kept for
    callers that name it.)"""
    if n_queries >= 2:
        if d > 64 and n > BATCH_DIRECT_MAX:
            return "gemv"
        return "mfma"
    return "short" if d <= 64 else "gemv"


def _rows_of(keys_rows) -> int:
    t = keys_rows.t if isinstance(keys_rows, DeviceRows) else keys_rows
    return int(t.shape[0])


def query_bounds(keys_rows, key_dtype: str, queries, metric: str, q_in_key_type: bool = False):
    """One ScoreBound per query row of `queries` (float64-convertible array,
    Q x d) for the path sense_retrieve takes with this batch over the rows
    of keys_rows (the whole store)."""
    q = np.asarray(queries, dtype=np.float64)
    path = retrieval_path(q.shape[0], q.shape[1], _rows_of(keys_rows), metric)
    return [ScoreBound(keys_rows, key_dtype, q[i], metric, path, q_in_key_type)
            for i in range(q.shape[0])]


class DeviceRows:
    """Row access to a device store for ScoreBound: rows[list] -> host bits."""

    def __init__(self, t: torch.Tensor):
        self.t = t

    def __getitem__(self, rows):
        idx = torch.as_tensor(np.asarray(rows, dtype=np.int64), device=self.t.device)
        return host_bits(self.t[idx])


def check_topk(g_ids, g_scores, o_scores_row, k, bound=None):
    """g_ids/g_scores: one query's GPU results; o_scores_row: oracle scores of
    every row; bound: a ScoreBound for this query (None: the 1e-3 rule).
    Returns the number of ranks whose id differs from the oracle's (each an
    excused near tie)."""
    g_ids = np.asarray(g_ids, dtype=np.int64)
    o_ids, o_sc = oracle.topk(o_scores_row, k)
    assert len(set(g_ids.tolist())) == k, "duplicate ids"
    assert g_ids.min() >= 0 and g_ids.max() < o_scores_row.shape[0], "id out of range"
    s_of = o_scores_row[g_ids]
    g = np.asarray(g_scores, dtype=np.float64)
    if bound is None:
        tol_g = REL_TIE * np.abs(s_of)
        tol_o = REL_TIE * np.abs(o_sc)
        np.testing.assert_allclose(g, s_of, rtol=REL_SCORE,
                                   atol=REL_SCORE * max(1e-30, float(np.abs(o_sc).max())) * 1e-3)
    else:
        tol_g = bound(g_ids)
        tol_o = bound(o_ids)
        err = np.abs(g - s_of)
        bad = np.nonzero(~(err <= tol_g))[0]
        assert bad.size == 0, (
            f"{bad.size} scores outside their bound; first at rank {bad[0]}: gpu {g[bad[0]]!r} "
            f"oracle {s_of[bad[0]]!r} bound {tol_g[bad[0]]:.3g}")
        np.testing.assert_allclose(g, s_of, rtol=REL_SCORE, atol=1e-30)
    diff = np.nonzero(g_ids != o_ids)[0]
    for r in diff:
        gap = abs(s_of[r] - o_sc[r])
        assert gap <= tol_g[r] + tol_o[r], (
            f"rank {r}: gpu id {g_ids[r]} (oracle score {s_of[r]!r}) vs oracle id {o_ids[r]} "
            f"({o_sc[r]!r}): gap {gap:.3g} beyond the allowance {tol_g[r] + tol_o[r]:.3g} "
            f"({diff.size} ranks differ)")
    outside = set(g_ids.tolist()) - set(o_ids.tolist())
    sk, tk = o_sc[k - 1], tol_o[k - 1]
    pos = {int(i): r for r, i in enumerate(g_ids.tolist())}
    for i in outside:
        assert o_scores_row[i] >= sk - tk - tol_g[pos[i]], (
            f"id {i} (oracle score {o_scores_row[i]!r}) is not a near tie of the k-th "
            f"({sk!r}); {len(outside)} ids outside the oracle's top {k}")
    return int(diff.size)


def check_verify(gpu: dict, ref: dict, gamma: float, draft_len=None):
    """Compare a GPU verify result (device tensors) with the oracle's dict."""
    acc = gpu["accept_len"].cpu().numpy()
    c, m = ref["masks"].shape
    lens = np.full(c, m) if draft_len is None else np.clip(np.asarray(draft_len), 0, m)
    gs = gpu["gate_score"].cpu().numpy().astype(np.float64) if "gate_score" in gpu else None
    if gs is not None:
        np.testing.assert_allclose(gs, ref["gate_score"], rtol=0, atol=GATE_ABS)
    near = np.abs(ref["gate_score"] - gamma) <= GATE_ABS
    for cc in range(c):
        near[cc, lens[cc]:] = False
    if "rank" in gpu:
        assert np.array_equal(gpu["rank"].cpu().numpy(), ref["rank"]), "ranks differ"
    masks = gpu["masks"].cpu().numpy() if "masks" in gpu else None
    if masks is not None:
        # em (1), topk (4), con depends on em only (8): exact everywhere
        assert np.array_equal(masks & 0b1101, ref["masks"] & 0b1101), "em/topk/con bits differ"
        ent_diff = (masks & 2) != (ref["masks"] & 2)
        assert not (ent_diff & ~near).any(), "entropy gate differs away from gamma"
    excused = np.zeros(c, dtype=bool)
    for cc in range(c):
        if near[cc, : min(ref["accept_len"][cc] + 1, lens[cc])].any():
            excused[cc] = True
    assert np.array_equal(acc[~excused], ref["accept_len"][~excused]), "accept_len differs"
    best = gpu["best"].cpu().numpy()
    n_groups = best.shape[0]
    gsz = c // max(n_groups, 1)
    for g in range(n_groups):
        grp = slice(g * gsz, (g + 1) * gsz)
        if not excused[grp].any():
            assert best[g] == ref["best"][g], f"best of group {g}"
    return int(excused.sum()), int(near.sum())
