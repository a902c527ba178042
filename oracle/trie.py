"""Loose-trie oracle (Sec. 3.2 Eq. 9 and the tree mask after it; Alg. 2's
LexSort step; Alg. 3; the static-KV tree mask of App. "Tree Attention Mask
for Static KV Cache"; Sec. 3.2 Eq. 11's aligned logits).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: imported by the test
suite, ``__graft_entry__.smoke()`` and the benchmark's ``cpu_baseline`` leg,
never by the HIP library.  Plain numpy, written from the algorithm's steps in
the paper's order; no blocking or fusion.

Readings (the same on the HIP side):
  * Drafts have lengths.  Position j of candidate i exists when j < len_i;
    a position that does not exist matches nothing, is no tree node, and its
    entry of Gamma is -1.  With every length equal to M this is Alg. 3
    literally.
  * LexSort is the lexicographic order of the token sequences (a proper
    prefix sorts first), ties (identical drafts) by original index.
  * Tree node u's logits row: the tree forward gives one row per node (the
    distribution after that node); the aligned rows of candidate c are
    [p_{t-1}; P[Gamma[c, 0]]; ...], so token j of c is judged by p_{t-1} for
    j = 0 and by P[Gamma[c, j-1]] otherwise.  A flat logits array holds
    p_{t-1} in row 0 and P[u] in row 1 + u.
"""
from __future__ import annotations

import numpy as np


def _lengths(drafts, draft_len):
    n, m = drafts.shape
    if draft_len is None:
        return np.full(n, m, dtype=np.int64)
    return np.clip(np.asarray(draft_len, dtype=np.int64), 0, m)


def lexsort_candidates(drafts, draft_len=None) -> np.ndarray:
    """Alg. 2's LexSort: the permutation pi listing candidates in
    lexicographic order of their token sequences (ties by index)."""
    drafts = np.asarray(drafts, dtype=np.int64)
    lens = _lengths(drafts, draft_len)
    seqs = [tuple(int(t) for t in drafts[i, :lens[i]]) for i in range(drafts.shape[0])]
    return np.array(sorted(range(len(seqs)), key=lambda i: (seqs[i], i)), dtype=np.int64)


def loose_trie(sorted_drafts, sorted_len=None):
    """Alg. 3 on lexicographically sorted candidates D (N x M).

    Returns (T, Gamma, mask): T the flattened tree tokens (L,), Gamma (N, M)
    the tree position of every existing (candidate, position) (-1 where the
    position does not exist), mask (L, L) uint8 with mask[Gamma[i, a],
    Gamma[i, b]] = 1 for b <= a on every candidate's path."""
    D = np.asarray(sorted_drafts, dtype=np.int64)
    n, m = D.shape
    lens = _lengths(D, sorted_len)
    exists = np.arange(m)[None, :] < lens[:, None]
    # Prefix detection: position j of row i repeats row i-1 at j, and so do
    # all positions before it (cumulative product along the row).
    match = np.zeros((n, m), dtype=np.int64)
    match[1:] = (D[1:] == D[:-1]) & exists[1:] & exists[:-1]
    is_prefix = np.cumprod(match, axis=1).astype(bool)
    unique = ~is_prefix & exists
    # Tree extraction in row-major order.
    T = D[unique]
    # Index mapping: running count of unique positions; shared positions
    # take the latest unique index above them in their column (cummax down
    # the rows).
    idx = np.cumsum(unique.ravel()) - 1
    gamma = idx.reshape(n, m)
    tmp = np.where(unique, gamma, -1)
    gamma = np.maximum.accumulate(tmp, axis=0)
    gamma = np.where(exists, gamma, -1)
    # Attention mask: along each candidate path, later positions see earlier
    # ones (lower-triangular index pairs).
    L = T.shape[0]
    mask = np.zeros((L, L), dtype=np.uint8)
    I, J = np.tril_indices(m)
    for i in range(n):
        ok = (I < lens[i]) & (J < lens[i])
        mask[gamma[i, I[ok]], gamma[i, J[ok]]] = 1
    return T, gamma, mask


def node_table(gamma, sorted_len=None):
    """Inverse map of Gamma: for every node u its parent (-1 at depth 0), its
    depth and the first sorted candidate whose path creates it."""
    gamma = np.asarray(gamma, dtype=np.int64)
    n, m = gamma.shape
    L = int(gamma.max()) + 1 if gamma.size and gamma.max() >= 0 else 0
    parent = np.full(L, -1, dtype=np.int64)
    depth = np.full(L, -1, dtype=np.int64)
    cand = np.full(L, -1, dtype=np.int64)
    for i in range(n):
        for j in range(m):
            u = gamma[i, j]
            if u >= 0 and cand[u] < 0:
                cand[u] = i
                depth[u] = j
                parent[u] = gamma[i, j - 1] if j > 0 else -1
    return parent, depth, cand


def full_mask(mask, prefix_len: int, cache_len: int) -> np.ndarray:
    """The static-KV mask (App.): row i of the L tree tokens sees every
    cached position j < m and tree position j - m when mask[i, j - m] = 1;
    everything else is -inf.  float64 (L x cache_len)."""
    L = mask.shape[0]
    out = np.full((L, cache_len), -np.inf)
    out[:, :min(prefix_len, cache_len)] = 0.0
    cols = np.arange(prefix_len, min(prefix_len + L, cache_len))
    block = out[:, cols]
    block[mask[:, cols - prefix_len] == 1] = 0.0
    out[:, cols] = block
    return out


def aligned_logits(flat_rows, gamma):
    """Gamma applied to the flattened logits (Sec. 3.2 Eq. 11): for every
    candidate c and position j the row judging token j, i.e. flat row 0 for
    j = 0 and flat row 1 + Gamma[c, j-1] otherwise.  Positions whose
    predecessor does not exist get row 0 (they are past the draft and never
    read).  Returns an (N, M, V) array."""
    gamma = np.asarray(gamma, dtype=np.int64)
    n, m = gamma.shape
    rows = np.zeros((n, m), dtype=np.int64)
    prev = gamma[:, :-1]
    rows[:, 1:] = np.where(prev >= 0, prev + 1, 0)
    return np.asarray(flat_rows)[rows]


def canonical_trie(sorted_drafts, sorted_len=None):
    """Brute-force trie for cross-checking: insert the sorted sequences one
    by one, numbering a prefix the first time it is seen.  Returns (T,
    Gamma, mask) in the same conventions as loose_trie."""
    D = np.asarray(sorted_drafts, dtype=np.int64)
    n, m = D.shape
    lens = _lengths(D, sorted_len)
    ids = {}
    tokens = []
    gamma = np.full((n, m), -1, dtype=np.int64)
    for i in range(n):
        for j in range(lens[i]):
            key = tuple(D[i, :j + 1].tolist())
            if key not in ids:
                ids[key] = len(tokens)
                tokens.append(int(D[i, j]))
            gamma[i, j] = ids[key]
    L = len(tokens)
    prefix_of = {v: k for k, v in ids.items()}
    mask = np.zeros((L, L), dtype=np.uint8)
    for u in range(L):
        pu = prefix_of[u]
        for v in range(L):
            pv = prefix_of[v]
            mask[u, v] = 1 if pu[:len(pv)] == pv else 0
    return np.array(tokens, dtype=np.int64), gamma, mask
