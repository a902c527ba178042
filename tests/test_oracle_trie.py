"""Pins for the loose-trie oracle (Sec. 3.2 Eq. 9; Alg. 2 LexSort; Alg. 3;
the static-KV mask of the appendix; Sec. 3.2 Eq. 11): a hand-worked example
(with a ragged variant), a brute-force canonical trie on random drafts with
heavy prefix sharing, Eq. 9's flattening read literally (first sorted draft,
then every next draft past its LCP with the previous one), and the
equivalence of verification through Gamma with verification of dense rows
that are equal wherever two drafts share a prefix."""
import json
import os

import numpy as np
import pytest

import oracle
from oracle import trie

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def golden():
    return json.load(open(os.path.join(GOLDEN, "loose_trie_example.json")))


def test_hand_worked_example():
    g = golden()
    D = np.array(g["drafts"])
    order = trie.lexsort_candidates(D)
    assert order.tolist() == g["order"]
    T, gamma, mask = trie.loose_trie(D[order])
    assert T.tolist() == g["tree_tokens"]
    assert gamma.tolist() == g["gamma"]
    parent, depth, cand = trie.node_table(gamma)
    assert parent.tolist() == g["parent"]
    assert depth.tolist() == g["depth"]
    for u, anc in enumerate(g["ancestors"]):
        assert np.flatnonzero(mask[u]).tolist() == anc
    fm = trie.full_mask(mask, g["prefix_len"], g["cache_len"])
    want = [0.0 if x == "0" else -np.inf for x in g["full_mask_row_6"]]
    assert fm[6].tolist() == want


def test_hand_worked_ragged_example():
    r = golden()["ragged"]
    D, lens = np.array(r["drafts"]), np.array(r["len"])
    order = trie.lexsort_candidates(D, lens)
    assert order.tolist() == r["order"]
    T, gamma, _ = trie.loose_trie(D[order], lens[order])
    assert T.tolist() == r["tree_tokens"]
    assert gamma.tolist() == r["gamma"]


def random_drafts(rng, n, m, vocab, ragged=True):
    D = rng.integers(0, vocab, (n, m))
    # heavy sharing: copy a prefix of another draft into most drafts
    for i in range(n):
        if rng.random() < 0.7 and i > 0:
            src = rng.integers(0, i)
            cut = rng.integers(0, m + 1)
            D[i, :cut] = D[src, :cut]
    lens = rng.integers(0, m + 1, n) if ragged else np.full(n, m)
    return D, lens


@pytest.mark.parametrize("seed", range(12))
def test_matches_brute_force_canonical_trie(seed):
    rng = np.random.default_rng(seed)
    n, m = int(rng.integers(1, 40)), int(rng.integers(1, 9))
    D, lens = random_drafts(rng, n, m, vocab=int(rng.integers(2, 6)), ragged=seed % 2 == 0)
    order = trie.lexsort_candidates(D, lens)
    T, gamma, mask = trie.loose_trie(D[order], lens[order])
    T2, gamma2, mask2 = trie.canonical_trie(D[order], lens[order])
    assert np.array_equal(T, T2)
    assert np.array_equal(gamma, gamma2)
    assert np.array_equal(mask, mask2)
    # node count = number of distinct non-empty prefixes
    prefixes = {tuple(D[i, :j + 1]) for i in range(n) for j in range(lens[i])}
    assert T.shape[0] == len(prefixes)


@pytest.mark.parametrize("seed", range(6))
def test_flattening_is_eq9_concatenation(seed):
    """T_flat = s_pi(1) followed by s_pi(j)[l_j:], l_j the LCP with the
    previous sorted draft (full-length drafts, as in the equation)."""
    rng = np.random.default_rng(100 + seed)
    D, _ = random_drafts(rng, 25, 6, vocab=3, ragged=False)
    S = D[trie.lexsort_candidates(D)]
    T, _, _ = trie.loose_trie(S)
    parts = [S[0]]
    for j in range(1, S.shape[0]):
        lcp = 0
        while lcp < S.shape[1] and S[j, lcp] == S[j - 1, lcp]:
            lcp += 1
        parts.append(S[j, lcp:])
    assert np.array_equal(T, np.concatenate(parts))


def test_lexsort_is_sequence_order():
    D = np.array([[3, 1], [2, 9], [3, 0], [2, 9], [-5, 4]])
    lens = np.array([2, 1, 2, 2, 2])
    # sequences: (3,1), (2,), (3,0), (2,9), (-5,4)
    assert trie.lexsort_candidates(D, lens).tolist() == [4, 1, 3, 2, 0]


def test_verify_through_gamma_equals_dense_rows_with_shared_prefixes():
    """Drafts that share a prefix see the same context, so a model gives
    them the same distribution: a dense C x M x V tensor built that way (one
    random row per distinct prefix, by dictionary) must verify exactly like
    the flat tree rows read through Gamma."""
    rng = np.random.default_rng(7)
    n, m, vocab = 24, 6, 40
    D, lens = random_drafts(rng, n, m, vocab=4)
    lens = np.maximum(lens, 1)
    order = trie.lexsort_candidates(D, lens)
    S, SL = D[order].astype(np.int32), lens[order].astype(np.int32)
    T, gamma, _ = trie.loose_trie(S, SL)
    rows_by_prefix = {}

    def row_for(prefix):
        if prefix not in rows_by_prefix:
            rows_by_prefix[prefix] = rng.normal(0, 2, vocab).astype(np.float32)
        return rows_by_prefix[prefix]
    dense = np.zeros((n, m, vocab), dtype=np.float32)
    for c in range(n):
        for j in range(m):
            dense[c, j] = row_for(tuple(S[c, :j].tolist()))   # context before token j
    flat = np.zeros((1 + T.shape[0], vocab), dtype=np.float32)
    flat[0] = row_for(())
    parent, depth, cand = trie.node_table(gamma)
    for u in range(T.shape[0]):
        flat[1 + u] = row_for(tuple(S[cand[u], :depth[u] + 1].tolist()))
    via = trie.aligned_logits(flat, gamma)
    a = oracle.soft_gate_verify(dense, "f32", S, SL, gamma=0.3, topk=2, window=2)
    b = oracle.soft_gate_verify(via, "f32", S, SL, gamma=0.3, topk=2, window=2)
    for key in ("accept_len", "best", "masks", "rank"):
        assert np.array_equal(a[key], b[key]), key
    assert np.array_equal(a["gate_score"], b["gate_score"])
