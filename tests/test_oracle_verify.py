"""Pins for the soft-gated evaluation half of the oracle (Alg. 4, Sec. 3.3).

The oracle is checked against closed forms (entropy of uniform and two-valued
distributions), the hand-worked look-ahead window fixture, special cases that
reduce the gate to textbook rules (gamma >= 1 gives plain greedy verification;
k = 1 makes top-k membership equal to exact match; k >= V makes it always
true; W >= M disables the window), hand-ranked ties, and the monotonicity
invariants of the definition over the paper's hyper-parameter grid
(gamma in {0.01, 0.05, 0.10, 0.30}, k in {2, 3, 4, 10}, W in {5..9}).
"""
import json
import math
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
EM, ENT, TOPK, CON, G = 1, 2, 4, 8, 16


def test_uniform_row_entropy_is_log_v_and_rank_is_index():
    v = 1000
    row = np.zeros(v, dtype=np.float32)
    y, e, r = oracle.row_stats(row, "f32", 437)
    assert y == 0 and r == 437
    assert abs(e - math.log(v)) < 1e-12
    out = oracle.soft_gate_verify(row.reshape(1, 1, v), "f32", np.array([[437]], np.int32))
    assert abs(out["gate_score"][0, 0] - 1.0) < 1e-13


@pytest.mark.parametrize("a", [0.5, 3.7, 20.0, 50.0])
def test_two_valued_row_closed_form(a):
    v, i0, b = 5000, 123, -1.25
    row = np.full(v, b, dtype=np.float32)
    row[i0] = a
    a = float(row[i0])                      # the value actually stored (float32)
    # p1 = 1/(1+r), p0 = e^(b-a)/(1+r) with r = (V-1) e^(b-a); then
    # -p1 ln p1 - (V-1) p0 ln p0 simplifies to log1p(r) + r (a-b) / (1+r)
    r = (v - 1) * math.exp(b - a)
    ent = math.log1p(r) + r * (a - b) / (1.0 + r)
    y, e, r = oracle.row_stats(row, "f32", i0)
    assert y == i0 and r == 0
    assert abs(e - ent) <= 1e-12 * max(1.0, ent)
    # every other token: one larger value ahead, ties broken by index
    for t in (0, 122, 124, v - 1):
        _, _, rt = oracle.row_stats(row, "f32", t)
        assert rt == (t + 1 if t < i0 else t)


def test_hand_ranked_ties():
    row = np.array([1.0, 3.0, 3.0, 2.0, 3.0], dtype=np.float32)
    # rank(d) = #{x_v > x_d} + #{v < d : x_v = x_d}
    expect = {0: 4, 1: 0, 2: 1, 3: 3, 4: 2}
    for tok, r in expect.items():
        y, _, got = oracle.row_stats(row, "f32", tok)
        assert y == 1 and got == r


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_half_precision_rows_decode_exactly(dt):
    rng = np.random.default_rng(1)
    ints = rng.integers(-8, 9, size=(4, 3, 257)).astype(np.float32) * 0.5  # exact in both
    bits = (ints.astype(np.float16).view(np.uint16) if dt == "f16"
            else (ints.view(np.uint32) >> 16).astype(np.uint16))
    drafts = rng.integers(0, 257, size=(4, 3)).astype(np.int32)
    a = oracle.soft_gate_verify(ints, "f32", drafts, n_groups=2)
    b = oracle.soft_gate_verify(bits, dt, drafts, n_groups=2)
    for key in a:
        assert np.array_equal(a[key], b[key]), key


def _row_exact(v, tok):
    """Low-entropy row whose argmax is tok (E_n ~ 0)."""
    row = np.zeros(v, dtype=np.float32)
    row[tok] = 50.0
    return row


def _row_mismatch(v, tok, other, high_entropy, tok_rank_ge3):
    """Row whose argmax is `other` != tok.  High entropy: near-uniform values;
    low entropy: `other` dominates.  tok_rank_ge3 puts three tokens above tok."""
    row = np.zeros(v, dtype=np.float32)
    if high_entropy:
        row[other] = 0.01
        if tok_rank_ge3:
            row[(tok + 1) % v] = 0.005
            row[(tok + 2) % v] = 0.005
            row[tok] = -0.01
        else:
            row[tok] = 0.005
    else:
        row[other] = 50.0
        row[tok] = -1.0 if tok_rank_ge3 else 40.0
    return row


def test_golden_window_example_end_to_end():
    g = json.load(open(os.path.join(GOLDEN, "bcon_window_example.json")))
    M, W, V = g["M"], g["W"], 64
    drafts = np.arange(M, dtype=np.int32).reshape(1, M) + 5
    for case in g["cases"]:
        mis = case["mismatch_at"]
        variants = []
        if not mis:
            variants.append(((False, False), case["n"]))
        elif mis == [2]:
            variants += [((True, True), case["n_if_ent_at_mismatch"]),
                         ((False, True), case["n_if_no_ent_at_mismatch"])]
        else:
            variants += [((True, False), case["n_if_ent_and_topk_at_mismatch"]),
                         ((True, True), case["n_if_ent_no_topk_at_mismatch"])]
        for (hi_ent, rank_ge3), n_expect in variants:
            logits = np.stack([
                _row_mismatch(V, drafts[0, j], 0, hi_ent, rank_ge3) if j in mis
                else _row_exact(V, drafts[0, j]) for j in range(M)])[None]
            out = oracle.soft_gate_verify(logits, "f32", drafts, window=W, topk=3, gamma=0.05)
            con = (out["masks"][0] & CON) > 0
            assert con.astype(int).tolist() == case["B_con"]
            assert out["accept_len"][0] == n_expect, (mis, hi_ent, rank_ge3)
            # Alg. 4's L is n - 1
            assert out["accept_len"][0] - 1 == n_expect - 1


def _structured(rng, c, m, v, p_match=0.6):
    """Logits with a spread of entropies and drafts that match the greedy
    token at a Bernoulli(p_match) subset of positions."""
    sig = rng.choice([0.3, 2.0, 6.0, 12.0], size=(c, m, 1))
    logits = (rng.normal(size=(c, m, v)) * sig).astype(np.float32)
    greedy = logits.argmax(-1)
    rand = rng.integers(0, v, size=(c, m))
    drafts = np.where(rng.random((c, m)) < p_match, greedy, rand).astype(np.int32)
    return logits, drafts


def _greedy_prefix(logits, drafts, lens):
    y = logits.argmax(-1)
    out = []
    for c in range(drafts.shape[0]):
        n = 0
        while n < lens[c] and drafts[c, n] == y[c, n]:
            n += 1
        out.append(n)
    return np.array(out)


def test_gamma_one_reduces_to_greedy_verification():
    rng = np.random.default_rng(21)
    logits, drafts = _structured(rng, 24, 10, 300, p_match=0.85)
    lens = rng.integers(0, 11, size=24).astype(np.int32)
    ref = _greedy_prefix(logits, drafts, lens)
    out = oracle.soft_gate_verify(logits, "f32", drafts, lens, gamma=1.0, topk=10, window=3, tau=2)
    assert np.array_equal(out["accept_len"], ref)
    raw = oracle.soft_gate_verify(logits, "f32", drafts, lens, gamma=math.log(300), topk=10,
                                  window=3, tau=2, entropy_normalized=False)
    assert np.array_equal(raw["accept_len"], ref)
    assert ref.max() > 2          # the case is not vacuous


def test_topk_special_cases():
    rng = np.random.default_rng(4)
    logits, drafts = _structured(rng, 16, 8, 50)
    k1 = oracle.soft_gate_verify(logits, "f32", drafts, topk=1)
    assert np.array_equal((k1["masks"] & TOPK) > 0, (k1["masks"] & EM) > 0)
    kv = oracle.soft_gate_verify(logits, "f32", drafts, topk=50)
    assert ((kv["masks"] & TOPK) > 0).all()


def test_window_not_shorter_than_draft_disables_lookahead():
    rng = np.random.default_rng(9)
    logits, drafts = _structured(rng, 16, 8, 50)
    for w in (8, 9, 20):
        out = oracle.soft_gate_verify(logits, "f32", drafts, window=w, tau=0)
        assert ((out["masks"] & CON) == 0).all()
    out = oracle.soft_gate_verify(logits, "f32", drafts, window=0)
    assert ((out["masks"] & CON) > 0).all()     # empty window: nothing to count


def test_out_of_range_draft_ids_match_nothing():
    rng = np.random.default_rng(6)
    logits, drafts = _structured(rng, 3, 4, 40)
    drafts[0, 0], drafts[1, 1], drafts[2, 3] = -1, 40, 10**6
    for k in (40, 45):                          # k >= V: every real token is in the set
        out = oracle.soft_gate_verify(logits, "f32", drafts, topk=k)
        for c, j in ((0, 0), (1, 1), (2, 3)):
            assert out["rank"][c, j] == 40
            assert out["masks"][c, j] & (EM | TOPK) == 0
        assert out["accept_len"][0] == 0


def test_positions_beyond_draft_length_are_rejected_and_never_read():
    rng = np.random.default_rng(8)
    logits, drafts = _structured(rng, 12, 6, 64, p_match=1.0)
    lens = np.array([0, 1, 2, 3, 4, 5, 6, 6, 3, 0, 1, 2], dtype=np.int32)
    for c in range(12):
        logits[c, lens[c]:] = np.nan              # must not influence anything
    out = oracle.soft_gate_verify(logits, "f32", drafts, lens, gamma=0.0, topk=64)
    assert np.array_equal(out["accept_len"], lens)  # every read position accepted
    for c in range(12):
        assert (out["masks"][c, lens[c]:] & (EM | ENT | TOPK | G) == 0).all()
        assert (out["gate_score"][c, lens[c]:] == 0).all()


GRID_G = [0.01, 0.05, 0.10, 0.30]
GRID_K = [2, 3, 4, 10]
GRID_W = [5, 6, 7, 8, 9]


def test_invariants_over_paper_grid():
    rng = np.random.default_rng(33)
    c, m, v = 32, 12, 200
    logits, drafts = _structured(rng, c, m, v, p_match=0.8)
    lens = rng.integers(0, m + 1, size=c).astype(np.int32)
    res = {}
    for g in GRID_G:
        for k in GRID_K:
            for w in GRID_W:
                for tau in (0, 1):
                    out = oracle.soft_gate_verify(logits, "f32", drafts, lens, gamma=g, topk=k,
                                                  window=w, tau=tau, n_groups=4)
                    n = out["accept_len"]
                    masks = out["masks"]
                    assert ((0 <= n) & (n <= lens) & (lens <= m)).all()
                    em = (masks & EM) > 0
                    assert not (em & ((masks & TOPK) == 0)).any()     # B_em => B_topk
                    assert not (em & ((masks & G) == 0)).any()        # G contains B_em
                    # best = first maximiser per group
                    for gi, b in enumerate(out["best"]):
                        grp = n[gi * 8:(gi + 1) * 8]
                        assert b == int(np.argmax(grp))
                    res[(g, k, w, tau)] = n
    greedy = _greedy_prefix(logits, drafts, lens)
    for key, n in res.items():
        assert (n >= greedy).all()                                    # SE >= exact match
    for k in GRID_K:
        for w in GRID_W:
            for tau in (0, 1):
                for g0, g1 in zip(GRID_G, GRID_G[1:]):                # non-increasing in gamma
                    assert (res[(g1, k, w, tau)] <= res[(g0, k, w, tau)]).all()
    for g in GRID_G:
        for w in GRID_W:
            for tau in (0, 1):
                for k0, k1 in zip(GRID_K, GRID_K[1:]):                # non-decreasing in k
                    assert (res[(g, k1, w, tau)] >= res[(g, k0, w, tau)]).all()
        for k in GRID_K:
            for tau in (0, 1):
                for w0, w1 in zip(GRID_W, GRID_W[1:]):                # non-increasing in W
                    assert (res[(g, k, w1, tau)] <= res[(g, k, w0, tau)]).all()
            for w in GRID_W:
                assert (res[(g, k, w, 1)] >= res[(g, k, w, 0)]).all()  # non-decreasing in tau
    # the sweep is not vacuous: the gate changes something somewhere
    assert any(not np.array_equal(res[(0.01, 10, 5, 1)], res[(0.30, 2, 9, 0)]) for _ in [0])


def test_candidate_permutation_permutes_lengths():
    rng = np.random.default_rng(12)
    logits, drafts = _structured(rng, 10, 8, 100, p_match=0.9)
    a = oracle.soft_gate_verify(logits, "f32", drafts)
    perm = rng.permutation(10)
    b = oracle.soft_gate_verify(logits[perm], "f32", drafts[perm])
    assert np.array_equal(b["accept_len"], a["accept_len"][perm])
    n = b["accept_len"]
    assert b["best"][0] == int(np.flatnonzero(n == n.max())[0])


def test_entropy_gate_is_strict():
    """Alg. 4 gates on a strict comparison, E / ln|V| > gamma.  A row with a
    single finite logit (the rest -inf) has softmax (1, 0, ..., 0) and entropy
    exactly 0, so at gamma = 0 the entropy bit is 0 in both entropy modes, and
    a mismatching draft with a clean look-ahead window is rejected."""
    v, m = 16, 4
    logits = np.full((1, m, v), -np.inf, dtype=np.float32)
    logits[0, :, 7] = 1.0
    drafts = np.array([[3, 7, 7, 7]], dtype=np.int32)        # position 0 mismatches
    for norm in (True, False):
        out = oracle.soft_gate_verify(logits, "f32", drafts, gamma=0.0, topk=v, window=2, tau=0,
                                      entropy_normalized=norm)
        assert out["gate_score"][0, 0] == 0.0
        assert (out["masks"][0] & ENT == 0).all()
        assert out["accept_len"][0] == 0


def test_plus_inf_logits():
    """+inf logits keep the stable order (logit desc, index asc) for the rank;
    the softmax of a row whose maximum is +inf is undefined, so its entropy is
    NaN and the entropy bit is 0 (the draft is then accepted only as the
    exact match)."""
    v = 10
    x = np.zeros((1, 3, v), dtype=np.float32)
    x[0, 0, 4] = np.inf                      # the draft itself: rank 0, B_em
    x[0, 1, [2, 4, 7]] = np.inf              # one +inf left of the draft: rank 1
    x[0, 2, 9] = np.inf                      # the draft finite: 1 above + 4 equal left = 5
    drafts = np.full((1, 3), 4, dtype=np.int32)
    out = oracle.soft_gate_verify(x, "f32", drafts, gamma=-1.0, topk=2, window=0)
    assert out["rank"].tolist() == [[0, 1, 5]]
    assert np.isnan(out["gate_score"]).all()
    assert ((out["masks"] & ENT) == 0).all()
    assert out["masks"][0, 0] & EM and not out["masks"][0, 1] & EM
    assert out["accept_len"][0] == 1
