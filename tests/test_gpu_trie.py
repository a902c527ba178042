"""GPU parity of the loose trie and of verification through it (Sec. 3.2
Eqs. 9 and 11; Alg. 2 LexSort; Alg. 3; App. tree attention mask; Sec. 3.3;
Alg. 4).

The trie is integer work: order, Gamma, the node table, the ancestor mask
and the static-KV mask must equal the oracle's exactly, and entries the
call must not write keep their sentinel.  Verification through Gamma is
compared with the oracle's dense verification of the Gamma-aligned rows,
under the same rules as the dense path.
"""
import numpy as np
import pytest
import torch

from oracle import trie as otrie
import oracle
from paper_2606_00021_amd import sense, synth
from parity import check_verify, dt_name, host_bits

pytestmark = pytest.mark.gpu

DEV = "cuda"

TRIE_CASES = [
    # n_groups, group size, M, vocab, ragged, p_share
    (1, 4, 3, 5, False, 0.7),
    (1, 64, 8, 3, True, 0.7),
    (3, 64, 8, 50, True, 0.5),
    (2, 1024, 4, 4, True, 0.8),       # largest group
    (1, 64, 64, 2, True, 0.9),        # 4096 tokens, M = 64
    (5, 7, 10, 6, True, 0.6),
    (1, 1, 1, 9, False, 0.0),
    (2, 33, 12, 1000, False, 0.0),    # almost no sharing
    (4, 16, 8, 2, False, 1.0),        # many identical drafts
]


def oracle_group(D, lens, g, gs, m):
    sl = slice(g * gs, (g + 1) * gs)
    order = otrie.lexsort_candidates(D[sl], lens[sl])
    S, SL = D[sl][order], lens[sl][order]
    T, gamma, mask = otrie.loose_trie(S, SL)
    parent, depth, cand = otrie.node_table(gamma)
    return order, S, np.clip(SL, 0, m), T, gamma, mask, parent, depth, cand


@pytest.mark.parametrize("case", TRIE_CASES, ids=[str(i) for i in range(len(TRIE_CASES))])
def test_trie_matches_oracle(case):
    G, gs, m, vocab, ragged, p_share = case
    print(f"[trie] case={case}", flush=True)
    c = G * gs
    nodes = gs * m
    drafts, lens = synth.make_drafts(17 + gs, c, m, vocab, DEV, p_share, ragged, n_groups=G)
    prefix, cache = 5, nodes + 9
    fspec = {"dtype": torch.float32, "prefix_len": prefix, "cache_len": cache}
    out = sense.sense_build_loose_trie(drafts, lens if ragged else None, n_groups=G,
                                       want_mask=True, full_mask=fspec)
    out["mask"].fill_(7)           # sentinel: only rows/columns < L may change
    out["full_mask"].fill_(3.0)
    out = sense.sense_build_loose_trie(drafts, lens if ragged else None, n_groups=G, out=out,
                                       full_mask=fspec)
    torch.cuda.synchronize()
    D = drafts.cpu().numpy()
    LN = lens.cpu().numpy() if ragged else np.full(c, m)
    h = {k: v.cpu().numpy() for k, v in out.items()}
    for g in range(G):
        order, S, SL, T, gamma, mask, parent, depth, cand = oracle_group(D, LN, g, gs, m)
        L = T.shape[0]
        sl = slice(g * gs, (g + 1) * gs)
        assert np.array_equal(h["order"][sl], order), f"group {g}: order"
        assert np.array_equal(h["gamma"][sl], gamma), f"group {g}: gamma"
        assert h["tree_len"][g] == L
        pad = -np.ones(nodes - L, dtype=np.int64)
        assert np.array_equal(h["tree_tokens"][g], np.r_[T, pad])
        assert np.array_equal(h["tree_parent"][g], np.r_[parent, pad])
        assert np.array_equal(h["tree_depth"][g], np.r_[depth, pad])
        assert np.array_equal(h["tree_cand"][g], np.r_[cand, pad])
        exist = np.arange(m)[None, :] < SL[:, None]
        assert np.array_equal(h["sorted_drafts"][sl], np.where(exist, S, -1))
        assert np.array_equal(h["sorted_len"][sl], SL)
        assert np.array_equal(h["mask"][g][:L, :L], mask)
        assert (h["mask"][g][L:] == 7).all() and (h["mask"][g][:, L:] == 7).all()
        fm = otrie.full_mask(mask, prefix, cache)
        assert np.array_equal(h["full_mask"][g][:L], fm.astype(np.float32))
        assert (h["full_mask"][g][L:] == 3.0).all()


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float16])
def test_full_mask_16bit(dtype):
    drafts, lens = synth.make_drafts(3, 32, 6, 4, DEV, 0.8, True)
    out = sense.sense_build_loose_trie(drafts, lens, full_mask={"dtype": dtype, "prefix_len": 0,
                                                                 "cache_len": 200})
    torch.cuda.synchronize()
    order, S, SL, T, gamma, mask, *_ = oracle_group(drafts.cpu().numpy(), lens.cpu().numpy(), 0,
                                                    32, 6)
    L = T.shape[0]
    got = out["full_mask"][0][:L].float().cpu().numpy()
    assert np.array_equal(got, otrie.full_mask(mask, 0, 200).astype(np.float32))


VERIFY_CASES = [
    # n_groups, group size, M, draft vocab, V, logits dtype, p_share, ragged
    (1, 64, 8, 6, 32000, "f32", 0.7, True),
    (2, 32, 10, 4, 5000, "bf16", 0.8, False),
    (1, 16, 8, 3, 152064, "bf16", 0.7, True),
    (3, 8, 12, 30, 1001, "f16", 0.5, True),
    (1, 128, 4, 2, 2048, "f32", 0.9, False),
]


@pytest.mark.parametrize("case", VERIFY_CASES, ids=[str(i) for i in range(len(VERIFY_CASES))])
def test_verify_tree_matches_oracle(case):
    G, gs, m, dv, vocab, ldt, p_share, ragged = case
    print(f"[verify-tree] case={case}", flush=True)
    c, nodes = G * gs, gs * m
    drafts, lens = synth.make_drafts(29 + gs, c, m, dv, DEV, p_share, ragged, n_groups=G)
    tr = sense.sense_build_loose_trie(drafts, lens if ragged else None, n_groups=G)
    D = drafts.cpu().numpy()
    LN = lens.cpu().numpy() if ragged else np.full(c, m)
    groups = [oracle_group(D, LN, g, gs, m) for g in range(G)]
    tok_h = [np.r_[gr[3], -np.ones(nodes - gr[3].shape[0], dtype=np.int64)] for gr in groups]
    par_h = [np.r_[gr[6], -np.ones(nodes - gr[3].shape[0], dtype=np.int64)] for gr in groups]
    tl_h = [gr[3].shape[0] for gr in groups]
    logits = synth.make_tree_logits(vocab, ldt, G, nodes, tok_h, par_h, tl_h, 31 + gs, DEV)
    out = sense.sense_soft_gate_verify_tree(logits, tr, n_groups=G, gamma=0.05, topk=3,
                                            window=3)
    torch.cuda.synchronize()
    bits = host_bits(logits)
    for g, (order, S, SL, T, gamma, mask, parent, depth, cand) in enumerate(groups):
        assert np.array_equal(tr["gamma"][g * gs:(g + 1) * gs].cpu().numpy(), gamma)
        dense = otrie.aligned_logits(bits[g], gamma)
        ref = oracle.soft_gate_verify(dense, ldt, S.astype(np.int32), SL.astype(np.int32),
                                      gamma=0.05, topk=3, window=3)
        sl = slice(g * gs, (g + 1) * gs)
        sub = {"accept_len": out["accept_len"][sl], "best": out["best"][g:g + 1],
               "gate_score": out["gate_score"][sl], "masks": out["masks"][sl],
               "rank": out["rank"][sl]}
        check_verify(sub, ref, 0.05, SL)


def test_verify_tree_full_length():
    """Groups of 16 drafts of 64 tokens (1024 tree rows) that pass the gate
    at every judged position (gamma below every entropy score, top-k over
    the whole vocabulary): every draft accepts all 64 positions through
    Gamma, and the result meets the oracle's dense verification."""
    G, gs, m, vocab = 2, 16, 64, 1000
    drafts, lens = synth.make_drafts(43, G * gs, m, 3, DEV, 0.8, False, n_groups=G)
    tr = sense.sense_build_loose_trie(drafts, None, n_groups=G)
    D = drafts.cpu().numpy()
    groups = [oracle_group(D, np.full(G * gs, m), g, gs, m) for g in range(G)]
    nodes = gs * m
    tok_h = [np.r_[gr[3], -np.ones(nodes - gr[3].shape[0], dtype=np.int64)] for gr in groups]
    par_h = [np.r_[gr[6], -np.ones(nodes - gr[3].shape[0], dtype=np.int64)] for gr in groups]
    tl_h = [gr[3].shape[0] for gr in groups]
    logits = synth.make_tree_logits(vocab, "bf16", G, nodes, tok_h, par_h, tl_h, 47, DEV)
    out = sense.sense_soft_gate_verify_tree(logits, tr, n_groups=G, gamma=-1.0, topk=1 << 20,
                                            window=3)
    torch.cuda.synchronize()
    bits = host_bits(logits)
    for g, (order, S, SL, T, gamma, mask, parent, depth, cand) in enumerate(groups):
        dense = otrie.aligned_logits(bits[g], gamma)
        ref = oracle.soft_gate_verify(dense, "bf16", S.astype(np.int32), SL.astype(np.int32),
                                      gamma=-1.0, topk=1 << 20, window=3)
        sl = slice(g * gs, (g + 1) * gs)
        sub = {"accept_len": out["accept_len"][sl], "best": out["best"][g:g + 1],
               "gate_score": out["gate_score"][sl], "masks": out["masks"][sl],
               "rank": out["rank"][sl]}
        check_verify(sub, ref, -1.0, SL)
    assert (out["accept_len"].cpu() == m).all()


def test_verify_tree_equals_dense_verify_bitwise():
    """The same row statistics read through Gamma or from a dense copy of
    the aligned rows give identical bits."""
    drafts, lens = synth.make_drafts(5, 48, 8, 5, DEV, 0.8, True)
    tr = sense.sense_build_loose_trie(drafts, lens)
    torch.cuda.synchronize()
    L = int(tr["tree_len"][0])
    nodes = 48 * 8
    logits = synth.make_tree_logits(4000, "bf16", 1, nodes, tr["tree_tokens"].cpu().numpy(),
                                    tr["tree_parent"].cpu().numpy(), [L], 9, DEV)
    gam = tr["gamma"].long()
    rows = torch.zeros_like(gam)
    rows[:, 1:] = torch.where(gam[:, :-1] >= 0, gam[:, :-1] + 1, torch.zeros_like(gam[:, :-1]))
    dense = logits[0][rows].contiguous()
    a = sense.sense_soft_gate_verify_tree(logits, tr)
    b = sense.sense_soft_gate_verify(dense, tr["sorted_drafts"], tr["sorted_len"])
    torch.cuda.synchronize()
    for k in ("accept_len", "best", "masks", "rank"):
        assert torch.equal(a[k], b[k]), k
    assert torch.equal(a["gate_score"].view(torch.int32), b["gate_score"].view(torch.int32))


def test_trie_is_deterministic():
    drafts, lens = synth.make_drafts(8, 512, 8, 3, DEV, 0.9, True)
    a = {k: v.clone() for k, v in sense.sense_build_loose_trie(drafts, lens, want_mask=True).items()}
    b = sense.sense_build_loose_trie(drafts, lens, want_mask=True)
    torch.cuda.synchronize()
    for k in a:
        assert torch.equal(a[k], b[k]), k
