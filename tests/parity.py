"""Parity rules between the HIP path and the oracle (shared by the GPU tests).

Retrieval: the ordered top-k ids must equal the oracle's, except that two
entries may differ where their oracle scores are within REL_TIE of each other
(a near tie), and at the k/k+1 boundary an id may differ only if its oracle
score is within REL_TIE of the oracle's k-th score.  Scores must match the
oracle's within REL_SCORE relative.  Drafts must match exactly for every id.
Verification: ranks, exact-match and top-k bits exactly; gate scores within
GATE_ABS; the entropy bit and the accepted length exactly unless a gate score
lies within GATE_ABS of gamma.
"""
import numpy as np
import torch

import oracle

REL_TIE = 1e-3
REL_SCORE = 1e-3
GATE_ABS = 1e-4
STRICT_TIE = 1e-5


def host_bits(t: torch.Tensor) -> np.ndarray:
    """Raw uint16 bit patterns (f16/bf16) or float32 array of a device tensor."""
    t = t.detach().cpu().contiguous()
    if t.dtype in (torch.float16, torch.bfloat16):
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def dt_name(t: torch.Tensor) -> str:
    return {torch.float32: "f32", torch.float16: "f16", torch.bfloat16: "bf16"}[t.dtype]


def check_topk(g_ids, g_scores, o_scores_row, k, strict_counter=None):
    """g_ids/g_scores: one query's GPU results; o_scores_row: oracle scores of
    every row.  Returns the number of excused near-tie differences."""
    g_ids = np.asarray(g_ids, dtype=np.int64)
    o_ids, o_sc = oracle.topk(o_scores_row, k)
    assert len(set(g_ids.tolist())) == k, "duplicate ids"
    assert g_ids.min() >= 0 and g_ids.max() < o_scores_row.shape[0], "id out of range"
    s_of = o_scores_row[g_ids]
    # scores of the returned ids
    np.testing.assert_allclose(np.asarray(g_scores, dtype=np.float64), s_of, rtol=REL_SCORE,
                               atol=REL_SCORE * max(1e-30, float(np.abs(o_sc).max())) * 1e-3)
    excused = 0
    sk = o_sc[k - 1]
    for r in range(k):
        if g_ids[r] == o_ids[r]:
            continue
        excused += 1
        gap = abs(s_of[r] - o_sc[r])
        assert gap <= REL_TIE * abs(o_sc[r]), (
            f"rank {r}: gpu id {g_ids[r]} (oracle score {s_of[r]!r}) vs oracle id {o_ids[r]} "
            f"({o_sc[r]!r})")
        if strict_counter is not None and gap > STRICT_TIE * abs(o_sc[r]):
            strict_counter.append((r, gap))
    outside = set(g_ids.tolist()) - set(o_ids.tolist())
    for i in outside:
        assert o_scores_row[i] >= sk - REL_TIE * abs(sk), f"id {i} is not a near tie of the k-th"
    return excused


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
