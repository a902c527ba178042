"""GPU parity of sense_soft_gate_verify against the oracle (Alg. 4).

Structured fixtures exercise every branch of the gate: a spread of
entropies, drafts that follow the greedy token at chosen rates, ties at the
draft token, out-of-vocabulary ids, ragged draft lengths, every logits dtype,
padded rows, unaligned rows (scalar path), vocabularies that are not a
multiple of the vector width, the paper's hyper-parameter grid, and the
full-size verify batches of the benchmark workloads.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_00021_amd import sense, synth
from parity import check_verify, dt_name, host_bits

pytestmark = pytest.mark.gpu
DEV = "cuda"
TDT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def structured(seed, c, m, v, p_match=0.7, dtype="f32"):
    g = torch.Generator().manual_seed(seed)
    sig = torch.tensor([0.05, 0.3, 2.0, 6.0, 12.0])[torch.randint(0, 5, (c, m, 1), generator=g)]
    x = torch.randn((c, m, v), generator=g) * sig
    greedy = x.argmax(-1)
    rand = torch.randint(0, v, (c, m), generator=g)
    drafts = torch.where(torch.rand((c, m), generator=g) < p_match, greedy, rand).int()
    # some rows: a tie at the draft token with a lower index
    tie = torch.rand((c, m), generator=g) < 0.1
    for cc, jj in tie.nonzero().tolist():
        t = int(drafts[cc, jj])
        if t > 0:
            x[cc, jj, t - 1] = x[cc, jj, t]
    x = x.to(TDT[dtype])
    return x, drafts


def run(logits, drafts, draft_len=None, n_groups=1, gamma=0.05, topk=3, window=6, tau=0,
        entropy_normalized=True, vocab=None):
    print(f"[verify] C={drafts.shape[0]} M={drafts.shape[1]} V={logits.shape[-1]} "
          f"{logits.dtype} g={gamma} k={topk} W={window} tau={tau}", flush=True)
    dl_dev = None if draft_len is None else torch.as_tensor(draft_len, dtype=torch.int32).to(DEV)
    ld = logits.to(DEV)
    out = sense.sense_soft_gate_verify(ld, drafts.to(DEV), dl_dev, n_groups=n_groups, gamma=gamma,
                                       topk=topk, window=window, tau=tau,
                                       entropy_normalized=entropy_normalized, vocab=vocab)
    torch.cuda.synchronize()
    ref = oracle.soft_gate_verify(host_bits(logits), dt_name(logits), drafts.numpy(),
                                  None if draft_len is None else np.asarray(draft_len, np.int32),
                                  n_groups=n_groups, gamma=gamma, topk=topk, window=window,
                                  tau=tau, entropy_normalized=entropy_normalized, vocab=vocab)
    excused, near = check_verify(out, ref, gamma, draft_len)
    print(f"[verify] ok (near-threshold positions {near}, excused candidates {excused})",
          flush=True)
    return out, ref


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_full_length_acceptance(dtype):
    """Drafts of 64 tokens (the longest) that pass the gate at every
    position: greedy drafts, gamma below every entropy score and the tied
    (or, in 16 bits, rounded-together) rows inside the top 10, so every
    candidate accepts its whole length
    (all 64 gate bits set) and the first one is the best; with ragged
    lengths each accepts exactly its own length."""
    logits, drafts = structured(37, 6, 64, 512, p_match=1.0, dtype=dtype)
    out, ref = run(logits, drafts, gamma=-1.0, topk=10, window=6)
    assert (out["accept_len"].cpu() == 64).all() and int(out["best"][0]) == 0
    lens = np.array([64, 63, 1, 0, 40, 64], dtype=np.int32)
    out, ref = run(logits, drafts, draft_len=lens, n_groups=2, gamma=-1.0, topk=10, window=6)
    assert np.array_equal(out["accept_len"].cpu().numpy(), lens)


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("v", [32000, 1001, 77])
def test_structured(dtype, v):
    logits, drafts = structured(11, 24, 10, v, dtype=dtype)
    run(logits, drafts, n_groups=3)


def test_ragged_lengths_and_bad_ids():
    logits, drafts = structured(3, 16, 12, 5000, p_match=0.9)
    drafts[0, 0] = -1
    drafts[1, 3] = 5000
    drafts[2, 5] = 1 << 30
    lens = np.array([12, 0, 1, 2, 3, 12, 11, 5, 6, 7, 8, 9, 10, 12, 4, 12], dtype=np.int32)
    lens[3] = 15                                     # clamped to M
    lens[4] = -2                                     # clamped to 0
    run(logits, drafts, lens, n_groups=4)


def test_padded_and_unaligned_rows():
    logits, drafts = structured(5, 8, 6, 3000, dtype="bf16")
    padded = torch.zeros((8, 6, 3011), dtype=torch.bfloat16)
    padded[..., :3000] = logits
    padded[..., 3000:] = 100.0                       # beyond vocab: must be ignored
    out, _ = run(padded, drafts, vocab=3000)         # row_stride 3011: scalar path


@pytest.mark.parametrize("gamma", [0.01, 0.05, 0.10, 0.30, 1.0])
@pytest.mark.parametrize("topk", [1, 2, 3, 4, 10])
def test_paper_grid(gamma, topk):
    logits, drafts = structured(17, 32, 12, 4096, p_match=0.8)
    for window in (5, 6, 9):
        run(logits, drafts, n_groups=4, gamma=gamma, topk=topk, window=window)
    run(logits, drafts, gamma=gamma, topk=topk, window=2, tau=1)


def test_raw_entropy_and_extremes():
    logits, drafts = structured(23, 8, 8, 2048)
    run(logits, drafts, gamma=2.5, entropy_normalized=False)
    run(logits, drafts, window=0)
    run(logits, drafts, window=64, tau=3)
    run(logits, drafts, topk=100000)
    one = torch.zeros((4, 3, 1))
    run(one, torch.zeros((4, 3), dtype=torch.int32), gamma=-1.0)   # |V| = 1


def test_low_entropy_rows_and_minus_inf():
    logits, drafts = structured(29, 8, 8, 1000, p_match=1.0)
    logits[0, 0] = -float("inf")
    logits[0, 0, drafts[0, 0]] = 3.0                 # a single finite logit: E = 0
    logits[1, :, 7] = 60.0                           # very confident rows
    run(logits, drafts)


def test_deterministic():
    logits, drafts = structured(31, 64, 8, 50000, dtype="bf16")
    ld, dd = logits.to(DEV), drafts.to(DEV)
    a = sense.sense_soft_gate_verify(ld, dd)
    b = sense.sense_soft_gate_verify(ld, dd)
    for key in a:
        assert torch.equal(a[key], b[key]), key


@pytest.mark.parametrize("name", ["tiny-16k-d4096", "llama3-8b-262k-d4096", "store-1m-d4096"])
def test_full_size_batches(name):
    w = synth.WORKLOADS[name]
    g = torch.Generator(device=DEV).manual_seed(5)
    drafts = torch.randint(0, w.vocab, (w.n_cand, w.span), generator=g, device=DEV,
                           dtype=torch.int32)
    logits = synth.make_logits(w, drafts, seed=5)
    # sharpen a third of the rows so that exact matches and low entropy occur
    sharp = torch.rand((w.n_cand, w.span), generator=g, device=DEV) < 0.33
    idx = drafts.long().unsqueeze(-1)
    logits.scatter_add_(2, idx, (sharp.to(logits.dtype) * 40).unsqueeze(-1))
    run(logits.cpu(), drafts.cpu(), n_groups=w.verify_queries)


@pytest.mark.parametrize("name", ["13b-batched-4m-d5120", "70b-8m-d8192"])
def test_full_size_batched_groups(name):
    """The verify batches of the batched workloads: 16 groups x 64 drafts x 8
    (fp32, V = 32000) and 4 groups x 128 drafts x 12 (fp32, V = 128256)."""
    w = synth.WORKLOADS[name]
    g = torch.Generator(device=DEV).manual_seed(9)
    drafts = torch.randint(0, w.vocab, (w.n_cand, w.span), generator=g, device=DEV,
                           dtype=torch.int32)
    logits = synth.make_logits(w, drafts, seed=9)
    sharp = torch.rand((w.n_cand, w.span), generator=g, device=DEV) < 0.4
    logits.scatter_add_(2, drafts.long().unsqueeze(-1), (sharp.to(logits.dtype) * 40).unsqueeze(-1))
    dl = torch.randint(0, w.span + 1, (w.n_cand,), generator=g, device=DEV, dtype=torch.int32)
    run(logits.cpu(), drafts.cpu(), dl.cpu().numpy(), n_groups=w.verify_queries)


@pytest.mark.parametrize("dtype,v", [("f32", 3000), ("bf16", 152064), ("f16", 3001)])
def test_plus_inf_logits_rank_in_stable_order(dtype, v):
    """+inf logits take their place in the order (logit desc, index asc) like
    any value: equal +inf values right of the draft token rank below it, left
    of it above it, in the draft's own 16-byte vector, in others and in other
    vocabulary slices; such a row's entropy is NaN on both sides (B_ent 0)."""
    logits, drafts = structured(41, 6, 4, v, dtype="f32")
    inf = float("inf")
    d = int(v * 0.6) | 1
    drafts[:, :] = d
    logits[0, 0, d] = inf                           # d alone at +inf: rank 0
    logits[0, 1, d] = inf
    logits[0, 1, d + 1] = inf                       # right of d, same vector
    logits[0, 1, v - 1] = inf                       # right of d, another slice
    logits[0, 2, d] = inf
    logits[0, 2, d - 1] = inf                       # left of d, same vector: rank 1
    logits[0, 3, d] = inf
    logits[0, 3, 5] = inf                           # left of d, first slice
    logits[0, 3, d - 2] = inf                       # rank 2
    logits[1, 0, d] = 1e4                           # d the largest finite logit
    logits[1, 0, 7] = inf                           # one +inf elsewhere: rank 1
    logits[1, 1, d] = 1e4
    logits[1, 1, v - 1] = inf
    logits[1, 1, 0] = inf                           # two above d
    logits = logits.to(TDT[dtype])
    out, ref = run(logits, drafts, gamma=0.05, topk=3, window=2)
    want = {(0, 0): 0, (0, 1): 0, (0, 2): 1, (0, 3): 2, (1, 0): 1, (1, 1): 2}
    for (cc, jj), r in want.items():
        assert ref["rank"][cc, jj] == r                 # the oracle's stable order
    sense_rank = out["rank"].cpu().numpy()
    for (cc, jj), r in want.items():
        assert sense_rank[cc, jj] == r


def test_nan_logits_stay_in_range():
    """NaN logits are outside the domain: the call still completes with every
    output in its range."""
    c, m, v = 8, 6, 4000
    logits, drafts = structured(43, c, m, v)
    logits[0, 0, :] = float("nan")
    logits[1, 2, 17] = float("nan")
    logits[2, 1, int(drafts[2, 1])] = float("nan")
    lens = torch.tensor([6, 6, 3, 0, 6, 2, 6, 6], dtype=torch.int32)
    out = sense.sense_soft_gate_verify(logits.to(DEV), drafts.to(DEV), lens.to(DEV), n_groups=2)
    torch.cuda.synchronize()
    acc = out["accept_len"].cpu().numpy()
    assert ((acc >= 0) & (acc <= lens.numpy())).all()
    best = out["best"].cpu().numpy()
    assert ((best >= 0) & (best < c // 2)).all()
    rank = out["rank"].cpu().numpy()
    assert ((rank >= 0) & (rank <= v)).all()
