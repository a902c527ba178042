"""Seeded synthetic workloads for the SENSE hot path.

Input generation only: nothing here computes similarity, top-k or any part of
the gate.  The same bytes feed both the HIP library and the CPU oracle.

The datastores stand in for hidden states of the paper's target models
(Llama-2/3 and Qwen families; their datastores and datasets are not
available).  Keys are a Gaussian mixture: centroids ~ N(0, 1), rows = a
uniformly chosen centroid + N(0, 0.3^2) noise, and a few "outlier" channels
(the first n_outliers entries of a seeded permutation of the dimensions)
scaled by 20, mimicking the large-magnitude channels of LLM hidden states.
A query is a stored row plus N(0, 0.05^2) noise (queries of a batch come from
distinct clusters).  Continuations are uniform token ids.  Logits are
N(0, 2^2) with the draft token boosted by +6 at a Bernoulli(0.6) subset of
positions.  Every normal law is written (mean, standard deviation).
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import torch

DTYPES = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


@dataclass(frozen=True)
class Workload:
    name: str
    n: int               # stored rows
    d: int               # key dimension (target hidden size)
    key_dtype: str       # "f16" | "bf16"
    n_queries: int
    k: int               # retrieval top-k
    span: int            # continuation length M
    vocab: int
    logits_dtype: str    # "f32" | "f16" | "bf16"
    n_clusters: int
    n_outliers: int
    verify_queries: int  # queries whose k drafts are verified (groups)
    metric: str = "cosine"
    proj: int = 0        # PCA dimension of the searched keys (0: the hidden states as-is)
    ivf_nlist: int = 0   # inverted lists (0: exact scan)
    ivf_nprobe: int = 0  # lists searched per query
    pq_m: int = 0        # PQ sub-quantizers (0: IVF-Flat)

    @property
    def key_bytes(self) -> int:
        return self.n * self.d * 2

    @property
    def n_cand(self) -> int:
        return self.verify_queries * self.k

    @property
    def logit_bytes(self) -> int:
        return self.n_cand * self.span * self.vocab * (4 if self.logits_dtype == "f32" else 2)


WORKLOADS = {
    w.name: w
    for w in [
        Workload("tiny-16k-d4096", 16_384, 4096, "f16", 1, 8, 8, 32_000, "f32", 256, 4, 1),
        Workload("llama3-8b-262k-d4096", 262_144, 4096, "bf16", 1, 32, 10, 128_256, "f32",
                 1024, 4, 1),
        Workload("qwen2-7b-1m-d3584", 1_048_576, 3584, "bf16", 1, 64, 8, 152_064, "bf16",
                 4096, 8, 1),
        # Headline shape: 1M keys at d = 4096, otherwise the Qwen2-7B shape.
        Workload("store-1m-d4096", 1_048_576, 4096, "bf16", 1, 64, 8, 152_064, "bf16",
                 4096, 8, 1),
        Workload("13b-batched-4m-d5120", 4_194_304, 5120, "f16", 16, 64, 8, 32_000, "f32",
                 16_384, 4, 16),
        Workload("70b-8m-d8192", 8_388_608, 8192, "bf16", 64, 128, 12, 128_256, "f32",
                 16_384, 16, 4),
        # The paper's own key geometry: the headline store projected 4096 -> 64 by
        # PCA and L2-normalised (bf16), the query projected the same way each step.
        Workload("store-1m-pca64", 1_048_576, 4096, "bf16", 1, 64, 8, 152_064, "bf16",
                 4096, 8, 1, proj=64),
        Workload("store-1m-pca64-q64", 1_048_576, 4096, "bf16", 64, 64, 8, 152_064, "bf16",
                 4096, 8, 1, proj=64),
        # The paper's retriever: FAISS-style IVF-PQ (nlist 4096, nprobe 32, pq_m 16)
        # over the PCA-64 keys, and IVF-Flat with the same lists.
        Workload("store-1m-pca64-ivfpq", 1_048_576, 4096, "bf16", 1, 64, 8, 152_064, "bf16",
                 4096, 8, 1, proj=64, ivf_nlist=4096, ivf_nprobe=32, pq_m=16),
        Workload("store-1m-pca64-ivfpq-q64", 1_048_576, 4096, "bf16", 64, 64, 8, 152_064,
                 "bf16", 4096, 8, 1, proj=64, ivf_nlist=4096, ivf_nprobe=32, pq_m=16),
        Workload("store-1m-pca64-ivfflat", 1_048_576, 4096, "bf16", 1, 64, 8, 152_064, "bf16",
                 4096, 8, 1, proj=64, ivf_nlist=4096, ivf_nprobe=32),
        # 64-dim keys straight from the cluster generator (no projection): the
        # short-key paths without a PCA fit in the set-up.
        Workload("store-1m-d64-q64", 1_048_576, 64, "bf16", 64, 64, 8, 152_064, "bf16",
                 4096, 2, 1),
        Workload("store-1m-d64", 1_048_576, 64, "bf16", 1, 64, 8, 152_064, "bf16",
                 4096, 2, 1),
    ]
}
HEADLINE = "store-1m-d4096"


def scaled(w: Workload, **changes) -> Workload:
    """A workload of the same recipe with some sizes changed."""
    return replace(w, **changes)


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


@dataclass
class Datastore:
    keys: torch.Tensor      # n x d (key dtype)
    assign: torch.Tensor    # n int64 cluster of each row
    outliers: torch.Tensor  # n_outliers int64 dims
    spans: torch.Tensor     # n x span int32
    span_len: torch.Tensor | None


def make_datastore(w: Workload, seed: int, device, chunk_rows: int = 1 << 15,
                   ragged_spans: bool = False, key_stride: int | None = None) -> Datastore:
    """Keys, cluster labels and continuations of a workload.  key_stride > d
    lays the rows out with padding (the padding holds a constant)."""
    g = _gen(seed, device)
    d = w.d
    cent = torch.randn(w.n_clusters, d, generator=g, device=device)
    assign = torch.randint(0, w.n_clusters, (w.n,), generator=g, device=device)
    outl = torch.randperm(d, generator=g, device=device)[: w.n_outliers]
    dt = DTYPES[w.key_dtype]
    ld = d if key_stride is None else key_stride
    if ld == d:
        store = torch.empty((w.n, ld), dtype=dt, device=device)
    else:
        store = torch.full((w.n, ld), 7.0, dtype=dt, device=device)
    keys = store[:, :d]
    for r in range(0, w.n, chunk_rows):
        c = min(chunk_rows, w.n - r)
        x = cent[assign[r:r + c]]
        x.add_(torch.randn(c, d, generator=g, device=device), alpha=0.3)
        x[:, outl] *= 20.0
        keys[r:r + c] = x.to(dt)
        del x
    spans = torch.randint(0, w.vocab, (w.n, w.span), generator=g, device=device, dtype=torch.int32)
    span_len = None
    if ragged_spans:
        span_len = torch.randint(0, w.span + 1, (w.n,), generator=g, device=device,
                                 dtype=torch.int32)
    return Datastore(keys, assign, outl, spans, span_len)


def make_queries(w: Workload, ds: Datastore, seed: int, n_queries: int | None = None):
    """Queries = stored rows + N(0, 0.05^2) noise, fp32.  Returns (queries,
    source rows).  Several queries come from distinct clusters."""
    device = ds.keys.device
    g = _gen(seed + 7919, device)
    nq = w.n_queries if n_queries is None else n_queries
    if nq == 1:
        rows = torch.randint(0, w.n, (1,), generator=g, device=device)
    else:
        present = torch.unique(ds.assign)
        pick = present[torch.randperm(present.numel(), generator=g, device=device)[:nq]]
        rows = []
        for c in pick.tolist():
            members = torch.nonzero(ds.assign == c).flatten()
            rows.append(members[torch.randint(0, members.numel(), (1,), generator=g,
                                              device=device)])
        rows = torch.cat(rows)
    q = ds.keys[rows].float()
    q.add_(torch.randn(q.shape, generator=g, device=device), alpha=0.05)
    return q.contiguous(), rows


def make_logits(w: Workload, drafts: torch.Tensor, seed: int, dtype: str | None = None,
                boost: float = 6.0, p_boost: float = 0.6, std: float = 2.0,
                chunk: int = 64) -> torch.Tensor:
    """C x M x V logits ~ N(0, std^2); the draft token of each position gets
    +boost with probability p_boost (draft ids outside [0, V) are skipped)."""
    device = drafts.device
    g = _gen(seed + 104729, device)
    c, m = drafts.shape
    dt = DTYPES[dtype or w.logits_dtype]
    out = torch.empty((c, m, w.vocab), dtype=dt, device=device)
    for c0 in range(0, c, chunk):
        c1 = min(c, c0 + chunk)
        x = torch.randn((c1 - c0, m, w.vocab), generator=g, device=device).mul_(std)
        dr = drafts[c0:c1].long()
        hit = (torch.rand((c1 - c0, m), generator=g, device=device) < p_boost)
        hit &= (dr >= 0) & (dr < w.vocab)
        idx = dr.clamp(0, w.vocab - 1).unsqueeze(-1)
        x.scatter_add_(2, idx, (hit.float() * boost).unsqueeze(-1))
        out[c0:c1] = x.to(dt)
        del x
    return out


@dataclass
class Context:
    keys: torch.Tensor      # length x d fp32 hidden states of generated positions
    tokens: torch.Tensor    # length int32: the token each state predicted
    near: torch.Tensor      # positions planted near the query's source row


def make_context(w: Workload, ds: Datastore, seed: int, length: int, source_row: int,
                 anchor: int, n_near: int = 8, p_anchor: float = 0.1) -> Context:
    """Generation context for a dynamic cache: `length` fp32 states, each a
    stored row chosen uniformly plus N(0, 0.1^2) noise, except n_near
    positions that revisit the query's source row (+ N(0, 0.05^2)), as when
    the generation repeats itself.  Tokens are uniform ids with a fraction
    p_anchor set to `anchor` (so first-token matches occur)."""
    device = ds.keys.device
    g = _gen(seed + 15485863, device)
    rows = torch.randint(0, w.n, (length,), generator=g, device=device)
    x = ds.keys[rows].float()
    x.add_(torch.randn(x.shape, generator=g, device=device), alpha=0.1)
    near = torch.randperm(length, generator=g, device=device)[:min(n_near, length)]
    src = ds.keys[source_row].float()
    x[near] = src + 0.05 * torch.randn((near.numel(), w.d), generator=g, device=device)
    tokens = torch.randint(0, w.vocab, (length,), generator=g, device=device, dtype=torch.int32)
    hit = torch.rand(length, generator=g, device=device) < p_anchor
    tokens[hit] = int(anchor)
    return Context(x.contiguous(), tokens, near)


@dataclass
class Pool:
    scores: torch.Tensor    # Q x n fp32 similarities
    drafts: torch.Tensor    # Q x n x M int32
    lengths: torch.Tensor   # Q x n int32 (may lie outside [0, M])


def make_pool(seed: int, n_queries: int, n: int, max_len: int, vocab: int,
              anchors: torch.Tensor, device, p_anchor: float = 0.3, ragged: bool = True,
              ties: bool = True, specials: bool = False) -> Pool:
    """Retrieval-shaped hits for candidate selection: scores ~ U(-1, 1) (a
    quarter rounded to multiples of 1/64, so exact ties occur), drafts of
    uniform token ids whose first token is the query's anchor with
    probability p_anchor, lengths uniform in [-1, M + 1] when ragged (tokens
    past the length are left as random ids), and, with specials, NaN, +-inf
    and -0 scores sprinkled in."""
    g = _gen(seed + 32452843, device)
    sc = torch.rand((n_queries, n), generator=g, device=device) * 2 - 1
    if ties:
        q = torch.rand((n_queries, n), generator=g, device=device) < 0.25
        sc = torch.where(q, torch.round(sc * 64) / 64, sc)
    if specials and n > 0:
        kind = torch.randint(0, 12, (n_queries, n), generator=g, device=device)
        sc = torch.where(kind == 0, torch.full_like(sc, float("nan")), sc)
        sc = torch.where(kind == 1, torch.full_like(sc, float("inf")), sc)
        sc = torch.where(kind == 2, torch.full_like(sc, float("-inf")), sc)
        sc = torch.where(kind == 3, torch.full_like(sc, -0.0), sc)
    dr = torch.randint(0, vocab, (n_queries, n, max_len), generator=g, device=device,
                       dtype=torch.int32)
    hit = torch.rand((n_queries, n), generator=g, device=device) < p_anchor
    first = torch.where(hit, anchors.view(-1, 1).to(torch.int32).expand(n_queries, n),
                        dr[:, :, 0])
    dr[:, :, 0] = first
    if ragged:
        ln = torch.randint(-1, max_len + 2, (n_queries, n), generator=g, device=device,
                           dtype=torch.int32)
    else:
        ln = torch.full((n_queries, n), max_len, dtype=torch.int32, device=device)
    return Pool(sc.float().contiguous(), dr.contiguous(), ln.contiguous())


def make_drafts(seed: int, n_cand: int, m: int, vocab: int, device, p_share: float = 0.7,
                ragged: bool = True, n_groups: int = 1):
    """Draft batches with shared prefixes, as retrieved continuations of
    neighbouring keys have: within each group, a draft copies the first
    `cut` tokens (cut uniform in [0, M]) of an earlier draft of its group
    with probability p_share; the rest are uniform ids.  Lengths uniform in
    [0, M] when ragged.  Returns (drafts C x M int32, lengths C int32)."""
    g = _gen(seed + 49979687, "cpu")
    d = torch.randint(0, vocab, (n_cand, m), generator=g, dtype=torch.int32)
    gs = n_cand // n_groups
    share = torch.rand(n_cand, generator=g) < p_share
    cut = torch.randint(0, m + 1, (n_cand,), generator=g)
    pick = torch.rand(n_cand, generator=g)
    for i in range(n_cand):
        r = i % gs
        if r > 0 and bool(share[i]):
            src = i - r + int(pick[i] * r)
            c = int(cut[i])
            d[i, :c] = d[src, :c]
    if ragged:
        ln = torch.randint(0, m + 1, (n_cand,), generator=g, dtype=torch.int32)
    else:
        ln = torch.full((n_cand,), m, dtype=torch.int32)
    return d.to(device), ln.to(device)


def make_tree_logits(vocab: int, dtype: str, n_groups: int, nodes: int, tokens, parent, tree_len,
                     seed: int, device, boost: float = 6.0, p_boost: float = 0.6,
                     std: float = 2.0) -> torch.Tensor:
    """Logits of a flattened tree, G x (1 + nodes) x V: rows ~ N(0, std^2);
    for each tree node u, the row that judges it (1 + parent, row 0 at depth
    0) gets +boost at u's token with probability p_boost.  tokens / parent
    are G x nodes host arrays (node u of group g), tree_len the node counts."""
    g = _gen(seed + 86028121, device)
    x = torch.randn((n_groups, 1 + nodes, vocab), generator=g, device=device).mul_(std)
    hit = torch.rand((n_groups, nodes), generator=g, device=device).cpu()
    gi_l, row_l, tok_l = [], [], []
    for gi in range(n_groups):
        for u in range(int(tree_len[gi])):
            tok = int(tokens[gi][u])
            if 0 <= tok < vocab and float(hit[gi, u]) < p_boost:
                gi_l.append(gi)
                row_l.append(1 + int(parent[gi][u]))
                tok_l.append(tok)
    if gi_l:
        idx = tuple(torch.tensor(a, dtype=torch.int64, device=device) for a in (gi_l, row_l, tok_l))
        x.index_put_(idx, torch.full((len(gi_l),), boost, device=device), accumulate=True)
    return x.to(DTYPES[dtype]).contiguous()


def make_shared_spans(w: Workload, ds: Datastore, seed: int, phrases: int = 4,
                      p_diverge: float = 0.25) -> torch.Tensor:
    """Continuations that overlap between neighbours, as text retrieved for
    similar hidden states does: each cluster has `phrases` base
    continuations; a row takes one of its cluster's phrases and, from a
    position onwards where each position diverges with probability
    p_diverge, uniform ids instead.  Returns n x M int32 (same device)."""
    device = ds.keys.device
    g = _gen(seed + 67867967, device)
    base = torch.randint(0, w.vocab, (w.n_clusters, phrases, w.span), generator=g, device=device,
                         dtype=torch.int32)
    pick = torch.randint(0, phrases, (w.n,), generator=g, device=device)
    # first diverging position ~ geometric(p_diverge), by inversion
    u = torch.rand(w.n, generator=g, device=device).clamp_min(1e-12)
    first = torch.floor(torch.log(u) / torch.log(torch.tensor(1.0 - p_diverge))).long()
    div = torch.arange(w.span, device=device)[None, :] >= first[:, None]
    rnd = torch.randint(0, w.vocab, (w.n, w.span), generator=g, device=device, dtype=torch.int32)
    return torch.where(div, rnd, base[ds.assign, pick]).contiguous()


def make_pca_basis(ds: Datastore, seed: int, d_out: int = 64, sample: int = 16384):
    """A PCA fit of the kind the paper's datastore construction uses (the
    fit is input preparation here, not part of the library): mean and the
    top-d_out principal directions of a uniform sample of stored keys, from
    the eigen-decomposition of the sample covariance in float64.  Returns
    (mean [d] fp32, basis [d_out, d] fp32) on the keys' device."""
    device = ds.keys.device
    g = _gen(seed + 32416189, device)
    n = ds.keys.shape[0]
    rows = torch.randint(0, n, (min(sample, n),), generator=g, device=device)
    x = ds.keys[rows].double()
    mean = x.mean(dim=0)
    xc = x - mean
    cov = xc.T @ xc / x.shape[0]
    w, v = torch.linalg.eigh(cov)
    top = torch.argsort(w, descending=True)[:d_out]
    basis = v[:, top].T.contiguous()
    return mean.float().contiguous(), basis.float().contiguous()


def fit_ivf(keys: torch.Tensor, seed: int, nlist: int, pq_m: int = 0, ksub: int = 256,
            iters: int = 6, sample: int = 65536):
    """Coarse centroids (spherical k-means: inner-product assignment, mean
    update) and, with pq_m > 0, PQ codebooks (k-means per sub-space on the
    residuals) of a uniform sample of the keys, in fp32 with torch: the
    FAISS-style training of the paper's index, here input preparation.
    Returns (centroids [nlist, d], codebooks [pq_m, ksub, d/pq_m] or None)."""
    device = keys.device
    g = _gen(seed + 15485867, device)
    n, d = keys.shape
    rows = torch.randint(0, n, (min(sample, n),), generator=g, device=device)
    x = keys[rows].float()
    cen = x[torch.randperm(x.shape[0], generator=g, device=device)[:nlist]].clone()
    for _ in range(iters):
        lab = torch.argmax(x @ cen.T, dim=1)
        sums = torch.zeros_like(cen).index_add_(0, lab, x)
        cnt = torch.bincount(lab, minlength=nlist).float().unsqueeze(1)
        cen = torch.where(cnt > 0, sums / cnt.clamp_min(1.0), cen)
    if pq_m <= 0:
        return cen.contiguous(), None
    lab = torch.argmax(x @ cen.T, dim=1)
    res = (x - cen[lab]).view(x.shape[0], pq_m, d // pq_m)
    books = []
    for j in range(pq_m):
        r = res[:, j, :]
        cb = r[torch.randperm(r.shape[0], generator=g, device=device)[:ksub]].clone()
        for _ in range(iters):
            dist = torch.cdist(r, cb)
            a = torch.argmin(dist, dim=1)
            sums = torch.zeros_like(cb).index_add_(0, a, r)
            cnt = torch.bincount(a, minlength=ksub).float().unsqueeze(1)
            cb = torch.where(cnt > 0, sums / cnt.clamp_min(1.0), cb)
        books.append(cb)
    return cen.contiguous(), torch.stack(books).contiguous()
