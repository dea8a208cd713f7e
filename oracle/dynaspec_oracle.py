"""Plain CPU oracle for DynaSpec's dynamic draft head (arXiv 2510.13847).

TEST INFRASTRUCTURE ONLY.  This module is the slow, obviously-correct
definition the HIP library is checked against.  Only the test-suite, the
smoke check and the CPU-baseline leg of the benchmark may import it; the
library never calls it and shares no code, table or helper with it.

Everything is evaluated in float64 from the exact input values: fp32 arrays
are widened, bf16 inputs arrive as raw uint16 bit patterns and are decoded
here (a bf16 value is the upper half of an fp32 word, so the decode is exact).

The path, in the paper's order (Sec. 4.2 "Context-aware dynamic sub-vocabulary
selection", Sec. 4.3 "Dynamic Drafting", Algorithm 1):

  partition      V = disjoint union of clusters C_1..C_M          (Sec. 4.2, "Vocabulary partition")
  router         s = r_theta(x), a small FFN                       (Sec. 4.2, "Low-cost router"; "Training the router")
  top-k          K = TopK_k(s)                                     (Sec. 4.2)
  shortlist      V_S = disjoint union of C_m over m in K           (Sec. 4.2)
  logits         z = h . W_LM[:, V_S]  (gathered head)             (Sec. 4.3; Algorithm 1, FUSED_INDEX_GEMM)
  select         log_softmax over V_S, TopK_{k_t}, remap to ids    (Algorithm 1; Sec. 5 restricted draft q_S)

Readings where the paper is silent (each is listed in the design notes):
  * the LM head is stored [V, d] row-major: paper column v is row v;
  * ties in any top-k go to the lower id (cluster id for routing, vocabulary
    id for tokens); NaN scores count as -inf; -0 equals +0;
  * the shortlist is ordered by ascending cluster id, then ascending
    vocabulary id inside a cluster;
  * log-probabilities and sampling use softmax(z / T) over the shortlist
    (T = 1 gives Algorithm 1's log_softmax(z)); sampling walks the CDF in
    shortlist order and returns the first j with F_j > u, else the last j
    with p_j > 0;
  * the router's hidden activation is not re-rounded (fp64 here);
  * clusters may be empty (no balance is enforced), so a context can select
    only empty clusters: its shortlist is empty and it proposes no token (no
    ids, no sample);
  * the partition itself comes from spherical k-means on the unit LM-head
    rows (Sec. 4.2): centroids start at caller-chosen points, each round
    assigns every point to its most similar centroid (cosine similarity in
    float64; ties to the lower id) and then sets each centroid to the mean
    direction of its points; an empty cluster keeps its centroid.

Every function below has a pin in tests/test_oracle_pins.py.
"""
from __future__ import annotations

import numpy as np

ACTS = ("none", "relu", "silu")


# --------------------------------------------------------------------------
# input decoding
# --------------------------------------------------------------------------
def as_f64(a) -> np.ndarray:
    """float64 view of an input: fp32/fp64 values, or bf16 bit patterns (uint16)."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    if a.dtype in (np.float32, np.float64):
        return a.astype(np.float64)
    raise TypeError(f"unsupported input dtype {a.dtype}")


# --------------------------------------------------------------------------
# vocabulary partition (Sec. 4.2, "Vocabulary partition")
# --------------------------------------------------------------------------
def cluster_layout(cluster_of, M: int):
    """Cluster-contiguous layout of a partition of the vocabulary.

    The paper partitions V into M disjoint clusters with no balance
    constraint.  Laid out cluster by cluster (ascending cluster id, ascending
    vocabulary id inside each cluster), every cluster is one contiguous run.

    Returns (sizes[M], offsets[M+1], perm[V], cap_by_k[M+1]):
      perm[j]     vocabulary id stored at layout row j;
      offsets[m]  first layout row of cluster m;
      cap_by_k[k] largest possible shortlist of k clusters (sum of the k
                  largest cluster sizes).
    """
    cluster_of = np.asarray(cluster_of, dtype=np.int64)
    if cluster_of.size and (cluster_of.min() < 0 or cluster_of.max() >= M):
        raise ValueError("cluster id out of range")
    sizes = np.bincount(cluster_of, minlength=M).astype(np.int64)
    offsets = np.zeros(M + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(sizes)
    perm = np.argsort(cluster_of, kind="stable").astype(np.int64)
    cap_by_k = np.zeros(M + 1, dtype=np.int64)
    cap_by_k[1:] = np.cumsum(np.sort(sizes)[::-1])
    return sizes, offsets, perm, cap_by_k


# --------------------------------------------------------------------------
# router (Sec. 4.2, "Low-cost router" and "Training the router")
# --------------------------------------------------------------------------
def activation(a: np.ndarray, act: str) -> np.ndarray:
    if act == "none":
        return a
    if act == "relu":
        return np.maximum(a, 0.0)
    if act == "silu":
        return a / (1.0 + np.exp(-a))
    raise ValueError(act)


def router_scores(x, W1, W2=None, b1=None, b2=None, act: str = "silu") -> np.ndarray:
    """Cluster scores s[B, M] from context features x[B, d_r].

    Two-layer FFN: s = W2 . act(W1 . x + b1) + b2, with W1 [H, d_r] and
    W2 [M, H].  With W2 = None the router is one linear map s = W1 . x + b1,
    W1 [M, d_r].  The sigmoid of the training loss is not part of scoring
    (top-k is invariant to it).
    """
    x = as_f64(x)
    W1 = as_f64(W1)
    pre = x @ W1.T
    if b1 is not None:
        pre = pre + as_f64(b1)
    if W2 is None:
        return pre
    a = activation(pre, act)
    s = a @ as_f64(W2).T
    if b2 is not None:
        s = s + as_f64(b2)
    return s


# --------------------------------------------------------------------------
# ordering rule shared by every top-k of the path (a reading, see header)
# --------------------------------------------------------------------------
def _canonical(values: np.ndarray) -> np.ndarray:
    v = np.where(np.isnan(values), -np.inf, values)
    return v + 0.0  # -0 + 0 = +0 under round-to-nearest


def rank_order(values, ids) -> np.ndarray:
    """Indices that sort (values desc, ids asc)."""
    v = _canonical(np.asarray(values, dtype=np.float64))
    return np.lexsort((np.asarray(ids), -v))


# --------------------------------------------------------------------------
# top-k clusters (Sec. 4.2, K(c,t) = TopK_{k_c(t)}(s))
# --------------------------------------------------------------------------
def topk_clusters(scores, k: int):
    """Per row, the k clusters with the highest scores, in rank order.

    Returns (ids[B, k], vals[B, k]).
    """
    s = np.atleast_2d(np.asarray(scores, dtype=np.float64))
    B, M = s.shape
    if not 1 <= k <= M:
        raise ValueError("k out of range")
    ids = np.empty((B, k), dtype=np.int64)
    vals = np.empty((B, k), dtype=np.float64)
    for b in range(B):
        order = rank_order(s[b], np.arange(M))[:k]
        ids[b] = order
        vals[b] = s[b, order]
    return ids, vals


# --------------------------------------------------------------------------
# shortlist (Sec. 4.2, V_S = disjoint union of the selected clusters)
# --------------------------------------------------------------------------
def shortlist(cluster_ids, offsets, perm):
    """Shortlist of one context from its selected cluster ids.

    Returns (sel_sorted[k], rowoff[k+1], layout_rows[n], vocab_ids[n]):
    clusters in ascending id, the start of each cluster inside the
    shortlist, the layout rows of the shortlist, and their vocabulary ids.
    """
    sel = np.sort(np.asarray(cluster_ids, dtype=np.int64))
    offsets = np.asarray(offsets, dtype=np.int64)
    sizes = offsets[sel + 1] - offsets[sel]
    rowoff = np.zeros(sel.size + 1, dtype=np.int64)
    rowoff[1:] = np.cumsum(sizes)
    rows = np.concatenate([np.arange(offsets[m], offsets[m + 1]) for m in sel]) \
        if sel.size else np.zeros(0, dtype=np.int64)
    return sel, rowoff, rows, np.asarray(perm, dtype=np.int64)[rows]


# --------------------------------------------------------------------------
# gathered head (Sec. 4.3; Algorithm 1, FUSED_INDEX_GEMM)
# --------------------------------------------------------------------------
def shortlist_logits(h, W_lm, vocab_ids) -> np.ndarray:
    """z[j] = h . W_LM[:, vocab_ids[j]] for one context row h[d].

    Read from the original (vocabulary-ordered) LM head, never from the
    permuted copy, so a layout error cannot hide in both sides.
    """
    Wg = as_f64(np.asarray(W_lm)[np.asarray(vocab_ids, dtype=np.int64)])
    return Wg @ as_f64(h)


# --------------------------------------------------------------------------
# draft selection (Algorithm 1: log_softmax, TopK_{k_t}, remap2realid;
# Sec. 5: the restricted, renormalised draft q_S)
# --------------------------------------------------------------------------
def log_softmax(z, temperature: float = 1.0) -> np.ndarray:
    """log q_S over the shortlist: z/T - log(sum exp(z/T)), shifted by the max.
    An empty shortlist has no log-probabilities."""
    t = np.asarray(z, dtype=np.float64) / float(temperature)
    if t.size == 0:
        return t
    mx = np.max(t)
    return t - (mx + np.log(np.sum(np.exp(t - mx))))


def topk_tokens(z, vocab_ids, k_t: int):
    """Positions of the k_t largest logits, ordered (z desc, vocabulary id asc)."""
    order = rank_order(z, vocab_ids)
    return order[:k_t]


def sample_inverse_cdf(z, u: float, temperature: float = 1.0) -> int:
    """Shortlist position drawn from softmax(z/T) by the inverse CDF at u.

    The CDF runs in shortlist order; the answer is the first j with F_j > u,
    else (when rounding leaves F_n <= u) the last j with p_j > 0.  An empty
    shortlist gives -1 (no token).
    """
    t = np.asarray(z, dtype=np.float64) / float(temperature)
    if t.size == 0:
        return -1
    p = np.exp(t - np.max(t))
    p = p / p.sum()
    F = np.cumsum(p)
    hit = np.nonzero(F > u)[0]
    if hit.size:
        return int(hit[0])
    return int(np.nonzero(p > 0)[0][-1])


def sample_cdf(z, temperature: float = 1.0) -> np.ndarray:
    """Normalised CDF in shortlist order (used to find near-boundary uniforms)."""
    t = np.asarray(z, dtype=np.float64) / float(temperature)
    p = np.exp(t - np.max(t))
    return np.cumsum(p / p.sum())


def draft_select(z, vocab_ids, k_t: int = 1, temperature: float = 1.0, u=None, beta: float = 0.0,
                 complement_ids=None):
    r"""Draft outputs of one context over its shortlist.

    Returns dict(ids[k_t], logprobs[k_t], positions[k_t], sample_id,
    sample_pos, sample_logprob); ids are vocabulary ids (remap2realid).

    With beta > 0 the proposal is the tail mixture of Sec. 5,
    q~ = (1 - beta) q_S + beta * omega, omega uniform on the complement
    V \ S given by complement_ids (in layout order).  Top-k positions stay in
    the shortlist, with log-probabilities under q~.  The sample takes the
    shortlist branch when u < 1 - beta (at u / (1 - beta)), else complement
    entry floor((u - (1 - beta)) / beta * |V \ S|) (sample_pos = -1).  An empty
    complement leaves q~ = q_S.
    """
    vocab_ids = np.asarray(vocab_ids, dtype=np.int64)
    if vocab_ids.size == 0 and (complement_ids is None or len(complement_ids) == 0 or beta <= 0.0):
        # only empty clusters were selected: nothing to propose
        e = np.zeros(0, dtype=np.int64)
        out = dict(ids=e, logprobs=np.zeros(0), positions=e)
        if u is not None:
            out.update(sample_id=-1, sample_pos=-1, sample_logprob=-np.inf)
        return out
    C = 0 if complement_ids is None else len(complement_ids)
    b = float(beta) if (beta > 0.0 and C > 0) else 0.0
    lp = log_softmax(z, temperature) + (np.log1p(-b) if b > 0.0 else 0.0)
    pos = topk_tokens(z, vocab_ids, k_t)
    out = dict(ids=vocab_ids[pos], logprobs=lp[pos], positions=pos)
    if u is not None:
        u = float(u)
        if u < 1.0 - b:
            j = sample_inverse_cdf(z, u / (1.0 - b), temperature)
            out.update(sample_id=int(vocab_ids[j]), sample_pos=j, sample_logprob=float(lp[j]))
        else:
            jj = min(C - 1, int(np.floor((u - (1.0 - b)) / b * C)))
            out.update(sample_id=int(complement_ids[jj]), sample_pos=-1,
                       sample_logprob=float(np.log(b) - np.log(C)))
    return out


def complement(offsets, perm, sel_sorted):
    """Vocabulary ids outside the shortlist of clusters sel_sorted, in layout order."""
    offsets = np.asarray(offsets, dtype=np.int64)
    keep = np.ones(int(offsets[-1]), dtype=bool)
    for m in np.asarray(sel_sorted, dtype=np.int64):
        keep[offsets[m]:offsets[m + 1]] = False
    return np.asarray(perm, dtype=np.int64)[np.nonzero(keep)[0]]


# --------------------------------------------------------------------------
# whole head and the two baselines
# --------------------------------------------------------------------------
def union_clusters(cluster_ids) -> np.ndarray:
    """Clusters selected by any row of a step, ascending (Sec. 4.2: with
    several tokens at a step, the union of their predicted clusters)."""
    return np.unique(np.asarray(cluster_ids, dtype=np.int64).ravel())


def draft_head(x, h, W1, W2, act, cluster_of, M, W_lm, k, k_t=1, temperature=1.0,
               u=None, b1=None, b2=None, beta: float = 0.0, union: bool = False):
    """The dynamic draft head for a batch: route, shortlist, logits, select.

    With union=True every row of the step shares one shortlist, the union of
    the rows' selected clusters (Sec. 4.2); otherwise each row has its own.
    Returns a list (one dict per context row) with the router's cluster ids,
    the shortlist and the draft outputs.
    """
    sizes, offsets, perm, _ = cluster_layout(cluster_of, M)
    s = router_scores(x, W1, W2, b1, b2, act)
    ids, vals = topk_clusters(s, k)
    h = np.atleast_2d(np.asarray(h))
    shared = union_clusters(ids) if union else None
    out = []
    for b in range(h.shape[0]):
        sel, rowoff, rows, vids = shortlist(shared if union else ids[b], offsets, perm)
        z = shortlist_logits(h[b], W_lm, vids)
        comp = complement(offsets, perm, sel) if beta > 0.0 else None
        r = draft_select(z, vids, k_t, temperature, None if u is None else u[b], beta, comp)
        r.update(clusters=ids[b], cluster_scores=vals[b], sel_sorted=sel, rowoff=rowoff,
                 layout_rows=rows, vocab_ids=vids, logits=z, scores=s[b])
        out.append(r)
    return out


def beam_expand(logprobs, ids, last_scores, n_out: int):
    """EAGLE-2 style expansion (Algorithm 1): cumulative scores
    cu[b, r] = logprobs[b, r] + last_scores[b] over the B x k_t candidates of a
    step; the n_out largest, ordered (cu desc, b asc, r asc), give the next
    beam: (scores[n_out], parent rows[n_out], token ids[n_out]).  Candidates
    with no token (id < 0) are never chosen."""
    lp = np.asarray(logprobs, dtype=np.float64)
    ids = np.asarray(ids, dtype=np.int64)
    B, kt = lp.shape
    last = np.zeros(B) if last_scores is None else np.asarray(last_scores, dtype=np.float64)
    cu = lp + last[:, None]
    cand = [(cu[b, r], b, r) for b in range(B) for r in range(kt) if ids[b, r] >= 0]
    cand.sort(key=lambda c: (-_canonical(np.array([c[0]]))[0], c[1], c[2]))
    cand = cand[:n_out]
    return (np.array([c[0] for c in cand]), np.array([c[1] for c in cand], dtype=np.int64),
            np.array([ids[c[1], c[2]] for c in cand], dtype=np.int64))


def draft_cycle(x0, h0, next_inputs, W1, W2, act, cluster_of, M, W_lm, k_first: int, k_second: int,
                k_t: int, gamma: int, k_min: int = 1, form: str = "equation"):
    """One verification cycle of drafting (Algorithm 1): positions j = 0..gamma.

    Position j routes each of its rows with the budget k_c(j) (k_schedule),
    evaluates every row over the union of the rows' clusters, keeps each
    row's k_t best log-probabilities (TopP_j, ids T~_j), adds the parent's
    score (cu_scores = TopP_j + last_step_scores, zero at j = 0) and keeps the
    k_t best cu_scores over the position (beam_expand): their scores are the
    next last_step_scores, their tokens x_j and their rows the parents whose
    hidden rows h~[TopC_j] the next position extends.

    x0 [1, d_r], h0 [1, d]: the router input and the drafter's hidden row of
    the first position.  next_inputs(h_parent_rows, tokens) -> (x, h) stands
    in for the draft layer (outside the head): the next position's router
    input and hidden rows from the parents' hidden rows and the new tokens.

    Returns (positions, draft_list).  positions[j] holds k, the union head's
    per-row results ("heads"), ids/logprobs [B, k_t] (-1 / -inf past a short
    shortlist), cu_scores [B, k_t] and the beam (scores, parents, tokens).
    draft_list re-ranks every drafted token by cu_score, descending; ties go
    to the earlier position, then the lower row, then the better rank.
    """
    x, h = np.atleast_2d(np.asarray(x0)), np.atleast_2d(np.asarray(h0))
    last = None
    positions = []
    for j in range(gamma + 1):
        k = k_schedule(j, k_first, k_second, k_min, form)
        heads = draft_head(x, h, W1, W2, act, cluster_of, M, W_lm, k, k_t=k_t, union=True)
        B = len(heads)
        ids = np.full((B, k_t), -1, dtype=np.int64)
        lp = np.full((B, k_t), -np.inf)
        for b, r in enumerate(heads):
            n = len(r["ids"])
            ids[b, :n] = r["ids"]
            lp[b, :n] = r["logprobs"]
        base = np.zeros(B) if last is None else np.asarray(last, dtype=np.float64)
        cu = lp + base[:, None]
        scores, parents, tokens = beam_expand(lp, ids, last, k_t)
        positions.append(dict(k=k, heads=heads, ids=ids, logprobs=lp, cu_scores=cu, scores=scores,
                              parents=parents, tokens=tokens))
        last = scores
        if j < gamma:
            x, h = next_inputs(h[parents], tokens)
    entries = [(positions[j]["cu_scores"][b, r], j, b, r, positions[j]["ids"][b, r])
               for j in range(len(positions)) for b in range(positions[j]["ids"].shape[0])
               for r in range(k_t) if positions[j]["ids"][b, r] >= 0]
    entries.sort(key=lambda e: (-e[0], e[1], e[2], e[3]))
    draft_list = dict(scores=np.array([e[0] for e in entries]),
                      position=np.array([e[1] for e in entries], dtype=np.int64),
                      row=np.array([e[2] for e in entries], dtype=np.int64),
                      rank=np.array([e[3] for e in entries], dtype=np.int64),
                      ids=np.array([e[4] for e in entries], dtype=np.int64))
    return positions, draft_list


def dense_head(h, W_lm, k_t=1, temperature=1.0, u=None, n_rows=None):
    """Full-vocabulary head O = H W_LM (Sec. 4.1), or, with n_rows, the static
    head over the first n_rows vocabulary ids (Sec. 4.1, the FR-Spec drafter,
    with an id prefix standing in for the frequency ranking)."""
    W = np.asarray(W_lm)
    if n_rows is not None:
        W = W[:n_rows]
    vids = np.arange(W.shape[0])
    h = np.atleast_2d(np.asarray(h))
    Wf = as_f64(W)
    out = []
    for b in range(h.shape[0]):
        z = Wf @ as_f64(h[b])
        r = draft_select(z, vids, k_t, temperature, None if u is None else u[b])
        r["logits"] = z
        out.append(r)
    return out


# --------------------------------------------------------------------------
# position-aware cluster budget (Sec. 4.2, eq. pos_schedule; Algorithm 1)
# --------------------------------------------------------------------------
def k_schedule(t: int, k0: int, k1: int, k_min: int = 1, form: str = "equation") -> int:
    """Cluster budget at draft position t: k0, k1, then floor((k1 + t) / (2t)),
    clamped below at k_min (the equation reaches 0 for large t while the
    text bounds the budget by k_min).  form="algorithm1" takes the appendix
    algorithm's floor(k1 / (2t)) for t >= 2 instead (its undefined index read
    as the draft position)."""
    if t == 0:
        return k0
    if t == 1:
        return k1
    if form == "equation":
        return max(k_min, (k1 + t) // (2 * t))
    if form == "algorithm1":
        return max(k_min, k1 // (2 * t))
    raise ValueError(form)


# --------------------------------------------------------------------------
# position-aware frequency-ranked static shortlist (appendix, PA-FR)
# --------------------------------------------------------------------------
def pa_fr_budget(t: int, k_max: int) -> int:
    """Static shortlist size at draft position t: k_max for t in {0, 1}, then
    floor(k_max / (t + 1)); the shortlist is the K most frequent ids (here the
    first K ids of the vocabulary, see dense_head)."""
    if t < 2:
        return k_max
    return k_max // (t + 1)


# --------------------------------------------------------------------------
# building the partition: spherical k-means (Sec. 4.2, "Vocabulary partition")
# --------------------------------------------------------------------------
def unit_rows(W) -> np.ndarray:
    """The paper's points: every LM-head column (here row) divided by its
    2-norm; an all-zero row stays zero (it has no direction)."""
    X = as_f64(W)
    n = np.sqrt((X * X).sum(axis=1))
    out = np.zeros_like(X)
    nz = n > 0
    out[nz] = X[nz] / n[nz, None]
    return out


def kmeans_assign(W, centroids):
    """Assignment step: each point goes to the centroid of largest cosine
    similarity, x_v . mu_m for unit mu_m; ties go to the lower cluster id.
    Everything in float64 from the exact inputs.  Returns (assign[V], S[V, M])."""
    X = unit_rows(W)
    S = X @ np.asarray(centroids, dtype=np.float64).T
    return np.argmax(_canonical(S), axis=1).astype(np.int64), S


def kmeans_update(W, assign, M: int, prev):
    """Update step: mu_m = sum of the unit points assigned to m, divided by
    its norm (the mean direction).  A cluster with no points (or a zero sum)
    keeps its previous centroid."""
    X = unit_rows(W)
    assign = np.asarray(assign, dtype=np.int64)
    mu = np.array(np.asarray(prev, dtype=np.float64), copy=True)
    for m in range(M):
        members = np.nonzero(assign == m)[0]
        if len(members) == 0:
            continue
        s = X[members].sum(axis=0)
        n = np.sqrt((s * s).sum())
        if n > 0:
            mu[m] = s / n
    return mu


def spherical_kmeans(W, M: int, init_ids, iters: int):
    """Spherical k-means on the unit LM-head rows: centroids start at the
    points init_ids (M distinct vocabulary ids, drawn by the caller), then
    `iters` rounds of assignment followed by update.  Returns the last
    assignment (the partition, cluster_of[V]) and the centroids after the
    last update."""
    X = unit_rows(W)
    mu = X[np.asarray(init_ids, dtype=np.int64)]
    assign = np.zeros(X.shape[0], dtype=np.int64)
    for _ in range(iters):
        assign, _ = kmeans_assign(W, mu)
        mu = kmeans_update(W, assign, M, mu)
    return assign, mu


def kmeans_objective(W, assign, centroids) -> float:
    """Sum over points of the cosine similarity to their own centroid."""
    X = unit_rows(W)
    mu = np.asarray(centroids, dtype=np.float64)
    return float((X * mu[np.asarray(assign, dtype=np.int64)]).sum())
