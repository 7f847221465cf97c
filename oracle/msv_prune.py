"""MSV-Prune (Sec. 4.1): multi-layer semantic visual token pruning, per tile.

Steps, in the order of Sec. 4.1 and Algorithm 1 (stage 1):

1. ``anchor_scores``  - Sec. 4.1.1: the ViT self-attention averaged over
   heads; for CLIP-like encoders the [CLS] row, one value per patch.
2. ``budget``         - Sec. 4.1.1 / 4.1.2: anchor budget n*R*r and
   complementary budget n*R*(1-r), as integers.
3. ``anchor_set``     - Eq. 1 read through Algorithm 1 ("top-nRr by attention
   score"): the k largest scores, ties to the lower patch index.
4. ``kmeans``         - Sec. 4.1.2 coarse clustering: Lloyd's K-means on the
   last-layer features of the non-anchor tokens.
5. ``quotas``         - Eq. 2: per-cluster quota.
6. ``complementary_scores`` - Eq. 3: pairwise multi-layer similarity S_ij
   (cosine of every tapped layer plus the two max-similarity-to-anchor
   terms), reduced to one score per token as its mean over the token's
   cluster.
7. ``select``         - Sec. 4.1.2: the N_k lowest-scoring tokens of each
   cluster, united with the anchors and put back in spatial order (Sec. 4.1).
8. ``assemble``       - Sec. 4.1 / Sec. 5 (AnyRes): kept rows of each tile,
   tiles in order, followed by the sample's text rows.

Readings where the paper is silent (each also listed in the design notes):
head-mean is a sequential float32 sum over heads then one division; the
anchor budget is floor(keep * r) with r rational; Eq. 1's threshold is the
exact top-k with ties to the lower index; K-means uses Euclidean distance on
the raw features, centroids initialised at rows floor(k*m/K), at most
``max_iter`` assignment passes with early exit, ties to the lower cluster,
empty clusters keep their centroid, and its decisions are taken in float32
(the kernel's precision); Eq. 2 rounds half to even, applies max(1, .) only
to non-empty clusters, clips to the cluster size and does not reconcile the
total; the per-token score is the mean of S_ij over its cluster (j = i
included); cosine with a zero vector is 0 and the anchor term is 0 when
there are no anchors.

Parity pins: anchors and selection against brute-force sorts and the Eq. 1
threshold set; K-means against scikit-learn's Lloyd with the same initial
centroids and against fixed-point properties; quotas against hand-worked
cases; scores against closed forms on constructed features (orthonormal and
collinear rows) and invariances (row scaling, permutation).
"""
from __future__ import annotations

import numpy as np


# --------------------------------------------------------------------------- 1
def anchor_scores(cls_attn_tile: np.ndarray, col0: int = 1, n: int | None = None) -> np.ndarray:
    """Head-averaged [CLS] attention per patch (Sec. 4.1.1).

    ``cls_attn_tile`` is [H, >= col0 + n] float32 (row 0 of each head's
    attention matrix).  Returns float32 [n]: a sequential float32 sum over
    heads h = 0..H-1 followed by a single IEEE division by H.
    """
    A = np.asarray(cls_attn_tile, dtype=np.float32)
    H = A.shape[0]
    if n is None:
        n = A.shape[1] - col0
    acc = np.zeros(n, dtype=np.float32)
    for h in range(H):
        acc = (acc + A[h, col0:col0 + n]).astype(np.float32)
    return (acc / np.float32(H)).astype(np.float32)


def cls_attention(q_cls: np.ndarray, keys: np.ndarray, scale: float) -> np.ndarray:
    """The [CLS] row of a ViT layer's self-attention rebuilt from its query and
    keys, for encoders that never store attention maps (Sec. 4.1.1 reads this
    row): per head h, softmax over tokens j of scale * q_cls[h] . keys[j, h].

    ``q_cls`` is [H, dh], ``keys`` [T, H, dh] (token 0 = [CLS]).  Returns
    float64 [H, T]; anchor_scores() then averages it over heads.
    """
    q = np.asarray(q_cls, dtype=np.float64)
    k = np.asarray(keys, dtype=np.float64)
    z = np.einsum("hc,jhc->hj", q, k) * float(scale)
    z = z - z.max(axis=1, keepdims=True)
    e = np.exp(z)
    return e / e.sum(axis=1, keepdims=True)


def anchor_scores_colmean(attn_tile: np.ndarray) -> np.ndarray:
    """Anchor scores of an encoder without [CLS] (Sec. 4.1.1): the attention each
    patch receives, averaged over heads and over the patches attending to it.

    ``attn_tile`` is [H, n, n] (head, query patch, key patch).  Returns float64
    [n]: a[j] = mean over h and i of attn[h, i, j].
    """
    A = np.asarray(attn_tile, dtype=np.float64)
    return A.mean(axis=(0, 1))


# --------------------------------------------------------------------------- 2
def budget_ratio(n: int, rv_num: int, rv_den: int, r_num: int = 7, r_den: int = 10):
    """Budgets from a retention ratio R_v of an input-dependent token count (the
    Qwen3-VL setting of the appendix): keep = floor(n * R_v), then budget(keep).
    Exact rational arithmetic; returns (keep, k_anc, n_cmp)."""
    if n < 0 or rv_den <= 0 or rv_num < 0 or rv_num > rv_den:
        raise ValueError("bad ratio arguments")
    keep = (n * rv_num) // rv_den
    k_anc, n_cmp = budget(keep, r_num, r_den)
    return keep, k_anc, n_cmp


def budget(keep: int, r_num: int = 7, r_den: int = 10):
    """Anchor and complementary budgets (Sec. 4.1.1-4.1.2): k = floor(keep*r), keep - k."""
    if keep < 0 or r_den <= 0 or r_num < 0 or r_num > r_den:
        raise ValueError("bad budget arguments")
    k_anc = (keep * r_num) // r_den
    return k_anc, keep - k_anc


# --------------------------------------------------------------------------- 3
def _canon(v: float) -> float:
    if v != v:
        raise ValueError("NaN attention score")
    return 0.0 if v == 0.0 else float(v)


def anchor_set(a: np.ndarray, k: int) -> list:
    """Top-k patch indices by score, ties to the lower index (Eq. 1 / Alg. 1)."""
    n = len(a)
    order = sorted(range(n), key=lambda i: (-_canon(a[i]), i))
    return sorted(order[:k])


def threshold_set(a: np.ndarray, k: int) -> list:
    """Eq. 1 literally: tau = the smallest attained value t with |{a_i >= t}| <= k.

    Equals ``anchor_set`` whenever no tie straddles the budget; used as a
    cross-check of the top-k reading on distinct values.
    """
    vals = sorted(set(float(v) for v in a))
    ok = [t for t in vals if sum(1 for v in a if v >= t) <= k]
    if not ok:
        return []
    tau = min(ok)
    return [i for i in range(len(a)) if a[i] >= tau]


# --------------------------------------------------------------------------- 4
def kmeans(X: np.ndarray, K: int, max_iter: int):
    """Lloyd's K-means on the rows of X (Sec. 4.1.2, coarse clustering).

    Distances and centroid means are float32.  Returns (assign [m] int,
    centroids [K, d] float32, passes, margin [m]) where ``margin`` is the
    relative gap between the nearest and second-nearest centroid distance of
    each row at the final pass (how far the decision is from a tie).
    """
    X = np.asarray(X, dtype=np.float32)
    m = X.shape[0]
    if m == 0:
        return np.zeros(0, dtype=np.int64), np.zeros((K, X.shape[1]), np.float32), 0, np.zeros(0)
    if max_iter < 1:
        raise ValueError("max_iter must be >= 1")
    c = X[[(k * m) // K for k in range(K)]].copy()
    assign = None
    passes = 0
    d2 = None
    for _ in range(max_iter):
        d2 = ((X[:, None, :] - c[None, :, :]) ** 2).sum(axis=-1, dtype=np.float32)
        new = np.argmin(d2, axis=1)            # first minimum: lower cluster wins ties
        passes += 1
        if assign is not None and np.array_equal(new, assign):
            break
        assign = new
        for k in range(K):
            members = X[assign == k]
            if len(members):
                c[k] = (members.sum(axis=0, dtype=np.float32) / np.float32(len(members))).astype(np.float32)
    srt = np.sort(d2, axis=1)
    if K > 1:
        margin = (srt[:, 1] - srt[:, 0]) / np.maximum(srt[:, 1], 1e-30)
    else:
        margin = np.full(m, np.inf)
    return assign.astype(np.int64), c, passes, margin


# --------------------------------------------------------------------------- 5
def _rne_div(p: int, q: int) -> int:
    """round(p / q), halves to even, exact in integers (p >= 0, q > 0)."""
    t, r = divmod(p, q)
    if 2 * r > q or (2 * r == q and (t & 1)):
        t += 1
    return t


def quotas(sizes, n_cmp: int, mode: str = "literal") -> list:
    """Per-cluster quota N_k (Eq. 2).

    literal: N_k = max(1, round(n_cmp*|C_k| / sum|C_j|)) for non-empty clusters,
             0 for empty ones, clipped to |C_k|; the total is not reconciled.
    exact:   largest-remainder apportionment of exactly n_cmp (ties to the
             lower cluster), clipped to |C_k| (a variant that fixes the budget).
    """
    sizes = [int(s) for s in sizes]
    D = sum(sizes)
    if n_cmp <= 0 or D == 0:
        return [0] * len(sizes)
    if mode == "literal":
        return [0 if s == 0 else min(s, max(1, _rne_div(n_cmp * s, D))) for s in sizes]
    if mode == "exact":
        n_cmp = min(n_cmp, D)
        base = [(n_cmp * s) // D for s in sizes]
        rem = [(n_cmp * s) % D for s in sizes]
        left = n_cmp - sum(base)
        order = sorted(range(len(sizes)), key=lambda k: (-rem[k], k))
        for k in order[:left]:
            base[k] += 1
        return [min(b, s) for b, s in zip(base, sizes)]
    raise ValueError(mode)


# --------------------------------------------------------------------------- 6
def _unit_rows(F: np.ndarray) -> np.ndarray:
    F = np.asarray(F, dtype=np.float64)
    nrm = np.sqrt((F * F).sum(axis=1))
    out = np.zeros_like(F)
    nz = nrm > 0
    out[nz] = F[nz] / nrm[nz, None]
    return out


def anchor_max_similarity(F_last: np.ndarray, anchors) -> np.ndarray:
    """max over anchors p of cos(F^L_i, F^L_p) for every token i (the anchor term of Eq. 3)."""
    U = _unit_rows(F_last)
    anchors = list(anchors)
    if not anchors:
        return np.zeros(U.shape[0])
    return (U @ U[anchors].T).max(axis=1)


def complementary_scores(feats, anchors, cluster: np.ndarray):
    """Per-token score from the pairwise multi-layer similarity of Eq. 3.

    ``feats`` is the list of tapped-layer features [n, d] (patch rows only),
    the last entry being F^L.  For tokens i, j of the same cluster:

        S_ij = sum_l cos(F^l_i, F^l_j) + max_p cos(F^L_i, F^L_p) + max_p cos(F^L_j, F^L_p)

    and the token score is the mean of S_ij over j in the cluster.  Returns
    (s [n] float64 with +inf for anchors, mvec [n] anchor-max similarity).
    """
    n = len(cluster)
    units = [_unit_rows(F) for F in feats]
    mvec = anchor_max_similarity(feats[-1], anchors)
    s = np.full(n, np.inf)
    for k in sorted(set(int(c) for c in cluster if c >= 0)):
        C = np.nonzero(cluster == k)[0]
        S = np.zeros((len(C), len(C)))
        for U in units:
            S += U[C] @ U[C].T
        S += mvec[C][:, None] + mvec[C][None, :]
        s[C] = S.mean(axis=1)
    return s, mvec


# --------------------------------------------------------------------------- 7
def select(cluster: np.ndarray, s32: np.ndarray, n_cmp: int, K: int, mode: str = "literal"):
    """Anchors plus the N_k lowest-scoring tokens of every cluster, in spatial order.

    ``cluster`` is [n] with -1 for anchors; ``s32`` the float32 scores used for
    the ranking (ties to the lower index).  Returns (idx ascending, N list).
    """
    cluster = np.asarray(cluster)
    s32 = np.asarray(s32, dtype=np.float32)
    anchors = [int(i) for i in np.nonzero(cluster < 0)[0]]
    sizes = [int((cluster == k).sum()) for k in range(K)]
    N = quotas(sizes, n_cmp, mode)
    chosen = []
    for k in range(K):
        members = [int(i) for i in np.nonzero(cluster == k)[0]]
        members.sort(key=lambda i: (float(s32[i]) if s32[i] != 0 else 0.0, i))
        chosen += members[:N[k]]
    return sorted(anchors + chosen), N


# --------------------------------------------------------------------------- tile
def prune_tile(cls_attn_tile, feats_tile, keep: int, r_num: int = 7, r_den: int = 10,
               K: int = 4, max_iter: int = 10, mode: str = "literal", col0: int = 1,
               row0: int = 1, cluster_override=None, a=None):
    """Whole MSV-Prune for one tile (Alg. 1, stage 1).

    ``feats_tile``: list of [row0 + n, d] arrays, last = F^L.  Returns a dict
    with a, anchors, cluster (-1 = anchor), s (float64, +inf for anchors),
    s32, mvec, kmeans margin, quotas, idx (ascending kept patch indices).
    ``cluster_override`` replaces the K-means assignment of the non-anchor
    tokens (used to score a known clustering).  ``a`` (length n) replaces the
    [CLS] anchor scores (e.g. anchor_scores_colmean for encoders without
    [CLS]); ``cls_attn_tile`` is then not read.
    """
    feats = [np.asarray(F, dtype=np.float64)[row0:] for F in feats_tile]
    n = feats[0].shape[0]
    a = anchor_scores(cls_attn_tile, col0, n) if a is None else np.asarray(a, np.float64)
    k_anc, n_cmp = budget(keep, r_num, r_den)
    k_anc = min(k_anc, n)
    anchors = anchor_set(a, k_anc)
    is_anchor = np.zeros(n, dtype=bool)
    is_anchor[anchors] = True
    U = np.nonzero(~is_anchor)[0]
    cluster = np.full(n, -1, dtype=np.int64)
    margin = np.zeros(0)
    # The clustering runs whenever there are non-anchor tokens (with a zero
    # complementary budget every quota is simply 0).
    if len(U):
        if cluster_override is not None:
            cluster[U] = np.asarray(cluster_override)[U]
        else:
            X = np.asarray(feats_tile[-1], dtype=np.float32)[row0:][U]
            assign, _, _, margin = kmeans(X, K, max_iter)
            cluster[U] = assign
    s, mvec = complementary_scores(feats, anchors, cluster)
    s32 = s.astype(np.float32)
    idx, N = select(cluster, s32, n_cmp, K, mode)
    return dict(a=a, anchors=anchors, cluster=cluster, s=s, s32=s32, mvec=mvec,
                margin=margin, quotas=N, idx=idx, k_anc=k_anc, n_cmp=n_cmp)


# --------------------------------------------------------------------------- 8
def assemble(src: np.ndarray, idx_per_tile, text: np.ndarray, tiles_per_sample: int):
    """Decoder input rows: per sample, kept rows of its tiles (tile order) then its text rows.

    ``src`` [G, n, d]; ``text`` [B, n_text, d].  Returns (x [rows, d], cu_seqlens [B+1]).
    """
    G = src.shape[0]
    B = G // tiles_per_sample
    rows, cu = [], [0]
    for b in range(B):
        for t in range(tiles_per_sample):
            g = b * tiles_per_sample + t
            rows.append(src[g][list(idx_per_tile[g])])
        rows.append(text[b])
        cu.append(cu[-1] + sum(len(idx_per_tile[b * tiles_per_sample + t])
                               for t in range(tiles_per_sample)) + text.shape[1])
    return np.concatenate(rows, axis=0), np.array(cu, dtype=np.int64)
