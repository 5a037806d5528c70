"""Plain, slow, float64 CPU oracle of the PQ-HSA decode-attention operator.

TEST INFRASTRUCTURE ONLY. This module is the reference that the HIP path is
checked against. Only the test suite, the package smoke check and the CPU
baseline leg of the benchmark may import it; the product path never calls it
and shares no code with it (no kernels, headers, tables or helpers).

Everything is written from the paper's statement of the method:

* Section 3 (opening paragraph), Eq. (1): dense decode attention and the
  exact/background decomposition y = (N_E + N_B) / (Z_E + Z_B).
* Section 3.1, Eq. (2): direction-norm residual IVF-PQ score of an indexed
  key, computed from a per-query lookup table (LUT) over the M subspaces plus
  the coarse term u_q . c_{a_i}.
* Section 3.2, Eq. (3): partition into sink prefix S, local window L and
  indexed region R; top-k selection T over R; E = S u L u T, B = R \\ T.
* Section 3.2, Eq. (4): per-list background masses M_j over B n R_j and the
  list value means; Eq. (5): the output.
* Appendix A ("Budgets"): 4 sinks, a 128-token local window, k = ceil(rho |R|)
  and the exact-set size rounded up to whole pages of 16 tokens.
* Section 3.1 (the index): a key k = r u is stored as its norm r, the list
  a of the centroid nearest to its direction u, and the codes of the
  residual u - c_a, the nearest codeword in each of the M subspaces
  (`encode_ref`). Section 3.3 (execution path): later tokens are encoded
  into the existing lists without re-clustering, and each update refreshes
  the list means (`update_ref`).
* Section 3.3 and Appendix "Index build": the index of each KV head is
  built from its keys' directions by k-means, one coarse problem over the
  directions and one problem per PQ subspace over the residual slices, with
  key norms kept apart and empty clusters re-seeded (`kmeans_ref`,
  `build_ref`; the paper's setting is one coarse and two PQ iterations).
* Appendix B (variant definitions, Table "mechanism variants"): variants T
  (no background), C (token-weighted global value mean) and Bx (mean of the
  unselected members of each list).

Readings where the paper is silent:
* the top-k tie-break is the smaller token id;
* r_q = 0 gives a score of 0 for every indexed token;
* an empty list, or a list whose members are all selected, contributes 0;
* "nearest" is the smallest squared Euclidean distance, ties going to the
  smaller list id or codeword index; a zero key has r = 0 and u = 0;
* an update from n_old to n_new tokens indexes the tokens that leave the
  local window, [max(n_sink, n_old - n_local), n_new - n_local);
* k-means starts from given data points (the caller draws them); one
  iteration assigns every point to its nearest center, then moves each
  center to the mean of its points; a center left without points takes the
  point farthest from its own center in that assignment (the farthest
  first, ties to the smaller index, one point per empty center in
  increasing center id);
* the build trains the coarse centers on the directions of R, assigns,
  trains each subspace's codewords on the residual slices starting from the
  residuals of given tokens, and ends with `encode_ref` against the trained
  model and the list means of the final lists.

Each function is pinned in tests/test_oracle_pins.py to something other
than itself:
* budget_paper: the budgets the paper prints (Appendix A);
* lut_ref, pq_scores_ref: explicit key reconstruction, exact-reconstruction
  keys, a zero query;
* topk_ref: brute-force ranking and exhaustive subsets;
* dense_attention_ref: torch's attention routine in float64, whole and
  truncated caches;
* list_means_ref: brute-force means;
* pqhsa_row_ref: rho = 1 against library attention, closed forms under exact
  reconstruction, the pseudo-token form of pure background, the variants'
  special cases, invariances, an mpmath re-evaluation;
* pqhsa_batch_ref: library attention with grouped query heads over ragged
  sequences (at rho = 1, and for any k under exact reconstruction with
  list-constant values);
* encode_ref, update_ref: scipy's vector quantizer, an exactly representable
  key, norm scaling, update composition;
* kmeans_ref: scipy's kmeans2, a brute-force re-seed;
* build_ref: zero-iteration closed forms, and scipy's kmeans2 for the coarse
  centers and for the codewords on residual slices the test forms itself.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "budget_paper",
    "split_positions",
    "lut_ref",
    "pq_scores_ref",
    "topk_ref",
    "dense_attention_ref",
    "list_means_ref",
    "pqhsa_row_ref",
    "pqhsa_batch_ref",
    "RowResult",
    "Encoding",
    "encode_ref",
    "update_ref",
    "kmeans_ref",
    "build_ref",
]


# ---------------------------------------------------------------------------
# Budget rule (Appendix A, "Budgets"; Section 3.2 for k = ceil(rho |R|)).
# ---------------------------------------------------------------------------
def budget_paper(n_ctx: int, rho: float, n_sink: int = 4, n_local: int = 128,
                 page: int = 16) -> tuple[int, int]:
    """Return (k, exact-set size rounded up to whole pages).

    |R| = n_ctx - n_sink - n_local, k = ceil(rho |R|) (Section 3.2), and the
    exact set S u L u T has n_sink + n_local + k tokens, rounded up to a
    multiple of `page` tokens (Appendix A).
    """
    n_r = n_ctx - n_sink - n_local
    if n_r < 0:
        raise ValueError("context shorter than sink + local window")
    # ceil of a decimal fraction without binary round-up surprises
    k = int(math.ceil(round(rho * n_r, 9)))
    exact = n_sink + n_local + k
    rounded = -(-exact // page) * page
    return k, rounded


def split_positions(n_seq: int, n_sink: int, n_local: int):
    """Sink prefix S, local window L and indexed region R (Section 3.2).

    S = [0, n_sink), L = [n_seq - n_local, n_seq), R = the positions between.
    """
    if n_seq < n_sink + n_local:
        raise ValueError("n_seq must be at least n_sink + n_local")
    S = np.arange(0, n_sink)
    L = np.arange(n_seq - n_local, n_seq)
    R = np.arange(n_sink, n_seq - n_local)
    return S, L, R


# ---------------------------------------------------------------------------
# Eq. (2): LUT and approximate logits.
# ---------------------------------------------------------------------------
def lut_ref(q: np.ndarray, centroids: np.ndarray, codebooks: np.ndarray):
    """Query norm, coarse table and fine LUT of Eq. (2).

    q [d]; centroids [n_list, d]; codebooks [M, ksub, d/M].
    Returns r_q = ||q||, coarse[j] = u_q . c_j and fine[m, z] = u_q^(m) . p_{m,z}
    where u_q = q / r_q and u_q^(m) is the m-th contiguous sub-vector of u_q.
    """
    q = np.asarray(q, dtype=np.float64)
    d = q.shape[0]
    n_m, ksub, dsub = codebooks.shape
    if n_m * dsub != d:
        raise ValueError("codebook subspaces do not tile the head dimension")
    r_q = float(np.sqrt(np.sum(q * q)))
    if r_q == 0.0:
        # reading: a zero query has no direction; every PQ score is 0
        return 0.0, np.zeros(centroids.shape[0]), np.zeros((n_m, ksub))
    u_q = q / r_q
    coarse = np.asarray(centroids, np.float64) @ u_q
    fine = np.empty((n_m, ksub))
    for m in range(n_m):
        sub = u_q[m * dsub:(m + 1) * dsub]
        fine[m] = np.asarray(codebooks[m], np.float64) @ sub
    return r_q, coarse, fine


def pq_scores_ref(q, list_ids, codes, norms, centroids, codebooks, positions):
    """Approximate logits of Eq. (2) for the given token positions.

    l~_i = (r_q r_i / sqrt(d)) (u_q . c_{a_i} + sum_m u_q^(m) . p_{m, z_im}),
    evaluated as one LUT lookup per subspace. list_ids [N] (a_i), codes [N, M]
    (z_im), norms [N] (r_i).
    """
    d = np.asarray(q).shape[0]
    r_q, coarse, fine = lut_ref(q, centroids, codebooks)
    positions = np.asarray(positions, dtype=np.int64)
    a = np.asarray(list_ids)[positions].astype(np.int64)
    z = np.asarray(codes)[positions].astype(np.int64)          # [n, M]
    r = np.asarray(norms, np.float64)[positions]
    n_m = fine.shape[0]
    total = coarse[a].copy()
    for m in range(n_m):
        total += fine[m, z[:, m]]
    return (r_q * r / math.sqrt(d)) * total


def topk_ref(scores: np.ndarray, token_ids: np.ndarray, k: int):
    """T = TopK_k over R (Eq. 3); ties go to the smaller token id.

    Returns (selected token ids sorted ascending, tau = k-th largest score or
    None when k = 0).
    """
    scores = np.asarray(scores, np.float64)
    token_ids = np.asarray(token_ids, np.int64)
    if not 0 <= k <= scores.shape[0]:
        raise ValueError("k out of range")
    order = np.lexsort((token_ids, -scores))   # primary: score desc; then id asc
    chosen = order[:k]
    tau = float(scores[order[k - 1]]) if k > 0 else None
    return np.sort(token_ids[chosen]), tau


# ---------------------------------------------------------------------------
# Dense attention (Section 3, opening paragraph).
# ---------------------------------------------------------------------------
def dense_attention_ref(q, K, V, n_seq: int | None = None):
    """y = sum_i e_i v_i / sum_i e_i with e_i = exp(q . k_i / sqrt(d))."""
    q = np.asarray(q, np.float64)
    K = np.asarray(K, np.float64)
    V = np.asarray(V, np.float64)
    if n_seq is not None:
        K, V = K[:n_seq], V[:n_seq]
    d = q.shape[0]
    logits = K @ q / math.sqrt(d)
    m0 = logits.max()
    e = np.exp(logits - m0)
    return (e @ V) / e.sum()


def list_means_ref(V, list_ids, n_list: int, R: np.ndarray):
    """v_bar_j = mean of v_i over R_j = {i in R : a_i = j} (Eq. 4); 0 if empty."""
    V = np.asarray(V, np.float64)
    a = np.asarray(list_ids)[R].astype(np.int64)
    sums = np.zeros((n_list, V.shape[1]))
    np.add.at(sums, a, V[R])
    cnt = np.bincount(a, minlength=n_list).astype(np.float64)
    means = np.zeros_like(sums)
    nz = cnt > 0
    means[nz] = sums[nz] / cnt[nz, None]
    return means


# ---------------------------------------------------------------------------
# Encoding keys into the existing index (Section 3.1) and the incremental
# update (Section 3.3).
# ---------------------------------------------------------------------------
def sq_dists(X, C):
    """Squared Euclidean distances ||x - c||^2 of every row of X [n, dim] to
    every row of C [k, dim], as ||x||^2 - 2 x . c + ||c||^2 with one matrix
    product per block of rows (float64; a negative rounding residue is set
    to 0)."""
    X = np.asarray(X, np.float64)
    C = np.asarray(C, np.float64)
    cc = (C * C).sum(axis=1)
    out = np.empty((X.shape[0], C.shape[0]))
    for s in range(0, X.shape[0], 8192):
        x = X[s:s + 8192]
        d2 = out[s:s + 8192]
        np.matmul(x, C.T, out=d2)
        d2 *= -2.0
        d2 += (x * x).sum(axis=1)[:, None]
        d2 += cc[None, :]
        np.maximum(d2, 0.0, out=d2)
    return out


@dataclass
class Encoding:
    a: np.ndarray          # [n] list id
    z: np.ndarray          # [n, M] code per subspace
    r: np.ndarray          # [n] key norm
    coarse_d2: np.ndarray  # [n, n_list] ||u - c_j||^2
    fine_d2: np.ndarray    # [n, M, K] ||(u - c_a)^(m) - p_{m,z}||^2


def encode_ref(keys, centroids, codebooks, tables: bool = True) -> Encoding:
    """Direction-norm residual IVF-PQ encoding of keys [n, d] (Section 3.1).

    r = ||k||, u = k / r; a = the list whose centroid is nearest to u; then
    for each subspace m the codeword nearest to the m-th slice of u - c_a.
    The distance tables are returned for validity checks of other encoders
    (None for both when tables=False, which keeps only the choices).
    """
    K = np.asarray(keys, np.float64)
    C = np.asarray(centroids, np.float64)
    P = np.asarray(codebooks, np.float64)
    n, d = K.shape
    M, ksub, dsub = P.shape
    r = np.sqrt((K * K).sum(axis=1))
    u = np.zeros_like(K)
    nz = r > 0
    u[nz] = K[nz] / r[nz, None]
    coarse = sq_dists(u, C)
    a = coarse.argmin(axis=1)            # the first minimum: the smaller id
    res = (u - C[a]).reshape(n, M, dsub)
    fine = np.empty((n, M, ksub)) if tables else None
    z = np.empty((n, M), np.int64)
    for m in range(M):
        dm = sq_dists(res[:, m, :], P[m])
        z[:, m] = dm.argmin(axis=1)
        if tables:
            fine[:, m, :] = dm
    return Encoding(a=a, z=z, r=r, coarse_d2=coarse if tables else None, fine_d2=fine)


def update_ref(list_ids, codes, norms, K, V, n_old: int, n_new: int, n_sink: int,
               n_local: int, centroids, codebooks):
    """Grow one (sequence, KV head) index from n_old to n_new cached tokens.

    list_ids [>= n_new], codes [>= n_new, M], norms [>= n_new]: the current
    token-major index (entries outside R ignored); K, V [>= n_new, d]. The
    tokens leaving the local window join R, encoded with `encode_ref` against
    the existing centroids and codebooks; the list means become the means
    over the grown lists. Returns (list_ids, codes, norms, list_means,
    Encoding of the new tokens) as new arrays.
    """
    if n_new < n_old:
        raise ValueError("an update cannot shrink the sequence")
    lo = max(n_sink, n_old - n_local)
    hi = max(n_sink, n_new - n_local)
    ids = np.array(list_ids, np.int64, copy=True)
    cds = np.array(codes, np.int64, copy=True)
    nrm = np.array(norms, np.float64, copy=True)
    enc = encode_ref(np.asarray(K, np.float64)[lo:hi], centroids, codebooks)
    ids[lo:hi] = enc.a
    cds[lo:hi] = enc.z
    nrm[lo:hi] = enc.r
    R = split_positions(n_new, n_sink, n_local)[2]
    means = list_means_ref(V, ids, np.asarray(centroids).shape[0], R)
    return ids, cds, nrm, means, enc


def kmeans_ref(X, init_idx, n_iter: int):
    """Lloyd's k-means on the rows of X [n, dim] from centers X[init_idx].

    Each iteration: nearest center of every point (squared distance, ties to
    the smaller center id), then each center becomes the mean of its points;
    centers without points are re-seeded with the points farthest from their
    assigned centers. Returns the centers [k, dim].
    """
    X = np.asarray(X, np.float64)
    C = X[np.asarray(init_idx, np.int64)].copy()
    n, k = X.shape[0], C.shape[0]
    for _ in range(n_iter):
        d2 = sq_dists(X, C)
        a = d2.argmin(axis=1)
        dmin = d2[np.arange(n), a]
        cnt = np.bincount(a, minlength=k)
        sums = np.zeros_like(C)
        np.add.at(sums, a, X)
        newC = C.copy()
        nz = cnt > 0
        newC[nz] = sums[nz] / cnt[nz, None]
        empty = np.flatnonzero(cnt == 0)
        if empty.size:
            far = np.lexsort((np.arange(n), -dmin))   # farthest first, then smaller index
            for e, j in enumerate(empty):
                newC[j] = X[far[e]]
        C = newC
    return C


def build_ref(K, V, R, n_list: int, M: int, ksub: int, init_coarse, init_pq,
              n_iter_coarse: int = 1, n_iter_pq: int = 2):
    """Build one (sequence, KV head) index from its keys over R.

    K, V [>= max(R) + 1, d]; R the indexed token ids; init_coarse [n_list] and
    init_pq [M, ksub] token ids of R whose direction (coarse) or residual
    slice (subspace m) starts each center. Returns a dict with token-major
    list_ids, codes, norms (entries outside R zero), centroids [n_list, d],
    codebooks [M, ksub, d/M] and list_means [n_list, d].
    """
    K = np.asarray(K, np.float64)
    R = np.asarray(R, np.int64)
    n_tok, d = K.shape
    ds = d // M
    r = np.sqrt((K[R] ** 2).sum(axis=1))
    U = np.zeros((R.size, d))
    nz = r > 0
    U[nz] = K[R][nz] / r[nz, None]
    pos = {int(t): i for i, t in enumerate(R)}
    C = kmeans_ref(U, [pos[int(t)] for t in init_coarse], n_iter_coarse)
    a = encode_ref(K[R], C, np.zeros((M, 1, ds)), tables=False).a
    res = U - C[a]
    P = np.stack([kmeans_ref(res[:, m * ds:(m + 1) * ds],
                             [pos[int(t)] for t in np.asarray(init_pq)[m]], n_iter_pq)
                  for m in range(M)])
    enc = encode_ref(K[R], C, P, tables=False)
    ids = np.zeros(n_tok, np.int64)
    codes = np.zeros((n_tok, M), np.int64)
    norms = np.zeros(n_tok)
    ids[R], codes[R], norms[R] = enc.a, enc.z, enc.r
    means = list_means_ref(V, ids, n_list, R)
    return dict(list_ids=ids, codes=codes, norms=norms, centroids=C, codebooks=P,
                list_means=means, encoding=enc)


# ---------------------------------------------------------------------------
# The operator, one query row (Section 3.2, Eqs. 3-5).
# ---------------------------------------------------------------------------
@dataclass
class RowResult:
    y: np.ndarray                 # output [d]
    T: np.ndarray                 # selected token ids (sorted)
    tau: float | None             # k-th largest approximate logit
    scores: np.ndarray            # approximate logits over R (aligned with R)
    R: np.ndarray                 # indexed token ids
    m0: float                     # common shift
    Z_E: float
    Z_B: float
    list_size: np.ndarray         # |R_j|
    unselected_per_list: np.ndarray  # |B n R_j|
    extra: dict = field(default_factory=dict)


def pqhsa_row_ref(q, K, V, list_ids, codes, norms, centroids, codebooks,
                  list_means, n_seq: int, n_sink: int, n_local: int, k: int,
                  variant: str = "B", force_T=None) -> RowResult:
    """PQ-HSA output for one query head against its KV head.

    q [d]; K, V [>= n_seq, d]; list_ids [>= n_seq]; codes [>= n_seq, M];
    norms [>= n_seq]; centroids [n_list, d]; codebooks [M, ksub, d/M];
    list_means [n_list, d]. Index entries outside R are ignored.

    variant: "B" (PQ-HSA, Eq. 5), "T" (background dropped), "C" (background
    values = token-weighted global value mean over R), "Bx" (background values
    = mean of the unselected members of each list, Appendix B).
    force_T: evaluate Eqs. 3-5 with this selected set instead of the top-k.
    """
    q = np.asarray(q, np.float64)
    d = q.shape[0]
    n_list = centroids.shape[0]
    S, L, R = split_positions(n_seq, n_sink, n_local)

    # Eq. (2): one approximate logit per indexed token
    scores = pq_scores_ref(q, list_ids, codes, norms, centroids, codebooks, R)

    # Eq. (3): selection over R only
    if force_T is None:
        T, tau = topk_ref(scores, R, k)
    else:
        T = np.sort(np.asarray(force_T, np.int64))
        if T.shape[0] != k or not np.all(np.isin(T, R)):
            raise ValueError("force_T must hold k distinct indexed positions")
        tau = None
    in_T = np.isin(R, T)
    B_ids = R[~in_T]
    B_scores = scores[~in_T]
    E_ids = np.concatenate([S, L, T]).astype(np.int64)

    # exact logits replace the approximate ones on E
    Kf = np.asarray(K, np.float64)
    Vf = np.asarray(V, np.float64)
    exact = Kf[E_ids] @ q / math.sqrt(d)

    a_all = np.asarray(list_ids).astype(np.int64)
    a_B = a_all[B_ids]
    list_size = np.bincount(a_all[R], minlength=n_list)
    unsel = np.bincount(a_B, minlength=n_list)

    use_background = variant != "T"
    # common shift: maximum over exact (E) and approximate (B) logits
    cands = [exact.max()] if exact.size else []
    if use_background and B_scores.size:
        cands.append(B_scores.max())
    m0 = float(max(cands)) if cands else 0.0

    e_E = np.exp(exact - m0)
    Z_E = float(e_E.sum())
    N_E = e_E @ Vf[E_ids] if E_ids.size else np.zeros(d)

    if use_background and B_ids.size:
        e_B = np.exp(B_scores - m0)
        # Eq. (4): M_j = sum of e~_i over B n R_j (0 for an empty list)
        M = np.zeros(n_list)
        np.add.at(M, a_B, e_B)
        if variant == "B":
            vbar = np.asarray(list_means, np.float64)
        elif variant == "C":
            glob = Vf[R].mean(axis=0) if R.size else np.zeros(d)
            vbar = np.broadcast_to(glob, (n_list, d))
        elif variant == "Bx":
            lm = np.asarray(list_means, np.float64)
            sel_sum = np.zeros((n_list, d))
            np.add.at(sel_sum, a_all[T], Vf[T])
            vbar = np.zeros((n_list, d))
            nz = unsel > 0
            vbar[nz] = (list_size[nz, None] * lm[nz] - sel_sum[nz]) / unsel[nz, None]
        else:
            raise ValueError(f"unknown variant {variant!r}")
        Z_B = float(M.sum())
        N_B = M @ vbar
    else:
        Z_B = 0.0
        N_B = np.zeros(d)

    # Eq. (5)
    y = (N_E + N_B) / (Z_E + Z_B)
    return RowResult(y=y, T=T, tau=tau, scores=scores, R=R, m0=m0, Z_E=Z_E,
                     Z_B=Z_B, list_size=list_size, unselected_per_list=unsel)


def pqhsa_batch_ref(inp: dict, topk, rows=None, variant: str = "B", force_T=None):
    """Run the row oracle over (batch element, query head) pairs.

    inp holds numpy-convertible arrays with the ABI's layouts:
    q [B, Hq, d]; k_cache, v_cache [B, Hkv, Nmax, d]; list_ids [B, Hkv, Nmax];
    codes [B, Hkv, Nmax, M]; norms [B, Hkv, Nmax]; centroids [B, Hkv, n_list, d];
    codebooks [B, Hkv, M, ksub, d/M]; list_means [B, Hkv, n_list, d];
    seq_lens [B]; n_sink, n_local (ints). topk: int per batch element.
    Query head h reads KV head h // G with G = Hq / Hkv (Section 3.3).
    rows: iterable of (b, h); default all. force_T: optional {(b, h): token ids}.
    Arrays may be numpy arrays or torch tensors on any device (read-only).
    Returns {(b, h): RowResult}.
    """
    q = inp["q"]
    B, Hq, _ = q.shape
    seq_lens = _np(inp["seq_lens"])
    Hkv = inp["k_cache"].shape[1]
    G = Hq // Hkv
    if rows is None:
        rows = [(b, h) for b in range(B) for h in range(Hq)]
    out = {}
    cache = {}
    for b, h in rows:
        g = h // G
        key = (b, g)
        if key not in cache:
            cache.clear()
            n = int(seq_lens[b])
            cache[key] = dict(
                K=_f64(inp["k_cache"][b, g, :n]), V=_f64(inp["v_cache"][b, g, :n]),
                list_ids=_np(inp["list_ids"][b, g, :n]),
                codes=_np(inp["codes"][b, g, :n]),
                norms=_f64(inp["norms"][b, g, :n]),
                centroids=_f64(inp["centroids"][b, g]),
                codebooks=_f64(inp["codebooks"][b, g]),
                list_means=_f64(inp["list_means"][b, g]), n=n)
        c = cache[key]
        out[(b, h)] = pqhsa_row_ref(
            _f64(q[b, h]), c["K"], c["V"], c["list_ids"], c["codes"], c["norms"],
            c["centroids"], c["codebooks"], c["list_means"], c["n"],
            int(inp["n_sink"]), int(inp["n_local"]), int(_np(topk)[b]),
            variant=variant, force_T=None if force_T is None else force_T.get((b, h)))
    return out


def _f64(x):
    """Exact upcast of a numpy array or a torch tensor (bf16 included)."""
    if hasattr(x, "detach"):
        return x.detach().to("cpu").double().numpy()
    return np.asarray(x, np.float64)


def _np(x):
    """A numpy copy of a numpy array or a torch tensor on any device."""
    if hasattr(x, "detach"):
        return x.detach().to("cpu").numpy()
    return np.asarray(x)
