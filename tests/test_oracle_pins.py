"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a library
attention routine, an explicit key reconstruction, brute-force ranking,
closed forms that the method reduces to in special cases, invariances, and
the budget numbers the paper prints. A plausible mistake in the oracle (a
dropped coarse term, a wrong sub-vector index, a missing norm factor, a
selection off by one, a wrong shift or normaliser, the background counting
selected tokens) fails at least one of them.
"""

import itertools
import json
import math
import os

import mpmath
import numpy as np
import pytest
import scipy.special
import torch

from oracle import pqhsa_ref as R

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# small float64 problem builder (independent of the product's generator)
# ---------------------------------------------------------------------------
def tiny_problem(seed=0, n=64, d=16, n_m=4, ksub=8, n_list=5, noise=0.0,
                 norms="one", values="random", q_scale=1.0, empty_list=None):
    rng = np.random.default_rng(seed)
    dsub = d // n_m
    cen = rng.standard_normal((n_list, d))
    cb = 0.4 * rng.standard_normal((n_m, ksub, dsub))
    a = rng.integers(0, n_list, size=n)
    if empty_list is not None:
        a[a == empty_list] = (empty_list + 1) % n_list
    z = rng.integers(0, ksub, size=(n, n_m))
    recon = cen[a] + np.concatenate([cb[m, z[:, m]] for m in range(n_m)], axis=1)
    if norms == "one":
        r = np.ones(n)
    else:
        r = np.exp(rng.uniform(np.log(0.5), np.log(2.0), size=n))
    K = r[:, None] * (recon + noise * rng.standard_normal((n, d)))
    off = rng.standard_normal((n_list, d))
    if values == "list_constant":
        V = 0.5 * off[a]
    else:
        V = rng.standard_normal((n, d)) + 0.5 * off[a]
    q = q_scale * K[rng.integers(0, n)] + 0.3 * rng.standard_normal(d)
    return dict(q=q, K=K, V=V, a=a, z=z.astype(np.uint8), r=r, cen=cen, cb=cb,
                n_list=n_list)


def run(p, n_sink, n_local, k, means=None, variant="B", force_T=None):
    n = p["K"].shape[0]
    _, _, Rr = R.split_positions(n, n_sink, n_local)
    if means is None:
        means = R.list_means_ref(p["V"], p["a"], p["n_list"], Rr)
    return R.pqhsa_row_ref(p["q"], p["K"], p["V"], p["a"], p["z"], p["r"], p["cen"],
                           p["cb"], means, n, n_sink, n_local, k, variant=variant,
                           force_T=force_T)


def sdpa(q, K, V):
    """Dense attention by torch's library routine (float64, CPU)."""
    qt = torch.from_numpy(np.asarray(q, np.float64))[None, None, None, :]
    kt = torch.from_numpy(np.asarray(K, np.float64))[None, None]
    vt = torch.from_numpy(np.asarray(V, np.float64))[None, None]
    return torch.nn.functional.scaled_dot_product_attention(qt, kt, vt)[0, 0, 0].numpy()


def reconstructed_logits(p, positions):
    """q . k_hat_i / sqrt(d) with k_hat_i = r_i (c_{a_i} + concat_m p_{m, z_im})."""
    d = p["q"].shape[0]
    n_m = p["cb"].shape[0]
    out = []
    for i in positions:
        k_hat = np.concatenate([p["cb"][m, p["z"][i, m]] for m in range(n_m)])
        k_hat = p["r"][i] * (p["cen"][p["a"][i]] + k_hat)
        out.append(float(np.dot(p["q"], k_hat)) / math.sqrt(d))
    return np.array(out)


def close(a, b, tol=1e-12):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    scale = max(np.max(np.abs(b)), 1e-300)
    return np.max(np.abs(a - b)) / scale <= tol


# ---------------------------------------------------------------------------
# budget numbers printed in Appendix A
# ---------------------------------------------------------------------------
def test_budget_rule_reproduces_paper_numbers():
    with open(os.path.join(GOLDEN, "budget_paper.json")) as f:
        gold = json.load(f)
    for case in gold["cases"]:
        _, rounded = R.budget_paper(case["n_ctx"], case["rho"])
        if "exact_tokens" in case:
            assert rounded == case["exact_tokens"], case
        else:
            assert abs(rounded - case["exact_tokens_about"]) <= case["about_tolerance"]
        assert rounded % 16 == 0


# ---------------------------------------------------------------------------
# Eq. (2): LUT score == inner product with the explicitly reconstructed key
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("norms", ["one", "random"])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_scores_equal_reconstructed_key_logits(norms, seed):
    p = tiny_problem(seed=seed, n=80, d=32, n_m=8, ksub=16, n_list=6, noise=0.1,
                     norms=norms)
    pos = np.arange(80)
    s = R.pq_scores_ref(p["q"], p["a"], p["z"], p["r"], p["cen"], p["cb"], pos)
    assert close(s, reconstructed_logits(p, pos), 1e-12)


def test_scores_zero_query_are_zero():
    p = tiny_problem()
    s = R.pq_scores_ref(np.zeros(16), p["a"], p["z"], p["r"], p["cen"], p["cb"],
                        np.arange(10))
    assert np.all(s == 0.0)


def test_scores_with_exact_reconstruction_equal_exact_logits():
    p = tiny_problem(noise=0.0, norms="random")
    pos = np.arange(p["K"].shape[0])
    s = R.pq_scores_ref(p["q"], p["a"], p["z"], p["r"], p["cen"], p["cb"], pos)
    exact = p["K"] @ p["q"] / math.sqrt(p["q"].shape[0])
    assert close(s, exact, 1e-12)


# ---------------------------------------------------------------------------
# Eq. (3): top-k by brute force ranking, including exact ties
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(5))
def test_topk_matches_brute_force_rank(seed):
    rng = np.random.default_rng(seed)
    n = 30
    scores = rng.integers(0, 6, size=n).astype(np.float64)   # many exact ties
    ids = rng.permutation(1000)[:n]
    for k in range(n + 1):
        T, tau = R.topk_ref(scores, ids, k)
        brute = []
        for i in range(n):
            rank = sum(1 for j in range(n)
                       if scores[j] > scores[i] or (scores[j] == scores[i] and ids[j] < ids[i]))
            if rank < k:
                brute.append(ids[i])
        assert list(T) == sorted(brute)
        if k:
            assert tau == sorted(scores, reverse=True)[k - 1]


def test_topk_is_max_sum_subset_for_distinct_scores():
    rng = np.random.default_rng(7)
    scores = rng.standard_normal(10)
    ids = np.arange(10)
    for k in range(0, 11):
        T, _ = R.topk_ref(scores, ids, k)
        best = max(itertools.combinations(range(10), k), key=lambda c: sum(scores[list(c)]))
        assert list(T) == sorted(best)


def test_operator_selects_only_from_R_with_ties_to_smaller_id():
    p = tiny_problem(seed=3, n=40)
    # duplicate index entries -> identical approximate logits
    p["a"][10:20] = p["a"][10]
    p["z"][10:20] = p["z"][10]
    res = run(p, n_sink=4, n_local=8, k=5)
    assert np.all((res.T >= 4) & (res.T < 32))
    # brute-force rank on the oracle's own logits (ties -> smaller id)
    rank_sel = [i for i, s in zip(res.R, res.scores)
                if sum(1 for j, t in zip(res.R, res.scores) if t > s or (t == s and j < i)) < 5]
    assert list(res.T) == sorted(rank_sel)


# ---------------------------------------------------------------------------
# Eq. (5) special cases
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("n_sink,n_local", [(0, 0), (4, 8), (2, 0)])
def test_rho_one_is_dense_attention(n_sink, n_local):
    """Section 3.2: at rho = 1 the background is empty and Eq. 5 is dense."""
    p = tiny_problem(seed=11, n=50, noise=0.2, norms="random")
    n_r = 50 - n_sink - n_local
    res = run(p, n_sink, n_local, n_r)
    assert res.Z_B == 0.0
    assert close(res.y, sdpa(p["q"], p["K"], p["V"]), 1e-12)


@pytest.mark.parametrize("k", [0, 1, 7, 20, 42])
def test_exact_reconstruction_and_list_constant_values_is_dense(k):
    """l~ = l and v_i = v_bar_{a_i}: every background term is exact."""
    p = tiny_problem(seed=5, n=50, noise=0.0, values="list_constant", norms="random")
    res = run(p, 4, 4, k)
    assert close(res.y, sdpa(p["q"], p["K"], p["V"]), 1e-12)


@pytest.mark.parametrize("k", [0, 3, 15])
def test_exact_reconstruction_closed_form(k):
    """With l~ = l, Eq. 5 is dense attention whose background values are
    replaced by their list means."""
    p = tiny_problem(seed=9, n=60, noise=0.0, norms="random", q_scale=0.5)
    n_sink, n_local = 3, 5
    res = run(p, n_sink, n_local, k)
    _, _, Rr = R.split_positions(60, n_sink, n_local)
    means = R.list_means_ref(p["V"], p["a"], p["n_list"], Rr)
    V2 = p["V"].copy()
    for i in Rr:
        if i not in set(res.T.tolist()):
            V2[i] = means[p["a"][i]]
    assert close(res.y, sdpa(p["q"], p["K"], V2), 1e-12)


def test_pure_background_is_attention_over_list_pseudo_tokens():
    """k = 0, S = L = empty: softmax over lists with logit log sum_{R_j} e^{l~}
    and value v_bar_j (Eq. 4 with every token in B)."""
    p = tiny_problem(seed=21, n=70, noise=0.3, norms="random", n_list=6)
    res = run(p, 0, 0, 0)
    logits = reconstructed_logits(p, range(70))
    lse = np.array([scipy.special.logsumexp(logits[p["a"] == j]) if np.any(p["a"] == j)
                    else -np.inf for j in range(6)])
    w = scipy.special.softmax(lse)
    means = R.list_means_ref(p["V"], p["a"], 6, np.arange(70))
    assert close(res.y, w @ means, 1e-12)


def test_variant_T_is_softmax_over_exact_set():
    p = tiny_problem(seed=4, n=50, noise=0.2)
    res = run(p, 4, 6, 9, variant="T")
    E = np.concatenate([np.arange(4), np.arange(44, 50), res.T])
    assert close(res.y, sdpa(p["q"], p["K"][E], p["V"][E]), 1e-12)


def test_single_list_equals_global_mean_variant():
    p = tiny_problem(seed=8, n=50, noise=0.2, n_list=1)
    yb = run(p, 4, 6, 9).y
    yc = run(p, 4, 6, 9, variant="C").y
    assert close(yb, yc, 1e-12)


def test_unselected_mean_variant_on_list_constant_values():
    p = tiny_problem(seed=12, n=50, noise=0.2, values="list_constant")
    assert close(run(p, 4, 6, 9, variant="Bx").y, run(p, 4, 6, 9).y, 1e-12)


def test_unselected_mean_variant_brute_force():
    p = tiny_problem(seed=13, n=50, noise=0.2)
    res = run(p, 4, 6, 9, variant="Bx")
    B = [i for i in range(4, 44) if i not in set(res.T.tolist())]
    logits = {i: s for i, s in zip(res.R, res.scores)}
    E = list(range(4)) + list(range(44, 50)) + list(res.T)
    d = 16
    num = np.zeros(d)
    den = 0.0
    for i in E:
        e = math.exp(float(np.dot(p["q"], p["K"][i])) / 4.0)
        num += e * p["V"][i]
        den += e
    for i in B:
        members = [t for t in B if p["a"][t] == p["a"][i]]
        e = math.exp(logits[i])
        num += e * p["V"][members].mean(axis=0)
        den += e
    assert close(res.y, num / den, 1e-12)


# ---------------------------------------------------------------------------
# Eq. (4) boundary rules and per-token form
# ---------------------------------------------------------------------------
def test_background_per_token_form():
    """Sum over B of e~_i v_bar_{a_i} equals the per-list form (Eq. 4)."""
    p = tiny_problem(seed=31, n=64, noise=0.3, norms="random", q_scale=0.3)
    res = run(p, 2, 4, 10)
    Tset = set(res.T.tolist())
    d = 16
    means = R.list_means_ref(p["V"], p["a"], p["n_list"], np.arange(2, 60))
    num = np.zeros(d)
    den = 0.0
    for i in list(range(2)) + list(range(60, 64)) + sorted(Tset):
        e = math.exp(float(np.dot(p["q"], p["K"][i])) / 4.0)
        num += e * p["V"][i]
        den += e
    for i, s in zip(res.R, res.scores):
        if i not in Tset:
            e = math.exp(s)
            num += e * means[p["a"][i]]
            den += e
    assert close(res.y, num / den, 1e-12)
    assert close(res.Z_B / (res.Z_E + res.Z_B),
                 sum(math.exp(s) for i, s in zip(res.R, res.scores) if i not in Tset) / den,
                 1e-12)


def test_empty_list_contributes_nothing():
    p = tiny_problem(seed=14, n=50, noise=0.2, empty_list=2)
    _, _, Rr = R.split_positions(50, 4, 6)
    means = R.list_means_ref(p["V"], p["a"], p["n_list"], Rr)
    y0 = run(p, 4, 6, 7, means=means).y
    means2 = means.copy()
    means2[2] = 1e6
    assert np.array_equal(run(p, 4, 6, 7, means=means2).y, y0)


def test_fully_selected_list_contributes_nothing():
    p = tiny_problem(seed=15, n=50, noise=0.05, n_list=5)
    # aim the query at list 0's centroid so its members rank first
    p["q"] = 6.0 * p["cen"][0]
    _, _, Rr = R.split_positions(50, 4, 6)
    members = [i for i in Rr if p["a"][i] == 0]
    k = len(members) + 2
    means = R.list_means_ref(p["V"], p["a"], p["n_list"], Rr)
    res = run(p, 4, 6, k, means=means)
    assert set(members) <= set(res.T.tolist())
    assert res.unselected_per_list[0] == 0
    means2 = means.copy()
    means2[0] = -1e6
    assert np.array_equal(run(p, 4, 6, k, means=means2).y, res.y)


def test_value_shift_and_scale_equivariance():
    p = tiny_problem(seed=16, n=50, noise=0.3, q_scale=0.4)
    _, _, Rr = R.split_positions(50, 4, 6)
    means = R.list_means_ref(p["V"], p["a"], p["n_list"], Rr)
    y = run(p, 4, 6, 8, means=means).y
    w = np.linspace(-2, 3, 16)
    p2 = dict(p, V=p["V"] + w)
    assert close(run(p2, 4, 6, 8, means=means + w).y, y + w, 1e-12)
    p3 = dict(p, V=-2.5 * p["V"])
    assert close(run(p3, 4, 6, 8, means=-2.5 * means).y, -2.5 * y, 1e-12)


def test_permutation_of_indexed_tokens():
    """Reordering the indexed region (with its index entries) leaves y alone."""
    p = tiny_problem(seed=17, n=50, noise=0.3, norms="random")
    y = run(p, 4, 6, 9).y
    perm = np.arange(50)
    rng = np.random.default_rng(0)
    perm[4:44] = 4 + rng.permutation(40)
    p2 = {k: (v[perm] if isinstance(v, np.ndarray) and v.shape[:1] == (50,) else v)
          for k, v in p.items()}
    assert close(run(p2, 4, 6, 9).y, y, 1e-12)


def test_list_means_helper_brute_force():
    p = tiny_problem(seed=18, n=40)
    Rr = np.arange(3, 35)
    means = R.list_means_ref(p["V"], p["a"], p["n_list"], Rr)
    for j in range(p["n_list"]):
        mem = [i for i in Rr if p["a"][i] == j]
        ref = p["V"][mem].mean(axis=0) if mem else np.zeros(16)
        assert np.allclose(means[j], ref, rtol=1e-14, atol=1e-14)


# ---------------------------------------------------------------------------
# precision: the float64 oracle against 50-digit arithmetic on tiny inputs
# ---------------------------------------------------------------------------
def test_float64_oracle_against_mpmath():
    mpmath.mp.dps = 50
    p = tiny_problem(seed=19, n=24, d=8, n_m=2, ksub=4, n_list=3, noise=0.2,
                     norms="random", q_scale=2.0)
    n_sink, n_local, k = 2, 3, 5
    res = run(p, n_sink, n_local, k)
    d = 8
    q = [mpmath.mpf(float(x)) for x in p["q"]]
    Rr = list(range(n_sink, 24 - n_local))
    Tset = set(res.T.tolist())
    means = R.list_means_ref(p["V"], p["a"], 3, np.array(Rr))
    num = [mpmath.mpf(0)] * d
    den = mpmath.mpf(0)
    for i in range(24):
        if i in Rr and i not in Tset:
            kh = [mpmath.mpf(float(x)) for x in p["cen"][p["a"][i]]]
            for m in range(2):
                for t in range(4):
                    kh[m * 4 + t] += mpmath.mpf(float(p["cb"][m, p["z"][i, m], t]))
            kh = [mpmath.mpf(float(p["r"][i])) * x for x in kh]
            logit = mpmath.fsum(a * b for a, b in zip(q, kh)) / mpmath.sqrt(d)
            val = [mpmath.mpf(float(x)) for x in means[p["a"][i]]]
        else:
            kk = [mpmath.mpf(float(x)) for x in p["K"][i]]
            logit = mpmath.fsum(a * b for a, b in zip(q, kk)) / mpmath.sqrt(d)
            val = [mpmath.mpf(float(x)) for x in p["V"][i]]
        e = mpmath.exp(logit)
        den += e
        num = [a + e * b for a, b in zip(num, val)]
    ref = np.array([float(x / den) for x in num])
    assert close(res.y, ref, 1e-13)


# ---------------------------------------------------------------------------
# encoding into the existing index (Section 3.1) and the incremental update
# (Section 3.3)
# ---------------------------------------------------------------------------
def _enc_problem(seed, n=300, d=32, n_m=4, ksub=16, n_list=12):
    rng = np.random.default_rng(seed)
    C = rng.standard_normal((n_list, d))
    C /= np.linalg.norm(C, axis=1, keepdims=True)
    P = 0.15 * rng.standard_normal((n_m, ksub, d // n_m))
    K = rng.standard_normal((n, d)) * np.exp(rng.uniform(-1, 1, size=(n, 1)))
    return K, C, P


def test_encode_matches_scipy_vq():
    """Nearest centroid and nearest codeword against scipy's own vector quantizer."""
    import scipy.cluster.vq as vq
    K, C, P = _enc_problem(1)
    enc = R.encode_ref(K, C, P)
    u = K / np.linalg.norm(K, axis=1, keepdims=True)
    a_vq, _ = vq.vq(u, C, check_finite=False)
    np.testing.assert_array_equal(enc.a, a_vq)
    np.testing.assert_allclose(enc.r, np.linalg.norm(K, axis=1), rtol=1e-14)
    res = u - C[a_vq]
    ds = P.shape[2]
    for m in range(P.shape[0]):
        z_vq, _ = vq.vq(res[:, m * ds:(m + 1) * ds], P[m], check_finite=False)
        np.testing.assert_array_equal(enc.z[:, m], z_vq)


def test_encode_recovers_an_exactly_representable_key():
    """A key whose direction is c_j0 + P(z0) exactly is stored as (j0, z0, ||k||)."""
    rng = np.random.default_rng(2)
    d, n_m, ksub, n_list = 32, 4, 8, 6
    ds = d // n_m
    u0 = rng.standard_normal(d)
    u0 /= np.linalg.norm(u0)
    delta = 0.05 * rng.standard_normal(d)
    C = 3.0 * rng.standard_normal((n_list, d))   # far from the unit sphere
    j0 = 4
    C[j0] = u0 - delta
    P = 0.5 + rng.standard_normal((n_m, ksub, ds))   # far from delta's slices
    z0 = rng.integers(0, ksub, size=n_m)
    for m in range(n_m):
        P[m, z0[m]] = delta[m * ds:(m + 1) * ds]
    r = np.array([0.5, 1.0, 1.7])
    enc = R.encode_ref(r[:, None] * u0[None], C, P)
    assert np.all(enc.a == j0)
    assert np.all(enc.z == z0[None])
    np.testing.assert_allclose(enc.r, r, rtol=1e-14)
    recon = C[enc.a] + np.concatenate([P[m, enc.z[:, m]] for m in range(n_m)], axis=1)
    np.testing.assert_allclose(enc.r[:, None] * recon, r[:, None] * u0[None], atol=1e-12)


def test_encode_norm_scaling_and_zero_key():
    K, C, P = _enc_problem(3, n=80)
    e1 = R.encode_ref(K, C, P)
    e2 = R.encode_ref(2.5 * K, C, P)
    np.testing.assert_array_equal(e1.a, e2.a)
    np.testing.assert_array_equal(e1.z, e2.z)
    np.testing.assert_allclose(e2.r, 2.5 * e1.r, rtol=1e-14)
    z0 = R.encode_ref(np.zeros((1, K.shape[1])), C, P)
    assert z0.r[0] == 0.0
    assert z0.a[0] == int(np.argmin((C ** 2).sum(axis=1)))   # the centroid nearest the origin


def test_update_composes_and_matches_an_encoding_from_scratch():
    """Two updates equal one; both equal encoding all of R at once, with the
    list means recomputed by brute force over each list's members."""
    K, C, P = _enc_problem(4, n=400)
    V = np.random.default_rng(5).standard_normal(K.shape)
    n_sink, n_local, n_list = 4, 16, C.shape[0]
    n0, n1, n2 = 150, 270, 400
    R0 = np.arange(n_sink, n0 - n_local)
    e0 = R.encode_ref(K[R0], C, P)
    ids = np.zeros(400, np.int64)
    codes = np.zeros((400, P.shape[0]), np.int64)
    norms = np.zeros(400)
    ids[R0], codes[R0], norms[R0] = e0.a, e0.z, e0.r
    a1 = R.update_ref(ids, codes, norms, K, V, n0, n1, n_sink, n_local, C, P)
    a2 = R.update_ref(*a1[:3], K, V, n1, n2, n_sink, n_local, C, P)
    b2 = R.update_ref(ids, codes, norms, K, V, n0, n2, n_sink, n_local, C, P)
    Rn = np.arange(n_sink, n2 - n_local)
    full = R.encode_ref(K[Rn], C, P)
    for got in (a2, b2):
        np.testing.assert_array_equal(got[0][Rn], full.a)
        np.testing.assert_array_equal(got[1][Rn], full.z)
        np.testing.assert_allclose(got[2][Rn], full.r, rtol=1e-14)
        for j in range(n_list):
            members = [i for i in Rn if full.a[i - n_sink] == j]
            want = V[members].mean(axis=0) if members else np.zeros(K.shape[1])
            np.testing.assert_allclose(got[3][j], want, atol=1e-12)
    same = R.update_ref(*a2[:3], K, V, n2, n2, n_sink, n_local, C, P)
    np.testing.assert_array_equal(same[0], a2[0])
    np.testing.assert_allclose(same[3], a2[3], atol=0)
    with pytest.raises(ValueError):
        R.update_ref(*a2[:3], K, V, n2, n1, n_sink, n_local, C, P)


# ---------------------------------------------------------------------------
# k-means and the index build (Section 3.3, Appendix "Index build")
# ---------------------------------------------------------------------------
def _blobs(seed, k=6, per=40, dim=8, spread=0.05):
    rng = np.random.default_rng(seed)
    centers = 3.0 * rng.standard_normal((k, dim))
    X = np.concatenate([c + spread * rng.standard_normal((per, dim)) for c in centers])
    return X, centers


def test_kmeans_matches_scipy_lloyd():
    """Without empty clusters the iteration is scipy's kmeans2 from given centers."""
    import scipy.cluster.vq as vq
    X, _ = _blobs(20)
    rng = np.random.default_rng(21)
    init = rng.choice(X.shape[0], 6, replace=False)
    for n_iter in (1, 2, 5):
        want, _ = vq.kmeans2(X, X[init].copy(), iter=n_iter, minit="matrix", missing="raise")
        np.testing.assert_allclose(R.kmeans_ref(X, init, n_iter), want, atol=1e-12)
    np.testing.assert_array_equal(R.kmeans_ref(X, init, 0), X[init])


def test_kmeans_reseeds_empty_clusters_with_the_farthest_points():
    X, _ = _blobs(22, k=3, per=30)
    init = [0, 0, 0, 31]          # centers 1 and 2 tie with 0 and lose every point
    C = R.kmeans_ref(X, init, 1)
    a = np.array([0 if np.sum((x - X[0]) ** 2) <= np.sum((x - X[31]) ** 2) else 3 for x in X])
    dist = np.array([np.sum((x - X[init][ai]) ** 2) for x, ai in zip(X, a)])
    far = sorted(range(len(X)), key=lambda i: (-dist[i], i))
    np.testing.assert_allclose(C[0], X[a == 0].mean(axis=0), atol=1e-12)
    np.testing.assert_allclose(C[3], X[a == 3].mean(axis=0), atol=1e-12)
    np.testing.assert_array_equal(C[1], X[far[0]])
    np.testing.assert_array_equal(C[2], X[far[1]])


def test_build_closed_forms_and_consistency():
    """Zero iterations keep the drawn points: the coarse centers are the init
    tokens' directions and each codeword the init token's residual slice; the
    codes are the encoding against the built model, the means brute force."""
    rng = np.random.default_rng(23)
    n, d, M, ksub, n_list = 300, 16, 4, 8, 5
    K = rng.standard_normal((n, d)) * rng.uniform(0.5, 2.0, size=(n, 1))
    V = rng.standard_normal((n, d))
    Rr = np.arange(4, n - 10)
    init_c = rng.choice(Rr, n_list, replace=False)
    init_p = np.stack([rng.choice(Rr, ksub, replace=False) for _ in range(M)])
    b0 = R.build_ref(K, V, Rr, n_list, M, ksub, init_c, init_p, 0, 0)
    U = K / np.linalg.norm(K, axis=1, keepdims=True)
    np.testing.assert_allclose(b0["centroids"], U[init_c], atol=1e-15)
    a = np.array([np.argmin(((U[t] - b0["centroids"]) ** 2).sum(axis=1)) for t in range(n)])
    ds = d // M
    for m in range(M):
        for z in range(ksub):
            t = init_p[m, z]
            np.testing.assert_allclose(b0["codebooks"][m, z],
                                       (U[t] - b0["centroids"][a[t]])[m * ds:(m + 1) * ds], atol=1e-15)
    for it in ((1, 2), (3, 1)):
        b = R.build_ref(K, V, Rr, n_list, M, ksub, init_c, init_p, *it)
        enc = R.encode_ref(K[Rr], b["centroids"], b["codebooks"])
        np.testing.assert_array_equal(b["list_ids"][Rr], enc.a)
        np.testing.assert_array_equal(b["codes"][Rr], enc.z)
        for j in range(n_list):
            mem = Rr[enc.a == j]
            want = V[mem].mean(axis=0) if mem.size else np.zeros(d)
            np.testing.assert_allclose(b["list_means"][j], want, atol=1e-12)
        # the coarse centers are one more k-means step over the directions of R
        np.testing.assert_allclose(
            b["centroids"], R.kmeans_ref(U[Rr], [int(np.flatnonzero(Rr == t)[0]) for t in init_c], it[0]),
            atol=1e-12)


# ---------------------------------------------------------------------------
# dense attention (Section 3, opening paragraph; Eq. 1 with B empty)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("n_seq", [None, 1, 37, 200])
def test_dense_attention_matches_library_attention(n_seq):
    """The dense oracle against torch's attention routine (float64, CPU), on
    the whole cache and truncated to its first n_seq rows; the rows past
    n_seq hold large values, so reading them fails the pin."""
    rng = np.random.default_rng(31)
    d, n = 32, 200
    K = rng.standard_normal((n, d))
    V = rng.standard_normal((n, d))
    q = 0.5 * K[5] + rng.standard_normal(d)   # a spread softmax: the 1/sqrt(d) matters
    want = sdpa(q, K if n_seq is None else K[:n_seq], V if n_seq is None else V[:n_seq])
    if n_seq is not None:
        K[n_seq:] = 50.0 * rng.standard_normal((n - n_seq, d))
        V[n_seq:] = 1e3
    assert close(R.dense_attention_ref(q, K, V, n_seq), want, 1e-12)


def _gqa_batch(seed, B=2, Hq=8, Hkv=2, d=16, n_m=4, ksub=8, n_list=5, lens=(150, 97),
               nmax=160, exact=False, list_constant=False):
    """A ragged batch in the ABI's layouts, built independently of the
    product's generator. Each (b, KV head) has its own index; padding rows
    past seq_lens[b] hold values that would show if they were read. With
    exact=True every key equals its PQ reconstruction (no noise), and with
    list_constant=True every value is its list's offset."""
    rng = np.random.default_rng(seed)
    ds = d // n_m
    q = np.zeros((B, Hq, d))
    Kc = np.zeros((B, Hkv, nmax, d))
    Vc = np.zeros((B, Hkv, nmax, d))
    ids = np.zeros((B, Hkv, nmax), np.int64)
    codes = np.zeros((B, Hkv, nmax, n_m), np.uint8)
    norms = np.ones((B, Hkv, nmax))
    cen = rng.standard_normal((B, Hkv, n_list, d))
    cb = 0.4 * rng.standard_normal((B, Hkv, n_m, ksub, ds))
    means = np.zeros((B, Hkv, n_list, d))
    for b in range(B):
        n = lens[b]
        for g in range(Hkv):
            a = rng.integers(0, n_list, size=nmax)
            z = rng.integers(0, ksub, size=(nmax, n_m))
            recon = cen[b, g, a] + np.concatenate([cb[b, g, m, z[:, m]] for m in range(n_m)], axis=1)
            Kc[b, g] = recon + (0.0 if exact else 0.1) * rng.standard_normal((nmax, d))
            off = rng.standard_normal((n_list, d))
            Vc[b, g] = off[a] if list_constant else rng.standard_normal((nmax, d)) + 0.5 * off[a]
            Kc[b, g, n:] = 40.0 * rng.standard_normal((nmax - n, d))
            Vc[b, g, n:] = 1e3
            ids[b, g], codes[b, g] = a, z
            means[b, g] = R.list_means_ref(Vc[b, g], a, n_list, np.arange(4, n - 8))
        for h in range(Hq):
            g = h // (Hq // Hkv)
            q[b, h] = 2.0 * Kc[b, g, rng.integers(4, n - 8)] + 0.3 * rng.standard_normal(d)
    return dict(q=q, k_cache=Kc, v_cache=Vc, list_ids=ids, codes=codes, norms=norms,
                centroids=cen, codebooks=cb, list_means=means,
                seq_lens=np.array(lens, np.int32), n_sink=4, n_local=8)


def _sdpa_gqa(inp, b):
    """Library attention of sequence b over its first seq_lens[b] tokens,
    with torch's own grouped-query head mapping (float64, CPU)."""
    n = int(inp["seq_lens"][b])
    qt = torch.from_numpy(inp["q"][b])[None, :, None, :]
    kt = torch.from_numpy(inp["k_cache"][b, :, :n])[None]
    vt = torch.from_numpy(inp["v_cache"][b, :, :n])[None]
    return torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, enable_gqa=True)[0, :, 0].numpy()


def test_batch_oracle_gqa_mapping_and_ragged_lengths_at_rho_one():
    """k = |R_b| makes every row dense attention (Section 3.2, rho = 1): the
    batch oracle must then equal library attention with grouped query heads
    (head h reads KV head h // G, Section 3.3) over each sequence's own
    length. A head mapped to the wrong KV head, or a sequence read past its
    length, fails."""
    inp = _gqa_batch(41)
    topk = [int(n) - 12 for n in inp["seq_lens"]]
    refs = R.pqhsa_batch_ref(inp, topk)
    for b in range(2):
        want = _sdpa_gqa(inp, b)
        for h in range(8):
            assert close(refs[(b, h)].y, want[h], 1e-12), (b, h)
            assert refs[(b, h)].Z_B == 0.0


@pytest.mark.parametrize("k", [0, 3, 40])
def test_batch_oracle_gqa_index_mapping_closed_form(k):
    """With exact reconstruction (l~ = l for every token) and list-constant
    values (v_i = v_bar of its list), the background of Eq. 4 equals the
    dense contribution of B exactly, so every row is dense attention for any
    k. The index tensors of the wrong KV head give other scores and fail."""
    inp = _gqa_batch(43, exact=True, list_constant=True)
    topk = [k, k]
    refs = R.pqhsa_batch_ref(inp, topk)
    for b in range(2):
        want = _sdpa_gqa(inp, b)
        for h in range(8):
            assert close(refs[(b, h)].y, want[h], 1e-10), (b, h)
            if k == 0:
                assert refs[(b, h)].Z_B > 0.0


# ---------------------------------------------------------------------------
# index build: the subspace problems at n_iter_pq >= 1 (appendix on the index
# build; Section 3.1 for the residual slices)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("it_c,it_p", [(1, 1), (1, 2), (2, 2)])
def test_build_codebooks_match_scipy_on_residual_slices(it_c, it_p):
    """The codewords after n_iter_pq iterations equal scipy's Lloyd iteration
    (kmeans2 from given centers) on the residual slices u - c_a, where the
    test forms u, the coarse centers (scipy too), the nearest-center lists and
    the residuals itself."""
    import scipy.cluster.vq as vq
    rng = np.random.default_rng(47)
    n, d, M, ksub, n_list = 400, 16, 4, 6, 4
    # clustered directions, so that no coarse center or codeword loses all points
    dirs = rng.standard_normal((n_list, d)) * 3.0
    lab = rng.integers(0, n_list, size=n)
    K = (dirs[lab] + rng.standard_normal((n, d))) * rng.uniform(0.5, 2.0, size=(n, 1))
    V = rng.standard_normal((n, d))
    Rr = np.arange(4, n - 10)
    init_c = np.array([Rr[np.flatnonzero(lab[Rr] == j)[0]] for j in range(n_list)])
    init_p = np.stack([rng.choice(Rr, ksub, replace=False) for _ in range(M)])
    got = R.build_ref(K, V, Rr, n_list, M, ksub, init_c, init_p, it_c, it_p)

    U = K[Rr] / np.sqrt((K[Rr] ** 2).sum(axis=1, keepdims=True))
    row = {int(t): i for i, t in enumerate(Rr)}
    C, _ = vq.kmeans2(U, U[[row[int(t)] for t in init_c]].copy(), iter=it_c, minit="matrix",
                      missing="raise")
    a, _ = vq.vq(U, C)
    res = U - C[a]
    ds = d // M
    for m in range(M):
        sl = res[:, m * ds:(m + 1) * ds]
        want, _ = vq.kmeans2(sl, sl[[row[int(t)] for t in init_p[m]]].copy(), iter=it_p,
                             minit="matrix", missing="raise")
        np.testing.assert_allclose(got["codebooks"][m], want, atol=1e-12)
    np.testing.assert_allclose(got["centroids"], C, atol=1e-12)
    np.testing.assert_array_equal(got["list_ids"][Rr], a)
