"""Pins of the fp64 oracle to facts it does not compute itself.

Each test checks the oracle against something fixed by the mathematics of the
scoring (Sec. 3.1 Eq. 1 for the log-prob and the cut mask; the full-vocabulary
KL(teacher || student) that distillation minimises, Sec. 6): exact rational
arithmetic at 50 digits, closed forms, invariants, limits and brute-force
enumeration. test_oracle_mutations.py plants plausible mistakes in a copy of the
oracle and checks that these pins catch them.
"""
import json
import math
import os
from decimal import Decimal, getcontext

import numpy as np
import pytest
import torch

from oracle import olive_oracle as O

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def bf16_values(shape, rng, std=1.0):
    """Random values exactly representable in bf16 (and hence in fp64)."""
    x = torch.from_numpy(rng.standard_normal(shape).astype(np.float32) * std)
    return x.to(torch.bfloat16).float().numpy().astype(np.float64)


def test_row_scores_without_extras_returns_the_same_values():
    """extras=False only leaves keys out: every returned value is bit-identical to the
    full call's (the GPU parity of large workloads uses it), and the left-out keys
    are the reverse KL and top-K ones."""
    rng = np.random.default_rng(7)
    n, V, ds, dt = 5, 300, 16, 24
    hs, ht = bf16_values((n, ds), rng, 2.0), bf16_values((n, dt), rng, 2.0)
    ws, wt = bf16_values((ds, V), rng), bf16_values((dt, V), rng)
    y = rng.integers(0, V, size=n)
    full = O.row_scores(hs, ws, y, 2.0, ht, wt, 0.5)
    core = O.row_scores(hs, ws, y, 2.0, ht, wt, 0.5, extras=False)
    assert set(full) - set(core) == {"kl_rev", "kl_rev_nonneg", "jsd", "overlap", "kl_topk",
                                     "topk_s", "topk_t"}
    for k, v in core.items():
        np.testing.assert_array_equal(v, full[k], err_msg=k)


# ----------------------------------------------------------------------------- exact arithmetic
def decimal_row(h, w, scale):
    """z, lse, log-softmax of one row in 50-digit decimal arithmetic, no max shift."""
    getcontext().prec = 50
    d, V = w.shape
    z = []
    for v in range(V):
        acc = Decimal(0)
        for k in range(d):
            acc += Decimal(float(h[k])) * Decimal(float(w[k, v]))
        z.append(Decimal(repr(float(scale))) * acc)
    tot = sum((zi.exp() for zi in z), Decimal(0))
    lse = tot.ln()
    logp = [zi - lse for zi in z]
    return z, lse, logp


@pytest.mark.parametrize("seed", range(6))
def test_decimal_brute_force(seed):
    rng = np.random.default_rng(100 + seed)
    V = int(rng.integers(2, 17))
    ds, dt = int(rng.integers(1, 9)), int(rng.integers(1, 9))
    n = 3
    hs = bf16_values((n, ds), rng, 2.0)
    ht = bf16_values((n, dt), rng, 2.0)
    ws = bf16_values((ds, V), rng, 1.0)
    wt = bf16_values((dt, V), rng, 1.0)
    y = rng.integers(0, V, size=n)
    sS, sT = [1.0, 4.0, 0.5][seed % 3], [1.0, 2.0, 4.0][seed % 3]
    r = O.row_scores(hs, ws, y, sS, ht, wt, sT)
    for i in range(n):
        zs, lse_s, lps = decimal_row(hs[i], ws, sS)
        zt, lse_t, lpt = decimal_row(ht[i], wt, sT)
        assert abs(r["lse_s"][i] - float(lse_s)) <= 1e-13 * max(1.0, abs(float(lse_s)))
        assert abs(r["lse_t"][i] - float(lse_t)) <= 1e-13 * max(1.0, abs(float(lse_t)))
        assert abs(r["logp_s"][i] - float(lps[y[i]])) <= 1e-13 * max(1.0, abs(float(lps[y[i]])))
        assert abs(r["logp_t"][i] - float(lpt[y[i]])) <= 1e-13 * max(1.0, abs(float(lpt[y[i]])))
        kl = sum((lt.exp() * (lt - ls) for lt, ls in zip(lpt, lps)), Decimal(0))
        assert abs(r["kl"][i] - float(kl)) <= 1e-13 * max(1.0, float(kl))
        assert abs(r["kl_nonneg"][i] - float(kl)) <= 1e-13 * max(1.0, float(kl))
        klr = sum((ls.exp() * (ls - lt) for lt, ls in zip(lpt, lps)), Decimal(0))
        assert abs(r["kl_rev"][i] - float(klr)) <= 1e-13 * max(1.0, float(klr))
        assert abs(r["kl_rev_nonneg"][i] - float(klr)) <= 1e-13 * max(1.0, float(klr))
        # greedy token: first index attaining the exact maximum
        ms = max(zs)
        assert r["argmax_s"][i] == min(v for v in range(V) if zs[v] == ms)
        mt = max(zt)
        assert r["argmax_t"][i] == min(v for v in range(V) if zt[v] == mt)


# ----------------------------------------------------------------------------- closed forms
def test_golden_worked_examples():
    with open(os.path.join(GOLDEN, "worked_examples.json")) as f:
        data = json.load(f)
    for c in data["cases"]:
        region = O.REGION_SPANS if c.get("region") == "spans" else O.REGION_TEACHER
        spans = [[tuple(x) for x in sp] for sp in c["spans"]] if "spans" in c else None
        out = O.score(np.array(c["h_student"]), np.array(c["w_student"]), np.array(c["targets"]),
                      np.array(c["cu_seqlens"]), np.array(c["cut"]),
                      None if c["valid_len"] is None else np.array(c["valid_len"]),
                      np.array(c["h_teacher"]), np.array(c["w_teacher"]), region=region,
                      spans=spans)
        e = c["expect"]
        for k in ("logp_s", "logp_t", "kl", "kl_rev", "ce", "lse_s", "lse_t"):
            if k in e:
                np.testing.assert_allclose(out[k], e[k], rtol=0, atol=1e-14, err_msg=c["name"] + k)
        for k in ("argmax_s", "argmax_t"):
            if k in e:
                np.testing.assert_array_equal(out[k], e[k], err_msg=c["name"] + k)
        assert out["n_scored"] == e["n_scored"] and out["t_valid"] == e["t_valid"]


@pytest.mark.parametrize("V", [1, 2, 7, 1000])
def test_equal_columns_give_uniform(V):
    rng = np.random.default_rng(V)
    d = 5
    col = bf16_values((d, 1), rng)
    w = np.repeat(col, V, axis=1)
    h = bf16_values((4, d), rng, 3.0)
    r = O.row_scores(h, w, np.zeros(4, dtype=np.int64), 1.0, h, w, 1.0)
    np.testing.assert_allclose(r["logp_s"], -math.log(V), rtol=0, atol=1e-12)
    np.testing.assert_array_equal(r["argmax_s"], 0)       # all tied: lowest index
    assert np.all(np.abs(r["kl"]) <= 1e-15)


def test_two_token_softplus_and_bernoulli_kl():
    rng = np.random.default_rng(7)
    for _ in range(20):
        a = bf16_values((1, 2), rng, 3.0)
        b = bf16_values((1, 2), rng, 3.0)
        y = int(rng.integers(0, 2))
        r = O.row_scores(np.ones((1, 1)), a, [y], 1.0, np.ones((1, 1)), b, 1.0)
        other = 1 - y
        want = -np.logaddexp(0.0, a[0, other] - a[0, y])
        assert abs(r["logp_s"][0] - want) <= 1e-14
        p = 1.0 / (1.0 + math.exp(b[0, 0] - b[0, 1]))   # teacher P(token 1)
        q = 1.0 / (1.0 + math.exp(a[0, 0] - a[0, 1]))   # student P(token 1)
        kl = p * math.log(p / q) + (1 - p) * math.log((1 - p) / (1 - q))
        assert abs(r["kl"][0] - kl) <= 1e-13
        klr = q * math.log(q / p) + (1 - q) * math.log((1 - q) / (1 - p))
        assert abs(r["kl_rev"][0] - klr) <= 1e-13


# ----------------------------------------------------------------------------- invariants
def plain_logits(h, w, scale):
    """Logits by explicit Python loops (tiny sizes only), independent of the oracle."""
    n, d = h.shape
    V = w.shape[1]
    return [[scale * math.fsum(h[i, k] * w[k, v] for k in range(d)) for v in range(V)]
            for i in range(n)]


def test_probabilities_sum_to_one_and_lse_bounds():
    rng = np.random.default_rng(3)
    h = bf16_values((6, 8), rng, 2.0)
    w = bf16_values((8, 50), rng, 1.5)
    r = O.row_scores(h, w, np.zeros(6, dtype=np.int64), 2.0)
    z = plain_logits(h, w, 2.0)
    for i in range(6):
        s = math.fsum(math.exp(zv - r["lse_s"][i]) for zv in z[i])
        assert abs(s - 1.0) <= 1e-12
        M = max(z[i])
        assert M <= r["lse_s"][i] <= M + math.log(50) + 1e-12
        assert abs(r["max_s"][i] - M) <= 1e-12
        srt = sorted(z[i])
        assert abs(r["gap_s"][i] - (srt[-1] - srt[-2])) <= 1e-12


def test_kl_nonnegative_and_two_forms_agree():
    rng = np.random.default_rng(4)
    n, V = 16, 3000
    hs, ht = bf16_values((n, 32), rng), bf16_values((n, 48), rng)
    ws, wt = bf16_values((32, V), rng, 0.4), bf16_values((48, V), rng, 0.4)
    r = O.row_scores(hs, ws, np.zeros(n, dtype=np.int64), 1.0, ht, wt, 4.0)
    assert np.all(r["kl_nonneg"] >= 0.0)
    assert np.all(r["kl"] >= -1e-12)
    np.testing.assert_allclose(r["kl"], r["kl_nonneg"], rtol=1e-12, atol=1e-12)
    assert np.all(r["kl_rev_nonneg"] >= 0.0)
    assert np.all(r["kl_rev"] >= -1e-12)
    np.testing.assert_allclose(r["kl_rev"], r["kl_rev_nonneg"], rtol=1e-12, atol=1e-12)
    # the two directions differ for distinct distributions
    assert np.all(np.abs(r["kl_rev"] - r["kl"]) > 1e-6)


def test_kl_cross_entropy_identity():
    """KL(p_T||p_S) = H(p_T, p_S) - H(p_T): cross-entropy minus entropy."""
    rng = np.random.default_rng(12)
    hs, ht = bf16_values((4, 16), rng), bf16_values((4, 24), rng)
    ws, wt = bf16_values((16, 200), rng), bf16_values((24, 200), rng)
    r = O.row_scores(hs, ws, np.zeros(4, dtype=np.int64), 1.0, ht, wt, 1.0)
    zs, zt = plain_logits(hs, ws, 1.0), plain_logits(ht, wt, 1.0)
    for i in range(4):
        lt = [v - r["lse_t"][i] for v in zt[i]]
        ls = [v - r["lse_s"][i] for v in zs[i]]
        pt = [math.exp(v) for v in lt]
        cross = -math.fsum(p * l for p, l in zip(pt, ls))
        ent = -math.fsum(p * l for p, l in zip(pt, lt))
        assert abs(r["kl"][i] - (cross - ent)) <= 1e-12
        # reverse: KL(p_S||p_T) = H(p_S, p_T) - H(p_S)
        ps = [math.exp(v) for v in ls]
        cross_r = -math.fsum(p * l for p, l in zip(ps, lt))
        ent_r = -math.fsum(p * l for p, l in zip(ps, ls))
        assert abs(r["kl_rev"][i] - (cross_r - ent_r)) <= 1e-12


def test_kl_zero_for_identical_models_and_row_shift():
    rng = np.random.default_rng(5)
    n, d, V = 8, 16, 777
    hs = bf16_values((n, d), rng)
    ws = bf16_values((d, V), rng, 0.5)
    r = O.row_scores(hs, ws, np.arange(n), 1.0, hs, ws, 1.0)
    assert np.all(r["kl"] == 0.0)
    assert np.all(r["kl_rev"] == 0.0)
    np.testing.assert_array_equal(r["logp_s"], r["logp_t"])
    # teacher logits = student logits + a per-row constant: identical distributions
    c = bf16_values((1, V), rng)[0] * 0 + 3.0
    ht = np.concatenate([hs, bf16_values((n, 1), rng)], axis=1)
    wt = np.concatenate([ws, np.full((1, V), c[0])], axis=0)
    r2 = O.row_scores(hs, ws, np.arange(n), 1.0, ht, wt, 1.0)
    assert np.all(np.abs(r2["kl"]) <= 1e-12)
    assert np.all(np.abs(r2["kl_rev"]) <= 1e-12)
    assert np.all(np.abs(r2["logp_t"] - r2["logp_s"]) <= 1e-12)


def test_peaked_teacher_limit():
    """As p_T becomes one-hot at v*, KL(p_T||p_S) -> -log p_S(v*)."""
    rng = np.random.default_rng(6)
    hs, ht = bf16_values((3, 8), rng), bf16_values((3, 8), rng)
    ws, wt = bf16_values((8, 64), rng), bf16_values((8, 64), rng)
    r = O.row_scores(hs, ws, np.zeros(3, dtype=np.int64), 1.0, ht, wt, 1.0)
    for s in (64.0, 256.0):
        rr = O.row_scores(hs, ws, r["argmax_t"], 1.0, ht, wt, s)
        np.testing.assert_allclose(rr["kl"], -rr["logp_s"], rtol=0, atol=1e-6 * (64.0 / s) + 1e-9)


def test_peaked_student_limit_of_reverse_kl():
    """As p_S becomes one-hot at v*, KL(p_S||p_T) -> -log p_T(v*)."""
    rng = np.random.default_rng(16)
    hs, ht = bf16_values((3, 8), rng), bf16_values((3, 8), rng)
    ws, wt = bf16_values((8, 64), rng), bf16_values((8, 64), rng)
    r = O.row_scores(hs, ws, np.zeros(3, dtype=np.int64), 1.0, ht, wt, 1.0)
    for s in (64.0, 256.0):
        rr = O.row_scores(hs, ws, r["argmax_s"], s, ht, wt, 1.0)
        np.testing.assert_allclose(rr["kl_rev"], -rr["logp_t"], rtol=0,
                                   atol=1e-6 * (64.0 / s) + 1e-9)


def _decimal_entropy(logp):
    """-sum p log p of a row given as exact decimal log-probs."""
    return -sum((lp.exp() * lp for lp in logp), Decimal(0))


@pytest.mark.parametrize("seed", range(4))
def test_jsd_decimal_entropy_form(seed):
    """JSD(p, q) = H((p + q) / 2) - (H(p) + H(q)) / 2: the entropy form of the
    Jensen-Shannon divergence, evaluated at 50 digits from decimal logits, against the
    oracle's sum of the two KLs to the mixture."""
    rng = np.random.default_rng(300 + seed)
    V = int(rng.integers(2, 17))
    ds, dt = int(rng.integers(1, 9)), int(rng.integers(1, 9))
    n = 3
    hs, ht = bf16_values((n, ds), rng, 2.0), bf16_values((n, dt), rng, 2.0)
    ws, wt = bf16_values((ds, V), rng), bf16_values((dt, V), rng)
    sS, sT = [1.0, 4.0, 0.5, 2.0][seed], [1.0, 0.5, 4.0, 2.0][seed]
    r = O.row_scores(hs, ws, np.zeros(n, dtype=np.int64), sS, ht, wt, sT)
    getcontext().prec = 50
    for i in range(n):
        _, _, lps = decimal_row(hs[i], ws, sS)
        _, _, lpt = decimal_row(ht[i], wt, sT)
        m = [(a.exp() + b.exp()) / 2 for a, b in zip(lps, lpt)]
        h_m = -sum((x * x.ln() for x in m if x > 0), Decimal(0))
        want = h_m - (_decimal_entropy(lps) + _decimal_entropy(lpt)) / 2
        assert abs(r["jsd"][i] - float(want)) <= 1e-13, (r["jsd"][i], float(want))


def test_jsd_bounds_symmetry_and_limits():
    """0 <= JSD <= ln 2; symmetric in the two models; 0 for identical models; ln 2 in
    the limit of one-hot distributions on different tokens; and at most a quarter of
    the symmetrised KL (each KL to the mixture is at most half the KL to the other
    distribution, by convexity of KL in its second argument)."""
    rng = np.random.default_rng(21)
    n, V = 6, 400
    hs, ht = bf16_values((n, 12), rng, 1.5), bf16_values((n, 20), rng, 1.5)
    ws, wt = bf16_values((12, V), rng), bf16_values((20, V), rng)
    y = np.zeros(n, dtype=np.int64)
    r = O.row_scores(hs, ws, y, 1.0, ht, wt, 2.0)
    assert np.all(r["jsd"] >= -1e-15) and np.all(r["jsd"] <= math.log(2.0) + 1e-15)
    assert np.all(r["jsd"] <= 0.25 * (r["kl"] + r["kl_rev"]) + 1e-12)
    swapped = O.row_scores(ht, wt, y, 2.0, hs, ws, 1.0)
    np.testing.assert_allclose(swapped["jsd"], r["jsd"], rtol=1e-12, atol=1e-15)
    same = O.row_scores(hs, ws, y, 1.0, hs, ws, 1.0)
    assert np.all(np.abs(same["jsd"]) <= 1e-15)
    # one-hot on different tokens: JSD -> ln 2
    w1 = np.zeros((1, V))
    w2 = np.zeros((1, V))
    w1[0, 3] = 1.0
    w2[0, 7] = 1.0
    h = np.ones((1, 1))
    for s, tol in ((40.0, 1e-12), (80.0, 1e-15)):
        rr = O.row_scores(h, w1, [0], s, h, w2, s)
        assert abs(rr["jsd"][0] - math.log(2.0)) <= tol + V * math.exp(-s) * 4, rr["jsd"][0]


def test_jsd_two_tokens_closed_form():
    """V = 2: with p = (a, 1 - a), q = (b, 1 - b) and the binary entropy h,
    JSD = h((a + b) / 2) - (h(a) + h(b)) / 2."""
    def hb(x):
        return -(x * math.log(x) + (1 - x) * math.log(1 - x))
    for zs, zt in ((0.3, -1.2), (2.5, 2.5), (-4.0, 1.0), (0.0, 7.0)):
        a = 1.0 / (1.0 + math.exp(-zs))
        b = 1.0 / (1.0 + math.exp(-zt))
        want = hb((a + b) / 2) - 0.5 * (hb(a) + hb(b))
        r = O.row_scores(np.ones((1, 1)), np.array([[zs, 0.0]]), [0], 1.0,
                         np.ones((1, 1)), np.array([[zt, 0.0]]), 1.0)
        assert abs(r["jsd"][0] - want) <= 1e-14, (zs, zt, r["jsd"][0], want)


def test_lse_of_iid_gaussian_logits():
    """For V iid N(0, sigma^2) logits, lse ~= ln V + sigma^2 / 2 (law of large numbers)."""
    rng = np.random.default_rng(8)
    V, sigma = 151936, 1.0
    z = rng.standard_normal((4, V)) * sigma
    for i in range(4):
        st = O.log_softmax_stats(z[i])
        assert abs(st["lse"] - (math.log(V) + sigma ** 2 / 2)) < 0.02


def test_argmax_exact_ties_take_lowest_index():
    rng = np.random.default_rng(9)
    d, V = 6, 40
    w = bf16_values((d, V), rng)
    h = bf16_values((5, d), rng)
    z = h @ w
    for i in range(5):
        j = int(np.argmax(z[i]))
        w2 = w.copy()
        lo = int(rng.integers(0, j + 1))
        w2[:, lo] = w[:, j]        # duplicate the best column at a lower or equal index
        r = O.row_scores(h[i:i + 1], w2, [0], 1.0)
        assert r["argmax_s"][0] == lo
        assert r["gap_s"][0] == (0.0 if lo != j else r["gap_s"][0])


# ----------------------------------------------------------------------------- masks and Eq. 1
def test_mask_counts_enumerated():
    """All (len, cut, valid_len) with len <= 12: counts equal their closed forms."""
    for L in range(0, 13):
        for cut in range(0, L + 1):
            for vl in range(0, L + 1):
                cu = np.array([0, L])
                mt = O.masks(cu, [cut], [vl], O.REGION_TEACHER)
                ms = O.masks(cu, [cut], [vl], O.REGION_STUDENT)
                ma = O.masks(cu, [cut], [vl], O.REGION_ALL)
                assert mt["n_scored"] == max(0, vl - cut)
                assert ms["n_scored"] == min(cut, vl)
                assert ma["n_scored"] == vl
                assert mt["t_valid"] == vl
                # the scored teacher positions are exactly local t in [cut, vl)
                np.testing.assert_array_equal(np.nonzero(mt["in_region"])[0],
                                              np.arange(cut, max(cut, vl)))


# ----------------------------------------------------------------------------- top-K statistics
def test_topk_set_ties_take_lower_indices():
    z = [1.0, 3.0, 3.0, 2.0, 3.0, -1.0]
    np.testing.assert_array_equal(O.topk_set(z, 2), [1, 2])
    np.testing.assert_array_equal(O.topk_set(z, 4), [1, 2, 4, 3])
    np.testing.assert_array_equal(O.topk_set([0.0] * 7, 3), [0, 1, 2])
    # brute force: every k-subset ordered by (value desc, index asc)
    rng = np.random.default_rng(21)
    for _ in range(50):
        V = int(rng.integers(1, 12))
        z = rng.integers(-3, 4, size=V).astype(np.float64)   # many ties
        k = int(rng.integers(1, V + 1))
        want = [v for _, v in sorted((-z[v], v) for v in range(V))][:k]
        np.testing.assert_array_equal(O.topk_set(z, k), want)


def test_topk_worked_example():
    """Teacher logits ln(1, 4, 2, 8, 1), student ln(4, 1, 2, 1, 8), K = 2:
    TopK_T = {3, 1}, TopK_S = {4, 0}: overlap 0; with Z_T = 16 and Z_S = 16,
    KL_top2 = (8/16) ln(8/1) + (4/16) ln(4/1)."""
    zt = np.log([1.0, 4.0, 2.0, 8.0, 1.0])
    zs = np.log([4.0, 1.0, 2.0, 1.0, 8.0])
    lse_t = lse_s = math.log(16.0)
    st, ss = O.topk_set(zt, 2), O.topk_set(zs, 2)
    np.testing.assert_array_equal(st, [3, 1])
    np.testing.assert_array_equal(ss, [4, 0])
    assert O.topk_overlap(ss, st, 2) == 0.0
    want = 0.5 * math.log(8.0) + 0.25 * math.log(4.0)
    assert abs(O.kl_topk(zt, lse_t, zs, lse_s, st) - want) <= 1e-14
    # a student sharing one of the two: ln(1, 2, 4, 8, 1) -> TopK_S = {3, 2}, overlap 1/2
    s2 = O.topk_set(np.log([1.0, 2.0, 4.0, 8.0, 1.0]), 2)
    np.testing.assert_array_equal(s2, [3, 2])
    assert O.topk_overlap(s2, st, 2) == 0.5


def test_topk_reduces_to_argmax_and_to_the_full_kl():
    rng = np.random.default_rng(22)
    hs, ht = bf16_values((6, 8), rng), bf16_values((6, 8), rng)
    for V in (5, 16, 40):
        ws, wt = bf16_values((8, V), rng), bf16_values((8, V), rng)
        r = O.row_scores(hs, ws, np.zeros(6, dtype=np.int64), 1.0, ht, wt, 2.0)
        zs, zt = O.project(hs, ws, 1.0), O.project(ht, wt, 2.0)
        for i in range(6):
            # K = 1: the greedy tokens
            s1, t1 = O.topk_set(zs[i], 1), O.topk_set(zt[i], 1)
            assert s1[0] == r["argmax_s"][i] and t1[0] == r["argmax_t"][i]
            a = t1[0]
            lp_t, lp_s = zt[i, a] - r["lse_t"][i], zs[i, a] - r["lse_s"][i]
            assert abs(O.kl_topk(zt[i], r["lse_t"][i], zs[i], r["lse_s"][i], t1)
                       - math.exp(lp_t) * (lp_t - lp_s)) <= 1e-14
            # K = V: every token, the full KL and overlap 1
            if V <= O.TOPK:
                assert r["overlap"][i] == 1.0
                assert abs(r["kl_topk"][i] - r["kl"][i]) <= 1e-12
            else:
                assert r["kl_topk"][i] != r["kl"][i]
    # identical models: overlap 1 and zero divergence
    ws = bf16_values((8, 300), rng)
    r = O.row_scores(hs, ws, np.zeros(6, dtype=np.int64), 1.0, hs, ws, 1.0)
    assert np.all(r["overlap"] == 1.0) and np.all(r["kl_topk"] == 0.0)


def test_span_masks_reduce_to_the_cut_regions_and_add_up():
    """Span masks (Sec. 3.2): a single span [cut, len) is the teacher region, [0, cut)
    the student region, [0, len) every valid position, no span scores nothing; the
    count of two disjoint span sets is the sum of their counts."""
    for L in range(0, 9):
        for c in range(0, L + 1):
            for vl in range(0, L + 1):
                cu, cut, v = [0, L], [c], [vl]
                for spans, region in (([(c, L)], O.REGION_TEACHER), ([(0, c)], O.REGION_STUDENT),
                                      ([(0, L)], O.REGION_ALL)):
                    a = O.masks(cu, cut, v, O.REGION_SPANS, [spans])
                    b = O.masks(cu, cut, v, region)
                    np.testing.assert_array_equal(a["in_region"], b["in_region"])
                    assert a["n_scored"] == b["n_scored"]
                e = O.masks(cu, cut, v, O.REGION_SPANS, [[]])
                assert e["n_scored"] == 0 and e["t_valid"] == vl
                # disjoint split of [0, L) at every point
                for x in range(0, L + 1):
                    s1 = O.masks(cu, cut, v, O.REGION_SPANS, [[(0, x)]])["n_scored"]
                    s2 = O.masks(cu, cut, v, O.REGION_SPANS, [[(x, L)]])["n_scored"]
                    assert s1 + s2 == min(L, vl)
                    both = O.masks(cu, cut, v, O.REGION_SPANS, [[(0, x), (x, L)]])["n_scored"]
                    assert both == s1 + s2


def test_eq1_masks_prefix_and_scores_continuation():
    """A stitched trace (prefix y_1..y_k, continuation c_1..c_l): the teacher region
    scores exactly the l continuation tokens, and the loss is minus the sum of their
    student log-probs (Eq. 1)."""
    rng = np.random.default_rng(10)
    V, d = 50, 8
    w = bf16_values((d, V), rng)
    seqs = [(5, 3), (1, 6), (0, 4), (7, 0)]          # (k prefix tokens, l continuation tokens)
    lengths = [k + l for k, l in seqs]
    cu = np.concatenate([[0], np.cumsum(lengths)])
    T = int(cu[-1])
    h = bf16_values((T, d), rng)
    prefix_tok, cont_tok = 1000, 2000                 # labels, mapped into [0, V) below
    labels = []
    for k, l in seqs:
        labels += [prefix_tok] * k + [cont_tok] * l
    labels = np.array(labels)
    y = rng.integers(0, V, size=T)
    out = O.score(h, w, y, cu, [k for k, _ in seqs], None, h, w)
    assert out["n_scored"] == sum(l for _, l in seqs)
    np.testing.assert_array_equal(labels[out["in_region"]], cont_tok)
    r = O.row_scores(h, w, y, 1.0)
    for b, (k, l) in enumerate(seqs):
        idx = np.arange(cu[b] + k, cu[b] + k + l)
        assert abs(out["ce"][b] - (-math.fsum(r["logp_s"][idx]))) <= 1e-12
    # cut = 0 (offline SFT on whole teacher traces) scores every valid position;
    # cut = len scores none
    o0 = O.score(h, w, y, cu, [0] * 4)
    assert o0["n_scored"] == T
    oL = O.score(h, w, y, cu, lengths)
    assert oL["n_scored"] == 0 and np.all(oL["ce"] == 0.0) and np.all(oL["kl"] == 0.0)


def test_masked_outputs_exact_values():
    rng = np.random.default_rng(11)
    cu = np.array([0, 10, 10, 25])                  # includes an empty sequence
    cut, vl = np.array([4, 0, 7]), np.array([8, 0, 13])
    T, d, V = 25, 4, 30
    h, w = bf16_values((T, d), rng), bf16_values((d, V), rng)
    y = rng.integers(0, V, size=T)
    out = O.score(h, w, y, cu, cut, vl, h * 0.5, w)
    inval = ~out["valid"]
    assert np.all(out["logp_s"][inval] == 0.0) and np.all(out["argmax_s"][inval] == -1)
    outside = ~out["in_region"]
    assert np.all(out["kl"][outside] == 0.0)
    assert not np.any(np.signbit(out["kl"][outside]))
    assert out["t_valid"] == 8 + 0 + 13 and out["n_scored"] == 4 + 0 + 6
    assert out["ce"][1] == 0.0


# ------------------------------------------------------------------ backward (grad)
def _tiny_batch(seed, V=11, d_s=4, d_t=3, lens=(5, 7)):
    rng = np.random.default_rng(seed)
    T = sum(lens)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    return dict(h_s=rng.standard_normal((T, d_s)), w_s=rng.standard_normal((d_s, V)),
                h_t=rng.standard_normal((T, d_t)), w_t=rng.standard_normal((d_t, V)),
                y=rng.integers(0, V, T), cu=cu, cut=np.array([2, 3]),
                vl=np.array([lens[0], lens[1] - 1]))


def _loss(b, h_s, w_s, region, spans, w_ce, w_kl, s_s, s_t):
    return O.loss(h_s, w_s, b["y"], b["cu"], b["cut"], b["vl"], b["h_t"], b["w_t"], s_s, s_t,
                  region, spans, w_ce, w_kl)


@pytest.mark.parametrize("region,spans", [(O.REGION_TEACHER, None), (O.REGION_ALL, None),
                                          (O.REGION_SPANS, [[(0, 2), (3, 5)], [(1, 4)]])])
def test_backward_matches_finite_differences(region, spans):
    """dL/dh_S and dL/dW_S against central differences of the oracle's forward loss
    L = w_ce sum_b CE_b + w_kl sum_t KL(p_T || p_S)[t] (Eq. 1 and the distillation
    divergence), with two different logit scales."""
    b = _tiny_batch(3)
    w_ce, w_kl, s_s, s_t = 1.0, 0.7, 2.0, 1.5
    g = O.backward(b["h_s"], b["w_s"], b["y"], b["cu"], b["cut"], b["vl"], b["h_t"], b["w_t"],
                   s_s, s_t, region, spans, w_ce, w_kl)
    eps = 1e-6
    for arr, grad in (("h", g["grad_h"]), ("w", g["grad_w"])):
        base = b["h_s"] if arr == "h" else b["w_s"]
        num = np.zeros_like(base)
        for idx in np.ndindex(base.shape):
            plus, minus = base.copy(), base.copy()
            plus[idx] += eps
            minus[idx] -= eps
            hp, wp = (plus, b["w_s"]) if arr == "h" else (b["h_s"], plus)
            hm, wm = (minus, b["w_s"]) if arr == "h" else (b["h_s"], minus)
            num[idx] = (_loss(b, hp, wp, region, spans, w_ce, w_kl, s_s, s_t) -
                        _loss(b, hm, wm, region, spans, w_ce, w_kl, s_s, s_t)) / (2 * eps)
        np.testing.assert_allclose(grad, num, rtol=1e-6, atol=1e-7, err_msg=arr)
    # positions outside the region get no gradient
    out = ~g["in_region"]
    assert np.all(g["grad_h"][out] == 0.0)


def test_backward_invariants():
    """Every row's dL/dz sums to 0 over the vocabulary (both distributions sum to 1),
    so dW's rows sum to 0; the KL part vanishes for identical models and the whole
    gradient for an empty region."""
    b = _tiny_batch(5)
    g = O.backward(b["h_s"], b["w_s"], b["y"], b["cu"], b["cut"], b["vl"], b["h_t"], b["w_t"],
                   1.5, 1.0, O.REGION_TEACHER, None, 0.8, 0.3)
    np.testing.assert_allclose(g["g"].sum(axis=1), 0.0, atol=1e-12)
    np.testing.assert_allclose(g["grad_w"].sum(axis=1), 0.0, atol=1e-12)
    # CE part alone: the target entry is p_S[y] - 1 < 0, every other entry p_S > 0
    g1 = O.backward(b["h_s"], b["w_s"], b["y"], b["cu"], b["cut"], b["vl"], scale_student=1.5,
                    w_ce=1.0, w_kl=0.0)
    for i, t in enumerate(g1["rows"]):
        row = g1["g"][i]
        assert row[b["y"][t]] < 0 and np.all(np.delete(row, b["y"][t]) > 0)
    # teacher == student (same hidden states, weights and scale), KL only: no gradient
    g2 = O.backward(b["h_s"], b["w_s"], b["y"], b["cu"], b["cut"], b["vl"], b["h_s"], b["w_s"],
                    1.5, 1.5, O.REGION_ALL, None, 0.0, 1.0)
    assert np.abs(g2["grad_h"]).max() < 1e-14 and np.abs(g2["grad_w"]).max() < 1e-14
    # empty region: cut at the end of every sequence
    g3 = O.backward(b["h_s"], b["w_s"], b["y"], b["cu"], np.array([5, 7]), b["vl"],
                    scale_student=1.0)
    assert not g3["grad_h"].any() and not g3["grad_w"].any()
