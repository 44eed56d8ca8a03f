"""Pins that tie the float64 oracle to the paper and to mathematics, not to itself.

Each test checks the oracle against something fixed independently of its code:
identities of Theorem 1, closed forms, the paper's worked example, exact
enumeration of the speculative-decoding procedure on tiny vocabularies, and
invariants of Hedge / NormalHedge. A plausible slip in the oracle (a dropped
term, a wrong sign or index, T applied the wrong way, the wrong p used for the
learner's loss) fails at least one of them.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _bf16(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest even (test-side helper)."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


def _softmax(z: np.ndarray, T: float) -> np.ndarray:
    x = z.astype(np.float64) / T
    x = x - x.max()
    e = np.exp(x)
    return e / e.sum()


# ------------------------------------------------------------------------------------------
# Theorem 1: alpha = sum min(p, q) = 1 - TV(p, q)
# ------------------------------------------------------------------------------------------

@pytest.mark.parametrize("T", [1.0, 0.7, 0.05, 20.0])
def test_alpha_of_identical_rows_is_one(T):
    rng = np.random.default_rng(1)
    z = rng.normal(0, 3, 5000).astype(np.float32)
    assert abs(oracle.alpha_pair(z, z, T) - 1.0) < 1e-12
    zb = _bf16(z)
    assert abs(oracle.alpha_pair(zb, zb, T) - 1.0) < 1e-12


def test_alpha_disjoint_supports_is_exactly_zero():
    rng = np.random.default_rng(2)
    V = 4096
    zt = rng.normal(0, 2, V).astype(np.float32)
    zi = rng.normal(0, 2, V).astype(np.float32)
    mask = rng.random(V) < 0.5
    zt[mask] = -np.inf
    zi[~mask] = -np.inf
    assert oracle.alpha_pair(zt, zi, 1.0) == 0.0


def test_alpha_of_a_row_without_a_distribution_is_nan():
    # Theorem 1 takes two distributions; a row of -inf logits has no softmax. Either side
    # degenerate gives NaN, and the same row in a pair with itself too. The argmax of such a
    # row is the lowest index (all entries attain the max), and its normaliser is NaN.
    rng = np.random.default_rng(21)
    V = 3000
    z = rng.normal(0, 1, V).astype(np.float32)
    dead = np.full(V, -np.inf, np.float32)
    assert math.isnan(oracle.alpha_pair(dead, z, 1.0))
    assert math.isnan(oracle.alpha_pair(z, dead, 1.0))
    assert math.isnan(oracle.alpha_pair(dead, dead, 1.0))
    assert oracle.alpha_pair(z, z, 1.0) == pytest.approx(1.0, abs=1e-12)
    x = np.stack([z, dead, z])[:, None, None, :]  # target, a dead drafter, a copy
    ref = oracle.evaluate(x, V=V, T=1.0, want_alpha=True)
    assert math.isnan(ref["alpha"][0, 0, 0]) and ref["alpha"][0, 0, 1] == pytest.approx(1.0)
    assert ref["argmax"][0, 0, 1] == 0


@pytest.mark.parametrize("T", [1.0, 0.5, 3.0])
def test_alpha_symmetric_bounded_and_equals_one_minus_tv(T):
    rng = np.random.default_rng(3)
    for V in [2, 17, 1000, 32000]:
        zt = rng.normal(0, 2, V).astype(np.float32)
        zi = (zt + rng.normal(0, 1.5, V)).astype(np.float32)
        a = oracle.alpha_pair(zt, zi, T)
        assert 0.0 <= a <= 1.0
        assert abs(a - oracle.alpha_pair(zi, zt, T)) < 1e-13
        p, q = _softmax(zt, T), _softmax(zi, T)
        tv = 0.5 * np.abs(p - q).sum()
        assert abs(a - (1.0 - tv)) < 1e-12
        # acceptance-rule form of the speculative-decoding box: sum_v q_v min(1, p_v / q_v)
        assert abs(a - np.sum(q * np.minimum(1.0, p / q))) < 1e-12


@pytest.mark.parametrize("T", [1.0, 0.5, 2.0])
@pytest.mark.parametrize("delta", [0.5, 3.0, 9.0])
def test_alpha_closed_form_one_boosted_token_full_vocab(T, delta):
    # p uniform over V; q uniform except one token boosted by delta:
    # alpha = 1/V + (V - 1) / (e^{delta/T} + V - 1)
    V = 151936
    zt = np.zeros(V, dtype=np.float32)
    zi = np.zeros(V, dtype=np.float32)
    zi[12345] = delta
    want = 1.0 / V + (V - 1) / (math.exp(delta / T) + V - 1)
    assert abs(oracle.alpha_pair(zt, zi, T) - want) < 1e-11
    assert abs(oracle.alpha_pair(zi, zt, T) - want) < 1e-11
    # the same in bf16 storage (0 and delta are exact in bf16)
    assert abs(oracle.alpha_pair(_bf16(zt), _bf16(zi), T) - want) < 1e-11


def test_alpha_single_token_vocab_is_one():
    assert oracle.alpha_pair(np.array([3.0], np.float32), np.array([-7.0], np.float32), 1.0) == 1.0


def test_alpha_temperature_to_zero_gives_greedy_indicator():
    rng = np.random.default_rng(4)
    V = 64
    for _ in range(20):
        zt = rng.normal(0, 1, V).astype(np.float32)
        zi = (zt + rng.normal(0, 1, V)).astype(np.float32)
        st, si = np.sort(zt), np.sort(zi)
        if st[-1] - st[-2] < 0.05 or si[-1] - si[-2] < 0.05:
            continue
        a = oracle.alpha_pair(zt, zi, 1e-3)
        g = float(np.argmax(zt) == np.argmax(zi))
        assert abs(a - g) < 1e-9


def test_row_stats_argmax_lowest_index_and_lse():
    z = np.array([0.5, 2.0, -1.0, 2.0, 2.0, 1.0], dtype=np.float32)
    m, a, l = oracle.row_stats(z, 0.5)
    assert m == 2.0 and a == 1
    want = math.log(sum(math.exp(float(v) / 0.5) for v in z))
    assert abs(l - want) < 1e-13
    # bf16 ties (0x4000 == 2.0), and a -inf entry
    zb = np.array([0x3F80, 0x4000, 0xFF80, 0x4000], dtype=np.uint16)
    m, a, l = oracle.row_stats(zb, 1.0)
    assert m == 2.0 and a == 1
    assert abs(l - math.log(math.e + 2 * math.e ** 2)) < 1e-13


def test_evaluate_greedy_indicators_and_shapes():
    # target argmax 3 (tie with 7 resolved to the lowest index)
    V = 10
    t = np.zeros(V, np.float32)
    t[3] = t[7] = 5.0
    d1 = np.zeros(V, np.float32)
    d1[3] = 1.0
    d2 = np.zeros(V, np.float32)
    d2[7] = 1.0
    d3 = t.copy()
    x = np.stack([t, d1, d2, d3])[:, None, :]  # [R][G=1][V]
    out = oracle.evaluate(x, T=1.0)
    assert list(out["argmax"][0]) == [3, 3, 7, 3]
    assert list(out["agree"][0]) == [1, 0, 1]
    assert abs(out["alpha"][0, 2] - 1.0) < 1e-12


# ------------------------------------------------------------------------------------------
# Speculative-decoding box (Section 2.2), enumerated exactly on tiny vocabularies
# ------------------------------------------------------------------------------------------

def _sd_box_enumeration(P, Q):
    """Exact expectation of the number of tokens one chunk emits, and the law of its first token,
    for the speculative-decoding procedure with position-wise distributions P[k], Q[k]."""
    K, V = len(P), len(P[0])
    expected = 0.0
    first = np.zeros(V)
    res0 = np.maximum(P[0] - Q[0], 0.0)
    for drafts in itertools.product(range(V), repeat=K):
        reach = float(np.prod([Q[k][d] for k, d in enumerate(drafts)]))
        if reach == 0.0:
            continue
        for k, d in enumerate(drafts):
            acc = min(1.0, P[k][d] / Q[k][d])
            rej = reach * (1.0 - acc)
            expected += rej * (k + 1)  # k accepted drafts + the resampled token
            if k == 0:
                first[d] += reach * acc
                if res0.sum() > 0:
                    first += rej * res0 / res0.sum()
            reach *= acc
        expected += reach * (K + 1)  # all K accepted + the bonus token
    return expected, first


@pytest.mark.parametrize("V,K,T", [(2, 1, 1.0), (3, 2, 1.0), (4, 3, 0.7), (5, 3, 1.6), (3, 3, 0.3)])
def test_bruteforce_sd_box_matches_alpha_and_eal(V, K, T):
    rng = np.random.default_rng(100 + 10 * V + K)
    for trial in range(3):
        zt = rng.normal(0, 1.5, (K, V)).astype(np.float32)
        zq = (zt + rng.normal(0, 1.0, (K, V))).astype(np.float32)
        if trial == 2:
            zq[0, 0] = -np.inf  # a token the drafter never proposes
        P = [_softmax(zt[k], T) for k in range(K)]
        Q = [_softmax(zq[k], T) for k in range(K)]
        expected, first = _sd_box_enumeration(P, Q)
        # Theorem 1: the first emitted token is distributed as p
        assert np.allclose(first, P[0], atol=1e-13)
        gam = [oracle.alpha_pair(zt[k], zq[k], T) for k in range(K)]
        # Theorem 3 with position-wise fixed distributions is exact
        assert abs(oracle.eal_path(gam) - expected) < 1e-12


def test_bruteforce_greedy_is_one_plus_leading_agreement_run():
    for bits in itertools.product([0.0, 1.0], repeat=5):
        run = 0
        for g in bits:
            if g == 0.0:
                break
            run += 1
        assert oracle.eal_path(list(bits)) == 1.0 + run


# ------------------------------------------------------------------------------------------
# Theorem 3 estimator
# ------------------------------------------------------------------------------------------

def test_worked_example_censoring_appendix():
    with open(os.path.join(GOLDEN, "censoring_example.json")) as f:
        gold = json.load(f)
    for case in gold["cases"]:
        assert len(case["gamma"]) == case["K"]
        assert abs(oracle.eal_path(case["gamma"]) - case["eal"]) < 1e-12, case["name"]


@pytest.mark.parametrize("K", [1, 2, 4, 8, 9])
def test_eal_constant_gamma_closed_form(K):
    for a in [0.0, 0.25, 0.6, 0.9, 0.999]:
        want = (1 - a ** (K + 1)) / (1 - a)
        assert abs(oracle.eal_path([a] * K) - want) < 1e-12
    assert abs(oracle.eal_path([1.0] * K) - (K + 1)) < 1e-12
    assert oracle.eal_path([0.3] + [1.0] * (K - 1)) == pytest.approx(1 + 0.3 * K, abs=1e-12)


def test_eal_range_is_one_to_k_plus_one():
    rng = np.random.default_rng(5)
    for K in [1, 3, 8, 20]:
        for _ in range(50):
            e = oracle.eal_path(rng.random(K))
            assert 1.0 - 1e-12 <= e <= K + 1 + 1e-12


def test_tree_prefix_products_and_path_eal_hand_computed():
    parent = [-1, 0, 0, 1, 1, 2]
    gam = np.array([0.9, 0.8, 0.7, 0.6, 0.5, 0.4])[None, None, :]  # [B=1][N=1][M=6]
    out = oracle.accept_len(gam, parent=parent, path_end=[4], want_prefix=True)
    # path 0 -> 1 -> 4; prefix products by hand
    assert np.allclose(out["prefix"][0, 0], [0.9, 0.72, 0.63, 0.432, 0.36, 0.252], atol=1e-15)
    assert abs(out["eal"][0, 0] - (1 + 0.9 + 0.72 + 0.36)) < 1e-12
    assert list(oracle.path(parent, 5)) == [0, 2, 5]
    # a path through the tree equals the chain of its gammas
    out = oracle.accept_len(gam, parent=parent, path_end=[5])
    assert abs(out["eal"][0, 0] - oracle.eal_path([0.9, 0.7, 0.4])) < 1e-15
    # length loss 1 - EAL / (K_path + 1) with K_path = 3
    assert abs(out["loss"][0, 0, 0] - (1 - out["eal"][0, 0] / 4)) < 1e-15


def test_chain_equals_tree_with_chain_parents():
    rng = np.random.default_rng(6)
    g = rng.random((3, 5, 8))
    a = oracle.accept_len(g)
    b = oracle.accept_len(g, parent=np.arange(-1, 7), path_end=[7, 7, 7])
    assert np.array_equal(a["eal"], b["eal"])


def test_loss_kinds_on_worked_example():
    g = np.array([1.0, 0.0])[None, None, :]
    assert abs(oracle.accept_len(g, loss_kind=oracle.LOSS_LENGTH)["loss"][0, 0, 0] - 1 / 3) < 1e-15
    tok = oracle.accept_len(g, loss_kind=oracle.LOSS_ACCEPT_TOKEN)["loss"]
    assert tok.shape == (2, 1, 1) and list(tok[:, 0, 0]) == [0.0, 1.0]
    assert oracle.accept_len(g, loss_kind=oracle.LOSS_ACCEPT_CHUNK)["loss"][0, 0, 0] == 0.5
    # all-accept gives zero loss; all-reject gives K/(K+1) length loss
    assert oracle.accept_len(np.ones((1, 1, 4)))["loss"][0, 0, 0] == 0.0
    assert abs(oracle.accept_len(np.zeros((1, 1, 4)))["loss"][0, 0, 0] - 0.8) < 1e-15


def test_out_of_range_path_end_gives_nan():
    out = oracle.accept_len(np.ones((1, 2, 4)), path_end=[9])
    assert not out["ok"] and np.isnan(out["eal"]).all()


# ------------------------------------------------------------------------------------------
# Hedge
# ------------------------------------------------------------------------------------------

def test_hedge_eta_zero_stays_uniform_and_sums_to_one():
    rng = np.random.default_rng(7)
    w = np.full((3, 6), 1 / 6)
    loss = rng.random((5, 3, 6))
    assert np.allclose(oracle.hedge(w, loss, 0.0), 1 / 6, atol=1e-15)
    w2 = oracle.hedge(w, loss, 0.7)
    assert np.allclose(w2.sum(axis=1), 1.0, atol=1e-14)


def test_hedge_closed_form_cumulative_loss_and_shift_invariance():
    rng = np.random.default_rng(8)
    B, N, steps, eta = 4, 9, 40, 0.3
    loss = rng.random((steps, 1, B, N))
    w = np.full((B, N), 1 / N)
    for t in range(steps):
        w = oracle.hedge(w, loss[t], eta)
    cum = loss.sum(axis=(0, 1))
    logits = -eta * cum
    want = np.exp(logits - logits.max(axis=1, keepdims=True))
    want /= want.sum(axis=1, keepdims=True)
    assert np.allclose(w, want, atol=1e-13)
    # adding a constant to every expert's loss changes nothing
    w_shift = np.full((B, N), 1 / N)
    for t in range(steps):
        w_shift = oracle.hedge(w_shift, loss[t] + 0.37, eta)
    assert np.allclose(w_shift, w, atol=1e-13)
    # L vectors in one call == L calls
    w_one = oracle.hedge(np.full((B, N), 1 / N), loss[:, 0], eta)
    assert np.allclose(w_one, w, atol=1e-13)


# ------------------------------------------------------------------------------------------
# NormalHedge
# ------------------------------------------------------------------------------------------

def test_normalhedge_single_positive_regret_closed_form():
    N = 4
    R0 = np.zeros((1, N))
    p0 = np.full((1, N), 1 / N)
    loss = np.array([[[0.0, 1.0, 1.0, 1.0]]])  # l_A = 0.75 -> R = (0.75, -0.25, -0.25, -0.25)
    R, p, c = oracle.normalhedge(R0, p0, loss)
    assert np.allclose(R, [[0.75, -0.25, -0.25, -0.25]], atol=1e-15)
    want_c = 0.75 ** 2 / (2 * math.log(N * (math.e - 1) + 1))
    assert abs(c[0] - want_c) < 1e-14 * want_c
    assert np.allclose(p, [[1.0, 0.0, 0.0, 0.0]], atol=1e-15)


def test_normalhedge_m_equal_positive_regrets_closed_form():
    N, m = 5, 2
    loss = np.array([[[0.0, 0.0, 1.0, 1.0, 1.0]]])  # l_A = 0.6 -> R = (.6, .6, -.4, -.4, -.4)
    R, p, c = oracle.normalhedge(np.zeros((1, N)), np.full((1, N), 1 / N), loss)
    want_c = 0.36 / (2 * math.log((N * (math.e - 1) + m) / m))
    assert abs(c[0] - want_c) < 1e-14 * want_c
    assert np.allclose(p, [[0.5, 0.5, 0, 0, 0]], atol=1e-15)


def test_normalhedge_all_nonpositive_regret_is_uniform():
    R, p, c = oracle.normalhedge(np.zeros((2, 3)), np.full((2, 3), 1 / 3), np.full((1, 2, 3), 0.4))
    assert np.allclose(p, 1 / 3) and np.all(c == 0.0)


def test_normalhedge_stream_invariants():
    rng = np.random.default_rng(9)
    B, N = 3, 16
    R = np.zeros((B, N))
    p = np.full((B, N), 1 / N)
    base = rng.random((B, N))
    cum = np.zeros((B, N))
    for t in range(200):
        loss = np.clip(base + rng.uniform(-0.3, 0.3, (B, N)), 0, 1)[None]
        cum += loss[0]
        R_new, p_new, c = oracle.normalhedge(R, p, loss)
        # the learner's loss uses the distribution before the update: sum_i p_i dR_i = 0
        assert np.all(np.abs(((R_new - R) * p).sum(axis=1)) < 1e-13)
        assert np.allclose(p_new.sum(axis=1), 1.0, atol=1e-13)
        for b in range(B):
            if c[b] > 0:
                assert abs(oracle.normalhedge_residual(R_new[b], c[b])) < 1e-12
            assert np.all(p_new[b][R_new[b] <= 0] == 0.0) or c[b] == 0
        R, p = R_new, p_new
    # p is increasing in the regret, so the best expert in hindsight carries the largest weight
    assert np.all(np.argmax(p, axis=1) == np.argmin(cum, axis=1))
    for b in range(B):
        order = np.argsort(R[b])
        assert np.all(np.diff(p[b][order]) >= -1e-15)


def test_normalhedge_scale_covariance_and_permutation():
    rng = np.random.default_rng(10)
    N = 7
    R0 = rng.normal(0, 1, (1, N))
    zero = np.zeros((1, 1, N))  # a zero loss leaves R unchanged and re-solves c
    _, p1, c1 = oracle.normalhedge(R0, np.full((1, N), 1 / N), zero)
    for lam in [0.01, 3.0, 250.0]:
        _, p2, c2 = oracle.normalhedge(lam * R0, np.full((1, N), 1 / N), zero)
        assert abs(c2[0] - lam ** 2 * c1[0]) < 1e-12 * lam ** 2 * c1[0]
        assert np.allclose(p2, p1, atol=1e-12)
    perm = rng.permutation(N)
    _, p3, c3 = oracle.normalhedge(R0[:, perm], np.full((1, N), 1 / N), zero)
    assert abs(c3[0] - c1[0]) < 1e-13 * c1[0]
    assert np.allclose(p3, p1[:, perm], atol=1e-13)


@pytest.mark.parametrize("seed", [21, 22, 23])
def test_normalhedge_weights_are_the_gradient_of_the_scale_equation(seed):
    # NormalHedge's weight on drafter i is the partial derivative, in R_i, of the potential
    # whose level set e fixes c: p_i is proportional to d/dR_i (1/N) sum_j exp([R_j]_+^2 / 2c)
    # at the solved c. The derivative is taken here by central differences of that left
    # side (a route independent of the oracle's weight formula), with several distinct
    # positive regrets, so a wrong exponent or a wrong prefactor in the weights fails.
    rng = np.random.default_rng(seed)
    N = 9
    R0 = rng.normal(0.2, 1.0, (1, N))
    R0[0, :3] = [1.3, 0.4, 2.1]  # at least three distinct positive regrets
    R0[0, 3] = -0.5
    zero = np.zeros((1, 1, N))  # a zero loss leaves R unchanged and re-solves c
    R, p, c = oracle.normalhedge(R0, np.full((1, N), 1 / N), zero)
    assert np.array_equal(R, R0) and c[0] > 0

    def lhs(r):
        rp = np.maximum(r, 0.0)
        return np.mean(np.exp(rp * rp / (2.0 * c[0])))

    h = 1e-6
    grad = np.zeros(N)
    for i in range(N):
        e = np.zeros(N)
        e[i] = h
        grad[i] = (lhs(R0[0] + e) - lhs(R0[0] - e)) / (2 * h)
    grad[R0[0] <= 0] = 0.0  # [R]_+ has no slope there (the one-sided kink at 0 is not hit)
    want = grad / grad.sum()
    assert np.allclose(p[0], want, rtol=1e-7, atol=1e-9)
    # and the solved c really is the root: the level set is e
    assert abs(lhs(R0[0]) - math.e) < 1e-12


def test_hedge_expected_regret_within_the_hedge_bound():
    # Hedge on losses in [0, 1]: sum_t <w_t, l_t> - min_i sum_t l_t,i <= ln N / eta + eta T / 8
    # (the standard bound, Hoeffding's lemma per round), for any loss sequence; a sign slip in
    # the update (weights growing with loss) breaks it on an adversarial stream.
    rng = np.random.default_rng(12)
    B, N, T = 4, 8, 400
    eta = math.sqrt(8 * math.log(N) / T)
    w = np.full((B, N), 1 / N)
    mix = np.zeros(B)
    cum = np.zeros((B, N))
    for t in range(T):
        # adversarial-ish: the drafter that currently has the most weight loses
        loss = rng.random((B, N)) * 0.3
        loss[np.arange(B), np.argmax(w, axis=1)] = 1.0
        loss[:, 0] = np.minimum(loss[:, 0], 0.25)  # drafter 0 stays the best in hindsight
        mix += (w * loss).sum(axis=1)
        cum += loss
        w = oracle.hedge(w, loss[None], eta)
    regret = mix - cum.min(axis=1)
    assert np.all(regret <= math.log(N) / eta + eta * T / 8 + 1e-9)


def test_normalhedge_equal_losses_leave_regrets_exactly_unchanged():
    # l_A = sum_i p_i l = l when every loss is equal: regrets must not move at all,
    # whatever p is (no spurious positive regret from rounding)
    rng = np.random.default_rng(11)
    N = 8
    p0 = rng.random((1, N))
    p0 /= p0.sum()
    for val in [0.1, 1 / 3, 0.7, 5 / 9]:
        R, p, c = oracle.normalhedge(np.zeros((1, N)), p0, np.full((1, 1, N), val))
        assert np.all(R == 0.0) and c[0] == 0.0 and np.allclose(p, 1 / N)
    # ties among the drafters that carry weight: the tied drafters' regret is exactly 0
    p1 = np.array([[0.5, 0.5, 0.0, 0.0]])
    R, _, _ = oracle.normalhedge(np.zeros((1, 4)), p1, np.array([[[1 / 3, 1 / 3, 0.9, 0.1]]]))
    assert R[0, 0] == 0.0 and R[0, 1] == 0.0 and R[0, 2] < 0 < R[0, 3]


# ---- token-level length loss and QFI-D (Section 3.3; Appendix, algorithm QFI-D) ----------------

@pytest.mark.parametrize("K", [1, 2, 5, 8])
def test_window_losses_closed_forms(K):
    rng = np.random.default_rng(K)
    T, N = 3 * K + 4, 3
    # all accepted: EAL = K + 1, loss 0; all rejected: EAL = 1, loss K / (K + 1)
    assert np.all(oracle.window_losses(np.ones((T, N)), K) == 0.0)
    assert np.allclose(oracle.window_losses(np.zeros((T, N)), K), K / (K + 1), rtol=0, atol=1e-15)
    # constant gamma a: EAL = (1 - a^(K+1)) / (1 - a), the geometric sum
    for a in (0.25, 0.6, 0.95):
        want = 1 - (1 - a ** (K + 1)) / (1 - a) / (K + 1)
        assert np.allclose(oracle.window_losses(np.full((T, N), a), K), want, rtol=0, atol=1e-14)
    # window count and order: window s uses tokens s .. s + K - 1 only
    g = rng.random((T, N))
    ls = oracle.window_losses(g, K)
    assert ls.shape == (T - K + 1, N)
    g2 = g.copy()
    g2[K:] = rng.random((T - K, N))  # change every token after the first window
    assert np.array_equal(oracle.window_losses(g2, K)[0], ls[0])
    assert oracle.window_losses(g[:K - 1], K).shape == (0, N)


def test_window_loss_k1_is_half_the_rejection_probability():
    g = np.random.default_rng(3).random((20, 4))
    assert np.allclose(oracle.window_losses(g, 1), (1 - g) / 2, rtol=0, atol=1e-15)


def test_window_loss_of_the_censoring_example():
    with open(os.path.join(GOLDEN, "censoring_example.json")) as f:
        gold = json.load(f)
    for case in gold["cases"]:
        g = np.asarray(case["gamma"], dtype=np.float64)[:, None]
        got = oracle.window_losses(g, case["K"])
        assert got.shape == (1, 1)
        assert abs(got[0, 0] - (1 - case["eal"] / (case["K"] + 1))) < 1e-12, case["name"]


def _stream_counts(rng, rounds, K, B):
    return rng.integers(0, K + 1, (rounds, B))


def test_qfid_is_the_base_learners_on_the_window_stream_whatever_the_chunking():
    # QFI-D feeds the base learners every window loss in token order, each as soon as its
    # window is complete: the state after any chunking of the same stream equals the base
    # learners run on the whole window-loss sequence at once, and no window is used early.
    rng = np.random.default_rng(11)
    B, N, K, eta = 3, 5, 4, 0.4
    T = 40
    gam = [rng.random((T, N)) for _ in range(B)]
    results = []
    for split in range(3):
        q = oracle.QfiD(B, N, K, eta)
        pos = [0] * B
        while min(pos) < T:
            cnt = [min(int(rng.integers(0, K + 1)), T - pos[b]) for b in range(B)]
            g = np.zeros((B, N, K))
            for b in range(B):
                g[b, :, :cnt[b]] = gam[b][pos[b]:pos[b] + cnt[b]].T
            used = q.push(g, cnt)
            for b in range(B):
                pos[b] += cnt[b]
                assert q.done[b] == max(0, pos[b] - K + 1)  # every complete window, none early
                assert used[b].shape[0] <= cnt[b]
        results.append(q)
    for b in range(B):
        ls = oracle.window_losses(gam[b], K)[:, None, :]
        w = oracle.hedge(np.full((1, N), 1.0 / N), ls, eta)
        R, p, c = oracle.normalhedge(np.zeros((1, N)), np.full((1, N), 1.0 / N), ls)
        for q in results:
            assert np.array_equal(q.w[b], w[0]) and np.array_equal(q.R[b], R[0])
            assert np.array_equal(q.p[b], p[0]) and q.c[b] == c[0]


# ------------------------------------------------------------------------------------------
# Theorem 2 (EAGLE): gamma = sum of the target's p over the drafter's Top_L tokens
# ------------------------------------------------------------------------------------------

def _known_target(w: np.ndarray, T: float) -> np.ndarray:
    """fp32 target logits whose softmax at temperature T is w (up to fp32 rounding)."""
    return (T * np.log(w)).astype(np.float32)


@pytest.mark.parametrize("T", [1.0, 0.5])
@pytest.mark.parametrize("L", [1, 3, 10])
def test_topl_closed_form_on_a_linear_target(T, L):
    V = 200
    w = np.arange(1, V + 1, dtype=np.float64)
    w /= w.sum()
    rising = np.arange(V, dtype=np.float32)  # ranks the last tokens first
    x = np.stack([_known_target(w, T), rising, -rising])[:, None, :]
    out = oracle.topl(x, L, T=T)
    tri = V * (V + 1) / 2
    assert abs(out["gamma"][0, 0] - sum(range(V - L + 1, V + 1)) / tri) < 1e-6
    assert abs(out["gamma"][0, 1] - L * (L + 1) / 2 / tri) < 1e-6
    assert list(out["idx"][0, 0]) == list(range(V - 1, V - 1 - L, -1))
    assert list(out["idx"][0, 1]) == list(range(L))
    # the target's argmax V-1 is the rising drafter's first choice, the falling one's last
    assert out["hit"][0, 0] == 1 and out["hit"][0, 1] == 0


@pytest.mark.parametrize("bf16", [False, True])
def test_topl_full_vocabulary_has_mass_one_and_a_valid_order(bf16):
    rng = np.random.default_rng(11)
    V = 300
    x = rng.normal(0, 3, (4, 2, V)).astype(np.float32)
    x[2] = np.round(x[2])  # a drafter with many equal logits
    if bf16:
        x = _bf16(x)
    out = oracle.topl(x, V, T=0.7)
    assert np.all(np.abs(out["gamma"] - 1.0) < 1e-12)
    assert np.all(out["hit"] == 1)
    q = x.view(np.uint16).astype(np.uint32) << 16 if bf16 else x
    q = q.view(np.float32) if bf16 else q
    for g in range(2):
        for i in range(3):
            idx = out["idx"][g, i]
            assert sorted(idx) == list(range(V))
            v = q[1 + i, g, idx].astype(np.float64)
            assert np.all(v[:-1] >= v[1:])
            eq = v[:-1] == v[1:]
            assert np.all(idx[:-1][eq] < idx[1:][eq])


@pytest.mark.parametrize("seed", range(5))
def test_topl_bruteforce_dominating_subset(seed):
    """Top_L is the one L-subset whose every member ranks above every non-member."""
    rng = np.random.default_rng(100 + seed)
    V, T = 7, 0.8
    zt = rng.normal(0, 2, V).astype(np.float32)
    q = rng.integers(-2, 3, V).astype(np.float32)  # few levels: many ties
    p = _softmax(zt, T)
    x = np.stack([zt, q])[:, None, :]
    for L in range(1, V + 1):
        found = []
        for S in itertools.combinations(range(V), L):
            out_ = [u for u in range(V) if u not in S]
            if all(q[v] > q[u] or (q[v] == q[u] and v < u) for v in S for u in out_):
                found.append(set(S))
        assert len(found) == 1
        o = oracle.topl(x, L, T=T)
        assert set(o["idx"][0, 0]) == found[0]
        assert abs(o["gamma"][0, 0] - sum(p[v] for v in found[0])) < 1e-12
        assert o["hit"][0, 0] == (int(np.argmax(zt)) in found[0])


def test_topl_signed_zeros_rank_as_equal_by_index():
    zt = np.zeros(4, dtype=np.float32)
    for q, want in ((np.array([-0.0, 0.0, -1.0, 0.0], np.float32), [0, 1, 3]),
                    (np.array([0.0, -0.0, -1.0, -0.0], np.float32), [0, 1, 3])):
        for x in (np.stack([zt, q])[:, None, :], _bf16(np.stack([zt, q]))[:, None, :]):
            assert list(oracle.topl(x, 3, T=1.0)["idx"][0, 0]) == want


def test_topl_depends_on_the_drafter_only_through_its_ranking():
    rng = np.random.default_rng(12)
    V, L = 1000, 10
    zt = rng.normal(0, 3, V).astype(np.float32)
    q = rng.integers(-50, 50, V).astype(np.float32)
    base = oracle.topl(np.stack([zt, q])[:, None, :], L, T=0.5)
    for q2 in (q * 4, q * 0.25, q + 64, q - 1024):  # exact in fp32: same order, same ties
        o = oracle.topl(np.stack([zt, q2.astype(np.float32)])[:, None, :], L, T=0.5)
        assert np.array_equal(o["idx"], base["idx"]) and o["gamma"][0, 0] == base["gamma"][0, 0]
    for T in (0.1, 3.0):  # the children do not depend on the temperature, only the mass does
        assert np.array_equal(oracle.topl(np.stack([zt, q])[:, None, :], L, T=T)["idx"],
                              base["idx"])


def test_topl_mass_grows_by_the_next_ranked_probability():
    rng = np.random.default_rng(13)
    V, T = 64, 0.5
    w = rng.dirichlet(np.ones(V))
    x = np.stack([_known_target(w, T), rng.normal(0, 1, V).astype(np.float32)])[:, None, :]
    prev = oracle.topl(x, 1, T=T)
    assert abs(prev["gamma"][0, 0] - w[prev["idx"][0, 0, 0]]) < 1e-6
    for L in range(2, V + 1):
        cur = oracle.topl(x, L, T=T)
        assert np.array_equal(cur["idx"][0, 0, :L - 1], prev["idx"][0, 0])
        assert abs(cur["gamma"][0, 0] - prev["gamma"][0, 0] - w[cur["idx"][0, 0, L - 1]]) < 1e-6
        prev = cur
    assert abs(prev["gamma"][0, 0] - 1.0) < 1e-6


def test_topl_single_child_hit_is_greedy_agreement():
    rng = np.random.default_rng(14)
    x = _bf16(rng.normal(0, 2, (6, 3, 500)).astype(np.float32))
    x[2] = x[0]           # a drafter that copies the target
    x[3, :, 17] = 0x7F7F  # and one whose argmax is planted away from the target's
    hit = oracle.topl(x, 1, want_mass=False)["hit"]
    agree = oracle.evaluate(x, want_alpha=False)["agree"]
    assert np.array_equal(hit, agree) and np.all(hit[:, 1] == 1) and np.all(hit[:, 2] == 0)


def test_topl_rejects_bad_arguments():
    x = np.zeros((2, 1, 8), dtype=np.float32)
    with pytest.raises(ValueError):
        oracle.topl(x, 9)
    with pytest.raises(ValueError):
        oracle.topl(x, 0)
    with pytest.raises(ValueError):
        oracle.topl(x, 2, T=0.0)
    assert oracle.topl(x, 2, T=0.0, want_mass=False)["hit"][0, 0] == 1


# ------------------------------------------------------------------------------------------
# Chunks of ragged verified length k_h (Appendix "Chunk-Level vs Token-Level")
# ------------------------------------------------------------------------------------------

def test_ragged_chunk_lengths_closed_forms_and_token_rows():
    rng = np.random.default_rng(31)
    B, N, K = 4, 3, 6
    alpha = np.array([0.3, 0.6, 0.9])
    g = np.broadcast_to(alpha[None, :, None], (B, N, K)).copy()  # constant gamma per drafter
    ends = np.array([0, 2, 5, 3], dtype=np.int32)  # k_h = 1, 3, 6, 4
    out = oracle.accept_len(g, path_end=ends, loss_kind=oracle.LOSS_LENGTH)
    for b, e in enumerate(ends):
        k = e + 1
        want = (1 - alpha ** (k + 1)) / (1 - alpha)  # constant-gamma closed form with K = k_h
        assert np.allclose(out["eal"][b], want, rtol=1e-13, atol=0)
        assert np.allclose(out["loss"][0, b], 1 - want / (k + 1), rtol=1e-13, atol=0)
    ch = oracle.accept_len(g, path_end=ends, loss_kind=oracle.LOSS_ACCEPT_CHUNK)
    assert np.allclose(ch["loss"][0], (1 - alpha)[None, :].repeat(B, 0), rtol=1e-13, atol=0)
    # token losses: one vector per verified token, zero vectors past the chunk
    gr = rng.random((B, N, K))
    tok = oracle.accept_len(gr, path_end=ends, loss_kind=oracle.LOSS_ACCEPT_TOKEN)["loss"]
    for b, e in enumerate(ends):
        assert np.array_equal(tok[: e + 1, b], (1 - gr[b]).T[: e + 1])
        assert np.all(tok[e + 1:, b] == 0.0)
    # zero vectors change neither learner: the first k_h vectors alone give the same state
    w0 = np.full((B, N), 1.0 / N)
    w_all = oracle.hedge(w0, tok, 0.5)
    for b, e in enumerate(ends):
        w_b = oracle.hedge(w0[b:b + 1], tok[: e + 1, b:b + 1], 0.5)
        assert np.allclose(w_all[b], w_b[0], rtol=0, atol=1e-15)
    R0, p0 = np.zeros((B, N)), np.full((B, N), 1.0 / N)
    R_all, p_all, _ = oracle.normalhedge(R0, p0, tok)
    for b, e in enumerate(ends):
        Rb, pb, _ = oracle.normalhedge(R0[b:b + 1], p0[b:b + 1], tok[: e + 1, b:b + 1])
        assert np.array_equal(R_all[b], Rb[0]) and np.allclose(p_all[b], pb[0], rtol=0, atol=1e-12)


def test_ragged_chunk_invalid_length_is_nan_in_every_token_row():
    g = np.full((2, 2, 4), 0.5)
    tok = oracle.accept_len(g, path_end=np.array([4, 1], np.int32), loss_kind=oracle.LOSS_ACCEPT_TOKEN)
    assert np.all(np.isnan(tok["loss"][:, 0])) and not np.any(np.isnan(tok["loss"][:, 1]))
    assert not tok["ok"]


# ------------------------------------------------------------------------------------------
# Hybrid losses (Appendix "Practical heuristics")
# ------------------------------------------------------------------------------------------

def test_hybrid_losses_limits_and_the_appendix_example():
    rng = np.random.default_rng(51)
    T, N, K = 20, 4, 8
    g = rng.random((T, N))
    assert np.array_equal(oracle.hybrid_losses(g, K, 0), oracle.window_losses(g, K))
    assert np.array_equal(oracle.hybrid_losses(g, K, T), 1.0 - g)
    h = oracle.hybrid_losses(g, K, 5)
    assert h.shape[0] == 5 + (T - K + 1 - 5)
    assert np.array_equal(h[:5], 1.0 - g[:5])
    assert np.array_equal(h[5:], oracle.window_losses(g, K)[5:])
    # the appendix's example: K = 8 and a first chunk of 4 tokens. The acceptance loss can
    # already update the learner 4 times; the length loss cannot update it at all yet.
    first = g[:4]
    assert oracle.hybrid_losses(first, 8, 4).shape[0] == 4
    assert oracle.hybrid_losses(first, 8, 0).shape[0] == 0


def test_hybrid_qfid_chunking_invariance():
    rng = np.random.default_rng(52)
    B, N, K, H, rounds = 3, 5, 4, 6, 9
    gam = rng.random((rounds, B, N, K))
    cnt = rng.integers(0, K + 1, (rounds, B))
    a = oracle.QfiD(B, N, K, 0.5, hybrid=H)
    for r in range(rounds):
        a.push(gam[r], cnt[r])
    streams = [np.concatenate([gam[r, b, :, :cnt[r, b]].T for r in range(rounds)]) for b in range(B)]
    for b in range(B):
        ls = oracle.hybrid_losses(streams[b], K, H)
        w = oracle.hedge(np.full((1, N), 1.0 / N), ls[:, None, :], 0.5)
        R, p, _ = oracle.normalhedge(np.zeros((1, N)), np.full((1, N), 1.0 / N), ls[:, None, :])
        assert np.allclose(a.w[b], w[0], rtol=0, atol=1e-13)
        assert np.allclose(a.p[b], p[0], rtol=0, atol=1e-12)


# ------------------------------------------------------------------------------------------
# Drafter play and regret bookkeeping (Section 3.1; Appendix, algorithm QFI-D)
# ------------------------------------------------------------------------------------------

def test_play_argmax_ties_point_masses_and_empty_rows():
    w = np.array([[0.2, 0.5, 0.5, 0.1], [0, 0, 1.0, 0], [0, 0, 0, 0], [1, np.nan, 0, 0]])
    assert list(oracle.play(w, 0)) == [1, 2, -1, -1]
    for u in (0.0, 0.3, 0.999999):
        assert oracle.play(w[1:2], 1, np.array([u]))[0] == 2


def test_play_sampling_frequencies_on_a_grid_of_draws_are_the_weights():
    # integer weights k_i summing to M and draws u = m / M: exactly k_i draws pick drafter i
    k = np.array([3, 0, 7, 1, 0, 5, 0, 24], dtype=np.float64)
    M = int(k.sum())
    u = np.arange(M) / M
    ch = oracle.play(np.tile(k, (M, 1)), 1, u)
    assert np.array_equal(np.bincount(ch, minlength=len(k)), k.astype(int))
    assert list(ch[:4]) == [0, 0, 0, 2]  # inverse CDF: the draws fill the drafters in order


def test_regret_hand_computed_and_fixed_play():
    f = np.array([[[0.2, 0.5]], [[0.7, 0.1]], [[0.3, 0.3]]])  # [L=3][B=1][N=2]
    r = oracle.Regret(1, 2)
    reg = r.update(f, np.array([[1], [0], [1]], dtype=np.int32))
    assert abs(r.played[0] - 1.5) < 1e-15 and np.allclose(r.cum[0], [1.2, 0.9], atol=1e-15)
    assert abs(reg[0] - 0.6) < 1e-15
    rng = np.random.default_rng(61)
    L, B, N = 50, 3, 6
    f = rng.random((L, B, N))
    best = f.sum(0).argmin(1)
    for j in range(N):
        rj = oracle.Regret(B, N)
        reg = rj.update(f, np.full((L, B), j, dtype=np.int32))
        assert np.allclose(reg, f.sum(0)[:, j] - f.sum(0).min(1), rtol=0, atol=1e-12)
        assert np.all(reg >= 0) and np.all(reg[best == j] == 0.0)
    # chunked updates give the same sums
    rc = oracle.Regret(B, N)
    pl = rng.integers(0, N, (L, B)).astype(np.int32)
    for l0 in range(0, L, 7):
        rc.update(f[l0:l0 + 7], pl[l0:l0 + 7])
    ro = oracle.Regret(B, N)
    ro.update(f, pl)
    assert np.allclose(rc.regret, ro.regret, rtol=0, atol=1e-12)


def test_regret_eal_of_the_played_drafter_and_bad_indices():
    r = oracle.Regret(2, 3)
    eal = np.array([[1.5, 2.5, 3.5], [4.0, 5.0, 6.0]])
    r.update(np.zeros((2, 2, 3)), np.array([[0, 2], [1, 0]], dtype=np.int32), eal=eal)
    assert list(r.eal_sum) == [2.5, 4.0]  # the drafter played with the last vector
    rb = oracle.Regret(1, 3)
    rb.update(np.zeros((1, 1, 3)), np.array([[3]], dtype=np.int32))
    assert np.isnan(rb.regret[0])


# ------------------------------------------------------------------------------------------
# Theorem 2 with dynamic pruning: the target's mass on a given candidate set
# ------------------------------------------------------------------------------------------

def test_candidate_mass_of_the_top_l_is_the_eagle_mass():
    rng = np.random.default_rng(31)
    x = rng.normal(0, 2, (4, 3, 2, 500)).astype(np.float32)  # [R][B][K][V]
    for T in (1.0, 0.8):
        t = oracle.topl(x, 7, T=T)
        cm = oracle.candidate_mass(x[0], t["idx"], T=T)  # [B][K][N]
        assert np.allclose(cm, t["gamma"], rtol=1e-12, atol=0)


def test_candidate_mass_full_and_empty_sets_and_bad_indices():
    rng = np.random.default_rng(32)
    V = 50
    x = rng.normal(0, 3, (2, V)).astype(np.float32)
    full = np.tile(np.arange(V, dtype=np.int32), (2, 1, 1))  # [G][N=1][C=V]
    assert np.allclose(oracle.candidate_mass(x, full, T=0.7), 1.0, rtol=0, atol=1e-12)
    empty = np.full((2, 3, 5), -1, np.int32)
    assert np.all(oracle.candidate_mass(x, empty) == 0.0)
    bad = np.array([[[3, V, 4]], [[1, 2, -1]]], np.int32)
    g = oracle.candidate_mass(x, bad)
    assert np.isnan(g[0, 0]) and np.isfinite(g[1, 0])


def test_candidate_mass_of_a_known_distribution():
    # logits log p (+ any shift) have softmax p at T = 1, up to the fp32 rounding of log p
    # (relative error below 1e-6 per token here)
    rng = np.random.default_rng(33)
    V = 40
    p = rng.dirichlet(np.full(V, 0.5))
    p = np.maximum(p, 1e-12)
    p /= p.sum()
    for shift in (0.0, 17.5):
        z = (np.log(p) + shift).astype(np.float32)[None, :]
        sets = [rng.choice(V, size=k, replace=False) for k in (1, 5, 13, V)]
        for s in sets:
            c = np.full((1, 1, V), -1, np.int32)
            c[0, 0, :len(s)] = s
            rng.shuffle(c[0, 0])  # empty slots anywhere in the list
            got = oracle.candidate_mass(z, c)[0, 0]
            assert abs(got - p[s].sum()) <= 5e-6 * p[s].sum() + 1e-15, (len(s), got, p[s].sum())
