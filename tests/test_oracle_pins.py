"""Pins of the fp64 oracle against things other than itself (CPU only).

Each test ties one oracle function to a library routine (torch SDPA, numpy cov,
Python's stable sort), a closed form the paper derives, an invariant, or brute force on
a tiny input.  They are chosen so that a plausible slip (dropped term, wrong sign or
index, transposed operand, wrong scale, off-by-one mask) fails at least one of them;
tests/test_oracle_mutants.py plants such slips and checks that they are caught.
"""
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def sdpa(q, K, V, scale, mask=None):
    """Textbook softmax attention via torch (fp64): q [m,d], K [n,d], V [n,e] -> [m,e]."""
    qt = torch.from_numpy(np.asarray(q, np.float64))[None, None]
    Kt = torch.from_numpy(np.asarray(K, np.float64))[None, None]
    Vt = torch.from_numpy(np.asarray(V, np.float64))[None, None]
    m = None if mask is None else torch.from_numpy(mask)[None, None]
    return F.scaled_dot_product_attention(qt, Kt, Vt, attn_mask=m, scale=scale)[0, 0].numpy()


def lse(x):
    return float(torch.logsumexp(torch.from_numpy(np.asarray(x, np.float64)), 0))


# ------------------------------------------------------------------------ window mass
def test_window_mass_equals_sdpa_probabilities():
    """a_j = mean over window rows of softmax probabilities (Sec. 5.1 protocol).

    SDPA with one-hot values returns each row's attention weights; the mask is torch's
    bottom-right causal band (row t of the window sits at position N-w+t)."""
    rng = np.random.default_rng(1)
    G, w, d, N = 3, 5, 8, 37
    q = rng.normal(size=(G, w, d)) * 1.5
    K = rng.normal(size=(N, d))
    scale = 1 / math.sqrt(d)
    band = torch.ones(w, N, dtype=torch.bool).tril(diagonal=N - w).numpy()
    mask = np.tile(band, (G, 1))
    P = sdpa(q.reshape(G * w, d), K, np.eye(N), scale, mask)
    expect = P[:, : N - w].mean(axis=0)
    got = O.window_attention_mass(q, K, scale)
    np.testing.assert_allclose(got, expect, rtol=1e-12, atol=1e-15)
    # every row is a distribution over its visible keys
    np.testing.assert_allclose(P.sum(axis=1), 1.0, rtol=1e-12)


def test_window_mass_bruteforce_loops():
    rng = np.random.default_rng(2)
    G, w, d, N = 2, 3, 4, 11
    q = rng.normal(size=(G, w, d))
    K = rng.normal(size=(N, d))
    scale = 0.37
    acc = [0.0] * (N - w)
    for g in range(G):
        for t in range(w):
            vis = N - w + t
            logit = [scale * sum(q[g, t, i] * K[j, i] for i in range(d)) for j in range(vis + 1)]
            z = sum(math.exp(x) for x in logit)
            for j in range(N - w):
                acc[j] += math.exp(logit[j]) / z / (G * w)
    np.testing.assert_allclose(O.window_attention_mass(q, K, scale), acc, rtol=1e-12)


# ------------------------------------------------------------------------ chunk pooling
@pytest.mark.parametrize("n_sink,chunk,n", [(1, 4, 23), (1, 4, 24), (0, 4, 9), (2, 3, 17), (1, 1, 10)])
def test_chunk_pool_invariants(n_sink, chunk, n):
    rng = np.random.default_rng(3)
    a = rng.random(n)
    ab = O.chunk_pool(a, n_sink, chunk)
    assert ab.shape == (n - n_sink,)
    pos = np.arange(n_sink, n)
    cid = pos // chunk
    for c in np.unique(cid):
        sel = cid == c
        assert np.ptp(ab[sel]) == 0.0                              # constant inside a chunk
        np.testing.assert_allclose(ab[sel].sum(), a[pos[sel]].sum(), rtol=1e-13)  # sum kept
    # locality: changing one candidate's mass moves only its own chunk
    a2 = a.copy()
    j = n - 2
    a2[j] += 1.0
    ab2 = O.chunk_pool(a2, n_sink, chunk)
    changed = np.nonzero(ab2 != ab)[0] + n_sink
    assert set(changed) == set(pos[cid == j // chunk])
    if chunk == 1:
        np.testing.assert_array_equal(ab, a[n_sink:])


# ------------------------------------------------------------------------ selection
def test_select_top_matches_python_stable_sort_with_ties():
    rng = np.random.default_rng(4)
    for trial in range(20):
        n = int(rng.integers(1, 60))
        s = rng.integers(0, 6, size=n).astype(np.float64) / 4.0   # many exact ties
        k = int(rng.integers(0, n + 1))
        expect = sorted(range(n), key=lambda j: (-s[j], j))[:k]
        assert list(O.select_top(s, k)) == expect


# ------------------------------------------------------------------------ moments
def test_moments_equal_sequential_rank_one_updates():
    """Batched sums == the per-eviction additive update of Eq. app_update, in a random order."""
    rng = np.random.default_rng(5)
    N, d = 40, 6
    K, V = rng.normal(size=(N, d)), rng.normal(size=(N, d))
    E = rng.choice(N, size=17, replace=False)
    n, sk, sv, S = 0, np.zeros(d), np.zeros(d), np.zeros((d, d))
    for i in rng.permutation(E):
        n += 1
        sk = sk + K[i]
        sv = sv + V[i]
        for a in range(d):
            for b in range(d):
                S[a, b] += V[i, a] * K[i, b]
    m = O.evicted_moments(K, V, E)
    assert m.n_e == n
    np.testing.assert_allclose(m.s_k, sk, rtol=1e-12)
    np.testing.assert_allclose(m.s_v, sv, rtol=1e-12)
    np.testing.assert_allclose(m.S, S, rtol=1e-12, atol=1e-13)


def test_covariance_identity_against_numpy_cov():
    """S_tilde = sum_E v_i (k_i - k_bar)^T = n_e * cross-covariance(v, k) (App. A.1)."""
    rng = np.random.default_rng(6)
    N, d = 50, 7
    K = rng.normal(size=(N, d)) + 2.0
    V = rng.normal(size=(N, d)) - 1.0
    E = np.arange(3, 41)
    m = O.evicted_moments(K, V, E)
    k_bar, v_bar, St = O.centered_moments(m, tau=0.0)
    C = np.cov(np.vstack([V[E].T, K[E].T]), bias=True)
    np.testing.assert_allclose(St, len(E) * C[:d, d:], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(k_bar, K[E].mean(axis=0), rtol=1e-13)
    np.testing.assert_allclose(v_bar, V[E].mean(axis=0), rtol=1e-13)


def test_single_evicted_token_closed_form():
    """n_e = 1: k_bar = k, v_bar = v and S_tilde = 0 exactly."""
    rng = np.random.default_rng(7)
    K, V = rng.normal(size=(5, 4)), rng.normal(size=(5, 4))
    m = O.evicted_moments(K, V, [3])
    k_bar, v_bar, St = O.centered_moments(m, tau=0.0)
    np.testing.assert_array_equal(k_bar, K[3])
    np.testing.assert_array_equal(v_bar, V[3])
    assert np.abs(St).max() <= 1e-15


def test_clamp_zeroes_entries_below_tau():
    d = 3
    S = np.array([[5e-7, -2e-6, 0.3], [-9.99e-7, 1e-6, 0.0], [1.0, -1.0, 2e-7]])
    m = O.Moments(1, np.zeros(d), np.zeros(d), S)   # zero means: S_tilde == S
    _, _, St = O.centered_moments(m, tau=1e-6)
    keep = np.abs(S) >= 1e-6
    np.testing.assert_array_equal(St, np.where(keep, S, 0.0))


def test_zero_sum_of_centered_logits():
    rng = np.random.default_rng(8)
    K = rng.normal(size=(30, 8)) * 3
    m = O.evicted_moments(K, K, np.arange(30))
    k_bar, _, _ = O.centered_moments(m, 0.0)
    q = rng.normal(size=8)
    delta = (K - k_bar) @ q / math.sqrt(8)
    assert abs(delta.sum()) < 1e-11


# ------------------------------------------------------------------------ decode
def _split_case(rng, n=60, d=16, n_ret=20, spread=1.0, q_norm=1.0):
    K = rng.normal(size=(n, d))
    V = rng.normal(size=(n, d))
    R = np.sort(rng.choice(n, size=n_ret, replace=False))
    E = np.setdiff1d(np.arange(n), R)
    kc = K[E].mean(axis=0)
    K[E] = kc + spread * (K[E] - kc)
    q = rng.normal(size=d) * q_norm
    return q, K, V, R, E


def test_decode_without_eviction_is_softmax_attention():
    rng = np.random.default_rng(9)
    d = 16
    q, K, V = rng.normal(size=d) * 2, rng.normal(size=(33, d)), rng.normal(size=(33, d))
    r = O.decode_head(q, K, V, O.Moments.zeros(d))
    np.testing.assert_allclose(r.out, sdpa(q[None], K, V, 1 / math.sqrt(d))[0], rtol=1e-12)
    assert r.w_R == 1.0
    np.testing.assert_allclose(r.log_Z_R, lse(K @ q / math.sqrt(d)), rtol=1e-13)


def test_decode_without_correction_is_softmax_attention_over_retained():
    """order = -1 (the ablation without the correction) returns textbook attention over
    the retained rows whatever the summary, with w_R = 1."""
    rng = np.random.default_rng(19)
    d = 12
    q, K, V, R, E = _split_case(rng, spread=1.0, q_norm=2.0)
    m = O.evicted_moments(K, V, E)
    assert m.n_e > 0
    r = O.decode_head(q, K[R], V[R], m, order=-1)
    np.testing.assert_allclose(r.out, sdpa(q[None], K[R], V[R], 1 / math.sqrt(len(q)))[0],
                               rtol=1e-12)
    assert r.w_R == 1.0


def test_eviction_diagnostics_against_library_attention():
    """The diagnostics are the paper's quantities: w_E from torch softmax weights, the
    relative error of f_R against SDPA over every row, and the corrected output closer to
    full attention than f_R on this planted-covariance case."""
    rng = np.random.default_rng(20)
    q, K, V, R, E = _split_case(rng, spread=0.3, q_norm=2.0)
    d = len(q)
    dg = O.eviction_diagnostics(q, K, V, R)
    w = torch.softmax(torch.from_numpy(K @ q / math.sqrt(d)), 0).numpy()
    np.testing.assert_allclose(dg["w_E"], w[E].sum(), rtol=1e-12)
    full = sdpa(q[None], K, V, 1 / math.sqrt(d))[0]
    f_R = sdpa(q[None], K[R], V[R], 1 / math.sqrt(d))[0]
    np.testing.assert_allclose(dg["rel_err_retained"],
                               np.linalg.norm(f_R - full) / np.linalg.norm(full), rtol=1e-10)
    assert dg["rel_err_corrected"] < dg["rel_err_retained"]
    assert dg["cos_fE_fEhat"] > 0.99


def test_decode_zero_key_spread_recovers_full_attention():
    """All evicted keys equal: delta = 0, f_E_hat = v_bar = f_E and Z_E_hat = Z_E, so the
    corrected output is exact full attention over R and E (Sec. 4.2, App. B.2)."""
    rng = np.random.default_rng(10)
    q, K, V, R, E = _split_case(rng, spread=0.0, q_norm=3.0)
    m = O.evicted_moments(K, V, E)
    r = O.decode_head(q, K[R], V[R], m, tau=0.0)
    full = sdpa(q[None], K, V, 1 / math.sqrt(len(q)))[0]
    np.testing.assert_allclose(r.out, full, rtol=1e-11, atol=1e-13)
    s = K @ q / math.sqrt(len(q))
    w_R = math.exp(lse(s[R]) - lse(s))
    np.testing.assert_allclose(r.w_R, w_R, rtol=1e-12)
    np.testing.assert_allclose(r.log_Z_E_hat, lse(s[E]), rtol=1e-12)


def test_decode_query_orthogonal_to_key_spread_is_exact():
    """q orthogonal to every k_i - k_bar: S_tilde != 0 but S_tilde q = 0 and delta = 0, so
    the output equals full attention; a transposed covariance would not vanish."""
    rng = np.random.default_rng(11)
    d, n = 12, 50
    q = rng.normal(size=d)
    K = rng.normal(size=(n, d))
    V = rng.normal(size=(n, d)) + K[:, ::-1]
    R = np.arange(0, n, 3)
    E = np.setdiff1d(np.arange(n), R)
    P = np.eye(d) - np.outer(q, q) / (q @ q)
    K[E] = K[E] @ P + 0.7 * q                     # spread lies in q's orthogonal complement
    m = O.evicted_moments(K, V, E)
    _, _, St = O.centered_moments(m, 0.0)
    assert np.abs(St).max() > 1.0
    r = O.decode_head(q, K[R], V[R], m, tau=0.0)
    np.testing.assert_allclose(r.out, sdpa(q[None], K, V, 1 / math.sqrt(d))[0], rtol=1e-10,
                               atol=1e-12)


def _err_ratios(errs):
    return [errs[i] / errs[i + 1] for i in range(len(errs) - 1)]


def test_decode_first_order_error_is_second_order_in_key_spread():
    """||f_E - f_E_hat|| = O(eps^2) when the evicted key deviations shrink by eps
    (App. A.2 Eq. app_error_bound): halving eps divides the error by ~4.  The
    zeroth-order variant (v_bar only) is only O(eps): ratio ~2."""
    d = 16
    errs1, errs0, errs_full = [], [], []
    eps_list = [0.4, 0.2, 0.1, 0.05, 0.025]
    for eps in eps_list:
        rng = np.random.default_rng(12)
        q, K, V, R, E = _split_case(rng, n=80, d=d, n_ret=10, spread=eps, q_norm=2.0)
        m = O.evicted_moments(K, V, E)
        f_E = sdpa(q[None], K[E], V[E], 1 / math.sqrt(d))[0]
        r1 = O.decode_head(q, K[R], V[R], m, tau=0.0, order=1)
        r0 = O.decode_head(q, K[R], V[R], m, tau=0.0, order=0)
        errs1.append(np.linalg.norm(f_E - r1.f_E_hat))
        errs0.append(np.linalg.norm(f_E - r0.f_E_hat))
        full = sdpa(q[None], K, V, 1 / math.sqrt(d))[0]
        errs_full.append(np.linalg.norm(full - r1.out))
        # explicit bound of Eq. app_error_bound (leading term; sigma small here)
        k_bar = K[E].mean(axis=0)
        sig = np.abs((K[E] - k_bar) @ q / math.sqrt(d)).max()
        vmax = np.linalg.norm(V[E], axis=1).max()
        bound = sig ** 2 * math.exp(sig) / 2 * (vmax + np.linalg.norm(r1.f_E_hat))
        assert errs1[-1] <= bound * 1.05
    for r in _err_ratios(errs1[1:]):
        assert 3.6 < r < 4.4, errs1
    for r in _err_ratios(errs_full[1:]):
        assert 3.6 < r < 4.4, errs_full
    for r in _err_ratios(errs0[2:]):
        assert 1.8 < r < 2.2, errs0


def test_jensen_lower_bound_and_weight_bias_identity():
    """Z_E_hat <= Z_E and w_R_hat >= w_R (Eq. jensen); the exact bias identity of
    Eq. app_weight_bias; Z_E/Z_E_hat -> 1 + Var(delta)/2 (Eq. app_ratio)."""
    rng = np.random.default_rng(13)
    for trial in range(10):
        q, K, V, R, E = _split_case(rng, spread=rng.uniform(0.1, 2.0), q_norm=2.0)
        d = len(q)
        m = O.evicted_moments(K, V, E)
        r = O.decode_head(q, K[R], V[R], m, tau=0.0)
        s = K @ q / math.sqrt(d)
        lZ, lZR, lZE = lse(s), lse(s[R]), lse(s[E])
        assert r.log_Z_E_hat <= lZE + 1e-12
        w_R = math.exp(lZR - lZ)
        assert r.w_R >= w_R - 1e-15
        eps = math.exp(lZE - r.log_Z_E_hat) - 1.0
        w_E_hat = 1.0 - r.w_R
        # Eq. app_weight_bias's middle line, simplified: w_R * w_E_hat * eps; the printed
        # closing form carries 1/(1 + eps w_E_hat), which belongs with w_R_hat in front.
        np.testing.assert_allclose(r.w_R - w_R, w_R * w_E_hat * eps, rtol=1e-8, atol=1e-15)
        np.testing.assert_allclose(r.w_R - w_R, r.w_R * w_E_hat * eps / (1 + eps * w_E_hat),
                                   rtol=1e-8, atol=1e-15)
    # logit-variance law at small spread
    q, K, V, R, E = _split_case(np.random.default_rng(14), spread=0.02, q_norm=2.0)
    d = len(q)
    m = O.evicted_moments(K, V, E)
    r = O.decode_head(q, K[R], V[R], m, tau=0.0)
    s = K @ q / math.sqrt(d)
    ratio = math.exp(lse(s[E]) - r.log_Z_E_hat)
    kc = K[E] - K[E].mean(axis=0)
    var = q @ (kc.T @ kc / len(E)) @ q / d
    np.testing.assert_allclose(ratio - 1.0, var / 2, rtol=2e-2)


def test_exact_decomposition_of_full_attention():
    rng = np.random.default_rng(15)
    q, K, V, R, E = _split_case(rng, q_norm=2.0)
    p = O.attention_parts(q, K, V, R)
    full = sdpa(q[None], K, V, 1 / math.sqrt(len(q)))[0]
    np.testing.assert_allclose(p["f"], full, rtol=1e-12)
    np.testing.assert_allclose(p["w_R"] * p["f_R"] + p["w_E"] * p["f_E"], full, rtol=1e-12)
    np.testing.assert_allclose(p["f_R"], sdpa(q[None], K[R], V[R], 1 / math.sqrt(len(q)))[0],
                               rtol=1e-12)
    np.testing.assert_allclose(np.linalg.norm(full - p["f_R"]), p["w_E"] * p["gamma"] *
                               np.linalg.norm(full), rtol=1e-10)


# ------------------------------------------------------------------------ residual
def test_residual_is_second_order_close_to_true_evicted_output_at_own_key():
    """r_j = v_j - f_E_hat(q = k_j): the residual's prediction term is the first-order
    estimate of the evicted attention output evaluated at token j's own key, so
    r_j - (v_j - f_E(k_j)) is O(eps^2) in the evicted key spread (Sec. 4.2, App. A.2)."""
    d = 8
    errs = []
    for eps in [0.2, 0.1, 0.05, 0.025]:
        rng = np.random.default_rng(16)
        _, K, V, R, E = _split_case(rng, n=70, d=d, n_ret=12, spread=eps)
        m = O.evicted_moments(K, V, E)
        r = O.moment_residuals(K[R], V[R], m, 1 / math.sqrt(d), tau=0.0)
        f_E = sdpa(K[R], K[E], V[E], 1 / math.sqrt(d))
        errs.append(np.abs(r - (V[R] - f_E)).max())
    for x in _err_ratios(errs):
        assert 3.5 < x < 4.5, errs


def test_residual_with_empty_summary_is_the_value():
    rng = np.random.default_rng(17)
    K, V = rng.normal(size=(9, 4)), rng.normal(size=(9, 4))
    s, rn = O.residual_scores(K, V, np.full(9, 0.5), np.arange(9), O.Moments.zeros(4), 0.5, 1e-6)
    np.testing.assert_allclose(rn, np.linalg.norm(V, axis=1), rtol=1e-14)
    np.testing.assert_allclose(s, 0.5 * rn, rtol=1e-14)


# ------------------------------------------------------------------------ compress
def _tiny_prefill(seed, G=2, w=4, d=8, N=48):
    rng = np.random.default_rng(seed)
    K = rng.normal(size=(N, d))
    V = rng.normal(size=(N, d)) + 0.5 * K
    q = K[rng.integers(0, N, size=(G, w))] + 0.3 * rng.normal(size=(G, w, d))
    return q, K, V


def test_compress_full_budget_keeps_everything():
    q, K, V = _tiny_prefill(18)
    r = O.compress_head(q, K, V, budget=len(K))
    np.testing.assert_array_equal(r.idx, np.arange(len(K)))
    assert r.moments.n_e == 0 and not r.moments.S.any()


@pytest.mark.parametrize("mi_rounds", [-1, 0, 1, 2])
def test_compress_structure(mi_rounds):
    q, K, V = _tiny_prefill(19)
    N, w, L = len(K), q.shape[1], 20
    r = O.compress_head(q, K, V, budget=L, mi_rounds=mi_rounds)
    assert len(r.idx) == L and np.all(np.diff(r.idx) > 0)
    assert 0 in r.idx and set(range(N - w, N)) <= set(r.idx)
    cand = set(range(1, N - w))
    assert set(r.retained) | set(r.evicted) == cand
    assert not set(r.retained) & set(r.evicted)
    assert r.moments.n_e == len(cand) - (L - 1 - w)
    np.testing.assert_array_equal(r.k_out, K[r.idx])
    np.testing.assert_array_equal(r.v_out, V[r.idx])
    m = O.evicted_moments(K, V, r.evicted)
    np.testing.assert_allclose(r.moments.S, m.S, rtol=1e-13)


def test_snapkv_mode_is_top_pooled_mass():
    q, K, V = _tiny_prefill(20)
    N, w, L = len(K), q.shape[1], 17
    r = O.compress_head(q, K, V, budget=L, mi_rounds=-1)
    a = O.window_attention_mass(q, K, 1 / math.sqrt(K.shape[1]))
    ab = O.chunk_pool(a, 1, 4)
    cand = list(range(1, N - w))
    best = sorted(range(len(cand)), key=lambda i: (-ab[i], i))[: L - 1 - w]
    assert sorted(cand[i] for i in best) == list(r.retained)


def test_provisional_round_is_greedy_first_eviction():
    """With an empty summary Algorithm 1 scores alpha_j ||v_j||; the greedy loop's first
    eviction is the lowest-scored candidate of the provisional round."""
    q, K, V = _tiny_prefill(21)
    N, w = len(K), q.shape[1]
    r = O.compress_head(q, K, V, budget=12, mi_rounds=0)
    alpha = np.zeros(N)
    alpha[1:N - w] = r.abar
    prot = [0] + list(range(N - w, N))
    kept, m = O.greedy_evict(alpha, K, V, prot, budget=N - 1)
    ev = int(np.setdiff1d(np.arange(N), kept)[0])
    order = sorted(range(len(r.sigma0)), key=lambda i: (r.sigma0[i], i))
    assert ev == order[0] + 1
    assert m.n_e == 1


def test_moment_round_evicts_tokens_the_summary_already_predicts():
    """Closed-form case of the moment round (Sec. 4.2): dyadic values make every sum exact.

    Candidates 0-5 share one key and one small value v_A (low mass): round 0 evicts them,
    so the summary is v_bar = v_A, S_tilde = 0.  Candidates 6-7 ("twins") carry v_A too
    but high mass, so round 0 keeps them; their residual is then exactly 0, like that of
    0-5.  Candidates 8-11 have large distinct values.  With k_keep = 6 the moment round
    keeps 8-11 plus the two lowest-index zero-score tokens (0, 1): the twins go."""
    d = 4
    k_A = np.array([1.0, 0.5, -0.25, 2.0])
    v_A = np.array([0.125, -0.25, 0.0, 0.0625])
    K = np.zeros((12, d))
    V = np.zeros((12, d))
    K[:6], V[:6] = k_A, v_A
    K[6:8] = np.array([[0.5, 1.0, 1.0, -1.0], [-2.0, 0.25, 0.5, 1.0]])
    V[6:8] = v_A
    K[8:] = np.array([[1, 2, 3, 4], [-1, 0, 2, 1], [3, -2, 1, 0], [0, 1, -1, 2]], float)
    V[8:] = np.array([[4, 0, 1, 2], [0, -4, 2, 1], [2, 2, -4, 0], [-3, 1, 0, 4]], float)
    abar = np.array([1.0] * 6 + [10.0] * 2 + [1.0] * 4)
    sel = O.select_candidates(abar, K, V, 6, mi_rounds=1, scale=0.5, tau=1e-6)
    assert list(sel["rounds"][0]) == [6, 7, 8, 9, 10, 11]
    np.testing.assert_array_equal(sel["sigma"][:8], 0.0)
    assert list(sel["rounds"][1]) == [0, 1, 8, 9, 10, 11]
    np.testing.assert_allclose(sel["sigma"][8:], np.linalg.norm(V[8:] - v_A, axis=1), rtol=1e-15)


def test_compress_is_permutation_equivariant_without_chunks():
    """Window mass, residuals and moments depend on the candidate multiset only: permuting
    candidate rows (chunk = 1) permutes the selection and leaves the moments unchanged."""
    q, K, V = _tiny_prefill(22, N=40)
    N, w = len(K), q.shape[1]
    rng = np.random.default_rng(23)
    perm = np.arange(N)
    perm[1:N - w] = 1 + rng.permutation(N - w - 1)
    r1 = O.compress_head(q, K, V, budget=14, chunk=1)
    r2 = O.compress_head(q, K[perm], V[perm], budget=14, chunk=1)
    assert sorted(perm[r2.retained]) == list(r1.retained)
    np.testing.assert_allclose(r2.moments.S, r1.moments.S, rtol=1e-12)
    np.testing.assert_allclose(r2.moments.s_k, r1.moments.s_k, rtol=1e-12)


def test_compress_rejects_budget_below_sink_plus_window():
    q, K, V = _tiny_prefill(24)
    with pytest.raises(ValueError):
        O.compress_head(q, K, V, budget=q.shape[1])


def test_moment_storage_matches_paper_table():
    with open(os.path.join(GOLDEN, "storage_table.json")) as f:
        g = json.load(f)
    for row in g["rows"]:
        b = O.moment_storage_bytes(row["layers"], row["kv_heads"], row["head_dim"], 2)
        assert round(b / 1e6, 1) == row["moment_overhead_MB"]
    assert 128 * 128 * 2 == g["S_bytes_per_head_d128_16bit"]


def test_corrected_output_beats_retained_only_on_average():
    """Quality check (reported in Sec. 4.2 as the purpose of the correction): over random
    queries the corrected output is closer to full attention than f_R on average."""
    rng = np.random.default_rng(25)
    q, K, V = _tiny_prefill(26, G=2, w=4, d=16, N=200)
    r = O.compress_head(q, K, V, budget=40)
    gains = []
    for _ in range(30):
        qq = K[rng.integers(0, len(K), 4)].mean(axis=0) + 0.5 * rng.normal(size=16)
        full = sdpa(qq[None], K, V, 0.25)[0]
        dec = O.decode_head(qq, r.k_out, r.v_out, r.moments)
        gains.append(np.linalg.norm(full - dec.f_R) - np.linalg.norm(full - dec.out))
    assert np.mean(gains) > 0


# ------------------------------------------------------------ decode-time eviction
def _evict_case(rng, d=6, G=2, n_hist=9, L=7, key=None):
    """History of n_hist evicted tokens (their moments) and L retained rows in a cache of
    L+3 slots, plus a new token.  key: a shared key for every token (zero spread)."""
    def keys(n):
        return np.tile(key, (n, 1)) if key is not None else rng.normal(size=(n, d))
    KE, VE = keys(n_hist), rng.normal(size=(n_hist, d))
    m = O.evicted_moments(KE, VE, np.arange(n_hist))
    kc = np.zeros((L + 3, d))
    vc = np.zeros((L + 3, d))
    kc[:L], vc[:L] = keys(L), rng.normal(size=(L, d))
    k_new, v_new = keys(1)[0], rng.normal(size=d)
    q = rng.normal(size=(G, d))
    return q, kc, vc, m, k_new, v_new, (KE, VE)


def test_evict_zero_key_spread_evicts_value_nearest_mean_and_stays_exact():
    """Every key equal: S_tilde = 0 and alpha is uniform, so score_j is ||v_j - v_bar||
    up to a constant and the step evicts the retained value nearest the evicted mean
    (brute force).  After the rank-one update the corrected output is still exact full
    attention over every token seen, i.e. the plain mean of all values."""
    rng = np.random.default_rng(40)
    d, L = 6, 7
    key = rng.normal(size=d)
    q, kc, vc, m, k_new, v_new, (KE, VE) = _evict_case(rng, d=d, L=L, key=key)
    r = O.decode_evict_head(q, kc, vc, L, k_new, v_new, m, L)
    rows = [vc[i] for i in range(L)] + [v_new]
    v_bar = VE.mean(axis=0)
    dist = [math.sqrt(sum((a - b) ** 2 for a, b in zip(row, v_bar))) for row in rows]
    want = min(range(len(dist)), key=lambda i: (dist[i], i))
    assert r["evicted"] == want
    assert r["length"] == L
    every = np.vstack([VE] + rows)
    for g in range(q.shape[0]):
        np.testing.assert_allclose(r["out"][g], every.mean(axis=0), rtol=1e-10, atol=1e-12)
    assert r["moments"].n_e == len(VE) + 1


def test_evict_scores_follow_softmax_weights_at_equal_residual_norms():
    """With an empty summary r_j = v_j; values of equal norm make the score the group-mean
    softmax weight alone (torch softmax over the rows of each query), so the evicted
    row is the least attended on average."""
    rng = np.random.default_rng(41)
    d, G, L = 8, 3, 11
    for trial in range(6):
        q = rng.normal(size=(G, d)) * 2.0
        kc = np.zeros((L + 2, d))
        vc = np.zeros((L + 2, d))
        kc[:L] = rng.normal(size=(L, d))
        V = rng.normal(size=(L + 1, d))
        V /= np.linalg.norm(V, axis=1, keepdims=True)
        vc[:L] = V[:L]
        k_new = rng.normal(size=d)
        r = O.decode_evict_head(q, kc, vc, L, k_new, V[L], O.Moments.zeros(d), L)
        K = np.vstack([kc[:L], k_new[None]])
        logits = torch.from_numpy(K @ q.T / math.sqrt(d))          # [n, G]
        alpha = torch.softmax(logits, dim=0).mean(dim=1).numpy()
        want = int(np.argmin(alpha))
        assert r["evicted"] == want, trial
        np.testing.assert_allclose(r["alpha"], alpha, rtol=1e-12)
        np.testing.assert_allclose(r["rnorm"], 1.0, rtol=1e-12)


def test_evict_equal_scores_evict_lowest_slot():
    """Two identical rows share the minimal score: the lower slot is evicted and the
    last row moves into it."""
    rng = np.random.default_rng(42)
    d, L = 5, 6
    q, kc, vc, m, k_new, v_new, _ = _evict_case(rng, d=d, G=1, L=L)
    vc[:L] *= 4.0
    kc[2], vc[2] = k_new, v_new * 0.01        # rows 2 and L (the new one) are twins
    v_new = v_new * 0.01
    r = O.decode_evict_head(q, kc, vc, L, k_new, v_new, O.Moments.zeros(d), L)
    s = r["score"]
    assert s[2] == s[L] and s[2] == s.min()
    assert r["evicted"] == 2
    np.testing.assert_array_equal(r["v_cache"][2], v_new)


def test_evict_without_overflow_is_plain_decode_with_append():
    """While the cache holds fewer than `budget` rows nothing is evicted and the step is
    the corrected decode with the append."""
    rng = np.random.default_rng(43)
    d, G, L = 6, 2, 7
    q, kc, vc, m, k_new, v_new, _ = _evict_case(rng, d=d, G=G, L=L)
    r = O.decode_evict_head(q, kc, vc, L, k_new, v_new, m, L + 1)
    assert r["evicted"] == -1 and r["length"] == L + 1
    out, lz, wr, _ = O.decode(q[None], kc[None, None], vc[None, None], np.array([[L]]),
                              [[m]], k_new=k_new[None, None], v_new=v_new[None, None])
    np.testing.assert_allclose(r["out"], out[0], rtol=1e-13)
    np.testing.assert_allclose(r["w_R"], wr[0], rtol=1e-13)


def test_evict_steps_conserve_tokens_and_moments_sum_everything_evicted():
    """Over several steps: the retained rows and the evicted rows together are exactly the
    tokens seen, the cache stays at `budget` rows, and the summary equals brute-force
    sums over every evicted token (the compressed history and each step's victim)."""
    rng = np.random.default_rng(44)
    d, G, L, T = 6, 2, 6, 8
    q, kc, vc, m, k_new, v_new, (KE, VE) = _evict_case(rng, d=d, G=G, L=L)
    kc = np.zeros((L + 1, d)); vc = np.zeros((L + 1, d))
    kc[:L], vc[:L] = rng.normal(size=(L, d)), rng.normal(size=(L, d))
    seen_k, seen_v = [KE[i] for i in range(len(KE))] + list(kc[:L]), \
        [VE[i] for i in range(len(VE))] + list(vc[:L])
    gone_k, gone_v = [KE[i] for i in range(len(KE))], [VE[i] for i in range(len(VE))]
    n = L
    for t in range(T):
        kn, vn = rng.normal(size=d), rng.normal(size=d)
        seen_k.append(kn); seen_v.append(vn)
        qt = rng.normal(size=(G, d))
        pre_k = kc.copy(); pre_v = vc.copy()
        pre_k[n], pre_v[n] = kn, vn
        r = O.decode_evict_head(qt, kc, vc, n, kn, vn, m, L)
        j = r["evicted"]
        assert 0 <= j <= n and r["length"] == L
        gone_k.append(pre_k[j]); gone_v.append(pre_v[j])
        kc, vc, n, m = r["k_cache"], r["v_cache"], r["length"], r["moments"]
    def as_set(rows):
        return sorted(tuple(np.round(x, 12)) for x in rows)
    assert as_set(list(kc[:n]) + gone_k) == as_set(seen_k)
    assert as_set(list(vc[:n]) + gone_v) == as_set(seen_v)
    S = np.zeros((d, d)); sk = np.zeros(d); sv = np.zeros(d)
    for kk, vv in zip(gone_k, gone_v):
        for a in range(d):
            sk[a] += kk[a]; sv[a] += vv[a]
            for b in range(d):
                S[a, b] += vv[a] * kk[b]
    assert m.n_e == len(gone_k)
    np.testing.assert_allclose(m.s_k, sk, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(m.s_v, sv, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(m.S, S, rtol=1e-12, atol=1e-12)


def test_evict_batched_matches_per_head():
    rng = np.random.default_rng(45)
    B, Hkv, G, d, L = 2, 2, 2, 5, 5
    kc = rng.normal(size=(B, Hkv, L + 2, d)); vc = rng.normal(size=(B, Hkv, L + 2, d))
    lens = np.array([[L, L - 1], [L, L]])
    q = rng.normal(size=(B, Hkv * G, d))
    kn, vn = rng.normal(size=(B, Hkv, d)), rng.normal(size=(B, Hkv, d))
    mom = [[O.evicted_moments(rng.normal(size=(4, d)), rng.normal(size=(4, d)), np.arange(4))
            for _ in range(Hkv)] for _ in range(B)]
    out, lz, wr, (kc2, vc2, ln2, mom2), ev, _ = O.decode_evict(q, kc, vc, lens, mom, kn, vn, L)
    for b in range(B):
        for h in range(Hkv):
            r = O.decode_evict_head(q[b, h * G:(h + 1) * G], kc[b, h], vc[b, h], lens[b, h],
                                    kn[b, h], vn[b, h], mom[b][h], L)
            assert ev[b, h] == r["evicted"] and ln2[b, h] == r["length"]
            np.testing.assert_array_equal(out[b, h * G:(h + 1) * G], r["out"])
            np.testing.assert_array_equal(kc2[b, h], r["k_cache"])
    assert ev[0, 1] == -1 and ln2[0, 1] == L


# ------------------------------------------------------------ head-adaptive budgets
def test_head_budgets_match_bruteforce_sort_with_ties():
    """Per-head counts equal a brute-force Python sort of (-mass, head, position) over the
    layer, with planted equal masses inside and across heads."""
    rng = np.random.default_rng(50)
    for trial in range(20):
        H, n = int(rng.integers(2, 5)), int(rng.integers(5, 14))
        a = rng.integers(0, 6, size=(H, n)).astype(float) / 7.0   # many ties
        k = int(rng.integers(0, n + 1))
        items = sorted((-a[h, j], h, j) for h in range(H) for j in range(n))[:H * k]
        want = [sum(1 for _, h, _ in items if h == hh) for hh in range(H)]
        got = O.head_budgets(a, k)
        assert list(got) == want, trial
        assert got.sum() == H * k


def test_head_budgets_one_head_is_the_uniform_budget():
    rng = np.random.default_rng(51)
    a = rng.random((1, 40))
    for k in (0, 1, 17, 40):
        assert list(O.head_budgets(a, k)) == [k]


def test_adaptive_compress_of_identical_heads_is_uniform():
    """Heads with identical queries, keys and values (no chunk pooling, continuous masses)
    split the layer budget evenly, so adaptive compress equals uniform compress."""
    q, K, V = _tiny_prefill(52, G=2, w=4, d=8, N=90)
    H = 3
    qq = np.concatenate([q] * H)[None]                  # [1, H*G, w, d]
    KK = np.stack([K] * H)[None]
    VV = np.stack([V] * H)[None]
    ada = O.compress(qq, KK, VV, 30, adaptive=True, chunk=1)
    uni = O.compress(qq, KK, VV, 30, chunk=1)
    for h in range(H):
        np.testing.assert_array_equal(ada[0][h].idx, uni[0][h].idx)
        np.testing.assert_allclose(ada[0][h].moments.S, uni[0][h].moments.S)


def test_adaptive_compress_counts_and_summaries():
    """Heads keep n_sink + w + k_h tokens with sum k_h = Hkv * k_keep; each head's summary is
    the brute-force moment sums over its own evicted candidates."""
    rng = np.random.default_rng(53)
    H, G, w, d, N, L = 3, 2, 4, 8, 80, 20
    q = rng.normal(size=(1, H * G, w, d))
    K = rng.normal(size=(1, H, N, d))
    K[0, 1] *= 2.5                                         # a sharper head
    V = rng.normal(size=(1, H, N, d))
    res = O.compress(q, K, V, L, adaptive=True)
    kh = [len(r.retained) for r in res[0]]
    assert sum(kh) == H * (L - 1 - w) and len(set(kh)) > 1
    for h in range(H):
        r = res[0][h]
        assert len(r.idx) == 1 + w + kh[h]
        E = np.setdiff1d(np.arange(1, N - w), r.retained)
        np.testing.assert_array_equal(E, r.evicted)
        S = sum(np.outer(V[0, h, i], K[0, h, i]) for i in E)
        np.testing.assert_allclose(r.moments.S, S, rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------ grouped-query head mapping
def sdpa_gqa(q, K, V, scale, mask=None):
    """torch SDPA with grouped queries (enable_gqa): q [B,Hq,m,d], K [B,Hkv,n,d],
    V [B,Hkv,n,e] -> [B,Hq,m,e], fp64."""
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x, np.float64))
    m = None if mask is None else torch.from_numpy(mask)
    return F.scaled_dot_product_attention(t(q), t(K), t(V), attn_mask=m, scale=scale,
                                          enable_gqa=True).numpy()


def torch_kv_head_of(Hq, Hkv):
    """The KV head torch's grouped-query SDPA gives each query head: every value row
    carries a one-hot of its head's index, so each query head's output names its head.
    This is the GQA layout (Sec. 5.1: 32 query heads over 8 KV heads) taken from a
    library, not from the oracle."""
    q = np.ones((1, Hq, 1, 4))
    K = np.zeros((1, Hkv, 1, 4))
    V = np.eye(Hkv)[None, :, None, :]
    return sdpa_gqa(q, K, V, 1.0)[0, :, 0, :].argmax(axis=-1)


def test_batched_decode_reads_the_kv_head_of_each_query_group():
    """oracle.decode over [B, Hq] queries and [B, Hkv] caches: without correction it is
    torch's grouped-query SDPA over each head's retained rows; with the correction each
    query head's output is decode_head against the KV head (lens, rows and summary)
    that torch assigns it."""
    rng = np.random.default_rng(60)
    B, Hq, Hkv, d, cap, n = 2, 8, 2, 8, 12, 10
    q = rng.normal(size=(B, Hq, d)) * 1.5
    kc = rng.normal(size=(B, Hkv, cap, d))
    vc = rng.normal(size=(B, Hkv, cap, d))
    kc[:, 1] += 2.0                                        # heads that differ in law
    mom = [[O.evicted_moments(rng.normal(size=(5, d)), rng.normal(size=(5, d)) + 3.0 * h,
                              np.arange(5)) for h in range(Hkv)] for _ in range(B)]
    scale = 1 / math.sqrt(d)
    want = sdpa_gqa(q[:, :, None], kc[:, :, :n], vc[:, :, :n], scale)[:, :, 0]
    lens = np.full((B, Hkv), n)
    out, lz, wr, _ = O.decode(q, kc, vc, lens, mom, order=-1)
    np.testing.assert_allclose(out, want, rtol=1e-12, atol=1e-14)
    zero = [[O.Moments.zeros(d) for _ in range(Hkv)] for _ in range(B)]
    out0, _, _, _ = O.decode(q, kc, vc, lens, zero)
    np.testing.assert_allclose(out0, want, rtol=1e-12, atol=1e-14)
    grp = torch_kv_head_of(Hq, Hkv)
    lens = np.array([[7, 11], [12, 3]])
    out1, lz1, wr1, _ = O.decode(q, kc, vc, lens, mom)
    for b in range(B):
        for hq in range(Hq):
            h = grp[hq]
            r = O.decode_head(q[b, hq], kc[b, h, :lens[b, h]], vc[b, h, :lens[b, h]], mom[b][h])
            np.testing.assert_allclose(out1[b, hq], r.out, rtol=1e-13)
            np.testing.assert_allclose(lz1[b, hq], r.log_Z_R, rtol=1e-13)
            np.testing.assert_allclose(wr1[b, hq], r.w_R, rtol=1e-13)


def test_batched_compress_window_mass_groups_queries_by_kv_head():
    """Each KV head's window mass is the mean of the softmax probabilities of the query
    heads torch's grouped-query SDPA sends to it: one-hot values over positions, plus a
    one-hot of the KV head's index that names the group."""
    rng = np.random.default_rng(61)
    B, Hq, Hkv, w, d, N = 2, 6, 3, 4, 8, 40
    q = rng.normal(size=(B, Hq, w, d)) * 1.5
    K = rng.normal(size=(B, Hkv, N, d)) * (1.0 + np.arange(Hkv))[None, :, None, None]
    V = rng.normal(size=(B, Hkv, N, d))
    scale = 1 / math.sqrt(d)
    onehot = np.zeros((B, Hkv, N, N + Hkv))
    onehot[:, :, :, :N] = np.eye(N)
    for h in range(Hkv):
        onehot[:, h, :, N + h] = 1.0
    band = torch.ones(w, N, dtype=torch.bool).tril(diagonal=N - w).numpy()
    P = sdpa_gqa(q, K, onehot, scale, band)                 # [B, Hq, w, N + Hkv]
    res = O.compress(q, K, V, 1 + w + 6)
    for b in range(B):
        head = P[b, :, 0, N:].argmax(axis=-1)              # the KV head of each query head
        for h in range(Hkv):
            rows = P[b, head == h, :, : N - w].reshape(-1, N - w)
            assert rows.shape[0] == w * Hq // Hkv
            np.testing.assert_allclose(res[b][h].a, rows.mean(axis=0), rtol=1e-12, atol=1e-15)


def test_batched_decode_evict_scores_each_kv_head_with_its_query_group():
    """With an empty summary and unit-norm values the evicted row of each KV head is the
    one with the lowest mean softmax weight over the query heads torch's grouped-query
    SDPA sends to that head; without correction the output is that SDPA over the cache
    left after the eviction."""
    rng = np.random.default_rng(62)
    B, Hq, Hkv, d, L = 1, 6, 2, 8, 9
    grp = torch_kv_head_of(Hq, Hkv)
    scale = 1 / math.sqrt(d)
    for trial in range(8):
        q = rng.normal(size=(B, Hq, d)) * 2.5
        kc = np.zeros((B, Hkv, L + 2, d))
        vc = np.zeros((B, Hkv, L + 2, d))
        kc[:, :, :L] = rng.normal(size=(B, Hkv, L, d))
        V = rng.normal(size=(B, Hkv, L + 1, d))
        V /= np.linalg.norm(V, axis=-1, keepdims=True)
        vc[:, :, :L] = V[:, :, :L]
        kn = rng.normal(size=(B, Hkv, d))
        lens = np.full((B, Hkv), L)
        zero = [[O.Moments.zeros(d) for _ in range(Hkv)] for _ in range(B)]
        out, _, _, (kc2, vc2, ln2, _), ev, _ = O.decode_evict(q, kc, vc, lens, zero, kn,
                                                              V[:, :, L], L, order=-1)
        for b in range(B):
            for h in range(Hkv):
                Kh = np.vstack([kc[b, h, :L], kn[b, h][None]])
                logits = torch.from_numpy(q[b, grp == h] @ Kh.T * scale)   # [G, n]
                alpha = torch.softmax(logits, dim=1).mean(dim=0).numpy()
                assert ev[b, h] == int(np.argmin(alpha)), (trial, h)
        want = sdpa_gqa(q[:, :, None], kc2[:, :, :L], vc2[:, :, :L], scale)[:, :, 0]
        assert (ln2 == L).all()
        np.testing.assert_allclose(out, want, rtol=1e-12, atol=1e-14)
