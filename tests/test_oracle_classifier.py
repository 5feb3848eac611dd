"""Pins of the classifier oracle (paper Sec. 4 and Algorithm 1) against facts
the mathematics fixes: the proxy spectrum against a dense SVD of M_h, planted
spectra with closed-form effective ranks, invariances, and hand-built layers
whose labels follow from the planted ranks."""
import math

import numpy as np
import pytest

from oracle import classifier as CL


def _orthonormal_rows(n, d_model, seed):
    """n x d_model matrix with orthonormal rows (QR of a Gaussian matrix)."""
    g = np.random.default_rng(seed).standard_normal((d_model, n))
    q, _ = np.linalg.qr(g)
    return q.T


def _planted(s, d_head, d_model, seed):
    """W_Q = diag(s) P, W_K = P with P orthonormal rows: M_h = P^T diag(s) P,
    whose singular values are exactly s (zero-padded to d_head)."""
    p = _orthonormal_rows(d_head, d_model, seed)
    s = np.concatenate([np.asarray(s, np.float64), np.zeros(d_head - len(s))])
    return s[:, None] * p, p


@pytest.mark.parametrize("d_head,d_model,seed", [(8, 40, 0), (16, 48, 1), (4, 4, 2), (32, 64, 3)])
def test_proxy_spectrum_equals_dense_svd(d_head, d_model, seed):
    r = np.random.default_rng(seed)
    wq = r.standard_normal((d_head, d_model))
    wk = r.standard_normal((d_head, d_model)) * np.linspace(0.2, 3.0, d_head)[:, None]
    full = CL.singular_values_full(wq, wk)
    proxy = CL.singular_values(wq, wk)
    np.testing.assert_allclose(proxy, full[:d_head], rtol=1e-9, atol=1e-9 * full[0])
    assert np.all(full[d_head:] <= 1e-9 * full[0])  # rank(M_h) <= d_head
    assert abs(CL.effective_rank(proxy) - CL.effective_rank(full[:d_head])) < 1e-9


@pytest.mark.parametrize("rank", [1, 3, 8])
def test_flat_spectrum_gives_its_rank(rank):
    wq, wk = _planted([2.5] * rank, 8, 32, rank)
    assert abs(CL.effective_rank(CL.singular_values(wq, wk)) - rank) < 1e-9


@pytest.mark.parametrize("s,want", [
    ([2, 1, 1], 2 ** 1.5),          # p = (1/2, 1/4, 1/4): entropy 1.5 ln 2
    ([4, 2, 1, 1], 2 ** 1.75),      # p = (1/2, 1/4, 1/8, 1/8): entropy 1.75 ln 2
    ([1, 1, 1, 1], 4.0),
    ([7], 1.0),
])
def test_closed_form_effective_ranks(s, want):
    wq, wk = _planted(s, 8, 24, 7)
    assert abs(CL.effective_rank(CL.singular_values(wq, wk)) - want) < 1e-9


def test_rank_one_query_projection():
    r = np.random.default_rng(4)
    wq = np.outer(r.standard_normal(16), r.standard_normal(64))
    wk = r.standard_normal((16, 64))
    assert abs(CL.effective_rank(CL.singular_values(wq, wk)) - 1.0) < 1e-6


def test_invariances_and_bounds():
    r = np.random.default_rng(5)
    d_head, d_model = 16, 48
    wq = r.standard_normal((d_head, d_model)) * np.geomspace(1, 0.05, d_head)[:, None]
    wk = r.standard_normal((d_head, d_model))
    er = CL.effective_rank(CL.singular_values(wq, wk))
    assert 1.0 <= er <= d_head
    # scaling either projection leaves the normalised spectrum unchanged
    assert abs(CL.effective_rank(CL.singular_values(3.0 * wq, 0.1 * wk)) - er) < 1e-9
    # an orthogonal change of basis of the model space: M -> R^T M R
    rot, _ = np.linalg.qr(r.standard_normal((d_model, d_model)))
    assert abs(CL.effective_rank(CL.singular_values(wq @ rot, wk @ rot)) - er) < 1e-9
    # the same orthogonal map on the head space of both projections cancels in W_K^T W_Q
    o, _ = np.linalg.qr(r.standard_normal((d_head, d_head)))
    assert abs(CL.effective_rank(CL.singular_values(o @ wq, o @ wk)) - er) < 1e-9
    # ... but not on one side only (the score depends on how Q and K align)
    assert abs(CL.effective_rank(CL.singular_values(o @ wq, wk)) - er) > 1e-3


def _layer(head_flat_ranks, n_kv, d_head=8, d_model=32, seed=0):
    """A layer whose query head h has a flat spectrum of the given rank with its
    group's key projection: W_K^g = P (orthonormal rows), W_Q^h = first r rows
    of P, padded with zero rows."""
    p = _orthonormal_rows(d_head, d_model, seed)
    wq = []
    for r in head_flat_ranks:
        w = np.zeros((d_head, d_model))
        w[:r] = p[:r]
        wq.append(w)
    return np.concatenate(wq), np.concatenate([p] * n_kv)


def test_group_mean_and_labels():
    wq, wk = _layer([8, 8, 2, 4, 5, 5, 1, 3], 4)
    out = CL.classify_layer(wq, wk, 8, sparsity=0.5)
    np.testing.assert_allclose(out["head_rank"], [8, 8, 2, 4, 5, 5, 1, 3], atol=1e-9)
    np.testing.assert_allclose(out["group_score"], [8, 3, 5, 2], atol=1e-9)
    assert out["head_is_streaming"].tolist() == [1, 0, 1, 0]
    # 25% sparsity: ceil(0.75 * 4) = 3 retrieval groups
    assert CL.classify_layer(wq, wk, 8, sparsity=0.25)["head_is_streaming"].tolist() == [1, 0, 0, 0]


def test_ties_keep_exactly_k_lowest_index_first():
    wq, wk = _layer([4] * 8, 4)
    assert CL.classify_layer(wq, wk, 8, n_retrieval=2)["head_is_streaming"].tolist() == [0, 0, 1, 1]
    wq, wk = _layer([6, 6, 3, 3, 3, 3, 6, 6], 4)
    assert CL.classify_layer(wq, wk, 8, n_retrieval=1)["head_is_streaming"].tolist() == [1, 0, 1, 1]


def test_model_stacks_layers():
    a, b = _layer([8, 8, 2, 4, 5, 5, 1, 3], 4, seed=1), _layer([1, 1, 2, 2, 3, 3, 4, 4], 4, seed=2)
    out = CL.classify_model(np.stack([a[0], b[0]]), np.stack([a[1], b[1]]), 8, sparsity=0.5)
    assert out["head_is_streaming"].tolist() == [[1, 0, 1, 0], [0, 0, 1, 1]]


def test_planted_mistakes_are_caught(monkeypatch):
    """Plausible mistakes planted in the oracle (CPU only) fail one of the pins."""
    def pins_hold():
        try:
            test_proxy_spectrum_equals_dense_svd(8, 40, 0)
            test_closed_form_effective_ranks([2, 1, 1], 2 ** 1.5)
            test_group_mean_and_labels()
            test_ties_keep_exactly_k_lowest_index_first()
        except AssertionError:
            return False
        return True

    good = {n: getattr(CL, n) for n in ("singular_values", "effective_rank", "group_scores", "select_retrieval")}
    assert pins_hold()

    def eig_not_sqrt(wq, wk):  # lambda used as sigma
        return np.sort(np.maximum(np.linalg.eigvals(CL.proxy_matrix(wq, wk)).real, 0))[::-1]

    def cross_gram(wq, wk):  # singular values of W_K W_Q^T instead of W_K^T W_Q
        return np.linalg.svd(np.asarray(wk) @ np.asarray(wq).T, compute_uv=False)

    def entropy_not_exp(sigma):  # entropy itself instead of its exponential
        return math.log(good["effective_rank"](sigma))

    def unnormalised(sigma):  # sigma not divided by its sum
        s = np.asarray(sigma, np.float64)
        s = s[s > 0]
        return float(np.exp(-np.sum(s * np.log(s))))

    def group_max(r, n_kv):
        return np.asarray(r).reshape(n_kv, -1).max(axis=1)

    def reverse(scores, k):  # highest scores kept as retrieval
        return good["select_retrieval"](-np.asarray(scores), k)

    def unstable(scores, k):  # ties broken toward the higher index
        s = np.asarray(scores)
        order = np.lexsort((-np.arange(len(s)), s))
        m = np.ones(len(s), np.uint8)
        m[order[:k]] = 0
        return m

    mutants = [("singular_values", eig_not_sqrt), ("singular_values", cross_gram),
               ("effective_rank", entropy_not_exp), ("effective_rank", unnormalised),
               ("group_scores", group_max), ("select_retrieval", reverse), ("select_retrieval", unstable)]
    for name, fn in mutants:
        monkeypatch.setattr(CL, name, fn)
        assert not pins_hold(), fn.__name__
        monkeypatch.setattr(CL, name, good[name])
    assert pins_hold()
