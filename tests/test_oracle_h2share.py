"""Pins of the H2Share oracle (cross-layer head mapping, anchor top-k,
reuse-layer sparse decode) against facts the paper and the mathematics fix."""
import numpy as np
import pytest

from oracle import attention as OA
from oracle import h2share as HS


def _weights(hq, hkv, d, dm, seed):
    r = np.random.default_rng(seed)
    return r.standard_normal((hq * d, dm)), r.standard_normal((hkv * d, dm))


@pytest.mark.parametrize("hq,hkv,d,dm,seed", [(4, 2, 8, 24, 0), (6, 3, 4, 16, 1), (2, 2, 8, 8, 2)])
def test_trace_form_equals_dense_frobenius(hq, hkv, d, dm, seed):
    wq_a, wk_a = _weights(hq, hkv, d, dm, seed)
    wq_r, wk_r = _weights(hq, hkv, d, dm, seed + 10)
    fast = HS.head_similarity(wq_a, wk_a, wq_r, wk_r, d)
    dense = HS.frobenius_similarity_dense(wq_a, wk_a, wq_r, wk_r, d)
    np.testing.assert_allclose(fast, dense, rtol=1e-9, atol=1e-12)


def test_self_similarity_bounds_and_transpose():
    wq_a, wk_a = _weights(8, 4, 8, 32, 3)
    wq_r, wk_r = _weights(8, 4, 8, 32, 4)
    self_sim = HS.head_similarity(wq_a, wk_a, wq_a, wk_a, 8)
    np.testing.assert_allclose(np.diag(self_sim), 1.0, atol=1e-12)
    m = HS.head_similarity(wq_a, wk_a, wq_r, wk_r, 8)
    assert np.all(np.abs(m) <= 1 + 1e-12)
    np.testing.assert_allclose(HS.head_similarity(wq_r, wk_r, wq_a, wk_a, 8), m.T, rtol=1e-12, atol=1e-14)


def _permuted_reuse(wq, wk, perm, d, gs, seed):
    """Reuse layer whose group g' is a rescaled copy of anchor group perm[g']
    (queries and key), plus small noise."""
    r = np.random.default_rng(seed)
    wq_r, wk_r = np.empty_like(wq), np.empty_like(wk)
    for g2, g in enumerate(perm):
        s = r.uniform(0.5, 2.0)
        wk_r[g2 * d:(g2 + 1) * d] = s * wk[g * d:(g + 1) * d]
        wq_r[g2 * gs * d:(g2 + 1) * gs * d] = r.uniform(0.5, 2.0) * wq[g * gs * d:(g + 1) * gs * d]
    return wq_r + 1e-3 * r.standard_normal(wq.shape), wk_r + 1e-3 * r.standard_normal(wk.shape)


def test_permuted_copies_map_back():
    d, gs, hkv = 8, 2, 4
    wq, wk = _weights(gs * hkv, hkv, d, 64, 5)
    perm = [2, 0, 3, 1]
    wq_r, wk_r = _permuted_reuse(wq, wk, perm, d, gs, 6)
    hsim = HS.head_similarity(wq, wk, wq_r, wk_r, d)
    gsim = HS.group_similarity(hsim, hkv)
    for g2, g in enumerate(perm):
        # copied head pairs are identical up to scale (similarity 1); the group
        # mean over the gs x gs head pairs is then about 1/gs, far above the rest
        for j in range(gs):
            assert hsim[g * gs + j, g2 * gs + j] > 0.99
        assert gsim[g, g2] > np.delete(gsim[:, g2], g).max() + 0.3
    assert HS.group_mapping(gsim, [0] * 4, [0] * 4).tolist() == perm
    # only retrieval anchors are candidates; streaming reuse groups get -1
    # reuse groups 1 and 2 copy anchor groups 0 and 3, the anchor's two retrieval groups
    m = HS.group_mapping(gsim, [0, 1, 1, 0], [1, 0, 0, 1])
    assert m.tolist() == [-1, 0, 3, -1]
    assert HS.mapping_to_rank(m, [0, 1, 1, 0]).tolist() == [-1, 0, 1, -1]


def test_group_similarity_is_block_mean():
    hs = np.arange(36, dtype=float).reshape(6, 6)
    gsim = HS.group_similarity(hs, 3)
    assert gsim[0, 0] == np.mean([0, 1, 6, 7]) and gsim[2, 1] == np.mean([26, 27, 32, 33])


def test_top_k_hand_listed():
    s = [0.1, 0.3, 0.3, 0.2, 0.3, 0.05]
    assert HS.top_k_positions(s, 2).tolist() == [1, 2]
    assert HS.top_k_positions(s, 4).tolist() == [1, 2, 3, 4]
    assert HS.top_k_positions(s, 6).tolist() == [0, 1, 2, 3, 4, 5]
    assert HS.top_k_positions(s, 8).tolist() == [0, 1, 2, 3, 4, 5, -1, -1]
    assert HS.top_k_positions([0.5], 1).tolist() == [0]


def test_top_k_brute_force():
    r = np.random.default_rng(7)
    for n, k in [(50, 7), (33, 33), (10, 3)]:
        s = np.round(r.random(n), 1)  # many ties
        got = set(HS.top_k_positions(s, k).tolist())
        # brute force: a position is kept iff fewer than k positions beat it,
        # counting equal scores at lower positions as beating it
        want = {j for j in range(n) if sum(1 for i in range(n) if s[i] > s[j] or (s[i] == s[j] and i < j)) < k}
        assert got == want


def _seq(B, L, hkv, d, seed):
    r = np.random.default_rng(seed)
    return r.standard_normal((B, L, hkv, d)), r.standard_normal((B, L, hkv, d))


def test_reuse_with_every_position_is_full_decode():
    B, L, hq, hkv, d = 2, 40, 4, 2, 8
    k, v = _seq(B, L, hkv, d, 8)
    q = np.random.default_rng(9).standard_normal((B, hq, d))
    lens = [40, 23]
    mask = [0, 0]
    idx = np.full((B, 2, L), -1)
    for b in range(B):
        idx[b, :, :lens[b]] = np.arange(lens[b])
    got = HS.reuse_decode(q, k, v, lens, mask, 4, 8, idx, [1, 0])
    want = OA.decode(q, k, v, lens, mask, 4, 8)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


def test_reuse_with_sink_and_window_is_streaming_decode():
    B, L, hq, hkv, d, n_sink, window = 1, 60, 4, 2, 8, 3, 10
    k, v = _seq(B, L, hkv, d, 10)
    q = np.random.default_rng(11).standard_normal((B, hq, d))
    lens = [57]
    p = lens[0] - 1
    keep = [j for j in range(lens[0]) if j < n_sink or p - j < window]
    idx = np.array([[keep + [-1] * 3]])
    got = HS.reuse_decode(q, k, v, lens, [0, 1], n_sink, window, idx, [0, -1])
    want = OA.decode(q, k, v, lens, [1, 1], n_sink, window)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


def test_reuse_follows_the_mapping():
    # anchor list 0 = every position, anchor list 1 = the last 6 positions;
    # reuse group 0 borrows list 1 (a window of 6, no sink), group 1 list 0 (full)
    B, L, hq, hkv, d = 1, 30, 4, 2, 8
    k, v = _seq(B, L, hkv, d, 14)
    q = np.random.default_rng(15).standard_normal((B, hq, d))
    lens = [25]
    idx = np.full((1, 2, 25), -1)
    idx[0, 0] = np.arange(25)
    idx[0, 1, :6] = np.arange(19, 25)
    got = HS.reuse_decode(q, k, v, lens, [0, 0], 0, 6, idx, [1, 0])
    window6 = OA.decode(q, k, v, lens, [1, 1], 0, 6)
    full = OA.decode(q, k, v, lens, [0, 0], 0, 6)
    np.testing.assert_allclose(got[0, :2], window6[0, :2], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(got[0, 2:], full[0, 2:], rtol=1e-12, atol=1e-12)


def test_anchor_scores_are_group_mean_probabilities():
    B, L, hq, hkv, d = 1, 30, 4, 2, 8
    k, _ = _seq(B, L, hkv, d, 12)
    q = np.random.default_rng(13).standard_normal((B, hq, d))
    lens = [30]
    sc = HS.group_scores(q, k, lens, 0, 1, hkv)
    w2 = OA.attention_weights(q[0, 2][None], [29], k[0, :, 1], False, 0, 1)[0]
    w3 = OA.attention_weights(q[0, 3][None], [29], k[0, :, 1], False, 0, 1)[0]
    np.testing.assert_allclose(sc, (w2 + w3) / 2, rtol=1e-12)
    assert abs(sc.sum() - 1) < 1e-12
    idx = HS.anchor_select(q, k, lens, [1, 0], 5)
    assert idx.shape == (1, 1, 5) and idx[0, 0].tolist() == HS.top_k_positions(sc, 5).tolist()


def test_planted_mistakes_are_caught(monkeypatch):
    def pins_hold():
        try:
            test_trace_form_equals_dense_frobenius(4, 2, 8, 24, 0)
            test_permuted_copies_map_back()
            test_top_k_hand_listed()
            test_top_k_brute_force()
            test_reuse_with_every_position_is_full_decode()
            test_reuse_follows_the_mapping()
            test_anchor_scores_are_group_mean_probabilities()
        except AssertionError:
            return False
        return True

    assert pins_hold()
    good = {n: getattr(HS, n) for n in ("head_similarity", "group_mapping", "top_k_positions", "reuse_decode")}

    def no_norm(wq_a, wk_a, wq_r, wk_r, d):  # inner product without the normalisation
        hq = wq_a.shape[0] // d
        hkv = wk_a.shape[0] // d
        out = np.empty((hq, hq))
        for h in range(hq):
            for h2 in range(hq):
                qa, ka = wq_a[h * d:(h + 1) * d], wk_a[(h // (hq // hkv)) * d:][:d]
                qr, kr = wq_r[h2 * d:(h2 + 1) * d], wk_r[(h2 // (hq // hkv)) * d:][:d]
                out[h, h2] = np.trace((qa @ qr.T) @ (kr @ ka.T))
        return out

    def keys_same_layer(wq_a, wk_a, wq_r, wk_r, d):  # anchor keys on both sides
        return good["head_similarity"](wq_a, wk_a, wq_r, wk_a, d)

    def argmin_map(gsim, a, r):
        return good["group_mapping"](-gsim, a, r)

    def ties_high(s, k):
        s = np.asarray(s)
        order = np.lexsort((-np.arange(len(s)), -s))
        sel = np.sort(order[:k])
        return np.concatenate([sel, np.full(k - len(sel), -1)]).astype(np.int64)

    def reuse_same_index(q, k, v, lens, mask, ns, w, idx, mapping):  # ignores the mapping
        return good["reuse_decode"](q, k, v, lens, mask, ns, w, idx, [0] * len(mapping))

    for name, fn in [("head_similarity", no_norm), ("head_similarity", keys_same_layer),
                     ("group_mapping", argmin_map), ("top_k_positions", ties_high),
                     ("reuse_decode", reuse_same_index)]:
        monkeypatch.setattr(HS, name, fn)
        assert not pins_hold(), fn.__name__
        monkeypatch.setattr(HS, name, good[name])
