"""Pins for oracle.attention: each check fixes the oracle against something
other than itself (a library routine, a closed form, a hand-listed mask, an
independent brute force, an invariant of the definition)."""
import numpy as np
import pytest
import torch

from oracle import attention as A


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def _sdpa_causal(q, k, v):
    """torch's scaled_dot_product_attention (float64, CPU, causal) with each KV
    head repeated over its group of Hq/Hkv consecutive query heads."""
    b, t, hq, d = q.shape
    gs = hq // k.shape[2]
    qt = torch.from_numpy(q).permute(0, 2, 1, 3)
    kt = torch.from_numpy(k).permute(0, 2, 1, 3).repeat_interleave(gs, dim=1)
    vt = torch.from_numpy(v).permute(0, 2, 1, 3).repeat_interleave(gs, dim=1)
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True)
    return o.permute(0, 2, 1, 3).numpy()


@pytest.mark.parametrize("b,t,hq,hkv,d", [(2, 97, 6, 2, 16), (1, 64, 4, 4, 8), (1, 33, 8, 1, 32)])
def test_all_retrieval_equals_library_causal_attention(b, t, hq, hkv, d):
    q, k, v = _rand((b, t, hq, d), 1), _rand((b, t, hkv, d), 2), _rand((b, t, hkv, d), 3)
    o = A.prefill(q, k, v, np.zeros(hkv, np.uint8), n_sink=4, window=8)
    np.testing.assert_allclose(o, _sdpa_causal(q, k, v), rtol=0, atol=1e-12)


@pytest.mark.parametrize("n_sink,window", [(0, 50), (3, 50), (50, 1), (60, 7)])
def test_window_or_sink_covering_sequence_equals_dense(n_sink, window):
    # window >= T or n_sink >= T: every causal key is visible
    b, t, hq, hkv, d = 1, 50, 4, 2, 16
    q, k, v = _rand((b, t, hq, d), 4), _rand((b, t, hkv, d), 5), _rand((b, t, hkv, d), 6)
    o = A.prefill(q, k, v, np.ones(hkv, np.uint8), n_sink=n_sink, window=window)
    np.testing.assert_allclose(o, _sdpa_causal(q, k, v), rtol=0, atol=1e-12)


def test_window_one_without_sink_returns_own_value_exactly():
    # n_sink = 0, window = 1: each query sees only itself, with weight exactly 1
    b, t, hq, hkv, d = 2, 40, 4, 2, 16
    q, k, v = _rand((b, t, hq, d), 7), _rand((b, t, hkv, d), 8), _rand((b, t, hkv, d), 9)
    o = A.prefill(q, k, v, np.ones(hkv, np.uint8), n_sink=0, window=1)
    for h in range(hq):
        assert np.array_equal(o[:, :, h, :], v[:, :, h // 2, :])


def _mean_visible_position(i, streaming, n_sink, window):
    # closed form with arithmetic series: recent block [lo, i], sink block [0, min(n_sink, lo))
    if not streaming:
        return i / 2.0
    lo = max(0, i - window + 1)
    s = min(n_sink, lo)
    n_recent, sum_recent = i - lo + 1, (lo + i) * (i - lo + 1) / 2.0
    n_sink_vis, sum_sink = s, s * (s - 1) / 2.0
    return (sum_recent + sum_sink) / (n_recent + n_sink_vis)


@pytest.mark.parametrize("n_sink,window", [(4, 32), (0, 5), (16, 16), (1, 200)])
def test_zero_keys_give_mean_of_visible_positions(n_sink, window):
    # K = 0 makes every visible weight equal; with V[j] = j the output is the
    # mean visible position, known in closed form
    b, t, hq, hkv, d = 1, 150, 4, 2, 8
    q = _rand((b, t, hq, d), 10)
    k = np.zeros((b, t, hkv, d))
    v = np.broadcast_to(np.arange(t, dtype=np.float64)[None, :, None, None], (b, t, hkv, d)).copy()
    mask = np.array([0, 1], np.uint8)
    o = A.prefill(q, k, v, mask, n_sink, window)
    for h in range(hq):
        st = bool(mask[h // 2])
        want = np.array([_mean_visible_position(i, st, n_sink, window) for i in range(t)])
        np.testing.assert_allclose(o[0, :, h, 0], want, rtol=0, atol=1e-9)


def test_hand_listed_visible_sets():
    # n_sink = 2, window = 3 over 10 positions, written out by hand
    want = {
        0: {0}, 1: {0, 1}, 2: {0, 1, 2}, 3: {0, 1, 2, 3}, 4: {0, 1, 2, 3, 4},
        5: {0, 1, 3, 4, 5}, 6: {0, 1, 4, 5, 6}, 7: {0, 1, 5, 6, 7},
        8: {0, 1, 6, 7, 8}, 9: {0, 1, 7, 8, 9},
    }
    m = A.visible_mask(np.arange(10), 10, True, 2, 3)
    for i in range(10):
        assert set(np.nonzero(m[i])[0].tolist()) == want[i], i
    r = A.visible_mask(np.arange(10), 10, False, 2, 3)
    for i in range(10):
        assert set(np.nonzero(r[i])[0].tolist()) == set(range(i + 1))


def test_weights_rows_sum_to_one_and_vanish_off_mask():
    t, d = 45, 16
    q, k = _rand((t, d), 11), _rand((t, d), 12)
    for st in (False, True):
        p = A.attention_weights(q, np.arange(t), k, st, 3, 9)
        np.testing.assert_allclose(p.sum(axis=1), 1.0, rtol=0, atol=1e-12)
        m = A.visible_mask(np.arange(t), t, st, 3, 9)
        assert np.all(p[~m] == 0)
        assert np.all(p[m] > 0)


@pytest.mark.parametrize("n_sink,window", [(2, 5), (0, 1), (4, 40), (7, 3)])
def test_brute_force_explicit_mask_agrees(n_sink, window):
    b, t, hq, hkv, d = 1, 24, 4, 2, 8
    q, k, v = _rand((b, t, hq, d), 13), _rand((b, t, hkv, d), 14), _rand((b, t, hkv, d), 15)
    mask = np.array([1, 0], np.uint8)
    o = A.prefill(q, k, v, mask, n_sink, window)
    ob = A.brute_force(q, k, v, mask, n_sink, window)
    np.testing.assert_allclose(o, ob, rtol=0, atol=1e-12)


def test_decode_equals_prefill_row():
    b, t, hq, hkv, d = 2, 70, 6, 3, 16
    q, k, v = _rand((b, t, hq, d), 16), _rand((b, t, hkv, d), 17), _rand((b, t, hkv, d), 18)
    mask = np.array([0, 1, 1], np.uint8)
    o = A.prefill(q, k, v, mask, 3, 10)
    for p in (0, 2, 3, 12, 13, 69):
        lens = np.array([p + 1, p + 1])
        od = A.decode(q[:, p], k, v, lens, mask, 3, 10)
        np.testing.assert_allclose(od, o[:, p], rtol=0, atol=1e-13)


def test_invisible_keys_do_not_matter():
    # perturbing keys/values a row cannot see leaves that row unchanged, bit for bit
    b, t, hq, hkv, d = 1, 60, 2, 2, 8
    q, k, v = _rand((b, t, hq, d), 19), _rand((b, t, hkv, d), 20), _rand((b, t, hkv, d), 21)
    mask = np.array([1, 0], np.uint8)
    n_sink, window, i = 3, 10, 40
    base = A.prefill(q, k, v, mask, n_sink, window, rows=[i])
    k2, v2 = k.copy(), v.copy()
    inv_stream = list(range(n_sink, i - window + 1)) + list(range(i + 1, t))
    k2[0, inv_stream, 0] += 100.0
    v2[0, inv_stream, 0] -= 50.0
    k2[0, i + 1:, 1] += 7.0
    pert = A.prefill(q, k2, v2, mask, n_sink, window, rows=[i])
    assert np.array_equal(base, pert)
    # and perturbing a visible key does change it
    k2[0, n_sink - 1, 0] += 1.0
    assert not np.array_equal(base, A.prefill(q, k2, v2, mask, n_sink, window, rows=[i]))


def test_head_permutation_equivariance():
    # permuting KV heads together with their query groups and the mask permutes the outputs
    b, t, hq, hkv, d = 1, 40, 6, 3, 8
    q, k, v = _rand((b, t, hq, d), 22), _rand((b, t, hkv, d), 23), _rand((b, t, hkv, d), 24)
    mask = np.array([1, 0, 1], np.uint8)
    perm = np.array([2, 0, 1])
    qperm = np.concatenate([np.arange(g * 2, g * 2 + 2) for g in perm])
    o = A.prefill(q, k, v, mask, 2, 5)
    op = A.prefill(q[:, :, qperm], k[:, :, perm], v[:, :, perm], mask[perm], 2, 5)
    np.testing.assert_allclose(op, o[:, :, qperm], rtol=0, atol=1e-14)


def test_planted_mistakes_are_caught(monkeypatch):
    """Plant plausible mistakes in the oracle (on the CPU) and check that the pins
    above reject each one."""
    b, t, hq, hkv, d = 1, 24, 4, 2, 8
    q, k, v = _rand((b, t, hq, d), 25), _rand((b, t, hkv, d), 26), _rand((b, t, hkv, d), 27)
    mask = np.array([1, 0], np.uint8)
    good_mask = A.visible_mask
    good_group = A.group_of

    def agree():
        return np.allclose(A.prefill(q, k, v, mask, 2, 5), A.brute_force(q, k, v, mask, 2, 5), atol=1e-12)

    def hand_sets_ok():
        try:
            test_hand_listed_visible_sets()
            return True
        except AssertionError:
            return False

    def sdpa_ok():
        o = A.prefill(q, k, v, np.zeros(hkv, np.uint8), 2, 5)
        return np.allclose(o, _sdpa_causal(q, k, v), atol=1e-12)

    mutants = {
        "window_off_by_one": lambda qp, n, s, ns, w, chunk=0: good_mask(qp, n, s, ns, w + 1, chunk),
        "sink_off_by_one": lambda qp, n, s, ns, w, chunk=0: good_mask(qp, n, s, ns + 1, w, chunk),
        "no_causal_limit": lambda qp, n, s, ns, w, chunk=0: np.ones((len(qp), n), bool),
    }
    assert agree() and hand_sets_ok() and sdpa_ok()
    for name, fn in mutants.items():
        monkeypatch.setattr(A, "visible_mask", fn)
        assert not (agree() and hand_sets_ok() and sdpa_ok()), name
        monkeypatch.setattr(A, "visible_mask", good_mask)
    monkeypatch.setattr(A, "group_of", lambda h, hq_, hkv_: h % hkv_)
    assert not (agree() and sdpa_ok()), "interleaved GQA grouping"
    monkeypatch.setattr(A, "group_of", good_group)
    assert agree() and sdpa_ok()


def test_chunk_eviction_hand_listed_sets():
    # chunk K = 4, n_sink = 1, window = 2 over 12 positions, written out by hand:
    # chunk 0 (rows 0-3) sees everything causal; chunk 1 (rows 4-7) sees the sink,
    # tokens 2,3 (the 2 before the chunk) and its own chunk; chunk 2 sees 0, 6, 7, own.
    want = {0: {0}, 1: {0, 1}, 2: {0, 1, 2}, 3: {0, 1, 2, 3},
            4: {0, 2, 3, 4}, 5: {0, 2, 3, 4, 5}, 6: {0, 2, 3, 4, 5, 6}, 7: {0, 2, 3, 4, 5, 6, 7},
            8: {0, 6, 7, 8}, 9: {0, 6, 7, 8, 9}, 10: {0, 6, 7, 8, 9, 10}, 11: {0, 6, 7, 8, 9, 10, 11}}
    m = A.visible_mask(np.arange(12), 12, True, 1, 2, chunk=4)
    for i in range(12):
        assert set(np.nonzero(m[i])[0].tolist()) == want[i], i


@pytest.mark.parametrize("n_sink,window", [(0, 1), (3, 5), (8, 40)])
def test_chunk_of_one_is_band_one_wider(n_sink, window):
    # evicting after every token keeps `window` tokens plus the current one
    t = 70
    a = A.visible_mask(np.arange(t), t, True, n_sink, window, chunk=1)
    b = A.visible_mask(np.arange(t), t, True, n_sink, window + 1)
    assert np.array_equal(a, b)


def test_chunk_covering_sequence_equals_dense():
    b, t, hq, hkv, d = 1, 50, 4, 2, 16
    q, k, v = _rand((b, t, hq, d), 30), _rand((b, t, hkv, d), 31), _rand((b, t, hkv, d), 32)
    o = A.prefill(q, k, v, np.ones(hkv, np.uint8), 2, 5, chunk=64)
    np.testing.assert_allclose(o, _sdpa_causal(q, k, v), rtol=0, atol=1e-12)


@pytest.mark.parametrize("chunk", [1, 3, 8, 13])
def test_chunk_eviction_brute_force_agrees(chunk):
    b, t, hq, hkv, d = 1, 26, 4, 2, 8
    q, k, v = _rand((b, t, hq, d), 33), _rand((b, t, hkv, d), 34), _rand((b, t, hkv, d), 35)
    mask = np.array([1, 0], np.uint8)
    o = A.prefill(q, k, v, mask, 2, 4, chunk=chunk)
    ob = A.brute_force(q, k, v, mask, 2, 4, chunk=chunk)
    np.testing.assert_allclose(o, ob, rtol=0, atol=1e-12)


def test_chunk_eviction_sees_superset_of_band():
    # the chunked mask keeps the band's keys plus the rest of the chunk's window
    t, n_sink, window = 200, 4, 16
    for chunk in (1, 5, 16, 37):
        band = A.visible_mask(np.arange(t), t, True, n_sink, window)
        ch = A.visible_mask(np.arange(t), t, True, n_sink, window, chunk=chunk)
        assert np.all(ch >= band)
        assert ch.sum(axis=1).max() <= n_sink + window + chunk
