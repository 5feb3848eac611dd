"""Pins for oracle.cache_model and oracle.accounting."""
import csv
import math
import os

import numpy as np
import pytest

from oracle import accounting as C
from oracle import attention as A
from oracle import cache_model as M

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return list(csv.DictReader(line for line in f if not line.startswith("#")))


def test_ring_slots_hand_listed():
    # n_sink = 2, window = 3: positions 0..9
    assert [M.ring_slot(p, 2, 3) for p in range(10)] == [0, 1, 2, 3, 4, 2, 3, 4, 2, 3]
    assert M.ring_tokens(10, 2, 3).tolist() == [0, 1, 8, 9, 7]
    assert M.ring_tokens(3, 2, 3).tolist() == [0, 1, 2, -1, -1]


@pytest.mark.parametrize("n_sink,window", [(0, 1), (2, 3), (4, 32), (64, 16), (5, 1)])
def test_ring_holds_exactly_what_the_last_query_sees(n_sink, window):
    # the ring of n_sink + window slots, after L appends, holds exactly the keys
    # visible to a streaming query at position L-1 (the cache-size reading)
    for length in range(1, 3 * (n_sink + window) + 5):
        held = M.ring_tokens(length, n_sink, window)
        held = set(held[held >= 0].tolist())
        vis = A.visible_mask([length - 1], length, True, n_sink, window)[0]
        assert held == set(np.nonzero(vis)[0].tolist()), length


def test_paged_and_ring_readers_follow_layout():
    # hand-placed tokens: write by explicit index arithmetic, read back through the readers
    d, n_pages = 4, 5
    kp = np.zeros((n_pages, 2, 16, d))
    vp = np.zeros((n_pages, 2, d, 16))
    bt = np.array([[3, 0, 4]])
    kp[0, 1, 2, :] = 7.0      # token 18 = page index 1 -> physical 0, row 2, rank 1
    vp[0, 1, :, 2] = 9.0
    k, v = M.paged_read_token(kp, vp, bt, 0, 1, 18)
    assert (k == 7).all() and (v == 9).all()
    kr = np.zeros((1, 1, 2, 16, d))
    vr = np.zeros((1, 1, 2, d, 16))
    kr[0, 0, 1, 1, :] = 5.0   # slot 17 -> block 1, row 1
    vr[0, 0, 1, :, 1] = 6.0
    k, v = M.ring_read_slot(kr, vr, 0, 0, 17)
    assert (k == 5).all() and (v == 6).all()
    assert M.ring_capacity_padded(64, 1024) == 1088 and M.ring_capacity_padded(4, 32) == 48


@pytest.mark.parametrize("t", [1, 2, 5, 31, 32, 33, 36, 37, 100, 256])
@pytest.mark.parametrize("n_sink,window", [(4, 32), (0, 1), (3, 3), (40, 2)])
def test_visible_pairs_closed_form_matches_mask_count(t, n_sink, window):
    for st in (False, True):
        m = A.visible_mask(np.arange(t), t, st, n_sink, window)
        assert C.visible_pairs(t, st, n_sink, window) == int(m.sum())
        assert [C.visible_pairs_row(i, st, n_sink, window) for i in range(t)] == m.sum(axis=1).tolist()


def test_tiny_workload_pair_counts():
    assert C.visible_pairs(256, False, 4, 32) == 32896
    assert C.visible_pairs(256, True, 4, 32) == 8586


def test_retrieval_group_count():
    assert C.n_retrieval_groups(4, 0.5) == 2
    assert C.n_retrieval_groups(8, 0.25) == 6
    assert C.n_retrieval_groups(8, 0.75) == 2
    assert C.n_retrieval_groups(4, 0.25) == 3
    assert C.n_retrieval_groups(4, 0.75) == 1
    assert C.n_retrieval_groups(7, 0.5) == 4


def test_kv_bytes_reproduce_efficiency_tables():
    rows = _rows("kv_memory_efficiency_tables.csv")
    assert len(rows) == 63
    for r in rows:
        L, G, d, T = int(r["n_layers"]), int(r["n_kv_heads"]), int(r["d_head"]), int(r["ctx_tokens"])
        g_ret = C.n_retrieval_groups(G, int(r["sparsity_pct"]) / 100.0)
        full = C.kv_cache_bytes(L, d, 2, G, 0, T, 128, 256) / 1e9
        aoh = C.kv_cache_bytes(L, d, 2, g_ret, G - g_ret, T, 128, 256) / 1e9
        tol = float(r["tol_gb"]) + 1e-9
        assert abs(full - float(r["full_gb"])) <= tol, r
        assert abs(aoh - float(r["aoh_gb"])) <= tol, r


def test_kv_bytes_reproduce_longbench_table():
    for r in _rows("kv_memory_longbench_32k.csv"):
        L, G, d, T = int(r["n_layers"]), int(r["n_kv_heads"]), int(r["d_head"]), int(r["ctx_tokens"])
        full = C.kv_cache_bytes(L, d, 2, G, 0, T, 128, 256) / 2**30
        aoh = C.kv_cache_bytes(L, d, 2, G // 2, G - G // 2, T, 128, 256) / 2**30
        assert abs(full - float(r["full_gib"])) <= float(r["full_tol"]) / 2 + 1e-9
        assert abs(aoh - float(r["aoh_gib"])) <= float(r["aoh_tol"]) / 2 + 1e-9
        # the 512-token reading of the surrounding text does not reproduce the table
        aoh512 = C.kv_cache_bytes(L, d, 2, G // 2, G - G // 2, T, 256, 256) / 2**30
        assert abs(aoh512 - float(r["aoh_gib"])) > float(r["aoh_tol"])


def test_prefill_flops_qwen_shape():
    # 28 query heads over 4 KV heads, KV heads 1 and 3 streaming: 14 + 14 query heads
    f = C.prefill_flops(32768, 128, 14, 14, 64, 1024)
    assert f == 4 * 128 * (14 * (32768 * 32769 // 2) + 14 * C.visible_pairs(32768, True, 64, 1024))
    assert math.isclose(f / 1e12, 4.100, abs_tol=5e-4)


def test_vectorised_readers_match_per_token_readers():
    rng = np.random.default_rng(0)
    d, n_pages, B = 8, 12, 2
    kp = rng.standard_normal((n_pages, 2, 16, d))
    vp = rng.standard_normal((n_pages, 2, d, 16))
    bt = rng.permutation(n_pages)[:10].reshape(B, 5)
    for b in range(B):
        for r in range(2):
            K, V = M.gather_paged(kp, vp, bt, b, r, 77)
            for p in range(77):
                kr, vr = M.paged_read_token(kp, vp, bt, b, r, p)
                assert np.array_equal(K[p], kr) and np.array_equal(V[p], vr)
    kr_ = rng.standard_normal((B, 1, 3, 16, d))
    vr_ = rng.standard_normal((B, 1, 3, d, 16))
    pos, K, V = M.gather_ring(kr_, vr_, 1, 0, 100, 5, 37)
    assert sorted(pos.tolist()) == sorted(set(range(5)) | set(range(63, 100)))
    for i, p in enumerate(pos):
        slot = M.ring_slot(int(p), 5, 37)
        kk, vv = M.ring_read_slot(kr_, vr_, 1, 0, slot)
        assert np.array_equal(K[i], kk) and np.array_equal(V[i], vv)
