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


def test_paged_reader_follows_the_token_major_v_layout():
    # the same hand-placed token with V pages [num_pages][n_ret][16][D]
    d, n_pages = 4, 5
    kp = np.zeros((n_pages, 2, 16, d))
    vp = np.zeros((n_pages, 2, 16, d))
    bt = np.array([[3, 0, 4]])
    kp[0, 1, 2, :] = 7.0      # token 18 = page index 1 -> physical 0, row 2, rank 1
    vp[0, 1, 2, :] = np.arange(d) + 1.0
    k, v = M.paged_read_token(kp, vp, bt, 0, 1, 18, v_token_major=True)
    assert (k == 7).all() and v.tolist() == [1.0, 2.0, 3.0, 4.0]
    K, V = M.gather_paged(kp, vp, bt, 0, 1, 19, v_token_major=True)
    assert V[18].tolist() == [1.0, 2.0, 3.0, 4.0] and (V[:18] == 0).all()


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


# ---------------------------------------------------------------- negative pins of the bit-exact checkers
#
# A correct cache image is built here by direct index arithmetic from the
# documented layout (not through the oracle's readers), the checkers must find
# no mismatch in it, and every planted fault must be counted.

def _cache_image(seed=0, B=2, lens=(45, 70), mask=(0, 1, 0, 1), n_sink=3, window=20, d=8, n_pages=16):
    rng = np.random.default_rng(seed)
    T = max(lens)
    hkv = len(mask)
    ks = rng.standard_normal((B, T, hkv, d)).astype(np.float32)
    vs = rng.standard_normal((B, T, hkv, d)).astype(np.float32)
    ret = [g for g in range(hkv) if not mask[g]]
    st = [g for g in range(hkv) if mask[g]]
    max_pages = (T + 15) // 16
    bt = rng.permutation(n_pages)[:B * max_pages].reshape(B, max_pages)
    kp = np.full((n_pages, len(ret), 16, d), np.nan, np.float32)
    vp = np.full((n_pages, len(ret), d, 16), np.nan, np.float32)
    cap = n_sink + window
    nblk = (cap + 15) // 16
    kr = np.full((B, len(st), nblk, 16, d), np.nan, np.float32)
    vr = np.full((B, len(st), nblk, d, 16), np.nan, np.float32)
    for b in range(B):
        for p in range(lens[b]):
            page, row = bt[b, p // 16], p % 16
            for r, g in enumerate(ret):
                kp[page, r, row] = ks[b, p, g]
                vp[page, r, :, row] = vs[b, p, g]
            # ring: sinks keep their slot; later tokens cycle through the window
            slot = p if p < n_sink else n_sink + (p - n_sink) % window
            for s, g in enumerate(st):
                kr[b, s, slot // 16, slot % 16] = ks[b, p, g]
                vr[b, s, slot // 16, :, slot % 16] = vs[b, p, g]
    return dict(ks=ks, vs=vs, kp=kp, vp=vp, kr=kr, vr=vr, bt=bt, lens=np.array(lens), mask=mask,
                n_sink=n_sink, window=window)


def _bad_paged(c):
    return M.check_paged(c["kp"], c["vp"], c["bt"], c["ks"], c["vs"], c["lens"], c["mask"])


def _bad_ring(c):
    return M.check_ring(c["kr"], c["vr"], c["ks"], c["vs"], c["lens"], c["mask"], c["n_sink"], c["window"])


def test_checkers_accept_a_correct_image():
    c = _cache_image()
    assert _bad_paged(c) == 0 and _bad_ring(c) == 0


def test_checker_counts_a_flipped_bit_in_a_k_row():
    c = _cache_image()
    page, row = c["bt"][1, 33 // 16], 33 % 16
    k = c["kp"][page, 1, row].view(np.uint32)
    k[3] ^= 1                                       # lowest mantissa bit of one element
    assert _bad_paged(c) == 1


def test_checker_counts_a_v_column_of_the_wrong_token():
    c = _cache_image()
    page = c["bt"][0, 0]
    c["vp"][page, 0, :, 5] = c["vs"][0, 6, 0]       # token 5's V column holds token 6
    assert _bad_paged(c) == 1


def _token_major(c):
    """The same image with token-major V pages, by index arithmetic."""
    c = dict(c)
    c["vp"] = np.ascontiguousarray(np.swapaxes(c["vp"], 2, 3))
    return c


def test_checker_reads_token_major_v_pages():
    c = _token_major(_cache_image())
    args = (c["kp"], c["vp"], c["bt"], c["ks"], c["vs"], c["lens"], c["mask"])
    assert M.check_paged(*args, v_token_major=True) == 0
    page = c["bt"][1, 50 // 16]
    c["vp"][page, 1, 50 % 16, 2] += 1.0             # one element of token 50's V row
    assert M.check_paged(*args, v_token_major=True) == 1


def test_checker_counts_a_stale_ring_slot_after_wrap():
    c = _cache_image()
    n_sink, window = c["n_sink"], c["window"]
    p = c["lens"][1] - 1                            # newest token of sequence 1, past the wrap
    slot = n_sink + (p - n_sink) % window
    stale = p - window                              # the token that slot held one lap earlier
    g = [h for h in range(4) if c["mask"][h]][1]
    c["kr"][1, 1, slot // 16, slot % 16] = c["ks"][1, stale, g]
    c["vr"][1, 1, slot // 16, :, slot % 16] = c["vs"][1, stale, g]
    assert _bad_ring(c) == 1


def test_checker_counts_swapped_retrieval_ranks():
    c = _cache_image()
    c["kp"][:, [0, 1]] = c["kp"][:, [1, 0]]
    c["vp"][:, [0, 1]] = c["vp"][:, [1, 0]]
    assert _bad_paged(c) == 2 * int(c["lens"].sum())


def test_checker_counts_swapped_streaming_ranks_and_sink_loss():
    c = _cache_image()
    c["kr"][:, [0, 1]] = c["kr"][:, [1, 0]]
    assert _bad_ring(c) == 2 * 2 * (c["n_sink"] + c["window"])
    c = _cache_image()
    c["vr"][0, 0, 0, :, 1] = c["vs"][0, 1 + c["window"], 1]   # sink slot 1 overwritten as if it cycled
    assert _bad_ring(c) == 1


# ---------------------------------------------------------------- decode bytes

def test_decode_kv_bytes_hand_cases():
    # (2 retrieval heads x 5 tokens + 1 ring of min(5, 2+3)) and (2 x 100 + min(100, 5)), d 4, bf16, K and V
    assert C.decode_kv_bytes([5, 100], 2, 1, 4, 2, 2, 3) == (15 + 205) * 4 * 2 * 2
    assert C.decode_kv_bytes([], 3, 1, 128, 2, 64, 1024) == 0
    assert C.decode_kv_bytes([1], 0, 4, 128, 4, 64, 1024) == 4 * 1 * 128 * 2 * 4
    # the batch-8 x 131072 Llama-3-8B-shaped step: 4 + 4 KV heads, ring 64 + 1024
    b = C.decode_kv_bytes([131072] * 8, 4, 4, 128, 2, 64, 1024)
    assert b == 8 * (4 * 131072 + 4 * 1088) * 128 * 2 * 2
    assert math.isclose(b / 1e9, 2.1653, abs_tol=5e-5)


@pytest.mark.parametrize("n_sink,window", [(0, 1), (3, 20), (64, 16)])
def test_decode_kv_bytes_equals_the_cache_image(n_sink, window):
    # bytes read by a step = tokens stored in the paged cache + live ring slots
    # (ring replay, independent of the min() in the formula), K and V
    for lens in ([1], [7, 50], [200, 3, 81]):
        live = sum(int((M.ring_tokens(n, n_sink, window) >= 0).sum()) for n in lens)
        want = (2 * sum(lens) + 3 * live) * 16 * 2 * 2
        assert C.decode_kv_bytes(lens, 2, 3, 16, 2, n_sink, window) == want
        # and one layer of the resident-KV formula per sequence
        assert C.decode_kv_bytes(lens, 2, 3, 16, 2, n_sink, window) == \
            sum(C.kv_cache_bytes(1, 16, 2, 2, 3, n, n_sink, window) for n in lens)


def test_decode_kv_bytes_rejects_planted_mistakes():
    lens, args = [37, 5000], (2, 3, 128, 2, 64, 1024)
    good = C.decode_kv_bytes(lens, *args)
    no_v = sum((2 * n + 3 * min(n, 1088)) * 128 * 2 for n in lens)          # K only
    full_ring = sum((2 * n + 3 * n) * 128 * 2 * 2 for n in lens)            # streaming heads read everything
    window_only = sum((2 * n + 3 * min(n, 1024)) * 128 * 2 * 2 for n in lens)  # sink forgotten
    assert good not in (no_v, full_ring, window_only)


# ---------------------------------------------------------------- the benchmark's own counters

def _bench():
    import importlib.util
    spec = importlib.util.spec_from_file_location("bench", os.path.join(os.path.dirname(GOLDEN), "..", "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_bench_counters_equal_the_oracle_accounting():
    bench = _bench()
    for t in (1, 2, 63, 64, 65, 255, 1000, 4096, 32768, 262144):
        for n_sink, window in ((0, 1), (4, 32), (64, 1024), (64, 2048), (2000, 10), (5, 100000)):
            for st in (False, True):
                assert bench.visible_pairs(t, st, n_sink, window) == C.visible_pairs(t, st, n_sink, window)
            for hr, hs in ((14, 14), (28, 0), (0, 28), (7, 21)):
                assert bench.useful_prefill_flops(t, 128, hr, hs, n_sink, window) == \
                    C.prefill_flops(t, 128, hr, hs, n_sink, window)
    for lens in ([131072] * 8, [1, 17, 1088, 1089], [262144]):
        for gr, gs in ((4, 4), (2, 2), (8, 0), (0, 8)):
            for n_sink, window in ((64, 1024), (64, 2048), (0, 1)):
                assert bench.decode_bytes(lens, gr, gs, 128, 2, n_sink, window) == \
                    C.decode_kv_bytes(lens, gr, gs, 128, 2, n_sink, window)


def _tiles_with_a_visible_pair(t, streaming, n_sink, window, chunk=0, rows=256, bn=64):
    """(query block, key tile) pairs, blocks of `rows` query rows and tiles of
    `bn` keys, in which the oracle's mask has at least one visible pair."""
    m = A.visible_mask(np.arange(t), t, streaming, n_sink, window, chunk)
    count = 0
    for i0 in range(0, t, rows):
        blk = m[i0:i0 + rows]
        for k0 in range(0, t, bn):
            count += bool(blk[:, k0:k0 + bn].any())
    return count


@pytest.mark.parametrize("t", [1, 63, 64, 65, 300, 700, 1000, 2113])
@pytest.mark.parametrize("n_sink,window,chunk", [(0, 1, 0), (4, 32, 0), (64, 128, 0), (70, 200, 0), (130, 5, 0),
                                                (4, 100, 7), (16, 256, 1024), (8, 64, 600)])
def test_bench_computed_tiles_are_the_tiles_holding_visible_pairs(t, n_sink, window, chunk):
    # The computed-tile FLOP count of the benchmark (the work the prefill
    # kernel issues: 256-row query blocks x 64-key tiles) equals 4 D x 256 x 64
    # per (block, tile) pair in which the mask of Sec. 5 has a visible
    # (query, key) pair: the kernel visits exactly those tiles, no others.
    bench = _bench()
    per_tile = 4 * 128 * 256 * 64
    ret = _tiles_with_a_visible_pair(t, False, n_sink, window, chunk)
    st = _tiles_with_a_visible_pair(t, True, n_sink, window, chunk)
    assert bench.computed_tile_flops(t, 128, 1, 0, n_sink, window, chunk=chunk) == per_tile * ret
    assert bench.computed_tile_flops(t, 128, 0, 1, n_sink, window, chunk=chunk) == per_tile * st
    assert bench.computed_tile_flops(t, 128, 3, 5, n_sink, window, chunk=chunk) == per_tile * (3 * ret + 5 * st)



def test_bench_traffic_figure_follows_its_kernel_sources():
    # roofline.traffic is reported only while the kernel sources it was
    # measured on are unchanged: the hash covers code lines, not comments.
    bench = _bench()
    root = os.path.join(os.path.dirname(GOLDEN), "..", "paper_2608_06849_amd", "csrc")

    def reader(edit):
        def read(name):
            with open(os.path.join(root, name)) as f:
                text = f.read()
            return edit(name, text)
        return read

    names = bench.PREFILL_SOURCES
    same = bench.kernel_source_hash(names)
    assert bench.kernel_source_hash(names, reader(lambda n, t: t)) == same
    commented = reader(lambda n, t: t.replace("\n", "\n// a comment line\n", 3) + "\n\n   // trailing\n")
    assert bench.kernel_source_hash(names, commented) == same
    changed = reader(lambda n, t: t + "\nint aoh_extra_symbol;\n" if n == "prefill.hip" else t)
    assert bench.kernel_source_hash(names, changed) != same
    # a figure keyed to another hash is dropped; one keyed to the current hash is kept
    saved = bench.TRAFFIC["prefill_mixed"]
    try:
        bench.TRAFFIC["prefill_mixed"] = dict(saved, source_hash="0" * 16)
        assert bench.traffic_for("prefill_mixed") is None
        bench.TRAFFIC["prefill_mixed"] = dict(saved, source_hash=same)
        want = round((saved["fetch_kib"] / bench.TRAFFIC["fetch_factor"] +
                      saved["write_kib"] / bench.TRAFFIC["write_factor"]) * 1024)
        assert bench.traffic_for("prefill_mixed") == want
    finally:
        bench.TRAFFIC["prefill_mixed"] = saved
    assert bench.traffic_for("no_such_kernel") is None
