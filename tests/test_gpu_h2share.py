"""H2Share on the GPU (through the C interface) against the float64 oracle.

* Head mapping: similarities within 1e-4 (Gram matrices of bf16 weights with
  fp32 accumulation; everything after in fp64), mapping exact (cases are built
  with separated maxima).
* Anchor decode: the attention output is bit-identical to aoh_decode (same
  kernels, the scores are only kept); the selected positions are checked
  against the oracle's group-mean probabilities: equal to the oracle's set
  where its k-th and (k+1)-th scores are further apart than the tolerance,
  else every selected score must reach the oracle's k-th score (and every
  unselected one must not exceed it) within the tolerance.  Format: ascending,
  distinct, < lens, min(lens, k) entries then -1.
* Reuse decode: borrowed lists drawn by a seeded generator, attention output
  against the oracle (bf16 bar); the anchor -> reuse chain end to end against
  the oracle's own chain where the selections coincide.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import h2share as HS
from oracle import attention as OA
from oracle import cache_model as CM
from paper_2608_06849_amd import (PagedCache, RingCache, aoh_decode, aoh_decode_anchor, aoh_decode_reuse,
                                  aoh_decode_workspace_bytes, aoh_head_mapping, aoh_kv_append)
from paper_2608_06849_amd import aoh as A
from tests.helpers import assert_parity, bits, f64

pytestmark = pytest.mark.gpu
DEV = "cuda"
BF = torch.bfloat16
SEL_RTOL = 1e-3   # relative tolerance on selection scores (fp32 scores of bf16 products vs fp64)
SEL_ATOL = 1e-9


def _bf(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(BF)


# ------------------------------------------------------------------------- head mapping

def _check_mapping(wq_a, wk_a, wq_r, wk_r, d, mask_a, mask_r, what):
    t = [_bf(w) for w in (wq_a, wk_a, wq_r, wk_r)]
    hs, gsim, mp = aoh_head_mapping(*[x.to(DEV) for x in t], d, mask_a, mask_r)
    torch.cuda.synchronize()
    w64 = [x.double().numpy() for x in t]
    want_h = HS.head_similarity(*w64, d)
    want_g = HS.group_similarity(want_h, len(mask_a))
    want_m = HS.mapping_to_rank(HS.group_mapping(want_g, mask_a, mask_r), mask_a)
    err = np.abs(hs.cpu().numpy() - want_h).max()
    assert err < 1e-4, f"{what}: head similarity error {err:.2e}"
    assert np.abs(gsim.cpu().numpy() - want_g).max() < 1e-4, what
    assert mp.cpu().numpy().tolist() == want_m.tolist(), what
    print(f"{what}: max similarity error {err:.2e}, mapping {want_m.tolist()}")
    return want_m


def test_mapping_permuted_copies():
    d, gs, hkv, dm = 128, 2, 4, 512
    r = np.random.default_rng(0)
    wq = r.standard_normal((gs * hkv * d, dm)) * 0.05
    wk = r.standard_normal((hkv * d, dm)) * 0.05
    perm = [3, 1, 0, 2]
    wq_r, wk_r = np.empty_like(wq), np.empty_like(wk)
    for g2, g in enumerate(perm):
        wk_r[g2 * d:(g2 + 1) * d] = r.uniform(0.5, 2) * wk[g * d:(g + 1) * d]
        wq_r[g2 * gs * d:(g2 + 1) * gs * d] = r.uniform(0.5, 2) * wq[g * gs * d:(g + 1) * gs * d]
    m = _check_mapping(wq, wk, wq_r, wk_r, d, [0, 0, 0, 0], [0, 0, 0, 0], "permuted copies")
    assert m.tolist() == perm
    # only the anchor's retrieval groups (0 and 3) are candidates: reuse group 0
    # copies anchor group 3 (rank 1), group 2 copies anchor group 0 (rank 0);
    # group 3 copies a streaming anchor group, so its choice is the oracle's
    m = _check_mapping(wq, wk, wq_r, wk_r, d, [0, 1, 1, 0], [0, 1, 0, 0], "permuted copies, mixed labels")
    assert m.tolist()[:3] == [1, -1, 0]


@pytest.mark.parametrize("hq,hkv,d,dm,seed", [(8, 2, 64, 192, 1), (4, 4, 128, 256, 2)])
def test_mapping_random(hq, hkv, d, dm, seed):
    r = np.random.default_rng(seed)
    w = [r.standard_normal((n * d, dm)) for n in (hq, hkv, hq, hkv)]
    _check_mapping(*w, d, [0] * hkv, [0] * hkv, f"random {hq, hkv, d, dm}")


def test_mapping_qwen_shaped_layers():
    # two consecutive layers of the Qwen2.5-7B-shaped classifier workload
    a = synth.projection_weights("qwen25_classify", 4)
    b = synth.projection_weights("qwen25_classify", 5)
    _check_mapping(a[0], a[1], b[0], b[1], 128, [0, 1, 0, 1], [1, 0, 0, 1], "qwen25 layers 4 -> 5")


# ------------------------------------------------------------------------- decode

def _decode_setup(B, L, hq, hkv, d, mask, n_sink, window, seed, k_boost=None, v_token_major=False):
    """Seeded K/V for L positions of B sequences in a paged cache (shuffled pages;
    V pages token-major on request) and a ring, appended from position 0."""
    kk = synth.gaussian((B, L, hkv, d), seed, "h2-k")
    vv = synth.gaussian((B, L, hkv, d), seed, "h2-v")
    if k_boost is not None:
        k_boost(kk)
    k, v = _bf(kk), _bf(vv)
    n_ret, n_str = mask.count(0), mask.count(1)
    max_pages = (L + 15) // 16
    perm = synth.page_permutation(B * max_pages, seed, "h2-pages")
    bt = torch.from_numpy(perm.reshape(B, max_pages).astype(np.int32))
    full = PagedCache.allocate(B * max_pages, n_ret, d, BF, bt, v_token_major=v_token_major) if n_ret else None
    ring = RingCache.allocate(B, n_str, n_sink, window, d, BF) if n_str else None
    return k, v, full, ring


def _fill(k, v, mask, lens, full, ring, n_sink, window):
    # append each sequence's first lens[b] tokens (the ring must end at lens[b])
    for b, n in enumerate(lens):
        f = full.rows(b, b + 1) if full else None
        rg = RingCache(ring.k[b:b + 1], ring.v[b:b + 1], ring.capacity) if ring else None
        aoh_kv_append(k[b:b + 1, :n].to(DEV), v[b:b + 1, :n].to(DEV), mask, torch.zeros(1, dtype=torch.int32, device=DEV),
                      f, rg, n_sink, window)


def _check_selection(got, q, k, lens, mask, top_k, what):
    """got [B, n_ret, top_k] (numpy) against the oracle's scores."""
    k64 = f64(k)
    q64 = f64(q)
    ret = [g for g in range(len(mask)) if not mask[g]]
    exact = 0
    for b in range(len(lens)):
        n = int(lens[b])
        for r, g in enumerate(ret):
            sel = got[b, r]
            m = min(n, top_k)
            assert np.all(sel[m:] == -1), f"{what}: padding"
            s = sel[:m]
            assert np.all(np.diff(s) > 0) and s[0] >= 0 and s[-1] < n, f"{what}: order/range"
            sc = HS.group_scores(q64, k64, lens, b, g, len(mask))
            if n <= top_k:
                continue
            srt = np.sort(sc)[::-1]
            kth, nxt = srt[top_k - 1], srt[top_k]
            tol = SEL_RTOL * kth + SEL_ATOL
            if kth - nxt > 2 * tol:
                assert s.tolist() == HS.top_k_positions(sc, top_k).tolist(), f"{what}: b{b} group {g}"
                exact += 1
            else:
                unsel = np.setdiff1d(np.arange(n), s)
                assert sc[s].min() >= kth - tol and sc[unsel].max() <= kth + tol, f"{what}: b{b} group {g}"
    return exact


@pytest.mark.parametrize("B,L,lens,hq,hkv,d,mask,top_k,seed", [
    (2, 700, [700, 413], 8, 2, 128, [0, 1], 64, 1),
    (1, 300, [300], 8, 4, 128, [0, 0, 1, 0], 300, 2),      # top_k = lens: everything
    (2, 500, [37, 500], 4, 2, 64, [0, 0], 100, 3),          # lens < top_k for one sequence
    (1, 2048, [2048], 28, 4, 128, [0, 1, 0, 1], 256, 4),    # Qwen-shaped heads
])
def test_anchor_decode(B, L, lens, hq, hkv, d, mask, top_k, seed):
    n_sink, window = 4, 64
    k, v, full, ring = _decode_setup(B, L, hq, hkv, d, mask, n_sink, window, seed)
    _fill(k, v, mask, lens, full, ring, n_sink, window)
    q = _bf(synth.gaussian((B, hq, d), seed, "h2-q"))
    lens_t = torch.tensor(lens, dtype=torch.int32, device=DEV)
    out_a, idx = aoh_decode_anchor(q.to(DEV), full, ring, mask, lens_t, n_sink, window, top_k)
    ws = torch.empty(aoh_decode_workspace_bytes(B, hq, d, full.block_table.shape[1], n_sink + window) // 4 + 4,
                     dtype=torch.float32, device=DEV)
    out_d = aoh_decode(q.to(DEV), full, ring, mask, lens_t, n_sink, window, workspace=ws)
    torch.cuda.synchronize()
    assert np.array_equal(bits(out_a), bits(out_d)), "anchor output differs from aoh_decode"
    n_exact = _check_selection(idx.cpu().numpy(), q, k, lens, mask, top_k, f"anchor {B, L, hq, hkv, d, top_k}")
    print(f"anchor {B, L, hq, hkv, d, top_k}: selections exact for {n_exact} separable lists")


def test_anchor_many_sequences_fixed_splits():
    # more sequences than the work-space split takes: the anchor runs on fixed
    # splits per (sequence, KV head); outputs equal aoh_decode bit for bit and
    # every list is a valid top-k of the oracle's scores
    B, L, hq, hkv, d, mask, top_k, seed = 70, 400, 8, 2, 128, [0, 1], 64, 14
    n_sink, window = 4, 64
    lens = [int(x) for x in synth.rng(seed, "h2-many-lens").integers(30, L + 1, size=B)]
    k, v, full, ring = _decode_setup(B, L, hq, hkv, d, mask, n_sink, window, seed)
    _fill(k, v, mask, lens, full, ring, n_sink, window)
    q = _bf(synth.gaussian((B, hq, d), seed, "h2-q"))
    lens_t = torch.tensor(lens, dtype=torch.int32, device=DEV)
    out_a, idx = aoh_decode_anchor(q.to(DEV), full, ring, mask, lens_t, n_sink, window, top_k)
    ws = torch.empty(aoh_decode_workspace_bytes(B, hq, d, full.block_table.shape[1], n_sink + window) // 4 + 4,
                     dtype=torch.float32, device=DEV)
    out_d = aoh_decode(q.to(DEV), full, ring, mask, lens_t, n_sink, window, workspace=ws)
    torch.cuda.synchronize()
    assert np.array_equal(bits(out_a), bits(out_d)), "anchor output differs from aoh_decode"
    n_exact = _check_selection(idx.cpu().numpy(), q, k, lens, mask, top_k, f"anchor B={B}")
    print(f"anchor B={B}: selections exact for {n_exact} separable lists")


def test_anchor_exact_ties_go_to_lower_positions():
    # K rows at positions 40, 90, 140, 190, 240 are identical and dominant: five
    # exactly tied scores for a top-3 selection -> positions 40, 90, 140
    B, L, hq, hkv, d = 1, 256, 4, 1, 128
    def boost(kk):
        row = kk[0, 7, 0] * 6.0
        for p in (40, 90, 140, 190, 240):
            kk[0, p, 0] = row
    k, v, full, ring = _decode_setup(B, L, hq, hkv, d, [0], 4, 16, 5, k_boost=boost)
    _fill(k, v, [0], [L], full, None, 4, 16)
    # queries aligned with the planted row so that it dominates
    q = _bf(np.repeat(k[0, 40, 0].float().numpy()[None, None], hq, axis=1) * 0.5)
    _, idx = aoh_decode_anchor(q.to(DEV), full, None, [0], torch.tensor([L], dtype=torch.int32, device=DEV), 4, 16, 3)
    torch.cuda.synchronize()
    assert idx.cpu().numpy()[0, 0].tolist() == [40, 90, 140]


@pytest.mark.parametrize("scale,top_k", [
    (1.0, 200),    # planted keys ~16-24 log2 units above the rest: the k-th score lies inside the code span
    (5.0, 48),     # ~80-120 units above: the selection reaches scores far below the span (saturated codes)
])
def test_anchor_wide_score_range(scale, top_k):
    # 24 planted K rows (a common direction times distinct factors) dominate
    # the seeded ones by tens of log2 units, spread over many 32-token chunks,
    # so a chunk holding one keeps the other positions' scores as large
    # offsets below it (saturated in the second case); the selection is
    # checked against the float64 oracle's group probabilities
    B, L, hq, hkv, d, mask = 1, 3000, 8, 2, 128, [0, 0]
    planted = synth.rng(11, "h2-wide").choice(L, 24, replace=False)

    kk0 = synth.gaussian((B, L, hkv, d), 11, "h2-k")[0, 5]   # the planted direction, before boosting

    def boost(kk):
        u = kk[0, 5, :].copy()
        for i, p in enumerate(planted):
            kk[0, p, :] = u * scale * (1.0 + 0.02 * i)
    k, v, full, ring = _decode_setup(B, L, hq, hkv, d, mask, 4, 16, 11, k_boost=boost)
    _fill(k, v, mask, [L], full, None, 4, 16)
    # query heads of group g aligned with the planted direction of KV head g
    qq = np.stack([kk0[h // (hq // hkv)] for h in range(hq)])[None]
    qq = qq + 0.2 * synth.gaussian((B, hq, d), 11, "h2-wide-q")
    q = _bf(qq)
    lens_t = torch.tensor([L], dtype=torch.int32, device=DEV)
    _, idx = aoh_decode_anchor(q.to(DEV), full, None, mask, lens_t, 4, 16, top_k)
    torch.cuda.synchronize()
    got = idx.cpu().numpy()
    n_exact = _check_selection(got, q, k, [L], mask, top_k, f"wide scores x{scale}")
    # every planted position holding more than the absolute tolerance of its
    # group's probability is selected (saturated codes only reorder positions
    # below ~2^-32 of their chunk's maximum, far under that tolerance)
    q64, k64 = f64(q), f64(k)
    for r in range(hkv):
        sc = HS.group_scores(q64, k64, [L], 0, r, hkv)
        big = [p for p in planted.tolist() if sc[p] > 10 * SEL_ATOL]
        assert big and set(big) <= set(got[0, r].tolist()), f"group {r}: a planted position was not selected"
    print(f"wide scores x{scale}, top {top_k}: selections exact for {n_exact} lists")


def _lists(B, n_lists, lens, top_k, seed):
    """Seeded borrowed lists: per (b, list) min(lens, top_k) distinct sorted positions, then -1."""
    out = np.full((B, n_lists, top_k), -1, dtype=np.int32)
    for b in range(B):
        for r in range(n_lists):
            n = int(lens[b])
            m = min(n, top_k)
            pick = synth.rng(seed, "h2-lists", b, r).choice(n, m, replace=False)
            out[b, r, :m] = np.sort(pick)
    return out


@pytest.mark.parametrize("B,L,lens,hq,hkv,d,mask,mapping,n_lists,top_k,seed", [
    (2, 900, [900, 611], 8, 2, 128, [0, 1], [1, -1], 2, 128, 6),
    (1, 400, [400], 8, 4, 128, [0, 0, 1, 0], [2, 0, -1, 2], 3, 77, 7),   # ragged list length
    (2, 300, [300, 20], 4, 2, 64, [0, 0], [0, 0], 1, 64, 8),             # lens < top_k
    (1, 3000, [3000], 28, 4, 128, [0, 1, 0, 1], [1, -1, 0, -1], 2, 1024, 9),
])
@pytest.mark.parametrize("vtm", [False, True], ids=["v_dim_major", "v_token_major"])
def test_reuse_decode(B, L, lens, hq, hkv, d, mask, mapping, n_lists, top_k, seed, vtm):
    n_sink, window = 8, 96
    k, v, full, ring = _decode_setup(B, L, hq, hkv, d, mask, n_sink, window, seed, v_token_major=vtm)
    _fill(k, v, mask, lens, full, ring, n_sink, window)
    q = _bf(synth.gaussian((B, hq, d), seed, "h2-q"))
    sel = _lists(B, n_lists, lens, top_k, seed)
    lens_t = torch.tensor(lens, dtype=torch.int32, device=DEV)
    out = aoh_decode_reuse(q.to(DEV), full, ring, mask, lens_t, n_sink, window,
                           torch.from_numpy(sel).to(DEV), mapping)
    torch.cuda.synchronize()
    want = HS.reuse_decode(f64(q), f64(k), f64(v), lens, mask, n_sink, window, sel, mapping)
    mx, mean = assert_parity(out, want, BF, f"reuse {B, L, hq, hkv, d, top_k}")
    print(f"reuse {B, L, hq, hkv, d, top_k}: max abs {mx:.2e} mean {mean:.2e}")


def test_reuse_token_major_v_equals_dimension_major():
    # the same tokens appended to a cache of each V layout (ragged prompt
    # chunks starting mid-page, then single-token steps): both caches hold every
    # token bit for bit in their own layout, and the reuse step reads them to
    # bit-identical outputs (same products in the same order)
    B, L, hq, hkv, d, mask = 2, 1000, 8, 2, 128, [0, 1]
    n_sink, window, seed = 4, 64, 12
    lens = [1000, 613]
    caches = [_decode_setup(B, L, hq, hkv, d, mask, n_sink, window, seed, v_token_major=t) for t in (False, True)]
    k, v = caches[0][0], caches[0][1]
    outs = []
    for _, _, full, ring in caches:
        full.k.fill_(float("nan"))
        full.v.fill_(float("nan"))
        for b, n in enumerate(lens):
            f = full.rows(b, b + 1)
            rg = RingCache(ring.k[b:b + 1], ring.v[b:b + 1], ring.capacity)
            cut = [0, 37, n - 3, n - 2, n - 1, n]            # 37 tokens, then up to the last 3, then 1 at a time
            for lo, hi in zip(cut, cut[1:]):
                start = torch.full((1,), lo, dtype=torch.int32, device=DEV)
                aoh_kv_append(k[b:b + 1, lo:hi].to(DEV), v[b:b + 1, lo:hi].to(DEV), mask, start, f, rg, n_sink, window)
        torch.cuda.synchronize()
        bad = CM.check_paged(bits(full.k), bits(full.v), full.block_table.cpu().numpy(), bits(k), bits(v), lens, mask,
                             v_token_major=full.v_token_major)
        assert bad == 0, f"{bad} tokens wrong in the cache (v_token_major={full.v_token_major})"
        q = _bf(synth.gaussian((B, hq, d), seed, "h2-q"))
        sel = _lists(B, 1, lens, 300, seed)
        out = aoh_decode_reuse(q.to(DEV), full, ring, mask, torch.tensor(lens, dtype=torch.int32, device=DEV), n_sink,
                               window, torch.from_numpy(sel).to(DEV), [0, -1])
        torch.cuda.synchronize()
        outs.append(out)
    assert np.array_equal(bits(outs[0]), bits(outs[1])), "reuse output depends on the V page layout"


def test_reuse_every_position_matches_oracle_full_decode():
    B, L, hq, hkv, d = 2, 640, 8, 2, 128
    mask = [0, 0]
    lens = [640, 333]
    k, v, full, _ = _decode_setup(B, L, hq, hkv, d, mask, 4, 32, 10)
    _fill(k, v, mask, lens, full, None, 4, 32)
    q = _bf(synth.gaussian((B, hq, d), 10, "h2-q"))
    sel = np.full((B, 1, L), -1, dtype=np.int32)
    for b in range(B):
        sel[b, 0, :lens[b]] = np.arange(lens[b])
    out = aoh_decode_reuse(q.to(DEV), full, None, mask, torch.tensor(lens, dtype=torch.int32, device=DEV), 4, 32,
                           torch.from_numpy(sel).to(DEV), [0, 0])
    torch.cuda.synchronize()
    assert_parity(out, OA.decode(f64(q), f64(k), f64(v), lens, mask, 4, 32), BF, "reuse over every position")


def test_anchor_then_reuse_chain():
    # Two layers of one block on the same sequences: the anchor's planted needles
    # (48 per sequence and retrieval group) make its top-48 set clear-cut; the
    # reuse layer (own K/V) borrows it through the mapping.
    B, L, hq, hkv, d, top_k = 2, 4096, 8, 2, 128, 48
    mask = [0, 0]
    lens = [4096, 2500]
    qa = synth.gaussian((B, hq, d), 11, "h2-qa")

    def needles(kk):
        for b in range(B):
            for g in range(hkv):
                pos = synth.rng(11, "h2-needles", b, g).choice(lens[b], top_k, replace=False)
                direction = qa[b, g * (hq // hkv)] / np.linalg.norm(qa[b, g * (hq // hkv)])
                kk[b, pos, g] = 3.0 * direction * np.sqrt(d)

    ka, va, fa, _ = _decode_setup(B, L, hq, hkv, d, mask, 4, 32, 11, k_boost=needles)
    kr, vr, fr, _ = _decode_setup(B, L, hq, hkv, d, mask, 4, 32, 12)
    _fill(ka, va, mask, lens, fa, None, 4, 32)
    _fill(kr, vr, mask, lens, fr, None, 4, 32)
    qr = _bf(synth.gaussian((B, hq, d), 12, "h2-qr"))
    q_a = _bf(qa)
    lens_t = torch.tensor(lens, dtype=torch.int32, device=DEV)
    _, idx = aoh_decode_anchor(q_a.to(DEV), fa, None, mask, lens_t, 4, 32, top_k)
    mapping = [1, 0]
    out = aoh_decode_reuse(qr.to(DEV), fr, None, mask, lens_t, 4, 32, idx, mapping)
    torch.cuda.synchronize()
    want_idx = HS.anchor_select(f64(q_a), f64(ka), lens, mask, top_k)
    assert np.array_equal(idx.cpu().numpy(), want_idx), "anchor selection differs from the oracle's"
    want = HS.reuse_decode(f64(qr), f64(kr), f64(vr), lens, mask, 4, 32, want_idx, mapping)
    assert_parity(out, want, BF, "anchor -> reuse chain")


# ------------------------------------------------------------------------- top-k over several segments
#
# The selection cuts each list into 8 segments of whole 4096-position tiles and
# combines per-segment histograms, counts and compaction offsets.  A list of
# 131072 positions has 8 full segments of 16384; one of 40000 has segments of
# 8192 with a ragged fifth and three empty ones.

def _plant_threshold_ties(kk, qa, lens, n_super, tie_at, n_tie, gs, seed):
    """Group 0 of every sequence: n_super planted keys of distinct strength,
    above n_tie identical keys centred on position tie_at[b] (a segment
    boundary); everything else stays N(0, 1).  With top_k = n_super + n_tie / 2
    the selection threshold falls inside the tied run."""
    d = kk.shape[-1]
    for b, n in enumerate(lens):
        u = qa[b, :gs].sum(0)
        u /= np.linalg.norm(u)
        ties = np.arange(tie_at[b] - n_tie // 2, tie_at[b] + n_tie // 2)
        free = np.setdiff1d(np.arange(n), ties)
        sup = synth.rng(seed, "h2-super", b).choice(free, n_super, replace=False)
        kk[b, sup, 0] = (4.0 + np.arange(n_super)[:, None] / n_super) * np.sqrt(d) * u
        kk[b, ties, 0] = 3.0 * np.sqrt(d) * u
    return kk


@pytest.mark.parametrize("planted", [False, True])
def test_anchor_topk_several_segments(planted):
    B, L, hq, hkv, d, top_k = 2, 131072, 8, 2, 128, 2048
    lens = [131072, 40000]
    mask, n_sink, window, seed = [0, 1], 64, 1024, 21
    gs = hq // hkv
    qa = synth.gaussian((B, hq, d), seed, "h2-q")
    tie_at = [16384, 32768]
    n_super, n_tie = top_k - 8, 16
    boost = (lambda kk: _plant_threshold_ties(kk, qa, lens, n_super, tie_at, n_tie, gs, seed)) if planted else None
    k, v, full, ring = _decode_setup(B, L, hq, hkv, d, mask, n_sink, window, seed, k_boost=boost)
    _fill(k, v, mask, lens, full, ring, n_sink, window)
    q = _bf(qa)
    lens_t = torch.tensor(lens, dtype=torch.int32, device=DEV)
    out_a, idx = aoh_decode_anchor(q.to(DEV), full, ring, mask, lens_t, n_sink, window, top_k)
    ws = torch.empty(aoh_decode_workspace_bytes(B, hq, d, full.block_table.shape[1], n_sink + window) // 4 + 4,
                     dtype=torch.float32, device=DEV)
    out_d = aoh_decode(q.to(DEV), full, ring, mask, lens_t, n_sink, window, workspace=ws)
    torch.cuda.synchronize()
    assert np.array_equal(bits(out_a), bits(out_d)), "anchor output differs from aoh_decode"
    got = idx.cpu().numpy()
    n_exact = _check_selection(got, q, k, lens, mask, top_k, f"anchor multi-segment planted={planted}")
    if planted:
        for b in range(B):
            sel = set(got[b, 0].tolist())
            ties = list(range(tie_at[b] - n_tie // 2, tie_at[b] + n_tie // 2))
            # exactly the 8 lowest tied positions (all before the boundary) are taken
            assert [p for p in ties if p in sel] == ties[:n_tie // 2], f"b{b}: tie order across the segment boundary"
            # every planted key above the tie level is taken
            assert len(sel) == top_k and len(sel - set(ties)) == n_super
    print(f"anchor multi-segment planted={planted}: {n_exact} lists exact")


def test_anchor_odd_page_count_full_last_page():
    # 19 pages per sequence (odd) with the length in the last page: the last
    # split of a row covers one block, and its second block's score slots lie
    # past the row.  Strong keys at positions 0..15 of every group make any
    # overwrite of a neighbouring row's first positions change the selection.
    B, L, hq, hkv, d, top_k = 2, 293, 8, 2, 128, 24
    lens = [293, 290]
    mask, n_sink, window, seed = [0, 0], 4, 32, 22
    qa = synth.gaussian((B, hq, d), seed, "h2-q")

    def early(kk):
        for b in range(B):
            for g in range(hkv):
                u = qa[b, g * 4:(g + 1) * 4].sum(0)
                u /= np.linalg.norm(u)
                kk[b, :16, g] = (2.0 + np.arange(16)[:, None] / 16.0) * np.sqrt(d) * u

    k, v, full, ring = _decode_setup(B, L, hq, hkv, d, mask, n_sink, window, seed, k_boost=early)
    assert full.block_table.shape[1] == 19
    _fill(k, v, mask, lens, full, ring, n_sink, window)
    q = _bf(qa)
    _, idx = aoh_decode_anchor(q.to(DEV), full, ring, mask, torch.tensor(lens, dtype=torch.int32, device=DEV),
                               n_sink, window, top_k)
    torch.cuda.synchronize()
    got = idx.cpu().numpy()
    _check_selection(got, q, k, lens, mask, top_k, "anchor odd page count")
    want = HS.anchor_select(f64(q), f64(k), lens, mask, top_k)
    assert np.array_equal(got, want), "selection differs from the oracle's"
    for b in range(B):
        for r in range(2):
            assert set(range(16)) <= set(got[b, r].tolist())


def test_anchor_and_reuse_replay_from_a_graph():
    # the anchor step (split keeping score codes, merge, three top-k launches)
    # and the reuse step on token-major V pages, captured as one HIP graph:
    # every replay, with eager calls and synchronisations between replays,
    # leaves the eager outputs bit for bit
    B, L, hq, hkv, d, mask = 2, 2500, 8, 2, 128, [0, 1]
    n_sink, window, seed, top_k = 4, 64, 13, 200
    lens = [2500, 1777]
    k, v, full, ring = _decode_setup(B, L, hq, hkv, d, mask, n_sink, window, seed)
    _fill(k, v, mask, lens, full, ring, n_sink, window)
    _, _, full_tm, ring_tm = _decode_setup(B, L, hq, hkv, d, mask, n_sink, window, seed, v_token_major=True)
    _fill(k, v, mask, lens, full_tm, ring_tm, n_sink, window)
    q = _bf(synth.gaussian((B, hq, d), seed, "h2-q")).to(DEV)
    lens_t = torch.tensor(lens, dtype=torch.int32, device=DEV)
    idx = torch.empty((B, 1, top_k), dtype=torch.int32, device=DEV)
    out_a, out_r = torch.empty_like(q), torch.empty_like(q)
    ws_a = torch.empty(A.aoh_decode_anchor_workspace_bytes(B, hq, d, full.block_table.shape[1], n_sink + window),
                       dtype=torch.uint8, device=DEV)
    ws_r = torch.empty(A.aoh_decode_reuse_workspace_bytes(B, hq, d, top_k, n_sink + window), dtype=torch.uint8,
                       device=DEV)

    def step():
        aoh_decode_anchor(q, full, ring, mask, lens_t, n_sink, window, top_k, indices=idx, out=out_a, workspace=ws_a)
        aoh_decode_reuse(q, full_tm, ring_tm, mask, lens_t, n_sink, window, idx, [0, -1], out=out_r, workspace=ws_r)

    step()
    torch.cuda.synchronize()
    want = [bits(out_a), idx.cpu().numpy().copy(), bits(out_r)]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(3):
        out_a.zero_(); out_r.zero_(); idx.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = [bits(out_a), idx.cpu().numpy(), bits(out_r)]
        for w, x, name in zip(want, got, ("anchor output", "indices", "reuse output")):
            assert np.array_equal(w, x), f"replay {rep}: {name} differs from the eager call"
        step()                                  # eager work between the replays
        torch.cuda.synchronize()
