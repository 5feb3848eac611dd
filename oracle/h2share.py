"""Oracle of H2Share, the AoH-guided cross-layer sparse attention (paper
Sec. "AoH-Guided Sparse Attention: H2Share", its Inference Phase, the GQA
appendix's group-level head mapping, and the trace-reduction appendix).
CPU, numpy float64.

TEST INFRASTRUCTURE: only tests/, the smoke check and the CPU baseline of the
benchmark use this module.

What is computed
  * Head similarity between an anchor layer l and a reuse layer l': the
    normalised Frobenius inner product of the kernel attention matrices,
        M_{h,h'} = <M_h, M_h'>_F / (|M_h|_F |M_h'|_F),  M_h = W_K^T W_Q,
    evaluated in d_head space by the trace identities
        <M_h, M_h'>_F = tr(W_Q^h W_Q'^h'^T . W_K'^g' W_K^g^T),
        |M_h|_F^2     = tr(W_Q^h W_Q^h^T . W_K^g W_K^g^T)
    (Eq. sim; trace-reduction proposition and corollary).
  * Group-level mapping (GQA appendix): the similarity of a KV-group pair is
    the mean of its query-head pairs; every reuse retrieval group takes the
    anchor retrieval group of highest similarity.
  * Anchor layer, per decode step: full attention for retrieval heads, and the
    top-k token positions "according to their attention scores" per retrieval
    group.
  * Reuse layer, per decode step: each retrieval head attends only to its own
    layer's K/V at the positions borrowed from its mapped anchor group;
    streaming heads attend to sink + window as in any layer.

Readings where the paper leaves room:
  * a group's selection score for position j is the mean, over the group's
    query heads, of their attention probabilities p_hj for this step;
  * top-k ties go to the lower position; fewer than k positions (lens < k)
    select them all; the index list is in ascending position order, padded
    with -1;
  * mapping ties go to the lower anchor group index;
  * the reuse layer attends exactly to the borrowed positions (its own
    current token only if borrowed);
  * selection happens on every decode step from that step's anchor attention.

Pins (tests/test_oracle_h2share.py): the trace form equals the Frobenius
inner product of explicitly formed M_h on small weights; a head's similarity
with itself is 1, every value lies in [-1, 1], and the matrix for (l', l) is
the transpose of the one for (l, l'); a reuse layer built from permuted and
rescaled copies of the anchor's groups is mapped back by the permutation; the
top-k equals a brute-force ranking with hand-listed ties; a reuse step whose
borrowed set is every position equals full decode, and one whose borrowed set
is the sink + window positions equals the streaming decode.
"""
import numpy as np

from .attention import attend_rows, group_of


def _slice(w, h, d_head):
    return np.asarray(w[h * d_head:(h + 1) * d_head], dtype=np.float64)


def head_similarity(wq_a, wk_a, wq_r, wk_r, d_head):
    """M^{(l -> l')} [Hq, Hq]: rows anchor query heads h, columns reuse query
    heads h' (Eq. sim, by the trace identities).  wq_* [Hq * d_head, d_model],
    wk_* [Hkv * d_head, d_model]."""
    hq = np.asarray(wq_a).shape[0] // d_head
    hkv = np.asarray(wk_a).shape[0] // d_head
    num = np.empty((hq, hq))
    norm_a = np.empty(hq)
    norm_r = np.empty(hq)
    for h in range(hq):
        g = group_of(h, hq, hkv)
        qa, ka = _slice(wq_a, h, d_head), _slice(wk_a, g, d_head)
        qr, kr = _slice(wq_r, h, d_head), _slice(wk_r, g, d_head)
        norm_a[h] = np.sqrt(np.trace((qa @ qa.T) @ (ka @ ka.T)))
        norm_r[h] = np.sqrt(np.trace((qr @ qr.T) @ (kr @ kr.T)))
    for h in range(hq):
        qa, ka = _slice(wq_a, h, d_head), _slice(wk_a, group_of(h, hq, hkv), d_head)
        for h2 in range(hq):
            qr, kr = _slice(wq_r, h2, d_head), _slice(wk_r, group_of(h2, hq, hkv), d_head)
            num[h, h2] = np.trace((qa @ qr.T) @ (kr @ ka.T))
    return num / np.outer(norm_a, norm_r)


def frobenius_similarity_dense(wq_a, wk_a, wq_r, wk_r, d_head):
    """The same matrix from explicitly formed d_model x d_model M_h (small
    inputs only; the definition the trace identities are checked against)."""
    hq = np.asarray(wq_a).shape[0] // d_head
    hkv = np.asarray(wk_a).shape[0] // d_head
    ma = [_slice(wk_a, group_of(h, hq, hkv), d_head).T @ _slice(wq_a, h, d_head) for h in range(hq)]
    mr = [_slice(wk_r, group_of(h, hq, hkv), d_head).T @ _slice(wq_r, h, d_head) for h in range(hq)]
    out = np.empty((hq, hq))
    for h in range(hq):
        for h2 in range(hq):
            out[h, h2] = np.sum(ma[h] * mr[h2]) / (np.linalg.norm(ma[h]) * np.linalg.norm(mr[h2]))
    return out


def group_similarity(head_sim, n_kv):
    """[Hkv, Hkv]: mean of the query-head similarities of each group pair."""
    hq = head_sim.shape[0]
    gs = hq // n_kv
    return head_sim.reshape(n_kv, gs, n_kv, gs).mean(axis=(1, 3))


def group_mapping(group_sim, anchor_is_streaming, reuse_is_streaming):
    """Anchor retrieval group of highest similarity for every reuse retrieval
    group (-1 for reuse streaming groups); ties to the lower anchor index."""
    anchors = [g for g in range(len(anchor_is_streaming)) if not anchor_is_streaming[g]]
    if not anchors:
        raise ValueError("the anchor layer has no retrieval group")
    out = np.full(len(reuse_is_streaming), -1, dtype=np.int64)
    for g2 in range(len(reuse_is_streaming)):
        if reuse_is_streaming[g2]:
            continue
        best = anchors[0]
        for g in anchors[1:]:
            if group_sim[g, g2] > group_sim[best, g2]:
                best = g
        out[g2] = best
    return out


def step_probabilities(q, k_seq, lens, b, h, n_kv):
    """Full-attention probabilities [lens_b] of query head h of sequence b
    over positions 0..lens_b - 1 (retrieval head of the anchor layer)."""
    hq = q.shape[1]
    g = group_of(h, hq, n_kv)
    n = int(lens[b])
    kk = np.asarray(k_seq[b, :n, g, :], dtype=np.float64)
    s = kk @ np.asarray(q[b, h], dtype=np.float64) / np.sqrt(kk.shape[1])
    p = np.exp(s - s.max())
    return p / p.sum()


def group_scores(q, k_seq, lens, b, g, n_kv):
    """Mean over the group's query heads of their probabilities (selection score)."""
    hq = q.shape[1]
    heads = [h for h in range(hq) if group_of(h, hq, n_kv) == g]
    return np.mean([step_probabilities(q, k_seq, lens, b, h, n_kv) for h in heads], axis=0)


def top_k_positions(scores, k):
    """k positions of highest score, ties to the lower position, ascending;
    padded with -1 when there are fewer than k positions."""
    scores = np.asarray(scores)
    order = np.lexsort((np.arange(len(scores)), -scores))  # score descending, position ascending
    sel = np.sort(order[:k])
    return np.concatenate([sel, np.full(k - len(sel), -1, dtype=np.int64)]).astype(np.int64)


def anchor_select(q, k_seq, lens, head_is_streaming, k):
    """Index lists [B, n_retrieval_groups, k] of one anchor decode step, in the
    order of the retrieval groups (ascending group id)."""
    n_kv = k_seq.shape[2]
    ret = [g for g in range(n_kv) if not head_is_streaming[g]]
    out = np.empty((q.shape[0], len(ret), k), dtype=np.int64)
    for b in range(q.shape[0]):
        for r, g in enumerate(ret):
            out[b, r] = top_k_positions(group_scores(q, k_seq, lens, b, g, n_kv), k)
    return out


def reuse_decode(q, k_seq, v_seq, lens, head_is_streaming, n_sink, window, indices, mapping_rank):
    """One reuse-layer decode step.  indices [B, n_anchor_retrieval, k] from
    the anchor (entries -1 are padding); mapping_rank[g] = the anchor retrieval
    rank whose list reuse retrieval group g borrows.  Streaming groups attend
    to sink + window.  Returns [B, Hq, D] float64."""
    b_n, hq, d = q.shape
    n_kv = k_seq.shape[2]
    out = np.empty((b_n, hq, d))
    for b in range(b_n):
        p = int(lens[b]) - 1
        for h in range(hq):
            g = group_of(h, hq, n_kv)
            qh = np.asarray(q[b, h][None, :], dtype=np.float64)
            if head_is_streaming[g]:
                kk = np.asarray(k_seq[b, :p + 1, g], dtype=np.float64)
                vv = np.asarray(v_seq[b, :p + 1, g], dtype=np.float64)
                out[b, h] = attend_rows(qh, [p], kk, vv, True, n_sink, window)[0]
                continue
            idx = np.asarray(indices[b, mapping_rank[g]])
            idx = idx[idx >= 0]
            kk = np.asarray(k_seq[b, idx, g], dtype=np.float64)
            vv = np.asarray(v_seq[b, idx, g], dtype=np.float64)
            s = (kk @ qh[0]) / np.sqrt(d)
            w = np.exp(s - s.max())
            out[b, h] = (w @ vv) / w.sum()
    return out


def mapping_to_rank(mapping, anchor_is_streaming):
    """Anchor group ids of group_mapping() -> their rank among the anchor's
    retrieval groups (the row of the anchor's index lists); -1 stays -1."""
    ret = [g for g in range(len(anchor_is_streaming)) if not anchor_is_streaming[g]]
    return np.array([ret.index(m) if m >= 0 else -1 for m in mapping], dtype=np.int64)
