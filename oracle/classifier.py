"""Oracle of the AoH head classifier (paper Sec. 4 and Algorithm 1; group-level
classification of the GQA appendix).  CPU, numpy float64.

TEST INFRASTRUCTURE: only tests/, the smoke check and the CPU baseline of the
benchmark use this module.

The classifier scores every query head h of a layer by the effective rank of
its kernel attention matrix M_h = W_K^T W_Q (Sec. 4, Eq. 2), where W_Q^h and
W_K^g are d_head x d_model slices of the projection weights (PyTorch Linear
layout: output rows x input columns; query head h owns rows h*d_head ...
(h+1)*d_head - 1 of W_Q, KV group g owns the same rows of W_K, and query head h
belongs to group g = h // (Hq / Hkv)).

  * singular values: from the d_head x d_head proxy
      C_h = (W_Q^h W_Q^h^T)(W_K^g W_K^g^T),  sigma_k = sqrt(max(lambda_k(C_h), 0))
    (Sec. 4 "Optimized Implementation", Eqs. 5-6; Algorithm 1);
  * effective rank: the exponential of the Shannon entropy of the singular
    values normalised to sum one, over the nonzero ones (Sec. 4, Eq. 4);
  * group score: the mean over the query heads of the group; the
    k = ceil((1 - s) G) groups with the lowest score are retrieval groups, the
    rest streaming (Sec. 4 "Group-level Classification"; GQA appendix).

Readings where the paper leaves room:
  * ties at the k-th score: exactly k groups are retrieval, chosen by a stable
    ascending sort, so the lower group index wins a tie (Algorithm 1's "<=" can
    select more than k on a tie; the prose says k);
  * "nonzero" singular values: the terms with sigma = 0 (after the clamp) are
    left out, i.e. 0 log 0 = 0.

Pins (tests/test_oracle_classifier.py): the proxy's spectrum equals the full
SVD of M_h on small random weights (Eq. 2-3 vs Eq. 5-6); a flat spectrum gives
eff_rank = rank exactly; rank one gives 1; singular values (2, 1, 1) give 2^1.5;
invariance under weight scaling and under a shared orthogonal change of basis;
1 <= eff_rank <= d_head; hand-built layers with planted flat spectra fix the
group means and the labels, ties included.
"""
import numpy as np

from .accounting import n_retrieval_groups


def kernel_attention_matrix(wq_h, wk_g):
    """M_h = W_K^T W_Q, d_model x d_model (Sec. 4, Eq. 2).  Small inputs only."""
    return np.asarray(wk_g, np.float64).T @ np.asarray(wq_h, np.float64)


def singular_values_full(wq_h, wk_g):
    """All singular values of M_h by a dense SVD (Sec. 4, Eq. 3), descending.
    Used only to pin the proxy on small inputs."""
    return np.linalg.svd(kernel_attention_matrix(wq_h, wk_g), compute_uv=False)


def proxy_matrix(wq_h, wk_g):
    """C_h = (W_Q W_Q^T)(W_K W_K^T), d_head x d_head (Sec. 4, Eq. 5)."""
    wq = np.asarray(wq_h, np.float64)
    wk = np.asarray(wk_g, np.float64)
    return (wq @ wq.T) @ (wk @ wk.T)


def singular_values(wq_h, wk_g):
    """sigma_k = sqrt(max(lambda_k(C_h), 0)), descending (Eq. 6, Algorithm 1).
    C_h is a product of two symmetric PSD matrices, so its eigenvalues are real
    and non-negative in exact arithmetic; the real part is kept."""
    lam = np.linalg.eigvals(proxy_matrix(wq_h, wk_g)).real
    return np.sort(np.sqrt(np.maximum(lam, 0.0)))[::-1]


def effective_rank(sigma):
    """exp(-sum_k p_k log p_k), p_k = sigma_k / sum_j sigma_j over the nonzero
    sigma (Sec. 4, Eq. 4).  Lies in [1, number of nonzero sigma]."""
    s = np.asarray(sigma, np.float64)
    s = s[s > 0]
    p = s / s.sum()
    return float(np.exp(-np.sum(p * np.log(p))))


def head_effective_ranks(wq, wk, d_head):
    """eff_rank of every query head of one layer.
    wq: [Hq * d_head, d_model]; wk: [Hkv * d_head, d_model]."""
    wq = np.asarray(wq, np.float64)
    wk = np.asarray(wk, np.float64)
    hq, hkv = wq.shape[0] // d_head, wk.shape[0] // d_head
    assert hq * d_head == wq.shape[0] and hkv * d_head == wk.shape[0] and hq % hkv == 0
    gs = hq // hkv
    out = np.empty(hq)
    for h in range(hq):
        g = h // gs
        out[h] = effective_rank(singular_values(wq[h * d_head:(h + 1) * d_head],
                                                wk[g * d_head:(g + 1) * d_head]))
    return out


def group_scores(head_ranks, n_kv):
    """Mean eff_rank over the query heads of each KV group (Sec. 4)."""
    r = np.asarray(head_ranks, np.float64)
    return r.reshape(n_kv, -1).mean(axis=1)


def select_retrieval(scores, n_retrieval):
    """head_is_streaming per group: the n_retrieval lowest scores are retrieval
    (0), the rest streaming (1); ties go to the lower index (stable sort)."""
    order = np.argsort(np.asarray(scores), kind="stable")
    mask = np.ones(len(scores), np.uint8)
    mask[order[:n_retrieval]] = 0
    return mask


def classify_layer(wq, wk, d_head, sparsity=None, n_retrieval=None):
    """One layer of Algorithm 1 at group level.  Give either the target
    sparsity s (k = ceil((1 - s) G)) or k itself."""
    hkv = np.asarray(wk).shape[0] // d_head
    if n_retrieval is None:
        n_retrieval = n_retrieval_groups(hkv, sparsity)
    hr = head_effective_ranks(wq, wk, d_head)
    gsc = group_scores(hr, hkv)
    return {"head_rank": hr, "group_score": gsc, "head_is_streaming": select_retrieval(gsc, n_retrieval)}


def classify_model(wq, wk, d_head, sparsity=None, n_retrieval=None):
    """Algorithm 1 over layers: wq [L, Hq * d_head, d_model], wk [L, Hkv * d_head, d_model]."""
    per = [classify_layer(wq[l], wk[l], d_head, sparsity, n_retrieval) for l in range(len(wq))]
    return {k: np.stack([p[k] for p in per]) for k in per[0]}
