"""Fused decode step (aoh_decode_step) on the GPU.

Two runs are built from the same seeded sequence: one takes every step as
aoh_kv_append at lens - 1 followed by aoh_decode, the other as one
aoh_decode_step.  Outputs and both caches must agree bit for bit after every
step; the fused run is also checked against the oracle's decode (Sec. 5,
Eq. 8) and against the oracle's cache placement model."""
import numpy as np
import pytest
import torch

from paper_2608_06849_amd import AohError, aoh_decode_step
from tests.helpers import assert_parity, bits
from tests.test_gpu_decode import DECODE_CASES, Run

pytestmark = pytest.mark.gpu
DEV = "cuda"


def step_tokens(run):
    pos = run.lens.cpu().numpy()
    kn = torch.stack([run.k_seq[b, int(pos[b])] for b in range(run.B)]).to(DEV)
    vn = torch.stack([run.v_seq[b, int(pos[b])] for b in range(run.B)]).to(DEV)
    return kn, vn


def fused_step(run, s):
    kn, vn = step_tokens(run)
    run.lens += 1
    q = run.q_steps[s].to(DEV)
    out = aoh_decode_step(q, kn, vn, run.full, run.ring, run.mask, run.lens, run.n_sink, run.window,
                          workspace=run.ws)
    torch.cuda.synchronize()
    return q, out


def assert_same_caches(a, b, what):
    for ca, cb in ((a.full, b.full), (a.ring, b.ring)):
        if ca is None:
            continue
        assert np.array_equal(bits(ca.k), bits(cb.k)), f"{what}: K caches differ"
        assert np.array_equal(bits(ca.v), bits(cb.v)), f"{what}: V caches differ"


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("B,Hq,Hkv,D,mask,n_sink,window,prompt,steps", DECODE_CASES)
def test_step_equals_append_then_decode(B, Hq, Hkv, D, mask, n_sink, window, prompt, steps, dtype):
    seed = B * 100 + Hq + steps
    ref = Run(B, Hq, Hkv, D, mask, n_sink, window, prompt, steps, dtype, seed=seed)
    run = Run(B, Hq, Hkv, D, mask, n_sink, window, prompt, steps, dtype, seed=seed)
    for r in (ref, run):
        r.append_prompts()
    for s in range(steps):
        _, want = ref.step(s)
        q, got = fused_step(run, s)
        assert np.array_equal(bits(got), bits(want)), f"step {s}: output differs from append + decode"
        assert_same_caches(ref, run, f"step {s}")
        assert_parity(got, run.expected(q), dtype, f"fused step {s}")
    run.check_caches()


def test_step_ragged_lengths_fill_pages():
    # one sequence per residue of the position within its page (0..15), so the
    # new token lands on every row of a page and on the first row of a fresh
    # page; the ring wraps for the longer prompts
    prompt = [16 * (i + 1) + i for i in range(16)]
    ref = Run(16, 8, 2, 128, [0, 1], 3, 29, prompt, 2, torch.bfloat16, seed=77)
    run = Run(16, 8, 2, 128, [0, 1], 3, 29, prompt, 2, torch.bfloat16, seed=77)
    for r in (ref, run):
        r.append_prompts()
    for s in range(2):
        _, want = ref.step(s)
        q, got = fused_step(run, s)
        assert np.array_equal(bits(got), bits(want)), f"step {s}: output differs"
        assert_same_caches(ref, run, f"step {s}")
        assert_parity(got, run.expected(q), torch.bfloat16, f"ragged step {s}")
    run.check_caches()


def test_step_first_token_of_empty_cache():
    # lens = 1 after the step: the cache held nothing before; the output is the
    # value of the new token itself
    run = Run(2, 4, 2, 64, [0, 1], 2, 8, [0, 0], 1, torch.bfloat16, seed=5)
    q, got = fused_step(run, 0)
    v0 = run.v_seq[:, 0].float()                       # [B, Hkv, D]
    want = v0.repeat_interleave(2, dim=1).numpy()      # query head h -> KV head h // 2
    assert np.abs(got.float().cpu().numpy() - want).max() <= 1e-2
    run.check_caches()


def test_step_rejects_misshapen_new_token():
    run = Run(1, 4, 2, 64, [0, 1], 2, 8, [10], 1, torch.bfloat16, seed=6)
    run.append_prompts()
    q = run.q_steps[0].to(DEV)
    kn = torch.zeros((1, 1, 2, 64), dtype=torch.bfloat16, device=DEV)  # [B, 1, Hkv, D]: one dim too many
    with pytest.raises(AohError):
        aoh_decode_step(q, kn, kn, run.full, run.ring, run.mask, run.lens, 2, 8, workspace=run.ws)
    kn = torch.zeros((1, 3, 64), dtype=torch.bfloat16, device=DEV)     # wrong Hkv
    with pytest.raises(AohError):
        aoh_decode_step(q, kn, kn, run.full, run.ring, run.mask, run.lens, 2, 8, workspace=run.ws)
    kn = torch.zeros((1, 2, 64), dtype=torch.float32, device=DEV)      # dtype of q required
    with pytest.raises(AohError):
        aoh_decode_step(q, kn, kn, run.full, run.ring, run.mask, run.lens, 2, 8, workspace=run.ws)
    # nothing was written by the rejected calls
    ref = Run(1, 4, 2, 64, [0, 1], 2, 8, [10], 1, torch.bfloat16, seed=6)
    ref.append_prompts()
    assert_same_caches(ref, run, "after rejected calls")
