"""GPU: smoes_mi_loss_noalloc (scratch in the library's fixed device array,
no workspace) against smoes_mi_loss with a caller workspace, through the C
ABI: the same kernels in the same order, so the outputs must agree bit for
bit (and so meet the MI bars of 1e-5 relative against the oracle). Two calls
in a row, the second with a smaller problem, so that the second reads
nothing the first left behind; then a problem beyond the fixed array is
refused on the host with SMOES_ERR_SCRATCH."""
from __future__ import annotations

import ctypes

import numpy as np
import pytest
import torch

import oracle as O
from paper_2604_23996_amd import smoes as S
from paper_2604_23996_amd import workloads as W
from tests.gpu_util import host, rel_err, say, t

pytestmark = pytest.mark.gpu


def _inputs(seed, T, E, B, n_batch):
    rng = np.random.default_rng(seed)
    probs = W.random_probs(rng, T, E, 0.5)
    M = W.random_soft_scores(rng, T)
    e2b = W.random_bin_map(rng, E, B, contiguous=False)
    tilt = np.where(e2b < B // 2, 1.0, -1.0)[None, :] * (M[:, :1] - 0.5)  # gate leaning with the score
    probs = probs * np.exp(2.0 * tilt)
    probs = (probs / probs.sum(axis=1, keepdims=True)).astype(np.float32)
    off = W.random_offsets(rng, T, n_batch) if n_batch > 1 else None
    return probs, M, off, e2b


@pytest.mark.parametrize("first,second", [((16384, 160, 8, 16), (3000, 64, 8, 3)),
                                          ((5000, 256, 64, 1), (1, 8, 2, 1))])
def test_noalloc_matches_workspace_call_twice(first, second):
    for seed, (T, E, B, nb) in enumerate((first, second)):
        probs, M, off, e2b = _inputs(50 + seed, T, E, B, nb)
        say("mi noalloc", T, E, B, nb)
        dp, dM, doff, de2b = t(probs), t(M), t(off), t(e2b)
        a = S.mi_loss(dp, dM, doff, de2b, B, grad_scale=0.7)
        b = S.mi_loss_noalloc(dp, dM, doff, de2b, B, grad_scale=0.7)
        torch.cuda.synchronize()
        for u, v in zip(a, b):
            assert torch.equal(u, v)
        off_ref = off if off is not None else np.array([0, T])
        I = O.mi_per_sample(probs, M, off_ref, e2b, B)
        assert np.all(np.abs(host(b[0]) - I) <= 1e-5 * np.abs(I) + 1e-14)
        G = O.mi_loss_grad_logits(probs, M, off_ref, e2b, B, grad_scale=0.7)
        assert rel_err(host(b[2]), G) <= 1e-5


def test_noalloc_without_gradient_and_refusal():
    probs, M, off, e2b = _inputs(60, 2000, 64, 8, 4)
    dp, dM, doff, de2b = t(probs), t(M), t(off), t(e2b)
    say("mi noalloc, no gradient")
    a = S.mi_loss(dp, dM, doff, de2b, 8, want_grad=False)
    b = S.mi_loss_noalloc(dp, dM, doff, de2b, 8, want_grad=False)
    torch.cuda.synchronize()
    assert b[2] is None and torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
    # beyond the fixed array: refused on the host before anything is launched
    L = S.lib()
    T_big, nb_big = 1 << 22, 16
    assert L.smoes_mi_workspace_size(T_big, 256, nb_big, 8) > S.SMOES_NOALLOC_SCRATCH_BYTES
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: the call returns before any launch
    rc = L.smoes_mi_loss_noalloc(fake, fake, T_big, 256, fake, nb_big, fake, 8, 1.0, fake, fake, fake, None)
    assert rc == S.SMOES_ERR_SCRATCH
    assert "scratch" in S.status_string(rc)
