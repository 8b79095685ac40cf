"""GPU parity of smoes_binning against the oracle: momentum-adaptive bins
(Eq. 10-11), the bin-level load balance loss and its logit gradient (Eq. 16)
and MSI (Eq. 18-19). Integer results and the float64 EMA are compared bit
for bit; the loss, its gradient and MSI within float64-accumulation /
float32-output rounding."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle as O
from paper_2604_23996_amd import smoes as S
from tests.gpu_util import DEV, host, rel_err, say, t

pytestmark = pytest.mark.gpu


def _inputs(seed, T, E, k, n_bins, skew=0.0, one_modality=None, bins="perm"):
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((T, E)).astype(np.float32)
    z += np.float32(skew) * np.linspace(0, 1, E, dtype=np.float32)[None, :]  # load imbalance
    g = O.softmax_rows(z).astype(np.float32)
    idx = O.topk_select(z, k).astype(np.int32)
    mid = (rng.random(T) < 0.3).astype(np.uint8) if one_modality is None else np.full(T, one_modality, np.uint8)
    NB = E // n_bins
    e2b = (np.arange(E) // NB).astype(np.int32)
    if bins == "perm":
        e2b = rng.permutation(e2b).astype(np.int32)
    ema = rng.integers(0, 50, size=(2, E)).astype(np.float64) * 7.25
    return g, idx, mid, e2b, ema


def _run(g, idx, mid, e2b, n_bins, ema, beta=0.99, scale=0.5, accumulate=False, base=None):
    dl = None
    if accumulate:
        dl = t(base.astype(np.float32))
    ema_d = t(ema) if ema is not None else None
    out = S.binning(t(g), t(idx), t(mid), t(e2b), n_bins, beta=beta, load_ema=ema_d, grad_scale=scale,
                    dlogits=dl, accumulate=accumulate)
    torch.cuda.synchronize()
    res = {k: host(v) for k, v in out.items() if v is not None}
    if ema_d is not None:
        res["load_ema"] = ema_d.cpu().numpy()
    return res


def _check(g, idx, mid, e2b, n_bins, ema, res, beta=0.99, scale=0.5, base=None):
    E = g.shape[1]
    C = O.modality_expert_counts(idx, mid, E)
    assert np.array_equal(res["counts"], C)
    cb = O.load_ema_update(ema, C, beta) if ema is not None else C.astype(np.float64)
    if ema is not None:
        assert np.array_equal(res["load_ema"], cb)  # bit for bit
    fs = O.f_spec(cb)
    assert np.array_equal(res["f_spec"], fs)
    assert np.array_equal(res["expert_to_bin_next"], O.adaptive_bins(fs, n_bins))
    L = O.bin_balance_loss(g, idx, e2b, n_bins)
    assert abs(res["bal_loss"][0] - L) <= 1e-6 * abs(L) + 1e-7, (res["bal_loss"][0], L)
    assert abs(res["msi"][0] - O.msi(C[1], C[0])) <= 1e-6
    if "dlogits" in res:
        ref = O.bin_balance_grad_logits(g, idx, e2b, n_bins, grad_scale=scale)
        if base is not None:
            ref = ref + base.astype(np.float32)
        assert rel_err(res["dlogits"], ref) <= 1e-6


CASES = [
    # seed, T, E, k, n_bins, skew, one_modality, bins
    (1, 300, 16, 4, 4, 0.0, None, "perm"),
    (2, 1000, 64, 6, 8, 3.0, None, "contig"),
    (3, 1, 8, 2, 2, 0.0, None, "perm"),         # one token: most bins unreached
    (4, 257, 12, 12, 3, 0.0, None, "perm"),     # k = E
    (5, 130, 10, 3, 1, 0.0, None, "perm"),      # one bin
    (6, 200, 20, 2, 20, 0.0, None, "perm"),     # N_B = 1
    (7, 500, 32, 4, 8, 0.0, 1, "perm"),         # text only
    (8, 700, 256, 16, 64, 2.0, None, "perm"),   # maxima
    (9, 513, 160, 6, 8, 4.0, None, "contig"),   # config-4 expert count, skewed
]


@pytest.mark.parametrize("seed,T,E,k,n_bins,skew,one_mod,bins", CASES)
def test_binning(seed, T, E, k, n_bins, skew, one_mod, bins):
    say("binning", seed, T, E, k, n_bins)
    g, idx, mid, e2b, ema = _inputs(seed, T, E, k, n_bins, skew, one_mod, bins)
    res = _run(g, idx, mid, e2b, n_bins, ema)
    _check(g, idx, mid, e2b, n_bins, ema, res)


def test_binning_accumulates_onto_a_gradient_and_without_ema():
    g, idx, mid, e2b, ema = _inputs(11, 400, 16, 4, 4)
    base = np.random.default_rng(12).standard_normal(g.shape)
    res = _run(g, idx, mid, e2b, 4, None, accumulate=True, base=base)
    _check(g, idx, mid, e2b, 4, None, res, base=base)


def test_binning_ties_and_idle_experts():
    """Equal loads tie (lower expert index first); experts without load get
    f_spec = 1/2."""
    T, E, k, nb = 64, 8, 2, 4
    g, idx, mid, e2b, _ = _inputs(13, T, E, k, nb)
    idx = np.tile(np.array([0, 1], np.int32), (T, 1))  # only experts 0 and 1 are used
    ema = np.zeros((2, E))
    ema[:, 4:6] = 3.0  # experts 4, 5: equal loads, f = 1/2, tying with the idle experts
    res = _run(g, idx, mid, e2b, nb, ema)
    _check(g, idx, mid, e2b, nb, ema, res)


def test_binning_empty_batch_decays_the_ema():
    E, nb = 16, 4
    rng = np.random.default_rng(14)
    ema = rng.random((2, E)) * 100
    e2b = (np.arange(E) // 4).astype(np.int32)
    ema_d = t(ema)
    empty_f = torch.empty((0, E), dtype=torch.float32, device=DEV)
    empty_i = torch.empty((0, 2), dtype=torch.int32, device=DEV)
    empty_u = torch.empty(0, dtype=torch.uint8, device=DEV)
    out = S.binning(empty_f, empty_i, empty_u, t(e2b), nb, beta=0.9, load_ema=ema_d, want_grad=False)
    torch.cuda.synchronize()
    cb = O.load_ema_update(ema, np.zeros((2, E)), 0.9)
    assert np.array_equal(ema_d.cpu().numpy(), cb)
    assert np.array_equal(host(out["expert_to_bin_next"]), O.adaptive_bins(O.f_spec(cb), nb))
    assert host(out["bal_loss"])[0] == 0.0


@pytest.mark.parametrize("T,E,k,n_bins", [(4096, 64, 6, 8), (16384, 160, 6, 8)])
def test_binning_full_size(T, E, k, n_bins):
    """The routing shapes of the benchmark workloads (64 experts, top-6 over
    4096 tokens; 160 experts, top-6 over 16384 tokens)."""
    say("binning full", T, E)
    g, idx, mid, e2b, ema = _inputs(15 + E, T, E, k, n_bins, 2.0, None, "contig")
    res = _run(g, idx, mid, e2b, n_bins, ema)
    _check(g, idx, mid, e2b, n_bins, ema, res)


def test_binning_deterministic():
    g, idx, mid, e2b, ema = _inputs(16, 900, 32, 4, 8)
    a = _run(g, idx, mid, e2b, 8, ema)
    b = _run(g, idx, mid, e2b, 8, ema)
    for key in a:
        assert np.array_equal(a[key], b[key]), key
