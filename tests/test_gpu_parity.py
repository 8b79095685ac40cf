"""GPU parity: every entry point of the C ABI against the CPU oracle on the
same seeded inputs, element by element.

Tolerances (from the layer's stated targets):
  * top-k indices and the permutation: bit-exact (top-k where the oracle's
    k-th vs (k+1)-th logit gap exceeds 1e-4; the permutation is fed the same
    index array on both sides);
  * modality scores and MI: relative error <= 1e-5 (fp32 outputs of fp64
    accumulations); dlogits: normwise relative error <= 1e-5;
  * layer outputs: |gpu - ref| <= 1e-2 + 2e-2 |ref| elementwise, plus a
    normwise relative error <= 2e-2 (bf16 operands, fp32 accumulation) or
    <= 1e-5 (fp32 layers), because the absolute bound alone is loose for
    outputs of magnitude ~1e-3; the norm is that of the routed part for layers
    without shared experts and of the whole output otherwise.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2604_23996_amd import smoes as S
from paper_2604_23996_amd import workloads as W
from tests.gpu_util import (DEV, check_expert_rows, check_topk, gate_rtol, gauss_state_dev, host, rel_err,
                            run_gpu_layer, run_oracle_layer, say, t)

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _name_case(request):
    say("case", request.node.nodeid)
    yield


# ---------------------------------------------------------------- router

ROUTE_CASES = [
    # (T, d, E, k, dtype, bias)
    (100, 136, 40, 5, W.BF16, False),   # ragged T, d % 16 == 8, E not a multiple of 32
    (257, 256, 64, 6, W.BF16, False),
    (64, 64, 160, 6, W.BF16, True),
    (33, 512, 256, 16, W.BF16, False),  # maximum E and k
    (300, 1032, 100, 8, W.BF16, True),  # 7 expert tiles: 4 per expert half, the last one empty;
                                        # 33 k-steps in 4 ranges (the last one shorter), partial last step
    (2000, 2048, 128, 8, W.BF16, False),  # 16 tiles of 128 tokens, 8 ranges of the hidden dimension
    (200, 512, 224, 8, W.BF16, True),   # 7 expert tiles per half: three ring slots
    (129, 320, 192, 4, W.BF16, False),  # 6 expert tiles per half, one token past a 128-token tile
    (5000, 512, 64, 6, W.BF16, False),  # ragged last token tile, 2 ranges
    (31, 2048, 8, 2, W.BF16, False),
    # many tokens: near-equal logits inside some tokens' top-k (their order is free), a last
    # 128-token tile past T, one range of the hidden dimension at d = 256
    (12289, 1032, 100, 8, W.BF16, True),
    (12288, 256, 256, 16, W.BF16, False),  # the maxima over many tokens
    (16384, 96, 8, 2, W.BF16, False),      # one expert tile, one k-step range of three steps
    (1, 8, 1, 1, W.BF16, False),        # degenerate: one token, one expert
    (100, 72, 8, 2, W.F32, False),
    (70, 256, 20, 3, W.F32, True),
]


@pytest.mark.parametrize("T,d,E,k,dt,bias", ROUTE_CASES)
@pytest.mark.parametrize("renorm", [False, True])
def test_route(T, d, E, k, dt, bias, renorm):
    rng = np.random.default_rng(T * 7 + d + E)
    x32 = rng.standard_normal((T, d)).astype(np.float32)
    x = W.f32_to_bf16_bits(x32) if dt == W.BF16 else x32
    w = (0.05 * rng.standard_normal((E, d))).astype(np.float32)
    b = rng.standard_normal(E).astype(np.float32) if bias else None
    z, g, idx, wt = O.route(x, w, k, b, renorm)
    r = S.route(t(x), t(w), k, t(b), renorm_topk=renorm)
    zg, gg, ig, wg = (host(r["logits"]), host(r["probs"]), host(r["topk_idx"]), host(r["topk_w"]))
    # fp32-faithful logits: error within a few fp32 ulps of sum |x w|
    scale = np.abs(O.widen(x)) @ np.abs(w.astype(np.float64)).T + (np.abs(b) if bias else 0)
    assert np.all(np.abs(zg - z) <= 4e-7 * scale + 1e-30), np.max(np.abs(zg - z) / scale)
    rt = gate_rtol(x, w, b)
    assert np.all(np.abs(gg - g) <= rt * g + 1e-12)
    assert np.allclose(gg.sum(axis=1), 1.0, atol=1e-5)
    clear = check_topk(ig, idx, z, k)
    assert np.all(np.abs(wg[clear] - wt[clear]) <= rt[clear] * wt[clear] + 1e-12)
    # every token: the weights are the GPU's own gate values at its own choice
    gsel = np.take_along_axis(gg, ig.astype(np.int64), axis=1)
    if renorm:
        want = gsel / gsel.sum(axis=1, keepdims=True)
        assert np.all(np.abs(wg - want) <= 1e-6 * want + 1e-12)
    else:
        assert np.array_equal(wg, gsel)


def test_route_partial_last_step_reads_no_next_row():
    # d = 40: the last 32-wide k-step is partly past d; its lanes past d must
    # not read the next token's row (an inf there would give 0 * inf = NaN)
    T, d, E, k = 40, 40, 64, 6
    rng = np.random.default_rng(11)
    x32 = rng.standard_normal((T, d)).astype(np.float32)
    x32[5, :8] = np.inf
    x = W.f32_to_bf16_bits(x32)
    w = (0.05 * rng.standard_normal((E, d))).astype(np.float32)
    r = S.route(t(x), t(w), k)
    ok = np.arange(T) != 5
    z, g, idx, _ = O.route(x[ok], w, k, None, False)
    zg, gg = host(r["logits"])[ok], host(r["probs"])[ok]
    assert np.all(np.isfinite(zg)) and np.all(np.isfinite(gg))
    scale = np.abs(O.widen(x[ok])) @ np.abs(w.astype(np.float64)).T
    assert np.all(np.abs(zg - z) <= 4e-7 * scale + 1e-30)
    check_topk(host(r["topk_idx"])[ok], idx, z, k)


# ---------------------------------------------------------------- modality score

MOD_CASES = [
    # (T, d, dtype, update, tau_scale, beta, state)
    (333, 200, W.BF16, False, 0.5, 0.99, "random"),
    (600, 1024, W.BF16, True, 0.5, 0.99, "zero"),
    (600, 1024, W.BF16, True, 0.05, 0.9, "random"),
    (257, 64, W.F32, True, 1.0, 0.99, "random"),
    (300, 256, W.BF16, True, 0.1, 0.99, "one-modality"),
    (1, 8, W.F32, True, 0.3, 0.5, "zero"),
]


@pytest.mark.parametrize("T,d,dt,update,tau_scale,beta,state", MOD_CASES)
def test_modality_score(T, d, dt, update, tau_scale, beta, state):
    rng = np.random.default_rng(T + d)
    mu = rng.standard_normal((2, d)).astype(np.float32) * 0.5
    mid = rng.integers(0, 2, size=T).astype(np.uint8)
    if state == "one-modality":
        mid[:] = 0
    x32 = (mu[mid] + rng.standard_normal((T, d)) * np.where(mid == 0, 1.0, 1.5)[:, None]).astype(np.float32)
    x = W.f32_to_bf16_bits(x32) if dt == W.BF16 else x32
    if state == "zero" or state == "one-modality":
        n0 = np.zeros(2, np.float32); smu0 = np.zeros((2, d), np.float32); ssig0 = np.zeros((2, d), np.float32)
        if state == "one-modality":
            n0, smu0, ssig0 = W.random_gauss_state(rng, d, count=50.0)
    else:
        n0, smu0, ssig0 = W.random_gauss_state(rng, d)
    tau = tau_scale * d
    st = O.GaussState.of(n0, smu0, ssig0)
    if update:
        st = O.gauss_update(st, x, mid, beta)
    mu_o, var_o = O.gauss_params(st, 1e-6)
    M_ref = O.modality_score(x, mu_o, var_o, tau)
    n, smu, ssig = t(n0), t(smu0), t(ssig0)
    M = host(S.modality_score(t(x), n, smu, ssig, t(mid), update=update, beta=beta, tau=tau, var_floor=1e-6))
    assert np.all(np.abs(M - M_ref) <= 1e-5 * M_ref + 1e-30), np.max(np.abs(M - M_ref) / M_ref)
    assert np.allclose(M.sum(axis=1), 1.0, atol=1e-6)
    if update:
        assert np.allclose(host(n), st.n, rtol=1e-6)
        assert np.allclose(host(smu), st.s_mu, rtol=2e-6, atol=1e-6 * np.abs(st.s_mu).max())
        assert np.allclose(host(ssig), st.s_sig, rtol=2e-6, atol=1e-6 * np.abs(st.s_sig).max())


def test_modality_tau_default_is_half_d():
    rng = np.random.default_rng(5)
    d, T = 128, 64
    x = rng.standard_normal((T, d)).astype(np.float32)
    n0, smu0, ssig0 = W.random_gauss_state(rng, d)
    a = host(S.modality_score(t(x), t(n0), t(smu0), t(ssig0), tau=0.0))
    b = host(S.modality_score(t(x), t(n0), t(smu0), t(ssig0), tau=0.5 * d))
    assert np.array_equal(a, b)


# ---------------------------------------------------------------- MI loss + gradient

MI_CASES = [
    # (T, E, B, offsets kind, bin map, score kind, concentration)
    (500, 64, 8, "with-empty", "random", "soft", 1.0),
    (2000, 160, 8, "16", "contiguous", "soft", 0.3),
    (1, 8, 2, "none", "contiguous", "soft", 1.0),
    (100, 256, 64, "3", "random", "hard", 0.1),
    (3000, 128, 16, "none", "contiguous", "soft", 2.0),
    (4096, 64, 8, "4", "contiguous", "aligned", 0.5),
]


def _mi_inputs(T, E, B, offk, binmap, scores, conc, seed=11):
    rng = np.random.default_rng(seed + T + E)
    probs = W.random_probs(rng, T, E, conc)
    if scores == "hard":
        mid = rng.integers(0, 2, size=T)
        M = np.stack([1.0 - mid, mid], axis=1).astype(np.float32)
    else:
        M = W.random_soft_scores(rng, T)
    e2b = W.random_bin_map(rng, E, B, contiguous=(binmap == "contiguous"))
    if scores == "aligned":  # gate mass leaning to the bins that match the score
        tilt = np.where(e2b < B // 2, 1.0, -1.0)[None, :] * (M[:, :1] - 0.5)
        probs = probs * np.exp(2.0 * tilt)
        probs = (probs / probs.sum(axis=1, keepdims=True)).astype(np.float32)
    if offk == "none":
        off = None
    elif offk == "with-empty":
        off = np.array([0, 120, 120, 371, 500], dtype=np.int32)
    else:
        off = W.random_offsets(rng, T, int(offk))
    return probs, M, off, e2b


@pytest.mark.parametrize("T,E,B,offk,binmap,scores,conc", MI_CASES)
def test_mi_loss(T, E, B, offk, binmap, scores, conc):
    probs, M, off, e2b = _mi_inputs(T, E, B, offk, binmap, scores, conc)
    off_ref = off if off is not None else np.array([0, T])
    I_ref = O.mi_per_sample(probs, M, off_ref, e2b, B)
    L_ref = -I_ref.mean()
    G_ref = O.mi_loss_grad_logits(probs, M, off_ref, e2b, B, grad_scale=0.37)
    mi, loss, dl = S.mi_loss(t(probs), t(M), t(off), t(e2b), B, grad_scale=0.37)
    mi, loss, dl = host(mi), host(loss), host(dl)
    assert np.all(np.abs(mi - I_ref) <= 1e-5 * np.abs(I_ref) + 1e-14), (mi, I_ref)
    assert abs(loss[0] - L_ref) <= 1e-5 * abs(L_ref) + 1e-14
    assert rel_err(dl, G_ref) <= 1e-5, rel_err(dl, G_ref)
    assert np.max(np.abs(dl.sum(axis=1))) <= 1e-6 * np.max(np.abs(G_ref)) + 1e-30


def test_mi_loss_without_gradient_and_determinism():
    probs, M, off, e2b = _mi_inputs(1000, 64, 8, "4", "contiguous", "soft", 1.0)
    a = S.mi_loss(t(probs), t(M), t(off), t(e2b), 8, want_grad=False)
    b = S.mi_loss(t(probs), t(M), t(off), t(e2b), 8)
    c = S.mi_loss(t(probs), t(M), t(off), t(e2b), 8)
    assert a[2] is None
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
    assert torch.equal(b[2], c[2])  # bit-for-bit reproducible


# ---------------------------------------------------------------- permutation

PERM_CASES = [
    # (T, E, k, skew, with_x)
    (1000, 64, 6, 0.0, True),
    (1, 4, 1, 0.0, True),
    (257, 160, 6, 6.0, False),  # skewed: many empty experts
    (300, 256, 16, 0.0, True),
    (4096, 128, 8, 1.0, False),
]


@pytest.mark.parametrize("T,E,k,skew,with_x", PERM_CASES)
@pytest.mark.parametrize("dt", [W.BF16, W.F32])
def test_permute(T, E, k, skew, with_x, dt):
    rng = np.random.default_rng(T + E + k)
    idx = W.random_topk(rng, T, E, k, skew)
    counts, off_ref, perm_ref, inv_ref = O.permutation(idx, E)
    x = None
    if with_x:
        x32 = rng.standard_normal((T, 64)).astype(np.float32)
        x = W.f32_to_bf16_bits(x32) if dt == W.BF16 else x32
    off, perm, inv, xp = S.permute(t(idx), E, t(x) if with_x else None)
    assert np.array_equal(host(off), off_ref)
    assert np.array_equal(host(perm), perm_ref)
    assert np.array_equal(host(inv), inv_ref)
    if with_x:
        xs = O.widen(x)
        assert np.array_equal(host(xp), xs[perm_ref])


# ---------------------------------------------------------------- whole layer

def _check_layer(inp, spec, outs, ref, rows=None, fp32=False, routed_outs=None, w_gate=None):
    """Routing, scores, permutation and output of one layer call against the
    oracle. routed_outs: for layers with shared experts, the outputs of the same
    call with the shared experts' down projection zeroed, whose `out` is the
    routed part alone (the shared output is then exactly 0)."""
    cfg = inp.cfg
    z = ref["logits"]
    idx_g = host(outs["topk_idx"])
    clear = check_topk(idx_g, ref["topk_idx"], z, cfg.k)
    g = host(outs["probs"])
    rt = gate_rtol(inp.x, inp.w_gate if w_gate is None else w_gate, inp.logit_bias)
    assert np.all(np.abs(g - ref["probs"]) <= rt * ref["probs"] + 1e-12)
    # combine weights: on every token, the GPU's own gate values at its own
    # choice (the same float32 expression, so bit for bit without renormalisation)
    gsel = np.take_along_axis(g, idx_g.astype(np.int64), axis=1)
    tw = host(outs["topk_w"])
    if spec.renorm_topk:
        want = gsel / gsel.sum(axis=1, keepdims=True)
        assert np.all(np.abs(tw - want) <= 1e-6 * want + 1e-12)
    else:
        assert np.array_equal(tw, gsel)
    assert np.all(np.abs(tw[clear] - ref["topk_w"][clear]) <= rt[clear] * ref["topk_w"][clear] + 1e-12)
    M = host(outs["M"])
    assert np.all(np.abs(M - ref["M"]) <= 1e-5 * ref["M"] + 1e-30), np.max(np.abs(M - ref["M"]) / ref["M"])
    # permutation: exactly the oracle's stable counting sort of the GPU's own
    # top-k (a flipped near tie moves every later row of its experts)
    _, off_r, perm_r, inv_r = O.permutation(idx_g, cfg.E)
    assert np.array_equal(host(outs["expert_offsets"]), off_r)
    assert np.array_equal(host(outs["perm_token"]), perm_r)
    assert np.array_equal(host(outs["perm_inv"]), inv_r)
    # layer output on the checked rows (tokens whose routing is the oracle's)
    out = host(outs["out"])
    sel = np.arange(cfg.T) if rows is None else rows
    ok = clear[sel]
    o = out[sel][ok]
    r_full = ref["out"][ok]
    assert np.all(np.abs(o - r_full) <= 1e-2 + 2e-2 * np.abs(r_full)), np.max(np.abs(o - r_full))
    bar = 1e-5 if fp32 else 2e-2
    if cfg.n_shared == 0:
        o_r = o
    else:
        # whole output against its own norm (the ungated shared experts dominate it) ...
        assert rel_err(o, r_full) <= bar, rel_err(o, r_full)
        # ... and the routed part on its own, from the run without the shared output
        assert routed_outs is not None, "layers with shared experts need the routed-only run"
        assert torch.equal(routed_outs["topk_idx"], outs["topk_idx"])
        o_r = host(routed_outs["out"])[sel][ok]
    r_r = ref["routed"][ok]
    assert np.all(np.abs(o_r - r_r) <= 1e-2 + 2e-2 * np.abs(r_r)), np.max(np.abs(o_r - r_r))
    routed_err = rel_err(o_r, r_r)
    assert routed_err <= bar, routed_err
    return clear


def _routed_run(inp, **kw):
    """The same layer call with the shared down projection zeroed, or None for
    a layer without shared experts."""
    if inp.cfg.n_shared == 0:
        return None
    return run_gpu_layer(inp, zero_shared_down=True, **kw)[2]


def _check_mi(outs, ref, inp, strict):
    mi = host(outs["mi_per_sample"])
    I = ref["mi_per_sample"]
    if strict:
        assert np.all(np.abs(mi - I) <= 1e-5 * np.abs(I) + 1e-14), (mi, I)
    else:
        # conditioning: MI from fp32-rounded oracle gates / scores vs exact
        off = inp.sample_offsets
        I32 = O.mi_per_sample(ref["probs"].astype(np.float32), ref["M"].astype(np.float32), off,
                              inp.expert_to_bin, inp.cfg.n_bins)
        tol = 1e-5 * np.abs(I) + 10 * np.abs(I32 - I) + 1e-13
        assert np.all(np.abs(mi - I) <= tol), (mi, I, tol)
    dl = host(outs["dlogits"])
    return rel_err(dl, ref["dlogits"])


SMALL_LAYERS = [
    dict(d=128, E=16, k=4, inter=96, n_shared=1, n_bins=4, samples=((200, 100), (40, 60)), dtype=W.BF16),
    dict(d=256, E=12, k=3, inter=64, n_shared=0, n_bins=3, samples=((500, 200),), dtype=W.BF16),
    dict(d=64, E=8, k=2, inter=48, n_shared=2, n_bins=2, samples=((90, 40), (10, 3), (60, 60)), dtype=W.F32),
    dict(d=512, E=64, k=6, inter=128, n_shared=2, n_bins=8, samples=((700, 300),), dtype=W.BF16,
         logit_bias=True),
    # ragged for the packed weights: inter % 32 == 16, d % 32 == 8 (partial GEMM2 groups, padded K)
    dict(d=136, E=10, k=3, inter=48, n_shared=2, n_bins=5, samples=((150, 70), (33, 17)), dtype=W.BF16),
    # three tokens
    dict(d=64, E=4, k=2, inter=32, n_shared=0, n_bins=2, samples=((2, 1),), dtype=W.BF16),
    # the maxima: 256 experts, top-16, 64 bins of 4 (about 25 rows per expert: short tiles everywhere)
    dict(d=256, E=256, k=16, inter=64, n_shared=1, n_bins=64, samples=((300, 100),), dtype=W.BF16),
    # no vision token at all (the vision statistics stay empty)
    dict(d=128, E=16, k=4, inter=64, n_shared=1, n_bins=4, samples=((0, 200), (0, 57)), dtype=W.BF16),
    # an empty sample between two others (its MI is 0)
    dict(d=128, E=16, k=4, inter=64, n_shared=0, n_bins=4, samples=((100, 50), (0, 0), (30, 20)), dtype=W.BF16),
    # at least 256 routed rows per expert on average: several full 128-row tiles
    # per expert and last tiles of every height (ragged d and inter too)
    dict(d=136, E=4, k=2, inter=48, n_shared=1, n_bins=2, samples=((500, 300),), dtype=W.BF16),
    dict(d=256, E=6, k=3, inter=160, n_shared=0, n_bins=3, samples=((700, 300), (200, 100)), dtype=W.BF16),
    # more than 12000 tokens: gate values over millions of entries against their derived
    # bar, near-equal logits inside some tokens' top-k; ragged d, a last token tile past T
    dict(d=264, E=40, k=5, inter=64, n_shared=1, n_bins=4, samples=((9000, 3301),), dtype=W.BF16),
    dict(d=512, E=160, k=6, inter=64, n_shared=2, n_bins=8, samples=((6000, 2144), (3000, 1144)), dtype=W.BF16,
         logit_bias=True),
]


@pytest.mark.parametrize("layer", range(len(SMALL_LAYERS)))
@pytest.mark.parametrize("update", [False, True])
def test_layer_small(layer, update):
    kw = dict(SMALL_LAYERS[layer])
    cfg = W.small_config(seed=100 + layer, **kw)
    inp = W.make_layer_inputs(cfg)
    wg = W.aligned_router(inp, 0.5)  # well-conditioned MI
    spec, _, outs, ws = run_gpu_layer(inp, w_gate=wg, update_stats=update, keep_workspace=True)
    ref = run_oracle_layer(inp, w_gate=wg, update_stats=update)
    fp32 = cfg.dtype == W.F32
    _check_layer(inp, spec, outs, ref, fp32=fp32, routed_outs=_routed_run(inp, w_gate=wg, update_stats=update),
                 w_gate=wg)
    check_expert_rows(inp, spec, ws, outs, fp32=fp32)
    assert _check_mi(outs, ref, inp, strict=True) <= 1e-5


@pytest.mark.parametrize("layer", [i for i, L in enumerate(SMALL_LAYERS) if L["dtype"] == W.BF16])
def test_layer_small_rowmajor_weights(layer):
    """bf16 layers with row-major expert weights (the path for weights that
    are not kept packed)."""
    kw = dict(SMALL_LAYERS[layer])
    cfg = W.small_config(seed=100 + layer, **kw)
    inp = W.make_layer_inputs(cfg)
    wg = W.aligned_router(inp, 0.5)
    spec, _, outs, ws = run_gpu_layer(inp, w_gate=wg, packed=False, keep_workspace=True)
    ref = run_oracle_layer(inp, w_gate=wg)
    _check_layer(inp, spec, outs, ref, fp32=False, routed_outs=_routed_run(inp, w_gate=wg, packed=False), w_gate=wg)
    check_expert_rows(inp, spec, ws, outs)


@pytest.mark.parametrize("layer", [i for i, L in enumerate(SMALL_LAYERS) if L["dtype"] == W.BF16])
def test_packed_weights_match_rowmajor(layer):
    """The packed path (16x16x32 matrix instructions) and the row-major path
    (32x32x16) multiply the same bf16 operands and differ only in the order of
    their float32 accumulation, so the outputs agree to a few bf16 roundings."""
    cfg = W.small_config(seed=100 + layer, **dict(SMALL_LAYERS[layer]))
    inp = W.make_layer_inputs(cfg)
    _, _, a = run_gpu_layer(inp, packed=True)
    _, _, b = run_gpu_layer(inp, packed=False)
    a, b = a["out"].float().cpu(), b["out"].float().cpu()
    assert torch.all(torch.isfinite(a))
    assert float((a - b).norm() / b.norm()) <= 4e-3
    assert torch.all((a - b).abs() <= 2.0 ** -6 * b.abs() + 1e-3)


def _pack_reference(w, n, k, interleave):
    """The packed layout written out with numpy: P[h][c][l][e] =
    W[16h + l%16][32c + 8(l/16) + e], rows padded to a multiple of 32; gate
    and up interleaved by 16-row groups in blocks of 32 columns (gate rows
    32q.., up rows 32q.., gate rows 32q+16.., up rows 32q+16..)."""
    batch = w.shape[0]
    rows = w.reshape(batch, -1, k)
    if interleave:
        ip = -(-n // 32) * 32
        gate = np.zeros((batch, ip, k), w.dtype)
        up = np.zeros((batch, ip, k), w.dtype)
        gate[:, :n] = rows[:, :n]
        up[:, :n] = rows[:, n:]
        src = np.stack([gate.reshape(batch, ip // 32, 2, 16, k), up.reshape(batch, ip // 32, 2, 16, k)], axis=3)
        src = src.reshape(batch, 2 * ip, k)
    else:
        np_ = -(-n // 32) * 32
        src = np.zeros((batch, np_, k), w.dtype)
        src[:, :n] = rows
    kp = -(-k // 32) * 32
    full = np.zeros((batch, src.shape[1], kp), w.dtype)
    full[:, :, :k] = src
    g = full.shape[1] // 16
    # [b][g][16 rows][kc][4 quads][8] -> [b][g][kc][quad][16 rows][8]
    v = full.reshape(batch, g, 16, kp // 32, 4, 8).transpose(0, 1, 3, 4, 2, 5)
    return v.reshape(-1)


def _split3(w):
    """fp32 -> three bf16 terms (hi, mid, lo), each rounded to nearest even."""
    hi = W.f32_to_bf16_bits(w)
    r1 = (w.astype(np.float32) - W.bf16_bits_to_f32(hi)).astype(np.float32)
    mid = W.f32_to_bf16_bits(r1)
    r2 = (r1 - W.bf16_bits_to_f32(mid)).astype(np.float32)
    return hi, mid, W.f32_to_bf16_bits(r2)


@pytest.mark.parametrize("d,E", [(128, 16), (136, 40), (2048, 64), (72, 3)])
def test_pack_router_weights_layout(d, E):
    rng = np.random.default_rng(6)
    w = rng.standard_normal((E, d)).astype(np.float32)
    spec = S.LayerSpec(T=16, d=d, E=E, k=1, inter=32, shared_inter=0, n_bins=1, n_batch=1,
                       act_dtype=S.SMOES_BF16, weights_packed=True)
    got = S.pack_weights(spec, S.SMOES_WGATE, t(w)).cpu().numpy().view(np.uint16)
    ep, dp = -(-E // 16) * 16, -(-d // 32) * 32
    parts = []
    for term in _split3(w):
        full = np.zeros((ep, dp), np.uint16)
        full[:E, :d] = term
        # [g][16 rows][c][2 halves... 4 quads][8] -> [g][c][quad][row][8]
        parts.append(full.reshape(ep // 16, 16, dp // 32, 4, 8).transpose(0, 2, 3, 1, 4).reshape(-1))
    assert np.array_equal(got, np.concatenate(parts))
    # the three terms reproduce the weights to ~2^-24 relative
    hi, mid, lo = _split3(w)
    back = (W.bf16_bits_to_f32(hi).astype(np.float64) + W.bf16_bits_to_f32(mid) + W.bf16_bits_to_f32(lo))
    assert np.all(np.abs(back - w) <= 2.0 ** -23 * np.abs(w))


@pytest.mark.parametrize("d,E,inter,shared", [(128, 3, 96, 96), (136, 2, 48, 64), (64, 1, 32, 0)])
def test_pack_weights_layout(d, E, inter, shared):
    rng = np.random.default_rng(5)
    spec = S.LayerSpec(T=16, d=d, E=E, k=1, inter=inter, shared_inter=shared, n_bins=1, n_batch=1,
                       act_dtype=S.SMOES_BF16, weights_packed=True)
    mats = {"w13": (E, 2 * inter, d, inter, 1), "w2": (E, d, inter, d, 0)}
    if shared:
        mats.update(ws13=(1, 2 * shared, d, shared, 1), ws2=(1, d, shared, d, 0))
    for name, (b, r, c, n, il) in mats.items():
        w = rng.integers(1, 1 << 15, size=(b, r, c), dtype=np.uint16)
        got = S.pack_weights(spec, S.WEIGHT_NAMES[name], t(w if b > 1 or name in ("w13", "w2") else w[0]))
        torch.cuda.synchronize()
        exp = _pack_reference(w, n, c, il)
        assert np.array_equal(got.cpu().numpy().view(np.uint16), exp), name


def test_layer_tiny_fp32_full():
    inp = W.make_layer_inputs(W.workload("tiny-fp32"))
    spec, _, outs, ws = run_gpu_layer(inp, keep_workspace=True)
    ref = run_oracle_layer(inp)
    _check_layer(inp, spec, outs, ref, fp32=True)
    check_expert_rows(inp, spec, ws, outs, fp32=True)
    assert _check_mi(outs, ref, inp, strict=False) <= 1e-3


@pytest.mark.parametrize("name", ["deepseekmoe-vlm", "finegrained-vlm", "deepseekmoe-vlm-train", "large-skewed-vlm"])
def test_layer_full_size(name):
    """The full-size bf16 workloads in the launch configuration the benchmark
    times (caller-owned side streams: merged GEMM launches and, with shared
    experts, the combine in the shared down GEMM's epilogue); routing, scores
    and MI on every token, the output on a seeded sample."""
    cfg = W.workload(name)
    inp = W.make_layer_inputs(cfg)
    st = S.Streams()
    try:
        spec, _, outs, ws = run_gpu_layer(inp, keep_workspace=True, streams=st)
        torch.cuda.synchronize()
    finally:
        st.close()
    rows = np.sort(np.random.default_rng(cfg.seed).choice(cfg.T, size=192, replace=False))
    ref = run_oracle_layer(inp, rows=rows)
    _check_layer(inp, spec, outs, ref, rows=rows, routed_outs=_routed_run(inp))
    err = _check_mi(outs, ref, inp, strict=False)
    assert err <= 1e-3, err
    # every routed row's expert output, on the most and least loaded experts
    # (an empty one included where there is one) and two more, 64 rows each
    counts = np.diff(host(outs["expert_offsets"]).astype(np.int64))
    pick = {int(np.argmax(counts)), int(np.argmin(counts)), int(np.argmin(np.where(counts > 0, counts, 1 << 30)))}
    pick |= set(np.random.default_rng(cfg.seed + 1).choice(cfg.E, size=2, replace=False).tolist())
    check_expert_rows(inp, spec, ws, outs, experts=sorted(pick), max_rows=64)


def test_layer_deepseekmoe_full_rowmajor_weights():
    """The DeepSeekMoE-like workload through the row-major bf16 weight path."""
    cfg = W.workload("deepseekmoe-vlm")
    inp = W.make_layer_inputs(cfg)
    spec, _, outs = run_gpu_layer(inp, packed=False)
    rows = np.sort(np.random.default_rng(11).choice(cfg.T, size=128, replace=False))
    ref = run_oracle_layer(inp, rows=rows)
    _check_layer(inp, spec, outs, ref, rows=rows, routed_outs=_routed_run(inp, packed=False))


def test_layer_deepseekmoe_aligned_router_strict_mi():
    """Config-1 shapes with a modality-aligned router: MI ~1e-3, so the
    end-to-end MI and gradient meet the 1e-5 bound directly."""
    cfg = W.workload("deepseekmoe-vlm")
    inp = W.make_layer_inputs(cfg)
    wg = W.aligned_router(inp, 0.5)
    spec, _, outs = run_gpu_layer(inp, w_gate=wg)
    ref = run_oracle_layer(inp, w_gate=wg, rows=np.arange(64))
    err = _check_mi(outs, ref, inp, strict=True)
    assert err <= 1e-5, err


def test_layer_deterministic():
    cfg = W.small_config(seed=7, d=128, E=16, k=4, inter=96, n_shared=1, n_bins=4,
                         samples=((200, 100),), dtype=W.BF16)
    inp = W.make_layer_inputs(cfg)
    _, _, a = run_gpu_layer(inp)
    _, _, b = run_gpu_layer(inp)
    for key in ("probs", "topk_idx", "M", "mi_per_sample", "loss", "dlogits", "perm_token", "out"):
        assert torch.equal(a[key], b[key]), key


def test_stage_events():
    cfg = W.small_config(seed=8, d=128, E=16, k=4, inter=96, n_shared=1, n_bins=4,
                         samples=((200, 100),), dtype=W.BF16)
    inp = W.make_layer_inputs(cfg)
    ev = S.Events()
    run_gpu_layer(inp, events=ev)
    times = [ev.stage_ms(s) for s in range(S.N_STAGES)]
    assert all(x >= 0 for x in times)
    ev.close()


SIDE_STREAM_LAYERS = [
    dict(seed=9, d=256, E=16, k=4, inter=96, n_shared=1, n_bins=4, samples=((300, 100), (50, 60))),
    # ragged for the combine in the shared down GEMM's epilogue: k % 4 != 0,
    # d % 256 != 0 (a partial column tile), T % 128 != 0, statistics fixed
    dict(seed=19, d=136, E=12, k=6, inter=48, n_shared=2, n_bins=3, samples=((150, 47), (61, 33)),
         update_stats=False),
    # the maxima through the fused combine: 256 experts, top-16 (four slot groups per token), 64 bins
    dict(seed=23, d=256, E=256, k=16, inter=64, n_shared=1, n_bins=64, samples=((300, 100),)),
    # top-1: one routed slot per token beside the shared expert
    dict(seed=29, d=128, E=8, k=1, inter=32, n_shared=1, n_bins=2, samples=((100, 28), (40, 9))),
]


@pytest.mark.parametrize("layer", range(len(SIDE_STREAM_LAYERS)))
def test_side_streams_match_single_stream(layer):
    """With caller-owned side streams the modality score, the MI chain and the
    shared GEMMs run beside the routed path (and the combine runs in the shared
    down GEMM's epilogue); several calls in a row, with outputs read right
    after each, give the oracle's results and are bit-identical to the
    single-stream order (the joins make them complete)."""
    kw = dict(SIDE_STREAM_LAYERS[layer])
    kw.setdefault("update_stats", True)
    cfg = W.small_config(dtype=W.BF16, **kw)
    inp = W.make_layer_inputs(cfg)
    wg = W.aligned_router(inp, 0.5)  # well-conditioned MI
    ref = run_oracle_layer(inp, w_gate=wg)
    _, _, serial = run_gpu_layer(inp, w_gate=wg)
    st = S.Streams()
    try:
        for _ in range(3):
            spec, _, outs = run_gpu_layer(inp, w_gate=wg, streams=st)
            assert np.all(np.abs(host(outs["M"]) - ref["M"]) <= 1e-5 * np.abs(ref["M"]) + 1e-6)
            assert rel_err(host(outs["dlogits"]), ref["dlogits"]) <= 1e-5
            for k in ("M", "dlogits", "loss", "mi_per_sample", "out", "probs", "perm_token"):
                assert torch.equal(outs[k], serial[k]), k
    finally:
        st.close()
