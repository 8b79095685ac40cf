"""GPU parity of the layer backward (smoes_moe_backward after
smoes_moe_forward) against oracle.layer_backward: combine-weight and logit
gradients, the router weight and bias gradients, the routed and shared
expert weight gradients and the input gradient.

The routing must agree with the oracle's wherever the oracle's k-th and
(k+1)-th logits are more than 1e-4 apart. The upstream gradient is zero on
tokens whose gap is below 1e-3, so that no gradient depends on how a near
tie was broken (such a token then contributes only its auxiliary logit
gradient, which does not depend on the routing). Bars,
normwise relative error (the GPU path stores the recomputed pre-activations,
their gradients, H and each routed row's dX in bf16, relative rounding
2^-9 per stored element, and scales dout by the combine weight in bf16):
  dw, dz, dw_gate          <= 5e-3  (observed 1e-3 .. 2.7e-3: the forward's
                                     Y and H are bf16, rms rounding 1.1e-3 each)
  dbias                    <= 1e-2  (column sums of signed logit gradients
                                     cancel, observed up to 3.9e-3)
  dx                       <= 1e-2  (observed up to 3.1e-3)
  dw13, dw2, dws13, dws2   <= 1e-2  (observed up to 3.3e-3)
plus an elementwise bar of 6e-2 x max|ref| on every gradient (no single
element far off while the norm is fine).

fp32 layers and bf16 layers with row-major weights take the float32 FMA
backward (float32 intermediates). For fp32 layers every stored value is
float32 and each gradient entry is a float32 sum of at most a few thousand
products, so the normwise error is a small multiple of the unit roundoff
6e-8 amplified by the cancellation in the sum: bars 1e-5 (dbias, a column
sum of signed logit gradients, 1e-4) and an elementwise bar of 1e-4 x
max|ref|. Row-major bf16 layers keep the packed layers' bars (their forward
Y and H are still bf16)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle as O
from paper_2604_23996_amd import smoes as S
from paper_2604_23996_amd import workloads as W
from tests.gpu_util import DEV, check_topk, host, layer_spec, rel_err, run_gpu_layer, say, t

pytestmark = pytest.mark.gpu

BARS = {"dw": 5e-3, "dz": 5e-3, "dbias": 1e-2, "dw_gate": 5e-3, "dx": 1e-2,
        "dw13": 1e-2, "dw2": 1e-2, "dws13": 1e-2, "dws2": 1e-2}
ELEM = 6e-2
BARS_F32 = {"dw": 1e-5, "dz": 1e-5, "dbias": 1e-4, "dw_gate": 1e-5, "dx": 1e-5,
            "dw13": 1e-5, "dw2": 1e-5, "dws13": 1e-5, "dws2": 1e-5}
ELEM_F32 = 1e-4

LAYERS = [
    dict(d=128, E=16, k=4, inter=96, n_shared=1, n_bins=4, samples=((200, 100), (40, 60))),
    dict(d=256, E=12, k=3, inter=64, n_shared=0, n_bins=3, samples=((500, 200),)),
    # ragged packed groups: d % 32 == 8, inter % 32 == 16
    dict(d=136, E=10, k=3, inter=48, n_shared=2, n_bins=5, samples=((150, 70), (33, 17))),
    dict(d=512, E=64, k=6, inter=128, n_shared=2, n_bins=8, samples=((700, 300),), logit_bias=True),
    # several experts without tokens
    dict(d=64, E=32, k=2, inter=32, n_shared=1, n_bins=4, samples=((9, 5),)),
    # three tokens
    dict(d=64, E=4, k=2, inter=32, n_shared=0, n_bins=2, samples=((2, 1),)),
    # the maxima: 256 experts, top-16 (about 25 rows per expert)
    dict(d=128, E=256, k=16, inter=64, n_shared=1, n_bins=64, samples=((300, 100),)),
]


def _inputs(case, seed, dtype=W.BF16):
    cfg = W.small_config(seed=seed, dtype=dtype, **case)
    return _inputs_of(cfg, seed)


def _inputs_of(cfg, seed):
    inp = W.make_layer_inputs(cfg)
    rng = np.random.default_rng(seed + 7)
    g = rng.standard_normal((cfg.T, cfg.d)).astype(np.float32)
    dout = _mask_ties(inp, W.f32_to_bf16_bits(g) if cfg.dtype == W.BF16 else g)
    aux = (1e-3 * rng.standard_normal((cfg.T, cfg.E))).astype(np.float32)
    return cfg, inp, dout, aux


def _dout_f(cfg, dout):
    return W.bf16_bits_to_f32(dout) if cfg.dtype == W.BF16 else dout


def _mask_ties(inp, dout, gap=1e-3):
    """Zero the upstream gradient of the tokens whose oracle top-k gap is
    below `gap`."""
    z, _, _, _ = O.route(inp.x, inp.w_gate, inp.cfg.k, inp.logit_bias)
    dout = dout.copy()
    dout[O.topk_gap(z, inp.cfg.k) < gap] = 0
    return dout


def run_gpu_backward(inp, dout, aux, renorm, want_dw=True, save_preact=False, streams=None, packed=None):
    """Forward then backward on the device (the backward's router and shared
    experts on side streams when `streams` is given); bf16 layers use packed
    weights unless packed=False; returns (spec, outs, grads)."""
    cfg = inp.cfg
    if packed is None:
        packed = cfg.dtype == W.BF16
    packed_t = None
    if packed:
        rowmajor = {"w13": t(inp.w13), "w2": t(inp.w2), "ws13": t(inp.ws13), "ws2": t(inp.ws2)}
        spec_t = layer_spec(cfg, weights_packed=True)
        packed_t = S.pack_transposed_weights(spec_t, rowmajor)
        torch.cuda.synchronize()
    spec, dev_in, outs, ws = run_gpu_layer(inp, renorm_topk=renorm, keep_workspace=True, save_preact=save_preact,
                                           packed=packed)
    g = S.moe_backward(spec, dev_in, outs, ws, packed_t, t(dout), None if aux is None else t(aux), want_dw=want_dw,
                       streams=streams)
    torch.cuda.synchronize()
    return spec, outs, g


def _compare(g, ref, inp, outs, cfg, extra="", bars=BARS, elem=ELEM):
    z_ref, _, idx_ref, _ = O.route(inp.x, inp.w_gate, cfg.k, inp.logit_bias)
    check_topk(host(outs["topk_idx"]), idx_ref, z_ref, cfg.k)
    errs = {}
    for name, bar in bars.items():
        r = ref[name]
        if r is None:
            assert g.get(name) is None
            continue
        if g.get(name) is None:
            continue
        got = host(g[name]).reshape(r.shape)
        e = rel_err(got, r)
        errs[name] = e
        scale = np.abs(r).max()
        assert e <= bar, (name, e, extra)
        assert np.abs(got - r).max() <= elem * scale + 1e-30, (name, np.abs(got - r).max(), scale, extra)
    say("backward errors", extra, {k: f"{v:.2e}" for k, v in errs.items()})
    return errs


@pytest.mark.parametrize("layer", range(len(LAYERS)))
@pytest.mark.parametrize("renorm", [False, True])
@pytest.mark.parametrize("with_aux", [False, True])
def test_backward_small(layer, renorm, with_aux):
    cfg, inp, dout, aux = _inputs(LAYERS[layer], 300 + layer)
    if not with_aux:
        aux = None
    say("backward", layer, "renorm", renorm, "aux", with_aux, "T", cfg.T)
    spec, outs, g = run_gpu_backward(inp, dout, aux, renorm)
    _compare(g, _ref(inp, cfg, dout, aux, renorm), inp, outs, cfg, extra=f"layer {layer}")


@pytest.mark.parametrize("dtype", [W.BF16, W.F32])
def test_backward_experts_without_tokens_have_zero_gradient(dtype):
    cfg, inp, dout, aux = _inputs(LAYERS[4], 304, dtype=dtype)
    say("backward empty experts", dtype)
    spec, outs, g = run_gpu_backward(inp, dout, None, False)
    idx = host(outs["topk_idx"])
    used = np.zeros(cfg.E, bool)
    used[idx.ravel()] = True
    # experts with a token whose upstream gradient is not masked to zero
    live = np.zeros(cfg.E, bool)
    live[idx[np.abs(_dout_f(cfg, dout)).max(axis=1) > 0].ravel()] = True
    assert (~used).any() and live.any()
    dw13, dw2 = host(g["dw13"]), host(g["dw2"])
    assert np.all(dw13[~used] == 0.0) and np.all(dw2[~used] == 0.0)
    assert np.all(np.abs(dw13[live]).reshape(int(live.sum()), -1).max(axis=1) > 0)


@pytest.mark.parametrize("layer", [0, 1, 2, 4])
def test_backward_with_kept_preactivations_matches_recompute(layer):
    # the forward that keeps the gate / up pre-activations (save_preact) runs
    # the same MFMA sequence as the backward's recompute: identical bits
    cfg, inp, dout, aux = _inputs(LAYERS[layer], 300 + layer)
    say("backward kept pre-activations", layer)
    _, o1, g1 = run_gpu_backward(inp, dout, aux, True)
    _, o2, g2 = run_gpu_backward(inp, dout, aux, True, save_preact=True)
    assert torch.equal(o1["out"], o2["out"])
    for name in g1:
        if g1[name] is not None:
            assert torch.equal(g1[name], g2[name]), name


@pytest.mark.parametrize("layer", [0, 2, 3])
def test_backward_side_streams_match_single_stream(layer):
    # the router and shared-expert gradients on a side stream run the same
    # kernels in the same order within each chain: identical bits
    cfg, inp, dout, aux = _inputs(LAYERS[layer], 300 + layer)
    say("backward side streams", layer)
    streams = S.Streams()
    _, _, a = run_gpu_backward(inp, dout, aux, True, save_preact=True)
    _, _, b = run_gpu_backward(inp, dout, aux, True, save_preact=True, streams=streams)
    _, _, c = run_gpu_backward(inp, dout, aux, True, save_preact=False, streams=streams)
    for name in a:
        if a[name] is not None:
            assert torch.equal(a[name], b[name]), name
            assert torch.equal(a[name], c[name]), name
    streams.close()


def test_backward_is_reproducible():
    cfg, inp, dout, aux = _inputs(LAYERS[0], 300)
    say("backward reproducible")
    _, _, a = run_gpu_backward(inp, dout, aux, False)
    _, _, b = run_gpu_backward(inp, dout, aux, False)
    for name in a:
        if a[name] is not None:
            assert torch.equal(a[name], b[name]), name


def test_backward_without_dw_output():
    cfg, inp, dout, aux = _inputs(LAYERS[2], 302)
    say("backward no dw")
    _, _, g = run_gpu_backward(inp, dout, aux, True, want_dw=False)
    _, _, h = run_gpu_backward(inp, dout, aux, True, want_dw=True)
    for name in g:
        if g[name] is not None:
            assert torch.equal(g[name], h[name]), name


def _ref(inp, cfg, dout, aux, renorm):
    return O.layer_backward(inp.x, inp.w_gate, inp.logit_bias, cfg.k, inp.w13, inp.w2, inp.ws13, inp.ws2,
                            _dout_f(cfg, dout), aux, renorm_topk=renorm)


@pytest.mark.parametrize("layer", range(len(LAYERS)))
@pytest.mark.parametrize("renorm", [False, True])
def test_backward_fp32(layer, renorm):
    cfg, inp, dout, aux = _inputs(LAYERS[layer], 400 + layer, dtype=W.F32)
    say("backward fp32", layer, "renorm", renorm, "T", cfg.T)
    spec, outs, g = run_gpu_backward(inp, dout, aux, renorm)
    assert g["dw13"].dtype == torch.float32
    _compare(g, _ref(inp, cfg, dout, aux, renorm), inp, outs, cfg, extra=f"fp32 layer {layer}", bars=BARS_F32,
             elem=ELEM_F32)


def test_backward_tiny_fp32_workload():
    # the small fp32 workload (T=512, d=256, E=8, top-2, inter=512, no shared experts) in full
    cfg = W.workload("tiny-fp32")
    cfg, inp, dout, aux = _inputs_of(cfg, cfg.seed)
    say("backward tiny-fp32", cfg.T)
    for renorm in (False, True):
        spec, outs, g = run_gpu_backward(inp, dout, aux, renorm)
        _compare(g, _ref(inp, cfg, dout, aux, renorm), inp, outs, cfg, extra=f"tiny-fp32 renorm {renorm}",
                 bars=BARS_F32, elem=ELEM_F32)


@pytest.mark.parametrize("layer", range(len(LAYERS)))
def test_backward_rowmajor_bf16(layer):
    cfg, inp, dout, aux = _inputs(LAYERS[layer], 300 + layer)
    say("backward row-major bf16", layer, "T", cfg.T)
    spec, outs, g = run_gpu_backward(inp, dout, aux, True, packed=False)
    assert g["dw13"].dtype == torch.bfloat16
    _compare(g, _ref(inp, cfg, dout, aux, True), inp, outs, cfg, extra=f"row-major layer {layer}")


def test_backward_fp32_is_reproducible():
    cfg, inp, dout, aux = _inputs(LAYERS[0], 400, dtype=W.F32)
    say("backward fp32 reproducible")
    _, _, a = run_gpu_backward(inp, dout, aux, True)
    _, _, b = run_gpu_backward(inp, dout, aux, True)
    for name in a:
        if a[name] is not None:
            assert torch.equal(a[name], b[name]), name


def test_backward_rejects_missing_weights():
    # the float32 path reads the row-major w2 / ws2; the packed path needs the transposed packs
    cfg = W.small_config(d=64, E=8, k=2, inter=32, n_shared=0, samples=((8, 8),), dtype=W.F32, seed=5)
    spec = layer_spec(cfg)
    ws = torch.empty(1 << 20, dtype=torch.uint8, device=DEV)
    x = torch.zeros((cfg.T, cfg.d), dtype=torch.float32, device=DEV)
    with pytest.raises(S.SmoesError):
        S.moe_backward(spec, {"x": x}, {}, ws, None, x)
    cfg = W.small_config(d=64, E=8, k=2, inter=32, n_shared=0, samples=((8, 8),), dtype=W.BF16, seed=5)
    spec = layer_spec(cfg, weights_packed=True)
    with pytest.raises(S.SmoesError):
        S.moe_backward(spec, {"x": x}, {}, ws, None, x)


@pytest.mark.parametrize("name", ["deepseekmoe-vlm", W.BENCH_WORKLOAD])
def test_backward_bench_layer_sampled(name):
    """The full-size layers in the launch configuration of the timed training
    step: the 4096-token DeepSeekMoE-like layer (d 2048, 64 experts, top-6,
    inter 1408, two shared experts) and the benchmark's 16384-token layer
    (d 4096, 160 experts, top-6, inter 1536, two shared experts, logit bias).
    The oracle computes dw, dz and dx of 128 sampled tokens (the per-token
    gradients depend on that token alone), the weight gradients of three
    routed experts over their rows and the shared experts' weight gradients
    over all tokens (at d 4096 on 64 sampled inner columns: the SwiGLU is
    separable over its inner columns, so the gradient rows and columns of a
    column subset are those of the sub-network of those columns); the router
    weight and bias gradients are checked as dz^T x and the column sums of
    dz in float64."""
    cfg = W.workload(name)
    inp = W.make_layer_inputs(cfg)
    rng = np.random.default_rng(77)
    dout = _mask_ties(inp, W.f32_to_bf16_bits(rng.standard_normal((cfg.T, cfg.d)).astype(np.float32)))
    say("backward bench layer")
    spec, outs, g = run_gpu_backward(inp, dout, None, False)
    X = O.widen(inp.x)
    dO = W.bf16_bits_to_f32(dout).astype(np.float64)
    z, _, idx, w = O.route(inp.x, inp.w_gate, cfg.k, inp.logit_bias)
    check_topk(host(outs["topk_idx"]), idx, z, cfg.k)
    # per-token gradients of sampled tokens
    sample = np.sort(rng.choice(cfg.T, size=128, replace=False))
    ref = O.layer_backward(inp.x[sample], inp.w_gate, inp.logit_bias, cfg.k, inp.w13, inp.w2, inp.ws13, inp.ws2,
                           dO[sample], None)
    for name in ("dw", "dz", "dx"):
        got = host(g[name])[sample]
        assert rel_err(got, ref[name]) <= BARS[name], (name, rel_err(got, ref[name]))
        assert np.abs(got - ref[name]).max() <= ELEM * np.abs(ref[name]).max()
    # routed experts over all their rows
    _, offsets, perm_token, inv = O.permutation(idx, cfg.E)
    for e in (0, cfg.E // 2 - 3, cfg.E - 1):
        a, b = offsets[e], offsets[e + 1]
        toks = perm_token[a:b]
        slot = np.argmax(inv[toks] == np.arange(a, b)[:, None], axis=1)
        dY = w[toks, slot][:, None] * dO[toks]
        _, dw13, dw2 = O.swiglu_backward(X[toks], inp.w13[e], inp.w2[e], dY)
        for name, got, r in (("dw13", host(g["dw13"][e]), dw13), ("dw2", host(g["dw2"][e]), dw2)):
            assert rel_err(got, r) <= BARS[name], (name, e, rel_err(got, r))
            assert np.abs(got - r).max() <= ELEM * np.abs(r).max(), (name, e)
    # shared experts over all tokens
    SI = cfg.shared_inter
    cols = np.arange(SI) if cfg.d <= 2048 else np.sort(rng.choice(SI, size=64, replace=False))
    _, dws13, dws2 = O.swiglu_backward(X, inp.ws13[np.concatenate([cols, SI + cols])], inp.ws2[:, cols], dO)
    got13 = host(g["dws13"])[np.concatenate([cols, SI + cols])]
    got2 = host(g["dws2"])[:, cols]
    for wname, got, r in (("dws13", got13, dws13), ("dws2", got2, dws2)):
        assert rel_err(got, r) <= BARS[wname], (wname, rel_err(got, r))
        assert np.abs(got - r).max() <= ELEM * np.abs(r).max(), wname
    # router: dW_gate = dz^T x and dbias = column sums of dz, float32 chunked sums
    dz = host(g["dz"]).astype(np.float64)
    assert rel_err(host(g["dw_gate"]), dz.T @ X) <= 1e-5
    assert rel_err(host(g["dbias"]), dz.sum(axis=0)) <= 1e-5
