"""GPU parity of the attention-accumulated modality score (Sec. 3.2.1,
Eq. 2-4) against the oracle: the one-hot start, the causal per-sample
attention with the scores carried as two extra value channels, and the
head-averaged norm-weighted update.

Bars: the per-head aggregated scores within 2e-5 absolute (float32
accumulation of float32 probabilities from bf16 x bf16 logits); the attention
output within 1e-2 + 2e-2 |ref| elementwise and 1e-2 normwise (the
probabilities enter the value product as bf16, as in any bf16 attention);
the updated scores within 1e-5; the one-hot start bit for bit."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle as O
from paper_2604_23996_amd import smoes as S
from paper_2604_23996_amd import workloads as W
from tests.gpu_util import host, rel_err, say, t

pytestmark = pytest.mark.gpu

M_TOL = 2e-5


def _run_attention(a: W.AttnInputs, scale=0.0):
    o, mh = S.attention_scores(t(a.q), t(a.k), t(a.v), t(a.sample_offsets), t(a.m_in), scale=scale)
    torch.cuda.synchronize()
    return host(o), host(mh)


def _check_attention(a: W.AttnInputs, o, mh, scale=None, rows=None):
    ref_o, ref_a = O.attention_heads(a.q, a.k, a.v, a.sample_offsets, a.m_in, scale=scale)
    if rows is not None:
        ref_o, ref_a, o, mh = ref_o[rows], ref_a[rows], o[rows], mh[rows]
    err_m = np.abs(mh - ref_a).max() if mh.size else 0.0
    assert err_m <= M_TOL, err_m
    assert np.all(np.abs(o - ref_o) <= 1e-2 + 2e-2 * np.abs(ref_o)), np.abs(o - ref_o).max()
    assert rel_err(o, ref_o) <= 1e-2, rel_err(o, ref_o)


@pytest.mark.parametrize("dh", [128, 64])
@pytest.mark.parametrize("H,Hkv", [(4, 4), (4, 2), (8, 1)])
def test_attention_ragged_samples(dh, H, Hkv):
    # sample lengths that are not multiples of the 128-row query blocks or
    # 64-key blocks, an empty sample, a one-token sample: query blocks
    # straddle sample boundaries
    samples = ((30, 20), (0, 0), (70, 67), (1, 0), (150, 41))
    a = W.make_attention_inputs(samples, 64, H, Hkv, dh, seed=dh + H + Hkv)
    say("attention ragged", dh, H, Hkv, a.T)
    o, mh = _run_attention(a)
    _check_attention(a, o, mh)


def test_attention_explicit_scale_and_flat_logits():
    samples = ((100, 60),)
    a = W.make_attention_inputs(samples, 64, 2, 2, 128, seed=5, logit_std=0.05)
    say("attention scale", a.T)
    o, mh = _run_attention(a, scale=0.3)
    _check_attention(a, o, mh, scale=0.3)


def test_attention_sharp_logits():
    # peaked attention: large logits exercise the running-maximum rescaling
    a = W.make_attention_inputs(((200, 100), (64, 64)), 64, 4, 4, 128, seed=6, logit_std=12.0)
    say("attention sharp", a.T)
    o, mh = _run_attention(a)
    _check_attention(a, o, mh)


def test_attention_single_token_and_empty():
    a = W.make_attention_inputs(((1, 0),), 64, 2, 1, 64, seed=7)
    say("attention T=1")
    o, mh = _run_attention(a)
    _check_attention(a, o, mh)
    # the one token attends only to itself
    assert np.allclose(mh[0], np.repeat(a.m_in[:1], 2, axis=0), atol=1e-7)
    e = W.make_attention_inputs(((0, 0),), 64, 2, 1, 64, seed=7)
    say("attention T=0")
    o, mh = S.attention_scores(t(e.q), t(e.k), t(e.v), t(e.sample_offsets), t(e.m_in))
    torch.cuda.synchronize()
    assert o.numel() == 0 and mh.numel() == 0


def test_attention_bench_shape_sampled_samples():
    # the bench workload's shape (16 samples x 1024 tokens, hidden 4096 as 32
    # heads of 128); samples are independent (pinned in the oracle), so the
    # oracle runs on the first and the last sample alone
    cfg = W.workload(W.BENCH_WORKLOAD)
    a = W.make_attention_inputs(cfg.samples, cfg.d, cfg.d // 128, cfg.d // 128, 128, seed=cfg.seed)
    say("attention bench shape", a.T)
    o, mh = _run_attention(a)
    for s in (0, len(cfg.samples) - 1):
        lo, hi = int(a.sample_offsets[s]), int(a.sample_offsets[s + 1])
        sub = W.AttnInputs(a.samples[s:s + 1], a.q[lo:hi], a.k[lo:hi], a.v[lo:hi], a.x[lo:hi], a.x_attn[lo:hi],
                           a.m_in[lo:hi], a.modality_id[lo:hi], np.array([0, hi - lo], np.int32))
        _check_attention(sub, o[lo:hi], mh[lo:hi])


def test_attention_is_reproducible():
    a = W.make_attention_inputs(((300, 200),), 64, 4, 2, 128, seed=8)
    say("attention reproducible", a.T)
    o1, m1 = _run_attention(a)
    o2, m2 = _run_attention(a)
    assert np.array_equal(o1, o2) and np.array_equal(m1, m2)


def test_attn_score_init_one_hot():
    mid = np.array([0, 1, 1, 0, 2, 1], np.uint8)
    say("attn init")
    M = host(S.attn_score_init(t(mid)))
    assert np.array_equal(M, O.attn_score_init(mid).astype(np.float32))
    assert M[4].tolist() == [0.0, 0.0]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_attn_score_update(dtype):
    rng = np.random.default_rng(9)
    T, d, H = 333, 264, 6
    x = rng.standard_normal((T, d)).astype(np.float32)
    xa = (rng.standard_normal((T, d)) * 0.3).astype(np.float32)
    x[5] = 0.0
    xa[5] = 0.0  # both norms 0: the score is kept
    xa[7] = 0.0  # no attention output: unchanged
    x[9] = 0.0  # no residual: the aggregate
    if dtype == "bf16":
        x, xa = W.f32_to_bf16_bits(x), W.f32_to_bf16_bits(xa)
    mh = rng.uniform(0, 1, (T, H, 2)).astype(np.float32)
    m_in = W.random_soft_scores(rng, T)
    say("attn update", dtype)
    out = host(S.attn_score_update(t(x), t(xa), t(mh), t(m_in)))
    ref = O.attn_score_update(x, xa, m_in, O.attn_aggregate(mh))
    assert np.abs(out - ref).max() <= 1e-5
    assert np.array_equal(out[5], m_in[5])
    # in place: m_out aliases m_in
    m_dev = t(m_in)
    S.attn_score_update(t(x), t(xa), t(mh), m_dev, out=m_dev)
    torch.cuda.synchronize()
    assert np.array_equal(host(m_dev), out)


def test_attention_score_layer_chain():
    # Eq. 2 -> Eq. 3 -> Eq. 4 for one layer, end to end on the device
    a = W.make_attention_inputs(((120, 80), (90, 30)), 128, 4, 2, 64, seed=10)
    say("attn chain", a.T)
    m0 = S.attn_score_init(t(a.modality_id))
    o, mh = S.attention_scores(t(a.q), t(a.k), t(a.v), t(a.sample_offsets), m0)
    m1 = S.attn_score_update(t(a.x), t(a.x_attn), mh, m0)
    torch.cuda.synchronize()
    M0 = O.attn_score_init(a.modality_id)
    _, A = O.attention_heads(a.q, a.k, a.v, a.sample_offsets, M0)
    M1 = O.attn_score_update(a.x, a.x_attn, M0, O.attn_aggregate(A))
    assert np.abs(host(m1) - M1).max() <= 2e-5
    assert np.allclose(host(m1).sum(axis=1), 1.0, atol=1e-5)
