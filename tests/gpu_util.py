"""Shared helpers of the GPU parity tests: moving the seeded inputs to the
device, running the oracle on the same arrays, and the tolerance checks."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle as O
from paper_2604_23996_amd import smoes as S
from paper_2604_23996_amd import workloads as W

DEV = "cuda:0"


def say(*a):
    """Name the case before a GPU step (flushed, so a crash still shows it)."""
    print("[gpu]", *a, file=sys.stderr, flush=True)


def t(a: np.ndarray, dtype=None) -> torch.Tensor:
    """numpy -> device tensor; uint16 arrays are bf16 bit patterns."""
    if a is None:
        return None
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(DEV).view(torch.bfloat16)
    x = torch.from_numpy(a)
    if dtype is not None:
        x = x.to(dtype)
    return x.to(DEV)


def host(x: torch.Tensor) -> np.ndarray:
    if x.dtype == torch.bfloat16:
        return W.bf16_bits_to_f32(x.view(torch.int16).cpu().numpy().view(np.uint16)).astype(np.float64)
    return x.cpu().numpy()


def rel_err(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.linalg.norm(b.ravel())
    return np.linalg.norm((a - b).ravel()) / (den if den > 0 else 1.0)


def gate_rtol(x, w_gate, bias=None):
    """Per-token relative tolerance of the gate values g = softmax(z). The
    logits are fp32-faithful: |z_gpu - z| <= 4e-7 sum_d |x_d w_ed| (+ |b_e|).
    The softmax turns an absolute logit error into a relative gate error,
    |dg_e / g_e| <= |dz_e| + |d logsumexp| <= 2 max_e |dz_e|, so the bar is
    8e-7 times the token's largest such sum, and never below 1e-5."""
    scale = np.abs(O.widen(x)) @ np.abs(np.asarray(w_gate, dtype=np.float64)).T
    if bias is not None:
        scale = scale + np.abs(np.asarray(bias, dtype=np.float64))
    return np.maximum(1e-5, 8e-7 * scale.max(axis=1))[:, None]


def check_topk(idx_gpu, idx_ref, z_ref, k, gap_tol=1e-4):
    """Top-k against the oracle. Wherever the oracle's k-th vs (k+1)-th logit
    gap exceeds gap_tol the chosen set is bit-exact, and the order is the
    oracle's except among chosen experts whose logits lie within gap_tol of
    each other (the s-th chosen logit equals the oracle's s-th within gap_tol):
    the logits are fp32-faithful, so keys closer than that may come in either
    order. Elsewhere every chosen expert must be a valid choice (its logit
    within gap_tol of the k-th largest). Returns the mask of clear tokens."""
    gap = O.topk_gap(z_ref, k)
    clear = gap > gap_tol
    same_set = np.all(np.sort(idx_gpu[clear], axis=1) == np.sort(idx_ref[clear], axis=1), axis=1)
    assert same_set.all(), f"top-k set mismatch on {np.sum(~same_set)} clear tokens"
    zg = np.take_along_axis(z_ref[clear], idx_gpu[clear].astype(np.int64), axis=1)
    zr = np.take_along_axis(z_ref[clear], idx_ref[clear].astype(np.int64), axis=1)
    assert np.all(np.abs(zg - zr) <= gap_tol), "top-k order differs beyond near-equal logits"
    assert np.all(zg[:, :-1] >= zg[:, 1:] - gap_tol), "top-k not in descending logit order"
    if (~clear).any():
        zs = -np.sort(-z_ref[~clear], axis=1)
        kth = zs[:, k - 1]
        chosen = np.take_along_axis(z_ref[~clear], idx_gpu[~clear].astype(np.int64), axis=1)
        assert np.all(chosen >= kth[:, None] - gap_tol)
        for row in idx_gpu[~clear]:
            assert len(set(row.tolist())) == k
    return clear


def gauss_state_dev(d):
    return (torch.zeros(2, dtype=torch.float32, device=DEV),
            torch.zeros((2, d), dtype=torch.float32, device=DEV),
            torch.zeros((2, d), dtype=torch.float32, device=DEV))


def layer_spec(cfg: W.LayerConfig, T=None, **kw) -> S.LayerSpec:
    return S.LayerSpec(T=cfg.T if T is None else T, d=cfg.d, E=cfg.E, k=cfg.k, inter=cfg.inter,
                       shared_inter=cfg.shared_inter, n_bins=cfg.n_bins, n_batch=cfg.n_batch,
                       act_dtype=S.SMOES_BF16 if cfg.dtype == W.BF16 else S.SMOES_F32,
                       tau=cfg.tau, beta=cfg.beta, **kw)


def pack_layer_weights(spec: S.LayerSpec, dev_in) -> None:
    """Replace the row-major bf16 expert weights in dev_in by their packed
    form (smoes_pack_weights); spec must have weights_packed set."""
    S.pack_layer_inputs(spec, dev_in)
    torch.cuda.synchronize()


def run_gpu_layer(inp: W.LayerInputs, w_gate=None, update_stats=None, events=None, packed=None,
                  streams=None, renorm_topk=False, keep_workspace=False, save_preact=False,
                  zero_shared_down=False, check_inputs=False):
    """The full layer through smoes_moe_forward. For layers that do not update
    their statistics in the call, the Gaussian state is first estimated from
    the batch by smoes_modality_score(update=1) from the zero state. bf16
    layers use packed expert weights unless packed=False. zero_shared_down
    replaces the shared experts' down projection by zeros: their output is
    then exactly 0 and `out` holds the routed part alone."""
    cfg = inp.cfg
    upd = cfg.update_stats if update_stats is None else update_stats
    if packed is None:
        packed = cfg.dtype == W.BF16
    spec = layer_spec(cfg, update_stats=upd, weights_packed=packed, renorm_topk=renorm_topk,
                      save_preact=save_preact, check_inputs=check_inputs)
    ws2 = inp.ws2
    if zero_shared_down and ws2 is not None:
        ws2 = np.zeros_like(ws2)
    dev_in = {
        "x": t(inp.x), "modality_id": t(inp.modality_id), "sample_offsets": t(inp.sample_offsets),
        "w_gate": t(inp.w_gate if w_gate is None else w_gate), "logit_bias": t(inp.logit_bias),
        "expert_to_bin": t(inp.expert_to_bin), "w13": t(inp.w13), "w2": t(inp.w2),
        "ws13": t(inp.ws13), "ws2": t(ws2),
    }
    if packed:
        pack_layer_weights(spec, dev_in)
    n, smu, ssig = gauss_state_dev(cfg.d)
    if not upd:
        S.modality_score(dev_in["x"], n, smu, ssig, dev_in["modality_id"], update=True, beta=cfg.beta,
                         tau=cfg.tau)
    dev_in.update(gauss_n=n, gauss_smu=smu, gauss_ssig=ssig)
    act = torch.bfloat16 if cfg.dtype == W.BF16 else torch.float32
    outs = S.alloc_outputs(spec, DEV, act)
    ws = torch.empty(S.workspace_bytes(spec), dtype=torch.uint8, device=DEV)
    S.moe_forward(spec, dev_in, outs, ws, events=events, streams=streams)
    torch.cuda.synchronize()
    if keep_workspace:
        return spec, dev_in, outs, ws
    return spec, dev_in, outs


def run_oracle_layer(inp: W.LayerInputs, w_gate=None, rows=None, update_stats=None):
    cfg = inp.cfg
    upd = cfg.update_stats if update_stats is None else update_stats
    st = O.GaussState.zeros(cfg.d)
    if not upd:
        st = O.gauss_update(st, inp.x, inp.modality_id, cfg.beta)
    return O.layer_forward(inp.x, inp.modality_id, inp.sample_offsets,
                           inp.w_gate if w_gate is None else w_gate, inp.logit_bias,
                           inp.expert_to_bin, cfg.n_bins, cfg.k, inp.w13, inp.w2, inp.ws13, inp.ws2,
                           st, update_stats=upd, beta=cfg.beta, tau=cfg.tau, rows=rows)


def routed_rows(spec: S.LayerSpec, ws: torch.Tensor) -> np.ndarray:
    """Y_r [T*k, d] of the last forward on `ws` (smoes_workspace_buffer), as
    float64; rows in the expert-contiguous order of perm_token."""
    buf = S.workspace_buffer(spec, ws, S.SMOES_BUF_Y_ROUTED)
    R = spec.T * spec.k
    if spec.act_dtype == S.SMOES_BF16:
        y = buf.view(torch.int16).reshape(R, spec.d).cpu().numpy().view(np.uint16)
        return W.bf16_bits_to_f32(y).astype(np.float64)
    return buf.view(torch.float32).reshape(R, spec.d).cpu().numpy().astype(np.float64)


def check_expert_rows(inp: W.LayerInputs, spec: S.LayerSpec, ws: torch.Tensor, outs, experts=None,
                      max_rows=None, fp32=False):
    """Every routed row's expert output Y_r[r] = FFN_e(x[perm_token[r]]) of the
    GPU's own permutation against the oracle's SwiGLU of the same rows, expert
    by expert: normwise relative error <= 2e-2 (bf16) / 1e-5 (fp32) and
    elementwise |gpu - ref| <= 1e-2 + 2e-2 |ref|. Returns the worst normwise error."""
    cfg = inp.cfg
    Y = routed_rows(spec, ws)
    off = host(outs["expert_offsets"]).astype(np.int64)
    perm = host(outs["perm_token"]).astype(np.int64)
    worst = 0.0
    for e in (range(cfg.E) if experts is None else experts):
        a, b = off[e], off[e + 1]
        if max_rows is not None:
            b = min(b, a + max_rows)
        if b <= a:
            continue
        ref = O.swiglu(inp.x[perm[a:b]], inp.w13[e], inp.w2[e])
        got = Y[a:b]
        err = rel_err(got, ref)
        assert err <= (1e-5 if fp32 else 2e-2), (e, err)
        assert np.all(np.abs(got - ref) <= 1e-2 + 2e-2 * np.abs(ref)), (e, np.max(np.abs(got - ref)))
        worst = max(worst, err)
    return worst
