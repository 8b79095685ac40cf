"""CPU oracle of one SMoES-routed MoE layer (test infrastructure only).

It is the reference the GPU path is checked against, not part of it: only the
tests, the smoke entry and the CPU-baseline leg of the benchmark may import it. It shares no code with the
HIP path. Everything is plain NumPy in float64 on the exact stored input values
(bf16 inputs are widened exactly), written step by step in the order and
notation of the paper, "Soft Modality-Guided Expert Specialization in
MoE-VLMs" (SMoES):

  * Sec. 3.1   router gating g = softmax(W_gate x) and top-k selection
  * Sec. 3.2.2 EMA variant of Welford's update (Eq. 5-7), per-modality
               log-likelihood (Eq. 8), temperature softmax score (Eq. 9)
  * Sec. 3.3   expert binning (bins of N_B = N_e / N_bins experts)
  * Sec. 3.4   per-sample bin-by-modality gating mass (Eq. 12), joint (Eq. 13),
               mutual information (Eq. 14), loss (Eq. 15, one layer)
  * derived    gradient of the MI loss with respect to the router logits
               (the paper does not print it; the closed form below follows from
               Eq. 12-15 by the chain rule and is pinned by finite differences)
  * MoE layer  expert-contiguous permutation, SwiGLU experts, shared experts,
               weighted combine (the backbones of the supplementary backbone
               table: DeepSeekMoE with 2 shared experts, gated-SiLU FFNs)
  * Sec. 3.3 / 3.5 / 4.1  momentum-adaptive binning (Eq. 10-11), bin-level
               load balance (Eq. 16) and its logit gradient, MSI (Eq. 18-19)
  * Sec. 3.2.1 attention-accumulated score: one-hot start (Eq. 2), head-averaged
               attention aggregation (Eq. 3), norm-weighted residual mix (Eq. 4)
  * Suppl. GMM estimator: a K-component diagonal mixture per modality in place
               of the single Gaussian of Sec. 3.2.2 (mixture log-likelihood,
               Eq. 9 score, stepwise-EM update built on Eq. 5-7)
  * backward   the layer's gradients for the training step of the
               supplementary cost table: experts (dgrad and wgrad), combine
               weights, softmax router with the auxiliary logit gradients added

Readings where the paper is silent (each also listed in the design notes):
  R1  logarithms are natural (MI in nats);
  R2  g inside the MI is the full softmax over all experts, not the top-k mask;
  R3  combine weights are the raw top-k gate values unless renorm is asked for;
  R4  top-k is decided on float32 logits, ordered by descending logit, ties to
      the lower expert index;
  R5  a per-expert logit bias, when given, is added before softmax and top-k;
  R6  shared experts have weight 1 and are ungated; S shared experts of inner
      size I are one SwiGLU of inner size S*I;
  R7  SwiGLU is down(silu(gate x) * up x), silu(a) = a / (1 + exp(-a));
  R8  samples are contiguous token ranges given by offsets;
  R9  the modality score is treated as a constant in the MI gradient;
  R10 statistics are updated with the current batch before scoring it;
  R11 the 2*pi constant of the log-likelihood is dropped (it cancels in Eq. 9),
      the variance is floored at var_floor, and a modality with N = 0 has
      mu = 0, sigma^2 = 1;
  R12 an MI term with P(m, B_k) = 0 contributes 0, and a modality with zero
      total score mass in a sample has S-bar = 0 for every bin;
  R13 column 0 of the modality score is vision, column 1 is text.
  R14 bin-level load balance (Eq. 16, one layer): the "tokens in bin B_k" are
      the tokens routed to bin k (at least one of their top-k experts lies in
      B_k), T_k of them; f_e = (tokens whose top-k holds e) / T_k and P_e is
      the mean gate value of e over those tokens; a bin no token reaches adds
      0. The top-k counts are constants for the gradient, as in the standard
      load-balance loss.
  R15 momentum-adaptive binning (Eq. 10-11): C_{m,e} counts the tokens of
      hard label m whose top-k holds e; the EMA is kept in float64 as
      beta * C_bar + (1 - beta) * C with both products rounded before the
      sum; f_spec = C_bar_text / (C_bar_text + C_bar_vision), 1/2 when both
      are 0; experts are sorted by ascending f_spec, ties to the lower expert
      index, and cut into consecutive bins: bin(e) = rank(e) // N_B.
  R16 MSI (Eq. 18-19) for one layer from the batch counts; a modality with
      no tokens has all normalised shares 0, and an expert that no token of
      either modality reaches counts as unspecialised (C_tilde_text = 1/2).
  R17 Attn in Eq. 3 is the decoder's causal softmax attention inside each
      sample (a sample never attends to another), with logits q.k * scale
      (scale 1/sqrt(d_head) by default), averaged over the query heads; with
      grouped KV heads, query head h reads KV head h // (H / H_kv). Both
      score columns are aggregated.
  R18 In Eq. 4, x_attn is the attention sublayer's output that is added to
      the residual stream (after its output projection) and x is that
      sublayer's residual input; norms are Euclidean over D; a token with
      both norms 0 keeps its score.
  R19 GMM estimator (the supplementary GMM ablation gives only K in {2, 4}):
      each modality is a mixture of K diagonal Gaussians with weights
      pi_mc = N_mc / sum_c' N_mc' (uniform when all are 0), mu and sigma^2 as
      in Sec. 3.2.2 per component (R11 per component); LL_m is the log of the
      mixture density without the 2 pi constant, and the score is Eq. 9 with
      it. The update is stepwise EM: responsibilities of the token's own
      modality under the parameters before the update, then Eq. 5-7 per
      component with |T_m|, mu_T and the centred sum of squares replaced by
      their responsibility-weighted forms. K = 1 is exactly Sec. 3.2.2.
      Components must be seeded apart by the caller (identical components
      stay identical under EM).
  R20 Layer backward: the top-k choice is piecewise constant (no gradient);
      the gradient reaches the router through the combine weights (the gate
      values at the chosen experts, or their renormalised form) and the full
      softmax; logit gradients of auxiliary losses (MI, bin balance) are
      added to the router's logit gradient; the modality scores are constants
      (R9). Given dL/d out, the outputs are dx, the router weight (and bias)
      gradient, the total logit gradient, the combine-weight gradient and the
      routed and shared expert weight gradients.

Parity pins live in tests/test_oracle_pins.py; no part of this file is
"parity unpinned" except the conventions R3-R5, R8, R11, R12, R14-R16 above,
which fix choices the paper does not make (both sides implement the same
stated choice; the formulas that follow each choice are pinned).
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Dict, Optional, Tuple

import numpy as np

VISION, TEXT = 0, 1


def widen(a) -> np.ndarray:
    """Exact float64 view of a stored array (uint16 = bf16 bit patterns)."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


# ----------------------------------------------------------------------------
# Sec. 3.1: router
# ----------------------------------------------------------------------------

def router_logits(x, w_gate, logit_bias=None) -> np.ndarray:
    """z_j = W_gate x_j (+ b): the pre-softmax router scores, float64."""
    z = widen(x) @ widen(w_gate).T
    if logit_bias is not None:
        z = z + widen(logit_bias)[None, :]
    return z


def softmax_rows(z) -> np.ndarray:
    """g_je = exp(z_je) / sum_e' exp(z_je') over all N_e experts (Sec. 3.1)."""
    z = np.asarray(z, dtype=np.float64)
    e = np.exp(z - z.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True)


def topk_select(z, k: int) -> np.ndarray:
    """Indices of the k highest scores per token (Sec. 3.1), decided on the
    float32 value of the logits (R4); descending order, ties to lower index."""
    z32 = np.asarray(z, dtype=np.float64).astype(np.float32)
    order = np.argsort(-z32, axis=1, kind="stable")
    return order[:, :k].astype(np.int32)


def topk_gap(z, k: int) -> np.ndarray:
    """z_(k) - z_(k+1) per token (inf when k = E): tokens with a small gap may
    legitimately pick a different k-th expert under rounding."""
    z = np.asarray(z, dtype=np.float64)
    if k >= z.shape[1]:
        return np.full(z.shape[0], np.inf)
    s = -np.sort(-z, axis=1)
    return s[:, k - 1] - s[:, k]


def route(x, w_gate, k: int, logit_bias=None, renorm_topk: bool = False):
    """Router step: logits, full softmax, top-k indices and combine weights."""
    z = router_logits(x, w_gate, logit_bias)
    g = softmax_rows(z)
    idx = topk_select(z, k)
    w = np.take_along_axis(g, idx.astype(np.int64), axis=1)
    if renorm_topk:
        w = w / w.sum(axis=1, keepdims=True)
    return z, g, idx, w


# ----------------------------------------------------------------------------
# Sec. 3.2.2: Gaussian-statistics modality score
# ----------------------------------------------------------------------------

@dataclass
class GaussState:
    """Per-layer EMA-Welford state for the two modalities: N_m, S_mu,m, S_sigma2,m."""

    n: np.ndarray  # [2]
    s_mu: np.ndarray  # [2, D]
    s_sig: np.ndarray  # [2, D]

    @staticmethod
    def zeros(d: int) -> "GaussState":
        return GaussState(np.zeros(2), np.zeros((2, d)), np.zeros((2, d)))

    @staticmethod
    def of(n, s_mu, s_sig) -> "GaussState":
        return GaussState(widen(n).copy(), widen(s_mu).copy(), widen(s_sig).copy())


def gauss_update(state: GaussState, x, modality_id, beta: float) -> GaussState:
    """One EMA-Welford step (Eq. 5-7) for each modality m:

        N_t      = beta N_{t-1} + |T_m|
        S_mu,t   = beta S_mu,t-1 + |T_m| mu_T
        S_sig,t  = beta S_sig,t-1 + sum_{x in T_m} (x - mu_T)^2
                   + (mu_T - S_mu,t-1 / N_{t-1})^2 beta N_{t-1} |T_m| / (beta N_{t-1} + |T_m|)

    with T_m the modality-m tokens of the batch and mu_T their mean. The last
    term is taken as 0 when N_{t-1} = 0 or |T_m| = 0 (its factor vanishes)."""
    X = widen(x)
    mid = np.asarray(modality_id)
    n_new = state.n.copy()
    s_mu_new = state.s_mu.copy()
    s_sig_new = state.s_sig.copy()
    for m in (VISION, TEXT):
        sel = X[mid == m]
        cnt = sel.shape[0]
        n_prev = state.n[m]
        if cnt > 0:
            mu_T = sel.mean(axis=0)
            sq = ((sel - mu_T) ** 2).sum(axis=0)
        else:
            mu_T = np.zeros(X.shape[1])
            sq = np.zeros(X.shape[1])
        if n_prev > 0 and cnt > 0:
            prev_mean = state.s_mu[m] / n_prev
            cross = (mu_T - prev_mean) ** 2 * (beta * n_prev * cnt) / (beta * n_prev + cnt)
        else:
            cross = np.zeros(X.shape[1])
        n_new[m] = beta * n_prev + cnt
        s_mu_new[m] = beta * state.s_mu[m] + cnt * mu_T
        s_sig_new[m] = beta * state.s_sig[m] + sq + cross
    return GaussState(n_new, s_mu_new, s_sig_new)


def gauss_params(state: GaussState, var_floor: float) -> Tuple[np.ndarray, np.ndarray]:
    """mu_m = S_mu / N and sigma^2_m = S_sigma2 / N (Sec. 3.2.2), floored (R11)."""
    d = state.s_mu.shape[1]
    mu = np.zeros((2, d))
    var = np.ones((2, d))
    for m in (VISION, TEXT):
        if state.n[m] > 0:
            mu[m] = state.s_mu[m] / state.n[m]
            var[m] = np.maximum(state.s_sig[m] / state.n[m], var_floor)
    return mu, var


def log_likelihood(x, mu, var) -> np.ndarray:
    """LL_jm = -1/2 sum_d (log sigma^2_md + (x_jd - mu_md)^2 / sigma^2_md)  (Eq. 8)."""
    X = widen(x)
    ll = np.empty((X.shape[0], 2))
    for m in (VISION, TEXT):
        ll[:, m] = -0.5 * (np.log(var[m]).sum() + (((X - mu[m]) ** 2) / var[m]).sum(axis=1))
    return ll


def modality_score(x, mu, var, tau: float) -> np.ndarray:
    """M_jm = exp(LL_jm / tau) / sum_m' exp(LL_jm' / tau)  (Eq. 9); [T, 2]."""
    ll = log_likelihood(x, mu, var) / tau
    ll = ll - ll.max(axis=1, keepdims=True)
    e = np.exp(ll)
    return e / e.sum(axis=1, keepdims=True)


def default_tau(d: int, tau: float) -> float:
    """tau <= 0 selects the paper's default tau = 0.5 D (Sec. 3.5)."""
    return 0.5 * d if tau <= 0 else tau


# ----------------------------------------------------------------------------
# Sec. 3.3 - 3.4: expert bins and inter-bin mutual information
# ----------------------------------------------------------------------------

def bin_members(expert_to_bin, n_bins: int):
    e2b = np.asarray(expert_to_bin)
    return [np.nonzero(e2b == k)[0] for k in range(n_bins)]


def mi_sample_terms(g, M, expert_to_bin, n_bins: int) -> Dict[str, np.ndarray]:
    """The quantities of Eq. 12-14 for ONE sample (rows of g and M).

    S_bar[m, k] = sum_{e in B_k} sum_j M_jm g_je / (N_B sum_j M_jm)   (Eq. 12)
    P[m, k]     = S_bar[m, k] / sum_{m', k'} S_bar[m', k']             (Eq. 13)
    I           = sum_{m, k} P log(P / (P(m) P(B_k)))                   (Eq. 14)
    """
    g = np.asarray(g, dtype=np.float64)
    M = np.asarray(M, dtype=np.float64)
    E = g.shape[1]
    n_b = E // n_bins
    members = bin_members(expert_to_bin, n_bins)
    S = np.zeros((2, n_bins))
    W = M.sum(axis=0)
    for m in (VISION, TEXT):
        if W[m] <= 0:
            continue
        for k in range(n_bins):
            mass = (M[:, m][:, None] * g[:, members[k]]).sum()
            S[m, k] = mass / (n_b * W[m])
    Z = S.sum()
    P = S / Z if Z > 0 else np.zeros_like(S)
    Pm = P.sum(axis=1)
    Pk = P.sum(axis=0)
    I = 0.0
    for m in (VISION, TEXT):
        for k in range(n_bins):
            if P[m, k] > 0:
                I += P[m, k] * np.log(P[m, k] / (Pm[m] * Pk[k]))
    return dict(S_bar=S, W=W, Z=Z, P=P, Pm=Pm, Pk=Pk, I=I)


def mi_per_sample(g, M, sample_offsets, expert_to_bin, n_bins: int) -> np.ndarray:
    """I_i(M; B) for every sample i (Eq. 14)."""
    off = np.asarray(sample_offsets)
    out = np.zeros(len(off) - 1)
    for i in range(len(off) - 1):
        a, b = int(off[i]), int(off[i + 1])
        if b > a:
            out[i] = mi_sample_terms(g[a:b], M[a:b], expert_to_bin, n_bins)["I"]
    return out


def mi_loss(g, M, sample_offsets, expert_to_bin, n_bins: int) -> float:
    """L_MI = -(1 / N_batch) sum_i I_i for one layer (Eq. 15)."""
    I = mi_per_sample(g, M, sample_offsets, expert_to_bin, n_bins)
    return -float(I.sum()) / len(I)


def mi_loss_grad_logits(g, M, sample_offsets, expert_to_bin, n_bins: int,
                        grad_scale: float = 1.0) -> np.ndarray:
    """grad_scale * dL_MI / dz for the router logits z (M held constant, R9).

    Chain rule through Eq. 12-15 and the softmax of Sec. 3.1:
      dI_i / dS_bar[m, k] = (log r_mk - I_i) / Z,  r_mk = P_mk / (P_m P_k)
      dI_i / dG_jk        = h_jk = sum_m M_jm (log r_mk - I_i) / (N_B W_m Z)
      dI_i / dz_je        = g_je (h_j,bin(e) - sum_k G_jk h_jk)
    where G_jk = sum_{e in B_k} g_je and W_m = sum_j M_jm; terms with W_m = 0 or
    P_mk = 0 are dropped (R12). L_MI = -(1/N_batch) sum_i I_i."""
    g = np.asarray(g, dtype=np.float64)
    M = np.asarray(M, dtype=np.float64)
    off = np.asarray(sample_offsets)
    n_batch = len(off) - 1
    E = g.shape[1]
    n_b = E // n_bins
    e2b = np.asarray(expert_to_bin)
    members = bin_members(e2b, n_bins)
    out = np.zeros_like(g)
    for i in range(n_batch):
        a, b = int(off[i]), int(off[i + 1])
        if b <= a:
            continue
        t = mi_sample_terms(g[a:b], M[a:b], e2b, n_bins)
        coef = np.zeros((2, n_bins))
        for m in (VISION, TEXT):
            if t["W"][m] <= 0:
                continue
            for k in range(n_bins):
                if t["P"][m, k] > 0:
                    log_r = np.log(t["P"][m, k] / (t["Pm"][m] * t["Pk"][k]))
                    coef[m, k] = (log_r - t["I"]) / (n_b * t["W"][m] * t["Z"])
        gi = g[a:b]
        G = np.stack([gi[:, members[k]].sum(axis=1) for k in range(n_bins)], axis=1)
        h = M[a:b] @ coef  # [rows, n_bins]
        hG = (h * G).sum(axis=1)
        out[a:b] = gi * (h[:, e2b] - hG[:, None])
    return (-grad_scale / n_batch) * out


# ----------------------------------------------------------------------------
# MoE experts: permutation, SwiGLU experts, shared experts, combine
# ----------------------------------------------------------------------------

def permutation(topk_idx, E: int):
    """Expert-contiguous order of the (token, slot) pairs: a stable counting
    sort by expert, tokens ascending inside each expert.

    Returns counts[E], offsets[E+1] (exclusive scan), perm_token[R] (token of
    each permuted row) and inv[T, k] (permuted row of each (token, slot))."""
    idx = np.asarray(topk_idx, dtype=np.int64)
    T, k = idx.shape
    counts = np.zeros(E, dtype=np.int64)
    for e in idx.reshape(-1):
        counts[e] += 1
    offsets = np.zeros(E + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    cursor = offsets[:-1].copy()
    perm_token = np.zeros(T * k, dtype=np.int64)
    inv = np.zeros((T, k), dtype=np.int64)
    # tokens in ascending order; each token visits its k experts
    for j in range(T):
        for s in range(k):
            e = idx[j, s]
            r = cursor[e]
            cursor[e] += 1
            perm_token[r] = j
            inv[j, s] = r
    return counts, offsets, perm_token, inv


def silu(a):
    return a / (1.0 + np.exp(-a))


def swiglu(x, w13, w2) -> np.ndarray:
    """down(silu(gate x) * up x) with w13 = [gate rows; up rows] ([2I, d]) and
    w2 = [d, I]  (R7)."""
    X = widen(x)
    W13 = widen(w13)
    inter = W13.shape[0] // 2
    a = X @ W13[:inter].T
    u = X @ W13[inter:].T
    return (silu(a) * u) @ widen(w2).T


def experts_grouped(x, topk_idx, topk_w, w13, w2, ws13=None, ws2=None, E=None):
    """Routed experts over the expert-contiguous permutation, then the weighted
    combine out_j = sum_s w_js Y[inv(j, s)] + shared(x_j)."""
    X = widen(x)
    idx = np.asarray(topk_idx)
    T, k = idx.shape
    E = E if E is not None else w13.shape[0]
    counts, offsets, perm_token, inv = permutation(idx, E)
    Y = np.zeros((T * k, X.shape[1]))
    for e in range(E):
        a, b = offsets[e], offsets[e + 1]
        if b > a:
            Y[a:b] = swiglu(X[perm_token[a:b]], w13[e], w2[e])
    w = np.asarray(topk_w, dtype=np.float64)
    out = np.zeros_like(X)
    for s in range(k):
        out += w[:, s:s + 1] * Y[inv[:, s]]
    shared = swiglu(X, ws13, ws2) if ws13 is not None else np.zeros_like(X)
    return out + shared, out, shared


def experts_naive(x, topk_idx, topk_w, w13, w2, ws13=None, ws2=None):
    """The same layer output by a plain loop: every token through each of its
    k experts, weighted, plus the shared experts."""
    X = widen(x)
    idx = np.asarray(topk_idx)
    w = np.asarray(topk_w, dtype=np.float64)
    out = np.zeros_like(X)
    for j in range(X.shape[0]):
        for s in range(idx.shape[1]):
            out[j] += w[j, s] * swiglu(X[j:j + 1], w13[idx[j, s]], w2[idx[j, s]])[0]
        if ws13 is not None:
            out[j] += swiglu(X[j:j + 1], ws13, ws2)[0]
    return out


# ----------------------------------------------------------------------------
# The whole layer
# ----------------------------------------------------------------------------

def layer_forward(x, modality_id, sample_offsets, w_gate, logit_bias, expert_to_bin,
                  n_bins, k, w13, w2, ws13, ws2, state: GaussState, *, update_stats: bool,
                  beta: float = 0.99, tau: float = 0.0, var_floor: float = 1e-6,
                  grad_scale: float = 1.0, renorm_topk: bool = False,
                  rows: Optional[np.ndarray] = None) -> Dict[str, np.ndarray]:
    """One SMoES MoE layer forward: route, (update and) score modality, MI loss
    and its logit gradient, permutation, experts, combine.

    `rows`, when given, restricts the expert computation to those tokens (the
    routing, modality score and MI always cover the whole batch)."""
    d = widen(w_gate).shape[1]
    z, g, idx, w = route(x, w_gate, k, logit_bias, renorm_topk)
    if update_stats:
        state = gauss_update(state, x, modality_id, beta)
    mu, var = gauss_params(state, var_floor)
    M = modality_score(x, mu, var, default_tau(d, tau))
    I = mi_per_sample(g, M, sample_offsets, expert_to_bin, n_bins)
    loss = -float(I.sum()) / len(I)
    dlogits = mi_loss_grad_logits(g, M, sample_offsets, expert_to_bin, n_bins, grad_scale)
    E = widen(w_gate).shape[0]
    counts, offsets, perm_token, inv = permutation(idx, E)
    out = {"logits": z, "probs": g, "topk_idx": idx, "topk_w": w, "gap": topk_gap(z, k),
           "state": state, "M": M, "mi_per_sample": I, "loss": loss, "dlogits": dlogits,
           "expert_counts": counts, "expert_offsets": offsets, "perm_token": perm_token, "inv": inv}
    if w13 is not None:
        if rows is None:
            full, routed, shared = experts_grouped(x, idx, w, w13, w2, ws13, ws2, E)
        else:
            xs = np.asarray(x)[rows]
            full, routed, shared = experts_grouped(xs, idx[rows], w[rows], w13, w2, ws13, ws2, E)
        out.update(out=full, routed=routed, shared=shared)
    return out


# ----------------------------------------------------------------------------
# Sec. 3.3: momentum-adaptive binning (Eq. 10-11); Sec. 3.5: bin-level load
# balance (Eq. 16); Sec. 4.1 diagnostic: modality specialization index
# (Eq. 18-19)
# ----------------------------------------------------------------------------

def modality_expert_counts(topk_idx, modality_id, E: int) -> np.ndarray:
    """C[m][e]: tokens of hard label m whose top-k holds expert e (Eq. 10)."""
    idx = np.asarray(topk_idx, dtype=np.int64)
    mid = np.asarray(modality_id, dtype=np.int64)
    C = np.zeros((2, E), dtype=np.int64)
    for m in (VISION, TEXT):
        rows = idx[mid == m]
        if rows.size:
            C[m] = np.bincount(rows.ravel(), minlength=E)
    return C


def load_ema_update(C_bar, C, beta: float) -> np.ndarray:
    """Eq. 10: C_bar <- beta * C_bar + (1 - beta) * C, float64 (R15)."""
    b = float(np.float32(beta))
    return b * np.asarray(C_bar, dtype=np.float64) + (1.0 - b) * np.asarray(C, dtype=np.float64)


def f_spec(C_bar) -> np.ndarray:
    """Eq. 11: text-bias score of each expert; 1/2 where no load (R15)."""
    cb = np.asarray(C_bar, dtype=np.float64)
    tot = cb[TEXT] + cb[VISION]
    out = np.full(cb.shape[1], 0.5)
    nz = tot > 0
    out[nz] = cb[TEXT][nz] / tot[nz]
    return out


def adaptive_bins(fs, n_bins: int) -> np.ndarray:
    """Sort experts by f_spec (ascending, ties to the lower index) and cut the
    order into n_bins consecutive bins of N_B experts (Sec. 3.3, R15)."""
    fs = np.asarray(fs, dtype=np.float64)
    E = fs.shape[0]
    NB = E // n_bins
    order = np.argsort(fs, kind="stable")
    e2b = np.empty(E, dtype=np.int32)
    e2b[order] = np.arange(E) // NB
    return e2b


def bin_balance_terms(g, topk_idx, expert_to_bin, n_bins: int) -> Dict[str, np.ndarray]:
    """Per-bin token sets and per-expert f_e, P_e of Eq. 16 (R14)."""
    g = np.asarray(g, dtype=np.float64)
    idx = np.asarray(topk_idx, dtype=np.int64)
    e2b = np.asarray(expert_to_bin, dtype=np.int64)
    T, E = g.shape
    in_bin = np.zeros((T, n_bins), dtype=bool)
    in_bin[np.repeat(np.arange(T), idx.shape[1]), e2b[idx.ravel()]] = True
    Tk = in_bin.sum(axis=0)
    counts = np.bincount(idx.ravel(), minlength=E).astype(np.float64)
    f = np.zeros(E)
    P = np.zeros(E)
    for e in range(E):
        k = e2b[e]
        if Tk[k] > 0:
            f[e] = counts[e] / Tk[k]
            P[e] = g[in_bin[:, k], e].sum() / Tk[k]
    return dict(in_bin=in_bin, Tk=Tk, counts=counts, f=f, P=P)


def bin_balance_loss(g, topk_idx, expert_to_bin, n_bins: int) -> float:
    """Eq. 16 for one layer: sum_k N_B sum_{e in B_k} f_e P_e (R14)."""
    E = np.asarray(g).shape[1]
    NB = E // n_bins
    t = bin_balance_terms(g, topk_idx, expert_to_bin, n_bins)
    return float(NB * np.sum(t["f"] * t["P"]))


def bin_balance_grad_logits(g, topk_idx, expert_to_bin, n_bins: int, grad_scale: float = 1.0) -> np.ndarray:
    """grad_scale * d L_bal / d z with the top-k sets fixed (R14): through
    P_e only, dL/dg_je = N_B f_e / T_k for tokens j routed to bin k = bin(e),
    then the softmax Jacobian dz = g (dg - sum_e g dg)."""
    g = np.asarray(g, dtype=np.float64)
    E = g.shape[1]
    NB = E // n_bins
    e2b = np.asarray(expert_to_bin, dtype=np.int64)
    t = bin_balance_terms(g, topk_idx, expert_to_bin, n_bins)
    coef = np.zeros(E)
    for e in range(E):
        k = e2b[e]
        if t["Tk"][k] > 0:
            coef[e] = NB * t["f"][e] / t["Tk"][k]
    dg = t["in_bin"][:, e2b] * coef[None, :]
    dz = g * (dg - np.sum(g * dg, axis=1, keepdims=True))
    return grad_scale * dz


def msi(counts_text, counts_vision) -> float:
    """MSI for one layer (Eq. 18-19) from per-expert token counts per
    modality (R16)."""
    ct = np.asarray(counts_text, dtype=np.float64)
    cv = np.asarray(counts_vision, dtype=np.float64)
    nt = ct / ct.sum() if ct.sum() > 0 else np.zeros_like(ct)
    nv = cv / cv.sum() if cv.sum() > 0 else np.zeros_like(cv)
    den = nt + nv
    c_text = np.full(ct.shape, 0.5)
    nz = den > 0
    c_text[nz] = nt[nz] / den[nz]
    return float(np.mean(2.0 * np.abs(c_text - 0.5)))


# ----------------------------------------------------------------------------
# Attention-accumulated modality score (Sec. 3.2.1, Eq. 2-4). The paper's
# implementation note carries the scores as extra value channels through the
# attention; here the attention matrix is formed explicitly, per sample and
# head, as the definition reads.
# ----------------------------------------------------------------------------

def attn_score_init(modality_id) -> np.ndarray:
    """Layer-0 scores (Eq. 2): the one-hot hard label; columns (vision, text) (R13)."""
    mid = np.asarray(modality_id)
    M = np.zeros((mid.shape[0], 2))
    M[mid == VISION, 0] = 1.0
    M[mid == TEXT, 1] = 1.0
    return M


def attention_heads(q, k, v, sample_offsets, M, scale: Optional[float] = None):
    """Per query head h: Attn_h = causal softmax(q_h k_h^T * scale) inside each
    sample (R17); returns O[T, H, d_head] = Attn_h v_h and A[T, H, 2] = Attn_h M
    (Eq. 3 before the head average). q: [T, H, d_head]; k, v: [T, H_kv, d_head]."""
    Q, K, V = widen(q), widen(k), widen(v)
    Ms = np.asarray(M, dtype=np.float64)
    T, H, dh = Q.shape
    Hkv = K.shape[1]
    group = H // Hkv
    sc = 1.0 / math.sqrt(dh) if scale is None else float(scale)
    O = np.zeros((T, H, V.shape[2]))
    A = np.zeros((T, H, 2))
    off = np.asarray(sample_offsets)
    for i in range(len(off) - 1):
        lo, hi = int(off[i]), int(off[i + 1])
        L = hi - lo
        if L == 0:
            continue
        causal = np.tril(np.ones((L, L), dtype=bool))
        for h in range(H):
            hk = h // group
            logits = (Q[lo:hi, h] @ K[lo:hi, hk].T) * sc
            logits = np.where(causal, logits, -np.inf)
            logits = logits - logits.max(axis=1, keepdims=True)
            P = np.exp(logits)
            P = P / P.sum(axis=1, keepdims=True)
            O[lo:hi, h] = P @ V[lo:hi, hk]
            A[lo:hi, h] = P @ Ms[lo:hi]
    return O, A


def attn_aggregate(A) -> np.ndarray:
    """M_tilde = Attn M with Attn averaged over heads (Eq. 3); A from attention_heads."""
    return np.asarray(A, dtype=np.float64).mean(axis=1)


def attn_score_update(x, x_attn, M, M_tilde) -> np.ndarray:
    """M^(l+1) = (|x_attn| M_tilde + |x| M) / (|x_attn| + |x|)  (Eq. 4, R18)."""
    nx = np.sqrt((widen(x) ** 2).sum(axis=1))
    na = np.sqrt((widen(x_attn) ** 2).sum(axis=1))
    M = np.asarray(M, dtype=np.float64)
    Mt = np.asarray(M_tilde, dtype=np.float64)
    out = M.copy()
    den = nx + na
    nz = den > 0
    out[nz] = (na[nz, None] * Mt[nz] + nx[nz, None] * M[nz]) / den[nz, None]
    return out


# ----------------------------------------------------------------------------
# GMM estimator (supplementary GMM ablation; R19): K diagonal components per
# modality in place of the single Gaussian of Sec. 3.2.2.
# ----------------------------------------------------------------------------

@dataclass
class GmmState:
    """EMA state per modality m and component c: N[2, K], S_mu[2, K, D], S_sigma2[2, K, D]."""

    n: np.ndarray
    s_mu: np.ndarray
    s_sig: np.ndarray

    @staticmethod
    def of(n, s_mu, s_sig) -> "GmmState":
        return GmmState(widen(n).copy(), widen(s_mu).copy(), widen(s_sig).copy())


def gmm_params(state: GmmState, var_floor: float):
    """pi_mc = N_mc / sum_c N_mc, mu_mc = S_mu / N, sigma^2_mc = S_sigma2 / N floored (R19)."""
    _, K, d = state.s_mu.shape
    pi = np.full((2, K), 1.0 / K)
    mu = np.zeros((2, K, d))
    var = np.ones((2, K, d))
    for m in (VISION, TEXT):
        tot = state.n[m].sum()
        if tot > 0:
            pi[m] = state.n[m] / tot
        for c in range(K):
            if state.n[m, c] > 0:
                mu[m, c] = state.s_mu[m, c] / state.n[m, c]
                var[m, c] = np.maximum(state.s_sig[m, c] / state.n[m, c], var_floor)
    return pi, mu, var


def gmm_component_loglik(x, pi, mu, var) -> np.ndarray:
    """log pi_mc - 1/2 sum_d (log sigma^2_mcd + (x_d - mu_mcd)^2 / sigma^2_mcd); [T, 2, K]."""
    X = widen(x)
    K = pi.shape[1]
    out = np.empty((X.shape[0], 2, K))
    for m in (VISION, TEXT):
        for c in range(K):
            with np.errstate(divide="ignore"):
                lp = np.log(pi[m, c])
            out[:, m, c] = lp - 0.5 * (np.log(var[m, c]).sum() + (((X - mu[m, c]) ** 2) / var[m, c]).sum(axis=1))
    return out


def _logsumexp_last(a) -> np.ndarray:
    mx = a.max(axis=-1, keepdims=True)
    mx = np.where(np.isfinite(mx), mx, 0.0)
    return (mx + np.log(np.exp(a - mx).sum(axis=-1, keepdims=True)))[..., 0]


def gmm_log_likelihood(x, pi, mu, var) -> np.ndarray:
    """LL_jm = log sum_c exp(component log-likelihood); [T, 2] (R19)."""
    return _logsumexp_last(gmm_component_loglik(x, pi, mu, var))


def gmm_modality_score(x, pi, mu, var, tau: float) -> np.ndarray:
    """Eq. 9 with the mixture log-likelihood; [T, 2]."""
    ll = gmm_log_likelihood(x, pi, mu, var) / tau
    ll = ll - ll.max(axis=1, keepdims=True)
    e = np.exp(ll)
    return e / e.sum(axis=1, keepdims=True)


def gmm_responsibilities(x, modality_id, pi, mu, var) -> np.ndarray:
    """r_jc = posterior of component c under the mixture of token j's own
    modality (the E-step); [T, K]."""
    cl = gmm_component_loglik(x, pi, mu, var)
    mid = np.asarray(modality_id)
    own = cl[np.arange(cl.shape[0]), mid]  # [T, K]
    return np.exp(own - _logsumexp_last(own)[:, None])


def gmm_update(state: GmmState, x, modality_id, beta: float, var_floor: float) -> GmmState:
    """Stepwise EM (R19): responsibilities under the current parameters, then
    per modality m and component c, with weights r_jc over the tokens T_m:
        n      = sum r,  mu_T = sum r x / n,  Q = sum r (x - mu_T)^2
        N_t    = beta N_{t-1} + n
        S_mu,t = beta S_mu,t-1 + n mu_T
        S_sig,t= beta S_sig,t-1 + Q + (mu_T - S_mu,t-1 / N_{t-1})^2 beta N_{t-1} n / (beta N_{t-1} + n)
    (Eq. 5-7 with weighted batch statistics; the last term is 0 when
    N_{t-1} = 0 or n = 0)."""
    X = widen(x)
    mid = np.asarray(modality_id)
    pi, mu, var = gmm_params(state, var_floor)
    r = gmm_responsibilities(X, mid, pi, mu, var)
    _, K, d = state.s_mu.shape
    n_new = state.n.copy()
    s_mu_new = state.s_mu.copy()
    s_sig_new = state.s_sig.copy()
    for m in (VISION, TEXT):
        sel = mid == m
        Xm = X[sel]
        for c in range(K):
            w = r[sel, c]
            n = w.sum()
            if n > 0:
                mu_T = (w[:, None] * Xm).sum(axis=0) / n
                Q = (w[:, None] * (Xm - mu_T) ** 2).sum(axis=0)
            else:
                mu_T = np.zeros(d)
                Q = np.zeros(d)
            n_prev = state.n[m, c]
            if n_prev > 0 and n > 0:
                prev_mean = state.s_mu[m, c] / n_prev
                cross = (mu_T - prev_mean) ** 2 * (beta * n_prev * n) / (beta * n_prev + n)
            else:
                cross = np.zeros(d)
            n_new[m, c] = beta * n_prev + n
            s_mu_new[m, c] = beta * state.s_mu[m, c] + n * mu_T
            s_sig_new[m, c] = beta * state.s_sig[m, c] + Q + cross
    return GmmState(n_new, s_mu_new, s_sig_new)


# ----------------------------------------------------------------------------
# Layer backward (R20): the gradients of a loss through the layer output,
# dL/d out given, with auxiliary logit gradients folded into the router.
# ----------------------------------------------------------------------------

def swiglu_backward(x, w13, w2, dy):
    """For rows y = W2 (silu(a) * b), a = W1 x, b = W3 x, given dy: returns dx,
    dW13 = [dW1; dW3] ([2I, d]) and dW2 ([d, I])."""
    X = widen(x)
    W13 = widen(w13)
    W2 = widen(w2)
    dY = np.asarray(dy, dtype=np.float64)
    inter = W13.shape[0] // 2
    a = X @ W13[:inter].T
    b = X @ W13[inter:].T
    sig = 1.0 / (1.0 + np.exp(-a))
    sa = a * sig
    h = sa * b
    dh = dY @ W2
    da = dh * b * (sig * (1.0 + a * (1.0 - sig)))  # d silu / da = sig (1 + a (1 - sig))
    db = dh * sa
    dx = da @ W13[:inter] + db @ W13[inter:]
    return dx, np.concatenate([da.T @ X, db.T @ X]), dY.T @ h


def layer_backward(x, w_gate, logit_bias, k: int, w13, w2, ws13, ws2, dout, dlogits_aux=None,
                   renorm_topk: bool = False) -> Dict[str, np.ndarray]:
    """Gradients of the layer (R20) given dout = dL/d out [T, d]:
    dw [T, k] combine weights, dz [T, E] logits (with dlogits_aux added),
    dw_gate [E, d], dbias [E], dw13 [E, 2I, d], dw2 [E, d, I], dws13, dws2 and
    dx [T, d] (experts, shared experts and router)."""
    X = widen(x)
    Wg = widen(w_gate)
    dO = np.asarray(dout, dtype=np.float64)
    z, g, idx, w = route(x, w_gate, k, logit_bias, renorm_topk)
    T, d = X.shape
    E = Wg.shape[0]
    counts, offsets, perm_token, inv = permutation(idx, E)
    Y = np.zeros((T * k, d))
    for e in range(E):
        a, b = offsets[e], offsets[e + 1]
        if b > a:
            Y[a:b] = swiglu(X[perm_token[a:b]], w13[e], w2[e])
    # combine: out_j = sum_s w_js Y[inv(j, s)] + shared_j
    dw = np.stack([(dO * Y[inv[:, s]]).sum(axis=1) for s in range(k)], axis=1)
    dY = np.zeros((T * k, d))
    for s in range(k):
        dY[inv[:, s]] = w[:, s:s + 1] * dO
    # routed experts
    dx = np.zeros((T, d))
    dw13 = np.zeros(widen(w13).shape)
    dw2 = np.zeros(widen(w2).shape)
    for e in range(E):
        a, b = offsets[e], offsets[e + 1]
        if b > a:
            dxe, dw13[e], dw2[e] = swiglu_backward(X[perm_token[a:b]], w13[e], w2[e], dY[a:b])
            np.add.at(dx, perm_token[a:b], dxe)
    dws13 = dws2 = None
    if ws13 is not None:
        dxs, dws13, dws2 = swiglu_backward(X, ws13, ws2, dO)
        dx += dxs
    # combine weights -> gates at the chosen experts -> full softmax -> logits
    gsel = np.take_along_axis(g, idx.astype(np.int64), axis=1)
    if renorm_topk:
        S = gsel.sum(axis=1, keepdims=True)
        dsel = (dw - (w * dw).sum(axis=1, keepdims=True)) / S
    else:
        dsel = dw
    dg = np.zeros((T, E))
    for s in range(k):
        dg[np.arange(T), idx[:, s]] += dsel[:, s]
    dz = g * (dg - (g * dg).sum(axis=1, keepdims=True))
    if dlogits_aux is not None:
        dz = dz + np.asarray(dlogits_aux, dtype=np.float64)
    dx += dz @ Wg
    return {"dw": dw, "dz": dz, "dw_gate": dz.T @ X, "dbias": dz.sum(axis=0), "dw13": dw13, "dw2": dw2,
            "dws13": dws13, "dws2": dws2, "dx": dx}
