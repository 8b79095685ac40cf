"""Python binding of libsmoes.so (ctypes; argument marshalling only).

Every function takes and returns torch tensors on the current HIP device and
enqueues on torch's current stream; all arithmetic runs in the HIP kernels of
libsmoes.so. There is no fallback: if the library is missing this module
raises when it is used.

Names follow the C ABI in include/smoes.h: route, modality_score, mi_loss,
permute, moe_forward (+ workspace helpers and the layer descriptor).
"""
from __future__ import annotations

import ctypes
import os
import re
from dataclasses import dataclass
from typing import Dict, Optional, Sequence

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libsmoes.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "smoes.h")

SMOES_OK, SMOES_ERR_ARG, SMOES_ERR_SHAPE, SMOES_ERR_WORKSPACE, SMOES_ERR_HIP = 0, -1, -2, -3, -4
SMOES_ERR_SCRATCH = -5
SMOES_NOALLOC_SCRATCH_BYTES = 8 << 20
SMOES_F32, SMOES_BF16 = 0, 1
N_STAGES = 9
STAGES = ("route", "modality", "mi", "permute", "gemm1", "gemm2", "combine", "gemm1_shared", "gemm2_shared")

_lib = None


class SmoesError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} ({status})")


c_i64, c_int, c_float, c_size, c_void = ctypes.c_int64, ctypes.c_int, ctypes.c_float, ctypes.c_size_t, ctypes.c_void_p


class SmoesLayer(ctypes.Structure):
    _fields_ = [("T", c_i64), ("d", c_int), ("E", c_int), ("k", c_int), ("inter", c_int),
                ("shared_inter", c_int), ("n_bins", c_int), ("n_batch", c_int), ("act_dtype", c_int),
                ("tau", c_float), ("beta", c_float), ("var_floor", c_float), ("grad_scale", c_float),
                ("renorm_topk", c_int), ("update_stats", c_int), ("weights_packed", c_int),
                ("save_preact", c_int), ("check_inputs", c_int)]


_IO_FIELDS = ["x", "modality_id", "sample_offsets", "w_gate", "logit_bias", "expert_to_bin", "w13",
              "w2", "ws13", "ws2", "w_gate_packed", "gauss_n", "gauss_smu", "gauss_ssig", "logits", "probs", "topk_idx",
              "topk_w", "M", "mi_per_sample", "loss", "dlogits", "expert_offsets", "perm_token",
              "perm_inv", "out", "stage_events"]


class SmoesLayerIO(ctypes.Structure):
    _fields_ = [(n, c_void) for n in _IO_FIELDS] + [("streams", c_void)]


_GRAD_FIELDS = ["dx", "dw_gate", "dbias", "dz", "dw", "dw13", "dw2", "dws13", "dws2"]


class SmoesLayerGrads(ctypes.Structure):
    _fields_ = [(n, c_void) for n in _GRAD_FIELDS]


class SmoesStreams(ctypes.Structure):
    _fields_ = [("side", c_void * 2), ("events", c_void * 4)]


def lib() -> ctypes.CDLL:
    """Load libsmoes.so (built by paper_2604_23996_amd.build); raise if absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: run `python -m paper_2604_23996_amd.build` "
                              "(there is no fallback path)")
        L = ctypes.CDLL(LIB_PATH)
        L.smoes_status_string.restype = ctypes.c_char_p
        L.smoes_status_string.argtypes = [c_int]
        L.smoes_version.restype = ctypes.c_char_p
        L.smoes_route_workspace_size.restype = c_size
        L.smoes_route_workspace_size.argtypes = [c_i64, c_int, c_int, c_int]
        L.smoes_route.restype = c_int
        L.smoes_route.argtypes = [c_void, c_int, c_i64, c_int, c_void, c_void, c_int, c_int, c_int,
                                  c_void, c_void, c_void, c_void, c_void, c_size, c_void]
        L.smoes_modality_workspace_size.restype = c_size
        L.smoes_modality_workspace_size.argtypes = [c_i64, c_int]
        L.smoes_modality_score.restype = c_int
        L.smoes_modality_score.argtypes = [c_void, c_int, c_i64, c_int, c_void, c_void, c_void, c_void,
                                           c_int, c_float, c_float, c_float, c_void, c_void, c_size, c_void]
        L.smoes_mi_workspace_size.restype = c_size
        L.smoes_mi_workspace_size.argtypes = [c_i64, c_int, c_int, c_int]
        L.smoes_mi_loss.restype = c_int
        L.smoes_mi_loss.argtypes = [c_void, c_void, c_i64, c_int, c_void, c_int, c_void, c_int, c_float,
                                    c_void, c_void, c_void, c_void, c_size, c_void]
        L.smoes_mi_loss_noalloc.restype = c_int
        L.smoes_mi_loss_noalloc.argtypes = [c_void, c_void, c_i64, c_int, c_void, c_int, c_void, c_int, c_float,
                                            c_void, c_void, c_void, c_void]
        L.smoes_permute_workspace_size.restype = c_size
        L.smoes_permute_workspace_size.argtypes = [c_i64, c_int, c_int]
        L.smoes_permute.restype = c_int
        L.smoes_permute.argtypes = [c_void, c_i64, c_int, c_int, c_void, c_void, c_void, c_void, c_int,
                                    c_int, c_void, c_void, c_size, c_void]
        L.smoes_workspace_bytes.restype = c_size
        L.smoes_workspace_bytes.argtypes = [ctypes.POINTER(SmoesLayer)]
        L.smoes_moe_forward.restype = c_int
        L.smoes_moe_forward.argtypes = [ctypes.POINTER(SmoesLayer), ctypes.POINTER(SmoesLayerIO),
                                        c_void, c_size, c_void]
        L.smoes_packed_weight_bytes.restype = c_size
        L.smoes_packed_weight_bytes.argtypes = [ctypes.POINTER(SmoesLayer), c_int]
        L.smoes_pack_weights.restype = c_int
        L.smoes_pack_weights.argtypes = [ctypes.POINTER(SmoesLayer), c_int, c_void, c_void, c_void]
        L.smoes_binning_workspace_size.restype = c_size
        L.smoes_binning_workspace_size.argtypes = [c_i64, c_int, c_int]
        L.smoes_binning.restype = c_int
        L.smoes_binning.argtypes = [c_void, c_void, c_void, c_i64, c_int, c_int, c_void, c_int, c_float, c_void,
                                    c_void, c_void, c_void, c_float, c_void, c_void, c_int, c_void, c_void,
                                    c_size, c_void]
        L.smoes_backward_workspace_bytes.restype = c_size
        L.smoes_backward_workspace_bytes.argtypes = [ctypes.POINTER(SmoesLayer)]
        L.smoes_moe_backward.restype = c_int
        L.smoes_moe_backward.argtypes = [ctypes.POINTER(SmoesLayer), ctypes.POINTER(SmoesLayerIO), c_void, c_void,
                                         c_void, c_void, c_void, c_void, ctypes.POINTER(SmoesLayerGrads), c_void,
                                         c_size, c_void, c_size, c_void]
        L.smoes_gmm_workspace_size.restype = c_size
        L.smoes_gmm_workspace_size.argtypes = [c_i64, c_int, c_int]
        L.smoes_gmm_modality_score.restype = c_int
        L.smoes_gmm_modality_score.argtypes = [c_void, c_int, c_i64, c_int, c_int, c_void, c_void, c_void, c_void,
                                               c_int, c_float, c_float, c_float, c_void, c_void, c_void, c_size,
                                               c_void]
        L.smoes_attn_score_init.restype = c_int
        L.smoes_attn_score_init.argtypes = [c_void, c_i64, c_void, c_void]
        L.smoes_attention_scores.restype = c_int
        L.smoes_attention_scores.argtypes = [c_void, c_void, c_void, c_i64, c_int, c_int, c_int, c_void, c_int,
                                             c_void, c_float, c_void, c_void, c_void]
        L.smoes_attn_score_update.restype = c_int
        L.smoes_attn_score_update.argtypes = [c_void, c_void, c_int, c_i64, c_int, c_void, c_int, c_void, c_void,
                                              c_void]
        L.smoes_workspace_buffer.restype = c_int
        L.smoes_workspace_buffer.argtypes = [ctypes.POINTER(SmoesLayer), c_void, c_int, ctypes.POINTER(c_void),
                                             ctypes.POINTER(c_size)]
        L.smoes_check_inputs.restype = c_int
        L.smoes_check_inputs.argtypes = [ctypes.POINTER(SmoesLayer), ctypes.POINTER(SmoesLayerIO), c_void, c_void]
        L.smoes_streams_create.restype = c_int
        L.smoes_streams_create.argtypes = [ctypes.POINTER(SmoesStreams)]
        L.smoes_streams_destroy.restype = c_int
        L.smoes_streams_destroy.argtypes = [ctypes.POINTER(SmoesStreams)]
        L.smoes_events_create.restype = c_int
        L.smoes_events_create.argtypes = [c_int, ctypes.POINTER(c_void)]
        L.smoes_events_destroy.restype = c_int
        L.smoes_events_destroy.argtypes = [c_int, ctypes.POINTER(c_void)]
        L.smoes_event_elapsed_ms.restype = c_int
        L.smoes_event_elapsed_ms.argtypes = [c_void, c_void, ctypes.POINTER(c_float)]
        _lib = L
    return _lib


def header_functions() -> Sequence[str]:
    """Names of the functions include/smoes.h declares."""
    text = open(HEADER_PATH).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(smoes_[a-z_0-9]+)\s*\(", text)))


def status_string(status: int) -> str:
    return lib().smoes_status_string(int(status)).decode()


def _check(status: int, where: str):
    if status != SMOES_OK:
        raise SmoesError(status, where)


def _p(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to libsmoes must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return SMOES_BF16
    if t.dtype == torch.float32:
        return SMOES_F32
    raise TypeError(f"unsupported activation dtype {t.dtype}")


def _workspace(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


# ---------------------------------------------------------------- entry points

def route(x: torch.Tensor, w_gate: torch.Tensor, k: int, logit_bias: Optional[torch.Tensor] = None,
          renorm_topk: bool = False, want_logits: bool = True) -> Dict[str, torch.Tensor]:
    T, d = x.shape
    E = w_gate.shape[0]
    dev = x.device
    logits = torch.empty((T, E), dtype=torch.float32, device=dev) if want_logits else None
    probs = torch.empty((T, E), dtype=torch.float32, device=dev)
    idx = torch.empty((T, k), dtype=torch.int32, device=dev)
    w = torch.empty((T, k), dtype=torch.float32, device=dev)
    dt = _dtype_code(x)
    nbytes = lib().smoes_route_workspace_size(T, d, E, dt)
    ws = _workspace(nbytes, dev)
    _check(lib().smoes_route(_p(x), dt, T, d, _p(w_gate), _p(logit_bias), E, k, int(renorm_topk),
                             _p(logits), _p(probs), _p(idx), _p(w), _p(ws), nbytes, _stream()),
           "smoes_route")
    return {"logits": logits, "probs": probs, "topk_idx": idx, "topk_w": w}


def modality_score(x: torch.Tensor, gauss_n: torch.Tensor, gauss_smu: torch.Tensor,
                   gauss_ssig: torch.Tensor, modality_id: Optional[torch.Tensor] = None,
                   update: bool = False, beta: float = 0.99, tau: float = 0.0,
                   var_floor: float = 1e-6) -> torch.Tensor:
    """Soft modality scores [T, 2]; with update=True the state tensors are updated in place."""
    T, d = x.shape
    M = torch.empty((T, 2), dtype=torch.float32, device=x.device)
    nbytes = lib().smoes_modality_workspace_size(T, d)
    ws = _workspace(nbytes, x.device)
    _check(lib().smoes_modality_score(_p(x), _dtype_code(x), T, d, _p(modality_id), _p(gauss_n),
                                      _p(gauss_smu), _p(gauss_ssig), int(update), beta, tau, var_floor,
                                      _p(M), _p(ws), nbytes, _stream()), "smoes_modality_score")
    return M


def mi_loss(probs: torch.Tensor, M: torch.Tensor, sample_offsets: Optional[torch.Tensor],
            expert_to_bin: torch.Tensor, n_bins: int, grad_scale: float = 1.0,
            want_grad: bool = True):
    """Returns (mi_per_sample [n_batch], loss [1], dlogits [T, E] or None)."""
    T, E = probs.shape
    n_batch = 1 if sample_offsets is None else sample_offsets.numel() - 1
    dev = probs.device
    mi = torch.empty(n_batch, dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    dl = torch.empty((T, E), dtype=torch.float32, device=dev) if want_grad else None
    nbytes = lib().smoes_mi_workspace_size(T, E, n_batch, n_bins)
    ws = _workspace(nbytes, dev)
    _check(lib().smoes_mi_loss(_p(probs), _p(M), T, E, _p(sample_offsets), n_batch, _p(expert_to_bin),
                               n_bins, grad_scale, _p(mi), _p(loss), _p(dl), _p(ws), nbytes, _stream()),
           "smoes_mi_loss")
    return mi, loss, dl


def mi_loss_noalloc(probs: torch.Tensor, M: torch.Tensor, sample_offsets: Optional[torch.Tensor],
                    expert_to_bin: torch.Tensor, n_bins: int, grad_scale: float = 1.0,
                    outputs: Optional[tuple] = None, want_grad: bool = True):
    """smoes_mi_loss_noalloc (no workspace: the library's fixed device array).
    `outputs` = (mi_per_sample, loss, dlogits or None) preallocated by the
    caller, or None to allocate them here. Returns the three."""
    T, E = probs.shape
    n_batch = 1 if sample_offsets is None else sample_offsets.numel() - 1
    if outputs is None:
        dev = probs.device
        outputs = (torch.empty(n_batch, dtype=torch.float32, device=dev),
                   torch.empty(1, dtype=torch.float32, device=dev),
                   torch.empty((T, E), dtype=torch.float32, device=dev) if want_grad else None)
    mi, loss, dl = outputs
    _check(lib().smoes_mi_loss_noalloc(_p(probs), _p(M), T, E, _p(sample_offsets), n_batch, _p(expert_to_bin),
                                       n_bins, grad_scale, _p(mi), _p(loss), _p(dl), _stream()),
           "smoes_mi_loss_noalloc")
    return mi, loss, dl


def binning(probs: torch.Tensor, topk_idx: torch.Tensor, modality_id: torch.Tensor, expert_to_bin: torch.Tensor,
            n_bins: int, beta: float = 0.99, load_ema: Optional[torch.Tensor] = None, grad_scale: float = 1.0,
            dlogits: Optional[torch.Tensor] = None, accumulate: bool = False,
            want_grad: bool = True) -> Dict[str, torch.Tensor]:
    """smoes_binning: adaptive bins for the next batch, the bin-level load
    balance loss (+ its logit gradient) and MSI. load_ema ([2, E] float64) is
    updated in place when given; dlogits is written (or added to) when given,
    else a new array is returned when want_grad."""
    T, E = probs.shape
    k = topk_idx.shape[1]
    dev = probs.device
    out = {
        "counts": torch.empty((2, E), dtype=torch.int32, device=dev),
        "f_spec": torch.empty(E, dtype=torch.float64, device=dev),
        "expert_to_bin_next": torch.empty(E, dtype=torch.int32, device=dev),
        "bal_loss": torch.empty(1, dtype=torch.float32, device=dev),
        "msi": torch.empty(1, dtype=torch.float32, device=dev),
    }
    if dlogits is None and want_grad:
        dlogits = torch.empty((T, E), dtype=torch.float32, device=dev)
    out["dlogits"] = dlogits
    nws = int(lib().smoes_binning_workspace_size(T, E, n_bins))
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
    _check(lib().smoes_binning(_p(probs), _p(topk_idx), _p(modality_id), T, E, k, _p(expert_to_bin), n_bins,
                               beta, _p(load_ema), _p(out["counts"]), _p(out["f_spec"]),
                               _p(out["expert_to_bin_next"]), grad_scale, _p(out["bal_loss"]), _p(dlogits),
                               int(accumulate), _p(out["msi"]), _p(ws), ws.numel(), _stream()), "smoes_binning")
    return out


def gmm_modality_score(x: torch.Tensor, gmm_n: torch.Tensor, gmm_smu: torch.Tensor, gmm_ssig: torch.Tensor,
                       modality_id: Optional[torch.Tensor] = None, update: bool = False, beta: float = 0.99,
                       tau: float = 0.0, var_floor: float = 1e-6, want_resp: bool = False):
    """smoes_gmm_modality_score: scores M [T, 2] under the K-component mixtures
    (state updated in place by one stepwise-EM step when update); returns
    (M, resp or None)."""
    T, d = x.shape
    K = gmm_n.shape[1]
    M = torch.empty((T, 2), dtype=torch.float32, device=x.device)
    resp = torch.empty((T, K), dtype=torch.float32, device=x.device) if want_resp else None
    nbytes = int(lib().smoes_gmm_workspace_size(T, d, K))
    ws = _workspace(max(nbytes, 1), x.device)
    _check(lib().smoes_gmm_modality_score(_p(x), _dtype_code(x), T, d, K, _p(modality_id), _p(gmm_n), _p(gmm_smu),
                                          _p(gmm_ssig), int(update), beta, tau, var_floor, _p(M), _p(resp), _p(ws),
                                          nbytes, _stream()), "smoes_gmm_modality_score")
    return M, resp


def attn_score_init(modality_id: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """smoes_attn_score_init: one-hot layer-0 scores [T, 2] (Eq. 2)."""
    T = modality_id.shape[0]
    if out is None:
        out = torch.empty((T, 2), dtype=torch.float32, device=modality_id.device)
    _check(lib().smoes_attn_score_init(_p(modality_id), T, _p(out), _stream()), "smoes_attn_score_init")
    return out


def attention_scores(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, sample_offsets: torch.Tensor,
                     m_in: torch.Tensor, scale: float = 0.0, o: Optional[torch.Tensor] = None,
                     m_heads: Optional[torch.Tensor] = None):
    """smoes_attention_scores: causal per-sample attention O [T, H, d_head] (bf16)
    and the per-head aggregated scores m_heads [T, H, 2] (Eq. 3 before the head mean)."""
    T, H, dh = q.shape
    Hkv = k.shape[1]
    dev = q.device
    if o is None:
        o = torch.empty((T, H, dh), dtype=torch.bfloat16, device=dev)
    if m_heads is None:
        m_heads = torch.empty((T, H, 2), dtype=torch.float32, device=dev)
    n_batch = sample_offsets.numel() - 1
    _check(lib().smoes_attention_scores(_p(q), _p(k), _p(v), T, H, Hkv, dh, _p(sample_offsets), n_batch,
                                        _p(m_in), scale, _p(o), _p(m_heads), _stream()), "smoes_attention_scores")
    return o, m_heads


def attn_score_update(x: torch.Tensor, x_attn: torch.Tensor, m_heads: torch.Tensor, m_in: torch.Tensor,
                      out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """smoes_attn_score_update: head mean (Eq. 3) and norm-weighted mix (Eq. 4) -> [T, 2]."""
    T, d = x.shape
    H = m_heads.shape[1]
    if out is None:
        out = torch.empty((T, 2), dtype=torch.float32, device=x.device)
    _check(lib().smoes_attn_score_update(_p(x), _p(x_attn), _dtype_code(x), T, d, _p(m_heads), H, _p(m_in),
                                         _p(out), _stream()), "smoes_attn_score_update")
    return out


def permute(topk_idx: torch.Tensor, E: int, x: Optional[torch.Tensor] = None):
    """Returns (expert_offsets [E+1], perm_token [T*k], perm_inv [T, k], x_perm or None)."""
    T, k = topk_idx.shape
    dev = topk_idx.device
    off = torch.empty(E + 1, dtype=torch.int32, device=dev)
    perm = torch.empty(T * k, dtype=torch.int32, device=dev)
    inv = torch.empty((T, k), dtype=torch.int32, device=dev)
    xp = None
    dt, d = SMOES_F32, 8
    if x is not None:
        d = x.shape[1]
        dt = _dtype_code(x)
        xp = torch.empty((T * k, d), dtype=x.dtype, device=dev)
    nbytes = lib().smoes_permute_workspace_size(T, E, k)
    ws = _workspace(nbytes, dev)
    _check(lib().smoes_permute(_p(topk_idx), T, E, k, _p(off), _p(perm), _p(inv), _p(x), dt, d, _p(xp),
                               _p(ws), nbytes, _stream()), "smoes_permute")
    return off, perm, inv, xp


# ---------------------------------------------------------------- whole layer

@dataclass
class LayerSpec:
    T: int
    d: int
    E: int
    k: int
    inter: int
    shared_inter: int
    n_bins: int
    n_batch: int
    act_dtype: int
    tau: float = 0.0
    beta: float = 0.99
    var_floor: float = 1e-6
    grad_scale: float = 1.0
    renorm_topk: bool = False
    update_stats: bool = False
    weights_packed: bool = False
    save_preact: bool = False
    check_inputs: bool = False

    def c(self) -> SmoesLayer:
        return SmoesLayer(self.T, self.d, self.E, self.k, self.inter, self.shared_inter, self.n_bins,
                          self.n_batch, self.act_dtype, self.tau, self.beta, self.var_floor,
                          self.grad_scale, int(self.renorm_topk), int(self.update_stats),
                          int(self.weights_packed), int(self.save_preact), int(self.check_inputs))


def workspace_bytes(spec: LayerSpec) -> int:
    desc = spec.c()
    return int(lib().smoes_workspace_bytes(ctypes.byref(desc)))


SMOES_BUF_H_ROUTED, SMOES_BUF_H_SHARED, SMOES_BUF_Y_ROUTED, SMOES_BUF_Y_SHARED, SMOES_BUF_CHECK_FLAGS = 0, 1, 2, 3, 4
SMOES_CHECK_MODALITY_ID, SMOES_CHECK_SAMPLE_OFFSETS, SMOES_CHECK_EXPERT_TO_BIN = 1, 2, 4


def workspace_buffer(spec: LayerSpec, workspace: torch.Tensor, which: int) -> torch.Tensor:
    """smoes_workspace_buffer: the bytes of one intermediate buffer of the
    forward (SMOES_BUF_*) as a uint8 view into `workspace`."""
    desc = spec.c()
    ptr, nb = c_void(), c_size()
    _check(lib().smoes_workspace_buffer(ctypes.byref(desc), _p(workspace), which, ctypes.byref(ptr),
                                        ctypes.byref(nb)), "smoes_workspace_buffer")
    off = (ptr.value or 0) - workspace.data_ptr()
    if nb.value == 0:
        return workspace[:0]
    if off < 0 or off + nb.value > workspace.numel():
        raise SmoesError(SMOES_ERR_WORKSPACE, "smoes_workspace_buffer")
    return workspace[off:off + nb.value]


def _layer_io(inputs, outputs=None) -> SmoesLayerIO:
    io = SmoesLayerIO()
    outputs = outputs or {}
    for name in _IO_FIELDS:
        if name == "stage_events":
            continue
        t = inputs.get(name) if name in inputs else outputs.get(name)
        setattr(io, name, None if t is None else _p(t).value)
    io.stage_events = None
    io.streams = None
    return io


def check_inputs(spec: LayerSpec, inputs: Dict[str, Optional[torch.Tensor]],
                 flags: Optional[torch.Tensor] = None) -> torch.Tensor:
    """smoes_check_inputs: the SMOES_CHECK_* bitmask of the device-resident
    inputs (modality_id, sample_offsets, expert_to_bin) as a device int32 [1]."""
    if flags is None:
        flags = torch.empty(1, dtype=torch.int32, device=inputs["expert_to_bin"].device)
    desc = spec.c()
    io = _layer_io(inputs)
    _check(lib().smoes_check_inputs(ctypes.byref(desc), ctypes.byref(io), _p(flags), _stream()),
           "smoes_check_inputs")
    return flags


SMOES_W13, SMOES_W2, SMOES_WS13, SMOES_WS2, SMOES_WGATE = 0, 1, 2, 3, 4
SMOES_W13T, SMOES_W2T, SMOES_WS13T, SMOES_WS2T = 5, 6, 7, 8
WEIGHT_NAMES = {"w13": SMOES_W13, "w2": SMOES_W2, "ws13": SMOES_WS13, "ws2": SMOES_WS2}


def pack_layer_inputs(spec: "LayerSpec", dev_in: Dict[str, Optional[torch.Tensor]]) -> None:
    """Add the packed forms of a bf16 layer's weights to dev_in: the expert
    weights replace w13/w2/ws13/ws2 and the router weights go to
    w_gate_packed (w_gate stays). spec.weights_packed must be set."""
    for name, which in WEIGHT_NAMES.items():
        if dev_in.get(name) is not None:
            dev_in[name] = pack_weights(spec, which, dev_in[name])
    dev_in["w_gate_packed"] = pack_weights(spec, SMOES_WGATE, dev_in["w_gate"])


def packed_weight_bytes(spec: LayerSpec, which: int) -> int:
    desc = spec.c()
    return int(lib().smoes_packed_weight_bytes(ctypes.byref(desc), which))


def pack_weights(spec: LayerSpec, which: int, src: torch.Tensor) -> torch.Tensor:
    """Pack one row-major bf16 expert weight tensor (device) into the
    fragment order read by the packed GEMMs; returns a new uint8 tensor."""
    n = packed_weight_bytes(spec, which)
    if n == 0:
        raise SmoesError(SMOES_ERR_ARG, "smoes_packed_weight_bytes")
    dst = torch.empty(n, dtype=torch.uint8, device=src.device)
    desc = spec.c()
    _check(lib().smoes_pack_weights(ctypes.byref(desc), which, _p(src), _p(dst), _stream()),
           "smoes_pack_weights")
    return dst


class Streams:
    """Caller-owned side streams for moe_forward (smoes_streams_create)."""

    def __init__(self):
        self.st = SmoesStreams()
        _check(lib().smoes_streams_create(ctypes.byref(self.st)), "smoes_streams_create")

    def close(self):
        if self.st is not None:
            torch.cuda.synchronize()
            lib().smoes_streams_destroy(ctypes.byref(self.st))
            self.st = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Events:
    """2 * SMOES_N_STAGES HIP events for the forward's stage timing: events
    2s and 2s + 1 bracket stage s on the stream that runs it."""

    def __init__(self, n: int = 2 * N_STAGES, only: Optional[int] = None):
        """only: make just the two events of that stage (the others stay NULL,
        so the forward records nothing for them)."""
        self.n = n
        self.arr = (c_void * n)()
        if only is None:
            self._own, self._own_n = self.arr, n
        else:
            self._own, self._own_n = (c_void * 2)(), 2
        _check(lib().smoes_events_create(self._own_n, self._own), "smoes_events_create")
        if only is not None:
            self.arr[2 * only], self.arr[2 * only + 1] = self._own[0], self._own[1]

    def stage_ms(self, stage: int) -> float:
        return self.elapsed_ms(2 * stage, 2 * stage + 1)

    def elapsed_ms(self, a: int, b: int) -> float:
        ms = c_float()
        _check(lib().smoes_event_elapsed_ms(self.arr[a], self.arr[b], ctypes.byref(ms)), "smoes_event_elapsed_ms")
        return float(ms.value)

    def close(self):
        if self.arr is not None:
            lib().smoes_events_destroy(self._own_n, self._own)
            self.arr = self._own = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def alloc_outputs(spec: LayerSpec, device, act_torch_dtype, want_logits=True, want_dlogits=True,
                  want_perm=True) -> Dict[str, torch.Tensor]:
    T, E, k = spec.T, spec.E, spec.k
    f = dict(dtype=torch.float32, device=device)
    i = dict(dtype=torch.int32, device=device)
    return {
        "logits": torch.empty((T, E), **f) if want_logits else None,
        "probs": torch.empty((T, E), **f),
        "topk_idx": torch.empty((T, k), **i),
        "topk_w": torch.empty((T, k), **f),
        "M": torch.empty((T, 2), **f),
        "mi_per_sample": torch.empty(spec.n_batch, **f),
        "loss": torch.empty(1, **f),
        "dlogits": torch.empty((T, E), **f) if want_dlogits else None,
        "expert_offsets": torch.empty(E + 1, **i) if want_perm else None,
        "perm_token": torch.empty(T * k, **i) if want_perm else None,
        "perm_inv": torch.empty((T, k), **i) if want_perm else None,
        "out": torch.empty((T, spec.d), dtype=act_torch_dtype, device=device),
    }


def backward_workspace_bytes(spec: LayerSpec) -> int:
    desc = spec.c()
    return int(lib().smoes_backward_workspace_bytes(ctypes.byref(desc)))


def pack_transposed_weights(spec: LayerSpec, dev_in: Dict[str, Optional[torch.Tensor]]) -> Dict[str, torch.Tensor]:
    """The transposed packed expert weights the backward reads (from the
    row-major bf16 weights in dev_in: w13, w2, ws13, ws2)."""
    out = {"w13t": pack_weights(spec, SMOES_W13T, dev_in["w13"]), "w2t": pack_weights(spec, SMOES_W2T, dev_in["w2"])}
    if spec.shared_inter > 0:
        out["ws13t"] = pack_weights(spec, SMOES_WS13T, dev_in["ws13"])
        out["ws2t"] = pack_weights(spec, SMOES_WS2T, dev_in["ws2"])
    return out


def moe_backward(spec: LayerSpec, inputs: Dict[str, Optional[torch.Tensor]],
                 outputs: Dict[str, Optional[torch.Tensor]], fwd_workspace: torch.Tensor,
                 packed_t: Optional[Dict[str, torch.Tensor]], dout: torch.Tensor,
                 dlogits_aux: Optional[torch.Tensor] = None, want_dw: bool = True,
                 grads: Optional[Dict[str, Optional[torch.Tensor]]] = None,
                 workspace: Optional[torch.Tensor] = None,
                 streams: Optional["Streams"] = None) -> Dict[str, torch.Tensor]:
    """smoes_moe_backward after moe_forward with the same inputs / outputs /
    workspace. `inputs` holds the layer's w13 / ws13 (packed when
    spec.weights_packed) and the float32 w_gate, and w2 / ws2 for fp32 layers
    and row-major bf16 layers; `packed_t` the transposed packed weights
    (pack_transposed_weights), needed for packed bf16 layers only (else None).
    Returns the gradients (dx, dw_gate, dbias, dz, dw, dw13, dw2, dws13, dws2;
    the expert weight gradients in the layer's dtype), written into `grads`
    when given (as returned by an earlier call), with `workspace` reused when
    given; `streams` (side streams) lets the router and shared-expert
    gradients of a packed bf16 layer run beside the routed ones."""
    desc = spec.c()
    io = SmoesLayerIO()
    for name in _IO_FIELDS:
        if name == "stage_events":
            continue
        t = inputs.get(name) if name in inputs else outputs.get(name)
        setattr(io, name, None if t is None else _p(t).value)
    io.stage_events = None
    io.streams = ctypes.cast(ctypes.byref(streams.st), c_void).value if streams is not None else None
    T, d, E, k, I, SI = spec.T, spec.d, spec.E, spec.k, spec.inter, spec.shared_inter
    dev = dout.device
    wdt = torch.bfloat16 if spec.act_dtype == SMOES_BF16 else torch.float32
    pt = packed_t or {}
    g = grads if grads is not None else {
         "dx": torch.empty((T, d), dtype=torch.float32, device=dev),
         "dw_gate": torch.empty((E, d), dtype=torch.float32, device=dev),
         "dbias": torch.empty(E, dtype=torch.float32, device=dev),
         "dz": torch.empty((T, E), dtype=torch.float32, device=dev),
         "dw": torch.empty((T, k), dtype=torch.float32, device=dev) if want_dw else None,
         "dw13": torch.empty((E, 2 * I, d), dtype=wdt, device=dev),
         "dw2": torch.empty((E, d, I), dtype=wdt, device=dev),
         "dws13": torch.empty((2 * SI, d), dtype=wdt, device=dev) if SI > 0 else None,
         "dws2": torch.empty((d, SI), dtype=wdt, device=dev) if SI > 0 else None}
    G = SmoesLayerGrads()
    for name in _GRAD_FIELDS:
        setattr(G, name, None if g[name] is None else _p(g[name]).value)
    nbytes = int(lib().smoes_backward_workspace_bytes(ctypes.byref(desc)))
    if workspace is not None and workspace.numel() >= nbytes:
        ws, nbytes = workspace, workspace.numel()
    else:
        ws = _workspace(nbytes, dev)
    _check(lib().smoes_moe_backward(ctypes.byref(desc), ctypes.byref(io), _p(pt.get("w13t")), _p(pt.get("w2t")),
                                    _p(pt.get("ws13t")), _p(pt.get("ws2t")), _p(dout), _p(dlogits_aux),
                                    ctypes.byref(G), _p(fwd_workspace), fwd_workspace.numel(), _p(ws), nbytes,
                                    _stream()), "smoes_moe_backward")
    return g


def moe_forward(spec: LayerSpec, inputs: Dict[str, Optional[torch.Tensor]],
                outputs: Dict[str, Optional[torch.Tensor]], workspace: torch.Tensor,
                events: Optional[Events] = None,
                streams: Optional[Streams] = None) -> Dict[str, Optional[torch.Tensor]]:
    """One layer forward. `inputs` holds x, modality_id, sample_offsets, w_gate,
    logit_bias, expert_to_bin, w13, w2, ws13, ws2, gauss_n, gauss_smu, gauss_ssig
    (the Gaussian state is updated in place when spec.update_stats)."""
    desc = spec.c()
    io = SmoesLayerIO()
    for name in _IO_FIELDS:
        if name == "stage_events":
            continue
        t = inputs.get(name) if name in inputs else outputs.get(name)
        setattr(io, name, None if t is None else _p(t).value)
    io.stage_events = ctypes.cast(events.arr, c_void).value if events is not None else None
    io.streams = ctypes.cast(ctypes.byref(streams.st), c_void).value if streams is not None else None
    _check(lib().smoes_moe_forward(ctypes.byref(desc), ctypes.byref(io), _p(workspace),
                                   workspace.numel(), _stream()), "smoes_moe_forward")
    return outputs
