"""The C ABI library: it loads, exports every function include/smoes.h
declares, and rejects bad arguments on the host before touching the GPU.
None of these calls launches a kernel, so they run without a GPU."""
import ctypes
import os

import pytest

from paper_2604_23996_amd import smoes as S

pytestmark = pytest.mark.skipif(not os.path.exists(S.LIB_PATH), reason="libsmoes.so not built")

FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: every call below fails validation first


def test_exports_every_declared_function():
    names = S.header_functions()
    assert {"smoes_route", "smoes_modality_score", "smoes_mi_loss", "smoes_permute",
            "smoes_moe_forward", "smoes_workspace_bytes"} <= set(names)
    L = S.lib()
    for n in names:
        assert hasattr(L, n), n


def test_status_strings():
    for code in (0, -1, -2, -3, -4, -5):
        s = S.status_string(code)
        assert s.startswith("SMOES_")
    assert "unknown" in S.status_string(-99)


def test_route_argument_checks():
    L = S.lib()
    # null x
    assert L.smoes_route(None, 1, 10, 64, FAKE, None, 8, 2, 0, None, FAKE, FAKE, FAKE, FAKE, 1 << 20, None) == S.SMOES_ERR_ARG
    # bad dtype
    assert L.smoes_route(FAKE, 7, 10, 64, FAKE, None, 8, 2, 0, None, FAKE, FAKE, FAKE, FAKE, 1 << 20, None) == S.SMOES_ERR_ARG
    # d not a multiple of 8, k > E, k > K_MAX, E > E_MAX
    for (d, E, k) in ((63, 8, 2), (64, 8, 9), (64, 64, 17), (64, 257, 2), (0, 8, 2)):
        assert L.smoes_route(FAKE, 1, 10, d, FAKE, None, E, k, 0, None, FAKE, FAKE, FAKE, FAKE, 1 << 20, None) == S.SMOES_ERR_SHAPE
    # workspace too small (bf16 needs the split router weights)
    need = L.smoes_route_workspace_size(10, 64, 8, 1)
    assert need > 0
    assert L.smoes_route(FAKE, 1, 10, 64, FAKE, None, 8, 2, 0, None, FAKE, FAKE, FAKE, FAKE, need - 1, None) == S.SMOES_ERR_WORKSPACE
    # T = 0 is a no-op success, even with null buffers
    assert L.smoes_route(None, 1, 0, 64, None, None, 8, 2, 0, None, None, None, None, None, 0, None) == S.SMOES_OK


def test_modality_argument_checks():
    L = S.lib()
    ws = L.smoes_modality_workspace_size(10, 64)
    args = lambda **kw: dict(dict(x=FAKE, dt=1, T=10, d=64, mid=FAKE, n=FAKE, smu=FAKE, ssig=FAKE,
                                   upd=1, beta=0.99, tau=0.0, vf=1e-6, M=FAKE, ws=FAKE, wsb=ws), **kw)
    call = lambda a: L.smoes_modality_score(a["x"], a["dt"], a["T"], a["d"], a["mid"], a["n"], a["smu"],
                                            a["ssig"], a["upd"], a["beta"], a["tau"], a["vf"], a["M"],
                                            a["ws"], a["wsb"], None)
    assert call(args(mid=None)) == S.SMOES_ERR_ARG  # update needs modality ids
    assert call(args(beta=1.5)) == S.SMOES_ERR_ARG
    assert call(args(vf=-1.0)) == S.SMOES_ERR_ARG
    assert call(args(d=20)) == S.SMOES_ERR_SHAPE
    assert call(args(wsb=ws - 1)) == S.SMOES_ERR_WORKSPACE
    assert call(args(M=None)) == S.SMOES_ERR_ARG
    assert call(args(T=0, x=None)) == S.SMOES_OK


def test_mi_argument_checks():
    L = S.lib()
    ws = L.smoes_mi_workspace_size(10, 8, 2, 2)
    call = lambda E=8, nb=2, bins=2, off=FAKE, wsb=ws, probs=FAKE: L.smoes_mi_loss(
        probs, FAKE, 10, E, off, nb, FAKE, bins, 1.0, FAKE, FAKE, None, FAKE, wsb, None)
    assert call(bins=3) == S.SMOES_ERR_SHAPE  # E % n_bins
    assert call(bins=65, E=130) == S.SMOES_ERR_SHAPE
    assert call(nb=0) == S.SMOES_ERR_SHAPE
    assert call(off=None) == S.SMOES_ERR_SHAPE  # several samples need offsets
    assert call(probs=None) == S.SMOES_ERR_ARG
    assert call(wsb=ws - 1) == S.SMOES_ERR_WORKSPACE


def test_permute_argument_checks():
    L = S.lib()
    ws = L.smoes_permute_workspace_size(10, 8, 2)
    call = lambda E=8, k=2, idx=FAKE, xp=None, x=FAKE, d=64, wsb=ws: L.smoes_permute(
        idx, 10, E, k, FAKE, FAKE, FAKE, x, 1, d, xp, FAKE, wsb, None)
    assert call(k=9) == S.SMOES_ERR_SHAPE
    assert call(idx=None) == S.SMOES_ERR_ARG
    assert call(xp=FAKE, x=None) == S.SMOES_ERR_ARG
    assert call(xp=FAKE, d=12) == S.SMOES_ERR_SHAPE
    assert call(wsb=ws - 1) == S.SMOES_ERR_WORKSPACE


def _spec(**kw):
    base = dict(T=300, d=128, E=16, k=4, inter=96, shared_inter=96, n_bins=4, n_batch=2, act_dtype=1)
    base.update(kw)
    return S.LayerSpec(**base)


def test_layer_workspace_and_checks():
    L = S.lib()
    assert S.workspace_bytes(_spec()) > 0
    for bad in (dict(inter=100), dict(inter=0), dict(shared_inter=24), dict(n_bins=3), dict(k=17),
                dict(d=100), dict(act_dtype=5), dict(beta=2.0)):
        assert S.workspace_bytes(_spec(**bad)) == 0, bad
    # operands past 32-bit byte offsets are refused: routed activations, x, and the shared block
    assert S.workspace_bytes(_spec(T=1 << 17, d=2048, k=8, inter=1408)) == 0
    assert S.workspace_bytes(_spec(T=1 << 18, d=4096, k=1, inter=512, shared_inter=0)) == 0
    assert S.workspace_bytes(_spec(T=1 << 16, d=2048, k=2, inter=512, shared_inter=16384)) == 0
    assert S.workspace_bytes(_spec(T=1 << 16, d=2048, k=2, inter=512, shared_inter=2816)) > 0
    desc = _spec().c()
    io = S.SmoesLayerIO()
    assert L.smoes_moe_forward(ctypes.byref(desc), ctypes.byref(io), FAKE, 1 << 30, None) == S.SMOES_ERR_ARG
    assert L.smoes_moe_forward(None, ctypes.byref(io), FAKE, 1 << 30, None) == S.SMOES_ERR_ARG
    # every required pointer present but the workspace too small
    for name in ("x", "w_gate", "expert_to_bin", "w13", "w2", "ws13", "ws2", "gauss_n", "gauss_smu",
                 "gauss_ssig", "probs", "topk_idx", "topk_w", "M", "mi_per_sample", "loss", "out",
                 "sample_offsets"):
        setattr(io, name, 0x1000)
    need = S.workspace_bytes(_spec())
    assert L.smoes_moe_forward(ctypes.byref(desc), ctypes.byref(io), FAKE, need - 1, None) == S.SMOES_ERR_WORKSPACE
    # side streams given but incomplete
    st = S.SmoesStreams()
    io.streams = ctypes.cast(ctypes.byref(st), ctypes.c_void_p).value
    assert L.smoes_moe_forward(ctypes.byref(desc), ctypes.byref(io), FAKE, need, None) == S.SMOES_ERR_ARG
    io.streams = None
    # shared experts declared but weights missing
    io.ws13 = None
    assert L.smoes_moe_forward(ctypes.byref(desc), ctypes.byref(io), FAKE, need, None) == S.SMOES_ERR_ARG
    # T = 0 is a no-op
    d0 = _spec(T=0).c()
    assert L.smoes_moe_forward(ctypes.byref(d0), ctypes.byref(S.SmoesLayerIO()), None, 0, None) == S.SMOES_OK


def test_struct_layout_matches_header():
    # smoes_layer: int64 + 8 int + 4 float + 5 int = 76 bytes, padded to 80; io: 28 pointers
    assert ctypes.sizeof(S.SmoesLayer) == 80
    assert ctypes.sizeof(S.SmoesLayerIO) == 28 * 8
    assert ctypes.sizeof(S.SmoesStreams) == 6 * 8
    text = open(S.HEADER_PATH).read()
    import re
    lay = text[text.index("typedef struct smoes_layer {"):text.index("} smoes_layer;")]
    lay = re.sub(r"/\*.*?\*/", "", lay, flags=re.S)
    names = re.findall(r"(?:int64_t|int|float)\s+([A-Za-z_0-9]+);", lay)
    assert names == [f[0] for f in S.SmoesLayer._fields_]
    io_block = text[text.index("typedef struct smoes_layer_io"):text.index("} smoes_layer_io;")]
    io_block = re.sub(r"/\*.*?\*/", "", io_block, flags=re.S)
    fields = re.findall(r"\*\s*(?:const\s*\*\s*)?([A-Za-z_0-9]+);", io_block)
    assert fields == S._IO_FIELDS + ["streams"]


def test_backward_struct_and_host_checks():
    text = open(S.HEADER_PATH).read()
    import re
    blk = text[text.index("typedef struct smoes_layer_grads"):text.index("} smoes_layer_grads;")]
    blk = re.sub(r"/\*.*?\*/", "", blk, flags=re.S)
    assert re.findall(r"\*\s*([A-Za-z_0-9]+);", blk) == S._GRAD_FIELDS
    assert ctypes.sizeof(S.SmoesLayerGrads) == 9 * 8
    L = S.lib()
    spec = _spec(d=128, inter=96, shared_inter=48, weights_packed=True)
    desc = spec.c()
    n = L.smoes_backward_workspace_bytes(ctypes.byref(desc))
    assert n > 0
    bad = _spec().c()
    bad.save_preact = 3
    assert L.smoes_backward_workspace_bytes(ctypes.byref(bad)) == 0
    kept = _spec(d=128, inter=96, shared_inter=48, weights_packed=True, save_preact=True).c()
    assert 0 < L.smoes_backward_workspace_bytes(ctypes.byref(kept)) < n
    io = S.SmoesLayerIO()
    G = S.SmoesLayerGrads()
    args = lambda d_: (ctypes.byref(d_), ctypes.byref(io), FAKE, FAKE, FAKE, FAKE, FAKE, None, ctypes.byref(G),
                       FAKE, 1 << 40, FAKE, 1 << 40, None)
    # float32 layers and row-major weights are not implemented; nothing is launched
    assert L.smoes_moe_backward(*args(_spec(act_dtype=0).c())) == S.SMOES_ERR_ARG
    assert L.smoes_moe_backward(*args(_spec(weights_packed=False).c())) == S.SMOES_ERR_ARG
    # missing pointers and short workspaces are rejected before any launch
    assert L.smoes_moe_backward(*args(desc)) == S.SMOES_ERR_ARG
    assert L.smoes_moe_backward(ctypes.byref(desc), None, FAKE, FAKE, FAKE, FAKE, FAKE, None, ctypes.byref(G),
                                FAKE, 1 << 40, FAKE, 1 << 40, None) == S.SMOES_ERR_ARG
    for name in S._IO_FIELDS:
        if name in ("x", "w13", "ws13", "w_gate", "probs", "topk_idx", "topk_w"):
            setattr(io, name, FAKE.value)
    for name in S._GRAD_FIELDS:
        setattr(G, name, FAKE.value)
    assert L.smoes_moe_backward(ctypes.byref(desc), ctypes.byref(io), FAKE, FAKE, FAKE, FAKE, FAKE, None,
                                ctypes.byref(G), FAKE, 16, FAKE, 1 << 40, None) == S.SMOES_ERR_WORKSPACE
    assert L.smoes_moe_backward(ctypes.byref(desc), ctypes.byref(io), FAKE, FAKE, FAKE, FAKE, FAKE, None,
                                ctypes.byref(G), FAKE, 1 << 40, FAKE, n - 1, None) == S.SMOES_ERR_WORKSPACE
    # the dX GEMM's A operand must stay inside 32-bit byte offsets
    big = _spec(T=1 << 17, d=64, E=8, k=8, inter=512, shared_inter=0, weights_packed=True).c()
    assert L.smoes_workspace_bytes(ctypes.byref(big)) > 0  # the forward accepts it
    assert L.smoes_moe_backward(*args(big)) == S.SMOES_ERR_SHAPE


def test_packed_weight_sizes_and_checks():
    L = S.lib()
    spec = _spec(d=128, inter=96, shared_inter=48)
    # w13: E experts of 2*32*ceil(inter/32) rows x ceil(d/16) slices x 128 bf16 per slice-group
    # pairs of 16-row groups x 32-wide K slices x 1024 bf16
    assert S.packed_weight_bytes(spec, S.SMOES_W13) == 16 * (2 * 3) * (128 // 32) * 1024 * 2
    assert S.packed_weight_bytes(spec, S.SMOES_W2) == 16 * (128 // 32) * (96 // 32) * 1024 * 2
    assert S.packed_weight_bytes(spec, S.SMOES_WS13) == (2 * 2) * (128 // 32) * 1024 * 2
    assert S.packed_weight_bytes(spec, S.SMOES_WS2) == (128 // 32) * (-(-48 // 32)) * 1024 * 2
    # router weights: 3 bf16 terms x ceil(E/16)*16 experts x ceil(d/32)*32
    assert S.packed_weight_bytes(spec, S.SMOES_WGATE) == 3 * 16 * 128 * 2
    # transposed forms for the backward: W13^T has d rows over 2 inter, W2^T inter rows over d
    assert S.packed_weight_bytes(spec, S.SMOES_W13T) == 16 * (128 // 32) * (192 // 32) * 1024 * 2
    assert S.packed_weight_bytes(spec, S.SMOES_W2T) == 16 * (96 // 32) * (128 // 32) * 1024 * 2
    assert S.packed_weight_bytes(spec, S.SMOES_WS13T) == (128 // 32) * (96 // 32) * 1024 * 2
    assert S.packed_weight_bytes(spec, S.SMOES_WS2T) == (48 // 32 + 1) * (128 // 32) * 1024 * 2
    assert S.packed_weight_bytes(spec, 9) == 0 and S.packed_weight_bytes(spec, -1) == 0
    assert S.packed_weight_bytes(_spec(shared_inter=0), S.SMOES_WS13) == 0
    assert S.packed_weight_bytes(_spec(shared_inter=0), S.SMOES_WS2T) == 0
    desc = spec.c()
    assert L.smoes_pack_weights(ctypes.byref(desc), S.SMOES_W13, None, FAKE, None) == S.SMOES_ERR_ARG
    assert L.smoes_pack_weights(ctypes.byref(desc), 9, FAKE, FAKE, None) == S.SMOES_ERR_ARG
    f32 = _spec(act_dtype=0).c()
    assert L.smoes_pack_weights(ctypes.byref(f32), S.SMOES_W13, FAKE, FAKE, None) == S.SMOES_ERR_ARG
    # packed weights are a bf16 layout; save_preact is 0 or 1
    assert S.workspace_bytes(_spec(act_dtype=0, weights_packed=True)) == 0
    bad = _spec().c()
    bad.save_preact = 2
    assert L.smoes_workspace_bytes(ctypes.byref(bad)) == 0
    # keeping the pre-activations is a packed bf16 feature, and it grows the workspace
    assert S.workspace_bytes(_spec(save_preact=True)) == 0
    assert S.workspace_bytes(_spec(weights_packed=True, save_preact=True)) > S.workspace_bytes(_spec(weights_packed=True))


def test_workspace_buffers_lie_inside_the_workspace():
    """smoes_workspace_buffer is host arithmetic: every buffer of the forward
    lies inside the workspace the size query asks for, with the documented
    byte size, and the buffers do not overlap."""
    L = S.lib()
    for sh, dt in ((48, S.SMOES_BF16), (0, S.SMOES_F32)):
        spec = _spec(d=128, inter=96, shared_inter=sh, act_dtype=dt)
        desc = spec.c()
        n = L.smoes_workspace_bytes(ctypes.byref(desc))
        base = 1 << 40
        es = 2 if dt == S.SMOES_BF16 else 4
        R = spec.T * spec.k
        want = {S.SMOES_BUF_H_ROUTED: es * R * spec.inter, S.SMOES_BUF_H_SHARED: es * spec.T * sh,
                S.SMOES_BUF_Y_ROUTED: es * R * spec.d, S.SMOES_BUF_Y_SHARED: es * spec.T * spec.d if sh else 0,
                S.SMOES_BUF_CHECK_FLAGS: 4}
        spans = []
        for which, nbytes in want.items():
            ptr, nb = ctypes.c_void_p(), ctypes.c_size_t()
            assert L.smoes_workspace_buffer(ctypes.byref(desc), ctypes.c_void_p(base), which, ctypes.byref(ptr),
                                            ctypes.byref(nb)) == S.SMOES_OK
            assert nb.value == nbytes
            assert base <= ptr.value and ptr.value + nb.value <= base + n
            if nb.value:
                spans.append((ptr.value, ptr.value + nb.value))
        spans.sort()
        assert all(a[1] <= b[0] for a, b in zip(spans, spans[1:]))
        ptr, nb = ctypes.c_void_p(), ctypes.c_size_t()
        assert L.smoes_workspace_buffer(ctypes.byref(desc), ctypes.c_void_p(base), 9, ctypes.byref(ptr),
                                        ctypes.byref(nb)) == S.SMOES_ERR_ARG
        assert L.smoes_workspace_buffer(ctypes.byref(desc), None, 0, ctypes.byref(ptr),
                                        ctypes.byref(nb)) == S.SMOES_ERR_ARG


def test_check_inputs_host_errors():
    L = S.lib()
    desc = _spec().c()
    io = S.SmoesLayerIO()
    # no expert_to_bin, no flags, no io: rejected on the host, nothing launched
    assert L.smoes_check_inputs(ctypes.byref(desc), ctypes.byref(io), FAKE, None) == S.SMOES_ERR_ARG
    io.expert_to_bin = FAKE.value
    assert L.smoes_check_inputs(ctypes.byref(desc), ctypes.byref(io), None, None) == S.SMOES_ERR_ARG
    assert L.smoes_check_inputs(ctypes.byref(desc), None, FAKE, None) == S.SMOES_ERR_ARG
    bad = _spec().c()
    bad.check_inputs = 2
    assert L.smoes_workspace_bytes(ctypes.byref(bad)) == 0
    assert L.smoes_check_inputs(ctypes.byref(bad), ctypes.byref(io), FAKE, None) == S.SMOES_ERR_ARG
