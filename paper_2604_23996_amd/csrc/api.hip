// C ABI of the SMoES layer: argument validation, workspace layout and the
// launch sequence on the caller's stream. No call allocates device memory or
// synchronises the host.
#include <stdio.h>

#include "smoes.h"
#include "common.h"
#include "kernels.h"

using namespace smoes;

namespace {

constexpr size_t kAlign = 256;

inline hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

// Carves aligned sub-buffers out of the caller's workspace.
struct Carver {
    char* base;
    size_t used = 0;
    explicit Carver(void* p) : base(static_cast<char*>(p)) {
        // align the start inside the workspace
        const uintptr_t a = reinterpret_cast<uintptr_t>(base);
        used = (kAlign - (a % kAlign)) % kAlign;
    }
    void* take(size_t bytes) {
        void* p = base + used;
        used += align_up(bytes, kAlign);
        return p;
    }
};

inline int hip_status(hipError_t e) { return e == hipSuccess ? SMOES_OK : SMOES_ERR_HIP; }

bool dtype_ok(int dt) { return dt == SMOES_F32 || dt == SMOES_BF16; }

int check_router_shape(int64_t T, int d, int E, int k) {
    if (T < 0 || d < 1 || d > SMOES_D_MAX || (d % 8) != 0) return SMOES_ERR_SHAPE;
    if (E < 1 || E > SMOES_E_MAX) return SMOES_ERR_SHAPE;
    if (k < 1 || k > E || k > SMOES_K_MAX) return SMOES_ERR_SHAPE;
    return SMOES_OK;
}

int check_mi_shape(int64_t T, int E, int n_batch, int n_bins) {
    if (T < 0 || E < 1 || E > SMOES_E_MAX) return SMOES_ERR_SHAPE;
    if (n_bins < 1 || n_bins > SMOES_BINS_MAX || (E % n_bins) != 0) return SMOES_ERR_SHAPE;
    if (n_batch < 1) return SMOES_ERR_SHAPE;
    return SMOES_OK;
}

// Total workspace of the standalone entry points (max alignment slack included).
size_t route_ws(int64_t T, int d, int E, int x_dtype) {
    return router_workspace_bytes(T, d, E, x_dtype) + 2 * kAlign;
}
size_t modality_ws(int64_t T, int d) { return modality_workspace_bytes(T, d) + 2 * kAlign; }
size_t mi_ws(int64_t T, int E, int n_batch, int n_bins) {
    return mi_workspace_bytes(T, E, n_batch, n_bins) + 2 * kAlign;
}
size_t permute_ws(int64_t T, int E, int k) { return permute_workspace_bytes(T, E, k) + 2 * kAlign; }

// Stage s timing: start event 2 s, end event 2 s + 1 (either may be NULL).
hipError_t record(void* const* ev, int idx, hipStream_t st) {
    if (ev == nullptr || ev[idx] == nullptr) return hipSuccess;
    return hipEventRecord(static_cast<hipEvent_t>(ev[idx]), st);
}

}  // namespace

extern "C" {

const char* smoes_status_string(int status) {
    switch (status) {
        case SMOES_OK: return "SMOES_OK: success";
        case SMOES_ERR_ARG: return "SMOES_ERR_ARG: a required pointer is NULL or a scalar/dtype is invalid";
        case SMOES_ERR_SHAPE: return "SMOES_ERR_SHAPE: inconsistent or unsupported sizes";
        case SMOES_ERR_WORKSPACE: return "SMOES_ERR_WORKSPACE: workspace smaller than the size query";
        case SMOES_ERR_HIP: return "SMOES_ERR_HIP: a HIP launch or runtime call failed";
        case SMOES_ERR_SCRATCH:
            return "SMOES_ERR_SCRATCH: the problem needs more scratch than the fixed device array of the "
                   "no-allocation entry point holds";
        default: return "SMOES: unknown status code";
    }
}

const char* smoes_version(void) { return "smoes-gfx950 0.1.0"; }

size_t smoes_route_workspace_size(int64_t T, int d, int E, int x_dtype) {
    return route_ws(T, d, E, x_dtype);
}

int smoes_route(const void* x, int x_dtype, int64_t T, int d, const float* w_gate,
                const float* logit_bias, int E, int k, int renorm_topk, float* logits, float* probs,
                int32_t* topk_idx, float* topk_w, void* workspace, size_t workspace_bytes,
                void* stream) {
    if (!dtype_ok(x_dtype)) return SMOES_ERR_ARG;
    int st = check_router_shape(T, d, E, k);
    if (st != SMOES_OK) return st;
    // bf16 activations are read through a buffer descriptor with 32-bit byte offsets
    if (x_dtype == SMOES_BF16 && T * d * 2 > INT32_MAX) return SMOES_ERR_SHAPE;
    if (T == 0) return SMOES_OK;
    if (x == nullptr || w_gate == nullptr || probs == nullptr || topk_idx == nullptr || topk_w == nullptr)
        return SMOES_ERR_ARG;
    const size_t need = route_ws(T, d, E, x_dtype);
    if (x_dtype == SMOES_BF16 && (workspace == nullptr || workspace_bytes < need)) return SMOES_ERR_WORKSPACE;
    Carver c(workspace);
    void* ws = x_dtype == SMOES_BF16 ? c.take(router_workspace_bytes(T, d, E, x_dtype)) : nullptr;
    return hip_status(launch_route(x, x_dtype, T, d, w_gate, nullptr, logit_bias, E, k, renorm_topk ? 1 : 0,
                                   logits, probs, topk_idx, topk_w, ws, as_stream(stream)));
}

size_t smoes_modality_workspace_size(int64_t T, int d) { return modality_ws(T, d); }

int smoes_modality_score(const void* x, int x_dtype, int64_t T, int d, const uint8_t* modality_id,
                         float* gauss_n, float* gauss_smu, float* gauss_ssig, int update, float beta,
                         float tau, float var_floor, float* M, void* workspace,
                         size_t workspace_bytes, void* stream) {
    if (!dtype_ok(x_dtype)) return SMOES_ERR_ARG;
    if (T < 0 || d < 1 || d > SMOES_D_MAX || (d % 8) != 0) return SMOES_ERR_SHAPE;
    if (!(beta >= 0.0f && beta <= 1.0f) || !(var_floor >= 0.0f) || tau != tau) return SMOES_ERR_ARG;
    if (T == 0) return SMOES_OK;
    if (x == nullptr || gauss_n == nullptr || gauss_smu == nullptr || gauss_ssig == nullptr || M == nullptr)
        return SMOES_ERR_ARG;
    if (update && modality_id == nullptr) return SMOES_ERR_ARG;
    if (workspace == nullptr || workspace_bytes < modality_ws(T, d)) return SMOES_ERR_WORKSPACE;
    Carver c(workspace);
    void* ws = c.take(modality_workspace_bytes(T, d));
    return hip_status(launch_modality(x, x_dtype, T, d, modality_id, gauss_n, gauss_smu, gauss_ssig,
                                      update ? 1 : 0, beta, tau, var_floor, M, ws, as_stream(stream)));
}

size_t smoes_mi_workspace_size(int64_t T, int E, int n_batch, int n_bins) {
    return mi_ws(T, E, n_batch, n_bins);
}

int smoes_mi_loss(const float* probs, const float* M, int64_t T, int E, const int32_t* sample_offsets,
                  int n_batch, const int32_t* expert_to_bin, int n_bins, float grad_scale,
                  float* mi_per_sample, float* loss, float* dlogits, void* workspace,
                  size_t workspace_bytes, void* stream) {
    int st = check_mi_shape(T, E, n_batch, n_bins);
    if (st != SMOES_OK) return st;
    if (sample_offsets == nullptr && n_batch != 1) return SMOES_ERR_SHAPE;
    if (grad_scale != grad_scale) return SMOES_ERR_ARG;
    if (probs == nullptr || M == nullptr || expert_to_bin == nullptr || mi_per_sample == nullptr ||
        loss == nullptr)
        return SMOES_ERR_ARG;
    if (workspace == nullptr || workspace_bytes < mi_ws(T, E, n_batch, n_bins)) return SMOES_ERR_WORKSPACE;
    Carver c(workspace);
    void* ws = c.take(mi_workspace_bytes(T, E, n_batch, n_bins));
    // T == 0 still defines the outputs (every I_i = 0, loss = 0)
    return hip_status(launch_mi(probs, M, T, E, sample_offsets, n_batch, expert_to_bin, n_bins,
                                grad_scale, mi_per_sample, loss, T > 0 ? dlogits : nullptr, ws,
                                as_stream(stream)));
}

size_t smoes_binning_workspace_size(int64_t T, int E, int n_bins) {
    if (check_mi_shape(T, E, 1, n_bins) != SMOES_OK) return 0;
    return binning_workspace_bytes(T, E, n_bins) + 2 * kAlign;
}

int smoes_binning(const float* probs, const int32_t* topk_idx, const uint8_t* modality_id, int64_t T, int E,
                  int k, const int32_t* expert_to_bin, int n_bins, float beta, double* load_ema,
                  int32_t* counts, double* f_spec, int32_t* expert_to_bin_next, float grad_scale,
                  float* bal_loss, float* dlogits, int accumulate, float* msi, void* workspace,
                  size_t workspace_bytes, void* stream) {
    int st = check_mi_shape(T, E, 1, n_bins);
    if (st != SMOES_OK) return st;
    if (k < 1 || k > E || k > SMOES_K_MAX) return SMOES_ERR_SHAPE;
    if (!(beta >= 0.0f && beta <= 1.0f) || (accumulate != 0 && accumulate != 1)) return SMOES_ERR_ARG;
    if (expert_to_bin == nullptr) return SMOES_ERR_ARG;
    if (T > 0 && (probs == nullptr || topk_idx == nullptr || modality_id == nullptr)) return SMOES_ERR_ARG;
    if (expert_to_bin_next != nullptr && expert_to_bin_next == expert_to_bin) return SMOES_ERR_ARG;
    if (workspace == nullptr || workspace_bytes < smoes_binning_workspace_size(T, E, n_bins))
        return SMOES_ERR_WORKSPACE;
    Carver c(workspace);
    void* ws = c.take(binning_workspace_bytes(T, E, n_bins));
    return hip_status(launch_binning(probs, topk_idx, modality_id, T, E, k, expert_to_bin, n_bins, beta, load_ema,
                                     counts, f_spec, expert_to_bin_next, grad_scale, bal_loss, dlogits, accumulate,
                                     msi, ws, as_stream(stream)));
}

// ------------------------------------------------------------------ GMM estimator

size_t smoes_gmm_workspace_size(int64_t T, int d, int K) {
    if (T < 0 || d < 1 || d > SMOES_D_MAX || (d % 8) != 0 || K < 1 || K > SMOES_GMM_K_MAX) return 0;
    return gmm_workspace_bytes(T, d, K) + 2 * kAlign;
}

int smoes_gmm_modality_score(const void* x, int x_dtype, int64_t T, int d, int K, const uint8_t* modality_id,
                             float* gmm_n, float* gmm_smu, float* gmm_ssig, int update, float beta, float tau,
                             float var_floor, float* M, float* resp, void* workspace, size_t workspace_bytes,
                             void* stream) {
    if (!dtype_ok(x_dtype)) return SMOES_ERR_ARG;
    if (T < 0 || d < 1 || d > SMOES_D_MAX || (d % 8) != 0 || K < 1 || K > SMOES_GMM_K_MAX) return SMOES_ERR_SHAPE;
    if (!(beta >= 0.0f && beta <= 1.0f) || !(var_floor >= 0.0f) || tau != tau) return SMOES_ERR_ARG;
    if (update != 0 && update != 1) return SMOES_ERR_ARG;
    if (T == 0) return SMOES_OK;
    if (x == nullptr || gmm_n == nullptr || gmm_smu == nullptr || gmm_ssig == nullptr || M == nullptr)
        return SMOES_ERR_ARG;
    if ((update || resp != nullptr) && modality_id == nullptr) return SMOES_ERR_ARG;
    if (workspace == nullptr || workspace_bytes < smoes_gmm_workspace_size(T, d, K)) return SMOES_ERR_WORKSPACE;
    Carver c(workspace);
    void* ws = c.take(gmm_workspace_bytes(T, d, K));
    return hip_status(launch_gmm(x, x_dtype, T, d, K, modality_id, gmm_n, gmm_smu, gmm_ssig, update, beta, tau,
                                 var_floor, M, resp, ws, as_stream(stream)));
}

// ------------------------------------------------------------------ attention-accumulated score

int smoes_attn_score_init(const uint8_t* modality_id, int64_t T, float* M, void* stream) {
    if (T < 0) return SMOES_ERR_SHAPE;
    if (T > 0 && (modality_id == nullptr || M == nullptr)) return SMOES_ERR_ARG;
    return hip_status(launch_attn_init(modality_id, T, M, as_stream(stream)));
}

int smoes_attention_scores(const void* q, const void* k, const void* v, int64_t T, int n_heads,
                           int n_kv_heads, int head_dim, const int32_t* sample_offsets, int n_batch,
                           const float* m_in, float scale, void* o, float* m_heads, void* stream) {
    if (T < 0 || n_batch < 1) return SMOES_ERR_SHAPE;
    if (n_heads < 1 || n_heads > 65535 || n_kv_heads < 1 || (n_heads % n_kv_heads) != 0) return SMOES_ERR_SHAPE;
    if (head_dim != 64 && head_dim != 128) return SMOES_ERR_SHAPE;
    if (T * n_heads * head_dim * 2 > INT32_MAX) return SMOES_ERR_SHAPE;
    if (scale != scale) return SMOES_ERR_ARG;
    if (T > 0 && (q == nullptr || k == nullptr || v == nullptr || sample_offsets == nullptr || m_in == nullptr ||
                  o == nullptr || m_heads == nullptr))
        return SMOES_ERR_ARG;
    const float sc = scale > 0.0f ? scale : 1.0f / sqrtf(static_cast<float>(head_dim));
    return hip_status(launch_attention(q, k, v, T, n_heads, n_kv_heads, head_dim, sample_offsets, n_batch, m_in,
                                       sc, o, m_heads, as_stream(stream)));
}

int smoes_attn_score_update(const void* x, const void* x_attn, int act_dtype, int64_t T, int d,
                            const float* m_heads, int n_heads, const float* m_in, float* m_out,
                            void* stream) {
    if (!dtype_ok(act_dtype)) return SMOES_ERR_ARG;
    if (T < 0 || d < 1 || d > SMOES_D_MAX || (d % 8) != 0 || n_heads < 1) return SMOES_ERR_SHAPE;
    if (T > 0 && (x == nullptr || x_attn == nullptr || m_heads == nullptr || m_in == nullptr || m_out == nullptr))
        return SMOES_ERR_ARG;
    return hip_status(launch_attn_update(x, x_attn, act_dtype, T, d, m_heads, n_heads, m_in, m_out,
                                         as_stream(stream)));
}

size_t smoes_permute_workspace_size(int64_t T, int E, int k) { return permute_ws(T, E, k); }

int smoes_permute(const int32_t* topk_idx, int64_t T, int E, int k, int32_t* expert_offsets,
                  int32_t* perm_token, int32_t* perm_inv, const void* x, int x_dtype, int d,
                  void* x_perm, void* workspace, size_t workspace_bytes, void* stream) {
    if (T < 0 || E < 1 || E > SMOES_E_MAX || k < 1 || k > E || k > SMOES_K_MAX) return SMOES_ERR_SHAPE;
    if (x_perm != nullptr) {
        if (!dtype_ok(x_dtype)) return SMOES_ERR_ARG;
        if (d < 1 || d > SMOES_D_MAX || (d % 8) != 0) return SMOES_ERR_SHAPE;
        if (x == nullptr) return SMOES_ERR_ARG;
    }
    if (T * k > INT32_MAX) return SMOES_ERR_SHAPE;
    if (topk_idx == nullptr || expert_offsets == nullptr || perm_token == nullptr || perm_inv == nullptr)
        return SMOES_ERR_ARG;
    if (workspace == nullptr || workspace_bytes < permute_ws(T, E, k)) return SMOES_ERR_WORKSPACE;
    hipStream_t s = as_stream(stream);
    if (T == 0) return hip_status(hipMemsetAsync(expert_offsets, 0, sizeof(int32_t) * (E + 1), s));
    Carver c(workspace);
    void* ws = c.take(permute_workspace_bytes(T, E, k));
    hipError_t err = launch_permute(topk_idx, T, E, k, expert_offsets, perm_token, perm_inv, ws, nullptr, s);
    if (err != hipSuccess) return SMOES_ERR_HIP;
    if (x_perm != nullptr) err = launch_gather_rows(x, x_dtype, d, perm_token, T * k, x_perm, s);
    return hip_status(err);
}

// ------------------------------------------------------------------ layer

namespace {

struct LayerWs {
    float* logits;
    float* probs_unused;
    int32_t* offsets;
    int32_t* perm_token;
    int32_t* perm_inv;
    void* route;
    void* modality;
    void* mi;
    void* permute;
    void* experts;
    void* ab_r;  // kept pre-activations (save_preact), else NULL
    void* ab_s;
    int32_t* flags;  // input-check flag word
};

int check_layer(const smoes_layer* L) {
    if (L == nullptr) return SMOES_ERR_ARG;
    if (!dtype_ok(L->act_dtype)) return SMOES_ERR_ARG;
    int st = check_router_shape(L->T, L->d, L->E, L->k);
    if (st != SMOES_OK) return st;
    st = check_mi_shape(L->T, L->E, L->n_batch, L->n_bins);
    if (st != SMOES_OK) return st;
    if (L->inter < 16 || (L->inter % 16) != 0) return SMOES_ERR_SHAPE;
    if (L->shared_inter < 0 || (L->shared_inter % 16) != 0) return SMOES_ERR_SHAPE;
    if (L->T * L->k > INT32_MAX) return SMOES_ERR_SHAPE;
    {
        // The GEMMs address each operand through a buffer descriptor with 32-bit byte offsets.
        const int64_t es = L->act_dtype == SMOES_BF16 ? 2 : 4;
        const int64_t lim = INT32_MAX;
        const int64_t wide = L->inter > L->d ? L->inter : L->d;
        if (L->T * L->d * es > lim || L->T * L->k * wide * es > lim ||
            L->T * static_cast<int64_t>(L->shared_inter) * es > lim ||
            2 * static_cast<int64_t>(L->inter > L->shared_inter ? L->inter : L->shared_inter) * L->d * es > lim)
            return SMOES_ERR_SHAPE;
    }
    if ((L->weights_packed != 0 && L->weights_packed != 1) || (L->save_preact != 0 && L->save_preact != 1))
        return SMOES_ERR_ARG;
    if (L->save_preact && !L->weights_packed) return SMOES_ERR_ARG;
    if (L->check_inputs != 0 && L->check_inputs != 1) return SMOES_ERR_ARG;
    if (L->weights_packed && L->act_dtype != SMOES_BF16) return SMOES_ERR_ARG;
    if (!(L->beta >= 0.0f && L->beta <= 1.0f) || !(L->var_floor >= 0.0f) || L->tau != L->tau ||
        L->grad_scale != L->grad_scale)
        return SMOES_ERR_ARG;
    return SMOES_OK;
}

size_t layer_ws_parts(const smoes_layer* L, LayerWs* out, void* base) {
    Carver c(base);
    const int64_t T = L->T;
    LayerWs w;
    w.logits = static_cast<float*>(c.take(sizeof(float) * T * L->E));
    w.probs_unused = nullptr;
    w.offsets = static_cast<int32_t*>(c.take(sizeof(int32_t) * (L->E + 1)));
    w.perm_token = static_cast<int32_t*>(c.take(sizeof(int32_t) * T * L->k));
    w.perm_inv = static_cast<int32_t*>(c.take(sizeof(int32_t) * T * L->k));
    w.route = c.take(router_workspace_bytes(T, L->d, L->E, L->act_dtype));
    w.modality = c.take(modality_workspace_bytes(T, L->d));
    w.mi = c.take(mi_workspace_bytes(T, L->E, L->n_batch, L->n_bins));
    w.permute = c.take(permute_workspace_bytes(T, L->E, L->k));
    w.experts = c.take(experts_workspace_bytes(T, L->d, L->E, L->k, L->inter, L->shared_inter, L->act_dtype));
    w.ab_r = w.ab_s = nullptr;
    if (L->save_preact) {
        w.ab_r = c.take(sizeof(uint16_t) * T * L->k * 2 * L->inter);
        w.ab_s = c.take(sizeof(uint16_t) * T * 2 * L->shared_inter);
    }
    w.flags = static_cast<int32_t*>(c.take(sizeof(int32_t)));
    if (out != nullptr) *out = w;
    return c.used + kAlign;
}

}  // namespace

size_t smoes_workspace_bytes(const smoes_layer* desc) {
    if (check_layer(desc) != SMOES_OK) return 0;
    // sizes only: carve from a fake aligned base
    return layer_ws_parts(desc, nullptr, reinterpret_cast<void*>(static_cast<uintptr_t>(kAlign)));
}

int smoes_moe_forward(const smoes_layer* L, const smoes_layer_io* io, void* workspace,
                      size_t workspace_bytes, void* stream) {
    int st = check_layer(L);
    if (st != SMOES_OK) return st;
    if (io == nullptr) return SMOES_ERR_ARG;
    if (L->T == 0) return SMOES_OK;
    if (io->x == nullptr || (L->weights_packed ? io->w_gate_packed == nullptr : io->w_gate == nullptr) ||
        io->expert_to_bin == nullptr || io->w13 == nullptr ||
        io->w2 == nullptr || io->gauss_n == nullptr || io->gauss_smu == nullptr ||
        io->gauss_ssig == nullptr || io->probs == nullptr || io->topk_idx == nullptr ||
        io->topk_w == nullptr || io->M == nullptr || io->mi_per_sample == nullptr ||
        io->loss == nullptr || io->out == nullptr)
        return SMOES_ERR_ARG;
    if (L->update_stats && io->modality_id == nullptr) return SMOES_ERR_ARG;
    if (L->shared_inter > 0 && (io->ws13 == nullptr || io->ws2 == nullptr)) return SMOES_ERR_ARG;
    if (io->sample_offsets == nullptr && L->n_batch != 1) return SMOES_ERR_SHAPE;
    if (workspace == nullptr || workspace_bytes < smoes_workspace_bytes(L)) return SMOES_ERR_WORKSPACE;
    if (io->streams != nullptr) {
        for (void* p : io->streams->side)
            if (p == nullptr) return SMOES_ERR_ARG;
        for (void* p : io->streams->events)
            if (p == nullptr) return SMOES_ERR_ARG;
    }

    hipStream_t s = as_stream(stream);
    LayerWs w;
    layer_ws_parts(L, &w, workspace);
    const int64_t T = L->T;
    if (L->check_inputs &&
        launch_check_inputs(io->modality_id, T, io->sample_offsets, L->n_batch, io->expert_to_bin, L->E, L->n_bins,
                            w.flags, s) != hipSuccess)
        return SMOES_ERR_HIP;
    float* logits = io->logits != nullptr ? io->logits : w.logits;
    int32_t* offsets = io->expert_offsets != nullptr ? io->expert_offsets : w.offsets;
    int32_t* perm_token = io->perm_token != nullptr ? io->perm_token : w.perm_token;
    int32_t* perm_inv = io->perm_inv != nullptr ? io->perm_inv : w.perm_inv;
    void* const* ev = io->stage_events;
    hipError_t err;
#define SMOES_TRY(expr)                          \
    do {                                         \
        if ((err = (expr)) != hipSuccess) return SMOES_ERR_HIP; \
    } while (0)

    ExpertArgs a;
    a.T = T;
    a.d = L->d;
    a.E = L->E;
    a.k = L->k;
    a.inter = L->inter;
    a.shared_inter = L->shared_inter;
    a.act_dtype = L->act_dtype;
    a.packed = L->weights_packed;
    a.x = io->x;
    a.w13 = io->w13;
    a.w2 = io->w2;
    a.ws13 = io->ws13;
    a.ws2 = io->ws2;
    a.expert_offsets = offsets;
    a.perm_token = perm_token;
    a.perm_inv = perm_inv;
    a.topk_w = io->topk_w;
    a.out = io->out;
    a.ab_r = w.ab_r;
    a.ab_s = L->shared_inter > 0 ? w.ab_s : nullptr;
    const WorkTables wt = experts_work_tables(a, w.experts);

    // Without side streams every stage runs on the caller's stream s, each
    // GEMM part in a launch of its own: shared GEMM1 -> shared GEMM2 ->
    // modality -> route -> MI -> permute -> routed GEMM1 -> routed GEMM2 ->
    // combine. With caller-owned side streams (io->streams) the modality
    // score and then the MI chain (after the route) run on side[0], forked
    // from s at the start of the call and joined back at its end, and each
    // GEMM covers the routed and the shared experts in one launch on s
    // (route -> permute -> GEMM1 -> GEMM2 -> combine): two concurrent GEMM
    // launches slow each other down more than they gain from overlapping.
    // For bf16 layers with packed weights and shared experts the GEMM2 stage
    // then runs the routed experts alone and the shared experts' GEMM2 follows
    // with the combine in its epilogue (the shared output never goes to HBM;
    // the combine stage is an empty pair).
    const smoes_streams* sides = io->streams;
    const bool merged = sides != nullptr;
    const bool fuse = merged && L->act_dtype == SMOES_BF16 && L->weights_packed && L->shared_inter > 0;
    hipStream_t b = s;
    hipEvent_t e_fork = nullptr, e_routed = nullptr, e_join = nullptr;
    if (sides != nullptr) {
        b = as_stream(sides->side[0]);
        e_fork = static_cast<hipEvent_t>(sides->events[0]);
        e_routed = static_cast<hipEvent_t>(sides->events[1]);
        e_join = static_cast<hipEvent_t>(sides->events[2]);
        SMOES_TRY(hipEventRecord(e_fork, s));
        SMOES_TRY(hipStreamWaitEvent(b, e_fork, 0));
    }
    if (!merged) {
        SMOES_TRY(record(ev, 2 * SMOES_STAGE_GEMM1_SHARED, s));
        SMOES_TRY(launch_experts_gemm1(a, w.experts, 2, s));
        SMOES_TRY(record(ev, 2 * SMOES_STAGE_GEMM1_SHARED + 1, s));
        SMOES_TRY(record(ev, 2 * SMOES_STAGE_GEMM2_SHARED, s));
        SMOES_TRY(launch_experts_gemm2(a, w.experts, 2, s));
        SMOES_TRY(record(ev, 2 * SMOES_STAGE_GEMM2_SHARED + 1, s));
    }
    SMOES_TRY(record(ev, 2 * SMOES_STAGE_MODALITY, b));
    SMOES_TRY(launch_modality(io->x, L->act_dtype, T, L->d, io->modality_id, io->gauss_n, io->gauss_smu,
                              io->gauss_ssig, L->update_stats ? 1 : 0, L->beta, L->tau, L->var_floor,
                              io->M, w.modality, b));
    SMOES_TRY(record(ev, 2 * SMOES_STAGE_MODALITY + 1, b));
    SMOES_TRY(record(ev, 2 * SMOES_STAGE_ROUTE, s));
    SMOES_TRY(launch_route(io->x, L->act_dtype, T, L->d, io->w_gate, L->weights_packed ? io->w_gate_packed : nullptr,
                           io->logit_bias, L->E, L->k, L->renorm_topk ? 1 : 0, logits, io->probs, io->topk_idx,
                           io->topk_w, w.route, s));
    SMOES_TRY(record(ev, 2 * SMOES_STAGE_ROUTE + 1, s));
    if (sides != nullptr) {
        SMOES_TRY(hipEventRecord(e_routed, s));
        SMOES_TRY(hipStreamWaitEvent(b, e_routed, 0));
    }
    SMOES_TRY(record(ev, 2 * SMOES_STAGE_MI, b));
    SMOES_TRY(launch_mi(io->probs, io->M, T, L->E, io->sample_offsets, L->n_batch, io->expert_to_bin,
                        L->n_bins, L->grad_scale, io->mi_per_sample, io->loss, io->dlogits, w.mi, b));
    SMOES_TRY(record(ev, 2 * SMOES_STAGE_MI + 1, b));
    if (sides != nullptr) SMOES_TRY(hipEventRecord(e_join, b));
    SMOES_TRY(record(ev, 2 * SMOES_STAGE_PERMUTE, s));
    SMOES_TRY(launch_permute(io->topk_idx, T, L->E, L->k, offsets, perm_token, perm_inv, w.permute, &wt, s));
    SMOES_TRY(record(ev, 2 * SMOES_STAGE_PERMUTE + 1, s));
    if (merged) {  // the shared stages are part of the merged launches: empty pairs
        for (int st2 : {SMOES_STAGE_GEMM1_SHARED, SMOES_STAGE_GEMM2_SHARED}) {
            if (fuse && st2 == SMOES_STAGE_GEMM2_SHARED) continue;
            SMOES_TRY(record(ev, 2 * st2, s));
            SMOES_TRY(record(ev, 2 * st2 + 1, s));
        }
    }
    SMOES_TRY(record(ev, 2 * SMOES_STAGE_GEMM1, s));
    SMOES_TRY(launch_experts_gemm1(a, w.experts, merged ? 0 : 1, s));
    SMOES_TRY(record(ev, 2 * SMOES_STAGE_GEMM1 + 1, s));
    SMOES_TRY(record(ev, 2 * SMOES_STAGE_GEMM2, s));
    SMOES_TRY(launch_experts_gemm2(a, w.experts, merged && !fuse ? 0 : 1, s));
    SMOES_TRY(record(ev, 2 * SMOES_STAGE_GEMM2 + 1, s));
    if (fuse) {
        SMOES_TRY(record(ev, 2 * SMOES_STAGE_GEMM2_SHARED, s));
        SMOES_TRY(launch_experts_gemm2_combine(a, w.experts, s));
        SMOES_TRY(record(ev, 2 * SMOES_STAGE_GEMM2_SHARED + 1, s));
        SMOES_TRY(record(ev, 2 * SMOES_STAGE_COMBINE, s));
        SMOES_TRY(record(ev, 2 * SMOES_STAGE_COMBINE + 1, s));
    } else {
        SMOES_TRY(record(ev, 2 * SMOES_STAGE_COMBINE, s));
        SMOES_TRY(launch_experts_combine(a, w.experts, s));
        SMOES_TRY(record(ev, 2 * SMOES_STAGE_COMBINE + 1, s));
    }
    if (sides != nullptr) SMOES_TRY(hipStreamWaitEvent(s, e_join, 0));
#undef SMOES_TRY
    return SMOES_OK;
}

int smoes_workspace_buffer(const smoes_layer* L, void* workspace, int which, void** ptr, size_t* bytes) {
    if (check_layer(L) != SMOES_OK || workspace == nullptr || ptr == nullptr || bytes == nullptr)
        return SMOES_ERR_ARG;
    LayerWs w;
    layer_ws_parts(L, &w, workspace);
    if (which == SMOES_BUF_CHECK_FLAGS) {
        *ptr = w.flags;
        *bytes = sizeof(int32_t);
        return SMOES_OK;
    }
    ExpertArgs a{};
    a.T = L->T;
    a.d = L->d;
    a.E = L->E;
    a.k = L->k;
    a.inter = L->inter;
    a.shared_inter = L->shared_inter;
    a.act_dtype = L->act_dtype;
    const ExpertFwdBuffers fb = experts_fwd_buffers(a, w.experts);
    const size_t es = L->act_dtype == SMOES_BF16 ? 2 : 4;
    const size_t R = static_cast<size_t>(L->T) * L->k, T = static_cast<size_t>(L->T);
    switch (which) {
        case SMOES_BUF_H_ROUTED: *ptr = fb.h_r; *bytes = es * R * L->inter; return SMOES_OK;
        case SMOES_BUF_H_SHARED: *ptr = fb.h_s; *bytes = es * T * L->shared_inter; return SMOES_OK;
        case SMOES_BUF_Y_ROUTED: *ptr = fb.y_r; *bytes = es * R * L->d; return SMOES_OK;
        case SMOES_BUF_Y_SHARED: *ptr = fb.y_s; *bytes = L->shared_inter > 0 ? es * T * L->d : 0; return SMOES_OK;
        default: return SMOES_ERR_ARG;
    }
}

int smoes_check_inputs(const smoes_layer* L, const smoes_layer_io* io, int32_t* flags, void* stream) {
    const int st = check_layer(L);
    if (st != SMOES_OK) return st;
    if (io == nullptr || flags == nullptr || io->expert_to_bin == nullptr) return SMOES_ERR_ARG;
    return hip_status(launch_check_inputs(io->modality_id, L->T, io->sample_offsets, L->n_batch, io->expert_to_bin,
                                          L->E, L->n_bins, flags, as_stream(stream)));
}

// ------------------------------------------------------------------ layer backward

namespace {
// fp32 layers and bf16 layers with row-major weights take the float32 FMA backward
bool generic_bwd(const smoes_layer* L) { return L->act_dtype != SMOES_BF16 || !L->weights_packed; }
// routed rows (T k) from which the packed backward runs on the caller's stream alone
constexpr int64_t kBwdOverlapRows = 65536;

struct BwdWs {
    void* ab_r;
    void* ab_s;
    void* dab_r;
    void* dab_s;
    void* dx_r;
    void* dx_s;
    float* wrow;
    void* wh_r;
    void* wh_s;  // float32 H of the shared experts (float32 backward only)
    int32_t* work4;
    void* router;
    // k-packed weight-gradient operands (packed bf16 path): routed rows (dout,
    // then x, gathered), w H, [dA dB]; the same for the shared experts' tokens
    int32_t* kp;
    int32_t* ranges;  // [2][9] XCD tile ranges of the two routed weight-gradient launches
    void* dxg;        // packed W_gate and dz fragments of the input gradient
    void* pt_rows_r;
    void* pt_wh_r;
    void* pt_dab_r;
    void* pt_rows_s;
    void* pt_h_s;
    void* pt_dab_s;
};
// padded row totals of the k-packed operands: routed (a bound: each expert
// pads to 16 rows) and shared
int64_t kpad_routed(const smoes_layer* L) { return L->T * L->k + 15 * static_cast<int64_t>(L->E); }
int64_t kpad_shared(const smoes_layer* L) { return ceil_div(L->T, 16) * 16; }
size_t bwd_ws_parts(const smoes_layer* L, BwdWs* out, void* base) {
    Carver c(base);
    const int64_t T = L->T, R = L->T * L->k;
    const bool gen = generic_bwd(L);
    // intermediates: bf16 on the packed matrix-core path, float32 on the FMA path
    const size_t es = gen ? sizeof(float) : sizeof(uint16_t);
    BwdWs w;
    // the pre-activations are recomputed here unless the forward kept them
    w.ab_r = c.take(L->save_preact ? 0 : es * R * 2 * L->inter);
    w.ab_s = c.take(L->save_preact ? 0 : es * T * 2 * L->shared_inter);
    w.dab_r = c.take(es * R * 2 * L->inter);
    w.dab_s = c.take(es * T * 2 * L->shared_inter);
    w.dx_r = c.take(es * R * L->d);
    w.dx_s = c.take(es * T * L->d);
    w.wrow = static_cast<float*>(c.take(sizeof(float) * R));
    w.wh_r = c.take(es * R * L->inter);
    w.wh_s = c.take(gen ? es * T * L->shared_inter : 0);
    w.work4 = static_cast<int32_t*>(c.take(sizeof(int32_t) * (L->E + 2)));
    w.router = c.take(router_bwd_workspace_bytes(T, L->d, L->E, L->act_dtype == SMOES_BF16 ? 1 : 0));
    const int64_t kr = gen ? 0 : kpad_routed(L), ksh = gen || L->shared_inter == 0 ? 0 : kpad_shared(L);
    w.kp = static_cast<int32_t*>(c.take(gen ? 0 : sizeof(int32_t) * (L->E + 1)));
    w.ranges = static_cast<int32_t*>(c.take(gen ? 0 : sizeof(int32_t) * 18));
    w.dxg = c.take(gen ? 0 : dx_mfma_workspace_bytes(T, L->d, L->E));
    w.pt_rows_r = c.take(2 * kpack_elems(L->d, kr));
    w.pt_wh_r = c.take(2 * kpack_elems(L->inter, kr));
    w.pt_dab_r = c.take(2 * kpack_elems(2 * L->inter, kr));
    w.pt_rows_s = c.take(2 * kpack_elems(L->d, ksh));
    w.pt_h_s = c.take(2 * kpack_elems(L->shared_inter, ksh));
    w.pt_dab_s = c.take(2 * kpack_elems(2 * L->shared_inter, ksh));
    if (out != nullptr) *out = w;
    return c.used + kAlign;
}
}  // namespace

size_t smoes_backward_workspace_bytes(const smoes_layer* desc) {
    if (check_layer(desc) != SMOES_OK) return 0;
    return bwd_ws_parts(desc, nullptr, reinterpret_cast<void*>(static_cast<uintptr_t>(kAlign)));
}

int smoes_moe_backward(const smoes_layer* L, const smoes_layer_io* io, const void* w13t, const void* w2t,
                       const void* ws13t, const void* ws2t, const void* dout, const float* dlogits_aux,
                       const smoes_layer_grads* G, void* fwd_workspace, size_t fwd_workspace_bytes,
                       void* workspace, size_t workspace_bytes, void* stream) {
    int st = check_layer(L);
    if (st != SMOES_OK) return st;
    if (io == nullptr || G == nullptr) return SMOES_ERR_ARG;
    const bool gen = generic_bwd(L);
    // dX = [dA dB] W13 of the packed path reads its A operand (2 inter columns
    // per row) through a buffer descriptor with 32-bit byte offsets
    if (!gen && (2 * L->T * L->k * 2 * static_cast<int64_t>(L->inter) > INT32_MAX ||
                 2 * L->T * 2 * static_cast<int64_t>(L->shared_inter) > INT32_MAX))
        return SMOES_ERR_SHAPE;
    // the k-packed weight-gradient operands are read with 32-bit byte offsets as well
    if (!gen) {
        const int64_t kr = kpad_routed(L), ks = kpad_shared(L);
        const int wide = L->d > 2 * L->inter ? L->d : 2 * L->inter;
        const int wide_s = L->d > 2 * L->shared_inter ? L->d : 2 * L->shared_inter;
        if (2 * kpack_elems(wide, kr) > INT32_MAX || (L->shared_inter > 0 && 2 * kpack_elems(wide_s, ks) > INT32_MAX))
            return SMOES_ERR_SHAPE;
    }
    if (L->T == 0) return SMOES_OK;
    const bool sh = L->shared_inter > 0;
    if (io->x == nullptr || io->w13 == nullptr || io->w_gate == nullptr || io->probs == nullptr ||
        io->topk_idx == nullptr || io->topk_w == nullptr || dout == nullptr || G->dx == nullptr ||
        G->dw_gate == nullptr || G->dz == nullptr || G->dw13 == nullptr || G->dw2 == nullptr)
        return SMOES_ERR_ARG;
    if (gen ? io->w2 == nullptr : (w13t == nullptr || w2t == nullptr)) return SMOES_ERR_ARG;
    if (sh && (io->ws13 == nullptr || G->dws13 == nullptr || G->dws2 == nullptr ||
               (gen ? io->ws2 == nullptr : (ws13t == nullptr || ws2t == nullptr))))
        return SMOES_ERR_ARG;
    if (fwd_workspace == nullptr || fwd_workspace_bytes < smoes_workspace_bytes(L)) return SMOES_ERR_WORKSPACE;
    if (workspace == nullptr || workspace_bytes < smoes_backward_workspace_bytes(L)) return SMOES_ERR_WORKSPACE;
    if (io->streams != nullptr) {
        for (void* p : io->streams->side)
            if (p == nullptr) return SMOES_ERR_ARG;
        for (void* p : io->streams->events)
            if (p == nullptr) return SMOES_ERR_ARG;
    }
    hipStream_t s = as_stream(stream);
    LayerWs fw;
    layer_ws_parts(L, &fw, fwd_workspace);
    BwdWs bw;
    bwd_ws_parts(L, &bw, workspace);
    const int64_t T = L->T;
    const int32_t* offsets = io->expert_offsets != nullptr ? io->expert_offsets : fw.offsets;
    const int32_t* perm_token = io->perm_token != nullptr ? io->perm_token : fw.perm_token;
    const int32_t* perm_inv = io->perm_inv != nullptr ? io->perm_inv : fw.perm_inv;
    ExpertArgs a;
    a.T = T;
    a.d = L->d;
    a.E = L->E;
    a.k = L->k;
    a.inter = L->inter;
    a.shared_inter = L->shared_inter;
    a.act_dtype = L->act_dtype;
    a.packed = gen ? 0 : 1;
    a.x = io->x;
    a.w13 = io->w13;
    a.w2 = io->w2;
    a.ws13 = io->ws13;
    a.ws2 = io->ws2;
    a.expert_offsets = offsets;
    a.perm_token = perm_token;
    a.perm_inv = perm_inv;
    a.topk_w = io->topk_w;
    a.out = nullptr;
    a.ab_r = a.ab_s = nullptr;
    const ExpertFwdBuffers fb = experts_fwd_buffers(a, fw.experts);
    hipError_t err;
#define SMOES_BTRY(expr)                                        \
    do {                                                        \
        if ((err = (expr)) != hipSuccess) return SMOES_ERR_HIP; \
    } while (0)
    const int bf16 = L->act_dtype == SMOES_BF16 ? 1 : 0;
    if (gen) {
        // float32 FMA path, every step on s: router backward and dW_gate, then
        // the experts (routed and shared in each launch), then the input gradient
        GenericBwdPtrs gp;
        gp.dout = dout;
        gp.ab_r = static_cast<float*>(bw.ab_r);
        gp.ab_s = static_cast<float*>(bw.ab_s);
        gp.dab_r = static_cast<float*>(bw.dab_r);
        gp.dab_s = static_cast<float*>(bw.dab_s);
        gp.wh_r = static_cast<float*>(bw.wh_r);
        gp.wh_s = static_cast<float*>(bw.wh_s);
        gp.dx_r = static_cast<float*>(bw.dx_r);
        gp.dx_s = static_cast<float*>(bw.dx_s);
        gp.wrow = bw.wrow;
        gp.work = bw.work4;
        gp.dw13 = G->dw13;
        gp.dw2 = G->dw2;
        gp.dws13 = G->dws13;
        gp.dws2 = G->dws2;
        SMOES_BTRY(launch_router_bwd(dout, fb.y_r, bf16, perm_inv, io->probs, io->topk_idx, io->topk_w, dlogits_aux,
                                     T, L->d, L->E, L->k, L->renorm_topk ? 1 : 0, G->dw, G->dz, s));
        SMOES_BTRY(launch_dwgate(G->dz, io->x, bf16, T, L->d, L->E, G->dw_gate, G->dbias, bw.router, s));
        SMOES_BTRY(launch_row_weights(perm_inv, io->topk_w, T, L->k, bw.wrow, s));
        for (int step = 0; step < 5; ++step) SMOES_BTRY(launch_generic_bwd(step, a, gp, s));
        SMOES_BTRY(launch_dx_gather(bw.dx_r, sh ? bw.dx_s : nullptr, 0, perm_inv, G->dz, io->w_gate, T, L->d, L->E,
                                    L->k, G->dx, nullptr, s));
        return SMOES_OK;
    }
    BwdGemmPtrs bp;
    bp.dout = dout;
    bp.w2t = w2t;
    bp.ws2t = ws2t;
    bp.w13t = w13t;
    bp.ws13t = ws13t;
    bp.ab_r = L->save_preact ? fw.ab_r : bw.ab_r;
    bp.ab_s = L->save_preact ? fw.ab_s : bw.ab_s;
    bp.dab_r = bw.dab_r;
    bp.dab_s = bw.dab_s;
    bp.dx_r = bw.dx_r;
    bp.dx_s = bw.dx_s;
    bp.wrow = bw.wrow;
    bp.wh_r = bw.wh_r;
    bp.work4 = bw.work4;
    // Caller's stream s: combine weights, the routed experts' dgrad GEMMs
    // (pre-activation recompute unless kept, dH with the SwiGLU backward,
    // dX) and weight gradients, then the input gradient. With caller-owned
    // side streams (io->streams) the router backward, dW_gate and the shared
    // experts' GEMMs and weight gradients (independent of the routed chain)
    // run on side[1], forked from s at the start of the call and joined back
    // before the input gradient, which needs both chains; without them every
    // step runs on s in the same dependency order.
    // Side streams only below kBwdOverlapRows routed rows: above it the routed
    // GEMMs alone fill the chip and the side chain only takes CUs from them.
    const smoes_streams* sides = L->T * L->k < kBwdOverlapRows ? io->streams : nullptr;
    hipStream_t c = s;
    hipEvent_t e_fork = nullptr, e_join = nullptr;
    if (sides != nullptr) {
        c = as_stream(sides->side[1]);
        e_fork = static_cast<hipEvent_t>(sides->events[0]);
        e_join = static_cast<hipEvent_t>(sides->events[3]);
        SMOES_BTRY(hipEventRecord(e_fork, s));
        SMOES_BTRY(hipStreamWaitEvent(c, e_fork, 0));
    }
    const int I = L->inter, SI = L->shared_inter, d = L->d;
    // side chain: router backward (dz, dw), dW_gate and dbias, shared experts
    SMOES_BTRY(launch_router_bwd(dout, fb.y_r, 1, perm_inv, io->probs, io->topk_idx, io->topk_w, dlogits_aux, T,
                                 L->d, L->E, L->k, L->renorm_topk ? 1 : 0, G->dw, G->dz, c));
    SMOES_BTRY(launch_dwgate(G->dz, io->x, 1, T, d, L->E, G->dw_gate, G->dbias, bw.router, c));
    if (sh) {
        for (int mode = L->save_preact ? 4 : 3; mode <= 5; ++mode)
            SMOES_BTRY(launch_bwd_gemm(mode, a, fw.experts, bp, 2, c));
        // dWs2 = dout^T H_s and dWs13 = [dA dB]_s^T X over all tokens, from k-packed copies
        const int64_t ksh = kpad_shared(L);
        SMOES_BTRY(launch_kpack(dout, d, nullptr, nullptr, nullptr, 1, T, ksh, bw.pt_rows_s, c));
        SMOES_BTRY(launch_kpack(fb.h_s, SI, nullptr, nullptr, nullptr, 1, T, ksh, bw.pt_h_s, c));
        SMOES_BTRY(launch_wgrad_pk(1, d, SI, nullptr, nullptr, T, bw.pt_rows_s, bw.pt_h_s, G->dws2, c));
        SMOES_BTRY(launch_kpack(bw.dab_s, 2 * SI, nullptr, nullptr, nullptr, 1, T, ksh, bw.pt_dab_s, c));
        SMOES_BTRY(launch_kpack(io->x, d, nullptr, nullptr, nullptr, 1, T, ksh, bw.pt_rows_s, c));
        SMOES_BTRY(launch_wgrad_pk(1, 2 * SI, d, nullptr, nullptr, T, bw.pt_dab_s, bw.pt_rows_s, G->dws13, c));
    }
    if (sides != nullptr) SMOES_BTRY(hipEventRecord(e_join, c));
    // routed chain
    SMOES_BTRY(launch_row_weights(perm_inv, io->topk_w, T, L->k, bw.wrow, s));
    for (int mode = L->save_preact ? 4 : 3; mode <= 5; ++mode)
        SMOES_BTRY(launch_bwd_gemm(mode, a, fw.experts, bp, 1, s));
    // dW2 = dout^T (w H) over each expert's rows (dout gathered); dW13 = [dA dB]^T X (x
    // gathered): both operands k-packed per expert first (rows padded to 16)
    const int64_t kr = kpad_routed(L);
    SMOES_BTRY(launch_kpad_offsets(offsets, L->E, bw.kp, wgrad_tiles_per_group(d, I), wgrad_tiles_per_group(2 * I, d),
                                   bw.ranges, s));
    SMOES_BTRY(launch_kpack(dout, d, perm_token, offsets, bw.kp, L->E, T, kr, bw.pt_rows_r, s));
    SMOES_BTRY(launch_kpack(bw.wh_r, I, nullptr, offsets, bw.kp, L->E, T, kr, bw.pt_wh_r, s));
    SMOES_BTRY(launch_wgrad_pk(L->E, d, I, bw.kp, bw.ranges, T, bw.pt_rows_r, bw.pt_wh_r, G->dw2, s));
    SMOES_BTRY(launch_kpack(bw.dab_r, 2 * I, nullptr, offsets, bw.kp, L->E, T, kr, bw.pt_dab_r, s));
    SMOES_BTRY(launch_kpack(io->x, d, perm_token, offsets, bw.kp, L->E, T, kr, bw.pt_rows_r, s));
    SMOES_BTRY(launch_wgrad_pk(L->E, 2 * I, d, bw.kp, bw.ranges + 9, T, bw.pt_dab_r, bw.pt_rows_r, G->dw13, s));
    if (sides != nullptr) SMOES_BTRY(hipStreamWaitEvent(s, e_join, 0));
    SMOES_BTRY(launch_dx_gather(bw.dx_r, sh ? bw.dx_s : nullptr, 1, perm_inv, G->dz, io->w_gate, T, L->d, L->E, L->k,
                                G->dx, bw.dxg, s));
#undef SMOES_BTRY
    return SMOES_OK;
}

namespace {
// batch, rows n, contraction k and gate/up interleave of each packed tensor; false if invalid
bool weight_dims(const smoes_layer* L, int which, int* batch, int* n, int* k, int* interleave, int* transpose) {
    *transpose = 0;
    switch (which) {
        case SMOES_W13: *batch = L->E; *n = L->inter; *k = L->d; *interleave = 1; return true;
        case SMOES_W2: *batch = L->E; *n = L->d; *k = L->inter; *interleave = 0; return true;
        case SMOES_WS13: *batch = 1; *n = L->shared_inter; *k = L->d; *interleave = 1; return L->shared_inter > 0;
        case SMOES_WS2: *batch = 1; *n = L->d; *k = L->shared_inter; *interleave = 0; return L->shared_inter > 0;
        case SMOES_WGATE: *batch = 1; *n = L->E; *k = L->d; *interleave = 0; return true;
        case SMOES_W13T: *batch = L->E; *n = L->d; *k = 2 * L->inter; *interleave = 0; *transpose = 1; return true;
        case SMOES_W2T: *batch = L->E; *n = L->inter; *k = L->d; *interleave = 0; *transpose = 1; return true;
        case SMOES_WS13T:
            *batch = 1; *n = L->d; *k = 2 * L->shared_inter; *interleave = 0; *transpose = 1;
            return L->shared_inter > 0;
        case SMOES_WS2T:
            *batch = 1; *n = L->shared_inter; *k = L->d; *interleave = 0; *transpose = 1;
            return L->shared_inter > 0;
        default: return false;
    }
}
}  // namespace

size_t smoes_packed_weight_bytes(const smoes_layer* desc, int which) {
    if (check_layer(desc) != SMOES_OK) return 0;
    int batch, n, k, il, tr;
    if (!weight_dims(desc, which, &batch, &n, &k, &il, &tr)) return 0;
    if (which == SMOES_WGATE) return router_packed_elems(desc->d, desc->E) * 2;
    return static_cast<size_t>(packed_weight_elems(batch, n, k, il)) * 2;
}

int smoes_pack_weights(const smoes_layer* desc, int which, const void* src, void* dst, void* stream) {
    const int st = check_layer(desc);
    if (st != SMOES_OK) return st;
    int batch, n, k, il, tr;
    if (desc->act_dtype != SMOES_BF16 || !weight_dims(desc, which, &batch, &n, &k, &il, &tr) || src == nullptr ||
        dst == nullptr)
        return SMOES_ERR_ARG;
    const hipError_t err = which == SMOES_WGATE
                               ? launch_split_wgate(static_cast<const float*>(src), desc->E, desc->d, dst, as_stream(stream))
                               : launch_pack_weights(src, batch, n, k, il, tr, dst, as_stream(stream));
    return err == hipSuccess ? SMOES_OK : SMOES_ERR_HIP;
}

int smoes_streams_create(smoes_streams* st) {
    if (st == nullptr) return SMOES_ERR_ARG;
    *st = smoes_streams{};
    for (void*& p : st->side) {
        hipStream_t h;
        if (hipStreamCreateWithFlags(&h, hipStreamNonBlocking) != hipSuccess) {
            smoes_streams_destroy(st);
            return SMOES_ERR_HIP;
        }
        p = h;
    }
    for (void*& p : st->events) {
        hipEvent_t e;
        if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) {
            smoes_streams_destroy(st);
            return SMOES_ERR_HIP;
        }
        p = e;
    }
    return SMOES_OK;
}

int smoes_streams_destroy(smoes_streams* st) {
    if (st == nullptr) return SMOES_ERR_ARG;
    int rc = SMOES_OK;
    for (void*& p : st->events) {
        if (p != nullptr && hipEventDestroy(static_cast<hipEvent_t>(p)) != hipSuccess) rc = SMOES_ERR_HIP;
        p = nullptr;
    }
    for (void*& p : st->side) {
        if (p != nullptr && hipStreamDestroy(static_cast<hipStream_t>(p)) != hipSuccess) rc = SMOES_ERR_HIP;
        p = nullptr;
    }
    return rc;
}

int smoes_events_create(int n, void** events) {
    if (n < 0 || (n > 0 && events == nullptr)) return SMOES_ERR_ARG;
    for (int i = 0; i < n; ++i) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) return SMOES_ERR_HIP;
        events[i] = e;
    }
    return SMOES_OK;
}

int smoes_events_destroy(int n, void** events) {
    if (n < 0 || (n > 0 && events == nullptr)) return SMOES_ERR_ARG;
    for (int i = 0; i < n; ++i)
        if (events[i] != nullptr && hipEventDestroy(static_cast<hipEvent_t>(events[i])) != hipSuccess)
            return SMOES_ERR_HIP;
    return SMOES_OK;
}

int smoes_event_elapsed_ms(void* start, void* end, float* ms) {
    if (start == nullptr || end == nullptr || ms == nullptr) return SMOES_ERR_ARG;
    if (hipEventSynchronize(static_cast<hipEvent_t>(end)) != hipSuccess) return SMOES_ERR_HIP;
    return hip_status(hipEventElapsedTime(ms, static_cast<hipEvent_t>(start), static_cast<hipEvent_t>(end)));
}

}  // extern "C"
