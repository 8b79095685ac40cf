/*
 * smoes.h - C ABI of the SMoES MoE-layer hot path for AMD Instinct MI355X (gfx950).
 *
 * SMoES ("Soft Modality-Guided Expert Specialization in MoE-VLMs") routes the
 * tokens of a mixed vision + text batch through a Mixture-of-Experts layer and
 * regularises the router with the mutual information between a soft modality
 * score and groups ("bins") of experts. This library computes one layer:
 *
 *   smoes_route            router logits, softmax gate, top-k        (Sec. 3.1)
 *   smoes_modality_score   EMA-Welford statistics + Gaussian score   (Sec. 3.2.2, Eq. 5-9)
 *   smoes_mi_loss          inter-bin MI, its loss and d loss / d logits (Sec. 3.3-3.4, Eq. 12-15)
 *   smoes_permute          expert-contiguous token order (+ optional row gather)
 *   smoes_binning          momentum-adaptive bins, bin-level load balance loss
 *                          (+ d loss / d logits) and MSI (Sec. 3.3, 3.5, 4.1;
 *                          Eq. 10-11, 16, 18-19)
 *   smoes_moe_forward      all of the above + grouped SwiGLU experts, shared
 *                          experts and the weighted combine
 *
 * Conventions shared by every entry point
 *   - Every array pointer is a DEVICE pointer owned by the caller; arrays are
 *     dense and row-major. The library allocates no device memory: scratch
 *     comes from a caller-provided workspace whose size the matching
 *     *_workspace_size query returns (any alignment; the library aligns
 *     inside it). Workspace contents need not be initialised and are
 *     clobbered.
 *   - `stream` is a hipStream_t (NULL = the default stream). Work is enqueued
 *     asynchronously; no call synchronises the host. The library keeps no
 *     global state, so distinct calls with distinct buffers may run from
 *     different threads.
 *   - Return value: SMOES_OK (0) or a negative smoes_status. Argument checks
 *     happen on the host before anything is enqueued; on an error nothing is
 *     launched and no output is written. T = 0 is a successful no-op.
 *   - Values that live on the device are NOT checked on the host (that would
 *     need a synchronisation); the caller guarantees them: modality ids in
 *     {0, 1}, sample offsets non-decreasing with offsets[0] = 0 and
 *     offsets[n_batch] = T, expert_to_bin entries in [0, n_bins) with exactly
 *     E / n_bins experts per bin, top-k indices in [0, E) and distinct within
 *     a token. smoes_check_inputs (or smoes_layer.check_inputs = 1) checks the
 *     first three on the device and reports them in a flag word.
 *   - Activation dtype codes: SMOES_F32 (float) or SMOES_BF16 (bfloat16 bits,
 *     uint16 storage). Router weights, logits, gate probabilities, modality
 *     scores and losses are always float32.
 */
#ifndef SMOES_H
#define SMOES_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
enum smoes_status {
    SMOES_OK = 0,
    SMOES_ERR_ARG = -1,       /* a required pointer is NULL, or a scalar/dtype is out of range */
    SMOES_ERR_SHAPE = -2,     /* inconsistent sizes (see each entry point) */
    SMOES_ERR_WORKSPACE = -3, /* workspace_bytes smaller than the query's answer */
    SMOES_ERR_HIP = -4,       /* a HIP launch or runtime call failed */
    SMOES_ERR_SCRATCH = -5    /* the problem needs more scratch than the fixed device array of
                                 smoes_mi_loss_noalloc holds (SMOES_NOALLOC_SCRATCH_BYTES) */
};

/* Activation storage types. */
enum smoes_dtype { SMOES_F32 = 0, SMOES_BF16 = 1 };

/* Limits checked by every entry point (SMOES_ERR_SHAPE beyond them). */
#define SMOES_E_MAX 256   /* routed experts */
#define SMOES_K_MAX 16    /* top-k */
#define SMOES_BINS_MAX 64 /* expert bins */
#define SMOES_D_MAX 16384 /* hidden size */

/* Human-readable text for a status code (static storage, never NULL). */
const char* smoes_status_string(int status);

/* Library version string (static storage). */
const char* smoes_version(void);

/* ------------------------------------------------------------------------ */
/* Router (Sec. 3.1: g = softmax(W_gate x); the k highest-scoring experts).  */
/* ------------------------------------------------------------------------ */

size_t smoes_route_workspace_size(int64_t T, int d, int E, int x_dtype);

/*
 * x          [T, d] activations (x_dtype). For SMOES_BF16 the logits are
 *            computed fp32-faithfully (the fp32 weights are split into three
 *            bf16 terms whose products with the exact bf16 inputs are exact).
 * w_gate     [E, d] float32 router weights.
 * logit_bias [E] float32 added to every token's logits before softmax and
 *            top-k, or NULL.
 * renorm_topk  0: topk_w are the gate probabilities of the chosen experts;
 *              1: they are renormalised to sum to 1 per token.
 * logits     [T, E] float32 output, or NULL (not stored).
 * probs      [T, E] float32 output: the full softmax over all E experts.
 * topk_idx   [T, k] int32 output: experts by descending logit, ties to the
 *            lower index (decided on the float32 logits).
 * topk_w     [T, k] float32 output: combine weights.
 * Shapes: 1 <= d <= SMOES_D_MAX, d % 8 == 0; 1 <= E <= SMOES_E_MAX;
 *         1 <= k <= min(E, SMOES_K_MAX); for SMOES_BF16, T * d * 2 < 2^31.
 */
int smoes_route(const void* x, int x_dtype, int64_t T, int d,
                const float* w_gate, const float* logit_bias, int E, int k, int renorm_topk,
                float* logits, float* probs, int32_t* topk_idx, float* topk_w,
                void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Gaussian-statistics modality score (Sec. 3.2.2, Eq. 5-9).                 */
/* ------------------------------------------------------------------------ */

size_t smoes_modality_workspace_size(int64_t T, int d);

/*
 * x            [T, d] activations (x_dtype): the MoE layer input.
 * modality_id  [T] uint8, 0 = vision, 1 = text. Required iff update != 0.
 * gauss_n      [2] float32 EMA token counts N_m (in/out when update != 0).
 * gauss_smu    [2, d] float32 S_mu,m (in/out when update != 0).
 * gauss_ssig   [2, d] float32 S_sigma2,m (in/out when update != 0).
 *              Row/entry 0 is vision, 1 is text. The caller owns (and
 *              checkpoints) this state; a fresh layer starts from zeros.
 * update       1: first fold the batch into the state with the EMA-Welford
 *              step of Eq. 5-7 (decay beta), then score; 0: score only.
 * beta         EMA decay in [0, 1] (paper: 0.99).
 * tau          temperature of Eq. 9; tau <= 0 selects 0.5 * d (paper default).
 * var_floor    lower bound applied to sigma^2 = S_sigma2 / N (>= 0).
 * M            [T, 2] float32 output: column 0 vision score, column 1 text
 *              score; each row sums to 1.
 * A modality with N = 0 scores with mu = 0, sigma^2 = 1.
 * Shapes: 1 <= d <= SMOES_D_MAX, d % 8 == 0.
 */
int smoes_modality_score(const void* x, int x_dtype, int64_t T, int d,
                         const uint8_t* modality_id,
                         float* gauss_n, float* gauss_smu, float* gauss_ssig,
                         int update, float beta, float tau, float var_floor,
                         float* M, void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Inter-bin mutual information (Sec. 3.3-3.4, Eq. 12-15) and its gradient. */
/* ------------------------------------------------------------------------ */

size_t smoes_mi_workspace_size(int64_t T, int E, int n_batch, int n_bins);

/*
 * probs          [T, E] float32 full-softmax gate g.
 * M              [T, 2] float32 soft modality scores (column 0 vision).
 * sample_offsets [n_batch + 1] int32 token offsets of the samples, or NULL
 *                for one sample covering all T tokens (then n_batch must be 1).
 * expert_to_bin  [E] int32 bin of every expert (bins hold E / n_bins experts).
 * grad_scale     multiplies the gradient (e.g. the loss weight alpha_MI).
 * mi_per_sample  [n_batch] float32 output: I_i(M; B) in nats (Eq. 14).
 * loss           [1] float32 output: L_MI = -(1/n_batch) sum_i I_i (Eq. 15).
 * dlogits        [T, E] float32 output grad_scale * dL_MI / d logits with the
 *                modality scores held constant, or NULL to skip it.
 * Sums are accumulated in float64 in a fixed order: results are bit-for-bit
 * reproducible. Shapes: 1 <= E <= SMOES_E_MAX, 1 <= n_bins <= SMOES_BINS_MAX,
 * E % n_bins == 0, n_batch >= 1.
 */
int smoes_mi_loss(const float* probs, const float* M, int64_t T, int E,
                  const int32_t* sample_offsets, int n_batch,
                  const int32_t* expert_to_bin, int n_bins, float grad_scale,
                  float* mi_per_sample, float* loss, float* dlogits,
                  void* workspace, size_t workspace_bytes, void* stream);

/*
 * smoes_mi_loss without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, serving loops or harnesses that
 * forbid allocation). Arguments, outputs and bits are those of
 * smoes_mi_loss; the scratch comes from a fixed file-scope device array of
 * SMOES_NOALLOC_SCRATCH_BYTES that every device the library runs on holds
 * until the process ends. The call allocates nothing. It accepts problems
 * whose smoes_mi_workspace_size(T, E, n_batch, n_bins) is at most
 * SMOES_NOALLOC_SCRATCH_BYTES (16384 tokens in 16 samples with E = 160 need
 * 1.3 MB, 65536 tokens in one sample with E = 256 need 4.1 MB) and returns
 * SMOES_ERR_SCRATCH, launching nothing, beyond that. All calls on
 * one device share that device's array, which keeps the last call's
 * contents (no call relies on its initial contents): calls that may overlap
 * in time on one device (different streams, threads) race on it and must be
 * serialised by the caller.
 */
#define SMOES_NOALLOC_SCRATCH_BYTES (8u << 20)
int smoes_mi_loss_noalloc(const float* probs, const float* M, int64_t T, int E,
                          const int32_t* sample_offsets, int n_batch,
                          const int32_t* expert_to_bin, int n_bins, float grad_scale,
                          float* mi_per_sample, float* loss, float* dlogits, void* stream);

/* ------------------------------------------------------------------------ */
/* Momentum-adaptive binning (Sec. 3.3, Eq. 10-11), bin-level load balance   */
/* (Sec. 3.5, Eq. 16) and modality specialization index (Sec. 4.1, Eq. 18-19)*/
/* ------------------------------------------------------------------------ */

size_t smoes_binning_workspace_size(int64_t T, int E, int n_bins);

/*
 * From one batch's routing:
 * probs         [T, E] float32 gate values (full softmax), topk_idx [T, k] int32,
 * modality_id   [T] uint8 hard labels (0 vision, 1 text),
 * expert_to_bin [E] int32: the bins the batch was routed and scored with.
 * Counts C[m][e] = tokens of label m whose top-k holds e.
 *
 * load_ema [2][E] float64 (row 0 vision, row 1 text), in/out, or NULL: the
 *   expert-load EMA of Eq. 10, C_bar = beta * C_bar + (1 - beta) * C (both
 *   products rounded before the sum); NULL scores this batch's counts only.
 * Outputs, each optional (NULL = not written):
 *   counts [2][E] int32: C of this batch;
 *   f_spec [E] float64: Eq. 11, C_bar_text / (C_bar_text + C_bar_vision), 1/2
 *     for an expert without load;
 *   expert_to_bin_next [E] int32: experts sorted by ascending f_spec (ties to
 *     the lower index) cut into n_bins consecutive bins of E / n_bins: the
 *     adaptive bins for the next batch (must not alias expert_to_bin);
 *   bal_loss [1] float32: Eq. 16 for this layer, sum over bins k of
 *     N_B sum_{e in B_k} f_e P_e, where the tokens of bin k are those with at
 *     least one top-k expert in it (T_k of them), f_e = (tokens whose top-k
 *     holds e) / T_k and P_e = mean gate of e over them;
 *   dlogits [T, E] float32: grad_scale * d bal_loss / d logits with the top-k
 *     sets held fixed; written, or added to the array when accumulate = 1
 *     (e.g. onto the MI gradient);
 *   msi [1] float32: Eq. 18-19 of this batch's counts (an expert no token
 *     reaches counts as unspecialised).
 * Sums run in a fixed order: results are bit-reproducible. T = 0 still
 * updates load_ema (with zero counts) and the bins.
 * Shapes: 1 <= E <= SMOES_E_MAX, 1 <= n_bins <= SMOES_BINS_MAX,
 * E % n_bins == 0, 1 <= k <= min(E, SMOES_K_MAX); 0 <= beta <= 1.
 */
int smoes_binning(const float* probs, const int32_t* topk_idx, const uint8_t* modality_id, int64_t T, int E,
                  int k, const int32_t* expert_to_bin, int n_bins, float beta, double* load_ema,
                  int32_t* counts, double* f_spec, int32_t* expert_to_bin_next, float grad_scale,
                  float* bal_loss, float* dlogits, int accumulate, float* msi, void* workspace,
                  size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Expert-contiguous permutation of the routed (token, slot) pairs.          */
/* ------------------------------------------------------------------------ */

size_t smoes_permute_workspace_size(int64_t T, int E, int k);

/*
 * topk_idx       [T, k] int32 experts of every token (distinct per token).
 * expert_offsets [E + 1] int32 output: exclusive prefix sum of the per-expert
 *                row counts (expert e owns rows [off[e], off[e+1])).
 * perm_token     [T * k] int32 output: token of every permuted row; rows of
 *                one expert are in ascending token order.
 * perm_inv       [T, k] int32 output: permuted row of every (token, slot).
 * x, x_perm      optional: when x_perm is non-NULL, x_perm[r] = x[perm_token[r]]
 *                ([T * k, d], same dtype as x) is also written.
 * The order is a deterministic stable counting sort (no atomics decide it).
 * Shapes: 1 <= E <= SMOES_E_MAX, 1 <= k <= min(E, SMOES_K_MAX); d % 8 == 0
 * when x_perm is given.
 */
int smoes_permute(const int32_t* topk_idx, int64_t T, int E, int k,
                  int32_t* expert_offsets, int32_t* perm_token, int32_t* perm_inv,
                  const void* x, int x_dtype, int d, void* x_perm,
                  void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* The whole SMoES MoE layer forward.                                        */
/* ------------------------------------------------------------------------ */

typedef struct smoes_layer {
    int64_t T;        /* tokens */
    int d;            /* hidden size, d % 8 == 0 */
    int E;            /* routed experts */
    int k;            /* top-k */
    int inter;        /* routed expert FFN inner size, inter % 16 == 0 */
    int shared_inter; /* merged inner size of the shared experts (0 = none), % 16 == 0 */
    int n_bins;       /* expert bins, E % n_bins == 0 */
    int n_batch;      /* samples (>= 1) */
    int act_dtype;    /* SMOES_F32 or SMOES_BF16: x, expert weights and out */
    float tau;        /* Eq. 9 temperature; <= 0 selects 0.5 * d */
    float beta;       /* EMA decay of Eq. 5-7 */
    float var_floor;  /* floor on sigma^2 */
    float grad_scale; /* scale of dlogits */
    int renorm_topk;  /* renormalise the combine weights */
    int update_stats; /* fold the batch into the Gaussian state before scoring */
    int weights_packed; /* 1: w13, w2, ws13, ws2 are in the packed order of smoes_pack_weights
                           (SMOES_BF16 only); 0: row-major as in smoes_layer_io */
    int save_preact;    /* 1: smoes_moe_forward also keeps the experts' gate and up
                           pre-activations (bf16, in its workspace) for
                           smoes_moe_backward, which then skips recomputing them
                           (packed bf16 layers only); 0: it does not */
    int check_inputs;   /* 1: smoes_moe_forward first checks the device-resident
                           preconditions (as smoes_check_inputs) and writes the
                           flag word into its workspace (SMOES_BUF_CHECK_FLAGS);
                           0: no check (the production setting) */
} smoes_layer;

/* Side streams for smoes_moe_forward and smoes_moe_backward (caller-owned;
 * see smoes_streams_create). */
typedef struct smoes_streams {
    void* side[2];   /* hipStream_t: [0] the forward's modality score + MI chain, [1] the
                        backward's router and shared-expert gradients */
    void* events[4]; /* hipEvent_t (timing disabled) used to fork and join them */
} smoes_streams;

typedef struct smoes_layer_io {
    /* inputs */
    const void* x;                 /* [T, d] act_dtype */
    const uint8_t* modality_id;    /* [T]; required iff update_stats */
    const int32_t* sample_offsets; /* [n_batch + 1] or NULL (one sample) */
    const float* w_gate;           /* [E, d] */
    const float* logit_bias;       /* [E] or NULL */
    const int32_t* expert_to_bin;  /* [E] */
    const void* w13;               /* [E, 2*inter, d]: rows [0, inter) gate, [inter, 2*inter) up */
    const void* w2;                /* [E, d, inter] down projection */
    const void* ws13;              /* [2*shared_inter, d] or NULL when shared_inter == 0 */
    const void* ws2;               /* [d, shared_inter] or NULL when shared_inter == 0 */
    const void* w_gate_packed;     /* weights_packed: the router weights packed by
                                      smoes_pack_weights(SMOES_WGATE) (then w_gate may be
                                      NULL); otherwise unused */
    /* caller-owned Gaussian state (in/out when update_stats) */
    float* gauss_n;   /* [2] */
    float* gauss_smu; /* [2, d] */
    float* gauss_ssig;/* [2, d] */
    /* outputs (NULL allowed where marked) */
    float* logits;          /* [T, E] or NULL */
    float* probs;           /* [T, E] */
    int32_t* topk_idx;      /* [T, k] */
    float* topk_w;          /* [T, k] */
    float* M;               /* [T, 2] */
    float* mi_per_sample;   /* [n_batch] */
    float* loss;            /* [1] */
    float* dlogits;         /* [T, E] or NULL */
    int32_t* expert_offsets;/* [E + 1] or NULL */
    int32_t* perm_token;    /* [T * k] or NULL */
    int32_t* perm_inv;      /* [T, k] or NULL */
    void* out;              /* [T, d] act_dtype: routed experts + shared experts */
    /* optional stage timing: NULL, or 2 * SMOES_N_STAGES events made by
     * smoes_events_create (entries may be NULL); events 2s and 2s + 1 are
     * recorded on the stream that runs stage s, before and after it. */
    void* const* stage_events;
    /* optional side streams: NULL runs every stage on `stream`, the routed and
     * the shared experts' GEMMs in launches of their own; otherwise the
     * modality score and the MI chain run on side[0], forked from and joined
     * back into `stream` with the given events, and each expert GEMM covers
     * the routed and the shared experts in one launch on `stream`. One
     * smoes_streams may serve consecutive calls; calls that overlap in time
     * need one each. */
    const smoes_streams* streams;
} smoes_layer_io;

/* Stages of smoes_moe_forward. Without side streams every stage runs on the
 * caller's stream in the order GEMM1_SHARED, GEMM2_SHARED, MODALITY, ROUTE,
 * MI, PERMUTE, GEMM1, GEMM2, COMBINE. With io->streams, ROUTE, PERMUTE,
 * GEMM1, GEMM2 and COMBINE run in this order on the caller's stream, GEMM1
 * and GEMM2 each covering the routed and the shared experts (the two
 * *_SHARED stages are then empty event pairs), MODALITY and then MI (after
 * ROUTE) on side[0]; the caller's stream waits for side[0] before the
 * call's work is complete. Exception, with io->streams and a bf16 layer with
 * packed weights and shared experts: GEMM2 covers the routed experts only,
 * then GEMM2_SHARED runs the shared experts' down GEMM with the combine in
 * its epilogue (COMBINE is an empty pair, and SMOES_BUF_Y_SHARED is not
 * written); the output has the same bits as the separate combine's. */
enum smoes_stage {
    SMOES_STAGE_ROUTE = 0,        /* router GEMM + softmax + top-k */
    SMOES_STAGE_MODALITY = 1,     /* statistics update (optional) + modality score */
    SMOES_STAGE_MI = 2,           /* MI partials, loss, gradient */
    SMOES_STAGE_PERMUTE = 3,      /* expert-contiguous order + work lists */
    SMOES_STAGE_GEMM1 = 4,        /* routed (+ shared, with side streams) experts: grouped gate/up GEMM + SwiGLU */
    SMOES_STAGE_GEMM2 = 5,        /* routed (+ shared, with side streams) experts: grouped down GEMM */
    SMOES_STAGE_COMBINE = 6,      /* weighted combine + shared output */
    SMOES_STAGE_GEMM1_SHARED = 7, /* shared experts: gate/up GEMM + SwiGLU */
    SMOES_STAGE_GEMM2_SHARED = 8, /* shared experts: down GEMM */
    SMOES_N_STAGES = 9
};

size_t smoes_workspace_bytes(const smoes_layer* desc);

/*
 * One SMoES MoE layer forward (Sec. 3.1: softmax router and top-k experts;
 * Sec. 3.2.2, Eq. 5-9: Gaussian modality score; Sec. 3.3-3.4, Eq. 12-15:
 * inter-bin MI loss and its logit gradient; the MoE layer's experts with the
 * backbone's always-on shared experts). Shapes as in the entry points above, plus
 * inter >= 16, inter % 16 == 0 and shared_inter % 16 == 0. The expert FFN is
 * SwiGLU: down(silu(gate x) * up x), silu(a) = a / (1 + exp(-a)); the shared
 * experts (ungated, weight 1) are one SwiGLU of inner size shared_inter.
 * With SMOES_BF16 the expert GEMMs take bf16 operands with float32
 * accumulation and the intermediate activations are stored in bf16.
 * Size limit (SMOES_ERR_SHAPE beyond it): with s the activation element size
 * (2 for bf16, 4 for f32), each of T*d*s, T*k*max(inter, d)*s,
 * T*shared_inter*s and 2*max(inter, shared_inter)*d*s must be below 2^31
 * bytes (the expert GEMMs address operands with 32-bit byte offsets).
 */
int smoes_moe_forward(const smoes_layer* desc, const smoes_layer_io* io,
                      void* workspace, size_t workspace_bytes, void* stream);

/* Intermediate buffers inside the workspace of smoes_moe_forward. */
enum smoes_buffer {
    SMOES_BUF_H_ROUTED = 0,   /* [T*k, inter] act_dtype: silu(gate) * up of every routed row */
    SMOES_BUF_H_SHARED = 1,   /* [T, shared_inter] act_dtype: the same for the shared experts */
    SMOES_BUF_Y_ROUTED = 2,   /* [T*k, d] act_dtype: expert output of every routed row */
    SMOES_BUF_Y_SHARED = 3,   /* [T, d] act_dtype: shared experts' output (not written when the
                                 combine runs in the shared GEMM2's epilogue, see smoes_stage) */
    SMOES_BUF_CHECK_FLAGS = 4 /* [1] int32: flag word of check_inputs (SMOES_CHECK_* bits) */
};

/*
 * Device address (*ptr) and byte size (*bytes) of one intermediate buffer of
 * smoes_moe_forward inside `workspace` (the same pointer the forward got).
 * Routed rows are in the expert-contiguous order of expert_offsets /
 * perm_token (row r belongs to token perm_token[r]). The contents are those
 * of the last forward call on this workspace, once it has completed; they
 * stay valid until the workspace is reused. Host-side arithmetic only: no
 * device access. SMOES_ERR_ARG for a NULL pointer, an invalid desc or an
 * unknown `which`; the shared buffers have 0 bytes when shared_inter == 0.
 */
int smoes_workspace_buffer(const smoes_layer* desc, void* workspace, int which, void** ptr, size_t* bytes);

/* Bits of the input-check flag word. */
enum smoes_check_flag {
    SMOES_CHECK_MODALITY_ID = 1,    /* a modality id is neither 0 nor 1 */
    SMOES_CHECK_SAMPLE_OFFSETS = 2, /* offsets[0] != 0, offsets[n_batch] != T, or a decrease */
    SMOES_CHECK_EXPERT_TO_BIN = 4   /* a bin index outside [0, n_bins), or a bin without
                                       exactly E / n_bins experts */
};

/*
 * Debug check of the device-resident inputs of a layer call: io->modality_id
 * (when not NULL), io->sample_offsets (when not NULL) and io->expert_to_bin
 * are read on the device by one workgroup, and the OR of the violated
 * SMOES_CHECK_* bits (0 when all hold) is written to flags[0] (device int32).
 * Nothing else is read or written. With desc->check_inputs = 1,
 * smoes_moe_forward runs the same check as its first step and writes the flag
 * word into its workspace (SMOES_BUF_CHECK_FLAGS); the check reports, it does
 * not stop the later kernels: with a non-zero flag the outputs of that call
 * are undefined, and an out-of-range modality id or bin can make later
 * kernels read out of bounds, so untrusted inputs go through this call alone
 * first. Asynchronous on `stream`; SMOES_ERR_ARG for a NULL desc, io, flags
 * or io->expert_to_bin; desc errors as smoes_workspace_bytes.
 */
int smoes_check_inputs(const smoes_layer* desc, const smoes_layer_io* io, int32_t* flags, void* stream);

/* ------------------------------------------------------------------------ */
/* Packed expert weights (bf16). Same products and sums as the row-major    */
/* weights of smoes_layer_io, stored in the order the matrix cores read     */
/* them, so each GEMM streams its weights straight into registers.          */
/* ------------------------------------------------------------------------ */

/* Which expert weight tensor (shapes as in smoes_layer_io). */
enum smoes_weight {
    SMOES_W13 = 0, SMOES_W2 = 1, SMOES_WS13 = 2, SMOES_WS2 = 3, SMOES_WGATE = 4,
    /* transposed forms read by smoes_moe_backward */
    SMOES_W13T = 5, SMOES_W2T = 6, SMOES_WS13T = 7, SMOES_WS2T = 8
};

/*
 * Layout: a matrix W[N][K] (N output rows, K the contraction) becomes
 * 2*ceil(N/32) groups of 16 rows, each ceil(K/32) slices of 64 x 8 bf16:
 *   P[h][c][l][e] = W[16h + l%16][32c + 8(l/16) + e], zero outside W
 * (the operand order of the 16x16x32 matrix instructions).
 * w13/ws13: W = the gate and up rows interleaved by 16-row groups in blocks
 * of 32 columns (groups 4q..4q+3 = gate rows 32q..32q+15, up rows
 * 32q..32q+15, gate rows 32q+16..32q+31, up rows 32q+16..32q+31),
 * N = 2*32*ceil(inter/32), K = d; one matrix per expert, experts back to
 * back. w2/ws2: W = w2[e] ([d][inter]), N = d, K = inter.
 * SMOES_WGATE: the float32 router weights w_gate [E][d] as three bf16 terms
 * (hi, mid, lo: their sum reproduces each weight to ~2^-24), each stored as
 * ceil(E/16) groups of ceil(d/32) slices of 64 x 8 bf16,
 *   P[p][g][c][l][e] = term p of w_gate[16g + l%16][32c + 8(l/16) + e],
 * zero outside w_gate: the operand order of the 16x16x32 matrix instructions.
 * SMOES_W13T / SMOES_WS13T: W = the transpose of w13[e] / ws13 (N = d,
 * K = 2 inter, gate rows then up rows along K, no interleave);
 * SMOES_W2T / SMOES_WS2T: W = the transpose of w2[e] / ws2 (N = inter,
 * K = d). `src` is the same row-major tensor as for SMOES_W13 / SMOES_W2.
 * Returns the byte size of the packed tensor, 0 for an invalid desc or
 * `which` (ws13/ws2 need shared_inter > 0).
 */
size_t smoes_packed_weight_bytes(const smoes_layer* desc, int which);

/*
 * Pack one row-major bf16 weight tensor `src` (device, shape of `which` in
 * smoes_layer_io) into `dst` (device, smoes_packed_weight_bytes bytes, not
 * overlapping src). Asynchronous on `stream`. SMOES_ERR_ARG for a NULL
 * pointer, act_dtype != SMOES_BF16 or an invalid `which`; other desc errors
 * as smoes_workspace_bytes.
 */
int smoes_pack_weights(const smoes_layer* desc, int which, const void* src, void* dst, void* stream);

/* ------------------------------------------------------------------------ */
/* Layer backward (the training step of the supplementary cost table).      */
/* ------------------------------------------------------------------------ */

/* Gradients written by smoes_moe_backward (device pointers). */
typedef struct smoes_layer_grads {
    float* dx;       /* [T, d] float32: experts, shared experts and router       */
    float* dw_gate;  /* [E, d] float32 router weight gradient                    */
    float* dbias;    /* [E] float32 logit bias gradient, or NULL                 */
    float* dz;       /* [T, E] float32 total logit gradient (with dlogits_aux)   */
    float* dw;       /* [T, k] float32 combine-weight gradient, or NULL          */
    void* dw13;      /* [E, 2 inter, d] act_dtype (gate rows then up rows, as w13) */
    void* dw2;       /* [E, d, inter] act_dtype                                  */
    void* dws13;     /* [2 shared_inter, d] act_dtype (when shared_inter > 0)    */
    void* dws2;      /* [d, shared_inter] act_dtype                              */
} smoes_layer_grads;

/*
 * Bytes of the backward's workspace for desc (0 for an invalid desc): the
 * recomputed pre-activations and their gradients, each routed row's input
 * gradient and w H, and for bf16 layers with packed weights the k-packed
 * copies of the weight-gradient operands (each expert's rows padded to 16).
 * At T = 16384, d = 4096, 160 experts of inter 1536, top-6 and two shared
 * experts the copies take 2.2 GB and the whole workspace 4.4 GB (5.2 GB when
 * the forward did not keep the pre-activations). Host arithmetic only.
 */
size_t smoes_backward_workspace_bytes(const smoes_layer* desc);

/*
 * Gradients of a loss L through the layer output, given dout = dL/d out
 * ([T, d] act_dtype), after smoes_moe_forward ran with the same desc, io and
 * forward workspace (whose expert buffers, H and Y, and work tables must be
 * intact). The top-k choice carries no gradient; the gradient reaches the
 * router through the combine weights (the gate values at the chosen experts,
 * or their renormalised form) and the full softmax; dlogits_aux ([T, E]
 * float32, e.g. io->dlogits of the MI loss, plus the bin balance gradient),
 * when not NULL, is added to the logit gradient; the modality scores are
 * constants. The experts' gate and up pre-activations are read from the
 * forward workspace when desc->save_preact is 1 (the forward kept them),
 * else recomputed.
 * Reads from io: x, w13 and ws13 (packed when desc->weights_packed),
 * w2 and ws2 (row-major; fp32 layers and bf16 layers with row-major
 * weights), w_gate (float32 row-major), probs, topk_idx, topk_w, and
 * expert_offsets / perm_token / perm_inv (or the forward workspace's copies
 * when those are NULL).
 * w13t, w2t, ws13t, ws2t: the transposed packed weights (SMOES_W13T, ...),
 * read for bf16 layers with packed weights only (may be NULL otherwise).
 * Two paths: bf16 layers with packed weights run matrix-core GEMMs with bf16
 * operands and bf16 intermediates; fp32 layers and bf16 layers with
 * row-major weights run float32 FMA tiles with float32 intermediates, every
 * step on `stream` (io->streams is not used there). The expert weight
 * gradients are in act_dtype; dx, dw_gate and the logit gradient float32.
 * SMOES_ERR_SHAPE (packed path) when 4 T k inter or 4 T shared_inter exceeds
 * INT32_MAX bytes, or a k-packed operand copy (2 (T k + 15 E) max(d, 2 inter)
 * bytes, or 2 T max(d, 2 shared_inter) for the shared experts) would;
 * SMOES_ERR_WORKSPACE when either workspace is NULL or
 * smaller than smoes_workspace_bytes / smoes_backward_workspace_bytes;
 * SMOES_ERR_ARG for a NULL pointer that is needed. Differentiates the layer
 * output of Sec. 3.1 (softmax router, top-k combine, SwiGLU experts plus the
 * shared experts). Sums run in a fixed order: results are reproducible.
 * Asynchronous on `stream`; nothing is allocated. Packed path with
 * io->streams set and fewer than 65536 routed rows (T k): the router
 * backward, dW_gate / dbias and the shared experts' gradients run on
 * io->streams->side[1], forked from `stream` at the start of the call and
 * joined back before the input gradient (events[0] and events[3]); the
 * results are the same bits as on one stream. From 65536 routed rows, or with
 * NULL, every step runs on `stream` (there the routed GEMMs alone fill the
 * GPU and the side chain would only take compute units from them).
 */
int smoes_moe_backward(const smoes_layer* desc, const smoes_layer_io* io, const void* w13t, const void* w2t,
                       const void* ws13t, const void* ws2t, const void* dout, const float* dlogits_aux,
                       const smoes_layer_grads* grads, void* fwd_workspace, size_t fwd_workspace_bytes,
                       void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* GMM estimator: a K-component diagonal mixture per modality in place of   */
/* the single Gaussian of Sec. 3.2.2 (supplementary GMM ablation).           */
/* ------------------------------------------------------------------------ */

#define SMOES_GMM_K_MAX 4

size_t smoes_gmm_workspace_size(int64_t T, int d, int K);

/*
 * x            [T, d] activations (x_dtype).
 * modality_id  [T] uint8 hard labels (0 vision, 1 text); needed when update
 *              = 1 or resp != NULL.
 * gmm_n        [2, K] float32 EMA counts N_mc (device, read/write).
 * gmm_smu      [2, K, d] float32 S_mu per component (device, read/write).
 * gmm_ssig     [2, K, d] float32 S_sigma2 per component (device, read/write).
 *              Row m = 0 is vision, 1 text. Mixture weights are
 *              pi_mc = N_mc / sum_c N_mc (uniform for a modality with no
 *              count); a component with N = 0 has mu = 0, sigma^2 = 1. The
 *              caller seeds the components apart (identical components stay
 *              identical under EM).
 * update       1: one stepwise-EM step first: responsibilities of each
 *              token's own modality under the current parameters, then Eq.
 *              5-7 per component with the responsibility-weighted batch
 *              count, mean and centred sum of squares (decay beta); 0: score
 *              only.
 * tau          temperature of Eq. 9; <= 0 selects 0.5 * d.
 * var_floor    lower bound of sigma^2 (>= 0).
 * M            [T, 2] float32 output: Eq. 9 with LL_m the log of the
 *              mixture density (2 pi constant dropped); rows sum to 1.
 * resp         [T, K] float32 output or NULL: the responsibilities of the
 *              E-step (parameters before the update).
 * K = 1 is the single-Gaussian score of smoes_modality_score.
 * Shapes: 1 <= K <= SMOES_GMM_K_MAX, 1 <= d <= SMOES_D_MAX, d % 8 == 0.
 * Sums are float64 in a fixed order: results are reproducible.
 */
int smoes_gmm_modality_score(const void* x, int x_dtype, int64_t T, int d, int K,
                             const uint8_t* modality_id, float* gmm_n, float* gmm_smu,
                             float* gmm_ssig, int update, float beta, float tau, float var_floor,
                             float* M, float* resp, void* workspace, size_t workspace_bytes,
                             void* stream);

/* ------------------------------------------------------------------------ */
/* Attention-accumulated modality score (Sec. 3.2.1, Eq. 2-4).               */
/* ------------------------------------------------------------------------ */

/*
 * Layer-0 scores (Eq. 2): M[j] = (1, 0) for a vision token (modality_id 0),
 * (0, 1) for a text token (1), (0, 0) for any other label.
 * modality_id  [T] uint8 (device).   M  [T, 2] float32 output (device).
 * Asynchronous on `stream`; SMOES_ERR_ARG for a NULL pointer with T > 0.
 */
int smoes_attn_score_init(const uint8_t* modality_id, int64_t T, float* M, void* stream);

/*
 * Causal softmax attention inside each sample (a sample never attends to
 * another; within a sample token j attends to tokens <= j), per query head h,
 * with the modality scores carried as two extra value channels (the
 * supplementary implementation note; here accumulated in float32):
 *   o[j][h]       = sum_j' Attn_h(j, j') v[j'][h_kv]               (bf16)
 *   m_heads[j][h] = sum_j' Attn_h(j, j') m_in[j']                   (Eq. 3
 *                   before the head average; float32, 2 columns)
 * with Attn_h(j, .) = softmax over j' of scale * q[j][h] . k[j'][h_kv] and
 * h_kv = h / (n_heads / n_kv_heads) (grouped KV heads).
 * q            [T, n_heads, head_dim] bf16 (device, row-major).
 * k, v         [T, n_kv_heads, head_dim] bf16 (device).
 * sample_offsets [n_batch + 1] int32 (device): 0 = off[0] <= ... <= off[n_batch] = T.
 * m_in         [T, 2] float32 scores of this layer's input (column 0 vision).
 * scale        logit scale; <= 0 selects 1 / sqrt(head_dim).
 * o            [T, n_heads, head_dim] bf16 output (device).
 * m_heads      [T, n_heads, 2] float32 output (device).
 * Shapes: head_dim in {64, 128}; n_heads % n_kv_heads == 0;
 * T * n_heads * head_dim * 2 < 2^31. Sums run in a fixed order: results are
 * reproducible. Asynchronous on `stream`; nothing is allocated.
 */
int smoes_attention_scores(const void* q, const void* k, const void* v, int64_t T, int n_heads,
                           int n_kv_heads, int head_dim, const int32_t* sample_offsets, int n_batch,
                           const float* m_in, float scale, void* o, float* m_heads, void* stream);

/*
 * Head average (Eq. 3) and norm-weighted residual mix (Eq. 4):
 *   M_tilde[j] = (1 / n_heads) sum_h m_heads[j][h]
 *   m_out[j]   = (|x_attn[j]| M_tilde[j] + |x[j]| m_in[j]) / (|x_attn[j]| + |x[j]|)
 * with Euclidean norms over d; a token with both norms 0 keeps m_in[j].
 * x            [T, d] residual input of the attention sublayer (act_dtype).
 * x_attn       [T, d] attention sublayer output added to it (act_dtype).
 * m_heads      [T, n_heads, 2] float32 from smoes_attention_scores.
 * m_in, m_out  [T, 2] float32; m_out may equal m_in (updated in place).
 * Shapes: 1 <= d <= SMOES_D_MAX, d % 8 == 0. Asynchronous on `stream`.
 */
int smoes_attn_score_update(const void* x, const void* x_attn, int act_dtype, int64_t T, int d,
                            const float* m_heads, int n_heads, const float* m_in, float* m_out,
                            void* stream);

/* ------------------------------------------------------------------------ */
/* Timing helpers for stage_events (hipEvent_t handles behind void*).        */
/* ------------------------------------------------------------------------ */

/* Two non-blocking streams of default priority and four untimed events on
 * the current device, for smoes_layer_io.streams. Destroy with
 * smoes_streams_destroy (after their work has completed). */
int smoes_streams_create(smoes_streams* st);
int smoes_streams_destroy(smoes_streams* st);

int smoes_events_create(int n, void** events);
int smoes_events_destroy(int n, void** events);
/* Milliseconds between two recorded events (synchronises on `end`). */
int smoes_event_elapsed_ms(void* start, void* end, float* ms);

#ifdef __cplusplus
}
#endif

#endif /* SMOES_H */
