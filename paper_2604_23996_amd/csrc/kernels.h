// Internal launchers of the SMoES kernels (host side). Every launcher enqueues
// on `stream` and returns the launch status; sizes are validated by the C ABI
// layer before any launcher runs.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace smoes {

// ---------------------------------------------------------------- router
size_t router_workspace_bytes(int64_t T, int d, int E, int x_dtype);
// w_split: router weights already in the split fragment order of
// launch_split_wgate (bf16 x only), or NULL to split w_gate into ws first
hipError_t launch_route(const void* x, int x_dtype, int64_t T, int d, const float* w_gate,
                        const void* w_split, const float* bias, int E, int k, int renorm, float* logits,
                        float* probs, int32_t* topk_idx, float* topk_w, void* ws, hipStream_t stream);
size_t router_packed_elems(int d, int E);
hipError_t launch_split_wgate(const float* w_gate, int E, int d, void* wpk, hipStream_t stream);

// ---------------------------------------------------------------- modality score
size_t modality_workspace_bytes(int64_t T, int d);
hipError_t launch_modality(const void* x, int x_dtype, int64_t T, int d, const uint8_t* modality_id,
                           float* gauss_n, float* gauss_smu, float* gauss_ssig, int update,
                           float beta, float tau, float var_floor, float* M, void* ws,
                           hipStream_t stream);

// ---------------------------------------------------------------- MI loss
size_t mi_workspace_bytes(int64_t T, int E, int n_batch, int n_bins);
hipError_t launch_mi(const float* probs, const float* M, int64_t T, int E,
                     const int32_t* sample_offsets, int n_batch, const int32_t* expert_to_bin,
                     int n_bins, float grad_scale, float* mi_per_sample, float* loss,
                     float* dlogits, void* ws, hipStream_t stream);

// ---------------------------------------------------------------- permutation
size_t permute_workspace_bytes(int64_t T, int E, int k);
// Work tables of the grouped GEMMs (filled by the permutation, which knows
// the per-expert row counts): work[g + 1] = work[g] + m_tiles(g) * n_tiles.
struct WorkTables {
    int32_t* work1;  // [E + 2] GEMM1 (NULL: not wanted)
    int32_t* work2;  // [E + 2] GEMM2
    int bm, nt1_r, nt1_s, nt2, has_shared;
};
hipError_t launch_permute(const int32_t* topk_idx, int64_t T, int E, int k,
                          int32_t* expert_offsets, int32_t* perm_token, int32_t* perm_inv,
                          void* ws, const WorkTables* work, hipStream_t stream);
hipError_t launch_gather_rows(const void* x, int x_dtype, int d, const int32_t* perm_token,
                              int64_t R, void* x_perm, hipStream_t stream);

// ---------------------------------------------------------------- experts
struct ExpertArgs {
    int64_t T;
    int d, E, k, inter, shared_inter, act_dtype;
    int packed;  // bf16 expert weights in the fragment order of launch_pack_weights
    const void* x;
    const void* w13;
    const void* w2;
    const void* ws13;
    const void* ws2;
    const int32_t* expert_offsets;  // [E + 1]
    const int32_t* perm_token;      // [T * k]
    const int32_t* perm_inv;        // [T, k]
    const float* topk_w;            // [T, k]
    void* out;                      // [T, d]
    void* ab_r;                     // NULL, or [T k][2 inter]: GEMM1 also keeps the gate | up
    void* ab_s;                     //   pre-activations (packed bf16 path); [T][2 shared_inter]
};
size_t experts_workspace_bytes(int64_t T, int d, int E, int k, int inter, int shared_inter,
                               int act_dtype);
// work tables of both grouped GEMMs: where they live and their tiling
WorkTables experts_work_tables(const ExpertArgs& a, void* ws);
// part: 0 every work item, 1 the routed experts only, 2 the shared expert only
// (the two parts can run on different streams once the work tables exist;
// the shared items' entries in the tables do not depend on the routing)
hipError_t launch_experts_gemm1(const ExpertArgs& a, void* ws, int part, hipStream_t stream);
hipError_t launch_experts_gemm2(const ExpertArgs& a, void* ws, int part, hipStream_t stream);
// The shared experts' GEMM2 with the combine in its epilogue (bf16, packed
// weights, shared experts present): writes `out`, not Y_s; every routed row
// of Y_r must be written before it runs.
hipError_t launch_experts_gemm2_combine(const ExpertArgs& a, void* ws, hipStream_t stream);
hipError_t launch_experts_combine(const ExpertArgs& a, void* ws, hipStream_t stream);
// packed bf16 expert weights: elements of `batch` packed n x k matrices
// (interleave: gate and up halves of a 2n-row source)
int64_t packed_weight_elems(int batch, int n, int k, int interleave);
hipError_t launch_pack_weights(const void* src, int batch, int n, int k, int interleave, int transpose, void* dst,
                               hipStream_t stream);

// Momentum-adaptive binning, bin-level load balance loss (+ logit gradient) and MSI
size_t binning_workspace_bytes(int64_t T, int E, int n_bins);
hipError_t launch_binning(const float* probs, const int32_t* topk_idx, const uint8_t* modality_id, int64_t T,
                          int E, int k, const int32_t* expert_to_bin, int n_bins, float beta, double* load_ema,
                          int32_t* counts, double* f_spec, int32_t* expert_to_bin_next, float grad_scale,
                          float* bal_loss, float* dlogits, int accumulate, float* msi, void* ws,
                          hipStream_t stream);

// ---------------------------------------------------------------- layer backward
// The forward's expert buffers inside its workspace (H, Y and the work tables).
struct ExpertFwdBuffers {
    void* h_r;
    void* h_s;
    void* y_r;
    void* y_s;
    int32_t* work1;
    int32_t* work2;
};
ExpertFwdBuffers experts_fwd_buffers(const ExpertArgs& a, void* ws);
struct BwdGemmPtrs {
    const void* dout;   // [T][d]
    const void* w2t;    // packed W2^T per expert
    const void* ws2t;
    const void* w13t;   // packed W13^T per expert
    const void* ws13t;
    void* ab_r;         // [R][2 inter]
    void* ab_s;         // [T][2 shared_inter]
    void* dab_r;
    void* dab_s;
    void* dx_r;         // [R][d]
    void* dx_s;         // [T][d]
    const float* wrow;  // [R]
    void* wh_r;         // [R][inter] w H of the routed rows (written by mode 4)
    int32_t* work4;     // [E + 2] table of mode 4
};
// mode 3: recomputed gate/up pre-activations; 4: dH = w dout W2 with the SwiGLU
// backward -> [dA dB] (and w H for routed rows); 5: dX = [dA dB] W13. part: 1
// routed, 2 shared.
hipError_t launch_bwd_gemm(int mode, const ExpertArgs& a, void* fwd_ws, const BwdGemmPtrs& bp, int part,
                           hipStream_t stream);
// Backward of fp32 layers and of bf16 layers with row-major weights: float32
// FMA tiles, float32 intermediates, weight gradients in the layer dtype.
struct GenericBwdPtrs {
    const void* dout;   // [T][d] layer dtype
    float* ab_r;        // [R][2 inter] gate | up pre-activations
    float* ab_s;        // [T][2 shared_inter]
    float* dab_r;       // their gradients
    float* dab_s;
    float* wh_r;        // [R][inter] w H
    float* wh_s;        // [T][shared_inter] H
    float* dx_r;        // [R][d]
    float* dx_s;        // [T][d]
    const float* wrow;  // [R] combine weight of each routed row
    int32_t* work;      // [E + 2] work table, rebuilt by each row step
    void* dw13;
    void* dw2;
    void* dws13;
    void* dws2;
};
// step 0: pre-activations; 1: dH and the SwiGLU backward (dA dB, w H); 2: dX;
// 3: dW2 and dWs2; 4: dW13 and dWs13. Routed and shared experts in one launch.
hipError_t launch_generic_bwd(int step, const ExpertArgs& a, const GenericBwdPtrs& bp, hipStream_t stream);
// k-packed operands (fragment order, rows contiguous, each group padded to 16
// rows) and the weight gradients from them: kp = padded row prefix of the
// groups given by off; kpack_elems = elements of a packed copy of C columns.
int64_t kpack_elems(int C, int64_t padded_rows);
// ranges (may be NULL): [2][9] first tiles of the 8 XCDs' work-balanced tile
// ranges for two launch_wgrad_pk calls over these groups with per0 and per1
// tiles per group (wgrad_tiles_per_group). 1 <= E <= 256.
int wgrad_tiles_per_group(int M, int N);
hipError_t launch_kpad_offsets(const int32_t* off, int E, int32_t* kp, int per0, int per1, int32_t* ranges,
                               hipStream_t stream);
// S [.][C] bf16 row-major; group g's rows are off[g] .. off[g + 1] (through map
// when given); off == NULL: one group of T rows. max_padded_rows bounds kp's
// total (the grid).
hipError_t launch_kpack(const void* S, int C, const int32_t* map, const int32_t* off, const int32_t* kp,
                        int n_groups, int64_t T, int64_t max_padded_rows, void* P, hipStream_t stream);
// out[g][m][n] = sum over group g's rows of A[row][m] B[row][n] (bf16), from the
// k-packed A (M columns) and B (N columns); kp == NULL: one group of T rows;
// ranges: 9 entries from launch_kpad_offsets, or NULL: equal tile counts per XCD.
hipError_t launch_wgrad_pk(int n_groups, int M, int N, const int32_t* kp, const int32_t* ranges, int64_t T,
                           const void* PA, const void* PB, void* out, hipStream_t stream);
size_t router_bwd_workspace_bytes(int64_t T, int d, int E, int bf16);  // bf16: x is bf16 (launch_dwgate)
hipError_t launch_row_weights(const int32_t* perm_inv, const float* topk_w, int64_t T, int k, float* wrow,
                              hipStream_t stream);
// bf16: dout and y_r (router_bwd), the row gradients dx_r / dx_s (dx_gather), x (dwgate) are
// bf16, else float32
hipError_t launch_router_bwd(const void* dout, const void* y_r, int bf16, const int32_t* perm_inv,
                             const float* probs, const int32_t* topk_idx, const float* topk_w,
                             const float* dlogits_aux, int64_t T, int d, int E, int k, int renorm, float* dw,
                             float* dz, hipStream_t stream);
// ws (bf16 only; NULL: the FMA kernel): dx_mfma_workspace_bytes for the packed W_gate and dz fragments
size_t dx_mfma_workspace_bytes(int64_t T, int d, int E);
hipError_t launch_dx_gather(const void* dx_r, const void* dx_s, int bf16, const int32_t* perm_inv, const float* dz,
                            const float* w_gate, int64_t T, int d, int E, int k, float* dx, void* ws,
                            hipStream_t stream);
hipError_t launch_dwgate(const float* dz, const void* x, int bf16, int64_t T, int d, int E, float* dw_gate,
                         float* dbias, void* ws, hipStream_t stream);

// ---------------------------------------------------------------- input checks
// One block: bitmask of violated device-resident preconditions (SMOES_CHECK_*) into flags[0].
hipError_t launch_check_inputs(const uint8_t* modality_id, int64_t T, const int32_t* sample_offsets, int n_batch,
                               const int32_t* expert_to_bin, int E, int n_bins, int32_t* flags,
                               hipStream_t stream);

// ---------------------------------------------------------------- GMM estimator
size_t gmm_workspace_bytes(int64_t T, int d, int K);
hipError_t launch_gmm(const void* x, int x_dtype, int64_t T, int d, int K, const uint8_t* modality_id, float* gmm_n,
                      float* gmm_smu, float* gmm_ssig, int update, float beta, float tau, float var_floor, float* M,
                      float* resp, void* ws, hipStream_t stream);

// ---------------------------------------------------------------- attention-accumulated score
hipError_t launch_attention(const void* q, const void* k, const void* v, int64_t T, int H, int Hkv, int head_dim,
                            const int32_t* sample_offsets, int n_batch, const float* m_in, float scale, void* o,
                            float* m_heads, hipStream_t stream);
hipError_t launch_attn_update(const void* x, const void* x_attn, int act_dtype, int64_t T, int d,
                              const float* m_heads, int H, const float* m_in, float* m_out, hipStream_t stream);
hipError_t launch_attn_init(const uint8_t* modality_id, int64_t T, float* M, hipStream_t stream);

}  // namespace smoes
