// Layer backward: the router and gather kernels around the expert GEMMs.
//
//  row_weights: the combine weight of each routed row (row r = inv(j, s)).
//  router_bwd: one wave per token: dw_js = <dout_j, Y[inv(j, s)]> (float32
//     sums, fixed butterfly), the gate gradient at the chosen experts (through
//     the renormalisation when it is on), the softmax backward
//     dz_je = g_je (dg_je - sum_e' g_je' dg_je'), plus the auxiliary logit
//     gradients (MI, bin balance) when given.
//  dx_gather: dx_j = dz_j W_gate + sum_s dX[inv(j, s)] + dXs_j in float32, in
//     that order (8 tokens x 1024 columns per block, dz staged in LDS).
//  dwgate: dW_gate[e][c] = sum_j dz_je x_jc and dbias_e = sum_j dz_je: per
//     256-token chunk partials, then a chunk-ordered sum.
#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

constexpr int kDxTok = 8;
constexpr int kDwChunk = 256;  // tokens per dwgate partial
constexpr int kDwExp = 16;     // experts per dwgate block

__global__ void row_weights_kernel(const int32_t* __restrict__ inv, const float* __restrict__ topk_w, int64_t n,
                                   float* __restrict__ wrow) {
    for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x)
        wrow[inv[i]] = topk_w[i];
}

template <bool BF16>
__global__ void __launch_bounds__(256)
router_bwd_kernel(const void* __restrict__ dout, const void* __restrict__ y_r, const int32_t* __restrict__ inv,
                  const float* __restrict__ probs, const int32_t* __restrict__ topk_idx,
                  const float* __restrict__ topk_w, const float* __restrict__ aux, int64_t T, int d, int E, int k,
                  int renorm, float* __restrict__ dw, float* __restrict__ dz) {
    const int64_t j = static_cast<int64_t>(blockIdx.x) * 4 + threadIdx.x / kWave;
    if (j >= T) return;  // whole waves
    const int lane = lane_id();
    // dw_s = <dout_j, Y[inv(j, s)]>: one pass over the columns loads dout once
    // and every slot's row chunk; each slot's partial runs over the columns in
    // order
    float dws[SMOES_K_MAX_DEV];
    int64_t rows[SMOES_K_MAX_DEV];
#pragma unroll
    for (int s = 0; s < SMOES_K_MAX_DEV; ++s) {
        rows[s] = s < k ? static_cast<int64_t>(inv[j * k + s]) : 0;
        dws[s] = 0.0f;
    }
    for (int c = lane * 8; c < d; c += kWave * 8) {
        float a[8];
        load8<BF16>(dout, j * d + c, a);
#pragma unroll
        for (int s = 0; s < SMOES_K_MAX_DEV; ++s) {
            if (s >= k) break;
            float y[8];
            load8<BF16>(y_r, rows[s] * d + c, y);
#pragma unroll
            for (int e = 0; e < 8; ++e) dws[s] = fmaf(a[e], y[e], dws[s]);
        }
    }
    for (int s = 0; s < k; ++s) dws[s] = wave_sum_u(dws[s]);
    // gradient at the chosen experts: dw itself, or through w = g_sel / S
    float dsel[SMOES_K_MAX_DEV], gsel[SMOES_K_MAX_DEV];
    float S = 0.0f, wd = 0.0f;
    for (int s = 0; s < k; ++s) {
        gsel[s] = probs[j * E + topk_idx[j * k + s]];
        S += gsel[s];
        wd += topk_w[j * k + s] * dws[s];
    }
    float gdg = 0.0f;  // sum_e g_e dg_e: only the chosen experts carry dg
    for (int s = 0; s < k; ++s) {
        dsel[s] = renorm ? (dws[s] - wd) / S : dws[s];
        gdg += gsel[s] * dsel[s];
    }
    for (int e = lane; e < E; e += kWave) {
        float dg = 0.0f;
        for (int s = 0; s < k; ++s)
            if (topk_idx[j * k + s] == e) dg += dsel[s];
        float v = probs[j * E + e] * (dg - gdg);
        if (aux != nullptr) v += aux[j * E + e];
        dz[j * E + e] = v;
    }
    if (dw != nullptr && lane == 0)
        for (int s = 0; s < k; ++s) dw[j * k + s] = dws[s];
}

// Each thread: 4 adjacent columns of kDxTok tokens (8-byte loads of bf16 row
// gradients or 16-byte loads of float32 ones, 16 bytes of W_gate per expert).
template <bool BF16>
__global__ void __launch_bounds__(256)
dx_gather_kernel(const void* __restrict__ dx_r, const void* __restrict__ dx_s, const int32_t* __restrict__ inv,
                 const float* __restrict__ dz, const float* __restrict__ w_gate, int64_t T, int d, int E, int k,
                 float* __restrict__ dx) {
    extern __shared__ float dz_s[];  // [kDxTok][E]
    const int64_t j0 = static_cast<int64_t>(blockIdx.x) * kDxTok;
    const int c = (blockIdx.y * 256 + threadIdx.x) * 4;
    const int nt = static_cast<int>(T - j0 < kDxTok ? T - j0 : kDxTok);
    for (int i = threadIdx.x; i < kDxTok * E; i += 256) {
        const int t = i / E;
        dz_s[i] = t < nt ? dz[(j0 + t) * E + i % E] : 0.0f;
    }
    __syncthreads();
    if (c >= d) return;
    float acc[kDxTok][4];
#pragma unroll
    for (int t = 0; t < kDxTok; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[t][q] = 0.0f;
    for (int e = 0; e < E; ++e) {
        const float4 w = *reinterpret_cast<const float4*>(w_gate + static_cast<int64_t>(e) * d + c);
#pragma unroll
        for (int t = 0; t < kDxTok; ++t) {
            const float z = dz_s[t * E + e];
            acc[t][0] = fmaf(z, w.x, acc[t][0]);
            acc[t][1] = fmaf(z, w.y, acc[t][1]);
            acc[t][2] = fmaf(z, w.z, acc[t][2]);
            acc[t][3] = fmaf(z, w.w, acc[t][3]);
        }
    }
    // the four columns of row r of a row-gradient matrix, added onto v
    auto add4 = [&](float (&v)[4], const void* m, int64_t r) {
        if constexpr (BF16) {
            const uint2 u = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(m) + r * d + c);
            v[0] += __uint_as_float(u.x << 16);
            v[1] += __uint_as_float(u.x & 0xffff0000u);
            v[2] += __uint_as_float(u.y << 16);
            v[3] += __uint_as_float(u.y & 0xffff0000u);
        } else {
            const float4 u = *reinterpret_cast<const float4*>(static_cast<const float*>(m) + r * d + c);
            v[0] += u.x;
            v[1] += u.y;
            v[2] += u.z;
            v[3] += u.w;
        }
    };
#pragma unroll
    for (int t = 0; t < kDxTok; ++t) {
        if (t >= nt) break;
        const int64_t j = j0 + t;
        float v[4] = {acc[t][0], acc[t][1], acc[t][2], acc[t][3]};
        for (int s2 = 0; s2 < k; ++s2) add4(v, dx_r, static_cast<int64_t>(inv[j * k + s2]));
        if (dx_s != nullptr) add4(v, dx_s, j);
        *reinterpret_cast<float4*>(dx + j * d + c) = make_float4(v[0], v[1], v[2], v[3]);
    }
}

// partial[chunk][e][c] = sum over the chunk's tokens of dz[j][e] x[j][c]; bias
// partials by the blocks of column tile 0.
template <bool BF16>
__global__ void __launch_bounds__(256)
dwgate_partial_kernel(const float* __restrict__ dz, const void* __restrict__ x, int64_t T, int d, int E,
                      float* __restrict__ part, float* __restrict__ bpart) {
    __shared__ float dz_s[kDwChunk][kDwExp];
    const int c = blockIdx.x * 256 + threadIdx.x;
    const int e0 = blockIdx.y * kDwExp;
    const int64_t chunk = blockIdx.z;
    const int64_t j0 = chunk * kDwChunk;
    const int nt = static_cast<int>(T - j0 < kDwChunk ? T - j0 : kDwChunk);
    for (int i = threadIdx.x; i < kDwChunk * kDwExp; i += 256) {
        const int t = i / kDwExp, e = e0 + i % kDwExp;
        dz_s[t][i % kDwExp] = (t < nt && e < E) ? dz[(j0 + t) * E + e] : 0.0f;
    }
    __syncthreads();
    if (blockIdx.x == 0 && threadIdx.x < kDwExp && e0 + static_cast<int>(threadIdx.x) < E) {
        float b = 0.0f;
        for (int t = 0; t < nt; ++t) b += dz_s[t][threadIdx.x];
        bpart[chunk * E + e0 + threadIdx.x] = b;
    }
    if (c >= d) return;
    float acc[kDwExp];
#pragma unroll
    for (int e = 0; e < kDwExp; ++e) acc[e] = 0.0f;
    for (int t = 0; t < nt; ++t) {
        const float xv = BF16 ? bf16_to_f32(static_cast<const uint16_t*>(x)[(j0 + t) * d + c])
                              : static_cast<const float*>(x)[(j0 + t) * d + c];
#pragma unroll
        for (int e = 0; e < kDwExp; ++e) acc[e] = fmaf(dz_s[t][e], xv, acc[e]);
    }
#pragma unroll
    for (int e = 0; e < kDwExp; ++e)
        if (e0 + e < E) part[(chunk * E + e0 + e) * d + c] = acc[e];
}

__global__ void dwgate_reduce_kernel(const float* __restrict__ part, const float* __restrict__ bpart, int64_t nchunk,
                                     int d, int E, float* __restrict__ dw_gate, float* __restrict__ dbias) {
    const int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x;
    if (i < static_cast<int64_t>(E) * d) {
        float acc = 0.0f;
        for (int64_t ch = 0; ch < nchunk; ++ch) acc += part[ch * E * d + i];
        dw_gate[i] = acc;
    }
    if (dbias != nullptr && i < E) {
        float acc = 0.0f;
        for (int64_t ch = 0; ch < nchunk; ++ch) acc += bpart[ch * E + i];
        dbias[i] = acc;
    }
}

}  // namespace

size_t router_bwd_workspace_bytes(int64_t T, int d, int E) {
    const int64_t nchunk = ceil_div(T, kDwChunk);
    return align_up(sizeof(float) * nchunk * E * d, 256) + align_up(sizeof(float) * nchunk * E, 256);
}

hipError_t launch_row_weights(const int32_t* perm_inv, const float* topk_w, int64_t T, int k, float* wrow,
                              hipStream_t stream) {
    const int64_t n = T * k;
    if (n == 0) return hipSuccess;
    const int64_t b = ceil_div(n, 256);
    hipLaunchKernelGGL(row_weights_kernel, dim3(static_cast<unsigned>(b < 4096 ? b : 4096)), dim3(256), 0, stream,
                       perm_inv, topk_w, n, wrow);
    return hipGetLastError();
}

hipError_t launch_router_bwd(const void* dout, const void* y_r, int bf16, const int32_t* perm_inv,
                             const float* probs, const int32_t* topk_idx, const float* topk_w,
                             const float* dlogits_aux, int64_t T, int d, int E, int k, int renorm, float* dw,
                             float* dz, hipStream_t stream) {
    if (T == 0) return hipSuccess;
    const dim3 grid(static_cast<unsigned>(ceil_div(T, 4)));
    if (bf16)
        hipLaunchKernelGGL(router_bwd_kernel<true>, grid, dim3(256), 0, stream, dout, y_r, perm_inv, probs, topk_idx,
                           topk_w, dlogits_aux, T, d, E, k, renorm, dw, dz);
    else
        hipLaunchKernelGGL(router_bwd_kernel<false>, grid, dim3(256), 0, stream, dout, y_r, perm_inv, probs, topk_idx,
                           topk_w, dlogits_aux, T, d, E, k, renorm, dw, dz);
    return hipGetLastError();
}

hipError_t launch_dx_gather(const void* dx_r, const void* dx_s, int bf16, const int32_t* perm_inv, const float* dz,
                            const float* w_gate, int64_t T, int d, int E, int k, float* dx, hipStream_t stream) {
    if (T == 0) return hipSuccess;
    const dim3 grid(static_cast<unsigned>(ceil_div(T, kDxTok)), static_cast<unsigned>(ceil_div(d, 256 * 4)));
    const size_t lds = sizeof(float) * kDxTok * E;
    if (bf16)
        hipLaunchKernelGGL(dx_gather_kernel<true>, grid, dim3(256), lds, stream, dx_r, dx_s, perm_inv, dz, w_gate, T, d,
                           E, k, dx);
    else
        hipLaunchKernelGGL(dx_gather_kernel<false>, grid, dim3(256), lds, stream, dx_r, dx_s, perm_inv, dz, w_gate, T,
                           d, E, k, dx);
    return hipGetLastError();
}

hipError_t launch_dwgate(const float* dz, const void* x, int bf16, int64_t T, int d, int E, float* dw_gate,
                         float* dbias, void* ws, hipStream_t stream) {
    const int64_t nchunk = ceil_div(T, kDwChunk);
    float* part = static_cast<float*>(ws);
    float* bpart = reinterpret_cast<float*>(static_cast<char*>(ws) + align_up(sizeof(float) * nchunk * E * d, 256));
    hipError_t err;
    if (nchunk > 0) {
        const dim3 grid(static_cast<unsigned>(ceil_div(d, 256)), static_cast<unsigned>(ceil_div(E, kDwExp)),
                        static_cast<unsigned>(nchunk));
        if (bf16)
            hipLaunchKernelGGL(dwgate_partial_kernel<true>, grid, dim3(256), 0, stream, dz, x, T, d, E, part, bpart);
        else
            hipLaunchKernelGGL(dwgate_partial_kernel<false>, grid, dim3(256), 0, stream, dz, x, T, d, E, part, bpart);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    const int64_t n = static_cast<int64_t>(E) * d;
    hipLaunchKernelGGL(dwgate_reduce_kernel, dim3(static_cast<unsigned>(ceil_div(n, 256))), dim3(256), 0, stream, part,
                       bpart, nchunk, d, E, dw_gate, dbias);
    return hipGetLastError();
}

}  // namespace smoes
