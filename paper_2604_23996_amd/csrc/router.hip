// Router: logits z = W_gate x (+ b), full softmax g and top-k (Sec. 3.1).
//
// One workgroup (8 waves) owns 32 tokens and every expert. For bf16
// activations the logits are fp32-faithful on the matrix cores: the fp32
// router weights are split into three bf16 terms (hi + mid + lo reproduces
// the weight to ~2^-24), each product with the exact bf16 activation is exact,
// and v_mfma_f32_32x32x16_bf16 accumulates in fp32. The eight waves split the
// hidden dimension; their partial tiles are summed in LDS in a fixed order,
// then every wave runs the softmax and a wave-wide top-k for 4 tokens.
// For fp32 activations the dot products are accumulated in fp64.
#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

constexpr int kRouterTokens = 32;
constexpr int kRouterWaves = 8;
constexpr int kRouterThreads = kRouterWaves * 64;
constexpr size_t kRouterLdsMax = 65536;

// Tree buffers that fit the LDS budget: up to 4, at least 2.
__host__ __device__ inline int router_slots(int E_pad) {
    const int per = kRouterTokens * E_pad * static_cast<int>(sizeof(float));
    const int s = static_cast<int>(kRouterLdsMax / per);
    return s >= 4 ? 4 : (s < 2 ? 2 : s);
}

// w_gate [E, d] f32 -> wsplit [3][E_pad][d] bf16 (hi, mid, lo); rows >= E are zero.
__global__ void split_wgate_kernel(const float* __restrict__ w, int E, int E_pad, int d,
                                   uint16_t* __restrict__ wsplit) {
    const int64_t n = static_cast<int64_t>(E_pad) * d;
    for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int e = static_cast<int>(i / d);
        float v = e < E ? w[i] : 0.0f;
        const uint16_t hi = f32_to_bf16(v);
        const float r1 = v - bf16_to_f32(hi);
        const uint16_t mid = f32_to_bf16(r1);
        const float r2 = r1 - bf16_to_f32(mid);
        const uint16_t lo = f32_to_bf16(r2);
        wsplit[i] = hi;
        wsplit[n + i] = mid;
        wsplit[2 * n + i] = lo;
    }
}

// Logits of one wave over its share of the hidden dimension (k-steps
// s = wave, wave + 8, ...), bf16x3 MFMA with the next step's fragments
// loaded before the current step's MFMAs; then a fixed-order tree over the 8
// waves through LDS (wave w adds wave w + half, half = 4, 2, 1), using `slots`
// buffers of [32][E_pad] floats. The logits end in buffer 0.
// Output layout of a 32x32 MFMA tile (lane l, element v):
//   column = l % 32, row = 8 * (v / 4) + 4 * (l / 32) + (v % 4).
template <int NT>
__device__ void router_mfma_logits(const uint16_t* __restrict__ x, int64_t T, int d,
                                   const uint16_t* __restrict__ wsplit, int E_pad,
                                   int64_t tok0, int wave, int slots, float* __restrict__ buf) {
    const int lane = lane_id();
    const int half = lane >> 5;
    const int r = lane & 31;
    int64_t tok = tok0 + r;
    if (tok >= T) tok = T - 1;
    const uint16_t* xrow = x + tok * d;
    const int64_t part = static_cast<int64_t>(E_pad) * d;
    f32x16_t acc[NT];
#pragma unroll
    for (int n = 0; n < NT; ++n) acc[n] = f32x16_t{};
    const int nsteps = static_cast<int>(ceil_div(d, 16));
    bf16x8_t a_cur = {}, b_cur[NT][3];
    auto fetch = [&](int s, bf16x8_t& a, bf16x8_t (&b)[NT][3]) {
        const int kk = s * 16 + half * 8;
        const bool valid = s < nsteps && kk < d;  // d % 8 == 0: an 8-chunk is all in or all out
        a = valid ? *reinterpret_cast<const bf16x8_t*>(xrow + kk) : bf16x8_t{};
#pragma unroll
        for (int n = 0; n < NT; ++n) {
            const int64_t off = static_cast<int64_t>(n * 32 + r) * d + kk;
#pragma unroll
            for (int p = 0; p < 3; ++p)
                b[n][p] = valid ? *reinterpret_cast<const bf16x8_t*>(wsplit + p * part + off) : bf16x8_t{};
        }
    };
    auto mfma3 = [&](const bf16x8_t& a, const bf16x8_t (&b)[NT][3]) {
#pragma unroll
        for (int n = 0; n < NT; ++n) {
            acc[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b[n][2], acc[n], 0, 0, 0);  // lo
            acc[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b[n][1], acc[n], 0, 0, 0);  // mid
            acc[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b[n][0], acc[n], 0, 0, 0);  // hi
        }
    };
    if constexpr (NT <= 5) {  // register double buffer: next step's loads overlap this step's MFMAs
        fetch(wave, a_cur, b_cur);
        for (int s = wave; s < nsteps; s += kRouterWaves) {
            bf16x8_t a_nxt, b_nxt[NT][3];
            fetch(s + kRouterWaves, a_nxt, b_nxt);
            mfma3(a_cur, b_cur);
            a_cur = a_nxt;
#pragma unroll
            for (int n = 0; n < NT; ++n)
#pragma unroll
                for (int p = 0; p < 3; ++p) b_cur[n][p] = b_nxt[n][p];
        }
    } else {  // wide expert counts: no room for a second fragment set
        for (int s = wave; s < nsteps; s += kRouterWaves) {
            fetch(s, a_cur, b_cur);
            mfma3(a_cur, b_cur);
        }
    }
    const int64_t tile = static_cast<int64_t>(kRouterTokens) * E_pad;
    auto at = [&](int which, int n, int v) -> float& {
        const int row = 8 * (v >> 2) + 4 * half + (v & 3);
        return buf[which * tile + row * E_pad + n * 32 + r];
    };
    for (int h = kRouterWaves / 2; h >= 1; h >>= 1) {
        // writers [h, 2h) hand their partials to readers [0, h), `slots` at a time
        for (int g = 0; g < h; g += slots) {
            if (wave >= h + g && wave < h + g + slots && wave < 2 * h) {
#pragma unroll
                for (int n = 0; n < NT; ++n)
#pragma unroll
                    for (int v = 0; v < 16; ++v) at(wave - h - g, n, v) = acc[n][v];
            }
            __syncthreads();
            if (wave >= g && wave < g + slots && wave < h) {
#pragma unroll
                for (int n = 0; n < NT; ++n)
#pragma unroll
                    for (int v = 0; v < 16; ++v) acc[n][v] += at(wave - g, n, v);
            }
            __syncthreads();
        }
    }
    if (wave == 0) {
#pragma unroll
        for (int n = 0; n < NT; ++n)
#pragma unroll
            for (int v = 0; v < 16; ++v) at(0, n, v) = acc[n][v];
    }
}

template <bool BF16, int NT>
__global__ void __launch_bounds__(kRouterThreads)
router_kernel(const void* __restrict__ x, int64_t T, int d, const float* __restrict__ w_gate,
              const uint16_t* __restrict__ wsplit, const float* __restrict__ bias, int E, int E_pad,
              int k, int renorm, float* __restrict__ logits, float* __restrict__ probs,
              int32_t* __restrict__ topk_idx, float* __restrict__ topk_w) {
    extern __shared__ float smem[];
    // bf16 path: smem = [slots][32][E_pad] tree buffers, the logits end in the first;
    // fp32 path: smem = [32][E_pad] logits.
    float* zrow = smem;
    const int wave = threadIdx.x / kWave;
    const int lane = lane_id();
    const int64_t tok0 = static_cast<int64_t>(blockIdx.x) * kRouterTokens;
    const int ntok = static_cast<int>(T - tok0 < kRouterTokens ? T - tok0 : kRouterTokens);

    if constexpr (BF16) {
        router_mfma_logits<NT>(static_cast<const uint16_t*>(x), T, d, wsplit, E_pad, tok0, wave,
                               router_slots(E_pad), smem);
    } else {
        const float* xf = static_cast<const float*>(x);
        for (int i = threadIdx.x; i < kRouterTokens * E_pad; i += kRouterThreads) {
            const int t = i / E_pad, e = i % E_pad;
            float z = 0.0f;
            if (t < ntok && e < E) {
                const float* xr = xf + (tok0 + t) * d;
                const float* wr = w_gate + static_cast<int64_t>(e) * d;
                double acc = 0.0;
                for (int c = 0; c < d; ++c) acc = fma(static_cast<double>(xr[c]), static_cast<double>(wr[c]), acc);
                z = static_cast<float>(acc);
            }
            zrow[i] = z;
        }
    }
    __syncthreads();

    // softmax + top-k: wave w handles tokens w, w + 8, ...
    const int QE = static_cast<int>(ceil_div(E, kWave));
    for (int t = wave; t < ntok; t += kRouterWaves) {
        const float* zr = zrow + t * E_pad;
        const int64_t tok = tok0 + t;
        float zq[4], gq[4];
        float m = -INFINITY;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = lane + q * kWave;
            zq[q] = -INFINITY;
            if (q < QE && e < E) zq[q] = zr[e] + (bias != nullptr ? bias[e] : 0.0f);
            m = fmaxf(m, zq[q]);
        }
        m = wave_max(m);
        float s = 0.0f;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = lane + q * kWave;
            gq[q] = (q < QE && e < E) ? expf(zq[q] - m) : 0.0f;
            s += gq[q];
        }
        s = wave_sum(s);
        const float inv = 1.0f / s;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = lane + q * kWave;
            gq[q] *= inv;
            if (q < QE && e < E) {
                probs[tok * E + e] = gq[q];
                if (logits != nullptr) logits[tok * E + e] = zq[q];
            }
        }
        // top-k: k rounds of a wave-wide argmax on (logit desc, index asc);
        // lane r keeps the r-th choice.
        unsigned taken = 0;
        int my_i = 0;
        float my_w = 0.0f;
        for (int r = 0; r < k; ++r) {
            float bv = -INFINITY;
            int bi = 0x7fffffff;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int e = lane + q * kWave;
                if (q < QE && e < E && !((taken >> q) & 1u)) {
                    if (bi == 0x7fffffff || zq[q] > bv) {
                        bv = zq[q];
                        bi = e;
                    }
                }
            }
#pragma unroll
            for (int o = 32; o > 0; o >>= 1) {
                const float ov = __shfl_xor(bv, o, kWave);
                const int oi = __shfl_xor(bi, o, kWave);
                const bool better = (oi != 0x7fffffff) &&
                                    (bi == 0x7fffffff || ov > bv || (ov == bv && oi < bi));
                if (better) {
                    bv = ov;
                    bi = oi;
                }
            }
            const int wq = bi / kWave;
            float gv = 0.0f;
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (q == wq) gv = gq[q];
            gv = __shfl(gv, bi % kWave, kWave);
            if ((bi % kWave) == lane) taken |= 1u << wq;
            if (lane == r) {
                my_i = bi;
                my_w = gv;
            }
        }
        if (renorm) {
            const float wsum = wave_sum(lane < k ? my_w : 0.0f);
            my_w = my_w / wsum;
        }
        if (lane < k) {
            topk_idx[tok * k + lane] = my_i;
            topk_w[tok * k + lane] = my_w;
        }
    }
}

template <bool BF16>
hipError_t launch_router_nt(int NT, const void* x, int64_t T, int d, const float* w_gate,
                            const uint16_t* wsplit, const float* bias, int E, int E_pad, int k,
                            int renorm, float* logits, float* probs, int32_t* topk_idx,
                            float* topk_w, hipStream_t stream) {
    const dim3 grid(static_cast<unsigned>(ceil_div(T, kRouterTokens)));
    const size_t lds = sizeof(float) * kRouterTokens * E_pad * (BF16 ? router_slots(E_pad) : 1);
#define SMOES_ROUTER_CASE(N)                                                                      \
    case N:                                                                                       \
        hipLaunchKernelGGL((router_kernel<BF16, N>), grid, dim3(kRouterThreads), lds, stream, x, \
                           T, d, w_gate, wsplit, bias, E, E_pad, k, renorm, logits, probs,       \
                           topk_idx, topk_w);                                                    \
        break;
    switch (NT) {
        SMOES_ROUTER_CASE(1)
        SMOES_ROUTER_CASE(2)
        SMOES_ROUTER_CASE(3)
        SMOES_ROUTER_CASE(4)
        SMOES_ROUTER_CASE(5)
        SMOES_ROUTER_CASE(6)
        SMOES_ROUTER_CASE(7)
        SMOES_ROUTER_CASE(8)
        default:
            return hipErrorInvalidValue;
    }
#undef SMOES_ROUTER_CASE
    return hipGetLastError();
}

}  // namespace

size_t router_workspace_bytes(int d, int E, int x_dtype) {
    if (x_dtype != 1) return 0;
    const int E_pad = static_cast<int>(ceil_div(E, 32) * 32);
    return align_up(sizeof(uint16_t) * 3 * static_cast<size_t>(E_pad) * d, 256);
}

size_t router_lds_bytes(int E, int x_dtype) {
    const int E_pad = static_cast<int>(ceil_div(E, 32) * 32);
    return sizeof(float) * kRouterTokens * E_pad * (x_dtype == 1 ? router_slots(E_pad) : 1);
}

hipError_t launch_route(const void* x, int x_dtype, int64_t T, int d, const float* w_gate,
                        const float* bias, int E, int k, int renorm, float* logits, float* probs,
                        int32_t* topk_idx, float* topk_w, void* ws, hipStream_t stream) {
    const int E_pad = static_cast<int>(ceil_div(E, 32) * 32);
    const int NT = E_pad / 32;
    if (x_dtype == 1) {
        uint16_t* wsplit = static_cast<uint16_t*>(ws);
        const int64_t n = static_cast<int64_t>(E_pad) * d;
        const unsigned blocks = static_cast<unsigned>(ceil_div(n, 256) < 4096 ? ceil_div(n, 256) : 4096);
        hipLaunchKernelGGL(split_wgate_kernel, dim3(blocks), dim3(256), 0, stream, w_gate, E, E_pad,
                           d, wsplit);
        hipError_t err = hipGetLastError();
        if (err != hipSuccess) return err;
        return launch_router_nt<true>(NT, x, T, d, w_gate, wsplit, bias, E, E_pad, k, renorm,
                                      logits, probs, topk_idx, topk_w, stream);
    }
    return launch_router_nt<false>(NT, x, T, d, w_gate, nullptr, bias, E, E_pad, k, renorm, logits,
                                   probs, topk_idx, topk_w, stream);
}

}  // namespace smoes
