// Router: logits z = W_gate x (+ b), full softmax g and top-k (Sec. 3.1).
//
// One workgroup (8 waves) owns 16 tokens and every expert, so a 4096-token
// batch already spreads over 256 workgroups. For bf16 activations the logits
// are fp32-faithful on the matrix cores: the fp32 router weights are split
// into three bf16 terms (hi + mid + lo reproduces the weight to ~2^-24), each
// product with the exact bf16 activation is exact, and
// v_mfma_f32_16x16x32_bf16 accumulates in fp32. The eight waves split the
// hidden dimension; their partial tiles are summed in LDS in a fixed order,
// then every wave runs the softmax and a wave-wide top-k for 2 tokens.
// For fp32 activations the dot products are accumulated in fp64.
#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

constexpr int kRouterTokens = 16;
constexpr int kRouterWaves = 8;
constexpr int kRouterThreads = kRouterWaves * 64;
constexpr int kRouterSlots = 4;  // LDS tree buffers of [16][E_pad] floats (<= 64 KB)

__host__ __device__ inline int router_epad(int E) { return static_cast<int>(ceil_div(E, 16) * 16); }

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

// Logits of one wave over its share of the hidden dimension (k-steps of 32,
// s = wave, wave + 8, ...), bf16x3 MFMA; for up to 6 expert tiles the next
// step's fragments are loaded before the current step's MFMAs. Then a
// fixed-order tree over the 8 waves through LDS (wave w adds wave w + h,
// h = 4, 2, 1). The logits end in buffer 0.
// 16x16x32 operands: lane l holds row (A) / column (B) l % 16 at k = 8 (l / 16) + 0..7;
// result element i of lane l sits at row 4 (l / 16) + i, column l % 16.
template <int NT>
__device__ void router_mfma_logits(const uint16_t* __restrict__ x, int64_t T, int d,
                                   const uint16_t* __restrict__ wsplit, int E_pad,
                                   int64_t tok0, int wave, float* __restrict__ buf) {
    const int lane = lane_id();
    const int quad = lane >> 4;
    const int r = lane & 15;
    int64_t tok = tok0 + r;
    if (tok >= T) tok = T - 1;
    const uint16_t* xrow = x + tok * d;
    const int64_t part = static_cast<int64_t>(E_pad) * d;
    f32x4_t acc[NT];
#pragma unroll
    for (int n = 0; n < NT; ++n) acc[n] = f32x4_t{};
    const int nsteps = static_cast<int>(ceil_div(d, 32));
    auto fetch = [&](int s, bf16x8_t& a, bf16x8_t (&b)[NT][3]) {
        const int kk = s * 32 + quad * 8;
        const bool valid = s < nsteps && kk < d;  // d % 8 == 0: an 8-chunk is all in or all out
        const int kc = valid ? kk : 0;
        a = *reinterpret_cast<const bf16x8_t*>(xrow + kc);
        if (!valid) a = bf16x8_t{};
#pragma unroll
        for (int n = 0; n < NT; ++n) {
            const int64_t off = static_cast<int64_t>(n * 16 + r) * d + kc;
#pragma unroll
            for (int p = 0; p < 3; ++p) {
                b[n][p] = *reinterpret_cast<const bf16x8_t*>(wsplit + p * part + off);
                if (!valid) b[n][p] = bf16x8_t{};
            }
        }
    };
    auto mfma3 = [&](const bf16x8_t& a, const bf16x8_t (&b)[NT][3]) {
#pragma unroll
        for (int n = 0; n < NT; ++n) {
            acc[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b[n][2], acc[n], 0, 0, 0);  // lo
            acc[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b[n][1], acc[n], 0, 0, 0);  // mid
            acc[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b[n][0], acc[n], 0, 0, 0);  // hi
        }
    };
    bf16x8_t a_cur, b_cur[NT][3];
    if constexpr (NT <= 6) {  // register double buffer
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
    auto at = [&](int which, int n, int i) -> float& {
        return buf[which * tile + (quad * 4 + i) * E_pad + n * 16 + r];
    };
    for (int h = kRouterWaves / 2; h >= 1; h >>= 1) {
        // writers [h, 2h) hand their partials to readers [0, h)
        if (wave >= h && wave < 2 * h) {
#pragma unroll
            for (int n = 0; n < NT; ++n)
#pragma unroll
                for (int i = 0; i < 4; ++i) at(wave - h, n, i) = acc[n][i];
        }
        __syncthreads();
        if (wave < h) {
#pragma unroll
            for (int n = 0; n < NT; ++n)
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[n][i] += at(wave, n, i);
        }
        __syncthreads();
    }
    if (wave == 0) {
#pragma unroll
        for (int n = 0; n < NT; ++n)
#pragma unroll
            for (int i = 0; i < 4; ++i) at(0, n, i) = acc[n][i];
    }
}

template <bool BF16, int NT>
__global__ void __launch_bounds__(kRouterThreads)
router_kernel(const void* __restrict__ x, int64_t T, int d, const float* __restrict__ w_gate,
              const uint16_t* __restrict__ wsplit, const float* __restrict__ bias, int E, int E_pad,
              int k, int renorm, float* __restrict__ logits, float* __restrict__ probs,
              int32_t* __restrict__ topk_idx, float* __restrict__ topk_w) {
    extern __shared__ float smem[];
    // bf16 path: smem = [4][16][E_pad] tree buffers, the logits end in the first;
    // fp32 path: smem = [16][E_pad] logits.
    float* zrow = smem;
    const int wave = threadIdx.x / kWave;
    const int lane = lane_id();
    const int64_t tok0 = static_cast<int64_t>(blockIdx.x) * kRouterTokens;
    const int ntok = static_cast<int>(T - tok0 < kRouterTokens ? T - tok0 : kRouterTokens);

    if constexpr (BF16) {
        router_mfma_logits<NT>(static_cast<const uint16_t*>(x), T, d, wsplit, E_pad, tok0, wave, smem);
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

    // softmax + top-k: wave w handles tokens w and w + 8
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
    const size_t lds = sizeof(float) * kRouterTokens * E_pad * (BF16 ? kRouterSlots : 1);
#define SMOES_ROUTER_CASE(N)                                                                      \
    case N:                                                                                       \
        hipLaunchKernelGGL((router_kernel<BF16, N>), grid, dim3(kRouterThreads), lds, stream, x, \
                           T, d, w_gate, wsplit, bias, E, E_pad, k, renorm, logits, probs,       \
                           topk_idx, topk_w);                                                    \
        break;
    if constexpr (BF16) {
        switch (NT) {
            SMOES_ROUTER_CASE(1)
            SMOES_ROUTER_CASE(2)
            SMOES_ROUTER_CASE(3)
            SMOES_ROUTER_CASE(4)
            SMOES_ROUTER_CASE(5)
            SMOES_ROUTER_CASE(6)
            SMOES_ROUTER_CASE(7)
            SMOES_ROUTER_CASE(8)
            SMOES_ROUTER_CASE(9)
            SMOES_ROUTER_CASE(10)
            SMOES_ROUTER_CASE(11)
            SMOES_ROUTER_CASE(12)
            SMOES_ROUTER_CASE(13)
            SMOES_ROUTER_CASE(14)
            SMOES_ROUTER_CASE(15)
            SMOES_ROUTER_CASE(16)
            default:
                return hipErrorInvalidValue;
        }
    } else {
        switch (1) { SMOES_ROUTER_CASE(1) }
    }
#undef SMOES_ROUTER_CASE
    return hipGetLastError();
}

}  // namespace

size_t router_workspace_bytes(int d, int E, int x_dtype) {
    if (x_dtype != 1) return 0;
    const int E_pad = router_epad(E);
    return align_up(sizeof(uint16_t) * 3 * static_cast<size_t>(E_pad) * d, 256);
}

size_t router_lds_bytes(int E, int x_dtype) {
    return sizeof(float) * kRouterTokens * router_epad(E) * (x_dtype == 1 ? kRouterSlots : 1);
}

hipError_t launch_route(const void* x, int x_dtype, int64_t T, int d, const float* w_gate,
                        const float* bias, int E, int k, int renorm, float* logits, float* probs,
                        int32_t* topk_idx, float* topk_w, void* ws, hipStream_t stream) {
    const int E_pad = router_epad(E);
    const int NT = E_pad / 16;
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
