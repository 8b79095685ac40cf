// Router: logits z = W_gate x (+ b), full softmax g and top-k (Sec. 3.1).
//
// One workgroup (8 waves) owns 16 * TT tokens (TT = 1) and every expert. For bf16 activations the logits are fp32-faithful on the
// matrix cores: the fp32 router weights are split into three bf16 terms
// (hi + mid + lo reproduces the weight to ~2^-24), each product with the
// exact bf16 activation is exact, and v_mfma_f32_16x16x32_bf16 accumulates in
// fp32. The split weights are stored in the order the MFMA reads them, so a
// wave loads each fragment as one contiguous 1 KB. The eight waves split the
// hidden dimension; their partial tiles are summed in LDS in a fixed order,
// then each wave runs the softmax and the top-k of its tokens (one lane per
// expert, DPP reductions).
// For fp32 activations the dot products are accumulated in fp64.
#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

constexpr int kRouterTokens = 16;  // tokens per MFMA tile
constexpr int kRouterWaves = 8;
constexpr int kRouterThreads = kRouterWaves * 64;
constexpr int kRouterSlots = 4;  // LDS tree buffers of [16 TT][E_pad] floats (<= 64 KB)

__host__ __device__ inline int router_epad(int E) { return static_cast<int>(ceil_div(E, 16) * 16); }
// Token tiles per workgroup. One (16 tokens) is fastest: larger tiles cut the
// weight traffic but leave fewer workgroups to share the per-token softmax
// and top-k, which then dominate.
__host__ __device__ constexpr int router_tt(int /*NT*/) { return 1; }

// w_gate [E, d] f32 -> three bf16 parts (hi, mid, lo) in MFMA fragment order:
// wpk[p][n][s][l][e] = part p of W[16 n + l % 16][32 s + 8 (l / 16) + e], zero
// outside W (n < E_pad / 16 expert tiles, s < ceil(d / 32) k-steps). One
// thread per 8-element fragment row.
__global__ void split_wgate_kernel(const float* __restrict__ w, int E, int E_pad, int d,
                                   uint16_t* __restrict__ wpk) {
    const int nsteps = static_cast<int>(ceil_div(d, 32));
    const int64_t frags = static_cast<int64_t>(E_pad / 16) * nsteps * 64;
    const int64_t part = frags * 8;
    for (int64_t f = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; f < frags;
         f += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int l = static_cast<int>(f % 64);
        const int st = static_cast<int>((f / 64) % nsteps);
        const int n = static_cast<int>(f / (64 * nsteps));
        const int e = n * 16 + (l % 16);
        const int k0 = st * 32 + 8 * (l / 16);
        uint16_t hi[8], mid[8], lo[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const float v = (e < E && k0 + q < d) ? w[static_cast<int64_t>(e) * d + k0 + q] : 0.0f;
            hi[q] = f32_to_bf16(v);
            const float r1 = v - bf16_to_f32(hi[q]);
            mid[q] = f32_to_bf16(r1);
            lo[q] = f32_to_bf16(r1 - bf16_to_f32(mid[q]));
        }
        auto pack = [](const uint16_t (&h)[8]) {
            return make_uint4(h[0] | (static_cast<uint32_t>(h[1]) << 16), h[2] | (static_cast<uint32_t>(h[3]) << 16),
                              h[4] | (static_cast<uint32_t>(h[5]) << 16), h[6] | (static_cast<uint32_t>(h[7]) << 16));
        };
        *reinterpret_cast<uint4*>(wpk + f * 8) = pack(hi);
        *reinterpret_cast<uint4*>(wpk + part + f * 8) = pack(mid);
        *reinterpret_cast<uint4*>(wpk + 2 * part + f * 8) = pack(lo);
    }
}

// Logits of one wave over its share of the hidden dimension (k-steps of 32,
// s = wave, wave + 8, ...), bf16x3 MFMA over TT token tiles and NT expert
// tiles; for small tiles the next step's fragments are loaded before the
// current step's MFMAs. Then a fixed-order tree over the 8 waves through LDS
// (wave w adds wave w + h, h = 4, 2, 1). The logits end at the start of the
// buffer as [16 TT][E_pad + 1] (odd pitch: one lane per token reads them
// without bank conflicts).
// 16x16x32 operands: lane l holds row (A) / column (B) l % 16 at k = 8 (l / 16) + 0..7;
// result element i of lane l sits at row 4 (l / 16) + i, column l % 16.
template <int TT, int NT>
__device__ __forceinline__ void router_mfma_logits(const uint16_t* __restrict__ x, int64_t T, int d,
                                   const uint16_t* __restrict__ wpk, int E_pad,
                                   int64_t tok0, int wave, float* __restrict__ buf) {
    const int lane = lane_id();
    const int quad = lane >> 4;
    const int r = lane & 15;
    // Buffer loads: an offset past the record count returns zeros, so the
    // k tail and the steps past the end need no selects on loaded values.
    constexpr int kOob = 0x7fffffff;
    const __amdgpu_buffer_rsrc_t rsx = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(x), 0, static_cast<int>(T * d * 2), 0x00020000);
    const int nsteps = static_cast<int>(ceil_div(d, 32));
    const int64_t part = static_cast<int64_t>(E_pad / 16) * nsteps * 512;
    const __amdgpu_buffer_rsrc_t rsw = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(wpk), 0, static_cast<int>(3 * part * 2), 0x00020000);
    int xoff[TT];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
        int64_t tok = tok0 + tt * 16 + r;
        if (tok >= T) tok = T - 1;
        xoff[tt] = static_cast<int>(tok * d * 2);
    }
    f32x4_t acc[TT][NT];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
#pragma unroll
        for (int n = 0; n < NT; ++n) acc[tt][n] = f32x4_t{};
    typedef int i32x4 __attribute__((ext_vector_type(4)));
    auto fetch = [&](int s, bf16x8_t (&a)[TT], bf16x8_t (&b)[NT][3]) {
        const int kk = s * 32 + quad * 8;
        const int oob = (s < nsteps && kk < d) ? 0 : kOob;  // d % 8 == 0: an 8-chunk is all in or all out
#pragma unroll
        for (int tt = 0; tt < TT; ++tt)
            a[tt] = __builtin_bit_cast(bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(rsx, (xoff[tt] + kk * 2) | oob, 0, 0));
        const int soob = s < nsteps ? 0 : kOob;
#pragma unroll
        for (int n = 0; n < NT; ++n) {
            const int off = static_cast<int>(((static_cast<int64_t>(n) * nsteps + s) * 64 + lane) * 16);
#pragma unroll
            for (int p = 0; p < 3; ++p)
                b[n][p] = __builtin_bit_cast(
                    bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(rsw, (static_cast<int>(p * part * 2) + off) | soob, 0, 0));
        }
    };
    auto mfma3 = [&](const bf16x8_t (&a)[TT], const bf16x8_t (&b)[NT][3]) {
#pragma unroll
        for (int n = 0; n < NT; ++n)
#pragma unroll
            for (int tt = 0; tt < TT; ++tt) {
                acc[tt][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[tt], b[n][2], acc[tt][n], 0, 0, 0);  // lo
                acc[tt][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[tt], b[n][1], acc[tt][n], 0, 0, 0);  // mid
                acc[tt][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[tt], b[n][0], acc[tt][n], 0, 0, 0);  // hi
            }
    };
    if constexpr (TT * 4 + NT * 12 <= 72) {
        // two named fragment sets: the loads of one step fly while the other's MFMAs run
        bf16x8_t a0[TT], b0[NT][3], a1[TT], b1[NT][3];
        fetch(wave, a0, b0);
        for (int s = wave; s < nsteps; s += 2 * kRouterWaves) {
            __builtin_amdgcn_sched_barrier(0);
            fetch(s + kRouterWaves, a1, b1);
            __builtin_amdgcn_sched_barrier(0);
            mfma3(a0, b0);
            __builtin_amdgcn_sched_barrier(0);
            fetch(s + 2 * kRouterWaves, a0, b0);
            __builtin_amdgcn_sched_barrier(0);
            mfma3(a1, b1);
        }
    } else {  // wide expert counts: no room for a second fragment set
        bf16x8_t a0[TT], b0[NT][3];
        for (int s = wave; s < nsteps; s += kRouterWaves) {
            fetch(s, a0, b0);
            mfma3(a0, b0);
        }
    }
    const int64_t tile = static_cast<int64_t>(kRouterTokens) * TT * E_pad;
    auto at = [&](int which, int tt, int n, int i) -> float& {
        return buf[which * tile + (tt * 16 + quad * 4 + i) * E_pad + n * 16 + r];
    };
    for (int h = kRouterWaves / 2; h >= 1; h >>= 1) {
        // writers [h, 2h) hand their partials to readers [0, h)
        if (wave >= h && wave < 2 * h) {
#pragma unroll
            for (int tt = 0; tt < TT; ++tt)
#pragma unroll
                for (int n = 0; n < NT; ++n)
#pragma unroll
                    for (int i = 0; i < 4; ++i) at(wave - h, tt, n, i) = acc[tt][n][i];
        }
        __syncthreads();
        if (wave < h) {
#pragma unroll
            for (int tt = 0; tt < TT; ++tt)
#pragma unroll
                for (int n = 0; n < NT; ++n)
#pragma unroll
                    for (int i = 0; i < 4; ++i) acc[tt][n][i] += at(wave, tt, n, i);
        }
        __syncthreads();
    }
    if (wave == 0) {  // final tile with an odd row pitch (the other tree slots are free by now)
        const int zp = E_pad + 1;
#pragma unroll
        for (int tt = 0; tt < TT; ++tt)
#pragma unroll
            for (int n = 0; n < NT; ++n)
#pragma unroll
                for (int i = 0; i < 4; ++i) buf[(tt * 16 + quad * 4 + i) * zp + n * 16 + r] = acc[tt][n][i];
    }
}

template <bool BF16, int NT, int TT>
__global__ void __launch_bounds__(kRouterThreads)
router_kernel(const void* __restrict__ x, int64_t T, int d, const float* __restrict__ w_gate,
              const uint16_t* __restrict__ wsplit, const float* __restrict__ bias, int E, int E_pad,
              int k, int renorm, float* __restrict__ logits, float* __restrict__ probs,
              int32_t* __restrict__ topk_idx, float* __restrict__ topk_w) {
    extern __shared__ float smem[];
    // bf16 path: smem = [4][16 TT][E_pad] tree buffers; fp32 path: the logits only.
    // Either way the logits end as [16 TT][E_pad + 1] at the start of smem.
    constexpr int WG_TOKENS = kRouterTokens * TT;
    const int zp = E_pad + 1;
    float* zrow = smem;
    const int wave = threadIdx.x / kWave;
    const int64_t tok0 = static_cast<int64_t>(blockIdx.x) * WG_TOKENS;
    const int ntok = static_cast<int>(T - tok0 < WG_TOKENS ? T - tok0 : WG_TOKENS);

    if constexpr (BF16) {
        router_mfma_logits<TT, NT>(static_cast<const uint16_t*>(x), T, d, wsplit, E_pad, tok0, wave, smem);
    } else {
        const float* xf = static_cast<const float*>(x);
        for (int i = threadIdx.x; i < WG_TOKENS * E_pad; i += kRouterThreads) {
            const int t = i / E_pad, e = i % E_pad;
            float z = 0.0f;
            if (t < ntok && e < E) {
                const float* xr = xf + (tok0 + t) * d;
                const float* wr = w_gate + static_cast<int64_t>(e) * d;
                double acc = 0.0;
                for (int c = 0; c < d; ++c) acc = fma(static_cast<double>(xr[c]), static_cast<double>(wr[c]), acc);
                z = static_cast<float>(acc);
            }
            zrow[t * zp + e] = z;
        }
    }
    __syncthreads();

    // Softmax and top-k: one wave per token, lane l holds experts l + 64 q.
    // Each top-k round takes the wave maximum of the untaken logits and then
    // the lowest expert index that holds it (ties to the lower index).
    constexpr int Q = BF16 ? (16 * NT + 63) / 64 : 4;
    const int lane = lane_id();
    for (int t = wave; t < ntok; t += kRouterWaves) {
        const float* zr = zrow + t * zp;
        const int64_t tok = tok0 + t;
        float z[Q];
        float lm = -INFINITY;
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            const int e = lane + q * kWave;
            z[q] = e < E ? zr[e] + (bias != nullptr ? bias[e] : 0.0f) : -INFINITY;
            lm = fmaxf(lm, z[q]);
        }
        const float m = wave_max_u(lm);
        float ls = 0.0f, g[Q];
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            const int e = lane + q * kWave;
            g[q] = e < E ? expf(z[q] - m) : 0.0f;
            ls += g[q];
        }
        const float inv = 1.0f / wave_sum_u(ls);
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            const int e = lane + q * kWave;
            if (e < E) {
                probs[tok * E + e] = g[q] * inv;
                if (logits != nullptr) logits[tok * E + e] = z[q];
            }
        }
        unsigned taken = 0;
        int my_i = 0;
        float my_w = 0.0f;
        for (int rr = 0; rr < k; ++rr) {
            float bv = -INFINITY;
            int bi = 0x7fffffff;
#pragma unroll
            for (int q = 0; q < Q; ++q) {
                const int e = lane + q * kWave;
                if (e < E && !((taken >> q) & 1u) && (bi == 0x7fffffff || z[q] > bv)) {
                    bv = z[q];
                    bi = e;
                }
            }
            const float gm = wave_max_u(bi == 0x7fffffff ? -INFINITY : bv);
            const int gi = wave_min_u(bi != 0x7fffffff && bv == gm ? bi : 0x7fffffff);
            if ((gi % kWave) == lane) taken |= 1u << (gi / kWave);
            if (lane == rr) {
                my_i = gi;
                my_w = expf(gm - m) * inv;  // the chosen expert's gate value, as in probs
            }
        }
        if (renorm) my_w = my_w / wave_sum_u(lane < k ? my_w : 0.0f);
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
    const int TT = BF16 ? router_tt(NT) : 1;
    const dim3 grid(static_cast<unsigned>(ceil_div(T, kRouterTokens * TT)));
    const size_t lds = router_lds_bytes(E, BF16 ? 1 : 0);
#define SMOES_ROUTER_CASE(N)                                                                        \
    case N:                                                                                         \
        hipLaunchKernelGGL((router_kernel<BF16, N, BF16 ? router_tt(N) : 1>), grid, dim3(kRouterThreads), \
                           lds, stream, x, T, d, w_gate, wsplit, bias, E, E_pad, k, renorm, logits, probs, \
                           topk_idx, topk_w);                                                     \
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
    return align_up(sizeof(uint16_t) * 3 * static_cast<size_t>(E_pad) * ceil_div(d, 32) * 32, 256);
}

size_t router_lds_bytes(int E, int x_dtype) {
    const int E_pad = router_epad(E);
    const int TT = x_dtype == 1 ? router_tt(E_pad / 16) : 1;
    const size_t tokens = static_cast<size_t>(kRouterTokens) * TT;
    const size_t tree = x_dtype == 1 ? tokens * E_pad * kRouterSlots : 0;
    const size_t fin = tokens * (E_pad + 1);  // logits with an odd row pitch
    return sizeof(float) * (tree > fin ? tree : fin);
}

size_t router_packed_elems(int d, int E) {
    return 3 * static_cast<size_t>(router_epad(E)) * ceil_div(d, 32) * 32;
}

hipError_t launch_split_wgate(const float* w_gate, int E, int d, void* wpk, hipStream_t stream) {
    const int E_pad = router_epad(E);
    const int64_t n = static_cast<int64_t>(E_pad / 16) * ceil_div(d, 32) * 64;  // fragments
    const unsigned blocks = static_cast<unsigned>(ceil_div(n, 256) < 4096 ? ceil_div(n, 256) : 4096);
    hipLaunchKernelGGL(split_wgate_kernel, dim3(blocks), dim3(256), 0, stream, w_gate, E, E_pad, d,
                       static_cast<uint16_t*>(wpk));
    return hipGetLastError();
}

hipError_t launch_route(const void* x, int x_dtype, int64_t T, int d, const float* w_gate,
                        const void* w_split, const float* bias, int E, int k, int renorm, float* logits,
                        float* probs, int32_t* topk_idx, float* topk_w, void* ws, hipStream_t stream) {
    const int E_pad = router_epad(E);
    const int NT = E_pad / 16;
    if (x_dtype == 1 && w_split != nullptr)
        return launch_router_nt<true>(NT, x, T, d, w_gate, static_cast<const uint16_t*>(w_split), bias, E,
                                      E_pad, k, renorm, logits, probs, topk_idx, topk_w, stream);
    if (x_dtype == 1) {
        uint16_t* wsplit = static_cast<uint16_t*>(ws);
        const int64_t n = static_cast<int64_t>(E_pad / 16) * ceil_div(d, 32) * 64;  // fragments
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
