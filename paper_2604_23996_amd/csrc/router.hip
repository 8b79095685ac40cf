// Router: logits z = W_gate x (+ b), full softmax g and top-k (Sec. 3.1).
//
// bf16 activations, two kernels:
//   router_logits_kernel: the logits on the matrix cores, fp32-faithful: the
//     fp32 router weights are split into three bf16 terms (hi + mid + lo
//     reproduces each weight to ~2^-24), every product of a term with an exact
//     bf16 activation is exact, and v_mfma_f32_16x16x32_bf16 accumulates in
//     fp32. The split weights are stored in the order the MFMA reads them, so
//     a wave loads a fragment as one contiguous 1 KB. A workgroup owns a tile
//     of 64 or 128 tokens and one of KS ranges of the hidden dimension (KS
//     chosen so that the grid fills the chip); its four waves split the
//     experts, so every weight byte reaches a workgroup once per token tile.
//     Each range's partial logits go to the workspace.
//   router_topk_kernel: one wave per token sums the KS partials in range
//     order, adds the bias, and runs the softmax and the top-k (one lane per
//     expert, DPP reductions).
// fp32 activations: one kernel, dot products accumulated in fp64, then the
// same per-token softmax and top-k.
#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

constexpr int kRouterTokens = 16;  // tokens per fp32-path workgroup
constexpr int kRouterWaves = 8;    // fp32 path
constexpr int kRouterThreads = kRouterWaves * 64;
constexpr int kLogitWaves = 4;     // bf16 logits kernel: waves split the expert tiles
constexpr int kTopkWaves = 4;      // top-k kernel: one wave per token

__host__ __device__ inline int router_epad(int E) { return static_cast<int>(ceil_div(E, 16) * 16); }

// Tiling of the bf16 logits kernel: NTW expert tiles of 16 per wave (4 waves
// cover E_pad), TMT token tiles of 16 per workgroup, KS ranges of the hidden
// dimension of `steps` 32-wide k-steps each (the last may be shorter).
struct RouterPlan {
    int ntw, tmt, ks, steps;
};
RouterPlan router_plan(int64_t T, int d, int E) {
    RouterPlan p;
    const int nt = router_epad(E) / 16;
    p.ntw = static_cast<int>(ceil_div(nt, kLogitWaves));
    p.tmt = (p.ntw == 2 || p.ntw == 3) ? 8 : 4;  // VGPRs: accumulators + the fragment sets
    const int64_t tiles = ceil_div(T, 16 * p.tmt);
    const int nsteps = static_cast<int>(ceil_div(d, 32));
    // about one workgroup per CU, each range at least 8 k-steps long (a sweep
    // of 1, 2, 4, 8 ranges and 32, 64, 128-token tiles at the four bf16
    // workload shapes found this the fastest or within 3 % of it)
    int ks = static_cast<int>(ceil_div(256, tiles > 0 ? tiles : 1));
    const int ks_max = nsteps / 8 > 1 ? nsteps / 8 : 1;
    ks = ks < 1 ? 1 : (ks > ks_max ? ks_max : ks);
    p.steps = static_cast<int>(ceil_div(nsteps, ks));
    p.ks = static_cast<int>(ceil_div(nsteps, p.steps));
    return p;
}

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

// Partial logits of 16 * TMT tokens over k-steps [s0, s1) of the hidden
// dimension (range blockIdx.y), all experts. Wave w owns expert tiles
// w, w + 4, ... (NTW of them) and computes D = W x^T on the matrix cores
// (experts as rows, tokens as columns), so a lane ends with four consecutive
// experts of one token and stores them as one 16-byte vector. Each k-step
// loads the wave's weight fragments (three bf16 terms) and the token
// fragments, the next step's while this step's MFMAs run; the terms are
// accumulated lo, mid, hi. NBUF fragment sets rotate, so the loads of the
// next NBUF - 1 steps are in flight while a step's MFMAs run (two sets
// measured as fast as three, four or six). Loads past the
// hidden dimension, the range or the expert tiles are out of range and
// return zeros (zero products add nothing).
// 16x16x32 operands: lane l holds row (A) / column (B) l % 16 at k = 8 (l / 16) + 0..7;
// result element i of lane l sits at row 4 (l / 16) + i, column l % 16.
template <int TMT, int NTW, int NBUF>
__global__ void __launch_bounds__(kLogitWaves * 64)
router_logits_kernel(const uint16_t* __restrict__ x, int64_t T, int d, const uint16_t* __restrict__ wpk, int E_pad,
                     int steps, float* __restrict__ part) {
    const int lane = lane_id();
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kWave);
    const int quad = lane >> 4, r = lane & 15;
    const int nt = E_pad / 16;
    const int nsteps = static_cast<int>(ceil_div(d, 32));
    const int s0 = static_cast<int>(blockIdx.y) * steps;
    const int s1 = s0 + steps < nsteps ? s0 + steps : nsteps;
    const int64_t tok0 = static_cast<int64_t>(blockIdx.x) * (16 * TMT);
    constexpr int kOob = 0x7fffffff;
    const __amdgpu_buffer_rsrc_t rsx = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(x), 0, static_cast<int>(T * d * 2), 0x00020000);
    const int64_t term = static_cast<int64_t>(nt) * nsteps * 512;  // elements per weight term
    const __amdgpu_buffer_rsrc_t rsw = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(wpk), 0, static_cast<int>(3 * term * 2), 0x00020000);
    int xoff[TMT];
#pragma unroll
    for (int tt = 0; tt < TMT; ++tt) {
        int64_t tok = tok0 + tt * 16 + r;
        if (tok >= T) tok = T - 1;  // computed but never stored
        xoff[tt] = static_cast<int>(tok * d * 2);
    }
    f32x4_t acc[NTW][TMT];
#pragma unroll
    for (int j = 0; j < NTW; ++j)
#pragma unroll
        for (int tt = 0; tt < TMT; ++tt) acc[j][tt] = f32x4_t{};
    auto fetch = [&](int s, bf16x8_t (&a)[TMT], bf16x8_t (&b)[NTW][3]) {
        const int kk = s * 32 + quad * 8;
        // d % 8 == 0: an 8-chunk is all in or all out; chunks past d would read
        // the next token's row (zero weights there, but 0 * inf is NaN)
        const int oob = (s < s1 && kk < d) ? 0 : kOob;
#pragma unroll
        for (int tt = 0; tt < TMT; ++tt)
            a[tt] = __builtin_bit_cast(bf16x8_t,
                                       __builtin_amdgcn_raw_buffer_load_b128(rsx, (xoff[tt] + kk * 2) | oob, 0, 0));
#pragma unroll
        for (int j = 0; j < NTW; ++j) {
            const int n = wave + kLogitWaves * j;
            const int noob = n < nt ? oob : kOob;
            const int off = static_cast<int>(((static_cast<int64_t>(n) * nsteps + s) * 64 + lane) * 16);
#pragma unroll
            for (int p = 0; p < 3; ++p)
                b[j][p] = __builtin_bit_cast(
                    bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(rsw, (static_cast<int>(p * term * 2) + off) | noob,
                                                                     0, 0));
        }
    };
    auto mfma3 = [&](const bf16x8_t (&a)[TMT], const bf16x8_t (&b)[NTW][3]) {
#pragma unroll
        for (int j = 0; j < NTW; ++j)
#pragma unroll
            for (int tt = 0; tt < TMT; ++tt) {
                acc[j][tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(b[j][2], a[tt], acc[j][tt], 0, 0, 0);  // lo
                acc[j][tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(b[j][1], a[tt], acc[j][tt], 0, 0, 0);  // mid
                acc[j][tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(b[j][0], a[tt], acc[j][tt], 0, 0, 0);  // hi
            }
    };
    bf16x8_t a[NBUF][TMT], b[NBUF][NTW][3];
#pragma unroll
    for (int u = 0; u < NBUF - 1; ++u) fetch(s0 + u, a[u], b[u]);
    for (int s = s0; s < s1; s += NBUF) {
#pragma unroll
        for (int u = 0; u < NBUF; ++u) {
            __builtin_amdgcn_sched_barrier(0);
            fetch(s + u + NBUF - 1, a[(u + NBUF - 1) % NBUF], b[(u + NBUF - 1) % NBUF]);
            __builtin_amdgcn_sched_barrier(0);
            mfma3(a[u], b[u]);
        }
    }
    float* out = part + static_cast<int64_t>(blockIdx.y) * T * E_pad;
#pragma unroll
    for (int j = 0; j < NTW; ++j) {
        const int n = wave + kLogitWaves * j;
        if (n >= nt) continue;
#pragma unroll
        for (int tt = 0; tt < TMT; ++tt) {
            const int64_t tok = tok0 + tt * 16 + r;
            if (tok < T)
                *reinterpret_cast<f32x4_t*>(out + tok * E_pad + n * 16 + quad * 4) = acc[j][tt];
        }
    }
}

// Softmax and top-k of one token by one wave: lane l holds experts l + 64 q
// (z[q], -inf past E). Each top-k round takes the wave maximum of the
// untaken logits and then the lowest expert index that holds it (ties to the
// lower index).
template <int Q>
__device__ __forceinline__ void softmax_topk_token(const float (&z)[Q], int64_t tok, int E, int k, int renorm,
                                                   float* __restrict__ logits, float* __restrict__ probs,
                                                   int32_t* __restrict__ topk_idx, float* __restrict__ topk_w) {
    const int lane = lane_id();
    float lm = -INFINITY;
#pragma unroll
    for (int q = 0; q < Q; ++q) lm = fmaxf(lm, z[q]);
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

// One wave per token: z = the KS partial logits summed in range order, plus
// the bias; then softmax and top-k.
template <int Q>
__global__ void __launch_bounds__(kTopkWaves * 64)
router_topk_kernel(const float* __restrict__ part, int ks_n, int64_t T, int E, int E_pad,
                   const float* __restrict__ bias, int k, int renorm, float* __restrict__ logits,
                   float* __restrict__ probs, int32_t* __restrict__ topk_idx, float* __restrict__ topk_w) {
    const int64_t tok = static_cast<int64_t>(blockIdx.x) * kTopkWaves + threadIdx.x / kWave;
    if (tok >= T) return;  // wave-uniform
    const int lane = lane_id();
    float z[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int e = lane + q * kWave;
        if (e < E) {
            float v = part[tok * E_pad + e];
#pragma unroll 4
            for (int ks = 1; ks < ks_n; ++ks) v += part[(static_cast<int64_t>(ks) * T + tok) * E_pad + e];
            z[q] = v + (bias != nullptr ? bias[e] : 0.0f);
        } else {
            z[q] = -INFINITY;
        }
    }
    softmax_topk_token<Q>(z, tok, E, k, renorm, logits, probs, topk_idx, topk_w);
}

// fp32 activations: 16 tokens per workgroup, dot products in fp64 into an
// LDS tile [16][E_pad + 1] (odd pitch), then one wave per token runs the
// softmax and the top-k.
__global__ void __launch_bounds__(kRouterThreads)
router_f32_kernel(const float* __restrict__ x, int64_t T, int d, const float* __restrict__ w_gate,
                  const float* __restrict__ bias, int E, int E_pad, int k, int renorm, float* __restrict__ logits,
                  float* __restrict__ probs, int32_t* __restrict__ topk_idx, float* __restrict__ topk_w) {
    extern __shared__ float smem[];
    const int zp = E_pad + 1;
    const int wave = threadIdx.x / kWave;
    const int64_t tok0 = static_cast<int64_t>(blockIdx.x) * kRouterTokens;
    const int ntok = static_cast<int>(T - tok0 < kRouterTokens ? T - tok0 : kRouterTokens);
    for (int i = threadIdx.x; i < kRouterTokens * E_pad; i += kRouterThreads) {
        const int t = i / E_pad, e = i % E_pad;
        float z = 0.0f;
        if (t < ntok && e < E) {
            const float* xr = x + (tok0 + t) * d;
            const float* wr = w_gate + static_cast<int64_t>(e) * d;
            double acc = 0.0;
            for (int c = 0; c < d; ++c) acc = fma(static_cast<double>(xr[c]), static_cast<double>(wr[c]), acc);
            z = static_cast<float>(acc);
        }
        smem[t * zp + e] = z;
    }
    __syncthreads();
    const int lane = lane_id();
    for (int t = wave; t < ntok; t += kRouterWaves) {
        float z[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = lane + q * kWave;
            z[q] = e < E ? smem[t * zp + e] + (bias != nullptr ? bias[e] : 0.0f) : -INFINITY;
        }
        softmax_topk_token<4>(z, tok0 + t, E, k, renorm, logits, probs, topk_idx, topk_w);
    }
}

// bf16 path: partial logits into part[KS][T][E_pad], then the top-k kernel.
hipError_t launch_router_bf16(const uint16_t* x, int64_t T, int d, const uint16_t* wsplit, const float* bias,
                              int E, int k, int renorm, float* part, float* logits, float* probs,
                              int32_t* topk_idx, float* topk_w, hipStream_t stream) {
    const int E_pad = router_epad(E);
    const RouterPlan p = router_plan(T, d, E);
    const dim3 grid(static_cast<unsigned>(ceil_div(T, 16 * p.tmt)), static_cast<unsigned>(p.ks));
    const dim3 block(kLogitWaves * 64);
    if (p.ntw == 1 && p.tmt == 4)
        hipLaunchKernelGGL((router_logits_kernel<4, 1, 2>), grid, block, 0, stream, x, T, d, wsplit, E_pad, p.steps, part);
    else if (p.ntw == 2 && p.tmt == 8)
        hipLaunchKernelGGL((router_logits_kernel<8, 2, 2>), grid, block, 0, stream, x, T, d, wsplit, E_pad, p.steps, part);
    else if (p.ntw == 3 && p.tmt == 8)
        hipLaunchKernelGGL((router_logits_kernel<8, 3, 2>), grid, block, 0, stream, x, T, d, wsplit, E_pad, p.steps, part);
    else if (p.ntw == 4 && p.tmt == 4)
        hipLaunchKernelGGL((router_logits_kernel<4, 4, 2>), grid, block, 0, stream, x, T, d, wsplit, E_pad, p.steps, part);
    else
        return hipErrorInvalidValue;
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    const dim3 tgrid(static_cast<unsigned>(ceil_div(T, kTopkWaves)));
    const dim3 tblock(kTopkWaves * 64);
    switch ((E + kWave - 1) / kWave) {
        case 1:
            hipLaunchKernelGGL(router_topk_kernel<1>, tgrid, tblock, 0, stream, part, p.ks, T, E, E_pad, bias, k,
                               renorm, logits, probs, topk_idx, topk_w);
            break;
        case 2:
            hipLaunchKernelGGL(router_topk_kernel<2>, tgrid, tblock, 0, stream, part, p.ks, T, E, E_pad, bias, k,
                               renorm, logits, probs, topk_idx, topk_w);
            break;
        case 3:
            hipLaunchKernelGGL(router_topk_kernel<3>, tgrid, tblock, 0, stream, part, p.ks, T, E, E_pad, bias, k,
                               renorm, logits, probs, topk_idx, topk_w);
            break;
        case 4:
            hipLaunchKernelGGL(router_topk_kernel<4>, tgrid, tblock, 0, stream, part, p.ks, T, E, E_pad, bias, k,
                               renorm, logits, probs, topk_idx, topk_w);
            break;
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

// bf16: the split weights (used when the caller passes row-major weights)
// and the partial logits [KS][T][E_pad]; fp32: nothing.
size_t router_workspace_bytes(int64_t T, int d, int E, int x_dtype) {
    if (x_dtype != 1) return 0;
    const int E_pad = router_epad(E);
    const RouterPlan p = router_plan(T, d, E);
    return align_up(sizeof(uint16_t) * 3 * static_cast<size_t>(E_pad) * ceil_div(d, 32) * 32, 256) +
           align_up(sizeof(float) * static_cast<size_t>(p.ks) * T * E_pad, 256);
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
    if (x_dtype == 1) {
        uint8_t* base = static_cast<uint8_t*>(ws);
        const size_t split_bytes = align_up(sizeof(uint16_t) * 3 * static_cast<size_t>(E_pad) * ceil_div(d, 32) * 32, 256);
        float* part = reinterpret_cast<float*>(base + split_bytes);
        const uint16_t* wsplit = static_cast<const uint16_t*>(w_split);
        if (wsplit == nullptr) {
            hipError_t err = launch_split_wgate(w_gate, E, d, base, stream);
            if (err != hipSuccess) return err;
            wsplit = reinterpret_cast<const uint16_t*>(base);
        }
        return launch_router_bf16(static_cast<const uint16_t*>(x), T, d, wsplit, bias, E, k, renorm, part, logits,
                                  probs, topk_idx, topk_w, stream);
    }
    const dim3 grid(static_cast<unsigned>(ceil_div(T, kRouterTokens)));
    const size_t lds = sizeof(float) * kRouterTokens * (E_pad + 1);
    hipLaunchKernelGGL(router_f32_kernel, grid, dim3(kRouterThreads), lds, stream, static_cast<const float*>(x), T,
                       d, w_gate, bias, E, E_pad, k, renorm, logits, probs, topk_idx, topk_w);
    return hipGetLastError();
}

}  // namespace smoes
