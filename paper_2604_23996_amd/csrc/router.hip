// Router: logits z = W_gate x (+ b), full softmax g and top-k (Sec. 3.1).
//
// bf16 activations, two kernels:
//   router_logits_kernel: the logits on the matrix cores, fp32-faithful: the
//     fp32 router weights are split into three bf16 terms (hi + mid + lo
//     reproduces each weight to ~2^-24), every product of a term with an exact
//     bf16 activation is exact, and v_mfma_f32_16x16x32_bf16 accumulates in
//     fp32 (per 32-wide k-step the terms lo, mid, hi). The split weights are
//     stored in the order the MFMA reads them (one contiguous 1 KB per
//     fragment). A workgroup owns 128 tokens and one of KS ranges of the
//     hidden dimension (KS chosen so that the grid fills the chip). Per
//     k-step every weight fragment (three terms of every 16-expert tile) and
//     every token fragment goes HBM -> LDS once, by buffer-to-LDS loads
//     through a ring of 2-4 slots, and its four waves split the work two by
//     two: expert half x token half, so each fragment read from LDS feeds four
//     (weights) or 3 x NE (tokens) MFMAs. Each range's partial logits go to the
//     workspace.
//   router_topk_row_kernel: 16 lanes per token (four tokens per wave) sum
//     the KS partials in range order, add the bias, and run the softmax and
//     the top-k (lane j holds experts j + 16 q; DPP reductions inside the
//     16-lane row).
// fp32 activations: one kernel, dot products accumulated in fp64, then the
// same per-token softmax and top-k.
#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

constexpr int kRouterTokens = 16;  // tokens per fp32-path workgroup
constexpr int kRouterWaves = 8;    // fp32 path
constexpr int kRouterThreads = kRouterWaves * 64;
constexpr int kLogitWaves = 4;     // bf16 logits kernel: expert half x token half
constexpr int kLogitTT = 4;        // 16-token tiles per wave: 128 tokens per workgroup
constexpr int kLogitTokens = 2 * kLogitTT * 16;
constexpr int kTopkWaves = 4;      // top-k kernel: one wave per token

__host__ __device__ inline int router_epad(int E) { return static_cast<int>(ceil_div(E, 16) * 16); }

// Expert tiles of 16 per wave (half of the E_pad / 16 tiles, rounded up).
__host__ __device__ inline int router_ne(int E) { return static_cast<int>(ceil_div(router_epad(E) / 16, 2)); }

// LDS per ring slot: three weight terms of 2 NE expert tiles and 2 TT token
// tiles, 1 KB each; the ring has as many slots (at most four) as fit in 160 KB.
__host__ __device__ constexpr int router_slot_bytes(int ne) { return (6 * ne + 2 * kLogitTT) * 1024; }
__host__ __device__ constexpr int router_ring(int ne) {
    return 4 * router_slot_bytes(ne) <= 160 * 1024 ? 4 : (3 * router_slot_bytes(ne) <= 160 * 1024 ? 3 : 2);
}

// KS ranges of the hidden dimension of `steps` 32-wide k-steps each (the last
// may be shorter): about one workgroup per CU, each range at least 8 k-steps.
struct RouterPlan {
    int ks, steps;
};
RouterPlan router_plan(int64_t T, int d, int /*E*/) {
    RouterPlan p;
    const int64_t tiles = ceil_div(T, kLogitTokens);
    const int nsteps = static_cast<int>(ceil_div(d, 32));
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

// Partial logits of 128 tokens over k-steps [s0, s1) of the hidden dimension
// (range blockIdx.y), all experts. Wave w takes expert tiles (w % 2) NE ..
// + NE - 1 and token tiles (w / 2) TT .. + TT - 1 and computes D = W x^T on
// the matrix cores (experts as rows, tokens as columns), so a lane ends with
// four consecutive experts of one token and stores them as one 16-byte
// vector. Ring slot layout: weight fragment (term p, tile n) at
// (p * 2 NE + n) KB, token tile t at (6 NE + t) KB; the weight fragments of a
// k-step are dealt to the waves round-robin, the token tiles two per wave.
// Fragments are read from LDS one k-step ahead: while k-step t's MFMAs run on
// registers, k-step t + 1's fragments come in. Before that, a wait for
// k-step t + 1's DMAs and a barrier show every wave's part of it landed and
// every wave done reading slot t % ST, which then takes k-step t + ST. Loads
// past the hidden dimension, the range, the tokens or the expert tiles are
// out of range and fill zeros (zero products add nothing; chunks past d are
// never read from the next token's row, where 0 * inf would be NaN).
// 16x16x32 operands: lane l holds row (A) / column (B) l % 16 at k = 8 (l / 16) + 0..7;
// result element i of lane l sits at row 4 (l / 16) + i, column l % 16.
template <int NE>
__global__ void __launch_bounds__(kLogitWaves * 64)
router_logits_kernel(const uint16_t* __restrict__ x, int64_t T, int d, const uint16_t* __restrict__ wpk, int E_pad,
                     int steps, float* __restrict__ part) {
    constexpr int TT = kLogitTT, ST = router_ring(NE), SLOT = router_slot_bytes(NE);
    constexpr int NW = 6 * NE;                            // weight fragments per k-step
    constexpr int QW = (NW + kLogitWaves - 1) / kLogitWaves;  // weight DMAs of waves 0 .. NW % 4 - 1
    constexpr int DMIN = NW / kLogitWaves + 2;            // DMAs every wave issues per k-step (at least)
    constexpr int NF = TT + 3 * NE;                       // fragments a wave reads per k-step
    static_assert(2 * TT == 2 * kLogitWaves, "two token tiles per wave");
    static_assert(3 * DMIN < 64, "vmcnt range");
    __shared__ __attribute__((aligned(1024))) uint8_t lds[ST * SLOT];
    const int lane = lane_id();
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kWave);
    const int eh = wave & 1, th = wave >> 1;
    const int quad = lane >> 4, r = lane & 15;
    const int nt = E_pad / 16;
    const int nsteps = static_cast<int>(ceil_div(d, 32));
    const int s0 = static_cast<int>(blockIdx.y) * steps;
    const int s1 = s0 + steps < nsteps ? s0 + steps : nsteps;
    const int nk = s1 - s0;
    const int64_t tok0 = static_cast<int64_t>(blockIdx.x) * kLogitTokens;
    const i32x4_t rsx = buf_rsrc(x, static_cast<int>(T * d * 2));
    const i32x4_t rsw = buf_rsrc(wpk, static_cast<int>(3 * static_cast<int64_t>(nt) * nsteps * 1024));
    const uint32_t lds0 = lds_address(lds);
    // Byte offsets at k-step 0 (weight fragments: + 1 KB per k-step; token
    // chunks: + 64 B) and LDS offsets of this wave's DMAs; -1: out of range.
    int wvo[QW], xvo[2];
    const bool last_w = wave + kLogitWaves * (QW - 1) < NW;  // this wave issues QW weight DMAs (else QW - 1)
#pragma unroll
    for (int q = 0; q < QW; ++q) {
        const int i = wave + kLogitWaves * q;
        const int pt = i / (2 * NE), n = i % (2 * NE);
        wvo[q] = (i < NW && n < nt) ? ((pt * nt + n) * nsteps + s0) * 1024 + lane * 16 : -1;
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int64_t tok = tok0 + (wave + kLogitWaves * q) * 16 + r;
        xvo[q] = tok < T ? static_cast<int>((tok * d + s0 * 32 + quad * 8) * 2) : -1;
    }
    const int kq = s0 * 32 + quad * 8;  // this lane's k at k-step 0 of the range
    auto issue = [&](int t) {
        const uint32_t slot = lds0 + static_cast<uint32_t>((t % ST) * SLOT);
#pragma unroll
        for (int q = 0; q < QW; ++q) {
            if (q == QW - 1 && !last_w) break;  // wave-uniform
            const int vo = wvo[q] >= 0 ? wvo[q] + t * 1024 : kOutOfRange;
            dma16(rsw, vo, slot + static_cast<uint32_t>(wave + kLogitWaves * q) * 1024u);
        }
        const bool kin = kq + t * 32 < d;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int vo = (xvo[q] >= 0 && kin) ? xvo[q] + t * 64 : kOutOfRange;
            dma16(rsx, vo, slot + static_cast<uint32_t>(NW + wave + kLogitWaves * q) * 1024u);
        }
    };
    // wait until at most `later` k-steps of this wave's DMAs issued after the awaited one fly
    auto wait_later = [&](int later) {
        if (later <= 0) wait_vm_lgkm0<0>();
        else if (later == 1) wait_vm_lgkm0<DMIN>();
        else if (later == 2) wait_vm_lgkm0<2 * DMIN>();
        else wait_vm_lgkm0<3 * DMIN>();
    };
    auto read_frags = [&](int t, bf16x8_t (&f)[NF]) {
        const uint8_t* base = lds + (t % ST) * SLOT + lane * 16;
#pragma unroll
        for (int i = 0; i < TT; ++i) f[i] = *reinterpret_cast<const bf16x8_t*>(base + (NW + th * TT + i) * 1024);
#pragma unroll
        for (int j = 0; j < NE; ++j)
#pragma unroll
            for (int pt = 0; pt < 3; ++pt)
                f[TT + 3 * j + pt] = *reinterpret_cast<const bf16x8_t*>(base + (pt * 2 * NE + eh * NE + j) * 1024);
    };
    auto lgkm_wait0 = [] { __builtin_amdgcn_s_waitcnt(0xc07f); };  // lgkmcnt(0), vmcnt and expcnt free
    f32x4_t acc[NE][TT];
#pragma unroll
    for (int j = 0; j < NE; ++j)
#pragma unroll
        for (int i = 0; i < TT; ++i) acc[j][i] = f32x4_t{};
    auto mma = [&](const bf16x8_t (&f)[NF]) {
#pragma unroll
        for (int j = 0; j < NE; ++j)
#pragma unroll
            for (int i = 0; i < TT; ++i) {
                acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f[TT + 3 * j + 2], f[i], acc[j][i], 0, 0, 0);  // lo
                acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f[TT + 3 * j + 1], f[i], acc[j][i], 0, 0, 0);  // mid
                acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f[TT + 3 * j + 0], f[i], acc[j][i], 0, 0, 0);  // hi
            }
    };
    // k-step t (t + 1 < nk) from registers `cur`; k-step t + 1's fragments into
    // `nxt`. The wait also completes `cur`'s reads (issued one step earlier),
    // so the MFMAs need no wait on the reads issued here.
    auto step = [&](int t, const bf16x8_t (&cur)[NF], bf16x8_t (&nxt)[NF]) {
        const int rest = nk - 2 - t;
        wait_later(rest < ST - 2 ? rest : ST - 2);
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");  // no LDS read moves above the barrier
        if (t + ST < nk) issue(t + ST);
        __builtin_amdgcn_sched_barrier(0);
        read_frags(t + 1, nxt);
        mma(cur);
        // one LDS read after every three MFMAs, the rest of the MFMAs after them
#pragma unroll
        for (int q = 0; q < NF; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x008, 3, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    };
    const int pro = nk < ST ? nk : ST;
    for (int t = 0; t < pro; ++t) issue(t);
    wait_later(pro - 1);
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    bf16x8_t fa[NF], fb[NF];
    read_frags(0, fa);
    int t = 0;
    for (; t + 2 < nk; t += 2) {
        step(t, fa, fb);
        step(t + 1, fb, fa);
    }
    if (t + 1 < nk) {  // two k-steps left
        step(t, fa, fb);
        lgkm_wait0();
        mma(fb);
    } else {
        lgkm_wait0();
        mma(fa);
    }
    float* out = part + static_cast<int64_t>(blockIdx.y) * T * E_pad;
#pragma unroll
    for (int j = 0; j < NE; ++j) {
        const int n = eh * NE + j;
        if (n >= nt) continue;
#pragma unroll
        for (int i = 0; i < TT; ++i) {
            const int64_t tok = tok0 + (th * TT + i) * 16 + r;
            if (tok < T) *reinterpret_cast<f32x4_t*>(out + tok * E_pad + n * 16 + quad * 4) = acc[j][i];
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

// bf16 path, 16 lanes per token (four tokens per wave): lane j of a row holds
// experts j + 16 q. z = the KS partial logits summed in range order plus the
// bias; the softmax and the top-k rounds reduce inside the row with DPP
// moves only (no cross-row reads), ties to the lower expert index.
template <int Q>
__global__ void __launch_bounds__(kTopkWaves * 64)
router_topk_row_kernel(const float* __restrict__ part, int ks_n, int64_t T, int E, int E_pad,
                       const float* __restrict__ bias, int k, int renorm, float* __restrict__ logits,
                       float* __restrict__ probs, int32_t* __restrict__ topk_idx, float* __restrict__ topk_w) {
    const int lane = lane_id(), l16 = lane & 15;
    const int64_t tok = (static_cast<int64_t>(blockIdx.x) * kTopkWaves + threadIdx.x / kWave) * 4 + (lane >> 4);
    const bool live = tok < T;  // uniform in the row; every lane takes part in the row reductions
    float z[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int e = l16 + 16 * q;
        float v = -INFINITY;
        if (live && e < E) {
            v = part[tok * E_pad + e];
            for (int ks = 1; ks < ks_n; ++ks) v += part[(static_cast<int64_t>(ks) * T + tok) * E_pad + e];
            v += bias != nullptr ? bias[e] : 0.0f;
        }
        z[q] = v;
    }
    float lm = -INFINITY;
#pragma unroll
    for (int q = 0; q < Q; ++q) lm = fmaxf(lm, z[q]);
    const float m = row_allreduce(lm, [](float a, float b) { return fmaxf(a, b); });
    float ls = 0.0f, g[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        g[q] = l16 + 16 * q < E ? expf(z[q] - m) : 0.0f;
        ls += g[q];
    }
    const float inv = 1.0f / row_allreduce(ls, [](float a, float b) { return a + b; });
    if (live) {
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            const int e = l16 + 16 * q;
            if (e < E) {
                probs[tok * E + e] = g[q] * inv;
                if (logits != nullptr) logits[tok * E + e] = z[q];
            }
        }
    }
    uint32_t taken = 0;
    int my_i = 0;
    float my_w = 0.0f;
    for (int rr = 0; rr < k; ++rr) {
        float bv = -INFINITY;
        int bi = 0x7fffffff;
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            const int e = l16 + 16 * q;
            if (e < E && !((taken >> q) & 1u) && (bi == 0x7fffffff || z[q] > bv)) {
                bv = z[q];
                bi = e;
            }
        }
        const float gm = row_allreduce(bi == 0x7fffffff ? -INFINITY : bv, [](float a, float b) { return fmaxf(a, b); });
        const int gi = row_allreduce(bi != 0x7fffffff && bv == gm ? bi : 0x7fffffff,
                                     [](int a, int b) { return a < b ? a : b; });
        if ((gi & 15) == l16) taken |= 1u << (gi >> 4);
        if (l16 == rr) {
            my_i = gi;
            my_w = expf(gm - m) * inv;  // the chosen expert's gate value, as in probs
        }
    }
    if (renorm) my_w = my_w / row_allreduce(l16 < k ? my_w : 0.0f, [](float a, float b) { return a + b; });
    if (live && l16 < k) {
        topk_idx[tok * k + l16] = my_i;
        topk_w[tok * k + l16] = my_w;
    }
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
    const dim3 grid(static_cast<unsigned>(ceil_div(T, kLogitTokens)), static_cast<unsigned>(p.ks));
    const dim3 block(kLogitWaves * 64);
    switch (router_ne(E)) {
#define SMOES_ROUTER_NE(NE)                                                                                     \
    case NE:                                                                                                    \
        hipLaunchKernelGGL(router_logits_kernel<NE>, grid, block, 0, stream, x, T, d, wsplit, E_pad, p.steps, part); \
        break;
        SMOES_ROUTER_NE(1)
        SMOES_ROUTER_NE(2)
        SMOES_ROUTER_NE(3)
        SMOES_ROUTER_NE(4)
        SMOES_ROUTER_NE(5)
        SMOES_ROUTER_NE(6)
        SMOES_ROUTER_NE(7)
        SMOES_ROUTER_NE(8)
#undef SMOES_ROUTER_NE
        default:
            return hipErrorInvalidValue;
    }
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    // four tokens per wave (16 lanes each), kTopkWaves waves per block
    const dim3 tgrid(static_cast<unsigned>(ceil_div(T, 4 * kTopkWaves)));
    const dim3 tblock(kTopkWaves * 64);
    switch ((E + 15) / 16) {
#define SMOES_TOPK_Q(Q)                                                                                     \
    case Q:                                                                                                 \
        hipLaunchKernelGGL(router_topk_row_kernel<Q>, tgrid, tblock, 0, stream, part, p.ks, T, E, E_pad, bias, k, \
                           renorm, logits, probs, topk_idx, topk_w);                                        \
        break;
        SMOES_TOPK_Q(1) SMOES_TOPK_Q(2) SMOES_TOPK_Q(3) SMOES_TOPK_Q(4) SMOES_TOPK_Q(5) SMOES_TOPK_Q(6)
        SMOES_TOPK_Q(7) SMOES_TOPK_Q(8) SMOES_TOPK_Q(9) SMOES_TOPK_Q(10) SMOES_TOPK_Q(11) SMOES_TOPK_Q(12)
        SMOES_TOPK_Q(13) SMOES_TOPK_Q(14) SMOES_TOPK_Q(15) SMOES_TOPK_Q(16)
#undef SMOES_TOPK_Q
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
