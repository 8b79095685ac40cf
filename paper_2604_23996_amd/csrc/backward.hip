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
//  dwgate: dW_gate[e][c] = sum_j dz_je x_jc and dbias_e = sum_j dz_je. For
//     bf16 x on the matrix cores: dz is split into three bf16 terms whose sum
//     is dz exactly (every product with a bf16 x is then exact in float32),
//     packed in MFMA fragment order; workgroups of 256 columns x up to 160
//     experts sum token ranges into partials; a range-ordered sum finishes.
//     float32 x: FMA partials per 256-token chunk, then a chunk-ordered sum.
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

// dw_gate = sum over the nchunk partials in chunk order (4 consecutive
// entries per thread, 8 partials in flight). dbias: workgroup b < ceil(E / 32)
// sums experts 32 b .. 32 b + 31, thread group j over the partials j, j + 8,
// ..., then the 8 group sums in order. The grid covers both.
__global__ void __launch_bounds__(256)
dwgate_reduce_kernel(const float* __restrict__ part, int64_t nchunk, const float* __restrict__ bpart, int64_t nbchunk,
                     int d, int E, float* __restrict__ dw_gate, float* __restrict__ dbias) {
    __shared__ float bsum[8][32];
    if (dbias != nullptr && static_cast<int>(blockIdx.x) * 32 < E) {  // uniform per workgroup
        const int j = threadIdx.x >> 5, e = blockIdx.x * 32 + (threadIdx.x & 31);
        float acc = 0.0f;
        if (e < E) {
            int64_t ch = j;
            for (; ch + 24 < nbchunk; ch += 32) {
                float v[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) v[u] = bpart[(ch + 8 * u) * E + e];
#pragma unroll
                for (int u = 0; u < 4; ++u) acc += v[u];
            }
            for (; ch < nbchunk; ch += 8) acc += bpart[ch * E + e];
        }
        bsum[j][threadIdx.x & 31] = acc;
        __syncthreads();
        if (threadIdx.x < 32 && e < E) {
            float t = 0.0f;
#pragma unroll
            for (int q = 0; q < 8; ++q) t += bsum[q][threadIdx.x];
            dbias[e] = t;
        }
    }
    const int64_t n = static_cast<int64_t>(E) * d;  // d % 8 == 0: n % 4 == 0
    const int64_t i = 4 * (blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x);
    if (i < n) {
        float4 acc = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        int64_t ch = 0;
        for (; ch + 8 <= nchunk; ch += 8) {
            float4 v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = *reinterpret_cast<const float4*>(part + (ch + u) * n + i);
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                acc.x += v[u].x;
                acc.y += v[u].y;
                acc.z += v[u].z;
                acc.w += v[u].w;
            }
        }
        for (; ch < nchunk; ++ch) {
            const float4 v = *reinterpret_cast<const float4*>(part + ch * n + i);
            acc.x += v.x;
            acc.y += v.y;
            acc.z += v.z;
            acc.w += v.w;
        }
        dw_gate[i] = acc.x;  // the caller's array may be only 4-byte aligned
        dw_gate[i + 1] = acc.y;
        dw_gate[i + 2] = acc.z;
        dw_gate[i + 3] = acc.w;
    }
}

// ---- dW_gate on the matrix cores (bf16 x)
//
// v_mfma_f32_32x32x16_bf16 with A = x (rows: 32 columns of x, contraction:
// 16 tokens) and B = dz (columns: 32 experts). A wave owns 64 columns as two
// interleaved tiles (tile q holds the columns c0 + 2 i + q), so each lane
// builds both A fragments from 8 dword reads (one token each) of x rows kept
// as rows in LDS. The three dz terms of an expert tile come pre-packed as B
// fragments. Both operands reach LDS by buffer-to-LDS DMA through a 3-slot
// ring of one 16-token slice each.
constexpr int kDgCols = 256;     // columns per workgroup (4 waves x 64)
constexpr int kDgMaxET = 5;      // 32-expert tiles per workgroup at most
constexpr int kDgSt = 3;         // ring slots
constexpr int kDgXPair = 1056;   // LDS bytes per token pair of x: two 512-byte rows + 32 (the two halves of a
                                 // wave then read disjoint banks)
constexpr int kDgTerms = 3;
__host__ __device__ constexpr int dg_slot_bytes(int et) { return et * kDgTerms * 1024 + 8 * kDgXPair; }
__host__ __device__ constexpr int dg_dmas(int et) { return (et * kDgTerms + 8 + 3) / 4; }  // per wave per slice

// Pz fragment (ks, et, term), lane l: dz[16 ks + 8 (l / 32) + i][32 et + l % 32] term, i < 8 (zero
// outside T x E). bpart[b][e]: sum of dz over the 64 tokens of slices 4 b .. 4 b + 3.
__global__ void __launch_bounds__(256)
dg_pack_kernel(const float* __restrict__ dz, int64_t T, int E, int ETt, int64_t KS, uint16_t* __restrict__ Pz,
               float* __restrict__ bpart) {
    __shared__ float red[4][64];
    const int lane = threadIdx.x & 63, sl = threadIdx.x >> 6;
    const int64_t ks = static_cast<int64_t>(blockIdx.x) * 4 + sl;
    const int et = blockIdx.y;
    const int64_t t0 = 16 * ks + 8 * (lane >> 5);
    const int e = 32 * et + (lane & 31);
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = (ks < KS && t0 + i < T && e < E) ? dz[(t0 + i) * E + e] : 0.0f;
    if (ks < KS) {
        uint32_t w[kDgTerms][4];
#pragma unroll
        for (int i = 0; i < 8; i += 2) {
            uint16_t h[kDgTerms][2];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                float r = v[i + u];
#pragma unroll
                for (int term = 0; term < kDgTerms; ++term) {  // r - bf16(r) is exact in float32
                    h[term][u] = f32_to_bf16(r);
                    r -= bf16_to_f32(h[term][u]);
                }
            }
#pragma unroll
            for (int term = 0; term < kDgTerms; ++term)
                w[term][i / 2] = static_cast<uint32_t>(h[term][0]) | (static_cast<uint32_t>(h[term][1]) << 16);
        }
#pragma unroll
        for (int term = 0; term < kDgTerms; ++term)
            *reinterpret_cast<uint4*>(Pz + (((ks * ETt + et) * kDgTerms + term) * 64 + lane) * 8) =
                make_uint4(w[term][0], w[term][1], w[term][2], w[term][3]);
    }
    float b = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) b += v[i];
    red[sl][lane] = b;
    __syncthreads();
    if (threadIdx.x < 32 && e < E) {
        float acc = 0.0f;
#pragma unroll
        for (int q = 0; q < 4; ++q) acc += red[q][threadIdx.x] + red[q][threadIdx.x + 32];
        bpart[static_cast<int64_t>(blockIdx.x) * E + e] = acc;
    }
}

// Workgroup (column block, token range s, expert group): part[s][e][c] for its 256
// columns and EG expert tiles over slices s * kps .. min(KS, (s + 1) * kps).
template <int EG>
__global__ void __launch_bounds__(256, 2)
dg_mfma_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ Pz, int64_t T, int d, int E, int ETt,
               int64_t KS, int kps, float* __restrict__ part) {
    constexpr int SLOT = dg_slot_bytes(EG), ND = dg_dmas(EG), NF = EG * kDgTerms + 8;
    constexpr int XOFF = EG * kDgTerms * 1024;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[kDgSt * SLOT + 1024];  // + 1 KB sink for padding DMAs
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = lane_id();
    const int cb = blockIdx.x, s = blockIdx.y, et0 = blockIdx.z * EG;
    const int64_t ks0 = static_cast<int64_t>(s) * kps;
    const int64_t ks1 = ks0 + kps < KS ? ks0 + kps : KS;
    const int nks = static_cast<int>(ks1 - ks0);
    const i32x4_t rsX = buf_rsrc(x, static_cast<int>(T * d * 2));
    const i32x4_t rsZ = buf_rsrc(Pz, static_cast<int>(KS * ETt * kDgTerms * 1024));
    const uint32_t lds0 = lds_address(lds);
    const int xcol = cb * kDgCols + (lane & 31) * 8;  // the 8 columns this lane's x DMA moves
    // the DMAs of slice n (relative to ks0) into ring slot `slot`: wave w moves fragments w, w + 4, ...
    auto issue = [&](int n, int slot) {
        const int64_t ks = ks0 + n;
#pragma unroll
        for (int i = 0; i < ND; ++i) {
            const int f = wave + 4 * i;
            int vo = kOutOfRange;
            uint32_t dst = lds0 + kDgSt * SLOT;  // sink
            if (f < EG * kDgTerms) {
                const int et = et0 + f / kDgTerms;
                if (ks < ks1 && et < ETt)
                    vo = static_cast<int>(((ks * ETt + et) * kDgTerms + f % kDgTerms) * 1024) + lane * 16;
                dst = lds0 + slot * SLOT + f * 1024;
            } else if (f < NF) {
                const int pr = f - EG * kDgTerms;  // token pair
                const int64_t t = 16 * ks + 2 * pr + (lane >> 5);
                if (ks < ks1 && t < T && xcol < d) vo = static_cast<int>((t * d + xcol) * 2);
                dst = lds0 + slot * SLOT + XOFF + pr * kDgXPair;
            }
            dma16(f < EG * kDgTerms ? rsZ : rsX, vo, dst);
        }
    };
    f32x16_t acc[2][EG];
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int et = 0; et < EG; ++et) acc[q][et] = f32x16_t{};
    issue(0, 0);
    issue(1, 1);
    int slot = 0;
    // Slice n waits for its own DMAs (only slice n + 1's, ND per wave, may fly);
    // the barrier frees the slot that slice n + 2 then overwrites.
    for (int n = 0; n < nks; ++n) {
        wait_vm_lgkm0<ND>();
        __builtin_amdgcn_s_barrier();
        issue(n + 2, slot == 0 ? 2 : slot - 1);
        const uint8_t* base = lds + slot * SLOT;
        // x: token 8 (lane / 32) + r of the slice, columns c0 + 2 (lane % 32) and + 1
        uint32_t w[8];
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            const int tt = 8 * (lane >> 5) + r;
            w[r] = *reinterpret_cast<const uint32_t*>(base + XOFF + (tt >> 1) * kDgXPair + (tt & 1) * 512 +
                                                      (wave * 64 + 2 * (lane & 31)) * 2);
        }
        bf16x8_t a[2];
        {
            uint32_t lo[4], hi[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                lo[r] = (w[2 * r] & 0xffffu) | (w[2 * r + 1] << 16);
                hi[r] = (w[2 * r] >> 16) | (w[2 * r + 1] & 0xffff0000u);
            }
            a[0] = __builtin_bit_cast(bf16x8_t, make_uint4(lo[0], lo[1], lo[2], lo[3]));
            a[1] = __builtin_bit_cast(bf16x8_t, make_uint4(hi[0], hi[1], hi[2], hi[3]));
        }
#pragma unroll
        for (int et = 0; et < EG; ++et)
#pragma unroll
            for (int term = 0; term < kDgTerms; ++term) {
                const bf16x8_t bz = *reinterpret_cast<const bf16x8_t*>(base + (et * kDgTerms + term) * 1024 + lane * 16);
#pragma unroll
                for (int q = 0; q < 2; ++q)
                    acc[q][et] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[q], bz, acc[q][et], 0, 0, 0);
            }
        slot = slot == 2 ? 0 : slot + 1;
    }
    wait_vm_lgkm0<0>();  // no DMA may still write LDS when the workgroup ends
    // element v of lane l of acc[q][et]: expert 32 (et0 + et) + l % 32, column c0 + 2 i + q with
    // i = 8 (v / 4) + 4 (l / 32) + v % 4: for each v / 4 the lane holds 8 consecutive columns
    const int c0 = cb * kDgCols + wave * 64;
    float* P = part + static_cast<int64_t>(s) * E * d;
#pragma unroll
    for (int et = 0; et < EG; ++et) {
        const int e = 32 * (et0 + et) + (lane & 31);
        if (e >= E) continue;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int c = c0 + 16 * g + 8 * (lane >> 5);
            if (c >= d) continue;  // d % 8 == 0: 8 columns are all in or all out
            const f32x16_t& u = acc[0][et];
            const f32x16_t& v = acc[1][et];
            float4* o = reinterpret_cast<float4*>(P + static_cast<int64_t>(e) * d + c);
            o[0] = make_float4(u[4 * g], v[4 * g], u[4 * g + 1], v[4 * g + 1]);
            o[1] = make_float4(u[4 * g + 2], v[4 * g + 2], u[4 * g + 3], v[4 * g + 3]);
        }
    }
}

// workgroups of dwgate_reduce_kernel: 4 entries per thread, and one per 32 experts for dbias
int64_t dwgate_reduce_blocks(int64_t n, int E) {
    const int64_t a = ceil_div(n / 4, 256), b = ceil_div(E, 32);
    return a > b ? a : b;
}

// ---- dx on the matrix cores (bf16 layers)
//
// dx_j = dz_j W_gate + sum_s dX_r[inv(j, s)] + dXs_j: D[c][j] = sum_e
// W_gate[e][c] dz[j][e] on v_mfma_f32_32x32x16_bf16 with both float32
// operands split into two bf16 terms (hi * hi + hi * lo + lo * hi: relative
// error about 2^-16 per product), from fragments packed beforehand. The 64
// tokens x 256 columns of a workgroup then go through LDS as rows, and the
// gathered row gradients are added in the order above with whole-row loads.
constexpr int kDxTerms = 2;
constexpr int kDxBT = 64;    // tokens per workgroup
constexpr int kDxBC = 256;   // columns per workgroup (4 waves x 2 tiles of 32)
constexpr int kDxPitch = kDxBC + 4;  // LDS row pitch in floats

// Fragment (a, ks, term), lane l, element r: src[m * sm + kk * sk] term with
// m = 32 a + l % 32 < M, kk = 16 ks + 8 (l / 32) + r < K (zero outside).
__global__ void __launch_bounds__(256)
frag_pack_kernel(const float* __restrict__ src, int64_t M, int K, int64_t sm, int64_t sk, int KS, int64_t n_frag,
                 uint16_t* __restrict__ out) {
    const int64_t q = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x;  // (fragment, lane)
    const int64_t f = q >> 6;
    if (f >= n_frag) return;
    const int lane = static_cast<int>(q & 63);
    const int64_t a = f / KS;
    const int ks = static_cast<int>(f % KS);
    const int64_t m = 32 * a + (lane & 31);
    const int kk0 = 16 * ks + 8 * (lane >> 5);
    uint32_t w[kDxTerms][4];
#pragma unroll
    for (int r = 0; r < 8; r += 2) {
        uint16_t h[kDxTerms][2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            float v = (m < M && kk0 + r + u < K) ? src[m * sm + static_cast<int64_t>(kk0 + r + u) * sk] : 0.0f;
#pragma unroll
            for (int term = 0; term < kDxTerms; ++term) {
                h[term][u] = f32_to_bf16(v);
                v -= bf16_to_f32(h[term][u]);
            }
        }
#pragma unroll
        for (int term = 0; term < kDxTerms; ++term)
            w[term][r / 2] = static_cast<uint32_t>(h[term][0]) | (static_cast<uint32_t>(h[term][1]) << 16);
    }
#pragma unroll
    for (int term = 0; term < kDxTerms; ++term)
        *reinterpret_cast<uint4*>(out + ((f * kDxTerms + term) * 64 + lane) * 8) =
            make_uint4(w[term][0], w[term][1], w[term][2], w[term][3]);
}

__global__ void __launch_bounds__(256, 2)
dx_mfma_kernel(const uint16_t* __restrict__ PW, const uint16_t* __restrict__ PZ, int KS, const uint16_t* __restrict__ dx_r,
               const uint16_t* __restrict__ dx_s, const int32_t* __restrict__ inv, int64_t T, int d, int k,
               float* __restrict__ dx) {
    __shared__ __attribute__((aligned(16))) float tile[kDxBT][kDxPitch];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = lane_id();
    const int64_t tb = blockIdx.x;
    const int cb = blockIdx.y;
    const int CT = static_cast<int>(ceil_div(d, 32));
    const int64_t TT = ceil_div(T, 32);
    const int ct0 = cb * (kDxBC / 32) + 2 * wave;
    const int64_t tt0 = 2 * tb;
    f32x16_t acc[2][2];
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int u = 0; u < 2; ++u) acc[q][u] = f32x16_t{};
    // D rows: 32 columns of W_gate (A = W_gate^T), D columns: 32 tokens (B = dz^T)
    for (int ks = 0; ks < KS; ++ks) {
        bf16x8_t a[2][kDxTerms], b[2][kDxTerms];
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
            for (int term = 0; term < kDxTerms; ++term) {
                const int ct = ct0 + q;
                a[q][term] = ct < CT ? *reinterpret_cast<const bf16x8_t*>(
                                           PW + ((static_cast<int64_t>(ct) * KS + ks) * kDxTerms + term) * 512 + lane * 8)
                                     : bf16x8_t{};
                const int64_t tt = tt0 + q;
                b[q][term] = tt < TT ? *reinterpret_cast<const bf16x8_t*>(
                                           PZ + ((tt * KS + ks) * kDxTerms + term) * 512 + lane * 8)
                                     : bf16x8_t{};
            }
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                acc[q][u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[q][0], b[u][0], acc[q][u], 0, 0, 0);
                acc[q][u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[q][0], b[u][1], acc[q][u], 0, 0, 0);
                acc[q][u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[q][1], b[u][0], acc[q][u], 0, 0, 0);
            }
    }
    // element v of lane l of acc[q][u]: column 64 wave + 32 q + 8 (v / 4) + 4 (l / 32) + v % 4 of the
    // workgroup, token 32 u + l % 32
    const int half = lane >> 5, l32 = lane & 31;
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int g = 0; g < 4; ++g)
                *reinterpret_cast<float4*>(&tile[32 * u + l32][64 * wave + 32 * q + 8 * g + 4 * half]) =
                    make_float4(acc[q][u][4 * g], acc[q][u][4 * g + 1], acc[q][u][4 * g + 2], acc[q][u][4 * g + 3]);
    __syncthreads();
    // 8 columns of one token per item; 32 threads cover a row
    constexpr int NIT = kDxBT * (kDxBC / 8) / 256;  // 8 items per thread
    constexpr int BATCH = 4;
#pragma unroll
    for (int p0 = 0; p0 < NIT; p0 += BATCH) {
        float v[BATCH][8];
        int64_t j[BATCH];
        int c[BATCH];
        bool ok[BATCH];
#pragma unroll
        for (int u = 0; u < BATCH; ++u) {
            const int it = static_cast<int>(threadIdx.x) + 256 * (p0 + u);
            const int r = it / (kDxBC / 8), ch = it % (kDxBC / 8);
            j[u] = tb * kDxBT + r;
            c[u] = cb * kDxBC + 8 * ch;
            ok[u] = j[u] < T && c[u] < d;  // d % 8 == 0: 8 columns are all in or all out
            const float4 x0 = *reinterpret_cast<const float4*>(&tile[r][8 * ch]);
            const float4 x1 = *reinterpret_cast<const float4*>(&tile[r][8 * ch + 4]);
            v[u][0] = x0.x; v[u][1] = x0.y; v[u][2] = x0.z; v[u][3] = x0.w;
            v[u][4] = x1.x; v[u][5] = x1.y; v[u][6] = x1.z; v[u][7] = x1.w;
        }
        auto add8 = [](float (&acc8)[8], const uint4 w) {
            acc8[0] += __uint_as_float(w.x << 16);
            acc8[1] += __uint_as_float(w.x & 0xffff0000u);
            acc8[2] += __uint_as_float(w.y << 16);
            acc8[3] += __uint_as_float(w.y & 0xffff0000u);
            acc8[4] += __uint_as_float(w.z << 16);
            acc8[5] += __uint_as_float(w.z & 0xffff0000u);
            acc8[6] += __uint_as_float(w.w << 16);
            acc8[7] += __uint_as_float(w.w & 0xffff0000u);
        };
        // four slots at a time: the row indices, then all their row loads, then the sums in slot order
        for (int s0 = 0; s0 < k; s0 += 4) {
            int row[BATCH][4];
#pragma unroll
            for (int u = 0; u < BATCH; ++u)
#pragma unroll
                for (int q = 0; q < 4; ++q) row[u][q] = (ok[u] && s0 + q < k) ? inv[j[u] * k + s0 + q] : -1;
            uint4 w[BATCH][4];
#pragma unroll
            for (int u = 0; u < BATCH; ++u)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    w[u][q] = row[u][q] >= 0
                                  ? *reinterpret_cast<const uint4*>(dx_r + static_cast<int64_t>(row[u][q]) * d + c[u])
                                  : make_uint4(0, 0, 0, 0);
#pragma unroll
            for (int u = 0; u < BATCH; ++u)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (s0 + q < k) add8(v[u], w[u][q]);
        }
        if (dx_s != nullptr) {
            uint4 w[BATCH];
#pragma unroll
            for (int u = 0; u < BATCH; ++u)
                w[u] = ok[u] ? *reinterpret_cast<const uint4*>(dx_s + j[u] * d + c[u]) : make_uint4(0, 0, 0, 0);
#pragma unroll
            for (int u = 0; u < BATCH; ++u) add8(v[u], w[u]);
        }
#pragma unroll
        for (int u = 0; u < BATCH; ++u)
            if (ok[u]) {
                float4* o = reinterpret_cast<float4*>(dx + j[u] * d + c[u]);
                o[0] = make_float4(v[u][0], v[u][1], v[u][2], v[u][3]);
                o[1] = make_float4(v[u][4], v[u][5], v[u][6], v[u][7]);
            }
    }
}

struct DgGeom {
    int ETt, G, EG, colb, S, kps;
    int64_t KS;
};

// Launch shape of the matrix-core dW_gate: expert tiles split into G groups of
// at most kDgMaxET, token ranges sized so there are about 512 workgroups.
DgGeom dg_geom(int64_t T, int d, int E) {
    DgGeom g;
    g.ETt = static_cast<int>(ceil_div(E, 32));
    g.G = static_cast<int>(ceil_div(g.ETt, kDgMaxET));
    g.EG = static_cast<int>(ceil_div(g.ETt, g.G));
    g.colb = static_cast<int>(ceil_div(d, kDgCols));
    g.KS = ceil_div(T, 16);
    int64_t S = ceil_div(512, static_cast<int64_t>(g.colb) * g.G);
    S = S < 64 ? S : 64;
    S = S < g.KS ? S : g.KS;
    S = S > 1 ? S : 1;
    g.kps = g.KS > 0 ? static_cast<int>(ceil_div(g.KS, S)) : 1;  // no tokens: S = 0 partial slabs
    g.S = static_cast<int>(ceil_div(g.KS, g.kps));
    return g;
}

// the packed dz is addressed with 32-bit byte offsets
bool dg_fits(int64_t T, int E) {
    return ceil_div(T, 16) * ceil_div(E, 32) * kDgTerms * 1024 <= INT32_MAX;
}

}  // namespace

size_t router_bwd_workspace_bytes(int64_t T, int d, int E, int bf16) {
    if (bf16 && dg_fits(T, E)) {
        const DgGeom g = dg_geom(T, d, E);
        return align_up(sizeof(float) * g.S * E * d, 256) + align_up(sizeof(uint16_t) * g.KS * g.ETt * kDgTerms * 512, 256) +
               align_up(sizeof(float) * ceil_div(g.KS, 4) * E, 256);
    }
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

size_t dx_mfma_workspace_bytes(int64_t T, int d, int E) {
    const int64_t KS = ceil_div(E, 16);
    return align_up(sizeof(uint16_t) * ceil_div(d, 32) * KS * kDxTerms * 512, 256) +
           align_up(sizeof(uint16_t) * ceil_div(T, 32) * KS * kDxTerms * 512, 256);
}

hipError_t launch_dx_gather(const void* dx_r, const void* dx_s, int bf16, const int32_t* perm_inv, const float* dz,
                            const float* w_gate, int64_t T, int d, int E, int k, float* dx, void* ws,
                            hipStream_t stream) {
    if (T == 0) return hipSuccess;
    if (bf16 && ws != nullptr) {
        const int KS = static_cast<int>(ceil_div(E, 16));
        const int64_t CT = ceil_div(d, 32), TT = ceil_div(T, 32);
        uint16_t* PW = static_cast<uint16_t*>(ws);
        uint16_t* PZ = reinterpret_cast<uint16_t*>(static_cast<char*>(ws) +
                                                   align_up(sizeof(uint16_t) * CT * KS * kDxTerms * 512, 256));
        hipError_t err;
        hipLaunchKernelGGL(frag_pack_kernel, dim3(static_cast<unsigned>(ceil_div(CT * KS * 64, 256))), dim3(256), 0,
                           stream, w_gate, static_cast<int64_t>(d), E, static_cast<int64_t>(1), static_cast<int64_t>(d),
                           KS, CT * KS, PW);
        if ((err = hipGetLastError()) != hipSuccess) return err;
        hipLaunchKernelGGL(frag_pack_kernel, dim3(static_cast<unsigned>(ceil_div(TT * KS * 64, 256))), dim3(256), 0,
                           stream, dz, T, E, static_cast<int64_t>(E), static_cast<int64_t>(1), KS, TT * KS, PZ);
        if ((err = hipGetLastError()) != hipSuccess) return err;
        const dim3 grid(static_cast<unsigned>(ceil_div(T, kDxBT)), static_cast<unsigned>(ceil_div(d, kDxBC)));
        hipLaunchKernelGGL(dx_mfma_kernel, grid, dim3(256), 0, stream, PW, PZ, KS,
                           static_cast<const uint16_t*>(dx_r), static_cast<const uint16_t*>(dx_s), perm_inv, T, d, k,
                           dx);
        return hipGetLastError();
    }
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
    hipError_t err;
    const int64_t n = static_cast<int64_t>(E) * d;
    if (bf16 && dg_fits(T, E)) {
        const DgGeom g = dg_geom(T, d, E);
        float* part = static_cast<float*>(ws);
        uint16_t* Pz = reinterpret_cast<uint16_t*>(static_cast<char*>(ws) + align_up(sizeof(float) * g.S * E * d, 256));
        float* bpart = reinterpret_cast<float*>(reinterpret_cast<char*>(Pz) +
                                                align_up(sizeof(uint16_t) * g.KS * g.ETt * kDgTerms * 512, 256));
        const int64_t nb = ceil_div(g.KS, 4);
        if (g.KS > 0) {
            hipLaunchKernelGGL(dg_pack_kernel, dim3(static_cast<unsigned>(nb), static_cast<unsigned>(g.ETt)), dim3(256),
                               0, stream, dz, T, E, g.ETt, g.KS, Pz, bpart);
            if ((err = hipGetLastError()) != hipSuccess) return err;
            const dim3 grid(static_cast<unsigned>(g.colb), static_cast<unsigned>(g.S), static_cast<unsigned>(g.G));
            const uint16_t* xb = static_cast<const uint16_t*>(x);
            switch (g.EG) {
                case 1: hipLaunchKernelGGL(dg_mfma_kernel<1>, grid, dim3(256), 0, stream, xb, Pz, T, d, E, g.ETt, g.KS, g.kps, part); break;
                case 2: hipLaunchKernelGGL(dg_mfma_kernel<2>, grid, dim3(256), 0, stream, xb, Pz, T, d, E, g.ETt, g.KS, g.kps, part); break;
                case 3: hipLaunchKernelGGL(dg_mfma_kernel<3>, grid, dim3(256), 0, stream, xb, Pz, T, d, E, g.ETt, g.KS, g.kps, part); break;
                case 4: hipLaunchKernelGGL(dg_mfma_kernel<4>, grid, dim3(256), 0, stream, xb, Pz, T, d, E, g.ETt, g.KS, g.kps, part); break;
                default: hipLaunchKernelGGL(dg_mfma_kernel<5>, grid, dim3(256), 0, stream, xb, Pz, T, d, E, g.ETt, g.KS, g.kps, part); break;
            }
            if ((err = hipGetLastError()) != hipSuccess) return err;
        }
        hipLaunchKernelGGL(dwgate_reduce_kernel, dim3(static_cast<unsigned>(dwgate_reduce_blocks(n, E))),
                           dim3(256), 0, stream, part, static_cast<int64_t>(g.KS > 0 ? g.S : 0), bpart, nb, d, E, dw_gate,
                           dbias);
        return hipGetLastError();
    }
    const int64_t nchunk = ceil_div(T, kDwChunk);
    float* part = static_cast<float*>(ws);
    float* bpart = reinterpret_cast<float*>(static_cast<char*>(ws) + align_up(sizeof(float) * nchunk * E * d, 256));
    if (nchunk > 0) {
        const dim3 grid(static_cast<unsigned>(ceil_div(d, 256)), static_cast<unsigned>(ceil_div(E, kDwExp)),
                        static_cast<unsigned>(nchunk));
        if (bf16)
            hipLaunchKernelGGL(dwgate_partial_kernel<true>, grid, dim3(256), 0, stream, dz, x, T, d, E, part, bpart);
        else
            hipLaunchKernelGGL(dwgate_partial_kernel<false>, grid, dim3(256), 0, stream, dz, x, T, d, E, part, bpart);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    hipLaunchKernelGGL(dwgate_reduce_kernel, dim3(static_cast<unsigned>(dwgate_reduce_blocks(n, E))),
                       dim3(256), 0, stream, part, nchunk, bpart, nchunk, d, E, dw_gate, dbias);
    return hipGetLastError();
}

}  // namespace smoes
