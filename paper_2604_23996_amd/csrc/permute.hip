// Expert-contiguous permutation of the routed (token, slot) pairs: a stable
// counting sort by expert with tokens ascending inside each expert.
//
//   perm_count  : per 256-token chunk, per-expert counts (LDS integer adds:
//                 counts do not depend on their order).
//   perm_scan   : one block; per expert, exclusive prefix over chunks, then an
//                 exclusive scan over experts -> expert_offsets and the base
//                 row of every (chunk, expert).
//   perm_scatter: per chunk; for every expert a wave ballot marks the lanes
//                 (tokens) that chose it, so the rank of a token among the
//                 chunk's earlier tokens is a popcount: the row order comes
//                 from prefix sums only, never from atomics.
// Row gathers (x_perm) copy 16-byte vectors with consecutive lanes on
// consecutive addresses of one row.
#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

constexpr int kChunk = 256;

struct PermWs {
    int32_t* hist;  // [nchunk][E]
    int32_t* base;  // [nchunk][E]
};

PermWs carve(void* ws, int64_t T, int E) {
    const int64_t nchunk = ceil_div(T, kChunk);
    PermWs w;
    char* p = static_cast<char*>(ws);
    w.hist = reinterpret_cast<int32_t*>(p);
    p += align_up(sizeof(int32_t) * nchunk * E, 256);
    w.base = reinterpret_cast<int32_t*>(p);
    return w;
}

__global__ void __launch_bounds__(kChunk)
perm_count_kernel(const int32_t* __restrict__ idx, int64_t T, int E, int k, int32_t* __restrict__ hist) {
    __shared__ int cnt[256];
    for (int e = threadIdx.x; e < E; e += blockDim.x) cnt[e] = 0;
    __syncthreads();
    const int64_t j = static_cast<int64_t>(blockIdx.x) * kChunk + threadIdx.x;
    if (j < T)
        for (int s = 0; s < k; ++s) atomicAdd(&cnt[idx[j * k + s]], 1);
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += blockDim.x) hist[static_cast<int64_t>(blockIdx.x) * E + e] = cnt[e];
}

__global__ void __launch_bounds__(256)
perm_scan_kernel(int64_t nchunk, int E, const int32_t* __restrict__ hist, int32_t* __restrict__ base,
                 int32_t* __restrict__ expert_offsets) {
    __shared__ int tot[256];
    const int e = threadIdx.x;
    int running = 0;
    if (e < E) {
        for (int64_t c = 0; c < nchunk; ++c) {
            base[c * E + e] = running;
            running += hist[c * E + e];
        }
    }
    tot[e] = e < E ? running : 0;
    __syncthreads();
    // exclusive scan of the per-expert totals (Hillis-Steele on 256 entries)
    int v = tot[e];
    for (int o = 1; o < 256; o <<= 1) {
        const int add = e >= o ? tot[e - o] : 0;
        __syncthreads();
        v += add;
        tot[e] = v;
        __syncthreads();
    }
    const int excl = v - (e < E ? running : 0);
    if (e < E) {
        expert_offsets[e] = excl;
        for (int64_t c = 0; c < nchunk; ++c) base[c * E + e] += excl;
    }
    if (e == E - 1) expert_offsets[E] = v;
}

__device__ __forceinline__ uint64_t lanemask_lt() {
    const int lane = lane_id();
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

__global__ void __launch_bounds__(kChunk)
perm_scatter_kernel(const int32_t* __restrict__ idx, int64_t T, int E, int k,
                    const int32_t* __restrict__ base, int32_t* __restrict__ perm_token,
                    int32_t* __restrict__ perm_inv) {
    __shared__ uint64_t masks[kChunk / kWave][256];
    const int wave = threadIdx.x / kWave;
    const int lane = lane_id();
    const int64_t j = static_cast<int64_t>(blockIdx.x) * kChunk + threadIdx.x;
    const bool live = j < T;
    int sel[SMOES_K_MAX_DEV];
    uint64_t b0 = 0, b1 = 0, b2 = 0, b3 = 0;
#pragma unroll
    for (int s = 0; s < SMOES_K_MAX_DEV; ++s) {
        sel[s] = 0;
        if (live && s < k) {
            const int e = idx[j * k + s];
            sel[s] = e;
            const uint64_t bit = 1ull << (e & 63);
            const int blk = e >> 6;
            b0 |= blk == 0 ? bit : 0ull;
            b1 |= blk == 1 ? bit : 0ull;
            b2 |= blk == 2 ? bit : 0ull;
            b3 |= blk == 3 ? bit : 0ull;
        }
    }
    // one ballot per expert: which tokens of this wave chose it
    const uint64_t bits[4] = {b0, b1, b2, b3};
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
        const int e0 = blk * 64;
        if (e0 >= E) break;
        const int ne = E - e0 < 64 ? E - e0 : 64;
        const uint64_t mine = bits[blk];
        for (int t = 0; t < ne; ++t) {
            const uint64_t m = __ballot(static_cast<int>((mine >> t) & 1ull));
            if (lane == 0) masks[wave][e0 + t] = m;
        }
    }
    __syncthreads();
    if (!live) return;
    const int32_t* bc = base + static_cast<int64_t>(blockIdx.x) * E;
    const uint64_t lt = lanemask_lt();
#pragma unroll
    for (int s = 0; s < SMOES_K_MAX_DEV; ++s) {
        if (s < k) {
            const int e = sel[s];
            int pos = bc[e] + __popcll(masks[wave][e] & lt);
            for (int w = 0; w < wave; ++w) pos += __popcll(masks[w][e]);
            perm_token[pos] = static_cast<int32_t>(j);
            perm_inv[j * k + s] = pos;
        }
    }
}

template <bool BF16>
__global__ void gather_rows_kernel(const void* __restrict__ x, int d, const int32_t* __restrict__ perm_token,
                                   int64_t R, void* __restrict__ x_perm) {
    const int per_row = d / 8;  // 8 elements per vector
    const int64_t n = R * per_row;
    for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t r = i / per_row;
        const int c = static_cast<int>(i % per_row) * 8;
        const int64_t src = static_cast<int64_t>(perm_token[r]) * d + c;
        if constexpr (BF16) {
            *reinterpret_cast<uint4*>(static_cast<uint16_t*>(x_perm) + r * d + c) =
                *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(x) + src);
        } else {
            const float4* s = reinterpret_cast<const float4*>(static_cast<const float*>(x) + src);
            float4* t = reinterpret_cast<float4*>(static_cast<float*>(x_perm) + r * d + c);
            t[0] = s[0];
            t[1] = s[1];
        }
    }
}

}  // namespace

size_t permute_workspace_bytes(int64_t T, int E, int /*k*/) {
    const int64_t nchunk = ceil_div(T, kChunk);
    return 2 * align_up(sizeof(int32_t) * nchunk * E, 256);
}

hipError_t launch_permute(const int32_t* topk_idx, int64_t T, int E, int k,
                          int32_t* expert_offsets, int32_t* perm_token, int32_t* perm_inv,
                          void* ws, hipStream_t stream) {
    PermWs w = carve(ws, T, E);
    const int64_t nchunk = ceil_div(T, kChunk);
    hipError_t err;
    hipLaunchKernelGGL(perm_count_kernel, dim3(static_cast<unsigned>(nchunk)), dim3(kChunk), 0, stream,
                       topk_idx, T, E, k, w.hist);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    hipLaunchKernelGGL(perm_scan_kernel, dim3(1), dim3(256), 0, stream, nchunk, E, w.hist, w.base,
                       expert_offsets);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    hipLaunchKernelGGL(perm_scatter_kernel, dim3(static_cast<unsigned>(nchunk)), dim3(kChunk), 0, stream,
                       topk_idx, T, E, k, w.base, perm_token, perm_inv);
    return hipGetLastError();
}

hipError_t launch_gather_rows(const void* x, int x_dtype, int d, const int32_t* perm_token,
                              int64_t R, void* x_perm, hipStream_t stream) {
    if (R == 0) return hipSuccess;
    const int64_t n = R * (d / 8);
    const unsigned blocks = static_cast<unsigned>(ceil_div(n, 256) < 8192 ? ceil_div(n, 256) : 8192);
    if (x_dtype == 1)
        hipLaunchKernelGGL(gather_rows_kernel<true>, dim3(blocks), dim3(256), 0, stream, x, d,
                           perm_token, R, x_perm);
    else
        hipLaunchKernelGGL(gather_rows_kernel<false>, dim3(blocks), dim3(256), 0, stream, x, d,
                           perm_token, R, x_perm);
    return hipGetLastError();
}

}  // namespace smoes
