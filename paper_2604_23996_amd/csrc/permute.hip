// Expert-contiguous permutation of the routed (token, slot) pairs: a stable
// counting sort by expert with tokens ascending inside each expert.
//
//   perm_count  : per 256-token chunk, per-expert counts: for every expert a
//                 wave ballot of the lanes (tokens) that chose it and a
//                 popcount, the four waves' counts summed in wave order.
//   perm_scatter: per chunk; every block sums the chunk counts itself (per
//                 expert: the total and the part before its chunk), scans the
//                 totals over experts, and places its rows: for every expert a
//                 wave ballot marks the lanes (tokens) that chose it, so the
//                 rank of a token among the chunk's earlier tokens is a
//                 popcount. Counts and row order come from ballots and
//                 prefix sums only, never from atomics. Block 0 also writes
//                 expert_offsets and, when asked, the grouped GEMMs' work
//                 tables.
// Row gathers (x_perm) copy 16-byte vectors with consecutive lanes on
// consecutive addresses of one row.
#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

constexpr int kChunk = 256;
static_assert(kChunk / kWave == 4, "per-wave counts are summed as four terms");

struct PermWs {
    int32_t* hist;  // [nchunk][E]
};

PermWs carve(void* ws) {
    PermWs w;
    w.hist = static_cast<int32_t*>(ws);
    return w;
}

// Bit e & 63 of word e >> 6: the experts a token chose (E <= 256).
struct ExpertBits {
    uint64_t w[4];
};

__device__ __forceinline__ ExpertBits chosen_bits(const int32_t* __restrict__ idx, int64_t j, bool live, int k,
                                                  int (&sel)[SMOES_K_MAX_DEV]) {
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
    return ExpertBits{{b0, b1, b2, b3}};
}

__global__ void __launch_bounds__(kChunk)
perm_count_kernel(const int32_t* __restrict__ idx, int64_t T, int E, int k, int32_t* __restrict__ hist) {
    __shared__ int32_t cnt[kChunk / kWave][256];
    const int wave = threadIdx.x / kWave, lane = lane_id();
    const int64_t j = static_cast<int64_t>(blockIdx.x) * kChunk + threadIdx.x;
    int sel[SMOES_K_MAX_DEV];
    const ExpertBits eb = chosen_bits(idx, j, j < T, k, sel);
    // lane t of the wave ends with the count of expert e0 + t (experts past E
    // are never chosen: their ballots are empty)
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
        const int e0 = blk * 64;
        if (e0 >= E) break;
        const uint32_t lo = static_cast<uint32_t>(eb.w[blk]), hi = static_cast<uint32_t>(eb.w[blk] >> 32);
        int c = 0;
#pragma unroll
        for (int t = 0; t < 64; ++t) {
            const uint32_t bit = t < 32 ? (lo >> t) & 1u : (hi >> (t - 32)) & 1u;
            const int n = __popcll(__ballot(static_cast<int>(bit)));  // every lane takes part in the ballot
            c = lane == t ? n : c;
        }
        if (e0 + lane < E) cnt[wave][e0 + lane] = c;
    }
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += blockDim.x)
        hist[static_cast<int64_t>(blockIdx.x) * E + e] = (cnt[0][e] + cnt[1][e]) + (cnt[2][e] + cnt[3][e]);
}

__device__ __forceinline__ uint64_t lanemask_lt() {
    const int lane = lane_id();
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Block-wide inclusive scan of one int per thread (256 threads = 4 waves):
// each wave scans with shuffles, then adds the totals of the waves before it.
// sc holds at least 4 ints; it is free again when the function returns.
__device__ __forceinline__ int block_scan_incl(int v, int32_t* sc) {
    const int lane = lane_id();
    const int wave = threadIdx.x / kWave;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int t = __shfl_up(v, o);
        if (lane >= o) v += t;
    }
    if (lane == kWave - 1) sc[wave] = v;
    __syncthreads();
    int add = 0;
    for (int w = 0; w < wave; ++w) add += sc[w];
    __syncthreads();
    return v + add;
}

__global__ void __launch_bounds__(kChunk)
perm_scatter_kernel(const int32_t* __restrict__ idx, int64_t T, int E, int k, int64_t nchunk,
                    const int32_t* __restrict__ hist, int32_t* __restrict__ expert_offsets,
                    int32_t* __restrict__ perm_token, int32_t* __restrict__ perm_inv, WorkTables wt) {
    __shared__ uint64_t masks[kChunk / kWave][256];
    __shared__ int32_t base_s[256];
    __shared__ int32_t sc[kChunk];
    const int wave = threadIdx.x / kWave;
    const int lane = lane_id();
    {
        // per expert: total over all chunks and the part before this chunk (fixed order)
        const int e = threadIdx.x;
        int tot = 0, pre = 0;
        if (e < E) {
            // 32 independent loads in flight, summed in chunk order
            for (int64_t c0 = 0; c0 < nchunk; c0 += 32) {
                int h[32];
#pragma unroll
                for (int q = 0; q < 32; ++q) h[q] = c0 + q < nchunk ? hist[(c0 + q) * E + e] : 0;
#pragma unroll
                for (int q = 0; q < 32; ++q) {
                    tot += h[q];
                    pre += c0 + q < blockIdx.x ? h[q] : 0;
                }
            }
        }
        const int incl = block_scan_incl(tot, sc);
        const int excl = incl - tot;
        if (e < E) base_s[e] = excl + pre;
        if (blockIdx.x == 0) {
            if (e < E) expert_offsets[e] = excl;
            if (e == E - 1) expert_offsets[E] = incl;
            if (wt.work1 != nullptr) {
                // GEMM work tables: work[g + 1] = work[g] + m_tiles(g) * n_tiles
                const int mt = e < E ? static_cast<int>(ceil_div(tot, wt.bm)) : 0;
                const int mt_incl = block_scan_incl(mt, sc);
                const int shared_mt = wt.has_shared ? static_cast<int>(ceil_div(T, wt.bm)) : 0;
                if (e == 0) {
                    wt.work1[0] = 0;
                    wt.work2[0] = 0;
                }
                if (e < E) {
                    wt.work1[e + 1] = mt_incl * wt.nt1_r;
                    wt.work2[e + 1] = mt_incl * wt.nt2;
                }
                if (e == E - 1) {
                    wt.work1[E + 1] = mt_incl * wt.nt1_r + shared_mt * wt.nt1_s;
                    wt.work2[E + 1] = mt_incl * wt.nt2 + shared_mt * wt.nt2;
                }
            }
        }
    }
    const int64_t j = static_cast<int64_t>(blockIdx.x) * kChunk + threadIdx.x;
    const bool live = j < T;
    int sel[SMOES_K_MAX_DEV];
    const ExpertBits eb = chosen_bits(idx, j, live, k, sel);
    // one ballot per expert: which tokens of this wave chose it
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
        const int e0 = blk * 64;
        if (e0 >= E) break;
        const int ne = E - e0 < 64 ? E - e0 : 64;
        const uint64_t mine = eb.w[blk];
        for (int t = 0; t < ne; ++t) {
            const uint64_t m = __ballot(static_cast<int>((mine >> t) & 1ull));
            if (lane == 0) masks[wave][e0 + t] = m;
        }
    }
    __syncthreads();
    if (!live) return;
    const int32_t* bc = base_s;
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
    return align_up(sizeof(int32_t) * nchunk * E, 256);
}

hipError_t launch_permute(const int32_t* topk_idx, int64_t T, int E, int k,
                          int32_t* expert_offsets, int32_t* perm_token, int32_t* perm_inv,
                          void* ws, const WorkTables* work, hipStream_t stream) {
    PermWs w = carve(ws);
    const int64_t nchunk = ceil_div(T, kChunk);
    WorkTables wt{};
    if (work != nullptr) wt = *work;
    hipError_t err;
    hipLaunchKernelGGL(perm_count_kernel, dim3(static_cast<unsigned>(nchunk)), dim3(kChunk), 0, stream,
                       topk_idx, T, E, k, w.hist);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    hipLaunchKernelGGL(perm_scatter_kernel, dim3(static_cast<unsigned>(nchunk)), dim3(kChunk), 0, stream,
                       topk_idx, T, E, k, nchunk, w.hist, expert_offsets, perm_token, perm_inv, wt);
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
