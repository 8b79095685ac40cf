// Expert weight gradients of the layer backward: for each group g (a routed
// expert over its expert-contiguous rows, or the merged shared expert over
// all tokens)
//   dW_g[m][n] = sum_r A[ra(r)][m] * sa(r) * B[rb(r)][n]
// with optional row maps (the permutation's token of a routed row) and a row
// scale (the combine weight): dW2 = (w dout)^T H, dW13 = [dA dB]^T X.
//
// Tiles of 128 (m) x 256 (n), 4 waves of 64 x 128, K = the group's rows in
// slices of 32. Both operands are staged row-major in LDS (rows = K) and the
// MFMA fragments, which need 8 consecutive rows of one column per lane, come
// from the transposing LDS read ds_read_b64_tr_b16 (in each 16-lane group,
// lane j gives the address of row j/4, columns 4 (j%4) .. + 3 and receives
// column j of those four rows). The accumulators hold n x m tiles, so each
// lane stores four adjacent n of one m as 8 bytes. bf16 operands, fp32
// accumulation, bf16 gradients.
#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

constexpr int WG_TM = 128, WG_TN = 256, WG_BK = 32, WG_THREADS = 256;
// row pitches (elements) at which the transposing reads hit distinct banks
constexpr int WG_PA = WG_TM + 32, WG_PB = WG_TN + 32;
constexpr int WG_ACH = WG_BK * WG_TM / 8 / WG_THREADS;  // 16-byte A chunks per thread per slice (2)
constexpr int WG_BCH = WG_BK * WG_TN / 8 / WG_THREADS;  // B chunks (4)

typedef int wg_i32x4 __attribute__((ext_vector_type(4)));
typedef short wg_v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) wg_v4i16 wg_lds_v4i16;

struct WgArgs {
    int64_t T;
    int n_groups;           // E routed experts, or 1 (shared)
    int M, N;               // output rows / columns of every group
    const int32_t* off;     // [E + 1] row ranges of the routed groups; NULL: one group of T rows
    const uint16_t* A;      // row-major, lda columns
    int64_t lda;
    const int32_t* amap;    // A row of each K row (NULL: identity)
    const float* ascale;    // scale of each K row (NULL: 1)
    const uint16_t* B;
    int64_t ldb;
    const int32_t* bmap;
    uint16_t* out;          // [n_groups][M][N]
};

__device__ __forceinline__ uint4 scale_bf16x8(uint4 v, float s) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float lo = __uint_as_float(w[i] << 16) * s, hi = __uint_as_float(w[i] & 0xffff0000u) * s;
        o[i] = static_cast<uint32_t>(f32_to_bf16(lo)) | (static_cast<uint32_t>(f32_to_bf16(hi)) << 16);
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
}

__global__ void __launch_bounds__(WG_THREADS) __attribute__((amdgpu_waves_per_eu(2, 2)))
wgrad_kernel(WgArgs p) {
    __shared__ __attribute__((aligned(16))) uint16_t a_lds[2][WG_BK * WG_PA];
    __shared__ __attribute__((aligned(16))) uint16_t b_lds[2][WG_BK * WG_PB];
    const int tiles_m = static_cast<int>(ceil_div(p.M, WG_TM)), tiles_n = static_cast<int>(ceil_div(p.N, WG_TN));
    const int per = tiles_m * tiles_n;
    const int nblk = p.n_groups * per;
    // the tiles of one group run back to back on one XCD (block b runs on XCD b % 8)
    const int nb8 = static_cast<int>(ceil_div(nblk, 8));
    const int b = (blockIdx.x & 7) * nb8 + (blockIdx.x >> 3);
    if (b >= nblk) return;
    const int g = b / per, tt = b % per;
    const int m0 = (tt / tiles_n) * WG_TM, n0 = (tt % tiles_n) * WG_TN;
    const int64_t r0 = p.off ? p.off[g] : 0, r1 = p.off ? p.off[g + 1] : p.T;
    const int nk = static_cast<int>(ceil_div(r1 - r0, WG_BK));
    const int wave = threadIdx.x / kWave, lane = lane_id();
    const int wm = wave >> 1, wn = wave & 1;

    uint4 ar[WG_ACH], br[WG_BCH];
    auto load_slice = [&](int kb) {
#pragma unroll
        for (int i = 0; i < WG_ACH; ++i) {
            const int id = threadIdx.x + i * WG_THREADS;
            const int row = id / (WG_TM / 8), c = id % (WG_TM / 8);
            const int64_t r = r0 + static_cast<int64_t>(kb) * WG_BK + row;
            const int col = m0 + c * 8;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (r < r1 && col < p.M) {
                const int64_t src = p.amap ? p.amap[r] : r;
                v = *reinterpret_cast<const uint4*>(p.A + src * p.lda + col);
                if (p.ascale) v = scale_bf16x8(v, p.ascale[r]);
            }
            ar[i] = v;
        }
#pragma unroll
        for (int i = 0; i < WG_BCH; ++i) {
            const int id = threadIdx.x + i * WG_THREADS;
            const int row = id / (WG_TN / 8), c = id % (WG_TN / 8);
            const int64_t r = r0 + static_cast<int64_t>(kb) * WG_BK + row;
            const int col = n0 + c * 8;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (r < r1 && col < p.N) {
                const int64_t src = p.bmap ? p.bmap[r] : r;
                v = *reinterpret_cast<const uint4*>(p.B + src * p.ldb + col);
            }
            br[i] = v;
        }
    };
    auto store_slice = [&](int buf) {
#pragma unroll
        for (int i = 0; i < WG_ACH; ++i) {
            const int id = threadIdx.x + i * WG_THREADS;
            *reinterpret_cast<uint4*>(&a_lds[buf][(id / (WG_TM / 8)) * WG_PA + (id % (WG_TM / 8)) * 8]) = ar[i];
        }
#pragma unroll
        for (int i = 0; i < WG_BCH; ++i) {
            const int id = threadIdx.x + i * WG_THREADS;
            *reinterpret_cast<uint4*>(&b_lds[buf][(id / (WG_TN / 8)) * WG_PB + (id % (WG_TN / 8)) * 8]) = br[i];
        }
    };

    f32x16_t acc[4][2];  // [n tile][m tile]: rows n, columns m
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int i = 0; i < 2; ++i) acc[q][i] = f32x16_t{};
    // per-lane part of the transposing reads: 16-lane group grp covers columns
    // 16 (grp & 1) .. + 15 of a 32-column tile and rows 8 (grp >> 1) .. + 7
    const int grp = lane >> 4, j = lane & 15;
    const int trow = 8 * (grp >> 1) + (j >> 2), tcol = 16 * (grp & 1) + 4 * (j & 3);
    auto frag = [&](const uint16_t* base, int pitch, int k0, int c0) {
        const wg_v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((wg_lds_v4i16*)(base + (k0 + trow) * pitch + c0 + tcol));
        const wg_v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((wg_lds_v4i16*)(base + (k0 + 4 + trow) * pitch + c0 + tcol));
        const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
        return __builtin_bit_cast(bf16x8_t, wg_i32x4{static_cast<int>(l2.x), static_cast<int>(l2.y),
                                                     static_cast<int>(h2.x), static_cast<int>(h2.y)});
    };

    if (nk > 0) load_slice(0);
    for (int kb = 0; kb < nk; ++kb) {
        const int buf = kb & 1;
        store_slice(buf);
        __syncthreads();  // the slice is visible; the other buffer's readers (slice kb - 1) are done
        if (kb + 1 < nk) load_slice(kb + 1);
        const uint16_t* al = a_lds[buf];
        const uint16_t* bl = b_lds[buf];
#pragma unroll
        for (int ks = 0; ks < WG_BK / 16; ++ks) {
            bf16x8_t mf[2], nf[4];
#pragma unroll
            for (int i = 0; i < 2; ++i) mf[i] = frag(al, WG_PA, ks * 16, wm * 64 + i * 32);
#pragma unroll
            for (int q = 0; q < 4; ++q) nf[q] = frag(bl, WG_PB, ks * 16, wn * 128 + q * 32);
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int i = 0; i < 2; ++i)
                    acc[q][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(nf[q], mf[i], acc[q][i], 0, 0, 0);
        }
    }
    // element v of lane l of acc[q][i]: n = 8 (v / 4) + 4 (l / 32) + v % 4 of tile q, m = l % 32 of tile i
    uint16_t* O = p.out + static_cast<int64_t>(g) * p.M * p.N;
    const int half = lane >> 5, l32 = lane & 31;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int m = m0 + wm * 64 + i * 32 + l32;
        if (m >= p.M) continue;
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int vq = 0; vq < 4; ++vq) {
                const int n = n0 + wn * 128 + q * 32 + 8 * vq + 4 * half;
                if (n >= p.N) continue;  // N % 4 == 0
                const f32x16_t& a = acc[q][i];
                *reinterpret_cast<uint2*>(O + static_cast<int64_t>(m) * p.N + n) = make_uint2(
                    static_cast<uint32_t>(f32_to_bf16(a[4 * vq])) | (static_cast<uint32_t>(f32_to_bf16(a[4 * vq + 1])) << 16),
                    static_cast<uint32_t>(f32_to_bf16(a[4 * vq + 2])) | (static_cast<uint32_t>(f32_to_bf16(a[4 * vq + 3])) << 16));
            }
    }
}

}  // namespace

hipError_t launch_wgrad(int64_t T, int n_groups, int M, int N, const int32_t* off, const void* A, int64_t lda,
                        const int32_t* amap, const float* ascale, const void* B, int64_t ldb, const int32_t* bmap,
                        void* out, hipStream_t stream) {
    if (n_groups == 0 || M == 0 || N == 0) return hipSuccess;
    WgArgs p;
    p.T = T;
    p.n_groups = n_groups;
    p.M = M;
    p.N = N;
    p.off = off;
    p.A = static_cast<const uint16_t*>(A);
    p.lda = lda;
    p.amap = amap;
    p.ascale = ascale;
    p.B = static_cast<const uint16_t*>(B);
    p.ldb = ldb;
    p.bmap = bmap;
    p.out = static_cast<uint16_t*>(out);
    const int64_t nblk = static_cast<int64_t>(n_groups) * ceil_div(M, WG_TM) * ceil_div(N, WG_TN);
    hipLaunchKernelGGL(wgrad_kernel, dim3(static_cast<unsigned>(8 * ceil_div(nblk, 8))), dim3(WG_THREADS), 0, stream,
                       p);
    return hipGetLastError();
}

}  // namespace smoes
