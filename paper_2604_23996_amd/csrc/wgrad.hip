// Expert weight gradients of the layer backward: for each group g (a routed
// expert over its expert-contiguous rows, or the merged shared expert over
// all tokens)
//   dW_g[m][n] = sum_r A[ra(r)][m] * B[rb(r)][n]
// where at most one operand has a row map (the permutation's token of a
// routed row): dW2 = dout^T (w H) with dout gathered, dW13 = [dA dB]^T X
// with x gathered.
//
// Tiles of 128 (m) x 256 (n), 4 waves of 64 x 128, K = the group's rows in
// stages of 32 through a 3-stage LDS ring filled by buffer loads straight to
// LDS (no staging registers), two stages in flight while one is consumed.
// Both operands sit row-major in LDS (rows = K, 256 or 512 bytes) with the
// 16-byte chunks of row r XOR-swizzled by 4 (r % 4); the MFMA fragments, 8
// consecutive rows of one column per lane, come from the transposing read
// ds_read_b64_tr_b16 (in each 16-lane group, lane j gives the address of row
// j / 4, columns 4 (j % 4) .. + 3, and receives column j of those four rows),
// which with that swizzle touches 64 distinct banks per 32 lanes. A row map
// is itself brought into LDS by a buffer load one stage ahead of the data it
// addresses. bf16 operands, fp32 accumulation, bf16 gradients written as
// full rows through LDS.
#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

constexpr int WG_TM = 128, WG_TN = 256, WG_BK = 32, WG_ST = 3, WG_THREADS = 256;
constexpr int WG_ARB = WG_TM * 2, WG_BRB = WG_TN * 2;          // row bytes in LDS
constexpr int WG_AB = WG_BK * WG_ARB, WG_BB = WG_BK * WG_BRB;  // 8 KB + 16 KB per stage
constexpr int WG_SB = WG_AB + WG_BB;
constexpr int WG_IA = WG_AB / 1024 / 4, WG_IB = WG_BB / 1024 / 4;  // 1 KB loads per wave per stage (2, 4)
constexpr int WG_IDX = 1024;                                      // row-map bytes per stage (4 waves x 256)
constexpr int WG_NI = 4;                                          // row-map slots
constexpr int WG_LDS = WG_ST * WG_SB + WG_NI * WG_IDX;
constexpr int WG_OP = WG_TN + 8;  // epilogue row pitch (elements)
static_assert(WG_TM * WG_OP * 2 <= WG_ST * WG_SB, "epilogue tile fits the ring");

typedef short wg_v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) wg_v4i16 wg_lds_v4i16;

struct WgArgs {
    int64_t T;
    int n_groups;           // E routed experts, or 1 (shared)
    int M, N;               // output rows / columns of every group
    const int32_t* off;     // [E + 1] row ranges of the routed groups; NULL: one group of T rows
    const uint16_t* A;      // row-major, lda columns, a_rows rows
    int lda, a_rows;
    const uint16_t* B;
    int ldb, b_rows;
    const int32_t* map;     // row map of the gathered operand ([map_len]); NULL: none
    int map_len;
    uint16_t* out;          // [n_groups][M][N]
};

__device__ __forceinline__ int wg_swz(int row) { return 4 * (row & 3); }

// G: 0 no row map, 1 A's rows through the map, 2 B's rows through the map.
template <int G>
__global__ void __launch_bounds__(WG_THREADS) __attribute__((amdgpu_waves_per_eu(2, 2)))
wgrad_kernel(WgArgs p) {
    __shared__ __attribute__((aligned(1024))) uint8_t lds[WG_LDS];
    const int tiles_m = static_cast<int>(ceil_div(p.M, WG_TM)), tiles_n = static_cast<int>(ceil_div(p.N, WG_TN));
    const int per = tiles_m * tiles_n;
    const int nblk = p.n_groups * per;
    // the tiles of one group run back to back on one XCD (block b runs on XCD b % 8)
    const int nb8 = static_cast<int>(ceil_div(nblk, 8));
    const int b = (blockIdx.x & 7) * nb8 + (blockIdx.x >> 3);
    if (b >= nblk) return;
    const int g = b / per, tt = b % per;
    const int m0 = (tt / tiles_n) * WG_TM, n0 = (tt % tiles_n) * WG_TN;
    const int r0 = uniform_int(p.off ? p.off[g] : 0);
    const int r1 = uniform_int(p.off ? p.off[g + 1] : static_cast<int>(p.T));
    const int nk = static_cast<int>(ceil_div(r1 - r0, WG_BK));
    const int wave = threadIdx.x / kWave, lane = lane_id();
    const int wm = wave >> 1, wn = wave & 1;
    uint8_t* idx_lds = lds + WG_ST * WG_SB;

    const i32x4_t rsA = buf_rsrc(p.A, p.a_rows * p.lda * 2);
    const i32x4_t rsB = buf_rsrc(p.B, p.b_rows * p.ldb * 2);
    const i32x4_t rsM = buf_rsrc(G ? p.map : nullptr, G ? p.map_len * 4 : 0);
    const uint32_t lds0 = lds_address(lds);

    // Load q of this wave (A: rows (wave * IA + q) * 4 + lane / 16, B: rows
    // (wave * IB + q) * 2 + lane / 32 of a stage) moves global chunk
    // (slot ^ swizzle(row)) of its row into slot lane % 16 (A) / lane % 32 (B).
    // Column offsets (elements) and the row in the stage are fixed per tile.
    int a_row[WG_IA], a_col[WG_IA], b_row[WG_IB], b_col[WG_IB];
#pragma unroll
    for (int q = 0; q < WG_IA; ++q) {
        a_row[q] = (wave * WG_IA + q) * 4 + lane / 16;
        const int col = m0 + ((lane % 16) ^ wg_swz(a_row[q])) * 8;
        a_col[q] = col < p.M ? col : -1;
    }
#pragma unroll
    for (int q = 0; q < WG_IB; ++q) {
        b_row[q] = (wave * WG_IB + q) * 2 + lane / 32;
        const int col = n0 + ((lane % 32) ^ wg_swz(b_row[q])) * 8;
        b_col[q] = col < p.N ? col : -1;
    }
    // Row map of stage s into index slot s % 4: wave w loads rows 8 w .. 8 w + 7
    // (lanes 0..7; the other lanes' loads are out of range and write zeros).
    auto issue_idx = [&](int s) {
        if constexpr (G != 0) {
            const int r = r0 + s * WG_BK + wave * 8 + lane;
            const int vo = (lane < 8 && r < r1) ? r * 4 : kOutOfRange;
            dma4(rsM, vo, lds0 + WG_ST * WG_SB + (s % WG_NI) * WG_IDX + wave * 256);
        }
    };
    auto map_of = [&](int s, int row) {
        return *reinterpret_cast<const int32_t*>(idx_lds + (s % WG_NI) * WG_IDX + (row / 8) * 256 + (row % 8) * 4);
    };
    // Byte offsets of this lane's loads for stage s (the map read from LDS);
    // kOutOfRange for rows past K and columns past the matrix.
    auto src_offs = [&](int s, int (&va)[WG_IA], int (&vb)[WG_IB]) {
#pragma unroll
        for (int q = 0; q < WG_IA; ++q) {
            const int r = r0 + s * WG_BK + a_row[q];
            const int src = r < r1 ? (G == 1 ? map_of(s, a_row[q]) : r) : -1;
            va[q] = (src >= 0 && a_col[q] >= 0) ? (src * p.lda + a_col[q]) * 2 : kOutOfRange;
        }
#pragma unroll
        for (int q = 0; q < WG_IB; ++q) {
            const int r = r0 + s * WG_BK + b_row[q];
            const int src = r < r1 ? (G == 2 ? map_of(s, b_row[q]) : r) : -1;
            vb[q] = (src >= 0 && b_col[q] >= 0) ? (src * p.ldb + b_col[q]) * 2 : kOutOfRange;
        }
    };
    auto issue_a = [&](int s, int q, int vo) {
        dma16(rsA, vo, lds0 + (s % WG_ST) * WG_SB + (wave * WG_IA + q) * 1024);
    };
    auto issue_b = [&](int s, int q, int vo) {
        dma16(rsB, vo, lds0 + (s % WG_ST) * WG_SB + WG_AB + (wave * WG_IB + q) * 1024);
    };

    f32x16_t acc[4][2];  // [n tile][m tile]: rows n, columns m
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int i = 0; i < 2; ++i) acc[q][i] = f32x16_t{};
    // per-lane part of the transposing reads: 16-lane group grp covers columns
    // 16 (grp & 1) .. + 15 of a 32-column tile and rows 8 (grp >> 1) .. + 7;
    // byte offsets in a stage for substep ks (rows 16 ks ..), the hi half 4
    // rows further (r % 4 is the same for both halves)
    const int grp = lane >> 4, j = lane & 15;
    const int trow = 8 * (grp >> 1) + (j >> 2), tcol = 16 * (grp & 1) + 4 * (j & 3);
    auto frag_off = [&](int rb, int k0, int c0) {
        const int col = c0 + tcol, r = k0 + trow;
        return static_cast<uint32_t>(r * rb + ((col >> 3) ^ wg_swz(r)) * 16 + (col & 7) * 2);
    };
    uint32_t fa[2][2], fb[2][4];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
        for (int i = 0; i < 2; ++i) fa[ks][i] = frag_off(WG_ARB, ks * 16, wm * 64 + i * 32);
#pragma unroll
        for (int q = 0; q < 4; ++q) fb[ks][q] = WG_AB + frag_off(WG_BRB, ks * 16, wn * 128 + q * 32);
    }
    auto frag = [&](uint32_t addr, auto rb4_c) {
        constexpr int RB4 = decltype(rb4_c)::value;
        const wg_v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((wg_lds_v4i16*)(uintptr_t)addr);
        const wg_v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((wg_lds_v4i16*)(uintptr_t)(addr + RB4));
        const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
        return __builtin_bit_cast(bf16x8_t, i32x4_t{static_cast<int>(l2.x), static_cast<int>(l2.y),
                                                    static_cast<int>(h2.x), static_cast<int>(h2.y)});
    };
    using RA4 = std::integral_constant<int, 4 * WG_ARB>;
    using RB4 = std::integral_constant<int, 4 * WG_BRB>;

    // Issue order: I(0), I(1) | D(0), I(2), D(1), I(3) | per stage s: I(s + 4),
    // D(s + 2). Stage s starts with its first substep's fragments in registers
    // (read at the end of stage s - 1). Halfway through it waits until at most
    // I(s + 4) and D(s + 2) may still fly (so D(s + 1) and I(s + 3) have
    // landed) and lgkmcnt is 0 (its second substep's fragments are in
    // registers), passes a barrier, and reads stage s + 1's first fragments
    // while its second substep's MFMAs run. After that barrier no wave reads
    // stage s's data slot any more (D(s + 3) overwrites it) nor the index slot
    // of stage s + 1 (I(s + 5) overwrites it). Past the end of K every load is
    // out of range and writes zeros, so the counts stay exact.
    constexpr int PEND = WG_IA + WG_IB + (G != 0 ? 1 : 0);
    const uint32_t sb0 = lds0;
    bf16x8_t mf[2][2], nf[2][4];
    auto read_frags = [&](uint32_t sb, int ks, bf16x8_t (&m)[2], bf16x8_t (&n)[4]) {
#pragma unroll
        for (int i = 0; i < 2; ++i) m[i] = frag(sb + fa[ks][i], RA4{});
#pragma unroll
        for (int q = 0; q < 4; ++q) n[q] = frag(sb + fb[ks][q], RB4{});
    };
    auto mfma_step = [&](const bf16x8_t (&m)[2], const bf16x8_t (&n)[4]) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int i = 0; i < 2; ++i)
                acc[q][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(n[q], m[i], acc[q][i], 0, 0, 0);
    };
    if constexpr (G != 0) {
        issue_idx(0);
        issue_idx(1);
        wait_vm_lgkm0<0>();
        __builtin_amdgcn_s_barrier();
    }
    {
        int va[WG_IA], vb[WG_IB];
        src_offs(0, va, vb);
#pragma unroll
        for (int q = 0; q < WG_IA; ++q) issue_a(0, q, va[q]);
#pragma unroll
        for (int q = 0; q < WG_IB; ++q) issue_b(0, q, vb[q]);
        issue_idx(2);
        src_offs(1, va, vb);
#pragma unroll
        for (int q = 0; q < WG_IA; ++q) issue_a(1, q, va[q]);
#pragma unroll
        for (int q = 0; q < WG_IB; ++q) issue_b(1, q, vb[q]);
        issue_idx(3);
        wait_vm_lgkm0<PEND>();  // D(0) and I(2) have landed
        __builtin_amdgcn_s_barrier();
        read_frags(sb0, 0, mf[0], nf[0]);
    }
    for (int s = 0; s < nk; ++s) {
        int va[WG_IA], vb[WG_IB];
        src_offs(s + 2, va, vb);
        issue_idx(s + 4);
        const uint32_t sb = lds0 + (s % WG_ST) * WG_SB;
#pragma unroll
        for (int q = 0; q < WG_IA; ++q) issue_a(s + 2, q, va[q]);
#pragma unroll
        for (int q = 0; q < WG_IB / 2; ++q) issue_b(s + 2, q, vb[q]);
        read_frags(sb, 1, mf[1], nf[1]);
        mfma_step(mf[0], nf[0]);
#pragma unroll
        for (int q = WG_IB / 2; q < WG_IB; ++q) issue_b(s + 2, q, vb[q]);
        wait_vm_lgkm0<PEND>();
        __builtin_amdgcn_s_barrier();
        if (s + 1 < nk) read_frags(lds0 + ((s + 1) % WG_ST) * WG_SB, 0, mf[0], nf[0]);
        mfma_step(mf[1], nf[1]);
    }
    wait_vm_lgkm0<0>();  // drain: the epilogue reuses the ring
    __builtin_amdgcn_s_barrier();

    // element v of lane l of acc[q][i]: n = 8 (v / 4) + 4 (l / 32) + v % 4 of
    // tile q, m = l % 32 of tile i; four adjacent n go to LDS as 8 bytes, then
    // whole 512-byte rows to memory
    uint16_t* ot = reinterpret_cast<uint16_t*>(lds);
    const int half = lane >> 5, l32 = lane & 31;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int vq = 0; vq < 4; ++vq) {
                const f32x16_t& a = acc[q][i];
                *reinterpret_cast<uint2*>(ot + (wm * 64 + i * 32 + l32) * WG_OP + wn * 128 + q * 32 + 8 * vq +
                                          4 * half) =
                    make_uint2(static_cast<uint32_t>(f32_to_bf16(a[4 * vq])) |
                                   (static_cast<uint32_t>(f32_to_bf16(a[4 * vq + 1])) << 16),
                               static_cast<uint32_t>(f32_to_bf16(a[4 * vq + 2])) |
                                   (static_cast<uint32_t>(f32_to_bf16(a[4 * vq + 3])) << 16));
            }
    __syncthreads();
    uint16_t* O = p.out + static_cast<int64_t>(g) * p.M * p.N;
    constexpr int CH = WG_TN / 8;
    for (int q = threadIdx.x; q < WG_TM * CH; q += WG_THREADS) {
        const int r = q / CH, c = (q % CH) * 8;
        if (m0 + r < p.M && n0 + c < p.N)  // N % 8 == 0: a chunk is all in or all out
            *reinterpret_cast<uint4*>(O + static_cast<int64_t>(m0 + r) * p.N + n0 + c) =
                *reinterpret_cast<const uint4*>(ot + r * WG_OP + c);
    }
}

}  // namespace

hipError_t launch_wgrad(int64_t T, int n_groups, int M, int N, const int32_t* off, const void* A, int lda,
                        int a_rows, const int32_t* amap, const void* B, int ldb, int b_rows, const int32_t* bmap,
                        int map_len, void* out, hipStream_t stream) {
    if (n_groups == 0 || M == 0 || N == 0) return hipSuccess;
    if (amap != nullptr && bmap != nullptr) return hipErrorInvalidValue;  // one row map at most
    WgArgs p;
    p.T = T;
    p.n_groups = n_groups;
    p.M = M;
    p.N = N;
    p.off = off;
    p.A = static_cast<const uint16_t*>(A);
    p.lda = lda;
    p.a_rows = a_rows;
    p.B = static_cast<const uint16_t*>(B);
    p.ldb = ldb;
    p.b_rows = b_rows;
    p.map = amap != nullptr ? amap : bmap;
    p.map_len = map_len;
    p.out = static_cast<uint16_t*>(out);
    const int64_t nblk = static_cast<int64_t>(n_groups) * ceil_div(M, WG_TM) * ceil_div(N, WG_TN);
    const dim3 grid(static_cast<unsigned>(8 * ceil_div(nblk, 8)));
    if (amap != nullptr) hipLaunchKernelGGL(wgrad_kernel<1>, grid, dim3(WG_THREADS), 0, stream, p);
    else if (bmap != nullptr) hipLaunchKernelGGL(wgrad_kernel<2>, grid, dim3(WG_THREADS), 0, stream, p);
    else hipLaunchKernelGGL(wgrad_kernel<0>, grid, dim3(WG_THREADS), 0, stream, p);
    return hipGetLastError();
}

}  // namespace smoes
