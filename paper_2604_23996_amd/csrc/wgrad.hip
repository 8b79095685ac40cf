// Expert weight gradients of the layer backward: for each group g (a routed
// expert over its expert-contiguous rows, or the merged shared expert over
// all tokens)
//   dW_g[m][n] = sum_r A[ra(r)][m] * B[rb(r)][n]
// where at most one operand's rows go through a row map (the permutation's
// token of a routed row): dW2 = dout^T (w H) with dout gathered, dW13 =
// [dA dB]^T X with x gathered. Both operands are first written once more in
// the matrix cores' fragment order with the contraction (the group's rows)
// contiguous, then multiplied with the forward's packed tiling.
#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

// ============================================================ k-packed weight gradients
//
// The same products from operands stored once more, per group, in the matrix
// cores' fragment order with the contraction (the group's rows) contiguous:
// for a row-major S with C columns and a group of rows [r0, r1) (rows taken
// through a row map when given),
//   P[cg][ks][l][e] = S[row(r0 + 16 ks + 8 (l / 32) + e)][32 cg + l % 32],
// zero past the group's rows and past C; the groups follow each other, each
// padded to a multiple of 16 rows (kp: the padded row prefix). A fragment is
// one 1 KB block: lane l's 16 bytes are an MFMA operand as they are.
// wgrad_pk_kernel then runs the forward's packed tiling: 128 (m) x 256 (n)
// tiles, the m operand brought to LDS by buffer-to-LDS loads through a
// three-stage ring of K = 64 slices and read with plain 16-byte LDS reads, the
// n operand loaded straight into registers one slice ahead.

constexpr int KP_COLS = 256;  // source columns per k-pack block (8 column groups)

// Padded row prefix of the routed groups: kp[g + 1] = kp[g] + 16 ceil(rows_g / 16).
// a weight-gradient tile's fixed cost in 16-row slices: its start and its output
constexpr int kWpTileCost = 8;

__global__ void __launch_bounds__(256)
kpad_offsets_kernel(const int32_t* __restrict__ off, int E, int32_t* __restrict__ kp, int per0, int per1,
                    int32_t* __restrict__ ranges) {
    __shared__ int32_t sc[256];
    const int g = threadIdx.x;
    const int32_t rows = g < E ? ((off[g + 1] - off[g] + 15) / 16) * 16 : 0;
    sc[g] = rows;
    __syncthreads();
    for (int o = 1; o < 256; o <<= 1) {  // inclusive scan
        const int32_t v = g >= o ? sc[g - o] : 0;
        __syncthreads();
        sc[g] += v;
        __syncthreads();
    }
    if (g == 0) kp[0] = 0;
    if (g < E) kp[g + 1] = sc[g];
    if (ranges == nullptr || g >= E) return;
    // Tile ranges of the 8 XCDs with equal work for the two weight-gradient
    // launches (per0 and per1 tiles per group): a tile of group g costs its
    // 16-row slices plus kWpTileCost for its start and its output, and range
    // x starts at the first tile whose work ends after x / 8 of the total.
    // The group holding a boundary writes it.
    const int64_t w = rows / 16 + kWpTileCost;
    const int64_t pre = (sc[g] - rows) / 16 + static_cast<int64_t>(kWpTileCost) * g;  // work before g, per tile
    const int64_t all = sc[E - 1] / 16 + static_cast<int64_t>(kWpTileCost) * E;
    for (int h = 0; h < 2; ++h) {
        const int64_t per = h == 0 ? per0 : per1;
        int32_t* rg = ranges + 9 * h;
        if (g == 0) {
            rg[0] = 0;
            rg[8] = static_cast<int32_t>(per * E);
        }
        for (int x = 1; x < 8; ++x) {
            const int64_t target = per * all * x / 8;
            if (per * pre <= target && target < per * (pre + w)) {
                const int64_t o = (target - per * pre + w - 1) / w;
                rg[x] = static_cast<int32_t>(per * g + (o < per ? o : per));
            }
        }
    }
}

// One block per (16-row slice of the padded row space, 256 source columns):
// the slice's rows come into LDS as rows, and each lane writes one fragment
// lane (8 consecutive rows of one column) as 16 bytes.
__global__ void __launch_bounds__(256)
kpack_kernel(const uint16_t* __restrict__ S, int C, const int32_t* __restrict__ map, const int32_t* __restrict__ off,
             const int32_t* __restrict__ kp, int n_groups, int64_t T, uint16_t* __restrict__ P) {
    __shared__ __attribute__((aligned(16))) uint16_t tile[16][KP_COLS + 8];
    const int64_t prow = static_cast<int64_t>(blockIdx.x) * 16;  // first padded row of the slice
    int64_t kp0, kp1, r0, r1;
    if (kp == nullptr) {  // one group of T rows
        kp0 = 0;
        kp1 = ceil_div(T, 16) * 16;
        r0 = 0;
        r1 = T;
        if (prow >= kp1) return;
    } else {
        if (prow >= kp[n_groups]) return;  // past the padded total (the grid is sized for a bound)
        int lo = 0, hi = n_groups - 1;     // last g with kp[g] <= prow
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (kp[mid] <= prow) lo = mid; else hi = mid - 1;
        }
        kp0 = kp[lo];
        kp1 = kp[lo + 1];
        r0 = off[lo];
        r1 = off[lo + 1];
    }
    const int64_t ks = (prow - kp0) / 16, Ks = (kp1 - kp0) / 16;
    const int CG = static_cast<int>(ceil_div(C, 32));
    const int c0 = blockIdx.y * KP_COLS;
    for (int q = threadIdx.x; q < 16 * (KP_COLS / 8); q += blockDim.x) {
        const int rr = q / (KP_COLS / 8), ch = q % (KP_COLS / 8);
        const int64_t r = r0 + 16 * ks + rr;
        const int c = c0 + ch * 8;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (r < r1 && c < C) {  // C % 8 == 0: a chunk is all in or all out
            const int64_t src = map != nullptr ? static_cast<int64_t>(map[r]) : r;
            v = *reinterpret_cast<const uint4*>(S + src * C + c);
        }
        *reinterpret_cast<uint4*>(&tile[rr][ch * 8]) = v;
    }
    __syncthreads();
    uint16_t* Pg = P + 32 * static_cast<int64_t>(CG) * kp0;
    for (int q = threadIdx.x; q < (KP_COLS / 32) * 64; q += blockDim.x) {
        const int f = q / 64, l = q % 64;
        const int cg = c0 / 32 + f;
        if (cg >= CG) continue;
        const int col = f * 32 + (l & 31), rb = 8 * (l >> 5);
        uint32_t w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
            w[e] = static_cast<uint32_t>(tile[rb + 2 * e][col]) | (static_cast<uint32_t>(tile[rb + 2 * e + 1][col]) << 16);
        *reinterpret_cast<uint4*>(Pg + (static_cast<int64_t>(cg) * Ks + ks) * 512 + l * 8) =
            make_uint4(w[0], w[1], w[2], w[3]);
    }
}

constexpr int WP_BM = 128, WP_TN = 256, WP_BK = 64, WP_ST = 3, WP_THREADS = 256;
// m tiles per super-row of the tile order (16: 1504 -> 1473 us per routed launch at 16384 x 4096,
// 160 experts, against 8; 4: 1492 us)
constexpr int kWpGroupM = 16;
constexpr int WP_A_BYTES = WP_BM * WP_BK * 2;  // 16 fragments of 1 KB per stage
constexpr int WP_OP = WP_TN + 8;               // epilogue row pitch (elements)
constexpr int WP_EPI = 2 * WP_A_BYTES;         // epilogue staging: past ring slots 0 and 1
constexpr int WP_LDS = WP_EPI + (WP_BM / 2) * WP_OP * 2;
static_assert(WP_LDS >= WP_ST * WP_A_BYTES, "the ring fits");

struct WpArgs {
    int n_groups, M, N;
    const int32_t* kp;   // [n_groups + 1] padded row prefix, or NULL: one group of T rows
    const int32_t* ranges;  // [9] first tile of each XCD's range (work-balanced), or NULL: equal counts
    int64_t T;
    const uint16_t* PA;  // k-packed m operand (M source columns)
    const uint16_t* PB;  // k-packed n operand (N source columns)
    uint16_t* out;       // [n_groups][M][N] bf16
};

// Persistent: block (x = blockIdx % 8, seat) runs on XCD x and takes the
// tiles seat, seat + S, ... of XCD x's range (S blocks per XCD), so the
// resident blocks of an XCD work on consecutive tiles. The first two stages
// of a block's next tile are requested before the output of the current one
// is written (staged through LDS past ring slots 0 and 1, half a tile at a
// time, with buffer stores that every lane issues whatever the bounds), so
// the next tile's first data arrives while the stores drain.
__global__ void __launch_bounds__(WP_THREADS) __attribute__((amdgpu_waves_per_eu(2, 2)))
wgrad_pk_kernel(WpArgs p) {
    __shared__ __attribute__((aligned(1024))) uint8_t lds[WP_LDS];
    const int tiles_m = static_cast<int>(ceil_div(p.M, WP_BM)), tiles_n = static_cast<int>(ceil_div(p.N, WP_TN));
    const int per = tiles_m * tiles_n;
    const int nblk = p.n_groups * per;
    const int xcd = blockIdx.x & 7, seat = blockIdx.x >> 3, seats = gridDim.x >> 3;
    int lo, hi;
    if (p.ranges != nullptr) {
        lo = p.ranges[xcd];
        hi = p.ranges[xcd + 1];
    } else {
        const int nb8 = static_cast<int>(ceil_div(nblk, 8));
        lo = xcd * nb8 < nblk ? xcd * nb8 : nblk;
        hi = lo + nb8 < nblk ? lo + nb8 : nblk;
    }
    lo = uniform_int(lo);
    hi = uniform_int(hi);
    int b = lo + seat;
    if (b >= hi) return;
    const int MG = static_cast<int>(ceil_div(p.M, 32)), NG = static_cast<int>(ceil_div(p.N, 32));
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = lane_id();
    const int half = lane >> 5, l32 = lane & 31;

    // the tile whose operands are being requested: its group, corner and
    // 16-row slice count, the operand descriptors, and this lane's byte
    // offsets of slice 0 of its m fragment and its two n fragments (out of
    // range past the matrix edge)
    struct Tile {
        int g, m0, n0, Ks, va, vb0, vb1;
        i32x4_t rsA;
        __amdgpu_buffer_rsrc_t rsB;
    };
    auto decode = [&](int bb) {
        Tile t;
        t.g = bb / per;
        const int tt = bb % per;
        // inside a group: super-rows of kWpGroupM m tiles; each n tile's operand slice serves the
        // m tiles of a super-row back to back
        const int sr = tt / (kWpGroupM * tiles_n), r8 = tt % (kWpGroupM * tiles_n);
        const int gm = tiles_m - sr * kWpGroupM < kWpGroupM ? tiles_m - sr * kWpGroupM : kWpGroupM;
        t.m0 = (sr * kWpGroupM + r8 % gm) * WP_BM;
        t.n0 = (r8 / gm) * WP_TN;
        const int64_t kp0 = p.kp != nullptr ? p.kp[t.g] : 0;
        const int64_t kp1 = p.kp != nullptr ? p.kp[t.g + 1] : ceil_div(p.T, 16) * 16;
        t.Ks = uniform_int(static_cast<int>((kp1 - kp0) / 16));  // 16-row slices of the group
        const uint16_t* PAg = p.PA + 32 * static_cast<int64_t>(MG) * kp0;
        const uint16_t* PBg = p.PB + 32 * static_cast<int64_t>(NG) * kp0;
        t.rsA = buf_rsrc(PAg, MG * t.Ks * 1024);
        t.rsB = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(uniform_ptr(PBg)), 0,
                                                  uniform_int(NG * t.Ks * 1024), kBufferFlags);
        const int mg = t.m0 / 32 + wave, ng = t.n0 / 32 + 2 * wave;
        t.va = mg < MG ? (mg * t.Ks * 64 + lane) * 16 : kOutOfRange;
        t.vb0 = ng < NG ? (ng * t.Ks * 64 + lane) * 16 : kOutOfRange;
        t.vb1 = ng + 1 < NG ? ((ng + 1) * t.Ks * 64 + lane) * 16 : kOutOfRange;
        return t;
    };
    const uint32_t lds_base = lds_address(lds);
    // A DMA q of stage s: fragment (m group m0 / 32 + wave, slice 4 s + q) into LDS block wave * 4 + q of the slot
    auto issue_aq = [&](const Tile& t, int slot, int s, int q) {
        const int ks = 4 * s + q;
        const int vo = (t.va + ks * 1024) | (ks < t.Ks ? 0 : kOutOfRange);
        dma16(t.rsA, vo, lds_base + slot * WP_A_BYTES + (wave * 4 + q) * 1024);
    };
    // the two n fragments (n groups n0 / 32 + 2 wave + gg) of slice 4 s + j
    auto issue_bj = [&](const Tile& t, i32x4_t (&bq)[4][2], int s, int j) {
        const int ks = 4 * s + j;
        const int past = ks < t.Ks ? 0 : kOutOfRange;
        bq[j][0] = __builtin_amdgcn_raw_buffer_load_b128(t.rsB, (t.vb0 + ks * 1024) | past, 0, 0);
        bq[j][1] = __builtin_amdgcn_raw_buffer_load_b128(t.rsB, (t.vb1 + ks * 1024) | past, 0, 0);
    };
    i32x4_t b0[4][2], b1[4][2];
    // stages 0 and 1 of the decoded tile: 16 loads per wave, the 4 DMAs of stage 0 first
    auto prologue = [&](const Tile& t) {
#pragma unroll
        for (int q = 0; q < 4; ++q) issue_aq(t, 0, 0, q);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            issue_bj(t, b0, 0, j);
            issue_aq(t, 1, 1, j);
        }
    };
    f32x16_t acc[4][2];
    // stage s from ring slot `slot`: substep j issues the n fragments of stage
    // s + 1 (2 loads) and the DMA q = j of stage s + 2, reads the m fragments
    // of substep j + 1 and runs 8 MFMAs
    auto stage_run = [&](const Tile& t, int slot, int s, const i32x4_t (&bc)[4][2], i32x4_t (&bn)[4][2]) {
        const uint8_t* base = lds + slot * WP_A_BYTES;
        const int nslot = slot == 0 ? 2 : slot - 1;  // (slot + 2) % 3
        bf16x8_t af[2][4];
        auto rd = [&](int j, bf16x8_t (&a)[4]) {
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = *reinterpret_cast<const bf16x8_t*>(base + (i * 4 + j) * 1024 + lane * 16);
        };
        rd(0, af[0]);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            __builtin_amdgcn_sched_barrier(0);
            issue_bj(t, bn, s + 1, j);
            issue_aq(t, nslot, s + 2, j);
            if (j < 3) rd(j + 1, af[(j + 1) & 1]);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int gg = 0; gg < 2; ++gg)  // rows of the MFMA tile: n, columns: m
                    acc[i][gg] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(bf16x8_t, bc[j][gg]), af[j & 1][i], acc[i][gg], 0, 0, 0);
#pragma unroll
            for (int q = 0; q < 3; ++q) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    };
    // Vector memory operations retire in order. Before stage s reads its
    // slot, at most the loads issued after the last DMA of stage s may still
    // fly: for s >= 2 the 12 of stage s - 1's run (n fragments of stage s,
    // DMA of stage s + 1); for s = 0 and 1 of every tile but a block's first
    // also the 16 output stores of the previous tile, issued after this
    // tile's first two stages were requested. The barrier makes every
    // wave's DMA visible and frees the slot the DMA of stage s + 2
    // overwrites. Past the group's rows every load is out of range and
    // returns zeros, so every stage issues the same count and the waits stay
    // exact.
    constexpr int kStoresPerTile = (WP_BM * WP_TN / 8) / WP_THREADS;  // 16-byte stores per lane
    Tile cur = decode(b);
    prologue(cur);
    bool after_stores = false;
    for (;;) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int gg = 0; gg < 2; ++gg) acc[i][gg] = f32x16_t{};
        const int nk = static_cast<int>(ceil_div(cur.Ks, 4));
        {
            int s = 0, slot = 0;
            if (nk > 0) {
                if (after_stores) wait_vm_lgkm0<12 + kStoresPerTile>();
                else wait_vm_lgkm0<12>();
                __builtin_amdgcn_s_barrier();
                stage_run(cur, 0, 0, b0, b1);
            }
            if (nk > 1) {
                if (after_stores) wait_vm_lgkm0<12 + kStoresPerTile>();
                else wait_vm_lgkm0<12>();
                __builtin_amdgcn_s_barrier();
                stage_run(cur, 1, 1, b1, b0);
            }
            s = 2;
            slot = 2;
            for (; s + 2 <= nk; s += 2) {
                wait_vm_lgkm0<12>();
                __builtin_amdgcn_s_barrier();
                stage_run(cur, slot, s, b0, b1);
                slot = slot == 2 ? 0 : slot + 1;
                wait_vm_lgkm0<12>();
                __builtin_amdgcn_s_barrier();
                stage_run(cur, slot, s + 1, b1, b0);
                slot = slot == 2 ? 0 : slot + 1;
            }
            if (s < nk) {
                wait_vm_lgkm0<12>();
                __builtin_amdgcn_s_barrier();
                stage_run(cur, slot, s, b0, b1);
            }
        }
        wait_vm_lgkm0<0>();  // drain: the next tile's DMA reuses the ring
        __builtin_amdgcn_s_barrier();
        // output of this tile, then the next tile's first two stages
        const int og = cur.g, om0 = cur.m0, on0 = cur.n0;
        const int nb = b + seats;
        if (nb < hi) {
            cur = decode(nb);
            prologue(cur);
        }
        const __amdgpu_buffer_rsrc_t rsO = __builtin_amdgcn_make_buffer_rsrc(
            uniform_ptr(p.out + static_cast<int64_t>(og) * p.M * p.N), 0, uniform_int(p.M * p.N * 2), kBufferFlags);
        uint16_t* ot = reinterpret_cast<uint16_t*>(lds + WP_EPI);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            // element v of lane l of acc[i][gg]: n = 8 (v / 4) + 4 half + v % 4 of n group
            // 2 wave + gg of the tile, m = l32 of m group i; four adjacent n go to LDS as
            // 8 bytes, then whole rows of the half tile to memory
#pragma unroll
            for (int i = 2 * h; i < 2 * h + 2; ++i)
#pragma unroll
                for (int vq = 0; vq < 4; ++vq)
#pragma unroll
                    for (int gg = 0; gg < 2; ++gg) {
                        const f32x16_t& a = acc[i][gg];
                        *reinterpret_cast<uint2*>(ot + ((i - 2 * h) * 32 + l32) * WP_OP + wave * 64 + gg * 32 + 8 * vq +
                                                  4 * half) =
                            make_uint2(static_cast<uint32_t>(f32_to_bf16(a[4 * vq])) |
                                           (static_cast<uint32_t>(f32_to_bf16(a[4 * vq + 1])) << 16),
                                       static_cast<uint32_t>(f32_to_bf16(a[4 * vq + 2])) |
                                           (static_cast<uint32_t>(f32_to_bf16(a[4 * vq + 3])) << 16));
                    }
            __syncthreads();
            constexpr int CH = WP_TN / 8;
#pragma unroll
            for (int u = 0; u < kStoresPerTile / 2; ++u) {
                const int q = u * WP_THREADS + static_cast<int>(threadIdx.x);
                const int r = q / CH, c = (q % CH) * 8;
                const int row = om0 + 64 * h + r, col = on0 + c;
                // N % 8 == 0: a chunk is all in or all out; out of range the store is dropped
                const int vo = (row < p.M && col < p.N) ? (row * p.N + col) * 2 : kOutOfRange;
                __builtin_amdgcn_raw_buffer_store_b128(*reinterpret_cast<const i32x4_t*>(ot + r * WP_OP + c), rsO,
                                                       vo, 0, kBufferNonTemporal);
            }
            __syncthreads();  // the half tile's LDS reads are done before the next writes
        }
        if (nb >= hi) break;
        b = nb;
        after_stores = true;
    }
}

}  // namespace

int64_t kpack_elems(int C, int64_t padded_rows) { return 32 * ceil_div(C, 32) * padded_rows; }

int wgrad_tiles_per_group(int M, int N) { return static_cast<int>(ceil_div(M, WP_BM) * ceil_div(N, WP_TN)); }

hipError_t launch_kpad_offsets(const int32_t* off, int E, int32_t* kp, int per0, int per1, int32_t* ranges,
                               hipStream_t stream) {
    if (E < 1 || E > 256) return hipErrorInvalidValue;
    hipLaunchKernelGGL(kpad_offsets_kernel, dim3(1), dim3(256), 0, stream, off, E, kp, per0, per1, ranges);
    return hipGetLastError();
}

hipError_t launch_kpack(const void* S, int C, const int32_t* map, const int32_t* off, const int32_t* kp,
                        int n_groups, int64_t T, int64_t max_padded_rows, void* P, hipStream_t stream) {
    const int64_t slices = ceil_div(max_padded_rows, 16);
    if (slices == 0 || C == 0) return hipSuccess;
    const dim3 grid(static_cast<unsigned>(slices), static_cast<unsigned>(ceil_div(C, KP_COLS)));
    hipLaunchKernelGGL(kpack_kernel, grid, dim3(256), 0, stream, static_cast<const uint16_t*>(S), C, map, off, kp,
                       n_groups, T, static_cast<uint16_t*>(P));
    return hipGetLastError();
}

hipError_t launch_wgrad_pk(int n_groups, int M, int N, const int32_t* kp, const int32_t* ranges, int64_t T,
                           const void* PA, const void* PB, void* out, hipStream_t stream) {
    if (n_groups == 0 || M == 0 || N == 0) return hipSuccess;
    WpArgs p;
    p.n_groups = n_groups;
    p.M = M;
    p.N = N;
    p.kp = kp;
    p.ranges = ranges;
    p.T = T;
    p.PA = static_cast<const uint16_t*>(PA);
    p.PB = static_cast<const uint16_t*>(PB);
    p.out = static_cast<uint16_t*>(out);
    // two resident workgroups per CU, 32 CUs per XCD; fewer when there are fewer tiles
    const int64_t nblk = static_cast<int64_t>(n_groups) * ceil_div(M, WP_BM) * ceil_div(N, WP_TN);
    const int64_t per_xcd = ceil_div(nblk, 8) < 64 ? ceil_div(nblk, 8) : 64;
    hipLaunchKernelGGL(wgrad_pk_kernel, dim3(static_cast<unsigned>(8 * per_xcd)), dim3(WP_THREADS), 0, stream, p);
    return hipGetLastError();
}

}  // namespace smoes
