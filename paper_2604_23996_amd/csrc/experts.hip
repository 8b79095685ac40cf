// Grouped SwiGLU experts, shared experts and the weighted combine.
//
// Groups: g < E is routed expert g over its expert-contiguous rows
// [off[g], off[g+1]) (rows gathered from x through perm_token inside the
// GEMM's loader, so no permuted copy of x is written); g = E is the merged
// shared expert over all T tokens. A work table (prefix over groups of
// m_tiles * n_tiles, written on the device by the permutation) lets one
// launch cover every group without any host synchronisation.
//
// Block -> tile mapping: blocks are dealt round-robin to the 8 XCDs, so block b
// runs on XCD b % 8. Each XCD takes one contiguous eighth of the work list,
// ordered (group, super-row of m-tiles, n-tile, m-tile): the tiles that share
// a weight slice run back to back on one XCD and hit its L2 (8 m-tiles per
// super-row for the row-major path; the packed path picks the count per
// product).
//
// bf16, packed weights (the fast path, gemm_bf16_pk_kernel): 16x16x32 MFMA
// tiles with the weights loaded straight into registers; its layout and
// schedule are described where it is defined.
// bf16, row-major weights: 128 x 128 tiles, 4 waves of 64 x 64 (2 x 2 MFMA
// 32x32x16 bf16 tiles), fp32 accumulation. Operand tiles are copied HBM ->
// LDS by buffer loads with an LDS destination (no register staging) through
// a three-stage ring of K = 32 slices; the MFMA fragments are read back with
// 16-byte LDS reads from XOR-swizzled rows. The results leave through LDS as
// 16-byte row chunks.
//   GEMM1: B rows 0..63 are gate rows, 64..127 the matching up rows, so a
//          wave holds gate and up outputs of the same (row, column) in the
//          same lane: the SwiGLU epilogue is register-local. H is bf16.
//   GEMM2: Y = H W2^T, bf16.
// f32 (exact path for float32 layers): 64 x 64 FMA tiles, same work table.
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

constexpr int kThreads = 256;
constexpr int kGroupM = 8;  // m-tiles per super-row in the work order

// f32 FMA tiles
constexpr int FBM = 64, FBNB = 64, FBK = 16;

struct ExpWs {
    void* h_r;   // [R, inter]
    void* h_s;   // [T, shared_inter]
    void* y_r;   // [R, d]
    void* y_s;   // [T, d]
    int32_t* work1;  // [E + 2]
    int32_t* work2;  // [E + 2]
};

size_t esz(int act_dtype) { return act_dtype == 1 ? 2 : 4; }

ExpWs carve(void* ws, int64_t T, int d, int k, int inter, int shared_inter, int act_dtype, int E) {
    ExpWs w;
    const int64_t R = T * k;
    char* p = static_cast<char*>(ws);
    const size_t s = esz(act_dtype);
    w.h_r = p;
    p += align_up(s * R * inter, 256);
    w.h_s = p;
    p += align_up(s * T * shared_inter, 256);
    w.y_r = p;
    p += align_up(s * R * d, 256);
    w.y_s = p;
    p += align_up(s * T * d, 256);
    w.work1 = reinterpret_cast<int32_t*>(p);
    p += align_up(sizeof(int32_t) * (E + 2), 256);
    w.work2 = reinterpret_cast<int32_t*>(p);
    return w;
}

struct Tile {
    int g;          // group (E = shared)
    int64_t row0;   // first row of the tile in the group's row space (global row index)
    int rows;       // valid rows in the tile
    int nt;         // n-tile
};

// Decode this block's tile; returns false when the block has no work.
// Block b runs on XCD b % 8. The routed items and the shared-expert items are
// each cut into 8 contiguous ranges, one per XCD, so every XCD gets the same
// share of both kinds (shared tiles can have a longer K than routed ones).
// Inside a group items run (super-row of group_m m-tiles, n-tile, m-tile).
// part: 0 every item, 1 routed items only, 2 shared items only. The shared
// part never reads the work table (its item count follows from T and the
// tiling), so it can run before the routing has been permuted.
__device__ __forceinline__ bool decode_tile(const int32_t* __restrict__ work, const int32_t* __restrict__ off,
                                            int E, int64_t T, int bm, int nt_routed, int nt_shared,
                                            int part, Tile& t, int group_m = kGroupM) {
    const int xcd = blockIdx.x & 7;
    const int slot = blockIdx.x >> 3;
    int g, local;
    if (part == 2) {
        const int ns = static_cast<int>(ceil_div(T, bm)) * nt_shared;
        const int s8 = (ns + 7) / 8;
        const int s_lo = min(xcd * s8, ns), s_hi = min(s_lo + s8, ns);
        if (slot >= s_hi - s_lo) return false;
        g = E;
        local = s_lo + slot;
    } else {
        const int routed = work[E];
        const int ns = part == 1 ? 0 : work[E + 1] - routed;
        const int r8 = (routed + 7) / 8, s8 = (ns + 7) / 8;
        const int r_lo = min(xcd * r8, routed), r_hi = min(r_lo + r8, routed);
        const int s_lo = min(xcd * s8, ns), s_hi = min(s_lo + s8, ns);
        // shared items first: their K can be longer (GEMM2), and blocks are
        // dispatched in index order, so the longest tiles start earliest
        int w;
        if (slot < s_hi - s_lo) w = routed + s_lo + slot;
        else if (slot < (s_hi - s_lo) + (r_hi - r_lo)) w = r_lo + (slot - (s_hi - s_lo));
        else return false;
        if (w >= routed) {
            g = E;
        } else {
            int lo = 0, hi = E - 1;  // last g with work[g] <= w
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (work[mid] <= w) lo = mid; else hi = mid - 1;
            }
            g = lo;
        }
        local = w - work[g];
    }
    int64_t base, rows_g;
    int ntn;
    if (g < E) {
        base = off[g];
        rows_g = off[g + 1] - off[g];
        ntn = nt_routed;
    } else {
        base = 0;
        rows_g = T;
        ntn = nt_shared;
    }
    const int m_tiles = static_cast<int>(ceil_div(rows_g, bm));
    const int sb = local / (group_m * ntn);
    const int r = local % (group_m * ntn);
    const int gm = m_tiles - sb * group_m < group_m ? m_tiles - sb * group_m : group_m;
    const int mt = sb * group_m + r % gm;
    t.g = g;
    t.nt = r / gm;
    t.row0 = base + static_cast<int64_t>(mt) * bm;
    const int64_t left = rows_g - static_cast<int64_t>(mt) * bm;
    t.rows = static_cast<int>(left < bm ? left : bm);
    return true;
}

__device__ __forceinline__ float silu(float a) { return a / (1.0f + expf(-a)); }

__device__ __forceinline__ uint4 as_uint4(i32x4_t v) {
    return make_uint4(static_cast<uint32_t>(v.x), static_cast<uint32_t>(v.y), static_cast<uint32_t>(v.z),
                      static_cast<uint32_t>(v.w));
}

struct GemmArgs {
    int64_t T;
    int d, E, k, inter, shared_inter;
    int packed;  // expert weights in the fragment order of pack_weights_kernel
    int part;    // work items of this launch: 0 all, 1 routed, 2 shared
    const void* x;
    const void* w13;
    const void* w2;
    const void* ws13;
    const void* ws2;
    const int32_t* off;
    const int32_t* perm_token;
    const int32_t* work;
    void* h_r;
    void* h_s;
    void* y_r;
    void* y_s;
    // backward (modes 3-5 of the packed kernel)
    const void* dout;   // [T][d] upstream gradient
    const void* w2t;    // packed W2^T per expert (N = inter, K = d)
    const void* ws2t;   // packed Ws2^T (N = shared_inter, K = d)
    const void* w13t;   // packed W13^T per expert (N = d, K = 2 inter)
    const void* ws13t;  // packed Ws13^T (N = d, K = 2 shared_inter)
    void* ab_r;         // [R][2 inter] pre-activations (gate | up), routed rows
    void* ab_s;         // [T][2 shared_inter]
    void* dab_r;        // [R][2 inter] their gradients
    void* dab_s;        // [T][2 shared_inter]
    void* dx_r;         // [R][d] input gradient of each routed row
    void* dx_s;         // [T][d] shared experts' input gradient
    const float* wrow;  // [R] combine weight of each routed row
    void* wh_r;         // [R][inter] w H of each routed row (mode 4 output)
    // shared down GEMM with the combine in its epilogue (mode 7)
    const int32_t* inv;    // [T][k] routed row of each (token, slot)
    const float* topk_w;   // [T][k] combine weights
    void* out;             // [T][d] layer output
};

// ============================================================== bf16 MFMA path

// The operand tiles go straight from HBM to LDS (buffer_load ... lds: each wave instruction writes
// 64 x 16 bytes contiguously), through a ring of STAGES buffers, with one
// barrier per K step and no VGPR staging. Rows are unpadded (BK bf16) and the
// 16-byte chunks of a row are XOR-swizzled with (row / SWZ_DIV) % CPR so that
// the MFMA fragment reads of consecutive rows fall in different banks.
template <int WAVES_M_, int WAVES_N_, int TM_, int TN_, int BK_, int STAGES_, int SWZ_DIV_>
struct DmaCfg {
    static constexpr int WAVES_M = WAVES_M_, WAVES_N = WAVES_N_, TM = TM_, TN = TN_, BK = BK_;
    static constexpr int STAGES = STAGES_, SWZ_DIV = SWZ_DIV_;
    static constexpr int THREADS = WAVES_M * WAVES_N * 64;
    static constexpr int BM = WAVES_M * TM * 32;
    static constexpr int BNB = WAVES_N * TN * 32;
    static constexpr int CPR = BK / 8;                 // 16-byte chunks per row
    static constexpr int RPI = 64 / CPR;               // rows per DMA instruction (1 KB)
    static constexpr int IA = BM / RPI / (THREADS / 64);   // A instructions per wave per stage
    static constexpr int IB = BNB / RPI / (THREADS / 64);  // B instructions per wave per stage
    static_assert(IA * RPI * (THREADS / 64) == BM && IB * RPI * (THREADS / 64) == BNB, "tile / wave mismatch");
    static_assert(TN % 2 == 0, "gate/up pairs need an even TN");
};

// 128 rows x 128 B-rows (GEMM1: 64 gate + 64 up rows; GEMM2: 128 output columns),
// 4 waves of 64 x 64, K step 32, three-stage ring (48 KB of LDS: 3 blocks per CU)
using DCfg = DmaCfg<2, 2, 2, 2, 32, 3, 2>;

template <class C>
constexpr int tile_cols(int mode) { return mode == 1 ? C::BNB / 2 : C::BNB; }

template <class C>
__device__ __forceinline__ int dma_slot(int row, int chunk) {
    return chunk ^ ((row / C::SWZ_DIV) % C::CPR);
}


template <int MODE, class C>
__global__ void __launch_bounds__(C::THREADS, 1)
gemm_bf16_dma_kernel(GemmArgs p) {
    constexpr int BM = C::BM, BNB = C::BNB, BK = C::BK, CPR = C::CPR, RPI = C::RPI;
    constexpr int TM = C::TM, TN = C::TN, IA = C::IA, IB = C::IB, ST = C::STAGES;
    constexpr int A_BYTES = BM * BK * 2, B_BYTES = BNB * BK * 2;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[ST][A_BYTES + B_BYTES];
    constexpr int TC = tile_cols<C>(MODE);
    const int nt_r = static_cast<int>(ceil_div(MODE == 1 ? p.inter : p.d, TC));
    const int nt_s = MODE == 1 ? static_cast<int>(ceil_div(p.shared_inter, TC)) : nt_r;
    Tile t;
    if (!decode_tile(p.work, p.off, p.E, p.T, BM, nt_r, nt_s, p.part, t)) return;
    const bool shared = t.g == p.E;
    const int wave = threadIdx.x / kWave, lane = lane_id();
    const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;

    int K, n_out;
    const uint16_t* Abase;
    const uint16_t* Bbase;
    int a_ld;
    int64_t a_rows, b_rows;
    if constexpr (MODE == 1) {
        K = p.d;
        n_out = shared ? p.shared_inter : p.inter;
        Abase = static_cast<const uint16_t*>(p.x);
        a_ld = p.d;
        a_rows = p.T;
        b_rows = 2 * static_cast<int64_t>(n_out);
        Bbase = shared ? static_cast<const uint16_t*>(p.ws13)
                       : static_cast<const uint16_t*>(p.w13) + static_cast<int64_t>(t.g) * 2 * p.inter * p.d;
    } else {
        K = shared ? p.shared_inter : p.inter;
        n_out = p.d;
        Abase = shared ? static_cast<const uint16_t*>(p.h_s) : static_cast<const uint16_t*>(p.h_r);
        a_ld = K;
        a_rows = shared ? p.T : p.T * p.k;
        b_rows = p.d;
        Bbase = shared ? static_cast<const uint16_t*>(p.ws2)
                       : static_cast<const uint16_t*>(p.w2) + static_cast<int64_t>(t.g) * p.d * p.inter;
    }
    const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(Abase), 0, static_cast<int>(a_rows * a_ld * 2), kBufferFlags);
    const __amdgpu_buffer_rsrc_t rsB = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(Bbase), 0, static_cast<int>(b_rows * K * 2), kBufferFlags);

    // Lane `lane` of this wave's q-th instruction fills LDS row R = (wave * I + q) * RPI + lane / CPR,
    // slot lane % CPR, with the row's chunk slot ^ swizzle(R).
    const int lrow = lane / CPR, lslot = lane % CPR;
    int aoff[IA], boff[IB];  // element offset of the row start
    int achk[IA], bchk[IB];  // k offset of the chunk this lane moves (after the swizzle)
#pragma unroll
    for (int q = 0; q < IA; ++q) {
        const int R = (wave * IA + q) * RPI + lrow;
        const int rr = R < t.rows ? R : 0;
        int src;
        if (MODE == 1 && !shared) src = p.perm_token[t.row0 + rr];
        else src = static_cast<int>(t.row0 + rr);
        aoff[q] = src * a_ld;
        achk[q] = (lslot ^ ((R / C::SWZ_DIV) % CPR)) * 8;
    }
#pragma unroll
    for (int q = 0; q < IB; ++q) {
        const int R = (wave * IB + q) * RPI + lrow;
        int bi;
        if constexpr (MODE == 1) {
            int cc = t.nt * TC + (R % (BNB / 2));
            if (cc >= n_out) cc = 0;
            bi = R < BNB / 2 ? cc : n_out + cc;
        } else {
            int cc = t.nt * TC + R;
            if (cc >= n_out) cc = 0;
            bi = cc;
        }
        boff[q] = bi * K;
        bchk[q] = (lslot ^ ((R / C::SWZ_DIV) % CPR)) * 8;
    }
    // a chunk past K (K % 8 == 0) gets an offset beyond the record count: the DMA writes zeros
    auto issue = [&](int stage, int k0) {
        uint8_t* base = lds[stage];
#pragma unroll
        for (int q = 0; q < IA; ++q) {
            const int k = k0 + achk[q];
            const int vo = k < K ? (aoff[q] + k) * 2 : kOutOfRange;
            auto* dst = (__attribute__((address_space(3))) void*)(base + (wave * IA + q) * 1024);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rsA, dst, 16, vo, 0, 0, 0);
        }
#pragma unroll
        for (int q = 0; q < IB; ++q) {
            const int k = k0 + bchk[q];
            const int vo = k < K ? (boff[q] + k) * 2 : kOutOfRange;
            auto* dst = (__attribute__((address_space(3))) void*)(base + A_BYTES + (wave * IB + q) * 1024);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rsB, dst, 16, vo, 0, 0, 0);
        }
    };
    int bsub[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        if constexpr (MODE == 1)
            bsub[j] = (j < TN / 2) ? (wn * (TN / 2) + j) * 32 : BNB / 2 + (wn * (TN / 2) + j - TN / 2) * 32;
        else
            bsub[j] = (wn * TN + j) * 32;
    }
    f32x16_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x16_t{};
    const int half = lane >> 5, l32 = lane & 31;
    auto compute = [&](int stage) {
        const uint8_t* base = lds[stage];
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            const int c = ks * 2 + half;
            bf16x8_t af[TM], bfr[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int R = (wm * TM + i) * 32 + l32;
                af[i] = *reinterpret_cast<const bf16x8_t*>(base + R * (BK * 2) + dma_slot<C>(R, c) * 16);
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int R = bsub[j] + l32;
                bfr[j] = *reinterpret_cast<const bf16x8_t*>(base + A_BYTES + R * (BK * 2) + dma_slot<C>(R, c) * 16);
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }
    };

    // K loop: ST-stage ring. Before reading stage kt, this wave waits until at
    // most (ST - 2) newer stages of its own loads are in flight and its LDS
    // reads are done, then a barrier makes every wave's loads visible and
    // frees the stage that the next loads overwrite.
    static_assert(ST == 3, "the loop below is written for three stages");
    constexpr int PER_STAGE = IA + IB;
    const int nk = static_cast<int>(ceil_div(K, BK));
    issue(0, 0);
    issue(1, BK);
    int kt = 0;
    for (; kt + 3 <= nk; kt += 3) {
        wait_vm_lgkm0<PER_STAGE>();
        __builtin_amdgcn_s_barrier();
        issue(2, (kt + 2) * BK);
        compute(0);
        wait_vm_lgkm0<PER_STAGE>();
        __builtin_amdgcn_s_barrier();
        issue(0, (kt + 3) * BK);
        compute(1);
        wait_vm_lgkm0<PER_STAGE>();
        __builtin_amdgcn_s_barrier();
        issue(1, (kt + 4) * BK);
        compute(2);
    }
    if (kt < nk) {
        wait_vm_lgkm0<PER_STAGE>();
        __builtin_amdgcn_s_barrier();
        issue(2, (kt + 2) * BK);
        compute(0);
    }
    if (kt + 1 < nk) {
        wait_vm_lgkm0<PER_STAGE>();
        __builtin_amdgcn_s_barrier();
        compute(1);
    }
    wait_vm_lgkm0<0>();  // drain the ring: the epilogue reuses its LDS
    __builtin_amdgcn_s_barrier();

    // Epilogue through LDS: each wave writes its bf16 results (GEMM1: the
    // SwiGLU output) into a [BM][TC + 8] tile, then every thread stores whole
    // 16-byte row chunks. Element v of a 32x32 MFMA tile sits at row
    // 8*(v/4) + 4*half + v%4, column l32.
    constexpr int OP = TC + 8;  // row pitch (bf16) of the output tile
    static_assert(BM * OP * 2 <= ST * (A_BYTES + B_BYTES), "output tile must fit the ring");
    uint16_t* otile = reinterpret_cast<uint16_t*>(&lds[0][0]);
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int r = (wm * TM + i) * 32 + 8 * (v >> 2) + 4 * half + (v & 3);
            if constexpr (MODE == 1) {
#pragma unroll
                for (int j = 0; j < TN / 2; ++j) {
                    const int c = (wn * (TN / 2) + j) * 32 + l32;
                    otile[r * OP + c] = f32_to_bf16(silu(acc[i][j][v]) * acc[i][j + TN / 2][v]);
                }
            } else {
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    const int c = (wn * TN + j) * 32 + l32;
                    otile[r * OP + c] = f32_to_bf16(acc[i][j][v]);
                }
            }
        }
    }
    __syncthreads();
    uint16_t* O;
    if constexpr (MODE == 1) O = shared ? static_cast<uint16_t*>(p.h_s) : static_cast<uint16_t*>(p.h_r);
    else O = shared ? static_cast<uint16_t*>(p.y_s) : static_cast<uint16_t*>(p.y_r);
    constexpr int CH = TC / 8;  // 16-byte chunks per output row
    const int col0 = t.nt * TC;
    for (int q = threadIdx.x; q < BM * CH; q += C::THREADS) {
        const int r = q / CH, ch = q % CH;
        const int c = col0 + ch * 8;
        if (r < t.rows && c < n_out)  // n_out % 8 == 0: a chunk is all in or all out
            *reinterpret_cast<uint4*>(O + (t.row0 + r) * n_out + c) =
                *reinterpret_cast<const uint4*>(otile + r * OP + ch * 8);
    }
}

// ============================================================== bf16 MFMA path, packed weights
//
// Packed weights: a matrix W[N][K] (N output rows, K contraction) is stored as
// 16-byte fragments P[2 ceil(N/32)][ceil(K/32)][64][8] with
//   P[h][c][l][e] = W[16 h + l % 16][32 c + 8 (l / 16) + e]   (zero outside W),
// which is exactly the A operand of v_mfma_f32_16x16x32_bf16 for output
// rows 16 h .. 16 h + 15 and contraction slice 32 c .. 32 c + 31: one wave
// loads it with one fully coalesced 1 KB buffer load, straight into VGPRs.
// (N is padded to a multiple of 32 so that a matrix holds the same number of
// 16-row groups in every packed form.) GEMM1 packs the gate and up rows
// interleaved by 16-row groups in blocks of 32 output columns (groups 4q ..
// 4q + 3 = gate rows 32q.., up rows 32q.., gate rows 32q + 16.., up rows
// 32q + 16..), so one wave holds gate and up outputs of the same (row,
// column) in the same lane.
//
// The 16x16x32 instruction rather than 32x32x16: both run at the same
// nominal rate and the tile below feeds them the same operand bytes, but with
// random bf16 operands and every SIMD busy the chip holds ~12 % more 16x16x32
// flops under its power limit (1.98 vs 1.76 PFLOP/s sustained from registers).
//
// Tiles: 128 rows x 4 waves; each wave owns all 128 rows and 64 B-rows (four
// 16-row groups: 8 x 4 MFMA tiles of 16 x 16). The weights never pass through
// LDS and no two waves read the same weight bytes; only the token rows (x
// gathered through perm_token for GEMM1, H for GEMM2) are staged HBM -> LDS by
// buffer_load ... lds through a three-stage ring of K = 64 slices. The
// weight loads of the next slice and the token-row DMA of the slice after
// are spread between the MFMAs of the current one.
//   GEMM1: 128 H columns per tile (32 per wave), SwiGLU in registers.
//   GEMM2: 256 output columns per tile (64 per wave).
constexpr int PK_BM = 128, PK_BK = 64, PK_WAVES = 4, PK_THREADS = PK_WAVES * 64, PK_ST = 3;
constexpr int PK_IA = PK_BM * PK_BK * 2 / 1024 / PK_WAVES;  // A DMA instructions per wave per stage
// Modes: 1 GEMM1 (+ SwiGLU), 2 GEMM2, and for the backward 3 GEMM1 with the
// raw gate and up outputs, 4 dH = dout W2 (rows gathered, scaled by the combine
// weight) with the SwiGLU backward in the epilogue, 5 dX = [dA dB] W13, and 6
// GEMM1 writing both H and the gate and up outputs (a forward that keeps them
// for the backward); 7 the shared experts' GEMM2 whose epilogue is the
// combine (run after the routed GEMM2 has written every routed row). Modes 1, 3 and 6 pair gate and up groups (32 H columns
// per wave); 2, 4 and 5 give each wave two consecutive 32-column groups.
constexpr int pk_family(int mode) { return (mode == 1 || mode == 3 || mode == 6) ? 1 : 2; }
// Row tiles per super-row of the work order (row tiles that take one weight
// slice back to back), chosen by same-box A/B at 16384 x 4096 with 160 + 2
// experts: 4 for the down products of the forward (modes 2, 7; 8 -> 4 took
// the routed launch from 1.29 to 1.27 ms), 16 for the rest (gate/up: the
// merged launch 2.83 -> 2.79 ms; the backward's dX 1.56 -> 1.53 ms, dH
// unchanged; 4 there made the backward 0.9 % slower).
constexpr int pk_group_m(int mode) { return (mode == 2 || mode == 7) ? 4 : 16; }
constexpr int pk_tile_cols(int mode) { return pk_family(mode) == 1 ? PK_WAVES * 32 : PK_WAVES * 64; }
constexpr int pk_out_cols(int mode) {
    return (mode == 3 || mode == 6) ? 2 * pk_tile_cols(mode) : pk_tile_cols(mode);
}
constexpr int pk_epi_bytes(int mode) {
    return mode == 4 ? 32 * (3 * pk_tile_cols(mode) + 8) * 2 : PK_BM * (pk_out_cols(mode) + 8) * 2;
}
constexpr int pk_lds_bytes(int mode) {
    return PK_ST * PK_BM * PK_BK * 2 > pk_epi_bytes(mode) ? PK_ST * PK_BM * PK_BK * 2 : pk_epi_bytes(mode);
}

// Elements of one packed matrix with n rows (n_groups = ceil(n / 32) pairs of 16-row groups) and
// contraction k.
__host__ __device__ inline int64_t packed_elems(int64_t n_groups, int k) {
    return n_groups * ((k + 31) / 32) * 1024;
}


template <int MODE>
__global__ void __launch_bounds__(PK_THREADS) __attribute__((amdgpu_waves_per_eu(2, 2)))
gemm_bf16_pk_kernel(GemmArgs p) {
    constexpr int BM = PK_BM, BK = PK_BK, IA = PK_IA;
    constexpr int A_BYTES = BM * BK * 2;
    constexpr int TC = pk_tile_cols(MODE);
    __shared__ __attribute__((aligned(1024))) uint8_t lds[pk_lds_bytes(MODE)];
    constexpr int FAM = pk_family(MODE);
    const int nt_r = static_cast<int>(ceil_div((FAM == 1 || MODE == 4) ? p.inter : p.d, TC));
    const int nt_s = (FAM == 1 || MODE == 4) ? static_cast<int>(ceil_div(p.shared_inter, TC)) : nt_r;
    Tile t;
    if (!decode_tile(p.work, p.off, p.E, p.T, BM, nt_r, nt_s, p.part, t, pk_group_m(MODE))) return;
    const bool shared = t.g == p.E;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = lane_id();

    int K, n_out;
    const uint16_t* Abase;
    int64_t a_rows;
    const uint16_t* Bw;  // this wave's first packed group
    int b_groups;        // packed groups of this wave that hold weights (0..2)
    if constexpr (FAM == 1) {
        K = p.d;
        n_out = shared ? p.shared_inter : p.inter;
        Abase = static_cast<const uint16_t*>(p.x);
        a_rows = p.T;
        const int ng = 2 * static_cast<int>(ceil_div(n_out, 32));  // gate + up groups
        const uint16_t* W = shared ? static_cast<const uint16_t*>(p.ws13)
                                   : static_cast<const uint16_t*>(p.w13) + t.g * packed_elems(ng, K);
        const int q = t.nt * PK_WAVES + wave;  // output group of this wave
        b_groups = 2 * q < ng ? 2 : 0;
        Bw = W + packed_elems(b_groups ? 2 * q : 0, K);
    } else {
        const uint16_t* Wr;
        const uint16_t* Ws;
        if constexpr (MODE == 4) {  // dH = dout W2: rows of dout, contraction over d
            K = p.d;
            n_out = shared ? p.shared_inter : p.inter;
            Abase = static_cast<const uint16_t*>(p.dout);
            a_rows = p.T;
            Wr = static_cast<const uint16_t*>(p.w2t);
            Ws = static_cast<const uint16_t*>(p.ws2t);
        } else if constexpr (MODE == 5) {  // dX = [dA dB] W13: contraction over 2 inter
            K = 2 * (shared ? p.shared_inter : p.inter);
            n_out = p.d;
            Abase = shared ? static_cast<const uint16_t*>(p.dab_s) : static_cast<const uint16_t*>(p.dab_r);
            a_rows = shared ? p.T : p.T * p.k;
            Wr = static_cast<const uint16_t*>(p.w13t);
            Ws = static_cast<const uint16_t*>(p.ws13t);
        } else {
            K = shared ? p.shared_inter : p.inter;
            n_out = p.d;
            Abase = shared ? static_cast<const uint16_t*>(p.h_s) : static_cast<const uint16_t*>(p.h_r);
            a_rows = shared ? p.T : p.T * p.k;
            Wr = static_cast<const uint16_t*>(p.w2);
            Ws = static_cast<const uint16_t*>(p.ws2);
        }
        const int ng = static_cast<int>(ceil_div(n_out, 32));
        const uint16_t* W = shared ? Ws : Wr + t.g * packed_elems(ng, K);
        const int g0 = t.nt * (2 * PK_WAVES) + 2 * wave;
        b_groups = ng - g0 >= 2 ? 2 : (ng - g0 > 0 ? ng - g0 : 0);
        Bw = W + packed_elems(b_groups ? g0 : 0, K);
    }
    K = uniform_int(K);
    const int kc_n = (K + 31) / 32;  // packed 32-wide contraction slices per 16-row group
    const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(uniform_ptr(Abase)), 0, uniform_int(static_cast<int>(a_rows * K * 2)), kBufferFlags);
    const __amdgpu_buffer_rsrc_t rsB = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(uniform_ptr(Bw)), 0, uniform_int(2 * b_groups * kc_n * 1024), kBufferFlags);

    // A DMA: instruction q of this wave fills LDS rows (wave * IA + q) * 8 .. + 7 of the stage;
    // lane moves the 16-byte chunk (lane % 8) ^ swizzle(row) of its row into slot lane % 8.
    // aoff: element offset of the row start; rows past the tile get 2^30, whose
    // byte offset (>= 2^31) is out of range: zero fill without memory traffic.
    uint32_t aoff[IA];
    int achk[IA];
#pragma unroll
    for (int q = 0; q < IA; ++q) {
        const int R = (wave * IA + q) * 8 + lane / 8;
        const int rr = R < t.rows ? R : 0;
        int src;
        if ((FAM == 1 || MODE == 4) && !shared) src = p.perm_token[t.row0 + rr];
        else src = static_cast<int>(t.row0 + rr);
        aoff[q] = R < t.rows ? static_cast<uint32_t>(src) * static_cast<uint32_t>(K) : (1u << 30);
        achk[q] = ((lane % 8) ^ ((R / 2) % 8)) * 8;
    }
    // One A DMA instruction (rows (wave * IA + q) * 8 ..) of stage s into ring slot `slot`.
    auto issue_aq = [&](int slot, int s, int q) {
        const int k = s * BK + achk[q];
        const int vo = static_cast<int>(((aoff[q] + static_cast<uint32_t>(k)) * 2u) |
                                        (k < K ? 0u : static_cast<uint32_t>(kOutOfRange)));
        auto* dst = (__attribute__((address_space(3))) void*)(lds + slot * A_BYTES + (wave * IA + q) * 1024);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsA, dst, 16, vo, 0, 0, 0);
    };
    // Weight fragments of stage s: b[j][h] is 16-row group h of K slice 32 (2 s + j).
    // Quarter q of a stage loads groups 2 (q % 2) and 2 (q % 2) + 1 of slice q / 2.
    auto issue_bq = [&](i32x4_t (&b)[2][4], int s, int q) {
        const int j = q >> 1;
        const int kc = s * 2 + j;
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int h = 2 * (q & 1) + u;
            const int vo = (((h * kc_n + kc) * 64 + lane) * 16) | (kc < kc_n ? 0 : kOutOfRange);
            b[j][h] = __builtin_amdgcn_raw_buffer_load_b128(rsB, vo, 0, 0);
        }
    };
    // acc[i][h]: token rows 16 i .. 16 i + 15 x weight rows 16 h .. 16 h + 15 of this wave
    f32x4_t acc[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int h = 0; h < 4; ++h) acc[i][h] = f32x4_t{};
    const int quad = lane >> 4, l16 = lane & 15;

    // Stage s from ring slot `slot` with weight registers bc, while the loads of
    // the next stages go out between the MFMAs. A stage (K = 64) runs in four
    // quarters q: K slice j = q / 2 against token tiles 2 u + q % 2 (u < MT);
    // quarter q issues the weight loads of stage s + 1 for
    // quarter q (2 loads) and the A DMA q of stage s + 2, reads the token
    // fragments of quarter q + 1 and runs 4 MT MFMAs. A wave issues in order,
    // so spreading the memory instructions over the MFMAs keeps the matrix
    // pipe fed while the address unit drains them.
    static_assert(IA == 4, "one A DMA per quarter stage");
    // MT: 32-row sub-tiles that take part (1-4: a short last tile of an
    // expert skips the MFMAs and fragment reads of its empty sub-tiles).
    auto stage_run = [&](auto mt_c, int slot, int s, const i32x4_t (&bc)[2][4], i32x4_t (&bn)[2][4]) {
        constexpr int MT = decltype(mt_c)::value;
        const uint8_t* base = lds + slot * A_BYTES;
        const int nslot = slot == 0 ? 2 : slot - 1;  // (slot + 2) % 3
        bf16x8_t af[2][4];
        // token fragment of tile 2 u + q % 2, K slice q / 2: row 16 i + l % 16, k 32 j + 8 (l / 16) ..
        auto rd = [&](int q, bf16x8_t (&a)[4]) {
            const int c = (q >> 1) * 4 + quad;
#pragma unroll
            for (int u = 0; u < MT; ++u) {
                const int R = (2 * u + (q & 1)) * 16 + l16;
                a[u] = *reinterpret_cast<const bf16x8_t*>(base + R * (BK * 2) + ((c ^ ((R / 2) % 8)) * 16));
            }
        };
        rd(0, af[0]);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            __builtin_amdgcn_sched_barrier(0);
            issue_bq(bn, s + 1, q);
            issue_aq(nslot, s + 2, q);
            if (q < 3) rd(q + 1, af[(q + 1) & 1]);
#pragma unroll
            for (int u = 0; u < MT; ++u)
#pragma unroll
                for (int h = 0; h < 4; ++h)  // transposed tile: rows = weight rows, columns = tokens
                    acc[2 * u + (q & 1)][h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(bf16x8_t, bc[q >> 1][h]), af[q & 1][u], acc[2 * u + (q & 1)][h], 0, 0, 0);
            // order: one VMEM after each of the first MFMAs, then one LDS read after each of
            // the following MFMAs, then the rest of the MFMAs
            constexpr int NM = 4 * MT;
#pragma unroll
            for (int v = 0; v < 3; ++v) {
                if (v < NM) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
            }
#pragma unroll
            for (int v = 0; v < MT; ++v) {
                if (3 + v < NM) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
            if (NM > 3 + MT) __builtin_amdgcn_sched_group_barrier(0x008, NM - 3 - MT, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    };

    // Loads retire in order. Issue order: A(0), then per quarter q of stage
    // s - 1: B(s)[q] (2), A(s + 1)[q] (1). Before stage s reads LDS slot s % 3,
    // at most the 12 loads issued after A(s)'s last DMA may still fly (B(s)
    // and A(s + 1)); the compiler waits for B(s)'s registers by itself. The
    // barrier makes every wave's DMA of A(s) visible and frees the slot that
    // A(s + 2) overwrites. Unrolled by two so the B register sets stay static.
    // Past the end of K the loads go out of range and return zeros, so every
    // stage issues the same count and the waits stay exact.
    const int nk = static_cast<int>(ceil_div(K, BK));
    auto kloop = [&](auto mt_c) {
        i32x4_t b0[2][4], b1[2][4];
#pragma unroll
        for (int q = 0; q < IA; ++q) issue_aq(0, 0, q);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            issue_bq(b0, 0, q);
            issue_aq(1, 1, q);
        }
        int s = 0, slot = 0;
        for (; s + 2 <= nk; s += 2) {
            wait_vm_lgkm0<12>();
            __builtin_amdgcn_s_barrier();
            stage_run(mt_c, slot, s, b0, b1);
            slot = slot == 2 ? 0 : slot + 1;
            wait_vm_lgkm0<12>();
            __builtin_amdgcn_s_barrier();
            stage_run(mt_c, slot, s + 1, b1, b0);
            slot = slot == 2 ? 0 : slot + 1;
        }
        if (s < nk) {
            wait_vm_lgkm0<12>();
            __builtin_amdgcn_s_barrier();
            stage_run(mt_c, slot, s, b0, b1);
        }
    };
    const int trows = uniform_int(t.rows);
    if (trows > 96) kloop(std::integral_constant<int, 4>{});
    else if (trows > 64) kloop(std::integral_constant<int, 3>{});
    else if (trows > 32) kloop(std::integral_constant<int, 2>{});
    else kloop(std::integral_constant<int, 1>{});
    wait_vm_lgkm0<0>();  // drain: the epilogue reuses the ring
    __builtin_amdgcn_s_barrier();

    // Epilogue through LDS: [BM][TC + 8] bf16 tile, then 16-byte row chunks.
    // The accumulators hold transposed 16x16 tiles: element e of lane l of
    // acc[i][h] is output column 16 h + 4 (l / 16) + e of the wave's columns,
    // token row 16 i + l % 16, so each lane writes four adjacent columns as
    // one 8-byte store.
    auto pack4 = [](float a, float b, float c, float d) {
        return make_uint2(static_cast<uint32_t>(f32_to_bf16(a)) | (static_cast<uint32_t>(f32_to_bf16(b)) << 16),
                          static_cast<uint32_t>(f32_to_bf16(c)) | (static_cast<uint32_t>(f32_to_bf16(d)) << 16));
    };
    if constexpr (MODE == 4) {
        // dH = w * (dout W2) and the SwiGLU backward with the saved gate (a)
        // and up (b) pre-activations: dA = dH b silu'(a), dB = dH silu(a),
        // plus w H = w silu(a) b for the dW2 product (routed rows). In four
        // passes of 32 rows: the rows' a | b slices come into LDS as whole
        // rows, each lane turns its four adjacent columns into dA | dB | w H
        // in place, and the three slices go out as whole rows.
        const uint16_t* AB = static_cast<const uint16_t*>(shared ? p.ab_s : p.ab_r);
        uint16_t* dAB = static_cast<uint16_t*>(shared ? p.dab_s : p.dab_r);
        uint16_t* WH = shared ? nullptr : static_cast<uint16_t*>(p.wh_r);
        const int64_t ld = 2 * static_cast<int64_t>(n_out);
        constexpr int EP = 3 * TC + 8;  // LDS row: a | b | w H (pitch = 4 mod 64 dwords)
        uint16_t* el = reinterpret_cast<uint16_t*>(lds);
        const int col0 = t.nt * TC;
        const int ncols = n_out - col0 < TC ? n_out - col0 : TC;  // multiple of 16
        // 16-byte chunks of a pass's a | b rows held by each thread; the next
        // pass's chunks are loaded while the current one is processed
        constexpr int LCH = 32 * (2 * TC / 8) / PK_THREADS;
        auto load_pass = [&](int i, uint4 (&v)[LCH]) {
            const int rows_here = t.rows - i * 32;
            const int64_t rbase = t.row0 + i * 32;
#pragma unroll
            for (int u = 0; u < LCH; ++u) {
                const int q = threadIdx.x + u * PK_THREADS;
                const int r = q / (2 * TC / 8), ch = q % (2 * TC / 8);
                const int part = ch / (TC / 8), c = (ch % (TC / 8)) * 8;
                v[u] = (r < rows_here && c < ncols)
                           ? *reinterpret_cast<const uint4*>(AB + (rbase + r) * ld + part * n_out + col0 + c)
                           : make_uint4(0, 0, 0, 0);
            }
        };
        uint4 cur[LCH], nxt[LCH];
        load_pass(0, cur);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int rows_here = t.rows - i * 32;
            if (rows_here <= 0) break;  // uniform
            const int64_t rbase = t.row0 + i * 32;
#pragma unroll
            for (int u = 0; u < LCH; ++u) {
                const int q = threadIdx.x + u * PK_THREADS;
                const int r = q / (2 * TC / 8), ch = q % (2 * TC / 8);
                *reinterpret_cast<uint4*>(el + r * EP + (ch / (TC / 8)) * TC + (ch % (TC / 8)) * 8) = cur[u];
            }
            if (i + 1 < 4) load_pass(i + 1, nxt);
            __syncthreads();
#pragma unroll
            for (int tt = 0; tt < 2; ++tt) {
                const int lr = 16 * tt + l16;  // row of the pass
                const float w = shared ? 1.0f : (lr < rows_here ? p.wrow[rbase + lr] : 0.0f);
                uint16_t* er = el + lr * EP;
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    const int col = wave * 64 + 16 * h + 4 * quad;
                    const uint2 av = *reinterpret_cast<const uint2*>(er + col);
                    const uint2 bv = *reinterpret_cast<const uint2*>(er + TC + col);
                    const float a[4] = {__uint_as_float(av.x << 16), __uint_as_float(av.x & 0xffff0000u),
                                        __uint_as_float(av.y << 16), __uint_as_float(av.y & 0xffff0000u)};
                    const float bb[4] = {__uint_as_float(bv.x << 16), __uint_as_float(bv.x & 0xffff0000u),
                                         __uint_as_float(bv.y << 16), __uint_as_float(bv.y & 0xffff0000u)};
                    float da[4], db[4], wh[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float dh = w * acc[2 * i + tt][h][e];
                        const float sg = 1.0f / (1.0f + __expf(-a[e]));
                        const float sa = a[e] * sg;  // silu(a)
                        da[e] = dh * bb[e] * (sg + sa * (1.0f - sg));
                        db[e] = dh * sa;
                        wh[e] = w * sa * bb[e];
                    }
                    *reinterpret_cast<uint2*>(er + col) = pack4(da[0], da[1], da[2], da[3]);
                    *reinterpret_cast<uint2*>(er + TC + col) = pack4(db[0], db[1], db[2], db[3]);
                    *reinterpret_cast<uint2*>(er + 2 * TC + col) = pack4(wh[0], wh[1], wh[2], wh[3]);
                }
            }
            __syncthreads();
            const int nparts = WH != nullptr ? 3 : 2;
            for (int q = threadIdx.x; q < 32 * (3 * TC / 8); q += PK_THREADS) {
                const int r = q / (3 * TC / 8), ch = q % (3 * TC / 8);
                const int part = ch / (TC / 8), c = (ch % (TC / 8)) * 8;
                if (r < rows_here && c < ncols && part < nparts) {
                    const uint4 v = *reinterpret_cast<const uint4*>(el + r * EP + part * TC + c);
                    if (part < 2) *reinterpret_cast<uint4*>(dAB + (rbase + r) * ld + part * n_out + col0 + c) = v;
                    else *reinterpret_cast<uint4*>(WH + (rbase + r) * n_out + col0 + c) = v;
                }
            }
            __syncthreads();
#pragma unroll
            for (int u = 0; u < LCH; ++u) cur[u] = nxt[u];
        }
        return;
    }
    // OK: 1 H = silu(gate) * up, 3 the gate | up pre-activations, 2 / 5 the
    // plain accumulators. Mode 6 writes H, then the pre-activations.
    auto epilogue = [&](auto ok_c) {
        constexpr int OK = decltype(ok_c)::value;
        constexpr int OC = OK == 3 ? 2 * TC : TC;  // tile columns written (3: gate block then up block)
        constexpr int OP = OC + 8;
        uint16_t* otile = reinterpret_cast<uint16_t*>(lds);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int r = i * 16 + l16;
            const int c0 = 4 * quad;
            if constexpr (OK == 1) {  // groups 2 p (gate) and 2 p + 1 (up): H columns 16 p ..
#pragma unroll
                for (int pq = 0; pq < 2; ++pq) {
                    float h[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) h[e] = silu(acc[i][2 * pq][e]) * acc[i][2 * pq + 1][e];
                    *reinterpret_cast<uint2*>(otile + r * OP + wave * 32 + 16 * pq + c0) = pack4(h[0], h[1], h[2], h[3]);
                }
            } else if constexpr (OK == 3) {  // gate block, then up block
#pragma unroll
                for (int h = 0; h < 4; ++h)
                    *reinterpret_cast<uint2*>(otile + r * OP + (h & 1) * TC + wave * 32 + 16 * (h >> 1) + c0) =
                        pack4(acc[i][h][0], acc[i][h][1], acc[i][h][2], acc[i][h][3]);
            } else {
#pragma unroll
                for (int h = 0; h < 4; ++h)
                    *reinterpret_cast<uint2*>(otile + r * OP + wave * 64 + 16 * h + c0) =
                        pack4(acc[i][h][0], acc[i][h][1], acc[i][h][2], acc[i][h][3]);
            }
        }
        __syncthreads();
        if constexpr (OK == 7) {
            // out_j = sum_s w_js Y_r[inv(j, s)] + Ys_j for the tile's tokens and
            // columns, in the combine kernel's order (float32, slots in order,
            // then the bf16 shared row from the tile): two 8-column items per
            // thread at a time, their row indices, then four row loads each
            const int kk = p.k;
            const int32_t* inv = p.inv;
            const float* tw = p.topk_w;
            const uint16_t* yr = static_cast<const uint16_t*>(p.y_r);
            uint16_t* out = static_cast<uint16_t*>(p.out);
            const int64_t dd = p.d;
            constexpr int CH = OC / 8;
            const int col0 = t.nt * TC;
            for (int q0 = threadIdx.x; q0 < BM * CH; q0 += 2 * PK_THREADS) {
                int64_t j[2];
                int c[2], r[2];
                bool ok[2];
                float v[2][8];
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    const int q = q0 + u * PK_THREADS;
                    r[u] = q / CH;
                    c[u] = col0 + (q % CH) * 8;
                    j[u] = t.row0 + r[u];
                    ok[u] = q < BM * CH && r[u] < t.rows && c[u] < n_out;  // d % 8 == 0
#pragma unroll
                    for (int e = 0; e < 8; ++e) v[u][e] = 0.0f;
                }
                for (int s0 = 0; s0 < kk; s0 += 4) {
                    int row[2][4];
                    float wt[2][4];
#pragma unroll
                    for (int u = 0; u < 2; ++u)
#pragma unroll
                        for (int sv = 0; sv < 4; ++sv) {
                            const bool in = ok[u] && s0 + sv < kk;
                            row[u][sv] = in ? inv[j[u] * kk + s0 + sv] : -1;
                            wt[u][sv] = in ? tw[j[u] * kk + s0 + sv] : 0.0f;
                        }
                    uint4 y[2][4];
#pragma unroll
                    for (int u = 0; u < 2; ++u)
#pragma unroll
                        for (int sv = 0; sv < 4; ++sv)
                            y[u][sv] = row[u][sv] >= 0
                                           ? *reinterpret_cast<const uint4*>(yr + static_cast<int64_t>(row[u][sv]) * dd + c[u])
                                           : make_uint4(0, 0, 0, 0);
#pragma unroll
                    for (int u = 0; u < 2; ++u)
#pragma unroll
                        for (int sv = 0; sv < 4; ++sv) {
                            if (s0 + sv >= kk) continue;
                            const uint32_t w4[4] = {y[u][sv].x, y[u][sv].y, y[u][sv].z, y[u][sv].w};
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                v[u][2 * e] = fmaf(wt[u][sv], __uint_as_float(w4[e] << 16), v[u][2 * e]);
                                v[u][2 * e + 1] = fmaf(wt[u][sv], __uint_as_float(w4[e] & 0xffff0000u), v[u][2 * e + 1]);
                            }
                        }
                }
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    if (!ok[u]) continue;
                    const uint4 ys = *reinterpret_cast<const uint4*>(otile + r[u] * OP + (c[u] - col0));
                    const uint32_t w4[4] = {ys.x, ys.y, ys.z, ys.w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        v[u][2 * e] += __uint_as_float(w4[e] << 16);
                        v[u][2 * e + 1] += __uint_as_float(w4[e] & 0xffff0000u);
                    }
                    *reinterpret_cast<uint4*>(out + j[u] * dd + c[u]) =
                        make_uint4(static_cast<uint32_t>(f32_to_bf16(v[u][0])) | (static_cast<uint32_t>(f32_to_bf16(v[u][1])) << 16),
                                   static_cast<uint32_t>(f32_to_bf16(v[u][2])) | (static_cast<uint32_t>(f32_to_bf16(v[u][3])) << 16),
                                   static_cast<uint32_t>(f32_to_bf16(v[u][4])) | (static_cast<uint32_t>(f32_to_bf16(v[u][5])) << 16),
                                   static_cast<uint32_t>(f32_to_bf16(v[u][6])) | (static_cast<uint32_t>(f32_to_bf16(v[u][7])) << 16));
                }
            }
            return;
        }
        uint16_t* O;
        if constexpr (OK == 1) O = shared ? static_cast<uint16_t*>(p.h_s) : static_cast<uint16_t*>(p.h_r);
        else if constexpr (OK == 3) O = shared ? static_cast<uint16_t*>(p.ab_s) : static_cast<uint16_t*>(p.ab_r);
        else if constexpr (OK == 5) O = shared ? static_cast<uint16_t*>(p.dx_s) : static_cast<uint16_t*>(p.dx_r);
        else O = shared ? static_cast<uint16_t*>(p.y_s) : static_cast<uint16_t*>(p.y_r);
        constexpr int CH = OC / 8;
        const int col0 = t.nt * TC;
        for (int q = threadIdx.x; q < BM * CH; q += PK_THREADS) {
            const int r = q / CH, ch = q % CH;
            if constexpr (OK == 3) {  // gate block to columns [0, n_out), up block to [n_out, 2 n_out)
                const int part = (ch * 8) / TC;
                const int c = col0 + ch * 8 - part * TC;
                if (r < t.rows && c < n_out)
                    *reinterpret_cast<uint4*>(O + (t.row0 + r) * (2 * static_cast<int64_t>(n_out)) + part * n_out +
                                              c) = *reinterpret_cast<const uint4*>(otile + r * OP + ch * 8);
            } else {
                const int c = col0 + ch * 8;
                if (r < t.rows && c < n_out)  // n_out % 8 == 0: a chunk is all in or all out
                    *reinterpret_cast<uint4*>(O + (t.row0 + r) * n_out + c) =
                        *reinterpret_cast<const uint4*>(otile + r * OP + ch * 8);
            }
        }
    };
    if constexpr (MODE == 6) {
        epilogue(std::integral_constant<int, 1>{});
        __syncthreads();  // every H row chunk has left the tile
        epilogue(std::integral_constant<int, 3>{});
    } else {
        epilogue(std::integral_constant<int, MODE>{});
    }
}

// Pack `batch` row-major matrices into the fragment order above. interleave:
// the source has 2 * n rows (gate rows then up rows) and 16-row group 4q + 2v
// + h takes rows 32q + 16v.. of half h; otherwise the source has n rows.
// transpose: the source is stored [k][n] (the packed matrix is its
// transpose). One thread per 16-byte fragment; k % 8 == 0.
__global__ void pack_weights_kernel(const uint16_t* __restrict__ src, int batch, int n, int k, int interleave,
                                    int transpose, uint16_t* __restrict__ dst) {
    const int ng = static_cast<int>((interleave ? 4 : 2) * ceil_div(n, 32));  // 16-row groups
    const int kc_n = (k + 31) / 32;
    const int64_t per = static_cast<int64_t>(ng) * kc_n * 64;  // fragments per matrix
    const int64_t total = per * batch;
    const int64_t src_rows = interleave ? 2 * static_cast<int64_t>(n) : n;
    for (int64_t f = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; f < total;
         f += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t b = f / per;
        const int64_t r = f % per;
        const int l = static_cast<int>(r % 64);
        const int c = static_cast<int>((r / 64) % kc_n);
        const int g = static_cast<int>(r / (64 * kc_n));
        int row;
        bool ok;
        if (interleave) {
            const int q = g / 4, v = (g / 2) % 2, h = g % 2;
            const int rr = q * 32 + v * 16 + l % 16;
            ok = rr < n;
            row = h * n + rr;
        } else {
            row = g * 16 + l % 16;
            ok = row < n;
        }
        const int kk = c * 32 + 8 * (l / 16);
        ok = ok && kk < k;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (ok && transpose) {
            uint16_t e8[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) e8[e] = src[(b * k + kk + e) * static_cast<int64_t>(n) + row];
            v = make_uint4(e8[0] | (static_cast<uint32_t>(e8[1]) << 16), e8[2] | (static_cast<uint32_t>(e8[3]) << 16),
                           e8[4] | (static_cast<uint32_t>(e8[5]) << 16), e8[6] | (static_cast<uint32_t>(e8[7]) << 16));
        } else if (ok) {
            v = *reinterpret_cast<const uint4*>(src + (b * src_rows + row) * k + kk);
        }
        *reinterpret_cast<uint4*>(dst + f * 8) = v;
    }
}

// ============================================================== f32 FMA path

template <int MODE>
__global__ void __launch_bounds__(kThreads)
gemm_f32_kernel(GemmArgs p) {
    __shared__ float As[FBK][FBM + 4];
    __shared__ float Bs[FBK][FBNB + 4];
    __shared__ float Cs[FBM][FBNB + 1];
    const int nt_r = MODE == 1 ? static_cast<int>(ceil_div(p.inter, 32)) : static_cast<int>(ceil_div(p.d, 64));
    const int nt_s = MODE == 1 ? static_cast<int>(ceil_div(p.shared_inter, 32)) : nt_r;
    Tile t;
    if (!decode_tile(p.work, p.off, p.E, p.T, FBM, nt_r, nt_s, p.part, t)) return;
    const bool shared = t.g == p.E;
    const int tid = threadIdx.x;
    int K, n_out;
    const float* Abase;
    const float* Bbase;
    int64_t a_ld;
    if constexpr (MODE == 1) {
        K = p.d;
        n_out = shared ? p.shared_inter : p.inter;
        Abase = static_cast<const float*>(p.x);
        a_ld = p.d;
        Bbase = shared ? static_cast<const float*>(p.ws13)
                       : static_cast<const float*>(p.w13) + static_cast<int64_t>(t.g) * 2 * p.inter * p.d;
    } else {
        K = shared ? p.shared_inter : p.inter;
        n_out = p.d;
        Abase = shared ? static_cast<const float*>(p.h_s) : static_cast<const float*>(p.h_r);
        a_ld = K;
        Bbase = shared ? static_cast<const float*>(p.ws2)
                       : static_cast<const float*>(p.w2) + static_cast<int64_t>(t.g) * p.d * p.inter;
    }
    // loaders: 64 rows x 16 k per tile, 4 elements per thread
    const int lr = tid >> 2;         // row 0..63
    const int lk = (tid & 3) * 4;    // k 0,4,8,12
    const int rr = lr < t.rows ? lr : 0;
    int64_t asrc;
    if (MODE == 1 && !shared) asrc = p.perm_token[t.row0 + rr];
    else asrc = t.row0 + rr;
    const float* arow = Abase + asrc * a_ld;
    int64_t bidx;
    if constexpr (MODE == 1) {
        int c = t.nt * 32 + (lr & 31);
        if (c >= n_out) c = 0;
        bidx = lr < 32 ? c : n_out + c;
    } else {
        int c = t.nt * 64 + lr;
        if (c >= n_out) c = 0;
        bidx = c;
    }
    const float* brow = Bbase + bidx * K;
    const int ty = tid >> 4, tx = tid & 15;
    float acc[4][4] = {};
    for (int k0 = 0; k0 < K; k0 += FBK) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int kk = k0 + lk + q;
            As[lk + q][lr] = kk < K ? arow[kk] : 0.0f;
            Bs[lk + q][lr] = kk < K ? brow[kk] : 0.0f;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < FBK; ++kk) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) Cs[ty * 4 + i][tx * 4 + j] = acc[i][j];
    __syncthreads();
    if constexpr (MODE == 1) {
        float* H = shared ? static_cast<float*>(p.h_s) : static_cast<float*>(p.h_r);
        for (int q = tid; q < FBM * 32; q += kThreads) {
            const int r = q / 32, c = q % 32;
            const int col = t.nt * 32 + c;
            if (r < t.rows && col < n_out)
                H[(t.row0 + r) * n_out + col] = silu(Cs[r][c]) * Cs[r][32 + c];
        }
    } else {
        float* Y = shared ? static_cast<float*>(p.y_s) : static_cast<float*>(p.y_r);
        for (int q = tid; q < FBM * FBNB; q += kThreads) {
            const int r = q / FBNB, c = q % FBNB;
            const int col = t.nt * 64 + c;
            if (r < t.rows && col < n_out) Y[(t.row0 + r) * n_out + col] = Cs[r][c];
        }
    }
}

// ============================================================== f32 FMA backward

// Backward of fp32 layers and of bf16 layers whose weights are row-major: the
// same contractions as the forward's f32 tiles (64 x 64 outputs per block, 4 x 4
// per thread, K steps of 16 through LDS), with float32 intermediates. Steps:
//   GB_AB   [A | B] = X W13^T          rows: routed rows (x gathered) / tokens
//   GB_DH   dH = w dout W2, then the SwiGLU backward: dA, dB and w H
//   GB_DX   dX = [dA dB] W13
//   GB_DW2  dW2[n][c]  = sum over the group's rows of dout[tok][n] (w H)[c]
//   GB_DW13 dW13[m][n] = sum over the group's rows of [dA dB][m] x[tok][n]
// Row steps take their tiles from the work table (decode_tile, both parts);
// weight steps run one block per (output tile, group), group E the shared
// experts. An expert without rows gets a zero gradient.
enum { GB_AB = 0, GB_DH = 1, GB_DX = 2, GB_DW2 = 3, GB_DW13 = 4 };

struct GenBwdArgs {
    int64_t T;
    int d, E, inter, shared_inter;
    const int32_t* off;
    const int32_t* perm_token;
    const int32_t* work;
    const void* x;     // [T][d] layer dtype
    const void* dout;  // [T][d]
    const void* w13;   // [E][2 inter][d]
    const void* w2;    // [E][d][inter]
    const void* ws13;  // [2 shared_inter][d]
    const void* ws2;   // [d][shared_inter]
    float* ab_r;       // [R][2 inter]
    float* ab_s;       // [T][2 shared_inter]
    float* dab_r;
    float* dab_s;
    float* wh_r;       // [R][inter]
    float* wh_s;       // [T][shared_inter]
    float* dx_r;       // [R][d]
    float* dx_s;       // [T][d]
    const float* wrow; // [R]
    void* dw13;        // layer dtype, shapes of w13 ...
    void* dw2;
    void* dws13;
    void* dws2;
};

template <bool BF16>
__device__ __forceinline__ float ldv(const void* p, int64_t i) {
    if constexpr (BF16) return bf16_to_f32(static_cast<const uint16_t*>(p)[i]);
    else return static_cast<const float*>(p)[i];
}

// output column tiles of a row step for a group with n_out inner columns
__host__ __device__ __forceinline__ int gb_row_tiles(int mode, int n_out, int d) {
    return static_cast<int>(ceil_div(mode == GB_AB ? 2 * n_out : mode == GB_DH ? n_out : d, FBNB));
}

template <int MODE, bool BF16>
__global__ void __launch_bounds__(kThreads)
gemm_f32_bwd_kernel(GenBwdArgs p) {
    __shared__ __align__(16) float As[FBK][FBM + 4];
    __shared__ __align__(16) float Bs[FBK][FBNB + 4];
    constexpr bool kRows = MODE <= GB_DX;
    const int tid = threadIdx.x;
    int g, m0, n0, M, N, K, rows = 0;
    int64_t row0;
    if constexpr (kRows) {
        Tile t;
        if (!decode_tile(p.work, p.off, p.E, p.T, FBM, gb_row_tiles(MODE, p.inter, p.d),
                         gb_row_tiles(MODE, p.shared_inter, p.d), 0, t))
            return;
        g = t.g;
        row0 = t.row0;
        rows = t.rows;
        m0 = 0;
        n0 = t.nt * FBNB;
        const int n_out = g == p.E ? p.shared_inter : p.inter;
        M = rows;
        N = MODE == GB_AB ? 2 * n_out : MODE == GB_DH ? n_out : p.d;
        K = MODE == GB_DX ? 2 * n_out : p.d;
    } else {
        g = blockIdx.y;
        const int n_out = g == p.E ? p.shared_inter : p.inter;
        M = MODE == GB_DW2 ? p.d : 2 * n_out;
        N = MODE == GB_DW2 ? n_out : p.d;
        const int tn = static_cast<int>(ceil_div(N, FBNB));
        if (static_cast<int>(blockIdx.x) >= static_cast<int>(ceil_div(M, FBM)) * tn) return;
        m0 = static_cast<int>(blockIdx.x) / tn * FBM;
        n0 = static_cast<int>(blockIdx.x) % tn * FBNB;
        row0 = g == p.E ? 0 : p.off[g];
        K = g == p.E ? static_cast<int>(p.T) : p.off[g + 1] - p.off[g];
    }
    const bool shared = g == p.E;
    const int n_out = shared ? p.shared_inter : p.inter;
    const int ldab = 2 * n_out;
    const void* W13 = shared ? p.ws13
                             : static_cast<const char*>(p.w13) + (BF16 ? 2 : 4) * static_cast<int64_t>(g) * 2 * p.inter * p.d;
    const void* W2 = shared ? p.ws2
                            : static_cast<const char*>(p.w2) + (BF16 ? 2 : 4) * static_cast<int64_t>(g) * p.d * p.inter;
    float* ab = shared ? p.ab_s : p.ab_r;
    float* dab = shared ? p.dab_s : p.dab_r;
    float* wh = shared ? p.wh_s : p.wh_r;
    // token of row r (row space of this group: routed rows in expert order, or tokens)
    auto token = [&](int64_t r) -> int64_t { return shared ? r : p.perm_token[r]; };

    // loader coordinates: "kc" operands are contiguous along K (thread: one row, 4 k),
    // "ic" operands along the output index (thread: one k, 4 indices)
    const int kc_i = tid >> 2, kc_k = (tid & 3) * 4;
    const int ic_k = tid >> 4, ic_i = (tid & 15) * 4;
    // row-step A operand (kc): x / dout gathered by token, or [dA dB] by row
    int64_t a_base = 0;
    const bool a_ok = kc_i < rows;
    if constexpr (kRows) {
        if (a_ok) a_base = MODE == GB_DX ? (row0 + kc_i) * ldab : token(row0 + kc_i) * p.d;
    }
    // GB_AB B operand (kc): row n0 + kc_i of W13
    const bool b_kc_ok = n0 + kc_i < N;
    const int64_t b_kc_base = static_cast<int64_t>(n0 + kc_i) * p.d;

    const int ty = tid >> 4, tx = tid & 15;
    float acc[4][4] = {};
    for (int k0 = 0; k0 < K; k0 += FBK) {
        float a[4], b[4];
        if constexpr (kRows) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int kk = k0 + kc_k + q;
                const bool ok = a_ok && kk < K;
                if constexpr (MODE == GB_DX) a[q] = ok ? dab[a_base + kk] : 0.0f;
                else if constexpr (MODE == GB_AB) a[q] = ok ? ldv<BF16>(p.x, a_base + kk) : 0.0f;
                else a[q] = ok ? ldv<BF16>(p.dout, a_base + kk) : 0.0f;
            }
            if constexpr (MODE == GB_AB) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int kk = k0 + kc_k + q;
                    b[q] = b_kc_ok && kk < K ? ldv<BF16>(W13, b_kc_base + kk) : 0.0f;
                }
            } else {
                // B(j, kk) = W2[kk][j] (dH) or W13[kk][j] (dX): contiguous along j
                const int kk = k0 + ic_k;
                const int ld = MODE == GB_DH ? n_out : p.d;
                const void* Wb = MODE == GB_DH ? W2 : W13;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int j = n0 + ic_i + q;
                    b[q] = kk < K && j < N ? ldv<BF16>(Wb, static_cast<int64_t>(kk) * ld + j) : 0.0f;
                }
            }
        } else {
            // contraction over the group's rows: row k0 + ic_k
            const int kk = k0 + ic_k;
            const bool rok = kk < K;
            const int64_t r = row0 + (rok ? kk : 0);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int i = m0 + ic_i + q, j = n0 + ic_i + q;
                if constexpr (MODE == GB_DW2) {
                    a[q] = rok && i < M ? ldv<BF16>(p.dout, token(r) * p.d + i) : 0.0f;
                    b[q] = rok && j < N ? wh[r * n_out + j] : 0.0f;
                } else {
                    a[q] = rok && i < M ? dab[r * ldab + i] : 0.0f;
                    b[q] = rok && j < N ? ldv<BF16>(p.x, token(r) * p.d + j) : 0.0f;
                }
            }
        }
        if constexpr (kRows) {
#pragma unroll
            for (int q = 0; q < 4; ++q) As[kc_k + q][kc_i] = a[q];
        } else {
            *reinterpret_cast<float4*>(&As[ic_k][ic_i]) = make_float4(a[0], a[1], a[2], a[3]);
        }
        if constexpr (MODE == GB_AB) {
#pragma unroll
            for (int q = 0; q < 4; ++q) Bs[kc_k + q][kc_i] = b[q];
        } else {
            *reinterpret_cast<float4*>(&Bs[ic_k][ic_i]) = make_float4(b[0], b[1], b[2], b[3]);
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < FBK; ++kk) {
            const float4 av = *reinterpret_cast<const float4*>(&As[kk][ty * 4]);
            const float4 bv = *reinterpret_cast<const float4*>(&Bs[kk][tx * 4]);
            const float ar[4] = {av.x, av.y, av.z, av.w}, br[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(ar[i], br[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int rr = m0 + ty * 4 + i;
        if (rr >= M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int col = n0 + tx * 4 + j;
            if (col >= N) continue;
            const float v = acc[i][j];
            if constexpr (MODE == GB_AB) {
                ab[(row0 + rr) * ldab + col] = v;
            } else if constexpr (MODE == GB_DH) {
                // SwiGLU backward of h = silu(a) b with dh = w (dout W2)
                const int64_t r = row0 + rr;
                const float w = shared ? 1.0f : p.wrow[r];
                const float dh = w * v;
                const float av = ab[r * ldab + col], bv = ab[r * ldab + n_out + col];
                const float sg = 1.0f / (1.0f + expf(-av));
                const float sa = av * sg;
                dab[r * ldab + col] = dh * bv * sg * (1.0f + av * (1.0f - sg));
                dab[r * ldab + n_out + col] = dh * sa;
                wh[r * n_out + col] = w * sa * bv;
            } else if constexpr (MODE == GB_DX) {
                (shared ? p.dx_s : p.dx_r)[(row0 + rr) * p.d + col] = v;
            } else {
                const int64_t gi = MODE == GB_DW2 ? static_cast<int64_t>(g) * p.d * p.inter
                                                  : static_cast<int64_t>(g) * 2 * p.inter * p.d;
                void* out = shared ? (MODE == GB_DW2 ? p.dws2 : p.dws13) : (MODE == GB_DW2 ? p.dw2 : p.dw13);
                const int64_t e = (shared ? 0 : gi) + static_cast<int64_t>(rr) * N + col;
                if constexpr (BF16) static_cast<uint16_t*>(out)[e] = f32_to_bf16(v);
                else static_cast<float*>(out)[e] = v;
            }
        }
    }
}

// ============================================================== combine

template <bool BF16>
__global__ void combine_kernel(int64_t T, int d, int k, const int32_t* __restrict__ inv,
                               const float* __restrict__ topk_w, const void* __restrict__ y_r,
                               const void* __restrict__ y_s, void* __restrict__ out) {
    const int per_row = d / 8;
    const int64_t n = T * per_row;
    for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t j = i / per_row;
        const int c = static_cast<int>(i % per_row) * 8;
        float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        for (int s = 0; s < k; ++s) {
            const float w = topk_w[j * k + s];
            float v[8];
            load8<BF16>(y_r, static_cast<int64_t>(inv[j * k + s]) * d + c, v);
#pragma unroll
            for (int q = 0; q < 8; ++q) acc[q] = fmaf(w, v[q], acc[q]);
        }
        if (y_s != nullptr) {
            float v[8];
            load8<BF16>(y_s, j * d + c, v);
#pragma unroll
            for (int q = 0; q < 8; ++q) acc[q] += v[q];
        }
        if constexpr (BF16) {
            uint4 o;
            o.x = static_cast<uint32_t>(f32_to_bf16(acc[0])) | (static_cast<uint32_t>(f32_to_bf16(acc[1])) << 16);
            o.y = static_cast<uint32_t>(f32_to_bf16(acc[2])) | (static_cast<uint32_t>(f32_to_bf16(acc[3])) << 16);
            o.z = static_cast<uint32_t>(f32_to_bf16(acc[4])) | (static_cast<uint32_t>(f32_to_bf16(acc[5])) << 16);
            o.w = static_cast<uint32_t>(f32_to_bf16(acc[6])) | (static_cast<uint32_t>(f32_to_bf16(acc[7])) << 16);
            *reinterpret_cast<uint4*>(static_cast<uint16_t*>(out) + j * d + c) = o;
        } else {
            float4* o = reinterpret_cast<float4*>(static_cast<float*>(out) + j * d + c);
            o[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
            o[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
        }
    }
}

GemmArgs make_args(const ExpertArgs& a, const ExpWs& w, const int32_t* work, int part) {
    GemmArgs g;
    g.part = part;
    g.T = a.T;
    g.d = a.d;
    g.E = a.E;
    g.k = a.k;
    g.inter = a.inter;
    g.shared_inter = a.shared_inter;
    g.packed = a.packed;
    g.x = a.x;
    g.w13 = a.w13;
    g.w2 = a.w2;
    g.ws13 = a.ws13;
    g.ws2 = a.ws2;
    g.off = a.expert_offsets;
    g.perm_token = a.perm_token;
    g.work = work;
    g.h_r = w.h_r;
    g.h_s = w.h_s;
    g.y_r = w.y_r;
    g.y_s = w.y_s;
    g.dout = nullptr;
    g.w2t = g.ws2t = g.w13t = g.ws13t = nullptr;
    g.ab_r = a.ab_r;
    g.ab_s = a.ab_s;
    g.dab_r = g.dab_s = g.dx_r = g.dx_s = nullptr;
    g.wrow = nullptr;
    g.wh_r = nullptr;
    g.inv = a.perm_inv;
    g.topk_w = a.topk_w;
    g.out = a.out;
    return g;
}

// Grid size: 8 XCD ranges, each at most a bound on the routed items over 8
// plus the shared items over 8 (host side; the exact split is made on the device).
int64_t work_bound(int64_t T, int k, int E, int bm, int nt_r, int nt_s, bool has_shared, int part) {
    const int64_t R = T * k;
    const int64_t routed = part == 2 ? 0 : (ceil_div(R, bm) + E) * nt_r;
    const int64_t shared = (has_shared && part != 1) ? ceil_div(T, bm) * nt_s : 0;
    return 8 * (ceil_div(routed, 8) + ceil_div(shared, 8));
}

struct Plan {
    int bm, bm2, nt1_r, nt1_s, nt2;
    bool has_shared;
};

Plan plan_of(const ExpertArgs& a) {
    Plan p;
    const bool bf16 = a.act_dtype == 1;
    const bool pk = bf16 && a.packed;
    p.bm = pk ? PK_BM : bf16 ? DCfg::BM : FBM;
    p.bm2 = p.bm;
    const int tn1 = pk ? pk_tile_cols(1) : bf16 ? tile_cols<DCfg>(1) : 32;  // H columns per GEMM1 tile
    const int tn2 = pk ? pk_tile_cols(2) : bf16 ? tile_cols<DCfg>(2) : 64;  // output columns per GEMM2 tile
    p.nt1_r = static_cast<int>(ceil_div(a.inter, tn1));
    p.nt1_s = static_cast<int>(ceil_div(a.shared_inter, tn1));
    p.nt2 = static_cast<int>(ceil_div(a.d, tn2));
    p.has_shared = a.shared_inter > 0;
    return p;
}

}  // namespace

size_t experts_workspace_bytes(int64_t T, int d, int E, int k, int inter, int shared_inter,
                               int act_dtype) {
    const int64_t R = T * k;
    const size_t s = esz(act_dtype);
    return align_up(s * R * inter, 256) + align_up(s * T * shared_inter, 256) +
           align_up(s * R * d, 256) + align_up(s * T * d, 256) +
           2 * align_up(sizeof(int32_t) * (E + 2), 256);
}

WorkTables experts_work_tables(const ExpertArgs& a, void* ws) {
    ExpWs w = carve(ws, a.T, a.d, a.k, a.inter, a.shared_inter, a.act_dtype, a.E);
    const Plan p = plan_of(a);
    WorkTables t;
    t.work1 = w.work1;
    t.work2 = w.work2;
    t.bm = p.bm;  // both GEMMs use the same tile height
    t.nt1_r = p.nt1_r;
    t.nt1_s = p.nt1_s;
    t.nt2 = p.nt2;
    t.has_shared = p.has_shared ? 1 : 0;
    return t;
}

hipError_t launch_experts_gemm1(const ExpertArgs& a, void* ws, int part, hipStream_t stream) {
    ExpWs w = carve(ws, a.T, a.d, a.k, a.inter, a.shared_inter, a.act_dtype, a.E);
    const Plan p = plan_of(a);
    const GemmArgs g = make_args(a, w, w.work1, part);
    const dim3 grid(static_cast<unsigned>(work_bound(a.T, a.k, a.E, p.bm, p.nt1_r, p.nt1_s, p.has_shared, part)));
    if (grid.x == 0) return hipSuccess;
    if (a.act_dtype == 1 && a.packed && a.ab_r != nullptr)
        hipLaunchKernelGGL(gemm_bf16_pk_kernel<6>, grid, dim3(PK_THREADS), 0, stream, g);
    else if (a.act_dtype == 1 && a.packed)
        hipLaunchKernelGGL(gemm_bf16_pk_kernel<1>, grid, dim3(PK_THREADS), 0, stream, g);
    else if (a.act_dtype == 1)
        hipLaunchKernelGGL((gemm_bf16_dma_kernel<1, DCfg>), grid, dim3(DCfg::THREADS), 0, stream, g);
    else
        hipLaunchKernelGGL(gemm_f32_kernel<1>, grid, dim3(kThreads), 0, stream, g);
    return hipGetLastError();
}

hipError_t launch_experts_gemm2_combine(const ExpertArgs& a, void* ws, hipStream_t stream) {
    if (!(a.act_dtype == 1 && a.packed && a.shared_inter > 0)) return hipErrorInvalidValue;
    ExpWs w = carve(ws, a.T, a.d, a.k, a.inter, a.shared_inter, a.act_dtype, a.E);
    const Plan p = plan_of(a);
    const GemmArgs g = make_args(a, w, w.work2, 2);
    const dim3 grid(static_cast<unsigned>(work_bound(a.T, a.k, a.E, p.bm2, p.nt2, p.nt2, p.has_shared, 2)));
    if (grid.x == 0) return hipSuccess;
    hipLaunchKernelGGL(gemm_bf16_pk_kernel<7>, grid, dim3(PK_THREADS), 0, stream, g);
    return hipGetLastError();
}

hipError_t launch_experts_gemm2(const ExpertArgs& a, void* ws, int part, hipStream_t stream) {
    ExpWs w = carve(ws, a.T, a.d, a.k, a.inter, a.shared_inter, a.act_dtype, a.E);
    const Plan p = plan_of(a);
    const GemmArgs g = make_args(a, w, w.work2, part);
    const dim3 grid(static_cast<unsigned>(work_bound(a.T, a.k, a.E, p.bm2, p.nt2, p.nt2, p.has_shared, part)));
    if (grid.x == 0) return hipSuccess;
    if (a.act_dtype == 1 && a.packed)
        hipLaunchKernelGGL(gemm_bf16_pk_kernel<2>, grid, dim3(PK_THREADS), 0, stream, g);
    else if (a.act_dtype == 1)
        hipLaunchKernelGGL((gemm_bf16_dma_kernel<2, DCfg>), grid, dim3(DCfg::THREADS), 0, stream, g);
    else
        hipLaunchKernelGGL(gemm_f32_kernel<2>, grid, dim3(kThreads), 0, stream, g);
    return hipGetLastError();
}

// ---------------------------------------------------------------- backward (modes 3-5)

// Work table of one tiling (bm rows x nt column tiles per routed expert, then
// the shared items): one block of 256 threads, thread g counts expert g's items
// and an LDS scan forms the prefix sums (E <= 256).
__global__ void __launch_bounds__(256)
bwd_work_kernel(const int32_t* __restrict__ off, int E, int64_t T, int bm, int nt_r, int nt_s, int has_shared,
                int32_t* __restrict__ work) {
    __shared__ int32_t sc[256];
    const int g = threadIdx.x;
    sc[g] = g < E ? static_cast<int32_t>(ceil_div(off[g + 1] - off[g], bm)) * nt_r : 0;
    __syncthreads();
    for (int o = 1; o < 256; o <<= 1) {  // inclusive scan
        const int32_t v = g >= o ? sc[g - o] : 0;
        __syncthreads();
        sc[g] += v;
        __syncthreads();
    }
    if (g == 0) work[0] = 0;
    if (g < E) work[g + 1] = sc[g];
    if (g == 0) work[E + 1] = sc[E - 1] + (has_shared ? static_cast<int32_t>(ceil_div(T, bm)) * nt_s : 0);
}

ExpertFwdBuffers experts_fwd_buffers(const ExpertArgs& a, void* ws) {
    const ExpWs w = carve(ws, a.T, a.d, a.k, a.inter, a.shared_inter, a.act_dtype, a.E);
    ExpertFwdBuffers b;
    b.h_r = w.h_r;
    b.h_s = w.h_s;
    b.y_r = w.y_r;
    b.y_s = w.y_s;
    b.work1 = w.work1;
    b.work2 = w.work2;
    return b;
}

hipError_t launch_bwd_gemm(int mode, const ExpertArgs& a, void* fwd_ws, const BwdGemmPtrs& bp, int part,
                           hipStream_t stream) {
    const ExpWs w = carve(fwd_ws, a.T, a.d, a.k, a.inter, a.shared_inter, a.act_dtype, a.E);
    const bool has_shared = a.shared_inter > 0;
    int nt_r, nt_s;
    const int32_t* work;
    if (mode == 3) {
        nt_r = static_cast<int>(ceil_div(a.inter, pk_tile_cols(3)));
        nt_s = static_cast<int>(ceil_div(a.shared_inter, pk_tile_cols(3)));
        work = w.work1;  // the forward GEMM1's table: same tiling
    } else if (mode == 4) {
        nt_r = static_cast<int>(ceil_div(a.inter, pk_tile_cols(4)));
        nt_s = static_cast<int>(ceil_div(a.shared_inter, pk_tile_cols(4)));
        work = bp.work4;
        if (part != 2) {
            hipLaunchKernelGGL(bwd_work_kernel, dim3(1), dim3(256), 0, stream, a.expert_offsets, a.E, a.T, PK_BM, nt_r,
                               nt_s, has_shared ? 1 : 0, bp.work4);
            const hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
    } else {
        nt_r = nt_s = static_cast<int>(ceil_div(a.d, pk_tile_cols(5)));
        work = w.work2;  // the forward GEMM2's table: same tiling
    }
    GemmArgs g = make_args(a, w, work, part);
    g.dout = bp.dout;
    g.w2t = bp.w2t;
    g.ws2t = bp.ws2t;
    g.w13t = bp.w13t;
    g.ws13t = bp.ws13t;
    g.ab_r = bp.ab_r;
    g.ab_s = bp.ab_s;
    g.dab_r = bp.dab_r;
    g.dab_s = bp.dab_s;
    g.dx_r = bp.dx_r;
    g.dx_s = bp.dx_s;
    g.wrow = bp.wrow;
    g.wh_r = bp.wh_r;
    const dim3 grid(static_cast<unsigned>(work_bound(a.T, a.k, a.E, PK_BM, nt_r, nt_s, has_shared, part)));
    if (grid.x == 0) return hipSuccess;
    if (mode == 3) hipLaunchKernelGGL(gemm_bf16_pk_kernel<3>, grid, dim3(PK_THREADS), 0, stream, g);
    else if (mode == 4) hipLaunchKernelGGL(gemm_bf16_pk_kernel<4>, grid, dim3(PK_THREADS), 0, stream, g);
    else hipLaunchKernelGGL(gemm_bf16_pk_kernel<5>, grid, dim3(PK_THREADS), 0, stream, g);
    return hipGetLastError();
}

hipError_t launch_generic_bwd(int step, const ExpertArgs& a, const GenericBwdPtrs& bp, hipStream_t stream) {
    GenBwdArgs g;
    g.T = a.T;
    g.d = a.d;
    g.E = a.E;
    g.inter = a.inter;
    g.shared_inter = a.shared_inter;
    g.off = a.expert_offsets;
    g.perm_token = a.perm_token;
    g.work = bp.work;
    g.x = a.x;
    g.dout = bp.dout;
    g.w13 = a.w13;
    g.w2 = a.w2;
    g.ws13 = a.ws13;
    g.ws2 = a.ws2;
    g.ab_r = bp.ab_r;
    g.ab_s = bp.ab_s;
    g.dab_r = bp.dab_r;
    g.dab_s = bp.dab_s;
    g.wh_r = bp.wh_r;
    g.wh_s = bp.wh_s;
    g.dx_r = bp.dx_r;
    g.dx_s = bp.dx_s;
    g.wrow = bp.wrow;
    g.dw13 = bp.dw13;
    g.dw2 = bp.dw2;
    g.dws13 = bp.dws13;
    g.dws2 = bp.dws2;
    const bool bf16 = a.act_dtype == 1;
    const bool has_shared = a.shared_inter > 0;
    dim3 grid;
    if (step <= GB_DX) {
        const int nt_r = gb_row_tiles(step, a.inter, a.d), nt_s = gb_row_tiles(step, a.shared_inter, a.d);
        hipLaunchKernelGGL(bwd_work_kernel, dim3(1), dim3(256), 0, stream, a.expert_offsets, a.E, a.T, FBM, nt_r, nt_s,
                           has_shared ? 1 : 0, bp.work);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        grid = dim3(static_cast<unsigned>(work_bound(a.T, a.k, a.E, FBM, nt_r, nt_s, has_shared, 0)));
    } else {
        auto tiles = [&](int n_out) {
            const int64_t M = step == GB_DW2 ? a.d : 2 * n_out, N = step == GB_DW2 ? n_out : a.d;
            return ceil_div(M, FBM) * ceil_div(N, FBNB);
        };
        const int64_t t_r = tiles(a.inter), t_s = has_shared ? tiles(a.shared_inter) : 0;
        grid = dim3(static_cast<unsigned>(t_r > t_s ? t_r : t_s), static_cast<unsigned>(a.E + (has_shared ? 1 : 0)));
    }
    if (grid.x == 0) return hipSuccess;
#define SMOES_GB(M)                                                                                    \
    do {                                                                                               \
        if (bf16) hipLaunchKernelGGL((gemm_f32_bwd_kernel<M, true>), grid, dim3(kThreads), 0, stream, g);  \
        else hipLaunchKernelGGL((gemm_f32_bwd_kernel<M, false>), grid, dim3(kThreads), 0, stream, g);      \
    } while (0)
    switch (step) {
        case GB_AB: SMOES_GB(GB_AB); break;
        case GB_DH: SMOES_GB(GB_DH); break;
        case GB_DX: SMOES_GB(GB_DX); break;
        case GB_DW2: SMOES_GB(GB_DW2); break;
        case GB_DW13: SMOES_GB(GB_DW13); break;
        default: return hipErrorInvalidValue;
    }
#undef SMOES_GB
    return hipGetLastError();
}

int64_t packed_weight_elems(int batch, int n, int k, int interleave) {
    const int64_t ng = interleave ? 2 * ceil_div(n, 32) : ceil_div(n, 32);
    return batch * packed_elems(ng, k);
}

hipError_t launch_pack_weights(const void* src, int batch, int n, int k, int interleave, int transpose, void* dst,
                               hipStream_t stream) {
    const int64_t frags = packed_weight_elems(batch, n, k, interleave) / 8;
    if (frags == 0) return hipSuccess;
    const unsigned blocks = static_cast<unsigned>(ceil_div(frags, 256) < 65536 ? ceil_div(frags, 256) : 65536);
    hipLaunchKernelGGL(pack_weights_kernel, dim3(blocks), dim3(256), 0, stream, static_cast<const uint16_t*>(src),
                       batch, n, k, interleave, transpose, static_cast<uint16_t*>(dst));
    return hipGetLastError();
}

hipError_t launch_experts_combine(const ExpertArgs& a, void* ws, hipStream_t stream) {
    ExpWs w = carve(ws, a.T, a.d, a.k, a.inter, a.shared_inter, a.act_dtype, a.E);
    const int64_t n = a.T * (a.d / 8);
    const unsigned blocks = static_cast<unsigned>(ceil_div(n, 256) < 16384 ? ceil_div(n, 256) : 16384);
    const void* ys = a.shared_inter > 0 ? w.y_s : nullptr;
    if (a.act_dtype == 1)
        hipLaunchKernelGGL(combine_kernel<true>, dim3(blocks), dim3(256), 0, stream, a.T, a.d, a.k,
                           a.perm_inv, a.topk_w, w.y_r, ys, a.out);
    else
        hipLaunchKernelGGL(combine_kernel<false>, dim3(blocks), dim3(256), 0, stream, a.T, a.d, a.k,
                           a.perm_inv, a.topk_w, w.y_r, ys, a.out);
    return hipGetLastError();
}

}  // namespace smoes
