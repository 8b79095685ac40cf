// Grouped SwiGLU experts, shared experts and the weighted combine.
//
// Groups: g < E is routed expert g over its expert-contiguous rows
// [off[g], off[g+1]) (rows gathered from x through perm_token inside the
// GEMM's loader, so no permuted copy of x is written); g = E is the merged
// shared expert over all T tokens. A device-built work table (prefix over
// groups of m_tiles * n_tiles) lets one launch cover every group without any
// host synchronisation.
//
// Block -> tile mapping: blocks are dealt round-robin to the 8 XCDs, so block b
// runs on XCD b % 8. Each XCD takes one contiguous eighth of the work list,
// ordered (group, super-row of 8 m-tiles, n-tile, m-tile): the tiles that
// share a weight slice run back to back on one XCD and hit its L2.
//
// bf16: 128 x 128 tiles, BK = 64, 4 waves of 64 x 64 (2 x 2 MFMA
// 32x32x16 bf16 tiles), LDS double-buffered (row pitch 72 bf16 = 144 B keeps
// the 16-byte fragment reads conflict-free), fp32 accumulation.
//   GEMM1: B rows 0..63 are gate rows, 64..127 the matching up rows, so a
//          wave holds gate and up outputs of the same (row, column) in the
//          same lane: the SwiGLU epilogue is register-local. H is bf16.
//   GEMM2: Y = H W2^T, bf16.
// f32 (exact path for float32 layers): 64 x 64 FMA tiles, same work table.
#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

constexpr int kThreads = 256;
constexpr int kGroupM = 8;  // m-tiles per super-row in the work order

// bf16 MFMA tiles
constexpr int BM = 128, BNB = 128, BK = 64, LDP = BK + 8;
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

// Work table: work[g + 1] = work[g] + m_tiles(g) * n_tiles(g) for g in [0, G):
// one thread per group and a block-wide inclusive scan (E + 1 <= 257 groups).
__global__ void __launch_bounds__(512)
build_work_kernel(const int32_t* __restrict__ off, int E, int64_t T, int has_shared, int bm,
                  int nt_routed, int nt_shared, int32_t* __restrict__ work) {
    __shared__ int32_t sc[512];
    const int g = threadIdx.x;
    int32_t v = 0;
    if (g < E) v = static_cast<int32_t>(ceil_div(off[g + 1] - off[g], bm)) * nt_routed;
    else if (g == E && has_shared) v = static_cast<int32_t>(ceil_div(T, bm)) * nt_shared;
    sc[g] = v;
    __syncthreads();
    for (int o = 1; o < 512; o <<= 1) {
        const int32_t add = g >= o ? sc[g - o] : 0;
        __syncthreads();
        v += add;
        sc[g] = v;
        __syncthreads();
    }
    if (g == 0) work[0] = 0;
    if (g <= E) work[g + 1] = v;
}

struct Tile {
    int g;          // group (E = shared)
    int64_t row0;   // first row of the tile in the group's row space (global row index)
    int rows;       // valid rows in the tile
    int nt;         // n-tile
};

// Decode this block's tile; returns false when the block has no work.
__device__ __forceinline__ bool decode_tile(const int32_t* __restrict__ work, const int32_t* __restrict__ off,
                                            int E, int64_t T, int G, int bm, int nt_routed, int nt_shared,
                                            Tile& t) {
    const int total = work[G];
    const int per_xcd = (total + 7) / 8;
    const int xcd = blockIdx.x & 7;
    const int slot = blockIdx.x >> 3;
    if (slot >= per_xcd) return false;
    const int w = xcd * per_xcd + slot;
    if (w >= total) return false;
    int lo = 0, hi = G - 1;  // last g with work[g] <= w
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (work[mid] <= w) lo = mid; else hi = mid - 1;
    }
    const int g = lo;
    const int local = w - work[g];
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
    const int sb = local / (kGroupM * ntn);
    const int r = local % (kGroupM * ntn);
    const int gm = m_tiles - sb * kGroupM < kGroupM ? m_tiles - sb * kGroupM : kGroupM;
    const int mt = sb * kGroupM + r % gm;
    t.g = g;
    t.nt = r / gm;
    t.row0 = base + static_cast<int64_t>(mt) * bm;
    const int64_t left = rows_g - static_cast<int64_t>(mt) * bm;
    t.rows = static_cast<int>(left < bm ? left : bm);
    return true;
}

__device__ __forceinline__ float silu(float a) { return a / (1.0f + expf(-a)); }

struct GemmArgs {
    int64_t T;
    int d, E, inter, shared_inter;
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
};

// ============================================================== bf16 MFMA path

template <int MODE>
__global__ void __launch_bounds__(kThreads, 2)
gemm_bf16_kernel(GemmArgs p) {
    __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * LDP];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BNB * LDP];
    const int G = p.E + (p.shared_inter > 0 ? 1 : 0);
    const int nt_r = MODE == 1 ? static_cast<int>(ceil_div(p.inter, 64)) : static_cast<int>(ceil_div(p.d, 128));
    const int nt_s = MODE == 1 ? static_cast<int>(ceil_div(p.shared_inter, 64)) : nt_r;
    Tile t;
    if (!decode_tile(p.work, p.off, p.E, p.T, G, BM, nt_r, nt_s, t)) return;
    const bool shared = t.g == p.E;
    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = lane_id();
    const int wm = wave >> 1, wn = wave & 1;

    // operand geometry
    int K, n_out;
    const uint16_t* Abase;
    const uint16_t* Bbase;
    int64_t a_ld;
    if constexpr (MODE == 1) {
        K = p.d;
        n_out = shared ? p.shared_inter : p.inter;
        Abase = static_cast<const uint16_t*>(p.x);
        a_ld = p.d;
        Bbase = shared ? static_cast<const uint16_t*>(p.ws13)
                       : static_cast<const uint16_t*>(p.w13) + static_cast<int64_t>(t.g) * 2 * p.inter * p.d;
    } else {
        K = shared ? p.shared_inter : p.inter;
        n_out = p.d;
        Abase = shared ? static_cast<const uint16_t*>(p.h_s) : static_cast<const uint16_t*>(p.h_r);
        a_ld = K;
        Bbase = shared ? static_cast<const uint16_t*>(p.ws2)
                       : static_cast<const uint16_t*>(p.w2) + static_cast<int64_t>(t.g) * p.d * p.inter;
    }
    // per-thread load slots: 4 A rows, 4 B rows, one 16-byte k-chunk each
    const int kc = (tid & 7) * 8;
    const uint16_t* arow[4];
    const uint16_t* brow[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = (tid >> 3) + 32 * i;
        const int rr = r < t.rows ? r : 0;
        int64_t src;
        if (MODE == 1 && !shared) src = p.perm_token[t.row0 + rr];
        else src = t.row0 + rr;
        arow[i] = Abase + src * a_ld;
        int64_t brow_idx;
        if constexpr (MODE == 1) {
            int c = t.nt * 64 + (r & 63);
            if (c >= n_out) c = 0;
            brow_idx = (r < 64) ? c : n_out + c;
        } else {
            int c = t.nt * 128 + r;
            if (c >= n_out) c = 0;
            brow_idx = c;
        }
        brow[i] = Bbase + brow_idx * K;
    }
    uint4 ra[4], rb[4];
    auto gload = [&](int k0) {
        const bool ok = k0 + kc < K;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            ra[i] = ok ? *reinterpret_cast<const uint4*>(arow[i] + k0 + kc) : make_uint4(0, 0, 0, 0);
            rb[i] = ok ? *reinterpret_cast<const uint4*>(brow[i] + k0 + kc) : make_uint4(0, 0, 0, 0);
        }
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = (tid >> 3) + 32 * i;
            *reinterpret_cast<uint4*>(&As[buf][r * LDP + kc]) = ra[i];
            *reinterpret_cast<uint4*>(&Bs[buf][r * LDP + kc]) = rb[i];
        }
    };
    // B rows read by this wave: two 32-row blocks
    int bsub[2];
    if constexpr (MODE == 1) {
        bsub[0] = wn * 32;
        bsub[1] = 64 + wn * 32;
    } else {
        bsub[0] = wn * 64;
        bsub[1] = wn * 64 + 32;
    }
    f32x16_t acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x16_t{};

    const int nk = static_cast<int>(ceil_div(K, BK));
    gload(0);
    sstore(0);
    __syncthreads();
    const int half = lane >> 5, l32 = lane & 31;
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < nk) gload((kt + 1) * BK);
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            const int kk = ks * 16 + half * 8;
            bf16x8_t af[2], bfr[2];
#pragma unroll
            for (int i = 0; i < 2; ++i)
                af[i] = *reinterpret_cast<const bf16x8_t*>(&As[cur][(wm * 64 + i * 32 + l32) * LDP + kk]);
#pragma unroll
            for (int j = 0; j < 2; ++j)
                bfr[j] = *reinterpret_cast<const bf16x8_t*>(&Bs[cur][(bsub[j] + l32) * LDP + kk]);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < nk) sstore(cur ^ 1);
        __syncthreads();
    }

    // epilogue: element v of a 32x32 tile sits at row 8*(v/4) + 4*half + v%4, column l32
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int r = wm * 64 + i * 32 + 8 * (v >> 2) + 4 * half + (v & 3);
            if (r >= t.rows) continue;
            const int64_t grow = t.row0 + r;
            if constexpr (MODE == 1) {
                const int c = t.nt * 64 + wn * 32 + l32;
                if (c < n_out) {
                    const float h = silu(acc[i][0][v]) * acc[i][1][v];
                    uint16_t* H = shared ? static_cast<uint16_t*>(p.h_s) : static_cast<uint16_t*>(p.h_r);
                    H[grow * n_out + c] = f32_to_bf16(h);
                }
            } else {
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const int c = t.nt * 128 + wn * 64 + j * 32 + l32;
                    if (c < n_out) {
                        uint16_t* Y = shared ? static_cast<uint16_t*>(p.y_s) : static_cast<uint16_t*>(p.y_r);
                        Y[grow * n_out + c] = f32_to_bf16(acc[i][j][v]);
                    }
                }
            }
        }
    }
}

// ============================================================== f32 FMA path

template <int MODE>
__global__ void __launch_bounds__(kThreads)
gemm_f32_kernel(GemmArgs p) {
    __shared__ float As[FBK][FBM + 4];
    __shared__ float Bs[FBK][FBNB + 4];
    __shared__ float Cs[FBM][FBNB + 1];
    const int G = p.E + (p.shared_inter > 0 ? 1 : 0);
    const int nt_r = MODE == 1 ? static_cast<int>(ceil_div(p.inter, 32)) : static_cast<int>(ceil_div(p.d, 64));
    const int nt_s = MODE == 1 ? static_cast<int>(ceil_div(p.shared_inter, 32)) : nt_r;
    Tile t;
    if (!decode_tile(p.work, p.off, p.E, p.T, G, FBM, nt_r, nt_s, t)) return;
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

GemmArgs make_args(const ExpertArgs& a, const ExpWs& w, const int32_t* work) {
    GemmArgs g;
    g.T = a.T;
    g.d = a.d;
    g.E = a.E;
    g.inter = a.inter;
    g.shared_inter = a.shared_inter;
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
    return g;
}

// Upper bound on the work items of one GEMM (host side; sizes the grid).
int64_t work_bound(int64_t T, int k, int E, int bm, int nt_r, int nt_s, bool has_shared) {
    const int64_t R = T * k;
    int64_t m_r = ceil_div(R, bm) + E;
    int64_t b = m_r * nt_r;
    if (has_shared) b += ceil_div(T, bm) * nt_s;
    return ceil_div(b, 8) * 8;
}

struct Plan {
    int bm, nt1_r, nt1_s, nt2;
    bool has_shared;
};

Plan plan_of(const ExpertArgs& a) {
    Plan p;
    const bool bf16 = a.act_dtype == 1;
    p.bm = bf16 ? BM : FBM;
    const int tn1 = bf16 ? 64 : 32;   // H columns per GEMM1 tile
    const int tn2 = bf16 ? 128 : 64;  // output columns per GEMM2 tile
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

hipError_t launch_experts_plan(const ExpertArgs& a, void* ws, hipStream_t stream) {
    ExpWs w = carve(ws, a.T, a.d, a.k, a.inter, a.shared_inter, a.act_dtype, a.E);
    const Plan p = plan_of(a);
    hipLaunchKernelGGL(build_work_kernel, dim3(1), dim3(512), 0, stream, a.expert_offsets, a.E, a.T,
                       p.has_shared ? 1 : 0, p.bm, p.nt1_r, p.nt1_s, w.work1);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(build_work_kernel, dim3(1), dim3(512), 0, stream, a.expert_offsets, a.E, a.T,
                       p.has_shared ? 1 : 0, p.bm, p.nt2, p.nt2, w.work2);
    return hipGetLastError();
}

hipError_t launch_experts_gemm1(const ExpertArgs& a, void* ws, hipStream_t stream) {
    ExpWs w = carve(ws, a.T, a.d, a.k, a.inter, a.shared_inter, a.act_dtype, a.E);
    const Plan p = plan_of(a);
    const GemmArgs g = make_args(a, w, w.work1);
    const dim3 grid(static_cast<unsigned>(work_bound(a.T, a.k, a.E, p.bm, p.nt1_r, p.nt1_s, p.has_shared)));
    if (a.act_dtype == 1)
        hipLaunchKernelGGL(gemm_bf16_kernel<1>, grid, dim3(kThreads), 0, stream, g);
    else
        hipLaunchKernelGGL(gemm_f32_kernel<1>, grid, dim3(kThreads), 0, stream, g);
    return hipGetLastError();
}

hipError_t launch_experts_gemm2(const ExpertArgs& a, void* ws, hipStream_t stream) {
    ExpWs w = carve(ws, a.T, a.d, a.k, a.inter, a.shared_inter, a.act_dtype, a.E);
    const Plan p = plan_of(a);
    const GemmArgs g = make_args(a, w, w.work2);
    const dim3 grid(static_cast<unsigned>(work_bound(a.T, a.k, a.E, p.bm, p.nt2, p.nt2, p.has_shared)));
    if (a.act_dtype == 1)
        hipLaunchKernelGGL(gemm_bf16_kernel<2>, grid, dim3(kThreads), 0, stream, g);
    else
        hipLaunchKernelGGL(gemm_f32_kernel<2>, grid, dim3(kThreads), 0, stream, g);
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
