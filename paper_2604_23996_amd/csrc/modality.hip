// Gaussian-statistics modality score (Sec. 3.2.2).
//
//  update (optional): per-modality batch count, mean and centred sum of
//     squares, folded into the caller's EMA-Welford state (Eq. 5-7).
//     gauss_partial: 4 waves share 512 columns (8 per lane) and split a
//       64-token chunk (rows loaded eight at a time); fp64 sums of
//       (x - shift) and (x - shift)^2, where the shift is the previous mean,
//       then a fixed-order LDS tree.
//     gauss_merge: one thread per (modality, column) adds the chunk partials
//       in chunk order and applies the EMA update.
//  score: gauss_prep turns the state into per-column mu_m and 1 / sigma^2_m
//     (fp64 division, stored fp32) and the fp64 constant sum_d log(s2_v / s2_t)
//     as per-block parts;
//     modality_score evaluates, per token,
//       Delta = sum_d [log s2_v - log s2_t + (x - mu_v)^2 / s2_v - (x - mu_t)^2 / s2_t]
//     (each column's two squared terms in fp32, accumulated in fp64);
//     M_vision = sigmoid(-Delta / (2 tau)), M_text = 1 - M_vision (Eq. 8-9).
//     The two squared terms are kept apart rather than expanded around a
//     common centre: with very different variances the expansion cancels
//     terms ~1/sigma^2 times larger than the result.
#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

constexpr int kChunkRows = 64;    // tokens per gauss_partial block (16 per wave)
constexpr int kColsPerBlock = 512; // 64 lanes x 8 columns
constexpr int kScoreTokPerWave = 2;
constexpr int kScoreThreads = 256;
constexpr int kPrepThreads = 256;   // columns per gauss_prep block
constexpr int kPrepMaxBlocks = 64;  // SMOES_D_MAX / kPrepThreads

struct ModalityWs {
    float* coef;       // [4][d]: mu_v, 1/s2_v, mu_t, 1/s2_t
    double* cst;       // [ceil(d / 256)]: per column block, sum (log s2_v - log s2_t)
    double* n_old;     // [2]: state counts before the update
    int32_t* counts;   // [nchunk][2]
    double* s1;        // [nchunk][2][d]
    double* s2;        // [nchunk][2][d]
};

ModalityWs carve(void* ws, int64_t T, int d) {
    char* p = static_cast<char*>(ws);
    ModalityWs w;
    const int64_t nchunk = ceil_div(T, kChunkRows);
    w.coef = reinterpret_cast<float*>(p);
    p += align_up(sizeof(float) * 4 * d, 256);
    w.cst = reinterpret_cast<double*>(p);
    p += sizeof(double) * kPrepMaxBlocks;
    w.n_old = reinterpret_cast<double*>(p);
    p += 256;
    w.counts = reinterpret_cast<int32_t*>(p);
    p += align_up(sizeof(int32_t) * 2 * nchunk, 256);
    w.s1 = reinterpret_cast<double*>(p);
    p += align_up(sizeof(double) * 2 * nchunk * d, 256);
    w.s2 = reinterpret_cast<double*>(p);
    return w;
}

__device__ __forceinline__ double shift_of(const float* smu, const float* n, int m, int d, int col) {
    const double nm = static_cast<double>(n[m]);
    return nm > 0.0 ? static_cast<double>(smu[static_cast<int64_t>(m) * d + col]) / nm : 0.0;
}

template <bool BF16>
__global__ void __launch_bounds__(256)
gauss_partial_kernel(const void* __restrict__ x, int64_t T, int d, const uint8_t* __restrict__ mid,
                     const float* __restrict__ gauss_n, const float* __restrict__ gauss_smu,
                     int32_t* __restrict__ counts, double* __restrict__ s1g, double* __restrict__ s2g,
                     double* __restrict__ n_old) {
    __shared__ double red[2][64][32];
    const int wave = threadIdx.x / kWave;
    const int lane = lane_id();
    const int64_t chunk = blockIdx.x;
    const int col0 = blockIdx.y * kColsPerBlock + lane * 8;
    const bool active = col0 < d;
    if (chunk == 0 && blockIdx.y == 0 && threadIdx.x < 2) n_old[threadIdx.x] = gauss_n[threadIdx.x];

    double sh[2][8];
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int i = 0; i < 8; ++i) sh[m][i] = active ? shift_of(gauss_smu, gauss_n, m, d, col0 + i) : 0.0;
    double s1[2][8], s2[2][8];
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int i = 0; i < 8; ++i) s1[m][i] = s2[m][i] = 0.0;
    int cnt[2] = {0, 0};
    const int64_t r0 = chunk * kChunkRows;
    const int64_t r1 = r0 + kChunkRows < T ? r0 + kChunkRows : T;
    // rows r0 + wave, + 4, ... in groups of U: the group's labels and row
    // chunks are loaded first, then accumulated in row order
    constexpr int U = 8;
    for (int64_t g = r0 + wave; g < r1; g += 4 * U) {
        int mm[U];
        float v[U][8];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t r = g + 4 * u;
            const int64_t rr = r < r1 ? r : g;
            mm[u] = mid[rr] ? 1 : 0;
            if (active) load8<BF16>(x, rr * d + col0, v[u]);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (g + 4 * u >= r1) break;  // wave-uniform
            const int m = mm[u];
            cnt[m] += 1;
            if (!active) continue;
            if (m == 0) {
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const double y = static_cast<double>(v[u][i]) - sh[0][i];
                    s1[0][i] += y;
                    s2[0][i] = fma(y, y, s2[0][i]);
                }
            } else {
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const double y = static_cast<double>(v[u][i]) - sh[1][i];
                    s1[1][i] += y;
                    s2[1][i] = fma(y, y, s2[1][i]);
                }
            }
        }
    }
    // fixed-order tree over the waves: (w0 + w2) + (w1 + w3)
    auto put = [&](int slot) {
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                red[slot][lane][m * 8 + i] = s1[m][i];
                red[slot][lane][16 + m * 8 + i] = s2[m][i];
            }
    };
    auto add = [&](int slot) {
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                s1[m][i] += red[slot][lane][m * 8 + i];
                s2[m][i] += red[slot][lane][16 + m * 8 + i];
            }
    };
    if (wave >= 2) put(wave - 2);
    __syncthreads();
    if (wave < 2) add(wave);
    __syncthreads();
    if (wave == 1) put(0);
    __syncthreads();
    if (wave == 0) {
        add(0);
        if (active) {
#pragma unroll
            for (int m = 0; m < 2; ++m)
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const int64_t o = (chunk * 2 + m) * d + col0 + i;
                    s1g[o] = s1[m][i];
                    s2g[o] = s2[m][i];
                }
        }
    }
    // token counts per modality: every wave counted its own rows
    __shared__ int wc[4][2];
    if (lane == 0) {
        wc[wave][0] = cnt[0];
        wc[wave][1] = cnt[1];
    }
    __syncthreads();
    if (blockIdx.y == 0 && threadIdx.x < 2)
        counts[chunk * 2 + threadIdx.x] = (wc[0][threadIdx.x] + wc[2][threadIdx.x]) +
                                          (wc[1][threadIdx.x] + wc[3][threadIdx.x]);
}

__global__ void gauss_merge_kernel(int d, int64_t nchunk, const int32_t* __restrict__ counts,
                                   const double* __restrict__ s1g, const double* __restrict__ s2g,
                                   const double* __restrict__ n_old, float beta,
                                   float* __restrict__ gauss_n, float* __restrict__ gauss_smu,
                                   float* __restrict__ gauss_ssig) {
    const int m = blockIdx.y;
    const int col = blockIdx.x * blockDim.x + threadIdx.x;
    if (col >= d) return;
    int64_t n = 0;
    double S1 = 0.0, S2 = 0.0;
    constexpr int B = 16;  // chunk loads in flight; the sums still run in chunk order
    for (int64_t c0 = 0; c0 < nchunk; c0 += B) {
        int32_t vn[B];
        double v1[B], v2[B];
#pragma unroll
        for (int q = 0; q < B; ++q) {
            const int64_t c = c0 + q < nchunk ? c0 + q : c0;
            vn[q] = counts[c * 2 + m];
            v1[q] = s1g[(c * 2 + m) * d + col];
            v2[q] = s2g[(c * 2 + m) * d + col];
        }
#pragma unroll
        for (int q = 0; q < B; ++q)
            if (c0 + q < nchunk) {
                n += vn[q];
                S1 += v1[q];
                S2 += v2[q];
            }
    }
    const double nprev = n_old[m];
    const double smu_old = gauss_smu[static_cast<int64_t>(m) * d + col];
    const double ssig_old = gauss_ssig[static_cast<int64_t>(m) * d + col];
    const double shift = nprev > 0.0 ? smu_old / nprev : 0.0;
    const double b = static_cast<double>(beta);
    const double nt = static_cast<double>(n);
    double mean_T = 0.0, m2_T = 0.0, cross = 0.0;
    if (n > 0) {
        mean_T = shift + S1 / nt;
        m2_T = S2 - S1 * (S1 / nt);
        if (m2_T < 0.0) m2_T = 0.0;
        if (nprev > 0.0) {
            const double dm = mean_T - shift;
            cross = dm * dm * (b * nprev * nt) / (b * nprev + nt);
        }
    }
    gauss_smu[static_cast<int64_t>(m) * d + col] = static_cast<float>(b * smu_old + nt * mean_T);
    gauss_ssig[static_cast<int64_t>(m) * d + col] = static_cast<float>(b * ssig_old + m2_T + cross);
    if (col == 0) gauss_n[m] = static_cast<float>(b * nprev + nt);
}

// Per-column score coefficients; each block of 256 columns also writes its
// part of the fp64 constant (a fixed-order LDS tree), summed in block order
// by modality_score.
__global__ void __launch_bounds__(kPrepThreads)
gauss_prep_kernel(int d, const float* __restrict__ gauss_n, const float* __restrict__ gauss_smu,
                  const float* __restrict__ gauss_ssig, float var_floor, float* __restrict__ coef,
                  double* __restrict__ cst_part) {
    __shared__ double part[kPrepThreads];
    const double nv = gauss_n[0], nt = gauss_n[1];
    const int c = blockIdx.x * kPrepThreads + threadIdx.x;
    double acc = 0.0;
    if (c < d) {
        double mv = 0.0, vv = 1.0, mt = 0.0, vt = 1.0;
        if (nv > 0.0) {
            mv = gauss_smu[c] / nv;
            vv = fmax(static_cast<double>(gauss_ssig[c]) / nv, static_cast<double>(var_floor));
        }
        if (nt > 0.0) {
            mt = gauss_smu[d + c] / nt;
            vt = fmax(static_cast<double>(gauss_ssig[d + c]) / nt, static_cast<double>(var_floor));
        }
        coef[c] = static_cast<float>(mv);
        coef[d + c] = static_cast<float>(1.0 / vv);
        coef[2 * d + c] = static_cast<float>(mt);
        coef[3 * d + c] = static_cast<float>(1.0 / vt);
        acc = log(vv) - log(vt);
    }
    part[threadIdx.x] = acc;
    __syncthreads();
    for (int s = kPrepThreads / 2; s > 0; s >>= 1) {
        if (threadIdx.x < s) part[threadIdx.x] += part[threadIdx.x + s];
        __syncthreads();
    }
    if (threadIdx.x == 0) cst_part[blockIdx.x] = part[0];
}

template <bool BF16>
__global__ void __launch_bounds__(kScoreThreads)
modality_score_kernel(const void* __restrict__ x, int64_t T, int d, const float* __restrict__ coef,
                      const double* __restrict__ cst_part, int n_part, double inv2tau, float* __restrict__ M) {
    __shared__ double red[kScoreThreads / kWave][kScoreTokPerWave][kWave];
    const int wave = threadIdx.x / kWave;
    const int lane = lane_id();
    const int64_t tok0 = (static_cast<int64_t>(blockIdx.x) * (kScoreThreads / kWave) + wave) * kScoreTokPerWave;
    if (tok0 >= T) return;  // whole waves only: the reduction below is wave-local
    int64_t rows[kScoreTokPerWave];
#pragma unroll
    for (int t = 0; t < kScoreTokPerWave; ++t) rows[t] = tok0 + t < T ? tok0 + t : T - 1;
    double acc[kScoreTokPerWave];
#pragma unroll
    for (int t = 0; t < kScoreTokPerWave; ++t) acc[t] = 0.0;
#pragma unroll 4
    for (int c0 = lane * 8; c0 < d; c0 += kWave * 8) {
        float mv[8], iv[8], mt[8], it[8];
        const float4* p0 = reinterpret_cast<const float4*>(coef + c0);
        const float4* p1 = reinterpret_cast<const float4*>(coef + d + c0);
        const float4* p2 = reinterpret_cast<const float4*>(coef + 2 * d + c0);
        const float4* p3 = reinterpret_cast<const float4*>(coef + 3 * d + c0);
        *reinterpret_cast<float4*>(&mv[0]) = p0[0];
        *reinterpret_cast<float4*>(&mv[4]) = p0[1];
        *reinterpret_cast<float4*>(&iv[0]) = p1[0];
        *reinterpret_cast<float4*>(&iv[4]) = p1[1];
        *reinterpret_cast<float4*>(&mt[0]) = p2[0];
        *reinterpret_cast<float4*>(&mt[4]) = p2[1];
        *reinterpret_cast<float4*>(&it[0]) = p3[0];
        *reinterpret_cast<float4*>(&it[4]) = p3[1];
#pragma unroll
        for (int t = 0; t < kScoreTokPerWave; ++t) {
            float v[8];
            load8<BF16>(x, rows[t] * d + c0, v);
            float part = 0.0f;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const float dv = v[i] - mv[i];
                const float dt = v[i] - mt[i];
                part += dv * dv * iv[i] - dt * dt * it[i];
            }
            acc[t] += static_cast<double>(part);
        }
    }
    // per token: the 64 lane partials in lane order, then the constant in block order
#pragma unroll
    for (int t = 0; t < kScoreTokPerWave; ++t) red[wave][t][lane] = acc[t];
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (lane < kScoreTokPerWave) {
        const int t = lane;
        double sum = 0.0;
        for (int l = 0; l < kWave; ++l) sum += red[wave][t][l];
        double c = 0.0;
        for (int b = 0; b < n_part; ++b) c += cst_part[b];
        const double delta = sum + c;
        if (tok0 + t < T) {
            const double s = -delta * inv2tau;
            double mv, mt;
            if (s >= 0.0) {
                const double e = exp(-s);
                mv = 1.0 / (1.0 + e);
                mt = e / (1.0 + e);
            } else {
                const double e = exp(s);
                mv = e / (1.0 + e);
                mt = 1.0 / (1.0 + e);
            }
            M[(tok0 + t) * 2] = static_cast<float>(mv);
            M[(tok0 + t) * 2 + 1] = static_cast<float>(mt);
        }
    }
}

}  // namespace

size_t modality_workspace_bytes(int64_t T, int d) {
    const int64_t nchunk = ceil_div(T, kChunkRows);
    return align_up(sizeof(float) * 4 * d, 256) + sizeof(double) * kPrepMaxBlocks + 256 +
           align_up(sizeof(int32_t) * 2 * nchunk, 256) +
           2 * align_up(sizeof(double) * 2 * nchunk * d, 256);
}

hipError_t launch_modality(const void* x, int x_dtype, int64_t T, int d, const uint8_t* modality_id,
                           float* gauss_n, float* gauss_smu, float* gauss_ssig, int update,
                           float beta, float tau, float var_floor, float* M, void* ws,
                           hipStream_t stream) {
    ModalityWs w = carve(ws, T, d);
    const bool bf16 = x_dtype == 1;
    hipError_t err;
    if (update) {
        const int64_t nchunk = ceil_div(T, kChunkRows);
        const dim3 grid(static_cast<unsigned>(nchunk), static_cast<unsigned>(ceil_div(d, kColsPerBlock)));
        if (bf16)
            hipLaunchKernelGGL(gauss_partial_kernel<true>, grid, dim3(256), 0, stream, x, T, d,
                               modality_id, gauss_n, gauss_smu, w.counts, w.s1, w.s2, w.n_old);
        else
            hipLaunchKernelGGL(gauss_partial_kernel<false>, grid, dim3(256), 0, stream, x, T, d,
                               modality_id, gauss_n, gauss_smu, w.counts, w.s1, w.s2, w.n_old);
        if ((err = hipGetLastError()) != hipSuccess) return err;
        hipLaunchKernelGGL(gauss_merge_kernel, dim3(static_cast<unsigned>(ceil_div(d, 64)), 2),
                           dim3(64), 0, stream, d, nchunk, w.counts, w.s1, w.s2, w.n_old, beta,
                           gauss_n, gauss_smu, gauss_ssig);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    const int n_part = static_cast<int>(ceil_div(d, kPrepThreads));
    hipLaunchKernelGGL(gauss_prep_kernel, dim3(n_part), dim3(kPrepThreads), 0, stream, d, gauss_n, gauss_smu,
                       gauss_ssig, var_floor, w.coef, w.cst);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    const double t = tau > 0.0f ? static_cast<double>(tau) : 0.5 * d;
    const double inv2tau = 1.0 / (2.0 * t);
    const int64_t tok_per_block = static_cast<int64_t>(kScoreThreads / kWave) * kScoreTokPerWave;
    const dim3 grid(static_cast<unsigned>(ceil_div(T, tok_per_block)));
    if (bf16)
        hipLaunchKernelGGL(modality_score_kernel<true>, grid, dim3(kScoreThreads), 0, stream, x, T,
                           d, w.coef, w.cst, n_part, inv2tau, M);
    else
        hipLaunchKernelGGL(modality_score_kernel<false>, grid, dim3(kScoreThreads), 0, stream, x,
                           T, d, w.coef, w.cst, n_part, inv2tau, M);
    return hipGetLastError();
}

}  // namespace smoes
