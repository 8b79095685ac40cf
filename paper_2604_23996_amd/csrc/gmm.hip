// GMM estimator: a K-component diagonal Gaussian mixture per modality in
// place of the single Gaussian of Sec. 3.2.2 (the supplementary GMM ablation,
// K in {2, 4}). The state per modality m and component c is (N, S_mu, S_sigma2)
// as in Eq. 5-7; pi_mc = N_mc / sum_c N_mc.
//
//  gmm_prep: state -> per (m, c, column) mu and 1 / sigma^2 (fp64 division,
//     stored fp32) and per column block the fp64 parts of sum_d log sigma^2.
//  gmm_loglik: per token and (m, c), q = sum_d (x - mu)^2 / sigma^2 (fp32 per
//     8-column stripe, accumulated in fp64, reduced by a fixed butterfly), the
//     component log-likelihood log pi - (sum log sigma^2 + q) / 2, then either
//     the score (Eq. 9 over the per-modality log-sum-exp) or the
//     responsibilities of the token's own modality (the E-step).
//  update (stepwise EM): gmm_partial sums r (x - shift), r (x - shift)^2 and r
//     per chunk of 64 tokens in fp64 (shift = the component's previous mean),
//     gmm_merge adds the chunks in order and applies Eq. 5-7 with the weighted
//     batch count, mean and centred sum of squares.
#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

constexpr int kGChunk = 64;         // tokens per gmm_partial block
constexpr int kGPartCols = 256;     // columns per gmm_partial block (64 lanes x 4)
constexpr int kGPrepThreads = 256;  // columns per gmm_prep block
constexpr int kGMaxParts = 64;      // SMOES_D_MAX / kGPrepThreads
constexpr int kGTokPerWave = 2;
constexpr int kGThreads = 256;

struct GmmWs {
    float* coef;      // [2K][2][d]: mu, 1 / sigma^2
    double* cst;      // [2K][kGMaxParts]: per column block, sum log sigma^2
    double* n_old;    // [2K]
    float* resp;      // [T][K] (when the caller passes none)
    double* wsum;     // [nchunk][2K]
    double* s1;       // [nchunk][2K][d]
    double* s2;       // [nchunk][2K][d]
};

GmmWs gmm_carve(void* ws, int64_t T, int d, int K) {
    char* p = static_cast<char*>(ws);
    const int64_t nchunk = ceil_div(T, kGChunk);
    GmmWs w;
    w.coef = reinterpret_cast<float*>(p);
    p += align_up(sizeof(float) * 2 * K * 2 * d, 256);
    w.cst = reinterpret_cast<double*>(p);
    p += align_up(sizeof(double) * 2 * K * kGMaxParts, 256);
    w.n_old = reinterpret_cast<double*>(p);
    p += 256;
    w.resp = reinterpret_cast<float*>(p);
    p += align_up(sizeof(float) * T * K, 256);
    w.wsum = reinterpret_cast<double*>(p);
    p += align_up(sizeof(double) * nchunk * 2 * K, 256);
    w.s1 = reinterpret_cast<double*>(p);
    p += align_up(sizeof(double) * nchunk * 2 * K * d, 256);
    w.s2 = reinterpret_cast<double*>(p);
    return w;
}

__global__ void __launch_bounds__(kGPrepThreads)
gmm_prep_kernel(int d, int K, const float* __restrict__ gn, const float* __restrict__ gsmu,
                const float* __restrict__ gssig, float var_floor, float* __restrict__ coef,
                double* __restrict__ cst) {
    __shared__ double part[kGPrepThreads];
    const int mc = blockIdx.y;  // m * K + c
    const double n = gn[mc];
    const int col = blockIdx.x * kGPrepThreads + threadIdx.x;
    double acc = 0.0;
    if (col < d) {
        double mu = 0.0, var = 1.0;
        if (n > 0.0) {
            mu = gsmu[static_cast<int64_t>(mc) * d + col] / n;
            var = fmax(static_cast<double>(gssig[static_cast<int64_t>(mc) * d + col]) / n, static_cast<double>(var_floor));
        }
        coef[(static_cast<int64_t>(mc) * 2) * d + col] = static_cast<float>(mu);
        coef[(static_cast<int64_t>(mc) * 2 + 1) * d + col] = static_cast<float>(1.0 / var);
        acc = log(var);
    }
    part[threadIdx.x] = acc;
    __syncthreads();
    for (int s = kGPrepThreads / 2; s > 0; s >>= 1) {
        if (threadIdx.x < s) part[threadIdx.x] += part[threadIdx.x + s];
        __syncthreads();
    }
    if (threadIdx.x == 0) cst[mc * kGMaxParts + blockIdx.x] = part[0];
}

// mode 0: scores M[T][2]; mode 1: responsibilities resp[T][K] of each token's own modality.
template <bool BF16, int K>
__global__ void __launch_bounds__(kGThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
gmm_loglik_kernel(const void* __restrict__ x, int64_t T, int d, const uint8_t* __restrict__ mid,
                  const float* __restrict__ coef, const double* __restrict__ cst, int n_part,
                  const float* __restrict__ gn, double inv_tau, int mode, float* __restrict__ M,
                  float* __restrict__ resp) {
    constexpr int MC = 2 * K;
    static_assert(kGTokPerWave == 2, "the token select below assumes two tokens per wave");
    const int wave = threadIdx.x / kWave;
    const int lane = lane_id();
    const int64_t tok0 = (static_cast<int64_t>(blockIdx.x) * (kGThreads / kWave) + wave) * kGTokPerWave;
    if (tok0 >= T) return;  // whole waves: the reduction below is wave-local
    int64_t rows[kGTokPerWave];
#pragma unroll
    for (int t = 0; t < kGTokPerWave; ++t) rows[t] = tok0 + t < T ? tok0 + t : T - 1;
    double acc[kGTokPerWave][MC];
#pragma unroll
    for (int t = 0; t < kGTokPerWave; ++t)
#pragma unroll
        for (int j = 0; j < MC; ++j) acc[t][j] = 0.0;
#pragma unroll 1
    for (int c0 = lane * 8; c0 < d; c0 += kWave * 8) {
        float v[kGTokPerWave][8];
#pragma unroll
        for (int t = 0; t < kGTokPerWave; ++t) load8<BF16>(x, rows[t] * d + c0, v[t]);
#pragma unroll
        for (int j = 0; j < MC; ++j) {
            float mu[8], iv[8];
            const float4* pm = reinterpret_cast<const float4*>(coef + (static_cast<int64_t>(j) * 2) * d + c0);
            const float4* pi = reinterpret_cast<const float4*>(coef + (static_cast<int64_t>(j) * 2 + 1) * d + c0);
            *reinterpret_cast<float4*>(&mu[0]) = pm[0];
            *reinterpret_cast<float4*>(&mu[4]) = pm[1];
            *reinterpret_cast<float4*>(&iv[0]) = pi[0];
            *reinterpret_cast<float4*>(&iv[4]) = pi[1];
#pragma unroll
            for (int t = 0; t < kGTokPerWave; ++t) {
                float part = 0.0f;
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const float dv = v[t][i] - mu[i];
                    part += dv * dv * iv[i];
                }
                acc[t][j] += static_cast<double>(part);
            }
        }
    }
    // lane partials -> per (token, component) sums: a fixed butterfly, the same in every lane
#pragma unroll
    for (int t = 0; t < kGTokPerWave; ++t)
#pragma unroll
        for (int j = 0; j < MC; ++j) acc[t][j] = wave_sum_u(acc[t][j]);
    if (lane >= kGTokPerWave) return;
    const int t = lane;
    if (tok0 + t >= T) return;
    double q[MC];
#pragma unroll
    for (int j = 0; j < MC; ++j) q[j] = t == 0 ? acc[0][j] : acc[kGTokPerWave - 1][j];
    double ll[MC];
    for (int j = 0; j < MC; ++j) {
        double slv = 0.0;
        for (int b = 0; b < n_part; ++b) slv += cst[j * kGMaxParts + b];
        ll[j] = -0.5 * (slv + q[j]);
    }
    // mixture weights pi_mc = N_mc / sum_c N_mc (uniform when the modality has no count)
#pragma unroll
    for (int m = 0; m < 2; ++m) {
        double tot = 0.0;
#pragma unroll
        for (int c = 0; c < K; ++c) tot += static_cast<double>(gn[m * K + c]);
#pragma unroll
        for (int c = 0; c < K; ++c)
            ll[m * K + c] += tot > 0.0 ? log(static_cast<double>(gn[m * K + c]) / tot) : -log(static_cast<double>(K));
    }
    const int64_t j = tok0 + t;
    if (mode == 0) {
        double lse[2];
#pragma unroll
        for (int m = 0; m < 2; ++m) {
            double mx = -INFINITY;
#pragma unroll
            for (int c = 0; c < K; ++c) mx = fmax(mx, ll[m * K + c]);
            double s = 0.0;
#pragma unroll
            for (int c = 0; c < K; ++c) s += exp(ll[m * K + c] - mx);
            lse[m] = mx + log(s);
        }
        const double sgn = (lse[0] - lse[1]) * inv_tau;  // M_vision = sigmoid(sgn)
        double mv, mt;
        if (sgn >= 0.0) {
            const double e = exp(-sgn);
            mv = 1.0 / (1.0 + e);
            mt = e / (1.0 + e);
        } else {
            const double e = exp(sgn);
            mv = e / (1.0 + e);
            mt = 1.0 / (1.0 + e);
        }
        M[j * 2] = static_cast<float>(mv);
        M[j * 2 + 1] = static_cast<float>(mt);
    } else {
        const int m = mid[j] ? 1 : 0;
        double mx = -INFINITY;
#pragma unroll
        for (int c = 0; c < K; ++c) mx = fmax(mx, ll[m * K + c]);
        double e[K], s = 0.0;
#pragma unroll
        for (int c = 0; c < K; ++c) {
            e[c] = exp(ll[m * K + c] - mx);
            s += e[c];
        }
#pragma unroll
        for (int c = 0; c < K; ++c) resp[j * K + c] = static_cast<float>(e[c] / s);
    }
}

// Weighted sums of one modality (blockIdx.z) over a chunk of tokens: 4 waves
// split the rows, each lane owns 4 columns; fixed-order tree over the waves.
template <bool BF16, int K>
__global__ void __launch_bounds__(256)
gmm_partial_kernel(const void* __restrict__ x, int64_t T, int d, const uint8_t* __restrict__ mid,
                   const float* __restrict__ resp, const float* __restrict__ gn, const float* __restrict__ gsmu,
                   double* __restrict__ wsum, double* __restrict__ s1g, double* __restrict__ s2g,
                   double* __restrict__ n_old) {
    constexpr int NV = K * 4 * 2;
    __shared__ double red[2][kWave][NV];
    __shared__ double wred[4][K];
    const int wave = threadIdx.x / kWave;
    const int lane = lane_id();
    const int m = blockIdx.z;
    const int64_t chunk = blockIdx.x;
    const int col0 = blockIdx.y * kGPartCols + lane * 4;
    const bool active = col0 < d;
    if (chunk == 0 && blockIdx.y == 0 && m == 0 && threadIdx.x < 2 * K) n_old[threadIdx.x] = gn[threadIdx.x];
    double sh[K][4], s1[K][4], s2[K][4], ws[K];
#pragma unroll
    for (int c = 0; c < K; ++c) {
        const double n = gn[m * K + c];
        ws[c] = 0.0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            sh[c][i] = (active && n > 0.0) ? static_cast<double>(gsmu[static_cast<int64_t>(m * K + c) * d + col0 + i]) / n : 0.0;
            s1[c][i] = s2[c][i] = 0.0;
        }
    }
    const int64_t r0 = chunk * kGChunk;
    const int64_t r1 = r0 + kGChunk < T ? r0 + kGChunk : T;
#pragma unroll 4
    for (int64_t r = r0 + wave; r < r1; r += 4) {
        if ((mid[r] ? 1 : 0) != m) continue;
        double w[K];
#pragma unroll
        for (int c = 0; c < K; ++c) {
            w[c] = static_cast<double>(resp[r * K + c]);
            ws[c] += w[c];
        }
        if (!active) continue;
        float v[4];
        if constexpr (BF16) {
            const uint2 q = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(x) + r * d + col0);
            v[0] = __uint_as_float(q.x << 16);
            v[1] = __uint_as_float(q.x & 0xffff0000u);
            v[2] = __uint_as_float(q.y << 16);
            v[3] = __uint_as_float(q.y & 0xffff0000u);
        } else {
            const float4 q = *reinterpret_cast<const float4*>(static_cast<const float*>(x) + r * d + col0);
            v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
        }
#pragma unroll
        for (int c = 0; c < K; ++c)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const double y = static_cast<double>(v[i]) - sh[c][i];
                const double wy = w[c] * y;
                s1[c][i] += wy;
                s2[c][i] = fma(wy, y, s2[c][i]);
            }
    }
    auto put = [&](int slot) {
#pragma unroll
        for (int c = 0; c < K; ++c)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                red[slot][lane][(c * 4 + i) * 2] = s1[c][i];
                red[slot][lane][(c * 4 + i) * 2 + 1] = s2[c][i];
            }
    };
    auto add = [&](int slot) {
#pragma unroll
        for (int c = 0; c < K; ++c)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                s1[c][i] += red[slot][lane][(c * 4 + i) * 2];
                s2[c][i] += red[slot][lane][(c * 4 + i) * 2 + 1];
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
            for (int c = 0; c < K; ++c)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int64_t o = (chunk * 2 * K + m * K + c) * d + col0 + i;
                    s1g[o] = s1[c][i];
                    s2g[o] = s2[c][i];
                }
        }
    }
    // weight sums: every lane of a wave saw the same rows; lane 0 reports
    if (lane == 0) {
#pragma unroll
        for (int c = 0; c < K; ++c) wred[wave][c] = ws[c];
    }
    __syncthreads();
    if (blockIdx.y == 0 && threadIdx.x < K)
        wsum[chunk * 2 * K + m * K + threadIdx.x] = (wred[0][threadIdx.x] + wred[2][threadIdx.x]) +
                                                    (wred[1][threadIdx.x] + wred[3][threadIdx.x]);
}

__global__ void gmm_merge_kernel(int d, int K, int64_t nchunk, const double* __restrict__ wsum,
                                 const double* __restrict__ s1g, const double* __restrict__ s2g,
                                 const double* __restrict__ n_old, float beta, float* __restrict__ gn,
                                 float* __restrict__ gsmu, float* __restrict__ gssig) {
    const int mc = blockIdx.y;
    const int col = blockIdx.x * blockDim.x + threadIdx.x;
    if (col >= d) return;
    double n = 0.0, S1 = 0.0, S2 = 0.0;
    constexpr int B = 8;  // chunk loads in flight; the sums still run in chunk order
    for (int64_t c0 = 0; c0 < nchunk; c0 += B) {
        double vn[B], v1[B], v2[B];
#pragma unroll
        for (int q = 0; q < B; ++q) {
            const int64_t ch = c0 + q < nchunk ? c0 + q : c0;
            vn[q] = wsum[ch * 2 * K + mc];
            v1[q] = s1g[(ch * 2 * K + mc) * d + col];
            v2[q] = s2g[(ch * 2 * K + mc) * d + col];
        }
#pragma unroll
        for (int q = 0; q < B; ++q)
            if (c0 + q < nchunk) {
                n += vn[q];
                S1 += v1[q];
                S2 += v2[q];
            }
    }
    const double nprev = n_old[mc];
    const int64_t o = static_cast<int64_t>(mc) * d + col;
    const double smu_old = gsmu[o];
    const double ssig_old = gssig[o];
    const double shift = nprev > 0.0 ? smu_old / nprev : 0.0;
    const double b = static_cast<double>(beta);
    double mean_T = 0.0, m2_T = 0.0, cross = 0.0;
    if (n > 0.0) {
        mean_T = shift + S1 / n;
        m2_T = S2 - S1 * (S1 / n);
        if (m2_T < 0.0) m2_T = 0.0;
        if (nprev > 0.0) {
            const double dm = mean_T - shift;
            cross = dm * dm * (b * nprev * n) / (b * nprev + n);
        }
    }
    gsmu[o] = static_cast<float>(b * smu_old + n * mean_T);
    gssig[o] = static_cast<float>(b * ssig_old + m2_T + cross);
    if (col == 0) gn[mc] = static_cast<float>(b * nprev + n);
}

template <bool BF16, int K>
hipError_t gmm_run(const void* x, int64_t T, int d, const uint8_t* mid, float* gn, float* gsmu, float* gssig,
                   int update, float beta, float tau, float var_floor, float* M, float* resp_out, const GmmWs& w,
                   hipStream_t stream) {
    hipError_t err;
    const int n_part = static_cast<int>(ceil_div(d, kGPrepThreads));
    const dim3 pgrid(static_cast<unsigned>(n_part), 2 * K);
    const int64_t tok_per_block = static_cast<int64_t>(kGThreads / kWave) * kGTokPerWave;
    const dim3 lgrid(static_cast<unsigned>(ceil_div(T, tok_per_block)));
    const double t = tau > 0.0f ? static_cast<double>(tau) : 0.5 * d;
    float* resp = resp_out != nullptr ? resp_out : w.resp;
    if (update || resp_out != nullptr) {
        hipLaunchKernelGGL(gmm_prep_kernel, pgrid, dim3(kGPrepThreads), 0, stream, d, K, gn, gsmu, gssig,
                           var_floor, w.coef, w.cst);
        if ((err = hipGetLastError()) != hipSuccess) return err;
        hipLaunchKernelGGL((gmm_loglik_kernel<BF16, K>), lgrid, dim3(kGThreads), 0, stream, x, T, d, mid, w.coef,
                           w.cst, n_part, gn, 1.0 / t, 1, M, resp);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    if (update) {
        const int64_t nchunk = ceil_div(T, kGChunk);
        const dim3 grid(static_cast<unsigned>(nchunk), static_cast<unsigned>(ceil_div(d, kGPartCols)), 2);
        hipLaunchKernelGGL((gmm_partial_kernel<BF16, K>), grid, dim3(256), 0, stream, x, T, d, mid, resp, gn, gsmu,
                           w.wsum, w.s1, w.s2, w.n_old);
        if ((err = hipGetLastError()) != hipSuccess) return err;
        hipLaunchKernelGGL(gmm_merge_kernel, dim3(static_cast<unsigned>(ceil_div(d, 256)), 2 * K), dim3(256), 0,
                           stream, d, K, nchunk, w.wsum, w.s1, w.s2, w.n_old, beta, gn, gsmu, gssig);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    hipLaunchKernelGGL(gmm_prep_kernel, pgrid, dim3(kGPrepThreads), 0, stream, d, K, gn, gsmu, gssig, var_floor,
                       w.coef, w.cst);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    hipLaunchKernelGGL((gmm_loglik_kernel<BF16, K>), lgrid, dim3(kGThreads), 0, stream, x, T, d, mid, w.coef, w.cst,
                       n_part, gn, 1.0 / t, 0, M, resp);
    return hipGetLastError();
}

template <bool BF16>
hipError_t gmm_dispatch(int K, const void* x, int64_t T, int d, const uint8_t* mid, float* gn, float* gsmu,
                        float* gssig, int update, float beta, float tau, float var_floor, float* M, float* resp,
                        const GmmWs& w, hipStream_t s) {
    switch (K) {
        case 1: return gmm_run<BF16, 1>(x, T, d, mid, gn, gsmu, gssig, update, beta, tau, var_floor, M, resp, w, s);
        case 2: return gmm_run<BF16, 2>(x, T, d, mid, gn, gsmu, gssig, update, beta, tau, var_floor, M, resp, w, s);
        case 3: return gmm_run<BF16, 3>(x, T, d, mid, gn, gsmu, gssig, update, beta, tau, var_floor, M, resp, w, s);
        default: return gmm_run<BF16, 4>(x, T, d, mid, gn, gsmu, gssig, update, beta, tau, var_floor, M, resp, w, s);
    }
}

}  // namespace

size_t gmm_workspace_bytes(int64_t T, int d, int K) {
    const int64_t nchunk = ceil_div(T, kGChunk);
    return align_up(sizeof(float) * 2 * K * 2 * d, 256) + align_up(sizeof(double) * 2 * K * kGMaxParts, 256) + 256 +
           align_up(sizeof(float) * T * K, 256) + align_up(sizeof(double) * nchunk * 2 * K, 256) +
           2 * align_up(sizeof(double) * nchunk * 2 * K * d, 256);
}

hipError_t launch_gmm(const void* x, int x_dtype, int64_t T, int d, int K, const uint8_t* modality_id, float* gmm_n,
                      float* gmm_smu, float* gmm_ssig, int update, float beta, float tau, float var_floor, float* M,
                      float* resp, void* ws, hipStream_t stream) {
    const GmmWs w = gmm_carve(ws, T, d, K);
    if (x_dtype == 1)
        return gmm_dispatch<true>(K, x, T, d, modality_id, gmm_n, gmm_smu, gmm_ssig, update, beta, tau, var_floor, M,
                                  resp, w, stream);
    return gmm_dispatch<false>(K, x, T, d, modality_id, gmm_n, gmm_smu, gmm_ssig, update, beta, tau, var_floor, M,
                               resp, w, stream);
}

}  // namespace smoes
