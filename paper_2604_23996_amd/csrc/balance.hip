// Momentum-adaptive binning (Sec. 3.3, Eq. 10-11), the bin-level load
// balance loss with its logit gradient (Sec. 3.5, Eq. 16) and the modality
// specialization index (Sec. 4.1, Eq. 18-19) of one layer, from one batch's
// routing.
//
//   bal_partial : per 256-token chunk: per token the bins its top-k reaches
//                 (kept for the gradient), counts C[m][e] of hard label m with
//                 e in the token's top-k and tokens routed to each bin (wave
//                 ballots and popcounts, summed over the four waves in wave
//                 order: no atomics), and per expert the gate mass over the tokens
//                 routed to its bin (fp64, fixed order).
//   bal_finalize: one block; sums the chunk partials in chunk order, then
//                 L_bal = sum_e N_B (n_e / T_k)(S_e / T_k), the gradient
//                 coefficients N_B n_e / T_k^2, the EMA of the expert loads
//                 (fp64, products rounded before the sum), f_spec, the stable
//                 ascending rank of f_spec -> next bin map, and MSI.
//   bal_grad    : one wave per token: dz = scale * g * (dg - sum_e g dg) with
//                 dg_e = coef_e for experts whose bin the token was routed to
//                 (the token's bin mask from bal_partial).
// Readings (the paper leaves them open): "tokens in bin B_k" are the tokens
// routed to bin k; f_e = n_e / T_k, P_e = mean gate of e over them; the top-k
// counts are constants for the gradient; f_spec = 1/2 for an expert with no
// load; MSI counts an expert no token reaches as unspecialised.
#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

constexpr int kBalChunk = 256;    // tokens per partial block
constexpr int kBalThreads = 256;  // 4 waves
constexpr int kBalWaves = kBalThreads / kWave;
static_assert(kBalWaves == 4, "per-wave counts are summed as four terms");

struct BalWs {
    int32_t* cnt;    // [nchunk][2][E]
    int32_t* tk;     // [nchunk][n_bins]
    double* mass;    // [nchunk][E]
    double* coef;    // [E]
    uint64_t* mask;  // [T]: bins each token's top-k reaches
};

BalWs carve(void* ws, int64_t nchunk, int E, int n_bins) {
    char* p = static_cast<char*>(ws);
    BalWs w;
    w.cnt = reinterpret_cast<int32_t*>(p);
    p += align_up(sizeof(int32_t) * nchunk * 2 * E, 256);
    w.tk = reinterpret_cast<int32_t*>(p);
    p += align_up(sizeof(int32_t) * nchunk * n_bins, 256);
    w.mass = reinterpret_cast<double*>(p);
    p += align_up(sizeof(double) * nchunk * E, 256);
    w.coef = reinterpret_cast<double*>(p);
    p += align_up(sizeof(double) * E, 256);
    w.mask = reinterpret_cast<uint64_t*>(p);
    return w;
}

// Phase 1, one thread per token of the chunk: its top-k row (k loads in
// flight), the bins it reaches as a bit mask (n_bins <= 64, bin map in LDS);
// counts by label and expert and tokens per bin from wave ballots (lane t of a
// wave ends with the count of expert e0 + t, or of bin t) and popcounts, one
// LDS row per wave. Phase 2, one wave per token with lanes over experts: gate
// mass of each expert over the tokens routed to its bin (fp64, fixed order).
__global__ void __launch_bounds__(kBalThreads)
bal_partial_kernel(const float* __restrict__ probs, const int32_t* __restrict__ idx,
                   const uint8_t* __restrict__ mid, int64_t T, int E, int k, const int32_t* __restrict__ e2b,
                   int n_bins, int32_t* __restrict__ cnt_out, int32_t* __restrict__ tk_out,
                   double* __restrict__ mass_out, uint64_t* __restrict__ mask_out) {
    __shared__ int32_t cnt[kBalWaves][2][256];
    __shared__ int32_t tk[kBalWaves][64];
    __shared__ int32_t bin_s[256];
    __shared__ uint64_t mask_s[kBalChunk];
    __shared__ double mass[kBalWaves][256];
    const int wave = threadIdx.x / kWave, lane = lane_id();
    for (int e = threadIdx.x; e < E; e += kBalThreads) bin_s[e] = e2b[e];
    __syncthreads();
    const int64_t j0 = static_cast<int64_t>(blockIdx.x) * kBalChunk;
    const int n = static_cast<int>(T - j0 < kBalChunk ? T - j0 : kBalChunk);
    {
        const int r = threadIdx.x;
        uint64_t m = 0;
        uint64_t b0 = 0, b1 = 0, b2 = 0, b3 = 0;  // experts chosen: bit e & 63 of word e >> 6
        int lab = 0;
        if (r < n) {
            const int64_t j = j0 + r;
            int ex[SMOES_K_MAX_DEV];
#pragma unroll
            for (int s = 0; s < SMOES_K_MAX_DEV; ++s) ex[s] = s < k ? idx[j * k + s] : 0;
            lab = mid[j] ? 1 : 0;
#pragma unroll
            for (int s = 0; s < SMOES_K_MAX_DEV; ++s) {
                if (s < k) {
                    const int e = ex[s];
                    m |= 1ull << bin_s[e];
                    const uint64_t bit = 1ull << (e & 63);
                    const int blk = e >> 6;
                    b0 |= blk == 0 ? bit : 0ull;
                    b1 |= blk == 1 ? bit : 0ull;
                    b2 |= blk == 2 ? bit : 0ull;
                    b3 |= blk == 3 ? bit : 0ull;
                }
            }
            mask_out[j] = m;
        }
        mask_s[r] = m;
        const uint64_t eb[4] = {b0, b1, b2, b3};
        const uint32_t l1 = static_cast<uint32_t>(lab), l0 = l1 ^ 1u;
        // lane t ends with the counts of expert e0 + t (experts past E are never chosen)
#pragma unroll
        for (int blk = 0; blk < 4; ++blk) {
            const int e0 = blk * 64;
            if (e0 >= E) break;
            const uint32_t lo = static_cast<uint32_t>(eb[blk]), hi = static_cast<uint32_t>(eb[blk] >> 32);
            int c0 = 0, c1 = 0;
#pragma unroll
            for (int t = 0; t < 64; ++t) {
                const uint32_t bit = t < 32 ? (lo >> t) & 1u : (hi >> (t - 32)) & 1u;
                const int n0 = __popcll(__ballot(static_cast<int>(bit & l0)));  // every lane takes part
                const int n1 = __popcll(__ballot(static_cast<int>(bit & l1)));
                c0 = lane == t ? n0 : c0;
                c1 = lane == t ? n1 : c1;
            }
            if (e0 + lane < E) {
                cnt[wave][0][e0 + lane] = c0;
                cnt[wave][1][e0 + lane] = c1;
            }
        }
        // lane b ends with the tokens routed to bin b (bins past n_bins are never reached)
        const uint32_t mlo = static_cast<uint32_t>(m), mhi = static_cast<uint32_t>(m >> 32);
        int cb = 0;
#pragma unroll
        for (int b = 0; b < 64; ++b) {
            const uint32_t bit = b < 32 ? (mlo >> b) & 1u : (mhi >> (b - 32)) & 1u;
            const int nb = __popcll(__ballot(static_cast<int>(bit)));  // every lane takes part
            cb = lane == b ? nb : cb;
        }
        if (lane < n_bins) tk[wave][lane] = cb;
    }
    __syncthreads();
    int bin_of[4];
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int e = lane + q * kWave;
        bin_of[q] = e < E ? bin_s[e] : 0;
    }
#pragma unroll 4
    for (int r = wave; r < n; r += kBalWaves) {
        const uint64_t bins = mask_s[r];
        const float* row = probs + (j0 + r) * E;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = lane + q * kWave;
            if (e < E && ((bins >> bin_of[q]) & 1ull)) acc[q] += static_cast<double>(row[e]);
        }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) mass[wave][lane + q * kWave] = acc[q];
    __syncthreads();
    int32_t* co = cnt_out + static_cast<int64_t>(blockIdx.x) * 2 * E;
    for (int i = threadIdx.x; i < 2 * E; i += kBalThreads) {
        const int l = i / E, e = i % E;
        co[i] = (cnt[0][l][e] + cnt[1][l][e]) + (cnt[2][l][e] + cnt[3][l][e]);
    }
    if (threadIdx.x < n_bins)
        tk_out[static_cast<int64_t>(blockIdx.x) * n_bins + threadIdx.x] =
            (tk[0][threadIdx.x] + tk[1][threadIdx.x]) + (tk[2][threadIdx.x] + tk[3][threadIdx.x]);
    for (int e = threadIdx.x; e < E; e += kBalThreads) {
        double sum = 0.0;
        for (int w = 0; w < kBalWaves; ++w) sum += mass[w][e];  // wave order
        mass_out[static_cast<int64_t>(blockIdx.x) * E + e] = sum;
    }
}

// Fixed-order sum of one double per thread over the block (256 threads).
__device__ __forceinline__ double block_sum_f64(double v, double* sh) {
    sh[threadIdx.x] = v;
    __syncthreads();
    for (int s = kBalThreads / 2; s > 0; s >>= 1) {
        if (threadIdx.x < s) sh[threadIdx.x] += sh[threadIdx.x + s];
        __syncthreads();
    }
    const double r = sh[0];
    __syncthreads();
    return r;
}

__global__ void __launch_bounds__(kBalThreads)
bal_finalize_kernel(int64_t nchunk, int E, int n_bins, const int32_t* __restrict__ cnt_in,
                    const int32_t* __restrict__ tk_in, const double* __restrict__ mass_in, double beta,
                    double* __restrict__ load_ema, int32_t* __restrict__ counts, double* __restrict__ fspec_out,
                    int32_t* __restrict__ e2b_next, const int32_t* __restrict__ e2b, float* __restrict__ bal_loss,
                    float* __restrict__ msi_out, double* __restrict__ coef) {
    __shared__ int32_t tk[64];
    __shared__ double fs[256];
    __shared__ double red[kBalThreads];
    const int e = threadIdx.x;  // E <= 256 = blockDim
    const int NB = E / n_bins;
    constexpr int B = 8;  // chunk loads in flight; the sums still run in chunk order
    if (e < n_bins) {
        int32_t s = 0;
        for (int64_t c0 = 0; c0 < nchunk; c0 += B) {
            int32_t v[B];
#pragma unroll
            for (int q = 0; q < B; ++q) v[q] = c0 + q < nchunk ? tk_in[(c0 + q) * n_bins + e] : 0;
#pragma unroll
            for (int q = 0; q < B; ++q) s += v[q];
        }
        tk[e] = s;
    }
    int32_t cv = 0, ct = 0;
    double S = 0.0;
    if (e < E) {
        for (int64_t c0 = 0; c0 < nchunk; c0 += B) {
            int32_t vv[B], vt[B];
            double vm[B];
#pragma unroll
            for (int q = 0; q < B; ++q) {
                const int64_t c = c0 + q < nchunk ? c0 + q : c0;
                vv[q] = cnt_in[c * 2 * E + e];
                vt[q] = cnt_in[c * 2 * E + E + e];
                vm[q] = mass_in[c * E + e];
            }
#pragma unroll
            for (int q = 0; q < B; ++q)
                if (c0 + q < nchunk) {
                    cv += vv[q];
                    ct += vt[q];
                    S += vm[q];
                }
        }
    }
    __syncthreads();
    // Eq. 16 and its gradient coefficients
    double term = 0.0;
    if (e < E) {
        const int32_t Tk = tk[e2b[e]];
        const double n_e = static_cast<double>(cv) + static_cast<double>(ct);
        double c = 0.0;
        if (Tk > 0) {
            const double t = static_cast<double>(Tk);
            term = NB * (n_e / t) * (S / t);
            c = NB * (n_e / t) / t;
        }
        coef[e] = c;
        if (counts != nullptr) {
            counts[e] = cv;
            counts[E + e] = ct;
        }
    }
    const double L = block_sum_f64(term, red);
    if (e == 0 && bal_loss != nullptr) bal_loss[0] = static_cast<float>(L);
    // Eq. 10: EMA of the expert loads (rows: vision, text), products rounded before the sum
    double f = 0.5;
    if (e < E) {
        double lv = cv, lt = ct;
        if (load_ema != nullptr) {
            const double a = 1.0 - beta;
            lv = __dadd_rn(__dmul_rn(beta, load_ema[e]), __dmul_rn(a, static_cast<double>(cv)));
            lt = __dadd_rn(__dmul_rn(beta, load_ema[E + e]), __dmul_rn(a, static_cast<double>(ct)));
            load_ema[e] = lv;
            load_ema[E + e] = lt;
        }
        const double tot = __dadd_rn(lt, lv);
        if (tot > 0.0) f = __ddiv_rn(lt, tot);  // Eq. 11
        fs[e] = f;
        if (fspec_out != nullptr) fspec_out[e] = f;
    }
    __syncthreads();
    // stable ascending rank -> consecutive bins of N_B
    if (e < E && e2b_next != nullptr) {
        int rank = 0;
        for (int q = 0; q < E; ++q) rank += (fs[q] < f || (fs[q] == f && q < e)) ? 1 : 0;
        e2b_next[e] = rank / NB;
    }
    // Eq. 18-19 on this batch's counts
    const double tot_v = block_sum_f64(e < E ? static_cast<double>(cv) : 0.0, red);
    const double tot_t = block_sum_f64(e < E ? static_cast<double>(ct) : 0.0, red);
    double dev = 0.0;
    if (e < E) {
        const double nv = tot_v > 0.0 ? cv / tot_v : 0.0;
        const double nt = tot_t > 0.0 ? ct / tot_t : 0.0;
        const double den = nt + nv;
        const double c_text = den > 0.0 ? nt / den : 0.5;
        dev = 2.0 * fabs(c_text - 0.5);
    }
    const double msi = block_sum_f64(dev, red) / E;
    if (e == 0 && msi_out != nullptr) msi_out[0] = static_cast<float>(msi);
}

__global__ void __launch_bounds__(kBalThreads)
bal_grad_kernel(const float* __restrict__ probs, const uint64_t* __restrict__ mask, int64_t T, int E,
                const int32_t* __restrict__ e2b, const double* __restrict__ coef, double scale, int accumulate,
                float* __restrict__ dlogits) {
    const int wave = threadIdx.x / kWave, lane = lane_id();
    double cf[4];
    int bin_of[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int e = lane + q * kWave;
        cf[q] = e < E ? coef[e] : 0.0;
        bin_of[q] = e < E ? e2b[e] : 0;
    }
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBalWaves;
    for (int64_t j = static_cast<int64_t>(blockIdx.x) * kBalWaves + wave; j < T; j += stride) {
        const uint64_t bins = mask[j];
        double g[4], dg[4], part = 0.0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = lane + q * kWave;
            g[q] = e < E ? static_cast<double>(probs[j * E + e]) : 0.0;
            dg[q] = (e < E && ((bins >> bin_of[q]) & 1ull)) ? cf[q] : 0.0;
            part += g[q] * dg[q];
        }
        const double s = wave_sum_u(part);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = lane + q * kWave;
            if (e < E) {
                float v = static_cast<float>(scale * g[q] * (dg[q] - s));
                if (accumulate) v += dlogits[j * E + e];
                dlogits[j * E + e] = v;
            }
        }
    }
}

}  // namespace

size_t binning_workspace_bytes(int64_t T, int E, int n_bins) {
    const int64_t nchunk = ceil_div(T, kBalChunk) > 0 ? ceil_div(T, kBalChunk) : 1;
    return align_up(sizeof(int32_t) * nchunk * 2 * E, 256) + align_up(sizeof(int32_t) * nchunk * n_bins, 256) +
           align_up(sizeof(double) * nchunk * E, 256) + align_up(sizeof(double) * E, 256) +
           align_up(sizeof(uint64_t) * (T > 0 ? T : 1), 256);
}

hipError_t launch_binning(const float* probs, const int32_t* topk_idx, const uint8_t* modality_id, int64_t T,
                          int E, int k, const int32_t* expert_to_bin, int n_bins, float beta, double* load_ema,
                          int32_t* counts, double* f_spec, int32_t* expert_to_bin_next, float grad_scale,
                          float* bal_loss, float* dlogits, int accumulate, float* msi, void* ws,
                          hipStream_t stream) {
    const int64_t nchunk = ceil_div(T, kBalChunk);
    BalWs w = carve(ws, nchunk > 0 ? nchunk : 1, E, n_bins);
    hipError_t err;
    if (nchunk > 0) {
        hipLaunchKernelGGL(bal_partial_kernel, dim3(static_cast<unsigned>(nchunk)), dim3(kBalThreads), 0, stream,
                           probs, topk_idx, modality_id, T, E, k, expert_to_bin, n_bins, w.cnt, w.tk, w.mass,
                           w.mask);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    const double b = static_cast<double>(beta);
    hipLaunchKernelGGL(bal_finalize_kernel, dim3(1), dim3(kBalThreads), 0, stream, nchunk, E, n_bins, w.cnt,
                       w.tk, w.mass, b, load_ema, counts, f_spec, expert_to_bin_next, expert_to_bin, bal_loss,
                       msi, w.coef);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    if (dlogits != nullptr && T > 0) {
        int64_t blocks = ceil_div(T, kBalWaves);
        if (blocks > 4096) blocks = 4096;
        hipLaunchKernelGGL(bal_grad_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kBalThreads), 0, stream,
                           probs, w.mask, T, E, expert_to_bin, w.coef, static_cast<double>(grad_scale),
                           accumulate, dlogits);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    return hipSuccess;
}

}  // namespace smoes
