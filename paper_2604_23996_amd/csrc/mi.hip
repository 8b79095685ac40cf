// Inter-bin mutual information between the soft modality score and expert
// bins (Sec. 3.3-3.4, Eq. 12-15) and its gradient with respect to the router
// logits.
//
// Eq. 12 is linear in the gate, so the per-sample work reduces to the
// per-expert, per-modality masses A[m][e] = sum_j M_jm g_je and the score
// totals W[m] = sum_j M_jm; bins only enter in the small finalize step.
//   mi_partial : (sample, chunk) blocks; threads own expert columns, rows are
//                split over row groups; fp64 sums, fixed-order LDS reduction.
//   mi_finalize: one block per sample; chunk partials in chunk order, bin
//                sums in ascending expert order, then S-bar (Eq. 12), the joint
//                (Eq. 13), I_i (Eq. 14) and the gradient coefficients
//                c[m][k] = (log r_mk - I_i) / (N_B W_m Z); the loss (Eq. 15)
//                is summed in sample order by the next kernel.
//   mi_grad    : one wave per token; G_k = bin masses of the token,
//                h_k = sum_m M_jm c[m][k], dlogit_e = s g_e (h_bin(e) - sum_k G_k h_k)
//                with s = -grad_scale / N_batch.
// No atomics: every result is reproducible bit for bit.
#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

constexpr int kMiThreads = 256;
constexpr int kRowsPerChunk = 32;

struct MiWs {
    double* part;     // [n_batch * C][2E + 2]
    double* coef;     // [n_batch][2][B]
    double* mi;       // [n_batch]
    int32_t* members; // [B][N_B]
    int C;
};

int mi_chunks(int64_t T, int n_batch) {
    int64_t c = ceil_div(T, static_cast<int64_t>(n_batch) * kRowsPerChunk);
    if (c < 1) c = 1;
    if (c > 1024) c = 1024;
    return static_cast<int>(c);
}

MiWs carve(void* ws, int64_t T, int E, int n_batch, int n_bins) {
    MiWs w;
    w.C = mi_chunks(T, n_batch);
    char* p = static_cast<char*>(ws);
    w.part = reinterpret_cast<double*>(p);
    p += align_up(sizeof(double) * static_cast<size_t>(n_batch) * w.C * (2 * E + 2), 256);
    w.coef = reinterpret_cast<double*>(p);
    p += align_up(sizeof(double) * static_cast<size_t>(n_batch) * 2 * n_bins, 256);
    w.mi = reinterpret_cast<double*>(p);
    p += align_up(sizeof(double) * static_cast<size_t>(n_batch), 256);
    w.members = reinterpret_cast<int32_t*>(p);
    return w;
}

__device__ __forceinline__ void sample_range(const int32_t* off, int64_t T, int i, int64_t& a, int64_t& b) {
    if (off == nullptr) {
        a = 0;
        b = T;
    } else {
        a = off[i];
        b = off[i + 1];
    }
}

__global__ void __launch_bounds__(kMiThreads)
mi_partial_kernel(const float* __restrict__ probs, const float* __restrict__ M, int64_t T, int E,
                  const int32_t* __restrict__ off, int C, double* __restrict__ part) {
    __shared__ double red[kMiThreads][2];
    __shared__ double wred[kMiThreads][2];
    const int i = blockIdx.y;
    const int c = blockIdx.x;
    const int EP = static_cast<int>(ceil_div(E, kWave) * kWave);
    const int RG = kMiThreads / EP;  // row groups (>= 1 since E <= 256)
    const int rg = threadIdx.x / EP;
    const int e = threadIdx.x % EP;
    int64_t a, b;
    sample_range(off, T, i, a, b);
    const int64_t len = b - a;
    const int64_t L = ceil_div(len, C);
    const int64_t s0 = a + c * L;
    const int64_t s1 = s0 + L < b ? s0 + L : b;
    double a0 = 0.0, a1 = 0.0, w0 = 0.0, w1 = 0.0;
    // rows in order; the loads of 8 rows go out before their sums
    auto add = [&](float2 mj, float gv) {
        const double m0 = mj.x, m1 = mj.y;
        if (e < E) {
            a0 = fma(m0, static_cast<double>(gv), a0);
            a1 = fma(m1, static_cast<double>(gv), a1);
        }
        w0 += m0;
        w1 += m1;
    };
    if (rg < RG) {
        constexpr int U = 8;
        int64_t j = s0 + rg;
        for (; j + (U - 1) * RG < s1; j += U * RG) {
            float2 mj[U];
            float gv[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                mj[u] = *reinterpret_cast<const float2*>(M + 2 * (j + u * RG));
                gv[u] = e < E ? probs[(j + u * RG) * E + e] : 0.0f;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) add(mj[u], gv[u]);
        }
        for (; j < s1; j += RG) add(*reinterpret_cast<const float2*>(M + 2 * j), e < E ? probs[j * E + e] : 0.0f);
    }
    red[threadIdx.x][0] = a0;
    red[threadIdx.x][1] = a1;
    wred[threadIdx.x][0] = w0;
    wred[threadIdx.x][1] = w1;
    __syncthreads();
    double* out = part + (static_cast<int64_t>(i) * C + c) * (2 * E + 2);
    if (rg == 0) {
        double s_0 = 0.0, s_1 = 0.0;
        for (int r = 0; r < RG; ++r) {
            s_0 += red[r * EP + e][0];
            s_1 += red[r * EP + e][1];
        }
        if (e < E) {
            out[e] = s_0;
            out[E + e] = s_1;
        }
        if (e == 0) {
            double t0 = 0.0, t1 = 0.0;
            for (int r = 0; r < RG; ++r) {
                t0 += wred[r * EP][0];
                t1 += wred[r * EP][1];
            }
            out[2 * E] = t0;
            out[2 * E + 1] = t1;
        }
    }
}

// One block per sample. The chunk partials are summed by (expert, chunk
// group) threads in chunk order, the groups combined in a fixed order; then
// thread (m, k) owns one cell of the joint, and sums over cells are taken by
// every thread in the same fixed order from LDS.
__global__ void __launch_bounds__(kMiThreads)
mi_finalize_kernel(int64_t T, int E, const int32_t* __restrict__ off, int n_batch, int C,
                   const int32_t* __restrict__ e2b, int n_bins, const double* __restrict__ part,
                   double* __restrict__ coef, double* __restrict__ mi64, int32_t* __restrict__ members,
                   float* __restrict__ mi_per_sample) {
    __shared__ double red[kMiThreads][2];
    __shared__ double wred[kMiThreads][2];
    __shared__ double A[2][256];
    __shared__ double P[2][64];    // S-bar, then the joint P(m, k)
    __shared__ double term[2][64];
    __shared__ double Wm[2];
    __shared__ int32_t mem[256];
    __shared__ int32_t bin_s[256];
    const int NB = E / n_bins;
    const int tid = threadIdx.x;
    const int i = blockIdx.x;
    // chunk partials: thread (cg, e) sums chunks cg, cg + RG, ... in order
    const int EP = static_cast<int>(ceil_div(E, kWave) * kWave);
    const int RG = kMiThreads / EP;
    const int cg = tid / EP, e = tid % EP;
    const double* pi = part + static_cast<int64_t>(i) * C * (2 * E + 2);
    double s0 = 0.0, s1 = 0.0, w0 = 0.0, w1 = 0.0;
    auto add = [&](const double* pc) {
        if (e < E) {
            s0 += pc[e];
            s1 += pc[E + e];
        }
        if (e == 0) {
            w0 += pc[2 * E];
            w1 += pc[2 * E + 1];
        }
    };
    if (cg < RG) {
        // chunks in order; the loads of 16 chunks go out before their sums
        constexpr int U = 16;
        int c = cg;
        for (; c + (U - 1) * RG < C; c += U * RG) {
            double v[U][2];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const double* pc = pi + static_cast<int64_t>(c + u * RG) * (2 * E + 2);
                v[u][0] = e < E ? pc[e] : 0.0;
                v[u][1] = e < E ? pc[E + e] : 0.0;
            }
            if (e == 0) {
                double q[U][2];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const double* pc = pi + static_cast<int64_t>(c + u * RG) * (2 * E + 2);
                    q[u][0] = pc[2 * E];
                    q[u][1] = pc[2 * E + 1];
                }
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    w0 += q[u][0];
                    w1 += q[u][1];
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (e < E) {
                    s0 += v[u][0];
                    s1 += v[u][1];
                }
            }
        }
        for (; c < C; c += RG) add(pi + static_cast<int64_t>(c) * (2 * E + 2));
    }
    // bin member lists in ascending expert order: expert e takes slot
    // (its bin, the number of lower experts in that bin); slots no expert
    // takes stay -1 (violated precondition: a bin with fewer than N_B experts)
    for (int q = tid; q < E; q += blockDim.x) {
        bin_s[q] = e2b[q];
        mem[q] = -1;
    }
    __syncthreads();
    for (int q = tid; q < E; q += blockDim.x) {
        const int k = bin_s[q];
        int rank = 0;
        for (int e = 0; e < q; ++e) rank += bin_s[e] == k ? 1 : 0;
        if (k >= 0 && k < n_bins && rank < NB) mem[k * NB + rank] = q;
    }
    red[tid][0] = s0;
    red[tid][1] = s1;
    wred[tid][0] = w0;
    wred[tid][1] = w1;
    __syncthreads();
    if (cg == 0) {
        double a0 = 0.0, a1 = 0.0;
        for (int g = 0; g < RG; ++g) {
            a0 += red[g * EP + e][0];
            a1 += red[g * EP + e][1];
        }
        if (e < E) {
            A[0][e] = a0;
            A[1][e] = a1;
        }
        if (e == 0) {
            double t0 = 0.0, t1 = 0.0;
            for (int g = 0; g < RG; ++g) {
                t0 += wred[g * EP][0];
                t1 += wred[g * EP][1];
            }
            Wm[0] = t0;
            Wm[1] = t1;
        }
    }
    __syncthreads();
    if (i == 0)
        for (int q = tid; q < E; q += blockDim.x) members[q] = mem[q];
    int64_t a, b;
    sample_range(off, T, i, a, b);
    const bool cell = tid < 2 * n_bins;
    const int cm = cell ? tid / n_bins : 0, ck = cell ? tid % n_bins : 0;
    // Eq. 12: S-bar[m][k] = sum_{e in B_k} A[m][e] / (N_B W_m)
    if (cell) {
        double s = 0.0;
        for (int n = 0; n < NB; ++n) {
            const int ee = mem[ck * NB + n];
            if (ee >= 0) s += A[cm][ee];
        }
        P[cm][ck] = (b > a && Wm[cm] > 0.0) ? s / (static_cast<double>(NB) * Wm[cm]) : 0.0;
    }
    __syncthreads();
    // Eq. 13: normalise; marginals
    double Z = 0.0;
    for (int m = 0; m < 2; ++m)
        for (int k = 0; k < n_bins; ++k) Z += P[m][k];
    double pmk = 0.0, pm = 0.0, pk = 0.0;
    if (cell && Z > 0.0) {
        for (int k = 0; k < n_bins; ++k) pm += P[cm][k] / Z;
        pk = P[0][ck] / Z + P[1][ck] / Z;
        pmk = P[cm][ck] / Z;
    }
    // Eq. 14
    const double lr = (cell && pmk > 0.0) ? log(pmk / (pm * pk)) : 0.0;
    if (cell) term[cm][ck] = pmk > 0.0 ? pmk * lr : 0.0;
    __syncthreads();
    double I = 0.0;
    for (int m = 0; m < 2; ++m)
        for (int k = 0; k < n_bins; ++k) I += term[m][k];
    if (cell) {
        double cv = 0.0;
        if (Wm[cm] > 0.0 && pmk > 0.0) cv = (lr - I) / (static_cast<double>(NB) * Wm[cm] * Z);
        coef[(static_cast<int64_t>(i) * 2 + cm) * n_bins + ck] = cv;
    }
    if (tid == 0) {
        mi64[i] = I;
        mi_per_sample[i] = static_cast<float>(I);
    }
}

// Eq. 15 for one layer: loss = -(1 / N_batch) sum_i I_i, summed in sample order.
__device__ __forceinline__ void write_loss(const double* mi64, int n_batch, float* loss) {
    double s = 0.0;
    for (int i = 0; i < n_batch; ++i) s += mi64[i];
    loss[0] = static_cast<float>(-s / n_batch);
}

__global__ void mi_loss_kernel(const double* __restrict__ mi64, int n_batch, float* __restrict__ loss) {
    if (threadIdx.x == 0) write_loss(mi64, n_batch, loss);
}

__global__ void __launch_bounds__(kMiThreads)
mi_grad_kernel(const float* __restrict__ probs, const float* __restrict__ M, int64_t T, int E,
               const int32_t* __restrict__ off, int n_batch, const int32_t* __restrict__ e2b,
               int n_bins, const int32_t* __restrict__ members, const double* __restrict__ coef,
               double scale, float* __restrict__ dlogits, const double* __restrict__ mi64,
               float* __restrict__ loss) {
    if (blockIdx.x == 0 && threadIdx.x == 0) write_loss(mi64, n_batch, loss);
    constexpr int kWaves = kMiThreads / kWave;
    __shared__ float gl[kWaves][256];
    __shared__ double hl[kWaves][64];
    __shared__ int32_t mem[256];
    __shared__ int32_t bin[256];
    const int wave = threadIdx.x / kWave;
    const int lane = lane_id();
    const int NB = E / n_bins;
    for (int e = threadIdx.x; e < E; e += blockDim.x) {
        mem[e] = members[e];
        bin[e] = e2b[e];
    }
    const int QE = static_cast<int>(ceil_div(E, kWave));
    // block b takes tokens [j_lo, j_hi); wave w every kWaves-th of them from j_lo + w
    const int64_t per_block = ceil_div(ceil_div(T, gridDim.x), kWaves) * kWaves;
    const int64_t j_lo = static_cast<int64_t>(blockIdx.x) * per_block;
    const int64_t j_hi = j_lo + per_block < T ? j_lo + per_block : T;
    // sample of the wave's token: last i with off[i] <= j, found once and then
    // advanced as the tokens pass the ends of samples
    int si = 0;
    int64_t next = INT64_MAX;
    const int64_t jw = j_lo + wave;
    if (off != nullptr && jw < j_hi) {
        int lo = 0, hi = n_batch - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (off[mid] <= jw) lo = mid; else hi = mid - 1;
        }
        si = lo;
        next = si + 1 < n_batch ? off[si + 1] : INT64_MAX;
    }
    // the coefficients c[m][lane] of the wave's current sample, reloaded when the sample changes
    auto load_coef = [&](int i, double& c0, double& c1) {
        c0 = c1 = 0.0;
        if (lane < n_bins) {
            const double* cf = coef + static_cast<int64_t>(i) * 2 * n_bins;
            c0 = cf[lane];
            c1 = cf[n_bins + lane];
        }
    };
    double cf0, cf1;
    load_coef(si, cf0, cf1);
    // the gates and scores of token j (0 past the wave's range)
    auto load_tok = [&](int64_t j, float (&g)[4], float2& mj) {
        const bool ok = j < j_hi;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = lane + q * kWave;
            g[q] = ok && q < QE && e < E ? probs[j * E + e] : 0.0f;
        }
        mj = ok ? *reinterpret_cast<const float2*>(M + 2 * j) : make_float2(0.0f, 0.0f);
    };
    __syncthreads();  // mem, bin
    auto wave_lds_sync = [] {
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    };
    float gn[4];
    float2 mn;
    load_tok(jw, gn, mn);
    for (int64_t j = jw; j < j_hi; j += kWaves) {
        const float g[4] = {gn[0], gn[1], gn[2], gn[3]};
        const float2 mj = mn;
        load_tok(j + kWaves, gn, mn);  // the wave's next token, in flight during this one
        if (j >= next) {
            while (j >= next) {
                ++si;
                next = si + 1 < n_batch ? off[si + 1] : INT64_MAX;
            }
            load_coef(si, cf0, cf1);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = lane + q * kWave;
            if (q < QE && e < E) gl[wave][e] = g[q];
        }
        wave_lds_sync();
        double gh = 0.0;
        if (lane < n_bins) {
            double G = 0.0;
            for (int n = 0; n < NB; ++n) {
                const int e = mem[lane * NB + n];
                if (e >= 0) G += static_cast<double>(gl[wave][e]);
            }
            const double h = static_cast<double>(mj.x) * cf0 + static_cast<double>(mj.y) * cf1;
            hl[wave][lane] = h;
            gh = G * h;
        }
        gh = wave_sum(gh);
        wave_lds_sync();
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = lane + q * kWave;
            if (q < QE && e < E) {
                const double dv = scale * static_cast<double>(g[q]) * (hl[wave][bin[e]] - gh);
                dlogits[j * E + e] = static_cast<float>(dv);
            }
        }
        wave_lds_sync();
    }
}

}  // namespace

size_t mi_workspace_bytes(int64_t T, int E, int n_batch, int n_bins) {
    const int C = mi_chunks(T, n_batch);
    return align_up(sizeof(double) * static_cast<size_t>(n_batch) * C * (2 * E + 2), 256) +
           align_up(sizeof(double) * static_cast<size_t>(n_batch) * 2 * n_bins, 256) +
           align_up(sizeof(double) * static_cast<size_t>(n_batch), 256) +
           align_up(sizeof(int32_t) * static_cast<size_t>(E), 256);
}

hipError_t launch_mi(const float* probs, const float* M, int64_t T, int E,
                     const int32_t* sample_offsets, int n_batch, const int32_t* expert_to_bin,
                     int n_bins, float grad_scale, float* mi_per_sample, float* loss,
                     float* dlogits, void* ws, hipStream_t stream) {
    MiWs w = carve(ws, T, E, n_batch, n_bins);
    hipError_t err;
    hipLaunchKernelGGL(mi_partial_kernel, dim3(w.C, n_batch), dim3(kMiThreads), 0, stream, probs, M,
                       T, E, sample_offsets, w.C, w.part);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    hipLaunchKernelGGL(mi_finalize_kernel, dim3(n_batch), dim3(kMiThreads), 0, stream, T, E,
                       sample_offsets, n_batch, w.C, expert_to_bin, n_bins, w.part, w.coef, w.mi,
                       w.members, mi_per_sample);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    if (dlogits != nullptr) {
        int64_t blocks = ceil_div(T, kMiThreads / kWave);
        if (blocks > 2048) blocks = 2048;
        const double scale = -static_cast<double>(grad_scale) / n_batch;
        hipLaunchKernelGGL(mi_grad_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kMiThreads), 0,
                           stream, probs, M, T, E, sample_offsets, n_batch, expert_to_bin, n_bins,
                           w.members, w.coef, scale, dlogits, w.mi, loss);
    } else {
        hipLaunchKernelGGL(mi_loss_kernel, dim3(1), dim3(64), 0, stream, w.mi, n_batch, loss);
    }
    if ((err = hipGetLastError()) != hipSuccess) return err;
    return hipSuccess;
}

}  // namespace smoes
