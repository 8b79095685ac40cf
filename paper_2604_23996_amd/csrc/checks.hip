// Device-side check of the layer's device-resident preconditions (the
// problem statement of Sec. 3.1-3.4: hard modality labels in {vision, text},
// samples as contiguous token ranges, bins of N_e / N_bins experts each).
// The host cannot see these values without a synchronisation, so one block
// reads them on the device and writes a bitmask; nothing else is touched.
#include "smoes.h"
#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

constexpr int kCheckThreads = 512;

__global__ void __launch_bounds__(kCheckThreads)
check_inputs_kernel(const uint8_t* __restrict__ mid, int64_t T, const int32_t* __restrict__ off, int n_batch,
                    const int32_t* __restrict__ e2b, int E, int n_bins, int32_t* __restrict__ flags) {
    const int tid = threadIdx.x;
    int bad_mid = 0, bad_off = 0, bad_bin = 0;
    if (mid != nullptr)
        for (int64_t j = tid; j < T; j += kCheckThreads) bad_mid |= mid[j] > 1 ? 1 : 0;
    if (off != nullptr) {
        if (tid == 0 && (off[0] != 0 || static_cast<int64_t>(off[n_batch]) != T)) bad_off = 1;
        for (int i = tid; i < n_batch; i += kCheckThreads) bad_off |= off[i + 1] < off[i] ? 1 : 0;
    }
    // every entry in range, and every bin holding exactly E / n_bins experts
    // (one thread counts one bin over the whole map: no atomics)
    const int nb = E / n_bins;
    for (int e = tid; e < E; e += kCheckThreads) bad_bin |= (e2b[e] < 0 || e2b[e] >= n_bins) ? 1 : 0;
    for (int b = tid; b < n_bins; b += kCheckThreads) {
        int c = 0;
        for (int e = 0; e < E; ++e) c += e2b[e] == b ? 1 : 0;
        bad_bin |= c != nb ? 1 : 0;
    }
    bad_mid = __syncthreads_or(bad_mid);
    bad_off = __syncthreads_or(bad_off);
    bad_bin = __syncthreads_or(bad_bin);
    if (tid == 0)
        flags[0] = (bad_mid ? SMOES_CHECK_MODALITY_ID : 0) | (bad_off ? SMOES_CHECK_SAMPLE_OFFSETS : 0) |
                   (bad_bin ? SMOES_CHECK_EXPERT_TO_BIN : 0);
}

}  // namespace

hipError_t launch_check_inputs(const uint8_t* modality_id, int64_t T, const int32_t* sample_offsets, int n_batch,
                               const int32_t* expert_to_bin, int E, int n_bins, int32_t* flags,
                               hipStream_t stream) {
    hipLaunchKernelGGL(check_inputs_kernel, dim3(1), dim3(kCheckThreads), 0, stream, modality_id, T,
                       sample_offsets, n_batch, expert_to_bin, E, n_bins, flags);
    return hipGetLastError();
}

}  // namespace smoes
