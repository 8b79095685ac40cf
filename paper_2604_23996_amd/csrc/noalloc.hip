// smoes_mi_loss_noalloc: the inter-bin MI loss and its logit gradient with
// the scratch memory taken from a fixed file-scope device array instead of a
// caller workspace, for callers that cannot allocate (code under HIP graph
// capture, serving loops that forbid allocation). Same kernels, same
// arithmetic and the same bits as smoes_mi_loss.
#include <atomic>
#include <mutex>

#include "smoes.h"
#include "common.h"
#include "kernels.h"

namespace {

// Each device that runs the library holds its own copy of this array for
// the life of the process. Host code never uses its name as an address: the
// device address comes from hipGetSymbolAddress, per device.
__device__ __align__(256) unsigned char scratch[SMOES_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_setup;

// Device address of the current device's copy of `scratch`, looked up once
// per device (with that device current) and kept.
int scratch_address(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return SMOES_ERR_HIP;
    void* p = g_scratch[dev].load(std::memory_order_acquire);
    if (p == nullptr) {
        std::lock_guard<std::mutex> lock(g_setup);
        p = g_scratch[dev].load(std::memory_order_relaxed);
        if (p == nullptr) {
            if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return SMOES_ERR_HIP;
            g_scratch[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return SMOES_OK;
}

}  // namespace

extern "C" int smoes_mi_loss_noalloc(const float* probs, const float* M, int64_t T, int E,
                                     const int32_t* sample_offsets, int n_batch, const int32_t* expert_to_bin,
                                     int n_bins, float grad_scale, float* mi_per_sample, float* loss,
                                     float* dlogits, void* stream) {
    // the same host checks as smoes_mi_loss, then the scratch bound
    if (T < 0 || E < 1 || E > SMOES_E_MAX || n_bins < 1 || n_bins > SMOES_BINS_MAX || (E % n_bins) != 0 ||
        n_batch < 1)
        return SMOES_ERR_SHAPE;
    if (sample_offsets == nullptr && n_batch != 1) return SMOES_ERR_SHAPE;
    if (grad_scale != grad_scale) return SMOES_ERR_ARG;
    if (probs == nullptr || M == nullptr || expert_to_bin == nullptr || mi_per_sample == nullptr || loss == nullptr)
        return SMOES_ERR_ARG;
    if (smoes_mi_workspace_size(T, E, n_batch, n_bins) > SMOES_NOALLOC_SCRATCH_BYTES) return SMOES_ERR_SCRATCH;
    void* base = nullptr;
    const int st = scratch_address(&base);
    if (st != SMOES_OK) return st;
    // the workspace query includes the slack for aligning its start; the
    // array is 256-byte aligned, so the kernels' buffers start at its base
    const hipError_t err = smoes::launch_mi(probs, M, T, E, sample_offsets, n_batch, expert_to_bin, n_bins,
                                            grad_scale, mi_per_sample, loss, T > 0 ? dlogits : nullptr, base,
                                            static_cast<hipStream_t>(stream));
    return err == hipSuccess ? SMOES_OK : SMOES_ERR_HIP;
}
