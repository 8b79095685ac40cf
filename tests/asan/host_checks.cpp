// Host-side checks of libsmoes under AddressSanitizer: every path here runs
// on the CPU only (descriptor validation, workspace arithmetic, argument
// errors that return before any device call), so the driver needs no GPU.
// Built together with a host-only, ASan-instrumented copy of the library by
// tests/test_asan_host.py; it prints one line per failed check and exits
// non-zero if any failed.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "smoes.h"

static int failures = 0;
#define EXPECT(cond)                                                           \
    do {                                                                       \
        if (!(cond)) {                                                         \
            std::printf("FAIL %s:%d: %s\n", __FILE__, __LINE__, #cond);        \
            ++failures;                                                        \
        }                                                                      \
    } while (0)

static smoes_layer layer(int64_t T, int d, int E, int k, int inter, int shared_inter, int n_bins, int n_batch,
                         int dtype, int packed, int save_preact) {
    smoes_layer L;
    std::memset(&L, 0, sizeof(L));
    L.T = T;
    L.d = d;
    L.E = E;
    L.k = k;
    L.inter = inter;
    L.shared_inter = shared_inter;
    L.n_bins = n_bins;
    L.n_batch = n_batch;
    L.act_dtype = dtype;
    L.tau = 0.0f;
    L.beta = 0.99f;
    L.var_floor = 1e-6f;
    L.grad_scale = 1.0f;
    L.weights_packed = packed;
    L.save_preact = save_preact;
    return L;
}

// The workspace buffers of a layer lie inside its workspace and do not
// overlap; writing each one in full on a host allocation of exactly the
// reported size lets the sanitizer catch a carve past the end.
static void check_buffers(const smoes_layer& L) {
    const size_t n = smoes_workspace_bytes(&L);
    EXPECT(n > 0);
    std::vector<unsigned char> heap(n);
    unsigned char* ws = heap.data();
    struct Span {
        size_t lo, hi;
    };
    std::vector<Span> spans;
    for (int which = SMOES_BUF_H_ROUTED; which <= SMOES_BUF_CHECK_FLAGS; ++which) {
        void* p = nullptr;
        size_t bytes = 0;
        EXPECT(smoes_workspace_buffer(&L, ws, which, &p, &bytes) == SMOES_OK);
        if (bytes == 0) continue;
        unsigned char* b = static_cast<unsigned char*>(p);
        EXPECT(b >= ws && b + bytes <= ws + n);
        if (b >= ws && b + bytes <= ws + n) {
            std::memset(b, 0x5a, bytes);
            spans.push_back({static_cast<size_t>(b - ws), static_cast<size_t>(b - ws) + bytes});
        }
    }
    for (size_t i = 0; i < spans.size(); ++i)
        for (size_t j = i + 1; j < spans.size(); ++j)
            EXPECT(spans[i].hi <= spans[j].lo || spans[j].hi <= spans[i].lo);
    void* p = nullptr;
    size_t bytes = 0;
    EXPECT(smoes_workspace_buffer(&L, ws, 99, &p, &bytes) == SMOES_ERR_ARG);
    EXPECT(smoes_workspace_buffer(nullptr, ws, 0, &p, &bytes) == SMOES_ERR_ARG);
    EXPECT(smoes_workspace_buffer(&L, ws, 0, nullptr, &bytes) == SMOES_ERR_ARG);
}

int main() {
    // status strings and version: static, never NULL
    for (int s = -6; s <= 1; ++s) EXPECT(smoes_status_string(s) != nullptr && std::strlen(smoes_status_string(s)) > 0);
    EXPECT(smoes_status_string(12345) != nullptr);
    EXPECT(smoes_version() != nullptr && std::strlen(smoes_version()) > 0);

    // standalone workspace sizes: shapes in range give a size, out of range 0
    EXPECT(smoes_route_workspace_size(16384, 4096, 160, SMOES_BF16) > 0);
    EXPECT(smoes_route_workspace_size(100, 72, 8, SMOES_F32) > 0);
    EXPECT(smoes_modality_workspace_size(16384, 4096) > 0);
    EXPECT(smoes_mi_workspace_size(16384, 160, 16, 8) > 0);
    EXPECT(smoes_permute_workspace_size(16384, 160, 6) > 0);
    EXPECT(smoes_binning_workspace_size(16384, 160, 8) > 0);
    EXPECT(smoes_gmm_workspace_size(4096, 2048, 2) > 0);

    // layer descriptors: the workloads' shapes, both dtypes, packed, kept pre-activations
    const smoes_layer good[] = {
        layer(512, 256, 8, 2, 512, 0, 2, 1, SMOES_F32, 0, 0),
        layer(4096, 2048, 64, 6, 1408, 2816, 8, 4, SMOES_BF16, 1, 0),
        layer(4096, 2048, 64, 6, 1408, 2816, 8, 4, SMOES_BF16, 1, 1),
        layer(8192, 2048, 128, 8, 768, 0, 16, 8, SMOES_BF16, 0, 0),
        layer(16384, 4096, 160, 6, 1536, 3072, 8, 16, SMOES_BF16, 1, 1),
        layer(3, 64, 4, 2, 32, 0, 2, 1, SMOES_BF16, 1, 0),
        layer(300, 136, 10, 3, 48, 96, 5, 2, SMOES_F32, 0, 0),
        layer(0, 64, 4, 2, 32, 32, 2, 1, SMOES_BF16, 1, 0),
    };
    for (const smoes_layer& L : good) {
        EXPECT(smoes_workspace_bytes(&L) > 0);
        EXPECT(smoes_backward_workspace_bytes(&L) > 0);
        for (int w = SMOES_W13; w <= SMOES_WS2T; ++w) (void)smoes_packed_weight_bytes(&L, w);
        check_buffers(L);
    }
    // invalid descriptors: every size query says 0, every entry point refuses
    smoes_layer bad[] = {
        layer(512, 256, 8, 2, 512, 0, 3, 1, SMOES_F32, 0, 0),      // E % n_bins != 0
        layer(512, 256, 8, 2, 500, 0, 2, 1, SMOES_F32, 0, 0),      // inter % 16 != 0
        layer(512, 260, 8, 2, 512, 0, 2, 1, SMOES_F32, 0, 0),      // d % 8 != 0
        layer(512, 256, 300, 2, 512, 0, 2, 1, SMOES_F32, 0, 0),    // E > SMOES_E_MAX
        layer(512, 256, 8, 9, 512, 0, 2, 1, SMOES_F32, 0, 0),      // k > E
        layer(512, 256, 8, 2, 512, 0, 2, 1, SMOES_F32, 1, 0),      // packed fp32
        layer(512, 256, 8, 2, 512, 0, 2, 1, SMOES_BF16, 0, 1),     // kept pre-activations, row-major
        layer(512, 256, 8, 2, 512, 0, 2, 1, 7, 0, 0),              // unknown dtype
        layer(512, 256, 8, 2, 512, 0, 2, 0, SMOES_F32, 0, 0),      // no samples
        layer(-1, 256, 8, 2, 512, 0, 2, 1, SMOES_F32, 0, 0),       // negative T
    };
    bad[0].beta = 0.99f;
    for (const smoes_layer& L : bad) {
        EXPECT(smoes_workspace_bytes(&L) == 0);
        EXPECT(smoes_backward_workspace_bytes(&L) == 0);
        smoes_layer_io io;
        std::memset(&io, 0, sizeof(io));
        EXPECT(smoes_moe_forward(&L, &io, nullptr, 0, nullptr) != SMOES_OK);
        EXPECT(smoes_moe_backward(&L, &io, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0,
                                  nullptr, 0, nullptr) != SMOES_OK);
    }
    smoes_layer nan_beta = good[0];
    nan_beta.beta = 2.0f;
    EXPECT(smoes_workspace_bytes(&nan_beta) == 0);
    EXPECT(smoes_workspace_bytes(nullptr) == 0);
    EXPECT(smoes_backward_workspace_bytes(nullptr) == 0);

    // argument errors of the entry points return before any device work
    EXPECT(smoes_moe_forward(&good[1], nullptr, nullptr, 0, nullptr) == SMOES_ERR_ARG);
    {
        smoes_layer_io io;
        std::memset(&io, 0, sizeof(io));
        EXPECT(smoes_moe_forward(&good[1], &io, nullptr, 0, nullptr) == SMOES_ERR_ARG);
        smoes_layer_grads g;
        std::memset(&g, 0, sizeof(g));
        EXPECT(smoes_moe_backward(&good[1], &io, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, &g, nullptr, 0,
                                  nullptr, 0, nullptr) == SMOES_ERR_ARG);
        EXPECT(smoes_check_inputs(&good[1], nullptr, nullptr, nullptr) == SMOES_ERR_ARG);
    }
    EXPECT(smoes_route(nullptr, SMOES_BF16, 16, 64, nullptr, nullptr, 8, 2, 0, nullptr, nullptr, nullptr, nullptr,
                       nullptr, 0, nullptr) == SMOES_ERR_ARG);
    EXPECT(smoes_route(nullptr, SMOES_BF16, 16, 64, nullptr, nullptr, 300, 2, 0, nullptr, nullptr, nullptr, nullptr,
                       nullptr, 0, nullptr) == SMOES_ERR_SHAPE);
    EXPECT(smoes_permute(nullptr, 16, 300, 2, nullptr, nullptr, nullptr, nullptr, SMOES_BF16, 64, nullptr, nullptr, 0,
                         nullptr) == SMOES_ERR_SHAPE);
    EXPECT(smoes_mi_loss(nullptr, nullptr, 16, 8, nullptr, 1, nullptr, 3, 1.0f, nullptr, nullptr, nullptr, nullptr, 0,
                         nullptr) == SMOES_ERR_SHAPE);
    EXPECT(smoes_modality_score(nullptr, SMOES_BF16, 16, 64, nullptr, nullptr, nullptr, nullptr, 0, 0.99f, 0.0f,
                                1e-6f, nullptr, nullptr, 0, nullptr) == SMOES_ERR_ARG);
    EXPECT(smoes_pack_weights(&good[0], SMOES_W13, nullptr, nullptr, nullptr) != SMOES_OK);  // fp32: nothing to pack
    EXPECT(smoes_streams_create(nullptr) == SMOES_ERR_ARG);
    EXPECT(smoes_events_create(2, nullptr) == SMOES_ERR_ARG);

    if (failures == 0) std::printf("host checks passed\n");
    return failures == 0 ? 0 : 1;
}
