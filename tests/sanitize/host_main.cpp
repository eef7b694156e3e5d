// Runs the host side of the C ABI (argument validation, LDS and split
// planning, workspace layout) under the sanitizers, with the device launches
// replaced by stubs that report no device.  Every entry point is called with
// valid descriptors (which reach a stub and return VD_ERR_HIP) and with
// invalid ones (which must be rejected before).  Built and run by
// tests/test_sanitizers.py.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstring>
#include <vector>

#include "vd.h"
#include "vd_launch.h"

namespace vd {
hipError_t launch_step(const UnitParams &, int, int, int, int, size_t, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_select(const UnitParams &, int, size_t, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_compact(const UnitParams &, int, int, int, size_t, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_attn(const UnitParams &, int, int, int, int, bool, size_t, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_geometry(const UnitParams &, int, int, int, size_t, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_stream_read(const void *, size_t, uint32_t *, hipStream_t) { return hipErrorNoDevice; }
hipError_t scratch_memory(hipStream_t, void **) { return hipErrorNoDevice; }
}  // namespace vd

static int failures = 0;
#define EXPECT(x)                                                                \
    do {                                                                         \
        if (!(x)) {                                                              \
            std::fprintf(stderr, "expectation failed at line %d: %s\n", __LINE__, #x); \
            ++failures;                                                          \
        }                                                                        \
    } while (0)

static vd_cache_desc desc(int S, int L, int H, int Hq, int D, int C, int dtype) {
    vd_cache_desc d;
    std::memset(&d, 0, sizeof d);
    d.k = reinterpret_cast<void *>(0x7f0000000000ull);
    d.v = reinterpret_cast<void *>(0x7f8000000000ull);
    d.dtype = dtype;
    d.num_seqs = S;
    d.num_layers = L;
    d.num_kv_heads = H;
    d.num_q_heads = Hq;
    d.head_dim = D;
    d.capacity = C;
    d.stride_slot = D;
    d.stride_head = int64_t(C) * D;
    d.stride_layer = int64_t(H) * C * D;
    d.stride_seq = int64_t(L) * H * C * D;
    return d;
}

int main() {
    void *dev = reinterpret_cast<void *>(0x7e0000000000ull);
    for (int dtype = 0; dtype < 2; ++dtype) {
        for (int D : {64, 128, 256}) {
            for (int S : {1, 3, 300}) {
                const int C = 5000;
                vd_cache_desc d = desc(S, 2, 2, 8, D, C, dtype);
                std::vector<int32_t> n(S), N(S);
                for (int s = 0; s < S; ++s) {
                    n[s] = (s * 997) % C;
                    N[s] = 1 + (s * 131) % C;
                }
                auto *f = static_cast<float *>(dev);
                auto *db = static_cast<double *>(dev);
                auto *u8 = static_cast<uint8_t *>(dev);
                auto *i32 = static_cast<int32_t *>(dev);
                for (int var = 0; var <= 5; ++var) {
                    EXPECT(vd_score(&d, n.data(), vd_variant(var), f, f, nullptr) == VD_ERR_HIP);
                    EXPECT(vd_evict_step(&d, n.data(), N.data(), vd_variant(var), db, i32, f, u8, nullptr,
                                         0, nullptr) == VD_ERR_HIP);
                }
                EXPECT(vd_select_topn(&d, f, n.data(), N.data(), u8, nullptr) == VD_ERR_HIP);
                EXPECT(vd_compact(&d, u8, n.data(), N.data(), i32, nullptr) != VD_ERR_INVALID_ARG);
                EXPECT(vd_geometry(&d, n.data(), nullptr, nullptr, db, nullptr) == VD_ERR_HIP);
                EXPECT(vd_geometry(&d, n.data(), db, db, db, nullptr) == VD_ERR_HIP);
                // decode step: n <= N + 1
                for (int s = 0; s < S; ++s) {
                    N[s] = 1 + (s * 131) % (C - 1);
                    n[s] = N[s] + (s & 1);
                }
                for (int var : {0, 6}) {
                    const size_t ws = vd_decode_attention_workspace_size(&d, vd_variant(var));
                    EXPECT(ws > 0);
                    EXPECT(vd_decode_attention_evict(&d, f, 0.1f, n.data(), N.data(), vd_variant(var), db,
                                                     i32, f, dev, ws, nullptr) == VD_ERR_HIP);
                    const vd_status st = vd_decode_attention_evict_noalloc(
                        &d, f, 0.1f, n.data(), N.data(), vd_variant(var), db, i32, f, nullptr);
                    EXPECT(st == VD_ERR_HIP || st == VD_ERR_WORKSPACE);
                }
                // rejections
                EXPECT(vd_evict_step(&d, n.data(), nullptr, VD_SCORE_L2, nullptr, nullptr, nullptr,
                                     nullptr, nullptr, 0, nullptr) == VD_ERR_INVALID_ARG);
                EXPECT(vd_evict_step(&d, n.data(), N.data(), vd_variant(9), nullptr, nullptr, nullptr,
                                     nullptr, nullptr, 0, nullptr) == VD_ERR_INVALID_ARG);
                n[0] = C + 1;
                EXPECT(vd_score(&d, n.data(), VD_SCORE_L2, f, nullptr, nullptr) == VD_ERR_INVALID_ARG);
            }
        }
    }
    // the slot limit: keys and lists that do not fit the LDS
    vd_cache_desc big = desc(1, 1, 1, 1, 256, VD_MAX_CAPACITY, 1);
    int32_t n1 = VD_MAX_CAPACITY, N1 = 1;
    vd_status st = vd_evict_step(&big, &n1, &N1, VD_SCORE_L2, nullptr, nullptr, nullptr, nullptr, nullptr,
                                 0, nullptr);
    EXPECT(st == VD_ERR_UNSUPPORTED || st == VD_ERR_HIP);
    vd_cache_desc over = desc(1, 1, 1, 1, 128, VD_MAX_CAPACITY + 1, 0);
    EXPECT(vd_evict_step(&over, &n1, &N1, VD_SCORE_L2, nullptr, nullptr, nullptr, nullptr, nullptr, 0,
                         nullptr) == VD_ERR_UNSUPPORTED);
    EXPECT(vd_stream_read(nullptr, 16, nullptr, nullptr) == VD_ERR_INVALID_ARG);
    for (int s = 0; s < 6; ++s) EXPECT(vd_status_string(vd_status(s)) != nullptr);
    if (failures) return 1;
    std::puts("host sanitizer run ok");
    return 0;
}
