// Kernel argument blocks and launchers shared between the HIP kernels and the C-ABI host code.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/qta.h"

namespace qta {

// One pyramid pass over up to three token maps (q, k, v): from a source level produce one or two
// coarser levels.
struct PyramidPassArgs {
    const void* src[3];
    void* dst1[3];
    void* dst2[3];
    int B, Hs, Ws, H1, W1, H2, W2;
    int chunks;                 // 16-byte chunks per token (C * sizeof(dtype) / 16)
};

struct CoarseArgs {
    const void* q;
    const void* k;
    const void* v;
    int B, heads, N, C;         // N = Hc * Wc tokens at the coarsest level
    int K;                      // 0: no selection
    float scale;
    float* msg;                 // fp32 [B][N][heads][d], or NULL when `out` is written instead
    int32_t* sel_idx;
    float* sel_key;
    void* out;                  // single-level problem: write out = w0 * m (B) or m (A) in dtype
    const float* w;
    int levels;
};

struct FineArgs {
    const void* q;
    const void* k;
    const void* v;
    int B, heads, H, W, Hp, Wp, C, K;
    float scale;
    const int32_t* parent_idx;
    const float* parent_key;
    // intermediate level: outputs
    float* msg;
    int32_t* sel_idx;
    float* sel_key;
    // finest level: fused combination
    void* out;
    const float* w;
    int levels;
    const float* coarser_msg[QTA_MAX_LEVELS];   // entry j: message of level j (j >= 1)
    int lvl_W[QTA_MAX_LEVELS];                  // map width of level j
    int lvl_N[QTA_MAX_LEVELS];                  // tokens of level j
};

struct TopkArgs {
    const float* keys;
    const int32_t* cand_idx;
    int rows, n, K;
    int32_t* idx_out;
    float* key_out;
};

// Largest dynamic LDS a workgroup may use on the current device (cached per device).
inline size_t device_max_lds()
{
    static int cached[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 64 * 1024;
    if (cached[dev] == 0) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess || v <= 0)
            v = 64 * 1024;
        cached[dev] = v;
    }
    return static_cast<size_t>(cached[dev]);
}

hipError_t launch_pyramid_pass(const PyramidPassArgs& a, int nlev, int ntensors, bool use_bf16, hipStream_t stream);
hipError_t launch_coarse_attn(const CoarseArgs& a, int d, bool variant_a, bool use_bf16, hipStream_t stream);
hipError_t launch_fine_attn(const FineArgs& a, int d, bool variant_a, bool use_bf16, bool finest, hipStream_t stream);
hipError_t launch_topk(const TopkArgs& a, hipStream_t stream);

}  // namespace qta
