// Step 3 as a standalone row-wise top-K (Sec. 3.2: each query keeps the K keys with the highest
// attention scores).
//
// One wave per row. Each lane holds NPER candidates of the row as 64-bit words (score, inverted
// name), so one unsigned comparison orders by (score descending, name ascending). K rounds of a
// wave-wide maximum pick the winners in order; the lowest lane holding the winning word retires
// it, so repeated names are kept as separate candidates. Rows are independent; a workgroup of
// four waves takes four rows.
#include "qta_device.h"
#include "qta_internal.h"

namespace qta {

namespace {

template <int NPER>
__global__ __launch_bounds__(256) void topk_kernel(TopkArgs a)
{
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= a.rows) return;                  // whole wave leaves; no workgroup barriers below
    const size_t base = static_cast<size_t>(row) * a.n;
    // every load unconditional (clamped into the row) so that all are in flight at once; slots
    // past the row and negative names are masked to 0 (no candidate)
    uint64_t word[NPER];
    float key[NPER];
    int32_t name[NPER];
#pragma unroll
    for (int e = 0; e < NPER; ++e) {
        const int j = min(lane + kWave * e, a.n - 1);
        key[e] = a.keys[base + j];
        name[e] = a.cand_idx ? a.cand_idx[base + j] : j;
    }
#pragma unroll
    for (int e = 0; e < NPER; ++e) {
        const bool live = lane + kWave * e < a.n && name[e] >= 0;
        word[e] = live ? rank_word(key[e], name[e]) : 0ull;
    }
    const size_t orow = static_cast<size_t>(row) * a.K;
    for (int r = 0; r < a.K; ++r) {
        uint64_t best = 0ull;
#pragma unroll
        for (int e = 0; e < NPER; ++e) best = word[e] > best ? word[e] : best;
        const uint64_t g = wave_max_u64(best);
        if (g == 0ull) {                         // fewer than K candidates: pad
            if (lane == 0) {
                a.idx_out[orow + r] = -1;
                if (a.key_out) a.key_out[orow + r] = 0.f;
            }
            continue;
        }
        const uint64_t owners = __ballot(best == g);
        const int owner = __ffsll(static_cast<unsigned long long>(owners)) - 1;
        if (lane == owner) {
            bool done = false;
#pragma unroll
            for (int e = 0; e < NPER; ++e)
                if (!done && word[e] == g) {
                    word[e] = 0ull;
                    done = true;
                }
        }
        if (lane == 0) {
            a.idx_out[orow + r] = rank_word_index(g);
            if (a.key_out) a.key_out[orow + r] = rank_word_score(g);
        }
    }
}

// In-place ordering of selection rows of K <= 64 entries (the stage calls' output contract): one
// wave per row, lane i holds entry i as a ranking word (0 for an empty slot, index -1), counts the
// entries ranked before it by reading every other lane's word, and writes itself to that place.
// Empty slots follow the kept keys. Every load of the row completes before any store (the ranks
// need all of them).
__global__ __launch_bounds__(256) void sort_rows_kernel(int32_t* idx, float* key, int rows, int K)
{
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= rows) return;                    // whole wave leaves; no workgroup barriers below
    const size_t base = static_cast<size_t>(row) * K;
    const int e = min(lane, K - 1);
    const int32_t my_idx = idx[base + e];
    const float my_key = key[base + e];
    const bool live = lane < K && my_idx >= 0;
    const uint64_t word = live ? rank_word(my_key, my_idx) : 0ull;
    int before = 0;
    for (int j = 0; j < K; ++j) {               // uniform trip count
        const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(word), j);
        const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(word >> 32), j);
        const uint64_t wj = (static_cast<uint64_t>(hi) << 32) | lo;
        before += wj > word ? 1 : 0;
    }
    const uint64_t live_mask = __ballot(live);
    const uint64_t dead_mask = __ballot(lane < K && !live);
    const int nlive = __popcll(live_mask);
    const int pos = live ? before : nlive + lanes_below(dead_mask);
    if (lane < K) {
        idx[base + pos] = live ? my_idx : -1;
        key[base + pos] = live ? my_key : 0.f;
    }
}

}  // namespace

hipError_t launch_sort_rows(int32_t* idx, float* key, long long rows, int K, hipStream_t stream)
{
    if (rows <= 0) return hipSuccess;
    if (K < 1 || K > kWave || rows > 0x7FFFFFFFLL - 3) return hipErrorInvalidValue;
    hipLaunchKernelGGL(sort_rows_kernel, dim3(static_cast<unsigned>((rows + 3) / 4)), dim3(256), 0, stream, idx, key,
                       static_cast<int>(rows), K);
    return hipGetLastError();
}

hipError_t launch_topk(const TopkArgs& a, hipStream_t stream)
{
    const unsigned blocks = static_cast<unsigned>((a.rows + 3) / 4);
    if (a.n <= 64) hipLaunchKernelGGL((topk_kernel<1>), dim3(blocks), dim3(256), 0, stream, a);
    else if (a.n <= 256) hipLaunchKernelGGL((topk_kernel<4>), dim3(blocks), dim3(256), 0, stream, a);
    else if (a.n <= 1024) hipLaunchKernelGGL((topk_kernel<16>), dim3(blocks), dim3(256), 0, stream, a);
    else if (a.n <= 4096) hipLaunchKernelGGL((topk_kernel<64>), dim3(blocks), dim3(256), 0, stream, a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace qta
