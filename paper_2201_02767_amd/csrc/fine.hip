// Gathered fine attention at the finer levels: one wave per (parent query, head) work item, or per
// pair of neighbouring parents on maps of one row; the per-item work (its independent loads in
// item_head, then gather, MFMA logits, softmax, top-K, messages, the finest level's combination in
// fine_item, both in fine_item.h). A workgroup holds up to four independent waves (fewer when a
// wave's LDS region is large: 256 fp32 slots of d = 64); nothing synchronises across waves.
#include "fine_item.h"

namespace qta {

namespace {

using namespace fine;

template <typename T, int D, int NSP, bool VA, bool FINEST, bool ROW, bool PE>
__global__ __launch_bounds__(256) void fine_attn_kernel(FineArgs a)
{
    const int wave = threadIdx.x >> 6;
    const int wpb = blockDim.x >> 6;
    const int np = a.Hp * a.Wp;
    const int nitems = a.B * a.heads * (ROW ? (np + 1) / 2 : np);   // below 2^31 (checked by the launcher)
    // the work item is the same for the whole wave: keep it (and all that derives from it) scalar
    const int item = __builtin_amdgcn_readfirstlane(xcd_remap(blockIdx.x, gridDim.x) * wpb + wave);
    if (item >= nitems) return;            // whole wave leaves; only wave-level syncs follow
    extern __shared__ __align__(16) unsigned char smem[];
    const int nsp = (4 * a.Kp + 15) & ~15;
    ItemHead<T, D, NSP, VA, ROW> hd;
    item_head<T, D, NSP, VA, ROW, FINEST>(a, item, hd);
    fine_item<T, D, NSP, VA, FINEST, ROW, PE>(a, hd, smem + static_cast<size_t>(wave) * wave_lds<T, D>(nsp).total);
}

template <typename T, int D, int NSP, bool VA, bool FINEST, bool ROW, bool PE>
hipError_t launch_one(const FineArgs& a, hipStream_t stream)
{
    const int nsp = (4 * a.Kp + 15) & ~15;
    const WaveLds lay = wave_lds<T, D>(nsp);
    const size_t wave_bytes = lay.total;
    int wpb = 4;
    while (wpb > 1 && wpb * wave_bytes > device_max_lds()) --wpb;
    if (wave_bytes > device_max_lds()) return hipErrorInvalidValue;
    // the fused position encoding stages a 4x4 token block of one head in the value-row region
    if (PE && static_cast<size_t>(lay.p - lay.v) < static_cast<size_t>(D) * kPeTokenPitch * sizeof(T))
        return hipErrorInvalidValue;
    static std::atomic<unsigned long long> configured{0};     // devices whose LDS limit is raised
    if (hipError_t e = set_max_lds_once(reinterpret_cast<const void*>(&fine_attn_kernel<T, D, NSP, VA, FINEST, ROW, PE>),
                                        configured);
        e != hipSuccess)
        return e;
    const long long np = static_cast<long long>(a.Hp) * a.Wp;
    const long long items = static_cast<long long>(a.B) * a.heads * (ROW ? (np + 1) / 2 : np);
    const long long blocks = (items + wpb - 1) / wpb;
    if (blocks * wpb >= 0x7FFFFFFFLL) return hipErrorInvalidValue;     // work items are int
    hipLaunchKernelGGL((fine_attn_kernel<T, D, NSP, VA, FINEST, ROW, PE>), dim3(static_cast<unsigned>(blocks)),
                       dim3(wpb * kWave), wpb * wave_bytes, stream, a);
    return hipGetLastError();
}

template <typename T, int D, bool VA, bool FINEST, bool ROW, bool PE>
hipError_t launch_nsp_pe(const FineArgs& a, hipStream_t stream)
{
    const int nslot = 4 * a.Kp;
    if (nslot <= 16) return launch_one<T, D, 16, VA, FINEST, ROW, PE>(a, stream);
    if (nslot <= 32) return launch_one<T, D, 32, VA, FINEST, ROW, PE>(a, stream);
    if (nslot <= 64) return launch_one<T, D, 64, VA, FINEST, ROW, PE>(a, stream);
    if constexpr (!PE) {
        if (nslot <= 128) return launch_one<T, D, 128, VA, FINEST, ROW, PE>(a, stream);
        if (nslot <= 256) return launch_one<T, D, 256, VA, FINEST, ROW, PE>(a, stream);
    }
    return hipErrorInvalidValue;
}

// Levels of maps with more than one row may fuse their position encoding (a.pe_w).
template <typename T, int D, bool VA, bool FINEST, bool ROW>
hipError_t launch_nsp_row(const FineArgs& a, hipStream_t stream)
{
    if constexpr (!ROW) {
        if (a.pe_w) return launch_nsp_pe<T, D, VA, FINEST, ROW, true>(a, stream);
    } else {
        if (a.pe_w) return hipErrorInvalidValue;
    }
    return launch_nsp_pe<T, D, VA, FINEST, ROW, false>(a, stream);
}

// Maps of one row (attention along epipolar lines) pack two parents into one item.
template <typename T, int D, bool VA, bool FINEST>
hipError_t launch_nsp(const FineArgs& a, hipStream_t stream)
{
    if (a.H == 1 && a.Hp == 1) return launch_nsp_row<T, D, VA, FINEST, true>(a, stream);
    return launch_nsp_row<T, D, VA, FINEST, false>(a, stream);
}

template <typename T, int D>
hipError_t launch_td(const FineArgs& a, bool variant_a, bool finest, hipStream_t stream)
{
    if (variant_a) return finest ? launch_nsp<T, D, true, true>(a, stream) : launch_nsp<T, D, true, false>(a, stream);
    return finest ? launch_nsp<T, D, false, true>(a, stream) : launch_nsp<T, D, false, false>(a, stream);
}

}  // namespace

hipError_t launch_fine_attn(const FineArgs& a, int d, bool variant_a, bool bf16_in, bool finest, hipStream_t stream)
{
    const int nslot = 4 * a.Kp;
    if (nslot > kMaxSlots || (a.pe_w && nslot > kMaxSlotsPe)) return hipErrorInvalidValue;
    if (finest && (a.q_blocked || a.kv_blocked)) return hipErrorInvalidValue;   // level 0 is NHWC
    FineArgs b = a;
    b.inv_levels = a.levels > 0 ? 1.0f / static_cast<float>(a.levels) : 0.f;
    b.div_Wp = make_fastdiv(a.Wp);
    b.div_heads = make_fastdiv(a.heads);
    const int np = a.Hp * a.Wp;
    b.div_items = make_fastdiv(a.H == 1 && a.Hp == 1 ? (np + 1) / 2 : np);   // one-row maps: parent pairs
    if (bf16_in) {
        if (d == 32) return launch_td<bf16, 32>(b, variant_a, finest, stream);
        if (d == 64) return launch_td<bf16, 64>(b, variant_a, finest, stream);
    } else {
        if (d == 32) return launch_td<float, 32>(b, variant_a, finest, stream);
        if (d == 64) return launch_td<float, 64>(b, variant_a, finest, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace qta
