// Device helpers shared by the QuadTree attention kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qta {

constexpr int kWave = 64;
constexpr int kNumXcd = 8;   // MI355X: 8 accelerator complex dies, workgroups dealt round-robin

// ---------------------------------------------------------------------------------------------
// storage types
// ---------------------------------------------------------------------------------------------

// bf16 is carried as its 16 raw bits.
struct bf16 {
    uint16_t bits;
};

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// fp32 -> bf16, round to nearest, ties to even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f)
{
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return u >> 16;
}

// An access at a 32-bit byte offset from a wave-uniform base: the address is the base in scalar
// registers plus the zero-extended per-lane offset, the form the hardware takes directly (a signed
// or 64-bit index costs a 64-bit add per lane). The offset must stay below 2^32.
template <typename V>
__device__ __forceinline__ V load_at(const void* base, uint32_t byte_off)
{
    return *reinterpret_cast<const V*>(static_cast<const unsigned char*>(base) + byte_off);
}
template <typename V>
__device__ __forceinline__ void store_at(void* base, uint32_t byte_off, V x)
{
    *reinterpret_cast<V*>(static_cast<unsigned char*>(base) + byte_off) = x;
}

template <typename T> struct Storage;

template <> struct Storage<float> {
    static constexpr int kPer16B = 4;      // elements per 16-byte chunk
    __device__ static __forceinline__ void unpack(const uint4& c, float* out)
    {
        out[0] = __uint_as_float(c.x);
        out[1] = __uint_as_float(c.y);
        out[2] = __uint_as_float(c.z);
        out[3] = __uint_as_float(c.w);
    }
    __device__ static __forceinline__ uint4 pack(const float* in)
    {
        return make_uint4(__float_as_uint(in[0]), __float_as_uint(in[1]), __float_as_uint(in[2]),
                          __float_as_uint(in[3]));
    }
    __device__ static __forceinline__ float load1(const void* base, size_t i)
    {
        return static_cast<const float*>(base)[i];
    }
    __device__ static __forceinline__ void store1(void* base, size_t i, float x)
    {
        static_cast<float*>(base)[i] = x;
    }
    // element i (below 2^30) of a wave-uniform base
    __device__ static __forceinline__ float load1_at(const void* base, uint32_t i) { return load_at<float>(base, i * 4u); }
    __device__ static __forceinline__ void store1_at(void* base, uint32_t i, float x) { store_at<float>(base, i * 4u, x); }
    // Round an fp32 value to this storage type and back.
    __device__ static __forceinline__ float round(float x) { return x; }
};

template <> struct Storage<bf16> {
    static constexpr int kPer16B = 8;
    __device__ static __forceinline__ void unpack(const uint4& c, float* out)
    {
        const uint32_t w[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            out[2 * i] = __uint_as_float(w[i] << 16);
            out[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
        }
    }
    __device__ static __forceinline__ uint4 pack(const float* in)
    {
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) w[i] = f32_to_bf16_bits(in[2 * i]) | (f32_to_bf16_bits(in[2 * i + 1]) << 16);
        return make_uint4(w[0], w[1], w[2], w[3]);
    }
    __device__ static __forceinline__ float load1(const void* base, size_t i)
    {
        return bf16_bits_to_f32(static_cast<const uint16_t*>(base)[i]);
    }
    __device__ static __forceinline__ void store1(void* base, size_t i, float x)
    {
        static_cast<uint16_t*>(base)[i] = static_cast<uint16_t>(f32_to_bf16_bits(x));
    }
    // element i (below 2^31) of a wave-uniform base
    __device__ static __forceinline__ float load1_at(const void* base, uint32_t i)
    {
        return bf16_bits_to_f32(load_at<uint16_t>(base, i * 2u));
    }
    __device__ static __forceinline__ void store1_at(void* base, uint32_t i, float x)
    {
        store_at<uint16_t>(base, i * 2u, static_cast<uint16_t>(f32_to_bf16_bits(x)));
    }
    __device__ static __forceinline__ float round(float x) { return __uint_as_float(f32_to_bf16_bits(x) << 16); }
};

// ---------------------------------------------------------------------------------------------
// launch mapping
// ---------------------------------------------------------------------------------------------

// Workgroups are dealt to the XCDs round-robin (block b runs on XCD b % 8), and each XCD has its
// own L2. Remap so that XCD x processes one contiguous range of logical tiles: neighbouring
// query tiles, which gather overlapping keys, then share an L2.
__device__ __forceinline__ int xcd_remap(int bid, int nblk)
{
    const int q = nblk / kNumXcd, r = nblk % kNumXcd;
    const int xcd = bid % kNumXcd, pos = bid / kNumXcd;
    return xcd * q + (xcd < r ? xcd : r) + pos;
}

// ---------------------------------------------------------------------------------------------
// wave-level communication
// ---------------------------------------------------------------------------------------------

// Make this wave's LDS writes visible to its other lanes (no cross-wave synchronisation).
__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// ---- register-only exchanges (DPP and permlane swaps; no LDS round trip) ----

// DPP controls used below.
constexpr int kDppXor1 = 0xB1;         // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;         // quad_perm [2,3,0,1]
constexpr int kDppRowShl4 = 0x104;
constexpr int kDppRowShr4 = 0x114;
constexpr int kDppRowRor4 = 0x124;     // within a 16-lane row: lane (lane + 4) mod 16
constexpr int kDppRowRor8 = 0x128;     // within a 16-lane row: lane ^ 8
constexpr int kDppRowMirror = 0x140;   // within a row: lane -> 15 - lane
constexpr int kDppRowHalfMirror = 0x141;  // within 8 lanes: lane -> 7 - lane

// The value held by lane (lane ^ M), M a power of two below 64.
template <int M>
__device__ __forceinline__ uint32_t xchg_u32(uint32_t x)
{
    if constexpr (M == 1) {
        return __builtin_amdgcn_update_dpp(0u, x, kDppXor1, 0xF, 0xF, false);
    } else if constexpr (M == 2) {
        return __builtin_amdgcn_update_dpp(0u, x, kDppXor2, 0xF, 0xF, false);
    } else if constexpr (M == 4) {
        // banks 1 and 3 of each row read four lanes down, banks 0 and 2 four lanes up
        const uint32_t t = __builtin_amdgcn_update_dpp(x, x, kDppRowShr4, 0xF, 0xA, false);
        return __builtin_amdgcn_update_dpp(t, x, kDppRowShl4, 0xF, 0x5, false);
    } else if constexpr (M == 8) {
        return __builtin_amdgcn_update_dpp(0u, x, kDppRowRor8, 0xF, 0xF, false);
    } else if constexpr (M == 16) {
        const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
        return (threadIdx.x & 16) ? r[0] : r[1];
    } else {
        static_assert(M == 32, "exchange distance");
        const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
        return (threadIdx.x & 32) ? r[0] : r[1];
    }
}

template <int M>
__device__ __forceinline__ float xchg_f32(float x) { return __uint_as_float(xchg_u32<M>(__float_as_uint(x))); }

// Sum over the four lanes n, n+4, n+8, n+12 of each 16-lane row (every one of them ends with it):
// two row rotations.
__device__ __forceinline__ float row_sum_stride4(float x)
{
    x += __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), kDppRowRor4, 0xF, 0xF, false));
    return x + __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), kDppRowRor8, 0xF, 0xF, false));
}

// Butterfly all-reduce over the 64 lanes (every lane ends with the same value).
template <typename Op>
__device__ __forceinline__ float wave_allreduce(float x, Op op)
{
    x = op(x, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), kDppXor1, 0xF, 0xF, false)));
    x = op(x, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), kDppXor2, 0xF, 0xF, false)));
    x = op(x, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), kDppRowHalfMirror, 0xF, 0xF, false)));
    x = op(x, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), kDppRowMirror, 0xF, 0xF, false)));
    const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = op(__uint_as_float(r16[0]), __uint_as_float(r16[1]));
    const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return op(__uint_as_float(r32[0]), __uint_as_float(r32[1]));
}

// 1/x on the hardware reciprocal (within one ulp) instead of the correctly rounded division
// sequence; used for softmax normalisers, which are at least 1.
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

// Natural logarithm from the hardware base-2 logarithm (about one ulp of log2 x); used for the
// log-sum-exp of softmax sums, which are at least 1.
__device__ __forceinline__ float fast_ln(float x) { return __builtin_amdgcn_logf(x) * 0.69314718056f; }

// All-ones if ok, else zero, in a form the compiler cannot see through. A visible "ok ? load : 0"
// is turned into a branch around the load, which then waits for it at once; x & mask with an
// opaque mask keeps a batch of loads (at clamped, always valid addresses) unconditional and in
// flight together.
__device__ __forceinline__ unsigned opaque_mask(bool ok)
{
    unsigned m = ok ? 0xFFFFFFFFu : 0u;
    asm volatile("" : "+v"(m));
    return m;
}
__device__ __forceinline__ float masked(float x, unsigned m) { return __uint_as_float(__float_as_uint(x) & m); }
__device__ __forceinline__ uint4 masked4(uint4 v, unsigned m) { return make_uint4(v.x & m, v.y & m, v.z & m, v.w & m); }

// A 4x4 transpose across the wave's four 16-lane rows: on entry lane n of row i holds M[i][j] in
// c[j]; on return lane n of row j holds M[i][j] in c[i]. Two rounds of row swaps: the first swaps
// row pairs (0,1) and (2,3) between c[0]/c[1] and c[2]/c[3], the second the wave halves between
// c[0]/c[2] and c[1]/c[3].
__device__ __forceinline__ void rows_transpose4(float (&c)[4])
{
    const auto s01 = __builtin_amdgcn_permlane16_swap(__float_as_uint(c[0]), __float_as_uint(c[1]), false, false);
    const auto s23 = __builtin_amdgcn_permlane16_swap(__float_as_uint(c[2]), __float_as_uint(c[3]), false, false);
    const auto s02 = __builtin_amdgcn_permlane32_swap(s01[0], s23[0], false, false);
    const auto s13 = __builtin_amdgcn_permlane32_swap(s01[1], s23[1], false, false);
    c[0] = __uint_as_float(s02[0]);
    c[1] = __uint_as_float(s13[0]);
    c[2] = __uint_as_float(s02[1]);
    c[3] = __uint_as_float(s13[1]);
}

// Butterfly all-reduce within each 16-lane row of the wave.
template <typename Op>
__device__ __forceinline__ float row_allreduce(float x, Op op)
{
    x = op(x, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), kDppXor1, 0xF, 0xF, false)));
    x = op(x, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), kDppXor2, 0xF, 0xF, false)));
    x = op(x, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), kDppRowHalfMirror, 0xF, 0xF, false)));
    return op(x, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), kDppRowMirror, 0xF, 0xF, false)));
}

// Butterfly all-reduce within each 32-lane half of the wave.
template <typename Op>
__device__ __forceinline__ float half_allreduce(float x, Op op)
{
    x = op(x, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), kDppXor1, 0xF, 0xF, false)));
    x = op(x, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), kDppXor2, 0xF, 0xF, false)));
    x = op(x, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), kDppRowHalfMirror, 0xF, 0xF, false)));
    x = op(x, __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), kDppRowMirror, 0xF, 0xF, false)));
    const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return op(__uint_as_float(r16[0]), __uint_as_float(r16[1]));
}

__device__ __forceinline__ float wave_max_fast(float x)
{
    return wave_allreduce(x, [](float a, float b) { return fmaxf(a, b); });
}

__device__ __forceinline__ float wave_sum_fast(float x)
{
    return wave_allreduce(x, [](float a, float b) { return a + b; });
}

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x)
{
    auto mn = [](uint32_t a, uint32_t b) { return a < b ? a : b; };
    x = mn(x, __builtin_amdgcn_update_dpp(0u, x, kDppXor1, 0xF, 0xF, false));
    x = mn(x, __builtin_amdgcn_update_dpp(0u, x, kDppXor2, 0xF, 0xF, false));
    x = mn(x, __builtin_amdgcn_update_dpp(0u, x, kDppRowHalfMirror, 0xF, 0xF, false));
    x = mn(x, __builtin_amdgcn_update_dpp(0u, x, kDppRowMirror, 0xF, 0xF, false));
    const auto r16 = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    x = mn(r16[0], r16[1]);
    const auto r32 = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    return mn(r32[0], r32[1]);
}

// Number of set bits of `mask` below this lane.
__device__ __forceinline__ int lanes_below(uint64_t mask)
{
    return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

__device__ __forceinline__ float wave_max(float x)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) x = fmaxf(x, __shfl_xor(x, m, kWave));
    return x;
}

__device__ __forceinline__ float wave_sum(float x)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, kWave);
    return x;
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t x, int m)
{
    const uint32_t lo = __shfl_xor(static_cast<uint32_t>(x), m, kWave);
    const uint32_t hi = __shfl_xor(static_cast<uint32_t>(x >> 32), m, kWave);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t x)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
        const uint64_t y = shfl_xor_u64(x, m);
        x = y > x ? y : x;
    }
    return x;
}

// ---------------------------------------------------------------------------------------------
// ranking keys for top-K
// ---------------------------------------------------------------------------------------------

// Monotone map of a float to uint32 (larger float -> larger integer); -0 and +0 map together.
__device__ __forceinline__ uint32_t ordered_bits(float f)
{
    const uint32_t u = __float_as_uint(f + 0.0f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float from_ordered_bits(uint32_t o)
{
    const uint32_t u = (o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o;
    return __uint_as_float(u);
}

// One 64-bit word per candidate: score in the high half, inverted index in the low half, so the
// unsigned order is (score descending, index ascending) when sorting for the maximum. Every valid
// candidate encodes to a nonzero word; 0 marks "no candidate".
__device__ __forceinline__ uint64_t rank_word(float score, int32_t idx)
{
    return (static_cast<uint64_t>(ordered_bits(score)) << 32) | static_cast<uint32_t>(~static_cast<uint32_t>(idx));
}

__device__ __forceinline__ int32_t rank_word_index(uint64_t w)
{
    return static_cast<int32_t>(~static_cast<uint32_t>(w));
}

__device__ __forceinline__ float rank_word_score(uint64_t w) { return from_ordered_bits(static_cast<uint32_t>(w >> 32)); }

// Exact top-`keff` selection over NPER candidates per lane, held as 32-bit ranking keys (larger is
// better, 0 = not a candidate) with distinct 32-bit names. Returns, per candidate, whether it is
// kept: every key above the cut, and at the cut the lowest names first. The cut (the keff-th
// largest key) is built bit by bit from the top with wave ballots; the search stops as soon as the
// keys at or above the partial cut number exactly keff, which for distinct scores happens after
// about log2(candidates) bits. No sorting and no LDS traffic. Requires 1 <= keff <= number of
// candidates.
template <int NPER>
__device__ __forceinline__ void wave_select_top(const uint32_t (&key)[NPER], const uint32_t (&name)[NPER], int keff,
                                                bool (&kept)[NPER])
{
    keff = __builtin_amdgcn_readfirstlane(keff);
    uint32_t cut = 0;
    int cnt = 0;                                     // keys at or above the cut, once the search ends
    if constexpr (NPER == 1) {
        // one candidate per lane: a constant trip count with an early exit, which the compiler
        // unrolls completely (a compare, a bit count and a test per bit)
        for (int bit = 31; bit >= 0; --bit) {
            const uint32_t c = cut | (1u << bit);
            const int n = __popcll(__ballot(key[0] >= c));
            if (n >= keff) {
                cut = c;
                if (n == keff) break;
            }
        }
    } else {
        // several candidates per lane: the loop stays rolled, so the cut and the bit under test
        // are kept wave-uniform in scalar registers explicitly (one scalar unit serves all the waves
        // of a compute unit, so the loop keeps its scalar work small); a bit that leaves exactly
        // keff keys at or above the cut ends the search by clearing the bit under test
        uint32_t bitv = 0x80000000u;
        while (bitv != 0u) {
            const uint32_t c = cut | bitv;
            int n = 0;
#pragma unroll
            for (int e = 0; e < NPER; ++e) n += __popcll(__ballot(key[e] >= c));
            n = __builtin_amdgcn_readfirstlane(n);
            cut = n >= keff ? c : cut;
            bitv = n == keff ? 0u : bitv >> 1;
        }
    }
#pragma unroll
    for (int e = 0; e < NPER; ++e) cnt += __popcll(__ballot(key[e] >= cut));
    if (cnt == keff) {
#pragma unroll
        for (int e = 0; e < NPER; ++e) kept[e] = key[e] >= cut;
        return;
    }
    // the cut is the keff-th largest key and more than one candidate sits on it
    int above = 0;
#pragma unroll
    for (int e = 0; e < NPER; ++e) {
        above += __popcll(__ballot(key[e] > cut));
        kept[e] = key[e] > cut;
    }
    const int need = keff - above;                   // places left for candidates at the cut
    bool open[NPER];
#pragma unroll
    for (int e = 0; e < NPER; ++e) open[e] = key[e] == cut;
    for (int r = 0; r < need; ++r) {
        uint32_t mine = 0xFFFFFFFFu;
#pragma unroll
        for (int e = 0; e < NPER; ++e)
            if (open[e] && name[e] < mine) mine = name[e];
        const uint32_t low = wave_min_u32(mine);
#pragma unroll
        for (int e = 0; e < NPER; ++e)
            if (open[e] && name[e] == low) {
                open[e] = false;
                kept[e] = true;
            }
    }
}

// Bitonic sort, descending, of NT*64 words held as word[t] in lane l at position t*64 + l.
template <int NT>
__device__ __forceinline__ void wave_bitonic_sort_desc(uint64_t (&word)[NT])
{
    const int lane = threadIdx.x & (kWave - 1);
    constexpr int n = NT * kWave;
#pragma unroll
    for (int k = 2; k <= n; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j >= 1; j >>= 1) {
            if (j >= kWave) {
                const int tj = j / kWave;
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    if (t & tj) continue;
                    const int e = t * kWave + lane;            // lower element of the pair
                    const bool desc = (e & k) == 0;
                    const uint64_t a = word[t], b = word[t | tj];
                    const bool swap = desc ? (b > a) : (a > b);
                    word[t] = swap ? b : a;
                    word[t | tj] = swap ? a : b;
                }
            } else {
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    const int e = t * kWave + lane;
                    const uint64_t other = shfl_xor_u64(word[t], j);
                    const bool lower = (e & j) == 0;
                    const bool desc = (e & k) == 0;
                    const bool take_max = (lower == desc);
                    const bool other_bigger = other > word[t];
                    word[t] = (take_max == other_bigger) ? other : word[t];
                }
            }
        }
    }
}

}  // namespace qta
