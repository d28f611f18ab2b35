// Device-side building blocks of the gfx950 routing kernels: 16-byte vector
// loads and stores with fp32 widening / bf16 narrowing, and wave64
// reductions.  Storage types: float, or uint16_t holding bf16 bits.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lrar {

constexpr int kWaveSize = 64;

typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned u32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Raw<T, VEC>::type is what one lane moves per access: 16 bytes for the
// vector paths (4 fp32 or 8 bf16), one element for the scalar paths.
template <typename T, int VEC> struct Raw;
template <> struct Raw<float, 4> { typedef f32x4_t type; };
template <> struct Raw<float, 1> { typedef float type; };
template <> struct Raw<uint16_t, 8> { typedef u32x4_t type; };
template <> struct Raw<uint16_t, 4> { typedef u32x2_t type; };  // 4 bf16 in 8 bytes
template <> struct Raw<uint16_t, 1> { typedef uint16_t type; };

template <typename T> struct VecOf;
template <> struct VecOf<float> { static constexpr int value = 4; };
template <> struct VecOf<uint16_t> { static constexpr int value = 8; };

__device__ __forceinline__ float bf16_lo(unsigned w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(unsigned w) { return __uint_as_float(w & 0xffff0000u); }

// Round two fp32 to bf16 (nearest even; gfx950 v_cvt_pk_bf16_f32) and pack.
__device__ __forceinline__ unsigned pack_bf16x2(float a, float b)
{
    f32x2_t v = {a, b};
    return __builtin_bit_cast(unsigned, __builtin_convertvector(v, bf16x2_t));
}

__device__ __forceinline__ uint16_t to_bf16(float a)
{
    return (uint16_t)(pack_bf16x2(a, 0.0f) & 0xffffu);
}

template <typename T, int VEC>
__device__ __forceinline__ typename Raw<T, VEC>::type load_raw(const T *p)
{
    return *reinterpret_cast<const typename Raw<T, VEC>::type *>(p);
}

template <typename T, int VEC>
__device__ __forceinline__ void store_raw(T *p, typename Raw<T, VEC>::type v)
{
    *reinterpret_cast<typename Raw<T, VEC>::type *>(p) = v;
}

// Streaming variants: data touched exactly once, marked non-temporal so it
// does not displace reusable lines (keys, the token's dH row) in the caches.
template <typename T, int VEC, bool NT>
__device__ __forceinline__ typename Raw<T, VEC>::type load_stream(const T *p)
{
    typedef typename Raw<T, VEC>::type raw_t;
    if constexpr (NT)
        return __builtin_nontemporal_load(reinterpret_cast<const raw_t *>(p));
    else
        return *reinterpret_cast<const raw_t *>(p);
}

template <typename T, int VEC, bool NT>
__device__ __forceinline__ void store_stream(T *p, typename Raw<T, VEC>::type v)
{
    typedef typename Raw<T, VEC>::type raw_t;
    if constexpr (NT)
        __builtin_nontemporal_store(v, reinterpret_cast<raw_t *>(p));
    else
        *reinterpret_cast<raw_t *>(p) = v;
}

// Raw (untyped) buffer accesses of 16 bytes.  A buffer resource describes
// one row: its base address and its size in bytes.  An access at or past
// the size is dropped by the hardware (a load returns zeros), so a range
// check becomes a size in the scalar descriptor instead of a branch around
// the access.  NT marks the access non-temporal.
constexpr int kRawBufferWord3 = 0x00020000;  // word 3 of a raw buffer resource (gfx9 family)

__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const void *base, int bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, bytes, kRawBufferWord3);
}

template <typename T, int VEC, bool NT>
__device__ __forceinline__ typename Raw<T, VEC>::type buffer_load16(__amdgpu_buffer_rsrc_t r,
                                                                    int byte_off)
{
    typedef typename Raw<T, VEC>::type raw_t;
    static_assert(sizeof(raw_t) == 16, "16-byte accesses only");
    return __builtin_bit_cast(raw_t, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, NT ? 2 : 0));
}

template <typename T, int VEC, bool NT>
__device__ __forceinline__ void buffer_store16(__amdgpu_buffer_rsrc_t r, int byte_off,
                                               typename Raw<T, VEC>::type v)
{
    static_assert(sizeof(v) == 16, "16-byte accesses only");
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, v), r, byte_off, 0,
                                           NT ? 2 : 0);
}

// Widen one raw access to VEC fp32 values (exact).
__device__ __forceinline__ void widen(const f32x4_t &r, float (&x)[4])
{
    x[0] = r.x; x[1] = r.y; x[2] = r.z; x[3] = r.w;
}
__device__ __forceinline__ void widen(const float &r, float (&x)[1]) { x[0] = r; }
__device__ __forceinline__ void widen(const u32x4_t &r, float (&x)[8])
{
    x[0] = bf16_lo(r.x); x[1] = bf16_hi(r.x);
    x[2] = bf16_lo(r.y); x[3] = bf16_hi(r.y);
    x[4] = bf16_lo(r.z); x[5] = bf16_hi(r.z);
    x[6] = bf16_lo(r.w); x[7] = bf16_hi(r.w);
}
__device__ __forceinline__ void widen(const u32x2_t &r, float (&x)[4])
{
    x[0] = bf16_lo(r.x); x[1] = bf16_hi(r.x);
    x[2] = bf16_lo(r.y); x[3] = bf16_hi(r.y);
}
__device__ __forceinline__ void widen(const uint16_t &r, float (&x)[1])
{
    x[0] = __uint_as_float((unsigned)r << 16);
}

// Narrow VEC fp32 values to one raw access (bf16: round to nearest even).
template <typename T, int VEC> struct Narrow;
template <> struct Narrow<float, 4> {
    __device__ static f32x4_t run(const float (&x)[4]) { return f32x4_t{x[0], x[1], x[2], x[3]}; }
};
template <> struct Narrow<float, 1> {
    __device__ static float run(const float (&x)[1]) { return x[0]; }
};
template <> struct Narrow<uint16_t, 8> {
    __device__ static u32x4_t run(const float (&x)[8])
    {
        return u32x4_t{pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]),
                       pack_bf16x2(x[4], x[5]), pack_bf16x2(x[6], x[7])};
    }
};
template <> struct Narrow<uint16_t, 4> {
    __device__ static u32x2_t run(const float (&x)[4])
    {
        return u32x2_t{pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3])};
    }
};
template <> struct Narrow<uint16_t, 1> {
    __device__ static uint16_t run(const float (&x)[1]) { return to_bf16(x[0]); }
};

// y += the VEC values of one stored raw access (accumulating outputs).
template <int VEC, typename R>
__device__ __forceinline__ void add_stored(float (&y)[VEC], const R &stored)
{
    float x[VEC];
    widen(stored, x);
#pragma unroll
    for (int e = 0; e < VEC; ++e)
        y[e] += x[e];
}

__device__ __forceinline__ float load_elem(const float *p) { return *p; }
__device__ __forceinline__ float load_elem(const uint16_t *p)
{
    return __uint_as_float((unsigned)*p << 16);
}
__device__ __forceinline__ void store_elem(float *p, float v) { *p = v; }
__device__ __forceinline__ void store_elem(uint16_t *p, float v) { *p = to_bf16(v); }

// One data-parallel-primitive move: lane i receives the value of the lane
// that CTRL selects within its row of 16 (every lane active).
template <int CTRL>
__device__ __forceinline__ float dpp_move(float v)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppXor1 = 0xB1;         // quad_perm [1, 0, 3, 2]: lane i^1
constexpr int kDppXor2 = 0x4E;         // quad_perm [2, 3, 0, 1]: lane i^2
constexpr int kDppHalfMirror = 0x141;  // row_half_mirror: lane 7 - i within each 8
constexpr int kDppMirror = 0x140;      // row_mirror: lane 15 - i within the row

// Sum over aligned groups of g lanes (g a power of two, 1..64, the same on
// every lane), every lane of a group receiving its group's sum, with the
// pairings of a xor butterfly over lane bits 1, 2, 4, ...: bits 1 and 2 are
// quad permutes; bits 4 and 8 mirror the quad within the half row and the
// half within the row, which pair exactly as xor 4 and xor 8 do once the
// earlier steps have made every quad (half row) hold one value; bits 16 and
// 32 cross rows through LDS permutes.  Same bits as the butterfly, with four
// of its six lane exchanges as DPP moves instead of LDS permutes.
__device__ __forceinline__ float group_sum(float v, int g)
{
    if (g > 1)
        v += dpp_move<kDppXor1>(v);
    if (g > 2)
        v += dpp_move<kDppXor2>(v);
    if (g > 4)
        v += dpp_move<kDppHalfMirror>(v);
    if (g > 8)
        v += dpp_move<kDppMirror>(v);
    if (g > 16)
        v += __shfl_xor(v, 16, kWaveSize);
    if (g > 32)
        v += __shfl_xor(v, 32, kWaveSize);
    return v;
}

__device__ __forceinline__ float group_max(float v, int g)
{
    if (g > 1)
        v = fmaxf(v, dpp_move<kDppXor1>(v));
    if (g > 2)
        v = fmaxf(v, dpp_move<kDppXor2>(v));
    if (g > 4)
        v = fmaxf(v, dpp_move<kDppHalfMirror>(v));
    if (g > 8)
        v = fmaxf(v, dpp_move<kDppMirror>(v));
    if (g > 16)
        v = fmaxf(v, __shfl_xor(v, 16, kWaveSize));
    if (g > 32)
        v = fmaxf(v, __shfl_xor(v, 32, kWaveSize));
    return v;
}

// Butterfly reductions over the 64 lanes of a wave; every lane gets the result.
__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1)
        v += __shfl_xor(v, m, kWaveSize);
    return v;
}

__device__ __forceinline__ float wave_max(float v)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1)
        v = fmaxf(v, __shfl_xor(v, m, kWaveSize));
    return v;
}

// Wave reductions with DPP moves for the lane bits within a row (DPP) or
// the LDS-permute butterflies above; the sum's order differs between the two.
template <bool DPP>
__device__ __forceinline__ float wave_sum_t(float v)
{
    return DPP ? group_sum(v, kWaveSize) : wave_sum(v);
}
template <bool DPP>
__device__ __forceinline__ float wave_max_t(float v)
{
    return DPP ? group_max(v, kWaveSize) : wave_max(v);
}

// Two sums over aligned groups of g lanes by the xor butterfly over lane
// bits 1, 2, 4, ..., step by step together so that the two chains overlap:
// with DPP moves for bits 1-8 (as group_sum) or with LDS lane permutes only
// (same bits either way).
template <bool DPP>
__device__ __forceinline__ void butterfly_sum2(float &a, float &b, int g)
{
    if constexpr (DPP) {
        if (g > 1) {
            a += dpp_move<kDppXor1>(a);
            b += dpp_move<kDppXor1>(b);
        }
        if (g > 2) {
            a += dpp_move<kDppXor2>(a);
            b += dpp_move<kDppXor2>(b);
        }
        if (g > 4) {
            a += dpp_move<kDppHalfMirror>(a);
            b += dpp_move<kDppHalfMirror>(b);
        }
        if (g > 8) {
            a += dpp_move<kDppMirror>(a);
            b += dpp_move<kDppMirror>(b);
        }
        for (int m = 16; m < g; m <<= 1) {
            a += __shfl_xor(a, m, kWaveSize);
            b += __shfl_xor(b, m, kWaveSize);
        }
        return;
    }
    for (int m = 1; m < g; m <<= 1) {
        a += __shfl_xor(a, m, kWaveSize);
        b += __shfl_xor(b, m, kWaveSize);
    }
}

// Sum M per-lane values (M a power of two, M <= 64) over the wave with
// log2(M) halving exchanges followed by plain butterflies: at each halving
// step a lane keeps the half of its values selected by one lane bit and
// receives its partner's copy of that half.  On return lane l holds the
// wave-wide sum of value index multi_sum_index<M>(l).
template <int M>
__device__ __forceinline__ float multi_sum(float (&v)[M], int lane)
{
    int bit = kWaveSize / 2;
#pragma unroll
    for (int half = M / 2; half >= 1; half >>= 1, bit >>= 1) {
        const bool upper = (lane & bit) != 0;
#pragma unroll
        for (int k = 0; k < half; ++k) {
            float keep = upper ? v[k + half] : v[k];
            float give = upper ? v[k] : v[k + half];
            v[k] = keep + __shfl_xor(give, bit, kWaveSize);
        }
    }
    float s = v[0];
    for (; bit >= 1; bit >>= 1)
        s += __shfl_xor(s, bit, kWaveSize);
    return s;
}

// Value index whose sum multi_sum<M> leaves in lane `lane`: the lane bits
// 32, 16, ... consumed by the halving steps, most significant first.
template <int M>
__device__ __forceinline__ int multi_sum_index(int lane)
{
    int idx = 0, bit = kWaveSize / 2;
#pragma unroll
    for (int half = M / 2; half >= 1; half >>= 1, bit >>= 1)
        idx += (lane & bit) ? half : 0;
    return idx;
}

// True on exactly one lane per value index after multi_sum<M>.
template <int M>
__device__ __forceinline__ bool multi_sum_writer(int lane)
{
    constexpr int low_bits = kWaveSize / M;  // lanes sharing one value index
    return (lane & (low_bits - 1)) == 0;
}

// After multi_sum<M>, the sum of value index k, read from one lane that holds
// it (the lane whose bits 32, 16, ... spell k, most significant first).
template <int M>
__device__ __forceinline__ float lane_value(float tot, int k)
{
    int src = 0, bit = kWaveSize / 2;
#pragma unroll
    for (int half = M / 2; half >= 1; half >>= 1, bit >>= 1)
        src += (k & half) ? bit : 0;
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(tot), src));
}

// Make this wave's LDS writes visible to its other lanes.
__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

}  // namespace lrar
