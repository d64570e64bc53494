// Device helpers for the gfx950 COUNTDOWN kernels: 16-byte bf16 row loads,
// bf16 dot products on v_dot2_f32_bf16, DPP wavefront reductions, SiLU.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cdk {

constexpr int kWave = 64;                     // CDNA wavefront width
constexpr int kBlock = 256;                   // threads per workgroup (4 waves)
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kColsPerLoad = kWave * 8;       // bf16 columns covered by one wave-wide 16 B load
constexpr int kMaxRowsPerBlock = 64;          // one ballot word of local rows

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4 load16(const uint16_t *p)
{
    return *reinterpret_cast<const u32x4 *>(p);
}

__device__ __forceinline__ u32x4 zero16()
{
    u32x4 z = {0u, 0u, 0u, 0u};
    return z;
}

// a.lo*b.lo + a.hi*b.hi + c for two packed bf16 pairs, fp32 accumulate
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c)
{
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                           __builtin_bit_cast(bf16x2_t, b), c, false);
}

// 8-element bf16 dot product of two 16-byte chunks added to acc
__device__ __forceinline__ float dot8(const u32x4 &w, const u32x4 &x, float acc)
{
    acc = dot2_bf16(w.x, x.x, acc);
    acc = dot2_bf16(w.y, x.y, acc);
    acc = dot2_bf16(w.z, x.z, acc);
    acc = dot2_bf16(w.w, x.w, acc);
    return acc;
}

// exact bf16 -> fp32 of the low / high half of a packed pair
__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }

// DPP move of v with controls CTRL; lanes outside ROW_MASK return 0
template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ float dpp0(float v)
{
    return __builtin_bit_cast(
        float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, ROW_MASK, 0xF, false));
}

constexpr int kDppQuadSwap1 = 0xB1;   // quad_perm [1,0,3,2]
constexpr int kDppQuadSwap2 = 0x4E;   // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // row_half_mirror
constexpr int kDppMirror = 0x140;     // row_mirror
constexpr int kDppBcast15 = 0x142;    // row_bcast:15
constexpr int kDppBcast31 = 0x143;    // row_bcast:31

// Sum over aligned segments of 2^LOG lanes (LOG in 0..6). Afterwards the
// last lane of every segment holds the segment sum (for LOG <= 4 every lane
// of the segment does).
template <int LOG>
__device__ __forceinline__ float segment_sum(float v)
{
    if constexpr (LOG >= 1) v += dpp0<kDppQuadSwap1>(v);
    if constexpr (LOG >= 2) v += dpp0<kDppQuadSwap2>(v);
    if constexpr (LOG >= 3) v += dpp0<kDppHalfMirror>(v);
    if constexpr (LOG >= 4) v += dpp0<kDppMirror>(v);
    if constexpr (LOG >= 5) v += dpp0<kDppBcast15, 0xA>(v);
    if constexpr (LOG >= 6) v += dpp0<kDppBcast31, 0xC>(v);
    return v;
}

// Sum over the 64 lanes of a wave, returned uniformly to every lane.
__device__ __forceinline__ float wave_sum(float v)
{
    v = segment_sum<6>(v);
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

// SiLU(z) = z * sigmoid(z) (the Gated-MLP activation); saturates to -0 / z
// without NaN for large |z|.
__device__ __forceinline__ float silu(float z)
{
    return z / (1.0f + expf(-z));
}

__device__ __forceinline__ uint64_t ballot(bool p)
{
    return __ballot(p);
}

// number of set bits of m below this lane
__device__ __forceinline__ int lanes_below(uint64_t m)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

} // namespace cdk
