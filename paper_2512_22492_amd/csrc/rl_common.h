// rl_common.h -- shared device helpers of the decode-attention library
// (gfx950).  Internal header: included by the library's .hip sources only.
#pragma once

#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include "rl_decode_attn.h"

namespace rl_da {

constexpr int kHeadDim = 128;
constexpr int kPageSize = 16;
constexpr int kWave = 64;
constexpr int kUnitWaves = 4;  // wavefronts per work unit (decode and extend)
constexpr float kLog2e = 1.4426950408889634f;
// The online softmax's reference max moves only when a page's max exceeds it
// by more than this (log2 units); probabilities then stay <= 2^kMaxSlack.
constexpr float kMaxSlack = 8.0f;

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx2_t __attribute__((ext_vector_type(2)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// RL_DA_LAYOUT_HND_KV keeps both pools in one allocation: the value pool must
// start one slab after the key pool (elt-byte elements).  Other layouts take
// any two pools.
inline bool pools_paired(int32_t layout, const void* k_pool, const void* v_pool, int32_t elt)
{
    return layout != RL_DA_LAYOUT_HND_KV ||
           (const uint8_t*)v_pool == (const uint8_t*)k_pool + kPageSize * kHeadDim * elt;
}

// Byte strides of a pool of elt-byte elements: per page, per kv head within a
// page, per token slot within a (page, kv head) slab.  Both pools use the
// same strides from their own base.
struct PoolStrides {
    int64_t page;
    int32_t head;
    int32_t row;
};

// false for an unknown layout
inline bool pool_strides(int32_t layout, int32_t num_kv_heads, int32_t elt, PoolStrides* s)
{
    const int32_t row = kHeadDim * elt;
    s->page = (int64_t)num_kv_heads * kPageSize * row;
    if (layout == RL_DA_LAYOUT_HND) {
        s->head = kPageSize * row;
        s->row = row;
        return true;
    }
    if (layout == RL_DA_LAYOUT_HND_KV) {  // K slab, then V slab, per (page, kv head)
        s->page *= 2;
        s->head = 2 * kPageSize * row;
        s->row = row;
        return true;
    }
    if (layout == RL_DA_LAYOUT_NHD) {
        s->head = row;
        s->row = num_kv_heads * row;
        return true;
    }
    return false;
}

// ------------------------------------------------------------ helpers ---

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two fp32 values as packed bf16 (one v_cvt_pk_bf16_f32, round to nearest
// even), a in the low half.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b)
{
    const f32x2_t v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 bits, round to nearest even (quiet NaN kept NaN).
__device__ __forceinline__ uint32_t f32_to_bf16(float f)
{
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u)
        return 0x7fc0u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c)
{
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                           __builtin_bit_cast(bf16x2_t, b), c, false);
}

// DPP lane permutations inside a 16-lane row.  quad_perm [1,0,3,2] and
// [2,3,0,1] pair lanes within a quad; row_half_mirror pairs the two quads of
// each 8-lane half; row_mirror pairs the two halves.  Applied in turn they
// combine all 16 lanes of a row.
constexpr int kDppQuadXor1 = 0xB1;
constexpr int kDppQuadXor2 = 0x4E;
constexpr int kDppRowHalfMirror = 0x141;
constexpr int kDppRowMirror = 0x140;

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v)
{
    return __int_as_float(
        __builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}

__device__ __forceinline__ float row16_sum(float v)
{
    v += dpp_f32<kDppQuadXor1>(v);
    v += dpp_f32<kDppQuadXor2>(v);
    v += dpp_f32<kDppRowHalfMirror>(v);
    v += dpp_f32<kDppRowMirror>(v);
    return v;
}

__device__ __forceinline__ float row16_max(float v)
{
    v = fmaxf(v, dpp_f32<kDppQuadXor1>(v));
    v = fmaxf(v, dpp_f32<kDppQuadXor2>(v));
    v = fmaxf(v, dpp_f32<kDppRowHalfMirror>(v));
    v = fmaxf(v, dpp_f32<kDppRowMirror>(v));
    return v;
}

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// Loads with the non-temporal hint: K/V bytes are read exactly once, so they
// are streamed past the caches rather than kept.
__device__ __forceinline__ uint4 load_stream16(const uint8_t* p)
{
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ uint2 load_stream8(const uint8_t* p)
{
    const u32x2_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(p));
    return make_uint2(v.x, v.y);
}

// Orders LDS traffic between the lanes of one wavefront (the work-group is
// a single wavefront, so no s_barrier and no wait on global loads is needed).
__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ void unpack8(const uint4& w, float (&v)[8])
{
    v[0] = bf16_lo(w.x); v[1] = bf16_hi(w.x);
    v[2] = bf16_lo(w.y); v[3] = bf16_hi(w.y);
    v[4] = bf16_lo(w.z); v[5] = bf16_hi(w.z);
    v[6] = bf16_lo(w.w); v[7] = bf16_hi(w.w);
}

}  // namespace rl_da
