// Shared device helpers of the GPU library (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint16_t bf16_t;  // raw bfloat16 bits in memory
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

#define EBRL_DEV __device__ __forceinline__

EBRL_DEV float bf16_to_f32(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// Round to nearest even (v_cvt_pk_bf16_f32).
EBRL_DEV bf16_t f32_to_bf16(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

// Element loads/stores templated on the storage type (float or bf16_t).
template <typename T> EBRL_DEV float ld_elem(const T* p);
template <> EBRL_DEV float ld_elem<float>(const float* p) { return *p; }
template <> EBRL_DEV float ld_elem<bf16_t>(const bf16_t* p) { return bf16_to_f32(*p); }
template <typename T> EBRL_DEV void st_elem(T* p, float v);
template <> EBRL_DEV void st_elem<float>(float* p, float v) { *p = v; }
template <> EBRL_DEV void st_elem<bf16_t>(bf16_t* p, float v) { *p = f32_to_bf16(v); }

// 4 consecutive elements.
template <typename T> EBRL_DEV void st4(T* p, float a, float b, float c, float d);
template <> EBRL_DEV void st4<float>(float* p, float a, float b, float c, float d) {
    *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
}
template <> EBRL_DEV void st4<bf16_t>(bf16_t* p, float a, float b, float c, float d) {
    typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
    const bf16x4_t v = {(__bf16)a, (__bf16)b, (__bf16)c, (__bf16)d};
    *reinterpret_cast<bf16x4_t*>(p) = v;
}

// Cross-lane reductions without LDS round trips where possible: DPP
// quad_perm / row_half_mirror / row_mirror / row_ror inside 16-lane rows,
// ds_swizzle (xor 16 inside 32 lanes) across rows, v_readlane across the two
// wave halves.  Float add and max are commutative, so the two lanes of every
// exchange compute the same value and a reduction leaves every lane of its
// group with the identical result.
template <int CTRL> EBRL_DEV float dpp_f(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
constexpr int DPP_SWAP1 = 0xB1;        // quad_perm [1, 0, 3, 2]
constexpr int DPP_SWAP2 = 0x4E;        // quad_perm [2, 3, 0, 1]
constexpr int DPP_HALF_MIRROR = 0x141; // lane i <-> 7 - i within 8
constexpr int DPP_MIRROR = 0x140;      // lane i <-> 15 - i within 16
constexpr int DPP_ROR8 = 0x128;        // lane i <- lane (i + 8) % 16 within 16
EBRL_DEV float swz_xor16_f(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x401F));
}
// sum over each aligned group of 8 / 16 lanes
EBRL_DEV float sum_lanes8(float v) {
    v += dpp_f<DPP_SWAP1>(v);
    v += dpp_f<DPP_SWAP2>(v);
    return v + dpp_f<DPP_HALF_MIRROR>(v);
}
EBRL_DEV float sum_lanes16(float v) { v = sum_lanes8(v); return v + dpp_f<DPP_MIRROR>(v); }
EBRL_DEV float max_lanes16(float v) {
    v = fmaxf(v, dpp_f<DPP_SWAP1>(v));
    v = fmaxf(v, dpp_f<DPP_SWAP2>(v));
    v = fmaxf(v, dpp_f<DPP_HALF_MIRROR>(v));
    return fmaxf(v, dpp_f<DPP_MIRROR>(v));
}
EBRL_DEV float readlane_f(float v, int l) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}
EBRL_DEV float wave_sum(float v) {
    v = sum_lanes16(v);
    v += swz_xor16_f(v);
    return readlane_f(v, 0) + readlane_f(v, 32);
}
EBRL_DEV float wave_max(float v) {
    v = max_lanes16(v);
    v = fmaxf(v, swz_xor16_f(v));
    return fmaxf(readlane_f(v, 0), readlane_f(v, 32));
}

// Block-wide sum over blockDim.x threads (multiple of 64, <= 1024); every
// thread gets the result.  `red` must hold 16 floats of shared memory.
EBRL_DEV float block_sum(float v, float* red) {
    v = wave_sum(v);
    const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int nw = blockDim.x >> 6;
    __syncthreads();
    if (lane == 0) red[w] = v;
    __syncthreads();
    float t = 0.f;
    for (int i = 0; i < nw; ++i) t += red[i];
    return t;
}

EBRL_DEV float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

constexpr int KV_BLOCK = 16;  // tokens per paged-KV block

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// Buffer accesses with the device-coherence cache policy bit (sc1): they
// bypass the per-XCD L2s, the same policy the compiler uses for agent-scope
// atomic loads and stores, so data one workgroup writes is read correctly by
// a workgroup on another XCD without cache-wide write-back or invalidation.
// Used for in-kernel hand-offs: the writer waits for its stores (vmcnt 0)
// before bumping a device-scope counter; the reader loads after seeing the
// final count.
constexpr int CPOL_SC1 = 16;
EBRL_DEV __amdgpu_buffer_rsrc_t coherent_rsrc(float* base) {
    return __builtin_amdgcn_make_buffer_rsrc(base, 0, 0x7fffffff, 0x00020000);
}
EBRL_DEV void st_coherent4(__amdgpu_buffer_rsrc_t r, int byte_off, f32x4 v) {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, byte_off, 0, CPOL_SC1);
}
EBRL_DEV f32x4 ld_coherent4(__amdgpu_buffer_rsrc_t r, int byte_off) {
    return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, CPOL_SC1));
}
EBRL_DEV void st_coherent1(__amdgpu_buffer_rsrc_t r, int byte_off, float v) {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), r, byte_off, 0, CPOL_SC1);
}
EBRL_DEV float ld_coherent1(__amdgpu_buffer_rsrc_t r, int byte_off) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, byte_off, 0, CPOL_SC1));
}
