// Device-side helpers shared by the attention kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <tuple>

namespace moa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr float kNegInf = -__builtin_inff();
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// 2^x on the hardware transcendental unit (v_exp_f32).
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// bf16 bit pattern -> fp32 (exact).
__device__ __forceinline__ float bf16lo_to_f32(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi_to_f32(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 bits, round to nearest even (finite inputs; NaN stays NaN-ish).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return f32_to_bf16_bits(lo) | (f32_to_bf16_bits(hi) << 16);
}

// Cross-lane moves inside a row of 16 lanes via DPP.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
constexpr int kDppQuadXor1 = 0xB1;      // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;      // quad_perm [2,3,0,1]
constexpr int kDppRowHalfMirror = 0x141;
constexpr int kDppRowMirror = 0x140;

// Sum over aligned groups of G lanes (G in {1,2,4,8,16,32,64}); every lane of a
// group ends with the group total.
template <int G>
__device__ __forceinline__ float group_sum(float x) {
    if constexpr (G >= 2) x += dpp_f32<kDppQuadXor1>(x);
    if constexpr (G >= 4) x += dpp_f32<kDppQuadXor2>(x);
    if constexpr (G >= 8) x += dpp_f32<kDppRowHalfMirror>(x);
    if constexpr (G >= 16) x += dpp_f32<kDppRowMirror>(x);
    if constexpr (G >= 32) x += __shfl_xor(x, 16);
    if constexpr (G >= 64) x += __shfl_xor(x, 32);
    return x;
}

// 16-byte streaming load with the non-temporal hint (data read once).
__device__ __forceinline__ uint4 load_nt16(const void* p) {
    const u32x4 v = __builtin_nontemporal_load(static_cast<const u32x4*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

// Enqueue a kernel and return the status of THIS launch.  (hipGetLastError()
// after a triple-chevron launch would also report errors left on the thread
// by unrelated earlier runtime calls, e.g. a not-ready event query.)
template <typename... Params, typename... Args>
inline hipError_t launch_kernel(void (*kernel)(Params...), dim3 grid, dim3 block,
                                hipStream_t stream, Args... args) {
    static_assert(sizeof...(Params) == sizeof...(Args), "argument count mismatch");
    auto typed = std::make_tuple(static_cast<Params>(args)...);
    void* argv[sizeof...(Params)];
    std::apply([&](auto&... a) {
        int i = 0;
        ((argv[i++] = static_cast<void*>(&a)), ...);
    }, typed);
    return hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, argv, 0, stream);
}

// Element offset of the (batch*head) slice bh of a tensor with batch stride
// sb and head stride sh, H heads.
__device__ __forceinline__ long long head_offset(int bh, int H, long long sb, long long sh) {
    const int b = bh / H;
    return (long long)b * sb + (long long)(bh - b * H) * sh;
}

// Bytes spanned by n rows of row_bytes each, row_stride_bytes apart (the
// extent a buffer descriptor over those rows must cover).
__device__ __forceinline__ uint32_t rows_extent(int n, uint32_t row_stride_bytes, uint32_t row_bytes) {
    return n > 0 ? (uint32_t)(n - 1) * row_stride_bytes + row_bytes : 0u;
}

// Raw buffer access: a descriptor over [base, base + bytes).  Loads beyond
// `bytes` return zeros instead of touching memory, which is how ragged tiles
// are padded without per-lane clamping.  (Descriptor word 3 for gfx9-family.)
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ uint4 buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t voffset) {
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voffset, 0, 0);
    return make_uint4(v.x, v.y, v.z, v.w);
}

// 16 bytes per lane from a buffer straight into LDS (buffer_load_dwordx4 ...
// lds): lane l's data lands at lds_base + 16*l, lds_base being wave-uniform.
// The builtin exists only for the device pass; in the host pass a call to it
// makes clang drop the kernel's host-side stub, so the host pass sees an empty
// body (it never runs device code).
__device__ __forceinline__ void buffer_load16_to_lds(__amdgpu_buffer_rsrc_t r, void* lds_base,
                                                     uint32_t voffset) {
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        r, (__attribute__((address_space(3))) void*)lds_base, 16, voffset, 0, 0, 0);
#else
    (void)r; (void)lds_base; (void)voffset;
#endif
}

// Combine the two half-waves (lanes l and l ^ 32) with v_permlane32_swap:
// swapping x with itself leaves {x[l % 32], x[l % 32 + 32]} in every lane.
__device__ __forceinline__ float half_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float half_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Wave-uniform "any lane" test.
__device__ __forceinline__ bool wave_any(bool pred) { return __ballot(pred) != 0; }

}  // namespace moa
