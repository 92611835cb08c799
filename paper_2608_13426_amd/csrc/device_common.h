// Device helpers shared by librmm's kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rmm {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned short u16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// fp32 -> bf16 bits, round to nearest even; NaN stays a quiet NaN with its
// sign and top payload bits (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

// two fp32 -> one register of packed bf16 (lo in bits 0-15), same rounding
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    bf16x2_t v;
    v.x = static_cast<__bf16>(lo);
    v.y = static_cast<__bf16>(hi);
    return __builtin_bit_cast(uint32_t, v);
}

constexpr int kWave = 64;

typedef short s16x4_t __attribute__((ext_vector_type(4)));

// Workgroup barrier for LDS hand-offs.  __syncthreads() also waits for every
// outstanding global load and store of the wave (its workgroup-scope fence),
// which stalls a kernel that streams stores out while it computes; this one
// waits only for the wave's own LDS accesses, and no instruction is
// scheduled across it.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_barrier" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

// The two gfx950 LDS instructions below exist only in the device pass; the
// host pass of a kernel that names them directly drops the kernel's launch
// stub, so they are wrapped here.

// ds_read_b64_tr_b16 at LDS byte address `lds`: within each 16-lane group,
// lane l receives element l%4 of the 8-byte words addressed by lanes
// 4v + (l%16)/4, v = 0..3 of its group (a 4x4 transpose of 16-bit values).
__device__ __forceinline__ s16x4_t lds_read_tr16(const void *lds) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t *)(lds));
#else
    (void)lds;
    return s16x4_t{};
#endif
}

// 16-byte buffer load straight into LDS: lane i's data lands at lds + 16*i
// (`lds` must be the same for the whole wave).  Offsets past the
// descriptor's range stage zeros.
__device__ __forceinline__ void lds_load16(__amdgpu_buffer_rsrc_t rsrc, void *lds, uint32_t voffset) {
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void *)(lds), 16,
                                             voffset, 0, 0, 0);
#else
    (void)rsrc; (void)lds; (void)voffset;
#endif
}

// x of the lane that the DPP control CTRL names within its row of 16 lanes
// (0xB1: lane ^ 1, 0x4E: lane ^ 2, 0x141: the mirror within 8 lanes), for a
// float64 value (two 32-bit moves); every lane must be active.
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x) {
#if defined(__HIP_DEVICE_COMPILE__)
    const uint64_t u = static_cast<uint64_t>(__double_as_longlong(x));
    const uint32_t lo = static_cast<uint32_t>(
        __builtin_amdgcn_update_dpp(0, static_cast<int>(static_cast<uint32_t>(u)), CTRL, 0xF, 0xF, false));
    const uint32_t hi = static_cast<uint32_t>(
        __builtin_amdgcn_update_dpp(0, static_cast<int>(static_cast<uint32_t>(u >> 32)), CTRL, 0xF, 0xF, false));
    return __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(hi) << 32) | lo));
#else
    return x;
#endif
}

}  // namespace rmm
