// device_common.h -- small device-side helpers shared by the gfx950 kernels:
// buffer-resource loads/stores (hardware range checking returns 0 for an
// out-of-range load and drops an out-of-range store), bf16 conversion, and
// the MFMA fragment types.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace caffe_hip {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
// LDS destination of the global -> LDS buffer copies
typedef __attribute__((address_space(3))) void lds_void;

// Word 3 of a raw (stride 0) buffer resource on gfx9-class parts: 32-bit
// data format, no swizzle.  With stride 0 the range check compares the byte
// offset with num_records.
constexpr uint32_t kBufferWord3 = 0x00020000u;
// Byte offset that is always out of range (every tensor is < 2^31 bytes).
constexpr uint32_t kOob = 0x80000000u;
// s_waitcnt immediate that waits for vmcnt(0) only (expcnt and lgkmcnt left
// at their maxima): all of this wave's vector-memory loads, including
// global-to-LDS copies, have completed.
constexpr int kVmcnt0 = 0x0F70;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                             (int)kBufferWord3);
}

__device__ __forceinline__ float buf_ld_f32(__amdgpu_buffer_rsrc_t r, uint32_t byte_off)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, byte_off, 0, 0));
}

__device__ __forceinline__ u32x4 buf_ld_b128(__amdgpu_buffer_rsrc_t r, uint32_t byte_off)
{
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0));
}

__device__ __forceinline__ uint16_t buf_ld_u16(__amdgpu_buffer_rsrc_t r, uint32_t byte_off)
{
    return __builtin_amdgcn_raw_buffer_load_b16(r, byte_off, 0, 0);
}

__device__ __forceinline__ uint8_t buf_ld_u8(__amdgpu_buffer_rsrc_t r, uint32_t byte_off)
{
    return __builtin_amdgcn_raw_buffer_load_b8(r, byte_off, 0, 0);
}

__device__ __forceinline__ void buf_st_f32(float v, __amdgpu_buffer_rsrc_t r, uint32_t byte_off)
{
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), r, byte_off, 0, 0);
}

// float -> bfloat16 bits, round to nearest even (a NaN stays a quiet NaN):
// gfx950's conversion instruction, one per value or per pair.
typedef __bf16 bf16x2_cvt __attribute__((ext_vector_type(2)));
typedef float f32x2_cvt __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f)
{
    return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// (lo, hi) -> their bfloat16 bits packed, lo in the low half
__device__ __forceinline__ uint32_t f32x2_to_bf16x2_rne(float lo, float hi)
{
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_cvt{lo, hi}, bf16x2_cvt));
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h)
{
    return __builtin_bit_cast(float, (uint32_t)h << 16);
}

// x / f.d for x < 2^31 (see FastDiv).
__device__ __forceinline__ uint32_t fdiv(uint32_t x, const FastDiv& f)
{
    return (uint32_t)(((uint64_t)x * f.mul) >> f.shift);
}

// MFMA results regrouped as output rows across the lanes.  A wave's NI
// accumulator blocks of MT columns (NI * MT == 64) hold, in register q,
//   MT = 32: row 8*(q/4) + q%4 + 4*(lane/32) of column 32*ni + lane%32,
//   MT = 16: row 4*(lane/16) + q of column 16*ni + lane%16.
// Lane swaps regroup them so that value h of get(acc, q) is row row(q, h)
// of column `lane` (0..63): a store of one value per lane then writes 64
// consecutive columns of one row instead of 32 columns of two rows.  Used by
// the fp32 GEMM epilogues (the CaffeNet fp32 step runs ~1% faster with it;
// the bf16 step ran 2% slower, so the bf16 kernels keep the MFMA layout).
//   v_permlane32_swap(x, y): x.lanes[32,64) <-> y.lanes[0,32)
//   v_permlane16_swap(x, y): x.lanes[16,32) <-> y.lanes[0,16), x.lanes[48,64) <-> y.lanes[32,48)
template <int MT>
struct WaveRows;

template <>
struct WaveRows<32> {
    static constexpr int kRows = 2;
    static __device__ __forceinline__ int row(int q, int h) { return 8 * (q >> 2) + (q & 3) + 4 * h; }
    // x[ni] = register q of accumulator block ni
    static __device__ __forceinline__ void get(const float* x, float* out)
    {
        const auto s = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, x[0]),
                                                        __builtin_bit_cast(uint32_t, x[1]), false,
                                                        false);
        out[0] = __builtin_bit_cast(float, (uint32_t)s[0]);
        out[1] = __builtin_bit_cast(float, (uint32_t)s[1]);
    }
};

template <>
struct WaveRows<16> {
    static constexpr int kRows = 4;
    static __device__ __forceinline__ int row(int q, int h) { return q + 4 * h; }
    // a 4 x 4 transpose of 16-lane groups: register ni, group j holds row
    // group j of columns 16*ni ..; the result h holds row group h of all 64
    static __device__ __forceinline__ void get(const float* x, float* out)
    {
        const auto s02 = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, x[0]),
                                                          __builtin_bit_cast(uint32_t, x[2]), false,
                                                          false);
        const auto s13 = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, x[1]),
                                                          __builtin_bit_cast(uint32_t, x[3]), false,
                                                          false);
        const auto t01 = __builtin_amdgcn_permlane16_swap((uint32_t)s02[0], (uint32_t)s13[0],
                                                          false, false);
        const auto t23 = __builtin_amdgcn_permlane16_swap((uint32_t)s02[1], (uint32_t)s13[1],
                                                          false, false);
        out[0] = __builtin_bit_cast(float, (uint32_t)t01[0]);
        out[1] = __builtin_bit_cast(float, (uint32_t)t01[1]);
        out[2] = __builtin_bit_cast(float, (uint32_t)t23[0]);
        out[3] = __builtin_bit_cast(float, (uint32_t)t23[1]);
    }
};

// Register q of the NI accumulator blocks of row block `acc` (an array of NI
// MFMA accumulators), regrouped as WaveRows rows.  The registers are passed
// to the swaps by value: read through a pointer to the accumulator array
// inside the swap helper, every q got the swaps of q = 0 (checked with a
// probe of known values).
template <int MT, int NI, typename Acc>
__device__ __forceinline__ void wave_rows(const Acc (&acc)[NI], int q, float* out)
{
    float x[NI];
#pragma unroll
    for (int ni = 0; ni < NI; ++ni)
        x[ni] = acc[ni][q];
    WaveRows<MT>::get(x, out);
}

__device__ __forceinline__ float wave_sum(float v)
{
    for (int off = 32; off > 0; off >>= 1)
        v += __shfl_xor(v, off, 64);
    return v;
}

}  // namespace caffe_hip
