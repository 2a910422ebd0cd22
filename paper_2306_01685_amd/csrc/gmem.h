// Device-side global-memory accessors.
//
// Buffer pointers reach the kernels inside descriptor tables, so the compiler
// cannot tell that they point to global memory and would emit flat
// instructions.  Flat loads count against the LDS wait counter as well as the
// vector-memory one, so a wait for an LDS read would also wait for every
// outstanding prefetch.  These helpers cast to the global address space (and
// use native vector types, which the cast needs to stay a single 16-byte
// access), so every access below is a global_load / global_store.
#pragma once

#include <hip/hip_runtime.h>

namespace mkor {

#define MKOR_GLOBAL __attribute__((address_space(1)))

typedef float        mk_f4 __attribute__((ext_vector_type(4)));
typedef unsigned int mk_u4 __attribute__((ext_vector_type(4)));
typedef unsigned int mk_u2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float gld(const float* p) { return *(const MKOR_GLOBAL float*)p; }

__device__ __forceinline__ int gld_i32(const int32_t* p) { return *(const MKOR_GLOBAL int32_t*)p; }

__device__ __forceinline__ unsigned short gld_u16(const unsigned short* p) {
    return *(const MKOR_GLOBAL unsigned short*)p;
}

__device__ __forceinline__ float4 gld4(const float* p) {
    const mk_f4 v = *(const MKOR_GLOBAL mk_f4*)p;
    return make_float4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ uint4 gld_u4(const void* p) {
    const mk_u4 v = *(const MKOR_GLOBAL mk_u4*)p;
    return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ uint2 gld_u2(const void* p) {
    const mk_u2 v = *(const MKOR_GLOBAL mk_u2*)p;
    return make_uint2(v.x, v.y);
}

// Streaming variants (non-temporal hint: the data is not re-read soon).
__device__ __forceinline__ float4 gld4_nt(const float* p) {
    const mk_f4 v = __builtin_nontemporal_load((const MKOR_GLOBAL mk_f4*)p);
    return make_float4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ void gst4_nt(float* p, const float4& v) {
    mk_f4 w;
    w.x = v.x; w.y = v.y; w.z = v.z; w.w = v.w;
    __builtin_nontemporal_store(w, (MKOR_GLOBAL mk_f4*)p);
}

__device__ __forceinline__ uint4 gld_u4_nt(const void* p) {
    const mk_u4 v = __builtin_nontemporal_load((const MKOR_GLOBAL mk_u4*)p);
    return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ void gst_u4_nt(void* p, const uint4& v) {
    mk_u4 w;
    w.x = v.x; w.y = v.y; w.z = v.z; w.w = v.w;
    __builtin_nontemporal_store(w, (MKOR_GLOBAL mk_u4*)p);
}

// base (wave-uniform) + 32-bit byte offset: the form of the scalar-base
// addressing mode, so per-thread addresses need one 32-bit register.
__device__ __forceinline__ float4 gld4_off(const void* base, unsigned byte_off) {
    const mk_f4 v = *(const MKOR_GLOBAL mk_f4*)((const MKOR_GLOBAL char*)base + byte_off);
    return make_float4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ uint2 gld_u2_off(const void* base, unsigned byte_off) {
    const mk_u2 v = *(const MKOR_GLOBAL mk_u2*)((const MKOR_GLOBAL char*)base + byte_off);
    return make_uint2(v.x, v.y);
}

__device__ __forceinline__ float gld_off(const void* base, unsigned byte_off) {
    return *(const MKOR_GLOBAL float*)((const MKOR_GLOBAL char*)base + byte_off);
}

__device__ __forceinline__ void gst(float* p, float v) { *(MKOR_GLOBAL float*)p = v; }

__device__ __forceinline__ void gst_u4(void* p, uint4 v) {
    mk_u4 w;
    w.x = v.x; w.y = v.y; w.z = v.z; w.w = v.w;
    *(MKOR_GLOBAL mk_u4*)p = w;
}

__device__ __forceinline__ void gst_u2(void* p, uint2 v) {
    mk_u2 w;
    w.x = v.x; w.y = v.y;
    *(MKOR_GLOBAL mk_u2*)p = w;
}

// bf16 <-> fp32.  The conversion to bf16 is the hardware's (v_cvt_pk_bf16_f32):
// round to nearest, ties to even; NaN stays NaN.
typedef __bf16 mk_bf2 __attribute__((ext_vector_type(2)));
typedef float  mk_f2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf2f(unsigned short h) { return __uint_as_float(((unsigned)h) << 16); }

// two floats -> packed bf16 pair (a in the low half)
__device__ __forceinline__ unsigned f2bf2(float a, float b) {
    const mk_f2 v = {a, b};
    return __builtin_bit_cast(unsigned, __builtin_convertvector(v, mk_bf2));
}

__device__ __forceinline__ unsigned short f2bf(float f) {
    return __builtin_bit_cast(unsigned short, (__bf16)f);
}

__device__ __forceinline__ void gst4(float* p, const float4& v) {
    mk_f4 w;
    w.x = v.x; w.y = v.y; w.z = v.z; w.w = v.w;
    *(MKOR_GLOBAL mk_f4*)p = w;
}

}  // namespace mkor
