// Device helpers shared by the gfx950 kernels: conversions, INT4 chunk
// decode, wave/block reductions and the coherent cross-workgroup exchange.
#pragma once

#include "common.h"

namespace stg {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// ------------------------------------------------------------------ conversions

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);  // quiet NaN
    u += 0x7fffu + ((u >> 16) & 1u);                                           // ties to even
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float f16_to_f32(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }
__device__ __forceinline__ uint16_t f32_to_f16(float f) { return __builtin_bit_cast(uint16_t, (_Float16)f); }

__device__ __forceinline__ float load_val(const void* p, int dt, size_t i) {
    if (dt == DT_F32) return ((const float*)p)[i];
    const uint16_t b = ((const uint16_t*)p)[i];
    return dt == DT_BF16 ? bf16_to_f32(b) : f16_to_f32(b);
}

// N values at element offsets off[i] of p (dtype dt, the same in every lane),
// every load issued before any is converted: the dtype branch sits outside the
// loads (a branch per value makes each load wait for the one before).
template <int N>
__device__ __forceinline__ void load_vals(const void* p, int dt, const size_t (&off)[N], float (&out)[N]) {
    if (dt == DT_F32) {
        const float* f = (const float*)p;
#pragma unroll
        for (int i = 0; i < N; ++i) out[i] = f[off[i]];
    } else {
        const uint16_t* h = (const uint16_t*)p;
        uint16_t bits[N];
#pragma unroll
        for (int i = 0; i < N; ++i) bits[i] = h[off[i]];
#pragma unroll
        for (int i = 0; i < N; ++i) out[i] = dt == DT_BF16 ? bf16_to_f32(bits[i]) : f16_to_f32(bits[i]);
    }
}

__device__ __forceinline__ uint16_t to_half_bits(float f, int dt) { return dt == DT_BF16 ? f32_to_bf16(f) : f32_to_f16(f); }
__device__ __forceinline__ float half_bits_to_f32(uint16_t b, int dt) { return dt == DT_BF16 ? bf16_to_f32(b) : f16_to_f32(b); }

__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
    return (uint32_t)f32_to_f16(lo) | ((uint32_t)f32_to_f16(hi) << 16);
}

// 16-byte chunk (32 codes) -> 16 fp16 pairs of consecutive k holding q = u - 8 exactly.
__device__ __forceinline__ void unpack_chunk(const u32x4 w, half2_t* out) {
    const half2_t sub = {(_Float16)1032.0f, (_Float16)1032.0f};
    const half2_t s16 = {(_Float16)0.0625f, (_Float16)0.0625f};
    const half2_t m72 = {(_Float16)-72.0f, (_Float16)-72.0f};
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        const uint32_t x = w[d];
        const uint32_t y = x >> 8;
        const uint32_t p0 = (x & 0x000F000Fu) | 0x64006400u;   // 1024 + u      (k, k+1)
        const uint32_t p1 = (x & 0x00F000F0u) | 0x64006400u;   // 1024 + 16 u   (k+2, k+3)
        const uint32_t p2 = (y & 0x000F000Fu) | 0x64006400u;   //               (k+4, k+5)
        const uint32_t p3 = (y & 0x00F000F0u) | 0x64006400u;   //               (k+6, k+7)
        out[4 * d + 0] = __builtin_bit_cast(half2_t, p0) - sub;
        out[4 * d + 1] = __builtin_elementwise_fma(__builtin_bit_cast(half2_t, p1), s16, m72);
        out[4 * d + 2] = __builtin_bit_cast(half2_t, p2) - sub;
        out[4 * d + 3] = __builtin_elementwise_fma(__builtin_bit_cast(half2_t, p3), s16, m72);
    }
}

// ------------------------------------------------------------------ reductions

template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

// Sum over the 16 lanes of a DPP row; every lane receives the identical value.
__device__ __forceinline__ float sum16(float v) {
    v += dpp_f<0xB1>(v);    // quad_perm [1,0,3,2]
    v += dpp_f<0x4E>(v);    // quad_perm [2,3,0,1]
    v += dpp_f<0x141>(v);   // row_half_mirror
    v += dpp_f<0x140>(v);   // row_mirror
    return v;
}

// Deterministic block sum (256 threads): fixed-order tree in LDS.
__device__ __forceinline__ float block_sum256(float v, float* buf) {
    const int tid = threadIdx.x;
    buf[tid] = v;
    __syncthreads();
#pragma unroll
    for (int w = 128; w > 0; w >>= 1) {
        if (tid < w) buf[tid] += buf[tid + w];
        __syncthreads();
    }
    const float r = buf[0];
    __syncthreads();
    return r;
}

// ------------------------------------------------------------------ coherent exchange
// Workgroups of one launch exchange split partials through device-scope
// ("sc1") stores and loads, which bypass the per-XCD L2s.  Before the ticket
// every wave waits for the acknowledgement of its own stores (s_waitcnt
// vmcnt(0): a device-scope store is acknowledged once it is visible at device
// scope), then the workgroup meets at a barrier, so every partial of the
// workgroup is visible before the counter moves.  A workgroup-scope release
// alone emits no such wait on gfx950, and an agent-scope fence would write
// back and invalidate the whole L2.

__device__ __forceinline__ void store_coherent(float* p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_coherent(const float* p) {
    return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Returns true in exactly one workgroup: the last of `n` to arrive at counter *c,
// which it resets.  Every thread of the workgroup must call it.
__device__ __forceinline__ bool last_arrival(unsigned* c, unsigned n, int* flag) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");          // this wave's coherent stores are acknowledged
    __syncthreads();
    if (threadIdx.x == 0) {
        const unsigned prev = atomicAdd(c, 1u);
        *flag = (prev == n - 1);
        if (prev == n - 1) __hip_atomic_store(c, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);  // next use starts from zero
    }
    __syncthreads();
    return *flag != 0;
}


}  // namespace stg
