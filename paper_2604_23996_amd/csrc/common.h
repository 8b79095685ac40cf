// Device helpers shared by the SMoES kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>
#include <stdint.h>

#define SMOES_K_MAX_DEV 16

namespace smoes {

constexpr int kWave = 64;

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

// ---------------------------------------------------------------- bf16 storage

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// float32 -> bf16, round to nearest even (NaN kept quiet).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

// Eight consecutive activations (16 bytes of bf16, or 2 x 16 bytes of f32) as floats.
template <bool BF16>
__device__ __forceinline__ void load8(const void* base, int64_t elem, float (&v)[8]) {
    if constexpr (BF16) {
        const uint4 q = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + elem);
        const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[2 * i] = __uint_as_float(w[i] << 16);
            v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    } else {
        const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(base) + elem);
        const float4 a = p[0], b = p[1];
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    }
}

// ---------------------------------------------------------------- wave reductions
// Fixed butterfly order: every lane ends with the same, reproducible value.

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// Wave reductions with a uniform result, built from DPP moves inside each
// 16-lane row (quad swaps, half-row and row mirrors: every lane of a row ends
// with the row's value) and one read of each row's lane 0; the four row
// values are combined in a fixed order. Needs all 64 lanes active.
template <int CTRL>
__device__ __forceinline__ int dpp_mov(int v) {
    return __builtin_amdgcn_mov_dpp(v, CTRL, 0xf, 0xf, false);
}
template <class T, class Op>
__device__ __forceinline__ T row_allreduce(T v, Op op) {
    auto mv = [](T x, auto ctrl) {
        constexpr int C = decltype(ctrl)::value;
        if constexpr (__is_same(T, double)) {
            const long long b = __double_as_longlong(x);
            const int lo = dpp_mov<C>(static_cast<int>(b)), hi = dpp_mov<C>(static_cast<int>(b >> 32));
            return __longlong_as_double((static_cast<long long>(hi) << 32) | static_cast<unsigned int>(lo));
        } else if constexpr (sizeof(T) == 4 && !__is_same(T, int)) {
            return __int_as_float(dpp_mov<C>(__float_as_int(x)));
        } else {
            return static_cast<T>(dpp_mov<C>(static_cast<int>(x)));
        }
    };
    v = op(v, mv(v, std::integral_constant<int, 0xB1>{}));   // quad_perm [1,0,3,2]
    v = op(v, mv(v, std::integral_constant<int, 0x4E>{}));   // quad_perm [2,3,0,1]
    v = op(v, mv(v, std::integral_constant<int, 0x141>{}));  // row_half_mirror
    v = op(v, mv(v, std::integral_constant<int, 0x140>{}));  // row_mirror
    return v;
}
__device__ __forceinline__ float wave_max_u(float v) {
    v = row_allreduce(v, [](float a, float b) { return fmaxf(a, b); });
    const int i = __float_as_int(v);
    const float a = __int_as_float(__builtin_amdgcn_readlane(i, 0)), b = __int_as_float(__builtin_amdgcn_readlane(i, 16));
    const float c = __int_as_float(__builtin_amdgcn_readlane(i, 32)), d = __int_as_float(__builtin_amdgcn_readlane(i, 48));
    return fmaxf(fmaxf(a, b), fmaxf(c, d));
}
__device__ __forceinline__ float wave_sum_u(float v) {
    v = row_allreduce(v, [](float a, float b) { return a + b; });
    const int i = __float_as_int(v);
    const float a = __int_as_float(__builtin_amdgcn_readlane(i, 0)), b = __int_as_float(__builtin_amdgcn_readlane(i, 16));
    const float c = __int_as_float(__builtin_amdgcn_readlane(i, 32)), d = __int_as_float(__builtin_amdgcn_readlane(i, 48));
    return (a + b) + (c + d);
}
__device__ __forceinline__ double wave_sum_u(double v) {
    v = row_allreduce(v, [](double a, double b) { return a + b; });
    auto rl = [](double x, int l) {
        const long long b = __double_as_longlong(x);
        const int lo = __builtin_amdgcn_readlane(static_cast<int>(b), l);
        const int hi = __builtin_amdgcn_readlane(static_cast<int>(b >> 32), l);
        return __longlong_as_double((static_cast<long long>(hi) << 32) | static_cast<unsigned int>(lo));
    };
    return (rl(v, 0) + rl(v, 16)) + (rl(v, 32) + rl(v, 48));
}
__device__ __forceinline__ int wave_min_u(int v) {
    v = row_allreduce(v, [](int a, int b) { return a < b ? a : b; });
    const int a = __builtin_amdgcn_readlane(v, 0), b = __builtin_amdgcn_readlane(v, 16);
    const int c = __builtin_amdgcn_readlane(v, 32), d = __builtin_amdgcn_readlane(v, 48);
    const int ab = a < b ? a : b, cd = c < d ? c : d;
    return ab < cd ? ab : cd;
}

__host__ __device__ __forceinline__ int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

__host__ __device__ __forceinline__ size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// ---------------------------------------------------------------- buffer loads and waits

// Raw buffer descriptors (gfx9 word 3) and an offset that is always past the record count.
constexpr int kBufferFlags = 0x00020000;
constexpr int kOutOfRange = 0x7fffffff;
constexpr int kBufferNonTemporal = 2;  // cache-policy operand of a buffer access: streaming (nt)
typedef int i32x4_t __attribute__((ext_vector_type(4)));

// s_waitcnt with vmcnt(N) and lgkmcnt(0) (gfx9 encoding; expcnt left free)
template <int N>
__device__ __forceinline__ void wait_vm_lgkm0() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 0xf) | ((N >> 4) << 14) | 0x70);
}

// ---------------------------------------------------------------- buffer-to-LDS loads as inline assembly
//
// With the builtin form the compiler sees the LDS writes of a buffer-to-LDS
// load and, unable to tell them apart from reads of other ring slots, may wait
// for every outstanding load before each LDS read, which drains the ring. The
// kernels that use these order them with explicit vmcnt waits and barriers.
// Descriptor words: base (48 bits, stride 0), record count in bytes, format.
__device__ __forceinline__ i32x4_t buf_rsrc(const void* base, int bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    return i32x4_t{__builtin_amdgcn_readfirstlane(static_cast<int>(a & 0xffffffffu)),
                   __builtin_amdgcn_readfirstlane(static_cast<int>((a >> 32) & 0xffffu)),
                   __builtin_amdgcn_readfirstlane(bytes), kBufferFlags};
}
__device__ __forceinline__ uint32_t lds_address(const void* p) {
    return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) uint8_t*)p));
}
// 16 bytes per lane from byte offset voff into LDS at lds + 16 lane (lds uniform;
// it goes in through M0 as an operand, so the compiler sets M0 itself)
__device__ __forceinline__ void dma16(i32x4_t rsrc, int voff, uint32_t lds) {
    asm volatile("buffer_load_dwordx4 %0, %1, 0 offen lds"
                 :
                 : "v"(voff), "s"(rsrc), "{m0}"(__builtin_amdgcn_readfirstlane(static_cast<int>(lds)))
                 : "memory");
}
// 4 bytes per lane into LDS at lds + 4 lane
__device__ __forceinline__ void dma4(i32x4_t rsrc, int voff, uint32_t lds) {
    asm volatile("buffer_load_dword %0, %1, 0 offen lds"
                 :
                 : "v"(voff), "s"(rsrc), "{m0}"(__builtin_amdgcn_readfirstlane(static_cast<int>(lds)))
                 : "memory");
}

// Values that are the same in every lane but that the compiler cannot prove
// uniform (they derive from loads): pin them to SGPRs so buffer descriptors
// built from them stay scalar.
__device__ __forceinline__ int uniform_int(int v) { return __builtin_amdgcn_readfirstlane(v); }
template <class T>
__device__ __forceinline__ T* uniform_ptr(T* p) {
    const uint64_t v = reinterpret_cast<uint64_t>(p);
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v >> 32));
    return reinterpret_cast<T*>((static_cast<uint64_t>(hi) << 32) | lo);
}

}  // namespace smoes
