// Device helpers for the gfx950 Physics-Attention kernels: matrix-core
// fragment types, the 16x16 MFMA wrappers and cross-lane reductions.
//
// Fragment convention (every MFMA in this library is 16x16 with a K step of
// 32): lane l of a wave64 owns row/column (l & 15) of an operand and "K slots"
// (g, t) with g = l >> 4 in 0..3 and t in 0..7.  A and B operands pair slot
// (g, t) with slot (g, t), so which reduction index a slot holds is a free
// choice made per contraction, as long as both operands agree.  Output
// fragment (4 floats): lane l holds D[4*g + r][l & 15], r = 0..3.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ts3 {

typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;

struct bf16_t {
    uint16_t bits;
};

// An 8-slot operand fragment for one K32 step.
template <typename T> struct Frag;

template <> struct Frag<float> {
    float v[8];
    __device__ __forceinline__ void set(int t, float x) { v[t] = x; }
    // slots t and t+1 (t even) from two floats
    __device__ __forceinline__ void set2(int t, float a, float b) { v[t] = a; v[t + 1] = b; }
};

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

template <> struct Frag<bf16_t> {
    bf16x8 v;
    __device__ __forceinline__ void set(int t, float x) { v[t] = (__bf16)x; }
    // slots t and t+1 (t even) from two floats with one packed conversion
    __device__ __forceinline__ void set2(int t, float a, float b) {
        const bf16x2 p{(__bf16)a, (__bf16)b};
        u32x4 u = __builtin_bit_cast(u32x4, v);
        u[t >> 1] = __builtin_bit_cast(uint32_t, p);
        v = __builtin_bit_cast(bf16x8, u);
    }
};

// IEEE half precision operands (the feed-forward's second product).  Same
// 16-bit fragment layout as bf16.
struct f16_t {
    uint16_t bits;
};
typedef __attribute__((ext_vector_type(8))) _Float16 f16x8;
typedef __attribute__((ext_vector_type(2))) _Float16 f16x2;

template <> struct Frag<f16_t> {
    f16x8 v;
};

// acc += A * B over one K32 step.
__device__ __forceinline__ void mma(f32x4 &acc, const Frag<f16_t> &a, const Frag<f16_t> &b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a.v, b.v, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma(f32x4 &acc, const Frag<bf16_t> &a, const Frag<bf16_t> &b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma(f32x4 &acc, const Frag<float> &a, const Frag<float> &b) {
#pragma unroll
    for (int t = 0; t < 8; ++t) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[t], b.v[t], acc, 0, 0, 0);
}

// Load the 8 consecutive storage elements at p (16 B for bf16, 32 B for fp32).
__device__ __forceinline__ void load8(Frag<bf16_t> &f, const bf16_t *p) {
    f.v = *reinterpret_cast<const bf16x8 *>(p);
}
__device__ __forceinline__ void load8(Frag<float> &f, const float *p) {
    const float4 a = reinterpret_cast<const float4 *>(p)[0];
    const float4 b = reinterpret_cast<const float4 *>(p)[1];
    f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w;
    f.v[4] = b.x; f.v[5] = b.y; f.v[6] = b.z; f.v[7] = b.w;
}
__device__ __forceinline__ void zero8(Frag<bf16_t> &f) {
    f.v = bf16x8{};
}
__device__ __forceinline__ void zero8(Frag<float> &f) {
#pragma unroll
    for (int t = 0; t < 8; ++t) f.v[t] = 0.f;
}
__device__ __forceinline__ void ones8(Frag<bf16_t> &f) {
#pragma unroll
    for (int t = 0; t < 8; ++t) f.v[t] = (__bf16)1.0f;
}
__device__ __forceinline__ void ones8(Frag<float> &f) {
#pragma unroll
    for (int t = 0; t < 8; ++t) f.v[t] = 1.f;
}

// Storage element <-> float.
__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t x) { return __uint_as_float(uint32_t(x.bits) << 16); }
__device__ __forceinline__ uint16_t raw16(bf16_t x) { return x.bits; }

// Element t of a loaded fragment as stored bits/values (for LDS transposes).
__device__ __forceinline__ uint16_t elem_bits(const Frag<bf16_t> &f, int t) {
    // Read element t through the packed dwords (element 2k is the low half of dword k).
    const u32x4 u = __builtin_bit_cast(u32x4, f.v);
    return (uint16_t)((t & 1) ? (u[t >> 1] >> 16) : (u[t >> 1] & 0xffffu));
}
__device__ __forceinline__ float elem_f32(const Frag<float> &f, int t) { return f.v[t]; }

// Cross-lane reductions among the 16 lanes of a DPP row (all lanes get the result).
template <int CTRL> __device__ __forceinline__ float dpp(float v) {
    return __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(v), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ float row16_max(float v) {
    v = fmaxf(v, dpp<0x128>(v));  // row_ror:8
    v = fmaxf(v, dpp<0x124>(v));  // row_ror:4
    v = fmaxf(v, dpp<0x4E>(v));   // quad_perm [2,3,0,1]
    v = fmaxf(v, dpp<0xB1>(v));   // quad_perm [1,0,3,2]
    return v;
}
__device__ __forceinline__ float row16_sum(float v) {
    v += dpp<0x128>(v);
    v += dpp<0x124>(v);
    v += dpp<0x4E>(v);
    v += dpp<0xB1>(v);
    return v;
}

// Reductions across the four 16-lane rows (lanes l, l^16, l^32, l^48).
__device__ __forceinline__ float xrow_max(float v) {
    auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float xrow_sum(float v) {
    auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// The slice softmax skips the max subtraction when a row's sum of exp2 terms
// lands in [2^-100, 2^100]: every term is then finite, the largest is a normal
// number, and terms that underflow weigh < 2^-20 of it.  Rows outside the
// window (or NaN) take the max-shifted path; both compute the same softmax.
__device__ __forceinline__ bool softmax_sum_ok(float s) {
    return s >= 0x1p-100f && s <= 0x1p100f;
}
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

// Scheduling hint for the region just emitted: alternate NMFMA matrix-core
// instructions with VPER vector-ALU instructions, pulling one LDS read ahead
// of every RPER MFMAs, so one wave keeps both units busy (in-order issue would
// otherwise run the MFMA cluster and the VALU cluster back to back).
template <int NMFMA, int VPER, int RPER>
__device__ __forceinline__ void interleave_mfma_valu() {
#pragma unroll
    for (int i = 0; i < NMFMA; ++i) {
        if (RPER > 0 && i % RPER == 0) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                                  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, VPER, 0);                               // VALU
    }
}

// Scheduling hint for a region holding a chain of NMFMA matrix-core
// instructions fed by LDS reads, next to an independent vector-ALU chain: the
// first PRE reads go up front, then each MFMA is followed by VPER vector-ALU
// instructions, and RN further reads are pulled in after every RPER MFMAs
// (starting after MFMA R0); NW LDS writes close the region.
template <int PRE, int NMFMA, int VPER, int R0, int RPER, int RN, int NW>
__device__ __forceinline__ void interleave_chain() {
    if constexpr (PRE > 0) __builtin_amdgcn_sched_group_barrier(0x100, PRE, 0);
#pragma unroll
    for (int i = 0; i < NMFMA; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, VPER, 0);
        if (i >= R0 && (i - R0) % RPER == 0) __builtin_amdgcn_sched_group_barrier(0x100, RN, 0);
    }
    if constexpr (NW > 0) __builtin_amdgcn_sched_group_barrier(0x200, NW, 0);
}

// Direct global->LDS copy of 16 bytes per lane: lane l's bytes land at LDS
// byte lds_base + 16*l (lds_base wave-uniform).  Issued as inline assembly so
// that the compiler's wait-count pass does not see an LDS write in flight and
// hold every later LDS access until it lands; callers track completion
// themselves with wait_vmcnt.  M0 carries the LDS base; the kernels that use
// this have no other M0 user (gfx950 LDS instructions do not read M0).
// The compiler inserts no wait states for hazards inside assembly, so the
// copies carry their own: one between the M0 write and the copy that reads
// it, and, where the global base is a scalar operand that vector code may
// have just written (v_readfirstlane), five before the copy reads it.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const void *src, uint32_t lds_base) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(lds_base)
                 : "memory", "m0");
}
// The same copy with a wave-uniform global base and a per-lane 32-bit offset.
template <int IMM> __device__ __forceinline__ void dma16s(uint32_t voff, const void *sbase, uint32_t lds_base) {
    static_assert(IMM >= 0 && IMM < 4096, "global offset field");
    const uint64_t b = (uint64_t)(uintptr_t)sbase;  // pin the base to scalar registers
    // readfirstlane yields a signed int: widen through uint32_t so the low
    // half is not sign-extended into the high one.
    const uint64_t ub = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32)) << 32) |
                        (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b);
    sbase = (const void *)(uintptr_t)ub;
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 3\n\tglobal_load_lds_dwordx4 %0, %1 offset:%3" ::"v"(voff), "s"(sbase),
                 "s"(lds_base), "n"(IMM)
                 : "memory", "m0");
}
#pragma clang diagnostic pop
__device__ __forceinline__ uint32_t lds_addr(const void *p) {
    return __builtin_amdgcn_readfirstlane(
        (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)p);
}

// Wait until at most N vector-memory operations of this wave are outstanding
// (other counters untouched).
template <int N> __device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// XCD-aware block index: consecutive logical indices land on the same XCD
// (workgroups are dispatched round-robin over the 8 XCDs of an MI355X).
__device__ __forceinline__ int xcd_remap(int i, int n) {
    const int xcd = i & 7, k = i >> 3;
    const int base = n >> 3, rem = n & 7;
    return xcd < rem ? xcd * (base + 1) + k : rem * (base + 1) + (xcd - rem) * base + k;
}

}  // namespace ts3
