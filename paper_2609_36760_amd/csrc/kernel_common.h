// Device helpers shared by the decode kernels (decode_attn.hip, decode_narrow.hip).
// Internal; not part of the public C ABI.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdint>

namespace mla {
namespace kc {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;
typedef const __attribute__((address_space(1))) void gbl_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};   // RNE
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
    const f16x2 v = {static_cast<_Float16>(lo), static_cast<_Float16>(hi)}; // v_cvt_pk_f16_f32, RNE
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint32_t bf16x2_to_f16x2(uint32_t w) {
    return pack_f16x2(__uint_as_float(w << 16), __uint_as_float(w & 0xFFFF0000u));
}

// Byte offset of buffer (j mod n) of `bytes` bytes, as an opaque scalar: the
// compiler then forms every LDS address as one per-lane base plus this offset
// plus an immediate, instead of keeping a per-lane address for every buffer.
__device__ __forceinline__ int slot_offset(int j, int n, int bytes) {
    int off = (j % n) * bytes;
    asm volatile("" : "+s"(off));
    return off;
}

// Direct-to-LDS load of 16 bytes per lane, marked non-temporal (the cache
// bytes are read once per step): lane l copies base + voff into LDS
// bytes [lds + 16 l, lds + 16 l + 16) (base and lds wave-uniform).  Written as
// inline assembly so that the compiler does not track it: it would otherwise
// wait for every such load in flight before any LDS read of the same array.
// Every read of staged data instead follows an explicit counted wait
// (s_waitcnt vmcnt), and a barrier when other waves read it.  M0 is saved and
// restored around the load.
__device__ __forceinline__ void dma16(const uint8_t* base, uint32_t voff, uint32_t lds) {
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %3\n\ts_nop 0\n\t"
        "global_load_lds_dwordx4 %1, %2 nt\n\ts_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(voff), "s"(base), "s"(lds)
        : "memory");
}

// The same load with its LDS destination handed to the compiler as M0 (which
// the compiler then sets and knows to be in use; the leading wait state covers
// the M0 write before the load reads it).
__device__ __forceinline__ void dma16_m0(const uint8_t* base, uint32_t voff, uint32_t lds) {
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 nt" : : "v"(voff), "s"(base), "{m0}"(lds) : "memory");
}

// (x & m) | o in one v_and_or_b32 (the compiler otherwise splits it in two
// when both constants are literals); m is a scalar, o a vector register.
__device__ __forceinline__ uint32_t and_or(uint32_t x, uint32_t m, uint32_t o) {
    uint32_t r;
    asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "s"(m), "v"(o));
    return r;
}

// 32-bit LDS address of a pointer into shared memory (uniform).
__device__ __forceinline__ uint32_t lds_addr(const uint8_t* p) {
    return __builtin_amdgcn_readfirstlane(
        static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) uint8_t*)p)));
}

// The same entry, waited for on the spot.
__device__ __forceinline__ int load_page_id(const int32_t* table, int index) {
    int v;
    asm volatile("s_load_dword %0, %1, %2\n\ts_waitcnt lgkmcnt(0)"
                 : "=&s"(v)
                 : "s"(table), "s"(__builtin_amdgcn_readfirstlane(index * 4))
                 : "memory");
    return v;
}

// Entries i0, i1, i2 of a page table, fetched through the scalar cache
// together (issue_page_ids3) and waited for once (wait_page_ids3, which names
// the results, so that no use is placed before it); other work can be issued
// in between.
__device__ __forceinline__ void issue_page_ids3(const int32_t* table, int i0, int i1, int i2, int& p0, int& p1,
                                                int& p2) {
    asm volatile("s_load_dword %0, %1, %2" : "=&s"(p0) : "s"(table), "s"(__builtin_amdgcn_readfirstlane(i0 * 4)));
    asm volatile("s_load_dword %0, %1, %2" : "=&s"(p1) : "s"(table), "s"(__builtin_amdgcn_readfirstlane(i1 * 4)));
    asm volatile("s_load_dword %0, %1, %2" : "=&s"(p2) : "s"(table), "s"(__builtin_amdgcn_readfirstlane(i2 * 4)));
}
__device__ __forceinline__ void wait_page_ids3(int& p0, int& p1, int& p2) {
    asm volatile("s_waitcnt lgkmcnt(0)" : "+s"(p0), "+s"(p1), "+s"(p2) : : "memory");
}

// Dequantization metadata as packed fp16 pairs (zz = 1024 + zero, ss = scale).
// Codes become fp16 values 1024 + q (the fp16 with bits 0x6400 | q, exact);
// (1024 + q) - (1024 + zero) = q - zero exactly, and one fp16 multiply by the
// stored scale rounds s * (q - zero) once.  Both in packed fp16 (2 per op).
//
// The paper's storage: scale (bf16 bits, or fp32 for the RoPE group) and a
// byte zero-point.  The bf16 scale converts to fp16 exactly inside the fp16
// range; the fp32 RoPE scale is rounded to fp16 once.
__device__ __forceinline__ void pmeta_to_f16(float scale, uint32_t zero, f16x2& zz, f16x2& ss) {
    const _Float16 s = static_cast<_Float16>(scale);
    const _Float16 zb = static_cast<_Float16>(static_cast<float>(zero) + 1024.0f);   // exact
    zz = f16x2{zb, zb};
    ss = f16x2{s, s};
}

// fp16 storage: {fp16 scale, fp16 zero} in one word.
__device__ __forceinline__ void meta_to_f16(uint32_t meta, f16x2& zz, f16x2& ss) {
    const _Float16 s = __builtin_bit_cast(_Float16, static_cast<uint16_t>(meta & 0xFFFFu));
    const _Float16 z = __builtin_bit_cast(_Float16, static_cast<uint16_t>(meta >> 16));
    const _Float16 zb = z + static_cast<_Float16>(1024.0f);    // exact: z is an integer in [0, 15]
    zz = f16x2{zb, zb};
    ss = f16x2{s, s};
}

// Host side: dispatch a decode kernel, attaching the events that
// mla_time_next_decode_launch left for this thread (if any) to the dispatch
// itself, so that they time the kernel's execution alone.
template <typename Kernel, typename Args>
void dispatch_decode(Kernel kernel, dim3 grid, dim3 block, hipStream_t stream, const LaunchEvents& ev,
                     const Args& a) {
    if (ev.start != nullptr)
        hipExtLaunchKernelGGL(kernel, grid, block, 0, stream, ev.start, ev.stop, 0, a);
    else
        hipLaunchKernelGGL(kernel, grid, block, 0, stream, a);
}

}  // namespace kc
}  // namespace mla
