// Device helpers of the quantize-and-append writer, shared by the writer
// kernels (quant_append.hip) and the decode kernel's in-launch append
// (decode_attn.hip).  Internal; not part of the public C ABI.
//
// Quantizer: Appendix C.4, "Affine group quantization" -- per token, groups of
// 64 consecutive channels, m = 2^b - 1,
//   s = max(xmax - xmin, 1e-8) / m,  z = clip(rint(-xmin / s), 0, m),
//   q = clip(rint(x / s + z), 0, m),
// round-half-to-even, constant groups not special-cased; the stored fp16
// scale and zero are what attention dequantizes with.  Every step is one IEEE
// fp32 operation in that order (explicitly rounded subtractions and divisions;
// no step multiplies, so no contraction can merge two), so the codes and fp16
// metadata are bit-identical to any IEEE implementation of the formula.
//
// Metadata: fp16(s) and fp16(z) per group (MLA_META_FP16); or the paper's
// storage (Appendix C.4, last sentence): bf16(s) (round-half-to-even) for the
// content groups and s itself (fp32) for the RoPE group, z as a byte, in one
// 32-byte record per token (layout in mla_lowbit.h).  The codes come from
// the unrounded fp32 s in both.
//
// Work split: 8 consecutive lanes per group of 64 channels, each lane owning 8
// channels (one 16-byte load); min/max are reduced across the 8 lanes, which
// must all be active.  A token has 9 groups: 8 content groups (d_c = 512) and
// one RoPE-key group (d_r = 64).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "internal.h"

namespace mla {
namespace wc {

constexpr int kGroup = 64;
constexpr int kLanesPerGroup = 8;
constexpr int kGroupsPerToken = 9;

__device__ __forceinline__ void widen_bf16x8(const uint4 raw, float x[8]) {
    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        x[2 * i] = __uint_as_float(w[i] << 16);
        x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
}

__device__ __forceinline__ uint16_t f16_bits(float v) {
    const _Float16 h = static_cast<_Float16>(v);   // v_cvt_f16_f32: round-half-to-even, subnormals kept
    return __builtin_bit_cast(uint16_t, h);
}

// Quantize the lane's 8 channels `raw` (bf16) of group g of a token (lane lig
// of the group's 8; rope: the RoPE-key group) and store its codes and
// metadata at token `off` of the page at `base`.
template <int CBITS, bool kPaper>
__device__ __forceinline__ void quantize_store(const uint4 raw, bool rope, int g, int lig, uint8_t* base,
                                               int64_t off, const PageGeom& geom) {
    float x[8];
    widen_bf16x8(raw, x);
    float lo = x[0], hi = x[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) {
        lo = fminf(lo, x[i]);
        hi = fmaxf(hi, x[i]);
    }
#pragma unroll
    for (int d = 1; d < kLanesPerGroup; d <<= 1) {
        lo = fminf(lo, __shfl_xor(lo, d, kLanesPerGroup));
        hi = fmaxf(hi, __shfl_xor(hi, d, kLanesPerGroup));
    }

    const int bits = rope ? 4 : CBITS;
    const float m = static_cast<float>((1 << bits) - 1);
    const float s = __fdiv_rn(fmaxf(__fsub_rn(hi, lo), 1e-8f), m);
    // integer zero-point in [0, m]; "+ 0.0f" turns a -0 from rint into +0
    const float z = fminf(fmaxf(rintf(__fdiv_rn(-lo, s)), 0.0f), m) + 0.0f;

    // Code layout: little-endian 32-bit words of 32 / bits consecutive
    // channels; channel 2i of a word in bits [bits i, bits (i+1)), channel
    // 2i+1 at the same place in the upper half (a decoder extracts a channel
    // pair with one shift and one mask).  A lane's 8 channels fill a 4-bit
    // word, or one half of each 16-bit half of a 2-bit word: the two lanes of
    // a 2-bit word merge their parts.
    uint32_t packed = 0;
    const int sh2 = 8 * (lig & 1);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const float t = __fadd_rn(__fdiv_rn(x[i], s), z);
        const uint32_t q = static_cast<uint32_t>(fminf(fmaxf(rintf(t), 0.0f), m));
        const int pos = bits == 4 ? 4 * (i >> 1) : sh2 + 2 * (i >> 1);
        packed |= q << (pos + 16 * (i & 1));
    }
    const uint32_t word2 = packed | static_cast<uint32_t>(__shfl_xor(static_cast<int>(packed), 1, kLanesPerGroup));

    if (rope) {
        *reinterpret_cast<uint32_t*>(base + geom.off_cr + off * geom.cr_bytes + lig * 4) = packed;
    } else if (CBITS == 4) {
        *reinterpret_cast<uint32_t*>(base + off * geom.cc_bytes + g * 32 + lig * 4) = packed;
    } else if ((lig & 1) == 0) {
        *reinterpret_cast<uint32_t*>(base + off * geom.cc_bytes + g * 16 + lig * 2) = word2;
    }
    if (lig == 0) {
        if constexpr (kPaper) {
            uint8_t* rec = base + geom.off_mc + off * 32;
            const uint32_t zb = static_cast<uint32_t>(z);
            if (rope) {
                // fp32 scale, byte zero-point, three zero bytes
                *reinterpret_cast<uint2*>(rec + 24) = make_uint2(__float_as_uint(s), zb);
            } else {
                const __bf16 sb = static_cast<__bf16>(s);     // round-half-to-even
                *reinterpret_cast<uint16_t*>(rec + 2 * g) = __builtin_bit_cast(uint16_t, sb);
                rec[16 + g] = static_cast<uint8_t>(zb);
            }
        } else {
            const uint32_t meta = static_cast<uint32_t>(f16_bits(s)) | (static_cast<uint32_t>(f16_bits(z)) << 16);
            uint8_t* mp = rope ? base + geom.off_mr + off * 4 : base + geom.off_mc + off * 32 + g * 4;
            *reinterpret_cast<uint32_t*>(mp) = meta;
        }
    }
}

}  // namespace wc
}  // namespace mla
