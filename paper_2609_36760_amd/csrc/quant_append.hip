// Quantize-and-append writer for the packed dual-path cache, and the plain
// BF16 append used by the unquantized comparison cache.
//
// Quantizer: Appendix C.4, "Affine group quantization" -- per token, groups of
// 64 consecutive channels, m = 2^b - 1,
//   s = max(xmax - xmin, 1e-8) / m,  z = clip(rint(-xmin / s), 0, m),
//   q = clip(rint(x / s + z), 0, m),
// round-half-to-even, constant groups not special-cased; the stored fp16
// scale and zero are what attention dequantizes with.  Every step is one IEEE
// fp32 operation in that order: this file is built with
// -ffp-contract=off and correctly rounded fp32 division, so the codes and
// fp16 metadata are bit-identical to any IEEE implementation of the formula.
//
// Metadata: fp16(s) and fp16(z) per group (MLA_META_FP16); or the paper's
// storage (Appendix C.4, last sentence): bf16(s) (round-half-to-even) for the
// content groups and s itself (fp32) for the RoPE group, z as a byte, in one
// 32-byte record per token (layout in mla_lowbit.h).  The codes come from
// the unrounded fp32 s in both.
//
// Work split: 8 lanes per group of 64 channels, each lane owning 8 channels
// (one 16-byte load); min/max are reduced across the 8 lanes.  A token has 9
// groups: 8 content groups (d_c = 512) and one RoPE-key group (d_r = 64).
//
// With BF16 protection (Sec. 3.3; Appendix C.5, "BF16 protection and cache
// lifecycle") the same lanes also store the bf16 values they loaded into the
// token's row of its sequence's protection buffer when the token is protected
// once the append is done: position p < sink (row p) or p >= L - recent
// (row sink + (p - sink) mod recent, a ring), L the sequence's new length.
// Tokens leaving the window keep the packed copy written here at insertion.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace mla {
namespace {

constexpr int kGroup = 64;
constexpr int kLanesPerGroup = 8;
constexpr int kGroupsPerToken = 9;
constexpr int kThreads = 256;

__device__ inline void widen_bf16x8(const uint4 raw, float x[8]) {
    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        x[2 * i] = __uint_as_float(w[i] << 16);
        x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
}

__device__ inline uint16_t f16_bits(float v) {
    const _Float16 h = static_cast<_Float16>(v);   // v_cvt_f16_f32: round-half-to-even, subnormals kept
    return __builtin_bit_cast(uint16_t, h);
}

template <int CBITS, bool kProt, bool kPaper>
__global__ __launch_bounds__(kThreads) void lowbit_append_kernel(AppendArgs a) {
    const int64_t tid = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    const int64_t gid = tid / kLanesPerGroup;           // the 8 lanes of a group share gid
    const int lig = static_cast<int>(threadIdx.x % kLanesPerGroup);
    if (gid >= static_cast<int64_t>(a.n) * kGroupsPerToken) return;
    const int64_t token = gid / kGroupsPerToken;
    const int g = static_cast<int>(gid % kGroupsPerToken);
    const int64_t slot = a.slot_mapping[token];
    if (slot < 0 || slot >= a.num_slots) return;        // skipped token

    const bool rope = (g == kGroupsPerToken - 1);
    const uint16_t* src = rope ? a.k_rope + token * a.k_rope_stride + lig * 8
                               : a.c_kv + token * a.c_kv_stride + g * kGroup + lig * 8;
    const uint4 raw = *reinterpret_cast<const uint4*>(src);
    float x[8];
    widen_bf16x8(raw, x);

    if constexpr (kProt) {
        const int bseq = a.token_seq[token];
        if (bseq >= 0 && bseq < a.B) {
            const int p = a.positions[token];
            const int L = a.seq_lens[bseq];
            const int64_t ps = a.prot_slot[bseq];
            // p >= L - recent with p < L implies recent >= 1
            if (p >= 0 && p < L && (p < a.sink || p >= L - a.recent) && ps >= 0 && ps < a.num_prot) {
                const int prow = p < a.sink ? p : a.sink + (p - a.sink) % a.recent;
                uint8_t* dst = a.prot + (ps * (a.sink + a.recent) + prow) * 1152 +
                               (rope ? 1024 + lig * 16 : (g * kGroup + lig * 8) * 2);
                *reinterpret_cast<uint4*>(dst) = raw;
            }
        }
    }

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
    const float s = fmaxf(hi - lo, 1e-8f) / m;
    // integer zero-point in [0, m]; "+ 0.0f" turns a -0 from rint into +0
    const float z = fminf(fmaxf(rintf(-lo / s), 0.0f), m) + 0.0f;

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

    const int64_t page = slot / a.g.page_size;
    const int64_t off = slot % a.g.page_size;
    uint8_t* base = a.cache + page * a.g.page_bytes;
    if (rope) {
        *reinterpret_cast<uint32_t*>(base + a.g.off_cr + off * a.g.cr_bytes + lig * 4) = packed;
    } else if (CBITS == 4) {
        *reinterpret_cast<uint32_t*>(base + off * a.g.cc_bytes + g * 32 + lig * 4) = packed;
    } else if ((lig & 1) == 0) {
        *reinterpret_cast<uint32_t*>(base + off * a.g.cc_bytes + g * 16 + lig * 2) = word2;
    }
    if (lig == 0) {
        if constexpr (kPaper) {
            uint8_t* rec = base + a.g.off_mc + off * 32;
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
            uint8_t* mp = rope ? base + a.g.off_mr + off * 4 : base + a.g.off_mc + off * 32 + g * 4;
            *reinterpret_cast<uint32_t*>(mp) = meta;
        }
    }
}

// BF16 comparison cache: row = [c_kv (512) | k_rope (64)] bf16; 72 lanes per
// token, 16 bytes each.
__global__ __launch_bounds__(kThreads) void bf16_append_kernel(AppendArgs a) {
    constexpr int kLanesPerToken = 72;
    const int64_t tid = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    const int64_t token = tid / kLanesPerToken;
    const int lane = static_cast<int>(tid % kLanesPerToken);
    if (token >= a.n) return;
    const int64_t slot = a.slot_mapping[token];
    if (slot < 0 || slot >= a.num_slots) return;
    const uint16_t* src = lane < 64 ? a.c_kv + token * a.c_kv_stride + lane * 8
                                    : a.k_rope + token * a.k_rope_stride + (lane - 64) * 8;
    const int64_t page = slot / a.g.page_size;
    const int64_t off = slot % a.g.page_size;
    uint8_t* dst = a.cache + page * a.g.page_bytes + off * 1152 + lane * 16;
    *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(src);
}

}  // namespace

namespace {

template <bool kProt>
hipError_t launch_append(const AppendArgs& a, hipStream_t stream) {
    if (a.n == 0) return hipSuccess;
    const int64_t threads = static_cast<int64_t>(a.n) * kGroupsPerToken * kLanesPerGroup;
    const dim3 grid(static_cast<unsigned>((threads + kThreads - 1) / kThreads));
    const bool paper = a.g.paper_meta != 0;
    if (a.g.c_bits == 4) {
        if (paper) hipLaunchKernelGGL((lowbit_append_kernel<4, kProt, true>), grid, dim3(kThreads), 0, stream, a);
        else hipLaunchKernelGGL((lowbit_append_kernel<4, kProt, false>), grid, dim3(kThreads), 0, stream, a);
    } else {
        if (paper) hipLaunchKernelGGL((lowbit_append_kernel<2, kProt, true>), grid, dim3(kThreads), 0, stream, a);
        else hipLaunchKernelGGL((lowbit_append_kernel<2, kProt, false>), grid, dim3(kThreads), 0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_lowbit_append(const AppendArgs& a, hipStream_t stream) { return launch_append<false>(a, stream); }

hipError_t launch_lowbit_append_protected(const AppendArgs& a, hipStream_t stream) {
    return launch_append<true>(a, stream);
}

hipError_t launch_bf16_append(const AppendArgs& a, hipStream_t stream) {
    if (a.n == 0) return hipSuccess;
    const int64_t threads = static_cast<int64_t>(a.n) * 72;
    const dim3 grid(static_cast<unsigned>((threads + kThreads - 1) / kThreads));
    hipLaunchKernelGGL(bf16_append_kernel, grid, dim3(kThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace mla
