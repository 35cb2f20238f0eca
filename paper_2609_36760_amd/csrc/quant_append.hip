// Quantize-and-append writer for the packed dual-path cache, and the plain
// BF16 append used by the unquantized comparison cache.  The quantizer, the
// code layout and the metadata storage are in writer_common.h (shared with the
// decode kernel's in-launch append); one group of 64 channels per 8 lanes.
//
// With BF16 protection (Sec. 3.3; Appendix C.5, "BF16 protection and cache
// lifecycle") the same lanes also store the bf16 values they loaded into the
// token's row of its sequence's protection buffer when the token is protected
// once the append is done: position p < sink (row p) or p >= L - recent
// (row sink + (p - sink) mod recent, a ring), L the sequence's new length.
// Tokens leaving the window keep the packed copy written here at insertion.
#include <hip/hip_runtime.h>

#include "internal.h"
#include "writer_common.h"

namespace mla {
namespace {

using wc::kGroup;
using wc::kGroupsPerToken;
using wc::kLanesPerGroup;
constexpr int kThreads = 256;
static_assert(kGroupsPerToken * kLanesPerGroup == kAppendThreadsPerToken, "launch shape the host checks");

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

    wc::quantize_store<CBITS, kPaper>(raw, rope, g, lig, a.cache + slot / a.g.page_size * a.g.page_bytes,
                                      slot % a.g.page_size, a.g);
}

// BF16 comparison cache: row = [c_kv (512) | k_rope (64)] bf16; 72 lanes per
// token, 16 bytes each.
__global__ __launch_bounds__(kThreads) void bf16_append_kernel(AppendArgs a) {
    constexpr int kLanesPerToken = 72;     // 64 content + 8 RoPE pieces of 16 bytes
    static_assert(kLanesPerToken == kAppendThreadsPerToken, "launch shape the host checks");
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
    const int64_t threads = static_cast<int64_t>(a.n) * kAppendThreadsPerToken;
    const dim3 grid(static_cast<unsigned>((threads + kThreads - 1) / kThreads));
    hipLaunchKernelGGL(bf16_append_kernel, grid, dim3(kThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace mla
