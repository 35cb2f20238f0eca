// Internal interface between the host ABI (mla_abi.cpp) and the HIP kernels.
// Not part of the public C ABI.
#pragma once

#include <cstdint>

#include <hip/hip_runtime_api.h>

namespace mla {

// Resolved byte geometry of a packed page (layout documented in mla_lowbit.h).
struct PageGeom {
    int32_t page_size;      // tokens per page
    int32_t c_bits;         // 4 or 2
    int32_t cc_bytes;       // content code bytes per token
    int32_t cr_bytes;       // RoPE code bytes per token
    int32_t off_cr;         // region offsets inside a page
    int32_t off_mc;
    int32_t off_mr;         // (fp16 metadata only)
    int64_t page_bytes;
    int32_t paper_meta;     // 1: the paper's metadata record at off_mc
};

struct AppendArgs {
    const uint16_t* c_kv;
    int64_t c_kv_stride;
    const uint16_t* k_rope;
    int64_t k_rope_stride;
    const int64_t* slot_mapping;
    int32_t n;
    uint8_t* cache;
    int64_t num_slots;      // num_pages * page_size
    PageGeom g;
    // BF16 protection writes (lowbit_append_kernel<CBITS, true> only)
    uint8_t* prot;
    int64_t num_prot;
    const int32_t* token_seq;   // [n] sequence of each token
    const int32_t* positions;   // [n] position of each token in its sequence
    const int32_t* seq_lens;    // [B] lengths after the append
    const int32_t* prot_slot;   // [B] buffer of each sequence
    int32_t B;
    int32_t sink, recent;
};

// Low-bit kinds: content bits and metadata storage (P: the paper's record).
enum CacheKind { KIND_C4R4 = 0, KIND_C2R4 = 1, KIND_BF16 = 2, KIND_C4R4P = 3, KIND_C2R4P = 4 };

struct DecodeArgs {
    const uint16_t* q_lat;
    const uint16_t* q_rope;
    const uint8_t* cache;
    int64_t num_pages;
    const int32_t* block_table;
    int32_t max_pages;
    const int32_t* seq_lens;
    int32_t B, s_q, H;
    float scale_log2;       // softmax_scale * log2(e)
    int32_t split_tokens;   // 0: unsplit
    const int32_t* split_indptr;
    int32_t num_work;       // B (unsplit) or total splits
    uint16_t* out;
    float* lse;
    float* part_m;
    float* part_s;
    uint16_t* part_o;       // fp16, normalized by part_s
    PageGeom g;             // for BF16: page_size and page_bytes only
    // BF16 protection (decode_kernel<KIND, true> only)
    const uint8_t* prot;    // protection buffers, num_prot x (sink + recent) rows of 1152 bytes
    int64_t num_prot;
    const int32_t* prot_slot;   // [B] buffer of each sequence
    int32_t sink, recent;
    // In-launch append (decode_kernel only; new_c == nullptr: none): token (b, i)
    // of [B][s_q], position seq_lens[b] - s_q + i of sequence b, quantized (or
    // copied, BF16) into slot new_slots[b * s_q + i] before it is read; under
    // protection also its bf16 row into the protection buffer.
    const uint16_t* new_c;
    int64_t new_c_stride;
    const uint16_t* new_k;
    int64_t new_k_stride;
    const int64_t* new_slots;
};

struct CombineArgs {
    const float* part_m;
    const float* part_s;
    const uint16_t* part_o;
    const int32_t* split_indptr;
    int32_t B, s_q, H;
    uint16_t* out;
    float* lse;
};

// Events for the next decode-kernel dispatch on this host thread (both null
// when none); take_launch_events() returns them and clears them.
struct LaunchEvents {
    hipEvent_t start, stop;
};
LaunchEvents take_launch_events();

hipError_t launch_lowbit_append(const AppendArgs& a, hipStream_t stream);
hipError_t launch_bf16_append(const AppendArgs& a, hipStream_t stream);
hipError_t launch_decode(CacheKind kind, const DecodeArgs& a, hipStream_t stream);
hipError_t launch_decode_protected(CacheKind kind, const DecodeArgs& a, hipStream_t stream);
// The same computation for few query rows (s_q * H <= kNarrowRows): 16 rows per one-wave workgroup.
constexpr int kNarrowRows = 32;

// Launch shapes, for the host's size checks (each kernel file asserts its own
// constants against these).  A dispatch packet holds the launch's work-item
// count in 32 bits, so a launch of more than kMaxDispatchItems work items
// cannot be expressed: the host refuses such shapes before any HIP call.
constexpr int64_t kMaxDispatchItems = 0xFFFFFFFFll;
constexpr int kDecodeThreads = 256;          // decode_attn.hip: 4 waves per workgroup
constexpr int kDecodeRowsPerBlock = 128;     // query rows per workgroup
constexpr int kNarrowThreads = 64;           // decode_narrow.hip: one wave per workgroup
constexpr int kNarrowRowsPerBlock = 16;
constexpr int kWorkGroupRound = 8;           // work items padded to a multiple of the 8 XCDs
constexpr int kCombineThreads = 256;         // combine.hip: at most one row per workgroup
constexpr int kAppendThreadsPerToken = 72;   // quant_append.hip: 9 groups x 8 lanes
constexpr int64_t kMaxAppendTokens = int64_t(1) << 25;
static_assert(kMaxAppendTokens * kAppendThreadsPerToken + 256 <= kMaxDispatchItems, "append launch size");

// Work items of a launch over the split (or unsplit) work list: padded to the
// XCD round, times the row blocks; the caller multiplies by the threads.
constexpr int64_t decode_workgroups(int64_t num_work, int64_t rows, int64_t rows_per_block) {
    return (num_work + kWorkGroupRound - 1) / kWorkGroupRound * kWorkGroupRound *
           ((rows + rows_per_block - 1) / rows_per_block);
}
hipError_t launch_decode_narrow(CacheKind kind, const DecodeArgs& a, hipStream_t stream);
hipError_t launch_decode_narrow_protected(CacheKind kind, const DecodeArgs& a, hipStream_t stream);
hipError_t launch_lowbit_append_protected(const AppendArgs& a, hipStream_t stream);
// num_splits (split_indptr[B]) chooses between one wave per row and four waves sharing a row.
hipError_t launch_combine(const CombineArgs& a, int32_t num_splits, hipStream_t stream);

// Split-partial storage owned by the library for the allocation-free decode
// entry point: at most kNoallocSplitRows partial rows (split x query row) of
// kNoallocRowBytes (fp16 latent, fp32 max and sum).  Returns this device's
// part_m / part_s / part_o addresses (resolved on the device's first call).
constexpr int64_t kNoallocSplitRows = 65536;
constexpr int64_t kNoallocRowBytes = 512 * 2 + 2 * 4;
hipError_t noalloc_partials(float** part_m, float** part_s, uint16_t** part_o);

}  // namespace mla
