// Host side of the C ABI declared in include/mla_lowbit.h: argument
// validation, page geometry, the split planner and kernel dispatch.
//
// This translation unit is plain C++ (it needs only the HIP runtime API
// types); every check below runs on the host before any HIP call is made.
#include "mla_lowbit.h"

#include <cmath>
#include <cstdint>

#include "internal.h"

namespace {

thread_local int g_last_hip_error = 0;
thread_local mla::LaunchEvents g_launch_events{nullptr, nullptr};

constexpr int32_t kDc = 512;
constexpr int32_t kDr = 64;
constexpr int32_t kGroup = 64;
constexpr int32_t kTile = 32;

constexpr int32_t kMaxProtRows = 65536;
constexpr int32_t kPaperMetaBytes = 32;
constexpr int64_t kReverseMapBytes = 8;     // per physical page, eq. physical_cache_storage
constexpr int64_t kProtRowBytes = (kDc + kDr) * 2;

bool aligned(const void* p, uintptr_t n) { return (reinterpret_cast<uintptr_t>(p) % n) == 0; }

int check_policy(const mla_protect_policy* p) {
    if (p == nullptr) return MLA_EINVAL;
    if (p->sink < 0 || p->recent < 0) return MLA_EINVAL;
    const int64_t rows = static_cast<int64_t>(p->sink) + p->recent;
    if (rows < 1 || rows > kMaxProtRows) return MLA_EINVAL;
    return MLA_OK;
}

// Tiles of 32 keys a sequence of length L is processed in under protection:
// packed tiles from the one holding token `sink` up to token L - recent - 1,
// then the protected rows (sink + recent of them, or all L when the packed
// range is empty).
int64_t protected_tile_count(int64_t L, int64_t sink, int64_t recent) {
    const bool has_packed = L - recent > sink;
    const int64_t n_pk = has_packed ? (L - recent + kTile - 1) / kTile - sink / kTile : 0;
    const int64_t n_prot = has_packed ? sink + recent : L;
    return n_pk + (n_prot + kTile - 1) / kTile;
}

// The protection arguments of a decode call (null: no protection).
struct ProtDecode {
    const mla_protect_policy* policy;
    const void* prot;
    int64_t num_prot;
    const int32_t* prot_slot;
};

constexpr int32_t kMaxPageSize = 1 << 20;

// Structural checks shared by both cache kinds.
int check_shape(const mla_cache_format* f) {
    if (f == nullptr) return MLA_EINVAL;
    if (f->d_c <= 0 || f->d_r <= 0 || f->page_size <= 0) return MLA_EINVAL;
    if (f->page_size % 16 != 0) return MLA_EINVAL;
    if (f->d_c != kDc || f->d_r != kDr) return MLA_ENOTSUP;
    if (f->page_size % kTile != 0) return MLA_ENOTSUP;
    if (f->page_size > kMaxPageSize) return MLA_ENOTSUP;      // a page's bytes fit 31 bits
    return MLA_OK;
}

int check_lowbit_format(const mla_cache_format* f) {
    const int st = check_shape(f);
    if (st != MLA_OK) return st;
    if (f->group <= 0 || f->d_c % f->group != 0 || f->d_r % f->group != 0) return MLA_EINVAL;
    if (f->c_bits != 4 && f->c_bits != 2) return MLA_EINVAL;
    if (f->r_bits != 4) return MLA_EINVAL;
    if (f->meta != MLA_META_FP16 && f->meta != MLA_META_PAPER) return MLA_EINVAL;
    if (f->group != kGroup) return MLA_ENOTSUP;
    return MLA_OK;
}

mla::PageGeom lowbit_geom(const mla_cache_format* f) {
    mla::PageGeom g{};
    const int32_t P = f->page_size;
    g.page_size = P;
    g.c_bits = f->c_bits;
    g.cc_bytes = f->d_c * f->c_bits / 8;
    g.cr_bytes = f->d_r * f->r_bits / 8;
    g.off_cr = P * g.cc_bytes;
    g.off_mc = g.off_cr + P * g.cr_bytes;
    int64_t end;
    if (f->meta == MLA_META_PAPER) {
        // one 32-byte record per token: bf16 scales, byte zeros, fp32 RoPE scale, byte RoPE zero
        g.paper_meta = 1;
        g.off_mr = g.off_mc;
        end = g.off_mc + static_cast<int64_t>(P) * kPaperMetaBytes;
    } else {
        g.off_mr = g.off_mc + P * (f->d_c / f->group) * 4;
        end = g.off_mr + static_cast<int64_t>(P) * (f->d_r / f->group) * 4;
    }
    g.page_bytes = (end + 255) / 256 * 256;
    return g;
}

mla::PageGeom bf16_geom(const mla_cache_format* f) {
    mla::PageGeom g{};
    g.page_size = f->page_size;
    g.page_bytes = static_cast<int64_t>(f->page_size) * (f->d_c + f->d_r) * 2;
    return g;
}

int hip_status(hipError_t e) {
    if (e == hipSuccess) return MLA_OK;
    g_last_hip_error = static_cast<int>(e);
    return MLA_EHIP;
}

int check_append(const uint16_t* c_kv, int64_t c_kv_stride, const uint16_t* k_rope, int64_t k_rope_stride,
                 const int64_t* slot_mapping, int32_t n, const void* cache, int64_t num_pages) {
    if (n < 0 || num_pages < 0) return MLA_EINVAL;
    if (n == 0) return MLA_OK;
    if (n > mla::kMaxAppendTokens) return MLA_ENOTSUP;   // the launch would not fit one dispatch
    if (c_kv == nullptr || k_rope == nullptr || slot_mapping == nullptr || cache == nullptr) return MLA_EINVAL;
    if (num_pages == 0) return MLA_EINVAL;
    if (c_kv_stride < kDc || k_rope_stride < kDr) return MLA_EINVAL;
    if (!aligned(cache, 256)) return MLA_EINVAL;
    // 16-byte vector loads of 8 channels
    if (c_kv_stride % 8 != 0 || k_rope_stride % 8 != 0 || !aligned(c_kv, 16) || !aligned(k_rope, 16))
        return MLA_ENOTSUP;
    return MLA_OK;
}

int append_common(const mla_cache_format* f, bool lowbit, const uint16_t* c_kv, int64_t c_kv_stride,
                  const uint16_t* k_rope, int64_t k_rope_stride, const int64_t* slot_mapping, int32_t n,
                  void* cache, int64_t num_pages, hipStream_t stream, mla::AppendArgs a = {}) {
    int st = lowbit ? check_lowbit_format(f) : check_shape(f);
    if (st != MLA_OK) return st;
    st = check_append(c_kv, c_kv_stride, k_rope, k_rope_stride, slot_mapping, n, cache, num_pages);
    if (st != MLA_OK || n == 0) return st;
    a.c_kv = c_kv;
    a.c_kv_stride = c_kv_stride;
    a.k_rope = k_rope;
    a.k_rope_stride = k_rope_stride;
    a.slot_mapping = slot_mapping;
    a.n = n;
    a.cache = static_cast<uint8_t*>(cache);
    a.num_slots = num_pages * f->page_size;
    a.g = lowbit ? lowbit_geom(f) : bf16_geom(f);
    if (a.prot != nullptr) return hip_status(mla::launch_lowbit_append_protected(a, stream));
    return hip_status(lowbit ? mla::launch_lowbit_append(a, stream) : mla::launch_bf16_append(a, stream));
}

struct NewTokens {
    const uint16_t* c_kv;
    int64_t c_kv_stride;
    const uint16_t* k_rope;
    int64_t k_rope_stride;
    const int64_t* slot_mapping;
};

// Whether the decode launch over num_work work items fits one dispatch (its
// work-item count is 32 bits): the wide kernel's 256-thread workgroups of 128
// rows, or the 16-row kernel's one-wave workgroups when s_q * H <= 32.
bool decode_fits(int64_t num_work, int32_t s_q, int32_t H) {
    const int64_t rows = static_cast<int64_t>(s_q) * H;
    const bool narrow = rows <= mla::kNarrowRows;
    const int64_t groups = mla::decode_workgroups(num_work, rows, narrow ? mla::kNarrowRowsPerBlock
                                                                         : mla::kDecodeRowsPerBlock);
    return groups * (narrow ? mla::kNarrowThreads : mla::kDecodeThreads) <= mla::kMaxDispatchItems;
}

// Host validation of a decode call (no HIP call); part_* are checked only when
// check_parts is set (the allocation-free entry point supplies its own).
int check_decode(const mla_cache_format* f, bool lowbit, const uint16_t* q_lat, const uint16_t* q_rope,
                 const void* cache, int64_t num_pages, const int32_t* block_table, int32_t max_pages_per_seq,
                 const int32_t* seq_lens, int32_t B, int32_t s_q, int32_t H, float softmax_scale,
                 int32_t split_tokens, const int32_t* split_indptr, int32_t num_splits, const uint16_t* out,
                 const float* part_m, const float* part_s, const uint16_t* part_o, const ProtDecode* pd,
                 bool check_parts) {
    int st = lowbit ? check_lowbit_format(f) : check_shape(f);
    if (st != MLA_OK) return st;
    if (pd != nullptr) {
        st = check_policy(pd->policy);
        if (st != MLA_OK) return st;
        if (pd->num_prot < 0) return MLA_EINVAL;
    }
    if (B < 0 || num_pages < 0 || max_pages_per_seq <= 0 || split_tokens < 0) return MLA_EINVAL;
    if (s_q != 1 && s_q != 2) return MLA_EINVAL;
    if (H <= 0 || H % 16 != 0) return MLA_EINVAL;
    if (!std::isfinite(softmax_scale) || !(softmax_scale > 0.0f)) return MLA_EINVAL;
    if (split_tokens % kTile != 0) return MLA_ENOTSUP;
    if (B == 0) return MLA_OK;   // nothing is read or written
    if (q_lat == nullptr || q_rope == nullptr || cache == nullptr || block_table == nullptr || seq_lens == nullptr)
        return MLA_EINVAL;
    if (num_pages == 0) return MLA_EINVAL;
    if (!aligned(cache, 256)) return MLA_EINVAL;
    if (!aligned(q_lat, 16) || !aligned(q_rope, 16)) return MLA_ENOTSUP;
    if (pd != nullptr) {
        if (pd->prot == nullptr || pd->prot_slot == nullptr || pd->num_prot == 0) return MLA_EINVAL;
        if (!aligned(pd->prot, 16)) return MLA_ENOTSUP;
    }
    if (split_tokens == 0) {
        if (out == nullptr) return MLA_EINVAL;
        if (!aligned(out, 16)) return MLA_ENOTSUP;
    } else {
        if (split_indptr == nullptr || num_splits < 0) return MLA_EINVAL;
        if (check_parts) {
            if (part_m == nullptr || part_s == nullptr || part_o == nullptr) return MLA_EINVAL;
            if (!aligned(part_o, 16)) return MLA_ENOTSUP;
        }
    }
    if (!decode_fits(split_tokens == 0 ? B : num_splits, s_q, H)) return MLA_ENOTSUP;
    return MLA_OK;
}

int decode_common(const mla_cache_format* f, bool lowbit, const uint16_t* q_lat, const uint16_t* q_rope,
                  const void* cache, int64_t num_pages, const int32_t* block_table, int32_t max_pages_per_seq,
                  const int32_t* seq_lens, int32_t B, int32_t s_q, int32_t H, float softmax_scale,
                  int32_t split_tokens, const int32_t* split_indptr, int32_t num_splits, uint16_t* out,
                  float* lse, float* part_m, float* part_s, uint16_t* part_o, const ProtDecode* pd,
                  hipStream_t stream, const NewTokens* nt = nullptr) {
    int st = check_decode(f, lowbit, q_lat, q_rope, cache, num_pages, block_table, max_pages_per_seq, seq_lens, B,
                          s_q, H, softmax_scale, split_tokens, split_indptr, num_splits, out, part_m, part_s, part_o,
                          pd, true);
    if (st != MLA_OK || B == 0) return st;
    mla::DecodeArgs a{};
    a.q_lat = q_lat;
    a.q_rope = q_rope;
    a.cache = static_cast<const uint8_t*>(cache);
    a.num_pages = num_pages;
    a.block_table = block_table;
    a.max_pages = max_pages_per_seq;
    a.seq_lens = seq_lens;
    a.B = B;
    a.s_q = s_q;
    a.H = H;
    a.scale_log2 = softmax_scale * 1.4426950408889634f;
    a.split_tokens = split_tokens;
    a.split_indptr = split_indptr;
    a.num_work = split_tokens == 0 ? B : num_splits;
    a.out = out;
    a.lse = lse;
    a.part_m = part_m;
    a.part_s = part_s;
    a.part_o = part_o;
    a.g = lowbit ? lowbit_geom(f) : bf16_geom(f);
    const bool paper = f->meta == MLA_META_PAPER;
    const mla::CacheKind kind = !lowbit ? mla::KIND_BF16
                                : f->c_bits == 4 ? (paper ? mla::KIND_C4R4P : mla::KIND_C4R4)
                                                 : (paper ? mla::KIND_C2R4P : mla::KIND_C2R4);
    const bool narrow = s_q * H <= mla::kNarrowRows;
    if (nt != nullptr && B > 0) {
        // the workgroups that read a new token write it inside the decode launch
        a.new_c = nt->c_kv;
        a.new_c_stride = nt->c_kv_stride;
        a.new_k = nt->k_rope;
        a.new_k_stride = nt->k_rope_stride;
        a.new_slots = nt->slot_mapping;
    }
    if (pd == nullptr)
        return hip_status(narrow ? mla::launch_decode_narrow(kind, a, stream) : mla::launch_decode(kind, a, stream));
    a.prot = static_cast<const uint8_t*>(pd->prot);
    a.num_prot = pd->num_prot;
    a.prot_slot = pd->prot_slot;
    a.sink = pd->policy->sink;
    a.recent = pd->policy->recent;
    return hip_status(narrow ? mla::launch_decode_narrow_protected(kind, a, stream)
                             : mla::launch_decode_protected(kind, a, stream));
}

}  // namespace

namespace mla {
LaunchEvents take_launch_events() {
    const LaunchEvents e = g_launch_events;
    g_launch_events = LaunchEvents{nullptr, nullptr};
    return e;
}
}  // namespace mla

// Append the step's new tokens, then decode (one launch for the wide kernel).
static int append_decode(const mla_cache_format* f, bool lowbit, const uint16_t* c_kv, int64_t c_kv_stride,
                  const uint16_t* k_rope, int64_t k_rope_stride, const int64_t* slot_mapping, const uint16_t* q_lat,
                  const uint16_t* q_rope, void* cache, int64_t num_pages, const int32_t* block_table,
                  int32_t max_pages_per_seq, const int32_t* seq_lens, int32_t B, int32_t s_q, int32_t H,
                  float softmax_scale, int32_t split_tokens, const int32_t* split_indptr, int32_t num_splits,
                  uint16_t* out, float* lse, float* part_m, float* part_s, uint16_t* part_o, hipStream_t stream) {
    int st = lowbit ? check_lowbit_format(f) : check_shape(f);
    if (st != MLA_OK) return st;
    if (B < 0 || s_q < 0) return MLA_EINVAL;
    if (s_q != 1 && s_q != 2) return MLA_EINVAL;
    if (static_cast<int64_t>(B) * s_q > mla::kMaxAppendTokens) return MLA_ENOTSUP;
    st = check_append(c_kv, c_kv_stride, k_rope, k_rope_stride, slot_mapping, B * s_q, cache, num_pages);
    if (st != MLA_OK) return st;
    const NewTokens nt{c_kv, c_kv_stride, k_rope, k_rope_stride, slot_mapping};
    return decode_common(f, lowbit, q_lat, q_rope, cache, num_pages, block_table, max_pages_per_seq, seq_lens, B,
                         s_q, H, softmax_scale, split_tokens, split_indptr, num_splits, out, lse, part_m, part_s,
                         part_o, nullptr, stream, &nt);
}

extern "C" {

int64_t mla_lowbit_page_bytes(const mla_cache_format* f) {
    if (check_lowbit_format(f) != MLA_OK) return -1;
    return lowbit_geom(f).page_bytes;
}

int64_t mla_bf16_page_bytes(const mla_cache_format* f) {
    if (check_shape(f) != MLA_OK) return -1;
    return bf16_geom(f).page_bytes;
}

int mla_lowbit_quant_append(const mla_cache_format* f, const uint16_t* c_kv, int64_t c_kv_stride,
                            const uint16_t* k_rope, int64_t k_rope_stride, const int64_t* slot_mapping,
                            int32_t n, void* cache, int64_t num_pages, hipStream_t stream) {
    return append_common(f, true, c_kv, c_kv_stride, k_rope, k_rope_stride, slot_mapping, n, cache, num_pages,
                         stream);
}

int mla_bf16_append(const mla_cache_format* f, const uint16_t* c_kv, int64_t c_kv_stride,
                    const uint16_t* k_rope, int64_t k_rope_stride, const int64_t* slot_mapping, int32_t n,
                    void* cache, int64_t num_pages, hipStream_t stream) {
    return append_common(f, false, c_kv, c_kv_stride, k_rope, k_rope_stride, slot_mapping, n, cache, num_pages,
                         stream);
}

int64_t mla_persistent_cache_bytes(const mla_cache_format* f, const mla_protect_policy* p, int64_t L) {
    if (f == nullptr || L < 0) return -1;
    constexpr int64_t kMax = INT64_MAX;
    if (f->c_bits == 16) {
        if (check_shape(f) != MLA_OK || p != nullptr) return -1;
        const int64_t pages = L / f->page_size + (L % f->page_size != 0);
        const int64_t per = bf16_geom(f).page_bytes;
        return pages > kMax / per ? -1 : pages * per;
    }
    if (check_lowbit_format(f) != MLA_OK) return -1;
    if (p != nullptr && check_policy(p) != MLA_OK) return -1;
    const int64_t pages = L / f->page_size + (L % f->page_size != 0);
    const int64_t prot = p == nullptr ? 0 : (static_cast<int64_t>(p->sink) + p->recent) * kProtRowBytes;
    const int64_t per = lowbit_geom(f).page_bytes + kReverseMapBytes;
    if (pages > (kMax - prot) / per) return -1;     // the result does not fit int64
    return pages * per + prot;
}

int64_t mla_protect_buffer_bytes(const mla_cache_format* f, const mla_protect_policy* p) {
    if (check_lowbit_format(f) != MLA_OK || check_policy(p) != MLA_OK) return -1;
    return (static_cast<int64_t>(p->sink) + p->recent) * kProtRowBytes;
}

int mla_lowbit_quant_append_protected(const mla_cache_format* f, const mla_protect_policy* p,
                                      const uint16_t* c_kv, int64_t c_kv_stride, const uint16_t* k_rope,
                                      int64_t k_rope_stride, const int64_t* slot_mapping, int32_t n, void* cache,
                                      int64_t num_pages, const int32_t* token_seq, const int32_t* positions,
                                      const int32_t* seq_lens, const int32_t* prot_slot, int32_t B, void* prot,
                                      int64_t num_prot, hipStream_t stream) {
    int st = check_policy(p);
    if (st != MLA_OK) return st;
    if (B < 0 || num_prot < 0) return MLA_EINVAL;
    if (n > 0) {
        if (token_seq == nullptr || positions == nullptr || seq_lens == nullptr || prot_slot == nullptr ||
            prot == nullptr || B == 0 || num_prot == 0)
            return MLA_EINVAL;
        if (!aligned(prot, 16)) return MLA_ENOTSUP;
    }
    mla::AppendArgs a{};
    a.prot = static_cast<uint8_t*>(prot);
    a.num_prot = num_prot;
    a.token_seq = token_seq;
    a.positions = positions;
    a.seq_lens = seq_lens;
    a.prot_slot = prot_slot;
    a.B = B;
    a.sink = p->sink;
    a.recent = p->recent;
    return append_common(f, true, c_kv, c_kv_stride, k_rope, k_rope_stride, slot_mapping, n, cache, num_pages,
                         stream, a);
}

int32_t mla_plan_splits_protected(const int32_t* seq_lens, int32_t B, int32_t split_tokens,
                                  const mla_protect_policy* p, int32_t* split_indptr) {
    if (seq_lens == nullptr || split_indptr == nullptr || B < 0 || split_tokens <= 0) return -MLA_EINVAL;
    if (check_policy(p) != MLA_OK) return -MLA_EINVAL;
    if (split_tokens % kTile != 0) return -MLA_ENOTSUP;
    const int64_t per_split = split_tokens / kTile;
    int64_t total = 0;
    split_indptr[0] = 0;
    for (int32_t b = 0; b < B; ++b) {
        if (seq_lens[b] < 1) return -MLA_EINVAL;
        total += (protected_tile_count(seq_lens[b], p->sink, p->recent) + per_split - 1) / per_split;
        if (total > INT32_MAX) return -MLA_EINVAL;
        split_indptr[b + 1] = static_cast<int32_t>(total);
    }
    return static_cast<int32_t>(total);
}

int mla_lowbit_decode_attn_protected(const mla_cache_format* f, const mla_protect_policy* p,
                                     const uint16_t* q_lat, const uint16_t* q_rope, const void* cache,
                                     int64_t num_pages, const int32_t* block_table, int32_t max_pages_per_seq,
                                     const int32_t* seq_lens, int32_t B, int32_t s_q, int32_t H,
                                     float softmax_scale, const void* prot, int64_t num_prot,
                                     const int32_t* prot_slot, int32_t split_tokens, const int32_t* split_indptr,
                                     int32_t num_splits, uint16_t* out, float* lse, float* part_m, float* part_s,
                                     uint16_t* part_o, hipStream_t stream) {
    const ProtDecode pd{p, prot, num_prot, prot_slot};
    return decode_common(f, true, q_lat, q_rope, cache, num_pages, block_table, max_pages_per_seq, seq_lens, B,
                         s_q, H, softmax_scale, split_tokens, split_indptr, num_splits, out, lse, part_m, part_s,
                         part_o, &pd, stream);
}

int mla_lowbit_append_decode_attn_protected(const mla_cache_format* f, const mla_protect_policy* p,
                                            const uint16_t* c_kv, int64_t c_kv_stride, const uint16_t* k_rope,
                                            int64_t k_rope_stride, const int64_t* slot_mapping,
                                            const uint16_t* q_lat, const uint16_t* q_rope, void* cache,
                                            int64_t num_pages, const int32_t* block_table,
                                            int32_t max_pages_per_seq, const int32_t* seq_lens, int32_t B,
                                            int32_t s_q, int32_t H, float softmax_scale, void* prot,
                                            int64_t num_prot, const int32_t* prot_slot, int32_t split_tokens,
                                            const int32_t* split_indptr, int32_t num_splits, uint16_t* out,
                                            float* lse, float* part_m, float* part_s, uint16_t* part_o,
                                            hipStream_t stream) {
    int st = check_lowbit_format(f);
    if (st != MLA_OK) return st;
    st = check_policy(p);
    if (st != MLA_OK) return st;
    if (B < 0 || s_q < 0) return MLA_EINVAL;
    if (s_q != 1 && s_q != 2) return MLA_EINVAL;
    if (static_cast<int64_t>(B) * s_q > mla::kMaxAppendTokens) return MLA_ENOTSUP;
    st = check_append(c_kv, c_kv_stride, k_rope, k_rope_stride, slot_mapping, B * s_q, cache, num_pages);
    if (st != MLA_OK) return st;
    const NewTokens nt{c_kv, c_kv_stride, k_rope, k_rope_stride, slot_mapping};
    const ProtDecode pd{p, prot, num_prot, prot_slot};
    return decode_common(f, true, q_lat, q_rope, cache, num_pages, block_table, max_pages_per_seq, seq_lens, B,
                         s_q, H, softmax_scale, split_tokens, split_indptr, num_splits, out, lse, part_m, part_s,
                         part_o, &pd, stream, &nt);
}

int32_t mla_plan_splits(const int32_t* seq_lens, int32_t B, int32_t split_tokens, int32_t* split_indptr) {
    if (seq_lens == nullptr || split_indptr == nullptr || B < 0 || split_tokens <= 0) return -MLA_EINVAL;
    if (split_tokens % kTile != 0) return -MLA_ENOTSUP;
    int64_t total = 0;
    split_indptr[0] = 0;
    for (int32_t b = 0; b < B; ++b) {
        if (seq_lens[b] < 1) return -MLA_EINVAL;
        total += (static_cast<int64_t>(seq_lens[b]) + split_tokens - 1) / split_tokens;
        if (total > INT32_MAX) return -MLA_EINVAL;
        split_indptr[b + 1] = static_cast<int32_t>(total);
    }
    return static_cast<int32_t>(total);
}

int mla_lowbit_decode_attn(const mla_cache_format* f, const uint16_t* q_lat, const uint16_t* q_rope,
                           const void* cache, int64_t num_pages, const int32_t* block_table,
                           int32_t max_pages_per_seq, const int32_t* seq_lens, int32_t B, int32_t s_q, int32_t H,
                           float softmax_scale, int32_t split_tokens, const int32_t* split_indptr,
                           int32_t num_splits, uint16_t* out, float* lse, float* part_m, float* part_s,
                           uint16_t* part_o, hipStream_t stream) {
    return decode_common(f, true, q_lat, q_rope, cache, num_pages, block_table, max_pages_per_seq, seq_lens, B,
                         s_q, H, softmax_scale, split_tokens, split_indptr, num_splits, out, lse, part_m, part_s,
                         part_o, nullptr, stream);
}

int mla_bf16_decode_attn(const mla_cache_format* f, const uint16_t* q_lat, const uint16_t* q_rope,
                         const void* cache, int64_t num_pages, const int32_t* block_table, int32_t max_pages_per_seq,
                         const int32_t* seq_lens, int32_t B, int32_t s_q, int32_t H, float softmax_scale,
                         int32_t split_tokens, const int32_t* split_indptr, int32_t num_splits, uint16_t* out,
                         float* lse, float* part_m, float* part_s, uint16_t* part_o, hipStream_t stream) {
    return decode_common(f, false, q_lat, q_rope, cache, num_pages, block_table, max_pages_per_seq, seq_lens, B,
                         s_q, H, softmax_scale, split_tokens, split_indptr, num_splits, out, lse, part_m, part_s,
                         part_o, nullptr, stream);
}

int mla_lowbit_append_decode_attn(const mla_cache_format* f, const uint16_t* c_kv, int64_t c_kv_stride,
                                  const uint16_t* k_rope, int64_t k_rope_stride, const int64_t* slot_mapping,
                                  const uint16_t* q_lat, const uint16_t* q_rope, void* cache, int64_t num_pages,
                                  const int32_t* block_table, int32_t max_pages_per_seq, const int32_t* seq_lens,
                                  int32_t B, int32_t s_q, int32_t H, float softmax_scale, int32_t split_tokens,
                                  const int32_t* split_indptr, int32_t num_splits, uint16_t* out, float* lse,
                                  float* part_m, float* part_s, uint16_t* part_o, hipStream_t stream) {
    return append_decode(f, true, c_kv, c_kv_stride, k_rope, k_rope_stride, slot_mapping, q_lat, q_rope, cache,
                         num_pages, block_table, max_pages_per_seq, seq_lens, B, s_q, H, softmax_scale, split_tokens,
                         split_indptr, num_splits, out, lse, part_m, part_s, part_o, stream);
}

int mla_bf16_append_decode_attn(const mla_cache_format* f, const uint16_t* c_kv, int64_t c_kv_stride,
                                const uint16_t* k_rope, int64_t k_rope_stride, const int64_t* slot_mapping,
                                const uint16_t* q_lat, const uint16_t* q_rope, void* cache, int64_t num_pages,
                                const int32_t* block_table, int32_t max_pages_per_seq, const int32_t* seq_lens,
                                int32_t B, int32_t s_q, int32_t H, float softmax_scale, int32_t split_tokens,
                                const int32_t* split_indptr, int32_t num_splits, uint16_t* out, float* lse,
                                float* part_m, float* part_s, uint16_t* part_o, hipStream_t stream) {
    return append_decode(f, false, c_kv, c_kv_stride, k_rope, k_rope_stride, slot_mapping, q_lat, q_rope, cache,
                         num_pages, block_table, max_pages_per_seq, seq_lens, B, s_q, H, softmax_scale, split_tokens,
                         split_indptr, num_splits, out, lse, part_m, part_s, part_o, stream);
}

int mla_lowbit_decode_attn_noalloc(const mla_cache_format* f, const uint16_t* q_lat, const uint16_t* q_rope,
                                   const void* cache, int64_t num_pages, const int32_t* block_table,
                                   int32_t max_pages_per_seq, const int32_t* seq_lens, int32_t B, int32_t s_q,
                                   int32_t H, float softmax_scale, int32_t split_tokens, const int32_t* split_indptr,
                                   int32_t num_splits, uint16_t* out, float* lse, hipStream_t stream) {
    if (split_tokens == 0)
        return decode_common(f, true, q_lat, q_rope, cache, num_pages, block_table, max_pages_per_seq, seq_lens, B,
                             s_q, H, softmax_scale, 0, nullptr, 0, out, lse, nullptr, nullptr, nullptr, nullptr,
                             stream);
    // every check of the decode and the combine, before any HIP call
    int st = check_decode(f, true, q_lat, q_rope, cache, num_pages, block_table, max_pages_per_seq, seq_lens, B, s_q,
                          H, softmax_scale, split_tokens, split_indptr, num_splits, out, nullptr, nullptr, nullptr,
                          nullptr, false);
    if (st != MLA_OK || B == 0) return st;
    if (static_cast<int64_t>(num_splits) * s_q * H > mla::kNoallocSplitRows) return MLA_ENOTSUP;
    if (out == nullptr) return MLA_EINVAL;
    if (!aligned(out, 16)) return MLA_ENOTSUP;
    float* part_m = nullptr;
    float* part_s = nullptr;
    uint16_t* part_o = nullptr;
    st = hip_status(mla::noalloc_partials(&part_m, &part_s, &part_o));
    if (st != MLA_OK) return st;
    st = decode_common(f, true, q_lat, q_rope, cache, num_pages, block_table, max_pages_per_seq, seq_lens, B, s_q, H,
                       softmax_scale, split_tokens, split_indptr, num_splits, out, lse, part_m, part_s, part_o,
                       nullptr, stream);
    if (st != MLA_OK) return st;
    return mla_splitkv_combine(part_m, part_s, part_o, split_indptr, num_splits, B, s_q, H, kDc, out, lse, stream);
}

int mla_splitkv_combine(const float* part_m, const float* part_s, const uint16_t* part_o, const int32_t* split_indptr,
                        int32_t num_splits, int32_t B, int32_t s_q, int32_t H, int32_t d_c, uint16_t* out,
                        float* lse, hipStream_t stream) {
    if (B < 0 || d_c <= 0 || num_splits < 0) return MLA_EINVAL;
    if (s_q != 1 && s_q != 2) return MLA_EINVAL;
    if (H <= 0 || H % 16 != 0) return MLA_EINVAL;
    if (d_c != kDc) return MLA_ENOTSUP;
    if (B == 0) return MLA_OK;   // nothing is read or written
    if (part_m == nullptr || part_s == nullptr || part_o == nullptr || split_indptr == nullptr || out == nullptr)
        return MLA_EINVAL;
    if (!aligned(part_o, 16) || !aligned(out, 16)) return MLA_ENOTSUP;
    // at most one row per 256-thread workgroup, workgroups padded to a multiple of 8
    const int64_t rows = static_cast<int64_t>(B) * s_q * H;
    if ((rows + mla::kWorkGroupRound - 1) / mla::kWorkGroupRound * mla::kWorkGroupRound * mla::kCombineThreads >
        mla::kMaxDispatchItems)
        return MLA_ENOTSUP;
    mla::CombineArgs a{};
    a.part_m = part_m;
    a.part_s = part_s;
    a.part_o = part_o;
    a.split_indptr = split_indptr;
    a.B = B;
    a.s_q = s_q;
    a.H = H;
    a.out = out;
    a.lse = lse;
    return hip_status(mla::launch_combine(a, num_splits, stream));
}

const char* mla_status_str(int status) {
    switch (status) {
        case MLA_OK: return "MLA_OK";
        case MLA_EINVAL: return "MLA_EINVAL: invalid argument";
        case MLA_ENOTSUP: return "MLA_ENOTSUP: shape or alignment not supported";
        case MLA_EHIP: return "MLA_EHIP: HIP launch failed";
        default: return "MLA: unknown status";
    }
}

int mla_last_hip_error(void) { return g_last_hip_error; }

int mla_time_next_decode_launch(hipEvent_t start, hipEvent_t stop) {
    if ((start == nullptr) != (stop == nullptr)) return MLA_EINVAL;
    g_launch_events = mla::LaunchEvents{start, stop};
    return MLA_OK;
}

}  // extern "C"
