// Host-only driver of the C ABI (csrc/mla_abi.cpp), built with AddressSanitizer
// and UndefinedBehaviorSanitizer by tests/test_abi_sanitized.py.  The kernel
// launchers are replaced by stubs that record their arguments, so every entry
// point runs its host code -- validation, geometry, planners, dispatch -- with
// no GPU and no HIP runtime.  Exits non-zero on the first failed check; the
// sanitizers abort on any memory error or undefined behaviour.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <limits>
#include <vector>

#include "internal.h"
#include "mla_lowbit.h"

namespace {

int g_failures = 0;
int g_decode_calls = 0, g_combine_calls = 0, g_append_calls = 0;
mla::DecodeArgs g_last_decode{};
mla::CombineArgs g_last_combine{};
mla::AppendArgs g_last_append{};
int32_t g_last_combine_splits = -1;
mla::CacheKind g_last_kind = mla::KIND_C4R4;
bool g_last_narrow = false, g_last_protected = false;
mla::LaunchEvents g_last_events{nullptr, nullptr};
alignas(256) uint8_t g_partials[1 << 16];

#define CHECK(cond)                                                              \
    do {                                                                         \
        if (!(cond)) {                                                           \
            std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
            ++g_failures;                                                        \
        }                                                                        \
    } while (0)

hipError_t record_decode(mla::CacheKind kind, const mla::DecodeArgs& a, bool narrow, bool prot) {
    ++g_decode_calls;
    g_last_decode = a;
    g_last_kind = kind;
    g_last_narrow = narrow;
    g_last_protected = prot;
    g_last_events = mla::take_launch_events();
    return hipSuccess;
}

}  // namespace

namespace mla {
hipError_t launch_lowbit_append(const AppendArgs& a, hipStream_t) { ++g_append_calls; g_last_append = a; return hipSuccess; }
hipError_t launch_bf16_append(const AppendArgs& a, hipStream_t) { ++g_append_calls; g_last_append = a; return hipSuccess; }
hipError_t launch_lowbit_append_protected(const AppendArgs& a, hipStream_t) {
    ++g_append_calls;
    g_last_append = a;
    return hipSuccess;
}
hipError_t launch_decode(CacheKind k, const DecodeArgs& a, hipStream_t) { return record_decode(k, a, false, false); }
hipError_t launch_decode_protected(CacheKind k, const DecodeArgs& a, hipStream_t) {
    return record_decode(k, a, false, true);
}
hipError_t launch_decode_narrow(CacheKind k, const DecodeArgs& a, hipStream_t) { return record_decode(k, a, true, false); }
hipError_t launch_decode_narrow_protected(CacheKind k, const DecodeArgs& a, hipStream_t) {
    return record_decode(k, a, true, true);
}
hipError_t launch_combine(const CombineArgs& a, int32_t num_splits, hipStream_t) {
    ++g_combine_calls;
    g_last_combine = a;
    g_last_combine_splits = num_splits;
    return hipSuccess;
}
hipError_t noalloc_partials(float** part_m, float** part_s, uint16_t** part_o) {
    *part_o = reinterpret_cast<uint16_t*>(g_partials);
    *part_m = reinterpret_cast<float*>(g_partials + 4096);
    *part_s = reinterpret_cast<float*>(g_partials + 8192);
    return hipSuccess;
}
}  // namespace mla

int main() {
    // fake device pointers: distinct, 256-byte aligned, never dereferenced
    auto dev = [](uintptr_t i) { return reinterpret_cast<void*>((i + 1) << 12); };
    mla_cache_format f{512, 64, 64, 4, 4, 64, MLA_META_FP16};

    // ---- geometry
    CHECK(mla_lowbit_page_bytes(&f) == 20736);
    mla_cache_format f2 = f;
    f2.c_bits = 2;
    CHECK(mla_lowbit_page_bytes(&f2) == 12544);
    mla_cache_format fp = f;
    fp.meta = MLA_META_PAPER;
    CHECK(mla_lowbit_page_bytes(&fp) == 20480);
    CHECK(mla_bf16_page_bytes(&f) == 73728);
    CHECK(mla_lowbit_page_bytes(nullptr) == -1);
    mla_cache_format bad = f;
    bad.page_size = std::numeric_limits<int32_t>::max();
    CHECK(mla_lowbit_page_bytes(&bad) == -1);
    bad = f;
    bad.group = 0;
    CHECK(mla_lowbit_page_bytes(&bad) == -1);
    bad = f;
    bad.d_c = -512;
    CHECK(mla_bf16_page_bytes(&bad) == -1);

    // ---- planners, including lengths near the int32 limit
    {
        const int32_t lens[4] = {1, 64, 65, 4096};
        int32_t indptr[5] = {};
        CHECK(mla_plan_splits(lens, 4, 64, indptr) == 1 + 1 + 2 + 64);
        CHECK(indptr[0] == 0 && indptr[4] == 68);
        CHECK(mla_plan_splits(lens, 4, 48, indptr) == -MLA_ENOTSUP);
        CHECK(mla_plan_splits(lens, 4, 0, indptr) == -MLA_EINVAL);
        CHECK(mla_plan_splits(nullptr, 4, 64, indptr) == -MLA_EINVAL);
        CHECK(mla_plan_splits(lens, 0, 64, indptr) == 0 && indptr[0] == 0);
        // 40 sequences of 2^31 - 1 keys in 32-key splits: 40 * 2^26 splits overflow int32
        const std::vector<int32_t> big(40, std::numeric_limits<int32_t>::max());
        std::vector<int32_t> ipb(41, 0);
        CHECK(mla_plan_splits(big.data(), 40, 32, ipb.data()) == -MLA_EINVAL);
        CHECK(mla_plan_splits(big.data(), 3, 32, ipb.data()) == 3 * (1 << 26));
        int32_t ip3[4] = {};
        const int32_t zero[1] = {0};
        CHECK(mla_plan_splits(zero, 1, 32, ip3) == -MLA_EINVAL);
        mla_protect_policy pol{4, 128};
        CHECK(mla_plan_splits_protected(lens, 4, 64, &pol, indptr) > 0);
        mla_protect_policy badp{-1, 128};
        CHECK(mla_plan_splits_protected(lens, 4, 64, &badp, indptr) == -MLA_EINVAL);
        mla_protect_policy hugep{std::numeric_limits<int32_t>::max(), std::numeric_limits<int32_t>::max()};
        CHECK(mla_plan_splits_protected(lens, 4, 64, &hugep, indptr) == -MLA_EINVAL);
        CHECK(mla_plan_splits_protected(big.data(), 40, 32, &pol, ipb.data()) == -MLA_EINVAL);
        CHECK(mla_plan_splits_protected(big.data(), 3, 32, &pol, ipb.data()) > 3 * ((1 << 26) - 5));
    }

    // ---- accounting
    {
        mla_protect_policy pol{4, 128};
        CHECK(mla_persistent_cache_bytes(&fp, &pol, 4096) == 64 * (20480 + 8) + 152064);
        CHECK(mla_persistent_cache_bytes(&fp, nullptr, 0) == 0);
        CHECK(mla_persistent_cache_bytes(&fp, &pol, -1) == -1);
        CHECK(mla_persistent_cache_bytes(&fp, &pol, std::numeric_limits<int64_t>::max() / 4) == -1);
        CHECK(mla_persistent_cache_bytes(&fp, &pol, std::numeric_limits<int64_t>::max()) == -1);
        CHECK(mla_persistent_cache_bytes(&fp, &pol, int64_t{1} << 40) == (int64_t{1} << 34) * (20480 + 8) + 152064);
        mla_cache_format fb = f;
        fb.c_bits = 16;
        CHECK(mla_persistent_cache_bytes(&fb, nullptr, std::numeric_limits<int64_t>::max()) == -1);
        CHECK(mla_persistent_cache_bytes(&fb, nullptr, 65) == 2 * 73728);
        CHECK(mla_protect_buffer_bytes(&f, &pol) == 152064);
        CHECK(mla_protect_buffer_bytes(&f, nullptr) == -1);
    }

    // ---- append: validation and dispatch
    {
        const auto* c = static_cast<const uint16_t*>(dev(1));
        const auto* k = static_cast<const uint16_t*>(dev(2));
        const auto* slots = static_cast<const int64_t*>(dev(3));
        void* cache = dev(4);
        CHECK(mla_lowbit_quant_append(&f, c, 512, k, 64, slots, 0, nullptr, 0, nullptr) == MLA_OK);
        CHECK(mla_lowbit_quant_append(&f, c, 512, k, 64, slots, -1, cache, 4, nullptr) == MLA_EINVAL);
        CHECK(mla_lowbit_quant_append(&f, nullptr, 512, k, 64, slots, 8, cache, 4, nullptr) == MLA_EINVAL);
        CHECK(mla_lowbit_quant_append(&f, c, 500, k, 64, slots, 8, cache, 4, nullptr) == MLA_EINVAL);
        CHECK(mla_lowbit_quant_append(&f, c, 520, k, 64, slots, 8,
                                      static_cast<uint8_t*>(cache) + 16, 4, nullptr) == MLA_EINVAL);
        CHECK(mla_lowbit_quant_append(&f, c, 516, k, 64, slots, 8, cache, 4, nullptr) == MLA_ENOTSUP);
        const int before = g_append_calls;
        CHECK(mla_lowbit_quant_append(&f, c, 512, k, 64, slots, 8, cache, 4, nullptr) == MLA_OK);
        CHECK(g_append_calls == before + 1 && g_last_append.n == 8 && g_last_append.num_slots == 4 * 64);
        CHECK(g_last_append.g.page_bytes == 20736 && g_last_append.g.off_cr == 64 * 256);
    }

    // ---- decode: validation, kind and launch selection, split plumbing
    {
        const auto* ql = static_cast<const uint16_t*>(dev(10));
        const auto* qr = static_cast<const uint16_t*>(dev(11));
        const void* cache = dev(12);
        const auto* bt = static_cast<const int32_t*>(dev(13));
        const auto* sl = static_cast<const int32_t*>(dev(14));
        const auto* ip = static_cast<const int32_t*>(dev(15));
        auto* out = static_cast<uint16_t*>(dev(16));
        auto* lse = static_cast<float*>(dev(17));
        auto* pm = static_cast<float*>(dev(18));
        auto* ps = static_cast<float*>(dev(19));
        auto* po = static_cast<uint16_t*>(dev(20));
        CHECK(mla_lowbit_decode_attn(&f, ql, qr, cache, 4, bt, 4, sl, 0, 1, 128, 0.1f, 0, nullptr, 0, nullptr, nullptr,
                                     nullptr, nullptr, nullptr, nullptr) == MLA_OK);
        CHECK(mla_lowbit_decode_attn(&f, ql, qr, cache, 4, bt, 4, sl, 2, 3, 128, 0.1f, 0, nullptr, 0, out, lse,
                                     nullptr, nullptr, nullptr, nullptr) == MLA_EINVAL);
        CHECK(mla_lowbit_decode_attn(&f, ql, qr, cache, 4, bt, 4, sl, 2, 1, 120, 0.1f, 0, nullptr, 0, out, lse,
                                     nullptr, nullptr, nullptr, nullptr) == MLA_EINVAL);
        CHECK(mla_lowbit_decode_attn(&f, ql, qr, cache, 4, bt, 4, sl, 2, 1, 128, NAN, 0, nullptr, 0, out, lse,
                                     nullptr, nullptr, nullptr, nullptr) == MLA_EINVAL);
        CHECK(mla_lowbit_decode_attn(&f, ql, qr, cache, 4, bt, 4, sl, 2, 1, 128, -1.0f, 0, nullptr, 0, out, lse,
                                     nullptr, nullptr, nullptr, nullptr) == MLA_EINVAL);
        CHECK(mla_lowbit_decode_attn(&f, ql, qr, cache, 4, bt, 4, sl, 2, 1, 128, 0.1f, 48, ip, 4, out, lse, pm, ps,
                                     po, nullptr) == MLA_ENOTSUP);
        CHECK(mla_lowbit_decode_attn(&f, ql, qr, cache, 4, bt, 4, sl, 2, 1, 128, 0.1f, 64, ip, 4, out, lse, pm, ps,
                                     nullptr, nullptr) == MLA_EINVAL);
        CHECK(mla_lowbit_decode_attn(&f, ql, qr, cache, 4, bt, 4, sl, 2, 1, 128, 0.1f, 0, nullptr, 0,
                                     out + 1, lse, nullptr, nullptr, nullptr, nullptr) == MLA_ENOTSUP);
        int before = g_decode_calls;
        CHECK(mla_lowbit_decode_attn(&f, ql, qr, cache, 4, bt, 4, sl, 2, 2, 128, 0.1f, 64, ip, 9, out, lse, pm, ps,
                                     po, nullptr) == MLA_OK);
        CHECK(g_decode_calls == before + 1 && !g_last_narrow && g_last_kind == mla::KIND_C4R4);
        CHECK(g_last_decode.num_work == 9 && g_last_decode.split_tokens == 64 && g_last_decode.part_o == po);
        CHECK(std::fabs(g_last_decode.scale_log2 - 0.1f * 1.4426950408889634f) < 1e-7f);
        CHECK(mla_lowbit_decode_attn(&f2, ql, qr, cache, 4, bt, 4, sl, 2, 1, 16, 0.1f, 0, nullptr, 0, out, lse,
                                     nullptr, nullptr, nullptr, nullptr) == MLA_OK);
        CHECK(g_last_narrow && g_last_kind == mla::KIND_C2R4 && g_last_decode.num_work == 2);
        CHECK(mla_lowbit_decode_attn(&fp, ql, qr, cache, 4, bt, 4, sl, 2, 1, 128, 0.1f, 0, nullptr, 0, out, lse,
                                     nullptr, nullptr, nullptr, nullptr) == MLA_OK);
        CHECK(g_last_kind == mla::KIND_C4R4P && g_last_decode.g.paper_meta == 1);
        CHECK(mla_bf16_decode_attn(&f, ql, qr, cache, 4, bt, 4, sl, 2, 1, 128, 0.1f, 0, nullptr, 0, out, lse,
                                   nullptr, nullptr, nullptr, nullptr) == MLA_OK);
        CHECK(g_last_kind == mla::KIND_BF16 && g_last_decode.g.page_bytes == 73728);

        // protected decode
        mla_protect_policy pol{4, 128};
        const void* prot = dev(21);
        const auto* pslot = static_cast<const int32_t*>(dev(22));
        CHECK(mla_lowbit_decode_attn_protected(&f, &pol, ql, qr, cache, 4, bt, 4, sl, 2, 1, 128, 0.1f, prot, 2, pslot,
                                               0, nullptr, 0, out, lse, nullptr, nullptr, nullptr, nullptr) == MLA_OK);
        CHECK(g_last_protected && g_last_decode.sink == 4 && g_last_decode.recent == 128 && g_last_decode.num_prot == 2);
        CHECK(mla_lowbit_decode_attn_protected(&f, &pol, ql, qr, cache, 4, bt, 4, sl, 2, 1, 128, 0.1f, nullptr, 2,
                                               pslot, 0, nullptr, 0, out, lse, nullptr, nullptr, nullptr,
                                               nullptr) == MLA_EINVAL);

        // append-and-decode: the writer inside the decode launch (wide and narrow)
        const auto* c = static_cast<const uint16_t*>(dev(23));
        const auto* k = static_cast<const uint16_t*>(dev(24));
        const auto* slots = static_cast<const int64_t*>(dev(25));
        before = g_append_calls;
        CHECK(mla_lowbit_append_decode_attn(&f, c, 512, k, 64, slots, ql, qr, const_cast<void*>(cache), 4, bt, 4, sl,
                                            2, 1, 128, 0.1f, 0, nullptr, 0, out, lse, nullptr, nullptr, nullptr,
                                            nullptr) == MLA_OK);
        CHECK(g_append_calls == before && g_last_decode.new_c == c && g_last_decode.new_slots == slots);
        CHECK(mla_lowbit_append_decode_attn(&f, c, 512, k, 64, slots, ql, qr, const_cast<void*>(cache), 4, bt, 4, sl,
                                            2, 1, 16, 0.1f, 0, nullptr, 0, out, lse, nullptr, nullptr, nullptr,
                                            nullptr) == MLA_OK);
        CHECK(g_append_calls == before && g_last_narrow && g_last_decode.new_c == c && g_last_decode.new_k == k);
        // the same under protection: one launch, the protection arguments and the new tokens together
        auto* wprot = dev(21);
        for (int heads : {128, 16}) {
            CHECK(mla_lowbit_append_decode_attn_protected(&f, &pol, c, 512, k, 64, slots, ql, qr, const_cast<void*>(cache),
                                                          4, bt, 4, sl, 2, 1, heads, 0.1f, wprot, 2, pslot, 0, nullptr,
                                                          0, out, lse, nullptr, nullptr, nullptr, nullptr) == MLA_OK);
            CHECK(g_append_calls == before && g_last_protected && g_last_narrow == (heads == 16));
            CHECK(g_last_decode.new_c == c && g_last_decode.new_slots == slots && g_last_decode.prot == wprot &&
                  g_last_decode.sink == 4 && g_last_decode.recent == 128 && g_last_decode.num_prot == 2);
        }
        CHECK(mla_lowbit_append_decode_attn_protected(&f, &pol, c, 512, k, 64, slots, ql, qr, const_cast<void*>(cache),
                                                      4, bt, 4, sl, 2, 1, 128, 0.1f, nullptr, 2, pslot, 0, nullptr, 0,
                                                      out, lse, nullptr, nullptr, nullptr, nullptr) == MLA_EINVAL);

        // timing hook: consumed by the next decode dispatch only
        CHECK(mla_time_next_decode_launch(reinterpret_cast<hipEvent_t>(dev(30)), nullptr) == MLA_EINVAL);
        CHECK(mla_time_next_decode_launch(reinterpret_cast<hipEvent_t>(dev(30)),
                                          reinterpret_cast<hipEvent_t>(dev(31))) == MLA_OK);
        CHECK(mla_lowbit_decode_attn(&f, ql, qr, cache, 4, bt, 4, sl, 2, 1, 128, 0.1f, 0, nullptr, 0, out, lse,
                                     nullptr, nullptr, nullptr, nullptr) == MLA_OK);
        CHECK(g_last_events.start == reinterpret_cast<hipEvent_t>(dev(30)));
        CHECK(mla_lowbit_decode_attn(&f, ql, qr, cache, 4, bt, 4, sl, 2, 1, 128, 0.1f, 0, nullptr, 0, out, lse,
                                     nullptr, nullptr, nullptr, nullptr) == MLA_OK);
        CHECK(g_last_events.start == nullptr);

        // combine
        CHECK(mla_splitkv_combine(pm, ps, po, ip, 9, 2, 2, 128, 512, out, lse, nullptr) == MLA_OK);
        CHECK(g_last_combine_splits == 9 && g_last_combine.B == 2 && g_last_combine.H == 128);
        CHECK(mla_splitkv_combine(pm, ps, po, ip, 9, 2, 2, 128, 256, out, lse, nullptr) == MLA_ENOTSUP);
        CHECK(mla_splitkv_combine(pm, ps, nullptr, ip, 9, 2, 2, 128, 512, out, lse, nullptr) == MLA_EINVAL);

        // allocation-free decode: storage limit, then decode into it and combine from it
        CHECK(mla_lowbit_decode_attn_noalloc(&f, ql, qr, cache, 4, bt, 4, sl, 2, 2, 128, 0.1f, 64, ip, 257, out, lse,
                                             nullptr) == MLA_ENOTSUP);
        const int cb = g_combine_calls;
        CHECK(mla_lowbit_decode_attn_noalloc(&f, ql, qr, cache, 4, bt, 4, sl, 2, 2, 128, 0.1f, 64, ip, 9, out, lse,
                                             nullptr) == MLA_OK);
        CHECK(g_combine_calls == cb + 1 && g_last_combine.part_o == g_last_decode.part_o);
        CHECK(reinterpret_cast<const uint8_t*>(g_last_decode.part_o) == g_partials);
    }

    CHECK(std::strcmp(mla_status_str(MLA_ENOTSUP), "MLA_ENOTSUP: shape or alignment not supported") == 0);
    CHECK(mla_status_str(12345) != nullptr);
    CHECK(mla_last_hip_error() == 0);

    if (g_failures != 0) {
        std::fprintf(stderr, "%d checks failed\n", g_failures);
        return 1;
    }
    std::printf("host ABI driver: all checks passed\n");
    return 0;
}
