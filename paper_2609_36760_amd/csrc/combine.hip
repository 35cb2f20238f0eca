// Split-KV combine: global softmax normalisation of per-split partials
// (Appendix C.5, "Global attention normalization"):
//   m = max_j m_j,  s = sum_j e^{m_j - m} s_j,  O = (sum_j e^{m_j - m} o_j) / s,
//   lse = m + ln s,
// skipping splits with m_j = -inf (no visible key).  A split's aggregation is
// stored normalized, u_j = o_j / s_j in fp16, so o_j = s_j u_j.
//
// One workgroup of 128 threads per output row (sequence, query token, head);
// each thread owns 4 of the 512 latent channels, so every split's partial row
// is read as one coalesced 1 KiB sweep.  The kernel is bound by HBM reads of
// the partials.
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace mla {
namespace {

constexpr int kDc = 512;
constexpr int kThreads = kDc / 4;
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
    return __builtin_bit_cast(uint32_t, v);
}

__global__ __launch_bounds__(kThreads) void combine_kernel(CombineArgs a) {
    // rows (b * s_q + i) * H + h in 8 contiguous ranges, range x on XCD x
    // (block id mod 8), the XCD whose decode workgroups wrote most of them
    const int64_t rows_all = static_cast<int64_t>(a.B) * a.s_q * a.H;
    const int64_t per_xcd = (rows_all + 7) / 8;
    const int64_t row = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
    if (row >= rows_all) return;
    const int rows_per_seq = a.s_q * a.H;
    const int b = static_cast<int>(row / rows_per_seq);
    const int r = static_cast<int>(row % rows_per_seq);
    const int j0 = a.split_indptr[b];
    const int j1 = a.split_indptr[b + 1];

    float mx = -INFINITY;
    for (int j = j0; j < j1; ++j) mx = fmaxf(mx, a.part_m[static_cast<int64_t>(j) * rows_per_seq + r]);

    float s = 0.0f;
    float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int j = j0; j < j1; ++j) {
        const int64_t pr = static_cast<int64_t>(j) * rows_per_seq + r;
        const float mj = a.part_m[pr];
        if (mj == -INFINITY) continue;
        const float ws = expf(mj - mx) * a.part_s[pr];
        s += ws;
        const uint2 u = *reinterpret_cast<const uint2*>(a.part_o + pr * kDc + threadIdx.x * 4);
        const f16x2 u0 = __builtin_bit_cast(f16x2, u.x), u1 = __builtin_bit_cast(f16x2, u.y);
        o.x += ws * static_cast<float>(u0[0]);
        o.y += ws * static_cast<float>(u0[1]);
        o.z += ws * static_cast<float>(u1[0]);
        o.w += ws * static_cast<float>(u1[1]);
    }
    const float inv = s > 0.0f ? 1.0f / s : 0.0f;
    *reinterpret_cast<uint2*>(a.out + row * kDc + threadIdx.x * 4) =
        make_uint2(pack_bf16x2(o.x * inv, o.y * inv), pack_bf16x2(o.z * inv, o.w * inv));
    if (a.lse != nullptr && threadIdx.x == 0) a.lse[row] = s > 0.0f ? mx + logf(s) : -INFINITY;
}

}  // namespace

hipError_t launch_combine(const CombineArgs& a, hipStream_t stream) {
    const int64_t rows = static_cast<int64_t>(a.B) * a.s_q * a.H;
    if (rows == 0) return hipSuccess;
    hipLaunchKernelGGL(combine_kernel, dim3(static_cast<unsigned>((rows + 7) / 8 * 8)), dim3(kThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace mla
