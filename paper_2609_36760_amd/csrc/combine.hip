// Split-KV combine: global softmax normalisation of per-split partials
// (Appendix C.5, "Global attention normalization"):
//   m = max_j m_j,  s = sum_j e^{m_j - m} s_j,  O = (sum_j e^{m_j - m} o_j) / s,
//   lse = m + ln s,
// skipping splits with m_j = -inf (no visible key).  A split's aggregation is
// stored normalized, u_j = o_j / s_j in fp16, so o_j = s_j u_j.
//
// One wave per output row (sequence, query token, head), four rows per
// workgroup; each lane owns 8 of the 512 latent channels, so a split's
// partial row is one coalesced 1 KiB read (16 bytes per lane).  The kernel is
// bound by the reads of the partials and their latency: every load of a batch
// of splits (maximum, sum, latent row) is issued before any is used, so a
// row costs two dependent rounds of loads (the split range, then the batch);
// an empty split holds zeros and weighs e^{-inf} s = 0.
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace mla {
namespace {

constexpr int kDc = 512;
constexpr int kRowsPerBlock = 4;
constexpr int kBatch = 8;       // splits whose loads are in flight together
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
    return __builtin_bit_cast(uint32_t, v);
}

__global__ __launch_bounds__(64 * kRowsPerBlock) void combine_kernel(CombineArgs a) {
    // rows (b * s_q + i) * H + h in 8 contiguous ranges, range x on XCD x
    // (block id mod 8), the XCD whose decode workgroups wrote most of them
    const int64_t rows_all = static_cast<int64_t>(a.B) * a.s_q * a.H;
    const int64_t blocks_all = (rows_all + kRowsPerBlock - 1) / kRowsPerBlock;
    const int64_t per_xcd = (blocks_all + 7) / 8;
    const int64_t blk = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
    const int lane = threadIdx.x & 63;
    const int64_t row = blk * kRowsPerBlock + (threadIdx.x >> 6);
    if (blk >= blocks_all || row >= rows_all) return;
    const int rows_per_seq = a.s_q * a.H;
    const int b = static_cast<int>(row / rows_per_seq);
    const int r = static_cast<int>(row % rows_per_seq);
    const int j0 = a.split_indptr[b];
    const int j1 = a.split_indptr[b + 1];

    // Splits in batches of kBatch: all loads of a batch (maxima, sums and the
    // latent rows) are issued together, then the running maximum moves to the
    // batch's and the running sums are rescaled (online, as within a split).
    float mx = -INFINITY, s = 0.0f;
    float o[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int jb = j0; jb < j1; jb += kBatch) {
        uint4 u[kBatch];
        float mk[kBatch], sk[kBatch];
#pragma unroll
        for (int k = 0; k < kBatch; ++k) {
            const int j = min(jb + k, j1 - 1);
            const int64_t pr = static_cast<int64_t>(j) * rows_per_seq + r;
            u[k] = *reinterpret_cast<const uint4*>(a.part_o + pr * kDc + lane * 8);
            mk[k] = jb + k < j1 ? a.part_m[pr] : -INFINITY;
            sk[k] = a.part_s[pr];
        }
        float bm = mk[0];
#pragma unroll
        for (int k = 1; k < kBatch; ++k) bm = fmaxf(bm, mk[k]);
        const float nm = fmaxf(mx, bm);
        if (nm == -INFINITY) continue;          // no visible key so far
        const float c = expf(mx - nm);          // 0 while mx = -inf
        s *= c;
#pragma unroll
        for (int q = 0; q < 8; ++q) o[q] *= c;
        mx = nm;
#pragma unroll
        for (int k = 0; k < kBatch; ++k) {
            const float ws = expf(mk[k] - mx) * sk[k];     // an empty split weighs 0
            s += ws;
            const uint32_t w4[4] = {u[k].x, u[k].y, u[k].z, u[k].w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const f16x2 h2 = __builtin_bit_cast(f16x2, w4[q]);
                o[2 * q] += ws * static_cast<float>(h2[0]);
                o[2 * q + 1] += ws * static_cast<float>(h2[1]);
            }
        }
    }
    const float inv = s > 0.0f ? 1.0f / s : 0.0f;
    *reinterpret_cast<uint4*>(a.out + row * kDc + lane * 8) =
        make_uint4(pack_bf16x2(o[0] * inv, o[1] * inv), pack_bf16x2(o[2] * inv, o[3] * inv),
                   pack_bf16x2(o[4] * inv, o[5] * inv), pack_bf16x2(o[6] * inv, o[7] * inv));
    if (a.lse != nullptr && lane == 0) a.lse[row] = s > 0.0f ? mx + logf(s) : -INFINITY;
}

}  // namespace

hipError_t launch_combine(const CombineArgs& a, hipStream_t stream) {
    const int64_t rows = static_cast<int64_t>(a.B) * a.s_q * a.H;
    if (rows == 0) return hipSuccess;
    const int64_t blocks = (rows + kRowsPerBlock - 1) / kRowsPerBlock;
    hipLaunchKernelGGL(combine_kernel, dim3(static_cast<unsigned>((blocks + 7) / 8 * 8)), dim3(64 * kRowsPerBlock), 0,
                       stream, a);
    return hipGetLastError();
}

}  // namespace mla
