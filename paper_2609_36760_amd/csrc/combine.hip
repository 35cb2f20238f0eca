// Split-KV combine: global softmax normalisation of per-split partials
// (Appendix C.5, "Global attention normalization"):
//   m = max_j m_j,  s = sum_j e^{m_j - m} s_j,  O = (sum_j e^{m_j - m} o_j) / s,
//   lse = m + ln s,
// skipping splits with m_j = -inf (no visible key).  A split's aggregation is
// stored normalized, u_j = o_j / s_j in fp16, so o_j = s_j u_j.
//
// Workgroups of four waves; each lane owns 8 of the 512 latent channels of an
// output row (sequence, query token, head), so a
// split's partial row is one coalesced 1 KiB read (16 bytes per lane).  The
// kernel is bound by the reads of the partials and their latency: a wave
// issues every load of a batch of splits (maximum, sum, latent row) before
// using any and keeps a running maximum across batches.  With few splits per
// sequence each wave combines one row alone; with many (kShare or more on
// average) a workgroup takes one row and its four waves share the row's splits
// (wave w takes j0 + w, j0 + w + 4, ..) and merge their (maximum, sum,
// weighted row) through LDS, so a row of S splits costs ceil(S / 32)
// dependent rounds of loads.  An empty split holds
// zeros and weighs e^{-inf} s = 0.
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace mla {
namespace {

constexpr int kDc = 512;
constexpr int kWaves = 4;         // waves (and rows) per workgroup
static_assert(64 * kWaves == kCombineThreads, "launch shape the host checks");
constexpr int kShare = 16;        // splits per sequence from which the waves share a row
// kBatch: splits whose loads are in flight together (4 when sequences have
// at most 4 splits on average, so that no load re-reads a split, else 8)
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
    return __builtin_bit_cast(uint32_t, v);
}

// One wave's combine state for one row over the splits j0 + first + step k.
struct RowState {
    float mx, s, o[8];
};

template <int kBatch>
__device__ __forceinline__ RowState combine_splits(const CombineArgs& a, int r, int rows_per_seq, int j0, int j1,
                                                   int first, int step, int lane) {
    RowState st{-INFINITY, 0.0f, {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f}};
    for (int jb = j0 + first; jb < j1; jb += step * kBatch) {
        uint4 u[kBatch];
        float mk[kBatch], sk[kBatch];
#pragma unroll
        for (int k = 0; k < kBatch; ++k) {
            const int jk = jb + step * k;
            const int j = min(jk, j1 - 1);
            const int64_t pr = static_cast<int64_t>(j) * rows_per_seq + r;
            u[k] = *reinterpret_cast<const uint4*>(a.part_o + pr * kDc + lane * 8);
            mk[k] = jk < j1 ? a.part_m[pr] : -INFINITY;
            sk[k] = a.part_s[pr];
        }
        float bm = mk[0];
#pragma unroll
        for (int k = 1; k < kBatch; ++k) bm = fmaxf(bm, mk[k]);
        const float nm = fmaxf(st.mx, bm);
        if (nm == -INFINITY) continue;          // no visible key so far
        const float c = expf(st.mx - nm);       // 0 while mx = -inf
        st.s *= c;
#pragma unroll
        for (int q = 0; q < 8; ++q) st.o[q] *= c;
        st.mx = nm;
#pragma unroll
        for (int k = 0; k < kBatch; ++k) {
            const float ws = expf(mk[k] - st.mx) * sk[k];     // an empty split weighs 0
            st.s += ws;
            const uint32_t w4[4] = {u[k].x, u[k].y, u[k].z, u[k].w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const f16x2 h2 = __builtin_bit_cast(f16x2, w4[q]);
                st.o[2 * q] += ws * static_cast<float>(h2[0]);
                st.o[2 * q + 1] += ws * static_cast<float>(h2[1]);
            }
        }
    }
    return st;
}

__device__ __forceinline__ void store_row(const CombineArgs& a, int64_t row, const float O[8], float M, float S,
                                          int lane) {
    const float inv = S > 0.0f ? 1.0f / S : 0.0f;
    *reinterpret_cast<uint4*>(a.out + row * kDc + lane * 8) =
        make_uint4(pack_bf16x2(O[0] * inv, O[1] * inv), pack_bf16x2(O[2] * inv, O[3] * inv),
                   pack_bf16x2(O[4] * inv, O[5] * inv), pack_bf16x2(O[6] * inv, O[7] * inv));
    if (a.lse != nullptr && lane == 0) a.lse[row] = S > 0.0f ? M + logf(S) : -INFINITY;
}

// kShared: one row per workgroup, its splits shared by the four waves (many
// splits per sequence); else four rows per workgroup, one per wave.
template <bool kShared, int kBatch>
__global__ __launch_bounds__(64 * kWaves) void combine_kernel(CombineArgs a) {
    // rows (b * s_q + i) * H + h in 8 contiguous ranges of blocks, range x on
    // XCD x (block id mod 8), the XCD whose decode workgroups wrote most of them
    constexpr int kRows = kShared ? 1 : kWaves;
    const int64_t rows_all = static_cast<int64_t>(a.B) * a.s_q * a.H;
    const int64_t blocks_all = (rows_all + kRows - 1) / kRows;
    const int64_t per_xcd = (blocks_all + 7) / 8;
    const int64_t blk = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
    if (blk >= blocks_all) return;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int rows_per_seq = a.s_q * a.H;
    const int64_t row = blk * kRows + (kShared ? 0 : wave);
    if (!kShared && row >= rows_all) return;
    const int b = static_cast<int>(row / rows_per_seq);
    const int r = static_cast<int>(row % rows_per_seq);
    const int j0 = a.split_indptr[b];
    const int j1 = a.split_indptr[b + 1];

    if constexpr (!kShared) {
        const RowState st = combine_splits<kBatch>(a, r, rows_per_seq, j0, j1, 0, 1, lane);
        store_row(a, row, st.o, st.mx, st.s, lane);
    } else {
        __shared__ float sh_o[kWaves][8][64];
        __shared__ float sh_ms[kWaves][2];
        const RowState st = combine_splits<kBatch>(a, r, rows_per_seq, j0, j1, wave, kWaves, lane);
#pragma unroll
        for (int q = 0; q < 8; ++q) sh_o[wave][q][lane] = st.o[q];
        if (lane == 0) {
            sh_ms[wave][0] = st.mx;
            sh_ms[wave][1] = st.s;
        }
        __syncthreads();
        if (wave != 0) return;
        float M = sh_ms[0][0];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) M = fmaxf(M, sh_ms[w][0]);
        float S = 0.0f;
        float O[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        if (M != -INFINITY) {
#pragma unroll
            for (int w = 0; w < kWaves; ++w) {
                const float c = expf(sh_ms[w][0] - M);      // 0 for a wave with no visible key
                S += c * sh_ms[w][1];
#pragma unroll
                for (int q = 0; q < 8; ++q) O[q] += c * sh_o[w][q][lane];
            }
        }
        store_row(a, row, O, M, S, lane);
    }
}

}  // namespace

hipError_t launch_combine(const CombineArgs& a, int32_t num_splits, hipStream_t stream) {
    const int64_t rows = static_cast<int64_t>(a.B) * a.s_q * a.H;
    if (rows == 0) return hipSuccess;
    if (num_splits >= static_cast<int64_t>(kShare) * a.B) {
        hipLaunchKernelGGL((combine_kernel<true, 8>), dim3(static_cast<unsigned>((rows + 7) / 8 * 8)),
                           dim3(64 * kWaves), 0, stream, a);
    } else {
        const int64_t blocks = (rows + kWaves - 1) / kWaves;
        const dim3 grid(static_cast<unsigned>((blocks + 7) / 8 * 8)), block(64 * kWaves);
        if (num_splits <= 4 * static_cast<int64_t>(a.B))
            hipLaunchKernelGGL((combine_kernel<false, 4>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((combine_kernel<false, 8>), grid, block, 0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace mla
