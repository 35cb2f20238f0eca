// Fused low-bit MLA decode attention for gfx950 (and the BF16-cache variant).
//
// Computes, for every query row r = (query token i, head h) of a sequence,
//   z_t = tau * (q_lat[r] . C_hat[t] + q_rope[r] . K_hat[t])      (Sec. 2.1,
//   out[r] = softmax(z) C_hat,  lse[r] = ln sum_t e^{z_t}          eq. mla_compact)
// straight from the packed paged cache: each tile of 32 tokens is gathered
// from its page, unpacked and dequantized (x_hat = scale * (q - zero), stored
// fp16 metadata; Appendix C.4) once into LDS as bf16, and that single
// reconstructed tile feeds both the score product and the latent aggregation
// (Appendix C.5, "Cache update and tile reuse").  Partials over a key split
// are the (max, sum, weighted sum) of Appendix C.5 "Global attention
// normalization".
//
// Mapping (one workgroup = 4 waves = 256 threads, one per CU):
//   * the workgroup owns one (sequence or key split, block of 128 rows);
//     wave w owns rows 32w..32w+31 of the block;
//   * the wave keeps its 32 query rows (576 channels) in registers as the B
//     operand of v_mfma_f32_32x32x16_bf16 and computes the transposed score
//     tile S^T[token][row] = K_tile . Q^T (M = 32 tokens, N = 32 rows,
//     K = 576), so every lane holds the scores of ONE row: the online
//     softmax needs no cross-lane reduction except one swap with lane ^ 32;
//   * the output is accumulated transposed, O^T[channel][row] += V^T . P^T
//     (M = 512 channels in 16 tiles, N = 32 rows, K = 32 tokens), the
//     probabilities coming straight from the score registers; the rescale
//     of the running output is one per-lane scalar;
//   * the dequantized tile is written to LDS twice: token-major (QK operand,
//     16 contiguous bytes per lane) and channel-major with tokens permuted to
//     match the score register layout (PV operand, 16 contiguous bytes per
//     lane);
//   * two LDS stages: tile i+1 is unpacked into one while tile i is consumed
//     from the other; packed bytes of tile i+2 are already in flight.
//   * no running rescale of the output: every row fixes its exponential
//     reference at the maximum of the first tile it sees and keeps it; the
//     result is exact for any reference (all terms share it).  If a later
//     tile exceeds the reference by more than 2^64 -- far below fp32
//     overflow of the sums -- the row's reference is raised and the whole
//     workgroup restarts the split (a block-uniform decision through LDS).
//     This keeps the 256 accumulator registers out of any branch.
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace mla {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kRowsPerBlock = 32 * kWaves;
constexpr int kTile = 32;                       // tokens per tile
constexpr int kDc = 512;
constexpr int kDk = 576;                        // d_c + d_r
constexpr int kKSteps = kDk / 16;               // 36 MFMA k-steps for the scores
constexpr int kKRow = kDk * 2 + 16;             // bytes per token row, token-major tile (padded)
constexpr int kVRow = kTile * 2 + 16;           // bytes per channel row, channel-major tile (padded)
constexpr int kKTileBytes = kTile * kKRow;      // 37376
constexpr int kVTileBytes = kDc * kVRow;        // 40960
constexpr int kStageBytes = kKTileBytes + kVTileBytes;
constexpr float kRefSlack = 64.0f;              // log2 units a score may exceed the reference
constexpr float kLn2 = 0.693147180559945309f;

static_assert(2 * kStageBytes <= 160 * 1024, "two LDS stages must fit the 160 KiB of a gfx950 CU");

// Natural token index (0..31) of element j (0..7) of token octet o (0..3).
// Octet o holds exactly the tokens that lane group (o & 1) of the score
// accumulator covers in PV k-step (o >> 1), in register order.
__device__ __forceinline__ int octet_token(int o, int j) {
    return 16 * (o >> 1) + 4 * (o & 1) + (j & 3) + 8 * (j >> 2);
}

__device__ __forceinline__ float f16lo(uint32_t w) {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w & 0xffffu)));
}
__device__ __forceinline__ float f16hi(uint32_t w) {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w >> 16)));
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};   // v_cvt_pk_bf16_f32, RNE
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float swap_halves(float v) {
    // exchange with lane ^ 32 (the other half of the wave holds the same row)
    return __shfl_xor(v, 32, 64);
}

// Per-thread registers of one tile's raw (packed or bf16) cache bytes.
template <int KIND> struct Raw;
template <> struct Raw<KIND_C4R4> { uint32_t code[8]; uint32_t meta[8]; uint32_t rcode; uint32_t rmeta; };
template <> struct Raw<KIND_C2R4> { uint32_t code[8]; uint32_t meta[8]; uint32_t rcode; uint32_t rmeta; };
template <> struct Raw<KIND_BF16> { uint4 c[8]; uint4 r; };

struct TileCtx {
    const uint8_t* page;   // page holding the tile
    int po;                // page offset of the tile's first token
    int nvalid;            // tokens of the tile inside the work range
};

template <int KIND>
__device__ __forceinline__ void load_raw(Raw<KIND>& raw, const TileCtx& tc, const PageGeom& g,
                                         int wave, int lane, int tid) {
    if constexpr (KIND == KIND_BF16) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int t = octet_token(wave, j);
            raw.c[j] = *reinterpret_cast<const uint4*>(tc.page + (tc.po + t) * 1152 + lane * 16);
        }
        const int t = tid >> 3;
        raw.r = *reinterpret_cast<const uint4*>(tc.page + (tc.po + t) * 1152 + 1024 + (tid & 7) * 16);
    } else {
        constexpr int cb = (KIND == KIND_C4R4) ? 4 : 2;        // code bytes per 8 channels
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int t = octet_token(wave, j);
            const uint8_t* p = tc.page + (tc.po + t) * g.cc_bytes + lane * cb;
            raw.code[j] = (cb == 4) ? *reinterpret_cast<const uint32_t*>(p)
                                    : static_cast<uint32_t>(*reinterpret_cast<const uint16_t*>(p));
            raw.meta[j] = *reinterpret_cast<const uint32_t*>(tc.page + g.off_mc + (tc.po + t) * 32 + (lane >> 3) * 4);
        }
        const int t = tid >> 3;
        raw.rcode = *reinterpret_cast<const uint32_t*>(tc.page + g.off_cr + (tc.po + t) * 32 + (tid & 7) * 4);
        raw.rmeta = *reinterpret_cast<const uint32_t*>(tc.page + g.off_mr + (tc.po + t) * 4);
    }
}

// Dequantize 8 codes of one group slice: x_hat = scale * (q - zero).
template <int BITS>
__device__ __forceinline__ void dequant8(uint32_t code, uint32_t meta, float v[8]) {
    const float sc = f16lo(meta);
    const float ze = f16hi(meta);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const float q = static_cast<float>((code >> (BITS * i)) & ((1u << BITS) - 1u));
        v[i] = sc * (q - ze);
    }
}

template <int KIND>
__device__ __forceinline__ void store_tile(const Raw<KIND>& raw, uint8_t* stage, int nvalid,
                                           int wave, int lane, int tid) {
    uint8_t* kt = stage;
    uint8_t* vt = stage + kKTileBytes;
    // content: this thread owns channels 8*lane..+8 of token octet `wave`
    uint32_t kw[8][4];      // [token j][channel pair]
    if constexpr (KIND == KIND_BF16) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const bool ok = octet_token(wave, j) < nvalid;
            kw[j][0] = ok ? raw.c[j].x : 0u;
            kw[j][1] = ok ? raw.c[j].y : 0u;
            kw[j][2] = ok ? raw.c[j].z : 0u;
            kw[j][3] = ok ? raw.c[j].w : 0u;
        }
    } else {
        constexpr int BITS = (KIND == KIND_C4R4) ? 4 : 2;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            float v[8];
            dequant8<BITS>(raw.code[j], raw.meta[j], v);
            const bool ok = octet_token(wave, j) < nvalid;
#pragma unroll
            for (int p = 0; p < 4; ++p) kw[j][p] = ok ? pack_bf16x2(v[2 * p], v[2 * p + 1]) : 0u;
        }
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int t = octet_token(wave, j);
        *reinterpret_cast<uint4*>(kt + t * kKRow + lane * 16) = make_uint4(kw[j][0], kw[j][1], kw[j][2], kw[j][3]);
    }
    // channel-major copy: row = channel, 8 tokens of this octet in register order
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int p = i >> 1;
        const int sh = (i & 1) * 16;
        uint32_t w[4];
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const uint32_t a = (kw[2 * jj][p] >> sh) & 0xffffu;
            const uint32_t b = (kw[2 * jj + 1][p] >> sh) & 0xffffu;
            w[jj] = a | (b << 16);
        }
        *reinterpret_cast<uint4*>(vt + (lane * 8 + i) * kVRow + wave * 16) = make_uint4(w[0], w[1], w[2], w[3]);
    }
    // RoPE key: token tid>>3, channels 512 + 8*(tid&7)..+8
    const int t = tid >> 3;
    const bool ok = t < nvalid;
    uint4 r;
    if constexpr (KIND == KIND_BF16) {
        r = ok ? raw.r : make_uint4(0u, 0u, 0u, 0u);
    } else {
        float v[8];
        dequant8<4>(raw.rcode, raw.rmeta, v);
        r = ok ? make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                            pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7]))
               : make_uint4(0u, 0u, 0u, 0u);
    }
    *reinterpret_cast<uint4*>(kt + t * kKRow + (kDc + (tid & 7) * 8) * 2) = r;
}

template <int KIND>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void decode_kernel(DecodeArgs a) {
    __shared__ __attribute__((aligned(16))) uint8_t smem[2 * kStageBytes];
    __shared__ int restart_flag;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int half = lane >> 5;
    const int rows_total = a.s_q * a.H;
    const int RB = (rows_total + kRowsPerBlock - 1) / kRowsPerBlock;

    // Block -> (work item, row block).  Row blocks of one work item read the
    // same tiles, so they are placed on the same XCD (block id = XCD mod 8).
    int w, rb;
    if (RB == 1) {
        w = blockIdx.x;
        rb = 0;
    } else {
        const int slot = blockIdx.x >> 3;
        w = (slot / RB) * 8 + (blockIdx.x & 7);
        rb = slot % RB;
    }
    if (w >= a.num_work) return;

    const int P = a.g.page_size;
    int b, t_begin, t_end;
    if (a.split_tokens == 0) {
        b = w;
        t_begin = 0;
        t_end = a.seq_lens[b];
    } else {
        int lo = 0, hi = a.B;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (a.split_indptr[mid] <= w) lo = mid; else hi = mid - 1;
        }
        b = lo < a.B ? lo : a.B - 1;
        t_begin = (w - a.split_indptr[b]) * a.split_tokens;
        t_end = t_begin + a.split_tokens;
        const int L = a.seq_lens[b];
        if (t_end > L) t_end = L;
    }
    const int L = min(max(a.seq_lens[b], 0), a.max_pages * P);
    if (t_end > L) t_end = L;
    if (t_begin < 0) t_begin = 0;
    const int n_tiles = t_end > t_begin ? (t_end - t_begin + kTile - 1) / kTile : 0;

    // this lane's query row
    const int row = rb * kRowsPerBlock + wave * 32 + (lane & 31);
    const bool row_ok = row < rows_total;
    const int qi = row_ok ? row / a.H : 0;
    const int h = row_ok ? row % a.H : 0;
    const int lim = row_ok ? min(L - a.s_q + qi + 1, t_end) : t_begin;   // keys t < lim are visible

    bf16x8 qf[kKSteps];
    {
        const int64_t qrow = (static_cast<int64_t>(b) * a.s_q + qi) * a.H + h;
        const uint16_t* ql = a.q_lat + qrow * kDc + 8 * half;
        const uint16_t* qr = a.q_rope + qrow * 64 + 8 * half;
#pragma unroll
        for (int kk = 0; kk < kKSteps; ++kk) {
            const uint16_t* p = kk < 32 ? ql + 16 * kk : qr + 16 * (kk - 32);
            qf[kk] = *reinterpret_cast<const bf16x8*>(p);   // rows past the end read row 0; never written
        }
    }

    f32x16 acc[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) acc[m] = f32x16{};
    float m_ref = -INFINITY;    // reference of the exponentials (log2 units)
    float m_true = -INFINITY;   // true running maximum (log2 units)
    float l_run = 0.0f;         // this lane's share of the exponential sum
    if (tid == 0) restart_flag = 0;

    auto tile_ctx = [&](int it) {
        TileCtx tc;
        const int t0 = t_begin + it * kTile;
        int pid = a.block_table[static_cast<int64_t>(b) * a.max_pages + t0 / P];
        pid = min(max(pid, 0), static_cast<int>(a.num_pages - 1));
        tc.page = a.cache + static_cast<int64_t>(pid) * a.g.page_bytes;
        tc.po = t0 % P;
        tc.nvalid = t_end - t0;
        return tc;
    };

    Raw<KIND> raw;
    if (n_tiles > 0) {
        const TileCtx tc = tile_ctx(0);
        load_raw<KIND>(raw, tc, a.g, wave, lane, tid);
        store_tile<KIND>(raw, smem, tc.nvalid, wave, lane, tid);
    }
    if (n_tiles > 1) load_raw<KIND>(raw, tile_ctx(1), a.g, wave, lane, tid);

    for (int it = 0; it < n_tiles; ++it) {
        __syncthreads();
        if (restart_flag != 0) {
            // some row met a score far above its reference: start the split
            // again with the raised references (uniform across the block)
#pragma unroll
            for (int m = 0; m < 16; ++m) acc[m] = f32x16{};
            l_run = 0.0f;
            const TileCtx tc = tile_ctx(0);
            load_raw<KIND>(raw, tc, a.g, wave, lane, tid);
            store_tile<KIND>(raw, smem, tc.nvalid, wave, lane, tid);
            if (n_tiles > 1) load_raw<KIND>(raw, tile_ctx(1), a.g, wave, lane, tid);
            it = 0;
            __syncthreads();
            if (tid == 0) restart_flag = 0;
        }
        const uint8_t* kt = smem + (it & 1) * kStageBytes;
        const uint8_t* vt = kt + kKTileBytes;
        const int t0 = t_begin + it * kTile;
        {
            // every wave computes, also one whose rows all lie past the end
            // (its results are never stored): a branch here would force the
            // accumulators through a register-class join
            // scores S^T[token][row], K = 576 in 36 steps
            f32x16 s0 = f32x16{};
            const uint8_t* krow = kt + (lane & 31) * kKRow + half * 16;
#pragma unroll
            for (int kk = 0; kk < kKSteps; kk += 2) {
                const bf16x8 k0 = *reinterpret_cast<const bf16x8*>(krow + kk * 32);
                const bf16x8 k1 = *reinterpret_cast<const bf16x8*>(krow + kk * 32 + 32);
                s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k0, qf[kk], s0, 0, 0, 0);
                s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k1, qf[kk + 1], s0, 0, 0, 0);
            }
            // online softmax over this lane's 16 tokens (the other 16 of the
            // row live in lane ^ 32)
            float x[16];
            float mt = -INFINITY;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int t = t0 + 8 * (v >> 2) + 4 * half + (v & 3);
                x[v] = t < lim ? s0[v] * a.scale_log2 : -INFINITY;
                mt = fmaxf(mt, x[v]);
            }
            mt = fmaxf(mt, swap_halves(mt));
            m_true = fmaxf(m_true, mt);
            if (m_ref == -INFINITY) m_ref = mt;           // first tile with a visible key
            if (mt > m_ref + kRefSlack) {                 // rare: raise and restart
                m_ref = mt;
                restart_flag = 1;
            }
            const float ref = m_ref == -INFINITY ? 0.0f : m_ref;
            float p[16];
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                p[v] = exp2f(x[v] - ref);
                l_run += p[v];
            }
            bf16x8 pb[2];
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                pb[ks] = bf16x8{static_cast<__bf16>(p[8 * ks + 0]), static_cast<__bf16>(p[8 * ks + 1]),
                                static_cast<__bf16>(p[8 * ks + 2]), static_cast<__bf16>(p[8 * ks + 3]),
                                static_cast<__bf16>(p[8 * ks + 4]), static_cast<__bf16>(p[8 * ks + 5]),
                                static_cast<__bf16>(p[8 * ks + 6]), static_cast<__bf16>(p[8 * ks + 7])};
            }
            // latent aggregation O^T[channel][row] += V^T . P^T
            const uint8_t* vrow = vt + (lane & 31) * kVRow + half * 16;
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
                for (int m = 0; m < 16; ++m) {
                    const bf16x8 v = *reinterpret_cast<const bf16x8*>(vrow + m * 32 * kVRow + ks * 32);
                    acc[m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v, pb[ks], acc[m], 0, 0, 0);
                }
            }
        }
        if (it + 1 < n_tiles) {
            const TileCtx tc = tile_ctx(it + 1);
            store_tile<KIND>(raw, smem + ((it + 1) & 1) * kStageBytes, tc.nvalid, wave, lane, tid);
            if (it + 2 < n_tiles) load_raw<KIND>(raw, tile_ctx(it + 2), a.g, wave, lane, tid);
        }
    }

    if (!row_ok) return;
    const float l_tot = l_run + swap_halves(l_run);
    const int64_t orow = (static_cast<int64_t>(b) * a.s_q + qi) * a.H + h;
    if (a.split_tokens == 0) {
        const float inv = l_tot > 0.0f ? 1.0f / l_tot : 0.0f;
        uint16_t* op = a.out + orow * kDc + 4 * half;
#pragma unroll
        for (int m = 0; m < 16; ++m) {
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                const int c = 32 * m + 8 * q4;
                const uint2 v = make_uint2(pack_bf16x2(acc[m][4 * q4] * inv, acc[m][4 * q4 + 1] * inv),
                                           pack_bf16x2(acc[m][4 * q4 + 2] * inv, acc[m][4 * q4 + 3] * inv));
                *reinterpret_cast<uint2*>(op + c) = v;
            }
        }
        if (a.lse != nullptr && half == 0)
            a.lse[orow] = l_tot > 0.0f ? (m_ref + log2f(l_tot)) * kLn2 : -INFINITY;
    } else {
        const int64_t prow = (static_cast<int64_t>(w) * a.s_q + qi) * a.H + h;
        const float f = m_true == -INFINITY ? 0.0f : exp2f(m_ref - m_true);
        float* op = a.part_o + prow * kDc + 4 * half;
#pragma unroll
        for (int m = 0; m < 16; ++m) {
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                const int c = 32 * m + 8 * q4;
                *reinterpret_cast<float4*>(op + c) = make_float4(acc[m][4 * q4] * f, acc[m][4 * q4 + 1] * f,
                                                                 acc[m][4 * q4 + 2] * f, acc[m][4 * q4 + 3] * f);
            }
        }
        if (half == 0) {
            a.part_m[prow] = m_true * kLn2;
            a.part_s[prow] = l_tot * f;
        }
    }
}

}  // namespace

hipError_t launch_decode(CacheKind kind, const DecodeArgs& a, hipStream_t stream) {
    if (a.num_work == 0) return hipSuccess;
    const int rows = a.s_q * a.H;
    const int RB = (rows + kRowsPerBlock - 1) / kRowsPerBlock;
    const int blocks = RB == 1 ? a.num_work : ((a.num_work + 7) / 8) * 8 * RB;
    const dim3 grid(static_cast<unsigned>(blocks)), block(kThreads);
    switch (kind) {
        case KIND_C4R4: hipLaunchKernelGGL(decode_kernel<KIND_C4R4>, grid, block, 0, stream, a); break;
        case KIND_C2R4: hipLaunchKernelGGL(decode_kernel<KIND_C2R4>, grid, block, 0, stream, a); break;
        case KIND_BF16: hipLaunchKernelGGL(decode_kernel<KIND_BF16>, grid, block, 0, stream, a); break;
    }
    return hipGetLastError();
}

}  // namespace mla
