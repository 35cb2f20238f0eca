// Fused low-bit MLA decode attention for gfx950 (and the BF16-cache variant).
//
// Computes, for every query row r = (query token i, head h) of a sequence,
//   z_t = tau * (q_lat[r] . C_hat[t] + q_rope[r] . K_hat[t])      (Sec. 2.1,
//   out[r] = softmax(z) C_hat,  lse[r] = ln sum_t e^{z_t}          eq. mla_compact)
// straight from the packed paged cache.  Each tile of 32 tokens is gathered
// from its page, unpacked and dequantized (x_hat = scale * (q - zero) with the
// stored fp16 metadata; Appendix C.4) once into LDS, and that single
// reconstructed tile feeds both the score product and the latent aggregation
// (Appendix C.5, "Cache update and tile reuse").  Partials over a key split
// are the (max, sum, weighted sum) of Appendix C.5 "Global attention
// normalization".
//
// Workgroup = 4 waves = 256 threads, one per CU; it owns one (sequence or key
// split, block of 128 query rows); wave w owns rows 32w..32w+31.
//
// Data path per 32-token tile:
//   1. the tile's packed bytes (codes and metadata regions of the page; raw
//      bf16 rows for the BF16 cache) are copied HBM -> LDS by direct-to-LDS
//      loads (global_load_lds_dwordx4), two tiles ahead of use;
//   2. all 256 threads unpack and dequantize them with packed fp16 math into
//      one token-major fp16 tile [32][576] (rows padded by 32 bytes to spread
//      LDS banks); invalid tokens become zeros;
//   3. scores: every wave computes S^T[token][row] = K_tile . Q^T with
//      v_mfma_f32_32x32x16_f16 (M = 32 tokens, N = its 32 rows, K = 576), the
//      rows' queries held in registers as the B operand.  A lane then holds
//      the 16 scores of one row, the other 16 live in lane ^ 32;
//   4. softmax weights p = 2^(x - ref) in fp32, rounded to fp16;
//   5. latent aggregation O^T[channel][row] += V^T . P^T (M = 512 channels in
//      16 tiles, N = 32 rows, K = 32 tokens): the V^T operand is read from the
//      SAME token-major tile with ds_read_b64_tr_b16 (transposing loads), the
//      P^T operand comes straight from the score registers.
//
// The fp16 datapath (instead of bf16) keeps the reconstructed latents and the
// probabilities to 11 significant bits; the result is accumulated in fp32 and
// rounded once to the bf16 output.  Inputs must lie within the fp16 range
// (|q|, |x_hat| < 65504), which also bounds the reference slack below.
//
// Online softmax with a lazy rescale: every row keeps a running reference
// (its maximum so far, log2 units) and the weights p = 2^(x - ref) stay below
// 2^10 (well inside fp16).  Only when a tile's maximum exceeds the reference by
// more than that slack does the wave rescale its rows' accumulators -- rare
// after the first tiles.  The rescale reads and writes the accumulator
// registers in place (the compiler would otherwise stage all 256 of them
// through vector registers at the branch).  The true maximum is tracked
// separately for the split partials.
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace mla {
namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;
typedef const __attribute__((address_space(1))) void gbl_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kRowsPerBlock = 32 * kWaves;
constexpr int kTile = 32;                       // tokens per tile
constexpr int kDc = 512;
constexpr int kDk = 576;                        // d_c + d_r
constexpr int kKSteps = kDk / 16;               // 36 MFMA k-steps for the scores
constexpr int kRowBytes = kDk * 2 + 32;         // fp16 tile row, padded (see below)
constexpr int kTileBytes = kTile * kRowBytes;   // 37888
constexpr float kRefSlack = 10.0f;              // log2 units a weight may exceed the reference
constexpr float kLn2 = 0.693147180559945309f;

// Staging bytes of one tile's raw cache data (regions in page order).
template <int KIND> struct Staging;
template <> struct Staging<KIND_C4R4> {
    static constexpr int cc = 256, rcodes = kTile * cc, meta = rcodes + kTile * 32,
                         rmeta = meta + kTile * 32, bytes = rmeta + kTile * 4;
};
template <> struct Staging<KIND_C2R4> {
    static constexpr int cc = 128, rcodes = kTile * cc, meta = rcodes + kTile * 32,
                         rmeta = meta + kTile * 32, bytes = rmeta + kTile * 4;
};
template <> struct Staging<KIND_BF16> { static constexpr int bytes = kTile * 1152; };

template <int KIND>
constexpr int lds_bytes() { return 2 * kTileBytes + 2 * Staging<KIND>::bytes; }
static_assert(lds_bytes<KIND_BF16>() + 16 <= 160 * 1024, "LDS budget of a gfx950 CU");

// Byte offset of the 16-byte chunk `chunk` (8 channels) of tile row `row`.
// The 32-byte row pad puts 4 consecutive rows reading two neighbouring chunks
// (the transposing reads) into 8 distinct 16-byte bank groups of a 128-byte
// window, and keeps every operand address a per-lane base plus a
// compile-time offset.
__device__ __forceinline__ int chunk_off(int row, int chunk) { return row * kRowBytes + (chunk << 4); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};   // RNE
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
    const f16x2 v = {static_cast<_Float16>(lo), static_cast<_Float16>(hi)}; // v_cvt_pk_f16_f32, RNE
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint32_t bf16x2_to_f16x2(uint32_t w) {
    return pack_f16x2(__uint_as_float(w << 16), __uint_as_float(w & 0xFFFF0000u));
}

__device__ __forceinline__ float swap_halves(float v) { return __shfl_xor(v, 32, 64); }

// acc *= alpha on an accumulator tile held in AGPRs, element by element in
// place.  Used only on the rare rescale path, hundreds of cycles after the
// last matrix instruction that wrote the tile and before the next one reads it.
__device__ __forceinline__ void scale_acc(f32x16& acc, float alpha) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        float t;
        asm volatile("v_accvgpr_read_b32 %1, %0\n\tv_mul_f32 %1, %1, %2\n\tv_accvgpr_write_b32 %0, %1"
                     : "+a"(acc[v]), "=&v"(t)
                     : "v"(alpha));
    }
}

// ---------------------------------------------------------------------------
// 1. HBM -> LDS staging of one tile (direct-to-LDS loads, 16 B per lane).
// Chunk j of the staging area is loaded by lane (j % 64) of wave ((j / 64) % 4)
// in round j / 256, so every wave instruction fills 1 KiB of contiguous LDS.
// The region sizes make every (round, wave) read from one region: the content
// codes fill whole rounds and the three small regions start a round at waves
// 0, 1 and 2.
__device__ __forceinline__ void dma16(const uint8_t* src, uint8_t* lds_wave_base) {
    __builtin_amdgcn_global_load_lds((gbl_void*)src, (lds_void*)lds_wave_base, 16, 0, 0);
}

template <int KIND>
__device__ __forceinline__ void stage_tile(const uint8_t* page, int po, const PageGeom& g, uint8_t* stage,
                                           int wave, int lane) {
    if constexpr (KIND == KIND_BF16) {
        constexpr int rounds = Staging<KIND>::bytes / (kThreads * 16);       // 9
        static_assert(rounds * kThreads * 16 == Staging<KIND>::bytes, "whole rounds");
        const uint8_t* src = page + po * 1152 + (wave * 64 + lane) * 16;
#pragma unroll
        for (int r = 0; r < rounds; ++r)
            dma16(src + r * kThreads * 16, stage + (r * kThreads + wave * 64) * 16);
    } else {
        using S = Staging<KIND>;
        constexpr int code_rounds = S::rcodes / (kThreads * 16);             // 2 (4-bit) or 1 (2-bit)
        static_assert(code_rounds * kThreads * 16 == S::rcodes, "content codes fill whole rounds");
        static_assert(S::meta - S::rcodes == 1024 && S::rmeta - S::meta == 1024, "one wave per small region");
        const uint8_t* src = page + po * S::cc + (wave * 64 + lane) * 16;
#pragma unroll
        for (int r = 0; r < code_rounds; ++r)
            dma16(src + r * kThreads * 16, stage + (r * kThreads + wave * 64) * 16);
        uint8_t* dst = stage + S::rcodes + wave * 1024;
        if (wave == 0) {
            dma16(page + g.off_cr + po * 32 + lane * 16, dst);
        } else if (wave == 1) {
            dma16(page + g.off_mc + po * 32 + lane * 16, dst);
        } else if (wave == 2 && lane < kTile * 4 / 16) {
            dma16(page + g.off_mr + po * 4 + lane * 16, dst);
        }
    }
}

// ---------------------------------------------------------------------------
// 2. Dequantization of a staged tile into the fp16 tile.
//
// Codes become fp16 values 1024 + q (the fp16 with bits 0x6400 | q, exact);
// (1024 + q) - (1024 + zero) = q - zero exactly, and one fp16 multiply by the
// stored scale rounds s * (q - zero) once.  Both in packed fp16 (2 per op).
__device__ __forceinline__ void meta_to_f16(uint32_t meta, f16x2& zz, f16x2& ss) {
    const _Float16 s = __builtin_bit_cast(_Float16, static_cast<uint16_t>(meta & 0xFFFFu));
    const _Float16 z = __builtin_bit_cast(_Float16, static_cast<uint16_t>(meta >> 16));
    const _Float16 zb = z + static_cast<_Float16>(1024.0f);    // exact: z is an integer in [0, 15]
    zz = f16x2{zb, zb};
    ss = f16x2{s, s};
}

// 8 four-bit codes (channel 2j in the low nibble of byte j) -> 4 fp16 pairs.
__device__ __forceinline__ uint4 codes4_to_f16(uint32_t w, f16x2 zz, f16x2 ss) {
    const uint32_t lo = w & 0x0F0F0F0Fu;          // channels 0, 2, 4, 6
    const uint32_t hi = (w >> 4) & 0x0F0F0F0Fu;   // channels 1, 3, 5, 7
    uint32_t o[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        // bytes [lo.b_k, 0, hi.b_k, 0]
        const uint32_t sel = static_cast<uint32_t>(k) | 0x0C000C00u | (static_cast<uint32_t>(4 + k) << 16);
        const uint32_t pair = __builtin_amdgcn_perm(hi, lo, sel) | 0x64006400u;
        o[k] = __builtin_bit_cast(uint32_t, (__builtin_bit_cast(f16x2, pair) - zz) * ss);
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
}

// 8 two-bit codes (channel 4j+k in bits 2k..2k+1 of byte j), low 16 bits of w.
__device__ __forceinline__ uint4 codes2_to_f16(uint32_t w, f16x2 zz, f16x2 ss) {
    uint32_t o[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {          // pair k: channels 2k, 2k+1
        const uint32_t sh = 4 * k;
        const uint32_t pair = ((w >> sh) & 3u) | (((w >> (sh + 2)) & 3u) << 16) | 0x64006400u;
        o[k] = __builtin_bit_cast(uint32_t, (__builtin_bit_cast(f16x2, pair) - zz) * ss);
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
}

__device__ __forceinline__ uint4 bf16x8_to_f16(uint4 v) {
    return make_uint4(bf16x2_to_f16x2(v.x), bf16x2_to_f16x2(v.y), bf16x2_to_f16x2(v.z), bf16x2_to_f16x2(v.w));
}

// Thread t: tile row (t >> 3) and part (t & 7); the part is one content group
// of 64 channels (8 chunks) plus one RoPE chunk of 8 channels.
template <int KIND>
__device__ __forceinline__ void dequant_tile(const uint8_t* stage, uint8_t* tile, int nvalid, int tid) {
    const int row = tid >> 3;
    const int part = tid & 7;
    uint4 w[9];
    if constexpr (KIND == KIND_BF16) {
        const uint4* src = reinterpret_cast<const uint4*>(stage + row * 1152);
#pragma unroll
        for (int j = 0; j < 8; ++j) w[j] = bf16x8_to_f16(src[part * 8 + j]);
        w[8] = bf16x8_to_f16(src[64 + part]);
    } else {
        using S = Staging<KIND>;
        f16x2 zz, ss;
        meta_to_f16(*reinterpret_cast<const uint32_t*>(stage + S::meta + row * 32 + part * 4), zz, ss);
        if constexpr (KIND == KIND_C4R4) {
            const uint4 c0 = *reinterpret_cast<const uint4*>(stage + row * 256 + part * 32);
            const uint4 c1 = *reinterpret_cast<const uint4*>(stage + row * 256 + part * 32 + 16);
            const uint32_t cw[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
#pragma unroll
            for (int j = 0; j < 8; ++j) w[j] = codes4_to_f16(cw[j], zz, ss);
        } else {
            const uint4 c0 = *reinterpret_cast<const uint4*>(stage + row * 128 + part * 16);
            const uint32_t cw[4] = {c0.x, c0.y, c0.z, c0.w};
#pragma unroll
            for (int j = 0; j < 8; ++j) w[j] = codes2_to_f16(cw[j >> 1] >> (16 * (j & 1)), zz, ss);
        }
        f16x2 rz, rs;
        meta_to_f16(*reinterpret_cast<const uint32_t*>(stage + S::rmeta + row * 4), rz, rs);
        w[8] = codes4_to_f16(*reinterpret_cast<const uint32_t*>(stage + S::rcodes + row * 32 + part * 4), rz, rs);
    }
    const bool ok = row < nvalid;
#pragma unroll
    for (int j = 0; j < 9; ++j) {
        const int chunk = j < 8 ? part * 8 + j : 64 + part;
        *reinterpret_cast<uint4*>(tile + chunk_off(row, chunk)) = ok ? w[j] : make_uint4(0u, 0u, 0u, 0u);
    }
}

// ---------------------------------------------------------------------------
template <int KIND>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void decode_kernel(DecodeArgs a) {
    __shared__ __attribute__((aligned(1024))) uint8_t smem[lds_bytes<KIND>()];
    uint8_t* tiles = smem;                              // 2 x kTileBytes
    uint8_t* stages = smem + 2 * kTileBytes;            // 2 x Staging::bytes
    constexpr int kStage = Staging<KIND>::bytes;

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
    const int full_lim = min(L - a.s_q + 1, t_end);    // every valid row sees keys t < full_lim

    // queries as fp16 B operands: k-step kk holds channels 16kk + 8*half .. +8
    f16x8 qf[kKSteps];
    {
        const int64_t qrow = (static_cast<int64_t>(b) * a.s_q + qi) * a.H + h;
        const uint16_t* ql = a.q_lat + qrow * kDc + 8 * half;
        const uint16_t* qr = a.q_rope + qrow * 64 + 8 * half;
#pragma unroll
        for (int kk = 0; kk < kKSteps; ++kk) {
            // rows past the end read row 0 of the sequence; they are never stored
            const uint4 v = *reinterpret_cast<const uint4*>(kk < 32 ? ql + 16 * kk : qr + 16 * (kk - 32));
            qf[kk] = __builtin_bit_cast(f16x8, bf16x8_to_f16(v));
        }
    }

    auto tile_page = [&](int it, int& po) {
        const int t0 = t_begin + it * kTile;
        int pid = a.block_table[static_cast<int64_t>(b) * a.max_pages + t0 / P];
        pid = min(max(pid, 0), static_cast<int>(a.num_pages - 1));
        po = t0 % P;
        return a.cache + static_cast<int64_t>(pid) * a.g.page_bytes;
    };

    // per-lane addressing of the transposing V^T reads: lane (group g, index i)
    // supplies the address of tile row k0 + i/4, channels n0 + 4(i%4) .. +3
    // and receives rows k0 .. k0+3 of channel n0 + i
    const int qk_row = lane & 31;
    const int tr_i = lane & 15;
    const int tr_g = lane >> 4;
    const int tr_kbase = 4 * (tr_g >> 1) + (tr_i >> 2);   // + 16 * ks (+ 8 for the second read)
    const int tr_col = 16 * (tr_g & 1) + 4 * (tr_i & 3);  // + 32 * m

    float m_ref = -INFINITY;    // reference of the exponentials (log2 units)
    float m_true = -INFINITY;   // true running maximum (log2 units)
    float l_run = 0.0f;         // this lane's share of the exponential sum
    f32x16 acc[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) acc[m] = f32x16{};

    {
        // prologue: stage tiles 0 and 1, dequantize tile 0
        int po;
        if (n_tiles > 0) {
            const uint8_t* pg = tile_page(0, po);
            stage_tile<KIND>(pg, po, a.g, stages, wave, lane);
        }
        if (n_tiles > 1) {
            const uint8_t* pg = tile_page(1, po);
            stage_tile<KIND>(pg, po, a.g, stages + kStage, wave, lane);
        }
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (n_tiles > 0) dequant_tile<KIND>(stages, tiles, t_end - t_begin, tid);

        for (int it = 0; it < n_tiles; ++it) {
            __builtin_amdgcn_s_waitcnt(0);   // this thread's staging of tile it+1 has landed
            __syncthreads();                 // tile it is in LDS; staging it+1 complete; tile (it+1)&1 free
            if (it + 2 < n_tiles) {
                const uint8_t* pg = tile_page(it + 2, po);
                stage_tile<KIND>(pg, po, a.g, stages + (it & 1) * kStage, wave, lane);
            }
            const uint8_t* kt = tiles + (it & 1) * kTileBytes;
            const int t0 = t_begin + it * kTile;

            // every wave computes, also one whose rows all lie past the end
            // (its results are never stored): a branch here would force the
            // accumulators through a register-class join.
            // scores S^T[token][row], K = 576 in 36 steps
            // The operand reads run kAhead steps ahead of the matrix
            // instructions; the group barriers pin that order (left alone, the
            // scheduler issues each read right before its use and the chain
            // waits on LDS latency at every step).
            f32x16 s = f32x16{};
            const uint8_t* krow = kt + chunk_off(qk_row, half);
            constexpr int kAhead = 3;
            f16x8 kb[kAhead];
#pragma unroll
            for (int j = 0; j < kAhead; ++j) kb[j] = *reinterpret_cast<const f16x8*>(krow + 32 * j);
            __builtin_amdgcn_sched_group_barrier(0x100, kAhead, 0);             // LDS reads
#pragma unroll
            for (int kk = 0; kk < kKSteps; ++kk) {
                const f16x8 k = kb[kk % kAhead];
                if (kk + kAhead < kKSteps) kb[kk % kAhead] = *reinterpret_cast<const f16x8*>(krow + 32 * (kk + kAhead));
                s = __builtin_amdgcn_mfma_f32_32x32x16_f16(k, qf[kk], s, 0, 0, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);              // one MFMA
                if (kk + kAhead < kKSteps) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
            // rows see every key of the tile except in the last tile of the
            // range or the tile holding the newest key (block-uniform test)
            if (t0 + kTile > full_lim) {
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int t = t0 + 8 * (v >> 2) + 4 * half + (v & 3);
                    s[v] = t < lim ? s[v] : -INFINITY;
                }
            }
            float mr = s[0];
#pragma unroll
            for (int v = 1; v < 16; ++v) mr = fmaxf(mr, s[v]);
            mr = fmaxf(mr, swap_halves(mr));
            const float mt = mr * a.scale_log2;           // scale > 0: max commutes
            m_true = fmaxf(m_true, mt);
            if (m_ref == -INFINITY) m_ref = mt;          // first visible key: nothing accumulated yet
            if (__builtin_amdgcn_ballot_w64(mt > m_ref + kRefSlack) != 0) {
                const float m_new = fmaxf(m_ref, mt);     // finite for every row that needs it
                const float alpha = exp2f(m_ref - m_new); // 1 for the other rows
#pragma unroll
                for (int m = 0; m < 16; ++m) scale_acc(acc[m], alpha);
                l_run *= alpha;
                m_ref = m_new;
            }
            const float nref = m_ref == -INFINITY ? 0.0f : -m_ref;
            uint32_t pw[8];
#pragma unroll
            for (int v = 0; v < 16; v += 2) {
                const float p0 = __builtin_amdgcn_exp2f(fmaf(s[v], a.scale_log2, nref));
                const float p1 = __builtin_amdgcn_exp2f(fmaf(s[v + 1], a.scale_log2, nref));
                l_run += p0 + p1;
                pw[v >> 1] = pack_f16x2(p0, p1);
            }
            const f16x8 pb0 = __builtin_bit_cast(f16x8, make_uint4(pw[0], pw[1], pw[2], pw[3]));
            const f16x8 pb1 = __builtin_bit_cast(f16x8, make_uint4(pw[4], pw[5], pw[6], pw[7]));

            // latent aggregation O^T[channel][row] += V^T . P^T; the V^T operand
            // is read transposed from the token-major tile
            const uint8_t* vbase = kt + chunk_off(tr_kbase, 0) + 2 * tr_col;
            auto vread = [&](int step) __attribute__((always_inline)) {
                const int ks = step >> 4, m = step & 15;
                const uint8_t* p = vbase + (16 * ks) * kRowBytes + 64 * m;
                const i16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p);
                const i16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 8 * kRowBytes));
                return __builtin_bit_cast(f16x8, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
            };
            constexpr int kVAhead = 2;
            f16x8 vb[kVAhead];
#pragma unroll
            for (int j = 0; j < kVAhead; ++j) vb[j] = vread(j);
            __builtin_amdgcn_sched_group_barrier(0x100, 2 * kVAhead, 0);
#pragma unroll
            for (int step = 0; step < 32; ++step) {
                const f16x8 va = vb[step % kVAhead];
                if (step + kVAhead < 32) vb[step % kVAhead] = vread(step + kVAhead);
                const int m = step & 15;
                acc[m] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va, step < 16 ? pb0 : pb1, acc[m], 0, 0, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                if (step + kVAhead < 32) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
            }
            // keep the unpacking of the next tile out of the operand loads of
            // this one: interleaving them overflows the register file
            __builtin_amdgcn_sched_barrier(0);
            if (it + 1 < n_tiles)
                dequant_tile<KIND>(stages + ((it + 1) & 1) * kStage, tiles + ((it + 1) & 1) * kTileBytes,
                                   t_end - t_begin - (it + 1) * kTile, tid);
            __builtin_amdgcn_sched_barrier(0);
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
                *reinterpret_cast<uint2*>(op + c) =
                    make_uint2(pack_bf16x2(acc[m][4 * q4] * inv, acc[m][4 * q4 + 1] * inv),
                               pack_bf16x2(acc[m][4 * q4 + 2] * inv, acc[m][4 * q4 + 3] * inv));
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
