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
// Workgroup = 4 waves = 256 threads, one per CU (one wave per SIMD); it owns
// one (sequence or key split, block of 128 query rows); wave w owns rows
// 32w..32w+31.
//
// Data path per 32-token tile:
//   1. its packed bytes (code and metadata regions of the page) are copied
//      HBM -> LDS by direct-to-LDS loads (global_load_lds_dwordx4) three tiles
//      ahead of use, every wave issuing the same number of loads so that one
//      counted wait covers a tile; the page id is fetched through the scalar
//      cache while the workgroup waits at the step barrier.  Rows past the
//      end of the range re-read the range's last token, so every staged row
//      decodes to finite values;
//   2. all 256 threads unpack and dequantize them with packed fp16 math into a
//      token-major fp16 tile [32][576] (the bank-conflict-free layout of
//      tile_bytes below);
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
// Software pipeline.  With one wave per SIMD no other wave hides a wave's
// latencies, so every step interleaves independent work explicitly:
//   step j:  scores of tile j   ||  dequantization of tile j+1
//            softmax of tile j  ||  latent aggregation of tile j-1 (and the
//                                   staging of tile j+3)
// (the aggregation trails the scores by one tile: three fp16 tile buffers,
// three staging buffers).  Scheduling barriers after every matrix
// instruction pin the interleaving.
//
// The BF16-cache kernel stages raw bf16 rows straight into padded tile
// buffers (four of them; staging distance two tiles) and runs the same steps
// on bf16 matrix instructions, the weights rounded to bf16 (cache values and
// queries are exact in bf16, so the weights are the only rounded operand).
//
// The fp16 datapath of the low-bit kernel keeps the reconstructed latents and
// the probabilities to 11 significant bits; the result is accumulated in fp32
// and rounded once to the bf16 output.  Inputs must lie within the fp16 range
// (|q|, |x_hat| < 65504), which also bounds the reference slack below.
//
// Online softmax with a lazy rescale: every row keeps a running reference
// (its maximum so far, log2 units) and the weights p = 2^(x - ref) stay below
// 2^10 (well inside fp16).  Only when a tile's maximum exceeds the reference by
// more than that slack does the wave move its rows to a new reference -- rare
// after the first tiles.  The tile's weights are then computed on the new
// reference, and the accumulators follow in the next step, just before that
// tile is aggregated (after the aggregation of the previous tile, still on the
// old reference).  The rescale reads and writes the accumulator registers in
// place (the compiler would otherwise stage all 256 of them through vector
// registers at the branch).  The true maximum is tracked separately for the
// split partials.
#include <hip/hip_runtime.h>

#include <cmath>
#include <type_traits>

#include "internal.h"
#include "kernel_common.h"
#include "writer_common.h"

namespace mla {
namespace {

using namespace kc;


constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kRowsPerBlock = 32 * kWaves;
static_assert(kThreads == kDecodeThreads && kRowsPerBlock == kDecodeRowsPerBlock, "launch shape the host checks");
constexpr int kTile = 32;                       // tokens per tile
constexpr int kDc = 512;
constexpr int kDk = 576;                        // d_c + d_r
constexpr int kKSteps = kDk / 16;               // 36 MFMA k-steps for the scores
constexpr float kRefSlack = 10.0f;              // log2 units a weight may exceed the reference
constexpr float kLn2 = 0.693147180559945309f;

// Per cache kind: NT tile buffers, NS staging buffers, staging distance D
// (tiles ahead), direct-to-LDS loads per wave per tile.
template <int KIND> struct Cfg;
template <> struct Cfg<KIND_C4R4> {
    static constexpr bool lowbit = true;
    static constexpr bool pmeta = false;                // fp16 {scale, zero} metadata regions
    static constexpr int cc = 256;                      // content code bytes per token
    static constexpr int code_rounds = 2;               // content codes: 2 x 256 chunks
    static constexpr int rcodes = kTile * cc, meta = rcodes + 1024, rmeta = meta + 1024,
                         spare = rmeta + 128, stage_bytes = spare + 128;
    static constexpr int NT = 3, NS = 3, D = 3, loads = code_rounds + 1;
    static constexpr int SC = 84;                       // tile row stride in 16-byte chunks
    static constexpr bool grouped = true;               // a pad chunk after every 8 content chunks
};
template <> struct Cfg<KIND_C2R4> {
    static constexpr bool lowbit = true;
    static constexpr bool pmeta = false;
    static constexpr int cc = 128;
    static constexpr int code_rounds = 1;
    static constexpr int rcodes = kTile * cc, meta = rcodes + 1024, rmeta = meta + 1024,
                         spare = rmeta + 128, stage_bytes = spare + 128;
    static constexpr int NT = 3, NS = 3, D = 3, loads = code_rounds + 1;
    static constexpr int SC = 84;
    static constexpr bool grouped = true;
};
// The paper's storage: one 32-byte metadata record per token (staged where
// the content metadata goes; the RoPE metadata slot only receives a dummy
// load that keeps the load count uniform).
template <> struct Cfg<KIND_C4R4P> : Cfg<KIND_C4R4> {
    static constexpr bool pmeta = true;
};
template <> struct Cfg<KIND_C2R4P> : Cfg<KIND_C2R4> {
    static constexpr bool pmeta = true;
};
template <> struct Cfg<KIND_BF16> {
    static constexpr bool lowbit = false;
    static constexpr int cc = 0;
    static constexpr int stage_bytes = 0;
    static constexpr int NT = 4, NS = 0, D = 2, loads = 10;   // 2432 chunks: 9 rounds of 256 + 128
    static constexpr int SC = 76;
    static constexpr bool grouped = false;
};

// Tile layout.  Row r (token) starts at 16 * (SC * r + ((r >> 2) & 3)) bytes;
// logical 16-byte chunk c (8 channels) sits at chunk c + c / 8 of the row in
// the grouped layout (low-bit tiles: a pad chunk after each 64-channel group,
// 80 chunks in all) and at chunk c otherwise (72 chunks).  With SC = 84 (or
// 76), the score operand reads (16 rows, one chunk each), the transposing reads
// (4 aligned rows, 4 consecutive chunks each) and the dequantization stores
// (8 consecutive groups of two rows r, r + 2) touch 16 distinct 16-byte bank
// groups per 256-byte access, i.e. no bank conflicts.
template <int KIND>
constexpr int tile_bytes() { return kTile * Cfg<KIND>::SC * 16; }
__host__ __device__ constexpr int row_off(int sc, int r) { return 16 * (sc * r + ((r >> 2) & 3)); }
__host__ __device__ constexpr int phys_chunk(bool grouped, int c) { return grouped ? c + (c >> 3) : c; }
static_assert(row_off(84, 31) + 16 * 80 <= 32 * 84 * 16, "grouped rows fit the tile");
static_assert(row_off(84, 16) - row_off(84, 15) >= 16 * 80, "grouped rows do not overlap");
static_assert(row_off(76, 31) + 16 * 72 <= 32 * 76 * 16, "plain rows fit the tile");
static_assert(row_off(76, 16) - row_off(76, 15) >= 16 * 72, "plain rows do not overlap");

template <int KIND>
constexpr int lds_bytes() { return Cfg<KIND>::NT * tile_bytes<KIND>() + Cfg<KIND>::NS * Cfg<KIND>::stage_bytes; }
constexpr int kLdsMax = 160 * 1024;     // LDS of a gfx950 workgroup
static_assert(lds_bytes<KIND_C4R4>() <= 160 * 1024, "LDS budget of a gfx950 CU");
static_assert(lds_bytes<KIND_C4R4P>() == lds_bytes<KIND_C4R4>(), "same staging for both metadata layouts");
static_assert(lds_bytes<KIND_BF16>() <= 160 * 1024, "LDS budget of a gfx950 CU");

// max / sum of a value and its copy in lane ^ 32 (v_permlane32_swap hands each
// lane the pair {own value, partner's value} in its two results)
// Score products accumulate in vector registers: the 256 accumulation
// registers hold the output tiles, and a score tile kept there would be copied
// out for the softmax (and an output tile copied in) on every step.  Issued as
// inline assembly, so the compiler inserts no hazard waits for these: the
// chain's first product writes the tile without reading it, the following
// ones accumulate back to back (no wait needed between products of one shape),
// and score_ready() supplies the wait before vector instructions read the
// result (12 wait states, what the compiler's hazard model places after a
// 32 x 32 x 16 product whose result a vector instruction reads).
__device__ __forceinline__ void mfma_v(f32x16& c, f16x8 a, f16x8 b, bool first) {
    if (first)
        asm volatile("v_mfma_f32_32x32x16_f16 %0, %1, %2, 0" : "=&v"(c) : "v"(a), "v"(b));
    else
        asm volatile("v_mfma_f32_32x32x16_f16 %0, %1, %2, %0" : "+v"(c) : "v"(a), "v"(b));
}
__device__ __forceinline__ void mfma_v(f32x16& c, bf16x8 a, bf16x8 b, bool first) {
    if (first)
        asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(c) : "v"(a), "v"(b));
    else
        asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(c) : "v"(a), "v"(b));
}
__device__ __forceinline__ void score_ready(f32x16& c) {
    asm volatile("s_nop 7\n\ts_nop 3" : "+v"(c));
}
__device__ __forceinline__ float max_halves(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_halves(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ f32x16 mfma(f16x8 a, f16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// acc *= alpha on an accumulator tile held in AGPRs, element by element in
// place.  Used only on the rare rescale path; the caller first waits out the
// latency of the matrix instructions that last wrote the tiles.
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
// 1. HBM -> LDS staging (direct-to-LDS loads: dma16 in kernel_common.h).
//
// Wait until at most N direct-to-LDS loads of this wave are in flight and all
// of its LDS accesses are done, then synchronize the workgroup.  Also fetches
// a page-table entry through the scalar cache (one cache line holds the ids
// of 16 consecutive pages): its latency hides behind the barrier, and the
// value is complete when the statement ends.
template <int N>
__device__ __forceinline__ int step_barrier(const int32_t* table, int index) {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    int v;
    asm volatile("s_load_dword %0, %1, %2\n\ts_waitcnt vmcnt(%3) lgkmcnt(0)\n\ts_barrier"
                 : "=&s"(v)
                 : "s"(table), "s"(__builtin_amdgcn_readfirstlane(index * 4)), "n"(N)
                 : "memory");
    return v;
}

// A page-table entry fetched through the scalar cache without waiting
// (issue_page_id), and the step's wait and barrier that deliver it
// (wait_barrier names the result, so that no use is placed before the wait).
__device__ __forceinline__ void issue_page_id(const int32_t* table, int index, int& v) {
    asm volatile("s_load_dword %0, %1, %2" : "=&s"(v) : "s"(table), "s"(__builtin_amdgcn_readfirstlane(index * 4)));
}
template <int N>
__device__ __forceinline__ int wait_barrier(int& v) {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%1) lgkmcnt(0)\n\ts_barrier" : "+s"(v) : "n"(N) : "memory");
    return v;
}

// The same wait and barrier without a page-table fetch.
template <int N>
__device__ __forceinline__ void plain_barrier() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" : : "n"(N) : "memory");
}

// Packed tile: the content codes in whole rounds (chunk i of the region by
// lane i % 64 of wave (i / 64) % 4), then one load per wave for the small
// regions: wave 0 the RoPE codes, wave 1 the content metadata (or the paper's
// 32-byte records), wave 2 the RoPE metadata, wave 3 the RoPE metadata again
// into a spare area (every wave issues Cfg::loads loads; under the paper's
// storage wave 2 too loads into the spare area).  Tokens at or past `nvalid` re-read token
// nvalid - 1 (per-token regions; a RoPE metadata chunk holds four tokens and
// is read as it is -- such a token's score is masked and its RoPE channels
// never enter the aggregation).  Load `k` of the Cfg::loads.
template <int KIND>
__device__ __forceinline__ void stage_lowbit(int k, const uint8_t* page, int po, int nvalid, const PageGeom& g,
                                             uint32_t st_lds, int wave, int wave_u, int lane) {
    using C = Cfg<KIND>;
    constexpr int cpt = C::cc / 16;                     // chunks per token
    static_assert(C::code_rounds * kThreads * 16 == C::rcodes, "content codes fill whole rounds");
    if (k < C::code_rounds) {
        const int i = k * kThreads + wave * 64 + lane;
        const int tok = min(i / cpt, nvalid - 1);
        dma16(page, (po + tok) * C::cc + (i % cpt) * 16, st_lds + (k * kThreads + wave_u * 64) * 16);
        return;
    }
    const int tok2 = min(lane >> 1, nvalid - 1);
    int src_off, dst_off;
    if (wave_u == 0) {
        src_off = g.off_cr + (po + tok2) * 32 + (lane & 1) * 16;
        dst_off = C::rcodes;
    } else if (wave_u == 1) {
        src_off = g.off_mc + (po + tok2) * 32 + (lane & 1) * 16;
        dst_off = C::meta;
    } else {
        src_off = g.off_mr + po * 4 + (lane & 7) * 16;
        dst_off = wave_u == 2 && !C::pmeta ? C::rmeta : C::spare;
    }
    if (wave_u < 2 || lane < 8) dma16(page, src_off, st_lds + dst_off);
}

// Raw bf16 rows into a tile of the plain layout (SC = 76): LDS chunk i of the
// tile belongs to row r (the last row starting at or before i) and column
// i - start(r); columns 72.. are padding and receive column 71 again.  Tokens
// at or past `nvalid` re-read token nvalid - 1.  Loads 0..8 cover chunks
// 0..2303 (chunk i by lane i % 64 of wave (i / 64) % 4); load 9 covers
// 2304..2431 with waves 0/2 and 1/3 loading the same chunks (same data to the
// same place), so that all waves issue the same number of loads.  Row tok of
// the tile starts at byte row_start(tok) of `src` (a page, or a protection
// buffer).
template <class RowStart>
__device__ __forceinline__ void stage_bf16(int k, const uint8_t* src, RowStart row_start, int nvalid,
                                           uint32_t tile_lds, int wave, int wave_u, int lane) {
    constexpr int sc = 76;
    const int base = k < 9 ? k * kThreads + wave * 64 : 2304 + 64 * (wave & 1);
    const int i = base + lane;
    int row = static_cast<int>((static_cast<unsigned>(i) * 3450u) >> 18);   // i / 76 for i < 2432
    if (i < row_off(sc, row) / 16) --row;
    const int col = min(i - row_off(sc, row) / 16, 71);
    const int tok = min(row, nvalid - 1);
    const int base_u = k < 9 ? k * kThreads + wave_u * 64 : 2304 + 64 * (wave_u & 1);
    dma16(src, row_start(tok) + col * 16, tile_lds + base_u * 16);
}

// ---------------------------------------------------------------------------
// 2. Dequantization of a staged tile into the fp16 tile (metadata as fp16
// pairs: meta_to_f16 / pmeta_to_f16 in kernel_common.h).
//
// Thread t dequantizes part (t & 7) -- one content group of 64 channels (8
// chunks) plus one RoPE chunk of 8 channels -- of tile row dq_row(t); the
// eight threads of a row and the row two further on share a 16-lane store
// group (conflict-free in the grouped layout).
//
// The 36 fp16 pairs (chunk j, pair p; task 4j + p) go through three stages --
// A extract the pair as 1024 + q (shift, mask-and-or), B subtract the biased
// zero, C scale (and store the chunk after its last pair) -- one stage per
// k-step of the score products, task t in stage A at step t: a step runs
// independent operations of three different tasks, which issue without
// waiting on each other while the matrix pipe works.  Steps 0..37; the staged
// bytes are read before step 0.
__device__ __forceinline__ int dq_row(int tid) {
    const int g16 = tid >> 4;
    return 4 * (g16 >> 1) + (g16 & 1) + 2 * ((tid >> 3) & 1);
}

template <int KIND> struct Dq {
    uint4 c0, c1;                   // content codes of the group (c1: 4-bit only)
    uint32_t meta, rcode, rmeta;    // content {scale, zero}, RoPE codes, RoPE {scale, zero}
                                    // (paper storage: meta = bf16 scale | zero << 16,
                                    // rmeta = fp32 scale bits, rzero)
    uint32_t rzero;
    f16x2 zz, ss, rz, rs;           // metadata as fp16 (zero + 1024, scale)
    f16x2 zo[3], rzo;               // -(1024 / 4^(k+1) + zero) for pairs at bit offset 2(k+1) (RoPE: offset 4)
    uint32_t pr[4];                 // pairs in flight (index task & 3)
    uint32_t o[4];                  // finished pairs of the chunk being stored
};

template <int KIND>
__device__ __forceinline__ void dq_read(Dq<KIND>& d, const uint8_t* st, int tid) {
    using C = Cfg<KIND>;
    const int row = dq_row(tid), part = tid & 7;
    if constexpr (C::cc == 256) {
        d.c0 = *reinterpret_cast<const uint4*>(st + row * 256 + part * 32);
        d.c1 = *reinterpret_cast<const uint4*>(st + row * 256 + part * 32 + 16);
    } else {
        d.c0 = *reinterpret_cast<const uint4*>(st + row * 128 + part * 16);
        d.c1 = make_uint4(0u, 0u, 0u, 0u);
    }
    d.rcode = *reinterpret_cast<const uint32_t*>(st + C::rcodes + row * 32 + part * 4);
    if constexpr (C::pmeta) {
        const uint8_t* rec = st + C::meta + row * 32;
        d.meta = static_cast<uint32_t>(*reinterpret_cast<const uint16_t*>(rec + 2 * part)) |
                 (static_cast<uint32_t>(rec[16 + part]) << 16);
        const uint2 r = *reinterpret_cast<const uint2*>(rec + 24);
        d.rmeta = r.x;
        d.rzero = r.y & 0xFFu;
    } else {
        d.meta = *reinterpret_cast<const uint32_t*>(st + C::meta + row * 32 + part * 4);
        d.rmeta = *reinterpret_cast<const uint32_t*>(st + C::rmeta + row * 4);
        d.rzero = 0;
    }
}

// chunk j holds 4-bit codes (channel 2i in the low nibble of byte i)?
template <int KIND>
__device__ __forceinline__ constexpr bool dq_is4(int j) { return Cfg<KIND>::cc == 256 || j == 8; }

// Code word holding chunk j (8 channels): 4-bit content, one word per chunk;
// 2-bit content, one word per two chunks; chunk 8 is the RoPE chunk (4-bit).
template <int KIND>
__device__ __forceinline__ uint32_t dq_word(const Dq<KIND>& d, int j) {
    if constexpr (Cfg<KIND>::cc == 256) {
        const uint32_t cw[9] = {d.c0.x, d.c0.y, d.c0.z, d.c0.w, d.c1.x, d.c1.y, d.c1.z, d.c1.w, d.rcode};
        return cw[j];
    } else {
        const uint32_t cw[4] = {d.c0.x, d.c0.y, d.c0.z, d.c0.w};
        return j < 8 ? cw[j >> 1] : d.rcode;
    }
}

// Bit offset of pair p of chunk j in its code word: in the code layout a
// channel pair sits at one bit offset of the two 16-bit halves of a word.
template <int KIND>
__device__ __forceinline__ constexpr int dq_shift(int j, int p) {
    return dq_is4<KIND>(j) ? 4 * p : 8 * (j & 1) + 2 * p;
}

// Pair p (channels 2p, 2p+1) of chunk j as the fp16 pair with bits
// 0x6400 | (q << o) = 1024 + 2^o q, o = dq_shift mod 8: the word is shifted
// only by the multiple of 8 (shared by the pairs of a byte), and the code is
// masked in place.  1024 + 2^o q is an integer below 2048, exact in fp16.
template <int KIND>
__device__ __forceinline__ uint32_t dq_pair(const Dq<KIND>& d, int j, int p) {
    const int sh = dq_shift<KIND>(j, p);
    const uint32_t m = (dq_is4<KIND>(j) ? 0x000F000Fu : 0x00030003u) << (sh & 7);
    return and_or(dq_word<KIND>(d, j) >> (sh & ~7), m, 0x64006400u);
}

// Dequantization steps 0 .. kDqSteps - 1 (36 pairs through three stages).
constexpr int kDqSteps = 38;

template <int KIND>
__device__ __forceinline__ void dq_step(Dq<KIND>& d, int s, uint8_t* tile, int tid) {
    if (s == 0) {
        if constexpr (Cfg<KIND>::pmeta) {
            pmeta_to_f16(__uint_as_float(d.meta << 16), d.meta >> 16, d.zz, d.ss);
            pmeta_to_f16(__uint_as_float(d.rmeta), d.rzero, d.rz, d.rs);
        } else {
            meta_to_f16(d.meta, d.zz, d.ss);
            meta_to_f16(d.rmeta, d.rz, d.rs);
        }
        // -(1024 / 2^o + zero) for the offsets o = 2, 4, 6 (from zero + 1024:
        // exact, integers and quarters below 1024)
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            const _Float16 c = static_cast<_Float16>(1024.0f - 1024.0f / static_cast<float>(4 << (2 * k)));
            d.zo[k] = f16x2{c, c} - d.zz;
        }
        d.rzo = f16x2{static_cast<_Float16>(960.0f), static_cast<_Float16>(960.0f)} - d.rz;
    }
    if (s >= 2 && s - 2 < 36) {                 // C: scale; store a finished chunk
        const int t = s - 2, j = t >> 2, p = t & 3;
        d.o[p] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, d.pr[t & 3]) * (j < 8 ? d.ss : d.rs));
        if (p == 3) {
            // content chunk 8 part + j sits at physical chunk 9 part + j of the
            // row, the RoPE chunk 64 + part at 72 + part: one per-thread base
            // each, the chunk index an immediate offset
            const int row = dq_row(tid), part = tid & 7;
            static_assert(phys_chunk(true, 8 * 7 + 5) == 9 * 7 + 5 && phys_chunk(true, 64 + 7) == 72 + 7,
                          "grouped layout");
            const int base = row_off(Cfg<KIND>::SC, row) + 16 * (j < 8 ? 9 * part : 72 + part);
            *reinterpret_cast<uint4*>(tile + base + 16 * (j < 8 ? j : 0)) = make_uint4(d.o[0], d.o[1], d.o[2], d.o[3]);
        }
    }
    if (s >= 1 && s - 1 < 36) {                 // B: q - zero, exact
        const int t = s - 1, j = t >> 2, o = dq_shift<KIND>(j, t & 3) & 7;
        const f16x2 x = __builtin_bit_cast(f16x2, d.pr[t & 3]);
        if (o == 0) {
            // (1024 + q) - (1024 + zero)
            d.pr[t & 3] = __builtin_bit_cast(uint32_t, x - (j < 8 ? d.zz : d.rz));
        } else {
            // (1024 + 2^o q) 2^-o is 1024 / 2^o + q exactly; adding -(1024 / 2^o + zero)
            // leaves q - zero, so the fused multiply-add rounds nothing
            const _Float16 w = static_cast<_Float16>(1.0f / static_cast<float>(1 << o));
            const f16x2 c = j < 8 ? d.zo[o / 2 - 1] : d.rzo;
            d.pr[t & 3] = __builtin_bit_cast(uint32_t, __builtin_elementwise_fma(x, f16x2{w, w}, c));
        }
    }
    if (s < 36) {                               // A: extract pair p of chunk j
        const int t = s;
        d.pr[t & 3] = dq_pair<KIND>(d, t >> 2, t & 3);
    }
}

template <int KIND>
__device__ __forceinline__ void dequant_tile(const uint8_t* st, uint8_t* tile, int tid) {
    Dq<KIND> d;
    dq_read<KIND>(d, st, tid);
#pragma unroll
    for (int s = 0; s < kDqSteps; ++s) dq_step<KIND>(d, s, tile, tid);
}

// ---------------------------------------------------------------------------
// In-launch append (the writer of mla_lowbit_quant_append / mla_bf16_append
// for the step's new tokens, run by the decode workgroups that read them).
// Token (b, i) sits at position L - s_q + i; the workgroup whose key range
// holds that position writes it (72 threads per token: 8 per group of 64
// channels, 9 groups; BF16: 72 16-byte pieces of the row) before its tile is
// staged.  A tile is read only by the work item that owns it, so no other
// workgroup waits for the write: every row block of a work item writes the
// same bytes itself.  The stores are older than every staging load of the
// work item, so the counted wait at the barrier before a tile's staging covers
// them; a tile staged in the prologue waits for them explicitly first.
template <int KIND>
__device__ __forceinline__ void append_in_launch(const DecodeArgs& a, int b, int L, int t_begin, int t_end,
                                                 int tid) {
    using C = Cfg<KIND>;
    constexpr int kDpro = C::D;                 // tiles staged in the prologue
    bool early = false;
    for (int i = 0; i < a.s_q; ++i) {
        const int pos = L - a.s_q + i;
        if (pos >= t_begin && pos < t_end && (pos - t_begin) / kTile < kDpro) early = true;
    }
    const int i = tid / 72, r = tid % 72;
    const int pos = L - a.s_q + i;
    if (i < a.s_q && pos >= 0 && pos >= t_begin && pos < t_end) {
        const int64_t tok = static_cast<int64_t>(b) * a.s_q + i;
        const int64_t slot = a.new_slots[tok];
        const int64_t num_slots = a.num_pages * a.g.page_size;
        if (slot >= 0 && slot < num_slots) {
            uint8_t* base = const_cast<uint8_t*>(a.cache) + slot / a.g.page_size * a.g.page_bytes;
            const int64_t off = slot % a.g.page_size;
            const bool rope = r >= 64;
            const uint16_t* src = rope ? a.new_k + tok * a.new_k_stride + (r - 64) * 8
                                       : a.new_c + tok * a.new_c_stride + r * 8;
            const uint4 raw = *reinterpret_cast<const uint4*>(src);
            if constexpr (C::lowbit)
                wc::quantize_store<C::cc == 256 ? 4 : 2, C::pmeta>(raw, rope, r >> 3, r & 7, base, off, a.g);
            else
                *reinterpret_cast<uint4*>(base + off * 1152 + r * 16) = raw;
        }
    }
    if (early) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
    }
}

// The same under BF16 protection: the key list of a work item (packed tiles,
// then the protected rows in position order; see below) decides which work
// item reads a new token, and that work item writes it: the packed copy, as
// the plain writer does for every token, and for a token that is protected
// after the step (position p < sink, or p >= L - recent) its bf16 row in the
// sequence's protection buffer, row p or sink + (p - sink) mod recent -- the
// ring row of the token leaving the window, which this launch reads from its
// packed copy.  A protection buffer index outside [0, num_prot) skips the row
// (as the protected writer does; the decode clamps it).  When a written token
// lies in the first tiles the work item stages, the stores land first.
template <int KIND>
__device__ __forceinline__ void append_in_launch_protected(const DecodeArgs& a, int b, int L, int u0, int u1,
                                                           int n_pk, int pk0, int tid) {
    using C = Cfg<KIND>;
    constexpr int kDpro = C::D > Cfg<KIND_BF16>::D ? C::D : Cfg<KIND_BF16>::D;
    const int sink = a.sink, recent = a.recent;
    const int nsink = min(sink, L), r0 = max(sink, L - recent);
    auto is_prot = [&](int p) { return p < sink || p >= L - recent; };
    // list tile of position p: a packed position by its tile (from the tile
    // holding token `sink`), a protected one by its index among the protected rows
    auto list_tile = [&](int p) {
        return is_prot(p) ? n_pk + (min(p, nsink) + max(0, p - r0)) / kTile : p / kTile - pk0;
    };
    bool early = false;
    for (int i = 0; i < a.s_q; ++i) {
        const int pos = L - a.s_q + i;
        const int u = list_tile(pos);
        if (pos >= 0 && u >= u0 && u < u1 && u - u0 < kDpro) early = true;
    }
    const int i = tid / 72, r = tid % 72;
    const int pos = L - a.s_q + i;
    if (i < a.s_q && pos >= 0 && list_tile(pos) >= u0 && list_tile(pos) < u1) {
        const int64_t tok = static_cast<int64_t>(b) * a.s_q + i;
        const int64_t slot = a.new_slots[tok];
        const int64_t num_slots = a.num_pages * a.g.page_size;
        if (slot >= 0 && slot < num_slots) {
            uint8_t* base = const_cast<uint8_t*>(a.cache) + slot / a.g.page_size * a.g.page_bytes;
            const int64_t off = slot % a.g.page_size;
            const bool rope = r >= 64;
            const uint16_t* src = rope ? a.new_k + tok * a.new_k_stride + (r - 64) * 8
                                       : a.new_c + tok * a.new_c_stride + r * 8;
            const uint4 raw = *reinterpret_cast<const uint4*>(src);
            wc::quantize_store<C::cc == 256 ? 4 : 2, C::pmeta>(raw, rope, r >> 3, r & 7, base, off, a.g);
            const int64_t ps = a.prot_slot[b];
            if (is_prot(pos) && ps >= 0 && ps < a.num_prot) {
                const int prow = pos < sink ? pos : sink + (pos - sink) % recent;
                // [c_kv | k_rope] row: piece r at byte 16 r (the RoPE key from byte 1024)
                uint8_t* dst = const_cast<uint8_t*>(a.prot) + (ps * (sink + recent) + prow) * 1152 + 16 * r;
                *reinterpret_cast<uint4*>(dst) = raw;
            }
        }
    }
    if (early) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// 3. The kernel.
//
// A work item is a sequence (unsplit launch) or one key split of it.  Under
// BF16 protection (kProt) the keys of a sequence of length L form a list of
// 32-token tiles: the packed tiles first (tokens sink .. L-recent-1, counted
// from the tile that holds token `sink`; its tokens below `sink` are masked),
// then the protected tiles, raw bf16 rows of the sequence's protection buffer
// in position order (the sink rows, then the recent window out of the ring).
// A work item takes a contiguous part of that list and runs it in at most two
// phases that carry one online-softmax state -- the low-bit pipeline over its
// packed tiles, then the BF16 pipeline over its protected tiles -- so every
// visible token enters one softmax in exactly one representation
// (Appendix C.5, "BF16 protection and cache lifecycle", "Global attention
// normalization").
template <int KIND, bool kProt>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void decode_kernel(DecodeArgs a) {
    // Low-bit kinds take the whole 160 KiB: the staging slots sit at the top,
    // so that the tile slots and the spare bytes below them form one region of
    // at least 128 KiB, which holds the workgroup's query rows in the prologue.
    constexpr int kLds = Cfg<KIND>::lowbit ? kLdsMax
                         : kProt && lds_bytes<KIND_BF16>() > lds_bytes<KIND>() ? lds_bytes<KIND_BF16>()
                                                                                : lds_bytes<KIND>();
    static_assert(lds_bytes<KIND>() <= kLds && lds_bytes<KIND_BF16>() <= kLdsMax, "LDS budget");
    __shared__ __attribute__((aligned(1024))) uint8_t smem[kLds];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int half = lane >> 5;
    const int rows_total = a.s_q * a.H;
    const int RB = (rows_total + kRowsPerBlock - 1) / kRowsPerBlock;

    // Block -> (work item, row block).  Workgroups are dispatched to the 8
    // XCDs round-robin (XCD = block id mod 8); each XCD gets a contiguous range
    // of work items -- the key splits of whole sequences, which share their
    // queries through that XCD's L2 -- and all row blocks of its work items
    // (which read the same tiles).
    const int per_xcd = (a.num_work + 7) / 8;
    const int slot = blockIdx.x >> 3;
    const int w = (blockIdx.x & 7) * per_xcd + slot / RB;
    const int rb = slot % RB;
    if (w >= a.num_work) return;

    const int P = a.g.page_size;
    int b, split = 0, Lraw;
    if (a.split_tokens == 0) {
        b = w;
        Lraw = a.seq_lens[b];
    } else {
        // The sequence of work item w is the last b with split_indptr[b] <= w
        // (the index is non-decreasing from 0): count those entries 64 at a
        // time, one lane per entry, loading the lengths alongside, so that the
        // search costs one round of loads instead of a chain of dependent ones.
        int cnt = 0, start = 0;
        Lraw = 0;
        for (int base = 0; base <= a.B; base += 64) {
            const int idx = base + lane;
            const int ip = idx <= a.B ? a.split_indptr[idx] : 0x7FFFFFFF;
            const int sl = idx < a.B ? a.seq_lens[idx] : 0;
            const int c = __builtin_popcountll(__builtin_amdgcn_ballot_w64(ip <= w));
            const int last = cnt + c - 1 - base;     // lane of the last such entry in this chunk
            if (c > 0 && last >= 0 && last < 64) {
                start = __builtin_amdgcn_readlane(ip, last);
                Lraw = __builtin_amdgcn_readlane(sl, last);
            }
            cnt += c;
        }
        b = min(cnt - 1, a.B - 1);
        split = w - start;
    }
    const int L = min(max(Lraw, 0), a.max_pages * P);
    const int32_t* bt = a.block_table + static_cast<int64_t>(b) * a.max_pages;

    // this lane's query row
    const int row = rb * kRowsPerBlock + wave * 32 + (lane & 31);
    const bool row_ok = row < rows_total;
    const int qi = row_ok ? row / a.H : 0;
    const int h = row_ok ? row % a.H : 0;

    float m_ref = -INFINITY;    // reference of the exponentials (log2 units)
    float m_true = -INFINITY;   // true running maximum (log2 units)
    float l_run = 0.0f;         // this lane's share of the exponential sum
    f32x16 acc[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) acc[m] = f32x16{};

    // the sequence's protection buffer (kProt): base, rows, sink rows in use
    // and the ring index of the first window position past the sink
    const uint8_t* ring_base = nullptr;
    int ring_rows = 1, ring_nsink = 0, ring_q0 = 0;

    // One phase over keys [t_begin, t_end) in one representation: PK is the
    // cache kind whose pipeline runs; kRing reads bf16 rows of the protection
    // buffer, t then counting protected positions in order.  This lane's row
    // sees keys t_lo <= t < lim; every valid row sees t < full_lim.
    auto run = [&](auto kind_c, auto ring_c, const int t_begin, const int t_end, const int t_lo, const int lim,
                   const int full_lim) __attribute__((always_inline)) {
        constexpr int PK = decltype(kind_c)::value;
        constexpr bool kRing = decltype(ring_c)::value;
        using C = Cfg<PK>;
        using OpT = std::conditional_t<C::lowbit, f16x8, bf16x8>;
        constexpr int kDqKind = C::lowbit ? PK : KIND_C4R4;     // unused by the BF16 pipeline
        constexpr int kTileBytes = tile_bytes<PK>();
        uint8_t* tiles = smem;                              // NT x kTileBytes
        uint8_t* stages = smem + kLds - C::NS * C::stage_bytes;   // NS x stage_bytes at the top (low-bit only)
        static_assert(!C::lowbit || C::NT * kTileBytes <= kLds - C::NS * C::stage_bytes, "tiles below the stages");
        const int n_tiles = t_end > t_begin ? (t_end - t_begin + kTile - 1) / kTile : 0;
        (void)t_lo;

        // Staging.  Step it stages tile it + D -- clamped to the last tile,
        // whose bytes then land once more in a free slot -- so that every step
        // issues Cfg::loads loads.  Buffer slots rotate with the step: tofs[q]
        // is the byte offset of the tile slot of tile it + q (q < NT), sofs[q]
        // that of the staging slot of tile it + q (low-bit, q < NS); both move
        // on by one slot at the end of a step, so the loop does no divisions.
        const int wave_u = __builtin_amdgcn_readfirstlane(wave);
        int tofs[C::NT], sofs[C::NS > 0 ? C::NS : 1];
#pragma unroll
        for (int q = 0; q < C::NT; ++q) tofs[q] = q * kTileBytes;
#pragma unroll
        for (int q = 0; q < (C::NS > 0 ? C::NS : 1); ++q) sofs[q] = q * C::stage_bytes;
        const uint32_t tiles_lds = lds_addr(tiles), stages_lds = lds_addr(stages);

        // Per-lane parts of the staging addresses, fixed for the whole run.
        // Packed: content chunk i of load k < code_rounds (i = 256 k + 64 wave +
        // lane) is chunk i % cpt of token i / cpt of the tile; a small region
        // (RoPE codes, metadata) is read 16 bytes per lane from its start.  BF16
        // rows: row and column of the lane's chunk, two loads per register.
        // Tokens at or past the range's end re-read its last token (nvalid - 1),
        // so the address is one clamp and one shift-add per load.
        constexpr int cpt = C::lowbit ? C::cc / 16 : 1;           // content chunks per token
        constexpr int kBfPairs = C::lowbit ? 1 : (C::loads + 1) / 2;
        uint32_t c_tok = 0, c_col = 0, s_tok = 0, s_col = 0;
        uint32_t bf_rc[kBfPairs];
        int s_reg = 0, s_shift = 0, dst_small = 0;
        if constexpr (C::lowbit) {
            c_tok = static_cast<uint32_t>(wave * 64 + lane) / cpt;
            c_col = (static_cast<uint32_t>(wave * 64 + lane) % cpt) * 16u;
            s_tok = wave_u < 2 ? static_cast<uint32_t>(lane >> 1) : 0u;
            s_col = static_cast<uint32_t>(wave_u < 2 ? (lane & 1) : (lane & 7)) * 16u;
            s_reg = wave_u == 0 ? a.g.off_cr : wave_u == 1 ? a.g.off_mc : a.g.off_mr;
            s_shift = wave_u < 2 ? 5 : 2;
            dst_small = wave_u == 0 ? C::rcodes : wave_u == 1 ? C::meta : (wave_u == 2 && !C::pmeta ? C::rmeta : C::spare);
        } else {
#pragma unroll
            for (int k = 0; k < kBfPairs; ++k) bf_rc[k] = 0;
#pragma unroll
            for (int k = 0; k < C::loads; ++k) {
                const int i = (k < 9 ? k * kThreads + wave * 64 : 2304 + 64 * (wave & 1)) + lane;
                int row = static_cast<int>((static_cast<unsigned>(i) * 3450u) >> 18);   // i / 76 for i < 2432
                if (i < row_off(76, row) / 16) --row;
                const int col = min(i - row_off(76, row) / 16, 71);
                bf_rc[k >> 1] |= static_cast<uint32_t>(row | (col << 5)) << (16 * (k & 1));
            }
        }
        const bool small_lane = wave_u < 2 || lane < 8;

        // Load k of the tile starting at token t0 (offset po in page pid), into
        // the slot at LDS address slot_lds.
        auto issue = [&](int k, int pid, int t0, int po, uint32_t slot_lds) __attribute__((always_inline)) {
            const int nvalid = min(t_end - t0, kTile);
            if constexpr (kRing) {
                // protected position order: the sink rows, then the window from the ring
                auto row_start = [&](int tok) {
                    const int v = t0 + tok;
                    const int x = ring_q0 + (v - ring_nsink);       // < 2 * recent
                    const int r = v < ring_nsink ? v : a.sink + (x >= a.recent ? x - a.recent : x);
                    return min(r, ring_rows - 1) * 1152;
                };
                stage_bf16(k, ring_base, row_start, nvalid, slot_lds, wave, wave_u, lane);
            } else {
                pid = min(max(pid, 0), static_cast<int>(a.num_pages - 1));
                // page_bytes < 2^31: one 32 x 32 -> 64-bit product, unsigned offsets
                const uint8_t* page = a.cache + static_cast<uint64_t>(static_cast<uint32_t>(pid)) *
                                                    static_cast<uint32_t>(a.g.page_bytes);
                const uint32_t upo = static_cast<uint32_t>(po);
                const uint32_t nv1 = static_cast<uint32_t>(nvalid - 1);
                if constexpr (C::lowbit) {
                    if (k < C::code_rounds) {
                        const uint32_t tok = min(c_tok + static_cast<uint32_t>(k * (kThreads / cpt)), nv1);
                        dma16_m0(page + upo * C::cc, tok * C::cc + c_col, slot_lds + (k * kThreads + wave_u * 64) * 16);
                    } else if (small_lane) {
                        dma16_m0(page + (static_cast<uint32_t>(s_reg) + (upo << s_shift)), (min(s_tok, nv1) << 5) + s_col,
                                 slot_lds + dst_small);
                    }
                } else {
                    const uint32_t rc = (bf_rc[k >> 1] >> (16 * (k & 1))) & 0xFFFFu;
                    const int base_u = k < 9 ? k * kThreads + wave_u * 64 : 2304 + 64 * (wave_u & 1);
                    dma16_m0(page + upo * 1152u, min(rc & 31u, nv1) * 1152u + (rc >> 5) * 16u, slot_lds + base_u * 16);
                }
            }
        };
        auto stage_slot = [&](int q) { return C::lowbit ? stages_lds + sofs[q] : tiles_lds + tofs[q]; };
        // prologue: the first D tiles' staging, the queries' loads and their
        // conversion (rows past the end read row 0 of the sequence; they are
        // never stored)
        static_assert(C::D <= 3, "prologue page ids");
        const int64_t qrow = (static_cast<int64_t>(b) * a.s_q + qi) * a.H + h;
        uint4 rawq[kKSteps];
        // The wave's 32 content rows (1 KiB each) are read whole, one
        // direct-to-LDS load per row, into LDS that the prologue's staging
        // leaves free: low-bit, the region below the staging slots (free until
        // tile 0 is dequantized), all rows at once; BF16, the tile slots past
        // the D being staged, 16 rows per round, in two rounds.  Lane l fetches
        // chunk l ^ (row & 15), so that chunk c of row j sits at slot
        // c ^ (j & 15) and the operand reads (32 rows, one chunk each) spread
        // over all banks.  Read straight from memory, the operands take 32
        // rows x 32 bytes per load, four loads per cache line.
        constexpr int kQRounds = C::lowbit ? 1 : 2;
        constexpr int kQRows = 32 / kQRounds;                  // rows per wave and round
        constexpr int kQOff = C::lowbit ? 0 : C::D * kTileBytes;
        static_assert(kQOff + kWaves * kQRows * kDc * 2 <= (C::lowbit ? kLds - C::NS * C::stage_bytes : kLds),
                      "query rows fit the free LDS");
        const uint8_t* qseq = reinterpret_cast<const uint8_t*>(a.q_lat) +
                              static_cast<int64_t>(b) * rows_total * (kDc * 2);
        const int qr0 = rb * kRowsPerBlock + wave_u * 32;
        const uint32_t qdst = lds_addr(smem) + kQOff + static_cast<uint32_t>(wave_u * kQRows) * (kDc * 2);
        auto q_round = [&](int r) __attribute__((always_inline)) {
#pragma unroll
            for (int j = 0; j < kQRows; ++j) {
                const int jr = r * kQRows + j;
                const uint32_t rr = qr0 + jr < rows_total ? static_cast<uint32_t>(qr0 + jr) : 0u;
                dma16_m0(qseq, rr * (kDc * 2) + 16u * static_cast<uint32_t>(lane ^ (jr & 15)),
                         qdst + static_cast<uint32_t>(j) * (kDc * 2));
            }
        };
        const uint8_t* qrow_lds = smem + kQOff + (wave * kQRows + (lane & 31) % kQRows) * (kDc * 2);
        auto q_read = [&](int r) __attribute__((always_inline)) {
            if ((lane & 31) / kQRows == r) {
#pragma unroll
                for (int kk = 0; kk < 32; ++kk)
                    rawq[kk] = *reinterpret_cast<const uint4*>(qrow_lds + 16 * ((2 * kk + half) ^ (lane & 15)));
            }
        };
        // Order: the page ids of the first D tiles (one scalar round trip),
        // the tiles' staging loads (the HBM latency that bounds the prologue),
        // then the query rows, which every workgroup fetches at the same time
        // (128 KiB each, mostly from L2) and which would otherwise hold the
        // staging loads behind them.
        int pids[3] = {0, 0, 0};
        if constexpr (!kRing) {
            auto pidx = [&](int j) { return (t_begin + (j < n_tiles ? j : 0) * kTile) / P; };
            issue_page_ids3(bt, pidx(0), pidx(1), pidx(2), pids[0], pids[1], pids[2]);
        }
        {
            const uint16_t* qr = a.q_rope + qrow * 64 + 8 * half;
#pragma unroll
            for (int kk = 32; kk < kKSteps; ++kk) rawq[kk] = *reinterpret_cast<const uint4*>(qr + 16 * (kk - 32));
        }
        if constexpr (!kRing) wait_page_ids3(pids[0], pids[1], pids[2]);
#pragma unroll
        for (int j = 0; j < C::D; ++j) {
            if (j < n_tiles) {
                const int t0 = t_begin + j * kTile;
#pragma unroll
                for (int k = 0; k < C::loads; ++k) issue(k, pids[j], t0, t0 % P, stage_slot(j));
            }
        }
        q_round(0);
        // the query rows are the youngest loads: every staged tile lands first
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        q_read(0);
        if constexpr (kQRounds == 2) {
            // the second round overwrites the first's rows once they are read
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            q_round(1);
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            q_read(1);
        }

        // queries as B operands: k-step kk holds channels 16kk + 8*half .. +8
        OpT qf[kKSteps];
        {
#pragma unroll
            for (int kk = 0; kk < kKSteps; ++kk) {
                const uint4 v = rawq[kk];
                if constexpr (C::lowbit)
                    qf[kk] = __builtin_bit_cast(f16x8, make_uint4(bf16x2_to_f16x2(v.x), bf16x2_to_f16x2(v.y),
                                                                  bf16x2_to_f16x2(v.z), bf16x2_to_f16x2(v.w)));
                else
                    qf[kk] = __builtin_bit_cast(bf16x8, v);
            }
        }

        int cur_t0 = t_begin + min(C::D, n_tiles - 1) * kTile;     // tile staged by the current step
        int cur_page = cur_t0 / P;
        int cur_po = cur_t0 - cur_page * P;

        // per-lane addressing of the transposing V^T reads: lane (group g, index i)
        // supplies the address of tile row k0 + i/4, channels n0 + 4(i%4) .. +3
        // and receives rows k0 .. k0+3 of channel n0 + i
        const int qk_row = lane & 31;
        const int tr_i = lane & 15;
        const int tr_g = lane >> 4;
        const int tr_kbase = 4 * (tr_g >> 1) + (tr_i >> 2);   // + 16 * ks (+ 8 for the second read)
        const int tr_col = 16 * (tr_g & 1) + 4 * (tr_i & 3);  // + 32 * m

        OpT pb_prev[2] = {OpT{}, OpT{}};   // weights of the previous tile (P^T operands)
        // BF16 pipeline over protected rows: the weights' residuals w - bf16(w),
        // rounded to bf16, as a second P^T operand, so that the aggregation sees
        // each weight to 16 significant bits (bf16 alone keeps 8).  Over the BF16
        // cache one bf16 operand, the normalizer summing the rounded weights.
        constexpr bool kPairW = !C::lowbit && kRing;
        OpT pl_prev[kPairW ? 2 : 1] = {};
        int pid_next = 0;                  // page id of the tile the next step stages
        bool move_pending = false;         // the previous tile moved the reference:
        float alpha_pending = 1.0f;        // accumulators *= alpha before its aggregation

        // One pipeline step.  QK: scores and softmax of tile `it` (low-bit: plus
        // the dequantization of tile it+1) and the staging of tile it+D; PV:
        // aggregation of tile it-1.
        auto step = [&](const int it, auto QK, auto PV) __attribute__((always_inline)) {
            constexpr bool kQK = decltype(QK)::value, kPV = decltype(PV)::value;
            // The previous step issued Cfg::loads staging loads (none before step
            // 0: the prologue's must all land); everything older must have landed.
            int pid = 0;
            if constexpr (kRing) {
                if (it == 0) plain_barrier<0>();
                else plain_barrier<C::loads>();
            } else {
                // the page of tile it + D, fetched at the end of the previous step
                if (it == 0) pid = wait_barrier<0>(pid_next);
                else pid = wait_barrier<C::loads>(pid_next);
            }
            const int stage_j = it + C::D;
            constexpr int kStageQ = C::D % (C::lowbit ? C::NS : C::NT);    // slot of tile it + D

            f32x16 s;
            if constexpr (kQK) {
                const uint8_t* kt = tiles + tofs[0];
                // every wave computes, also one whose rows all lie past the end
                // (its results are never stored): a branch here would force the
                // accumulators through a register-class join.
                // Scores S^T[token][row], K = 576 in 36 steps, the operands read
                // two k-steps ahead of the matrix instructions, in pairs: the pair
                // (2p, 2p+1) is multiplied in the order 2p+1, 2p, so that one wait
                // for the later read covers both.  Low-bit: the 36 pieces of the
                // next tile's dequantization (reading the staging slot of tile
                // it+1, writing its tile slot, which the aggregation of tile it-2
                // released before this step's barrier) fill the matrix pipe's
                // shadow, one per k-step.
                Dq<kDqKind> dq;
                uint8_t* next_tile = tiles + tofs[1];
                if constexpr (C::lowbit) {
                    dq_read<kDqKind>(dq, stages + sofs[1], tid);
                }
                // k-step kk reads logical chunk 2kk + half: physical 2kk + half (+ kk/4 grouped)
                const uint8_t* krow = kt + row_off(C::SC, qk_row) + 16 * half;
                auto kread_off = [](int kk) { return 16 * (2 * kk + (C::grouped ? kk >> 2 : 0)); };
                constexpr int kAhead = 4;
                OpT kb[kAhead];
#pragma unroll
                for (int j = 0; j < kAhead; ++j) kb[j] = *reinterpret_cast<const OpT*>(krow + kread_off(j));
                // Scheduling barriers after every k-step keep this order (left
                // free, the scheduler trades the read-ahead for registers and every
                // product then waits on LDS latency).
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int kk = 0; kk < kKSteps; ++kk) {
                    const int ko = kk ^ 1;          // 2p+1 first, then 2p
                    mfma_v(s, kb[ko % kAhead], qf[ko], kk == 0);
                    if (kk & 1) {
#pragma unroll
                        for (int j = kk - 1; j <= kk; ++j)
                            if (j + kAhead < kKSteps) kb[j % kAhead] = *reinterpret_cast<const OpT*>(krow + kread_off(j + kAhead));
                    }
                    if constexpr (C::lowbit) dq_step<kDqKind>(dq, kk, next_tile, tid);
                    __builtin_amdgcn_sched_barrier(0);
                }
                score_ready(s);
                if constexpr (C::lowbit) {
#pragma unroll
                    for (int s = kKSteps; s < kDqSteps; ++s) dq_step<kDqKind>(dq, s, next_tile, tid);
                }
                // rows see every key of the tile except in the last tile of the
                // range or the tile holding the newest key (block-uniform test)
                // (and, in a packed phase under protection, the tile holding the
                // last sink token)
                const int t0 = t_begin + it * kTile;
                bool edge = t0 + kTile > full_lim;
                if constexpr (kProt) edge = edge || t0 < t_lo;
                if (edge) {
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int t = t0 + 8 * (v >> 2) + 4 * half + (v & 3);
                        bool ok = t < lim;
                        if constexpr (kProt) ok = ok && t >= t_lo;
                        s[v] = ok ? s[v] : -INFINITY;
                    }
                }
            }
            if constexpr (kPV) {
                if (move_pending) {
                    // the previous tile moved the reference: its weights are on the
                    // new one, the accumulators follow before they are added
#pragma unroll
                    for (int m = 0; m < 16; ++m) scale_acc(acc[m], alpha_pending);
                }
            }

            // Softmax of tile it in pieces (interleaved with the aggregation of
            // tile it-1 when there is one, a piece every second product, the
            // staging loads after them): 0-1 the tile maximum, 2 the reference
            // (a move reaches the accumulators in the next step), 3-10 the
            // weights, two per piece.
            float mr = -INFINITY, nref = 0.0f;
            bool move = false;
            float alpha = 1.0f;
            uint32_t pw[8];
            uint32_t pwl[kPairW ? 8 : 1];
            // (The empty statements pin each piece's results where it is computed:
            // the compiler would otherwise sink the work next to its first use,
            // after the aggregation.)
            auto softmax_piece = [&](int q) __attribute__((always_inline)) {
                if (q == 0) {
                    mr = s[0];
#pragma unroll
                    for (int v = 1; v < 8; ++v) mr = fmaxf(mr, s[v]);
                    asm volatile("" : "+v"(mr));
                } else if (q == 1) {
#pragma unroll
                    for (int v = 8; v < 16; ++v) mr = fmaxf(mr, s[v]);
                    mr = max_halves(mr);
                    asm volatile("" : "+v"(mr));
                } else if (q == 2) {
                    const float mt = mr * a.scale_log2;           // scale > 0: max commutes
                    m_true = fmaxf(m_true, mt);
                    if (m_ref == -INFINITY) m_ref = mt;          // first visible key: nothing accumulated yet
                    move = __builtin_amdgcn_ballot_w64(mt > m_ref + kRefSlack) != 0;
                    const float m_new = move ? fmaxf(m_ref, mt) : m_ref;   // finite for a row that moves
                    alpha = m_new == m_ref ? 1.0f : __builtin_amdgcn_exp2f(m_ref - m_new);
                    m_ref = m_new;
                    l_run *= alpha;
                    nref = m_ref == -INFINITY ? 0.0f : -m_ref;
                    asm volatile("" : "+v"(nref), "+v"(l_run), "+v"(m_ref), "+v"(m_true), "+v"(alpha));
                } else if (q < 11) {
                    const int v2 = q - 3;
                    const float p0 = __builtin_amdgcn_exp2f(fmaf(s[2 * v2], a.scale_log2, nref));
                    const float p1 = __builtin_amdgcn_exp2f(fmaf(s[2 * v2 + 1], a.scale_log2, nref));
                    if constexpr (C::lowbit) {
                        // the sum of the fp16 weights the aggregation uses, one dot2 per pair
                        pw[v2] = pack_f16x2(p0, p1);
                        l_run = __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, pw[v2]), f16x2{1.0f16, 1.0f16}, l_run,
                                                       false);
                    } else if constexpr (kPairW) {
                        l_run += p0 + p1;
                        pw[v2] = pack_bf16x2(p0, p1);
                        // w - bf16(w) is exact in fp32 (|r| <= 2^-9 |w|); its bf16 rounding
                        // leaves each weight to a relative 2^-17
                        const float h0 = __uint_as_float(pw[v2] << 16), h1 = __uint_as_float(pw[v2] & 0xFFFF0000u);
                        pwl[v2 % (kPairW ? 8 : 1)] = pack_bf16x2(p0 - h0, p1 - h1);
                        asm volatile("" : "+v"(pwl[v2 % (kPairW ? 8 : 1)]));
                    } else {
                        // the sum of the bf16 weights the aggregation uses, one dot2 per pair
                        typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
                        pw[v2] = pack_bf16x2(p0, p1);
                        l_run = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pw[v2]),
                                                                bf16x2{static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)},
                                                                l_run, false);
                    }
                    asm volatile("" : "+v"(pw[v2]), "+v"(l_run));
                }
            };
            constexpr int kStageSlot0 = C::lowbit ? 23 : 13, kStageGap = C::lowbit ? 3 : 2;

            if constexpr (kPV) {
                // latent aggregation of tile it-1: O^T[channel][row] += V^T . P^T;
                // the V^T operand is read transposed from the token-major tile.
                // Rows tr_kbase + 16 ks (+ 8): the row shift term of row + 8 is
                // that of row + 2 (tr_kbase < 8), of row + 16 that of the row;
                // channels 32 m + tr_col ..: logical chunk 4m + (0..3), physical
                // + m/2 in the grouped layout
                const uint8_t* vt = tiles + tofs[C::NT - 1];
                const uint8_t* vbase = vt + row_off(C::SC, tr_kbase) + 2 * tr_col;
                auto vread = [&](int stp) __attribute__((always_inline)) {
                    const int ks = stp >> 4, m = stp & 15;
                    const uint8_t* p = vbase + 16 * C::SC * 16 * ks + 64 * m + (C::grouped ? 16 * (m >> 1) : 0);
                    const i16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p);
                    const i16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 16 * C::SC * 8 + 32));
                    return __builtin_bit_cast(OpT, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
                };
                // operands read in pairs one pair ahead; the pair (2p, 2p+1) is
                // multiplied in the order 2p+1, 2p (one wait covers both)
                constexpr int kVAhead = 4;
                OpT vb[kVAhead];
#pragma unroll
                for (int j = 0; j < kVAhead; ++j) vb[j] = vread(j);
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int stp = 0; stp < 32; ++stp) {
                    const int so = stp ^ 1;
                    const int m = so & 15;
                    acc[m] = mfma(vb[so % kVAhead], pb_prev[so >> 4], acc[m]);
                    if constexpr (kPairW) acc[m] = mfma(vb[so % kVAhead], pl_prev[(so >> 4) % 2], acc[m]);
                    if (stp & 1) {
#pragma unroll
                        for (int j = stp - 1; j <= stp; ++j)
                            if (j + kVAhead < 32) vb[j % kVAhead] = vread(j + kVAhead);
                    }
                    if constexpr (kQK) {
                        if (stp % 2 == 0) softmax_piece(stp / 2);
                        // the staging of tile it+D, one load per kStageGap k-steps
                        const int k = (stp - kStageSlot0) / kStageGap;
                        if (stp >= kStageSlot0 && (stp - kStageSlot0) % kStageGap == 0 && k < C::loads)
                            issue(k, pid, cur_t0, cur_po, stage_slot(kStageQ));
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            } else if constexpr (kQK) {
#pragma unroll
                for (int q = 0; q < 11; ++q) softmax_piece(q);
#pragma unroll
                for (int k = 0; k < C::loads; ++k) issue(k, pid, cur_t0, cur_po, stage_slot(kStageQ));
            }
            if constexpr (kQK) {
                pb_prev[0] = __builtin_bit_cast(OpT, make_uint4(pw[0], pw[1], pw[2], pw[3]));
                pb_prev[1] = __builtin_bit_cast(OpT, make_uint4(pw[4], pw[5], pw[6], pw[7]));
                if constexpr (kPairW) {
                    constexpr int n = kPairW ? 8 : 1;
                    pl_prev[0] = __builtin_bit_cast(OpT, make_uint4(pwl[0 % n], pwl[1 % n], pwl[2 % n], pwl[3 % n]));
                    pl_prev[1 % (kPairW ? 2 : 1)] =
                        __builtin_bit_cast(OpT, make_uint4(pwl[4 % n], pwl[5 % n], pwl[6 % n], pwl[7 % n]));
                }
                move_pending = move;
                alpha_pending = alpha;
                // advance the staging cursor (it stays on the last tile)
                if (stage_j + 1 < n_tiles) {
                    cur_t0 += kTile;
                    cur_po += kTile;
                    if (cur_po == P) {
                        cur_po = 0;
                        ++cur_page;
                    }
                }
                if constexpr (!kRing) issue_page_id(bt, cur_page, pid_next);
            }
            // the buffer slots move on by one tile
            {
                const int t = tofs[0];
#pragma unroll
                for (int q = 0; q + 1 < C::NT; ++q) tofs[q] = tofs[q + 1];
                tofs[C::NT - 1] = t;
            }
            if constexpr (C::NS > 1) {
                const int t = sofs[0];
#pragma unroll
                for (int q = 0; q + 1 < C::NS; ++q) sofs[q] = sofs[q + 1];
                sofs[C::NS - 1] = t;
            }
        };

        if (n_tiles > 0) {
            // prologue part 2: tile 0 decoded (low-bit) before the first step
            if constexpr (C::lowbit) {
                pid_next = step_barrier<0>(bt, cur_page);
                dequant_tile<kDqKind>(stages, tiles, tid);
            } else if constexpr (!kRing) {
                issue_page_id(bt, cur_page, pid_next);
            }
            step(0, std::true_type{}, std::false_type{});
            for (int it = 1; it < n_tiles; ++it) step(it, std::true_type{}, std::true_type{});
            step(n_tiles, std::false_type{}, std::true_type{});
            // no direct-to-LDS load may outlive the workgroup's LDS
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        }

    };

    if constexpr (!kProt) {
        int t_begin = 0, t_end = L;
        if (a.split_tokens != 0) {
            t_begin = max(split * a.split_tokens, 0);
            t_end = min(split * a.split_tokens + a.split_tokens, L);
        }
        const int lim = row_ok ? min(L - a.s_q + qi + 1, t_end) : t_begin;   // keys t < lim are visible
        const int full_lim = min(L - a.s_q + 1, t_end);    // every valid row sees keys t < full_lim
        if (a.new_c != nullptr) append_in_launch<KIND>(a, b, L, t_begin, t_end, tid);
        run(std::integral_constant<int, KIND>{}, std::false_type{}, t_begin, t_end, t_begin, lim, full_lim);
    } else {
        const int sink = a.sink, recent = a.recent;
        const bool has_packed = L - recent > sink;          // else every token is protected
        const int pk0 = has_packed ? sink / kTile : 0;
        const int n_pk = has_packed ? (L - recent + kTile - 1) / kTile - pk0 : 0;
        const int n_prot = has_packed ? sink + recent : L;
        const int n_list = n_pk + (n_prot + kTile - 1) / kTile;
        int u0 = 0, u1 = n_list;
        if (a.split_tokens != 0) {
            u0 = split * (a.split_tokens / kTile);
            u1 = min(u0 + a.split_tokens / kTile, n_list);
        }
        if constexpr (Cfg<KIND>::lowbit) {
            if (a.new_c != nullptr) append_in_launch_protected<KIND>(a, b, L, u0, u1, n_pk, pk0, tid);
        }
        if (u0 < n_pk) {
            const int tb = kTile * (pk0 + u0);
            const int te = min(kTile * (pk0 + min(u1, n_pk)), L - recent);
            const int lim = row_ok ? min(L - a.s_q + qi + 1, te) : tb;
            const int full_lim = min(L - a.s_q + 1, te);
            run(std::integral_constant<int, KIND>{}, std::false_type{}, tb, te, sink, lim, full_lim);
        }
        if (u1 > n_pk) {
            // every wave is done with the packed phase's LDS before the
            // protected phase stages into the same memory
            if (u0 < n_pk) __syncthreads();
            ring_rows = sink + recent;
            ring_nsink = min(sink, L);
            const int r0 = max(sink, L - recent);       // first window position past the sink
            ring_q0 = recent > 0 ? (r0 - sink) % recent : 0;
            int64_t pslot = a.prot_slot[b];
            pslot = pslot < 0 ? 0 : (pslot >= a.num_prot ? a.num_prot - 1 : pslot);
            ring_base = a.prot + pslot * ring_rows * 1152;
            // protected positions below x
            auto below = [&](int x) { return min(max(x, 0), ring_nsink) + max(0, x - r0); };
            const int vb = kTile * (max(u0, n_pk) - n_pk);
            const int ve = min(kTile * (u1 - n_pk), n_prot);
            const int lim = row_ok ? min(below(L - a.s_q + qi + 1), ve) : vb;
            const int full_lim = min(below(L - a.s_q + 1), ve);
            run(std::integral_constant<int, KIND_BF16>{}, std::true_type{}, vb, ve, 0, lim, full_lim);
        }
    }

    // Epilogue.  A lane holds row (lane & 31) of its wave, channels 32 m +
    // 8 q + 4 half .. +3 of the accumulators.  The rows go out through LDS so
    // that each store writes one whole row (1 KiB, 64 lanes x 16 bytes) instead
    // of 16-byte pieces of 32 rows: wave w stages its 32 rows at 1040-byte
    // pitch (the 16-byte shift per row spreads the 32 rows of a write over the
    // banks), then reads them back row by row.
    const float l_tot = sum_halves(l_run);
    const bool split_out = a.split_tokens != 0;
    const float inv = l_tot > 0.0f ? 1.0f / l_tot : 0.0f;
    __syncthreads();        // every wave is done with the tiles (no staging load is in flight)
    constexpr int kRowPitch = 1040;
    static_assert(kWaves * 32 * kRowPitch <= kLds, "epilogue rows fit the LDS");
    uint8_t* ep = smem + wave * 32 * kRowPitch;
#pragma unroll
    for (int m = 0; m < 16; ++m) {
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
            const float x0 = acc[m][4 * q4] * inv, x1 = acc[m][4 * q4 + 1] * inv;
            const float x2 = acc[m][4 * q4 + 2] * inv, x3 = acc[m][4 * q4 + 3] * inv;
            // partials: the split's normalized aggregation in fp16 (the combine
            // weighs it by part_s); unsplit: the output in bf16
            const uint2 u = split_out ? make_uint2(pack_f16x2(x0, x1), pack_f16x2(x2, x3))
                                      : make_uint2(pack_bf16x2(x0, x1), pack_bf16x2(x2, x3));
            *reinterpret_cast<uint2*>(ep + (lane & 31) * kRowPitch + 2 * (32 * m + 8 * q4 + 4 * half)) = u;
        }
    }
    // rows r = row block + 32 wave + i are (b, i, h) rows of the output, or of
    // work item w's partials
    const int row0 = rb * kRowsPerBlock + wave * 32;
    uint16_t* dst = split_out ? a.part_o + (static_cast<int64_t>(w) * rows_total + row0) * kDc
                              : a.out + (static_cast<int64_t>(b) * rows_total + row0) * kDc;
    // Non-temporal stores: every workgroup writes its rows at about the same
    // time, at the end of the launch, and the write burst is the epilogue's
    // bound; written as streaming data they cost less.
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
#pragma unroll
    for (int i = 0; i < 32; ++i) {
        if (row0 + i < rows_total)
            __builtin_nontemporal_store(*reinterpret_cast<const u32x4*>(ep + i * kRowPitch + 16 * lane),
                                        reinterpret_cast<u32x4*>(dst + i * kDc + 8 * lane));
    }
    if (!row_ok || half != 0) return;
    if (!split_out) {
        if (a.lse != nullptr) {
            const int64_t orow = (static_cast<int64_t>(b) * a.s_q + qi) * a.H + h;
            a.lse[orow] = l_tot > 0.0f ? (m_ref + log2f(l_tot)) * kLn2 : -INFINITY;
        }
    } else {
        const int64_t prow = (static_cast<int64_t>(w) * a.s_q + qi) * a.H + h;
        const float f = m_true == -INFINITY ? 0.0f : exp2f(m_ref - m_true);
        a.part_m[prow] = m_true * kLn2;
        a.part_s[prow] = l_tot * f;
    }
}

}  // namespace

hipError_t launch_decode(CacheKind kind, const DecodeArgs& a, hipStream_t stream) {
    if (a.num_work == 0) return hipSuccess;
    const LaunchEvents ev = take_launch_events();
    const int64_t blocks = decode_workgroups(a.num_work, static_cast<int64_t>(a.s_q) * a.H, kRowsPerBlock);
    const dim3 grid(static_cast<unsigned>(blocks)), block(kThreads);
    switch (kind) {
        case KIND_C4R4: dispatch_decode(decode_kernel<KIND_C4R4, false>, grid, block, stream, ev, a); break;
        case KIND_C2R4: dispatch_decode(decode_kernel<KIND_C2R4, false>, grid, block, stream, ev, a); break;
        case KIND_C4R4P: dispatch_decode(decode_kernel<KIND_C4R4P, false>, grid, block, stream, ev, a); break;
        case KIND_C2R4P: dispatch_decode(decode_kernel<KIND_C2R4P, false>, grid, block, stream, ev, a); break;
        case KIND_BF16: dispatch_decode(decode_kernel<KIND_BF16, false>, grid, block, stream, ev, a); break;
    }
    return hipGetLastError();
}

hipError_t launch_decode_protected(CacheKind kind, const DecodeArgs& a, hipStream_t stream) {
    if (a.num_work == 0) return hipSuccess;
    const LaunchEvents ev = take_launch_events();
    const int64_t blocks = decode_workgroups(a.num_work, static_cast<int64_t>(a.s_q) * a.H, kRowsPerBlock);
    const dim3 grid(static_cast<unsigned>(blocks)), block(kThreads);
    switch (kind) {
        case KIND_C4R4: dispatch_decode(decode_kernel<KIND_C4R4, true>, grid, block, stream, ev, a); break;
        case KIND_C2R4: dispatch_decode(decode_kernel<KIND_C2R4, true>, grid, block, stream, ev, a); break;
        case KIND_C4R4P: dispatch_decode(decode_kernel<KIND_C4R4P, true>, grid, block, stream, ev, a); break;
        case KIND_C2R4P: dispatch_decode(decode_kernel<KIND_C2R4P, true>, grid, block, stream, ev, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace mla
