// Decode attention for few query rows per sequence (16 per workgroup), the
// regime of 16 heads and one query token (Appendix F.1, "Native Attention"),
// where the 128-row kernel of decode_attn.hip would leave 7/8 of every matrix
// instruction idle.  Same computation and results contract: absorbed MLA
// scores z_t = tau (q_lat . C_hat_t + q_rope . K_hat_t), softmax, latent
// aggregation O = A C_hat (Sec. 2.1, eq. mla_compact), split partials as in
// Appendix C.5 "Global attention normalization", BF16 protection of sink and
// recent tokens as in Appendix C.5 "BF16 protection and cache lifecycle".
//
// Workgroup = one wave (64 lanes), several per CU; no workgroup barriers.
// It owns one (sequence or key split, block of 16 query rows).  Lane l works
// on query row l % 16 and lane group g = l / 16.
//
// Per 16-token tile (low-bit cache):
//   1. the packed bytes are copied HBM -> LDS by direct-to-LDS loads two tiles
//      ahead, gathered chunk-major (16-byte chunk j of token m at chunk slot
//      16 j + m) so that the per-lane code reads below are bank-conflict-free;
//   2. scores S^T[token][row] = K_tile . Q^T with v_mfma_f32_16x16x32_f16: the
//      A operand of k-step kk is token l % 16, channels 32 kk + 8 g .. +8 --
//      one 32-bit word of 4-bit codes, dequantized in registers (x_hat =
//      scale * (q - zero), one fp16 rounding); the dequantized content
//      channels are also stored to an fp16 tile in LDS;
//   3. softmax: a lane holds tokens 4 g .. 4 g + 3 of its row; maxima and sums
//      combine the four lane groups with v_permlane16/32_swap;
//   4. aggregation O^T[channel][row] += V^T . P^T with v_mfma_f32_16x16x16_f16
//      (32 channel blocks, K = the 16 tokens): V^T read transposed from the
//      fp16 tile with ds_read_b64_tr_b16, P^T straight from the score
//      registers (the lane's four tokens are the B operand's K slice).
// BF16 rows (the BF16 cache, and protected rows from a protection buffer)
// are staged raw into a padded tile and feed both products directly.
//
// Online softmax as in decode_attn.hip: a per-row reference (log2 units) that
// moves only when a tile exceeds it by more than 2^10, the accumulators
// rescaled on the move; the true maximum is tracked for the split partials.
#include <hip/hip_runtime.h>

#include <cmath>
#include <type_traits>

#include "internal.h"
#include "kernel_common.h"
#include "writer_common.h"

namespace mla {
namespace {

using namespace kc;

typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kRows = 16;           // query rows per workgroup
static_assert(kRows == kNarrowRowsPerBlock, "launch shape the host checks");
constexpr int kTok = 16;            // tokens per tile
constexpr int kQSteps = 18;         // 576 channels / 32 per k-step
constexpr int kDc = 512;
constexpr float kRefSlack = 10.0f;
constexpr float kLn2 = 0.693147180559945309f;

// LDS tiles, in 16-byte units.  Row r of the fp16 content tile starts at unit
// 66 r + r / 8, row r of a raw bf16 tile at 74 r + r / 8: the dequantization
// stores and score reads (16 rows, one chunk each) and the transposing reads
// (8 rows, two chunks each, per half wave) then fall on distinct banks.
__host__ __device__ constexpr int f16_row(int r) { return 66 * r + (r >> 3); }
__host__ __device__ constexpr int bf_row(int r) { return 74 * r + (r >> 3); }
constexpr int kF16TileBytes = 16 * (f16_row(15) + 64);
constexpr int kBfUnits = (bf_row(15) + 72 + 63) / 64 * 64;
constexpr int kBfTileBytes = 16 * kBfUnits;
constexpr int kBfLoads = kBfUnits / 64;
static_assert(kBfLoads == 19, "bf16 tile staging loads");

// Narrow configuration per cache kind.  Low-bit staging slot (units): content
// codes chunk-major [cc/16 chunks][16 tokens], RoPE codes [2][16], metadata
// [2][16] (fp16 content pairs, or the paper's 32-byte record), and for fp16
// metadata the RoPE pairs token-major (4 units).
template <int KIND> struct NCfg {
    static constexpr bool lowbit = true;
    static constexpr bool pmeta = KIND == KIND_C4R4P || KIND == KIND_C2R4P;
    static constexpr int cbits = (KIND == KIND_C4R4 || KIND == KIND_C4R4P) ? 4 : 2;
    static constexpr int cc = 512 * cbits / 8;            // content code bytes per token
    static constexpr int u_rc = cc, u_mc = cc + 32, u_mr = cc + 64;
    static constexpr int units = u_mr + (pmeta ? 0 : 4);
    static constexpr int loads = (units + 63) / 64;
    static constexpr int stage_bytes = 16 * units;
    static constexpr int NS = 3, D = 2;                   // staging slots, tiles ahead
    static constexpr int lds = NS * stage_bytes + kF16TileBytes;
};
template <> struct NCfg<KIND_BF16> {
    static constexpr bool lowbit = false;
    static constexpr int loads = kBfLoads;
    static constexpr int NS = 2, D = 1;                   // tile slots, tiles ahead
    static constexpr int lds = NS * kBfTileBytes;
};

template <int KIND>
constexpr int narrow_lds(bool prot) {
    return prot && NCfg<KIND_BF16>::lds > NCfg<KIND>::lds ? NCfg<KIND_BF16>::lds : NCfg<KIND>::lds;
}

template <int N>
__device__ __forceinline__ void wait_loads() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" : : "n"(N) : "memory");
}

// value and its copies in lanes ^16, ^32, ^48 combined
__device__ __forceinline__ float max4(float v) {
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
    r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum4(float v) {
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Staging of one low-bit tile: load k (of NCfg::loads) covers slot units
// 64 k .. 64 k + 63 (lane = unit - 64 k).  Tokens at or past nvalid re-read
// token nvalid - 1 (the RoPE pairs: four tokens per chunk, read as they are).
// The content codes fill whole loads (cc / 64 of them); the next load carries
// the RoPE codes (lanes 0-31) and the metadata (lanes 32-63); with fp16
// metadata a last load brings the RoPE pairs (lanes 0-3).
template <int KIND>
__device__ __forceinline__ void stage_narrow_lowbit(int k, const uint8_t* page, int po, int nvalid,
                                                    const PageGeom& g, uint32_t lds, int lane) {
    using C = NCfg<KIND>;
    static_assert(C::u_rc % 64 == 0 && C::u_mr == C::u_rc + 64, "region boundaries on load boundaries");
    const int last = nvalid - 1;
    if (k < C::u_rc / 64) {
        const int u = 64 * k + lane;
        dma16_m0(page, (po + min(u & 15, last)) * C::cc + 16 * (u >> 4), lds + 64 * 16 * k);
    } else if (k == C::u_rc / 64) {
        const int v = lane & 31;
        const int base = lane < 32 ? g.off_cr : g.off_mc;
        dma16_m0(page, base + (po + min(v & 15, last)) * 32 + 16 * (v >> 4), lds + 64 * 16 * k);
    } else if (lane < 4) {
        dma16_m0(page, g.off_mr + po * 4 + 16 * lane, lds + 64 * 16 * k);
    }
}

// Staging of one raw bf16 tile (576 channels per row) into the padded layout:
// unit u belongs to the last row starting at or before it; padding units
// re-read column 71.  Row tok of the tile starts at byte row_start(tok).
template <class RowStart>
__device__ __forceinline__ void stage_narrow_bf16(int k, const uint8_t* src, RowStart row_start, int nvalid,
                                                  uint32_t lds, int lane) {
    const int u = 64 * k + lane;
    int r = min(u / 74, 15);
    if (u < bf_row(r)) --r;
    const int col = min(u - bf_row(r), 71);
    dma16_m0(src, row_start(min(r, nvalid - 1)) + 16 * col, lds + 64 * 16 * k);
}

// Dequantize 8 channels into fp16 pairs (2p, 2p+1).  In the code layout a
// channel pair sits at one bit offset of the two 16-bit halves of a word: the
// 8 channels are the word's pairs at bit offsets sh0 + CBITS p (a 4-bit word
// holds exactly 8 channels, sh0 = 0; a 2-bit word 16, sh0 = 0 or 8).  A pair
// is extracted in place at its offset o within a byte: masked and or'ed with
// 0x6400 it is the fp16 value 1024 + 2^o q.  For o = 0, subtracting
// zz = 1024 + zero leaves q - zero; otherwise one fused multiply-add by 2^-o
// adds zo = -(1024 / 2^o + zero) (zo[o / 2 - 1]).  Both are exact, so the
// word is shifted only by whole bytes, and the one rounding is the multiply
// by the scale.
template <int CBITS>
__device__ __forceinline__ f16x8 dequant8(uint32_t w, int sh0, f16x2 zz, const f16x2* zo, f16x2 ss) {
    uint32_t o[4];
    if constexpr (CBITS == 4) {
        const uint32_t w8 = w >> 8;
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const uint32_t src = p < 2 ? w : w8;
            const f16x2 x = __builtin_bit_cast(f16x2, and_or(src, (p & 1) ? 0x00F000F0u : 0x000F000Fu, 0x64006400u));
            const f16x2 d = (p & 1) ? __builtin_elementwise_fma(x, f16x2{0.0625f16, 0.0625f16}, zo[1]) : x - zz;
            o[p] = __builtin_bit_cast(uint32_t, d * ss);
        }
    } else {
        const uint32_t ws = w >> sh0;
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const f16x2 x = __builtin_bit_cast(f16x2, and_or(ws, 0x00030003u << (2 * p), 0x64006400u));
            constexpr _Float16 kInv[4] = {1.0f16, 0.25f16, 0.0625f16, 0.015625f16};
            const f16x2 d = p == 0 ? x - zz : __builtin_elementwise_fma(x, f16x2{kInv[p], kInv[p]}, zo[p - 1]);
            o[p] = __builtin_bit_cast(uint32_t, d * ss);
        }
    }
    return __builtin_bit_cast(f16x8, make_uint4(o[0], o[1], o[2], o[3]));
}

// zo[k] = -(1024 / 2^o + zero) for o = 2 (k + 1), from zz = 1024 + zero
// (exact: integers and quarters below 1024).
__device__ __forceinline__ void zero_offsets(f16x2 zz, f16x2* zo) {
    zo[0] = f16x2{768.0f16, 768.0f16} - zz;
    zo[1] = f16x2{960.0f16, 960.0f16} - zz;
    zo[2] = f16x2{1008.0f16, 1008.0f16} - zz;
}

// In-launch append (the writer of mla_lowbit_quant_append / mla_bf16_append,
// and under protection of mla_lowbit_quant_append_protected, for the step's
// new tokens), as in decode_attn.hip: the work item that reads a new token
// (`reads(p)`: its key range, or under protection its key list, holds
// position p) writes it before it stages any tile -- the packed copy (BF16:
// the row), and under protection, for a token protected after the step, its
// bf16 row into ring row p or sink + (p - sink) mod recent of the sequence's
// buffer (skipped for a buffer index outside [0, num_prot)).  One 16-byte
// piece per lane and round (72 per token; a group's 8 lanes stay together,
// as the quantizer needs); the wave's stores land before its first staging
// load.
template <int KIND, bool kProt, class Reads>
__device__ __forceinline__ void narrow_append(const DecodeArgs& a, int b, int L, Reads reads, int lane) {
    using C = NCfg<KIND>;
    bool any = false;
    for (int i = 0; i < a.s_q; ++i) {
        const int pos = L - a.s_q + i;
        if (pos >= 0 && reads(pos)) any = true;
    }
    if (!any) return;
    const int64_t num_slots = a.num_pages * a.g.page_size;
    for (int piece = lane; piece < 72 * a.s_q; piece += 64) {
        const int i = piece / 72, r = piece % 72;
        const int pos = L - a.s_q + i;
        if (pos < 0 || !reads(pos)) continue;
        const int64_t tok = static_cast<int64_t>(b) * a.s_q + i;
        const int64_t slot = a.new_slots[tok];
        if (slot < 0 || slot >= num_slots) continue;
        uint8_t* base = const_cast<uint8_t*>(a.cache) + slot / a.g.page_size * a.g.page_bytes;
        const int64_t off = slot % a.g.page_size;
        const bool rope = r >= 64;
        const uint16_t* src = rope ? a.new_k + tok * a.new_k_stride + (r - 64) * 8
                                   : a.new_c + tok * a.new_c_stride + r * 8;
        const uint4 raw = *reinterpret_cast<const uint4*>(src);
        if constexpr (C::lowbit) {
            wc::quantize_store<C::cbits, C::pmeta>(raw, rope, r >> 3, r & 7, base, off, a.g);
            if constexpr (kProt) {
                const int64_t ps = a.prot_slot[b];
                if ((pos < a.sink || pos >= L - a.recent) && ps >= 0 && ps < a.num_prot) {
                    const int prow = pos < a.sink ? pos : a.sink + (pos - a.sink) % a.recent;
                    uint8_t* dst = const_cast<uint8_t*>(a.prot) + (ps * (a.sink + a.recent) + prow) * 1152 + 16 * r;
                    *reinterpret_cast<uint4*>(dst) = raw;
                }
            }
        } else {
            *reinterpret_cast<uint4*>(base + off * 1152 + r * 16) = raw;
        }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// ---------------------------------------------------------------------------
template <int KIND, bool kProt>
__global__ __launch_bounds__(64) void narrow_kernel(DecodeArgs a) {
    __shared__ __attribute__((aligned(1024))) uint8_t smem[narrow_lds<KIND>(kProt)];

    const int lane = threadIdx.x;
    const int g = lane >> 4;            // lane group: tokens 4g..4g+3 of a tile, k slice 8g..8g+7
    const int li = lane & 15;           // query row within the block; token of the score A operand
    const int rows_total = a.s_q * a.H;
    const int RB = (rows_total + kRows - 1) / kRows;

    // Block -> (work item, row block): contiguous work items per XCD (block
    // id mod 8), as in decode_attn.hip.
    const int per_xcd = (a.num_work + 7) / 8;
    const int slot = blockIdx.x >> 3;
    const int w = (blockIdx.x & 7) * per_xcd + slot / RB;
    const int rb = slot % RB;
    if (w >= a.num_work) return;

    const int P = a.g.page_size;
    int b, split = 0;
    int Lraw;
    if (a.split_tokens == 0) {
        b = w;
        Lraw = a.seq_lens[b];
    } else {
        // the last b with split_indptr[b] <= w, counted 64 entries at a time
        // with the lengths loaded alongside: one round of loads instead of a
        // chain of dependent ones (as in decode_attn.hip)
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

    const int row = rb * kRows + li;
    const bool row_ok = row < rows_total;
    const int qi = row_ok ? row / a.H : 0;
    const int h = row_ok ? row % a.H : 0;
    const int64_t qrow = (static_cast<int64_t>(b) * a.s_q + qi) * a.H + h;

    float m_ref = -INFINITY, m_true = -INFINITY, l_run = 0.0f;
    f32x4 acc[32];
#pragma unroll
    for (int m = 0; m < 32; ++m) acc[m] = f32x4{};

    const uint8_t* ring_base = nullptr;
    int ring_rows = 1, ring_nsink = 0, ring_q0 = 0;

    // One phase over keys [t_begin, t_end) in one representation (see
    // decode_attn.hip): PK is the cache kind whose pipeline runs; kRing reads
    // bf16 rows of the protection buffer.  This lane's row sees keys
    // t_lo <= t < lim.
    auto run = [&](auto kind_c, auto ring_c, const int t_begin, const int t_end, const int t_lo,
                   const int lim) __attribute__((always_inline)) {
        constexpr int PK = decltype(kind_c)::value;
        constexpr bool kRing = decltype(ring_c)::value;
        using C = NCfg<PK>;
        using OpT = std::conditional_t<C::lowbit, f16x8, bf16x8>;
        const int n_tiles = t_end > t_begin ? (t_end - t_begin + kTok - 1) / kTok : 0;
        (void)t_lo;

        // queries (B operand of the scores): k-step kk holds channels 32 kk + 8 g .. +8 of row li
        OpT qf[kQSteps];
        {
            const uint16_t* ql = a.q_lat + qrow * kDc + 8 * g;
            const uint16_t* qr = a.q_rope + qrow * 64 + 8 * g;
#pragma unroll
            for (int kk = 0; kk < kQSteps; ++kk) {
                // rows past the end read a valid row; their results are never stored
                const uint4 v = *reinterpret_cast<const uint4*>(kk < 16 ? ql + 32 * kk : qr + 32 * (kk - 16));
                if constexpr (C::lowbit)
                    qf[kk] = __builtin_bit_cast(f16x8, make_uint4(bf16x2_to_f16x2(v.x), bf16x2_to_f16x2(v.y),
                                                                  bf16x2_to_f16x2(v.z), bf16x2_to_f16x2(v.w)));
                else
                    qf[kk] = __builtin_bit_cast(bf16x8, v);
                // kept in accumulation registers, which the score products read
                // directly as their B operand
                asm volatile("" : "+a"(qf[kk]));
            }
        }

        auto slot_base = [&](int j) {
            if constexpr (C::lowbit) return smem + slot_offset(j, C::NS, C::stage_bytes);
            else return smem + slot_offset(j, C::NS, kBfTileBytes);
        };
        int st_pg = t_begin / P, st_po = t_begin % P, pid_pg = -1, pid = 0;   // next tile to stage
        auto issue_tile = [&](int j) __attribute__((always_inline)) {
            const int t0 = t_begin + min(j, n_tiles - 1) * kTok;   // past the end: the last tile again
            const int nvalid = min(t_end - t0, kTok);
            const uint32_t lds = lds_addr(slot_base(j));
            if constexpr (kRing) {
                auto row_start = [&](int tok) {
                    const int v = t0 + tok;
                    const int x = ring_q0 + (v - ring_nsink);       // < 2 * recent
                    const int r = v < ring_nsink ? v : a.sink + (x >= a.recent ? x - a.recent : x);
                    return min(r, ring_rows - 1) * 1152;
                };
#pragma unroll
                for (int k = 0; k < C::loads; ++k) stage_narrow_bf16(k, ring_base, row_start, nvalid, lds, lane);
            } else {
                // tiles are issued in order; a 16-token tile never crosses a page
                // (t_begin and the page size are multiples of 32), and the page
                // id is fetched once per page
                if (st_pg != pid_pg) {
                    pid = load_page_id(bt, st_pg);
                    pid = min(max(pid, 0), static_cast<int>(a.num_pages - 1));
                    pid_pg = st_pg;
                }
                const uint8_t* page = a.cache + static_cast<int64_t>(pid) * a.g.page_bytes;
                const int po = st_po;
                if (j < n_tiles - 1) {
                    st_po += kTok;
                    if (st_po == P) {
                        st_po = 0;
                        ++st_pg;
                    }
                }
                if constexpr (C::lowbit) {
#pragma unroll
                    for (int k = 0; k < C::loads; ++k) stage_narrow_lowbit<PK>(k, page, po, nvalid, a.g, lds, lane);
                } else {
                    auto row_start = [&](int tok) { return (po + tok) * 1152; };
#pragma unroll
                    for (int k = 0; k < C::loads; ++k) stage_narrow_bf16(k, page, row_start, nvalid, lds, lane);
                }
            }
        };

        if (n_tiles == 0) return;
#pragma unroll
        for (int j = 0; j < C::D; ++j) issue_tile(j);

        // online softmax of one tile's scores (lane: tokens 4g+v of row li):
        // masks, moves the reference (rescaling the accumulators, which hold
        // every earlier tile) when needed, returns the weights
        auto softmax = [&](int it, f32x4 s, float p[4]) __attribute__((always_inline)) {
            const int t0 = t_begin + it * kTok;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int t = t0 + 4 * g + v;
                bool ok = t < lim;
                if constexpr (kProt) ok = ok && t >= t_lo;
                s[v] = ok ? s[v] : -INFINITY;
            }
            const float mr = max4(fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3])));
            const float mt = mr * a.scale_log2;
            m_true = fmaxf(m_true, mt);
            if (m_ref == -INFINITY) m_ref = mt;
            const bool move = __builtin_amdgcn_ballot_w64(mt > m_ref + kRefSlack) != 0;
            if (move) {
                const float m_new = fmaxf(m_ref, mt);
                const float alpha = m_new == m_ref ? 1.0f : __builtin_amdgcn_exp2f(m_ref - m_new);
                m_ref = m_new;
                l_run *= alpha;
#pragma unroll
                for (int m = 0; m < 32; ++m) acc[m] *= alpha;
            }
            const float nref = m_ref == -INFINITY ? 0.0f : -m_ref;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                p[v] = __builtin_amdgcn_exp2f(fmaf(s[v], a.scale_log2, nref));
                // the normalizer sums the weights the aggregation uses: fp16-rounded
                // (low-bit), bf16-rounded (the BF16 cache), or to 16 significant bits
                // (protected rows, a bf16 pair)
                if constexpr (C::lowbit) p[v] = static_cast<float>(static_cast<_Float16>(p[v]));
                else if constexpr (!kRing) p[v] = static_cast<float>(static_cast<__bf16>(p[v]));
                l_run += p[v];
            }
        };

        if constexpr (C::lowbit) {
            // Software pipeline: step it computes the scores of tile it (its
            // operands dequantized in registers) interleaved with the aggregation
            // of tile it-1 (read transposed from the fp16 tile); once the
            // aggregation's reads are done, tile it's content channels replace
            // tile it-1's in the fp16 tile.
            uint8_t* tile = smem + C::NS * C::stage_bytes;
            const uint8_t* vbase = tile + 16 * f16_row(4 * g + (li >> 2)) + 8 * (li & 3);
            uint32_t words[kQSteps];
            uint4 mc0, mc1;
            uint32_t rmw = 0;
            auto read_stage = [&](const uint8_t* st) __attribute__((always_inline)) {
#pragma unroll
                for (int kk = 0; kk < kQSteps; ++kk) {
                    if (kk >= 16)
                        words[kk] = *reinterpret_cast<const uint32_t*>(st + 16 * (C::u_rc + 16 * (kk - 16) + li) + 4 * g);
                    else if constexpr (C::cbits == 4)
                        words[kk] = *reinterpret_cast<const uint32_t*>(st + 16 * (16 * kk + li) + 4 * g);
                    else    // channels 32 kk + 8 g ..: word 2 kk + g / 2, upper or lower 8 (sh0)
                        words[kk] = *reinterpret_cast<const uint32_t*>(st + 16 * (16 * (kk >> 1) + li) + 8 * (kk & 1) +
                                                                       4 * (g >> 1));
                }
                mc0 = *reinterpret_cast<const uint4*>(st + 16 * (C::u_mc + li));
                mc1 = *reinterpret_cast<const uint4*>(st + 16 * (C::u_mc + 16 + li));
                if constexpr (!C::pmeta) rmw = *reinterpret_cast<const uint32_t*>(st + 16 * C::u_mr + 4 * li);
            };
            // dequantization constants of the group holding k-step kk (its
            // scale, 1024 + zero, and the zero offsets of the in-place extraction)
            struct Gm { f16x2 zz, ss, zo[3]; };
            auto group_meta = [&](int kk) __attribute__((always_inline)) {
                Gm m;
                if (kk >= 16) {
                    if constexpr (C::pmeta) pmeta_to_f16(__uint_as_float(mc1.z), mc1.w & 0xFFu, m.zz, m.ss);
                    else meta_to_f16(rmw, m.zz, m.ss);
                } else {
                    const int grp = kk >> 1;
                    if constexpr (C::pmeta) {
                        const uint32_t sw = grp < 4 ? (grp < 2 ? mc0.x : mc0.y) : (grp < 6 ? mc0.z : mc0.w);
                        const uint32_t sbits = (sw >> (16 * (grp & 1))) & 0xFFFFu;
                        const uint32_t zw = grp < 4 ? mc1.x : mc1.y;
                        pmeta_to_f16(__uint_as_float(sbits << 16), (zw >> (8 * (grp & 3))) & 0xFFu, m.zz, m.ss);
                    } else {
                        const uint32_t mw = grp < 4 ? (grp < 2 ? (grp == 0 ? mc0.x : mc0.y) : (grp == 2 ? mc0.z : mc0.w))
                                                    : (grp < 6 ? (grp == 4 ? mc1.x : mc1.y) : (grp == 6 ? mc1.z : mc1.w));
                        meta_to_f16(mw, m.zz, m.ss);
                    }
                }
                zero_offsets(m.zz, m.zo);
                return m;
            };
            auto dq = [&](int kk, const Gm& m) __attribute__((always_inline)) {
                if (kk >= 16) return dequant8<4>(words[kk], 0, m.zz, m.zo, m.ss);
                return dequant8<C::cbits>(words[kk], C::cbits == 4 ? 0 : 8 * (g & 1), m.zz, m.zo, m.ss);
            };
            float p[4] = {0.0f, 0.0f, 0.0f, 0.0f};
            constexpr int kVAhead = 8;
            s16x4 vb[kVAhead];
            auto vread = [&](int m) {
                return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vbase + 32 * m));
            };
            auto pv = [&](int m, f16x4 pbh) __attribute__((always_inline)) {
                acc[m] = __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(f16x4, vb[m % kVAhead]), pbh, acc[m],
                                                               0, 0, 0);
                if (m + kVAhead < 32) vb[m % kVAhead] = vread(m + kVAhead);
            };
            // one step: scores of tile it (QK) and aggregation of tile it-1 (PV).
            // Tile it's content channels 32 kk + 8 g .. +8 (channel blocks 2 kk and
            // 2 kk + 1) replace tile it-1's as soon as they are dequantized: the
            // transposing reads of those blocks were issued before (in the previous
            // k-steps, or before the loop), and LDS serves one wave's accesses in
            // the order they are issued.
            auto step = [&](int it, auto QK, auto PV) __attribute__((always_inline)) {
                constexpr bool kQK = decltype(QK)::value, kPV = decltype(PV)::value;
                const f16x4 pbh = {static_cast<_Float16>(p[0]), static_cast<_Float16>(p[1]),
                                   static_cast<_Float16>(p[2]), static_cast<_Float16>(p[3])};
                f32x4 s = f32x4{};
                // tile it's code words were read at the end of the previous step;
                // its staging slot is free (the slot of tile it + D held tile it - 1)
                if constexpr (kQK) issue_tile(it + C::D);
                if constexpr (kPV) {
#pragma unroll
                    for (int m = 0; m < kVAhead; ++m) vb[m] = vread(m);
                }
                __builtin_amdgcn_sched_barrier(0);
                // the dequantization runs one k-step ahead of the score product,
                // so that vector work separates the products (each 16 cycles on the
                // matrix unit) instead of issuing them back to back
                Gm gm;
                f16x8 kv_next;
                if constexpr (kQK) {
                    gm = group_meta(0);
                    kv_next = dq(0, gm);
                }
#pragma unroll
                for (int kk = 0; kk < kQSteps; ++kk) {
                    f16x8 kv;
                    if constexpr (kQK) {
                        kv = kv_next;
                        s = __builtin_amdgcn_mfma_f32_16x16x32_f16(kv, qf[kk], s, 0, 0, 0);
                    }
                    if constexpr (kPV) {
                        if (kk < 16) pv(2 * kk, pbh);
                    }
                    if constexpr (kQK) {
                        if (kk + 1 < kQSteps) {
                            if (((kk + 1) & 1) == 0) gm = group_meta(kk + 1);
                            kv_next = dq(kk + 1, gm);
                        }
                    }
                    if constexpr (kPV) {
                        if (kk < 16) pv(2 * kk + 1, pbh);
                    }
                    if constexpr (kQK) {
                        if (kk < 16) *reinterpret_cast<f16x8*>(tile + 16 * (f16_row(li) + 4 * kk + g)) = kv;
                    }
                    if constexpr (kQK && kPV) {
                        if (kk < 16) {
                            // product, 5 vector, product, 5 vector, product, the rest
                            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                            __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);
                            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                            __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);
                            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                        }
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
                if constexpr (kQK) {
                    if (it + 1 < n_tiles) {
                        // tile it+1 has landed: its code words are read while the
                        // softmax runs
                        wait_loads<(C::D - 1) * C::loads>();
                        read_stage(slot_base(it + 1));
                    }
                    softmax(it, s, p);
                }
            };
            wait_loads<(C::D - 1) * C::loads>();
            read_stage(slot_base(0));
            step(0, std::true_type{}, std::false_type{});
            for (int it = 1; it < n_tiles; ++it) step(it, std::true_type{}, std::true_type{});
            step(n_tiles, std::false_type{}, std::true_type{});
        } else {
            // raw bf16 rows: both products read the staged tile directly
            for (int it = 0; it < n_tiles; ++it) {
                // tile it has landed and every LDS access of the previous step is
                // done; then stage tile it+D into the slot tile it-1 used
                wait_loads<(C::D - 1) * C::loads>();
                issue_tile(it + C::D);
                const uint8_t* st = slot_base(it);
                bf16x8 kv[kQSteps];
#pragma unroll
                for (int kk = 0; kk < kQSteps; ++kk)
                    kv[kk] = *reinterpret_cast<const bf16x8*>(st + 16 * (bf_row(li) + 4 * kk + g));
                f32x4 s = f32x4{};
#pragma unroll
                for (int kk = 0; kk < kQSteps; ++kk) s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kv[kk], qf[kk], s, 0, 0, 0);
                float p[4];
                softmax(it, s, p);
                // aggregation: O^T[16 channels][16 rows] += V^T . P^T per block,
                // transposing reads eight blocks ahead of the products
                const uint8_t* vbase = st + 16 * bf_row(4 * g + (li >> 2)) + 8 * (li & 3);
                constexpr int kVAhead = 8;
                s16x4 vb[kVAhead];
#pragma unroll
                for (int m = 0; m < kVAhead; ++m) vb[m] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vbase + 32 * m));
                // protected rows: the weights to 16 significant bits, bf16(w) and the
                // bf16 rounding of the exact residual w - bf16(w), two products per
                // block; the BF16 cache: the bf16 weights alone (already rounded)
                const uint32_t h01 = pack_bf16x2(p[0], p[1]), h23 = pack_bf16x2(p[2], p[3]);
                const s16x4 pbb = __builtin_bit_cast(s16x4, make_uint2(h01, h23));
                const s16x4 pbl = __builtin_bit_cast(
                    s16x4, make_uint2(pack_bf16x2(p[0] - __uint_as_float(h01 << 16), p[1] - __uint_as_float(h01 & 0xFFFF0000u)),
                                      pack_bf16x2(p[2] - __uint_as_float(h23 << 16), p[3] - __uint_as_float(h23 & 0xFFFF0000u))));
#pragma unroll
                for (int m = 0; m < 32; ++m) {
                    acc[m] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vb[m % kVAhead], pbb, acc[m], 0, 0, 0);
                    if constexpr (kRing)
                        acc[m] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vb[m % kVAhead], pbl, acc[m], 0, 0, 0);
                    if (m + kVAhead < 32)
                        vb[m % kVAhead] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vbase + 32 * (m + kVAhead)));
                }
            }
        }
        // no direct-to-LDS load may outlive the workgroup's LDS
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    };

    if constexpr (!kProt) {
        int t_begin = 0, t_end = L;
        if (a.split_tokens != 0) {
            t_begin = max(split * a.split_tokens, 0);
            t_end = min(split * a.split_tokens + a.split_tokens, L);
        }
        const int lim = row_ok ? min(L - a.s_q + qi + 1, t_end) : t_begin;
        if (a.new_c != nullptr)
            narrow_append<KIND, false>(a, b, L, [&](int pos) { return pos >= t_begin && pos < t_end; }, lane);
        run(std::integral_constant<int, KIND>{}, std::false_type{}, t_begin, t_end, t_begin, lim);
    } else {
        // the tile list of mla_plan_splits_protected (32-key list tiles)
        const int sink = a.sink, recent = a.recent;
        const bool has_packed = L - recent > sink;
        const int pk0 = has_packed ? sink / 32 : 0;
        const int n_pk = has_packed ? (L - recent + 31) / 32 - pk0 : 0;
        const int n_prot = has_packed ? sink + recent : L;
        const int n_list = n_pk + (n_prot + 31) / 32;
        int u0 = 0, u1 = n_list;
        if (a.split_tokens != 0) {
            u0 = split * (a.split_tokens / 32);
            u1 = min(u0 + a.split_tokens / 32, n_list);
        }
        if constexpr (NCfg<KIND>::lowbit) {
            if (a.new_c != nullptr) {
                // list tile of position p: a packed position by its tile (from the
                // tile holding token `sink`), a protected one by its index among
                // the protected rows
                const int nsink = min(sink, L), r0 = max(sink, L - recent);
                auto reads = [&](int pos) {
                    const bool prot = pos < sink || pos >= L - recent;
                    const int u = prot ? n_pk + (min(pos, nsink) + max(0, pos - r0)) / 32 : pos / 32 - pk0;
                    return u >= u0 && u < u1;
                };
                narrow_append<KIND, true>(a, b, L, reads, lane);
            }
        }
        if (u0 < n_pk) {
            const int tb = 32 * (pk0 + u0);
            const int te = min(32 * (pk0 + min(u1, n_pk)), L - recent);
            const int lim = row_ok ? min(L - a.s_q + qi + 1, te) : tb;
            run(std::integral_constant<int, KIND>{}, std::false_type{}, tb, te, sink, lim);
        }
        if (u1 > n_pk) {
            ring_rows = sink + recent;
            ring_nsink = min(sink, L);
            const int r0 = max(sink, L - recent);
            ring_q0 = recent > 0 ? (r0 - sink) % recent : 0;
            int64_t pslot = a.prot_slot[b];
            pslot = pslot < 0 ? 0 : (pslot >= a.num_prot ? a.num_prot - 1 : pslot);
            ring_base = a.prot + pslot * ring_rows * 1152;
            auto below = [&](int x) { return min(max(x, 0), ring_nsink) + max(0, x - r0); };
            const int vb = 32 * (max(u0, n_pk) - n_pk);
            const int ve = min(32 * (u1 - n_pk), n_prot);
            const int lim = row_ok ? min(below(L - a.s_q + qi + 1), ve) : vb;
            run(std::integral_constant<int, KIND_BF16>{}, std::true_type{}, vb, ve, 0, lim);
        }
    }

    // ---- epilogue: this lane holds channels 16 m + 4 g .. +3 of row li
    const float l_tot = sum4(l_run);
    if (!row_ok) return;
    const int64_t orow = qrow;
    if (a.split_tokens == 0) {
        const float inv = l_tot > 0.0f ? 1.0f / l_tot : 0.0f;
        uint16_t* op = a.out + orow * kDc + 4 * g;
#pragma unroll
        for (int m = 0; m < 32; ++m)
            *reinterpret_cast<uint2*>(op + 16 * m) =
                make_uint2(pack_bf16x2(acc[m][0] * inv, acc[m][1] * inv), pack_bf16x2(acc[m][2] * inv, acc[m][3] * inv));
        if (a.lse != nullptr && g == 0)
            a.lse[orow] = l_tot > 0.0f ? (m_ref + log2f(l_tot)) * kLn2 : -INFINITY;
    } else {
        const int64_t prow = (static_cast<int64_t>(w) * a.s_q + qi) * a.H + h;
        const float f = m_true == -INFINITY ? 0.0f : exp2f(m_ref - m_true);
        const float inv = l_tot > 0.0f ? 1.0f / l_tot : 0.0f;
        uint16_t* op = a.part_o + prow * kDc + 4 * g;
#pragma unroll
        for (int m = 0; m < 32; ++m)
            *reinterpret_cast<uint2*>(op + 16 * m) =
                make_uint2(pack_f16x2(acc[m][0] * inv, acc[m][1] * inv), pack_f16x2(acc[m][2] * inv, acc[m][3] * inv));
        if (g == 0) {
            a.part_m[prow] = m_true * kLn2;
            a.part_s[prow] = l_tot * f;
        }
    }
}

template <bool kProt>
hipError_t launch(CacheKind kind, const DecodeArgs& a, hipStream_t stream) {
    if (a.num_work == 0) return hipSuccess;
    const LaunchEvents ev = take_launch_events();
    static_assert(kNarrowThreads == 64, "one wave per workgroup");
    const int64_t blocks = decode_workgroups(a.num_work, static_cast<int64_t>(a.s_q) * a.H, kRows);
    const dim3 grid(static_cast<unsigned>(blocks)), block(kNarrowThreads);
    switch (kind) {
        case KIND_C4R4: dispatch_decode(narrow_kernel<KIND_C4R4, kProt>, grid, block, stream, ev, a); break;
        case KIND_C2R4: dispatch_decode(narrow_kernel<KIND_C2R4, kProt>, grid, block, stream, ev, a); break;
        case KIND_C4R4P: dispatch_decode(narrow_kernel<KIND_C4R4P, kProt>, grid, block, stream, ev, a); break;
        case KIND_C2R4P: dispatch_decode(narrow_kernel<KIND_C2R4P, kProt>, grid, block, stream, ev, a); break;
        case KIND_BF16:
            if constexpr (kProt) return hipErrorInvalidValue;
            else dispatch_decode(narrow_kernel<KIND_BF16, false>, grid, block, stream, ev, a);
            break;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_decode_narrow(CacheKind kind, const DecodeArgs& a, hipStream_t stream) {
    return launch<false>(kind, a, stream);
}

hipError_t launch_decode_narrow_protected(CacheKind kind, const DecodeArgs& a, hipStream_t stream) {
    return launch<true>(kind, a, stream);
}

}  // namespace mla
