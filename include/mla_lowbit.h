/*
 * mla_lowbit.h -- C ABI of the low-bit MLA decode library for AMD MI355X (gfx950).
 *
 * The library computes absorbed-form Multi-head Latent Attention decode
 * (Sec. 2.1, eq. mla_compact) directly over a packed low-bit, paged cache of
 * the two MLA cache paths: the shared content latent C (d_c = 512 channels,
 * 4- or 2-bit codes) and the decoupled RoPE key K_P (d_r = 64 channels, 4-bit
 * codes).  Unpacking and dequantization are fused into attention
 * (Sec. 3.3; Appendix C.5, "Cache update and tile reuse").  The cache holds
 * latents already in the offline-fused coordinates, so no transformation is
 * applied here.
 *
 * Conventions for every entry point
 *   - Pointers named as device buffers must be device memory of the current
 *     HIP device; host pointers are marked "host".  The caller owns every
 *     buffer; the library allocates nothing and keeps no state between calls
 *     except, per host thread, a copy of the last HIP error and the event
 *     pair armed by mla_time_next_decode_launch (two handles, cleared by the
 *     decode dispatch that consumes them).
 *   - bf16 tensors are passed as uint16_t bit patterns.  All tensors are dense
 *     and row-major in the index order given, unless a stride is an argument.
 *     Query, output and partial tensors must be 16-byte aligned (else
 *     MLA_ENOTSUP).
 *   - GPU work is enqueued on `stream` (0 = the null stream) and is
 *     asynchronous; no call synchronizes.
 *   - Arguments are validated on the host before any HIP call.  Return codes:
 *       MLA_OK      success (work enqueued)
 *       MLA_EINVAL  a null pointer, a negative size or an ill-formed format
 *       MLA_ENOTSUP well-formed, but a shape the library does not implement
 *       MLA_EHIP    a HIP launch failed; mla_last_hip_error() gives the code
 *   - Launch sizes.  A dispatch counts its work items in 32 bits, so shapes
 *     whose launch would need more are refused with MLA_ENOTSUP: an append of
 *     more than 2^25 tokens in one call (also B * s_q new tokens of an
 *     append-and-decode call); a decode whose work items (B unsplit, else
 *     num_splits), rounded up to a multiple of 8, times ceil(s_q * H / 128)
 *     exceed 2^24 - 1 (the 16-row kernel, s_q * H <= 32: 2^26 - 1 times
 *     ceil(s_q * H / 16)); a combine of more than 2^24 - 8 rows (B * s_q * H).
 *   - Device-resident values (page ids, sequence lengths, split offsets) are
 *     not readable by the host without a synchronization and are preconditions:
 *     s_q <= seq_lens[b] <= max_pages_per_seq * page_size, 0 <= page id <
 *     num_pages, split_indptr as produced by mla_plan_splits, finite inputs.
 *     Kernels clamp every index into its buffer, so a violated precondition
 *     gives unspecified results but no out-of-bounds access.
 */
#ifndef MLA_LOWBIT_H
#define MLA_LOWBIT_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { MLA_OK = 0, MLA_EINVAL = 1, MLA_ENOTSUP = 2, MLA_EHIP = 3 };

/*
 * Cache format (Appendix C.4 "Affine group quantization", Appendix C.5
 * "Storage layout").  Supported: d_c = 512, d_r = 64, group = 64,
 * c_bits in {4, 2}, r_bits = 4, page_size a positive multiple of 32 (at most 2^20),
 * meta in {MLA_META_FP16, MLA_META_PAPER}.  The BF16 cache calls read only
 * d_c, d_r and page_size.
 */
enum { MLA_META_FP16 = 0, MLA_META_PAPER = 1 };

typedef struct mla_cache_format {
    int32_t d_c;        /* content latent channels                         */
    int32_t d_r;        /* decoupled RoPE key channels                     */
    int32_t group;      /* quantization group (consecutive channels)       */
    int32_t c_bits;     /* content code width                              */
    int32_t r_bits;     /* RoPE key code width                             */
    int32_t page_size;  /* tokens per page                                 */
    int32_t meta;       /* metadata storage, MLA_META_*                    */
} mla_cache_format;

/*
 * Packed page layout, MLA_META_FP16.  A page of P tokens holds four
 * token-major regions:
 *   codes_c[P][d_c*c_bits/8]   content codes
 *   codes_r[P][d_r*r_bits/8]   RoPE key codes
 *   meta_c [P][d_c/group]{fp16 scale, fp16 zero}
 *   meta_r [P][d_r/group]{fp16 scale, fp16 zero}
 * MLA_META_PAPER, the paper's storage (content scales in BF16, RoPE scales in
 * FP32; Appendix C.4 last sentence), holds three:
 *   codes_c[P][d_c*c_bits/8], codes_r[P][d_r*r_bits/8],
 *   meta   [P][32]: bf16 content scales [8] (bytes 0-15), byte content
 *          zero-points [8] (16-23), fp32 RoPE scale (24-27), byte RoPE
 *          zero-point (28), zero (29-31)
 * The page size is rounded up to 256 bytes; the cache is num_pages such
 * pages back to back from a 256-byte aligned base.  Codes form little-endian
 * 32-bit words of 32/bits consecutive channels (8 at 4 bits, 16 at 2 bits);
 * in a word, channel 2i occupies bits [bits*i, bits*(i+1)) and channel 2i+1
 * the same bits of the upper 16-bit half, so that a decoder extracts a
 * channel pair with one shift and one mask (a 4-bit word holds channels
 * 0, 2, 4, 6 in bytes 0-1 and 1, 3, 5, 7 in bytes 2-3).  Token t of page p is slot
 * p*P + t.  For d_c=512, d_r=64, P=64: 20736 bytes per page with 4-bit
 * content (324 B/token), 12544 with 2-bit content (196 B/token); with the
 * paper's metadata 20480 (320 B/token, the paper's figure) and 12288.
 * A BF16 cache page holds P rows of d_c + d_r bf16 values (73728 B at P=64).
 * Both return -1 for an invalid format.
 */
int64_t mla_lowbit_page_bytes(const mla_cache_format* f);
int64_t mla_bf16_page_bytes(const mla_cache_format* f);

/*
 * Quantize-and-append (Appendix C.4 quantizer; Appendix C.5 "Cache update and
 * tile reuse": quantization, integer packing, slot-mapped page insertion).
 * For each of n tokens and each group of 64 consecutive channels of both
 * paths, in IEEE fp32 with round-half-to-even:
 *   s = max(xmax - xmin, 1e-8) / m     (m = 2^bits - 1, a true division)
 *   z = clip(rint(-xmin / s), 0, m)
 *   q = clip(rint(x / s + z), 0, m)    (divide, then add: two roundings)
 * stores q packed and the metadata: fp16(s), fp16(z) (fp16 subnormals kept)
 * under MLA_META_FP16; bf16(s) (round-half-to-even) for content groups, s
 * itself (fp32) for the RoPE group and z as a byte under MLA_META_PAPER.
 *   c_kv     device, bf16 [n][c_kv_stride], first d_c used
 *   k_rope   device, bf16 [n][k_rope_stride], first d_r used (post-RoPE key)
 *   slot_mapping device, int64 [n]: destination slot; a negative slot skips
 *            the token; a slot >= num_pages*page_size is skipped too
 *   cache    device, num_pages packed pages (layout above)
 * Codes and metadata are bit-identical to the quantizer above.  n = 0 is a
 * no-op.  Tokens with equal slots race; the last writer is unspecified.
 */
int mla_lowbit_quant_append(const mla_cache_format* f,
                            const uint16_t* c_kv, int64_t c_kv_stride,
                            const uint16_t* k_rope, int64_t k_rope_stride,
                            const int64_t* slot_mapping, int32_t n,
                            void* cache, int64_t num_pages, hipStream_t stream);

/*
 * Append into the BF16 comparison cache: row = [c_kv(d_c) | k_rope(d_r)],
 * copied bit for bit.  Arguments as for mla_lowbit_quant_append.
 */
int mla_bf16_append(const mla_cache_format* f,
                    const uint16_t* c_kv, int64_t c_kv_stride,
                    const uint16_t* k_rope, int64_t k_rope_stride,
                    const int64_t* slot_mapping, int32_t n,
                    void* cache, int64_t num_pages, hipStream_t stream);

/*
 * Split planner (host only; no HIP call).  Split k of sequence b covers keys
 * [k*split_tokens, min((k+1)*split_tokens, seq_lens[b])), so sequence b has
 * ceil(seq_lens[b] / split_tokens) splits and its partials live at indices
 * split_indptr[b] .. split_indptr[b+1]-1 (Appendix C.5, "Global attention
 * normalization": any partition of the keys merges to the same result).
 *   seq_lens     host, int32 [B], each >= 1
 *   split_indptr host, int32 [B+1], written
 * Returns the total number of splits (>= 0), or -MLA_EINVAL / -MLA_ENOTSUP
 * (split_tokens must be a positive multiple of 32).
 */
int32_t mla_plan_splits(const int32_t* seq_lens, int32_t B, int32_t split_tokens,
                        int32_t* split_indptr);

/*
 * Low-bit decode attention (Sec. 2.1, eq. mla_compact, up to the latent
 * aggregation O_h = A_h C; value/output projections stay outside).
 * For sequence b of length L = seq_lens[b], query token i < s_q sits at
 * position L - s_q + i and sees keys t <= L - s_q + i (causal within the
 * s_q new tokens).  For head h:
 *   z_t = softmax_scale * (q_lat[b,i,h,:] . C_hat[t,:] + q_rope[b,i,h,:] . K_hat[t,:])
 *   out[b,i,h,:] = sum_t softmax(z)_t C_hat[t,:],   lse[b,i,h] = ln sum_t e^{z_t}
 * where C_hat, K_hat are dequantized from the packed cache with the stored
 * scale and zero: x_hat = scale * (q - zero).
 *   q_lat   device, bf16 [B][s_q][H][d_c]  absorbed content query
 *   q_rope  device, bf16 [B][s_q][H][d_r]  RoPE-encoded query
 *   cache   device, packed pages; num_pages of them
 *   block_table device, int32 [B][max_pages_per_seq]: page id of each
 *           page_size-token block of each sequence
 *   seq_lens    device, int32 [B]
 *   H       heads, a positive multiple of 16; s_q in {1, 2}; softmax_scale > 0
 *   B = 0 is a no-op after the scalar arguments are checked (pointers may be NULL)
 * Unsplit (split_tokens == 0): writes out (device, bf16 [B][s_q][H][d_c]) and,
 *   if lse != NULL, lse (device, fp32 [B][s_q][H]); split_indptr,
 *   num_splits and part_* are ignored.
 * Split (split_tokens > 0): split_indptr (device, int32 [B+1]) and
 *   num_splits = split_indptr[B] come from mla_plan_splits; writes for every
 *   split j and row (i, h) the partials of Appendix C.5 "Global attention
 *   normalization", in natural-log units, with the weighted sum stored
 *   normalized by the split's own exponential sum:
 *     part_m[j][i][h]    = max_t z_t over the split's visible keys      (fp32)
 *     part_s[j][i][h]    = sum_t e^{z_t - part_m}                        (fp32)
 *     part_o[j][i][h][:] = fp16( sum_t e^{z_t - part_m} C_hat[t,:] / part_s )
 *   (device; a split with no visible key gives (-inf, 0, 0)); the paper's
 *   unnormalized sum is part_s * part_o.  out and lse are not touched -- call
 *   mla_splitkv_combine.
 * Scores and latent aggregation run as fp16 matrix products with fp32
 * accumulation: the dequantized cache (x_hat, one fp16 rounding) and the
 * softmax weights are fp16 operands, so queries and x_hat must lie within the
 * fp16 range.  Past it the result is not finite, never a plausible value: a
 * row that sees a key with |x_hat| >= 65520 in some channel comes out NaN or
 * inf (output and lse), and a row of the same launch work item that does not
 * see the key is non-finite in that key's overflowing channels.  Under
 * MLA_META_PAPER the RoPE scale enters as fp16(scale) (a
 * second rounding of the RoPE key, relative 2^-11).  The output is rounded to
 * bf16 once.
 */
int mla_lowbit_decode_attn(const mla_cache_format* f,
                           const uint16_t* q_lat, const uint16_t* q_rope,
                           const void* cache, int64_t num_pages,
                           const int32_t* block_table, int32_t max_pages_per_seq,
                           const int32_t* seq_lens, int32_t B, int32_t s_q, int32_t H,
                           float softmax_scale,
                           int32_t split_tokens, const int32_t* split_indptr, int32_t num_splits,
                           uint16_t* out, float* lse,
                           float* part_m, float* part_s, uint16_t* part_o,
                           hipStream_t stream);

/*
 * Same computation over a BF16 cache (the unquantized comparison; row layout
 * in mla_bf16_page_bytes).  Arguments as for mla_lowbit_decode_attn.  The
 * products run in bf16 (cache rows and queries exact), the softmax weights
 * rounded to bf16.  With split partials, the cache values must lie within the
 * fp16 range (part_o is fp16).
 */
int mla_bf16_decode_attn(const mla_cache_format* f,
                         const uint16_t* q_lat, const uint16_t* q_rope,
                         const void* cache, int64_t num_pages,
                         const int32_t* block_table, int32_t max_pages_per_seq,
                         const int32_t* seq_lens, int32_t B, int32_t s_q, int32_t H,
                         float softmax_scale,
                         int32_t split_tokens, const int32_t* split_indptr, int32_t num_splits,
                         uint16_t* out, float* lse,
                         float* part_m, float* part_s, uint16_t* part_o,
                         hipStream_t stream);

/*
 * The step's append and decode in one call (Appendix C.5, "Cache update and
 * tile reuse": the writer's quantization and insertion, then the fused
 * decode): equivalent to mla_lowbit_quant_append (or mla_bf16_append) of the
 * n = B * s_q new tokens followed by mla_lowbit_decode_attn (or
 * mla_bf16_decode_attn), with identical cache bytes and outputs.  New token
 * (b, i), row b * s_q + i of c_kv / k_rope (bf16, strides as for the append),
 * is position seq_lens[b] - s_q + i of sequence b and is written at slot
 * slot_mapping[b * s_q + i] (device, int64; < 0 skips the token), which must
 * be that position's slot under block_table (a device-resident precondition).
 * The writer runs inside the decode launch: the workgroups that read a new
 * token's tile quantize and store it first.  Arguments and errors as for the
 * two calls.
 */
int mla_lowbit_append_decode_attn(const mla_cache_format* f,
                                  const uint16_t* c_kv, int64_t c_kv_stride,
                                  const uint16_t* k_rope, int64_t k_rope_stride,
                                  const int64_t* slot_mapping,
                                  const uint16_t* q_lat, const uint16_t* q_rope,
                                  void* cache, int64_t num_pages,
                                  const int32_t* block_table, int32_t max_pages_per_seq,
                                  const int32_t* seq_lens, int32_t B, int32_t s_q, int32_t H,
                                  float softmax_scale,
                                  int32_t split_tokens, const int32_t* split_indptr, int32_t num_splits,
                                  uint16_t* out, float* lse,
                                  float* part_m, float* part_s, uint16_t* part_o,
                                  hipStream_t stream);
int mla_bf16_append_decode_attn(const mla_cache_format* f,
                                const uint16_t* c_kv, int64_t c_kv_stride,
                                const uint16_t* k_rope, int64_t k_rope_stride,
                                const int64_t* slot_mapping,
                                const uint16_t* q_lat, const uint16_t* q_rope,
                                void* cache, int64_t num_pages,
                                const int32_t* block_table, int32_t max_pages_per_seq,
                                const int32_t* seq_lens, int32_t B, int32_t s_q, int32_t H,
                                float softmax_scale,
                                int32_t split_tokens, const int32_t* split_indptr, int32_t num_splits,
                                uint16_t* out, float* lse,
                                float* part_m, float* part_s, uint16_t* part_o,
                                hipStream_t stream);

/*
 * Split-KV combine (Appendix C.5, "Global attention normalization"):
 *   m = max_j part_m[j],  s = sum_j e^{part_m[j]-m} part_s[j],
 *   out = (sum_j e^{part_m[j]-m} part_s[j] part_o[j]) / s  as bf16,
 *   lse = m + ln s
 * over the splits j of each sequence; splits with part_m = -inf are skipped.
 *   part_*  device, as written by the decode call
 *   split_indptr, num_splits  as passed to the decode call (num_splits =
 *           split_indptr[B], from mla_plan_splits; host value, it chooses
 *           how the rows' splits are spread over the waves)
 *   out     device, bf16 [B][s_q][H][d_c];  lse device fp32 [B][s_q][H] or NULL
 * Every row must have at least one split with a visible key.  B = 0 is a no-op.
 */
int mla_splitkv_combine(const float* part_m, const float* part_s, const uint16_t* part_o,
                        const int32_t* split_indptr, int32_t num_splits, int32_t B, int32_t s_q, int32_t H,
                        int32_t d_c, uint16_t* out, float* lse, hipStream_t stream);

/*
 * BF16 protection of sink and recent tokens (Sec. 3.3; Appendix C.5, "BF16
 * protection and cache lifecycle", "Global attention normalization",
 * "Storage layout").  Besides the packed copy of every token, the writer keeps
 * the pre-quantization bf16 content latent and RoPE key of the first `sink`
 * and the last `recent` tokens of every sequence.  For a sequence of length L
 * the protected positions are
 *   P_L = {0 .. min(sink, L) - 1}  U  {max(0, L - recent) .. L - 1}
 * (overlap counted once; the paper's policy is sink = 4, recent = 128).
 * Attention reads every token once: bf16 values for positions in P_L, the
 * packed copy otherwise, all in one softmax.  Constraints: sink, recent >= 0,
 * 1 <= sink + recent <= 65536.
 *
 * Protection buffer of one sequence: sink + recent rows of d_c + d_r bf16
 * values ([c_kv | k_rope], 1152 B at d_c = 512, d_r = 64; 152,064 B for the
 * paper's policy).  Row p holds position p < sink; row
 * sink + (p - sink) mod recent holds position p >= sink (a ring: the token
 * entering the window overwrites the one leaving it, which attention then
 * reads from its packed copy).  Rows not yet written are never read.
 */
typedef struct mla_protect_policy {
    int32_t sink;       /* leading tokens kept in bf16                    */
    int32_t recent;     /* most recent tokens kept in bf16                */
} mla_protect_policy;

/* Bytes of one sequence's protection buffer; -1 for an invalid format or
 * policy (low-bit formats only). */
int64_t mla_protect_buffer_bytes(const mla_cache_format* f, const mla_protect_policy* p);

/*
 * Quantize-and-append with protection: exactly mla_lowbit_quant_append for
 * the packed cache, and in the same pass the bf16 row of every appended token
 * that is protected once the call is done, i.e. position p < sink, or
 * L - recent <= p < L with L = seq_lens[b] the sequence's length after the
 * call (a prefill thus writes only the rows that stay protected, and no two
 * tokens of one call share a row).  Rows are copied bit for bit.
 *   token_seq  device, int32 [n]: sequence b of each token (outside [0, B):
 *              no protection write)
 *   positions  device, int32 [n]: the token's position in its sequence
 *   seq_lens   device, int32 [B]: lengths after this call
 *   prot_slot  device, int32 [B]: protection buffer index of each sequence
 *              (outside [0, num_prot): no protection write)
 *   prot       device, num_prot buffers of mla_protect_buffer_bytes each,
 *              back to back, 16-byte aligned
 * A token with a skipped slot (negative or past the cache) is skipped
 * entirely.  Other arguments and errors as for mla_lowbit_quant_append.
 */
int mla_lowbit_quant_append_protected(const mla_cache_format* f, const mla_protect_policy* p,
                                      const uint16_t* c_kv, int64_t c_kv_stride,
                                      const uint16_t* k_rope, int64_t k_rope_stride,
                                      const int64_t* slot_mapping, int32_t n,
                                      void* cache, int64_t num_pages,
                                      const int32_t* token_seq, const int32_t* positions,
                                      const int32_t* seq_lens, const int32_t* prot_slot, int32_t B,
                                      void* prot, int64_t num_prot, hipStream_t stream);

/*
 * Split planner for protected decode (host only).  Under protection the keys
 * of a sequence of length L are processed as a list of 32-key tiles: the
 * packed tiles first -- from the tile holding token `sink` through token
 * L - recent - 1, when L - recent > sink -- then ceil(n_prot / 32) tiles of
 * protected rows (n_prot = sink + recent, or L when every token is
 * protected).  Split k of a sequence covers list tiles
 * [k * split_tokens / 32, (k + 1) * split_tokens / 32); the partials of all
 * splits merge to the single softmax (Appendix C.5).  Returns the total
 * number of splits, or -MLA_EINVAL / -MLA_ENOTSUP as mla_plan_splits.
 */
int32_t mla_plan_splits_protected(const int32_t* seq_lens, int32_t B, int32_t split_tokens,
                                  const mla_protect_policy* p, int32_t* split_indptr);

/*
 * Low-bit decode attention under protection: as mla_lowbit_decode_attn, with
 * positions in P_L read as bf16 rows from the sequence's protection buffer
 * (prot_slot[b], clamped into [0, num_prot)) instead of the packed cache.
 * Split partials follow mla_plan_splits_protected; mla_splitkv_combine
 * merges them unchanged.  Products over protected rows run in bf16 (rows and
 * queries exact, weights rounded to bf16), over packed rows in fp16 as in
 * mla_lowbit_decode_attn.  Precondition: the buffer holds every position of
 * P_L (written by mla_lowbit_quant_append_protected).
 *   prot  device, num_prot protection buffers (16-byte aligned)
 */
int mla_lowbit_decode_attn_protected(const mla_cache_format* f, const mla_protect_policy* p,
                                     const uint16_t* q_lat, const uint16_t* q_rope,
                                     const void* cache, int64_t num_pages,
                                     const int32_t* block_table, int32_t max_pages_per_seq,
                                     const int32_t* seq_lens, int32_t B, int32_t s_q, int32_t H,
                                     float softmax_scale,
                                     const void* prot, int64_t num_prot, const int32_t* prot_slot,
                                     int32_t split_tokens, const int32_t* split_indptr, int32_t num_splits,
                                     uint16_t* out, float* lse,
                                     float* part_m, float* part_s, uint16_t* part_o,
                                     hipStream_t stream);

/*
 * The step's append and decode under protection in one call (Appendix C.5,
 * "BF16 protection and cache lifecycle", "Cache update and tile reuse"):
 * equivalent to mla_lowbit_quant_append_protected of the n = B * s_q new
 * tokens -- token (b, i), row b * s_q + i of c_kv / k_rope, at position
 * seq_lens[b] - s_q + i of sequence b and slot slot_mapping[b * s_q + i] --
 * followed by mla_lowbit_decode_attn_protected, with identical cache bytes,
 * protection buffer rows and outputs.  A buffer index outside [0, num_prot)
 * skips the token's protection row (as the writer does) and is clamped for
 * the decode (as the decode does).  The writer runs inside the decode
 * launch: the workgroups that read a new token quantize and store it first
 * (its protection row too, for a token protected after the step).  Arguments
 * and errors as for the two calls; prot is written (device, 16-byte aligned).
 * Precondition: the sequences' protection buffers are distinct (a sequence
 * whose index is clamped onto another's buffer may read that buffer's new
 * rows before or after they are written).
 */
int mla_lowbit_append_decode_attn_protected(const mla_cache_format* f, const mla_protect_policy* p,
                                            const uint16_t* c_kv, int64_t c_kv_stride,
                                            const uint16_t* k_rope, int64_t k_rope_stride,
                                            const int64_t* slot_mapping,
                                            const uint16_t* q_lat, const uint16_t* q_rope,
                                            void* cache, int64_t num_pages,
                                            const int32_t* block_table, int32_t max_pages_per_seq,
                                            const int32_t* seq_lens, int32_t B, int32_t s_q, int32_t H,
                                            float softmax_scale,
                                            void* prot, int64_t num_prot, const int32_t* prot_slot,
                                            int32_t split_tokens, const int32_t* split_indptr, int32_t num_splits,
                                            uint16_t* out, float* lse,
                                            float* part_m, float* part_s, uint16_t* part_o,
                                            hipStream_t stream);

/*
 * Per-layer persistent cache bytes of one request of L tokens
 * (Appendix C.5, eq. physical_cache_storage):
 *   ceil(L / page_size) * (page bytes + 8) + protection buffer bytes
 * with this library's page geometry for `f`, the 8-byte reverse page mapping
 * a paging allocator keeps per physical page (counted by the equation, not
 * allocated by this library), and the protection buffer of `p` (NULL: no
 * protection).  With MLA_META_PAPER, c_bits = 4 and the paper's policy this is
 * the paper's M_C4R4(L); for a BF16 format (c_bits = 16) it returns the
 * equation's M_BF16(L) = ceil(L / page_size) * mla_bf16_page_bytes.
 * Returns -1 for an invalid format, policy, L < 0, or a byte count beyond
 * INT64_MAX.
 */
int64_t mla_persistent_cache_bytes(const mla_cache_format* f, const mla_protect_policy* p, int64_t L);

/*
 * Decode attention without any allocation, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops, harnesses that
 * forbid hipMalloc): mla_lowbit_decode_attn followed by mla_splitkv_combine,
 * with the split partials held in storage the library owns -- one static
 * device array per GPU, for at most 65536 partial rows (num_splits * s_q * H;
 * 64.5 MiB, held from module load until the process ends).  The caller passes
 * inputs and the final outputs only.  Arguments as for mla_lowbit_decode_attn
 * without part_m / part_s / part_o: split_tokens = 0 decodes unsplit (no
 * storage used); split_tokens > 0 needs split_indptr and num_splits from
 * mla_plan_splits and writes out (bf16 [B][s_q][H][d_c]) and lse (NULL
 * allowed) as the combine does.  Returns MLA_ENOTSUP when num_splits * s_q * H
 * exceeds 65536, before any HIP call.  No hipMalloc, hipFree or allocating
 * library routine is called.  Every call on one GPU shares that GPU's storage
 * (each call writes every partial it reads, so nothing carries over between
 * calls): calls that overlap on one GPU, on different streams or host
 * threads, race and give unspecified results.
 */
int mla_lowbit_decode_attn_noalloc(const mla_cache_format* f,
                                   const uint16_t* q_lat, const uint16_t* q_rope,
                                   const void* cache, int64_t num_pages,
                                   const int32_t* block_table, int32_t max_pages_per_seq,
                                   const int32_t* seq_lens, int32_t B, int32_t s_q, int32_t H,
                                   float softmax_scale,
                                   int32_t split_tokens, const int32_t* split_indptr, int32_t num_splits,
                                   uint16_t* out, float* lse, hipStream_t stream);

/* Human-readable name of a status code (static string). */
const char* mla_status_str(int status);

/* hipError_t of this thread's last MLA_EHIP return (0 if none). */
int mla_last_hip_error(void);

/* Measurement hook (not part of the computation).  The next decode-kernel
 * dispatch made by the calling host thread -- from any *_decode_attn entry
 * point, the append-and-decode ones included -- carries `start` and `stop`
 * on its own dispatch packet (hipExtLaunchKernel), so that
 * hipEventElapsedTime(start, stop) is that kernel's execution time, free of
 * the dispatch latency that events recorded around the call would include.
 * Writer and combine launches do not consume it.  One-shot: the pair is
 * cleared by that dispatch (a call that returns an error or has no work
 * dispatches nothing and leaves it set); passing two nulls clears it.
 * Both events belong to the caller, must stay valid until the dispatch has
 * completed, and must be both null or both non-null (else MLA_EINVAL). */
int mla_time_next_decode_launch(hipEvent_t start, hipEvent_t stop);

#ifdef __cplusplus
}
#endif

#endif /* MLA_LOWBIT_H */
