/*
 * wushkv.h -- C ABI of the WUSH-KV online hot path on AMD Instinct MI355X
 * (gfx950).
 *
 * WUSH-KV ("KV Cache Quantization with Data-Adaptive Transforms") caches, for
 * every key/value head h of a grouped-query attention layer, the quantised
 * transformed keys Q(T_K(h) k) and values Q(T_V(h) v) (Eq. (3)).  The value
 * transform is folded into the projection weights offline, so values arrive
 * here already transformed; the key transform is applied online after norm
 * and RoPE.  Queries are compensated with T_K^{-T} (Alg. 2, step 3).  The
 * quantiser is the per-token percentile-clipped affine quantiser of Eq. (7)
 * or, per cache, the RMS-scaled symmetric QuEST quantiser of Eq. (5) (the
 * one the paper's analysis and reconstruction-error experiments use), and
 * the cache keeps two bf16 windows, a sink and a recent window, with
 * quantisation in multiples of S_flush (Sec. 4.4, Alg. 2).
 *
 * Entry points:
 *   wushkv_append            Alg. 2 steps 3 (keys), 4 and 7-11
 *   wushkv_decode_attention  Alg. 2 steps 3 (queries) and 5, Eq. (2)
 *   wushkv_dequant           the reconstruction of Eq. (7) for stored tokens
 *   wushkv_wush_transform    the transform T of Eq. (1) (calibration, Alg. 1)
 *
 * Conventions
 *   - Every pointer is a DEVICE pointer unless marked (host), and must be
 *     16-byte aligned.  bf16 and fp16 values are passed as uint16_t bit
 *     patterns.
 *   - The caller owns all memory.  The library never allocates device memory
 *     on these paths, never frees and never synchronises; all work is
 *     enqueued on the caller's stream.  The only library state the compute
 *     calls touch is a per-variant cache of the decode kernel's occupancy,
 *     filled on first use (thread-safe: racing first calls store the same
 *     value); calls on different streams with disjoint caches may therefore
 *     run concurrently.  The opt-in kernel timer (wushkv_timing_enable) is
 *     global and not thread-safe.
 *   - Argument checks happen on the host before anything is enqueued; a
 *     failing check returns a negative status and enqueues nothing.
 *   - Device-resident values (seq_len, quant_end, n_new, page_table) cannot
 *     be checked on the host.  The kernels never access memory outside the
 *     bounds the descriptor states (a page index outside [0, n_pages) or a
 *     logical page beyond max_pages_per_seq is skipped), but the results of
 *     a call that breaks the capacity contract are unspecified.
 *
 * Status codes: WUSHKV_OK (0) or a negative WUSHKV_E* value;
 * wushkv_status_string() names them.
 */
#ifndef WUSHKV_H
#define WUSHKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t *wushkv_stream_t; /* same type as hipStream_t */

enum {
    WUSHKV_OK = 0,
    WUSHKV_EINVAL = -1,       /* null pointer or value out of range */
    WUSHKV_EUNSUPPORTED = -2, /* valid per the paper but not built here */
    WUSHKV_EWORKSPACE = -3,   /* workspace too small */
    WUSHKV_ELAUNCH = -4,      /* the HIP runtime refused a launch */
    WUSHKV_ENODEVICE = -5     /* no usable gfx950 device */
};

#define WUSHKV_PAGE_TOKENS 64
#define WUSHKV_ABI_VERSION 4

/* Per-token quantisers (wushkv_cache.codec). */
enum {
    WUSHKV_CODEC_PCLIP = 0, /* Eq. (7): percentile-clipped affine */
    WUSHKV_CODEC_QUEST = 1  /* Eq. (5): RMS-scaled, symmetric, bin centres */
};

/*
 * Cache descriptor.  Sizes are host values; the arrays are device memory.
 *
 * Positions p of sequence b are counted from 0.  With S = seq_len[b] and
 * S_quant = quant_end[b] (the paper's inclusive 1-based boundary is the same
 * integer as this exclusive 0-based end):
 *   p <  s_sink                       sink window, bf16, slot p
 *   s_sink <= p < max(S_quant,s_sink) quantised (Eq. (7)), in pages
 *   max(S_quant, s_sink) <= p < S     recent window, bf16, ring slot
 *                                     s_sink + (p - s_sink) mod R,
 *                                     R = win_slots - s_sink
 *
 * Quantised positions live in pages of 64 tokens.  Logical page i of
 * sequence b holds positions s_sink + 64 i .. s_sink + 64 i + 63 and is
 * physical page page_table[b * max_pages_per_seq + i].
 *
 * pages: uint8 [n_pages][n_kv_heads][page_bytes], page_bytes =
 *   wushkv_page_bytes(head_dim, bits) = 64 * (2 * head_dim * sb / 8 + 8), where
 *   sb = bits for 2- and 4-bit codes and sb = 4 for 3-bit codes: a 3-bit code
 *   is stored in the 4-bit format below, in a 4-bit field whose top bit is
 *   zero (136 bytes per token-head at d = 128 instead of the dense 104).
 *   In the rest of this layout description, bits stands for sb.
 *   One (page, head) block is, in order:
 *     K codes   8 * head_dim * bits bytes
 *     V codes   8 * head_dim * bits bytes
 *     K params  64 tokens x 4 bytes: fp16 scale, fp16 zero (token t at 4 t)
 *     V params  64 tokens x 4 bytes, same form
 *   Reconstruction of a stored entry: x = scale * code + zero (fp32 fma),
 *   for both codecs (the QuEST codec stores its bin-centre offset as the
 *   zero, see wushkv_append).
 *
 *   Code words.  Both code regions are arrays of little-endian 32-bit
 *   words; a word holds B = 32 / bits codes.  Each region is a sequence of
 *   16-byte chunks: chunk q holds words 4q .. 4q+3 of every "lane" in lane
 *   order, so the k-th word of lane L is word (k / 4) * 4 * lanes + 4 L +
 *   k % 4 of the region (lanes = 16 * head_dim / 32 for K, 64 for V).
 *
 *   K region: lanes L = 16 j + n (j < head_dim / 32, n = 0..15) of
 *   4 * bits words each.  Word k = bits * t + w of lane L (t = 0..3,
 *   w = 0..bits-1) holds token 4 n + t, channels 32 j + B w + e for
 *   e = 0..B-1; code e = h * B/2 + i (h = 0, 1) sits at bit
 *   2 * bits * i + bits * h.  A mask then spreads a word, or the word
 *   shifted right by bits, into one code per nibble (2-bit) or per byte
 *   (4-bit): the fp4 / fp8 operands of the decode kernel's scaled matrix
 *   instruction.
 *
 *   V region: element e of a word is slot i = e % 8 of operand o = e / 8
 *   and sits at bit 16 * (i % 2) + F(o, i / 2): slot pairs share a field
 *   position, the even slot in the low half word.  F = (6, 10, 8, 12) for
 *   operand 0 and (2, 0, 4, 14) for operand 1 of a 2-bit word, F =
 *   (4, 0, 8, 12) for a 4-bit word (one operand).  With
 *   nw = head_dim * bits / 128, the region holds 64 lanes L = 16 j + m
 *   (j = 0..3, m = 0..15) of 4 nw words each; word k = kc * 2nw + u of
 *   lane L (kc = 0..1, u = 0..2nw-1) holds
 *     token    32 kc + 8 j + i
 *     channel  16 nt + m,  nt = u * (B / 8) + o
 *   (the operand order of the 16x16x32 fp16 product: a few shifts and one
 *   mask per operand register move each code near the top of an fp16
 *   fraction).
 *
 * win_k: bf16 [batch][n_kv_heads][win_slots][head_dim]   (token-major)
 * win_v: bf16 [batch][n_kv_heads][head_dim][win_slots]   (channel-major)
 *   Keys in transformed coordinates (T_K k, rounded to bf16), values as
 *   given (already transformed).  Slots that hold no live position may hold
 *   any bit pattern, NaN included; they are never read into a result.
 */
typedef struct wushkv_cache {
    int32_t batch;             /* sequences, >= 1 */
    int32_t n_kv_heads;        /* >= 1 */
    int32_t head_dim;          /* 64 or 128 */
    int32_t bits;              /* 2, 3 or 4, for keys and values (3: stored as 4) */
    int32_t s_sink;            /* >= 0 */
    int32_t s_keep;            /* >= 0 */
    int32_t s_flush;           /* >= 1 */
    int32_t win_slots;         /* multiple of 64, >= s_sink + max(1, s_keep + s_flush - 1) */
    int32_t max_pages_per_seq; /* row length of page_table, >= 0 */
    int32_t n_pages;           /* pages in the pool, >= 0 */
    float kappa_k;             /* Eq. (7) clipping quantile for keys, (0, 1] (PCLIP) */
    float kappa_v;             /* same for values */
    int32_t codec;             /* WUSHKV_CODEC_PCLIP or WUSHKV_CODEC_QUEST */
    float quest_alpha;         /* Eq. (5) clip multiplier alpha_b > 0, finite (QUEST);
                                  wushkv_quest_alpha(bits) is the paper's choice */
    uint8_t *pages;
    int32_t *page_table;       /* [batch][max_pages_per_seq] */
    uint16_t *win_k;
    uint16_t *win_v;
    int32_t *seq_len;          /* [batch] S; read and advanced by wushkv_append */
    int32_t *quant_end;        /* [batch] S_quant; read and advanced by wushkv_append */
    int32_t *commit;           /* [batch] caller-owned scratch, zero before the first
                                  append: the append's workgroups count their arrivals
                                  here so that the last of each sequence advances S and
                                  S_quant (an append of more than 64 tiles per sequence
                                  advances them in a one-workgroup launch of its own
                                  instead); every completed call leaves it zero */
} wushkv_cache;

/* Bytes of one (page, head) block, or 0 for unsupported (head_dim, bits):
 * head_dim 64 or 128, bits 2, 3 or 4. */
size_t wushkv_page_bytes(int32_t head_dim, int32_t bits);

/*
 * wushkv_append -- append new tokens to every sequence (Alg. 2 steps 3-4)
 * and quantise the newly eligible positions (Alg. 2 steps 7-11).
 *
 *   k_new   bf16 [batch][max_new][n_kv_heads][head_dim]: keys after headwise
 *           norm and RoPE.  Row t of sequence b is position seq_len[b] + t.
 *   v_new   bf16, same shape: values, already in transformed coordinates.
 *   n_new   int32 [batch]: tokens appended to each sequence, 0..max_new.
 *   max_new (host) upper bound of n_new, sizes the grid; 0 is a no-op.
 *   t_k     bf16 [n_kv_heads][head_dim][head_dim] row-major: the stored key
 *           is k~ = T_K k, i.e. k~[o] = sum_i t_k[o][i] k[i], accumulated in
 *           fp32 and rounded once to bf16 (Alg. 2 step 3).
 *   k_tilde_out  nullable; bf16 of k_new's shape: receives k~ for every
 *           appended token (a verification aid; costs one extra write).
 *
 * Effect, per sequence b with S = seq_len[b], S' = n_new[b]:
 *   S_new = S + S'; S_start = max(S_quant, s_sink);
 *   S_quant_new = max(S_quant, S_start + floor((S_new - s_keep - S_start)
 *                 / s_flush) * s_flush)          (floor toward -infinity);
 *   positions [S_start, S_quant_new) are quantised from their bf16 values
 *   with the cache's codec; new positions below s_sink go to the sink, new
 *   positions at or after S_quant_new go to the recent ring;
 *   seq_len[b] = S_new; quant_end[b] = S_quant_new.
 *
 * Codecs, per group x (one token-head of keys or values, fp32 from bf16,
 * every step one correctly rounded operation):
 *   PCLIP (Eq. (7)): q = type-7 quantile of |x| at kappa_k / kappa_v;
 *     x_min = max(min x, -q), x_max = min(max x, q);
 *     scale = fp16(fp32((x_max - x_min) / (2^bits - 1))), zero = fp16(x_min);
 *     code = clamp(rne((x - zero) / scale), 0, 2^bits - 1), with the
 *     division as a product by 1 / scale (codes 0 when scale is 0).
 *   QUEST (Eq. (5)): with h = 2^(bits-1),
 *     step = fp32(2 quest_alpha / (2^bits - 1) * sqrt(sum_i x_i^2 / head_dim))
 *     evaluated in fp64 (the sum in any order), scale = fp16(step),
 *     zero = fp16(scale * (1/2 - h));
 *     code = clamp(floor(x * (1 / scale)) + h, 0, 2^bits - 1)  (code h when
 *     scale is 0), so that scale * code + zero is the bin centre
 *     scale (floor(x / scale) + 1/2) up to the fp16 rounding of the zero.
 * Capacity (caller's contract): page_table holds valid pages for every
 *   logical page the new S_quant reaches.
 */
int wushkv_append(const wushkv_cache *c,
                  const uint16_t *k_new, const uint16_t *v_new,
                  const int32_t *n_new, int32_t max_new,
                  const uint16_t *t_k, uint16_t *k_tilde_out,
                  wushkv_stream_t stream);

/*
 * wushkv_append_norm_rope -- wushkv_append with Alg. 2 step 1 fused in
 * front of it: the keys arrive as projected, BEFORE the headwise
 * normalisation and the rotary embedding of Eq. (2), K = RoPE(Norm(W_K^T X)).
 *
 *   k_raw   bf16 [batch][max_new][n_kv_heads][head_dim]: projected keys.
 *           Row t of sequence b is position s = seq_len[b] + t.
 *   norm_gain  fp32 [head_dim] device, or NULL for a gain of one.
 *   norm_eps   (host) >= 0, added to the mean square inside the root.
 *   rope_table fp32 [rope_positions][head_dim] device: for position s,
 *              column j < head_dim/2 holds cos(s w_j) and column
 *              head_dim/2 + j holds sin(s w_j) (the model's own rotary table).
 *   rope_positions (host) rows of rope_table; must be at least the cache's
 *              capacity, max_pages_per_seq * 64 + s_sink.
 *   The other arguments are wushkv_append's.
 *
 * Per key row x (fp32 from bf16), each step rounded to nearest-even fp32:
 *   r = 1 / sqrt(sum_i x_i^2 / head_dim + norm_eps)   (sum in any order);
 *   y_i = (x_i * r) * gain_i;
 *   for j < h = head_dim/2, with c, s the table's cos and sin at (s, j):
 *     k'_j = y_j c - y_{j+h} s,   k'_{j+h} = y_{j+h} c + y_j s;
 * k' is rounded once to bf16 and then appended exactly as wushkv_append
 * appends k_new (k~ = T_K k', windows, quantisation).  This is the RMS form
 * of Norm and the pairwise rotation R(s w_j) of the coordinate pairs
 * (j, j + h) written in the paper's appendix on RoPE-commuting transforms.
 * Returns WUSHKV_EINVAL for a null table, a negative or non-finite eps or a
 * table shorter than the capacity, besides wushkv_append's checks.
 */
int wushkv_append_norm_rope(const wushkv_cache *c,
                            const uint16_t *k_raw, const uint16_t *v_new,
                            const int32_t *n_new, int32_t max_new,
                            const uint16_t *t_k,
                            const float *norm_gain, float norm_eps,
                            const float *rope_table, int32_t rope_positions,
                            uint16_t *k_tilde_out, wushkv_stream_t stream);

/*
 * wushkv_decode_attention -- one decode query per query head (Eq. (2)).
 *
 *   q          bf16 [batch][n_q_heads][head_dim]: queries after norm and RoPE.
 *              Query head (h, g) is flat index h * G + g, G = n_q / n_kv.
 *   n_q_heads  (host) multiple of n_kv_heads; G <= 8.
 *   max_seq_len (host) >= every seq_len[b]; sizes the split-K grid.
 *   t_k_inv    fp32 [n_kv_heads][head_dim][head_dim] row-major T_K^{-1}:
 *              the compensated query is q~[j] = sum_i q[i] t_k_inv[i][j]
 *              (the row form of T_K^{-T} q, Eq. (3)).
 *   sm_scale   softmax scale 1 / tau (usually 1 / sqrt(head_dim)).
 *   out        fp32 [batch][n_q_heads][head_dim]: attention output in
 *              transformed value coordinates (the folded W_O consumes it).
 *              A sequence with seq_len 0 gets zeros.
 *   workspace  device scratch of at least wushkv_decode_workspace_bytes();
 *              contents need not be initialised and are clobbered.
 *
 * The query of sequence b attends to all positions [0, seq_len[b]): sink
 * and recent windows at bf16, the middle through the stored codes.
 * Returns WUSHKV_EUNSUPPORTED (and the workspace size is 0) when max_seq_len
 * would need a page run longer than 64 pages per wave, beyond about
 * 16.7 M tokens (chunk attention: about 4.19 M).
 */
int wushkv_decode_attention(const wushkv_cache *c,
                            const uint16_t *q, int32_t n_q_heads,
                            int32_t max_seq_len,
                            const float *t_k_inv, float sm_scale,
                            float *out, void *workspace,
                            size_t workspace_bytes,
                            wushkv_stream_t stream);

/* Workspace bytes wushkv_decode_attention needs for these sizes (0 on bad
 * arguments). */
size_t wushkv_decode_workspace_bytes(const wushkv_cache *c,
                                     int32_t n_q_heads, int32_t max_seq_len);

/*
 * wushkv_decode_attention_noalloc -- wushkv_decode_attention for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation): the same arguments without the
 * workspace, the same kernels and the same results.  Its workspace is a
 * static device array of WUSHKV_NOALLOC_SCRATCH_BYTES inside the library,
 * one per GPU, held until the process ends; its address is looked up on the
 * first call on each device (hipGetSymbolAddress, no allocation).  The call
 * allocates and frees nothing.
 *   - A call whose plan needs more than WUSHKV_NOALLOC_SCRATCH_BYTES
 *     (wushkv_decode_workspace_bytes for the same arguments) returns
 *     WUSHKV_EWORKSPACE and enqueues nothing: for example batch 64, 32 query
 *     heads at 32768 tokens need about 14 MB, well inside the limit.
 *   - Nothing in the array has to start at zero: every call writes all it
 *     reads (the q~ rows and every split's partial) before reading it.
 *   - Every call on one GPU shares that GPU's array, which keeps the last
 *     call's contents: calls that overlap on one GPU (different streams, or
 *     host threads, without ordering between them) race on it and must not
 *     be issued.
 * Returns WUSHKV_ENODEVICE when no device is current or the array cannot be
 * located, besides wushkv_decode_attention's statuses.
 */
#define WUSHKV_NOALLOC_SCRATCH_BYTES (32u << 20)
int wushkv_decode_attention_noalloc(const wushkv_cache *c, const uint16_t *q,
                                    int32_t n_q_heads, int32_t max_seq_len,
                                    const float *t_k_inv, float sm_scale, float *out,
                                    wushkv_stream_t stream);

/*
 * wushkv_decode_step -- one decode step of Alg. 2 (S' = 1) in the
 * algorithm's own order, in two launches on the stream:
 *   1. each sequence's new token is appended at bf16 (steps 3-4: k~ = T_K k
 *      into its window slot) and attention runs over the cache including it
 *      (step 5), the positions that this step moves out of the recent window
 *      still at bf16;
 *   2. the attention splits are merged into out, those positions are
 *      quantised into their pages (steps 7-11) and seq_len / quant_end
 *      advance.
 * On a step that quantises nothing the output and the cache equal those of
 * wushkv_append followed by wushkv_decode_attention; on a step that does,
 * that pair (which flushes first) attends to the flushed positions through
 * their codes instead.
 *
 *   k_new, v_new  bf16 [batch][n_kv_heads][head_dim]: each sequence's new key
 *              (after norm and RoPE) and value.
 *   n_new      int32 [batch] device: 1 appends sequence b's token, 0 leaves the
 *              sequence as it is (its query still attends); clamped to [0, 1].
 *   t_k        bf16 [n_kv_heads][head_dim][head_dim] T_K, 16-byte aligned.
 *   max_seq_len (host) >= every seq_len[b] + n_new[b]; sizes the split-K grid.
 *   The other arguments are wushkv_decode_attention's; the workspace needs
 *   wushkv_decode_workspace_bytes() for the same max_seq_len.
 * The position seq_len[b] must lie inside the cache's capacity, as for
 * wushkv_append.  Returns WUSHKV_EUNSUPPORTED when win_slots - s_sink <
 * s_keep + s_flush (the new token's ring slot could still be live), and
 * WUSHKV_EINVAL for null or misaligned new-token arguments, besides
 * wushkv_decode_attention's checks; nothing is enqueued then.
 */
int wushkv_decode_step(const wushkv_cache *c, const uint16_t *k_new, const uint16_t *v_new,
                       const int32_t *n_new, const uint16_t *t_k, const uint16_t *q,
                       int32_t n_q_heads, int32_t max_seq_len, const float *t_k_inv,
                       float sm_scale, float *out, void *workspace, size_t workspace_bytes,
                       wushkv_stream_t stream);

/*
 * wushkv_chunk_attention -- attention of a chunk of new tokens per sequence
 * (Alg. 2 step 5 with S' > 1): Eq. (2) with its causal mask, over the cache
 * as stored after the append that brought the chunk.
 *
 *   q          bf16 [batch][max_tok][n_q_heads][head_dim]: queries after norm
 *              and RoPE; row t of sequence b is its chunk token t.
 *   n_tok      int32 [batch] device, or NULL for max_tok everywhere: the
 *              chunk of sequence b is its last n_tok[b] positions (clamped to
 *              [0, min(max_tok, seq_len[b])]); token t sits at position
 *              p = seq_len[b] - n_tok[b] + t and attends to positions [0, p].
 *   max_tok    (host) 1 <= max_tok <= s_keep: the chunk lies inside the
 *              recent window, so every quantised position precedes it.
 *   out        fp32 [batch][max_tok][n_q_heads][head_dim]; rows beyond a
 *              sequence's chunk are zero.
 *   The other arguments are wushkv_decode_attention's; the workspace needs
 *   wushkv_chunk_workspace_bytes().  Decode is the case max_tok = 1.
 */
int wushkv_chunk_attention(const wushkv_cache *c, const uint16_t *q,
                           const int32_t *n_tok, int32_t max_tok, int32_t n_q_heads,
                           int32_t max_seq_len, const float *t_k_inv, float sm_scale,
                           float *out, void *workspace, size_t workspace_bytes,
                           wushkv_stream_t stream);

/* Workspace of wushkv_chunk_attention, or 0 for invalid arguments. */
size_t wushkv_chunk_workspace_bytes(const wushkv_cache *c, int32_t n_q_heads,
                                    int32_t max_tok, int32_t max_seq_len);

/*
 * wushkv_dequant -- reconstruct stored entries x = scale * code + zero
 * (Eq. (7), last term) of sequence b, positions [start, start + count).
 *   k_out, v_out  fp32 [n_kv_heads][count][head_dim] (either may be null;
 *                 16-byte aligned, or the call fails with WUSHKV_EINVAL).
 * Positions must satisfy start >= s_sink and start + count <= s_sink + 64 *
 * max_pages_per_seq (host-checked).  The pages are decoded as stored,
 * whether or not quant_end has reached the position; a logical page whose
 * physical index lies outside [0, n_pages) yields NaN.
 */
int wushkv_dequant(const wushkv_cache *c, int32_t b, int32_t start,
                   int32_t count, float *k_out, float *v_out,
                   wushkv_stream_t stream);

/* Name of a status code. */
const char *wushkv_status_string(int status);

/*
 * wushkv_wush_transform -- the WUSH transform of Eq. (1), T = Wush(M, H,
 * gamma), for `count` independent pairs (one per key or value head, Eq. (4),
 * Alg. 1):
 *   L L^T = H + gamma tr(H)/d I,  U Lam U^T = L^T (M + gamma tr(M)/d I) L,
 *   c = ((1 + gamma) tr(M))^(1/2) tr(Lam^(1/2))^(-1/2),
 *   T = c Had Lam^(-1/4) U^T L^T   (Had: normalised Sylvester Hadamard).
 * The eigenpairs are taken in ascending order of Lam, and each eigenvector's
 * sign makes the largest-magnitude entry of L u_k positive (first on ties);
 * T depends on both and the paper fixes neither.
 *
 *   m, h        fp32 [count][d][d] device, row-major, symmetric (only the
 *               lower triangle is read): the Gram matrix of the tensor
 *               quantised and the Hessian of its perturbation.  Both damped
 *               matrices must be positive definite.
 *   count       >= 0 pairs; 0 is a no-op.
 *   d           64 or 128.
 *   gamma       (host) damping ratio >= 0, finite (the paper uses 1e-2).
 *   t_out       fp32 [count][d][d]: T (k~ = T k); convert to bf16 for
 *               wushkv_append's t_k.
 *   t_inv_out   nullable fp32 [count][d][d]: T^{-1}, as wushkv_decode_attention
 *               takes it.
 *   sweeps_out  nullable int32 [count]: Jacobi sweeps each pair took, or -1
 *               when a damped matrix was not positive definite (its outputs
 *               are then NaN).
 * Computed in fp32 with a one-sided Jacobi eigensolver; see the source for
 * the method.  Errors: WUSHKV_EINVAL for a negative count, bad gamma, null or
 * unaligned pointers; WUSHKV_EUNSUPPORTED for other d.
 */
int wushkv_wush_transform(const float *m, const float *h, int32_t count, int32_t d,
                          float gamma, float *t_out, float *t_inv_out,
                          int32_t *sweeps_out, wushkv_stream_t stream);

/*
 * wushkv_quest_alpha -- the clip multiplier alpha_b of Eq. (5): the endpoint
 * of the 2^bits evenly spaced levels that minimises the mean squared error of
 * rounding a standard Gaussian to the nearest level (Sec. 4.3).  Host only;
 * returns NaN for bits outside 1..8.
 */
double wushkv_quest_alpha(int32_t bits);

/*
 * wushkv_read_probe -- a plain streaming read of `bytes` (a positive multiple
 * of 65536) at `buf`: the reference for how much of the nominal HBM peak a
 * kernel that only reads reaches on this device.  mode 0 reads with 16-byte
 * vector loads into registers, mode 1 with 16-byte direct-to-LDS loads, the
 * path of the decode kernel's pages.  sink: uint32 [bytes / 65536] device,
 * receives one XOR of the data per 64 KB block.  Measurement aid only.
 */
int wushkv_read_probe(const void *buf, size_t bytes, int32_t mode, uint32_t *sink,
                      wushkv_stream_t stream);

/* WUSHKV_ABI_VERSION of the loaded library. */
int wushkv_abi_version(void);

/*
 * Kernel timing for measurement.  While enabled (slots > 0), each of the
 * next `slots` launches the library makes records a pair of HIP events on
 * its stream that the runtime stamps when that kernel starts and when it
 * ends (hipExtLaunchKernelGGL); disabling (slots = 0) releases them.  This
 * is the only library state and it is not thread-safe; leave it off in
 * production.  wushkv_timing_read synchronises on the recorded events and
 * returns, for launches whose kernel name contains `name_substr` (all
 * launches for NULL), the count and the summed milliseconds.  Reading does
 * not clear the record; calling wushkv_timing_enable again does.
 */
int wushkv_timing_enable(int32_t slots);
int wushkv_timing_read(const char *name_substr, int32_t *count, double *total_ms);
/* Launches recorded so far, and the kernel name and milliseconds of the
 * index-th of them (synchronising on its events; WUSHKV_EINVAL for an index
 * out of range). */
int wushkv_timing_count(void);
int wushkv_timing_launch(int32_t index, const char **name, double *ms);

#ifdef __cplusplus
}
#endif

#endif /* WUSHKV_H */
