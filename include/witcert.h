/*
 * witcert.h -- C-ABI of the WitCert hot path on MI355X (gfx950).
 *
 * WitCert meters, per (layer, head, decode step), a provable bound on how far
 * the softmax attention over the compressed cache can move, in total-variation
 * distance, from the one over the uncompressed cache (paper:
 * "WitCert: Sound Runtime Risk Observability and Gating for KV-Cache
 * Quantization").  This library implements the meter loop of Sec. 6:
 *
 *   write path  wc_quantize_write   dithered INT8 (Sec. 4.2) or raw fp8 cast,
 *                                   plus the residual witness (Sec. 4.1, Eq. witness)
 *               wc_witness          witness of any cache-preserving scheme (Sec. 4.1)
 *               wc_select_outlier_pairs
 *                                   the fixed outlier RoPE pairs of each KV head that the
 *                                   INT8 key cache keeps in fp16 (Sec. 4.2, Sec. 6.2)
 *   read path   wc_metered_decode_attention
 *                                   GQA decode attention over the compressed cache
 *                                   fused with the Tier-A meter (Theorem black-box
 *                                   logit bound + Theorem sound replacement), split
 *                                   over the KV axis and merged under the softmax
 *                                   LSE weights (Sec. 6.2, SGLang decode kernel)
 *   gate        wc_gate             meter (raw score when tau >= 1) > tau, routed per
 *                                   KV head by any-of-G (Sec. 4.3, Sec. 5)
 *               wc_exact_decode_attention
 *                                   exact attention from an uncompressed bf16 cache for
 *                                   the routed heads (the fallback of the meter loop)
 *   step        wc_step_metered_decode_gate, wc_step_certified_decode,
 *               wc_step_certified_decode_speculative
 *                                   a decode step's token write with the read path and
 *                                   gate (and, certified, the exact fallback) fused
 *               wc_block_repair     repair of routed heads from the exact cache at block
 *                                   granularity (Sec. 6.3)
 *               wc_repair_write_back
 *                                   persistent repair: repaired pages are served from the
 *                                   exact cache by every later decode (Sec. 6, Sec. 6.3)
 *
 * Conventions shared by every entry point
 *   - All tensor pointers are DEVICE pointers owned by the caller; the library
 *     never allocates, frees, synchronizes or reads results back.  Scratch
 *     memory is a caller-provided workspace sized by wc_decode_workspace_size.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and
 *     returns immediately; results are valid once the stream reaches them.
 *     Every call is safe to capture in a HIP graph (no host synchronization,
 *     no memset nodes).
 *   - Return value: WC_OK (0) or a negative WC_E* code; nothing is enqueued
 *     when an argument check fails.  wc_strerror names the codes.  No C++
 *     exception crosses this boundary.  The library keeps no state (apart from
 *     the static scratch of wc_step_metered_decode_gate_noalloc) and is
 *     thread-safe.
 *   - Pointers must be 16-byte aligned; shapes are row-major, innermost last.
 *   - Preconditions not checked on the device: finite inputs, |x| <= 8.28e6
 *     (keeps fp16 scales finite; the decode handles every fp16 value scale and
 *     every finite bf16 value of the exact cache), |x| <= 448 for the fp8 cache,
 *     |q| < 65504,
 *     block-table entries < num_blocks, slots < num_blocks * 16, every
 *     seq_lens[b] <= max_seq_len and <= max_blocks_per_seq * 16, outlier pair
 *     lists ascending and distinct (out-of-range pair indices are clamped, so a
 *     bad list gives wrong values, never a fault), |x| <= 65504 on bypassed
 *     channels.
 */
#ifndef WITCERT_H
#define WITCERT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---------------------------------------------------- */
#define WC_OK              0
#define WC_EINVAL         -1   /* null/misaligned pointer, bad shape or enum    */
#define WC_EUNSUPPORTED   -2   /* valid but not built (e.g. head_dim 96)        */
#define WC_EHIP           -3   /* the HIP runtime rejected a launch             */
#define WC_EWORKSPACE     -4   /* workspace smaller than wc_decode_workspace_size */
#define WC_ESCRATCH       -5   /* sizes need more than WC_NOALLOC_SCRATCH_BYTES  */

/* ---- element types ---------------------------------------------------- */
#define WC_F32   0
#define WC_BF16  1
#define WC_F16   2

/* ---- cache kinds ------------------------------------------------------ */
#define WC_KIND_INT8_DITHER  0   /* int8 codes + fp16 per-token scales + fp16 key witness */
#define WC_KIND_FP8_RAW      1   /* fp8 E4M3 raw cast (no scale) + fp16 key witness       */
#define WC_KIND_BF16         2   /* uncompressed bf16 (the exact fallback cache)          */

/* ---- RoPE pair layouts (they decide the band map) ---------------------- */
#define WC_ROPE_HALF         0   /* pair j = channels (j, j + d/2)  (rotate-half)  */
#define WC_ROPE_INTERLEAVED  1   /* pair j = channels (2j, 2j + 1)                 */

#define WC_BLOCK_TOKENS 16       /* tokens per paged block */

/*
 * One layer's paged cache.  Slot s lives in block s/16 at offset s%16.
 * Memory layout (sizes from wc_cache_bytes):
 *   k_data,
 *   v_data     [num_blocks][n_kv_heads][page], a page (16 tokens, 16*head_dim elements
 *              of E bytes: 1 for the quantized kinds, 2 for BF16) stored as 16-byte
 *              pieces [CL][4][16][16 bytes], CL = head_dim*E/64: piece (i, g, r) at byte
 *              ((i*4 + g)*16 + r)*16 of the page, so that each 16-byte load of a wave
 *              covers whole cache lines.
 *              k_data: piece (i, g, r) = bytes (g*CL + i)*16 .. +15 of token r's row
 *                (its head_dim elements in channel order): token r, channel c at byte
 *                ((p%CL*4 + p/CL)*16 + r)*16 + (c*E)%16, p = c*E/16.
 *              v_data: token quad q (tokens 4q .. 4q+3) has a row of head_dim x 4
 *                elements (channel c, token 4q+u at element 4c + u); piece (i, q, r) =
 *                bytes (r*CL + i)*16 .. +15 of that row: token t, channel c at byte
 *                ((p%CL*4 + t/4)*16 + p/CL)*16 + b%16, b = (4c + t%4)*E, p = b/16.
 *   k_scale,
 *   v_scale    [num_blocks][n_kv_heads][16] fp16              INT8_DITHER only, else NULL;
 *              with group_scales [num_blocks][n_kv_heads][16][head_dim/32] fp16
 *   k_witness  [num_blocks][n_kv_heads][16][n_bands] fp16     NULL for BF16
 *   k_outlier  [num_blocks][n_kv_heads][16][2m] fp16          keys of the bypassed pairs
 *              (m = n_outlier_pairs > 0 only, else NULL)
 *   v_resid,
 *   v_norm     [num_blocks][n_kv_heads][16] fp16              value side (optional, both or
 *              neither, quantized kinds only): ||vhat_t - v_t|| rounded up and ||v_t||
 *              rounded down, from float64 norms (Sec. 3 output bound; Sec. 4.2 value side)
 * Element type of k_data/v_data: int8 code stored excess-128, i.e. the byte code + 128
 * (INT8_DITHER; codes lie in [-127, 127]), E4M3 byte (FP8_RAW), bf16 (BF16).
 * Band b holds the channels of RoPE pairs b*P .. b*P+P-1, P = head_dim/(2*n_bands)
 * (Sec. 4.1; Lemma RoPE band unitarity).  `seed` keys the Philox dither; `layer`
 * enters its counter (Sec. 6.2: counter (layer, kv_head, slot, channel)).
 *
 * Outlier-pair bypass (INT8_DITHER; Sec. 4.2 outlier RoPE pairs, Sec. 6.2
 * fixed-channel bypass): a fixed set of m RoPE pairs per KV head,
 * outlier_pairs[h][0..m-1] (ascending, distinct, < head_dim/2; see
 * wc_select_outlier_pairs), is kept in fp16 instead of INT8: both channels of
 * each pair leave the key's amax, their codes are 0, and their values, rounded to
 * nearest fp16, are stored in k_outlier in the order (pair 0 first channel, pair 0
 * second channel, pair 1 first, ...); the pair channels are (j, j + head_dim/2)
 * for WC_ROPE_HALF and (2j, 2j + 1) for WC_ROPE_INTERLEAVED.  Values stay within
 * +-65504.  Values are not bypassed.  m is even, 0 <= m <= 16.
 *
 * Group scales (INT8_DITHER; Sec. 6.2 storage side: per token, per group of 32
 * channels; Table 4: 272 bytes per token-head for K + V): with group_scales = 1,
 * every token has one fp16 scale per 32-channel group g (channels 32g..32g+31) and
 * tensor, s_g = fp16_round_up(fl32(amax_g / 126.5)) over the group's quantized
 * channels (bypassed channels leave amax_g), stored in k_scale / v_scale in place
 * of the token scale; codes use fl32(1/s_g).  The decode of a group-scaled cache
 * takes the same paths as a per-token one (matrix cores for head_dim 128 and bf16
 * queries); its value operands carry one more fp16 rounding there (outputs within
 * 2e-3 of the oracle, relative to the largest output; logits and meters exact).
 *
 * Persistent repair (quantized kinds; the meter loop's gate, Sec. 6: repaired slots
 * keep their exact values and their witnesses are cleared; Sec. 6.3 gated evaluation
 * (c): each slot is repaired once and skipped afterwards): repaired[blk * n_kv_heads +
 * h] != 0 marks page blk of KV head h as served from the exact store, whose bf16
 * pages (the k_data / v_data of a WC_KIND_BF16 cache with the same num_blocks,
 * n_kv_heads and head_dim, written by wc_quantize_write_pair) are exact_k /
 * exact_v.  Every decode of the cache reads a marked page's keys and values from
 * the exact store with bound 0 (no witness, no radius, no value residual), for
 * every token of the page, also tokens written after the mark; block repair ranks
 * only blocks that hold an unmarked token.  wc_repair_write_back sets the marks
 * (and zeroes the marked slots' witness); the caller allocates the array (one
 * byte per page and KV head) and zeroes it with the cache.  With repaired NULL,
 * exact_k and exact_v are ignored.
 */
typedef struct wc_cache {
    int32_t  kind;          /* WC_KIND_*                                       */
    int32_t  head_dim;      /* 64 or 128                                       */
    int32_t  n_kv_heads;    /* 1 .. 65535                                      */
    int32_t  n_bands;       /* B, head_dim % (2*B) == 0, 1 <= B <= 16           */
    int32_t  rope_layout;   /* WC_ROPE_*                                       */
    int32_t  layer;         /* 0 .. 65535, Philox counter field                */
    int64_t  num_blocks;    /* pages of 16 slots                               */
    uint64_t seed;          /* Philox4x32-10 key (low word = key[0])           */
    void *k_data, *v_data, *k_scale, *v_scale, *k_witness;
    int32_t  n_outlier_pairs;          /* m: bypassed RoPE pairs per KV head (0: none) */
    int32_t  group_scales;             /* 1: one fp16 scale per 32-channel group, 0: per token */
    const int32_t* outlier_pairs;      /* [n_kv_heads][m] device, or NULL when m == 0  */
    void*    k_outlier;                /* see above, or NULL when m == 0               */
    void    *v_resid, *v_norm;          /* value side, or both NULL                     */
    uint8_t* repaired;                 /* persistent repair marks, or NULL (see below)  */
    const void *exact_k, *exact_v;     /* the exact store's k_data / v_data, with marks */
} wc_cache;

const char* wc_strerror(int status);
int         wc_version(void);   /* 100*major + minor */

/*
 * Bytes of each array of a cache (k_data, v_data, k_scale, v_scale, k_witness,
 * k_outlier, v_resid, v_norm) written to sizes[0..7]; returns their sum, 0 on bad
 * arguments.  The "exact byte account" of the cache (Sec. 5 memory saving; Sec.
 * 6.2 acceptance; Table 4: 2 bytes per scale, one per token or one per 32-channel
 * group and side when group_scales != 0; Table 6: 4m bytes per token and KV head
 * for the bypassed pairs; 2 + 2 bytes for the value side when value_side != 0).
 */
size_t wc_cache_bytes(int kind, int64_t num_blocks, int n_kv_heads, int head_dim,
                      int n_bands, int n_outlier_pairs, int value_side, int group_scales,
                      size_t sizes[8]);

/*
 * Fixed outlier-pair set of each KV head (Sec. 6.2 fixed-channel bypass; Sec. 4.2
 * pairs selected by energy): the m RoPE pairs j of largest energy
 * E_j = sum_i ||(k_i)_pair j||^2 over the n_tok rows given (e.g. a prefill),
 * ties to the lower j, written in ascending order to pairs_out[h][0..m-1].
 * The energies are summed in float64, over fixed row chunks in a fixed order, so
 * the result does not depend on scheduling.  RoPE does not change E_j, so the set
 * is the same before and after the rotation.
 *   k          [n_tok][n_kv_heads][head_dim], in_dtype WC_F32 or WC_BF16, n_tok >= 1
 *   m          0 <= m <= head_dim/2 (m = 0 writes nothing)
 *   pairs_out  [n_kv_heads][m] int32 device
 *   ws         device workspace of ws_bytes >= wc_select_workspace_size(n_tok,
 *              n_kv_heads, head_dim) bytes, 8-byte aligned, no initialization needed
 */
size_t wc_select_workspace_size(int64_t n_tok, int n_kv_heads, int head_dim);
int wc_select_outlier_pairs(const void* k, int in_dtype, int64_t n_tok, int n_kv_heads,
                            int head_dim, int rope_layout, int m, int32_t* pairs_out, void* ws,
                            size_t ws_bytes, void* stream);

/*
 * Write path (Sec. 4.2 subtractive dither; Sec. 6.2 research kernels and storage
 * side; Sec. 4.1 Eq. witness).  For every token i < n_tok and KV head h:
 *   INT8_DITHER: s = fp16_round_up(fl32(amax/126.5)) per (token, head, tensor), or
 *                per 32-channel group with group scales;
 *                xi_c = (u_c - 127.5)/256 with u_c the Philox4x32-10 byte of channel c
 *                (key = seed, counter = (c/16, slot lo, slot hi, layer<<16 | h)),
 *                shared by K and V; code = rint_even(fl32(fl32(x*inv) + xi)) with
 *                inv = fl32(1/s) (of the channel's group);
 *                with bypassed pairs (n_outlier_pairs > 0) the amax and the codes
 *                skip their channels and k_outlier receives fp16(x) of them;
 *   FP8_RAW:     code = E4M3(x), nearest-even, saturating at +-448;
 *   BF16:        x rounded to bf16 (nearest-even);
 * and, except for BF16, the key witness w_b = ||(khat - k)_b|| rounded up to fp16
 * (the residual, its squares, sums and square root in float64; one round-up), and,
 * when the cache has a value side, ||vhat - v|| rounded up and ||v|| rounded down to
 * fp16 (float64 norms).
 *   k, v          [n_tok][n_kv_heads][head_dim], in_dtype WC_F32 or WC_BF16 (post-RoPE keys)
 *   slot_mapping  [n_tok] int64 device; a slot < 0 or >= num_blocks * 16 skips the token
 *                 (no write outside the cache)
 */
int wc_quantize_write(const wc_cache* cache, const void* k, const void* v, int in_dtype,
                      const int64_t* slot_mapping, int64_t n_tok, void* stream);

/*
 * wc_quantize_write into `cache` (INT8_DITHER or FP8_RAW) and into the bf16 exact
 * cache `exact` that the fallback reads (Sec. 6: the gated heads are recomputed
 * from an exact copy), in one pass over k and v.  The result equals
 * wc_quantize_write(cache, ...) followed by wc_quantize_write(exact, ...).
 * exact must be a BF16 cache with the same head_dim and n_kv_heads and at least
 * cache->num_blocks blocks; both are addressed by the same slot_mapping.
 */
int wc_quantize_write_pair(const wc_cache* cache, const wc_cache* exact, const void* k, const void* v,
                           int in_dtype, const int64_t* slot_mapping, int64_t n_tok, void* stream);

/*
 * Black-box witness (Sec. 4.1, Tier A scope: any scheme that writes back a
 * per-token reconstruction): w[i][b] = fp16_round_up(||(xhat_i - x_i)_b||).
 *   x, xhat  [n_vec][head_dim] in x_dtype / xhat_dtype (WC_F32, WC_BF16 or WC_F16)
 *   w_out    [n_vec][n_bands] fp16 bits
 */
int wc_witness(const void* x, int x_dtype, const void* xhat, int xhat_dtype, int64_t n_vec,
               int head_dim, int n_bands, int rope_layout, uint16_t* w_out, void* stream);

/*
 * Workspace bytes needed by wc_metered_decode_attention / wc_exact_decode_attention
 * for these sizes.  split_tokens as passed to the decode call (0 = library choice).
 * The workspace holds the per-split partial records, for the fused gate one int32
 * per (sequence, KV head), and the meter numerators of the block segments that
 * wc_block_repair reads; it needs no initialization.  Calls that share a
 * workspace must not run concurrently.
 */
size_t wc_decode_workspace_size(int batch, int n_q_heads, int n_kv_heads, int head_dim,
                                int64_t max_seq_len, int split_tokens);

/*
 * Tokens per KV split that the decode calls use for these sizes: split_tokens
 * rounded up to a multiple of 64, or, for 0, the library's choice (about 512
 * workgroups over the batch's KV heads, at least 256 tokens).  With
 * total_tokens > 0 (the sum of the batch's
 * sequence lengths, known to the caller on the host) and split_tokens = 0 the
 * choice balances the workgroups over the total instead of the longest
 * sequence: pass the result as split_tokens to the decode calls and
 * wc_decode_workspace_size for ragged batches (the same value as the default for
 * equal lengths).  Returns 0 for invalid sizes.
 */
int wc_decode_split_tokens(int batch, int n_kv_heads, int64_t max_seq_len, int64_t total_tokens,
                           int split_tokens);

/*
 * Tokens per KV split for wc_step_certified_decode_speculative, whose one launch
 * holds the metered and the exact workgroups of every split (twice a decode's):
 * as wc_decode_split_tokens with about 256 instead of 512 (sequence, KV head,
 * split) workgroups, so that the launch fills the GPU's two workgroups per compute
 * unit once rather than twice with a ragged second round (at 32k tokens x 4
 * sequences: 2112 tokens, 16 splits, against 1088 for the decode calls).  A
 * throughput choice only: any split gives results within rounding of any other.
 * Pass the result as split_tokens to the speculative step and to
 * wc_certified_workspace_size.  Returns 0 for invalid sizes.
 */
int wc_speculative_split_tokens(int batch, int n_kv_heads, int64_t max_seq_len, int64_t total_tokens,
                                int split_tokens);

/*
 * Metered decode attention (the read path of the meter loop, Sec. 6).  For each
 * sequence b and query head h (KV head h / (n_q_heads / n_kv_heads)), over the
 * seq_lens[b] tokens whose slots are block_table[b][t/16]*16 + t%16:
 *   khat_t, vhat_t  reconstructions (INT8: s*(code - xi), xi regenerated from the slot;
 *                   the stored fp16 value on the channels of bypassed pairs)
 *   ptilde         = softmax(sm_scale * q . khat_t)
 *   out[b][h]      = sum_t ptilde_t vhat_t
 *   c_t            = sm_scale * sum_b ||q_b|| w_{t,b}      (Theorem black-box logit bound)
 *   A - 1          = sum_t ptilde_t (e^{c_t} - 1)            (Theorem sound replacement)
 *   raw[b][h]      = (A - 1)(A + 1)/2, +inf on overflow
 *   meter[b][h]    = min(1, raw)                             (Sec. 4.3)
 * The KV axis is split into chunks whose partial (max, sum, A-1 numerator, output)
 * are merged under the LSE weights; A merges exactly like the output (Sec. 6.2).
 *   q            [batch][n_q_heads][head_dim], q_dtype WC_F32 or WC_BF16
 *   block_table  [batch][max_blocks_per_seq] int32 entries in [0, cache->num_blocks);
 *                the kernels never read outside the cache, but the result for a
 *                token whose entry lies outside it is unspecified
 *   seq_lens     [batch] int32 (>= 0)
 *   max_seq_len  host-side upper bound of seq_lens (sizes the split grid)
 *   out          [batch][n_q_heads][head_dim], out_dtype WC_F32 or WC_BF16
 *   meter, raw   [batch][n_q_heads] fp32 (raw may be NULL)
 *   split_tokens tokens per KV split, multiple of 64 (0 = library choice)
 *   ws           workspace of ws_bytes >= wc_decode_workspace_size(...)
 * A sequence with seq_lens[b] == 0 gets out = 0, meter = raw = 0.
 * cache->kind must be INT8_DITHER or FP8_RAW.
 */
int wc_metered_decode_attention(const wc_cache* cache, const void* q, int q_dtype, int batch,
                                int n_q_heads, const int32_t* block_table,
                                int max_blocks_per_seq, const int32_t* seq_lens,
                                int64_t max_seq_len, float sm_scale, void* out, int out_dtype,
                                float* meter, float* raw, int split_tokens, void* ws,
                                size_t ws_bytes, void* stream);

/*
 * Tier-B certified decode (Sec. 4.2, Tier B: Lemma uniform sub-Gaussian proxy and
 * the request-level budget) over an INT8_DITHER cache: as
 * wc_metered_decode_attention, with the witness bound c_t replaced by the
 * sub-Gaussian radius of the subtractive-dither residual,
 *   u_t = (alpha_h + beta_h) * s_t,
 *   alpha_h = sm_scale * ||q_h|| * sqrt(2 log(2 S_b / delta_loc) / 12),
 *   beta_h  = sm_scale * ||q_h||_1 / 256 (bound on the residual mean of the 8-bit
 *             dither lattice),
 * s_t the token's stored key scale and S_b = seq_lens[b].  With bypassed pairs,
 * ||q_h|| and ||q_h||_1 are taken over the other channels and u_t gains the fp16
 * rounding bound of the bypassed ones,
 *   sm_scale * sum_{c bypassed} |q_c| (2^-11 |khat_{t,c}| + 2^-25).
 * A = sum_t ptilde_t e^{u_t}, raw = (A^2 - 1)/2, meter = min(1, raw).  No witness
 * is read (k_witness may be NULL).  With probability at least 1 - delta_loc (over the dither, for a query
 * that does not depend on it) raw bounds the TV of every query head of the call;
 * delta_loc in (0, 1) is the per-(layer, head, step) budget, e.g. delta_req /
 * (layers * query heads * steps).
 */
/*
 * Per-(layer, head, step) failure budget of Tier B (Sec. 4.2, request-level
 * budget by the union bound over the request's certificates):
 *   delta_loc = delta_req / (n_layers * n_q_heads * n_steps),
 * delta_req in (0, 1) the request's budget, n_steps the decode steps it runs
 * (the serving experiments of Sec. 6.2 take 256).  Returns -1 for invalid
 * arguments.  Pass the result (rounded to float) as wc_tierb_decode_attention's
 * delta_loc.
 */
double wc_tierb_delta_loc(double delta_req, int n_layers, int n_q_heads, int n_steps);

int wc_tierb_decode_attention(const wc_cache* cache, const void* q, int q_dtype, int batch,
                              int n_q_heads, const int32_t* block_table, int max_blocks_per_seq,
                              const int32_t* seq_lens, int64_t max_seq_len, float sm_scale,
                              void* out, int out_dtype, float* meter, float* raw, int split_tokens,
                              float delta_loc, void* ws, size_t ws_bytes, void* stream);

/*
 * wc_metered_decode_attention with the gate applied in its split merge (one
 * launch fewer): same arguments, then tau, mask_q, mask_kv and n_gated as in
 * wc_gate below.  Results equal wc_metered_decode_attention followed by
 * wc_gate(meter, raw, batch, n_q_heads, n_q_heads / n_kv_heads, tau, mask_q,
 * mask_kv, n_gated).  raw may be NULL also when tau >= 1.
 */
int wc_metered_decode_gate(const wc_cache* cache, const void* q, int q_dtype, int batch,
                           int n_q_heads, const int32_t* block_table, int max_blocks_per_seq,
                           const int32_t* seq_lens, int64_t max_seq_len, float sm_scale, void* out,
                           int out_dtype, float* meter, float* raw, int split_tokens, float tau,
                           uint8_t* mask_q, uint8_t* mask_kv, int32_t* n_gated, void* ws,
                           size_t ws_bytes, void* stream);

/*
 * One decode step of the meter loop (Sec. 6, boxed meter loop: write the step's
 * token, then the metered read path and the gate): results equal
 *   wc_quantize_write_pair(cache, exact, new_k, new_v, in_dtype, new_slots, batch)
 * followed by wc_metered_decode_gate(cache, q, ...) with the remaining arguments.
 * Where the decode runs on the matrix cores, in_dtype is WC_BF16 and the cache has
 * no bypassed pairs and no group scales, this is one launch: the workgroup whose
 * KV split holds a sequence's new token quantizes and stores it (codes, scales,
 * witness, exact copy) before it reads its pages; otherwise the two calls run
 * back to back on `stream`.
 *   new_k, new_v [batch][n_kv_heads][head_dim] in in_dtype (WC_BF16 or WC_F32),
 *                the step's token of each sequence
 *   new_slots    [batch] int64: the slot of each sequence's last position
 *                (seq_lens[b] - 1: block_table[b][(seq_lens[b] - 1) / 16] * 16 +
 *                (seq_lens[b] - 1) % 16), or < 0 for a sequence without a new
 *                token (seq_lens[b] == 0 needs < 0); any other slot makes the
 *                result unspecified (the write may land after the read)
 *   exact        the bf16 exact cache that the fallback reads (as in
 *                wc_quantize_write_pair)
 * Other arguments and checks as wc_quantize_write_pair and wc_metered_decode_gate.
 */
int wc_step_metered_decode_gate(const wc_cache* cache, const wc_cache* exact, const void* new_k,
                                const void* new_v, int in_dtype, const int64_t* new_slots, const void* q,
                                int q_dtype, int batch, int n_q_heads, const int32_t* block_table,
                                int max_blocks_per_seq, const int32_t* seq_lens, int64_t max_seq_len,
                                float sm_scale, void* out, int out_dtype, float* meter, float* raw,
                                int split_tokens, float tau, uint8_t* mask_q, uint8_t* mask_kv,
                                int32_t* n_gated, void* ws, size_t ws_bytes, void* stream);

/*
 * Joint key + value certificate with its gate (Sec. 3 output bound; Sec. 4.2 value
 * side and joint event): wc_metered_decode_gate (delta_loc == 0: Tier A, the
 * witness bound) or Tier B (0 < delta_loc < 1, as wc_tierb_decode_attention), plus
 * the value meter of each query head over its KV head's cache,
 *   meter_v[b][h] = (sum_t ptilde_t rho_t) / max_t nu_t,
 * rho_t, nu_t the stored value residual (up) and value norm (down), so that
 *   ||y - yhat|| <= (2 meter + meter_v) * max_t ||v_t||
 * (the key-side TV bound times 2 plus the value term, in units of the largest value
 * norm; 0/0 = 0, x/0 = +inf), and the joint gate
 *   mask_q[b][h] = !(pass_K && pass_V),  pass_K = (tau_k < 1 ? meter : raw) <= tau_k,
 *                                        pass_V = meter_v <= tau_v,
 * routed per KV head (any-of-G), n_gated counted as in wc_gate.  The cache must
 * carry the value side (v_resid and v_norm) and, for Tier A, the key witness.
 */
int wc_joint_decode_gate(const wc_cache* cache, const void* q, int q_dtype, int batch,
                         int n_q_heads, const int32_t* block_table, int max_blocks_per_seq,
                         const int32_t* seq_lens, int64_t max_seq_len, float sm_scale, void* out,
                         int out_dtype, float* meter, float* raw, float* meter_v, int split_tokens,
                         float delta_loc, float tau, float tau_v, uint8_t* mask_q, uint8_t* mask_kv,
                         int32_t* n_gated, void* ws, size_t ws_bytes, void* stream);

/*
 * Block-granular repair of routed KV heads (Sec. 6.3, block-level paging; the
 * meter loop's gate pages in the top-contributing blocks).  Run after a metered
 * decode call (Tier A, or Tier B with delta_loc > 0) over the same cache, queries,
 * table, lengths and split_tokens, whose workspace `ws` still holds its partial
 * records, and whose gate set mask_kv.  For every KV head with mask_kv != 0:
 *   blocks are fixed runs of 256 tokens of the sequence (Sec. 6.3: S = 32768 in 128
 *   blocks), block i holding positions 256i .. 256i+255 (the last one shorter),
 *   whatever split_tokens the decode used;
 *   share_{h,i} = sum_{t in i} ptilde_{h,t} (e^{c_{h,t}} - 1) (they add up to A_h - 1),
 *   from the block segments the decode recorded in its workspace,
 *   taken in decreasing order of sum_h share_{h,i} (ties to the lower i), at most
 *   max_repair_blocks (1 .. 64) of them, among the blocks that hold a position not
 *   yet marked as repaired (cache->repaired; all blocks without marks);
 *   a taken block contributes exact logits and values (from the bf16 cache `exact`)
 *   with bound 0; after each block A_h is recomputed, and the repair stops as soon
 *   as every query head h of the KV head passes: (tau < 1 ? meter : raw) <= tau.
 * A repaired KV head gets its G outputs, meter and raw rewritten for the repaired
 * state and its mask_kv cleared (no whole-head fallback needed); otherwise nothing
 * of it changes.  repaired[b][g][0..max_repair_blocks-1] receives the block order
 * (-1 padded; may be NULL) and n_repaired[b][g] the number of blocks taken (0: not
 * routed, -1: the budget did not suffice; may be NULL).  At most 4096 blocks
 * (1,048,576 tokens) per sequence.  out must be the decode's output array (out_dtype as there).
 * repair_ws (repair_ws_bytes >= wc_block_repair_workspace_size for the same sizes,
 * caller-owned device memory, no initialization needed) holds the per-KV-head
 * state and the block corrections; the blocks' corrections are computed in
 * parallel and added in the repair order, so the result does not depend on how
 * they are scheduled.  Calls that share a repair workspace must not overlap.
 */
int wc_block_repair(const wc_cache* cache, const wc_cache* exact, const void* q, int q_dtype,
                    int batch, int n_q_heads, const int32_t* block_table, int max_blocks_per_seq,
                    const int32_t* seq_lens, int64_t max_seq_len, float sm_scale, int split_tokens,
                    float delta_loc, float tau, int max_repair_blocks, const void* ws,
                    size_t ws_bytes, void* out, int out_dtype, float* meter, float* raw,
                    uint8_t* mask_kv, int32_t* repaired, int32_t* n_repaired, void* repair_ws,
                    size_t repair_ws_bytes, void* stream);

/*
 * Bytes of the repair workspace of wc_block_repair for these sizes; 0 for invalid
 * sizes.
 */
size_t wc_block_repair_workspace_size(int batch, int n_q_heads, int n_kv_heads, int head_dim,
                                      int max_repair_blocks);

/*
 * Write-back of a repair (the meter loop's gate, Sec. 6; incremental persistent
 * repair, Sec. 6.3 gated evaluation (c)): marks pages of cache->repaired and zeroes
 * the witness of their slots (when the cache has one), so that every later decode
 * serves them from the exact store with bound 0.  For every (b, g) of the batch:
 *   n_repaired[b][g] > 0: the pages holding positions 0 .. seq_lens[b]-1 of the
 *     blocks repaired_blocks[b][g][0 .. n-1] (256-token blocks, block i = positions
 *     256i .. 256i+255, as wc_block_repair reports them in `repaired`);
 *   whole_kv != NULL and whole_kv[b][g] != 0 (a KV head served by the whole-head
 *     fallback): every page holding positions 0 .. seq_lens[b]-1.
 * Block ids outside [0, 4096), table entries outside the cache and positions past
 * max_blocks_per_seq * 16 are skipped.  n_repaired may be NULL (then only
 * whole_kv counts).  cache->repaired must be set.
 */
int wc_repair_write_back(const wc_cache* cache, int batch, const int32_t* block_table,
                         int max_blocks_per_seq, const int32_t* seq_lens, const int32_t* repaired_blocks,
                         const int32_t* n_repaired, int max_repair_blocks, const uint8_t* whole_kv,
                         void* stream);

/*
 * Gate (the meter loop's gate, Sec. 6; certified vs risk-ranked, Sec. 4.3):
 *   mask_q[b][h]   = (tau < 1 ? meter : raw)[b][h] > tau      (strict)
 *   mask_kv[b][g]  = OR over the `group` query heads of KV head g (any-of-G, Sec. 5)
 *   n_gated[0] += number of set mask_q, n_gated[1] += number of set mask_kv
 *                  (device int32[2], may be NULL; the caller zeroes it)
 * raw may be NULL when tau < 1.
 */
int wc_gate(const float* meter, const float* raw, int batch, int n_q_heads, int group,
            float tau, uint8_t* mask_q, uint8_t* mask_kv, int32_t* n_gated, void* stream);

/*
 * Exact fallback (the meter loop: a gated head is served from the exact store).
 * For every (b, g) with mask_kv[b][g] != 0, overwrites out[b][h] for the G query
 * heads h of KV head g with softmax(sm_scale * q . k_t) v over the bf16 cache
 * `exact` (kind WC_KIND_BF16); other rows of `out` are not touched.
 * Arguments as in wc_metered_decode_attention.
 */
int wc_exact_decode_attention(const wc_cache* exact, const void* q, int q_dtype, int batch,
                              int n_q_heads, const int32_t* block_table,
                              int max_blocks_per_seq, const int32_t* seq_lens,
                              int64_t max_seq_len, float sm_scale, const uint8_t* mask_kv,
                              void* out, int out_dtype, int split_tokens, void* ws,
                              size_t ws_bytes, void* stream);

/*
 * Workspace bytes of wc_step_certified_decode: that of the metered decode plus one
 * more region of split records (0 for invalid sizes).
 */
size_t wc_certified_workspace_size(int batch, int n_q_heads, int n_kv_heads, int head_dim,
                                   int64_t max_seq_len, int split_tokens);

/*
 * One whole decode step of the meter loop (Sec. 6: write the step's token, the
 * metered read path, the gate, the exact fallback for what the gate routes):
 * results equal wc_step_metered_decode_gate(...) followed by
 * wc_exact_decode_attention(exact, q, ..., mask_kv, out, ...) with the same
 * arguments, bit for bit (out, meter, raw, mask_q, mask_kv, n_gated), in three
 * launches instead of four: the metered decode writes its split records, the exact
 * fallback's workgroups first decide their KV head's gate from those records
 * (the split merge's own statistics, in the same bits; the workgroup of the first
 * split stores mask_q and mask_kv) and only the routed ones read the exact cache,
 * and one merge forms every output row (a routed KV head's query heads from the
 * exact records) with meter and raw.  The gate is Tier A's (as
 * wc_metered_decode_gate).
 *   ws     at least wc_certified_workspace_size(batch, n_q_heads, cache->n_kv_heads,
 *          cache->head_dim, max_seq_len, split_tokens) bytes
 *   exact  the bf16 exact cache (kind WC_KIND_BF16, same n_kv_heads and head_dim,
 *          addressed by the same block table)
 * Other arguments and checks as wc_step_metered_decode_gate.
 */
int wc_step_certified_decode(const wc_cache* cache, const wc_cache* exact, const void* new_k,
                             const void* new_v, int in_dtype, const int64_t* new_slots, const void* q,
                             int q_dtype, int batch, int n_q_heads, const int32_t* block_table,
                             int max_blocks_per_seq, const int32_t* seq_lens, int64_t max_seq_len,
                             float sm_scale, void* out, int out_dtype, float* meter, float* raw,
                             int split_tokens, float tau, uint8_t* mask_q, uint8_t* mask_kv,
                             int32_t* n_gated, void* ws, size_t ws_bytes, void* stream);

/*
 * wc_step_certified_decode for steps where most KV heads are routed: the exact
 * fallback of EVERY KV head runs beside the metered decode instead of after it, and
 * the final merge decides the gate (Sec. 6 meter loop; the same gate, any of a KV
 * head's query heads above tau, from the same statistics) and takes each routed KV
 * head's rows from the exact records.  Results are bit for bit those of
 * wc_step_certified_decode (out, meter, raw, mask_q, mask_kv, n_gated and both
 * caches); only the work differs.  With a plain Tier A cache (INT8 dithered or raw
 * fp8, no bypassed pairs, group scales, value side or repair marks), bf16 queries
 * and head_dim 128 both decodes share one launch, their workgroups interleaved on
 * every compute unit, and each writes the step's new tokens (bf16 inputs) into the
 * cache it reads; otherwise the two decodes run one after the other.  It reads the
 * whole exact cache of the active tokens (512 bytes per token and KV head at
 * head_dim 128) whatever the gate decides: the caller picks it when the routed
 * fraction it observes (n_gated) is high.  Arguments, workspace and checks as
 * wc_step_certified_decode.
 */
int wc_step_certified_decode_speculative(const wc_cache* cache, const wc_cache* exact, const void* new_k,
                                         const void* new_v, int in_dtype, const int64_t* new_slots, const void* q,
                                         int q_dtype, int batch, int n_q_heads, const int32_t* block_table,
                                         int max_blocks_per_seq, const int32_t* seq_lens, int64_t max_seq_len,
                                         float sm_scale, void* out, int out_dtype, float* meter, float* raw,
                                         int split_tokens, float tau, uint8_t* mask_q, uint8_t* mask_kv,
                                         int32_t* n_gated, void* ws, size_t ws_bytes, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): wc_step_metered_decode_gate
 * without a workspace argument.  The split records and gate counters live in a
 * static device array of WC_NOALLOC_SCRATCH_BYTES bytes inside the library, one copy
 * per GPU, held until the process ends; the call allocates and frees nothing.
 *   - Returns WC_ESCRATCH (nothing enqueued) when wc_decode_workspace_size(batch,
 *     n_q_heads, cache->n_kv_heads, cache->head_dim, max_seq_len, split_tokens)
 *     exceeds WC_NOALLOC_SCRATCH_BYTES (e.g. 4 sequences of 32k tokens x 28 query
 *     heads need about 2 MiB; 64 sequences up to 32k with a balanced split about 9 MiB).
 *   - Every call on one GPU uses that GPU's array: calls that overlap on one GPU
 *     (other streams, other threads) race and give undefined results.  The array
 *     needs no initialization (the decode clears what it reads back).
 *   - The array's device address is looked up on the first call on each device
 *     (that device current); make that first call outside a graph capture.
 * Other arguments, checks and results as wc_step_metered_decode_gate.
 */
#define WC_NOALLOC_SCRATCH_BYTES (16u << 20)
int wc_step_metered_decode_gate_noalloc(const wc_cache* cache, const wc_cache* exact, const void* new_k,
                                        const void* new_v, int in_dtype, const int64_t* new_slots,
                                        const void* q, int q_dtype, int batch, int n_q_heads,
                                        const int32_t* block_table, int max_blocks_per_seq,
                                        const int32_t* seq_lens, int64_t max_seq_len, float sm_scale,
                                        void* out, int out_dtype, float* meter, float* raw, int split_tokens,
                                        float tau, uint8_t* mask_q, uint8_t* mask_kv, int32_t* n_gated,
                                        void* stream);

#ifdef __cplusplus
}
#endif
#endif /* WITCERT_H */
