/*
 * moe_quant.h -- C ABI of the MI355X (gfx950) mixed-precision MoE expert-FFN
 * kernel library.
 *
 * The library implements the inference hot path of DynaMo ("Runtime Switchable
 * Quantization for MoE with Cross-Dataset Adaptation", arXiv 2503.21135):
 *   - top-k expert selection (Sec. II-A, "MoE Model"),
 *   - expert-level mixed-precision uniform quantization with codes packed into
 *     32-bit words (Sec. IV-A, last paragraph; Sec. V-B "Quantized Weight
 *     Packing Load"),
 *   - the channel-level switch that replaces channels of a quantized expert by
 *     cached higher-precision copies located through (expert, channel) index
 *     headers (Sec. IV-B "Channel Weights Replacement based on Caching";
 *     Sec. V-A "Data Format in the Channel Cache"),
 *   - requantization of the cached original channels at each expert's new
 *     precision when the dataset changes (Sec. IV-B "Channel Weights
 *     Requantization for New Datasets"),
 *   - on the host, the expert significance of Eq. (1) and the precision of
 *     each expert from Alg. 1 (Sec. III-B, Sec. IV-A),
 *   - dequantization fused with the matrix-core contraction (Sec. V-B
 *     "Channel-Grained Dequantization"), applied to the routed expert FFN.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *   - Every buffer is owned by the caller.  "device" pointers are HIP device
 *     memory, "host" pointers are ordinary host memory read only during the
 *     call.  The library allocates no device memory and keeps no state about
 *     any layer or batch between calls.  It caches three host-side facts:
 *     the compute-unit count of each device (read once per device, used to
 *     size the prefill grid), the MOE_DEBUG setting (read once), and
 *     per-thread scratch vectors that moe_set_channel_switch reuses for its
 *     host validation.  moe_expert_ffn_mixed_noalloc additionally owns one
 *     fixed device array per GPU (see there).
 *   - All device work is enqueued on `stream` (a hipStream_t, passed as void*;
 *     NULL is the default stream) and is asynchronous to the host.  No entry
 *     point reads device memory back to the host.
 *   - Arguments are validated on the host before any device work is enqueued;
 *     a call that returns an error has had no effect.  A HIP launch failure is
 *     reported as MOE_ERR_HIP; the stream's state is then undefined.
 *   - bf16 values are passed as uint16_t bit patterns, fp16 values likewise.
 *   - Setting the environment variable MOE_DEBUG=1 makes every entry point
 *     synchronise its stream after each launch and check for errors.
 *
 * Packed code layout (the contract between moe_quant_pack and the FFN)
 * ---------------------------------------------------------------------
 * A row of K codes of bit-width b is stored as K*b/32 little-endian uint32
 * words.  For b in {2, 4, 8} each word holds 32/b consecutive codes; the
 * codes of even local index 2i sit at bits [b*i, b*i+b) and the codes of odd
 * local index 2i+1 at bits [16+b*i, 16+b*i+b) ("half-split" order: the low
 * half-word holds the even codes, the high half-word the odd ones, each least
 * significant field first).  For b = 3 every block of 32 codes takes three
 * words: word 0 holds bits 0..1 of codes 0..15 and word 1 bits 0..1 of codes
 * 16..31, both in the 2-bit half-split order; word 2 holds bit 2 of codes
 * 0..31 in the 1-bit half-split order (code 2i at bit i, code 2i+1 at bit
 * 16+i).  For b = 6 every block of 32 codes takes six words: words 0..3 hold
 * bits 0..3 of codes 8w..8w+7 (word w) in the 4-bit half-split order, words
 * 4 and 5 bits 4..5 of codes 0..15 and 16..31 in the 2-bit half-split order.
 * b = 16 is the unquantized reference layout (the 16-bit model that the
 * paper's speedups are measured against, Sec. VI-C): word i holds the bf16
 * values (round to nearest even) of weights 2i (low half) and 2i+1 (high
 * half), and every {scale, zero} word is {1.0, 0}.
 * Quantization groups run along K: group j covers codes
 * [j*group, (j+1)*group) of a row.
 *
 * Quantizer (per row and group; Sec. IV-A, uniform quantization)
 * ----------------------------------------------------------------
 *   mn = min(0, min w), mx = max(0, max w), qmax = 2^b - 1,
 *   s  = (mx - mn) / qmax in IEEE binary64,
 *   s16 = the smallest fp16 value >= s (1.0 when s == 0),
 *   z  = rint(-mn / s16)            (ties to even, an integer in [0, qmax]),
 *   q  = clamp(rint(w / s16) + z, 0, qmax),
 *   dequantized weight = s16 * (q - z)   (exact in fp32).
 * {s16, z} are stored as one uint32: bits 0..15 the fp16 scale, bits 16..31
 * the fp16 zero point.
 *
 * FFN numerics
 * ------------
 * The hidden activation h = silu(g) * u is rounded to bf16 (round to nearest
 * even) before the down projection, as the paper feeds 16-bit activations to
 * the matrix cores (Sec. V-B); accumulation is fp32.  The weights enter in
 * one of two ways, chosen per launch from the expected tokens per expert:
 *   - up to 28 expected tokens per routed expert (48 for experts narrower
 *     than d_ff 4096), and shared experts over up to 512 tokens (decode):
 *     exactly -- the matrix cores multiply the integer
 *     codes (exact in bf16) by the bf16 activations, and each group's scale
 *     and zero point are applied to the fp32 partial sum;
 *   - more tokens (prefill): as the 16-bit dequantized
 *     operand of the paper (Sec. V-B), fp16(s * (q - z)) -- one rounding per
 *     weight -- multiplied by fp16 copies of the activations and of h.  A
 *     bf16 value converts to fp16 exactly when it is 0 or its magnitude lies
 *     in [2^-17, 65504]; below 2^-17 it is rounded to the fp16 subnormal grid
 *     (absolute error <= 2^-25); beyond 65504 (and for inf or NaN) it has no
 *     finite fp16 value, and the call reports it through its status word
 *     (MOE_ERR_RANGE) instead of silently producing infinities.
 * Unquantized experts (bits 16) take the same two routes: the streaming
 * kernel multiplies their bf16 weights as stored; the tile kernel converts
 * them to fp16 rounding toward zero, exact for magnitudes in [2^-17, 65504]
 * (smaller ones truncate to the fp16 subnormal grid, absolute error < 2^-24;
 * larger ones clamp to +-65504).
 * Either way the FFN output matches the exact definition to within 2e-3
 * relative L2 (measured: ~1e-4 for the first, ~1.1e-3 for the second).
 */
#ifndef MOE_QUANT_H
#define MOE_QUANT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define MOE_OK             0
#define MOE_ERR_ARG       -1  /* bad size, NULL pointer or inconsistent arguments      */
#define MOE_ERR_BITS      -2  /* bit-width outside {2, 3, 4, 6, 8} (or 16 where allowed) */
#define MOE_ERR_ALIGN     -3  /* a pointer that must be 16-byte aligned is not          */
#define MOE_ERR_WORKSPACE -4  /* workspace NULL or smaller than the size helper returns */
#define MOE_ERR_SLOT      -5  /* switch slot out of range, duplicated, or two slots
                                 naming the same (expert, row)                          */
#define MOE_ERR_RANGE     -6  /* a value outside fp16's range: a scale in moe_quant_pack
                                 or moe_requant_channels, an activation or hidden value
                                 of the FFN's fp16 operand path (device status words) */
#define MOE_ERR_HIP       -7  /* a HIP call or kernel launch failed                    */

/* Limits checked by the host validation. */
#define MOE_MAX_EXPERTS  256  /* routed + shared experts of one layer */
#define MOE_MAX_TOPK      16

/* Kinds of expert weight matrix. */
#define MOE_KIND_GATE 0   /* [d_ff][d_model]  rows = hidden neurons, K = d_model */
#define MOE_KIND_UP   1   /* [d_ff][d_model]                                     */
#define MOE_KIND_DOWN 2   /* [d_model][d_ff]  rows = output channels, K = d_ff   */

/*
 * moe_code_row_words -- row stride, in 32-bit words, of the packed code
 * matrices moe_expert_ffn_mixed reads (base codes and 8-bit copies): K*bits/32
 * words of codes followed by padding of 16 words (32 words at bits >= 8), so
 * that consecutive rows never start a power of two of bytes apart.  The
 * padding words are never read.  Returns 0 for bits outside {2, 3, 4, 6, 8, 16}
 * or K not a positive multiple of 128.
 */
int64_t moe_code_row_words(int32_t K, int32_t bits);

/*
 * One kind (gate, up or down) of every expert of a layer.
 *
 * Base codes: expert e (routed experts 0..E-1 first, then shared experts
 * E..E+S-1) stores its R_e x K_e matrix row-major in the packed layout above
 * at word offset code_off[e] of `codes`, row stride
 * moe_code_row_words(K_e, bits[e]) words.
 * code_off[e] must be a multiple of 4 (16-byte aligned rows start).
 * Its scales and zeros are group-major: the {s16, z} word of (row r, group j)
 * is sz[sz_off[e] + j*R_e + r].
 *
 * Resident copies (the channel cache of Sec. IV-B / V-A, kept in the 8-bit
 * code format: 8-bit codes quantized from the original rows, or b-bit codes
 * one per byte after moe_requant_channels): slot s holds one row of
 * a routed expert, K/4 words at copy_codes[s*moe_code_row_words(K, 8)], its
 * {s16, z} words at
 * copy_sz[s*(K/group) + j], and its header (expert, row) at copy_hdr[2s],
 * copy_hdr[2s+1].  A layer may have n_slots = 0 (copy pointers then NULL).
 *
 * Switch state, written only by moe_set_channel_switch: row_slot[e*R + r] is
 * the copy slot that row r of routed expert e currently reads, or -1 for its
 * base codes.
 */
typedef struct moe_kind_desc {
  const uint32_t* codes;          /* device */
  const uint32_t* sz;             /* device */
  const int64_t*  code_off;       /* device [E+S] */
  const int64_t*  sz_off;         /* device [E+S] */
  const int64_t*  code_off_host;  /* host   [E+S] (validation) */
  int32_t         n_slots;
  int32_t         reserved0;
  const uint32_t* copy_codes;     /* device [n_slots][K/4]      */
  const uint32_t* copy_sz;        /* device [n_slots][K/group]  */
  const int32_t*  copy_hdr;       /* device [n_slots][2]        */
  const int32_t*  copy_hdr_host;  /* host   [n_slots][2]        */
  int32_t*        row_slot;       /* device [E][R]              */
} moe_kind_desc_t;

/*
 * One MoE layer.  Routed experts have hidden size d_ff, shared experts
 * d_ff_shared (shared experts are always applied with weight 1 and are never
 * switched).  bits[e] in {2, 3, 4, 6, 8}, or 16 for an unquantized expert
 * (bf16 weights); bit-widths 3 and 6 need group == 128, 16 needs group == 64.
 *
 * order_gu[e*d_ff + i] and order_dn[e*d_model + i] (routed experts only) are
 * the orders in which the FFN visits hidden neurons and output channels.  They
 * are rebuilt by moe_set_channel_switch as stable partitions by source class:
 * for a hidden neuron, class bit 0 = its gate row reads a cached copy, bit 1 =
 * its up row does; for an output channel, class 1 = its down row does.  Rows
 * of class 0 come first (ascending), then class 1, 2, 3.  class_cnt[e*4 + c]
 * (gate/up) and class_cnt[4*E + e*4 + c] (down) count the rows of each class.
 * Any permutation gives the same result.
 */
typedef struct moe_layer {
  int32_t n_experts;     /* E, routed  */
  int32_t n_shared;      /* S          */
  int32_t d_model;
  int32_t d_ff;
  int32_t d_ff_shared;
  int32_t group;         /* 64 or 128  */
  const int32_t* bits_host;   /* host   [E+S] */
  const int32_t* bits;        /* device [E+S] */
  moe_kind_desc_t kind[3];
  int32_t* order_gu;          /* device [E][d_ff]    */
  int32_t* order_dn;          /* device [E][d_model] */
  int32_t* class_cnt;         /* device [2][E][4]: rows per source class of the orders */
  int32_t* staging;           /* device scratch of at least max(kind[].n_slots)+1 int32 */
} moe_layer_t;

/*
 * moe_quant_pack -- quantize rows of an fp32 matrix and pack the codes.
 * Sec. IV-A (uniform quantization of each expert at its precision) and
 * Sec. V-B (several low-bit codes packed into one 32-bit word).
 *
 *   w        device fp32 [R][ld_w]; the rows to quantize are rows[0..n-1]
 *            (device int32 list) or, when rows == NULL, rows 0..n-1 (n <= R).
 *   K        codes per row; K % group == 0, K % 32 == 0.
 *   bits     2, 3, 4, 6 or 8, or 16 (the bf16 values, {1.0, 0} words).
 *   group    64 or 128 (3- and 6-bit need 128).
 *   codes    device; list row i is written to codes[i*ld_codes ...], K*bits/32
 *            words; ld_codes >= K*bits/32; codes and ld_codes*4 16-byte aligned.
 *   sz       device; {s16, z} word of (list row i, group j) is written to
 *            sz[i*sz_row_stride + j*sz_group_stride].
 *   status   device int32 or NULL; set to MOE_ERR_RANGE by any group whose
 *            scale overflows fp16 (that group's scale is then +inf).  Never
 *            cleared by the library.
 */
int moe_quant_pack(const float* w, int64_t ld_w, int32_t R, int32_t K,
                   int32_t bits, int32_t group,
                   const int32_t* rows, int32_t n,
                   uint32_t* codes, int64_t ld_codes,
                   uint32_t* sz, int64_t sz_row_stride, int64_t sz_group_stride,
                   int32_t* status, void* stream);

/*
 * moe_route_permute -- router, top-k selection and token permutation.
 * Sec. II-A (a fixed number K of experts selected per token); the paper's
 * one-to-many mapping of a token to the channels of several experts
 * (Sec. I, Sec. II-A "Data-Weight Mappings") becomes per-expert segments.
 *
 *   x         device bf16 [T][d]
 *   w_router  device fp32 [E][d];  bias  device fp32 [E] or NULL
 *   logit[t][e] = (sum_c x[t][c]*w_router[e][c]) + bias[e], computed in fp32
 *             in this fixed order: 64 partial sums, partial l accumulating
 *             fmaf over c = l, l+64, l+128, ... in increasing c; then for
 *             off = 32, 16, 8, 4, 2, 1: partial[l] += partial[l+off] (l < off).
 *   topk_ids  device int32 [T][k]: the k experts of largest logit, ordered by
 *             (logit descending, expert index ascending); a NaN logit ranks as
 *             -inf (in the softmax too), so the k ids are always distinct
 *             experts in [0, E).
 *   topk_w    device fp32 [T][k]: softmax over the k selected logits,
 *             m = logit of slot 0, e_j = cexp(l_j - m), S = e_0 + e_1 + ...
 *             summed left to right, w_j = e_j / S.  cexp is the library's
 *             exponential for arguments <= 0: 0 below -80, otherwise
 *             n = rint(x*fl(log2 e)), r = x - n*ln2 by a two-constant
 *             Cody-Waite reduction with fmaf (ln2 split into its leading 12
 *             significant bits and the fp32 remainder), the degree-7 Taylor
 *             polynomial of e^r with fp32 coefficients 1/i! by Horner fmaf,
 *             scaled by 2^n.
 *   offsets   device int32 [E+S+1]: segment e (routed) holds the rows of the
 *             tokens that selected e, tokens in increasing order; segment E+s
 *             (shared expert s) holds all T tokens in order.  offsets[0] = 0.
 *   perm_token device int32 [T*(k+S)]: token of each permuted row.
 *   inv_perm  device int32 [T][k+S]: row of (t, topk slot j) for j < k, and of
 *             (t, shared expert s) at j = k+s.
 *   x_perm    device bf16 [T*(k+S)][d] or NULL: x[perm_token[p]] (bit copy).
 *   ws        device workspace of at least moe_route_workspace_bytes(T,E,k,S).
 *   Requires d % 64 == 0, d <= 8192, 1 <= k <= min(E, MOE_MAX_TOPK),
 *   E+S <= MOE_MAX_EXPERTS.
 *   Results are bitwise reproducible.
 */
int moe_route_permute(const uint16_t* x, int32_t T, int32_t d,
                      const float* w_router, const float* bias,
                      int32_t E, int32_t k, int32_t S,
                      int32_t* topk_ids, float* topk_w,
                      int32_t* offsets, int32_t* perm_token, int32_t* inv_perm,
                      uint16_t* x_perm,
                      void* ws, size_t ws_bytes, void* stream);

/*
 * moe_route_workspace_bytes -- bytes of device workspace moe_route_permute
 * needs for this batch: two int32 [ceil(T/64)][E] tables (per-chunk expert
 * counts and bases) and, from 256 tokens or 16 experts on, the fp32 [T][E]
 * logits that the router writes before its top-k pass, each region 256-byte
 * aligned.  Returns 0 for T < 0 or
 * E <= 0.  The contents need no initialization and are scratch between calls.
 */
size_t moe_route_workspace_bytes(int32_t T, int32_t E, int32_t k, int32_t S);

/*
 * moe_ffn_plan -- the output split count and workspace size of
 * moe_expert_ffn_mixed for this layer and batch.  Depends only on host-known
 * shapes.  Either output pointer may be NULL.
 */
int moe_ffn_plan(const moe_layer_t* L, int32_t T, int32_t k,
                 int32_t* n_split, size_t* ws_bytes);

/*
 * moe_expert_ffn_mixed -- the routed (and shared) expert FFNs of one layer
 * over per-expert mixed-precision packed weights, with the channel switch
 * applied row by row.  Sec. IV-A (expert-level precisions), Sec. IV-B and
 * V-A (switched channels read their cached copy), Sec. V-B (packed loads,
 * on-chip unpacking, dequantization fused into the matrix-core contraction).
 *
 * For permuted row p of segment e (token t = perm_token[p]):
 *   g = Wg_e x_t,  u = Wu_e x_t,  h = bf16(silu(g) * u),  o_p = Wd_e h
 * where each row of W*_e is the dequantized copy slot row_slot[e][row] when
 * that is >= 0 and the dequantized base codes otherwise.
 *
 *   x          device bf16 [T][d_model], original token order.
 *   offsets, perm_token   from moe_route_permute (T*k routed rows, S*T shared).
 *   o          device fp32 [n_split][T*(k+S)][d_model]; the FFN output of row p
 *              is the sum over the n_split slices (moe_ffn_plan), which
 *              moe_unpermute_combine adds.  16-byte aligned.
 *   ws         device workspace of at least moe_ffn_plan()'s ws_bytes; scratch
 *              between calls (no initialization needed).
 *   status     device int32 or NULL; set to MOE_ERR_RANGE when the fp16 operand
 *              path (prefill sizes, see "FFN numerics") meets an activation or
 *              a hidden value with no finite fp16 value (|v| > 65504, inf,
 *              NaN); the outputs of that call are then not valid.  Never
 *              cleared by the library; the streaming (decode) path never sets it.
 *   Never reads offsets on the host: the grid covers the worst case and idle
 *   waves exit.
 */
int moe_expert_ffn_mixed(const moe_layer_t* L, const uint16_t* x, int32_t T,
                         int32_t k, const int32_t* offsets,
                         const int32_t* perm_token, float* o,
                         void* ws, size_t ws_bytes, int32_t* status, void* stream);

/*
 * moe_expert_ffn_mixed_ev -- moe_expert_ffn_mixed that also records HIP
 * events on `stream`, so a caller can time the FFN's stages on the stream
 * they run on.  The events are attached to the kernel dispatches themselves
 * (they take the dispatch's begin or end timestamp; no marker packets are
 * added between kernels).  Not on the hot path of a production caller; same
 * arguments, results and errors otherwise.
 *   events    host array of n_events hipEvent_t handles (as void*), each
 *             created by the caller; NULL entries are skipped:
 *             [0] begin of the activation group-sum launch,
 *             [1] begin of the first gate/up launch,
 *             [2] end of the last gate/up launch,
 *             [3] begin of the first down launch,
 *             [4] end of the last down launch.
 *             A stage with no launch records its events as stream markers.
 */
int moe_expert_ffn_mixed_ev(const moe_layer_t* L, const uint16_t* x, int32_t T,
                            int32_t k, const int32_t* offsets,
                            const int32_t* perm_token, float* o,
                            void* ws, size_t ws_bytes, int32_t* status, void* stream,
                            void* const* events, int32_t n_events);

/*
 * moe_expert_ffn_mixed_noalloc -- moe_expert_ffn_mixed without a workspace
 * argument, for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation.  It
 * calls no hipMalloc, hipFree or allocating library routine.
 *
 * Its workspace is one fixed device array of MOE_NOALLOC_SCRATCH_BYTES (64
 * MiB) per GPU, part of the library's code object: each GPU the library runs
 * on holds it until the process ends.  Its device address is looked up once
 * per device, on the first call made with that device current.  Batches
 * whose workspace (moe_ffn_plan's ws_bytes) exceeds the array are rejected
 * with MOE_ERR_WORKSPACE before any device work: decode and mid-size batches
 * fit (the Mixtral-shaped layer at 64 tokens needs ~4 MB, the Qwen-shaped
 * layer at 512 tokens ~12 MB), prefill batches of thousands of tokens use
 * moe_expert_ffn_mixed with a caller workspace.  Nothing in the array needs
 * to start at zero.  Every call on one GPU shares that GPU's array: calls
 * that overlap in time on one GPU (different streams, or different host
 * threads without ordering) race and give undefined results; calls ordered
 * on one stream do not.  Same arguments (minus ws, ws_bytes), results and
 * errors as moe_expert_ffn_mixed otherwise; MOE_ERR_HIP if the array's
 * address cannot be obtained.
 */
#define MOE_NOALLOC_SCRATCH_BYTES (64u << 20)
int moe_expert_ffn_mixed_noalloc(const moe_layer_t* L, const uint16_t* x, int32_t T,
                                 int32_t k, const int32_t* offsets,
                                 const int32_t* perm_token, float* o,
                                 int32_t* status, void* stream);

/*
 * moe_set_channel_switch -- install a set of cached copies.
 * Sec. IV-B "Channel Weights Replacement based on Caching" and Sec. V-A "Data
 * Format in the Channel Cache": the copy of each listed slot replaces the row
 * named by its (expert, row) header; every other row of that kind reverts to
 * its base codes.  No requantization takes place.
 *
 *   kind      MOE_KIND_GATE/UP/DOWN, or -1 with n_on == 0 to reset all kinds.
 *   slots_on  host int32 list of n_on distinct slots in [0, n_slots) whose
 *             headers name distinct rows; copied before the call returns.
 *   Rewrites kind[kind].row_slot, order_gu and class_cnt[0..4E) (gate/up) or
 *   order_dn and class_cnt[4E..8E) (down).
 */
int moe_set_channel_switch(moe_layer_t* L, int32_t kind,
                           const int32_t* slots_on, int32_t n_on, void* stream);

/*
 * moe_requant_channels -- requantize cached 16-bit channels into the copy
 * slots of one kind, each at the new precision of the expert its header names.
 * Sec. IV-B "Channel Weights Requantization for New Datasets": once the
 * experts' precisions are determined again for a new dataset, the retained
 * original channels of every expert whose precision changed are quantized
 * afresh at that precision, which may be higher or lower than before; Sec.
 * V-A: the cache of original channels lives in device memory, entries keyed by
 * (expert, channel) headers.
 *
 *   kind         MOE_KIND_GATE, MOE_KIND_UP or MOE_KIND_DOWN.
 *   cache        device binary16 [n_slots][ld_cache] (4-byte aligned,
 *                ld_cache even and >= K): row s is the original channel named
 *                by slot s's header (copy_hdr[2s], copy_hdr[2s+1]).
 *   expert_bits  host int32 [n_experts]: new precision of each routed expert
 *                in {2, 3, 4, 6, 8}, or 0 to leave its slots untouched; read
 *                before the call returns.
 *   status       device int32 or NULL: set to MOE_ERR_RANGE when a scale
 *                overflows binary16 (the group is still written).
 * Every slot whose expert has expert_bits[e] = b > 0 is rewritten with the
 * moe_quant_pack quantizer at b bits applied to the binary16 values of its
 * cache row (group size L->group, exactly as moe_quant_pack with bits = b
 * produces for those values); the b-bit codes are stored in the 8-bit copy
 * format (one code per byte, kind[kind].copy_codes row stride
 * moe_code_row_words(K, 8)) with their {s16, z} words in kind[kind].copy_sz,
 * so the FFN reads them unchanged.  copy_codes and copy_sz must be writable.
 * The switch state is not touched: rows whose slots are switched on read the
 * new codes from the next FFN call on the same stream.  Returns MOE_ERR_SLOT
 * for a header naming an expert outside [0, n_experts).
 */
int moe_requant_channels(moe_layer_t* L, int32_t kind, const uint16_t* cache,
                         int64_t ld_cache, const int32_t* expert_bits,
                         int32_t* status, void* stream);

/*
 * moe_unpermute_combine -- the MoE output of each token, Sec. II-A: the
 * outputs of the k selected experts weighted by the router's combine weights
 * (plus the shared experts with weight 1), back in token order:
 *   y[t] = sum_j topk_w[t][j] * o[inv_perm[t][j]] + sum_s o[inv_perm[t][k+s]],
 * where o[p] = sum over the n_split slices at o + i*split_stride (slice 0
 * first).  fp32, fused multiply-adds in the order written (slot 0 first), so
 * the result is bitwise reproducible.
 *   o         device fp32 [n_split] slices of [T*(k+S)][d] (moe_expert_ffn_mixed)
 *   inv_perm, topk_w   from moe_route_permute
 *   y         device fp32 [T][d]; o, y 16-byte aligned, d % 4 == 0.
 */
int moe_unpermute_combine(const float* o, int32_t n_split, int64_t split_stride,
                          const int32_t* inv_perm, const float* topk_w,
                          int32_t T, int32_t k, int32_t S, int32_t d,
                          float* y, void* stream);

/*
 * moe_expert_significance -- expert significance of one dataset, Eq. (1)
 * (Sec. III-B), and each expert's token share.  Host only, no device work.
 *
 *   sig       host float [T]: significance of token i's combined top-K channel
 *             output (finite, >= 0).
 *   topk_ids  host int32 [T][k]: the experts the router chose for each token
 *             (an expert repeated in a row counts once).
 *   s_exp     host double [E] out: sum of sig over the tokens routed to expert
 *             e divided by the sum over all T tokens (0 when that sum is 0);
 *             the values add up to k.
 *   share     host double [E] out or NULL: fraction of the T tokens routed to e.
 * Sums run over tokens in ascending order.  MOE_ERR_ARG for an id outside
 * [0, E), a negative or non-finite sig, k outside [1, MOE_MAX_TOPK] or E
 * outside [1, MOE_MAX_EXPERTS].
 */
int moe_expert_significance(const float* sig, const int32_t* topk_ids, int32_t T,
                            int32_t k, int32_t E, double* s_exp, double* share);

/*
 * moe_allocate_bits -- expert-level precision from significance: the fuzzy
 * c-means of Alg. 1 (Sec. IV-A), one precision per cluster, and the
 * low-precision-first rule for experts in the overlap of clusters.  Host only.
 *
 *   x, share  host double [n]: each expert's significance and token share.
 *   levels    host int32 [c]: bit-widths from the most to the least
 *             significant cluster, each in [1, 8] (the FFN runs {2, 3, 4, 6, 8}).
 *   c         clusters, 1..8 (the paper uses 4);  m > 1 fuzzifier;
 *   eps > 0   stop when the Frobenius norm of the change of U is below eps,
 *             or after max_iter >= 1 rounds.
 *   alpha     membership from which an expert counts as inside a cluster.
 *   bits      host int32 [n] out;  V host double [c], U host double [n][c] and
 *             rounds (all optional, NULL to skip) receive the final centers,
 *             memberships and the number of rounds.
 * Initial U: experts sorted by ascending significance (ties by index) are cut
 * into c consecutive runs of equal token share, each expert joining, with
 * membership 1, the run that holds the midpoint of its own share (by rank when
 * every share is 0).  Each round updates the centers (membership^m weighted
 * means), then the memberships (the textbook FCM update; an expert that
 * coincides with centers splits its membership equally among them).  The
 * cluster with the largest center takes levels[0], the next levels[1], ...
 * (ties by cluster index).  An expert takes the lowest precision among the
 * clusters where its membership is >= alpha, or, if there is none, that of
 * its largest membership (first on ties).
 */
int moe_allocate_bits(const double* x, const double* share, int32_t n,
                      const int32_t* levels, int32_t c, double m, double eps,
                      int32_t max_iter, double alpha, int32_t* bits, double* V,
                      double* U, int32_t* rounds);

/* Human-readable name of a status code. */
const char* moe_status_str(int status);

#ifdef __cplusplus
}
#endif

#endif /* MOE_QUANT_H */
