/*
 * kvk.h — C ABI of the per-layer compressed KV-cache library (KV-Kaizen decode path).
 *
 * The library implements the inference-time hot path of KV-Kaizen
 * (arXiv 2609.37988): a plan assigns every layer one action, either `inherit`
 * (read the nearest earlier anchor's cache, §2.1 "Depth") or a kept width and
 * bit-width (d, b) (§2.2, eq. (1)–(3)).  Anchor layers write their K/V cache once
 * at prefill, compressed as the plan says (§2.1 "Precision", App. C.3); every
 * decode step then runs single-query softmax attention of each layer's own
 * query against its anchor's compressed cache (§2.1).
 *
 * Conventions that hold for every entry point:
 *   - All device buffers (inputs, arena, workspace, outputs) are owned by the
 *     caller.  They must be device pointers valid on the current HIP device and
 *     16-byte aligned.  The library never allocates or frees device memory and
 *     never synchronises the stream on these calls.
 *   - Calls that launch work enqueue it on `stream` and return at once.  All
 *     argument validation happens synchronously on the host before any launch;
 *     a failing call launches nothing.
 *   - Errors are returned as kvk_status codes, never as aborts or C++
 *     exceptions.  kvk_last_error() returns a thread-local message for the
 *     last failing call on the calling thread.
 *   - A kvk_table is immutable after creation; it may be shared between
 *     threads for concurrent calls.
 *   - Keys handed to the library are taken as they are (post-RoPE); the
 *     library never applies a rotary embedding.
 *   - GQA head map: query head h reads KV head h / (Hq / Hkv).
 */
#ifndef KVK_H
#define KVK_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KVK_MAX_LAYERS 64
#define KVK_MAX_BATCH_PLANS 256  /* sequences of a batch with per-sequence plans */
#define KVK_GROUP 32 /* quantisation group: 32 tokens (keys) / 32 channels (values) */

typedef enum {
  KVK_OK = 0,
  KVK_ERR_INVALID = -1,     /* a plan, shape, pointer or size violates this header */
  KVK_ERR_UNSUPPORTED = -2, /* valid in the paper's terms, not provided by this library */
  KVK_ERR_DEVICE = -3,      /* a HIP launch or query failed; see kvk_last_error() */
  KVK_ERR_BUFFER = -4       /* a caller buffer is too small (workspace) */
} kvk_status;

typedef enum { KVK_GQA = 0, KVK_MLA = 1 } kvk_kind;

/* Quantiser used by every quantised layer of a table.
 *  KVK_Q_KIVI32 — grouped asymmetric (App. C.3 "grouped asymmetric quantizer"):
 *    keys: one (scale, zero) pair of fp16 per channel per 32 consecutive stored
 *    tokens; values: one pair per token per 32 consecutive channels; codes use
 *    all 2^b levels.
 *  KVK_Q_SYMROW — the paper's own quantiser (App. B "Quantization", App. C.3):
 *    symmetric, one bf16 scale per 128-element token-head row (per token, per
 *    KV head, separately for K and V), codes in [-q, q] with q = 2^(b-1) - 1.
 *  KVK_Q_GROUP64 — grouped asymmetric per token (App. C.3's on-device grouped
 *    cache, 4 + 32/64 = 4.5 bits per element at 4 bits): keys and values alike,
 *    one fp16 (scale, zero) pair per token per 64 consecutive channels.  GQA
 *    tables only, head_dim a multiple of 64. */
typedef enum { KVK_Q_KIVI32 = 0, KVK_Q_SYMROW = 1, KVK_Q_GROUP64 = 2 } kvk_qscheme;

typedef enum { KVK_BF16 = 0, KVK_F32 = 1 } kvk_dtype;

/* One plan entry (§2.2, eq. (3)).  inherit != 0 selects the zero-cost action;
 * otherwise bits is b in {2, 4, 8, 16} and rank is the kept width d.  For GQA
 * the rank axis does not exist (§2.2): rank must be 0 or 2*Hkv*d_h.  For MLA
 * rank is d in {r/8, r/4, r/2, r} (eq. (3)). */
typedef struct {
  int32_t inherit;
  int32_t bits;
  int32_t rank;
} kvk_action;

/* Geometry of the cached model and of the arena. */
typedef struct {
  int32_t kind;        /* kvk_kind */
  int32_t n_layers;    /* L, 1..KVK_MAX_LAYERS */
  int32_t n_q_heads;   /* Hq; MLA: a multiple of 8, at most 256 */
  int32_t n_kv_heads;  /* GQA: Hkv; Hq % Hkv == 0; Hq/Hkv * (readers of one anchor) <= 64.
                          MLA: KV heads of the bf16 GQA model the ratio eq. (2) is
                          quoted against (C0 = L * 2 * Hkv * d_h * 16); >= 1 */
  int32_t head_dim;    /* GQA: d_h in {64, 128}.  MLA: d_h of that reference model, >= 1 */
  int32_t latent_dim;  /* MLA r: a multiple of 256; kept widths at most 1024 (unused for GQA, pass 0) */
  int32_t rope_dim;    /* MLA d_R: 64 (unused for GQA, pass 0) */
  int32_t nope_dim;    /* MLA per-head no-RoPE query/key width: a multiple of 32, <= 256 */
  int32_t v_dim;       /* MLA per-head value width: a multiple of 16, <= 256 */
  int32_t qscheme;     /* kvk_qscheme */
  int32_t batch;       /* B >= 1 */
  int32_t max_tokens;  /* prefill length capacity per sequence, >= 1 */
  int32_t keep_tokens; /* 0: no eviction; else stored tokens per stream (GQA: per
                          (sequence, KV head); MLA: per sequence) */
} kvk_dims;

typedef struct kvk_table kvk_table;

/* Everything the host needs to allocate and account for a table. */
typedef struct {
  int64_t arena_bytes;          /* bytes the caller allocates for the compressed cache */
  int64_t workspace_bytes;      /* decode workspace for the full layer range [0, L) */
  int32_t n_anchors;            /* layers that own a cache */
  int32_t stored_tokens_cap;    /* stored tokens per stream: keep_tokens or max_tokens */
  double cost_bits_per_token;   /* sum over layers of c(a_l), eq. (1) */
  double c0_bits_per_token;     /* C0 = L * 2 * Hkv * d_h * 16, eq. (2) */
  double rho;                   /* eq. (2): C0 / sum c(a_l), metadata excluded (§3) */
  double rho_realized;          /* bf16 cache bytes / arena bytes actually stored at
                                   capacity (metadata and bf16 tail included, eviction
                                   included) */
  int32_t anchor_of[KVK_MAX_LAYERS];   /* nearest anchor at or before l (§2.1) */
  int64_t layer_offset[KVK_MAX_LAYERS];/* byte offset of the layer's region; -1 if it inherits */
  int64_t layer_bytes[KVK_MAX_LAYERS]; /* region size (0 if it inherits) */
  int64_t stream_bytes[KVK_MAX_LAYERS];/* bytes of one stream of the layer (GQA: one
                                          (b, KV head); MLA: one sequence b) */
  double layer_cost_bits[KVK_MAX_LAYERS]; /* c(a_l), eq. (1), bits per token */
  double layer_bits_per_elt[KVK_MAX_LAYERS]; /* stored bits per cached scalar at capacity,
                                                metadata included (App. C.3 accounting) */
} kvk_table_info;

/*
 * ARENA LAYOUT (GQA).  All multi-byte fields are little-endian.
 *
 * The region of anchor layer l (layer_offset[l], layer_bytes[l]) holds B*Hkv
 * streams, stream s = b*Hkv + kvh at offset s*stream_bytes[l].  A stream holds
 * the layer's stored tokens of one (sequence, KV head) in order: NB = cap/32
 * full blocks of 32 tokens (cap = stored_tokens_cap), followed by one tail
 * block.  With n stored tokens, blocks 0 .. n/32-1 are full and the tail block
 * holds tokens 32*(n/32) .. n-1 (fewer than 32) in the bf16 block format, its
 * unused slots zero.  Stream and region sizes are rounded up to 256 bytes.
 * Regions follow each other in layer order from offset 0; arena_bytes is their
 * total.
 *
 * Within a 32-token block, positions are described by "lanes" lam = 16*kg + i
 * with kg in 0..3 and i in 0..15, D = d_h, and
 *   K slot map: lane lam, tile tau in {0,1}, sub-chunk j in 0..D/32-1, slot s in 0..7
 *               holds token 16*tau + i, channel 32*j + 8*kg + s;
 *   V slot map: lane lam, tile m in 0..D/16-1, slot s in 0..7
 *               holds channel 16*m + i, token 16*(s/4) + 4*kg + (s%4).
 *
 * Each lane owns a share of P bytes of a part (a K tile's codes or values, or
 * the V codes or values).  "Share byte o of lane lam" below is stored at part
 * byte 1024*(o/16) + 16*lam + o%16 when P > 16 (the shares are dealt out to the
 * 64 lanes in 16-byte pieces, so that each 16-byte load of all lanes reads one
 * contiguous kilobyte), and at part byte lam*P + o when P <= 16.
 *
 * bf16 block (bits = 16, and every tail block), 128*D bytes:
 *   [K: 64*D bytes][V: 64*D bytes]
 *   K: tile tau is the part at byte 32*D*tau (P = D/2); sub-chunk j of lane lam
 *      is share bytes 16*j .. 16*j + 15, slot s the bf16 at share byte 16*j + 2*s.
 *   V: the part at byte 64*D (P = D); tile m of lane lam is share bytes
 *      16*m .. 16*m + 15, slot s the bf16 at share byte 16*m + 2*s.
 *   A bf16 value is the round-to-nearest-even bf16 of the input value.
 *
 * quantised block (bits b in {2, 4, 8}):
 *   [K codes: 4*D*b][V codes: 4*D*b][K meta][V meta]
 *   K codes: tile tau is the part at byte 2*D*b*tau (P = D*b/32); sub-chunk j of
 *      lane lam occupies share bytes j*b .. j*b + b - 1.
 *   V codes: the part at byte 4*D*b (P = D*b/16); tile m of lane lam occupies
 *      share bytes m*b .. m*b + b - 1.
 *   Each such b-byte "chunk" holds 8 codes of b bits (slots s = 0..7):
 *      b = 8: slot s is byte s.
 *      b = 4: the chunk is one 32-bit word; slot s at bit 16*(s%2) + 4*(s/2).
 *      b = 2: chunk pairs (j or m even, then odd) form one 32-bit word at the even
 *             chunk's byte; slot s of chunk x at bit 16*(s%2) + 2*(s/2) + 8*(x%2).
 *   KIVI32 meta (4*D bytes each):
 *      K meta: fp16 scale[D] then fp16 zero[D], natural channel order; the pair
 *              of channel c covers this block's 32 tokens.
 *      V meta: fp16 at index ((g*2 + w)*4 + kg)*8 + s, w = 0 scale / 1 zero, for
 *              channel group g (channels 32g..32g+31) and token
 *              16*(s/4) + 4*kg + (s%4).
 *   SYMROW meta (64 bytes each): K meta bf16 scale[32], V meta bf16 scale[32],
 *      natural token order.
 *   GROUP64 meta (2*D bytes each), NG = D/64 channel groups g (channels
 *      64g..64g+63), w = 0 scale / 1 zero:
 *      K meta: fp16 at index ((tau*4 + kg)*NG*2 + g*2 + w)*4 + e for token
 *              16*tau + 4*kg + e (the token order of a lane's score tile);
 *      V meta: fp16 at index ((g*2 + w)*4 + kg)*8 + s for token
 *              16*(s/4) + 4*kg + (s%4) (as KIVI32's V meta, over the NG groups).
 *   Block bytes: KIVI32 8*D*(b+1); SYMROW 8*D*b + 128; GROUP64 8*D*b + 4*D.
 *
 * Codes (unsigned, b bits):
 *   KIVI32 (App. C.3 grouped asymmetric): for a group x_1..x_32 (a channel over a
 *   block's tokens for K, a token over 32 channels for V; GROUP64: a token over
 *   64 channels, K and V), in IEEE fp32 arithmetic with round-to-nearest-even:
 *      mn = min x, mx = max x
 *      scale = fp16( (mx - mn) / (2^b - 1) ),  zero = fp16( mn )
 *      u = 0 if scale == 0 else clamp( rint( (x - zero) / scale ), 0, 2^b - 1 )
 *      dequantised value = fmaf(u, scale, zero)
 *   SYMROW (App. C.3 symmetric): for a 128-element row, q = 2^(b-1) - 1,
 *      scale = bf16( max|x| / q ),
 *      code = 0 if scale == 0 else clamp( rint( x / scale ), -q, q ),
 *      u = code + 2^(b-1), dequantised value = code * scale.
 *   Inputs with |x| beyond the fp16 range are outside the supported domain of
 *   KIVI32 (the scale and zero are fp16).
 */

/*
 * ARENA LAYOUT (MLA).  Rank axis, §2.1 and App. C.2: an MLA layer stores per token
 * the first d coordinates of its latent c (d = the action's rank; the remaining
 * r - d are never written) and the positional key k^R of width d_R (stored as
 * given, after RoPE).  The W = d + d_R stored channels of a token are, in order,
 * c[0..d-1] then k^R[0..d_R-1].
 *
 * The region of anchor layer l holds B streams, stream b (sequence b) at offset
 * b*stream_bytes[l].  A stream holds NB = cap/32 full blocks of 32 tokens and one
 * bf16 tail block, as for GQA; stream and region sizes are rounded up to 256.
 *
 * Inside a block the bytes are ordered by the decode kernel's MFMA operand
 * lanes, so that each of its load instructions reads one contiguous run.  Token t
 * (0..31) of a block lies in tile T = t/16 at row i = t%16; stored channel c lies
 * in k-step K = c/32 (NK = W/32 k-steps), sub-group g = (c/8)%4, position s = c%8.
 * The slot of (t, c) is  S = (T*NK + K)*64 + i + 16*g.
 *
 * bf16 block (bits = 16, and every tail block), 64*W bytes: the 8 values of slot
 *   S at bytes 16*S .. 16*S + 15, channel position s at byte 16*S + 2*s
 *   (round-to-nearest-even bf16 of the input).  Unused tail rows are zero.
 * quantised block (bits b in {2, 4, 8}): [codes: 4*W*b bytes][meta]
 *   codes (32-bit little-endian words):
 *     b = 8: slot S fills words 2*S and 2*S + 1; position s at word 2*S + s/4,
 *            bit 8*(s%4);
 *     b = 4: slot S is word S; position s at bit 16*(s%2) + 4*(s/2);
 *     b = 2: sub-groups g = 2*y + x (x in {0,1}) of (t, K) share word
 *            ((T*NK + K)*16 + i)*2 + y; position s at bit 16*(s%2) + 2*(s/2) + 8*x.
 *   KIVI32 meta, 4*W bytes: for token t and channel group K (stored channels
 *     32K .. 32K+31; d and d_R are multiples of 32 so no group mixes the latent
 *     and k^R), the fp16 scale at byte 4*((T*NK + K)*16 + i) and the fp16 zero 2
 *     bytes after it.  Codes and values follow the KIVI32 rules above with the
 *     group being these 32 channels of one token.
 *   SYMROW meta, 128 bytes: for token t the bf16 scale of c[0..d-1] at byte 4*t
 *     and the bf16 scale of k^R at byte 4*t + 2 (one scale per stored vector,
 *     App. C.3), each under the SYMROW rules above with the vector as the row.
 *   Block bytes: KIVI32 4*W*(b+1); SYMROW 4*W*b + 128; bf16 64*W.
 */

/* Build the layer table of a plan (§2.2): validate every action against
 * eq. (3) (layer 0 must own a cache, §2.2/§2.3), resolve anchor_of, compute the
 * per-layer cost eq. (1), the compression ratio eq. (2), the arena layout and
 * the decode workspace size.  Host only; touches no device.
 * Errors: KVK_ERR_INVALID on any violation (message via kvk_last_error()). */
kvk_status kvk_layer_table(const kvk_dims* dims, const kvk_action* plan, kvk_table** out);

/* A batch whose sequences carry their own plans (§2.3: the selector maps each
 * input sequence to its own configuration; eq. (4) takes the realized cost per
 * sequence).  plans: host [batch][n_layers] actions, sequence b's plan at
 * plans + b * n_layers, each validated as by kvk_layer_table (for MLA the plans
 * may differ in kept width too, §2.2 eq. (3)); batch 1..KVK_MAX_BATCH_PLANS.  Sequence b is stored exactly as a one-sequence table
 * (dims with batch 1) of plans[b] would store it, at byte base_b of the arena:
 * base_0 = 0, base_{b+1} = base_b + that table's arena_bytes rounded up to 256.
 * Every other entry point accepts the table: kvk_compress_layer, kvk_append_token
 * and kvk_debug_dequantize take the batch's tensors as for one plan and serve each
 * sequence by its own plan (a sequence whose layer inherits writes nothing there);
 * GQA: one kvk_decode_attention call decodes the whole batch in one launch, each
 * sequence reading its own anchors once (its work list, one item per sequence and
 * anchor, sits at the head of the workspace, written there once per workspace and
 * layer range by kvk_decode_setup; decode calls then copy nothing).  MLA: likewise
 * one launch per phase for the batch (A1 over every (layer, sequence) at its own
 * kept width, D2 over every (sequence, anchor), C2 over every (layer, sequence)),
 * from the work list kvk_decode_setup writes; sequence b's absorbed queries and
 * partials sit in its own part of the workspace, after the list, as its one-sequence
 * table lays them out, so each sequence's output equals that table's bit for bit;
 * kvk_compress_layer_project takes the table with latent_out NULL.  kvk_read_bytes sums the sequences.  kvk_table_query reports the batch (arena_bytes, workspace_bytes,
 * n_anchors over all sequences, rho of the mean plan); its per-layer fields are
 * empty (anchor_of and layer_offset -1): use kvk_table_sequence_query.
 * Errors: KVK_ERR_INVALID, and those of kvk_layer_table for a sequence's plan. */
kvk_status kvk_layer_table_batched(const kvk_dims* dims, const kvk_action* plans, kvk_table** out);

/* Per-sequence plans: the accounting of sequence b as its one-sequence table
 * reports it, with layer_offset made absolute (base_b added): stream h of layer l
 * of sequence b starts at layer_offset[l] + h * stream_bytes[l].
 * Errors: KVK_ERR_INVALID (not a per-sequence table, b out of range). */
kvk_status kvk_table_sequence_query(const kvk_table* table, int32_t b, kvk_table_info* out);

/* Copy the table's accounting and layout into *out.  Host only. */
kvk_status kvk_table_query(const kvk_table* table, kvk_table_info* out);

/* Free a table (NULL is accepted). */
void kvk_table_destroy(kvk_table* table);

/* Workspace bytes needed by kvk_decode_attention over [layer_begin, layer_end). */
kvk_status kvk_workspace_bytes(const kvk_table* table, int32_t layer_begin, int32_t layer_end,
                               size_t* out_bytes);

/* Prefill write of one layer's cache (§2.1: an anchor writes its cache, an
 * inheriting layer writes nothing; App. C.3 quantisers).
 * GQA:
 *   k, v      : device [B][Hkv][n_tokens][d_h], dtype in_dtype (bf16 or fp32), contiguous.
 *   keep_idx  : NULL when the table has no eviction; else device int32
 *               [B][Hkv][keep_tokens], strictly increasing positions in
 *               [0, n_tokens): the stored stream is k/v at these positions, in
 *               order (composition with token eviction, §3 long context).
 * MLA (rank axis, §2.1, App. C.2):
 *   k         : the latent, device [B][n_tokens][r], dtype in_dtype; only the
 *               first d = rank coordinates of each token are read and stored.
 *   v         : the positional key k^R after RoPE, device [B][n_tokens][d_R].
 *   keep_idx  : NULL, or device int32 [B][keep_tokens] as above, per sequence.
 * Both:
 *   n_tokens  : prefill length, 1..max_tokens.
 *   arena     : device, arena_bytes; only this layer's region is written.
 * An inheriting layer returns KVK_OK without launching anything.
 * keep_idx contents are trusted: the host cannot read device memory without a
 * synchronisation, so out-of-range positions are clamped by the kernel.
 * Errors: KVK_ERR_INVALID (layer, sizes, NULL pointers, keep_idx presence),
 *         KVK_ERR_DEVICE (launch failure). */
kvk_status kvk_compress_layer(const kvk_table* table, int32_t layer, const void* k, const void* v,
                              int32_t in_dtype, int32_t n_tokens, const int32_t* keep_idx,
                              void* arena, hipStream_t stream);

/* Prefill write with the down-projection (§2.1 "Rank", App. C.2), MLA tables: each
 * stored token's latent is computed from its hidden state on the matrix cores, only
 * its first d coordinates (the layer's kept width; a deployed kernel writes only
 * those): c[:d] = W_DKV[:d, :] x, bf16 operands, fp32 accumulation, rounded to bf16.
 * [c[:d] ; k^R] is then stored exactly as kvk_compress_layer stores a latent input
 * (eviction gather, quantiser, block layout).
 *   x         : device bf16 [B][n_tokens][d_model], the hidden states; d_model a
 *               positive multiple of 32.
 *   w_dkv     : device bf16 [r][d_model]; row i maps a hidden state to latent
 *               coordinate i (rows 0 .. d-1 are read).
 *   k_rope    : device bf16 [B][n_tokens][64], the positional keys after RoPE.
 *   keep_idx  : as for kvk_compress_layer.
 *   latent_out: NULL, or device bf16 [B][n_stored][d]: the bf16 latent the write
 *               stored (test support; NULL for per-sequence tables, whose
 *               sequences may keep different widths).
 * An inheriting layer is a no-op returning KVK_OK (per sequence under
 * per-sequence plans).  All buffers 16-byte aligned.
 * Errors: KVK_ERR_INVALID (GQA table, sizes, NULL, misalignment, host memory,
 *         latent_out with per-sequence plans), KVK_ERR_DEVICE. */
kvk_status kvk_compress_layer_project(const kvk_table* table, int32_t layer, const void* x, const void* w_dkv,
                                      int32_t d_model, const void* k_rope, int32_t n_tokens,
                                      const int32_t* keep_idx, void* arena, void* latent_out, hipStream_t stream);

/* W_UK in the layout the query absorption reads (App. C.2: the content-key
 * projection folds into the query, q~ = W_UK[h]^T q_nope, so the library reads
 * W_UK[h] latent-major).  Transposes every (layer, head) matrix on the device.
 *   w_uk : device bf16 [n_layers][n_heads][nope_dim][latent_dim], the model's layout
 *          (row i of W_UK[h] maps the latent to content-key channel i).
 *   out  : device bf16 [n_layers][n_heads][latent_dim][nope_dim]; must not alias w_uk.
 * nope_dim and latent_dim multiples of 32; both buffers 16-byte aligned.  Asynchronous
 * on `stream`.  Errors: KVK_ERR_INVALID (sizes, NULL, aliasing, misalignment, host
 * memory), KVK_ERR_DEVICE. */
kvk_status kvk_mla_arrange_w_uk(const void* w_uk, int32_t n_layers, int32_t n_heads, int32_t nope_dim,
                                int32_t latent_dim, void* out, hipStream_t stream);

/* Attach an MLA table's up-projections for all its layers (App. C.2): w_uk as
 * kvk_mla_arrange_w_uk writes it, [n_layers][Hq][r][nope_dim], and w_uv
 * [n_layers][Hq][v_dim][r], both device bf16, 16-byte aligned.  Decode calls that
 * pass NULL for both weights then use these from their first layer on.  The
 * buffers stay owned by the caller and must outlive their use; NULL for both
 * detaches.  Not to be called while a decode call on the table runs on another
 * thread.  Errors: KVK_ERR_INVALID (GQA table, one weight NULL, misalignment, host
 * memory). */
kvk_status kvk_set_mla_weights(kvk_table* table, const void* w_uk, const void* w_uv);

/* Decode-time append of one generated token to every anchor layer in
 * [layer_begin, layer_end).  The plan chosen at prefill holds for the whole
 * generation (§2.3), so each anchor keeps its configuration: the new token enters
 * the stream's bf16 tail (the recent-token window that grouped quantisers keep in
 * full precision, App. C.3), and the token that fills the tail completes a
 * 32-token group, which is quantised into the next full block exactly as the
 * prefill write quantises a block (keys per channel over the group's tokens,
 * values per token).  The group is quantised from its bf16 values, so a stream
 * built by appends equals the prefill write of the same tokens rounded to bf16.
 * GQA:
 *   k, v     : device [layer_end-layer_begin][B][Hkv][d_h], dtype in_dtype: the
 *              new token's key and value per layer (rows of inheriting layers are
 *              not read).
 * MLA:
 *   k        : the new latent, device [nl][B][r] (first d = rank coordinates used);
 *   v        : the new positional key after RoPE, device [nl][B][d_R].
 * Both:
 *   n_stored : tokens stored per stream before the call (the new token's
 *              position in the stream), 0 .. stored_tokens_cap - 1; the same for
 *              every layer of the range.  Afterwards the streams hold n_stored + 1.
 *   arena    : device; only the anchors' tails and, when n_stored % 32 == 31,
 *              their full block n_stored / 32 are written.  Tail slots at and after
 *              (n_stored + 1) % 32 are left undefined; nothing reads them.
 * Under eviction the appended token is always kept (the keep list applies at
 * prefill).  Layers that inherit an anchor outside the range see the new token
 * only once that anchor's layer has been appended.
 * Errors: KVK_ERR_INVALID (range, NULL pointers, dtype, n_stored + 1 beyond the
 *         capacity, misalignment: k, v and arena 16 B), KVK_ERR_DEVICE. */
kvk_status kvk_append_token(const kvk_table* table, int32_t layer_begin, int32_t layer_end,
                            const void* k, const void* v, int32_t in_dtype, int32_t n_stored,
                            void* arena, hipStream_t stream);

/* Query-aware keep list of one anchor layer at prefill, for a table that evicts
 * (keep_tokens > 0): the eviction the paper composes with its configurations
 * (§3.4: the configurations drop no positions, so an evictor runs on the same
 * cache and the reductions multiply), computed as its eviction implementations do,
 * by summing attention over a 32-query observation window (App. F.3).  Per
 * sequence and KV head: the queries of the last 32 prompt positions of the G query
 * heads attend causally (window slot w sees positions <= n_tokens - 32 + w) with
 * softmax(scale q.k); a position's importance is the sum of its probabilities over
 * those 32 G rows; the 32 window positions are kept, plus the keep_tokens - 32
 * earlier positions of largest importance (ties to the lower position).  No
 * pooling (the paper names none).  The result feeds kvk_compress_layer's keep_idx.
 *   k         : device bf16 [B][Hkv][n_tokens][d_h], the prompt's keys after RoPE
 *               (the same tensor kvk_compress_layer takes).
 *   q_obs     : device bf16 [B][Hq][32][d_h], the queries of the last 32 positions.
 *   n_tokens  : keep_tokens .. max_tokens.
 *   scale     : softmax scale.
 *   keep_out  : device int32 [B][Hkv][keep_tokens], written in increasing order.
 *   importance: NULL, or device fp32 [B][Hkv][n_tokens] receiving the importances.
 *   workspace : device, >= kvk_snapkv_workspace_bytes(table, n_tokens), 256-byte aligned.
 * Scores are products of the bf16 inputs accumulated in fp32; the selection is
 * exact for the importances it computes (fp32).  An inheriting layer returns
 * KVK_OK and writes nothing.
 * Errors: KVK_ERR_INVALID (table without eviction or keep_tokens < 32, sizes, NULL
 *         pointers, misalignment), KVK_ERR_UNSUPPORTED (MLA table: kvk_snapkv_select_mla; dtype other than
 *         bf16, more than 8 query heads per KV head, d_h other than 64 or 128),
 *         KVK_ERR_BUFFER (workspace), KVK_ERR_DEVICE. */
kvk_status kvk_snapkv_workspace_bytes(const kvk_table* table, int32_t n_tokens, size_t* out_bytes);

/* The query-aware keep list of one MLA anchor layer (§3.4, App. F.3 as above; the
 * rank axis of §2.1 and App. C.2): the latent is shared by every head, so a
 * sequence keeps one list of positions.  Head h's key at position t is
 * [W_UK[h] c_t ; k^R_t] with the latent at its full width r (the layer then stores
 * the first d coordinates of the kept tokens); a position's importance sums the
 * causal softmax probabilities of the 32 window queries of every query head; the
 * selection rule is kvk_snapkv_select's.  Computed in the absorbed form: the window
 * queries are absorbed (q~ = W_UK[h]^T q_nope, fp16) and scored against the latent
 * on the matrix cores (fp16 products, fp32 accumulation).
 *   latent    : device bf16 [B][n_tokens][r] (the tensor kvk_compress_layer takes).
 *   k_rope    : device bf16 [B][n_tokens][64], the positional keys after RoPE.
 *   q_obs     : device bf16 [B][32][Hq][nope_dim + 64], the window queries (per head
 *               the no-RoPE part, then the RoPE part).
 *   w_uk      : device bf16 [Hq][r][nope_dim], this layer's W_UK as
 *               kvk_mla_arrange_w_uk writes it; NULL: the attached weights' layer.
 *   keep_out  : device int32 [B][keep_tokens], increasing.
 *   importance: NULL, or device fp32 [B][n_tokens].
 *   workspace : device, >= kvk_snapkv_workspace_bytes(table, n_tokens), 256-byte aligned.
 * latent_dim 256, 512, 768 or 1024.  An inheriting layer (one-plan tables) returns
 * KVK_OK and writes nothing; per-sequence tables score every sequence.
 * Errors: KVK_ERR_INVALID (GQA table, no eviction or keep_tokens < 32, sizes, NULL,
 *         no weights, misalignment), KVK_ERR_UNSUPPORTED (latent_dim),
 *         KVK_ERR_BUFFER (workspace), KVK_ERR_DEVICE. */
kvk_status kvk_snapkv_select_mla(const kvk_table* table, int32_t layer, const void* latent, const void* k_rope,
                                 const void* q_obs, const void* w_uk, int32_t n_tokens, float scale,
                                 int32_t* keep_out, float* importance, void* workspace, size_t ws_bytes,
                                 hipStream_t stream);
kvk_status kvk_snapkv_select(const kvk_table* table, int32_t layer, const void* k, const void* q_obs,
                             int32_t in_dtype, int32_t n_tokens, float scale, int32_t* keep_out,
                             float* importance, void* workspace, size_t ws_bytes, hipStream_t stream);

/* The selector's forward pass (§2.3; App. B "Selector architecture"): the prompt's
 * token embeddings (the backbone's own) -> a linear map to width 256 -> two
 * bidirectional pre-norm transformer blocks -> a final RMSNorm -> the average over
 * the prompt -> an optional budget scale and shift (App. B "Budget conditioning":
 * z * (1 + gamma) + beta) -> one linear head per layer -> the argmax action of each
 * layer.  Run once per prompt at prefill; the actions build the plan that is held
 * for the whole generation.
 * Block: x += W_o Attn(RMSNorm(x)), then x += W_down (SiLU(W_gate n) * W_up n) with
 * n = RMSNorm(x); RMSNorm is x / sqrt(mean(x^2) + 1e-6) * gain; attention has 4
 * heads of 64 over every position with scale 1/8 and rotary embeddings on q and k
 * (token t at position t, base 10000, channel i of a head paired with i + 32 and
 * turned by t * 10000^(-i/32)); the trunk's linear maps have no bias, the heads do.
 * Actions (eq. (3)): index 0 = inherit (depth); 1 + 4 j + k = produce with kept
 * width r / 2^j at 16 / 2^k bits (j, k = 0..3): 17 actions for the composed space;
 * a GQA selector (precision and depth) uses the first 5 (inherit, bf16, int8, int4,
 * int2).  The depth logit is -inf at layer 0, and at every layer when depth = 0.
 *   d_model  : the embedding width, a multiple of 32; n_layers 1..64;
 *   n_actions: 2..32 logits per layer;
 *   weights  : device bf16, kvk_selector_weight_elems(d_model, n_layers, n_actions)
 *              elements, packed in this order, each matrix [out][in] row-major:
 *              w_in [256][d_model]; then per block (two): g_attn [256],
 *              w_qkv [768][256] (q, k, v rows; head h uses rows 64h .. 64h+63 of
 *              each), w_o [256][256], g_ffn [256], w_gate [1024][256],
 *              w_up [1024][256], w_down [256][1024]; then g_final [256],
 *              w_head [n_layers][n_actions][256], b_head [n_layers][n_actions].
 *   emb      : device bf16 [n_tokens][d_model].
 *   film     : NULL (no conditioning), or device fp32 [2][256]: gamma, then beta.
 *   logits   : NULL, or device fp32 [n_layers][n_actions] (fp32; bf16 operands).
 *   actions  : device int32 [n_layers], the argmax (lowest index on ties).
 *   workspace: device, >= kvk_selector_workspace_bytes(...), 256-byte aligned.
 * kvk_selector_weight_elems returns -1 for sizes outside those ranges.
 * Errors: KVK_ERR_INVALID (sizes, NULL pointers, misalignment), KVK_ERR_BUFFER,
 *         KVK_ERR_DEVICE. */
int64_t kvk_selector_weight_elems(int32_t d_model, int32_t n_layers, int32_t n_actions);
kvk_status kvk_selector_workspace_bytes(int32_t d_model, int32_t n_layers, int32_t n_tokens, size_t* out_bytes);
kvk_status kvk_selector_forward(int32_t d_model, int32_t n_layers, int32_t n_actions, int32_t depth,
                                const void* weights, const void* emb, int32_t n_tokens, const float* film,
                                float* logits, int32_t* actions, void* workspace, size_t ws_bytes,
                                hipStream_t stream);

/* Set-up for decoding layers [layer_begin, layer_end) with `workspace` (§2.3: a
 * plan is chosen once per prompt and held for every decode step, so this runs once
 * per table, layer range and workspace, not per step).  Per-sequence tables
 * (kvk_layer_table_batched): writes the decode work list (one item per sequence and
 * anchor of its plan, laid out for the capacity, so valid for every n_stored) to the
 * head of `workspace` (kvk_workspace_bytes of the range) and waits for the copy (it
 * synchronises `stream`; do not call it inside graph capture).  The table records
 * the workspace; kvk_decode_attention, kvk_decode_splits and kvk_decode_merge on a
 * per-sequence table then require a prior set-up of the same workspace and layer
 * range (else KVK_ERR_INVALID), copy nothing and never synchronise.  The workspace
 * must keep its list (and stay allocated) while it is used for decoding: a set-up
 * of another range on the same workspace replaces the record; a list that does not
 * match the call's (a workspace overwritten since) makes the kernels write NaN
 * outputs and read nothing through it.  MLA per-sequence tables: the list holds a
 * row per (layer, sequence) (kept width, where its absorbed queries and split
 * partials sit, its anchor's split rule) and an item per (sequence, anchor) for each
 * decode launch; the splits of a call follow from its n_stored in the kernels.
 * One-plan tables: a no-op (the work list travels in the kernel arguments).
 * Errors: KVK_ERR_INVALID (range, NULL), KVK_ERR_BUFFER (workspace too small),
 *         KVK_ERR_DEVICE (the copy). */
kvk_status kvk_decode_setup(const kvk_table* table, int32_t layer_begin, int32_t layer_end, void* workspace,
                            size_t workspace_bytes, hipStream_t stream);

/* One decode step of attention for layers [layer_begin, layer_end) (§2.1): layer l
 * uses its own query and the cache of anchor_of[l].  Layers in the range that
 * share an anchor are served by one read of that anchor's bytes.
 * GQA:
 *   q        : device [layer_end-layer_begin][B][Hq][d_h], dtype q_dtype.
 *   w_uk, w_uv: must be NULL.
 *   out      : device fp32 [layer_end-layer_begin][B][Hq][d_h].
 * MLA (§2.1, App. C.2), with nl = layer_end - layer_begin:
 *   q        : device [nl][B][Hq][nope_dim + d_R], dtype q_dtype: per head the
 *              no-RoPE part q_nope then the RoPE part q_rope.
 *   w_uk     : device bf16 [nl][Hq][r][nope_dim]: layer l's W_UK, the map from the
 *              latent to head h's content key (k = W_UK[h] c), stored transposed
 *              (latent-major: element (i, c) of W_UK[h] at [h][c][i]), the layout the
 *              query absorption reads contiguously (kvk_mla_arrange_w_uk makes it
 *              from the model's layout once, at weight load).
 *   w_uv     : device bf16 [nl][Hq][v_dim][r]: layer l's W_UV (v = W_UV[h] c).
 *   Both NULL: the weights attached by kvk_set_mla_weights, from layer_begin on
 *              (KVK_ERR_INVALID if none are attached); pass both or neither.
 *   out      : device fp32 [nl][B][Hq][v_dim].
 *   Head h of layer l attends with query [q_nope ; q_rope] to keys
 *   [W_UK[h] c_t ; k^R_t] and values W_UV[h] c_t, where c_t is the stored latent
 *   of token t zero-extended from the anchor's d to r.  The library computes it
 *   with the projections moved onto the query and the output (App. C.2):
 *   q~ = W_UK[h][:, :d]^T q_nope, scores over [c_t[:d] ; k^R_t], then
 *   out = W_UV[h][:, :d] (softmax-weighted sum of c_t[:d]).
 * Both:
 *   n_stored : stored tokens per stream, 0..stored_tokens_cap (the prefill
 *              n_tokens, or keep_tokens under eviction).  n_stored = 0 yields zeros.
 *   scale    : softmax scale applied to the query-key dot product.
 *   workspace: device, >= kvk_workspace_bytes(...) bytes, 256-byte aligned; its
 *              contents on entry are ignored.
 * Calls that overlap on one workspace race.
 * Errors: KVK_ERR_INVALID, KVK_ERR_BUFFER (workspace too small), KVK_ERR_DEVICE. */
kvk_status kvk_decode_attention(const kvk_table* table, int32_t layer_begin, int32_t layer_end,
                                const void* q, int32_t q_dtype, int32_t n_stored, float scale,
                                const void* w_uk, const void* w_uv, const void* arena,
                                float* out, void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

/* The two phases of kvk_decode_attention, for callers that schedule or time them
 * separately.  kvk_decode_splits runs the attention split along the context and
 * leaves the split partials in `workspace` (GQA: over the full 32-token blocks;
 * MLA: the absorbed queries, then every stored token, tail included);
 * kvk_decode_merge merges the partials by log-sum-exp into `out` (GQA: after
 * attending to the bf16 tail tokens; MLA: followed by the W_UV up-projection).
 * The merge must use the same table, layer range, q, n_stored, scale, weights,
 * arena and workspace as the splits call before it on the same stream.  Errors
 * as for kvk_decode_attention. */
kvk_status kvk_decode_splits(const kvk_table* table, int32_t layer_begin, int32_t layer_end,
                             const void* q, int32_t q_dtype, int32_t n_stored, float scale,
                             const void* w_uk, const void* w_uv, const void* arena,
                             void* workspace, size_t workspace_bytes, hipStream_t stream);
kvk_status kvk_decode_merge(const kvk_table* table, int32_t layer_begin, int32_t layer_end,
                            const void* q, int32_t q_dtype, int32_t n_stored, float scale,
                            const void* w_uk, const void* w_uv, const void* arena,
                            const void* workspace, size_t workspace_bytes, float* out,
                            hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): kvk_decode_attention with
 * no workspace argument.  The split partials (and, for MLA tables, the absorbed
 * queries) go to a static device array of KVK_NOALLOC_SCRATCH_BYTES that the
 * library holds on each GPU it runs on, from the first call on that GPU until the
 * process ends.  The call allocates nothing (no hipMalloc, no host heap on this
 * path) and runs the same kernels, so its output equals kvk_decode_attention's.
 * Arguments as for kvk_decode_attention; the GPU is the stream's (the current
 * device for the null stream).
 * Every call on one GPU shares that GPU's scratch: calls that overlap on one GPU
 * (on different streams, or from different threads) race.
 * Errors: those of kvk_decode_attention; KVK_ERR_UNSUPPORTED for a per-sequence
 * table, or when the layer range needs more than KVK_NOALLOC_SCRATCH_BYTES of
 * scratch (kvk_workspace_bytes of the range; decode fewer layers per call), before
 * any launch. */
#define KVK_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
kvk_status kvk_decode_attention_noalloc(const kvk_table* table, int32_t layer_begin, int32_t layer_end,
                                        const void* q, int32_t q_dtype, int32_t n_stored, float scale,
                                        const void* w_uk, const void* w_uv, const void* arena, float* out,
                                        hipStream_t stream);

/* Algorithmic bytes one decode call over [layer_begin, layer_end) reads from the
 * arena with n_stored tokens per stream: each distinct anchor's full blocks and
 * bf16 tail tokens, counted once (split partials, queries, MLA up-projection
 * weights and outputs excluded).  Host only. */
kvk_status kvk_read_bytes(const kvk_table* table, int32_t layer_begin, int32_t layer_end,
                          int32_t n_stored, int64_t* out_bytes);

/* Test support: dequantise the cache read by `layer` (its anchor's) into fp32,
 * using the rules above bit for bit.  GQA: k_out, v_out [B][Hkv][n_stored][d_h].
 * MLA: k_out = the stored latent [B][n_stored][d], v_out = k^R [B][n_stored][d_R];
 * under per-sequence plans sequence b's latent starts at b * n_stored * r, in rows of
 * its own anchor's kept width d_b. */
kvk_status kvk_debug_dequantize(const kvk_table* table, int32_t layer, int32_t n_stored,
                                const void* arena, float* k_out, float* v_out, hipStream_t stream);

/* Storage accounting of App. C.3 (table of storage cost with quantisation
 * metadata): bits per cached element for `bits`-bit codes with 32 bits of
 * metadata per `group` elements (grouped schemes, KVK_Q_KIVI32 and KVK_Q_GROUP64, the
 * latter with group 64 as stored) or one bf16 scale
 * per 128-element row (KVK_Q_SYMROW, group ignored), with `window` of the
 * `context` tokens kept in bf16.  Returns a negative value on invalid input. */
double kvk_realized_bits(int32_t qscheme, int32_t bits, int32_t group, int64_t window,
                         int64_t context);

/* eq. (5): rho_min / rho_max over the actions a layer may take.
 *   axes bit 0 = precision (B = {2,4,8,16}, else {16}), bit 1 = rank (MLA,
 *   D = {r/8, r/4, r/2, r}, else {r} for MLA / the full GQA width), bit 2 = depth.
 *   mla selects the MLA cost (d + d_R) b with r = latent_dim, else the GQA cost
 *   2*Hkv*d_h*b.  C0 = L * kv_width * 16 with kv_width = 2*Hkv*d_h. */
kvk_status kvk_rho_range(int32_t n_layers, int32_t kv_width, int32_t latent_dim, int32_t rope_dim,
                         int32_t mla, int32_t axes, double* rho_min, double* rho_max);

const char* kvk_last_error(void);
const char* kvk_version(void);

#ifdef __cplusplus
}
#endif
#endif /* KVK_H */
