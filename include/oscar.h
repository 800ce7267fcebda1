/*
 * liboscar -- INT2 KV-cache append and paged decode attention for OSCAR
 * (arXiv 2605.17757) on AMD Instinct MI355X (gfx950).
 *
 * The cache stores every key and value row rotated by a fixed orthogonal matrix,
 * clipped, and quantized to asymmetric 2-bit codes per group of G channels with
 * a binary16 scale and zero (Sec. 4 "KV Cache Update"; App. "Scale
 * Determination and Per-token Clipping Details").  Decode attention reads the
 * codes through a block table (paged cache, Sec. 4 "KV Cache Layout") and
 * computes softmax(q K^T / sqrt(d)) V against the reconstructed rows
 * K^ = Q(K R_k) R_k^T, V^ = Q(V R_v) R_v^T (Sec. 2 quantization notation;
 * Alg. 1 DecodeStep) as a split-K flash-decoding pass with a log-sum-exp merge
 * (Sec. 4 "Decoding Attention Kernel").
 *
 * Plain C, no HIP include: load it with any FFI.
 *
 * Conventions for every entry point
 *   - Pointers named in the argument lists are DEVICE pointers unless marked
 *     "host".  The caller owns and allocates every buffer: pages, inputs,
 *     rotation matrices, workspace and output.  The library never allocates.
 *   - Calls are asynchronous on `stream` (a hipStream_t passed as void*; NULL
 *     is the default stream).  OSCAR_OK means "validated and launched".
 *     OSCAR_ERR_HIP reports a launch error (hipGetLastError right after the
 *     launch); asynchronous faults surface at the caller's next synchronization.
 *   - Host arguments are validated before anything is launched; on any error
 *     nothing is launched and no memory is touched.  Device-resident indices
 *     (slot_mapping, block_table, seq_lens, seq_idx) are not validated by
 *     default: they must lie in range (slot < num_pages*page_size, 0 <= page id
 *     < num_pages, 1 <= seq_lens[b] <= max_pages_per_seq*page_size, 0 <=
 *     seq_idx < B).  With the environment variable OSCAR_DEBUG set (and not
 *     "0", read at every call) the entry points that take them synchronize the
 *     stream, copy them to host memory and check them first: seq_lens[b] in
 *     [0, max_pages_per_seq*page_size], the block-table entries of the pages a
 *     sequence uses in [0, num_pages), slots below num_pages*page_size
 *     (negative slots are skipped by the cache update), seq_idx in [0, B); an
 *     index out of range returns OSCAR_ERR_INVALID_ARG with nothing launched,
 *     a failed copy OSCAR_ERR_HIP.
 *   - Inputs must be finite.  Scales and zeros that fall outside the range of
 *     their storage format are saturated to its largest finite value (+-65504
 *     for binary16).
 *   - A rotation matrix argument (R_k, R_v) may be NULL: the identity, e.g.
 *     R_V absorbed into the value and output projections (Sec. 4 "KV Cache
 *     Update").  The same choice must be used for the cache update and decode.
 *   - L->rot_per_head = 1: every non-NULL R_k, R_v is an fp32 [Hkv][d][d] array,
 *     one matrix per KV head (row (token, h) and the query heads of KV head h use
 *     matrix h); 0 (default): one [d][d] matrix for all heads, as the paper
 *     deploys it (one rotation per layer, GQA-averaged).
 *   - Supported shapes: head_dim 128, page_size 64, group_size 32, 64 or 128.  Other values
 *     return OSCAR_ERR_UNSUPPORTED; an unknown clip_mode or meta_dtype returns
 *     OSCAR_ERR_INVALID_ARG.
 *
 * Page byte layout (an ABI: any producer/consumer of the pool must follow it).
 *   A pool of num_pages pages; page p, kv-head h is the block starting at byte
 *   (p*Hkv + h) * B_ph, B_ph = 2*P*d/4 + 2*(d/G)*P*4  (6144 bytes for d=128,
 *   P=64, G=32).  Inside a block, for token slot t in [0,P) and channel c:
 *     [K codes]  P*d/4 bytes, token-major:  byte t*(d/4) + c/4
 *     [V codes]  P*d/4 bytes, quad-major:   byte P*d/4 + (c/4)*P + t
 *     [K s,z]    (d/G)*P 4-byte entries, group-major: entry (c/G)*P + t
 *     [V s,z]    same, after the K entries
 *   A code byte holds the four channels 4j..4j+3 of one token; channel c sits
 *   in bits 2*(c%4)..2*(c%4)+1.  An s,z entry is the scale followed by the
 *   zero point, each a little-endian binary16 (meta_dtype F16) or bfloat16
 *   (BF16).  The stored row is
 *   Q(x~)_c = s * (code_c - z).
 */
#ifndef OSCAR_H
#define OSCAR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  OSCAR_OK = 0,
  OSCAR_ERR_INVALID_ARG = 1,         /* null pointer, negative size, bad ratio ... */
  OSCAR_ERR_UNSUPPORTED = 2,         /* valid but unsupported shape               */
  OSCAR_ERR_WORKSPACE_TOO_SMALL = 3, /* workspace_bytes below the required size   */
  OSCAR_ERR_HIP = 4                  /* the HIP runtime reported an error         */
} oscar_status;

typedef enum { OSCAR_OUT_BF16 = 0, OSCAR_OUT_F32 = 1 } oscar_dtype;

/* Clip threshold of the quantizer (App. "Scale Determination and Per-token
 * Clipping Details"), with clip = clip_k or clip_v of the call:
 *   GROUP_ABSMAX   : tau = clip * max|x~| over each group of G channels;
 *   TOKEN_QUANTILE : tau = the clip-quantile of |x~| over the token's d channels
 *                    (the same tau for every group): sorted a_0 <= ... <= a_{d-1},
 *                    pos = clip * (d - 1), k = floor(pos), f = pos - k,
 *                    tau = a_k + f * (a_{k+1} - a_k) (tau = a_{d-1} if k = d - 1),
 *                    each step one fp32 operation. */
typedef enum { OSCAR_CLIP_GROUP_ABSMAX = 0, OSCAR_CLIP_TOKEN_QUANTILE = 1 } oscar_clip_mode;

/* Storage format of the per-group scale and zero point. */
typedef enum { OSCAR_META_F16 = 0, OSCAR_META_BF16 = 1 } oscar_meta_dtype;

/* Geometry and quantizer format of one layer's page pool.  Host struct, read
 * only.  Zero-initialized trailing fields give the default format. */
typedef struct {
  int32_t head_dim;     /* d, channels per head (128)                 */
  int32_t num_kv_heads; /* Hkv >= 1                                   */
  int32_t page_size;    /* P, token slots per page (64)               */
  int32_t group_size;   /* G, channels per quantization group (32)    */
  int64_t num_pages;    /* pages in the pool (>= 1)                   */
  int32_t clip_mode;    /* oscar_clip_mode (default GROUP_ABSMAX)     */
  int32_t meta_dtype;   /* oscar_meta_dtype (default F16)             */
  int32_t rot_per_head; /* 0: one R_k, R_v per layer; 1: one per KV head */
} oscar_layout;

/* Human-readable name of a status code (static storage). */
const char *oscar_status_string(int status);

/* Bytes of one page (all kv-heads): Hkv * B_ph.  0 if L is invalid. */
size_t oscar_page_bytes(const oscar_layout *L);

/* Bytes of the whole pool: num_pages * oscar_page_bytes(L). */
size_t oscar_pool_bytes(const oscar_layout *L);

/* Check a layout; OSCAR_OK if the library supports it. */
int oscar_layout_check(const oscar_layout *L);

/*
 * oscar_kv_append -- the cache update (Sec. 4 "KV Cache Update"; App. "Scale
 * Determination and Per-token Clipping Details"; Alg. 1 QuantizeAndWrite).
 * For each new token i and kv-head h, and for X in {K, V}:
 *   x~ = x R_X                      rotation, x~_j = sum_c x_c R_X[c][j]
 *                                   (summed in fp64, rounded once to fp32;
 *                                   R_X NULL: x~ = x)
 *   tau                             clipping threshold of L->clip_mode with
 *                                   clip_X (see oscar_clip_mode)
 *   per group g of G channels:
 *     y   = min(max(x~, -tau), tau)
 *     a = min y, b = max y, s = M((b - a)/3), z = M(-a / s)
 *     code = clamp(round_half_even(y / s + z), 0, 3)
 *   where M rounds to the metadata format (L->meta_dtype, nearest even); a
 *   group whose stored scale is 0 stores s = 1, z = M(-a), codes 0; a zero
 *   point of 0 is stored as +0.  Packed into the slot per the page layout.
 *   k_new, v_new : bf16 [n_tok, Hkv, d], row-major
 *   slot_mapping : int64 [n_tok], slot = page_id * P + offset; slots must be
 *                  distinct within one call
 *   R_k, R_v     : fp32 [d, d], row-major, orthogonal, or NULL (identity)
 *   clip_k/_v    : ratios in (0, 1]; 1 disables clipping
 * n_tok == 0 launches nothing.  Only the addressed slots are written.
 */
int oscar_kv_append(const oscar_layout *L, void *pages, const void *k_new, const void *v_new,
                    const int64_t *slot_mapping, int32_t n_tok, const float *R_k,
                    const float *R_v, float clip_k, float clip_v, void *stream);

/*
 * Workspace for decode: bytes needed by oscar_decode_attn (and its stages) for
 * B sequences, Hq query heads and num_splits splits per sequence.
 */
size_t oscar_decode_workspace_bytes(const oscar_layout *L, int32_t B, int32_t Hq,
                                    int32_t num_splits);

/*
 * A split count for B sequences whose longest context is max_seq_len tokens
 * (>= 1).  oscar_decode_attn divides the pages of all sequences evenly among the
 * GPU's resident waves (about 16 per compute unit, ranges of at least 4 pages);
 * num_splits bounds the number of partial states of one (sequence, head) row,
 * and the returned value allows the cut that an average sequence length of half
 * the longest produces (>= 2 unless the longest sequence has < 4 pages).
 */
int32_t oscar_default_num_splits(const oscar_layout *L, int32_t B, int32_t Hq,
                                 int32_t max_seq_len);

/*
 * oscar_decode_attn -- one decode step of attention for B sequences over the
 * INT2 cache (Alg. 1 DecodeStep; Sec. 4 "Decoding Attention Kernel").
 * For sequence b and query head h (kv-head h / (Hq/Hkv)):
 *   o = softmax(sm_scale * q K^T) V,  K^ = Q(K~) R_k^T,  V^ = Q(V~) R_v^T,
 * over the cached tokens t < seq_lens[b], evaluated as
 *   q~ = q R_k;  scores against Q(K~);  o~ = softmax-weighted sum of Q(V~);
 *   o = o~ R_v^T,
 * split along the sequences and merged with a log-sum-exp reduce: the pages of
 * all sequences are laid end to end and cut into equal ranges (one wave per
 * range and kv-head, about 16 waves per compute unit in all), each range at
 * least ceil(max_pages_per_seq / (num_splits - 1)) pages so that a row gets at
 * most num_splits partial states (num_splits == 1: one range per sequence).  The result does not
 * depend on the cut beyond fp32 rounding.  No host synchronization, no
 * allocation.
 *   q            : bf16 [B, Hq, d]; Hq % Hkv == 0, Hq/Hkv <= 16
 *   block_table  : int32 [B, max_pages_per_seq]; token t of sequence b is in
 *                  page block_table[b][t / P], slot t % P
 *   seq_lens     : int32 [B], tokens in cache, 1 <= seq_lens[b] <=
 *                  max_pages_per_seq * P (the current token already appended);
 *                  values outside are clamped to [0, max_pages_per_seq * P],
 *                  and a sequence of length 0 gives a zero output
 *   sm_scale     : logit scale, 1/sqrt(d) for standard attention
 *   num_splits   : >= 1, or 0 for oscar_default_num_splits(L, B, Hq,
 *                  max_pages_per_seq * P)
 *   workspace    : >= oscar_decode_workspace_bytes(L, B, Hq, num_splits) bytes,
 *                  256-byte aligned, contents need no initialization
 *   out          : [B, Hq, d] of out_dtype (bf16 is the round-to-nearest-even
 *                  of the fp32 result)
 */
int oscar_decode_attn(const oscar_layout *L, const void *pages, const void *q, int32_t B,
                      int32_t Hq, const int32_t *block_table, int32_t max_pages_per_seq,
                      const int32_t *seq_lens, const float *R_k, const float *R_v,
                      float sm_scale, int32_t num_splits, void *workspace,
                      size_t workspace_bytes, void *out, oscar_dtype out_dtype, void *stream);

/* Size of the device scratch array behind oscar_decode_attn_noalloc. */
#define OSCAR_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

/*
 * oscar_decode_attn_noalloc -- oscar_decode_attn without a workspace argument,
 * for callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc).  It computes exactly
 * what oscar_decode_attn computes with the same arguments (same kernels) and
 * allocates nothing: the workspace is a 64 MiB array in the library's device
 * data (OSCAR_NOALLOC_SCRATCH_BYTES), one copy per GPU, held from the library's
 * load until the process ends; its address is looked up once per device on the
 * first call made with that device current.
 *   Arguments as in oscar_decode_attn.  A call whose workspace
 *   (oscar_decode_workspace_bytes(L, B, Hq, num_splits) with num_splits
 *   resolved) exceeds OSCAR_NOALLOC_SCRATCH_BYTES returns
 *   OSCAR_ERR_WORKSPACE_TOO_SMALL with nothing launched; a failed address
 *   lookup returns OSCAR_ERR_HIP.
 *   Every call on one GPU uses that GPU's one array (no initialization is
 *   needed: each call writes every entry it reads), so calls that may overlap
 *   on one GPU (other streams, other host threads) race: order them on one
 *   stream or serialize them.
 */
int oscar_decode_attn_noalloc(const oscar_layout *L, const void *pages, const void *q, int32_t B,
                              int32_t Hq, const int32_t *block_table, int32_t max_pages_per_seq,
                              const int32_t *seq_lens, const float *R_k, const float *R_v,
                              float sm_scale, int32_t num_splits, void *out,
                              oscar_dtype out_dtype, void *stream);

/*
 * oscar_decode_step -- one serving decode step (Alg. 1 DecodeStep): write the
 * n_new newest tokens' K/V into the cache (exactly oscar_kv_append), then
 * decode attention over the cache including them (exactly oscar_decode_attn),
 * in three launches instead of four: the cache update and the query rotation
 * share one launch.  Arguments as in oscar_kv_append and oscar_decode_attn; n_new
 * may be 0 (no update; k_new, v_new, slot_mapping may then be NULL).  Every
 * argument is validated before anything is launched.
 */
int oscar_decode_step(const oscar_layout *L, void *pages, const void *k_new, const void *v_new,
                      const int64_t *slot_mapping, int32_t n_new, float clip_k, float clip_v,
                      const void *q, int32_t B, int32_t Hq, const int32_t *block_table,
                      int32_t max_pages_per_seq, const int32_t *seq_lens, const float *R_k,
                      const float *R_v, float sm_scale, int32_t num_splits, void *workspace,
                      size_t workspace_bytes, void *out, oscar_dtype out_dtype, void *stream);

/*
 * The three stages of oscar_decode_attn, for callers that schedule or time
 * them separately.  Called in this order on one stream with the same
 * arguments they equal one oscar_decode_attn call.
 *   prepare : q~ = q R_k scaled by sm_scale*log2(e), into the workspace.
 *   split   : partial softmax states over page ranges (see above), into the
 *             workspace.
 *   reduce  : log-sum-exp merge of the splits, o = o~ R_v^T, into out.
 */
int oscar_decode_prepare(const oscar_layout *L, const void *q, int32_t B, int32_t Hq,
                         const float *R_k, float sm_scale, int32_t num_splits,
                         void *workspace, size_t workspace_bytes, void *stream);
int oscar_decode_split(const oscar_layout *L, const void *pages, int32_t B, int32_t Hq,
                       const int32_t *block_table, int32_t max_pages_per_seq,
                       const int32_t *seq_lens, int32_t num_splits, void *workspace,
                       size_t workspace_bytes, void *stream);
int oscar_decode_reduce(const oscar_layout *L, int32_t B, int32_t Hq, const float *R_v,
                        int32_t num_splits, void *workspace, size_t workspace_bytes, void *out,
                        oscar_dtype out_dtype, void *stream);

/*
 * Mixed-precision cache (Sec. 4 "KV Cache Layout"; Alg. 1 DecodeStep): the
 * first S0 tokens of a sequence (attention sink) and its W most recent tokens
 * stay in bf16; only the history between them is INT2.  At length n the cache
 * of a sequence is
 *   bf16 sink [0, lo), INT2 history [lo, hi), bf16 window [hi, n),
 *   lo = min(S0, n), hi = max(lo, n - W)
 * (S0 = W = 0: everything INT2, as oscar_kv_append / oscar_decode_attn).  The
 * history lives in the paged pool at its own positions (block table as above);
 * pool slots of sink and window positions are never written or read.  The bf16
 * rows live in a segment store owned by the caller, an ABI like the page layout:
 *   K(b, h, slot, c) at bf16 element (((b*Hkv + h)*2 + 0)*(S0+W) + slot)*d + c
 *   V(b, h, slot, c) at bf16 element (((b*Hkv + h)*2 + 1)*(S0+W) + slot)*d + c
 * position p < S0 uses slot p, a window position p >= S0 uses slot
 * S0 + (p - S0) mod W.  S0 and W are arguments of every call and must stay the
 * same for the life of a cache; 0 <= S0, 0 <= W, S0 + W <= 65536.
 */

/* Bytes of the segment store for B sequences: B * Hkv * 2 * (S0+W) * d * 2. */
size_t oscar_seg_bytes(const oscar_layout *L, int32_t B, int32_t S0, int32_t W);

/* Workspace of oscar_decode_attn_mixed / oscar_decode_step_mixed: rows of
 * num_splits + 1 partial states (the INT2 pieces and one for the bf16 tokens). */
size_t oscar_mixed_workspace_bytes(const oscar_layout *L, int32_t B, int32_t Hq,
                                   int32_t num_splits);

/*
 * oscar_mixed_append -- build the mixed cache from a prompt: token i of sequence
 * seq_idx[i] (int32, in [0, B)) at position pos[i] (int64) is written where a
 * cache of length seq_lens[b] keeps it: positions in the history [lo, hi) are
 * rotated, clipped and INT2-quantized into the pool exactly as by
 * oscar_kv_append (slot block_table[b][p / P] * P + p % P); sink and window
 * positions are copied into their segment slot; positions outside
 * [0, seq_lens[b]) are skipped.  Tokens already in the cache are not moved: call
 * it once with a sequence's whole prompt, then advance with
 * oscar_decode_step_mixed.  Two tokens of one call must not share a slot (pool
 * or segment).  k, v: bf16 [n_tok, Hkv, d]; other arguments as in
 * oscar_kv_append and oscar_decode_attn.  n_tok == 0 launches nothing.
 */
int oscar_mixed_append(const oscar_layout *L, void *pages, void *seg, int32_t B, int32_t S0,
                       int32_t W, const void *k, const void *v, const int32_t *seq_idx,
                       const int64_t *pos, int32_t n_tok, const int32_t *block_table,
                       int32_t max_pages_per_seq, const int32_t *seq_lens, const float *R_k,
                       const float *R_v, float clip_k, float clip_v, void *stream);

/*
 * oscar_decode_attn_mixed -- decode attention over the mixed cache (Alg. 1
 * DecodeStep): o = softmax(sm_scale * q K^T) V over all n = seq_lens[b] tokens,
 * with bf16 K, V rows for the sink and window and K^ = Q(K~) R_k^T,
 * V^ = Q(V~) R_v^T for the history.  The history is split and evaluated in the
 * rotated basis as in oscar_decode_attn (num_splits pieces at most); the bf16
 * tokens give one more partial state in the original basis; the merge computes
 *   o = (sum_pieces e_s o~_s R_v^T + e_b o_b) / (sum_pieces e_s l_s + e_b l_b).
 * Arguments as in oscar_decode_attn, plus seg (may be NULL when S0 = W = 0) and
 * S0, W; workspace >= oscar_mixed_workspace_bytes(L, B, Hq, num_splits).
 */
int oscar_decode_attn_mixed(const oscar_layout *L, const void *pages, const void *seg,
                            int32_t S0, int32_t W, const void *q, int32_t B, int32_t Hq,
                            const int32_t *block_table, int32_t max_pages_per_seq,
                            const int32_t *seq_lens, const float *R_k, const float *R_v,
                            float sm_scale, int32_t num_splits, void *workspace,
                            size_t workspace_bytes, void *out, oscar_dtype out_dtype,
                            void *stream);

/*
 * oscar_decode_step_mixed -- one serving decode step over the mixed cache (Alg.
 * 1 DecodeStep): every sequence b gains one token, k_new[b], v_new[b] (bf16
 * [B, Hkv, d]), at position p = seq_lens[b] - 1 (seq_lens counts it):
 *   p < S0          -> it joins the bf16 sink (slot p);
 *   p >= S0, W = 0  -> it is INT2-quantized into the pool at position p;
 *   otherwise       -> it joins the bf16 window; when p - W >= S0 the window's
 *                      oldest token (position p - W, in the same segment slot)
 *                      is first INT2-quantized into the pool at position p - W
 *                      (QuantizeAndWrite of its bf16 row).
 * Then decode attention over the updated cache, exactly oscar_decode_attn_mixed.
 * Four launches: update + query rotation, INT2 split, bf16 partial, merge.  A
 * sequence with seq_lens[b] = 0 gets no update and a zero output.  Arguments as
 * in oscar_decode_attn_mixed and oscar_kv_append.
 */
int oscar_decode_step_mixed(const oscar_layout *L, void *pages, void *seg, int32_t S0,
                            int32_t W, const void *k_new, const void *v_new, float clip_k,
                            float clip_v, const void *q, int32_t B, int32_t Hq,
                            const int32_t *block_table, int32_t max_pages_per_seq,
                            const int32_t *seq_lens, const float *R_k, const float *R_v,
                            float sm_scale, int32_t num_splits, void *workspace,
                            size_t workspace_bytes, void *out, oscar_dtype out_dtype,
                            void *stream);

/*
 * bf16 paged-decode baseline (same paging, uncompressed cache), for comparing
 * against the INT2 path on the same GPU.  A bf16 page-head block (page p,
 * kv-head h) starts at element (p*Hkv + h) * 2*P*d and holds K then V in the
 * order of the decode's matrix-core operands (P = 64, d = 128; each of K and V
 * is 16 tiles of 64 lanes x 8 elements, one contiguous 1 KB load per tile):
 *   K(t, c) at ((u*4 + kc)*64 + lo + 16*hi)*8 + e,
 *           t = 4*lo + u, c = 32*hi + 8*kc + e;
 *   V(t, c) at P*d + ((ct*2 + kt)*64 + lo + 16*hi)*8 + e,
 *           t = 16*hi + 8*kt + e, c = 16*ct + lo.
 * Token slots never written are read as 0 weight (their V is masked).
 */
size_t oscar_bf16_page_bytes(const oscar_layout *L);
int oscar_bf16_kv_append(const oscar_layout *L, void *pages, const void *k_new,
                         const void *v_new, const int64_t *slot_mapping, int32_t n_tok,
                         void *stream);
size_t oscar_bf16_decode_workspace_bytes(const oscar_layout *L, int32_t B, int32_t Hq,
                                         int32_t num_splits);
int oscar_bf16_decode_attn(const oscar_layout *L, const void *pages, const void *q, int32_t B,
                           int32_t Hq, const int32_t *block_table, int32_t max_pages_per_seq,
                           const int32_t *seq_lens, float sm_scale, int32_t num_splits,
                           void *workspace, size_t workspace_bytes, void *out,
                           oscar_dtype out_dtype, void *stream);

/*
 * Offline calibration (Sec. 3 "Algorithm Design: Offline Calibration and
 * Justification"; App. "Hadamard transform", "P_K" and the worked example;
 * Alg. 1 Calibrate).  From one layer's calibration activations (bf16
 * q [T, Hq, d], k and v [T, Hkv, d], row-major, d = 128, Hq % Hkv == 0,
 * g = Hq / Hkv) the rotations and clip ratios the cache update takes.
 * All matrices are row-major [d][d]; fp64 unless stated.  Device pointers,
 * 16-byte aligned; asynchronous on `stream`; nothing is allocated.
 */
#define OSCAR_CALIB_MAX_CANDS 32  /* candidate clip ratios per call */
#define OSCAR_CALIB_MAX_SWEEPS 32 /* Jacobi sweeps before giving up   */

/*
 * oscar_calib_query_cov -- query-aware key target covariance, GQA-averaged as
 * in the appendix worked example:
 *   C = (1/Hkv) sum_h (1/(T g)) sum_{i in group h} sum_t q_{t,i}^T q_{t,i}
 * Products of the bf16 inputs are exact; they are summed in fp32 over chunks of
 * rows and the chunks in fp64.  workspace >= oscar_calib_workspace_bytes(T, Hq,
 * Hkv).  C: fp64 [d][d], exactly symmetric.
 */
size_t oscar_calib_workspace_bytes(int64_t T, int32_t Hq, int32_t Hkv);
int oscar_calib_query_cov(const void *q, int64_t T, int32_t Hq, int32_t Hkv, double *C,
                          void *workspace, size_t workspace_bytes, void *stream);

/*
 * oscar_calib_attn -- the calibration pass's attention rows (Alg. 1 Calibrate):
 *   out[t][i] = softmax_row(q_{t,i} K_h^T / sqrt(d) + M) V_h,  h = i / g,
 * M = -inf on keys j > t when causal != 0 (0 otherwise).  fp32 out [T, Hq, d].
 * Scores are exact products summed in fp32; softmax in fp32 with the running row
 * maximum; the probabilities enter the value product with ~16 significant bits.
 */
int oscar_calib_attn(const void *q, const void *k, const void *v, int64_t T, int32_t Hq,
                     int32_t Hkv, int32_t causal, float *out, void *stream);

/*
 * oscar_calib_score_cov -- score-aware value target covariance (Sec. 3):
 *   C = (1/N) V^T S^T S V, i.e. the GQA-averaged second moment of the rows
 *   o_{t,i} of oscar_calib_attn (averaged like oscar_calib_query_cov).
 * The rows are kept in the workspace (>= oscar_calib_workspace_bytes(T, Hq, Hkv)).
 */
int oscar_calib_score_cov(const void *q, const void *k, const void *v, int64_t T, int32_t Hq,
                          int32_t Hkv, int32_t causal, double *C, void *workspace,
                          size_t workspace_bytes, void *stream);

/*
 * oscar_calib_rotation -- for each of n_mats symmetric matrices C (fp64
 * [n_mats][d][d]): the eigen-decomposition C = U diag(lam) U^T with lam
 * descending (ties: lower index first) and each eigenvector's largest-magnitude
 * entry (the first such) positive, then the composed rotation
 * (Eq. method_composed_rot)
 *   R = U H_Had P_br,   H_Had the normalized Sylvester Walsh-Hadamard matrix,
 *                       P_br[k][bitrev(k)] = 1 (App. "P_K")
 * evaluated as R[i][j] = sum_c U[i][c] H[c][bitrev(j)] in fp64, ascending c.
 * Eigen-decomposition by cyclic Jacobi in fp64.
 *   lam  : [n_mats][d]             U   : [n_mats][d][d] (eigenvectors in columns)
 *   R64  : [n_mats][d][d] or NULL  R32 : fp32 [n_mats][d][d] or NULL (R64 rounded)
 *   info : int32 [n_mats], sweeps run, or -1 if OSCAR_CALIB_MAX_SWEEPS sweeps did
 *          not converge (lam, U and R are then not reliable)
 *   workspace >= oscar_calib_rotation_workspace_bytes(n_mats)
 */
size_t oscar_calib_rotation_workspace_bytes(int32_t n_mats);
int oscar_calib_rotation(const double *C, int32_t n_mats, double *lam, double *U, double *R64,
                         float *R32, int32_t *info, void *workspace, size_t workspace_bytes,
                         void *stream);

/*
 * oscar_calib_clip -- clip calibration (Alg. 1 CalibrateClip; the paper gives no
 * procedure: read as the candidate with the smallest quantization error of the
 * rotated calibration rows).  For rows x [n_tok, Hkv = L->num_kv_heads, d] bf16,
 * rotated by R (fp32, [Hkv][d][d] when L->rot_per_head, NULL: identity) exactly
 * as oscar_kv_append does, and
 * quantized with L's group size, clip mode and metadata format at each
 * candidate ratio cands[n] (fp32, in (0, 1], n_cands <= OSCAR_CALIB_MAX_CANDS):
 *   err[n] = mean over rows and channels of (x~_c - s (code_c - z))^2   (fp64)
 *   best   = cands[first n minimizing err] (fp32 [1], may be NULL)
 * workspace >= oscar_calib_clip_workspace_bytes(n_tok, Hkv, n_cands).
 */
size_t oscar_calib_clip_workspace_bytes(int64_t n_tok, int32_t Hkv, int32_t n_cands);
int oscar_calib_clip(const oscar_layout *L, const void *x, int64_t n_tok, const float *R,
                     const float *cands, int32_t n_cands, double *err, float *best,
                     void *workspace, size_t workspace_bytes, void *stream);

/*
 * oscar_calibrate_layer -- Alg. 1 Calibrate for one layer, in the paper's order:
 * C_Q (oscar_calib_query_cov), C_S (oscar_calib_score_cov), their rotations
 * R_K = U_Q H_Had P_br and R_V = U_S H_Had P_br (oscar_calib_rotation), and the
 * clip ratios c_K, c_V (oscar_calib_clip of k by R_K and of v by R_V, in L's
 * quantizer format).  L->num_kv_heads is Hkv.  With L->rot_per_head = 1 every KV
 * head h gets its own C_Q and C_S (the average over its g query heads only) and
 * its own R_K, R_V; the clip ratios stay one per tensor (all heads' rows).
 *   R_k, R_v : fp32 [d][d], or [Hkv][d][d] per head (what oscar_kv_append and
 *              decode take)
 *   clip     : fp32 [2] = (c_K, c_V)
 *   lam      : fp64 [2][d] (spectra of C_Q, C_S), [2][Hkv][d] per head, or NULL
 *   info     : int32 [2] (oscar_calib_rotation's), [2][Hkv] per head, or NULL
 * workspace >= oscar_calibrate_layer_workspace_bytes(L, T, Hq, n_cands).
 */
size_t oscar_calibrate_layer_workspace_bytes(const oscar_layout *L, int64_t T, int32_t Hq,
                                             int32_t n_cands);
int oscar_calibrate_layer(const oscar_layout *L, const void *q, const void *k, const void *v,
                          int64_t T, int32_t Hq, int32_t causal, const float *cands,
                          int32_t n_cands, float *R_k, float *R_v, float *clip, double *lam,
                          int32_t *info, void *workspace, size_t workspace_bytes,
                          void *stream);

/* ------------------------------------------------------------------------- */
/* Measurement helper (not part of the method)                                */
/* ------------------------------------------------------------------------- */

/*
 * oscar_hbm_read_probe -- a plain streaming read of `bytes` bytes at src (device,
 * 16-byte aligned, bytes a multiple of 16) by `blocks` blocks of 256 threads,
 * each thread reading 16-byte words grid-stride and writing the xor of its words
 * to sink[thread] (device, uint32 [blocks * 256], caller-owned).  The xor of all
 * sink words is the xor of all source words.  Its rate is the reference for the
 * decode kernel's HBM read rate.  Asynchronous on `stream`; invalid arguments
 * return OSCAR_ERR_INVALID_ARG with nothing launched.
 */
int oscar_hbm_read_probe(const void *src, size_t bytes, uint32_t *sink, int32_t blocks,
                         void *stream);

/* Access-pattern flags of oscar_hbm_read_probe_ex. */
enum {
  OSCAR_PROBE_NONTEMPORAL = 1, /* non-temporal loads (lines not kept for reuse)     */
  OSCAR_PROBE_WAVE_CHUNKS = 2  /* each wave reads loads_per_thread KiB contiguous   */
};

/*
 * oscar_hbm_read_probe_ex -- the same read with a chosen access pattern:
 * loads_per_thread (4, 8 or 16) independent 16-byte loads in flight per thread
 * and iteration; flags a combination of OSCAR_PROBE_* (0: grid-stride words,
 * plain loads, as oscar_hbm_read_probe with 4 loads).  With
 * OSCAR_PROBE_WAVE_CHUNKS wave w reads words [w*64*U, (w+1)*64*U) of each
 * iteration's span of 64*U words per wave (lane l, load u: word 64u + l).
 * The sink contract is the one above.  Any other loads_per_thread or flag bit
 * returns OSCAR_ERR_INVALID_ARG with nothing launched.
 */
int oscar_hbm_read_probe_ex(const void *src, size_t bytes, uint32_t *sink, int32_t blocks,
                            int32_t loads_per_thread, int32_t flags, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* OSCAR_H */
