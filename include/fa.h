/*
 * fa.h -- C ABI of the MI355X (gfx950) FlashAttention forward library.
 *
 * Computes exact softmax attention, o = softmax(scale * q k^T) v, per query
 * head (the scaled dot-product definition of Sec. 2), for multi-head,
 * grouped-query and multi-query attention (Sec. 1; Sec. 4.1.1: a key/value
 * row is shared by the query heads of its group), in prefill (many query
 * rows) and decode (one query row against a long key/value cache, Sec. 4.1:
 * "(1 x D)" operands).  The result is reached with the streaming softmax of
 * Alg. 1 carried over key blocks as in Alg. 2 (running row maximum, running
 * row sum, rescaled accumulator, one final 1/l normalisation); decode splits
 * the key range over workgroups and merges the partial results by their
 * log-sum-exp.
 *
 * Tensors (all dense, row-major, D fastest, device memory owned by the
 * caller):
 *   q   [B][Nq][Hq][D]    element type = in_dtype          read only
 *   k   [B][Nk][Hkv][D]   element type = in_dtype          read only
 *   v   [B][Nk][Hkv][D]   element type = in_dtype          read only
 *   o   [B][Nq][Hq][D]    element type = out_dtype         written
 *   lse [B][Hq][Nq]       float32, may be NULL (then not written)
 *                         lse = ln(sum over visible keys of exp(scale*q.k))
 *
 * Head map: query head h reads key/value head h / (Hq / Hkv) (contiguous
 * groups); Hq must be a multiple of Hkv.
 * Causal mask (bottom-right): key j is visible to query row i iff
 * j <= i + (Nk - Nq).  With Nq == Nk this is the usual lower triangle; with
 * Nq == 1 every key is visible.  causal with Nq > Nk is rejected (it would
 * leave rows with no visible key).
 * Precision: fp16 / bf16 inputs use fp32 accumulation and fp32 softmax state;
 * the probabilities enter the second product as fp16 (bf16 values are
 * converted to fp16 there, exact for |v| <= 65504 and within 2^-25 absolute
 * below 2^-14).  fp32 inputs are computed in fp32 throughout.  Outputs are
 * rounded to nearest even.
 *
 * Calls enqueue work on `stream` (a hipStream_t; NULL = the null stream) and
 * return without synchronising.  Argument errors are reported synchronously,
 * before any HIP call; device faults surface at the caller's next
 * synchronisation.  No exception crosses this interface.
 *
 * Decode needs a device workspace for the per-split partial results
 * (fa_workspace_bytes()).  There are three ways to provide it:
 *  - the *_ws entry points take it with each call (caller-owned, checked
 *    before any HIP call, never allocated by the library): calls running
 *    concurrently on different streams each pass their own;
 *  - otherwise the library owns one buffer per (device, stream), allocated on
 *    first use and grown when a call needs more (make one warm-up call before
 *    timing or graph capture: no buffer is allocated while the stream is
 *    being captured, and such a call returns FA_ERR_WORKSPACE).  An outgrown
 *    buffer is kept, not freed, until fa_release_workspace(), so that work
 *    queued earlier and graphs captured earlier stay valid; calls on
 *    different streams never share a buffer (the buffer of a stream is kept
 *    after the stream is destroyed, again until fa_release_workspace());
 *  - fa_set_workspace() installs one caller-owned buffer for a device, which
 *    then serves every call on that device that does not pass its own.
 */
#ifndef FA_H_
#define FA_H_

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
/* In C++ the enumerations below get int as their fixed underlying type, so
 * that any int a C caller passes is a valid value of the type (the library
 * then rejects unknown codes instead of reading an out-of-range enum). */
#define FA_ENUM_BASE : int
#else
#define FA_ENUM_BASE
#endif

typedef enum FA_ENUM_BASE {
    FA_F16 = 0,  /* IEEE binary16 */
    FA_BF16 = 1, /* bfloat16 */
    FA_F32 = 2   /* IEEE binary32 */
} fa_dtype_t;

typedef enum FA_ENUM_BASE {
    FA_OK = 0,
    FA_ERR_NULL = 1,         /* q, k, v or o is NULL */
    FA_ERR_DIM = 2,          /* a size is < 1, or an index would overflow int64 */
    FA_ERR_GQA_RATIO = 3,    /* Hq is not a multiple of Hkv */
    FA_ERR_HEAD_DIM = 4,     /* D unsupported: D % 8 != 0 or D > 256 */
    FA_ERR_CAUSAL_SHAPE = 5, /* causal with Nq > Nk */
    FA_ERR_SCALE = 6,        /* scale is NaN or infinite */
    FA_ERR_ALIGN = 7,        /* a tensor pointer is not 16-byte aligned */
    FA_ERR_ALIAS = 8,        /* o or lse overlaps q, k, v, or each other */
    FA_ERR_DTYPE = 9,        /* unknown dtype, or out_dtype not in {in_dtype, FA_F32} */
    FA_ERR_WORKSPACE = 10,   /* workspace allocation failed or not allowed (stream capture), or a caller-owned one is too small */
    FA_ERR_HIP = 11,         /* a HIP runtime call or kernel launch failed */
    FA_ERR_SPLITS = 12,      /* num_splits outside [0, FA_MAX_SPLITS] */
    FA_ERR_PACKING = 13      /* slots or heads per workgroup not allowed (see fa_fwd_slots) */
} fa_status_t;

#define FA_MAX_SPLITS 256

/* Human-readable name of a status code (static string, never NULL). */
const char *fa_status_string(fa_status_t status);

/* Library version, (major << 16) | (minor << 8) | patch. */
int fa_version(void);

/* Argument checks alone (no HIP call, no device access): returns the status
 * fa_fwd would return for these arguments before touching the GPU.  Pointers
 * are compared and tested for alignment only, never dereferenced. */
fa_status_t fa_validate(const void *q, const void *k, const void *v, const void *o,
                        const float *lse, int B, int Hq, int Hkv, int Nq, int Nk, int D,
                        int causal, float scale, fa_dtype_t in_dtype, fa_dtype_t out_dtype);

/* Attention forward with input and output in the same element type. */
fa_status_t fa_fwd_f16(const void *q, const void *k, const void *v, void *o, float *lse,
                       int B, int Hq, int Hkv, int Nq, int Nk, int D, int causal,
                       float scale, void *stream);
fa_status_t fa_fwd_bf16(const void *q, const void *k, const void *v, void *o, float *lse,
                        int B, int Hq, int Hkv, int Nq, int Nk, int D, int causal,
                        float scale, void *stream);
fa_status_t fa_fwd_f32(const void *q, const void *k, const void *v, void *o, float *lse,
                       int B, int Hq, int Hkv, int Nq, int Nk, int D, int causal,
                       float scale, void *stream);

/* Generic form: out_dtype is in_dtype, or FA_F32 to receive the kernel's fp32
 * result before the final rounding (same kernels, same arithmetic). */
fa_status_t fa_fwd(const void *q, const void *k, const void *v, void *o, float *lse, int B,
                   int Hq, int Hkv, int Nq, int Nk, int D, int causal, float scale,
                   void *stream, fa_dtype_t in_dtype, fa_dtype_t out_dtype);

/* Decode path with an explicit split count (Nq == 1 and fp16 / bf16 with
 * D in {64, 128} only; otherwise behaves like fa_fwd).  num_splits = 0 picks
 * the count fa_fwd would use; 1..FA_MAX_SPLITS forces it (splits left
 * without keys are allowed and contribute nothing to the merge). */
fa_status_t fa_fwd_splitkv(const void *q, const void *k, const void *v, void *o, float *lse,
                           int B, int Hq, int Hkv, int Nq, int Nk, int D, int causal,
                           float scale, void *stream, fa_dtype_t in_dtype,
                           fa_dtype_t out_dtype, int num_splits);

/* Prefill with an explicit query-head packing (the inter-head packing of
 * Sec. 4.1.1 and the GQA K/V reuse of Sec. 4.1.2 (iv)).  With a nonzero
 * heads_per_workgroup a prefill workgroup owns four 32-row query slots that
 * read one key/value head;
 * heads_per_workgroup of them are different query heads of that key/value
 * group (at the same rows), so each K/V tile staged in LDS serves that many
 * heads, and the rest are consecutive row blocks.  1 is the per-head
 * schedule (four consecutive row blocks of one head); 0 does what fa_fwd
 * does (fa_fwd_slots with 0, 0: at D = 64 on a large grid eight slots, and
 * otherwise four, with 4 heads when 4 divides Hq / Hkv, else 2 when 2 does,
 * else 1).  The result
 * is the same, bit for bit, for every packing.  Only the fp16 / bf16 prefill
 * kernels (Nq > 1, D in {64, 128}) take the packing; other calls ignore it.
 * Errors: FA_ERR_PACKING for a value other than 0, 1, 2, 4 or one that does
 * not divide Hq / Hkv; otherwise as fa_fwd.  (fa_fwd_slots also sets the
 * number of slots.) */
fa_status_t fa_fwd_packed(const void *q, const void *k, const void *v, void *o, float *lse,
                          int B, int Hq, int Hkv, int Nq, int Nk, int D, int causal,
                          float scale, void *stream, fa_dtype_t in_dtype,
                          fa_dtype_t out_dtype, int heads_per_workgroup);

/* Prefill with an explicit workgroup layout, for the packing ablation: each
 * prefill workgroup holds slots_per_workgroup query slots of 32 rows that all
 * read one key/value head, so every K/V tile it stages in LDS serves that many
 * slots (the reuse the inter-head packing of Sec. 4.1.1 and Fig. 1 is about:
 * one load of a key/value row serving several query heads), and
 * heads_per_workgroup of them are different query heads of the group (the
 * rest consecutive row blocks).  slots_per_workgroup: 0 (what fa_fwd uses:
 * 8 at D = 64 when that still gives every compute unit two or more
 * workgroups, the K/V is contiguous and heads_per_workgroup is 0; else 4),
 * 1 (no sharing: every slot
 * stages its own tiles), 2, 4 or 8;
 * heads_per_workgroup: 0 (the most heads, up to 4, that divide both the slots
 * and Hq / Hkv), 1, 2, 4 or 8, dividing Hq / Hkv and the slots.  The result
 * is the same, bit for bit, for every layout.  Only the fp16 / bf16 prefill
 * kernels (Nq > 1, D in {64, 128}) take the layout; other calls ignore it.
 * Errors: FA_ERR_PACKING for a value not allowed; otherwise as fa_fwd. */
fa_status_t fa_fwd_slots(const void *q, const void *k, const void *v, void *o, float *lse, int B,
                         int Hq, int Hkv, int Nq, int Nk, int D, int causal, float scale, void *stream,
                         fa_dtype_t in_dtype, fa_dtype_t out_dtype, int slots_per_workgroup,
                         int heads_per_workgroup);

/* Attention against a key/value cache with per-sequence lengths (decode,
 * and chunked prefill of Nq new tokens).  k and v are [B][Nk][Hkv][D]
 * caches of which the first seqlens_k[b] rows of batch element b are valid;
 * seqlens_k is a device array of B int32 values (read by the kernels; values
 * are clamped to [0, Nk]).  The Nq queries of batch element b are the last
 * Nq positions of its sequence: with causal = 1, query i sees keys
 * j <= i + seqlens_k[b] - Nq (the bottom-right alignment of fa_fwd applied to
 * each sequence).  A query row that sees no key (causal with
 * seqlens_k[b] < Nq, or seqlens_k[b] = 0) gets 0 and a log-sum-exp of -inf.
 * With seqlens_k[b] = Nk for every b the result equals fa_fwd's bit for bit.
 * Decode calls (Nq = 1) take the split-KV path with the workspace of
 * fa_workspace_bytes(…, Nk, …).  Errors: FA_ERR_NULL for a NULL seqlens_k,
 * FA_ERR_ALIGN if it is not 4-byte aligned, FA_ERR_ALIAS if o or lse overlaps
 * it; otherwise as fa_fwd (with Nk the cache length). */
fa_status_t fa_fwd_kvcache(const void *q, const void *k, const void *v, void *o, float *lse,
                           const int *seqlens_k, int B, int Hq, int Hkv, int Nq, int Nk, int D,
                           int causal, float scale, void *stream, fa_dtype_t in_dtype,
                           fa_dtype_t out_dtype);

/* Attention against a paged key/value cache (decode, and chunked prefill of
 * Nq new tokens), the cache layout of serving systems: keys and values live
 * in a pool of fixed-size pages,
 *   k_pages, v_pages  [num_pages][page_size][Hkv][D]   element type = in_dtype, read only
 *   block_table       [B][max_pages] int32 (device): page of each block of
 *                     page_size keys of each sequence; key j of batch element
 *                     b is row j % page_size of page block_table[b][j / page_size]
 *   seqlens_k         [B] int32 (device): valid keys of each sequence
 * and otherwise the semantics of fa_fwd_kvcache with Nk = page_size *
 * max_pages (lengths clamped to [0, Nk], the Nq queries are each sequence's
 * last positions, bottom-right causal alignment per sequence, rows that see no
 * key give 0 and -inf).  Only table entries for blocks that hold valid keys
 * are read; an entry outside [0, num_pages) is clamped into that range (a
 * wrong table gives wrong results, never an access outside the pool).  With
 * every sequence's pages laid out in order the result equals fa_fwd_kvcache's
 * on the gathered cache bit for bit.  fp16 / bf16 with D in {64, 128} only.
 * Decode calls (Nq = 1) use the decode workspace of fa_workspace_bytes(B, Hq,
 * Hkv, 1, Nk, D, in_dtype, 0).  Errors: FA_ERR_NULL for a NULL table or
 * length array, FA_ERR_DIM for page_size not a positive multiple of 64,
 * max_pages or num_pages < 1 or page_size * max_pages above 2^31 - 1,
 * FA_ERR_ALIGN for a table or length array not 4-byte aligned, FA_ERR_DTYPE
 * for fp32 data, FA_ERR_HEAD_DIM for another D, FA_ERR_ALIAS when o or lse
 * overlaps the pools, the table or the lengths; otherwise as fa_fwd. */
fa_status_t fa_fwd_kvcache_paged(const void *q, const void *k_pages, const void *v_pages, void *o,
                                 float *lse, const int *seqlens_k, const int *block_table, int B,
                                 int Hq, int Hkv, int Nq, int D, int page_size, int max_pages,
                                 int num_pages, int causal, float scale, void *stream,
                                 fa_dtype_t in_dtype, fa_dtype_t out_dtype);

/* Bytes of decode workspace a call with these sizes needs (0 when the call
 * takes no split-KV path).  num_splits as in fa_fwd_splitkv. */
size_t fa_workspace_bytes(int B, int Hq, int Hkv, int Nq, int Nk, int D, fa_dtype_t in_dtype,
                          int num_splits);

/* Frees every library-owned workspace buffer of the current device (those of
 * all its streams, and outgrown ones), after synchronising the device.  Safe
 * to call when none is held.  Graphs captured with library-owned workspaces
 * of this device must not be replayed afterwards.  Returns FA_ERR_HIP if the
 * device cannot be read, synchronised or a buffer freed. */
fa_status_t fa_release_workspace(void);

/* Caller-owned decode workspace for the current device (the split-KV
 * partial results of the decode path, which otherwise live in a
 * library-owned, grow-only device buffer allocated on first use).
 * dev_ptr: device memory on the current device, 16-byte aligned, at least
 * `bytes` long, owned by the caller and left untouched by the library except
 * as scratch during calls; it must stay allocated until it is replaced or
 * cleared.  After a successful call every decode call on this device uses
 * it and never allocates; a call that needs more than `bytes` (see
 * fa_workspace_bytes) returns FA_ERR_WORKSPACE without launching anything.
 * Every call on the device that does not pass its own workspace shares this
 * one, so such calls must be ordered (one stream, or synchronised streams);
 * concurrent streams should use the *_ws entry points instead.
 * fa_set_workspace(NULL, 0) returns the device to the library-owned
 * per-stream workspaces.  Errors: FA_ERR_NULL for a NULL pointer with
 * bytes > 0 or a non-NULL pointer with bytes == 0, FA_ERR_ALIGN for a
 * misaligned pointer, FA_ERR_HIP when the current device cannot be read. */
fa_status_t fa_set_workspace(void *dev_ptr, size_t bytes);

/* The forward with a caller-owned decode workspace passed with the call (the
 * split-KV partial results of Sec. 4.1's one-row decode, merged by their
 * log-sum-exp): otherwise fa_fwd_splitkv (num_splits as there).  Calls that
 * take no split-KV path (prefill, fp32, other D) ignore the workspace, which
 * may then be NULL.
 *   workspace        device memory on the current device, 16-byte aligned,
 *                    owned by the caller; at least workspace_bytes long
 *   workspace_bytes  its size; the call needs fa_workspace_bytes(B, Hq, Hkv,
 *                    Nq, Nk, D, in_dtype, num_splits)
 * The library never allocates for these calls and uses the workspace only as
 * scratch during the call's kernels; calls running concurrently (e.g. on
 * different streams) must pass disjoint workspaces.  Errors (before any HIP
 * call), on the split-KV path: FA_ERR_NULL for a NULL workspace,
 * FA_ERR_ALIGN for a misaligned one, FA_ERR_WORKSPACE when workspace_bytes is
 * too small, FA_ERR_ALIAS when it overlaps q, k, v, o or lse; otherwise as
 * fa_fwd_splitkv. */
fa_status_t fa_fwd_ws(const void *q, const void *k, const void *v, void *o, float *lse, int B,
                      int Hq, int Hkv, int Nq, int Nk, int D, int causal, float scale, void *stream,
                      fa_dtype_t in_dtype, fa_dtype_t out_dtype, int num_splits, void *workspace,
                      size_t workspace_bytes);

/* For callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): fa_fwd_splitkv whose
 * split-KV partial results go to a fixed device array inside the library
 * (32 MiB, one copy per GPU, held until the process ends) instead of a
 * workspace; it calls no hipMalloc, hipFree or other allocating routine.  The
 * first call on a device reads that array's device address (a HIP query; the
 * runtime places the array in that device's memory then, once), later calls
 * touch no allocator at all.  Every call on one GPU shares its array, so calls that overlap
 * on one GPU (e.g. on two streams) race: order them.  Errors: those of
 * fa_fwd_splitkv, then FA_ERR_WORKSPACE (before any HIP call) when the
 * partial results, fa_workspace_bytes(B, Hq, Hkv, Nq, Nk, D, in_dtype,
 * num_splits), exceed 32 MiB, and FA_ERR_HIP when the array's address cannot
 * be read.  Calls that take no split-KV path behave as fa_fwd_splitkv. */
fa_status_t fa_fwd_splitkv_noalloc(const void *q, const void *k, const void *v, void *o, float *lse,
                                   int B, int Hq, int Hkv, int Nq, int Nk, int D, int causal,
                                   float scale, void *stream, fa_dtype_t in_dtype,
                                   fa_dtype_t out_dtype, int num_splits);

/* fa_fwd_kvcache with a caller-owned decode workspace passed with the call
 * (fa_workspace_bytes(B, Hq, Hkv, Nq, Nk, D, in_dtype, 0) bytes; semantics
 * and errors of the workspace as for fa_fwd_ws). */
fa_status_t fa_fwd_kvcache_ws(const void *q, const void *k, const void *v, void *o, float *lse,
                              const int *seqlens_k, int B, int Hq, int Hkv, int Nq, int Nk, int D,
                              int causal, float scale, void *stream, fa_dtype_t in_dtype,
                              fa_dtype_t out_dtype, void *workspace, size_t workspace_bytes);

/* fa_fwd_kvcache_paged with a caller-owned decode workspace passed with the
 * call (fa_workspace_bytes(B, Hq, Hkv, 1, page_size * max_pages, D,
 * in_dtype, 0) bytes for decode; semantics and errors of the workspace as for
 * fa_fwd_ws). */
fa_status_t fa_fwd_kvcache_paged_ws(const void *q, const void *k_pages, const void *v_pages, void *o,
                                    float *lse, const int *seqlens_k, const int *block_table, int B,
                                    int Hq, int Hkv, int Nq, int D, int page_size, int max_pages,
                                    int num_pages, int causal, float scale, void *stream,
                                    fa_dtype_t in_dtype, fa_dtype_t out_dtype, void *workspace,
                                    size_t workspace_bytes);

/* Unfused self-attention: the same result as fa_fwd, computed the way the
 * paper's optimised self-attention does it (Sec. 4.2), with the score matrix
 * materialised -- the comparison point of its fused kernel (Sec. 6.2).  Three
 * kernels run in order on `stream`, each leaving its result in the workspace:
 * S = scale * Q K^T (fp32), P = the row-wise softmax of S (fp16, normalised;
 * lse from the fp32 maximum and sum), O = P V (fp32 accumulation, one
 * rounding to out_dtype).  GQA/MQA heads share K and V as in fa_fwd; causal
 * is bottom-right aligned; score tiles past the causal edge are not computed.
 *   workspace  device, 256-byte aligned, at least
 *              fa_unfused_workspace_bytes(B, Hq, Nq, Nk) bytes, owned by the
 *              caller; scratch only (its contents after the call are the
 *              scores [B][Hq][Nq][NkP] fp32 followed by the weights
 *              [B][Hq][Nq][NkP] fp16, NkP = Nk rounded up to 64, defined on
 *              each row's visible keys).  Calls sharing one workspace must be
 *              ordered.
 * fp16 / bf16 inputs with D in {64, 128}, Nk <= 2^23 and B * Hq * Nq < 2^31
 * only.  Errors: those of fa_fwd, then FA_ERR_DTYPE for fp32 inputs,
 * FA_ERR_HEAD_DIM for another D, FA_ERR_DIM for Nk > 2^23 or B * Hq * Nq >=
 * 2^31, FA_ERR_NULL for a NULL workspace, FA_ERR_ALIGN
 * for a misaligned one, FA_ERR_DIM when the workspace size overflows, FA_ERR_WORKSPACE when workspace_bytes is too
 * small, FA_ERR_ALIAS when it overlaps a tensor; all before any HIP call. */
fa_status_t fa_fwd_unfused(const void *q, const void *k, const void *v, void *o, float *lse,
                           int B, int Hq, int Hkv, int Nq, int Nk, int D, int causal,
                           float scale, void *stream, fa_dtype_t in_dtype,
                           fa_dtype_t out_dtype, void *workspace, size_t workspace_bytes);

/* Bytes of workspace fa_fwd_unfused needs: 6 * B * Hq * Nq * NkP (0 when a
 * size is < 1 or the product overflows). */
size_t fa_unfused_workspace_bytes(int B, int Hq, int Nq, int Nk);

/* Q8_0 matrix-vector product y = W x, the form the linear projection and
 * feed-forward layers take in decode, where a single token is processed
 * (Sec. 4.3).  W (M x K, row-major) is in the 8-bit block format Q8_0 of
 * Sec. 4.3 and Sec. 7: each row is K / 32 consecutive 34-byte blocks, a block
 * being one IEEE binary16 scale d (bytes 0-1, little-endian) followed by 32
 * signed 8-bit values q_0 .. q_31 (bytes 2-33), weight j of the block being
 * d * q_j (symmetric, no zero point).  The scale comes first as Sec. 7 lays
 * the block out (Sec. 4.3 places it after the values).
 *   w  device, M * (K / 32) * 34 bytes, 4-byte aligned          read only
 *   x  device, K elements of x_dtype (FA_F16, FA_BF16 or FA_F32),
 *      16-byte aligned; used as given (not quantized)            read only
 *   y  device, M elements of y_dtype (x_dtype or FA_F32)        written
 * y[m] = sum over blocks b of d[m][b] * (sum_j q[m][b][j] * x[32 b + j]),
 * accumulated in fp32 (products of the exact int8 values and fp32 x, one
 * rounding per multiply-add), then rounded to nearest even in y_dtype.
 * Non-finite scales give non-finite results whose sign and NaN-ness may
 * differ from the term-by-term sum.  Enqueued on `stream`; allocates nothing.
 * Errors (before any HIP call): FA_ERR_NULL for a NULL pointer, FA_ERR_DIM
 * for M < 1, K < 32, K > 2^30 or K not a multiple of 32, FA_ERR_DTYPE for another dtype
 * pair, FA_ERR_ALIGN for a misaligned pointer, FA_ERR_ALIAS when y overlaps w
 * or x, FA_ERR_HIP when the launch fails. */
fa_status_t fa_q8_0_gemv(const void *w, const void *x, void *y, int M, int K, fa_dtype_t x_dtype,
                         fa_dtype_t y_dtype, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* FA_H_ */
