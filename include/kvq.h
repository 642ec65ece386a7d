/*
 * kvq.h -- C ABI of the MI355X (gfx950) packed low-bit KV-cache decode path.
 *
 * Hot path of "Quality Recovery for Quantized KV Caches via Low-Rank
 * Attention Adaptation" (Abdellatif): the adapted Q/K/V projection
 * (Sec. 3, Eq. (1)-(2)), quantize-and-pack append into a physically packed
 * incremental cache (Sec. 3.1, Eq. (3)), and decode attention over the
 * reconstruction (Sec. 3.1-3.2), each a hand-written HIP kernel.
 *
 * Conventions for every call:
 *   - Tensor arguments are DEVICE pointers owned by the caller; the library
 *     never allocates or frees device memory.  A cache handle is host memory.
 *   - Work is enqueued on the caller's HIP stream (passed as void*, NULL =
 *     the default stream) and runs asynchronously; the call returns once
 *     enqueued.  Calls on one handle must be ordered by the caller (one
 *     stream, or explicit events); a handle is not thread-safe.
 *   - Every argument is checked on the host before anything is enqueued; a
 *     call that returns an error has changed no state and launched nothing.
 *     KVQ_ERR_DEVICE reports a HIP launch error (state is then undefined).
 *   - Device pointers must be 16-byte aligned.  bf16 and fp16 tensors are
 *     16-bit IEEE-style storage (bfloat16 / binary16).
 *   - Non-finite inputs are outside the contract (results are undefined).
 */
#ifndef KVQ_H
#define KVQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    KVQ_OK = 0,
    KVQ_ERR_ARG = 1,       /* null/misaligned pointer, bad size or shape, empty cache */
    KVQ_ERR_FORMAT = 2,    /* unsupported format, or format differs from the cache's */
    KVQ_ERR_CAPACITY = 3,  /* append would exceed T_max tokens */
    KVQ_ERR_WORKSPACE = 4, /* workspace smaller than the *_workspace_bytes query */
    KVQ_ERR_DEVICE = 5,    /* HIP runtime/launch error */
    KVQ_ERR_SCRATCH = 6    /* kvq_decode_attn_noalloc: partials cannot fit KVQ_SCRATCH_BYTES (reserved) */
} kvq_status;

enum { KVQ_AFFINE = 0, KVQ_SYMMETRIC = 1 };
enum { KVQ_PER_TOKEN = 0, KVQ_PER_CHANNEL = 1 };

/* Cache format (Sec. 3.1).
 *   *_bits   2, 4 or 8: code width (8 only as k_bits = v_bits = 8, the
 *            8-bit ablation of Sec. 4 and Sec. 5.4).
 *   *_mode   KVQ_AFFINE: Eq. (3), s = max((max-min)/(2^b-1), 1e-8),
 *            c = clip(round_half_even((x-min)/s), 0, 2^b-1), offset = min.
 *            KVQ_SYMMETRIC (the symmetric control, "max-magnitude scale, no
 *            offset"; formula is this library's reading): s = max(max|x| /
 *            (2^(b-1)-1), 1e-8), q = clip(round(x/s), -(2^(b-1)-1), ...),
 *            stored code q + 2^(b-1).
 *   *_axis   KVQ_PER_TOKEN: groups of *_group consecutive head_dim elements
 *            of one token.  KVQ_PER_CHANNEL (keys only, KIVI): groups of 32
 *            consecutive tokens of one channel (k_group must be 32).
 *   *_group  32..head_dim, power of two (per token); 32 (per channel).
 *   residual, flush   fp16 window (KIVI, Sec. 3.1): with flush F > 0, the
 *            newest tokens stay fp16 and tokens are coded F at a time; the
 *            number coded at length n is floor(max(0, n - residual)/F) * F.
 *            F must be a multiple of 32; both 0 = no window.
 *   rotate   0, or head_dim: apply the fixed normalized Hadamard transform
 *            (KVarN, Sec. 3.1) to K and V before coding, to queries before
 *            attention and to outputs after it.
 *   meta_fp16  0: scales and offsets stored as fp32.  1: stored as fp16, as
 *            the paper stores them (Sec. 3.1): the fp32 scale and offset
 *            are rounded to nearest fp16 (scale clamped to [2^-24, 65504],
 *            offset to +-65504) and the codes are computed from the rounded
 *            values (this rounding rule is this library's reading).
 *   sink     0, or S, a multiple of 32: KVarN's protected first tokens
 *            (Sec. 3.1).  Tokens t < S are kept as fp16 rows (rotated first
 *            when the format rotates) and never coded; tokens from S on
 *            form the coded tail, tail token i = t - S, and every rule
 *            above (groups, the window, the ring slot, the coded count
 *            over n - S tail tokens) applies to tail indices.  The storage
 *            rule is this library's reading of the paper. */
typedef struct {
    int32_t k_bits, v_bits;
    int32_t k_mode, v_mode;
    int32_t k_axis, v_axis;
    int32_t k_group, v_group;
    int32_t residual, flush;
    int32_t rotate;
    int32_t meta_fp16;
    int32_t sink;
} kvq_format;

/* Opaque host handle: format, dimensions, storage pointer, token count. */
typedef struct kvq_cache kvq_cache;

/* Bytes of cache storage for B sequences, H_kv heads of size D (64, 128 or
 * 256) and up to T_max tokens.  The storage image has ten sections, each
 * starting at a multiple of 256 bytes (T_alloc = max(T_max - sink, 0)
 * rounded up to 32, the tail capacity; "token" in sections 0-7 is a tail
 * token):
 *   0 Kc key codes           D*k_bits/8 bytes per token
 *   1 Ks key scales          per token: D/k_group per token; per channel: D per 32 tokens
 *                            (fp32, or fp16 when meta_fp16; element i at byte 4i or 2i)
 *   2 Kz key offsets, like Ks; affine keys only (else 0 bytes)
 *   3 Vc value codes         D*v_bits/8 bytes per token
 *   4 Vs value scales        D/v_group per token (fp32 or fp16, like Ks)
 *   5 Vz value offsets, like Vs; affine values only
 *   6 Kr f16 [B][H_kv][residual+flush][D]  fp16 window, slot t mod (R+F)
 *   7 Vr f16, like Kr
 *   8 Kq f16 [B][H_kv][sink][D]  fp16 sink tokens, row t (sink > 0 only)
 *   9 Vq f16, like Kq
 * Sections 0-5 are blocked by 32-token blocks: with u = b*H_kv + h,
 * NB = T_alloc/32, token t at position tau = t%32 of block beta = t/32, and
 * i = u*NB + beta:
 *   Codes come in pieces of eight codes (code j at bits [bits*j, +bits); a
 *   piece is 64 bits for 8-bit codes, 32 for 4-bit, 16 for 2-bit; piece index
 *   x starts at byte x*bits of its section).  Token tau has row
 *   r = 4*(tau/8) + tau%4 and half e = (tau/4)%2 of its block.
 *   Kc piece (t, P), channels 8P..8P+7 of token t, is at index
 *       ((i*2 + e)*64 + r + 16*(P%4)) * (D/32) + P/4
 *   Vc piece (octet o = tau/8, channel d), tokens 8o..8o+7 of channel d,
 *       is at index (i*64 + d%16 + 16*o) * (D/16) + d/16
 *   Ks/Kz per token, group g: element index (i*(D/k_group) + g)*32 + tau;
 *       per channel (32-token group beta, channel d): i*D + d
 *   Vs/Vz group g: element index (i*(D/v_group) + g)*32 + tau
 * This is the order in which the decode kernel consumes the codes (a
 * 64-lane MFMA operand layout), so attention reads them without any
 * rearrangement; the paper fixes the codes and metadata, not this order. */
kvq_status kvq_cache_bytes(const kvq_format* fmt, int B, int H_kv, int D, int T_max, size_t* bytes);

/* Create a handle over caller storage (at least kvq_cache_bytes bytes,
 * 256-byte aligned).  Host-only: enqueues nothing.  The cache starts empty
 * (n = 0).  No result depends on what the storage holds at init: appends
 * write every byte of a token's codes and metadata (clearing the code bits
 * of later tokens in pieces they share), and attention masks every slot at
 * or past the cached length, whatever it contains.  Only the bytes of dead
 * slots do: storage zero-filled before init gives an image that is a
 * function of the appended tokens alone (what byte-for-byte comparisons
 * with a reference need). */
kvq_status kvq_cache_init(const kvq_format* fmt, int B, int H_kv, int D, int T_max, void* storage,
                          size_t bytes, kvq_cache** out);

/* Byte offset and length of storage section 0..9 (see kvq_cache_bytes). */
kvq_status kvq_cache_section(const kvq_cache* cache, int index, size_t* offset, size_t* length);

/* n = 0: start a new window (the paper resets the cache per evaluation
 * window, Sec. 4).  Storage is not cleared; slots at or past n are dead. */
kvq_status kvq_cache_reset(kvq_cache* cache);

/* Tokens cached (n) and tokens held as codes (n_coded <= n - min(n, sink)). */
kvq_status kvq_cache_len(const kvq_cache* cache, int* n, int* n_coded);

/* Shrink n to n_new <= n without touching storage.  Valid only for formats
 * without an fp16 window (flush == 0), where the first n_new tokens' bytes
 * are unchanged by later appends; otherwise KVQ_ERR_FORMAT. */
kvq_status kvq_cache_rewind(kvq_cache* cache, int n_new);

/* Set the length to n (0 <= n <= T_max) after the caller has made the
 * storage hold the image this cache had at length n, for example by copying
 * back a snapshot of the storage taken then (the fp16 window of formats that
 * have one is only consistent with such a snapshot).  The bytes are not
 * checked.  Host-only. */
kvq_status kvq_cache_restore(kvq_cache* cache, int n);

/* Free the host handle (not the storage). */
void kvq_cache_destroy(kvq_cache* cache);

/* Workspace bytes kvq_project_qkv and kvq_project_append need for M rows and
 * adapter rank r: the fp32 adapter activations A h, M x 3r, times 16 for
 * M <= 32 (partial sums over up to 16 slices of d_in).  0 when r is 0. */
kvq_status kvq_project_workspace_bytes(int M, int rank, size_t* bytes);

/* Adapted Q/K/V projection, Eq. (1)-(2) with the explicit adapter branch of
 * Sec. 3.4: for each row h of H and projection p in {Q, K, V},
 *     y_p = W_p h + lora_scale * B_p (A_p h),   lora_scale = alpha / r.
 *   H  bf16 [M][d_in]             (M = tokens; d_in a multiple of 64)
 *   W  bf16 [d_q + 2 d_kv][d_in]  rows of W_Q, then W_K, then W_V
 *   A  bf16 [3 rank][d_in]        A_Q, A_K, A_V (ignored when rank == 0)
 *   Bm bf16 [d_q + 2 d_kv][rank]  B_Q, B_K, B_V rows aligned with W's rows
 *   Q  bf16 [M][d_q], K and V bf16 [M][d_kv]: outputs, fp32 accumulation,
 *      rounded once to bf16 (round to nearest even).
 * rank 0 disables the adapter.  rank <= 64.  d_q, d_kv multiples of 16. */
kvq_status kvq_project_qkv(const void* H, int M, int d_in, const void* W, int d_q, int d_kv,
                           const void* A, const void* Bm, int rank, float lora_scale, void* Q,
                           void* K, void* V, void* workspace, size_t ws_bytes, void* stream);

/* Projection fused with the append of its K and V (Sec. 3 and 3.1: the new
 * states are projected, then coded, packed and appended): the same Q as
 * kvq_project_qkv, and the cache image kvq_append of its bf16 K and V would
 * write, without the bf16 K and V ever reaching memory.  The rows of H are
 * (sequence, token) pairs, sequence-major: M = B * n_new, n_new new tokens
 * of each of the cache's B sequences.  Arguments as kvq_project_qkv, plus
 * the cache (d_kv = H_kv * D).  Two cases are supported:
 *   - window formats (flush > 0, e.g. KIVI), one decode step: n_new = 1,
 *     M = B <= 32, no rotation or sink.  K and V go straight into the fp16
 *     window; a flush that falls due is coded from the window in the same
 *     call.
 *   - formats without a window, prefill chunks: M >= 256 (the tiled path),
 *     d_q and d_kv multiples of 256, n_new and the cache length multiples
 *     of 32, per-token key groups, no rotation or sink.
 * Otherwise KVQ_ERR_FORMAT (format) or KVQ_ERR_ARG (shapes) and nothing
 * changes.  On success the cache length grows by n_new. */
kvq_status kvq_project_append(const void* H, int M, int d_in, const void* W, int d_q, int d_kv,
                              const void* A, const void* Bm, int rank, float lora_scale, void* Q,
                              kvq_cache* cache, int n_new, void* workspace, size_t ws_bytes,
                              void* stream);

/* Dense-merge deployment of the adapter (Sec. 3.4 "Deployment overhead": the
 * dense-base update can be folded into the weights, leaving the projection
 * shapes unchanged and removing the adapter branch at inference):
 *     W'_p = W_p + lora_scale * B_p A_p   for p in {Q, K, V},
 * accumulated in fp32 and rounded once to bf16 (round to nearest even).
 * kvq_project_qkv with rank 0 on W' then computes the adapted projection.
 *   W     bf16 [d_q + 2 d_kv][d_in]  base weights, rows as in kvq_project_qkv
 *   A     bf16 [3 rank][d_in],  Bm bf16 [d_q + 2 d_kv][rank]
 *   Wout  bf16 [d_q + 2 d_kv][d_in]  result; may be W itself (in place);
 *         must not otherwise overlap W, A or Bm.
 * d_in a multiple of 64; d_q, d_kv multiples of 32; 1 <= rank <= 64.
 * All pointers 16-byte aligned device memory owned by the caller; nothing is
 * allocated.  Invalid arguments return KVQ_ERR_ARG before any launch. */
kvq_status kvq_merge_adapter(const void* W, int d_in, int d_q, int d_kv, const void* A, const void* Bm,
                             int rank, float lora_scale, void* Wout, void* stream);

/* Append n_new tokens per sequence (Sec. 3.1: new states are coded, packed
 * and appended; the cache keeps no unquantized copy beyond the fp16 window).
 *   K, V  bf16 [B][n_new][H_kv][D] (the natural view of the projection's
 *         [B * n_new][d_kv] output).
 *   fmt   must equal the cache's format (KVQ_ERR_FORMAT otherwise).
 * The resulting storage bytes depend only on the tokens appended since the
 * last reset, not on how they were split into calls.  Codes and metadata
 * are bit-exact functions of the input (IEEE fp32, fixed operation order).
 * n + n_new > T_max returns KVQ_ERR_CAPACITY.  n_new == 0 is a no-op. */
kvq_status kvq_append(kvq_cache* cache, const void* K, const void* V, int n_new,
                      const kvq_format* fmt, void* stream);

/* Workspace bytes kvq_decode_attn needs for H_q query heads at any length
 * up to the cache's T_max (split-K partial results; contents need no
 * initialization).  Calls that share a workspace must not overlap. */
kvq_status kvq_decode_workspace_bytes(const kvq_cache* cache, int H_q, size_t* bytes);

/* Decode attention for one new query per sequence over the reconstructed
 * cache (Sec. 3.1-3.2: attention sees the stored reconstruction).
 *   Q  bf16 [B][H_q][D]; query head h reads KV head h / (H_q / H_kv);
 *      H_q a multiple of H_kv with H_q / H_kv <= 16.
 *   O  fp32 [B][H_q][D]: sum_t softmax_t(sm_scale * q . k_t) v_t over all n
 *      cached tokens (coded tokens reconstructed in-kernel, window tokens
 *      from fp16).  With a rotating format q is rotated first and the
 *      output rotated back.
 * Products are formed from binary16 MFMA operands and accumulated in fp32:
 * query elements (after rotation), query x key channel scale x sm_scale x
 * log2(e) for per-channel keys, and each value group's scale must have
 * magnitude below 65504 (binary16's largest finite value).
 * An empty cache (n == 0) returns KVQ_ERR_ARG. */
kvq_status kvq_decode_attn(const kvq_cache* cache, const void* Q, int H_q, float sm_scale, void* O,
                           void* workspace, size_t ws_bytes, void* stream);

/* Bytes of the library's static split-partial scratch: one array per GPU,
 * held from the first kvq_decode_attn_noalloc call on that GPU until the
 * process ends. */
#define KVQ_SCRATCH_BYTES (4u << 20)

/* kvq_decode_attn for callers that cannot allocate device memory (code
 * under HIP graph capture, serving loops that forbid allocation): the same
 * attention, with the split-K partials in the library's static scratch
 * instead of a caller workspace.  Nothing is allocated or freed and no
 * memory is cleared (every split writes its own partials before the merge
 * reads them).  The split plan is kvq_decode_attn's, with the split count
 * capped so that the partials, B * H_q * (D + 2) floats per split, fit in
 * KVQ_SCRATCH_BYTES; when not even two splits fit, one split per (sequence,
 * KV head) computes the outputs directly and the scratch is not used.  A
 * capped plan sums in another order than kvq_decode_attn, within the same
 * bound.  KVQ_ERR_SCRATCH is reserved for a plan that cannot fit (the
 * planner above always finds one).  Every call on one GPU shares that GPU's
 * scratch: calls that overlap on one GPU (different streams, or threads)
 * race and must be ordered by the caller.  Arguments, results and other
 * errors as kvq_decode_attn. */
kvq_status kvq_decode_attn_noalloc(const kvq_cache* cache, const void* Q, int H_q, float sm_scale, void* O,
                                   void* stream);

/* Chunked prefill attention (Sec. 3.1: evaluation runs chunk by chunk; the
 * chunk's states are coded and appended first, then the reconstruction of
 * everything stored feeds attention).  The chunk is the newest C tokens of
 * the cache (1 <= C <= n); query i of the chunk, at position n - C + i,
 * attends causally to the reconstructed tokens 0 .. n - C + i, otherwise
 * exactly as kvq_decode_attn (same head grouping, rotation and softmax).
 *   Q  bf16 [B][C][H_q][D]
 *   O  fp32 [B][C][H_q][D], normalized
 * Reconstructed keys and values (after rotation, for a rotating format)
 * enter the products as binary16 MFMA operands, so their magnitudes must
 * stay below 65504 (binary16's largest finite value).
 * H_q a multiple of H_kv.  Pointers 16-byte aligned device memory owned by
 * the caller; invalid arguments return KVQ_ERR_ARG before any launch.
 *   workspace  device scratch for the reconstructed blocks of each (b, h):
 *              every visible 32-token block is reconstructed once per call
 *              (192 D bytes each) and read back by all the chunk's query
 *              tiles.  kvq_prefill_workspace_bytes gives the size that
 *              serves all B H_kv units in one pass; a smaller workspace
 *              (at least one unit's share, that size / (B H_kv)) makes the
 *              call process the units in groups that fit, with more
 *              launches.  Below one unit's share: KVQ_ERR_WORKSPACE.
 *              Calls that share a workspace must not overlap. */
kvq_status kvq_prefill_attn(const kvq_cache* cache, const void* Q, int C, int H_q, float sm_scale, void* O,
                            void* workspace, size_t ws_bytes, void* stream);
/* Workspace bytes for kvq_prefill_attn on the cache at its current length
 * (all units in one pass). */
kvq_status kvq_prefill_workspace_bytes(const kvq_cache* cache, size_t* bytes);

/* Measurement hook for benchmarks (not part of the method).  While set
 * (both events non-null), every kernel the library launches from this host
 * thread records stop_event when it completes, and the first of them after
 * this call also records start_event when it begins, both from the
 * kernels' own dispatch timestamps (hipExtLaunchKernel).  After one library
 * call, hipEventElapsedTime(start, stop) is that call's device time, from
 * its first kernel's start to its last kernel's end, without the marker
 * packets that hipEventRecord would add on either side.  The events are
 * hipEvent_t values created by the caller with timing enabled and owned by
 * it; kvq_time_launches(NULL, NULL) clears the request.  The request is
 * per host thread and launches nothing itself.  Returns KVQ_ERR_ARG when
 * exactly one of the two events is null. */
kvq_status kvq_time_launches(void* start_event, void* stop_event);

/* Static description of a status code. */
const char* kvq_strerror(kvq_status status);

#ifdef __cplusplus
}
#endif

#endif /* KVQ_H */
