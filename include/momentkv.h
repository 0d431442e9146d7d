/*
 * momentkv.h - C ABI of libmomentkv.so, the MomentKV hot path on MI355X (gfx950).
 *
 * MomentKV (arXiv 2606.01563) keeps, per KV head, four running sums over the evicted
 * tokens E: the count n_e, the key sum s_k, the value sum s_v and the value-key
 * outer-product sum S = sum_E v_i k_i^T (Sec. 4.1; App. A.1 Eq. app_sufficient).
 * This library implements the two data-parallel halves of the method:
 *
 *   momentkv_compress     one-shot prefill eviction: observation-window scoring
 *                         (Sec. 5.1 prefill protocol), moment-informed selection of the
 *                         retained set (Sec. 4.2 Eq. residual; Algorithm 1 Phase 1 in
 *                         batched form), and the moments of the evicted set.
 *   momentkv_decode_attn  attention over the retained cache fused with the first-order
 *                         correction for the evicted tokens (Algorithm 1 Phase 2;
 *                         Eqs. fhat, jensen, fused; log-domain weight of App. C.2).
 *   momentkv_prepare_summary  the centred, clamped covariance of a summary in the form
 *                         the decode reads fastest; the summary is fixed between
 *                         compressions, so this runs once per compression.
 *   momentkv_decode_evict a decoding step with moment-informed eviction: the new token
 *                         joins the cache, the row with the lowest alpha_j ||r_j|| is
 *                         folded into the summary (Algorithm 1 Phase 1, run at every
 *                         generated token), then the corrected attention of Phase 2.
 *
 * Conventions shared by every entry point
 *   - Tensors are dense, contiguous, row-major, in device memory (HBM) unless stated.
 *     Parameter structs are host memory.  Shapes use B = batch, Hq = query heads,
 *     Hkv = KV heads, G = Hq / Hkv (query head hq reads KV head hq / G), d = head dim.
 *   - K/V/Q tensors and outputs use the element type `dtype` (fp32, or bf16 stored as
 *     uint16 bit patterns, round-to-nearest-even).  Moments are always fp32 (n_e int32).
 *   - The caller owns every buffer, including the workspace sized by the matching
 *     *_workspace_bytes query (the *_workspace_size names are the same functions).
 *     The library never allocates, frees or synchronises; all work is enqueued on
 *     `stream` (a hipStream_t; NULL = the default stream) and is stream-ordered.  There is no global mutable state: calls on different streams
 *     with different buffers may run concurrently.
 *   - Every argument is validated on the host before the first launch.  On any error
 *     nothing is launched and the status says why.  A launch failure reported by HIP
 *     returns MKV_ERR_HIP.
 *   - Results are deterministic: all reductions run in a fixed order (no float
 *     atomics), so identical inputs give bit-identical outputs.
 */
#ifndef MOMENTKV_H
#define MOMENTKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MOMENTKV_ABI_VERSION 7

typedef enum {
  MKV_OK = 0,
  MKV_ERR_NULL = 1,        /* a required pointer is NULL                               */
  MKV_ERR_SHAPE = 2,       /* non-positive size, Hq % Hkv != 0, bad d/window/chunk ... */
  MKV_ERR_BUDGET = 3,      /* budget < n_sink + window; eviction budget < 1            */
  MKV_ERR_DTYPE = 4,       /* dtype is not MKV_F32 or MKV_BF16                          */
  MKV_ERR_WORKSPACE = 5,   /* workspace NULL or smaller than the size query            */
  MKV_ERR_CAPACITY = 6,    /* output cache rows too few, or max_len > cap              */
  MKV_ERR_ALIAS = 7,       /* an output overlaps an input it must not overwrite        */
  MKV_ERR_HIP = 8,         /* a HIP launch failed                                       */
  MKV_ERR_UNSUPPORTED = 9  /* valid request outside this build's limits (see below)    */
} mkv_status;

typedef enum { MKV_F32 = 0, MKV_BF16 = 1 } mkv_dtype;

/* Limits of this build: head_dim in {64, 128}; G = Hq/Hkv <= 16; G * window <= 512;
 * at most 1048576 eviction candidates (ctx_len - window - n_sink) per head (per layer with
 * head-adaptive budgets); a decode grid
 * of at most 2^24 waves (B * Hkv * (token slices + head_dim / 32)). */

/* ------------------------------------------------------------------------------------
 * Prefill compression (Sec. 5.1 protocol; Sec. 4.2; App. A.1)
 *
 * Per (sequence b, KV head h), with N = ctx_len, w = window, n_s = n_sink:
 *   1. Window scoring.  The G*w window queries of the group attend causally to the
 *      prefix (row t of the window sits at position N-w+t and sees keys 0..N-w+t);
 *      a_j is the mean over those rows of the softmax probability on key j, j < N-w.
 *      Logits are scale * q.k (scale = 1/sqrt(d) when the field is 0).
 *   2. Candidates are C = [n_s, N-w); the sinks [0, n_s) and the window [N-w, N) are
 *      always kept.  k_keep = budget - n_s - w candidates survive.
 *   3. Chunk pooling: abar_j = mean of a over the candidates of j's aligned chunk
 *      [c*m, c*m+c) of absolute positions (chunk = 1 disables pooling).
 *   4. Selection (batched Algorithm 1 Phase 1):
 *        provisional round: score0_j = abar_j * ||v_j|| (the empty summary gives
 *        r_j = v_j); keep the k_keep best; E0 = the other candidates;
 *        moment rounds (mi_rounds >= 1): summary = moments of the previous round's
 *        evicted set, k_bar/v_bar = sums / n, S_tilde = S - s_v s_k^T / n with entries
 *        |S_tilde_ab| < tau set to 0 (App. C.2), r_j = v_j - v_bar - scale/n *
 *        S_tilde k_j (Eq. residual), score_j = abar_j * ||r_j||; keep the k_keep best.
 *        "Best" = larger score; equal scores keep the lower position.
 *      mi_rounds = -1 keeps the k_keep largest abar (attention only); 0 stops after the
 *      provisional round; mi_rounds = r >= 1 runs r moment rounds, each with the
 *      moments of the round before.  This build supports mi_rounds in [-1, 8].
 *   5. Outputs: the retained positions idx (ascending: sinks, kept candidates, window)
 *      and their K/V rows copied to k_out/v_out; lens = min(budget, N); the raw sums of
 *      the final evicted set E (n_e = |E|, s_k, s_v, S = sum_E v_i k_i^T), accumulated
 *      in fp32; S is stored in fp32 or, with moment_dtype = MKV_BF16, in bf16.
 *   budget >= N keeps every token: idx = 0..N-1, n_e = 0 and zero moments.
 *   adaptive = 1 (head-adaptive budgets, Sec. 5.1 after Ada-KV): per sequence, the
 *      Hkv * k_keep candidates with the largest abar over all the layer's heads (equal
 *      values in (head, position) order) are counted per head, k_h; head h then selects
 *      k_h candidates as in step 4 and keeps n_s + w + k_h tokens (lens).  Requires
 *      cap >= n_s + w + min(n_c, Hkv * k_keep) and Hkv * n_c <= 1048576; idx_out then has
 *      cap entries per head, of which the first lens are written.
 * ---------------------------------------------------------------------------------- */
typedef struct {
  int32_t batch;        /* B                                                         */
  int32_t n_q_heads;    /* Hq                                                        */
  int32_t n_kv_heads;   /* Hkv, divides Hq                                           */
  int32_t head_dim;     /* d in {64, 128}                                            */
  int32_t ctx_len;      /* N, prefill length                                         */
  int32_t budget;       /* L, retained tokens per KV head (sinks and window included) */
  int32_t window;       /* w, 1 <= w < N                                             */
  int32_t n_sink;       /* n_s >= 0 attention-sink tokens kept at the start          */
  int32_t chunk;        /* c >= 1 pooling chunk                                      */
  int32_t mi_rounds;    /* -1 .. 8 (see step 4)                                      */
  int32_t cap;          /* rows per head of k_out/v_out, >= min(budget, N)           */
  int32_t dtype;        /* mkv_dtype of q_win, k, v, k_out, v_out                    */
  float scale;          /* logit scale; 0 selects 1/sqrt(d)                          */
  float tau;            /* covariance clamp threshold (paper: 1e-6); >= 0            */
  int32_t adaptive;     /* 0 = budget per head; 1 = head-adaptive split (step 5)     */
  int32_t moment_dtype; /* mkv_dtype of the output S: MKV_F32, or MKV_BF16 = the fp32 */
                        /* sum rounded once to bf16 (RNE), the 16-bit moment storage */
                        /* of App. C.2 (s_k, s_v stay fp32: 2d of the d^2 + 2d)      */
} mkv_compress_params;

/* Optional per-candidate diagnostics (any field may be NULL).  n_c = N - w - n_s.
 * Written only when budget < N (otherwise nothing is scored).                         */
typedef struct {
  float* abar;          /* [B, Hkv, n_c] pooled window mass                           */
  float* score0;        /* [B, Hkv, n_c] provisional score abar * ||v||               */
  float* score;         /* [B, Hkv, n_c] last moment round's score (mi_rounds >= 1)   */
  int32_t* kept0;       /* [B, Hkv, k_keep] provisional kept positions, ascending    */
                        /* (adaptive: [B, Hkv, min(n_c, Hkv*k_keep)], first k_h set) */
} mkv_compress_debug;

/* Bytes of device workspace momentkv_compress needs for these parameters (0 on invalid
 * parameters).  Pure host computation.  momentkv_compress_workspace_size is the same
 * function under its earlier name. */
size_t momentkv_compress_workspace_bytes(const mkv_compress_params* p);
size_t momentkv_compress_workspace_size(const mkv_compress_params* p);

/* q_win   [B, Hq, w, d]      window queries (post-RoPE), read only
 * k, v    [B, Hkv, N, d]     prefill keys (post-RoPE) and values, read only
 * k_out, v_out [B, Hkv, cap, d]  retained rows written to rows 0..min(L,N)-1; must not
 *                            overlap k or v (MKV_ERR_ALIAS)
 * idx_out [B, Hkv, min(L,N)] int32 retained positions, ascending ([B, Hkv, cap] when
 *                            adaptive)
 * lens_out [B, Hkv]          int32, set to min(L, N) (n_s + w + k_h when adaptive)
 * n_e [B, Hkv] int32, s_k, s_v [B, Hkv, d] fp32, S [B, Hkv, d, d] fp32: outputs,
 *                            overwritten (zero-initialised summary per generation)
 * dbg                        NULL or optional diagnostics
 * workspace                  >= momentkv_compress_workspace_bytes(p) bytes, 256-aligned */
mkv_status momentkv_compress(const mkv_compress_params* p, const void* q_win, const void* k,
                             const void* v, void* k_out, void* v_out, int32_t* idx_out,
                             int32_t* lens_out, int32_t* n_e, float* s_k, float* s_v, void* S,
                             const mkv_compress_debug* dbg, void* workspace,
                             size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------------------
 * Corrected decode attention (Algorithm 1 Phase 2; Eqs. fhat, jensen, fused; App. C.2)
 *
 * Per (b, query head hq), KV head h = hq / G, one query q:
 *   0. if k_new/v_new are given, append them at row lens[b,h] of the cache and
 *      increment lens[b,h] (the new token joins the retained set; the summary is
 *      unchanged);
 *   1. f_R, log Z_R = softmax attention of q over rows 0..lens-1 (logits scale * q.k);
 *   2. if n_e = 0: out = f_R, w_R = 1;
 *   3. else k_bar = s_k/n_e, v_bar = s_v/n_e, S_tilde = S - s_v s_k^T/n_e clamped at tau,
 *      log Z_E_hat = log n_e + scale * q.k_bar (Jensen lower bound),
 *      f_E_hat = v_bar + scale/n_e * S_tilde q (first-order estimate; order 0 drops the
 *      covariance term), w_R = exp(log Z_R - logsumexp(log Z_R, log Z_E_hat)),
 *      out = w_R f_R + (1 - w_R) f_E_hat.
 * ---------------------------------------------------------------------------------- */
typedef struct {
  int32_t batch;        /* B (any number of independent caches, e.g. layers x seqs)  */
  int32_t n_q_heads;    /* Hq                                                        */
  int32_t n_kv_heads;   /* Hkv                                                       */
  int32_t head_dim;     /* d in {64, 128}                                            */
  int32_t cap;          /* rows per head of the cache                                */
  int32_t max_len;      /* upper bound of lens after the append, 1 <= max_len <= cap */
  int32_t order;        /* 1 = first order (default), 0 = v_bar only, -1 = no        */
                        /* correction (out = f_R, w_R = 1: the uncorrected ablation) */
  int32_t dtype;        /* mkv_dtype of q, caches, k_new, v_new, out                 */
  float scale;          /* logit scale; 0 selects 1/sqrt(d)                          */
  float tau;            /* covariance clamp threshold, >= 0                          */
  int32_t n_split;      /* work split over each KV head's cache: 1 = one workgroup   */
                        /* per KV head; k > 1 = k token slices of one wave each      */
                        /* (rows rounded up to a multiple of 32), merged in the same */
                        /* launch by the last wave of the head to finish; 0 =        */
                        /* automatic (one workgroup per KV head up to max_len 384,   */
                        /* else about 768 slices in the whole grid).  One launch     */
                        /* either way.                                               */
  int32_t summary;      /* form of the S argument: 0 = the raw sum S (fp32); 1 = the */
                        /* prepared form written by momentkv_prepare_summary; 2 =    */
                        /* its half-precision form (bf16 caches only); 3 = the raw   */
                        /* sum stored in bf16 (compress with moment_dtype MKV_BF16), */
                        /* centred and clamped in fp32 as for 0                      */
} mkv_decode_params;

/* Bytes of device workspace momentkv_decode_attn needs for these parameters (0 on invalid
 * parameters; pure host computation); momentkv_decode_workspace_size is the same function. */
size_t momentkv_decode_workspace_bytes(const mkv_decode_params* p);
size_t momentkv_decode_workspace_size(const mkv_decode_params* p);

/* Leading bytes of that workspace that must be zero before a call (0 on invalid
 * parameters): the sticky flag, then one arrival counter per KV head that the split shape
 * uses to find the last slice of a head to finish.  Every call leaves the counters at zero,
 * so a workspace zeroed once serves any number of calls; a workspace reused for a call
 * with a larger value here needs the bytes beyond the previous value zeroed first (they
 * may hold partial results of earlier calls). */
size_t momentkv_decode_workspace_zero_bytes(const mkv_decode_params* p);

/* Decode form of a summary (Eq. fhat's covariance term; clamp of App. C.2).
 *
 * Per (b, h) with n_e > 0: S_tilde = S - s_v s_k^T / n_e in fp32, entries with
 * |S_tilde| < tau set to 0 (the same arithmetic the decode applies to a raw S), stored as
 *   dtype bf16: two bf16 planes [B, Hkv, 2, d, d]: hi = RNE(S_tilde), lo = RNE(S_tilde - hi),
 *               so hi + lo equals S_tilde to within 2^-16 of its magnitude;
 *   dtype bf16, p->summary = 2: the hi plane alone, [B, Hkv, d, d] bf16 (the moments in
 *               half precision as in App. C.2, rounded after the fp32 centring, so the
 *               cancellation of S - s_v s_k^T / n_e happens before the rounding);
 *   dtype fp32: S_tilde itself, fp32 [B, Hkv, d, d].
 * Heads with n_e = 0 get zeros.  Uses batch, n_q_heads, n_kv_heads, head_dim, dtype and
 * tau of p (the other fields are validated as for the decode).  `prepared` holds
 * momentkv_prepared_summary_size(p) bytes (16-byte aligned) and must not overlap the
 * inputs.  Decode calls with p->summary = 1 (2) read it in place of S.  S is the fp32 raw
 * sum; p->summary = 3 (a bf16 raw sum) has no prepared form (MKV_ERR_SHAPE, size 0). */
size_t momentkv_prepared_summary_size(const mkv_decode_params* p);
mkv_status momentkv_prepare_summary(const mkv_decode_params* p, const int32_t* n_e,
                                    const float* s_k, const float* s_v, const float* S,
                                    void* prepared, void* stream);

/* q         [B, Hq, d]
 * k_cache, v_cache [B, Hkv, cap, d]  retained cache; row lens[b,h] is written when
 *           appending (a head whose lens >= cap skips the append and is flagged)
 * lens      [B, Hkv] int32 device, 0 <= lens (+1 when appending) <= max_len; updated.
 *           An empty retained set gives log Z_R = -inf, w_R = 0 and out = f_E_hat
 *           (out = 0 when n_e = 0 as well).
 * k_new, v_new [B, Hkv, d] or both NULL
 * n_e [B, Hkv] int32, s_k, s_v [B, Hkv, d] fp32: the summary, read only
 * S         p->summary = 0: the raw sum, fp32 [B, Hkv, d, d]; p->summary = 1 or 2: the
 *           output of momentkv_prepare_summary for the same summary, tau, dtype and form;
 *           p->summary = 3: the raw sum in bf16 [B, Hkv, d, d]
 * out       [B, Hq, d]
 * lse_out   NULL or [B, Hq] fp32: log Z_R (retained partition function, logits scaled)
 * w_r_out   NULL or [B, Hq] fp32: the mixing weight w_R
 * workspace >= momentkv_decode_workspace_bytes(p) bytes, 256-aligned, whose first
 *           momentkv_decode_workspace_zero_bytes(p) bytes are zero (see there).  Its first
 *           int32 is a sticky overflow flag (set to 1 when an append found a full cache).
 *           Calls that share a workspace must be stream-ordered. */
mkv_status momentkv_decode_attn(const mkv_decode_params* p, const void* q, void* k_cache,
                                void* v_cache, int32_t* lens, const void* k_new,
                                const void* v_new, const int32_t* n_e, const float* s_k,
                                const float* s_v, const void* S, void* out, float* lse_out,
                                float* w_r_out, void* workspace, size_t workspace_bytes,
                                void* stream);

/* ------------------------------------------------------------------------------------
 * Decode without a workspace argument.  For callers that cannot allocate device memory:
 * code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 *
 * Computes exactly what momentkv_decode_attn computes (the same kernels, so the same bits)
 * with the same arguments, except:
 *   - the workspace is a library-owned device array of MOMENTKV_NOALLOC_SCRATCH_BYTES on
 *     each GPU the library runs on, held until the process ends; calls for which
 *     momentkv_decode_workspace_bytes(p) exceeds it return MKV_ERR_WORKSPACE (at 16 MiB:
 *     e.g. 2048 KV heads at G = 4, d = 128 and max_len <= 384);
 *   - flag: NULL, or a device int32 set to 1 when an append finds a full cache (sticky,
 *     the caller zeroes it); with NULL that event is not reported.
 * No hipMalloc, hipFree or allocating library routine is called.  The array's device
 * address is looked up once per device, on the first call with that device current;
 * `stream` must belong to the current device (MKV_ERR_UNSUPPORTED otherwise).  Every call
 * on one GPU uses that GPU's array, which keeps the last call's contents: its arrival
 * counters (a fixed region at its start, zero when the library is loaded) are back at zero
 * when a call completes.  Calls that overlap in time on one GPU (on different streams, or
 * from host threads without ordering between them) race on it and must not be issued;
 * calls on one stream are ordered.
 * ---------------------------------------------------------------------------------- */
#define MOMENTKV_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)

mkv_status momentkv_decode_attn_noalloc(const mkv_decode_params* p, const void* q,
                                        void* k_cache, void* v_cache, int32_t* lens,
                                        const void* k_new, const void* v_new,
                                        const int32_t* n_e, const float* s_k, const float* s_v,
                                        const void* S, void* out, float* lse_out,
                                        float* w_r_out, int32_t* flag, void* stream);

/* ------------------------------------------------------------------------------------
 * Decode step with moment-informed eviction (Algorithm 1, Phase 1 then Phase 2)
 *
 * Per (b, h) and its G queries q_g (query heads hG .. hG + G - 1):
 *   0. the new token joins R at row lens[b,h] (Algorithm 1, before Phase 1);
 *   1. Phase 1, when R now holds more than `budget` rows.  One eviction per call: a cache
 *      that held at most `budget` rows before the append (every step after a
 *      compression to `budget`) is back at `budget` rows, so Algorithm 1's loop runs once;
 *      a cache that already held more keeps its length and is flagged:
 *        alpha_j = mean over g of softmax_j(scale q_g . k_j) over R (the group mean is this
 *                  library's reading for grouped queries),
 *        r_j = v_j - v_bar - (scale / n_e) S_tilde k_j (Sec. 4.2 Eq. residual; v_bar and
 *              S_tilde are zero when n_e = 0), S_tilde clamped at tau as in the decode,
 *        j* = the row with the lowest alpha_j ||r_j|| (the lowest row among equal scores),
 *        n_e += 1, s_k += k_j*, s_v += v_j*, S += v_j* k_j*^T (App. A.1 Eq. app_update),
 *        the last row of R moves into row j*, lens -= 1;
 *   2. Phase 2: the corrected attention of momentkv_decode_attn (no append) on the
 *      updated cache and summary.
 * The decision is taken on fp32 scores in the log domain (log alpha_j + log ||r_j||, so
 * no weight underflows); near-equal scores may order differently from exact arithmetic.
 * ---------------------------------------------------------------------------------- */
size_t momentkv_decode_evict_workspace_bytes(const mkv_decode_params* p);
size_t momentkv_decode_evict_workspace_size(const mkv_decode_params* p);  /* same function */

/* p         as for momentkv_decode_attn with summary = 0: S is the raw sum, updated in
 *           place.  max_len bounds lens after the append (budget < max_len <= cap leaves
 *           room for the new row).  n_split selects the launch shape: 0 = automatic; for
 *           max_len >= 320 (or n_split > 0) one read of the cache, the attention computed
 *           in the scoring pass over about one workgroup per CU (n_split per KV head when
 *           n_split > 0) and the evicted row's term removed from it afterwards, then a
 *           finishing launch; for shorter caches one launch with one workgroup per KV
 *           head that scores, selects, updates and then attends to the new cache.
 *           Results agree within the dtype's tolerance either way
 * budget    rows per KV head kept by Phase 1, >= 1 (MKV_ERR_BUDGET otherwise)
 * q, k_cache, v_cache, lens, out, lse_out, w_r_out: as momentkv_decode_attn; row lens (the
 *           new token) and row j* of the caches are written, lens is updated
 * k_new, v_new [B, Hkv, d]: required
 * n_e, s_k, s_v, S: the raw summary (fp32; n_e int32), read and updated in place
 * evicted_out  NULL or [B, Hkv] int32: the row j* evicted by this call (it now holds what
 *           was the last row, unless j* was the last row itself), -1 if none
 * workspace >= momentkv_decode_evict_workspace_bytes(p) bytes, 256-aligned.  Its first
 *           int32 is a sticky flag: bit 0 = a full cache (lens >= cap) skipped the append
 *           and the eviction; bit 1 = lens + 1 exceeded max_len (appended, no eviction);
 *           bit 2 = no finite score (nothing evicted); bit 3 = lens was above budget
 *           before the append (one row evicted, the length kept).  Zero it before first
 *           use. */
mkv_status momentkv_decode_evict(const mkv_decode_params* p, int32_t budget, const void* q,
                                 void* k_cache, void* v_cache, int32_t* lens,
                                 const void* k_new, const void* v_new, int32_t* n_e,
                                 float* s_k, float* s_v, float* S, void* out, float* lse_out,
                                 float* w_r_out, int32_t* evicted_out, void* workspace,
                                 size_t workspace_bytes, void* stream);

/* Static description of a status code. */
const char* momentkv_status_string(int32_t status);

/* MOMENTKV_ABI_VERSION of the loaded library. */
int32_t momentkv_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* MOMENTKV_H */
