/*
 * dfa.h -- C ABI of the DiTFastAttn attention hot path on AMD MI355X (gfx950).
 *
 * DiTFastAttn (arXiv 2406.08552) compresses the self-attention of a diffusion
 * transformer with three techniques that this library executes on the GPU:
 *
 *   WA-RS  Window Attention with Residual Sharing (Sec. 3.2, Eq. 1-2).  At the
 *          first step r of a residual-sharing set the layer computes full
 *          attention O_r and window attention W_r and keeps R_r = O_r - W_r;
 *          at every later step k of the set it computes only W_k and emits
 *          O_k = W_k + R_r.
 *   AST    Attention Sharing across Timesteps (Sec. 3.3): a step reuses the
 *          cached attention output of an earlier step of the same layer.
 *   ASC    Attention Sharing across CFG (Sec. 3.4): the attention output of
 *          the conditional evaluation is reused for the unconditional one.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *   Tensors  Q, K, V, O and Ocache are DEVICE pointers to bf16 values
 *            (16-bit storage, round-to-nearest-even on output); the residual
 *            R is a DEVICE pointer to fp32 values.  All are contiguous
 *            [B][H][L][d] with d fastest, and each pointer must be 16-byte
 *            aligned.  The softmax scale is fixed at 1/sqrt(d).  R is kept in
 *            fp32 because it is reused unchanged by every later step of its
 *            set: with a narrow band R is as large as V itself, and bf16
 *            storage alone would put about 1e-3 mean error into every reuse.
 *   Window   Window attention attends, for query token i, to the keys j with
 *            |i - j| <= w over the flattened token index (a band along the
 *            diagonal of the attention matrix, Sec. 3.2), truncated at 0 and
 *            L-1.  w is the HALF-width; w >= L-1 covers every key.
 *   Numerics Scores and softmax statistics are fp32; the probabilities enter
 *            the PV product as bf16 and every accumulation is fp32.  Rows of
 *            at most 32 keys (windows with w <= 15, in window attention and in
 *            the window pass of a refresh, and every sequence of at most 32
 *            tokens) add the bf16 rounding residual of each probability as a
 *            second PV operand: with so few keys the rounding of the weights
 *            does not average out.
 *   CFG      A classifier-free-guidance batch holds B = 2P entries: entries
 *            0..P-1 are the conditional evaluations and entry b + P is the
 *            unconditional partner of entry b (Sec. 3.4).
 *   Sizes    B, H, L >= 1; w >= 0; d in {64, 72} (others return
 *            DFA_ERR_UNSUPPORTED).  L is arbitrary: ragged tiles are masked.
 *            Limits (DFA_ERR_INVALID_ARG beyond them): L <= 2^30, B*H <= 2^24,
 *            B*H*L*d <= 2^40 elements, and B*L <= 2^30 tokens for the
 *            projection and module entry points.
 *   Streams  Every call is asynchronous on `stream` (0 = the null stream).
 *            Outputs are valid once the caller has synchronised the stream.
 *            The attention, plan-step, projection and module calls only
 *            launch kernels (no copy, memset or synchronisation), so they may
 *            be captured into a HIP graph on `stream` and replayed.
 *   Memory   The caller allocates and owns every buffer and the stream.  The
 *            library never allocates or frees (dfa_mrae_noalloc's array is a
 *            static part of the library's device code) and keeps no pointer after
 *            returning; only dfa_plan_search synchronises (its stream, to read
 *            each trial's loss).  The state kept between calls is the
 *            thread-local message of dfa_last_error() and, for
 *            dfa_mrae_noalloc only, its fixed per-device scratch array (and
 *            that array's address).  Calls are re-entrant,
 *            and calls on different streams may run concurrently as long as
 *            their output buffers do not overlap.
 *   Errors   Every function returns a dfa_status; nothing else crosses the
 *            ABI.  Arguments are validated before any HIP call is made, so a
 *            bad argument is reported without touching a device.  After a
 *            non-OK status dfa_last_error() describes it.
 */
#ifndef DFA_H
#define DFA_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DFA_OK = 0,
    DFA_ERR_INVALID_ARG = 1,  /* NULL/misaligned pointer, bad size, bad code, aliasing */
    DFA_ERR_UNSUPPORTED = 2,  /* valid but not built (head dim outside the supported set) */
    DFA_ERR_HIP = 3           /* a HIP launch or query failed; see dfa_last_error() */
} dfa_status;

/* Plan codes: the strategy one layer runs at one denoising step (the entries
 * of the per-(step, layer) plan dictionary produced by the plan search of
 * Sec. 3.5, Alg. 1). */
enum {
    DFA_FULL = 0,          /* full attention                                  */
    DFA_WARS_REFRESH = 1,  /* WA-RS, first step of a set: O = Attn, R = O - W  (Eq. 1) */
    DFA_WARS_REUSE = 2,    /* WA-RS, later step:          O = W + R            (Eq. 2) */
    DFA_AST_REUSE = 3,     /* AST: O = the layer's cached output (Sec. 3.3)    */
    DFA_ASC_REUSE = 4,     /* ASC: conditional half computed, copied to the unconditional half (Sec. 3.4) */
    DFA_WARS_ASC_REFRESH = 5,  /* WA-RS + ASC: REFRESH on the conditional half, output copied */
    DFA_WARS_ASC_REUSE = 6     /* WA-RS + ASC: REUSE on the conditional half, output copied   */
};

/* Full self-attention (Sec. 3.2, first line of Eq. 1):
 *   O[b,h,i,:] = sum_j softmax_j(Q[b,h,i,:] . K[b,h,j,:] / sqrt(d)) V[b,h,j,:]
 * In:  Q, K, V.  Out: O (must not overlap Q, K or V).
 * R and w are accepted for signature symmetry with the other calls and are
 * ignored (R may be NULL; w must still be >= 0). */
dfa_status dfa_attn_full(const void* Q, const void* K, const void* V, void* O, void* R,
                         int B, int H, int L, int d, int w, hipStream_t stream);

/* WA-RS refresh (Sec. 3.2, Eq. 1) in one pass over K and V:
 *   O := Attention(Q, K, V)                       (full attention, O_r)
 *   R := O_full - WindowAttention(Q, K, V; w)     (the residual R_r)
 * Both outputs are computed from the same scores; R (fp32) is the difference
 * of the two fp32 results.  O and R must not overlap each other or Q, K, V.
 * w >= L-1 gives R == 0 exactly. */
dfa_status dfa_attn_full_and_residual(const void* Q, const void* K, const void* V, void* O, void* R,
                                      int B, int H, int L, int d, int w, hipStream_t stream);

/* WA-RS reuse (Sec. 3.2, Eq. 2):
 *   O := WindowAttention(Q, K, V; w) + R
 * Only key tiles that intersect the band are visited.  R is the residual of
 * the layer's latest refresh; R == NULL gives plain window attention.  O must
 * not overlap Q, K, V or R. */
dfa_status dfa_attn_window_plus_residual(const void* Q, const void* K, const void* V, void* O,
                                         const void* R, int B, int H, int L, int d, int w,
                                         hipStream_t stream);

/* One plan entry of one layer at one step: dispatches `code` and maintains the
 * caller's per-layer caches.
 *   R       the layer's fp32 residual buffer [B,H,L,d]: written by the two
 *           REFRESH codes, read by the two REUSE codes (required for all four;
 *           ignored otherwise).  The WA-RS + ASC codes touch only its first
 *           B/2 entries (the conditional half).
 *   Ocache  the layer's output cache [B,H,L,d] for AST (Sec. 3.3).  Every
 *           computed step (all codes except AST) also writes its output here,
 *           and DFA_AST_REUSE copies it to O.  Ocache == O makes AST a no-op
 *           and computed steps write once.  Ocache == NULL is allowed for
 *           every code except DFA_AST_REUSE.
 *   code    FULL      O = Attention
 *           REFRESH   O = Attention, R = O - W
 *           REUSE     O = W + R
 *           AST       O = Ocache
 *           ASC       O[b] = O[b+B/2] = Attention on the conditional entry b
 *                     (b < B/2; B must be even)
 *           WARS_ASC_REFRESH   (WA-RS and ASC together, the strategy list of
 *                     Sec. 3.5 and Table 2)  for b < B/2:
 *                     O[b] = O[b+B/2] = Attention, R[b] = O[b] - W[b];
 *                     R[b+B/2] is left untouched
 *           WARS_ASC_REUSE     for b < B/2: O[b] = O[b+B/2] = W[b] + R[b]
 * A WARS_ASC_REUSE may follow either refresh code (it reads only R's
 * conditional half).  A whole-batch WARS_REUSE must follow a whole-batch
 * WARS_REFRESH: after a WARS_ASC_REFRESH the unconditional half of R is stale,
 * and the library, which keeps no state, cannot detect that misuse.
 * The ASC copy and the cache write are fused into the attention kernel's
 * store (each output tile is written to every destination), not separate
 * passes.  Returns DFA_ERR_INVALID_ARG for an unknown code, odd B with a
 * half-batch code (ASC, WARS_ASC_*), a missing R or Ocache, or overlapping
 * outputs. */
dfa_status dfa_plan_step(int code, const void* Q, const void* K, const void* V, void* O, void* R,
                         void* Ocache, int B, int H, int L, int d, int w, hipStream_t stream);

/* The attention module around the path (Sec. 3.1; the module whose FLOPs
 * Table 2 counts): a fused QKV projection, attention, an output projection.
 *   X, Y      [B][L][C] bf16 token-major hidden states, C = H * d
 *   Wqkv      [3C][C] bf16, Linear layout (y = x W^T + b); output feature
 *             f = which * C + head * d + dim with which 0/1/2 = q/k/v
 *   bqkv      [3C] fp32 (may be NULL: no bias)
 *   Wo, bo    [C][C] bf16 and [C] fp32 (bo may be NULL)
 * Supported shapes: d in {64, 72} and C a multiple of 128 (else
 * DFA_ERR_UNSUPPORTED).  Outputs must not overlap inputs or each other. */

/* QKV projection: Q, K, V [B][H][L][d] = split(X Wqkv^T + bqkv). */
dfa_status dfa_qkv_proj(const void* X, const void* Wqkv, const void* bqkv, void* Q, void* K, void* V,
                        int B, int H, int L, int d, hipStream_t stream);

/* Output projection: Y = merge(O) Wo^T + bo, merge reading O [B][H][L][d] as the
 * [B][L][H * d] concatenation of heads. */
dfa_status dfa_out_proj(const void* O, const void* Wo, const void* bo, void* Y, int B, int H, int L, int d,
                        hipStream_t stream);

/* One attention module of one layer at one step under plan `code` (the codes
 * of dfa_plan_step), with the module-level caches:
 *   AST          the whole module is skipped: Y = Ycache (a no-op when
 *                Ycache == Y; X, weights and workspaces are not read and may
 *                be NULL)
 *   ASC, WARS_ASC_REFRESH, WARS_ASC_REUSE
 *                the module, projections included, runs on the conditional
 *                half (b < B/2) only; its output is stored to both halves
 *                (Sec. 3.4).  B must be even.
 *   other codes  QKV projection, the attention step of dfa_plan_step, output
 *                projection, on the whole batch.
 * Q, K, V, O are caller-owned [B][H][L][d] bf16 workspaces (the half-batch
 * codes use their first halves); R is the layer's fp32 residual [B][H][L][d]
 * in the space of the attention output before the output projection (Eq. 1-2;
 * required by the four WA-RS codes, ignored otherwise).  Every computed step
 * also writes its output to Ycache (unless Ycache is NULL or equal to Y).
 * The kernels run back to back on `stream`. */
dfa_status dfa_module_step(int code, const void* X, const void* Wqkv, const void* bqkv, const void* Wo,
                           const void* bo, void* Q, void* K, void* V, void* O, void* R, void* Y, void* Ycache,
                           int B, int H, int L, int d, int w, hipStream_t stream);

/* Mean relative absolute error of the plan search (Sec. 3.5):
 *   L(A, B) = mean_i clip(|A_i - B_i| / (max(|A_i|, |B_i|) + 1e-6), 0, 10)
 * over n bf16 elements (DEVICE pointers, 16-byte aligned).  The result is
 * written as one fp64 value to the DEVICE pointer `result` (8-byte aligned).  `workspace` is a
 * caller-owned DEVICE buffer of DFA_MRAE_WORKSPACE_BYTES (per-workgroup
 * partial sums; calls that share it must not overlap).  Each lane sums its
 * share in fp32, the partial sums are added in fp64 in a fixed order: the
 * result is deterministic. */
#define DFA_MRAE_WORKSPACE_BYTES 8192
dfa_status dfa_mrae(const void* A, const void* B, size_t n, void* workspace, double* result, hipStream_t stream);

/* dfa_mrae without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): same arguments otherwise, same kernels and grid, so
 * the same result bit for bit.  It calls no hipMalloc, hipFree or other
 * allocating routine.  Its per-workgroup partial sums live in a fixed device
 * array of the library, 8 KiB (1024 fp64 values) per device, held from the
 * first call on a device until the process ends; its address is looked up on
 * that first call, with the calling thread's current device (the device of
 * `stream`).  The grid of the reduction is capped at 1024 workgroups, so every
 * n up to DFA_MRAE_NOALLOC_MAX_ELEMS fits; a larger n returns
 * DFA_ERR_INVALID_ARG.  Every call on a device shares that device's array and
 * leaves its partial sums there (each call writes every partial sum it reads,
 * so nothing needs clearing); calls that overlap in time on one device, e.g.
 * on two streams, race on it and must be serialised by the caller. */
#define DFA_MRAE_NOALLOC_MAX_ELEMS (1ULL << 40)
dfa_status dfa_mrae_noalloc(const void* A, const void* B, size_t n, double* result, hipStream_t stream);

/* Bytes of DEVICE workspace dfa_plan_search needs (0 for bad sizes). */
size_t dfa_plan_search_workspace_bytes(int n_layers, int B, int H, int L, int d);

/* The greedy plan search of Alg. 1 (Sec. 3.5) on a surrogate model: a stack of
 * n_layers attention modules (dfa_module_step), each with a residual
 * connection, X <- X + module_i(X), evaluated at the hidden states
 * X_steps[t] ([B][L][C] bf16 DEVICE pointers, one per denoising step).
 * Per step t the output O of the uncompressed model is formed; then for each
 * layer i the strategies AST, WA-RS + ASC, WA-RS, ASC, ordered from the
 * largest computation reduction to the smallest (the module FLOP fractions at
 * this L, C and w; ties keep that order), are applied to layer i alone on top
 * of the choices already made for layers < i at this step, and the first with
 * dfa_mrae(O, O') < ((i + 1) / n_layers) * delta is kept.  An uncompressed
 * layer runs as DFA_WARS_REFRESH, so it is the residual source of later reuse
 * steps; WA-RS needs such a refresh, AST a computed step before, ASC an even B.
 *   Wqkv, bqkv, Wo, bo  HOST arrays of n_layers DEVICE pointers (bqkv, bo may
 *                       be NULL arrays: no biases)
 *   workspace           caller-owned DEVICE buffer, 256-byte aligned, of at
 *                       least dfa_plan_search_workspace_bytes() (module caches
 *                       and scratch; its contents are overwritten)
 *   plan, loss          HOST outputs [n_steps][n_layers]: the plan code per
 *                       layer and step, and the accepted strategy's loss (NaN
 *                       where the layer is not compressed)
 * The host loop synchronises `stream` after each loss evaluation. */
dfa_status dfa_plan_search(int n_layers, int n_steps, const void* const* X_steps, const void* const* Wqkv,
                           const void* const* bqkv, const void* const* Wo, const void* const* bo, double delta,
                           int B, int H, int L, int d, int w, void* workspace, size_t workspace_bytes,
                           int32_t* plan, double* loss, hipStream_t stream);

/* Host only (no device is touched).  Draws a seeded per-(step, layer) plan in
 * place of the searched plan dictionary of Alg. 1 and resolves its cache
 * sources.  Output arrays are int32, step-major [n_steps][n_layers]:
 *   code[t][l]   executed plan code (DFA_FULL .. DFA_ASC_REUSE)
 *   r_src[t][l]  for DFA_WARS_REUSE the step whose residual is read, else -1
 *   o_src[t][l]  for DFA_AST_REUSE the step whose output is returned, else t
 * Drawing: a SplitMix64 stream (Steele, Lea and Flood 2014) seeded with
 * `seed`, one draw per entry in step-major order; the draw's upper 32 bits
 * map to a code by ((x >> 32) * 5) >> 32.  Legality repair, in order:
 *   1. AST before the layer has a cached output             -> FULL
 *   2. refresh_every > 0: REFRESH and REUSE draws both mean WA-RS; the entry
 *      is REFRESH when the layer has no residual or its residual is at least
 *      refresh_every steps old, else REUSE
 *   3. refresh_every == 0: REUSE before the layer's first refresh -> REFRESH
 *   4. ASC drawn with an odd B                             -> DFA_ERR_INVALID_ARG
 *      (the entries before it are already written; the arrays' contents are
 *      then unspecified)
 * n_layers, n_steps, B >= 1 and refresh_every >= 0 are required. */
dfa_status dfa_plan_make(uint64_t seed, int n_layers, int n_steps, int refresh_every, int B,
                         int32_t* code, int32_t* r_src, int32_t* o_src);

/* Message for the last non-OK status returned on the calling thread (an empty
 * string if there was none).  The pointer stays valid until the next call on
 * the same thread. */
const char* dfa_last_error(void);

/* Library version as "major.minor.patch". */
const char* dfa_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DFA_H */
