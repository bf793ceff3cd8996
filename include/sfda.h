/*
 * libsfda -- Semidirect Fourier Delta Attention (SFDA) forward and decode on AMD MI355X (gfx950).
 *
 * Plain C ABI: device pointers, sizes and a HIP stream passed as an opaque pointer.  No C++,
 * HIP or framework types cross this boundary.
 *
 * The operation (Sec. 3, Eq. (sfda) and the readout that follows it), per batch b and head h,
 * over complex coordinates, with x^* the conjugate transpose:
 *
 *   Lambda_t = diag(alpha_t * exp(i theta_t))             alpha_t, theta_t real, m channels
 *   S_t      = (I - beta_t k_t k_t^*) Lambda_t S_{t-1} + beta_t k_t v_t^*      S_t in C^{m x n}
 *   o_t      = S_t^* q_t                                  (state after token t's update)
 *
 * so that (k v^*)_{ij} = k_i conj(v_j) and o_{t,j} = sum_i conj(S_t[i][j]) q_t[i].
 *
 * Memory layouts (row-major, contiguous; complex = interleaved (re, im) scalar pairs):
 *   q, k          [B, H, T, m] complex     v, o   [B, H, T, n] complex
 *   alpha, theta  [B, H, T, m] real        beta   [B, H, T]    real
 *   S0, S_T, S    [B, H, m, n] complex, always float32
 * Element type of q, k, v, alpha, theta, beta is `in_dtype`; of o it is `out_dtype`.
 * For the decode step drop the T axis: q, k [B, H, m], v, o [B, H, n], alpha, theta [B, H, m],
 * beta [B, H].
 *
 * Ownership: the caller allocates and frees every buffer (including the workspaces of
 * sfda_chunk_fwd_segmented and sfda_chunk_bwd) and owns the stream; the library allocates
 * no device memory and keeps no state between calls (calls are reentrant; calls
 * that write the same buffers on different streams race, as any two kernels would).
 *
 * Errors: all argument checks run on the host before anything is enqueued; on any error
 * nothing is launched and a status code is returned.  A launch failure returns
 * SFDA_ERR_HIP.  Faults inside a kernel surface at the caller's next synchronisation.
 * Nothing aborts, throws or prints.
 *
 * Determinism: no atomics; for identical inputs, sizes and dtypes results are bitwise
 * identical from run to run.
 */
#ifndef SFDA_H
#define SFDA_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SFDA_ABI_VERSION 3

/* Element types and status codes are plain ints (the names below are their values), so
 * any value a caller passes is well defined: an unknown dtype is SFDA_ERR_DTYPE, an unknown
 * status has its own text. */
enum { SFDA_F32 = 0, SFDA_BF16 = 1 };
typedef int sfda_dtype_t;

enum {
    SFDA_OK = 0,
    SFDA_ERR_NULL = 1,   /* a required pointer is NULL                                   */
    SFDA_ERR_SHAPE = 2,  /* a size is out of range (see each entry point)                 */
    SFDA_ERR_CHUNK = 3,  /* chunk length C not supported                                  */
    SFDA_ERR_DTYPE = 4,  /* unknown dtype                                                 */
    SFDA_ERR_ALIGN = 5,  /* a pointer is not 16-byte aligned                              */
    SFDA_ERR_ALIAS = 6,  /* an output overlaps an input or another output                 */
    SFDA_ERR_HIP = 7,    /* the HIP runtime reported an error when launching              */
    SFDA_ERR_SCRATCH = 8 /* sfda_chunk_fwd_segmented_noalloc: the call needs more workspace
                            than SFDA_NOALLOC_SCRATCH_BYTES                                */
};
typedef int sfda_status_t;

/* A hipStream_t passed as an opaque pointer; NULL means the default (null) stream. */
typedef void* sfda_stream_t;

/*
 * sfda_chunk_fwd -- the whole forward pass over T tokens, evaluated chunk by chunk through
 * the constructive chunk-WY factorisation P = Gamma - Y M W^* (Thm 4.2, Cor. 4.3) with the
 * exact affine chunk transfer (Thm 4.4), the intra-chunk prefix outputs (Thm 4.5) and a
 * sequential boundary-state scan across chunks (Thm 6.1, eq. (apply-transfer)).  The result
 * equals the token-by-token recurrence above up to floating-point rounding.
 *
 *   q, k, v, alpha, theta, beta : inputs (device, in_dtype), layouts above.
 *   S0   : initial state [B,H,m,n] complex float32, or NULL for the zero state.
 *   o    : output [B,H,T,n] complex (device, out_dtype); every element is written.
 *   S_T  : state after token T [B,H,m,n] complex float32, or NULL if not wanted.
 *          S_T == S0 (same pointer) is allowed and updates the state in place; any other
 *          overlap between S_T and another buffer is SFDA_ERR_ALIAS.
 *   B, H >= 0 (B*H == 0 is a no-op); T >= 0 (T == 0 writes S_T = S0, or zeros);
 *   1 <= m <= 64; n >= 1 with m * n < 2^28 and n < 2^23 (one head's state and 32 tokens'
 *   rows of v and o are addressed with 32-bit byte offsets; SFDA_ERR_SHAPE otherwise);
 *   C in {16, 32, 64, 128} (SFDA_ERR_CHUNK otherwise).  The last chunk may be ragged
 *   (T mod C != 0).
 *   Chunk length: C fixes the paper's chunking; the result does not depend on it (Thm 6.1,
 *   up to rounding), and the kernels choose their own blocking.  bf16 inputs with m > 4 run
 *   64-token steps of four 16-token blocks for every C (bitwise the same result for every
 *   C); float32 inputs, and bf16 inputs with m <= 4, run 16-token chunks for every C.
 *   Numerical range (App. C.4, local renormalisation): the decay is referenced to the start
 *   of each aligned 16-token block (tokens 16 j .. 16 j + 15), so the kernels divide by at
 *   most the decay over part of one block.  The result is exact to rounding for every
 *   alpha in (0, 1] whose product over each aligned 16-token block, per channel, is at
 *   least 2^-126 (e.g. any alpha >= 0.0043; alpha may be exactly 1 or vary per channel and
 *   token; the decay over longer stretches is unbounded).  Past that the outputs are NaN
 *   rather than wrong: with bf16 inputs (m > 4) from the 64-token step holding such a block
 *   on, otherwise from the first token whose block decay so far is below 2^-126 (its
 *   16-token chunk's earlier rows may be NaN too); S_T is NaN in both cases.
 *   Accumulation and state are float32 for both dtypes; with in_dtype == SFDA_BF16 and
 *   m > 4 the matrix products take bfloat16 operands (with m <= 4 they take float32 ones:
 *   there 1 - beta |k|^2 can sit near 0, and the erase factor would amplify the operand
 *   rounding of bfloat16 past its own precision); each head's share of q, k, v and o must
 *   stay below 2 GiB (T * max(m, n) * 2 * sizeof(out element) < 2^31; SFDA_ERR_SHAPE
 *   otherwise).
 */
sfda_status_t sfda_chunk_fwd(const void* q, const void* k, const void* v,
                             const void* alpha, const void* theta, const void* beta,
                             const float* S0, void* o, float* S_T,
                             int B, int H, int T, int m, int n, int C,
                             sfda_dtype_t in_dtype, sfda_dtype_t out_dtype,
                             sfda_stream_t stream);

/*
 * sfda_chunk_fwd_sliced -- sfda_chunk_fwd with an explicit number of value columns per
 * workgroup, `slice` (a multiple of 8 in [8, 64]; SFDA_ERR_SHAPE otherwise).  The n value
 * columns are independent in the recurrence (column j of S only mixes with column j of
 * v^*), so the library splits them into ceil(n / slice) workgroups per (b, h); a smaller
 * slice gives more workgroups at the cost of repeating the chunk factors per slice.
 * sfda_chunk_fwd uses slice = min(64, n rounded up to a multiple of 8), halved to 32 when
 * the heads alone would leave more than half of the device's compute units idle
 * (2 * B * H * ceil(n / slice) <= compute units).  Every column's arithmetic is the same for
 * every slice, so the results are bitwise the same.
 */
sfda_status_t sfda_chunk_fwd_sliced(const void* q, const void* k, const void* v,
                                    const void* alpha, const void* theta, const void* beta,
                                    const float* S0, void* o, float* S_T,
                                    int B, int H, int T, int m, int n, int C, int slice,
                                    sfda_dtype_t in_dtype, sfda_dtype_t out_dtype,
                                    sfda_stream_t stream);

/*
 * sfda_chunk_fwd_gated -- sfda_chunk_fwd on pre-activations: the kernels map them to the
 * recurrence's parameters as they load them (the stable parameterization of Sec. 3,
 * equations param-alpha, param-theta, param-beta and param-key), with no separate pass:
 *   alpha_t = alpha_min + (alpha_max - alpha_min) * sigmoid(a_t)    a:     [B,H,T,m] real
 *   theta_t = theta_max * tanh(b_t)                                  b:     [B,H,T,m] real
 *   beta_t  = sigmoid(c_t)                                           c:     [B,H,T]   real
 *   k_t     = k_raw_t / (||k_raw_t||_2 + eps)   (norm over the m complex channels)
 * q, v, S0, o, S_T, sizes, dtypes, layouts, errors and results as sfda_chunk_fwd (a, b, c,
 * k_raw take the places of alpha, theta, beta, k).  Requires 0 < alpha_min <= alpha_max
 * <= 1, alpha_min >= 0.0042719 (so that alpha_min^16 >= 2^-126: every input is inside
 * sfda_chunk_fwd's numerical range) and finite theta_max, eps >= 0 (SFDA_ERR_SHAPE
 * otherwise).  With eps == 0 an all-zero raw key gives k = 0.
 */
sfda_status_t sfda_chunk_fwd_gated(const void* q, const void* k_raw, const void* v,
                                   const void* a, const void* b, const void* c,
                                   const float* S0, void* o, float* S_T,
                                   int B, int H, int T, int m, int n, int C,
                                   float alpha_min, float alpha_max, float theta_max, float eps,
                                   sfda_dtype_t in_dtype, sfda_dtype_t out_dtype,
                                   sfda_stream_t stream);

/*
 * sfda_chunk_fwd_decoupled -- the write-decoupled variant (Sec. 3, write-decoupled
 * variant): the erase direction and strength are separate from the write direction and
 * strength,
 *   S_t = (I - eta_t k_t k_t^*) Lambda_t S_{t-1} + beta_t r_t v_t^*,   o_t = S_t^* q_t,
 * evaluated chunk by chunk (the erase rows solve a unit lower-triangular system in the
 * k-k Gram block, the write rows are known; outputs and the state update add the q-r and
 * r-state products).  r = k with eta = beta gives sfda_chunk_fwd's result.
 *   r   : [B,H,T,m] complex write directions (device, in_dtype).
 *   eta : [B,H,T] erase strengths; beta : [B,H,T] write strengths (device, in_dtype).
 *   Other arguments, errors and the numerical range as sfda_chunk_fwd's float32 path:
 *   every C runs 16-token chunks (the result does not depend on C).
 */
sfda_status_t sfda_chunk_fwd_decoupled(const void* q, const void* k, const void* r, const void* v,
                                       const void* alpha, const void* theta, const void* eta,
                                       const void* beta, const float* S0, void* o, float* S_T,
                                       int B, int H, int T, int m, int n, int C,
                                       sfda_dtype_t in_dtype, sfda_dtype_t out_dtype,
                                       sfda_stream_t stream);

/*
 * sfda_chunk_fwd_segmented -- sfda_chunk_fwd with each head's sequence cut into G
 * segments of T / G tokens that are scanned in parallel (for few heads over long
 * sequences, where one workgroup per head leaves most of the GPU idle).  It uses the
 * exact affine law of a stretch of tokens (Thm 4.4: S_end = P S_in + B, P the product of
 * the stretch's transitions, B its write from the zero state) composed along the segments
 * (Lemma A.2, the boundary-state scan of Thm 6.1 at segment granularity): chunk passes give
 * every segment's P_g (final state from S0 = I with v = 0) and B_g (final state from
 * S0 = 0), and a fold gives S_in[g + 1] = P_g S_in[g] + B_g and S_T = S_in[G].  With
 * float32 inputs the same two passes also give the readouts X_t = P_t^* q_t and the
 * zero-state outputs o0_t, and a join writes o_t = o0_t + S_in^* X_t (the same law token by
 * token; a bfloat16 o is then rounded twice); with bfloat16 inputs a third pass writes o
 * from the exact incoming states.  With float32 inputs and n <= 64 the two passes run as
 * one scan per segment (one copy of the chunk factors, twice the columns).  Up to two
 * (float32) or three (bfloat16) times the scan work of sfda_chunk_fwd, spread over G times
 * as many workgroups; results agree with it to rounding.
 *   Arguments and errors as sfda_chunk_fwd, plus:
 *   G >= 1 with T a multiple of G * C (SFDA_ERR_SHAPE otherwise; T == 0 is as
 *   sfda_chunk_fwd).
 *   workspace : device memory of at least sfda_chunk_fwd_segmented_workspace_bytes(B, H,
 *               T, m, n, G, in_dtype) bytes (SFDA_ERR_SHAPE if smaller, SFDA_ERR_NULL if
 *               NULL), 16-byte aligned, not overlapping any other argument
 *               (SFDA_ERR_ALIAS); no initial contents needed.  Holds, per segment, P_g
 *               (m x m), B_g and the incoming state (m x n), and with float32 inputs per
 *               token X_t (m), complex float32 (0 for sizes or a dtype out of range).
 *   S_T == S0 (in place) is allowed.
 */
size_t sfda_chunk_fwd_segmented_workspace_bytes(int B, int H, int T, int m, int n, int G,
                                                sfda_dtype_t in_dtype);

/*
 * sfda_chunk_fwd_auto_segments -- the segment count G that the library suggests for
 * sfda_chunk_fwd_segmented on the current device and input dtype: the largest power of two
 * for which the segments' workgroups (B * H * G * ceil(n / 64)) still fit the compute units
 * once each, T is a multiple of G * C and every segment keeps at least 256 tokens; 1 (use
 * sfda_chunk_fwd) when that G is below 4 for float32 inputs or below 8 for bfloat16 ones.
 * The segmented scan does two (float32) or three (bfloat16) times the scan work of
 * sfda_chunk_fwd spread over G times the workgroups, so it pays only when few heads would
 * leave most compute units idle.  Sizes or a dtype out of range, or no device, give 1.
 * Launches nothing and allocates nothing.
 */
int sfda_chunk_fwd_auto_segments(int B, int H, int T, int m, int n, int C, sfda_dtype_t in_dtype);

/*
 * sfda_chunk_fwd_segmented_noalloc -- sfda_chunk_fwd_segmented for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the workspace is a static device array of SFDA_NOALLOC_SCRATCH_BYTES
 * inside the library, one per GPU, held until the process ends.  The call itself allocates
 * nothing (no hipMalloc, hipFree or allocating library routine); its first call on a device
 * looks up that device's scratch address (hipGetSymbolAddress, with the device current).
 *   Arguments, results and errors as sfda_chunk_fwd_segmented without the workspace; a call
 *   whose workspace (sfda_chunk_fwd_segmented_workspace_bytes) exceeds
 *   SFDA_NOALLOC_SCRATCH_BYTES returns SFDA_ERR_SCRATCH before anything is launched.
 *   Every call on one GPU shares that GPU's scratch (no initial contents are needed; each
 *   call overwrites what it uses): calls that overlap in time on one GPU (different
 *   streams, or different host threads without ordering) race.
 */
#define SFDA_NOALLOC_SCRATCH_BYTES (32u * 1024u * 1024u)

sfda_status_t sfda_chunk_fwd_segmented_noalloc(const void* q, const void* k, const void* v,
                                               const void* alpha, const void* theta,
                                               const void* beta, const float* S0, void* o,
                                               float* S_T, int B, int H, int T, int m, int n,
                                               int C, int G, sfda_dtype_t in_dtype,
                                               sfda_dtype_t out_dtype, sfda_stream_t stream);

sfda_status_t sfda_chunk_fwd_segmented(const void* q, const void* k, const void* v,
                                       const void* alpha, const void* theta, const void* beta,
                                       const float* S0, void* o, float* S_T,
                                       int B, int H, int T, int m, int n, int C, int G,
                                       sfda_dtype_t in_dtype, sfda_dtype_t out_dtype,
                                       void* workspace, size_t workspace_bytes,
                                       sfda_stream_t stream);

/*
 * sfda_chunk_bwd -- reverse-mode gradients through sfda_chunk_fwd for a real scalar loss L
 * (the backward of the chunkwise forward, recomputing the chunk factors of Thm 4.2 /
 * Cor. 4.3 instead of storing them).  Given dO = dL/do and dS_T = dL/dS_T it returns the
 * gradients with respect to every input; the gradient of a complex variable z is
 * dL/dRe(z) + i dL/dIm(z).  Three launches on the stream: a forward scan recording the
 * state entering each chunk and the chunk's solve result, a reverse scan carrying dL/dS
 * through the chunks (the adjoint of the boundary-state map of Thm 6.1; it writes dv and
 * dS0), and one workgroup per (head, chunk) forming dq, dk, dalpha, dtheta and dbeta.
 *   q, k, v, alpha, theta, beta, S0 : as sfda_chunk_fwd (in_dtype; S0 NULL = zero state).
 *   dO   : [B,H,T,n] complex (device, out_dtype); dS_T : [B,H,m,n] complex float32 or NULL
 *          (zero).
 *   dq, dk : [B,H,T,m] complex; dv : [B,H,T,n] complex; dalpha, dtheta : [B,H,T,m];
 *          dbeta : [B,H,T] (device, in_dtype, written).  dS0 : [B,H,m,n] complex float32
 *          or NULL (not wanted).  No output may overlap an input, another output or the
 *          workspace (SFDA_ERR_ALIAS).
 *   workspace : device memory of at least sfda_chunk_bwd_workspace_bytes(B, H, T, m, n, C)
 *          bytes (SFDA_ERR_SHAPE if smaller, SFDA_ERR_NULL if NULL and needed), 16-byte
 *          aligned, no initial contents; holds per chunk the state entering it and dL/dS
 *          leaving it (m x n) and two C x n blocks, complex float32.
 *   Sizes, C and dtypes as sfda_chunk_fwd; T == 0 writes dS0 = dS_T (or zeros).  The
 *   chunk length only fixes how the work is blocked (every C gives the same gradients up
 *   to rounding): every C runs 16-token chunks, so that the numerical range is
 *   sfda_chunk_fwd's (each aligned 16-token block decaying by at least 2^-126 per channel;
 *   past it the gradients of that chunk and of the earlier ones are NaN), and the
 *   workspace function sizes for that.
 *   alpha must be nonzero wherever T > 0 (dalpha divides by it).
 */
size_t sfda_chunk_bwd_workspace_bytes(int B, int H, int T, int m, int n, int C);

sfda_status_t sfda_chunk_bwd(const void* q, const void* k, const void* v, const void* alpha,
                             const void* theta, const void* beta, const float* S0,
                             const void* dO, const float* dS_T, void* dq, void* dk, void* dv,
                             void* dalpha, void* dtheta, void* dbeta, float* dS0,
                             int B, int H, int T, int m, int n, int C, sfda_dtype_t in_dtype,
                             sfda_dtype_t out_dtype, void* workspace, size_t workspace_bytes,
                             sfda_stream_t stream);

/*
 * sfda_step -- one recurrent decode token per (b, h) (Sec. 3, Eq. (sfda) and the readout),
 * updating the state in place:
 *   S <- (I - beta k k^*) Lambda S + beta k v^*,   o = S^* q   (post-update S).
 *
 *   q, k, v, alpha, theta, beta : one token per head (device, in_dtype), layouts above.
 *   S : [B,H,m,n] complex float32, read and overwritten.
 *   o : [B,H,n] complex (device, out_dtype).  o must not overlap S or any input.
 *   B, H >= 0; 1 <= m <= 64; 1 <= n < 2^22 (each head's state rows are addressed with
 *   32-bit offsets); SFDA_ERR_SHAPE otherwise.
 */
sfda_status_t sfda_step(const void* q, const void* k, const void* v,
                        const void* alpha, const void* theta, const void* beta,
                        float* S, void* o, int B, int H, int m, int n,
                        sfda_dtype_t in_dtype, sfda_dtype_t out_dtype,
                        sfda_stream_t stream);

/* Static, human-readable text for a status code. */
const char* sfda_status_string(sfda_status_t s);

/*
 * sfda_chunk_solve_monitor -- the conditioning watch that Prop. 6.4 asks for (its bound
 * ||M||_2 <= 1 / (1 - eta) holds when ||L||_2 <= eta < 1, which the gates do not enforce):
 * for every 16-token block of every head (the blocking of the chunk kernels), the
 * triangular solve that forms N = (I + D_beta L')^{-1} is repeated exactly as the float32
 * path's kernels do it (same load stage, Gram products and substitution; with bfloat16
 * inputs and m > 4 the Gram products take bfloat16 operands, as in the backward's scans), and
 *   residual[b, h, blk] = max_ij |((I + D_beta L') N - I)_ij|   (on the L' it used)
 *   lnorm[b, h, blk]    = ||D_beta L'||_F   (an upper bound of the spectral norm)
 * are written, float32, [B, H, ceil(T / 16)].  L'[t, j] = k_t^* diag(g_t / g_j) k_j for j < t
 * inside the block (the chunk relations of Thm 4.2).  A block outside the decay range of
 * sfda_chunk_fwd gives NaN.
 *   k, alpha, theta, beta: as sfda_chunk_fwd's (device, in_dtype); residual, lnorm: device
 *   float32 (either may be NULL, not both; SFDA_ERR_NULL), 16-byte aligned, not
 *   overlapping the inputs or each other (SFDA_ERR_ALIAS).  Sizes as sfda_chunk_fwd (m in
 *   1..64); B, H or T == 0 is a no-op.
 */
sfda_status_t sfda_chunk_solve_monitor(const void* k, const void* alpha, const void* theta,
                                       const void* beta, float* residual, float* lnorm, int B,
                                       int H, int T, int m, sfda_dtype_t in_dtype,
                                       sfda_stream_t stream);

/* SFDA_ABI_VERSION of the built library. */
int sfda_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SFDA_H */
