/*
 * flarepp.h -- C ABI of libflarepp.so, the FLARE++ mixer forward and
 * backward on AMD MI355X (gfx950).
 *
 * The operations follow "FLARE++: Low-rank attention with dynamic attention
 * routing" (arXiv 2608.11519):
 *
 *   project   K = X W_K, V = X W_V, K~ = X W~_K, V~ = X W~_V, each split into
 *             H heads of width D = C / H                (Sec. 3.1 Eq. (4);
 *                                                         Sec. 3.2 Eqs. (7), (9))
 *   route     rectangular SDPA, softmax(Q K^T / sqrt(D)) V, with the softmax
 *             over the keys (Sec. 3.1 Eq. (3)).  ENCODE: M route queries over
 *             N token keys (Eqs. (8), (10)); DECODE: N token queries over the
 *             M routes (Eq. (11)).
 *   mixer     project; Q = SDPA(Q~, K~, V~); Z = SDPA(Q, K, V);
 *             Y = SDPA(K, Q, Z); O = [Y_1 .. Y_H] W_O  (Fig. 1; Sec. 3.2)
 *
 * Conventions shared by every entry point:
 *   - All tensors are dense, row-major, in device memory (hipMalloc or any
 *     allocation the device can address), 16-byte aligned.
 *   - dtype selects the storage type of X, the weights, the seeds, the
 *     token-side tensors and the outputs: FLAREPP_F32 (float) or FLAREPP_BF16
 *     (bfloat16 bits).  Accumulation and softmax are always fp32.  With bf16,
 *     MFMA operands (including the softmax numerators and the synthesised
 *     queries / latents) are rounded to bf16; with f32 they stay fp32.
 *   - Head h owns channels [h*D, (h+1)*D).  Weights are [C_in][C_out] and act
 *     as out = X W (no biases).  The softmax scale is 1/sqrt(D) in every call.
 *   - D must be 16, 32 or 64, and C = H*D a multiple of 32 for the project
 *     and mixer entry points.  Every size must be >= 1.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream).
 *     The library never allocates, frees or synchronises; the caller owns
 *     every buffer, including the workspace, which must stay alive until the
 *     enqueued work has finished.  Calls that share a workspace must not
 *     overlap.
 *   - Results are deterministic: the same inputs on the same device give
 *     bitwise identical outputs (fixed reduction orders, no float atomics).
 *   - Return value: FLAREPP_OK (0) or a negative FLAREPP_ERR_* code.
 *     Arguments are validated before anything is enqueued: on an error
 *     nothing is launched.  flarepp_last_error() describes the last failure
 *     of the calling thread.  Faults inside kernels surface at the caller's
 *     next synchronisation.
 */
#ifndef FLAREPP_H_
#define FLAREPP_H_

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__)
#define FLAREPP_API __attribute__((visibility("default")))
#else
#define FLAREPP_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

#define FLAREPP_OK 0
#define FLAREPP_ERR_INVALID_ARG (-1) /* size < 1, C % H != 0, null or misaligned pointer */
#define FLAREPP_ERR_UNSUPPORTED (-2) /* D not in {16,32,64}, unknown dtype/kind, too large */
#define FLAREPP_ERR_WORKSPACE (-3)   /* workspace null or smaller than required */
#define FLAREPP_ERR_HIP (-4)         /* a kernel launch failed */

#define FLAREPP_F32 0
#define FLAREPP_BF16 1

#define FLAREPP_ENCODE 0 /* softmax over the N token keys (routes gather tokens) */
#define FLAREPP_DECODE 1 /* softmax over the M route keys (tokens read routes) */

/* Description of the last error on the calling thread ("" if none). */
FLAREPP_API const char* flarepp_last_error(void);

/* Library version string. */
FLAREPP_API const char* flarepp_version(void);

/* ---------------------------------------------------------------------------
 * Project (Sec. 3.1 Eq. (4); Sec. 3.2 Eqs. (7), (9)).
 *
 * X [B][N][C] and W* [C][C] in dtype.  For each non-null (W, out) pair,
 * out [B][H][N][D] = X W split into heads.  At least one pair must be given;
 * a pair with exactly one null pointer is INVALID_ARG.  The workspace holds
 * the weights re-laid out as MFMA fragments.
 * ------------------------------------------------------------------------- */
FLAREPP_API size_t flarepp_project_workspace_bytes(int dtype, int64_t C);
FLAREPP_API int flarepp_project(int dtype, int64_t B, int64_t N, int64_t C, int64_t H,
                    const void* X, const void* Wk, const void* Wv, const void* Wkt,
                    const void* Wvt, void* K, void* V, void* Kt, void* Vt,
                    void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Route: one rectangular SDPA call with M routes and N tokens per (b, h)
 * (Sec. 3.1 Eq. (3)).
 *
 * FLAREPP_ENCODE (Eqs. (8), (10)):
 *   q    route queries, float32 [B][H][M][D]; route_batch_stride is the
 *        element stride between batch entries: H*M*D, or 0 when one [H][M][D]
 *        set is shared by the whole batch (the learned seeds, App. A.1).
 *   k, v token keys and values, dtype [B][H][N][D].
 *   out  float32 [B][H][M][D] = softmax_N(q k^T / sqrt(D)) v.
 *   lse  float32 [B][H][M] natural-log normaliser
 *        log sum_n exp(q . k_n / sqrt(D)) (App. A.2 Eq. (20)), or NULL.
 * FLAREPP_DECODE (Eq. (11)):
 *   q    token queries, dtype [B][H][N][D] (the keys K of the mixer).
 *   k, v route keys and values, float32 [B][H][M][D] (Q(X) and Z);
 *        route_batch_stride as above applies to both.
 *   out  dtype [B][N][H*D]: token n, head h at channels [h*D, (h+1)*D) =
 *        softmax_M(q_n k^T / sqrt(D)) v (heads merged, Sec. 3.1).
 *   lse  must be NULL.
 * Route-side inputs are rounded to the MFMA operand type inside the call.
 * ------------------------------------------------------------------------- */
FLAREPP_API size_t flarepp_route_workspace_bytes(int kind, int dtype, int64_t B, int64_t H,
                                     int64_t N, int64_t M, int64_t D);
FLAREPP_API int flarepp_route(int kind, int dtype, int64_t B, int64_t H, int64_t N, int64_t M,
                  int64_t D, const void* q, int64_t route_batch_stride,
                  const void* k, const void* v, void* out, float* lse,
                  void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Whole mixer forward (Fig. 1; Sec. 3.2 Eqs. (7)-(11)).
 *
 * X [B][N][C]; Wk, Wv, Wkt (W~_K), Wvt (W~_V), Wo [C][C]; seeds (the learned
 * Q~, shared by the batch) [H][M][D]; O [B][N][C] -- all in dtype.
 * M may exceed N.  The workspace holds the projections, the split-key
 * partials, Q(X), Z and Y; size it with flarepp_mixer_workspace_bytes.
 * ------------------------------------------------------------------------- */
FLAREPP_API size_t flarepp_mixer_workspace_bytes(int dtype, int64_t B, int64_t N, int64_t C,
                                     int64_t H, int64_t M);
FLAREPP_API int flarepp_mixer_forward(int dtype, int64_t B, int64_t N, int64_t C, int64_t H,
                          int64_t M, const void* X, const void* Wk, const void* Wv,
                          const void* Wkt, const void* Wvt, const void* Wo,
                          const void* seeds, void* O, void* ws, size_t ws_bytes,
                          void* stream);

/* ---------------------------------------------------------------------------
 * Allocation-free mixer forward, for callers that cannot allocate device
 * memory (work recorded under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  It computes exactly what
 * flarepp_mixer_forward computes (bit for bit, same kernels) without a
 * workspace argument: its workspace is a static scratch array of
 * flarepp_mixer_noalloc_max_bytes() bytes (32 MiB) in the library's device
 * code, so every device the library runs on holds its own copy until the
 * process ends.  The caller passes inputs and outputs as for
 * flarepp_mixer_forward; nothing is allocated or freed.
 *
 * The work runs on the current device, and `stream` (NULL = the null
 * stream) must belong to it (FLAREPP_ERR_INVALID_ARG otherwise).  Every call
 * on a device shares that device's array and leaves its contents behind:
 * calls that overlap in time on one device (on two streams, or from two
 * threads) race on it and must not be issued.  Only shapes that take the
 * fused kernels are covered (FLAREPP_ERR_UNSUPPORTED otherwise, see
 * flarepp_mixer_path), and only while flarepp_mixer_workspace_bytes(...) of
 * the shape is at most the array's size (FLAREPP_ERR_WORKSPACE otherwise);
 * both are checked before anything is enqueued.  Other errors as
 * flarepp_mixer_forward.
 * ------------------------------------------------------------------------- */
FLAREPP_API size_t flarepp_mixer_noalloc_max_bytes(void);
FLAREPP_API int flarepp_mixer_forward_noalloc(int dtype, int64_t B, int64_t N, int64_t C, int64_t H,
                                              int64_t M, const void* X, const void* Wk, const void* Wv,
                                              const void* Wkt, const void* Wvt, const void* Wo,
                                              const void* seeds, void* O, void* stream);

/* Which kernel sequence flarepp_mixer_forward runs for this shape:
 * FLAREPP_PATH_FUSED (projections inside the routing kernels, decode fused
 * with the merge; used when C is 64, 128 or 256 and the per-wave register
 * and LDS budgets allow) or FLAREPP_PATH_UNFUSED (projection GEMM, three
 * routing calls over materialised K, V, K~, V~, merge GEMM).  Both compute
 * the same function.  Negative FLAREPP_ERR_* for an invalid shape. */
#define FLAREPP_PATH_UNFUSED 0
#define FLAREPP_PATH_FUSED 1
FLAREPP_API int flarepp_mixer_path(int dtype, int64_t B, int64_t N, int64_t C, int64_t H,
                                   int64_t M);

/* As flarepp_mixer_forward, and also copies the stage results for checking:
 * Q_out, Z_out float32 [B][H][M][D] (the synthesised queries Q(X) and the
 * latents Z), Y_out dtype [B][N][C] (decoded tokens, heads merged, before
 * W_O).  Each may be NULL. */
FLAREPP_API int flarepp_mixer_forward_debug(int dtype, int64_t B, int64_t N, int64_t C, int64_t H,
                                int64_t M, const void* X, const void* Wk, const void* Wv,
                                const void* Wkt, const void* Wvt, const void* Wo,
                                const void* seeds, void* O, float* Q_out, float* Z_out,
                                void* Y_out, void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Fixed-query FLARE mixer forward (Sec. 3.1, Eqs. (4)-(5)): the baseline
 * that FLARE++ generalises.  Per head h, with learned queries Q_h:
 *   K = X Wk, V = X Wv (head h = columns [hD, (h+1)D)),
 *   Z_h = softmax_N(Q_h K_h^T / sqrt(D)) V_h        (encode, softmax over N),
 *   Y_h = softmax_M(K_h Q_h^T / sqrt(D)) Z_h        (decode, softmax over M),
 *   O = [Y_1 .. Y_H] Wo.
 * It is FLARE++ without the query synthesis (call 1): the same kernels, with
 * `queries` in place of Q(X).
 *
 * X [B][N][C]; Wk, Wv, Wo [C][C] (out = X W); queries [H][M][D], shared by
 * the batch; O [B][N][C] -- all in dtype.  Sizes, layouts, ownership,
 * determinism and errors as flarepp_mixer_forward; size the workspace with
 * flarepp_flare_workspace_bytes (0 for an invalid shape).
 * flarepp_flare_forward_debug also writes Z_out float32 [B][H][M][D] and
 * Y_out dtype [B][N][C] (decoded tokens, heads merged, before Wo); each may
 * be NULL.
 * ------------------------------------------------------------------------- */
FLAREPP_API size_t flarepp_flare_workspace_bytes(int dtype, int64_t B, int64_t N, int64_t C,
                                                 int64_t H, int64_t M);
FLAREPP_API int flarepp_flare_forward(int dtype, int64_t B, int64_t N, int64_t C, int64_t H,
                                      int64_t M, const void* X, const void* Wk, const void* Wv,
                                      const void* Wo, const void* queries, void* O, void* ws,
                                      size_t ws_bytes, void* stream);
FLAREPP_API int flarepp_flare_forward_debug(int dtype, int64_t B, int64_t N, int64_t C, int64_t H,
                                            int64_t M, const void* X, const void* Wk,
                                            const void* Wv, const void* Wo, const void* queries,
                                            void* O, float* Z_out, void* Y_out, void* ws,
                                            size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Mixer block: O = X + mixer(LN(X)), the pre-norm residual block around the
 * mixer (the residual stream that Sec. 3.2 leaves as it is; only the mixer
 * changes).  LN normalises every token over its C channels:
 * (x - mean) / sqrt(var + eps) * gamma + beta with the biased variance;
 * gamma, beta [C] in dtype, eps > 0.  The normalised tokens go to a
 * workspace buffer (one pass) and through the same kernels as
 * flarepp_mixer_forward; the residual is added where O is stored (the
 * decode's merge, or the merge product on the unfused path).  O must not
 * alias X.  Workspace: flarepp_block_workspace_bytes(...) bytes.  Errors as
 * for flarepp_mixer_forward, plus FLAREPP_ERR_INVALID_ARG for eps <= 0.
 * ------------------------------------------------------------------------- */
FLAREPP_API size_t flarepp_block_workspace_bytes(int dtype, int64_t B, int64_t N, int64_t C, int64_t H,
                                                 int64_t M);
FLAREPP_API int flarepp_block_forward(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M,
                                      const void* X, const void* gamma, const void* beta, float eps,
                                      const void* Wk, const void* Wv, const void* Wkt, const void* Wvt,
                                      const void* Wo, const void* seeds, void* O, void* ws,
                                      size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Backward of the pre-norm residual block O = X + mixer(LayerNorm(X)): the
 * gradients of <O, dO> with respect to X, gamma, beta, the five weights and
 * the seeds.  The layer norm runs again (keeping each token's mean and
 * 1 / sqrt(var + eps)), the mixer backward runs on the normalised tokens, and
 * dX = dO + rstd (g - mean_c(g) - xhat mean_c(g xhat)) with g = dXn * gamma,
 * xhat the normalised token and dXn the mixer's input gradient; dgamma =
 * sum_tokens dXn * xhat and dbeta = sum_tokens dXn in fixed-order sums.
 * Inputs as for flarepp_block_forward plus dO [B][N][C] (dtype); outputs
 * fp32, overwritten: dX [B][N][C], dgamma and dbeta [C], the rest as for
 * flarepp_mixer_backward.  Workspace:
 * flarepp_block_backward_workspace_bytes(...) bytes (0 for an invalid shape).
 * Errors as for flarepp_mixer_backward, plus FLAREPP_ERR_INVALID_ARG for
 * eps <= 0.
 * ------------------------------------------------------------------------- */
FLAREPP_API size_t flarepp_block_backward_workspace_bytes(int dtype, int64_t B, int64_t N, int64_t C,
                                                          int64_t H, int64_t M);
FLAREPP_API int flarepp_block_backward(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M,
                                       const void* X, const void* gamma, const void* beta, float eps,
                                       const void* Wk, const void* Wv, const void* Wkt, const void* Wvt,
                                       const void* Wo, const void* seeds, const void* dO, float* dX,
                                       float* dgamma, float* dbeta, float* dWk, float* dWv, float* dWkt,
                                       float* dWvt, float* dWo, float* dseeds, void* ws, size_t ws_bytes,
                                       void* stream);

/* ---------------------------------------------------------------------------
 * Shared-projection mixer: FLARE++ with the query-synthesis keys and values
 * tied to the physical ones (K~ = K, V~ = V), the variant the paper's cost
 * model leaves open (App. C.2): call 1 is Q = SDPA(Q~, K, V).  Same
 * arguments, workspace (flarepp_mixer_workspace_bytes) and errors as
 * flarepp_mixer_forward without Wkt and Wvt; the result equals
 * flarepp_mixer_forward(..., Wkt = Wk, Wvt = Wv, ...) bit for bit.  Every
 * routing kernel projects its own operands from X, so no projection work is
 * saved on this path; what the variant removes is the two C x C parameters.
 * ------------------------------------------------------------------------- */
FLAREPP_API int flarepp_mixer_forward_shared(int dtype, int64_t B, int64_t N, int64_t C, int64_t H,
                                             int64_t M, const void* X, const void* Wk,
                                             const void* Wv, const void* Wo, const void* seeds,
                                             void* O, void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Mixer backward (App. A.5): the gradients of the scalar <O, dO> with respect
 * to every input of flarepp_mixer_forward, for the output gradient
 * dO [B][N][C] (dtype).
 *
 * Each routing call is differentiated from its global output and
 * log-normaliser: with P = exp(s S - L) and c = <dOut, Out> per query row,
 * dV = P^T dOut, dS = P (dOut V^T - c), dK = s dS^T Q, dQ = s dS K.  The
 * decode's query gradient (on the synthesised queries Q) is added to the
 * physical-value encode's before the query-synthesis encode is
 * differentiated; the seed gradient is summed over the batch.  The call runs
 * the forward again itself (nothing needs to be kept from an earlier
 * forward), then the merge, call 3, call 2, call 1 and the projections in
 * reverse order.  Reductions over tokens and key chunks use fixed orders:
 * the results are bitwise reproducible.
 *
 * Inputs as for flarepp_mixer_forward, plus dO.  Outputs, all fp32 and
 * row-major, overwritten: dX [B][N][C]; dWk, dWv, dWkt, dWvt, dWo [C][C]
 * (the layout of the weights, out = X W); dseeds [H][M][D].  With bf16 the
 * MFMA operands, and the token gradients dY, dK, dK~ kept between the
 * kernels, are rounded to bf16; the value gradients dV, dV~ are kept as two
 * bf16 parts (hi + lo, ~16 bits), because the weight gradients X^T dV are
 * made of their small token-dependent part; accumulation is fp32.
 *
 * Sizes as for the mixer; in addition B*N <= 2^30 (FLAREPP_ERR_UNSUPPORTED
 * otherwise).  Workspace:
 * flarepp_mixer_backward_workspace_bytes(...) bytes (0 for an invalid or
 * unsupported shape); it holds the forward's K, V, K~, V~, Y and the token
 * gradients dY, dK, dV, dK~, dV~ (and the low parts of dV, dV~ with bf16),
 * about 10 * bytes(dtype) * B * N * C bytes (12 with bf16).
 * flarepp_mixer_backward_debug also writes the summed latent gradient dZ and
 * the summed query gradient dQ (fp32 [B][H][M][D] each) when non-null.
 * ------------------------------------------------------------------------- */
FLAREPP_API size_t flarepp_mixer_backward_workspace_bytes(int dtype, int64_t B, int64_t N,
                                                          int64_t C, int64_t H, int64_t M);
FLAREPP_API int flarepp_mixer_backward(int dtype, int64_t B, int64_t N, int64_t C, int64_t H,
                                       int64_t M, const void* X, const void* Wk, const void* Wv,
                                       const void* Wkt, const void* Wvt, const void* Wo,
                                       const void* seeds, const void* dO, float* dX, float* dWk,
                                       float* dWv, float* dWkt, float* dWvt, float* dWo,
                                       float* dseeds, void* ws, size_t ws_bytes, void* stream);
FLAREPP_API int flarepp_mixer_backward_debug(int dtype, int64_t B, int64_t N, int64_t C, int64_t H,
                                             int64_t M, const void* X, const void* Wk,
                                             const void* Wv, const void* Wkt, const void* Wvt,
                                             const void* Wo, const void* seeds, const void* dO,
                                             float* dX, float* dWk, float* dWv, float* dWkt,
                                             float* dWvt, float* dWo, float* dseeds, float* dZ_out,
                                             float* dQ_out, void* ws, size_t ws_bytes,
                                             void* stream);

/* ---------------------------------------------------------------------------
 * Backward of the shared-projection mixer (flarepp_mixer_forward_shared,
 * K~ = K and V~ = V; App. C.2): the gradients of <O, dO> with respect to X,
 * the tied W_K and W_V, W_O and the seeds.  A tied weight's gradient is the
 * sum of its two uses, dWk = X^T (dK + dK~) and dWv = X^T (dV + dV~), formed
 * in one fixed-order reduction.  Arguments, outputs, precision, workspace
 * (flarepp_mixer_backward_workspace_bytes) and errors as for
 * flarepp_mixer_backward without Wkt, Wvt, dWkt and dWvt.
 * ------------------------------------------------------------------------- */
FLAREPP_API int flarepp_mixer_backward_shared(int dtype, int64_t B, int64_t N, int64_t C, int64_t H,
                                              int64_t M, const void* X, const void* Wk, const void* Wv,
                                              const void* Wo, const void* seeds, const void* dO, float* dX,
                                              float* dWk, float* dWv, float* dWo, float* dseeds, void* ws,
                                              size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Training pair: a forward that keeps what the backward needs, and a backward
 * that reads it instead of running the forward again.
 *
 * flarepp_mixer_forward_train computes O like flarepp_mixer_forward (on the
 * unfused kernels, the results agree within rounding) and leaves in `ws`
 * (flarepp_mixer_backward_workspace_bytes bytes) the projections K, V, K~,
 * V~, the decoded tokens Y, Q(X), Z and the three log-normalisers.
 * flarepp_mixer_backward_from_saved then computes exactly what
 * flarepp_mixer_backward computes for the same inputs (bit for bit), given a
 * workspace that a flarepp_mixer_forward_train with the same sizes and inputs
 * filled and that nothing has written since; it does not modify the saved
 * state, so one forward can serve several output gradients.  Arguments,
 * outputs and errors as for flarepp_mixer_forward and flarepp_mixer_backward.
 * ------------------------------------------------------------------------- */
FLAREPP_API int flarepp_mixer_forward_train(int dtype, int64_t B, int64_t N, int64_t C, int64_t H, int64_t M,
                                            const void* X, const void* Wk, const void* Wv, const void* Wkt,
                                            const void* Wvt, const void* Wo, const void* seeds, void* O,
                                            void* ws, size_t ws_bytes, void* stream);
FLAREPP_API int flarepp_mixer_backward_from_saved(int dtype, int64_t B, int64_t N, int64_t C, int64_t H,
                                                  int64_t M, const void* X, const void* Wk, const void* Wv,
                                                  const void* Wkt, const void* Wvt, const void* Wo,
                                                  const void* seeds, const void* dO, float* dX, float* dWk,
                                                  float* dWv, float* dWkt, float* dWvt, float* dWo,
                                                  float* dseeds, void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Profiling variant of flarepp_mixer_forward for timing each stage on the
 * device.  `events` holds FLAREPP_PROFILE_EVENTS caller-created hipEvent_t
 * handles (created with timing enabled); events[0] is recorded on `stream`
 * before the first launch and events[i] after stage i:
 *   1 weight fragments and seed operands   5 call 2 (encode) partials
 *   2 project K, V, K~, V~                 6 call 2 combine -> Z
 *   3 call 1 (query synthesis) partials    7 call 3 (decode) -> Y
 *   4 call 1 combine -> Q(X)               8 merge O = Y W_O
 * On the fused path stages 2 and 8 are empty: the projections run inside
 * stages 3, 5 and 7, and the merge inside stage 7.
 * The library only records the events; reading them (hipEventElapsedTime
 * after a synchronisation) is the caller's.  n_events must be
 * FLAREPP_PROFILE_EVENTS, or 0 (then this is flarepp_mixer_forward).
 * ------------------------------------------------------------------------- */
#define FLAREPP_PROFILE_EVENTS 9
FLAREPP_API int flarepp_mixer_forward_profiled(int dtype, int64_t B, int64_t N, int64_t C,
                                   int64_t H, int64_t M, const void* X, const void* Wk,
                                   const void* Wv, const void* Wkt, const void* Wvt,
                                   const void* Wo, const void* seeds, void* O, void* ws,
                                   size_t ws_bytes, void* stream, void* const* events,
                                   int n_events);

/* Runs stage `stage` (1 .. FLAREPP_PROFILE_EVENTS - 1, numbered as for
 * flarepp_mixer_forward_profiled) of flarepp_mixer_forward alone, for timing
 * one kernel in isolation.  The workspace must hold what a complete
 * flarepp_mixer_forward with the same arguments left in it; the stage then
 * recomputes and rewrites exactly the values it wrote there (its inputs are
 * unchanged), so it may be launched any number of times or captured into a
 * graph.  An empty stage launches nothing.  Errors as flarepp_mixer_forward,
 * and FLAREPP_ERR_INVALID_ARG for a stage outside that range. */
FLAREPP_API int flarepp_mixer_stage(int stage, int dtype, int64_t B, int64_t N, int64_t C,
                                    int64_t H, int64_t M, const void* X, const void* Wk,
                                    const void* Wv, const void* Wkt, const void* Wvt,
                                    const void* Wo, const void* seeds, void* O, void* ws,
                                    size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FLAREPP_H_ */
