/*
 * libmlstm: the mLSTM matrix-memory cell of xLSTM 7B (arXiv 2503.13427) on
 * AMD Instinct MI355X (gfx950).
 *
 * The cell (Sec. 2 of the paper, Eqs. 2-5 with the gate activations of
 * Eqs. 7-8), per independent (batch, head) sequence with q^ = q / sqrt(DQK):
 *
 *   m_t  = max(logsig(f~_t) + m_{t-1}, i~_t)
 *   f_t  = exp(logsig(f~_t) + m_{t-1} - m_t),   i_t = exp(i~_t - m_t)
 *   C_t  = f_t C_{t-1} + i_t k_t v_t^T          (DQK x DV, fp32)
 *   n_t  = f_t n_{t-1} + i_t k_t                (DQK, fp32)
 *   h_t  = C_t^T q^_t / max(|n_t^T q^_t|, exp(-m_t))
 *
 * h is the h~ of Eq. 5.  The output gate and Norm of Eq. 6 are a separate
 * entry point, mlstm_output_norm, applied to h~ and o~ afterwards.
 * h_{t-1} is not an input (Eq. 1 lists it, Eqs. 2-9 never use it).
 *
 * Conventions shared by every entry point:
 *  - All tensor pointers are DEVICE pointers, contiguous and row-major, with
 *    16-byte aligned base addresses.  The caller owns every buffer; the
 *    library allocates nothing.
 *  - q, k, v and h share one element type, mlstm_dtype; gates and the state
 *    (C, n, m) are always fp32.
 *  - Arguments are validated on the host before anything is launched; a
 *    rejected call touches no memory and launches nothing.
 *  - Work is enqueued on `hip_stream` (a hipStream_t; NULL = the null stream)
 *    and the call returns after enqueue.  Launch failures are reported as
 *    MLSTM_ERR_HIP; faults during execution surface at the caller's next
 *    synchronisation.
 *  - Inputs are assumed finite, except that i~ = -inf (nothing written),
 *    f~ = +inf (nothing forgotten) and f~ = -inf are allowed.  f~ = -inf is a
 *    forget gate of exactly zero: the state restarts from the zero matrix at
 *    that token, the reset at document borders of packed sequences (App. B,
 *    "Sequence packing"); both entry points support it.  A restart token with
 *    i~ = -inf as well leaves an empty state (m = -inf), for which Eqs. 7-8
 *    are undefined; such rows get h = 0.  NaN/Inf are not checked on the hot
 *    path and propagate.
 *  - The library is stateless and re-entrant.
 */
#ifndef LIBMLSTM_MLSTM_H
#define LIBMLSTM_MLSTM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MLSTM_OK = 0,
    MLSTM_ERR_NULL_PTR = 1,     /* a required pointer is NULL                         */
    MLSTM_ERR_BAD_SHAPE = 2,    /* negative/zero size, or a size product overflows    */
    MLSTM_ERR_UNSUPPORTED = 3,  /* (dtype, DQK, DV, L) combination not built          */
    MLSTM_ERR_MISALIGNED = 4,   /* a tensor base pointer is not 16-byte aligned       */
    MLSTM_ERR_ALIAS = 5,        /* outputs overlap inputs in a way that is not allowed */
    MLSTM_ERR_WORKSPACE = 6,    /* workspace given but smaller than required          */
    MLSTM_ERR_HIP = 7           /* the HIP runtime reported an error at launch         */
} mlstm_status;

typedef enum {
    MLSTM_F32 = 0,   /* q, k, v, h in IEEE fp32                     */
    MLSTM_BF16 = 1   /* q, k, v, h in bfloat16 (bit pattern uint16) */
} mlstm_dtype;

/*
 * Chunkwise-parallel prefill (Sec. 2, "Training Mode": the hidden states are
 * computed chunk by chunk without materialising the per-step states; the
 * sub-steps are those of the FLOP count in App. D.1).
 *
 * Shapes (S = B * NH independent sequences):
 *   q, k  [B, NH, T, DQK]   (dt)        v  [B, NH, T, DV]   (dt)
 *   ipre, fpre [B, NH, T]   fp32 gate pre-activations i~, f~
 *   C0 [B, NH, DQK, DV], n0 [B, NH, DQK], m0 [B, NH]   fp32 initial state;
 *       all three NULL = zero state with m0 = 0; giving only some of them is
 *       MLSTM_ERR_NULL_PTR.
 *   h  [B, NH, T, DV]       (dt)       output h~ for every step
 *   CT [B, NH, DQK, DV], nT [B, NH, DQK], mT [B, NH]   fp32 final state
 *
 * L is the chunk size.  T need not be a multiple of L: the last chunk is
 * then partial, its missing tokens taken as neutral (no input, no decay:
 * i~ = -inf, f~ = +inf), which leaves the state unchanged, and their h rows
 * are not written.
 * T == 0 copies the initial state to the final state; q, k, v, ipre, fpre
 * and h are then not accessed and may be NULL.  The result does not
 * depend on L except through rounding; mT equals the recurrent m_T of Eq. 2.
 *
 * Built combinations (else MLSTM_ERR_UNSUPPORTED):
 *   - MLSTM_BF16, DQK = 256, DV = 512, L in {64, 128}, T < 2^21: the bf16
 *     MFMA kernel (the xLSTM 7B head shape);
 *   - otherwise any dtype and sizes whose fp32 working set (a DQK x DVt state
 *     tile, the chunk's Q, K and V, the L x L gate matrix) fits in 64 KB of
 *     LDS for some power-of-two tile DVt dividing DV, e.g. DQK = DV = 16 with
 *     L = 16: the fp32 VALU kernel.
 *
 * workspace: optional device scratch.  workspace_bytes == 0 runs the fused
 * single-pass kernel.  Otherwise it must be at least
 * mlstm_chunkwise_workspace_bytes(...) (else MLSTM_ERR_WORKSPACE), and the
 * sequence is split into segments processed in parallel, with the segment
 * boundary states passed through the workspace.  Contents on entry are
 * ignored; on return they are undefined.
 *
 * Aliasing: no output may overlap any input or another output
 * (MLSTM_ERR_ALIAS).
 */
mlstm_status mlstm_chunkwise_fwd(const void* q, const void* k, const void* v, mlstm_dtype dt,
                                 const float* ipre, const float* fpre,
                                 const float* C0, const float* n0, const float* m0,
                                 int B, int NH, int T, int DQK, int DV, int L,
                                 void* h, float* CT, float* nT, float* mT,
                                 void* workspace, size_t workspace_bytes, void* hip_stream);

/*
 * mlstm_chunkwise_fwd on strided q, k, v (for instance per-head views of one
 * projection output [B, T, NH, D], which a layer then need not copy into
 * head-major order).  qkv_strides holds 9 element strides: q's for the
 * batch, head and token axes, then k's, then v's; the D elements of a row are
 * contiguous.  Every stride must be a multiple of 8 (16-byte rows;
 * MLSTM_ERR_MISALIGNED), non-negative, with token strides of at least D
 * (MLSTM_ERR_BAD_SHAPE), and one sequence's rows plus 127 more token
 * strides must span under 2^31 bytes and B NH^2 stay under 2^32
 * (MLSTM_ERR_UNSUPPORTED).  The other
 * arguments, results and workspace (mlstm_chunkwise_workspace_bytes) are
 * those of mlstm_chunkwise_fwd; the alias checks cover the element ranges
 * the views span.  Built for the bf16
 * MFMA path (dt = MLSTM_BF16, DQK = 256, DV = 512, L in {64, 128}); other
 * shapes return MLSTM_ERR_UNSUPPORTED.  qkv_strides NULL is MLSTM_ERR_NULL_PTR.
 */
mlstm_status mlstm_chunkwise_fwd_strided(const void* q, const void* k, const void* v,
                                         const int64_t* qkv_strides, mlstm_dtype dt,
                                         const float* ipre, const float* fpre,
                                         const float* C0, const float* n0, const float* m0,
                                         int B, int NH, int T, int DQK, int DV, int L,
                                         void* h, float* CT, float* nT, float* mT,
                                         void* workspace, size_t workspace_bytes, void* hip_stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * mlstm_chunkwise_fwd with no workspace argument and no allocation.  Same
 * arguments (less the workspace), validation, kernels and results as
 * mlstm_chunkwise_fwd given a workspace of mlstm_chunkwise_workspace_bytes
 * bytes: the segment slots live in a fixed device array of
 * mlstm_chunkwise_scratch_bytes() bytes (64 MiB), one per device, which the
 * library holds from the first call on that device until the process ends.
 * A call whose segment schedule needs more than that returns
 * MLSTM_ERR_WORKSPACE and does nothing (mlstm_chunkwise_fwd serves it).
 * Nothing in the array needs clearing between calls (every slot a call
 * reads is written earlier in that call), but calls that overlap in time on
 * one device share it and race: order them (one stream, or events).
 * It calls no hipMalloc or hipFree.
 */
mlstm_status mlstm_chunkwise_fwd_noalloc(const void* q, const void* k, const void* v, mlstm_dtype dt,
                                         const float* ipre, const float* fpre,
                                         const float* C0, const float* n0, const float* m0,
                                         int B, int NH, int T, int DQK, int DV, int L,
                                         void* h, float* CT, float* nT, float* mT, void* hip_stream);
size_t mlstm_chunkwise_scratch_bytes(void);

/*
 * Workspace size (bytes) for the segment-parallel schedule of
 * mlstm_chunkwise_fwd with these arguments; 0 when that schedule would not be
 * used (the call then runs the fused kernel whatever workspace is given).
 */
size_t mlstm_chunkwise_workspace_bytes(int B, int NH, int T, int DQK, int DV, int L, mlstm_dtype dt);

/*
 * One recurrent step (Sec. 2, "Generation Mode", Eqs. 2-5, 7-8), fused into
 * one kernel that streams C once (Sec. 3.1, "Fused Generation Kernels").
 *
 *   q, k [B, NH, DQK] (dt)   v [B, NH, DV] (dt)   ipre, fpre [B, NH] fp32
 *   C [B, NH, DQK, DV], n [B, NH, DQK], m [B, NH]   fp32 state in
 *   h [B, NH, DV] (dt)   C_out, n_out, m_out: the state after the step
 *
 * DQK >= 1 and DV a multiple of 4, DQK * DV <= 2^20.  In-place is allowed:
 * C_out == C, n_out == n and m_out == m may each be equal (exactly, not
 * partially overlapping); any other overlap is MLSTM_ERR_ALIAS.
 */
mlstm_status mlstm_step(const void* q, const void* k, const void* v, mlstm_dtype dt,
                        const float* ipre, const float* fpre,
                        const float* C, const float* n, const float* m,
                        int B, int NH, int DQK, int DV,
                        void* h, float* C_out, float* n_out, float* m_out, void* hip_stream);

typedef enum {
    MLSTM_NORM_LAYER = 0,   /* LayerNorm: (x - mean(x)) / sqrt(var(x) + eps)  */
    MLSTM_NORM_RMS = 1      /* RMSNorm:   x / sqrt(mean(x^2) + eps)           */
} mlstm_norm;

/*
 * Hidden-state output of the cell (Eq. 6 with the output gate of Eq. 9):
 * for every (b, head, t) row of DV values
 *
 *   h_row = sigmoid(o~_row) * (Norm(h~_row) * weight[head] + bias[head])
 *
 * Norm is the headwise norm (Sec. 2 allows RMSNorm or LayerNorm; the 7B
 * model uses LayerNorm), computed in fp32 over the row; var is the mean
 * squared deviation.
 *
 *   h_tilde, o_pre, h [B, NH, T, DV] (dt)   (a decode step is T = 1)
 *   weight, bias [NH, DV] fp32, either may be NULL (weight 1, bias 0)
 *
 * eps must be finite and > 0; norm is MLSTM_NORM_LAYER or MLSTM_NORM_RMS
 * (else MLSTM_ERR_BAD_SHAPE).  Built: DV a multiple of 4, DV <= 2048 (else
 * MLSTM_ERR_UNSUPPORTED).  T == 0 launches nothing.  h may equal h_tilde
 * (in place: each row is read before it is written); any other overlap of h
 * with an input is MLSTM_ERR_ALIAS.
 */
mlstm_status mlstm_output_norm(const void* h_tilde, const void* o_pre, mlstm_dtype dt,
                               const float* weight, const float* bias, float eps, mlstm_norm norm,
                               int B, int NH, int T, int DV, void* h, void* hip_stream);

/*
 * The same output (Eq. 6 with the output gate of Eq. 9) in the token-major
 * layouts of a layer's projections, so that neither o~ nor the result needs a
 * head-major copy:
 *
 *   h_tilde [B, NH, T, DV] (dt)        the cell output, head-major
 *   o_pre   row (b, h, t) at element (b T + t) o_token_stride + h DV: the
 *           o~ columns of a token-major projection output (o_token_stride is
 *           its row length in elements, >= NH DV, a multiple of 4)
 *   y       [B, T, NH, DV] (dt)        token-major, the input layout of the
 *           output projection
 *
 * Same arithmetic, norms, limits and errors as mlstm_output_norm; y may not
 * overlap any input (MLSTM_ERR_ALIAS), and a bad o_token_stride is
 * MLSTM_ERR_BAD_SHAPE.
 */
mlstm_status mlstm_output_norm_tokens(const void* h_tilde, const void* o_pre, int64_t o_token_stride,
                                      mlstm_dtype dt, const float* weight, const float* bias, float eps,
                                      mlstm_norm norm, int B, int NH, int T, int DV, void* y,
                                      void* hip_stream);

/*
 * One decode step that returns the cell's hidden-state output instead of h~
 * (Sec. 2, Eqs. 2-5 for the step; Eq. 6 with the output gate of Eq. 9 for the
 * output; Sec. 3.1, "Fused Generation Kernels"):
 *
 *   h_row = sigmoid(o~_row) * (Norm(h~_row) * weight[head] + bias[head])
 *
 * with the state update and arguments of mlstm_step, and o~, weight, bias,
 * eps and norm as in mlstm_output_norm (o_pre [B, NH, DV] in dt).  When one
 * workgroup owns each sequence (enough sequences to fill the chip, e.g. a
 * decode batch of 256 x 8 heads) the norm runs on the h~ row in the step
 * kernel itself, from the unrounded fp32 h~, and h~ never goes to memory;
 * otherwise the step writes h~ into h and the output pass runs on it in place,
 * on the same stream.  Limits and state aliasing as mlstm_step, plus DV <=
 * 2048; h may not overlap o_pre, weight or bias (MLSTM_ERR_ALIAS), a bad eps
 * or norm is MLSTM_ERR_BAD_SHAPE and a NULL o_pre is MLSTM_ERR_NULL_PTR.
 */
mlstm_status mlstm_step_output(const void* q, const void* k, const void* v, mlstm_dtype dt,
                               const float* ipre, const float* fpre,
                               const float* C, const float* n, const float* m,
                               const void* o_pre, const float* weight, const float* bias, float eps,
                               mlstm_norm norm, int B, int NH, int DQK, int DV,
                               void* h, float* C_out, float* n_out, float* m_out, void* hip_stream);

/*
 * Gate pre-activations of an mLSTM layer, the inputs ipre and fpre of the two
 * cell entry points (Eq. 11: one input and one forget gate column per head,
 * each with a bias; Eq. 13: the soft-cap; App. B: the reset at document
 * borders of packed sequences).  For token (b, t) with x = x[b, t, :] and head h:
 *
 *   ipre[b, h, t] = softcap(x . w_t[h, :]      + bias[0, h])
 *   fpre[b, h, t] = softcap(x . w_t[NH + h, :] + bias[1, h]),  or -inf where
 *                   border[b, t] != 0 (a forget gate of exactly zero)
 *
 * with softcap(z) = cap * tanh(z / cap), or z itself when cap == 0.  The
 * products are bf16 with fp32 accumulation; the gates stay fp32.
 *
 *   x      [B, T, d] (dt, MLSTM_BF16 only)
 *   w_t    [2 NH, d] bf16: row h holds head h's input gate weights, row NH + h
 *          its forget gate weights (the transpose of a [d, 2 NH] projection)
 *   bias   [2, NH] fp32, or NULL (zero)
 *   border [B, T] uint8, or NULL (no document borders)
 *   ipre, fpre [B, NH, T] fp32 outputs (head-major: the cell's layout)
 *
 * cap must be finite and >= 0 (else MLSTM_ERR_BAD_SHAPE).  Built: d a
 * multiple of 128 and 2 NH <= 64 (else MLSTM_ERR_UNSUPPORTED).  B T == 0
 * launches nothing.  The outputs may not overlap each other or any input
 * (MLSTM_ERR_ALIAS).
 */
mlstm_status mlstm_gate_preact(const void* x, mlstm_dtype dt, const void* w_t, const float* bias, float cap,
                               const unsigned char* border, int B, int T, int d, int NH,
                               float* ipre, float* fpre, void* hip_stream);

/*
 * Backward pass of the cell for training (Sec. 2, "Training Mode"): the
 * gradients of a loss with respect to q, k, v, ipre and fpre, given its
 * gradient dh with respect to the outputs h~ of a forward call from the zero
 * initial state (C0, n0, m0 all NULL in mlstm_chunkwise_fwd).  It works on the
 * parallel form (Eq. 10): h~_t = N_t / max(|D_t|, 1) in unscaled units with
 * N_t, D_t sums over s <= t of exp(b_t - b_s + i~_s) (k_s . q^_t) (times v_s
 * for N), b the prefix sums of logsig(f~), every exponential evaluated
 * relative to the max state of Eq. 2.  Work is O(T^2 (DQK + DV)) per
 * sequence, in fp32.
 *
 *   q, k [B, NH, T, DQK], v [B, NH, T, DV] (dt)   ipre, fpre [B, NH, T] fp32
 *   dh [B, NH, T, DV] fp32
 *   dq, dk [B, NH, T, DQK], dv [B, NH, T, DV], dipre, dfpre [B, NH, T] fp32
 *   workspace: device scratch of at least mlstm_parallel_bwd_workspace_bytes
 *   bytes (else MLSTM_ERR_WORKSPACE); its contents on entry do not matter.
 *
 * fpre must not hold -inf (a document border): the parallel form's prefix
 * sums cannot restart there, and every gradient of that sequence would be
 * NaN.  The chunkwise backward takes borders.
 *
 * Built: DQK and DV multiples of 16, DQK <= 256, DV <= 512 (else
 * MLSTM_ERR_UNSUPPORTED).  T == 0 launches nothing.  No output may overlap
 * an input, another output or the workspace (MLSTM_ERR_ALIAS).
 */
size_t mlstm_parallel_bwd_workspace_bytes(int B, int NH, int T, int DV);
mlstm_status mlstm_parallel_bwd(const void* q, const void* k, const void* v, mlstm_dtype dt,
                                const float* ipre, const float* fpre, const float* dh,
                                int B, int NH, int T, int DQK, int DV,
                                float* dq, float* dk, float* dv, float* dipre, float* dfpre,
                                void* workspace, size_t workspace_bytes, void* hip_stream);

/*
 * Chunkwise backward pass of the cell for training (Sec. 2, "Training Mode";
 * App. D.2 counts it as twice the forward's work): the gradients of a loss
 * with respect to q, k, v, ipre, fpre and the initial state, given its
 * gradient dh with respect to the outputs h~ of mlstm_chunkwise_fwd on the same
 * inputs.  The entry state of every 64-token chunk is recomputed (the forward's
 * segment passes), then per chunk the intra-chunk terms, the terms through the
 * entry state, and the gradient of the state (C, n) carried backwards through
 * the chunk recurrence of App. D.1; document borders (fpre = -inf, App. B)
 * restart that recurrence as in the forward.  The forward's output is not
 * needed: dh . h~ is formed from the recomputed numerator in fp32.  Products
 * run on bf16 MFMA with fp32 accumulation; the recomputed states enter them
 * as bf16 hi + lo pairs, the carried state gradients (accumulated in fp32)
 * rounded once to bf16.  No float atomics: the
 * result is deterministic.
 *
 *   q, k [B, NH, T, DQK], v [B, NH, T, DV] (dt)   ipre, fpre [B, NH, T] fp32
 *   C0 [B, NH, DQK, DV], n0 [B, NH, DQK], m0 [B, NH] fp32: the forward's
 *        initial state, or all NULL for the zero state (m0 = 0)
 *   dh [B, NH, T, DV] (dt): the gradient of the loss with respect to h~
 *   dq, dk [B, NH, T, DQK], dv [B, NH, T, DV], dipre, dfpre [B, NH, T] fp32
 *   dC0 [B, NH, DQK, DV], dn0 [B, NH, DQK], dm0 [B, NH] fp32: the gradients
 *        of the initial state (also of the zero state), or all NULL
 *   workspace: device scratch of at least mlstm_chunkwise_bwd_workspace_bytes
 *   bytes (else MLSTM_ERR_WORKSPACE); its contents on entry do not matter.
 *   About 1 MiB per 64 tokens per (batch, head) plus 36 bytes per token.
 *
 * The loss is taken not to depend on the final state (CT, nT, mT).  dfpre is
 * zero where fpre = -inf.  A partially given initial state or gradient
 * triple is MLSTM_ERR_NULL_PTR.
 *
 * Built: dt = MLSTM_BF16, DQK = 256, DV = 512, L = 64 (the backward's own
 * chunk length, independent of the forward call's), T DV 2 < 2^31 and
 * B NH <= 65535 (else MLSTM_ERR_UNSUPPORTED).  T == 0 launches at most a fill
 * of zeros into dC0, dn0, dm0.  No output may overlap an input, another
 * output or the workspace (MLSTM_ERR_ALIAS).
 */
size_t mlstm_chunkwise_bwd_workspace_bytes(int B, int NH, int T, int DQK, int DV, int L, mlstm_dtype dt);
mlstm_status mlstm_chunkwise_bwd(const void* q, const void* k, const void* v, mlstm_dtype dt,
                                 const float* ipre, const float* fpre,
                                 const float* C0, const float* n0, const float* m0,
                                 int B, int NH, int T, int DQK, int DV, int L,
                                 const void* dh,
                                 float* dq, float* dk, float* dv, float* dipre, float* dfpre,
                                 float* dC0, float* dn0, float* dm0,
                                 void* workspace, size_t workspace_bytes, void* hip_stream);

/* Static, human-readable name of a status code. */
const char* mlstm_status_string(mlstm_status s);

/* Library version: major * 10000 + minor * 100 + patch. */
int mlstm_version(void);

/*
 * Debug builds only (compiled with -DMLSTM_DEBUG, libmlstm_debug.so): the
 * kernels check their computed indices (state slots, LDS tiles, sequence and
 * row offsets) against the extents of what they address, and a failed check
 * sets a bit instead of faulting.  This call returns the bits set since the
 * previous call and clears them: 1 chunkwise prefill (bf16 MFMA, including the
 * segment passes), 2 chunkwise prefill (fp32), 4 decode step, 8 output norm,
 * 16 gate pre-activations, 32 chunkwise backward, 64 parallel-form backward.
 * 0 means no check failed.  The caller synchronises the device first (the
 * words are read with a synchronous copy on the default stream).  A library
 * built without the checks returns MLSTM_DEBUG_NOT_BUILT.
 */
#define MLSTM_DEBUG_NOT_BUILT 0x80000000u
unsigned int mlstm_debug_flags(void);

#ifdef __cplusplus
}
#endif

#endif /* LIBMLSTM_MLSTM_H */
