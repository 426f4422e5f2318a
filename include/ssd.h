/*
 * ssd.h -- C ABI of the MI355X (gfx950) SSD layer: forward, decode step,
 * block steps, span state passing, and gradients.
 *
 * Computes y = SSM(A, B, C)(x) for the scalar-transition selective SSM of the
 * SSD layer (Section 5 of "Transformers are SSMs"), by the chunked block
 * decomposition of its 1-semiseparable matrix (Section 6): per chunk of Q
 * tokens, the diagonal block in its quadratic (masked-attention) form, the
 * chunk-final states (right factors), a scan of the states over chunks (centre
 * factors, the scalar SSM scan of Appendix B) and the state-to-output term
 * (left factors).  The problem statement follows the paper's
 *   Y, final_state = ssd(X, A, B, C, block_len, initial_states)
 * with discretisation exp(dt*A) / dt*x, a per-head skip D, grouped B/C heads
 * (Section 7) and packed variable-length rows (Section 8.3) added.
 *
 * Per head h (group g = h / (H/G)), with A_h = -exp(A_log[h]) and state S (P x N):
 *     S_t = exp(dt_t A_h) S_{t-1} + (dt_t x_t) B_t^T,    y_t = S_t C_t + D_h x_t,
 * S_{-1} = initial state (zero when none).  With seq_idx the state entering
 * the first token of every sequence is that sequence's initial state.
 *
 * Layouts (row-major, contiguous, element strides implied by the shape):
 *   x, y            (batch, seqlen, nheads, headdim)      dtype
 *   dt              (batch, seqlen, nheads)               dtype, already positive
 *                                                         (softplus applied by the caller)
 *   A_log           (nheads)                              float32
 *   B, C            (batch, seqlen, ngroups, dstate)      dtype
 *   D               (nheads)                              float32, may be NULL (= 0)
 *   seq_idx         (1, seqlen)                           int32, may be NULL
 *   initial_states  (batch, nheads, headdim, dstate)      float32, may be NULL (= 0);
 *                   (nseq, nheads, headdim, dstate) when seq_idx is given
 *   final_states    same shape as initial_states          float32, may be NULL (not written)
 * "dtype" is SSD_DTYPE_F32 (float) or SSD_DTYPE_BF16 (bfloat16 bits).  All
 * arithmetic accumulates in float32; y is rounded to dtype (nearest even).
 *
 * seq_idx contract (not checked on the device): non-decreasing, starting at 0,
 * consecutive ids, last value nseq - 1; batch must be 1.  Ids that break it
 * give unspecified values in y and final_states but no access outside the
 * buffers described here.
 *
 * Ownership: every pointer is device memory owned by the caller; the library
 * allocates nothing on the call path.  `workspace` is caller-provided device
 * memory of at least ssd_workspace_bytes() bytes; its contents on entry do not
 * matter, and on exit only its first int is specified: the status word that
 * ssd_workspace_status() reads.  The call is asynchronous on `stream`
 * (a hipStream_t; NULL = the null stream); it keeps no global mutable state
 * (apart from the test settings of ssd_set_tuning), so concurrent calls with
 * distinct workspaces are safe.  Results are
 * deterministic (no floating-point atomics).
 *
 * Errors: functions return SSD_OK (0) or a negative ssd_status.  On error no
 * device work has been enqueued, except SSD_ERR_LAUNCH (a launch failed after
 * earlier kernels of the call were enqueued).
 */
#ifndef SSD_H_
#define SSD_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SSD_DTYPE_F32 = 0,
    SSD_DTYPE_BF16 = 1
} ssd_dtype;

typedef enum {
    SSD_OK = 0,
    SSD_ERR_NULL_ARG = -1,         /* a required pointer is NULL                     */
    SSD_ERR_BAD_SHAPE = -2,        /* a dimension < 1, or nheads % ngroups != 0,
                                      or nseq < 1 with seq_idx                        */
    SSD_ERR_BAD_CHUNK = -3,        /* chunk_size not in {32, 64, 128, 256}           */
    SSD_ERR_BAD_DTYPE = -4,        /* dtype not an ssd_dtype                         */
    SSD_ERR_UNSUPPORTED_DIMS = -5, /* headdim not a multiple of 16 in [16, 128], or
                                      dstate not a multiple of 16 in [16, 256]       */
    SSD_ERR_SEQIDX_BATCH = -6,     /* seq_idx given with batch != 1                  */
    SSD_ERR_WORKSPACE = -7,        /* workspace NULL or smaller than required        */
    SSD_ERR_LAUNCH = -8,           /* a kernel launch failed                         */
    SSD_ERR_TOO_LARGE = -9,        /* a tensor exceeds the supported index range     */
    SSD_ERR_BAD_OPTION = -10,      /* an ssd_block_opts field out of range, or an
                                      unknown ssd_set_tuning name or value           */
    SSD_ERR_STATE_TIMEOUT = -11,   /* reported by ssd_workspace_status only: a chunk
                                      kernel's wait for the state of the chunk before
                                      it gave up; that call's y and final_states are
                                      wrong                                          */
    SSD_ERR_SCRATCH_TOO_SMALL = -12 /* ssd_forward_noalloc: the problem needs more
                                      workspace than SSD_NOALLOC_SCRATCH_BYTES       */
} ssd_status;

typedef struct {
    int64_t batch;       /* b                                        */
    int64_t seqlen;      /* T (any length >= 1; the last chunk may be partial) */
    int64_t nheads;      /* H                                        */
    int64_t headdim;     /* P                                        */
    int64_t dstate;      /* N                                        */
    int64_t ngroups;     /* G, divides H                             */
    int64_t chunk_size;  /* Q, the block length of the decomposition */
    int64_t nseq;        /* number of sequences; read only when seq_idx != NULL */
    int32_t dtype;       /* ssd_dtype of x, dt, B, C, y              */
} ssd_problem;

/* Workspace size in bytes for `prob` (Section 6 intermediates: chunk cumsums,
 * chunk states, the packed row's chunk table).  The size covers calls with and
 * without seq_idx; with batch 1 it depends on prob->nseq, so size it with the
 * nseq the call will pass.  It is the size of the kernels the call will run:
 * at the shapes of the fused kernels (bf16, headdim 64, dstate 64/128/256,
 * chunk 256) a fraction of the general kernels' (which keep every chunk
 * state), so a test setting that forces the general path (ssd_set_tuning)
 * must be made before the size is asked.  A workspace too small for the path
 * a call takes fails with SSD_ERR_WORKSPACE, never overruns.  Returns SSD_OK
 * and writes *bytes, or a validation error. */
int ssd_workspace_bytes(const ssd_problem* prob, size_t* bytes);

/* The SSD forward (Section 6 algorithm; definition above).  `D`,
 * `initial_states`, `seq_idx` and `final_states` may be NULL.  `stream` is a
 * hipStream_t. */
int ssd_forward(const ssd_problem* prob,
                const void* x, const void* dt, const float* A_log,
                const void* B, const void* C, const float* D,
                const float* initial_states, const int32_t* seq_idx,
                void* y, float* final_states,
                void* workspace, size_t workspace_bytes, void* stream);

/* ssd_forward, plus two hipEvent_t (either may be NULL) recorded on `stream`
 * immediately before and immediately after the launch of the dominant kernel
 * of the call (the chunk kernel, which evaluates the diagonal blocks, the
 * chunk states, the state passing and the state-to-output term), so that a
 * profiler or benchmark can time that kernel alone with hipEventElapsedTime.
 * Results, errors and ownership are those of ssd_forward; the events are
 * owned by the caller and must have been created on the stream's device. */
int ssd_forward_timed(const ssd_problem* prob,
                      const void* x, const void* dt, const float* A_log,
                      const void* B, const void* C, const float* D,
                      const float* initial_states, const int32_t* seq_idx,
                      void* y, float* final_states,
                      void* workspace, size_t workspace_bytes, void* stream,
                      void* event_begin, void* event_end);

/* ssd_forward for one packed row (batch 1) of nseq sequences given by host
 * offsets instead of the device seq_idx: seq_starts (host memory) holds nseq +
 * 1 token offsets, seq_starts[0] = 0, strictly increasing, seq_starts[nseq] =
 * seqlen (else SSD_ERR_BAD_SHAPE); token t belongs to sequence s when
 * seq_starts[s] <= t < seq_starts[s + 1].  At the fused kernels' shapes and
 * up to 511 sequences the offsets are handed to the device by value and the
 * row runs as one launch, as ssd_forward with seq_idx does; otherwise each
 * sequence runs as a problem of its own on its slice of the packed tensors.
 * Either way the result equals ssd_forward with the matching seq_idx.  initial_states / final_states are (nseq, nheads, headdim, dstate)
 * (either may be NULL).  Workspace: ssd_forward_varlen_workspace_bytes().
 * Errors as for ssd_forward. */
int ssd_forward_varlen_workspace_bytes(const ssd_problem* prob, const int64_t* seq_starts, size_t* bytes);

int ssd_forward_varlen(const ssd_problem* prob, const int64_t* seq_starts,
                       const void* x, const void* dt, const float* A_log,
                       const void* B, const void* C, const float* D,
                       const float* initial_states, void* y, float* final_states,
                       void* workspace, size_t workspace_bytes, void* stream);

/* One decode step (one new token per sequence) of the same layer, in the
 * recurrent form of eq. s6 with scalar A (the per-token inference cost of
 * Section 6.3): per batch row and head h (group g = h / (H/G)),
 *     S <- exp(dt A_h) S + (dt x) B^T,    y = S C + D_h x.
 * `prob` gives batch, nheads, headdim, dstate, ngroups and dtype (seqlen,
 * chunk_size and nseq are ignored; the limits on headdim and dstate are those
 * of ssd_forward).  Layouts (row-major, contiguous):
 *   x, y    (batch, nheads, headdim)            dtype
 *   dt      (batch, nheads)                     dtype, already positive
 *   A_log   (nheads) float32;  D (nheads) float32, may be NULL (= 0)
 *   B, C    (batch, ngroups, dstate)            dtype
 *   state   (batch, nheads, headdim, dstate)    float32, read and updated in
 *           place, 16-byte aligned (else SSD_ERR_UNSUPPORTED_DIMS)
 * A state carried through a sequence of decode steps equals the final state
 * of ssd_forward over the same tokens.  Asynchronous on `stream`; needs no
 * workspace; errors as for ssd_forward. */
int ssd_decode_step(const ssd_problem* prob,
                    const void* x, const void* dt, const float* A_log,
                    const void* B, const void* C, const float* D,
                    float* state, void* y, void* stream);

/* Steps of the Mamba-2 block fused on either side of the layer.
 *
 * Before the layer, the discretisation parameter (left to the caller by the
 * paper, which has Delta come out of the block's input projection, Section 7):
 *     dt = min(max(softplus(dt_in + dt_bias), dt_min), dt_max)   (dt_softplus != 0)
 *     dt = min(max(dt_in + dt_bias, dt_min), dt_max)             (dt_softplus == 0)
 * with softplus(v) = log(1 + e^v) and dt_bias NULL meaning 0.
 * After the layer (y including D x), the gate and the normalisation of the
 * block equations of Section 8.1 (the norm after the gate, as in Section 7.1):
 *     y = y * z * sigmoid(z)                                     (z != NULL)
 *     y = y / sqrt(mean over its group of y^2 + norm_eps) * norm_weight
 *                                                      (norm_group_size > 0)
 * where a token's groups are consecutive runs of norm_group_size channels of
 * its nheads * headdim channel row (head-major).  A zero-initialised struct
 * with dt_max = INFINITY is the plain layer.
 *
 * Limits (else SSD_ERR_BAD_OPTION): 0 <= dt_min <= dt_max (dt_max may be
 * INFINITY); norm_group_size 0 or a multiple of headdim that divides
 * nheads * headdim; norm_eps >= 0 and finite. */
typedef struct {
    const float* dt_bias;      /* (nheads) float32, or NULL                          */
    int32_t dt_softplus;       /* nonzero: softplus after the bias                   */
    float dt_min;              /* clamp of dt (0 = none from below)                  */
    float dt_max;              /* clamp of dt (INFINITY = none from above)           */
    const void* z;             /* (batch, seqlen, nheads, headdim) dtype, or NULL    */
    const float* norm_weight;  /* (nheads * headdim) float32, or NULL (= 1)          */
    int64_t norm_group_size;   /* channels per normalisation group, 0 = no norm      */
    float norm_eps;            /* added to each group's mean square                  */
} ssd_block_opts;

/* Workspace size for ssd_forward_block (at least ssd_workspace_bytes). */
int ssd_block_workspace_bytes(const ssd_problem* prob, const ssd_block_opts* opts, size_t* bytes);

/* The layer with the block steps above around it.  Arguments, layouts,
 * ownership and errors as for ssd_forward, except that `dt` holds dt_in (any
 * sign when dt_softplus != 0) and `opts` (host memory, read during the call;
 * its device pointers must stay valid until the work completes) selects the
 * steps; y receives the block's output.  On the Mamba-2 layer shapes of the
 * fused path the dt step runs inside the chunk kernel and the gate (and a
 * normalisation of one head per group) inside its output stage; larger
 * groups are normalised by one more pass over y. */
int ssd_forward_block(const ssd_problem* prob, const ssd_block_opts* opts,
                      const void* x, const void* dt, const float* A_log,
                      const void* B, const void* C, const float* D,
                      const float* initial_states, const int32_t* seq_idx,
                      void* y, float* final_states,
                      void* workspace, size_t workspace_bytes, void* stream);

/* ssd_forward_block with the two events of ssd_forward_timed around its
 * chunk kernel. */
int ssd_forward_block_timed(const ssd_problem* prob, const ssd_block_opts* opts,
                            const void* x, const void* dt, const float* A_log,
                            const void* B, const void* C, const float* D,
                            const float* initial_states, const int32_t* seq_idx,
                            void* y, float* final_states,
                            void* workspace, size_t workspace_bytes, void* stream,
                            void* event_begin, void* event_end);

/* Sequence spans (context parallelism, Section 8.2).  A sequence cut into
 * consecutive spans (one per GPU, say) is computed span by span from zero
 * states with ssd_forward, giving each span's outputs and final state; then
 *   ssd_span_decay     the span's total decay exp(A_h sum_t dt_t), per
 *                      (batch, head);
 *   ssd_span_combine   from every span's (decay, final state) pair, the state
 *                      entering every span and the final state of the whole
 *                      sequence: the exclusive scan under the scalar-SSM
 *                      operator of Appendix B, (a, h) then (a', h') =
 *                      (a a', a' h + h');
 *   ssd_span_correct   y_t += exp(A_h sum_{s<=t} dt_s) (h_in C_t) over the
 *                      span (sums from its first token), which turns the
 *                      zero-state outputs into those of the whole sequence.
 * Across GPUs the (decay, final state) pairs are exchanged between the first
 * and the second step (an all-gather); that exchange is not part of this
 * library.  `prob` describes one span (seqlen = its length); chunk_size and
 * nseq are ignored; packed rows are not supported.  Layouts: dt (batch,
 * seqlen, nheads) dtype, already positive; A_log (nheads) float32; decay
 * (batch, nheads) float32; states (batch, nheads, headdim, dstate) float32,
 * 16-byte aligned; for ssd_span_combine, decay (nspans, batch, nheads) and
 * local_final / entering (nspans, batch, nheads, headdim, dstate), span
 * order; initial_states may be NULL (zero), final_states may be NULL; C
 * (batch, seqlen, ngroups, dstate) dtype; y (batch, seqlen, nheads, headdim)
 * dtype, updated in place (rounded to dtype).  bf16 products run on the
 * matrix cores with the entering state rounded to bf16.  Errors as for
 * ssd_forward. */
int ssd_span_decay(const ssd_problem* prob, const void* dt, const float* A_log, float* decay, void* stream);

int ssd_span_combine(int64_t nspans, const ssd_problem* prob, const float* decay,
                     const float* local_final, const float* initial_states, float* entering,
                     float* final_states, void* stream);

/* Workspace of ssd_span_correct (per-chunk dt sums). */
int ssd_span_correct_workspace_bytes(const ssd_problem* prob, size_t* bytes);

int ssd_span_correct(const ssd_problem* prob, const void* dt, const float* A_log, const void* C,
                     const float* entering, void* y, void* workspace, size_t workspace_bytes,
                     void* stream);

/* ---- Gradients (training; the cost of Section 6.3) --------------------------
 *
 * ssd_backward: the gradients of a scalar loss L with respect to every input
 * of ssd_forward, given dy = dL/dy and dfinal_states = dL/d(final_states)
 * (NULL = 0), for the layer defined at the top of this header without packed
 * rows (no seq_idx).  The paper states no backward algorithm; this is the
 * adjoint of the recurrence, evaluated chunk by chunk like the forward of
 * Section 6 (chunk-local terms, then a scan over chunks in each direction).
 *   Inputs: prob, x, dt, A_log, B, C, D (may be NULL = 0), initial_states
 *           (may be NULL = 0) exactly as given to ssd_forward, and dy (layout
 *           and dtype of y).  prob->chunk_size and prob->nseq are not used
 *           (the backward has its own chunking; the result does not depend on it).
 *   Outputs (every one overwritten):
 *     dx  (batch, seqlen, nheads, headdim)   dtype
 *     ddt (batch, seqlen, nheads)            dtype (gradient of dt as given,
 *                                            i.e. after any softplus)
 *     dA_log (nheads)                        float32 (through A = -exp(A_log))
 *     dB, dC (batch, seqlen, ngroups, dstate) dtype (summed over a group's heads)
 *     dD (nheads)                            float32; not written when D or dD is NULL
 *     dinitial_states (batch, nheads, headdim, dstate) float32; may be NULL
 * x, B, C, dy, dx, initial_states, dfinal_states and dinitial_states must be
 * 16-byte aligned (else SSD_ERR_UNSUPPORTED_DIMS).  Arithmetic in float32; dtype outputs are
 * rounded to nearest even.  Workspace: ssd_backward_workspace_bytes() bytes of
 * device memory (it holds a state per 64 tokens and head twice in bf16
 * for bf16 with headdim 64 and dstate 64 or 128, which run on the matrix
 * cores; otherwise one per 32 tokens and head twice in float32).  Ownership,
 * asynchrony, determinism and errors as for ssd_forward. */
int ssd_backward_workspace_bytes(const ssd_problem* prob, size_t* bytes);

int ssd_backward(const ssd_problem* prob,
                 const void* x, const void* dt, const float* A_log,
                 const void* B, const void* C, const float* D,
                 const float* initial_states,
                 const void* dy, const float* dfinal_states,
                 void* dx, void* ddt, float* dA_log, void* dB, void* dC,
                 float* dD, float* dinitial_states,
                 void* workspace, size_t workspace_bytes, void* stream);

/* ssd_backward, plus two hipEvent_t (either may be NULL) recorded right before
 * and right after the launch of its dominant kernel (the per-chunk gradient
 * kernel), as in ssd_forward_timed. */
int ssd_backward_timed(const ssd_problem* prob,
                       const void* x, const void* dt, const float* A_log,
                       const void* B, const void* C, const float* D,
                       const float* initial_states,
                       const void* dy, const float* dfinal_states,
                       void* dx, void* ddt, float* dA_log, void* dB, void* dC,
                       float* dD, float* dinitial_states,
                       void* workspace, size_t workspace_bytes, void* stream,
                       void* event_begin, void* event_end);

/* ssd_backward_varlen: ssd_backward for one packed row of nseq sequences
 * (Section 8.3; batch must be 1, else SSD_ERR_SEQIDX_BATCH).  seq_starts is
 * host memory: nseq + 1 token offsets, seq_starts[0] = 0, strictly
 * increasing, seq_starts[nseq] = seqlen (else SSD_ERR_BAD_SHAPE); token t
 * belongs to sequence s when seq_starts[s] <= t < seq_starts[s + 1] (the
 * seq_idx of ssd_forward).  initial_states, dfinal_states and
 * dinitial_states are (nseq, nheads, headdim, dstate).  The sequences do not
 * interact.  On the matrix-core path (bf16, headdim 64, dstate 64 or 128) and
 * up to 511 sequences the offsets are handed to the device by value and the
 * row runs as one backward over per-sequence chunks; otherwise each sequence
 * runs as a problem of its own on its slice of the packed tensors and dA_log
 * and dD are summed over the sequences in order.
 * Workspace: ssd_backward_varlen_workspace_bytes() bytes.  Otherwise as
 * ssd_backward (every check is made before any work is enqueued). */
int ssd_backward_varlen_workspace_bytes(const ssd_problem* prob, const int64_t* seq_starts, size_t* bytes);

int ssd_backward_varlen(const ssd_problem* prob, const int64_t* seq_starts,
                        const void* x, const void* dt, const float* A_log,
                        const void* B, const void* C, const float* D,
                        const float* initial_states,
                        const void* dy, const float* dfinal_states,
                        void* dx, void* ddt, float* dA_log, void* dB, void* dC,
                        float* dD, float* dinitial_states,
                        void* workspace, size_t workspace_bytes, void* stream);

/* ssd_backward_block: the gradients of ssd_forward_block (same `prob`,
 * `opts` and inputs; no packed rows), given dout = dL/d(block output) and
 * dfinal_states (NULL = 0).  The paper gives no backward; this is the chain
 * rule through the normalisation, the gate (Section 8.1), the layer
 * (ssd_backward) and the dt step, with the layer's output recomputed from the
 * inputs.  What the steps exchange with the layer -- dt after the dt step, the
 * layer's output, its gradient and the layer's dt gradient -- stays float32
 * (as in ssd_forward_block), with bf16 activations too: only inputs and
 * outputs have the activation dtype, and the result is the gradient of
 * ssd_forward_block itself.  (bf16 at headdim 64 and dstate 64 or 128 runs on
 * the matrix cores; other bf16 shapes run in float32 on widened copies of the
 * activations.)  Outputs as for ssd_backward with `ddt` the gradient of `dt`
 * as given (before bias, softplus and clamp), plus
 *   ddt_bias      (nheads) float32, written when opts->dt_bias (may be NULL)
 *   dz            like y, dtype; required when opts->z
 *   dnorm_weight  (nheads * headdim) float32, written when the normalisation
 *                 and its weight are on (may be NULL)
 * x, B, C, dout, dx, dz and the state arrays must be 16-byte aligned (else
 * SSD_ERR_UNSUPPORTED_DIMS).  Workspace: ssd_backward_block_workspace_bytes()
 * bytes.  Ownership, asynchrony, determinism and errors as for ssd_forward. */
int ssd_backward_block_workspace_bytes(const ssd_problem* prob, const ssd_block_opts* opts, size_t* bytes);

int ssd_backward_block(const ssd_problem* prob, const ssd_block_opts* opts,
                       const void* x, const void* dt, const float* A_log,
                       const void* B, const void* C, const float* D,
                       const float* initial_states,
                       const void* dout, const float* dfinal_states,
                       void* dx, void* ddt, float* dA_log, void* dB, void* dC,
                       float* dD, float* dinitial_states,
                       float* ddt_bias, void* dz, float* dnorm_weight,
                       void* workspace, size_t workspace_bytes, void* stream);

/* Status of the state passing of the last call that used `workspace`.
 *
 * On the fused path the chunk kernel passes each chunk's final state to the
 * next chunk's workgroup through device memory (the centre factors of
 * Section 6, as the sequential scan of Appendix B): a workgroup waits for the
 * state of the chunk before it.  That wait is bounded (2^22 polls with a short
 * sleep in between, far beyond any normal wait) so that a fault can never hang
 * the GPU; when it gives up, the kernel sets the status word, the first int of
 * the workspace, and finishes with a wrong entering state.  Every call of
 * ssd_forward, ssd_forward_timed, ssd_forward_block(_timed),
 * ssd_forward_varlen and ssd_backward_block writes that word (0 when no wait
 * gave up); the general path, which has no such wait, writes 0.
 *
 * ssd_workspace_status waits for `stream` (a hipStream_t) to finish, then
 * reads the word: SSD_OK, SSD_ERR_STATE_TIMEOUT, SSD_ERR_NULL_ARG (workspace
 * NULL) or SSD_ERR_LAUNCH (the synchronisation or the read failed).  After any
 * other call on the workspace the result is unspecified. */
int ssd_workspace_status(const void* workspace, void* stream);

/* Testing and measurement hook; normal use never needs it.  Overrides one of
 * the library's internal choices for every later call in this process, until
 * it is set back to 0 (each choice's default: the library decides).  The
 * results stay within the stated tolerances whatever the setting; only the
 * kernels and launch shapes that compute them change.
 *   "force_general_path"   1: every call takes the general kernels (one
 *                          launch per step of Section 6), also where the
 *                          fused or matrix-core kernels apply
 *   "heads_per_item"       k >= 1: heads per work item of the fused chunk
 *                          kernel (ignored unless k divides nheads/ngroups)
 *   "early_state_flag"     1: a chunk's state flag is set after its output
 *                          stage, 2: right after its state is stored
 *   "max_workgroups"       k >= 1: at most k persistent workgroups of the
 *                          fused chunk kernel
 *   "separate_block_post"  1: the block's gate and normalisation always run
 *                          as their own pass over y
 *   "bwd_heads_per_slice"  k >= 1: heads per workgroup of the backward's
 *                          per-chunk gradient kernel
 *   "varlen_per_sequence"  1: ssd_forward_varlen and ssd_backward_varlen run
 *                          one problem per sequence
 *   "state_wait_limit"     k >= 1: polls before a state wait gives up (see
 *                          ssd_workspace_status; 1 gives up at the first
 *                          poll that finds the state missing)
 *   "fused_right_factor"   1: the fused chunk kernel computes the right
 *                          factor in a pass of its own, 2: in the diagonal
 *                          block's pass (plain rows with the late state flag;
 *                          elsewhere 2 acts as 1)
 *   "packed_order"         1: the fused chunk kernel takes a packed row's
 *                          chunks in token order, 2: by their index within
 *                          their sequence (every sequence's first chunk,
 *                          then every second chunk, ...)
 * Returns SSD_OK, SSD_ERR_NULL_ARG, or SSD_ERR_BAD_OPTION (unknown name, or a
 * value out of range).  The settings are process-wide and not ordered with
 * calls made concurrently on other host threads. */
int ssd_set_tuning(const char* name, int64_t value);

/* For callers that cannot allocate device memory -- code under HIP graph
 * capture, serving loops that must not call hipMalloc, harnesses that forbid
 * it: ssd_forward without a workspace argument.  Its workspace is a fixed
 * device array of SSD_NOALLOC_SCRATCH_BYTES inside the library (one per GPU
 * it runs on, held until the process ends); the call itself allocates nothing
 * (no hipMalloc, hipFree or allocating library routine).  Problems whose
 * ssd_workspace_bytes() exceed that size return SSD_ERR_SCRATCH_TOO_SMALL
 * before anything is enqueued (the 2.7B and 130M layer shapes need about 35
 * and 27 MB).  Every call on one GPU shares that GPU's array: calls that
 * overlap in time on one GPU (different streams, or host threads) race and
 * give wrong results; calls in order on one stream are safe (each call's
 * kernels reset what must start at zero).  `status` (device memory, may be
 * NULL) receives, when the call's work completes, 0 or -- when a chunk's wait
 * for the state before it gave up (see ssd_workspace_status) -- a nonzero
 * value; with NULL that report is lost.  Everything else as ssd_forward. */
#define SSD_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

int ssd_forward_noalloc(const ssd_problem* prob,
                        const void* x, const void* dt, const float* A_log,
                        const void* B, const void* C, const float* D,
                        const float* initial_states, const int32_t* seq_idx,
                        void* y, float* final_states, int32_t* status, void* stream);

/* Static, NUL-terminated description of a status code. */
const char* ssd_error_string(int code);

#ifdef __cplusplus
}
#endif

#endif /* SSD_H_ */
