/*
 * solo_readout.h -- C ABI of the SOLO shared-readout local loss on MI355X (gfx950).
 *
 * The operation (the paper: Section 3.2 "SOLO: local learning with a shared
 * readout", Eq. 2 and Eq. 3; Appendix A, Algorithm 1, the readout lines of one
 * SOLO step; Appendix C: a head ends in an RMSNorm with an element-wise gain):
 * every module k in [0, K) sends its hidden states h_k through RMSNorm(gain)
 * and the shared read-only copy of the final module's readout W (V x d) into
 * a softmax cross-entropy over the full vocabulary, averaged over the module's
 * T tokens (temperature 1, no bias):
 *
 *     r_t    = 1 / sqrt(mean_j h_tj^2 + eps),   n_t = r_t h_t,   hhat_t = gain * n_t
 *     z_tv   = <W_v, hhat_t>                                      (Eq. 2)
 *     loss_k = (1/T) sum_t ( log sum_v exp z_tv  -  z_{t, y_t} )
 *
 * and returns, per module, d loss_k / d h_k only (the residual goes back
 * through the readout, Eq. 3, then the RMSNorm backward).  The read-only
 * copies get no gradient; the final module (k = K-1) also returns the
 * gradients of its own trained readout W and gain (the FLOP table of the
 * paper's systems appendix: 2r per auxiliary readout, 3r for the terminal).
 *
 * solo_readout_general extends this to everything Algorithm 1 and Eq. 2 put
 * into a head's loss, and to the readout sources of the paper's variant
 * tables (Section 3.3, table of readout sources; Appendix D, table of readout
 * content and basis):
 *
 *     z_tv = tau_k <R_kv, g_k * n_t> + b_kv
 *
 * with a temperature tau_k and bias b_k per module (Alg. 1: the heads train
 * (phi_k, tau_k, b_k), the terminal trains (W, b)), a gain g_k per module or
 * one shared gain, and the heads' readout R_k (k < K-1) taken from W itself
 * (SOLO), one other matrix shared by the heads (SOLO's copy from an earlier
 * step when it is refreshed every S > 1 steps; RSHARE), one matrix per head
 * (RAND frozen, PRIV trained), or the shared matrix in a fixed orthogonal
 * basis per head, Wbar R_k (ROT: same content and range, another basis;
 * Appendix D).  The terminal always reads W.  solo_readout_exit_eval is the forward pass alone: every
 * exit's loss and top-1 prediction through its readout (early exit through
 * the shared readout, Section 4).
 *
 * All compute runs in hand-written HIP kernels on the caller's stream; the
 * T x V logit or probability matrix is never written to memory.
 */
#ifndef SOLO_READOUT_H
#define SOLO_READOUT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SOLO_READOUT_ABI_VERSION 3

/* Element type of h, gain, W, Wbar and dh.  Statistics, exponentials and
 * accumulation are fp32 in both cases; the bf16 path multiplies bf16
 * operands (rounded to nearest even) on the matrix cores. */
typedef enum {
    SOLO_BF16 = 0,
    SOLO_F32 = 1
} solo_dtype;

typedef enum {
    SOLO_OK = 0,
    SOLO_ERR_NULL = 1,      /* a required pointer is NULL                                  */
    SOLO_ERR_SHAPE = 2,     /* K, T or V < 1; d < 8, d % 8 != 0 or d > 4096; size overflow */
    SOLO_ERR_DTYPE = 3,     /* dtype is not a solo_dtype                                   */
    SOLO_ERR_ALIGN = 4,     /* a pointer violates the alignment stated below               */
    SOLO_ERR_WORKSPACE = 5, /* workspace_bytes below the size the workspace query returns  */
    SOLO_ERR_ARG = 6,       /* eps < 0 or not finite; a flag not 0 or 1; flags that do not
                               go together (see solo_readout_args)                       */
    SOLO_ERR_HIP = 7        /* a HIP runtime call or kernel launch failed                  */
} solo_status;

/* SOLO_READOUT_ABI_VERSION of the loaded library. */
int solo_readout_abi_version(void);

/* Static, NUL-terminated description of a status code (never NULL). */
const char* solo_status_string(int status);

/*
 * Bytes of device workspace one solo_readout_fwd_bwd call needs.  A function
 * of (K, T, d, V, dtype, final_module_dW) with no T*V term: per-token
 * statistics, per-tile partial sums of the gain gradient and, on the
 * matrix-core families, a bf16 copy of gain * h of the modules whose readout or
 * bias gradient is computed (T*d*2 bytes each, rounded up to 16 rows); on the
 * "mfma_wide" family also one tiled bf16 copy of W (V*d*2 bytes, V rounded up
 * to 16), and the same for each distinct heads' readout of the general
 * entry point.  Returns 0 for arguments that solo_readout_fwd_bwd would reject.
 */
size_t solo_readout_workspace_size(int K, int T, int d, int V, int dtype, int final_module_dW);

/*
 * Name of the kernel family one call with these sizes runs on:
 * "mfma" (bf16 matrix-core kernels: d a multiple of 256 up to 2048; tiles of
 * 64 rows up to d = 1024 and 32 above, twice that in the forward-only
 * passes), "mfma_wide" (bf16 matrix-core kernels, d = 2560; 16-row tiles, 48
 * in the forward-only passes) or
 * "valu" (fp32 vector-ALU kernels, used for SOLO_F32 and for every other bf16
 * width).  Returns "invalid" for arguments solo_readout_fwd_bwd would reject.
 */
const char* solo_readout_kernel_family(int K, int T, int d, int V, int dtype);

/*
 * Forward and local backward of the shared-readout loss for K modules.
 *
 * Sizes: K >= 1 modules, T >= 1 tokens per module, 8 <= d <= 4096 with
 * d % 8 == 0, V >= 1.  All arrays are dense row-major device memory
 * (hipMalloc or torch CUDA/HIP tensors), except where noted.
 *
 *   eps             RMSNorm epsilon, finite and >= 0.
 *   h               [K][T][d] dtype, 16-byte aligned.  Pre-norm hidden states.
 *   gain            [d] dtype, 16-byte aligned.  RMSNorm gain (shared, read-only
 *                   for modules 0..K-2, trained by module K-1).
 *   W               [V][d] dtype, 16-byte aligned.  Readout; the read-only copy
 *                   of every head and the trained readout of module K-1.
 *   targets         [K][T] int32, 4-byte aligned.  Next-token ids, each in [0, V).
 *                   An id outside [0, V) is not checked on the host; the
 *                   kernels never index out of bounds for it and report it
 *                   as a NaN row loss (and hence a NaN module loss).
 *   final_module_dW 1: also compute dW and dgain of module K-1; 0: all frozen.
 *   losses          [K] float, out.  Mean cross-entropy of each module.
 *   row_loss        [K][T] float, out, optional (NULL to skip).  Per-token
 *                   cross-entropy (losses[k] is its mean over t).
 *   dh              [K][T][d] dtype, out, 16-byte aligned.  d losses[k] / d h_k.
 *   dW              [V][d] float, out, 16-byte aligned; required iff
 *                   final_module_dW, ignored otherwise.  d losses[K-1] / d W.
 *   dgain           [d] float, out, 4-byte aligned; required iff final_module_dW.
 *                   d losses[K-1] / d gain.
 *   workspace       device scratch of at least solo_readout_workspace_size(...)
 *                   bytes, 256-byte aligned.  Owned by the caller; its
 *                   contents on entry do not matter and are clobbered.
 *   hip_stream      hipStream_t to enqueue on (NULL = default stream).
 *
 * Semantics: outputs are overwritten (never accumulated).  Inputs, outputs
 * and workspace must not overlap.  The call only enqueues work and returns;
 * outputs are valid once the stream has reached this point, and inputs must
 * stay unchanged until then.  The library allocates no memory, keeps no
 * pointer after returning and holds no global mutable state; concurrent
 * calls on different streams with different workspaces are safe.  Results are
 * bitwise reproducible for identical inputs (no floating-point atomics).
 *
 * Errors: every argument check runs on the host before any launch; on error
 * nothing is enqueued and no output is touched.  SOLO_ERR_HIP means a launch
 * failed (outputs then undefined).
 */
int solo_readout_fwd_bwd(int K, int T, int d, int V, int dtype, float eps,
                         const void* h, const void* gain, const void* W,
                         const int32_t* targets, int final_module_dW,
                         float* losses, float* row_loss, void* dh,
                         float* dW, float* dgain,
                         void* workspace, size_t workspace_bytes,
                         void* hip_stream);

/*
 * Stages of one call, in launch order (all on hip_stream).  Every stage
 * event is recorded: right after its stage's work, or right after the
 * previous event when the stage has no work in this call.
 */
#define SOLO_NUM_STAGES 6
/*   0  per-token inverse RMS of h (and the tiled readout copies; with rot, */
/*      the heads' rotated rows)                                             */
/*   1  local-loss pass (logits, online log-sum-exp, dh; all K), or the     */
/*      forward-only exit evaluation; with rot also the heads' gradient     */
/*      rotated back and their RMSNorm backward                              */
/*   2  per-module sums in fixed order: losses, temperature gradients        */
/*   3  readout-gradient pass (modules whose readout is trained), after the */
/*      gain-scaled copy of h the matrix-core gradient passes stream         */
/*   4  bias-gradient pass (modules whose bias but not readout is trained)   */
/*   5  gain gradients (fixed-order sum of per-tile partials)                */

/*
 * solo_readout_fwd_bwd, and for profiling: stage_events[i], if not NULL, is a
 * hipEvent_t recorded on hip_stream as stated above.  stage_events itself
 * may be NULL.  Same arguments, semantics and errors otherwise; a failed
 * event record returns SOLO_ERR_HIP.
 */
int solo_readout_fwd_bwd_profiled(int K, int T, int d, int V, int dtype, float eps,
                                  const void* h, const void* gain, const void* W,
                                  const int32_t* targets, int final_module_dW,
                                  float* losses, float* row_loss, void* dh,
                                  float* dW, float* dgain,
                                  void* workspace, size_t workspace_bytes,
                                  void* hip_stream, void* const* stage_events);

/*
 * solo_readout_fwd_bwd without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  The workspace is a static device array
 * inside the library, one per GPU, of solo_readout_scratch_limit() bytes
 * (128 MiB), held from the first call on a device until the process ends.
 * Same arguments (minus workspace), kernels, semantics and results as
 * solo_readout_fwd_bwd, on the current device (which must own hip_stream).
 * Errors: as solo_readout_fwd_bwd; SOLO_ERR_WORKSPACE when the call needs
 * more workspace than the limit (solo_readout_workspace_size tells).  The
 * function calls no allocating routine.  Every call on one GPU shares that
 * GPU's scratch: calls that overlap on one GPU (different streams, or
 * threads) race and must be serialised by the caller; one stream in order is
 * safe.  Nothing in the scratch needs to start at zero.
 */
size_t solo_readout_scratch_limit(void);
int solo_readout_fwd_bwd_noalloc(int K, int T, int d, int V, int dtype, float eps,
                                 const void* h, const void* gain, const void* W,
                                 const int32_t* targets, int final_module_dW,
                                 float* losses, float* row_loss, void* dh,
                                 float* dW, float* dgain, void* hip_stream);

/*
 * Arguments of solo_readout_general and solo_readout_exit_eval.  Zero-fill
 * the struct, then set what the call uses; NULL pointers and 0 flags mean
 * "absent".  Sizes, dtype, eps, h, targets, losses, row_loss, workspace and
 * the stream are as in solo_readout_fwd_bwd.
 *
 * Inputs:
 *   gain            [d] dtype (gain_per_module = 0: one gain, trained by the
 *                   terminal only, read-only for the heads) or [K][d]
 *                   (gain_per_module = 1: g_k owned by module k, every module
 *                   gets its gradient); 16-byte aligned.
 *   W               [V][d] dtype: the terminal readout (module K-1), 16-byte aligned.
 *   Wbar            the heads' readout (modules 0..K-2), 16-byte aligned:
 *                   NULL -> W itself (SOLO with the copy refreshed every step);
 *                   [V][d] dtype with readout_per_head = 0 -> one matrix shared
 *                   by the heads; [K-1][V][d] dtype with readout_per_head = 1
 *                   -> one matrix per head.
 *   tau             [K] float or NULL (every tau_k = 1; the paper's terminal
 *                   has none, so pass tau[K-1] = 1 for that).  Not checked for
 *                   finiteness.  4-byte aligned.
 *   bias            [K][V] float or NULL (no bias).  4-byte aligned.
 *   rot             [K-1][d][d] dtype or NULL, 16-byte aligned (ROT): head k
 *                   reads Wbar R_k (Wbar = W when Wbar is NULL; needs
 *                   readout_per_head = 0), i.e. z_tv = tau_k <Wbar_v, R_k hhat_t>
 *                   + b_kv.  R_k is used as given (orthogonality is not
 *                   checked).  The library rotates the heads' normalised
 *                   rows instead of forming Wbar R_k: u_t = R_k (g_k * h_t)
 *                   (rounded to bf16 on the bf16 path, as the product
 *                   g_k * h_t is there) and, backward, R_k^T applied to
 *                   sum_v delta_tv Wbar_v (2 T d^2 multiply-adds per head each
 *                   way).  The workspace then also holds (K-1) T d elements of
 *                   u and, for fwd_bwd, 2 (K-1) T d floats and (K-1) d^2
 *                   elements.  Ignored when K = 1.
 *
 * Which gradients (fwd_bwd only; exit evaluation computes none):
 *   final_module_dW      dW of the terminal, and with a shared gain its dgain.
 *   heads_train_readout  PRIV: dWbar of every head; needs readout_per_head.
 *   dtau != NULL         d losses[k] / d tau_k for every k (at tau = 1 if tau is NULL).
 *   dbias != NULL        d losses[k] / d b_k for every k (at b = 0 if bias is NULL).
 *                        The heads whose readout is not trained then run an
 *                        extra logits-only pass (the bias-gradient pass): the
 *                        column sums of the softmax need the final log-sum-exp.
 *
 * Outputs (fwd_bwd):
 *   dh              [K][T][d] dtype, 16-byte aligned, required.
 *   dW              [V][d] float, 16-byte aligned, required iff final_module_dW.
 *   dWbar           [K-1][V][d] float, 16-byte aligned, required iff
 *                   heads_train_readout and K > 1.
 *   dgain           float, 4-byte aligned: [K][d] iff gain_per_module
 *                   (required); else [d], required iff final_module_dW.
 *   dtau            [K] float or NULL, 4-byte aligned.
 *   dbias           [K][V] float or NULL, 4-byte aligned.
 * Outputs (exit evaluation):
 *   losses, row_loss as above; top1 [K][T] int32 or NULL, 4-byte aligned:
 *   argmax_v z_tv in fp32 arithmetic, the lowest v on ties.
 *
 *   stage_events    NULL or SOLO_NUM_STAGES hipEvent_t, as for
 *                   solo_readout_fwd_bwd_profiled.
 *
 * Semantics and errors as for solo_readout_fwd_bwd.  SOLO_ERR_ARG also for:
 * a flag not 0 or 1, readout_per_head without Wbar, heads_train_readout
 * without readout_per_head, rot with readout_per_head.
 *
 * ABI version 3 appended rot to the end of the struct (a caller built against
 * version 2 that zero-fills a version-2 struct must not pass it to a
 * version-3 library: the library reads the new field).
 */
typedef struct solo_readout_args {
    int K, T, d, V;
    int dtype;
    float eps;
    const void* h;
    const void* gain;
    const void* W;
    const void* Wbar;
    const float* tau;
    const float* bias;
    const int32_t* targets;
    int gain_per_module;
    int readout_per_head;
    int final_module_dW;
    int heads_train_readout;
    float* losses;
    float* row_loss;
    void* dh;
    float* dW;
    float* dWbar;
    float* dgain;
    float* dtau;
    float* dbias;
    int32_t* top1;
    void* workspace;
    size_t workspace_bytes;
    void* hip_stream;
    void* const* stage_events;
    const void* rot;
} solo_readout_args;

/* Workspace bytes of solo_readout_general with these arguments (only the
 * sizes, dtype, flags and which optional pointers are NULL matter); 0 if the
 * call would be rejected for its sizes, dtype or flags. */
size_t solo_readout_general_workspace_size(const solo_readout_args* args);

/* Forward and local backward with every option above. */
int solo_readout_general(const solo_readout_args* args);

/* Workspace bytes of solo_readout_exit_eval: per-token statistics (K T
 * floats each), the tiled readout copies of the matrix-core families (V d
 * terms, as for the general entry point) and, with rot, the rotated rows. */
size_t solo_readout_exit_eval_workspace_size(const solo_readout_args* args);

/* Forward-only exit evaluation: losses, row_loss and top1 of every module. */
int solo_readout_exit_eval(const solo_readout_args* args);

#ifdef __cplusplus
}
#endif

#endif /* SOLO_READOUT_H */
