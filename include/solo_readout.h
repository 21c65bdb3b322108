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

#define SOLO_READOUT_ABI_VERSION 1

/* Element type of h, gain, W and dh.  Statistics, exponentials and
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
    SOLO_ERR_WORKSPACE = 5, /* workspace_bytes < solo_readout_workspace_size(...)           */
    SOLO_ERR_ARG = 6,       /* eps < 0 or not finite; final_module_dW not 0 or 1           */
    SOLO_ERR_HIP = 7        /* a HIP runtime call or kernel launch failed                  */
} solo_status;

/* SOLO_READOUT_ABI_VERSION of the loaded library. */
int solo_readout_abi_version(void);

/* Static, NUL-terminated description of a status code (never NULL). */
const char* solo_status_string(int status);

/*
 * Bytes of device workspace one call needs.  A function of (K, T, d, V,
 * dtype, final_module_dW) with no T*V term: the largest piece is a V x d
 * copy of the readout with the gain folded in.  Returns 0 for arguments that
 * solo_readout_fwd_bwd would reject.
 */
size_t solo_readout_workspace_size(int K, int T, int d, int V, int dtype, int final_module_dW);

/*
 * Name of the kernel family one call with these sizes runs on:
 * "mfma" (bf16 matrix-core kernels) or "valu" (fp32 vector-ALU kernels,
 * used for SOLO_F32 and for bf16 widths the matrix-core kernels do not tile).
 * Returns "invalid" for arguments solo_readout_fwd_bwd would reject.
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
 * Stages of one call, in launch order (all on hip_stream).
 */
#define SOLO_NUM_STAGES 6
/*   0  fold the gain into the readout copy (workspace)          */
/*   1  per-token inverse RMS of h                                */
/*   2  local-loss pass: logits, online log-sum-exp, dh (all K)   */
/*   3  module losses (fixed-order mean of the per-token losses)  */
/*   4  readout-gradient pass of module K-1 (dW, dgain partials)  */
/*   5  dgain (fixed-order sum of the partials)                   */

/*
 * solo_readout_fwd_bwd, and for profiling: stage_events[i], if not NULL, is a
 * hipEvent_t that is recorded on hip_stream right after stage i has been
 * enqueued (stages 4 and 5 only run when final_module_dW = 1; their events
 * are then not recorded).  stage_events itself may be NULL.  Same arguments,
 * semantics and errors otherwise; a failed event record returns SOLO_ERR_HIP.
 */
int solo_readout_fwd_bwd_profiled(int K, int T, int d, int V, int dtype, float eps,
                                  const void* h, const void* gain, const void* W,
                                  const int32_t* targets, int final_module_dW,
                                  float* losses, float* row_loss, void* dh,
                                  float* dW, float* dgain,
                                  void* workspace, size_t workspace_bytes,
                                  void* hip_stream, void* const* stage_events);

#ifdef __cplusplus
}
#endif

#endif /* SOLO_READOUT_H */
