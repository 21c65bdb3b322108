// Internal declarations of the SOLO readout library (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace solo {

typedef __bf16 bf16;

// Everything one fused pass needs.  The fused kernels keep a tile of
// "stationary" rows (X) on chip and stream "streamed" rows (Y) in chunks:
//   local-loss pass:    X = h of module k (rows t), Y = readout rows (v)
//   readout-grad pass:  X = readout rows (v),       Y = h of the final module (rows t)
struct FusedArgs {
    int K, T, d, V;
    float inv_T;
    const void* h;        // [K][T][d] elem
    const void* Wg;       // [V][d] elem: readout with the gain folded in (workspace)
    const void* W;        // [V][d] elem: readout as given (dgain epilogue)
    const void* gain;     // [d] elem
    const int32_t* targets;  // [K][T]
    const float* rstd;    // [K][T] 1/sqrt(mean h^2 + eps)
    float* lse;           // [K][T] log-sum-exp (written by the local-loss pass)
    float* rowrec;        // [T][4] final module: {lse log2 e, rstd log2 e, target bits, rstd / T} per token
    float* rowloss;       // [K][T] per-token cross-entropy
    void* dh;             // [K][T][d] elem
    float* dW;            // [V][d]
    float* dgain_part;    // [ceil(V / vtile)][d] per-vocab-tile partial sums of W * D
};

// Tile sizes of the two kernel families (the workspace depends on them).
constexpr int kMfmaRows = 32;      // stationary rows per workgroup (matrix-core kernels)
constexpr int kValuRows = 8;       // stationary rows per workgroup (vector-ALU kernels)

// small kernels (k_small.hip)
hipError_t launch_prep_readout(int dtype, const void* W, const void* gain, void* Wg, int V, int d, hipStream_t s);
hipError_t launch_row_rstd(int dtype, const void* h, float* rstd, long long rows, int d, float eps, hipStream_t s);
hipError_t launch_module_loss(const float* rowloss, float* losses, int K, int T, hipStream_t s);
hipError_t launch_dgain_reduce(const float* part, float* dgain, int ntiles, int d, hipStream_t s);

// fused passes
bool mfma_supported(int dtype, int d);
hipError_t launch_local_loss_mfma(const FusedArgs& a, hipStream_t s);
hipError_t launch_readout_grad_mfma(const FusedArgs& a, hipStream_t s);
hipError_t launch_local_loss_valu(int dtype, const FusedArgs& a, hipStream_t s);
hipError_t launch_readout_grad_valu(int dtype, const FusedArgs& a, hipStream_t s);

}  // namespace solo
