// Internal declarations of the SOLO readout library (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace solo {

typedef __bf16 bf16;

// Tiled copy of a streamed matrix Y [nY][d] (bf16), the operand layout of the
// matrix-core passes: rows are grouped in chunks of 16, and chunk c occupies
// 16 d contiguous elements, one 1 KiB block per 32 columns; inside a block,
// 16-byte granule q = 16 g + r holds Y[16 c + r][32 b + 8 g .. + 7].  Lane l of
// a wave that loads 16 bytes at block + 16 l therefore receives exactly the
// A operand of a 16x16x32 MFMA over those 32 columns (row l % 16, columns
// 8 (l / 16) .. + 7).  Rows past nY up to the chunk boundary are zeros.
__host__ __device__ inline long long tiled_elems(long long nY, int d) { return (nY + 15) / 16 * 16 * (long long)d; }

// Everything one fused pass needs.  The fused kernels keep a tile of
// "stationary" rows (X) on chip and stream "streamed" rows (Y) in chunks:
//   local-loss pass:      X = g_k * h_k (rows t),     Y = readout of module k (rows v)
//   exit evaluation:      same, forward only
//   readout-grad pass:    X = readout_k (rows v),       Y = g_k * h_k (rows t)
//   bias-grad pass:       same, without the second product
// In the matrix-core passes both products see the same rounded operands
// bf16(g_k * h_k) and R_k: the local-loss pass rounds g_k * h_k while it loads
// its stationary tile, and the readout-/bias-gradient passes stream a tiled
// copy that a small kernel wrote with the same rounding (so their recomputed
// logits match the stored log-sum-exp).  The register-fed matrix-core passes
// stream Y from its tiled copy (see tiled_elems); the others read Y row-major.
struct FusedArgs {
    int K, T, d, V;
    int m0;               // module of grid row 0 (module = m0 + blockIdx.y)
    float inv_T;
    const void* h;        // [K][T][d] elem
    const void* Wt;       // [V][d] elem: readout of module K-1 (the terminal)
    const void* Wh;       // elem: readout of module k < K-1 at Wh + k * wh_stride
    long long wh_stride;  // elements; 0 when every head reads the same matrix
    const void* Wtt;      // tiled copy of Wt (register-fed matrix-core passes)
    const void* Wht;      // tiled copy of the heads' readout(s): module k < K-1 at Wht + k * wht_stride
    long long wht_stride; // elements; 0 when every head reads the same matrix
    const void* hg;       // copies of bf16(g_k * h_k), modules hg_m0.., tiled_elems(T, d) apart: row-major for
                          // the direct-to-LDS passes, tiled for the register-fed ones
    int hg_m0;
    const void* gain;     // elem: gain of module k at gain + k * g_stride
    int g_stride;         // 0 (one gain) or d (one per module)
    const float* tau;     // [K] or null (temperature 1)
    const float* bias;    // [K][V] or null (no bias)
    const int32_t* targets;  // [K][T]
    const float* rstd;    // [K][T] 1/sqrt(mean h^2 + eps)
    float* lse;           // [K][T] log-sum-exp of the logits (written by the local-loss pass)
    float* rowrec;        // [K][T][4] or null: {lse log2 e, r tau log2 e, target bits, p_y - 1} per token
                          // (the vector-ALU family reads only p_y - 1)
    float* rowloss;       // [K][T] per-token cross-entropy
    float* rowdtau;       // [K][T] or null: per-token share of d loss / d tau
    int32_t* top1;        // [K][T] or null: exit evaluation, argmax of the logits (lowest index on ties)
    void* dh;             // [K][T][d] elem
    float* dgain_part;    // [slots][gridDim.x][d]: per-tile partial sums of dhhat * n
    int dg_mode;          // 0: no gain gradient; 1: module K-1 only (slot 0); 2: every module (slot k)
    float* dWt;           // [V][d] or null: d loss_{K-1} / d W
    float* dWh;           // [K-1][V][d] or null: d loss_k / d readout_k of the heads
    float* dbias;         // [K][V] or null: d loss_k / d b_k
    void* ebuf;           // null, or: the local-loss pass writes e_t = sum_v delta_tv R_kv there instead of
                          // the RMSNorm backward (ROT heads: their stationary rows are rotated states, whose
                          // gradient is rotated back afterwards).  Row m = k T + t holds 4 d bytes: the
                          // matrix-core families write two bf16 planes, hi = bf16(e) at [0, d) and
                          // lo = bf16(e - hi) at [d, 2d) (the rotate-back product's operand as a 2d-deep
                          // bf16 row); the vector-ALU family writes e in fp32
};

// Tile sizes of the two kernel families (the workspace depends on them).
constexpr int kMfmaRows = 32;      // stationary rows per workgroup of the matrix-core kernels at d > 1024
constexpr int kMfmaWideRows = 16;  // stationary rows per workgroup (wide matrix-core kernels, d = 2560)
constexpr int kValuRows = 8;       // stationary rows per workgroup (vector-ALU kernels)

// small kernels (k_small.hip)
hipError_t launch_row_rstd(int dtype, const void* h, float* rstd, long long rows, int d, float eps, hipStream_t s);
// tiled copies (layout of tiled_elems) of nmat row-major matrices [nY][d], src_stride
// elements apart; with a gain, of bf16(Y * gain[m g_stride + j]) (the rounding of the
// local-loss pass's stationary tile)
hipError_t launch_tile(const bf16* src, long long src_stride, const bf16* gain, int g_stride, bf16* dst, int nmat,
                       int nY, int d, hipStream_t s);
// row-major copies hg[m][t][j] = bf16(h[m][t][j] gain[m g_stride + j]), matrices src_stride / dst_stride apart
hipError_t launch_gain_rows(const bf16* h, long long src_stride, const bf16* gain, int g_stride, bf16* hg,
                            long long dst_stride, int nmat, int T, int d, hipStream_t s);
// out[k] = scale * sum_t rows[k][t], fixed order
hipError_t launch_module_sum(const float* rows, float* out, int K, int T, double scale, hipStream_t s);
// dgain[slot][j] = sum over tiles of part[slot][tile][j], fixed order
hipError_t launch_dgain_reduce(const float* part, float* dgain, int slots, int ntiles, int d, hipStream_t s);

// fused passes; `ext` selects the local-loss variant with per-chunk biases,
// `nmod` is the number of modules of a readout-/bias-gradient launch
bool mfma_supported(int dtype, int d);
int mfma_rows(int d);  // stationary rows per workgroup of the matrix-core kernels at width d (64 or 32)
// local-loss and exit passes: modules m0 .. m0 + nmod - 1
hipError_t launch_local_loss_mfma(const FusedArgs& a, bool ext, int nmod, hipStream_t s);
hipError_t launch_exit_eval_mfma(const FusedArgs& a, int nmod, hipStream_t s);
hipError_t launch_readout_grad_mfma(const FusedArgs& a, int nmod, hipStream_t s);
hipError_t launch_bias_grad_mfma(const FusedArgs& a, int nmod, hipStream_t s);
// the wide matrix-core kernels (k_mfma_wide.hip): d = 2560
bool mfma_wide_supported(int dtype, int d);
hipError_t launch_local_loss_mfma_wide(const FusedArgs& a, bool ext, int nmod, hipStream_t s);
hipError_t launch_exit_eval_mfma_wide(const FusedArgs& a, int nmod, hipStream_t s);
hipError_t launch_readout_grad_mfma_wide(const FusedArgs& a, int nmod, hipStream_t s);
hipError_t launch_bias_grad_mfma_wide(const FusedArgs& a, int nmod, hipStream_t s);
hipError_t launch_local_loss_valu(int dtype, const FusedArgs& a, int nmod, hipStream_t s);
hipError_t launch_exit_eval_valu(int dtype, const FusedArgs& a, int nmod, hipStream_t s);
// ROT (k_rot.hip): C = A B^T per matrix; transposes; a vector of ones; the
// heads' RMSNorm backward from the rotated-back gradient D = e R_k
// u[m] = bf16(R_m bf16(g_m * h_m)) per row, heads m < nmat (gain g_m at gain + m g_stride)
hipError_t launch_rot_rows(int dtype, const void* h, const void* gain, int g_stride, const void* R, void* u,
                           int nmat, int T, int d, hipStream_t s);
// D[m] = e_m R_m from R_m^T (Rt); e as the matrix-core families' bf16 planes or in fp32
hipError_t launch_rot_back(int dtype, bool planes, const void* e, const void* Rt, float* D, int nmat, int T, int d,
                           hipStream_t s);
// whether launch_rot_back takes the planes form at this dtype and width
bool rot_back_planes(int dtype, int d);
hipError_t launch_transpose(int dtype, const void* in, void* out, int nmat, int d, hipStream_t s);
hipError_t launch_fill_one(int dtype, void* p, int n, hipStream_t s);
hipError_t launch_rot_post(int dtype, const float* D, const void* h, const void* gain, int g_stride,
                           const float* rstd, const float* tau, void* dh, float* dgain_part, int nmod, int T, int d,
                           int rows, hipStream_t s);
hipError_t launch_readout_grad_valu(int dtype, const FusedArgs& a, int nmod, hipStream_t s);
hipError_t launch_bias_grad_valu(int dtype, const FusedArgs& a, int nmod, hipStream_t s);

}  // namespace solo
