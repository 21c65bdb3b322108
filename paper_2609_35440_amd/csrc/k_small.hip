// Bandwidth-light kernels around the two fused passes:
//   - fold the RMSNorm gain into a copy of the readout (Wg = W diag(gain)),
//   - per-row inverse RMS of the hidden states,
//   - fixed-order reductions for the module losses and the gain gradient.
#include "solo_internal.h"

namespace solo {

namespace {

__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }
__device__ __forceinline__ float to_f32(float x) { return x; }
template <typename E> __device__ __forceinline__ E from_f32(float x);
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }

// Wg[v][j] = W[v][j] * gain[j], rounded once to the storage type.
// z_tv = <W_v, gain * n_t> = <Wg_v, n_t>, so the gain multiplies the readout
// once per call instead of every row of every module.
template <typename E>
__global__ void k_prep_readout(const E* __restrict__ W, const E* __restrict__ gain, E* __restrict__ Wg,
                               long long n, int d) {
    long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    long long stride = (long long)gridDim.x * blockDim.x;
    for (; i < n; i += stride) {
        int j = (int)(i % d);
        Wg[i] = from_f32<E>(to_f32(W[i]) * to_f32(gain[j]));
    }
}

// rstd[row] = 1 / sqrt(mean_j h[row][j]^2 + eps); one wave per row.
template <typename E>
__global__ void k_row_rstd(const E* __restrict__ h, float* __restrict__ rstd, long long rows, int d, float eps) {
    const int lane = threadIdx.x & 63;
    long long row = (long long)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
    if (row >= rows) return;
    const E* x = h + row * (long long)d;
    float acc = 0.f;
    for (int j = lane; j < d; j += 64) {
        float v = to_f32(x[j]);
        acc = fmaf(v, v, acc);
    }
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
    if (lane == 0) {
        double ms = (double)acc / (double)d;
        rstd[row] = (float)(1.0 / sqrt(ms + (double)eps));
    }
}

// losses[k] = (1/T) sum_t rowloss[k][t], fixed order, fp64 accumulation.
__global__ void k_module_loss(const float* __restrict__ rowloss, float* __restrict__ losses, int T) {
    __shared__ double red[256];
    const int k = blockIdx.x;
    const float* r = rowloss + (long long)k * T;
    double acc = 0.0;
    for (int t = threadIdx.x; t < T; t += 256) acc += (double)r[t];
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) losses[k] = (float)(red[0] / (double)T);
}

// dgain[j] = sum over vocabulary tiles of part[tile][j], fixed order: a
// block of 256 threads covers 32 columns; its 8 thread groups sum every
// eighth tile, then the 8 group sums are added in group order.
__global__ void k_dgain_reduce(const float* __restrict__ part, float* __restrict__ dgain, int ntiles, int d) {
    __shared__ double red[8][32];
    const int jl = threadIdx.x & 31, grp = threadIdx.x >> 5;
    const int j = blockIdx.x * 32 + jl;
    double acc = 0.0;
    if (j < d)
        for (int i = grp; i < ntiles; i += 8) acc += (double)part[(long long)i * d + j];
    red[grp][jl] = acc;
    __syncthreads();
    if (grp == 0 && j < d) {
        double s = 0.0;
        for (int g = 0; g < 8; ++g) s += red[g][jl];
        dgain[j] = (float)s;
    }
}

}  // namespace

hipError_t launch_prep_readout(int dtype, const void* W, const void* gain, void* Wg, int V, int d, hipStream_t s) {
    long long n = (long long)V * d;
    long long blocks = (n + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (dtype == 0)
        hipLaunchKernelGGL(k_prep_readout<bf16>, dim3((unsigned)blocks), dim3(256), 0, s, (const bf16*)W,
                           (const bf16*)gain, (bf16*)Wg, n, d);
    else
        hipLaunchKernelGGL(k_prep_readout<float>, dim3((unsigned)blocks), dim3(256), 0, s, (const float*)W,
                           (const float*)gain, (float*)Wg, n, d);
    return hipGetLastError();
}

hipError_t launch_row_rstd(int dtype, const void* h, float* rstd, long long rows, int d, float eps, hipStream_t s) {
    long long blocks = (rows + 3) / 4;
    if (dtype == 0)
        hipLaunchKernelGGL(k_row_rstd<bf16>, dim3((unsigned)blocks), dim3(256), 0, s, (const bf16*)h, rstd, rows, d, eps);
    else
        hipLaunchKernelGGL(k_row_rstd<float>, dim3((unsigned)blocks), dim3(256), 0, s, (const float*)h, rstd, rows, d, eps);
    return hipGetLastError();
}

hipError_t launch_module_loss(const float* rowloss, float* losses, int K, int T, hipStream_t s) {
    hipLaunchKernelGGL(k_module_loss, dim3(K), dim3(256), 0, s, rowloss, losses, T);
    return hipGetLastError();
}

hipError_t launch_dgain_reduce(const float* part, float* dgain, int ntiles, int d, hipStream_t s) {
    hipLaunchKernelGGL(k_dgain_reduce, dim3((d + 31) / 32), dim3(256), 0, s, part, dgain, ntiles, d);
    return hipGetLastError();
}

}  // namespace solo
