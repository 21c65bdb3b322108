// Bandwidth-light kernels around the fused passes:
//   - per-row inverse RMS of the hidden states,
//   - the copies the matrix-core passes stream: tiled readouts, and the
//     gain-scaled bf16(g_k * h_k) of the gradient passes (tiled, or row-major
//     for the direct-to-LDS readout-gradient pass),
//   - fixed-order reductions for the module losses, the temperature gradients
//     and the gain gradients.
#include "mfma_layout.h"
#include "solo_internal.h"

namespace solo {

namespace {

__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }
__device__ __forceinline__ float to_f32(float x) { return x; }

// rstd[row] = 1 / sqrt(mean_j h[row][j]^2 + eps); one wave per row.
template <typename E>
__global__ void k_row_rstd(const E* __restrict__ h, float* __restrict__ rstd, long long rows, int d, float eps) {
    // one wave per row, 16 bytes per lane per load (d % 8 == 0 and 16-byte aligned rows)
    constexpr int VE = 16 / (int)sizeof(E);
    typedef E ev __attribute__((ext_vector_type(VE)));
    const int lane = threadIdx.x & 63;
    long long row = (long long)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
    if (row >= rows) return;
    const E* x = h + row * (long long)d;
    float acc = 0.f;
    for (int j = lane * VE; j < d; j += 64 * VE) {
        const ev v = *(const ev*)(x + j);
#pragma unroll
        for (int e = 0; e < VE; ++e) {
            const float f = to_f32(v[e]);
            acc = fmaf(f, f, acc);
        }
    }
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
    if (lane == 0) {
        double ms = (double)acc / (double)d;
        rstd[row] = (float)(1.0 / sqrt(ms + (double)eps));
    }
}

// Tiled copy of nmat row-major matrices (the streamed-operand layout of the
// matrix-core passes, see tiled_elems and layout::tile_row / tile_col):
// thread o of chunk c writes output granule o (zeros past the last row).  With a
// gain, the copy is bf16(y * g): the same product and rounding as the
// stationary-tile load of the local-loss pass.
__global__ void k_tile(const bf16* __restrict__ src, long long src_stride, const bf16* __restrict__ gain,
                       int g_stride, bf16* __restrict__ dst, int nY, int d) {
    typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
    const int c = blockIdx.x;
    const int m = blockIdx.z;
    const int o = blockIdx.y * blockDim.x + threadIdx.x;
    if (o >= 2 * d) return;  // 2 d granules of 16 bytes per chunk
    const int row = 16 * c + layout::tile_row(o);
    const int j = layout::tile_col(o);
    bf16x8 v;
    if (row < nY) {
        v = *(const bf16x8*)(src + (long long)m * src_stride + (long long)row * d + j);
        if (gain) {
            const bf16x8 g = *(const bf16x8*)(gain + (long long)m * g_stride + j);
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = (bf16)((float)v[e] * (float)g[e]);
        }
    } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = (bf16)0.f;
    }
    *(bf16x8*)(dst + (long long)m * tiled_elems(nY, d) + (long long)c * 16 * d + 8LL * o) = v;
}

// Row-major gain-scaled copies hg[m][t][j] = bf16(h[m][t][j] g[m g_stride + j])
// (the stream of the direct-to-LDS readout-gradient pass), matrices dst_stride
// elements apart; 8 elements per thread (d % 8 == 0).
__global__ void k_gain_rows(const bf16* __restrict__ h, long long src_stride, const bf16* __restrict__ gain,
                            int g_stride, bf16* __restrict__ hg, long long dst_stride, long long per_mod, int d) {
    typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
    const long long n8 = per_mod / 8;
    const int m = blockIdx.y;
    const bf16* hm = h + (long long)m * src_stride;
    const bf16* gm = gain + (long long)m * g_stride;
    bf16* om = hg + (long long)m * dst_stride;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n8; i += (long long)gridDim.x * blockDim.x) {
        const int j = (int)((i * 8) % d);
        const bf16x8 hv = *(const bf16x8*)(hm + i * 8);
        const bf16x8 gv = *(const bf16x8*)(gm + j);
        bf16x8 o;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = (bf16)((float)hv[e] * (float)gv[e]);
        *(bf16x8*)(om + i * 8) = o;
    }
}

// out[k] = scale * sum_t rows[k][t], fixed order, fp64 accumulation
// (module losses: the per-token losses with scale 1/T; temperature gradients:
// the per-token shares with scale 1).
__global__ __launch_bounds__(1024) void k_module_sum(const float* __restrict__ rows, float* __restrict__ out, int T,
                                                    double scale) {
    __shared__ double red[1024];
    const int k = blockIdx.x;
    const float* r = rows + (long long)k * T;
    double acc = 0.0;
#pragma unroll 8
    for (int t = threadIdx.x; t < T; t += 1024) acc += (double)r[t];
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int w = 512; w > 0; w >>= 1) {
        if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) out[k] = (float)(red[0] * scale);
}

// dgain[slot][j] = sum over token tiles of part[slot][tile][j], fixed order:
// a block of 256 threads covers 32 columns of one slot; its 8 thread groups
// sum every eighth tile, then the 8 group sums are added in group order.
__global__ void k_dgain_reduce(const float* __restrict__ part, float* __restrict__ dgain, int ntiles, int d) {
    __shared__ double red[8][32];
    const int jl = threadIdx.x & 31, grp = threadIdx.x >> 5;
    const int j = blockIdx.x * 32 + jl;
    part += (long long)blockIdx.y * ntiles * d;
    dgain += (long long)blockIdx.y * d;
    double acc = 0.0;
    if (j < d) {
#pragma unroll 8
        for (int i = grp; i < ntiles; i += 8) acc += (double)part[(long long)i * d + j];
    }
    red[grp][jl] = acc;
    __syncthreads();
    if (grp == 0 && j < d) {
        double s = 0.0;
        for (int g = 0; g < 8; ++g) s += red[g][jl];
        dgain[j] = (float)s;
    }
}

}  // namespace

hipError_t launch_row_rstd(int dtype, const void* h, float* rstd, long long rows, int d, float eps, hipStream_t s) {
    long long blocks = (rows + 3) / 4;
    if (dtype == 0)
        hipLaunchKernelGGL(k_row_rstd<bf16>, dim3((unsigned)blocks), dim3(256), 0, s, (const bf16*)h, rstd, rows, d, eps);
    else
        hipLaunchKernelGGL(k_row_rstd<float>, dim3((unsigned)blocks), dim3(256), 0, s, (const float*)h, rstd, rows, d, eps);
    return hipGetLastError();
}

hipError_t launch_tile(const bf16* src, long long src_stride, const bf16* gain, int g_stride, bf16* dst, int nmat,
                       int nY, int d, hipStream_t s) {
    const unsigned nchunks = (unsigned)((nY + 15) / 16);
    const unsigned parts = (unsigned)((2 * d + 255) / 256);
    hipLaunchKernelGGL(k_tile, dim3(nchunks, parts, (unsigned)nmat), dim3(256), 0, s, src, src_stride, gain, g_stride,
                       dst, nY, d);
    return hipGetLastError();
}

hipError_t launch_gain_rows(const bf16* h, long long src_stride, const bf16* gain, int g_stride, bf16* hg,
                            long long dst_stride, int nmat, int T, int d, hipStream_t s) {
    const long long per_mod = (long long)T * d;
    long long blocks = (per_mod / 8 + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(k_gain_rows, dim3((unsigned)blocks, (unsigned)nmat), dim3(256), 0, s, h, src_stride, gain,
                       g_stride, hg, dst_stride, per_mod, d);
    return hipGetLastError();
}

hipError_t launch_module_sum(const float* rows, float* out, int K, int T, double scale, hipStream_t s) {
    hipLaunchKernelGGL(k_module_sum, dim3(K), dim3(1024), 0, s, rows, out, T, scale);
    return hipGetLastError();
}

hipError_t launch_dgain_reduce(const float* part, float* dgain, int slots, int ntiles, int d, hipStream_t s) {
    hipLaunchKernelGGL(k_dgain_reduce, dim3((d + 31) / 32, slots), dim3(256), 0, s, part, dgain, ntiles, d);
    return hipGetLastError();
}

}  // namespace solo
