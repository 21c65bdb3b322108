// Kernels of the ROT readout source (the paper's table of readout content and
// basis, Appendix D): head k reads sg(Wbar) R_k through a fixed d x d matrix
// R_k.  Since z_v = <Wbar_v R_k, hhat> = <Wbar_v, R_k hhat>, the library
// rotates the head's normalised states instead of forming the V x d product:
//
//   u_t     = R_k (g_k * h_t)                  (bf16, the head's stationary rows)
//   e_t     = sum_v delta_tv Wbar_v / tau_k    (the local-loss pass on u)
//   dhhat_t = tau_k R_k^T e_t                  (back to the hidden states' basis)
//   dh_t    = r_t (g_k * dhhat_t - c_t n_t),  c_t = mean_j g_kj dhhat_tj n_tj
//
// with r_t, n_t = r_t h_t of the original hidden states (the rotation commutes
// with the row scale r_t).  Both products are C = A B^T of row-major A [M][K]
// and B [N][K]: u = (g * h) R_k^T and dhhat / tau = e (R_k^T)^T.
#include "mfma_common.h"

namespace solo {

namespace {

using mfma::bf16x8;
using mfma::f32x16;
using mfma::f32x4;

// C[m][n] = sum_k A[m][k] B[n][k] on 32x32x16 bf16 matrix instructions.  A
// workgroup of 4 waves owns a 64 x 128 tile of C; wave (wm, wn) a 32 x 64
// block (two products per 16-deep step).  Operands come straight from global
// memory: lane l holds A[m0 + l % 32][k0 + 8 (l / 32) .. + 7] and
// B[n0 + l % 32][k0 + 8 (l / 32) .. + 7], 16 contiguous bytes each.
// AT: bf16 A (times a per-column gain, rounded once to bf16, when gain is not
// null) or fp32 A (split into two bf16 parts); CT: bf16 or fp32 C.  N % 128 == 0,
// K % 16 == 0; rows m >= M read as zero and are not written.
template <typename AT, typename CT>
__global__ __launch_bounds__(256) void k_gemm_nt_mfma(const AT* __restrict__ A, long long a_mat, const bf16* gain,
                                                     int g_stride, const bf16* __restrict__ B, long long b_mat,
                                                     CT* __restrict__ C, long long c_mat, int M, int N, int Kd) {
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int mat = blockIdx.z;
    A += mat * a_mat;
    B += mat * b_mat;
    C += mat * c_mat;
    const bf16* g = gain ? gain + (long long)mat * g_stride : nullptr;
    const int m0 = blockIdx.x * 64 + 32 * (w & 1);
    const int n0 = blockIdx.y * 128 + 64 * (w >> 1);
    const int mr = m0 + (lane & 31);
    const bool mok = mr < M;
    const int kl = 8 * (lane >> 5);
    f32x16 acc[2];
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[b][i] = 0.f;
    for (int k0 = 0; k0 < Kd; k0 += 16) {
        const int kk = k0 + kl;
        bf16x8 av, alo;
        if constexpr (sizeof(AT) == 2) {
            av = mok ? *(const bf16x8*)((const bf16*)A + (long long)mr * Kd + kk) : bf16x8{};
            if (g) {
                const bf16x8 gv = *(const bf16x8*)(g + kk);
#pragma unroll
                for (int e = 0; e < 8; ++e) av[e] = (bf16)((float)av[e] * (float)gv[e]);
            }
        } else {
            // fp32 A as the sum of two bf16 parts, hi = bf16(x) and lo = bf16(x - hi):
            // the product then keeps about 16 bits of A (B is bf16 already)
            f32x4 x0 = {0.f, 0.f, 0.f, 0.f}, x1 = x0;
            if (mok) {
                x0 = *(const f32x4*)((const float*)A + (long long)mr * Kd + kk);
                x1 = *(const f32x4*)((const float*)A + (long long)mr * Kd + kk + 4);
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float xv = e < 4 ? x0[e] : x1[e - 4];
                av[e] = (bf16)xv;
                alo[e] = (bf16)(xv - (float)av[e]);
            }
        }
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const bf16x8 bv = *(const bf16x8*)(B + (long long)(n0 + 32 * b + (lane & 31)) * Kd + kk);
            acc[b] = mfma::mfma32(av, bv, acc[b]);
            if constexpr (sizeof(AT) == 4) acc[b] = mfma::mfma32(alo, bv, acc[b]);
        }
    }
    // C layout: lane holds C[m0 + 8 (i / 4) + 4 (lane / 32) + i % 4][n0 + 32 b + lane % 32]
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int m = m0 + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
            if (m < M) C[(long long)m * N + n0 + 32 * b + (lane & 31)] = (CT)acc[b][i];
        }
}

// The same product in fp32 on the vector ALU (fp32 storage, and bf16 widths
// the matrix-core tiling does not cover): one thread per element of C.
template <typename AT, typename BT, typename CT>
__global__ void k_gemm_nt_valu(const AT* __restrict__ A, long long a_mat, const BT* gain, int g_stride,
                               const BT* __restrict__ B, long long b_mat, CT* __restrict__ C, long long c_mat, int M,
                               int N, int Kd) {
    const int mat = blockIdx.z;
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (long long)M * N) return;
    const int m = (int)(i / N), n = (int)(i % N);
    const AT* a = A + mat * a_mat + (long long)m * Kd;
    const BT* b = B + mat * b_mat + (long long)n * Kd;
    const BT* g = gain ? gain + (long long)mat * g_stride : nullptr;
    float s = 0.f;
    for (int k = 0; k < Kd; ++k) {
        float av = (float)a[k];
        if (g) {
            av *= (float)g[k];
            if (sizeof(BT) == 2) av = (float)(bf16)av;  // the product the bf16 local-loss pass rounds
        }
        s = fmaf(av, (float)b[k], s);
    }
    C[mat * c_mat + (long long)m * N + n] = (CT)s;
}

// out[k][j][i] = in[k][i][j] for nmat d x d matrices
template <typename E>
__global__ void k_transpose(const E* __restrict__ in, E* __restrict__ out, int d) {
    __shared__ E tile[32][33];
    const long long off = (long long)blockIdx.z * d * d;
    const int i0 = blockIdx.y * 32, j0 = blockIdx.x * 32;
    for (int r = threadIdx.y; r < 32; r += blockDim.y) {
        const int i = i0 + r, j = j0 + threadIdx.x;
        if (i < d && j < d) tile[r][threadIdx.x] = in[off + (long long)i * d + j];
    }
    __syncthreads();
    for (int r = threadIdx.y; r < 32; r += blockDim.y) {
        const int j = j0 + r, i = i0 + threadIdx.x;
        if (i < d && j < d) out[off + (long long)j * d + i] = tile[threadIdx.x][r];
    }
}

template <typename E>
__global__ void k_fill_one(E* __restrict__ p, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = (E)1.f;
}

// The RMSNorm backward of ROT heads from the rotated-back gradient D = e R_k
// (fp32, [T][d] per head): dhhat = tau D, dn = g * dhhat, c = mean(dn * n),
// dh = r (dn - c n); with a per-module gain also the tile's partial sums of
// dhhat * n (rows tiles of the local-loss pass).  One workgroup per tile of
// rows rows of one head; thread t takes columns t + 256 q.
template <typename E>
__global__ __launch_bounds__(256) void k_rot_post(const float* __restrict__ D, const E* __restrict__ h,
                                                 const E* __restrict__ gain, int g_stride, const float* __restrict__ rstd,
                                                 const float* __restrict__ tau, E* __restrict__ dh, float* dgain_part,
                                                 int T, int d, int rows) {
    constexpr int NQ = 16;  // d <= 4096
    __shared__ float red[8];
    const int k = blockIdx.y;
    const int tile = blockIdx.x;
    const int tid = threadIdx.x;
    const float tk = tau ? tau[k] : 1.f;
    const E* g = gain + (long long)k * g_stride;
    float part[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q) part[q] = 0.f;
    for (int tr = 0; tr < rows; ++tr) {
        const int t = tile * rows + tr;
        if (t >= T) break;
        const long long row = (long long)k * T + t;
        const float r = rstd[row];
        float c = 0.f;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int j = tid + 256 * q;
            if (j < d) c = fmaf((float)g[j] * tk * D[row * d + j], r * (float)h[row * d + j], c);
        }
        for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off, 64);
        if ((tid & 63) == 0) red[tid >> 6] = c;
        __syncthreads();
        const float cm = (red[0] + red[1] + red[2] + red[3]) / (float)d;
        __syncthreads();
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int j = tid + 256 * q;
            if (j < d) {
                const float dhat = tk * D[row * d + j];
                const float n = r * (float)h[row * d + j];
                dh[row * d + j] = (E)(r * ((float)g[j] * dhat - cm * n));
                part[q] = fmaf(dhat, n, part[q]);
            }
        }
    }
    if (dgain_part) {
        float* p = dgain_part + ((long long)k * gridDim.x + tile) * d;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int j = tid + 256 * q;
            if (j < d) p[j] = part[q];
        }
    }
}

}  // namespace

// C = A B^T per matrix (nmat of them, strides in elements): A bf16 (times
// gain) or fp32, B in the storage dtype, C bf16/fp32 as named.
hipError_t launch_rot_gemm(int dtype, bool a_f32, const void* A, long long a_mat, const void* gain, int g_stride,
                           const void* B, long long b_mat, void* C, bool c_f32, long long c_mat, int nmat, int M,
                           int N, int Kd, hipStream_t s) {
    if (dtype == 0 && N % 128 == 0 && Kd % 16 == 0) {
        dim3 grid((unsigned)((M + 63) / 64), (unsigned)(N / 128), (unsigned)nmat);
        if (!a_f32 && !c_f32)
            hipLaunchKernelGGL((k_gemm_nt_mfma<bf16, bf16>), grid, dim3(256), 0, s, (const bf16*)A, a_mat,
                               (const bf16*)gain, g_stride, (const bf16*)B, b_mat, (bf16*)C, c_mat, M, N, Kd);
        else if (a_f32 && c_f32)
            hipLaunchKernelGGL((k_gemm_nt_mfma<float, float>), grid, dim3(256), 0, s, (const float*)A, a_mat,
                               (const bf16*)gain, g_stride, (const bf16*)B, b_mat, (float*)C, c_mat, M, N, Kd);
        else
            return hipErrorInvalidValue;
        return hipGetLastError();
    }
    const long long n = (long long)M * N;
    dim3 grid((unsigned)((n + 255) / 256), 1, (unsigned)nmat);
    if (dtype == 0) {
        if (!a_f32 && !c_f32)
            hipLaunchKernelGGL((k_gemm_nt_valu<bf16, bf16, bf16>), grid, dim3(256), 0, s, (const bf16*)A, a_mat,
                               (const bf16*)gain, g_stride, (const bf16*)B, b_mat, (bf16*)C, c_mat, M, N, Kd);
        else if (a_f32 && c_f32)
            hipLaunchKernelGGL((k_gemm_nt_valu<float, bf16, float>), grid, dim3(256), 0, s, (const float*)A, a_mat,
                               (const bf16*)gain, g_stride, (const bf16*)B, b_mat, (float*)C, c_mat, M, N, Kd);
        else
            return hipErrorInvalidValue;
    } else {
        hipLaunchKernelGGL((k_gemm_nt_valu<float, float, float>), grid, dim3(256), 0, s, (const float*)A, a_mat,
                           (const float*)gain, g_stride, (const float*)B, b_mat, (float*)C, c_mat, M, N, Kd);
    }
    return hipGetLastError();
}

hipError_t launch_transpose(int dtype, const void* in, void* out, int nmat, int d, hipStream_t s) {
    dim3 grid((unsigned)((d + 31) / 32), (unsigned)((d + 31) / 32), (unsigned)nmat);
    if (dtype == 0)
        hipLaunchKernelGGL(k_transpose<bf16>, grid, dim3(32, 8), 0, s, (const bf16*)in, (bf16*)out, d);
    else
        hipLaunchKernelGGL(k_transpose<float>, grid, dim3(32, 8), 0, s, (const float*)in, (float*)out, d);
    return hipGetLastError();
}

hipError_t launch_fill_one(int dtype, void* p, int n, hipStream_t s) {
    if (dtype == 0)
        hipLaunchKernelGGL(k_fill_one<bf16>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, (bf16*)p, n);
    else
        hipLaunchKernelGGL(k_fill_one<float>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, (float*)p, n);
    return hipGetLastError();
}

hipError_t launch_rot_post(int dtype, const float* D, const void* h, const void* gain, int g_stride,
                           const float* rstd, const float* tau, void* dh, float* dgain_part, int nmod, int T, int d,
                           int rows, hipStream_t s) {
    dim3 grid((unsigned)((T + rows - 1) / rows), (unsigned)nmod);
    if (dtype == 0)
        hipLaunchKernelGGL(k_rot_post<bf16>, grid, dim3(256), 0, s, D, (const bf16*)h, (const bf16*)gain, g_stride,
                           rstd, tau, (bf16*)dh, dgain_part, T, d, rows);
    else
        hipLaunchKernelGGL(k_rot_post<float>, grid, dim3(256), 0, s, D, (const float*)h, (const float*)gain,
                           g_stride, rstd, tau, (float*)dh, dgain_part, T, d, rows);
    return hipGetLastError();
}

}  // namespace solo
