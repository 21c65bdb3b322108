// Kernels of the ROT readout source (the paper's table of readout content and
// basis, Appendix D): head k reads sg(Wbar) R_k through a fixed d x d matrix
// R_k.  Since z_v = <Wbar_v R_k, hhat> = <Wbar_v, R_k hhat>, the library
// rotates the head's normalised states instead of forming the V x d product:
//
//   u_t     = R_k (g_k * h_t)                  (bf16, the head's stationary rows)
//   e_t     = sum_v delta_tv Wbar_v            (the local-loss pass on u)
//   dhhat_t = tau_k R_k^T e_t                  (back to the hidden states' basis)
//   dh_t    = r_t (g_k * dhhat_t - c_t n_t),  c_t = mean_j g_kj dhhat_tj n_tj
//
// with r_t, n_t = r_t h_t of the original hidden states (the rotation commutes
// with the row scale r_t).  Both products are C = A B^T of row-major A [M][K]
// and B [N][K]: u = (g * h) R_k^T and dhhat / tau = e (R_k^T)^T, the latter
// with e as two bf16 planes (hi | lo, a 2d-deep row) on the matrix cores.
#include "mfma_common.h"

namespace solo {

namespace {

using mfma::bf16x8;
using mfma::f32x16;
using mfma::f32x4;

// C[m][n] = sum_k A[m][k] B[n][k mod ldb] on 32x32x16 bf16 matrix
// instructions, A [M][Kd] and B [N][ldb] row-major bf16 (Kd = ldb, or
// Kd = 2 ldb for the rotate-back product, whose A rows are e's two bf16
// planes hi | lo and whose B is then read twice).  Workgroup tile 256 x 128
// (4 waves, each a 128 x 64 block: 4 x 2 products of 32 x 32), k in steps of
// 64 staged through LDS: each 16-byte granule of the 256 x 64 and 128 x 64
// operand tiles is loaded by one thread into registers a step ahead, then
// written to LDS, whose rows have a 144-byte pitch (8 lanes of a 16-byte
// access, rows r..r+7 at one column, fall in 8 distinct 4-bank groups).  Lane
// l of a product reads A[row l % 32][k + 8 (l / 32) .. + 7] and B[col l % 32][same k].
// With a gain, A is bf16(A * gain[k]) (the rounding of the local-loss pass's
// stationary tile).  CT: bf16 or fp32 C.  N % 128 == 0, ldb % 64 == 0;
// rows m >= M read as zero and are not written.  Row tile of workgroup
// (x, y, z): mtile0 + y (launches of at most 65535 row tiles).
constexpr int GM = 256;          // tile rows
constexpr int GN = 128;          // tile columns
constexpr int GK = 64;           // k per staged step
constexpr int GP = GK + 8;       // LDS row pitch in elements (144 bytes)

template <typename CT>
__global__ __launch_bounds__(256, 2) void k_gemm_nt_mfma(const bf16* __restrict__ A, long long a_mat, int Kd,
                                                        const bf16* __restrict__ gain, int g_stride,
                                                        const bf16* __restrict__ B, long long b_mat, int ldb,
                                                        CT* __restrict__ C, long long c_mat, int M, int N,
                                                        int mtile0) {
    __shared__ __attribute__((aligned(16))) bf16 As[GM * GP];
    __shared__ __attribute__((aligned(16))) bf16 Bs[GN * GP];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = tid >> 6;
    const int mat = blockIdx.z;
    const int n0 = blockIdx.x * GN;
    const int m0 = (mtile0 + (int)blockIdx.y) * GM;
    A += mat * a_mat;
    B += mat * b_mat;
    C += mat * c_mat;
    const bf16* g = gain ? gain + (long long)mat * g_stride : nullptr;

    // staging: granule q = tid + 256 i of a tile is row q / 8, columns 8 (q % 8) .. + 7
    const int kc = tid & 7;
    const int r0 = tid >> 3;
    bf16x8 ast[GM / 32], bst[GN / 32];
    auto load = [&](int k0) __attribute__((always_inline)) {
        const int kb = k0 >= ldb ? k0 - ldb : k0;
#pragma unroll
        for (int i = 0; i < GN / 32; ++i)
            bst[i] = *(const bf16x8*)(B + (long long)(n0 + r0 + 32 * i) * ldb + kb + 8 * kc);
        bf16x8 gv = {};
        if (g) gv = *(const bf16x8*)(g + k0 + 8 * kc);
#pragma unroll
        for (int i = 0; i < GM / 32; ++i) {
            const int m = m0 + r0 + 32 * i;
            bf16x8 av = {};
            if (m < M) av = *(const bf16x8*)(A + (long long)m * Kd + k0 + 8 * kc);
            if (g) {
#pragma unroll
                for (int e = 0; e < 8; ++e) av[e] = (bf16)((float)av[e] * (float)gv[e]);
            }
            ast[i] = av;
        }
    };
    auto store = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < GN / 32; ++i) *(bf16x8*)(Bs + (r0 + 32 * i) * GP + 8 * kc) = bst[i];
#pragma unroll
        for (int i = 0; i < GM / 32; ++i) *(bf16x8*)(As + (r0 + 32 * i) * GP + 8 * kc) = ast[i];
    };

    const int wm = 128 * (w & 1), wn = 64 * (w >> 1);
    f32x16 acc[4][2];
#pragma unroll
    for (int bi = 0; bi < 4; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[bi][bj][i] = 0.f;

    load(0);
    store();
    __syncthreads();
    const int ro = (lane & 31) * GP + 8 * (lane >> 5);
    for (int k0 = 0; k0 < Kd; k0 += GK) {
        const bool more = k0 + GK < Kd;
        if (more) load(k0 + GK);  // in flight during this step's products
#pragma unroll
        for (int s = 0; s < GK / 16; ++s) {
            bf16x8 bf[2];
#pragma unroll
            for (int bj = 0; bj < 2; ++bj) bf[bj] = *(const bf16x8*)(Bs + (wn + 32 * bj) * GP + ro + 16 * s);
#pragma unroll
            for (int bi = 0; bi < 4; ++bi) {
                const bf16x8 af = *(const bf16x8*)(As + (wm + 32 * bi) * GP + ro + 16 * s);
#pragma unroll
                for (int bj = 0; bj < 2; ++bj) acc[bi][bj] = mfma::mfma32(af, bf[bj], acc[bi][bj]);
            }
        }
        __syncthreads();
        if (more) {
            store();
            __syncthreads();
        }
    }
    // C layout: lane holds C[8 (i / 4) + 4 (lane / 32) + i % 4][lane % 32] of each 32 x 32 block
#pragma unroll
    for (int bi = 0; bi < 4; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int m = m0 + wm + 32 * bi + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
                if (m < M) C[(long long)m * N + n0 + wn + 32 * bj + (lane & 31)] = (CT)acc[bi][bj][i];
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
// (fp32, [T][d] per head): dhat = tau D, dn = g * dhat, c = mean(dn * n),
// dh = r (dn - c n); with a per-module gain also the tile's partial sums of
// dhat * n (tiles of rows rows, those of the local-loss pass).  One workgroup
// per tile of one head; wave w takes the tile's rows w, w + 4, ..., one row at
// a time with lane l on columns 4 l + 256 q .. + 3 (a row's mean is a wave reduction:
// no barrier inside the loop); the row is read twice, the second time from
// cache.  Each wave sums its gain partials in its own LDS row; the four rows
// meet in a fixed order at the end.
typedef float V4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ V4 ld4(const float* p) { return *(const V4*)p; }
__device__ __forceinline__ V4 ld4(const bf16* p) {
    typedef __bf16 b4 __attribute__((ext_vector_type(4)));
    const b4 v = *(const b4*)p;
    return V4{(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
}
__device__ __forceinline__ void st4(float* p, V4 v) { *(V4*)p = v; }
__device__ __forceinline__ void st4(bf16* p, V4 v) {
    typedef __bf16 b4 __attribute__((ext_vector_type(4)));
    *(b4*)p = b4{(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3]};
}

template <typename E>
__global__ __launch_bounds__(256) void k_rot_post(const float* __restrict__ D, const E* __restrict__ h,
                                                 const E* __restrict__ gain, int g_stride, const float* __restrict__ rstd,
                                                 const float* __restrict__ tau, E* __restrict__ dh, float* dgain_part,
                                                 int T, int d, int rows) {
    extern __shared__ __attribute__((aligned(16))) float pbuf[];  // [4][d] when dgain_part is not null
    const int k = blockIdx.y;
    const int tile = blockIdx.x;
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const float tk = tau ? tau[k] : 1.f;
    const E* g = gain + (long long)k * g_stride;
    float* pw = pbuf + w * d;
    if (dgain_part)
        for (int j = lane; j < d; j += 64) pw[j] = 0.f;
    for (int tr = w; tr < rows; tr += 4) {
        const int t = tile * rows + tr;
        if (t >= T) break;
        const long long row = (long long)k * T + t;
        const float r = rstd[row];
        const float* Dr = D + row * d;
        const E* hr = h + row * d;
        // four adjacent columns per lane and access (d % 8 == 0)
        float c = 0.f;
#pragma unroll 4
        for (int j = 4 * lane; j < d; j += 256) {
            const f32x4 dv = *(const f32x4*)(Dr + j);
            const V4 hv = ld4(hr + j), gv = ld4(g + j);
#pragma unroll
            for (int e = 0; e < 4; ++e) c = fmaf(gv[e] * (tk * dv[e]), r * hv[e], c);
        }
        for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off, 64);
        const float cm = c / (float)d;
        E* out = dh + row * d;
#pragma unroll 4
        for (int j = 4 * lane; j < d; j += 256) {
            const f32x4 dv = *(const f32x4*)(Dr + j);
            const V4 hv = ld4(hr + j), gv = ld4(g + j);
            f32x4 o, pv;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float dhat = tk * dv[e];
                const float n = r * hv[e];
                o[e] = r * (gv[e] * dhat - cm * n);
                pv[e] = dhat * n;
            }
            st4(out + j, o);
            if (dgain_part) {
                f32x4 a = *(f32x4*)(pw + j);
#pragma unroll
                for (int e = 0; e < 4; ++e) a[e] += pv[e];
                *(f32x4*)(pw + j) = a;
            }
        }
    }
    if (dgain_part) {
        __syncthreads();
        float* p = dgain_part + ((long long)k * gridDim.x + tile) * d;
        for (int j = threadIdx.x; j < d; j += 256) p[j] = ((pbuf[j] + pbuf[d + j]) + pbuf[2 * d + j]) + pbuf[3 * d + j];
    }
}

}  // namespace

bool rot_back_planes(int dtype, int d) { return dtype == 0 && d % GN == 0 && d % GK == 0; }

// the matrix-core product over all row tiles, in launches of at most 65535 of them
template <typename CT>
hipError_t gemm_mfma(const bf16* A, long long a_mat, int Kd, const bf16* gain, int g_stride, const bf16* B,
                     long long b_mat, int ldb, CT* C, long long c_mat, int nmat, int M, int N, hipStream_t s) {
    const int mtiles = (M + GM - 1) / GM;
    for (int t0 = 0; t0 < mtiles; t0 += 65535) {
        const int nt = mtiles - t0 < 65535 ? mtiles - t0 : 65535;
        dim3 grid((unsigned)(N / GN), (unsigned)nt, (unsigned)nmat);
        hipLaunchKernelGGL(k_gemm_nt_mfma<CT>, grid, dim3(256), 0, s, A, a_mat, Kd, gain, g_stride, B, b_mat, ldb, C,
                           c_mat, M, N, t0);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// the vector-ALU product, one thread per element of C
template <typename AT, typename BT, typename CT>
hipError_t gemm_valu(const AT* A, long long a_mat, const BT* gain, int g_stride, const BT* B, long long b_mat, CT* C,
                     long long c_mat, int nmat, int M, int N, int Kd, hipStream_t s) {
    const long long blocks = ((long long)M * N + 255) / 256;
    if (blocks > 2147483647LL) return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_gemm_nt_valu<AT, BT, CT>), dim3((unsigned)blocks, 1, (unsigned)nmat), dim3(256), 0, s, A,
                       a_mat, gain, g_stride, B, b_mat, C, c_mat, M, N, Kd);
    return hipGetLastError();
}

hipError_t launch_rot_rows(int dtype, const void* h, const void* gain, int g_stride, const void* R, void* u,
                           int nmat, int T, int d, hipStream_t s) {
    const long long td = (long long)T * d, dd = (long long)d * d;
    if (rot_back_planes(dtype, d))
        return gemm_mfma<bf16>((const bf16*)h, td, d, (const bf16*)gain, g_stride, (const bf16*)R, dd, d, (bf16*)u,
                               td, nmat, T, d, s);
    if (dtype == 0)
        return gemm_valu<bf16, bf16, bf16>((const bf16*)h, td, (const bf16*)gain, g_stride, (const bf16*)R, dd,
                                           (bf16*)u, td, nmat, T, d, d, s);
    return gemm_valu<float, float, float>((const float*)h, td, (const float*)gain, g_stride, (const float*)R, dd,
                                          (float*)u, td, nmat, T, d, d, s);
}

hipError_t launch_rot_back(int dtype, bool planes, const void* e, const void* Rt, float* D, int nmat, int T, int d,
                           hipStream_t s) {
    const long long td = (long long)T * d, dd = (long long)d * d;
    if (planes) {
        if (!rot_back_planes(dtype, d)) return hipErrorInvalidValue;
        return gemm_mfma<float>((const bf16*)e, 2 * td, 2 * d, nullptr, 0, (const bf16*)Rt, dd, d, D, td, nmat, T, d,
                                s);
    }
    if (dtype == 0)
        return gemm_valu<float, bf16, float>((const float*)e, td, nullptr, 0, (const bf16*)Rt, dd, D, td, nmat, T, d,
                                             d, s);
    return gemm_valu<float, float, float>((const float*)e, td, nullptr, 0, (const float*)Rt, dd, D, td, nmat, T, d, d,
                                          s);
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
    const size_t lds = dgain_part ? (size_t)4 * d * 4 : 0;
    if (dtype == 0)
        hipLaunchKernelGGL(k_rot_post<bf16>, grid, dim3(256), lds, s, D, (const bf16*)h, (const bf16*)gain, g_stride,
                           rstd, tau, (bf16*)dh, dgain_part, T, d, rows);
    else
        hipLaunchKernelGGL(k_rot_post<float>, grid, dim3(256), lds, s, D, (const float*)h, (const float*)gain,
                           g_stride, rstd, tau, (float*)dh, dgain_part, T, d, rows);
    return hipGetLastError();
}

}  // namespace solo
