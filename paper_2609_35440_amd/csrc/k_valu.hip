// Vector-ALU versions of the two fused passes (fp32 arithmetic on fp32 or
// bf16 storage).  They serve the fp32 configuration, where the products must
// be true fp32 products, and bf16 widths that the matrix-core kernels do not
// tile.  Same structure as the matrix-core passes: a tile of stationary rows
// stays in LDS/registers, the other operand streams in chunks, the T x V
// logits are never written.
//
//   local-loss pass: 8 rows t of h_k; online max / sum-exp over the readout
//     rows; acc_t += sum_v exp(z_tv - m_t) Wg_v; RMSNorm backward at the end.
//   readout-gradient pass: 8 readout rows v; delta from the stored lse;
//     D_v += sum_t delta_tv r_t h_t; dW_v = gain * D_v; dgain partial W_v * D_v.
#include "solo_internal.h"

namespace solo {

namespace {

constexpr int RX = kValuRows;  // stationary rows per workgroup (8)
constexpr int YC = 64;         // streamed rows per chunk
constexpr int NTHR = 256;
constexpr int NQ = 16;         // columns per thread: j = tid + 256 q, d <= 4096

__device__ __forceinline__ float ld(const float* p, long long i) { return p[i]; }
__device__ __forceinline__ float ld(const bf16* p, long long i) { return (float)p[i]; }
template <typename E> __device__ __forceinline__ void st(E* p, long long i, float v);
template <> __device__ __forceinline__ void st<float>(float* p, long long i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void st<bf16>(bf16* p, long long i, float v) { p[i] = (bf16)v; }

template <typename E, int MODE>
__global__ __launch_bounds__(NTHR) void k_fused_valu(FusedArgs a) {
    extern __shared__ __attribute__((aligned(16))) float sm[];
    const int d = a.d;
    float* xs = sm;                    // [RX][d] stationary rows (fp32)
    float* sS = xs + RX * d;           // [RX][YC] logits, then probabilities / deltas
    float* sc = sS + RX * YC;          // [RX] alpha, then 1/s
    float* sy = sc + RX;               // [3][YC] per-streamed-row scalars (MODE 1)
    float* red = sy + 3 * YC;          // [RX][NTHR/64] reductions

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wv = tid >> 6;
    const int x0 = blockIdx.x * RX;
    const int k = (MODE == 0) ? (int)blockIdx.y : a.K - 1;
    const long long modoff = (long long)k * a.T;
    const E* hk = (const E*)a.h + modoff * d;
    const E* Wg = (const E*)a.Wg;
    const E* Y = (MODE == 0) ? Wg : hk;
    const int nX = (MODE == 0) ? a.T : a.V;
    const int nY = (MODE == 0) ? a.V : a.T;

    // stationary tile: MODE 0 -> n_t = r_t h_t ; MODE 1 -> Wg_v
    for (int i = tid; i < RX * d; i += NTHR) {
        const int r = i / d, j = i - r * d;
        const int xg = x0 + r;
        float v = 0.f;
        if (xg < nX) {
            if (MODE == 0) v = a.rstd[modoff + xg] * ld(hk, (long long)xg * d + j);
            else v = ld(Wg, (long long)xg * d + j);
        }
        xs[i] = v;
    }

    float acc[RX][NQ];
#pragma unroll
    for (int r = 0; r < RX; ++r)
#pragma unroll
        for (int q = 0; q < NQ; ++q) acc[r][q] = 0.f;

    // online softmax state (MODE 0): thread (r = tid/32) keeps row r's copy
    const int sr = tid >> 5;          // row handled in the elementwise step
    const int sq = tid & 31;          // columns sq and sq + 32 of the chunk
    float m_run = -INFINITY, s_run = 0.f, zy = 0.f;
    int own_tgt = -1;
    if (MODE == 0 && x0 + sr < nX) own_tgt = a.targets[modoff + x0 + sr];
    __syncthreads();

    for (int y0 = 0; y0 < nY; y0 += YC) {
        if (MODE == 1 && tid < YC) {
            const int yg = y0 + tid;
            const bool ok = yg < nY;
            sy[tid] = ok ? a.rstd[modoff + yg] : 0.f;
            sy[YC + tid] = ok ? a.lse[modoff + yg] : 0.f;
            sy[2 * YC + tid] = ok ? __int_as_float(a.targets[modoff + yg]) : __int_as_float(-1);
        }
        // logits: wave wv handles streamed rows y0 + 16 wv .. +15; lanes split j
        for (int yy = 16 * wv; yy < 16 * wv + 16; ++yy) {
            const int yg = y0 + yy;
            float part[RX];
#pragma unroll
            for (int r = 0; r < RX; ++r) part[r] = 0.f;
            if (yg < nY) {
                const E* yrow = Y + (long long)yg * d;
                for (int j = lane; j < d; j += 64) {
                    const float yv = ld(yrow, j);
#pragma unroll
                    for (int r = 0; r < RX; ++r) part[r] = fmaf(xs[r * d + j], yv, part[r]);
                }
            }
#pragma unroll
            for (int r = 0; r < RX; ++r) {
                float v = part[r];
                for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
                part[r] = v;
            }
            if (lane == 0) {
#pragma unroll
                for (int r = 0; r < RX; ++r) sS[r * YC + yy] = (yg < nY) ? part[r] : -INFINITY;
            }
        }
        __syncthreads();

        // elementwise step: thread (sr, sq) handles columns sq, sq + 32 of row sr
        if (MODE == 0) {
            const float z0 = sS[sr * YC + sq], z1 = sS[sr * YC + sq + 32];
            float cmax = fmaxf(z0, z1);
            for (int off = 16; off > 0; off >>= 1) cmax = fmaxf(cmax, __shfl_xor(cmax, off, 32));
            const float m_new = fmaxf(m_run, cmax);
            const float alpha = __expf(m_run - m_new);
            m_run = m_new;
            const float p0 = (z0 == -INFINITY) ? 0.f : __expf(z0 - m_run);
            const float p1 = (z1 == -INFINITY) ? 0.f : __expf(z1 - m_run);
            float ps = p0 + p1;
            for (int off = 16; off > 0; off >>= 1) ps += __shfl_xor(ps, off, 32);
            s_run = s_run * alpha + ps;
            if (y0 + sq == own_tgt) zy = z0;
            if (y0 + sq + 32 == own_tgt) zy = z1;
            sS[sr * YC + sq] = p0;
            sS[sr * YC + sq + 32] = p1;
            if (sq == 0) sc[sr] = alpha;
        } else {
            const int xg = x0 + sr;
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
                const int yy = sq + 32 * hh;
                const int yg = y0 + yy;
                float g = 0.f;
                if (yg < nY && xg < nX) {
                    const float ry = sy[yy];
                    const float p = __expf(sS[sr * YC + yy] * ry - sy[YC + yy]);
                    const int tg = __float_as_int(sy[2 * YC + yy]);
                    g = (p - (tg == xg ? 1.f : 0.f)) * ry * a.inv_T;
                }
                sS[sr * YC + yy] = g;
            }
        }
        __syncthreads();

        // second product: thread owns columns j = tid + 256 q of all RX rows
        if (MODE == 0) {
#pragma unroll
            for (int r = 0; r < RX; ++r) {
                const float al = sc[r];
#pragma unroll
                for (int q = 0; q < NQ; ++q) acc[r][q] *= al;
            }
        }
        const int yend = (nY - y0) < YC ? (nY - y0) : YC;
        for (int yy = 0; yy < yend; ++yy) {
            const E* yrow = Y + (long long)(y0 + yy) * d;
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const int j = tid + NTHR * q;
                if (j < d) {
                    const float yv = ld(yrow, j);
#pragma unroll
                    for (int r = 0; r < RX; ++r) acc[r][q] = fmaf(sS[r * YC + yy], yv, acc[r][q]);
                }
            }
        }
        __syncthreads();
    }

    if (MODE == 0) {
        // finish rows: lse, row loss, 1/s (the target logit sits in one thread of the row group)
        for (int off = 16; off > 0; off >>= 1) zy += __shfl_xor(zy, off, 32);
        if (sq == 0) {
            const float lse = m_run + logf(s_run);
            const bool tok = own_tgt >= 0 && own_tgt < nY;
            if (x0 + sr < nX) {
                a.lse[modoff + x0 + sr] = lse;
                a.rowloss[modoff + x0 + sr] = tok ? lse - zy : __int_as_float(0x7fc00000);
            }
            sc[sr] = 1.f / s_run;
        }
        __syncthreads();
        // dn = (acc / s - Wg[y]) / T; c = mean(dn * n); dh = r (dn - c n)
        float cp[RX];
#pragma unroll
        for (int r = 0; r < RX; ++r) {
            const int xg = x0 + r;
            const int tg = (xg < nX) ? a.targets[modoff + xg] : -1;
            const bool tok = tg >= 0 && tg < nY;
            cp[r] = 0.f;
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const int j = tid + NTHR * q;
                if (j < d) {
                    const float wy = tok ? ld(Wg, (long long)tg * d + j) : 0.f;
                    const float dn = (acc[r][q] * sc[r] - wy) * a.inv_T;
                    acc[r][q] = dn;
                    cp[r] = fmaf(dn, xs[r * d + j], cp[r]);
                }
            }
            float v = cp[r];
            for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
            if (lane == 0) red[r * (NTHR / 64) + wv] = v;
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < RX; ++r) {
            const int xg = x0 + r;
            if (xg >= nX) continue;
            float csum = 0.f;
            for (int i = 0; i < NTHR / 64; ++i) csum += red[r * (NTHR / 64) + i];
            const float cmean = csum / (float)d;
            const float rx = a.rstd[modoff + xg];
            E* out = (E*)a.dh + (modoff + xg) * (long long)d;
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const int j = tid + NTHR * q;
                if (j < d) st<E>(out, j, rx * (acc[r][q] - cmean * xs[r * d + j]));
            }
        }
    } else {
        const E* W = (const E*)a.W;
        const E* gain = (const E*)a.gain;
        float* dgp = a.dgain_part + (long long)blockIdx.x * d;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int j = tid + NTHR * q;
            if (j >= d) continue;
            const float gj = ld(gain, j);
            float pr = 0.f;
#pragma unroll
            for (int r = 0; r < RX; ++r) {
                const int v = x0 + r;
                if (v < nX) {
                    a.dW[(long long)v * d + j] = gj * acc[r][q];
                    pr = fmaf(ld(W, (long long)v * d + j), acc[r][q], pr);
                }
            }
            dgp[j] = pr;
        }
    }
}

template <typename E, int MODE>
hipError_t launch_t(const FusedArgs& a, hipStream_t s) {
    const size_t lds = sizeof(float) * ((size_t)RX * a.d + RX * YC + RX + 3 * YC + RX * (NTHR / 64));
    hipError_t e = hipFuncSetAttribute((const void*)k_fused_valu<E, MODE>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds);
    if (e != hipSuccess) return e;
    dim3 grid = (MODE == 0) ? dim3((unsigned)((a.T + RX - 1) / RX), (unsigned)a.K) : dim3((unsigned)((a.V + RX - 1) / RX));
    hipLaunchKernelGGL((k_fused_valu<E, MODE>), grid, dim3(NTHR), lds, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_local_loss_valu(int dtype, const FusedArgs& a, hipStream_t s) {
    return dtype == 0 ? launch_t<bf16, 0>(a, s) : launch_t<float, 0>(a, s);
}
hipError_t launch_readout_grad_valu(int dtype, const FusedArgs& a, hipStream_t s) {
    return dtype == 0 ? launch_t<bf16, 1>(a, s) : launch_t<float, 1>(a, s);
}

}  // namespace solo
