// Vector-ALU versions of the fused passes (fp32 arithmetic on fp32 or bf16
// storage).  They serve the fp32 configuration, where the products must be
// true fp32 products, and bf16 widths that the matrix-core kernels do not
// tile.  Same passes and notation as k_mfma.hip (z_tv = tau_k <R_kv, hhat_t> + b_kv,
// hhat = g_k * r_t h_t): a tile of stationary rows stays in LDS, the other
// operand streams in chunks, the T x V logits are never written.
//
//   local-loss pass: 8 rows t with hhat in LDS; online max / sum-exp over the
//     readout rows; acc_t += sum_v exp(z_tv - m_t) R_kv; dhat, the RMSNorm
//     backward and the tile's gain-gradient partial at the end.
//   exit evaluation: the same without the second product, plus the top-1.
//   readout-gradient pass: 8 readout rows v (times g_k); delta from the stored
//     lse; D_v += sum_t delta_tv tau r_t h_t; dR_v = g_k * D_v; db_v = sum_t delta_tv.
//   bias-gradient pass: the same without the second product.
#include "solo_internal.h"

namespace solo {

namespace {

constexpr int RX = kValuRows;  // stationary rows per workgroup (8)
constexpr int YC = 64;         // streamed rows per chunk
constexpr int NTHR = 256;
constexpr int NQ = 16;         // columns per thread: j = tid + 256 q, d <= 4096

enum Mode { LOCAL = 0, RGRAD = 1, BGRAD = 2, EVAL = 3 };

__device__ __forceinline__ float ld(const float* p, long long i) { return p[i]; }
__device__ __forceinline__ float ld(const bf16* p, long long i) { return (float)p[i]; }
template <typename E> __device__ __forceinline__ void st(E* p, long long i, float v);
template <> __device__ __forceinline__ void st<float>(float* p, long long i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void st<bf16>(bf16* p, long long i, float v) { p[i] = (bf16)v; }

template <typename E, int MODE>
__global__ __launch_bounds__(NTHR) void k_fused_valu(FusedArgs a) {
    constexpr bool LL = MODE == LOCAL || MODE == EVAL;   // X = hhat, Y = readout
    constexpr bool PC = MODE == LOCAL || MODE == RGRAD;  // second product
    extern __shared__ __attribute__((aligned(16))) float sm[];
    const int d = a.d;
    float* xs = sm;                    // [RX][d] stationary rows (fp32)
    float* sS = xs + RX * d;           // [RX][YC] logits, then probabilities / deltas
    float* sc = sS + RX * YC;          // [RX] alpha, then 1/s
    float* sy = sc + RX;               // [4][YC] per-streamed-row scalars (readout-/bias-gradient passes)
    float* red = sy + 4 * YC;          // [RX][NTHR/64] reductions
    float* spy = red + RX * (NTHR / 64);  // [RX] p_y - 1 of the local-loss rows

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wv = tid >> 6;
    const int x0 = blockIdx.x * RX;
    const int k = a.m0 + (int)blockIdx.y;
    const long long modoff = (long long)k * a.T;
    const float tau = a.tau ? a.tau[k] : 1.f;
    const E* hk = (const E*)a.h + modoff * d;
    const E* Rk = k == a.K - 1 ? (const E*)a.Wt : (const E*)a.Wh + (long long)k * a.wh_stride;
    const E* gk = (const E*)a.gain + (long long)k * a.g_stride;
    const float* bk = a.bias ? a.bias + (long long)k * a.V : nullptr;
    const E* Y = LL ? Rk : hk;
    const int nX = LL ? a.T : a.V;
    const int nY = LL ? a.V : a.T;

    // stationary tile: LL -> hhat_t = g r_t h_t ; otherwise g * R_v
    for (int i = tid; i < RX * d; i += NTHR) {
        const int r = i / d, j = i - r * d;
        const int xg = x0 + r;
        float v = 0.f;
        if (xg < nX) {
            if (LL) v = ld(gk, j) * a.rstd[modoff + xg] * ld(hk, (long long)xg * d + j);
            else v = ld(gk, j) * ld(Rk, (long long)xg * d + j);
        }
        xs[i] = v;
    }

    float acc[PC ? RX : 1][NQ];
#pragma unroll
    for (int r = 0; r < (PC ? RX : 1); ++r)
#pragma unroll
        for (int q = 0; q < NQ; ++q) acc[r][q] = 0.f;

    // elementwise step: thread (sr = tid/32, sq = tid%32) handles columns sq and sq + 32 of row sr
    const int sr = tid >> 5;
    const int sq = tid & 31;
    float m_run = -INFINITY, s_run = 0.f, zy = 0.f;
    float best = -INFINITY;
    int best_v = -1;
    float dbp = 0.f;
    int own_tgt = -1;
    if (LL && x0 + sr < nX) own_tgt = a.targets[modoff + x0 + sr];
    const float bx = (!LL && bk && x0 + sr < nX) ? bk[x0 + sr] : 0.f;
    __syncthreads();

    for (int y0 = 0; y0 < nY; y0 += YC) {
        if (!LL && tid < YC) {
            const int yg = y0 + tid;
            const bool ok = yg < nY;
            sy[tid] = ok ? a.rstd[modoff + yg] : 0.f;
            sy[YC + tid] = ok ? a.lse[modoff + yg] : 0.f;
            sy[2 * YC + tid] = ok ? __int_as_float(a.targets[modoff + yg]) : __int_as_float(-1);
            // the exact p_y - 1 of the local-loss pass (the target's entry of delta)
            sy[3 * YC + tid] = ok ? a.rowrec[4 * (modoff + yg) + 3] : 0.f;
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
                for (int r = 0; r < RX; ++r) sS[r * YC + yy] = part[r];
            }
        }
        __syncthreads();

        if (LL) {
            float u[2], z[2];
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
                const int yg = y0 + sq + 32 * hh;
                u[hh] = sS[sr * YC + sq + 32 * hh];
                z[hh] = (yg < nY) ? tau * u[hh] + (bk ? bk[yg] : 0.f) : -INFINITY;
                if (MODE == EVAL && z[hh] > best) {  // columns come in increasing order: ties keep the first
                    best = z[hh];
                    best_v = yg;
                }
                if (yg == own_tgt) zy = z[hh];
            }
            float cmax = fmaxf(z[0], z[1]);
            for (int off = 16; off > 0; off >>= 1) cmax = fmaxf(cmax, __shfl_xor(cmax, off, 32));
            const float m_new = fmaxf(m_run, cmax);
            const float alpha = __expf(m_run - m_new);
            m_run = m_new;
            // the target's term joins the running sum only at the end of the row,
            // and its probability the input gradient only in the epilogue
            const float p0 = (z[0] == -INFINITY || y0 + sq == own_tgt) ? 0.f : __expf(z[0] - m_run);
            const float p1 = (z[1] == -INFINITY || y0 + sq + 32 == own_tgt) ? 0.f : __expf(z[1] - m_run);
            float ps = p0 + p1;
            for (int off = 16; off > 0; off >>= 1) ps += __shfl_xor(ps, off, 32);
            s_run = s_run * alpha + ps;
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
                    const float p = __expf(tau * ry * sS[sr * YC + yy] + bx - sy[YC + yy]);
                    const int tg = __float_as_int(sy[2 * YC + yy]);
                    const float dl = tg == xg ? sy[3 * YC + yy] : p;
                    dbp += dl;
                    g = dl * ry * tau * a.inv_T;
                }
                sS[sr * YC + yy] = g;
            }
        }
        __syncthreads();

        if (PC) {
            // second product: thread owns columns j = tid + 256 q of all RX rows
            if (MODE == LOCAL) {
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
                        for (int r = 0; r < RX; ++r) acc[PC ? r : 0][q] = fmaf(sS[r * YC + yy], yv, acc[PC ? r : 0][q]);
                    }
                }
            }
        }
        __syncthreads();
    }

    if (LL) {
        // finish rows: lse, row loss, top-1; the target logit sits in one thread of the row group
        for (int off = 16; off > 0; off >>= 1) {
            zy += __shfl_xor(zy, off, 32);
            if (MODE == EVAL) {
                const float ob = __shfl_xor(best, off, 32);
                const int ov = __shfl_xor(best_v, off, 32);
                if (ob > best || (ob == best && (unsigned)ov < (unsigned)best_v)) {
                    best = ob;
                    best_v = ov;
                }
            }
        }
        if (sq == 0) {
            // s_run holds every column but the target's: adding the target's term
            // here gives p_y - 1 = -s_run / s and the row loss without cancellation
            const bool tok = own_tgt >= 0 && own_tgt < nY;
            const float ey = tok ? __expf(zy - m_run) : 0.f;
            const float s = s_run + ey;
            const float lse = m_run + logf(s);
            const float py1 = tok ? -s_run / s : 0.f;
            if (x0 + sr < nX) {
                const long long t = modoff + x0 + sr;
                a.lse[t] = lse;
                a.rowloss[t] = !tok ? __int_as_float(0x7fc00000) : (ey > s_run ? log1pf(s_run / ey) : (m_run - zy) + logf(s));
                if (MODE == EVAL && a.top1) a.top1[t] = best_v;
                if (MODE == LOCAL && a.rowrec) a.rowrec[4 * t + 3] = py1;
            }
            sc[sr] = 1.f / s;
            spy[sr] = py1;
        }
        __syncthreads();
    }
    if (MODE == LOCAL) {
        // e = (acc / s - R_y) / T, dhat = tau e, dn = g dhat; the row sum of
        // e g n is both tau^-1 d mean(dn n) and the token's d loss / d tau
        // (sum_v delta_v u_v = <sum_v delta_v R_v, g n>); dh = r (dn - c n)
        const bool want_dg = a.dg_mode == 2 || (a.dg_mode == 1 && k == a.K - 1);
        float dgp[NQ];
#pragma unroll
        for (int q = 0; q < NQ; ++q) dgp[q] = 0.f;
        float cp[RX];
#pragma unroll
        for (int r = 0; r < RX; ++r) {
            const int xg = x0 + r;
            const int tg = (xg < nX) ? a.targets[modoff + xg] : -1;
            const bool tok = tg >= 0 && tg < nY;
            const float rx = (xg < nX) ? a.rstd[modoff + xg] : 0.f;
            cp[r] = 0.f;
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const int j = tid + NTHR * q;
                if (j < d) {
                    const float wy = tok ? ld(Rk, (long long)tg * d + j) : 0.f;
                    const float ev = fmaf(acc[r][q], sc[r], spy[r] * wy) * a.inv_T;
                    const float n = (xg < nX) ? rx * ld(hk, (long long)xg * d + j) : 0.f;
                    const float gj = ld(gk, j);
                    acc[r][q] = a.ebuf ? ev : tau * gj * ev;  // dn (e itself for the buffer)
                    cp[r] = fmaf(gj * ev, n, cp[r]);
                    dgp[q] = fmaf(tau * ev, n, dgp[q]);
                }
            }
            float v = cp[r];
            for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
            if (lane == 0) red[r * (NTHR / 64) + wv] = v;
        }
        if (want_dg) {
            float* part = a.dgain_part + ((long long)(a.dg_mode == 2 ? k : 0) * gridDim.x + blockIdx.x) * d;
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const int j = tid + NTHR * q;
                if (j < d) part[j] = dgp[q];
            }
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < RX; ++r) {
            const int xg = x0 + r;
            if (xg >= nX) continue;
            float csum = 0.f;
            for (int i = 0; i < NTHR / 64; ++i) csum += red[r * (NTHR / 64) + i];
            const float cmean = tau * csum / (float)d;
            if (a.rowdtau && tid == 0) {
                const int tg = a.targets[modoff + xg];
                a.rowdtau[modoff + xg] = (tg >= 0 && tg < nY) ? csum : 0.f;
            }
            if (a.ebuf) {
                // e to the buffer; the RMSNorm backward follows the rotation back (ROT heads)
#pragma unroll
                for (int q = 0; q < NQ; ++q) {
                    const int j = tid + NTHR * q;
                    if (j < d) ((float*)a.ebuf)[(modoff + xg) * (long long)d + j] = acc[r][q];
                }
                continue;
            }
            const float rx = a.rstd[modoff + xg];
            E* out = (E*)a.dh + (modoff + xg) * (long long)d;
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const int j = tid + NTHR * q;
                if (j < d) st<E>(out, j, rx * (acc[r][q] - cmean * rx * ld(hk, (long long)xg * d + j)));
            }
        }
    }
    if (!LL) {
        // bias gradient of readout row sr: sum over the 32 threads of the row group
        for (int off = 16; off > 0; off >>= 1) dbp += __shfl_xor(dbp, off, 32);
        if (a.dbias && sq == 0 && x0 + sr < nX) a.dbias[(long long)k * a.V + x0 + sr] = dbp * a.inv_T;
    }
    if (MODE == RGRAD) {
        float* dR = (k == a.K - 1) ? a.dWt : a.dWh + (long long)k * a.V * d;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int j = tid + NTHR * q;
            if (j >= d) continue;
            const float gj = ld(gk, j);
#pragma unroll
            for (int r = 0; r < RX; ++r) {
                const int v = x0 + r;
                if (v < nX) dR[(long long)v * d + j] = gj * acc[PC ? r : 0][q];
            }
        }
    }
}

template <typename E, int MODE>
hipError_t launch_t(const FusedArgs& a, int nmod, hipStream_t s) {
    const size_t lds = sizeof(float) * ((size_t)RX * a.d + RX * YC + RX + 4 * YC + RX * (NTHR / 64) + RX);
    hipError_t e = hipFuncSetAttribute((const void*)k_fused_valu<E, MODE>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds);
    if (e != hipSuccess) return e;
    const bool ll = MODE == LOCAL || MODE == EVAL;
    dim3 grid = ll ? dim3((unsigned)((a.T + RX - 1) / RX), (unsigned)nmod)
                   : dim3((unsigned)((a.V + RX - 1) / RX), (unsigned)nmod);
    hipLaunchKernelGGL((k_fused_valu<E, MODE>), grid, dim3(NTHR), lds, s, a);
    return hipGetLastError();
}

template <int MODE>
hipError_t launch_dt(int dtype, const FusedArgs& a, int nmod, hipStream_t s) {
    return dtype == 0 ? launch_t<bf16, MODE>(a, nmod, s) : launch_t<float, MODE>(a, nmod, s);
}

}  // namespace

hipError_t launch_local_loss_valu(int dtype, const FusedArgs& a, int nmod, hipStream_t s) {
    return launch_dt<LOCAL>(dtype, a, nmod, s);
}
hipError_t launch_exit_eval_valu(int dtype, const FusedArgs& a, int nmod, hipStream_t s) {
    return launch_dt<EVAL>(dtype, a, nmod, s);
}
hipError_t launch_readout_grad_valu(int dtype, const FusedArgs& a, int nmod, hipStream_t s) {
    return launch_dt<RGRAD>(dtype, a, nmod, s);
}
hipError_t launch_bias_grad_valu(int dtype, const FusedArgs& a, int nmod, hipStream_t s) {
    return launch_dt<BGRAD>(dtype, a, nmod, s);
}

}  // namespace solo
