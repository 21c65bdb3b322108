// Fused matrix-core passes of the SOLO shared-readout loss (bf16 operands, fp32
// accumulate) for gfx950.
//
// Both passes have the shape "logit tile -> elementwise -> second product":
//
//   local-loss pass (every module, Eq. 2 and Eq. 3 of the paper):
//     stationary X = 32 rows t of h_k, streamed Y = the readout rows v,
//     z_tv = r_t <Wg_v, h_t>, online (max, sum-exp) per row, and
//     acc_t += sum_v exp(z_tv - m_t) Wg_v        (Wg = W diag(gain))
//     so that dn_t = (acc_t / s_t - Wg_{y_t}) / T at the end, followed by the
//     RMSNorm backward.  The T x V logits and probabilities stay on chip.
//
//   readout-gradient pass (final module only; the copies get no gradient):
//     stationary X = 32 readout rows v, streamed Y = the rows t of h_{K-1},
//     delta_tv = (exp(z_tv - lse_t) - [v = y_t]) / T and
//     D_v += sum_t delta_tv r_t h_t,  dW_v = gain * D_v,  dgain += W_v * D_v.
//
// Work split: a workgroup of 8 waves owns the 32 stationary rows; wave w owns
// the d/8 columns [w d/8, (w+1) d/8).  Per chunk of 16 streamed rows, every
// wave multiplies its column slice (split-K partial of the logit tile), the
// partials meet in LDS, each wave finishes the elementwise step for 4 of the
// 32 stationary rows, and every wave then accumulates its own column slice of
// the second product.  The accumulator (32 rows x d/8 columns, fp32) and the
// stationary operand stay in registers for the whole pass; the streamed
// chunk goes HBM/L2 -> LDS directly and is read twice from LDS: row-wise for
// the logit product and with the transposing read for the second product.
#include "mfma_common.h"

namespace solo {

namespace {

using namespace mfma;

constexpr int NW = layout::NW;  // waves per workgroup
constexpr int NTHR = NW * 64;
constexpr int XR = kMfmaRows;  // stationary rows per workgroup (32)
constexpr int YC = layout::YC;  // streamed rows per chunk
constexpr int PP = 20;       // row pitch (floats) of the partial logit tiles: conflict-free 16 B writes

template <int DS>
struct Geo : layout::Geo<DS> {
    static constexpr int NB = DS / 32;                 // 32-column accumulator blocks per wave
    static constexpr int NK = DS / 32;                 // 32-deep k-steps of the logit product
    static constexpr int YBUF = NW * layout::Geo<DS>::SLICE;  // one chunk buffer (all waves)
    static constexpr int TOTAL = 2 * YBUF + NW * XR * PP * 4 + XR * YC * 2 + 2 * XR * 4 + NW * XR * 4;
    static_assert(TOTAL <= 160 * 1024, "LDS budget");
};

// MODE 0: local-loss pass, grid (ceil(T/32), K).
// MODE 1: readout-gradient pass of module K-1, grid (ceil(V/32)).
template <int MODE, int DS>
__global__ __launch_bounds__(NTHR, 1) void k_fused(FusedArgs a) {
    using G = Geo<DS>;
    // the stream of a chunk is issued in batches [0, kDma1), [kDma1, kDma2), [kDma2, NI)
    constexpr int kDma1 = (3 * G::NI + 7) / 8, kDma2 = (6 * G::NI + 7) / 8;
    // Separate LDS objects, so that the compiler can tell the chunk being read
    // from the chunk being prefetched (no needless waits on the prefetch).
    __shared__ __attribute__((aligned(16))) char ybufA[G::YBUF];
    __shared__ __attribute__((aligned(16))) char ybufB[G::YBUF];
    __shared__ __attribute__((aligned(16))) float part[NW * XR * PP];
    __shared__ __attribute__((aligned(16))) bf16 gbuf[XR * YC];
    __shared__ float abuf[XR];
    __shared__ float sbuf[XR];
    __shared__ float cbuf[NW * XR];
    __shared__ __attribute__((aligned(16))) float recA[YC * 4];  // readout-gradient pass: per-token records
    __shared__ __attribute__((aligned(16))) float recB[YC * 4];

    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int d = a.d;
    const int js = w * DS;
    const int x0 = blockIdx.x * XR;
    const int k = (MODE == 0) ? (int)blockIdx.y : a.K - 1;
    const long long modoff = (long long)k * a.T;

    const bf16* __restrict__ hk = (const bf16*)a.h + modoff * d;
    const bf16* __restrict__ Wg = (const bf16*)a.Wg;
    const bf16* __restrict__ X = (MODE == 0) ? hk : Wg;
    const bf16* __restrict__ Y = (MODE == 0) ? Wg : hk;
    const int nX = (MODE == 0) ? a.T : a.V;
    const int nY = (MODE == 0) ? a.V : a.T;
    const int nchunks = (nY + YC - 1) / YC;

    LDS_AS char* sliceA = (LDS_AS char*)(LDS_AS void*)ybufA + w * G::SLICE;
    LDS_AS char* sliceB = (LDS_AS char*)(LDS_AS void*)ybufB + w * G::SLICE;

    // per-lane scalars of the rows this wave finishes in the elementwise step
    const int xo = 4 * w + (lane >> 4);   // stationary row (0..31) owned in the elementwise step
    const int yy = lane & 15;             // streamed row within the chunk
    float own_r = 0.f;                    // MODE 0: r_t of row xo
    int own_tgt = -1;                     // MODE 0: target of row xo
    if (MODE == 0 && x0 + xo < nX) {
        own_r = a.rstd[modoff + x0 + xo];
        own_tgt = a.targets[modoff + x0 + xo];
    }
    const float own_r2 = own_r * kLog2e;

    ChunkStream<DS> stream;
    stream.init(d, js, lane);
    // first chunk in flight before the stationary operand is read
    const unsigned sliceA_u = lds_addr(sliceA), sliceB_u = lds_addr(sliceB);
    stream.issue(Y, nY, d, 0, sliceA_u);
    // readout-gradient pass: the 16 per-token records {lse, rstd, target, 0}
    // of a chunk stream into recA / recB next to the chunk itself
    const unsigned recA_u = lds_addr((LDS_AS char*)(LDS_AS void*)recA);
    const unsigned recB_u = lds_addr((LDS_AS char*)(LDS_AS void*)recB);
    auto issue_rec = [&](int y0, unsigned dst) __attribute__((always_inline)) {
        if (MODE == 1 && w == 0 && lane < YC) {
            const int rows = nY - y0;
            const unsigned rem = rows > 0 ? (unsigned)rows * 16u : 0u;
            buffer_load_lds16(make_rsrc(a.rowrec + 4 * (long long)y0, rem), dst, lane * 16);
        }
    };
    issue_rec(0, recA_u);

    // stationary operand: B of the 16x16x32 logit product, lane holds
    // X[x0 + 16 xb + lane%16][js + 32 kk + 8 (lane/16) .. +7]
    bf16x8 xr[2][G::NK];
#pragma unroll
    for (int xb = 0; xb < 2; ++xb) {
        const int xrow = x0 + 16 * xb + (lane & 15);
#pragma unroll
        for (int kk = 0; kk < G::NK; ++kk) {
            if (xrow < nX) {
                xr[xb][kk] = *(const bf16x8*)(X + (long long)xrow * d + js + 32 * kk + 8 * (lane >> 4));
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e) xr[xb][kk][e] = (bf16)0.f;
            }
        }
    }

    f32x16 acc[G::NB];
#pragma unroll
    for (int b = 0; b < G::NB; ++b)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[b][i] = 0.f;

    // online softmax state (MODE 0, base 2), per lane: row xo, streamed column yy
    float m_run = -INFINITY, s_part = 0.f, zy_part = 0.f;

    // per-lane parts of the LDS addresses; the unrolled loops add 64 * kk or 64 * b
    const int a_off = layout::rowread_off<DS>(lane);
    const int c_lo = layout::trread_off<DS>(lane, 0);
    const int c_hi = layout::trread_off<DS>(lane, 1);

    auto step = [&](LDS_AS char* cur, unsigned nxt, LDS_AS float* rec, unsigned rec_nxt, int c)
                    __attribute__((always_inline)) {
        const int y0 = c * YC;
        const bool more = c + 1 < nchunks;
        const i32x4 nrs = ChunkStream<DS>::rsrc(Y, nY, d, y0 + YC);

        // ---- split-K partial of the logit tile S[y][x] over this wave's columns.
        // All operand reads go out first, ahead of the data of the next chunk,
        // whose stream is issued in three batches (here, after these products
        // and after the elementwise step) so that neither the texture unit's
        // queue nor the LDS write port sees the whole chunk at once.
        bf16x8 ay[G::NK];
#pragma unroll
        for (int kk = 0; kk < G::NK; ++kk) ay[kk] = *(LDS_AS bf16x8*)(cur + a_off + 64 * kk);
        if (more) {
            stream.template issue_range<0, kDma1>(nrs, d, nxt);
            issue_rec(y0 + YC, rec_nxt);
        }
        f32x4 S0 = {0.f, 0.f, 0.f, 0.f}, S1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < G::NK; ++kk) {
            S0 = mfma16(ay[kk], xr[0][kk], S0);
            S1 = mfma16(ay[kk], xr[1][kk], S1);
        }
        if (more) stream.template issue_range<kDma1, kDma2>(nrs, d, nxt);
        // C layout: lane holds S[y = 4 (lane/16) + i][x = 16 xb + lane%16]; store as part[w][x][y]
        *(f32x4*)(part + (w * XR + (lane & 15)) * PP + 4 * (lane >> 4)) = S0;
        *(f32x4*)(part + (w * XR + 16 + (lane & 15)) * PP + 4 * (lane >> 4)) = S1;
        lds_barrier();

        // ---- elementwise step for rows xo = 4w .. 4w+3 (lane: row xo, column yy)
        float q[NW];
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) q[ww] = part[(ww * XR + xo) * PP + yy];
        static_assert(NW == 8, "partial-sum tree");
        const float sxy = ((q[0] + q[1]) + (q[2] + q[3])) + ((q[4] + q[5]) + (q[6] + q[7]));
        const int yg = y0 + yy;
        float gval;
        if (MODE == 0) {
            // columns past the end of the vocabulary get z = -inf (an additive
            // mask rather than a branch, so the partial reads stay unconditional)
            const float ymask = (yg < nY) ? 0.f : -INFINITY;
            const float zc = __builtin_fmaf(sxy, own_r2, ymask);
            float alpha = 1.f;
            if (__builtin_expect(__any(zc > m_run + kLazyThresh2), 0)) {  // wave-uniform
                const float cmax = row16_max(zc);
                if (cmax > m_run + kLazyThresh2) {
                    alpha = __builtin_amdgcn_exp2f(m_run - cmax);
                    s_part *= alpha;
                    m_run = cmax;
                }
            }
            const float p = __builtin_amdgcn_exp2f(zc - m_run);
            s_part += p;
            if (yg == own_tgt) zy_part = zc;
            gval = p;
            abuf[xo] = alpha;  // the 16 lanes of a row store the same value
        } else {
            // record {lse log2 e, r log2 e, target, r / T}; rows past the end
            // read as zeros and give gval = 0
            const f32x4 r4 = *(LDS_AS f32x4*)(rec + 4 * yy);
            const float p = __builtin_amdgcn_exp2f(sxy * r4[1] - r4[0]);
            gval = (p - (__float_as_int(r4[2]) == x0 + xo ? 1.f : 0.f)) * r4[3];
        }
        gbuf[xo * YC + yy] = (bf16)gval;
        if (more) stream.template issue_range<kDma2, G::NI>(nrs, d, nxt);
        lds_barrier();

        // ---- second product: acc[j][x] += sum_y Y[y][j] G[x][y] over this wave's columns
        const bf16x8 gfrag = *(bf16x8*)(gbuf + (lane & 31) * YC + 8 * (lane >> 5));
        if (MODE == 0) {
            const float al = abuf[lane & 31];
            if (__any(al != 1.f)) {
#pragma unroll
                for (int b = 0; b < G::NB; ++b)
#pragma unroll
                    for (int i = 0; i < 16; ++i) acc[b][i] *= al;
            }
        }
        bf16x4 tlo[G::NB], thi[G::NB];
#pragma unroll
        for (int b = 0; b < G::NB; ++b) {
            tlo[b] = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LDS_AS bf16x4*)(cur + c_lo + 64 * b));
            thi[b] = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LDS_AS bf16x4*)(cur + c_hi + 64 * b));
        }
#pragma unroll
        for (int b = 0; b < G::NB; ++b) {
            bf16x8 at;
            at[0] = tlo[b][0]; at[1] = tlo[b][1]; at[2] = tlo[b][2]; at[3] = tlo[b][3];
            at[4] = thi[b][0]; at[5] = thi[b][1]; at[6] = thi[b][2]; at[7] = thi[b][3];
            acc[b] = mfma32(at, gfrag, acc[b]);
        }
        __builtin_amdgcn_sched_barrier(0);
        wait_vm();
    };

    wait_vm();
    for (int c = 0; c < nchunks; c += 2) {
        step(sliceA, sliceB_u, (LDS_AS float*)(LDS_AS void*)recA, recB_u, c);
        if (c + 1 < nchunks) step(sliceB, sliceA_u, (LDS_AS float*)(LDS_AS void*)recB, recA_u, c + 1);
    }

    // ---- epilogues.  acc[b] lane layout: x = lane%32,
    //      j = js + 32 b + 8 (i/4) + 4 (lane/32) + i%4 for i = 0..15
    const int ex = lane & 31;
    const int ehh = lane >> 5;
    if (MODE == 0) {
        // finish the online softmax of rows 4w..4w+3
        float s = s_part, zy = zy_part;
        s = row16_sum(s);
        zy = row16_sum(zy);
        if (yy == 0) {
            const float lse2 = m_run + __log2f(s);
            const bool tok = own_tgt >= 0 && own_tgt < nY;
            const float rl = tok ? (lse2 - zy) * kLn2 : __int_as_float(0x7fc00000);
            if (x0 + xo < nX) {
                a.lse[modoff + x0 + xo] = lse2 * kLn2;
                a.rowloss[modoff + x0 + xo] = rl;
                if (a.rowrec && k == a.K - 1) {
                    f32x4 rec4 = {lse2, own_r2, __int_as_float(own_tgt), own_r * a.inv_T};
                    *(f32x4*)(a.rowrec + 4 * (long long)(x0 + xo)) = rec4;
                }
            }
            sbuf[xo] = 1.f / s;
        }
        __syncthreads();

        const int xg = x0 + ex;
        const bool xok = xg < nX;
        const float rx = xok ? a.rstd[modoff + xg] : 0.f;
        const int tgt = xok ? a.targets[modoff + xg] : -1;
        const bool tok = tgt >= 0 && tgt < nY;
        const float inv_s = sbuf[ex];
        const bf16* hrow = hk + (long long)(xok ? xg : 0) * d;
        const bf16* wrow = Wg + (long long)(tok ? tgt : 0) * d;
        float cp = 0.f;
#pragma unroll
        for (int b = 0; b < G::NB; ++b) {
#pragma unroll
            for (int i4 = 0; i4 < 4; ++i4) {
                const int j = js + 32 * b + 8 * i4 + 4 * ehh;
                u16x4 hv = {0, 0, 0, 0}, wv = {0, 0, 0, 0};
                if (xok) hv = *(const u16x4*)(hrow + j);
                if (tok) wv = *(const u16x4*)(wrow + j);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float dn = (acc[b][4 * i4 + e] * inv_s - bf16_bits_to_f32(wv[e])) * a.inv_T;
                    cp += dn * (rx * bf16_bits_to_f32(hv[e]));
                    acc[b][4 * i4 + e] = dn;
                }
            }
        }
        cp += __shfl_xor(cp, 32, 64);
        if (ehh == 0) cbuf[w * XR + ex] = cp;
        __syncthreads();
        float csum = 0.f;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) csum += cbuf[ww * XR + ex];
        const float cmean = csum / (float)d;
        if (xok) {
            bf16* dhrow = (bf16*)a.dh + (modoff + xg) * (long long)d;
#pragma unroll
            for (int b = 0; b < G::NB; ++b) {
#pragma unroll
                for (int i4 = 0; i4 < 4; ++i4) {
                    const int j = js + 32 * b + 8 * i4 + 4 * ehh;
                    const u16x4 hv = *(const u16x4*)(hrow + j);
                    bf16x4 o;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float n = rx * bf16_bits_to_f32(hv[e]);
                        o[e] = (bf16)(rx * (acc[b][4 * i4 + e] - cmean * n));
                    }
                    *(bf16x4*)(dhrow + j) = o;
                }
            }
        }
    } else {
        const int v = x0 + ex;
        const bool vok = v < nX;
        const bf16* wrow = (const bf16*)a.W + (long long)(vok ? v : 0) * d;
        const bf16* gain = (const bf16*)a.gain;
        float* dwrow = a.dW + (long long)(vok ? v : 0) * d;
        float* dgp = a.dgain_part + (long long)blockIdx.x * d;
#pragma unroll
        for (int b = 0; b < G::NB; ++b) {
#pragma unroll
            for (int i4 = 0; i4 < 4; ++i4) {
                const int j = js + 32 * b + 8 * i4 + 4 * ehh;
                const u16x4 gv = *(const u16x4*)(gain + j);
                u16x4 wv = {0, 0, 0, 0};
                if (vok) wv = *(const u16x4*)(wrow + j);
                f32x4 o;
                float pr[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float D = acc[b][4 * i4 + e];
                    o[e] = bf16_bits_to_f32(gv[e]) * D;
                    pr[e] = bf16_bits_to_f32(wv[e]) * D;
                }
                if (vok) *(f32x4*)(dwrow + j) = o;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    float t = pr[e];
                    t += __shfl_xor(t, 1, 64);
                    t += __shfl_xor(t, 2, 64);
                    t += __shfl_xor(t, 4, 64);
                    t += __shfl_xor(t, 8, 64);
                    t += __shfl_xor(t, 16, 64);
                    pr[e] = t;
                }
                if (ex == 0) {
                    f32x4 pv = {pr[0], pr[1], pr[2], pr[3]};
                    *(f32x4*)(dgp + j) = pv;
                }
            }
        }
    }
}

template <int MODE, int DS>
hipError_t launch_ds(const FusedArgs& a, hipStream_t s) {
    dim3 grid = (MODE == 0) ? dim3((unsigned)((a.T + XR - 1) / XR), (unsigned)a.K) : dim3((unsigned)((a.V + XR - 1) / XR));
    hipLaunchKernelGGL((k_fused<MODE, DS>), grid, dim3(NTHR), 0, s, a);
    return hipGetLastError();
}

template <int MODE>
hipError_t launch_mode(const FusedArgs& a, hipStream_t s) {
    switch (a.d / NW) {
        case 32: return launch_ds<MODE, 32>(a, s);
        case 64: return launch_ds<MODE, 64>(a, s);
        case 96: return launch_ds<MODE, 96>(a, s);
        case 128: return launch_ds<MODE, 128>(a, s);
        case 160: return launch_ds<MODE, 160>(a, s);
        case 192: return launch_ds<MODE, 192>(a, s);
        case 224: return launch_ds<MODE, 224>(a, s);
        case 256: return launch_ds<MODE, 256>(a, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

bool mfma_supported(int dtype, int d) { return dtype == 0 && d % (NW * 32) == 0 && d >= NW * 32 && d <= NW * 256; }

hipError_t launch_local_loss_mfma(const FusedArgs& a, hipStream_t s) { return launch_mode<0>(a, s); }
hipError_t launch_readout_grad_mfma(const FusedArgs& a, hipStream_t s) { return launch_mode<1>(a, s); }

}  // namespace solo
