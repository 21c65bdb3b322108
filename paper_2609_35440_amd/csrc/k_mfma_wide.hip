// Fused matrix-core passes of the SOLO shared-readout loss for wide hidden
// states, d = 2560 (bf16 operands, fp32 accumulate, gfx950).
//
// Same passes and algebra as k_mfma.hip: module k predicts through its
// readout R_k, gain g_k, temperature tau_k and bias b_k (Eq. 2 of the paper,
// with the bias of Algorithm 1):  z_tv = tau_k r_t <R_kv, g_k * h_t> + b_kv.
// What the width changes is what fits on a CU:
//
//   - 16 stationary rows per workgroup in the passes with a second product:
//     wave w owns the d/8 columns [w d/8, (w+1) d/8) of a 16 x d/8 fp32
//     accumulator (80 registers per lane at d = 2560) and of the stationary
//     operand; the passes without one (exit evaluation, bias gradient) hold
//     48 stationary rows, three 16-row blocks of the logit product;
//   - the second product runs on the 16x16x16 instruction (its contraction
//     over the 16 streamed rows of a chunk), its streamed operand read with
//     one ds_read_b64_tr_b16 per product;
//   - the streamed rows come from their tiled copy (see tiled_elems): each
//     wave loads its 10 k-steps of a chunk, one contiguous 1 KiB per
//     instruction, straight into the registers that feed the logit product.
//
// Per chunk each wave (1) computes its split-K partial of the 16 x XR logit
// tile from its operand registers, writes them into its private LDS slice
// (passes with a second product) and reloads them with the next chunk;
// (2) the 8 partials meet in LDS and each wave finishes the elementwise step
// for XR / 8 of the stationary rows; (3) every wave accumulates its column
// slice of the second product, reading its slice back transposed.
#include "mfma_common.h"
#include "mfma_layout_wide.h"

namespace solo {

namespace {

using namespace mfma;

constexpr int NW = layoutw::NW;  // waves per workgroup
constexpr int NTHR = NW * 64;
constexpr int YC = layoutw::YC;    // streamed rows per chunk
// Partial logit tiles part[w][x][y]: rows of PP = 16 floats, the 16-byte
// group y / 4 of row x stored at (y / 4) ^ ((x >> 1) & 3): conflict-free
// 16-byte writes and row reads.  The probability tile gbuf[x][y] (bf16, rows
// of YC) keeps the 8-byte group y / 4 of row x at (y / 4) ^ (2 ((x >> 3) & 1)),
// so that the 8-byte reads of its 16 rows spread over all 64 banks.
constexpr int PP = 16;

// Stationary rows per workgroup: 16 in the passes with a second product (the
// accumulator and the stationary operand fill the register file), 48 in the
// passes without one (exit evaluation, bias gradient: 120 registers of
// stationary operand), which cuts the readout streamed per flop to a third.
template <bool PC>
constexpr int wide_rows() { return PC ? kMfmaWideRows : 48; }
static_assert(kMfmaWideRows == 16, "one 16-row block of stationary rows with a second product");

enum Mode { LOCAL = 0, RGRAD = 1, BGRAD = 2, EVAL = 3 };

template <int DS, int XR>
struct Geo : layoutw::Geo<DS> {
    static constexpr int NK = DS / 32;  // 32-deep k-steps of the logit product
    static constexpr int NB = DS / 16;  // 16-column accumulator blocks per wave
    static constexpr int YBUF = NW * layoutw::Geo<DS>::SLICE;
    static constexpr int TOTAL = YBUF + NW * XR * PP * 4 + XR * YC * 2 + 2 * XR * 4 + NW * XR * 4 + 2 * YC * 16;
    static_assert(TOTAL <= 160 * 1024, "LDS budget");
};

typedef __bf16 bf16x4w __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma16k16(bf16x4w a, bf16x4w b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ const bf16* readout_of(const FusedArgs& a, int k) {
    return k == a.K - 1 ? (const bf16*)a.Wt : (const bf16*)a.Wh + (long long)k * a.wh_stride;
}

// MODE LOCAL / EVAL: grid (ceil(T/XR), nmod); MODE RGRAD / BGRAD: grid
// (ceil(V/XR), nmod); module k = m0 + blockIdx.y.
// XR = 16 with a second product (LOCAL, RGRAD), 48 without (EVAL, BGRAD).
// EXT (LOCAL and EVAL): the variant with per-chunk biases, launched when the call has biases.
template <int MODE, int DS, bool EXT>
__global__ __launch_bounds__(NTHR, 1) void k_fused_wide(FusedArgs a) {
    constexpr bool LL = MODE == LOCAL || MODE == EVAL;           // X = h, Y = readout
    constexpr bool PC = MODE == LOCAL || MODE == RGRAD;          // second product
    constexpr int XR = wide_rows<PC>();
    constexpr int NXB = XR / 16;                                 // 16-row blocks of the logit product
    static_assert((PC && XR == 16) || (!PC && (XR == 16 || XR == 32 || XR == 48)), "tile height");
    using G = Geo<DS, XR>;
    constexpr bool BZ = (MODE == LOCAL || MODE == EVAL) && EXT;  // per-chunk biases through LDS
    __shared__ __attribute__((aligned(16))) char ybuf[PC ? G::YBUF : 16];
    __shared__ __attribute__((aligned(16))) float part[NW * XR * PP];
    __shared__ __attribute__((aligned(16))) bf16 gbuf[XR * YC];
    __shared__ float abuf[XR];
    __shared__ float sbuf[XR];
    __shared__ float pybuf[XR];
    __shared__ float cbuf[NW * XR];
    __shared__ __attribute__((aligned(16))) float recA[YC * 4];
    __shared__ __attribute__((aligned(16))) float recB[YC * 4];

    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int d = a.d;
    const int js = w * DS;
    const int x0 = blockIdx.x * XR;
    const int k = a.m0 + (int)blockIdx.y;
    const long long modoff = (long long)k * a.T;
    const float tau_k = a.tau ? a.tau[k] : 1.f;

    const bf16* __restrict__ hk = (const bf16*)a.h + modoff * d;
    const bf16* __restrict__ Rk = readout_of(a, k);
    const bf16* __restrict__ gk = (const bf16*)a.gain + (long long)k * a.g_stride;
    const bf16* __restrict__ X = LL ? hk : Rk;
    const int nX = LL ? a.T : a.V;
    const int nY = LL ? a.V : a.T;
    const int nchunks = (nY + YC - 1) / YC;
    // this wave's k-step 0 of chunk 0 in the tiled streamed operand; k-step kk
    // of chunk c is 512 kk + 16 d c elements further, the lane's 16 bytes 8 lane
    const bf16* __restrict__ Yw =
        (LL ? (k == a.K - 1 ? (const bf16*)a.Wtt : (const bf16*)a.Wht + (long long)k * a.wht_stride)
            : (const bf16*)a.hg + (long long)(k - a.hg_m0) * tiled_elems(a.T, d)) +
        w * (G::NK * 512);
    const long long cstride = 16LL * d;
    // buffer loads over this wave's NK KiB of a chunk, one lane offset shared by
    // every load and the k-step as a scalar offset
    auto rsrc_of = [&](const bf16* __restrict__ base) __attribute__((always_inline)) {
        return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, G::NK * 1024, 0x00020000);
    };
    auto ld_op = [&](__amdgpu_buffer_rsrc_t rs, int kk) __attribute__((always_inline)) {
        return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rs, lane * 16, kk * 1024, 0));
    };
    // operand registers: k-step kk of the current chunk (lane: streamed row
    // lane % 16, columns js + 32 kk + 8 (lane / 16) .. + 7)
    bf16x8 ay[G::NK];
#pragma unroll
    for (int kk = 0; kk < G::NK; ++kk) ay[kk] = ld_op(rsrc_of(Yw), kk);

    LDS_AS char* slice = (LDS_AS char*)(LDS_AS void*)ybuf + w * G::SLICE;

    // elementwise ownership: the lane finishes stationary rows xo[r], r < ER,
    // at streamed column yy; only lanes with wr[r] write row xo[r].  16 rows:
    // row 2w + (l/16)%2, computed by lanes l and l + 32, written by l < 32;
    // 32 rows: row 4w + l/16; 48 rows: rows 6w + l/16 and 6w + 4 + (l/16)%2,
    // the second one again computed twice and written by l < 32
    constexpr int ER = XR == 48 ? 2 : 1;
    int xo[ER];
    bool wr[ER];
    xo[0] = XR == 16 ? 2 * w + ((lane >> 4) & 1) : (XR == 32 ? 4 * w : 6 * w) + (lane >> 4);
    wr[0] = XR != 16 || lane < 32;
    if constexpr (ER == 2) {
        xo[ER - 1] = 6 * w + 4 + ((lane >> 4) & 1);
        wr[ER - 1] = lane < 32;
    }
    const int yy = lane & 15;
    float own_r2[ER];  // LL: r_t tau_k log2 e of row xo[r]
    int own_tgt[ER];   // LL: target of row xo[r]
    float bx2[ER];     // RGRAD / BGRAD: bias of the stationary readout row, base 2
#pragma unroll
    for (int r = 0; r < ER; ++r) {
        own_r2[r] = 0.f;
        own_tgt[r] = -1;
        bx2[r] = 0.f;
        if (LL && x0 + xo[r] < nX) {
            own_r2[r] = a.rstd[modoff + x0 + xo[r]] * tau_k * kLog2e;
            own_tgt[r] = a.targets[modoff + x0 + xo[r]];
        }
        if (!LL && a.bias && x0 + xo[r] < nX) bx2[r] = a.bias[(long long)k * a.V + x0 + xo[r]] * kLog2e;
    }
    const bool has_bias = BZ || a.bias != nullptr;  // the bias variant always has one

    const unsigned recA_u = lds_addr((LDS_AS char*)(LDS_AS void*)recA);
    const unsigned recB_u = lds_addr((LDS_AS char*)(LDS_AS void*)recB);
    auto issue_side = [&](int y0, unsigned dst) __attribute__((always_inline)) {
        // rows of this chunk only (a range over all remaining rows could pass 2^32 bytes)
        const int rows = nY - y0 < YC ? nY - y0 : YC;
        if (!LL && w == 0 && lane < YC) {
            // the 16 per-token records of the chunk
            const unsigned rem = rows > 0 ? (unsigned)rows * 16u : 0u;
            buffer_load_lds16(make_rsrc(a.rowrec + 4 * (modoff + y0), rem), dst, lane * 16);
        }
        if (BZ && has_bias && w == 0 && lane < YC) {
            // the 16 biases of the chunk (zeros past the vocabulary)
            const unsigned rem = rows > 0 ? (unsigned)rows * 4u : 0u;
            buffer_load_lds4(make_rsrc(a.bias + (long long)k * a.V + y0, rem), dst, lane * 4);
        }
    };

    issue_side(0, recA_u);

    // stationary operand (local loss and exit evaluation: times the gain,
    // rounded once): B of the 16x16x32 logit product, lane holds
    // X[x0 + 16 xb + lane%16][js + 32 kk + 8 (lane/16) .. +7]
    bf16x8 xr[NXB][G::NK];
#pragma unroll
    for (int kk = 0; kk < G::NK; ++kk) {
        const int j0 = js + 32 * kk + 8 * (lane >> 4);
        const bf16x8 gv = *(const bf16x8*)(gk + j0);
#pragma unroll
        for (int xb = 0; xb < NXB; ++xb) {
            const int xrow = x0 + 16 * xb + (lane & 15);
            bf16x8 xv;
            if (xrow < nX) {
                xv = *(const bf16x8*)(X + (long long)xrow * d + j0);
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e) xv[e] = (bf16)0.f;
            }
            if (LL) {
#pragma unroll
                for (int e = 0; e < 8; ++e) xr[xb][kk][e] = (bf16)((float)xv[e] * (float)gv[e]);
            } else {
                xr[xb][kk] = xv;
            }
        }
    }

    f32x4 acc[PC ? G::NB : 1];
#pragma unroll
    for (int b = 0; b < (PC ? G::NB : 1); ++b) acc[b] = (f32x4){0.f, 0.f, 0.f, 0.f};

    // online softmax state (LL, base 2), per lane: row xo[r], streamed column yy
    float m_run[ER], s_part[ER], zy_part[ER];
    float best[ER];  // EVAL: largest logit seen by this lane, and its column
    int best_v[ER];
    float db_part[ER];  // RGRAD / BGRAD: sum_t (p - onehot) for row xo[r]
#pragma unroll
    for (int r = 0; r < ER; ++r) {
        m_run[r] = -INFINITY;
        s_part[r] = zy_part[r] = db_part[r] = 0.f;
        best[r] = -INFINITY;
        best_v[r] = -1;
    }

    // the operand registers of k-step kk go where the row-wise read of the slice
    // layout finds them: rd_even + 64 kk (kk even) or rd_odd + 64 kk (kk odd);
    // the swizzle flips bit 2 of the granule index for rows with (r & 4)
    const int rd_even = layoutw::rowread_off<DS>(lane, 0);
    const int rd_odd = layoutw::rowread_off<DS>(lane, 1) - 64;

    auto step = [&](LDS_AS float* side, unsigned side_nxt, int c) __attribute__((always_inline)) {
        const int y0 = c * YC;
        const bool more = c + 1 < nchunks;
        // reload with the next chunk (the last chunk reloads itself, unused)
        const __amdgpu_buffer_rsrc_t yn = rsrc_of(Yw + (more ? (long long)(c + 1) : (long long)c) * cstride);

        // ---- (1) split-K partial of the logit tile S[y][x] over this wave's columns
        if (more) issue_side(y0 + YC, side_nxt);
        f32x4 S[NXB];
#pragma unroll
        for (int xb = 0; xb < NXB; ++xb) S[xb] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < G::NK; ++kk) {
#pragma unroll
            for (int xb = 0; xb < NXB; ++xb) S[xb] = mfma16(ay[kk], xr[xb][kk], S[xb]);
            if (PC) *(LDS_AS bf16x8*)(slice + ((kk & 1) ? rd_odd : rd_even) + 64 * kk) = ay[kk];
            ay[kk] = ld_op(yn, kk);
            __builtin_amdgcn_sched_barrier(0);  // keeps the reload behind this k-step's uses
        }
        // C layout: lane holds S[y = 4 (lane/16) + i][x = 16 xb + lane%16]; store as part[w][x][y]
#pragma unroll
        for (int xb = 0; xb < NXB; ++xb) {
            const int xl = 16 * xb + (lane & 15);
            *(f32x4*)(part + (w * XR + xl) * PP + 4 * ((lane >> 4) ^ ((xl >> 1) & 3))) = S[xb];
        }
        lds_barrier();

        // ---- (2) elementwise step (lane: rows xo[r], column yy)
#pragma unroll
        for (int r = 0; r < ER; ++r) {
            float q[NW];
#pragma unroll
            for (int ww = 0; ww < NW; ++ww) q[ww] = part[(ww * XR + xo[r]) * PP + (yy ^ (4 * ((xo[r] >> 1) & 3)))];
            static_assert(NW == 8, "partial-sum tree");
            const float sxy = ((q[0] + q[1]) + (q[2] + q[3])) + ((q[4] + q[5]) + (q[6] + q[7]));
            const int yg = y0 + yy;
            float gval = 0.f;
            if (LL) {
                // columns past the end of the vocabulary get z = -inf
                float ymask = (yg < nY) ? 0.f : -INFINITY;
                if (BZ && has_bias) ymask += side[yy] * kLog2e;
                const float zc = __builtin_fmaf(sxy, own_r2[r], ymask);
                float alpha = 1.f;
                if (__builtin_expect(__any(zc > m_run[r] + kLazyThresh2), 0)) {  // wave-uniform
                    const float cmax = row16_max(zc);
                    if (cmax > m_run[r] + kLazyThresh2) {
                        alpha = __builtin_amdgcn_exp2f(m_run[r] - cmax);
                        s_part[r] *= alpha;
                        m_run[r] = cmax;
                    }
                }
                const float p = __builtin_amdgcn_exp2f(zc - m_run[r]);
                s_part[r] += yg == own_tgt[r] ? 0.f : p;  // the target's term joins at the end (finish_row)
                if (yg == own_tgt[r]) zy_part[r] = zc;
                if (MODE == EVAL && zc > best[r]) {  // strict: the first (lowest) column keeps a tie
                    best[r] = zc;
                    best_v[r] = yg;
                }
                // the target's probability enters the input gradient in the
                // epilogue, in fp32 together with its one-hot term
                gval = yg == own_tgt[r] ? 0.f : p;
                if (MODE == LOCAL && wr[r]) abuf[xo[r]] = alpha;  // the 16 lanes of a row store the same value
            } else {
                // record {lse log2 e, r tau log2 e, target, p_y - 1}; tokens past
                // the end of the module read as zeros and are masked.  The target's
                // entry of delta is the exact p_y - 1 of the local-loss pass.
                const f32x4 r4 = *(LDS_AS f32x4*)(side + 4 * yy);
                const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sxy, r4[1], bx2[r] - r4[0]));
                // (a padded token's zero record would match readout row 0 as its target)
                const float dlt = (yg < nY) ? (__float_as_int(r4[2]) == x0 + xo[r] ? r4[3] : p) : 0.f;
                gval = dlt * (r4[1] * (kLn2 * a.inv_T));  // times r tau / T
                db_part[r] += dlt;
            }
            if (PC && wr[r]) gbuf[xo[r] * YC + (yy ^ (8 * ((xo[r] >> 3) & 1)))] = (bf16)gval;
        }
        lds_barrier();

        if (PC) {
            // ---- (3) second product: acc[j][x] += sum_y Y[y][j] G[x][y] over this wave's columns
            // B operand: lane holds G[x = lane%16][y = 4 (lane/16) .. +3]
            const bf16x4w gfrag =
                *(LDS_AS bf16x4w*)(gbuf + (lane & 15) * YC + 4 * ((lane >> 4) ^ (2 * ((lane >> 3) & 1))));
            if (MODE == LOCAL) {
                const float al = abuf[lane & 15];
                if (__any(al != 1.f)) {
#pragma unroll
                    for (int b = 0; b < G::NB; ++b) acc[b] *= al;
                }
            }
#pragma unroll
            for (int b = 0; b < G::NB; ++b) {
                const bf16x4w t = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                    (LDS_AS bf16x4w*)(slice + layoutw::trread_off<DS>(lane, b)));
                acc[PC ? b : 0] = mfma16k16(t, gfrag, acc[PC ? b : 0]);
            }
        }
        // the next chunk's operand registers and side data have arrived; the
        // slice is rewritten by the next logit product only after this
        // chunk's transposing reads (LDS operations of a wave run in order)
        __builtin_amdgcn_sched_barrier(0);
        wait_vm();
    };

    wait_vm();

    for (int c = 0; c < nchunks; c += 2) {
        step((LDS_AS float*)(LDS_AS void*)recA, recB_u, c);
        if (c + 1 < nchunks) step((LDS_AS float*)(LDS_AS void*)recB, recA_u, c + 1);
    }

    // ---- epilogues.  acc[b] lane layout: x = lane%16, j = js + 16 b + 4 (lane/16) + i
    const int ex = lane & 15;
    const int eg = lane >> 4;
    if (LL) {
        // finish the online softmax of rows xo[r]
#pragma unroll
        for (int r = 0; r < ER; ++r) {
            const float sx = row16_sum(s_part[r]);
            const float zy = row16_sum(zy_part[r]);
            float bst = best[r];
            int bv = best_v[r];
            if (MODE == EVAL) {
                // argmax over the 16 lanes of the row: larger logit, then lower column
#pragma unroll
                for (int off = 1; off < 16; off <<= 1) {
                    const float ob = __shfl_xor(bst, off, 64);
                    const int ov = __shfl_xor(bv, off, 64);
                    if (ob > bst || (ob == bst && (unsigned)ov < (unsigned)bv)) {
                        bst = ob;
                        bv = ov;
                    }
                }
            }
            if (yy == 0 && wr[r]) {
                const int xr_ = x0 + xo[r];
                const bool tok = own_tgt[r] >= 0 && own_tgt[r] < nY;
                const RowEnd re = finish_row(m_run[r], sx, zy, tok);
                if (xr_ < nX) {
                    const long long t = modoff + xr_;
                    a.lse[t] = re.lse2 * kLn2;
                    a.rowloss[t] = re.loss;
                    if (MODE == EVAL && a.top1) a.top1[t] = bv;
                    if (MODE == LOCAL && a.rowrec) {
                        f32x4 rec4 = {re.lse2, own_r2[r], __int_as_float(own_tgt[r]), re.py1};
                        *(f32x4*)(a.rowrec + 4 * t) = rec4;
                    }
                }
                sbuf[xo[r]] = re.inv_s;
                // p_y - 1: the target's probability was left out of the probability tile
                if (MODE == LOCAL) pybuf[xo[r]] = re.py1;
            }
        }
    }
    if (MODE == LOCAL) {
        __syncthreads();
        const int xg = x0 + ex;
        const bool xok = xg < nX;
        const float rx = xok ? a.rstd[modoff + xg] : 0.f;
        const int tgt = xok ? a.targets[modoff + xg] : -1;
        const bool tok = tgt >= 0 && tgt < nY;
        const float inv_s = sbuf[ex];
        const float py1 = pybuf[ex];

        const bf16* hrow = hk + (long long)(xok ? xg : 0) * d;
        const bf16* wrow = Rk + (long long)(tok ? tgt : 0) * d;
        const bool want_dg = a.dg_mode == 2 || (a.dg_mode == 1 && k == a.K - 1);
        float* dgp = want_dg ? a.dgain_part + ((long long)(a.dg_mode == 2 ? k : 0) * gridDim.x + blockIdx.x) * d
                             : nullptr;
        // sweep 1: acc <- e = (acc / s + (p_y - 1) R_y) / T, so that dhhat = tau e
        // (the target's probability term joins its one-hot term in fp32), and
        // the row sums of e * g * n (n = r h): the RMSNorm backward's
        // mean(dn * n) = tau sum / d and the token's share of d loss / d tau
        float cp = 0.f;
#pragma unroll
        for (int b = 0; b < G::NB; ++b) {
            const int j = js + 16 * b + 4 * eg;
            const u16x4 hv = *(const u16x4*)(hrow + j);
            const u16x4 wv = *(const u16x4*)(wrow + j);
            const u16x4 gv = *(const u16x4*)(gk + j);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float wy = tok ? bf16_bits_to_f32(wv[e]) : 0.f;
                const float ev = __builtin_fmaf(acc[b][e], inv_s, py1 * wy) * a.inv_T;
                cp += bf16_bits_to_f32(gv[e]) * ev * (rx * bf16_bits_to_f32(hv[e]));
                acc[b][e] = ev;
            }
        }
        cp += __shfl_xor(cp, 16, 64);
        cp += __shfl_xor(cp, 32, 64);
        if (eg == 0) cbuf[w * XR + ex] = cp;
        __syncthreads();
        float csum = 0.f;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) csum += cbuf[ww * XR + ex];
        const float cmean = tau_k * csum / (float)d;
        if (a.rowdtau && w == 0 && eg == 0 && xok) a.rowdtau[modoff + xg] = tok ? csum : 0.f;

        // sweep 2: dh = r (dn - c n); or e to the buffer, whose RMSNorm backward
        // follows the rotation back (ROT heads)
        if (xok && a.ebuf) {
            bf16* er = (bf16*)a.ebuf + (modoff + xg) * (long long)(2 * d);
#pragma unroll
            for (int b = 0; b < G::NB; ++b) {
                const int j = js + 16 * b + 4 * eg;
                bf16x4w hi, lo;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    hi[e] = (bf16)acc[b][e];
                    lo[e] = (bf16)(acc[b][e] - (float)hi[e]);
                }
                *(bf16x4w*)(er + j) = hi;
                *(bf16x4w*)(er + d + j) = lo;
            }
        }
        if (xok && !a.ebuf) {
            bf16* dhrow = (bf16*)a.dh + (modoff + xg) * (long long)d;
#pragma unroll
            for (int b = 0; b < G::NB; ++b) {
                const int j = js + 16 * b + 4 * eg;
                const u16x4 hv = *(const u16x4*)(hrow + j);
                const u16x4 gv = *(const u16x4*)(gk + j);
                bf16x4 o;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float n = rx * bf16_bits_to_f32(hv[e]);
                    o[e] = (bf16)(rx * (tau_k * bf16_bits_to_f32(gv[e]) * acc[b][e] - cmean * n));
                }
                *(bf16x4*)(dhrow + j) = o;
            }
        }
        // sweep 3, for a module that trains its gain: the tile's partial sums
        // of dhhat * n = tau e * n over its 16 rows
        if (want_dg && !a.ebuf) {
#pragma unroll
            for (int b = 0; b < G::NB; ++b) {
                const int j = js + 16 * b + 4 * eg;
                const u16x4 hv = *(const u16x4*)(hrow + j);  // rx = 0 masks rows past the end
                f32x4 pv;
#pragma unroll
                for (int e = 0; e < 4; ++e) pv[e] = row16_sum(tau_k * acc[b][e] * (rx * bf16_bits_to_f32(hv[e])));
                if (ex == 0) *(f32x4*)(dgp + j) = pv;
            }
        }
    }
    if (!LL) {
        // bias gradient of the stationary readout rows: sum over the 16 lanes of the row
#pragma unroll
        for (int r = 0; r < ER; ++r) {
            const float db = row16_sum(db_part[r]);
            if (a.dbias && yy == 0 && wr[r] && x0 + xo[r] < nX)
                a.dbias[(long long)k * a.V + x0 + xo[r]] = db * a.inv_T;
        }
    }
    if (MODE == RGRAD) {
        const int v = x0 + ex;
        if (v < nX) {
            float* dR = (k == a.K - 1) ? a.dWt : a.dWh + (long long)k * a.V * d;
            float* dwrow = dR + (long long)v * d;
#pragma unroll
            for (int b = 0; b < G::NB; ++b) *(f32x4*)(dwrow + js + 16 * b + 4 * eg) = acc[b];
        }
    }
}

template <int MODE, int DS, bool EXT>
hipError_t launch_ds(const FusedArgs& a, int nmod, hipStream_t s) {
    const bool ll = MODE == LOCAL || MODE == EVAL;
    constexpr int XR = wide_rows<MODE == LOCAL || MODE == RGRAD>();
    dim3 grid = ll ? dim3((unsigned)((a.T + XR - 1) / XR), (unsigned)nmod)
                   : dim3((unsigned)((a.V + XR - 1) / XR), (unsigned)nmod);
    hipLaunchKernelGGL((k_fused_wide<MODE, DS, EXT>), grid, dim3(NTHR), 0, s, a);
    return hipGetLastError();
}

template <int MODE, bool EXT>
hipError_t launch_mode(const FusedArgs& a, int nmod, hipStream_t s) {
    switch (a.d) {
        case 2560: return launch_ds<MODE, 320, EXT>(a, nmod, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

bool mfma_wide_supported(int dtype, int d) { return dtype == 0 && d == 2560; }

hipError_t launch_local_loss_mfma_wide(const FusedArgs& a, bool ext, int nmod, hipStream_t s) {
    return ext ? launch_mode<LOCAL, true>(a, nmod, s) : launch_mode<LOCAL, false>(a, nmod, s);
}
hipError_t launch_exit_eval_mfma_wide(const FusedArgs& a, int nmod, hipStream_t s) {
    return a.bias ? launch_mode<EVAL, true>(a, nmod, s) : launch_mode<EVAL, false>(a, nmod, s);
}
hipError_t launch_readout_grad_mfma_wide(const FusedArgs& a, int nmod, hipStream_t s) {
    return launch_mode<RGRAD, false>(a, nmod, s);
}
hipError_t launch_bias_grad_mfma_wide(const FusedArgs& a, int nmod, hipStream_t s) {
    return launch_mode<BGRAD, false>(a, nmod, s);
}

}  // namespace solo
