// Fused matrix-core passes of the SOLO shared-readout loss (bf16 operands, fp32
// accumulate) for gfx950.
//
// Every pass has the shape "logit tile -> elementwise -> (second product)".
// Module k predicts through its readout R_k (the terminal's W for k = K-1,
// the heads' read-only copy otherwise), its gain g_k, temperature tau_k and
// bias b_k (Eq. 2 of the paper, with the bias of Algorithm 1):
//
//   z_tv = tau_k r_t <R_kv, g_k * h_t> + b_kv
//
//   local-loss pass (every module; Eq. 2 and Eq. 3):
//     stationary X = XR rows t of g_k * h_k, streamed Y = the readout rows v,
//     online (max, sum-exp) per row, and acc_t += sum_{v != y_t} exp(z_tv - m_t) R_kv,
//     so that dhhat_t = tau_k (acc_t / s_t + (p_{t,y} - 1) R_{k,y_t}) / T at the
//     end (the target's whole entry of delta in fp32, see finish_row), followed
//     by the RMSNorm backward and, for a module that trains its gain, the
//     tile's partial of dgain = sum_t dhhat_t * n_t.  The T x V logits and
//     probabilities stay on chip.
//
//   exit evaluation: the same without the second product; the top-1 of each
//     row (lowest index on ties) next to its loss.
//
//   readout-gradient pass (modules whose readout is trained):
//     stationary X = XR readout rows v, streamed Y = the rows t of g_k * h_k
//     (a copy rounded like the local-loss pass's stationary tile, so both
//     passes multiply the same operands), delta_tv = (exp(z_tv - lse_t) -
//     [v = y_t]) / T and dR_v = sum_t delta_tv tau_k r_t (g_k * h_t),
//     db_v = sum_t delta_tv.
//
//   bias-gradient pass: the readout-gradient pass without the second product,
//     for modules whose bias is trained but whose readout is not.
//
// Work split: a workgroup of 8 waves owns XR stationary rows (32, 64 or 128 where
// the register file allows it: see rows_of); wave w owns the d/8 columns
// [w d/8, (w+1) d/8).  Per chunk of 16 streamed rows, every wave multiplies
// its column slice (split-K partial of the logit tile), the partials meet in
// LDS, each wave finishes the elementwise step for XR/8 of the stationary
// rows, and every wave then accumulates its own column slice of the second
// product.  The accumulator (XR rows x d/8 columns, fp32) and the stationary
// operand stay in registers for the whole pass.
//
// Streaming: in the passes with a second product the chunk goes HBM/L2 ->
// LDS directly and is read twice from LDS: row-wise for the logit product and
// with the transposing read for the second product.  The passes without one
// (exit evaluation, bias gradient) stream the tiled copy of Y (see
// tiled_elems) straight into the registers that feed the logit product, one
// contiguous 1 KiB per wave and instruction, and need no LDS for the chunk,
// which measured faster at d = 2048.  With a second product the registers
// would still have to be written to LDS for the transposing read, and those
// ds_write_b128 measured slower than the direct-to-LDS stream and the
// row-wise reads together at d = 2048, so those passes keep the stream.
#include "mfma_common.h"

namespace solo {

namespace {

using namespace mfma;

constexpr int NW = layout::NW;  // waves per workgroup
constexpr int NTHR = NW * 64;
constexpr int YC = layout::YC;  // streamed rows per chunk
// Partial logit tiles part[w][x][y]: rows of PP = 16 floats, the 16-byte
// group y / 4 of row x stored at (y / 4) ^ ((x >> 1) & 3), so that the 16-byte
// writes (8 rows at one group per pass) and the elementwise step's reads (4
// whole rows per wave) are both free of bank conflicts.  The probability tile
// gbuf[x][y] (bf16, rows of YC) keeps the 16-byte half y / 8 of row x at
// (y / 8) ^ ((x >> 2) & 1), for its 16-byte reads of 8 rows per pass.
constexpr int PP = 16;

enum Mode { LOCAL = 0, RGRAD = 1, BGRAD = 2, EVAL = 3 };

// Stationary rows per workgroup: 64 while the accumulator (64 rows x d/8
// columns) and the stationary operand fit the register file (d <= 1024), 32
// otherwise.  The passes without a second product (no accumulator) hold as
// many rows as 128 registers of stationary operand take: 128 up to d = 1024,
// 64 at d = 2048.  The readout streamed per flop halves with each doubling.
template <int DS, bool PC>
constexpr int rows_of() { return (!PC && DS <= 128) ? 128 : ((DS <= 128 || (!PC && DS <= 256)) ? 64 : 32); }

template <int DS, bool PC>
struct Geo : layout::Geo<DS> {
    static constexpr int XR = rows_of<DS, PC>();       // stationary rows per workgroup
    static constexpr int PR = XR;                      // rows of the partial-logit exchange buffer
    static constexpr int NXB = XR / 16;                // 16-row blocks of the logit product
    static constexpr int NR = XR / 32;                 // 32-row halves of the second product
    // elementwise step: a lane takes EWC adjacent streamed columns of ER
    // stationary rows, LPR lanes share a row (64-row tiles: one row and two
    // columns per lane)
    static constexpr int EWC = XR == 64 ? 2 : 1;
    static constexpr int ER = NR / EWC;
    static constexpr int LPR = 16 / EWC;
    static constexpr int NB = DS / 32;                 // 32-column accumulator blocks per wave
    static constexpr int NK = DS / 32;                 // 32-deep k-steps of the logit product
    // one chunk buffer (all waves); the passes without a second product keep no chunk in LDS
    static constexpr int YBUF = PC ? NW * layout::Geo<DS>::SLICE : 16;
    static constexpr int GB = PC ? XR * YC : 8;        // elements of the probability tile (second product only)
    static constexpr int TOTAL = 2 * YBUF + NW * PR * PP * 4 + GB * 2 + 3 * XR * 4 + NW * XR * 4 + 4 * YC * 4;
    static_assert(TOTAL <= 160 * 1024, "LDS budget");
};

__device__ __forceinline__ const bf16* readout_of(const FusedArgs& a, int k) {
    return k == a.K - 1 ? (const bf16*)a.Wt : (const bf16*)a.Wh + (long long)k * a.wh_stride;
}

// the tiled copy of module k's readout (exit evaluation)
__device__ __forceinline__ const bf16* tiled_readout_of(const FusedArgs& a, int k) {
    return k == a.K - 1 ? (const bf16*)a.Wtt : (const bf16*)a.Wht + (long long)k * a.wht_stride;
}

// MODE LOCAL / EVAL: grid (ceil(T/XR), nmod); MODE RGRAD / BGRAD: grid
// (ceil(V/XR), nmod); module k = m0 + blockIdx.y.
// EXT (LOCAL and EVAL): the variant with per-chunk biases, launched when the call has biases.
template <int MODE, int DS, bool EXT>
__global__ __launch_bounds__(NTHR, 1) void k_fused(FusedArgs a) {
    constexpr bool PC = MODE == LOCAL || MODE == RGRAD;     // second product
    using G = Geo<DS, PC>;
    constexpr int XR = G::XR;
    constexpr int NR = G::NR;
    constexpr int PR = G::PR;
    constexpr bool LL = MODE == LOCAL || MODE == EVAL;      // X = h, Y = readout
    constexpr bool RF = !PC;                                // operand registers fed from the tiled copy
    constexpr bool BZ = (MODE == LOCAL || MODE == EVAL) && EXT;  // per-chunk biases through LDS
    // the stream of the next chunk: instructions [0, kDmaA) one per k-step of
    // the logit products, [kDmaA, NI) after the elementwise step.  Measured:
    // with a second product, at d = 2048 5 of 8 inside the products (3 and 8
    // are 3-5% slower, 4 and 6 within box-to-box noise), at d = 1024 2 of 4 (3%
    // faster than 3 of 4); without one (64-row tiles, twice the products per
    // chunk) all of them, 12-14% faster than 5 of 8 at d = 2048
    constexpr int kDmaA = ((DS <= 128 ? 4 : 5) * G::NI + 7) / 8;
    // Separate LDS objects, so that the compiler can tell the chunk being read
    // from the chunk being prefetched (no needless waits on the prefetch).
    __shared__ __attribute__((aligned(16))) char ybufA[G::YBUF];
    __shared__ __attribute__((aligned(16))) char ybufB[G::YBUF];
    __shared__ __attribute__((aligned(16))) float part[NW * PR * PP];
    __shared__ __attribute__((aligned(16))) bf16 gbuf[G::GB];
    __shared__ float abuf[XR];
    __shared__ float sbuf[XR];
    __shared__ float pybuf[XR];
    __shared__ float cbuf[NW * XR];
    // per-chunk side data streamed next to the chunk: the per-token records
    // (readout-/bias-gradient passes) or the chunk's 16 biases (local loss)
    __shared__ __attribute__((aligned(16))) float recA[YC * 4];
    __shared__ __attribute__((aligned(16))) float recB[YC * 4];

    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
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
    // the streamed rows: the readout, or the copy of g_k * h_k (row-major for
    // the direct-to-LDS stream, tiled for the register-fed passes); module
    // copies sit tiled_elems(T, d) apart either way
    const bf16* __restrict__ Y = LL ? (RF ? tiled_readout_of(a, k) : Rk)
                                    : (const bf16*)a.hg + (long long)(k - a.hg_m0) * tiled_elems(a.T, d);
    const int nX = LL ? a.T : a.V;
    const int nY = LL ? a.V : a.T;
    const int nchunks = (nY + YC - 1) / YC;

    LDS_AS char* sliceA = (LDS_AS char*)(LDS_AS void*)ybufA + w * G::SLICE;
    LDS_AS char* sliceB = (LDS_AS char*)(LDS_AS void*)ybufB + w * G::SLICE;

    // per-lane scalars of the rows this wave finishes in the elementwise step:
    // stationary rows xo[r] = 4 w + lane/16 + 32 r and streamed column yy of
    // the chunk, or, two columns per lane, row 8 w + lane/8 and columns yy, yy + 1
    constexpr int EWC = G::EWC, ER = G::ER, LPR = G::LPR;
    int xo[ER];
#pragma unroll
    for (int r = 0; r < ER; ++r) xo[r] = EWC == 2 ? 8 * w + (lane >> 3) : 4 * w + (lane >> 4) + 32 * r;
    const int yy = EWC == 2 ? 2 * (lane & 7) : (lane & 15);
    const int lane16 = lane & 15;  // the 16 lanes that stream a chunk's side data
    float own_r2[ER];  // LL: r_t tau_k log2 e of row xo (r_t is read again after the loop)
    // LL: target of row xo minus yy, the chunk start y0 at which this lane meets
    // it (the target itself is read again after the loop)
    int tgt_rel[ER];
    float bx2[ER];     // readout-/bias-gradient passes: bias of the stationary readout row, base 2
#pragma unroll
    for (int r = 0; r < ER; ++r) {
        own_r2[r] = 0.f;
        tgt_rel[r] = -1 - yy;
        bx2[r] = 0.f;
        if (LL && x0 + xo[r] < nX) {
            own_r2[r] = a.rstd[modoff + x0 + xo[r]] * tau_k * kLog2e;
            tgt_rel[r] = a.targets[modoff + x0 + xo[r]] - yy;
        }
        if (!LL && a.bias && x0 + xo[r] < nX) bx2[r] = a.bias[(long long)k * a.V + x0 + xo[r]] * kLog2e;
    }
    const bool has_bias = BZ || a.bias != nullptr;  // the bias variant always has one

    ChunkStream<DS> stream;
    if (PC) stream.init(d, js, lane);
    // first chunk in flight before the stationary operand is read
    const unsigned sliceA_u = lds_addr(sliceA), sliceB_u = lds_addr(sliceB);
    if (PC) stream.issue(Y, nY, d, 0, sliceA_u);
    // register-fed passes: k-step kk of chunk c of this wave's slice is NK KiB
    // into chunk c of the tiled copy plus 1 KiB kk; buffer loads over those NK
    // KiB, one lane offset shared by every load and the k-step as a scalar offset
    const bf16* __restrict__ Yw = Y + w * (G::NK * 512);
    auto rsrc_of = [&](int c) __attribute__((always_inline)) {
        return __builtin_amdgcn_make_buffer_rsrc((void*)(Yw + (long long)c * 16 * d), (short)0, G::NK * 1024,
                                                 0x00020000);
    };
    auto ld_op = [&](__amdgpu_buffer_rsrc_t rs, int kk) __attribute__((always_inline)) {
        return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rs, lane * 16, kk * 1024, 0));
    };
    // operand registers of the register-fed passes: k-step kk of the current
    // chunk (lane: streamed row lane % 16, columns js + 32 kk + 8 (lane / 16) .. + 7)
    bf16x8 ay_rf[RF ? G::NK : 1];
    if (RF) {
#pragma unroll
        for (int kk = 0; kk < G::NK; ++kk) ay_rf[kk] = ld_op(rsrc_of(0), kk);
    }
    const unsigned recA_u = lds_addr((LDS_AS char*)(LDS_AS void*)recA);
    const unsigned recB_u = lds_addr((LDS_AS char*)(LDS_AS void*)recB);
    auto issue_side = [&](int y0, unsigned dst) __attribute__((always_inline)) {
        // rows of this chunk only (a range over all remaining rows could pass 2^32 bytes)
        const int rows = nY - y0 < YC ? nY - y0 : YC;
        if (!LL && w == 0 && lane < YC) {
            // the 16 per-token records of the chunk
            const unsigned rem = rows > 0 ? (unsigned)rows * 16u : 0u;
            buffer_load_lds16(make_rsrc(a.rowrec + 4 * (modoff + y0), rem), dst, lane16 * 16);
        }
        if (BZ && has_bias && w == 0 && lane < YC) {
            // the 16 biases of the chunk (zeros past the vocabulary)
            const unsigned rem = rows > 0 ? (unsigned)rows * 4u : 0u;
            buffer_load_lds4(make_rsrc(a.bias + (long long)k * a.V + y0, rem), dst, lane16 * 4);
        }
    };
    issue_side(0, recA_u);

    // stationary operand (local loss and exit evaluation: times the gain,
    // rounded once): B of the 16x16x32 logit product, lane holds
    // X[x0 + 16 xb + lane%16][js + 32 kk + 8 (lane/16) .. +7]
    bf16x8 xr[G::NXB][G::NK];
#pragma unroll
    for (int kk = 0; kk < G::NK; ++kk) {
        const int j0 = js + 32 * kk + 8 * (lane >> 4);
        const bf16x8 gv = *(const bf16x8*)(gk + j0);
#pragma unroll
        for (int xb = 0; xb < G::NXB; ++xb) {
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

    // accumulator: 32-column block b of this wave's slice, 32-row half h of the tile
    f32x16 acc[PC ? G::NB : 1][NR];
#pragma unroll
    for (int b = 0; b < (PC ? G::NB : 1); ++b)
#pragma unroll
        for (int h = 0; h < NR; ++h)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[b][h][i] = 0.f;

    // online softmax state (LL, base 2), per lane and row r: row xo[r], streamed column yy
    float m_run[ER], s_part[ER], zy_part[ER];
    float best[ER];   // EVAL: largest logit seen by this lane, and its column
    int best_v[ER];
    float db_part[ER];  // RGRAD / BGRAD: sum_t (p - onehot) for row xo[r]
#pragma unroll
    for (int r = 0; r < ER; ++r) {
        m_run[r] = -INFINITY;
        s_part[r] = zy_part[r] = db_part[r] = 0.f;
        best[r] = -INFINITY;
        best_v[r] = -1;
    }

    // per-lane parts of the LDS addresses; the unrolled loops add 64 * kk or 64 * b
    const int a_off = layout::rowread_off<DS>(lane);
    const int c_lo = layout::trread_off<DS>(lane, 0);
    const int c_hi = layout::trread_off<DS>(lane, 1);

    auto step = [&](LDS_AS char* cur, unsigned nxt, LDS_AS float* side, unsigned side_nxt, int c)
                    __attribute__((always_inline)) {
        const int y0 = c * YC;
        const bool more = c + 1 < nchunks;
        const i32x4 nrs = ChunkStream<DS>::rsrc(Y, nY, d, y0 + YC);
        // register-fed passes reload the operand registers with the next chunk
        // (the last chunk reloads itself: no branch around the loads)
        const __amdgpu_buffer_rsrc_t yn = rsrc_of(more ? c + 1 : c);

        // ---- split-K partial of the logit tile S[y][x] over this wave's columns.
        // All operand reads go out first, ahead of the data of the next chunk,
        // whose stream is spread over the products (and the end of the
        // elementwise step), so that neither the texture unit's queue nor the
        // LDS write port sees the whole chunk at once.
        bf16x8 ay[PC ? G::NK : 1];
        if (PC) {
            // the widest slices recompute the per-lane part of the row-wise read
            // address each step (no register left to hold it)
            const int ao = DS >= 224 ? layout::rowread_off<DS>(lane_now()) : a_off;
#pragma unroll
            for (int kk = 0; kk < G::NK; ++kk) ay[kk] = *(LDS_AS bf16x8*)(cur + ao + 64 * kk);
        }
        if (more) issue_side(y0 + YC, side_nxt);
        f32x4 S[G::NXB];
#pragma unroll
        for (int xb = 0; xb < G::NXB; ++xb) S[xb] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < G::NK; ++kk) {
            if constexpr (RF) {
#pragma unroll
                for (int xb = 0; xb < G::NXB; ++xb) S[xb] = mfma16(ay_rf[kk], xr[xb][kk], S[xb]);
                ay_rf[kk] = ld_op(yn, kk);
                __builtin_amdgcn_sched_barrier(0);  // keeps the reload behind this k-step's products
            } else {
#pragma unroll
                for (int xb = 0; xb < G::NXB; ++xb) S[xb] = mfma16(ay[kk], xr[xb][kk], S[xb]);
                if (kk < kDmaA) {
                    if (more) stream.issue_one(nrs, d, nxt, kk);
                    __builtin_amdgcn_sched_barrier(0);  // keeps the instruction between these products
                }
            }
        }
        const int ylim = nY - y0;  // columns yy >= ylim of this chunk are past the last streamed row
        // C layout: lane holds S[y = 4 (lane/16) + i][x = 16 xb + lane%16]; store as part[w][x][y]
#pragma unroll
        for (int xb = 0; xb < G::NXB; ++xb) {
            const int xl = 16 * xb + (lane & 15);
            *(LDS_AS f32x4*)((LDS_AS float*)(LDS_AS void*)part + (w * PR + xl) * PP + 4 * ((lane >> 4) ^ ((xl >> 1) & 3))) =
                S[xb];
        }
        lds_barrier();
        {
            // ---- elementwise step for rows xo[r] (lane: row xo[r], columns yy .. yy + EWC - 1)
#pragma unroll
            for (int r = 0; r < ER; ++r) {
                float q[EWC][NW];
                const int xl = xo[r];
                const int yq = yy ^ (4 * ((xl >> 1) & 3));  // (yy even for two columns: both in one group)
#pragma unroll
                for (int ww = 0; ww < NW; ++ww) {
                    if constexpr (EWC == 2) {
                        const f32x2 v = *(LDS_AS f32x2*)((LDS_AS float*)(LDS_AS void*)part + (ww * PR + xl) * PP + yq);
                        q[0][ww] = v[0];
                        q[EWC - 1][ww] = v[1];
                    } else {
                        q[0][ww] = ((LDS_AS float*)(LDS_AS void*)part)[(ww * PR + xl) * PP + yq];
                    }
                }
                static_assert(NW == 8, "partial-sum tree");
                float sxy[EWC], gval[EWC];
#pragma unroll
                for (int e = 0; e < EWC; ++e) {
                    sxy[e] = ((q[e][0] + q[e][1]) + (q[e][2] + q[e][3])) + ((q[e][4] + q[e][5]) + (q[e][6] + q[e][7]));
                    gval[e] = 0.f;
                }
                if (LL) {
                    // columns past the end of the vocabulary get z = -inf (an additive
                    // mask rather than a branch, so the partial reads stay unconditional)
                    float zc[EWC];
                    float zmax = -INFINITY;
#pragma unroll
                    for (int e = 0; e < EWC; ++e) {
                        float ymask = (yy + e < ylim) ? 0.f : -INFINITY;
                        if (BZ && has_bias) ymask += side[yy + e] * kLog2e;
                        zc[e] = __builtin_fmaf(sxy[e], own_r2[r], ymask);
                        zmax = fmaxf(zmax, zc[e]);
                    }
                    float alpha = 1.f;
                    if (__builtin_expect(__any(zmax > m_run[r] + kLazyThresh2), 0)) {  // wave-uniform
                        const float cmax = group_max<LPR>(zmax);
                        if (cmax > m_run[r] + kLazyThresh2) {
                            alpha = __builtin_amdgcn_exp2f(m_run[r] - cmax);
                            s_part[r] *= alpha;
                            m_run[r] = cmax;
                        }
                    }
#pragma unroll
                    for (int e = 0; e < EWC; ++e) {
                        const float p = __builtin_amdgcn_exp2f(zc[e] - m_run[r]);
                        const bool is_y = tgt_rel[r] - e == y0;
                        s_part[r] += is_y ? 0.f : p;  // the target's term joins at the end (finish_row)
                        if (is_y) zy_part[r] = zc[e];
                        if (MODE == EVAL && zc[e] > best[r]) {  // strict: the first (lowest) column keeps a tie
                            best[r] = zc[e];
                            best_v[r] = y0 + yy + e;
                        }
                        // the target's probability enters the input gradient in
                        // the epilogue, in fp32 together with its one-hot term
                        gval[e] = is_y ? 0.f : p;
                    }
                    if (MODE == LOCAL) abuf[xo[r]] = alpha;  // the lanes of a row store the same value
                } else {
#pragma unroll
                    for (int e = 0; e < EWC; ++e) {
                        // record {lse log2 e, r tau log2 e, target, p_y - 1}; tokens past
                        // the end of the module read as zeros and are masked.  The
                        // target's entry of delta is the exact p_y - 1 of the local-loss pass.
                        const f32x4 r4 = *(LDS_AS f32x4*)(side + 4 * (yy + e));
                        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sxy[e], r4[1], bx2[r] - r4[0]));
                        // (a padded token's zero record would match readout row 0 as its target)
                        const float dlt =
                            (yy + e < ylim) ? (__float_as_int(r4[2]) == x0 + xo[r] ? r4[3] : p) : 0.f;
                        gval[e] = dlt * (r4[1] * (kLn2 * a.inv_T));  // times r tau / T
                        db_part[r] += dlt;
                    }
                }
                if (PC) {
                    bf16* gp = gbuf + xo[r] * YC + (yy ^ (8 * ((xo[r] >> 2) & 1)));
                    if constexpr (EWC == 2) {
                        bf16x2 g2;
                        g2[0] = (bf16)gval[0];
                        g2[1] = (bf16)gval[EWC - 1];
                        *(bf16x2*)gp = g2;
                    } else {
                        *gp = (bf16)gval[0];
                    }
                }
            }
        }
        if (PC && more) stream.template issue_range<kDmaA, G::NI>(nrs, d, nxt);
        lds_barrier();

        // 64-row tiles: the second product runs at raised wave priority, so that
        // a wave's products for the next chunk do not overtake the other wave's
        // second product on the SIMD (measured 2.3% faster at d = 1024; at
        // d = 2048 with 32-row tiles it is 0.5% slower and not used)
        constexpr bool PRIO = PC && XR == 64;
        if (PRIO) __builtin_amdgcn_s_setprio(2);
        if (PC) {
            // ---- second product: acc[j][x] += sum_y Y[y][j] G[x][y] over this wave's columns
            bf16x8 gfrag[NR];
#pragma unroll
            for (int h = 0; h < NR; ++h) {
                const int xg = 32 * h + (lane & 31);
                gfrag[h] = *(bf16x8*)(gbuf + xg * YC + 8 * ((lane >> 5) ^ ((xg >> 2) & 1)));
            }
            if (MODE == LOCAL) {
#pragma unroll
                for (int h = 0; h < NR; ++h) {
                    const float al = abuf[32 * h + (lane & 31)];
                    if (__any(al != 1.f)) {
#pragma unroll
                        for (int b = 0; b < G::NB; ++b)
#pragma unroll
                            for (int i = 0; i < 16; ++i) acc[b][h][i] *= al;
                    }
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
#pragma unroll
                for (int h = 0; h < NR; ++h) acc[PC ? b : 0][h] = mfma32(at, gfrag[h], acc[PC ? b : 0][h]);
            }
        }
        if (PRIO) __builtin_amdgcn_s_setprio(0);
        __builtin_amdgcn_sched_barrier(0);
        wait_vm();
    };

    wait_vm();
    for (int c = 0; c < nchunks; c += 2) {
        step(sliceA, sliceB_u, (LDS_AS float*)(LDS_AS void*)recA, recB_u, c);
        if (c + 1 < nchunks) step(sliceB, sliceA_u, (LDS_AS float*)(LDS_AS void*)recB, recA_u, c + 1);
    }

    // ---- epilogues.  acc[b][h] lane layout: x = 32 h + lane%32,
    //      j = js + 32 b + 8 (i/4) + 4 (lane/32) + i%4 for i = 0..15
    const int ex = lane & 31;
    const int ehh = lane >> 5;
    if (LL) {
        // finish the online softmax of rows xo[r]
#pragma unroll
        for (int r = 0; r < ER; ++r) {
            const int own_tgt = x0 + xo[r] < nX ? a.targets[modoff + x0 + xo[r]] : -1;
            const float sx = group_sum<LPR>(s_part[r]);
            const float zy = group_sum<LPR>(zy_part[r]);
            float bst = best[r];
            int bv = best_v[r];
            if (MODE == EVAL) {
                // argmax over the lanes of the row: larger logit, then lower column
#pragma unroll
                for (int off = 1; off < LPR; off <<= 1) {
                    const float ob = __shfl_xor(bst, off, 64);
                    const int ov = __shfl_xor(bv, off, 64);
                    if (ob > bst || (ob == bst && (unsigned)ov < (unsigned)bv)) {
                        bst = ob;
                        bv = ov;
                    }
                }
            }
            if (lane % LPR == 0) {
                const int xr_ = x0 + xo[r];
                const bool tok = own_tgt >= 0 && own_tgt < nY;
                const RowEnd re = finish_row(m_run[r], sx, zy, tok);
                if (xr_ < nX) {
                    const long long t = modoff + xr_;
                    a.lse[t] = re.lse2 * kLn2;
                    a.rowloss[t] = re.loss;
                    if (MODE == EVAL && a.top1) a.top1[t] = bv;
                    if (MODE == LOCAL && a.rowrec) {
                        f32x4 rec4 = {re.lse2, own_r2[r], __int_as_float(own_tgt), re.py1};
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
        const bool want_dg = a.dg_mode == 2 || (a.dg_mode == 1 && k == a.K - 1);
        float* dgp = want_dg ? a.dgain_part + ((long long)(a.dg_mode == 2 ? k : 0) * gridDim.x + blockIdx.x) * d
                             : nullptr;
        bool xok[NR], tok[NR];
        float rx[NR];
        const bf16* hrow[NR];
        // sweep 1: acc <- e = (acc / s + (p_y - 1) R_y) / T, so that dhhat = tau e
        // (acc holds every column but the target's, whose probability term
        // joins its one-hot term here in fp32), and the row sums of e * g * n
        // (n = r h).  That row sum is both the RMSNorm backward's mean(dn * n)
        // = tau sum / d and the token's share of d loss / d tau = sum_v
        // delta_v u_v = <sum_v delta_v R_v, g * n>.
#pragma unroll
        for (int h = 0; h < NR; ++h) {
            const int xg = x0 + 32 * h + ex;
            xok[h] = xg < nX;
            rx[h] = xok[h] ? a.rstd[modoff + xg] : 0.f;
            const int tgt = xok[h] ? a.targets[modoff + xg] : -1;
            tok[h] = tgt >= 0 && tgt < nY;
            const float inv_s = sbuf[32 * h + ex];
            const float py1 = pybuf[32 * h + ex];
            hrow[h] = hk + (long long)(xok[h] ? xg : 0) * d;
            const bf16* wrow = Rk + (long long)(tok[h] ? tgt : 0) * d;
            float cp = 0.f;
#pragma unroll
            for (int b = 0; b < (PC ? G::NB : 1); ++b) {
#pragma unroll
                for (int i4 = 0; i4 < 4; ++i4) {
                    const int j = js + 32 * b + 8 * i4 + 4 * ehh;
                    // unconditional loads (the row pointers are clamped to row 0), masked
                    // afterwards: no control flow inside the sweep
                    const u16x4 hv = *(const u16x4*)(hrow[h] + j);
                    const u16x4 wv = *(const u16x4*)(wrow + j);
                    const u16x4 gv = *(const u16x4*)(gk + j);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float wy = tok[h] ? bf16_bits_to_f32(wv[e]) : 0.f;
                        const float ev = __builtin_fmaf(acc[b][h][4 * i4 + e], inv_s, py1 * wy) * a.inv_T;
                        cp += bf16_bits_to_f32(gv[e]) * ev * (rx[h] * bf16_bits_to_f32(hv[e]));
                        acc[b][h][4 * i4 + e] = ev;
                    }
                }
                __builtin_amdgcn_sched_barrier(0);  // one block's loads at a time
            }
            cp += __shfl_xor(cp, 32, 64);
            if (ehh == 0) cbuf[w * XR + 32 * h + ex] = cp;
        }
        __syncthreads();
        // sweep 2: dh = r (dn - c n).  The accumulator layout gives a lane 8
        // bytes of a row per store (16 contiguous bytes per row and
        // instruction), which the memory system writes back as partial lines.
        // The 32 rows of a half-tile are staged in this wave's two (now idle)
        // chunk slices instead, 16 rows each, granule g of row r at g ^ (r & SM),
        // and leave as whole row segments of the wave's columns.
        constexpr int GS = DS / 8;  // 16-byte granules per row of the wave's columns
        constexpr int SM = (GS % 16 == 0) ? 15 : ((GS % 8 == 0) ? 7 : 3);
        static_assert(GS % 4 == 0 && 16 * 2 * DS <= G::SLICE, "staging rows fit a chunk slice");
#pragma unroll
        for (int h = 0; h < NR; ++h) {
            const int xg = x0 + 32 * h + ex;
            float csum = 0.f;
#pragma unroll
            for (int ww = 0; ww < NW; ++ww) csum += cbuf[ww * XR + 32 * h + ex];
            const float cmean = tau_k * csum / (float)d;
            if (a.rowdtau && w == 0 && ehh == 0 && xok[h]) a.rowdtau[modoff + xg] = tok[h] ? csum : 0.f;
            if (a.ebuf) {
                // e to the buffer as bf16 planes hi | lo; the RMSNorm backward follows
                // the rotation back
                if (xok[h]) {
                    bf16* er = (bf16*)a.ebuf + (modoff + xg) * (long long)(2 * d);
#pragma unroll
                    for (int b = 0; b < (PC ? G::NB : 1); ++b)
#pragma unroll
                        for (int i4 = 0; i4 < 4; ++i4) {
                            const int j = js + 32 * b + 8 * i4 + 4 * ehh;
                            mfma::bf16x4 hi, lo;
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                hi[e] = (bf16)acc[b][h][4 * i4 + e];
                                lo[e] = (bf16)(acc[b][h][4 * i4 + e] - (float)hi[e]);
                            }
                            *(mfma::bf16x4*)(er + j) = hi;
                            *(mfma::bf16x4*)(er + d + j) = lo;
                        }
                }
                continue;
            }
            LDS_AS char* srow = (ex < 16 ? sliceA : sliceB) + (ex & 15) * (2 * DS);
#pragma unroll
            for (int b = 0; b < (PC ? G::NB : 1); ++b) {
#pragma unroll
                for (int i4 = 0; i4 < 4; ++i4) {
                    const int j = js + 32 * b + 8 * i4 + 4 * ehh;
                    const u16x4 hv = *(const u16x4*)(hrow[h] + j);  // row 0 for rows past the end
                    const u16x4 gv = *(const u16x4*)(gk + j);
                    bf16x4 o;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float n = rx[h] * bf16_bits_to_f32(hv[e]);
                        o[e] = (bf16)(rx[h] * (tau_k * bf16_bits_to_f32(gv[e]) * acc[b][h][4 * i4 + e] - cmean * n));
                    }
                    *(LDS_AS bf16x4*)(srow + 16 * ((4 * b + i4) ^ (ex & SM)) + 8 * ehh) = o;
                }
                __builtin_amdgcn_sched_barrier(0);
            }
            // lane p of store q moves granule slot 64 q + p of the 32 x GS staged granules
#pragma unroll
            for (int q = 0; q < GS / 2; ++q) {
                const int sl = 64 * q + lane, row = sl / GS, g = sl % GS;
                const i32x4 v = *(LDS_AS i32x4*)((row < 16 ? sliceA : sliceB) + (row & 15) * (2 * DS) +
                                                 16 * (g ^ (row & SM)));
                const int xr = x0 + 32 * h + row;
                if (xr < nX) *(i32x4*)((bf16*)a.dh + (modoff + xr) * (long long)d + js + 8 * g) = v;
            }
        }
        // sweep 3, for a module that trains its gain: the tile's partial sums
        // of dhhat * n = tau e * n over its rows (the 16-lane row, the other row
        // of the half-wave, then the other 32-row half of the tile)
        if (want_dg && !a.ebuf) {
#pragma unroll
            for (int b = 0; b < (PC ? G::NB : 1); ++b) {
#pragma unroll
                for (int i4 = 0; i4 < 4; ++i4) {
                    const int j = js + 32 * b + 8 * i4 + 4 * ehh;
                    f32x4 pv = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int h = 0; h < NR; ++h) {
                        const u16x4 hv = *(const u16x4*)(hrow[h] + j);  // rx = 0 masks rows past the end
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const float t = row16_sum(tau_k * acc[b][h][4 * i4 + e] * (rx[h] * bf16_bits_to_f32(hv[e])));
                            pv[e] += t + __shfl_xor(t, 16, 64);
                        }
                    }
                    if (ex == 0) *(f32x4*)(dgp + j) = pv;
                }
            }
        }
    }
    if (!LL) {
        // bias gradient of the stationary readout rows: sum over the lanes of the row
#pragma unroll
        for (int r = 0; r < ER; ++r) {
            const float db = group_sum<LPR>(db_part[r]);
            if (a.dbias && lane % LPR == 0 && x0 + xo[r] < nX)
                a.dbias[(long long)k * a.V + x0 + xo[r]] = db * a.inv_T;
        }
    }
    if (MODE == RGRAD) {
        // dR_v = D_v
#pragma unroll
        for (int h = 0; h < NR; ++h) {
            const int v = x0 + 32 * h + ex;
            const bool vok = v < nX;
            float* dR = (k == a.K - 1) ? a.dWt : a.dWh + (long long)k * a.V * d;
            float* dwrow = dR + (long long)(vok ? v : 0) * d;
#pragma unroll
            for (int b = 0; b < (PC ? G::NB : 1); ++b) {
#pragma unroll
                for (int i4 = 0; i4 < 4; ++i4) {
                    const int j = js + 32 * b + 8 * i4 + 4 * ehh;
                    f32x4 o;
#pragma unroll
                    for (int e = 0; e < 4; ++e) o[e] = acc[b][h][4 * i4 + e];
                    if (vok) *(f32x4*)(dwrow + j) = o;
                }
            }
        }
    }
}

template <int MODE, int DS, bool EXT>
hipError_t launch_ds(const FusedArgs& a, int nmod, hipStream_t s) {
    const bool ll = MODE == LOCAL || MODE == EVAL;
    constexpr int XR = Geo<DS, MODE == LOCAL || MODE == RGRAD>::XR;
    dim3 grid = ll ? dim3((unsigned)((a.T + XR - 1) / XR), (unsigned)nmod)
                   : dim3((unsigned)((a.V + XR - 1) / XR), (unsigned)nmod);
    hipLaunchKernelGGL((k_fused<MODE, DS, EXT>), grid, dim3(NTHR), 0, s, a);
    return hipGetLastError();
}

template <int MODE, bool EXT>
hipError_t launch_mode(const FusedArgs& a, int nmod, hipStream_t s) {
    switch (a.d / NW) {
        case 32: return launch_ds<MODE, 32, EXT>(a, nmod, s);
        case 64: return launch_ds<MODE, 64, EXT>(a, nmod, s);
        case 96: return launch_ds<MODE, 96, EXT>(a, nmod, s);
        case 128: return launch_ds<MODE, 128, EXT>(a, nmod, s);
        case 160: return launch_ds<MODE, 160, EXT>(a, nmod, s);
        case 192: return launch_ds<MODE, 192, EXT>(a, nmod, s);
        case 224: return launch_ds<MODE, 224, EXT>(a, nmod, s);
        case 256: return launch_ds<MODE, 256, EXT>(a, nmod, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

bool mfma_supported(int dtype, int d) { return dtype == 0 && d % (NW * 32) == 0 && d >= NW * 32 && d <= NW * 256; }

int mfma_rows(int d) { return d <= NW * 128 ? rows_of<128, true>() : rows_of<256, true>(); }

hipError_t launch_local_loss_mfma(const FusedArgs& a, bool ext, int nmod, hipStream_t s) {
    return ext ? launch_mode<LOCAL, true>(a, nmod, s) : launch_mode<LOCAL, false>(a, nmod, s);
}
hipError_t launch_exit_eval_mfma(const FusedArgs& a, int nmod, hipStream_t s) {
    return a.bias ? launch_mode<EVAL, true>(a, nmod, s) : launch_mode<EVAL, false>(a, nmod, s);
}
hipError_t launch_readout_grad_mfma(const FusedArgs& a, int nmod, hipStream_t s) {
    return launch_mode<RGRAD, false>(a, nmod, s);
}
hipError_t launch_bias_grad_mfma(const FusedArgs& a, int nmod, hipStream_t s) {
    return launch_mode<BGRAD, false>(a, nmod, s);
}

}  // namespace solo
