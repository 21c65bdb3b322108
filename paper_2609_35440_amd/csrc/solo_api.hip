// C ABI of the SOLO shared-readout local loss: argument checks, workspace
// layout and the launch sequence on the caller's stream.
#include <cmath>
#include <cstdint>
#include <mutex>

#include "solo_readout.h"
#include "solo_internal.h"

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool shape_ok(int K, int T, int d, int V) {
    if (K < 1 || T < 1 || V < 1) return false;
    if (d < 8 || d % 8 != 0 || d > 4096) return false;
    if (K > 65535 || T > (1 << 30) || V > (1 << 30)) return false;
    if ((long long)K * (long long)T > 2147483647LL) return false;
    return true;
}

bool flag_ok(int f) { return f == 0 || f == 1; }

// What one call launches, and where its workspace pieces sit.
struct Plan {
    bool mfma = false;         // matrix-core family (either tiling)
    bool wide = false;         // the 16-row wide tiling of the matrix-core family (d = 2560)
    bool eval = false;
    bool ext = false;          // local-loss variant with per-chunk biases
    int dg_mode = 0;           // 0 none, 1 terminal only, 2 every module
    int slots = 0;             // gain-gradient partial slots
    int ntiles = 0;            // token tiles of the local-loss pass
    int rg_lo = 0, rg_hi = 0;  // modules of the readout-gradient pass
    int bg_lo = 0, bg_hi = 0;  // modules of the bias-gradient pass
    int hg_lo = 0, hg_hi = 0;  // modules whose gain-scaled copy the matrix-core gradient passes stream
    int nhead_tiles = 0;       // tiled copies of the heads' readouts (0: the heads read W's copy)
    int rows = 0;              // token rows per tile of the local-loss pass
    bool rot = false;          // ROT heads: modules 0..K-2 read Wbar R_k through rotated rows
    size_t rstd = 0, lse = 0, rowloss = 0, rowrec = 0, rowdtau = 0, dgp = 0, hg = 0;
    size_t wtile = 0, whtile = 0, total = 0;
    // ROT pieces: a vector of ones (the rotated rows' gain), the rotated rows
    // u, the heads' e = sum_v delta_v Wbar_v (4 bytes per element: two bf16
    // planes, or fp32 on the vector-ALU family), D = e R_k (fp32), R_k^T
    size_t ones = 0, ubuf = 0, ebuf = 0, dbuf = 0, rtr = 0;
};

// Which passes stream tiled copies: every pass of the wide tiling; in the
// 16-row tiling the passes without a second product (exit evaluation, bias
// gradient), which read their operand straight into registers.  The others
// (and the vector-ALU family) read the row-major matrices.
bool tiled_readout(const Plan& P) { return P.wide || (P.mfma && P.eval); }
bool tiled_rgrad(const Plan& P) { return P.wide; }

// Sizes, dtype and flags only (no pointer is dereferenced).
bool make_plan(const solo_readout_args& a, bool eval, Plan* P) {
    if (a.dtype != SOLO_BF16 && a.dtype != SOLO_F32) return false;
    if (!shape_ok(a.K, a.T, a.d, a.V)) return false;
    if (!flag_ok(a.gain_per_module) || !flag_ok(a.readout_per_head) || !flag_ok(a.final_module_dW) ||
        !flag_ok(a.heads_train_readout))
        return false;
    if (a.rot && a.readout_per_head) return false;
    const int K = a.K, T = a.T, d = a.d;
    P->wide = solo::mfma_wide_supported(a.dtype, d);
    P->mfma = solo::mfma_supported(a.dtype, d) || P->wide;
    P->eval = eval;
    const size_t kt = (size_t)K * T;
    size_t off = 0;
    P->rstd = off;
    off = align_up(off + kt * 4);
    P->lse = off;
    off = align_up(off + kt * 4);
    P->rowloss = off;
    off = align_up(off + kt * 4);
    // tiled copies of the readouts the local-loss pass and exit evaluation
    // stream: the terminal's W, and the heads' own matrix or matrices
    if (tiled_readout(*P)) {
        const size_t tv = (size_t)solo::tiled_elems(a.V, d) * 2;
        P->nhead_tiles = (a.Wbar && K > 1) ? (a.readout_per_head ? K - 1 : 1) : 0;
        P->wtile = off;
        off = align_up(off + tv);
        P->whtile = off;
        off = align_up(off + tv * P->nhead_tiles);
    }
    const int rows = P->wide ? solo::kMfmaWideRows : (P->mfma ? solo::mfma_rows(d) : solo::kValuRows);
    P->rows = rows;
    P->ntiles = (T + rows - 1) / rows;
    P->rot = a.rot != nullptr && K > 1;
    if (P->rot) {
        const size_t es = a.dtype == SOLO_BF16 ? 2 : 4;
        const size_t htd = (size_t)(K - 1) * T * d;
        P->ones = off;
        off = align_up(off + (size_t)d * es);
        P->ubuf = off;
        off = align_up(off + htd * es);
        if (!eval) {
            P->ebuf = off;
            off = align_up(off + htd * 4);
            P->dbuf = off;
            off = align_up(off + htd * 4);
            P->rtr = off;
            off = align_up(off + (size_t)(K - 1) * d * d * es);
        }
    }
    if (eval) {
        P->total = off;
        return true;
    }
    const bool priv = a.heads_train_readout && K > 1;
    const bool fdw = a.final_module_dW;
    // readout-gradient modules: the terminal if its dW is asked for, the heads under PRIV
    P->rg_lo = priv ? 0 : K - 1;
    P->rg_hi = fdw ? K : (priv ? K - 1 : K - 1);
    if (!fdw && !priv) P->rg_lo = P->rg_hi = 0;
    // bias-gradient modules: every other module, if the bias gradient is asked for
    if (a.dbias) {
        if (P->rg_hi == P->rg_lo) {
            P->bg_lo = 0;
            P->bg_hi = K;
        } else if (P->rg_lo == 0 && P->rg_hi == K) {
            P->bg_lo = P->bg_hi = 0;
        } else if (P->rg_lo == 0) {
            P->bg_lo = K - 1;
            P->bg_hi = K;
        } else {
            P->bg_lo = 0;
            P->bg_hi = K - 1;
        }
    }
    P->ext = a.bias != nullptr;
    P->dg_mode = a.gain_per_module ? 2 : (fdw ? 1 : 0);
    P->slots = P->dg_mode == 2 ? K : (P->dg_mode == 1 ? 1 : 0);
    const bool second = P->rg_hi > P->rg_lo || P->bg_hi > P->bg_lo;
    if (P->mfma && second) {
        // the two ranges are disjoint parts of [0, K): their union is one range
        const bool rg = P->rg_hi > P->rg_lo, bg = P->bg_hi > P->bg_lo;
        P->hg_lo = rg && bg ? (P->rg_lo < P->bg_lo ? P->rg_lo : P->bg_lo) : (rg ? P->rg_lo : P->bg_lo);
        P->hg_hi = rg && bg ? (P->rg_hi > P->bg_hi ? P->rg_hi : P->bg_hi) : (rg ? P->rg_hi : P->bg_hi);
    }
    P->rowrec = off;
    off = align_up(off + (second ? kt * 16 : 0));
    P->hg = off;
    off = align_up(off + (size_t)(P->hg_hi - P->hg_lo) * (size_t)solo::tiled_elems(T, d) * 2);
    P->rowdtau = off;
    off = align_up(off + (a.dtau ? kt * 4 : 0));
    P->dgp = off;
    off = align_up(off + (size_t)P->slots * P->ntiles * d * 4);
    P->total = off;
    return true;
}

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }
bool aligned_or_null(const void* p, uintptr_t a) { return !p || aligned(p, a); }

int check(const solo_readout_args& a, bool eval, Plan* P) {
    if (a.dtype != SOLO_BF16 && a.dtype != SOLO_F32) return SOLO_ERR_DTYPE;
    if (!shape_ok(a.K, a.T, a.d, a.V)) return SOLO_ERR_SHAPE;
    if (!std::isfinite(a.eps) || a.eps < 0.f) return SOLO_ERR_ARG;
    if (!flag_ok(a.gain_per_module) || !flag_ok(a.readout_per_head) || !flag_ok(a.final_module_dW) ||
        !flag_ok(a.heads_train_readout))
        return SOLO_ERR_ARG;
    if (a.readout_per_head && !a.Wbar) return SOLO_ERR_ARG;
    if (a.heads_train_readout && !a.readout_per_head) return SOLO_ERR_ARG;
    if (a.rot && a.readout_per_head) return SOLO_ERR_ARG;
    if (!a.h || !a.gain || !a.W || !a.targets || !a.losses || !a.workspace) return SOLO_ERR_NULL;
    if (!eval) {
        if (!a.dh) return SOLO_ERR_NULL;
        if (a.final_module_dW && !a.dW) return SOLO_ERR_NULL;
        if (a.heads_train_readout && a.K > 1 && !a.dWbar) return SOLO_ERR_NULL;
        if ((a.gain_per_module || a.final_module_dW) && !a.dgain) return SOLO_ERR_NULL;
    }
    if (!aligned(a.h, 16) || !aligned(a.gain, 16) || !aligned(a.W, 16) || !aligned_or_null(a.Wbar, 16) ||
        !aligned(a.targets, 4) || !aligned(a.losses, 4) || !aligned_or_null(a.row_loss, 4) ||
        !aligned_or_null(a.tau, 4) || !aligned_or_null(a.bias, 4) || !aligned_or_null(a.rot, 16) ||
        !aligned(a.workspace, kAlign))
        return SOLO_ERR_ALIGN;
    if (eval) {
        if (!aligned_or_null(a.top1, 4)) return SOLO_ERR_ALIGN;
    } else {
        if (!aligned(a.dh, 16) || !aligned_or_null(a.dtau, 4) || !aligned_or_null(a.dbias, 4))
            return SOLO_ERR_ALIGN;
        if (a.final_module_dW && !aligned(a.dW, 16)) return SOLO_ERR_ALIGN;
        if (a.heads_train_readout && a.K > 1 && !aligned(a.dWbar, 16)) return SOLO_ERR_ALIGN;
        if ((a.gain_per_module || a.final_module_dW) && !aligned(a.dgain, 4)) return SOLO_ERR_ALIGN;
    }
    if (!make_plan(a, eval, P)) return SOLO_ERR_SHAPE;
    if (a.workspace_bytes < P->total) return SOLO_ERR_WORKSPACE;
    return SOLO_OK;
}

int run(const solo_readout_args& x, bool eval) {
    Plan P;
    const int st = check(x, eval, &P);
    if (st != SOLO_OK) return st;
    const int K = x.K, T = x.T, d = x.d, V = x.V;
    hipStream_t s = (hipStream_t)x.hip_stream;
    char* ws = (char*)x.workspace;

    solo::FusedArgs a = {};
    a.K = K;
    a.T = T;
    a.d = d;
    a.V = V;
    a.m0 = 0;
    a.inv_T = (float)(1.0 / (double)T);
    a.h = x.h;
    a.Wt = x.W;
    // heads: W itself, one shared matrix, or one per head
    a.Wh = x.Wbar ? x.Wbar : x.W;
    a.wh_stride = (x.Wbar && x.readout_per_head) ? (long long)V * d : 0;
    a.Wtt = ws + P.wtile;
    a.Wht = P.nhead_tiles ? ws + P.whtile : ws + P.wtile;
    a.wht_stride = P.nhead_tiles > 1 ? solo::tiled_elems(V, d) : 0;
    a.hg = ws + P.hg;
    a.hg_m0 = P.hg_lo;
    a.gain = x.gain;
    a.g_stride = x.gain_per_module ? d : 0;
    a.tau = x.tau;
    a.bias = x.bias;
    a.targets = x.targets;
    a.rstd = (const float*)(ws + P.rstd);
    a.lse = (float*)(ws + P.lse);
    a.rowloss = x.row_loss ? x.row_loss : (float*)(ws + P.rowloss);
    a.rowrec = (!eval && (P.rg_hi > P.rg_lo || P.bg_hi > P.bg_lo)) ? (float*)(ws + P.rowrec) : nullptr;
    a.rowdtau = (!eval && x.dtau) ? (float*)(ws + P.rowdtau) : nullptr;
    a.top1 = eval ? x.top1 : nullptr;
    a.dh = eval ? nullptr : x.dh;
    a.dgain_part = P.slots ? (float*)(ws + P.dgp) : nullptr;
    a.dg_mode = eval ? 0 : P.dg_mode;
    a.dWt = (!eval && x.final_module_dW) ? x.dW : nullptr;
    a.dWh = (!eval && x.heads_train_readout) ? x.dWbar : nullptr;
    a.dbias = eval ? nullptr : x.dbias;

    auto mark = [&](int stage) -> bool {
        if (!x.stage_events || !x.stage_events[stage]) return true;
        return hipEventRecord((hipEvent_t)x.stage_events[stage], s) == hipSuccess;
    };
    const int dt = x.dtype;
    // a failure left pending by earlier work on this thread is not this call's
    (void)hipGetLastError();
    if (solo::launch_row_rstd(dt, x.h, (float*)(ws + P.rstd), (long long)K * T, d, x.eps, s) != hipSuccess)
        return SOLO_ERR_HIP;
    if (tiled_readout(P)) {
        if (solo::launch_tile((const solo::bf16*)x.W, 0, nullptr, 0, (solo::bf16*)(ws + P.wtile), 1, V, d, s) !=
            hipSuccess)
            return SOLO_ERR_HIP;
        if (P.nhead_tiles && solo::launch_tile((const solo::bf16*)x.Wbar, (long long)V * d, nullptr, 0,
                                               (solo::bf16*)(ws + P.whtile), P.nhead_tiles, V, d, s) != hipSuccess)
            return SOLO_ERR_HIP;
    }
    // ROT heads: their stationary rows are u = R_k (g_k * h) (gain one from
    // then on), which the passes of the heads read in place of h
    solo::FusedArgs ah = a;
    if (P.rot) {
        if (solo::launch_fill_one(dt, ws + P.ones, d, s) != hipSuccess) return SOLO_ERR_HIP;
        if (solo::launch_rot_rows(dt, x.h, x.gain, a.g_stride, x.rot, ws + P.ubuf, K - 1, T, d, s) != hipSuccess)
            return SOLO_ERR_HIP;
        ah.h = ws + P.ubuf;
        ah.gain = ws + P.ones;
        ah.g_stride = 0;
        ah.ebuf = eval ? nullptr : (void*)(ws + P.ebuf);
    }
    if (!mark(0)) return SOLO_ERR_HIP;
    // one launch over modules [m0, m0 + n) of a pass, with the arguments g
    auto pass = [&](int which, const solo::FusedArgs& g, int m0, int n) -> hipError_t {
        if (n <= 0) return hipSuccess;
        solo::FusedArgs b = g;
        b.m0 = m0;
        switch (which) {
            case 0:
                return P.wide   ? solo::launch_exit_eval_mfma_wide(b, n, s)
                       : P.mfma ? solo::launch_exit_eval_mfma(b, n, s)
                                : solo::launch_exit_eval_valu(dt, b, n, s);
            case 1:
                return P.wide   ? solo::launch_local_loss_mfma_wide(b, P.ext, n, s)
                       : P.mfma ? solo::launch_local_loss_mfma(b, P.ext, n, s)
                                : solo::launch_local_loss_valu(dt, b, n, s);
            case 2:
                return P.wide   ? solo::launch_readout_grad_mfma_wide(b, n, s)
                       : P.mfma ? solo::launch_readout_grad_mfma(b, n, s)
                                : solo::launch_readout_grad_valu(dt, b, n, s);
            default:
                return P.wide   ? solo::launch_bias_grad_mfma_wide(b, n, s)
                       : P.mfma ? solo::launch_bias_grad_mfma(b, n, s)
                                : solo::launch_bias_grad_valu(dt, b, n, s);
        }
    };
    // modules [lo, hi) of a pass: under ROT the heads and the terminal are two launches
    auto pass_range = [&](int which, int lo, int hi) -> bool {
        if (!P.rot || hi <= K - 1 || lo >= K - 1) return pass(which, P.rot && lo < K - 1 ? ah : a, lo, hi - lo) == hipSuccess;
        return pass(which, ah, lo, K - 1 - lo) == hipSuccess && pass(which, a, K - 1, hi - K + 1) == hipSuccess;
    };
    if (!pass_range(eval ? 0 : 1, 0, K)) return SOLO_ERR_HIP;
    if (P.rot && !eval) {
        // back to the basis of h: D = e R_k = e (R_k^T)^T, then the heads' RMSNorm
        // backward (and their gain partials when every module trains its gain)
        if (solo::launch_transpose(dt, x.rot, ws + P.rtr, K - 1, d, s) != hipSuccess ||
            solo::launch_rot_back(dt, P.mfma, ws + P.ebuf, ws + P.rtr, (float*)(ws + P.dbuf), K - 1, T, d, s) !=
                hipSuccess ||
            solo::launch_rot_post(dt, (const float*)(ws + P.dbuf), x.h, x.gain, a.g_stride, (const float*)(ws + P.rstd),
                                  x.tau, x.dh, P.dg_mode == 2 ? a.dgain_part : nullptr, K - 1, T, d, P.rows,
                                  s) != hipSuccess)
            return SOLO_ERR_HIP;
    }
    if (!mark(1)) return SOLO_ERR_HIP;
    if (solo::launch_module_sum(a.rowloss, x.losses, K, T, 1.0 / (double)T, s) != hipSuccess) return SOLO_ERR_HIP;
    if (a.rowdtau && solo::launch_module_sum(a.rowdtau, x.dtau, K, T, 1.0, s) != hipSuccess) return SOLO_ERR_HIP;
    if (!mark(2)) return SOLO_ERR_HIP;
    // the gain-scaled copies of h the gradient passes stream, module m at
    // hg + (m - hg_lo) tiled_elems(T, d): tiled for the register-fed passes,
    // row-major for the direct-to-LDS readout-gradient pass
    // (ROT heads: of their rotated rows, times the gain of ones)
    auto copies = [&](const solo::FusedArgs& g, int lo, int hi, bool as_tiles) -> bool {
        if (hi <= lo) return true;
        const solo::bf16* src = (const solo::bf16*)g.h + (long long)lo * T * d;
        const solo::bf16* gn = (const solo::bf16*)g.gain + (long long)lo * g.g_stride;
        solo::bf16* dst = (solo::bf16*)(ws + P.hg) + (long long)(lo - P.hg_lo) * solo::tiled_elems(T, d);
        return (as_tiles ? solo::launch_tile(src, (long long)T * d, gn, g.g_stride, dst, hi - lo, T, d, s)
                         : solo::launch_gain_rows(src, (long long)T * d, gn, g.g_stride, dst,
                                                  solo::tiled_elems(T, d), hi - lo, T, d, s)) == hipSuccess;
    };
    auto gain_copies = [&](int lo, int hi, bool as_tiles) -> bool {
        if (!P.rot || hi <= K - 1 || lo >= K - 1) return copies(P.rot && lo < K - 1 ? ah : a, lo, hi, as_tiles);
        return copies(ah, lo, K - 1, as_tiles) && copies(a, K - 1, hi, as_tiles);
    };
    if (!eval && P.mfma &&
        (!gain_copies(P.rg_lo, P.rg_hi, tiled_rgrad(P)) || !gain_copies(P.bg_lo, P.bg_hi, true)))
        return SOLO_ERR_HIP;
    if (!eval && !pass_range(2, P.rg_lo, P.rg_hi)) return SOLO_ERR_HIP;
    if (!mark(3)) return SOLO_ERR_HIP;
    if (!eval && !pass_range(3, P.bg_lo, P.bg_hi)) return SOLO_ERR_HIP;
    if (!mark(4)) return SOLO_ERR_HIP;
    if (!eval && P.slots) {
        if (solo::launch_dgain_reduce(a.dgain_part, x.dgain, P.slots, P.ntiles, d, s) != hipSuccess)
            return SOLO_ERR_HIP;
    }
    if (!mark(5)) return SOLO_ERR_HIP;
    return SOLO_OK;
}

solo_readout_args headline(int K, int T, int d, int V, int dtype, float eps, const void* h, const void* gain,
                           const void* W, const int32_t* targets, int final_module_dW, float* losses,
                           float* row_loss, void* dh, float* dW, float* dgain, void* workspace,
                           size_t workspace_bytes, void* hip_stream, void* const* stage_events) {
    solo_readout_args a = {};
    a.K = K;
    a.T = T;
    a.d = d;
    a.V = V;
    a.dtype = dtype;
    a.eps = eps;
    a.h = h;
    a.gain = gain;
    a.W = W;
    a.targets = targets;
    a.final_module_dW = final_module_dW;
    a.losses = losses;
    a.row_loss = row_loss;
    a.dh = dh;
    a.dW = dW;
    a.dgain = dgain;
    a.workspace = workspace;
    a.workspace_bytes = workspace_bytes;
    a.hip_stream = hip_stream;
    a.stage_events = stage_events;
    return a;
}

// Scratch of the entry point that allocates nothing: a file-scope device
// array, one copy per GPU, held until the process ends.  Host code never
// passes the array's name to a kernel (on the host it is a stand-in, not a
// device address): the device address is fetched once per device, with that
// device current, and kept.
constexpr size_t kScratchBytes = size_t(128) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void* scratch_ptr[kMaxDevices] = {};

// The current device's scratch address (nullptr on a HIP error).
void* scratch_of_current_device() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (!scratch_ptr[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
        scratch_ptr[dev] = ptr;
    }
    return scratch_ptr[dev];
}

}  // namespace

extern "C" {

size_t solo_readout_scratch_limit(void) { return kScratchBytes; }

int solo_readout_fwd_bwd_noalloc(int K, int T, int d, int V, int dtype, float eps, const void* h, const void* gain,
                                 const void* W, const int32_t* targets, int final_module_dW, float* losses,
                                 float* row_loss, void* dh, float* dW, float* dgain, void* hip_stream) {
    if (dtype != SOLO_BF16 && dtype != SOLO_F32) return SOLO_ERR_DTYPE;
    if (!shape_ok(K, T, d, V)) return SOLO_ERR_SHAPE;
    solo_readout_args a = headline(K, T, d, V, dtype, eps, h, gain, W, targets, final_module_dW, losses, row_loss,
                                   dh, dW, dgain, nullptr, 0, hip_stream, nullptr);
    Plan P;
    if (!make_plan(a, false, &P)) return SOLO_ERR_SHAPE;
    if (P.total > kScratchBytes) return SOLO_ERR_WORKSPACE;
    // every other host check before the first HIP call (a stand-in, aligned
    // workspace of the limit's size: only the scratch's address is unknown yet)
    a.workspace = (void*)(uintptr_t)kAlign;
    a.workspace_bytes = kScratchBytes;
    const int st = check(a, false, &P);
    if (st != SOLO_OK) return st;
    (void)hipGetLastError();
    void* ws = scratch_of_current_device();
    if (!ws) return SOLO_ERR_HIP;
    a.workspace = ws;
    a.workspace_bytes = kScratchBytes;
    return run(a, false);
}

int solo_readout_abi_version(void) { return SOLO_READOUT_ABI_VERSION; }

const char* solo_status_string(int status) {
    switch (status) {
        case SOLO_OK: return "ok";
        case SOLO_ERR_NULL: return "a required pointer is NULL";
        case SOLO_ERR_SHAPE: return "invalid sizes (need K,T,V >= 1, 8 <= d <= 4096, d % 8 == 0, K <= 65535, K*T < 2^31)";
        case SOLO_ERR_DTYPE: return "unknown dtype";
        case SOLO_ERR_ALIGN: return "misaligned pointer";
        case SOLO_ERR_WORKSPACE: return "workspace too small";
        case SOLO_ERR_ARG:
            return "invalid argument (eps must be finite and >= 0; flags must be 0 or 1; readout_per_head needs "
                   "Wbar; heads_train_readout needs readout_per_head; rot excludes readout_per_head)";
        case SOLO_ERR_HIP: return "HIP launch failed";
        default: return "unknown status";
    }
}

size_t solo_readout_workspace_size(int K, int T, int d, int V, int dtype, int final_module_dW) {
    const solo_readout_args a = headline(K, T, d, V, dtype, 0.f, nullptr, nullptr, nullptr, nullptr, final_module_dW,
                                         nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0, nullptr, nullptr);
    Plan P;
    return make_plan(a, false, &P) ? P.total : 0;
}

const char* solo_readout_kernel_family(int K, int T, int d, int V, int dtype) {
    if ((dtype != SOLO_BF16 && dtype != SOLO_F32) || !shape_ok(K, T, d, V)) return "invalid";
    if (solo::mfma_wide_supported(dtype, d)) return "mfma_wide";
    return solo::mfma_supported(dtype, d) ? "mfma" : "valu";
}

int solo_readout_fwd_bwd(int K, int T, int d, int V, int dtype, float eps, const void* h, const void* gain,
                         const void* W, const int32_t* targets, int final_module_dW, float* losses, float* row_loss,
                         void* dh, float* dW, float* dgain, void* workspace, size_t workspace_bytes,
                         void* hip_stream) {
    return solo_readout_fwd_bwd_profiled(K, T, d, V, dtype, eps, h, gain, W, targets, final_module_dW, losses,
                                         row_loss, dh, dW, dgain, workspace, workspace_bytes, hip_stream, nullptr);
}

int solo_readout_fwd_bwd_profiled(int K, int T, int d, int V, int dtype, float eps, const void* h, const void* gain,
                                  const void* W, const int32_t* targets, int final_module_dW, float* losses,
                                  float* row_loss, void* dh, float* dW, float* dgain, void* workspace,
                                  size_t workspace_bytes, void* hip_stream, void* const* stage_events) {
    if (dtype != SOLO_BF16 && dtype != SOLO_F32) return SOLO_ERR_DTYPE;
    if (!shape_ok(K, T, d, V)) return SOLO_ERR_SHAPE;
    const solo_readout_args a = headline(K, T, d, V, dtype, eps, h, gain, W, targets, final_module_dW, losses,
                                         row_loss, dh, dW, dgain, workspace, workspace_bytes, hip_stream,
                                         stage_events);
    return run(a, false);
}

size_t solo_readout_general_workspace_size(const solo_readout_args* args) {
    Plan P;
    return (args && make_plan(*args, false, &P)) ? P.total : 0;
}

int solo_readout_general(const solo_readout_args* args) {
    if (!args) return SOLO_ERR_NULL;
    return run(*args, false);
}

size_t solo_readout_exit_eval_workspace_size(const solo_readout_args* args) {
    Plan P;
    return (args && make_plan(*args, true, &P)) ? P.total : 0;
}

int solo_readout_exit_eval(const solo_readout_args* args) {
    if (!args) return SOLO_ERR_NULL;
    return run(*args, true);
}

}  // extern "C"
