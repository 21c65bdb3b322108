// C ABI of the SOLO shared-readout local loss: argument checks, workspace
// layout and the launch sequence on the caller's stream.
#include <cmath>
#include <cstdint>

#include "solo_readout.h"
#include "solo_internal.h"

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Layout {
    size_t wg, rstd, lse, rowloss, rowrec, dgp, total;
    int ntiles;
    bool mfma;
};

bool shape_ok(int K, int T, int d, int V) {
    if (K < 1 || T < 1 || V < 1) return false;
    if (d < 8 || d % 8 != 0 || d > 4096) return false;
    if (K > 65535 || T > (1 << 30) || V > (1 << 30)) return false;
    if ((long long)K * (long long)T > 2147483647LL) return false;
    return true;
}

bool make_layout(int K, int T, int d, int V, int dtype, int fdw, Layout* L) {
    if (dtype != SOLO_BF16 && dtype != SOLO_F32) return false;
    if (!shape_ok(K, T, d, V)) return false;
    const size_t elem = dtype == SOLO_BF16 ? 2 : 4;
    L->mfma = solo::mfma_supported(dtype, d);
    const int vtile = L->mfma ? solo::kMfmaRows : solo::kValuRows;
    size_t off = 0;
    L->wg = off;
    off = align_up(off + (size_t)V * d * elem);
    L->rstd = off;
    off = align_up(off + (size_t)K * T * 4);
    L->lse = off;
    off = align_up(off + (size_t)K * T * 4);
    L->rowloss = off;
    off = align_up(off + (size_t)K * T * 4);
    L->rowrec = off;
    off = align_up(off + (fdw ? (size_t)T * 16 : 0));
    L->ntiles = fdw ? (V + vtile - 1) / vtile : 0;
    L->dgp = off;
    off = align_up(off + (size_t)L->ntiles * d * 4);
    L->total = off;
    return true;
}

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

}  // namespace

extern "C" {

int solo_readout_abi_version(void) { return SOLO_READOUT_ABI_VERSION; }

const char* solo_status_string(int status) {
    switch (status) {
        case SOLO_OK: return "ok";
        case SOLO_ERR_NULL: return "a required pointer is NULL";
        case SOLO_ERR_SHAPE: return "invalid sizes (need K,T,V >= 1, 8 <= d <= 4096, d % 8 == 0, K <= 65535, K*T < 2^31)";
        case SOLO_ERR_DTYPE: return "unknown dtype";
        case SOLO_ERR_ALIGN: return "misaligned pointer";
        case SOLO_ERR_WORKSPACE: return "workspace too small";
        case SOLO_ERR_ARG: return "invalid argument (eps must be finite and >= 0; final_module_dW must be 0 or 1)";
        case SOLO_ERR_HIP: return "HIP launch failed";
        default: return "unknown status";
    }
}

size_t solo_readout_workspace_size(int K, int T, int d, int V, int dtype, int final_module_dW) {
    if (final_module_dW != 0 && final_module_dW != 1) return 0;
    Layout L;
    if (!make_layout(K, T, d, V, dtype, final_module_dW, &L)) return 0;
    return L.total;
}

const char* solo_readout_kernel_family(int K, int T, int d, int V, int dtype) {
    Layout L;
    if (!make_layout(K, T, d, V, dtype, 0, &L)) return "invalid";
    return L.mfma ? "mfma" : "valu";
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
    if (!std::isfinite(eps) || eps < 0.f) return SOLO_ERR_ARG;
    if (final_module_dW != 0 && final_module_dW != 1) return SOLO_ERR_ARG;
    if (!h || !gain || !W || !targets || !losses || !dh || !workspace) return SOLO_ERR_NULL;
    if (final_module_dW && (!dW || !dgain)) return SOLO_ERR_NULL;
    if (!aligned(h, 16) || !aligned(gain, 16) || !aligned(W, 16) || !aligned(dh, 16) || !aligned(targets, 4) ||
        !aligned(losses, 4) || (row_loss && !aligned(row_loss, 4)) || !aligned(workspace, kAlign))
        return SOLO_ERR_ALIGN;
    if (final_module_dW && (!aligned(dW, 16) || !aligned(dgain, 4))) return SOLO_ERR_ALIGN;
    Layout L;
    if (!make_layout(K, T, d, V, dtype, final_module_dW, &L)) return SOLO_ERR_SHAPE;
    if (workspace_bytes < L.total) return SOLO_ERR_WORKSPACE;

    hipStream_t s = (hipStream_t)hip_stream;
    char* ws = (char*)workspace;
    solo::FusedArgs a;
    a.K = K;
    a.T = T;
    a.d = d;
    a.V = V;
    a.inv_T = (float)(1.0 / (double)T);
    a.h = h;
    a.Wg = ws + L.wg;
    a.W = W;
    a.gain = gain;
    a.targets = targets;
    a.rstd = (const float*)(ws + L.rstd);
    a.lse = (float*)(ws + L.lse);
    a.rowloss = row_loss ? row_loss : (float*)(ws + L.rowloss);
    a.rowrec = final_module_dW ? (float*)(ws + L.rowrec) : nullptr;
    a.dh = dh;
    a.dW = final_module_dW ? dW : nullptr;
    a.dgain_part = (float*)(ws + L.dgp);

    auto mark = [&](int stage) -> bool {
        if (!stage_events || !stage_events[stage]) return true;
        return hipEventRecord((hipEvent_t)stage_events[stage], s) == hipSuccess;
    };
    if (solo::launch_prep_readout(dtype, W, gain, ws + L.wg, V, d, s) != hipSuccess || !mark(0)) return SOLO_ERR_HIP;
    if (solo::launch_row_rstd(dtype, h, (float*)(ws + L.rstd), (long long)K * T, d, eps, s) != hipSuccess || !mark(1))
        return SOLO_ERR_HIP;
    hipError_t e = L.mfma ? solo::launch_local_loss_mfma(a, s) : solo::launch_local_loss_valu(dtype, a, s);
    if (e != hipSuccess || !mark(2)) return SOLO_ERR_HIP;
    if (solo::launch_module_loss(a.rowloss, losses, K, T, s) != hipSuccess || !mark(3)) return SOLO_ERR_HIP;
    if (final_module_dW) {
        e = L.mfma ? solo::launch_readout_grad_mfma(a, s) : solo::launch_readout_grad_valu(dtype, a, s);
        if (e != hipSuccess || !mark(4)) return SOLO_ERR_HIP;
        if (solo::launch_dgain_reduce(a.dgain_part, dgain, L.ntiles, d, s) != hipSuccess || !mark(5))
            return SOLO_ERR_HIP;
    }
    return SOLO_OK;
}

}  // extern "C"
