"""Host-side checks of the C ABI: the library loads, exports what the header
declares, sizes its workspace without a T*V term, and rejects bad arguments
on the host before any launch (these calls never reach the GPU)."""
import ctypes
import os
import subprocess

import pytest

from paper_2609_35440_amd import binding as B

LIB = B.library_path()
pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="library not built (run __graft_entry__.build())")

# fake, aligned, never dereferenced: every call below fails validation first
P = 0x10000
WS = 1 << 40


def call(**kw):
    args = dict(K=2, T=8, d=64, V=32, dtype=B.SOLO_BF16, eps=1e-6, h=P, gain=P, W=P, targets=P, final_module_dW=1,
                losses=P, row_loss=0, dh=P, dW=P, dgain=P, workspace=P, workspace_bytes=WS, stream=0)
    args.update(kw)
    return B.readout_fwd_bwd_raw(**args)


def test_exports_match_header():
    names = B.header_functions()
    assert set(names) == {"solo_readout_abi_version", "solo_status_string", "solo_readout_workspace_size",
                          "solo_readout_kernel_family", "solo_readout_fwd_bwd", "solo_readout_fwd_bwd_profiled",
                          "solo_readout_general_workspace_size", "solo_readout_general",
                          "solo_readout_exit_eval_workspace_size", "solo_readout_exit_eval",
                          "solo_readout_scratch_limit", "solo_readout_fwd_bwd_noalloc"}
    lib = ctypes.CDLL(LIB)
    for n in names:
        assert hasattr(lib, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True).stdout
    exported = {l.split()[-1] for l in out.splitlines() if " T " in l}
    assert set(names) <= exported
    assert B.abi_version() == 3


def test_status_strings():
    for name, code in B.STATUS.items():
        s = B.status_string(code)
        assert isinstance(s, str) and s
    assert B.status_string(99) == "unknown status"


def al(x):
    return (x + 255) // 256 * 256


def tiled(n, d):
    # bytes of a bf16 tiled copy of an [n][d] matrix: rows padded to chunks of 16
    return -(-n // 16) * 16 * d * 2


def test_workspace_has_no_TV_term():
    # bf16 matrix-core families: rstd, lse, row_loss (3 K T 4) + per-token records of
    # every module (K T 16) + the terminal's bf16 copy of gain * h (T d 2, rows padded
    # to chunks of 16) + its gain-gradient partials (one row of d fp32 per token tile:
    # 64-row tiles at d <= 1024, 32-row tiles up to 2048, 16-row tiles at d = 2560).
    # The wide tiling (d = 2560) also streams a tiled copy of the readout (V d 2).
    # No T x V piece.
    for K, T, d, V, rows in [(4, 16384, 2048, 32000, 32), (2, 32768, 2048, 128256, 32), (4, 8192, 1024, 32000, 64),
                             (1, 1, 256, 1, 64), (3, 100, 1536, 50, 32), (8, 16384, 2560, 32000, 16)]:
        wt = al(tiled(V, d)) if d == 2560 else 0
        want = 3 * al(K * T * 4) + wt + al(K * T * 16) + al(tiled(T, d)) + al(-(-T // rows) * d * 4)
        assert B.workspace_size(K, T, d, V, B.SOLO_BF16, True) == want
        assert B.workspace_size(K, T, d, V, B.SOLO_BF16, False) == 3 * al(K * T * 4) + wt
    # the 16-row tiling's workspace does not depend on V at all; the wide tiling's
    # only through the readout copy
    a = B.workspace_size(4, 16384, 2048, 32000, B.SOLO_BF16, True)
    assert B.workspace_size(4, 16384, 2048, 128256, B.SOLO_BF16, True) == a
    aw = B.workspace_size(8, 16384, 2560, 32000, B.SOLO_BF16, True)
    assert B.workspace_size(8, 16384, 2560, 64000, B.SOLO_BF16, True) - aw == 32000 * 2560 * 2
    # doubling T grows it by K T (12 + 16) + (T/32) d 4 + T d 2 bytes
    b = B.workspace_size(4, 32768, 2048, 32000, B.SOLO_BF16, True)
    assert b - a == 4 * 16384 * 28 + 512 * 2048 * 4 + 16384 * 2048 * 2
    # well below one module's T x V fp32 logits (2.1 GB at the 1B shape)
    assert a < 16384 * 32000 * 4 / 20
    # vector-ALU family: 8-row token tiles, per-token records (p_y - 1 for the readout-gradient pass)
    K, T, d, V = 2, 256, 64, 512
    assert B.workspace_size(K, T, d, V, B.SOLO_F32, True) == 3 * al(K * T * 4) + al(K * T * 16) + al(-(-T // 8) * d * 4)
    # invalid arguments -> 0
    assert B.workspace_size(0, 8, 64, 32, B.SOLO_BF16, True) == 0
    assert B.workspace_size(1, 8, 63, 32, B.SOLO_BF16, True) == 0
    assert B.workspace_size(1, 8, 64, 32, 7, True) == 0
    assert B.workspace_size(1, 8, 64, 32, B.SOLO_BF16, 2) == 0


def test_kernel_family():
    assert B.kernel_family(4, 16384, 2048, 32000, B.SOLO_BF16) == "mfma"
    assert B.kernel_family(4, 8192, 1024, 32000, B.SOLO_BF16) == "mfma"
    assert B.kernel_family(2, 256, 64, 512, B.SOLO_F32) == "valu"
    assert B.kernel_family(8, 16384, 2560, 32000, B.SOLO_BF16) == "mfma_wide"
    assert B.kernel_family(8, 16384, 3072, 32000, B.SOLO_BF16) == "valu"
    assert B.kernel_family(8, 16384, 2560, 32000, B.SOLO_F32) == "valu"
    assert B.kernel_family(1, 1, 72, 3, B.SOLO_BF16) == "valu"
    assert B.kernel_family(0, 1, 64, 3, B.SOLO_BF16) == "invalid"


def test_profiled_entry_point_validates_identically():
    # same host checks; stage events are never touched on an argument error
    for kw, code in [(dict(K=0), "SOLO_ERR_SHAPE"), (dict(h=0), "SOLO_ERR_NULL"), (dict(workspace_bytes=1), "SOLO_ERR_WORKSPACE")]:
        assert call(stage_events=[0x1234] * B.NUM_STAGES, **kw) == B.STATUS[code]


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=2), "SOLO_ERR_DTYPE"),
    (dict(dtype=-1), "SOLO_ERR_DTYPE"),
    (dict(K=0), "SOLO_ERR_SHAPE"),
    (dict(T=0), "SOLO_ERR_SHAPE"),
    (dict(V=0), "SOLO_ERR_SHAPE"),
    (dict(d=0), "SOLO_ERR_SHAPE"),
    (dict(d=60), "SOLO_ERR_SHAPE"),
    (dict(d=4104), "SOLO_ERR_SHAPE"),
    (dict(K=70000), "SOLO_ERR_SHAPE"),
    (dict(K=65535, T=1 << 30), "SOLO_ERR_SHAPE"),
    (dict(eps=-1.0), "SOLO_ERR_ARG"),
    (dict(eps=float("nan")), "SOLO_ERR_ARG"),
    (dict(eps=float("inf")), "SOLO_ERR_ARG"),
    (dict(final_module_dW=2), "SOLO_ERR_ARG"),
    (dict(h=0), "SOLO_ERR_NULL"),
    (dict(gain=0), "SOLO_ERR_NULL"),
    (dict(W=0), "SOLO_ERR_NULL"),
    (dict(targets=0), "SOLO_ERR_NULL"),
    (dict(losses=0), "SOLO_ERR_NULL"),
    (dict(dh=0), "SOLO_ERR_NULL"),
    (dict(workspace=0), "SOLO_ERR_NULL"),
    (dict(dW=0), "SOLO_ERR_NULL"),
    (dict(dgain=0), "SOLO_ERR_NULL"),
    (dict(h=P + 8), "SOLO_ERR_ALIGN"),
    (dict(W=P + 2), "SOLO_ERR_ALIGN"),
    (dict(gain=P + 4), "SOLO_ERR_ALIGN"),
    (dict(dh=P + 8), "SOLO_ERR_ALIGN"),
    (dict(targets=P + 2), "SOLO_ERR_ALIGN"),
    (dict(losses=P + 1), "SOLO_ERR_ALIGN"),
    (dict(row_loss=P + 2), "SOLO_ERR_ALIGN"),
    (dict(workspace=P + 128), "SOLO_ERR_ALIGN"),
    (dict(dW=P + 4), "SOLO_ERR_ALIGN"),
    (dict(dgain=P + 2), "SOLO_ERR_ALIGN"),
    (dict(workspace_bytes=1000), "SOLO_ERR_WORKSPACE"),
])
def test_validation_errors(kw, code):
    assert call(**kw) == B.STATUS[code]


def test_frozen_only_call_ignores_dW_pointers():
    # with final_module_dW = 0, NULL dW/dgain are accepted; the too-small
    # workspace then fails before any launch
    assert call(final_module_dW=0, dW=0, dgain=0, workspace_bytes=16) == B.STATUS["SOLO_ERR_WORKSPACE"]
    assert call(final_module_dW=0, dW=P + 1, dgain=P + 1, workspace_bytes=16) == B.STATUS["SOLO_ERR_WORKSPACE"]


def test_workspace_size_boundary():
    need = B.workspace_size(2, 8, 64, 32, B.SOLO_BF16, True)
    assert call(workspace_bytes=need - 1) == B.STATUS["SOLO_ERR_WORKSPACE"]


# ---- solo_readout_general / solo_readout_exit_eval (host checks only)

def gargs(**kw):
    a = B.SoloReadoutArgs()
    base = dict(K=3, T=40, d=256, V=100, dtype=B.SOLO_BF16, eps=1e-6, h=P, gain=P, W=P, targets=P, losses=P,
                dh=P, dW=P, dgain=P, final_module_dW=1, workspace=P, workspace_bytes=WS)
    base.update(kw)
    for k, v in base.items():
        setattr(a, k, v)
    return a


def test_args_struct_layout_matches_header(tmp_path):
    # offsets of every field as the C compiler lays the struct out
    fields = [f for f, _ in B.SoloReadoutArgs._fields_]
    src = tmp_path / "layout.c"
    body = "\n".join(f'    printf("%s %zu\\n", "{f}", offsetof(solo_readout_args, {f}));' for f in fields)
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "solo_readout.h"\nint main(void) {\n'
                   f'{body}\n    printf("size %zu\\n", sizeof(solo_readout_args));\n    return 0;\n}}\n')
    inc = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", f"-I{inc}", str(src), "-o", str(exe)], check=True)
    got = dict(l.split() for l in subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.splitlines())
    for f in fields:
        assert int(got[f]) == getattr(B.SoloReadoutArgs, f).offset, f
    assert int(got["size"]) == ctypes.sizeof(B.SoloReadoutArgs)


def test_status_values_match_header(tmp_path):
    # the numbering of solo_status as the C compiler sees it (SOLO_ERR_ARG = 6 and
    # SOLO_ERR_HIP = 7 are this boundary's own choice) against the binding's table
    names = sorted(B.STATUS)
    src = tmp_path / "status.c"
    body = "\n".join(f'    printf("{n} %d\\n", (int){n});' for n in names)
    src.write_text('#include <stdio.h>\n#include "solo_readout.h"\nint main(void) {\n'
                   f'{body}\n    printf("ABI %d\\n", SOLO_READOUT_ABI_VERSION);\n    return 0;\n}}\n')
    inc = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
    exe = tmp_path / "status"
    subprocess.run(["gcc", "-std=c99", f"-I{inc}", str(src), "-o", str(exe)], check=True)
    got = dict(l.split() for l in subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.splitlines())
    for n in names:
        assert int(got[n]) == B.STATUS[n], n
    assert B.STATUS["SOLO_ERR_ARG"] == 6 and B.STATUS["SOLO_ERR_HIP"] == 7
    assert int(got["ABI"]) == B.abi_version()


def test_general_workspace_sizes():
    K, T, d, V = 3, 40, 256, 100
    kt = K * T
    tiles = -(-T // 64)  # 64-row token tiles of the matrix-core kernels at d <= 1024
    wt = al(tiled(V, d))  # a tiled copy of a readout (exit evaluation streams it)
    head = B.workspace_size(K, T, d, V, B.SOLO_BF16, True)
    # the headline arguments through the general entry point: same workspace
    assert B.general_workspace_size(gargs()) == head
    # per-module gains: one partial slot per module
    assert B.general_workspace_size(gargs(gain_per_module=1)) == \
        3 * al(kt * 4) + al(kt * 16) + al(tiled(T, d)) + al(K * tiles * d * 4)
    # temperature gradient: per-token shares
    assert B.general_workspace_size(gargs(dtau=P)) == head + al(kt * 4)
    # bias gradient without any readout gradient: records and gain * h copies of all K
    # modules for the bias-gradient pass, no gain partials
    assert B.general_workspace_size(gargs(final_module_dW=0, dW=0, dgain=0, dbias=P)) == \
        3 * al(kt * 4) + al(kt * 16) + al(K * tiled(T, d))
    # a separate copy for the heads: the local-loss pass reads it in place
    assert B.general_workspace_size(gargs(Wbar=P)) == head
    # PRIV: every module's copy
    assert B.general_workspace_size(gargs(heads_train_readout=1, readout_per_head=1, Wbar=P, dWbar=P)) == \
        head - al(tiled(T, d)) + al(K * tiled(T, d))
    # exit evaluation: per-token statistics and the tiled readout it streams; with one
    # readout per head, one tiled copy each
    assert B.exit_eval_workspace_size(gargs()) == 3 * al(kt * 4) + wt
    assert B.exit_eval_workspace_size(gargs(readout_per_head=1, Wbar=P)) == 3 * al(kt * 4) + wt + al((K - 1) * tiled(V, d))
    # the vector-ALU family (fp32) reads the row-major readout: no tiled copies
    assert B.exit_eval_workspace_size(gargs(dtype=B.SOLO_F32)) == 3 * al(kt * 4)
    # ROT: ones (d elements), the heads' rotated rows ((K-1) T d elements); fwd_bwd also
    # e and D ((K-1) T d floats each) and the transposed rotations ((K-1) d^2 elements)
    htd = (K - 1) * T * d
    rot = al(d * 2) + al(htd * 2)
    assert B.exit_eval_workspace_size(gargs(rot=P)) == 3 * al(kt * 4) + wt + rot
    assert B.general_workspace_size(gargs(rot=P)) == head + rot + 2 * al(htd * 4) + al((K - 1) * d * d * 2)
    assert B.exit_eval_workspace_size(gargs(rot=P, dtype=B.SOLO_F32)) == 3 * al(kt * 4) + al(d * 4) + al(htd * 4)
    # one module has no head: rot is ignored
    assert B.general_workspace_size(gargs(K=1, rot=P)) == B.general_workspace_size(gargs(K=1))
    # rejected flags -> 0
    assert B.general_workspace_size(gargs(gain_per_module=2)) == 0
    assert B.general_workspace_size(gargs(rot=P, readout_per_head=1, Wbar=P)) == 0
    assert B.general_workspace_size(gargs(K=0)) == 0


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=5), "SOLO_ERR_DTYPE"),
    (dict(K=0), "SOLO_ERR_SHAPE"),
    (dict(d=100), "SOLO_ERR_SHAPE"),
    (dict(eps=-1.0), "SOLO_ERR_ARG"),
    (dict(gain_per_module=3), "SOLO_ERR_ARG"),
    (dict(readout_per_head=1), "SOLO_ERR_ARG"),                       # per-head readout without Wbar
    (dict(heads_train_readout=1, Wbar=P), "SOLO_ERR_ARG"),            # PRIV without per-head readouts
    (dict(rot=P, readout_per_head=1, Wbar=P), "SOLO_ERR_ARG"),        # ROT rotates one shared readout
    (dict(rot=P + 8), "SOLO_ERR_ALIGN"),
    (dict(h=0), "SOLO_ERR_NULL"),
    (dict(dh=0), "SOLO_ERR_NULL"),
    (dict(dW=0), "SOLO_ERR_NULL"),
    (dict(dgain=0), "SOLO_ERR_NULL"),
    (dict(final_module_dW=0, dgain=0, gain_per_module=1), "SOLO_ERR_NULL"),   # per-module gains need dgain
    (dict(heads_train_readout=1, readout_per_head=1, Wbar=P, dWbar=0), "SOLO_ERR_NULL"),
    (dict(Wbar=P + 8), "SOLO_ERR_ALIGN"),
    (dict(tau=P + 2), "SOLO_ERR_ALIGN"),
    (dict(bias=P + 1), "SOLO_ERR_ALIGN"),
    (dict(dtau=P + 2), "SOLO_ERR_ALIGN"),
    (dict(dbias=P + 2), "SOLO_ERR_ALIGN"),
    (dict(heads_train_readout=1, readout_per_head=1, Wbar=P, dWbar=P + 4), "SOLO_ERR_ALIGN"),
    (dict(workspace_bytes=100), "SOLO_ERR_WORKSPACE"),
])
def test_general_validation_errors(kw, code):
    assert B.readout_general_raw(gargs(**kw)) == B.STATUS[code]


def test_general_null_args_pointer():
    lib = B.load_library()
    assert lib.solo_readout_general(None) == B.STATUS["SOLO_ERR_NULL"]
    assert lib.solo_readout_exit_eval(None) == B.STATUS["SOLO_ERR_NULL"]
    assert lib.solo_readout_general_workspace_size(None) == 0


@pytest.mark.parametrize("kw,code", [
    (dict(h=0), "SOLO_ERR_NULL"),
    (dict(losses=0), "SOLO_ERR_NULL"),
    (dict(top1=P + 2), "SOLO_ERR_ALIGN"),
    (dict(workspace_bytes=10), "SOLO_ERR_WORKSPACE"),
])
def test_exit_eval_validation_errors(kw, code):
    # exit evaluation needs no gradient outputs: dh, dW, dgain may be NULL
    assert B.exit_eval_raw(gargs(dh=0, dW=0, dgain=0, **kw)) == B.STATUS[code]


def test_noalloc_entry_point_validates_on_the_host():
    # argument errors and calls beyond the static scratch are refused before any HIP call
    assert B.scratch_limit() == 128 << 20
    def na(**kw):
        a = dict(K=2, T=8, d=64, V=32, dtype=B.SOLO_BF16, eps=1e-6, h=P, gain=P, W=P, targets=P, final_module_dW=1,
                 losses=P, row_loss=0, dh=P, dW=P, dgain=P, stream=0)
        a.update(kw)
        return B.readout_fwd_bwd_noalloc_raw(**a)
    assert na(dtype=5) == B.STATUS["SOLO_ERR_DTYPE"]
    assert na(K=0) == B.STATUS["SOLO_ERR_SHAPE"]
    assert na(d=60) == B.STATUS["SOLO_ERR_SHAPE"]
    assert na(h=0) == B.STATUS["SOLO_ERR_NULL"]
    assert na(dW=0) == B.STATUS["SOLO_ERR_NULL"]
    assert na(dh=P + 2) == B.STATUS["SOLO_ERR_ALIGN"]
    assert na(eps=-1.0) == B.STATUS["SOLO_ERR_ARG"]
    big = dict(K=4, T=65536, d=2048, V=32000)
    assert B.workspace_size(big["K"], big["T"], big["d"], big["V"], B.SOLO_BF16, True) > B.scratch_limit()
    assert na(**big) == B.STATUS["SOLO_ERR_WORKSPACE"]
