"""The allocation-free entry point (solo_readout_fwd_bwd_noalloc) against the
workspace entry point (solo_readout_fwd_bwd) through the C ABI: the same
kernels on the same inputs give the same bits, on two calls in a row (the
second smaller, so the library's scratch still holds the first call's
contents), for both matrix-core tilings and the fp32 family; a call that
needs more than the scratch limit is refused before anything is enqueued."""
import numpy as np
import pytest

from solo_inputs import make_inputs
from tests.gpu_helpers import log, run_gpu, to_device

pytestmark = pytest.mark.gpu


def _noalloc(x, final_module_dW=True, eps=1e-6):
    import torch

    from paper_2609_35440_amd import binding

    h, gain, W, targets = to_device(x)
    K, T, d = h.shape
    V = W.shape[0]
    dev = h.device
    losses = torch.empty(K, dtype=torch.float32, device=dev)
    row_loss = torch.empty((K, T), dtype=torch.float32, device=dev)
    dh = torch.empty_like(h)
    dW = torch.empty((V, d), dtype=torch.float32, device=dev)
    dgain = torch.empty(d, dtype=torch.float32, device=dev)
    dt = binding.SOLO_BF16 if h.dtype == torch.bfloat16 else binding.SOLO_F32
    st = binding.readout_fwd_bwd_noalloc_raw(K, T, d, V, dt, eps, h.data_ptr(), gain.data_ptr(), W.data_ptr(),
                                             targets.data_ptr(), int(final_module_dW), losses.data_ptr(),
                                             row_loss.data_ptr(), dh.data_ptr(), dW.data_ptr(), dgain.data_ptr(),
                                             torch.cuda.current_stream().cuda_stream)
    assert st == 0, binding.status_string(st)
    torch.cuda.synchronize()
    return {"losses": losses.double().cpu().numpy(), "row_loss": row_loss.double().cpu().numpy(),
            "dh": dh.float().cpu().numpy().astype(np.float64), "dW": dW.double().cpu().numpy(),
            "dgain": dgain.double().cpu().numpy()}


# (config, first call's sizes, second call's smaller sizes)
CASES = [("1b", dict(K=3, T=300, d=2048, V=1000), dict(K=2, T=70, d=2048, V=300)),
         ("2b", dict(K=3, T=100, d=2560, V=500), dict(K=2, T=37, d=2560, V=130)),
         ("tiny", dict(K=2, T=256, d=64, V=512), dict(K=1, T=33, d=64, V=45))]


@pytest.mark.parametrize("cfg,first,second", CASES, ids=[c[0] for c in CASES])
def test_noalloc_matches_workspace_entry_point(cfg, first, second):
    for i, ov in enumerate((first, second)):
        x = make_inputs(cfg, seed=61 + i, **ov)
        log(f"no-alloc {cfg} call {i}: {ov}")
        a = _noalloc(x)
        b = run_gpu(x, True)
        for key in ("losses", "row_loss", "dh", "dW", "dgain"):
            np.testing.assert_array_equal(a[key], b[key], err_msg=f"{cfg} call {i} {key}")


def test_noalloc_refuses_calls_beyond_the_scratch():
    import torch

    from paper_2609_35440_amd import binding

    limit = binding.scratch_limit()
    assert limit == 128 << 20
    # the 1B shape with 4 times the tokens needs more than the limit
    K, T, d, V = 4, 65536, 2048, 32000
    need = binding.workspace_size(K, T, d, V, binding.SOLO_BF16, True)
    assert need > limit
    losses = torch.full((K,), 7.0, dtype=torch.float32, device="cuda:0")
    p = losses.data_ptr()
    st = binding.readout_fwd_bwd_noalloc_raw(K, T, d, V, binding.SOLO_BF16, 1e-6, p, p, p, p, 1, p, 0, p, p, p, 0)
    assert st == binding.STATUS["SOLO_ERR_WORKSPACE"]
    torch.cuda.synchronize()
    assert (losses.cpu() == 7.0).all()   # nothing was enqueued


def test_noalloc_under_graph_capture():
    """What the entry point is for: a call captured into a HIP graph (nothing is
    allocated inside the capture; the scratch address was fetched by an earlier
    eager call) and replayed gives the eager call's bits on every replay, with
    the program's own eager work and synchronisations between the replays."""
    import torch

    from paper_2609_35440_amd import binding

    x = make_inputs("1b", seed=71, K=2, T=100, d=2048, V=500)
    h, gain, W, targets = to_device(x)
    K, T, d = h.shape
    V = W.shape[0]
    dev = h.device
    out = {"losses": torch.empty(K, dtype=torch.float32, device=dev),
           "row_loss": torch.empty((K, T), dtype=torch.float32, device=dev),
           "dh": torch.empty_like(h),
           "dW": torch.empty((V, d), dtype=torch.float32, device=dev),
           "dgain": torch.empty(d, dtype=torch.float32, device=dev)}

    def call(stream):
        return binding.readout_fwd_bwd_noalloc_raw(
            K, T, d, V, binding.SOLO_BF16, 1e-6, h.data_ptr(), gain.data_ptr(), W.data_ptr(), targets.data_ptr(), 1,
            out["losses"].data_ptr(), out["row_loss"].data_ptr(), out["dh"].data_ptr(), out["dW"].data_ptr(),
            out["dgain"].data_ptr(), stream.cuda_stream)

    assert call(torch.cuda.current_stream()) == 0
    torch.cuda.synchronize()
    eager = {k: v.clone() for k, v in out.items()}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        st = call(side)
    assert st == 0, binding.status_string(st)
    torch.cuda.synchronize()
    for rep in range(3):
        for v in out.values():
            v.fill_(float("nan"))  # the program's own eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for key, v in out.items():
            assert torch.equal(v, eager[key]), (rep, key)
        log(f"graph replay {rep}: outputs equal the eager call's")
