"""The Python binding's host-side contract on the GPU: calls on a side stream
with inputs that need converting (non-contiguous h, int64 targets) give the
same bits as the plain call, and malformed output, workspace or target
arguments are refused before anything is enqueued."""
import numpy as np
import pytest

from solo_inputs import make_extras, make_inputs
from tests.gpu_helpers import log, to_device

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.float().cpu().numpy()


def test_side_stream_with_converted_inputs_matches_plain_call():
    import torch

    from paper_2609_35440_amd import binding

    x = make_inputs("1b", seed=21, K=2, T=70, d=2048, V=333)
    h, gain, W, targets = to_device(x)
    log("plain call")
    ref = binding.readout_fwd_bwd(h, gain, W, targets, True, row_loss=True)
    torch.cuda.synchronize()
    # the same values through a transposed copy (non-contiguous view) and int64 targets,
    # enqueued on a side stream while the default stream is still busy making them
    side = torch.cuda.Stream()
    h_nc = h.transpose(1, 2).contiguous().transpose(1, 2)
    assert not h_nc.is_contiguous()
    t64 = targets.to(torch.int64)
    log("side-stream call")
    got = binding.readout_fwd_bwd(h_nc, gain, W, t64, True, row_loss=True, stream=side)
    side.synchronize()
    torch.cuda.synchronize()
    for name in ("losses", "row_loss", "dh", "dW", "dgain"):
        np.testing.assert_array_equal(_bits(getattr(got, name)), _bits(getattr(ref, name)), err_msg=name)


def test_general_and_exit_eval_on_side_stream_match_plain_call():
    import torch

    from paper_2609_35440_amd import binding

    from tests.test_gpu_general import _dev

    x = make_extras(make_inputs("1b", seed=22, K=3, T=40, d=2048, V=200), 5, tau=True, bias=True,
                    per_module_gain=True)
    f = _dev(x)
    h, gk, W, targets, tau, bias = f["h"], f["gain"], f["W"], f["targets"], f["tau"], f["bias"]
    assert gk.dim() == 2
    kw = dict(tau=tau, bias=bias, want_dtau=True, want_dbias=True, row_loss=True)
    ref = binding.readout_general(h, gk, W, targets, **kw)
    ev_ref = binding.exit_eval(h, gk, W, targets, tau=tau, bias=bias)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    got = binding.readout_general(h, gk, W, targets.to(torch.int64), stream=side, **kw)
    ev = binding.exit_eval(h, gk, W, targets.to(torch.int64), tau=tau, bias=bias, stream=side)
    side.synchronize()
    for name in ("losses", "row_loss", "dh", "dW", "dgain", "dtau", "dbias"):
        np.testing.assert_array_equal(_bits(getattr(got, name)), _bits(getattr(ref, name)), err_msg=name)
    for name in ("losses", "row_loss", "top1"):
        np.testing.assert_array_equal(getattr(ev, name).cpu().numpy(), getattr(ev_ref, name).cpu().numpy(),
                                      err_msg=name)


def test_malformed_arguments_are_refused_before_launch():
    import torch

    from paper_2609_35440_amd import binding

    x = make_inputs("340m", seed=23, K=2, T=32, d=256, V=100)
    h, gain, W, targets = to_device(x)
    dev = h.device
    K, T, d, V = 2, 32, 256, 100
    f32 = dict(dtype=torch.float32, device=dev)
    good = binding.ReadoutResult(losses=torch.empty(K, **f32), dh=torch.empty_like(h),
                                 dW=torch.empty((V, d), **f32), dgain=torch.empty(d, **f32), row_loss=None)
    bad_outs = {
        "dh too small": good._replace(dh=torch.empty((K, T - 1, d), dtype=h.dtype, device=dev)),
        "dh wrong dtype": good._replace(dh=torch.empty((K, T, d), **f32)),
        "dW missing": good._replace(dW=None),
        "dW non-contiguous": good._replace(dW=torch.empty((d, V), **f32).t()),
        "dgain too small": good._replace(dgain=torch.empty(d - 8, **f32)),
        "row_loss wrong shape": good._replace(row_loss=torch.empty((K, T + 1), **f32)),
    }
    for what, out in bad_outs.items():
        with pytest.raises(ValueError):
            binding.readout_fwd_bwd(h, gain, W, targets, True, out=out)
        log(f"refused: {what}")
    with pytest.raises(TypeError):
        binding.readout_fwd_bwd(h, gain, W, targets.float(), True)
    with pytest.raises(ValueError):
        ws = torch.empty(2 * binding.workspace_size(K, T, d, V, binding.SOLO_BF16, True), dtype=torch.uint8,
                         device=dev)[::2]
        binding.readout_fwd_bwd(h, gain, W, targets, True, workspace=ws)
    with pytest.raises(ValueError):
        binding.exit_eval(h, gain, W, targets, out=binding.EvalResult(
            losses=torch.empty(K, **f32), row_loss=None, top1=torch.empty((K, T), **f32)))
    # the well-formed outputs still work after the refusals
    torch.cuda.synchronize()
    r = binding.readout_fwd_bwd(h, gain, W, targets, True, out=good)
    torch.cuda.synchronize()
    assert np.all(np.isfinite(r.losses.cpu().numpy()))
