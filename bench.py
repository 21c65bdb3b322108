#!/usr/bin/env python3
"""Throughput of the SOLO shared-readout local loss on one MI355X.

One step = one call of the whole hot path (readout prep, row statistics, the
local-loss pass of all K modules, module losses, the final module's
readout-gradient pass and its gain reduction) over one batch of synthetic
input already resident in HBM.  Default workload: the 1B-class shape
(K=4 modules, T=16384 tokens = 8 x 2048 per module, d=2048, V=32000, bf16).

Prints one JSON line (rank 0, N=1 only).  ``roofline`` is for the dominant
kernel (the local-loss pass), timed live with HIP events recorded on the
library's stream around that stage; ``cpu_baseline`` is the fp64 oracle on
a bounded sample of the same workload, on this host's cores.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6     # MI355X dense bf16 MFMA (256 CU x 4096 flop/clk x 2.4 GHz)
PEAK_HBM_GBS = 8000.0

METRIC = "readout fwd+bwd tokens/sec and % of bf16 MFMA peak (1B-class, V=32000)"


# variant -> (input extras for solo_inputs.make_extras, call flags, description)
VARIANTS = {
    "headline": (None, dict(final_module_dW=True), "SOLO readout, one shared gain, tau = 1, no bias"),
    "tau_bias": (dict(tau=True, bias=True),
                 dict(final_module_dW=True, want_dtau=True, want_dbias=True),
                 "SOLO readout with temperatures and biases and their gradients (heads' bias gradients "
                 "through the bias-gradient pass)"),
    "per_module_gain": (dict(per_module_gain=True, tau=True, bias=True),
                        dict(final_module_dW=True, want_dtau=True, want_dbias=True),
                        "per-module gains, temperatures and biases, all their gradients"),
    "rand": (dict(wbar="per_head", tau=True, bias=True),
             dict(final_module_dW=True, want_dtau=True, want_dbias=True),
             "one frozen readout per head (RAND), temperatures and biases"),
    "priv": (dict(wbar="per_head", tau=True, bias=True),
             dict(final_module_dW=True, heads_train_readout=True, want_dtau=True, want_dbias=True),
             "one trained readout per head (PRIV): every module's readout gradient"),
    "rot": (dict(rot=True, tau=True, bias=True),
            dict(final_module_dW=True, want_dtau=True, want_dbias=True),
            "the shared readout in a fixed orthogonal basis per head (ROT, Wbar R_k), temperatures and biases"),
    "exit_eval": (dict(), None, "forward-only exit evaluation: losses and top-1 of every exit"),
}


def _hip():
    import torch  # noqa: F401  (same HIP runtime as torch)

    lib = ctypes.CDLL("libamdhip64.so.7")
    lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
    lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
    lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    lib.hipEventSynchronize.argtypes = [ctypes.c_void_p]
    lib.hipMemGetInfo.argtypes = [ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(ctypes.c_size_t)]
    return lib


class EventSet:
    """NUM_STAGES + 1 hipEvents per step: a start event and one after each stage."""

    def __init__(self, hip, n):
        self.hip = hip
        self.ev = []
        for _ in range(n):
            e = ctypes.c_void_p()
            assert hip.hipEventCreate(ctypes.byref(e)) == 0
            self.ev.append(e.value)

    def elapsed(self, a, b) -> float:
        ms = ctypes.c_float()
        assert self.hip.hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(self.ev[a]), ctypes.c_void_p(self.ev[b])) == 0
        return float(ms.value)

    def destroy(self):
        for e in self.ev:
            self.hip.hipEventDestroy(ctypes.c_void_p(e))


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg_name: str, sample_T: int, seed: int = 0, variant: str = "headline") -> dict:
    """fp64 oracle on the same workload restricted to sample_T tokens per module."""
    import numpy as np

    import oracle
    from solo_inputs import make_inputs

    try:
        from threadpoolctl import threadpool_info

        threads = max([i.get("num_threads", 0) for i in threadpool_info() if i.get("user_api") == "blas"] or [0])
    except Exception:
        threads = 0
    if not threads:
        threads = len(os.sched_getaffinity(0))
    x = make_inputs(cfg_name, seed=seed, T=sample_T)
    h = x["h"].astype(np.float64)
    W = x["W"].astype(np.float64)
    g = x["gain"].astype(np.float64)
    extras, flags, _ = VARIANTS[variant]
    t0 = time.perf_counter()
    if extras is None:
        oracle.readout_fwd_bwd(h, g, W, x["targets"], True)
    else:
        from solo_inputs import make_extras

        e = make_extras(x, seed, **extras)
        Wbar = e.get("Wbar")
        if e.get("rot") is not None:
            # the oracle reads ROT heads as one readout each, Wbar R_k (formed before the clock starts)
            base = W if Wbar is None else Wbar.astype(np.float64)
            Wbar = np.stack([base @ r.astype(np.float64) for r in e["rot"]])
        kw = dict(Wbar=Wbar, tau=e.get("tau"), bias=e.get("bias"))
        t0 = time.perf_counter()
        if flags is None:
            oracle.exit_eval(h, e["gain"], W, x["targets"], **kw)
        else:
            oracle.general_fwd_bwd(h, e["gain"], W, x["targets"], final_module_dW=flags.get("final_module_dW", True),
                                   heads_train_readout=flags.get("heads_train_readout", False), **kw)
    dt = time.perf_counter() - t0
    cfg = x["cfg"]
    from paper_2609_35440_amd import costmodel

    fl = dict(final_module_dW=True) if flags is None else flags
    alg = costmodel.general_flops(cfg.K, sample_T, cfg.V, cfg.d, final_module_dW=fl.get("final_module_dW", True),
                                  heads_train_readout=fl.get("heads_train_readout", False),
                                  exit_eval=extras is not None and flags is None)
    return {
        "value": sample_T / dt,
        "unit": "tokens/s",
        "cores": int(threads),
        "cpu_model": _cpu_model(),
        "gflops_algorithmic": alg / dt / 1e9,
        "kind": "oracle",
        "sample": f"{cfg_name} shape with T={sample_T} tokens per module (K={cfg.K}, d={cfg.d}, V={cfg.V}, "
                  f"{'final-module dW included' if variant == 'headline' else 'variant ' + variant}), "
                  f"fp64 NumPy oracle, {dt:.2f} s",
        "seconds": dt,
    }


def kernel_sources_hash(read=None, files=None) -> str:
    """Hash of every library source (paper_2609_35440_amd/csrc), comments and
    whitespace removed (stamps counter-derived traffic and profiles: a comment
    edit does not void a measurement)."""
    import hashlib
    import re

    csrc = os.path.join(ROOT, "paper_2609_35440_amd", "csrc")
    if read is None:
        def read(f):
            with open(os.path.join(csrc, f), "rb") as fh:
                return fh.read().decode()
    if files is None:
        files = sorted(f for f in os.listdir(csrc) if f.endswith((".hip", ".h")))

    h = hashlib.sha256()
    for f in files:
        text = re.sub(r"/\*.*?\*/", " ", read(f), flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def copy_probe(mib: int) -> int:
    """A plain device-to-device copy of known size: reads and writes mib MiB per launch."""
    import torch

    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_each_way": n * 4, "launches": 5}), flush=True)
    return 0


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="1b", help="workload shape (solo_inputs.CONFIGS key)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--variant", default="headline", choices=sorted(VARIANTS),
                    help="headline: the shared-readout loss as the paper's headline runs it; the others time the "
                         "general call (temperatures, biases, per-module gains, readout sources) or the "
                         "forward-only exit evaluation on the same shapes")
    ap.add_argument("--cpu-sample-tokens", type=int, default=8192,
                    help="tokens per module of the oracle's bounded sample (0 to skip)")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "traffic_local_loss_1b.json"),
                    help="fabric traffic (L2 to memory system) of the dominant kernel measured with rocprofv3 "
                         "counters (JSON), if present")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="instead of the benchmark, run a plain device copy of MIB MiB a few times "
                         "(calibrates the FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args(argv)
    if args.copy_probe:
        return copy_probe(args.copy_probe)

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (no collectives, no sharding); "
              "run with --gpus 1", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2609_35440_amd import binding, costmodel
    from solo_inputs import make_inputs

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    binding.load_library()
    dev = torch.device("cuda:0")

    x = make_inputs(args.config, seed=args.seed)
    cfg = x["cfg"]
    K, T, d, V = cfg.K, cfg.T, cfg.d, cfg.V
    if cfg.dtype == "bf16":
        def up(bits):
            return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(dev)

        h, gain, W = up(x["h_bits"]), up(x["gain_bits"]), up(x["W_bits"])
        elem = 2
    else:
        h, gain, W = (torch.from_numpy(x[k]).to(dev) for k in ("h", "gain", "W"))
        elem = 4
    targets = torch.from_numpy(x["targets"]).to(dev)
    extras, flags, vdesc = VARIANTS[args.variant]
    Wbar = tau = bias = rot = None
    if extras is not None:
        from solo_inputs import make_extras

        e = make_extras(x, args.seed, **extras)
        bf = cfg.dtype == "bf16"

        def up_any(name):
            if e.get(name) is None:
                return None
            if bf:
                return torch.from_numpy(np.ascontiguousarray(e[name + "_bits"]).view(np.int16)).view(
                    torch.bfloat16).to(dev)
            return torch.from_numpy(np.ascontiguousarray(e[name])).to(dev)

        gain = up_any("gain")
        Wbar = up_any("Wbar")
        rot = up_any("rot")
        tau = torch.from_numpy(e["tau"]).to(dev) if e.get("tau") is not None else None
        bias = torch.from_numpy(e["bias"]).to(dev) if e.get("bias") is not None else None
        del e
    del x
    dt = binding.SOLO_BF16 if cfg.dtype == "bf16" else binding.SOLO_F32
    family = binding.kernel_family(K, T, d, V, dt)
    out = binding.ReadoutResult(
        losses=torch.empty(K, dtype=torch.float32, device=dev),
        dh=torch.empty_like(h),
        dW=torch.empty((V, d), dtype=torch.float32, device=dev),
        dgain=torch.empty(d, dtype=torch.float32, device=dev),
        row_loss=None,
    )
    stream = torch.cuda.current_stream(dev)
    hip = _hip()
    n_ev = binding.NUM_STAGES + 1
    events = [EventSet(hip, n_ev) for _ in range(args.steps)]
    gout = [None]
    if args.variant == "headline":
        ws = torch.empty(binding.workspace_size(K, T, d, V, dt, True), dtype=torch.uint8, device=dev)
    else:
        del out
        # first call sizes and allocates the workspace and outputs; the timed calls reuse them
        if flags is None:
            r = binding.exit_eval(h, gain, W, targets, Wbar=Wbar, tau=tau, bias=bias, rot=rot, stream=stream)
        else:
            r = binding.readout_general(h, gain, W, targets, Wbar=Wbar, tau=tau, bias=bias, rot=rot, stream=stream,
                                        **flags)
        gout[0] = r
        torch.cuda.synchronize()
        a = binding._fill_inputs(h, gain, W, targets, Wbar, tau, bias, 1e-6, rot)[0]
        if flags is None:
            nbytes = binding.exit_eval_workspace_size(a)
        else:
            a.final_module_dW = int(flags.get("final_module_dW", True))
            a.heads_train_readout = int(flags.get("heads_train_readout", False))
            a.dtau = 1 if flags.get("want_dtau") else None
            a.dbias = 1 if flags.get("want_dbias") else None
            nbytes = binding.general_workspace_size(a)
        ws = torch.empty(nbytes, dtype=torch.uint8, device=dev)

    def step(ev=None):
        stage = None
        if ev is not None:
            assert hip.hipEventRecord(ctypes.c_void_p(ev.ev[0]), ctypes.c_void_p(stream.cuda_stream)) == 0
            stage = ev.ev[1:]
        if args.variant == "headline":
            binding.readout_fwd_bwd(h, gain, W, targets, True, 1e-6, workspace=ws, out=out, stream=stream,
                                    stage_events=stage)
        elif flags is None:
            binding.exit_eval(h, gain, W, targets, Wbar=Wbar, tau=tau, bias=bias, rot=rot, workspace=ws,
                              stream=stream, stage_events=stage, out=gout[0])
        else:
            binding.readout_general(h, gain, W, targets, Wbar=Wbar, tau=tau, bias=bias, rot=rot, workspace=ws,
                                    stream=stream, stage_events=stage, out=gout[0], **flags)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # device memory: torch's allocator peak over one call (the library itself
    # allocates nothing), and the driver's free-memory reading around it
    free0 = ctypes.c_size_t(0)
    total = ctypes.c_size_t(0)
    assert hip.hipMemGetInfo(ctypes.byref(free0), ctypes.byref(total)) == 0
    base_alloc = torch.cuda.memory_allocated(dev)
    torch.cuda.reset_peak_memory_stats(dev)
    step()
    torch.cuda.synchronize()
    peak_delta = torch.cuda.max_memory_allocated(dev) - base_alloc
    free1 = ctypes.c_size_t(0)
    assert hip.hipMemGetInfo(ctypes.byref(free1), ctypes.byref(total)) == 0
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(events[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    # per-step and per-stage times from the events (stage i ends at event i + 1)
    step_ms = [e.elapsed(0, n_ev - 1) for e in events]
    stage_ms = {name: float(np.mean([e.elapsed(i, i + 1) for e in events]))
                for i, name in enumerate(binding.STAGE_NAMES)}
    for e in events:
        e.destroy()
    ms_per_step = wall * 1e3 / args.steps
    losses = (out if args.variant == "headline" else gout[0]).losses.cpu().tolist()
    if not all(np.isfinite(losses)):
        print(f"non-finite losses {losses}", file=sys.stderr)
        return 1

    is_eval = flags is None
    fl = dict(final_module_dW=True) if is_eval else flags
    alg_flops = costmodel.general_flops(K, T, V, d, final_module_dW=fl.get("final_module_dW", True),
                                        heads_train_readout=fl.get("heads_train_readout", False), exit_eval=is_eval)
    exe_flops = costmodel.executed_flops(K, T, V, d, final_module_dW=fl.get("final_module_dW", True),
                                         heads_train_readout=fl.get("heads_train_readout", False),
                                         bias_grad=fl.get("want_dbias", False), exit_eval=is_eval,
                                         rot=rot is not None)
    tokens_per_s = T / (ms_per_step / 1e3)
    # dominant kernel: the local-loss pass, 2r per token of every module (logits + input
    # gradient), or the exit evaluation's forward pass (1r)
    ll_ms = stage_ms["local_loss"]
    ll_flops = (1 if is_eval else 2) * 2 * K * T * V * d
    achieved = ll_flops / (ll_ms / 1e3) / 1e12
    traffic = None
    mfma_busy = None  # counter-measured busy fraction of the matrix units in that kernel
    if os.path.exists(args.traffic):
        try:
            with open(args.traffic) as f:
                tr = json.load(f)
            # counters count only for the kernel source they were taken on
            if (tr.get("config") == args.config and tr.get("family") == family and args.variant == "headline"
                    and tr.get("kernel_sources_sha256_16") == kernel_sources_hash()):
                traffic = tr.get("bytes_per_launch")
                mfma_busy = tr.get("mfma_busy")
        except Exception:
            traffic = mfma_busy = None

    result = {
        "metric": METRIC,
        "value": tokens_per_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded N(0,1) hidden states, N(0,0.02^2) readout, 1+N(0,0.1^2) gain, Zipf(1.1) targets)",
        "config": {"workload": f"{cfg.name}: K={K} modules, T={T} tokens/module, d={d}, V={V}, "
                               + ("final-module dW" if args.variant == "headline" else f"{args.variant}: {vdesc}"),
                   "K": K, "T": T, "d": d, "V": V, "kernel_family": family, "variant": args.variant},
        "executed_flops": exe_flops,
        "tflops_algorithmic": alg_flops / (ms_per_step / 1e3) / 1e12,
        "frac_bf16_peak_algorithmic": alg_flops / (ms_per_step / 1e3) / 1e12 / PEAK_BF16_TFLOPS,
        "tflops_executed": exe_flops / (ms_per_step / 1e3) / 1e12,
        "module_tokens_per_s": K * tokens_per_s,
        "stage_ms": stage_ms,
        "event_ms_per_step": float(np.median(step_ms)),
        "event_ms_per_step_min": float(np.min(step_ms)),
        "workspace_bytes": int(ws.numel()),
        "peak_alloc_delta_bytes": int(peak_delta),
        "driver_free_delta_bytes": int(free0.value) - int(free1.value),
        "one_module_tv_bf16_bytes": int(T) * int(V) * 2,
        "roofline": {
            "bound": "mfma",
            "kernel": ("exit evaluation (logits + online log-sum-exp + top-1), all K modules" if is_eval else
                       "local-loss pass (logits + online log-sum-exp + dh), all K modules"),
            "achieved": achieved,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS,
            # counter-measured bytes per launch between the L2 and the memory system
            # (Infinity Cache hits included, so an upper bound on DRAM bytes)
            "traffic": traffic,
            "traffic_kind": "fabric",
            "fabric_gb_per_s": (traffic / (ll_ms / 1e3) / 1e9) if traffic else None,
            "mfma_busy_counter": mfma_busy,
            "algorithmic_flops_per_launch": ll_flops,
            "launch_ms": ll_ms,
        },
        "losses": losses,
    }
    if args.cpu_sample_tokens > 0:
        result["cpu_baseline"] = cpu_baseline(args.config, args.cpu_sample_tokens, args.seed, args.variant)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
