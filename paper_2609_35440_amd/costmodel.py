"""FLOP and byte accounting of the SOLO readout path, and the paper's cost model.

Units follow the paper's FLOP table (appendix on training FLOPs, Table
"Training FLOPs per token"): a forward pass is one unit, a block costs
``3b`` with ``b = 12 d^2 + 2 T d`` multiply-accumulates per token, the
terminal readout costs ``3r`` with ``r = V d``, an auxiliary readout costs
``2r`` because no gradient with respect to its detached weights is computed,
and one multiply-accumulate is two FLOPs.  Proposition 2 (work ratio rho) and
Eq. "win" (crossover M*) of the pipeline appendix are written out below.
"""
from __future__ import annotations

__all__ = [
    "readout_flops",
    "general_flops",
    "executed_flops",
    "readout_bytes",
    "block_macs",
    "flops_per_token",
    "rho",
    "mstar",
]


def readout_flops(K: int, T: int, V: int, d: int, final_module_dW: bool = True) -> int:
    """Algorithmic FLOPs of one call of the shared-readout local loss.

    K-1 read-only heads cost 2r MACs per token (logits + input gradient) and
    the final module 3r (plus the weight gradient); r = V d.  Without the
    final module's weight gradient every module costs 2r.
    """
    units = 2 * K + (1 if final_module_dW else 0)
    return 2 * units * T * V * d


def general_flops(K: int, T: int, V: int, d: int, *, final_module_dW: bool = True,
                  heads_train_readout: bool = False, exit_eval: bool = False) -> int:
    """Algorithmic FLOPs of the general call (the same units as readout_flops).

    Every module costs 2r (logits + input gradient); a module whose readout is
    trained (the terminal with final_module_dW, every head under PRIV) one r
    more for the weight gradient.  Temperatures, biases and gains add only
    O(T V) or O(T d) work.  Exit evaluation is the forward product alone: 1r
    per module.
    """
    if exit_eval:
        return 2 * K * T * V * d
    trained = (1 if final_module_dW else 0) + ((K - 1) if heads_train_readout else 0)
    return 2 * (2 * K + trained) * T * V * d


def executed_flops(K: int, T: int, V: int, d: int, *, final_module_dW: bool = True,
                   heads_train_readout: bool = False, bias_grad: bool = False, exit_eval: bool = False,
                   rot: bool = False) -> int:
    """Matrix-product FLOPs the fused kernels execute for the same call.

    Local-loss pass: 2r per module (logits and the input-gradient product).
    Readout-gradient pass: 2r per module in it (the logits again, with the
    stored log-sum-exp, and the weight-gradient product).  Bias-gradient pass
    (modules whose bias but not readout gets a gradient): 1r per module, the
    logits again.  Exit evaluation: 1r per module.  ROT (head k reads Wbar R_k)
    adds the rotation of each head's rows, 2 T d^2, and in the backward pass
    the rotation of its gradient back, 2 T d^2 more.
    """
    rotf = (K - 1) * 2 * T * d * d if rot and K > 1 else 0
    if exit_eval:
        return 2 * K * T * V * d + rotf
    rg = (1 if final_module_dW else 0) + ((K - 1) if heads_train_readout else 0)
    bg = (K - rg) if bias_grad else 0
    return 2 * (2 * K + 2 * rg + bg) * T * V * d + 2 * rotf


def readout_bytes(K: int, T: int, V: int, d: int, elem_bytes: int = 2, final_module_dW: bool = True) -> int:
    """Algorithmic HBM bytes of one call: every input read once, every output written once.

    h [K,T,d] and W [V,d] and gain [d] in the storage dtype, targets int32,
    dh [K,T,d] in the storage dtype, dW [V,d] and dgain [d] fp32, losses fp32.
    """
    b = 2 * K * T * d * elem_bytes + V * d * elem_bytes + d * elem_bytes + K * T * 4 + K * 4
    if final_module_dW:
        b += V * d * 4 + d * 4
    return b


def block_macs(d: int, T: int) -> int:
    """Multiply-accumulates per token of one Transformer block: b = 12 d^2 + 2 T d."""
    return 12 * d * d + 2 * T * d


def flops_per_token(L: int, d: int, K: int, H: int, T: int, V: int) -> dict:
    """Per-token training FLOPs of BP and SOLO (the paper's FLOP table).

    Returns GFLOP/token for: BP total and layers, SOLO total, auxiliary
    blocks, readouts, and rho = SOLO / BP.
    """
    b = block_macs(d, T)
    r = V * d
    layers = 3 * L * b
    bp = layers + 3 * r
    aux = 3 * (K - 1) * H * b
    readouts = (2 * K + 1) * r
    solo = layers + aux + readouts
    g = 2e-9
    return {
        "bp_total": bp * g,
        "bp_layers": layers * g,
        "solo_total": solo * g,
        "aux_blocks": aux * g,
        "readouts": readouts * g,
        "rho": solo / bp,
    }


def _gamma(L: int, d: int, T: int, V: int) -> float:
    # cost of one readout relative to the L blocks: gamma = r / (L b) = V / (L (12 d + 2 T))
    return V / (L * (12 * d + 2 * T))


def rho(L: int, d: int, K: int, H: int, T: int, V: int) -> float:
    """Work ratio of Proposition 2: (1 + (K-1)H/L + (2K+1)gamma/3) / (1 + gamma)."""
    g = _gamma(L, d, T, V)
    return (1.0 + (K - 1) * H / L + (2 * K + 1) * g / 3.0) / (1.0 + g)


def mstar(L: int, d: int, H: int, T: int, V: int) -> float:
    """Crossover micro-batch count of Eq. "win": (1 + gamma) / (H/L + 2 gamma / 3)."""
    g = _gamma(L, d, T, V)
    return (1.0 + g) / (H / L + 2.0 * g / 3.0)
