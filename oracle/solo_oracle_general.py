"""fp64 CPU oracle of the full readout lines of one SOLO step (test infrastructure only).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call this module.  The GPU
product path never touches it and shares no code with it.

This extends the headline oracle (``solo_oracle.py``: temperature 1, no bias,
one gain, the heads reading the live readout) to everything the paper's
Algorithm 1 and Eq. 2 put into a head's loss, and to the readout sources of
the variant table (Section 3.3, the table of readout sources; Appendix D, the
table of readout content and basis):

  head k < K-1:  z = tau_k * Wh_k phi_k(h_k) + b_k      (Eq. 2 plus the bias of Alg. 1)
  terminal K-1:  z = tau_{K-1} * W phi_{K-1}(h_{K-1}) + b   (Alg. 1 has tau = 1 there;
                                                           pass tau[K-1] = 1 for that)

with ``phi_k(h) = g_k * h / sqrt(mean h^2 + eps)`` (the head's final RMSNorm with
an element-wise gain, Appendix C) and the heads' readout ``Wh_k``:

  * ``Wbar is None``      -> Wh_k = W (SOLO, the copy equals W when the step starts)
  * ``Wbar`` [V, d]       -> one read-only matrix shared by the heads (SOLO with a
                             refresh period S > 1: the copy from an earlier step;
                             RSHARE: one frozen random matrix)
  * ``Wbar`` [K-1, V, d]  -> one matrix per head (RAND: frozen; PRIV: learned,
                             ``heads_train_readout``; ROT: the caller's W R_k)

Gradients of the mean cross-entropy of each module (delta = (p - onehot) / T):

  dhhat = tau_k delta Wh_k,  dn = g_k * dhhat,  dh = r (dn - mean(dn n) n)
  dtau_k = sum_t sum_v delta_tv u_tv  with u = Wh_k hhat (the logits before tau, b)
  dbias_k = sum_t delta_t                        (every module: heads train b_k, Alg. 1)
  dW = tau_{K-1} delta^T hhat                    (terminal, if final_module_dW)
  dWbar_k = tau_k delta^T hhat                   (heads, PRIV only)
  dgain: one shared gain -> the terminal's sum_t dhhat * n (the heads' gain is the
         read-only copy); per-module gains [K, d] -> every module's own sum.

Forward-only exit evaluation (Section 4, early exit through the shared
readout): per module the loss, the perplexity exp(loss), and the top-1
prediction argmax_v z_tv with ties going to the lowest index.

Plain NumPy float64; rows of T are blocked, which the definition allows since
rows are independent.  Pins: tests/oracle_general_pins.py.
"""
from __future__ import annotations

import numpy as np

__all__ = ["readout_matrix", "general_fwd_bwd", "general_bruteforce", "exit_eval"]

DEFAULT_EPS = 1e-6


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def readout_matrix(k, K, W, Wbar):
    """The readout module k predicts through (Alg. 1; the readout-source table)."""
    if k == K - 1 or Wbar is None:
        return W
    return Wbar if Wbar.ndim == 2 else Wbar[k]


def _check(h, gain, W, targets, Wbar, tau, bias, heads_train_readout):
    K, T, d = h.shape
    V = W.shape[0]
    if W.shape != (V, d):
        raise ValueError("W shape")
    if gain.shape not in ((d,), (K, d)):
        raise ValueError("gain shape")
    if Wbar is not None and Wbar.shape not in ((V, d), (K - 1, V, d)):
        raise ValueError("Wbar shape")
    if heads_train_readout and (Wbar is None or Wbar.ndim != 3):
        raise ValueError("heads_train_readout needs one readout per head")
    if tau is not None and tau.shape != (K,):
        raise ValueError("tau shape")
    if bias is not None and bias.shape != (K, V):
        raise ValueError("bias shape")
    if np.any(targets < 0) or np.any(targets >= V):
        raise ValueError("targets out of range")
    for x in (h, gain, W, Wbar, tau, bias):
        if x is not None and not np.all(np.isfinite(x)):
            raise ValueError("non-finite input")


def general_fwd_bwd(h, gain, W, targets, *, Wbar=None, tau=None, bias=None, final_module_dW=True,
                    heads_train_readout=False, eps=DEFAULT_EPS, row_chunk=1024):
    """All K modules with temperatures, biases, per-module gains and readout sources.

    Returns a dict: ``losses`` [K], ``row_loss`` [K, T], ``dh`` [K, T, d],
    ``dW`` [V, d] or None, ``dWbar`` [K-1, V, d] or None, ``dgain`` ([d], [K, d]
    or None), ``dtau`` [K], ``dbias`` [K, V].
    """
    h, gain, W = _f64(h), _f64(gain), _f64(W)
    Wbar = None if Wbar is None else _f64(Wbar)
    tau = None if tau is None else _f64(tau)
    bias = None if bias is None else _f64(bias)
    targets = np.asarray(targets, dtype=np.int64)
    _check(h, gain, W, targets, Wbar, tau, bias, heads_train_readout)
    K, T, d = h.shape
    V = W.shape[0]
    per_module_gain = gain.ndim == 2

    losses = np.empty(K)
    row_loss = np.empty((K, T))
    dh = np.empty((K, T, d))
    dtau = np.zeros(K)
    dbias = np.zeros((K, V))
    dW = np.zeros((V, d)) if final_module_dW else None
    dWbar = np.zeros((K - 1, V, d)) if heads_train_readout else None
    if per_module_gain:
        dgain = np.zeros((K, d))
    else:
        dgain = np.zeros(d) if final_module_dW else None

    for k in range(K):
        Wk = readout_matrix(k, K, W, Wbar)
        gk = gain[k] if per_module_gain else gain
        tk = 1.0 if tau is None else float(tau[k])
        bk = np.zeros(V) if bias is None else bias[k]
        for t0 in range(0, T, row_chunk):
            t1 = min(T, t0 + row_chunk)
            rows = np.arange(t1 - t0)
            yc = targets[k, t0:t1]
            x = h[k, t0:t1]
            r = 1.0 / np.sqrt(np.mean(x * x, axis=1) + float(eps))     # RMSNorm
            n = x * r[:, None]
            hhat = gk * n                                              # element-wise gain
            u = hhat @ Wk.T                                            # readout product
            z = tk * u + bk                                            # Eq. 2 with the bias of Alg. 1
            m = z.max(axis=1)
            lse = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
            row_loss[k, t0:t1] = lse - z[rows, yc]
            delta = np.exp(z - lse[:, None])
            delta[rows, yc] -= 1.0
            delta /= float(T)                                          # mean over the module's tokens
            dhhat = tk * (delta @ Wk)                                  # Eq. 3 through the readout
            dn = dhhat * gk
            c = np.mean(dn * n, axis=1)
            dh[k, t0:t1] = r[:, None] * (dn - c[:, None] * n)
            dtau[k] += float(np.sum(delta * u))
            dbias[k] += delta.sum(axis=0)
            if k == K - 1 and final_module_dW:
                dW += tk * (delta.T @ hhat)
            if k < K - 1 and heads_train_readout:
                dWbar[k] += tk * (delta.T @ hhat)
            if per_module_gain:
                dgain[k] += np.sum(dhhat * n, axis=0)
            elif k == K - 1 and final_module_dW:
                dgain += np.sum(dhhat * n, axis=0)
        losses[k] = row_loss[k].sum() / T
    return {"losses": losses, "row_loss": row_loss, "dh": dh, "dW": dW, "dWbar": dWbar, "dgain": dgain,
            "dtau": dtau, "dbias": dbias}


def general_bruteforce(h, gain, W, targets, *, Wbar=None, tau=None, bias=None, final_module_dW=True,
                       heads_train_readout=False, eps=DEFAULT_EPS):
    """Per-element loops for tiny shapes; shares no expression with general_fwd_bwd."""
    h, gain, W = _f64(h), _f64(gain), _f64(W)
    K, T, d = h.shape
    V = W.shape[0]
    pm = gain.ndim == 2
    out = {"losses": np.zeros(K), "row_loss": np.zeros((K, T)), "dh": np.zeros((K, T, d)),
           "dtau": np.zeros(K), "dbias": np.zeros((K, V)),
           "dW": np.zeros((V, d)) if final_module_dW else None,
           "dWbar": np.zeros((K - 1, V, d)) if heads_train_readout else None,
           "dgain": np.zeros((K, d)) if pm else (np.zeros(d) if final_module_dW else None)}
    for k in range(K):
        if k == K - 1 or Wbar is None:
            Wk = W
        else:
            Wk = _f64(Wbar) if np.ndim(Wbar) == 2 else _f64(Wbar)[k]
        g = gain[k] if pm else gain
        tk = 1.0 if tau is None else float(tau[k])
        for t in range(T):
            ms = sum(h[k, t, j] ** 2 for j in range(d)) / d
            r = (ms + eps) ** -0.5
            n = [h[k, t, j] * r for j in range(d)]
            hh = [g[j] * n[j] for j in range(d)]
            u = [sum(Wk[v, j] * hh[j] for j in range(d)) for v in range(V)]
            z = [tk * u[v] + (0.0 if bias is None else float(bias[k][v])) for v in range(V)]
            zmax = max(z)
            lse = zmax + np.log(sum(np.exp(zv - zmax) for zv in z))
            y = int(targets[k][t])
            out["row_loss"][k, t] = lse - z[y]
            dl = [(np.exp(z[v] - lse) - (1.0 if v == y else 0.0)) / T for v in range(V)]
            dhh = [tk * sum(dl[v] * Wk[v, j] for v in range(V)) for j in range(d)]
            dn = [dhh[j] * g[j] for j in range(d)]
            c = sum(dn[j] * n[j] for j in range(d)) / d
            for j in range(d):
                out["dh"][k, t, j] = r * (dn[j] - c * n[j])
            for v in range(V):
                out["dtau"][k] += dl[v] * u[v]
                out["dbias"][k, v] += dl[v]
            grad_w = None
            if k == K - 1 and final_module_dW:
                grad_w = out["dW"]
            elif k < K - 1 and heads_train_readout:
                grad_w = out["dWbar"][k]
            if grad_w is not None:
                for v in range(V):
                    for j in range(d):
                        grad_w[v, j] += tk * dl[v] * hh[j]
            if pm:
                for j in range(d):
                    out["dgain"][k, j] += dhh[j] * n[j]
            elif k == K - 1 and final_module_dW:
                for j in range(d):
                    out["dgain"][j] += dhh[j] * n[j]
        out["losses"][k] = out["row_loss"][k].sum() / T
    return out


def exit_eval(h, gain, W, targets, *, Wbar=None, tau=None, bias=None, eps=DEFAULT_EPS, row_chunk=1024):
    """Forward-only evaluation of every exit through its readout.

    Returns ``losses`` [K], ``row_loss`` [K, T], ``ppl`` [K] = exp(losses),
    ``top1`` [K, T] (argmax of z, lowest index on ties), ``zmax`` [K, T] (the
    largest logit, for checking another implementation's argmax against the
    fp64 logits), ``logits_of`` (a function (k, t, v) -> z_ktv in fp64) and
    ``accuracy`` [K] (fraction of tokens whose top-1 equals the target).
    """
    h, gain, W = _f64(h), _f64(gain), _f64(W)
    Wbar = None if Wbar is None else _f64(Wbar)
    tau = None if tau is None else _f64(tau)
    bias = None if bias is None else _f64(bias)
    targets = np.asarray(targets, dtype=np.int64)
    _check(h, gain, W, targets, Wbar, tau, bias, False)
    K, T, d = h.shape
    V = W.shape[0]
    pm = gain.ndim == 2
    row_loss = np.empty((K, T))
    top1 = np.empty((K, T), dtype=np.int64)
    zmax = np.empty((K, T))

    def logits(k, rows):
        Wk = readout_matrix(k, K, W, Wbar)
        gk = gain[k] if pm else gain
        x = h[k, rows]
        r = 1.0 / np.sqrt(np.mean(x * x, axis=1) + float(eps))
        z = (gk * x * r[:, None]) @ Wk.T
        z = z * (1.0 if tau is None else float(tau[k]))
        return z + (0.0 if bias is None else bias[k])

    for k in range(K):
        for t0 in range(0, T, row_chunk):
            t1 = min(T, t0 + row_chunk)
            rows = np.arange(t0, t1)
            z = logits(k, rows)
            m = z.max(axis=1)
            lse = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
            row_loss[k, t0:t1] = lse - z[np.arange(t1 - t0), targets[k, t0:t1]]
            top1[k, t0:t1] = np.argmax(z, axis=1)          # first maximum: lowest index
            zmax[k, t0:t1] = m
    losses = row_loss.mean(axis=1)
    return {"losses": losses, "row_loss": row_loss, "ppl": np.exp(losses), "top1": top1, "zmax": zmax,
            "accuracy": (top1 == targets).mean(axis=1),
            "logits_of": lambda k, t, v: float(logits(k, np.array([t]))[0, v])}
