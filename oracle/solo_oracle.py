"""fp64 CPU oracle of the SOLO shared-readout local loss.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call this module.  The GPU
product path never touches it and shares no code with it.

What is computed (the paper: Section 3.2 "SOLO: local learning with a shared
readout", Eq. 2 and Eq. 3; Appendix A, Algorithm 1; Appendix C, head =
blocks + final RMSNorm with an element-wise gain; Appendix B, the
cross-entropy residual ``delta = p - onehot(y)``):

For every module k and token t, with the same read-only readout ``W`` (V x d)
and RMSNorm gain ``g`` (d) shared by all modules (temperature tau_k = 1, no
bias):

  1. ``ms = mean_j h_tj^2``, ``r = 1/sqrt(ms + eps)``, ``n = r h``,
     ``hhat = g * n``                                (RMSNorm, element-wise gain)
  2. ``z_v = <W_v, hhat>`` for every v                (Eq. 2, tau = 1)
  3. ``lse = log sum_v exp(z_v)``, ``l_t = lse - z_{y_t}``,
     ``p_v = exp(z_v - lse)``                         (softmax cross-entropy)
  4. ``delta_v = (p_v - [v = y_t]) / T``              (residual of the mean CE)
     ``dhhat = sum_v delta_v W_v``                    (Eq. 3: readout transposed)
     ``dn = g * dhhat``, ``c = mean_j dn_j n_j``,
     ``dh = r (dn - c n)``                            (RMSNorm backward)
  5. final module only: ``dW += delta^T hhat``, ``dgain += sum_t dhhat * n``.
     The read-only copies used by the other modules receive no gradient
     (Section 3.2; the FLOP table counts no weight gradient for them).
  6. ``loss_k = mean_t l_t``.

Readings where the paper is silent: eps is an explicit argument; the
cross-entropy is the mean over the module's T tokens; tau_k = 1 and no bias;
one gain shared with the readout (gradient only from the final module).

Everything is plain NumPy float64.  The only blocking is over rows of T, which
the definition allows since rows are independent; the T x V logits of a chunk
are materialised and discarded.  Parity pins: see ``tests/test_oracle.py``
(finite differences, torch fp64 autograd, closed forms at W = 0, softplus at
V = 2, V = 1, invariants, brute force).
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "rmsnorm_forward",
    "module_fwd_bwd",
    "readout_fwd_bwd",
    "readout_bruteforce",
    "softmax_rows",
]

DEFAULT_EPS = 1e-6


def _f64(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


def rmsnorm_forward(h, gain, eps):
    """RMSNorm with element-wise gain over the last axis.

    Returns ``(hhat, n, r)`` with ``n = h / sqrt(mean(h^2) + eps)`` and
    ``hhat = gain * n``.
    """
    h = _f64(h)
    ms = np.mean(h * h, axis=-1)
    r = 1.0 / np.sqrt(ms + float(eps))
    n = h * r[..., None]
    return _f64(gain) * n, n, r


def softmax_rows(z):
    """Row softmax of a logit matrix (max-shifted)."""
    z = _f64(z)
    m = z.max(axis=-1, keepdims=True)
    e = np.exp(z - m)
    return e / e.sum(axis=-1, keepdims=True)


def module_fwd_bwd(h, y, W, gain, eps=DEFAULT_EPS, want_readout_grads=False, T_total=None,
                   row_chunk=1024):
    """Local loss and gradients of one module through the shared readout.

    ``h`` [R, d] are R rows of the module (all of them unless a row subset is
    passed together with ``T_total``), ``y`` [R] their targets.  ``T_total`` is
    the module's token count that the mean CE divides by (defaults to R).

    Returns ``(row_loss [R], dh [R, d], dW [V, d] or None, dgain [d] or None)``;
    the module loss is ``row_loss.sum() / T_total``.
    """
    h = _f64(h)
    W = _f64(W)
    g = _f64(gain)
    y = np.asarray(y, dtype=np.int64)
    R, d = h.shape
    V = W.shape[0]
    if T_total is None:
        T_total = R
    if np.any(y < 0) or np.any(y >= V):
        raise ValueError("targets out of range")
    if not (np.all(np.isfinite(h)) and np.all(np.isfinite(W)) and np.all(np.isfinite(g))):
        raise ValueError("non-finite input")

    row_loss = np.empty(R)
    dh = np.empty((R, d))
    dW = np.zeros((V, d)) if want_readout_grads else None
    dgain = np.zeros(d) if want_readout_grads else None

    for t0 in range(0, R, row_chunk):
        t1 = min(R, t0 + row_chunk)
        rows = np.arange(t1 - t0)
        yc = y[t0:t1]
        hhat, n, r = rmsnorm_forward(h[t0:t1], g, eps)
        z = hhat @ W.T                                   # Eq. 2 (tau = 1)
        m = z.max(axis=1)
        lse = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
        row_loss[t0:t1] = lse - z[rows, yc]
        delta = np.exp(z - lse[:, None])                 # p
        delta[rows, yc] -= 1.0                           # p - onehot(y)
        delta /= float(T_total)                          # mean over the module's tokens
        dhhat = delta @ W                                # Eq. 3: W^T delta, per row
        dn = dhhat * g
        c = np.mean(dn * n, axis=1)
        dh[t0:t1] = r[:, None] * (dn - c[:, None] * n)
        if want_readout_grads:
            dW += delta.T @ hhat
            dgain += np.sum(dhhat * n, axis=0)
    return row_loss, dh, dW, dgain


def readout_fwd_bwd(h, gain, W, targets, final_module_dW=True, eps=DEFAULT_EPS, row_chunk=1024):
    """All K modules (Algorithm 1, the readout lines of one SOLO step).

    Modules 0..K-2 predict through the read-only copy (no readout gradient);
    module K-1 is the final module and, if ``final_module_dW``, also returns
    the gradients of the trained readout (``dW``) and gain (``dgain``).

    Returns a dict: ``losses`` [K], ``row_loss`` [K, T], ``dh`` [K, T, d],
    ``dW`` [V, d] or None, ``dgain`` [d] or None.
    """
    h = _f64(h)
    K, T, d = h.shape
    targets = np.asarray(targets)
    losses = np.empty(K)
    row_loss = np.empty((K, T))
    dh = np.empty((K, T, d))
    dW = dgain = None
    for k in range(K):
        want = bool(final_module_dW) and k == K - 1
        rl, dhk, dWk, dgk = module_fwd_bwd(h[k], targets[k], W, gain, eps, want, T, row_chunk)
        row_loss[k] = rl
        losses[k] = rl.sum() / T
        dh[k] = dhk
        if want:
            dW, dgain = dWk, dgk
    return {"losses": losses, "row_loss": row_loss, "dh": dh, "dW": dW, "dgain": dgain}


def readout_bruteforce(h, gain, W, targets, final_module_dW=True, eps=DEFAULT_EPS):
    """Unblocked version for tiny shapes: every intermediate as a full array.

    Written per element with explicit Python loops for the normalisation and
    the residual, so that it does not share the vectorised expressions of
    :func:`readout_fwd_bwd`.  Only for tiny K, T, d, V.
    """
    h = _f64(h)
    W = _f64(W)
    g = _f64(gain)
    K, T, d = h.shape
    V = W.shape[0]
    losses = np.zeros(K)
    row_loss = np.zeros((K, T))
    dh = np.zeros((K, T, d))
    dW = np.zeros((V, d)) if final_module_dW else None
    dgain = np.zeros(d) if final_module_dW else None
    for k in range(K):
        for t in range(T):
            x = h[k, t]
            ms = 0.0
            for j in range(d):
                ms += x[j] * x[j]
            ms /= d
            r = 1.0 / np.sqrt(ms + eps)
            n = [x[j] * r for j in range(d)]
            hh = [g[j] * n[j] for j in range(d)]
            z = [sum(W[v, j] * hh[j] for j in range(d)) for v in range(V)]
            zmax = max(z)
            s = sum(np.exp(zv - zmax) for zv in z)
            lse = zmax + np.log(s)
            y = int(targets[k, t])
            row_loss[k, t] = lse - z[y]
            delta = [(np.exp(z[v] - lse) - (1.0 if v == y else 0.0)) / T for v in range(V)]
            dhh = [sum(delta[v] * W[v, j] for v in range(V)) for j in range(d)]
            dn = [dhh[j] * g[j] for j in range(d)]
            c = sum(dn[j] * n[j] for j in range(d)) / d
            for j in range(d):
                dh[k, t, j] = r * (dn[j] - c * n[j])
            if final_module_dW and k == K - 1:
                for v in range(V):
                    for j in range(d):
                        dW[v, j] += delta[v] * hh[j]
                for j in range(d):
                    dgain[j] += dhh[j] * n[j]
        losses[k] = row_loss[k].sum() / T
    return {"losses": losses, "row_loss": row_loss, "dh": dh, "dW": dW, "dgain": dgain}
