"""Gradients of the masked second-order HLA, fp64 (test infrastructure only).

Sec. 4.2 states only that a reverse scan of the adjoint of (+), checkpointed
at tile boundaries, gives the gradients of the serial recurrence.  It prints
no formulas, so this module writes the vector-Jacobian product out from the
forward definition (Sec. 3.1)

    o_t = sum_{j<=t} sum_{i<=j} (q_t.k_i)(q_j.k_i) v_j = q_t^T Phi_t,
    Phi_t = sum_{j<=t} S_j q_j v_j^T,   S_j = sum_{i<=j} k_i k_i^T,

for a loss with upstream gradient g_t = dL/do_t.  Differentiating the double
sum term by term (q_t as the reading query, q_j inside Phi, k_i in both
factors, v_j linearly) and collecting the sums over the later tokens into the
reverse prefixes

    U_j = sum_{t>=j} q_t g_t^T   (d x dv),    u_j = U_j v_j,
    Z_i = sum_{j>=i} u_j q_j^T   (d x d),     r_j = S_j q_j,

gives

    dq_j = Phi_j g_j + S_j u_j,
    dv_j = U_j^T r_j,
    dk_i = (Z_i + Z_i^T) k_i.

The forward prefixes (S, Phi) run forward in time and the adjoint prefixes
(U, Z) run backward: the reverse scan of Sec. 4.2.

Functions
  hla2_vjp_autograd  torch autograd (fp64, CPU) through the dense definition
                     O = [(W W^T) (.) L] V, W = L (.) Q K^T: the reference the
                     written-out form is pinned against.
  hla2_vjp_serial    the three passes above, token by token.
  hla2_loss          sum_t g_t . o_t (for finite differences and identities).
Masked, unnormalised operator only.
"""
import numpy as np
import torch

from oracle.hla2 import hla2_definition


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def hla2_loss(q, k, v, g):
    """L = sum_t g_t . o_t for the masked operator."""
    return float((hla2_definition(q, k, v) * _f64(g)).sum())


def hla2_vjp_autograd(q, k, v, g):
    """(dq, dk, dv) of L = sum_t g_t . o_t by torch autograd in fp64 through
    the dense masked definition, per head over leading batch axes."""
    qt, kt, vt = (torch.tensor(_f64(x), dtype=torch.float64, requires_grad=True) for x in (q, k, v))
    gt = torch.tensor(_f64(g), dtype=torch.float64)
    n = qt.shape[-2]
    L = torch.tril(torch.ones(n, n, dtype=torch.float64))
    W = L * (qt @ kt.transpose(-1, -2))
    O = ((W @ W.transpose(-1, -2)) * L) @ vt
    (O * gt).sum().backward()
    return qt.grad.numpy(), kt.grad.numpy(), vt.grad.numpy()


def hla2_vjp_serial(q, k, v, g):
    """The written-out VJP (module header): a reverse pass for u_j = U_j v_j,
    a forward pass for dq_j = Phi_j g_j + S_j u_j (and r_j = S_j q_j), and a
    reverse pass for dv_j = U_j^T r_j and dk_i = (Z_i + Z_i^T) k_i.  Per head
    over leading batch axes; returns (dq, dk, dv)."""
    q, k, v, g = _f64(q), _f64(k), _f64(v), _f64(g)
    batch = q.shape[:-2]
    n, d = q.shape[-2:]
    dv_ = v.shape[-1]
    outer = lambda a, b: a[..., :, None] * b[..., None, :]
    mv = lambda M, x: np.einsum('...ab,...b->...a', M, x)
    u = np.empty(batch + (n, d))
    U = np.zeros(batch + (d, dv_))
    for j in range(n - 1, -1, -1):                  # U_j includes token j
        U = U + outer(q[..., j, :], g[..., j, :])
        u[..., j, :] = mv(U, v[..., j, :])
    dq = np.empty(batch + (n, d))
    r = np.empty(batch + (n, d))
    S = np.zeros(batch + (d, d))
    Phi = np.zeros(batch + (d, dv_))
    for j in range(n):                               # S_j and Phi_j include token j
        S = S + outer(k[..., j, :], k[..., j, :])
        r[..., j, :] = mv(S, q[..., j, :])
        Phi = Phi + outer(r[..., j, :], v[..., j, :])
        dq[..., j, :] = mv(Phi, g[..., j, :]) + mv(S, u[..., j, :])
    dk = np.empty(batch + (n, d))
    dv = np.empty(batch + (n, dv_))
    U = np.zeros(batch + (d, dv_))
    Z = np.zeros(batch + (d, d))
    for j in range(n - 1, -1, -1):                   # U_j and Z_j include token j
        U = U + outer(q[..., j, :], g[..., j, :])
        dv[..., j, :] = np.einsum('...ab,...a->...b', U, r[..., j, :])
        Z = Z + outer(u[..., j, :], q[..., j, :])
        dk[..., j, :] = mv(Z + np.swapaxes(Z, -1, -2), k[..., j, :])
    return dq, dk, dv
