"""Torch-facing helpers over the C ABI.

torch supplies device memory and the current HIP stream; every step of the
computation runs in libhla.so.  Tensors must be contiguous CUDA (HIP) tensors;
q/k/v are float32 or bfloat16, outputs and states are float32.
"""
import torch

from . import capi


def _code(t):
    if t.dtype == torch.bfloat16:
        return capi.HLA_BF16
    if t.dtype == torch.float32:
        return capi.HLA_FP32
    raise TypeError(f"q/k/v must be float32 or bfloat16, got {t.dtype}")


def _check(*ts):
    for t in ts:
        if not t.is_cuda:
            raise ValueError("tensors must be on the GPU")
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous")


def _stream():
    return torch.cuda.current_stream().cuda_stream


def state_floats(d, dv):
    return capi.hla2_state_floats(d, dv)


def new_state(B, H, d, dv, device="cuda"):
    """Zero state [B, H, F] (the identity segment)."""
    return torch.zeros(B, H, state_floats(d, dv), dtype=torch.float32, device=device)


def split_state(state, d, dv):
    """Views (S, C, m, G, h) of a state tensor [..., F]."""
    o = [0, d * d, d * d + d * dv, d * d + d * dv + d, d * d + 2 * d * dv + d, d * d + 2 * d * dv + 2 * d]
    shp = state.shape[:-1]
    return (state[..., o[0]:o[1]].reshape(*shp, d, d), state[..., o[1]:o[2]].reshape(*shp, d, dv),
            state[..., o[2]:o[3]], state[..., o[3]:o[4]].reshape(*shp, d, dv), state[..., o[4]:o[5]])


def workspace_bytes(B, H, n, d, dv, chunk, dtype_code, algo=capi.HLA_ALGO_AUTO):
    return capi.hla2_workspace_bytes_ex(B, H, n, d, dv, chunk, dtype_code, algo)


def forward(q, k, v, chunk, masked=True, normalized=False, eps=1e-6, algo=capi.HLA_ALGO_AUTO, out=None,
            workspace=None):
    """hla2_forward_ex on torch tensors q, k [B,H,n,d], v [B,H,n,dv] -> out fp32 [B,H,n,dv]."""
    _check(q, k, v)
    B, H, n, d = q.shape
    dv = v.shape[-1]
    code = _code(q)
    if out is None:
        out = torch.empty(B, H, n, dv, dtype=torch.float32, device=q.device)
    wsb = capi.hla2_workspace_bytes_ex(B, H, n, d, dv, chunk, code, algo)
    if workspace is None:
        workspace = torch.empty(max(wsb, 1), dtype=torch.uint8, device=q.device)
    capi.hla2_forward_ex(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), B, H, n, d, dv, chunk,
                         int(masked), int(normalized), float(eps), code, workspace.data_ptr(),
                         workspace.numel(), int(algo), _stream())
    return out


def chunk_summaries(q, k, v, chunk):
    """Per-chunk summaries [B, H, M, F]."""
    _check(q, k, v)
    B, H, n, d = q.shape
    dv = v.shape[-1]
    M = (n + chunk - 1) // chunk
    states = torch.empty(B, H, M, state_floats(d, dv), dtype=torch.float32, device=q.device)
    capi.hla2_chunk_summaries(q.data_ptr(), k.data_ptr(), v.data_ptr(), states.data_ptr(), B, H, n, d, dv, chunk,
                              _code(q), _stream())
    return states


def scan(states, d, dv, init=None):
    """Exclusive (+)-scan of states [B, H, M, F] -> (prefix [B,H,M,F], total [B,H,F])."""
    _check(states)
    B, H, M, F = states.shape
    prefix = torch.empty_like(states)
    total = torch.empty(B, H, F, dtype=torch.float32, device=states.device)
    if init is not None:
        _check(init)
    capi.hla2_scan(states.data_ptr(), init.data_ptr() if init is not None else None, prefix.data_ptr(),
                   total.data_ptr(), B, H, M, d, dv, _stream())
    return prefix, total


def prefill(state, q, k, v, chunk, masked=True, normalized=False, eps=1e-6, want_out=True, workspace=None):
    """state <- state (+) summary(q, k, v) in place; returns the outputs (or None)."""
    _check(state, q, k, v)
    B, H, n, d = q.shape
    dv = v.shape[-1]
    code = _code(q)
    out = torch.empty(B, H, n, dv, dtype=torch.float32, device=q.device) if want_out else None
    wsb = capi.hla2_prefill_workspace_bytes(B, H, n, d, dv, chunk, code)
    if workspace is None:
        workspace = torch.empty(wsb, dtype=torch.uint8, device=q.device)
    capi.hla2_prefill(state.data_ptr(), q.data_ptr(), k.data_ptr(), v.data_ptr(),
                      out.data_ptr() if out is not None else None, B, H, n, d, dv, chunk, int(masked),
                      int(normalized), float(eps), code, workspace.data_ptr(), workspace.numel(), _stream())
    return out


def step(state, q_t, k_t, v_t, masked=True, normalized=False, eps=1e-6, out=None):
    """One decode step: q_t, k_t [B,H,d], v_t [B,H,dv]; state [B,H,F] updated in place."""
    _check(state, q_t, k_t, v_t)
    B, H, d = q_t.shape
    dv = v_t.shape[-1]
    if out is None:
        out = torch.empty(B, H, dv, dtype=torch.float32, device=q_t.device)
    capi.hla2_step(state.data_ptr(), q_t.data_ptr(), k_t.data_ptr(), v_t.data_ptr(), out.data_ptr(), B, H, d, dv,
                   int(masked), int(normalized), float(eps), _code(q_t), _stream())
    return out


def forward_decay(q, k, v, chunk, gamma, masked=True, normalized=False, eps=1e-6, out=None, workspace=None):
    """Second-order HLA with decay gamma, q, k [B,H,n,d], v [B,H,n,dv] -> out fp32."""
    _check(q, k, v)
    B, H, n, d = q.shape
    dv = v.shape[-1]
    code = _code(q)
    if out is None:
        out = torch.empty(B, H, n, dv, dtype=torch.float32, device=q.device)
    wsb = capi.hla2_forward_decay_workspace_bytes(B, H, n, d, dv, chunk, code)
    if workspace is None:
        workspace = torch.empty(max(wsb, 1), dtype=torch.uint8, device=q.device)
    capi.hla2_forward_decay(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), B, H, n, d, dv, chunk,
                            int(masked), int(normalized), float(eps), float(gamma), code, workspace.data_ptr(),
                            workspace.numel(), _stream())
    return out


def backward(q, k, v, g, chunk=64, workspace=None):
    """Gradients (dq, dk, dv), fp32, of the masked unnormalised second-order HLA
    for upstream gradient g [B,H,n,dv] fp32; q, k, v [B,H,n,d] bf16."""
    g = g.float().contiguous()
    _check(q, k, v, g)
    B, H, n, d = q.shape
    dv_dim = v.shape[-1]
    code = _code(q)
    dq = torch.empty(B, H, n, d, dtype=torch.float32, device=q.device)
    dk = torch.empty_like(dq)
    dv = torch.empty(B, H, n, dv_dim, dtype=torch.float32, device=q.device)
    wsb = capi.hla2_backward_workspace_bytes(B, H, n, d, dv_dim, chunk, code)
    if workspace is None:
        workspace = torch.empty(max(wsb, 1), dtype=torch.uint8, device=q.device)
    capi.hla2_backward(q.data_ptr(), k.data_ptr(), v.data_ptr(), g.data_ptr(), dq.data_ptr(), dk.data_ptr(),
                       dv.data_ptr(), B, H, n, d, dv_dim, chunk, code, workspace.data_ptr(), workspace.numel(),
                       _stream())
    return dq, dk, dv


class HLA2(torch.autograd.Function):
    """Masked second-order HLA as a differentiable op: forward by the library's
    forward, backward by hla2_backward (bf16 q, k, v; fp32 output)."""

    @staticmethod
    def forward(ctx, q, k, v, chunk):
        ctx.save_for_backward(q, k, v)
        ctx.chunk = chunk
        return forward(q, k, v, chunk)

    @staticmethod
    def backward(ctx, g):
        q, k, v = ctx.saved_tensors
        dq, dk, dv = backward(q, k, v, g, ctx.chunk)
        return dq.to(q.dtype), dk.to(k.dtype), dv.to(v.dtype), None


def hla2_attention(q, k, v, chunk=64):
    """Differentiable masked second-order HLA (see HLA2)."""
    return HLA2.apply(q, k, v, chunk)


def ahla_forward(q, k, v, chunk, normalized=False, eps=1e-6, out=None, workspace=None):
    """AHLA (Sec. 6), ((A A) (.) L) V with A = L (.) Q K^T; q, k, v [B,H,n,d] bf16 -> out fp32."""
    _check(q, k, v)
    B, H, n, d = q.shape
    dv = v.shape[-1]
    code = _code(q)
    if out is None:
        out = torch.empty(B, H, n, dv, dtype=torch.float32, device=q.device)
    wsb = capi.ahla_workspace_bytes(B, H, n, d, dv, chunk, code)
    if workspace is None:
        workspace = torch.empty(max(wsb, 1), dtype=torch.uint8, device=q.device)
    capi.ahla_forward(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), B, H, n, d, dv, chunk,
                      int(normalized), float(eps), code, workspace.data_ptr(), workspace.numel(), _stream())
    return out


def hla3_forward(q, k, v, chunk, masked=True, normalized=False, eps=1e-6, out=None, workspace=None):
    """Third-order HLA (masked or unmasked), q, k [B,H,n,d], v [B,H,n,dv] -> out fp32."""
    _check(q, k, v)
    B, H, n, d = q.shape
    dv = v.shape[-1]
    code = _code(q)
    if out is None:
        out = torch.empty(B, H, n, dv, dtype=torch.float32, device=q.device)
    wsb = capi.hla3_workspace_bytes(B, H, n, d, dv, chunk, code)
    if workspace is None:
        workspace = torch.empty(max(wsb, 1), dtype=torch.uint8, device=q.device)
    capi.hla3_forward(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), B, H, n, d, dv, chunk,
                      int(masked), int(normalized), float(eps), code, workspace.data_ptr(), workspace.numel(),
                      _stream())
    return out
