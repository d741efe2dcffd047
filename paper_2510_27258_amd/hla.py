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


def _qkv(q, k, v, rank=4):
    """Shapes, dtypes and devices of q, k [..., d] and v [..., dv] (rank 4 for
    sequences [B, H, n, *], 3 for decode tokens [B, H, *]).  The C ABI sees
    only pointers and sizes taken from q, so a mismatched k or v would be read
    out of bounds: these checks run before any launch."""
    for name, t in (("q", q), ("k", k), ("v", v)):
        if t.dim() != rank:
            raise ValueError(f"{name} must have {rank} dimensions, got shape {tuple(t.shape)}")
    if k.shape != q.shape:
        raise ValueError(f"k must have q's shape {tuple(q.shape)}, got {tuple(k.shape)}")
    if v.shape[:-1] != q.shape[:-1]:
        raise ValueError(f"v must match q on {tuple(q.shape[:-1])}, got {tuple(v.shape)}")
    if k.dtype != q.dtype or v.dtype != q.dtype:
        raise ValueError(f"q, k and v must share one dtype, got {q.dtype}, {k.dtype}, {v.dtype}")
    if k.device != q.device or v.device != q.device:
        raise ValueError("q, k and v must be on one device")
    _code(q)
    _check(q, k, v)


def _fp32_out(out, shape, device, name="out"):
    """A caller's output tensor must be contiguous fp32 of exactly `shape` on `device`."""
    if out is None:
        return torch.empty(*shape, dtype=torch.float32, device=device)
    if out.dtype != torch.float32 or tuple(out.shape) != tuple(shape):
        raise ValueError(f"{name} must be float32 {tuple(shape)}, got {out.dtype} {tuple(out.shape)}")
    if out.device != device:
        raise ValueError(f"{name} must be on {device}")
    _check(out)
    return out


def _workspace(ws, nbytes, device):
    if ws is None:
        return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)
    if ws.device != device:
        raise ValueError(f"workspace must be on {device}")
    _check(ws)
    return ws


def _ws_bytes(ws):
    return ws.numel() * ws.element_size()


def _stream():
    return torch.cuda.current_stream().cuda_stream


def state_floats(d, dv):
    return capi.hla2_state_floats(d, dv)


def split_state(state, d, dv):
    """Views (S, C, m, G, h) of a state tensor [..., F]."""
    o = [0, d * d, d * d + d * dv, d * d + d * dv + d, d * d + 2 * d * dv + d, d * d + 2 * d * dv + 2 * d]
    shp = state.shape[:-1]
    return (state[..., o[0]:o[1]].reshape(*shp, d, d), state[..., o[1]:o[2]].reshape(*shp, d, dv),
            state[..., o[2]:o[3]], state[..., o[3]:o[4]].reshape(*shp, d, dv), state[..., o[4]:o[5]])


class State:
    """A decode state (the hla2_state descriptor of the C ABI): per-head
    records `data` [B, H, FP] fp32 in device memory (S packed symmetric, see
    include/hla.h), zeroed at creation (the identity segment), and the
    operator (masked, normalized, eps) and token dtype that every prefill and
    step on it uses.  `export()` returns the full records [B, H, F]."""

    def __init__(self, B, H, d, dv, masked=True, normalized=False, eps=1e-6, dtype=torch.bfloat16,
                 device="cuda"):
        code = _code(torch.empty(0, dtype=dtype))
        nbytes = capi.hla2_state_bytes(B, H, d, dv)
        if nbytes == 0:
            raise capi.HLAError(capi.HLA_ERR_INVALID, capi.hla_last_error())
        self.B, self.H, self.d, self.dv = B, H, d, dv
        self.dtype = dtype
        self.data = torch.empty(B, H, nbytes // (4 * B * H), dtype=torch.float32, device=device)
        self.desc = capi.HLA2State()
        capi.hla2_state_init(self.desc, self.data.data_ptr(), nbytes, B, H, d, dv, int(masked), int(normalized),
                             float(eps), code, _stream())

    def export(self):
        """The state as full records [B, H, F] (S as a d x d matrix), made by hla2_state_export."""
        full = torch.empty(self.B, self.H, state_floats(self.d, self.dv), dtype=torch.float32,
                           device=self.data.device)
        capi.hla2_state_export(self.desc, full.data_ptr(), _stream())
        return full

    def _tokens(self, q, k, v, rank):
        _qkv(q, k, v, rank)
        if q.dtype != self.dtype:
            raise ValueError(f"this state takes {self.dtype} tokens, got {q.dtype}")
        if q.device != self.data.device:
            raise ValueError(f"tokens must be on {self.data.device}")
        if tuple(q.shape[:2]) != (self.B, self.H) or q.shape[-1] != self.d or v.shape[-1] != self.dv:
            raise ValueError(f"tokens must be [{self.B}, {self.H}, ..., {self.d}] and [..., {self.dv}], "
                             f"got {tuple(q.shape)} and {tuple(v.shape)}")


def workspace_bytes(B, H, n, d, dv, chunk, dtype_code, algo=capi.HLA_ALGO_AUTO):
    return capi.hla2_workspace_bytes_ex(B, H, n, d, dv, chunk, dtype_code, algo)


def forward(q, k, v, chunk, masked=True, normalized=False, eps=1e-6, algo=capi.HLA_ALGO_AUTO, out=None,
            workspace=None, den=None):
    """hla2_forward_ex on torch tensors q, k [B,H,n,d], v [B,H,n,dv] -> out fp32 [B,H,n,dv].
    den: an fp32 [B,H,n] tensor that receives den_t (normalized only), or None."""
    _qkv(q, k, v)
    B, H, n, d = q.shape
    dv = v.shape[-1]
    code = _code(q)
    out = _fp32_out(out, (B, H, n, dv), q.device)
    if den is not None:
        den = _fp32_out(den, (B, H, n), q.device, "den")
    workspace = _workspace(workspace, capi.hla2_workspace_bytes_ex(B, H, n, d, dv, chunk, code, algo), q.device)
    capi.hla2_forward_ex(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                         den.data_ptr() if den is not None else None, B, H, n, d, dv, chunk,
                         int(masked), int(normalized), float(eps), code, workspace.data_ptr(),
                         _ws_bytes(workspace), int(algo), _stream())
    return out


def chunk_summaries(q, k, v, chunk):
    """Per-chunk summaries [B, H, M, F]."""
    _qkv(q, k, v)
    B, H, n, d = q.shape
    dv = v.shape[-1]
    M = (n + chunk - 1) // chunk
    states = torch.empty(B, H, M, state_floats(d, dv), dtype=torch.float32, device=q.device)
    capi.hla2_chunk_summaries(q.data_ptr(), k.data_ptr(), v.data_ptr(), states.data_ptr(), B, H, n, d, dv, chunk,
                              _code(q), _stream())
    return states


def scan(states, d, dv, init=None):
    """Exclusive (+)-scan of states [B, H, M, F] -> (prefix [B,H,M,F], total [B,H,F])."""
    if states.dim() != 4 or states.dtype != torch.float32 or states.shape[-1] != state_floats(d, dv):
        raise ValueError(f"states must be float32 [B, H, M, {state_floats(d, dv)}], got {states.dtype} "
                         f"{tuple(states.shape)}")
    _check(states)
    B, H, M, F = states.shape
    if init is not None:
        if init.dtype != torch.float32 or tuple(init.shape) != (B, H, F) or init.device != states.device:
            raise ValueError(f"init must be float32 [{B}, {H}, {F}] on {states.device}")
        _check(init)
    prefix = torch.empty_like(states)
    total = torch.empty(B, H, F, dtype=torch.float32, device=states.device)
    capi.hla2_scan(states.data_ptr(), init.data_ptr() if init is not None else None, prefix.data_ptr(),
                   total.data_ptr(), B, H, M, d, dv, _stream())
    return prefix, total


def prefill(state, q, k, v, chunk, want_out=True, workspace=None):
    """state <- state (+) summary(q, k, v) in place (a State); returns the
    outputs of those tokens under the state's operator (or None)."""
    state._tokens(q, k, v, 4)
    B, H, n, d = q.shape
    dv = v.shape[-1]
    out = torch.empty(B, H, n, dv, dtype=torch.float32, device=q.device) if want_out else None
    wsb = capi.hla2_prefill_workspace_bytes(state.desc, n, chunk)
    if wsb == 0:
        raise capi.HLAError(capi.HLA_ERR_INVALID, capi.hla_last_error())
    workspace = _workspace(workspace, wsb, q.device)
    capi.hla2_prefill(state.desc, q.data_ptr(), k.data_ptr(), v.data_ptr(), n, chunk,
                      out.data_ptr() if out is not None else None, workspace.data_ptr(), _ws_bytes(workspace),
                      _stream())
    return out


def step(state, q_t, k_t, v_t, out=None):
    """One decode step on a State: q_t, k_t [B,H,d], v_t [B,H,dv] -> out fp32 [B,H,dv]."""
    state._tokens(q_t, k_t, v_t, 3)
    out = _fp32_out(out, (state.B, state.H, state.dv), q_t.device)
    capi.hla2_step(state.desc, q_t.data_ptr(), k_t.data_ptr(), v_t.data_ptr(), out.data_ptr(), _stream())
    return out


def forward_decay(q, k, v, chunk, gamma, masked=True, normalized=False, eps=1e-6, out=None, workspace=None):
    """Second-order HLA with decay gamma, q, k [B,H,n,d], v [B,H,n,dv] -> out fp32."""
    _qkv(q, k, v)
    B, H, n, d = q.shape
    dv = v.shape[-1]
    code = _code(q)
    out = _fp32_out(out, (B, H, n, dv), q.device)
    workspace = _workspace(workspace, capi.hla2_forward_decay_workspace_bytes(B, H, n, d, dv, chunk, code), q.device)
    capi.hla2_forward_decay(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), B, H, n, d, dv, chunk,
                            int(masked), int(normalized), float(eps), float(gamma), code, workspace.data_ptr(),
                            _ws_bytes(workspace), _stream())
    return out


def backward(q, k, v, g, chunk=64, workspace=None):
    """Gradients (dq, dk, dv), fp32, of the masked unnormalised second-order HLA
    for upstream gradient g [B,H,n,dv] fp32; q, k, v [B,H,n,d] bf16."""
    _qkv(q, k, v)
    if tuple(g.shape) != tuple(v.shape):
        raise ValueError(f"g must have v's shape {tuple(v.shape)}, got {tuple(g.shape)}")
    if g.device != q.device:
        raise ValueError(f"g must be on {q.device}")
    g = g.float().contiguous()
    B, H, n, d = q.shape
    dv_dim = v.shape[-1]
    code = _code(q)
    dq = torch.empty(B, H, n, d, dtype=torch.float32, device=q.device)
    dk = torch.empty_like(dq)
    dv = torch.empty(B, H, n, dv_dim, dtype=torch.float32, device=q.device)
    workspace = _workspace(workspace, capi.hla2_backward_workspace_bytes(B, H, n, d, dv_dim, chunk, code), q.device)
    capi.hla2_backward(q.data_ptr(), k.data_ptr(), v.data_ptr(), g.data_ptr(), dq.data_ptr(), dk.data_ptr(),
                       dv.data_ptr(), B, H, n, d, dv_dim, chunk, code, workspace.data_ptr(), _ws_bytes(workspace),
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
    _qkv(q, k, v)
    B, H, n, d = q.shape
    dv = v.shape[-1]
    code = _code(q)
    out = _fp32_out(out, (B, H, n, dv), q.device)
    workspace = _workspace(workspace, capi.ahla_workspace_bytes(B, H, n, d, dv, chunk, code), q.device)
    capi.ahla_forward(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), B, H, n, d, dv, chunk,
                      int(normalized), float(eps), code, workspace.data_ptr(), _ws_bytes(workspace), _stream())
    return out


def hla3_forward(q, k, v, chunk, masked=True, normalized=False, eps=1e-6, out=None, workspace=None):
    """Third-order HLA (masked or unmasked), q, k [B,H,n,d], v [B,H,n,dv] -> out fp32."""
    _qkv(q, k, v)
    B, H, n, d = q.shape
    dv = v.shape[-1]
    code = _code(q)
    out = _fp32_out(out, (B, H, n, dv), q.device)
    workspace = _workspace(workspace, capi.hla3_workspace_bytes(B, H, n, d, dv, chunk, code), q.device)
    capi.hla3_forward(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), B, H, n, d, dv, chunk,
                      int(masked), int(normalized), float(eps), code, workspace.data_ptr(), _ws_bytes(workspace),
                      _stream())
    return out
