"""Python binding of libdfssm.so, the MI355X (gfx950) DF-SSM scaffold + int8
LoRA linear (include/dfssm.h).

Argument marshalling only: every step runs in the library's HIP kernels.
PyTorch provides device memory and the current HIP stream.  Importing this
package loads the in-tree library and fails loudly if it has not been built
(``python paper_2606_10932_amd/build.py``); there is no fallback.
"""
from __future__ import annotations

import ctypes
import weakref
import os
from typing import List, Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdfssm.so")

OK, ERR_NULL, ERR_SHAPE, ERR_ALIGN, ERR_WORKSPACE, ERR_DEVICE, ERR_UNSUPPORTED = range(7)
F16, F32 = 0, 1
PATH_AUTO, PATH_DECODE, PATH_MFMA, PATH_MFMA_FEW = 0, 1, 2, 3

EXPORTS = ["dfssm_quantize_act", "dfssm_linear_workspace_bytes", "dfssm_scaffold_lora_linear",
           "dfssm_scaffold_lora_linear_ex", "dfssm_chain_workspace_bytes",
           "dfssm_scaffold_lora_chain", "dfssm_chain_prepare", "dfssm_chain_run", "dfssm_chain_status",
           "dfssm_chain_stream_floor", "dfssm_read_floor", "dfssm_read_floor_sink_words",
           "dfssm_exchange_pingpong", "dfssm_exchange_pingpong_bytes",
           "dfssm_embed_gather", "dfssm_lm_head", "dfssm_add_rmsnorm_quant", "dfssm_gate_norm_quant",
           "dfssm_ssm_step", "dfssm_linear_i4_workspace_bytes", "dfssm_scaffold_lora_linear_i4",
           "dfssm_mamba2_state_bytes", "dfssm_mamba2_workspace_bytes",
           "dfssm_mamba2_decode_step", "dfssm_mamba2_prepare", "dfssm_mamba2_release", "dfssm_mamba2_status", "dfssm_mamba2_fused_path", "dfssm_scaffold_lora_linear_noalloc", "dfssm_noalloc_scratch_bytes",
           "dfssm_test_switch", "dfssm_status_string", "dfssm_last_error",
           "dfssm_version"]
TEST_LOCAL_LORA, TEST_PREFILL_KERNEL, TEST_LM_HEAD_MFMA_TOKENS, TEST_STEP_PER_KERNEL = 1, 2, 3, 4
TEST_LM_HEAD_TILED_TOKENS = 5


class DfssmError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"dfssm status {status} ({msg})")
        self.status = status


class Layer(ctypes.Structure):
    """dfssm_layer: one projection of a chain (device pointers + sizes)."""
    _fields_ = [("w_bits", ctypes.c_void_p), ("alpha", ctypes.c_void_p), ("A", ctypes.c_void_p),
                ("B", ctypes.c_void_p), ("beta", ctypes.c_void_p), ("K", ctypes.c_int64),
                ("N", ctypes.c_int64), ("r", ctypes.c_int64), ("lora_bits", ctypes.c_int64)]


class Mamba2Layer(ctypes.Structure):
    """dfssm_mamba2_layer: one Mamba-2 layer (device pointers)."""
    _fields_ = [("norm_w", ctypes.c_void_p), ("in_proj", Layer), ("conv_w", ctypes.c_void_p),
                ("conv_b", ctypes.c_void_p), ("dt_bias", ctypes.c_void_p), ("A_log", ctypes.c_void_p),
                ("D", ctypes.c_void_p), ("gate_w", ctypes.c_void_p), ("out_proj", Layer),
                ("lora_bits", ctypes.c_int64)]


class Mamba2Model(ctypes.Structure):
    """dfssm_mamba2_model."""
    _fields_ = [("d_model", ctypes.c_int64), ("d_state", ctypes.c_int64), ("n_layers", ctypes.c_int64),
                ("vocab", ctypes.c_int64), ("eps", ctypes.c_float), ("E", ctypes.c_void_p),
                ("E_scale", ctypes.c_void_p), ("norm_f", ctypes.c_void_p),
                ("layers", ctypes.POINTER(Mamba2Layer))]


def _load(path: str = LIB_PATH) -> ctypes.CDLL:
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python paper_2606_10932_amd/build.py`")
    lib = ctypes.CDLL(path)
    vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_size_t
    lib.dfssm_quantize_act.argtypes = [vp, i32, i64, i64, i64, vp, vp, vp]
    lib.dfssm_quantize_act.restype = i32
    lib.dfssm_linear_workspace_bytes.argtypes = [i64, i64, i64, i64]
    lib.dfssm_linear_workspace_bytes.restype = sz
    lib.dfssm_scaffold_lora_linear.argtypes = [vp, vp, i64, i64, i64, i64, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.dfssm_scaffold_lora_linear.restype = i32
    lib.dfssm_scaffold_lora_linear_ex.argtypes = [vp, vp, i64, i64, i64, i64, vp, vp, vp, vp, vp, vp, i32,
                                                  vp, vp, vp, vp, sz, vp]
    lib.dfssm_scaffold_lora_linear_ex.restype = i32
    lib.dfssm_chain_workspace_bytes.argtypes = [ctypes.POINTER(Layer), i32, i64]
    lib.dfssm_chain_workspace_bytes.restype = sz
    lib.dfssm_scaffold_lora_chain.argtypes = [ctypes.POINTER(Layer), i32, i64, vp, vp, vp, vp, sz, vp]
    lib.dfssm_scaffold_lora_chain.restype = i32
    lib.dfssm_chain_prepare.argtypes = [ctypes.POINTER(Layer), i32, i64, vp, sz, vp]
    lib.dfssm_chain_prepare.restype = i32
    lib.dfssm_chain_run.argtypes = [ctypes.POINTER(Layer), i32, i64, vp, vp, vp, vp, sz, vp]
    lib.dfssm_chain_run.restype = i32
    lib.dfssm_chain_status.argtypes = [ctypes.POINTER(Layer), i32, i64, vp, sz, ctypes.POINTER(ctypes.c_uint), vp]
    lib.dfssm_chain_status.restype = i32
    lib.dfssm_chain_stream_floor.argtypes = [ctypes.POINTER(Layer), i32, vp, sz, vp]
    lib.dfssm_chain_stream_floor.restype = i32
    lib.dfssm_read_floor.argtypes = [vp, sz, vp, sz, vp]
    lib.dfssm_read_floor.restype = i32
    lib.dfssm_read_floor_sink_words.argtypes = [sz]
    lib.dfssm_read_floor_sink_words.restype = sz
    lib.dfssm_exchange_pingpong_bytes.argtypes = []
    lib.dfssm_exchange_pingpong_bytes.restype = sz
    lib.dfssm_exchange_pingpong.argtypes = [i32, i32, i32, vp, sz, ctypes.POINTER(ctypes.c_double), vp]
    lib.dfssm_exchange_pingpong.restype = i32
    lib.dfssm_embed_gather.argtypes = [vp, vp, i64, i64, vp, i64, vp, vp]
    lib.dfssm_embed_gather.restype = i32
    lib.dfssm_lm_head.argtypes = [vp, vp, i64, i64, vp, vp, i64, vp, vp, vp]
    lib.dfssm_lm_head.restype = i32
    f32 = ctypes.c_float
    lib.dfssm_add_rmsnorm_quant.argtypes = [vp, vp, vp, f32, i64, i64, vp, vp, vp, vp]
    lib.dfssm_add_rmsnorm_quant.restype = i32
    lib.dfssm_gate_norm_quant.argtypes = [vp, vp, i64, vp, f32, i64, i64, vp, vp, vp]
    lib.dfssm_gate_norm_quant.restype = i32
    lib.dfssm_ssm_step.argtypes = [vp, i64, i64, i64, i64, i64, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.dfssm_ssm_step.restype = i32
    lib.dfssm_linear_i4_workspace_bytes.argtypes = [i64, i64, i64, i64]
    lib.dfssm_linear_i4_workspace_bytes.restype = sz
    lib.dfssm_scaffold_lora_linear_i4.argtypes = [vp, vp, i64, i64, i64, i64, vp, vp, vp, vp, vp, vp, i32,
                                                  vp, vp, vp, vp, sz, vp]
    lib.dfssm_scaffold_lora_linear_i4.restype = i32
    mp = ctypes.POINTER(Mamba2Model)
    lib.dfssm_mamba2_state_bytes.argtypes = [mp, i64, ctypes.POINTER(sz), ctypes.POINTER(sz)]
    lib.dfssm_mamba2_state_bytes.restype = i32
    lib.dfssm_mamba2_workspace_bytes.argtypes = [mp, i64]
    lib.dfssm_mamba2_workspace_bytes.restype = sz
    lib.dfssm_mamba2_decode_step.argtypes = [mp, i64, vp, i64, vp, vp, vp, vp, sz, vp]
    lib.dfssm_mamba2_decode_step.restype = i32
    lib.dfssm_mamba2_prepare.argtypes = [mp, i64, vp, sz, vp]
    lib.dfssm_mamba2_prepare.restype = i32
    lib.dfssm_mamba2_release.argtypes = [vp]
    lib.dfssm_mamba2_release.restype = i32
    lib.dfssm_mamba2_status.argtypes = [mp, i64, vp, sz, ctypes.POINTER(ctypes.c_uint), vp]
    lib.dfssm_mamba2_status.restype = i32
    lib.dfssm_mamba2_fused_path.argtypes = [mp, i64, vp, sz, ctypes.POINTER(ctypes.c_int)]
    lib.dfssm_mamba2_fused_path.restype = i32
    lib.dfssm_scaffold_lora_linear_noalloc.argtypes = [vp, vp, i64, i64, i64, i64, vp, vp, vp, vp, vp, vp, vp]
    lib.dfssm_scaffold_lora_linear_noalloc.restype = i32
    lib.dfssm_noalloc_scratch_bytes.argtypes = []
    lib.dfssm_noalloc_scratch_bytes.restype = sz
    lib.dfssm_test_switch.argtypes = [i32, i32]
    lib.dfssm_test_switch.restype = i32
    lib.dfssm_status_string.argtypes = [i32]
    lib.dfssm_status_string.restype = ctypes.c_char_p
    lib.dfssm_last_error.restype = ctypes.c_char_p
    lib.dfssm_version.restype = ctypes.c_char_p
    return lib


lib = _load()


def last_error() -> str:
    return lib.dfssm_last_error().decode()


def _check(status: int):
    if status != OK:
        raise DfssmError(status, f"{lib.dfssm_status_string(status).decode()}: {last_error()}")


# ------------------------------------------------------------------ torch glue
def _torch():
    import torch
    return torch


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream=None) -> int:
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _need(t, dtype, name, ndim=None):
    torch = _torch()
    if t is None:
        return
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must be {ndim}-D")
    del torch


def linear_workspace_bytes(M: int, K: int, N: int, r: int) -> int:
    return int(lib.dfssm_linear_workspace_bytes(M, K, N, r))


def linear_workspace(M: int, K: int, N: int, r: int, device="cuda"):
    """A zero-filled workspace for the linear (zeros before its first use;
    pass it back unchanged to later calls)."""
    return _torch().zeros(max(linear_workspace_bytes(M, K, N, r), 1), dtype=_torch().uint8, device=device)


def test_switch(which: int, value: int):
    """Test-only kernel-family switch (dfssm_test_switch); 0 restores the
    automatic choice."""
    _check(lib.dfssm_test_switch(which, value))


def quantize_act(x, K: Optional[int] = None, q=None, s=None, stream=None):
    """Per-token absmax int8 quantisation of x ([M, ldx] fp16/fp32 device
    tensor, unit stride along K).  Returns (q int8 [M,K], s fp32 [M])."""
    torch = _torch()
    if x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be 2-D with unit column stride")
    M, ldx = x.shape[0], x.stride(0) if x.shape[0] > 1 else x.shape[1]
    K = x.shape[1] if K is None else K
    dt = {torch.float16: F16, torch.float32: F32}[x.dtype]
    q = torch.empty((M, K), dtype=torch.int8, device=x.device) if q is None else q
    s = torch.empty((M,), dtype=torch.float32, device=x.device) if s is None else s
    _need(q, torch.int8, "q", 2)
    _need(s, torch.float32, "s", 1)
    _check(lib.dfssm_quantize_act(x.data_ptr(), dt, M, K, ldx, q.data_ptr(), s.data_ptr(), _stream(stream)))
    return q, s


def scaffold_lora_linear(q, s, w_bits, alpha, A=None, B=None, beta=None, y=None, workspace=None,
                         path: int = PATH_AUTO, acc: bool = False, stream=None):
    """y = s*(alpha*acc_s + beta*acc_b) for int8 codes q [M,K], scales s [M],
    packed signs w_bits [N,K/32] (int32 or uint32 storage), alpha/beta [N],
    A [r,K], B [N,r].  With acc=True also returns (acc_s, acc_a, acc_b)."""
    torch = _torch()
    M, K = q.shape
    N = w_bits.shape[0]
    r = 0 if A is None else A.shape[0]
    _need(q, torch.int8, "q", 2)
    _need(s, torch.float32, "s", 1)
    if w_bits.dtype not in (torch.int32, torch.uint32):
        raise ValueError("w_bits must be int32/uint32 storage")
    _need(w_bits, w_bits.dtype, "w_bits", 2)
    if w_bits.shape[1] * 32 != K:
        raise ValueError("w_bits must be [N, K/32]")
    _need(alpha, torch.float32, "alpha", 1)
    if r:
        _need(A, torch.int8, "A", 2)
        _need(B, torch.int8, "B", 2)
        _need(beta, torch.float32, "beta", 1)
        if tuple(A.shape) != (r, K) or tuple(B.shape) != (N, r):
            raise ValueError("A must be [r,K] and B [N,r]")
    dev = q.device
    y = torch.empty((M, N), dtype=torch.float32, device=dev) if y is None else y
    _need(y, torch.float32, "y", 2)
    if workspace is None:
        workspace = linear_workspace(M, K, N, r, device=dev)
    acc_s = acc_a = acc_b = None
    if acc:
        acc_s = torch.empty((M, N), dtype=torch.int32, device=dev)
        acc_a = torch.empty((M, max(r, 1)), dtype=torch.int32, device=dev)
        acc_b = torch.empty((M, N), dtype=torch.int64, device=dev)
    st = lib.dfssm_scaffold_lora_linear_ex(
        q.data_ptr(), s.data_ptr(), M, K, N, r, w_bits.data_ptr(), alpha.data_ptr(),
        _ptr(A) if r else None, _ptr(B) if r else None, _ptr(beta) if r else None, y.data_ptr(),
        path, _ptr(acc_s), _ptr(acc_a) if r else None, _ptr(acc_b), workspace.data_ptr(),
        workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st)
    if acc:
        return y, acc_s, acc_a[:, :r], acc_b
    return y


def scaffold_lora_linear_noalloc(q, s, w_bits, alpha, A, B, beta, y, stream=None):
    """The linear on the library's own scratch array (no workspace; the
    library allocates nothing).  y [M, N] fp32 must be given."""
    torch = _torch()
    M, K = q.shape
    N = w_bits.shape[0]
    r = 0 if A is None else A.shape[0]
    _need(q, torch.int8, "q", 2)
    _need(s, torch.float32, "s", 1)
    _need(y, torch.float32, "y", 2)
    if tuple(y.shape) != (M, N):
        raise ValueError("y must be [M, N]")
    _check(lib.dfssm_scaffold_lora_linear_noalloc(
        q.data_ptr(), s.data_ptr(), M, K, N, r, w_bits.data_ptr(), alpha.data_ptr(), _ptr(A) if r else None,
        _ptr(B) if r else None, _ptr(beta) if r else None, y.data_ptr(), _stream(stream)))
    return y


def make_layers(layers: Sequence[dict]):
    """ctypes array of dfssm_layer from dicts of device tensors.  The array
    holds references to the tensors, so their memory lives as long as it."""
    arr = (Layer * len(layers))()
    for i, ly in enumerate(layers):
        arr[i] = _proj(ly)
    arr._tensors = [dict(ly) for ly in layers]
    return arr


def chain_workspace_bytes(layer_arr, M: int) -> int:
    return int(lib.dfssm_chain_workspace_bytes(layer_arr, len(layer_arr), M))


def scaffold_lora_chain(layers, q0, s0, y_all=None, workspace=None, layer_arr=None, stream=None) -> List:
    """Run the re-quantising chain.  Returns the list of per-linear outputs
    (views into y_all)."""
    torch = _torch()
    arr = make_layers(layers) if layer_arr is None else layer_arr
    M = q0.shape[0]
    Ns = [ly["w_bits"].shape[0] for ly in layers]
    total = M * sum(Ns)
    if y_all is None:
        y_all = torch.empty(total, dtype=torch.float32, device=q0.device)
    if workspace is None:
        workspace = torch.zeros(max(chain_workspace_bytes(arr, M), 1), dtype=torch.uint8, device=q0.device)
    _check(lib.dfssm_scaffold_lora_chain(arr, len(arr), M, q0.data_ptr(), s0.data_ptr(), y_all.data_ptr(),
                                         workspace.data_ptr(), workspace.numel(), _stream(stream)))
    outs, off = [], 0
    for N in Ns:
        outs.append(y_all[off:off + M * N].view(M, N))
        off += M * N
    return outs


def chain_prepare(layer_arr, M: int, workspace, stream=None):
    """Prepare `workspace` (device uint8 tensor) for chain_run on these layers."""
    _check(lib.dfssm_chain_prepare(layer_arr, len(layer_arr), M, workspace.data_ptr(), workspace.numel(),
                                   _stream(stream)))


def chain_run(layer_arr, q0, s0, y_all, workspace, stream=None):
    """Run a prepared chain: q0 [M,K0] int8, s0 [M] fp32 -> y_all (flat fp32)."""
    _check(lib.dfssm_chain_run(layer_arr, len(layer_arr), q0.shape[0], q0.data_ptr(), s0.data_ptr(),
                               y_all.data_ptr(), workspace.data_ptr(), workspace.numel(), _stream(stream)))


def chain_status(layer_arr, M: int, workspace, stream=None) -> int:
    """Synchronise and read the persistent chain's status word (0 = fine)."""
    out = ctypes.c_uint(0)
    _check(lib.dfssm_chain_status(layer_arr, len(layer_arr), M, workspace.data_ptr(), workspace.numel(),
                                  ctypes.byref(out), _stream(stream)))
    return int(out.value)


def chain_stream_floor(layer_arr, workspace, stream=None):
    """Diagnostic: the persistent chain's operand loads alone (no arithmetic,
    no exchange, no output) on a workspace prepared for these layers at M=1."""
    _check(lib.dfssm_chain_stream_floor(layer_arr, len(layer_arr), workspace.data_ptr(), workspace.numel(),
                                        _stream(stream)))


def exchange_pingpong(npairs: int = 1, iters: int = 2000, fence: bool = False, stream=None) -> float:
    """Diagnostic: ns per round trip (two hops) of one agent-scope word
    between workgroups on two XCDs, median over npairs concurrent pairs."""
    torch = _torch()
    ws = torch.empty(int(lib.dfssm_exchange_pingpong_bytes()), dtype=torch.uint8, device="cuda")
    out = ctypes.c_double(0.0)
    _check(lib.dfssm_exchange_pingpong(int(npairs), int(iters), 1 if fence else 0, ws.data_ptr(), ws.numel(),
                                       ctypes.byref(out), _stream(stream)))
    return float(out.value)


def read_floor_sink_words(nbytes: int) -> int:
    return int(lib.dfssm_read_floor_sink_words(int(nbytes)))


def read_floor(buf, sink, nbytes=None, stream=None):
    """Diagnostic: one launch reading nbytes (default: all) of the device
    tensor buf; the XOR of sink's first read_floor_sink_words(nbytes) words
    (int32, device) is then the XOR of the buffer's 32-bit words.  nbytes = 0
    is an empty launch."""
    torch = _torch()
    _need(sink, torch.int32, "sink", 1)
    n = buf.numel() * buf.element_size() if nbytes is None else int(nbytes)
    _check(lib.dfssm_read_floor(buf.data_ptr() if n > 0 else None, n, sink.data_ptr(), sink.numel(),
                                _stream(stream)))


def embed_gather(E, scale, tok, x=None, stream=None):
    """x [M, d] fp32 = scale[tok] * E[tok, :] for the int8 table E [V, d],
    row scales scale [V] and int32 ids tok [M]; ids outside [0, V) give zero
    rows."""
    torch = _torch()
    _need(E, torch.int8, "E", 2)
    _need(scale, torch.float32, "scale", 1)
    _need(tok, torch.int32, "tok", 1)
    V, d = E.shape
    M = tok.shape[0]
    x = torch.empty((M, d), dtype=torch.float32, device=E.device) if x is None else x
    _need(x, torch.float32, "x", 2)
    if tuple(x.shape) != (M, d) or scale.shape[0] != V:
        raise ValueError("x must be [M, d] and scale [V]")
    _check(lib.dfssm_embed_gather(E.data_ptr(), scale.data_ptr(), V, d, tok.data_ptr(), M, x.data_ptr(),
                                  _stream(stream)))
    return x


def lm_head(q, s, E, scale, logits=None, acc: bool = False, stream=None):
    """logits [M, V] fp32 = s[m] * (scale[v] * (E Q^T)[m, v]) for int8 codes
    q [M, d], scales s [M] and the tied int8 table E [V, d] with row scales
    scale [V].  With acc=True returns (logits, acc int32 [M, V])."""
    torch = _torch()
    _need(q, torch.int8, "q", 2)
    _need(s, torch.float32, "s", 1)
    _need(E, torch.int8, "E", 2)
    _need(scale, torch.float32, "scale", 1)
    M, d = q.shape
    V = E.shape[0]
    if E.shape[1] != d or scale.shape[0] != V or s.shape[0] != M:
        raise ValueError("E must be [V, d], scale [V] and s [M]")
    logits = torch.empty((M, V), dtype=torch.float32, device=q.device) if logits is None else logits
    _need(logits, torch.float32, "logits", 2)
    a = torch.empty((M, V), dtype=torch.int32, device=q.device) if acc else None
    _check(lib.dfssm_lm_head(q.data_ptr(), s.data_ptr(), M, d, E.data_ptr(), scale.data_ptr(), V,
                             logits.data_ptr(), _ptr(a), _stream(stream)))
    return (logits, a) if acc else logits


def add_rmsnorm_quant(u, w, eps: float = 1e-5, delta=None, u_out=None, q=None, s=None, stream=None):
    """(q int8 [M,d], s fp32 [M]) of rmsnorm(u + delta) * w; u_out (optional,
    may be u) receives u + delta."""
    torch = _torch()
    _need(u, torch.float32, "u", 2)
    _need(w, torch.float32, "w", 1)
    _need(delta, torch.float32, "delta", 2)
    _need(u_out, torch.float32, "u_out", 2)
    M, d = u.shape
    q = torch.empty((M, d), dtype=torch.int8, device=u.device) if q is None else q
    s = torch.empty((M,), dtype=torch.float32, device=u.device) if s is None else s
    _need(q, torch.int8, "q", 2)
    _need(s, torch.float32, "s", 1)
    _check(lib.dfssm_add_rmsnorm_quant(u.data_ptr(), _ptr(delta), w.data_ptr(), float(eps), M, d, _ptr(u_out),
                                       q.data_ptr(), s.data_ptr(), _stream(stream)))
    return q, s


def gate_norm_quant(y, z, w, eps: float = 1e-5, q=None, s=None, stream=None):
    """(q, s) of rmsnorm(y * silu(z)) * w; z may be a column slice of a wider
    row-major tensor (unit column stride)."""
    torch = _torch()
    _need(y, torch.float32, "y", 2)
    _need(w, torch.float32, "w", 1)
    if z.dim() != 2 or z.stride(1) != 1 or z.dtype != torch.float32 or not z.is_cuda:
        raise ValueError("z must be a 2-D fp32 device tensor with unit column stride")
    M, d = y.shape
    if tuple(z.shape) != (M, d):
        raise ValueError("z must have y's shape")
    ldz = z.stride(0) if M > 1 else max(z.stride(0), d)   # a single row's stride may be reported as anything
    q = torch.empty((M, d), dtype=torch.int8, device=y.device) if q is None else q
    s = torch.empty((M,), dtype=torch.float32, device=y.device) if s is None else s
    _check(lib.dfssm_gate_norm_quant(y.data_ptr(), z.data_ptr(), ldz, w.data_ptr(), float(eps), M, d, q.data_ptr(),
                                     s.data_ptr(), _stream(stream)))
    return q, s


def ssm_step(zxbcdt, step: int, conv_ring, ssm_state, conv_w, conv_b, dt_bias, A_log, D, d_state: int = 128,
             headdim: int = 64, y=None, xbc=None, stream=None):
    """Convolution + SSM step of one token per sequence; conv_ring
    [M, 4, conv_dim] and ssm_state [M, H, P, N] are updated in place.
    Returns y [M, d_inner]."""
    torch = _torch()
    _need(zxbcdt, torch.float32, "zxbcdt", 2)
    M, ld = zxbcdt.shape
    H = dt_bias.shape[0]
    d_inner = H * headdim
    for t, n in ((conv_ring, "conv_ring"), (ssm_state, "ssm_state"), (conv_w, "conv_w"), (conv_b, "conv_b"),
                 (dt_bias, "dt_bias"), (A_log, "A_log"), (D, "D")):
        _need(t, torch.float32, n)
    y = torch.empty((M, d_inner), dtype=torch.float32, device=zxbcdt.device) if y is None else y
    _need(y, torch.float32, "y", 2)
    _need(xbc, torch.float32, "xbc", 2)
    _check(lib.dfssm_ssm_step(zxbcdt.data_ptr(), ld, M, d_inner, d_state, headdim, int(step), conv_ring.data_ptr(),
                              conv_w.data_ptr(), conv_b.data_ptr(), dt_bias.data_ptr(), A_log.data_ptr(),
                              D.data_ptr(), ssm_state.data_ptr(), y.data_ptr(), _ptr(xbc), _stream(stream)))
    return y


class Mamba2:
    """A Mamba-2 model for dfssm_mamba2_decode_step: the host structs over
    the caller's device tensors (kept referenced here).

    layers: list of dicts with norm_w, conv_w, conv_b, dt_bias, A_log, D,
    gate_w (fp32 device tensors) and in_proj / out_proj (dicts of w_bits,
    alpha, A, B, beta as for scaffold_lora_linear, or w_bits, alpha, A4,
    B4, beta as for scaffold_lora_linear_i4; both projections of a layer
    alike)."""

    def __init__(self, E, E_scale, norm_f, layers, d_state: int = 128, eps: float = 1e-5):
        self._keep = [E, E_scale, norm_f, layers]
        self.vocab, self.d_model = E.shape
        self.n_layers = len(layers)
        self._layers = (Mamba2Layer * self.n_layers)()
        for i, L in enumerate(layers):
            i4 = "A4" in L["in_proj"]
            if i4 != ("A4" in L["out_proj"]):
                raise ValueError(f"layer {i}: in_proj and out_proj must both have int4 (A4, B4) or int8 factors")
            self._layers[i] = Mamba2Layer(L["norm_w"].data_ptr(), _proj(L["in_proj"]), L["conv_w"].data_ptr(),
                                          L["conv_b"].data_ptr(), L["dt_bias"].data_ptr(), L["A_log"].data_ptr(),
                                          L["D"].data_ptr(), L["gate_w"].data_ptr(), _proj(L["out_proj"]),
                                          4 if i4 else 8)
        self.struct = Mamba2Model(self.d_model, d_state, self.n_layers, self.vocab, eps, E.data_ptr(),
                                  E_scale.data_ptr(), norm_f.data_ptr(), self._layers)

    def state_bytes(self, M: int):
        c, s = ctypes.c_size_t(0), ctypes.c_size_t(0)
        _check(lib.dfssm_mamba2_state_bytes(ctypes.byref(self.struct), M, ctypes.byref(c), ctypes.byref(s)))
        return int(c.value), int(s.value)

    def new_state(self, M: int, device="cuda"):
        """Zero (conv_ring, ssm_state) for M new sequences."""
        torch = _torch()
        c, s = self.state_bytes(M)
        return (torch.zeros(c // 4, dtype=torch.float32, device=device),
                torch.zeros(s // 4, dtype=torch.float32, device=device))

    def workspace(self, M: int, device="cuda", prepare: bool = True, stream=None):
        """A zero-filled workspace (zeros before its first use), prepared for
        the fused step (dfssm_mamba2_prepare: at M = 1 for models of its
        shape; a no-op otherwise) unless prepare is False."""
        torch = _torch()
        ws = torch.zeros(int(lib.dfssm_mamba2_workspace_bytes(ctypes.byref(self.struct), M)), dtype=torch.uint8,
                         device=device)
        if prepare:
            self.prepare(M, ws, stream=stream)
        return ws

    def prepare(self, M: int, workspace, stream=None):
        """dfssm_mamba2_prepare; the record is dropped again (dfssm_mamba2_release)
        when the workspace tensor is freed, so a later tensor at the same
        address is not taken for a prepared one."""
        _check(lib.dfssm_mamba2_prepare(ctypes.byref(self.struct), M, workspace.data_ptr(), workspace.numel(),
                                        _stream(stream)))
        weakref.finalize(workspace, lib.dfssm_mamba2_release, ctypes.c_void_p(workspace.data_ptr()))

    def status(self, M: int, workspace, stream=None) -> int:
        """Synchronise and read the fused step's status word (0 = fine)."""
        out = ctypes.c_uint(0)
        _check(lib.dfssm_mamba2_status(ctypes.byref(self.struct), M, workspace.data_ptr(), workspace.numel(),
                                       ctypes.byref(out), _stream(stream)))
        return int(out.value)

    def fused_path(self, M: int, workspace) -> bool:
        """Whether decode_step at M on this workspace takes the fused step."""
        out = ctypes.c_int(0)
        _check(lib.dfssm_mamba2_fused_path(ctypes.byref(self.struct), M, workspace.data_ptr(), workspace.numel(),
                                           ctypes.byref(out)))
        return bool(out.value)

    def decode_step(self, tok, step: int, conv_ring, ssm_state, workspace, logits=None, stream=None):
        """One token for each of the M sequences (tok int32 [M]); returns
        logits [M, vocab]."""
        torch = _torch()
        _need(tok, torch.int32, "tok", 1)
        M = tok.shape[0]
        logits = torch.empty((M, self.vocab), dtype=torch.float32, device=tok.device) if logits is None else logits
        _check(lib.dfssm_mamba2_decode_step(ctypes.byref(self.struct), M, tok.data_ptr(), int(step),
                                            conv_ring.data_ptr(), ssm_state.data_ptr(), logits.data_ptr(),
                                            workspace.data_ptr(), workspace.numel(), _stream(stream)))
        return logits


def _proj(w) -> Layer:
    """dfssm_layer of a projection: int8 factors A, B or packed int4 A4, B4."""
    i4 = w.get("A4") is not None
    A = w.get("A4") if i4 else w.get("A")
    B = w.get("B4") if i4 else w.get("B")
    r = 0 if A is None else A.shape[0]
    return Layer(w["w_bits"].data_ptr(), w["alpha"].data_ptr(), _ptr(A) if r else None, _ptr(B) if r else None,
                 _ptr(w.get("beta")) if r else None, w["w_bits"].shape[1] * 32, w["w_bits"].shape[0], r,
                 4 if i4 else 0)


def scaffold_lora_linear_i4(q, s, w_bits, alpha, A4=None, B4=None, beta=None, y=None, workspace=None,
                            path: int = PATH_AUTO, acc: bool = False, stream=None):
    """The linear with int4 LoRA factors: A4 uint8 [r, K/2], B4 uint8 [N, r/2]
    (two's-complement nibbles, low nibble first).  Same results as
    scaffold_lora_linear on the unpacked factors."""
    torch = _torch()
    M, K = q.shape
    N = w_bits.shape[0]
    r = 0 if A4 is None else A4.shape[0]
    _need(q, torch.int8, "q", 2)
    _need(s, torch.float32, "s", 1)
    _need(alpha, torch.float32, "alpha", 1)
    if r:
        _need(A4, torch.uint8, "A4", 2)
        _need(B4, torch.uint8, "B4", 2)
        _need(beta, torch.float32, "beta", 1)
        if tuple(A4.shape) != (r, K // 2) or tuple(B4.shape) != (N, r // 2):
            raise ValueError("A4 must be [r, K/2] and B4 [N, r/2] bytes")
    dev = q.device
    y = torch.empty((M, N), dtype=torch.float32, device=dev) if y is None else y
    nbytes = int(lib.dfssm_linear_i4_workspace_bytes(M, K, N, r))
    if workspace is None:
        workspace = torch.zeros(max(nbytes, 1), dtype=torch.uint8, device=dev)
    acc_s = acc_a = acc_b = None
    if acc:
        acc_s = torch.empty((M, N), dtype=torch.int32, device=dev)
        acc_a = torch.empty((M, max(r, 1)), dtype=torch.int32, device=dev)
        acc_b = torch.empty((M, N), dtype=torch.int64, device=dev)
    _check(lib.dfssm_scaffold_lora_linear_i4(
        q.data_ptr(), s.data_ptr(), M, K, N, r, w_bits.data_ptr(), alpha.data_ptr(), _ptr(A4) if r else None,
        _ptr(B4) if r else None, _ptr(beta) if r else None, y.data_ptr(), path, _ptr(acc_s),
        _ptr(acc_a) if r else None, _ptr(acc_b), workspace.data_ptr(), workspace.numel(), _stream(stream)))
    if acc:
        return y, acc_s, acc_a[:, :r], acc_b
    return y
