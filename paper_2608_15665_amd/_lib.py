"""ctypes binding of libzo (the C ABI declared in include/zo.h).

Argument marshalling only: every computation runs in the library's HIP
kernels.  Tensors are torch tensors on the GPU (PyTorch provides device
memory and the current stream); they are checked for device, dtype and
contiguity and handed over as raw pointers.  There is no CPU fallback: if
libzo.so is missing or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
import threading
from typing import Optional, Sequence

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libzo.so")

ZO_F32, ZO_BF16, ZO_F16 = 0, 1, 2
ZO_MAX_RANK = 128
ZO_MAX_QR_RANK = 128
ZO_MAX_BLOCKS = 256
STATUS = {0: "ok", 1: "invalid argument", 2: "unsupported", 3: "rank deficient",
          4: "non-finite value", 5: "HIP runtime error", 6: "workspace too small"}

ABI_SYMBOLS = (
    "zo_abi_version", "zo_status_str", "zo_last_error_detail",
    "zo_subspace_refresh_workspace", "zo_subspace_refresh",
    "zo_perturbed_linear_workspace", "zo_perturbed_linear",
    "zo_perturbed_linear_prepare", "zo_perturbed_linear_apply",
    "zo_lora_perturbed_linear_workspace", "zo_lora_perturbed_linear",
    "zo_lora_perturbed_linear_prepare",
    "zo_subspace_adam_update_workspace", "zo_subspace_adam_update",
    "zo_subspace_sgd_update_workspace", "zo_subspace_sgd_update",
    "zo_sq_loss_workspace", "zo_sq_loss", "zo_combine_central", "zo_combine_forward",
    "zo_perturbed_linear_apply_ex", "zo_layernorm", "zo_causal_attention",
    "zo_decoder_layer_workspace", "zo_decoder_layer_forward",
    "zo_rmsnorm", "zo_rope", "zo_llama_layer_workspace", "zo_llama_layer_forward",
    "zo_causal_attention_gqa", "zo_llama_lora_layer_workspace", "zo_llama_lora_layer_forward",
    "zo_perturbed_linear_group_workspace", "zo_perturbed_linear_prepare_group",
    "zo_subspace_refresh_noalloc",
)
ZO_NOALLOC_SCRATCH_BYTES = 64 << 20
ZO_EPI_NONE, ZO_EPI_RELU, ZO_EPI_RESIDUAL, ZO_EPI_SILU_MUL = 0, 1, 2, 3


class Matrix(ctypes.Structure):
    """zo_matrix: one perturbed matrix (device pointers)."""
    _fields_ = [("W", ctypes.c_void_p), ("U", ctypes.c_void_p), ("V", ctypes.c_void_p), ("Z", ctypes.c_void_p)]


class DecoderLayerDesc(ctypes.Structure):
    """zo_decoder_layer: six perturbed matrices and the two layer norms' parameters."""
    _fields_ = [(nm, Matrix) for nm in ("q", "k", "v", "o", "fc1", "fc2")] + [
        (nm, ctypes.c_void_p) for nm in ("ln1_gamma", "ln1_beta", "ln2_gamma", "ln2_beta")]


class LlamaLayerDesc(ctypes.Structure):
    """zo_llama_layer: seven perturbed matrices and the two RMS norms' gamma."""
    _fields_ = [(nm, Matrix) for nm in ("q", "k", "v", "o", "gate", "up", "down")] + [
        (nm, ctypes.c_void_p) for nm in ("rms1_gamma", "rms2_gamma")]


class LoraMatrix(ctypes.Structure):
    """zo_lora_matrix: a frozen W and its LoRA factors with their subspaces and coefficients."""
    _fields_ = [(nm, ctypes.c_void_p) for nm in ("W", "A", "U_A", "V_A", "Z_A", "B", "U_B", "V_B", "Z_B")]


class LlamaLoraLayerDesc(ctypes.Structure):
    """zo_llama_lora_layer: adapted q and v, the frozen k, o, gate, up, down, the RMS gammas."""
    _fields_ = [("q", LoraMatrix), ("v", LoraMatrix)] + [
        (nm, ctypes.c_void_p) for nm in ("k", "o", "gate", "up", "down", "rms1_gamma", "rms2_gamma")]


class ZoError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"libzo: {STATUS.get(status, status)}: {detail}")
        self.status = status
        self.detail = detail


class Panel(ctypes.Structure):
    _fields_ = [("rows", ctypes.c_int), ("omega", ctypes.c_void_p),
                ("q", ctypes.c_void_p), ("r_diag", ctypes.c_void_p)]


class UpdateItem(ctypes.Structure):
    _fields_ = [("m", ctypes.c_int), ("n", ctypes.c_int), ("W", ctypes.c_void_p),
                ("U", ctypes.c_void_p), ("V", ctypes.c_void_p), ("Z", ctypes.c_void_p),
                ("M1", ctypes.c_void_p), ("M2", ctypes.c_void_p),
                ("zbar_out", ctypes.c_void_p), ("w_f32_out", ctypes.c_void_p)]


_lib = None
_lock = threading.Lock()


def lib() -> ctypes.CDLL:
    """The loaded libzo.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                                   "`python -m paper_2608_15665_amd._build` (or __graft_entry__.build())")
            L = ctypes.CDLL(LIB_PATH)
            c_int, c_vp, c_sz, c_f, c_ll = (ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t,
                                           ctypes.c_float, ctypes.c_longlong)
            L.zo_abi_version.restype = c_int
            L.zo_status_str.restype = ctypes.c_char_p
            L.zo_status_str.argtypes = [c_int]
            L.zo_last_error_detail.restype = ctypes.c_char_p
            L.zo_subspace_refresh_workspace.restype = c_sz
            L.zo_subspace_refresh_workspace.argtypes = [c_int, ctypes.POINTER(Panel), c_int]
            L.zo_subspace_refresh.restype = c_int
            L.zo_subspace_refresh.argtypes = [c_int, ctypes.POINTER(Panel), c_int, c_vp, c_vp, c_sz, c_vp]
            L.zo_subspace_refresh_noalloc.restype = c_int
            L.zo_subspace_refresh_noalloc.argtypes = [c_int, ctypes.POINTER(Panel), c_int, c_vp, c_vp]
            L.zo_perturbed_linear_workspace.restype = c_sz
            L.zo_perturbed_linear_workspace.argtypes = [c_int] * 6 + [c_ll, c_int]
            L.zo_perturbed_linear.restype = c_int
            L.zo_perturbed_linear.argtypes = ([c_int] * 6 + [ctypes.POINTER(ctypes.c_int),
                                               ctypes.POINTER(ctypes.c_int8), c_f, c_int, c_vp, c_ll,
                                               c_vp, c_vp, c_vp, c_vp, c_int, c_vp, c_vp, c_sz, c_vp])
            L.zo_perturbed_linear_prepare.restype = c_int
            L.zo_perturbed_linear_prepare.argtypes = ([c_int] * 6 + [ctypes.POINTER(ctypes.c_int),
                                                       ctypes.POINTER(ctypes.c_int8), c_f, c_int, c_vp,
                                                       c_ll, c_vp, c_vp, c_vp, c_vp, c_sz, c_vp])
            L.zo_perturbed_linear_apply.restype = c_int
            L.zo_perturbed_linear_apply.argtypes = [c_int] * 7 + [c_vp, c_ll, c_vp, c_int, c_vp, c_vp, c_sz,
                                                                  c_vp]
            L.zo_lora_perturbed_linear_workspace.restype = c_sz
            L.zo_lora_perturbed_linear_workspace.argtypes = [c_int] * 7 + [c_ll, c_int]
            L.zo_lora_perturbed_linear.restype = c_int
            L.zo_lora_perturbed_linear.argtypes = ([c_int] * 7 + [ctypes.POINTER(ctypes.c_int),
                                                    ctypes.POINTER(ctypes.c_int8), c_f, c_f, c_int, c_vp,
                                                    c_ll, c_vp] + [c_vp] * 8 + [c_int, c_vp, c_vp, c_sz, c_vp])
            L.zo_lora_perturbed_linear_prepare.restype = c_int
            L.zo_lora_perturbed_linear_prepare.argtypes = ([c_int] * 7 + [ctypes.POINTER(ctypes.c_int),
                                                            ctypes.POINTER(ctypes.c_int8), c_f, c_f, c_int,
                                                            c_vp, c_ll] + [c_vp] * 8 + [c_vp, c_sz, c_vp])
            L.zo_subspace_adam_update_workspace.restype = c_sz
            L.zo_subspace_adam_update_workspace.argtypes = [c_int, ctypes.POINTER(UpdateItem), c_int,
                                                            c_int, c_int]
            L.zo_subspace_adam_update.restype = c_int
            L.zo_subspace_adam_update.argtypes = [c_int, ctypes.POINTER(UpdateItem), c_int, c_int, c_int,
                                                  c_vp, c_int, c_f, c_f, c_f, c_f, c_vp, c_vp, c_sz, c_vp]
            L.zo_subspace_sgd_update_workspace.restype = c_sz
            L.zo_subspace_sgd_update_workspace.argtypes = [c_int, ctypes.POINTER(UpdateItem), c_int,
                                                           c_int, c_int]
            L.zo_subspace_sgd_update.restype = c_int
            L.zo_subspace_sgd_update.argtypes = [c_int, ctypes.POINTER(UpdateItem), c_int, c_int, c_int,
                                                 c_vp, c_f, c_vp, c_vp, c_sz, c_vp]
            L.zo_sq_loss_workspace.restype = c_sz
            L.zo_sq_loss_workspace.argtypes = [c_int, c_int, c_int]
            L.zo_sq_loss.restype = c_int
            L.zo_sq_loss.argtypes = [c_int, c_int, c_int, c_int, c_vp, c_vp, c_vp, c_vp, c_sz, c_vp]
            L.zo_combine_central.restype = c_int
            L.zo_combine_central.argtypes = [c_int, c_vp, c_f, c_vp, c_vp]
            L.zo_combine_forward.restype = c_int
            L.zo_combine_forward.argtypes = [c_int, c_vp, c_f, c_vp, c_vp]
            L.zo_perturbed_linear_apply_ex.restype = c_int
            L.zo_perturbed_linear_apply_ex.argtypes = ([c_int] * 7 + [c_vp, c_ll, c_vp, c_int, c_vp, c_int, c_vp,
                                                                      c_ll, c_vp, c_sz, c_vp])
            L.zo_layernorm.restype = c_int
            L.zo_layernorm.argtypes = [c_ll, c_int, c_int, c_vp, c_vp, c_vp, c_f, c_vp, c_vp]
            L.zo_causal_attention.restype = c_int
            L.zo_causal_attention.argtypes = [c_int] * 6 + [c_vp] * 5
            L.zo_decoder_layer_workspace.restype = c_sz
            L.zo_decoder_layer_workspace.argtypes = [c_int] * 9
            L.zo_decoder_layer_forward.restype = c_int
            L.zo_decoder_layer_forward.argtypes = ([c_int] * 8 + [ctypes.POINTER(ctypes.c_int),
                                                                  ctypes.POINTER(ctypes.c_int8), c_f, c_f, c_int,
                                                                  c_vp, c_ll, ctypes.POINTER(DecoderLayerDesc),
                                                                  c_vp, c_vp, c_sz, c_vp])
            L.zo_rmsnorm.restype = c_int
            L.zo_rmsnorm.argtypes = [c_ll, c_int, c_int, c_vp, c_vp, c_f, c_vp, c_vp]
            L.zo_rope.restype = c_int
            L.zo_rope.argtypes = [c_ll, c_int, c_int, c_int, c_int, c_vp, c_f, c_vp]
            L.zo_llama_layer_workspace.restype = c_sz
            L.zo_llama_layer_workspace.argtypes = [c_int] * 9
            L.zo_llama_layer_forward.restype = c_int
            L.zo_llama_layer_forward.argtypes = ([c_int] * 8 + [ctypes.POINTER(ctypes.c_int),
                                                                ctypes.POINTER(ctypes.c_int8), c_f, c_f, c_f, c_int,
                                                                c_vp, c_ll, ctypes.POINTER(LlamaLayerDesc),
                                                                c_vp, c_vp, c_sz, c_vp])
            L.zo_perturbed_linear_group_workspace.restype = c_sz
            L.zo_perturbed_linear_group_workspace.argtypes = [c_int] * 6 + [c_ll, c_int]
            L.zo_perturbed_linear_prepare_group.restype = c_int
            L.zo_perturbed_linear_prepare_group.argtypes = [c_int, ctypes.POINTER(c_int)] + [c_int] * 5 + [
                ctypes.POINTER(c_int), ctypes.POINTER(ctypes.c_int8), c_f, c_int, c_vp, c_ll] + [
                ctypes.POINTER(c_vp)] * 4 + [ctypes.POINTER(c_sz), c_vp, c_sz, c_vp]
            L.zo_causal_attention_gqa.restype = c_int
            L.zo_causal_attention_gqa.argtypes = [c_int] * 7 + [c_vp] * 5
            L.zo_llama_lora_layer_workspace.restype = c_sz
            L.zo_llama_lora_layer_workspace.argtypes = [c_int] * 11
            L.zo_llama_lora_layer_forward.restype = c_int
            L.zo_llama_lora_layer_forward.argtypes = ([c_int] * 10 + [ctypes.POINTER(ctypes.c_int),
                                                                      ctypes.POINTER(ctypes.c_int8), c_f, c_f, c_f,
                                                                      c_f, c_int, c_vp, c_ll,
                                                                      ctypes.POINTER(LlamaLoraLayerDesc), c_vp, c_vp,
                                                                      c_sz, c_vp])
            _lib = L
    return _lib


def _check(status: int) -> None:
    if status != 0:
        raise ZoError(status, lib().zo_last_error_detail().decode())


def _stream_handle() -> int:
    return torch.cuda.current_stream().cuda_stream


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _need(t: torch.Tensor, name: str, dtype=None, numel=None) -> torch.Tensor:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must live on the GPU (got {t.device})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} must hold {numel} elements (got {t.numel()})")
    return t


_DT = {torch.float32: ZO_F32, torch.bfloat16: ZO_BF16, torch.float16: ZO_F16}


class Workspace:
    """Grow-only device scratch buffer, one per (device, stream).

    Calls enqueued on one stream run in order, so reusing one buffer between
    them is safe; calls on different streams get different buffers.
    """
    _bufs: dict = {}

    @classmethod
    def get(cls, nbytes: int) -> torch.Tensor:
        dev = torch.cuda.current_device()
        key = (dev, _stream_handle())
        buf = cls._bufs.get(key)
        if buf is None or buf.numel() < nbytes:
            buf = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=f"cuda:{dev}")
            cls._bufs[key] = buf
        return buf

    @classmethod
    def clear(cls):
        cls._bufs.clear()


# ---------------------------------------------------------------------------
def abi_version() -> int:
    return lib().zo_abi_version()


def subspace_refresh(omegas: Sequence[torch.Tensor], r: int, out: Optional[Sequence[torch.Tensor]] = None,
                     r_diag: Optional[Sequence[torch.Tensor]] = None, info: Optional[torch.Tensor] = None):
    """Haar factors Q_p of the Gaussian panels Omega_p (rows_p x r, fp32).  See zo_subspace_refresh."""
    n = len(omegas)
    if out is None:
        out = [torch.empty_like(o) for o in omegas]
    arr = (Panel * max(n, 1))()
    for p, om in enumerate(omegas):
        _need(om, f"omega[{p}]", torch.float32)
        if om.dim() != 2 or om.shape[1] != r:
            raise ValueError(f"omega[{p}] must be rows x {r}")
        _need(out[p], f"out[{p}]", torch.float32, om.numel())
        rd = None
        if r_diag is not None:
            rd = _need(r_diag[p], f"r_diag[{p}]", torch.float32, r)
        arr[p] = Panel(int(om.shape[0]), om.data_ptr(), out[p].data_ptr(), _ptr(rd))
    if info is not None:
        _need(info, "info", torch.int32, n)
    L = lib()
    ws_n = L.zo_subspace_refresh_workspace(n, arr, r)
    if ws_n == 0 and n > 0:
        _check(L.zo_subspace_refresh(n, arr, r, None, None, 0, None))  # raises with the reason
    ws = Workspace.get(ws_n)
    _check(L.zo_subspace_refresh(n, arr, r, _ptr(info), ws.data_ptr(), ws.numel(), _stream_handle()))
    return out


def subspace_refresh_noalloc(omegas: Sequence[torch.Tensor], r: int, out: Sequence[torch.Tensor],
                             r_diag: Optional[Sequence[torch.Tensor]] = None,
                             info: Optional[torch.Tensor] = None):
    """subspace_refresh through zo_subspace_refresh_noalloc: the library's static per-GPU scratch
    instead of a workspace, so nothing is allocated here either (out is required)."""
    n = len(omegas)
    arr = (Panel * max(n, 1))()
    for p, om in enumerate(omegas):
        _need(om, f"omega[{p}]", torch.float32)
        if om.dim() != 2 or om.shape[1] != r:
            raise ValueError(f"omega[{p}] must be rows x {r}")
        _need(out[p], f"out[{p}]", torch.float32, om.numel())
        rd = None
        if r_diag is not None:
            rd = _need(r_diag[p], f"r_diag[{p}]", torch.float32, r)
        arr[p] = Panel(int(om.shape[0]), om.data_ptr(), out[p].data_ptr(), _ptr(rd))
    if info is not None:
        _need(info, "info", torch.int32, n)
    _check(lib().zo_subspace_refresh_noalloc(n, arr, r, _ptr(info), _stream_handle()))
    return out


class PerturbedLinear:
    """One perturbed-linear problem (shapes, blocks, eps) with its arguments checked once.

    __call__ runs prepare + apply; prepare()/apply() run the two phases
    separately (same workspace, same stream, in that order).
    """

    def __init__(self, X: torch.Tensor, W: torch.Tensor, U: torch.Tensor, V: torch.Tensor, Z: torch.Tensor,
                 blk_query: Sequence[int], blk_sign: Sequence[int], eps: float, T: int,
                 x_block_stride: Optional[int] = None, out_dtype=None, Y: Optional[torch.Tensor] = None,
                 workspace: Optional[torch.Tensor] = None):
        nblk = len(blk_query)
        if len(blk_sign) != nblk:
            raise ValueError("blk_query and blk_sign differ in length")
        m, n = W.shape
        r = U.shape[1]
        q = Z.shape[0]
        dt = W.dtype
        if dt not in _DT:
            raise TypeError(f"unsupported dtype {dt}")
        _need(W, "W", dt)
        _need(X, "X", dt)
        if x_block_stride is None:
            x_block_stride = 0 if X.numel() == T * n else T * n
        if X.numel() < (T * n if x_block_stride == 0 else x_block_stride * (nblk - 1) + T * n):
            raise ValueError("X is too small for the block layout")
        _need(U, "U", torch.float32, m * r)
        _need(V, "V", torch.float32, n * r)
        _need(Z, "Z", torch.float32, q * r * r)
        out_dtype = dt if out_dtype is None else out_dtype
        if Y is None:
            Y = torch.empty((nblk * T, m), dtype=out_dtype, device=W.device)
        _need(Y, "Y", out_dtype, nblk * T * m)
        self.dims = (T, m, n, r, q, nblk)
        self.bq = (ctypes.c_int * nblk)(*[int(v) for v in blk_query])
        self.bs = (ctypes.c_int8 * nblk)(*[int(v) for v in blk_sign])
        self.eps = float(eps)
        self.dt, self.odt = _DT[dt], _DT[out_dtype]
        self.xs = int(x_block_stride)
        self.X, self.W, self.U, self.V, self.Z, self.Y = X, W, U, V, Z, Y
        need = lib().zo_perturbed_linear_workspace(T, m, n, r, q, nblk, self.xs, self.dt)
        if workspace is None:
            workspace = Workspace.get(need)
        _need(workspace, "workspace", torch.uint8)
        if workspace.numel() < need:
            raise ValueError(f"workspace holds {workspace.numel()} bytes, {need} needed")
        self.ws = workspace

    def prepare(self):
        _check(lib().zo_perturbed_linear_prepare(*self.dims, self.bq, self.bs, self.eps, self.dt, self.X.data_ptr(),
                                                 self.xs, self.U.data_ptr(), self.V.data_ptr(), self.Z.data_ptr(),
                                                 self.ws.data_ptr(), self.ws.numel(), _stream_handle()))

    def apply(self, epilogue: int = ZO_EPI_NONE, R: Optional[torch.Tensor] = None,
              r_block_stride: Optional[int] = None):
        """The fused GEMM (zo_perturbed_linear_apply_ex): epilogue ZO_EPI_RELU, ZO_EPI_RESIDUAL
        adding R, or ZO_EPI_SILU_MUL multiplying by silu(R) (R in Y's type; one T x m block shared
        by all blocks, or nblk blocks)."""
        T, m = self.dims[0], self.dims[1]
        nblk = self.dims[5]
        rs = 0
        if epilogue in (ZO_EPI_RESIDUAL, ZO_EPI_SILU_MUL):
            _need(R, "R", self.Y.dtype)
            rs = r_block_stride if r_block_stride is not None else (0 if R.numel() == T * m else T * m)
            if R.numel() < (T * m if rs == 0 else rs * (nblk - 1) + T * m):
                raise ValueError("R is too small for the block layout")
        _check(lib().zo_perturbed_linear_apply_ex(*self.dims, self.dt, self.X.data_ptr(), self.xs, self.W.data_ptr(),
                                                  self.odt, self.Y.data_ptr(), int(epilogue), _ptr(R), int(rs),
                                                  self.ws.data_ptr(), self.ws.numel(), _stream_handle()))
        return self.Y

    def __call__(self):
        _check(lib().zo_perturbed_linear(*self.dims, self.bq, self.bs, self.eps, self.dt, self.X.data_ptr(), self.xs,
                                         self.W.data_ptr(), self.U.data_ptr(), self.V.data_ptr(), self.Z.data_ptr(),
                                         self.odt, self.Y.data_ptr(), self.ws.data_ptr(), self.ws.numel(),
                                         _stream_handle()))
        return self.Y


def prepare_group(plins: Sequence["PerturbedLinear"], group_ws: Optional[torch.Tensor] = None):
    """zo_perturbed_linear_prepare_group for PerturbedLinear objects that read the same X (a
    layer's q, k, v): one projection pass for all of them, each keeping its own workspace."""
    p0 = plins[0]
    T, n, r, q, nblk = p0.dims[0], p0.dims[2], p0.dims[3], p0.dims[4], p0.dims[5]
    for p in plins:
        if (p.dims[0], p.dims[2], p.dims[3], p.dims[4], p.dims[5]) != (T, n, r, q, nblk) or p.dt != p0.dt \
                or p.X.data_ptr() != p0.X.data_ptr() or p.xs != p0.xs:
            raise ValueError("prepare_group: the linears must share T, n, r, q, nblk, dtype and X")
        if list(p.bq) != list(p0.bq) or list(p.bs) != list(p0.bs) or p.eps != p0.eps:
            raise ValueError("prepare_group: the linears must share their blocks and eps")
    cnt = len(plins)
    need = lib().zo_perturbed_linear_group_workspace(cnt, T, n, r, q, nblk, p0.xs, p0.dt)
    if need and group_ws is None:
        group_ws = torch.empty(need, dtype=torch.uint8, device=p0.X.device)
    if need and group_ws.numel() < need:
        raise ValueError(f"group workspace holds {group_ws.numel()} bytes, {need} needed")
    arr = lambda vals: (ctypes.c_void_p * cnt)(*vals)
    _check(lib().zo_perturbed_linear_prepare_group(
        cnt, (ctypes.c_int * cnt)(*[p.dims[1] for p in plins]), T, n, r, q, nblk, p0.bq, p0.bs, p0.eps, p0.dt,
        p0.X.data_ptr(), p0.xs, arr([p.U.data_ptr() for p in plins]), arr([p.V.data_ptr() for p in plins]),
        arr([p.Z.data_ptr() for p in plins]), arr([p.ws.data_ptr() for p in plins]),
        (ctypes.c_size_t * cnt)(*[p.ws.numel() for p in plins]), group_ws.data_ptr() if need else None,
        group_ws.numel() if need else 0, _stream_handle()))
    return group_ws


def perturbed_linear(X: torch.Tensor, W: torch.Tensor, U: torch.Tensor, V: torch.Tensor, Z: torch.Tensor,
                     blk_query: Sequence[int], blk_sign: Sequence[int], eps: float, T: int,
                     x_block_stride: Optional[int] = None, out_dtype=None, Y: Optional[torch.Tensor] = None):
    """Y_b = X_b (W + s_b eps U Z_{j(b)} V^T)^T for every block b.  See zo_perturbed_linear.

    X holds the stacked blocks (nblk*T x n), or a single T x n block shared by
    all blocks (x_block_stride = 0).  Returns Y (nblk*T x m).
    """
    return PerturbedLinear(X, W, U, V, Z, blk_query, blk_sign, eps, T, x_block_stride, out_dtype, Y)()


def layernorm(X: torch.Tensor, gamma: torch.Tensor, beta: torch.Tensor, eps_ln: float = 1e-5,
              out: Optional[torch.Tensor] = None):
    """Row-wise layer normalisation of X (rows x d).  See zo_layernorm."""
    d = X.shape[-1]
    _need(X, "X", X.dtype)
    if X.dtype not in _DT:
        raise TypeError(f"unsupported dtype {X.dtype}")
    _need(gamma, "gamma", torch.float32, d)
    _need(beta, "beta", torch.float32, d)
    if out is None:
        out = torch.empty_like(X)
    _need(out, "out", X.dtype, X.numel())
    _check(lib().zo_layernorm(X.numel() // d, d, _DT[X.dtype], X.data_ptr(), gamma.data_ptr(), beta.data_ptr(),
                              float(eps_ln), out.data_ptr(), _stream_handle()))
    return out


def rmsnorm(X: torch.Tensor, gamma: torch.Tensor, eps: float = 1e-6, out: Optional[torch.Tensor] = None):
    """Row-wise RMS normalisation of X (rows x d).  See zo_rmsnorm."""
    d = X.shape[-1]
    _need(X, "X", X.dtype)
    if X.dtype not in _DT:
        raise TypeError(f"unsupported dtype {X.dtype}")
    _need(gamma, "gamma", torch.float32, d)
    if out is None:
        out = torch.empty_like(X)
    _need(out, "out", X.dtype, X.numel())
    _check(lib().zo_rmsnorm(X.numel() // d, d, _DT[X.dtype], X.data_ptr(), gamma.data_ptr(), float(eps),
                            out.data_ptr(), _stream_handle()))
    return out


def rope(X: torch.Tensor, seq_len: int, heads: int, base: float = 10000.0):
    """Rotary position embedding of X (rows x d, sequences of seq_len rows), in place.
    See zo_rope."""
    d = X.shape[-1]
    _need(X, "X", X.dtype)
    if X.dtype not in _DT:
        raise TypeError(f"unsupported dtype {X.dtype}")
    _check(lib().zo_rope(X.numel() // d, seq_len, d, heads, _DT[X.dtype], X.data_ptr(), float(base),
                         _stream_handle()))
    return X


def causal_attention(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, nblk: int, T: int, seq_len: int,
                     heads: int, out: Optional[torch.Tensor] = None, kv_heads: Optional[int] = None):
    """Multi-head causal self-attention of nblk blocks of T rows (T / seq_len sequences each);
    with kv_heads, K and V hold kv_heads grouped key/value heads.  See zo_causal_attention(_gqa)."""
    d = Q.shape[-1]
    if Q.dtype not in _DT:
        raise TypeError(f"unsupported dtype {Q.dtype}")
    dkv = d if kv_heads is None else d // heads * kv_heads
    _need(Q, "Q", Q.dtype, nblk * T * d)
    for nm, t in (("K", K), ("V", V)):
        _need(t, nm, Q.dtype, nblk * T * dkv)
    if out is None:
        out = torch.empty_like(Q)
    _need(out, "out", Q.dtype, nblk * T * d)
    if kv_heads is None:
        _check(lib().zo_causal_attention(nblk, T, seq_len, d, heads, _DT[Q.dtype], Q.data_ptr(), K.data_ptr(),
                                         V.data_ptr(), out.data_ptr(), _stream_handle()))
    else:
        _check(lib().zo_causal_attention_gqa(nblk, T, seq_len, d, heads, kv_heads, _DT[Q.dtype], Q.data_ptr(),
                                             K.data_ptr(), V.data_ptr(), out.data_ptr(), _stream_handle()))
    return out


class DecoderLayer:
    """A pre-LN decoder layer whose six matrices are perturbed per block.  See
    zo_decoder_layer_forward.  ``mats`` maps q, k, v, o, fc1, fc2 to dicts with W (the
    layer's dtype), U, V, Z (fp32); ``ln`` holds ln1_gamma, ln1_beta, ln2_gamma, ln2_beta."""

    NAMES = ("q", "k", "v", "o", "fc1", "fc2")

    def __init__(self, mats: dict, ln: dict, blk_query: Sequence[int], blk_sign: Sequence[int], eps: float,
                 T: int, seq_len: int, heads: int, eps_ln: float = 1e-5, workspace: Optional[torch.Tensor] = None):
        nblk = len(blk_query)
        if len(blk_sign) != nblk:
            raise ValueError("blk_query and blk_sign differ in length")
        Wq = mats["q"]["W"]
        d = Wq.shape[0]
        ffn = mats["fc1"]["W"].shape[0]
        r = mats["q"]["U"].shape[1]
        q = mats["q"]["Z"].shape[0]
        dt = Wq.dtype
        if dt not in _DT:
            raise TypeError(f"unsupported dtype {dt}")
        shapes = {"q": (d, d), "k": (d, d), "v": (d, d), "o": (d, d), "fc1": (ffn, d), "fc2": (d, ffn)}
        desc = DecoderLayerDesc()
        for nm in self.NAMES:
            m, n = shapes[nm]
            mt = mats[nm]
            _need(mt["W"], f"{nm}.W", dt, m * n)
            _need(mt["U"], f"{nm}.U", torch.float32, m * r)
            _need(mt["V"], f"{nm}.V", torch.float32, n * r)
            _need(mt["Z"], f"{nm}.Z", torch.float32, q * r * r)
            setattr(desc, nm, Matrix(mt["W"].data_ptr(), mt["U"].data_ptr(), mt["V"].data_ptr(), mt["Z"].data_ptr()))
        for nm in ("ln1_gamma", "ln1_beta", "ln2_gamma", "ln2_beta"):
            _need(ln[nm], nm, torch.float32, d)
            setattr(desc, nm, ln[nm].data_ptr())
        self.desc, self.keep = desc, (mats, ln)
        self.dims = (T, seq_len, d, heads, ffn, r, q, nblk)
        self.bq = (ctypes.c_int * nblk)(*[int(v) for v in blk_query])
        self.bs = (ctypes.c_int8 * nblk)(*[int(v) for v in blk_sign])
        self.eps, self.eps_ln, self.dt, self.dtype = float(eps), float(eps_ln), _DT[dt], dt
        need = lib().zo_decoder_layer_workspace(*self.dims, self.dt)
        if need == 0:
            _check(lib().zo_decoder_layer_forward(*self.dims, self.bq, self.bs, self.eps, self.eps_ln, self.dt,
                                                  None, 0, ctypes.byref(self.desc), None, None, 0, None))
        if workspace is None:
            workspace = Workspace.get(need)
        _need(workspace, "workspace", torch.uint8)
        if workspace.numel() < need:
            raise ValueError(f"workspace holds {workspace.numel()} bytes, {need} needed")
        self.ws = workspace

    def __call__(self, H: torch.Tensor, out: Optional[torch.Tensor] = None):
        """H: one T x d input shared by all blocks, or nblk blocks; returns nblk blocks of T x d."""
        T, d, nblk = self.dims[0], self.dims[2], self.dims[7]
        _need(H, "H", self.dtype)
        if H.numel() == T * d:
            hs = 0
        elif H.numel() == nblk * T * d:
            hs = T * d
        else:
            raise ValueError("H must hold T*d or nblk*T*d elements")
        if out is None:
            out = torch.empty((nblk * T, d), dtype=self.dtype, device=H.device)
        _need(out, "out", self.dtype, nblk * T * d)
        _check(lib().zo_decoder_layer_forward(*self.dims, self.bq, self.bs, self.eps, self.eps_ln, self.dt,
                                              H.data_ptr(), hs, ctypes.byref(self.desc), out.data_ptr(),
                                              self.ws.data_ptr(), self.ws.numel(), _stream_handle()))
        return out


class LlamaLayer:
    """A LLaMA-family decoder layer (RMS norms, rotary positions, SwiGLU MLP) whose seven
    matrices are perturbed per block.  See zo_llama_layer_forward.  ``mats`` maps q, k, v, o,
    gate, up, down to dicts with W (the layer's dtype), U, V, Z (fp32); ``norms`` holds
    rms1_gamma and rms2_gamma."""

    NAMES = ("q", "k", "v", "o", "gate", "up", "down")

    def __init__(self, mats: dict, norms: dict, blk_query: Sequence[int], blk_sign: Sequence[int], eps: float,
                 T: int, seq_len: int, heads: int, eps_rms: float = 1e-6, rope_base: float = 10000.0,
                 workspace: Optional[torch.Tensor] = None):
        nblk = len(blk_query)
        if len(blk_sign) != nblk:
            raise ValueError("blk_query and blk_sign differ in length")
        Wq = mats["q"]["W"]
        d = Wq.shape[0]
        ffn = mats["gate"]["W"].shape[0]
        r = mats["q"]["U"].shape[1]
        q = mats["q"]["Z"].shape[0]
        dt = Wq.dtype
        if dt not in _DT:
            raise TypeError(f"unsupported dtype {dt}")
        shapes = {"q": (d, d), "k": (d, d), "v": (d, d), "o": (d, d), "gate": (ffn, d), "up": (ffn, d),
                  "down": (d, ffn)}
        desc = LlamaLayerDesc()
        for nm in self.NAMES:
            m, n = shapes[nm]
            mt = mats[nm]
            _need(mt["W"], f"{nm}.W", dt, m * n)
            _need(mt["U"], f"{nm}.U", torch.float32, m * r)
            _need(mt["V"], f"{nm}.V", torch.float32, n * r)
            _need(mt["Z"], f"{nm}.Z", torch.float32, q * r * r)
            setattr(desc, nm, Matrix(mt["W"].data_ptr(), mt["U"].data_ptr(), mt["V"].data_ptr(), mt["Z"].data_ptr()))
        for nm in ("rms1_gamma", "rms2_gamma"):
            _need(norms[nm], nm, torch.float32, d)
            setattr(desc, nm, norms[nm].data_ptr())
        self.desc, self.keep = desc, (mats, norms)
        self.dims = (T, seq_len, d, heads, ffn, r, q, nblk)
        self.bq = (ctypes.c_int * nblk)(*[int(v) for v in blk_query])
        self.bs = (ctypes.c_int8 * nblk)(*[int(v) for v in blk_sign])
        self.eps, self.eps_rms, self.base = float(eps), float(eps_rms), float(rope_base)
        self.dt, self.dtype = _DT[dt], dt
        need = lib().zo_llama_layer_workspace(*self.dims, self.dt)
        if need == 0:
            _check(lib().zo_llama_layer_forward(*self.dims, self.bq, self.bs, self.eps, self.eps_rms, self.base,
                                                self.dt, None, 0, ctypes.byref(self.desc), None, None, 0, None))
        if workspace is None:
            workspace = Workspace.get(need)
        _need(workspace, "workspace", torch.uint8)
        if workspace.numel() < need:
            raise ValueError(f"workspace holds {workspace.numel()} bytes, {need} needed")
        self.ws = workspace

    def __call__(self, H: torch.Tensor, out: Optional[torch.Tensor] = None):
        """H: one T x d input shared by all blocks, or nblk blocks; returns nblk blocks of T x d."""
        T, d, nblk = self.dims[0], self.dims[2], self.dims[7]
        _need(H, "H", self.dtype)
        if H.numel() == T * d:
            hs = 0
        elif H.numel() == nblk * T * d:
            hs = T * d
        else:
            raise ValueError("H must hold T*d or nblk*T*d elements")
        if out is None:
            out = torch.empty((nblk * T, d), dtype=self.dtype, device=H.device)
        _need(out, "out", self.dtype, nblk * T * d)
        _check(lib().zo_llama_layer_forward(*self.dims, self.bq, self.bs, self.eps, self.eps_rms, self.base,
                                            self.dt, H.data_ptr(), hs, ctypes.byref(self.desc), out.data_ptr(),
                                            self.ws.data_ptr(), self.ws.numel(), _stream_handle()))
        return out


class LlamaLoraLayer:
    """The LoRA-scheme LLaMA-family layer (grouped key/value heads, frozen base, adapters on q
    and v perturbed per block).  See zo_llama_lora_layer_forward.  ``mats`` maps q and v to
    dicts with W (the layer's dtype), A, UA, VA, ZA, B, UB, VB, ZB (fp32), and k, o, gate, up,
    down to dicts with W; ``norms`` holds rms1_gamma and rms2_gamma."""

    FROZEN = ("k", "o", "gate", "up", "down")

    def __init__(self, mats: dict, norms: dict, blk_query: Sequence[int], blk_sign: Sequence[int], eps: float,
                 scale: float, T: int, seq_len: int, heads: int, kv_heads: int, eps_rms: float = 1e-6,
                 rope_base: float = 1e6, workspace: Optional[torch.Tensor] = None):
        nblk = len(blk_query)
        if len(blk_sign) != nblk:
            raise ValueError("blk_query and blk_sign differ in length")
        Wq = mats["q"]["W"]
        d, dt = Wq.shape[0], Wq.dtype
        if dt not in _DT:
            raise TypeError(f"unsupported dtype {dt}")
        dkv = d // heads * kv_heads
        ffn = mats["gate"]["W"].shape[0]
        rl, r = mats["q"]["A"].shape[0], mats["q"]["UA"].shape[1]
        q = mats["q"]["ZA"].shape[0]
        desc = LlamaLoraLayerDesc()
        for nm, m in (("q", d), ("v", dkv)):
            mt = mats[nm]
            _need(mt["W"], f"{nm}.W", dt, m * d)
            for key, numel in (("A", rl * d), ("UA", rl * r), ("VA", d * r), ("ZA", q * r * r), ("B", m * rl),
                               ("UB", m * r), ("VB", rl * r), ("ZB", q * r * r)):
                _need(mt[key], f"{nm}.{key}", torch.float32, numel)
            setattr(desc, nm, LoraMatrix(*[mt[k].data_ptr() for k in ("W", "A", "UA", "VA", "ZA", "B", "UB", "VB",
                                                                      "ZB")]))
        shapes = {"k": (dkv, d), "o": (d, d), "gate": (ffn, d), "up": (ffn, d), "down": (d, ffn)}
        for nm in self.FROZEN:
            m, n = shapes[nm]
            _need(mats[nm]["W"], f"{nm}.W", dt, m * n)
            setattr(desc, nm, mats[nm]["W"].data_ptr())
        for nm in ("rms1_gamma", "rms2_gamma"):
            _need(norms[nm], nm, torch.float32, d)
            setattr(desc, nm, norms[nm].data_ptr())
        self.desc, self.keep = desc, (mats, norms)
        self.dims = (T, seq_len, d, heads, kv_heads, ffn, rl, r, q, nblk)
        self.bq = (ctypes.c_int * nblk)(*[int(v) for v in blk_query])
        self.bs = (ctypes.c_int8 * nblk)(*[int(v) for v in blk_sign])
        self.eps, self.scale, self.eps_rms, self.base = float(eps), float(scale), float(eps_rms), float(rope_base)
        self.dt, self.dtype = _DT[dt], dt
        need = lib().zo_llama_lora_layer_workspace(*self.dims, self.dt)
        if need == 0:
            _check(lib().zo_llama_lora_layer_forward(*self.dims, self.bq, self.bs, self.eps, self.scale, self.eps_rms,
                                                     self.base, self.dt, None, 0, ctypes.byref(self.desc), None, None,
                                                     0, None))
        if workspace is None:
            workspace = Workspace.get(need)
        _need(workspace, "workspace", torch.uint8)
        if workspace.numel() < need:
            raise ValueError(f"workspace holds {workspace.numel()} bytes, {need} needed")
        self.ws = workspace

    def __call__(self, H: torch.Tensor, out: Optional[torch.Tensor] = None):
        """H: one T x d input shared by all blocks, or nblk blocks; returns nblk blocks of T x d."""
        T, d, nblk = self.dims[0], self.dims[2], self.dims[9]
        _need(H, "H", self.dtype)
        if H.numel() == T * d:
            hs = 0
        elif H.numel() == nblk * T * d:
            hs = T * d
        else:
            raise ValueError("H must hold T*d or nblk*T*d elements")
        if out is None:
            out = torch.empty((nblk * T, d), dtype=self.dtype, device=H.device)
        _need(out, "out", self.dtype, nblk * T * d)
        _check(lib().zo_llama_lora_layer_forward(*self.dims, self.bq, self.bs, self.eps, self.scale, self.eps_rms,
                                                 self.base, self.dt, H.data_ptr(), hs, ctypes.byref(self.desc),
                                                 out.data_ptr(), self.ws.data_ptr(), self.ws.numel(),
                                                 _stream_handle()))
        return out


class LoraPerturbedLinear:
    """One perturbed LoRA-adapted layer (frozen base W, adapter A: rl x n, B: m x rl, each factor
    with its own subspace U_*, V_* and coefficients Z_*).  See zo_lora_perturbed_linear.

    __call__ runs prepare + apply; prepare()/apply() run the two phases separately (apply is
    zo_perturbed_linear_apply at rank rl + r).
    """

    def __init__(self, X: torch.Tensor, W: torch.Tensor, A: torch.Tensor, UA: torch.Tensor, VA: torch.Tensor,
                 ZA: torch.Tensor, B: torch.Tensor, UB: torch.Tensor, VB: torch.Tensor, ZB: torch.Tensor,
                 blk_query: Sequence[int], blk_sign: Sequence[int], eps: float, scale: float, T: int,
                 x_block_stride: Optional[int] = None, out_dtype=None, Y: Optional[torch.Tensor] = None,
                 workspace: Optional[torch.Tensor] = None):
        nblk = len(blk_query)
        if len(blk_sign) != nblk:
            raise ValueError("blk_query and blk_sign differ in length")
        m, n = W.shape
        rl = A.shape[0]
        r = UA.shape[1]
        q = ZA.shape[0]
        dt = W.dtype
        if dt not in _DT:
            raise TypeError(f"unsupported dtype {dt}")
        _need(W, "W", dt)
        _need(X, "X", dt)
        if x_block_stride is None:
            x_block_stride = 0 if X.numel() == T * n else T * n
        if X.numel() < (T * n if x_block_stride == 0 else x_block_stride * (nblk - 1) + T * n):
            raise ValueError("X is too small for the block layout")
        _need(A, "A", torch.float32, rl * n)
        _need(B, "B", torch.float32, m * rl)
        _need(UA, "U_A", torch.float32, rl * r)
        _need(VA, "V_A", torch.float32, n * r)
        _need(UB, "U_B", torch.float32, m * r)
        _need(VB, "V_B", torch.float32, rl * r)
        _need(ZA, "Z_A", torch.float32, q * r * r)
        _need(ZB, "Z_B", torch.float32, q * r * r)
        out_dtype = dt if out_dtype is None else out_dtype
        if Y is None:
            Y = torch.empty((nblk * T, m), dtype=out_dtype, device=W.device)
        _need(Y, "Y", out_dtype, nblk * T * m)
        self.T, self.m, self.n, self.rl, self.r, self.q, self.nblk = T, m, n, rl, r, q, nblk
        self.bq = (ctypes.c_int * nblk)(*[int(v) for v in blk_query])
        self.bs = (ctypes.c_int8 * nblk)(*[int(v) for v in blk_sign])
        self.eps, self.scale = float(eps), float(scale)
        self.dt, self.odt = _DT[dt], _DT[out_dtype]
        self.xs = int(x_block_stride)
        self.X, self.W, self.Y = X, W, Y
        self.factors = (A, UA, VA, ZA, B, UB, VB, ZB)
        need = lib().zo_lora_perturbed_linear_workspace(T, m, n, rl, r, q, nblk, self.xs, self.dt)
        if workspace is None:
            workspace = Workspace.get(need)
        _need(workspace, "workspace", torch.uint8)
        if workspace.numel() < need:
            raise ValueError(f"workspace holds {workspace.numel()} bytes, {need} needed")
        self.ws = workspace

    def _dims(self):
        return (self.T, self.m, self.n, self.rl, self.r, self.q, self.nblk)

    def prepare(self):
        _check(lib().zo_lora_perturbed_linear_prepare(
            *self._dims(), self.bq, self.bs, self.eps, self.scale, self.dt, self.X.data_ptr(), self.xs,
            *[f.data_ptr() for f in self.factors], self.ws.data_ptr(), self.ws.numel(), _stream_handle()))

    def apply(self):
        _check(lib().zo_perturbed_linear_apply(
            self.T, self.m, self.n, self.rl + self.r, self.q, self.nblk, self.dt, self.X.data_ptr(), self.xs,
            self.W.data_ptr(), self.odt, self.Y.data_ptr(), self.ws.data_ptr(), self.ws.numel(), _stream_handle()))
        return self.Y

    def __call__(self):
        _check(lib().zo_lora_perturbed_linear(
            *self._dims(), self.bq, self.bs, self.eps, self.scale, self.dt, self.X.data_ptr(), self.xs,
            self.W.data_ptr(), *[f.data_ptr() for f in self.factors], self.odt, self.Y.data_ptr(),
            self.ws.data_ptr(), self.ws.numel(), _stream_handle()))
        return self.Y


def lora_perturbed_linear(X, W, A, UA, VA, ZA, B, UB, VB, ZB, blk_query, blk_sign, eps, scale, T,
                          x_block_stride=None, out_dtype=None, Y=None):
    """Y_b = X_b (W + scale B'_b A'_b)^T for every block b.  See zo_lora_perturbed_linear."""
    return LoraPerturbedLinear(X, W, A, UA, VA, ZA, B, UB, VB, ZB, blk_query, blk_sign, eps, scale, T,
                               x_block_stride, out_dtype, Y)()


def _update_items(items: Sequence[dict], g: torch.Tensor, moments: bool):
    n = len(items)
    dt = items[0]["W"].dtype
    if dt not in _DT:
        raise TypeError(f"unsupported dtype {dt}")
    r = items[0]["U"].shape[1]
    q = items[0]["Z"].shape[0]
    _need(g, "g", torch.float32, q)
    arr = (UpdateItem * n)()
    for i, it in enumerate(items):
        W = _need(it["W"], f"W[{i}]", dt)
        m, nn = W.shape
        _need(it["U"], f"U[{i}]", torch.float32, m * r)
        _need(it["V"], f"V[{i}]", torch.float32, nn * r)
        _need(it["Z"], f"Z[{i}]", torch.float32, q * r * r)
        m1, m2 = it.get("M1"), it.get("M2")
        if moments or m1 is not None:
            _need(m1, f"M1[{i}]", torch.float32, r * r)
        if moments or m2 is not None:
            _need(m2, f"M2[{i}]", torch.float32, r * r)
        zb = it.get("zbar_out")
        wo = it.get("w_f32_out")
        if zb is not None:
            _need(zb, f"zbar_out[{i}]", torch.float32, r * r)
        if wo is not None:
            _need(wo, f"w_f32_out[{i}]", torch.float32, m * nn)
        arr[i] = UpdateItem(m, nn, W.data_ptr(), it["U"].data_ptr(), it["V"].data_ptr(), it["Z"].data_ptr(),
                            _ptr(m1), _ptr(m2), _ptr(zb), _ptr(wo))
    return arr, _DT[dt], r, q


def subspace_adam_update(items: Sequence[dict], g: torch.Tensor, t: int, lr: float, beta1: float,
                         beta2: float, eps_adam: float, nonfinite_flag: Optional[torch.Tensor] = None):
    """Subspace Adam step for every item (dict with W, U, V, Z, M1, M2 and optional
    zbar_out, w_f32_out).  See zo_subspace_adam_update."""
    n = len(items)
    if n == 0:
        return
    arr, dt, r, q = _update_items(items, g, True)
    if nonfinite_flag is not None:
        _need(nonfinite_flag, "nonfinite_flag", torch.int32, 1)
    L = lib()
    ws_n = L.zo_subspace_adam_update_workspace(n, arr, r, q, dt)
    if ws_n == 0:  # the arguments failed validation: the call (which launches nothing) says why
        _check(L.zo_subspace_adam_update(n, arr, dt, r, q, g.data_ptr(), t, lr, beta1, beta2,
                                         eps_adam, None, None, 0, None))
        return
    ws = Workspace.get(ws_n)
    _check(L.zo_subspace_adam_update(n, arr, dt, r, q, g.data_ptr(), int(t), float(lr), float(beta1),
                                     float(beta2), float(eps_adam), _ptr(nonfinite_flag), ws.data_ptr(),
                                     ws.numel(), _stream_handle()))


def subspace_sgd_update(items: Sequence[dict], g: torch.Tensor, lr: float,
                        nonfinite_flag: Optional[torch.Tensor] = None):
    """Subspace SGD step W <- W - lr U Zbar V^T for every item (dict with W, U, V, Z and optional
    zbar_out, w_f32_out; moments not used).  See zo_subspace_sgd_update."""
    n = len(items)
    if n == 0:
        return
    arr, dt, r, q = _update_items(items, g, False)
    if nonfinite_flag is not None:
        _need(nonfinite_flag, "nonfinite_flag", torch.int32, 1)
    L = lib()
    ws_n = L.zo_subspace_sgd_update_workspace(n, arr, r, q, dt)
    if ws_n == 0:  # the arguments failed validation: the call (which launches nothing) says why
        _check(L.zo_subspace_sgd_update(n, arr, dt, r, q, g.data_ptr(), lr, None, None, 0, None))
        return
    ws = Workspace.get(ws_n)
    _check(L.zo_subspace_sgd_update(n, arr, dt, r, q, g.data_ptr(), float(lr), _ptr(nonfinite_flag),
                                    ws.data_ptr(), ws.numel(), _stream_handle()))


def sq_loss(Y: torch.Tensor, Ystar: torch.Tensor, nblk: int, T: int, out: Optional[torch.Tensor] = None):
    """Per-block 0.5 ||Y_b - Y*||^2 / T as a float64 device tensor [nblk]."""
    dt = Y.dtype
    m = Ystar.shape[-1]
    _need(Y, "Y", dt, nblk * T * m)
    _need(Ystar, "Ystar", dt, T * m)
    if out is None:
        out = torch.empty(nblk, dtype=torch.float64, device=Y.device)
    _need(out, "out", torch.float64, nblk)
    L = lib()
    ws = Workspace.get(L.zo_sq_loss_workspace(nblk, T, m))
    _check(L.zo_sq_loss(nblk, T, m, _DT[dt], Y.data_ptr(), Ystar.data_ptr(), out.data_ptr(),
                        ws.data_ptr(), ws.numel(), _stream_handle()))
    return out


def combine_central(Lpm: torch.Tensor, eps: float, out: Optional[torch.Tensor] = None):
    """g_j = (L[2j] - L[2j+1]) / (2 eps) as float32 [q]."""
    _need(Lpm, "L", torch.float64)
    q = Lpm.numel() // 2
    if out is None:
        out = torch.empty(q, dtype=torch.float32, device=Lpm.device)
    _need(out, "g", torch.float32, q)
    _check(lib().zo_combine_central(q, Lpm.data_ptr(), float(eps), out.data_ptr(), _stream_handle()))
    return out


def combine_forward(L: torch.Tensor, eps: float, out: Optional[torch.Tensor] = None):
    """g_j = (L[1 + j] - L[0]) / eps as float32 [q] (L[0]: the baseline block)."""
    _need(L, "L", torch.float64)
    q = L.numel() - 1
    if out is None:
        out = torch.empty(q, dtype=torch.float32, device=L.device)
    _need(out, "g", torch.float32, q)
    _check(lib().zo_combine_forward(q, L.data_ptr(), float(eps), out.data_ptr(), _stream_handle()))
    return out
