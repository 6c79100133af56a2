"""ctypes binding of libsq.so (include/sq.h).

Argument marshalling only: tensors become device pointers, sizes become int64, the
current torch HIP stream becomes the `stream` argument.  Every step of the path runs in
the library's HIP kernels; there is no fallback.  A missing library raises.
Outputs are allocated with torch (device memory is torch's job here) unless passed in.
"""

import ctypes
import os

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsq.so")

SQ_OK, SQ_ERR_NULL, SQ_ERR_SHAPE, SQ_ERR_UNSUPPORTED, SQ_ERR_ALIGN, SQ_ERR_ALIAS, SQ_ERR_HIP = range(7)
STATUS_NAMES = {0: "SQ_OK", 1: "SQ_ERR_NULL", 2: "SQ_ERR_SHAPE", 3: "SQ_ERR_UNSUPPORTED",
                4: "SQ_ERR_ALIGN", 5: "SQ_ERR_ALIAS", 6: "SQ_ERR_HIP"}

EXPORTS = ("sq_abi_version", "sq_last_error", "sq_time_next_call", "sq_hadamard_factor", "sq_had_quant_act",
           "sq_had_quant_act_ex", "sq_pack_w4", "sq_pack_w4_ex", "sq_w4a4_linear", "sq_w4a8_linear",
           "sq_w4a4_linear_swiglu", "sq_qk_had_kvquant", "sq_qk_had_kvquant_ex", "sq_attn_decode_kv4",
           "sq_attn_decode_kv4_ex", "sq_attn_decode_workspace", "sq_attn_decode_kv4_split",
           "sq_attn_decode_kv4_split_noalloc")


class SqError(RuntimeError):
    def __init__(self, status: int, where: str, msg: str):
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


_lib = None
_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I32 = ctypes.c_int32
_F32 = ctypes.c_float


def lib() -> ctypes.CDLL:
    """Load libsq.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2405_16406_amd.build`")
    _lib = load(LIB_PATH)
    return _lib


def load(path: str) -> ctypes.CDLL:
    """Open a build of the library at `path` and declare the signatures of include/sq.h."""
    L = ctypes.CDLL(path)
    L.sq_abi_version.restype = _I32
    L.sq_abi_version.argtypes = []
    L.sq_last_error.restype = ctypes.c_char_p
    L.sq_last_error.argtypes = []
    L.sq_time_next_call.restype = _I32
    L.sq_time_next_call.argtypes = [_P, _P]
    L.sq_hadamard_factor.restype = _I32
    L.sq_hadamard_factor.argtypes = [_I32, _P]
    L.sq_had_quant_act.restype = _I32
    L.sq_had_quant_act.argtypes = [_P, _I64, _I64, _I64, _I32, _P, _I32, _I32, _I32, _P, _P, _P, _P, _P]
    L.sq_had_quant_act_ex.restype = _I32
    L.sq_had_quant_act_ex.argtypes = [_P, _I64, _I64, _I64, _I32, _P, _I32, _P, _I32, _I32, _F32,
                                      _P, _P, _P, _P, _P]
    L.sq_pack_w4.restype = _I32
    L.sq_pack_w4.argtypes = [_P, _I64, _I64, _I64, _I32, _P, _I32, _P, _P, _P, _P]
    L.sq_pack_w4_ex.restype = _I32
    L.sq_pack_w4_ex.argtypes = [_P, _I64, _I64, _I64, _I32, _P, _I32, _P, _P, _P, _P, _P]
    L.sq_w4a4_linear.restype = _I32
    L.sq_w4a4_linear.argtypes = [_P, _P, _P, _I64, _P, _P, _P, _I64, _I64, _P, _P, _I64, _P, _P]
    L.sq_w4a8_linear.restype = _I32
    L.sq_w4a8_linear.argtypes = [_P, _P, _P, _I64, _P, _P, _P, _I64, _I64, _P, _P, _I64, _P, _P]
    L.sq_w4a4_linear_swiglu.restype = _I32
    L.sq_w4a4_linear_swiglu.argtypes = [_P, _P, _P, _I64, _P, _P, _P, _I64, _I64, _P, _P, _I64, _P]
    L.sq_qk_had_kvquant.restype = _I32
    L.sq_qk_had_kvquant.argtypes = [_P, _P, _P, _I64, _I64, _I64, _I64, _I32, _I32,
                                    _P, _P, _P, _P, _P, _P, _P, _P, _P]
    L.sq_qk_had_kvquant_ex.restype = _I32
    L.sq_qk_had_kvquant_ex.argtypes = [_P, _P, _P, _I64, _I64, _I64, _I64, _I32, _I32, _F32, _F32, _I32,
                                       _P, _P, _P, _P, _P, _P, _P, _P, _P]
    L.sq_attn_decode_kv4.restype = _I32
    L.sq_attn_decode_kv4.argtypes = [_P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I64, _F32, _P, _P]
    L.sq_attn_decode_kv4_ex.restype = _I32
    L.sq_attn_decode_kv4_ex.argtypes = [_P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I64, _F32, _I32, _P, _P]
    L.sq_attn_decode_workspace.restype = _I32
    L.sq_attn_decode_workspace.argtypes = [_I64, _I64, _I64, _I64, _P]
    L.sq_attn_decode_kv4_split.restype = _I32
    L.sq_attn_decode_kv4_split.argtypes = [_P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I64, _F32, _I32, _P, _P,
                                           ctypes.c_uint64, _P]
    L.sq_attn_decode_kv4_split_noalloc.restype = _I32
    L.sq_attn_decode_kv4_split_noalloc.argtypes = [_P, _P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _I64, _F32, _I32,
                                                   _P, _P]
    return L


def _check(status: int, where: str) -> None:
    if status != SQ_OK:
        raise SqError(status, where, lib().sq_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(t: torch.Tensor):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _need(t: torch.Tensor, dtype, name: str):
    if not isinstance(t, torch.Tensor) or t.dtype != dtype or not t.is_cuda:
        raise TypeError(f"{name} must be a {dtype} tensor on the GPU")


def abi_version() -> int:
    return int(lib().sq_abi_version())


def time_next_call(start: "torch.cuda.Event", stop: "torch.cuda.Event") -> None:
    """Arm two timing events (torch.cuda.Event(enable_timing=True)) for this thread's next
    library call: start.elapsed_time(stop) is then that call's kernel time on the device."""
    for e in (start, stop):
        if e.cuda_event == 0:  # torch creates the HIP event on its first record
            e.record()
    _check(lib().sq_time_next_call(ctypes.c_void_p(start.cuda_event), ctypes.c_void_p(stop.cuda_event)),
           "sq_time_next_call")


def hadamard_factor(n: int) -> np.ndarray:
    """The library's +-1 Hadamard matrix of order n (1, 28, 172) as int8 [n, n] (host)."""
    out = np.empty((n, n), dtype=np.int8)
    _check(lib().sq_hadamard_factor(n, out.ctypes.data_as(ctypes.c_void_p)), "sq_hadamard_factor")
    return out


def had_quant_act(x: torch.Tensor, had: torch.Tensor | None = None, pow2: int = 1,
                  group: int | None = None, bits: int = 4, dbg: bool = False, out=None,
                  clip: float = 1.0, signs: torch.Tensor | None = None):
    """Rotate rows of x (fp16 [M, K], row stride x.stride(0)) and quantize (asym, 4 or 8 bits).

    had: int8 +-1 [a, a] on the device or None.  clip (range clipping ratio in (0, 1]) and
    signs (int8 +-1 [a * pow2] on the device: the random Hadamard S H) select sq_had_quant_act_ex.
    Returns (q uint8 [M, K/2] (4-bit) or [M, K] (8-bit), alpha fp32 [M, K/group],
    beta fp32 [M, K/group], dbg_rot fp32 [M, K] or None).
    """
    _need(x, torch.float16, "x")
    if x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be 2-D with unit column stride")
    M, K = x.shape
    group = K if group is None else group
    a = 1 if had is None else had.shape[0]
    if had is not None:
        _need(had, torch.int8, "had")
    dev = x.device
    if out is None:
        q = torch.empty((M, K * bits // 8), dtype=torch.uint8, device=dev)
        al = torch.empty((M, K // group), dtype=torch.float32, device=dev)
        be = torch.empty((M, K // group), dtype=torch.float32, device=dev)
    else:
        q, al, be = out
    rot = torch.empty((M, K), dtype=torch.float32, device=dev) if dbg else None
    if clip == 1.0 and signs is None:
        _check(lib().sq_had_quant_act(_ptr(x), M, K, x.stride(0), a, _ptr(had), pow2, bits, group,
                                      _ptr(q), _ptr(al), _ptr(be), _ptr(rot), _stream(x)), "sq_had_quant_act")
    else:
        if signs is not None:
            _need(signs, torch.int8, "signs")
        _check(lib().sq_had_quant_act_ex(_ptr(x), M, K, x.stride(0), a, _ptr(had), pow2, _ptr(signs), bits, group,
                                         float(clip), _ptr(q), _ptr(al), _ptr(be), _ptr(rot), _stream(x)),
               "sq_had_quant_act_ex")
    return q, al, be, rot


def pack_w4(w: torch.Tensor, had: torch.Tensor | None = None, pow2: int = 1, signs: torch.Tensor | None = None):
    """Offline: W' = W R (optional), symmetric per-row 4-bit quant, pack.

    signs (int8 +-1 [a * pow2] on the device) fold the random Hadamard S H instead
    (sq_pack_w4_ex).  Returns (wq uint8 [N, K/2], w_alpha fp32 [N], w_rowsum int32 [N]).
    """
    _need(w, torch.float16, "w")
    if w.dim() != 2 or w.stride(1) != 1:
        raise ValueError("w must be 2-D with unit column stride")
    N, K = w.shape
    a = 1 if had is None else had.shape[0]
    dev = w.device
    wq = torch.empty((N, K // 2), dtype=torch.uint8, device=dev)
    wa = torch.empty((N,), dtype=torch.float32, device=dev)
    rs = torch.empty((N,), dtype=torch.int32, device=dev)
    if signs is None:
        _check(lib().sq_pack_w4(_ptr(w), N, K, w.stride(0), a, _ptr(had), pow2, _ptr(wq), _ptr(wa), _ptr(rs),
                                _stream(w)), "sq_pack_w4")
    else:
        _need(signs, torch.int8, "signs")
        _check(lib().sq_pack_w4_ex(_ptr(w), N, K, w.stride(0), a, _ptr(had), pow2, _ptr(signs), _ptr(wq), _ptr(wa),
                                   _ptr(rs), _stream(w)), "sq_pack_w4_ex")
    return wq, wa, rs


def w4a4_linear(xq, x_alpha, x_beta, wq, w_alpha, w_rowsum, bias=None, out=None, dbg=False):
    """y = fp16(s_n (alpha_m acc + beta_m rowsum_n) + bias_n) with acc the exact int GEMM.

    Returns (y fp16 [M, N], acc int32 [M, N] or None).
    """
    _need(xq, torch.uint8, "xq")
    _need(wq, torch.uint8, "wq")
    M, KB = xq.shape
    N = wq.shape[0]
    if wq.shape[1] != KB:
        raise ValueError("xq and wq disagree on K")
    K = 2 * KB
    dev = xq.device
    y = torch.empty((M, N), dtype=torch.float16, device=dev) if out is None else out
    acc = torch.empty((M, N), dtype=torch.int32, device=dev) if dbg else None
    x_alpha = x_alpha.reshape(-1)
    x_beta = x_beta.reshape(-1)
    _check(lib().sq_w4a4_linear(_ptr(xq), _ptr(x_alpha), _ptr(x_beta), M, _ptr(wq), _ptr(w_alpha), _ptr(w_rowsum),
                                N, K, _ptr(bias), _ptr(y), y.stride(0), _ptr(acc), _stream(xq)), "sq_w4a4_linear")
    return y, acc


def w4a8_linear(xq, x_alpha, x_beta, wq, w_alpha, w_rowsum, bias=None, out=None, dbg=False):
    """y = fp16(s_n (alpha_m acc + beta_m rowsum_n) + bias_n) with 8-bit activation codes
    xq uint8 [M, K] (had_quant_act bits=8) and packed 4-bit weights wq uint8 [N, K/2].
    Returns (y fp16 [M, N], acc int32 [M, N] or None).
    """
    _need(xq, torch.uint8, "xq")
    _need(wq, torch.uint8, "wq")
    M, K = xq.shape
    N = wq.shape[0]
    if 2 * wq.shape[1] != K:
        raise ValueError("xq and wq disagree on K")
    dev = xq.device
    y = torch.empty((M, N), dtype=torch.float16, device=dev) if out is None else out
    acc = torch.empty((M, N), dtype=torch.int32, device=dev) if dbg else None
    _check(lib().sq_w4a8_linear(_ptr(xq), _ptr(x_alpha.reshape(-1)), _ptr(x_beta.reshape(-1)), M, _ptr(wq),
                                _ptr(w_alpha), _ptr(w_rowsum), N, K, _ptr(bias), _ptr(y), y.stride(0), _ptr(acc),
                                _stream(xq)), "sq_w4a8_linear")
    return y, acc


def w4a4_linear_swiglu(xq, x_alpha, x_beta, wq, w_alpha, w_rowsum, bias=None, out=None):
    """h = fp16(SiLU(gate) * up) from gate/up weights packed as one matrix whose rows
    interleave them in blocks of 32 (see interleave_gate_up).  Returns h fp16 [M, N/2].
    """
    _need(xq, torch.uint8, "xq")
    _need(wq, torch.uint8, "wq")
    M, KB = xq.shape
    N = wq.shape[0]
    if wq.shape[1] != KB:
        raise ValueError("xq and wq disagree on K")
    h = torch.empty((M, N // 2), dtype=torch.float16, device=xq.device) if out is None else out
    _check(lib().sq_w4a4_linear_swiglu(_ptr(xq), _ptr(x_alpha.reshape(-1)), _ptr(x_beta.reshape(-1)), M, _ptr(wq),
                                       _ptr(w_alpha), _ptr(w_rowsum), N, 2 * KB, _ptr(bias), _ptr(h), h.stride(0),
                                       _stream(xq)), "sq_w4a4_linear_swiglu")
    return h


def interleave_gate_up(gate: torch.Tensor, up: torch.Tensor) -> torch.Tensor:
    """Rows of gate [I, ...] and up [I, ...] interleaved in blocks of 32 (I % 32 == 0): the
    row order sq_w4a4_linear_swiglu expects of its weights, scales, row sums and bias."""
    I = gate.shape[0]
    if up.shape != gate.shape or I % 32:
        raise ValueError("gate and up need the same shape with a multiple of 32 rows")
    return torch.stack([gate.reshape(I // 32, 32, *gate.shape[1:]), up.reshape(I // 32, 32, *up.shape[1:])],
                       dim=1).reshape(2 * I, *gate.shape[1:])


def qk_had_kvquant(q, k, v, dbg: bool = False, out=None, bits: int = 4, k_clip: float = 1.0,
                   v_clip: float = 1.0, param_dtype=torch.float32):
    """R3 on Q and K per head (D = 128) + 4-bit (or 8-bit) asymmetric K/V quantization, group 128.

    k_clip, v_clip: range clipping ratios in (0, 1]; param_dtype torch.float32 or
    torch.float16 for the group parameters (either away from the default:
    sq_qk_had_kvquant_ex).  Returns dict(q_rot, k_q, k_alpha, k_beta, v_q, v_alpha, v_beta,
    k_rot (or None)).
    """
    for t, nme in ((q, "q"), (k, "k"), (v, "v")):
        _need(t, torch.float16, nme)
        if not t.is_contiguous():
            raise ValueError(f"{nme} must be contiguous")
    B, S, H, D = q.shape
    dev = q.device
    if out is None:
        out = dict(q_rot=torch.empty_like(q),
                   k_q=torch.empty((B, S, H, D * bits // 8), dtype=torch.uint8, device=dev),
                   k_alpha=torch.empty((B, S, H, 1), dtype=param_dtype, device=dev),
                   k_beta=torch.empty((B, S, H, 1), dtype=param_dtype, device=dev),
                   v_q=torch.empty((B, S, H, D * bits // 8), dtype=torch.uint8, device=dev),
                   v_alpha=torch.empty((B, S, H, 1), dtype=param_dtype, device=dev),
                   v_beta=torch.empty((B, S, H, 1), dtype=param_dtype, device=dev))
    pbits = {torch.float32: 32, torch.float16: 16}[param_dtype]
    for nme in ("k_alpha", "k_beta", "v_alpha", "v_beta"):
        _need(out[nme], param_dtype, nme)
    kr = torch.empty((B, S, H, D), dtype=torch.float32, device=dev) if dbg else None
    outs = (_ptr(out["q_rot"]), _ptr(out["k_q"]), _ptr(out["k_alpha"]), _ptr(out["k_beta"]), _ptr(out["v_q"]),
            _ptr(out["v_alpha"]), _ptr(out["v_beta"]), _ptr(kr), _stream(q))
    if k_clip == 1.0 and v_clip == 1.0 and pbits == 32:
        _check(lib().sq_qk_had_kvquant(_ptr(q), _ptr(k), _ptr(v), B, S, H, D, bits, 128, *outs), "sq_qk_had_kvquant")
    else:
        _check(lib().sq_qk_had_kvquant_ex(_ptr(q), _ptr(k), _ptr(v), B, S, H, D, bits, 128, float(k_clip),
                                          float(v_clip), pbits, *outs), "sq_qk_had_kvquant_ex")
    out = dict(out)
    out["k_rot"] = kr
    return out


def attn_decode_workspace_bytes(B, S, H, D=128):
    """Device bytes of the workspace attn_decode_kv4_split needs on the current device."""
    n = ctypes.c_uint64(0)
    _check(lib().sq_attn_decode_workspace(B, S, H, D, ctypes.byref(n)), "sq_attn_decode_workspace")
    return n.value


def attn_decode_kv4_split(q_rot, k_q, k_alpha, k_beta, v_q, v_alpha, v_beta, scale=None, out=None, workspace=None):
    """attn_decode_kv4 split over the sequence (sq_attn_decode_kv4_split).  workspace: a
    uint8 device tensor of at least attn_decode_workspace_bytes() bytes, allocated here
    when None.  Returns out fp16 [B, H, 128]."""
    _need(q_rot, torch.float16, "q_rot")
    for t, nme in ((q_rot, "q_rot"), (k_q, "k_q"), (v_q, "v_q"), (k_alpha, "k_alpha"), (k_beta, "k_beta"),
                   (v_alpha, "v_alpha"), (v_beta, "v_beta")):
        if not t.is_contiguous():
            raise ValueError(f"{nme} must be contiguous")
    B, H, D = q_rot.shape
    S = k_q.shape[1]
    scale = 1.0 / D ** 0.5 if scale is None else scale
    out = torch.empty_like(q_rot) if out is None else out
    pdt = k_alpha.dtype
    for t, nme in ((k_alpha, "k_alpha"), (k_beta, "k_beta"), (v_alpha, "v_alpha"), (v_beta, "v_beta")):
        _need(t, pdt, nme)
    if workspace is None:
        workspace = torch.empty(max(attn_decode_workspace_bytes(B, S, H, D), 1), dtype=torch.uint8,
                                device=q_rot.device)
    _need(workspace, torch.uint8, "workspace")
    _check(lib().sq_attn_decode_kv4_split(_ptr(q_rot), _ptr(k_q), _ptr(k_alpha), _ptr(k_beta), _ptr(v_q),
                                          _ptr(v_alpha), _ptr(v_beta), B, S, H, D, float(scale),
                                          {torch.float32: 32, torch.float16: 16}[pdt], _ptr(out), _ptr(workspace),
                                          workspace.numel(), _stream(q_rot)), "sq_attn_decode_kv4_split")
    return out


def attn_decode_kv4_split_noalloc(q_rot, k_q, k_alpha, k_beta, v_q, v_alpha, v_beta, scale=None, out=None):
    """attn_decode_kv4_split with the library's own scratch (sq_attn_decode_kv4_split_noalloc):
    the call allocates no device memory (out must then be given).  Returns out."""
    _need(q_rot, torch.float16, "q_rot")
    for t, nme in ((q_rot, "q_rot"), (k_q, "k_q"), (v_q, "v_q"), (k_alpha, "k_alpha"), (k_beta, "k_beta"),
                   (v_alpha, "v_alpha"), (v_beta, "v_beta")):
        if not t.is_contiguous():
            raise ValueError(f"{nme} must be contiguous")
    B, H, D = q_rot.shape
    S = k_q.shape[1]
    scale = 1.0 / D ** 0.5 if scale is None else scale
    out = torch.empty_like(q_rot) if out is None else out
    pdt = k_alpha.dtype
    for t, nme in ((k_alpha, "k_alpha"), (k_beta, "k_beta"), (v_alpha, "v_alpha"), (v_beta, "v_beta")):
        _need(t, pdt, nme)
    _check(lib().sq_attn_decode_kv4_split_noalloc(_ptr(q_rot), _ptr(k_q), _ptr(k_alpha), _ptr(k_beta), _ptr(v_q),
                                                  _ptr(v_alpha), _ptr(v_beta), B, S, H, D, float(scale),
                                                  {torch.float32: 32, torch.float16: 16}[pdt], _ptr(out),
                                                  _stream(q_rot)), "sq_attn_decode_kv4_split_noalloc")
    return out


def attn_decode_kv4(q_rot, k_q, k_alpha, k_beta, v_q, v_alpha, v_beta, scale=None, out=None):
    """Attention of one rotated query per (batch, head), q_rot fp16 [B, H, 128], over the
    4-bit cache of qk_had_kvquant (k_q, v_q uint8 [B, S, H, 64], group parameters fp32, or
    fp16 through sq_attn_decode_kv4_ex, [B, S, H(, 1)]).  Returns out fp16 [B, H, 128]."""
    _need(q_rot, torch.float16, "q_rot")
    for t, nme in ((q_rot, "q_rot"), (k_q, "k_q"), (v_q, "v_q"), (k_alpha, "k_alpha"), (k_beta, "k_beta"),
                   (v_alpha, "v_alpha"), (v_beta, "v_beta")):
        if not t.is_contiguous():
            raise ValueError(f"{nme} must be contiguous")
    B, H, D = q_rot.shape
    S = k_q.shape[1]
    scale = 1.0 / D ** 0.5 if scale is None else scale
    out = torch.empty_like(q_rot) if out is None else out
    pdt = k_alpha.dtype
    for t, nme in ((k_alpha, "k_alpha"), (k_beta, "k_beta"), (v_alpha, "v_alpha"), (v_beta, "v_beta")):
        _need(t, pdt, nme)
    if pdt == torch.float32:
        _check(lib().sq_attn_decode_kv4(_ptr(q_rot), _ptr(k_q), _ptr(k_alpha), _ptr(k_beta), _ptr(v_q),
                                        _ptr(v_alpha), _ptr(v_beta), B, S, H, D, float(scale), _ptr(out),
                                        _stream(q_rot)), "sq_attn_decode_kv4")
    else:
        _check(lib().sq_attn_decode_kv4_ex(_ptr(q_rot), _ptr(k_q), _ptr(k_alpha), _ptr(k_beta), _ptr(v_q),
                                           _ptr(v_alpha), _ptr(v_beta), B, S, H, D, float(scale),
                                           {torch.float16: 16}[pdt], _ptr(out), _stream(q_rot)),
               "sq_attn_decode_kv4_ex")
    return out
