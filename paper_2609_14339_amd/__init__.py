"""Python binding of libacsc.so (include/acsc.h): argument marshalling only.

Every step of the hot path runs in the HIP library; this module turns torch
tensors into device pointers and the current HIP stream, calls the C entry
point of the same name, and raises ``AcscError`` on a non-zero return code.
There is no fallback: if the library is not built, importing this package
raises ``ImportError``.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libacsc.so")

F32, BF16 = 0, 1
SC_KMAX = 192

ACSC_OK, ACSC_EINVAL, ACSC_EDTYPE, ACSC_EALIGN, ACSC_EHIP, ACSC_ENOSPC, ACSC_ENOCONV = 0, -1, -2, -3, -4, -5, -6


class AcscError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"acsc error {code}: {msg}")
        self.code = code


class MaskKey(C.Structure):
    """ac_mask_key: the fields of the paper's g(layer, step, B, S, H) plus a
    seed and a microbatch id."""
    _fields_ = [("seed", C.c_uint64), ("step", C.c_uint64), ("layer", C.c_uint32),
                ("microbatch", C.c_uint32), ("B", C.c_uint32), ("S", C.c_uint32),
                ("H", C.c_uint32)]


class ScMatrix(C.Structure):
    """sc_matrix: one weight matrix of a batched sc_* call."""
    _fields_ = [("G", C.c_void_p), ("M", C.c_void_p), ("m", C.c_int), ("n", C.c_int),
                ("U", C.c_void_p), ("s", C.c_void_p), ("V", C.c_void_p), ("d", C.c_void_p),
                ("V_warm", C.c_void_p), ("G_proj", C.c_void_p), ("ws", C.c_void_p),
                ("ws_bytes", C.c_size_t)]


class AdamwState(C.Structure):
    """sc_adamw_state: one matrix's fp32 weights and Adam moments (in place)."""
    _fields_ = [("W", C.c_void_p), ("m1", C.c_void_p), ("m2", C.c_void_p)]


class AdamwHparams(C.Structure):
    """sc_adamw_hparams: one step's AdamW hyperparameters."""
    _fields_ = [("lr", C.c_float), ("beta1", C.c_float), ("beta2", C.c_float), ("eps", C.c_float),
                ("weight_decay", C.c_float), ("step", C.c_int64), ("max_norm", C.c_float)]


class PsgdMatrix(C.Structure):
    """psgd_matrix: one matrix of a PowerSGD call."""
    _fields_ = [("G", C.c_void_p), ("E", C.c_void_p), ("P", C.c_void_p), ("Q", C.c_void_p),
                ("out", C.c_void_p), ("m", C.c_int), ("n", C.c_int), ("ws", C.c_void_p),
                ("ws_bytes", C.c_size_t)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                          "(or python paper_2609_14339_amd/build.py)")
    lib = C.CDLL(LIB_PATH)
    vp, i32, i64, u64, f32, sz = C.c_void_p, C.c_int, C.c_int64, C.c_uint64, C.c_float, C.c_size_t
    lib.acsc_last_error.restype = C.c_char_p
    lib.acsc_last_error.argtypes = []
    lib.acsc_version.restype = i32
    lib.ac_keep_count.restype = i32
    lib.ac_keep_count.argtypes = [i32, C.c_double, C.POINTER(i32)]
    lib.ac_mask_pack.restype = i32
    lib.ac_mask_pack.argtypes = [vp, i32, i64, i32, i64, i32, C.POINTER(MaskKey), vp, vp, vp]
    lib.ac_unpack_scatter.restype = i32
    lib.ac_unpack_scatter.argtypes = [vp, vp, i32, i64, i32, i32, C.POINTER(MaskKey), f32, vp,
                                      i64, vp]
    lib.ac_mask_pack_batched.restype = i32
    lib.ac_mask_pack_batched.argtypes = [vp, i32, i32, i64, i32, i64, i64, i32, C.POINTER(MaskKey), vp, i64,
                                         vp, vp, i64, vp]
    lib.ac_unpack_scatter_batched.restype = i32
    lib.ac_unpack_scatter_batched.argtypes = [vp, i64, i32, i32, i64, i32, i32, C.POINTER(MaskKey), vp, vp, i64,
                                              f32, vp, i64, i64, vp]
    lib.ac_bern_mask.restype = i32
    lib.ac_bern_mask.argtypes = [i64, i32, C.c_double, C.POINTER(MaskKey), vp, vp, vp]
    lib.ac_bern_pack.restype = i32
    lib.ac_bern_pack.argtypes = [vp, i32, i64, i32, i64, vp, vp, vp, vp, i64, vp]
    lib.ac_bern_unpack.restype = i32
    lib.ac_bern_unpack.argtypes = [vp, i32, i64, i32, vp, vp, i64, f32, vp, i64, vp]
    lib.sc_workspace_size.restype = i32
    lib.sc_workspace_size.argtypes = [i32, i32, i32, i32, i32, C.POINTER(sz)]
    lib.sc_build_prior.restype = i32
    lib.sc_build_prior.argtypes = [vp, i32, vp, i32, i32, f32, i32, i32, i32, f32, vp, u64,
                                   vp, vp, vp, vp, vp, sz, vp]
    lib.sc_correct.restype = i32
    lib.sc_correct.argtypes = [vp, i32, i32, i32, vp, vp, vp, i32, f32, vp, vp, sz, vp]
    lib.sc_correct_static.restype = i32
    lib.sc_correct_static.argtypes = [vp, i32, i32, i32, vp, vp, vp, i32, f32, vp, vp]
    for fn in (lib.sc_build_prior_batched, lib.sc_build_subspace_batched, lib.sc_build_ritz_batched):
        fn.restype = i32
        fn.argtypes = [i32, C.POINTER(ScMatrix), i32, f32, i32, i32, i32, f32, u64, vp]
    lib.sc_build_status.restype = i32
    lib.sc_build_status.argtypes = [i32, C.POINTER(ScMatrix), vp, vp, vp]
    lib.sc_correct_batched.restype = i32
    lib.sc_correct_batched.argtypes = [i32, C.POINTER(ScMatrix), i32, i32, f32, vp]
    lib.sc_adamw_workspace_size.restype = i32
    lib.sc_adamw_workspace_size.argtypes = [i32, i32, i32, i32, C.POINTER(sz)]
    lib.sc_correct_adamw_batched.restype = i32
    lib.sc_correct_adamw_batched.argtypes = [i32, C.POINTER(ScMatrix), C.POINTER(AdamwState), i32, i32, f32,
                                             C.POINTER(AdamwHparams), vp, vp]
    lib.psgd_workspace_size.restype = i32
    lib.psgd_workspace_size.argtypes = [i32, i32, i32, i32, C.POINTER(sz)]
    for name in ("psgd_project", "psgd_orthogonalize", "psgd_decompress", "psgd_step"):
        fn = getattr(lib, name)
        fn.restype = i32
        fn.argtypes = [i32, C.POINTER(PsgdMatrix), i32, i32, vp]
    lib.acsc_stats_enable.restype = i32
    lib.acsc_stats_enable.argtypes = [i32]
    lib.acsc_stats_only.restype = i32
    lib.acsc_stats_only.argtypes = [C.c_char_p]
    lib.acsc_stats_read.restype = i32
    lib.acsc_stats_read.argtypes = [i32, C.c_char_p, sz, C.POINTER(i64), C.POINTER(C.c_double)]
    return lib


lib = _load()

EXPORTED = ("acsc_last_error", "acsc_version", "acsc_stats_enable", "acsc_stats_only", "acsc_stats_read",
            "ac_keep_count", "ac_mask_pack", "ac_unpack_scatter", "ac_mask_pack_batched",
            "ac_unpack_scatter_batched", "sc_workspace_size",
            "sc_build_prior", "sc_correct", "sc_correct_static", "sc_build_prior_batched", "sc_correct_batched",
            "sc_build_subspace_batched", "sc_build_ritz_batched", "sc_build_status",
            "sc_adamw_workspace_size", "sc_correct_adamw_batched",
            "ac_bern_mask", "ac_bern_pack", "ac_bern_unpack",
            "psgd_workspace_size", "psgd_project", "psgd_orthogonalize", "psgd_decompress", "psgd_step")


def _check(rc: int):
    if rc != 0:
        raise AcscError(rc, lib.acsc_last_error().decode())


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise AcscError(ACSC_EDTYPE, f"unsupported dtype {t.dtype}")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _need_cuda(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise AcscError(ACSC_EINVAL, "tensors must live on the GPU")


def _in(t: Optional[torch.Tensor]) -> Optional[torch.Tensor]:
    """Row-major copy of an input if it is not already contiguous."""
    return None if t is None else t.contiguous()


def _out(*ts):
    for t in ts:
        if t is not None and not t.is_contiguous():
            raise AcscError(ACSC_EINVAL, "output and in/out tensors must be contiguous")


def acsc_stats_enable(on: bool = True) -> None:
    """Start (resetting the counters) or stop per-kernel event timing."""
    _check(lib.acsc_stats_enable(1 if on else 0))


def acsc_stats_only(tag=None) -> None:
    """Time only the launches of kernel name `tag` (None: every launch)."""
    _check(lib.acsc_stats_only(tag.encode() if tag else None))


def acsc_stats_read() -> dict:
    """{kernel name: (launches, total milliseconds)} of the timed launches."""
    out = {}
    i = 0
    buf = C.create_string_buffer(128)
    n = C.c_int64(0)
    ms = C.c_double(0.0)
    while lib.acsc_stats_read(i, buf, 128, C.byref(n), C.byref(ms)) == 0:
        out[buf.value.decode()] = (n.value, ms.value)
        i += 1
    return out


def make_key(seed: int, layer: int, step: int, microbatch: int, B: int, S: int, H: int) -> MaskKey:
    return MaskKey(seed=seed, step=step, layer=layer, microbatch=microbatch, B=B, S=S, H=H)


def ac_keep_count(H: int, keep: float) -> int:
    k = C.c_int(0)
    _check(lib.ac_keep_count(H, keep, C.byref(k)))
    return k.value


def ac_mask_pack(x: torch.Tensor, K: int, key: MaskKey, vals: Optional[torch.Tensor] = None,
                 idx: Optional[torch.Tensor] = None, with_idx: bool = True, stream=None):
    """x: [rows, H] (row stride x.stride(0)).  Returns (vals [rows, K], idx
    [rows, K] int16 holding uint16 patterns, or None)."""
    _need_cuda(x)
    if x.dim() != 2 or x.stride(1) != 1:
        raise AcscError(ACSC_EINVAL, "x must be 2-D with unit column stride")
    rows, H = x.shape
    if vals is None:
        vals = torch.empty(rows, K, dtype=x.dtype, device=x.device)
    if idx is None and with_idx:
        idx = torch.empty(rows, K, dtype=torch.int16, device=x.device)
    _need_cuda(vals, idx)
    _check(lib.ac_mask_pack(_ptr(x), _dt(x), rows, H, x.stride(0), K, C.byref(key), _ptr(vals),
                            _ptr(idx), _stream(stream)))
    return vals, idx


def ac_unpack_scatter(vals: torch.Tensor, H: int, key: MaskKey, scale: float = 1.0,
                      idx: Optional[torch.Tensor] = None, y: Optional[torch.Tensor] = None,
                      stream=None) -> torch.Tensor:
    """Dense [rows, H] output (or into ``y``, row stride y.stride(0))."""
    _need_cuda(vals, idx)
    rows, K = vals.shape
    if y is None:
        y = torch.empty(rows, H, dtype=vals.dtype, device=vals.device)
    _need_cuda(y)
    if y.dim() != 2 or y.stride(1) != 1 or not vals.is_contiguous():
        raise AcscError(ACSC_EINVAL, "vals must be contiguous and y 2-D with unit column stride")
    _check(lib.ac_unpack_scatter(_ptr(vals), _ptr(idx), _dt(vals), rows, H, K, C.byref(key),
                                 float(scale), _ptr(y), y.stride(0), _stream(stream)))
    return y


def _layer_stride(t: torch.Tensor) -> int:
    return t.stride(0) if t.shape[0] > 1 else 0


def ac_mask_pack_batched(x: torch.Tensor, K: int, key: MaskKey, vals: Optional[torch.Tensor] = None,
                         idx_in: Optional[torch.Tensor] = None, idx_out: Optional[torch.Tensor] = None,
                         stream=None) -> torch.Tensor:
    """x: [nlayers, rows, H] (unit column stride; row and layer strides taken
    from the tensor).  Boundary l is keyed with key.layer + l.  Returns vals
    [nlayers, rows, K].  idx_in: [nlayers, rows, K] index lists to pack at
    (no mask evaluated); idx_out: receives the kept positions (int16 holding
    uint16 patterns)."""
    _need_cuda(x, vals, idx_in, idx_out)
    if x.dim() != 3 or x.stride(2) != 1:
        raise AcscError(ACSC_EINVAL, "x must be [nlayers, rows, H] with unit column stride")
    nl, rows, H = x.shape
    if vals is None:
        vals = torch.empty(nl, rows, K, dtype=x.dtype, device=x.device)
    _need_cuda(vals)
    idx_stride = 0
    for t in (idx_in, idx_out):
        if t is not None:
            if tuple(t.shape) != (nl, rows, K) or t.stride(2) != 1 or t.stride(1) != K:
                raise AcscError(ACSC_EINVAL, "index lists must be [nlayers, rows, K] with contiguous rows")
            idx_stride = _layer_stride(t)
    if tuple(vals.shape) != (nl, rows, K) or vals.stride(2) != 1 or vals.stride(1) != K:
        raise AcscError(ACSC_EINVAL, "vals must be [nlayers, rows, K] with contiguous rows")
    _check(lib.ac_mask_pack_batched(_ptr(x), _dt(x), nl, rows, H, x.stride(1), _layer_stride(x), K, C.byref(key),
                                    _ptr(vals), _layer_stride(vals), _ptr(idx_in), _ptr(idx_out), idx_stride,
                                    _stream(stream)))
    return vals


def ac_unpack_scatter_batched(vals: torch.Tensor, H: int, key: MaskKey, scale: float = 1.0,
                              idx_in: Optional[torch.Tensor] = None, idx_out: Optional[torch.Tensor] = None,
                              y: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """vals: [nlayers, rows, K].  Returns (or fills) y [nlayers, rows, H].
    idx_in: transmitted or kept index lists; idx_out: receives the positions
    rebuilt from the key."""
    _need_cuda(vals, idx_in, idx_out)
    if vals.dim() != 3 or vals.stride(2) != 1 or vals.stride(1) != vals.shape[2]:
        raise AcscError(ACSC_EINVAL, "vals must be [nlayers, rows, K] with contiguous rows")
    nl, rows, K = vals.shape
    if y is None:
        y = torch.empty(nl, rows, H, dtype=vals.dtype, device=vals.device)
    _need_cuda(y)
    if y.dim() != 3 or y.stride(2) != 1 or tuple(y.shape) != (nl, rows, H):
        raise AcscError(ACSC_EINVAL, "y must be [nlayers, rows, H] with unit column stride")
    idx_stride = 0
    for t in (idx_in, idx_out):
        if t is not None:
            if tuple(t.shape) != (nl, rows, K) or t.stride(2) != 1 or t.stride(1) != K:
                raise AcscError(ACSC_EINVAL, "index lists must be [nlayers, rows, K] with contiguous rows")
            idx_stride = _layer_stride(t)
    _check(lib.ac_unpack_scatter_batched(_ptr(vals), _layer_stride(vals), _dt(vals), nl, rows, H, K, C.byref(key),
                                         _ptr(idx_in), _ptr(idx_out), idx_stride, float(scale), _ptr(y), y.stride(1),
                                         _layer_stride(y), _stream(stream)))
    return y


def ac_bern_mask(rows: int, H: int, keep: float, key: MaskKey, device="cuda", stream=None):
    """The Bernoulli mask of a [rows, H] tensor: (row_ptr int64 [rows + 1],
    bits int32 [rows, ceil(H / 32)] holding uint32 patterns)."""
    row_ptr = torch.empty(rows + 1, dtype=torch.int64, device=device)
    bits = torch.empty(max(rows, 1), (H + 31) // 32, dtype=torch.int32, device=device)[:rows]
    _check(lib.ac_bern_mask(rows, H, float(keep), C.byref(key), _ptr(row_ptr), _ptr(bits), _stream(stream)))
    return row_ptr, bits


def ac_bern_pack(x: torch.Tensor, row_ptr: torch.Tensor, bits: torch.Tensor, nnz: Optional[int] = None,
                 with_idx: bool = True, stream=None):
    """Packed values [nnz] (and uint16 indices as int16, or None) of x [rows, H]
    under the mask (row_ptr, bits).  nnz defaults to row_ptr[-1] (a host
    read, which synchronises)."""
    _need_cuda(x, row_ptr, bits)
    if x.dim() != 2 or x.stride(1) != 1:
        raise AcscError(ACSC_EINVAL, "x must be 2-D with unit column stride")
    rows, H = x.shape
    if nnz is None:
        nnz = int(row_ptr[-1].item())
    vals = torch.empty(max(nnz, 1), dtype=x.dtype, device=x.device)[:nnz]
    idx = torch.empty(max(nnz, 1), dtype=torch.int16, device=x.device)[:nnz] if with_idx else None
    _check(lib.ac_bern_pack(_ptr(x), _dt(x), rows, H, x.stride(0), _ptr(row_ptr), _ptr(bits), _ptr(vals),
                            _ptr(idx), nnz, _stream(stream)))
    return vals, idx


def ac_bern_unpack(vals: torch.Tensor, H: int, row_ptr: torch.Tensor, bits: torch.Tensor, scale: float = 1.0,
                   y: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Dense [rows, H]: scale * value at the kept entries, +0 elsewhere."""
    _need_cuda(vals, row_ptr, bits)
    rows = row_ptr.numel() - 1
    if y is None:
        y = torch.empty(rows, H, dtype=vals.dtype, device=vals.device)
    _need_cuda(y)
    if y.dim() != 2 or y.stride(1) != 1 or not vals.is_contiguous():
        raise AcscError(ACSC_EINVAL, "vals must be contiguous and y 2-D with unit column stride")
    _check(lib.ac_bern_unpack(_ptr(vals), _dt(vals), rows, H, _ptr(row_ptr), _ptr(bits), vals.numel(),
                              float(scale), _ptr(y), y.stride(0), _stream(stream)))
    return y


def sc_workspace_size(m: int, n: int, r: int, oversample: int, dtype: torch.dtype) -> int:
    b = C.c_size_t(0)
    code = BF16 if dtype == torch.bfloat16 else F32
    _check(lib.sc_workspace_size(m, n, r, oversample, code, C.byref(b)))
    return b.value


def workspace(m: int, n: int, r: int, oversample: int, dtype: torch.dtype, device="cuda"):
    nbytes = sc_workspace_size(m, n, r, oversample, dtype)
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


def sc_build_prior(G_anc: Optional[torch.Tensor], M: torch.Tensor, r: int, beta: float,
                   tau: float, oversample: int, power_iters: int, seed: int = 0,
                   V_warm: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                   out=None, dtype: Optional[torch.dtype] = None, stream=None):
    """EMA of G_anc into M (fp32, in place), then (U, s, V, d).  Returns them."""
    _need_cuda(G_anc, M, V_warm)
    G_anc, V_warm = _in(G_anc), _in(V_warm)
    _out(M)
    m, n = M.shape
    dt = dtype if dtype is not None else (G_anc.dtype if G_anc is not None else torch.float32)
    if out is None:
        out = (torch.empty(m, r, device=M.device), torch.empty(r, device=M.device),
               torch.empty(n, r, device=M.device), torch.empty(r, device=M.device))
    U, s, V, d = out
    _out(U, s, V, d)
    if ws is None:
        ws = workspace(m, n, r, oversample, dt, M.device)
    code = BF16 if dt == torch.bfloat16 else F32
    _check(lib.sc_build_prior(_ptr(G_anc), code, _ptr(M), m, n, float(beta), r, oversample,
                              power_iters, float(tau), _ptr(V_warm), seed, _ptr(U), _ptr(s),
                              _ptr(V), _ptr(d), _ptr(ws), ws.numel(), _stream(stream)))
    return U, s, V, d


def sc_correct(G: torch.Tensor, U: torch.Tensor, d: torch.Tensor, V: torch.Tensor, alpha: float,
               out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
               stream=None) -> torch.Tensor:
    """G_proj = alpha G + (1 - alpha) U diag(d) U^T G V diag(d) V^T."""
    _need_cuda(G, U, d, V, out)
    G, U, d, V = _in(G), _in(U), _in(d), _in(V)
    _out(out)
    m, n = G.shape
    r = U.shape[1]
    if out is None:
        out = torch.empty_like(G)
    if ws is None:
        ws = workspace(m, n, r, 0, G.dtype, G.device)
    _check(lib.sc_correct(_ptr(G), _dt(G), m, n, _ptr(U), _ptr(d), _ptr(V), r, float(alpha),
                          _ptr(out), _ptr(ws), ws.numel(), _stream(stream)))
    return out


SC_STATIC_SCRATCH_BYTES = 96 * 1024 * 1024


def sc_correct_static(G: torch.Tensor, U: torch.Tensor, d: torch.Tensor, V: torch.Tensor, alpha: float,
                      out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """sc_correct on the library's own device scratch (no workspace; for
    callers that cannot allocate).  ``out`` must be given by a caller that
    cannot allocate; calls that overlap on one GPU race."""
    _need_cuda(G, U, d, V, out)
    for t in (G, U, d, V):
        if not t.is_contiguous():
            raise AcscError(ACSC_EINVAL, "G, U, d, V must be contiguous (no copies are made)")
    _out(out)
    m, n = G.shape
    r = U.shape[1]
    if out is None:
        out = torch.empty_like(G)
    _check(lib.sc_correct_static(_ptr(G), _dt(G), m, n, _ptr(U), _ptr(d), _ptr(V), r, float(alpha), _ptr(out),
                                 _stream(stream)))
    return out


def _p(t):
    return None if t is None else t.data_ptr()


def sc_build_prior_batched(items, r: int, beta: float, tau: float, oversample: int,
                           power_iters: int, seed: int = 0, dtype: torch.dtype = torch.bfloat16,
                           stream=None):
    """items: list of dicts with G_anc (or None), M, out=(U, s, V, d), ws, and
    optionally V_warm.  Matrix i starts from the random block of seed + i."""
    _build_batched(lib.sc_build_prior_batched, items, r, beta, tau, oversample, power_iters, seed, dtype, stream)


def sc_build_subspace_batched(items, r: int, beta: float, tau: float, oversample: int,
                              power_iters: int, seed: int = 0, dtype: torch.dtype = torch.bfloat16,
                              stream=None):
    """First phase of sc_build_prior_batched (EMA, power passes, Z = M^T Q);
    the same arguments.  Follow it with sc_build_ritz_batched."""
    _build_batched(lib.sc_build_subspace_batched, items, r, beta, tau, oversample, power_iters, seed, dtype,
                   stream)


def sc_build_ritz_batched(items, r: int, beta: float, tau: float, oversample: int,
                          power_iters: int, seed: int = 0, dtype: torch.dtype = torch.bfloat16,
                          stream=None):
    """Second phase of sc_build_prior_batched (Rayleigh-Ritz on Z: U, s, V, d);
    the same arguments and workspaces as the sc_build_subspace_batched call
    it follows."""
    _build_batched(lib.sc_build_ritz_batched, items, r, beta, tau, oversample, power_iters, seed, dtype, stream)


def _build_batched(fn, items, r, beta, tau, oversample, power_iters, seed, dtype, stream):
    arr = (ScMatrix * max(len(items), 1))()
    keep = []
    for i, it in enumerate(items):
        G, M, (U, s, V, d), ws = _in(it.get("G_anc")), it["M"], it["out"], it["ws"]
        Vw = _in(it.get("V_warm"))
        _need_cuda(G, M, U, s, V, d, ws, Vw)
        _out(M, U, s, V, d)
        keep += [G, Vw]
        m, n = M.shape
        arr[i] = ScMatrix(_p(G), _p(M), m, n, _p(U), _p(s), _p(V), _p(d), _p(Vw), None, _p(ws),
                          ws.numel())
    code = BF16 if dtype == torch.bfloat16 else F32
    _check(fn(len(items), arr, code, float(beta), r, oversample, power_iters, float(tau), seed, _stream(stream)))


def sc_build_status(workspaces, stream=None):
    """Synchronise and read the status the last build left in each workspace:
    a list of (sweeps, residual) per workspace.  Raises AcscError with code
    ACSC_ENOCONV when a build stopped at its sweep cap above tolerance or ran
    its Rayleigh-Ritz phase without a subspace phase."""
    n = len(workspaces)
    arr = (ScMatrix * max(n, 1))()
    for i, ws in enumerate(workspaces):
        _need_cuda(ws)
        arr[i] = ScMatrix(None, None, 0, 0, None, None, None, None, None, None, _p(ws), ws.numel())
    sweeps = (C.c_int * max(n, 1))()
    res = (C.c_float * max(n, 1))()
    rc = lib.sc_build_status(n, arr, sweeps, res, _stream(stream))
    out = [(sweeps[i], res[i]) for i in range(n)]
    if rc != 0:
        err = AcscError(rc, lib.acsc_last_error().decode())
        err.status = out
        raise err
    return out


def sc_correct_batched(items, r: int, alpha: float, dtype: torch.dtype = torch.bfloat16,
                       stream=None):
    """items: list of dicts with G, prior=(U, d, V), out (G_proj) and ws."""
    arr = (ScMatrix * max(len(items), 1))()
    keep = []
    for i, it in enumerate(items):
        G, (U, d, V), out, ws = _in(it["G"]), it["prior"], it["out"], it["ws"]
        U, d, V = _in(U), _in(d), _in(V)
        _need_cuda(G, U, d, V, out, ws)
        _out(out)
        keep += [G, U, d, V]
        m, n = G.shape
        arr[i] = ScMatrix(_p(G), None, m, n, _p(U), _p(d), _p(V), _p(d), None, _p(out), _p(ws),
                          ws.numel())
    code = BF16 if dtype == torch.bfloat16 else F32
    _check(lib.sc_correct_batched(len(items), arr, code, r, float(alpha), _stream(stream)))


def sc_adamw_workspace_size(m: int, n: int, r: int, dtype: torch.dtype) -> int:
    b = C.c_size_t(0)
    code = BF16 if dtype == torch.bfloat16 else F32
    _check(lib.sc_adamw_workspace_size(m, n, r, code, C.byref(b)))
    return b.value


def sc_correct_adamw_batched(items, r: int, alpha: float, lr: float, beta1: float = 0.9,
                             beta2: float = 0.999, eps: float = 1e-8, weight_decay: float = 0.0,
                             step: int = 1, max_norm: float = 0.0, dtype: torch.dtype = torch.bfloat16,
                             norm_out: Optional[torch.Tensor] = None, stream=None):
    """items: list of dicts with G, prior=(U, d, V), ws and state=(W, m1, m2)
    (fp32, updated in place).  norm_out: optional fp32 device scalar that
    receives the global norm of the G_proj before clipping."""
    arr = (ScMatrix * max(len(items), 1))()
    st = (AdamwState * max(len(items), 1))()
    keep = []
    for i, it in enumerate(items):
        G, (U, d, V), ws, (W, m1, m2) = _in(it["G"]), it["prior"], it["ws"], it["state"]
        U, d, V = _in(U), _in(d), _in(V)
        _need_cuda(G, U, d, V, ws, W, m1, m2, norm_out)
        _out(W, m1, m2)
        for t in (W, m1, m2):
            if t.dtype != torch.float32 or tuple(t.shape) != tuple(G.shape):
                raise AcscError(ACSC_EINVAL, "W, m1, m2 must be fp32 tensors of G's shape")
        keep += [G, U, d, V]
        m, n = G.shape
        arr[i] = ScMatrix(_p(G), None, m, n, _p(U), _p(d), _p(V), _p(d), None, None, _p(ws), ws.numel())
        st[i] = AdamwState(_p(W), _p(m1), _p(m2))
    hp = AdamwHparams(float(lr), float(beta1), float(beta2), float(eps), float(weight_decay), int(step),
                      float(max_norm))
    code = BF16 if dtype == torch.bfloat16 else F32
    _check(lib.sc_correct_adamw_batched(len(items), arr, st, code, r, float(alpha), C.byref(hp),
                                        _ptr(norm_out), _stream(stream)))


def psgd_workspace_size(m: int, n: int, r: int, dtype: torch.dtype) -> int:
    b = C.c_size_t(0)
    code = BF16 if dtype == torch.bfloat16 else F32
    _check(lib.psgd_workspace_size(m, n, r, code, C.byref(b)))
    return b.value


def psgd_workspace(m: int, n: int, r: int, dtype: torch.dtype, device="cuda"):
    return torch.empty(max(psgd_workspace_size(m, n, r, dtype), 256), dtype=torch.uint8, device=device)


def _psgd(name: str, items, r: int, dtype: torch.dtype, stream):
    arr = (PsgdMatrix * max(len(items), 1))()
    keep = []
    for i, it in enumerate(items):
        G, E, P, Q, out, ws = _in(it.get("G")), it["E"], it["P"], it["Q"], it.get("out"), it["ws"]
        _need_cuda(G, E, P, Q, out, ws)
        _out(E, P, Q, out)
        for t, shape in ((E, None), (P, (E.shape[0], r)), (Q, (E.shape[1], r))):
            if t.dtype != torch.float32 or (shape is not None and tuple(t.shape) != shape):
                raise AcscError(ACSC_EINVAL, "E [m, n], P [m, r], Q [n, r] must be fp32")
        keep.append(G)
        m, n = E.shape
        arr[i] = PsgdMatrix(_p(G), _p(E), _p(P), _p(Q), _p(out), m, n, _p(ws), ws.numel())
    code = BF16 if dtype == torch.bfloat16 else F32
    _check(getattr(lib, name)(len(items), arr, code, r, _stream(stream)))


def psgd_project(items, r: int, dtype: torch.dtype = torch.bfloat16, stream=None):
    """items: dicts with G, E, P, Q, ws (out unused): E <- E + G, P <- E Q."""
    _psgd("psgd_project", items, r, dtype, stream)


def psgd_orthogonalize(items, r: int, dtype: torch.dtype = torch.bfloat16, stream=None):
    """P <- orth(P), Q <- M^T P (M held in E and in the workspace)."""
    _psgd("psgd_orthogonalize", items, r, dtype, stream)


def psgd_decompress(items, r: int, dtype: torch.dtype = torch.bfloat16, stream=None):
    """out <- P Q^T (in dtype), E <- M - out."""
    _psgd("psgd_decompress", items, r, dtype, stream)


def psgd_step(items, r: int, dtype: torch.dtype = torch.bfloat16, stream=None):
    """The three phases on one worker (items: dicts with G, E, P, Q, out, ws)."""
    _psgd("psgd_step", items, r, dtype, stream)
