"""Python binding of the stage-boundary subspace codec (libsn.so, gfx950).

Argument marshalling only: each function turns torch tensors into the plain
pointers, sizes and strides of the C ABI in ``include/sn.h`` (same names) and
launches on the current torch stream.  Every step of the codec runs in the
library's HIP kernels; there is no fallback.  If the library has not been
built the first call raises ``RuntimeError``.

    basis = sn_basis_pack(U)                         # U: d x k, cuda, bf16 / fp32
    C  = sn_compress(basis, X, tok=tok, E=E, P=P, seq_len=S)
    Xr = sn_decompress(basis, C, tok=tok, E=E, P=P, seq_len=S)
    Cg = sn_grad_compress(basis, G)
    Gr = sn_decompress(basis, Cg)
    sn_project_weights(basis, W)                     # in place

    proj = sn_embed_project(basis, E=E, P=P)         # T_fixed U, P U (once per basis)
    C  = sn_compress_projected(basis, X, proj, tok=tok, seq_len=S)

    state = sn_grassmann_state(basis)                # subspace update (Sec. 4.5)
    Cg = sn_grassmann_accumulate(basis, G, state, want_cg=True)   # per iteration
    U2 = sn_grassmann_step(basis, state, eta)        # every few hundred iterations

    sn_adamw_step(W2, grad, M, V, t, lr, weight_decay=wd)   # modified AdamW (Sec. 5)
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# SN_LIBRARY names another build of the same C ABI (the host-sanitizer build
# of the CPU tests); by default the library built next to this file.
LIB_PATH = os.environ.get("SN_LIBRARY") or os.path.join(_HERE, "libsn.so")

SN_F32, SN_BF16 = 0, 1
SN_ERR_INDEX = 6
STATUS = {0: "SN_OK", 1: "SN_ERR_NULL", 2: "SN_ERR_SHAPE", 3: "SN_ERR_DTYPE", 4: "SN_ERR_ALIGN",
          5: "SN_ERR_ALIAS", 6: "SN_ERR_INDEX", 7: "SN_ERR_HIP", 8: "SN_ERR_UNSUPPORTED",
          9: "SN_ERR_WORKSPACE"}

_lib = None

_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I32 = ctypes.c_int32
_SZ = ctypes.c_size_t

_SIGNATURES = {
    "sn_basis_packed_bytes": (_SZ, [_I64, _I64, _I32]),
    "sn_basis_pack": (_I32, [_P, _I64, _I64, _I64, _I32, _P, _SZ, _P]),
    "sn_compress": (_I32, [_P, _I64, _I64, _I32, _P, _I64, _I64, _P, _P, _I64, _I64, _P, _P,
                           _I64, _I64, _I64, _P, _I64, _P, _P]),
    "sn_decompress": (_I32, [_P, _I64, _I64, _I32, _P, _I64, _I64, _P, _P, _I64, _I64, _P, _P,
                             _I64, _I64, _I64, _P, _I64, _P, _P]),
    "sn_grad_compress": (_I32, [_P, _I64, _I64, _I32, _P, _I64, _I64, _P, _I64, _P]),
    "sn_embed_projected_bytes": (_SZ, [_I64, _I64, _I64]),
    "sn_embed_project": (_I32, [_P, _I64, _I64, _I32, _P, _I64, _I64, _P, _I64, _I64, _P, _SZ,
                                _P]),
    "sn_compress_projected": (_I32, [_P, _I64, _I64, _I32, _P, _I64, _I64, _P, _P, _I64, _P,
                                     _I64, _I64, _P, _I64, _P, _P]),
    "sn_project_weights_workspace_bytes": (_SZ, [_I64, _I64, _I32, _I64]),
    "sn_project_weights": (_I32, [_P, _I64, _I64, _I32, _P, _I64, _I64, _P, _SZ, _P]),
    "sn_project_weights_noalloc": (_I32, [_P, _I64, _I64, _I32, _P, _I64, _I64, _P]),
    "sn_project_weights_multi_workspace_bytes": (_SZ, [_I64, _I64, _I32, _I32, _P]),
    "sn_project_weights_multi": (_I32, [_P, _I64, _I64, _I32, _I32, _P, _P, _P, _P, _SZ, _P]),
    "sn_grassmann_state_bytes": (_SZ, [_I64, _I64]),
    "sn_grassmann_workspace_bytes": (_SZ, [_I64, _I64, _I32, _I64]),
    "sn_grassmann_reset": (_I32, [_P, _I64, _I64, _P]),
    "sn_grassmann_accumulate": (_I32, [_P, _I64, _I64, _I32, _P, _I64, _I64, _P, _I64, _I32, _P,
                                       _P, _SZ, _P]),
    "sn_grassmann_step": (_I32, [_P, _I64, _I64, _I32, _P, ctypes.c_double, _P, _I64, _I32, _P,
                                 _SZ, _P, _P]),
    "sn_embed_lowrank_workspace_bytes": (_SZ, [_I64, _I64, _I32, _I64, _I64]),
    "sn_embed_lowrank_forward": (_I32, [_P, _I64, _I64, _I32, _P, _I64, _I64, _P, _P, _I64, _P,
                                        _P, _I64, _I64, _I64, _P, _I64, _I64, _P, _P, _SZ, _P]),
    "sn_embed_lowrank_backward": (_I32, [_P, _I64, _I64, _I32, _P, _I64, _I64, _P, _I64, _P,
                                         _I64, _P, _P, _SZ, _P]),
    "sn_adamw_workspace_bytes": (_SZ, [_I64, _I64]),
    "sn_adamw_step": (_I32, [_P, _I64, _P, _I64, _I32, _P, _P, _I64, _I64, _I64, _I64,
                             ctypes.c_double, ctypes.c_double, ctypes.c_double, ctypes.c_double,
                             ctypes.c_double, _I32, _P, _SZ, _P]),
    "sn_status_string": (ctypes.c_char_p, [_I32]),
    "sn_last_error": (ctypes.c_char_p, []),
    "sn_version": (ctypes.c_char_p, []),
}


# Id checking (debug / test mode): the kernels clamp out-of-range token and
# position ids and report them only through a device flag.  With checking on
# (set_check_ids(True), or SN_CHECK_IDS=1 in the environment) every call that
# takes ids gets a private flag, waits for the call to finish, ORs the flag
# into the caller's err_flag (if any) and raises SnError(SN_ERR_INDEX) when an
# id was out of range.  The wait serialises the stream: for tests and
# debugging, not for production loops.
_CHECK_IDS = os.environ.get("SN_CHECK_IDS", "") not in ("", "0")


def set_check_ids(on: bool = True) -> None:
    global _CHECK_IDS
    _CHECK_IDS = bool(on)


def check_ids_enabled() -> bool:
    return _CHECK_IDS


class SnError(RuntimeError):
    def __init__(self, status: int, message: str):
        self.status = status
        super().__init__(f"{STATUS.get(status, status)}: {message}")


def lib():
    """The loaded libsn.so (built by paper_2506_01260_amd.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run paper_2506_01260_amd.build.build()")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(status: int):
    if status != 0:
        raise SnError(status, lib().sn_last_error().decode())


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return SN_F32
    if t.dtype == torch.bfloat16:
        return SN_BF16
    raise SnError(3, f"unsupported dtype {t.dtype}")


def _torch_dtype(dt: int):
    return torch.float32 if dt == SN_F32 else torch.bfloat16


def _mat(t: torch.Tensor, name: str):
    if not t.is_cuda:
        raise SnError(2, f"{name} must be a device tensor")
    if t.dim() != 2:
        raise SnError(2, f"{name} must be a 2-D matrix")
    rows, cols = t.shape
    if cols > 1 and t.stride(1) != 1:
        raise SnError(2, f"{name} must be row-major (unit column stride)")
    ld = t.stride(0) if rows > 1 else cols
    return t.data_ptr(), rows, cols, max(ld, cols)


def _ids(t, name, n):
    if t is None:
        return None
    if not t.is_cuda or t.dtype != torch.int32 or t.dim() != 1 or t.shape[0] != n or \
            (n > 1 and t.stride(0) != 1):
        raise SnError(2, f"{name} must be a contiguous int32 device vector of length {n}")
    return t.data_ptr()


def _id_flag(err_flag, device):
    """(flag to pass to the C call, private flag or None): the caller's flag
    itself, or with checking on a private zeroed flag."""
    if not _CHECK_IDS:
        return err_flag, None
    own = torch.zeros(1, dtype=torch.int32, device=device)
    return own, own


def _id_check(own, caller, what: str):
    """With checking on (own = the private flag): pass the bits on to the
    caller's flag and raise if any id was out of range."""
    if own is None:
        return
    if caller is not None:
        caller.bitwise_or_(own)
    bits = int(own.item())  # waits for the call
    if bits:
        raise SnError(SN_ERR_INDEX, f"{what}: out-of-range ids were clamped (flag bits {bits}: "
                                    f"1 = token id, 2 = position id)")


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


class Basis:
    """A packed basis (the device buffer the codec calls read) plus its shape."""

    def __init__(self, packed: torch.Tensor, d: int, k: int, dt: int):
        self.packed, self.d, self.k, self.dt = packed, d, k, dt

    @property
    def ptr(self):
        return self.packed.data_ptr()


def sn_basis_packed_bytes(d: int, k: int, dt: int) -> int:
    return lib().sn_basis_packed_bytes(d, k, dt)


def sn_basis_pack(U: torch.Tensor, stream=None) -> Basis:
    """Pack U (d x k) for the codec calls; re-pack whenever U changes."""
    ptr, d, k, ldu = _mat(U, "U")
    dt = _dt(U)
    nbytes = sn_basis_packed_bytes(d, k, dt)
    if nbytes == 0:
        raise SnError(2, f"invalid basis shape {d} x {k}")
    packed = torch.empty(nbytes, dtype=torch.uint8, device=U.device)
    _check(lib().sn_basis_pack(ptr, d, k, ldu, dt, packed.data_ptr(), nbytes, _stream(stream)))
    return Basis(packed, d, k, dt)


def _tables(N, tok, E, pos, P, seq_len):
    e_ptr = vocab = lde = 0
    if E is not None:
        e_ptr, vocab, _, lde = _mat(E, "E")
    p_ptr = n_pos = ldp = 0
    if P is not None:
        p_ptr, n_pos, _, ldp = _mat(P, "P")
    tok_ptr = _ids(tok, "tok", N) if E is not None else None
    pos_ptr = _ids(pos, "pos", N) if P is not None else None
    return (tok_ptr, e_ptr or None, vocab, lde, pos_ptr, p_ptr or None, n_pos, ldp,
            int(seq_len or 0))


def _same_d(basis: Basis, d: int, *tables):
    if d != basis.d:
        raise SnError(2, f"matrix has {d} columns, basis has d = {basis.d}")
    for name, t in tables:
        if t is not None and (t.dim() != 2 or t.shape[1] != basis.d):
            raise SnError(2, f"{name} must have d = {basis.d} columns")


def _same_dtype(basis: Basis, *tensors):
    for name, t in tensors:
        if t is not None and _dt(t) != basis.dt:
            raise SnError(3, f"{name} has dtype {t.dtype}; the basis was packed as "
                             f"{_torch_dtype(basis.dt)}")


def _out_shape(out, shape, name):
    if tuple(out.shape) != tuple(shape):
        raise SnError(2, f"{name} must have shape {tuple(shape)}, got {tuple(out.shape)}")


def sn_compress(basis: Basis, X: torch.Tensor, tok=None, E=None, P=None, pos=None,
                seq_len=None, out=None, err_flag=None, stream=None) -> torch.Tensor:
    """C = (X - P[pos] - E[tok]) U."""
    xp, N, d, ldx = _mat(X, "X")
    _same_d(basis, d, ("E", E), ("P", P))
    if out is None:
        out = torch.empty((N, basis.k), dtype=_torch_dtype(basis.dt), device=X.device)
    _out_shape(out, (N, basis.k), "out")
    _same_dtype(basis, ("X", X), ("E", E), ("P", P), ("out", out))
    cp, _, _, ldc = _mat(out, "out")
    flag, own = _id_flag(err_flag, X.device)
    _check(lib().sn_compress(basis.ptr, basis.d, basis.k, basis.dt, xp, N, ldx,
                             *_tables(N, tok, E, pos, P, seq_len), cp, ldc,
                             None if flag is None else flag.data_ptr(), _stream(stream)))
    _id_check(own, err_flag, "sn_compress")
    return out


def sn_decompress(basis: Basis, C: torch.Tensor, tok=None, E=None, P=None, pos=None,
                  seq_len=None, out=None, err_flag=None, stream=None) -> torch.Tensor:
    """X = C U^T + P[pos] + E[tok]; with no tables, the gradient recovery C U^T."""
    cp, N, k, ldc = _mat(C, "C")
    if k != basis.k:
        raise SnError(2, f"C has {k} columns, basis has k = {basis.k}")
    _same_d(basis, basis.d, ("E", E), ("P", P))
    if out is None:
        out = torch.empty((N, basis.d), dtype=_torch_dtype(basis.dt), device=C.device)
    _out_shape(out, (N, basis.d), "out")
    _same_dtype(basis, ("C", C), ("E", E), ("P", P), ("out", out))
    xp, _, _, ldx = _mat(out, "out")
    flag, own = _id_flag(err_flag, C.device)
    _check(lib().sn_decompress(basis.ptr, basis.d, basis.k, basis.dt, cp, N, ldc,
                               *_tables(N, tok, E, pos, P, seq_len), xp, ldx,
                               None if flag is None else flag.data_ptr(),
                               _stream(stream)))
    _id_check(own, err_flag, "sn_decompress")
    return out


def sn_grad_compress(basis: Basis, G: torch.Tensor, out=None, stream=None) -> torch.Tensor:
    """Cg = G U."""
    gp, N, d, ldg = _mat(G, "G")
    _same_d(basis, d)
    if out is None:
        out = torch.empty((N, basis.k), dtype=_torch_dtype(basis.dt), device=G.device)
    _out_shape(out, (N, basis.k), "out")
    _same_dtype(basis, ("G", G), ("out", out))
    cp, _, _, ldc = _mat(out, "out")
    _check(lib().sn_grad_compress(basis.ptr, basis.d, basis.k, basis.dt, gp, N, ldg, cp, ldc,
                                  _stream(stream)))
    return out


class Projected:
    """Projected tables T_fixed U and P U (fp32, one device buffer) of a basis."""

    def __init__(self, buf: torch.Tensor, basis: Basis, vocab: int, n_pos: int):
        self.buf, self.basis, self.vocab, self.n_pos = buf, basis, vocab, n_pos

    @property
    def ptr(self):
        return self.buf.data_ptr() if self.buf.numel() else None

    def _view(self, off: int, rows: int) -> torch.Tensor:
        kp = 16 * ((self.basis.k + 15) // 16)
        return self.buf[off:off + rows * kp * 4].view(torch.float32).view(rows, kp)

    def tables(self):
        """(T_fixed U, P U) as fp32 views of shape (rows, 16 * ceil(k / 16))."""
        kp = 16 * ((self.basis.k + 15) // 16)
        off_pu = (self.vocab * kp * 4 + 255) // 256 * 256
        return self._view(0, self.vocab), self._view(off_pu, self.n_pos)


def sn_embed_projected_bytes(k: int, vocab: int, n_pos: int) -> int:
    return lib().sn_embed_projected_bytes(k, vocab, n_pos)


def sn_embed_project(basis: Basis, E=None, P=None, stream=None) -> Projected:
    """Build the projected tables T_fixed U and P U once per basis."""
    _same_d(basis, basis.d, ("E", E), ("P", P))
    _same_dtype(basis, ("E", E), ("P", P))
    e_ptr = vocab = lde = 0
    if E is not None:
        e_ptr, vocab, _, lde = _mat(E, "E")
    p_ptr = n_pos = ldp = 0
    if P is not None:
        p_ptr, n_pos, _, ldp = _mat(P, "P")
    nbytes = sn_embed_projected_bytes(basis.k, vocab, n_pos)
    dev = (E if E is not None else P).device if (E is not None or P is not None) else "cuda"
    buf = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    _check(lib().sn_embed_project(basis.ptr, basis.d, basis.k, basis.dt, e_ptr or None, vocab,
                                  lde, p_ptr or None, n_pos, ldp,
                                  buf.data_ptr() if nbytes else None, nbytes, _stream(stream)))
    return Projected(buf, basis, vocab, n_pos)


def sn_compress_projected(basis: Basis, X: torch.Tensor, proj: Projected, tok=None, pos=None,
                          seq_len=None, out=None, err_flag=None, stream=None) -> torch.Tensor:
    """C = X U - (P U)[pos] - (T_fixed U)[tok] against tables from sn_embed_project."""
    xp, N, d, ldx = _mat(X, "X")
    _same_d(basis, d)
    if proj.basis is not basis:
        raise SnError(2, "proj was built for another basis")
    if out is None:
        out = torch.empty((N, basis.k), dtype=_torch_dtype(basis.dt), device=X.device)
    _out_shape(out, (N, basis.k), "out")
    _same_dtype(basis, ("X", X), ("out", out))
    cp, _, _, ldc = _mat(out, "out")
    tok_ptr = _ids(tok, "tok", N) if proj.vocab else None
    pos_ptr = _ids(pos, "pos", N) if proj.n_pos else None
    flag, own = _id_flag(err_flag, X.device)
    _check(lib().sn_compress_projected(basis.ptr, basis.d, basis.k, basis.dt, xp, N, ldx,
                                       tok_ptr, pos_ptr, int(seq_len or 0), proj.ptr,
                                       proj.vocab, proj.n_pos, cp, ldc,
                                       None if flag is None else flag.data_ptr(),
                                       _stream(stream)))
    _id_check(own, err_flag, "sn_compress_projected")
    return out


def sn_project_weights_workspace_bytes(d: int, k: int, dt: int, m: int) -> int:
    return lib().sn_project_weights_workspace_bytes(d, k, dt, m)


def sn_project_weights(basis: Basis, W: torch.Tensor, workspace=None, stream=None) -> torch.Tensor:
    """W <- U (U^T W) in place; returns W."""
    wp, d, m, ldw = _mat(W, "W")
    if d != basis.d:
        raise SnError(2, f"W has {d} rows, basis has d = {basis.d}")
    _same_dtype(basis, ("W", W))
    need = sn_project_weights_workspace_bytes(basis.d, basis.k, basis.dt, m)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=W.device)
    if workspace.numel() < need or not workspace.is_cuda:
        raise SnError(9, f"workspace needs {need} device bytes")
    _check(lib().sn_project_weights(basis.ptr, d, basis.k, basis.dt, wp, m, ldw,
                                    workspace.data_ptr(), workspace.numel(), _stream(stream)))
    return W


def sn_project_weights_noalloc(basis: Basis, W: torch.Tensor, stream=None) -> torch.Tensor:
    """W <- U (U^T W) in place with the library's static scratch (no workspace,
    no allocation); returns W."""
    wp, d, m, ldw = _mat(W, "W")
    if d != basis.d:
        raise SnError(2, f"W has {d} rows, basis has d = {basis.d}")
    _same_dtype(basis, ("W", W))
    _check(lib().sn_project_weights_noalloc(basis.ptr, d, basis.k, basis.dt, wp, m, ldw,
                                            _stream(stream)))
    return W


def _i64_array(vals):
    arr = (ctypes.c_int64 * max(1, len(vals)))(*vals)
    return arr


def sn_project_weights_multi_workspace_bytes(d: int, k: int, dt: int, widths) -> int:
    m = _i64_array(widths)
    return lib().sn_project_weights_multi_workspace_bytes(d, k, dt, len(widths), m)


def sn_project_weights_multi(basis: Basis, Ws, workspace=None, stream=None):
    """W <- U (U^T W) in place for every matrix of the list Ws (each d x m_i),
    in one set of launches when the widths allow; returns Ws."""
    ptrs, widths, lds = [], [], []
    for i, W in enumerate(Ws):
        wp, d, m, ldw = _mat(W, f"W[{i}]")
        if d != basis.d:
            raise SnError(2, f"W[{i}] has {d} rows, basis has d = {basis.d}")
        _same_dtype(basis, (f"W[{i}]", W))
        ptrs.append(wp)
        widths.append(m)
        lds.append(ldw)
    need = sn_project_weights_multi_workspace_bytes(basis.d, basis.k, basis.dt, widths)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=Ws[0].device)
    if workspace.numel() < need or not workspace.is_cuda:
        raise SnError(9, f"workspace needs {need} device bytes")
    parr = (ctypes.c_void_p * max(1, len(ptrs)))(*ptrs)
    _check(lib().sn_project_weights_multi(basis.ptr, basis.d, basis.k, basis.dt, len(Ws), parr,
                                          _i64_array(widths), _i64_array(lds),
                                          workspace.data_ptr(), workspace.numel(), _stream(stream)))
    return Ws


class GrassmannState:
    """Accumulator of the subspace update (one device buffer, see include/sn.h):
    float64 [loss sum, K_L, L, K_S] and Y = sum_t G_t^T (G_t U) (d x k)."""

    HEAD = 256

    def __init__(self, buf: torch.Tensor, d: int, k: int):
        self.buf, self.d, self.k = buf, d, k

    @property
    def ptr(self):
        return self.buf.data_ptr()

    def scalars(self) -> torch.Tensor:
        """Device view of [loss sum, K_L, L, K_S] (float64)."""
        return self.buf[:32].view(torch.float64)

    def Y(self) -> torch.Tensor:
        """Device view of Y (d x k, float64)."""
        n = self.d * self.k * 8
        return self.buf[self.HEAD:self.HEAD + n].view(torch.float64).view(self.d, self.k)


def sn_grassmann_state_bytes(d: int, k: int) -> int:
    return lib().sn_grassmann_state_bytes(d, k)


def sn_grassmann_workspace_bytes(d: int, k: int, dt: int, N: int) -> int:
    return lib().sn_grassmann_workspace_bytes(d, k, dt, N)


def sn_grassmann_reset(state: GrassmannState, stream=None) -> GrassmannState:
    _check(lib().sn_grassmann_reset(state.ptr, state.d, state.k, _stream(stream)))
    return state


def sn_grassmann_state(basis: Basis, device="cuda", stream=None) -> GrassmannState:
    """A zeroed accumulator state for the basis's (d, k)."""
    nbytes = sn_grassmann_state_bytes(basis.d, basis.k)
    if nbytes == 0:
        raise SnError(8, f"no subspace-update state for d = {basis.d}, k = {basis.k}")
    buf = torch.empty(nbytes, dtype=torch.uint8, device=device)
    return sn_grassmann_reset(GrassmannState(buf, basis.d, basis.k), stream)


def _grass_ws(basis: Basis, N: int, workspace, device):
    need = sn_grassmann_workspace_bytes(basis.d, basis.k, basis.dt, N)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=device)
    if workspace.numel() < need or not workspace.is_cuda:
        raise SnError(9, f"workspace needs {need} device bytes")
    return workspace


def sn_grassmann_accumulate(basis: Basis, G: torch.Tensor, state: GrassmannState,
                            with_su: bool = True, want_cg: bool = False, out=None,
                            workspace=None, stream=None):
    """Add one iteration's gradient G (N x d) to the state: the off-subspace
    loss always, Y += G^T (G U) when with_su.  With want_cg (or out given)
    also returns the gradient coefficients G U as sn_grad_compress writes them."""
    gp, N, d, ldg = _mat(G, "G")
    _same_d(basis, d)
    if (state.d, state.k) != (basis.d, basis.k):
        raise SnError(2, "state was made for another basis shape")
    if out is None and want_cg:
        out = torch.empty((N, basis.k), dtype=_torch_dtype(basis.dt), device=G.device)
    cp = ldc = 0
    if out is not None:
        _out_shape(out, (N, basis.k), "out")
        _same_dtype(basis, ("out", out))
        cp, _, _, ldc = _mat(out, "out")
    _same_dtype(basis, ("G", G))
    ws = _grass_ws(basis, N, workspace, G.device)
    _check(lib().sn_grassmann_accumulate(basis.ptr, basis.d, basis.k, basis.dt, gp, N, ldg,
                                         cp or None, ldc, 1 if with_su else 0, state.ptr,
                                         ws.data_ptr(), ws.numel(), _stream(stream)))
    return out


def sn_grassmann_step(basis: Basis, state: GrassmannState, eta: float, out_dtype=None, out=None,
                      workspace=None, err_flag=None, stream=None) -> torch.Tensor:
    """U_new: one Riemannian gradient step of size eta on the accumulated loss,
    retracted by QR (diag(R) > 0).  out_dtype defaults to the basis dtype."""
    if (state.d, state.k) != (basis.d, basis.k):
        raise SnError(2, "state was made for another basis shape")
    tdt = out.dtype if out is not None else (out_dtype or _torch_dtype(basis.dt))
    if out is None:
        out = torch.empty((basis.d, basis.k), dtype=tdt, device=state.buf.device)
    _out_shape(out, (basis.d, basis.k), "out")
    up, _, _, ldu = _mat(out, "out")
    ws = _grass_ws(basis, 0, workspace, state.buf.device)
    _check(lib().sn_grassmann_step(basis.ptr, basis.d, basis.k, basis.dt, state.ptr, float(eta),
                                   up, ldu, _dt(out), ws.data_ptr(), ws.numel(),
                                   None if err_flag is None else err_flag.data_ptr(),
                                   _stream(stream)))
    return out


def sn_embed_lowrank_workspace_bytes(d: int, k: int, dt: int, N: int, vocab: int) -> int:
    return lib().sn_embed_lowrank_workspace_bytes(d, k, dt, N, vocab)


def sn_embed_lowrank_forward(basis: Basis, CS: torch.Tensor, tok: torch.Tensor, E=None, P=None,
                             pos=None, seq_len=None, out=None, err_flag=None, workspace=None,
                             stream=None) -> torch.Tensor:
    """X0 = P[pos] + E[tok] + CS[tok] U^T (the low-rank token table T_S = CS U^T)."""
    cp, vocab, k, ldcs = _mat(CS, "CS")
    if k != basis.k:
        raise SnError(2, f"CS has {k} columns, basis has k = {basis.k}")
    N = tok.shape[0]
    _same_d(basis, basis.d, ("E", E), ("P", P))
    if E is not None and E.shape[0] != vocab:
        raise SnError(2, "E and CS must have the same number of rows")
    if out is None:
        out = torch.empty((N, basis.d), dtype=_torch_dtype(basis.dt), device=CS.device)
    _out_shape(out, (N, basis.d), "out")
    _same_dtype(basis, ("CS", CS), ("E", E), ("P", P), ("out", out))
    xp, _, _, ldx = _mat(out, "out")
    tok_ptr = _ids(tok, "tok", N)
    _, e_ptr, _, lde, pos_ptr, p_ptr, n_pos, ldp, sl = _tables(N, tok, E, pos, P, seq_len)
    need = sn_embed_lowrank_workspace_bytes(basis.d, basis.k, basis.dt, N, vocab)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=CS.device)
    flag, own = _id_flag(err_flag, CS.device)
    _check(lib().sn_embed_lowrank_forward(basis.ptr, basis.d, basis.k, basis.dt, cp, vocab, ldcs,
                                          tok_ptr, e_ptr, lde, pos_ptr, p_ptr, n_pos, ldp, sl,
                                          xp, N, ldx,
                                          None if flag is None else flag.data_ptr(),
                                          workspace.data_ptr(), workspace.numel(),
                                          _stream(stream)))
    _id_check(own, err_flag, "sn_embed_lowrank_forward")
    return out


def sn_embed_lowrank_backward(basis: Basis, dX0: torch.Tensor, tok: torch.Tensor, gCS: torch.Tensor,
                              err_flag=None, workspace=None, stream=None) -> torch.Tensor:
    """gCS += scatter over tok of dX0 U (float32 gCS, vocab x k); returns gCS."""
    gp, N, d, ldg = _mat(dX0, "dX0")
    _same_d(basis, d)
    _same_dtype(basis, ("dX0", dX0))
    cp, vocab, k, ldgc = _mat(gCS, "gCS")
    if k != basis.k or gCS.dtype != torch.float32:
        raise SnError(2, f"gCS must be float32 with k = {basis.k} columns")
    tok_ptr = _ids(tok, "tok", N)
    need = sn_embed_lowrank_workspace_bytes(basis.d, basis.k, basis.dt, N, vocab)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dX0.device)
    flag, own = _id_flag(err_flag, dX0.device)
    _check(lib().sn_embed_lowrank_backward(basis.ptr, basis.d, basis.k, basis.dt, gp, N, ldg,
                                           tok_ptr, vocab, cp, ldgc,
                                           None if flag is None else flag.data_ptr(),
                                           workspace.data_ptr(), workspace.numel(),
                                           _stream(stream)))
    _id_check(own, err_flag, "sn_embed_lowrank_backward")
    return gCS


def sn_adamw_workspace_bytes(rows: int, cols: int) -> int:
    return lib().sn_adamw_workspace_bytes(rows, cols)


def sn_adamw_step(W: torch.Tensor, G: torch.Tensor, M: torch.Tensor, V: torch.Tensor, t: int,
                  lr: float, beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8,
                  weight_decay: float = 0.0, subspace: bool = True, workspace=None,
                  stream=None) -> torch.Tensor:
    """One AdamW step in place on W (rows x cols, stored [out, in]) with fp32
    moments M, V; subspace=True uses the column-constant rate of Sec. 5."""
    wp, rows, cols, ldw = _mat(W, "W")
    gp, gr, gc, ldg = _mat(G, "G")
    mp, mr, mc, ldm = _mat(M, "M")
    vp, vr, vc, ldv = _mat(V, "V")
    if (gr, gc) != (rows, cols) or (mr, mc) != (rows, cols) or (vr, vc) != (rows, cols):
        raise SnError(2, "W, G, M and V must have the same shape")
    if ldv != ldm:
        raise SnError(2, "M and V must share a row stride")
    if M.dtype != torch.float32 or V.dtype != torch.float32:
        raise SnError(3, "M and V must be float32")
    dt = _dt(W)
    if _dt(G) != dt:
        raise SnError(3, "W and G must have the same dtype")
    need = sn_adamw_workspace_bytes(rows, cols) if subspace else 0
    if need and workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=W.device)
    if need and (workspace.numel() < need or not workspace.is_cuda):
        raise SnError(9, f"workspace needs {need} device bytes")
    _check(lib().sn_adamw_step(wp, ldw, gp, ldg, dt, mp, vp, ldm, rows, cols, int(t), float(lr),
                               float(beta1), float(beta2), float(eps), float(weight_decay),
                               1 if subspace else 0,
                               workspace.data_ptr() if need else None, need,
                               _stream(stream)))
    return W


def sn_version() -> str:
    return lib().sn_version().decode()
