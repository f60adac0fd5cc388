"""Python binding of libckkslinear.so (gfx950 CKKS ct x pt linear layer).

Argument marshalling only: each function has the name of the C entry point it
calls (declared in include/ckks_linear.h), takes torch tensors for device
buffers and passes their data pointers and the current HIP stream through.
All arithmetic runs in the library's HIP kernels; there is no fallback.  The
binding checks that every tensor is a contiguous cuda tensor of the right
element size and at least as large as the shape the call implies, so that no
kernel is launched over a buffer too small for its grid.

Importing this package raises ImportError when the library has not been
built (``python paper_2606_17421_amd/build.py`` or ``__graft_entry__.build()``).
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libckkslinear.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build the HIP library first "
                      "(python paper_2606_17421_amd/build.py)")

# torch (device memory and streams) brings its HIP runtime up first: loaded
# before it, the library's runtime finds no devices in a later torch session.
import torch  # noqa: E402,F401

_lib = ctypes.CDLL(LIB_PATH)

CKKS_OK = 0
CKKS_E_INVALID_ARG = -1
CKKS_E_UNSUPPORTED = -2
CKKS_E_HIP = -3
CKKS_E_WORKSPACE = -4

CKKS_OP_MAC_SCALAR = 1
CKKS_OP_RESCALE = 2
CKKS_OP_ENCODE_POLY = 3
CKKS_OP_ROTATE = 4

CKKS_MAC_AUTO = 0
CKKS_MAC_VALU = 1
CKKS_MAC_MFMA = 2

_u32, _i32, _sz, _vp, _dbl = ctypes.c_uint32, ctypes.c_int, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_double
_SIGS = {
    "ckks_ctx_create": (_i32, [ctypes.POINTER(_vp), _u32, _u32, ctypes.POINTER(_u32), _i32]),
    "ckks_ctx_destroy": (_i32, [_vp]),
    "ckks_ctx_moduli": (_i32, [_vp, ctypes.POINTER(_u32)]),
    "ckks_ctx_roots": (_i32, [_vp, ctypes.POINTER(_u32)]),
    "ckks_ctx_info": (_i32, [_vp, ctypes.POINTER(_u32), ctypes.POINTER(_u32)]),
    "ckks_ctx_set_mac_algo": (_i32, [_vp, _i32]),
    "ckks_ntt": (_i32, [_vp, _vp, _u32, _u32, _vp]),
    "ckks_intt": (_i32, [_vp, _vp, _u32, _u32, _vp]),
    "ckks_linear_encode_scalar": (_i32, [_vp, _vp, _u32, _u32, _u32, _dbl, _vp, _vp]),
    "ckks_linear_encode_poly": (_i32, [_vp, _vp, _u32, _u32, _dbl, _vp, _vp]),
    "ckks_linear_mac_scalar": (_i32, [_vp, _vp, _vp, _vp, _u32, _u32, _u32, _vp, _sz, _vp]),
    "ckks_linear_mac_scalar_noalloc": (_i32, [_vp, _vp, _vp, _vp, _u32, _u32, _u32, _vp]),
    "ckks_linear_mac_poly": (_i32, [_vp, _vp, _vp, _vp, _u32, _u32, _u32, _vp]),
    "ckks_rescale": (_i32, [_vp, _vp, _vp, _u32, _u32, _vp, _sz, _vp]),
    "ckks_encrypt": (_i32, [_vp, _vp, _vp, _vp, _vp, _u32, _u32, _vp, _vp]),
    "ckks_decrypt": (_i32, [_vp, _vp, _vp, _u32, _u32, _vp, _vp]),
    "ckks_refresh": (_i32, [_vp, _vp, _u32, _vp, _vp, _vp, _u32, _u32, _vp, _vp]),
    "ckks_automorphism": (_i32, [_vp, _vp, _u32, _u32, _vp, _vp]),
    "ckks_keygen_rotation": (_i32, [_vp, _vp, _u32, _u32, _u32, _vp, _vp, _vp, _vp]),
    "ckks_rotate": (_i32, [_vp, _vp, _u32, _u32, _u32, _i32, _vp, _vp, _sz, _vp, _vp]),
    "ckks_linear_bsgs": (_i32, [_vp, _vp, _vp, _u32, _u32, _u32, _vp, _vp, _sz, _vp, _vp]),
    "ckks_bsgs_workspace_bytes": (_sz, [_vp, _u32, _u32, _u32]),
    "ckks_add": (_i32, [_vp, _vp, _vp, _u32, _u32, _vp, _vp]),
    "ckks_workspace_bytes": (_sz, [_vp, _i32, _u32, _u32, _u32]),
    "ckks_rescaled_scale": (_dbl, [_vp, _dbl, _u32]),
    "ckks_last_error": (ctypes.c_char_p, []),
}
for _name, (_res, _args) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args

EXPORTS = tuple(_SIGS)


class CkksError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        msg = _lib.ckks_last_error().decode(errors="replace")
        super().__init__(f"{where} failed with status {code}: {msg}")


def _check(rc: int, where: str) -> None:
    if rc != CKKS_OK:
        raise CkksError(rc, where)


def _stream(stream):
    import torch
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t, name: str, nbytes: int, itemsize: int, allow_none: bool = False):
    """Data pointer of a contiguous cuda tensor holding at least nbytes."""
    if t is None:
        if allow_none or nbytes == 0:
            return None
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a cuda tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.element_size() != itemsize:
        raise ValueError(f"{name} must have {itemsize}-byte elements (got {t.dtype})")
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{name} holds {have} bytes, needs {nbytes}")
    return ctypes.c_void_p(t.data_ptr())


class Context:
    """Owns a ckks_ctx (modulus chain + device tables) on one device."""

    def __init__(self, log_n: int, limbs: int, moduli=None, device: int = 0):
        h = ctypes.c_void_p()
        arr = None
        if moduli is not None:
            arr = (_u32 * limbs)(*[int(m) for m in moduli])
        _check(_lib.ckks_ctx_create(ctypes.byref(h), log_n, limbs, arr, device), "ckks_ctx_create")
        self.handle = h
        self.log_n, self.n, self.limbs, self.device = log_n, 1 << log_n, limbs, device
        buf = (_u32 * limbs)()
        _check(_lib.ckks_ctx_moduli(h, buf), "ckks_ctx_moduli")
        self.moduli = tuple(int(x) for x in buf)
        _check(_lib.ckks_ctx_roots(h, buf), "ckks_ctx_roots")
        self.roots = tuple(int(x) for x in buf)

    def close(self) -> None:
        if self.handle:
            _check(_lib.ckks_ctx_destroy(self.handle), "ckks_ctx_destroy")
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def ckks_ctx_create(log_n: int, limbs: int, moduli=None, device: int = 0) -> Context:
    return Context(log_n, limbs, moduli, device)


def ckks_ctx_destroy(ctx: Context) -> None:
    ctx.close()


def ckks_ctx_set_mac_algo(ctx: Context, algo: int) -> None:
    _check(_lib.ckks_ctx_set_mac_algo(ctx.handle, algo), "ckks_ctx_set_mac_algo")


def ckks_ntt(ctx: Context, polys, count: int, limbs: int, stream=None) -> None:
    nb = count * limbs * ctx.n * 4
    _check(_lib.ckks_ntt(ctx.handle, _ptr(polys, "polys", nb, 4), count, limbs, _stream(stream)), "ckks_ntt")


def ckks_intt(ctx: Context, polys, count: int, limbs: int, stream=None) -> None:
    nb = count * limbs * ctx.n * 4
    _check(_lib.ckks_intt(ctx.handle, _ptr(polys, "polys", nb, 4), count, limbs, _stream(stream)), "ckks_intt")


def ckks_linear_encode_scalar(ctx: Context, w, d_out: int, d_in: int, limbs: int, scale: float, w_enc,
                              stream=None) -> None:
    cnt = d_out * d_in
    _check(_lib.ckks_linear_encode_scalar(ctx.handle, _ptr(w, "w", cnt * 8, 8), d_out, d_in, limbs, float(scale),
                                          _ptr(w_enc, "w_enc", cnt * limbs * 4, 4), _stream(stream)),
           "ckks_linear_encode_scalar")


def ckks_linear_encode_poly(ctx: Context, slots, count: int, limbs: int, scale: float, pt, stream=None) -> None:
    _check(_lib.ckks_linear_encode_poly(ctx.handle, _ptr(slots, "slots", count * (ctx.n // 2) * 8, 8), count, limbs,
                                        float(scale), _ptr(pt, "pt", count * limbs * ctx.n * 4, 4), _stream(stream)),
           "ckks_linear_encode_poly")


def ckks_workspace_bytes(ctx: Context, op: int, a: int, b: int, limbs: int) -> int:
    v = _lib.ckks_workspace_bytes(ctx.handle, op, a, b, limbs)
    if v == ctypes.c_size_t(-1).value:
        raise ValueError("invalid workspace request")
    return int(v)


def ckks_linear_mac_scalar(ctx: Context, w_enc, ct_in, ct_out, d_out: int, d_in: int, limbs: int,
                           workspace=None, workspace_bytes: int | None = None, stream=None) -> None:
    ct_words = 2 * limbs * ctx.n if d_out else 0          # d_out == 0: nothing is touched
    wb = workspace.numel() * workspace.element_size() if workspace is not None else 0
    if workspace_bytes is None:
        workspace_bytes = wb
    elif workspace_bytes > wb:
        raise ValueError("workspace_bytes exceeds the workspace tensor")
    ws = _ptr(workspace, "workspace", 0, workspace.element_size(), True) if workspace is not None else None
    _check(_lib.ckks_linear_mac_scalar(
        ctx.handle, _ptr(w_enc, "w_enc", d_out * d_in * limbs * 4, 4),
        _ptr(ct_in, "ct_in", d_in * ct_words * 4, 4), _ptr(ct_out, "ct_out", d_out * ct_words * 4, 4),
        d_out, d_in, limbs, ws, workspace_bytes, _stream(stream)), "ckks_linear_mac_scalar")


def ckks_linear_mac_scalar_noalloc(ctx: Context, w_enc, ct_in, ct_out, d_out: int, d_in: int, limbs: int,
                                   stream=None) -> None:
    """ckks_linear_mac_scalar with the library's own per-GPU scratch as workspace."""
    ct_words = 2 * limbs * ctx.n if d_out else 0
    _check(_lib.ckks_linear_mac_scalar_noalloc(
        ctx.handle, _ptr(w_enc, "w_enc", d_out * d_in * limbs * 4, 4),
        _ptr(ct_in, "ct_in", d_in * ct_words * 4, 4), _ptr(ct_out, "ct_out", d_out * ct_words * 4, 4),
        d_out, d_in, limbs, _stream(stream)), "ckks_linear_mac_scalar_noalloc")


NOALLOC_SCRATCH_BYTES = 64 << 20


def ckks_linear_mac_poly(ctx: Context, pt, ct_in, ct_out, d_out: int, d_in: int, limbs: int, stream=None) -> None:
    ct_words = 2 * limbs * ctx.n if d_out else 0
    _check(_lib.ckks_linear_mac_poly(
        ctx.handle, _ptr(pt, "pt", d_out * d_in * limbs * ctx.n * 4, 4),
        _ptr(ct_in, "ct_in", d_in * ct_words * 4, 4), _ptr(ct_out, "ct_out", d_out * ct_words * 4, 4),
        d_out, d_in, limbs, _stream(stream)), "ckks_linear_mac_poly")


def ckks_rescale(ctx: Context, ct_in, ct_out, count: int, limbs: int, workspace=None,
                 workspace_bytes: int | None = None, stream=None) -> None:
    wb = workspace.numel() * workspace.element_size() if workspace is not None else 0
    if workspace_bytes is None:
        workspace_bytes = wb
    elif workspace_bytes > wb:
        raise ValueError("workspace_bytes exceeds the workspace tensor")
    ws = _ptr(workspace, "workspace", 0, workspace.element_size(), True) if workspace is not None else None
    _check(_lib.ckks_rescale(
        ctx.handle, _ptr(ct_in, "ct_in", count * 2 * limbs * ctx.n * 4, 4),
        _ptr(ct_out, "ct_out", count * 2 * (limbs - 1) * ctx.n * 4, 4), count, limbs, ws, workspace_bytes,
        _stream(stream)), "ckks_rescale")


def ckks_encrypt(ctx: Context, pt, s_ntt, a, e, count: int, limbs: int, ct, stream=None) -> None:
    """pt may be None (zero plaintext); e holds int32 error coefficients [count][N]."""
    rows = count * limbs * ctx.n * 4
    _check(_lib.ckks_encrypt(
        ctx.handle, _ptr(pt, "pt", rows, 4, True), _ptr(s_ntt, "s_ntt", limbs * ctx.n * 4 if count else 0, 4),
        _ptr(a, "a", rows, 4), _ptr(e, "e", count * ctx.n * 4, 4), count, limbs, _ptr(ct, "ct", 2 * rows, 4),
        _stream(stream)), "ckks_encrypt")


def ckks_decrypt(ctx: Context, ct, s_ntt, count: int, limbs: int, m, stream=None) -> None:
    rows = count * limbs * ctx.n * 4
    _check(_lib.ckks_decrypt(
        ctx.handle, _ptr(ct, "ct", 2 * rows, 4), _ptr(s_ntt, "s_ntt", limbs * ctx.n * 4 if count else 0, 4),
        count, limbs, _ptr(m, "m", rows, 4), _stream(stream)), "ckks_decrypt")


def ckks_refresh(ctx: Context, ct_in, limbs_in: int, s_ntt, a, e, count: int, limbs_out: int, ct_out,
                 stream=None) -> None:
    n4 = ctx.n * 4
    _check(_lib.ckks_refresh(
        ctx.handle, _ptr(ct_in, "ct_in", count * 2 * limbs_in * n4, 4), limbs_in,
        _ptr(s_ntt, "s_ntt", max(limbs_out, 2) * n4 if count else 0, 4), _ptr(a, "a", count * limbs_out * n4, 4),
        _ptr(e, "e", count * n4, 4), count, limbs_out, _ptr(ct_out, "ct_out", count * 2 * limbs_out * n4, 4),
        _stream(stream)), "ckks_refresh")


def ckks_automorphism(ctx: Context, src, rows: int, galois: int, out, stream=None) -> None:
    nb = rows * ctx.n * 4
    _check(_lib.ckks_automorphism(ctx.handle, _ptr(src, "in", nb, 4), rows, galois, _ptr(out, "out", nb, 4),
                                  _stream(stream)), "ckks_automorphism")


def ckks_keygen_rotation(ctx: Context, s_ntt, r0: int, r_step: int, count: int, a, e, ksk, stream=None) -> None:
    L, n4 = ctx.limbs, ctx.n * 4
    lk = L - 1
    _check(_lib.ckks_keygen_rotation(
        ctx.handle, _ptr(s_ntt, "s_ntt", L * n4 if count else 0, 4), r0 % (ctx.n // 2), r_step % (ctx.n // 2), count,
        _ptr(a, "a", count * lk * L * n4, 4), _ptr(e, "e", count * lk * n4, 4),
        _ptr(ksk, "ksk", count * lk * 2 * L * n4, 4), _stream(stream)), "ckks_keygen_rotation")


def rotate_workspace_bytes(ctx: Context, count: int, hoisted: bool) -> int:
    return int(_lib.ckks_workspace_bytes(ctx.handle, CKKS_OP_ROTATE, count, int(hoisted), ctx.limbs - 1))


def ckks_rotate(ctx: Context, ct_in, count: int, r0: int, r_step: int, hoisted: bool, ksk, workspace, ct_out,
                stream=None) -> None:
    L, n4 = ctx.limbs, ctx.n * 4
    lk = L - 1
    wb = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(_lib.ckks_rotate(
        ctx.handle, _ptr(ct_in, "ct_in", (1 if hoisted else count) * 2 * lk * n4, 4), count, r0 % (ctx.n // 2),
        r_step % (ctx.n // 2), int(hoisted), _ptr(ksk, "ksk", count * lk * 2 * L * n4, 4),
        _ptr(workspace, "workspace", 0, workspace.element_size() if workspace is not None else 1, allow_none=True),
        wb, _ptr(ct_out, "ct_out", count * 2 * lk * n4, 4), _stream(stream)), "ckks_rotate")


def bsgs_workspace_bytes(ctx: Context, count: int, n1: int, n2: int) -> int:
    return int(_lib.ckks_bsgs_workspace_bytes(ctx.handle, count, n1, n2))


def ckks_linear_bsgs(ctx: Context, pt, ct_in, count: int, n1: int, n2: int, ksk, workspace, ct_out,
                     stream=None) -> None:
    L, n4 = ctx.limbs, ctx.n * 4
    lk = L - 1
    wb = workspace.numel() * workspace.element_size() if workspace is not None else 0
    keys = n1 + n2 - 2
    _check(_lib.ckks_linear_bsgs(
        ctx.handle, _ptr(pt, "pt", n1 * n2 * lk * n4, 4), _ptr(ct_in, "ct_in", count * 2 * lk * n4, 4), count, n1, n2,
        _ptr(ksk, "ksk", keys * lk * 2 * L * n4, 4, allow_none=keys == 0),
        _ptr(workspace, "workspace", 0, workspace.element_size() if workspace is not None else 1, allow_none=True),
        wb, _ptr(ct_out, "ct_out", count * 2 * (lk - 1) * n4, 4), _stream(stream)), "ckks_linear_bsgs")


def ckks_add(ctx: Context, ct_a, ct_b, count: int, limbs: int, ct_out, stream=None) -> None:
    nb = count * 2 * limbs * ctx.n * 4
    _check(_lib.ckks_add(ctx.handle, _ptr(ct_a, "ct_a", nb, 4), _ptr(ct_b, "ct_b", nb, 4), count, limbs,
                         _ptr(ct_out, "ct_out", nb, 4), _stream(stream)), "ckks_add")


def empty_workspace(nbytes: int, device: int = 0):
    """Device workspace of at least nbytes (torch's allocations are 256-byte aligned)."""
    import torch
    return torch.empty((max(nbytes, 1) + 3) // 4, dtype=torch.int32, device=f"cuda:{device}")


def ckks_rescaled_scale(ctx: Context, scale_in: float, limbs: int) -> float:
    return float(_lib.ckks_rescaled_scale(ctx.handle, float(scale_in), limbs))


def ckks_last_error() -> str:
    return _lib.ckks_last_error().decode(errors="replace")


# ---- host <-> device helpers (uint32 residues travel as int32 tensors) ----

def to_device(a, device: int = 0):
    """numpy uint32/float64 array -> contiguous cuda tensor with the same bits."""
    import numpy as np
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint32:
        a = a.view(np.int32)
    return torch.from_numpy(a).to(f"cuda:{device}")


def to_host_u32(t):
    """cuda int32 tensor -> numpy uint32 array with the same bits."""
    import numpy as np
    return t.cpu().numpy().view(np.uint32)


def empty_u32(shape, device: int = 0):
    import torch
    return torch.empty(shape, dtype=torch.int32, device=f"cuda:{device}")
