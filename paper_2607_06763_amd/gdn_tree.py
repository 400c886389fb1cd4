"""Python binding of libgdntree (include/gdn_tree.h): argument marshalling only.

Every step of the path runs in the HIP kernels of ``libgdntree.so``; this
module checks tensor shapes, dtypes and devices, passes raw device pointers
and the current HIP stream through ctypes, and turns error codes into
exceptions.  There is no fallback: if the library is missing the calls raise.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgdntree.so")

GDN_OK, GDN_EINVAL, GDN_EUNSUPPORTED, GDN_EHIP = 0, -1, -2, -3
GDN_F32, GDN_BF16 = 0, 1
TREE_OK, TREE_NO_ROOT, TREE_MULTI_ROOT, TREE_BAD_PARENT, TREE_CYCLE, TREE_BAD_ACCEPTED = range(6)
MAX_T = 512

EXPORTS = ("gdn_tree_meta_bytes", "gdn_tree_prepare", "gdn_tree_verify",
           "gdn_tree_verify_noalloc", "gdn_tree_verify_chunked", "gdn_tree_commit",
           "gdn_tree_step", "gdn_last_error", "gdn_version")
NOALLOC_SCRATCH_BYTES = 64 << 20  # GDN_NOALLOC_SCRATCH_BYTES of gdn_tree.h


class GdnError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"gdntree error {code}: {msg}")
        self.code = code


class Dims(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("T", ctypes.c_int32), ("Hk", ctypes.c_int32),
                ("Hv", ctypes.c_int32), ("dk", ctypes.c_int32), ("dv", ctypes.c_int32),
                ("in_dtype", ctypes.c_int32), ("scale", ctypes.c_float)]

    @property
    def C(self) -> int:
        return 2 * self.Hk * self.dk + self.Hv * self.dv

    def __repr__(self):
        return (f"Dims(B={self.B}, T={self.T}, Hk={self.Hk}, Hv={self.Hv}, dk={self.dk}, "
                f"dv={self.dv}, in_dtype={self.in_dtype}, scale={self.scale})")


def make_dims(B, T, Hk, Hv, dk, dv, in_dtype="bf16", scale=0.0) -> Dims:
    dt = GDN_BF16 if in_dtype in ("bf16", GDN_BF16) else GDN_F32
    return Dims(B, T, Hk, Hv, dk, dv, dt, float(scale))


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"libgdntree.so not built ({LIB_PATH}); run __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32 = ctypes.c_void_p, ctypes.c_int32
        L.gdn_tree_meta_bytes.restype = ctypes.c_size_t
        L.gdn_tree_meta_bytes.argtypes = [i32, i32]
        L.gdn_tree_prepare.restype = ctypes.c_int
        L.gdn_tree_prepare.argtypes = [ctypes.POINTER(Dims), vp, vp, vp, vp]
        L.gdn_tree_verify.restype = ctypes.c_int
        L.gdn_tree_verify.argtypes = [ctypes.POINTER(Dims)] + [vp] * 11
        L.gdn_tree_verify_noalloc.restype = ctypes.c_int
        L.gdn_tree_verify_noalloc.argtypes = [ctypes.POINTER(Dims)] + [vp] * 11
        L.gdn_tree_verify_chunked.restype = ctypes.c_int
        L.gdn_tree_verify_chunked.argtypes = [ctypes.POINTER(Dims)] + [vp] * 11
        L.gdn_tree_commit.restype = ctypes.c_int
        L.gdn_tree_commit.argtypes = [ctypes.POINTER(Dims)] + [vp] * 12
        L.gdn_tree_step.restype = ctypes.c_int
        L.gdn_tree_step.argtypes = [ctypes.POINTER(Dims)] + [vp] * 20
        L.gdn_last_error.restype = ctypes.c_char_p
        L.gdn_last_error.argtypes = []
        L.gdn_version.restype = ctypes.c_char_p
        L.gdn_version.argtypes = []
        _lib = L
    return _lib


def last_error() -> str:
    return lib().gdn_last_error().decode()


def _check(rc: int) -> None:
    if rc != GDN_OK:
        raise GdnError(rc, last_error())


def meta_bytes(B: int, T: int) -> int:
    return int(lib().gdn_tree_meta_bytes(B, T))


# ---------------------------------------------------------------------------
# tensor marshalling
# ---------------------------------------------------------------------------
def _ptr(t, shape, dtype, name, allow_none=False):
    import torch
    if t is None:
        if allow_none:
            return None
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name}: must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if t.data_ptr() % 16:
        raise ValueError(f"{name}: must be 16-byte aligned")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _in_dtype(d: Dims):
    import torch
    return torch.bfloat16 if d.in_dtype == GDN_BF16 else torch.float32


def prepare(d: Dims, parent, meta, tree_status=None, stream=None) -> None:
    """gdn_tree_prepare: parent int32 [B][T] -> meta (uint8, meta_bytes) and
    tree_status int32 [B] (optional)."""
    import torch
    _check(lib().gdn_tree_prepare(
        ctypes.byref(d), _ptr(parent, (d.B, d.T), torch.int32, "parent"),
        _ptr(meta, (meta_bytes(d.B, d.T),), torch.uint8, "meta"),
        _ptr(tree_status, (d.B,), torch.int32, "tree_status", allow_none=True), _stream(stream)))


def verify(d: Dims, meta, q, k, v, alpha, beta, conv_w, conv_state, S0, out, stream=None,
           chunked: bool = False, noalloc: bool = False) -> None:
    """gdn_tree_verify (or gdn_tree_verify_chunked, the paper's chunked
    form, or gdn_tree_verify_noalloc, which allocates nothing): per-node
    outputs out fp32 [B][T][Hv][dv]."""
    import torch
    f32, it = torch.float32, _in_dtype(d)
    if chunked and noalloc:
        raise ValueError("chunked and noalloc are separate entry points")
    fn = (lib().gdn_tree_verify_chunked if chunked else
          lib().gdn_tree_verify_noalloc if noalloc else lib().gdn_tree_verify)
    _check(fn(
        ctypes.byref(d), _ptr(meta, (meta_bytes(d.B, d.T),), torch.uint8, "meta"),
        _ptr(q, (d.B, d.T, d.Hk, d.dk), it, "q"), _ptr(k, (d.B, d.T, d.Hk, d.dk), it, "k"),
        _ptr(v, (d.B, d.T, d.Hv, d.dv), it, "v"), _ptr(alpha, (d.B, d.T, d.Hv), it, "alpha"),
        _ptr(beta, (d.B, d.T, d.Hv), it, "beta"), _ptr(conv_w, (d.C, 4), f32, "conv_w"),
        _ptr(conv_state, (d.B, 3, d.C), f32, "conv_state"),
        _ptr(S0, (d.B, d.Hv, d.dv, d.dk), f32, "S0"),
        _ptr(out, (d.B, d.T, d.Hv, d.dv), f32, "out"), _stream(stream)))


def commit(d: Dims, meta, accepted, q, k, v, alpha, beta, conv_w, conv_state, S,
           commit_status=None, stream=None) -> None:
    """gdn_tree_commit: in-place update of S [B][Hv][dv][dk] and conv_state
    [B][3][C] for the accepted slot of each sequence."""
    import torch
    f32, it = torch.float32, _in_dtype(d)
    _check(lib().gdn_tree_commit(
        ctypes.byref(d), _ptr(meta, (meta_bytes(d.B, d.T),), torch.uint8, "meta"),
        _ptr(accepted, (d.B,), torch.int32, "accepted"),
        _ptr(q, (d.B, d.T, d.Hk, d.dk), it, "q"), _ptr(k, (d.B, d.T, d.Hk, d.dk), it, "k"),
        _ptr(v, (d.B, d.T, d.Hv, d.dv), it, "v"), _ptr(alpha, (d.B, d.T, d.Hv), it, "alpha"),
        _ptr(beta, (d.B, d.T, d.Hv), it, "beta"), _ptr(conv_w, (d.C, 4), f32, "conv_w"),
        _ptr(conv_state, (d.B, 3, d.C), f32, "conv_state"),
        _ptr(S, (d.B, d.Hv, d.dv, d.dk), f32, "S"),
        _ptr(commit_status, (d.B,), torch.int32, "commit_status", allow_none=True),
        _stream(stream)))


def step(d: Dims, prev_meta, prev_accepted, prev_q, prev_k, prev_v, prev_alpha, prev_beta,
         commit_status, meta, q, k, v, alpha, beta, conv_w, conv_state, conv_state_out, S, out,
         stream=None) -> None:
    """gdn_tree_step: commit of the previous step's accepted node, then
    verification of the current tree; S is updated in place, the committed
    conv state goes to conv_state_out (conv_state is read-only)."""
    import torch
    f32, it = torch.float32, _in_dtype(d)
    mb = (meta_bytes(d.B, d.T),)
    qk, vs, gs = (d.B, d.T, d.Hk, d.dk), (d.B, d.T, d.Hv, d.dv), (d.B, d.T, d.Hv)
    _check(lib().gdn_tree_step(
        ctypes.byref(d), _ptr(prev_meta, mb, torch.uint8, "prev_meta"),
        _ptr(prev_accepted, (d.B,), torch.int32, "prev_accepted"),
        _ptr(prev_q, qk, it, "prev_q"), _ptr(prev_k, qk, it, "prev_k"),
        _ptr(prev_v, vs, it, "prev_v"), _ptr(prev_alpha, gs, it, "prev_alpha"),
        _ptr(prev_beta, gs, it, "prev_beta"),
        _ptr(commit_status, (d.B,), torch.int32, "commit_status", allow_none=True),
        _ptr(meta, mb, torch.uint8, "meta"), _ptr(q, qk, it, "q"), _ptr(k, qk, it, "k"),
        _ptr(v, vs, it, "v"), _ptr(alpha, gs, it, "alpha"), _ptr(beta, gs, it, "beta"),
        _ptr(conv_w, (d.C, 4), f32, "conv_w"),
        _ptr(conv_state, (d.B, 3, d.C), f32, "conv_state"),
        _ptr(conv_state_out, (d.B, 3, d.C), f32, "conv_state_out"),
        _ptr(S, (d.B, d.Hv, d.dv, d.dk), f32, "S"),
        _ptr(out, (d.B, d.T, d.Hv, d.dv), f32, "out"), _stream(stream)))


# ---------------------------------------------------------------------------
# workload upload (host arrays -> device tensors)
# ---------------------------------------------------------------------------
class DeviceTree:
    """Device copies of one workload's tensors plus meta/out/status buffers."""

    def __init__(self, w, device="cuda", scale: float = 0.0):
        import numpy as np
        import torch

        def up(a):
            a = np.ascontiguousarray(a)
            if a.dtype == np.uint16:  # bf16 bit patterns
                return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device)
            return torch.from_numpy(a).to(device)

        self.dims = make_dims(w.B, w.T, w.Hk, w.Hv, w.dk, w.dv, w.in_dtype, scale)
        self.parent = up(w.parent.astype(np.int32))
        self.q, self.k, self.v = up(w.q), up(w.k), up(w.v)
        self.alpha, self.beta = up(w.alpha), up(w.beta)
        self.S0 = up(w.S0.astype(np.float32))
        self.conv_w = up(w.conv_w.astype(np.float32))
        self.conv_state = up(w.conv_state.astype(np.float32))
        self.accepted = up(w.accepted.astype(np.int32))
        self.meta = torch.zeros(meta_bytes(w.B, w.T), dtype=torch.uint8, device=device)
        self.tree_status = torch.full((w.B,), -7, dtype=torch.int32, device=device)
        self.commit_status = torch.full((w.B,), -7, dtype=torch.int32, device=device)
        self.out = torch.full((w.B, w.T, w.Hv, w.dv), float("nan"), dtype=torch.float32,
                              device=device)

    def prepare(self, stream=None):
        prepare(self.dims, self.parent, self.meta, self.tree_status, stream)

    def verify(self, S0=None, conv_state=None, out=None, stream=None, chunked=False,
               noalloc=False):
        verify(self.dims, self.meta, self.q, self.k, self.v, self.alpha, self.beta, self.conv_w,
               self.conv_state if conv_state is None else conv_state,
               self.S0 if S0 is None else S0, self.out if out is None else out, stream, chunked,
               noalloc)

    def commit(self, S, conv_state, accepted=None, stream=None):
        commit(self.dims, self.meta, self.accepted if accepted is None else accepted, self.q,
               self.k, self.v, self.alpha, self.beta, self.conv_w, conv_state, S,
               self.commit_status, stream)

    def step_from(self, prev: "DeviceTree", S, conv_state, conv_state_out, out=None,
                  accepted=None, stream=None):
        """Fused step: commit prev's accepted node, then verify this tree."""
        step(self.dims, prev.meta, prev.accepted if accepted is None else accepted, prev.q,
             prev.k, prev.v, prev.alpha, prev.beta, prev.commit_status, self.meta, self.q,
             self.k, self.v, self.alpha, self.beta, self.conv_w, conv_state, conv_state_out, S,
             self.out if out is None else out, stream)

    def meta_arrays(self):
        """Host views of the metadata blob (layout of gdn_tree.h)."""
        B, T = self.dims.B, self.dims.T
        raw = self.meta.cpu().numpy()
        return unpack_meta(raw, B, T)


def meta_layout(B: int, T: int) -> dict:
    """Byte offsets of the metadata arrays (gdn_tree.h)."""
    def a16(x):
        return (x + 15) & ~15
    W = (T + 63) // 64
    off = {"anc": 0}
    off["depth"] = a16(8 * B * T * W)
    off["order"] = a16(off["depth"] + 4 * B * T)
    off["pos"] = a16(off["order"] + 4 * B * T)
    off["parent"] = a16(off["pos"] + 4 * B * T)
    off["status"] = a16(off["parent"] + 4 * B * T)
    off["nvalid"] = a16(off["status"] + 4 * B)
    off["pdep"] = a16(off["nvalid"] + 4 * B)
    off["ppos"] = a16(off["pdep"] + 4 * B * T)
    off["W"] = W
    return off


def unpack_meta(raw, B: int, T: int) -> dict:
    import numpy as np
    off = meta_layout(B, T)
    W = off["W"]

    def arr(name, dt, n, shape):
        return np.frombuffer(raw, dtype=dt, count=n, offset=off[name]).reshape(shape)
    return dict(anc=arr("anc", np.uint64, B * T * W, (B, T, W)),
                depth=arr("depth", np.int32, B * T, (B, T)),
                order=arr("order", np.int32, B * T, (B, T)),
                pos=arr("pos", np.int32, B * T, (B, T)),
                parent=arr("parent", np.int32, B * T, (B, T)),
                status=arr("status", np.int32, B, (B,)),
                nvalid=arr("nvalid", np.int32, B, (B,)),
                pdep=arr("pdep", np.int32, B * T, (B, T)),
                ppos=arr("ppos", np.int32, B * T, (B, T)))
