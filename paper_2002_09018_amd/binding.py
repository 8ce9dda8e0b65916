"""ctypes binding of libshampoo.so (the C ABI in include/shampoo.h).

Argument marshalling only: every step of the computation runs in the HIP
kernels behind the C entry points.  Functions carry the C names.  Tensors are
torch tensors on the handle's device (torch is used for device memory and
streams); the binding passes their data pointers and the current stream.
There is no CPU fallback: if the library cannot be loaded, importing this
module raises.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("SHAMPOO_LIB", os.path.join(HERE, "libshampoo.so"))

if not os.path.exists(LIB_PATH):
    raise ImportError(f"libshampoo.so not found at {LIB_PATH}: build it with "
                      f"`python -c 'import __graft_entry__ as g; g.build()'`")
_lib = C.CDLL(LIB_PATH)

SHAMPOO_OK, SHAMPOO_EINVAL, SHAMPOO_EUNSUPPORTED, SHAMPOO_EHIP, SHAMPOO_ENOMEM = 0, -1, -2, -3, -4
SHAMPOO_F32, SHAMPOO_BF16 = 0, 1
ROOT_CONVERGED, ROOT_STAGNATED, ROOT_MAXITER, ROOT_DIVERGED, ROOT_NOT_PD = 0, 1, 2, 3, 4
PRECISION_FP32, PRECISION_AUTO, PRECISION_FP64 = 0, 1, 2
SCALING_FROBENIUS, SCALING_POWER4 = 0, 1
(KCLASS_NEWTON_F32, KCLASS_NEWTON_F64, KCLASS_STATS, KCLASS_PRECOND, KCLASS_GRAFT, KCLASS_ROOT_AUX, KCLASS_EMB,
 KCLASS_NEWTON_WARM) = range(8)
KCLASS_NAMES = ["newton_f32", "newton_f64", "stats", "precond", "graft", "root_aux", "emb", "newton_warm"]


class shampoo_block(C.Structure):
    _fields_ = [("rows", C.c_int32), ("cols", C.c_int32), ("ld", C.c_int64),
                ("G", C.c_void_p), ("W", C.c_void_p), ("D", C.c_void_p), ("P", C.c_void_p),
                ("Mg", C.c_void_p), ("Ps", C.c_void_p), ("L", C.c_void_p), ("R", C.c_void_p),
                ("Lr", C.c_void_p), ("Rr", C.c_void_p)]


class shampoo_root_job(C.Structure):
    _fields_ = [("n", C.c_int32), ("reserved", C.c_int32), ("A", C.c_void_p), ("X", C.c_void_p)]


class shampoo_root_params(C.Structure):
    _fields_ = [("p", C.c_int32), ("eps", C.c_float), ("eps_relative", C.c_int32), ("tol", C.c_float),
                ("max_iters", C.c_int32), ("precision", C.c_int32), ("kappa32", C.c_float),
                ("maxsv_steps", C.c_int32), ("maxsv_tol", C.c_float), ("poll", C.c_int32),
                ("scaling", C.c_int32)]


class shampoo_root_info(C.Structure):
    _fields_ = [("status", C.c_int32), ("iters", C.c_int32), ("precision", C.c_int32),
                ("iters_fp32", C.c_int32), ("resid", C.c_float), ("lambda_max", C.c_float),
                ("cond_est", C.c_float), ("eps_eff", C.c_float)]


ROOT_INFO_FIELDS = [f for f, _ in shampoo_root_info._fields_]

_vp, _i, _f, _sz, _i64 = C.c_void_p, C.c_int, C.c_float, C.c_size_t, C.c_int64
_sig = {
    "shampoo_create": (_i, [C.POINTER(_vp), _i]),
    "shampoo_destroy": (_i, [_vp]),
    "shampoo_last_error": (C.c_char_p, [_vp]),
    "shampoo_version": (C.c_char_p, []),
    "shampoo_root_params_default": (None, [C.POINTER(shampoo_root_params)]),
    "shampoo_update_stats": (_i, [_vp, C.POINTER(shampoo_block), _i, _i, _f, _vp]),
    "shampoo_inv_root_workspace_bytes": (_sz, [C.POINTER(shampoo_root_job), _i, _i]),
    "shampoo_inv_root_batched": (_i, [_vp, C.POINTER(shampoo_root_job), _i, C.POINTER(shampoo_root_params),
                                      _vp, _sz, _vp, _vp]),
    "shampoo_inv_root_warm_batched": (_i, [_vp, C.POINTER(shampoo_root_job), _i, C.POINTER(shampoo_root_params),
                                           _f, _vp, _sz, _vp, _vp, _vp]),
    "shampoo_precondition": (_i, [_vp, C.POINTER(shampoo_block), _i, _i, _vp]),
    "shampoo_graft": (_i, [_vp, C.POINTER(shampoo_block), _i, _i, _f, _f, _i, _vp, _vp]),
    "shampoo_graft_lamb": (_i, [_vp, C.POINTER(shampoo_block), _i, _i, _f, _f, _i, _vp, _vp]),
    "shampoo_graft_noalloc": (_i, [_vp, C.POINTER(shampoo_block), _i, _i, _f, _f, _i, _vp, _vp]),
    "shampoo_precondition_graft": (_i, [_vp, C.POINTER(shampoo_block), _i, _i, _f, _vp, _vp]),
    "shampoo_embedding_workspace_bytes": (_sz, [_i, _i]),
    "shampoo_embedding_rows": (_i, [_vp, _vp, _vp, _vp, _i, _i64, _vp, _i, _i, _i64, _vp, _vp, _vp, _vp, _sz, _vp]),
    "shampoo_embedding_stats": (_i, [_vp, _vp, _vp, _i, _i, _vp, _f, _vp, _sz, _vp]),
    "shampoo_embedding_precondition": (_i, [_vp, _vp, _vp, _i, _i, _vp, _vp, _vp]),
    "shampoo_embedding_graft": (_i, [_vp, _vp, _vp, _i, _i, _vp, _vp, _vp, _vp, _i64, _i64, _f, _i, _vp, _vp]),
    "shampoo_timing_enable": (_i, [_vp, _i]),
    "shampoo_timing_read": (_i, [_vp, _i, C.POINTER(C.c_double), C.POINTER(C.c_int64)]),
}
for _name, (_res, _args) in _sig.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args

EXPORTED = tuple(_sig)


class ShampooError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"shampoo error {code}: {msg}")
        self.code = code


def _ptr(t):
    return None if t is None else t.data_ptr()


# ------------------------------------------------------------------ argument checks
# The C side cannot see shapes, strides, element types or devices: it gets
# raw pointers.  Every entry point below therefore checks its tensors against
# the layout include/shampoo.h states and raises ValueError before any C call.
# Device placement is checked last, so that a layout mistake is reported as
# such whatever the device.
_handle_device = {}


def _is_dtype(t, *names):
    return str(t.dtype).replace("torch.", "") in names


def _need(cond, msg):
    if not cond:
        raise ValueError(msg)


def _fp32(t, what):
    _need(_is_dtype(t, "float32"), f"{what}: dtype {t.dtype}, expected float32")


def _int32(t, what):
    _need(_is_dtype(t, "int32"), f"{what}: dtype {t.dtype}, expected int32")


def _contig(t, what):
    _need(t.is_contiguous(), f"{what}: must be contiguous (row-major, no gaps)")


def _square(t, n, what):
    _need(t.dim() == 2 and tuple(t.shape) == (n, n), f"{what}: shape {tuple(t.shape)}, expected ({n}, {n})")


def _min_numel(t, k, what):
    _need(t.numel() >= k, f"{what}: {t.numel()} elements, at least {k} needed")


def _devices(handle, tensors):
    """Every tensor must be a GPU tensor on the handle's device (one device
    for the call when the handle's device is not known)."""
    want = _handle_device.get(getattr(handle, "value", handle))
    for what, t in tensors:
        if t is None:
            continue
        _need(t.device.type == "cuda", f"{what}: on {t.device}, expected a GPU tensor")
        if want is None:
            want = t.device.index
        _need(t.device.index == want, f"{what}: on cuda:{t.device.index}, expected cuda:{want}")


_STATE_FIELDS = ("W", "D", "P", "Mg", "Ps")


_torch_mod = None


def _torch():
    global _torch_mod
    if _torch_mod is None:
        import torch
        _torch_mod = torch
    return _torch_mod


def _check_blocks(handle, blocks, norms=None):
    """Fast pass over the blocks (cheap accessors, no per-check calls); the
    detailed checker below runs only when something fails, to raise with the
    exact reason."""
    torch = _torch()
    f32, bf16 = torch.float32, torch.bfloat16
    want = _handle_device.get(getattr(handle, "value", handle))
    dev0 = None
    ok = True
    g_dtype = None
    for b in blocks:
        g = b.G
        if g is None or g.dim() != 2:
            ok = False
            break
        gd = g.dtype
        if g_dtype is None:
            g_dtype = gd
        if gd is not g_dtype or (gd is not f32 and gd is not bf16):
            ok = False
            break
        gs = g.size()
        m, n = gs[0], gs[1]
        gst = g.stride()
        ld = gst[0] if m > 1 else n
        dev = g.get_device()
        if dev0 is None:
            dev0 = dev
        if (n != 1 and gst[1] != 1) or dev != dev0:
            ok = False
            break
        for t in (b.W, b.D, b.P, b.Mg, b.Ps):
            if t is None:
                continue
            st = t.stride()
            if (t.dtype is not f32 or t.size() != gs or t.get_device() != dev0 or (n != 1 and st[1] != 1)
                    or (m != 1 and st[0] != ld)):
                ok = False
                break
        if not ok:
            break
        for t, k in ((b.L, m), (b.R, n), (b.Lr, m), (b.Rr, n)):
            if t is None:
                continue
            if t.dtype is not f32 or t.size() != (k, k) or not t.is_contiguous() or t.get_device() != dev0:
                ok = False
                break
        if not ok:
            break
    if ok and norms is not None:
        ok = (norms.dtype is f32 and norms.is_contiguous() and norms.numel() >= 3 * len(blocks)
              and (dev0 is None or norms.get_device() == dev0))
    if ok and (dev0 is None or (dev0 >= 0 and (want is None or dev0 == want))):
        if dev0 is None and norms is not None:
            _devices(handle, [("norms", norms)])
        return
    _check_blocks_detailed(handle, blocks, norms)
    raise ValueError("tensors of one call must all be on one GPU, the handle's")


def _check_blocks_detailed(handle, blocks, norms=None):
    tensors = []
    g_dtype = None
    for i, b in enumerate(blocks):
        g = b.G
        _need(g is not None, f"block {i}: G is required")
        _need(g.dim() == 2, f"block {i}: G has {g.dim()} dimensions, expected 2")
        _need(_is_dtype(g, "float32", "bfloat16"), f"block {i}: G dtype {g.dtype}, expected float32 or bfloat16")
        if g_dtype is None:
            g_dtype = g.dtype
        _need(g.dtype == g_dtype, f"block {i}: G dtype {g.dtype} differs from block 0's {g_dtype}: one call "
                                  f"takes one gradient type")
        m, n = int(g.shape[0]), int(g.shape[1])
        _need(n == 1 or g.stride(1) == 1, f"block {i}: G columns must be adjacent (stride(1) == 1)")
        ld = int(g.stride(0)) if m > 1 else n
        tensors.append((f"block {i}: G", g))
        for name in _STATE_FIELDS:
            t = getattr(b, name)
            if t is None:
                continue
            what = f"block {i}: {name}"
            _fp32(t, what)
            _need(tuple(t.shape) == (m, n), f"{what}: shape {tuple(t.shape)}, expected G's {(m, n)}")
            _need((n == 1 or t.stride(1) == 1) and (m == 1 or int(t.stride(0)) == ld),
                  f"{what}: strides {tuple(t.stride())}, expected G's row stride ({ld}, 1): the views of a "
                  f"block share one ld")
            tensors.append((what, t))
        for name, k in (("L", m), ("R", n), ("Lr", m), ("Rr", n)):
            t = getattr(b, name)
            if t is None:
                continue
            what = f"block {i}: {name}"
            _fp32(t, what)
            _square(t, k, what)
            _contig(t, what)
            tensors.append((what, t))
    _check_norms(handle, norms, len(blocks), tensors)


def _check_norms(handle, norms, nblocks, tensors=()):
    tensors = list(tensors)
    if norms is not None:
        _fp32(norms, "norms")
        _contig(norms, "norms")
        _min_numel(norms, 3 * nblocks, "norms")
        tensors.append(("norms", norms))
    _devices(handle, tensors)


def _check_jobs(handle, As, Xs, workspace, info, warm_out=None):
    """Fast pass (see _check_blocks); the detailed checks raise the reason."""
    torch = _torch()
    f32 = torch.float32
    want = _handle_device.get(getattr(handle, "value", handle))
    ok = len(As) == len(Xs) and workspace is not None
    dev0 = None
    if ok:
        for a, x in zip(As, Xs):
            sz = a.size()
            dev = a.get_device()
            if dev0 is None:
                dev0 = dev
            if (len(sz) != 2 or sz[0] != sz[1] or a.dtype is not f32 or x.dtype is not f32 or x.size() != sz
                    or not a.is_contiguous() or not x.is_contiguous() or dev != dev0 or x.get_device() != dev0
                    or a.data_ptr() == x.data_ptr()):
                ok = False
                break
    if ok:
        ok = (workspace.is_contiguous() and info.dtype is torch.int32 and info.is_contiguous()
              and info.numel() >= 8 * len(As) and (warm_out is None or (warm_out.dtype is torch.int32 and
                                                                        warm_out.is_contiguous() and
                                                                        warm_out.numel() >= 2 * len(As))))
        devs = [workspace.get_device(), info.get_device()] + ([] if warm_out is None else [warm_out.get_device()])
        if dev0 is None:
            dev0 = devs[0]
        ok = ok and all(d == dev0 for d in devs) and dev0 >= 0 and (want is None or dev0 == want)
    if ok:
        return
    _check_jobs_detailed(handle, As, Xs, workspace, info, warm_out)
    raise ValueError("tensors of one call must all be on one GPU, the handle's")


def _job_list_tensors(As, Xs):
    """Layout checks of the As / Xs of a root call (raise with the reason);
    returns the tensors for the device check."""
    _need(len(As) == len(Xs), f"{len(As)} statistics but {len(Xs)} outputs")
    tensors = []
    for i, (a, x) in enumerate(zip(As, Xs)):
        _need(a.dim() == 2, f"job {i}: A has {a.dim()} dimensions, expected 2")
        n = int(a.shape[0])
        for what, t in ((f"job {i}: A", a), (f"job {i}: X", x)):
            _fp32(t, what)
            _square(t, n, what)
            _contig(t, what)
            tensors.append((what, t))
        _need(a.data_ptr() != x.data_ptr() or n == 0, f"job {i}: A and X must be distinct buffers")
    return tensors


def _job_buffer_tensors(njobs, workspace, info, warm_out):
    """Layout checks of the workspace / info / warm_out of a root call of
    njobs jobs; returns the tensors for the device check."""
    _need(workspace is not None, "workspace is required")
    _contig(workspace, "workspace")
    _int32(info, "info")
    _contig(info, "info")
    _min_numel(info, 8 * njobs, "info (8 int32 per job)")
    tensors = [("workspace", workspace), ("info", info)]
    if warm_out is not None:
        _int32(warm_out, "warm_out")
        _contig(warm_out, "warm_out")
        _min_numel(warm_out, 2 * njobs, "warm_out (2 int32 per job)")
        tensors.append(("warm_out", warm_out))
    return tensors


def _check_jobs_detailed(handle, As, Xs, workspace, info, warm_out=None):
    As, Xs = list(As), list(Xs)
    tensors = _job_list_tensors(As, Xs) + _job_buffer_tensors(len(As), workspace, info, warm_out)
    _devices(handle, tensors)


def _stream(stream):
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def _check(handle, code):
    if code != SHAMPOO_OK:
        msg = _lib.shampoo_last_error(handle)
        raise ShampooError(code, msg.decode() if msg else "")


@dataclass
class Block:
    """One block view.  Tensors must share the row stride of G (``ld``)."""
    G: object
    W: Optional[object] = None
    D: Optional[object] = None
    P: Optional[object] = None
    Mg: Optional[object] = None
    Ps: Optional[object] = None
    L: Optional[object] = None
    R: Optional[object] = None
    Lr: Optional[object] = None
    Rr: Optional[object] = None


_BLOCK_PTRS = ("G", "W", "D", "P", "Mg", "Ps", "L", "R", "Lr", "Rr")


def _blocks(blocks: Sequence[Block]):
    """The shampoo_block array of a call, packed as 12 int64 words per block
    (rows | cols << 32, ld, then the ten pointers), as a ctypes pointer into a
    numpy buffer that the caller keeps alive over the C call."""
    import numpy as np
    rec = []
    for b in blocks:
        g = b.G
        m, n = g.size()
        ld = g.stride(0) if m > 1 else n   # one row: no stride used
        rec.append([m | (n << 32), ld] + [0 if t is None else t.data_ptr() for t in
                                          (b.G, b.W, b.D, b.P, b.Mg, b.Ps, b.L, b.R, b.Lr, b.Rr)])
    buf = np.array(rec if rec else [[0] * 12], dtype=np.uint64)
    assert buf.shape[1] * 8 == C.sizeof(shampoo_block)
    return _Packed(buf, buf.ctypes.data_as(C.POINTER(shampoo_block)))


class _Packed:
    """A packed host table and its ctypes pointer (the table lives as long as this object)."""
    def __init__(self, buf, ptr):
        self._buf, self._as_parameter_ = buf, ptr


def _dtype_code(blocks):
    if not blocks:
        return SHAMPOO_F32
    import torch
    dt = blocks[0].G.dtype
    return SHAMPOO_BF16 if dt == torch.bfloat16 else SHAMPOO_F32


class PackedBlocks:
    """A block list checked and packed once, for calls that repeat with the
    same views (a training loop passes the same blocks every step): every
    entry point that takes a block list accepts it in its place and skips the
    per-call checks and packing.  It records each tensor's pointer, size and
    row stride as they are when packed and keeps those tensors alive (a field
    of a Block reassigned later still leaves the packed tensor valid, if
    stale); pack again after any of them is reallocated, resized or
    replaced."""

    def __init__(self, handle, blocks):
        blocks = list(blocks)
        _check_blocks(handle, blocks)
        self.blocks = blocks
        self._tensors = [getattr(b, f) for b in blocks for f in _BLOCK_PTRS]
        self._handle = getattr(handle, "value", handle)
        self._arr = _blocks(blocks)
        self._dtype = _dtype_code(blocks)
        self._device = blocks[0].G.get_device() if blocks else None

    def __len__(self):
        return len(self.blocks)


class PackedJobs:
    """Inverse-root jobs (As, Xs) checked and packed once, as PackedBlocks:
    accepted by shampoo_inv_root_batched and shampoo_inv_root_warm_batched in
    place of As (Xs is then None).  Pack again after any tensor is
    reallocated or replaced."""

    def __init__(self, handle, As, Xs):
        As, Xs = list(As), list(Xs)
        _need(len(As) > 0, "PackedJobs: no jobs")
        _devices(handle, _job_list_tensors(As, Xs))
        self.As, self.Xs = As, Xs  # the packed tensors stay alive with this object
        self._handle = getattr(handle, "value", handle)
        self._arr = _jobs(As, Xs)
        self._device = As[0].get_device()

    def __len__(self):
        return len(self.As)


def _block_args(handle, blocks, norms=None):
    """(packed table, count, G dtype code) of a call's blocks: a PackedBlocks
    as it was packed (only norms is checked), a list checked and packed now."""
    if isinstance(blocks, PackedBlocks):
        _need(blocks._handle == getattr(handle, "value", handle), "PackedBlocks was packed for another handle")
        if norms is not None:
            _check_norms(handle, norms, len(blocks))
            _need(blocks._device is None or norms.get_device() == blocks._device,
                  "norms: not on the blocks' device")
        return blocks._arr, len(blocks), blocks._dtype
    _check_blocks(handle, blocks, norms)
    return _blocks(blocks), len(blocks), _dtype_code(blocks)


def _job_args(handle, As, Xs, workspace, info, warm_out=None):
    """(packed table, count) of a root call: a PackedJobs as it was packed (the
    workspace, info and warm_out checked now), lists checked and packed now."""
    if isinstance(As, PackedJobs):
        _need(Xs is None, "with PackedJobs, Xs must be None (the outputs are packed)")
        _need(As._handle == getattr(handle, "value", handle), "PackedJobs was packed for another handle")
        tensors = _job_buffer_tensors(len(As), workspace, info, warm_out)
        _devices(handle, tensors)
        for what, t in tensors:
            _need(t.get_device() == As._device, f"{what}: not on the jobs' device")
        return As._arr, len(As)
    _check_jobs(handle, As, Xs, workspace, info, warm_out)
    return _jobs(As, Xs), len(As)


# ------------------------------------------------------------------ entry points
def shampoo_version():
    return _lib.shampoo_version().decode()


def shampoo_root_params_default(**overrides):
    p = shampoo_root_params()
    _lib.shampoo_root_params_default(C.byref(p))
    for k, v in overrides.items():
        setattr(p, k, v)
    return p


def shampoo_create(device=0):
    h = C.c_void_p()
    code = _lib.shampoo_create(C.byref(h), int(device))
    if code != SHAMPOO_OK:
        raise ShampooError(code, f"shampoo_create(device={device}) failed")
    _handle_device[h.value] = int(device)
    return h


def shampoo_destroy(handle):
    _check(handle, _lib.shampoo_destroy(handle))
    _handle_device.pop(getattr(handle, "value", handle), None)


def shampoo_update_stats(handle, blocks, beta2=1.0, stream=None):
    """blocks: a list of Block, or a PackedBlocks."""
    arr, nb, dt = _block_args(handle, blocks)
    _check(handle, _lib.shampoo_update_stats(handle, arr, nb, dt, float(beta2), _stream(stream)))


def _jobs(As, Xs):
    """The shampoo_root_job array, packed as 3 int64 words per job (n, A, X)."""
    import numpy as np
    rec = [[a.size(0), a.data_ptr(), x.data_ptr()] for a, x in zip(As, Xs)]
    buf = np.array(rec if rec else [[0] * 3], dtype=np.uint64)
    assert buf.shape[1] * 8 == C.sizeof(shampoo_root_job)
    return _Packed(buf, buf.ctypes.data_as(C.POINTER(shampoo_root_job)))


def shampoo_inv_root_workspace_bytes(ns, precision=PRECISION_AUTO):
    arr = (shampoo_root_job * max(1, len(ns)))()
    for i, n in enumerate(ns):
        arr[i].n = int(n)
    return int(_lib.shampoo_inv_root_workspace_bytes(arr, len(ns), int(precision)))


def shampoo_inv_root_batched(handle, As, Xs, params, workspace, info, stream=None):
    """As, Xs: lists of contiguous n x n fp32 device tensors (or As a
    PackedJobs and Xs None); workspace: a uint8 device tensor; info: an int32
    device tensor of 8 * len(As)."""
    arr, nj = _job_args(handle, As, Xs, workspace, info)
    _check(handle, _lib.shampoo_inv_root_batched(handle, arr, nj, C.byref(params), _ptr(workspace),
                                                 int(workspace.numel() * workspace.element_size()),
                                                 _ptr(info), _stream(stream)))


def shampoo_inv_root_warm_batched(handle, As, Xs, params, workspace, info, warm_out=None, comm_tol=1e-3,
                                  stream=None):
    """As shampoo_inv_root_batched; Xs hold the warm starts X0 on entry.
    warm_out: None or an int32 device tensor of 2 * len(As)."""
    arr, nj = _job_args(handle, As, Xs, workspace, info, warm_out)
    _check(handle, _lib.shampoo_inv_root_warm_batched(handle, arr, nj, C.byref(params), float(comm_tol),
                                                      _ptr(workspace),
                                                      int(workspace.numel() * workspace.element_size()),
                                                      _ptr(info), _ptr(warm_out), _stream(stream)))


def shampoo_precondition(handle, blocks, stream=None):
    arr, nb, dt = _block_args(handle, blocks)
    _check(handle, _lib.shampoo_precondition(handle, arr, nb, dt, _stream(stream)))


def shampoo_graft(handle, blocks, eta0, beta1=0.0, use_shampoo=True, norms=None, stream=None):
    arr, nb, dt = _block_args(handle, blocks, norms)
    _check(handle, _lib.shampoo_graft(handle, arr, nb, dt, float(eta0), float(beta1), int(bool(use_shampoo)),
                                      _ptr(norms), _stream(stream)))


def shampoo_graft_noalloc(handle, blocks, eta0, beta1=0.0, use_shampoo=True, norms=None, stream=None):
    """shampoo_graft without any device allocation (fixed scratch; see the header for its limits)."""
    arr, nb, dt = _block_args(handle, blocks, norms)
    _check(handle, _lib.shampoo_graft_noalloc(handle, arr, nb, dt, float(eta0), float(beta1), int(bool(use_shampoo)),
                                              _ptr(norms), _stream(stream)))


def _nbytes(t):
    return 0 if t is None else int(t.numel() * t.element_size())


def shampoo_embedding_workspace_bytes(nnz, dim):
    return int(_lib.shampoo_embedding_workspace_bytes(int(nnz), int(dim)))


def _check_vec(t, k, what, kind):
    (_int32 if kind == "int32" else _fp32)(t, what)
    _contig(t, what)
    _min_numel(t, k, what)


def _check_compact(U, what="U"):
    _need(U.dim() == 2, f"{what}: {U.dim()} dimensions, expected nnz x dim")
    _fp32(U, what)
    _contig(U, what)
    return int(U.shape[0]), int(U.shape[1])


def shampoo_embedding_rows(handle, idx, feat, weight, vocab, dy, rows, U, count, workspace, stream=None):
    """idx, feat (or None): int32 [nnz]; weight: fp32 [nnz] or None; dy: m x dim
    fp32 (row-major view); rows int32 [nnz], U fp32 nnz x dim (contiguous),
    count int32 [2]; workspace: uint8 device tensor."""
    nnz = int(idx.numel())
    _check_vec(idx, nnz, "idx", "int32")
    if feat is not None:
        _need(feat.numel() == nnz, f"feat: {feat.numel()} entries, idx has {nnz}")
        _check_vec(feat, nnz, "feat", "int32")
    if weight is not None:
        _need(weight.numel() == nnz, f"weight: {weight.numel()} entries, idx has {nnz}")
        _check_vec(weight, nnz, "weight", "float32")
    _need(dy.dim() == 2, f"dy: {dy.dim()} dimensions, expected 2")
    _fp32(dy, "dy")
    _need(dy.shape[1] == 1 or dy.stride(1) == 1, "dy: columns must be adjacent (stride(1) == 1)")
    m, dim = int(dy.shape[0]), int(dy.shape[1])
    _check_vec(rows, nnz, "rows", "int32")
    u_rows, u_dim = _check_compact(U)
    _need(u_rows >= nnz and u_dim == dim, f"U: shape {tuple(U.shape)}, expected at least ({nnz}, {dim})")
    _check_vec(count, 2, "count", "int32")
    _need(workspace is not None, "workspace is required")
    _contig(workspace, "workspace")
    _devices(handle, [("idx", idx), ("feat", feat), ("weight", weight), ("dy", dy), ("rows", rows), ("U", U),
                      ("count", count), ("workspace", workspace)])
    _check(handle, _lib.shampoo_embedding_rows(handle, _ptr(idx), _ptr(feat), _ptr(weight), nnz, int(vocab),
                                               _ptr(dy), m, dim, int(dy.stride(0)), _ptr(rows), _ptr(U),
                                               _ptr(count), _ptr(workspace), _nbytes(workspace), _stream(stream)))


def shampoo_embedding_stats(handle, U, count, R, beta2=1.0, workspace=None, stream=None):
    nnz, dim = _check_compact(U)
    _check_vec(count, 2, "count", "int32")
    _fp32(R, "R")
    _square(R, dim, "R")
    _contig(R, "R")
    _need(workspace is not None, "workspace is required")
    _contig(workspace, "workspace")
    _devices(handle, [("U", U), ("count", count), ("R", R), ("workspace", workspace)])
    _check(handle, _lib.shampoo_embedding_stats(handle, _ptr(U), _ptr(count), nnz, dim, _ptr(R), float(beta2),
                                                _ptr(workspace), _nbytes(workspace), _stream(stream)))


def shampoo_embedding_precondition(handle, U, count, Rr, P, stream=None):
    nnz, dim = _check_compact(U)
    _check_vec(count, 2, "count", "int32")
    _fp32(Rr, "Rr")
    _square(Rr, dim, "Rr")
    _contig(Rr, "Rr")
    _need(_check_compact(P, "P") == (nnz, dim), f"P: shape {tuple(P.shape)}, expected U's ({nnz}, {dim})")
    _devices(handle, [("U", U), ("count", count), ("Rr", Rr), ("P", P)])
    _check(handle, _lib.shampoo_embedding_precondition(handle, _ptr(U), _ptr(count), nnz, dim, _ptr(Rr), _ptr(P),
                                                       _stream(stream)))


def shampoo_embedding_graft(handle, rows, count, U, P, W, D, eta0, use_shampoo=True, norms=None, stream=None):
    """W, D: vocab x dim fp32 tables (same row stride)."""
    nnz, dim = _check_compact(U)
    _check_vec(rows, nnz, "rows", "int32")
    _check_vec(count, 2, "count", "int32")
    _need(_check_compact(P, "P") == (nnz, dim), f"P: shape {tuple(P.shape)}, expected U's ({nnz}, {dim})")
    for what, t in (("W", W), ("D", D)):
        _fp32(t, what)
        _need(t.dim() == 2 and int(t.shape[1]) == dim, f"{what}: shape {tuple(t.shape)}, expected (vocab, {dim})")
        _need(dim == 1 or t.stride(1) == 1, f"{what}: columns must be adjacent (stride(1) == 1)")
    _need(tuple(W.shape) == tuple(D.shape) and (W.shape[0] == 1 or W.stride(0) == D.stride(0)),
          f"W {tuple(W.shape)} / {tuple(W.stride())} and D {tuple(D.shape)} / {tuple(D.stride())} must share "
          f"shape and row stride")
    _check_norms(handle, norms, 1, [("rows", rows), ("count", count), ("U", U), ("P", P), ("W", W), ("D", D)])
    _check(handle, _lib.shampoo_embedding_graft(handle, _ptr(rows), _ptr(count), nnz, dim, _ptr(U), _ptr(P),
                                                _ptr(W), _ptr(D), int(W.shape[0]), int(W.stride(0)), float(eta0),
                                                int(bool(use_shampoo)), _ptr(norms), _stream(stream)))


def shampoo_precondition_graft(handle, blocks, eta0, norms=None, stream=None):
    arr, nb, dt = _block_args(handle, blocks, norms)
    _check(handle, _lib.shampoo_precondition_graft(handle, arr, nb, dt, float(eta0), _ptr(norms), _stream(stream)))


def shampoo_graft_lamb(handle, blocks, eta0, beta1=0.0, use_shampoo=True, norms=None, stream=None):
    arr, nb, dt = _block_args(handle, blocks, norms)
    _check(handle, _lib.shampoo_graft_lamb(handle, arr, nb, dt, float(eta0), float(beta1), int(bool(use_shampoo)),
                                           _ptr(norms), _stream(stream)))


def shampoo_timing_enable(handle, enable=True):
    _check(handle, _lib.shampoo_timing_enable(handle, int(bool(enable))))


def shampoo_timing_read(handle, kclass):
    ms, n = C.c_double(), C.c_int64()
    _check(handle, _lib.shampoo_timing_read(handle, int(kclass), C.byref(ms), C.byref(n)))
    return ms.value, n.value


def decode_root_info(info_tensor):
    """Host view of a root-info device array: list of dicts."""
    import numpy as np
    raw = info_tensor.detach().cpu().numpy().astype(np.int32).reshape(-1, 8)
    fl = raw.view(np.float32)
    out = []
    for r, f in zip(raw, fl):
        out.append(dict(status=int(r[0]), iters=int(r[1]), precision=int(r[2]), iters_fp32=int(r[3]),
                        resid=float(f[4]), lambda_max=float(f[5]), cond_est=float(f[6]), eps_eff=float(f[7])))
    return out
