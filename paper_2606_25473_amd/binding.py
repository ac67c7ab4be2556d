"""ctypes binding of libattnjvp.so (argument marshalling only).

Every step of the computation runs in the HIP library.  Torch tensors supply
device memory and the current HIP stream; outputs are allocated here with
``torch.empty``.  There is no fallback: if the library is missing or a call
fails, an exception is raised.
"""
import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
_LIBPATH = os.path.join(_PKG, "lib", "libattnjvp.so")

DTYPE_F32, DTYPE_BF16 = 0, 1
MASK_KINDS = {"full": 0, "block_causal": 1, "teacher_forcing": 2, "ranges": 3}
MAX_CHUNKS = 64
ERR_NAMES = {1: "invalid argument", 2: "unsupported", 3: "HIP error"}


class AttnError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{ERR_NAMES.get(code, code)}: {msg}")
        self.code = code


MAX_GROUPS = 128
MAX_RANGES = 256


class _Layout(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("num_chunks", ctypes.c_int32),
                ("chunk_offsets", ctypes.POINTER(ctypes.c_int32)),
                ("range_offsets", ctypes.POINTER(ctypes.c_int32)),
                ("ranges", ctypes.POINTER(ctypes.c_int32))]


_lib = None
_vp = ctypes.c_void_p
_i = ctypes.c_int


def library_path():
    return _LIBPATH


def load_library():
    """Load libattnjvp.so once; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIBPATH):
        raise RuntimeError(f"HIP library not built: {_LIBPATH} is missing "
                           "(run `python -m paper_2606_25473_amd.build`)")
    lib = ctypes.CDLL(_LIBPATH)
    lib.attn_jvp_fwd.argtypes = [_i, _i, _i, _i, _i, _vp, _vp, _vp, _vp, _vp, _vp,
                                 ctypes.POINTER(_Layout), ctypes.c_float, _vp, _vp, _vp, _vp]
    lib.attn_jvp_fwd.restype = _i
    lib.attn_jvp_fwd_zero_clean.argtypes = lib.attn_jvp_fwd.argtypes
    lib.attn_jvp_fwd_zero_clean.restype = _i
    lib.attn_fwd.argtypes = [_i, _i, _i, _i, _i, _vp, _vp, _vp,
                             ctypes.POINTER(_Layout), ctypes.c_float, _vp, _vp, _vp]
    lib.attn_fwd.restype = _i
    lib.attn_bwd.argtypes = [_i, _i, _i, _i, _i, _vp, _vp, _vp, _vp, _vp, _vp,
                             ctypes.POINTER(_Layout), ctypes.c_float, _vp, _vp, _vp, _vp, _vp]
    lib.attn_bwd.restype = _i
    _ip = ctypes.POINTER(ctypes.c_int32)
    lib.attn_key_tile_plan.argtypes = [ctypes.POINTER(_Layout), _i, _i, _ip, _ip, _i]
    lib.attn_key_tile_plan.restype = _i
    lib.attn_count_unmasked_pairs.argtypes = [ctypes.POINTER(_Layout), _i]
    lib.attn_count_unmasked_pairs.restype = ctypes.c_int64
    lib.attn_count_computed_pairs.argtypes = [ctypes.POINTER(_Layout), _i, _i]
    lib.attn_count_computed_pairs.restype = ctypes.c_int64
    lib.attn_query_groups.argtypes = [ctypes.POINTER(_Layout), _i, _ip, _ip, _ip, _i, _i]
    lib.attn_query_groups.restype = _i
    lib.attn_tile_shape.argtypes = [ctypes.POINTER(_i), ctypes.POINTER(_i)]
    lib.attn_tile_shape.restype = None
    lib.attn_tile_plan.argtypes = [ctypes.POINTER(_Layout), _i, _i, ctypes.POINTER(ctypes.c_int32),
                                   ctypes.POINTER(ctypes.c_int32), _i]
    lib.attn_tile_plan.restype = _i
    lib.attn_tile_order.argtypes = [ctypes.POINTER(_Layout), _i, _i, ctypes.POINTER(ctypes.c_int32), _i]
    lib.attn_tile_order.restype = _i
    lib.attn_last_error.argtypes = []
    lib.attn_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _i32(vals):
    return (ctypes.c_int32 * max(1, len(vals)))(*vals)


def make_layout(kind, offsets=None):
    """C layout struct for mask ``kind`` ('full' | 'block_causal' | 'teacher_forcing' |
    'ranges', or its code).  ``offsets``: chunk prefix offsets, or for 'ranges' the
    query groups [(q0, q1, [(k0, k1), ...]), ...] in increasing order, each starting
    where the previous one ends (rows that see no key form a group with no range)."""
    code = MASK_KINDS[kind] if isinstance(kind, str) else int(kind)
    if code == MASK_KINDS["ranges"]:
        groups = list(offsets or [])
        bounds, roffs, flat = [], [0], []
        for i, (q0, q1, ks) in enumerate(groups):
            if i == 0:
                bounds.append(int(q0))
            elif int(q0) != bounds[-1]:
                raise ValueError(f"query group {i} starts at {q0}, not where group {i - 1} ends ({bounds[-1]})")
            bounds.append(int(q1))
            for k0, k1 in ks:
                flat += [int(k0), int(k1)]
            roffs.append(len(flat) // 2)
        arrs = (_i32(bounds), _i32(roffs), _i32(flat))
        lay = _Layout(code, len(groups), arrs[0], arrs[1], arrs[2])
        lay._keep = arrs  # keep the arrays alive with the struct
        return lay
    offs = [] if offsets is None else [int(x) for x in offsets]
    arr = _i32(offs) if offs else None
    lay = _Layout(code, max(0, len(offs) - 1), arr, None, None)
    lay._keep = arr
    return lay


def last_error():
    return load_library().attn_last_error().decode()


def _check(rc):
    if rc != 0:
        raise AttnError(rc, last_error())


def _dtype_code(t):
    if t.dtype == torch.float32:
        return DTYPE_F32
    if t.dtype == torch.bfloat16:
        return DTYPE_BF16
    raise TypeError(f"unsupported dtype {t.dtype} (float32 or bfloat16)")


def _check_inputs(ts, shape=None):
    """All of ``ts`` on q's device with q's dtype, contiguous, of ``shape`` (q's by default)."""
    q = ts[0]
    if q.dim() != 4:
        raise ValueError("tensors must be [B, H, L, D]")
    shape = q.shape if shape is None else shape
    for t in ts:
        if not t.is_cuda:
            raise ValueError("tensors must live on a GPU")
        if t.device != q.device or t.dtype != q.dtype or t.shape != shape:
            raise ValueError("all inputs need the same device, dtype and shape")
        if not t.is_contiguous():
            raise ValueError("inputs must be contiguous")


def _check_out(t, name, shape, dtype, device):
    """A caller-supplied output: contiguous, of the shape, dtype and device the call writes."""
    if not isinstance(t, torch.Tensor) or t.device != device or t.dtype != dtype \
            or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"out tensor {name} must be a contiguous {dtype} tensor of shape {tuple(shape)} on {device}")


def _check_outs(outs, specs, q):
    if len(outs) != len(specs):
        raise ValueError(f"out must hold {len(specs)} tensors")
    for t, (name, shape, dtype) in zip(outs, specs):
        _check_out(t, name, shape, dtype, q.device)


def attn_jvp_fwd(q, k, v, dq, dk, dv, kind="teacher_forcing", offsets=None, scale=None,
                 out=None, stream=None):
    """(O, dO, LSE) of masked softmax attention and its forward-mode tangent.

    q..dv: contiguous [B, H, L, D] float32 or bfloat16 GPU tensors.  ``out`` may
    supply preallocated (O, dO, LSE).  Work is queued on ``stream`` (default:
    the current stream of q's device).
    """
    lib = load_library()
    _check_inputs([q, k, v, dq, dk, dv])
    B, H, L, D = q.shape
    if out is None:
        o, do = torch.empty_like(q), torch.empty_like(q)
        lse = torch.empty((B, H, L), device=q.device, dtype=torch.float32)
    else:
        _check_outs(out, [("O", q.shape, q.dtype), ("dO", q.shape, q.dtype), ("LSE", (B, H, L), torch.float32)], q)
        o, do, lse = out
    lay = make_layout(kind, offsets)
    st = stream if stream is not None else torch.cuda.current_stream(q.device)
    with torch.cuda.device(q.device):
        rc = lib.attn_jvp_fwd(_dtype_code(q), B, H, L, D, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                              dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), ctypes.byref(lay),
                              float(scale or 0.0), o.data_ptr(), do.data_ptr(), lse.data_ptr(),
                              st.cuda_stream)
    _check(rc)
    return o, do, lse


def attn_jvp_fwd_zero_clean(q, k, v, dqn, dkn, dvn, offsets, scale=None, out=None, stream=None):
    """(O, dOn, LSE) of teacher-forcing attention whose clean half has zero tangent.

    q, k, v: contiguous [B, H, L, D] GPU tensors over the packed [clean | noisy]
    sequence; dqn, dkn, dvn: [B, H, L/2, D] tangents of the noisy half only.
    Returns O [B, H, L, D], dOn [B, H, L/2, D] (dO of the noisy half; the clean
    half's is zero) and LSE [B, H, L].  ``offsets``: chunk prefix offsets.
    """
    lib = load_library()
    _check_inputs([q, k, v])
    B, H, L, D = q.shape
    nshape = torch.Size((B, H, L - L // 2, D))
    _check_inputs([dqn, dkn, dvn], nshape)
    if dqn.device != q.device or dqn.dtype != q.dtype:
        raise ValueError("tangents need q's device and dtype")
    if out is None:
        o = torch.empty_like(q)
        don = torch.empty(nshape, device=q.device, dtype=q.dtype)
        lse = torch.empty((B, H, L), device=q.device, dtype=torch.float32)
    else:
        _check_outs(out, [("O", q.shape, q.dtype), ("dOn", nshape, q.dtype), ("LSE", (B, H, L), torch.float32)], q)
        o, don, lse = out
    lay = make_layout("teacher_forcing", offsets)
    st = stream if stream is not None else torch.cuda.current_stream(q.device)
    with torch.cuda.device(q.device):
        rc = lib.attn_jvp_fwd_zero_clean(_dtype_code(q), B, H, L, D, q.data_ptr(), k.data_ptr(),
                                         v.data_ptr(), dqn.data_ptr(), dkn.data_ptr(), dvn.data_ptr(),
                                         ctypes.byref(lay), float(scale or 0.0), o.data_ptr(),
                                         don.data_ptr(), lse.data_ptr(), st.cuda_stream)
    _check(rc)
    return o, don, lse


def attn_fwd(q, k, v, kind="teacher_forcing", offsets=None, scale=None, out=None, stream=None):
    """(O, LSE) of masked softmax attention (forward only)."""
    lib = load_library()
    _check_inputs([q, k, v])
    B, H, L, D = q.shape
    if out is None:
        o = torch.empty_like(q)
        lse = torch.empty((B, H, L), device=q.device, dtype=torch.float32)
    else:
        _check_outs(out, [("O", q.shape, q.dtype), ("LSE", (B, H, L), torch.float32)], q)
        o, lse = out
    lay = make_layout(kind, offsets)
    st = stream if stream is not None else torch.cuda.current_stream(q.device)
    with torch.cuda.device(q.device):
        rc = lib.attn_fwd(_dtype_code(q), B, H, L, D, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                          ctypes.byref(lay), float(scale or 0.0), o.data_ptr(), lse.data_ptr(),
                          st.cuda_stream)
    _check(rc)
    return o, lse


def attn_bwd(q, k, v, o, go, lse, kind="teacher_forcing", offsets=None, scale=None, out=None, stream=None):
    """(gQ, gK, gV, Delta): gradients of masked attention for the cotangent ``go`` of ``o``.

    q, k, v, o, go: contiguous [B, H, L, D] GPU tensors of one dtype; lse: fp32 [B, H, L]
    from the forward call that produced ``o``.  ``out`` may supply (gQ, gK, gV, Delta).
    """
    lib = load_library()
    _check_inputs([q, k, v, o, go])
    B, H, L, D = q.shape
    if lse.dtype != torch.float32 or tuple(lse.shape) != (B, H, L) or not lse.is_contiguous() \
            or lse.device != q.device:
        raise ValueError("lse must be a contiguous fp32 [B, H, L] tensor on q's device")
    if out is None:
        gq, gk, gv = torch.empty_like(q), torch.empty_like(q), torch.empty_like(q)
        delta = torch.empty((B, H, L), device=q.device, dtype=torch.float32)
    else:
        _check_outs(out, [("gQ", q.shape, q.dtype), ("gK", q.shape, q.dtype), ("gV", q.shape, q.dtype),
                          ("Delta", (B, H, L), torch.float32)], q)
        gq, gk, gv, delta = out
    lay = make_layout(kind, offsets)
    st = stream if stream is not None else torch.cuda.current_stream(q.device)
    with torch.cuda.device(q.device):
        rc = lib.attn_bwd(_dtype_code(q), B, H, L, D, q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                          go.data_ptr(), lse.data_ptr(), ctypes.byref(lay), float(scale or 0.0), gq.data_ptr(),
                          gk.data_ptr(), gv.data_ptr(), delta.data_ptr(), st.cuda_stream)
    _check(rc)
    return gq, gk, gv, delta


def _read_table(fn, kind, offsets, L):
    bounds = (ctypes.c_int32 * (MAX_GROUPS + 1))()
    roffs = (ctypes.c_int32 * (MAX_GROUPS + 1))()
    ranges = (ctypes.c_int32 * (2 * MAX_RANGES))()
    n = fn(ctypes.byref(make_layout(kind, offsets)), int(L), bounds, roffs, ranges, MAX_GROUPS, MAX_RANGES)
    if n < 0:
        raise AttnError(1, last_error())
    return [(bounds[g], bounds[g + 1], [(ranges[2 * r], ranges[2 * r + 1]) for r in range(roffs[g], roffs[g + 1])])
            for g in range(n)]


def count_unmasked_pairs(kind, offsets, L):
    """Admissible (query, key) pairs per (batch, head) (host-only library call)."""
    n = load_library().attn_count_unmasked_pairs(ctypes.byref(make_layout(kind, offsets)), int(L))
    if n < 0:
        raise AttnError(1, last_error())
    return int(n)


def count_computed_pairs(kind, offsets, L, D=128):
    """Pairs the bf16 kernel evaluates per (batch, head), masked lanes included."""
    n = load_library().attn_count_computed_pairs(ctypes.byref(make_layout(kind, offsets)), int(L), int(D))
    if n < 0:
        raise AttnError(1, last_error())
    return int(n)


def query_groups(kind, offsets, L):
    """Query-group table [(q0, q1, [(k0, k1), ...]), ...] derived by the library (normalised:
    each group's ranges sorted, empty ones dropped, touching ones merged)."""
    return _read_table(load_library().attn_query_groups, kind, offsets, L)


def tile_shape():
    """(query rows per tile, keys per block) of the bf16 kernels."""
    r, k = _i(), _i()
    load_library().attn_tile_shape(ctypes.byref(r), ctypes.byref(k))
    return r.value, k.value


def tile_order(kind, offsets, L, zero_clean=False):
    """Query tile taken by the t-th work-group of a (batch, head), for t = 0, 1, ..."""
    R, _ = tile_shape()
    cap = (int(L) + R - 1) // R
    buf = (ctypes.c_int32 * max(cap, 1))()
    n = load_library().attn_tile_order(ctypes.byref(make_layout(kind, offsets)), int(L),
                                       1 if zero_clean else 0, buf, cap)
    if n < 0:
        raise AttnError(1, last_error())
    return list(buf[:n])


def key_tile_plan(kind, offsets, L, ktile):
    """[(query_block, is_full), ...] visited by key tile ``ktile`` of the bf16 backward
    (128 keys per tile, 64-row query blocks)."""
    cap = (int(L) + 63) // 64 + 8
    blocks = (ctypes.c_int32 * cap)()
    full = (ctypes.c_int32 * cap)()
    n = load_library().attn_key_tile_plan(ctypes.byref(make_layout(kind, offsets)), int(L), int(ktile),
                                          blocks, full, cap)
    if n < 0:
        raise AttnError(1, last_error())
    return [(blocks[i], bool(full[i])) for i in range(n)]


def tile_plan(kind, offsets, L, qtile):
    """[(key_block, is_full), ...] visited by query tile ``qtile`` of the bf16 kernels."""
    cap = (int(L) + 31) // 32 + 8
    blocks = (ctypes.c_int32 * cap)()
    full = (ctypes.c_int32 * cap)()
    n = load_library().attn_tile_plan(ctypes.byref(make_layout(kind, offsets)), int(L), int(qtile),
                                      blocks, full, cap)
    if n < 0:
        raise AttnError(1, last_error())
    return [(blocks[i], bool(full[i])) for i in range(n)]
