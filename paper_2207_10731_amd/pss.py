"""Python binding of libpss.so (ctypes): argument marshalling only.

The function names are those of the C ABI.  Tensors must be contiguous and
live on the current GPU; work is enqueued on torch's current stream unless a
stream is given.  Every computation happens in the HIP library: if it cannot
be loaded, the first call raises.
"""
from __future__ import annotations

import atexit
import ctypes
import os
import re

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libpss.so")
INCLUDE = os.path.join(os.path.dirname(_PKG), "include")
HEADER = os.path.join(INCLUDE, "pss.h")

PSS_PRIME = 2**31 - 1
PSS_F32, PSS_BF16 = 0, 1
PSS_OK, PSS_ERR_INVALID_ARG, PSS_ERR_UNSUPPORTED, PSS_ERR_HIP, PSS_ERR_NO_MEMORY = 0, 1, 2, 3, 4
PSS_ERR_SCRATCH_LIMIT = 5
PSS_NOALLOC_SCRATCH_BYTES = 64 << 20
PSS_BWD_AUTO, PSS_BWD_ATOMIC, PSS_BWD_SORTED, PSS_BWD_SPARSE = 0, 1, 2, 3
PSS_BWD_MASK = 3
PSS_SIGN_PM1, PSS_SIGN_SPARSE, PSS_SIGN_MASK = 1 << 2, 2 << 2, 3 << 2
PSS_POOL_MEAN, PSS_INDEX_I32, PSS_ROWS_BF16 = 1 << 4, 1 << 5, 1 << 6
PSS_PREPARE_BACKWARD = 1 << 7
PSS_DEPOSIT_BY_ADDRESS = 1 << 8


class PssError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {status_string(status)} (status {status})")
        self.status = status


class pss_hash_params(ctypes.Structure):
    _fields_ = [
        ("a", ctypes.c_uint32),
        ("b", ctypes.c_uint32),
        ("num_tables", ctypes.c_uint32),
        ("batch", ctypes.c_uint32),
        ("num_indices", ctypes.c_int64),
        ("weight_dtype", ctypes.c_int32),
        ("eps", ctypes.c_float),
        ("flags", ctypes.c_uint32),
        ("sign_a", ctypes.c_uint32),
        ("sign_b", ctypes.c_uint32),
    ]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads libpss.so once.  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with python -m paper_2207_10731_amd.build")
    lib = ctypes.CDLL(path)
    vp, i32, i64, u64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
    hp = ctypes.POINTER(pss_hash_params)
    lib.pss_hash_params_from_seed.argtypes = [u64, hp]
    lib.pss_forward.argtypes = [vp, i64, i32, i32, hp, vp, vp, vp, vp]
    lib.pss_backward_update.argtypes = [vp, vp, i64, i32, i32, hp, vp, vp, vp, ctypes.c_float, vp]
    lib.pss_backward_update_noalloc.argtypes = lib.pss_backward_update.argtypes
    lib.pss_prepare_backward.argtypes = [i64, i32, i32, hp, vp, vp, vp]
    lib.pss_debug_addresses.argtypes = [i64, i32, i32, hp, vp, vp, vp, vp]
    lib.pss_debug_signs.argtypes = [i64, i32, i32, hp, vp, vp, vp, vp]
    lib.pss_hash_signs_host.argtypes = [i64, i32, i32, hp, vp, vp, vp]
    lib.pss_gradient_sparse.argtypes = [i64, i32, i32, hp, vp, vp, vp, vp, vp, i64, vp, vp]
    lib.pss_hash_bases_host.argtypes = [i64, i32, i32, hp, vp, vp, vp]
    lib.pss_validate_offsets_host.argtypes = [vp, i64, i64]
    lib.pss_status_string.argtypes = [ctypes.c_int]
    lib.pss_status_string.restype = ctypes.c_char_p
    lib.pss_release_scratch.argtypes = []
    lib.pss_debug_reduce_events.argtypes = [vp, vp]
    for name in ("pss_hash_params_from_seed", "pss_forward", "pss_backward_update",
                 "pss_backward_update_noalloc",
                 "pss_prepare_backward", "pss_debug_addresses", "pss_debug_signs",
                 "pss_gradient_sparse",
                 "pss_hash_bases_host", "pss_hash_signs_host", "pss_validate_offsets_host",
                 "pss_release_scratch", "pss_debug_reduce_events"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    # Return the library's runtime objects (kept scratch, prepared-grouping
    # streams and events, memory pools) while the interpreter still runs,
    # before the HIP runtime's own teardown at process exit.
    atexit.register(_release_at_exit)
    return lib


def _release_at_exit():
    if _lib is not None:
        try:
            _lib.pss_release_scratch()
        except Exception:  # nothing useful to do at exit
            pass


BENCH_LIB_PATH = os.path.join(_PKG, "libpss_bench.so")
_bench = None


def load_bench_library(path: str = BENCH_LIB_PATH) -> ctypes.CDLL:
    """Loads libpss_bench.so (measurement kernels beside the layer) once."""
    global _bench
    if _bench is not None:
        return _bench
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with python -m paper_2207_10731_amd.build")
    lib = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
    lib.pss_bench_copy.argtypes = [vp, vp, ctypes.c_size_t, vp]
    lib.pss_bench_read.argtypes = [vp, ctypes.c_size_t, i32, i32, vp, vp]
    lib.pss_bench_gather.argtypes = [vp, ctypes.c_size_t, i32, i32, ctypes.c_uint32, vp,
                                     ctypes.POINTER(i64), vp]
    for name in ("pss_bench_copy", "pss_bench_read", "pss_bench_gather"):
        getattr(lib, name).restype = ctypes.c_int
    _bench = lib
    return lib


def header_functions(paths=None) -> list[str]:
    """Names of the functions declared in the headers (default: include/*.h)."""
    if paths is None:
        paths = sorted(os.path.join(INCLUDE, f) for f in os.listdir(INCLUDE) if f.endswith(".h"))
    names = set()
    for path in paths:
        with open(path) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)  # drop comments
        names.update(re.findall(r"\b(pss_\w+)\s*\(", text))
    return sorted(names)


def status_string(status: int) -> str:
    return load_library().pss_status_string(int(status)).decode()


def _check(status: int, where: str):
    if status != PSS_OK:
        raise PssError(status, where)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _need(t, dtype, name, device=True):
    if t is None:
        return
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if device and not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")


def _need_len(t, n, name):
    """The kernels trust the sizes the call declares (M, N, T*B, d): a tensor
    shorter than that would be read or written past its end."""
    if t is not None and t.numel() < n:
        raise ValueError(f"{name} has {t.numel()} elements, the call needs {n}")


def _same_device(*ts):
    """Scratch, pools and launches follow the current device."""
    dev = torch.cuda.current_device()
    for t in ts:
        if t is not None and t.is_cuda and t.device.index != dev:
            raise ValueError(f"tensor on {t.device}, current device is cuda:{dev}")


def _need_batch(hash_params, M, Z, d, indices, offsets, rows=None, rows_name="out"):
    """Sizes the call implies: indices N, offsets T*B + 1, rows B x T*d."""
    bags = int(hash_params.num_tables) * int(hash_params.batch)
    _need_len(indices, int(hash_params.num_indices), "indices")
    _need_len(offsets, bags + 1, "offsets")
    if rows is not None:
        _need_len(rows, bags * int(d), rows_name)


def make_hash_params(seed=None, *, a=None, b=None, sign_a=None, sign_b=None, num_tables, batch,
                     num_indices, weight_dtype=PSS_F32, eps=1e-10,
                     flags=PSS_BWD_AUTO) -> pss_hash_params:
    """Fills the parameter block; (a, b, sign_a, sign_b) from ``seed`` via
    pss_hash_params_from_seed, then any given explicitly."""
    hp = pss_hash_params(0, 0, num_tables, batch, num_indices, weight_dtype, eps, flags, 1, 0)
    if seed is not None:
        _check(load_library().pss_hash_params_from_seed(ctypes.c_uint64(seed), ctypes.byref(hp)),
               "pss_hash_params_from_seed")
    for name, v in (("a", a), ("b", b), ("sign_a", sign_a), ("sign_b", sign_b)):
        if v is not None:
            setattr(hp, name, v)
    return hp


def _index_dtype(hp):
    return torch.int32 if hp.flags & PSS_INDEX_I32 else torch.int64


def _row_dtype(hp):
    return torch.bfloat16 if hp.flags & PSS_ROWS_BF16 else torch.float32


def _weight_dtype(shared):
    return PSS_BF16 if shared.dtype == torch.bfloat16 else PSS_F32


def pss_forward(shared, M, Z, d, hash_params, indices, offsets, out, stream=None):
    lib = load_library()
    _need(shared, shared.dtype, "shared")
    if shared.dtype not in (torch.float32, torch.bfloat16):
        raise TypeError("shared must be float32 or bfloat16")
    if hash_params.weight_dtype != _weight_dtype(shared):
        raise TypeError("hash_params.weight_dtype does not match shared")
    _need(indices, _index_dtype(hash_params), "indices")
    _need(offsets, _index_dtype(hash_params), "offsets")
    _need(out, _row_dtype(hash_params), "out")
    _need_len(shared, M, "shared")
    _need_batch(hash_params, M, Z, d, indices, offsets, out, "out")
    _same_device(shared, indices, offsets, out)
    _check(lib.pss_forward(_ptr(shared), M, Z, d, ctypes.byref(hash_params), _ptr(indices),
                           _ptr(offsets), _ptr(out), _stream(stream)), "pss_forward")
    return out


def pss_prepare_backward(M, Z, d, hash_params, indices, offsets, stream=None):
    """Starts the backward's grouping of this batch on a library stream (the
    work PSS_PREPARE_BACKWARD adds to pss_forward, as a call of its own)."""
    lib = load_library()
    _need(indices, _index_dtype(hash_params), "indices")
    _need(offsets, _index_dtype(hash_params), "offsets")
    _need_batch(hash_params, M, Z, d, indices, offsets)
    _same_device(indices, offsets)
    _check(lib.pss_prepare_backward(M, Z, d, ctypes.byref(hash_params), _ptr(indices),
                                    _ptr(offsets), _stream(stream)), "pss_prepare_backward")


def pss_backward_update(shared, state, M, Z, d, hash_params, indices, offsets, grad_out, lr,
                        stream=None):
    _backward("pss_backward_update", shared, state, M, Z, d, hash_params, indices, offsets,
              grad_out, lr, stream)


def pss_backward_update_noalloc(shared, state, M, Z, d, hash_params, indices, offsets, grad_out,
                                lr, stream=None):
    """The allocation-free backward: scratch in the library's static device
    array (PSS_ERR_SCRATCH_LIMIT when the call needs more)."""
    _backward("pss_backward_update_noalloc", shared, state, M, Z, d, hash_params, indices,
              offsets, grad_out, lr, stream)


def _backward(name, shared, state, M, Z, d, hash_params, indices, offsets, grad_out, lr, stream):
    lib = load_library()
    _need(shared, shared.dtype, "shared")
    if hash_params.weight_dtype != _weight_dtype(shared):
        raise TypeError("hash_params.weight_dtype does not match shared")
    _need(state, torch.float32, "state")
    _need(indices, _index_dtype(hash_params), "indices")
    _need(offsets, _index_dtype(hash_params), "offsets")
    _need(grad_out, _row_dtype(hash_params), "grad_out")
    _need_len(shared, M, "shared")
    _need_len(state, M, "state")
    _need_batch(hash_params, M, Z, d, indices, offsets, grad_out, "grad_out")
    _same_device(shared, state, indices, offsets, grad_out)
    _check(getattr(lib, name)(_ptr(shared), _ptr(state), M, Z, d, ctypes.byref(hash_params),
                              _ptr(indices), _ptr(offsets), _ptr(grad_out), ctypes.c_float(lr),
                              _stream(stream)), name)


def pss_gradient_sparse(M, Z, d, hash_params, indices, offsets, grad_out, locations, values,
                        num_unique, stream=None):
    """locations: int32 tensor (uint32 bit patterns), values: float32, both of
    length >= min(M, N*d); num_unique: int64 tensor of one element."""
    lib = load_library()
    _need(indices, _index_dtype(hash_params), "indices")
    _need(offsets, _index_dtype(hash_params), "offsets")
    _need(grad_out, _row_dtype(hash_params), "grad_out")
    _need(locations, torch.int32, "locations")
    _need(values, torch.float32, "values")
    _need(num_unique, torch.int64, "num_unique")
    if locations.numel() != values.numel():
        raise ValueError("locations and values must have the same length")
    _need_len(num_unique, 1, "num_unique")
    _need_batch(hash_params, M, Z, d, indices, offsets, grad_out, "grad_out")
    _same_device(indices, offsets, grad_out, locations, values, num_unique)
    _check(lib.pss_gradient_sparse(M, Z, d, ctypes.byref(hash_params), _ptr(indices), _ptr(offsets),
                                   _ptr(grad_out), _ptr(locations), _ptr(values),
                                   locations.numel(), _ptr(num_unique), _stream(stream)),
           "pss_gradient_sparse")


def pss_debug_addresses(M, Z, d, hash_params, indices, offsets, base_out, stream=None):
    lib = load_library()
    _need(indices, _index_dtype(hash_params), "indices")
    _need(offsets, _index_dtype(hash_params), "offsets")
    _need(base_out, torch.int32, "base_out")  # uint32 bit patterns
    _need_batch(hash_params, M, Z, d, indices, offsets)
    if Z > 0 and d % Z == 0:
        _need_len(base_out, int(hash_params.num_indices) * (d // Z), "base_out")
    _same_device(indices, offsets, base_out)
    _check(lib.pss_debug_addresses(M, Z, d, ctypes.byref(hash_params), _ptr(indices),
                                   _ptr(offsets), _ptr(base_out), _stream(stream)),
           "pss_debug_addresses")
    return base_out


def pss_debug_signs(M, Z, d, hash_params, indices, offsets, sign_out, stream=None):
    lib = load_library()
    _need(indices, _index_dtype(hash_params), "indices")
    _need(offsets, _index_dtype(hash_params), "offsets")
    _need(sign_out, torch.int8, "sign_out")
    _need_batch(hash_params, M, Z, d, indices, offsets)
    if Z > 0 and d % Z == 0:
        _need_len(sign_out, int(hash_params.num_indices) * (d // Z), "sign_out")
    _same_device(indices, offsets, sign_out)
    _check(lib.pss_debug_signs(M, Z, d, ctypes.byref(hash_params), _ptr(indices), _ptr(offsets),
                               _ptr(sign_out), _stream(stream)), "pss_debug_signs")
    return sign_out


def pss_hash_bases_host(M, Z, d, hash_params, indices, offsets):
    """Host evaluation of the library's hash code on NumPy arrays: uint32 [N, C]."""
    import numpy as np
    lib = load_library()
    idx = np.ascontiguousarray(indices, dtype=np.int64)
    off = np.ascontiguousarray(offsets, dtype=np.int64)
    out = np.zeros((idx.shape[0], d // Z if Z > 0 and d % Z == 0 else 1), dtype=np.uint32)
    if idx.shape[0] < int(hash_params.num_indices):
        raise ValueError(f"indices has {idx.shape[0]} entries, the call needs {hash_params.num_indices}")
    if off.shape[0] < int(hash_params.num_tables) * int(hash_params.batch) + 1:
        raise ValueError("offsets must hold T*B + 1 entries")
    _check(lib.pss_hash_bases_host(M, Z, d, ctypes.byref(hash_params),
                                   idx.ctypes.data_as(ctypes.c_void_p),
                                   off.ctypes.data_as(ctypes.c_void_p),
                                   out.ctypes.data_as(ctypes.c_void_p)), "pss_hash_bases_host")
    return out


def pss_hash_signs_host(M, Z, d, hash_params, indices, offsets):
    """Host evaluation of the library's chunk-sign code: int8 [N, C] of +1, -1, 0."""
    import numpy as np
    lib = load_library()
    idx = np.ascontiguousarray(indices, dtype=np.int64)
    off = np.ascontiguousarray(offsets, dtype=np.int64)
    out = np.zeros((idx.shape[0], d // Z if Z > 0 and d % Z == 0 else 1), dtype=np.int8)
    if idx.shape[0] < int(hash_params.num_indices):
        raise ValueError(f"indices has {idx.shape[0]} entries, the call needs {hash_params.num_indices}")
    if off.shape[0] < int(hash_params.num_tables) * int(hash_params.batch) + 1:
        raise ValueError("offsets must hold T*B + 1 entries")
    _check(lib.pss_hash_signs_host(M, Z, d, ctypes.byref(hash_params),
                                   idx.ctypes.data_as(ctypes.c_void_p),
                                   off.ctypes.data_as(ctypes.c_void_p),
                                   out.ctypes.data_as(ctypes.c_void_p)), "pss_hash_signs_host")
    return out


def pss_validate_offsets_host(offsets, num_bags, N) -> int:
    import numpy as np
    off = np.ascontiguousarray(offsets, dtype=np.int64)
    if num_bags < 0 or off.shape[0] < num_bags + 1:
        return PSS_ERR_INVALID_ARG
    return load_library().pss_validate_offsets_host(off.ctypes.data_as(ctypes.c_void_p),
                                                    num_bags, N)


def pss_debug_reduce_events(before=None, after=None):
    """Timing hook: in later backward calls the dispatch of the
    reduce-and-deposit kernel records the two events (torch.cuda.Event objects
    with timing, recorded once already so that their HIP events exist, or raw
    hipEvent_t handles) at the kernel's start and end; no arguments switch it
    off.  The events must stay alive while the hook is set."""
    handles = []
    for ev in (before, after):
        if ev is None:
            handles.append(None)
            continue
        if hasattr(ev, "cuda_event"):  # torch.cuda.Event
            h = int(ev.cuda_event)
        else:  # a raw hipEvent_t: int or ctypes.c_void_p
            h = int((ev.value or 0) if isinstance(ev, ctypes.c_void_p) else ev)
        if h == 0:
            raise ValueError("pss_debug_reduce_events: a null event (a torch event must be "
                             "recorded once before it is passed)")
        handles.append(ctypes.c_void_p(h))
    _check(load_library().pss_debug_reduce_events(handles[0], handles[1]),
           "pss_debug_reduce_events")


def pss_release_scratch():
    """Frees the scratch buffers the library keeps per (device, stream)."""
    _check(load_library().pss_release_scratch(), "pss_release_scratch")


def pss_status_string(status: int) -> str:
    return status_string(status)


def _table_lookups(T, n, device):
    """One-item bags over every (t, i) of T tables of n rows, table-major.

    The mapping's key is (i*T + t)*C + j.  Presenting row i of table t as
    token i*T + t of a single table (T = 1) gives the same key, so bag
    g = t*n + i reads exactly the chunks of (t, i) and its pooled row
    [g, 0:d] is element (t, i, :) of a [T, n, d] tensor."""
    if T * n >= 2**31:
        raise ValueError("T * n must stay below 2^31")
    ii = torch.arange(n, dtype=torch.int64, device=device) * T
    indices = (ii.unsqueeze(0) + torch.arange(T, dtype=torch.int64, device=device).unsqueeze(1))
    offsets = torch.arange(T * n + 1, dtype=torch.int64, device=device)
    return indices.reshape(-1), offsets


def compress_table(table, M, Z, hash_params, variant=PSS_BWD_SPARSE, out=None, stream=None):
    """Post-hoc PSS of given tables (Sec. 2.4 with Thm. 2: M = S E).

    table: float32 [T, n, d] on the GPU.  Returns the float32 flat array of
    M elements whose element m is the sum of every table entry (t, i, c)
    that the mapping sends to m (``out`` if given, which is overwritten),
    times the chunk's sign factor when ``hash_params.flags`` selects a sign.
    Only (a, b), the sign option and (sign_a, sign_b) of ``hash_params`` are
    used.  One deposit pass of the
    library: every row is a one-item bag whose output gradient is the row,
    applied by SGD with lr = -1 to a zeroed array.  The default SPARSE
    backward sums each location in a fixed order (bitwise reproducible);
    PSS_BWD_SORTED / PSS_BWD_ATOMIC are faster and sum in arrival order.
    """
    if table.dim() != 3:
        raise ValueError("table must be [T, n, d]")
    _need(table, torch.float32, "table")
    T, n, d = table.shape
    indices, offsets = _table_lookups(T, n, table.device)
    sign = hash_params.flags & PSS_SIGN_MASK
    hp = pss_hash_params(hash_params.a, hash_params.b, 1, T * n, T * n, PSS_F32,
                         hash_params.eps, variant | sign, hash_params.sign_a, hash_params.sign_b)
    if out is None:
        out = torch.empty(M, dtype=torch.float32, device=table.device)
    _need(out, torch.float32, "out")
    if out.numel() != M:
        raise ValueError("out must hold M elements")
    if isinstance(stream, torch.cuda.Stream):
        with torch.cuda.stream(stream):
            out.zero_()
    else:
        out.zero_()
    pss_backward_update(out, None, M, Z, d, hp, indices, offsets, table.contiguous().view(T * n, d),
                        -1.0, stream)
    return out


def lookup_rows(shared, M, Z, d, num_tables, rows, hash_params, stream=None):
    """Retrieved rows (S e_(t,i))^T M of rows 0 .. rows-1 of every table:
    float32 [num_tables, rows, d] (one forward pass of one-item bags)."""
    T = num_tables
    indices, offsets = _table_lookups(T, rows, shared.device)
    sign = hash_params.flags & PSS_SIGN_MASK
    hp = pss_hash_params(hash_params.a, hash_params.b, 1, T * rows, T * rows,
                         _weight_dtype(shared), hash_params.eps, PSS_BWD_AUTO | sign,
                         hash_params.sign_a, hash_params.sign_b)
    out = torch.empty((T, rows, d), dtype=torch.float32, device=shared.device)
    pss_forward(shared, M, Z, d, hp, indices, offsets, out.view(T * rows, d), stream)
    return out
