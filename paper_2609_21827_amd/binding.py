"""Python binding of librheo.so (the C ABI in include/rheo.h).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  torch supplies device buffers (``data_ptr``) and the HIP stream
(``torch.cuda.current_stream().cuda_stream``).  Importing this module fails
loudly when the library has not been built.
"""

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librheo.so")

RHEO_OK, RHEO_EINVAL, RHEO_ENOMEM, RHEO_EHIP, RHEO_ESTATE = 0, -1, -2, -3, -4
RHEO_F32, RHEO_BF16 = 0, 1
RHEO_METHOD_RHEO, RHEO_METHOD_RRSW, RHEO_METHOD_TOPK = 0, 1, 2
METHODS = {"rheo": RHEO_METHOD_RHEO, "rrsw": RHEO_METHOD_RRSW, "topk": RHEO_METHOD_TOPK}
ERROR_NAMES = {RHEO_EINVAL: "EINVAL", RHEO_ENOMEM: "ENOMEM", RHEO_EHIP: "EHIP",
               RHEO_ESTATE: "ESTATE"}

# every symbol the header declares
EXPORTS = ["rheo_create", "rheo_create_static", "rheo_destroy", "rheo_begin_step", "rheo_expand_level",
           "rheo_frontier", "rheo_frontier_view", "rheo_prune", "rheo_pruned_view",
           "rheo_tree_mask", "rheo_verify",
           "rheo_read_nodes", "rheo_device_error", "rheo_node_count",
           "rheo_last_error"]


class RheoConfig(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("pool", ctypes.c_int32), ("leads", ctypes.c_int32),
                ("depth", ctypes.c_int32), ("n_expand", ctypes.c_int32),
                ("support", ctypes.c_int32), ("construct_tempered", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("method", ctypes.c_int32),
                ("construct_full", ctypes.c_int32),
                ("row_stride", ctypes.c_int64), ("eps_m0", ctypes.c_double)]


class RheoError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{ERROR_NAMES.get(code, code)}: {msg}")
        self.code = code


_LIB = None


def load_library(path=LIB_PATH):
    """Loads librheo.so (raises if it is missing) and declares signatures."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with "
                          "`python -m paper_2609_21827_amd.build` first")
    lib = ctypes.CDLL(path)
    vp, i32, u64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64, ctypes.c_float
    sig = {
        "rheo_create": ([ctypes.POINTER(RheoConfig), ctypes.POINTER(vp)], ctypes.c_int),
        "rheo_create_static": ([ctypes.POINTER(RheoConfig), ctypes.POINTER(vp)], ctypes.c_int),
        "rheo_destroy": ([vp], ctypes.c_int),
        "rheo_begin_step": ([vp], ctypes.c_int),
        "rheo_expand_level": ([vp, vp, f32, u64, vp], ctypes.c_int),
        "rheo_frontier": ([vp, vp, vp, vp], ctypes.c_int),
        "rheo_frontier_view": ([vp, ctypes.POINTER(vp), ctypes.POINTER(vp)], ctypes.c_int),
        "rheo_prune": ([vp, i32, vp], ctypes.c_int),
        "rheo_pruned_view": ([vp, vp, vp, vp], ctypes.c_int),
        "rheo_tree_mask": ([vp, vp, vp, vp], ctypes.c_int),
        "rheo_verify": ([vp, vp, f32, u64, vp, vp, vp, vp], ctypes.c_int),
        "rheo_read_nodes": ([vp] * 10, ctypes.c_int),
        "rheo_device_error": ([vp, ctypes.POINTER(ctypes.c_int32)], ctypes.c_int),
        "rheo_node_count": ([vp], ctypes.c_int32),
        "rheo_last_error": ([], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _LIB = lib
    return lib


def _check(code):
    if code != RHEO_OK:
        raise RheoError(code, _LIB.rheo_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


class _CudaArray:
    """A device int32 array exposed through __cuda_array_interface__."""

    def __init__(self, ptr, shape):
        self.__cuda_array_interface__ = {"shape": tuple(shape), "typestr": "<i4",
                                         "data": (int(ptr), False), "version": 3,
                                         "strides": None}


def _device_view(ptr, shape, device):
    return torch.as_tensor(_CudaArray(ptr, shape), device=device)


class Tree:
    """One tree handle: B sequences, fixed shape, reused step after step."""

    def __init__(self, batch, vocab, pool, leads, depth, support, dtype,
                 n_expand=0, construct_tempered=False, row_stride=None,
                 eps_m0=0.0, method="rheo", construct_full=False, device="cuda",
                 static=False):
        lib = load_library()
        self.device = torch.device(device)
        self.B, self.V, self.K, self.m, self.D = batch, vocab, pool, leads, depth
        self.NE = n_expand or pool
        self.dtype = dtype
        self.row_stride = row_stride or vocab
        cfg = RheoConfig(batch, vocab, pool, leads, depth, n_expand, support,
                         int(construct_tempered),
                         RHEO_BF16 if dtype == torch.bfloat16 else RHEO_F32,
                         METHODS[method] if isinstance(method, str) else int(method),
                         int(construct_full), self.row_stride, eps_m0)
        h = ctypes.c_void_p()
        # static: the device state in the library's static scratch array
        create = lib.rheo_create_static if static else lib.rheo_create
        _check(create(ctypes.byref(cfg), ctypes.byref(h)))
        self._h = h
        self.N = lib.rheo_node_count(h)
        self.R = None

    def close(self):
        if getattr(self, "_h", None):
            _LIB.rheo_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def begin_step(self):
        _check(_LIB.rheo_begin_step(self._h))

    def expand_level(self, draft_logits, T, rng_key, stream=None):
        _check(_LIB.rheo_expand_level(self._h, _ptr(draft_logits), float(T),
                                      int(rng_key) & (2 ** 64 - 1), _stream(stream)))

    def frontier(self, out=None, stream=None):
        if out is None:
            out = (torch.empty((self.B, self.NE), dtype=torch.int32, device=self.device),
                   torch.empty((self.B, self.NE), dtype=torch.int32, device=self.device))
        par, tok = out
        _check(_LIB.rheo_frontier(self._h, _ptr(par), _ptr(tok), _stream(stream)))
        return par, tok

    def frontier_view(self):
        """The tree-owned frontier arrays as int32 [B, n_expand] tensors
        (zero-copy views; contents change with every expand below the last
        level)."""
        par, tok = ctypes.c_void_p(), ctypes.c_void_p()
        _check(_LIB.rheo_frontier_view(self._h, ctypes.byref(par), ctypes.byref(tok)))
        return (_device_view(par.value, (self.B, self.NE), self.device),
                _device_view(tok.value, (self.B, self.NE), self.device))

    def prune(self, budget, stream=None):
        _check(_LIB.rheo_prune(self._h, int(budget), _stream(stream)))
        self.R = int(budget)

    def pruned_view(self, out=None, stream=None):
        if out is None:
            out = (torch.empty((self.B, self.R + 1), dtype=torch.int32, device=self.device),
                   torch.empty((self.B, self.R + 1), dtype=torch.int32, device=self.device))
        par, tok = out
        _check(_LIB.rheo_pruned_view(self._h, _ptr(par), _ptr(tok), _stream(stream)))
        return par, tok

    def tree_mask(self, out=None, stream=None):
        """(mask [B][R+1][R+1] uint8, depth [B][R+1] int32) of the pruned tree."""
        n = self.R + 1
        if out is None:
            out = (torch.empty((self.B, n, n), dtype=torch.uint8, device=self.device),
                   torch.empty((self.B, n), dtype=torch.int32, device=self.device))
        mask, depth = out
        _check(_LIB.rheo_tree_mask(self._h, _ptr(mask), _ptr(depth), _stream(stream)))
        return mask, depth

    def verify(self, target_logits, T, rng_key, out=None, stream=None):
        if out is None:
            out = (torch.empty((self.B, self.D), dtype=torch.int32, device=self.device),
                   torch.empty((self.B,), dtype=torch.int32, device=self.device),
                   torch.empty((self.B,), dtype=torch.int32, device=self.device))
        acc, alen, fin = out
        _check(_LIB.rheo_verify(self._h, _ptr(target_logits), float(T),
                                int(rng_key) & (2 ** 64 - 1), _ptr(acc), _ptr(alen),
                                _ptr(fin), _stream(stream)))
        return acc, alen, fin

    def read_nodes(self, stream=None):
        shape = (self.B, self.N)
        dev = self.device
        out = {k: torch.empty(shape, dtype=torch.int32, device=dev)
               for k in ("token", "parent", "depth", "slot", "kind")}
        out.update({k: torch.empty(shape, dtype=torch.float64, device=dev)
                    for k in ("proxy", "qtrue", "score")})
        _check(_LIB.rheo_read_nodes(self._h, *[_ptr(out[k]) for k in (
            "token", "parent", "depth", "slot", "kind", "proxy", "qtrue", "score")],
            _stream(stream)))
        return out

    def device_error(self):
        flag = ctypes.c_int32(0)
        _check(_LIB.rheo_device_error(self._h, ctypes.byref(flag)))
        return flag.value
