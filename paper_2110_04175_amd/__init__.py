"""RelaySum round on MI355X: thin Python binding of librelaysum.so.

The functions mirror the C ABI of ``include/relaysum.h`` one to one and only
marshal arguments; every step of the round runs in the library's HIP
kernels.  Device buffers are passed as torch CUDA tensors (float32,
C-contiguous, shape [n, d]) or raw device addresses.  If the library is not
built this module raises on first use: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "librelaysum.so")

RELAYSUM_OK = 0
RELAYSUM_ERR_INVALID_ARG = -1
RELAYSUM_ERR_NOT_A_TREE = -2
RELAYSUM_ERR_OUT_OF_MEMORY = -3
RELAYSUM_ERR_DEVICE = -4
RELAYSUM_MAX_WORKERS = 1 << 24   # largest n a handle takes (nbar exact in binary32)

RELAYSUM_UPDATE_MODEL = 0
RELAYSUM_UPDATE_ROBUST = 1
RELAYSUM_UPDATE_GRAD = 2
RELAYSUM_UPDATE_MEAN = 3
RELAYSUM_OPT_SGD = 0
RELAYSUM_OPT_ADAM = 1

UPDATES = {"model": RELAYSUM_UPDATE_MODEL, "robust": RELAYSUM_UPDATE_ROBUST,
           "grad": RELAYSUM_UPDATE_GRAD, "mean": RELAYSUM_UPDATE_MEAN}
OPTIMIZERS = {"sgd": RELAYSUM_OPT_SGD, "adam": RELAYSUM_OPT_ADAM}

# Every symbol include/relaysum.h declares.
EXPORTED = (
    "relaysum_create", "relaysum_create_double", "relaysum_destroy", "relaysum_set_stream",
    "relaysum_step", "relaysum_step_ex", "relaysum_reset", "relaysum_round",
    "relaysum_num_trees", "relaysum_num_directed_edges", "relaysum_directed_edge",
    "relaysum_message_length", "relaysum_get_counts", "relaysum_get_samples",
    "relaysum_get_message", "relaysum_state_size", "relaysum_save_state",
    "relaysum_load_state", "relaysum_poison_next", "relaysum_strerror", "relaysum_last_error",
    "relaysum_step_static", "relaysum_kernel_path", "relaysum_consensus_distance",
)

PATHS = ("tile", "dtree", "wide_dtree", "cluster", "wide", "two_pass", "dtree_seq",
         "cluster_dtree")   # relaysum_path, by value
# Values the library keeps reserved but never returns: trees with a hub of
# more than 32 neighbours, which those kernels took, now take "two_pass".
RETIRED_PATHS = ("wide_dtree", "wide")


class RoundArgs(ctypes.Structure):
    """struct relaysum_round_args of relaysum.h."""
    _fields_ = [("update", ctypes.c_int32), ("optimizer", ctypes.c_int32),
                ("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("adam_step", ctypes.c_int64),
                ("dropped", ctypes.c_void_p)]


class RelaySumError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {strerror(code)} ({code})")
        self.code = code


_lib = None


def _hip_runtimes_mapped():
    try:
        with open("/proc/self/maps") as f:
            return sorted({ln.split()[-1] for ln in f if "libamdhip64" in ln})
    except OSError:
        return []


def load_library(path: Optional[str] = None):
    """Load librelaysum.so (raises if it has not been built).

    torch is imported first: its wheel carries its own HIP runtime, and the
    library must bind to that same runtime (same soname) so that torch's
    device memory and streams are valid in both.  Loading the library first
    would map a second HIP runtime into the process.
    """
    global _lib
    if _lib is not None and path is None:
        return _lib
    import torch  # noqa: F401  (binds libamdhip64 before the library does)
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(
            f"{p} is missing: build it with `python -m paper_2110_04175_amd.build` "
            "(there is no CPU fallback)")
    lib = ctypes.CDLL(p)
    runtimes = _hip_runtimes_mapped()
    if len(runtimes) > 1:
        raise RuntimeError(f"two HIP runtimes are mapped into this process: {runtimes}; "
                           "import torch before loading librelaysum.so")
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    pi32 = ctypes.POINTER(ctypes.c_int32)
    sig = {
        "relaysum_create": (ctypes.c_int, [i32, i64, pi32, i32, ctypes.POINTER(vp)]),
        "relaysum_create_double": (ctypes.c_int, [i32, i64, pi32, pi32, i32, ctypes.POINTER(vp)]),
        "relaysum_destroy": (ctypes.c_int, [vp]),
        "relaysum_set_stream": (ctypes.c_int, [vp, vp]),
        "relaysum_step": (ctypes.c_int, [vp, vp, vp, vp, ctypes.c_float, ctypes.c_float]),
        "relaysum_step_ex": (ctypes.c_int, [vp, vp, vp, vp, vp, ctypes.POINTER(RoundArgs)]),
        "relaysum_get_samples": (ctypes.c_int, [vp, ctypes.POINTER(i64)]),
        "relaysum_consensus_distance": (ctypes.c_int, [vp, vp, ctypes.POINTER(ctypes.c_double),
                                                       ctypes.POINTER(ctypes.c_double)]),
        "relaysum_reset": (ctypes.c_int, [vp]),
        "relaysum_round": (ctypes.c_int, [vp, ctypes.POINTER(i64)]),
        "relaysum_num_trees": (ctypes.c_int, [vp, pi32]),
        "relaysum_kernel_path": (ctypes.c_int, [vp, pi32]),
        "relaysum_num_directed_edges": (ctypes.c_int, [vp, pi32]),
        "relaysum_message_length": (ctypes.c_int, [vp, i32, ctypes.POINTER(i64)]),
        "relaysum_directed_edge": (ctypes.c_int, [vp, i32, pi32, pi32]),
        "relaysum_get_counts": (ctypes.c_int, [vp, pi32, pi32]),
        "relaysum_get_message": (ctypes.c_int, [vp, i32, ctypes.POINTER(ctypes.c_float)]),
        "relaysum_state_size": (ctypes.c_int, [vp, ctypes.POINTER(ctypes.c_size_t)]),
        "relaysum_save_state": (ctypes.c_int, [vp, vp, ctypes.c_size_t]),
        "relaysum_load_state": (ctypes.c_int, [vp, vp, ctypes.c_size_t]),
        "relaysum_poison_next": (ctypes.c_int, [vp]),
        "relaysum_strerror": (ctypes.c_char_p, [ctypes.c_int]),
        "relaysum_last_error": (ctypes.c_char_p, [vp]),
        "relaysum_step_static": (ctypes.c_int, [i32, i64, pi32, i32, i64, vp, vp, vp,
                                                ctypes.c_float, ctypes.c_float, vp]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    if path is None:
        _lib = lib
    return lib


def strerror(code: int) -> str:
    return load_library().relaysum_strerror(int(code)).decode()


def _addr(t) -> Optional[int]:
    """Device address of a tensor (or an int address, or None)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return int(t.data_ptr())


def _check_tensor(t, n, d, name):
    import torch
    if t is None:
        return
    if isinstance(t, int):
        return
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != torch.float32 or not t.is_contiguous() or tuple(t.shape) != (n, d):
        raise ValueError(f"{name} must be a contiguous float32 tensor of shape [{n}, {d}]")


def _check_mask(t, slots):
    """A loss mask must be a contiguous uint8 CUDA tensor with one byte per
    directed-edge slot: the kernels read exactly that many bytes."""
    import torch
    if t is None or isinstance(t, int):
        return
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError("dropped must be a CUDA (HIP) tensor")
    if t.dtype != torch.uint8 or not t.is_contiguous() or t.numel() != slots:
        raise ValueError(f"dropped must be a contiguous uint8 tensor of {slots} elements "
                         "(one per directed-edge slot)")


# ---- functions with the C names ---------------------------------------------


def relaysum_create(n: int, d: int, edges) -> int:
    """Handle (an opaque int) for n workers with d-float models on a tree."""
    lib = load_library()
    e = np.ascontiguousarray(np.asarray(edges, dtype=np.int32).reshape(-1, 2))
    out = ctypes.c_void_p()
    rc = lib.relaysum_create(int(n), int(d),
                             e.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)) if e.size else None,
                             int(e.shape[0]), ctypes.byref(out))
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, "relaysum_create")
    return out.value


def relaysum_create_double(n: int, d: int, edges_a, edges_b) -> int:
    """Handle for double binary trees: odd coordinates on tree A, even on B."""
    lib = load_library()
    ea = np.ascontiguousarray(np.asarray(edges_a, dtype=np.int32).reshape(-1, 2))
    eb = np.ascontiguousarray(np.asarray(edges_b, dtype=np.int32).reshape(-1, 2))
    if ea.shape != eb.shape:
        raise ValueError("both trees need the same number of edges")
    ptr = ctypes.POINTER(ctypes.c_int32)
    out = ctypes.c_void_p()
    rc = lib.relaysum_create_double(int(n), int(d),
                                    ea.ctypes.data_as(ptr) if ea.size else None,
                                    eb.ctypes.data_as(ptr) if eb.size else None,
                                    int(ea.shape[0]), ctypes.byref(out))
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, "relaysum_create_double")
    return out.value


def relaysum_destroy(h: int) -> None:
    rc = load_library().relaysum_destroy(h)
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, "relaysum_destroy")


def relaysum_set_stream(h: int, stream) -> None:
    """`stream`: a torch.cuda.Stream, a raw hipStream_t address, or None."""
    s = stream.cuda_stream if hasattr(stream, "cuda_stream") else stream
    rc = load_library().relaysum_set_stream(h, s)
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, "relaysum_set_stream")


def _last_error(h) -> str:
    return load_library().relaysum_last_error(h).decode()


def relaysum_step(h: int, x, g, mom, lr: float, beta: float) -> None:
    """One RelaySum round for all workers (see relaysum.h)."""
    rc = load_library().relaysum_step(h, _addr(x), _addr(g), _addr(mom), float(lr), float(beta))
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, f"relaysum_step ({_last_error(h)})")


def relaysum_step_ex(h: int, x, g, state1, state2, *, update="model", optimizer="sgd",
                     lr=0.0, beta1=0.0, beta2=0.0, eps=0.0, adam_step=0, dropped=None) -> None:
    """One round under an update rule and local optimizer (see relaysum.h).

    dropped: None, a device tensor / address of one uint8 per directed-edge
    slot, tree-major (nonzero = that message is lost this round).
    """
    args = RoundArgs(UPDATES[update], OPTIMIZERS[optimizer], float(lr), float(beta1),
                     float(beta2), float(eps), int(adam_step), _addr(dropped))
    rc = load_library().relaysum_step_ex(h, _addr(x), _addr(g), _addr(state1), _addr(state2),
                                         ctypes.byref(args))
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, f"relaysum_step_ex ({_last_error(h)})")


def relaysum_get_samples(h: int, n: int) -> np.ndarray:
    """Mean estimation: s_i, samples summed into each worker's y so far
    (n per tree, tree-major)."""
    out = np.zeros(n * relaysum_num_trees(h), np.int64)
    rc = load_library().relaysum_get_samples(h, out.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)))
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, "relaysum_get_samples")
    return out


def relaysum_consensus_distance(h: int, x) -> tuple:
    """(1/n) sum_i ||x_i - xbar||^2 and max |x_ic - xbar_c| of the models in
    x (a device tensor or address of n*d floats), computed on the GPU."""
    dist, spread = ctypes.c_double(), ctypes.c_double()
    rc = load_library().relaysum_consensus_distance(h, _addr(x), ctypes.byref(dist),
                                                    ctypes.byref(spread))
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, f"relaysum_consensus_distance ({_last_error(h)})")
    return dist.value, spread.value


def relaysum_reset(h: int) -> None:
    rc = load_library().relaysum_reset(h)
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, "relaysum_reset")


def relaysum_round(h: int) -> int:
    t = ctypes.c_int64()
    rc = load_library().relaysum_round(h, ctypes.byref(t))
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, "relaysum_round")
    return int(t.value)


def relaysum_num_trees(h: int) -> int:
    c = ctypes.c_int32()
    rc = load_library().relaysum_num_trees(h, ctypes.byref(c))
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, "relaysum_num_trees")
    return int(c.value)


def relaysum_kernel_path(h: int) -> str:
    """Name of the kernel path the handle's rounds take (see PATHS)."""
    c = ctypes.c_int32()
    rc = load_library().relaysum_kernel_path(h, ctypes.byref(c))
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, "relaysum_kernel_path")
    return PATHS[int(c.value)]


def relaysum_message_length(h: int, slot: int) -> int:
    n = ctypes.c_int64()
    rc = load_library().relaysum_message_length(h, int(slot), ctypes.byref(n))
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, "relaysum_message_length")
    return int(n.value)


def relaysum_num_directed_edges(h: int) -> int:
    c = ctypes.c_int32()
    rc = load_library().relaysum_num_directed_edges(h, ctypes.byref(c))
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, "relaysum_num_directed_edges")
    return int(c.value)


def relaysum_directed_edge(h: int, slot: int):
    s, t = ctypes.c_int32(), ctypes.c_int32()
    rc = load_library().relaysum_directed_edge(h, int(slot), ctypes.byref(s), ctypes.byref(t))
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, "relaysum_directed_edge")
    return int(s.value), int(t.value)


def relaysum_get_counts(h: int, n: int):
    """(nbar[n per tree], edge_counts[one per slot]) of the last round, as
    int32 numpy arrays (tree-major)."""
    e2 = relaysum_num_directed_edges(h)
    nbar = np.zeros(n * relaysum_num_trees(h), np.int32)
    cnt = np.zeros(max(e2, 1), np.int32)
    rc = load_library().relaysum_get_counts(
        h, nbar.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
        cnt.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)))
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, "relaysum_get_counts")
    return nbar, cnt[:e2]


def relaysum_get_message(h: int, slot: int) -> np.ndarray:
    d = relaysum_message_length(h, slot)
    out = np.zeros(max(int(d), 1), np.float32)
    rc = load_library().relaysum_get_message(
        h, int(slot), out.ctypes.data_as(ctypes.POINTER(ctypes.c_float)))
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, "relaysum_get_message")
    return out[:int(d)]


def relaysum_state_size(h: int) -> int:
    n = ctypes.c_size_t()
    rc = load_library().relaysum_state_size(h, ctypes.byref(n))
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, "relaysum_state_size")
    return int(n.value)


def _buffer(buf):
    """(address, bytes) of a snapshot buffer: a numpy uint8 array (host), a
    contiguous uint8 torch tensor (host or device), or (address, bytes)."""
    if isinstance(buf, tuple):
        return int(buf[0]), int(buf[1])
    if isinstance(buf, np.ndarray):
        if buf.dtype != np.uint8 or not buf.flags["C_CONTIGUOUS"]:
            raise ValueError("a snapshot buffer must be a contiguous uint8 array")
        return int(buf.ctypes.data), int(buf.nbytes)
    import torch
    if not isinstance(buf, torch.Tensor) or buf.dtype != torch.uint8 or not buf.is_contiguous():
        raise TypeError("a snapshot buffer must be a contiguous uint8 array or tensor")
    return int(buf.data_ptr()), int(buf.numel())


def relaysum_save_state(h: int, buf=None):
    """Snapshot of the handle's state (see relaysum.h) into `buf`, or into a
    new host numpy array that is returned."""
    if buf is None:
        buf = np.zeros(relaysum_state_size(h), np.uint8)
    addr, nbytes = _buffer(buf)
    rc = load_library().relaysum_save_state(h, addr, nbytes)
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, f"relaysum_save_state ({_last_error(h)})")
    return buf


def relaysum_load_state(h: int, buf) -> None:
    addr, nbytes = _buffer(buf)
    rc = load_library().relaysum_load_state(h, addr, nbytes)
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, f"relaysum_load_state ({_last_error(h)})")


def relaysum_poison_next(h: int) -> None:
    rc = load_library().relaysum_poison_next(h)
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, f"relaysum_poison_next ({_last_error(h)})")


def relaysum_step_static(n: int, d: int, edges, t: int, x, g, mom, lr: float, beta: float,
                         stream=None) -> None:
    """Round t of relaysum_step with the state in the library's static device
    buffer (no allocation; see relaysum.h)."""
    lib = load_library()
    e = np.ascontiguousarray(np.asarray(edges, dtype=np.int32).reshape(-1, 2))
    s = stream.cuda_stream if hasattr(stream, "cuda_stream") else stream
    rc = lib.relaysum_step_static(int(n), int(d),
                                  e.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)) if e.size else None,
                                  int(e.shape[0]), int(t), _addr(x), _addr(g), _addr(mom),
                                  float(lr), float(beta), s)
    if rc != RELAYSUM_OK:
        raise RelaySumError(rc, f"relaysum_step_static ({_last_error(None)})")


# ---- convenience wrapper ------------------------------------------------------


class RelaySum:
    """Owns one handle; `step(x, g, mom, lr, beta)` runs one round on torch
    tensors, on torch's current stream unless `stream` is given.  With
    `edges_b`, the handle relays over double binary trees (odd coordinates on
    `edges`, even ones on `edges_b`)."""

    def __init__(self, n: int, d: int, edges, stream=None, edges_b=None):
        self.n, self.d = int(n), int(d)
        self.h = None
        if edges_b is None:
            self.h = relaysum_create(n, d, edges)
        else:
            self.h = relaysum_create_double(n, d, edges, edges_b)
        self._stream = None
        if stream is not None:
            self.set_stream(stream)

    def set_stream(self, stream) -> None:
        self._stream = stream
        relaysum_set_stream(self.h, stream)

    def step(self, x, g, mom, lr: float, beta: float) -> None:
        _check_tensor(x, self.n, self.d, "x")
        _check_tensor(g, self.n, self.d, "g")
        _check_tensor(mom, self.n, self.d, "mom")
        if self._stream is None:
            import torch
            relaysum_set_stream(self.h, torch.cuda.current_stream())
        relaysum_step(self.h, x, g, mom, lr, beta)

    def step_ex(self, x, g, state1=None, state2=None, **kw) -> None:
        """One round under an update rule (model, robust, grad, mean) and a
        local optimizer (sgd, adam); keyword arguments as relaysum_step_ex."""
        for t, nm in ((x, "x"), (g, "g"), (state1, "state1"), (state2, "state2")):
            _check_tensor(t, self.n, self.d, nm)
        _check_mask(kw.get("dropped"), self.num_directed_edges)
        if self._stream is None:
            import torch
            relaysum_set_stream(self.h, torch.cuda.current_stream())
        relaysum_step_ex(self.h, x, g, state1, state2, **kw)

    def samples(self) -> np.ndarray:
        return relaysum_get_samples(self.h, self.n)

    def consensus_distance(self, x) -> tuple:
        """(consensus distance, largest coordinate deviation) of the models x."""
        _check_tensor(x, self.n, self.d, "x")
        if self._stream is None:
            import torch
            relaysum_set_stream(self.h, torch.cuda.current_stream())
        return relaysum_consensus_distance(self.h, x)

    def reset(self) -> None:
        relaysum_reset(self.h)

    @property
    def t(self) -> int:
        return relaysum_round(self.h)

    @property
    def num_trees(self) -> int:
        return relaysum_num_trees(self.h)

    @property
    def path(self) -> str:
        return relaysum_kernel_path(self.h)

    @property
    def num_directed_edges(self) -> int:
        return relaysum_num_directed_edges(self.h)

    def directed_edge(self, slot: int):
        return relaysum_directed_edge(self.h, slot)

    def counts(self):
        return relaysum_get_counts(self.h, self.n)

    def message(self, slot: int) -> np.ndarray:
        return relaysum_get_message(self.h, slot)

    @property
    def state_size(self) -> int:
        return relaysum_state_size(self.h)

    def save_state(self, buf=None):
        return relaysum_save_state(self.h, buf)

    def load_state(self, buf) -> None:
        relaysum_load_state(self.h, buf)

    def poison_next(self) -> None:
        relaysum_poison_next(self.h)

    def close(self) -> None:
        if getattr(self, "h", None):
            relaysum_destroy(self.h)
            self.h = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
