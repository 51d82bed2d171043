"""RelaySum oracle (test infrastructure only).

Plain CPU implementations of what one RelaySGD round computes, written from
the paper's Alg. 1 (RelaySum/Model) and its Nesterov-momentum local step
(Appendix D.2):

* ``Oracle``          -- the C oracle (relaysum_oracle.c) in float or double,
                         through ctypes;
* ``oracle.exact``    -- the same round in exact rational arithmetic,
                         pure-Python loops, for tiny trees.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline
leg may import this package.  The product library never does, and this
package never imports the product.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
_SRC = os.path.join(_HERE, "relaysum_oracle.c")
_INC = os.path.join(_HERE, "relaysum_round.inc")

# -O2, IEEE semantics: no contraction into FMA, no reassociation, no FTZ.
CFLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-shared", "-fPIC",
          "-std=c11", "-Wall", "-Wextra"]
LDLIBS = ["-lm"]


def build(verbose: bool = False) -> str:
    """Compile liboracle.so next to its source (always recompiles)."""
    tmp = LIB_PATH + ".tmp"
    cmd = ["gcc", *CFLAGS, "-o", tmp, _SRC, *LDLIBS]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True, cwd=_HERE)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH) or os.path.getmtime(LIB_PATH) < max(
            os.path.getmtime(_SRC), os.path.getmtime(_INC)):
        build()
    lib = ctypes.CDLL(LIB_PATH)
    for p, real in (("f32", ctypes.c_float), ("f64", ctypes.c_double)):
        ptr = ctypes.POINTER(real)
        f = getattr(lib, f"oracle_{p}_create")
        f.restype = ctypes.c_void_p
        f.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.c_int, ctypes.POINTER(ctypes.c_int)]
        f = getattr(lib, f"oracle_{p}_destroy")
        f.restype = None
        f.argtypes = [ctypes.c_void_p]
        f = getattr(lib, f"oracle_{p}_reset")
        f.restype = None
        f.argtypes = [ctypes.c_void_p]
        f = getattr(lib, f"oracle_{p}_round")
        f.restype = ctypes.c_int
        f.argtypes = [ctypes.c_void_p, ptr, ptr, ptr, real, real]
        f = getattr(lib, f"oracle_{p}_round_ex")
        f.restype = ctypes.c_int
        f.argtypes = [ctypes.c_void_p, ptr, ptr, ptr, ptr, ctypes.c_int, ctypes.c_int, real, real,
                      real, real, ctypes.c_int64, ctypes.POINTER(ctypes.c_ubyte)]
        f = getattr(lib, f"oracle_{p}_samples")
        f.restype = ctypes.c_int64
        f.argtypes = [ctypes.c_void_p, ctypes.c_int]
        f = getattr(lib, f"oracle_{p}_rounds")
        f.restype = ctypes.c_int64
        f.argtypes = [ctypes.c_void_p]
        f = getattr(lib, f"oracle_{p}_count")
        f.restype = ctypes.c_int
        f.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int]
        f = getattr(lib, f"oracle_{p}_nbar")
        f.restype = ctypes.c_int
        f.argtypes = [ctypes.c_void_p, ctypes.c_int]
        f = getattr(lib, f"oracle_{p}_message")
        f.restype = ctypes.c_int
        f.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ptr]
    lib.oracle_set_threads.restype = None
    lib.oracle_set_threads.argtypes = [ctypes.c_int]
    lib.oracle_get_threads.restype = ctypes.c_int
    lib.oracle_get_threads.argtypes = []
    _lib = lib
    return lib


def set_threads(k: int) -> None:
    _load().oracle_set_threads(int(k))


def get_threads() -> int:
    return int(_load().oracle_get_threads())


class Oracle:
    """RelaySum state of n workers on a tree, in float32 or float64.

    ``round(x, g, mom, lr, beta)`` performs one Alg. 1 iteration for every
    worker; ``x`` and ``mom`` ([n, d] C-contiguous numpy arrays of the
    oracle's dtype) are updated in place, as in the paper's algorithm
    statement.  ``mom`` may be None when beta == 0.
    """

    def __init__(self, n: int, d: int, edges, dtype=np.float32):
        self.lib = _load()
        self.dtype = np.dtype(dtype)
        if self.dtype == np.float32:
            self.p, self.real = "f32", ctypes.c_float
        elif self.dtype == np.float64:
            self.p, self.real = "f64", ctypes.c_double
        else:
            raise ValueError("oracle dtype must be float32 or float64")
        self.n, self.d = int(n), int(d)
        e = np.ascontiguousarray(np.asarray(edges, dtype=np.int32).reshape(-1, 2))
        self.edges = e
        self.h = getattr(self.lib, f"oracle_{self.p}_create")(
            self.n, self.d, int(e.shape[0]),
            e.ctypes.data_as(ctypes.POINTER(ctypes.c_int)) if e.size else None)
        if not self.h:
            raise ValueError("not a tree on n nodes (or out of memory)")

    def _fn(self, name):
        return getattr(self.lib, f"oracle_{self.p}_{name}")

    def _ptr(self, a):
        return a.ctypes.data_as(ctypes.POINTER(self.real))

    def _check(self, a, name, writable):
        if a.dtype != self.dtype or a.shape != (self.n, self.d) or not a.flags.c_contiguous:
            raise ValueError(f"{name} must be a C-contiguous {self.dtype} array [{self.n}, {self.d}]")
        if writable and not a.flags.writeable:
            raise ValueError(f"{name} must be writable")

    def round(self, x, g, mom, lr: float, beta: float) -> None:
        self._check(x, "x", True)
        self._check(g, "g", False)
        if mom is not None:
            self._check(mom, "mom", True)
        elif beta != 0.0:
            raise ValueError("mom is required when beta != 0")
        rc = self._fn("round")(self.h, self._ptr(x), self._ptr(g),
                               self._ptr(mom) if mom is not None else None,
                               self.real(lr), self.real(beta))
        if rc != 0:
            raise RuntimeError(f"oracle round failed ({rc})")

    UPDATES = {"model": 0, "robust": 1, "grad": 2, "mean": 3}
    OPTIMIZERS = {"sgd": 0, "adam": 1}

    def round_ex(self, x, g, s1=None, s2=None, *, update="model", optimizer="sgd", lr=0.0,
                 beta1=0.0, beta2=0.0, eps=0.0, adam_step=0, dropped=None) -> None:
        """One round of Alg. 1 (update="model"), eq. robust ("robust"), Alg. 4
        ("grad") or Alg. 3 ("mean"), with SGD/Nesterov or Adam local steps.

        s1, s2: optimizer state ([n, d]): Nesterov buffer in s1; Adam's first
        and second moments in s1, s2; for "mean", the running sums y in s1.
        dropped: None, or an [n, n] array whose (k, i) entry is nonzero when
        the message k -> i of this round is lost.
        """
        self._check(x, "x", True)
        self._check(g, "g", False)
        for a, nm in ((s1, "s1"), (s2, "s2")):
            if a is not None:
                self._check(a, nm, True)
        drop_ptr = None
        if dropped is not None:
            dm = np.ascontiguousarray(np.asarray(dropped, dtype=np.uint8).reshape(self.n, self.n))
            drop_ptr = dm.ctypes.data_as(ctypes.POINTER(ctypes.c_ubyte))
        rc = self._fn("round_ex")(
            self.h, self._ptr(x), self._ptr(g),
            self._ptr(s1) if s1 is not None else None, self._ptr(s2) if s2 is not None else None,
            self.UPDATES[update], self.OPTIMIZERS[optimizer], self.real(lr), self.real(beta1),
            self.real(beta2), self.real(eps), int(adam_step), drop_ptr)
        if rc != 0:
            raise RuntimeError(f"oracle round_ex failed ({rc})")

    def samples(self, i: int) -> int:
        """Mean estimation: number of samples summed into worker i's y so far."""
        return int(self._fn("samples")(self.h, int(i)))

    @property
    def t(self) -> int:
        return int(self._fn("rounds")(self.h))

    def count(self, src: int, dst: int) -> int:
        """c_{src->dst} sent in the last round (-1 if not an edge)."""
        return int(self._fn("count")(self.h, int(src), int(dst)))

    def nbar(self, i: int) -> int:
        """nbar_i of the last round's average."""
        return int(self._fn("nbar")(self.h, int(i)))

    def nbars(self) -> np.ndarray:
        return np.array([self.nbar(i) for i in range(self.n)], dtype=np.int32)

    def message(self, src: int, dst: int) -> np.ndarray:
        """m_{src->dst} sent in the last round."""
        out = np.empty(self.d, dtype=self.dtype)
        if self._fn("message")(self.h, int(src), int(dst), self._ptr(out)) != 0:
            raise ValueError(f"({src},{dst}) is not an edge")
        return out

    def reset(self) -> None:
        self._fn("reset")(self.h)

    def close(self) -> None:
        if getattr(self, "h", None):
            self._fn("destroy")(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
