"""ctypes front end of the plain C oracle (``se_a_ref.c``).

``build()`` compiles it with gcc (-O2 -ffp-contract=off -fopenmp) into
``oracle/_build/libse_a_ref.so``; ``forward``/``backward`` run it over a
range of atoms.  Tables come from ``oracle.table`` and are flattened into the
oracle's own layout [pair][l][m][q] (q = power of t).
"""
import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "se_a_ref.c")
_LIB = os.path.join(_HERE, "_build", "libse_a_ref.so")
_lib = None


def compile_source(src, out):
    """Compile a C oracle source file into the shared library ``out``."""
    tmp = out + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-fPIC",
                           "-shared", "-std=c11", src, "-o", tmp, "-lm"])
    os.replace(tmp, out)
    return out


def build(force=True):
    os.makedirs(os.path.dirname(_LIB), exist_ok=True)
    if force or not os.path.exists(_LIB):
        compile_source(_SRC, _LIB)
    return _LIB


class _Args(C.Structure):
    _fields_ = [("nloc", C.c_int), ("nnei", C.c_int), ("ntypes", C.c_int),
                ("M", C.c_int), ("M2", C.c_int),
                ("sel", C.c_void_p), ("lo", C.c_void_p), ("d1", C.c_void_p),
                ("L1", C.c_void_p), ("d2", C.c_void_p), ("L2", C.c_void_p),
                ("off", C.c_void_p), ("coef", C.c_void_p), ("atype", C.c_void_p),
                ("nlist", C.c_void_p), ("em", C.c_void_p)]


def load_library(path):
    """ctypes handle of a compiled C oracle (the default one, or a copy built
    from a modified source by a test)."""
    lib = C.CDLL(path)
    for fn in (lib.ref_forward, lib.ref_backward):
        fn.restype = None
    lib.ref_num_threads.restype = C.c_int
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        _lib = load_library(_LIB)
    return _lib


def num_threads():
    return int(_load().ref_num_threads())


class Problem:
    """Holds contiguous inputs and the flattened tables for the C oracle."""

    def __init__(self, em, nlist, atype, tables, sel, m2, lib=None):
        self._lib = lib
        self.em = np.ascontiguousarray(em, np.float64)
        self.nlist = np.ascontiguousarray(nlist, np.int32)
        self.atype = np.ascontiguousarray(atype, np.int32)
        self.sel = np.ascontiguousarray(sel, np.int32)
        self.m2 = int(m2)
        self.M = tables[0].M
        self.lo = np.array([t.lo for t in tables], np.float64)
        self.d1 = np.array([t.d1 for t in tables], np.float64)
        self.L1 = np.array([t.L1 for t in tables], np.int64)
        self.d2 = np.array([t.d2 for t in tables], np.float64)
        self.L2 = np.array([t.L2 for t in tables], np.int64)
        sizes = [t.coef.size for t in tables]
        self.off = np.concatenate([[0], np.cumsum(sizes)[:-1]]).astype(np.int64)
        self.coef = np.ascontiguousarray(np.concatenate([t.coef.ravel() for t in tables]))
        a = _Args()
        a.nloc, a.nnei = self.nlist.shape
        a.ntypes, a.M, a.M2 = len(self.sel), self.M, self.m2
        for name in ("sel", "lo", "d1", "L1", "d2", "L2", "off", "coef", "atype", "nlist", "em"):
            setattr(a, name, getattr(self, name).ctypes.data)
        self._args = a

    def forward(self, i0=0, i1=None):
        i1 = self.nlist.shape[0] if i1 is None else i1
        T = np.empty((i1 - i0, self.M, 4))
        D = np.empty((i1 - i0, self.M, self.m2))
        (self._lib or _load()).ref_forward(C.byref(self._args), C.c_int64(i0), C.c_int64(i1),
                            T.ctypes.data_as(C.c_void_p), D.ctypes.data_as(C.c_void_p))
        return T, D

    def backward(self, dT, i0=0, i1=None):
        """dT holds the rows of atoms i0..i1-1."""
        i1 = self.nlist.shape[0] if i1 is None else i1
        dT = np.ascontiguousarray(dT, np.float64)
        assert dT.shape == (i1 - i0, self.M, 4)
        dR = np.empty((i1 - i0, self.nlist.shape[1], 4))
        (self._lib or _load()).ref_backward(C.byref(self._args), C.c_int64(i0), C.c_int64(i1),
                             dT.ctypes.data_as(C.c_void_p), dR.ctypes.data_as(C.c_void_p))
        return dR
