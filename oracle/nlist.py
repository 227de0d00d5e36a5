"""ctypes front end of the brute-force neighbour-list oracle (``nlist_ref.c``).

Paper Sec. II, the environment matrix: neighbours of atom i within r_c,
grouped by type into sel_beta slots each, sorted by distance inside a group,
unused slots empty (-1).  ``build()`` compiles the C file with gcc
(-O2 -ffp-contract=off -fopenmp); ``neighbour_list`` runs it for some or all
centre atoms.  Test infrastructure only.
"""
import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "nlist_ref.c")
_LIB = os.path.join(_HERE, "_build", "libnlist_ref.so")
_lib = None


def compile_source(src, out):
    tmp = out + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-fPIC",
                           "-shared", "-std=c11", src, "-o", tmp, "-lm"])
    os.replace(tmp, out)
    return out


def build(force=True):
    os.makedirs(os.path.dirname(_LIB), exist_ok=True)
    if force or not os.path.exists(_LIB):
        compile_source(SRC, _LIB)
    return _LIB


def load_library(path):
    lib = C.CDLL(path)
    lib.ref_nlist.restype = C.c_int
    lib.ref_nlist.argtypes = [C.c_int, C.c_void_p, C.c_void_p, C.c_int, C.c_void_p, C.c_double,
                              C.c_double, C.c_int, C.c_void_p, C.c_void_p, C.c_void_p]
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        _lib = load_library(_LIB)
    return _lib


def neighbour_list(coord, atype, sel, box, rc, centres=None, lib=None):
    """(nlist [n][sum(sel)] int32, counts [n][ntypes] int32, n_truncated) for
    the centre atoms ``centres`` (default: all)."""
    coord = np.ascontiguousarray(coord, np.float64)
    atype = np.ascontiguousarray(atype, np.int32)
    sel = np.ascontiguousarray(sel, np.int32)
    natoms = coord.shape[0]
    centres = np.arange(natoms, dtype=np.int64) if centres is None else \
        np.ascontiguousarray(centres, np.int64)
    nnei = int(sel.sum())
    nl = np.empty((len(centres), nnei), np.int32)
    cnt = np.empty((len(centres), len(sel)), np.int32)
    over = (lib or _load()).ref_nlist(natoms, coord.ctypes.data, atype.ctypes.data, len(sel),
                                      sel.ctypes.data, float(box), float(rc), len(centres),
                                      centres.ctypes.data, nl.ctypes.data, cnt.ctypes.data)
    return nl, cnt, int(over)
