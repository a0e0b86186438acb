"""CPU oracle for the local-shard SBP linear layer.

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg may import this package; the product path
(``paper_2301_06813_amd``) never does, and this package imports nothing from
it. The arithmetic lives in ``oracle.c`` (plain C, fp64 accumulation, and an
fp32-accumulating form of the same loop); this module only builds it, loads
it and marshals numpy arrays.

What it computes follows AutoDDL Sec. 4.2 (the SBP matrix multiplication and
its local matmul) and Sec. 4.3 (a broadcast weight receives partial-sum
gradients), on a 1-D mesh of p devices and on d-dimensional meshes (one state
per mesh axis, the ``nd_*`` functions); see the header of ``oracle.c``.

Parity status: pinned by ``tests/test_oracle_pins.py`` and, for meshes,
``tests/test_oracle_nd_pins.py`` (reassembly
invariant against brute-force global products, exact integer inputs, closed
forms, the p = 1 textbook case, Listing 1 shard shapes, bf16 rounding against
a library conversion). ``orc_round_bf16`` does not model bf16 subnormals
(never produced by the tests): parity unpinned below 2^-126.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
# ORACLE_SANITIZE=1: the default build is instrumented with AddressSanitizer
# and UndefinedBehaviorSanitizer (any finding aborts); the process must then
# preload the ASan runtime (tests/test_oracle_sanitized.py runs the oracle
# pins that way)
SANITIZE = os.environ.get("ORACLE_SANITIZE") == "1"
LIB = os.path.join(HERE, "liboracle_san.so" if SANITIZE else "liboracle.so")
SAN_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=all"]

# signature ids (the oracle's own numbering)
DP, COL, KS, PB, BP, BB = 0, 1, 2, 3, 4, 5
SIGNATURES = {"DP": DP, "COL": COL, "KS": KS, "PB": PB, "BP": BP, "BB": BB}
# operation ids
FWD, BWD_DATA, BWD_WEIGHT = 0, 1, 2
OPS = {"fwd": FWD, "bwd_data": BWD_DATA, "bwd_weight": BWD_WEIGHT}
# state kinds
SPLIT, BCAST, PARTIAL = 0, 1, 2
# attention-core products (see oracle.c)
ATT_S, ATT_O, ATT_DQ, ATT_DK, ATT_DP, ATT_DV = 0, 1, 2, 3, 4, 5
# input encodings
IN_BF16, IN_F32 = 0, 1


def build(force: bool = False, src: str = SRC, out: str = LIB) -> str:
    """Compile oracle.c (or a given copy of it) into a shared library with gcc.

    OpenMP parallelises over output elements only; -ffp-contract=off keeps
    every product and sum a separately rounded fp64 operation.
    """
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(src):
        tmp = out + ".tmp%d" % os.getpid()
        opt = SAN_FLAGS if (SANITIZE and out == LIB) else ["-O2"]
        cmd = ["gcc"] + opt + ["-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
                               "-std=c11", "-o", tmp, src, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, out)
    return out


class Oracle:
    """Handle on one build of the oracle library (the default build, or a
    mutated copy that a test compiles to check that the pins catch it)."""

    def __init__(self, path: str):
        lib = ctypes.CDLL(path)
        i64, i32 = ctypes.c_int64, ctypes.c_int32
        p64 = ctypes.POINTER(ctypes.c_int64)
        p32 = ctypes.POINTER(ctypes.c_int32)
        vp = ctypes.c_void_p
        lib.orc_split.argtypes = [i64, i64, i64, p64, p64]
        lib.orc_split.restype = None
        lib.orc_tags.argtypes = [ctypes.c_int, p32, p32]
        lib.orc_tags.restype = ctypes.c_int
        lib.orc_out_shape.argtypes = [ctypes.c_int, ctypes.c_int, i64, i64, i64, i64, i64,
                                      p64, p64, p32, p32]
        lib.orc_out_shape.restype = ctypes.c_int
        lib.orc_linear_block.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, i64, i64, i64,
                                         i64, i64, vp, vp, vp, i64, i64, i64, i64, vp]
        lib.orc_linear_block.restype = ctypes.c_int
        lib.orc_linear_samples.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, i64, i64, i64,
                                           i64, i64, vp, vp, vp, i64, vp, vp, vp]
        lib.orc_linear_samples.restype = ctypes.c_int
        lib.orc_linear_block_f32.argtypes = lib.orc_linear_block.argtypes
        lib.orc_linear_block_f32.restype = ctypes.c_int
        lib.orc_threads.argtypes = []
        lib.orc_threads.restype = ctypes.c_int
        lib.orc_set_threads.argtypes = [ctypes.c_int]
        lib.orc_set_threads.restype = None
        lib.orc_round_bf16.argtypes = [vp, vp, i64]
        lib.orc_round_bf16.restype = None
        ci = ctypes.c_int
        lib.orc_mesh_coord.argtypes = [ci, p32, p32, i64, i64, p32]
        lib.orc_mesh_coord.restype = ci
        lib.orc_nd_tags.argtypes = [ci, p32, p32, p32, p32, p32, p32]
        lib.orc_nd_tags.restype = ci
        lib.orc_nd_share.argtypes = [ci, p32, p32, p32, p32, i64, i64, p64]
        lib.orc_nd_share.restype = ci
        lib.orc_nd_out_shape.argtypes = [ci, i64, i64, i64, ci, p32, p32, p32, p32, p32, p32,
                                         p64, p64, p32, p32]
        lib.orc_nd_out_shape.restype = ci
        lib.orc_nd_linear_block.argtypes = [ci, ci, i64, i64, i64, ci, p32, p32, p32, p32, p32,
                                            p32, vp, vp, vp, i64, i64, i64, i64, vp]
        lib.orc_nd_linear_block.restype = ci
        lib.orc_nd_linear_samples.argtypes = [ci, ci, i64, i64, i64, ci, p32, p32, p32, p32, p32,
                                              p32, vp, vp, vp, i64, vp, vp, vp]
        lib.orc_nd_linear_samples.restype = ci
        lib.orc_attn.argtypes = [ci, ci, i64, i64, i64, i64, i64, i64, i64, vp, vp, vp]
        lib.orc_attn.restype = ci
        self.lib = lib

    def split(self, D: int, p: int, r: int) -> tuple[int, int]:
        """(offset, length) of rank r's contiguous block of an extent D over p ranks."""
        off, ln = ctypes.c_int64(), ctypes.c_int64()
        self.lib.orc_split(D, p, r, ctypes.byref(off), ctypes.byref(ln))
        return off.value, ln.value

    def tags(self, sig: int) -> list[tuple[int, int]]:
        """(kind, axis) of X, W, Y, dY, dX, dW under signature sig."""
        k = (ctypes.c_int32 * 6)()
        a = (ctypes.c_int32 * 6)()
        if self.lib.orc_tags(sig, k, a) != 0:
            raise ValueError("unknown signature %r" % sig)
        return [(k[t], a[t]) for t in range(6)]

    def out_shape(self, sig: int, op: int, M: int, K: int, N: int, p: int, r: int):
        """(rows, cols, kind, axis) of rank r's output of op under sig."""
        rows, cols = ctypes.c_int64(), ctypes.c_int64()
        kind, axis = ctypes.c_int32(), ctypes.c_int32()
        rc = self.lib.orc_out_shape(sig, op, M, K, N, p, r, ctypes.byref(rows),
                                    ctypes.byref(cols), ctypes.byref(kind), ctypes.byref(axis))
        if rc != 0:
            raise ValueError("bad oracle arguments")
        return rows.value, cols.value, kind.value, axis.value

    def linear(self, sig: int, op: int, X, W, dY, p: int, r: int, rows=None, cols=None,
               M=None, K=None, N=None) -> np.ndarray:
        """Rank r's output of op under sig, as fp64.

        X (M x K), W (K x N) and dY (M x N) are the global tensors: uint16 bf16
        bit patterns or float32, row-major. Pass None for a tensor the op does
        not read, together with the global sizes M, K, N. rows/cols select a
        block (Python ranges with step 1) of the local output.
        """
        (X, W, dY), enc = _prep(X, W, dY)
        M, K, N = _dims(X, W, dY, M, K, N)
        orow, ocol, _, _ = self.out_shape(sig, op, M, K, N, p, r)
        rows = range(orow) if rows is None else rows
        cols = range(ocol) if cols is None else cols
        out = np.empty((len(rows), len(cols)), dtype=np.float64)
        rc = self.lib.orc_linear_block(sig, op, enc, M, K, N, p, r, _ptr(X), _ptr(W), _ptr(dY),
                                       rows.start, rows.start + len(rows),
                                       cols.start, cols.start + len(cols), out.ctypes.data)
        if rc != 0:
            raise ValueError("bad oracle arguments")
        return out

    def linear_f32(self, sig: int, op: int, X, W, dY, p: int, r: int, rows=None, cols=None,
                   M=None, K=None, N=None) -> np.ndarray:
        """As linear(), with an fp32 accumulator (the plain fp32 triple loop):
        returns float32."""
        (X, W, dY), enc = _prep(X, W, dY)
        M, K, N = _dims(X, W, dY, M, K, N)
        orow, ocol, _, _ = self.out_shape(sig, op, M, K, N, p, r)
        rows = range(orow) if rows is None else rows
        cols = range(ocol) if cols is None else cols
        out = np.empty((len(rows), len(cols)), dtype=np.float32)
        rc = self.lib.orc_linear_block_f32(sig, op, enc, M, K, N, p, r, _ptr(X), _ptr(W),
                                           _ptr(dY), rows.start, rows.start + len(rows),
                                           cols.start, cols.start + len(cols), out.ctypes.data)
        if rc != 0:
            raise ValueError("bad oracle arguments")
        return out

    def threads(self) -> int:
        """Threads the oracle's parallel loops use."""
        return self.lib.orc_threads()

    def set_threads(self, n: int) -> None:
        self.lib.orc_set_threads(n)

    def linear_samples(self, sig: int, op: int, X, W, dY, p: int, r: int, ii, jj,
                       M=None, K=None, N=None) -> np.ndarray:
        """Single elements (ii[s], jj[s]) of rank r's output of op under sig, as fp64."""
        (X, W, dY), enc = _prep(X, W, dY)
        M, K, N = _dims(X, W, dY, M, K, N)
        ii = np.ascontiguousarray(ii, dtype=np.int64)
        jj = np.ascontiguousarray(jj, dtype=np.int64)
        out = np.empty(ii.shape[0], dtype=np.float64)
        rc = self.lib.orc_linear_samples(sig, op, enc, M, K, N, p, r, _ptr(X), _ptr(W),
                                         _ptr(dY), ii.shape[0], ii.ctypes.data,
                                         jj.ctypes.data, out.ctypes.data)
        if rc != 0:
            raise ValueError("bad oracle arguments")
        return out

    # --------------------------------------------------------- meshes
    def mesh_coord(self, nodes, gpus=None, node=0, gpu=0) -> list[int]:
        """Mesh coordinate of device (node, gpu); gpus None means one GPU per node."""
        d = len(nodes)
        gpus = [1] * d if gpus is None else list(gpus)
        c = (ctypes.c_int32 * d)()
        if self.lib.orc_mesh_coord(d, _i32(nodes), _i32(gpus), node, gpu, c) != 0:
            raise ValueError("bad mesh or device")
        return list(c)

    def nd_tags(self, xstates, wstates) -> list[list[tuple[int, int]]]:
        """Per tensor (X, W, Y, dY, dX, dW), the per-mesh-axis (kind, axis)
        states for X and W in the given per-axis (kind, axis) states."""
        d = len(xstates)
        kinds = (ctypes.c_int32 * (6 * d))()
        axes = (ctypes.c_int32 * (6 * d))()
        xk, xa = zip(*xstates)
        wk, wa = zip(*wstates)
        if self.lib.orc_nd_tags(d, _i32(xk), _i32(xa), _i32(wk), _i32(wa), kinds, axes) != 0:
            raise ValueError("no nd signature for these states")
        return [[(kinds[t * d + a], axes[t * d + a]) for a in range(d)] for t in range(6)]

    def nd_share(self, states, mesh, coord, rows, cols) -> tuple[int, int, int, int]:
        """(row offset, col offset, rows, cols) of the device's share."""
        d = len(mesh)
        k, a = zip(*states)
        out = (ctypes.c_int64 * 4)()
        if self.lib.orc_nd_share(d, _i32(k), _i32(a), _i32(mesh), _i32(coord), rows, cols,
                                 out) != 0:
            raise ValueError("bad nd layout")
        return tuple(out)

    def _nd_args(self, xstates, wstates, mesh, coord):
        xk, xa = zip(*xstates)
        wk, wa = zip(*wstates)
        return (len(mesh), _i32(mesh), _i32(coord), _i32(xk), _i32(xa), _i32(wk), _i32(wa))

    def nd_out_shape(self, op, M, K, N, xstates, wstates, mesh, coord):
        """(rows, cols, per-axis (kind, axis) states) of the device's output of op."""
        d = len(mesh)
        rows, cols = ctypes.c_int64(), ctypes.c_int64()
        kind, axis = (ctypes.c_int32 * d)(), (ctypes.c_int32 * d)()
        rc = self.lib.orc_nd_out_shape(op, M, K, N, *self._nd_args(xstates, wstates, mesh, coord),
                                       ctypes.byref(rows), ctypes.byref(cols), kind, axis)
        if rc != 0:
            raise ValueError("bad nd oracle arguments")
        return rows.value, cols.value, list(zip(kind, axis))

    def nd_linear(self, op, X, W, dY, xstates, wstates, mesh, coord, rows=None, cols=None,
                  M=None, K=None, N=None) -> np.ndarray:
        """The device's output of op (fp64) for X and W in per-axis states
        xstates and wstates ((kind, axis) per mesh axis) on mesh `mesh`, at
        mesh coordinate `coord`. Inputs as for linear()."""
        (X, W, dY), enc = _prep(X, W, dY)
        M, K, N = _dims(X, W, dY, M, K, N)
        orow, ocol, _ = self.nd_out_shape(op, M, K, N, xstates, wstates, mesh, coord)
        rows = range(orow) if rows is None else rows
        cols = range(ocol) if cols is None else cols
        out = np.empty((len(rows), len(cols)), dtype=np.float64)
        rc = self.lib.orc_nd_linear_block(op, enc, M, K, N,
                                          *self._nd_args(xstates, wstates, mesh, coord),
                                          _ptr(X), _ptr(W), _ptr(dY), rows.start,
                                          rows.start + len(rows), cols.start,
                                          cols.start + len(cols), out.ctypes.data)
        if rc != 0:
            raise ValueError("bad nd oracle arguments")
        return out

    def nd_linear_samples(self, op, X, W, dY, xstates, wstates, mesh, coord, ii, jj,
                          M=None, K=None, N=None) -> np.ndarray:
        """Single elements (ii[s], jj[s]) of the device's output of op, as fp64."""
        (X, W, dY), enc = _prep(X, W, dY)
        M, K, N = _dims(X, W, dY, M, K, N)
        ii = np.ascontiguousarray(ii, dtype=np.int64)
        jj = np.ascontiguousarray(jj, dtype=np.int64)
        out = np.empty(ii.shape[0], dtype=np.float64)
        rc = self.lib.orc_nd_linear_samples(op, enc, M, K, N,
                                            *self._nd_args(xstates, wstates, mesh, coord),
                                            _ptr(X), _ptr(W), _ptr(dY), ii.shape[0],
                                            ii.ctypes.data, jj.ctypes.data, out.ctypes.data)
        if rc != 0:
            raise ValueError("bad nd oracle arguments")
        return out

    # ------------------------------------------------ attention core
    def attn(self, which, T1, T2, p, r, sq, sk, d) -> np.ndarray:
        """Device r's output of attention product `which` (ATT_*) under a head
        split over p devices, as fp64 [batch][local heads][rows][cols]. T1 and
        T2 are the operands in the order of the product's definition,
        contiguous [batch][heads][rows][cols], bf16 bits (uint16) or fp32."""
        (T1, T2, _), enc = _prep(T1, T2, None)
        nb, nh = T1.shape[:2]
        _, hr = self.split(nh, p, r)
        shapes = {ATT_S: (sq, sk), ATT_O: (sq, d), ATT_DQ: (sq, d), ATT_DK: (sk, d),
                  ATT_DP: (sq, sk), ATT_DV: (sk, d)}
        if which not in shapes:
            raise ValueError("unknown attention product %r" % which)
        rows, cols = shapes[which]
        out = np.empty((nb, hr, rows, cols), dtype=np.float64)
        rc = self.lib.orc_attn(which, enc, nb, nh, sq, sk, d, p, r, _ptr(T1), _ptr(T2),
                               out.ctypes.data)
        if rc != 0:
            raise ValueError("bad attention oracle arguments")
        return out

    def round_bf16(self, x) -> np.ndarray:
        """Round fp64 values to bf16 (nearest, ties to even); returns uint16 bit patterns."""
        x = np.ascontiguousarray(x, dtype=np.float64)
        out = np.empty(x.shape, dtype=np.uint16)
        self.lib.orc_round_bf16(x.ctypes.data, out.ctypes.data, x.size)
        return out


def _encode(a):
    """Return (contiguous array, encoding) for bf16 bit patterns (uint16) or fp32."""
    if a is None:
        return None, None
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return a, IN_BF16
    if a.dtype == np.float32:
        return a, IN_F32
    raise TypeError("oracle inputs are uint16 bf16 bit patterns or float32, got %s" % a.dtype)


def _prep(X, W, dY):
    arrs, encs = [], set()
    for a in (X, W, dY):
        c, e = _encode(a)
        arrs.append(c)
        if e is not None:
            encs.add(e)
    if len(encs) != 1:
        raise TypeError("oracle inputs must share one encoding")
    return arrs, encs.pop()


def _dims(X, W, dY, M, K, N):
    if X is not None:
        M, K = X.shape
    if W is not None:
        K, N = W.shape
    if dY is not None:
        M, N = dY.shape
    return M, K, N


def _ptr(a):
    return None if a is None else a.ctypes.data


def _i32(vals):
    vals = list(vals)
    return (ctypes.c_int32 * max(1, len(vals)))(*vals)


_default = None


def default() -> Oracle:
    """The oracle built from oracle.c (built on first use if missing)."""
    global _default
    if _default is None:
        if not os.path.exists(LIB):
            build()
        _default = Oracle(LIB)
    return _default


def split(D, p, r):
    return default().split(D, p, r)


def tags(sig):
    return default().tags(sig)


def out_shape(sig, op, M, K, N, p, r):
    return default().out_shape(sig, op, M, K, N, p, r)


def linear(sig, op, X, W, dY, p, r, rows=None, cols=None, M=None, K=None, N=None):
    return default().linear(sig, op, X, W, dY, p, r, rows, cols, M, K, N)


def linear_samples(sig, op, X, W, dY, p, r, ii, jj, M=None, K=None, N=None):
    return default().linear_samples(sig, op, X, W, dY, p, r, ii, jj, M, K, N)


def linear_f32(sig, op, X, W, dY, p, r, rows=None, cols=None, M=None, K=None, N=None):
    return default().linear_f32(sig, op, X, W, dY, p, r, rows, cols, M, K, N)


def threads() -> int:
    return default().threads()


def set_threads(n: int) -> None:
    default().set_threads(n)


def round_bf16(x) -> np.ndarray:
    return default().round_bf16(x)


def attn(which, T1, T2, p, r, sq, sk, d):
    return default().attn(which, T1, T2, p, r, sq, sk, d)


def mesh_coord(nodes, gpus=None, node=0, gpu=0):
    return default().mesh_coord(nodes, gpus, node, gpu)


def nd_tags(xstates, wstates):
    return default().nd_tags(xstates, wstates)


def nd_share(states, mesh, coord, rows, cols):
    return default().nd_share(states, mesh, coord, rows, cols)


def nd_out_shape(op, M, K, N, xstates, wstates, mesh, coord):
    return default().nd_out_shape(op, M, K, N, xstates, wstates, mesh, coord)


def nd_linear(op, X, W, dY, xstates, wstates, mesh, coord, rows=None, cols=None,
              M=None, K=None, N=None):
    return default().nd_linear(op, X, W, dY, xstates, wstates, mesh, coord, rows, cols, M, K, N)


def nd_linear_samples(op, X, W, dY, xstates, wstates, mesh, coord, ii, jj, M=None, K=None,
                      N=None):
    return default().nd_linear_samples(op, X, W, dY, xstates, wstates, mesh, coord, ii, jj,
                                       M, K, N)


def bf16_to_f64(bits) -> np.ndarray:
    """Decode uint16 bf16 bit patterns exactly."""
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
