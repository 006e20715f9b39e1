"""CPU oracle for the causal KATA-M1 forward, backward and decode step, for the
block-diagonal KATA-Mg variant, and for normalised linear attention with the
linear (n_psi ~ d) feature maps (test infrastructure).

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never does: it
shares no code with it, and it never falls back to it.

The arithmetic lives in ``kata_oracle.c`` (plain C, IEEE double, OpenMP over
independent rows); this module only builds that file with ``gcc`` and
marshals numpy arrays through ``ctypes``.  Every function cites the passage of
the paper it follows in the C source.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kata_oracle.c")
_LIB = os.path.join(_HERE, "libkata_oracle.so")
_lib = None

_dp = ctypes.POINTER(ctypes.c_double)
_lp = ctypes.POINTER(ctypes.c_long)
_L = ctypes.c_long


def build(src: str = _SRC, out: str = _LIB, extra_flags=()) -> str:
    """Compile the oracle into a shared library with gcc (-O2, OpenMP)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
           "-fvisibility=hidden", *extra_flags, src, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def load(path: str | None = None):
    """Load (building first if needed) the oracle library."""
    global _lib
    if path is None and _lib is not None:
        return _lib
    p = path or _LIB
    if path is None and (not os.path.exists(p) or
                         os.path.getmtime(p) < os.path.getmtime(_SRC)):
        build()
    lib = ctypes.CDLL(p)
    lib.kata_oracle_num_threads.restype = ctypes.c_int
    lib.kata_oracle_packed_dim.restype = _L
    lib.kata_oracle_packed_dim.argtypes = [_L]
    lib.kata_oracle_packed_index.restype = _L
    lib.kata_oracle_packed_index.argtypes = [_L, _L, _L]
    lib.kata_oracle_phi.argtypes = [_dp, _L, ctypes.c_int, _dp]
    lib.kata_oracle_fwd.argtypes = [_dp, _dp, _dp, _dp, _L, _L, _L, _L, _L]
    lib.kata_oracle_den.argtypes = [_dp, _dp, _dp, _L, _L, _L, _L]
    lib.kata_oracle_fwd_rows.argtypes = [_dp, _dp, _dp, _L, _L, _L, _L, _L,
                                         _lp, _lp, _L, _dp]
    lib.kata_oracle_scan_exclusive.argtypes = [_dp, _L, _L, ctypes.c_int]
    lib.kata_oracle_fwd_chunked.argtypes = [_dp, _dp, _dp, _dp, _L, _L, _L, _L,
                                            _L, _L, ctypes.c_int]
    lib.kata_oracle_state.argtypes = [_dp, _dp, _dp, _dp, _L, _L, _L, _L, _L]
    lib.kata_oracle_decode_step.argtypes = [_dp, _dp, _dp, _dp, _dp, _dp,
                                            _L, _L, _L, _L]
    lib.kata_oracle_packed_dim_mg.restype = _L
    lib.kata_oracle_packed_dim_mg.argtypes = [_L, _L]
    lib.kata_oracle_phi_mg.argtypes = [_dp, _L, _L, ctypes.c_int, _dp]
    lib.kata_oracle_fwd_mg.argtypes = [_dp, _dp, _dp, _dp, _L, _L, _L, _L, _L, _L]
    lib.kata_oracle_fwd_mg_rows.argtypes = [_dp, _dp, _dp, _L, _L, _L, _L, _L, _L,
                                            _lp, _lp, _L, _dp]
    lib.kata_oracle_fwd_chunked_mg.argtypes = [_dp, _dp, _dp, _dp, _L, _L, _L, _L,
                                               _L, _L, _L, ctypes.c_int]
    lib.kata_oracle_state_mg.argtypes = [_dp, _dp, _dp, _dp, _L, _L, _L, _L, _L, _L]
    lib.kata_oracle_decode_step_mg.argtypes = [_dp, _dp, _dp, _dp, _dp, _dp,
                                               _L, _L, _L, _L, _L]
    lib.kata_oracle_bwd_mg.argtypes = [_dp, _dp, _dp, _dp, _dp, _dp, _dp, _L, _L, _L, _L, _L,
                                       _L]
    lib.kata_oracle_bwd_chunked_mg.argtypes = [_dp, _dp, _dp, _dp, _dp, _dp, _dp, _L, _L, _L,
                                               _L, _L, _L, _L, ctypes.c_int]
    lib.kata_oracle_lin_dim.restype = _L
    lib.kata_oracle_lin_dim.argtypes = [_L, ctypes.c_int]
    lib.kata_oracle_lin_feature.argtypes = [_dp, _L, ctypes.c_int, ctypes.c_double, _dp]
    lib.kata_oracle_lin_fwd.argtypes = [_dp, _dp, _dp, _dp, _L, _L, _L, _L, _L,
                                        ctypes.c_int, ctypes.c_double, ctypes.c_int]
    lib.kata_oracle_lin_fwd_rows.argtypes = [_dp, _dp, _dp, _L, _L, _L, _L, _L,
                                             ctypes.c_int, ctypes.c_double, ctypes.c_int,
                                             _lp, _lp, _L, _dp]
    lib.kata_oracle_lin_fwd_chunked.argtypes = [_dp, _dp, _dp, _dp, _L, _L, _L, _L, _L,
                                                _L, ctypes.c_int, ctypes.c_double,
                                                ctypes.c_int, ctypes.c_int]
    if path is None:
        _lib = lib
    return lib


class Oracle:
    """numpy front end over one loaded copy of the oracle library."""

    def __init__(self, lib=None):
        self.lib = lib if lib is not None else load()

    @staticmethod
    def _f64(a):
        return np.ascontiguousarray(np.asarray(a, dtype=np.float64))

    @staticmethod
    def _p(a):
        return a.ctypes.data_as(_dp)

    def num_threads(self) -> int:
        return int(self.lib.kata_oracle_num_threads())

    def packed_dim(self, d: int) -> int:
        return int(self.lib.kata_oracle_packed_dim(d))

    def packed_index(self, a: int, b: int, d: int) -> int:
        return int(self.lib.kata_oracle_packed_index(a, b, d))

    def phi(self, x, weighted: bool = False):
        x = self._f64(x)
        d = x.shape[-1]
        out = np.empty(self.packed_dim(d))
        self.lib.kata_oracle_phi(self._p(x), d, int(weighted), self._p(out))
        return out

    def fwd(self, q, k, v):
        """Definition forward; q, k: [B,H,T,d], v: [B,H,T,dv] -> [B,H,T,dv]."""
        q, k, v = self._f64(q), self._f64(k), self._f64(v)
        B, H, T, d = q.shape
        dv = v.shape[-1]
        out = np.empty((B, H, T, dv))
        self.lib.kata_oracle_fwd(self._p(q), self._p(k), self._p(v), self._p(out),
                                 B, H, T, d, dv)
        return out

    def den(self, q, k):
        """Row denominators of the definition, sum_{i<=t} (q_t . k_i)^2:
        q, k [B,H,T,d] -> [B,H,T]."""
        q, k = self._f64(q), self._f64(k)
        B, H, T, d = q.shape
        out = np.empty((B, H, T))
        self.lib.kata_oracle_den(self._p(q), self._p(k), self._p(out), B, H, T, d)
        return out

    def fwd_rows(self, q, k, v, bh_idx, t_idx):
        """Definition at listed (flattened head, token) rows -> [nrows, dv]."""
        q, k, v = self._f64(q), self._f64(k), self._f64(v)
        B, H, T, d = q.shape
        dv = v.shape[-1]
        bh = np.ascontiguousarray(np.asarray(bh_idx, dtype=np.int64))
        tt = np.ascontiguousarray(np.asarray(t_idx, dtype=np.int64))
        assert bh.shape == tt.shape and bh.ndim == 1
        assert (bh >= 0).all() and (bh < B * H).all() and (tt >= 0).all() and (tt < T).all()
        out = np.empty((bh.size, dv))
        self.lib.kata_oracle_fwd_rows(self._p(q), self._p(k), self._p(v), B, H, T, d, dv,
                                      bh.ctypes.data_as(_lp), tt.ctypes.data_as(_lp),
                                      bh.size, self._p(out))
        return out

    def scan_exclusive(self, x, mode: int):
        """Exclusive prefix over axis 0 of x ([N, ...]); mode 0 sequential, 1 tree."""
        x = self._f64(x).copy()
        N = x.shape[0]
        E = int(np.prod(x.shape[1:])) if x.ndim > 1 else 1
        self.lib.kata_oracle_scan_exclusive(self._p(x), N, E, mode)
        return x

    def fwd_chunked(self, q, k, v, C: int, scan_mode: int = 1):
        q, k, v = self._f64(q), self._f64(k), self._f64(v)
        B, H, T, d = q.shape
        dv = v.shape[-1]
        out = np.empty((B, H, T, dv))
        self.lib.kata_oracle_fwd_chunked(self._p(q), self._p(k), self._p(v), self._p(out),
                                         B, H, T, d, dv, C, scan_mode)
        return out

    def state(self, k, v):
        """Packed state after all T tokens: S [B,H,n,dv], z [B,H,n]."""
        k, v = self._f64(k), self._f64(v)
        B, H, T, d = k.shape
        dv = v.shape[-1]
        n = self.packed_dim(d)
        S = np.empty((B, H, n, dv))
        z = np.empty((B, H, n))
        self.lib.kata_oracle_state(self._p(k), self._p(v), self._p(S), self._p(z),
                                   B, H, T, d, dv)
        return S, z

    def decode_step(self, S, z, q, k, v):
        """One decode step; returns (out [B,H,dv], S', z') without touching inputs."""
        S, z = self._f64(S).copy(), self._f64(z).copy()
        q, k, v = self._f64(q), self._f64(k), self._f64(v)
        B, H, d = q.shape
        dv = v.shape[-1]
        out = np.empty((B, H, dv))
        self.lib.kata_oracle_decode_step(self._p(S), self._p(z), self._p(q), self._p(k),
                                         self._p(v), self._p(out), B, H, d, dv)
        return out, S, z

    # ---- KATA-Mg (g blocks of d/g coordinates; g = 1 is KATA-M1) ----------

    def packed_dim_mg(self, d: int, g: int) -> int:
        return int(self.lib.kata_oracle_packed_dim_mg(d, g))

    def phi_mg(self, x, g: int, weighted: bool = False):
        x = self._f64(x)
        d = x.shape[-1]
        out = np.empty(self.packed_dim_mg(d, g))
        self.lib.kata_oracle_phi_mg(self._p(x), d, g, int(weighted), self._p(out))
        return out

    def fwd_mg(self, q, k, v, g: int):
        q, k, v = self._f64(q), self._f64(k), self._f64(v)
        B, H, T, d = q.shape
        dv = v.shape[-1]
        assert d % g == 0
        out = np.empty((B, H, T, dv))
        self.lib.kata_oracle_fwd_mg(self._p(q), self._p(k), self._p(v), self._p(out),
                                    B, H, T, d, dv, g)
        return out

    def fwd_mg_rows(self, q, k, v, g: int, bh_idx, t_idx):
        q, k, v = self._f64(q), self._f64(k), self._f64(v)
        B, H, T, d = q.shape
        dv = v.shape[-1]
        assert d % g == 0
        bh = np.ascontiguousarray(np.asarray(bh_idx, dtype=np.int64))
        tt = np.ascontiguousarray(np.asarray(t_idx, dtype=np.int64))
        assert bh.shape == tt.shape and bh.ndim == 1
        assert (bh >= 0).all() and (bh < B * H).all() and (tt >= 0).all() and (tt < T).all()
        out = np.empty((bh.size, dv))
        self.lib.kata_oracle_fwd_mg_rows(self._p(q), self._p(k), self._p(v), B, H, T, d, dv,
                                         g, bh.ctypes.data_as(_lp), tt.ctypes.data_as(_lp),
                                         bh.size, self._p(out))
        return out

    def fwd_chunked_mg(self, q, k, v, C: int, g: int, scan_mode: int = 1):
        q, k, v = self._f64(q), self._f64(k), self._f64(v)
        B, H, T, d = q.shape
        dv = v.shape[-1]
        assert d % g == 0
        out = np.empty((B, H, T, dv))
        self.lib.kata_oracle_fwd_chunked_mg(self._p(q), self._p(k), self._p(v), self._p(out),
                                            B, H, T, d, dv, C, g, scan_mode)
        return out

    def state_mg(self, k, v, g: int):
        k, v = self._f64(k), self._f64(v)
        B, H, T, d = k.shape
        dv = v.shape[-1]
        n = self.packed_dim_mg(d, g)
        S = np.empty((B, H, n, dv))
        z = np.empty((B, H, n))
        self.lib.kata_oracle_state_mg(self._p(k), self._p(v), self._p(S), self._p(z),
                                      B, H, T, d, dv, g)
        return S, z

    def decode_step_mg(self, S, z, q, k, v, g: int):
        S, z = self._f64(S).copy(), self._f64(z).copy()
        q, k, v = self._f64(q), self._f64(k), self._f64(v)
        B, H, d = q.shape
        dv = v.shape[-1]
        out = np.empty((B, H, dv))
        self.lib.kata_oracle_decode_step_mg(self._p(S), self._p(z), self._p(q), self._p(k),
                                            self._p(v), self._p(out), B, H, d, dv, g)
        return out, S, z

    # ---- backward of KATA-Mg (g = 1: KATA-M1) ----------------------------

    def bwd_mg(self, q, k, v, dout, g: int = 1):
        """Gradients (dq, dk, dv) of sum_t <dout_t, o_t> by the definition."""
        q, k, v, dout = self._f64(q), self._f64(k), self._f64(v), self._f64(dout)
        B, H, T, d = q.shape
        dv = v.shape[-1]
        assert d % g == 0 and dout.shape == v.shape
        gq, gk, gv = np.empty(q.shape), np.empty(k.shape), np.empty(v.shape)
        self.lib.kata_oracle_bwd_mg(self._p(q), self._p(k), self._p(v), self._p(dout),
                                    self._p(gq), self._p(gk), self._p(gv), B, H, T, d, dv, g)
        return gq, gk, gv

    def bwd_chunked_mg(self, q, k, v, dout, C: int, g: int = 1, scan_mode: int = 1):
        """The same gradients by the chunked reverse-scan form."""
        q, k, v, dout = self._f64(q), self._f64(k), self._f64(v), self._f64(dout)
        B, H, T, d = q.shape
        dv = v.shape[-1]
        assert d % g == 0 and dout.shape == v.shape
        gq, gk, gv = np.empty(q.shape), np.empty(k.shape), np.empty(v.shape)
        self.lib.kata_oracle_bwd_chunked_mg(self._p(q), self._p(k), self._p(v), self._p(dout),
                                            self._p(gq), self._p(gk), self._p(gv), B, H, T, d,
                                            dv, C, g, scan_mode)
        return gq, gk, gv

    # ---- linear features (identity, ReLU+eps, ELU+1, Lorentz lift) --------

    LIN_FEATURES = {"identity": 0, "relu": 1, "elu": 2, "lorentz": 3, "lorentz_s": 4}

    def lin_dim(self, d: int, feature: int) -> int:
        return int(self.lib.kata_oracle_lin_dim(d, feature))

    def lin_feature(self, x, feature: int, eps: float = 0.0):
        x = self._f64(x)
        d = x.shape[-1]
        out = np.empty(self.lin_dim(d, feature))
        self.lib.kata_oracle_lin_feature(self._p(x), d, feature, eps, self._p(out))
        return out

    def lin_fwd(self, q, k, v, feature: int, eps: float = 0.0, normalize: bool = True):
        q, k, v = self._f64(q), self._f64(k), self._f64(v)
        B, H, T, d = q.shape
        dv = v.shape[-1]
        out = np.empty((B, H, T, dv))
        self.lib.kata_oracle_lin_fwd(self._p(q), self._p(k), self._p(v), self._p(out),
                                     B, H, T, d, dv, feature, eps, int(normalize))
        return out

    def lin_fwd_rows(self, q, k, v, feature: int, eps: float, normalize: bool, bh_idx, t_idx):
        q, k, v = self._f64(q), self._f64(k), self._f64(v)
        B, H, T, d = q.shape
        dv = v.shape[-1]
        bh = np.ascontiguousarray(np.asarray(bh_idx, dtype=np.int64))
        tt = np.ascontiguousarray(np.asarray(t_idx, dtype=np.int64))
        assert bh.shape == tt.shape and bh.ndim == 1
        assert (bh >= 0).all() and (bh < B * H).all() and (tt >= 0).all() and (tt < T).all()
        out = np.empty((bh.size, dv))
        self.lib.kata_oracle_lin_fwd_rows(self._p(q), self._p(k), self._p(v), B, H, T, d, dv,
                                          feature, eps, int(normalize),
                                          bh.ctypes.data_as(_lp), tt.ctypes.data_as(_lp),
                                          bh.size, self._p(out))
        return out

    def lin_fwd_chunked(self, q, k, v, C: int, feature: int, eps: float = 0.0,
                        normalize: bool = True, scan_mode: int = 1):
        q, k, v = self._f64(q), self._f64(k), self._f64(v)
        B, H, T, d = q.shape
        dv = v.shape[-1]
        out = np.empty((B, H, T, dv))
        self.lib.kata_oracle_lin_fwd_chunked(self._p(q), self._p(k), self._p(v), self._p(out),
                                             B, H, T, d, dv, C, feature, eps, int(normalize),
                                             scan_mode)
        return out
