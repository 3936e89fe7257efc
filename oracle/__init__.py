"""Python access to the CPU oracle of the PHub exchange step.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the
benchmark's CPU-baseline leg use this module; the library path never does.
It loads the plain C oracle (``phub_oracle.c``, built by ``build()``) with
ctypes and marshals numpy arrays.  It imports nothing from the GPU library.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "phub_oracle.c")
LIB = os.path.join(HERE, "libphub_oracle.so")

CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared"]


def build(force: bool = True, src: str = SRC, out: str = LIB) -> str:
    """Compile the oracle with gcc into ``out`` (``libphub_oracle.so``)."""
    if force or not os.path.exists(out):
        tmp = out + ".tmp"
        subprocess.check_call(["gcc", *CFLAGS, "-o", tmp, src, "-lm"])
        os.replace(tmp, out)
    return out


class OracleLib:
    """The oracle's two entry points, loaded from one built library."""

    def __init__(self, path: str = LIB):
        lib = ctypes.CDLL(path)
        vp = ctypes.c_void_p
        lib.oracle_step_f32.argtypes = [ctypes.c_int, ctypes.c_int, vp, vp, vp, vp,
                                        ctypes.c_float, ctypes.c_float, ctypes.c_float, ctypes.c_int]
        lib.oracle_step_f32.restype = ctypes.c_int
        lib.oracle_step_f64.argtypes = [ctypes.c_int, ctypes.c_int, vp, vp, vp, vp,
                                        ctypes.c_double, ctypes.c_double, ctypes.c_double, ctypes.c_int]
        lib.oracle_step_f64.restype = ctypes.c_int
        f32 = ctypes.c_float
        lib.oracle_step_sgd_f32.argtypes = [ctypes.c_int, ctypes.c_int, vp, vp, vp, f32, f32]
        lib.oracle_step_sgd_f32.restype = ctypes.c_int
        lib.oracle_step_adam_f32.argtypes = [ctypes.c_int, ctypes.c_int, vp, vp, vp, vp, vp,
                                             f32, f32, f32, f32, f32, ctypes.c_int64]
        lib.oracle_step_adam_f32.restype = ctypes.c_int
        self.lib = lib
        self.path = path

    def step(self, grads, weights, moms, lr, momentum, weight_decay, nesterov, dtype=np.float32):
        """One exchange step, in place on ``weights`` and ``moms``.

        grads[w][k] is worker w's gradient for key k; weights[k] and moms[k]
        are key k's master weights and momentum.  All arrays must be
        contiguous 1-D arrays of ``dtype`` (float32 for the fp32 oracle,
        float64 for the double-precision one) with matching lengths per key.
        """
        num_workers = len(grads)
        num_keys = len(weights)
        if num_workers < 1 or num_keys < 1 or len(moms) != num_keys:
            raise ValueError("need at least one worker and one key, and one momentum array per key")
        elems = np.array([a.size for a in weights], dtype=np.int64)
        flat_g = []
        for w in range(num_workers):
            if len(grads[w]) != num_keys:
                raise ValueError("every worker must give one gradient per key")
            for k in range(num_keys):
                flat_g.append(grads[w][k])
        for a in list(flat_g) + list(weights) + list(moms):
            if a.dtype != dtype or not a.flags.c_contiguous or a.ndim != 1:
                raise ValueError(f"oracle arrays must be contiguous 1-D {np.dtype(dtype).name}")
        for k in range(num_keys):
            if moms[k].size != elems[k] or any(grads[w][k].size != elems[k] for w in range(num_workers)):
                raise ValueError(f"key {k}: length mismatch")
        gp, wp, mp = _ptrs(flat_g), _ptrs(weights), _ptrs(moms)
        if dtype == np.float32:
            rc = self.lib.oracle_step_f32(num_workers, num_keys, elems.ctypes.data, gp, wp, mp,
                                          float(np.float32(lr)), float(np.float32(momentum)),
                                          float(np.float32(weight_decay)), int(bool(nesterov)))
        elif dtype == np.float64:
            rc = self.lib.oracle_step_f64(num_workers, num_keys, elems.ctypes.data, gp, wp, mp,
                                          float(lr), float(momentum), float(weight_decay),
                                          int(bool(nesterov)))
        else:
            raise ValueError("dtype must be float32 or float64")
        if rc != 0:
            raise ValueError(f"oracle rejected its arguments (code {rc})")

    def _check_args(self, grads, weights, states):
        num_workers, num_keys = len(grads), len(weights)
        if num_workers < 1 or num_keys < 1:
            raise ValueError("need at least one worker and one key")
        elems = np.array([a.size for a in weights], dtype=np.int64)
        flat_g = []
        for w in range(num_workers):
            if len(grads[w]) != num_keys:
                raise ValueError("every worker must give one gradient per key")
            flat_g.extend(grads[w][k] for k in range(num_keys))
        for st in states:
            if len(st) != num_keys or any(st[k].size != elems[k] for k in range(num_keys)):
                raise ValueError("one state array per key, of the key's length")
        for a in flat_g + list(weights) + [x for st in states for x in st]:
            if a.dtype != np.float32 or not a.flags.c_contiguous or a.ndim != 1:
                raise ValueError("oracle arrays must be contiguous 1-D float32")
        for k in range(num_keys):
            if any(grads[w][k].size != elems[k] for w in range(num_workers)):
                raise ValueError(f"key {k}: length mismatch")
        return num_workers, num_keys, elems, flat_g

    def step_sgd(self, grads, weights, lr, weight_decay):
        """One step with plain SGD (no state), in place on ``weights`` (fp32)."""
        n, k, elems, flat_g = self._check_args(grads, weights, [])
        rc = self.lib.oracle_step_sgd_f32(n, k, elems.ctypes.data, _ptrs(flat_g), _ptrs(weights),
                                          float(np.float32(lr)), float(np.float32(weight_decay)))
        if rc != 0:
            raise ValueError(f"oracle rejected its arguments (code {rc})")

    def step_adam(self, grads, weights, m1, m2, lr, beta1, beta2, eps, weight_decay, step):
        """Step number ``step`` (from 1) of Adam, in place on ``weights`` and
        the two moment arrays ``m1``, ``m2`` (fp32)."""
        n, k, elems, flat_g = self._check_args(grads, weights, [m1, m2])
        rc = self.lib.oracle_step_adam_f32(n, k, elems.ctypes.data, _ptrs(flat_g), _ptrs(weights),
                                           _ptrs(m1), _ptrs(m2), float(np.float32(lr)),
                                           float(np.float32(beta1)), float(np.float32(beta2)),
                                           float(np.float32(eps)), float(np.float32(weight_decay)),
                                           int(step))
        if rc != 0:
            raise ValueError(f"oracle rejected its arguments (code {rc})")

    def step_flat(self, grads, weight, mom, lr, momentum, weight_decay, nesterov, dtype=np.float32):
        """One step over a single flat array (one key): grads[w] is worker w's."""
        self.step([[g] for g in grads], [weight], [mom], lr, momentum, weight_decay, nesterov, dtype)


def _ptrs(arrays):
    arr = (ctypes.c_void_p * len(arrays))()
    for i, a in enumerate(arrays):
        arr[i] = a.ctypes.data
    return arr


_default = None


def _load() -> OracleLib:
    global _default
    if _default is None:
        if not os.path.exists(LIB):
            build(force=False)
        _default = OracleLib(LIB)
    return _default


def step(grads: Sequence[Sequence[np.ndarray]], weights: Sequence[np.ndarray],
         moms: Sequence[np.ndarray], lr: float, momentum: float, weight_decay: float,
         nesterov: bool, dtype=np.float32) -> None:
    """One exchange step with the built oracle (see ``OracleLib.step``)."""
    _load().step(grads, weights, moms, lr, momentum, weight_decay, nesterov, dtype)


def step_flat(grads: Sequence[np.ndarray], weight: np.ndarray, mom: np.ndarray, lr: float,
              momentum: float, weight_decay: float, nesterov: bool, dtype=np.float32) -> None:
    """One step over a single flat array (one key): grads[w] is worker w's."""
    _load().step_flat(grads, weight, mom, lr, momentum, weight_decay, nesterov, dtype)


def step_sgd(grads, weights, lr, weight_decay) -> None:
    """Plain SGD step of the fp32 oracle; see ``OracleLib.step_sgd``."""
    _load().step_sgd(grads, weights, lr, weight_decay)


def step_adam(grads, weights, m1, m2, lr, beta1, beta2, eps, weight_decay, step) -> None:
    """Adam step of the fp32 oracle; see ``OracleLib.step_adam``."""
    _load().step_adam(grads, weights, m1, m2, lr, beta1, beta2, eps, weight_decay, step)
