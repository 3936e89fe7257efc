"""Python binding of the C interface in ``include/phub.h`` (ctypes).

Argument marshalling only: every step of the exchange runs in the HIP
library ``libphub.so``.  The functions keep the C names; each returns the C
status code, raising ``PhubError`` for a nonzero one unless ``check=False``.
Pointers are plain integers (torch's ``tensor.data_ptr()``, a stream's
``cuda_stream``).  If the library is not built, loading raises ImportError:
there is no fallback.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

PKG = os.path.dirname(os.path.abspath(__file__))
DEFAULT_LIB = os.path.join(PKG, "libphub.so")

PHUB_OK = 0
PHUB_EINVAL = -1
PHUB_ENOTREADY = -2
PHUB_ENOMEM = -3
PHUB_EHIP = -4
PHUB_ESTATE = -5

STATUS_NAMES = {0: "PHUB_OK", -1: "PHUB_EINVAL", -2: "PHUB_ENOTREADY", -3: "PHUB_ENOMEM",
                -4: "PHUB_EHIP", -5: "PHUB_ESTATE"}

PHUB_SCHEDULE_SPLIT = 0
PHUB_SCHEDULE_LPT = 1
PHUB_SCHEDULE_DYNAMIC = 2

PHUB_OPT_MOMENTUM = 0
PHUB_OPT_SGD = 1
PHUB_OPT_ADAM = 2
OPTIMIZERS = {"momentum": PHUB_OPT_MOMENTUM, "sgd": PHUB_OPT_SGD, "adam": PHUB_OPT_ADAM}

# Every symbol the header declares.
EXPORTED = ("phub_init", "phub_init_ex", "phub_set_weights", "phub_push", "phub_push_event",
            "phub_push_keys", "phub_push_keys_event", "phub_push_all", "phub_pushpull",
            "phub_pushpull_keys",
            "phub_step", "phub_pull", "phub_get_state", "phub_get_second_moment", "phub_sync",
            "phub_get_stream",
            "phub_job_info", "phub_destroy", "phub_last_error", "phub_plan_count",
            "phub_plan_build", "phub_step_noalloc")


class PhubError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(code, code)}: {message}")
        self.code = code


class PhubSegment(ctypes.Structure):
    _fields_ = [("key", ctypes.c_int32), ("count", ctypes.c_int32), ("offset", ctypes.c_int64)]


class PhubOptions(ctypes.Structure):
    _fields_ = [("schedule", ctypes.c_int), ("resident_bytes", ctypes.c_int64),
                ("num_groups", ctypes.c_int), ("key_group", ctypes.POINTER(ctypes.c_int)),
                ("optimizer", ctypes.c_int), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("workgroups", ctypes.c_int), ("unfused", ctypes.c_int),
                ("ordered_events", ctypes.c_int), ("whole_chunks", ctypes.c_int)]


class Library:
    """The C functions of one built ``libphub.so``."""

    def __init__(self, path: str = DEFAULT_LIB):
        if not os.path.exists(path):
            raise ImportError(f"HIP library {path} is not built; run __graft_entry__.build()")
        self.path = path
        lib = ctypes.CDLL(path)
        vp, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_float
        pp = ctypes.POINTER(ctypes.c_void_p)
        sig = {
            "phub_init": ([pp, i32, i32, vp, i64, f32, f32, f32, i32, vp], i32),
            "phub_init_ex": ([pp, i32, i32, vp, i64, f32, f32, f32, i32, vp,
                              ctypes.POINTER(PhubOptions)], i32),
            "phub_set_weights": ([vp, i32, vp], i32),
            "phub_push": ([vp, i32, i32, vp], i32),
            "phub_push_event": ([vp, i32, i32, vp, vp], i32),
            "phub_push_keys": ([vp, i32, i32, vp, vp], i32),
            "phub_push_all": ([vp, vp], i32),
            "phub_push_keys_event": ([vp, i32, i32, vp, vp, vp], i32),
            "phub_pushpull": ([vp, i32, i32, vp, vp], i32),
            "phub_pushpull_keys": ([vp, i32, i32, vp, vp, vp, vp], i32),
            "phub_step": ([vp], i32),
            "phub_pull": ([vp, i32, pp], i32),
            "phub_get_state": ([vp, i32, pp, pp], i32),
            "phub_get_second_moment": ([vp, i32, pp], i32),
            "phub_sync": ([vp], i32),
            "phub_get_stream": ([vp, pp], i32),
            "phub_job_info": ([vp, ctypes.POINTER(i32), ctypes.POINTER(i32), ctypes.POINTER(i64),
                               ctypes.POINTER(i64), ctypes.POINTER(i64)], i32),
            "phub_destroy": ([vp], i32),
            "phub_last_error": ([], ctypes.c_char_p),
            "phub_plan_count": ([i32, i32, vp, i64, i32, i32, i32, ctypes.POINTER(i64),
                                 ctypes.POINTER(i32), ctypes.POINTER(i64)], i32),
            "phub_plan_build": ([i32, i32, vp, i64, i32, i32, i32, vp, vp, vp], i32),
            "phub_step_noalloc": ([i32, i32, vp, i64, f32, f32, f32, i32, vp, vp, vp, vp], i32),
        }
        for name, (args, res) in sig.items():
            fn = getattr(lib, name)
            fn.argtypes = args
            fn.restype = res
        self.lib = lib

    def _check(self, rc: int, check: bool) -> int:
        if rc != 0 and check:
            raise PhubError(rc, self.last_error())
        return rc

    def last_error(self) -> str:
        return self.lib.phub_last_error().decode()

    # -- job lifecycle -----------------------------------------------------
    def phub_init(self, num_workers: int, key_elems: Sequence[int], chunk_bytes: int,
                  lr: float, momentum: float, weight_decay: float, nesterov: bool,
                  hip_stream: Optional[int] = None, check: bool = True,
                  schedule: Optional[int] = None, resident_bytes: Optional[int] = None,
                  key_group: Optional[Sequence[int]] = None, num_groups: Optional[int] = None,
                  unfused: bool = False, optimizer: Optional[int] = None, beta1: float = 0.9,
                  beta2: float = 0.999, eps: float = 1e-8, workgroups: Optional[int] = None,
                  ordered_events: int = 0, whole_chunks: int = 0):
        """Returns the job handle (an int), or (rc, None) with check=False on
        error.  With ``schedule``, ``resident_bytes`` or readiness groups
        (``key_group``: the group of each key; ``num_groups`` defaults to
        max + 1) given, calls phub_init_ex with those options."""
        elems = (ctypes.c_int64 * len(key_elems))(*[int(n) for n in key_elems])
        out = ctypes.c_void_p()
        args = (ctypes.byref(out), int(num_workers), len(key_elems),
                ctypes.cast(elems, ctypes.c_void_p), int(chunk_bytes), float(lr), float(momentum),
                float(weight_decay), int(bool(nesterov)), hip_stream)
        if (schedule is None and resident_bytes is None and key_group is None and num_groups is None
                and not unfused and optimizer is None and workgroups is None
                and not ordered_events and not whole_chunks):
            rc = self.lib.phub_init(*args)
        else:
            groups = None
            if key_group is not None:
                groups = (ctypes.c_int * max(len(key_group), 1))(*[int(g) for g in key_group])
                if num_groups is None:
                    num_groups = max((int(g) for g in key_group), default=-1) + 1
            opts = PhubOptions(PHUB_SCHEDULE_LPT if schedule is None else int(schedule),
                               -1 if resident_bytes is None else int(resident_bytes),
                               0 if num_groups is None else int(num_groups),
                               ctypes.cast(groups, ctypes.POINTER(ctypes.c_int)) if groups else None,
                               PHUB_OPT_MOMENTUM if optimizer is None else int(optimizer),
                               float(beta1), float(beta2), float(eps),
                               0 if workgroups is None else int(workgroups), int(bool(unfused)),
                               int(ordered_events), int(whole_chunks))
            rc = self.lib.phub_init_ex(*args, ctypes.byref(opts))
        if rc != 0:
            self._check(rc, check)
            return rc, None
        return out.value

    def phub_set_weights(self, job, key: int, src_ptr: int, check: bool = True) -> int:
        return self._check(self.lib.phub_set_weights(job, int(key), src_ptr), check)

    def phub_push(self, job, worker: int, key: int, grad_ptr: int, check: bool = True) -> int:
        return self._check(self.lib.phub_push(job, int(worker), int(key), grad_ptr), check)

    def phub_push_event(self, job, worker: int, key: int, grad_ptr: int, hip_event: Optional[int],
                        check: bool = True) -> int:
        """hip_event: a hipEvent_t handle as an int (torch.cuda.Event.cuda_event) or None."""
        return self._check(self.lib.phub_push_event(job, int(worker), int(key), grad_ptr, hip_event),
                           check)

    def phub_push_all(self, job, grad_ptrs, check: bool = True) -> int:
        """grad_ptrs: num_workers * num_keys device pointers, worker-major (a
        ctypes c_void_p array, see ``pointer_array``, or a sequence of ints;
        None is passed on as NULL)."""
        if grad_ptrs is not None and not isinstance(grad_ptrs, ctypes.Array):
            grad_ptrs = pointer_array(grad_ptrs)
        return self._check(self.lib.phub_push_all(job, grad_ptrs), check)

    def phub_push_keys(self, job, worker: int, grad_ptrs, keys=None, check: bool = True) -> int:
        """grad_ptrs: a ctypes c_void_p array (see ``pointer_array``) or a
        sequence of ints; keys: None (0..count-1) or a sequence of ints."""
        if not isinstance(grad_ptrs, ctypes.Array):
            grad_ptrs = pointer_array(grad_ptrs)
        karr = None
        if keys is not None:
            karr = (ctypes.c_int * len(keys))(*[int(k) for k in keys])
        return self._check(self.lib.phub_push_keys(job, int(worker), len(grad_ptrs),
                                                   karr, grad_ptrs), check)

    def phub_pushpull(self, job, worker: int, key: int, grad_ptr: int, out_ptr: int,
                      check: bool = True) -> int:
        return self._check(self.lib.phub_pushpull(job, int(worker), int(key), grad_ptr, out_ptr),
                           check)

    def phub_pushpull_keys(self, job, worker: int, grad_ptrs, out_ptrs, keys=None,
                           hip_event: Optional[int] = None, check: bool = True) -> int:
        if not isinstance(grad_ptrs, ctypes.Array):
            grad_ptrs = pointer_array(grad_ptrs)
        if not isinstance(out_ptrs, ctypes.Array):
            out_ptrs = pointer_array(out_ptrs)
        karr = keys
        if keys is not None and not isinstance(keys, ctypes.Array):
            karr = (ctypes.c_int * len(keys))(*[int(k) for k in keys])
        return self._check(self.lib.phub_pushpull_keys(job, int(worker), len(grad_ptrs), karr,
                                                       grad_ptrs, out_ptrs, hip_event), check)

    def phub_push_keys_event(self, job, worker: int, grad_ptrs, keys, hip_event: Optional[int],
                             check: bool = True) -> int:
        """As phub_push_keys, all ready once ``hip_event`` (a hipEvent_t as an
        int, or None) has completed.  ``keys`` may be a prebuilt ctypes int
        array."""
        if not isinstance(grad_ptrs, ctypes.Array):
            grad_ptrs = pointer_array(grad_ptrs)
        karr = keys
        if keys is not None and not isinstance(keys, ctypes.Array):
            karr = (ctypes.c_int * len(keys))(*[int(k) for k in keys])
        return self._check(self.lib.phub_push_keys_event(job, int(worker), len(grad_ptrs), karr,
                                                         grad_ptrs, hip_event), check)

    def phub_step(self, job, check: bool = True) -> int:
        return self._check(self.lib.phub_step(job), check)

    def phub_pull(self, job, key: int) -> int:
        out = ctypes.c_void_p()
        self._check(self.lib.phub_pull(job, int(key), ctypes.byref(out)), True)
        return out.value or 0

    def phub_get_state(self, job, key: int):
        w, m = ctypes.c_void_p(), ctypes.c_void_p()
        self._check(self.lib.phub_get_state(job, int(key), ctypes.byref(w), ctypes.byref(m)), True)
        return (w.value or 0), (m.value or 0)

    def phub_get_second_moment(self, job, key: int) -> int:
        v = ctypes.c_void_p()
        self._check(self.lib.phub_get_second_moment(job, int(key), ctypes.byref(v)), True)
        return v.value or 0

    def phub_sync(self, job, check: bool = True) -> int:
        return self._check(self.lib.phub_sync(job), check)

    def phub_get_stream(self, job) -> int:
        out = ctypes.c_void_p()
        self._check(self.lib.phub_get_stream(job, ctypes.byref(out)), True)
        return out.value or 0

    def phub_job_info(self, job):
        """(workgroups, threads per workgroup, segments, state bytes,
        cache-resident state bytes)."""
        g, t, s, sb, r = (ctypes.c_int(), ctypes.c_int(), ctypes.c_int64(), ctypes.c_int64(),
                          ctypes.c_int64())
        self._check(self.lib.phub_job_info(job, ctypes.byref(g), ctypes.byref(t), ctypes.byref(s),
                                           ctypes.byref(sb), ctypes.byref(r)), True)
        return g.value, t.value, s.value, sb.value, r.value

    def phub_destroy(self, job, check: bool = True) -> int:
        return self._check(self.lib.phub_destroy(job), check)

    def phub_step_noalloc(self, num_workers: int, key_elems: Sequence[int], chunk_bytes: int,
                          lr: float, momentum: float, weight_decay: float, nesterov: bool,
                          grad_ptrs: Sequence[int], weights_ptr: int, moments_ptr: int,
                          stream: Optional[int] = None, check: bool = True) -> int:
        """One step without allocation over caller arenas (see phub.h);
        grad_ptrs[w * K + k] is worker w's gradient for key k."""
        elems = (ctypes.c_int64 * len(key_elems))(*[int(n) for n in key_elems])
        return self._check(self.lib.phub_step_noalloc(
            int(num_workers), len(key_elems), elems, int(chunk_bytes), float(lr), float(momentum),
            float(weight_decay), int(bool(nesterov)), pointer_array(grad_ptrs), weights_ptr,
            moments_ptr, stream), check)

    # -- schedule (host only) ----------------------------------------------
    def phub_plan_count(self, num_workers: int, key_elems: Sequence[int], chunk_bytes: int,
                        num_bins: int, min_items: int = 0, schedule: int = PHUB_SCHEDULE_SPLIT):
        elems = (ctypes.c_int64 * len(key_elems))(*[int(n) for n in key_elems])
        nseg, used, item = ctypes.c_int64(), ctypes.c_int(), ctypes.c_int64()
        self._check(self.lib.phub_plan_count(int(num_workers), len(key_elems),
                                             ctypes.cast(elems, ctypes.c_void_p), int(chunk_bytes),
                                             int(schedule), int(num_bins), int(min_items),
                                             ctypes.byref(nseg), ctypes.byref(used),
                                             ctypes.byref(item)), True)
        return nseg.value, used.value, item.value

    def phub_plan_build(self, num_workers: int, key_elems: Sequence[int], chunk_bytes: int,
                        num_bins: int, min_items: int = 0, schedule: int = PHUB_SCHEDULE_SPLIT):
        """Returns (segments as a list of (key, count, offset), bin_begin,
        bin_cost, item_elems)."""
        nseg, used, item = self.phub_plan_count(num_workers, key_elems, chunk_bytes, num_bins,
                                                min_items, schedule)
        elems = (ctypes.c_int64 * len(key_elems))(*[int(n) for n in key_elems])
        segs = (PhubSegment * max(nseg, 1))()
        bb = (ctypes.c_int64 * (used + 1))()
        bc = (ctypes.c_int64 * max(used, 1))()
        self._check(self.lib.phub_plan_build(int(num_workers), len(key_elems),
                                             ctypes.cast(elems, ctypes.c_void_p), int(chunk_bytes),
                                             int(schedule), int(num_bins), int(min_items), segs,
                                             bb, bc), True)
        seg_list = [(segs[i].key, segs[i].count, segs[i].offset) for i in range(nseg)]
        return seg_list, list(bb), list(bc[:used]), item


def pointer_array(ptrs: Sequence[int]):
    arr = (ctypes.c_void_p * len(ptrs))()
    for i, p in enumerate(ptrs):
        arr[i] = int(p)
    return arr


_default: Optional[Library] = None


def load(path: Optional[str] = None) -> Library:
    """The library at ``path`` (default: the in-tree build)."""
    global _default
    if path is not None and path != DEFAULT_LIB:
        return Library(path)
    if _default is None:
        _default = Library(DEFAULT_LIB)
    return _default
