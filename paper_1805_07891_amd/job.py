"""One exchange job over torch-allocated device memory.

Plumbing only: torch allocates the worker gradient arenas and the stream,
this class turns them into the pointers the C interface takes, and copies
the job's state out for inspection.  All arithmetic of the step runs in the
HIP library.
"""

from __future__ import annotations

import ctypes
from typing import List, Optional, Sequence

import numpy as np

from . import phub as _phub
from .workloads import Job, key_offsets

HIP_MEMCPY_DEFAULT = 4

_hip = None


def hip_runtime():
    """The HIP runtime torch loaded (same SONAME as the library links)."""
    global _hip
    if _hip is None:
        import torch  # noqa: F401  (loads torch's libamdhip64.so.7 first)
        lib = ctypes.CDLL("libamdhip64.so.7")
        lib.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
        lib.hipMemcpy.restype = ctypes.c_int
        _hip = lib
    return _hip


def copy_to_host(dst: np.ndarray, src_ptr: int) -> None:
    """Synchronous copy of dst.nbytes from device address src_ptr."""
    rc = hip_runtime().hipMemcpy(dst.ctypes.data, src_ptr, dst.nbytes, HIP_MEMCPY_DEFAULT)
    if rc != 0:
        raise RuntimeError(f"hipMemcpy to host failed with code {rc}")


def load_library(path: Optional[str] = None) -> _phub.Library:
    import torch  # noqa: F401  (one HIP runtime for torch and the library)
    return _phub.load(path)


class TorchJob:
    """A phub job plus the torch buffers of its N workers.

    Gradients of worker w live in one arena tensor of ``arena_elems`` fp32
    values, key k at element offset ``offsets[k]`` (256-byte aligned); the
    job's own W and M arenas use the same layout.
    """

    def __init__(self, spec: Job, device, stream=None, chunk_bytes: Optional[int] = None,
                 lib: Optional[_phub.Library] = None, schedule: Optional[int] = None,
                 resident_bytes: Optional[int] = None,
                 key_group: Optional[Sequence[int]] = None, unfused: bool = False,
                 optimizer: Optional[str] = None, betas=(0.9, 0.999), eps: float = 1e-8,
                 workgroups: Optional[int] = None, ordered_events: bool = False,
                 whole_chunks: bool = False):
        import torch
        self.torch = torch
        self.spec = spec
        self.device = torch.device(device)
        self.lib = lib or load_library()
        self.stream = stream if stream is not None else torch.cuda.Stream(device=self.device)
        self.offsets, self.arena_elems = key_offsets(spec.key_elems)
        self.chunk_bytes = spec.chunk_bytes if chunk_bytes is None else int(chunk_bytes)
        with torch.cuda.device(self.device):
            self.handle = self.lib.phub_init(spec.num_workers, spec.key_elems, self.chunk_bytes,
                                             spec.lr, spec.momentum, spec.weight_decay,
                                             spec.nesterov, self.stream.cuda_stream,
                                             schedule=schedule, resident_bytes=resident_bytes,
                                             key_group=key_group, unfused=unfused,
                                             optimizer=None if optimizer is None
                                             else _phub.OPTIMIZERS[optimizer],
                                             beta1=betas[0], beta2=betas[1], eps=eps,
                                             workgroups=workgroups,
                                             ordered_events=int(bool(ordered_events)),
                                             whole_chunks=int(bool(whole_chunks)))
        self.optimizer = optimizer or "momentum"
        self.key_group = None if key_group is None else [int(g) for g in key_group]
        self._ptr_arrays: List = [None] * spec.num_workers
        self._grad_refs: List = [None] * spec.num_workers
        # every worker's key pointers in one table (worker-major) for phub_push_all
        self._all_ptrs = (ctypes.c_void_p * (spec.num_workers * spec.num_keys))()
        self._attached = 0
        # the two calls of every step, bound once and without ctypes argument
        # conversion (their arguments are prepared ctypes objects): a step of
        # a small job costs a few microseconds, and each layer of Python adds
        # to it (the conversion about 0.1-0.2 us per call)
        dll = self.lib.lib
        self._raw_push_all = dll._FuncPtr(("phub_push_all", dll))
        self._raw_push_all.restype = ctypes.c_int
        self._raw_step = dll._FuncPtr(("phub_step", dll))
        self._raw_step.restype = ctypes.c_int
        self._handle_arg = ctypes.c_void_p(self.handle)

    # -- inputs ----------------------------------------------------------------
    def key_pointers(self, arena) -> List[int]:
        base = arena.data_ptr()
        return [base + 4 * off for off in self.offsets]

    def attach_grads(self, worker: int, arena) -> None:
        """Use ``arena`` (a device fp32 tensor of arena_elems values) as
        worker ``worker``'s gradients from now on."""
        if arena.numel() != self.arena_elems or arena.dtype != self.torch.float32:
            raise ValueError("gradient arena has the wrong size or dtype")
        if self._grad_refs[worker] is None:
            self._attached += 1
        self._grad_refs[worker] = arena
        ptrs = self.key_pointers(arena)
        self._ptr_arrays[worker] = _phub.pointer_array(ptrs)
        k = self.spec.num_keys
        self._all_ptrs[worker * k:(worker + 1) * k] = ptrs

    def set_weights(self, arena) -> None:
        """Load every key's weights from a device arena (and zero M).  The
        job's stream first waits for work already queued on torch's current
        stream (which typically produced ``arena``)."""
        self.stream.wait_stream(self.torch.cuda.current_stream(self.device))
        self._weights_src = arena
        ptrs = self.key_pointers(arena)
        for k in range(self.spec.num_keys):
            self.lib.phub_set_weights(self.handle, k, ptrs[k])

    # -- the step --------------------------------------------------------------
    def push_all(self) -> None:
        """Every worker pushes every key from its attached arena (one call)."""
        if self._attached != self.spec.num_workers:
            missing = [w for w, a in enumerate(self._ptr_arrays) if a is None]
            raise RuntimeError(f"workers {missing} have no gradient arena attached")
        rc = self._raw_push_all(self._handle_arg, self._all_ptrs)
        if rc:
            self.lib._check(rc, True)

    def push_key(self, worker: int, key: int, event=None) -> None:
        """Push one key of worker ``worker`` from its attached arena; with
        ``event`` (a torch.cuda.Event recorded by the producer) the gradient
        counts as ready once the event completes."""
        ptr = self.key_pointers(self._grad_refs[worker])[key]
        if event is None:
            self.lib.phub_push(self.handle, worker, key, ptr)
        else:
            self.lib.phub_push_event(self.handle, worker, key, ptr, event.cuda_event)

    def bucket(self, worker: int, keys: Sequence[int]):
        """Prebuilt arguments for push_bucket: (key array, pointer array) of
        ``keys`` in worker ``worker``'s attached arena."""
        ptrs = self.key_pointers(self._grad_refs[worker])
        return ((ctypes.c_int * len(keys))(*[int(k) for k in keys]),
                _phub.pointer_array([ptrs[k] for k in keys]))

    def push_bucket(self, worker: int, bucket, event=None) -> None:
        """Push a prebuilt bucket (see ``bucket``) in one call, ready once
        ``event`` (a torch.cuda.Event) has completed."""
        keys, ptrs = bucket
        self.lib.phub_push_keys_event(self.handle, worker, ptrs, keys,
                                      None if event is None else event.cuda_event)

    def attach_models(self, worker: int, arena) -> None:
        """Use ``arena`` (arena_elems fp32 values) as worker ``worker``'s model
        buffer for pushpull: every key's updated weights land at its offset."""
        if arena.numel() != self.arena_elems or arena.dtype != self.torch.float32:
            raise ValueError("model arena has the wrong size or dtype")
        if not hasattr(self, "_model_refs"):
            self._model_refs = [None] * self.spec.num_workers
            self._model_ptrs = [None] * self.spec.num_workers
        self._model_refs[worker] = arena
        self._model_ptrs[worker] = _phub.pointer_array(self.key_pointers(arena))

    def pushpull_all(self) -> None:
        """Every worker pushes all its keys and asks for the updated weights
        in its attached model buffer."""
        for w, arr in enumerate(self._ptr_arrays):
            self.lib.phub_pushpull_keys(self.handle, w, arr, self._model_ptrs[w])

    def step(self) -> None:
        rc = self._raw_step(self._handle_arg)
        if rc:
            self.lib._check(rc, True)

    def push_and_step(self) -> None:
        self.push_all()
        self.step()

    def sync(self) -> None:
        self.lib.phub_sync(self.handle)

    # -- outputs ---------------------------------------------------------------
    def state_arenas(self):
        """(W, M) copied to host as numpy arenas of arena_elems values (M is
        None for plain SGD; for Adam it is the first moment)."""
        self.sync()
        w_ptr, m_ptr = self.lib.phub_get_state(self.handle, 0)
        W = np.empty(self.arena_elems, dtype=np.float32)
        copy_to_host(W, w_ptr)
        M = None
        if m_ptr:
            M = np.empty(self.arena_elems, dtype=np.float32)
            copy_to_host(M, m_ptr)
        return W, M

    def second_moment_arena(self):
        """Adam's second moment V as a host arena (None for other optimizers)."""
        self.sync()
        v_ptr = self.lib.phub_get_second_moment(self.handle, 0)
        if not v_ptr:
            return None
        V = np.empty(self.arena_elems, dtype=np.float32)
        copy_to_host(V, v_ptr)
        return V

    def key_state_pointers(self, key: int):
        """Device addresses of key ``key``'s state as the library hands them
        out: (phub_pull's W, phub_get_state's W and M, phub_get_second_moment's
        V); 0 where the optimizer keeps no such array."""
        w_pull = self.lib.phub_pull(self.handle, key)
        w_state, m = self.lib.phub_get_state(self.handle, key)
        v = self.lib.phub_get_second_moment(self.handle, key)
        return w_pull, w_state, m, v

    def pulled_keys(self):
        """Every key's state copied to the host through the per-key pointers
        of the Pull interface: a list of (W, M, V) per key, W read from
        phub_pull, M from phub_get_state, V from phub_get_second_moment (None
        where the optimizer keeps no such array).  Raises if phub_pull and
        phub_get_state disagree on a key's weights."""
        self.sync()
        out = []
        for k, n in enumerate(self.spec.key_elems):
            w_pull, w_state, m_ptr, v_ptr = self.key_state_pointers(k)
            if w_pull != w_state:
                raise RuntimeError(f"key {k}: phub_pull gives {w_pull:#x}, "
                                   f"phub_get_state {w_state:#x}")
            arrays = []
            for ptr in (w_pull, m_ptr, v_ptr):
                if not ptr:
                    arrays.append(None)
                    continue
                a = np.empty(n, dtype=np.float32)
                if n:
                    copy_to_host(a, ptr)
                arrays.append(a)
            out.append(tuple(arrays))
        return out

    def split(self, arena: np.ndarray) -> List[np.ndarray]:
        return [arena[o:o + n] for o, n in zip(self.offsets, self.spec.key_elems)]

    def info(self):
        """(workgroups, threads per workgroup, segments, state bytes,
        cache-resident state bytes) of the job's launch."""
        return self.lib.phub_job_info(self.handle)

    def cached_fraction(self) -> float:
        """Share of the optimizer state (unpadded) scheduled as cache-resident."""
        states = {"momentum": 2, "sgd": 1, "adam": 3}[self.optimizer]
        total = states * 4 * self.spec.num_params
        return self.info()[4] / total if total else 1.0

    def destroy(self) -> None:
        if self.handle is not None:
            self.lib.phub_destroy(self.handle)
            self.handle = None
            self._handle_arg = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass
