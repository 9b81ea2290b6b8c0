"""Thin ctypes binding of libmure.so (``include/mure.h``).

Argument marshalling only: every step of the mutation-testing path runs in
the library's HIP kernels.  torch supplies device memory (inputs, kill bits,
logits) and the stream; the library never links torch.  If the library is not
built the import of this module succeeds but constructing ``Mure`` raises.
"""
from __future__ import annotations

import ctypes as C
import itertools
import operator
import os
from typing import Dict, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmure.so")

# mure.h enums
MURE_OK, MURE_E_INVALID, MURE_E_STATE, MURE_E_NOMEM, MURE_E_DEVICE, MURE_E_UNSUPPORTED = 0, -1, -2, -3, -4, -5
STATUS_NAMES = {0: "MURE_OK", -1: "MURE_E_INVALID", -2: "MURE_E_STATE", -3: "MURE_E_NOMEM",
                -4: "MURE_E_DEVICE", -5: "MURE_E_UNSUPPORTED"}
MURE_F32, MURE_BF16 = 0, 1
MURE_VERSION = 6
N_KERNELS = 9                                   # kernel families in mure_stats (MURE_N_KERNELS)
OP_GAUSS_FUZZ, OP_EFFECT_BLOCK, OP_ACT_INVERSE, OP_NEURON_SWITCH, OP_WEIGHT_SHUFFLE = 0, 1, 2, 3, 4
INPUT, DENSE, CONV2D, ADD, GAP, FLATTEN, DWCONV, EMBED, LSTM = 0, 1, 2, 3, 4, 5, 6, 7, 8

EXPORTED = ["mure_version", "mure_create", "mure_load_model", "mure_apply_mutants",
            "mure_run_original", "mure_run_mutants", "mure_run_mutants_noalloc",
            "mure_get_logits", "mure_mutant_plan",
            "mure_get_stats", "mure_set_option", "mure_last_error", "mure_destroy"]


class mure_layer(C.Structure):
    _fields_ = [("kind", C.c_int32), ("n_in", C.c_int32), ("in_", C.c_int32 * 2),
                ("c_in", C.c_int32), ("c_out", C.c_int32), ("kh", C.c_int32), ("kw", C.c_int32),
                ("stride", C.c_int32), ("pad", C.c_int32), ("relu", C.c_int32),
                ("maxpool", C.c_int32), ("shortcut", C.c_int32), ("seq", C.c_int32)]


class mure_record(C.Structure):
    _fields_ = [("mutant", C.c_int32), ("op", C.c_int32), ("layer", C.c_int32),
                ("neuron", C.c_int32), ("partner", C.c_int32), ("reserved", C.c_int32),
                ("noise", C.POINTER(C.c_float)), ("noise_len", C.c_int64),
                ("perm", C.POINTER(C.c_int32))]


class mure_score(C.Structure):
    _fields_ = [("ms_num", C.c_int64), ("ms_den", C.c_int64), ("ms", C.c_double),
                ("killed_mutants", C.c_int64), ("n_mutants", C.c_int64), ("n_labels", C.c_int64),
                ("n_inputs", C.c_int64), ("nonfinite_logits", C.c_int64)]


class mure_stats(C.Structure):
    _fields_ = [("n_groups", C.c_int64), ("n_identity_mutants", C.c_int64),
                ("macs_original", C.c_int64), ("macs_vanilla", C.c_int64),
                ("macs_memoized", C.c_int64), ("macs_algorithmic", C.c_int64),
                ("macs_executed", C.c_int64), ("cache_bytes", C.c_int64),
                ("workspace_bytes", C.c_int64), ("launches", C.c_int64),
                ("ms_apply", C.c_double), ("ms_run_original", C.c_double),
                ("ms_run_mutants", C.c_double), ("gemm_launches", C.c_int64),
                ("ms_gemm", C.c_double), ("gemm_macs_algorithmic", C.c_int64),
                ("gemm_macs_executed", C.c_int64), ("kernel_launches", C.c_int64 * N_KERNELS),
                ("kernel_ms", C.c_double * N_KERNELS), ("kernel_macs_algorithmic", C.c_int64 * N_KERNELS),
                ("kernel_bytes_algorithmic", C.c_double * N_KERNELS),
                ("n_classes", C.c_int64), ("n_inputs", C.c_int64), ("n_mutants", C.c_int64),
                ("group_planes", C.c_int64), ("ms_mmi", C.c_double)]


def _pack(arrays, R: int, dtype):
    """Addresses and lengths of the non-None entries of ``arrays`` (length R,
    or None) for the records' pointer fields; returns (the arrays to keep
    alive while the call runs, address of each record's entry or 0, length of
    each record's entry or 0).  Entries already of ``dtype`` and contiguous
    are passed in place, without a copy: GF noise is fan-in long for every
    record (hundreds of MB on the large models).  The per-record iteration
    runs in C (map, itemgetter) rather than in Python loops."""
    addr = np.zeros(R, np.uint64)
    lens = np.zeros(R, np.int64)
    if arrays is None or len(arrays) == 0:
        return [], addr, lens
    idx = np.flatnonzero(np.fromiter(map(operator.is_not, arrays, itertools.repeat(None)), bool, R))
    if idx.size == 0:
        return [], addr, lens
    parts = operator.itemgetter(*idx.tolist())(arrays) if idx.size > 1 else (arrays[int(idx[0])],)
    dt = np.dtype(dtype)
    parts = [p if isinstance(p, np.ndarray) and p.dtype == dt and p.ndim == 1 and p.flags.c_contiguous
             else np.ascontiguousarray(p, dt).reshape(-1) for p in parts]
    ln = np.fromiter(map(len, parts), np.int64, idx.size)
    ad = np.fromiter((p.__array_interface__["data"][0] for p in parts), np.uint64, idx.size)
    addr[idx] = np.where(ln > 0, ad, 0).astype(np.uint64)
    lens[idx] = ln
    return parts, addr, lens


class MureError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status
        self.message = message


_lib = None


def load_library(path: str = LIB_PATH) -> C.CDLL:
    """Load libmure.so; raises if it has not been built (no fallback path)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it first (python -m paper_2607_18582_amd.build)")
    # One HIP runtime per process: torch ships its own libamdhip64, and the
    # streams and device memory it hands to the library belong to that
    # runtime.  Loading torch first makes libmure bind to the same runtime.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = C.CDLL(path)
    P = C.c_void_p
    sig = {
        "mure_version": (C.c_int32, []),
        "mure_create": (C.c_int, [C.POINTER(P), C.c_int32, P]),
        "mure_load_model": (C.c_int, [P, C.POINTER(mure_layer), C.c_int32, C.POINTER(C.c_int32),
                                      C.c_int32, C.POINTER(P), C.POINTER(P)]),
        "mure_apply_mutants": (C.c_int, [P, C.c_int32, C.POINTER(mure_record), C.c_int64]),
        "mure_run_original": (C.c_int, [P, P, C.c_int64, C.POINTER(C.c_int32)]),
        "mure_run_mutants": (C.c_int, [P, P, C.POINTER(C.c_int64), C.POINTER(mure_score)]),
        "mure_run_mutants_noalloc": (C.c_int, [P, P, C.POINTER(C.c_int64), C.POINTER(mure_score)]),
        "mure_get_logits": (C.c_int, [P, C.c_int32, P]),
        "mure_mutant_plan": (C.c_int, [P, C.c_int32, C.POINTER(C.c_int32), C.POINTER(C.c_int32),
                                       C.POINTER(C.c_int32), C.c_int32, C.POINTER(C.c_int32)]),
        "mure_get_stats": (C.c_int, [P, C.POINTER(mure_stats)]),
        "mure_set_option": (C.c_int, [P, C.c_char_p, C.c_int64]),
        "mure_last_error": (C.c_char_p, [P]),
        "mure_destroy": (None, [P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def layer_descriptors(nodes) -> "C.Array":
    """mure_layer array from node objects with the fields of ``mure_layer``
    (kind, inputs, c_in, c_out, kh, kw, stride, pad, relu, maxpool, shortcut)."""
    arr = (mure_layer * len(nodes))()
    for i, n in enumerate(nodes):
        L = arr[i]
        L.kind = int(n.kind)
        ins = list(n.inputs)
        L.n_in = len(ins)
        L.in_[0] = ins[0] if len(ins) > 0 else 0
        L.in_[1] = ins[1] if len(ins) > 1 else 0
        if n.kind in (CONV2D, DENSE, DWCONV):
            L.c_in, L.c_out = int(n.c_in), int(n.c_out)
            L.kh, L.kw, L.stride, L.pad = int(n.kh), int(n.kw), int(n.stride), int(n.pad)
            L.maxpool = int(n.maxpool)
        elif n.kind in (EMBED, LSTM):
            L.c_in, L.c_out = int(n.c_in), int(n.c_out)
            L.seq = int(getattr(n, "seq", 0)) if n.kind == LSTM else 0
        elif n.kind in (ADD, GAP, FLATTEN):
            L.c_in, L.c_out = int(n.c_in), int(n.c_out)
        L.relu = int(n.relu)
        L.shortcut = int(n.shortcut) if n.kind == ADD else 0
    return arr


class Mure:
    """One library context on a GPU (``device`` >= 0) or a planning-only
    context (``device`` = -1)."""

    def __init__(self, device: int = 0, stream=None):
        self.lib = load_library()
        self.device = device
        if device >= 0 and stream is None:
            import torch
            stream = torch.cuda.current_stream(device).cuda_stream
        self.ctx = C.c_void_p()
        st = self.lib.mure_create(C.byref(self.ctx), device, C.c_void_p(stream or 0))
        if st != MURE_OK:
            raise MureError(st, self.lib.mure_last_error(None).decode())
        self._keep = []
        self.n_mutants = 0
        self.n_inputs = 0
        self.classes = 0

    def close(self):
        if getattr(self, "ctx", None):
            self.lib.mure_destroy(self.ctx)
            self.ctx = None

    __del__ = close

    def _check(self, st: int):
        if st != MURE_OK:
            raise MureError(st, self.lib.mure_last_error(self.ctx).decode())

    # -- calls --------------------------------------------------------------
    def load_model(self, nodes, in_hwc, dtype: str, weights: Sequence, biases: Sequence):
        arr = layer_descriptors(nodes)
        hwc = (C.c_int32 * 3)(*[int(v) for v in in_hwc])
        n = len(nodes)
        wp = (C.c_void_p * n)()
        bp = (C.c_void_p * n)()
        keep = []
        for i in range(n):
            if weights[i] is not None:
                w = np.ascontiguousarray(weights[i])
                b = np.ascontiguousarray(biases[i], dtype=np.float32)
                keep += [w, b]
                wp[i] = w.ctypes.data
                bp[i] = b.ctypes.data
        dt = MURE_F32 if dtype == "f32" else MURE_BF16
        self._check(self.lib.mure_load_model(self.ctx, arr, n, hwc, dt, wp, bp))
        self.classes = self._shapes()[0]

    RECORD_DTYPE = np.dtype([("mutant", "<i4"), ("op", "<i4"), ("layer", "<i4"), ("neuron", "<i4"),
                             ("partner", "<i4"), ("reserved", "<i4"), ("noise", "<u8"),
                             ("noise_len", "<i8"), ("perm", "<u8")])

    def apply_mutants(self, n_mutants: int, mutant_id, op, layer, neuron, partner, noise, perm=None):
        R = len(mutant_id)
        recs = np.zeros(max(R, 1), dtype=self.RECORD_DTYPE)
        recs["mutant"][:R] = mutant_id
        recs["op"][:R] = op
        recs["layer"][:R] = layer
        recs["neuron"][:R] = neuron
        recs["partner"][:R] = partner
        # per-record arrays (GF noise, WS permutation) are referenced by
        # address and length, in place where their type allows
        pool, ppool = _pack(noise, R, np.float32), _pack(perm, R, np.int32)
        recs["noise"][:R], recs["noise_len"][:R] = pool[1], pool[2]
        wsr = ppool[2] > 0
        recs["perm"][:R] = ppool[1]
        recs["noise_len"][:R][wsr] = ppool[2][wsr]
        pool, ppool = pool[0], ppool[0]
        assert self.RECORD_DTYPE.itemsize == C.sizeof(mure_record)
        ptr = recs.ctypes.data_as(C.POINTER(mure_record))
        self._keep_params = (pool, ppool)
        self._check(self.lib.mure_apply_mutants(self.ctx, int(n_mutants), ptr, R))
        self.n_mutants = int(n_mutants)

    def apply(self, mutants):
        """``apply_mutants`` from an object with mutant_id/op/layer/neuron/partner/noise."""
        self.apply_mutants(mutants.n_mutants, mutants.mutant_id, mutants.op, mutants.layer,
                           mutants.neuron, mutants.partner, mutants.noise,
                           getattr(mutants, "perm", None))

    def run_original(self, inputs, labels: Optional[np.ndarray] = None):
        """``inputs``: a contiguous CUDA tensor [N][H][W][C] (float32, or int16/bfloat16
        holding bfloat16 bits)."""
        assert inputs.is_cuda and inputs.is_contiguous()
        n = int(inputs.shape[0])
        lp = None
        if labels is not None:
            lab = np.ascontiguousarray(labels, dtype=np.int32)
            self._keep_labels = lab
            lp = lab.ctypes.data_as(C.POINTER(C.c_int32))
        self._check(self.lib.mure_run_original(self.ctx, C.c_void_p(inputs.data_ptr()), n, lp))
        self.n_inputs = n

    def _shapes(self):
        """(classes, inputs, mutants) as the library holds them."""
        st = mure_stats()
        self._check(self.lib.mure_get_stats(self.ctx, C.byref(st)))
        return int(st.n_classes), int(st.n_inputs), int(st.n_mutants)

    @staticmethod
    def _check_device_buffer(t, nbytes: int, what: str):
        if not (t.is_cuda and t.is_contiguous()):
            raise ValueError(f"{what} must be a contiguous CUDA tensor")
        if t.numel() * t.element_size() < nbytes:
            raise ValueError(f"{what} holds {t.numel() * t.element_size()} bytes; the library writes {nbytes}")

    def run_mutants(self, kill_bits=None, noalloc: bool = False):
        """Returns (kill_bits [M][ceil(N/64)] int64 CUDA tensor holding the uint64
        words, kills per mutant (numpy int64), score dict).  noalloc: call
        mure_run_mutants_noalloc (the library allocates no device memory)."""
        import torch
        _, n, mutants = self._shapes()
        nw = (n + 63) // 64
        if kill_bits is None:
            kill_bits = torch.empty((max(mutants, 1), nw), dtype=torch.int64,
                                    device=f"cuda:{self.device}")
        self._check_device_buffer(kill_bits, mutants * nw * 8, "kill_bits")
        kills = np.zeros(max(mutants, 1), np.int64)
        sc = mure_score()
        fn = self.lib.mure_run_mutants_noalloc if noalloc else self.lib.mure_run_mutants
        self._check(fn(self.ctx, C.c_void_p(kill_bits.data_ptr()),
                       kills.ctypes.data_as(C.POINTER(C.c_int64)), C.byref(sc)))
        score = {k: getattr(sc, k) for k, _ in mure_score._fields_}
        return kill_bits[:mutants], kills[:mutants], score

    def get_logits(self, mutant_id: int, out=None):
        """float32 logits [N][classes] of one mutant (-1: the original)."""
        import torch
        classes, n, _ = self._shapes()
        if out is None:
            out = torch.empty((n, classes), dtype=torch.float32, device=f"cuda:{self.device}")
        self._check_device_buffer(out, n * classes * 4, "out")
        self._check(self.lib.mure_get_logits(self.ctx, int(mutant_id), C.c_void_p(out.data_ptr())))
        return out

    def mutant_plan(self, mutant_id: int):
        mmi, grp, nk = C.c_int32(), C.c_int32(), C.c_int32()
        ks = (C.c_int32 * 64)()
        self._check(self.lib.mure_mutant_plan(self.ctx, int(mutant_id), C.byref(mmi), C.byref(grp),
                                              ks, 64, C.byref(nk)))
        return mmi.value, grp.value, [ks[i] for i in range(min(nk.value, 64))]

    def stats(self) -> Dict[str, float]:
        s = mure_stats()
        self._check(self.lib.mure_get_stats(self.ctx, C.byref(s)))
        out = {}
        for k, _ in mure_stats._fields_:
            v = getattr(s, k)
            out[k] = list(v) if isinstance(v, C.Array) else v
        return out

    def set_option(self, name: str, value: int):
        self._check(self.lib.mure_set_option(self.ctx, name.encode(), int(value)))
