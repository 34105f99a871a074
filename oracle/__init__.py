"""Test infrastructure: the CPU oracle of the backoff n-gram query.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` import this package; the library under test never does.  The
arithmetic lives in ``oracle.c`` (plain C, built with gcc into
``liboracle.so``); ``bruteforce.py`` is a second, pure-Python statement of the
definition on histories, for tiny models.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

MODE_PLAIN, MODE_CTC, MODE_TRANSDUCER, MODE_AED = 0, 1, 2, 3

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
SRC_PATH = os.path.join(_HERE, "oracle.c")
CFLAGS = ["-O2", "-ffp-contract=off", "-fPIC", "-shared", "-pthread", "-Wall", "-Wextra"]


def build(src: str = SRC_PATH, out: str = LIB_PATH, extra=()) -> str:
    """Compile the oracle with gcc (no GPU code involved)."""
    cmd = ["gcc", *CFLAGS, *extra, "-o", out + ".tmp", src, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


_lib_cache = {}


def load(path: str = LIB_PATH):
    if path in _lib_cache:
        return _lib_cache[path]
    if not os.path.exists(path):
        if path != LIB_PATH:
            raise FileNotFoundError(path)
        build()
    lib = ctypes.CDLL(path)
    i32p = ctypes.POINTER(ctypes.c_int32)
    vp = ctypes.c_void_p
    lib.oracle_create.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int64, vp, vp, vp, vp,
                                  ctypes.c_float, ctypes.c_int, ctypes.POINTER(vp)]
    lib.oracle_final.argtypes = [vp, vp, ctypes.c_int64, vp]
    lib.oracle_final.restype = ctypes.c_int
    lib.oracle_start_state.argtypes = [vp]
    lib.oracle_start_state.restype = ctypes.c_int64
    lib.oracle_create.restype = ctypes.c_int
    lib.oracle_free.argtypes = [vp]
    lib.oracle_num_states.argtypes = [vp]
    lib.oracle_num_states.restype = ctypes.c_int64
    lib.oracle_state_context.argtypes = [vp, ctypes.c_int64, i32p]
    lib.oracle_state_context.restype = ctypes.c_int
    lib.oracle_state_of.argtypes = [vp, i32p, ctypes.c_int]
    lib.oracle_state_of.restype = ctypes.c_int64
    lib.oracle_advance.argtypes = [vp, vp, ctypes.c_int64, vp, vp, vp, ctypes.c_int]
    lib.oracle_advance.restype = ctypes.c_int
    lib.oracle_greedy_step.argtypes = [vp, vp, ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                                       ctypes.c_float, vp, vp, vp]
    lib.oracle_greedy_step.restype = ctypes.c_int
    lib.oracle_decode.argtypes = [vp, vp, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                  ctypes.c_int, ctypes.c_float, vp, vp, vp, vp, vp, ctypes.c_int]
    lib.oracle_decode.restype = ctypes.c_int
    lib.oracle_fused_topk.argtypes = [vp, vp, ctypes.c_int64, ctypes.c_int64, ctypes.c_float, ctypes.c_int,
                                      vp, vp, vp, vp]
    lib.oracle_fused_topk.restype = ctypes.c_int
    lib.oracle_last_error.restype = ctypes.c_char_p
    lib.oracle_repair.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int64, vp, vp, vp, vp, ctypes.c_float,
                                  ctypes.c_int, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(vp),
                                  ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp)]
    lib.oracle_repair.restype = ctypes.c_int
    lib.oracle_free_buffer.argtypes = [vp]
    _lib_cache[path] = lib
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


class OracleError(RuntimeError):
    def __init__(self, code, msg=""):
        super().__init__(f"oracle error {code}: {msg}")
        self.code = code


def repair_list(vocab_size, max_order, order, tokens, logprob, backoff, unk_logprob=float("nan"),
                bos_eos: bool = False, lib_path: str = LIB_PATH):
    """The closed list of a list that is not closed: the listed rows, then every
    missing prefix and suffix with backoff 0 and the backoff rule's weight
    (``oracle_repair``).  Returns (order, tokens, logprob, backoff)."""
    lib = load(lib_path)
    N = int(max_order)
    order = np.ascontiguousarray(order, np.int32)
    tokens = np.ascontiguousarray(tokens, np.int32).reshape(len(order), N)
    logprob = np.ascontiguousarray(logprob, np.float32)
    backoff = np.ascontiguousarray(backoff, np.float32)
    m = ctypes.c_int64()
    po, pt, pw, pb = ctypes.c_void_p(), ctypes.c_void_p(), ctypes.c_void_p(), ctypes.c_void_p()
    rc = lib.oracle_repair(int(vocab_size), N, len(order), _ptr(order), _ptr(tokens), _ptr(logprob), _ptr(backoff),
                           float(unk_logprob), int(bool(bos_eos)), ctypes.byref(m), ctypes.byref(po),
                           ctypes.byref(pt), ctypes.byref(pw), ctypes.byref(pb))
    if rc != 0:
        raise OracleError(rc, lib.oracle_last_error().decode())
    n = int(m.value)
    out = []
    for p, ct, shape in ((po, ctypes.c_int32, (n,)), (pt, ctypes.c_int32, (n, N)), (pw, ctypes.c_float, (n,)),
                         (pb, ctypes.c_float, (n,))):
        arr = np.ctypeslib.as_array(ctypes.cast(p, ctypes.POINTER(ct)), shape=shape).copy()
        lib.oracle_free_buffer(p)
        out.append(arr)
    return tuple(out)


class Oracle:
    """The oracle over an n-gram list (natural-log fp32 weights)."""

    def __init__(self, vocab_size, max_order, order, tokens, logprob, backoff,
                 unk_logprob=float("nan"), lib_path: str = LIB_PATH, bos_eos: bool = False):
        self._lib = load(lib_path)
        self.V = int(vocab_size)
        self.N = int(max_order)
        order = np.ascontiguousarray(order, np.int32)
        tokens = np.ascontiguousarray(tokens, np.int32).reshape(len(order), self.N)
        logprob = np.ascontiguousarray(logprob, np.float32)
        backoff = np.ascontiguousarray(backoff, np.float32)
        h = ctypes.c_void_p()
        rc = self._lib.oracle_create(self.V, self.N, len(order), _ptr(order), _ptr(tokens),
                                     _ptr(logprob), _ptr(backoff), float(unk_logprob), int(bool(bos_eos)),
                                     ctypes.byref(h))
        if rc != 0:
            raise OracleError(rc, self._lib.oracle_last_error().decode())
        self._h = h

    @classmethod
    def from_model(cls, model, lib_path: str = LIB_PATH, shuffle_seed=None):
        order, tokens, logprob, backoff = model.to_list(shuffle_seed)
        return cls(model.vocab_size, model.max_order, order, tokens, logprob, backoff,
                   model.unk_logprob, lib_path, bos_eos=getattr(model, "bos_eos", False))

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self._lib.oracle_free(h)
            self._h = None

    @property
    def num_states(self) -> int:
        return int(self._lib.oracle_num_states(self._h))

    def state_context(self, s: int) -> tuple:
        buf = (ctypes.c_int32 * max(1, self.N))()
        n = self._lib.oracle_state_context(self._h, int(s), buf)
        if n < 0:
            raise OracleError(-12, f"bad state {s}")
        return tuple(buf[i] for i in range(n))

    def state_of(self, ctx) -> int:
        ctx = list(ctx)
        buf = (ctypes.c_int32 * max(1, len(ctx)))(*ctx)
        return int(self._lib.oracle_state_of(self._h, buf, len(ctx)))

    @property
    def start_state(self) -> int:
        return int(self._lib.oracle_start_state(self._h))

    def final(self, states):
        """The </s> score of each state (models with <s>/</s>)."""
        states = np.ascontiguousarray(states, np.int32)
        out = np.empty(len(states), np.float32)
        rc = self._lib.oracle_final(self._h, _ptr(states), len(states), _ptr(out))
        if rc != 0:
            raise OracleError(rc, "final")
        return out

    def advance(self, states, nthreads: int = 1, want64: bool = False):
        """Rows for a batch of states: (scores fp32 [B,V], next int32 [B,V], scores double or None)."""
        states = np.ascontiguousarray(states, np.int32)
        B = len(states)
        s32 = np.empty((B, self.V), np.float32)
        nx = np.empty((B, self.V), np.int32)
        s64 = np.empty((B, self.V), np.float64) if want64 else None
        rc = self._lib.oracle_advance(self._h, _ptr(states), B, _ptr(s32),
                                      _ptr(s64) if want64 else None, _ptr(nx), int(nthreads))
        if rc != 0:
            raise OracleError(rc, "advance")
        return s32, nx, s64

    def greedy_step(self, asr, mode, lam, states, prev=None):
        """One fused step; ``states``/``prev`` (int32 arrays) are updated in place."""
        asr = np.ascontiguousarray(asr, np.float32)
        B, ld = asr.shape
        assert states.dtype == np.int32 and states.flags.c_contiguous and len(states) == B
        if prev is not None:
            assert prev.dtype == np.int32 and prev.flags.c_contiguous and len(prev) == B
        tok = np.empty(B, np.int32)
        rc = self._lib.oracle_greedy_step(self._h, _ptr(asr), B, ld, int(mode), float(lam),
                                          _ptr(states), _ptr(prev) if prev is not None else None,
                                          _ptr(tok))
        if rc != 0:
            raise OracleError(rc, "greedy_step")
        return tok

    def fused_topk(self, asr, lam, k, states):
        """k best fused tokens per hypothesis: (tokens, scores, next states), each [B, k]."""
        asr = np.ascontiguousarray(asr, np.float32)
        B, ld = asr.shape
        states = np.ascontiguousarray(states, np.int32)
        tok = np.empty((B, k), np.int32)
        sc = np.empty((B, k), np.float32)
        nx = np.empty((B, k), np.int32)
        rc = self._lib.oracle_fused_topk(self._h, _ptr(asr), B, ld, float(lam), int(k), _ptr(states),
                                         _ptr(tok), _ptr(sc), _ptr(nx))
        if rc != 0:
            raise OracleError(rc, "fused_topk")
        return tok, sc, nx

    def decode(self, asr, mode, lam, starts=None, nthreads: int = 1, lengths=None, prev=None):
        """Greedy decode of ``asr`` [B, T, C] from ``starts`` [B] (default: the empty context).

        ``lengths`` [B] limits the frames per utterance (later labels are -1);
        ``prev`` [B] is the label before frame 0 (default blank = V).
        Returns per-frame labels and the state after each frame, both [B, T]."""
        asr = np.ascontiguousarray(asr, np.float32)
        B, T, C = asr.shape
        labels = np.empty((B, T), np.int32)
        st = np.empty((B, T), np.int32)
        arrs = []
        for a in (starts, lengths, prev):
            if a is not None:
                a = np.ascontiguousarray(a, np.int32)
                assert len(a) == B
            arrs.append(a)
        rc = self._lib.oracle_decode(self._h, _ptr(asr), B, T, C, int(mode), float(lam),
                                     *[_ptr(a) if a is not None else None for a in arrs],
                                     _ptr(labels), _ptr(st), int(nthreads))
        if rc != 0:
            raise OracleError(rc, "decode")
        return labels, st


__all__ = ["Oracle", "OracleError", "build", "load",
           "MODE_PLAIN", "MODE_CTC", "MODE_TRANSDUCER", "MODE_AED", "LIB_PATH", "SRC_PATH"]
