"""Batched backoff n-gram language model for MI355X (the NGPU-LM query, arXiv 2505.22857).

A thin ctypes binding of ``libngpu_lm.so`` (C ABI in ``include/ngpu_lm.h``).
Every step of a query runs in the library's HIP kernels; this module only
marshals arguments.  PyTorch supplies device memory and the current HIP
stream.  The library must be built first (``__graft_entry__.build()`` or
``python -m paper_2505_22857_amd.build``); without it every call raises.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libngpu_lm.so")

NGPU_FUSION_PLAIN, NGPU_FUSION_CTC, NGPU_FUSION_TRANSDUCER, NGPU_FUSION_AED = 0, 1, 2, 3
NGPU_BUILD_BOS_EOS = 1
NGPU_BUILD_REPAIR_CLOSURE = 2
MAX_ORDER = 10
MAX_VOCAB = 8192
MAX_BATCH = (1 << 26) - 256      # NGPU_LM_MAX_BATCH

ERROR_NAMES = {
    -1: "INVALID_ARG", -2: "TOKEN_RANGE", -3: "ORDER_RANGE", -4: "DUPLICATE_NGRAM",
    -5: "MISSING_PREFIX", -6: "MISSING_SUFFIX", -7: "MISSING_UNIGRAM", -8: "NOT_UPLOADED",
    -9: "HIP", -10: "NONFINITE", -11: "TOO_LARGE", -12: "BAD_STATE", -13: "NO_MEMORY",
}

EXPORTED = [
    "ngpu_lm_build", "ngpu_lm_free", "ngpu_lm_info", "ngpu_lm_state_context", "ngpu_lm_device_bytes",
    "ngpu_lm_upload", "ngpu_lm_advance", "ngpu_lm_fused_greedy_step", "ngpu_lm_fused_greedy_decode",
    "ngpu_lm_fused_topk", "ngpu_lm_start_state", "ngpu_lm_final_weights",
    "ngpu_lm_check_states", "ngpu_lm_sync_check",
    "ngpu_lm_query_bytes", "ngpu_lm_host_image", "ngpu_lm_last_error",
    "ngpu_arpa_parse", "ngpu_arpa_list", "ngpu_arpa_free",
]


class NgpuError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"NGPU_E_{ERROR_NAMES.get(code, code)}: {msg}")
        self.code = code


class _NgramList(ctypes.Structure):
    _fields_ = [("num_ngrams", ctypes.c_int64), ("max_order", ctypes.c_int32),
                ("order", ctypes.c_void_p), ("tokens", ctypes.c_void_p),
                ("logprob", ctypes.c_void_p), ("backoff", ctypes.c_void_p)]


class _Info(ctypes.Structure):
    _fields_ = [("num_states", ctypes.c_int64), ("num_arcs", ctypes.c_int64),
                ("max_order", ctypes.c_int32), ("vocab_size", ctypes.c_int32),
                ("device_bytes", ctypes.c_int64)]


_lib = None


def load_library(path: str = LIB_PATH):
    """Load the HIP library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build() "
                           "(there is no fallback path)")
    lib = ctypes.CDLL(path)
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    lib.ngpu_lm_build.argtypes = [ctypes.POINTER(_NgramList), i32, ctypes.c_float, ctypes.c_uint32,
                                  ctypes.POINTER(vp)]
    lib.ngpu_lm_free.argtypes = [vp]
    lib.ngpu_lm_free.restype = None
    lib.ngpu_lm_info.argtypes = [vp, ctypes.POINTER(_Info)]
    lib.ngpu_lm_state_context.argtypes = [vp, i64, vp, ctypes.POINTER(i32)]
    lib.ngpu_lm_device_bytes.argtypes = [vp]
    lib.ngpu_lm_device_bytes.restype = ctypes.c_size_t
    lib.ngpu_lm_upload.argtypes = [vp, vp, ctypes.c_size_t, vp]
    lib.ngpu_lm_advance.argtypes = [vp, vp, i64, vp, vp, vp]
    lib.ngpu_lm_fused_greedy_step.argtypes = [vp, vp, i64, i64, i32, ctypes.c_float, vp, vp, vp, vp]
    lib.ngpu_lm_fused_greedy_decode.argtypes = [vp, vp, i64, i64, i64, i64, vp, i32, ctypes.c_float,
                                                vp, vp, vp, vp, vp]
    lib.ngpu_lm_start_state.argtypes = [vp, ctypes.POINTER(i64)]
    lib.ngpu_lm_final_weights.argtypes = [vp, vp, i64, vp, vp]
    lib.ngpu_lm_fused_topk.argtypes = [vp, vp, i64, i64, ctypes.c_float, i32, vp, vp, vp, vp, vp]
    lib.ngpu_lm_check_states.argtypes = [vp, vp, ctypes.POINTER(i64)]
    lib.ngpu_lm_sync_check.argtypes = [vp, vp]
    lib.ngpu_lm_query_bytes.argtypes = [vp, vp, i64, ctypes.POINTER(i64), ctypes.POINTER(i64)]
    lib.ngpu_lm_host_image.argtypes = [vp, ctypes.POINTER(vp), ctypes.POINTER(ctypes.c_size_t)]
    lib.ngpu_arpa_parse.argtypes = [ctypes.c_char_p, ctypes.c_size_t, vp, i32, ctypes.c_uint32,
                                    ctypes.POINTER(vp)]
    lib.ngpu_arpa_list.argtypes = [vp, ctypes.POINTER(_NgramList), ctypes.POINTER(ctypes.c_float)]
    lib.ngpu_arpa_free.argtypes = [vp]
    lib.ngpu_arpa_free.restype = None
    lib.ngpu_lm_last_error.argtypes = []
    lib.ngpu_lm_last_error.restype = ctypes.c_char_p
    for name in EXPORTED:
        if name not in ("ngpu_lm_free", "ngpu_lm_device_bytes", "ngpu_lm_last_error", "ngpu_arpa_free"):
            getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _check(rc: int):
    if rc != 0:
        raise NgpuError(rc, load_library().ngpu_lm_last_error().decode())


_torch = None


def _torch_mod():
    global _torch
    if _torch is None:
        import torch
        _torch = torch
    return _torch


def _stream_handle(stream, device: int = -1) -> int:
    """Raw HIP stream of ``stream``, or of the current stream of ``device`` (the
    current device when -1).  The raw query skips building a stream object,
    which costs more than the kernel launch itself for one small step."""
    torch = _torch_mod()
    if stream is not None:
        return stream.cuda_stream
    raw = getattr(torch._C, "_cuda_getCurrentRawStream", None)
    if raw is not None:
        return raw(device if device >= 0 else torch.cuda.current_device())
    return torch.cuda.current_stream().cuda_stream


def _dptr(t, dtype, name) -> int:
    """Device address of a contiguous device tensor of ``dtype`` (dtypes are
    singletons, so ``is`` compares them)."""
    try:
        ok = t.dtype is dtype and t.is_cuda and t.is_contiguous()
    except AttributeError:
        ok = False
    if not ok:
        raise TypeError(f"{name} must be a contiguous {dtype} device tensor")
    return t.data_ptr()


def parse_arpa(text, vocab, bos_eos: bool = False):
    """Parse ARPA text with the library's reader.

    Returns ``(max_order, order, tokens, logprob, backoff, unk_logprob)`` as
    numpy copies (natural-log fp32 weights), ready for ``NgpuLM``."""
    lib = load_library()
    data = text.encode() if isinstance(text, str) else bytes(text)
    words = [w.encode() for w in vocab]
    arr = (ctypes.c_char_p * len(words))(*words)
    h = ctypes.c_void_p()
    _check(lib.ngpu_arpa_parse(data, len(data), ctypes.cast(arr, ctypes.c_void_p), len(words),
                               NGPU_BUILD_BOS_EOS if bos_eos else 0, ctypes.byref(h)))
    try:
        lst = _NgramList()
        unk = ctypes.c_float()
        _check(lib.ngpu_arpa_list(h, ctypes.byref(lst), ctypes.byref(unk)))
        M, N = int(lst.num_ngrams), int(lst.max_order)

        def arr_of(ptr, ct, n):
            if n == 0:
                return np.zeros(0, np.dtype(ct))
            return np.ctypeslib.as_array(ctypes.cast(ptr, ctypes.POINTER(ct)), shape=(n,)).copy()
        order = arr_of(lst.order, ctypes.c_int32, M)
        tokens = arr_of(lst.tokens, ctypes.c_int32, M * N).reshape(M, N)
        logprob = arr_of(lst.logprob, ctypes.c_float, M)
        backoff = arr_of(lst.backoff, ctypes.c_float, M)
        return N, order, tokens, logprob, backoff, float(unk.value)
    finally:
        lib.ngpu_arpa_free(h)


class NgpuLM:
    """A trie built from an n-gram list (natural-log fp32 weights)."""

    def __init__(self, vocab_size: int, max_order: int, order, tokens, logprob, backoff,
                 unk_logprob: float = float("nan"), bos_eos: bool = False, repair: bool = False):
        self._lib = load_library()
        self._h = None
        order = np.ascontiguousarray(order, np.int32)
        tokens = np.ascontiguousarray(tokens, np.int32).reshape(len(order), int(max_order))
        logprob = np.ascontiguousarray(logprob, np.float32)
        backoff = np.ascontiguousarray(backoff, np.float32)
        lst = _NgramList(len(order), int(max_order), order.ctypes.data, tokens.ctypes.data,
                         logprob.ctypes.data, backoff.ctypes.data)
        h = ctypes.c_void_p()
        _check(self._lib.ngpu_lm_build(ctypes.byref(lst), int(vocab_size), float(unk_logprob),
                                       (NGPU_BUILD_BOS_EOS if bos_eos else 0) |
                                       (NGPU_BUILD_REPAIR_CLOSURE if repair else 0), ctypes.byref(h)))
        self._h = h
        info = _Info()
        _check(self._lib.ngpu_lm_info(h, ctypes.byref(info)))
        self.num_states = int(info.num_states)
        self.num_arcs = int(info.num_arcs)
        self.max_order = int(info.max_order)
        self.vocab_size = int(info.vocab_size)
        self.device_bytes = int(info.device_bytes)
        self.bos_eos = bool(bos_eos)
        st = ctypes.c_int64()
        _check(self._lib.ngpu_lm_start_state(h, ctypes.byref(st)))
        self.start_state = int(st.value)
        self._dev = None

    @classmethod
    def from_model(cls, model, shuffle_seed: Optional[int] = None):
        return cls(model.vocab_size, model.max_order, *model.to_list(shuffle_seed), model.unk_logprob,
                   bos_eos=getattr(model, "bos_eos", False))

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self._lib.ngpu_lm_free(h)
            self._h = None

    def state_context(self, state: int) -> tuple:
        buf = (ctypes.c_int32 * max(1, self.max_order))()
        k = ctypes.c_int32()
        _check(self._lib.ngpu_lm_state_context(self._h, int(state), buf, ctypes.byref(k)))
        return tuple(buf[i] for i in range(k.value))

    def upload(self, device="cuda", stream=None):
        """Allocate the device image with torch and copy the trie into it."""
        import torch
        buf = torch.empty(self.device_bytes + 256, dtype=torch.uint8, device=device)
        off = (-buf.data_ptr()) % 256
        view = buf[off:off + self.device_bytes]
        with torch.cuda.device(buf.device):
            _check(self._lib.ngpu_lm_upload(self._h, ctypes.c_void_p(view.data_ptr()), self.device_bytes,
                                            _stream_handle(stream)))
        self._dev = buf
        self.device = buf.device
        return self

    def advance(self, states, scores=None, next_states=None, stream=None):
        """Scores [B, V] fp32 and next states [B, V] int32 for device int32 ``states`` [B]."""
        import torch
        B = states.numel()
        if scores is None:
            scores = torch.empty((B, self.vocab_size), dtype=torch.float32, device=states.device)
        if next_states is None:
            next_states = torch.empty((B, self.vocab_size), dtype=torch.int32, device=states.device)
        if scores.numel() < B * self.vocab_size or next_states.numel() < B * self.vocab_size:
            raise ValueError("output tensors are too small")
        _check(self._lib.ngpu_lm_advance(self._h, _dptr(states, torch.int32, "states"), B,
                                         _dptr(scores, torch.float32, "scores"),
                                         _dptr(next_states, torch.int32, "next_states"),
                                         _stream_handle(stream)))
        return scores, next_states

    def _classes(self, mode: int) -> int:
        """Classes an ASR row holds in ``mode``: V, plus blank (or <eos>) outside plain fusion."""
        return self.vocab_size + (0 if mode == NGPU_FUSION_PLAIN else 1)

    def fused_greedy_step(self, asr, lam: float, states, prev=None, mode: int = NGPU_FUSION_PLAIN,
                          tokens=None, stream=None):
        """One greedy fusion step; ``states`` (and ``prev`` for CTC) are updated in place."""
        import torch
        if asr.dim() != 2 or asr.stride(1) != 1:
            raise TypeError("asr must be a [B, ld] tensor with unit stride in the last dimension")
        B, C = asr.shape
        if C < self.vocab_size + (mode != NGPU_FUSION_PLAIN):
            raise ValueError(f"asr rows must hold {self._classes(mode)} classes for mode {mode}")
        if states.numel() != B or (prev is not None and prev.numel() != B):
            raise ValueError("states/prev must hold B entries")
        if tokens is None:
            tokens = torch.empty(B, dtype=torch.int32, device=asr.device)
        if tokens.numel() < B:
            raise ValueError("tokens must hold at least B entries")
        if asr.dtype is not torch.float32 or not asr.is_cuda:
            raise TypeError("asr must be a float32 device tensor")
        _check(self._lib.ngpu_lm_fused_greedy_step(
            self._h, asr.data_ptr(), B, asr.stride(0), int(mode), float(lam),
            _dptr(states, torch.int32, "states"),
            _dptr(prev, torch.int32, "prev") if prev is not None else None,
            _dptr(tokens, torch.int32, "tokens"), _stream_handle(stream)))
        return tokens

    def final_weights(self, states, out=None, stream=None):
        """fp32 final (</s>) weight of each state of device int32 ``states``."""
        import torch
        if out is None:
            out = torch.empty(states.numel(), dtype=torch.float32, device=states.device)
        if out.numel() < states.numel():
            raise ValueError("out must hold one entry per state")
        _check(self._lib.ngpu_lm_final_weights(self._h, _dptr(states, torch.int32, "states"), states.numel(),
                                               _dptr(out, torch.float32, "out"), _stream_handle(stream)))
        return out

    def fused_topk(self, asr, lam: float, k: int, states, tokens=None, scores=None, next_states=None,
                   stream=None):
        """k best fused tokens per hypothesis: (tokens int32, scores fp32, next states int32), each [B, k]
        (allocated unless given)."""
        import torch
        if asr.dim() != 2 or asr.stride(1) != 1 or asr.dtype != torch.float32 or not asr.is_cuda:
            raise TypeError("asr must be a float32 [B, ld] device tensor with unit stride in the last dimension")
        B = asr.shape[0]
        if asr.shape[1] < self.vocab_size:
            raise ValueError(f"asr rows must hold {self.vocab_size} classes")
        if states.numel() != B:
            raise ValueError("states must hold B entries")
        tok = torch.empty((B, k), dtype=torch.int32, device=asr.device) if tokens is None else tokens
        sc = torch.empty((B, k), dtype=torch.float32, device=asr.device) if scores is None else scores
        nx = torch.empty((B, k), dtype=torch.int32, device=asr.device) if next_states is None else next_states
        if tok.numel() < B * k or sc.numel() < B * k or nx.numel() < B * k:
            raise ValueError("output tensors are too small")
        _check(self._lib.ngpu_lm_fused_topk(self._h, asr.data_ptr(), B, asr.stride(0), float(lam),
                                            int(k), _dptr(states, torch.int32, "states"),
                                            _dptr(tok, torch.int32, "tokens"), _dptr(sc, torch.float32, "scores"),
                                            _dptr(nx, torch.int32, "next"), _stream_handle(stream)))
        return tok, sc, nx

    def fused_greedy_decode(self, asr, lam: float, states, prev=None, lengths=None,
                            mode: int = NGPU_FUSION_PLAIN, labels=None, label_states=None, stream=None):
        """Greedy decode of ``asr`` [B, T, C] (last dimension contiguous) in one launch.

        ``states`` (and ``prev`` for CTC) are updated in place to the final
        state (and label).  Returns labels [B, T] int32 (-1 past ``lengths``)."""
        import torch
        if asr.dim() != 3 or asr.stride(2) != 1 or asr.dtype != torch.float32 or not asr.is_cuda:
            raise TypeError("asr must be a float32 [B, T, C] device tensor with unit class stride")
        B, T, C = asr.shape
        if C < self._classes(mode):
            raise ValueError(f"asr rows must hold {self._classes(mode)} classes for mode {mode}")
        if states.numel() != B or (prev is not None and prev.numel() != B):
            raise ValueError("states/prev must hold B entries")
        if labels is None:
            labels = torch.empty((B, T), dtype=torch.int32, device=asr.device)
        if labels.numel() != B * T:
            raise ValueError("labels must hold B * T entries")
        if label_states is not None and label_states.numel() != B * T:
            raise ValueError("label_states must hold B * T entries")
        if lengths is not None and lengths.numel() != B:
            raise ValueError("lengths must hold B entries")
        _check(self._lib.ngpu_lm_fused_greedy_decode(
            self._h, asr.data_ptr(), B, T, asr.stride(0), asr.stride(1),
            _dptr(lengths, torch.int32, "lengths") if lengths is not None else None, int(mode), float(lam),
            _dptr(states, torch.int32, "states"),
            _dptr(prev, torch.int32, "prev") if prev is not None else None,
            _dptr(labels, torch.int32, "labels"),
            _dptr(label_states, torch.int32, "label_states") if label_states is not None else None,
            _stream_handle(stream)))
        return labels

    def check_states(self, stream=None) -> int:
        n = ctypes.c_int64()
        rc = self._lib.ngpu_lm_check_states(self._h, _stream_handle(stream), ctypes.byref(n))
        if rc not in (0, -12):
            _check(rc)
        return int(n.value)

    def sync_check(self, stream=None) -> None:
        """Raise NgpuError (BAD_STATE) if queries since the last check met out-of-range states."""
        _check(self._lib.ngpu_lm_sync_check(self._h, _stream_handle(stream)))

    def host_image(self) -> np.ndarray:
        """Copy of the host trie image (uint8), the bytes ``upload`` copies to the device."""
        p, n = ctypes.c_void_p(), ctypes.c_size_t()
        _check(self._lib.ngpu_lm_host_image(self._h, ctypes.byref(p), ctypes.byref(n)))
        return np.ctypeslib.as_array((ctypes.c_uint8 * n.value).from_address(p.value)).copy()

    def query_bytes(self, states) -> tuple:
        """(algorithmic HBM bytes, total bytes) of ``advance`` on host ``states``."""
        s = np.ascontiguousarray(states, np.int32)
        hbm, tot = ctypes.c_int64(), ctypes.c_int64()
        _check(self._lib.ngpu_lm_query_bytes(self._h, s.ctypes.data, len(s), ctypes.byref(hbm),
                                             ctypes.byref(tot)))
        return int(hbm.value), int(tot.value)


__all__ = ["NgpuLM", "NgpuError", "load_library", "parse_arpa", "LIB_PATH", "EXPORTED", "NGPU_BUILD_BOS_EOS",
           "NGPU_BUILD_REPAIR_CLOSURE",
           "NGPU_FUSION_PLAIN", "NGPU_FUSION_CTC", "NGPU_FUSION_TRANSDUCER", "NGPU_FUSION_AED"]
