"""Python binding of libpsc.so (include/psc.h): argument marshalling only.

Every step of the mask path runs in the library's HIP kernels; torch is used
for device memory and streams.  There is no fallback: if the library is
missing or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpsc.so")

PSC_F32, PSC_BF16 = 0, 1
ADV_OK, ADV_REJECTED, ADV_EOS, ADV_OVERFLOW, ADV_BAD_INPUT, ADV_SKIPPED = range(6)
_STATUS = {0: "PSC_OK", -1: "PSC_E_INVALID_ARG", -2: "PSC_E_GRAMMAR", -3: "PSC_E_NOT_LALR1", -4: "PSC_E_OOM",
           -5: "PSC_E_DEVICE", -6: "PSC_E_NOT_BOUND", -7: "PSC_E_LIMIT", -8: "PSC_E_IO", -9: "PSC_E_FORMAT",
           -10: "PSC_E_NOT_VIABLE"}

EXPORTED = ["psc_build", "psc_info", "psc_device_bytes", "psc_bind_device", "psc_compute_masks",
            "psc_apply_mask", "psc_compute_and_apply", "psc_state_reset", "psc_advance",
            "psc_compute_masks_dense", "psc_compute_and_apply_dense", "psc_compute_and_argmax",
            "psc_compute_and_argmax_dense", "psc_compute_classes", "psc_compute_classes_dense", "psc_decode_step",
            "psc_save", "psc_load", "psc_device_error_count", "psc_classify_host", "psc_class_mask_host",
            "psc_host_state", "psc_free", "psc_last_error", "psc_device_bytes_ex", "psc_bind_device_ex",
            "psc_compute_masks_n", "psc_compute_classes_n", "psc_compute_and_apply_n", "psc_compute_and_argmax_n",
            "psc_predictor_fill", "psc_predictor_updates", "psc_timeline_records", "psc_compute_and_apply_timeline",
            "psc_set_options", "psc_compute_and_argmax_noalloc", "psc_grammar_compile", "psc_grammar_view",
            "psc_grammar_symbol_name", "psc_grammar_free", "psc_build_from_text"]

BIND_FLAT, BIND_SLICED = 1, 2
OPT_SPECULATE = 1
_LAYOUTS = {None: 0, "default": 0, "flat": BIND_FLAT, "sliced": BIND_SLICED}


class PscError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_STATUS.get(status, status)}: {msg}")
        self.status = status


# Argument checks (not asserts, so that python -O keeps them): the library
# trusts the sizes it is given, so a tensor of the wrong shape, dtype or
# device must never reach it.  (The lengths of ragged stacks live on the
# device: the calls pass stacks.numel() to the *_n entry points, which
# reject a sequence whose stack would reach past it.)
def _require(ok: bool, what: str) -> None:
    if not ok:
        raise ValueError(f"psc: expected {what}")


_T = {}   # torch types, looked up once


def _torch_types():
    if not _T:
        import torch
        _T.update(tensor=torch.Tensor, i32=torch.int32,
                  codes={torch.float32: PSC_F32, torch.bfloat16: PSC_BF16})
    return _T


def _i32(t, name: str, dev: int, numel: int | None = None, shape: tuple | None = None):
    """t as a contiguous int32 tensor on device index `dev` (get_device(): -1
    for host memory), with numel elements or the given shape."""
    T = _T or _torch_types()
    # one cheap test on the common path; the message is built only on failure
    if (type(t) is T["tensor"] and t.dtype is T["i32"] and t.get_device() == dev and t.is_contiguous()
            and (numel is None or t.numel() == numel) and (shape is None or t.shape == shape)):
        return t
    _require(isinstance(t, T["tensor"]) and t.dtype is T["i32"] and t.is_contiguous(),
             f"{name} to be a contiguous int32 tensor")
    _require(t.get_device() == dev, f"{name} on device {dev} (the bound device), not {t.get_device()}")
    _require(numel is None or t.numel() == numel, f"{name} to hold {numel} elements, not {t.numel()}")
    _require(shape is None or tuple(t.shape) == tuple(shape),
             f"{name} of shape {shape and tuple(shape)}, not {tuple(t.shape)}")
    return t


def _logits(t, dev: int, B: int, V: int) -> int:
    """The dtype code of contiguous logits [B, V] on device index `dev`."""
    T = _T or _torch_types()
    code = T["codes"].get(getattr(t, "dtype", None))
    if (code is not None and type(t) is T["tensor"] and t.get_device() == dev and t.is_contiguous()
            and t.shape == (B, V)):
        return code
    _require(isinstance(t, T["tensor"]) and t.is_contiguous() and tuple(t.shape) == (B, V),
             f"logits to be a contiguous tensor of shape ({B}, {V})")
    _require(t.get_device() == dev, f"logits on device {dev} (the bound device), not {t.get_device()}")
    _require(code is not None, f"float32 or bfloat16 logits, not {t.dtype}")
    return code


def _step_args(dev: int, stacks, lens, qs, logits=None, V: int = 0, out=None, out_cols: int = 0):
    """The checks of one mask-step call in one test on the common path:
    ragged states, optional logits [B, V], optional int32 out ([B, out_cols],
    or [B] when out_cols is 0).  Returns (B, logits dtype code or None)."""
    T = _T or _torch_types()
    i32 = T["i32"]
    try:
        B = lens.numel()
        code = T["codes"].get(logits.dtype) if logits is not None else None
        ok = (lens.dtype is i32 and lens.get_device() == dev and lens.is_contiguous()
              and qs.dtype is i32 and qs.get_device() == dev and qs.is_contiguous() and qs.numel() == B
              and stacks.dtype is i32 and stacks.get_device() == dev and stacks.is_contiguous()
              and (logits is None or (code is not None and logits.get_device() == dev and logits.is_contiguous()
                                      and logits.shape == (B, V)))
              and (out is None or (out.dtype is i32 and out.get_device() == dev and out.is_contiguous()
                                   and out.shape == ((B, out_cols) if out_cols else (B,)))))
    except AttributeError:
        ok = False
    if ok:
        return B, code
    # the slow path names what is wrong
    B = int(_i32(lens, "stack_lens", dev).numel())
    _i32(qs, "lexer_states", dev, numel=B)
    _i32(stacks, "stacks", dev)
    code = _logits(logits, dev, B, V) if logits is not None else None
    if out is not None:
        _i32(out, "out", dev, shape=(B, out_cols) if out_cols else (B,))
    return B, code


class _Grammar(C.Structure):
    _fields_ = [
        ("n_lex_states", C.c_int32), ("lex_next", C.c_void_p), ("lex_accept", C.c_void_p),
        ("n_terminals", C.c_int32), ("terminal_ignored", C.c_void_p), ("end_terminal", C.c_int32),
        ("n_lr_states", C.c_int32), ("n_nonterminals", C.c_int32), ("action", C.c_void_p),
        ("goto_table", C.c_void_p), ("n_productions", C.c_int32), ("prod_lhs", C.c_void_p),
        ("prod_len", C.c_void_p),
    ]


class _Vocab(C.Structure):
    _fields_ = [("n_tokens", C.c_int32), ("bytes", C.c_void_p), ("offsets", C.c_void_p),
                ("eos_id", C.c_int32)]


class Info(C.Structure):
    _fields_ = [
        ("vocab_size", C.c_int32), ("mask_words", C.c_int32), ("mask_stride_words", C.c_int32),
        ("n_lex_states", C.c_int32), ("n_lr_states", C.c_int32), ("n_classes", C.c_int32),
        ("dfa_states_built", C.c_int64), ("dfa_states", C.c_int32), ("dfa_rows", C.c_int32),
        ("dense_rows", C.c_int32), ("max_sparse_edges", C.c_int32), ("table_bytes", C.c_int64),
        ("mask_table_bytes", C.c_int64), ("device_bytes", C.c_int64), ("build_seconds", C.c_double),
        ("chain_states", C.c_int32), ("chains", C.c_int32), ("mask_slices_unique", C.c_int32),
        ("bound_mask_layout", C.c_int32), ("sliced_mask_bytes", C.c_int64),
        ("skip_edges", C.c_int64),
    ]

    def as_dict(self) -> dict:
        return {k: getattr(self, k) for k, _ in self._fields_}


_lib = None


def lib() -> C.CDLL:
    """Load libpsc.so; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: run __graft_entry__.build() "
                              "(or python paper_2608_03065_amd/build.py) first")
        L = C.CDLL(LIB_PATH)
        P, I32, I64 = C.c_void_p, C.c_int32, C.c_int64
        L.psc_build.argtypes = [P, P, C.POINTER(P)]
        L.psc_info.argtypes = [P, P]
        L.psc_device_bytes.argtypes = [P]
        L.psc_device_bytes.restype = C.c_size_t
        L.psc_bind_device.argtypes = [P, P, C.c_size_t, P]
        L.psc_compute_masks.argtypes = [P, P, P, P, I32, P, P]
        L.psc_apply_mask.argtypes = [P, C.c_int, P, I32, I32, P]
        L.psc_compute_and_apply.argtypes = [P, P, P, P, I32, P, P, C.c_int, I32, P]
        L.psc_compute_and_argmax.argtypes = [P, P, P, P, I32, P, C.c_int, I32, P, P]
        L.psc_compute_and_argmax_dense.argtypes = [P, P, I32, P, P, I32, P, C.c_int, I32, P, P]
        L.psc_compute_classes.argtypes = [P, P, P, P, I32, P, P]
        L.psc_compute_classes_dense.argtypes = [P, P, I32, P, P, I32, P, P]
        L.psc_decode_step.argtypes = [P, P, P, P, P, P, P, I32, I32, P, P, P, P, C.c_int, I32, P]
        L.psc_save.argtypes = [P, C.c_char_p]
        L.psc_load.argtypes = [C.c_char_p, C.POINTER(P)]
        L.psc_state_reset.argtypes = [P, P, I32, P, P, I32, P]
        L.psc_advance.argtypes = [P, P, I32, P, P, I32, P, P, P]
        L.psc_compute_masks_dense.argtypes = [P, P, I32, P, P, I32, P, P]
        L.psc_compute_and_apply_dense.argtypes = [P, P, I32, P, P, I32, P, P, C.c_int, I32, P]
        L.psc_device_error_count.argtypes = [P, P, I32, P]
        L.psc_classify_host.argtypes = [P, P, P, P, I32, P]
        L.psc_class_mask_host.argtypes = [P, I32, P]
        L.psc_host_state.argtypes = [P, C.c_char_p, C.c_size_t, P, P, I32, P]
        L.psc_device_bytes_ex.argtypes = [P, C.c_uint32]
        L.psc_device_bytes_ex.restype = C.c_size_t
        L.psc_bind_device_ex.argtypes = [P, P, C.c_size_t, C.c_uint32, P]
        L.psc_compute_masks_n.argtypes = [P, P, I64, P, P, I32, P, P]
        L.psc_compute_classes_n.argtypes = [P, P, I64, P, P, I32, P, P]
        L.psc_compute_and_apply_n.argtypes = [P, P, I64, P, P, I32, P, P, C.c_int, I32, P]
        L.psc_compute_and_argmax_n.argtypes = [P, P, I64, P, P, I32, P, C.c_int, I32, P, P]
        L.psc_compute_and_argmax_noalloc.argtypes = [P, P, I64, P, P, I32, P, C.c_int, I32, P, P]
        L.psc_grammar_compile.argtypes = [C.c_char_p, C.c_size_t, C.POINTER(P)]
        L.psc_grammar_view.argtypes = [P, P]
        L.psc_grammar_symbol_name.argtypes = [P, I32, I32]
        L.psc_grammar_symbol_name.restype = C.c_char_p
        L.psc_grammar_free.argtypes = [P]
        L.psc_grammar_free.restype = None
        L.psc_build_from_text.argtypes = [C.c_char_p, C.c_size_t, P, C.POINTER(P)]
        L.psc_predictor_fill.argtypes = [P, I32, P]
        L.psc_set_options.argtypes = [P, C.c_uint32]
        L.psc_predictor_updates.argtypes = [P, P, I32, P]
        L.psc_timeline_records.argtypes = [P, I32, C.c_int]
        L.psc_timeline_records.restype = I64
        L.psc_compute_and_apply_timeline.argtypes = [P, P, I64, P, P, I32, P, P, C.c_int, I32, P, I64, P]
        L.psc_free.argtypes = [P]
        L.psc_free.restype = None
        L.psc_last_error.restype = C.c_char_p
        for name in ("psc_build", "psc_info", "psc_bind_device", "psc_compute_masks", "psc_apply_mask",
                     "psc_compute_and_apply", "psc_state_reset", "psc_advance", "psc_compute_masks_dense",
                     "psc_compute_and_apply_dense", "psc_compute_and_argmax", "psc_compute_and_argmax_dense",
                     "psc_compute_classes", "psc_compute_classes_dense", "psc_decode_step", "psc_save", "psc_load", "psc_device_error_count",
                     "psc_classify_host", "psc_class_mask_host", "psc_host_state", "psc_bind_device_ex",
                     "psc_compute_masks_n", "psc_compute_classes_n", "psc_compute_and_apply_n",
                     "psc_compute_and_argmax_n", "psc_predictor_fill", "psc_predictor_updates",
                     "psc_compute_and_apply_timeline", "psc_set_options", "psc_compute_and_argmax_noalloc",
                     "psc_grammar_compile", "psc_grammar_view", "psc_build_from_text"):
            getattr(L, name).restype = C.c_int
        _lib = L
    return _lib


def _check(status: int):
    if status != 0:
        raise PscError(status, lib().psc_last_error().decode(errors="replace"))


def _stream_ptr(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def pack_states(states, device=None):
    """[(q, stack bottom->top), ...] -> (stacks int32 [sum len], lens int32 [B], qs int32 [B]),
    numpy on the host, or torch tensors on `device` when given."""
    lens = np.array([len(s[1]) for s in states], dtype=np.int32)
    qs = np.array([s[0] for s in states], dtype=np.int32)
    stacks = (np.concatenate([np.asarray(s[1], dtype=np.int32) for s in states])
              if len(states) else np.zeros(0, np.int32))
    if device is None:
        return stacks, lens, qs
    import torch
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)
    return t(stacks if stacks.size else np.zeros(1, np.int32)), t(lens), t(qs)


class CompiledGrammar:
    """Grammar text compiled by the library (psc_grammar_compile): the lexer
    and LALR(1) tables psc_build takes, as numpy arrays, with the symbol
    names.  Raises PscError (PSC_E_NOT_LALR1 on a conflict)."""

    def __init__(self, text):
        data = text.encode("latin-1") if isinstance(text, str) else bytes(text)
        h = C.c_void_p()
        _check(lib().psc_grammar_compile(data, len(data), C.byref(h)))
        try:
            v = _Grammar()
            _check(lib().psc_grammar_view(h, C.addressof(v)))

            def arr(ptr, n, ct, dt):
                return np.ctypeslib.as_array(C.cast(ptr, C.POINTER(ct)), shape=(n,)).astype(dt).copy() \
                    if n else np.zeros(0, dt)
            nq, nt, ns, nn, npr = v.n_lex_states, v.n_terminals, v.n_lr_states, v.n_nonterminals, v.n_productions
            self.lex_next = arr(v.lex_next, nq * 256, C.c_int32, np.int32).reshape(nq, 256)
            self.lex_accept = arr(v.lex_accept, nq, C.c_int32, np.int32)
            self.terminal_ignored = arr(v.terminal_ignored, nt, C.c_uint8, np.uint8)
            self.end_terminal = int(v.end_terminal)
            self.action = arr(v.action, ns * nt, C.c_int32, np.int32).reshape(ns, nt)
            self.goto = arr(v.goto_table, ns * nn, C.c_int32, np.int32).reshape(ns, nn)
            self.prod_lhs = arr(v.prod_lhs, npr, C.c_int32, np.int32)
            self.prod_len = arr(v.prod_len, npr, C.c_int32, np.int32)
            name = lambda term, i: lib().psc_grammar_symbol_name(h, term, i).decode("latin-1")
            self.terminal_names = [name(1, i) for i in range(nt)]
            self.nonterminal_names = [name(0, i) for i in range(nn)]
        finally:
            lib().psc_grammar_free(h)


def _vocab_struct(vocab):
    toks = vocab.tokens
    offs = np.zeros(len(toks) + 1, dtype=np.int64)
    np.cumsum([len(t) for t in toks], out=offs[1:])
    blob = np.frombuffer(b"".join(toks) + b"\0", dtype=np.uint8).copy()
    return _Vocab(len(toks), blob.ctypes.data, offs.ctypes.data, int(vocab.eos_id)), (blob, offs)


class Classifier:
    """A built (grammar, vocabulary) classifier: psc_build .. psc_free; one
    built from grammar text with Classifier.from_text; or one read back with
    Classifier.load(path)."""

    @classmethod
    def from_text(cls, text, vocab) -> "Classifier":
        """psc_build_from_text: compile the grammar text, then build."""
        data = text.encode("latin-1") if isinstance(text, str) else bytes(text)
        vs, keep = _vocab_struct(vocab)
        h = C.c_void_p()
        _check(lib().psc_build_from_text(data, len(data), C.addressof(vs), C.byref(h)))
        self = cls.__new__(cls)
        self._h = h
        self._dev = None
        self.V = len(vocab.tokens)
        self.W = (self.V + 31) // 32
        return self

    @classmethod
    def load(cls, path: str) -> "Classifier":
        h = C.c_void_p()
        _check(lib().psc_load(os.fsencode(path), C.byref(h)))
        self = cls.__new__(cls)
        self._h = h
        self._dev = None
        inf = self.info()
        self.V = inf["vocab_size"]
        self.W = inf["mask_words"]
        return self

    def save(self, path: str) -> None:
        _check(lib().psc_save(self._h, os.fsencode(path)))

    def __init__(self, grammar, vocab):
        g = grammar
        arrs = dict(
            lex_next=np.ascontiguousarray(g.lexer.next, dtype=np.int32),
            lex_accept=np.ascontiguousarray(g.lexer.accept, dtype=np.int32),
            ignored=np.ascontiguousarray(g.terminal_ignored, dtype=np.uint8),
            action=np.ascontiguousarray(g.action, dtype=np.int32),
            goto=np.ascontiguousarray(g.goto, dtype=np.int32),
            lhs=np.ascontiguousarray(g.prod_lhs, dtype=np.int32),
            plen=np.ascontiguousarray(g.prod_len, dtype=np.int32),
        )
        toks = vocab.tokens
        offs = np.zeros(len(toks) + 1, dtype=np.int64)
        np.cumsum([len(t) for t in toks], out=offs[1:])
        blob = np.frombuffer(b"".join(toks) + b"\0", dtype=np.uint8).copy()
        gs = _Grammar(arrs["lex_next"].shape[0], arrs["lex_next"].ctypes.data, arrs["lex_accept"].ctypes.data,
                      arrs["action"].shape[1], arrs["ignored"].ctypes.data, int(g.end_terminal),
                      arrs["action"].shape[0], arrs["goto"].shape[1], arrs["action"].ctypes.data,
                      arrs["goto"].ctypes.data, arrs["lhs"].shape[0], arrs["lhs"].ctypes.data,
                      arrs["plen"].ctypes.data)
        vs = _Vocab(len(toks), blob.ctypes.data, offs.ctypes.data, int(vocab.eos_id))
        h = C.c_void_p()
        _check(lib().psc_build(C.addressof(gs), C.addressof(vs), C.byref(h)))
        self._h = h
        self._dev = None
        self.V = len(toks)
        self.W = (self.V + 31) // 32

    def __del__(self):
        if getattr(self, "_h", None) is not None and _lib is not None:
            _lib.psc_free(self._h)
            self._h = None

    # ---------------------------------------------------------------- host
    def info(self) -> dict:
        inf = Info()
        _check(lib().psc_info(self._h, C.byref(inf)))
        return inf.as_dict()

    def classify_host(self, states) -> np.ndarray:
        stacks, lens, qs = pack_states(states)
        out = np.zeros(len(states), np.int32)
        st = stacks if stacks.size else np.zeros(1, np.int32)
        _check(lib().psc_classify_host(self._h, st.ctypes.data, lens.ctypes.data, qs.ctypes.data,
                                       len(states), out.ctypes.data))
        return out

    def class_mask(self, cls: int) -> np.ndarray:
        row = np.zeros(self.W, np.uint32)
        _check(lib().psc_class_mask_host(self._h, int(cls), row.ctypes.data))
        return row

    def host_state(self, text: bytes, cap: int = 1 << 16):
        """psc_host_state: the prefix state (q, stack bottom->top) of `text`."""
        _require(isinstance(text, (bytes, bytearray)), "text as bytes")
        stack = np.zeros(max(int(cap), 1), np.int32)
        q, n = C.c_int32(0), C.c_int32(0)
        _check(lib().psc_host_state(self._h, bytes(text), len(text), C.byref(q), stack.ctypes.data, len(stack),
                                    C.byref(n)))
        return int(q.value), stack[:n.value].copy()

    def masks_host(self, states) -> np.ndarray:
        """Host walk + mask lookup (triage; not a device path)."""
        cls = self.classify_host(states)
        out = np.zeros((len(states), self.W), np.uint32)
        for i, c in enumerate(cls):
            if c >= 0:
                out[i] = self.class_mask(c)
        return out

    # -------------------------------------------------------------- device
    def bind(self, device="cuda", stream=None, layout=None):
        """Copy the tables to `device`; layout "flat" or "sliced" chooses the
        mask table's layout (psc_bind_device_ex), None the library default."""
        import torch
        _require(layout in _LAYOUTS, "layout None, 'flat' or 'sliced'")
        flags = _LAYOUTS[layout]
        n = int(lib().psc_device_bytes_ex(self._h, flags))
        buf = torch.empty(n + 256, dtype=torch.uint8, device=device)
        off = (-buf.data_ptr()) % 256
        ptr = buf.data_ptr() + off
        _check(lib().psc_bind_device_ex(self._h, ptr, n, flags, _stream_ptr(stream)))
        self._dev = buf
        self._device = buf.device
        self._dev_index = buf.get_device()
        self._dev_ptr = ptr
        return self

    def set_options(self, speculate: bool = False):
        """psc_set_options: PSC_OPT_SPECULATE when `speculate`."""
        _check(lib().psc_set_options(self._h, OPT_SPECULATE if speculate else 0))
        return self

    def predictor_fill(self, cls: int = -1, stream=None):
        """Every class-predictor entry to `cls` (-1: no prediction)."""
        _check(lib().psc_predictor_fill(self._h, int(cls), _stream_ptr(stream)))

    def predictor_updates(self, reset: bool = False, stream=None) -> int:
        """Walks whose class differed from the prediction since the last reset."""
        v = C.c_uint32()
        _check(lib().psc_predictor_updates(self._h, C.byref(v), int(reset), _stream_ptr(stream)))
        return int(v.value)

    def timeline_records(self, B: int, dtype) -> int:
        code = (_T or _torch_types())["codes"][dtype]
        return int(lib().psc_timeline_records(self._h, int(B), code))

    def compute_and_apply_timeline(self, stacks, stack_lens, lexer_states, logits, records, out=None, stream=None):
        """psc_compute_and_apply_timeline: the fused step with per-wavefront
        clock records (records: int64 device tensor [n, 4])."""
        B, dt = _step_args(self._idx, stacks, stack_lens, lexer_states, logits, self.V, out, self.W)
        T = _T or _torch_types()
        import torch
        _require(isinstance(records, T["tensor"]) and records.dtype == torch.int64 and records.is_contiguous()
                 and records.dim() == 2 and records.shape[1] == 4 and records.get_device() == self._idx,
                 "records as a contiguous int64 device tensor [n, 4]")
        out_ptr = None if out is None else out.data_ptr()
        _check(lib().psc_compute_and_apply_timeline(self._h, stacks.data_ptr(), stacks.numel(),
                                                    stack_lens.data_ptr(), lexer_states.data_ptr(), B, out_ptr,
                                                    logits.data_ptr(), dt, self.V, records.data_ptr(),
                                                    records.shape[0], _stream_ptr(stream)))
        return logits

    @property
    def device(self):
        """The device the tables are bound to (PSC_E_NOT_BOUND before bind)."""
        dev = getattr(self, "_device", None)
        if dev is None:
            raise PscError(-6, "the classifier is not bound to a device (call bind first)")
        return dev

    @property
    def _idx(self) -> int:
        idx = getattr(self, "_dev_index", None)
        if idx is None:
            raise PscError(-6, "the classifier is not bound to a device (call bind first)")
        return idx

    def compute_masks(self, stacks, stack_lens, lexer_states, out=None, stream=None):
        """Device int32 tensors -> uint32 bitmask [B, W] (torch.int32 view)."""
        import torch
        if out is None:
            out = torch.empty((int(stack_lens.shape[0]), self.W), dtype=torch.int32, device=self.device)
        B, _ = _step_args(self._idx, stacks, stack_lens, lexer_states, out=out, out_cols=self.W)
        _check(lib().psc_compute_masks_n(self._h, stacks.data_ptr(), stacks.numel(), stack_lens.data_ptr(),
                                         lexer_states.data_ptr(), B, out.data_ptr(), _stream_ptr(stream)))
        return out

    def compute_classes(self, stacks, stack_lens, lexer_states, out=None, stream=None):
        """Device int32 tensors -> class ids int32 [B] (-1 for a rejected input)."""
        import torch
        if out is None:
            out = torch.empty(int(stack_lens.shape[0]), dtype=torch.int32, device=self.device)
        B, _ = _step_args(self._idx, stacks, stack_lens, lexer_states, out=out)
        _check(lib().psc_compute_classes_n(self._h, stacks.data_ptr(), stacks.numel(), stack_lens.data_ptr(),
                                           lexer_states.data_ptr(), B, out.data_ptr(), _stream_ptr(stream)))
        return out

    def compute_and_apply(self, stacks, stack_lens, lexer_states, logits, out=None, stream=None):
        """One launch: masks for the B prefix states applied to logits [B, V] in
        place; the bitmask is also written to `out` when given.  Returns logits."""
        B, dt = _step_args(self._idx, stacks, stack_lens, lexer_states, logits, self.V, out, self.W)
        out_ptr = None if out is None else out.data_ptr()
        _check(lib().psc_compute_and_apply_n(self._h, stacks.data_ptr(), stacks.numel(), stack_lens.data_ptr(),
                                             lexer_states.data_ptr(), B, out_ptr, logits.data_ptr(), dt,
                                             self.V, _stream_ptr(stream)))
        return logits

    def compute_and_argmax(self, stacks, stack_lens, lexer_states, logits, out=None, stream=None):
        """Greedy token per sequence under its mask (int32 [B]; -1 = none
        allowed); the logits are only read."""
        import torch
        if out is None:
            out = torch.empty(int(stack_lens.shape[0]), dtype=torch.int32, device=self.device)
        B, dt = _step_args(self._idx, stacks, stack_lens, lexer_states, logits, self.V, out)
        _check(lib().psc_compute_and_argmax_n(self._h, stacks.data_ptr(), stacks.numel(), stack_lens.data_ptr(),
                                              lexer_states.data_ptr(), B, logits.data_ptr(), dt, self.V,
                                              out.data_ptr(), _stream_ptr(stream)))
        return out

    def compute_and_argmax_noalloc(self, stacks, stack_lens, lexer_states, logits, out, stream=None):
        """compute_and_argmax whose records live in the library's fixed
        per-GPU array (the call allocates nothing; B <= 4096; calls on one
        GPU must not overlap).  `out` is required: int32 [B]."""
        B, dt = _step_args(self._idx, stacks, stack_lens, lexer_states, logits, self.V, out)
        _check(lib().psc_compute_and_argmax_noalloc(self._h, stacks.data_ptr(), stacks.numel(),
                                                    stack_lens.data_ptr(), lexer_states.data_ptr(), B,
                                                    logits.data_ptr(), dt, self.V, out.data_ptr(),
                                                    _stream_ptr(stream)))
        return out

    def error_count(self, reset: bool = False, stream=None) -> int:
        v = C.c_uint32()
        _check(lib().psc_device_error_count(self._h, C.byref(v), int(reset), _stream_ptr(stream)))
        return int(v.value)


class DecodeStates:
    """B device-resident prefix states in the dense layout of psc_advance:
    stacks int32 [B, cap], lens int32 [B], qs int32 [B] (torch tensors)."""

    def __init__(self, clf: Classifier, B: int, cap: int, device="cuda", stream=None):
        import torch
        self.clf, self.B, self.cap = clf, int(B), int(cap)
        self.stacks = torch.zeros((self.B, self.cap), dtype=torch.int32, device=device)
        self.lens = torch.zeros(self.B, dtype=torch.int32, device=device)
        self.qs = torch.zeros(self.B, dtype=torch.int32, device=device)
        self.status = torch.zeros(self.B, dtype=torch.int32, device=device)
        _require(self.stacks.device == clf.device, f"the states on the classifier's device {clf.device}")
        self.reset(stream)

    def reset(self, stream=None):
        """Every sequence to the empty prefix (q0, stack [0])."""
        _check(lib().psc_state_reset(self.clf._h, self.stacks.data_ptr(), self.cap, self.lens.data_ptr(),
                                     self.qs.data_ptr(), self.B, _stream_ptr(stream)))
        return self

    def load(self, states):
        """Set the states from host (q, stack bottom->top) pairs."""
        import torch
        _require(len(states) == self.B, f"{self.B} states, not {len(states)}")
        st = np.zeros((self.B, self.cap), np.int32)
        for b, (q, a) in enumerate(states):
            _require(1 <= len(a) <= self.cap, f"stacks of 1 to {self.cap} symbols, not {len(a)}")
            st[b, :len(a)] = a
        self.stacks.copy_(torch.from_numpy(st))
        self.lens.copy_(torch.tensor([len(a) for _, a in states], dtype=torch.int32))
        self.qs.copy_(torch.tensor([q for q, _ in states], dtype=torch.int32))
        return self

    def advance(self, tokens, stream=None):
        """One token per sequence (int32 device tensor [B], < 0 = skip);
        returns the status tensor (ADV_*)."""
        _i32(tokens, "tokens", self.clf._idx, numel=self.B)
        _check(lib().psc_advance(self.clf._h, self.stacks.data_ptr(), self.cap, self.lens.data_ptr(),
                                 self.qs.data_ptr(), self.B, tokens.data_ptr(), self.status.data_ptr(),
                                 _stream_ptr(stream)))
        return self.status

    def compute_masks(self, out=None, stream=None):
        import torch
        if out is None:
            out = torch.empty((self.B, self.clf.W), dtype=torch.int32, device=self.lens.device)
        _i32(out, "out", self.clf._idx, shape=(self.B, self.clf.W))
        _check(lib().psc_compute_masks_dense(self.clf._h, self.stacks.data_ptr(), self.cap, self.lens.data_ptr(),
                                             self.qs.data_ptr(), self.B, out.data_ptr(), _stream_ptr(stream)))
        return out

    def compute_classes(self, out=None, stream=None):
        import torch
        if out is None:
            out = torch.empty(self.B, dtype=torch.int32, device=self.lens.device)
        _i32(out, "out", self.clf._idx, numel=self.B)
        _check(lib().psc_compute_classes_dense(self.clf._h, self.stacks.data_ptr(), self.cap, self.lens.data_ptr(),
                                               self.qs.data_ptr(), self.B, out.data_ptr(), _stream_ptr(stream)))
        return out

    def compute_and_apply(self, logits, out=None, stream=None):
        dt = _logits(logits, self.clf._idx, self.B, self.clf.V)
        out_ptr = None
        if out is not None:
            out_ptr = _i32(out, "out", self.clf._idx, shape=(self.B, self.clf.W)).data_ptr()
        _check(lib().psc_compute_and_apply_dense(self.clf._h, self.stacks.data_ptr(), self.cap,
                                                 self.lens.data_ptr(), self.qs.data_ptr(), self.B, out_ptr,
                                                 logits.data_ptr(), dt, self.clf.V, _stream_ptr(stream)))
        return logits

    def argmax(self, logits, out=None, stream=None):
        """Greedy token per sequence under its mask (int32 [B]; -1 = none)."""
        import torch
        dt = _logits(logits, self.clf._idx, self.B, self.clf.V)
        if out is None:
            out = torch.empty(self.B, dtype=torch.int32, device=logits.device)
        _i32(out, "out", self.clf._idx, numel=self.B)
        _check(lib().psc_compute_and_argmax_dense(self.clf._h, self.stacks.data_ptr(), self.cap,
                                                  self.lens.data_ptr(), self.qs.data_ptr(), self.B,
                                                  logits.data_ptr(), dt, self.clf.V, out.data_ptr(),
                                                  _stream_ptr(stream)))
        return out

    def decode_step(self, tokens, logits, out=None, stream=None):
        """psc_decode_step: advance by `tokens` (int32 [B], < 0 = skip), then
        mask `logits` [B, V] for the new states in place, in one launch.  The
        new states go to a second set of buffers, which then become this
        object's; returns the status tensor (ADV_*)."""
        import torch
        dev, T = self.clf._idx, (_T or _torch_types())
        dt = T["codes"].get(getattr(logits, "dtype", None))
        try:
            ok = (tokens.dtype is T["i32"] and tokens.get_device() == dev and tokens.is_contiguous()
                  and tokens.numel() == self.B and dt is not None and logits.get_device() == dev
                  and logits.is_contiguous() and logits.shape == (self.B, self.clf.V))
        except AttributeError:
            ok = False
        if not ok:      # names what is wrong
            _i32(tokens, "tokens", dev, numel=self.B)
            dt = _logits(logits, dev, self.B, self.clf.V)
        if getattr(self, "_spare", None) is None:
            self._spare = (torch.empty_like(self.stacks), torch.empty_like(self.lens), torch.empty_like(self.qs))
        so, lo, qo = self._spare
        out_ptr = None
        if out is not None:
            out_ptr = _i32(out, "out", self.clf._idx, shape=(self.B, self.clf.W)).data_ptr()
        _check(lib().psc_decode_step(self.clf._h, self.stacks.data_ptr(), self.lens.data_ptr(), self.qs.data_ptr(),
                                     so.data_ptr(), lo.data_ptr(), qo.data_ptr(), self.cap, self.B,
                                     tokens.data_ptr(), self.status.data_ptr(), out_ptr, logits.data_ptr(), dt,
                                     self.clf.V, _stream_ptr(stream)))
        self._spare = (self.stacks, self.lens, self.qs)
        self.stacks, self.lens, self.qs = so, lo, qo
        return self.status

    def host_states(self):
        """The states as host (q, stack) pairs (synchronises)."""
        st = self.stacks.cpu().numpy()
        lens = self.lens.cpu().numpy()
        qs = self.qs.cpu().numpy()
        return [(int(qs[b]), st[b, :lens[b]].copy()) for b in range(self.B)]


def apply_mask(logits, bitmask, stream=None):
    """In place: logits[b, v] = -inf where bit v of bitmask[b] is 0."""
    import torch
    _require(isinstance(logits, torch.Tensor) and logits.is_cuda and logits.dim() == 2,
             "logits to be a 2-D device tensor")
    B, V = logits.shape
    dt = _logits(logits, logits.get_device(), B, V)
    _i32(bitmask, "bitmask", logits.get_device(), shape=(B, (V + 31) // 32))
    _check(lib().psc_apply_mask(logits.data_ptr(), dt, bitmask.data_ptr(), B, V, _stream_ptr(stream)))
    return logits
