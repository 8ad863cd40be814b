"""Thin ctypes binding of libtbias.so (include/tbias.h).

Argument marshalling only: every computation happens in the library. The
functions keep the C names; torch tensors are accepted for device buffers and
passed as raw pointers together with the current HIP stream. If the library is
not built, importing this module raises: there is no fallback path.
"""

from __future__ import annotations

import ctypes as C
import os
from pathlib import Path
from typing import Optional, Sequence, Tuple

import numpy as np

_PKG = Path(__file__).resolve().parent
LIB_PATH = _PKG / "libtbias.so"

TB_OK, TB_EINVAL, TB_ENOMEM, TB_EHIP, TB_ERANGE, TB_EIO = 0, -1, -2, -3, -4, -5
TB_F32, TB_BF16 = 0, 1
TB_COMMIT, TB_PURE_POTENTIAL = 0, 1
TB_STATE_NONE, TB_STATE_INVALID, TB_STATE_TIMEOUT = -1, -2, -3
TB_MAX_BEAM = 32
# tb_debug_select_kernels choices
GREEDY_AUTO, GREEDY_REF = 0, 1
BEAM_AUTO, BEAM_REF, BEAM_NO_PIPE = 0, 1, 2


class tb_arena_layout(C.Structure):
    _fields_ = [
        ("total_bytes", C.c_int64),
        ("n_models", C.c_int32),
        ("v_plus_blank", C.c_int32),
        ("n_states", C.c_int64),
        ("off_model_off", C.c_int64), ("off_model_n", C.c_int64),
        ("off_first_child", C.c_int64), ("off_n_child", C.c_int64),
        ("off_link", C.c_int64), ("off_label", C.c_int64),
        ("off_phi", C.c_int64), ("off_psi", C.c_int64),
        ("off_root_psi", C.c_int64), ("off_root_dst", C.c_int64),
        ("off_class_map", C.c_int64), ("off_cls_ptr", C.c_int64), ("off_cls_tok", C.c_int64),
        ("off_arc_mem", C.c_int64),
        ("max_children", C.c_int32),
        ("max_depth", C.c_int32),
        ("max_override", C.c_int32),
        ("off_value_tab", C.c_int64), ("off_state_rec", C.c_int64),
    ]


class tb_arena(C.Structure):
    _fields_ = [("base", C.c_void_p), ("layout", tb_arena_layout)]


class TbError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"tbias error {code}: {msg}")
        self.code = code


def _load() -> C.CDLL:
    # torch carries its own HIP runtime. Importing it first makes libtbias bind
    # to that same runtime (same soname), so the device buffers and HIP
    # streams torch hands over belong to the runtime the library launches on.
    import torch  # noqa: F401
    if not LIB_PATH.exists():
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2608_21343_amd.build`")
    lib = C.CDLL(str(LIB_PATH))
    P, I32, I64 = C.c_void_p, C.c_int32, C.c_int64
    sig = {
        "tb_compile_graphs": [I32, P, P, P, P, P, P, P, I32, I32, I32, C.POINTER(C.c_void_p)],
        "tb_compile_variative": [I32, P, P, P, P, P, P, P, P, I32, P, I32, C.c_float, I32, I32,
                                 C.POINTER(C.c_void_p)],
        "tb_graphs_layout": [P, C.POINTER(tb_arena_layout)],
        "tb_graphs_host_image": [P, P, I64],
        "tb_graphs_upload": [P, P, I64, P, C.POINTER(tb_arena)],
        "tb_validate_image": [P, C.POINTER(tb_arena_layout)],
        "tb_init_states": [C.POINTER(tb_arena), I32, I32, P, P, P, P],
        "tb_boost_step_greedy": [C.POINTER(tb_arena), P, I32, I32, I32, I64, P, P, P, P, P, P],
        "tb_boost_step_beam": [C.POINTER(tb_arena), P, I32, I32, I32, I32, I64, P, P, P, P, P, P,
                               P, P, P],
        "tb_reset_stream": [C.POINTER(tb_arena), I32, I32, I32, I32, P, P, P, P],
        "tb_init_beam_stream": [C.POINTER(tb_arena), I32, I32, P, P, P, P, P, P],
        "tb_boost_step_beam_stream": [C.POINTER(tb_arena), P, I32, I32, I32, I32, I64, P, P, P,
                                      P, P, I32, P, I32, P, P, P, P, P, P],
        "tb_debug_select_kernels": [I32, I32],
        "tb_debug_set_spin_limit": [C.c_uint32],
        "tb_debug_launch_empty": [I32, I32, I32, P],
        "tb_registry_layout": [I32, I64, I32, C.POINTER(tb_arena_layout)],
        "tb_registry_create": [I32, I64, P, I32, P, I64, P, C.POINTER(C.c_void_p)],
        "tb_registry_arena": [P, C.POINTER(tb_arena)],
        "tb_registry_model": [P, I32, C.POINTER(C.c_int64), C.POINTER(C.c_int32)],
        "tb_register_models": [P, P, P, P],
        "tb_unregister_model": [P, I32, P, I64, P],
        "tb_unregister_model_noalloc": [P, I32, P],
        "tb_graphs_cache_create": [P, I32, I64, C.POINTER(C.c_void_p)],
        "tb_graphs_cache_compile": [P, I32, P, P, P, P, P, P, I32, I32, P,
                                    C.POINTER(C.c_void_p)],
        "tb_graphs_cache_stats": [P, P],
        "tb_graphs_save": [P, C.c_char_p],
        "tb_graphs_load": [C.c_char_p, C.POINTER(C.c_void_p)],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = C.c_int
    lib.tb_graphs_free.argtypes = [P]
    lib.tb_graphs_free.restype = None
    lib.tb_registry_free.argtypes = [P]
    lib.tb_registry_free.restype = None
    lib.tb_graphs_cache_free.argtypes = [P]
    lib.tb_graphs_cache_free.restype = None
    for name in ("tb_registry_used_states", "tb_unregister_workspace_bytes"):
        getattr(lib, name).restype = C.c_int64
    lib.tb_registry_used_states.argtypes = [P]
    lib.tb_unregister_workspace_bytes.argtypes = [P, I32]
    lib.tb_last_error.argtypes = []
    lib.tb_last_error.restype = C.c_char_p
    return lib


LIB = _load()

EXPORTED = ("tb_compile_graphs", "tb_graphs_layout", "tb_graphs_host_image", "tb_graphs_upload",
            "tb_graphs_free", "tb_validate_image", "tb_init_states", "tb_boost_step_greedy",
            "tb_boost_step_beam", "tb_reset_stream", "tb_last_error",
            "tb_debug_select_kernels", "tb_debug_set_spin_limit", "tb_debug_launch_empty",
            "tb_registry_layout", "tb_registry_create", "tb_registry_arena", "tb_registry_model",
            "tb_registry_used_states", "tb_register_models", "tb_unregister_workspace_bytes",
            "tb_unregister_model", "tb_registry_free", "tb_unregister_model_noalloc",
            "tb_init_beam_stream", "tb_boost_step_beam_stream", "tb_compile_variative",
            "tb_graphs_cache_create", "tb_graphs_cache_compile", "tb_graphs_cache_stats",
            "tb_graphs_cache_free", "tb_graphs_save", "tb_graphs_load")


def _check(code: int) -> None:
    if code != TB_OK:
        raise TbError(code, LIB.tb_last_error().decode(errors="replace"))


def _np_ptr(a: np.ndarray) -> C.c_void_p:
    return C.c_void_p(a.ctypes.data)


def _dptr(t, dtype=None, name="tensor") -> Optional[int]:
    """Device pointer of a torch tensor (None passes NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must have dtype {dtype}, got {t.dtype}")
    return t.data_ptr()


def _need(t, n: int, name: str, exact: bool = True) -> None:
    """Reject a buffer whose element count does not fit the call (the kernels
    trust these sizes)."""
    if t is None:
        raise ValueError(f"{name} is required")
    k = t.numel()
    if (k != n) if exact else (k < n):
        raise ValueError(f"{name} holds {k} elements, needs {'' if exact else 'at least '}{n}")


def _stream(stream) -> Optional[int]:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


# ---------------------------------------------------------------------------
# host-side compile


class Graphs:
    """Library-owned compiled graphs (tb_graphs*)."""

    def __init__(self, handle: int):
        self._h = C.c_void_p(handle)
        self.layout = tb_arena_layout()
        _check(LIB.tb_graphs_layout(self._h, C.byref(self.layout)))

    def host_image(self) -> np.ndarray:
        img = np.empty(self.layout.total_bytes, dtype=np.uint8)
        _check(LIB.tb_graphs_host_image(self._h, _np_ptr(img), img.nbytes))
        return img

    def free(self) -> None:
        if self._h:
            LIB.tb_graphs_free(self._h)
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def _list_args(model_phrase_ptr, phrase_tok_ptr, phrase_tokens, token_w, end_bonus, scale):
    """Host arrays of the phrase-list arguments (weights broadcast per model)."""
    mp = np.ascontiguousarray(model_phrase_ptr, dtype=np.int64)
    tp = np.ascontiguousarray(phrase_tok_ptr, dtype=np.int64)
    tk = np.ascontiguousarray(phrase_tokens, dtype=np.int32)
    n_models = len(mp) - 1
    tw = np.ascontiguousarray(np.broadcast_to(np.asarray(token_w, np.float32), (n_models,)))
    eb = np.ascontiguousarray(np.broadcast_to(np.asarray(end_bonus, np.float32), (n_models,)))
    sc = None if scale is None else np.ascontiguousarray(
        np.broadcast_to(np.asarray(scale, np.float32), (n_models,)))
    keep = (mp, tp, tk, tw, eb, sc)  # alive for the call
    ptrs = (n_models, _np_ptr(mp), _np_ptr(tp), _np_ptr(tk) if tk.size else None, _np_ptr(tw),
            _np_ptr(eb), _np_ptr(sc) if sc is not None else None)
    return keep, ptrs


def tb_compile_graphs(model_phrase_ptr, phrase_tok_ptr, phrase_tokens, token_w, end_bonus,
                      class_map, scale=None, semantics: int = TB_COMMIT,
                      n_threads: int = 0) -> Graphs:
    keep, ptrs = _list_args(model_phrase_ptr, phrase_tok_ptr, phrase_tokens, token_w, end_bonus,
                            scale)
    cm = np.ascontiguousarray(class_map, dtype=np.int32)
    out = C.c_void_p()
    _check(LIB.tb_compile_graphs(*ptrs, _np_ptr(cm), len(cm), semantics, n_threads,
                                 C.byref(out)))
    del keep
    return Graphs(out.value)


class GraphsCache:
    """Host-memory cache of compiled models for one class map
    (tb_graphs_cache_*). compile() returns what tb_compile_graphs would, byte
    for byte, taking the models it has compiled before from the cache."""

    def __init__(self, class_map, capacity_bytes: int = 256 << 20):
        cm = np.ascontiguousarray(class_map, dtype=np.int32)
        h = C.c_void_p()
        _check(LIB.tb_graphs_cache_create(_np_ptr(cm), len(cm), int(capacity_bytes), C.byref(h)))
        self._h = h

    def compile(self, model_phrase_ptr, phrase_tok_ptr, phrase_tokens, token_w, end_bonus,
                scale=None, semantics: int = TB_COMMIT, n_threads: int = 0):
        """(Graphs, number of models taken from the cache)."""
        keep, ptrs = _list_args(model_phrase_ptr, phrase_tok_ptr, phrase_tokens, token_w,
                                end_bonus, scale)
        out, hits = C.c_void_p(), C.c_int32()
        _check(LIB.tb_graphs_cache_compile(self._h, *ptrs, semantics, n_threads, C.byref(hits),
                                           C.byref(out)))
        del keep
        return Graphs(out.value), int(hits.value)

    def stats(self) -> dict:
        st = np.zeros(5, dtype=np.int64)
        _check(LIB.tb_graphs_cache_stats(self._h, _np_ptr(st)))
        return dict(zip(("hits", "misses", "models", "bytes", "dropped"), (int(x) for x in st)))

    def free(self) -> None:
        if self._h:
            LIB.tb_graphs_cache_free(self._h)
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def tb_graphs_save(graphs: Graphs, path) -> None:
    _check(LIB.tb_graphs_save(graphs._h, os.fsencode(os.fspath(path))))


def tb_graphs_load(path) -> Graphs:
    out = C.c_void_p()
    _check(LIB.tb_graphs_load(os.fsencode(os.fspath(path)), C.byref(out)))
    return Graphs(out.value)


def tb_compile_variative(model_phrase_ptr, phrase_char_ptr, phrase_chars, token_w, end_bonus,
                         token_char_ptr, token_chars, lower, tau: float, scale=None,
                         semantics: int = TB_COMMIT, n_threads: int = 0) -> Graphs:
    """Variative BPE graphs of character-coded phrase lists over a piece
    vocabulary (token v spells token_chars[token_char_ptr[v]:token_char_ptr[v+1]])."""
    mp = np.ascontiguousarray(model_phrase_ptr, dtype=np.int64)
    pp = np.ascontiguousarray(phrase_char_ptr, dtype=np.int64)
    pc = np.ascontiguousarray(phrase_chars, dtype=np.int32)
    n_models = len(mp) - 1
    tw = np.ascontiguousarray(np.broadcast_to(np.asarray(token_w, np.float32), (n_models,)))
    eb = np.ascontiguousarray(np.broadcast_to(np.asarray(end_bonus, np.float32), (n_models,)))
    sc = None if scale is None else np.ascontiguousarray(
        np.broadcast_to(np.asarray(scale, np.float32), (n_models,)))
    tp = np.ascontiguousarray(token_char_ptr, dtype=np.int64)
    tc = np.ascontiguousarray(token_chars, dtype=np.int32)
    lo = np.ascontiguousarray(lower, dtype=np.int32)
    out = C.c_void_p()
    _check(LIB.tb_compile_variative(n_models, _np_ptr(mp), _np_ptr(pp),
                                    _np_ptr(pc) if pc.size else None, _np_ptr(tw), _np_ptr(eb),
                                    _np_ptr(sc) if sc is not None else None, _np_ptr(tp),
                                    _np_ptr(tc) if tc.size else None, len(tp), _np_ptr(lo),
                                    len(lo), float(tau), semantics, n_threads, C.byref(out)))
    return Graphs(out.value)


def tb_validate_image(image: np.ndarray, layout: tb_arena_layout) -> None:
    img = np.ascontiguousarray(image, dtype=np.uint8)
    _check(LIB.tb_validate_image(_np_ptr(img), C.byref(layout)))


# ---------------------------------------------------------------------------
# device side


class Arena:
    """A device arena: caller-owned (torch) device buffer plus tb_arena."""

    def __init__(self, buf, arena: tb_arena):
        self.buf = buf          # keeps the device memory alive
        self.arena = arena

    @property
    def layout(self) -> tb_arena_layout:
        return self.arena.layout


def tb_graphs_upload(graphs: Graphs, device="cuda", stream=None) -> Arena:
    import torch
    nbytes = graphs.layout.total_bytes
    buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
    base = buf.data_ptr()
    pad = (-base) % 256
    arena = tb_arena()
    _check(LIB.tb_graphs_upload(graphs._h, C.c_void_p(base + pad), nbytes, _stream(stream),
                                C.byref(arena)))
    return Arena(buf, arena)


def tb_init_states(arena: Arena, B: int, K: int, model_ids, states, scores=None,
                   stream=None) -> None:
    import torch
    _check(LIB.tb_init_states(C.byref(arena.arena), B, K,
                              _dptr(model_ids, torch.int32, "model_ids"),
                              _dptr(states, torch.int32, "states"),
                              _dptr(scores, torch.float32, "scores"), _stream(stream)))


def _logits_args(logits):
    """(dtype code, row stride) of a logits tensor; shape and layout checks only."""
    import torch
    if logits.dtype == torch.float32:
        dt = TB_F32
    elif logits.dtype == torch.bfloat16:
        dt = TB_BF16
    else:
        raise ValueError("logits must be float32 or bfloat16")
    if logits.stride(-1) != 1:
        raise ValueError("logits rows must be contiguous")
    return dt, logits.stride(-2)


def _logits_ptr(logits) -> int:
    if not logits.is_cuda:
        raise ValueError("logits must be a device tensor")
    return logits.data_ptr()


def tb_boost_step_greedy(arena: Arena, logits, model_ids, states, out_tok, out_state, out_score,
                         T: Optional[int] = None, B: Optional[int] = None,
                         row_stride: Optional[int] = None, stream=None) -> None:
    """logits: [T, B, V+1] (or [T, B, 1, V+1]) device tensor, rows contiguous."""
    import torch
    dt, rs = _logits_args(logits)
    if logits.dim() == 4:
        if logits.shape[2] != 1:
            raise ValueError("greedy logits must have K = 1")
        rs = logits.stride(1)
    if logits.dim() not in (3, 4):
        raise ValueError("greedy logits must be [T, B, V+1] or [T, B, 1, V+1]")
    if logits.shape[-1] != arena.layout.v_plus_blank:
        raise ValueError(f"logits rows hold {logits.shape[-1]} values, the arena has "
                         f"V+1 = {arena.layout.v_plus_blank}")
    if T is not None and not 0 <= T <= logits.shape[0]:
        raise ValueError(f"T = {T} outside [0, {logits.shape[0]}]")
    if B is not None and B != logits.shape[1]:
        raise ValueError(f"B = {B} differs from the logits' {logits.shape[1]} streams")
    T = logits.shape[0] if T is None else T
    B = logits.shape[1]
    if T > 1 and logits.stride(0) != B * rs:
        raise ValueError("logits steps must be laid out as (t*B + b) * row_stride")
    if row_stride is not None and row_stride != rs:
        raise ValueError(f"row_stride {row_stride} differs from the logits' {rs}")
    _need(model_ids, B, "model_ids")
    _need(states, B, "states")
    for name, o in (("out_tok", out_tok), ("out_state", out_state), ("out_score", out_score)):
        _need(o, T * B, name, exact=False)
    ptr = _logits_ptr(logits)
    _check(LIB.tb_boost_step_greedy(C.byref(arena.arena), C.c_void_p(ptr), dt, T, B, rs,
                                    _dptr(model_ids, torch.int32, "model_ids"),
                                    _dptr(states, torch.int32, "states"),
                                    _dptr(out_tok, torch.int32, "out_tok"),
                                    _dptr(out_state, torch.int32, "out_state"),
                                    _dptr(out_score, torch.float32, "out_score"),
                                    _stream(stream)))


def tb_boost_step_beam(arena: Arena, logits, model_ids, states, scores, out_tok, out_parent,
                       out_state, out_step, out_cum, stream=None) -> None:
    """logits: [T, B, K, V+1] device tensor with (t, b, k) rows at ((t*B+b)*K+k)*row_stride."""
    import torch
    dt, rs = _logits_args(logits)
    if logits.dim() != 4:
        raise ValueError("beam logits must be [T, B, K, V+1]")
    T, B, K, Vp1 = logits.shape
    if Vp1 != arena.layout.v_plus_blank:
        raise ValueError(f"logits rows hold {Vp1} values, the arena has "
                         f"V+1 = {arena.layout.v_plus_blank}")
    if logits.stride(1) != K * rs or (T > 1 and logits.stride(0) != B * K * rs):
        raise ValueError("beam logits must be laid out as ((t*B + b)*K + k) * row_stride")
    _need(model_ids, B, "model_ids")
    _need(states, B * K, "states")
    _need(scores, B * K, "scores")
    for name, o in (("out_tok", out_tok), ("out_parent", out_parent), ("out_state", out_state),
                    ("out_step", out_step), ("out_cum", out_cum)):
        _need(o, T * B * K, name, exact=False)
    ptr = _logits_ptr(logits)
    _check(LIB.tb_boost_step_beam(C.byref(arena.arena), C.c_void_p(ptr), dt, T, B, K, rs,
                                  _dptr(model_ids, torch.int32, "model_ids"),
                                  _dptr(states, torch.int32, "states"),
                                  _dptr(scores, torch.float32, "scores"),
                                  _dptr(out_tok, torch.int32, "out_tok"),
                                  _dptr(out_parent, torch.int32, "out_parent"),
                                  _dptr(out_state, torch.int32, "out_state"),
                                  _dptr(out_step, torch.float32, "out_step"),
                                  _dptr(out_cum, torch.float32, "out_cum"),
                                  _stream(stream)))


# tb_hyp: 24 bytes, held as three int64 words (hash, prefix hash, last | node << 32)
HYP_WORDS = 3
TB_HASH_MUL = 0x9E3779B97F4A7C15


def hyp_fields(hyps) -> Tuple[np.ndarray, np.ndarray, np.ndarray, np.ndarray]:
    """(hash, prefix_hash, last, node) of a host copy of tb_hyp records
    (an int64 array of shape [..., 3])."""
    h = np.ascontiguousarray(np.asarray(hyps, dtype=np.int64))
    words = h.view(np.uint64)
    ln = h[..., 2:3].copy().view(np.int32)
    return words[..., 0], words[..., 1], ln[..., 0], ln[..., 1]


def sequence_hash(seq) -> int:
    """The tb_hyp hash of a label sequence (empty: 0; appending v: h*MUL + v + 1 mod 2^64)."""
    h = 0
    for v in seq:
        h = (h * TB_HASH_MUL + int(v) + 1) & 0xFFFFFFFFFFFFFFFF
    return h


def tb_init_beam_stream(arena: Arena, B: int, K: int, model_ids, states, scores, hyps, tree_len,
                        stream=None) -> None:
    """hyps: device int64 [B*K, 3] (tb_hyp records); tree_len: device int32 [B]."""
    import torch
    _need(model_ids, B, "model_ids")
    _need(states, B * K, "states")
    _need(scores, B * K, "scores")
    _need(hyps, B * K * HYP_WORDS, "hyps")
    _need(tree_len, B, "tree_len")
    _check(LIB.tb_init_beam_stream(C.byref(arena.arena), B, K,
                                   _dptr(model_ids, torch.int32, "model_ids"),
                                   _dptr(states, torch.int32, "states"),
                                   _dptr(scores, torch.float32, "scores"),
                                   _dptr(hyps, torch.int64, "hyps"),
                                   _dptr(tree_len, torch.int32, "tree_len"), _stream(stream)))


def tb_boost_step_beam_stream(arena: Arena, logits, model_ids, states, scores, hyps, tree,
                              tree_len, out_tok, out_parent, out_state, out_step, out_cum,
                              recombine: bool = True, stream=None) -> None:
    """tb_boost_step_beam with the hypothesis carry: hyps device int64 [B*K, 3],
    tree device int32 [B, tree_cap, 2] (or None with tree_cap 0), tree_len
    device int32 [B]."""
    import torch
    dt, rs = _logits_args(logits)
    if logits.dim() != 4:
        raise ValueError("beam logits must be [T, B, K, V+1]")
    T, B, K, Vp1 = logits.shape
    if Vp1 != arena.layout.v_plus_blank:
        raise ValueError(f"logits rows hold {Vp1} values, the arena has "
                         f"V+1 = {arena.layout.v_plus_blank}")
    if logits.stride(1) != K * rs or (T > 1 and logits.stride(0) != B * K * rs):
        raise ValueError("beam logits must be laid out as ((t*B + b)*K + k) * row_stride")
    _need(model_ids, B, "model_ids")
    _need(states, B * K, "states")
    _need(scores, B * K, "scores")
    _need(hyps, B * K * HYP_WORDS, "hyps")
    _need(tree_len, B, "tree_len")
    if tree is None:
        cap = 0
    else:
        if tree.dim() != 3 or tree.shape[0] != B or tree.shape[2] != 2:
            raise ValueError("tree must be [B, tree_cap, 2]")
        cap = tree.shape[1]
    for name, o in (("out_tok", out_tok), ("out_parent", out_parent), ("out_state", out_state),
                    ("out_step", out_step), ("out_cum", out_cum)):
        _need(o, T * B * K, name, exact=False)
    ptr = _logits_ptr(logits)
    _check(LIB.tb_boost_step_beam_stream(
        C.byref(arena.arena), C.c_void_p(ptr), dt, T, B, K, rs,
        _dptr(model_ids, torch.int32, "model_ids"), _dptr(states, torch.int32, "states"),
        _dptr(scores, torch.float32, "scores"), _dptr(hyps, torch.int64, "hyps"),
        _dptr(tree, torch.int32, "tree"), cap, _dptr(tree_len, torch.int32, "tree_len"),
        1 if recombine else 0, _dptr(out_tok, torch.int32, "out_tok"),
        _dptr(out_parent, torch.int32, "out_parent"), _dptr(out_state, torch.int32, "out_state"),
        _dptr(out_step, torch.float32, "out_step"), _dptr(out_cum, torch.float32, "out_cum"),
        _stream(stream)))


def tb_reset_stream(arena: Arena, b: int, new_model_id: int, K: int, model_ids, states,
                    scores=None, stream=None) -> None:
    import torch
    B = model_ids.numel()
    if states.numel() != B * K or (scores is not None and scores.numel() != B * K):
        raise ValueError("states/scores must hold B*K entries")
    _check(LIB.tb_reset_stream(C.byref(arena.arena), B, b, new_model_id, K,
                               _dptr(model_ids, torch.int32, "model_ids"),
                               _dptr(states, torch.int32, "states"),
                               _dptr(scores, torch.float32, "scores"), _stream(stream)))


class Registry:
    """Model lifecycle on a device arena with free capacity (tb_registry_*).

    The device buffer is a torch tensor owned by this object. ``arena`` is the
    current tb_arena for step calls (the same object is updated in place
    after every lifecycle call, so Arena wrappers built from it stay valid)."""

    def __init__(self, max_models: int, max_states: int, class_map, device="cuda", stream=None):
        import torch
        cm = np.ascontiguousarray(class_map, dtype=np.int32)
        lay = tb_arena_layout()
        _check(LIB.tb_registry_layout(max_models, max_states, len(cm), C.byref(lay)))
        self.buf = torch.empty(lay.total_bytes + 256, dtype=torch.uint8, device=device)
        base = self.buf.data_ptr()
        self._base = base + (-base) % 256
        h = C.c_void_p()
        _check(LIB.tb_registry_create(max_models, max_states, _np_ptr(cm), len(cm),
                                      C.c_void_p(self._base), lay.total_bytes, _stream(stream),
                                      C.byref(h)))
        self._h = h
        self.max_models = max_models
        self.device = device
        self.arena = Arena(self.buf, tb_arena())
        self._refresh()

    def _refresh(self):
        _check(LIB.tb_registry_arena(self._h, C.byref(self.arena.arena)))

    def model(self, model_id: int):
        """(first state, state count) of an id; count 0 for a free id."""
        f, n = C.c_int64(), C.c_int32()
        _check(LIB.tb_registry_model(self._h, model_id, C.byref(f), C.byref(n)))
        return f.value, n.value

    @property
    def used_states(self) -> int:
        return int(LIB.tb_registry_used_states(self._h))

    def register(self, graphs: Graphs, stream=None) -> list:
        ids = np.zeros(graphs.layout.n_models, dtype=np.int32)
        _check(LIB.tb_register_models(self._h, graphs._h, _np_ptr(ids), _stream(stream)))
        self._refresh()
        return [int(i) for i in ids]

    def workspace_bytes(self, model_id: int) -> int:
        return int(LIB.tb_unregister_workspace_bytes(self._h, model_id))

    def unregister(self, model_id: int, workspace=None, stream=None) -> None:
        """Remove a model; ``workspace`` is a device tensor of at least
        workspace_bytes(model_id) bytes (allocated here when None)."""
        import torch
        need = self.workspace_bytes(model_id)
        if workspace is None and need > 0:
            workspace = torch.empty(need, dtype=torch.uint8, device=self.device)
        ptr = None if workspace is None else workspace.data_ptr()
        nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
        _check(LIB.tb_unregister_model(self._h, model_id, ptr, nbytes, _stream(stream)))
        self._refresh()
        self._last_workspace = workspace  # alive until the stream has used it

    def unregister_noalloc(self, model_id: int, stream=None) -> None:
        """Remove a model through the library's own scratch (no allocation)."""
        _check(LIB.tb_unregister_model_noalloc(self._h, model_id, _stream(stream)))
        self._refresh()

    def free(self) -> None:
        if getattr(self, "_h", None):
            LIB.tb_registry_free(self._h)
            self._h = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def tb_debug_select_kernels(greedy: int = GREEDY_AUTO, beam: int = BEAM_AUTO) -> None:
    """Test hook: force a kernel family (see tbias.h)."""
    _check(LIB.tb_debug_select_kernels(greedy, beam))


def tb_debug_set_spin_limit(polls: int = 0) -> None:
    """Test hook: poll limit of the greedy hand-off wait (0 = default)."""
    _check(LIB.tb_debug_set_spin_limit(polls))


def tb_debug_launch_empty(grid: int, block: int, lds_bytes: int = 0, stream=None) -> None:
    """Measurement hook: enqueue a kernel that does nothing (see tbias.h)."""
    _check(LIB.tb_debug_launch_empty(grid, block, lds_bytes, _stream(stream)))


class kernels:
    """Context manager for tests: ``with capi.kernels(greedy=GREEDY_REF): ...``."""

    def __init__(self, greedy: int = GREEDY_AUTO, beam: int = BEAM_AUTO):
        self.choice = (greedy, beam)

    def __enter__(self):
        tb_debug_select_kernels(*self.choice)
        return self

    def __exit__(self, *exc):
        tb_debug_select_kernels(GREEDY_AUTO, BEAM_AUTO)
        return False


def image_arrays(image: np.ndarray, layout: tb_arena_layout) -> dict:
    """Views of the arrays inside a host arena image (see tb_arena_layout)."""
    L = layout
    N, M, V1 = L.n_states, L.n_models, L.v_plus_blank

    def arr(off, n, dt):
        return np.frombuffer(image, dtype=dt, count=n, offset=off)

    return {
        "model_off": arr(L.off_model_off, M, np.int32),
        "model_n": arr(L.off_model_n, M, np.int32),
        "first_child": arr(L.off_first_child, N, np.int32),
        "n_child": arr(L.off_n_child, N, np.int32),
        "link": arr(L.off_link, N, np.int32),
        "label": arr(L.off_label, N, np.int32),
        "phi": arr(L.off_phi, N, np.float32),
        "psi": arr(L.off_psi, N, np.float32),
        "root_psi": arr(L.off_root_psi, M * V1, np.float32).reshape(M, V1),
        "root_dst": arr(L.off_root_dst, M * V1, np.int32).reshape(M, V1),
        "class_map": arr(L.off_class_map, V1, np.int32),
        "cls_ptr": arr(L.off_cls_ptr, V1, np.int32),
        "cls_tok": arr(L.off_cls_tok, V1 - 1, np.int32),
        "arc_mem": arr(L.off_arc_mem, 2 * L.n_states, np.uint32),
        "value_tab": arr(L.off_value_tab, 512 * M, np.float32).reshape(M, 512),
        "state_rec": arr(L.off_state_rec, 3 * N, np.uint32).reshape(N, 3),
    }
