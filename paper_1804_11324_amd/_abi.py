"""ctypes binding of liblmbr.so: the C ABI of include/lmbr.h, argument marshalling only.

Every function here has the name of the C entry point it calls and does no
arithmetic of its own: device buffers are torch tensors (or raw pointers),
streams are torch streams, and every compute step runs in the HIP library.
The binding refuses to run when the library is missing: there is no CPU path.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import (POINTER, Structure, byref, c_char_p, c_double, c_float, c_int32, c_int64,
                    c_size_t, c_uint32, c_uint64, c_void_p)
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liblmbr.so")

LMBR_OK, LMBR_E_INVALID, LMBR_E_CAPACITY, LMBR_E_HIP, LMBR_E_STATE, LMBR_E_DEVICE = 0, -1, -2, -3, -4, -5
LMBR_DEV_NONFINITE, LMBR_DEV_TABLE = 1, 2
LMBR_MAX_K, LMBR_MAX_V, LMBR_MAX_ORDER = 16, 262144, 4
LMBR_STATIC_SCRATCH_BYTES = 4194304

EXPORTS = [
    "lmbr_last_error", "lmbr_create", "lmbr_destroy", "lmbr_device_bytes", "lmbr_workspace_bytes",
    "lmbr_device_status", "lmbr_static_scratch_bytes", "lmbr_beam_step_logits_static",
    "lmbr_set_projection", "lmbr_load_posteriors", "lmbr_state_init", "lmbr_state_probe",
    "lmbr_synth_hidden", "lmbr_project", "lmbr_beam_step", "lmbr_beam_step_logits",
    "lmbr_score", "lmbr_score_logits", "lmbr_select", "lmbr_traceback",
    "lmbr_decode", "lmbr_gather_rows", "lmbr_table_build", "lmbr_table_free",
    "lmbr_set_decode_options", "lmbr_set_sentence_steps", "lmbr_set_constraints",
    "lmbr_set_step_path", "lmbr_projected_rows", "lmbr_set_lmbr_layout", "lmbr_table_dense",
    "lmbr_table_history_count", "lmbr_plan_batches", "lmbr_table_bytes", "lmbr_load_posteriors_into",
]
LMBR_FINISH_AT_T, LMBR_FINISH_EOS_BACKUP = 0, 1
LMBR_STEP_TWO_PASS, LMBR_STEP_FUSED = 0, 1
LMBR_L_SPARSE, LMBR_L_DENSE = 0, 1


class LmbrError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"lmbr error {code}: {msg}")
        self.code = code


class lmbr_config(Structure):
    _fields_ = [("B", c_int32), ("K", c_int32), ("V", c_int32), ("H", c_int32),
                ("T_max", c_int32), ("eos_id", c_int32), ("lam", c_float),
                ("theta", c_float * 5), ("load_factor", c_float)]


class lmbr_beam_state(Structure):
    _fields_ = [("q", c_void_p), ("ctx", c_void_p), ("hhash", c_void_p), ("len", c_void_p),
                ("ranges", c_void_p), ("bp", c_void_p), ("tok", c_void_p), ("qhist", c_void_p),
                ("sent", c_void_p), ("t", c_int32)]


class lmbr_decode_options(Structure):
    _fields_ = [("length_norm", c_int32), ("finish", c_int32), ("early_prune", c_int32),
                ("prune_width", c_double)]


class lmbr_table_image(Structure):
    _fields_ = [("n_slots", c_int64), ("n_entries", c_int64),
                ("slot_key", POINTER(c_uint64)), ("slot_off", POINTER(c_uint32)),
                ("slot_cnt", POINTER(c_uint32)), ("entry_tok", POINTER(c_int32)),
                ("entry_post", POINTER(c_float)), ("uni_off", c_uint32), ("uni_cnt", c_uint32)]


# int32_t (*lmbr_state_fn)(void *user, int32_t t, const lmbr_beam_state *st,
#                          uint16_t *hidden_out, hipStream_t stream)
LMBR_STATE_FN = ctypes.CFUNCTYPE(c_int32, c_void_p, c_int32, POINTER(lmbr_beam_state), c_void_p, c_void_p)

_lib = None


def lib():
    """Load liblmbr.so once (after torch, so both share torch's HIP runtime)."""
    global _lib
    if _lib is not None:
        return _lib
    import torch  # noqa: F401  (binds libamdhip64 first)
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_1804_11324_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    P = c_void_p
    sig = {
        "lmbr_last_error": (c_char_p, [P]),
        "lmbr_workspace_bytes": (c_size_t, [POINTER(lmbr_config)]),
        "lmbr_create": (c_int32, [POINTER(lmbr_config), P, c_size_t, POINTER(c_void_p)]),
        "lmbr_device_status": (c_int32, [P, POINTER(c_int32), P]),
        "lmbr_static_scratch_bytes": (c_size_t, [POINTER(lmbr_config)]),
        "lmbr_beam_step_logits_static": (c_int32, [P, POINTER(lmbr_beam_state), P, c_int64, P, P, P, P, P]),
        "lmbr_destroy": (None, [P]),
        "lmbr_device_bytes": (c_size_t, [P]),
        "lmbr_set_projection": (c_int32, [P, P, c_int32, P, P]),
        "lmbr_load_posteriors": (c_int32, [P, c_int32, c_int64, P, P, P, P]),
        "lmbr_table_bytes": (c_size_t, [P, c_int64, P, P, P]),
        "lmbr_load_posteriors_into": (c_int32, [P, c_int32, c_int64, P, P, P, P, c_size_t, P]),
        "lmbr_state_init": (c_int32, [P, POINTER(lmbr_beam_state), c_uint64, P]),
        "lmbr_state_probe": (c_int32, [P, POINTER(lmbr_beam_state), P]),
        "lmbr_synth_hidden": (c_int32, [P, POINTER(lmbr_beam_state), P, P]),
        "lmbr_project": (c_int32, [P, P, P, c_int64, P]),
        "lmbr_beam_step": (c_int32, [P, POINTER(lmbr_beam_state), P, P, P, P, P, P]),
        "lmbr_beam_step_logits": (c_int32, [P, POINTER(lmbr_beam_state), P, c_int64, P, P, P, P, P]),
        "lmbr_score": (c_int32, [P, POINTER(lmbr_beam_state), P, P, P]),
        "lmbr_score_logits": (c_int32, [P, POINTER(lmbr_beam_state), P, c_int64, P, P]),
        "lmbr_select": (c_int32, [P, POINTER(lmbr_beam_state), P, P, P, P]),
        "lmbr_traceback": (c_int32, [P, POINTER(lmbr_beam_state), P, P, P, P, P, P]),
        "lmbr_decode": (c_int32, [P, POINTER(lmbr_beam_state), c_int32, LMBR_STATE_FN, P, P, P, P, P, P]),
        "lmbr_gather_rows": (c_int32, [P, P, P, c_int32, c_size_t, P]),
        "lmbr_table_build": (c_int32, [c_int32, c_int64, P, P, P, c_float,
                                       POINTER(lmbr_table_image), ctypes.c_char_p, c_size_t]),
        "lmbr_table_free": (None, [POINTER(lmbr_table_image)]),
        "lmbr_set_decode_options": (c_int32, [P, POINTER(lmbr_decode_options)]),
        "lmbr_set_sentence_steps": (c_int32, [P, P]),
        "lmbr_set_constraints": (c_int32, [P, P]),
        "lmbr_set_step_path": (c_int32, [P, c_int32]),
        "lmbr_projected_rows": (c_int32, [P, POINTER(c_int32), P]),
        "lmbr_set_lmbr_layout": (c_int32, [P, c_int32]),
        "lmbr_table_history_count": (c_int64, [POINTER(lmbr_table_image)]),
        "lmbr_plan_batches": (c_int32, [c_int64, P, c_int32, c_int32, P, P]),
        "lmbr_table_dense": (c_int32, [POINTER(lmbr_table_image), c_int32, c_int64, c_float, P, P, P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


# --------------------------------------------------------------------------
# marshalling helpers
# --------------------------------------------------------------------------
def _ptr(t) -> Optional[int]:
    """Device (or host) address of a tensor/array, None for None."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(rc: int, ctx=None):
    if rc != LMBR_OK:
        msg = lib().lmbr_last_error(ctx.handle if ctx is not None else None)
        raise LmbrError(rc, msg.decode() if msg else "")


class Context:
    """Owner of an lmbr_ctx* (destroyed with the object)."""

    def __init__(self, handle: int, cfg: lmbr_config):
        self.handle = handle
        self.cfg = cfg

    def close(self):
        if self.handle:
            lib().lmbr_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class BeamState:
    """Device buffers of lmbr_beam_state as torch tensors, plus the C struct."""

    def __init__(self, cfg: lmbr_config, device="cuda"):
        import torch
        M, T = cfg.B * cfg.K, cfg.T_max
        self.q = torch.empty(M, dtype=torch.float64, device=device)
        self.ctx = torch.empty(M, dtype=torch.int64, device=device)
        self.hhash = torch.empty(M, dtype=torch.int64, device=device)
        self.len = torch.empty(M, dtype=torch.int32, device=device)
        self.ranges = torch.zeros(M * 6, dtype=torch.int32, device=device)
        self.bp = torch.zeros(T * M, dtype=torch.int32, device=device)
        self.tok = torch.zeros(T * M, dtype=torch.int32, device=device)
        self.qhist = torch.zeros(T * M, dtype=torch.float64, device=device)
        # lmbr_sentence_record [B]: {double best_final, backup_score; int32 backup_step, backup_slot}
        self.sent = torch.zeros(cfg.B * 3, dtype=torch.float64, device=device)
        self.c = lmbr_beam_state(self.q.data_ptr(), self.ctx.data_ptr(), self.hhash.data_ptr(),
                                 self.len.data_ptr(), self.ranges.data_ptr(), self.bp.data_ptr(),
                                 self.tok.data_ptr(), self.qhist.data_ptr(), self.sent.data_ptr(), 0)

    @property
    def t(self) -> int:
        return self.c.t

    @t.setter
    def t(self, v: int):
        self.c.t = int(v)


def make_config(B, K, V, H, T_max, eos_id=1, lam=1.0, theta=(-0.5, 1.0, 0.8, 0.6, 0.4),
                load_factor=0.5) -> lmbr_config:
    return lmbr_config(B, K, V, H, T_max, eos_id, lam, (c_float * 5)(*theta), load_factor)


# --------------------------------------------------------------------------
# entry points (same names as the C ABI)
# --------------------------------------------------------------------------
def lmbr_workspace_bytes(cfg: lmbr_config) -> int:
    """Device bytes of a context's workspace (0 for an invalid config)."""
    return int(lib().lmbr_workspace_bytes(byref(cfg)))


def lmbr_create(cfg: lmbr_config, workspace=None) -> Context:
    """workspace: a caller-owned device buffer (e.g. a uint8 tensor) of at least
    lmbr_workspace_bytes(cfg) bytes, 256-byte aligned, kept referenced by the
    context; None lets the library allocate its own."""
    h = c_void_p()
    nbytes = 0 if workspace is None else int(workspace.numel() * workspace.element_size())
    _check(lib().lmbr_create(byref(cfg), _ptr(workspace), nbytes, byref(h)))
    ctx = Context(h.value, cfg)
    ctx._ws_ref = workspace
    return ctx


def lmbr_device_status(ctx: Context, stream=None) -> int:
    """Waits for the stream, reads and clears the device fault flag; returns its
    LMBR_DEV_* bits (0: none).  Raises nothing: the caller decides."""
    bits = c_int32(0)
    rc = lib().lmbr_device_status(ctx.handle, byref(bits), _stream(stream))
    if rc not in (LMBR_OK, LMBR_E_DEVICE):
        _check(rc, ctx)
    return int(bits.value)


def lmbr_destroy(ctx: Context):
    ctx.close()


def lmbr_device_bytes(ctx: Context) -> int:
    return int(lib().lmbr_device_bytes(ctx.handle))


def lmbr_set_projection(ctx: Context, w, layout: int = 0, bias=None, stream=None):
    _check(lib().lmbr_set_projection(ctx.handle, _ptr(w), layout, _ptr(bias), _stream(stream)), ctx)
    ctx._w_ref = (w, bias)                         # referenced by the library


def _ngrams(order, tokens, post):
    order = np.ascontiguousarray(order, dtype=np.int32)
    tokens = np.ascontiguousarray(tokens, dtype=np.int32).reshape(-1, 4)
    post = np.ascontiguousarray(post, dtype=np.float32)
    n = order.shape[0]
    if tokens.shape[0] != n or post.shape[0] != n:
        raise ValueError("order, tokens and post must have the same length")
    return n, order, tokens, post


def lmbr_load_posteriors(ctx: Context, sentence: int, order, tokens, post, stream=None):
    n, order, tokens, post = _ngrams(order, tokens, post)
    _check(lib().lmbr_load_posteriors(ctx.handle, sentence, n, _ptr(order), _ptr(tokens),
                                      _ptr(post), _stream(stream)), ctx)


def lmbr_table_bytes(ctx: Context, order, tokens, post) -> int:
    """Host-only: the device bytes of the sentence's table (0 on invalid input)."""
    n, order, tokens, post = _ngrams(order, tokens, post)
    return int(lib().lmbr_table_bytes(ctx.handle, n, _ptr(order), _ptr(tokens), _ptr(post)))


def lmbr_load_posteriors_into(ctx: Context, sentence: int, order, tokens, post, table_mem, nbytes=None,
                              stream=None):
    """lmbr_load_posteriors into caller-owned device memory (a torch tensor, kept
    alive by the caller while the context may read it)."""
    n, order, tokens, post = _ngrams(order, tokens, post)
    if nbytes is None:
        nbytes = table_mem.numel() * table_mem.element_size()
    _check(lib().lmbr_load_posteriors_into(ctx.handle, sentence, n, _ptr(order), _ptr(tokens), _ptr(post),
                                           _ptr(table_mem), int(nbytes), _stream(stream)), ctx)


def lmbr_state_init(ctx: Context, st: BeamState, seed: int, stream=None):
    _check(lib().lmbr_state_init(ctx.handle, byref(st.c), seed & (2 ** 64 - 1), _stream(stream)), ctx)


def lmbr_state_probe(ctx: Context, st: BeamState, stream=None):
    _check(lib().lmbr_state_probe(ctx.handle, byref(st.c), _stream(stream)), ctx)


def lmbr_synth_hidden(ctx: Context, st: BeamState, hidden, stream=None):
    _check(lib().lmbr_synth_hidden(ctx.handle, byref(st.c), _ptr(hidden), _stream(stream)), ctx)


def lmbr_project(ctx: Context, hidden, logits, ld: int, stream=None):
    _check(lib().lmbr_project(ctx.handle, _ptr(hidden), _ptr(logits), ld, _stream(stream)), ctx)


def lmbr_beam_step(ctx: Context, st: BeamState, hidden, eos_bias=None, parent_out=None,
                   token_out=None, score_out=None, stream=None):
    _check(lib().lmbr_beam_step(ctx.handle, byref(st.c), _ptr(hidden), _ptr(eos_bias),
                                _ptr(parent_out), _ptr(token_out), _ptr(score_out),
                                _stream(stream)), ctx)


def lmbr_beam_step_logits(ctx: Context, st: BeamState, logits, ld: int, eos_bias=None,
                          parent_out=None, token_out=None, score_out=None, stream=None):
    _check(lib().lmbr_beam_step_logits(ctx.handle, byref(st.c), _ptr(logits), ld, _ptr(eos_bias),
                                       _ptr(parent_out), _ptr(token_out), _ptr(score_out),
                                       _stream(stream)), ctx)


def lmbr_static_scratch_bytes(cfg: lmbr_config) -> int:
    return int(lib().lmbr_static_scratch_bytes(byref(cfg)))


def lmbr_beam_step_logits_static(ctx: Context, st: BeamState, logits, ld: int, eos_bias=None,
                                 parent_out=None, token_out=None, score_out=None, stream=None):
    """lmbr_beam_step_logits with its partials in the library's static scratch
    (allocates nothing; overlapping calls on one GPU race)."""
    _check(lib().lmbr_beam_step_logits_static(ctx.handle, byref(st.c), _ptr(logits), ld, _ptr(eos_bias),
                                              _ptr(parent_out), _ptr(token_out), _ptr(score_out),
                                              _stream(stream)), ctx)


def lmbr_score(ctx: Context, st: BeamState, hidden, eos_bias=None, stream=None):
    _check(lib().lmbr_score(ctx.handle, byref(st.c), _ptr(hidden), _ptr(eos_bias), _stream(stream)), ctx)


def lmbr_score_logits(ctx: Context, st: BeamState, logits, ld: int, eos_bias=None, stream=None):
    _check(lib().lmbr_score_logits(ctx.handle, byref(st.c), _ptr(logits), ld, _ptr(eos_bias),
                                   _stream(stream)), ctx)


def lmbr_select(ctx: Context, st: BeamState, parent_out=None, token_out=None, score_out=None, stream=None):
    _check(lib().lmbr_select(ctx.handle, byref(st.c), _ptr(parent_out), _ptr(token_out), _ptr(score_out),
                             _stream(stream)), ctx)


def lmbr_traceback(ctx: Context, st: BeamState, tokens_out, len_out, score_out, step_out=None,
                   slot_out=None, stream=None):
    _check(lib().lmbr_traceback(ctx.handle, byref(st.c), _ptr(tokens_out), _ptr(len_out),
                                _ptr(score_out), _ptr(step_out), _ptr(slot_out),
                                _stream(stream)), ctx)


def lmbr_decode(ctx: Context, st: BeamState, T: int, eos_bias, tokens_out, len_out, score_out,
                state_fn=None, stream=None):
    """DecodeNMT: T steps, then GetBestHypothesis into HOST arrays tokens_out
    int32 [B, T_max], len_out int32 [B], score_out float64 [B] (numpy).
    state_fn(t, st_ptr, hidden_ptr, stream_handle) -> int fills the bf16 decoder
    states [M, H] of step t on the stream (None: the built-in stand-in model)."""
    for a, dt in ((tokens_out, np.int32), (len_out, np.int32), (score_out, np.float64)):
        if not (isinstance(a, np.ndarray) and a.dtype == dt and a.flags.c_contiguous):
            raise TypeError("lmbr_decode writes host numpy arrays (int32, int32, float64)")
    B, Tm = ctx.cfg.B, ctx.cfg.T_max
    if tokens_out.size < B * Tm or len_out.size < B or score_out.size < B:
        raise ValueError("decode outputs too small")
    cb = None
    if state_fn is not None:
        def _fn(user, t, stp, hidden, strm):
            try:
                return int(state_fn(int(t), stp, hidden, strm))
            except Exception:                       # an exception must not cross the C frame
                import traceback
                traceback.print_exc()
                return LMBR_E_STATE
        cb = LMBR_STATE_FN(_fn)
    _check(lib().lmbr_decode(ctx.handle, byref(st.c), T, cb if cb is not None else LMBR_STATE_FN(),
                             None, _ptr(eos_bias), _ptr(tokens_out), _ptr(len_out), _ptr(score_out),
                             _stream(stream)), ctx)


def lmbr_set_decode_options(ctx: Context, length_norm: int = 0, finish: int = LMBR_FINISH_AT_T,
                            prune_width: Optional[float] = None):
    """prune_width None: no early pruning."""
    opt = lmbr_decode_options(int(length_norm), int(finish), 0 if prune_width is None else 1,
                              0.0 if prune_width is None else float(prune_width))
    _check(lib().lmbr_set_decode_options(ctx.handle, byref(opt)), ctx)


def lmbr_set_sentence_steps(ctx: Context, steps=None):
    """steps: host int32 [B] (copied by the call), or None for T_max everywhere."""
    if steps is None:
        _check(lib().lmbr_set_sentence_steps(ctx.handle, None), ctx)
        return
    steps = np.ascontiguousarray(steps, dtype=np.int32)
    if steps.shape != (ctx.cfg.B,):
        raise ValueError(f"steps must have shape ({ctx.cfg.B},)")
    _check(lib().lmbr_set_sentence_steps(ctx.handle, _ptr(steps)), ctx)


def lmbr_set_constraints(ctx: Context, allowed=None):
    """allowed: device uint32 bits [B, ceil(V/32)] (an int32 tensor), kept referenced; None clears."""
    _check(lib().lmbr_set_constraints(ctx.handle, _ptr(allowed)), ctx)
    ctx._allowed_ref = allowed                     # read by every later step


def lmbr_set_step_path(ctx: Context, path: int = LMBR_STEP_TWO_PASS):
    """LMBR_STEP_TWO_PASS (projection into the context's logits workspace, then the
    score pass) or LMBR_STEP_FUSED (one kernel, logits kept on chip)."""
    _check(lib().lmbr_set_step_path(ctx.handle, int(path)), ctx)


def lmbr_set_lmbr_layout(ctx: Context, layout: int = LMBR_L_SPARSE):
    """LMBR_L_SPARSE (default) or LMBR_L_DENSE for the tables loaded from now on."""
    _check(lib().lmbr_set_lmbr_layout(ctx.handle, int(layout)), ctx)


def lmbr_projected_rows(ctx: Context, stream=None) -> int:
    """Rows the last step from decoder states projected (waits for the stream)."""
    v = c_int32(0)
    _check(lib().lmbr_projected_rows(ctx.handle, byref(v), _stream(stream)), ctx)
    return int(v.value)


def lmbr_gather_rows(dst, src, rows, n: int, row_bytes: int, stream=None):
    _check(lib().lmbr_gather_rows(_ptr(dst), _ptr(src), _ptr(rows), n, row_bytes, _stream(stream)))


def lmbr_plan_batches(lengths, B: int, sorted: bool = True):
    """Host-only: (order int64 [n], batch_steps int32 [ceil(n/B)]) for a corpus
    whose sentences have decode lengths `lengths`."""
    lengths = np.ascontiguousarray(lengths, dtype=np.int32)
    n = lengths.shape[0]
    order = np.empty(n, dtype=np.int64)
    steps = np.empty(max(1, -(-n // B)), dtype=np.int32)
    rc = lib().lmbr_plan_batches(n, _ptr(lengths), int(B), int(bool(sorted)), _ptr(order), _ptr(steps))
    if rc != LMBR_OK:
        raise LmbrError(rc, "lmbr_plan_batches: bad arguments")
    return order, steps[:-(-n // B)]


def lmbr_table_build(V: int, order, tokens, post, load_factor: float = 0.5, dense_ld=None,
                     dense_lambda=1.0, dense_theta=(-0.5, 1.0, 0.8, 0.6, 0.4)) -> dict:
    """Host-only: the table image lmbr_load_posteriors would upload, as numpy arrays;
    with dense_ld, also its dense rows (lmbr_table_dense) under "dense"."""
    order = np.ascontiguousarray(order, dtype=np.int32)
    tokens = np.ascontiguousarray(tokens, dtype=np.int32).reshape(-1, 4)
    post = np.ascontiguousarray(post, dtype=np.float32)
    img = lmbr_table_image()
    err = ctypes.create_string_buffer(256)
    rc = lib().lmbr_table_build(V, order.shape[0], _ptr(order), _ptr(tokens), _ptr(post),
                                load_factor, byref(img), err, 256)
    if rc != LMBR_OK:
        raise LmbrError(rc, err.value.decode())
    try:
        ns, ne = img.n_slots, img.n_entries
        dense = None
        if dense_ld is not None:
            nrows = int(lib().lmbr_table_history_count(byref(img))) + 1
            rows = np.zeros((nrows, dense_ld), dtype=np.float32)
            slot_row = np.zeros(ns, dtype=np.uint32)
            th = np.ascontiguousarray(dense_theta, dtype=np.float32)
            rc = lib().lmbr_table_dense(byref(img), V, dense_ld, float(dense_lambda), _ptr(th), _ptr(rows),
                                        _ptr(slot_row))
            if rc != LMBR_OK:
                raise LmbrError(rc, "lmbr_table_dense")
            dense = {"rows": rows, "slot_row": slot_row}
        out = {
            "slot_key": np.ctypeslib.as_array(img.slot_key, (ns,)).copy(),
            "slot_off": np.ctypeslib.as_array(img.slot_off, (ns,)).copy(),
            "slot_cnt": np.ctypeslib.as_array(img.slot_cnt, (ns,)).copy(),
            "entry_tok": np.ctypeslib.as_array(img.entry_tok, (max(ne, 1),))[:ne].copy(),
            "entry_post": np.ctypeslib.as_array(img.entry_post, (max(ne, 1),))[:ne].copy(),
            "uni_off": int(img.uni_off), "uni_cnt": int(img.uni_cnt),
        }
        if dense is not None:
            out["dense"] = dense
    finally:
        lib().lmbr_table_free(byref(img))
    return out
