"""ctypes binding of libpard.so (include/pard.h): argument marshalling only.

Every computation runs in the HIP library; this module converts Python /
numpy / torch arguments to the C ABI and raises ``PardError`` on a non-OK
status.  PyTorch is used only to allocate the device arena and to name the
HIP stream.  Importing fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpard.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2504_18583_amd.csrc.build` "
                      "(or __graft_entry__.build())")

lib = C.CDLL(LIB_PATH)

PARD_OK, PARD_ERR_ARG, PARD_ERR_STATE, PARD_ERR_CAPACITY = 0, -1, -2, -3
PARD_ERR_NOMEM, PARD_ERR_DEVICE, PARD_ERR_UNSUPPORTED, PARD_ERR_RANGE = -4, -5, -6, -7
PARD_F32, PARD_BF16 = 0, 1
PARD_TARGET, PARD_DRAFT = 0, 1
PARD_MODE_PARALLEL, PARD_MODE_VANILLA = 0, 1
OP_EMBED, OP_QKV, OP_ATTN, OP_O, OP_GATEUP, OP_DOWN, OP_LM, OP_TAIL = range(8)


class pard_model_spec(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn_dim", C.c_int32),
                ("vocab", C.c_int32), ("rms_eps", C.c_float), ("rope_theta", C.c_float),
                ("init_std", C.c_float), ("qkv_bias", C.c_int32), ("tied_embeddings", C.c_int32),
                ("dtype", C.c_int32), ("weight_stream", C.c_uint32), ("seed", C.c_uint64),
                ("rope_factor", C.c_float), ("rope_low_freq_factor", C.c_float),
                ("rope_high_freq_factor", C.c_float), ("rope_original_max_pos", C.c_int32)]


class pard_stats(C.Structure):
    _fields_ = [("steps", C.c_int64), ("tokens", C.c_int64), ("elapsed_ms", C.c_double),
                ("draft_ms", C.c_double), ("verify_ms", C.c_double), ("accept_ms", C.c_double),
                ("step_ms_p50", C.c_double), ("step_ms_p90", C.c_double),
                ("accept_hist", C.c_int64 * 33)]


_I32P = C.POINTER(C.c_int32)
_SPECP = C.POINTER(pard_model_spec)
_CTX = C.c_void_p

_sig = {
    "pard_arena_bytes": (C.c_size_t, [_SPECP, _SPECP, C.c_int32, C.c_int32, C.c_int32]),
    "pard_model_load": (C.c_int, [_SPECP, _SPECP, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                  C.c_void_p, C.c_size_t, C.c_void_p, C.POINTER(_CTX)]),
    "pard_prefill": (C.c_int, [_CTX, C.c_int32, _I32P, C.c_int32, _I32P]),
    "pard_draft": (C.c_int, [_CTX, C.c_int32, _I32P, C.c_int32, C.c_int32, _I32P]),
    "pard_verify": (C.c_int, [_CTX, C.c_int32, _I32P, C.c_int32, _I32P, _I32P]),
    "pard_kv_truncate": (C.c_int, [_CTX, C.c_int32, C.c_int32, C.c_int32]),
    "pard_kv_len": (C.c_int, [_CTX, C.c_int32, C.c_int32, _I32P]),
    "pard_generate": (C.c_int, [_CTX, C.c_int32, _I32P, C.c_int32, C.c_int32, C.c_int32, _I32P,
                                C.POINTER(pard_stats)]),
    "pard_generate_ex": (C.c_int, [_CTX, C.c_int32, _I32P, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                   _I32P, C.POINTER(pard_stats)]),
    "pard_set_sampling": (C.c_int, [_CTX, C.c_float, C.c_uint64]),
    "pard_cod_capacity": (C.c_int64, [C.c_int32, C.c_int32, C.c_double, C.c_double]),
    "pard_cod_layout": (C.c_int64, [C.POINTER(C.c_int64), C.c_int32, C.c_int32, C.c_double, C.c_double,
                                    C.POINTER(C.c_int64)]),
    "pard_cod_workspace_bytes": (C.c_size_t, [C.c_int32]),
    "pard_cod_build": (C.c_int, [C.c_void_p, C.POINTER(C.c_int64), C.c_int32, C.c_int32, C.c_double,
                                 C.c_double, C.c_int32, C.c_uint64, C.POINTER(C.c_int64), C.c_void_p,
                                 C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                 C.c_void_p, C.c_size_t, C.POINTER(C.c_float), C.c_void_p]),
    "pard_cod_build_noalloc": (C.c_int, [C.c_void_p, C.POINTER(C.c_int64), C.c_int32, C.c_int32, C.c_double,
                                         C.c_double, C.c_int32, C.c_uint64, C.POINTER(C.c_int64), C.c_void_p,
                                         C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]),
    "pard_read_logits": (C.c_int, [_CTX, C.c_int32, C.c_int32, C.POINTER(C.c_float), C.c_int32,
                                   C.c_int32]),
    "pard_read_weight": (C.c_int, [_CTX, C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                   C.POINTER(C.c_float)]),
    "pard_timer_enable": (C.c_int, [_CTX, C.c_int32, C.c_int32]),
    "pard_timer_read": (C.c_int, [_CTX, _I32P, C.POINTER(C.c_double)]),
    "pard_last_error": (C.c_char_p, [_CTX]),
    "pard_status_string": (C.c_char_p, [C.c_int]),
    "pard_free": (None, [_CTX]),
}
for _name, (_res, _args) in _sig.items():
    _f = getattr(lib, _name)
    _f.restype = _res
    _f.argtypes = _args

EXPORTED = tuple(_sig)


class PardError(RuntimeError):
    def __init__(self, status: int, message: str):
        self.status = status
        name = lib.pard_status_string(status).decode()
        super().__init__(f"{name}: {message}")


def spec_from(s) -> pard_model_spec:
    """C spec from a ``pard_inputs.ModelSpec`` (the library always stores bf16)."""
    return pard_model_spec(
        n_layers=s.n_layers, d_model=s.d_model, n_heads=s.n_heads, n_kv_heads=s.n_kv_heads,
        head_dim=s.head_dim, ffn_dim=s.ffn_dim, vocab=s.vocab, rms_eps=s.rms_eps,
        rope_theta=s.rope_theta, init_std=s.init_std, qkv_bias=int(s.qkv_bias),
        tied_embeddings=int(s.tied), dtype=PARD_BF16, weight_stream=s.stream, seed=s.seed,
        **_rope_fields(s))


def _rope_fields(s) -> dict:
    if s.rope_scaling is None:
        return {}
    factor, low, high, orig = s.rope_scaling
    return dict(rope_factor=float(factor), rope_low_freq_factor=float(low), rope_high_freq_factor=float(high),
                rope_original_max_pos=int(orig))


def _i32(a) -> Tuple[np.ndarray, object]:
    arr = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return arr, arr.ctypes.data_as(_I32P)


# ---- the C calls, same names --------------------------------------------------

def pard_arena_bytes(target: pard_model_spec, draft: pard_model_spec, max_batch: int,
                     max_ctx: int, max_k: int) -> int:
    return int(lib.pard_arena_bytes(C.byref(target), C.byref(draft), max_batch, max_ctx, max_k))


def pard_model_load(target, draft, mask_id, max_batch, max_ctx, max_k, dev_arena_ptr: int,
                    arena_bytes: int, hip_stream: Optional[int]) -> int:
    ctx = _CTX()
    st = lib.pard_model_load(C.byref(target), C.byref(draft), mask_id, max_batch, max_ctx, max_k,
                             C.c_void_p(dev_arena_ptr), arena_bytes, C.c_void_p(hip_stream or 0),
                             C.byref(ctx))
    if st != PARD_OK:
        raise PardError(st, "pard_model_load failed")
    return ctx.value


def cod_capacity(n_tokens: int, k: int, r: float, r_min: float) -> int:
    return int(lib.pard_cod_capacity(int(n_tokens), int(k), float(r), float(r_min)))


def cod_build(tokens, tok_offsets: Sequence[int], k: int, r: float, r_min: float, mask_id: int, seed: int,
              stream=None, timing: bool = False):
    """COD training-data processing on the device (pard_cod_build).

    tokens: 1-D int32 device tensor of the samples back to back; tok_offsets:
    host offsets (n_samples + 1).  Returns (out_offsets, dict of the five int32
    device tensors ids/labels/pos/section/column, out_len device tensor), and
    the kernel's device milliseconds when timing is set."""
    import torch
    offs = np.ascontiguousarray(np.asarray(tok_offsets, np.int64))
    n = len(offs) - 1
    out_offs = np.zeros(max(n, 0) + 1, np.int64)
    total = lib.pard_cod_layout(offs.ctypes.data_as(C.POINTER(C.c_int64)), n, k, float(r), float(r_min),
                                out_offs.ctypes.data_as(C.POINTER(C.c_int64))) if n >= 1 else -1
    if total < 0:
        raise PardError(PARD_ERR_ARG, "cod_build: empty batch, bad parameters or a sample outside the lengths")
    dev = tokens.device
    out = {name: torch.empty(total, dtype=torch.int32, device=dev)
           for name in ("ids", "labels", "pos", "section", "column")}
    out_len = torch.empty(n, dtype=torch.int32, device=dev)
    ws_bytes = int(lib.pard_cod_workspace_bytes(n))
    ws = torch.empty(ws_bytes + 256, dtype=torch.uint8, device=dev)
    ws_ptr = ws.data_ptr() + (-ws.data_ptr()) % 256
    ms = C.c_float(0.0)
    st = stream if stream is not None else torch.cuda.current_stream(dev).cuda_stream
    rc = lib.pard_cod_build(C.c_void_p(tokens.data_ptr()), offs.ctypes.data_as(C.POINTER(C.c_int64)), n, k,
                            float(r), float(r_min), mask_id, int(seed) & ((1 << 64) - 1),
                            out_offs.ctypes.data_as(C.POINTER(C.c_int64)),
                            *[C.c_void_p(out[name].data_ptr()) for name in ("ids", "labels", "pos", "section",
                                                                            "column")],
                            C.c_void_p(out_len.data_ptr()), C.c_void_p(ws_ptr), ws_bytes,
                            C.byref(ms) if timing else None, C.c_void_p(st))
    if rc != PARD_OK:
        raise PardError(rc, "pard_cod_build failed")
    return (out_offs, out, out_len, ms.value) if timing else (out_offs, out, out_len)


PARD_COD_NOALLOC_MAX_SAMPLES = 65535


def cod_build_noalloc(tokens, tok_offsets: Sequence[int], k: int, r: float, r_min: float, mask_id: int, seed: int,
                      stream=None):
    """pard_cod_build_noalloc: as cod_build, with the offsets staged in the
    library's fixed device scratch instead of a workspace.  The output tensors
    are allocated here (by the caller of the C function)."""
    import torch
    offs = np.ascontiguousarray(np.asarray(tok_offsets, np.int64))
    n = len(offs) - 1
    out_offs = np.zeros(max(n, 0) + 1, np.int64)
    total = lib.pard_cod_layout(offs.ctypes.data_as(C.POINTER(C.c_int64)), n, k, float(r), float(r_min),
                                out_offs.ctypes.data_as(C.POINTER(C.c_int64))) if n >= 1 else -1
    if total < 0:
        raise PardError(PARD_ERR_ARG, "cod_build_noalloc: empty batch, bad parameters or a sample outside the lengths")
    dev = tokens.device
    out = {name: torch.empty(total, dtype=torch.int32, device=dev)
           for name in ("ids", "labels", "pos", "section", "column")}
    out_len = torch.empty(n, dtype=torch.int32, device=dev)
    st = stream if stream is not None else torch.cuda.current_stream(dev).cuda_stream
    rc = lib.pard_cod_build_noalloc(C.c_void_p(tokens.data_ptr()), offs.ctypes.data_as(C.POINTER(C.c_int64)), n, k,
                                    float(r), float(r_min), mask_id, int(seed) & ((1 << 64) - 1),
                                    out_offs.ctypes.data_as(C.POINTER(C.c_int64)),
                                    *[C.c_void_p(out[name].data_ptr()) for name in ("ids", "labels", "pos", "section",
                                                                                    "column")],
                                    C.c_void_p(out_len.data_ptr()), C.c_void_p(st))
    if rc != PARD_OK:
        raise PardError(rc, "pard_cod_build_noalloc failed")
    return out_offs, out, out_len


class Engine:
    """A loaded target/draft pair: owns the torch arena and the context."""

    def __init__(self, target_spec, draft_spec, mask_id: int, max_ctx: int, max_k: int,
                 max_batch: int = 1, device: str = "cuda:0", stream=None):
        import torch
        self.target_spec, self.draft_spec = target_spec, draft_spec
        self.vocab = target_spec.vocab
        self.mask_id = mask_id
        self._t, self._d = spec_from(target_spec), spec_from(draft_spec)
        nbytes = pard_arena_bytes(self._t, self._d, max_batch, max_ctx, max_k)
        if nbytes == 0:
            raise PardError(PARD_ERR_ARG, "invalid specs or capacities")
        self.device = torch.device(device)
        self.arena = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
        base = self.arena.data_ptr()
        base += (-base) % 256
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        self.ctx = pard_model_load(self._t, self._d, mask_id, max_batch, max_ctx, max_k, base,
                                   nbytes, self.stream.cuda_stream)
        self.max_ctx, self.max_k, self.max_batch = max_ctx, max_k, max_batch

    def close(self) -> None:
        if getattr(self, "ctx", None):
            lib.pard_free(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _check(self, st: int, what: str) -> None:
        if st != PARD_OK:
            raise PardError(st, f"{what}: {lib.pard_last_error(self.ctx).decode()}")

    def prefill(self, prompt: Sequence[int], seq: int = 0) -> int:
        arr, ptr = _i32(prompt)
        first = C.c_int32()
        self._check(lib.pard_prefill(self.ctx, seq, ptr, len(arr), C.byref(first)), "pard_prefill")
        return first.value

    def draft(self, prefix: Sequence[int], k: int, seq: int = 0) -> list:
        arr, ptr = _i32(prefix)
        out = np.zeros(max(k, 1), np.int32)
        self._check(lib.pard_draft(self.ctx, seq, ptr, len(arr), k, out.ctypes.data_as(_I32P)),
                    "pard_draft")
        return [int(x) for x in out[:k]]

    def verify(self, cand: Sequence[int], seq: int = 0) -> Tuple[int, int]:
        arr, ptr = _i32(list(cand) if len(cand) else [0])
        a, bonus = C.c_int32(), C.c_int32()
        self._check(lib.pard_verify(self.ctx, seq, ptr, len(cand), C.byref(a), C.byref(bonus)),
                    "pard_verify")
        return a.value, bonus.value

    def set_sampling(self, temperature: float, seed: int = 0) -> None:
        """Speculative sampling at temperature T > 0 for later calls; 0 = greedy."""
        self._check(lib.pard_set_sampling(self.ctx, float(temperature), int(seed) & ((1 << 64) - 1)),
                    "pard_set_sampling")

    def kv_len(self, which: int, seq: int = 0) -> int:
        n = C.c_int32()
        self._check(lib.pard_kv_len(self.ctx, seq, which, C.byref(n)), "pard_kv_len")
        return n.value

    def kv_truncate(self, which: int, new_len: int, seq: int = 0) -> None:
        self._check(lib.pard_kv_truncate(self.ctx, seq, which, new_len), "pard_kv_truncate")

    def generate(self, k: int, n_tokens: int, max_steps: int = 0, seq: int = 0,
                 mode: int = PARD_MODE_PARALLEL):
        out = np.zeros(n_tokens, np.int32)
        stats = pard_stats()
        seqs, sptr = _i32([seq])
        self._check(lib.pard_generate_ex(self.ctx, 1, sptr, k, mode, n_tokens, max_steps,
                                         out.ctypes.data_as(_I32P), C.byref(stats)), "pard_generate_ex")
        return out[:stats.tokens].tolist(), stats

    def generate_batch(self, seqs: Sequence[int], k: int, n_tokens: int, max_steps: int = 0,
                       mode: int = PARD_MODE_PARALLEL):
        """Fused loop over several slots at once (batched passes).  Returns one
        token list per slot (the pending token first) and the summed stats."""
        before = [self.kv_len(PARD_TARGET, seq=s) for s in seqs]
        out = np.zeros((len(seqs), n_tokens), np.int32)
        stats = pard_stats()
        arr, sptr = _i32(list(seqs))
        self._check(lib.pard_generate_ex(self.ctx, len(seqs), sptr, k, mode, n_tokens, max_steps,
                                         out.ctypes.data_as(_I32P), C.byref(stats)), "pard_generate_ex")
        res = []
        for i, s in enumerate(seqs):
            n = min(n_tokens, 1 + self.kv_len(PARD_TARGET, seq=s) - before[i])
            res.append(out[i, :n].tolist())
        return res, stats

    def read_logits(self, which: int, rows: int, seq: int = 0) -> np.ndarray:
        out = np.zeros((rows, self.vocab), np.float32)
        self._check(lib.pard_read_logits(self.ctx, which, seq,
                                         out.ctypes.data_as(C.POINTER(C.c_float)), rows,
                                         self.vocab), "pard_read_logits")
        return out

    def read_weight(self, which: int, tensor: int, row: int, col0: int, n: int) -> np.ndarray:
        out = np.zeros(n, np.float32)
        self._check(lib.pard_read_weight(self.ctx, which, tensor, row, col0, n,
                                         out.ctypes.data_as(C.POINTER(C.c_float))),
                    "pard_read_weight")
        return out

    def timer_enable(self, kernel_class: int, max_launches: int) -> None:
        self._check(lib.pard_timer_enable(self.ctx, kernel_class, max_launches), "pard_timer_enable")

    def timer_read(self) -> Tuple[int, float]:
        n, ms = C.c_int32(), C.c_double()
        self._check(lib.pard_timer_read(self.ctx, C.byref(n), C.byref(ms)), "pard_timer_read")
        return n.value, ms.value
