"""Python binding of libdvs.so (ctypes; argument marshalling only).

Every entry point has the name of its C function and forwards device
pointers of torch tensors plus sizes.  All computation happens in the HIP
kernels; there is no fallback of any kind: if the library is missing or a
call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libdvs.so")

DVS_F32 = 0
DVS_BF16 = 1
ERR_POOL_EXHAUSTED = 1
ERR_MAX_PAGES = 2
ERR_NONFINITE = 4
ERR_BAD_PAGE = 8

_lib = None

# Model-level calls default to aligned 256-key attention chunks: a row's
# arithmetic then does not depend on the call's other rows, so the
# self-speculative stream equals greedy AR bit for bit.  chunk_keys = 0 (the
# balanced split) fills the chip better but drops that guarantee.
MODEL_CHUNK_KEYS = 256

_c_int, _c_ptr, _c_f32, _c_size = ctypes.c_int32, ctypes.c_void_p, ctypes.c_float, ctypes.c_size_t

_SIGS = {
    "dvs_version": ([], _c_int),
    "dvs_last_error": ([], ctypes.c_char_p),
    "dvs_attn_workspace_bytes": ([_c_int] * 9, _c_size),
    "attn_hybrid_block": ([_c_ptr] * 7 + [_c_int] * 8 + [_c_f32, _c_int, _c_int, _c_ptr, _c_ptr,
                                                          _c_ptr, _c_size, _c_ptr], _c_int),
    "attn_hybrid_block_noalloc": ([_c_ptr] * 7 + [_c_int] * 8 + [_c_f32, _c_int, _c_int, _c_ptr,
                                                                  _c_ptr, _c_ptr], _c_int),
    "argmax_accept": ([_c_ptr, _c_int, _c_int, _c_int, _c_int, _c_int, _c_ptr, _c_int, _c_ptr,
                       _c_ptr, _c_ptr, _c_ptr], _c_int),
    "kv_commit": ([_c_int, _c_int, _c_int, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_int, _c_ptr,
                   _c_ptr, _c_int, _c_ptr, _c_ptr, _c_int, _c_ptr, _c_ptr, _c_int, _c_int, _c_ptr,
                   _c_ptr, _c_ptr], _c_int),
    "accept_commit": ([_c_int, _c_int, _c_int, _c_int, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_int,
                       _c_ptr, _c_ptr, _c_int, _c_ptr, _c_ptr, _c_int, _c_ptr, _c_ptr, _c_int,
                       _c_int, _c_ptr, _c_ptr, _c_ptr], _c_int),
    "kv_commit_round": ([_c_int, _c_int, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_int,
                         _c_ptr, _c_ptr, _c_int, _c_ptr, _c_ptr, _c_int, _c_ptr, _c_ptr, _c_int,
                         _c_int, _c_ptr, _c_ptr, _c_ptr], _c_int),
    "top1_confidence": ([_c_ptr, _c_int, _c_int, _c_int, _c_ptr, _c_ptr, _c_ptr, _c_ptr], _c_int),
    "kv_commit_block": ([_c_int, _c_int, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_int, _c_ptr, _c_ptr,
                         _c_int, _c_ptr, _c_ptr, _c_ptr, _c_int, _c_int, _c_ptr, _c_ptr, _c_ptr],
                        _c_int),
}

class DvsLayer(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("wq", "wk", "wv", "wo", "g_attn", "g_mlp", "w_gate",
                                                "w_up", "w_down", "k_pool", "v_pool")]


class DvsModel(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("n_layers", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("hidden", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("ffn", ctypes.c_int32), ("rope_theta", ctypes.c_float),
                ("rms_eps", ctypes.c_float), ("embed", ctypes.c_void_p),
                ("g_final", ctypes.c_void_p), ("lm_head", ctypes.c_void_p),
                ("layers", ctypes.POINTER(DvsLayer))]


class DvsState(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("S", "max_pages", "num_pool_pages", "draft_width",
                                              "max_new", "eos_id")] + \
               [(n, ctypes.c_void_p) for n in ("kv_len", "page_table", "num_pages", "free_stack",
                                               "free_top", "boundary", "draft", "out_tokens",
                                               "out_count", "finished", "err_word")]


_SIGS["dvs_step_workspace_bytes"] = ([ctypes.POINTER(DvsModel), _c_int, _c_int, _c_int, _c_int,
                                      _c_int], _c_size)
_SIGS["draft_verify_step"] = ([ctypes.POINTER(DvsModel), ctypes.POINTER(DvsState), _c_int, _c_int,
                               _c_int, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_size, _c_ptr], _c_int)

_SIGS["multidraft_step"] = ([ctypes.POINTER(DvsModel), ctypes.POINTER(DvsState), _c_int, _c_int,
                             _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_size, _c_ptr], _c_int)
_SIGS["attn_hybrid_block_grouped"] = ([_c_ptr] * 7 + [_c_int] * 9 + [_c_f32, _c_int, _c_int,
                                                                     _c_ptr, _c_ptr, _c_ptr,
                                                                     _c_size, _c_ptr], _c_int)
_SIGS["literal_round"] = ([ctypes.POINTER(DvsModel), ctypes.POINTER(DvsState), _c_int, _c_int,
                           _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_size, _c_ptr], _c_int)

_SIGS["dvs_diffusion_workspace_bytes"] = ([ctypes.POINTER(DvsModel), _c_int, _c_int, _c_int,
                                           _c_int], _c_size)
_SIGS["diffusion_denoise"] = ([ctypes.POINTER(DvsModel), ctypes.POINTER(DvsState), _c_int, _c_f32,
                               _c_ptr, _c_ptr, _c_int, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_size,
                               _c_ptr], _c_int)
_SIGS["diffusion_block"] = ([ctypes.POINTER(DvsModel), ctypes.POINTER(DvsState), _c_int, _c_f32,
                             _c_ptr, _c_int, ctypes.POINTER(ctypes.c_int32), _c_ptr, _c_size,
                             _c_ptr], _c_int)

_SIGS["literal_round_refined"] = ([ctypes.POINTER(DvsModel), ctypes.POINTER(DvsState), _c_int,
                                   _c_f32, _c_int, _c_ptr, _c_ptr, _c_ptr,
                                   ctypes.POINTER(ctypes.c_int32), _c_ptr, _c_size, _c_ptr], _c_int)

_SIGS["dvs_sampled_round_workspace_bytes"] = ([ctypes.POINTER(DvsModel), _c_int, _c_int, _c_int,
                                               _c_int], _c_size)
_SIGS["literal_round_sampled"] = ([ctypes.POINTER(DvsModel), ctypes.POINTER(DvsState), _c_int,
                                   _c_f32, _c_ptr, _c_int, _c_ptr, _c_ptr, _c_ptr, _c_size,
                                   _c_ptr], _c_int)

_SIGS["dvs_prefill_workspace_bytes"] = ([ctypes.POINTER(DvsModel), _c_int, _c_int, _c_int, _c_int,
                                         _c_int], _c_size)
_SIGS["dvs_prefill"] = ([ctypes.POINTER(DvsModel), ctypes.POINTER(DvsState), _c_int, _c_int, _c_ptr,
                         _c_ptr, _c_int, _c_ptr, _c_ptr, _c_size, _c_ptr], _c_int)

EXPORTED = tuple(_SIGS)


class DvsError(RuntimeError):
    pass


def lib():
    """Load libdvs.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise DvsError(f"{LIB_PATH} not found: build it with "
                           "`python -m paper_2609_26638_amd.build` (no fallback exists)")
        l = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            f = getattr(l, name)
            f.argtypes = args
            f.restype = res
        _lib = l
    return _lib


def _check(rc: int, what: str):
    if rc != 0:
        msg = lib().dvs_last_error().decode(errors="replace")
        raise DvsError(f"{what} failed ({rc}): {msg}")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dev(t, dtype, name, ndim=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise DvsError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise DvsError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise DvsError(f"{name} must be contiguous")
    if ndim is not None and t.dim() != ndim:
        raise DvsError(f"{name} must have {ndim} dims, got {tuple(t.shape)}")
    return t


def _dtype_code(t):
    if t.dtype == torch.float32:
        return DVS_F32
    if t.dtype == torch.bfloat16:
        return DVS_BF16
    raise DvsError(f"unsupported dtype {t.dtype}")


# ---------------------------------------------------------------------------
# attention
# ---------------------------------------------------------------------------

def attn_workspace_bytes(S, n_causal, n_mask, Hq, Hkv, D, max_pages, chunk_keys=0,
                         dtype=DVS_BF16) -> int:
    return int(lib().dvs_attn_workspace_bytes(S, n_causal, n_mask, Hq, Hkv, D, max_pages,
                                              chunk_keys, dtype))


class Workspace:
    """Zero-initialised device scratch.  attn_hybrid_block keeps split-merge
    counters at its start, which must be zero when a call shape first uses
    it and which every call leaves zero; `shape` remembers the last shape so
    a change of shape clears the buffer again."""

    def __init__(self, nbytes: int, device="cuda"):
        self.buf = torch.zeros(max(int(nbytes), 256), dtype=torch.uint8, device=device)
        self.shape = None

    def prepare(self, nbytes: int, shape):
        self.ensure(nbytes)
        if shape != self.shape:
            self.buf.zero_()
            self.shape = shape
        return self

    @property
    def nbytes(self):
        return self.buf.numel()

    def ensure(self, nbytes: int):
        if nbytes > self.nbytes:
            self.buf = torch.zeros(int(nbytes), dtype=torch.uint8, device=self.buf.device)
            self.shape = None
        return self


def _attn_args(q, k_new, v_new, k_pool, v_pool, page_table, kv_len, n_causal, n_mask, out, err):
    """Shape and dtype checks shared by the two attention entry points."""
    dt = q.dtype
    _dev(q, dt, "q", 4)
    S, R, Hq, D = q.shape
    _dev(k_new, dt, "k_new", 4)
    _dev(v_new, dt, "v_new", 4)
    Hkv = k_new.shape[2]
    if tuple(k_new.shape) != (S, R, Hkv, D) or tuple(v_new.shape) != (S, R, Hkv, D):
        raise DvsError("k_new / v_new must be [S, R, Hkv, D]")
    _dev(k_pool, dt, "k_pool", 4)
    _dev(v_pool, dt, "v_pool", 4)
    P = k_pool.shape[0]
    if tuple(k_pool.shape) != (P, Hkv, 16, D) or tuple(v_pool.shape) != (P, Hkv, D, 16):
        raise DvsError("pools must be k [P,Hkv,16,D] and v [P,Hkv,D,16]")
    _dev(page_table, torch.int32, "page_table", 2)
    _dev(kv_len, torch.int32, "kv_len", 1)
    if page_table.shape[0] != S or kv_len.shape[0] != S:
        raise DvsError("page_table / kv_len must have S rows")
    if R != n_causal + n_mask:
        raise DvsError("R must equal n_causal + n_mask")
    if out is None:
        out = torch.empty_like(q)
    _dev(out, dt, "out", 4)
    if err is not None:
        _dev(err, torch.int32, "err", 1)
    return S, R, Hq, Hkv, D, P, page_table.shape[1], out


def attn_hybrid_block_noalloc(q, k_new, v_new, k_pool, v_pool, page_table, kv_len, n_causal: int,
                              n_mask: int, softmax_scale: float, out=None, err=None,
                              chunk_keys: int = 0, stream=None):
    """attn_hybrid_block with the library's own scratch array as workspace (the C
    call allocates nothing; ``out`` is allocated here when not given)."""
    S, R, Hq, Hkv, D, P, max_pages, out = _attn_args(q, k_new, v_new, k_pool, v_pool, page_table,
                                                     kv_len, n_causal, n_mask, out, err)
    rc = lib().attn_hybrid_block_noalloc(_ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_pool),
                                         _ptr(v_pool), _ptr(page_table), _ptr(kv_len), S, n_causal,
                                         n_mask, Hq, Hkv, D, max_pages, P, float(softmax_scale),
                                         _dtype_code(q), int(chunk_keys), _ptr(out), _ptr(err),
                                         _stream(stream))
    _check(rc, "attn_hybrid_block_noalloc")
    return out


def attn_hybrid_block(q, k_new, v_new, k_pool, v_pool, page_table, kv_len, n_causal: int,
                      n_mask: int, softmax_scale: float, out=None, err=None, workspace=None,
                      chunk_keys: int = 0, stream=None):
    """q [S,R,Hq,D], k_new/v_new [S,R,Hkv,D], k_pool [P,Hkv,16,D],
    v_pool [P,Hkv,D,16] (updated), page_table [S,max_pages] int32, kv_len [S] int32."""
    dt = q.dtype
    _dev(q, dt, "q", 4)
    S, R, Hq, D = q.shape
    _dev(k_new, dt, "k_new", 4)
    _dev(v_new, dt, "v_new", 4)
    Hkv = k_new.shape[2]
    if tuple(k_new.shape) != (S, R, Hkv, D) or tuple(v_new.shape) != (S, R, Hkv, D):
        raise DvsError("k_new / v_new must be [S, R, Hkv, D]")
    _dev(k_pool, dt, "k_pool", 4)
    _dev(v_pool, dt, "v_pool", 4)
    P = k_pool.shape[0]
    if tuple(k_pool.shape) != (P, Hkv, 16, D) or tuple(v_pool.shape) != (P, Hkv, D, 16):
        raise DvsError("pools must be k [P,Hkv,16,D] and v [P,Hkv,D,16]")
    _dev(page_table, torch.int32, "page_table", 2)
    _dev(kv_len, torch.int32, "kv_len", 1)
    if page_table.shape[0] != S or kv_len.shape[0] != S:
        raise DvsError("page_table / kv_len must have S rows")
    if R != n_causal + n_mask:
        raise DvsError("R must equal n_causal + n_mask")
    max_pages = page_table.shape[1]
    if out is None:
        out = torch.empty_like(q)
    _dev(out, dt, "out", 4)
    if err is not None:
        _dev(err, torch.int32, "err", 1)
    code = _dtype_code(q)
    need = attn_workspace_bytes(S, n_causal, n_mask, Hq, Hkv, D, max_pages, chunk_keys, code)
    if workspace is None:
        workspace = Workspace(need, device=q.device)
    workspace.prepare(need, ("attn", S, R, Hq, Hkv, D, max_pages, int(chunk_keys), code))
    rc = lib().attn_hybrid_block(_ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_pool), _ptr(v_pool),
                                 _ptr(page_table), _ptr(kv_len), S, n_causal, n_mask, Hq, Hkv, D,
                                 max_pages, P, float(softmax_scale), code, int(chunk_keys),
                                 _ptr(out), _ptr(err), _ptr(workspace.buf), workspace.nbytes,
                                 _stream(stream))
    _check(rc, "attn_hybrid_block")
    return out


# ---------------------------------------------------------------------------
# argmax + acceptance
# ---------------------------------------------------------------------------

def argmax_accept(logits, n_causal: int, draft, argmax_out=None, accept_len=None, err=None,
                  stream=None, accept: bool = True):
    """logits [S,R,V] (f32/bf16), draft [S,W] int32 -> (argmax [S,R], accept_len [S]).
    accept=False: top-1 only (accept_len is None), for accept_commit."""
    _dev(logits, logits.dtype, "logits", 3)
    S, R, V = logits.shape
    _dev(draft, torch.int32, "draft", 2)
    if argmax_out is None:
        argmax_out = torch.empty((S, R), dtype=torch.int32, device=logits.device)
    if accept and accept_len is None:
        accept_len = torch.empty((S,), dtype=torch.int32, device=logits.device)
    if not accept:
        accept_len = None
    _dev(argmax_out, torch.int32, "argmax_out", 2)
    if accept_len is not None:
        _dev(accept_len, torch.int32, "accept_len", 1)
    if err is not None:
        _dev(err, torch.int32, "err", 1)
    rc = lib().argmax_accept(_ptr(logits), _dtype_code(logits), S, R, V, n_causal, _ptr(draft),
                             draft.shape[1], _ptr(argmax_out), _ptr(accept_len), _ptr(err),
                             _stream(stream))
    _check(rc, "argmax_accept")
    return argmax_out, accept_len


def top1_confidence(logits, argmax_out=None, conf_out=None, err=None, stream=None):
    """logits [..., V] (f32/bf16) -> (top-1 [...] int32, softmax probability of it [...] f32)."""
    if logits.device.type != "cuda" or not logits.is_contiguous():
        raise DvsError("logits must be a contiguous device tensor")
    lead, V = logits.shape[:-1], logits.shape[-1]
    rows = int(np.prod(lead)) if len(lead) else 1
    if argmax_out is None:
        argmax_out = torch.empty(lead, dtype=torch.int32, device=logits.device)
    if conf_out is None:
        conf_out = torch.empty(lead, dtype=torch.float32, device=logits.device)
    _dev(argmax_out, torch.int32, "argmax_out")
    _dev(conf_out, torch.float32, "conf_out")
    if argmax_out.numel() != rows or conf_out.numel() != rows:
        raise DvsError("argmax_out / conf_out must have one entry per row")
    if err is not None:
        _dev(err, torch.int32, "err", 1)
    rc = lib().top1_confidence(_ptr(logits), _dtype_code(logits), rows, V, _ptr(argmax_out),
                               _ptr(conf_out), _ptr(err), _stream(stream))
    _check(rc, "top1_confidence")
    return argmax_out, conf_out


# ---------------------------------------------------------------------------
# commit / rollback over a device-resident decode state
# ---------------------------------------------------------------------------

class DeviceState:
    """Device copy of the integer decode state (see synth.PagedState).

    All fields are views into one flat int32 buffer, so a whole state can be
    saved or restored with a single device-to-device copy."""

    FIELDS = ("kv_len", "page_table", "num_pages", "free_stack", "boundary", "draft",
              "out_tokens", "out_count", "finished")

    def __init__(self, host, device="cuda"):
        parts = [np.ascontiguousarray(getattr(host, f), dtype=np.int32).reshape(-1)
                 for f in self.FIELDS]
        parts += [np.array([host.free_top], np.int32), np.zeros(1, np.int32)]
        flat = np.concatenate(parts)
        self.flat = torch.from_numpy(flat).to(device)
        off = 0
        for f, a in zip(self.FIELDS + ("free_top", "err"), parts):
            shape = getattr(host, f).shape if f in self.FIELDS else (1,)
            setattr(self, f, self.flat[off:off + a.size].view(shape))
            off += a.size
        self.pool_pages = int(host.pool_pages)
        self.max_pages = int(host.max_pages)

    def copy_from(self, other: "DeviceState"):
        self.flat.copy_(other.flat, non_blocking=True)
        return self

    def to_host(self, host_like):
        h = host_like.copy()
        for f in self.FIELDS:
            setattr(h, f, getattr(self, f).cpu().numpy().copy())
        h.free_top = int(self.free_top.item())
        return h


def accept_commit(st: DeviceState, argmax, n_causal: int, n_mask: int, accept_out=None,
                  eos_id: int = -1, draft_group: int = 0, stream=None):
    """Acceptance, commit and rollback in one kernel; returns accept_out [S] int32."""
    S = st.kv_len.shape[0]
    _dev(argmax, torch.int32, "argmax", 2)
    if argmax.shape != (S, n_causal + n_mask):
        raise DvsError("argmax must be [S, n_causal + n_mask]")
    if accept_out is None:
        accept_out = torch.empty((S,), dtype=torch.int32, device=argmax.device)
    _dev(accept_out, torch.int32, "accept_out", 1)
    rc = lib().accept_commit(S, n_causal, n_mask, int(draft_group), _ptr(argmax), _ptr(accept_out), _ptr(st.kv_len),
                             _ptr(st.page_table), _ptr(st.num_pages), st.max_pages,
                             _ptr(st.free_stack), _ptr(st.free_top), st.pool_pages,
                             _ptr(st.boundary), _ptr(st.draft), st.draft.shape[1],
                             _ptr(st.out_tokens), _ptr(st.out_count), st.out_tokens.shape[1],
                             int(eos_id), _ptr(st.finished), _ptr(st.err), _stream(stream))
    _check(rc, "accept_commit")
    return accept_out


def kv_commit(st: DeviceState, accept_len, argmax, n_causal: int, n_mask: int,
              eos_id: int = -1, max_new: int | None = None, stream=None):
    S = st.kv_len.shape[0]
    _dev(accept_len, torch.int32, "accept_len", 1)
    _dev(argmax, torch.int32, "argmax", 2)
    if argmax.shape != (S, n_causal + n_mask):
        raise DvsError("argmax must be [S, n_causal + n_mask]")
    cap = st.out_tokens.shape[1]
    max_new = cap if max_new is None else min(int(max_new), cap)
    if max_new != cap:
        raise DvsError("max_new must equal the out_tokens row length")
    rc = lib().kv_commit(S, n_causal, n_mask, _ptr(accept_len), _ptr(argmax), _ptr(st.kv_len),
                         _ptr(st.page_table), _ptr(st.num_pages), st.max_pages,
                         _ptr(st.free_stack), _ptr(st.free_top), st.pool_pages,
                         _ptr(st.boundary), _ptr(st.draft), st.draft.shape[1],
                         _ptr(st.out_tokens), _ptr(st.out_count), max_new, int(eos_id),
                         _ptr(st.finished), _ptr(st.err), _stream(stream))
    _check(rc, "kv_commit")


def kv_commit_round(st: DeviceState, B: int, lead, accept_len, argmax, eos_id: int = -1,
                    max_new: int | None = None, stream=None):
    """Commit of the two-forward round: a0 (lead), d_1..d_A, a_{A+1}."""
    S = st.kv_len.shape[0]
    _dev(lead, torch.int32, "lead", 1)
    _dev(accept_len, torch.int32, "accept_len", 1)
    _dev(argmax, torch.int32, "argmax", 2)
    if argmax.shape != (S, B + 1):
        raise DvsError("argmax must be [S, B + 1]")
    cap = st.out_tokens.shape[1]
    max_new = cap if max_new is None else min(int(max_new), cap)
    if max_new != cap:
        raise DvsError("max_new must equal the out_tokens row length")
    rc = lib().kv_commit_round(S, B, _ptr(lead), _ptr(accept_len), _ptr(argmax), _ptr(st.kv_len),
                               _ptr(st.page_table), _ptr(st.num_pages), st.max_pages,
                               _ptr(st.free_stack), _ptr(st.free_top), st.pool_pages,
                               _ptr(st.boundary), _ptr(st.draft), st.draft.shape[1],
                               _ptr(st.out_tokens), _ptr(st.out_count), max_new, int(eos_id),
                               _ptr(st.finished), _ptr(st.err), _stream(stream))
    _check(rc, "kv_commit_round")


def kv_commit_block(st: DeviceState, block, eos_id: int = -1, max_new: int | None = None,
                    stream=None):
    """Commit of one direct block-diffusion block: b_1..b_B (block [S, B])."""
    S = st.kv_len.shape[0]
    _dev(block, torch.int32, "block", 2)
    if block.shape[0] != S:
        raise DvsError("block must be [S, B]")
    cap = st.out_tokens.shape[1]
    max_new = cap if max_new is None else min(int(max_new), cap)
    if max_new != cap:
        raise DvsError("max_new must equal the out_tokens row length")
    rc = lib().kv_commit_block(S, block.shape[1], _ptr(block), _ptr(st.kv_len),
                               _ptr(st.page_table), _ptr(st.num_pages), st.max_pages,
                               _ptr(st.free_stack), _ptr(st.free_top), st.pool_pages,
                               _ptr(st.boundary), _ptr(st.out_tokens), _ptr(st.out_count),
                               max_new, int(eos_id), _ptr(st.finished), _ptr(st.err),
                               _stream(stream))
    _check(rc, "kv_commit_block")


# ---------------------------------------------------------------------------
# whole-step decoder
# ---------------------------------------------------------------------------

def _to_dev_weight(a: np.ndarray, dtype: str, transpose: bool, device="cuda"):
    """float32 host array -> device tensor in the model dtype (bf16 by RNE)."""
    a = np.ascontiguousarray(a.T if transpose else a, dtype=np.float32)
    if dtype == "bf16":
        from . import synth
        bits = synth.f32_to_bf16_bits(a)
        return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(a).to(device)


class DeviceModel:
    """Decoder weights (uploaded as [out, in]) and per-layer KV pools on the
    device, described to the library by a dvs_model struct."""

    def __init__(self, w, k_pools, v_pools, dtype: str = "f32", device="cuda"):
        self.dtype = dtype
        tw = lambda a: _to_dev_weight(a, dtype, True, device)      # [in,out] -> [out,in]
        tv = lambda a: _to_dev_weight(a, dtype, False, device)
        self.embed = tv(w.embed)
        self.g_final = tv(w.g_final)
        self.lm_head = tw(w.lm_head)
        self.keep = []
        self.k_pools, self.v_pools = [], []
        layers = (DvsLayer * w.n_layers)()
        for l in range(w.n_layers):
            kp = k_pools[l] if isinstance(k_pools[l], torch.Tensor) else tv(k_pools[l])
            vp = v_pools[l] if isinstance(v_pools[l], torch.Tensor) else tv(v_pools[l])
            self.k_pools.append(kp)
            self.v_pools.append(vp)
            t = dict(wq=tw(w.wq[l]), wk=tw(w.wk[l]), wv=tw(w.wv[l]), wo=tw(w.wo[l]),
                     g_attn=tv(w.g_attn[l]))
            if w.ffn:
                t.update(g_mlp=tv(w.g_mlp[l]), w_gate=tw(w.w_gate[l]), w_up=tw(w.w_up[l]),
                         w_down=tw(w.w_down[l]))
            self.keep.append(t)
            for n, v in t.items():
                setattr(layers[l], n, v.data_ptr())
            layers[l].k_pool = kp.data_ptr()
            layers[l].v_pool = vp.data_ptr()
        self.layers = layers
        self.desc = DvsModel(DVS_BF16 if dtype == "bf16" else DVS_F32, w.n_layers, w.V, w.H, w.Hq,
                             w.Hkv, w.D, w.ffn, float(w.rope_theta), float(w.eps),
                             self.embed.data_ptr(), self.g_final.data_ptr(),
                             self.lm_head.data_ptr(), layers)
        self.V, self.H = w.V, w.H
        self.ws = None

    def workspace_bytes(self, S, n_causal, n_mask, max_pages, chunk_keys=MODEL_CHUNK_KEYS) -> int:
        return int(lib().dvs_step_workspace_bytes(ctypes.byref(self.desc), S, n_causal, n_mask,
                                                  max_pages, chunk_keys))


def _state_desc(st: DeviceState, eos_id: int) -> DvsState:
    S = st.kv_len.shape[0]
    return DvsState(S, st.max_pages, st.pool_pages, st.draft.shape[1], st.out_tokens.shape[1],
                    int(eos_id), st.kv_len.data_ptr(), st.page_table.data_ptr(),
                    st.num_pages.data_ptr(), st.free_stack.data_ptr(), st.free_top.data_ptr(),
                    st.boundary.data_ptr(), st.draft.data_ptr(), st.out_tokens.data_ptr(),
                    st.out_count.data_ptr(), st.finished.data_ptr(), st.err.data_ptr())


def draft_verify_step(model: DeviceModel, st: DeviceState, n_causal: int, n_mask: int,
                      chunk_keys: int = MODEL_CHUNK_KEYS, eos_id: int = -1, logits_out=None, argmax_out=None,
                      accept_out=None, stream=None):
    """One fused step (or an AR step with n_causal=1, n_mask=0) on the device."""
    S = st.kv_len.shape[0]
    need = model.workspace_bytes(S, n_causal, n_mask, st.max_pages, chunk_keys)
    if need == 0:
        raise DvsError("draft_verify_step: invalid configuration")
    if model.ws is None or model.ws.nbytes < need:
        model.ws = Workspace(need, device=st.kv_len.device)
    for t, name in ((logits_out, "logits_out"), (argmax_out, "argmax_out"), (accept_out, "accept_out")):
        if t is not None:
            _dev(t, torch.float32 if name == "logits_out" else torch.int32, name)
    sd = _state_desc(st, eos_id)
    rc = lib().draft_verify_step(ctypes.byref(model.desc), ctypes.byref(sd), n_causal, n_mask,
                                 int(chunk_keys), _ptr(logits_out), _ptr(argmax_out),
                                 _ptr(accept_out), _ptr(model.ws.buf), model.ws.nbytes,
                                 _stream(stream))
    _check(rc, "draft_verify_step")


def multidraft_step(model: DeviceModel, st: DeviceState, B: int,
                    chunk_keys: int = MODEL_CHUNK_KEYS, eos_id: int = -1, logits_out=None,
                    argmax_out=None, accept_out=None, stream=None):
    """One fused step with a draft block per possible acceptance (B groups of
    B mask rows; the next draft comes from group A) on the device."""
    S = st.kv_len.shape[0]
    need = model.workspace_bytes(S, B, B * B, st.max_pages, chunk_keys)
    if need == 0:
        raise DvsError("multidraft_step: invalid configuration")
    if model.ws is None or model.ws.nbytes < need:
        model.ws = Workspace(need, device=st.kv_len.device)
    for t, name in ((logits_out, "logits_out"), (argmax_out, "argmax_out"), (accept_out, "accept_out")):
        if t is not None:
            _dev(t, torch.float32 if name == "logits_out" else torch.int32, name)
    sd = _state_desc(st, eos_id)
    rc = lib().multidraft_step(ctypes.byref(model.desc), ctypes.byref(sd), B, int(chunk_keys),
                               _ptr(logits_out), _ptr(argmax_out), _ptr(accept_out),
                               _ptr(model.ws.buf), model.ws.nbytes, _stream(stream))
    _check(rc, "multidraft_step")


def attn_hybrid_block_grouped(q, k_new, v_new, k_pool, v_pool, page_table, kv_len, n_causal: int,
                              n_mask: int, mask_group: int, softmax_scale: float, out=None,
                              err=None, workspace=None, chunk_keys: int = 0, stream=None):
    """attn_hybrid_block with the mask rows in groups of mask_group rows."""
    S, R, Hq, Hkv, D, P, max_pages, out = _attn_args(q, k_new, v_new, k_pool, v_pool, page_table,
                                                     kv_len, n_causal, n_mask, out, err)
    code = _dtype_code(q)
    need = attn_workspace_bytes(S, n_causal, n_mask, Hq, Hkv, D, max_pages, chunk_keys, code)
    if workspace is None:
        workspace = Workspace(need, device=q.device)
    workspace.prepare(need, ("attn", S, R, Hq, Hkv, D, max_pages, int(chunk_keys), code))
    rc = lib().attn_hybrid_block_grouped(_ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_pool),
                                         _ptr(v_pool), _ptr(page_table), _ptr(kv_len), S, n_causal,
                                         n_mask, int(mask_group), Hq, Hkv, D, max_pages, P,
                                         float(softmax_scale), code, int(chunk_keys), _ptr(out),
                                         _ptr(err), _ptr(workspace.buf), workspace.nbytes,
                                         _stream(stream))
    _check(rc, "attn_hybrid_block_grouped")
    return out


def literal_round(model: DeviceModel, st: DeviceState, B: int, chunk_keys: int = MODEL_CHUNK_KEYS,
                  eos_id: int = -1, logits_out=None, argmax_out=None, accept_out=None, stream=None):
    """One round of the paper's two-forward decoding (draft forward, verify
    forward, commit of a0, d_1..d_A, a_{A+1}) on the device."""
    S = st.kv_len.shape[0]
    need = model.workspace_bytes(S, B + 1, 0, st.max_pages, chunk_keys)
    if need == 0:
        raise DvsError("literal_round: invalid configuration")
    if model.ws is None or model.ws.nbytes < need:
        model.ws = Workspace(need, device=st.kv_len.device)
    for t, name in ((logits_out, "logits_out"), (argmax_out, "argmax_out"), (accept_out, "accept_out")):
        if t is not None:
            _dev(t, torch.float32 if name == "logits_out" else torch.int32, name)
    sd = _state_desc(st, eos_id)
    rc = lib().literal_round(ctypes.byref(model.desc), ctypes.byref(sd), int(B), int(chunk_keys),
                             _ptr(logits_out), _ptr(argmax_out), _ptr(accept_out),
                             _ptr(model.ws.buf), model.ws.nbytes, _stream(stream))
    _check(rc, "literal_round")


def capture(fn) -> "torch.cuda.CUDAGraph":
    """Record the launches of ``fn`` (calls of this module that only enqueue:
    draft_verify_step, literal_round, attn_hybrid_block, argmax_accept, the
    commits; not diffusion_block or literal_round_refined, which read a count
    back from the device) into a HIP graph.  ``replay()`` re-runs them on the
    buffers' current contents: every input of a step (kv_len, pages, boundary,
    draft, ...) is read from device memory, so a replay is the next step.
    The library clears its counters with kernels, never with a memset node.
    Workspaces must be allocated before the capture (one eager call does it)
    and must not be replaced (by a call needing a larger one) while the
    graph is replayed."""
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    return g


def literal_round_refined(model: DeviceModel, st: DeviceState, B: int, tau_d: float,
                          chunk_keys: int = MODEL_CHUNK_KEYS, eos_id: int = -1, logits_out=None, argmax_out=None,
                          accept_out=None, stream=None) -> int:
    """The two-forward round with its draft refined at threshold tau_d over
    several draft forwards; returns the number of draft forwards."""
    S = st.kv_len.shape[0]
    need = max(model.workspace_bytes(S, 1, B, st.max_pages, chunk_keys),
               model.workspace_bytes(S, B + 1, 0, st.max_pages, chunk_keys))
    if need == 0:
        raise DvsError("literal_round_refined: invalid configuration")
    if model.ws is None or model.ws.nbytes < need:
        model.ws = Workspace(need, device=st.kv_len.device)
    for t, name in ((logits_out, "logits_out"), (argmax_out, "argmax_out"), (accept_out, "accept_out")):
        if t is not None:
            _dev(t, torch.float32 if name == "logits_out" else torch.int32, name)
    steps = ctypes.c_int32(0)
    sd = _state_desc(st, eos_id)
    rc = lib().literal_round_refined(ctypes.byref(model.desc), ctypes.byref(sd), int(B),
                                     float(tau_d), int(chunk_keys), _ptr(logits_out),
                                     _ptr(argmax_out), _ptr(accept_out), ctypes.byref(steps),
                                     _ptr(model.ws.buf), model.ws.nbytes, _stream(stream))
    _check(rc, "literal_round_refined")
    return int(steps.value)


def literal_round_sampled(model: DeviceModel, st: DeviceState, B: int, temperature: float, u,
                          chunk_keys: int = MODEL_CHUNK_KEYS, eos_id: int = -1, logits_out=None,
                          accept_out=None, stream=None):
    """The two-forward round under sampling (stochastic acceptance); u is a
    device float32 [S, 2B + 2] of uniforms in [0, 1)."""
    S = st.kv_len.shape[0]
    _dev(u, torch.float32, "u", 2)
    if tuple(u.shape) != (S, 2 * B + 2):
        raise DvsError("u must be [S, 2B + 2]")
    need = int(lib().dvs_sampled_round_workspace_bytes(ctypes.byref(model.desc), S, int(B),
                                                       st.max_pages, int(chunk_keys)))
    if need == 0:
        raise DvsError("literal_round_sampled: invalid configuration")
    if model.ws is None or model.ws.nbytes < need:
        model.ws = Workspace(need, device=st.kv_len.device)
    if logits_out is not None:
        _dev(logits_out, torch.float32, "logits_out")
    if accept_out is not None:
        _dev(accept_out, torch.int32, "accept_out", 1)
    sd = _state_desc(st, eos_id)
    rc = lib().literal_round_sampled(ctypes.byref(model.desc), ctypes.byref(sd), int(B),
                                     float(temperature), _ptr(u), int(chunk_keys),
                                     _ptr(logits_out), _ptr(accept_out), _ptr(model.ws.buf),
                                     model.ws.nbytes, _stream(stream))
    _check(rc, "literal_round_sampled")


def diffusion_denoise(model: DeviceModel, st: DeviceState, block, tau_c: float, n_open=None,
                      chunk_keys: int = MODEL_CHUNK_KEYS, eos_id: int = -1, logits_out=None, argmax_out=None,
                      conf_out=None, stream=None):
    """One denoising forward of direct block diffusion and its reveal; block
    [S, B] int32 (-1 = masked) is updated in place.  Returns n_open (a device
    int32 [1]: live sequences whose block is still open)."""
    S = st.kv_len.shape[0]
    _dev(block, torch.int32, "block", 2)
    B = block.shape[1]
    if block.shape[0] != S:
        raise DvsError("block must be [S, B]")
    need = model.workspace_bytes(S, 1, B, st.max_pages, chunk_keys)
    if need == 0:
        raise DvsError("diffusion_denoise: invalid configuration")
    if model.ws is None or model.ws.nbytes < need:
        model.ws = Workspace(need, device=st.kv_len.device)
    if n_open is None:
        n_open = torch.empty(1, dtype=torch.int32, device=st.kv_len.device)
    _dev(n_open, torch.int32, "n_open", 1)
    for t, name, dt in ((logits_out, "logits_out", torch.float32),
                        (argmax_out, "argmax_out", torch.int32), (conf_out, "conf_out", torch.float32)):
        if t is not None:
            _dev(t, dt, name)
    sd = _state_desc(st, eos_id)
    rc = lib().diffusion_denoise(ctypes.byref(model.desc), ctypes.byref(sd), int(B), float(tau_c),
                                 _ptr(block), _ptr(n_open), int(chunk_keys), _ptr(logits_out),
                                 _ptr(argmax_out), _ptr(conf_out), _ptr(model.ws.buf),
                                 model.ws.nbytes, _stream(stream))
    _check(rc, "diffusion_denoise")
    return n_open


def diffusion_block(model: DeviceModel, st: DeviceState, B: int, tau_c: float, block=None,
                    chunk_keys: int = MODEL_CHUNK_KEYS, eos_id: int = -1, stream=None):
    """Decode and commit one block by direct block diffusion.  Returns
    (block [S, B] int32, denoising forwards); the block cost one more
    forward (the cache write)."""
    S = st.kv_len.shape[0]
    need = int(lib().dvs_diffusion_workspace_bytes(ctypes.byref(model.desc), S, int(B),
                                                   st.max_pages, int(chunk_keys)))
    if need == 0:
        raise DvsError("diffusion_block: invalid configuration")
    if model.ws is None or model.ws.nbytes < need:
        model.ws = Workspace(need, device=st.kv_len.device)
    if block is None:
        block = torch.empty((S, B), dtype=torch.int32, device=st.kv_len.device)
    _dev(block, torch.int32, "block", 2)
    if tuple(block.shape) != (S, B):
        raise DvsError("block must be [S, B]")
    steps = ctypes.c_int32(0)
    sd = _state_desc(st, eos_id)
    rc = lib().diffusion_block(ctypes.byref(model.desc), ctypes.byref(sd), int(B), float(tau_c),
                               _ptr(block), int(chunk_keys), ctypes.byref(steps),
                               _ptr(model.ws.buf), model.ws.nbytes, _stream(stream))
    _check(rc, "diffusion_block")
    return block, int(steps.value)


def prefill(model: DeviceModel, st: DeviceState, P: int, n_mask: int, prefix_tokens=None,
            x_prefix=None, chunk_keys: int = MODEL_CHUNK_KEYS, eos_id: int = -1, logits_out=None, stream=None):
    """Prefill P prefix rows (token ids and/or given fp32 embeddings) plus
    n_mask mask rows; sets kv_len, boundary, first draft and first token."""
    S = st.kv_len.shape[0]
    if prefix_tokens is not None:
        _dev(prefix_tokens, torch.int32, "prefix_tokens", 2)
    if x_prefix is not None:
        _dev(x_prefix, torch.float32, "x_prefix", 3)
    need = int(lib().dvs_prefill_workspace_bytes(ctypes.byref(model.desc), S, P, n_mask,
                                                 st.max_pages, chunk_keys))
    if need == 0:
        raise DvsError("dvs_prefill: invalid configuration")
    if model.ws is None or model.ws.nbytes < need:
        model.ws = Workspace(need, device=st.kv_len.device)
    sd = _state_desc(st, eos_id)
    rc = lib().dvs_prefill(ctypes.byref(model.desc), ctypes.byref(sd), P, n_mask,
                           _ptr(prefix_tokens), _ptr(x_prefix), int(chunk_keys), _ptr(logits_out),
                           _ptr(model.ws.buf), model.ws.nbytes, _stream(stream))
    _check(rc, "dvs_prefill")
