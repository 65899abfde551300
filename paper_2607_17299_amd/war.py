"""Thin ctypes binding over libwar.so (the C ABI declared in include/war.h).

Argument marshalling only: every step of the verify path runs in the HIP
kernels behind the C ABI.  torch provides device memory and the stream; arrays
are passed as raw device pointers (``tensor.data_ptr()``).  Importing this
module fails loudly when the library has not been built -- there is no
fallback path.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, List, Optional, Sequence

import torch

from .synth import ModelConfig, weight_shapes

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libwar.so")

WAR_OK = 0
_ERRORS = {-1: "WAR_ERR_INVALID_ARG", -2: "WAR_ERR_OUT_OF_PAGES", -3: "WAR_ERR_HIP",
           -4: "WAR_ERR_UNSUPPORTED", -5: "WAR_ERR_DEVICE"}

EXPORTS = ["war_weight_count", "war_model_create", "war_model_destroy", "war_kv_pool_create",
           "war_kv_pool_destroy", "war_kv_alloc", "war_kv_fork", "war_kv_free", "war_kv_load",
           "war_prefill_append", "war_verify_step", "war_verify_step_sampled", "war_verify_step_tree",
           "war_verify_step_noalloc",
           "war_kv_commit", "war_pool_state",
           "war_last_error", "war_debug_mfma16", "war_debug_workspace", "war_debug_sample",
           "war_debug_pool_waits", "war_profile", "war_profile_read"]


class WarError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_ERRORS.get(status, status)}: {msg}")
        self.status = status


class _Config(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn_dim", C.c_int32),
                ("vocab", C.c_int32), ("rms_eps", C.c_float), ("rope_base", C.c_float),
                ("page_size", C.c_int32), ("max_rows", C.c_int32)]


def load_library(path: str = LIB_PATH) -> C.CDLL:
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2607_17299_amd.build`")
    lib = C.CDLL(path)
    vp, i32, pi32 = C.c_void_p, C.c_int32, C.POINTER(C.c_int32)
    sig = {
        "war_weight_count": (i32, [C.POINTER(_Config)]),
        "war_model_create": (i32, [C.POINTER(_Config), C.POINTER(vp), i32, C.POINTER(vp)]),
        "war_model_destroy": (None, [vp]),
        "war_kv_pool_create": (i32, [C.POINTER(_Config), vp, i32, vp, i32, i32, vp, C.POINTER(vp)]),
        "war_kv_pool_destroy": (None, [vp]),
        "war_kv_alloc": (i32, [vp, i32, pi32, pi32, vp]),
        "war_kv_fork": (i32, [vp, i32, i32, i32, vp]),
        "war_kv_free": (i32, [vp, i32, pi32, vp]),
        "war_kv_load": (i32, [vp, i32, i32, i32, i32, vp, vp]),
        "war_prefill_append": (i32, [vp, vp, i32, vp, vp, pi32, vp, vp, vp, vp]),
        "war_verify_step": (i32, [vp, vp, i32, vp, vp, vp, vp, vp, i32, vp, vp, vp, vp]),
        "war_verify_step_sampled": (i32, [vp, vp, i32, vp, vp, vp, vp, vp, i32, vp, C.c_float, i32,
                                          vp, vp, vp, vp]),
        "war_verify_step_tree": (i32, [vp, vp, i32, vp, vp, vp, vp, vp, vp, i32, vp, vp, vp, vp, vp]),
        "war_verify_step_noalloc": (i32, [vp, vp, i32, vp, vp, vp, vp, vp, i32, vp, vp, vp, vp]),
        "war_kv_commit": (i32, [vp, i32, vp, vp, vp, vp]),
        "war_pool_state": (i32, [vp, pi32, pi32, pi32, pi32, pi32, vp]),
        "war_last_error": (C.c_char_p, []),
        "war_debug_sample": (i32, [vp, i32, i32, i32, vp, vp, vp, C.c_float, i32, vp, vp, vp]),
        "war_debug_mfma16": (i32, [vp, vp, vp, vp]),
        "war_debug_workspace": (i32, [vp, C.c_char_p, C.POINTER(vp), C.POINTER(C.c_int64)]),
        "war_debug_pool_waits": (i32, [vp, C.POINTER(C.c_int64)]),
        "war_profile": (i32, [vp, i32]),
        "war_profile_read": (i32, [vp, C.c_char_p, i32]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype, f.argtypes = res, args
    return lib


_LIB: Optional[C.CDLL] = None


def lib() -> C.CDLL:
    global _LIB
    if _LIB is None:
        _LIB = load_library()
    return _LIB


def _check(status: int) -> None:
    if status != WAR_OK:
        raise WarError(status, lib().war_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _host_i32(xs: Sequence[int]):
    arr = (C.c_int32 * len(xs))(*[int(x) for x in xs])
    return arr


def config_struct(cfg: ModelConfig, max_rows: int) -> _Config:
    return _Config(cfg.n_layers, cfg.d_model, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim,
                   cfg.ffn_dim, cfg.vocab, cfg.rms_eps, cfg.rope_base, cfg.page_size, max_rows)


class Model:
    """A decoder over bf16 device weights (canonical order).  The library copies
    (and repacks) them at creation; the tensors may be dropped afterwards."""

    def __init__(self, cfg: ModelConfig, weights: Dict[str, torch.Tensor], max_rows: int = 1024):
        self.cfg, self.max_rows = cfg, max_rows
        names = [n for n, _ in weight_shapes(cfg)]
        ws = [weights[n] for n in names]
        for t in ws:
            assert t.is_cuda and t.dtype == torch.bfloat16 and t.is_contiguous()
        arr = (C.c_void_p * len(ws))(*[t.data_ptr() for t in ws])
        self._cfg = config_struct(cfg, max_rows)
        h = C.c_void_p()
        torch.cuda.synchronize()                    # the weights are complete before the copy
        _check(lib().war_model_create(C.byref(self._cfg), arr, len(ws), C.byref(h)))
        self.handle = h

    def close(self):
        if getattr(self, "handle", None):
            lib().war_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Pool:
    """A paged KV pool: caller-owned KV storage and block tables (torch tensors)."""

    def __init__(self, cfg: ModelConfig, num_pages: int, max_seqs: int, max_pages_per_seq: int,
                 device="cuda", stream=None):
        self.cfg = cfg
        self.num_pages, self.max_seqs, self.max_pages = num_pages, max_seqs, max_pages_per_seq
        n = cfg.n_layers * num_pages * cfg.n_kv_heads * 2 * cfg.page_size * cfg.head_dim
        self.kv = torch.empty(n, dtype=torch.bfloat16, device=device)
        self.block_tables = torch.empty((max_seqs, max_pages_per_seq), dtype=torch.int32, device=device)
        self._cfg = config_struct(cfg, 1)
        h = C.c_void_p()
        _check(lib().war_kv_pool_create(C.byref(self._cfg), _ptr(self.kv), num_pages,
                                        _ptr(self.block_tables), max_seqs, max_pages_per_seq,
                                        _stream(stream), C.byref(h)))
        self.handle = h

    # ---- layout helpers (views of the caller-owned storage)
    def kv_view(self) -> torch.Tensor:
        c = self.cfg
        return self.kv.view(c.n_layers, self.num_pages, c.n_kv_heads, 2, c.page_size, c.head_dim)

    def _key_order(self) -> torch.Tensor:
        """Element index, inside a page's K region, of key slot s and dim d
        ([P, D]): the fragment order of include/war.h (groups of eight slots
        by (s / 4) % 2, 32-dim k-steps, eight 64-byte rows per run)."""
        c = self.cfg
        s = torch.arange(c.page_size).view(-1, 1)
        d = torch.arange(c.head_dim).view(1, -1)
        t, s8 = (s // 4) % 2, (s // 8) * 4 + s % 4
        return ((t * (c.head_dim // 32) + d // 32) * 8 + s8) * 32 + d % 32

    def gather_kv(self, seq: int, n_tokens: int, layer: int) -> torch.Tensor:
        """[2, Hkv, n_tokens, D] keys/values of a sequence read back from its pages."""
        c = self.cfg
        pages = self.block_tables[seq, : -(-n_tokens // c.page_size)].long()
        v = self.kv_view()[layer, pages]                       # [np, H, 2, P, D]
        kraw = v[:, :, 0].reshape(len(pages), c.n_kv_heads, c.page_size * c.head_dim)
        korder = self._key_order().to(kraw.device).reshape(-1)
        k = kraw[:, :, korder].reshape(len(pages), c.n_kv_heads, c.page_size, c.head_dim)
        k = k.permute(1, 0, 2, 3).reshape(c.n_kv_heads, -1, c.head_dim)
        vt = v[:, :, 1].reshape(len(pages), c.n_kv_heads, c.head_dim, c.page_size)
        vv = vt.permute(1, 0, 3, 2).reshape(c.n_kv_heads, -1, c.head_dim)
        return torch.stack([k[:, :n_tokens], vv[:, :n_tokens]])

    # ---- operations
    def alloc(self, seq_ids: Sequence[int], n_tokens: Sequence[int], stream=None):
        _check(lib().war_kv_alloc(self.handle, len(seq_ids), _host_i32(seq_ids), _host_i32(n_tokens),
                                  _stream(stream)))

    def fork(self, src: int, dst: int, n_tokens: int, stream=None):
        _check(lib().war_kv_fork(self.handle, src, dst, n_tokens, _stream(stream)))

    def free(self, seq_ids: Sequence[int], stream=None):
        _check(lib().war_kv_free(self.handle, len(seq_ids), _host_i32(seq_ids), _stream(stream)))

    def load(self, seq: int, layer: int, pos0: int, kv: torch.Tensor, stream=None):
        assert kv.dtype == torch.bfloat16 and kv.is_contiguous() and kv.dim() == 4
        _check(lib().war_kv_load(self.handle, seq, layer, pos0, kv.shape[2], _ptr(kv), _stream(stream)))

    def state(self, stream=None) -> Dict:
        fc = C.c_int32()
        stack = (C.c_int32 * self.num_pages)()
        ref = (C.c_int32 * self.num_pages)()
        held = (C.c_int32 * self.max_seqs)()
        base = (C.c_int32 * self.max_seqs)()
        st = lib().war_pool_state(self.handle, C.byref(fc), stack, ref, held, base, _stream(stream))
        import numpy as np
        out = {"stack": np.array(stack[: fc.value], dtype=np.int32), "refcount": np.array(ref[:], np.int32),
               "held": np.array(held[:], np.int32), "base": np.array(base[:], np.int32),
               "table": self.block_tables.cpu().numpy(), "status": st}
        return out

    def waits(self) -> int:
        """Verify steps that waited to read the exact free page count."""
        n = C.c_int64()
        _check(lib().war_debug_pool_waits(self.handle, C.byref(n)))
        return n.value

    def close(self):
        if getattr(self, "handle", None):
            lib().war_kv_pool_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def verify_step(model: Model, pool: Pool, seq_ids: torch.Tensor, ctx_lens: torch.Tensor,
                last_tokens: torch.Tensor, draft_tokens: Optional[torch.Tensor],
                draft_lens: Optional[torch.Tensor], k_max: int, accept_lens: torch.Tensor,
                next_tokens: torch.Tensor, logits: Optional[torch.Tensor] = None, stream=None) -> None:
    B = seq_ids.numel()
    _check(lib().war_verify_step(model.handle, pool.handle, B, _ptr(seq_ids), _ptr(ctx_lens),
                                 _ptr(last_tokens), _ptr(draft_tokens), _ptr(draft_lens), k_max,
                                 _ptr(accept_lens), _ptr(next_tokens), _ptr(logits), _stream(stream)))


def verify_step_noalloc(model: Model, pool: Pool, seq_ids: torch.Tensor, ctx_lens: torch.Tensor,
                        last_tokens: torch.Tensor, draft_tokens: Optional[torch.Tensor],
                        draft_lens: Optional[torch.Tensor], k_max: int, accept_lens: torch.Tensor,
                        next_tokens: torch.Tensor, logits: Optional[torch.Tensor] = None, stream=None) -> None:
    """war_verify_step over the library's static device scratch (allocates nothing)."""
    B = seq_ids.numel()
    _check(lib().war_verify_step_noalloc(model.handle, pool.handle, B, _ptr(seq_ids), _ptr(ctx_lens),
                                         _ptr(last_tokens), _ptr(draft_tokens), _ptr(draft_lens), k_max,
                                         _ptr(accept_lens), _ptr(next_tokens), _ptr(logits), _stream(stream)))


def verify_step_sampled(model: Model, pool: Pool, seq_ids: torch.Tensor, ctx_lens: torch.Tensor,
                        last_tokens: torch.Tensor, draft_tokens: Optional[torch.Tensor],
                        draft_lens: Optional[torch.Tensor], k_max: int, uniforms: torch.Tensor,
                        temperature: float, top_k: int, accept_lens: torch.Tensor, next_tokens: torch.Tensor,
                        logits: Optional[torch.Tensor] = None, stream=None) -> None:
    """Sampled verification; uniforms fp32 [B * (k_max + 1), 2] on the device."""
    assert uniforms.dtype == torch.float32 and uniforms.is_contiguous()
    B = seq_ids.numel()
    _check(lib().war_verify_step_sampled(model.handle, pool.handle, B, _ptr(seq_ids), _ptr(ctx_lens),
                                         _ptr(last_tokens), _ptr(draft_tokens), _ptr(draft_lens), k_max,
                                         _ptr(uniforms), float(temperature), int(top_k), _ptr(accept_lens),
                                         _ptr(next_tokens), _ptr(logits), _stream(stream)))


def verify_step_tree(model: Model, pool: Pool, seq_ids: torch.Tensor, ctx_lens: torch.Tensor,
                     last_tokens: torch.Tensor, draft_tokens: Optional[torch.Tensor],
                     draft_parents: Optional[torch.Tensor], draft_lens: Optional[torch.Tensor], k_max: int,
                     accept_lens: torch.Tensor, next_tokens: torch.Tensor,
                     accept_path: Optional[torch.Tensor] = None, logits: Optional[torch.Tensor] = None,
                     stream=None) -> None:
    """Tree drafts: draft_parents int32 [B, k_max], node i's parent in [0, i)."""
    B = seq_ids.numel()
    _check(lib().war_verify_step_tree(model.handle, pool.handle, B, _ptr(seq_ids), _ptr(ctx_lens),
                                      _ptr(last_tokens), _ptr(draft_tokens), _ptr(draft_parents),
                                      _ptr(draft_lens), k_max, _ptr(accept_lens), _ptr(next_tokens),
                                      _ptr(accept_path), _ptr(logits), _stream(stream)))


def kv_commit(pool: Pool, seq_ids: torch.Tensor, ctx_lens: torch.Tensor, accept_lens: torch.Tensor,
              stream=None) -> None:
    _check(lib().war_kv_commit(pool.handle, seq_ids.numel(), _ptr(seq_ids), _ptr(ctx_lens),
                               _ptr(accept_lens), _stream(stream)))


def prefill_append(model: Model, pool: Pool, seq_ids: torch.Tensor, ctx_lens: torch.Tensor,
                   n_new: Sequence[int], new_tokens: torch.Tensor, next_tokens: torch.Tensor,
                   last_logits: Optional[torch.Tensor] = None, stream=None) -> None:
    n = seq_ids.numel()
    _check(lib().war_prefill_append(model.handle, pool.handle, n, _ptr(seq_ids), _ptr(ctx_lens),
                                    _host_i32(n_new), _ptr(new_tokens), _ptr(next_tokens),
                                    _ptr(last_logits), _stream(stream)))


def debug_mfma16(A: torch.Tensor, B: torch.Tensor, stream=None) -> torch.Tensor:
    """C = A @ B (A bf16 [16, 32], B bf16 [32, 16]) through one matrix-core instruction."""
    out = torch.empty((16, 16), dtype=torch.float32, device=A.device)
    _check(lib().war_debug_mfma16(_ptr(A.contiguous()), _ptr(B.contiguous()), _ptr(out), _stream(stream)))
    return out


def debug_sample(logits: torch.Tensor, ntok: torch.Tensor, drafts: torch.Tensor, k_max: int,
                 uniforms: torch.Tensor, temperature: float, top_k: int, accept_lens: torch.Tensor,
                 next_tokens: torch.Tensor, stream=None) -> None:
    """The sampled-verification decisions alone on given logit rows (war_debug.h)."""
    B, V = ntok.numel(), logits.shape[-1]
    _check(lib().war_debug_sample(_ptr(logits), V, B, k_max, _ptr(ntok), _ptr(drafts), _ptr(uniforms),
                                  float(temperature), int(top_k), _ptr(accept_lens), _ptr(next_tokens),
                                  _stream(stream)))


def debug_workspace(model: Model, name: str, dtype: torch.dtype, shape) -> torch.Tensor:
    """Copy of a model workspace buffer (see war_debug.h), reinterpreted."""
    p, n = C.c_void_p(), C.c_int64()
    _check(lib().war_debug_workspace(model.handle, name.encode(), C.byref(p), C.byref(n)))
    numel = 1
    for s in shape:
        numel *= s
    nbytes = numel * torch.tensor([], dtype=dtype).element_size()
    assert nbytes <= n.value, (nbytes, n.value)
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipMemcpy(C.c_void_p(buf.data_ptr()), p, C.c_size_t(nbytes), 3)   # device to device
    return buf.view(dtype).view(*shape).clone()


def profile(model: Model, enable: bool) -> None:
    _check(lib().war_profile(model.handle, 1 if enable else 0))


def profile_read(model: Model) -> Dict[str, tuple]:
    """{kernel name: (calls, total_ms)} since the last read; synchronises."""
    buf = C.create_string_buffer(1 << 16)
    _check(lib().war_profile_read(model.handle, buf, len(buf)))
    out = {}
    for line in buf.value.decode().splitlines():
        name, calls, ms = line.split()
        out[name] = (int(calls), float(ms))
    return out
