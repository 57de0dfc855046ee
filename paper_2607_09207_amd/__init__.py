"""MI355X (gfx950) decode attention over a paged KV cache.

The computation is the one that dominates the rollout stage of the RL
post-training loop the paper schedules (Sec. 2.3, App. A.1.2): one query token per
sequence attending over a paged KV cache with long-tailed lengths and GRPO groups
that share prompt pages.  All arithmetic runs in the HIP kernels of
librl_decode_attn.so; this module only marshals torch tensors (device memory and
the current stream) into the C ABI of include/rl_decode_attn.h.
"""
from __future__ import annotations

import ctypes
from typing import Optional

from . import _abi

__all__ = ["DecodeAttention", "decode_attention", "RldaError", "library_path"]

RldaError = _abi.RldaError
library_path = _abi.LIB_PATH


def _torch():
    import torch
    return torch


def _torch_dtype(code: int):
    torch = _torch()
    return {_abi.RLDA_F32: torch.float32, _abi.RLDA_BF16: torch.bfloat16,
            _abi.RLDA_FP8_E4M3FN: torch.float8_e4m3fn}[code]


def _dtype_code(t) -> int:
    torch = _torch()
    if t in (torch.float32, "f32"):
        return _abi.RLDA_F32
    if t in (torch.bfloat16, "bf16"):
        return _abi.RLDA_BF16
    if t in (torch.float8_e4m3fn, "fp8_e4m3fn"):
        return _abi.RLDA_FP8_E4M3FN
    raise TypeError(f"unsupported dtype {t}")


class DecodeAttention:
    """A configured decode-attention layer (a library handle).

    k_cache / v_cache passed to __call__ are 4-D tensors of shape
    [num_pages, num_kv_heads, page_size, head_dim] with head_dim contiguous; any
    other strides (e.g. a [num_pages, page_size, num_kv_heads, head_dim] buffer
    viewed with .transpose(1, 2)) are given here as `kv_strides` (elements).
    """

    def __init__(self, num_q_heads: int, num_kv_heads: int, head_dim: int, max_batch: int,
                 max_pages_per_seq: int, q_dtype="bf16", kv_dtype="bf16", out_dtype="f32",
                 kv_head_of_q=None, softmax_scale: float = 0.0, kv_strides=None,
                 num_work_ranges: int = 0, page_size: int = 16):
        lib = _abi.load()
        cfg = _abi.Config()
        cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim = num_q_heads, num_kv_heads, head_dim
        cfg.page_size, cfg.max_batch, cfg.max_pages_per_seq = page_size, max_batch, max_pages_per_seq
        cfg.q_dtype, cfg.kv_dtype, cfg.out_dtype = _dtype_code(q_dtype), _dtype_code(kv_dtype), _dtype_code(out_dtype)
        self._head_map = None
        if kv_head_of_q is not None:
            self._head_map = (ctypes.c_int32 * num_q_heads)(*[int(x) for x in kv_head_of_q])
            cfg.kv_head_of_q = self._head_map
        cfg.softmax_scale = float(softmax_scale)
        if kv_strides is not None:
            cfg.kv_stride_page, cfg.kv_stride_head, cfg.kv_stride_slot = [int(x) for x in kv_strides]
        cfg.num_work_ranges = int(num_work_ranges)
        P, d = page_size, head_dim
        self._kv_strides = (tuple(int(x) for x in kv_strides) if kv_strides is not None
                            else (num_kv_heads * P * d, P * d, d))
        h = ctypes.c_void_p()
        _abi.check(lib.rl_decode_attn_create(ctypes.byref(cfg), ctypes.byref(h)), "rl_decode_attn_create")
        self._lib, self._h, self.config = lib, h, cfg
        n = ctypes.c_size_t()
        _abi.check(lib.rl_decode_attn_workspace_size(h, ctypes.byref(n)), "rl_decode_attn_workspace_size")
        self.workspace_bytes = int(n.value)
        _abi.check(lib.rl_decode_attn_grouped_workspace_size(h, ctypes.byref(n)),
                   "rl_decode_attn_grouped_workspace_size")
        self.grouped_workspace_bytes = int(n.value)
        self._ws = {}

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self._lib.rl_decode_attn_destroy(h)
            self._h = None

    def workspace(self, device, grouped: bool = False):
        """Zero-filled workspace for `device`, allocated once and reused (grown once
        for grouped calls, which need more)."""
        torch = _torch()
        key = str(device)
        need = (self.grouped_workspace_bytes if grouped else self.workspace_bytes) + 256
        ws = self._ws.get(key)
        if ws is None or ws.numel() < need:
            ws = torch.zeros(need, dtype=torch.uint8, device=device)
            self._ws[key] = ws
        return ws

    # ---------------------------------------------------------------- argument checks
    # The kernels index the tensors by the handle's configuration; a tensor of the
    # wrong device, dtype, shape or layout is rejected here, before any launch.

    def _fail(self, what: str, msg: str):
        raise RldaError(-1, f"{what}: {msg}")

    def _tensor(self, what, name, t, dtype, shape, device, contiguous=True):
        if t is None:
            self._fail(what, f"{name} is required")
        if not t.is_cuda or t.device != device:
            self._fail(what, f"{name} must be on {device}, got {t.device}")
        if t.dtype != dtype:
            self._fail(what, f"{name} must be {dtype}, got {t.dtype}")
        if tuple(t.shape) != tuple(shape):
            self._fail(what, f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
        if contiguous and not t.is_contiguous():
            self._fail(what, f"{name} must be contiguous")

    def _check_cache(self, what, k_cache, v_cache, k_scale, v_scale, npages, device):
        cfg = self.config
        kvd = _torch_dtype(cfg.kv_dtype)
        for name, t in (("k_cache", k_cache), ("v_cache", v_cache)):
            if t is None:
                self._fail(what, f"{name} is required")
            if not t.is_cuda or t.device != device:
                self._fail(what, f"{name} must be on {device}, got {t.device}")
            if t.dtype != kvd:
                self._fail(what, f"{name} must be {kvd}, got {t.dtype}")
            if t.dim() != 4 or tuple(t.shape[1:]) != (cfg.num_kv_heads, cfg.page_size, cfg.head_dim):
                self._fail(what, f"{name} must be [pages, {cfg.num_kv_heads}, {cfg.page_size}, {cfg.head_dim}], "
                                 f"got {tuple(t.shape)}")
            # A dimension of size 1 is never stepped through, and torch may report any
            # stride for it (a single KV head of a [page][slot][head][d] cache, a
            # one-page pool), so only the strides of longer dimensions must match.
            want = self._kv_strides + (1,)
            if any(t.stride(i) != want[i] for i in range(4) if t.shape[i] > 1):
                self._fail(what, f"{name} strides {tuple(t.stride())} differ from the handle's {self._kv_strides} "
                                 "(head_dim contiguous)")
            if t.shape[0] < npages:
                self._fail(what, f"{name} holds {t.shape[0]} pages, fewer than num_pages = {npages}")
        if cfg.kv_dtype == _abi.RLDA_FP8_E4M3FN:
            torch = _torch()
            for name, t in (("k_scale", k_scale), ("v_scale", v_scale)):
                if t is None:
                    self._fail(what, f"{name} is required for fp8 caches")
                if t.dim() != 2 or t.shape[1] != cfg.num_kv_heads or t.shape[0] < npages:
                    self._fail(what, f"{name} must be [>= {npages}, {cfg.num_kv_heads}], got {tuple(t.shape)}")
                self._tensor(what, name, t, torch.float32, tuple(t.shape), device)

    def _check_rows(self, what, q, out, rows, device):
        cfg = self.config
        shape = (rows, cfg.num_q_heads, cfg.head_dim)
        self._tensor(what, "q", q, _torch_dtype(cfg.q_dtype), shape, device)
        self._tensor(what, "out", out, _torch_dtype(cfg.out_dtype), shape, device)

    def _check_table(self, what, block_table, seq_lens, batch, device):
        torch = _torch()
        if batch > self.config.max_batch:
            self._fail(what, f"batch {batch} exceeds max_batch {self.config.max_batch}")
        self._tensor(what, "block_table", block_table, torch.int32, (batch, self.config.max_pages_per_seq), device)
        self._tensor(what, "seq_lens", seq_lens, torch.int32, (batch,), device)

    def _check_workspace(self, what, ws, device):
        torch = _torch()
        if not ws.is_cuda or ws.device != device or ws.dtype != torch.uint8 or not ws.is_contiguous():
            self._fail(what, f"workspace must be a contiguous uint8 tensor on {device}")

    @staticmethod
    def _aligned_ptr(ws) -> int:
        p = ws.data_ptr()
        return (p + 255) // 256 * 256

    @staticmethod
    def _event_handle(ev) -> int:
        """Raw hipEvent_t of a torch.cuda.Event (created on first record)."""
        if not ev.cuda_event:
            ev.record()
        return ev.cuda_event

    def __call__(self, q, k_cache, v_cache, block_table, seq_lens, k_scale=None, v_scale=None, out=None,
                 workspace=None, stream=None, num_pages: Optional[int] = None, events=None,
                 group_size: Optional[int] = None, prefix_pages=None, prompt_pages_hint: int = -1):
        """Queue the attention on `stream` (default: the current stream).  With
        events=(begin, end) (torch.cuda.Event, timing enabled) the two events bracket
        the library's kernels.  With group_size and prefix_pages (int32 device tensor,
        one entry per group of group_size consecutive sequences) the call shares each
        group's prompt pages (rl_decode_attn_run_grouped); prompt_pages_hint (host value,
        e.g. the largest prefix_pages entry, <= 0 unknown) picks its packed or
        prompt-pass form."""
        torch = _torch()
        B = int(q.shape[0])
        cfg = self.config
        what = "rl_decode_attn_run_grouped" if group_size is not None else "rl_decode_attn_run"
        if not q.is_cuda:
            self._fail(what, f"q must be on a GPU, got {q.device}")
        if out is None:
            odt = torch.float32 if cfg.out_dtype == _abi.RLDA_F32 else torch.bfloat16
            out = torch.empty((B, cfg.num_q_heads, cfg.head_dim), dtype=odt, device=q.device)
        npages = int(k_cache.shape[0]) if num_pages is None else int(num_pages)
        self._check_rows(what, q, out, B, q.device)
        self._check_table(what, block_table, seq_lens, B, q.device)
        self._check_cache(what, k_cache, v_cache, k_scale, v_scale, npages, q.device)
        grouped = group_size is not None
        if grouped:
            if int(group_size) < 1:
                self._fail(what, "group_size must be >= 1")
            ng = (B + int(group_size) - 1) // int(group_size)
            self._tensor(what, "prefix_pages", prefix_pages, torch.int32, (ng,), q.device)
        ws = workspace if workspace is not None else self.workspace(q.device, grouped=grouped)
        self._check_workspace(what, ws, q.device)
        if stream is None:
            stream = torch.cuda.current_stream(q.device).cuda_stream
        elif hasattr(stream, "cuda_stream"):
            stream = stream.cuda_stream
        ptr = lambda t: None if t is None else t.data_ptr()
        wp = self._aligned_ptr(ws)
        args = (self._h, B, npages, ptr(q), ptr(k_cache), ptr(v_cache), ptr(k_scale), ptr(v_scale),
                ptr(block_table), ptr(seq_lens), ptr(out), wp, ws.numel() - (wp - ws.data_ptr()), stream)
        if grouped:
            e0, e1 = (None, None) if events is None else tuple(self._event_handle(e) for e in events)
            gargs = args[:3] + (int(group_size), ptr(prefix_pages), int(prompt_pages_hint)) + args[3:] + (e0, e1)
            _abi.check(self._lib.rl_decode_attn_run_grouped(*gargs), "rl_decode_attn_run_grouped")
        elif events is None:
            _abi.check(self._lib.rl_decode_attn_run(*args), "rl_decode_attn_run")
        else:
            e0, e1 = (self._event_handle(e) for e in events)
            _abi.check(self._lib.rl_decode_attn_run_profiled(*args, e0, e1), "rl_decode_attn_run_profiled")
        return out

    def run_noalloc(self, q, k_cache, v_cache, block_table, seq_lens, k_scale=None, v_scale=None, out=None,
                    flags=None, stream=None, num_pages: Optional[int] = None):
        """The same attention through rl_decode_attn_run_noalloc, which takes no
        workspace: its flags, segment counters and partials live in the library's static
        device array (limits: batch * Hkv <= 65536, head_dim <= 128).  `flags`: None, or
        a one-element int32 device tensor that receives the contract bits (OR-ed in)."""
        torch = _torch()
        B = int(q.shape[0])
        cfg = self.config
        what = "rl_decode_attn_run_noalloc"
        if not q.is_cuda:
            self._fail(what, f"q must be on a GPU, got {q.device}")
        if out is None:
            odt = torch.float32 if cfg.out_dtype == _abi.RLDA_F32 else torch.bfloat16
            out = torch.empty((B, cfg.num_q_heads, cfg.head_dim), dtype=odt, device=q.device)
        npages = int(k_cache.shape[0]) if num_pages is None else int(num_pages)
        self._check_rows(what, q, out, B, q.device)
        self._check_table(what, block_table, seq_lens, B, q.device)
        self._check_cache(what, k_cache, v_cache, k_scale, v_scale, npages, q.device)
        if flags is not None:
            self._tensor(what, "flags", flags, torch.int32, (1,), q.device)
        if stream is None:
            stream = torch.cuda.current_stream(q.device).cuda_stream
        elif hasattr(stream, "cuda_stream"):
            stream = stream.cuda_stream
        ptr = lambda t: None if t is None else t.data_ptr()
        _abi.check(self._lib.rl_decode_attn_run_noalloc(self._h, B, npages, ptr(q), ptr(k_cache), ptr(v_cache),
                                                        ptr(k_scale), ptr(v_scale), ptr(block_table), ptr(seq_lens),
                                                        ptr(out), ptr(flags), stream),
                   "rl_decode_attn_run_noalloc")
        return out

    def multi(self, q, k_cache, v_cache, block_table, seq_lens, q_start, k_scale=None, v_scale=None, out=None,
              workspace=None, stream=None, num_pages: Optional[int] = None, events=None, max_q_len: int = 0):
        """Multi-token queries (rl_decode_attn_run_multi): q [total_q][Hq][d], q_start
        [batch + 1] int32 device tensor; sequence b's rows q[q_start[b]:q_start[b+1]]
        are its last tokens and attend causally.  max_q_len (host value) bounds the
        rows per sequence; with max_q_len <= 16 and max_q_len * G <= 64 the decode
        kernel's page stream runs the call.  Returns out [total_q][Hq][d]."""
        torch = _torch()
        total = int(q.shape[0])
        B = int(q_start.shape[0]) - 1
        cfg = self.config
        what = "rl_decode_attn_run_multi"
        if not q.is_cuda:
            self._fail(what, f"q must be on a GPU, got {q.device}")
        if out is None:
            odt = torch.float32 if cfg.out_dtype == _abi.RLDA_F32 else torch.bfloat16
            out = torch.empty((total, cfg.num_q_heads, cfg.head_dim), dtype=odt, device=q.device)
        npages = int(k_cache.shape[0]) if num_pages is None else int(num_pages)
        self._check_rows(what, q, out, total, q.device)
        self._tensor(what, "q_start", q_start, torch.int32, (B + 1,), q.device)
        self._check_table(what, block_table, seq_lens, B, q.device)
        self._check_cache(what, k_cache, v_cache, k_scale, v_scale, npages, q.device)
        ws = workspace if workspace is not None else self.workspace(q.device)
        self._check_workspace(what, ws, q.device)
        if stream is None:
            stream = torch.cuda.current_stream(q.device).cuda_stream
        elif hasattr(stream, "cuda_stream"):
            stream = stream.cuda_stream
        ptr = lambda t: None if t is None else t.data_ptr()
        wp = self._aligned_ptr(ws)
        e0, e1 = (None, None) if events is None else tuple(self._event_handle(e) for e in events)
        _abi.check(self._lib.rl_decode_attn_run_multi(self._h, B, npages, total, int(max_q_len), ptr(q), ptr(k_cache),
                                                      ptr(v_cache),
                                                      ptr(k_scale), ptr(v_scale), ptr(block_table), ptr(seq_lens),
                                                      ptr(q_start), ptr(out), wp, ws.numel() - (wp - ws.data_ptr()),
                                                      stream, e0, e1),
                   "rl_decode_attn_run_multi")
        return out

    def append(self, k_new, v_new, k_cache, v_cache, block_table, seq_lens, k_scale=None, v_scale=None,
               workspace=None, stream=None, num_pages: Optional[int] = None):
        """Write one decode step's K/V rows ([B][Hkv][d], the q dtype) into the caches at
        token seq_lens[b] - 1 of every sequence (rl_decode_attn_append); fp8 caches also
        update their per-page scales."""
        torch = _torch()
        B = int(k_new.shape[0])
        cfg = self.config
        what = "rl_decode_attn_append"
        if not k_new.is_cuda:
            self._fail(what, f"k_new must be on a GPU, got {k_new.device}")
        dev = k_new.device
        npages = int(k_cache.shape[0]) if num_pages is None else int(num_pages)
        for name, t in (("k_new", k_new), ("v_new", v_new)):
            self._tensor(what, name, t, _torch_dtype(cfg.q_dtype), (B, cfg.num_kv_heads, cfg.head_dim), dev)
        self._check_table(what, block_table, seq_lens, B, dev)
        self._check_cache(what, k_cache, v_cache, k_scale, v_scale, npages, dev)
        ws = workspace if workspace is not None else self.workspace(dev)
        self._check_workspace(what, ws, dev)
        if stream is None:
            stream = torch.cuda.current_stream(dev).cuda_stream
        elif hasattr(stream, "cuda_stream"):
            stream = stream.cuda_stream
        ptr = lambda t: None if t is None else t.data_ptr()
        wp = self._aligned_ptr(ws)
        _abi.check(self._lib.rl_decode_attn_append(self._h, B, npages, ptr(k_new), ptr(v_new), ptr(k_cache),
                                                   ptr(v_cache), ptr(k_scale), ptr(v_scale), ptr(block_table),
                                                   ptr(seq_lens), wp, ws.numel() - (wp - ws.data_ptr()), stream),
                   "rl_decode_attn_append")

    def read_flags(self, workspace=None, device=None, stream=None) -> int:
        torch = _torch()
        ws = workspace if workspace is not None else self.workspace(device)
        if stream is None:
            stream = torch.cuda.current_stream(ws.device).cuda_stream
        v = ctypes.c_uint32()
        _abi.check(self._lib.rl_decode_attn_read_flags(self._h, self._aligned_ptr(ws), stream, ctypes.byref(v)),
                   "rl_decode_attn_read_flags")
        return int(v.value)


_handles = {}


def decode_attention(q, k_cache, v_cache, block_table, seq_lens, *, k_scale=None, v_scale=None,
                     kv_head_of_q=None, scale: float = 0.0, out=None, out_dtype=None, stream=None):
    """Functional form: q [B][Hq][d], caches [NP][Hkv][P][d] (d contiguous, any other
    strides), block_table [B][MP] int32, seq_lens [B] int32, fp8 scales [NP][Hkv]."""
    torch = _torch()
    NP, Hkv, P, d = k_cache.shape
    B, Hq = int(q.shape[0]), int(q.shape[1])
    if out_dtype is None:
        out_dtype = out.dtype if out is not None else torch.float32
    strides = tuple(int(s) for s in k_cache.stride()[:3])
    if tuple(v_cache.stride()[:3]) != strides or k_cache.stride(3) != 1:
        raise ValueError("k_cache and v_cache need identical strides with head_dim contiguous")
    hm = None if kv_head_of_q is None else tuple(int(x) for x in kv_head_of_q)
    key = (Hq, Hkv, d, P, int(block_table.shape[1]), q.dtype, k_cache.dtype, out_dtype, hm, float(scale), strides)
    h = _handles.get(key)
    if h is None or h.config.max_batch < B:
        h = DecodeAttention(Hq, Hkv, d, max(B, 1), int(block_table.shape[1]), q.dtype, k_cache.dtype, out_dtype,
                            kv_head_of_q=hm, softmax_scale=scale, kv_strides=strides, page_size=P)
        _handles[key] = h
    return h(q, k_cache, v_cache, block_table, seq_lens, k_scale=k_scale, v_scale=v_scale, out=out, stream=stream)
