"""Python binding of libspla.so, the SPLA decode-step C ABI (include/spla.h).

Argument marshalling only: every step of the append and decode paths runs in
the library's HIP kernels. PyTorch provides device memory and the stream
(the current torch stream of the tensors' device); nothing here computes.
The binding fails loudly when the HIP library has not been built.
"""

from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_float, c_int32, c_size_t, c_uint32, c_void_p
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libspla.so")
HOST_LIB_PATH = os.path.join(_HERE, "libspla_host.so")

F32, BF16 = 0, 1
FLAG_NO_RLA, FLAG_FIRST_ORDER, FLAG_RLA_NORMALIZE, FLAG_SEPARATE_KERNELS = 1, 2, 4, 8
DEVERR_CAPACITY, DEVERR_SYNC, DEVERR_PAGE = 1, 2, 4
MAX_GROUP, MAX_TOP_K, MAX_BLOCKS, WORKSPACE_ALIGN = 16, 256, 32768, 256
PHASES = {"append": 0, "score": 1, "select": 2, "sparse": 3, "merge": 4, "decode": 5,
          "linear": 6}
NUM_PHASES = 8
STATUS = {0: "ok", -1: "invalid argument", -2: "unsupported shape",
          -3: "capacity or library limit exceeded", -4: "workspace missing, too small or misaligned",
          -5: "HIP runtime error"}

# every symbol include/spla.h declares
HOST_EXPORTS = ["spla_status_string", "spla_phase_name", "spla_validate", "spla_cache_bytes",
                "spla_workspace_bytes", "spla_append_workspace_bytes", "spla_decode_phase_mask",
                "spla_prefill_workspace_bytes"]
EXPORTS = HOST_EXPORTS + ["spla_workspace_init", "spla_reset", "spla_append", "spla_decode",
                          "spla_decode_ex", "spla_step", "spla_step_ex", "spla_prefill",
                          "spla_prefill_ex", "spla_decode_noalloc"]


class SplaError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {STATUS.get(status, 'unknown status')} ({status})")
        self.status = status


class SplaConfig(ctypes.Structure):
    _fields_ = [("batch", c_int32), ("n_q_heads", c_int32), ("n_kv_heads", c_int32),
                ("head_dim", c_int32), ("block_size", c_int32), ("top_k", c_int32),
                ("n_sink_blocks", c_int32), ("n_local_blocks", c_int32),
                ("max_seq_len", c_int32), ("dtype", c_int32), ("softmax_scale", c_float),
                ("rms_eps", c_float), ("flags", c_uint32), ("sel_window", c_int32),
                ("sel_stride", c_int32), ("kv_pages", c_int32)]


class SplaCacheStruct(ctypes.Structure):
    _fields_ = [("k_cache", c_void_p), ("v_cache", c_void_p), ("blk_stats", c_void_p),
                ("lin_state", c_void_p), ("lin_norm", c_void_p), ("seq_lens", c_void_p),
                ("err_flags", c_void_p), ("block_table", c_void_p)]


class SplaEvents(ctypes.Structure):
    _fields_ = [("start", c_void_p * NUM_PHASES), ("stop", c_void_p * NUM_PHASES)]


def _declare(lib, host_only=False):
    cfgp = POINTER(SplaConfig)
    cachep = POINTER(SplaCacheStruct)
    lib.spla_status_string.restype = ctypes.c_char_p
    lib.spla_status_string.argtypes = [c_int32]
    lib.spla_phase_name.restype = ctypes.c_char_p
    lib.spla_phase_name.argtypes = [c_int32]
    lib.spla_validate.restype = c_int32
    lib.spla_validate.argtypes = [cfgp]
    lib.spla_cache_bytes.restype = c_int32
    lib.spla_cache_bytes.argtypes = [cfgp, POINTER(c_size_t)]
    lib.spla_workspace_bytes.restype = c_int32
    lib.spla_workspace_bytes.argtypes = [cfgp, POINTER(c_size_t)]
    lib.spla_append_workspace_bytes.restype = c_int32
    lib.spla_append_workspace_bytes.argtypes = [cfgp, c_int32, POINTER(c_size_t)]
    lib.spla_decode_phase_mask.restype = c_int32
    lib.spla_decode_phase_mask.argtypes = [cfgp, POINTER(c_uint32)]
    lib.spla_prefill_workspace_bytes.restype = c_int32
    lib.spla_prefill_workspace_bytes.argtypes = [cfgp, c_int32, POINTER(c_size_t)]
    if host_only:
        return lib
    lib.spla_workspace_init.restype = c_int32
    lib.spla_workspace_init.argtypes = [cfgp, c_void_p, c_size_t, c_void_p]
    lib.spla_reset.restype = c_int32
    lib.spla_reset.argtypes = [cfgp, cachep, c_void_p]
    lib.spla_append.restype = c_int32
    lib.spla_append.argtypes = [cfgp, cachep, c_void_p, c_void_p, c_int32, c_void_p, c_void_p,
                                c_size_t, c_void_p]
    lib.spla_decode.restype = c_int32
    lib.spla_decode.argtypes = [cfgp, cachep, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                c_size_t, c_void_p]
    lib.spla_decode_ex.restype = c_int32
    lib.spla_decode_ex.argtypes = [cfgp, cachep, c_void_p, c_void_p, c_void_p, c_void_p,
                                   c_void_p, c_size_t, POINTER(SplaEvents), c_void_p]
    lib.spla_step.restype = c_int32
    lib.spla_step.argtypes = [cfgp, cachep, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                              c_void_p, c_void_p, c_size_t, c_void_p]
    lib.spla_step_ex.restype = c_int32
    lib.spla_step_ex.argtypes = [cfgp, cachep, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                 c_void_p, c_void_p, c_size_t, POINTER(SplaEvents), c_void_p]
    lib.spla_prefill_ex.restype = c_int32
    lib.spla_prefill_ex.argtypes = [cfgp, cachep, c_int32, c_void_p, c_void_p, c_void_p,
                                    c_void_p, c_void_p, c_void_p, c_void_p, c_size_t,
                                    POINTER(SplaEvents), c_void_p]
    lib.spla_decode_noalloc.restype = c_int32
    lib.spla_decode_noalloc.argtypes = [cfgp, cachep, c_void_p, c_void_p, c_void_p, c_void_p,
                                        c_void_p]
    lib.spla_prefill.restype = c_int32
    lib.spla_prefill.argtypes = [cfgp, cachep, c_int32, c_void_p, c_void_p, c_void_p, c_void_p,
                                 c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]
    return lib


_LIB = None
_HOST_LIB = None


def lib():
    """The HIP library (raises ImportError if it has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2601_22379_amd.build`")
        _LIB = _declare(ctypes.CDLL(LIB_PATH))
    return _LIB


def host_lib():
    """The host-only validation library (loads without a GPU or HIP runtime)."""
    global _HOST_LIB
    if _HOST_LIB is None:
        if not os.path.exists(HOST_LIB_PATH):
            raise ImportError(f"{HOST_LIB_PATH} is missing: build it with "
                              "`python -m paper_2601_22379_amd.build --host-only`")
        _HOST_LIB = _declare(ctypes.CDLL(HOST_LIB_PATH), host_only=True)
    return _HOST_LIB


def _check(status: int, where: str):
    if status != 0:
        raise SplaError(status, where)


def make_config(batch, n_q_heads, n_kv_heads, head_dim, block_size, top_k, max_seq_len,
                dtype="bf16", n_sink=1, n_local=4, softmax_scale=0.0, rms_eps=1e-6,
                flags=0, sel_window=0, sel_stride=0, kv_pages=0) -> SplaConfig:
    dt = {"f32": F32, "fp32": F32, "float32": F32, "bf16": BF16, "bfloat16": BF16}.get(dtype, dtype)
    return SplaConfig(batch, n_q_heads, n_kv_heads, head_dim, block_size, top_k, n_sink, n_local,
                      max_seq_len, int(dt), float(softmax_scale), float(rms_eps), int(flags),
                      int(sel_window), int(sel_stride), int(kv_pages))


def validate(cfg: SplaConfig, library=None) -> int:
    return int((library or lib()).spla_validate(ctypes.byref(cfg)))


def cache_bytes(cfg: SplaConfig, library=None) -> list:
    out = (c_size_t * 6)()
    _check((library or lib()).spla_cache_bytes(ctypes.byref(cfg), out), "spla_cache_bytes")
    return list(out)


def workspace_bytes(cfg: SplaConfig, library=None) -> int:
    n = c_size_t(0)
    _check((library or lib()).spla_workspace_bytes(ctypes.byref(cfg), ctypes.byref(n)),
           "spla_workspace_bytes")
    return int(n.value)


def append_workspace_bytes(cfg: SplaConfig, max_new: int, library=None) -> int:
    n = c_size_t(0)
    _check((library or lib()).spla_append_workspace_bytes(ctypes.byref(cfg), int(max_new),
                                                          ctypes.byref(n)),
           "spla_append_workspace_bytes")
    return int(n.value)


def prefill_workspace_bytes(cfg: SplaConfig, n_tokens: int, library=None) -> int:
    n = c_size_t(0)
    _check((library or lib()).spla_prefill_workspace_bytes(ctypes.byref(cfg), int(n_tokens),
                                                           ctypes.byref(n)),
           "spla_prefill_workspace_bytes")
    return int(n.value)


def decode_phases(cfg: SplaConfig, library=None) -> list:
    """Names of the phases whose events spla_decode_ex records for cfg."""
    mask = c_uint32(0)
    _check((library or lib()).spla_decode_phase_mask(ctypes.byref(cfg), ctypes.byref(mask)),
           "spla_decode_phase_mask")
    return [n for n, p in PHASES.items() if mask.value >> p & 1]


def torch_dtype(cfg: SplaConfig):
    return torch.float32 if cfg.dtype == F32 else torch.bfloat16


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else c_void_p(t.data_ptr())


def _stream(device) -> c_void_p:
    return c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _aligned_workspace(nbytes: int, device) -> torch.Tensor:
    # torch's caching allocator returns 512-byte aligned blocks
    t = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)
    assert t.data_ptr() % WORKSPACE_ALIGN == 0
    return t


class SplaCache:
    """Device buffers of one SPLA cache, allocated with torch, plus the
    workspaces the calls need. Thin wrapper over the C ABI."""

    def __init__(self, cfg: SplaConfig, device="cuda", block_table: Optional[torch.Tensor] = None):
        """block_table: int32 [batch, max_seq_len / block_size] on the device,
        page of each block, required when cfg.kv_pages > 0 (paged pool)."""
        self.cfg = cfg
        self.device = torch.device(device)
        if (cfg.kv_pages > 0) != (block_table is not None):
            raise ValueError("a block table goes with kv_pages > 0, and only then")
        if block_table is not None:
            assert block_table.dtype == torch.int32 and block_table.is_contiguous()
            assert block_table.shape == (cfg.batch, cfg.max_seq_len // cfg.block_size)
            assert block_table.device == self.device
        self.block_table = block_table
        sz = cache_bytes(cfg)
        dt = torch_dtype(cfg)
        e = 4 if cfg.dtype == F32 else 2
        self.k = torch.zeros(sz[0] // e, dtype=dt, device=self.device)
        self.v = torch.zeros(sz[1] // e, dtype=dt, device=self.device)
        self.stats = torch.zeros(sz[2] // 4, dtype=torch.float32, device=self.device)
        self.state = torch.zeros(sz[3] // 4, dtype=torch.float32, device=self.device)
        self.norm = torch.zeros(sz[4] // 4, dtype=torch.float32, device=self.device)
        self.seq_lens = torch.zeros(cfg.batch, dtype=torch.int32, device=self.device)
        self.err = torch.zeros(1, dtype=torch.int32, device=self.device)
        self.workspace = _aligned_workspace(workspace_bytes(cfg), self.device)
        _check(lib().spla_workspace_init(ctypes.byref(cfg), _ptr(self.workspace),
                                         self.workspace.numel(), _stream(self.device)),
               "spla_workspace_init")
        self._append_ws = None
        self._prefill_ws = None
        self._struct = SplaCacheStruct(self.k.data_ptr(), self.v.data_ptr(),
                                       self.stats.data_ptr(), self.state.data_ptr(),
                                       self.norm.data_ptr(), self.seq_lens.data_ptr(),
                                       self.err.data_ptr(),
                                       None if block_table is None else block_table.data_ptr())

    @property
    def struct(self) -> SplaCacheStruct:
        return self._struct

    def device_errors(self) -> int:
        """The SPLA_DEVERR_* bits the device has set in this cache's error
        word (waits for the work queued on the current stream)."""
        return int(self.err.item())

    def clear_device_errors(self):
        self.err.zero_()

    def check_device_errors(self, allowed: int = 0):
        """Raises SplaError when a bit outside `allowed` is set: after a
        SPLA_DEVERR_SYNC the outputs of the call that set it are undefined."""
        e = self.device_errors()
        if e & ~allowed:
            names = [n for n, v in (("CAPACITY", DEVERR_CAPACITY), ("SYNC", DEVERR_SYNC),
                                    ("PAGE", DEVERR_PAGE)) if e & v]
            raise SplaError(-5, "device error word: " + "|".join(names))

    def reset(self):
        _check(lib().spla_reset(ctypes.byref(self.cfg), ctypes.byref(self._struct),
                                _stream(self.device)), "spla_reset")

    def append(self, k_new: torch.Tensor, v_new: torch.Tensor,
               n_new: Optional[torch.Tensor] = None):
        """k_new, v_new: [batch, Hkv, max_new, d] in the cache dtype."""
        c = self.cfg
        assert k_new.shape == v_new.shape and k_new.dim() == 4
        assert k_new.shape[0] == c.batch and k_new.shape[1] == c.n_kv_heads
        assert k_new.shape[3] == c.head_dim
        assert k_new.dtype == torch_dtype(c) and v_new.dtype == torch_dtype(c)
        assert k_new.is_contiguous() and v_new.is_contiguous()
        max_new = int(k_new.shape[2])
        need = append_workspace_bytes(c, max_new)
        if self._append_ws is None or self._append_ws.numel() < need:
            self._append_ws = _aligned_workspace(need, self.device)
        if n_new is not None:
            assert n_new.dtype == torch.int32 and n_new.numel() == c.batch and n_new.is_contiguous()
        _check(lib().spla_append(ctypes.byref(c), ctypes.byref(self._struct), _ptr(k_new),
                                 _ptr(v_new), max_new, _ptr(n_new), _ptr(self._append_ws),
                                 self._append_ws.numel(), _stream(self.device)), "spla_append")

    def _decode_args(self, q, gamma, out, sel):
        c = self.cfg
        assert q.shape == (c.batch, c.n_q_heads, c.head_dim) and q.dtype == torch_dtype(c)
        assert q.is_contiguous()
        assert gamma.shape == (c.n_q_heads, c.head_dim) and gamma.dtype == torch.float32
        assert gamma.is_contiguous()
        if out is None:
            out = torch.empty_like(q)
        if sel is None:
            sel = torch.empty((c.batch, c.n_kv_heads, c.top_k), dtype=torch.int32,
                              device=self.device)
        return out, sel

    def decode(self, q: torch.Tensor, gamma: torch.Tensor, out=None, sel=None, events=None):
        """q [batch, Hq, d] (cache dtype), gamma [Hq, d] fp32 -> (out, sel)."""
        out, sel = self._decode_args(q, gamma, out, sel)
        ev = None if events is None else ctypes.byref(events)
        _check(lib().spla_decode_ex(ctypes.byref(self.cfg), ctypes.byref(self._struct), _ptr(q),
                                    _ptr(gamma), _ptr(out), _ptr(sel), _ptr(self.workspace),
                                    self.workspace.numel(), ev, _stream(self.device)),
               "spla_decode")
        return out, sel

    def decode_noalloc(self, q: torch.Tensor, gamma: torch.Tensor, out, sel=None):
        """spla_decode_noalloc: the decode on the library's own device scratch
        (no workspace); out must be given (nothing is allocated here either)."""
        c = self.cfg
        assert q.shape == (c.batch, c.n_q_heads, c.head_dim) and q.dtype == torch_dtype(c)
        assert gamma.shape == (c.n_q_heads, c.head_dim) and gamma.dtype == torch.float32
        assert out is not None and out.shape == q.shape and out.dtype == q.dtype
        assert q.is_contiguous() and gamma.is_contiguous() and out.is_contiguous()
        if sel is not None:
            assert sel.shape == (c.batch, c.n_kv_heads, c.top_k) and sel.dtype == torch.int32
            assert sel.is_contiguous()
        _check(lib().spla_decode_noalloc(ctypes.byref(c), ctypes.byref(self._struct), _ptr(q),
                                         _ptr(gamma), _ptr(out), _ptr(sel),
                                         _stream(self.device)), "spla_decode_noalloc")
        return out, sel

    def step(self, k_new, v_new, q, gamma, out=None, sel=None, events=None):
        """Append one token per (sequence, KV head) ([batch, Hkv, d]), then decode."""
        c = self.cfg
        assert k_new.shape == (c.batch, c.n_kv_heads, c.head_dim) and k_new.is_contiguous()
        assert v_new.shape == k_new.shape and v_new.is_contiguous()
        assert k_new.dtype == torch_dtype(c) and v_new.dtype == torch_dtype(c)
        out, sel = self._decode_args(q, gamma, out, sel)
        ev = None if events is None else ctypes.byref(events)
        _check(lib().spla_step_ex(ctypes.byref(c), ctypes.byref(self._struct), _ptr(k_new),
                                  _ptr(v_new), _ptr(q), _ptr(gamma), _ptr(out), _ptr(sel),
                                  _ptr(self.workspace), self.workspace.numel(), ev,
                                  _stream(self.device)), "spla_step")
        return out, sel

    def prefill(self, k_new, v_new, q, gamma, out=None, sel=None, events=None):
        """Causal prefill of T tokens per sequence: k_new, v_new [T, batch,
        Hkv, d], q [T, batch, Hq, d] (cache dtype) -> out [T, batch, Hq, d],
        sel [T, batch, Hkv, top_k]; position t is appended, then decoded."""
        c = self.cfg
        T = k_new.shape[0]
        assert k_new.shape == (T, c.batch, c.n_kv_heads, c.head_dim) and k_new.is_contiguous()
        assert v_new.shape == k_new.shape and v_new.is_contiguous()
        assert k_new.dtype == torch_dtype(c) and v_new.dtype == torch_dtype(c)
        assert q.shape == (T, c.batch, c.n_q_heads, c.head_dim) and q.dtype == torch_dtype(c)
        assert q.is_contiguous()
        assert gamma.shape == (c.n_q_heads, c.head_dim) and gamma.dtype == torch.float32
        if out is None:
            out = torch.empty_like(q)
        if sel is None:
            sel = torch.empty((T, c.batch, c.n_kv_heads, c.top_k), dtype=torch.int32,
                              device=self.device)
        need = prefill_workspace_bytes(c, T)
        if self._prefill_ws is None or self._prefill_ws.numel() < need:
            self._prefill_ws = _aligned_workspace(need, self.device)
        ws = self._prefill_ws
        ev = None if events is None else ctypes.byref(events)
        _check(lib().spla_prefill_ex(ctypes.byref(c), ctypes.byref(self._struct), int(T),
                                     _ptr(k_new), _ptr(v_new), _ptr(q), _ptr(gamma), _ptr(out),
                                     _ptr(sel), _ptr(ws), ws.numel(), ev,
                                     _stream(self.device)), "spla_prefill")
        return out, sel

    # ---- layout views (for checks; pure indexing) ----
    def stats_logical(self):
        """(mean, M2) as [batch, Hkv, n_units, d] fp32 tensors: one unit per
        block, or per selection window with strided selection."""
        c = self.cfg
        nb = c.max_seq_len // (c.sel_stride if c.sel_stride else c.block_size)
        nt = -(-nb // 64)
        s = self.stats.view(c.batch, c.n_kv_heads, nt, 2, c.head_dim // 4, 64, 4)
        s = s.permute(0, 1, 3, 2, 5, 4, 6).reshape(c.batch, c.n_kv_heads, 2, nt * 64, c.head_dim)
        return s[:, :, 0, :nb], s[:, :, 1, :nb]

    def _per_sequence(self, pool):
        """A K or V buffer in the per-sequence layout ([batch][Hkv][nb][B d]):
        the buffer itself, or the pages of a paged pool gathered through the
        block table (entries outside the pool give zeros)."""
        c = self.cfg
        if c.kv_pages == 0:
            return pool
        bd = c.block_size * c.head_dim
        pages = pool.view(c.kv_pages, c.n_kv_heads, bd)
        tab = self.block_table.long()
        ok = (tab >= 0) & (tab < c.kv_pages)
        g = pages[tab.clamp(0, c.kv_pages - 1)] * ok[..., None, None].to(pool.dtype)
        return g.permute(0, 2, 1, 3).contiguous().view(-1)

    def k_logical(self):
        """Keys as [batch][Hkv][max_seq_len][d] (undoing the bf16 step order)."""
        c = self.cfg
        B, H, T, d = c.batch, c.n_kv_heads, c.max_seq_len, c.head_dim
        kbuf = self._per_sequence(self.k)
        if c.dtype == F32:
            return kbuf.view(B, H, T, d)
        # step chunk (mt, ks, g, a, b) holds token 8a + 4mt + b, coordinates 32ks + 8g ..
        k = kbuf.view(B, H, T // 32, 2, d // 32, 4, 4, 4, 8)
        return k.permute(0, 1, 2, 6, 3, 7, 4, 5, 8).reshape(B, H, T, d)

    def v_logical(self):
        """Values as [batch][Hkv][max_seq_len][d] (undoing the block transpose
        of fp32 caches and the step order of bf16 ones)."""
        c = self.cfg
        B, H, T, d = c.batch, c.n_kv_heads, c.max_seq_len, c.head_dim
        vbuf = self._per_sequence(self.v)
        if c.dtype == F32:
            v = vbuf.view(B, H, T // c.block_size, d, c.block_size)
            return v.permute(0, 1, 2, 4, 3).reshape(B, H, T, d)
        # step chunk (t, g, i) holds coordinate 16t + i, tokens 8g .. 8g + 7
        v = vbuf.view(B, H, T // 32, d // 16, 4, 16, 8)
        return v.permute(0, 1, 2, 4, 6, 3, 5).reshape(B, H, T, d)

    def state_logical(self):
        c = self.cfg
        return (self.state.view(c.batch, c.n_kv_heads, c.head_dim, c.head_dim),
                self.norm.view(c.batch, c.n_kv_heads, c.head_dim))


def make_events(phases: Sequence[str] = ("score", "select", "sparse", "merge", "decode",
                                        "append")):
    """torch.cuda.Event pairs for the given phases, and the SplaEvents that
    points at their HIP events. Returns (events_struct, {phase: (start, stop)})."""
    ev = SplaEvents()
    pairs = {}
    for name in phases:
        p = PHASES[name]
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        b.record()   # materialise the underlying events
        ev.start[p] = c_void_p(a.cuda_event)
        ev.stop[p] = c_void_p(b.cuda_event)
        pairs[name] = (a, b)
    return ev, pairs
