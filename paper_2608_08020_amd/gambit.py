"""Python binding of libgambit (ctypes).  Argument marshalling only.

Every step of the hot path runs in the library's HIP kernels; this module
allocates the caller-owned device buffers with torch and passes pointers
and the current HIP stream.  Method names follow the C entry points in
include/gambit.h without the ``gambit_`` prefix.  There is no fallback: a
missing library raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch  # loads the HIP runtime that libgambit binds to

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgambit.so")

OK, ERR_INVALID, ERR_OUT_OF_BLOCKS, ERR_SHARED_WRITE, ERR_UNSUPPORTED, ERR_DEVICE, ERR_WORKSPACE = (
    0, -1, -2, -3, -4, -5, -6)
KV_BF16, KV_FP8_E4M3 = 0, 1
OUT_BF16, OUT_F32 = 0, 1
NEW_CACHE, NEW_BF16 = 0, 1
UNIT_NARROW, UNIT_COOP_ONE, UNIT_COOP_TWO, UNIT_TAIL_SLOT, UNIT_NARROW_TWO = 1, 2, 4, 16, 32
CODE_NAMES = {ERR_INVALID: "INVALID", ERR_OUT_OF_BLOCKS: "OUT_OF_BLOCKS",
              ERR_SHARED_WRITE: "SHARED_WRITE", ERR_UNSUPPORTED: "UNSUPPORTED",
              ERR_DEVICE: "DEVICE", ERR_WORKSPACE: "WORKSPACE"}
MAX_RANK = 4096


class GambitError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{CODE_NAMES.get(status, status)}: {msg}")
        self.status = status
        self.code = CODE_NAMES.get(status, str(status))


class PoolDesc(ctypes.Structure):
    _fields_ = [("num_blocks", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("kv_dtype", ctypes.c_int32),
                ("max_traces", ctypes.c_int32), ("max_blocks_per_trace", ctypes.c_int32),
                ("max_splits", ctypes.c_int32), ("fp8_append_scale", ctypes.c_float),
                ("num_layers", ctypes.c_int32),
                ("k_cache", ctypes.c_void_p), ("v_cache", ctypes.c_void_p),
                ("kv_scale", ctypes.c_void_p), ("block_table", ctypes.c_void_p),
                ("seq_len", ctypes.c_void_p), ("refcount", ctypes.c_void_p),
                ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t)]


class Round(ctypes.Structure):
    _fields_ = [("case_taken", ctypes.c_int32), ("n_active", ctypes.c_int32),
                ("n_pruned", ctypes.c_int32), ("n_children", ctypes.c_int32)]


class Mlp(ctypes.Structure):
    _fields_ = [("dim", ctypes.c_int32), ("hidden", ctypes.c_int32), ("activation", ctypes.c_int32),
                ("w1", ctypes.c_void_p), ("b1", ctypes.c_void_p), ("w2", ctypes.c_void_p),
                ("b2", ctypes.c_float)]


ACT_RELU, ACT_GELU = 0, 1


class ScorerDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("input_dim", "d_model", "n_heads", "n_layers", "d_ff", "max_steps",
                                              "max_traces")] + \
               [(n, ctypes.c_void_p) for n in ("ln_in_g", "ln_in_b", "w_in", "ln1_g", "ln1_b", "w_qkv", "w_o",
                                               "ln2_g", "ln2_b", "w_13", "w_2", "ln_out_g", "ln_out_b", "w_out",
                                               "workspace")] + \
               [("workspace_bytes", ctypes.c_size_t)]


class Stats(ctypes.Structure):
    _fields_ = [("total_tokens", ctypes.c_int64), ("unique_tokens", ctypes.c_int64),
                ("unique_blocks", ctypes.c_int64), ("table_entries", ctypes.c_int64),
                ("n_units", ctypes.c_int32),
                ("max_splits_used", ctypes.c_int32)]


_lib = None
EXPORTS = ["gambit_workspace_size", "gambit_pool_create", "gambit_pool_destroy", "gambit_kv_alloc",
           "gambit_kv_write", "gambit_kv_fork", "gambit_kv_free", "gambit_decode_attn", "gambit_decode_attn_layer",
           "gambit_score_prune_branch", "gambit_rank_topk", "gambit_pool_check",
           "gambit_plan_stats", "gambit_seq_len", "gambit_free_blocks", "gambit_status_str",
           "gambit_last_error", "gambit_profile_begin", "gambit_profile_end", "gambit_score_update",
           "gambit_evict", "gambit_tournament", "gambit_trace_state", "gambit_record_scores",
           "gambit_mlp_workspace_size", "gambit_mlp_score", "gambit_scorer_workspace_size", "gambit_scorer_create",
           "gambit_scorer_destroy", "gambit_scorer_step", "gambit_scorer_fork", "gambit_scorer_free",
           "gambit_scorer_steps", "gambit_scorer_check", "gambit_scorer_last_error", "gambit_stream_read",
           "gambit_plan_kinds", "gambit_mlp_score_static"]


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2608_08020_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float
    sig = {
        "gambit_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(PoolDesc)]),
        "gambit_pool_create": (i32, [ctypes.POINTER(PoolDesc), vp, ctypes.POINTER(vp)]),
        "gambit_pool_destroy": (i32, [vp]),
        "gambit_kv_alloc": (i32, [vp, i32, vp, vp, vp]),
        "gambit_kv_write": (i32, [vp, i32, i32, i32, vp, vp, vp, vp]),
        "gambit_kv_fork": (i32, [vp, i32, vp, vp, vp]),
        "gambit_kv_free": (i32, [vp, i32, vp, vp]),
        "gambit_decode_attn": (i32, [vp, i32, vp, vp, vp, vp, vp, i32, f32, vp]),
        "gambit_decode_attn_layer": (i32, [vp, i32, i32, vp, vp, vp, vp, i32, vp, i32, f32, vp]),
        "gambit_score_prune_branch": (i32, [vp, i32, vp, vp, i32, vp, f32, i32, i32, vp, vp, vp, vp]),
        "gambit_rank_topk": (i32, [i32, vp, vp, i32, vp, vp]),
        "gambit_pool_check": (i32, [vp, vp]),
        "gambit_plan_stats": (i32, [vp, i32, vp, ctypes.POINTER(Stats)]),
        "gambit_seq_len": (i32, [vp, i32]),
        "gambit_free_blocks": (i32, [vp]),
        "gambit_status_str": (ctypes.c_char_p, [i32]),
        "gambit_last_error": (ctypes.c_char_p, [vp]),
        "gambit_profile_begin": (i32, [vp, i32]),
        "gambit_profile_end": (i32, [vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i32)]),
        "gambit_score_update": (i32, [vp, i32, vp, vp, i32, vp, f32, vp, vp]),
        "gambit_evict": (i32, [vp, i32, vp, vp, vp]),
        "gambit_tournament": (i32, [vp, i32, i32, i32, ctypes.POINTER(Round), vp, vp, vp, vp]),
        "gambit_trace_state": (i32, [vp, i32, vp, vp, vp, vp, vp, vp]),
        "gambit_record_scores": (i32, [vp, i32, vp, vp, vp]),
        "gambit_mlp_workspace_size": (ctypes.c_size_t, [i32, i32]),
        "gambit_mlp_score": (i32, [i32, vp, ctypes.POINTER(Mlp), vp, vp, i32, vp, vp, ctypes.c_size_t, vp]),
        "gambit_scorer_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(ScorerDesc)]),
        "gambit_scorer_create": (i32, [ctypes.POINTER(ScorerDesc), vp, ctypes.POINTER(vp)]),
        "gambit_scorer_destroy": (i32, [vp]),
        "gambit_scorer_step": (i32, [vp, i32, vp, vp, vp, vp]),
        "gambit_scorer_fork": (i32, [vp, i32, vp, vp, vp]),
        "gambit_scorer_free": (i32, [vp, i32, vp, vp]),
        "gambit_scorer_steps": (i32, [vp, i32]),
        "gambit_scorer_check": (i32, [vp, vp]),
        "gambit_scorer_last_error": (ctypes.c_char_p, [vp]),
        "gambit_stream_read": (i32, [vp, ctypes.c_size_t, i32, i32, vp, vp]),
        "gambit_plan_kinds": (i32, [vp, i32, vp, vp]),
        "gambit_mlp_score_static": (i32, [i32, vp, ctypes.POINTER(Mlp), vp, vp, i32, vp, vp]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype, fn.argtypes = res, args
    _lib = L
    return L


def workspace_size(desc: PoolDesc) -> int:
    return int(lib().gambit_workspace_size(ctypes.byref(desc)))


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _host_i32(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32))


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _spec(t: torch.Tensor, dtype=None, shape=None, what: str = "tensor"):
    """Check a tensor argument's dtype(s), shape and contiguity.  The kernels
    trust these sizes (the C ABI takes bare pointers), so every device
    argument of an entry point is checked before the library sees any."""
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{what}: expected a tensor, got {type(t).__name__}")
    if dtype is not None:
        ok = t.dtype in dtype if isinstance(dtype, tuple) else t.dtype == dtype
        if not ok:
            raise ValueError(f"{what}: expected dtype {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{what}: expected shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{what}: expected a contiguous tensor")


def _dev(t: torch.Tensor, dtype=None, shape=None, what: str = "tensor"):
    """Pointer of a contiguous device tensor (checked as by _spec)."""
    _spec(t, dtype, shape, what)
    if not t.is_cuda:
        raise ValueError(f"{what}: expected a device tensor")
    return ctypes.c_void_p(t.data_ptr())


def rank_topk(ids: torch.Tensor, scores: torch.Tensor, keep: int, stream=None) -> torch.Tensor:
    """gambit_rank_topk: ids of the top `keep` by (score desc, id asc), on the device."""
    n = ids.numel()
    _spec(ids, torch.int32, (n,), "ids")
    _spec(scores, torch.float32, (n,), "scores")
    out = torch.empty(keep, dtype=torch.int32, device=ids.device)
    st = lib().gambit_rank_topk(n, _dev(ids), _dev(scores), keep, _dev(out), _stream(stream))
    if st != OK:
        raise GambitError(st, "rank_topk")
    return out


def mlp_score(h: torch.Tensor, w1: torch.Tensor, b1: torch.Tensor, w2: torch.Tensor, b2: float,
              activation: str = "relu", ids: torch.Tensor | None = None, keep: int = 0, stream=None):
    """gambit_mlp_score: (scores [n] fp32, top-`keep` ids or None), on the device."""
    if h.dim() != 2 or w1.dim() != 2:
        raise ValueError("h: expected [n][dim], w1: expected [hidden][dim]")
    n, dim = h.shape
    hidden = w1.shape[0]
    _spec(h, torch.bfloat16, (n, dim), "h")
    _spec(w1, torch.bfloat16, (hidden, dim), "w1")
    _spec(b1, torch.float32, (hidden,), "b1")
    _spec(w2, torch.float32, (hidden,), "w2")
    if activation not in ("relu", "gelu"):
        raise ValueError(f"activation: {activation!r}")
    if keep > 0 and ids is None:
        raise ValueError("ids: needed when keep > 0")
    if ids is not None:
        _spec(ids, torch.int32, (n,), "ids")
    m = Mlp(dim, hidden, ACT_RELU if activation == "relu" else ACT_GELU, _dev(w1).value, _dev(b1).value,
            _dev(w2).value, float(b2))
    ws_bytes = int(lib().gambit_mlp_workspace_size(n, hidden))
    ws = torch.empty(max(ws_bytes, 4), dtype=torch.uint8, device=h.device)
    scores = torch.empty(n, dtype=torch.float32, device=h.device)
    keep_out = torch.empty(max(keep, 1), dtype=torch.int32, device=h.device)
    st = lib().gambit_mlp_score(n, _dev(h, torch.bfloat16), ctypes.byref(m), _dev(scores),
                                None if ids is None else _dev(ids, torch.int32), keep, _dev(keep_out), _dev(ws),
                                ws_bytes, _stream(stream))
    if st != OK:
        raise GambitError(st, "mlp_score")
    return scores, (keep_out[:keep] if keep > 0 else None)


MLP_STATIC_SCRATCH_BYTES = 16 << 20


def mlp_score_static(h: torch.Tensor, w1: torch.Tensor, b1: torch.Tensor, w2: torch.Tensor, b2: float,
                     activation: str = "relu", ids: torch.Tensor | None = None, keep: int = 0,
                     scores_out: torch.Tensor | None = None, keep_out: torch.Tensor | None = None, stream=None):
    """gambit_mlp_score_static: as mlp_score, with the library's own device
    scratch instead of a workspace (no device allocation inside the call when
    the outputs are passed in)."""
    if h.dim() != 2 or w1.dim() != 2:
        raise ValueError("h: expected [n][dim], w1: expected [hidden][dim]")
    n, dim = h.shape
    hidden = w1.shape[0]
    _spec(h, torch.bfloat16, (n, dim), "h")
    _spec(w1, torch.bfloat16, (hidden, dim), "w1")
    _spec(b1, torch.float32, (hidden,), "b1")
    _spec(w2, torch.float32, (hidden,), "w2")
    if activation not in ("relu", "gelu"):
        raise ValueError(f"activation: {activation!r}")
    if keep > 0 and ids is None:
        raise ValueError("ids: needed when keep > 0")
    if ids is not None:
        _spec(ids, torch.int32, (n,), "ids")
    if scores_out is None:
        scores_out = torch.empty(n, dtype=torch.float32, device=h.device)
    _spec(scores_out, torch.float32, (n,), "scores_out")
    if keep > 0:
        if keep_out is None:
            keep_out = torch.empty(keep, dtype=torch.int32, device=h.device)
        _spec(keep_out, torch.int32, (keep,), "keep_out")
    m = Mlp(dim, hidden, ACT_RELU if activation == "relu" else ACT_GELU, _dev(w1).value, _dev(b1).value,
            _dev(w2).value, float(b2))
    st = lib().gambit_mlp_score_static(n, _dev(h), ctypes.byref(m), _dev(scores_out),
                                       None if ids is None else _dev(ids), keep,
                                       _dev(keep_out) if keep > 0 else None, _stream(stream))
    if st != OK:
        raise GambitError(st, "mlp_score_static")
    return scores_out, (keep_out if keep > 0 else None)


def stream_read(buf: torch.Tensor, nontemporal: bool, grid: int, sink: torch.Tensor, stream=None) -> None:
    """gambit_stream_read: read every byte of buf once (timing of the memory
    system's read rate); sink (int32, zeroed, >= grid entries) receives each
    workgroup's XOR of the dwords it read."""
    if not buf.is_contiguous() or sink.dtype != torch.int32 or sink.numel() < grid:
        raise ValueError("buf must be contiguous; sink int32 with >= grid entries")
    st = lib().gambit_stream_read(buf.data_ptr(), buf.numel() * buf.element_size(), int(bool(nontemporal)),
                                  int(grid), sink.data_ptr(), _stream(stream))
    if st != OK:
        raise GambitError(st, "stream_read")


class Pool:
    """A refcounted paged KV pool on one GPU; all buffers are torch tensors."""

    def __init__(self, *, num_blocks: int, num_q_heads: int, num_kv_heads: int,
                 max_traces: int, max_blocks_per_trace: int, kv_dtype: str = "bf16",
                 head_dim: int = 128, max_splits: int = 0, fp8_append_scale: float = 0.0,
                 num_layers: int = 1, device: str = "cuda", stream=None):
        fp8 = kv_dtype == "fp8_e4m3"
        if kv_dtype not in ("bf16", "fp8_e4m3"):
            raise ValueError(kv_dtype)
        self.kv_dtype = kv_dtype
        self.Hq, self.Hkv, self.D = num_q_heads, num_kv_heads, head_dim
        self.max_traces, self.max_blocks = max_traces, max_blocks_per_trace
        self.num_layers = num_layers
        cache_dtype = torch.uint8 if fp8 else torch.bfloat16
        self.cache_dtype = cache_dtype
        # one layer: [num_blocks][Hkv][16][D]; several: a leading layer axis
        lead = (num_layers,) if num_layers > 1 else ()
        shape = lead + (num_blocks, num_kv_heads, 16, head_dim)
        self.k_cache = torch.empty(shape, dtype=cache_dtype, device=device)
        self.v_cache = torch.empty(shape, dtype=cache_dtype, device=device)
        self.kv_scale = torch.ones(lead + (num_blocks, 2), dtype=torch.float32, device=device) if fp8 else None
        self.block_table = torch.empty((max_traces, max_blocks_per_trace), dtype=torch.int32, device=device)
        self.seq_len = torch.empty(max_traces, dtype=torch.int32, device=device)
        self.refcount = torch.empty(num_blocks, dtype=torch.int32, device=device)
        d = PoolDesc(num_blocks, 16, num_q_heads, num_kv_heads, head_dim,
                     KV_FP8_E4M3 if fp8 else KV_BF16, max_traces, max_blocks_per_trace, max_splits,
                     fp8_append_scale,
                     num_layers, self.k_cache.data_ptr(), self.v_cache.data_ptr(),
                     self.kv_scale.data_ptr() if fp8 else None, self.block_table.data_ptr(),
                     self.seq_len.data_ptr(), self.refcount.data_ptr(), None, 0)
        ws = workspace_size(d)
        if ws == 0:
            raise GambitError(ERR_INVALID, "invalid pool description")
        self.workspace = torch.empty(ws + 256, dtype=torch.uint8, device=device)
        base = self.workspace.data_ptr()
        d.workspace = base + (-base) % 256
        d.workspace_bytes = ws
        self.desc = d
        h = ctypes.c_void_p()
        st = lib().gambit_pool_create(ctypes.byref(d), _stream(stream), ctypes.byref(h))
        if st != OK:
            raise GambitError(st, "pool_create")
        self._h = h

    # -- plumbing
    def _check(self, st: int, what: str):
        if st != OK:
            raise GambitError(st, f"{what}: {lib().gambit_last_error(self._h).decode()}")

    def close(self):
        if getattr(self, "_h", None):
            torch.cuda.current_stream().synchronize()
            lib().gambit_pool_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- entry points
    def kv_alloc(self, ids, n_tokens, stream=None):
        ids, nt = _host_i32(ids), _host_i32(n_tokens)
        self._check(lib().gambit_kv_alloc(self._h, ids.size, _ptr(ids), _ptr(nt), _stream(stream)),
                    "kv_alloc")

    def kv_write(self, trace: int, pos0: int, k: torch.Tensor, v: torch.Tensor, scales=None, stream=None):
        """k, v: [n][Hkv][D] (one layer) or [num_layers][n][Hkv][D]; fp8 scales
        [m][2] or [num_layers][m][2]."""
        if k.dim() not in (3, 4):
            raise ValueError("k: expected [n][Hkv][D] or [num_layers][n][Hkv][D]")
        n = k.shape[-3]
        shape = ((self.num_layers,) if self.num_layers > 1 or k.dim() == 4 else ()) + (n, self.Hkv, self.D)
        _spec(k, self.cache_dtype, shape, "k")
        _spec(v, self.cache_dtype, shape, "v")
        sc = None
        if scales is not None:
            if self.kv_dtype != "fp8_e4m3":
                raise ValueError("scales: only fp8 pools take block scales")
            sc = np.ascontiguousarray(np.asarray(scales, np.float32))
            # one (K, V) pair per block whose first position lies in [pos0, pos0 + n), per layer
            m = -(-(pos0 + n) // 16) - -(-pos0 // 16)
            want = (self.num_layers, m, 2)
            if not (sc.shape == want or (self.num_layers == 1 and sc.shape == want[1:])):
                raise ValueError(f"scales: expected shape {want if self.num_layers > 1 else want[1:]}, got {sc.shape}")
        self._check(lib().gambit_kv_write(self._h, trace, pos0, n, _dev(k), _dev(v),
                                          None if sc is None else _ptr(sc), _stream(stream)),
                    "kv_write")

    def kv_fork(self, parents, children, stream=None):
        p, c = _host_i32(parents), _host_i32(children)
        self._check(lib().gambit_kv_fork(self._h, c.size, _ptr(p), _ptr(c), _stream(stream)), "kv_fork")

    def kv_free(self, ids, stream=None):
        ids = _host_i32(ids)
        self._check(lib().gambit_kv_free(self._h, ids.size, _ptr(ids), _stream(stream)), "kv_free")

    def decode_attn(self, ids, q: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor,
                    out: torch.Tensor | None = None, out_dtype=torch.bfloat16, sm_scale=None,
                    stream=None) -> torch.Tensor:
        ids = _host_i32(ids)
        n = ids.size
        if out is None:
            out = torch.empty((n, self.Hq, self.D), dtype=out_dtype, device=q.device)
        _spec(out, (torch.float32, torch.bfloat16), (n, self.Hq, self.D), "out")
        od = OUT_F32 if out.dtype == torch.float32 else OUT_BF16
        sm = float(self.D ** -0.5 if sm_scale is None else sm_scale)
        _spec(q, torch.bfloat16, (n, self.Hq, self.D), "q")
        _spec(k_new, self.cache_dtype, (n, self.Hkv, self.D), "k_new")
        _spec(v_new, self.cache_dtype, (n, self.Hkv, self.D), "v_new")
        self._check(lib().gambit_decode_attn(self._h, n, _ptr(ids), _dev(q), _dev(k_new), _dev(v_new),
                                             _dev(out), od, sm, _stream(stream)), "decode_attn")
        return out

    def decode_attn_layer(self, layer: int, ids, q: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor,
                          new_dtype: str = "cache", out: torch.Tensor | None = None, out_dtype=torch.bfloat16,
                          sm_scale=None, stream=None) -> torch.Tensor:
        """gambit_decode_attn_layer: layer `layer` of a decode step; new_dtype
        "bf16" quantises bf16 k_new / v_new on append (fp8 pools)."""
        ids = _host_i32(ids)
        n = ids.size
        if out is None:
            out = torch.empty((n, self.Hq, self.D), dtype=out_dtype, device=q.device)
        _spec(out, (torch.float32, torch.bfloat16), (n, self.Hq, self.D), "out")
        od = OUT_F32 if out.dtype == torch.float32 else OUT_BF16
        if new_dtype not in ("cache", "bf16"):
            raise ValueError(f"new_dtype: {new_dtype!r}")
        nd = {"cache": NEW_CACHE, "bf16": NEW_BF16}[new_dtype]
        ndt = torch.bfloat16 if nd == NEW_BF16 else self.cache_dtype
        _spec(k_new, ndt, (n, self.Hkv, self.D), "k_new")
        _spec(v_new, ndt, (n, self.Hkv, self.D), "v_new")
        sm = float(self.D ** -0.5 if sm_scale is None else sm_scale)
        _spec(q, torch.bfloat16, (n, self.Hq, self.D), "q")
        self._check(lib().gambit_decode_attn_layer(self._h, layer, n, _ptr(ids), _dev(q), _dev(k_new), _dev(v_new),
                                                   nd, _dev(out), od, sm, _stream(stream)), "decode_attn_layer")
        return out

    def score_prune_branch(self, ids, h: torch.Tensor, w: torch.Tensor, b: float, keep: int,
                           n_parents: int, stream=None):
        """Returns device tensors (scores [n], keep ids [keep], child/parent pairs [n-keep][2])."""
        ids = _host_i32(ids)
        n = ids.size
        if h.dim() != 2:
            raise ValueError("h: expected [n][Dh]")
        Dh = h.shape[1]
        _spec(h, torch.bfloat16, (n, Dh), "h")
        _spec(w, torch.float32, (Dh,), "w")
        if not 0 <= keep <= n:
            raise ValueError(f"keep: {keep} not in [0, {n}]")
        dev = h.device
        scores = torch.empty(n, dtype=torch.float32, device=dev)
        keep_out = torch.empty(max(keep, 1), dtype=torch.int32, device=dev)
        pairs = torch.empty((max(n - keep, 1), 2), dtype=torch.int32, device=dev)
        self._check(lib().gambit_score_prune_branch(self._h, n, _ptr(ids), _dev(h), h.shape[1],
                                                    _dev(w, torch.float32), float(b), keep, n_parents,
                                                    _dev(scores), _dev(keep_out), _dev(pairs),
                                                    _stream(stream)), "score_prune_branch")
        return scores, keep_out[:keep], pairs[:n - keep]

    # -- the full tournament of Alg. 1
    def score_update(self, ids, h: torch.Tensor, w: torch.Tensor, b: float, stream=None) -> torch.Tensor:
        """gambit_score_update: thought scores f [n] (device); running means update in the pool."""
        ids = _host_i32(ids)
        n = ids.size
        if h.dim() != 2 or h.shape[0] < n:
            raise ValueError("h: expected [>= n][Dh]")
        Dh = h.shape[1]
        _spec(h, torch.bfloat16, None, "h")
        _spec(w, torch.float32, (Dh,), "w")
        scores = torch.empty(max(n, 1), dtype=torch.float32, device=h.device)
        self._check(lib().gambit_score_update(self._h, n, _ptr(ids), _dev(h), Dh if n else 8,
                                              _dev(w, torch.float32), float(b), _dev(scores),
                                              _stream(stream)), "score_update")
        return scores[:n]

    def evict(self, ids, stream=None) -> int:
        """gambit_evict: the listed running trace of lowest running score becomes a ghost."""
        ids = _host_i32(ids)
        v = np.zeros(1, np.int32)
        self._check(lib().gambit_evict(self._h, ids.size, _ptr(ids), _ptr(v), _stream(stream)), "evict")
        return int(v[0])

    def tournament(self, capacity: int, swap_k: int, warmup: int, want_ranked: bool = False, stream=None):
        """gambit_tournament: (case, n_active, pruned ids, [(child, parent)], ranked ids or None)."""
        r = Round()
        pruned = np.zeros(max(swap_k, 1), np.int32)
        pairs = np.zeros((self.max_traces, 2), np.int32)
        ranked = torch.empty(self.max_traces, dtype=torch.int32, device="cuda") if want_ranked else None
        self._check(lib().gambit_tournament(self._h, capacity, swap_k, warmup, ctypes.byref(r), _ptr(pruned),
                                            _ptr(pairs), None if ranked is None else _dev(ranked),
                                            _stream(stream)), "tournament")
        pl = [(int(c), int(p)) for c, p in pairs[:r.n_children]]
        rk = ranked[:r.n_active].cpu().numpy().tolist() if ranked is not None else None
        return r.case_taken, r.n_active, pruned[:r.n_pruned].tolist(), pl, rk

    def record_scores(self, ids, f: torch.Tensor, stream=None):
        """gambit_record_scores: running means from device thought scores f [n]."""
        ids = _host_i32(ids)
        if f.dim() != 1 or f.shape[0] < ids.size:
            raise ValueError("f: expected [>= n] fp32")
        self._check(lib().gambit_record_scores(self._h, ids.size, _ptr(ids), _dev(f, torch.float32, None, "f"),
                                               _stream(stream)), "record_scores")

    def trace_state(self, ids, stream=None):
        """gambit_trace_state: (s_bar fp32, scored thoughts, GenLen, ghost) per listed slot."""
        ids = _host_i32(ids)
        n = ids.size
        sb, ns, ge, gh = (np.zeros(n, np.float32), np.zeros(n, np.int32), np.zeros(n, np.int32),
                          np.zeros(n, np.int32))
        self._check(lib().gambit_trace_state(self._h, n, _ptr(ids), _ptr(sb), _ptr(ns), _ptr(ge), _ptr(gh),
                                             _stream(stream)), "trace_state")
        return sb, ns, ge, gh

    def pool_check(self, stream=None):
        self._check(lib().gambit_pool_check(self._h, _stream(stream)), "pool_check")

    def plan_stats(self, ids) -> Stats:
        ids = _host_i32(ids)
        s = Stats()
        self._check(lib().gambit_plan_stats(self._h, ids.size, _ptr(ids), ctypes.byref(s)), "plan_stats")
        return s

    def plan_kinds(self, ids) -> np.ndarray:
        """gambit_plan_kinds: UNIT_* bits per listed trace in the current plan."""
        ids = _host_i32(ids)
        out = np.zeros(ids.size, np.int32)
        self._check(lib().gambit_plan_kinds(self._h, ids.size, _ptr(ids), _ptr(out)), "plan_kinds")
        return out

    def profile_begin(self, max_launches: int):
        """gambit_profile_begin: time the split-K attention kernel of each decode step."""
        self._check(lib().gambit_profile_begin(self._h, max_launches), "profile_begin")

    def profile_end(self):
        """gambit_profile_end: (summed attention-kernel ms, timed launches)."""
        ms, n = ctypes.c_double(), ctypes.c_int32()
        self._check(lib().gambit_profile_end(self._h, ctypes.byref(ms), ctypes.byref(n)), "profile_end")
        return ms.value, n.value

    def seq_len_of(self, t: int) -> int:
        return int(lib().gambit_seq_len(self._h, t))

    def free_blocks(self) -> int:
        return int(lib().gambit_free_blocks(self._h))


def _interleave16(w1: np.ndarray, w3: np.ndarray) -> np.ndarray:
    """Rows 32c .. 32c+15 = w1 rows 16c .. 16c+15, rows 32c+16 .. 32c+31 = w3's."""
    f, d = w1.shape
    return np.stack([w1.reshape(f // 16, 16, d), w3.reshape(f // 16, 16, d)], axis=1).reshape(2 * f, d)


class Scorer:
    """The sequence scorer with per-slot step histories (gambit_scorer_*).

    weights: dict of fp32 arrays - ln_in_g, ln_in_b [D], W_in [d][D],
    ln_out_g, ln_out_b, w_out [d], and "layers": a list of dicts with ln1_g,
    ln1_b, Wq, Wk, Wv, Wo, ln2_g, ln2_b, W1, W3 ([d_ff][d]), W2 ([d][d_ff]).
    The binding only packs them into the library's layout on the device."""

    def __init__(self, weights: dict, *, n_heads: int, max_steps: int, max_traces: int, device: str = "cuda",
                 stream=None):
        f32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(device)  # noqa: E731
        L = weights["layers"]
        d, D = weights["W_in"].shape
        d_ff = L[0]["W1"].shape[0] if L else 64
        stack = lambda key: np.stack([x[key] for x in L]) if L else np.zeros((1, 1), np.float32)  # noqa: E731
        self.t = {"ln_in_g": f32(weights["ln_in_g"]), "ln_in_b": f32(weights["ln_in_b"]),
                  "w_in": f32(weights["W_in"]), "ln_out_g": f32(weights["ln_out_g"]),
                  "ln_out_b": f32(weights["ln_out_b"]), "w_out": f32(weights["w_out"]),
                  "ln1_g": f32(stack("ln1_g")), "ln1_b": f32(stack("ln1_b")),
                  "ln2_g": f32(stack("ln2_g")), "ln2_b": f32(stack("ln2_b")),
                  "w_o": f32(stack("Wo")), "w_2": f32(stack("W2")),
                  "w_qkv": f32(np.stack([np.concatenate([x["Wq"], x["Wk"], x["Wv"]]) for x in L]) if L
                               else np.zeros((1, 1), np.float32)),
                  "w_13": f32(np.stack([_interleave16(x["W1"], x["W3"]) for x in L]) if L
                              else np.zeros((1, 1), np.float32))}
        self.D, self.d = D, d
        desc = ScorerDesc(D, d, n_heads, len(L), d_ff, max_steps, max_traces,
                          *[self.t[k].data_ptr() for k in ("ln_in_g", "ln_in_b", "w_in", "ln1_g", "ln1_b", "w_qkv",
                                                           "w_o", "ln2_g", "ln2_b", "w_13", "w_2", "ln_out_g",
                                                           "ln_out_b", "w_out")], None, 0)
        ws = int(lib().gambit_scorer_workspace_size(ctypes.byref(desc)))
        if ws == 0:
            raise GambitError(ERR_INVALID, "invalid scorer description")
        self.workspace = torch.empty(ws + 256, dtype=torch.uint8, device=device)
        base = self.workspace.data_ptr()
        desc.workspace = base + (-base) % 256
        desc.workspace_bytes = ws
        self.desc = desc
        h = ctypes.c_void_p()
        st = lib().gambit_scorer_create(ctypes.byref(desc), _stream(stream), ctypes.byref(h))
        if st != OK:
            raise GambitError(st, "scorer_create")
        self._h = h

    def _check(self, st: int, what: str):
        if st != OK:
            raise GambitError(st, f"{what}: {lib().gambit_scorer_last_error(self._h).decode()}")

    def close(self):
        if getattr(self, "_h", None):
            torch.cuda.current_stream().synchronize()
            lib().gambit_scorer_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def step(self, ids, h: torch.Tensor, stream=None) -> torch.Tensor:
        """Scores [n] (device fp32) of the listed slots' new step states h [n][D] bf16."""
        ids = _host_i32(ids)
        n = ids.size
        out = torch.empty(max(n, 1), dtype=torch.float32, device=h.device)
        _dev(h, torch.bfloat16, (n, self.D))
        self._check(lib().gambit_scorer_step(self._h, n, _ptr(ids), _dev(h), _dev(out), _stream(stream)), "step")
        return out[:n]

    def fork(self, parents, children, stream=None):
        p, c = _host_i32(parents), _host_i32(children)
        self._check(lib().gambit_scorer_fork(self._h, c.size, _ptr(p), _ptr(c), _stream(stream)), "fork")

    def free(self, ids, stream=None):
        ids = _host_i32(ids)
        self._check(lib().gambit_scorer_free(self._h, ids.size, _ptr(ids), _stream(stream)), "free")

    def steps(self, trace: int) -> int:
        return int(lib().gambit_scorer_steps(self._h, trace))

    def check(self, stream=None):
        self._check(lib().gambit_scorer_check(self._h, _stream(stream)), "check")
