"""Chunked-prefill attention over a paged KV cache, and chunked prefill of a KDA (gated
delta-rule) layer with recurrent-state snapshots, on AMD MI355X (gfx950).

Thin Python binding of libwavepp_attn.so (C ABI declared in include/wavepp_attn.h and
include/wavepp_kda.h).  Every step of
the computation runs in the library's HIP kernels; this module only marshals arguments: torch
tensors are passed as device pointers, the stream is torch's current HIP stream.

Per wave:
    p = plan(...)                       # host: validate the spans, build the work list
    ws = new_workspace(p)               # device scratch for metadata and split partials
    plan_upload(p, ws)                  # enqueue the metadata copy
    append_kv(p, k_new, v_new, k_pool, v_pool, ws)
    chunked_prefill(p, q, k_pool, v_pool, out, lse, ws)

Per wave of a KDA layer:
    kp = kda_plan(...)                  # host: validate chunk lengths and snapshot slots
    ws = new_workspace(kp)
    kda_upload(kp, ws)
    kda_chunked_prefill(kp, q, k, v, alpha, beta, state_pool, out, ws)
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libwavepp_attn.so")

WAVEPP_OK = 0
STATUS_NAMES = {0: "WAVEPP_OK", -1: "WAVEPP_EINVAL", -2: "WAVEPP_EUNSUPPORTED", -3: "WAVEPP_ERANGE",
                -4: "WAVEPP_EALIAS", -5: "WAVEPP_EPOSITION", -6: "WAVEPP_ENOSPACE", -7: "WAVEPP_EHIP"}

EXPORTED_SYMBOLS = [
    "wavepp_attn_plan", "wavepp_plan_workspace_bytes", "wavepp_plan_get_info", "wavepp_plan_get_items",
    "wavepp_attn_plan_upload", "wavepp_attn_append_kv", "wavepp_attn_chunked_prefill", "wavepp_plan_destroy",
    "wavepp_status_string", "wavepp_last_error", "wavepp_attn_chunked_prefill_noalloc",
]
MPU_SYMBOLS = [
    "wavepp_mpu_budget_ladder", "wavepp_mpu_create", "wavepp_mpu_admit", "wavepp_mpu_plan", "wavepp_mpu_commit",
    "wavepp_mpu_retire", "wavepp_mpu_get_state", "wavepp_mpu_destroy",
]
HINT_SYMBOLS = [
    "wavepp_block_hashes", "wavepp_hint_index_create", "wavepp_hint_index_add", "wavepp_hint_index_detach",
    "wavepp_hint_index_size", "wavepp_hint_probe_prefix", "wavepp_hint_probe_prefix_linear",
    "wavepp_hint_probe_recurrent", "wavepp_hint_index_destroy",
]
KDA_SYMBOLS = [
    "wavepp_kda_plan", "wavepp_kda_workspace_bytes", "wavepp_kda_get_info", "wavepp_kda_upload",
    "wavepp_kda_chunked_prefill", "wavepp_kda_destroy",
]
PROBE_SYMBOLS = ["wavepp_probe_mfma", "wavepp_probe_hbm_read"]


class WaveppError(RuntimeError):
    def __init__(self, status, detail):
        self.status = status
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {detail}")


class _Shape(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim_qk", ctypes.c_int32), ("head_dim_v", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("num_pages", ctypes.c_int32),
                ("kv_shared", ctypes.c_int32), ("softmax_scale", ctypes.c_float)]


class _Batch(ctypes.Structure):
    _fields_ = [("num_requests", ctypes.c_int32), ("prefix_lens", ctypes.POINTER(ctypes.c_int32)),
                ("chunk_lens", ctypes.POINTER(ctypes.c_int32)), ("block_table", ctypes.POINTER(ctypes.c_int32)),
                ("bt_stride", ctypes.c_int32)]


class _Info(ctypes.Structure):
    _fields_ = [("total_tokens", ctypes.c_int64), ("num_items", ctypes.c_int32),
                ("num_real_items", ctypes.c_int32), ("num_merge_items", ctypes.c_int32),
                ("max_splits", ctypes.c_int32), ("rows_per_item", ctypes.c_int32), ("kv_tile", ctypes.c_int32),
                ("partial_rows", ctypes.c_int64), ("metadata_bytes", ctypes.c_int64),
                ("workspace_bytes", ctypes.c_int64)]


class _KdaShape(ctypes.Structure):
    _fields_ = [("num_heads", ctypes.c_int32), ("head_dim_k", ctypes.c_int32), ("head_dim_v", ctypes.c_int32),
                ("num_state_slots", ctypes.c_int32)]


class _KdaBatch(ctypes.Structure):
    _fields_ = [("num_requests", ctypes.c_int32), ("chunk_lens", ctypes.POINTER(ctypes.c_int32)),
                ("state_in", ctypes.POINTER(ctypes.c_int32)), ("state_out", ctypes.POINTER(ctypes.c_int32))]


class _KdaInfo(ctypes.Structure):
    _fields_ = [("total_tokens", ctypes.c_int64), ("num_items", ctypes.c_int32), ("block_tokens", ctypes.c_int32),
                ("metadata_bytes", ctypes.c_int64), ("workspace_bytes", ctypes.c_int64)]


class _MpuConfig(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("max_budget", "min_budget", "block", "stages", "fills", "max_lanes",
                                               "split_permille", "count_inflight")]


class _Span(ctypes.Structure):
    _fields_ = [("request", ctypes.c_int32), ("start", ctypes.c_int32), ("length", ctypes.c_int32)]


class _MpuState(ctypes.Structure):
    _fields_ = [("work", ctypes.c_int64), ("budget", ctypes.c_int32), ("ring", ctypes.c_int32),
                ("requests", ctypes.c_int32), ("up_count", ctypes.c_int32), ("down_count", ctypes.c_int32)]


_lib = None


def load_library(path: str = None) -> ctypes.CDLL:
    """Load the built HIP library; raise if it has not been built (there is no fallback path)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    path = path or os.environ.get("WAVEPP_LIB") or LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it first (python -m paper_2609_35263_amd.build)")
    lib = ctypes.CDLL(path)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    lib.wavepp_attn_plan.argtypes = [ctypes.POINTER(_Shape), ctypes.POINTER(_Batch), i32, ctypes.POINTER(vp)]
    lib.wavepp_attn_plan.restype = ctypes.c_int
    lib.wavepp_plan_workspace_bytes.argtypes = [vp]
    lib.wavepp_plan_workspace_bytes.restype = sz
    lib.wavepp_plan_get_info.argtypes = [vp, ctypes.POINTER(_Info)]
    lib.wavepp_plan_get_info.restype = ctypes.c_int
    lib.wavepp_plan_get_items.argtypes = [vp, ctypes.POINTER(i32), i32]
    lib.wavepp_plan_get_items.restype = ctypes.c_int
    lib.wavepp_attn_plan_upload.argtypes = [vp, vp, sz, vp]
    lib.wavepp_attn_plan_upload.restype = ctypes.c_int
    lib.wavepp_attn_append_kv.argtypes = [vp, vp, vp, vp, vp, vp, sz, vp]
    lib.wavepp_attn_append_kv.restype = ctypes.c_int
    lib.wavepp_attn_chunked_prefill.argtypes = [vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.wavepp_attn_chunked_prefill.restype = ctypes.c_int
    lib.wavepp_attn_chunked_prefill_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.wavepp_attn_chunked_prefill_noalloc.restype = ctypes.c_int
    lib.wavepp_plan_destroy.argtypes = [vp]
    lib.wavepp_plan_destroy.restype = None
    lib.wavepp_status_string.argtypes = [ctypes.c_int]
    lib.wavepp_status_string.restype = ctypes.c_char_p
    lib.wavepp_last_error.argtypes = []
    lib.wavepp_last_error.restype = ctypes.c_char_p
    lib.wavepp_kda_plan.argtypes = [ctypes.POINTER(_KdaShape), ctypes.POINTER(_KdaBatch), ctypes.POINTER(vp)]
    lib.wavepp_kda_plan.restype = ctypes.c_int
    lib.wavepp_kda_workspace_bytes.argtypes = [vp]
    lib.wavepp_kda_workspace_bytes.restype = sz
    lib.wavepp_kda_get_info.argtypes = [vp, ctypes.POINTER(_KdaInfo)]
    lib.wavepp_kda_get_info.restype = ctypes.c_int
    lib.wavepp_kda_upload.argtypes = [vp, vp, sz, vp]
    lib.wavepp_kda_upload.restype = ctypes.c_int
    lib.wavepp_kda_chunked_prefill.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.wavepp_kda_chunked_prefill.restype = ctypes.c_int
    lib.wavepp_kda_destroy.argtypes = [vp]
    lib.wavepp_kda_destroy.restype = None
    cfgp, spanp = ctypes.POINTER(_MpuConfig), ctypes.POINTER(_Span)
    lib.wavepp_mpu_budget_ladder.argtypes = [cfgp, ctypes.POINTER(i32), i32]
    lib.wavepp_mpu_create.argtypes = [cfgp, ctypes.POINTER(vp)]
    lib.wavepp_mpu_admit.argtypes = [vp, i32, i32, i32]
    lib.wavepp_mpu_plan.argtypes = [vp, i32, spanp, i32, ctypes.POINTER(i32)]
    lib.wavepp_mpu_commit.argtypes = [vp, spanp, i32]
    lib.wavepp_mpu_retire.argtypes = [vp]
    lib.wavepp_mpu_get_state.argtypes = [vp, ctypes.POINTER(_MpuState)]
    lib.wavepp_mpu_destroy.argtypes = [vp]
    lib.wavepp_mpu_destroy.restype = None
    i64, u64p, u8p = ctypes.c_int64, ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(ctypes.c_uint8)
    lib.wavepp_block_hashes.argtypes = [ctypes.POINTER(i32), i64, i32, ctypes.POINTER(i64), i32, u8p, i32, u8p, u64p]
    lib.wavepp_block_hashes.restype = i64
    lib.wavepp_hint_index_create.argtypes = [i32, ctypes.POINTER(vp)]
    lib.wavepp_hint_index_add.argtypes = [vp, i32, u64p, i64]
    lib.wavepp_hint_index_detach.argtypes = [vp, i32, u64p, i64]
    lib.wavepp_hint_index_size.argtypes = [vp]
    lib.wavepp_hint_index_size.restype = i64
    for name in ("wavepp_hint_probe_prefix", "wavepp_hint_probe_prefix_linear", "wavepp_hint_probe_recurrent"):
        getattr(lib, name).argtypes = [vp, i32, u64p, i64, ctypes.POINTER(i64), ctypes.POINTER(i32)]
        getattr(lib, name).restype = ctypes.c_int
    for name in ("wavepp_hint_index_create", "wavepp_hint_index_add", "wavepp_hint_index_detach"):
        getattr(lib, name).restype = ctypes.c_int
    lib.wavepp_hint_index_destroy.argtypes = [vp]
    lib.wavepp_hint_index_destroy.restype = None
    for name in ("wavepp_mpu_budget_ladder", "wavepp_mpu_create", "wavepp_mpu_admit", "wavepp_mpu_plan",
                 "wavepp_mpu_commit", "wavepp_mpu_retire", "wavepp_mpu_get_state"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _check(status):
    if status != WAVEPP_OK:
        raise WaveppError(status, load_library().wavepp_last_error().decode())


class Plan:
    """A validated wave and its work list (host object owned by the library)."""

    def __init__(self, handle, shape):
        self._h = ctypes.c_void_p(handle)
        self.shape = shape

    @property
    def handle(self):
        if not self._h:
            raise ValueError("plan was destroyed")
        return self._h

    @property
    def workspace_bytes(self) -> int:
        return int(load_library().wavepp_plan_workspace_bytes(self.handle))

    def info(self) -> dict:
        info = _Info()
        _check(load_library().wavepp_plan_get_info(self.handle, ctypes.byref(info)))
        return {name: int(getattr(info, name)) for name, _ in _Info._fields_}

    def items(self) -> np.ndarray:
        n = self.info()["num_items"]
        buf = np.zeros((max(n, 1), 8), dtype=np.int32)
        got = load_library().wavepp_plan_get_items(self.handle, buf.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), n)
        if got < 0:
            _check(got)
        return buf[:got]

    def destroy(self):
        if self._h:
            load_library().wavepp_plan_destroy(self._h)
            self._h = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def plan(*, num_q_heads, num_kv_heads, head_dim_qk, head_dim_v, page_size, num_pages, softmax_scale,
         prefix_lens, chunk_lens, block_table, kv_shared=False, max_splits=0) -> Plan:
    lib = load_library()
    prefix = np.ascontiguousarray(prefix_lens, dtype=np.int32)
    chunk = np.ascontiguousarray(chunk_lens, dtype=np.int32)
    bt = np.ascontiguousarray(block_table, dtype=np.int32)
    if bt.ndim != 2:
        raise ValueError("block_table must be 2-D [num_requests, bt_stride]")
    if not (prefix.shape == chunk.shape == (bt.shape[0],)):
        raise ValueError("prefix_lens, chunk_lens and block_table rows must have the same length")
    shape = _Shape(num_q_heads, num_kv_heads, head_dim_qk, head_dim_v, page_size, num_pages, int(bool(kv_shared)),
                   float(softmax_scale))
    p32 = ctypes.POINTER(ctypes.c_int32)
    batch = _Batch(int(prefix.shape[0]), prefix.ctypes.data_as(p32), chunk.ctypes.data_as(p32),
                   bt.ctypes.data_as(p32), int(bt.shape[1]))
    out = ctypes.c_void_p()
    _check(lib.wavepp_attn_plan(ctypes.byref(shape), ctypes.byref(batch), int(max_splits), ctypes.byref(out)))
    return Plan(out.value, dict(num_q_heads=num_q_heads, num_kv_heads=num_kv_heads, head_dim_qk=head_dim_qk,
                                head_dim_v=head_dim_v, page_size=page_size, num_pages=num_pages,
                                kv_shared=bool(kv_shared), softmax_scale=float(softmax_scale),
                                total_tokens=int(chunk.sum())))


def plan_for(spec, max_splits=0) -> Plan:
    """Plan a wave described by a workloads.WaveSpec-like object."""
    return plan(num_q_heads=spec.num_q_heads, num_kv_heads=spec.num_kv_heads, head_dim_qk=spec.head_dim_qk,
                head_dim_v=spec.head_dim_v, page_size=spec.page_size, num_pages=spec.num_pages,
                softmax_scale=spec.softmax_scale, prefix_lens=spec.prefix_lens, chunk_lens=spec.chunk_lens,
                block_table=spec.block_table, kv_shared=spec.kv_shared, max_splits=max_splits)


# ------------------------------------------------------------------------------------------------
# Device calls (torch tensors for memory and the current stream)
# ------------------------------------------------------------------------------------------------

def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _check_shapes(**named):
    """Every tensor (name=(tensor or None, shape)) has the plan's shape.  Checked for all buffers of
    a call before anything else: the kernels index every buffer by the plan's sizes, so a tensor of
    any other shape would be read or written out of bounds."""
    for name, (t, shape) in named.items():
        if t is not None and tuple(t.shape) != tuple(int(x) for x in shape):
            raise ValueError(f"{name} has shape {tuple(t.shape)}, the plan needs {tuple(int(x) for x in shape)}")


def _ptr(t, dtype=None, name="", shape=None):
    """Device pointer of a contiguous tensor of the given dtype and shape (None: no buffer)."""
    if t is None:
        return ctypes.c_void_p(None)
    if shape is not None:
        _check_shapes(**{name: (t, shape)})
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    return ctypes.c_void_p(t.data_ptr())


def new_workspace(p: Plan, device=None):
    import torch
    n = max(p.workspace_bytes, 256)
    return torch.empty(n, dtype=torch.uint8, device=device or "cuda")


def plan_upload(p: Plan, workspace, stream=None):
    _check(load_library().wavepp_attn_plan_upload(p.handle, _ptr(workspace, name="workspace"),
                                                  workspace.numel() * workspace.element_size(), _stream(stream)))


def _attn_shapes(p: Plan) -> dict:
    s = p.shape
    T, Hq, Hkv = s["total_tokens"], s["num_q_heads"], s["num_kv_heads"]
    P, B, dq, dv = s["num_pages"], s["page_size"], s["head_dim_qk"], s["head_dim_v"]
    return {"q": (T, Hq, dq), "k_new": (T, Hkv, dq), "v_new": (T, Hkv, dv), "k_pool": (P, Hkv, B, dq),
            "v_pool": (P, Hkv, B, dv), "out": (T, Hq, dv), "lse": (T, Hq)}


def _shared_kv_none(p: Plan, **bufs):
    for name, t in bufs.items():
        if p.shape["kv_shared"] and t is not None:
            raise ValueError(f"{name} must be None for a latent (kv_shared) cache")
        if not p.shape["kv_shared"] and t is None:
            raise ValueError(f"{name} is required")


def append_kv(p: Plan, k_new, v_new, k_pool, v_pool, workspace, stream=None):
    import torch
    bf = torch.bfloat16
    sh = _attn_shapes(p)
    _shared_kv_none(p, v_new=v_new, v_pool=v_pool)
    _check_shapes(k_new=(k_new, sh["k_new"]), v_new=(v_new, sh["v_new"]), k_pool=(k_pool, sh["k_pool"]),
                  v_pool=(v_pool, sh["v_pool"]))
    _check(load_library().wavepp_attn_append_kv(
        p.handle, _ptr(k_new, bf, "k_new", sh["k_new"]), _ptr(v_new, bf, "v_new", sh["v_new"]),
        _ptr(k_pool, bf, "k_pool", sh["k_pool"]), _ptr(v_pool, bf, "v_pool", sh["v_pool"]),
        _ptr(workspace, name="workspace"), workspace.numel() * workspace.element_size(), _stream(stream)))


def chunked_prefill(p: Plan, q, k_pool, v_pool, out, lse, workspace, stream=None):
    import torch
    bf = torch.bfloat16
    sh = _attn_shapes(p)
    _shared_kv_none(p, v_pool=v_pool)
    _check_shapes(q=(q, sh["q"]), k_pool=(k_pool, sh["k_pool"]), v_pool=(v_pool, sh["v_pool"]),
                  out=(out, sh["out"]), lse=(lse, sh["lse"]))
    _check(load_library().wavepp_attn_chunked_prefill(
        p.handle, _ptr(q, bf, "q", sh["q"]), _ptr(k_pool, bf, "k_pool", sh["k_pool"]),
        _ptr(v_pool, bf, "v_pool", sh["v_pool"]), _ptr(out, bf, "out", sh["out"]),
        _ptr(lse, torch.float32, "lse", sh["lse"]), _ptr(workspace, name="workspace"),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def chunked_prefill_noalloc(p: Plan, q, k_pool, v_pool, out, lse, k_new=None, v_new=None, stream=None):
    """Append (when k_new is given) and attention with no workspace: the library's static per-GPU
    scratch holds the metadata and split partials.  Calls on one GPU must not overlap."""
    import torch
    bf = torch.bfloat16
    sh = _attn_shapes(p)
    _shared_kv_none(p, v_pool=v_pool)
    if p.shape["kv_shared"] and v_new is not None:
        raise ValueError("v_new must be None for a latent (kv_shared) cache")
    _check_shapes(q=(q, sh["q"]), k_new=(k_new, sh["k_new"]), v_new=(v_new, sh["v_new"]),
                  k_pool=(k_pool, sh["k_pool"]), v_pool=(v_pool, sh["v_pool"]), out=(out, sh["out"]),
                  lse=(lse, sh["lse"]))
    _check(load_library().wavepp_attn_chunked_prefill_noalloc(
        p.handle, _ptr(q, bf, "q"), _ptr(k_new, bf, "k_new"), _ptr(v_new, bf, "v_new"), _ptr(k_pool, bf, "k_pool"),
        _ptr(v_pool, bf, "v_pool"), _ptr(out, bf, "out"), _ptr(lse, torch.float32, "lse"), _stream(stream)))


# ------------------------------------------------------------------------------------------------
# KDA chunked prefill
# ------------------------------------------------------------------------------------------------

class KdaPlan:
    """A validated KDA wave: chunk lengths and snapshot slots (host object owned by the library)."""

    def __init__(self, handle, shape):
        self._h = ctypes.c_void_p(handle)
        self.shape = shape

    @property
    def handle(self):
        if not self._h:
            raise ValueError("plan was destroyed")
        return self._h

    @property
    def workspace_bytes(self) -> int:
        return int(load_library().wavepp_kda_workspace_bytes(self.handle))

    def info(self) -> dict:
        info = _KdaInfo()
        _check(load_library().wavepp_kda_get_info(self.handle, ctypes.byref(info)))
        return {name: int(getattr(info, name)) for name, _ in _KdaInfo._fields_}

    def destroy(self):
        if self._h:
            load_library().wavepp_kda_destroy(self._h)
            self._h = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def kda_plan(*, num_heads, head_dim_k, head_dim_v, num_state_slots, chunk_lens, state_in, state_out) -> KdaPlan:
    lib = load_library()
    chunk = np.ascontiguousarray(chunk_lens, dtype=np.int32)
    s_in = np.ascontiguousarray(state_in, dtype=np.int32)
    s_out = np.ascontiguousarray(state_out, dtype=np.int32)
    if not (chunk.ndim == 1 and chunk.shape == s_in.shape == s_out.shape):
        raise ValueError("chunk_lens, state_in and state_out must be 1-D of the same length")
    shape = _KdaShape(num_heads, head_dim_k, head_dim_v, num_state_slots)
    p32 = ctypes.POINTER(ctypes.c_int32)
    batch = _KdaBatch(int(chunk.shape[0]), chunk.ctypes.data_as(p32), s_in.ctypes.data_as(p32),
                      s_out.ctypes.data_as(p32))
    out = ctypes.c_void_p()
    _check(lib.wavepp_kda_plan(ctypes.byref(shape), ctypes.byref(batch), ctypes.byref(out)))
    return KdaPlan(out.value, dict(num_heads=num_heads, head_dim_k=head_dim_k, head_dim_v=head_dim_v,
                                   num_state_slots=num_state_slots, total_tokens=int(chunk.sum())))


def kda_plan_for(spec) -> KdaPlan:
    """Plan a wave described by a workloads.kda.KdaSpec-like object."""
    return kda_plan(num_heads=spec.num_heads, head_dim_k=spec.head_dim_k, head_dim_v=spec.head_dim_v,
                    num_state_slots=spec.num_slots, chunk_lens=spec.chunk_lens, state_in=spec.state_in,
                    state_out=spec.state_out)


def kda_upload(p: KdaPlan, workspace, stream=None):
    _check(load_library().wavepp_kda_upload(p.handle, _ptr(workspace, name="workspace"),
                                            workspace.numel() * workspace.element_size(), _stream(stream)))


def kda_chunked_prefill(p: KdaPlan, q, k, v, alpha, beta, state_pool, out, workspace, stream=None):
    import torch
    bf, f32 = torch.bfloat16, torch.float32
    s = p.shape
    T, H, dk, dv = s["total_tokens"], s["num_heads"], s["head_dim_k"], s["head_dim_v"]
    for name, t in (("q", q), ("k", k), ("v", v), ("alpha", alpha), ("beta", beta), ("state_pool", state_pool),
                    ("out", out)):
        if t is None:
            raise ValueError(f"{name} is required")
    _check_shapes(q=(q, (T, H, dk)), k=(k, (T, H, dk)), v=(v, (T, H, dv)), alpha=(alpha, (T, H, dk)),
                  beta=(beta, (T, H)), state_pool=(state_pool, (s["num_state_slots"], H, dk, dv)),
                  out=(out, (T, H, dv)))
    _check(load_library().wavepp_kda_chunked_prefill(
        p.handle, _ptr(q, bf, "q", (T, H, dk)), _ptr(k, bf, "k", (T, H, dk)), _ptr(v, bf, "v", (T, H, dv)),
        _ptr(alpha, f32, "alpha", (T, H, dk)), _ptr(beta, f32, "beta", (T, H)),
        _ptr(state_pool, f32, "state_pool", (s["num_state_slots"], H, dk, dv)), _ptr(out, bf, "out", (T, H, dv)),
        _ptr(workspace, name="workspace"), workspace.numel() * workspace.element_size(), _stream(stream)))


# ------------------------------------------------------------------------------------------------
# MPU wave planner (host only)
# ------------------------------------------------------------------------------------------------

def _mpu_config(max_budget, min_budget, block, stages, fills, max_lanes, split_permille=125, count_inflight=True):
    return _MpuConfig(max_budget, min_budget, block, stages, fills, max_lanes, split_permille, int(bool(count_inflight)))


def mpu_budget_ladder(max_budget, min_budget, block) -> list:
    cfg = _mpu_config(max_budget, min_budget, block, 1, 1, 1)
    buf = (ctypes.c_int32 * 64)()
    n = load_library().wavepp_mpu_budget_ladder(ctypes.byref(cfg), buf, 64)
    if n < 0:
        _check(n)
    return list(buf[:n])


class MpuPlanner:
    """The native wave planner: admit requests, then plan / commit waves and retire them."""

    def __init__(self, *, max_budget, min_budget, block, stages, fills, max_lanes, split_permille=125,
                 count_inflight=True):
        self.config = _mpu_config(max_budget, min_budget, block, stages, fills, max_lanes, split_permille,
                                  count_inflight)
        h = ctypes.c_void_p()
        _check(load_library().wavepp_mpu_create(ctypes.byref(self.config), ctypes.byref(h)))
        self._h = h
        self._spans = (_Span * max(1, max_lanes))()

    def admit(self, request, start, end):
        _check(load_library().wavepp_mpu_admit(self._h, int(request), int(start), int(end)))

    def plan(self, admission_pending=False):
        b = ctypes.c_int32()
        n = load_library().wavepp_mpu_plan(self._h, int(bool(admission_pending)), self._spans, len(self._spans),
                                            ctypes.byref(b))
        if n < 0:
            _check(n)
        return [(s.request, s.start, s.length) for s in self._spans[:n]], int(b.value)

    def commit(self, spans):
        arr = (_Span * max(1, len(spans)))(*[_Span(int(r), int(s), int(l)) for r, s, l in spans])
        serial = load_library().wavepp_mpu_commit(self._h, arr, len(spans))
        if serial < 0:
            _check(serial)
        return serial

    def retire(self):
        _check(load_library().wavepp_mpu_retire(self._h))

    def state(self) -> dict:
        st = _MpuState()
        _check(load_library().wavepp_mpu_get_state(self._h, ctypes.byref(st)))
        return {name: int(getattr(st, name)) for name, _ in _MpuState._fields_}

    def __del__(self):
        try:
            if self._h:
                load_library().wavepp_mpu_destroy(self._h)
                self._h = None
        except Exception:
            pass


# ------------------------------------------------------------------------------------------------
# Reuse hints (host only)
# ------------------------------------------------------------------------------------------------

def block_hashes(tokens, block, extra_keys=None, salt=b""):
    """Chained block hashes of the full blocks: (digests uint8 [n, 32], keys uint64 [n])."""
    toks = np.ascontiguousarray(tokens, dtype=np.int32)
    nb = len(toks) // int(block)
    extra = None if extra_keys is None else np.ascontiguousarray(extra_keys, dtype=np.int64).reshape(nb, -1)
    per = 0 if extra is None else int(extra.shape[1])
    dig = np.zeros((max(nb, 1), 32), dtype=np.uint8)
    keys = np.zeros(max(nb, 1), dtype=np.uint64)
    salt_arr = np.frombuffer(bytes(salt), dtype=np.uint8) if salt else np.zeros(1, dtype=np.uint8)
    n = load_library().wavepp_block_hashes(
        toks.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), len(toks), int(block),
        None if extra is None else extra.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), per,
        salt_arr.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)), len(salt),
        dig.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)), keys.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)))
    if n < 0:
        _check(int(n))
    return dig[:n], keys[:n]


class HintIndex:
    """The native sharded counted index of (window, key)."""

    def __init__(self, num_shards=64):
        h = ctypes.c_void_p()
        _check(load_library().wavepp_hint_index_create(int(num_shards), ctypes.byref(h)))
        self._h = h

    @staticmethod
    def _keys(keys):
        k = np.ascontiguousarray(keys, dtype=np.uint64)
        return k, k.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64))

    def add(self, window, keys):
        k, p = self._keys(keys)
        _check(load_library().wavepp_hint_index_add(self._h, int(window), p, len(k)))

    def detach(self, window, keys):
        k, p = self._keys(keys)
        _check(load_library().wavepp_hint_index_detach(self._h, int(window), p, len(k)))

    def size(self):
        return int(load_library().wavepp_hint_index_size(self._h))

    def _probe(self, fn, window, keys, n):
        k, p = self._keys(keys)
        e, np_ = ctypes.c_int64(), ctypes.c_int32()
        _check(getattr(load_library(), fn)(self._h, int(window), p, int(n), ctypes.byref(e), ctypes.byref(np_)))
        return int(e.value), int(np_.value)

    def probe_prefix(self, window, keys):
        """(endpoint in blocks, probes) by gallop and bisect."""
        return self._probe("wavepp_hint_probe_prefix", window, keys, len(keys))

    def probe_prefix_linear(self, window, keys):
        return self._probe("wavepp_hint_probe_prefix_linear", window, keys, len(keys))

    def probe_recurrent(self, window, keys, limit):
        if not 0 <= limit <= len(keys):
            raise ValueError("limit outside [0, len(keys)]")
        return self._probe("wavepp_hint_probe_recurrent", window, keys, limit)

    def __del__(self):
        try:
            if self._h:
                load_library().wavepp_hint_index_destroy(self._h)
                self._h = None
        except Exception:
            pass
