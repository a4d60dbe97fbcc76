"""ctypes binding of libepic_link (declared in include/epic_link.h).

Argument marshalling only: every step of the link step runs in the library
(host planner in C++, device work in HIP kernels).  PyTorch supplies device
memory and the current HIP stream.  Importing this module fails loudly when the
library has not been built; there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libepic_link.so")

EPIC_OK = 0
BLOCK = 16
WORK_INTS = 8     # int32 per attention work item in the plan


class EpicError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: {detail} (status {status})")
        self.status = status


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is not built; run `python -m paper_2410_15332_amd.build`")
    # Device memory and streams come from PyTorch, which ships its own HIP runtime
    # under the same soname (libamdhip64.so.7).  Load torch first so that this
    # library binds to the runtime already in the process; the other order would
    # leave torch on a second runtime that sees no device.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    return C.CDLL(_LIB_PATH)


_lib = _load()
_i32p = C.POINTER(C.c_int32)


class epic_attn_cfg(C.Structure):
    _fields_ = [("num_q_heads", C.c_int32), ("num_kv_heads", C.c_int32), ("head_dim", C.c_int32),
                ("block_size", C.c_int32), ("softmax_scale", C.c_float), ("kv_split_blocks", C.c_int32),
                ("tile_rows", C.c_int32), ("rope_theta", C.c_float)]


class epic_link_request(C.Structure):
    _fields_ = [("num_chunks", C.c_int32), ("chunk_len", _i32p), ("chunk_block_off", _i32p),
                ("chunk_blocks", _i32p), ("suffix_len", C.c_int32), ("k", C.c_int32), ("rerotate", C.c_int32)]


class epic_compile_batch(C.Structure):
    _fields_ = [("num_chunks", C.c_int32), ("chunk_len", _i32p), ("chunk_block_off", _i32p),
                ("chunk_blocks", _i32p), ("n_dummy", C.c_int32)]


class epic_plan_sizes(C.Structure):
    _fields_ = [("batch", C.c_int32), ("n_s", C.c_int32), ("n_linked_blocks", C.c_int32),
                ("n_private", C.c_int32), ("n_tiles", C.c_int32), ("n_work", C.c_int32),
                ("n_partials", C.c_int32), ("tile_rows", C.c_int32), ("max_pos", C.c_int32),
                ("n_rerotated", C.c_int32), ("total_ints", C.c_int64)]


PLAN_FIELDS = ["s_pos", "s_req", "s_slot", "s_off", "linked_blocks", "block_pos0", "block_len", "blk_off",
               "priv_block", "priv_src", "priv_rows", "tiles", "work", "priv_rot"]


class epic_plan(C.Structure):
    _fields_ = [(n, _i32p) for n in PLAN_FIELDS]


class epic_model_cfg(C.Structure):
    _fields_ = [("attn", epic_attn_cfg), ("hidden", C.c_int32), ("ffn", C.c_int32), ("n_layers", C.c_int32),
                ("rope_theta", C.c_float), ("rms_eps", C.c_float)]


class epic_layer_weights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("attn_norm", "wqkv", "wo", "mlp_norm", "w_gate_up", "w_down")]


def _proto(name, restype, argtypes):
    f = getattr(_lib, name)
    f.restype = restype
    f.argtypes = argtypes
    return f


_P = C.POINTER
_status_string = _proto("epic_status_string", C.c_char_p, [C.c_int])
_last_error = _proto("epic_last_error", C.c_char_p, [])
_version = _proto("epic_version", C.c_char_p, [])
_plan_sizes_get = _proto("epic_plan_sizes_get", C.c_int,
                         [_P(epic_link_request), C.c_int32, _P(epic_attn_cfg), C.c_int32, _P(epic_plan_sizes)])
_plan_layout = _proto("epic_plan_layout", C.c_int, [_P(epic_plan_sizes), C.c_void_p, _P(epic_plan)])
_plan_link = _proto("epic_plan_link", C.c_int,
                    [_P(epic_link_request), C.c_int32, _P(epic_attn_cfg), _i32p, C.c_int32, C.c_int32,
                     _P(epic_plan_sizes), _P(epic_plan)])
_plan_decode_sizes = _proto("epic_plan_decode_sizes", C.c_int,
                            [_P(epic_plan_sizes), _P(epic_plan), _i32p, _P(epic_attn_cfg), C.c_int32,
                             _P(epic_plan_sizes)])
_plan_decode = _proto("epic_plan_decode", C.c_int,
                      [_P(epic_plan_sizes), _P(epic_plan), _i32p, _P(epic_attn_cfg), _i32p, C.c_int32, C.c_int32,
                       _P(epic_plan_sizes), _P(epic_plan)])
_plan_compile_sizes = _proto("epic_plan_compile_sizes", C.c_int,
                             [_P(epic_compile_batch), _P(epic_attn_cfg), C.c_int32, _P(epic_plan_sizes)])
_plan_compile = _proto("epic_plan_compile", C.c_int,
                       [_P(epic_compile_batch), _P(epic_attn_cfg), _i32p, C.c_int32, C.c_int32,
                        _P(epic_plan_sizes), _P(epic_plan)])
_link_ws = _proto("epic_link_workspace_bytes", C.c_size_t, [_P(epic_attn_cfg), _P(epic_plan_sizes)])
_link_attention = _proto("epic_link_attention", C.c_int,
                         [_P(epic_attn_cfg), _P(epic_plan_sizes), _P(epic_plan), C.c_void_p, C.c_void_p,
                          C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t,
                          C.c_void_p])
_link_attention_noalloc = _proto("epic_link_attention_noalloc", C.c_int,
                                 [_P(epic_attn_cfg), _P(epic_plan_sizes), _P(epic_plan), C.c_void_p, C.c_void_p,
                                  C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p])
_set_prof = _proto("epic_set_profile_events", C.c_int, [C.c_void_p])
_model_ws = _proto("epic_model_workspace_bytes", C.c_size_t, [_P(epic_model_cfg), _P(epic_plan_sizes)])
_link_layer = _proto("epic_link_layer", C.c_int,
                     [_P(epic_model_cfg), _P(epic_layer_weights), _P(epic_plan_sizes), _P(epic_plan), C.c_void_p,
                      C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p])
_link_model = _proto("epic_link_model", C.c_int,
                     [_P(epic_model_cfg), _P(epic_layer_weights), C.c_void_p, _P(epic_plan_sizes), _P(epic_plan),
                      C.c_void_p, _P(C.c_void_p), _P(C.c_void_p), C.c_void_p, C.c_void_p, C.c_size_t,
                      C.c_void_p])

_gemm_ws = _proto("epic_gemm_workspace_bytes", C.c_size_t, [])
_gemm = _proto("epic_gemm", C.c_int,
               [C.c_int32, C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_int32, C.c_void_p, C.c_void_p,
                C.c_void_p, C.c_size_t, C.c_void_p])

EXPORTED = ["epic_status_string", "epic_last_error", "epic_version", "epic_plan_sizes_get", "epic_plan_layout",
            "epic_plan_link", "epic_link_workspace_bytes", "epic_link_attention", "epic_set_profile_events",
            "epic_model_workspace_bytes", "epic_link_layer", "epic_link_model", "epic_gemm_workspace_bytes",
            "epic_gemm", "epic_plan_decode_sizes", "epic_plan_decode", "epic_plan_compile_sizes",
            "epic_plan_compile", "epic_link_attention_noalloc"]

NOALLOC_SCRATCH_BYTES = 96 << 20      # EPIC_NOALLOC_SCRATCH_BYTES

GEMM_STORE, GEMM_RESIDUAL, GEMM_SWIGLU = 0, 1, 2


def _check(st: int, where: str):
    if st != EPIC_OK:
        raise EpicError(st, where, f"{_status_string(st).decode()}: {_last_error().decode()}")


def epic_version() -> str:
    return _version().decode()


def epic_status_string(st: int) -> str:
    return _status_string(st).decode()


# ---------------------------------------------------------------- requests and plans

@dataclass
class Request:
    """One request: chunks (lengths and physical block ids, in linked order), suffix length, k."""

    chunk_lens: List[int]
    chunk_blocks: List[List[int]]
    suffix_len: int
    k: int
    rerotate: bool = False


def attn_cfg(hq: int, hkv: int, d: int, scale: float = 0.0, split_blocks: int = 0, tile_rows: int = 0,
             rope_theta: float = 0.0) -> epic_attn_cfg:
    return epic_attn_cfg(hq, hkv, d, BLOCK, scale, split_blocks, tile_rows, rope_theta)


class _ReqArray:
    """Keeps the ctypes request array and the int32 buffers it points into alive."""

    def __init__(self, reqs: Sequence[Request]):
        self.keep = []
        self.arr = (epic_link_request * max(1, len(reqs)))()
        for i, r in enumerate(reqs):
            lens = np.asarray(r.chunk_lens, np.int32)
            off = np.zeros(len(r.chunk_lens) + 1, np.int32)
            off[1:] = np.cumsum([len(b) for b in r.chunk_blocks])
            blocks = np.asarray([x for b in r.chunk_blocks for x in b] or [0], np.int32)
            self.keep += [lens, off, blocks]
            self.arr[i] = epic_link_request(len(r.chunk_lens), lens.ctypes.data_as(_i32p),
                                            off.ctypes.data_as(_i32p), blocks.ctypes.data_as(_i32p),
                                            r.suffix_len, r.k, int(r.rerotate))
        self.n = len(reqs)


def epic_plan_sizes_get(reqs: Sequence[Request], cfg: epic_attn_cfg, n_free: int) -> epic_plan_sizes:
    ra = _ReqArray(reqs)
    s = epic_plan_sizes()
    _check(_plan_sizes_get(ra.arr, ra.n, C.byref(cfg), n_free, C.byref(s)), "epic_plan_sizes_get")
    return s


def epic_plan_layout(sizes: epic_plan_sizes, base_ptr: int) -> epic_plan:
    p = epic_plan()
    _check(_plan_layout(C.byref(sizes), C.c_void_p(base_ptr), C.byref(p)), "epic_plan_layout")
    return p


def epic_plan_link(reqs: Sequence[Request], cfg: epic_attn_cfg, free_blocks: Sequence[int], num_blocks: int):
    """Host planner.  Returns (sizes, host int32 buffer, dict of numpy views per plan array)."""
    ra = _ReqArray(reqs)
    free = np.ascontiguousarray(free_blocks, np.int32)
    sizes = epic_plan_sizes()
    _check(_plan_sizes_get(ra.arr, ra.n, C.byref(cfg), len(free), C.byref(sizes)), "epic_plan_sizes_get")
    buf = np.zeros(max(1, sizes.total_ints), np.int32)
    plan = epic_plan_layout(sizes, buf.ctypes.data)
    _check(_plan_link(ra.arr, ra.n, C.byref(cfg), free.ctypes.data_as(_i32p), len(free), num_blocks,
                      C.byref(sizes), C.byref(plan)), "epic_plan_link")
    return sizes, buf, plan_views(sizes, buf)


def epic_plan_decode(prev_sizes: epic_plan_sizes, prev_buf: np.ndarray, new_tokens: Sequence[int],
                     cfg: epic_attn_cfg, free_blocks: Sequence[int], num_blocks: int):
    """Decode planner: append new_tokens[b] tokens to request b of the previous plan
    (host buffer prev_buf of the link or a previous decode plan).  Returns (sizes,
    host int32 buffer, numpy views) of the new plan."""
    prev = epic_plan_layout(prev_sizes, prev_buf.ctypes.data)
    nt = np.ascontiguousarray(new_tokens, np.int32)
    if len(nt) != prev_sizes.batch:
        raise ValueError("new_tokens needs one entry per request")
    free = np.ascontiguousarray(free_blocks, np.int32)
    sizes = epic_plan_sizes()
    _check(_plan_decode_sizes(C.byref(prev_sizes), C.byref(prev), nt.ctypes.data_as(_i32p), C.byref(cfg), len(free),
                              C.byref(sizes)), "epic_plan_decode_sizes")
    buf = np.zeros(max(1, sizes.total_ints), np.int32)
    plan = epic_plan_layout(sizes, buf.ctypes.data)
    _check(_plan_decode(C.byref(prev_sizes), C.byref(prev), nt.ctypes.data_as(_i32p), C.byref(cfg),
                        free.ctypes.data_as(_i32p), len(free), num_blocks, C.byref(sizes), C.byref(plan)),
           "epic_plan_decode")
    return sizes, buf, plan_views(sizes, buf)


def epic_plan_compile(chunk_lens: Sequence[int], chunk_blocks: Sequence[Sequence[int]], n_dummy: int,
                      cfg: epic_attn_cfg, free_blocks: Sequence[int], num_blocks: int):
    """Compile planner: one request per chunk, S = n_dummy dummy tokens then the
    chunk's tokens; chunk_blocks[j] receive chunk j's cache (dummies dropped);
    with n_dummy > 0 the attention stages through blocks taken from free_blocks.
    Returns (sizes, host int32 buffer, numpy views)."""
    lens = np.ascontiguousarray(chunk_lens, np.int32)
    off = np.zeros(len(lens) + 1, np.int32)
    off[1:] = np.cumsum([len(b) for b in chunk_blocks])
    blocks = np.asarray([x for b in chunk_blocks for x in b] or [0], np.int32)
    cb = epic_compile_batch(len(lens), lens.ctypes.data_as(_i32p), off.ctypes.data_as(_i32p),
                            blocks.ctypes.data_as(_i32p), n_dummy)
    free = np.ascontiguousarray(free_blocks if len(free_blocks) else [0], np.int32)
    n_free = len(free_blocks)
    sizes = epic_plan_sizes()
    _check(_plan_compile_sizes(C.byref(cb), C.byref(cfg), n_free, C.byref(sizes)), "epic_plan_compile_sizes")
    buf = np.zeros(max(1, sizes.total_ints), np.int32)
    plan = epic_plan_layout(sizes, buf.ctypes.data)
    _check(_plan_compile(C.byref(cb), C.byref(cfg), free.ctypes.data_as(_i32p), n_free, num_blocks,
                         C.byref(sizes), C.byref(plan)), "epic_plan_compile")
    return sizes, buf, plan_views(sizes, buf)


def plan_views(sizes: epic_plan_sizes, buf: np.ndarray) -> dict:
    """numpy views of the plan arrays inside a host plan buffer."""
    plan = epic_plan_layout(sizes, buf.ctypes.data)
    base = buf.ctypes.data
    lens = {"s_pos": sizes.n_s, "s_req": sizes.n_s, "s_slot": sizes.n_s, "s_off": sizes.batch + 1,
            "linked_blocks": sizes.n_linked_blocks, "block_pos0": sizes.n_linked_blocks,
            "block_len": sizes.n_linked_blocks, "blk_off": sizes.batch + 1, "priv_block": sizes.n_private,
            "priv_src": sizes.n_private, "priv_rows": sizes.n_private * BLOCK, "tiles": 4 * sizes.n_tiles,
            "work": WORK_INTS * sizes.n_work, "priv_rot": sizes.n_private}
    out = {}
    for name in PLAN_FIELDS:
        addr = C.cast(getattr(plan, name), C.c_void_p).value or base
        i0 = (addr - base) // 4
        out[name] = buf[i0:i0 + lens[name]]
    return out


class DevicePlan:
    """A plan uploaded to device memory (one int32 tensor) and its device struct."""

    def __init__(self, sizes: epic_plan_sizes, host_buf: np.ndarray, device="cuda"):
        import torch

        self.sizes = sizes
        self.host = host_buf
        self.dev = torch.from_numpy(host_buf).to(device)
        self.plan = epic_plan_layout(sizes, self.dev.data_ptr())


def epic_link_workspace_bytes(cfg: epic_attn_cfg, sizes: epic_plan_sizes) -> int:
    return int(_link_ws(C.byref(cfg), C.byref(sizes)))


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    import torch

    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def epic_link_attention(cfg: epic_attn_cfg, dplan: DevicePlan, q_s, k_s, v_s, k_cache, v_cache, out, lse,
                        workspace, stream=None):
    """Enqueue one attention layer of the link step (see include/epic_link.h)."""
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_link_attention(C.byref(cfg), C.byref(dplan.sizes), C.byref(dplan.plan), _ptr(q_s), _ptr(k_s),
                           _ptr(v_s), _ptr(k_cache), _ptr(v_cache), _ptr(out), _ptr(lse), _ptr(workspace),
                           ws_bytes, _stream(stream)), "epic_link_attention")


def epic_link_attention_noalloc(cfg: epic_attn_cfg, dplan: DevicePlan, q_s, k_s, v_s, k_cache, v_cache, out, lse,
                                stream=None):
    """epic_link_attention without a workspace: split-KV partials in the library's fixed
    device array (see include/epic_link.h)."""
    _check(_link_attention_noalloc(C.byref(cfg), C.byref(dplan.sizes), C.byref(dplan.plan), _ptr(q_s), _ptr(k_s),
                                   _ptr(v_s), _ptr(k_cache), _ptr(v_cache), _ptr(out), _ptr(lse), _stream(stream)),
           "epic_link_attention_noalloc")


def epic_set_profile_events(events=None):
    """events: None, or 4 torch.cuda.Event (or None entries) recorded around the step's kernels.

    torch creates an event's HIP handle on its first record(); record each event once beforehand."""
    if events is None:
        _check(_set_prof(None), "epic_set_profile_events")
        return
    handles = [None if e is None else e.cuda_event for e in events]
    if any(h == 0 for h in handles):
        raise ValueError("epic_set_profile_events: an event has no HIP handle yet (record it once first)")
    arr = (C.c_void_p * 4)(*handles)
    _check(_set_prof(C.cast(arr, C.c_void_p)), "epic_set_profile_events")


def epic_model_workspace_bytes(cfg: epic_model_cfg, sizes: epic_plan_sizes) -> int:
    return int(_model_ws(C.byref(cfg), C.byref(sizes)))


def epic_link_layer(cfg: epic_model_cfg, weights: epic_layer_weights, dplan: DevicePlan, hidden_s, k_cache,
                    v_cache, workspace, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_link_layer(C.byref(cfg), C.byref(weights), C.byref(dplan.sizes), C.byref(dplan.plan), _ptr(hidden_s),
                       _ptr(k_cache), _ptr(v_cache), _ptr(workspace), ws_bytes, _stream(stream)),
           "epic_link_layer")


def epic_link_model(cfg: epic_model_cfg, layers: Sequence[epic_layer_weights], final_norm, dplan: DevicePlan,
                    hidden_s, k_caches: Sequence, v_caches: Sequence, out_hidden, workspace, stream=None):
    n = len(layers)
    warr = (epic_layer_weights * n)(*layers)
    karr = (C.c_void_p * n)(*[t.data_ptr() for t in k_caches])
    varr = (C.c_void_p * n)(*[t.data_ptr() for t in v_caches])
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_link_model(C.byref(cfg), warr, _ptr(final_norm), C.byref(dplan.sizes), C.byref(dplan.plan),
                       _ptr(hidden_s), karr, varr, _ptr(out_hidden), _ptr(workspace), ws_bytes, _stream(stream)),
           "epic_link_model")


def epic_gemm_workspace_bytes() -> int:
    return int(_gemm_ws())


def epic_gemm(epilogue: int, a, w, c=None, act=None, workspace=None, stream=None):
    """Enqueue the projection GEMM (see include/epic_link.h): a bf16 [m, k], w bf16 [n, k];
    c fp32 [m, n] (store / residual) or act bf16 [m, n/2] (SwiGLU)."""
    m, k = a.shape
    n = w.shape[0]
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_gemm(epilogue, _ptr(a), _ptr(w), m, n, k, _ptr(c), _ptr(act), _ptr(workspace), ws_bytes,
                 _stream(stream)), "epic_gemm")


# ---------------------------------------------------------------- cache layout helpers

def pack_blocks(k_rows: np.ndarray, v_rows: np.ndarray):
    """Token-major K/V [L, Hkv, D] (bf16 bits) -> block layouts for ceil(L/16) blocks:
    K [nb, Hkv, 16, D] and V [nb, Hkv, D, 16]; slots past L are zero."""
    L, hkv, d = k_rows.shape
    nb = -(-L // BLOCK)
    kp = np.zeros((nb * BLOCK, hkv, d), np.uint16)
    vp = np.zeros((nb * BLOCK, hkv, d), np.uint16)
    kp[:L] = k_rows
    vp[:L] = v_rows
    kb = kp.reshape(nb, BLOCK, hkv, d).transpose(0, 2, 1, 3)
    vb = vp.reshape(nb, BLOCK, hkv, d).transpose(0, 2, 3, 1)
    return np.ascontiguousarray(kb), np.ascontiguousarray(vb)


def read_linked_kv(k_cache: np.ndarray, v_cache: np.ndarray, views: dict, req: int):
    """Token-major K/V [N, Hkv, D] of request `req` read through its linked block table."""
    b0, b1 = int(views["blk_off"][req]), int(views["blk_off"][req + 1])
    ks, vs = [], []
    for b in range(b0, b1):
        phys, n = int(views["linked_blocks"][b]), int(views["block_len"][b])
        ks.append(k_cache[phys].transpose(1, 0, 2)[:n])
        vs.append(v_cache[phys].transpose(2, 0, 1)[:n])
    return np.concatenate(ks), np.concatenate(vs)
