"""ctypes binding of the C-ABI declared in include/boost_cap.h.

Argument marshalling only: every function below converts Python values to C
arguments, calls the entry point of the same name and turns a negative status
into ``BoostError``.  No computation happens here and there is no fallback:
if the library is missing, ``load()`` raises.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# BOOST_LIB may name another build of the same library: the host-sanitizer
# build used by the CPU tests (python -m paper_2609_13592_amd.build --sanitize)
_LIB_PATH = os.environ.get("BOOST_LIB") or os.path.join(HERE, "_lib", "libboostcap.so")

OK, EINVAL, ENOMEM, EAGAIN, ENODEV, EHIP = 0, -22, -12, -11, -19, -5
KV_LPP, KV_ALL_HBM, KV_ALL_HOST, KV_BUDGET = 0, 1, 2, 3
KV_LOCAL, KV_SHH = 0, 1
TIER_HBM, TIER_HOST = 0, 1
PLACE_MPP, PLACE_MPP_GLOBAL, PLACE_LINEAR, PLACE_RANDOM = 0, 1, 2, 3
DTYPE_F32, DTYPE_BF16 = 0, 1
SCHED_ADDRESS, SCHED_CAP = 0, 1
PAGE_BYTES = 2 * 1024 * 1024

_vp = C.c_void_p
_u64 = C.c_uint64
_u32 = C.c_uint32
_i32 = C.c_int
_dbl = C.c_double


class BoostError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"boost error {code}: {msg}")
        self.code = code


class KVCfg(C.Structure):
    _fields_ = [("layers", _u32), ("kv_heads", _u32), ("head_dim", _u32),
                ("block_tokens", _u32), ("n_blocks", _u32), ("M", _u32),
                ("tier_mode", _i32), ("q_heads", _u32), ("max_batch", _u32),
                ("max_blocks_per_seq", _u32), ("hbm_budget_bytes", _u64)]


class KVInfo(C.Structure):
    _fields_ = [("nb_pool", _u32), ("blocks_per_page", _u32),
                ("pages_per_tensor", _u64), ("host_pages_per_tensor", _u64),
                ("n_shh", _u32), ("shh_host_heads", _u32),
                ("local_host_heads", _u32), ("tau", _dbl)]


class KVStats(C.Structure):
    _fields_ = [("free_shh", _u32), ("free_local", _u32),
                ("used_blocks", _u64), ("used_host_head_blocks", _u64),
                ("requests", _u32), ("shh_requests", _u32)]


_SIGS = {
    "boost_last_error": (C.c_char_p, []),
    "boost_version": (_i32, []),
    "boost_init": (_i32, [_i32, C.POINTER(_vp)]),
    "boost_shutdown": (_i32, [_vp]),
    "boost_ctx_info": (_i32, [_vp, C.POINTER(_i32), C.POINTER(_i32)]),
    "boost_set_host_coherent": (_i32, [_vp, _i32]),
    "boost_set_host_numa": (_i32, [_vp, _i32]),
    "boost_host_numa_info": (_i32, [_vp, C.POINTER(_i32), C.POINTER(_i32), C.POINTER(_i32)]),
    "boost_calibrate": (_i32, [_vp, _u64, _u64, _i32, C.POINTER(_dbl),
                               C.POINTER(_dbl), C.POINTER(_dbl)]),
    "boost_stream_read_gbps": (_i32, [_vp, _vp, _u64, _i32, _i32, C.POINTER(_dbl)]),
    "boost_cap_sweep": (_i32, [_vp, _u64, _u64, _i32, _vp, _i32, _vp]),
    "boost_modulus_from_alpha": (_i32, [_dbl, C.POINTER(_u32)]),
    "boost_superpage_pages": (_i32, [_u64, C.POINTER(_u32)]),
    "boost_plan_mpp": (_i32, [_u64, _u32, _u64, _vp, _u64, C.POINTER(_u64)]),
    "boost_plan_contrast": (_i32, [_i32, _u64, _u32, _u64, _vp, _vp, _u64,
                                   C.POINTER(_u64)]),
    "boost_modulus_from_budget": (_i32, [_vp, _vp, C.c_size_t, _u64, _u32,
                                         C.POINTER(_u32)]),
    "boost_place_weights": (_i32, [_vp, _vp, _u64, _u32, _u64, C.POINTER(_vp)]),
    "boost_place_weights_map": (_i32, [_vp, _vp, _u64, _vp, _u64, C.POINTER(_vp)]),
    "boost_tensor_tiers": (_i32, [_vp, _vp, _u64, C.POINTER(_u64)]),
    "boost_tensor_layout": (_i32, [_vp, C.POINTER(_i32), C.POINTER(_i32)]),
    "boost_tensor_read": (_i32, [_vp, _u64, _vp, _u64]),
    "boost_tensor_free": (_i32, [_vp]),
    "boost_gemv_set_schedule": (_i32, [_vp, _i32, _i32]),
    "boost_embed_gather": (_i32, [_vp, _vp, _i32, _i32, _vp, _i32, _vp, _vp]),
    "boost_rmsnorm": (_i32, [_vp, _vp, _vp, _i32, _i32, C.c_float, _vp, _vp]),
    "boost_add_rmsnorm": (_i32, [_vp, _vp, _vp, _vp, _i32, _i32, C.c_float, _vp, _vp]),
    "boost_add_rmsnorm_slices": (_i32, [_vp, _vp, _vp, _i32, _i32, _vp, _i32, _i32, C.c_float,
                                        _vp, _vp]),
    "boost_rope_qkv": (_i32, [_vp, _vp, _vp, _i32, _i32, _i32, _i32, _dbl, _vp, _vp,
                              _vp, _vp]),
    "boost_kv_append": (_i32, [_vp, _vp, _i32, _vp, _i32, _vp, _vp, _vp, _i32, _vp]),
    "boost_rope_kv_append": (_i32, [_vp, _vp, _i32, _vp, _vp, _i32, _i32, _dbl, _vp, _i32,
                                    _vp, _vp]),
    "boost_rope_kv_append_slices": (_i32, [_vp, _vp, _i32, _vp, _i32, _i32, _vp, _i32, _i32,
                                           _dbl, _vp, _i32, _vp, _vp]),
    "boost_silu_mul": (_i32, [_vp, _vp, _i32, _i32, _vp, _vp]),
    "boost_residual_add": (_i32, [_vp, _vp, _vp, C.c_int64, _vp]),
    "boost_argmax": (_i32, [_vp, _vp, _i32, _i32, _vp, _vp]),
    "boost_staged_view": (_i32, [_vp, _vp, _vp, _u64, C.POINTER(_vp)]),
    "boost_prefetch": (_i32, [_vp, _vp, _vp]),
    "boost_kv_pool_create": (_i32, [_vp, C.POINTER(KVCfg), C.POINTER(_vp)]),
    "boost_kv_pool_info": (_i32, [_vp, C.POINTER(KVInfo)]),
    "boost_kv_pool_destroy": (_i32, [_vp]),
    "boost_kv_block_host_heads": (_i32, [_vp, C.c_int32, C.POINTER(_u32)]),
    "boost_kv_alloc": (_i32, [_vp, _u64, _u32, _vp]),
    "boost_kv_free": (_i32, [_vp, _u64]),
    "boost_kv_request_type": (_i32, [_vp, _u64, C.POINTER(_i32)]),
    "boost_kv_stats": (_i32, [_vp, C.POINTER(KVStats)]),
    "boost_kv_write": (_i32, [_vp, _vp, _i32, _vp, _vp, _vp, _i32, _vp]),
    "boost_paged_attn_decode": (_i32, [_vp, _vp, _i32, _vp, _i32, _i32, _vp, _i32,
                                       _vp, C.c_float, _vp, _i32, _vp]),
    "boost_paged_attn_decode_noalloc": (_i32, [_vp, _vp, _i32, _vp, _i32, _i32, _vp, _i32,
                                               _vp, C.c_float, _vp, _i32, _vp]),
    "boost_decode_gemv": (_i32, [_vp, _vp, _i32, _i32, _vp, _i32, _vp, _i32, _vp]),
    "boost_decode_gemv_slices": (_i32, [_vp, _vp, _i32, _i32, _vp, _i32, _vp, _i32,
                                        C.POINTER(_i32), _vp]),
    "boost_gemv_slices_floats": (_i32, [_i32, _i32, _i32, _i32, C.POINTER(_u64)]),
}

_lib = None


def lib_path() -> str:
    return _LIB_PATH


def load():
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is missing: build it with "
                          "`python -m paper_2609_13592_amd.build`")
    # One HIP runtime per process: torch ships its own libamdhip64 (same
    # soname).  Loading torch first makes the library bind to that copy
    # instead of pulling in a second runtime that would see no device.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = C.CDLL(_LIB_PATH)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name, None)
        if fn is None:
            continue
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(rc: int):
    if rc < 0:
        msg = load().boost_last_error().decode(errors="replace")
        raise BoostError(rc, msg)
    return rc


def _ptr(a) -> int:
    """Address of a numpy array, torch tensor or integer."""
    if a is None:
        return 0
    if isinstance(a, int):
        return a
    if isinstance(a, np.ndarray):
        assert a.flags["C_CONTIGUOUS"]
        return a.ctypes.data
    if hasattr(a, "data_ptr"):
        return a.data_ptr()
    raise TypeError(type(a))


def _stream(s) -> int:
    if s is None:
        return 0
    if isinstance(s, int):
        return s
    return s.cuda_stream


# ------------------------------------------------------------------ context
def boost_version() -> int:
    return load().boost_version()


def _runtime_first(device: int):
    """PyTorch and the library share one HIP runtime in this process; let
    torch create its device context before the library touches the device."""
    import sys
    torch = sys.modules.get("torch")
    if torch is None or device < 0:
        return
    torch.cuda.init()
    torch.empty(1, device=f"cuda:{device}")


def boost_init(device: int) -> int:
    _runtime_first(device)
    h = _vp()
    _check(load().boost_init(device, C.byref(h)))
    return h.value


def boost_shutdown(ctx: int):
    _check(load().boost_shutdown(ctx))


def boost_ctx_info(ctx: int):
    d, n = _i32(), _i32()
    _check(load().boost_ctx_info(ctx, C.byref(d), C.byref(n)))
    return d.value, n.value


def boost_set_host_coherent(ctx: int, coherent: bool):
    _check(load().boost_set_host_coherent(ctx, int(bool(coherent))))


NUMA_DEVICE = -1


def boost_set_host_numa(ctx: int, node: int):
    _check(load().boost_set_host_numa(ctx, node))


def boost_host_numa_info(ctx: int) -> dict:
    dn, n, node = C.c_int32(0), C.c_int32(0), C.c_int32(0)
    _check(load().boost_host_numa_info(ctx, C.byref(dn), C.byref(n), C.byref(node)))
    return {"device_node": dn.value, "n_nodes": n.value, "node": node.value}


# -------------------------------------------------------------- calibration
def boost_calibrate(ctx: int, hbm_bytes: int, host_bytes: int, iters: int):
    d, h, a = _dbl(), _dbl(), _dbl()
    _check(load().boost_calibrate(ctx, hbm_bytes, host_bytes, iters, C.byref(d),
                                  C.byref(h), C.byref(a)))
    return d.value, h.value, a.value


def boost_stream_read_gbps(ctx: int, src, nbytes: int, grid: int, iters: int) -> float:
    g = _dbl()
    _check(load().boost_stream_read_gbps(ctx, _ptr(src), nbytes, grid, iters,
                                         C.byref(g)))
    return g.value


CAP_POINT = np.dtype([("hbm_bytes", np.uint64), ("host_bytes", np.uint64),
                      ("hbm_wgs", np.int32), ("host_wgs", np.int32),
                      ("host_stride", np.int32), ("host_depth", np.int32),
                      ("host_policy", np.int32), ("dma", np.int32),
                      ("hbm_chunk_kib", np.int32), ("chunk_static", np.int32)])


def boost_cap_sweep(ctx: int, hbm_bytes: int, host_bytes: int, points, iters: int):
    """points: dicts with the fields of boost_cap_point (missing ones: bytes and
    workgroups 0, stride 1, depth 8, policy 0, dma 0, chunk 0); returns an array
    [n_points, 16] laid out as the header states."""
    n = len(points)
    arr = np.zeros(n, dtype=CAP_POINT)
    for i, p in enumerate(points):
        arr[i] = (p.get("hbm_bytes", 0), p.get("host_bytes", 0), p.get("hbm_wgs", 0),
                  p.get("host_wgs", 0), p.get("host_stride", 1), p.get("host_depth", 8),
                  p.get("host_policy", 0), p.get("dma", 0), p.get("hbm_chunk_kib", 0),
                  p.get("chunk_static", 0))
    res = np.zeros((n, 16), dtype=np.float64)
    _check(load().boost_cap_sweep(ctx, hbm_bytes, host_bytes, n, arr.ctypes.data, iters,
                                  res.ctypes.data))
    return res


def boost_modulus_from_alpha(alpha: float) -> int:
    m = _u32()
    _check(load().boost_modulus_from_alpha(alpha, C.byref(m)))
    return m.value


# ---------------------------------------------------------------- placement
def boost_superpage_pages(footprint: int) -> int:
    s = _u32()
    _check(load().boost_superpage_pages(footprint, C.byref(s)))
    return s.value


def boost_plan_mpp(nbytes: int, M: int, footprint: int = 0) -> np.ndarray:
    n = _u64()
    _check(load().boost_plan_mpp(nbytes, M, footprint, None, 0, C.byref(n)))
    out = np.zeros(n.value, dtype=np.uint8)
    _check(load().boost_plan_mpp(nbytes, M, footprint, _ptr(out), out.size,
                                 C.byref(n)))
    return out


def boost_plan_contrast(kind: int, nbytes: int, M: int, phase: int = 0,
                        uniforms=None) -> np.ndarray:
    n = -(-int(nbytes) // PAGE_BYTES)
    u = None if uniforms is None else np.ascontiguousarray(uniforms, dtype=np.float64)
    if u is not None and u.size < n:
        raise ValueError(f"{n} uniforms needed, {u.size} given")
    out = np.zeros(max(n, 1), dtype=np.uint8)
    got = _u64()
    _check(load().boost_plan_contrast(kind, nbytes, M, phase, _ptr(u), _ptr(out),
                                      out.size, C.byref(got)))
    return out[:got.value]


def boost_modulus_from_budget(sizes, budget: int, M_alpha: int, footprints=None) -> int:
    s = np.ascontiguousarray(sizes, dtype=np.uint64)
    f = None if footprints is None else np.ascontiguousarray(footprints, dtype=np.uint64)
    m = _u32()
    _check(load().boost_modulus_from_budget(_ptr(s), _ptr(f), s.size, budget,
                                            M_alpha, C.byref(m)))
    return m.value


def boost_place_weights(ctx: int, src, nbytes: int, M: int, footprint: int = 0) -> int:
    h = _vp()
    _check(load().boost_place_weights(ctx, _ptr(src), nbytes, M, footprint,
                                      C.byref(h)))
    return h.value


def boost_place_weights_map(ctx: int, src, nbytes: int, tiers) -> int:
    t = np.ascontiguousarray(tiers, dtype=np.uint8)
    h = _vp()
    _check(load().boost_place_weights_map(ctx, _ptr(src), nbytes, _ptr(t), t.size,
                                          C.byref(h)))
    return h.value


def boost_tensor_layout(t: int):
    """(M, SP) of the tensor's closed-form map, M = -1 when it has none."""
    m, sp = C.c_int32(0), C.c_int32(0)
    _check(load().boost_tensor_layout(t, C.byref(m), C.byref(sp)))
    return m.value, sp.value


def boost_tensor_tiers(t: int) -> np.ndarray:
    n = _u64()
    _check(load().boost_tensor_tiers(t, None, 0, C.byref(n)))
    out = np.zeros(n.value, dtype=np.uint8)
    _check(load().boost_tensor_tiers(t, _ptr(out), out.size, C.byref(n)))
    return out


def boost_tensor_read(t: int, offset: int, nbytes: int) -> np.ndarray:
    out = np.zeros(nbytes, dtype=np.uint8)
    _check(load().boost_tensor_read(t, offset, _ptr(out), nbytes))
    return out


def boost_tensor_free(t: int):
    _check(load().boost_tensor_free(t))


# ------------------------------------------------------- prefetch baseline
def boost_staged_view(ctx: int, t: int, staging, staging_bytes: int) -> int:
    h = _vp()
    _check(load().boost_staged_view(ctx, t, _ptr(staging), staging_bytes, C.byref(h)))
    return h.value


def boost_prefetch(ctx: int, view: int, stream=None):
    _check(load().boost_prefetch(ctx, view, _stream(stream)))


# -------------------------------------------------------------------- GEMV
def boost_gemv_set_schedule(ctx: int, schedule: int, host_workers: int = 0):
    _check(load().boost_gemv_set_schedule(ctx, schedule, host_workers))


def boost_decode_gemv(ctx: int, W: int, N: int, K: int, x, B: int, y,
                      y_dtype: int = DTYPE_F32, stream=None):
    _check(load().boost_decode_gemv(ctx, W, N, K, _ptr(x), B, _ptr(y), y_dtype,
                                    _stream(stream)))


MAX_GEMV_SLICES = 8


def boost_gemv_slices_floats(N: int, K: int, B: int, max_slices: int) -> int:
    n = _u64(0)
    _check(load().boost_gemv_slices_floats(N, K, B, max_slices, C.byref(n)))
    return n.value


def boost_decode_gemv_slices(ctx: int, W: int, N: int, K: int, x, B: int, slices,
                             max_slices: int, stream=None) -> int:
    """Writes the split-K partial slices (fp32 [S][B][N], then the parts of
    rows that cross a page) and returns S."""
    n = C.c_int32(0)
    _check(load().boost_decode_gemv_slices(ctx, W, N, K, _ptr(x), B, _ptr(slices), max_slices,
                                           C.byref(n), _stream(stream)))
    return n.value


# ------------------------------------------------------------- KV pool / DSR
def boost_kv_pool_create(ctx: int, layers: int, kv_heads: int, head_dim: int,
                         n_blocks: int, M: int, tier_mode: int = KV_LPP,
                         q_heads: int = 0, max_batch: int = 0,
                         max_blocks_per_seq: int = 0, block_tokens: int = 16,
                         hbm_budget_bytes: int = 0) -> int:
    cfg = KVCfg(layers, kv_heads, head_dim, block_tokens, n_blocks, M, tier_mode,
                q_heads or kv_heads, max_batch, max_blocks_per_seq, hbm_budget_bytes)
    h = _vp()
    _check(load().boost_kv_pool_create(ctx, C.byref(cfg), C.byref(h)))
    return h.value


def boost_kv_pool_info(pool: int) -> dict:
    i = KVInfo()
    _check(load().boost_kv_pool_info(pool, C.byref(i)))
    return {f: getattr(i, f) for f, _ in KVInfo._fields_}


def boost_kv_pool_destroy(pool: int):
    _check(load().boost_kv_pool_destroy(pool))


def boost_kv_block_host_heads(pool: int, block: int) -> int:
    n = _u32()
    _check(load().boost_kv_block_host_heads(pool, block, C.byref(n)))
    return n.value


def boost_kv_alloc(pool: int, request_id: int, n_blocks: int):
    """Block ids as a list, or EAGAIN (the int) when the pool cannot serve."""
    out = np.zeros(max(n_blocks, 1), dtype=np.int32)
    rc = load().boost_kv_alloc(pool, request_id, n_blocks, _ptr(out))
    if rc == EAGAIN:
        return EAGAIN
    _check(rc)
    return out[:n_blocks].tolist()


def boost_kv_free(pool: int, request_id: int):
    _check(load().boost_kv_free(pool, request_id))


def boost_kv_request_type(pool: int, request_id: int) -> int:
    t = _i32()
    _check(load().boost_kv_request_type(pool, request_id, C.byref(t)))
    return t.value


def boost_kv_stats(pool: int) -> dict:
    st = KVStats()
    _check(load().boost_kv_stats(pool, C.byref(st)))
    return {f: getattr(st, f) for f, _ in KVStats._fields_}


def boost_kv_write(ctx: int, pool: int, layer: int, slots, k, v, n: int, stream=None):
    _check(load().boost_kv_write(ctx, pool, layer, _ptr(slots), _ptr(k), _ptr(v), n,
                                 _stream(stream)))


def boost_paged_attn_decode(ctx: int, pool: int, layer: int, q, B: int, Hq: int,
                            block_tables, max_blocks: int, ctx_lens, scale: float,
                            out, out_dtype: int = DTYPE_F32, stream=None):
    _check(load().boost_paged_attn_decode(ctx, pool, layer, _ptr(q), B, Hq,
                                          _ptr(block_tables), max_blocks,
                                          _ptr(ctx_lens), scale, _ptr(out), out_dtype,
                                          _stream(stream)))


def boost_paged_attn_decode_noalloc(ctx: int, pool: int, layer: int, q, B: int, Hq: int,
                                    block_tables, max_blocks: int, ctx_lens, scale: float,
                                    out, out_dtype: int = DTYPE_F32, stream=None):
    _check(load().boost_paged_attn_decode_noalloc(ctx, pool, layer, _ptr(q), B, Hq,
                                                  _ptr(block_tables), max_blocks,
                                                  _ptr(ctx_lens), scale, _ptr(out),
                                                  out_dtype, _stream(stream)))


# ---------------------------------------------------------- decode-step glue
def boost_embed_gather(ctx: int, E: int, V: int, d: int, tokens, B: int, out, stream=None):
    _check(load().boost_embed_gather(ctx, E, V, d, _ptr(tokens), B, _ptr(out),
                                     _stream(stream)))


def boost_rmsnorm(ctx: int, x, w, B: int, d: int, eps: float, out, stream=None):
    _check(load().boost_rmsnorm(ctx, _ptr(x), _ptr(w), B, d, eps, _ptr(out),
                                _stream(stream)))


def boost_add_rmsnorm(ctx: int, x, r, w, B: int, d: int, eps: float, out, stream=None):
    _check(load().boost_add_rmsnorm(ctx, _ptr(x), _ptr(r), _ptr(w), B, d, eps, _ptr(out),
                                    _stream(stream)))


def boost_add_rmsnorm_slices(ctx: int, x, r, S: int, K: int, w, B: int, d: int, eps: float,
                             out, stream=None):
    _check(load().boost_add_rmsnorm_slices(ctx, _ptr(x), _ptr(r), S, K, _ptr(w), B, d, eps,
                                           _ptr(out), _stream(stream)))


def boost_rope_qkv(ctx: int, qkv, positions, B: int, Hq: int, H: int, D: int,
                   theta: float, q, k, v, stream=None):
    _check(load().boost_rope_qkv(ctx, _ptr(qkv), _ptr(positions), B, Hq, H, D, theta,
                                 _ptr(q), _ptr(k), _ptr(v), _stream(stream)))


def boost_kv_append(ctx: int, pool: int, layer: int, block_tables, max_blocks: int,
                    positions, k, v, B: int, stream=None):
    _check(load().boost_kv_append(ctx, pool, layer, _ptr(block_tables), max_blocks,
                                  _ptr(positions), _ptr(k), _ptr(v), B, _stream(stream)))


def boost_rope_kv_append(ctx: int, pool: int, layer: int, qkv, positions, B: int, Hq: int,
                         theta: float, block_tables, max_blocks: int, q, stream=None):
    _check(load().boost_rope_kv_append(ctx, pool, layer, _ptr(qkv), _ptr(positions), B, Hq,
                                       theta, _ptr(block_tables), max_blocks, _ptr(q),
                                       _stream(stream)))


def boost_rope_kv_append_slices(ctx: int, pool: int, layer: int, qkv, S: int, K: int,
                                positions, B: int, Hq: int, theta: float, block_tables,
                                max_blocks: int, q, stream=None):
    _check(load().boost_rope_kv_append_slices(ctx, pool, layer, _ptr(qkv), S, K,
                                              _ptr(positions), B, Hq, theta, _ptr(block_tables),
                                              max_blocks, _ptr(q), _stream(stream)))


def boost_silu_mul(ctx: int, gu, B: int, F: int, out, stream=None):
    _check(load().boost_silu_mul(ctx, _ptr(gu), B, F, _ptr(out), _stream(stream)))


def boost_residual_add(ctx: int, x, y, n: int, stream=None):
    _check(load().boost_residual_add(ctx, _ptr(x), _ptr(y), n, _stream(stream)))


def boost_argmax(ctx: int, logits, B: int, V: int, ids, stream=None):
    _check(load().boost_argmax(ctx, _ptr(logits), B, V, _ptr(ids), _stream(stream)))
