"""ctypes binding of ``include/pallas.h``.

Argument marshalling only: torch tensors become device pointers, Python
lists become host arrays, the current torch stream becomes the hipStream_t.
Every step of the computation runs in the HIP library.
"""
from __future__ import annotations

import ctypes as C
import enum
import os
from typing import List, Optional, Sequence

PKG = os.path.dirname(os.path.abspath(__file__))


def library_path() -> str:
    return os.path.join(PKG, "libpallas.so")


class Status(enum.IntEnum):
    OK = 0
    INVALID_ARG = 1
    OUT_OF_RANGE = 2
    COVERAGE = 3
    STALE_EPOCH = 4
    WRONG_REQUEST = 5
    UNSUPPORTED = 6
    HIP = 7
    WORKSPACE = 8


class PallasError(RuntimeError):
    def __init__(self, status: int, msg: str):
        self.status = Status(status)
        super().__init__(f"{self.status.name}: {msg}")


# ------------------------------------------------------------------ structs
class ModelConfigC(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("hidden", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn", C.c_int32),
                ("vocab", C.c_int32), ("rms_eps", C.c_float), ("rope_theta", C.c_float),
                ("qk_norm", C.c_int32), ("page_size", C.c_int32)]


class LayerWeightsC(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("attn_norm", "w_qkv", "q_norm", "k_norm", "w_o",
                                          "mlp_norm", "w_gate_up", "w_down")]


class WeightsC(C.Structure):
    _fields_ = [("embed", C.c_void_p), ("final_norm", C.c_void_p), ("lm_head", C.c_void_p),
                ("layers", C.POINTER(LayerWeightsC))]


class KVPoolC(C.Structure):
    _fields_ = [("base", C.c_void_p), ("num_pages", C.c_int32), ("page_size", C.c_int32),
                ("n_layers", C.c_int32), ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32)]


class ChunkDesc(C.Structure):
    _fields_ = [("start_pos", C.c_int32), ("num_tokens", C.c_int32), ("arena_offset", C.c_uint64)]


class ChunkHeader(C.Structure):
    _fields_ = [("request_id", C.c_uint64), ("epoch", C.c_uint64), ("start_pos", C.c_int32),
                ("num_tokens", C.c_int32), ("arena_offset", C.c_uint64), ("n_layers", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("elem_bytes", C.c_int32)]


class WindowParams(C.Structure):
    _fields_ = [(n, C.c_double) for n in ("r_p", "r_d", "goodput", "s_kv", "t_load", "t_0", "alpha",
                                          "t_max", "dt")]


class WindowDecision(C.Structure):
    _fields_ = [(n, C.c_double) for n in ("t_w", "cost", "t_sit", "t_early", "t_hist", "t_res",
                                          "l_hist")] + [("n_candidates", C.c_int32), ("trigger", C.c_int32)]


class Ewma(C.Structure):
    _fields_ = [("value", C.c_double), ("primed", C.c_int32)]


_vp, _i32, _u64, _sz = C.c_void_p, C.c_int32, C.c_uint64, C.c_size_t
_pi32 = C.POINTER(C.c_int32)

# name -> (restype, argtypes); mirrors include/pallas.h
EXPORTS = {
    "pallas_abi_version": (_i32, []),
    "pallas_last_error": (C.c_char_p, []),
    "pallas_model_create": (C.c_int, [C.POINTER(ModelConfigC), C.POINTER(WeightsC), C.POINTER(_vp)]),
    "pallas_model_destroy": (None, [_vp]),
    "pallas_workspace_size": (_sz, [_vp, _i32, _i32]),
    "pallas_prefill_prefix": (C.c_int, [_vp, _i32, _vp, _pi32, _vp, _i32, C.POINTER(KVPoolC),
                                        _vp, _sz, _vp, _vp]),
    "pallas_prefill_chunk": (C.c_int, [_vp, _i32, _vp, _pi32, _pi32, _vp, _i32, C.POINTER(KVPoolC),
                                       _vp, _sz, _vp, _vp]),
    "pallas_pack_suffix_blocks": (C.c_int, [C.POINTER(KVPoolC), _vp, _i32, C.POINTER(ChunkDesc),
                                            _i32, _vp, _sz, _vp, _vp]),
    "pallas_assemble_kv": (C.c_int, [C.POINTER(KVPoolC), _vp, _i32, C.POINTER(ChunkHeader), _vp,
                                     _sz, _i32, _u64, _u64, _vp, _vp]),
    "pallas_decode_step": (C.c_int, [_vp, _i32, _vp, _pi32, _vp, _i32, C.POINTER(KVPoolC), _vp,
                                     _vp, _sz, _vp, _vp]),
    "pallas_decode_step_static": (C.c_int, [_vp, _i32, _vp, _pi32, _vp, _i32, C.POINTER(KVPoolC), _vp,
                                            _vp, _vp]),
    "pallas_check_coverage": (C.c_int, [_i32, _pi32, _pi32, _i32, _i32]),
    "pallas_window_evaluate": (C.c_int, [C.POINTER(WindowParams), C.c_double, C.c_double, C.c_double,
                                         C.POINTER(WindowDecision)]),
    "pallas_window_select": (C.c_int, [C.POINTER(WindowParams), C.c_double, C.c_double,
                                       C.POINTER(WindowDecision)]),
    "pallas_ewma_update": (C.c_double, [C.POINTER(Ewma), C.c_double, C.c_double]),
    "pallas_admit": (_i32, [_i32, C.c_double, C.c_double, C.c_double, C.c_double, C.c_double]),
    "pallas_waste_bound": (C.c_double, [C.c_double, C.c_double, C.c_double]),
    "pallas_profile_enable": (None, [C.c_uint32]),
    "pallas_profile_read": (C.c_int, [C.POINTER(C.c_double), C.POINTER(C.c_int64)]),
    "pallas_profile_reset": (None, []),
    "pallas_profile_clock": (C.c_int, [_i32, C.POINTER(C.c_double), C.POINTER(C.c_int64)]),
}

KERNEL_CLASSES = ("embed", "rmsnorm", "rope_table", "gemm_qkv", "qkv_epilogue", "attention",
                  "gemm_o", "gemm_gate_up", "gemm_down", "pack", "assemble", "decode_proj",
                  "decode_attention")

_LIB = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _LIB
    if _LIB is None:
        path = library_path()
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with `python -m "
                               "paper_2608_16477_amd.build` (there is no fallback path)")
        h = C.CDLL(path)
        for name, (res, args) in EXPORTS.items():
            f = getattr(h, name)
            f.restype = res
            f.argtypes = args
        _LIB = h
    return _LIB


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _i32_array(vals: Sequence[int]):
    arr = (C.c_int32 * max(1, len(vals)))(*[int(v) for v in vals])
    return arr


def _check(rc: int):
    if rc != 0:
        raise PallasError(rc, pallas_last_error())


def pallas_abi_version() -> int:
    return lib().pallas_abi_version()


def pallas_last_error() -> str:
    return lib().pallas_last_error().decode()


def pallas_check_coverage(prefix_len: int, starts: Sequence[int], lens: Sequence[int], n: int) -> Status:
    """Returns the status (OK or COVERAGE / INVALID_ARG); does not raise."""
    return Status(lib().pallas_check_coverage(prefix_len, _i32_array(starts), _i32_array(lens),
                                              len(starts), n))


def kv_pool_struct(pool) -> KVPoolC:
    """``pool``: bf16 tensor [L, 2, P, page, Hkv, d]."""
    L, two, P, page, hkv, d = pool.shape
    assert two == 2
    return KVPoolC(pool.data_ptr(), P, page, L, hkv, d)


def pallas_pack_suffix_blocks(pool, src_block_table, descs: Sequence[ChunkDesc], arena,
                              err=None, stream=None):
    arr = (ChunkDesc * max(1, len(descs)))(*descs)
    ps = kv_pool_struct(pool)
    _check(lib().pallas_pack_suffix_blocks(C.byref(ps), _ptr(src_block_table),
                                           src_block_table.shape[-1], arr, len(descs),
                                           _ptr(arena), arena.numel() * arena.element_size(),
                                           _ptr(err), _stream(stream)))


def pallas_assemble_kv(pool, dst_block_table, hdrs: Sequence[ChunkHeader], arena,
                       expected_request_id: int, expected_epoch: int, err=None, stream=None):
    arr = (ChunkHeader * max(1, len(hdrs)))(*hdrs)
    ps = kv_pool_struct(pool)
    nbytes = 0 if arena is None else arena.numel() * arena.element_size()
    _check(lib().pallas_assemble_kv(C.byref(ps), _ptr(dst_block_table), dst_block_table.shape[-1],
                                    arr, _ptr(arena), nbytes, len(hdrs), expected_request_id,
                                    expected_epoch, _ptr(err), _stream(stream)))


def pallas_model_create(cfg, glob, layers):
    """Returns ``(handle, keepalive)``; ``glob``/``layers`` are dicts of bf16
    device tensors named as in ``pallas_layer_weights`` / ``pallas_weights``."""
    c = ModelConfigC(cfg.n_layers, cfg.hidden, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim,
                     cfg.ffn, cfg.vocab, cfg.rms_eps, cfg.rope_theta, int(bool(cfg.qk_norm)),
                     cfg.page_size)
    la = (LayerWeightsC * cfg.n_layers)()
    for i, l in enumerate(layers):
        for name, _ in LayerWeightsC._fields_:
            setattr(la[i], name, l[name].data_ptr())
    w = WeightsC(glob["embed"].data_ptr(), glob["final_norm"].data_ptr(),
                 glob["lm_head"].data_ptr(), la)
    h = C.c_void_p()
    _check(lib().pallas_model_create(C.byref(c), C.byref(w), C.byref(h)))
    return h


def pallas_model_destroy(h):
    lib().pallas_model_destroy(h)


def pallas_workspace_size(h, max_tokens: int, max_seqs: int) -> int:
    return int(lib().pallas_workspace_size(h, max_tokens, max_seqs))


def pallas_prefill_prefix(h, token_ids, cu_seqlens: Sequence[int], block_tables, pool,
                          workspace, err=None, stream=None):
    ps = kv_pool_struct(pool)
    _check(lib().pallas_prefill_prefix(h, len(cu_seqlens) - 1, _ptr(token_ids),
                                       _i32_array(cu_seqlens), _ptr(block_tables),
                                       block_tables.shape[-1], C.byref(ps), _ptr(workspace),
                                       workspace.numel() * workspace.element_size(), _ptr(err),
                                       _stream(stream)))


def pallas_prefill_chunk(h, token_ids, cu_seqlens: Sequence[int], start_pos: Sequence[int],
                         block_tables, pool, workspace, err=None, stream=None):
    assert len(start_pos) == len(cu_seqlens) - 1
    ps = kv_pool_struct(pool)
    _check(lib().pallas_prefill_chunk(h, len(cu_seqlens) - 1, _ptr(token_ids),
                                      _i32_array(cu_seqlens), _i32_array(start_pos),
                                      _ptr(block_tables), block_tables.shape[-1], C.byref(ps),
                                      _ptr(workspace), workspace.numel() * workspace.element_size(),
                                      _ptr(err), _stream(stream)))


def pallas_decode_step(h, tokens, positions: Sequence[int], block_tables, pool, logits,
                       workspace, err=None, stream=None):
    ps = kv_pool_struct(pool)
    _check(lib().pallas_decode_step(h, len(positions), _ptr(tokens), _i32_array(positions),
                                    _ptr(block_tables), block_tables.shape[-1], C.byref(ps),
                                    _ptr(logits), _ptr(workspace),
                                    workspace.numel() * workspace.element_size(), _ptr(err),
                                    _stream(stream)))


def pallas_decode_step_static(h, tokens, positions: Sequence[int], block_tables, pool, logits,
                              err=None, stream=None):
    """pallas_decode_step with the library's static scratch (no workspace)."""
    ps = kv_pool_struct(pool)
    _check(lib().pallas_decode_step_static(h, len(positions), _ptr(tokens), _i32_array(positions),
                                           _ptr(block_tables), block_tables.shape[-1], C.byref(ps),
                                           _ptr(logits), _ptr(err), _stream(stream)))


def _window_params(r_p, r_d, goodput, s_kv, t_load=0.0, t_0=0.0, alpha=0.8, t_max=5.0, dt=0.01):
    return WindowParams(r_p, r_d, goodput, s_kv, t_load, t_0, alpha, t_max, dt)


def pallas_window_select(k_curr: float, t_remain: float, **params) -> WindowDecision:
    """Algorithm 1's window decision; ``params`` are the fields of
    pallas_window_params (r_p, r_d, goodput, s_kv, t_load, t_0, alpha,
    t_max, dt)."""
    p = _window_params(**params)
    d = WindowDecision()
    _check(lib().pallas_window_select(C.byref(p), k_curr, t_remain, C.byref(d)))
    return d


def pallas_window_evaluate(k_curr: float, t_remain: float, t_w: float, **params) -> WindowDecision:
    p = _window_params(**params)
    d = WindowDecision()
    _check(lib().pallas_window_evaluate(C.byref(p), k_curr, t_remain, t_w, C.byref(d)))
    return d


def pallas_ewma_update(state: Ewma, sample: float, weight: float) -> float:
    return lib().pallas_ewma_update(C.byref(state), sample, weight)


def pallas_admit(model_compatible: bool, vram_free_bytes: float, s_kv: float, k_curr: float,
                 r_d: float, t_remain: float) -> bool:
    return bool(lib().pallas_admit(int(bool(model_compatible)), vram_free_bytes, s_kv, k_curr, r_d,
                                   t_remain))


def pallas_waste_bound(t_max: float, e_early: float, t_avail: float) -> float:
    return lib().pallas_waste_bound(t_max, e_early, t_avail)


def pallas_profile_enable(classes=KERNEL_CLASSES):
    """Time every launch of the named kernel classes (empty: disable)."""
    mask = 0
    for c in classes:
        mask |= 1 << KERNEL_CLASSES.index(c)
    lib().pallas_profile_enable(mask)


def pallas_profile_reset():
    lib().pallas_profile_reset()


def pallas_profile_clock(kernel_class: str):
    """(mean shader clock in GHz, workgroups sampled) inside the timed
    launches of one kernel class since the last reset."""
    ghz = C.c_double()
    wgs = C.c_int64()
    _check(lib().pallas_profile_clock(KERNEL_CLASSES.index(kernel_class), C.byref(ghz), C.byref(wgs)))
    return ghz.value, wgs.value


def pallas_profile_read():
    """{class: (total_ms, launches)} since the last reset."""
    n = len(KERNEL_CLASSES)
    ms = (C.c_double * n)()
    cnt = (C.c_int64 * n)()
    _check(lib().pallas_profile_read(ms, cnt))
    return {k: (ms[i], cnt[i]) for i, k in enumerate(KERNEL_CLASSES)}


class Model:
    """A model handle over caller-owned bf16 device weights."""

    def __init__(self, cfg, glob, layers):
        self.cfg = cfg
        self._keep = (glob, layers)
        self.handle = pallas_model_create(cfg, glob, layers)

    def close(self):
        if self.handle:
            pallas_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def workspace_size(self, max_tokens: int, max_seqs: int = 1) -> int:
        return pallas_workspace_size(self.handle, max_tokens, max_seqs)

    def workspace(self, max_tokens: int, max_seqs: int = 1, device="cuda"):
        import torch
        return torch.empty(self.workspace_size(max_tokens, max_seqs), dtype=torch.uint8, device=device)

    def prefill_prefix(self, token_ids, cu_seqlens, block_tables, pool, workspace, err=None,
                       stream=None):
        pallas_prefill_prefix(self.handle, token_ids, cu_seqlens, block_tables, pool, workspace,
                              err, stream)

    def prefill_chunk(self, token_ids, cu_seqlens, start_pos, block_tables, pool, workspace,
                      err=None, stream=None):
        pallas_prefill_chunk(self.handle, token_ids, cu_seqlens, start_pos, block_tables, pool,
                             workspace, err, stream)

    def decode_step(self, tokens, positions, block_tables, pool, logits, workspace, err=None,
                    stream=None):
        pallas_decode_step(self.handle, tokens, positions, block_tables, pool, logits, workspace,
                           err, stream)

    def decode_step_static(self, tokens, positions, block_tables, pool, logits, err=None, stream=None):
        pallas_decode_step_static(self.handle, tokens, positions, block_tables, pool, logits, err, stream)
