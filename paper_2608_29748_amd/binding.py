"""ctypes binding of libretrace.so: the C ABI of include/retrace.h under the same names.

Argument marshalling only; every step of the round runs in the library's HIP kernels.
Importing this module loads the in-tree library and fails loudly if it is missing.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Sequence, Tuple

import numpy as np
# torch first: its bundled HIP runtime (soname libamdhip64.so.7) is then the one the
# library binds to, so the process holds a single HIP / HSA runtime.
import torch  # noqa: F401

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libretrace.so")

RT_OK, RT_ERR_INVALID, RT_ERR_STATE, RT_ERR_CAPACITY, RT_ERR_WORKSPACE, RT_ERR_HIP, RT_ERR_TOKEN = \
    0, -1, -2, -3, -4, -5, -6
RT_F32, RT_BF16 = 0, 1
RT_COND_OFF, RT_COND_RETRACE, RT_COND_RAW_GATED, RT_COND_OVERWRITE, RT_COND_LOWRANK = 0, 1, 2, 3, 4
COND_MODES = {"off": RT_COND_OFF, "retrace": RT_COND_RETRACE, "raw_gated": RT_COND_RAW_GATED,
              "overwrite": RT_COND_OVERWRITE, "lowrank": RT_COND_LOWRANK}
RT_MAX_COND_LAYERS = 8
(RT_T_DRAFT_LOGITS, RT_T_VERIFY_LOGITS, RT_T_HD, RT_T_HT, RT_T_ETILDE, RT_T_DRAFT_TOKENS,
 RT_T_TARGET_TOKENS, RT_T_STATE, RT_T_G, RT_T_AR_LOGITS, RT_T_DRAFT_DIST_IDS, RT_T_DRAFT_DIST_P,
 RT_T_VERIFY_DIST_IDS, RT_T_VERIFY_DIST_P) = range(14)
RT_MAX_TOP_K = 64
RT_AR_MAX_STEPS = 256
RT_T_TARGET_K, RT_T_TARGET_V, RT_T_DRAFT_K, RT_T_DRAFT_V = 100, 200, 300, 400
RT_T_TRACE_DRAFT_X, RT_T_TRACE_TARGET_X, RT_T_TRACE_DRAFT_HEAD, RT_T_TRACE_VERIFY_HEAD = 500, 600, 700, 701
RT_T_TRACE_DRAFT_Q, RT_T_TRACE_DRAFT_ATTN, RT_T_TRACE_DRAFT_XMID, RT_T_TRACE_DRAFT_H2, RT_T_TRACE_DRAFT_MLP = \
    1100, 1200, 1300, 1400, 1500
RT_T_TRACE_TARGET_Q, RT_T_TRACE_TARGET_ATTN, RT_T_TRACE_TARGET_XMID, RT_T_TRACE_TARGET_H2, RT_T_TRACE_TARGET_MLP = \
    2100, 2200, 2300, 2400, 2500
(RT_K_GEMM_QKV, RT_K_GEMM_O, RT_K_GEMM_GATE_UP, RT_K_GEMM_DOWN, RT_K_GEMM_CONTEXT, RT_K_GEMM_COND,
 RT_K_ATTENTION, RT_K_ATTN_MERGE, RT_K_NORM, RT_K_QKV_POST, RT_K_LM_HEAD, RT_K_MISC) = range(12)
RT_K_KINDS = 12
KERNEL_KIND_NAMES = ["gemm_qkv", "gemm_o", "gemm_gate_up", "gemm_down", "gemm_context", "gemm_cond",
                     "attention", "attn_merge", "rmsnorm", "qkv_post", "lm_head", "misc"]
STAGE_NAMES = ["condition", "draft", "draft_lm_head", "verify", "verify_lm_head", "accept", "context_append"]
RT_PROF_STAGES = 7

EXPORTS = ["rt_workspace_bytes", "rt_weight_count", "rt_init_models", "rt_prefill", "rt_spec_round",
           "rt_destroy", "rt_last_error", "rt_set_debug", "rt_spec_round_forced", "rt_debug_read",
           "rt_debug_write", "rt_profile_round", "rt_time_kernel", "rt_ar_steps", "rt_debug_read_rows",
           "rt_spec_round_static", "rt_stream_read", "rt_weight_elements"]


class RetraceError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"[{code}] {msg}")
        self.code = code


class rt_config(C.Structure):
    _fields_ = [("vocab", C.c_int32), ("hidden", C.c_int32), ("n_layers", C.c_int32),
                ("n_q_heads", C.c_int32), ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32),
                ("ffn", C.c_int32), ("rope_theta", C.c_float), ("rms_eps", C.c_float),
                ("draft_layers", C.c_int32), ("n_cond_layers", C.c_int32),
                ("cond_layer_ids", C.c_int32 * RT_MAX_COND_LAYERS), ("block_size", C.c_int32),
                ("mask_token_id", C.c_int32), ("beta", C.c_float), ("cond_mode", C.c_int32),
                ("dtype", C.c_int32), ("max_batch", C.c_int32), ("max_seq_len", C.c_int32),
                ("page_size", C.c_int32), ("temperature", C.c_float), ("top_k", C.c_int32),
                ("top_p", C.c_float), ("sample_seed", C.c_uint64)]


class rt_kernel_stat(C.Structure):
    _fields_ = [("kind", C.c_int32), ("launches", C.c_int32), ("ms", C.c_double), ("bytes", C.c_double),
                ("flops", C.c_double)]


def load_library(path: str = LIB_PATH) -> C.CDLL:
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python paper_2608_29748_amd/build.py` "
                           "(there is no fallback path)")
    # refuse a library built from other sources than the ones in the tree
    from .build import STAMP, source_hash
    stamp = path + ".sha256" if path != LIB_PATH else STAMP
    built = open(stamp).read().strip() if os.path.exists(stamp) else None
    if built != source_hash():
        raise RuntimeError(f"{path} was not built from the current sources (stamp {stamp}: "
                           f"{'missing' if built is None else 'different hash'}); rebuild it with "
                           "`python paper_2608_29748_amd/build.py`")
    lib = C.CDLL(path)
    P = C.c_void_p
    i32p = C.POINTER(C.c_int32)
    lib.rt_workspace_bytes.argtypes = [C.POINTER(rt_config)]
    lib.rt_workspace_bytes.restype = C.c_size_t
    lib.rt_weight_count.argtypes = [C.POINTER(rt_config)]
    lib.rt_weight_count.restype = C.c_int32
    lib.rt_weight_elements.argtypes = [C.POINTER(rt_config), C.c_int32]
    lib.rt_weight_elements.restype = C.c_int64
    lib.rt_init_models.argtypes = [C.POINTER(rt_config), C.POINTER(P), C.c_int32, P, C.c_size_t, P,
                                   C.POINTER(P)]
    lib.rt_prefill.argtypes = [P, C.c_int32, i32p, i32p, C.c_int32, i32p]
    lib.rt_spec_round.argtypes = [P, i32p, i32p, i32p]
    lib.rt_spec_round_forced.argtypes = [P, i32p, i32p, i32p, i32p]
    lib.rt_spec_round_static.argtypes = [P, P, P, P]
    lib.rt_stream_read.argtypes = [P, C.c_size_t, C.c_size_t, C.c_int32, C.c_int32, P, C.POINTER(C.c_double)]
    lib.rt_destroy.argtypes = [P]
    lib.rt_last_error.argtypes = []
    lib.rt_last_error.restype = C.c_char_p
    lib.rt_set_debug.argtypes = [P, C.c_int32]
    lib.rt_debug_read.argtypes = [P, C.c_int32, C.c_int32, P, C.c_size_t]
    lib.rt_debug_read_rows.argtypes = [P, C.c_int32, C.c_int32, C.c_int32, P, C.c_size_t]
    lib.rt_debug_write.argtypes = [P, C.c_int32, C.c_int32, P, C.c_size_t]
    lib.rt_profile_round.argtypes = [P, C.POINTER(rt_kernel_stat), C.POINTER(C.c_double), i32p, i32p, i32p]
    lib.rt_time_kernel.argtypes = [P, C.c_int32, C.c_int32, C.POINTER(rt_kernel_stat)]
    lib.rt_ar_steps.argtypes = [P, C.c_int32, i32p, i32p]
    for name in ("rt_init_models", "rt_prefill", "rt_spec_round", "rt_spec_round_forced", "rt_spec_round_static",
                 "rt_stream_read", "rt_destroy",
                 "rt_set_debug", "rt_debug_read", "rt_debug_read_rows", "rt_debug_write", "rt_profile_round",
                 "rt_time_kernel", "rt_ar_steps"):
        getattr(lib, name).restype = C.c_int
    return lib


_lib = load_library()


def _check(status: int) -> None:
    if status != RT_OK:
        raise RetraceError(status, rt_last_error())


def _i32(a) -> Tuple[np.ndarray, C.POINTER(C.c_int32)]:
    arr = np.ascontiguousarray(a, dtype=np.int32)
    return arr, arr.ctypes.data_as(C.POINTER(C.c_int32))


def make_config(**kw) -> rt_config:
    """rt_config from keyword fields (cond_layer_ids given as a sequence)."""
    ids = list(kw.pop("cond_layer_ids"))
    cfg = rt_config(**kw)
    cfg.n_cond_layers = len(ids)
    for i, v in enumerate(ids):
        cfg.cond_layer_ids[i] = v
    return cfg


def rt_last_error() -> str:
    m = _lib.rt_last_error()
    return m.decode() if m else ""


def rt_workspace_bytes(cfg: rt_config) -> int:
    return int(_lib.rt_workspace_bytes(C.byref(cfg)))


def rt_weight_count(cfg: rt_config) -> int:
    return int(_lib.rt_weight_count(C.byref(cfg)))


def rt_weight_elements(cfg: rt_config, index: int) -> int:
    return int(_lib.rt_weight_elements(C.byref(cfg), index))


def rt_init_models(cfg: rt_config, weight_ptrs: Sequence[int], ws_ptr: int, ws_bytes: int,
                   stream_ptr: int = 0) -> int:
    arr = (C.c_void_p * len(weight_ptrs))(*[C.c_void_p(p) for p in weight_ptrs])
    h = C.c_void_p()
    _check(_lib.rt_init_models(C.byref(cfg), arr, len(weight_ptrs), C.c_void_p(ws_ptr), ws_bytes,
                               C.c_void_p(stream_ptr), C.byref(h)))
    return h.value


def rt_prefill(h: int, prompts: Sequence[np.ndarray], gen_budget: int) -> np.ndarray:
    lens, lp = _i32([len(p) for p in prompts])
    ids, ip = _i32(np.concatenate([np.asarray(p) for p in prompts]) if len(prompts) else [])
    first = np.zeros(len(prompts), np.int32)
    _check(_lib.rt_prefill(C.c_void_p(h), len(prompts), lp, ip, gen_budget,
                           first.ctypes.data_as(C.POINTER(C.c_int32))))
    return first


def rt_spec_round(h: int, n_seqs: int, block_size: int):
    tok = np.full((n_seqs, block_size), -1, np.int32)
    n = np.zeros(n_seqs, np.int32)
    a = np.zeros(n_seqs, np.int32)
    _check(_lib.rt_spec_round(C.c_void_p(h), tok.ctypes.data_as(C.POINTER(C.c_int32)),
                              n.ctypes.data_as(C.POINTER(C.c_int32)), a.ctypes.data_as(C.POINTER(C.c_int32))))
    return tok, n, a


def rt_spec_round_static(h: int, d_tokens: int, d_n_committed: int, d_accept_len: int) -> None:
    """The allocation-free round: outputs to device buffers (pointers), enqueued only."""
    _check(_lib.rt_spec_round_static(C.c_void_p(h), C.c_void_p(d_tokens), C.c_void_p(d_n_committed),
                                     C.c_void_p(d_accept_len)))


def rt_spec_round_forced(h: int, drafts: np.ndarray, block_size: int):
    d, dp = _i32(drafts)
    n_seqs = d.shape[0]
    tok = np.full((n_seqs, block_size), -1, np.int32)
    n = np.zeros(n_seqs, np.int32)
    a = np.zeros(n_seqs, np.int32)
    _check(_lib.rt_spec_round_forced(C.c_void_p(h), dp, tok.ctypes.data_as(C.POINTER(C.c_int32)),
                                     n.ctypes.data_as(C.POINTER(C.c_int32)),
                                     a.ctypes.data_as(C.POINTER(C.c_int32))))
    return tok, n, a


def rt_ar_steps(h: int, n_seqs: int, n_steps: int):
    """Target-only greedy steps: (tokens [n_seqs][n_steps] with -1 past the budget,
    tokens generated per sequence)."""
    tok = np.full((n_seqs, n_steps), -1, np.int32)
    n = np.zeros(n_seqs, np.int32)
    _check(_lib.rt_ar_steps(C.c_void_p(h), n_steps, tok.ctypes.data_as(C.POINTER(C.c_int32)),
                            n.ctypes.data_as(C.POINTER(C.c_int32))))
    return tok, n


def rt_profile_round(h: int, n_seqs: int, block_size: int):
    """One round with an event pair on every launch: returns (per-kind stats list of
    dicts, per-stage ms list, tokens, n_committed, accept_len)."""
    stats = (rt_kernel_stat * RT_K_KINDS)()
    stages = (C.c_double * RT_PROF_STAGES)()
    tok = np.full((n_seqs, block_size), -1, np.int32)
    n = np.zeros(n_seqs, np.int32)
    a = np.zeros(n_seqs, np.int32)
    _check(_lib.rt_profile_round(C.c_void_p(h), stats, stages, tok.ctypes.data_as(C.POINTER(C.c_int32)),
                                 n.ctypes.data_as(C.POINTER(C.c_int32)), a.ctypes.data_as(C.POINTER(C.c_int32))))
    out = [dict(kind=KERNEL_KIND_NAMES[s.kind], launches=s.launches, ms=s.ms, bytes=s.bytes, flops=s.flops)
           for s in stats]
    return out, list(stages), tok, n, a


def rt_time_kernel(h: int, kind: int, reps: int) -> dict:
    """Replay timing of one launch class: dict(kind, launches per round, ms of those
    launches per replay, algorithmic bytes, flops)."""
    st = rt_kernel_stat()
    _check(_lib.rt_time_kernel(C.c_void_p(h), kind, reps, C.byref(st)))
    return dict(kind=KERNEL_KIND_NAMES[st.kind], launches=st.launches, ms=st.ms, bytes=st.bytes, flops=st.flops)


def rt_stream_read(ptr: int, buf_bytes: int, nbytes: int, grid: int, reps: int, stream_ptr: int = 0) -> float:
    """Average microseconds of a plain read of nbytes, rotating over the buf_bytes at ptr."""
    us = C.c_double()
    _check(_lib.rt_stream_read(C.c_void_p(ptr), buf_bytes, nbytes, grid, reps, C.c_void_p(stream_ptr), C.byref(us)))
    return us.value


def rt_set_debug(h: int, flags: int) -> None:
    _check(_lib.rt_set_debug(C.c_void_p(h), flags))


def rt_debug_read(h: int, tensor_id: int, seq: int, nbytes: int) -> bytes:
    buf = C.create_string_buffer(nbytes)
    _check(_lib.rt_debug_read(C.c_void_p(h), tensor_id, seq, buf, nbytes))
    return buf.raw


def rt_debug_read_rows(h: int, tensor_id: int, seq: int, pos0: int, nbytes: int) -> bytes:
    buf = C.create_string_buffer(nbytes)
    _check(_lib.rt_debug_read_rows(C.c_void_p(h), tensor_id, seq, pos0, buf, nbytes))
    return buf.raw


def rt_debug_write(h: int, tensor_id: int, seq: int, data: bytes) -> None:
    buf = C.create_string_buffer(data, len(data))
    _check(_lib.rt_debug_write(C.c_void_p(h), tensor_id, seq, buf, len(data)))


def rt_destroy(h: int) -> None:
    _check(_lib.rt_destroy(C.c_void_p(h)))
