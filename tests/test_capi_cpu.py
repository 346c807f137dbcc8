"""The C-ABI library without a GPU: it loads, exports every function include/retrace.h
declares, and its host-side checks return the documented status codes before any
device work."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "retrace.h")
LIB = os.path.join(ROOT, "paper_2608_29748_amd", "libretrace.so")


@pytest.fixture(scope="module")
def B():
    if not os.path.exists(LIB):
        from paper_2608_29748_amd import build
        build.build()
    from paper_2608_29748_amd import binding
    return binding


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rt_[a-z_]+)\s*\(", text)))


def test_every_declared_function_is_exported(B):
    names = declared_functions()
    assert len(names) >= 12
    lib = C.CDLL(LIB)
    for n in names:
        assert hasattr(lib, n), f"{n} declared in retrace.h but not exported"
    assert sorted(B.EXPORTS) == names


def cfg(B, **over):
    base = dict(vocab=1024, hidden=256, n_layers=2, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn=688,
                rope_theta=1e6, rms_eps=1e-6, draft_layers=1, cond_layer_ids=[0, 1], block_size=8,
                mask_token_id=1023, beta=1.0, cond_mode=B.RT_COND_RETRACE, dtype=B.RT_F32, max_batch=1,
                max_seq_len=208, page_size=16)
    base.update(over)
    return B.make_config(**base)


def test_workspace_and_weight_count(B):
    c = cfg(B)
    assert B.rt_workspace_bytes(c) > 0
    assert B.rt_weight_count(c) == 1 + 11 * 2 + 4 + 11 * 1 + 1 + 3
    assert B.rt_weight_count(cfg(B, cond_mode=B.RT_COND_LOWRANK)) == 1 + 11 * 2 + 4 + 11 * 1 + 1 + 3 + 5
    assert B.rt_workspace_bytes(cfg(B, cond_mode=B.RT_COND_LOWRANK)) > B.rt_workspace_bytes(c)
    big = cfg(B, dtype=B.RT_BF16, max_batch=4)
    assert B.rt_workspace_bytes(big) > B.rt_workspace_bytes(cfg(B, dtype=B.RT_BF16))


@pytest.mark.parametrize("over,msg", [
    (dict(n_q_heads=3), "multiple of n_kv_heads"),
    (dict(head_dim=96), "head_dim"),
    (dict(block_size=1), "block_size"),
    (dict(block_size=65), "block_size"),
    (dict(page_size=8), "page_size"),
    (dict(hidden=250), "hidden"),
    (dict(ffn=100), "ffn"),
    (dict(vocab=1000), "vocab"),
    (dict(cond_layer_ids=[0, 2]), "out of range"),
    (dict(cond_layer_ids=[1, 0]), "increase"),
    (dict(draft_layers=0), "draft_layers"),
    (dict(dtype=7), "dtype"),
    (dict(cond_mode=5), "cond_mode"),
    (dict(temperature=-1.0), "temperature"),
    (dict(temperature=1.0, top_k=0, top_p=0.9), "top_k"),
    (dict(temperature=1.0, top_k=65, top_p=0.9), "top_k"),
    (dict(temperature=1.0, top_k=20, top_p=0.0), "top_p"),
    (dict(temperature=1.0, top_k=20, top_p=1.5), "top_p"),
    (dict(cond_mode=-1), "cond_mode"),
    (dict(max_seq_len=4), "max_seq_len"),
    (dict(max_batch=0), "max_batch"),
    (dict(dtype=0, max_seq_len=16385), "fp32 storage"),
])
def test_invalid_configs_are_rejected(B, over, msg):
    c = cfg(B, **over)
    assert B.rt_workspace_bytes(c) == 0
    assert msg in B.rt_last_error()


def test_mask_token_out_of_range(B):
    c = cfg(B, mask_token_id=1024)
    assert B.rt_workspace_bytes(c) == 0
    assert "mask_token_id" in B.rt_last_error()


def _init(B, c, n_weights=None, ws=0x100000, ws_bytes=None, weights_ok=True):
    n = B.rt_weight_count(c) if n_weights is None else n_weights
    arr = (C.c_void_p * max(n, 1))(*[C.c_void_p(0x1000 if weights_ok else 0) for _ in range(max(n, 1))])
    h = C.c_void_p()
    wsb = B.rt_workspace_bytes(c) if ws_bytes is None else ws_bytes
    return B._lib.rt_init_models(C.byref(c), arr, n, C.c_void_p(ws), wsb, None, C.byref(h))


def test_init_models_argument_checks(B):
    c = cfg(B)
    assert _init(B, c, n_weights=3) == B.RT_ERR_INVALID and "weight tensors" in B.rt_last_error()
    assert _init(B, c, weights_ok=False) == B.RT_ERR_INVALID and "is null" in B.rt_last_error()
    assert _init(B, c, ws=0) == B.RT_ERR_WORKSPACE
    assert _init(B, c, ws=0x100010) == B.RT_ERR_WORKSPACE and "aligned" in B.rt_last_error()
    assert _init(B, c, ws_bytes=1024) == B.RT_ERR_WORKSPACE and "needs" in B.rt_last_error()
    bad = cfg(B, head_dim=32)
    assert _init(B, bad, n_weights=B.rt_weight_count(c)) == B.RT_ERR_INVALID
    h = C.c_void_p()
    assert B._lib.rt_init_models(C.byref(c), None, 0, None, 0, None, None) == B.RT_ERR_INVALID


def test_calls_on_null_handle(B):
    i32 = C.POINTER(C.c_int32)
    z = (C.c_int32 * 8)()
    p = C.cast(z, i32)
    assert B._lib.rt_prefill(None, 1, p, p, 4, p) == B.RT_ERR_INVALID
    assert B._lib.rt_spec_round(None, p, p, p) == B.RT_ERR_INVALID
    assert B._lib.rt_spec_round_forced(None, p, p, p, p) == B.RT_ERR_INVALID
    assert B._lib.rt_ar_steps(None, 1, p, p) == B.RT_ERR_INVALID
    assert B._lib.rt_set_debug(None, 0) == B.RT_ERR_INVALID
    assert B._lib.rt_debug_read(None, 0, 0, None, 0) == B.RT_ERR_INVALID
    assert B._lib.rt_debug_write(None, 0, 0, None, 0) == B.RT_ERR_INVALID
    assert B._lib.rt_destroy(None) == B.RT_ERR_INVALID
    assert "null model" in B.rt_last_error()


def test_error_message_is_thread_local(B):
    import threading
    B.rt_workspace_bytes(cfg(B, page_size=8))
    seen = {}

    def other():
        B.rt_workspace_bytes(cfg(B, block_size=1))
        seen["msg"] = B.rt_last_error()

    t = threading.Thread(target=other)
    t.start()
    t.join()
    assert "block_size" in seen["msg"]
    assert "page_size" in B.rt_last_error()


def test_library_from_other_sources_is_refused(B, tmp_path):
    """The binding loads only a library whose build stamp matches the tree's sources."""
    import shutil
    from paper_2608_29748_amd.build import source_hash
    lib = tmp_path / "libretrace.so"
    shutil.copy(LIB, lib)
    (tmp_path / "libretrace.so.sha256").write_text("0" * 64 + "\n")
    with pytest.raises(RuntimeError, match="not built from the current sources"):
        B.load_library(str(lib))
    (tmp_path / "libretrace.so.sha256").unlink()
    with pytest.raises(RuntimeError, match="missing"):
        B.load_library(str(lib))
    (tmp_path / "libretrace.so.sha256").write_text(source_hash() + "\n")
    assert B.load_library(str(lib)) is not None


@pytest.mark.parametrize("name,mode", [("tiny-f32", "retrace"), ("mini-bf16-gqa5", "retrace"),
                                       ("mini-bf16", "lowrank"), ("qwen3-14b-shape-b16", "retrace")])
def test_weight_elements_follow_the_canonical_order(B, name, mode):
    """rt_weight_elements gives every tensor's size in the order rt_init_models reads them."""
    from workloads import get, weight_specs
    import numpy as np
    wl = get(name, cond_mode=mode)
    c = B.make_config(vocab=wl.target.vocab, hidden=wl.target.hidden, n_layers=wl.target.n_layers,
                      n_q_heads=wl.target.n_q_heads, n_kv_heads=wl.target.n_kv_heads, head_dim=wl.target.head_dim,
                      ffn=wl.target.ffn, rope_theta=1e6, rms_eps=1e-6, draft_layers=wl.draft_layers,
                      cond_layer_ids=list(wl.cond_layers), block_size=wl.block_size, mask_token_id=wl.mask_token_id,
                      beta=1.0, cond_mode=B.COND_MODES[mode], dtype=B.RT_BF16 if wl.dtype == "bf16" else B.RT_F32,
                      max_batch=wl.batch, max_seq_len=wl.max_seq_len, page_size=16, temperature=0.0, top_k=20,
                      top_p=0.95, sample_seed=1)
    specs = weight_specs(wl)
    assert B.rt_weight_count(c) == len(specs)
    for i, (_, shape, _) in enumerate(specs):
        assert B.rt_weight_elements(c, i) == int(np.prod(shape)), (i, specs[i])
    assert B.rt_weight_elements(c, len(specs)) == 0 and B.rt_weight_elements(c, -1) == 0


def test_stream_read_argument_checks(B):
    """rt_stream_read rejects its documented invalid arguments before any device work."""
    us = C.c_double()
    buf = 1 << 20   # a 256-byte-aligned stand-in address: never dereferenced on these paths

    def call(ptr=buf, buf_bytes=1 << 20, nbytes=4096, grid=64, reps=1, out=True):
        return B._lib.rt_stream_read(C.c_void_p(ptr), buf_bytes, nbytes, grid, reps, None,
                                     C.byref(us) if out else None)

    assert call(ptr=0) == B.RT_ERR_INVALID and "null" in B.rt_last_error()
    assert call(out=False) == B.RT_ERR_INVALID
    assert call(nbytes=0) == B.RT_ERR_INVALID and "multiple of 16" in B.rt_last_error()
    assert call(nbytes=4100) == B.RT_ERR_INVALID
    assert call(ptr=buf + 16) == B.RT_ERR_INVALID and "aligned" in B.rt_last_error()
    assert call(nbytes=2 << 20) == B.RT_ERR_INVALID and "exceed" in B.rt_last_error()
    assert call(grid=0) == B.RT_ERR_INVALID and "grid" in B.rt_last_error()
    assert call(grid=65537) == B.RT_ERR_INVALID
    assert call(reps=0) == B.RT_ERR_INVALID and "reps" in B.rt_last_error()
    assert call(reps=1001) == B.RT_ERR_INVALID
