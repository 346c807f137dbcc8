"""Device-memory plumbing around the C ABI: uploads weights, owns the workspace and
stream (PyTorch), and marshals calls.  Every step of the round runs in the library."""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

from . import binding as B


def config_from(shape, *, dtype: str, draft_layers: int, cond_layers: Sequence[int], block_size: int,
                mask_token_id: int, max_batch: int, max_seq_len: int, rope_theta: float = 1e6,
                rms_eps: float = 1e-6, beta: float = 1.0, cond_mode: int = B.RT_COND_RETRACE,
                page_size: int = 16, temperature: float = 0.0, top_k: int = 20, top_p: float = 0.95,
                sample_seed: int = 42) -> B.rt_config:
    """rt_config from a model-shape object with vocab / hidden / n_layers / n_q_heads /
    n_kv_heads / head_dim / ffn attributes."""
    return B.make_config(
        vocab=shape.vocab, hidden=shape.hidden, n_layers=shape.n_layers, n_q_heads=shape.n_q_heads,
        n_kv_heads=shape.n_kv_heads, head_dim=shape.head_dim, ffn=shape.ffn, rope_theta=rope_theta,
        rms_eps=rms_eps, draft_layers=draft_layers, cond_layer_ids=list(cond_layers),
        block_size=block_size, mask_token_id=mask_token_id, beta=beta, cond_mode=cond_mode,
        dtype=B.RT_BF16 if dtype == "bf16" else B.RT_F32, max_batch=max_batch,
        max_seq_len=max_seq_len, page_size=page_size, temperature=temperature, top_k=top_k, top_p=top_p,
        sample_seed=sample_seed)


class RoundEngine:
    """One model instance on cuda:`device`.  `weights` are host arrays in the canonical
    order (uint16 bf16 bit patterns or float32); they are uploaded, packed by the
    library into its workspace, and the uploaded copies are released."""

    def __init__(self, cfg: B.rt_config, weights: Sequence[np.ndarray], device: int = 0,
                 stream: Optional[torch.cuda.Stream] = None):
        if not torch.cuda.is_available():
            raise RuntimeError("RoundEngine needs a GPU")
        self.cfg = cfg
        self.device = torch.device("cuda", device)
        self.stream = stream or torch.cuda.Stream(device=self.device)
        n = B.rt_weight_count(cfg)
        if n != len(weights):
            raise ValueError(f"expected {n} weight tensors, got {len(weights)}")
        nbytes = B.rt_workspace_bytes(cfg)
        if nbytes == 0:
            raise B.RetraceError(B.RT_ERR_INVALID, B.rt_last_error())
        self.ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
        base = self.ws.data_ptr()
        off = (-base) % 256
        self.ws_ptr, self.ws_bytes = base + off, nbytes
        tdt = torch.int16 if cfg.dtype == B.RT_BF16 else torch.float32
        with torch.cuda.stream(self.stream):
            dev = [torch.from_numpy(np.ascontiguousarray(w).view(np.int16 if w.dtype == np.uint16 else w.dtype))
                   .to(self.device, non_blocking=False) for w in weights]
            for t in dev:
                assert t.dtype == tdt, f"weight dtype {t.dtype} does not match config"
        torch.cuda.synchronize(self.device)
        self.h = B.rt_init_models(cfg, [t.data_ptr() for t in dev], self.ws_ptr, self.ws_bytes,
                                  self.stream.cuda_stream)
        del dev
        torch.cuda.synchronize(self.device)
        self.n_seqs = 0

    def prefill(self, prompts: Sequence[np.ndarray], gen_budget: int) -> np.ndarray:
        first = B.rt_prefill(self.h, prompts, gen_budget)
        self.n_seqs = len(prompts)
        return first

    def spec_round(self):
        return B.rt_spec_round(self.h, self.n_seqs, self.cfg.block_size)

    def spec_round_forced(self, drafts: np.ndarray):
        return B.rt_spec_round_forced(self.h, drafts, self.cfg.block_size)

    def ar_steps(self, n_steps: int):
        return B.rt_ar_steps(self.h, self.n_seqs, n_steps)

    def profile_round(self):
        return B.rt_profile_round(self.h, self.n_seqs, self.cfg.block_size)

    def time_kernel(self, kind: int, reps: int = 20) -> dict:
        return B.rt_time_kernel(self.h, kind, reps)

    def set_debug(self, flags: int) -> None:
        B.rt_set_debug(self.h, flags)

    def read(self, tensor_id: int, seq: int, shape, dtype) -> np.ndarray:
        dt = np.dtype(dtype)
        n = int(np.prod(shape)) * dt.itemsize
        return np.frombuffer(B.rt_debug_read(self.h, tensor_id, seq, n), dtype=dt).reshape(shape).copy()

    def read_rows(self, tensor_id: int, seq: int, pos0: int, shape, dtype) -> np.ndarray:
        """KV cache rows pos0.. of one sequence ([n][Hkv][hd])."""
        dt = np.dtype(dtype)
        n = int(np.prod(shape)) * dt.itemsize
        return np.frombuffer(B.rt_debug_read_rows(self.h, tensor_id, seq, pos0, n), dtype=dt).reshape(shape).copy()

    def write(self, tensor_id: int, seq: int, arr: np.ndarray) -> None:
        B.rt_debug_write(self.h, tensor_id, seq, np.ascontiguousarray(arr).tobytes())

    def close(self) -> None:
        if getattr(self, "h", None):
            B.rt_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
