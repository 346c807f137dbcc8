"""In rounds and target-only steps the attention kernel applies the q / k-norm and the
rotation itself and writes the block's K / V rows to the caches; debug flag 16 keeps the
separate post-processing kernel.  Both paths round the same operations in the same
order, so everything downstream must agree bit for bit: logits of both LM heads,
committed tokens, round state, retained states, the layer trace's q, and the K / V
caches of every target and drafter layer."""
import numpy as np
import pytest

from paper_2608_29748_amd import binding as B
from workloads import ModelShape, get, make_weights

from gpu_parity import engine_for, keep_dtype, log

pytestmark = pytest.mark.gpu

FUSED_OFF = 16


def _prompts(wl, lens):
    g = np.random.default_rng(wl.seed + 1000)
    return [g.integers(0, wl.target.vocab - 1, size=n).astype(np.int32) for n in lens]


def _snapshot(eng, wl, trace):
    t, bk, V = wl.target, wl.block_size, wl.target.vocab
    kd = keep_dtype(wl)
    sd = np.uint16
    out = []
    for b in range(eng.n_seqs):
        st = eng.read(B.RT_T_STATE, b, (9,), np.int32)
        n_pos = int(st[0]) + bk
        item = {"state": st,
                "draft_logits": eng.read(B.RT_T_DRAFT_LOGITS, b, (bk, V), np.float32),
                "verify_logits": eng.read(B.RT_T_VERIFY_LOGITS, b, (bk, V), np.float32),
                "hd": eng.read(B.RT_T_HD, b, (bk, t.hidden), kd).view(np.uint8),
                "ht": eng.read(B.RT_T_HT, b, (bk, t.hidden), kd).view(np.uint8)}
        for l in range(t.n_layers):
            for name, base in (("tk", B.RT_T_TARGET_K), ("tv", B.RT_T_TARGET_V)):
                item[f"{name}{l}"] = eng.read_rows(base + l, b, 0, (n_pos, t.n_kv_heads, t.head_dim), sd)
        for l in range(wl.draft_layers):
            for name, base in (("dk", B.RT_T_DRAFT_K), ("dv", B.RT_T_DRAFT_V)):
                item[f"{name}{l}"] = eng.read_rows(base + l, b, 0, (n_pos, t.n_kv_heads, t.head_dim), sd)
        if trace:
            qw = t.n_q_heads * t.head_dim
            for l in range(wl.draft_layers):
                item[f"dq{l}"] = eng.read(B.RT_T_TRACE_DRAFT_Q + l, b, (bk, qw), sd)
            for l in range(t.n_layers):
                item[f"tq{l}"] = eng.read(B.RT_T_TRACE_TARGET_Q + l, b, (bk, qw), sd)
        out.append(item)
    return out


def _same(a, b, what):
    for s, (x, y) in enumerate(zip(a, b)):
        assert x.keys() == y.keys()
        for k in x:
            assert np.array_equal(x[k], y[k]), f"{what}: sequence {s} {k} differs " \
                f"({np.count_nonzero(x[k] != y[k])} of {x[k].size} elements)"


CASES = [
    # hd 64, GQA 2, one 64-row block per KV head; the first block straddles a 64-key chunk
    ("mini-bf16", {}, [57]),
    # hd 64, GQA 4, three sequences, blocks inside and across chunk boundaries
    ("mini-bf16-ragged", {}, [49, 63, 130]),
    # hd 128, four sequences (64 round rows, the largest batch on this path)
    ("mini-bf16-b4", {}, [30, 60, 64, 90]),
    # GQA 5: 80 query rows per block (the 96-row kernel, three LDS stages)
    ("mini-bf16-gqa5", {}, [55, 150]),
    # GQA 8: 128 query rows per block, two row blocks per KV head
    ("mini-bf16", {"target": ModelShape(vocab=2048, hidden=256, n_layers=2, n_q_heads=16, n_kv_heads=2,
                                        head_dim=64, ffn=512), "cond_layers": (0, 1), "batch": 2}, [61, 300]),
]


@pytest.mark.parametrize("name,over,lens", CASES)
def test_fused_qk_post_equals_separate_kernel(name, over, lens):
    wl = get(name, norm_init="perturbed", **over)
    wl = wl.with_(batch=len(lens), prompt_len=(min(lens), max(lens)))
    W = make_weights(wl)
    prompts = _prompts(wl, lens)
    for trace in (False, True):
        base = 1 | (8 if trace else 0)
        fused, sep = engine_for(wl, W), engine_for(wl, W)
        fused.set_debug(base)
        sep.set_debug(base | FUSED_OFF)
        assert list(fused.prefill(prompts, wl.new_tokens)) == list(sep.prefill(prompts, wl.new_tokens))
        for t in range(4):
            r_f, r_s = fused.spec_round(), sep.spec_round()
            for x, y in zip(r_f, r_s):
                assert np.array_equal(x, y), (name, trace, t, r_f, r_s)
            _same(_snapshot(fused, wl, trace), _snapshot(sep, wl, trace), f"{name} trace={trace} round {t}")
        log(f"[{name} {lens} trace={trace}] 4 rounds equal bit for bit")
        if not trace:
            # target-only greedy steps (one query row per sequence)
            a_f, a_s = fused.ar_steps(3), sep.ar_steps(3)
            for x, y in zip(a_f, a_s):
                assert np.array_equal(x, y), (name, a_f, a_s)
            for b in range(len(lens)):
                lf = fused.read(B.RT_T_AR_LOGITS, b, (wl.target.vocab,), np.float32)
                ls = sep.read(B.RT_T_AR_LOGITS, b, (wl.target.vocab,), np.float32)
                assert np.array_equal(lf, ls), (name, b)
            log(f"[{name} {lens}] 3 target-only steps equal bit for bit")
        fused.close()
        sep.close()
