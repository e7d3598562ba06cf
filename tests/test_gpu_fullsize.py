"""Full-size parity: the 7B-class workload exactly as bench.py runs it (32 layers, 256+1 library
segments in HBM, ~4.3K grafted tokens, 64 patch tokens), checked on sampled layers and decode steps.

Same calls, same sizes and therefore the same split plans and launch configurations as the bench.
"""
import numpy as np
import pytest
import torch

from gpuutil import check_attn, check_keys, oracle_items, oracle_run, read_cache, say, storage_np
from oracle import graft as ograft, numerics, rope

pytestmark = pytest.mark.gpu

LAYERS = (0, 17, 31)
N_DEC = 3


@pytest.mark.parametrize("task", [0, 3])
def test_7b_full_size_sampled(task):
    from paper_2606_13097_amd import runner, synth
    w = synth.workload("7b", seed=1, task=task)
    sh = w.shape
    say(f"[gpu] full-size 7b task {task}: {len(w.lib_lengths)} segments, {w.grafted_tokens} grafted tokens")
    s = runner.GpuSetup(w)
    try:
        s.graft()
        torch.cuda.synchronize()
        say("[gpu]   graft done")
        winv = rope.inv_freq(sh.head_dim, sh.rope_theta)
        for layer in LAYERS:
            K, V, wr = ograft.compose(w.max_tokens, sh.n_kv_heads, sh.head_dim, oracle_items(w, 0, layer), winv,
                                      sh.dtype)
            pos = np.flatnonzero(wr)
            gk, gv = read_cache(s.cache, w, layer, 0, pos)
            np.testing.assert_array_equal(numerics.decode(gv, sh.dtype), V[pos])
            check_keys(gk, K[pos], sh.dtype, f"graft keys layer {layer}")
        outs = {}
        for layer in range(sh.n_layers):
            q, k, v = s.fresh_inputs(layer)
            out = torch.empty_like(q)
            s.prefill(layer, q, k, v, out)
            if layer in LAYERS:
                outs[layer] = out
        torch.cuda.synchronize()
        say("[gpu]   prefill done")
        dec = {}
        dins = {l: s.decode_inputs(l, N_DEC) for l in range(sh.n_layers)}
        for t in range(N_DEC):
            for layer in range(sh.n_layers):
                dq, dk, dv = dins[layer]
                o = torch.empty_like(dq[t])
                s.decode(layer, dq[t], dk[t], dv[t], o)
                if layer in LAYERS:
                    dec[(layer, t)] = o
        torch.cuda.synchronize()
        say("[gpu]   decode done")
        for layer in LAYERS:
            ref = oracle_run(w, 0, layer, N_DEC)
            check_attn(storage_np(outs[layer]), ref["prefill"], sh.dtype, f"prefill layer {layer}")
            for t in range(N_DEC):
                check_attn(storage_np(dec[(layer, t)][0]), ref["decode"][t], sh.dtype, f"decode layer {layer} step {t}")
        say("[gpu]   parity ok")
    finally:
        s.close()


# The other full-size workloads: the plans are not trimmed (every segment, every
# patch token, the library at its full size in HBM); prefill and two decode steps
# run on the first, a middle and the last layer, and the oracle checks sampled
# sequences there (layout of every sequence bit for bit, grafted and final keys and
# values, prefill and decode outputs).

def _sampled_layers(n_layers):
    return [0, n_layers // 2, n_layers - 1]


@pytest.mark.timeout(900)
def test_long16k_full_size_sampled():
    """~16K-token context: 2048-token prefix + 20 segments of U[400,1200] with 0-32 fresh gap
    tokens before each, 256 patch tokens prefilled in the same call."""
    from test_gpu_parity import run_pipeline
    from paper_2606_13097_amd import synth
    w = synth.workload("long16k", seed=1, n_decode=2)
    say(f"[gpu] full-size long16k: {w.grafted_tokens} grafted, {len(w.fresh_pos)} fresh tokens")
    run_pipeline(w, _sampled_layers(w.shape.n_layers), 2, [0])


@pytest.mark.timeout(900)
@pytest.mark.parametrize("alias", [False, True])
def test_batched_full_size_sampled(alias):
    """32 tasks x 8 Zipf-drawn segments from the 512-segment library, 16-token pages, 32 patch
    tokens per task; values copied or read from the library (FCG_ALIAS_V)."""
    from test_gpu_parity import run_pipeline
    from paper_2606_13097_amd import synth
    w = synth.workload("batched", seed=1, n_decode=2)
    say(f"[gpu] full-size batched alias={alias}: {w.grafted_tokens} grafted tokens over {w.n_seqs} tasks")
    run_pipeline(w, _sampled_layers(w.shape.n_layers), 2, [0, 13, 31], alias=alias)


@pytest.mark.timeout(1200)
def test_34b_full_size_sampled():
    """48 layers, 64/8 heads, 1024-segment library (~182 GB) with 1% outlier pairs x8; 4 tasks
    of 24 segments and 512 patch tokens each."""
    from test_gpu_parity import run_pipeline
    from paper_2606_13097_amd import synth
    w = synth.workload("34b", seed=1, n_decode=2)
    say(f"[gpu] full-size 34b: {w.grafted_tokens} grafted tokens over {w.n_seqs} tasks")
    run_pipeline(w, _sampled_layers(w.shape.n_layers), 2, [0, 3])
