"""Parity of the HIP path (through the C ABI) with the CPU oracle, on seeded synthetic workloads.

Bars: layout and placement bit-exact; grafted and copied values bit-exact; grafted keys
within 1e-5 normwise (fp32) or one bf16 ulp; attention outputs within 1e-5 normwise per
head (fp32) or max-abs 2e-2 plus relative Frobenius 1e-2 (bf16).
"""
import dataclasses

import numpy as np
import pytest
import torch

from gpuutil import (check_attn, check_keys, oracle_items, oracle_run, read_cache, say, storage_np, to_device)
from oracle import graft as ograft, numerics, rope, task
from oracle.layout import Layout
from paper_2606_13097_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    from paper_2606_13097_amd import fcg, runner, synth  # noqa: F401  (fails loudly if unbuilt)
    yield


def _oracle_layout(w, n_decode, layers, alias=False):
    ora = Layout(w.shape.n_layers, w.n_seqs, w.max_tokens, w.page_size, w.n_pages, w.lib_lengths, w.lib_src_pos0,
                 alias_v=alias)
    ora.graft(w.graft_seq, w.graft_seg, w.graft_dst)
    for layer in layers:
        ora.append(layer, w.fresh_seq, w.fresh_pos)
        for _ in range(n_decode):
            ora.decode(layer, list(range(w.n_seqs)))
    return ora


def _compare_layout(cache, ora, w, layers):
    from paper_2606_13097_amd import fcg
    for s in range(w.n_seqs):
        for layer in layers:
            pt, n, wr = fcg.fcg_cache_export_layout(cache, s, layer)
            np.testing.assert_array_equal(wr.astype(bool), ora.written[s, layer])
            assert n == ora.seq_len(s, layer)
            if w.page_size:
                np.testing.assert_array_equal(pt, ora.page_table[s])
                np.testing.assert_array_equal(fcg.fcg_cache_export_v_alias(cache, s), ora.v_alias[s])


def run_pipeline(w, layers, n_decode, check_seqs, q_mult=1.0, shuffle=False, alias=False):
    from paper_2606_13097_amd import fcg, runner
    sh = w.shape
    say(f"[gpu] pipeline {w.name} L={sh.n_layers} seqs={w.n_seqs} decode={n_decode} q_mult={q_mult} "
        f"shuffle={shuffle} page={w.page_size} alias={alias}")
    setup = runner.GpuSetup(w, cache_flags=fcg.FCG_ALIAS_V if alias else 0)
    try:
        setup.graft()
        torch.cuda.synchronize()
        say("[gpu]   graft done")
        w_items = {}
        for layer in layers:
            w_inv = rope.inv_freq(sh.head_dim, sh.rope_theta)
            for s in check_seqs:
                items = oracle_items(w, s, layer)
                w_items[(s, layer)] = items
                K, V, wr = ograft.compose(w.max_tokens, sh.n_kv_heads, sh.head_dim, items, w_inv, sh.dtype)
                pos = np.flatnonzero(wr)
                gk, gv = read_cache(setup.cache, w, layer, s, pos, setup.lib)
                np.testing.assert_array_equal(numerics.decode(gv, sh.dtype), V[pos])
                check_keys(gk, K[pos], sh.dtype, f"graft keys seq {s} layer {layer}")
                # segments whose delta is 0 are copied bit for bit
                for dst, src, k_lib, _ in items:
                    if dst == src:
                        gk0, _ = read_cache(setup.cache, w, layer, s, np.arange(dst, dst + k_lib.shape[0]))
                        np.testing.assert_array_equal(gk0, k_lib)
        outs = {}
        order = np.arange(len(w.fresh_pos))
        if shuffle:
            order = np.random.default_rng(0).permutation(order)
        for layer in layers:
            q, k, v = setup.fresh_inputs(layer)
            if q_mult != 1.0:
                q = q * q_mult
            q, k, v = q[order].contiguous(), k[order].contiguous(), v[order].contiguous()
            out = torch.empty_like(q)
            from paper_2606_13097_amd import fcg
            fcg.fcg_patch_prefill(setup.cache, layer, w.fresh_seq[order], w.fresh_pos[order], q, k, v, out)
            res = torch.empty_like(out)
            res[torch.from_numpy(order).cuda()] = out
            outs[("prefill", layer)] = res
        torch.cuda.synchronize()
        say("[gpu]   prefill done")
        for layer in layers:
            dq, dk, dv = setup.decode_inputs(layer, n_decode)
            if q_mult != 1.0:
                dq = dq * q_mult
            douts = []
            for t in range(n_decode):
                o = torch.empty_like(dq[t])
                setup.decode(layer, dq[t], dk[t], dv[t], o)
                douts.append(o)
            outs[("decode", layer)] = douts
        torch.cuda.synchronize()
        say("[gpu]   decode done")
        ora = _oracle_layout(w, n_decode, layers, alias)
        _compare_layout(setup.cache, ora, w, layers)
        for layer in layers:
            for s in check_seqs:
                ref = oracle_run(w, s, layer, n_decode, q_mult)
                idx = np.flatnonzero(w.fresh_seq == s)
                got = storage_np(outs[("prefill", layer)][idx])
                check_attn(got, ref["prefill"], sh.dtype, f"prefill seq {s} layer {layer}")
                for t in range(n_decode):
                    got = storage_np(outs[("decode", layer)][t][s])
                    check_attn(got, ref["decode"][t], sh.dtype, f"decode seq {s} layer {layer} step {t}")
                # final cache: fresh and decode keys/values placed at their positions
                pos = np.flatnonzero(ref["written"])
                gk, gv = read_cache(setup.cache, w, layer, s, pos, setup.lib)
                np.testing.assert_array_equal(numerics.decode(gv, sh.dtype), ref["V"][pos])
                check_keys(gk, ref["K"][pos], sh.dtype, f"final keys seq {s} layer {layer}")
        say("[gpu]   parity ok")
    finally:
        setup.close()


def test_tiny_fp32_pipeline():
    from paper_2606_13097_amd import synth
    w = synth.workload("tiny", seed=1)
    run_pipeline(w, [0], 8, [0])


def test_tiny_fp32_shuffled_tokens_and_seed():
    from paper_2606_13097_amd import synth
    w = synth.workload("tiny", seed=3)
    run_pipeline(w, [0], 3, [0], shuffle=True)


def test_7b_shape_bf16_two_layers():
    from paper_2606_13097_amd import synth
    w = synth.workload("7b", seed=1, n_layers=2, n_lib=24)
    run_pipeline(w, [0, 1], 5, [0])


def test_7b_shape_bf16_peaked_queries():
    """Q x 8 gives score std ~4: attention far from uniform, so a tolerance of 2e-2 is not vacuous."""
    from paper_2606_13097_amd import synth
    w = synth.workload("7b", seed=2, n_layers=1, n_lib=16)
    run_pipeline(w, [0], 3, [0], q_mult=8.0)


def test_negative_and_positive_deltas_bf16():
    from paper_2606_13097_amd import synth
    w = synth.workload("7b", seed=4, n_layers=1, n_lib=16)
    rng = np.random.default_rng(4)
    w.lib_src_pos0 = rng.integers(0, 9000, size=len(w.lib_lengths)).astype(np.int32)
    run_pipeline(w, [0], 2, [0], shuffle=True)


def test_long_context_gap_tokens_bf16():
    from paper_2606_13097_amd import synth
    w = synth.workload("long16k", seed=1, n_layers=1, n_lib=24)
    run_pipeline(w, [0], 2, [0])


def test_batched_paged_bf16():
    from paper_2606_13097_amd import synth
    w = synth.workload("batched", seed=1, n_layers=1, n_lib=48)
    run_pipeline(w, [0], 3, [0, 7, 31])


def test_batched_paged_bf16_values_read_from_the_library():
    """The batched paged workload with value pages mapped onto the library
    (FCG_ALIAS_V): page tables and aliases bit-exact, values bit-exact where
    they are read (library or cache page), outputs within the bf16 bars."""
    from paper_2606_13097_amd import synth
    w = synth.workload("batched", seed=2, n_layers=1, n_lib=48)
    run_pipeline(w, [0], 3, [0, 5, 31], alias=True)


def test_tiny_fp32_paged_values_read_from_the_library():
    from paper_2606_13097_amd import synth
    w = dataclasses.replace(synth.workload("tiny", seed=3), page_size=16)
    run_pipeline(w, [0], 4, list(range(w.n_seqs)), alias=True)


def test_34b_shape_outliers_bf16():
    from paper_2606_13097_amd import synth
    w = synth.workload("34b", seed=1, n_layers=1, n_lib=40)
    # keep the oracle quick: 6 segments and 64 patch tokens per task
    keep = np.zeros(len(w.graft_seq), bool)
    for t in range(w.n_seqs):
        keep[np.flatnonzero(w.graft_seq == t)[:6]] = True
    w.graft_seq, w.graft_seg, w.graft_dst = w.graft_seq[keep], w.graft_seg[keep], w.graft_dst[keep]
    fresh = []
    for t in range(w.n_seqs):
        end = int((w.graft_dst[w.graft_seq == t] + w.lib_lengths[w.graft_seg[w.graft_seq == t]]).max())
        fresh += [(t, end + j, j) for j in range(64)]
    w.fresh_seq = np.array([f[0] for f in fresh], np.int32)
    w.fresh_pos = np.array([f[1] for f in fresh], np.int32)
    w.fresh_row = np.array([f[2] for f in fresh], np.int32)
    run_pipeline(w, [0], 2, [0, 3])


def test_causality_future_positions_do_not_change_outputs():
    """A segment grafted beyond every query position leaves prefill outputs bit-identical."""
    from paper_2606_13097_amd import fcg, runner, synth
    w = synth.workload("7b", seed=5, n_layers=1, n_lib=16)
    w.max_tokens += 2048
    say("[gpu] causality")
    a = runner.GpuSetup(w, n_caches=2)
    try:
        a.graft(a.caches[0])
        a.graft(a.caches[1])
        top = int(w.fresh_pos.max()) + 1
        fcg.fcg_graft(a.caches[1], a.lib, [0], [0], [top + 5])
        q, k, v = a.fresh_inputs(0)
        o1, o2 = torch.empty_like(q), torch.empty_like(q)
        a.prefill(0, q, k, v, o1, cache=a.caches[0])
        a.prefill(0, q, k, v, o2, cache=a.caches[1])
        torch.cuda.synchronize()
        assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    finally:
        a.close()


def test_needle_through_gpu_graft():
    """Keys encoded at 0..63, grafted at 3000: a query aimed at one of them retrieves its value."""
    from paper_2606_13097_amd import fcg
    D, Hkv, Hq, theta, dt = 128, 2, 8, 1e6, "bf16"
    say("[gpu] needle")
    desc = fcg.model_desc(1, Hq, Hkv, D, theta, dt)
    rng = np.random.default_rng(12)
    w = rope.inv_freq(D, theta)
    n = 64
    k_raw = rng.standard_normal((n, Hkv, D)) * 0.5
    j = 23
    k_raw[j] *= 2.0
    k_raw[j, :, 16:64] = 0.0
    k_raw[j, :, 80:] = 0.0
    k_lib = numerics.encode(rope.rotate(k_raw, np.arange(n)[:, None], w), dt)
    v_lib = np.zeros((n, Hkv, D))
    v_lib[j] = 1.0
    v_lib = numerics.encode(v_lib, dt)
    filler_k = numerics.encode(rng.standard_normal((3000, Hkv, D)) * 0.5, dt)
    filler_v = numerics.encode(np.zeros((3000, Hkv, D)), dt)
    lib = fcg.Library(desc, 3064, 2)
    fcg.fcg_lib_add_segment(lib, 3000, 0, to_device(filler_k, dt), to_device(filler_v, dt))
    fcg.fcg_lib_add_segment(lib, n, 0, to_device(k_lib, dt), to_device(v_lib, dt))
    cache = fcg.Cache(desc, 1, 4096)
    fcg.fcg_graft(cache, lib, [0, 0], [0, 1], [0, 3000])
    p_q = 3064
    p_k = 3000 + j
    q_raw = np.zeros((1, Hq, D))
    for hq in range(Hq):
        q_raw[0, hq] = 8.0 * rope.rotate(k_raw[j, hq // (Hq // Hkv)], p_k - p_q, w)
    q = to_device(numerics.encode(q_raw, dt), dt)
    kk = to_device(numerics.encode(np.zeros((1, Hkv, D)), dt), dt)
    out = torch.empty_like(q)
    fcg.fcg_patch_prefill(cache, 0, [0], [p_q], q, kk, kk, out)
    o = numerics.decode(storage_np(out), dt)
    assert np.all(o > 0.98), o.min()
    cache.close()
    lib.close()


def test_errors_on_device_cache_change_nothing():
    from paper_2606_13097_amd import fcg, runner, synth
    w = synth.workload("tiny", seed=1)
    say("[gpu] errors")
    s = runner.GpuSetup(w)
    try:
        s.graft()
        before = fcg.fcg_cache_export_layout(s.cache, 0, 0)
        with pytest.raises(fcg.FcgError) as e:
            s.graft()
        assert e.value.status == fcg.FCG_EOVERLAP
        q, k, v = s.fresh_inputs(0)
        out = torch.empty_like(q)
        with pytest.raises(fcg.FcgError) as e:
            fcg.fcg_patch_prefill(s.cache, 0, [0], [int(w.fresh_pos.max()) + 3], q[:1], k[:1], v[:1], out[:1])
        assert e.value.status == fcg.FCG_EHOLE
        with pytest.raises(fcg.FcgError) as e:
            fcg.fcg_decode(s.cache, 1, [0], q[:1], k[:1], v[:1], out[:1])
        assert e.value.status == fcg.FCG_ERANGE
        after = fcg.fcg_cache_export_layout(s.cache, 0, 0)
        assert after[1] == before[1] and np.array_equal(after[2], before[2])
        # empty calls are no-ops
        fcg.fcg_graft(s.cache, s.lib, [], [], [])
        fcg.fcg_patch_prefill(s.cache, 0, [], [], q, k, v, out)
        assert len(fcg.fcg_decode(s.cache, 0, [], q, k, v, out)) == 0
        torch.cuda.synchronize()
    finally:
        s.close()


def test_synth_gpu_twin_matches_host_bits():
    from paper_2606_13097_amd import synth
    from paper_2606_13097_amd.synth import gpu as sg
    say("[gpu] synth twin")
    for tag, dt, rate in (("lib_k", "f32", 0.0), ("lib_v", "bf16", 0.0), ("lib_k", "bf16", 0.05),
                          ("fresh_q", "bf16", 0.05), ("dec_v", "bf16", 0.05)):
        t = torch.empty((37, 8, 128), dtype=torch.float32 if dt == "f32" else torch.bfloat16, device="cuda")
        sg.fill_rows(t, dt, 7, tag, 3, 11, 5, 0.5, rate)
        ref = synth.tensor_values(7, tag, 3, 11, np.arange(5, 42), 8, 128, 0.5, dt, rate)
        np.testing.assert_array_equal(storage_np(t), ref)


def test_kernel_timing_counts_calls():
    from paper_2606_13097_amd import fcg, runner, synth
    w = synth.workload("7b", seed=6, n_layers=2, n_lib=8)
    say("[gpu] timing")
    s = runner.GpuSetup(w)
    try:
        fcg.fcg_cache_timing(s.cache, True)
        s.graft()
        for layer in range(2):
            q, k, v = s.fresh_inputs(layer)
            s.prefill(layer, q, k, v, torch.empty_like(q))
        dq, dk, dv = s.decode_inputs(0, 3)
        for t in range(3):
            s.decode(0, dq[t], dk[t], dv[t], torch.empty_like(dq[t]))
        counts = [fcg.fcg_cache_timing_read(s.cache, k) for k in range(5)]
        assert [c[0] for c in counts] == [1, 2, 2, 3, 3]
        assert all(c[1] > 0 for c in counts)
        assert counts[2][1] >= counts[1][1]            # the whole prefill includes its attention kernel
        assert counts[3][1] >= counts[4][1]            # the whole decode includes its attention kernel
    finally:
        s.close()


@pytest.mark.gpu
@pytest.mark.parametrize("hq,hkv,d,dtype", [(32, 8, 128, "bf16"), (64, 8, 128, "bf16"), (8, 4, 64, "bf16"),
                                            (4, 4, 128, "bf16"), (16, 1, 64, "bf16"),
                                            (4, 2, 64, "f32")])
def test_decode_split_edges(hq, hkv, d, dtype):
    """Decode positions on and next to the 64-key split boundaries (a last split holding only
    the new token, a split ending on the last cached key), in a batch whose sequences have
    different split counts (empty padding splits), plus three-token prefills."""
    from paper_2606_13097_amd import synth
    shape = synth.Shape(1, hq, hkv, d, 1e4, dtype)
    lengths = [58, 61, 124, 125, 197, 252]       # contexts 61, 64, 127, 128, 200, 255 after 3 fresh tokens
    w = synth.custom(shape, 11, lengths, [[i] for i in range(len(lengths))], n_fresh=3, n_decode=3)
    run_pipeline(w, [0], 3, list(range(w.n_seqs)))


@pytest.mark.gpu
@pytest.mark.parametrize("hq,d,dtype", [(16, 128, "bf16"), (8, 128, "bf16"), (16, 128, "f32"), (4, 64, "f32")])
def test_decode_merge_of_many_splits(hq, d, dtype):
    """One kv head and a ~3K-token context: 47 splits of 64 keys, so the last block's
    merge of the splits takes several rounds of loads (large query groups) and several
    rounds of LDS sums (16 query heads)."""
    shape = synth.Shape(1, hq, 1, d, 1e4, dtype)
    w = synth.custom(shape, 19, [2990], [[0]], n_fresh=3, n_decode=3)
    run_pipeline(w, [0], 3, [0])


@pytest.mark.gpu
def test_many_sequences_split_over_launches():
    """130 sequences: the prefill row blocks fill two attention launches (128 row blocks
    each at most) and decode runs in three launch groups (64 sequences each at most)."""
    from paper_2606_13097_amd import synth
    shape = synth.Shape(1, 32, 8, 128, 1e6, "bf16")
    n = 130
    lengths = [40 + 7 * (i % 9) for i in range(n)]
    w = synth.custom(shape, 13, lengths, [[i] for i in range(n)], n_fresh=2, n_decode=2)
    run_pipeline(w, [0], 2, [0, 63, 64, 127, 128, 129])


@pytest.mark.gpu
def test_prefill_one_block_per_cu_path():
    """64 sequences x 64 patch tokens at g = 4: 64 row blocks of 256 rows per kv head, 512
    (row block, kv head) pairs, so the planner keeps one 8-wave block per CU (smaller calls
    take two 4-wave blocks per CU)."""
    from paper_2606_13097_amd import synth
    shape = synth.Shape(1, 32, 8, 128, 1e6, "bf16")
    n = 64
    lengths = [60 + 5 * (i % 7) for i in range(n)]
    w = synth.custom(shape, 17, lengths, [[i] for i in range(n)], n_fresh=64, n_decode=1)
    run_pipeline(w, [0], 1, [0, 31, 63])


@pytest.mark.gpu
def test_paged_prefill_split_past_the_page_window():
    """64 sequences share one 8,500-token segment (paged), 16 patch tokens each at g = 16: one
    256-row block per sequence, 512 (row block, kv head) pairs, so one block per CU and one
    unsplit key range of 533 pages, more than the 520 page entries a block keeps in LDS; the
    blocks then read page-table entries per row."""
    from paper_2606_13097_amd import synth
    shape = synth.Shape(1, 128, 8, 64, 1e4, "bf16")
    n = 64
    w = synth.custom(shape, 23, [8500], [[0]] * n, n_fresh=16, n_decode=1, page_size=16)
    run_pipeline(w, [0], 1, [0, 63])


def _tokens(w, tag, layer, item, rows):
    sh = w.shape
    q = tag.endswith("q")
    return synth.tensor_values(w.seed, tag, layer, item, np.asarray(rows), sh.n_q_heads if q else sh.n_kv_heads,
                               sh.head_dim, w.q_scale if q else w.kv_scale, sh.dtype, w.outlier_rate)


@pytest.mark.gpu
@pytest.mark.parametrize("dtype,page,alias", [("bf16", 0, False), ("bf16", 16, False), ("f32", 16, False),
                                               ("bf16", 16, True), ("f32", 16, True)])
def test_cache_patching_cut_regenerate_decode(dtype, page, alias):
    """Cache-patching (Sec. 4.2, Eq. 6): after graft -> prefill -> two decode steps,
    each sequence is cut back to an error position -- inside its grafted context on
    a page boundary, inside its fresh span, at its full length (nothing cut), at 0
    (nothing kept) -- a new span is prefilled from there in one call and two more
    decode steps follow.  Outputs, layout (freed pages taken again) and cache
    contents match the oracle's patch step run on the oracle's own first pass."""
    from paper_2606_13097_amd import fcg, runner
    shape = synth.Shape(2, 32, 8, 128, 1e6, "bf16") if dtype == "bf16" else synth.Shape(2, 4, 2, 64, 1e4, "f32")
    w = synth.custom(shape, 17, [90, 130, 200, 64], [[0, 1], [2], [3, 1], [2, 0]], n_fresh=5, n_decode=2,
                     page_size=page)
    # contexts 220, 200, 194, 290; 5 fresh tokens, 2 decoded.  With value
    # aliasing, the cut at 100 splits a page whose values are read from the
    # library: its kept rows are copied into the page before new tokens follow
    keep = [100 if alias else 96, 203, 201, 0]
    n_new = [37, 9, 1, 70]
    layers = [0, 1]
    sh = w.shape
    say(f"[gpu] cache patching {dtype} page={page} alias={alias} keep={keep} new={n_new}")
    setup = runner.GpuSetup(w, cache_flags=fcg.FCG_ALIAS_V if alias else 0)
    try:
        setup.graft()
        for layer in layers:
            q, k, v = setup.fresh_inputs(layer)
            setup.prefill(layer, q, k, v, torch.empty_like(q))
        for layer in layers:
            dq, dk, dv = setup.decode_inputs(layer, 2)
            for t in range(2):
                setup.decode(layer, dq[t], dk[t], dv[t], torch.empty_like(dq[t]))
        torch.cuda.synchronize()
        for s, e in enumerate(keep):
            fcg.fcg_cache_truncate(setup.cache, s, e)
        seqs = np.concatenate([np.full(n, s, np.int32) for s, n in enumerate(n_new)])
        pos = np.concatenate([np.arange(e, e + n, dtype=np.int32) for e, n in zip(keep, n_new)])
        outs = {}
        for layer in layers:
            q, k, v = (to_device(np.concatenate([_tokens(w, "fresh_" + x, layer, 100 + s, np.arange(n))
                                                 for s, n in enumerate(n_new)]), dtype) for x in "qkv")
            out = torch.empty_like(q)
            fcg.fcg_patch_prefill(setup.cache, layer, seqs, pos, q, k, v, out)
            outs[("prefill", layer)] = out
        for layer in layers:
            for t in range(2):
                q, k, v = (to_device(np.stack([_tokens(w, "dec_" + x, layer, 100 + s, [t])[0]
                                               for s in range(w.n_seqs)]), dtype) for x in "qkv")
                out = torch.empty_like(q)
                p = fcg.fcg_decode(setup.cache, layer, np.arange(w.n_seqs), q, k, v, out)
                assert list(p) == [e + n + t for e, n in zip(keep, n_new)]
                outs[("decode", layer, t)] = out
        torch.cuda.synchronize()
        say("[gpu]   patch done")
        ora = _oracle_layout(w, 2, layers, alias)
        for s, e in enumerate(keep):
            ora.truncate(s, e)
        for layer in layers:
            ora.append(layer, seqs, pos)
        for layer in layers:
            for _ in range(2):
                ora.decode(layer, list(range(w.n_seqs)))
        _compare_layout(setup.cache, ora, w, layers)
        for layer in layers:
            for s, (e, n) in enumerate(zip(keep, n_new)):
                state = oracle_run(w, s, layer, 2)
                rows = np.arange(n)
                ref = task.patch_layer(state, sh.n_q_heads, sh.head_dim, sh.rope_theta, dtype, e,
                                       np.arange(e, e + n), *(_tokens(w, "fresh_" + x, layer, 100 + s, rows)
                                                              for x in "qkv"),
                                       *([_tokens(w, "dec_" + x, layer, 100 + s, [t])[0] for t in range(2)]
                                         for x in "qkv"))
                got = storage_np(outs[("prefill", layer)][torch.from_numpy(np.flatnonzero(seqs == s)).cuda()])
                check_attn(got, ref["prefill"], dtype, f"patch prefill seq {s} layer {layer}")
                for t in range(2):
                    check_attn(storage_np(outs[("decode", layer, t)][s]), ref["decode"][t], dtype,
                               f"patch decode seq {s} layer {layer} step {t}")
                wpos = np.flatnonzero(ref["written"])
                gk, gv = read_cache(setup.cache, w, layer, s, wpos, setup.lib)
                np.testing.assert_array_equal(numerics.decode(gv, dtype), ref["V"][wpos])
                check_keys(gk, ref["K"][wpos], dtype, f"patched keys seq {s} layer {layer}")
        say("[gpu]   patch parity ok")
    finally:
        setup.close()


@pytest.mark.gpu
def test_offload_reload_round_trip_is_bit_exact():
    """Segments offloaded to the pinned host tier and reloaded at other device offsets
    (a new segment took their old range) graft exactly as before: every grafted key and
    value of the cache is bit-identical to the first graft's."""
    from paper_2606_13097_amd import fcg, runner
    w = synth.workload("7b", seed=5, n_layers=2, n_lib=12)
    segs = sorted(set(int(g) for g in w.graft_seg))
    spare = int(sum(int(w.lib_lengths[g]) for g in segs))   # room to reload every one past the others
    say(f"[gpu] offload/reload segs={segs}")
    setup = runner.GpuSetup(w, lib_spare_tokens=spare)
    try:
        fcg.fcg_lib_host_reserve(setup.lib, int(w.lib_lengths.sum()))
        setup.graft()
        pos = np.flatnonzero(fcg.fcg_cache_export_layout(setup.cache, 0, 0)[2])
        ref = [read_cache(setup.cache, w, layer, 0, pos) for layer in range(2)]
        before = {g: fcg.fcg_lib_segment_info(setup.lib, g)[0] for g in segs}
        for g in segs:
            fcg.fcg_lib_offload(setup.lib, g)
        # a new segment as long as the first offloaded one takes the lowest freed range
        fcg.fcg_lib_add_segment(setup.lib, int(w.lib_lengths[segs[0]]), 0)
        for g in reversed(segs):
            fcg.fcg_lib_reload(setup.lib, g)
        after = {g: fcg.fcg_lib_segment_info(setup.lib, g)[0] for g in segs}
        assert any(after[g] != before[g] for g in segs), (before, after)
        assert all(fcg.fcg_lib_segment_state(setup.lib, g) == (True, True) for g in segs)
        setup.reset()
        setup.graft()
        torch.cuda.synchronize()
        for layer in range(2):
            gk, gv = read_cache(setup.cache, w, layer, 0, pos)
            np.testing.assert_array_equal(gk, ref[layer][0])
            np.testing.assert_array_equal(gv, ref[layer][1])
        say("[gpu]   round trip bit-exact")
    finally:
        setup.close()


def _random_case(i):
    rng = np.random.default_rng(1000 + i)
    shape = [synth.Shape(1, 4, 2, 64, 1e4, "f32"), synth.Shape(1, 8, 2, 128, 1e6, "bf16"),
             synth.Shape(1, 16, 1, 64, 1e4, "bf16"), synth.Shape(1, 32, 8, 128, 1e6, "bf16")][i % 4]
    n_seg = int(rng.integers(1, 7))
    lengths = [int(x) for x in rng.integers(1, 300, size=n_seg)]
    n_seqs = int(rng.integers(1, 9))
    segs = [list(rng.choice(n_seg, size=int(rng.integers(1, min(n_seg, 3) + 1)), replace=False))
            for _ in range(n_seqs)]
    page = int(rng.choice([0, 16]))
    alias = bool(page and rng.integers(0, 2))
    n_fresh, n_dec = int(rng.integers(1, 100)), int(rng.integers(1, 4))
    w = synth.custom(shape, 2000 + i, lengths, segs, n_fresh=n_fresh, n_decode=n_dec, page_size=page)
    return w, n_dec, alias


@pytest.mark.gpu
@pytest.mark.parametrize("i", range(24))
def test_random_small_plans(i):
    """Seeded random plans: 1-8 sequences grafting 1-3 of up to 6 segments of 1-299 tokens,
    1-99 fresh tokens (one to a dozen MFMA row blocks per sequence, so both prefill block
    orders), 1-3 decode steps, over four head layouts, contiguous or paged caches, values
    copied or read from the library; every sequence checked against the oracle."""
    w, n_dec, alias = _random_case(i)
    run_pipeline(w, [0], n_dec, list(range(w.n_seqs)), alias=alias)


@pytest.mark.gpu
def test_residency_updates_on_a_side_stream_keep_grafts_exact():
    """The cache-management loop under a tight device budget (Alg. 1: update after each
    task; Sec. 4.1 and App. C.5: low-scored entries to DRAM, reloaded only when needed):
    after every task the locality update offloads and reloads segments on a side stream,
    the next task reloads the segments it needs there too, and its graft on the main
    stream -- ordered after those copies by the library's events -- equals the oracle's
    graft of the generated library values (keys within the key bar, values bit for bit),
    though the segments now sit at other device offsets."""
    from paper_2606_13097_amd import fcg, runner
    w = synth.workload("7b", seed=5, n_layers=2, n_lib=16)
    sh = w.shape
    b_tok = sh.token_bytes
    tasks = [synth.workload("7b", seed=5, n_layers=2, n_lib=16, task=t) for t in range(6)]
    w.max_tokens = max(t.max_tokens for t in tasks)
    setup = runner.GpuSetup(w, lib_spare_tokens=int(w.lib_lengths.sum()) // 2)
    side = torch.cuda.Stream()
    loc = fcg.Locality(len(w.lib_lengths))
    rng = np.random.default_rng(5)
    try:
        lib = setup.lib
        fcg.fcg_lib_host_reserve(lib, int(w.lib_lengths.sum()))
        for f in range(len(w.lib_lengths)):
            fcg.fcg_locality_set_ppl(loc, f, float(rng.uniform(2.0, 30.0)))
        budget = int(w.lib_lengths.sum() * b_tok * 0.45)
        winv = rope.inv_freq(sh.head_dim, sh.rope_theta)
        moves = [0, 0, 0]
        for t, tw in enumerate(tasks):
            need = [int(g) for g in tw.graft_seg]
            for g in need:
                if not fcg.fcg_lib_segment_state(lib, g)[0]:
                    fcg.fcg_lib_reload(lib, g, side)
                    moves[2] += 1
            setup.reset()
            fcg.fcg_graft(setup.cache, lib, tw.graft_seq, tw.graft_seg, tw.graft_dst)
            # the update step right away, on the side stream, beside the graft
            fcg.fcg_locality_record(loc, need)
            n_off, n_re = fcg.fcg_lib_update_residency(lib, loc, budget, 15.0, side)
            moves[0] += n_off
            moves[1] += n_re
            torch.cuda.synchronize()
            for layer in range(sh.n_layers):
                items = oracle_items(tw, 0, layer)
                K, V, wr = ograft.compose(tw.max_tokens, sh.n_kv_heads, sh.head_dim, items, winv, sh.dtype)
                pos = np.flatnonzero(wr)
                gk, gv = read_cache(setup.cache, tw, layer, 0, pos)
                np.testing.assert_array_equal(numerics.decode(gv, sh.dtype), V[pos])
                check_keys(gk, K[pos], sh.dtype, f"task {t} layer {layer} keys after residency updates")
        say(f"[gpu]   offloads {moves[0]}, reloads by the update {moves[1]}, reloads on demand {moves[2]}")
        assert moves[0] > 0 and moves[1] + moves[2] > 0
    finally:
        loc.close()
        setup.close()
