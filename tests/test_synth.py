"""The seeded input generator (paper_2606_13097_amd/synth): definition and workload plans."""
import os

import numpy as np
import pytest
import torch

from paper_2606_13097_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_splitmix64_reference_outputs():
    with open(os.path.join(GOLDEN, "splitmix64_seed1234567.txt")) as f:
        want = [int(l) for l in f if l.strip() and not l.startswith("#")]
    s = np.uint64(1234567)
    with np.errstate(over="ignore"):
        got = [int(synth.mix64(s + np.uint64(k) * synth.GAMMA)) for k in range(1, 6)]
    assert got == want


def test_values_exact_deterministic_and_normal():
    c = np.arange(1_000_000, dtype=np.uint64)
    x = synth.normal_f32(1, c)
    np.testing.assert_array_equal(x, synth.normal_f32(1, c))
    assert not np.array_equal(x, synth.normal_f32(2, c))
    # (sum - 393210) / 65536 is exact in fp32
    np.testing.assert_array_equal(x.astype(np.float64) * 65536, np.rint(x.astype(np.float64) * 65536))
    assert abs(x.mean()) < 5e-3 and abs(x.var() - 1.0) < 5e-3
    assert np.abs(x).max() < 6.0


def test_counter_fields_do_not_collide():
    t, l, i, r, c = np.meshgrid([0, 1, 15], [0, 1, 255], [0, 1, 65535], [0, 1, 2**20 - 1],
                                [0, 1, 8191], indexing="ij")
    cs = synth.counter(t, l, i, r, c).ravel()
    assert len(np.unique(cs)) == cs.size
    with pytest.raises(ValueError):
        synth.counter(0, 0, 0, 2**20, 0)


def test_bf16_storage_is_rne():
    x = synth.tensor_values(3, "lib_k", 0, 0, np.arange(64), 8, 128, 0.5, "f32")
    b = synth.tensor_values(3, "lib_k", 0, 0, np.arange(64), 8, 128, 0.5, "bf16")
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(b, ref)


def test_outlier_pairs_rate_and_factor():
    m = np.stack([synth.outlier_pairs(5, l, 8, 128, 0.01) for l in range(48)])
    n = m.size
    assert abs(m.mean() - 0.01) < 4 * np.sqrt(0.01 * 0.99 / n)
    x = synth.tensor_values(5, "lib_k", 7, 3, np.arange(4), 8, 128, 1.0, "f32", outlier_rate=0.01)
    y = synth.tensor_values(5, "lib_k", 7, 3, np.arange(4), 8, 128, 1.0, "f32")
    mm = synth.outlier_pairs(5, 7, 8, 128, 0.01)
    full = np.concatenate([mm, mm], axis=1)
    np.testing.assert_array_equal(x[:, full], 8 * y[:, full])
    np.testing.assert_array_equal(x[:, ~full], y[:, ~full])


def _check_plan(w):
    for s in range(w.n_seqs):
        occ = np.zeros(w.max_tokens, int)
        m = w.graft_seq == s
        for g, d in zip(w.graft_seg[m], w.graft_dst[m]):
            occ[d:d + w.lib_lengths[g]] += 1
        pos, rows = w.fresh_of_seq(s)
        occ[pos] += 1
        end = w.seq_len_after_prefill(s)
        assert occ.max() == 1 and occ[:end].min() == 1        # disjoint, no holes
        assert end + w.n_decode <= w.max_tokens
        assert sorted(rows.tolist()) == list(range(len(rows)))


@pytest.mark.parametrize("name", synth.WORKLOADS)
def test_workload_plans(name):
    w = synth.workload(name, seed=1)
    _check_plan(w)
    sh = w.shape
    if name == "tiny":
        assert (sh.n_layers, sh.n_q_heads, sh.n_kv_heads, sh.head_dim, sh.dtype) == (1, 4, 2, 64, "f32")
        assert set(w.lib_lengths[:8].tolist()) <= {96, 128, 160} and w.lib_lengths[8] == 64
        assert len(w.graft_seg) == 4 and w.graft_seg[0] == 8 and len(w.fresh_pos) == 16 and w.n_decode == 8
    elif name == "7b":
        assert (sh.n_layers, sh.n_q_heads, sh.n_kv_heads, sh.head_dim, sh.dtype) == (32, 32, 8, 128, "bf16")
        assert w.lib_lengths[:256].min() >= 200 and w.lib_lengths[:256].max() <= 800
        assert w.lib_lengths[256] == 1024 and len(w.graft_seg) == 7 and len(w.fresh_pos) == 64
        assert w.n_decode == 256 and 3000 < w.grafted_tokens < 6000
    elif name == "long16k":
        assert len(w.graft_seg) == 21 and w.lib_lengths[w.graft_seg[0]] == 2048
        gaps = len(w.fresh_pos) - 256
        assert 0 <= gaps <= 20 * 32 and w.n_decode == 128
    elif name == "batched":
        assert w.n_seqs == 32 and w.page_size == 16 and len(w.graft_seg) == 256
        assert len(np.unique(w.graft_seg)) < 256                 # segments shared by tasks
        assert len(w.fresh_pos) == 32 * 32 and w.n_decode == 128
    elif name == "34b":
        assert (sh.n_layers, sh.n_q_heads, sh.n_kv_heads) == (48, 64, 8) and w.outlier_rate == 0.01
        assert w.n_seqs == 4 and len(w.graft_seg) == 96 and len(w.fresh_pos) == 2048
