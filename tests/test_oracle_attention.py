"""Pins of the oracle's causal GQA attention (oracle/attention.py, oracle/task.py)."""
import numpy as np
import pytest
import torch

from oracle import attention, graft, numerics, rope, task


def _rand_cache(N, Hkv, D, seed=0):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((N, Hkv, D)), rng.standard_normal((N, Hkv, D)), np.ones(N, bool)


def _sdpa(q, pos, K, V, g):
    """torch's scaled_dot_product_attention, float64 on CPU, explicit boolean mask."""
    n, Hq, D = q.shape
    N = K.shape[0]
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]                      # [1][Hq][n][D]
    kt = torch.from_numpy(K).permute(1, 0, 2).repeat_interleave(g, 0)[None].contiguous()
    vt = torch.from_numpy(V).permute(1, 0, 2).repeat_interleave(g, 0)[None].contiguous()
    mask = torch.from_numpy(np.arange(N)[None, :] <= np.asarray(pos)[:, None])
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask)
    return o[0].permute(1, 0, 2).numpy()


@pytest.mark.parametrize("Hq,Hkv,D", [(4, 2, 64), (32, 8, 128), (8, 8, 32), (8, 1, 16)])
def test_matches_torch_sdpa(Hq, Hkv, D):
    K, V, wr = _rand_cache(300, Hkv, D, seed=Hq)
    rng = np.random.default_rng(5)
    q = rng.standard_normal((20, Hq, D)) * 2.0
    pos = rng.integers(0, 300, 20)
    got = attention.attend(q, pos, K, V, wr)
    np.testing.assert_allclose(got, _sdpa(q, pos, K, V, Hq // Hkv), rtol=0, atol=1e-12)


def test_rows_sum_to_one_and_single_key():
    K, _, wr = _rand_cache(64, 2, 32, seed=1)
    V = np.ones_like(K)
    q = np.random.default_rng(2).standard_normal((5, 4, 32)) * 5
    pos = [0, 3, 10, 40, 63]
    np.testing.assert_allclose(attention.attend(q, pos, K, V, wr), 1.0, rtol=0, atol=1e-13)
    Vr = np.random.default_rng(3).standard_normal(K.shape)
    o = attention.attend_row(q[0], 0, K, Vr, wr)                  # only position 0 visible
    np.testing.assert_array_equal(o, np.repeat(Vr[0], 2, axis=0))


def test_zero_query_gives_mean_of_visible_values():
    K, V, wr = _rand_cache(100, 2, 16, seed=4)
    o = attention.attend_row(np.zeros((4, 16)), 57, K, V, wr)
    for hq in range(4):
        np.testing.assert_allclose(o[hq], V[:58, hq // 2].mean(axis=0), rtol=0, atol=1e-13)


def test_causality_and_unwritten_rejection():
    K, V, wr = _rand_cache(80, 2, 16, seed=5)
    q = np.random.default_rng(6).standard_normal((4, 16))
    o1 = attention.attend_row(q, 40, K, V, wr)
    K2, V2 = K.copy(), V.copy()
    K2[41:] += 100.0
    V2[41:] -= 3.0
    np.testing.assert_array_equal(attention.attend_row(q, 40, K2, V2, wr), o1)
    wr2 = wr.copy()
    wr2[12] = False
    with pytest.raises(ValueError):
        attention.attend_row(q, 40, K, V, wr2)


def _task_inputs(seed, D=64, Hq=4, Hkv=2, dtype="f32", n_fresh=6):
    rng = np.random.default_rng(seed)
    enc = lambda a: numerics.encode(a, dtype)
    items = [(0, 0, enc(rng.standard_normal((30, Hkv, D))), enc(rng.standard_normal((30, Hkv, D)))),
             (30, 0, enc(rng.standard_normal((20, Hkv, D))), enc(rng.standard_normal((20, Hkv, D))))]
    fq = enc(rng.standard_normal((n_fresh, Hq, D)))
    fk = enc(rng.standard_normal((n_fresh, Hkv, D)))
    fv = enc(rng.standard_normal((n_fresh, Hkv, D)))
    return items, fq, fk, fv


def test_shift_invariance():
    """Encoding every key and query c positions later leaves the outputs unchanged."""
    D, Hkv, Hq, N = 64, 2, 4, 120
    rng = np.random.default_rng(7)
    w = rope.inv_freq(D, 1e4)
    k_raw = rng.standard_normal((N, Hkv, D))
    V = rng.standard_normal((N, Hkv, D))
    q_raw = rng.standard_normal((5, Hq, D)) * 2
    pos = np.array([10, 40, 77, 100, 119])
    wr = np.ones(N, bool)
    outs = []
    for c in (0, 37, 5000):
        K = rope.rotate(k_raw, (np.arange(N) + c)[:, None], w)
        q = rope.rotate(q_raw, (pos + c)[:, None], w)
        outs.append(attention.attend(q, pos, K, V, wr))
    np.testing.assert_allclose(outs[1], outs[0], rtol=0, atol=1e-11)
    np.testing.assert_allclose(outs[2], outs[0], rtol=0, atol=1e-10)


def test_decode_step_equals_last_prefill_row():
    D = 64
    items, fq, fk, fv = _task_inputs(9)
    full = task.run_layer(4, 2, D, 1e4, "f32", 200, items, np.arange(50, 56), fq, fk, fv)
    part = task.run_layer(4, 2, D, 1e4, "f32", 200, items, np.arange(50, 55), fq[:5], fk[:5], fv[:5],
                          dec_q=[fq[5]], dec_k=[fk[5]], dec_v=[fv[5]])
    assert part["decode_pos"].tolist() == [55]
    np.testing.assert_array_equal(part["decode"][0], full["prefill"][5])
    np.testing.assert_array_equal(part["prefill"], full["prefill"][:5])


def test_group_one_is_multi_head_attention():
    K, V, wr = _rand_cache(90, 8, 32, seed=10)
    q = np.random.default_rng(11).standard_normal((3, 8, 32))
    got = attention.attend(q, [10, 50, 89], K, V, wr)
    for h in range(8):
        ref = _sdpa(q[:, h:h + 1], [10, 50, 89], K[:, h:h + 1], V[:, h:h + 1], 1)
        np.testing.assert_allclose(got[:, h:h + 1], ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_needle_through_graft(dtype):
    """A query aimed at one grafted key finds it only if the key was turned to its new position."""
    D, Hkv, Hq, theta = 128, 2, 4, 1e6
    rng = np.random.default_rng(12)
    w = rope.inv_freq(D, theta)
    n = 64
    k_raw = rng.standard_normal((n, Hkv, D)) * 0.5
    j = 23                                                    # the needle token
    # the needle lives on the 16 fastest-turning pairs only, so a key left unturned is lost
    k_raw[j] *= 2.0
    k_raw[j, :, 16:64] = 0.0
    k_raw[j, :, 80:] = 0.0
    k_lib = numerics.encode(rope.rotate(k_raw, np.arange(n)[:, None], w), dtype)   # captured at 0..63
    v_lib = np.zeros((n, Hkv, D))
    v_lib[j] = 1.0
    v_lib = numerics.encode(v_lib, dtype)
    other_k = numerics.encode(rng.standard_normal((500, Hkv, D)) * 0.5, dtype)
    other_v = numerics.encode(np.zeros((500, Hkv, D)), dtype)
    dst = 500                                                 # grafted behind 500 other tokens
    items = [(0, 0, other_k, other_v), (dst, 0, k_lib, v_lib)]
    p_q = 700
    # query (pre-encoding) = c * R(p_k - p_q) k_raw so that R(p_q) q = c * R(p_k) k_raw
    p_k = dst + j
    q_raw = np.zeros((1, Hq, D))
    for hq in range(Hq):
        q_raw[0, hq] = 8.0 * rope.rotate(k_raw[j, hq // 2], p_k - p_q, w)
    fill = numerics.encode(rng.standard_normal((p_q - dst - n + 1, Hkv, D)) * 0.5, dtype)
    fpos = np.arange(dst + n, p_q + 1)
    fq = numerics.encode(np.repeat(q_raw, len(fpos), axis=0), dtype)
    out = task.run_layer(Hq, Hkv, D, theta, dtype, 800, items, fpos, fq, fill,
                         numerics.encode(np.zeros((len(fpos), Hkv, D)), dtype))
    o = out["prefill"][-1]
    assert np.all(o > 0.99)                                   # the needle's value, 1.0
    # a graft that forgot to turn the keys loses the needle
    K_bad = out["K"].copy()
    K_bad[dst:dst + n] = numerics.decode(k_lib, dtype)
    q_enc = graft.encode_fresh(fq[-1:], [p_q], w, dtype)[0]
    o_bad = attention.attend_row(q_enc, p_q, K_bad, out["V"], out["written"])
    assert np.all(o_bad < 0.5)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("keep", [0, 17, 30, 50, 53, 57, 58])
def test_patch_equals_a_fresh_run_on_the_kept_prefix(dtype, keep):
    """Cache-patching (Sec. 4.2, Eq. 6): cutting a finished run back to ``keep`` and
    prefilling a new span there gives what a run built from scratch on the kept
    prefix gives, whether the cut falls in the grafted context (on or off a segment
    boundary), in the fresh span, among the decoded tokens, at 0 or past the end."""
    D, Hq, Hkv, theta = 64, 4, 2, 1e4
    items, fq, fk, fv = _task_inputs(21, D, Hq, Hkv, dtype)
    rng = np.random.default_rng(22)
    enc = lambda a: numerics.encode(a, dtype)
    dq, dk, dv = (enc(rng.standard_normal((2, h, D))) for h in (Hq, Hkv, Hkv))
    full = task.run_layer(Hq, Hkv, D, theta, dtype, 200, items, np.arange(50, 56), fq, fk, fv,
                          list(dq), list(dk), list(dv))
    m = 9
    cq, ck, cv = (enc(rng.standard_normal((m, h, D))) for h in (Hq, Hkv, Hkv))
    eq, ek, ev = (enc(rng.standard_normal((2, h, D))) for h in (Hq, Hkv, Hkv))
    cot = np.arange(keep, keep + m)
    got = task.patch_layer(full, Hq, D, theta, dtype, keep, cot, cq, ck, cv, list(eq), list(ek), list(ev))
    # from scratch: graft only the kept part of each segment; kept fresh and decoded
    # tokens (positions 50..57, encoded alike) become fresh tokens before the new span
    cut = [(d, s, k[:keep - d], v[:keep - d]) for d, s, k, v in items if d < keep]
    tq, tk, tv = np.concatenate([fq, dq]), np.concatenate([fk, dk]), np.concatenate([fv, dv])
    n_old = max(0, keep - 50)
    ref = task.run_layer(Hq, Hkv, D, theta, dtype, 200, cut, np.concatenate([np.arange(50, 50 + n_old), cot]),
                         np.concatenate([tq[:n_old], cq]), np.concatenate([tk[:n_old], ck]),
                         np.concatenate([tv[:n_old], cv]), list(eq), list(ek), list(ev))
    np.testing.assert_allclose(got["prefill"], ref["prefill"][n_old:], rtol=0, atol=1e-12)
    np.testing.assert_allclose(got["decode"], ref["decode"], rtol=0, atol=1e-12)
    np.testing.assert_array_equal(got["written"], ref["written"])
    np.testing.assert_array_equal(got["K"][ref["written"]], ref["K"][ref["written"]])
    np.testing.assert_array_equal(got["V"][ref["written"]], ref["V"][ref["written"]])
    # the input state is left as it was
    assert full["written"][:58].all() and not full["written"][58:].any()
