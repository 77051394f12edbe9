"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a worked
example derived by hand (tests/golden), a closed form, an invariant the
definitions imply, a brute-force loop on tiny inputs, or a library routine in
a special case that reduces to it.  A planted-mistake test at the end shows
that the parity bar used by the GPU tests separates a correct result from the
plausible mistakes (mask off by one, wrong position, dropped LoRA term,
transposed head map).
"""

import math
import os

import numpy as np
import pytest
import torch

import oracle
import synthdata as sd
from tests._tol import o_within

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, rhs = (t.strip() for t in line.split("=", 1))
            nums = [float(t) for t in rhs.split()]
            vals.setdefault(key, []).append(nums)
    return {k: (v if len(v) > 1 else v[0]) for k, v in vals.items()}


# ----------------------------------------------------------------------------
# storage and integer work
# ----------------------------------------------------------------------------

def test_decode_bf16_known_patterns():
    bits = np.array([0x3F80, 0xC000, 0x3F00, 0x4049, 0x0000, 0x8000, 0x7F7F], np.uint16)
    want = [1.0, -2.0, 0.5, 3.140625, 0.0, -0.0, 3.3895313892515355e38]
    assert oracle.decode_bf16(bits).tolist() == want


def test_bf16_generator_round_trip_is_nearest_even():
    # the generator's rounding must land on the nearest bf16; ties go to the even pattern
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5e-3], np.float32)
    bits = sd.f32_to_bf16_bits(x)
    back = oracle.decode_bf16(bits)
    assert back[0] == 1.0
    assert back[1] == 1.0                  # tie between 1 and 1 + 2^-7 -> even (1.0)
    assert back[2] == 1.0 + 2 ** -6        # tie between 1+2^-7 and 1+2^-6 -> even (1+2^-6)
    assert back[3] == 1.0
    rng = np.random.default_rng(0)
    y = rng.standard_normal(100000).astype(np.float32)
    yb = oracle.decode_bf16(sd.f32_to_bf16_bits(y))
    # nearest: error at most half an ulp (2^-8 relative to the leading power of two)
    ulp = 2.0 ** (np.floor(np.log2(np.abs(y.astype(np.float64)))) - 7)
    assert np.all(np.abs(yb - y) <= ulp / 2 + 1e-30)


def test_page_counts():
    assert oracle.page_valid_counts(1, 16) == [1]
    assert oracle.page_valid_counts(16, 16) == [16]
    assert oracle.page_valid_counts(17, 16) == [16, 1]
    assert oracle.page_valid_counts(1024, 16) == [16] * 64
    with pytest.raises(ValueError):
        oracle.page_valid_counts(0, 16)


def test_golden_block_table():
    g = _golden("block_table_small.txt")
    lengths = [int(v) for v in g["lengths"]]
    reqs = [([int(v) for v in g["req0_ids"]], int(g["req0_cap"][0])),
            ([int(v) for v in g["req1_ids"]], int(g["req1_cap"][0]))]
    entries, cu = oracle.block_table(lengths, reqs, int(g["page_tokens"][0]))
    assert entries.tolist() == [[int(v) for v in e] for e in g["entry"]]
    assert cu.tolist() == [int(v) for v in g["cu_ctx"]]


def test_block_table_brute_force_rows():
    # every token of every artifact lands on exactly one row, in prompt order
    rng = np.random.default_rng(5)
    lengths = rng.integers(1, 70, size=9).tolist()
    reqs = [([int(a) for a in rng.integers(0, 9, size=int(n))], int(c))
            for n, c in zip(rng.integers(0, 6, size=5), rng.integers(0, 20, size=5))]
    entries, cu = oracle.block_table(lengths, reqs, 16)
    owner = {}
    for a, p, nv, r, dst in entries.tolist():
        for t in range(nv):
            owner[dst + t] = (r, a, 16 * p + t)
    for r, (ids, cap) in enumerate(reqs):
        row = int(cu[r])
        for a in ids:
            for t in range(lengths[a]):
                assert owner.pop(row) == (r, a, t)
                row += 1
        assert row + cap == cu[r + 1]
    assert not owner


def test_assemble_is_concatenation_bit_exact():
    rng = np.random.default_rng(1)
    lengths = [5, 17, 32, 1]
    n_layers, n_kv, d = 2, 2, 8
    ks = {a: rng.integers(0, 2 ** 16, size=(n_layers, L, n_kv, d), dtype=np.uint16) for a, L in enumerate(lengths)}
    vs = {a: rng.integers(0, 2 ** 16, size=(n_layers, L, n_kv, d), dtype=np.uint16) for a, L in enumerate(lengths)}
    reqs = [([2, 0, 3], 4), ([], 3), ([1, 1], 0)]   # empty request and a duplicated artifact
    cache, cu = oracle.assemble(ks, vs, reqs, n_kv, d)
    # per-token loop written independently of the vectorised copy
    for r, (ids, cap) in enumerate(reqs):
        row = int(cu[r])
        for a in ids:
            for t in range(lengths[a]):
                for l in range(n_layers):
                    for g in range(n_kv):
                        assert np.array_equal(cache[l, 0, g, row], ks[a][l, t, g])
                        assert np.array_equal(cache[l, 1, g, row], vs[a][l, t, g])
                row += 1
        for _ in range(cap):
            assert not cache[:, :, :, row].any()
            row += 1
    assert row == cache.shape[3]


# ----------------------------------------------------------------------------
# O3 projection
# ----------------------------------------------------------------------------

def test_golden_lora():
    g = _golden("lora_small.txt")
    x = np.array(g["x"]).reshape(1, 2)
    w = np.array(g["w"]).reshape(2, 2)
    a = np.array(g["a"]).reshape(1, 2)
    b = np.array(g["b"]).reshape(2, 1)
    out = oracle.qproj_lora(x, w, a, b, g["scale"][0])
    assert out.tolist() == [g["out"]]


def _rand(rng, *shape, std=1.0):
    return rng.standard_normal(shape) * std


def test_lora_zero_b_is_base_projection():
    # zero-initialised B: the update is zero (section 4; appendix A.5)
    rng = np.random.default_rng(2)
    x, w, a = _rand(rng, 7, 40), _rand(rng, 24, 40), _rand(rng, 4, 40)
    b = np.zeros((24, 4))
    assert np.array_equal(oracle.qproj_lora(x, w, a, b, 2.0), x @ w.T)
    assert np.array_equal(oracle.qproj_lora(x, w, None, None), x @ w.T)


def test_lora_merged_equals_unmerged():
    # deployment merge W <- W + (alpha/r) B A (appendix A.5) computes the same map
    rng = np.random.default_rng(3)
    x, w, a, b = _rand(rng, 9, 48), _rand(rng, 32, 48), _rand(rng, 8, 48), _rand(rng, 32, 8)
    s = 16 / 8
    merged = x @ (w + s * b @ a).T
    got = oracle.qproj_lora(x, w, a, b, s)
    assert np.max(np.abs(got - merged)) <= 1e-12 * np.max(np.abs(merged))


def test_lora_only_on_query_columns():
    # fused [Wq; Wk; Wv]: the low-rank term touches the query block only
    rng = np.random.default_rng(4)
    x, w, a, b = _rand(rng, 5, 16), _rand(rng, 40, 16), _rand(rng, 2, 16), _rand(rng, 24, 2)
    got = oracle.qproj_lora(x, w, a, b, 1.5, lora_cols=24)
    assert np.array_equal(got[:, 24:], x @ w[24:].T)
    assert np.allclose(got[:, :24], x @ (w[:24] + 1.5 * b @ a).T, rtol=0, atol=1e-12)


# ----------------------------------------------------------------------------
# O4 RMSNorm
# ----------------------------------------------------------------------------

def test_golden_rmsnorm():
    g = _golden("rmsnorm_small.txt")
    out = oracle.rms_norm_heads(np.array(g["u"]), np.array(g["gamma"]), g["eps"][0])
    assert np.allclose(out, g["out"], rtol=0, atol=1e-15)


def test_rmsnorm_unit_gamma_rms_and_scale_invariance():
    rng = np.random.default_rng(6)
    u = _rand(rng, 50, 4, 128)
    eps = 1e-6
    out = oracle.rms_norm_heads(u, np.ones(128), eps)
    m = np.mean(u * u, axis=-1)
    rms_out = np.sqrt(np.mean(out * out, axis=-1))
    assert np.allclose(rms_out, np.sqrt(m / (m + eps)), rtol=1e-13, atol=0)
    # scaling the input by c acts like dividing eps by c^2: norm(c u) = u / sqrt(m + eps / c^2)
    out2 = oracle.rms_norm_heads(1000.0 * u, np.ones(128), eps)
    assert np.max(np.abs(out2 - u / np.sqrt(m + eps / 1e6)[..., None])) < 1e-13
    # constant vector c: gamma * c / sqrt(c^2 + eps), elementwise gamma
    gam = rng.uniform(0.5, 1.5, 128)
    c = np.full((1, 128), -0.25)
    assert np.allclose(oracle.rms_norm_heads(c, gam, eps), gam * -0.25 / math.sqrt(0.0625 + eps), atol=1e-15)


# ----------------------------------------------------------------------------
# O5 RoPE
# ----------------------------------------------------------------------------

def test_golden_rope_unit_vectors():
    g = _golden("rope_unit.txt")
    e = np.zeros((3, 1, 128))
    e[0, 0, 32] = 1.0
    e[1, 0, 96] = 1.0
    e[2, 0, 0] = 1.0
    pos = np.array([1000, 1000, 3])
    out = oracle.rope(e, pos, 1e6)
    c1, s1, c3, s3 = g["cos1"][0], g["sin1"][0], g["cos3"][0], g["sin3"][0]
    want = np.zeros((3, 1, 128))
    want[0, 0, 32], want[0, 0, 96] = c1, s1
    want[1, 0, 32], want[1, 0, 96] = -s1, c1
    want[2, 0, 0], want[2, 0, 64] = c3, s3
    assert np.max(np.abs(out - want)) < 1e-12


def test_rope_equals_complex_rotation():
    # pairs (j, j + d/2) as complex numbers z_j = u_j + i u_{j+d/2}, multiplied by exp(i p w_j)
    rng = np.random.default_rng(7)
    u = _rand(rng, 6, 3, 128)
    pos = rng.integers(0, 40000, size=6)
    z = u[..., :64] + 1j * u[..., 64:]
    w = np.exp(-np.log(1e6) * np.arange(0, 128, 2) / 128.0)
    zr = z * np.exp(1j * pos[:, None, None] * w[None, None, :])
    want = np.concatenate([zr.real, zr.imag], axis=-1)
    assert np.max(np.abs(oracle.rope(u, pos, 1e6) - want)) < 1e-9


def test_rope_identity_norm_and_composition():
    rng = np.random.default_rng(8)
    u = _rand(rng, 5, 2, 128)
    assert np.array_equal(oracle.rope(u, np.zeros(5), 1e6), u)
    r = oracle.rope(u, np.array([1, 7, 100, 5000, 33000]), 1e6)
    pair_norm = lambda t: t[..., :64] ** 2 + t[..., 64:] ** 2
    assert np.allclose(pair_norm(r), pair_norm(u), rtol=1e-12)
    a, b = np.array([3, 11, 250, 4000, 20000]), np.array([5, 2, 900, 123, 13000])
    assert np.max(np.abs(oracle.rope(oracle.rope(u, a, 1e6), b, 1e6) - oracle.rope(u, a + b, 1e6))) < 1e-9


def test_rope_scores_depend_on_relative_position():
    rng = np.random.default_rng(9)
    q, k = _rand(rng, 1, 1, 128), _rand(rng, 1, 1, 128)
    def score(p, pk):
        return float(np.sum(oracle.rope(q, np.array([p]), 1e6) * oracle.rope(k, np.array([pk]), 1e6)))
    assert abs(score(700, 200) - score(500, 0)) < 1e-9
    assert abs(score(33000, 32999) - score(1, 0)) < 1e-9


# ----------------------------------------------------------------------------
# O6 attention
# ----------------------------------------------------------------------------

def test_golden_attention():
    g = _golden("attention_small.txt")
    q = np.array(g["q"]).reshape(2, 1, 4)
    k = np.array(g["k"]).reshape(4, 1, 4)
    v = np.array(g["v"]).reshape(4, 1, 4)
    o, lse = oracle.attention(q, k, v, int(g["art_len"][0]), return_lse=True)
    assert np.max(np.abs(o.reshape(2, 4) - np.array(g["o"]).reshape(2, 4))) < 1e-14
    assert np.max(np.abs(lse.reshape(2) - np.array(g["lse"]))) < 1e-14


def _brute_attention(q, k, v, art_len):
    """Row-by-row loop with math.exp; written without numpy reductions."""
    S, Hq, d = q.shape
    Hkv = k.shape[1]
    out = np.zeros_like(q)
    for i in range(S):
        for h in range(Hq):
            g = h // (Hq // Hkv)
            zs = []
            for j in range(art_len + i + 1):
                zs.append(sum(q[i, h, t] * k[j, g, t] for t in range(d)) / math.sqrt(d))
            m = max(zs)
            ws = [math.exp(z - m) for z in zs]
            tot = sum(ws)
            for t in range(d):
                out[i, h, t] = sum(w * v[j, g, t] for j, w in enumerate(ws)) / tot
    return out


@pytest.mark.parametrize("art_len,S,Hq,Hkv,d", [(0, 5, 4, 2, 8), (3, 4, 4, 2, 8), (7, 6, 4, 1, 8),
                                                   (5, 1, 2, 2, 4), (4, 3, 8, 2, 6)])
def test_attention_brute_force(art_len, S, Hq, Hkv, d):
    rng = np.random.default_rng(art_len * 100 + S)
    q, k, v = _rand(rng, S, Hq, d, std=2.0), _rand(rng, art_len + S, Hkv, d), _rand(rng, art_len + S, Hkv, d)
    got = oracle.attention(q, k, v, art_len)
    assert np.max(np.abs(got - _brute_attention(q, k, v, art_len))) <= 1e-12


def test_softmax_rows_sum_to_one_and_mask():
    rng = np.random.default_rng(10)
    S, L = 6, 9
    q, k = _rand(rng, S, 4, 8, std=3.0), _rand(rng, L + S, 2, 8)
    p = oracle.attention_probs(q, k, L)
    assert np.max(np.abs(p.sum(axis=-1) - 1.0)) <= 1e-12
    for i in range(S):
        assert np.all(p[i, :, L + i + 1:] == 0.0)       # future suffix keys carry no weight
        assert np.all(p[i, :, :L + i + 1] > 0.0)        # every cached key and the past are visible


def test_constant_and_one_hot_values():
    rng = np.random.default_rng(11)
    S, L = 4, 6
    q, k = _rand(rng, S, 4, 8), _rand(rng, L + S, 2, 8)
    v = np.ones((L + S, 2, 8)) * 0.375
    assert np.max(np.abs(oracle.attention(q, k, v, L) - 0.375)) <= 1e-15
    p = oracle.attention_probs(q, k, L)
    for j in (0, L - 1, L + 2):
        vj = np.zeros((L + S, 2, 8))
        vj[j, :, 0] = 1.0
        o = oracle.attention(q, k, vj, L)
        assert np.max(np.abs(o[:, :, 0] - p[:, :, j])) <= 1e-15


def test_gqa_equals_sdpa_with_repeated_kv_heads():
    # library routine: torch scaled_dot_product_attention (float64, CPU), explicit mask
    rng = np.random.default_rng(12)
    S, L, Hq, Hkv, d = 5, 11, 8, 2, 16
    q, k, v = _rand(rng, S, Hq, d), _rand(rng, L + S, Hkv, d), _rand(rng, L + S, Hkv, d)
    G = Hq // Hkv
    kr = np.repeat(k, G, axis=1)  # head h reads kv head h // G
    vr = np.repeat(v, G, axis=1)
    mask = np.arange(L + S)[None, :] <= (L + np.arange(S))[:, None]
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q).permute(1, 0, 2), torch.from_numpy(kr).permute(1, 0, 2),
        torch.from_numpy(vr).permute(1, 0, 2), attn_mask=torch.from_numpy(mask)).permute(1, 0, 2).numpy()
    assert np.max(np.abs(oracle.attention(q, k, v, L) - ref)) <= 1e-12


def test_no_artifacts_is_textbook_causal_attention():
    rng = np.random.default_rng(13)
    S, H, d = 9, 4, 8
    q, k, v = _rand(rng, S, H, d), _rand(rng, S, H, d), _rand(rng, S, H, d)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q).permute(1, 0, 2), torch.from_numpy(k).permute(1, 0, 2),
        torch.from_numpy(v).permute(1, 0, 2), is_causal=True).permute(1, 0, 2).numpy()
    assert np.max(np.abs(oracle.attention(q, k, v, 0) - ref)) <= 1e-12


def test_lse_matches_logsumexp():
    rng = np.random.default_rng(14)
    S, L = 3, 5
    q, k, v = _rand(rng, S, 2, 8), _rand(rng, L + S, 1, 8), _rand(rng, L + S, 1, 8)
    _, lse = oracle.attention(q, k, v, L, return_lse=True)
    for i in range(S):
        for h in range(2):
            z = [float(q[i, h] @ k[j, 0]) / math.sqrt(8) for j in range(L + i + 1)]
            m = max(z)
            assert abs(lse[i, h] - (m + math.log(sum(math.exp(t - m) for t in z)))) < 1e-12


def test_row_subset_matches_all_rows():
    rng = np.random.default_rng(15)
    S, L = 8, 13
    q, k, v = _rand(rng, S, 4, 8), _rand(rng, L + S, 2, 8), _rand(rng, L + S, 2, 8)
    full = oracle.attention(q, k, v, L)
    rows = np.array([0, 3, 7])
    assert np.array_equal(oracle.attention(q, k, v, L, rows=rows), full[rows])


# ----------------------------------------------------------------------------
# whole layer: PIC construction vs Full (eq. 2), permutation, position shift
# ----------------------------------------------------------------------------

def _tiny_layer(rng, H=32, Hq=4, Hkv=2, d=8, r=2):
    return dict(wq=_rand(rng, Hq * d, H, std=0.2), wk=_rand(rng, Hkv * d, H, std=0.2),
                wv=_rand(rng, Hkv * d, H, std=0.2), a=_rand(rng, r, H, std=0.2),
                b=_rand(rng, Hq * d, r, std=0.3), gamma_q=rng.uniform(0.5, 1.5, d),
                gamma_k=rng.uniform(0.5, 1.5, d))


GEOM = dict(n_q_heads=4, n_kv_heads=2, theta=1e4, eps=1e-6)


def _encode(xa, w, pos0):
    f = oracle.full_prefill(xa, w["wq"], w["wk"], w["wv"], w["gamma_q"], w["gamma_k"], pos0, **GEOM)
    return f["k_hat"], f["v"]


def test_single_artifact_at_offset_zero_equals_full_prefill():
    # one artifact at position 0 followed by the suffix: PIC and Full coincide in one layer
    rng = np.random.default_rng(16)
    w = _tiny_layer(rng)
    xa, xs = _rand(rng, 7, 32), _rand(rng, 5, 32)
    ka, va = _encode(xa, w, 0)
    sfx = oracle.suffix_layer(xs, w["wq"], w["wk"], w["wv"], w["a"], w["b"], 2.0, w["gamma_q"], w["gamma_k"],
                              ka, va, 7, **GEOM)
    full = oracle.full_prefill(np.concatenate([xa, xs]), w["wq"], w["wk"], w["wv"], w["gamma_q"], w["gamma_k"], 0,
                               a=w["a"], b=w["b"], scale=2.0, **GEOM)
    assert np.max(np.abs(sfx["o"] - full["o"][7:])) <= 1e-12
    assert np.max(np.abs(sfx["k_hat"] - full["k_hat"][7:])) <= 1e-12


def test_pic_pos_equals_full_prefill_in_one_layer():
    # artifacts encoded alone at their target offsets (appendix C.1, PIC-Pos): in a single
    # layer keys depend only on their own token and position, so this matches Full exactly
    rng = np.random.default_rng(17)
    w = _tiny_layer(rng)
    lens = [4, 9, 3]
    xs_art = [_rand(rng, L, 32) for L in lens]
    xs = _rand(rng, 6, 32)
    ks, vs, off = [], [], 0
    for xa in xs_art:
        ka, va = _encode(xa, w, off)
        ks.append(ka)
        vs.append(va)
        off += xa.shape[0]
    sfx = oracle.suffix_layer(xs, w["wq"], w["wk"], w["wv"], w["a"], w["b"], 1.0, w["gamma_q"], w["gamma_k"],
                              np.concatenate(ks), np.concatenate(vs), off, **GEOM)
    full = oracle.full_prefill(np.concatenate(xs_art + [xs]), w["wq"], w["wk"], w["wv"], w["gamma_q"],
                               w["gamma_k"], 0, a=w["a"], b=w["b"], scale=1.0, **GEOM)
    assert np.max(np.abs(sfx["o"] - full["o"][off:])) <= 1e-12
    # the PIC construction (local positions) differs from PIC-Pos once artifacts are off zero
    ks_pic = [_encode(xa, w, 0)[0] for xa in xs_art]
    pic = oracle.suffix_layer(xs, w["wq"], w["wk"], w["wv"], w["a"], w["b"], 1.0, w["gamma_q"], w["gamma_k"],
                              np.concatenate(ks_pic), np.concatenate(vs), off, **GEOM)
    assert np.max(np.abs(pic["o"] - sfx["o"])) > 1e-6


def test_artifact_order_does_not_change_output():
    # every cached key is visible and positions are baked into the keys, so the order of
    # the assembled artifacts does not matter to the suffix rows
    rng = np.random.default_rng(18)
    w = _tiny_layer(rng)
    arts = [(_rand(rng, L, 2, 8), _rand(rng, L, 2, 8)) for L in (5, 3, 8)]
    xs = _rand(rng, 4, 32)
    outs = []
    for order in ([0, 1, 2], [2, 0, 1], [1, 2, 0]):
        ka = np.concatenate([arts[i][0] for i in order])
        va = np.concatenate([arts[i][1] for i in order])
        outs.append(oracle.suffix_layer(xs, w["wq"], w["wk"], w["wv"], w["a"], w["b"], 1.0, w["gamma_q"],
                                        w["gamma_k"], ka, va, 16, **GEOM)["o"])
    assert max(np.max(np.abs(o - outs[0])) for o in outs) <= 1e-12


def test_full_prefill_is_invariant_to_a_global_position_shift():
    rng = np.random.default_rng(19)
    w = _tiny_layer(rng)
    x = _rand(rng, 10, 32)
    o0 = oracle.full_prefill(x, w["wq"], w["wk"], w["wv"], w["gamma_q"], w["gamma_k"], 0, **GEOM)["o"]
    o1 = oracle.full_prefill(x, w["wq"], w["wk"], w["wv"], w["gamma_q"], w["gamma_k"], 12345, **GEOM)["o"]
    assert np.max(np.abs(o0 - o1)) <= 1e-9


# ----------------------------------------------------------------------------
# the parity bar separates plausible mistakes (planted in the oracle, on the CPU)
# ----------------------------------------------------------------------------

def _c1_layer(gamma="uniform", b_std=None):
    wl = sd.make_workload("c1", gamma=gamma, **({} if b_std is None else {"b_std": b_std}))
    s = wl.shape
    w = {k: oracle.decode_bf16(v) for k, v in sd.layer_weights(wl, 0).items()}
    kv = [sd.artifact_kv(wl, a, 0) for a in wl.requests[0].artifact_ids]
    ka = np.concatenate([oracle.decode_bf16(k) for k, _ in kv])
    va = np.concatenate([oracle.decode_bf16(v) for _, v in kv])
    x = oracle.decode_bf16(sd.suffix_hidden(wl, 0, 0))
    return wl, s, w, ka, va, x


def _run(wl, s, w, ka, va, x, pos0=None, scale=None):
    return oracle.suffix_layer(x, w["wq"], w["wk"], w["wv"], w["a"], w["b"],
                               wl.scale if scale is None else scale, w["gamma_q"], w["gamma_k"], ka, va,
                               wl.pos0(wl.requests[0]) if pos0 is None else pos0, s.n_q_heads, s.n_kv_heads,
                               s.rope_theta, s.rms_eps)


def test_parity_bar_catches_planted_mistakes():
    # C1 shapes with gamma ~ U(0.5, 1.5).  (A sharper gamma_q = 8 cannot be a parity case:
    # bf16 storage of the projected q alone moves O beyond the absolute mean bar there.)
    wl, s, w, ka, va, x = _c1_layer("uniform")
    ref = _run(wl, s, w, ka, va, x)
    L = ka.shape[0]
    keys = np.concatenate([ka, ref["k_hat"]])
    vals = np.concatenate([va, ref["v"]])
    # mask off by one: each suffix row also sees its next token
    leak = oracle.attention(ref["q_hat"], np.concatenate([keys, keys[-1:]]),
                            np.concatenate([vals, vals[-1:]]), L + 1)
    assert not o_within(leak, ref["o"])
    # suffix positions off by one
    assert not o_within(_run(wl, s, w, ka, va, x, pos0=L + 1)["o"], ref["o"])
    # head map h % Hkv instead of h // G
    qh = ref["q_hat"]
    perm = np.array([(h % 8) * 4 + h // 8 for h in range(32)])
    wrong = oracle.attention(qh[:, perm, :], keys, vals, L)[:, np.argsort(perm), :]
    assert not o_within(wrong, ref["o"])
    # the bar itself accepts bf16 storage of every intermediate of the pipeline
    # (projected q/k/v, q_hat, k_hat and O)
    rnd = lambda t: oracle.decode_bf16(sd.f32_to_bf16_bits(np.asarray(t, np.float32)))
    pos = L + np.arange(x.shape[0])
    qh = rnd(oracle.rope(oracle.rms_norm_heads(rnd(ref["q"]), w["gamma_q"], s.rms_eps), pos, s.rope_theta))
    kh = rnd(oracle.rope(oracle.rms_norm_heads(rnd(ref["k"]), w["gamma_k"], s.rms_eps), pos, s.rope_theta))
    o_b = oracle.attention(qh, np.concatenate([ka, kh]), np.concatenate([va, rnd(ref["v"])]), L)
    assert o_within(rnd(o_b), ref["o"])


def test_lora_delta_case_catches_a_dropped_update():
    # with the paper-scale B ~ N(0, 0.01) the low-rank term is small; the dedicated delta
    # case (B ~ N(0, 1)) makes a dropped or mis-scaled update fail the bar
    wl, s, w, ka, va, x = _c1_layer("uniform", b_std=1.0)
    ref = _run(wl, s, w, ka, va, x)
    assert not o_within(_run(wl, s, w, ka, va, x, scale=0.0)["o"], ref["o"])
    assert not o_within(_run(wl, s, w, ka, va, x, scale=wl.scale * 0.5)["o"], ref["o"])


# ----------------------------------------------------------------------------
# the decoder layer around the path
# ----------------------------------------------------------------------------

def test_silu_identity_limits_and_minimum():
    z = np.linspace(-30.0, 30.0, 6001)
    # silu(z) - silu(-z) = z, since sigma(-z) = 1 - sigma(z)
    assert np.max(np.abs(oracle.silu(z) - oracle.silu(-z) - z)) <= 1e-12
    assert oracle.silu(np.array([0.0]))[0] == 0.0
    assert abs(oracle.silu(np.array([60.0]))[0] - 60.0) < 1e-20 * 60 + 1e-24
    assert oracle.silu(np.array([-800.0]))[0] == 0.0          # e^800 overflows: the limit, no NaN
    # the minimum sits at x* with 1 + e^x* = -x* (derivative zero), where silu(x*) = x* + 1;
    # solve that fixed point by bisection and compare with a fine grid search of the oracle
    lo, hi = -2.0, -1.0
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if 1.0 + math.exp(mid) + mid > 0.0:
            hi = mid
        else:
            lo = mid
    x_star = 0.5 * (lo + hi)
    grid = np.linspace(-1.5, -1.0, 500001)
    vals = oracle.silu(grid)
    i = int(np.argmin(vals))
    assert abs(grid[i] - x_star) <= 2e-6
    assert abs(vals[i] - (x_star + 1.0)) <= 1e-11


def test_swiglu_brute_force():
    rng = np.random.default_rng(21)
    x, wg, wu = rng.standard_normal((3, 4)), rng.standard_normal((5, 4)), rng.standard_normal((5, 4))
    got = oracle.swiglu(x, wg, wu)
    for t in range(3):
        for j in range(5):
            g = sum(x[t, k] * wg[j, k] for k in range(4))
            u = sum(x[t, k] * wu[j, k] for k in range(4))
            assert abs(got[t, j] - g / (1.0 + math.exp(-g)) * u) <= 1e-12


def _tiny_layer_weights(rng, H=256, I=128, Hq=32, Hkv=8, d=128):
    f = lambda *s, std=1.0: rng.standard_normal(s) * std
    return {"wq": f(Hq * d, H, std=0.02), "wk": f(Hkv * d, H, std=0.02), "wv": f(Hkv * d, H, std=0.02),
            "a": None, "b": None, "gamma_q": 1.0 + 0.1 * f(d), "gamma_k": 1.0 + 0.1 * f(d),
            "gamma_in": 1.0 + 0.1 * f(H), "wo": f(H, Hq * d, std=0.02), "gamma_post": 1.0 + 0.1 * f(H),
            "w_gate": f(I, H, std=0.05), "w_up": f(I, H, std=0.05), "w_down": f(H, I, std=0.05)}


def test_decoder_layer_residual_identities():
    rng = np.random.default_rng(22)
    w = _tiny_layer_weights(rng)
    h = rng.standard_normal((5, 256))
    k_art, v_art = rng.standard_normal((7, 8, 128)), rng.standard_normal((7, 8, 128))
    args = (k_art, v_art, 7, 32, 8, 1e6, 1e-6)
    # no attention output projection and no MLP output: the residual stream passes unchanged
    w0 = dict(w, wo=np.zeros_like(w["wo"]), w_down=np.zeros_like(w["w_down"]))
    assert np.array_equal(oracle.decoder_layer(h, w0, *args)["h"], h)
    # a zero gate makes silu(0) = 0: the MLP adds nothing to h1
    wg0 = dict(w, w_gate=np.zeros_like(w["w_gate"]))
    r = oracle.decoder_layer(h, wg0, *args)
    assert np.array_equal(r["h"], r["h1"]) and not r["mlp"].any()
    # the attention part only enters through o W_o^T: scaling W_o by 2 doubles h1 - h
    r1 = oracle.decoder_layer(h, w, *args)
    r2 = oracle.decoder_layer(h, dict(w, wo=2.0 * w["wo"]), *args)
    assert np.max(np.abs((r2["h1"] - h) - 2.0 * (r1["h1"] - h))) <= 1e-12


def test_first_token_brute_force_and_ties():
    rng = np.random.default_rng(23)
    H, V = 16, 40
    h = rng.standard_normal((3, H))
    g = 1.0 + 0.1 * rng.standard_normal(H)
    w = rng.standard_normal((V, H))
    ids, logits = oracle.first_token(h, g, w, 1e-6)
    for r in range(3):
        x = [g[k] * h[r, k] / math.sqrt(sum(v * v for v in h[r]) / H + 1e-6) for k in range(H)]
        lg = [sum(x[k] * w[v, k] for k in range(H)) for v in range(V)]
        best = max(range(V), key=lambda v: (lg[v], -v))
        assert ids[r] == best and abs(logits[r, best] - lg[best]) <= 1e-12
    # two identical vocabulary rows at the top: the smaller index wins
    w2 = w.copy()
    top = int(ids[0])
    w2[V - 1] = w2[top]
    ids2, _ = oracle.first_token(h[:1], g, w2, 1e-6)
    assert ids2[0] == min(top, V - 1)


# ----------------------------------------------------------------------------
# interleaved online spans
# ----------------------------------------------------------------------------

def test_block_table_segments_worked_example():
    # prompt of request 0: 3 online | artifact 0 (20 tokens: pages of 16 and 4) |
    # 2 online | artifact 1 (5) | 4 online; request 1: artifact 1 alone.
    # Offsets by hand: art0 at 3 (rows 3..18, 19..22), span at 23, art1 at 25,
    # span at 30; request 0 spans 34 rows, request 1 rows 34..38.
    e, cu, sp = oracle.block_table_segments([20, 5], [[-3, 0, -2, 1, -4], [1]], 16)
    assert e.tolist() == [[0, 0, 16, 0, 3], [0, 1, 4, 0, 19], [1, 0, 5, 0, 25], [1, 0, 5, 1, 34]]
    assert cu.tolist() == [0, 34, 39]
    assert sp.tolist() == [[0, 0, 3], [0, 23, 2], [0, 30, 4]]


def test_block_table_segments_trailing_span_is_the_suffix_layout():
    lengths = [17, 40, 1, 16]
    reqs = [([1, 0, 3], 5), ([], 3), ([2, 2, 1], 0)]
    segs = [ids + ([-cap] if cap else []) for ids, cap in reqs]
    e, cu, sp = oracle.block_table_segments(lengths, segs, 16)
    e2, cu2 = oracle.block_table(lengths, reqs, 16)
    assert np.array_equal(e, e2) and np.array_equal(cu, cu2)
    assert sp.tolist() == [[0, 73, 5], [1, 0, 3]]


def _tiny_interleaved(seed, segments, lengths, H=16, Hq=4, Hkv=2, d=8):
    rng = np.random.default_rng(seed)
    n_online = sum(-s for s in segments if s < 0)
    w = {"wq": rng.standard_normal((Hq * d, H)) * 0.3, "wk": rng.standard_normal((Hkv * d, H)) * 0.3,
         "wv": rng.standard_normal((Hkv * d, H)), "a": rng.standard_normal((2, H)) * 0.3,
         "b": rng.standard_normal((Hq * d, 2)) * 0.3, "gq": rng.uniform(0.5, 1.5, d), "gk": rng.uniform(0.5, 1.5, d)}
    art_k = {i: rng.standard_normal((L, Hkv, d)) for i, L in enumerate(lengths)}
    art_v = {i: rng.standard_normal((L, Hkv, d)) for i, L in enumerate(lengths)}
    x = rng.standard_normal((n_online, H))
    return w, art_k, art_v, x, (Hq, Hkv)


def _run_interleaved(segments, w, art_k, art_v, x, heads, scale=0.7):
    return oracle.interleaved_layer(segments, x, w["wq"], w["wk"], w["wv"], w["a"], w["b"], scale, w["gq"], w["gk"],
                                    art_k, art_v, heads[0], heads[1], 1e4, 1e-6)


def test_interleaved_trailing_span_equals_suffix_layer():
    segs = [1, 0, -6]
    w, ak, av, x, heads = _tiny_interleaved(61, segs, [5, 9])
    got = _run_interleaved(segs, w, ak, av, x, heads)
    ref = oracle.suffix_layer(x, w["wq"], w["wk"], w["wv"], w["a"], w["b"], 0.7, w["gq"], w["gk"],
                              np.concatenate([ak[1], ak[0]]), np.concatenate([av[1], av[0]]), 14, heads[0],
                              heads[1], 1e4, 1e-6)
    assert np.max(np.abs(got["o"] - ref["o"])) <= 1e-12
    assert got["pos"].tolist() == list(range(14, 20))


def test_interleaved_single_span_without_artifacts_equals_full_prefill():
    w, ak, av, x, heads = _tiny_interleaved(62, [-7], [])
    got = _run_interleaved([-7], w, ak, av, x, heads)
    ref = oracle.full_prefill(x, w["wq"], w["wk"], w["wv"], w["gq"], w["gk"], 0, heads[0], heads[1], 1e4, 1e-6,
                              a=w["a"], b=w["b"], scale=0.7)
    assert np.max(np.abs(got["o"] - ref["o"])) <= 1e-12


def test_interleaved_split_span_is_invariant():
    w, ak, av, x, heads = _tiny_interleaved(63, [-3, 0, -5], [6])
    one = _run_interleaved([-3, 0, -5], w, ak, av, x, heads)
    two = _run_interleaved([-3, 0, -2, -3], w, ak, av, x, heads)
    assert np.max(np.abs(one["o"] - two["o"])) <= 1e-12


def test_interleaved_brute_force_mask_and_order():
    # the test lays the prompt out itself (its own walk over the segments) and
    # runs a per-row math.exp softmax over the keys each online token may see
    segs = [-2, 1, -3, 0, 0, -1]
    lengths = [3, 4]
    w, ak, av, x, heads = _tiny_interleaved(64, segs, lengths)
    out = _run_interleaved(segs, w, ak, av, x, heads)
    Hq, Hkv = heads
    G, d = Hq // Hkv, 8
    keys, vals, qpos = [], [], []
    t = 0
    for s in segs:
        if s >= 0:
            for i in range(lengths[s]):
                keys.append(ak[s][i])
                vals.append(av[s][i])
        else:
            for _ in range(-s):
                qpos.append(len(keys))
                keys.append(out["k_hat"][t])
                vals.append(out["v"][t])
                t += 1
    for r, p in enumerate(qpos):
        for h in range(Hq):
            g = h // G
            sc = [sum(out["q_hat"][r, h, j] * keys[kk][g, j] for j in range(d)) / math.sqrt(d) for kk in range(p + 1)]
            mx = max(sc)
            e = [math.exp(z - mx) for z in sc]
            den = sum(e)
            want = [sum(e[kk] * vals[kk][g, j] for kk in range(p + 1)) / den for j in range(d)]
            assert np.max(np.abs(out["o"][r, h] - np.array(want))) <= 1e-12


def test_interleaved_causality_and_leading_token():
    segs = [-4, 0, -3]
    w, ak, av, x, heads = _tiny_interleaved(65, segs, [5])
    base = _run_interleaved(segs, w, ak, av, x, heads)
    av2 = {0: av[0] + 1.0}
    moved = _run_interleaved(segs, w, ak, av2, x, heads)
    # the artifact sits after the first span: that span cannot see it, the last one does
    assert np.array_equal(base["o"][:4], moved["o"][:4])
    assert np.max(np.abs(base["o"][4:] - moved["o"][4:])) > 1e-3
    # the first online token sees only its own key: O = its value (GQA repeat)
    G = heads[0] // heads[1]
    assert np.max(np.abs(base["o"][0] - np.repeat(base["v"][0], G, axis=0))) <= 1e-12


def test_merge_lora_equals_the_unmerged_projection():
    # merged deployment (W_Q + s B A) against the adapter applied on the fly,
    # and the k/v rows untouched
    rng = np.random.default_rng(91)
    x, w = rng.standard_normal((5, 24)), rng.standard_normal((40, 24))
    a, b = rng.standard_normal((3, 24)), rng.standard_normal((32, 3))
    wm = oracle.merge_lora(w, a, b, 0.37, 32)
    assert np.array_equal(wm[32:], w[32:])
    got = oracle.qproj_lora(x, wm)
    want = oracle.qproj_lora(x, w, a, b, 0.37, 32)
    assert np.max(np.abs(got - want)) <= 1e-12
    # element (n, k) of the update by a plain loop
    n, k = 7, 11
    assert abs(wm[n, k] - w[n, k] - 0.37 * sum(b[n, j] * a[j, k] for j in range(3))) <= 1e-14
