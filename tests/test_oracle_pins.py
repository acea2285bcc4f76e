"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these re-type the oracle's own formula: each compares it with a library routine
on a special case the visibility rule reduces to, a closed form, an invariant, or brute
force over explicit predicates written here (Avatar V §1 contributions, §2.1, §4.3, §8).
"""
import math

import numpy as np
import pytest
import torch

import oracle
from sra_inputs import SampleGeom

RNG = np.random.default_rng(1234)


def rand_inputs(samples, H, d, rng=None, dtype=np.float64, grads=False):
    rng = RNG if rng is None else rng
    G = sum(s.n_gen for s in samples)
    R = sum(s.n_ref for s in samples)
    names = ["q_gen", "k_gen", "v_gen", "q_ref", "k_ref", "v_ref"]
    if grads:
        names += ["do_gen", "do_ref"]
    return {n: rng.standard_normal(((G if n.endswith("gen") else R), H, d)).astype(dtype) for n in names}


# --------------------------------------------------------------------- predicates (independent)
def ref_token_ok(geom, j):
    """Reference token j takes part: its frame is valid and, with a token mask, so is it."""
    F = geom.ref_h * geom.ref_w
    if geom.frame_valid is not None and not geom.frame_valid[j // F]:
        return False
    tv = getattr(geom, "ref_token_valid", None)
    return tv is None or bool(tv[j])


def pred_visible(geom, qi, ki):
    """Visibility of one (query, key) pair written as predicates, [gen ; ref] indexing."""
    G = geom.gen_frames * geom.gen_h * geom.gen_w
    F = geom.ref_h * geom.ref_w
    q_is_gen, k_is_gen = qi < G, ki < G
    if q_is_gen and k_is_gen:
        w = getattr(geom, "gen_window", None)
        if w is None:
            return True
        fg = geom.gen_h * geom.gen_w
        return abs(qi // fg - ki // fg) <= w
    if q_is_gen:
        return ref_token_ok(geom, ki - G)
    if k_is_gen:
        return False
    fq, fk = (qi - G) // F, (ki - G) // F
    return (ref_token_ok(geom, qi - G) and ref_token_ok(geom, ki - G)
            and (fq // geom.group_frames) == (fk // geom.group_frames))


def visible_count_closed_form(geom, qi):
    G = geom.gen_frames * geom.gen_h * geom.gen_w
    F = geom.ref_h * geom.ref_w
    R = geom.ref_frames * F
    n_valid = sum(ref_token_ok(geom, j) for j in range(R))
    if qi < G:
        w = getattr(geom, "gen_window", None)
        if w is None:
            return G + n_valid
        t, T = qi // (geom.gen_h * geom.gen_w), geom.gen_frames
        return (min(T - 1, t + w) - max(0, t - w) + 1) * geom.gen_h * geom.gen_w + n_valid
    j = qi - G
    if not ref_token_ok(geom, j):
        return 0
    g = geom.group_frames
    lo, hi = (j // F) // g * g * F, min(R, ((j // F) // g + 1) * g * F)
    return sum(ref_token_ok(geom, i) for i in range(lo, hi))


def torch_sdpa64(q, k, v, scale):
    """Dense softmax attention via torch's library routine (float64, CPU). q [n,d], k/v [m,d]."""
    qt, kt, vt = (torch.from_numpy(np.ascontiguousarray(a))[None, None] for a in (q, k, v))
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=scale)[0, 0].numpy()
    lse = torch.logsumexp(qt[0, 0] @ kt[0, 0].T * scale, dim=-1).numpy()
    return o, lse


GEOMS = [
    SampleGeom(2, 3, 5, 4, 3, 4),                                  # F = 12, all valid
    SampleGeom(3, 2, 4, 5, 2, 5, group_frames=1, frame_valid=[1, 0, 1, 1, 0]),
    SampleGeom(1, 4, 4, 6, 3, 3, group_frames=2, frame_valid=[1, 1, 0, 1, 1, 1]),
    SampleGeom(2, 2, 2, 3, 2, 2, group_frames=3),
]


# --------------------------------------------------------------------- special cases = library
@pytest.mark.parametrize("geom", GEOMS)
def test_gen_rows_equal_dense_attention_over_gen_and_valid_ref(geom):
    H, d = 2, 8
    x = rand_inputs([geom], H, d)
    o_gen, _, lse_gen, _ = oracle.sra_forward(x, [geom])
    F = geom.ref_h * geom.ref_w
    valid = np.ones(geom.ref_frames, bool) if geom.frame_valid is None else np.asarray(geom.frame_valid, bool)
    keep = np.repeat(valid, F)
    for h in range(H):
        k = np.concatenate([x["k_gen"][:, h], x["k_ref"][keep, h]])
        v = np.concatenate([x["v_gen"][:, h], x["v_ref"][keep, h]])
        o, lse = torch_sdpa64(x["q_gen"][:, h], k, v, 1 / math.sqrt(d))
        np.testing.assert_allclose(o_gen[:, h], o, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(lse_gen[h], lse, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("geom", GEOMS)
def test_ref_rows_equal_per_group_dense_attention(geom):
    H, d = 2, 8
    x = rand_inputs([geom], H, d)
    _, o_ref, _, lse_ref = oracle.sra_forward(x, [geom])
    F = geom.ref_h * geom.ref_w
    g = geom.group_frames
    valid = np.ones(geom.ref_frames, bool) if geom.frame_valid is None else np.asarray(geom.frame_valid, bool)
    for h in range(H):
        for g0 in range(0, geom.ref_frames, g):
            frames = [f for f in range(g0, min(g0 + g, geom.ref_frames)) if valid[f]]
            idx = np.concatenate([np.arange(f * F, (f + 1) * F) for f in frames]) if frames else np.zeros(0, int)
            if idx.size:
                o, lse = torch_sdpa64(x["q_ref"][idx, h], x["k_ref"][idx, h], x["v_ref"][idx, h], 1 / math.sqrt(d))
                np.testing.assert_allclose(o_ref[idx, h], o, rtol=1e-12, atol=1e-12)
                np.testing.assert_allclose(lse_ref[h, idx], lse, rtol=1e-12, atol=1e-12)
        for f in range(geom.ref_frames):
            if not valid[f]:
                assert np.all(o_ref[f * F:(f + 1) * F, h] == 0)
                assert np.all(np.isneginf(lse_ref[h, f * F:(f + 1) * F]))


def test_whole_reference_group_is_dense_ref_self_attention():
    geom = SampleGeom(2, 2, 3, 4, 2, 3, group_frames=4)
    x = rand_inputs([geom], 1, 8)
    _, o_ref, _, lse_ref = oracle.sra_forward(x, [geom])
    o, lse = torch_sdpa64(x["q_ref"][:, 0], x["k_ref"][:, 0], x["v_ref"][:, 0], 1 / math.sqrt(8))
    np.testing.assert_allclose(o_ref[:, 0], o, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse_ref[0], lse, rtol=1e-12, atol=1e-12)


def test_no_reference_is_plain_self_attention():
    geom = SampleGeom(3, 4, 4, 0, 4, 4)
    x = rand_inputs([geom], 2, 16)
    o_gen, o_ref, lse_gen, _ = oracle.sra_forward(x, [geom])
    assert o_ref.shape[0] == 0
    for h in range(2):
        o, lse = torch_sdpa64(x["q_gen"][:, h], x["k_gen"][:, h], x["v_gen"][:, h], 1 / math.sqrt(16))
        np.testing.assert_allclose(o_gen[:, h], o, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(lse_gen[h], lse, rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------------- invariants / closed forms
@pytest.mark.parametrize("geom", GEOMS)
def test_rows_sum_to_one(geom):
    x = rand_inputs([geom], 2, 8)
    x["v_gen"][:] = 1.0
    x["v_ref"][:] = 1.0
    o_gen, o_ref, _, lse_ref = oracle.sra_forward(x, [geom])
    np.testing.assert_allclose(o_gen, 1.0, rtol=0, atol=1e-13)
    live = np.isfinite(lse_ref[0])
    np.testing.assert_allclose(o_ref[live], 1.0, rtol=0, atol=1e-13)


@pytest.mark.parametrize("geom", GEOMS)
def test_zero_keys_give_log_visible_count(geom):
    """K = 0 makes every visible logit 0, so LSE_q = ln |vis(q)| exactly."""
    x = rand_inputs([geom], 1, 8)
    x["k_gen"][:] = 0.0
    x["k_ref"][:] = 0.0
    _, _, lse_gen, lse_ref = oracle.sra_forward(x, [geom])
    G = geom.n_gen
    lse = np.concatenate([lse_gen[0], lse_ref[0]])
    for qi in range(G + geom.n_ref):
        n = visible_count_closed_form(geom, qi)
        if n == 0:
            assert np.isneginf(lse[qi])
        else:
            assert abs(lse[qi] - math.log(n)) < 1e-12
            assert round(math.exp(lse[qi])) == n


@pytest.mark.parametrize("geom", [SampleGeom(1, 2, 3, 3, 2, 2, frame_valid=[1, 0, 1]),
                                  SampleGeom(2, 2, 2, 4, 2, 2, group_frames=2, frame_valid=[1, 1, 0, 1]),
                                  SampleGeom(1, 3, 3, 2, 2, 3, group_frames=2)])
def test_one_hot_values_recover_the_mask(geom):
    """K = 0 and V = one-hot per key: O[q, c] = 1/|vis(q)| exactly where key c is visible."""
    n = geom.n_gen + geom.n_ref
    d = n
    x = rand_inputs([geom], 1, d)
    x["k_gen"][:] = 0.0
    x["k_ref"][:] = 0.0
    eye = np.eye(n)
    x["v_gen"][:, 0] = eye[:geom.n_gen]
    x["v_ref"][:, 0] = eye[geom.n_gen:]
    o_gen, o_ref, _, _ = oracle.sra_forward(x, [geom])
    O = np.concatenate([o_gen[:, 0], o_ref[:, 0]])
    for qi in range(n):
        cnt = visible_count_closed_form(geom, qi)
        for ki in range(n):
            want = (1.0 / cnt) if pred_visible(geom, qi, ki) else 0.0
            assert abs(O[qi, ki] - want) < 1e-14, (qi, ki)


def test_mask_equals_predicates_and_pair_counts_close():
    for geom in GEOMS + [SampleGeom(2, 3, 3, 7, 2, 2, group_frames=3, frame_valid=[0, 1, 1, 0, 1, 1, 1])] + WINDOW_GEOMS:
        M = oracle.visibility_mask(geom)
        n = geom.n_gen + geom.n_ref
        P = np.array([[pred_visible(geom, i, j) for j in range(n)] for i in range(n)])
        assert np.array_equal(M, P)
        gp, rp = oracle.pair_counts([geom], block_rows=5)
        G = geom.n_gen
        assert gp + rp == int(P.sum())
        assert gp == sum(visible_count_closed_form(geom, q) for q in range(G))
        assert rp == sum(visible_count_closed_form(geom, q) for q in range(G, n))


def test_linear_pair_law_at_sweep_shape():
    """pairs(R) = G (G + R) + R F at group 1: slope G + F per ref token, intercept G^2."""
    G, F = 32760, 1560
    for n in (4, 16):
        gp, rp = oracle.pair_counts([SampleGeom(21, 30, 52, n, 30, 52)], block_rows=8192)
        R = n * F
        assert gp + rp == G * (G + R) + R * F
    assert G + F == 34320 and G * G == 1073217600


def test_gen_permutation_invariance():
    geom = GEOMS[1]
    x = rand_inputs([geom], 2, 8)
    o_gen, o_ref, lse_gen, lse_ref = oracle.sra_forward(x, [geom])
    perm = RNG.permutation(geom.n_gen)
    y = dict(x)
    for n in ("q_gen", "k_gen", "v_gen"):
        y[n] = x[n][perm]
    p_gen, p_ref, plg, plr = oracle.sra_forward(y, [geom])
    np.testing.assert_allclose(p_gen, o_gen[perm], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(plg, lse_gen[:, perm], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(p_ref, o_ref, rtol=1e-12, atol=1e-13)


def test_within_frame_permutation_invariance():
    geom = SampleGeom(2, 2, 3, 3, 3, 4, group_frames=1)
    x = rand_inputs([geom], 1, 8)
    o_gen, o_ref, _, lse_ref = oracle.sra_forward(x, [geom])
    F = 12
    perm = np.concatenate([f * F + RNG.permutation(F) for f in range(3)])
    y = dict(x)
    for n in ("q_ref", "k_ref", "v_ref"):
        y[n] = x[n][perm]
    p_gen, p_ref, _, plr = oracle.sra_forward(y, [geom])
    np.testing.assert_allclose(p_gen, o_gen, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(p_ref, o_ref[perm], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(plr, lse_ref[:, perm], rtol=1e-12, atol=1e-13)


def test_cross_frame_permutation_changes_ref_rows():
    """Moving a reference token to another frame must change reference outputs (groups matter)."""
    geom = SampleGeom(1, 2, 2, 2, 2, 2)
    x = rand_inputs([geom], 1, 4)
    _, o_ref, _, _ = oracle.sra_forward(x, [geom])
    y = dict(x)
    perm = np.array([0, 1, 2, 4, 3, 5, 6, 7])
    for n in ("q_ref", "k_ref", "v_ref"):
        y[n] = x[n][perm]
    _, p_ref, _, _ = oracle.sra_forward(y, [geom])
    assert not np.allclose(p_ref, o_ref[perm])


@pytest.mark.parametrize("geom", GEOMS)
def test_asymmetry_gen_inputs_never_reach_reference_outputs(geom):
    x = rand_inputs([geom], 2, 8, grads=True)
    _, o_ref, _, lse_ref = oracle.sra_forward(x, [geom])
    y = dict(x)
    for n in ("q_gen", "k_gen", "v_gen"):
        y[n] = RNG.standard_normal(x[n].shape)
    _, p_ref, _, plr = oracle.sra_forward(y, [geom])
    assert np.array_equal(p_ref, o_ref) and np.array_equal(plr, lse_ref)
    # backward: with dO_gen = 0 every gen gradient is exactly 0 ...
    z = dict(x)
    z["do_gen"] = np.zeros_like(x["do_gen"])
    g = oracle.sra_backward(z, [geom])
    for n in ("dq_gen", "dk_gen", "dv_gen"):
        assert np.all(g[n] == 0)
    # ... and the ref gradients equal those of per-group reference-only attention (torch autograd)
    F, gf = geom.ref_h * geom.ref_w, geom.group_frames
    valid = np.ones(geom.ref_frames, bool) if geom.frame_valid is None else np.asarray(geom.frame_valid, bool)
    for h in range(2):
        for g0 in range(0, geom.ref_frames, gf):
            frames = [f for f in range(g0, min(g0 + gf, geom.ref_frames)) if valid[f]]
            if not frames:
                continue
            idx = np.concatenate([np.arange(f * F, (f + 1) * F) for f in frames])
            q, k, v = (torch.tensor(x[n][idx, h], requires_grad=True) for n in ("q_ref", "k_ref", "v_ref"))
            o = torch.nn.functional.scaled_dot_product_attention(q[None], k[None], v[None], scale=1 / math.sqrt(8))[0]
            o.backward(torch.tensor(x["do_ref"][idx, h]))
            np.testing.assert_allclose(g["dq_ref"][idx, h], q.grad.numpy(), rtol=1e-10, atol=1e-12)
            np.testing.assert_allclose(g["dk_ref"][idx, h], k.grad.numpy(), rtol=1e-10, atol=1e-12)
            np.testing.assert_allclose(g["dv_ref"][idx, h], v.grad.numpy(), rtol=1e-10, atol=1e-12)


# --------------------------------------------------------------------- brute force
@pytest.mark.parametrize("g,w", [(1, None), (2, None), (3, None), (1, 0), (2, 1)])
def test_brute_force_quadruple_loop(g, w):
    geom = SampleGeom(3, 2, 2, 3, 2, 2, group_frames=g, frame_valid=[1, 0, 1], gen_window=w)
    H, d = 2, 4
    x = rand_inputs([geom], H, d)
    o_gen, o_ref, lse_gen, lse_ref = oracle.sra_forward(x, [geom])
    G, n = geom.n_gen, geom.n_gen + geom.n_ref
    Q = np.concatenate([x["q_gen"], x["q_ref"]])
    K = np.concatenate([x["k_gen"], x["k_ref"]])
    V = np.concatenate([x["v_gen"], x["v_ref"]])
    O = np.concatenate([o_gen, o_ref])
    L = np.concatenate([lse_gen, lse_ref], axis=1)
    sc = 1 / math.sqrt(d)
    for h in range(H):
        for qi in range(n):
            logits = []
            for ki in range(n):
                if pred_visible(geom, qi, ki):
                    s = 0.0
                    for c in range(d):
                        s += Q[qi, h, c] * K[ki, h, c]
                    logits.append((ki, s * sc))
            if not logits:
                assert np.all(O[qi, h] == 0) and np.isneginf(L[h, qi])
                continue
            mx = max(s for _, s in logits)
            den = sum(math.exp(s - mx) for _, s in logits)
            for c in range(d):
                num = sum(math.exp(s - mx) * V[ki, h, c] for ki, s in logits)
                assert abs(O[qi, h, c] - num / den) < 1e-12
            assert abs(L[h, qi] - (mx + math.log(den))) < 1e-12


# --------------------------------------------------------------------- backward
def _loss(x, geom, W):
    o_gen, o_ref, _, _ = oracle.sra_forward(x, [geom])
    return float((o_gen * W["gen"]).sum() + (o_ref * W["ref"]).sum())


@pytest.mark.parametrize("geom", [SampleGeom(2, 2, 2, 3, 2, 2, frame_valid=[1, 0, 1]),
                                  SampleGeom(1, 2, 3, 4, 2, 2, group_frames=2)])
def test_backward_central_finite_differences(geom):
    H, d = 2, 4
    rng = np.random.default_rng(7)
    x = rand_inputs([geom], H, d, rng=rng)
    W = {"gen": rng.standard_normal((geom.n_gen, H, d)), "ref": rng.standard_normal((geom.n_ref, H, d))}
    x["do_gen"], x["do_ref"] = W["gen"], W["ref"]
    g = oracle.sra_backward(x, [geom])
    eps = 1e-6
    for name in ("q_gen", "k_gen", "v_gen", "q_ref", "k_ref", "v_ref"):
        grad = g["d" + name]
        num = np.zeros_like(grad)
        for idx in np.ndindex(*x[name].shape):
            old = x[name][idx]
            x[name][idx] = old + eps
            lp = _loss(x, geom, W)
            x[name][idx] = old - eps
            lm = _loss(x, geom, W)
            x[name][idx] = old
            num[idx] = (lp - lm) / (2 * eps)
        err = np.abs(num - grad).max() / max(1e-12, np.abs(num).max())
        assert err < 1e-6, (name, err)


def test_backward_matches_torch_autograd_masked_softmax():
    geom = SampleGeom(2, 3, 3, 4, 2, 3, group_frames=2, frame_valid=[1, 1, 0, 1])
    H, d = 3, 8
    x = rand_inputs([geom], H, d, grads=True)
    g = oracle.sra_backward(x, [geom])
    n = geom.n_gen + geom.n_ref
    M = torch.tensor([[pred_visible(geom, i, j) for j in range(n)] for i in range(n)])
    live = M.any(dim=1)
    for h in range(H):
        cat = lambda a, b: torch.tensor(np.concatenate([x[a][:, h], x[b][:, h]]), requires_grad=True)
        q, k, v = cat("q_gen", "q_ref"), cat("k_gen", "k_ref"), cat("v_gen", "v_ref")
        do = torch.tensor(np.concatenate([x["do_gen"][:, h], x["do_ref"][:, h]]))
        s = (q @ k.T) / math.sqrt(d)
        s = s.masked_fill(~M, float("-inf"))
        p = torch.softmax(s[live], dim=-1)
        o = p @ v
        o.backward(do[live])
        G = geom.n_gen
        for nm, t in (("dq", q), ("dk", k), ("dv", v)):
            full = np.concatenate([g[nm + "_gen"][:, h], g[nm + "_ref"][:, h]])
            np.testing.assert_allclose(full, t.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_row_block_mode_matches_full():
    geom = SampleGeom(2, 4, 4, 3, 4, 4, frame_valid=[1, 0, 1])
    samples = [geom, SampleGeom(1, 4, 4, 2, 4, 4)]
    x = rand_inputs(samples, 2, 8, grads=True)
    o_gen, o_ref, lse_gen, lse_ref = oracle.sra_forward(x, samples)
    g = oracle.sra_backward(x, samples)
    rows = np.array([0, 5, 31, 32, 40, 70, 79])
    for b, off_g, off_r in ((0, 0, 0), (1, 32, 48)):
        G = samples[b].n_gen
        rws = rows[rows < G + samples[b].n_ref]
        o, lse = oracle.forward_rows(x, samples, b, 1, rws)
        dq = oracle.dq_rows(x, samples, b, 1, rws)
        for i, r in enumerate(rws):
            if r < G:
                ref_o, ref_l, ref_dq = o_gen[off_g + r, 1], lse_gen[1, off_g + r], g["dq_gen"][off_g + r, 1]
            else:
                ref_o, ref_l, ref_dq = o_ref[off_r + r - G, 1], lse_ref[1, off_r + r - G], g["dq_ref"][off_r + r - G, 1]
            np.testing.assert_allclose(o[i], ref_o, rtol=1e-12, atol=1e-13)
            np.testing.assert_allclose(dq[i], ref_dq, rtol=1e-10, atol=1e-13)
            assert (np.isneginf(ref_l) and np.isneginf(lse[i])) or abs(lse[i] - ref_l) < 1e-12


def test_key_block_mode_matches_full():
    """dK/dV of sampled keys (full softmax rows in blocks) equal the full backward's columns."""
    rng = np.random.default_rng(31)
    tok = (rng.random(3 * 16) < 0.7).astype(np.uint8).tolist()
    samples = [SampleGeom(3, 4, 4, 3, 4, 4, frame_valid=[1, 0, 1], ref_token_valid=tok),
               SampleGeom(4, 2, 4, 2, 4, 4, gen_window=1),
               SampleGeom(2, 4, 4, 3, 4, 4, group_frames=2)]
    x = rand_inputs(samples, 2, 8, grads=True)
    g = oracle.sra_backward(x, samples)
    go, ro = [0, 48, 80], [0, 48, 80]
    for b, geom in enumerate(samples):
        G, R = geom.n_gen, geom.n_ref
        keys = np.array(sorted(set(rng.integers(0, G + R, 12).tolist()) | {0, G - 1, G, G + R - 1}))
        for block in (5, 64):
            dk, dv = oracle.dkv_keys(x, samples, b, 1, keys, block_rows=block)
            for i, kk in enumerate(keys):
                if kk < G:
                    want_k, want_v = g["dk_gen"][go[b] + kk, 1], g["dv_gen"][go[b] + kk, 1]
                else:
                    want_k, want_v = g["dk_ref"][ro[b] + kk - G, 1], g["dv_ref"][ro[b] + kk - G, 1]
                np.testing.assert_allclose(dk[i], want_k, rtol=1e-10, atol=1e-13)
                np.testing.assert_allclose(dv[i], want_v, rtol=1e-10, atol=1e-13)

def test_mask_blocks_of_rows_and_columns_are_the_full_mask():
    """The mask built for a block of rows and a selection of key columns (the block mode that
    dkv_keys uses to find the query rows seeing its keys) is that block of the full mask, for
    contiguous and scattered selections, with windows, groups and token masks."""
    rng = np.random.default_rng(5)
    tok = (rng.random(4 * 12) < 0.6).astype(np.uint8).tolist()
    for geom in (SampleGeom(3, 4, 5, 4, 3, 4, group_frames=2, frame_valid=[1, 0, 1, 1], ref_token_valid=tok),
                 SampleGeom(5, 2, 3, 2, 3, 3, gen_window=1), SampleGeom(2, 3, 3, 0, 1, 1)):
        full = oracle.visibility_mask(geom)
        n = full.shape[0]
        for rows, cols in ((np.arange(n), np.arange(n)), (np.arange(3, n - 2), np.arange(1, n)),
                           (np.sort(rng.choice(n, 7, replace=False)), np.sort(rng.choice(n, 9, replace=False))),
                           (np.arange(n), np.array([0, n - 1])), (np.array([n - 1]), np.arange(n))):
            np.testing.assert_array_equal(oracle.visibility_mask(geom, rows, cols), full[np.ix_(rows, cols)])
        np.testing.assert_array_equal(oracle.visibility_mask(geom, np.arange(n)), full)


def test_varlen_samples_do_not_interact():
    samples = [SampleGeom(1, 2, 4, 2, 2, 4), SampleGeom(2, 2, 2, 1, 2, 4)]
    x = rand_inputs(samples, 1, 8, grads=True)
    o_gen, o_ref, _, _ = oracle.sra_forward(x, samples)
    # sample 1 alone
    one = {k: v[8:] if k.endswith("gen") else v[16:] for k, v in x.items()}
    p_gen, p_ref, _, _ = oracle.sra_forward(one, samples[1:])
    assert np.array_equal(p_gen, o_gen[8:]) and np.array_equal(p_ref, o_ref[16:])


def test_float32_mode_tracks_float64():
    geom = GEOMS[1]
    x = rand_inputs([geom], 2, 16)
    a = oracle.sra_forward(x, [geom])
    b = oracle.sra_forward({k: v.astype(np.float32) for k, v in x.items()}, [geom], dtype=np.float32)
    for u, v in zip(a, b):
        fin = np.isfinite(u)
        assert np.abs(u[fin] - v[fin]).max() < 1e-5


# --------------------------------------------------------------- refiner temporal window
# §2.4: the refiner keeps each frame's receptive field to a local temporal neighbourhood; its
# width is a parameter (gen_window latent frames on each side); gen queries still see the full
# valid reference.
WINDOW_GEOMS = [
    SampleGeom(4, 2, 3, 2, 2, 2, gen_window=0),
    SampleGeom(5, 2, 2, 3, 2, 2, frame_valid=[1, 0, 1], gen_window=1),
    SampleGeom(3, 3, 2, 0, 1, 1, gen_window=1),
    SampleGeom(6, 1, 3, 4, 1, 3, group_frames=2, gen_window=2),
]


def test_window_covering_every_frame_is_full_attention():
    base = SampleGeom(4, 3, 2, 3, 2, 2, frame_valid=[1, 1, 0])
    wide = SampleGeom(4, 3, 2, 3, 2, 2, frame_valid=[1, 1, 0], gen_window=3)
    assert np.array_equal(oracle.visibility_mask(base), oracle.visibility_mask(wide))
    x = rand_inputs([base], 2, 8)
    a, b = oracle.sra_forward(x, [base]), oracle.sra_forward(x, [wide])
    for u, v in zip(a, b):
        assert np.array_equal(u, v)


def test_window_zero_without_reference_is_per_frame_attention():
    """w = 0 and R = 0: every generation frame attends only to itself (dense SDPA per frame)."""
    geom = SampleGeom(3, 2, 3, 0, 1, 1, gen_window=0)
    H, d = 2, 8
    x = rand_inputs([geom], H, d)
    o_gen, _, lse_gen, _ = oracle.sra_forward(x, [geom])
    fg = geom.gen_h * geom.gen_w
    for t in range(geom.gen_frames):
        sl = slice(t * fg, (t + 1) * fg)
        for h in range(H):
            q, k, v = (torch.tensor(x[n][sl, h]) for n in ("q_gen", "k_gen", "v_gen"))
            o = torch.nn.functional.scaled_dot_product_attention(q[None], k[None], v[None], scale=1 / math.sqrt(d))[0]
            np.testing.assert_allclose(o_gen[sl, h], o.numpy(), rtol=1e-12, atol=1e-13)
            s = (q @ k.T).numpy() / math.sqrt(d)
            m = s.max(axis=1)
            np.testing.assert_allclose(lse_gen[h, sl], m + np.log(np.exp(s - m[:, None]).sum(axis=1)), rtol=1e-12)


def test_window_pair_count_closed_form():
    """Gen pairs = sum over gen frames t of F_g^2 (frames within w of t) + G * valid ref tokens."""
    for geom in WINDOW_GEOMS:
        fg, T, w = geom.gen_h * geom.gen_w, geom.gen_frames, geom.gen_window
        F = geom.ref_h * geom.ref_w
        nv = geom.ref_frames if geom.frame_valid is None else sum(geom.frame_valid)
        want = sum(fg * fg * (min(T - 1, t + w) - max(0, t - w) + 1) for t in range(T)) + geom.n_gen * F * nv
        assert oracle.pair_counts([geom], block_rows=7)[0] == want


# --------------------------------------------------------------------- token-level validity
def _token_mask(geom, seed, p=0.3):
    """Random reference token mask (1 = valid) with about a fraction p of invalid tokens."""
    rng = np.random.default_rng(seed)
    return tuple(int(x) for x in (rng.random(geom.n_ref) >= p))


def _with_tokens(geom, seed, p=0.3):
    import dataclasses
    return dataclasses.replace(geom, ref_token_valid=_token_mask(geom, seed, p))


TOKEN_GEOMS = [
    _with_tokens(SampleGeom(2, 3, 5, 4, 3, 4), 11),
    _with_tokens(SampleGeom(3, 2, 4, 5, 2, 5, frame_valid=[1, 0, 1, 1, 0]), 12),
    _with_tokens(SampleGeom(1, 4, 4, 6, 3, 3, group_frames=2, frame_valid=[1, 1, 0, 1, 1, 1]), 13, 0.5),
    _with_tokens(SampleGeom(3, 2, 2, 3, 2, 2, group_frames=3, gen_window=1), 14),
    SampleGeom(2, 2, 3, 3, 2, 3, ref_token_valid=(0,) * 18),           # every reference token invalid
    SampleGeom(1, 2, 2, 2, 2, 2, ref_token_valid=(1, 1, 1, 1, 0, 1, 1, 1)),  # one invalid token
]


def test_token_mask_predicates_pair_counts_and_closed_form():
    for geom in TOKEN_GEOMS:
        M = oracle.visibility_mask(geom)
        n = geom.n_gen + geom.n_ref
        P = np.array([[pred_visible(geom, i, j) for j in range(n)] for i in range(n)])
        assert np.array_equal(M, P)
        gp, rp = oracle.pair_counts([geom], block_rows=7)
        G = geom.n_gen
        assert gp == sum(visible_count_closed_form(geom, q) for q in range(G))
        assert rp == sum(visible_count_closed_form(geom, q) for q in range(G, n))


@pytest.mark.parametrize("fv", [[1, 0, 1, 1], [0, 0, 1, 0], [1, 1, 1, 1]])
def test_token_mask_constant_per_frame_equals_the_frame_mask(fv):
    """A token mask that repeats a frame mask over each frame's tokens is that frame mask."""
    a = SampleGeom(2, 2, 3, 4, 2, 3, group_frames=2, frame_valid=fv)
    b = SampleGeom(2, 2, 3, 4, 2, 3, group_frames=2, ref_token_valid=tuple(np.repeat(fv, 6)))
    x = rand_inputs([a], 2, 8, grads=True)
    fa, fb = oracle.sra_forward(x, [a]), oracle.sra_forward(x, [b])
    for u, w in zip(fa, fb):
        assert np.array_equal(u, w)
    ga, gb = oracle.sra_backward(x, [a]), oracle.sra_backward(x, [b])
    for k in ga:
        assert np.array_equal(ga[k], gb[k])


@pytest.mark.parametrize("geom", TOKEN_GEOMS)
def test_invalid_tokens_are_dropped_keys_and_dead_queries(geom):
    """Gen rows = dense attention over gen keys (window frames) and the valid reference tokens;
    valid ref rows = dense attention over the valid tokens of their group; invalid ref rows are
    O = 0, LSE = -inf (library SDPA over explicit key lists)."""
    H, d = 2, 8
    x = rand_inputs([geom], H, d)
    o_gen, o_ref, lse_gen, lse_ref = oracle.sra_forward(x, [geom])
    G, R, F = geom.n_gen, geom.n_ref, geom.ref_h * geom.ref_w
    ok = np.array([ref_token_ok(geom, j) for j in range(R)], dtype=bool)
    fg = geom.gen_h * geom.gen_w
    w = geom.gen_window
    for h in range(H):
        for qi in range(G):
            gk = np.arange(G) if w is None else np.nonzero(np.abs(np.arange(G) // fg - qi // fg) <= w)[0]
            k = np.concatenate([x["k_gen"][gk, h], x["k_ref"][ok, h]])
            v = np.concatenate([x["v_gen"][gk, h], x["v_ref"][ok, h]])
            o, lse = torch_sdpa64(x["q_gen"][qi:qi + 1, h], k, v, 1 / math.sqrt(d))
            np.testing.assert_allclose(o_gen[qi, h], o[0], rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(lse_gen[h, qi], lse[0], rtol=1e-12, atol=1e-12)
        g = geom.group_frames
        for j in range(R):
            if not ok[j]:
                assert np.all(o_ref[j, h] == 0) and np.isneginf(lse_ref[h, j])
                continue
            grp = (j // F) // g
            keys = [i for i in range(grp * g * F, min(R, (grp + 1) * g * F)) if ok[i]]
            o, lse = torch_sdpa64(x["q_ref"][j:j + 1, h], x["k_ref"][keys, h], x["v_ref"][keys, h], 1 / math.sqrt(d))
            np.testing.assert_allclose(o_ref[j, h], o[0], rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(lse_ref[h, j], lse[0], rtol=1e-12, atol=1e-12)


def test_token_mask_backward_finite_differences_and_dead_rows():
    geom = SampleGeom(1, 2, 2, 3, 2, 2, group_frames=2, frame_valid=[1, 1, 0],
                      ref_token_valid=(1, 0, 1, 1, 0, 1, 1, 1, 1, 1, 1, 1))
    H, d = 1, 4
    rng = np.random.default_rng(21)
    x = rand_inputs([geom], H, d, rng=rng)
    W = {"gen": rng.standard_normal((geom.n_gen, H, d)), "ref": rng.standard_normal((geom.n_ref, H, d))}
    x["do_gen"], x["do_ref"] = W["gen"], W["ref"]
    g = oracle.sra_backward(x, [geom])
    ok = np.array([ref_token_ok(geom, j) for j in range(geom.n_ref)])
    for nm in ("dq_ref", "dk_ref", "dv_ref"):
        assert np.all(g[nm][~ok] == 0)
    eps = 1e-6
    for name in ("q_gen", "k_ref", "v_ref", "q_ref"):
        grad = g["d" + name]
        num = np.zeros_like(grad)
        for idx in np.ndindex(*x[name].shape):
            old = x[name][idx]
            x[name][idx] = old + eps
            lp = _loss(x, geom, W)
            x[name][idx] = old - eps
            lm = _loss(x, geom, W)
            x[name][idx] = old
            num[idx] = (lp - lm) / (2 * eps)
        err = np.abs(num - grad).max() / max(1e-12, np.abs(num).max())
        assert err < 1e-6, (name, err)
