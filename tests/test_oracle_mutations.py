"""Planted mistakes in the oracle (on the CPU) must each be caught by a pin.

Each mutant replaces one piece of the oracle with a plausible error (a dropped term, a
wrong sign or index, a transposed operand); the test runs a pin from
test_oracle_pins against the mutant and requires it to fail.
"""
import numpy as np
import pytest

import oracle
import oracle.sra_oracle as so
from sra_inputs import SampleGeom

import test_oracle_pins as pins

_orig_mask = so.visibility_mask
_orig_bwd = so.attention_backward_full
_orig_rows = so.attention_rows


def mask_gen_drops_ref(geom, rows=None):
    M = _orig_mask(geom, rows)
    G = geom.n_gen
    r = np.arange(G + geom.n_ref) if rows is None else np.asarray(rows)
    M[np.ix_(r < G, np.arange(G, M.shape[1]))] = False
    return M


def mask_ref_sees_gen(geom, rows=None):
    M = _orig_mask(geom, rows)
    G = geom.n_gen
    r = np.arange(G + geom.n_ref) if rows is None else np.asarray(rows)
    M[np.ix_(r >= G, np.arange(G))] = True
    return M


def mask_ref_sees_all_ref(geom, rows=None):
    M = _orig_mask(geom, rows)
    G = geom.n_gen
    r = np.arange(G + geom.n_ref) if rows is None else np.asarray(rows)
    M[np.ix_(r >= G, np.arange(G, M.shape[1]))] = True
    return M


def mask_group_modulo(geom, rows=None):
    class G2:
        pass
    g = G2()
    for k in ("gen_frames", "gen_h", "gen_w", "ref_frames", "ref_h", "ref_w", "frame_valid"):
        setattr(g, k, getattr(geom, k))
    g.n_gen, g.n_ref = geom.n_gen, geom.n_ref
    # wrong index: group of frame f taken as f % group_frames through a permuted frame order
    g.group_frames = geom.group_frames
    M = _orig_mask(g, rows)
    F = geom.ref_h * geom.ref_w
    G = geom.n_gen
    if geom.group_frames > 1 and geom.ref_frames > geom.group_frames:
        r = np.arange(G + geom.n_ref) if rows is None else np.asarray(rows)
        fr = (np.arange(geom.n_ref) // F)
        grp = fr % geom.group_frames
        for i, q in enumerate(r):
            if q >= G and M[i, G:].any():
                fq = (q - G) // F
                M[i, G:] = grp == (fq % geom.group_frames)
    return M


def mask_ignores_validity(geom, rows=None):
    class G2:
        pass
    g = G2()
    for k in ("gen_frames", "gen_h", "gen_w", "ref_frames", "ref_h", "ref_w", "group_frames", "gen_window"):
        setattr(g, k, getattr(geom, k))
    g.frame_valid = None
    return _orig_mask(g, rows)


def mask_window_strict(geom, rows=None):
    # off by one: |frame difference| < w instead of <= w
    w = getattr(geom, "gen_window", None)
    if w is None:
        return _orig_mask(geom, rows)
    M = _orig_mask(geom, rows)
    G, fg = geom.n_gen, geom.gen_h * geom.gen_w
    r = np.arange(G + geom.n_ref) if rows is None else np.asarray(rows)
    for i, q in enumerate(r):
        if q < G:
            M[i, :G] &= np.abs(q // fg - np.arange(G) // fg) < w
    return M


def mask_window_ignored(geom, rows=None):
    class G2:
        pass
    g = G2()
    for k in ("gen_frames", "gen_h", "gen_w", "ref_frames", "ref_h", "ref_w", "group_frames", "frame_valid"):
        setattr(g, k, getattr(geom, k))
    g.gen_window = None
    return _orig_mask(g, rows)


_orig_token_valid = so.token_valid


def tok_ignored(geom):
    # the token mask is dropped: only the frame mask counts
    G, R, F = so.sample_sizes(geom)
    return np.repeat(so.frame_valid(geom), F) if R > 0 else np.zeros(0, dtype=bool)


def tok_shifted(geom):
    # wrong index: the mask of token j is read at j + 1
    return np.roll(_orig_token_valid(geom), -1)


def mask_token_keys_only(geom, rows=None):
    # invalid tokens are dropped as keys but still answer as queries (in valid frames)
    M = _orig_mask(geom, rows)
    G, R, F = so.sample_sizes(geom)
    tv = _orig_token_valid(geom)
    fv = np.repeat(so.frame_valid(geom), F)
    r = np.arange(G + R) if rows is None else np.asarray(rows)
    grp = (np.arange(R) // F) // geom.group_frames
    for i, q in enumerate(r):
        if q >= G and fv[q - G] and not tv[q - G]:
            M[i, G:] = tv & (grp == grp[q - G])
    return M


def rows_no_scale(q, k, v, M, scale):
    return _orig_rows(q, k, v, M, 1.0)


def rows_lse_without_max(q, k, v, M, scale):
    o, lse, P = _orig_rows(q, k, v, M, scale)
    S = np.where(M, (q @ k.T) * scale, -np.inf)
    m = S.max(axis=1)
    return o, np.where(np.isfinite(lse), lse - m, lse), P


def bwd_sign(q, k, v, do, M, scale):
    o, lse, P = so.attention_rows(q, k, v, M, scale)
    D = (do * o).sum(axis=1)
    dS = P * (do @ v.T + D[:, None])
    return dS @ k * scale, dS.T @ q * scale, P.T @ do, o, lse


def bwd_transposed(q, k, v, do, M, scale):
    o, lse, P = so.attention_rows(q, k, v, M, scale)
    D = (do * o).sum(axis=1)
    dS = P * (do @ v.T - D[:, None])
    return dS @ k * scale, dS @ q * scale, P.T @ do, o, lse


def bwd_drop_D(q, k, v, do, M, scale):
    o, lse, P = so.attention_rows(q, k, v, M, scale)
    dS = P * (do @ v.T)
    return dS @ k * scale, dS.T @ q * scale, P.T @ do, o, lse


_orig_dkv = so.dkv_keys
_orig_dq = so.dq_rows


def dkv_unscaled(x, samples, b, h, keys, scale=None, dtype=np.float64, block_rows=4096):
    # dropped factor: dK without the softmax scale
    dk, dv = _orig_dkv(x, samples, b, h, keys, scale, dtype, block_rows)
    d = x["q_gen"].shape[2]
    return dk / (so.default_scale(d) if scale is None else scale), dv


def dkv_swapped(x, samples, b, h, keys, scale=None, dtype=np.float64, block_rows=4096):
    dk, dv = _orig_dkv(x, samples, b, h, keys, scale, dtype, block_rows)
    return dv, dk


def dkv_last_block_only(x, samples, b, h, keys, scale=None, dtype=np.float64, block_rows=4096):
    # the block sums overwrite instead of accumulate (only the last query block survives)
    import torch

    d = x["q_gen"].shape[2]
    scale = so.default_scale(d) if scale is None else scale
    cat, _, _ = so._sample_head(x, samples, b, h, dtype)
    q, do = torch.from_numpy(cat("q_gen", "q_ref")), torch.from_numpy(cat("do_gen", "do_ref"))
    k, v = torch.from_numpy(cat("k_gen", "k_ref")), torch.from_numpy(cat("v_gen", "v_ref"))
    kt = torch.from_numpy(np.asarray(keys, dtype=np.int64))
    dk = torch.zeros((len(keys), d), dtype=q.dtype)
    dv = torch.zeros((len(keys), d), dtype=q.dtype)
    for r0 in range(0, q.shape[0], block_rows):
        rows = np.arange(r0, min(q.shape[0], r0 + block_rows))
        M = so.visibility_mask(samples[b], rows)
        sees = M[:, keys].any(axis=1)
        if not sees.any():
            continue
        rows, M = torch.from_numpy(rows[sees]), torch.from_numpy(M[sees])
        S = ((q[rows] @ k.T) * scale).masked_fill(~M, float("-inf"))
        P = torch.softmax(S, dim=1)
        D = (do[rows] * (P @ v)).sum(dim=1, keepdim=True)
        Pk = P[:, kt]
        dS = Pk * (do[rows] @ v[kt].T - D)
        dv = Pk.T @ do[rows]
        dk = (dS.T @ q[rows]) * scale
    return dk.numpy(), dv.numpy()


def dq_rows_sign(x, samples, b, h, rows, scale=None, dtype=np.float64):
    return -_orig_dq(x, samples, b, h, rows, scale, dtype)


G_INVALID = SampleGeom(3, 2, 4, 5, 2, 5, group_frames=1, frame_valid=[1, 0, 1, 1, 0])
G_GROUP2 = SampleGeom(1, 4, 4, 6, 3, 3, group_frames=2, frame_valid=[1, 1, 0, 1, 1, 1])
G_BWD = SampleGeom(2, 2, 2, 3, 2, 2, frame_valid=[1, 0, 1])


def _all_forward_pins():
    for geom in (G_INVALID, G_GROUP2):
        pins.test_gen_rows_equal_dense_attention_over_gen_and_valid_ref(geom)
        pins.test_ref_rows_equal_per_group_dense_attention(geom)
        pins.test_zero_keys_give_log_visible_count(geom)
    pins.test_brute_force_quadruple_loop(2, None)
    pins.test_brute_force_quadruple_loop(1, 0)
    pins.test_brute_force_quadruple_loop(2, 1)
    pins.test_window_zero_without_reference_is_per_frame_attention()
    pins.test_window_pair_count_closed_form()
    pins.test_token_mask_predicates_pair_counts_and_closed_form()
    for geom in pins.TOKEN_GEOMS[:3]:
        pins.test_invalid_tokens_are_dropped_keys_and_dead_queries(geom)


def _all_backward_pins():
    pins.test_backward_central_finite_differences(G_BWD)
    pins.test_backward_matches_torch_autograd_masked_softmax()


def _all_sampled_pins():
    pins.test_row_block_mode_matches_full()
    pins.test_key_block_mode_matches_full()


@pytest.mark.parametrize("attr,mutant,which", [
    ("visibility_mask", mask_gen_drops_ref, "fwd"),
    ("visibility_mask", mask_ref_sees_gen, "fwd"),
    ("visibility_mask", mask_ref_sees_all_ref, "fwd"),
    ("visibility_mask", mask_group_modulo, "fwd"),
    ("visibility_mask", mask_ignores_validity, "fwd"),
    ("visibility_mask", mask_window_strict, "fwd"),
    ("visibility_mask", mask_window_ignored, "fwd"),
    ("token_valid", tok_ignored, "fwd"),
    ("token_valid", tok_shifted, "fwd"),
    ("visibility_mask", mask_token_keys_only, "fwd"),
    ("attention_rows", rows_no_scale, "fwd"),
    ("attention_rows", rows_lse_without_max, "fwd"),
    ("attention_backward_full", bwd_sign, "bwd"),
    ("attention_backward_full", bwd_transposed, "bwd"),
    ("attention_backward_full", bwd_drop_D, "bwd"),
    ("dkv_keys", dkv_unscaled, "sampled"),
    ("dkv_keys", dkv_swapped, "sampled"),
    ("dkv_keys", dkv_last_block_only, "sampled"),
    ("dq_rows", dq_rows_sign, "sampled"),
])
def test_planted_mistake_is_caught(monkeypatch, attr, mutant, which):
    monkeypatch.setattr(so, attr, mutant)
    if hasattr(oracle, attr):  # names the package re-exports are called through it
        monkeypatch.setattr(oracle, attr, mutant)
    run = {"fwd": _all_forward_pins, "bwd": _all_backward_pins, "sampled": _all_sampled_pins}[which]
    with pytest.raises(AssertionError):
        run()


def test_unmutated_oracle_passes_the_same_pins():
    _all_forward_pins()
    _all_backward_pins()
    _all_sampled_pins()
