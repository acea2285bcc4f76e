"""Host schedules vs the oracle's explicit visibility mask, bit-exact.

The library's three tile schedules (forward, dQ, dK/dV) are expanded through the C ABI
into per-pair coverage counts; each must equal the oracle's 0/1 mask exactly: every
visible pair computed once, nothing else computed. Pair counts are checked against the
closed form and the golden values the oracle wrote.
"""
import heapq
import json
import os

import numpy as np
import pytest

import oracle
from paper_2606_13872_amd import sra
from sra_inputs import SWEEP_POINTS, SampleGeom, box_token_mask, workload

SCHEDS = [sra.SCHED_FORWARD, sra.SCHED_BWD_DQ, sra.SCHED_BWD_DKDV]


def _rand_tokens(n, seed, p):
    return tuple(int(x) for x in (np.random.default_rng(seed).random(n) >= p))


GEOMS = [
    [SampleGeom(2, 8, 8, 4, 8, 8)],                                        # tiny workload shape
    [SampleGeom(1, 3, 5, 0, 1, 1)],                                        # no reference
    [SampleGeom(3, 7, 11, 5, 6, 9)],                                       # F = 54: ragged tiles
    [SampleGeom(2, 9, 9, 6, 5, 7, frame_valid=[1, 0, 0, 1, 1, 0])],        # invalid frames
    [SampleGeom(2, 9, 9, 6, 5, 7, group_frames=2, frame_valid=[1, 0, 1, 1, 0, 0])],
    [SampleGeom(1, 16, 20, 7, 4, 9, group_frames=3)],                      # groups 3,3,1
    [SampleGeom(1, 8, 8, 5, 8, 8, group_frames=5)],                        # whole reference
    [SampleGeom(1, 4, 4, 3, 4, 4, frame_valid=[0, 0, 0])],                 # all reference invalid
    [SampleGeom(2, 10, 13, 3, 10, 13), SampleGeom(1, 17, 3, 2, 7, 7),      # varlen batch
     SampleGeom(3, 5, 5, 0, 5, 5), SampleGeom(1, 20, 20, 4, 6, 6, group_frames=2, frame_valid=[1, 1, 0, 1])],
    [SampleGeom(1, 16, 16, 2, 16, 16, group_frames=1)],                    # tile-aligned sizes
    [SampleGeom(5, 9, 13, 3, 6, 9, gen_window=1)],                         # temporal window
    [SampleGeom(6, 7, 7, 4, 5, 5, group_frames=2, frame_valid=[1, 0, 1, 1], gen_window=0),
     SampleGeom(4, 20, 15, 2, 9, 9, gen_window=2), SampleGeom(3, 6, 6, 1, 6, 6)],
    [SampleGeom(3, 10, 10, 2, 4, 4, gen_window=5)],                        # window >= all frames
    # token-level validity: random masks, box masks, with frame masks, groups and windows
    [SampleGeom(2, 9, 9, 4, 5, 7, ref_token_valid=_rand_tokens(4 * 35, 1, 0.3))],
    [SampleGeom(2, 9, 9, 6, 5, 7, group_frames=2, frame_valid=[1, 0, 1, 1, 0, 1],
                ref_token_valid=_rand_tokens(6 * 35, 2, 0.5))],
    [SampleGeom(1, 8, 8, 5, 8, 8, ref_token_valid=box_token_mask(5, 8, 8, 3)),
     SampleGeom(3, 6, 6, 3, 9, 9, group_frames=3, gen_window=1, ref_token_valid=box_token_mask(3, 9, 9, 4)),
     SampleGeom(2, 5, 5, 2, 4, 4, ref_token_valid=(0,) * 32)],
    [SampleGeom(1, 6, 6, 3, 6, 6, ref_token_valid=tuple([0] * 36 + [1] * 35 + [0] + [1] * 36))],
]


@pytest.mark.parametrize("gi", range(len(GEOMS)))
def test_dense_mask_is_the_oracle_mask(gi):
    """sra_dense_mask (the rule written out by the library) equals the oracle's mask, bit-exact."""
    samples = GEOMS[gi]
    for b, g in enumerate(samples):
        want = oracle.visibility_mask(g).astype(np.uint8)
        assert np.array_equal(sra.dense_mask(samples, b), want), b
    with pytest.raises(sra.SRAError):
        sra.dense_mask(samples, len(samples))


@pytest.mark.parametrize("gi", range(len(GEOMS)))
@pytest.mark.parametrize("which", SCHEDS)
def test_schedule_mask_is_the_visibility_mask(gi, which):
    samples = GEOMS[gi]
    for b, g in enumerate(samples):
        want = oracle.visibility_mask(g).astype(np.uint8)
        got = sra.schedule_mask(samples, which, b)
        assert got.shape == want.shape
        assert np.array_equal(got, want), (which, b, np.argwhere(got != want)[:5])


@pytest.mark.parametrize("gi", range(len(GEOMS)))
def test_pair_counts_closed_form_equals_mask(gi):
    samples = GEOMS[gi]
    assert sra.pair_counts(samples) == oracle.pair_counts(samples)
    total = sum(oracle.pair_counts(samples))
    for which in SCHEDS:
        _, _, covered = sra.schedule_info(samples, which)
        assert covered == total


@pytest.mark.parametrize("gi", range(len(GEOMS)))
@pytest.mark.parametrize("which", SCHEDS)
def test_gen_queries_only_schedules_drop_exactly_the_reference_rows(gi, which):
    """With reference tokens as context only (cached reference K/V, §4.3), every schedule
    covers exactly the gen rows of the visibility mask and no reference query row."""
    samples = GEOMS[gi]
    for b, g in enumerate(samples):
        want = oracle.visibility_mask(g).astype(np.uint8)
        want[g.n_gen:, :] = 0
        got = sra.schedule_mask(samples, which, b, flags=sra.FLAG_GEN_QUERIES_ONLY)
        assert np.array_equal(got, want), (which, b, np.argwhere(got != want)[:5])
    gp, rp = oracle.pair_counts(samples)
    assert sra.pair_counts(samples, flags=sra.FLAG_GEN_QUERIES_ONLY) == (gp, 0)
    assert sra.schedule_info(samples, which, flags=sra.FLAG_GEN_QUERIES_ONLY)[2] == gp


def _golden():
    with open(os.path.join(os.path.dirname(__file__), "golden", "pair_counts.json")) as f:
        return json.load(f)


@pytest.mark.parametrize("name", ["tiny", "480p"] + [f"sweep_{n}" for n in SWEEP_POINTS]
                         + ["720p", "varlen", "varlen_window", "varlen_tokens"])
def test_full_size_pair_counts_and_coverage(name):
    w = workload(name)
    gold = _golden()[name]
    gp, rp = sra.pair_counts(w.samples, w.heads, w.head_dim)
    assert (gp, rp) == (gold["gen_pairs"], gold["ref_pairs"])
    for which in SCHEDS:
        _, _, covered = sra.schedule_info(w.samples, which, w.heads, w.head_dim)
        assert covered == gp + rp


def test_hand_derived_pair_counts():
    """Hand-derived closed forms G(G+R) + R F for the named workloads."""
    g = _golden()
    assert g["tiny"]["gen_pairs"] + g["tiny"]["ref_pairs"] == 128 * 384 + 256 * 64 == 65536
    assert g["480p"]["gen_pairs"] == 32760 * (32760 + 14040)
    assert g["720p"]["gen_pairs"] + g["720p"]["ref_pairs"] == 75600 * 151200 + 75600 * 3600
    assert g["varlen"]["gen_pairs"] + g["varlen"]["ref_pairs"] == 13849804800


@pytest.mark.parametrize("which", SCHEDS)
def test_schedule_tables_are_well_formed(which):
    samples = GEOMS[8]
    heads = 8
    items, spans = sra.schedule_export(samples, which, heads=heads)
    tile = {sra.SCHED_FORWARD: 256, sra.SCHED_BWD_DQ: 256, sra.SCHED_BWD_DKDV: 256}[which]
    n_gen = sum(g.n_gen for g in samples)
    n_ref = sum(g.n_ref for g in samples)
    rows = (n_gen, n_ref)
    real = items[items[:, 0] >= 0]
    assert np.all((real[:, 3] > 0) & (real[:, 3] <= tile))
    assert np.all(real[:, 1] < heads)
    for s in (0, 1):
        sel = real[real[:, 0] == s]
        assert np.all(sel[:, 2] + sel[:, 3] <= rows[s])
    assert np.all(spans[:, 2] > 0)
    for s in (0, 1):
        sel = spans[spans[:, 0] == s]
        assert np.all((sel[:, 1] >= 0) & (sel[:, 1] + sel[:, 2] <= rows[s]))
    assert np.all(real[:, 4] + real[:, 5] <= len(spans))
    # every (head, row) of every valid row is covered by exactly one tile
    for s in (0, 1):
        for h in range(heads):
            cov = np.zeros(rows[s], dtype=np.int32)
            for it in real[(real[:, 0] == s) & (real[:, 1] == h)]:
                cov[it[2]:it[2] + it[3]] += 1
            assert cov.max() <= 1


@pytest.mark.parametrize("which", [0, 1, 2])
def test_xcd_order_pins_heads_and_puts_long_items_first(which):
    """Each XCD's subsequence (items k, k + 8, ...) holds the heads pinned to it. Query tiles
    (forward, dQ) run longest-first over the XCD's heads; key tiles (dK/dV) run the heads one
    after another, each head's items longest-first."""
    w = workload("480p")
    items, spans = sra.schedule_export(w.samples, which, w.heads, w.head_dim)
    assert len(items) % 8 == 0
    key_major = which == sra.SCHED_BWD_DKDV
    for x in range(8):
        sub = items[x::8]
        sub = sub[sub[:, 0] >= 0]
        assert np.all(sub[:, 1] % 8 == x)
        cost = np.array([spans[i[4]:i[4] + i[5], 2].sum() for i in sub])
        if not key_major:
            assert np.all(np.diff(cost) <= 0)
            continue
        assert np.all(np.diff(sub[:, 1]) >= 0)
        for h in np.unique(sub[:, 1]):
            assert np.all(np.diff(cost[sub[:, 1] == h]) <= 0)


def test_token_masks_that_split_frames_run_on_the_compacted_stream():
    """A token mask that splits frames into runs: the gen queries of each sample see its valid
    reference tokens as one span of the compacted stream (the valid tokens of the batch back
    to back). A mask that removes only whole frames keeps the frame runs of the packed stream."""
    F = 6 * 7
    tok = (np.random.default_rng(5).random(3 * F) >= 0.3).astype(np.uint8)
    split = [SampleGeom(2, 5, 6, 3, 6, 7, ref_token_valid=tuple(tok.tolist())), SampleGeom(1, 4, 4, 2, 6, 7)]
    n_valid = [int(tok.sum()), 2 * F]
    items, spans = sra.schedule_export(split, sra.SCHED_FORWARD)
    for b in range(2):
        it = items[(items[:, 0] == 0) & (items[:, 6] == b)][0]
        own = spans[it[4]:it[4] + it[5]]
        ref = own[own[:, 0] == 1]
        assert len(ref) == 1 and ref[0, 2] == n_valid[b] and ref[0, 1] == sum(n_valid[:b])
    # every compacted reference row is covered once per head by the reference query tiles
    cov = np.zeros(sum(n_valid), dtype=np.int32)
    for it in items[(items[:, 0] == 1) & (items[:, 1] == 0)]:
        cov[it[2]:it[2] + it[3]] += 1
    assert np.all(cov == 1)
    whole = [SampleGeom(2, 5, 6, 3, 6, 7, ref_token_valid=tuple([1] * F + [0] * F + [1] * F))]
    items, spans = sra.schedule_export(whole, sra.SCHED_FORWARD)
    it = items[items[:, 0] == 0][0]
    own = spans[it[4]:it[4] + it[5]]
    assert [tuple(r[1:3]) for r in own[own[:, 0] == 1]] == [(0, F), (2 * F, F)]


def test_key_tiles_cross_reference_groups_with_key_ranges():
    """dK/dV tiles of reference keys run across frames (groups) inside a run of valid rows; each
    group's reference-query span of a crossing tile carries the range of the tile's keys in
    that group, so every (query, key) pair is still covered exactly once."""
    F = 100  # 10 x 10 tokens per frame: a 256-key tile spans three frames
    samples = [SampleGeom(1, 4, 4, 5, 10, 10)]
    items, spans = sra.schedule_export(samples, sra.SCHED_BWD_DKDV)
    ref = items[(items[:, 0] == 1) & (items[:, 1] == 0)]
    assert sorted(ref[:, 2].tolist()) == [0, 256]          # 500 ref keys: tiles of 256 and 244
    ranged = []
    for it in ref:
        for sp in spans[it[4]:it[4] + it[5]]:
            if sp[0] == 1:
                lo, hi = sp[3] & 0xFFFF, sp[3] >> 16
                if sp[3] == 0:
                    lo, hi = 0, it[3]
                # the span's queries are the frame holding the tile's keys [lo, hi)
                f = (it[2] + lo) // F
                assert sp[1] == f * F and sp[2] == F and (it[2] + hi - 1) // F == f
                ranged.append((it[2] + lo, it[2] + hi))
    assert sorted(ranged) == [(0, 100), (100, 200), (200, 256), (256, 300), (300, 400), (400, 500)]
    assert sra.schedule_info(samples, sra.SCHED_BWD_DKDV)[2] == sum(sra.pair_counts(samples))


@pytest.mark.parametrize("which,step", [(0, 64), (1, 32), (2, 32)])
def test_tile_phases_rotate_the_gen_span_and_keep_every_pair(which, step):
    """With heads pinned to XCDs, each tile whose first span is the sample's gen rows (dK/dV key
    tiles: gen queries; forward and dQ gen query tiles: gen keys) starts that span at the step
    its compute unit is predicted to reach (the XCD's launch order replayed on 32 compute
    units, one resident tile each, time in inner steps), and wraps around: the span is cut in
    two and the tile's other spans are unchanged."""
    samples = [SampleGeom(4, 48, 48, 3, 48, 48)]  # 36 gen + 27 ref tiles per head
    g = samples[0]
    aligned, a_spans = sra.schedule_export(samples, which, heads=8)
    plain, p_spans = sra.schedule_export(samples, which, heads=1)  # 1 % 8: no phases
    canon = {(int(i[0]), int(i[2]), int(i[3])): p_spans[i[4]:i[4] + i[5]] for i in plain}
    steps = -(-g.n_gen // step)
    rotated = 0
    for x in range(8):
        free = [0] * 32
        for it in aligned[x::8]:
            if it[0] < 0:
                continue
            own = a_spans[it[4]:it[4] + it[5]]
            ref = canon[(int(it[0]), int(it[2]), int(it[3]))]
            t0 = heapq.heappop(free)
            heapq.heappush(free, t0 + int(sum(-(-int(s[2]) // step) for s in own)))
            phase = (t0 % steps) * step if ref[0][0] == 0 else 0
            if phase == 0:
                assert np.array_equal(own, ref)
                continue
            rotated += 1
            assert it[5] == len(ref) + 1
            assert tuple(own[0]) == (0, phase, g.n_gen - phase, 0)
            assert tuple(own[1]) == (0, 0, phase, 0)
            assert np.array_equal(own[2:], ref[1:])
    assert rotated >= 8 * 4  # every tile past the first 32 of each XCD starts late


def test_whole_reference_group_pair_counts():
    """With one self-attention group over the whole reference (g = T_r), every valid reference
    query sees every valid reference key: G (G + R) + R^2 pairs per head, and every schedule
    covers exactly those."""
    w = workload("720p_whole_ref")
    g = w.samples[0]
    G, R = g.n_gen, g.n_ref
    assert sra.pair_counts(w.samples, w.heads, w.head_dim) == (G * (G + R), R * R)
    for which in SCHEDS:
        assert sra.schedule_info(w.samples, which, w.heads, w.head_dim)[2] == G * (G + R) + R * R


def _random_geom(rng):
    """A sample big enough that head 0 alone has more work items than one XCD has compute
    units, so the phases of the pinned order come into play."""
    gf, gh, gw = int(rng.integers(3, 6)), int(rng.integers(30, 49)), int(rng.integers(40, 57))
    rf = int(rng.integers(2, 7))
    g = int(rng.integers(1, 4))
    fv = tuple(int(v) for v in (rng.random(rf) >= 0.25)) if rng.random() < 0.5 else None
    win = int(rng.integers(0, 3)) if rng.random() < 0.4 else None
    return SampleGeom(gf, gh, gw, rf, gh, gw, group_frames=g, frame_valid=fv, gen_window=win)


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("which", SCHEDS)
def test_random_pinned_schedules_cover_the_mask(seed, which):
    """Random geometries (groups, invalid frames, windows) with 8 heads, so that heads are
    pinned to XCDs and the phases rotate spans: head 0's schedule still covers exactly the
    oracle's mask, and the covered pair count over all heads equals the closed form."""
    rng = np.random.default_rng(100 + seed)
    samples = [_random_geom(rng)]
    items, _ = sra.schedule_export(samples, which, heads=8)
    assert (items[:, 0] >= 0).sum() > 8 * 32
    want = oracle.visibility_mask(samples[0]).astype(np.uint8)
    got = sra.schedule_mask(samples, which, 0, heads=8)
    assert np.array_equal(got, want), np.argwhere(got != want)[:5]
    assert sra.schedule_info(samples, which, heads=8)[2] == sum(sra.pair_counts(samples))
