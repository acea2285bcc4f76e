"""The forward's mid-span rescale, forced and checked against the oracle.

The forward does not track the running max per 32-key half: P is computed against the current
max m, and a lane whose 16 values of the half sum to more than 2^16 sends its whole wave down
the exact path (recompute S of the half, move m to the true running max, scale O and l by
alpha = 2^(m_old - m_new), recompute P). At the first half m = -inf, so alpha = 0 and O is
still zero; only a later half (O already holding the P V of earlier halves) exercises
0 < alpha < 1. Logits with a large spread reach it: unit softmax scale on unnormalised inputs,
where a row's max keeps rising by more than 16 log2 units as keys stream past.

`mid_span_triggers` replays the kernel's key order on the host (each span's full 64-key tiles
in span order, as two 32-key halves; lanes l and l + 32 hold the keys 8a + b and 8a + 4 + b of
a half, b < 4; a wave is 32 query rows of a 256-row work item, rows past the item are zero) and
counts the halves after the first whose overflow check fires with a finite m: the test asserts
that there are many, in generation and in reference work items. Ragged span tails run a
separate masked step and are not counted.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_13872_amd import sra
from sra_inputs import SampleGeom, make_inputs, to_numpy64

pytestmark = pytest.mark.gpu

LOG2E = 1.4426950408889634
BIG = 65536.0
REL, LSE_ABS = 1e-2, 1e-3


def _lane_keys():
    k0 = [8 * a + b for a in range(4) for b in range(4)]
    return np.array(k0), np.array(k0) + 4


def mid_span_triggers(x, samples, scale, head=0):
    """(gen, ref) counts of (wave, half) events after a wave's first half where the overflow
    check fires for some row whose m is finite, with the sum above 2^17 (a margin over the
    kernel's 2^16, so fp32 against fp64 logits cannot change the count)."""
    items, spans = sra.schedule_export(samples, sra.SCHED_FORWARD, heads=x["q_gen"].shape[1],
                                       head_dim=x["q_gen"].shape[2])
    lanes = _lane_keys()
    q = {0: to_numpy64(x["q_gen"][:, head]), 1: to_numpy64(x["q_ref"][:, head])}
    k = {0: to_numpy64(x["k_gen"][:, head]), 1: to_numpy64(x["k_ref"][:, head])}
    sl2 = scale * LOG2E
    counts = [0, 0]
    for it in items:
        stream, h, start, length, soff, scnt = (int(v) for v in it[:6])
        if stream < 0 or h != head:
            continue
        keys = []  # full 64-key tiles of every span, in span order
        for sp in spans[soff:soff + scnt]:
            ks, kstart, klen = int(sp[0]), int(sp[1]), int(sp[2])
            for off in range(0, klen - 63, 64):
                keys.append(k[ks][kstart + off:kstart + off + 64])
        if not keys:
            continue
        kk = np.concatenate(keys)
        for w in range(0, 256, 32):
            rows = np.zeros((32, q[stream].shape[1]))
            n = max(0, min(32, length - w))
            if n == 0:
                continue
            rows[:n] = q[stream][start + w:start + w + n]
            s = rows @ kk.T * sl2  # [32 rows, keys] in log2 units
            m = np.full(32, -np.inf)
            for hf in range(s.shape[1] // 32):
                blk = s[:, 32 * hf:32 * hf + 32]
                with np.errstate(over="ignore", invalid="ignore"):
                    sums = [np.exp2(blk[:, lk] - m[:, None]).sum(1) for lk in lanes]
                fires = ~((sums[0] <= BIG) & (sums[1] <= BIG))
                if fires.any():
                    if hf > 0 and (np.isfinite(m) & ((sums[0] > 2 * BIG) | (sums[1] > 2 * BIG))).any():
                        counts[stream] += 1
                    m = np.maximum(m, blk.max(1))
    return counts


CASES = {
    "d128": ([SampleGeom(2, 8, 16, 3, 8, 16), SampleGeom(1, 12, 16, 2, 8, 16)], 2, 128, 1.0),
    "d64": ([SampleGeom(2, 8, 16, 3, 8, 16), SampleGeom(1, 12, 16, 2, 8, 16)], 2, 64, 1.5),
}


@pytest.mark.parametrize("case", list(CASES))
def test_mid_span_rescale_matches_the_oracle(case):
    samples, H, d, scale = CASES[case]
    x = make_inputs(samples, H, d, 31)
    gen_fires, ref_fires = mid_span_triggers(x, samples, scale)
    print(f"{case}: mid-span rescales in gen waves {gen_fires}, ref waves {ref_fires}", flush=True)
    assert gen_fires >= 8 and ref_fires >= 4, (gen_fires, ref_fires)
    dev = torch.device("cuda")
    y = {n: v.to(dev) for n, v in x.items()}
    got = sra.forward(y["q_gen"], y["k_gen"], y["v_gen"], y["q_ref"], y["k_ref"], y["v_ref"], samples, scale)
    torch.cuda.synchronize()
    want = oracle.sra_forward({n: to_numpy64(v) for n, v in x.items()}, samples, scale)
    for name, g, w in zip(("o_gen", "o_ref"), got[:2], want[:2]):
        g = g.float().cpu().numpy().astype(np.float64)
        assert np.all(np.isfinite(g)), name
        for h in range(H):
            rel = np.linalg.norm(g[:, h] - w[:, h]) / np.linalg.norm(w[:, h])
            assert rel <= REL, (name, h, rel)
    for name, g, w in zip(("lse_gen", "lse_ref"), got[2:], want[2:]):
        err = np.abs(g.cpu().numpy().astype(np.float64) - w).max()
        assert err <= LSE_ABS, (name, err)
