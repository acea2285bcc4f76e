"""Plain CPU oracle for Sparse Reference Attention (SRA).

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the CPU-baseline leg of
the benchmark may import this module. The product path never calls it, and it shares
no code with the HIP library.

What it computes (Avatar V, §1 contributions; §2.1 "Sparse Reference Attention";
§4.3 reference KV caching and invalid-token skipping; §8 related work):

  * Generation (gen) queries attend to every generation key and to every valid
    reference (ref) key, through ONE softmax over the concatenation of the two key sets
    (§4.3: the cached reference K/V are concatenated with the generation K/V).
  * Reference queries attend only to reference keys, never to generation keys
    (§1 and §8.2 state that the reference side attends only within itself). The group a reference query sees is its own latent frame
    by default (group_frames = 1); see the module note below.
  * Invalid reference frames (§4.3: e.g. frames where the face is not visible) are
    removed as keys for every query and as queries (output 0, log-sum-exp -inf,
    no gradient). §4.3 speaks of invalid tokens: a per-token mask of the reference
    tokens (optional, ANDed with the frame mask) removes single tokens the same way.

The oracle is the plain definition: an explicit boolean visibility mask M over the
concatenated token order [gen ; ref] of one sample, logits S = scale * Q K^T, S = -inf
where M is false, a row softmax, O = P V and LSE = log sum exp(S) (natural log). The
backward pass is the textbook gradient of that masked softmax attention. Everything is
computed in float64 by default (float32 on request), with numpy matmul as the only
library primitive; dkv_keys, which sums over billions of (query, key) pairs at full sizes,
runs the same formulas with torch CPU ops instead.

Reading of the paper taken here (it gives no formula): reference-only attention for
reference queries, combined with the claim of cost linear in reference length means a
reference query cannot see all reference keys (that would be quadratic in reference
length); the smallest grouping consistent with both is one latent frame, which is the
default. Larger groups (up to the whole reference clip) are a parameter.
This grouping is parity-unpinned by the paper: only the linearity claim supports it.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

NEG_INF = -np.inf


# ----------------------------------------------------------------------------- geometry
def sample_sizes(geom) -> Tuple[int, int, int]:
    """(G, R, F): gen tokens, ref tokens, tokens per ref latent frame (§2: patchified latents)."""
    G = geom.gen_frames * geom.gen_h * geom.gen_w
    F = geom.ref_h * geom.ref_w
    R = geom.ref_frames * F
    return G, R, F


def frame_valid(geom) -> np.ndarray:
    """Per-reference-frame validity, §4.3 (None means every frame is valid)."""
    if geom.frame_valid is None:
        return np.ones(geom.ref_frames, dtype=bool)
    v = np.asarray(geom.frame_valid).astype(bool)
    assert v.shape == (geom.ref_frames,)
    return v


def token_valid(geom) -> np.ndarray:
    """Per-reference-token validity (§4.3 invalid tokens): the token's frame is valid and, when
    the sample carries a token mask (ref_token_valid, one entry per reference token in packed
    frame-major order), its own entry is nonzero."""
    G, R, F = sample_sizes(geom)
    v = np.repeat(frame_valid(geom), F) if R > 0 else np.zeros(0, dtype=bool)
    t = getattr(geom, "ref_token_valid", None)
    if t is not None:
        t = np.asarray(t).astype(bool)
        assert t.shape == (R,)
        v = v & t
    return v


def _as_index(idx: np.ndarray):
    """A run of consecutive indices as a slice (basic indexing, fast), any other set as is."""
    if idx.size and int(idx[-1]) - int(idx[0]) + 1 == idx.size and np.all(np.diff(idx) == 1):
        return slice(int(idx[0]), int(idx[-1]) + 1)
    return idx


def _put(M: np.ndarray, r: np.ndarray, c: np.ndarray, val) -> None:
    """M[r x c] = val for row indices r and column indices c (val broadcasts to [len r, len c])."""
    if r.size == 0 or c.size == 0:
        return
    rs, cs = _as_index(r), _as_index(c)
    if isinstance(rs, slice) or isinstance(cs, slice):
        M[rs, cs] = val
    else:
        M[np.ix_(rs, cs)] = val


def visibility_mask(geom, rows: Optional[np.ndarray] = None, cols: Optional[np.ndarray] = None) -> np.ndarray:
    """Explicit visibility mask of one sample, rows and columns in [gen ; ref] order.

    M[q, k] is True when query q may attend to key k:
      gen q, gen k : True                               (full base self-attention), or
                     |gframe(q) - gframe(k)| <= w when the sample has gen_window = w
                     (§2.4: the refiner's sparse temporal attention keeps each frame's
                     receptive field to a local neighbourhood of latent frames)
      gen q, ref k : valid(k)                           (§1: gen sees every reference token)
      ref q, gen k : False                              (§1, §8.2: reference attends only within itself)
      ref q, ref k : valid(q) and valid(k) and group(q) == group(k)
    where valid(t) is the token validity of token_valid (its frame's, and its own entry of
    the token mask when there is one).
    `rows` selects a subset of query rows and `cols` a subset of key columns (block mode for
    large shapes); the result is [len(rows), len(cols)].
    """
    G, R, F = sample_sizes(geom)
    tv = token_valid(geom)
    g = int(geom.group_frames)
    assert g >= 1
    rows = np.arange(G + R) if rows is None else np.asarray(rows, dtype=np.int64)
    cols = np.arange(G + R) if cols is None else np.asarray(cols, dtype=np.int64)
    M = np.zeros((rows.size, cols.size), dtype=bool)
    qg, qr = np.nonzero(rows < G)[0], np.nonzero(rows >= G)[0]   # gen / ref query rows
    kg, kr = np.nonzero(cols < G)[0], np.nonzero(cols >= G)[0]   # gen / ref key columns
    kref = cols[kr] - G                                          # reference token of each ref column
    # generation query rows
    w = getattr(geom, "gen_window", None)
    if w is None:
        _put(M, qg, kg, True)
    else:
        assert w >= 0
        Fg = geom.gen_h * geom.gen_w
        _put(M, qg, kg, np.abs((rows[qg] // Fg)[:, None] - (cols[kg] // Fg)[None, :]) <= w)
    _put(M, qg, kr, tv[kref][None, :])
    # reference query rows (no generation key is visible to them)
    if qr.size and kr.size:
        j = rows[qr] - G
        same_group = ((j // F) // g)[:, None] == ((kref // F) // g)[None, :]
        _put(M, qr, kr, tv[j][:, None] & tv[kref][None, :] & same_group)
    return M


def pair_counts(samples: Sequence, block_rows: int = 2048) -> Tuple[int, int]:
    """Visible (query, key) pairs per head, summed over samples, counted on the mask.

    Returns (pairs of gen queries, pairs of ref queries). Counts True entries of the
    explicit mask, built in row blocks, so it is exact (integer) at any size.
    """
    gen_pairs = 0
    ref_pairs = 0
    for geom in samples:
        G, R, F = sample_sizes(geom)
        for r0 in range(0, G + R, block_rows):
            rows = np.arange(r0, min(G + R, r0 + block_rows))
            cnt = visibility_mask(geom, rows).sum(axis=1, dtype=np.int64)
            gen_pairs += int(cnt[rows < G].sum())
            ref_pairs += int(cnt[rows >= G].sum())
    return gen_pairs, ref_pairs


# ----------------------------------------------------------------------------- kernels
def _masked_softmax_rows(S: np.ndarray, M: np.ndarray):
    """Row softmax of S restricted to M. Rows with no visible key give P = 0, LSE = -inf."""
    S = np.where(M, S, NEG_INF)
    m = S.max(axis=1) if S.shape[1] else np.full(S.shape[0], NEG_INF, dtype=S.dtype)
    has = np.isfinite(m)
    m_safe = np.where(has, m, 0.0).astype(S.dtype)
    E = np.where(M, np.exp(S - m_safe[:, None]), 0.0).astype(S.dtype)
    l = E.sum(axis=1)
    P = np.zeros_like(E)
    P[has] = E[has] / l[has, None]
    lse = np.full(S.shape[0], NEG_INF, dtype=S.dtype)
    lse[has] = m[has] + np.log(l[has])
    return P, lse


def attention_rows(q: np.ndarray, k: np.ndarray, v: np.ndarray, M: np.ndarray, scale: float):
    """Masked attention for a block of query rows: returns (O, LSE, P)."""
    S = (q @ k.T) * q.dtype.type(scale)
    P, lse = _masked_softmax_rows(S, M)
    return P @ v, lse, P


def attention_backward_full(q, k, v, do, M, scale):
    """Gradient of O = softmax_M(scale Q K^T) V for one (sample, head), all rows at once.

    D = rowsum(dO * O); dV = P^T dO; dP = dO V^T; dS = P * (dP - D); dQ = scale dS K;
    dK = scale dS^T Q. Rows with no visible key have P = 0 and contribute nothing.
    """
    o, lse, P = attention_rows(q, k, v, M, scale)
    D = (do * o).sum(axis=1)
    dv = P.T @ do
    dP = do @ v.T
    dS = P * (dP - D[:, None])
    s = q.dtype.type(scale)
    dq = (dS @ k) * s
    dk = (dS.T @ q) * s
    return dq, dk, dv, o, lse


# ----------------------------------------------------------------------------- problem level
def _offsets(samples):
    go, ro = [0], [0]
    for geom in samples:
        G, R, _ = sample_sizes(geom)
        go.append(go[-1] + G)
        ro.append(ro[-1] + R)
    return go, ro


def default_scale(head_dim: int) -> float:
    return 1.0 / math.sqrt(head_dim)


def sra_forward(x: Dict[str, np.ndarray], samples: Sequence, scale: Optional[float] = None,
                dtype=np.float64):
    """Full forward over a packed batch.

    x holds q_gen, k_gen, v_gen [sumG, H, d] and q_ref, k_ref, v_ref [sumR, H, d].
    Returns o_gen [sumG,H,d], o_ref [sumR,H,d], lse_gen [H,sumG], lse_ref [H,sumR].
    """
    H, d = x["q_gen"].shape[1:]
    scale = default_scale(d) if scale is None else scale
    go, ro = _offsets(samples)
    o_gen = np.zeros((go[-1], H, d), dtype)
    o_ref = np.zeros((ro[-1], H, d), dtype)
    lse_gen = np.full((H, go[-1]), NEG_INF, dtype)
    lse_ref = np.full((H, ro[-1]), NEG_INF, dtype)
    for b, geom in enumerate(samples):
        G, R, _ = sample_sizes(geom)
        M = visibility_mask(geom)
        gs, rs = slice(go[b], go[b + 1]), slice(ro[b], ro[b + 1])
        for h in range(H):
            qh = np.concatenate([x["q_gen"][gs, h], x["q_ref"][rs, h]]).astype(dtype)
            kh = np.concatenate([x["k_gen"][gs, h], x["k_ref"][rs, h]]).astype(dtype)
            vh = np.concatenate([x["v_gen"][gs, h], x["v_ref"][rs, h]]).astype(dtype)
            o, lse, _ = attention_rows(qh, kh, vh, M, scale)
            o_gen[gs, h], o_ref[rs, h] = o[:G], o[G:]
            lse_gen[h, gs], lse_ref[h, rs] = lse[:G], lse[G:]
    return o_gen, o_ref, lse_gen, lse_ref


def sra_backward(x: Dict[str, np.ndarray], samples: Sequence, scale: Optional[float] = None,
                 dtype=np.float64):
    """Full backward over a packed batch; x additionally holds do_gen, do_ref.

    Returns dict dq_gen, dk_gen, dv_gen, dq_ref, dk_ref, dv_ref (same shapes as inputs),
    plus the forward outputs o_gen, o_ref, lse_gen, lse_ref it recomputed.
    """
    H, d = x["q_gen"].shape[1:]
    scale = default_scale(d) if scale is None else scale
    go, ro = _offsets(samples)
    out = {n: np.zeros(((go if n.endswith("gen") else ro)[-1], H, d), dtype)
           for n in ("dq_gen", "dk_gen", "dv_gen", "dq_ref", "dk_ref", "dv_ref", "o_gen", "o_ref")}
    out["lse_gen"] = np.full((H, go[-1]), NEG_INF, dtype)
    out["lse_ref"] = np.full((H, ro[-1]), NEG_INF, dtype)
    for b, geom in enumerate(samples):
        G, R, _ = sample_sizes(geom)
        M = visibility_mask(geom)
        gs, rs = slice(go[b], go[b + 1]), slice(ro[b], ro[b + 1])
        for h in range(H):
            cat = lambda a, c: np.concatenate([x[a][gs, h], x[c][rs, h]]).astype(dtype)
            q, k, v = cat("q_gen", "q_ref"), cat("k_gen", "k_ref"), cat("v_gen", "v_ref")
            do = cat("do_gen", "do_ref")
            dq, dk, dv, o, lse = attention_backward_full(q, k, v, do, M, scale)
            for name, val in (("dq", dq), ("dk", dk), ("dv", dv), ("o", o)):
                out[name + "_gen"][gs, h] = val[:G]
                out[name + "_ref"][rs, h] = val[G:]
            out["lse_gen"][h, gs], out["lse_ref"][h, rs] = lse[:G], lse[G:]
    return out


# ----------------------------------------------------------------------------- sampled rows
def _sample_head(x, samples, b, h, dtype):
    go, ro = _offsets(samples)
    gs, rs = slice(go[b], go[b + 1]), slice(ro[b], ro[b + 1])
    cat = lambda a, c: np.concatenate([np.asarray(x[a][gs, h]), np.asarray(x[c][rs, h])]).astype(dtype)
    return cat, go, ro


def forward_rows(x, samples, b: int, h: int, rows: np.ndarray, scale=None, dtype=np.float64):
    """O and LSE of selected query rows of sample b, head h (rows index [gen ; ref] of the sample).

    x entries may be any array-likes of shape [T, H, d] (numpy or CPU torch views).
    """
    d = x["q_gen"].shape[2]
    scale = default_scale(d) if scale is None else scale
    geom = samples[b]
    cat, _, _ = _sample_head(x, samples, b, h, dtype)
    q = cat("q_gen", "q_ref")[rows]
    k, v = cat("k_gen", "k_ref"), cat("v_gen", "v_ref")
    M = visibility_mask(geom, rows)
    o, lse, _ = attention_rows(q, k, v, M, scale)
    return o, lse


def dq_rows(x, samples, b: int, h: int, rows: np.ndarray, scale=None, dtype=np.float64):
    """dQ of selected query rows (each row's gradient depends only on that row)."""
    d = x["q_gen"].shape[2]
    scale = default_scale(d) if scale is None else scale
    geom = samples[b]
    cat, _, _ = _sample_head(x, samples, b, h, dtype)
    q = cat("q_gen", "q_ref")[rows]
    do = cat("do_gen", "do_ref")[rows]
    k, v = cat("k_gen", "k_ref"), cat("v_gen", "v_ref")
    M = visibility_mask(geom, rows)
    o, lse, P = attention_rows(q, k, v, M, scale)
    D = (do * o).sum(axis=1)
    dS = P * (do @ v.T - D[:, None])
    return (dS @ k) * dtype(scale)


def dkv_keys(x, samples, b: int, h: int, keys: np.ndarray, scale=None, dtype=np.float64,
             block_rows: int = 4096):
    """dK and dV of selected keys of sample b, head h (keys index [gen ; ref] of the sample).

    A key's gradient sums over every query that sees it: dV_k = sum_q P_qk dO_q and
    dK_k = scale * sum_q dS_qk Q_q, with dS_qk = P_qk (dP_qk - D_q), dP = dO V^T and
    D = rowsum(dO * O). P_qk needs the whole softmax row of q, so every query row that sees one
    of the keys goes through the full masked softmax; rows are taken in blocks to bound memory
    (the sums over q are then added block by block). At full workload sizes that is billions
    of exponentials per head, so this function does its arithmetic with torch CPU ops
    (vectorised and multithreaded), one op per step of the formulas above; the visibility mask
    is the same explicit one as everywhere else in this module.
    """
    import torch

    d = x["q_gen"].shape[2]
    scale = default_scale(d) if scale is None else scale
    geom = samples[b]
    tdt = torch.float64 if np.dtype(dtype) == np.float64 else torch.float32
    cat, _, _ = _sample_head(x, samples, b, h, dtype)
    q, do = torch.from_numpy(cat("q_gen", "q_ref")), torch.from_numpy(cat("do_gen", "do_ref"))
    k, v = torch.from_numpy(cat("k_gen", "k_ref")), torch.from_numpy(cat("v_gen", "v_ref"))
    keys = np.asarray(keys, dtype=np.int64)
    kt = torch.from_numpy(keys)
    dk = torch.zeros((len(keys), d), dtype=tdt)
    dv = torch.zeros((len(keys), d), dtype=tdt)
    # the query rows that see at least one of the keys (mask restricted to the key columns)
    seers = np.concatenate([r0 + np.nonzero(visibility_mask(geom, np.arange(r0, min(q.shape[0], r0 + block_rows)),
                                                              keys).any(axis=1))[0]
                            for r0 in range(0, q.shape[0], block_rows)])
    for i0 in range(0, seers.size, block_rows):
        rows = seers[i0:i0 + block_rows]
        M = torch.from_numpy(visibility_mask(geom, rows))
        rows = torch.from_numpy(rows)
        # masked softmax of the block's full rows (every row here sees at least one key):
        # P = exp(S - rowmax) / rowsum, torch's softmax of the masked logits
        S = (q[rows] @ k.T) * scale
        P = torch.softmax(S.masked_fill(~M, float("-inf")), dim=1)
        o = P @ v
        D = (do[rows] * o).sum(dim=1, keepdim=True)
        Pk = P[:, kt]
        dS = Pk * (do[rows] @ v[kt].T - D)
        dv += Pk.T @ do[rows]
        dk += (dS.T @ q[rows]) * scale
    return dk.numpy(), dv.numpy()
