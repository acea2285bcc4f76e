"""The C-ABI library loads, exports what include/sra.h declares, and validates on the host.

No device work happens here: every call either fails validation before anything is
enqueued or is a host-only hook.
"""
import ctypes
import os

import pytest

from paper_2606_13872_amd import sra
from sra_inputs import SampleGeom


HOST_ONLY = bool(os.environ.get("SRA_HOST_LIB"))  # the sanitizer run's host-only library


@pytest.mark.skipif(HOST_ONLY, reason="the host-only sanitizer build has no device entry points")
def test_library_exports_every_declared_function():
    names = sra.header_functions()
    assert set(names) >= {"sra_workspace_size", "sra_forward", "sra_backward", "sra_pair_counts",
                          "sra_schedule_info", "sra_schedule_mask", "sra_schedule_export",
                          "sra_release_caches", "sra_status_string", "sra_last_error", "sra_version",
                          "sra_kernel_timing_enable", "sra_kernel_timing", "sra_dense_mask"}
    L = sra.lib()
    for n in names:
        assert hasattr(L, n), n
    assert L.sra_version() >= 200
    assert sra.status_string(0) == "SRA_OK"
    assert sra.status_string(3) == "SRA_ERR_WORKSPACE_TOO_SMALL"


GOOD = [SampleGeom(2, 8, 8, 4, 8, 8)]


@pytest.mark.parametrize("samples,heads,d,stride,status", [
    ([SampleGeom(0, 8, 8, 4, 8, 8)], 1, 64, 0, sra.SRA_ERR_INVALID_ARGUMENT),
    ([SampleGeom(2, 8, 8, -1, 8, 8)], 1, 64, 0, sra.SRA_ERR_INVALID_ARGUMENT),
    ([SampleGeom(2, 8, 8, 4, 8, 8, group_frames=0)], 1, 64, 0, sra.SRA_ERR_INVALID_ARGUMENT),
    ([SampleGeom(2, 8, 8, 2, 0, 8)], 1, 64, 0, sra.SRA_ERR_INVALID_ARGUMENT),
    (GOOD, 0, 64, 0, sra.SRA_ERR_INVALID_ARGUMENT),
    (GOOD, 1, 96, 0, sra.SRA_ERR_UNSUPPORTED),
    (GOOD, 1, 0, 0, sra.SRA_ERR_INVALID_ARGUMENT),
    (GOOD, 2, 64, 64, sra.SRA_ERR_INVALID_ARGUMENT),      # stride < H*d
    (GOOD, 2, 64, 132, sra.SRA_ERR_INVALID_ARGUMENT),     # stride not a multiple of 8
    ([SampleGeom(70000, 200, 200, 0, 1, 1)], 1, 64, 0, sra.SRA_ERR_INVALID_ARGUMENT),  # > int32 rows
    # heads * rows above 2^31 - 1: 40 heads x 53,687,092 gen rows, then 40 x that many ref rows
    ([SampleGeom(1, 53687092, 1, 0, 1, 1)], 40, 128, 0, sra.SRA_ERR_UNSUPPORTED),
    ([SampleGeom(1, 1, 1, 1, 53687092, 1)], 40, 128, 0, sra.SRA_ERR_UNSUPPORTED),
    # the largest accepted: heads * rows = 2^31 - 1 exactly (gen), and just below (ref)
    ([SampleGeom(1, 2147483647, 1, 0, 1, 1)], 1, 64, 0, None),
    ([SampleGeom(1, 1, 1, 1, 53687091, 1)], 40, 128, 0, None),
    # token strides whose offsets inside a tile (63 rows past its first) would overflow int32
    (GOOD, 2, 64, 33554432, sra.SRA_ERR_UNSUPPORTED),
    (GOOD, 2, 64, 1 << 40, sra.SRA_ERR_UNSUPPORTED),
    (GOOD, 2, 64, 33554424, "ok"),                        # the largest accepted multiple of 8
])
def test_invalid_problems_are_rejected(samples, heads, d, stride, status):
    p = sra.Problem(samples, heads, d, gen_token_stride=stride)
    n = ctypes.c_size_t(0)
    if status is None:  # at the limit: accepted (checked on the geometry only, no schedule)
        gp, rp = ctypes.c_int64(0), ctypes.c_int64(0)
        assert sra.lib().sra_pair_counts(p.ptr, ctypes.byref(gp), ctypes.byref(rp)) == sra.SRA_OK
        G, R = p.n_gen, p.n_ref
        F = samples[0].ref_h * samples[0].ref_w
        assert (gp.value, rp.value) == (G * (G + R), R * F)
        return
    st = sra.lib().sra_workspace_size(p.ptr, 0, ctypes.byref(n))
    if status == "ok":
        assert st == sra.SRA_OK and n.value > 0
        return
    assert st == status
    assert len(sra.lib().sra_last_error()) > 0


def test_flags_and_batch_validation():
    for bad in (4, 8, 0x80000000, 7):
        p = sra.Problem(GOOD, 1, 64, flags=bad)
        with pytest.raises(sra.SRAError) as e:
            p.workspace_size(False)
        assert e.value.status == sra.SRA_ERR_INVALID_ARGUMENT
    assert sra.Problem(GOOD, 1, 64, flags=sra.FLAG_GEN_QUERIES_ONLY).workspace_size(False) > 0
    p = sra.Problem([], 1, 64)
    with pytest.raises(sra.SRAError):
        p.workspace_size(False)


def test_workspace_size_is_host_only_and_grows_for_backward():
    p = sra.Problem(GOOD, 1, 64)
    f, b = p.workspace_size(False), p.workspace_size(True)
    assert f > 0 and b > f and f % 256 == 0 and b % 256 == 0


def test_forward_rejects_null_and_unaligned_pointers_before_any_launch():
    p = sra.Problem(GOOD, 1, 64)
    L = sra.lib()
    fake = ctypes.c_void_p(1 << 20)
    null = ctypes.c_void_p(0)
    args = [fake] * 6 + [fake, fake, fake, fake]
    # null gen pointer
    st = L.sra_forward(p.ptr, null, *args[1:], fake, ctypes.c_size_t(1 << 20), null)
    assert st == sra.SRA_ERR_INVALID_ARGUMENT
    # unaligned pointer
    st = L.sra_forward(p.ptr, ctypes.c_void_p((1 << 20) + 2), *args[1:], fake, ctypes.c_size_t(1 << 20), null)
    assert st == sra.SRA_ERR_INVALID_ARGUMENT
    # workspace too small
    st = L.sra_forward(p.ptr, *args, fake, ctypes.c_size_t(16), null)
    assert st == sra.SRA_ERR_WORKSPACE_TOO_SMALL
    # workspace misaligned
    st = L.sra_forward(p.ptr, *args, ctypes.c_void_p((1 << 20) + 16), ctypes.c_size_t(1 << 20), null)
    assert st == sra.SRA_ERR_INVALID_ARGUMENT
    # reference pointers may be NULL only when there is no reference
    ref_null = [fake] * 3 + [null] * 3 + [fake, null, fake, null]
    st = L.sra_forward(p.ptr, *ref_null, fake, ctypes.c_size_t(1 << 20), null)
    assert st == sra.SRA_ERR_INVALID_ARGUMENT


def test_backward_rejects_small_workspace():
    p = sra.Problem(GOOD, 1, 64)
    fake = ctypes.c_void_p(1 << 20)
    st = sra.lib().sra_backward(p.ptr, *([fake] * 18), fake, ctypes.c_size_t(p.workspace_size(True) - 256),
                                ctypes.c_void_p(0))
    assert st == sra.SRA_ERR_WORKSPACE_TOO_SMALL


def test_flag_constant_matches_the_header():
    import re
    text = open(sra.HEADER_PATH).read()
    m = re.search(r"SRA_FLAG_GEN_QUERIES_ONLY\s*=\s*(\d+)u", text)
    assert m and int(m.group(1)) == sra.FLAG_GEN_QUERIES_ONLY


def test_window_flag_constant_and_struct_layout():
    import re
    text = open(sra.HEADER_PATH).read()
    m = re.search(r"SRA_FLAG_GEN_WINDOW\s*=\s*(\d+)u", text)
    assert m and int(m.group(1)) == sra.FLAG_GEN_WINDOW
    # gen_window fills the padding before the first pointer; the token mask pointer follows it
    assert ctypes.sizeof(sra._SampleGeom) == 48 and sra._SampleGeom.ref_frame_valid.offset == 32
    assert sra._SampleGeom.ref_token_valid.offset == 40
    bad = SampleGeom(3, 2, 2, 1, 2, 2, gen_window=-1)
    with pytest.raises(sra.SRAError) as e:
        sra.Problem([bad], 1, 64).workspace_size(False)
    assert e.value.status == sra.SRA_ERR_INVALID_ARGUMENT


def test_cu_seqlens_are_checked_against_the_geometry():
    """Optional packed-row offsets must equal the geometry's; a mismatch is rejected before
    anything reaches the library (CPU tensors here: no device work can happen)."""
    import numpy as np
    import torch

    samples = [SampleGeom(1, 2, 4, 2, 2, 2), SampleGeom(2, 2, 2, 0, 1, 1)]
    g, r = sra.cu_seqlens(samples)
    assert g.tolist() == [0, 8, 16] and r.tolist() == [0, 8, 8]
    x = torch.zeros((16, 1, 64), dtype=torch.bfloat16)
    y = torch.zeros((8, 1, 64), dtype=torch.bfloat16)
    for bad in ({"cu_seqlens_gen": [0, 8, 17]}, {"cu_seqlens_ref": torch.tensor([0, 4, 8])},
                {"cu_seqlens_gen": np.array([0, 16])}):
        with pytest.raises(sra.SRAError) as e:
            sra.forward(x, x, x, y, y, y, samples, **bad)
        assert e.value.status == sra.SRA_ERR_INVALID_ARGUMENT
        with pytest.raises(sra.SRAError):
            sra.backward(x, x, x, y, y, y, x, y, None, None, x, y, samples, **bad)


def test_compacted_plans_reserve_the_compacted_reference_tensors():
    """A token mask that splits frames runs on the compacted reference stream: the workspace
    holds 4 (forward) or 8 (backward) compacted [rows, H, d] bf16 tensors more; a mask that
    only removes whole frames does not."""
    F, H, d = 16, 2, 64
    tok = [1, 0] * (F // 2) + [1] * F
    split = sra.Problem([SampleGeom(1, 4, 4, 2, 4, 4, ref_token_valid=tok)], H, d)
    plain = sra.Problem([SampleGeom(1, 4, 4, 2, 4, 4)], H, d)
    whole = sra.Problem([SampleGeom(1, 4, 4, 2, 4, 4, ref_token_valid=[0] * F + [1] * F)], H, d)
    n_valid = sum(tok)
    rows = (n_valid * H * d * 2 + 255) // 256 * 256
    assert split.workspace_size(False) >= plain.workspace_size(False) - 4096 + 4 * rows
    assert split.workspace_size(True) >= plain.workspace_size(True) - 4096 + 8 * rows
    assert whole.workspace_size(False) < plain.workspace_size(False) + 4 * rows


# ---------------------------------------------------------------- binding argument checks (CPU)
def _tensors(H=1, d=64, G=128, R=256, device="cpu"):
    import torch

    def t(n):
        return torch.zeros((n, H, d), dtype=torch.bfloat16, device=device)
    return [t(G), t(G), t(G), t(R), t(R), t(R)]


def _rejects(fn, *args, match=None, **kw):
    with pytest.raises(sra.SRAError) as e:
        fn(*args, **kw)
    assert e.value.status == sra.SRA_ERR_INVALID_ARGUMENT
    if match:
        assert match in str(e.value), str(e.value)


def test_binding_rejects_bad_inputs_before_the_library():
    """dtype, shape and layout of q/k/v are checked against the geometry, then the device: a CPU
    tensor never reaches the library (a device pointer of the wrong kind would fault the GPU)."""
    import torch

    qg, kg, vg, qr, kr, vr = _tensors()
    _rejects(sra.forward, qg.float(), kg, vg, qr, kr, vr, GOOD, match="dtype")
    _rejects(sra.forward, qg, kg[:100], vg, qr, kr, vr, GOOD, match="shape")
    _rejects(sra.forward, qg, kg, vg, qr, kr[:, :, :32], vr, GOOD, match="shape")
    q2, k2, v2, qr2, kr2, vr2 = _tensors(H=2)
    _rejects(sra.forward, q2, k2, v2, qr2, kr2, vr2.transpose(1, 2).contiguous().transpose(1, 2), GOOD,
             match="contiguous heads")
    _rejects(sra.forward, qg, kg, vg, None, kr, vr, GOOD, match="q_ref")
    _rejects(sra.forward, qg, kg, vg, qr, kr, vr, GOOD, match="GPU")
    _rejects(sra.forward, qg.unsqueeze(0), kg, vg, qr, kr, vr, GOOD, match="q_gen")
    # a tensor on another device than q_gen (the meta device stands in for a second GPU)
    meta = torch.zeros((256, 1, 64), dtype=torch.bfloat16, device="meta")
    with pytest.raises(sra.SRAError):
        sra.forward(qg, kg, vg, qr, meta, vr, GOOD)


def test_binding_rejects_bad_output_buffers():
    import torch

    qg, kg, vg, qr, kr, vr = _tensors()
    bad = {
        "o_gen": torch.zeros((128, 1, 64), dtype=torch.float32),
        "lse_gen": torch.zeros((128, 1), dtype=torch.float32),
        "o_ref": torch.zeros((256, 1, 128), dtype=torch.bfloat16)[:, :, :64],  # not dense
        "lse_ref": torch.zeros((1, 256), dtype=torch.bfloat16),
    }
    for name, t in bad.items():
        with pytest.raises(sra.SRAError) as e:
            sra._forward_args(qg, kg, vg, qr, kr, vr, GOOD, None, {name: t}, False, None, None)
        assert e.value.status == sra.SRA_ERR_INVALID_ARGUMENT and name in str(e.value)
    with pytest.raises(sra.SRAError):
        sra._workspace({"workspace": torch.zeros(16, dtype=torch.float32)}, 16, torch.device("cpu"))


def test_binding_backward_checks_every_tensor():
    import torch

    qg, kg, vg, qr, kr, vr = _tensors()
    og, org, dog, dor = qg, qr, qg, qr
    lg, lr = torch.zeros((1, 128)), torch.zeros((1, 256))
    args = [qg, kg, vg, qr, kr, vr, og, org, lg, lr, dog, dor]
    cases = {6: og.float(), 8: lg.t(), 9: torch.zeros((1, 255)), 10: dog[:, :, :32],
             11: qr.transpose(0, 1).contiguous().transpose(0, 1)}
    for i, t in cases.items():
        a = list(args)
        a[i] = t
        _rejects(sra.backward, *a, GOOD)
    _rejects(sra.backward, *args, GOOD, match="GPU")
    _rejects(sra.backward, *args, GOOD, out={"dk_ref": torch.zeros((256, 1, 64))}, match="dk_ref")


@pytest.mark.skipif(HOST_ONLY, reason="the host-only sanitizer build has no device entry points")
def test_noalloc_forward_rejects_oversized_problems_on_the_host():
    """The allocation-free forward takes its workspace from a static array of
    SRA_NOALLOC_WORKSPACE_MAX bytes; a problem needing more (here a token mask that forces the
    compacted reference stream at 40 heads) is rejected before any device call."""
    tok = [1, 0] * 1024 + [1] * 2048
    p = sra.Problem([SampleGeom(1, 4, 4, 2, 32, 64, ref_token_valid=tok)], 40, 128)
    assert p.workspace_size(False) > sra.noalloc_workspace_max() == 32 << 20
    fake = ctypes.c_void_p(1 << 20)
    st = sra.lib().sra_forward_noalloc(p.ptr, *([fake] * 10), ctypes.c_void_p(0))
    assert st == sra.SRA_ERR_WORKSPACE_TOO_SMALL
    assert b"static scratch maximum" in sra.lib().sra_last_error()
    # validation errors come first, as for sra_forward
    bad = sra.Problem([SampleGeom(0, 4, 4, 2, 4, 4)], 1, 64)
    assert sra.lib().sra_forward_noalloc(bad.ptr, *([fake] * 10), ctypes.c_void_p(0)) == sra.SRA_ERR_INVALID_ARGUMENT
