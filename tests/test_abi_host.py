"""C ABI checks that need no GPU: the library loads, exports every function
declared in include/flexmoe.h, and rejects bad arguments on the host before
any device work (no call here reaches a kernel launch)."""
import ctypes
import math
import os
import re
from fractions import Fraction

import pytest

from paper_2606_27866_amd import flexmoe as fm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "flexmoe.h")
FAKE = 0x100000  # never dereferenced: every call below fails its host checks first


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(flexmoe_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    L = fm.lib()
    names = declared_functions()
    assert set(names) == set(fm.EXPORTED)
    for n in names:
        assert hasattr(L, n), n


def good_desc(**kw):
    a = dict(d=64, E=8, I=128, top_k=2, I_shared=0, dtype=fm.FLEXMOE_BF16, norm_topk=1,
             max_tokens=100)
    a.update(kw)
    return fm.make_desc(**a)


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=7), -5),
    (dict(d=60), -2), (dict(d=0), -2), (dict(I=100), -2), (dict(I_shared=12), -2),
    (dict(I_shared=-8), -2), (dict(E=0), -2), (dict(E=257), -2), (dict(top_k=0), -2),
    (dict(top_k=9), -2), (dict(E=32, top_k=17), -2), (dict(max_tokens=-1), -2),
    (dict(norm_topk=2), -1), (dict(max_tokens=1 << 29), -2),
    # bf16 operand blocks of 2^30 elements or more
    (dict(d=1 << 14, max_tokens=1 << 16), -2), (dict(I=1 << 15, d=1 << 15), -2),
    (dict(I_shared=1 << 13, max_tokens=1 << 17), -2),
])
def test_bad_descriptor(kw, code):
    desc = good_desc(**kw)
    assert fm.lib().flexmoe_workspace_bytes(ctypes.byref(desc), 1) == 0
    with pytest.raises(fm.FlexMoEError) as ei:
        fm.flexmoe_layer_forward(desc, 1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, None,
                                 FAKE, FAKE, workspace_bytes=1 << 40, stream=0)
    assert ei.value.code == code


def test_fp32_has_no_operand_block_limit():
    desc = good_desc(d=1 << 14, max_tokens=1 << 16, dtype=fm.FLEXMOE_F32)
    assert fm.lib().flexmoe_workspace_bytes(ctypes.byref(desc), 1) > 0


def test_workspace_monotone_in_T():
    desc = good_desc(I_shared=64)
    sizes = [fm.flexmoe_workspace_bytes(desc, T) for T in (0, 1, 2, 63, 64, 65, 100)]
    assert sizes == sorted(sizes)
    assert all(s % 256 == 0 for s in sizes)
    with pytest.raises(fm.FlexMoEError):
        fm.flexmoe_workspace_bytes(desc, 101)


@pytest.mark.parametrize("shape", [
    dict(d=2048, E=60, I=1408, top_k=4, I_shared=5632),   # split at T <= 3840
    dict(d=256, E=8, I=128, top_k=2, I_shared=3080),      # split 3 ways, ragged chunk
    dict(d=4096, E=8, I=14336, top_k=2, I_shared=0),
    dict(d=256, E=8, I=128, top_k=2, I_shared=3080, dtype=fm.FLEXMOE_F32),
])
def test_workspace_monotone_across_shared_splits(shape):
    """The shared expert's down reduction is split into more chunks (each
    with its own rows) at smaller T; a workspace sized for max_tokens must
    still serve every smaller T."""
    desc = good_desc(max_tokens=20000, **shape)
    Ts = list(range(0, 700)) + list(range(700, 20001, 37)) + [20000]
    sizes = [fm.flexmoe_workspace_bytes(desc, T) for T in Ts]
    assert all(a <= b for a, b in zip(sizes, sizes[1:]))


def test_forward_argument_errors():
    desc = good_desc()
    need = fm.flexmoe_workspace_bytes(desc, 10)
    f = fm.flexmoe_layer_forward

    def call(T=10, x=FAKE, ws=FAKE, nbytes=need, shared=(None, None, None), y=FAKE, keep=FAKE):
        f(desc, T, x, FAKE, FAKE, FAKE, FAKE, keep, *shared, y, ws, workspace_bytes=nbytes, stream=0)

    for kwargs, code in [(dict(x=None), -1), (dict(y=None), -1), (dict(keep=None), -1),
                         (dict(T=-1), -1), (dict(T=101), -2), (dict(nbytes=need - 1), -4),
                         (dict(ws=None), -4), (dict(ws=FAKE + 8), -4),
                         (dict(shared=(FAKE, FAKE, FAKE)), -1)]:
        with pytest.raises(fm.FlexMoEError) as ei:
            call(**kwargs)
        assert ei.value.code == code, kwargs
        assert fm.flexmoe_last_error()
    call(T=0)  # T = 0 is a valid no-op: nothing is launched


def test_shared_weights_required_iff_shared_expert():
    desc = good_desc(I_shared=64)
    need = fm.flexmoe_workspace_bytes(desc, 4)
    with pytest.raises(fm.FlexMoEError) as ei:
        fm.flexmoe_layer_forward(desc, 4, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE,
                                 FAKE, FAKE, workspace_bytes=need, stream=0)
    assert ei.value.code == -1


def test_set_budget_rejects_out_of_range_on_host():
    desc = good_desc()
    for bad in ([0] * 7 + [129], [-1] + [0] * 7):
        with pytest.raises(fm.FlexMoEError) as ei:
            fm.flexmoe_set_budget(desc, FAKE, bad, stream=0)
        assert ei.value.code == -3
    with pytest.raises(fm.FlexMoEError) as ei:
        fm.flexmoe_set_budget(desc, None, [1] * 8, stream=0)
    assert ei.value.code == -1


def test_rank_reorder_null_pointer():
    with pytest.raises(fm.FlexMoEError) as ei:
        fm.flexmoe_rank_reorder(good_desc(), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, stream=0)
    assert ei.value.code == -1


def test_keep_from_ratio_matches_exact_ceil():
    for I in (14336, 2560, 1408, 512, 1000, 7):
        for r in ("0.1", "0.4", "0.7", "1.0", "0.25", "0.5", "0.75", "0", "0.333"):
            assert fm.flexmoe_keep_from_ratio(float(r), I) == math.ceil(Fraction(r) * I)
    assert fm.flexmoe_keep_from_ratio(-0.1, 10) == -1
    assert fm.flexmoe_keep_from_ratio(float("nan"), 10) == -1


def test_one_hip_runtime_in_process():
    """The library must share torch's HIP runtime (a second copy would not see
    the GPU and could not use torch's pointers and streams)."""
    fm.lib()
    maps = open("/proc/self/maps").read()
    hips = set(re.findall(r"\S*libamdhip64\S*", maps))
    hsas = set(re.findall(r"\S*libhsa-runtime64\S*", maps))
    assert len(hips) == 1 and len(hsas) == 1, (hips, hsas)


def test_noalloc_rejects_what_its_scratch_cannot_hold():
    """The no-allocation forward refuses, on the host and before any device
    call, a batch whose workspace regions exceed its 64 MiB static scratch,
    and null pointers; T = 0 is a no-op."""
    desc = good_desc(d=3584, E=64, I=2560, top_k=8, I_shared=20480, max_tokens=1024)
    assert fm.flexmoe_workspace_bytes(desc, 1024) > 64 << 20
    assert fm.flexmoe_workspace_bytes(desc, 64) <= 64 << 20
    f = fm.flexmoe_layer_forward_noalloc
    with pytest.raises(fm.FlexMoEError) as ei:
        f(desc, 1024, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, stream=0)
    assert ei.value.code == -4 and "static scratch" in fm.flexmoe_last_error()
    for T, code in ((-1, -1), (1025, -2)):
        with pytest.raises(fm.FlexMoEError) as ei:
            f(desc, T, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, stream=0)
        assert ei.value.code == code
    with pytest.raises(fm.FlexMoEError) as ei:
        f(desc, 4, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, stream=0)
    assert ei.value.code == -1
    f(desc, 0, None, None, None, None, None, None, None, None, None, None, stream=0)
