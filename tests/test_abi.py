"""C-ABI checks that need no GPU: the library loads, exports every symbol the
public header declares, sizes workspaces, and rejects bad arguments on the
host before anything is enqueued (fake, never-dereferenced device pointers)."""

import ctypes
import os
import re

import pytest

import paper_2609_32114_amd as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hagdn.h")

needs_lib = pytest.mark.skipif(not os.path.exists(P.library_path()),
                               reason="libhagdn.so not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("gdn_prefill", "kda_prefill", "gdn_prefill_workspace_size",
              "kda_prefill_workspace_size", "hagdn_last_error", "hagdn_device_status"):
        assert n in names


@needs_lib
def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(P.library_path())
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


@needs_lib
def test_workspace_size():
    n1 = P.workspace_size("gdn", 1, 4096, 16, 16, 128, 128, P.HAGDN_BF16)
    n2 = P.workspace_size("gdn", 1, 4096, 16, 16, 128, 128, P.HAGDN_F32)
    assert n1 > 0 and n2 > n1
    assert P.workspace_size("kda", 1, 0, 1, 1, 64, 64, P.HAGDN_F32) > 0
    for bad in [(0, 64, 1, 1, 64, 64, 1), (1, 64, 2, 3, 64, 64, 1), (1, 64, 1, 1, 96, 64, 1),
                (1, 64, 1, 1, 64, 64, 7), (1, -1, 1, 1, 64, 64, 1)]:
        with pytest.raises(P.HagdnError):
            P.workspace_size("gdn", *bad)


FAKE = 0x100000  # 16-byte aligned, never dereferenced


def _call(lib, kind="gdn", N=1, T=100, Hqk=1, Hv=1, Dk=64, Dv=64, dtype=0, ws_bytes=1 << 40,
          **over):
    ptrs = dict(q=FAKE, k=FAKE, v=FAKE, g=FAKE, beta=FAKE, s0=None, cu=FAKE, o=FAKE, sf=None,
                ws=FAKE)
    ptrs.update(over)
    vp = lambda x: None if x is None else ctypes.c_void_p(x)
    fn = lib.gdn_prefill if kind == "gdn" else lib.kda_prefill
    rc = fn(vp(ptrs["q"]), vp(ptrs["k"]), vp(ptrs["v"]), vp(ptrs["g"]), vp(ptrs["beta"]),
            vp(ptrs["s0"]), vp(ptrs["cu"]), N, T, Hqk, Hv, Dk, Dv, 1.0, dtype, vp(ptrs["o"]),
            vp(ptrs["sf"]), vp(ptrs["ws"]), ws_bytes, None)
    return rc, lib.hagdn_last_error().decode()


@needs_lib
@pytest.mark.parametrize("kind", ["gdn", "kda"])
def test_host_validation(kind):
    lib = P.load_library()
    EINVAL, EUNSUP, EWS = 1, 2, 3
    assert _call(lib, kind, q=None)[0] == EINVAL
    assert _call(lib, kind, o=None)[0] == EINVAL
    assert _call(lib, kind, cu=None)[0] == EINVAL
    assert _call(lib, kind, ws=None)[0] == EINVAL
    assert _call(lib, kind, N=0)[0] == EINVAL
    assert _call(lib, kind, T=-5)[0] == EINVAL
    assert _call(lib, kind, Hqk=2, Hv=3)[0] == EINVAL
    assert _call(lib, kind, Dk=32)[0] == EUNSUP
    assert _call(lib, kind, Dv=256)[0] == EUNSUP
    assert _call(lib, kind, dtype=2)[0] == EUNSUP
    assert _call(lib, kind, q=FAKE + 8)[0] == EINVAL            # misaligned
    assert _call(lib, kind, s0=FAKE + 4, sf=FAKE + 4)[0] == EINVAL
    assert _call(lib, kind, g=FAKE + 2)[0] == EINVAL
    rc, msg = _call(lib, kind, ws_bytes=64)
    assert rc == EWS and "workspace too small" in msg
    # s_final overlapping s0 without aliasing it exactly
    assert _call(lib, kind, s0=FAKE, sf=FAKE + 64)[0] == EINVAL


@needs_lib
def test_profile_requires_begin():
    lib = P.load_library()
    arr = (ctypes.c_double * 4)()
    calls = ctypes.c_int()
    assert lib.hagdn_profile_end(arr, 4, ctypes.byref(calls)) == 1
    assert lib.hagdn_profile_begin(0) == 1


@needs_lib
def test_segment_rule_depends_on_the_cu_count():
    """The automatic segment length is a function of the device's compute
    units: half the walks' share of the CUs moves the threshold, and L puts
    about one segment workgroup on each CU."""
    # 16 heads x 8 column tiles = 128 walk workgroups
    assert P.segment_chunks_for(1, 7680, 16, 128, 256) == 12        # 120 chunks on 256 CUs: segments
    assert P.segment_chunks_for(1, 7680, 16, 128, 128) == 120       # on 128 CUs the walks fill it
    assert P.segment_chunks_for(1, 32768, 16, 128, 256) == 32       # 512 chunks: L = 512 x 16 / 256
    assert P.segment_chunks_for(1, 32768, 16, 128, 128) == 64       # L = 512 x 16 / 128
    assert P.segment_chunks_for(1, 32768, 16, 128, 80) == 103       # an 80-CU partition
    assert P.segment_chunks_for(1, 32768, 16, 128, 64) == 512       # threshold 624 chunks: whole
    assert P.segment_chunks_for(1, 8192, 16, 128, 256, kind="kda") == 8
    assert P.segment_chunks_for(1, 8192, 16, 128, 128, kind="kda") == 128
    with pytest.raises(P.HagdnError):
        P.segment_chunks_for(1, 8192, 16, 128, 0)
    # with no device to query (this host) the queries answer for 256 CUs
    import torch
    if not torch.cuda.is_available():
        assert P.segment_chunks(1, 32768, 16, 128) == P.segment_chunks_for(1, 32768, 16, 128, 256)


@needs_lib
def test_overlap_rule():
    """Which calls take the overlapped launch: GDN in bf16 with d_k = d_v = 128,
    chains walked whole, walks on at most half the CUs of a device of 8 XCDs,
    and (by default) more chunk-local blocks than one round of 3 per CU."""
    bf, f32 = P.HAGDN_BF16, P.HAGDN_F32
    assert P.overlap_for(1, 4096, 16, 128, 128, bf, "gdn", 256)           # 1040 blocks > 768
    assert P.overlap_for(1, 6144, 16, 128, 128, bf, "gdn", 256)
    assert not P.overlap_for(1, 2048, 16, 128, 128, bf, "gdn", 256)       # 528 blocks: one round
    assert not P.overlap_for(1, 4096, 8, 128, 128, bf, "gdn", 256)        # 520 blocks
    assert not P.overlap_for(1, 4096, 16, 128, 128, bf, "kda", 256)       # no KDA instance
    assert not P.overlap_for(1, 4096, 16, 128, 128, f32, "gdn", 256)      # no fp32 instance
    assert not P.overlap_for(1, 4096, 16, 64, 128, bf, "gdn", 256)        # no d_k = 64 instance
    assert not P.overlap_for(1, 4096, 32, 128, 128, bf, "gdn", 256)       # 256 walks: every CU
    assert not P.overlap_for(1, 32768, 16, 128, 128, bf, "gdn", 256)      # segment maps
    assert not P.overlap_for(1, 4096, 16, 128, 128, bf, "gdn", 128)       # fewer than 8 x 32 CUs
    assert not P.overlap_for(1, 0, 16, 128, 128, bf, "gdn", 256)          # nothing to launch
    try:
        P.set_overlap(True, force=True)
        assert P.overlap_for(1, 2048, 16, 128, 128, bf, "gdn", 256)
        assert P.overlap_for(5, 900, 2, 128, 128, bf, "gdn", 256)
        assert not P.overlap_for(1, 4096, 16, 128, 128, bf, "kda", 256)
        P.set_overlap(False)
        assert not P.overlap_for(1, 4096, 16, 128, 128, bf, "gdn", 256)
    finally:
        P.set_overlap(True)
    with pytest.raises(P.HagdnError):
        P.overlap_for(1, 4096, 16, 128, 128, bf, "gdn", 0)


def test_segment_length_knob():
    import paper_2609_32114_amd as P
    P.load_library()

    def seg_len(N, T, Hv, Dv, dtype=None, kind="gdn"):  # the rule on a 256-CU device
        return P.segment_chunks_for(N, T, Hv, Dv, 256, dtype, kind)

    try:
        # automatic (for a 256-CU device): short chains stay one segment; long
        # ones get about one segment workgroup per CU (n Hv / 256 chunks, at least 12)
        assert seg_len(1, 256, 1, 64) == 4
        assert seg_len(1, 0, 1, 64) == 1
        assert seg_len(1, 4096, 16, 128) == 64
        assert seg_len(1, 7616, 16, 128) == 119    # below 120 chunks: whole
        assert seg_len(1, 7680, 16, 128) == 12     # 120 chunks
        assert seg_len(1, 9216, 16, 128) == 12     # 144 chunks
        assert seg_len(1, 12288, 16, 128) == 12
        assert seg_len(1, 16384, 16, 128) == 16
        assert seg_len(1, 32768, 16, 128) == 32
        assert seg_len(1, 131072, 16, 128) == 128  # 2048 chunks
        assert seg_len(1, 16384, 32, 128) == 256   # 256 walk workgroups: threshold 288
        assert seg_len(1, 18368, 32, 128) == 287
        assert seg_len(1, 18432, 32, 128) == 36    # 288 chunks: 288 x 32 / 256
        assert seg_len(8, 34816, 32, 128) == 544   # short average chains: whole
        # KDA segments from 112 chunks, L at least 8
        assert seg_len(1, 5568, 16, 128, kind="kda") == 87
        assert seg_len(1, 5632, 16, 128, kind="kda") == 8
        assert seg_len(1, 8192, 16, 128, kind="kda") == 8
        assert seg_len(1, 12288, 16, 128, kind="kda") == 12
        assert seg_len(1, 8192, 16, 128, kind="gdn") == 12
        assert seg_len(1, 6144, 16, 128, kind="gdn") == 96
        with pytest.raises(ValueError):
            seg_len(1, 8192, 16, 128, kind="mamba")
        P.set_segment_chunks(8)
        auto = seg_len(1, 4096, 16, 128)
        assert auto == 8
        ws_auto = P.workspace_size("gdn", 1, 4096, 16, 16, 128, 128, P.HAGDN_BF16)  # L = 8
        P.set_segment_chunks(2)
        assert seg_len(1, 4096, 16, 128) == 2
        ws_small = P.workspace_size("gdn", 1, 4096, 16, 16, 128, 128, P.HAGDN_BF16)
        assert ws_small > ws_auto  # more segment maps
        P.set_segment_chunks(64)   # one segment: no maps at all
        ws_one = P.workspace_size("gdn", 1, 4096, 16, 16, 128, 128, P.HAGDN_BF16)
        assert ws_one < ws_auto
        with pytest.raises(P.HagdnError):
            P.set_segment_chunks(-1)
        # the cap: 64 L Hv Dv elements stay below 2 GiB, forced or automatic
        import torch
        P.set_segment_chunks(1 << 20)
        assert seg_len(1, 4096, 16, 128) == 8191                      # bf16: 2^31 / 256 KiB
        assert seg_len(1, 4096, 16, 128, torch.float32) == 4095       # fp32: 2^31 / 512 KiB
        assert seg_len(1, 32832, 128, 128, torch.float32) == 511
        assert seg_len(1, 4096, 65535, 128, torch.float32) == 1       # 64 rows: 2147450880 B
        P.set_segment_chunks(0)
        L = seg_len(4096, 4096 * 2048, 16, 128)   # short chains, 8M tokens: whole, then capped
        assert L == 8191 and 64 * L * 16 * 128 * 2 < 2 ** 31 <= 64 * (L + 1) * 16 * 128 * 2
        assert seg_len(1, 32832, 128, 128, torch.float32) == 511    # whole (1024 walks), capped
    finally:
        P.set_segment_chunks(0)
    assert P.segment_chunks_for(1, 4096, 16, 128, 256) == 64


def _call_ex(lib, kind="gdn", pre=0, **kw):
    ptrs = dict(q=FAKE, k=FAKE, v=FAKE, g=FAKE, beta=FAKE, s0=None, cu=FAKE, o=FAKE, sf=None, ws=FAKE)
    vp = lambda x: None if x is None else ctypes.c_void_p(x)
    fn = lib.gdn_prefill_ex if kind == "gdn" else lib.kda_prefill_ex
    rc = fn(vp(ptrs["q"]), vp(ptrs["k"]), vp(ptrs["v"]), vp(ptrs["g"]), vp(ptrs["beta"]),
            vp(ptrs["s0"]), vp(ptrs["cu"]), 1, 100, 1, 1, 64, 64, 1.0, 0, pre, vp(ptrs["o"]),
            vp(ptrs["sf"]), vp(ptrs["ws"]), kw.get("ws_bytes", 64), None)
    return rc, lib.hagdn_last_error().decode()


@needs_lib
@pytest.mark.parametrize("kind", ["gdn", "kda"])
def test_prefill_ex_rejects_unknown_flags(kind):
    lib = P.load_library()
    rc, msg = _call_ex(lib, kind, pre=8)
    assert rc == 1 and "preprocessing" in msg
    # valid flags pass the flag check and stop at the (too small) workspace
    assert _call_ex(lib, kind, pre=7)[0] == 3


def _call_dec(lib, kind="gdn", N=4, Hqk=1, Hv=1, Dk=64, Dv=64, dtype=0, pre=0, num_slots=4, **over):
    ptrs = dict(q=FAKE, k=FAKE, v=FAKE, g=FAKE, beta=FAKE, state=FAKE, slots=None, o=FAKE)
    ptrs.update(over)
    vp = lambda x: None if x is None else ctypes.c_void_p(x)
    fn = lib.gdn_decode if kind == "gdn" else lib.kda_decode
    rc = fn(vp(ptrs["q"]), vp(ptrs["k"]), vp(ptrs["v"]), vp(ptrs["g"]), vp(ptrs["beta"]),
            vp(ptrs["state"]), vp(ptrs["slots"]), num_slots, N, Hqk, Hv, Dk, Dv, 1.0, dtype, pre,
            vp(ptrs["o"]), None)
    return rc, lib.hagdn_last_error().decode()


@needs_lib
@pytest.mark.parametrize("kind", ["gdn", "kda"])
def test_decode_host_validation(kind):
    lib = P.load_library()
    EINVAL, EUNSUP = 1, 2
    assert _call_dec(lib, kind, N=0)[0] == 0            # no-op, nothing launched
    assert _call_dec(lib, kind, N=-1)[0] == EINVAL
    assert _call_dec(lib, kind, state=None)[0] == EINVAL
    assert _call_dec(lib, kind, o=None)[0] == EINVAL
    assert _call_dec(lib, kind, Hqk=2, Hv=3)[0] == EINVAL
    assert _call_dec(lib, kind, Dk=96)[0] == EUNSUP
    assert _call_dec(lib, kind, dtype=5)[0] == EUNSUP
    assert _call_dec(lib, kind, pre=16)[0] == EINVAL
    assert _call_dec(lib, kind, state=FAKE + 4)[0] == EINVAL   # misaligned
    assert _call_dec(lib, kind, slots=FAKE + 2)[0] == EINVAL
    assert _call_dec(lib, kind, slots=FAKE, num_slots=0)[0] == EINVAL
