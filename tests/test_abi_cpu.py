"""The C ABI library on a host without a GPU: it loads, exports every entry
point that include/convfirst.h declares, and rejects bad arguments before any
HIP call.  No compute call is made here."""
import ctypes
import os
import re

import pytest

import paper_2404_03617_amd as cf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "convfirst.h")

pytestmark = pytest.mark.skipif(not os.path.exists(cf.library_path()),
                                reason="libconvfirst.so not built")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(cf_[a-z0-9_]+)\s*\(", src)))


def test_header_declares_the_binding_symbols():
    assert set(declared_functions()) == set(cf.EXPORTED_SYMBOLS)


def test_library_exports_every_declared_symbol():
    L = ctypes.CDLL(cf.library_path())
    for name in declared_functions():
        assert hasattr(L, name), name


def test_abi_version_and_status_strings():
    L = cf.lib()
    assert L.cf_abi_version() == 1
    for s, name in enumerate(["CF_OK", "CF_ERR_INVALID", "CF_ERR_UNSUPPORTED", "CF_ERR_WORKSPACE",
                              "CF_ERR_HIP"]):
        assert L.cf_status_string(s).decode() == name


# Fake, aligned, non-overlapping "device" addresses: validation never touches them.
X, Y, WS = 0x10000000, 0x20000000, 0x30000000
DW, W1, W2 = 0x40000000, 0x41000000, 0x42000000


def params(**kw):
    base = dict(dw_w=DW, dw_scale=None, dw_bias=None, w1=W1, s1=None, b1=None, w2=W2, s2=None,
                b2=None)
    base.update(kw)
    return cf._BlockParams(**base)


def block(x=X, y=Y, p=None, N=1, H=8, W=8, C=64, E=4, k=3, dt=0, act=0):
    p = params() if p is None else p
    return cf.lib().cf_block_forward(x, y, ctypes.byref(p), N, H, W, C, E, k, dt, act, None)


@pytest.mark.parametrize("kw,status", [
    (dict(x=None), cf.CF_ERR_INVALID),
    (dict(y=None), cf.CF_ERR_INVALID),
    (dict(p=params(dw_w=None)), cf.CF_ERR_INVALID),
    (dict(p=params(w1=None)), cf.CF_ERR_INVALID),
    (dict(p=params(w2=None)), cf.CF_ERR_INVALID),
    (dict(N=0), cf.CF_ERR_INVALID),
    (dict(H=-1), cf.CF_ERR_INVALID),
    (dict(E=0), cf.CF_ERR_INVALID),
    (dict(k=2), cf.CF_ERR_INVALID),
    (dict(k=9), cf.CF_ERR_INVALID),
    (dict(dt=7), cf.CF_ERR_INVALID),
    (dict(act=5), cf.CF_ERR_INVALID),
    (dict(x=X + 8), cf.CF_ERR_INVALID),                      # misaligned
    (dict(p=params(b1=W1 + 4)), cf.CF_ERR_INVALID),          # misaligned bias
    (dict(y=X + 64), cf.CF_ERR_INVALID),                     # overlaps x
    (dict(C=48), cf.CF_ERR_UNSUPPORTED),
    (dict(C=96), cf.CF_ERR_UNSUPPORTED),
    (dict(W=4096), cf.CF_ERR_UNSUPPORTED),                   # halo does not fit LDS
])
def test_block_forward_rejects(kw, status):
    assert block(**kw) == status
    assert cf.lib().cf_last_error().decode().startswith("cf_block_forward")


def test_workspace_queries():
    L = cf.lib()
    P = 2 * 5 * 7
    assert L.cf_stage_workspace_bytes(1, 2, 5, 7, 64, 0) == 0
    assert L.cf_stage_workspace_bytes(3, 2, 5, 7, 64, 0) == (P * 64 * 2 + 255) // 256 * 256
    # C = 512 fp16: room for fp32 partials of up to 4 hidden groups (recommended size)
    assert L.cf_stage_workspace_bytes(1, 2, 5, 7, 512, 0) == 4 * P * 512 * 4
    assert L.cf_stage_workspace_bytes(2, 2, 5, 7, 512, 0) == P * 512 * 2 + 4 * P * 512 * 4
    assert L.cf_stage_workspace_bytes(2, 2, 5, 7, 512, 1) == P * 512 * 2
    need = L.cf_unfused_workspace_bytes(2, 5, 7, 64, 4, 0)
    assert need >= P * 64 * 2 + P * 256 * 2
    assert L.cf_split_workspace_bytes(1, 7, 7, 512, 4, 8) == 8 * 49 * 512 * 4


def test_stage_and_unfused_and_split_reject_short_workspace():
    L = cf.lib()
    p = params()
    arr = (cf._BlockParams * 2)(p, p)
    assert L.cf_stage_forward(X, Y, WS, 16, arr, 2, 1, 8, 8, 64, 4, 3, 0, 0, None) == cf.CF_ERR_WORKSPACE
    assert L.cf_stage_forward(X, Y, None, 0, arr, 2, 1, 8, 8, 64, 4, 3, 0, 0, None) == cf.CF_ERR_INVALID
    assert L.cf_stage_forward(X, Y, X, 1 << 20, arr, 2, 1, 8, 8, 64, 4, 3, 0, 0, None) == cf.CF_ERR_INVALID
    assert L.cf_block_forward_unfused(X, Y, WS, 16, ctypes.byref(p), 1, 8, 8, 64, 4, 3, 0, 0,
                                      None) == cf.CF_ERR_WORKSPACE
    assert L.cf_block_forward_split(X, Y, WS, 16, ctypes.byref(p), 1, 8, 8, 64, 4, 3, 2, 0, 0,
                                    None) == cf.CF_ERR_WORKSPACE
    # groups must divide E*C/32 = 8
    assert L.cf_block_forward_split(X, Y, WS, 1 << 30, ctypes.byref(p), 1, 8, 8, 64, 4, 3, 3, 0, 0,
                                    None) == cf.CF_ERR_INVALID


def test_downsample_rejects():
    L = cf.lib()
    dp = cf._DownParams(w=W1, scale=None, bias=None)
    ok = dict(N=1, H=8, W=8, Cin=64, Cout=128)
    def call(x=X, y=Y, p=dp, N=1, H=8, W=8, Cin=64, Cout=128, dt=0):
        return L.cf_downsample_forward(x, y, ctypes.byref(p) if p is not None else None, N, H, W,
                                       Cin, Cout, dt, None)
    assert call(H=7) == cf.CF_ERR_UNSUPPORTED
    assert call(Cout=96) == cf.CF_ERR_UNSUPPORTED
    assert call(x=None) == cf.CF_ERR_INVALID
    assert call(p=cf._DownParams(w=None)) == cf.CF_ERR_INVALID
    assert call(y=X + 16) == cf.CF_ERR_INVALID
    assert call(dt=3) == cf.CF_ERR_INVALID


def _sigma(m):
    return 16 * (m >> 4) + 8 * ((m >> 2) & 1) + 4 * ((m >> 3) & 1) + (m & 3)


def _tau(m):
    return 16 * ((m >> 2) & 1) + 4 * (m >> 3) + (m & 3)


def test_c512_dma_layouts_are_conflict_free():
    """The C = 512 kernel's LDS weight layouts (restated from its DMA and
    fragment-read address formulas): every DMA instruction fills one
    contiguous KB at a 1040-byte pitch, every byte of the chunk has exactly one
    place, and each 16-lane group of an A-fragment read hits 16 distinct
    16-byte bank groups."""
    PITCH, C = 1040, 512
    assert sorted(_sigma(m) for m in range(32)) == list(range(32))
    assert sorted(_tau(m) for m in range(32)) == list(range(32))
    # W1: row r of the chunk (1 KB) is instruction r; fragment (ks, lane h, m) = row sigma(m), bytes 32 ks + 16 h
    seen = set()
    for r in range(32):
        for b in range(0, 2 * C, 16):
            a = r * PITCH + b
            assert a not in seen
            seen.add(a)
    for ks in range(C // 16):
        for h in range(2):
            for grp in (range(16), range(16, 32)):
                banks = {((_sigma(m) * PITCH + 32 * ks + 16 * h) // 16) % 16 for m in grp}
                assert len(banks) == 16
    # W2: instruction j = 8 * set + i; lane l -> slot l // 4 (block of the set slot // 4, row m = 4 i + slot % 4),
    # 16-byte piece l % 4 of the row's 64 bytes
    W2OFF = 32 * PITCH
    where = {}
    for j in range(32):
        st, i = j >> 3, j & 7
        for lane in range(64):
            sl, pc = lane >> 2, lane & 3
            o = (4 * st + (sl >> 2)) * 32 + _tau(4 * i + (sl & 3))
            key = (o, pc)
            assert key not in where
            where[key] = W2OFF + j * PITCH + 16 * lane
    assert len(where) == C * 4
    for cb in range(C // 32):
        for kk in range(2):
            for h in range(2):
                for grp in (range(16), range(16, 32)):
                    addrs = []
                    for m in grp:
                        # the kernel's read address: per-lane base + (cb, kk) offset
                        a = W2OFF + (m >> 2) * PITCH + (m & 3) * 64 + 16 * h + (cb >> 2) * 8 * PITCH + (cb & 3) * 256 + 32 * kk
                        # it must be where the DMA put row cb*32 + tau(m), piece 2 kk + h
                        assert a == where[(cb * 32 + _tau(m), 2 * kk + h)]
                        addrs.append(a)
                    assert len({(a // 16) % 16 for a in addrs}) == 16


@pytest.mark.parametrize("C", [128, 256])
def test_pair_kernel_dma_layouts_map_fragments_without_conflicts(C):
    """The C = 128 / 256 pair kernel's weight buffers (restated from its DMA
    and fragment-read address formulas): every 16-byte piece of a step's 64 W1
    rows and C W2 row segments is copied to exactly one place, every fragment
    read finds there the W1 / W2 elements its MFMA needs, and each 16-lane
    group of a read hits 16 distinct 16-byte bank groups."""
    PITCH, RPI = 1040, 1024 // (2 * C)
    NIA, NIB = 64 // RPI, C // 8
    CBH, KST = C // 64, C // 16
    # A: instruction I, lane l -> 16-row group g, piece p of W1 row 32 (I >> 4) + (I & 15) + 16 g of the step
    per = 64 // RPI
    where_a = {}
    for I in range(NIA):
        for lane in range(64):
            g, p = lane // per, lane % per
            key = (32 * (I >> 4) + (I & 15) + 16 * g, p)
            assert key not in where_a
            where_a[key] = I * PITCH + 16 * lane
    assert len(where_a) == 64 * (C // 8)
    for r in range(2):  # the chunk a wave expands
        for ks in range(KST):
            for h in range(2):
                for grp in (range(16), range(16, 32)):
                    addrs = []
                    for m in grp:
                        rho = _sigma(m)
                        q, u = 2 * r + (rho >> 4), rho & 15
                        a = (u + 16 * (q // RPI)) * PITCH + (q % RPI) * 2 * C + 16 * h + 32 * ks
                        assert a == where_a[(32 * r + rho, 2 * ks + h)]
                        addrs.append(a)
                    assert len({(a // 16) % 16 for a in addrs}) == 16
    # B: instruction I = 8 set + i, lane l -> slot l >> 3, piece l & 7 of the step's 64 columns of W2 row
    # (2 set + bb) * 32 + tau(16 mhi + 2 i + mlo); the kernel forms that row as a wave-uniform
    # 64 set + T(i) plus the lane's 32 bb + 8 mhi + mlo
    def T(i):
        return 16 * ((i >> 1) & 1) + 4 * (i >> 2) + 2 * (i & 1)
    where_b = {}
    for I in range(NIB):
        st, i = I >> 3, I & 7
        for lane in range(64):
            slot, piece = lane >> 3, lane & 7
            bb, mhi, mlo = slot >> 2, (slot >> 1) & 1, slot & 1
            o = (2 * st + bb) * 32 + _tau(16 * mhi + 2 * i + mlo)
            assert o == 64 * st + T(i) + 32 * bb + 8 * mhi + mlo
            assert (o, piece) not in where_b
            where_b[(o, piece)] = I * PITCH + 16 * lane
    assert len(where_b) == C * 8
    for r in range(2):  # the output half a wave projects
        for c in range(CBH):
            for j in range(2):
                for kk in range(2):
                    for h in range(2):
                        for grp in (range(16), range(16, 32)):
                            addrs = []
                            for m in grp:
                                base = ((m >> 1) & 7) * PITCH + (2 * (m >> 4) + (m & 1)) * 128 + 16 * h \
                                    + 4 * CBH * r * PITCH
                                a = base + 8 * (c >> 1) * PITCH + 4 * (c & 1) * 128 + 64 * j + 32 * kk
                                assert a == where_b[((CBH * r + c) * 32 + _tau(m), 4 * j + 2 * kk + h)]
                                addrs.append(a)
                            assert len({(a // 16) % 16 for a in addrs}) == 16


@pytest.mark.parametrize("C", [128, 256, 512])
def test_per_wave_copy_bases_match_the_layout_numbering(C):
    """The kernels issue a wave's copies from a per-wave base plus fixed
    offsets (restated here from their address formulas); wave wv's i-th copy
    must be exactly layout instruction I = wv + NW i, whose source row the
    layout tests above check.  Pair kernel (C = 128 / 256, NW = 8): A copy i
    reads W1 row wv + 32 (i >> 1) + 8 (i & 1) of the step, B copy i output
    row T(wv) + 64 i.  C = 512 ring (NW = 4): W1 copy q reads chunk row
    wv + 4 q, W2 copy q output row R(wv) + 128 (q >> 1) + 8 (q & 1)."""
    def T(i):
        return 16 * ((i >> 1) & 1) + 4 * (i >> 2) + 2 * (i & 1)
    PITCH = 1040
    if C < 512:
        NW, RPI = 8, 1024 // (2 * C)
        NIA, NIB = 64 // RPI, C // 8
        covered_a, covered_b = set(), set()
        for wv in range(NW):
            for i in range(NIA // NW):
                I = wv + NW * i
                assert wv + 32 * (i >> 1) + 8 * (i & 1) == 32 * (I >> 4) + (I & 15)
                assert wv * PITCH + i * NW * PITCH == I * PITCH  # LDS destination
                covered_a.add(I)
            for i in range(NIB // NW):
                I = wv + NW * i
                assert T(wv) + 64 * i == 64 * (I >> 3) + T(I & 7)
                covered_b.add(I)
        assert covered_a == set(range(NIA)) and covered_b == set(range(NIB))
    else:
        NWS, NI1, NI2 = 4, 32, 2 * (C // 32)
        covered1, covered2 = set(), set()
        for wv in range(NWS):
            R = 16 * (wv & 1) + 4 * (wv >> 1)
            for q in range(NI1 // NWS):
                covered1.add(wv + NWS * q)
            for q in range(NI2 // NWS):
                j = wv + NWS * q
                st, i = j >> 3, j & 7
                assert R + 128 * (q >> 1) + 8 * (q & 1) == 128 * st + 16 * (i & 1) + 4 * (i >> 1)
                covered2.add(j)
        assert covered1 == set(range(NI1)) and covered2 == set(range(NI2))


def test_c64_next_halo_rows_and_masks():
    """The C = 64 kernel's per-tile halo set-up (restated from next_halo and
    issue_row): buffer row r holds image row g_lo - PAD + r; rows rlo ..
    rlo + span - 1 are exactly the ones inside the images and the tile; the
    base row rlo is always a real image row (a skipped copy reads it); and the
    branch-free mask ~(d >> 31) & ((d - span) >> 31) (32-bit arithmetic
    shifts) selects exactly 0 <= d < span."""
    def asr(v):  # 32-bit arithmetic shift right by 31
        v &= 0xFFFFFFFF
        return 0xFFFFFFFF if v & 0x80000000 else 0
    for PAD in (0, 1, 2, 3):
        for NH in (1, 2, 5, 56, 7168):
            for g_lo in sorted({0, 1, 2, NH // 2, NH - 2, NH - 1} & set(range(NH))):
                for rows in (0, 1, 4, 10, 14):
                    rlo = max(PAD - g_lo, 0)
                    rhi = min(NH - g_lo + PAD, rows)
                    if rhi < rlo:
                        rhi = rlo
                    span = rhi - rlo
                    assert 0 <= g_lo - PAD + rlo < NH
                    for r in range(rows + 3):
                        want = r < rows and 0 <= g_lo - PAD + r < NH
                        d = r - rlo
                        okm = (~asr(d) & 0xFFFFFFFF) & asr(d - span)
                        assert (okm == 0xFFFFFFFF) == want and okm in (0, 0xFFFFFFFF)


def test_split_noalloc_rejects_before_any_launch():
    """The allocation-free split entry point: partials beyond its static
    scratch return CF_ERR_WORKSPACE, bad groups CF_ERR_INVALID, both on the
    host before any HIP call."""
    L = cf.lib()
    p = params()
    # N = 3, 14x14, C = 256, E = 4, 32 groups: 3*196*256*4*32 bytes = 19.3 MB > 16 MiB
    assert L.cf_block_forward_split_noalloc(X, Y, ctypes.byref(p), 3, 14, 14, 256, 4, 3, 32, 0, 0,
                                            None) == cf.CF_ERR_WORKSPACE
    assert "scratch" in L.cf_last_error().decode()
    assert L.cf_block_forward_split_noalloc(X, Y, ctypes.byref(p), 1, 8, 8, 64, 4, 3, 3, 0, 0,
                                            None) == cf.CF_ERR_INVALID
    assert L.cf_block_forward_split_noalloc(None, Y, ctypes.byref(p), 1, 8, 8, 64, 4, 3, 2, 0, 0,
                                            None) == cf.CF_ERR_INVALID


def test_gblock_forward_rejects():
    """The paper's block entry point: every check happens on the host."""
    L = cf.lib()
    GW = 0x43000000

    def call(x=X, y=Y, gw=GW, N=1, H=8, W=8, C=64, E=6, k=3, dt=0, act=1, **kw):
        p = cf._GBlockParams(gw_w=gw, gw_scale=None, gw_bias=None, w1=W1, s1=None, b1=None, w2=W2, s2=None,
                             b2=None)
        for f, v in kw.items():
            setattr(p, f, v)
        return L.cf_gblock_forward(x, y, ctypes.byref(p), N, H, W, C, E, k, dt, act, None)

    assert call(gw=None) == cf.CF_ERR_INVALID
    assert call(x=None) == cf.CF_ERR_INVALID
    assert call(C=20) == cf.CF_ERR_INVALID          # not a multiple of the group width 8
    assert call(k=4) == cf.CF_ERR_INVALID
    assert call(act=9) == cf.CF_ERR_INVALID
    assert call(y=X + 32) == cf.CF_ERR_INVALID      # overlaps x
    assert call(b1=W1 + 4) == cf.CF_ERR_INVALID     # misaligned
    assert call(C=24) == cf.CF_ERR_UNSUPPORTED      # multiple of 8, not of 16
    assert call(C=128) == cf.CF_ERR_UNSUPPORTED
    assert call(C=256) == cf.CF_ERR_UNSUPPORTED
    assert call(k=5) == cf.CF_ERR_UNSUPPORTED
    assert call(H=1, W=6_000_000, y=0x400000000) == cf.CF_ERR_UNSUPPORTED  # 32-bit row offsets
    assert L.cf_last_error().decode().startswith("cf_gblock_forward")


def test_microbatch_stage_workspace_and_rejects():
    L = cf.lib()
    # explicit micro-batch: two buffers of m images for depth > 2, one for depth 2, none for one block
    img = 7 * 9 * 64 * 2
    assert L.cf_stage_microbatch_workspace_bytes(3, 10, 7, 9, 64, 4, 0) == 2 * ((4 * img + 255) // 256 * 256)
    assert L.cf_stage_microbatch_workspace_bytes(2, 10, 7, 9, 64, 4, 0) == (4 * img + 255) // 256 * 256
    assert L.cf_stage_microbatch_workspace_bytes(1, 10, 7, 9, 64, 4, 0) == 0
    # a micro-batch larger than the batch is the batch
    assert L.cf_stage_microbatch_workspace_bytes(2, 3, 7, 9, 64, 50, 0) == (3 * img + 255) // 256 * 256
    # default: one micro-batch's input and output within 128 MiB (56x56x64 fp16: 167 images,
    # so the whole batch of 128; at 224x224x64, 10 images)
    assert L.cf_stage_microbatch_workspace_bytes(2, 128, 56, 56, 64, 0, 0) == 128 * 56 * 56 * 64 * 2
    assert L.cf_stage_microbatch_workspace_bytes(2, 128, 224, 224, 64, 0, 0) == 10 * 224 * 224 * 64 * 2
    p = params()
    arr = (cf._BlockParams * 3)(p, p, p)
    args = (arr, 3, 10, 7, 9, 64, 4, 3, 4, 0, 0, None)
    assert L.cf_stage_forward_microbatch(X, Y, WS, 16, *args) == cf.CF_ERR_WORKSPACE
    assert L.cf_stage_forward_microbatch(X, Y, None, 0, *args) == cf.CF_ERR_INVALID
    assert L.cf_stage_forward_microbatch(X, Y, X, 1 << 20, *args) == cf.CF_ERR_INVALID   # ws overlaps x
    assert L.cf_stage_forward_microbatch(X, Y, WS, 1 << 30, arr, 0, 10, 7, 9, 64, 4, 3, 4, 0, 0,
                                         None) == cf.CF_ERR_INVALID


def test_mbconv_forward_rejects():
    """The MBConv + SE entry point: every check happens on the host, and the
    workspace size is a function of the shape (one image in flight without a
    device to ask)."""
    L = cf.lib()
    GW, WR, WE = 0x43000000, 0x44000000, 0x45000000

    def need(N, H, W, C, E, R):
        G = E * C // 64
        return 256 + 2048 * 128 + (N * G * R * 4 + 255) // 256 * 256 + 2 * H * W * E * C * 2

    def call(x=X, y=Y, ws=WS, ws_bytes=1 << 30, N=2, H=8, W=8, C=64, E=4, R=16, k=3, dt=0, launch=0, **kw):
        p = cf._MBConvParams(w1=W1, s1=None, b1=None, gw_w=GW, s2=None, b2=None, wr=WR, br=None, we=WE, be=None,
                             w2=W2, s3=None, b3=None)
        for f, v in kw.items():
            setattr(p, f, v)
        return L.cf_mbconv_forward(x, y, ws, ws_bytes, ctypes.byref(p), N, H, W, C, E, R, k, dt, launch, None)

    assert L.cf_mbconv_workspace_bytes(2, 8, 8, 64, 4, 16, 0) >= need(2, 8, 8, 64, 4, 16)
    assert L.cf_mbconv_workspace_bytes(2, 17, 8, 64, 4, 16, 0) == 0     # H > 16
    assert L.cf_mbconv_workspace_bytes(2, 8, 8, 48, 1, 16, 0) == 0      # E*C not a multiple of 64
    assert L.cf_mbconv_workspace_bytes(2, 8, 8, 64, 4, 300, 0) == 0     # R > 256
    assert call(x=None) == cf.CF_ERR_INVALID
    assert call(gw_w=None) == cf.CF_ERR_INVALID
    assert call(we=None) == cf.CF_ERR_INVALID
    assert call(R=0) == cf.CF_ERR_INVALID
    assert call(C=20) == cf.CF_ERR_INVALID           # not a multiple of the group width
    assert call(k=4) == cf.CF_ERR_INVALID
    assert call(dt=5) == cf.CF_ERR_INVALID
    assert call(launch=2) == cf.CF_ERR_INVALID
    assert call(y=X + 32) == cf.CF_ERR_INVALID       # overlaps x without being x
    assert call(b3=W1 + 4) == cf.CF_ERR_INVALID      # misaligned
    assert call(ws=X) == cf.CF_ERR_INVALID           # ws overlaps x
    assert call(k=5) == cf.CF_ERR_UNSUPPORTED
    assert call(H=17) == cf.CF_ERR_UNSUPPORTED
    assert call(W=32) == cf.CF_ERR_UNSUPPORTED
    assert call(C=40, E=8) == cf.CF_ERR_UNSUPPORTED  # C not a multiple of 16
    assert call(C=48, E=1) == cf.CF_ERR_UNSUPPORTED  # E*C not a multiple of 64
    assert call(R=257) == cf.CF_ERR_UNSUPPORTED
    assert call(C=512, E=16) == cf.CF_ERR_UNSUPPORTED   # E*C > 4096
    assert call(C=1024, E=1) == cf.CF_ERR_UNSUPPORTED   # W1 rows, gates, staged V and vectors exceed 160 KB of LDS
    assert call(C=512, E=8) == cf.CF_ERR_UNSUPPORTED
    n = need(2, 8, 8, 64, 4, 16)
    assert call(ws_bytes=n - 1) == cf.CF_ERR_WORKSPACE
    assert call(ws=None, ws_bytes=0) == cf.CF_ERR_WORKSPACE
    assert L.cf_last_error().decode().startswith("cf_mbconv_forward")


def test_mbconv_s2_forward_rejects():
    """The stride-2 MBConv entry point: the stride-1 checks plus K, the 2 x 2
    minimum image (reflect padding) and no overlap of x and y at all; its
    workspace holds the down-sampled map."""
    L = cf.lib()
    GW, WR, WE = 0x43000000, 0x44000000, 0x45000000

    def need(N, H, W, C, E, R):
        G = E * C // 64
        return 256 + 2048 * 128 + (N * G * R * 4 + 255) // 256 * 256 + 2 * ((H + 1) // 2) * ((W + 1) // 2) * E * C * 2

    def call(x=X, y=Y, ws=WS, ws_bytes=1 << 30, N=2, H=8, W=8, C=64, E=4, R=16, K=128, k=3, dt=0, launch=0, **kw):
        p = cf._MBConvParams(w1=W1, s1=None, b1=None, gw_w=GW, s2=None, b2=None, wr=WR, br=None, we=WE, be=None,
                             w2=W2, s3=None, b3=None)
        for f, v in kw.items():
            setattr(p, f, v)
        return L.cf_mbconv_s2_forward(x, y, ws, ws_bytes, ctypes.byref(p), N, H, W, C, E, R, K, k, dt, launch, None)

    assert L.cf_mbconv_s2_workspace_bytes(2, 8, 8, 64, 4, 16, 128, 0) >= need(2, 8, 8, 64, 4, 16)
    assert L.cf_mbconv_s2_workspace_bytes(2, 7, 5, 64, 4, 16, 32, 1) >= need(2, 7, 5, 64, 4, 16)
    assert L.cf_mbconv_s2_workspace_bytes(2, 8, 8, 64, 4, 16, 0, 0) == 0      # K = 0
    assert L.cf_mbconv_s2_workspace_bytes(2, 8, 8, 64, 4, 16, 40, 0) == 0     # K not a multiple of 16
    assert L.cf_mbconv_s2_workspace_bytes(2, 1, 8, 64, 4, 16, 64, 0) == 0     # H < 2
    assert L.cf_mbconv_s2_workspace_bytes(2, 17, 8, 64, 4, 16, 64, 0) == 0    # H > 16
    assert call(x=None) == cf.CF_ERR_INVALID
    assert call(w2=None) == cf.CF_ERR_INVALID
    assert call(K=0) == cf.CF_ERR_INVALID
    assert call(K=-16) == cf.CF_ERR_INVALID
    assert call(H=1) == cf.CF_ERR_INVALID           # reflect padding needs a second row
    assert call(W=1) == cf.CF_ERR_INVALID
    assert call(C=20) == cf.CF_ERR_INVALID
    assert call(k=4) == cf.CF_ERR_INVALID
    assert call(dt=5) == cf.CF_ERR_INVALID
    assert call(launch=2) == cf.CF_ERR_INVALID
    assert call(y=X) == cf.CF_ERR_INVALID            # no in-place form
    assert call(y=X + 4096) == cf.CF_ERR_INVALID     # y overlaps x
    assert call(s3=W1 + 4) == cf.CF_ERR_INVALID      # misaligned
    assert call(ws=X) == cf.CF_ERR_INVALID           # ws overlaps x
    assert call(k=5) == cf.CF_ERR_UNSUPPORTED
    assert call(K=40) == cf.CF_ERR_UNSUPPORTED       # not a multiple of 16
    assert call(H=17) == cf.CF_ERR_UNSUPPORTED
    assert call(C=48, E=1) == cf.CF_ERR_UNSUPPORTED
    assert call(C=512, E=4, H=16, W=16, K=512) == cf.CF_ERR_UNSUPPORTED  # V's LDS copy exceeds 160 KB
    n = need(2, 8, 8, 64, 4, 16)
    assert call(ws_bytes=n - 1) == cf.CF_ERR_WORKSPACE
    assert call(ws=None, ws_bytes=0) == cf.CF_ERR_WORKSPACE
    assert L.cf_last_error().decode().startswith("cf_mbconv_s2_forward")


def test_convfirst_s2_forward_rejects():
    """The stride-2 ConvFirst entry point: every check happens on the host."""
    L = cf.lib()
    GW = 0x43000000

    def call(x=X, y=Y, N=2, H=8, W=8, C=16, R=96, K=32, k=3, dt=0, act=1, **kw):
        p = cf._GBlockParams(gw_w=GW, gw_scale=None, gw_bias=None, w1=W1, s1=None, b1=None, w2=W2, s2=None,
                             b2=None)
        for f, v in kw.items():
            setattr(p, f, v)
        return L.cf_convfirst_s2_forward(x, y, ctypes.byref(p), N, H, W, C, R, K, k, dt, act, None)

    assert call(x=None) == cf.CF_ERR_INVALID
    assert call(w1=None) == cf.CF_ERR_INVALID
    assert call(R=0) == cf.CF_ERR_INVALID
    assert call(k=4) == cf.CF_ERR_INVALID
    assert call(H=1) == cf.CF_ERR_INVALID           # reflect padding needs a second row
    assert call(W=1) == cf.CF_ERR_INVALID
    assert call(C=20) == cf.CF_ERR_INVALID          # not a multiple of the group width
    assert call(dt=5) == cf.CF_ERR_INVALID
    assert call(act=7) == cf.CF_ERR_INVALID
    assert call(y=X + 1024) == cf.CF_ERR_INVALID    # y overlaps x
    assert call(s2=W1 + 4) == cf.CF_ERR_INVALID     # misaligned
    assert call(k=5) == cf.CF_ERR_UNSUPPORTED
    assert call(C=40) == cf.CF_ERR_UNSUPPORTED      # no kernel for C = 40
    assert call(C=128) == cf.CF_ERR_UNSUPPORTED
    assert call(R=104) == cf.CF_ERR_UNSUPPORTED     # R not a multiple of 16
    assert call(R=2048) == cf.CF_ERR_UNSUPPORTED
    assert call(K=36) == cf.CF_ERR_UNSUPPORTED      # K not a multiple of 8
    assert call(K=136) == cf.CF_ERR_UNSUPPORTED
    assert L.cf_last_error().decode().startswith("cf_convfirst_s2_forward")


def test_stem_entry_points_reject():
    """The stem and the stem + first block: every check happens on the host."""
    L = cf.lib()
    SW, GW = 0x46000000, 0x43000000

    def stem(x=X, y=Y, w=SW, N=2, Hin=16, Win=16, C=16, dt=0, **kw):
        p = cf._StemParams(w=w, scale=None, bias=None)
        for f, v in kw.items():
            setattr(p, f, v)
        return L.cf_stem_forward(x, y, ctypes.byref(p), N, Hin, Win, C, dt, None)

    def fused(x=X, y=Y, w=SW, gw=GW, N=2, Hin=16, Win=16, C=16, E=3, k=3, dt=0, act=1):
        sp = cf._StemParams(w=w, scale=None, bias=None)
        gp = cf._GBlockParams(gw_w=gw, gw_scale=None, gw_bias=None, w1=W1, s1=None, b1=None, w2=W2, s2=None, b2=None)
        return L.cf_stem_gblock_forward(x, y, ctypes.byref(sp), ctypes.byref(gp), N, Hin, Win, C, E, k, dt, act, None)

    assert stem(x=None) == cf.CF_ERR_INVALID
    assert stem(w=None) == cf.CF_ERR_INVALID
    assert stem(Hin=0) == cf.CF_ERR_INVALID
    assert stem(C=20) == cf.CF_ERR_INVALID            # not a multiple of 8
    assert stem(dt=3) == cf.CF_ERR_INVALID
    assert stem(y=X + 64) == cf.CF_ERR_INVALID        # overlaps the image
    assert stem(scale=W1 + 4) == cf.CF_ERR_INVALID    # misaligned
    assert stem(C=64) == cf.CF_ERR_UNSUPPORTED
    assert stem(C=40) == cf.CF_ERR_UNSUPPORTED
    assert L.cf_last_error().decode().startswith("cf_stem_forward")
    assert fused(gw=None) == cf.CF_ERR_INVALID
    assert fused(E=0) == cf.CF_ERR_INVALID
    assert fused(k=4) == cf.CF_ERR_INVALID
    assert fused(act=7) == cf.CF_ERR_INVALID
    assert fused(C=24) == cf.CF_ERR_UNSUPPORTED        # a paper stem width without a block kernel
    assert fused(k=5) == cf.CF_ERR_UNSUPPORTED
    assert L.cf_last_error().decode().startswith("cf_stem_gblock_forward")
