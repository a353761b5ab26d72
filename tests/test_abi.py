"""The C ABI on the CPU: the library loads without a GPU, exports every
function the header declares, and rejects invalid arguments before making
any HIP call (so nothing is launched and no output is touched)."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "vitattn.h")

va = pytest.importorskip("paper_2405_15780_amd")


def lib():
    try:
        return va.library()
    except ImportError as e:  # the library must be built before the tests run
        pytest.fail(str(e))


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(vitattn_\w+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert {"vitattn_fwd", "vitattn_bwd", "vitattn_bwd_workspace_bytes", "vitattn_status_str",
            "vitattn_version", "vitattn_fwd_kv", "vitattn_bwd_kv", "vitattn_merge"} <= set(names)
    raw = ctypes.CDLL(va.LIB_PATH)
    for n in names:
        assert hasattr(raw, n), n


def test_status_strings_and_version():
    assert va.version() == "0.3.0"
    for s in range(7):
        assert va.status_str(s).startswith("VITATTN")
    assert "unknown" in va.status_str(99)


def test_workspace_bytes():
    assert va.workspace_bytes(1, 2, 188416, 128) == 2 * 4 * 2 * 188416
    assert va.workspace_bytes(1, 1, 1, 64) == 512
    assert va.workspace_bytes(1, 1, 65, 64) == 1024
    assert va.workspace_bytes(1, 1, 8388351, 128) > 0
    assert va.workspace_bytes(1, 1, 8388352, 128) == 0
    assert va.workspace_bytes(1, 1, 0, 64) == 0
    assert va.workspace_bytes(1, 1, 10, 100) == 0
    assert va.workspace_bytes(1, 1, 10, 168) == 0
    assert va.workspace_bytes(1, 1, 10, 72) == 512


class Bufs:
    """Aligned host buffers standing in for device pointers: validation must
    reject the call before anything could dereference them."""

    def __init__(self, n=4096):
        self.arrays = [np.full(n, 7.0, dtype=np.float32) for _ in range(12)]
        for a in self.arrays:
            assert a.ctypes.data % 16 == 0

    def p(self, i):
        return self.arrays[i].ctypes.data

    def untouched(self):
        return all((a == 7.0).all() for a in self.arrays)


E_INVAL, E_UNSUP, E_WS = 1, 2, 3


def fwd(b, B=1, H=1, N=8, d=64, scale=0.125, override=None):
    ptrs = [b.p(i) for i in range(5)]
    if override:
        for i, val in override.items():
            ptrs[i] = val
    return lib().vitattn_fwd(*ptrs, B, H, N, d, scale, None)


@pytest.mark.parametrize("kw,expected", [
    (dict(B=0), E_INVAL), (dict(H=0), E_INVAL), (dict(N=0), E_INVAL), (dict(N=-5), E_INVAL),
    (dict(d=100), E_UNSUP), (dict(d=4), E_UNSUP), (dict(d=0), E_UNSUP), (dict(d=168), E_UNSUP),
    (dict(d=256), E_UNSUP),
    (dict(scale=float("nan")), E_INVAL), (dict(scale=float("inf")), E_INVAL), (dict(scale=0.0), E_INVAL),
    (dict(scale=-0.125), E_INVAL), (dict(B=65536, H=65536, N=2), E_INVAL),
    # B*H*N below 2^31 but 2*B*H*(N + 383) work-items past 2^32
    (dict(B=2, H=2_800_000, N=1, d=8), E_INVAL),
])
def test_fwd_rejects_bad_sizes_and_scale(kw, expected):
    b = Bufs()
    assert fwd(b, **kw) == expected
    assert b.untouched()


@pytest.mark.parametrize("which", range(5))
def test_fwd_rejects_null_and_misaligned_pointers(which):
    b = Bufs()
    assert fwd(b, override={which: None}) == E_INVAL
    assert fwd(b, override={which: b.p(which) + 8}) == E_INVAL
    assert b.untouched()


def bwd(b, B=1, H=1, N=8, d=64, scale=0.125, ws_bytes=None, override=None):
    ptrs = [b.p(i) for i in range(9)]
    if override:
        for i, val in override.items():
            if i < 9:
                ptrs[i] = val
    ws = b.p(9)
    if override and 9 in override:
        ws = override[9]
    wsb = va.workspace_bytes(max(B, 1), max(H, 1), max(N, 1), d if d in (64, 128) else 64) if ws_bytes is None \
        else ws_bytes
    return lib().vitattn_bwd(*ptrs, B, H, N, d, scale, ws, wsb, None)


@pytest.mark.parametrize("kw,expected", [
    (dict(N=0), E_INVAL), (dict(d=84), E_UNSUP), (dict(scale=float("nan")), E_INVAL),
    (dict(ws_bytes=31), E_WS), (dict(ws_bytes=0), E_WS), (dict(override={9: None}), E_WS),
    (dict(override={9: 12345}), E_WS),
    # launches past 2^32 work-items: the row-dot pass (8 per row at d = 8)
    # and the dK/dV kernel (4 per key row plus padding), with B*H*N < 2^31
    (dict(B=8, H=8, N=1 << 23, d=8, ws_bytes=1 << 40), E_INVAL),
    (dict(B=4, H=1_125_000, N=64, d=8, ws_bytes=1 << 40), E_INVAL),
])
def test_bwd_rejects_bad_arguments(kw, expected):
    b = Bufs()
    assert bwd(b, **kw) == expected
    assert b.untouched()


@pytest.mark.parametrize("which", range(9))
def test_bwd_rejects_null_pointers(which):
    b = Bufs()
    assert bwd(b, override={which: None}) == E_INVAL
    assert bwd(b, override={which: b.p(which) + 4}) == E_INVAL
    assert b.untouched()


def noalloc(b, B=1, H=1, N=8, d=64, scale=0.125, override=None):
    ptrs = [b.p(i) for i in range(9)]
    for i, val in (override or {}).items():
        ptrs[i] = val
    return lib().vitattn_bwd_noalloc(*ptrs, B, H, N, d, scale, None)


@pytest.mark.parametrize("kw,expected", [
    (dict(N=0), E_INVAL), (dict(d=84), E_UNSUP), (dict(scale=float("nan")), E_INVAL),
    (dict(override={3: None}), E_INVAL), (dict(override={8: 12346}), E_INVAL),
    # one row past the static scratch, and the same rows as B*H*N in another split
    (dict(N=va.VITATTN_NOALLOC_MAX_ROWS + 1), 6), (dict(B=2, H=2, N=va.VITATTN_NOALLOC_MAX_ROWS // 4 + 1), 6),
])
def test_bwd_noalloc_rejects_bad_arguments_before_any_hip_call(kw, expected):
    b = Bufs()
    assert noalloc(b, **kw) == expected
    assert b.untouched()
    assert "VITATTN_NOALLOC_MAX_ROWS" in va.status_str(6)


def test_bwd_stages_validate():
    b = Bufs()
    L = lib()
    wsb = va.workspace_bytes(1, 1, 8, 64)
    assert L.vitattn_bwd_rowdot(b.p(0), b.p(1), b.p(3), 1, 1, 8, 64, b.p(2), wsb - 1, None) == E_WS
    assert L.vitattn_bwd_rowdot(None, b.p(1), b.p(3), 1, 1, 8, 64, b.p(2), wsb, None) == E_INVAL
    assert L.vitattn_bwd_rowdot(b.p(0), b.p(1), None, 1, 1, 8, 64, b.p(2), wsb, None) == E_INVAL
    assert L.vitattn_bwd_dkdv(b.p(0), b.p(1), b.p(2), b.p(3), b.p(4), b.p(5), b.p(6), 1, 1, 8, 100, 0.1, b.p(7), wsb,
                              None) == E_UNSUP
    assert L.vitattn_bwd_dkdv(b.p(0), b.p(1), b.p(2), b.p(3), None, b.p(5), b.p(6), 1, 1, 8, 64, 0.1, b.p(7), wsb,
                              None) == E_INVAL
    assert L.vitattn_bwd_dq(b.p(0), b.p(1), b.p(2), b.p(3), b.p(4), b.p(5), 1, 1, 8, 64, -1.0, b.p(7), wsb,
                            None) == E_INVAL
    assert L.vitattn_bwd_dq(b.p(0), b.p(1), b.p(2), b.p(3), b.p(4), b.p(5), 1, 1, 8, 64, 0.1, b.p(7), 0,
                            None) == E_WS
    assert b.untouched()


def fwd_kv(b, B=1, H=1, Nq=8, Nk=5, d=64, scale=0.125, override=None):
    ptrs = [b.p(i) for i in range(5)]
    if override:
        for i, val in override.items():
            ptrs[i] = val
    return lib().vitattn_fwd_kv(*ptrs, B, H, Nq, Nk, d, scale, None)


@pytest.mark.parametrize("kw,expected", [
    (dict(Nk=0), E_INVAL), (dict(Nq=0), E_INVAL), (dict(Nk=-1), E_INVAL), (dict(d=76), E_UNSUP),
    (dict(Nk=8388352, d=128), E_INVAL), (dict(scale=float("nan")), E_INVAL),
    (dict(override={1: None}), E_INVAL), (dict(override={2: 4100}), E_INVAL),
])
def test_fwd_kv_rejects_bad_arguments(kw, expected):
    b = Bufs()
    assert fwd_kv(b, **kw) == expected
    assert b.untouched()


def bwd_kv(b, B=1, H=1, Nq=8, Nk=5, d=64, scale=0.125, flags=0, ws_bytes=None, override=None):
    ptrs = [b.p(i) for i in range(9)]
    if override:
        for i, val in override.items():
            ptrs[i] = val
    wsb = va.workspace_bytes(1, 1, max(Nq, 1), 64) if ws_bytes is None else ws_bytes
    return lib().vitattn_bwd_kv(*ptrs, B, H, Nq, Nk, d, scale, flags, b.p(9), wsb, None)


@pytest.mark.parametrize("kw,expected", [
    (dict(Nk=0), E_INVAL), (dict(flags=4), E_INVAL), (dict(flags=-1), E_INVAL), (dict(d=168), E_UNSUP),
    (dict(flags=2), E_WS), (dict(flags=3), E_WS),  # the dS mode needs its larger workspace
    (dict(ws_bytes=1), E_WS), (dict(override={6: None}), E_INVAL), (dict(override={7: 4102}), E_INVAL),
])
def test_bwd_kv_rejects_bad_arguments(kw, expected):
    b = Bufs()
    assert bwd_kv(b, **kw) == expected
    assert b.untouched()


def test_bwd_kv_workspace_is_sized_by_query_rows():
    b = Bufs(n=1 << 16)
    # 200 query rows need more workspace than 8: too small for Nq = 200
    assert bwd_kv(b, Nq=200, Nk=8, ws_bytes=va.workspace_bytes(1, 1, 8, 64)) == E_WS
    assert b.untouched()


@pytest.mark.parametrize("kw,expected", [
    (dict(P=0), E_INVAL), (dict(P=-3), E_INVAL), (dict(P=65537), E_INVAL), (dict(N=0), E_INVAL),
    (dict(d=100), E_UNSUP), (dict(d=168), E_UNSUP), (dict(d=0), E_UNSUP), (dict(override={0: None}), E_INVAL),
    (dict(override={3: 4104}), E_INVAL),
    (dict(H=128, N=1 << 20, d=160), E_INVAL),  # B*H*N*d/4 work-items past 2^32
])
def test_merge_rejects_bad_arguments(kw, expected):
    b = Bufs()
    args = dict(P=2, B=1, H=1, N=8, d=64)
    args.update({k: v for k, v in kw.items() if k != "override"})
    ptrs = [b.p(i) for i in range(4)]
    for i, val in kw.get("override", {}).items():
        ptrs[i] = val
    assert lib().vitattn_merge(ptrs[0], ptrs[1], args["P"], ptrs[2], ptrs[3], args["B"], args["H"], args["N"],
                               args["d"], None) == expected
    assert b.untouched()


@pytest.mark.parametrize("name", ["vitattn_ulysses_pack", "vitattn_ulysses_unpack", "vitattn_ulysses_pack_out",
                                  "vitattn_ulysses_unpack_out"])
@pytest.mark.parametrize("kw", [dict(H=6, P=4), dict(P=0), dict(B=0), dict(Nl=0), dict(row_bytes=24),
                                dict(row_bytes=0), dict(src=None), dict(dst=None), dict(src="dst"),
                                dict(src=4100), dict(B=70000, P=2, H=2),
                                dict(Nl=1 << 24, H=1 << 16, P=1, row_bytes=16),
                                dict(Nl=1 << 20, H=64, P=1, row_bytes=1024)])  # 2^24 blocks of 256: 2^32 items
def test_ulysses_layouts_reject_bad_arguments(name, kw):
    b = Bufs()
    args = dict(src=b.p(0), dst=b.p(1), B=1, Nl=4, H=4, P=2, row_bytes=32)
    args.update(kw)
    if args["src"] == "dst":
        args["src"] = args["dst"]
    fn = getattr(lib(), name)
    assert fn(args["src"], args["dst"], args["B"], args["Nl"], args["H"], args["P"], args["row_bytes"], None) == E_INVAL
    assert b.untouched()


@pytest.mark.parametrize("kw,expected", [
    (dict(M=0), E_INVAL), (dict(H=0), E_INVAL), (dict(C=0), E_INVAL), (dict(d=72), E_UNSUP),
    (dict(scale=float("inf")), E_INVAL), (dict(scale=-1.0), E_INVAL), (dict(M=70000, H=70000), E_INVAL),
    (dict(M=1 << 24, H=4), E_INVAL),  # (M + 3) * H * 64 work-items past 2^32
    (dict(override={0: None}), E_INVAL), (dict(override={3: 4100}), E_INVAL),
])
def test_agg_fwd_rejects_bad_arguments(kw, expected):
    b = Bufs()
    a = dict(M=2, H=2, C=5, d=64, scale=0.125)
    a.update({k: v for k, v in kw.items() if k != "override"})
    ptrs = [b.p(i) for i in range(5)]
    for i, val in kw.get("override", {}).items():
        ptrs[i] = val
    assert lib().vitattn_agg_fwd(*ptrs, a["M"], a["H"], a["C"], a["d"], a["scale"], None) == expected
    assert b.untouched()


def test_agg_bwd_validates_workspace_and_pointers():
    b = Bufs()
    L = lib()
    wsb = L.vitattn_agg_bwd_workspace_bytes(3, 2, 5, 64)
    assert wsb == 1 * 2 * 64 * 4  # one group of four patches
    assert L.vitattn_agg_bwd_workspace_bytes(5000, 2, 5, 64) == 1250 * 2 * 64 * 4
    assert L.vitattn_agg_bwd_workspace_bytes(5001, 2, 5, 64) == 1251 * 2 * 64 * 4
    assert L.vitattn_agg_bwd_workspace_bytes(0, 2, 5, 64) == 0
    ptrs = [b.p(i) for i in range(9)]
    assert L.vitattn_agg_bwd(*ptrs, 3, 2, 5, 64, 0.1, b.p(9), wsb - 4, None) == E_WS
    assert L.vitattn_agg_bwd(*ptrs, 3, 2, 5, 64, 0.1, None, wsb, None) == E_WS
    ptrs[6] = None
    assert L.vitattn_agg_bwd(*ptrs, 3, 2, 5, 64, 0.1, b.p(9), wsb, None) == E_INVAL
    assert b.untouched()


def test_binding_helpers_reject_wrong_tensors():
    torch = pytest.importorskip("torch")
    x = torch.zeros(1, 1, 8, 64, dtype=torch.bfloat16)
    with pytest.raises(TypeError):
        va.fwd(x, x, x)  # CPU tensors are refused before any library call


def test_product_package_does_not_import_the_oracle():
    pkg_dir = os.path.join(ROOT, "paper_2405_15780_amd")
    for dirpath, _, files in os.walk(pkg_dir):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"^\s*(from|import)\s+oracle\b", text, flags=re.M), f
                assert "oracle/" not in text, f


# ------------------------------------------------------------ strided entry points


def S(batch, head, row):
    return va.Strides(batch, head, row)


def fwd_strided(b, sq=None, sk=None, sv=None, so=None, B=2, H=2, Nq=8, Nk=8, d=72, scale=0.125):
    dq = S(H * Nq * d, Nq * d, d)
    dk = S(H * Nk * d, Nk * d, d)
    return lib().vitattn_fwd_strided(b.p(0), sq or dq, b.p(1), sk or dk, b.p(2), sv or dk, b.p(3), so or dq, b.p(4),
                                     B, H, Nq, Nk, d, scale, None)


@pytest.mark.parametrize("kw,expected", [
    (dict(sq=S(0, 0, 64)), E_INVAL),                  # row stride below d
    (dict(sk=S(-8, 72, 144)), E_INVAL),               # negative stride
    (dict(sv=S(1152, 576, 76)), E_INVAL),             # bf16 row stride not a multiple of 8
    (dict(sq=S(1152, 572, 72)), E_INVAL),             # head stride misaligned
    (dict(so=S(1152, 576, 74)), E_INVAL),             # fp32 row stride not a multiple of 4
    (dict(so=S(576, 576, 72)), E_INVAL),              # output heads overlap batches
    (dict(so=S(1152, 72, 72)), E_INVAL),              # output heads overlap rows
    (dict(so=S(0, 576, 72)), E_INVAL),                # output batches repeat
    (dict(sq=S(0, 0, 1 << 27)), E_INVAL),             # (rows + 256) * row bytes past 2^31
    (dict(sk=S(0, 0, 131064), Nk=7937), E_INVAL),     # the same, one legal pitch past the largest (131,056)
    (dict(d=100), E_UNSUP), (dict(d=168), E_UNSUP), (dict(B=0), E_INVAL), (dict(scale=0.0), E_INVAL),
])
def test_fwd_strided_rejects_bad_layouts(kw, expected):
    b = Bufs()
    assert fwd_strided(b, **kw) == expected
    assert b.untouched()


def bwd_strided(b, bad=None, B=2, H=2, N=8, d=72, flags=0, ws_bytes=None):
    dense = S(H * N * d, N * d, d)
    st = [dense] * 8  # q k v o dout dq dk dv
    if bad:
        i, val = bad
        st[i] = val
    wsb = va.workspace_bytes(B, H, N, d) if ws_bytes is None else ws_bytes
    return lib().vitattn_bwd_strided(b.p(0), st[0], b.p(1), st[1], b.p(2), st[2], b.p(3), st[3], b.p(4), st[4],
                                     b.p(5), b.p(6), st[5], b.p(7), st[6], b.p(8), st[7], B, H, N, N, d, 0.125, flags,
                                     b.p(9), wsb, None)


@pytest.mark.parametrize("which", range(8))
def test_bwd_strided_rejects_a_bad_layout_on_any_operand(which):
    b = Bufs()
    assert bwd_strided(b, bad=(which, S(1152, 576, 64))) == E_INVAL  # row stride below d
    assert bwd_strided(b, bad=(which, S(1152, 576, 76 if which in (0, 1, 2, 4) else 74))) == E_INVAL
    assert b.untouched()


def test_bwd_strided_output_overlap_and_workspace():
    b = Bufs()
    for i in (5, 6, 7):  # dq, dk, dv may not overlap themselves
        assert bwd_strided(b, bad=(i, S(576, 0, 72))) == E_INVAL
    assert bwd_strided(b, flags=4) == E_INVAL
    assert bwd_strided(b, ws_bytes=16) == E_WS
    assert b.untouched()


# ------------------------------------------------------------ dS mode


def test_ds_mode_workspace_sizes():
    base = va.workspace_bytes(1, 2, 300, 64)
    assert va.workspace_bytes_kv(1, 2, 300, 300, 64, 0) == base
    assert va.workspace_bytes_kv(1, 2, 300, 300, 64, 1) == base
    # 2 heads x (300 keys -> 3 x 128 -> 12 blocks) x (300 queries -> 5 x 64 -> 10 blocks) x 2 KB
    assert va.workspace_bytes_kv(1, 2, 300, 300, 64, 2) == base + 2 * 12 * 10 * 2048
    assert va.workspace_bytes_kv(1, 2, 188416, 188416, 128, 2) > 140e9
    assert va.workspace_bytes_kv(1, 2, 300, 300, 64, 4) == 0
    assert va.workspace_bytes_kv(1, 2, 300, 300, 100, 2) == 0


def test_ds_mode_stages_validate():
    b = Bufs()
    L = lib()
    need = va.workspace_bytes_kv(1, 1, 8, 8, 64, 2)
    assert L.vitattn_bwd_dkdv_ds(b.p(0), b.p(1), b.p(2), b.p(3), b.p(4), b.p(5), b.p(6), 1, 1, 8, 64, 0.1, b.p(7),
                                 need - 1, None) == E_WS
    assert L.vitattn_bwd_dkdv_ds(b.p(0), b.p(1), b.p(2), None, b.p(4), b.p(5), b.p(6), 1, 1, 8, 64, 0.1, b.p(7),
                                 need, None) == E_INVAL
    assert L.vitattn_bwd_dkdv_ds(b.p(0), b.p(1), b.p(2), b.p(3), b.p(4), b.p(5), b.p(6), 1, 1, 8, 100, 0.1, b.p(7),
                                 need, None) == E_UNSUP
    assert L.vitattn_bwd_dq_from_ds(b.p(1), b.p(5), 1, 1, 8, 64, 0.1, b.p(7), need - 1, None) == E_WS
    assert L.vitattn_bwd_dq_from_ds(b.p(1), None, 1, 1, 8, 64, 0.1, b.p(7), need, None) == E_INVAL
    assert L.vitattn_bwd_dq_from_ds(b.p(1), b.p(5), 1, 1, 8, 64, float("nan"), b.p(7), need, None) == E_INVAL
    assert b.untouched()
