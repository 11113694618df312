"""Host-only checks of the C-ABI library: it loads, exports every function the
header declares, and rejects invalid arguments before making any HIP call (so
these run without a GPU)."""
import ctypes
import os
import re

import pytest

from paper_2508_21706_amd import binding as bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "specmoe_verify.h")
HEADERS = [os.path.join(ROOT, "include", h) for h in sorted(os.listdir(os.path.join(ROOT, "include")))
           if h.endswith(".h")]

FAKE = 0x10000          # 16-byte aligned, never dereferenced by these tests


@pytest.fixture(scope="module")
def lib():
    return bd.load_library()


def header_functions():
    text = "".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(specmoe_\w+)\s*\(", text)))


def test_exports_every_declared_function(lib):
    names = header_functions()
    assert {"specmoe_verify_attn", "specmoe_verify_attn_workspace_bytes", "specmoe_verify_attn_tree",
            "specmoe_accept_greedy", "specmoe_accept_workspace_bytes", "specmoe_accept_workspace_init",
            "specmoe_status_str"} <= set(names)
    for n in names:
        assert hasattr(lib, n), f"{n} is declared in the header but not exported"


def test_status_codes_match_header(lib):
    text = open(HEADER).read()
    codes = dict((n, int(v)) for n, v in re.findall(r"(SPECMOE_(?:OK|ERR_\w+))\s*=\s*(-?\d+)", text))
    assert codes == {v: k for k, v in bd.STATUS.items()}
    for code in codes.values():
        assert lib.specmoe_status_str(code).decode() not in ("", "unknown status")
    assert lib.specmoe_status_str(12345).decode() == "unknown status"


def _desc(**kw):
    base = dict(B=2, Hq=32, Hkv=8, D=128, C_max=5, S_max=2304, dtype=bd.SPECMOE_BF16, grid_blocks=0)
    base.update(kw)
    return bd.make_desc(**base)


def _call(lib, desc, q=FAKE, k=FAKE, v=FAKE, ctx=FAKE, chunk=FAKE, scale=0.088, out=FAKE, lse=FAKE):
    return lib.specmoe_verify_attn(q, k, v, ctx, chunk, scale, out, lse, None,
                                   ctypes.byref(desc) if desc is not None else None)


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=7), -5),
    (dict(D=96), -4),
    (dict(D=256), -4),
    (dict(B=-1), -2),
    (dict(Hq=0), -2),
    (dict(Hkv=0), -2),
    (dict(C_max=0), -2),
    (dict(S_max=4, C_max=5), -2),
    (dict(Hq=30, Hkv=8), -3),
    (dict(C_max=17, Hq=32, Hkv=4), -6),          # 17 * 8 = 136 rows > 128
    (dict(grid_blocks=-1), -7),
    (dict(grid_blocks=2049), -7),
    (dict(flags=2), -12),                        # only SPECMOE_FLAG_NO_WAIT is defined
    (dict(flags=3), -12),
    (dict(S_max=1 << 23), -2),                   # slab offsets would pass 2^31 bytes
    (dict(S_max=1 << 24, dtype=bd.SPECMOE_BF16, D=64), -2),   # packed lengths need T < 2^24
])
def test_invalid_descriptor(lib, kw, code):
    assert _call(lib, _desc(**kw)) == code
    assert lib.specmoe_verify_attn_workspace_bytes(ctypes.byref(_desc(**kw))) == 0


def test_null_and_alignment_and_scale(lib):
    d = _desc()
    d.workspace, d.workspace_bytes = FAKE, 1 << 30
    assert _call(lib, None) == -1
    for arg in ("q", "k", "v", "ctx", "chunk", "out", "lse"):
        assert _call(lib, d, **{arg: None}) == -1, arg
    for arg in ("q", "k", "v", "out"):
        assert _call(lib, d, **{arg: FAKE + 4}) == -9, arg
    assert _call(lib, d, scale=float("nan")) == -10
    assert _call(lib, d, scale=float("inf")) == -10
    # the kernels track the running maximum of scale * q.k as scale times the
    # maximum of q.k, which needs scale > 0
    for bad in (0.0, -0.0, -0.088, -float("inf")):
        assert _call(lib, d, scale=bad) == -10, bad
    assert _call(lib, d, scale=1e-30) != -10


def test_descriptor_struct_matches_header():
    """The binding's mirror of specmoe_verify_desc has the header's fields, in
    order (no timing or other hidden fields)."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    body = re.search(r"typedef struct specmoe_verify_desc \{(.*?)\} specmoe_verify_desc;", text, re.S).group(1)
    fields = re.findall(r"(\w+)\s*;", body)
    assert fields == [f[0] for f in bd.Desc._fields_]
    assert ctypes.sizeof(bd.Desc) == 56


def _call_tree(lib, desc, mask=FAKE, **kw):
    args = dict(q=FAKE, k=FAKE, v=FAKE, ctx=FAKE, chunk=FAKE, scale=0.088, out=FAKE, lse=FAKE)
    args.update(kw)
    return lib.specmoe_verify_attn_tree(args["q"], args["k"], args["v"], args["ctx"], args["chunk"], mask,
                                        args["scale"], args["out"], args["lse"], None,
                                        ctypes.byref(desc) if desc is not None else None)


def test_tree_entry_point_host_checks(lib):
    d = _desc(C_max=16, Hq=32, Hkv=4)           # 128 rows, 16 draft tokens
    d.workspace, d.workspace_bytes = FAKE, 1 << 30
    assert _call_tree(lib, None) == -1
    assert _call_tree(lib, d, mask=None) == -1
    for arg in ("q", "k", "v", "ctx", "chunk", "out", "lse"):
        assert _call_tree(lib, d, **{arg: None}) == -1, arg
    assert _call_tree(lib, d, mask=FAKE + 4) == -9          # words are 8-byte aligned
    assert _call_tree(lib, d, q=FAKE + 4) == -9
    assert _call_tree(lib, d, scale=float("nan")) == -10
    # one 64-bit word per draft token: at most 64 draft tokens
    wide = _desc(C_max=65, Hq=1, Hkv=1, S_max=2304)
    wide.workspace, wide.workspace_bytes = FAKE, 1 << 30
    assert _call_tree(lib, wide) == -13
    # the chain entry point has no such limit: with a too-small workspace it
    # gets as far as the workspace check (and launches nothing)
    wide.workspace_bytes = 1
    assert _call(lib, wide) == -8
    wide.B = 0
    assert _call_tree(lib, wide) == -13                     # a descriptor error even for B = 0
    # B = 0 with a valid descriptor: no pointer is looked at
    empty = _desc(B=0, C_max=16, Hq=32, Hkv=4)
    assert _call_tree(lib, empty, mask=None, q=None, out=None) == 0
    # descriptor errors come first, as in the chain entry point
    assert _call_tree(lib, _desc(D=96)) == -4
    assert lib.specmoe_status_str(-13).decode().startswith("draft masks")


def test_workspace_contract(lib):
    d = _desc(B=64, grid_blocks=256)
    need = lib.specmoe_verify_attn_workspace_bytes(ctypes.byref(d))
    rows = 5 * 4                                # C_max * g
    slots = 2 * 256 * rows                      # two pieces per workgroup
    counters = 1024 * 8 * 4                     # one per (sequence, KV head) of a launch
    header = 256                                # the sticky status word
    assert need >= header + counters + slots * (128 + 1) * 4
    assert need < header + counters + slots * (128 + 1) * 4 + 512
    # the workspace grows with the grid
    d2 = _desc(B=64, grid_blocks=1024)
    assert lib.specmoe_verify_attn_workspace_bytes(ctypes.byref(d2)) > need
    # default grid = 256 workgroups
    assert lib.specmoe_verify_attn_workspace_bytes(ctypes.byref(_desc(B=64))) == need
    assert _call(lib, d) == -1                  # workspace needed but NULL
    d.workspace, d.workspace_bytes = FAKE, need - 1
    assert _call(lib, d) == -8
    d.workspace, d.workspace_bytes = FAKE + 8, need
    assert _call(lib, d) == -9
    # the counter-zeroing entry point validates before launching anything
    init = lib.specmoe_verify_attn_workspace_init
    assert init(None, need, None, ctypes.byref(_desc(B=64))) == -1
    assert init(FAKE, need - 1, None, ctypes.byref(_desc(B=64))) == -8
    assert init(FAKE + 4, need, None, ctypes.byref(_desc(B=64))) == -9
    assert init(FAKE, need, None, ctypes.byref(_desc(B=64, D=80))) == -4
    # the status query validates before its copy
    status = lib.specmoe_verify_attn_status
    assert status(None, need, None) == -1
    assert status(FAKE + 4, need, None) == -9
    assert status(FAKE, 255, None) == -8


def test_key_tile(lib):
    assert lib.specmoe_verify_attn_key_tile(ctypes.byref(_desc())) == 128    # 32 KB of bf16 D=128 rows
    assert lib.specmoe_verify_attn_key_tile(ctypes.byref(_desc(D=64))) == 256
    assert lib.specmoe_verify_attn_key_tile(ctypes.byref(_desc(dtype=bd.SPECMOE_F32, D=64))) == 128
    assert lib.specmoe_verify_attn_key_tile(ctypes.byref(_desc(dtype=bd.SPECMOE_F32, D=128))) == 64
    assert lib.specmoe_verify_attn_key_tile(ctypes.byref(_desc(D=80))) == -4
    assert lib.specmoe_verify_attn_key_tile(ctypes.byref(_desc(dtype=bd.SPECMOE_F16))) == 128   # f16 as bf16
    assert lib.specmoe_verify_attn_key_tile(ctypes.byref(_desc(dtype=3))) == -5


def test_noalloc_host_checks(lib):
    """The allocation-free entry point validates like the others and refuses
    a problem whose workspace would not fit its static scratch, before any
    HIP call."""
    call = lib.specmoe_verify_attn_noalloc
    args = (FAKE, FAKE, FAKE, FAKE, FAKE, 0.088, FAKE, FAKE, None)
    assert call(*args, None) == -1
    assert call(*args, ctypes.byref(_desc(D=96))) == -4
    assert call(*args, ctypes.byref(_desc(flags=2))) == -12
    # 2 * 2048 workgroups * 128 rows * (128 + 1) * 4 bytes > 48 MiB of scratch
    assert call(*args, ctypes.byref(_desc(C_max=16, Hq=32, Hkv=4, grid_blocks=2048))) == -8
    assert call(None, None, None, None, None, 0.088, None, None, None, ctypes.byref(_desc(B=0))) == 0
    assert call(*args[:5], -1.0, *args[6:], ctypes.byref(_desc(B=0))) == 0   # B = 0: nothing is looked at


def test_empty_batch_is_a_no_op(lib):
    # B = 0 returns before any HIP call and before looking at data pointers
    assert _call(lib, _desc(B=0)) == 0
    assert _call(lib, _desc(B=0), q=None, k=None, v=None, ctx=None, chunk=None, out=None, lse=None) == 0
    assert _call(lib, _desc(B=0, dtype=9)) == -5    # the descriptor is still validated


# ------------------------------------------------------------ acceptance step

def _adesc(**kw):
    base = dict(B=4, C_max=5, V=32000, dtype=bd.SPECMOE_BF16, split=0)
    base.update(kw)
    return bd.accept_desc(**base)


def _acall(lib, desc, logits=FAKE, tokens=FAKE, ctx=FAKE, chunk=FAKE, am=FAKE, acc=FAKE, nxt=FAKE, new=FAKE):
    return lib.specmoe_accept_greedy(logits, tokens, ctx, chunk, am, acc, nxt, new, None,
                                     ctypes.byref(desc) if desc is not None else None)


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=3), -5),
    (dict(B=-1), -2),
    (dict(B=65537), -2),
    (dict(C_max=0), -2),
    (dict(C_max=1025), -2),
    (dict(V=0), -2),
    (dict(V=32001), -2),                          # rows are read in 16-byte vectors
    (dict(V=1002, dtype=bd.SPECMOE_F32), -2),
    (dict(split=1000), -2),
    (dict(split=-2048), -2),
    (dict(B=4096, C_max=1024, V=32000), -2),      # element offsets would pass 2^31
])
def test_accept_invalid_descriptor(lib, kw, code):
    assert _acall(lib, _adesc(**kw)) == code
    assert lib.specmoe_accept_workspace_bytes(ctypes.byref(_adesc(**kw))) == 0


def test_accept_host_checks_and_workspace(lib):
    d = _adesc()
    need = lib.specmoe_accept_workspace_bytes(ctypes.byref(d))
    items = (32000 + 4095) // 4096                # default: 8 KB of bf16 logits per item
    assert need == 65536 * 4 + 4 * 5 * items * 8
    d32 = _adesc(dtype=bd.SPECMOE_F32, V=32000)
    assert lib.specmoe_accept_workspace_bytes(ctypes.byref(d32)) == 65536 * 4 + 4 * 5 * 16 * 8
    assert lib.specmoe_accept_workspace_bytes(ctypes.byref(_adesc(split=1024))) == 65536 * 4 + 4 * 5 * 32 * 8
    assert _acall(lib, None) == -1
    d.flags = 1
    assert _acall(lib, d) == -12
    d.flags = 0
    assert _acall(lib, d) == -1                   # workspace needed but NULL
    d.workspace, d.workspace_bytes = FAKE, need - 1
    assert _acall(lib, d) == -8
    d.workspace, d.workspace_bytes = FAKE + 8, need
    assert _acall(lib, d) == -9
    d.workspace = FAKE
    for arg in ("logits", "tokens", "ctx", "chunk", "am", "acc", "nxt", "new"):
        assert _acall(lib, d, **{arg: None}) == -1, arg
    assert _acall(lib, d, logits=FAKE + 4) == -9
    assert _acall(lib, _adesc(B=0), logits=None, tokens=None) == 0
    init = lib.specmoe_accept_workspace_init
    assert init(None, need, None, ctypes.byref(_adesc())) == -1
    assert init(FAKE, need - 1, None, ctypes.byref(_adesc())) == -8
    assert init(FAKE + 4, need, None, ctypes.byref(_adesc())) == -9


def test_tree_acceptance_and_compaction_host_checks(lib):
    d = _adesc(C_max=65)
    d.workspace, d.workspace_bytes = FAKE, 1 << 30
    assert lib.specmoe_accept_greedy_tree(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None,
                                          ctypes.byref(d)) == -13
    d = _adesc(C_max=16)
    d.workspace, d.workspace_bytes = FAKE, 1 << 30
    for i in (2, 9):   # draft_mask, path
        args = [FAKE] * 11
        args[i] = None
        args[10] = None
        assert lib.specmoe_accept_greedy_tree(*args, ctypes.byref(d)) == -1
    args = [FAKE] * 10 + [None]
    args[2] = FAKE + 4
    assert lib.specmoe_accept_greedy_tree(*args, ctypes.byref(d)) == -9
    compact = lib.specmoe_compact_accepted_kv
    vd = _desc()
    assert compact(FAKE, FAKE, FAKE, FAKE, None, None) == -1
    assert compact(None, FAKE, FAKE, FAKE, None, ctypes.byref(vd)) == -1
    assert compact(FAKE, FAKE, FAKE, None, None, ctypes.byref(vd)) == -1
    assert compact(FAKE + 4, FAKE, FAKE, FAKE, None, ctypes.byref(vd)) == -9
    assert compact(FAKE, FAKE, FAKE, FAKE + 4, None, ctypes.byref(vd)) == -9
    assert compact(FAKE, FAKE, FAKE, FAKE, None, ctypes.byref(_desc(dtype=5))) == -5
    assert compact(FAKE, FAKE, FAKE, FAKE, None, ctypes.byref(_desc(D=96))) == -4
    assert compact(None, None, None, None, None, ctypes.byref(_desc(B=0))) == 0

