"""C ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and rejects invalid arguments on the host with the documented
status before any device work (null device pointers are never dereferenced)."""

import ctypes
import os
import re
import subprocess

import pytest

from paper_2609_27373_amd import wise

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "wise.h")


def header_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(wise_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(wise.LIB_PATH):
        from paper_2609_27373_amd import build
        build.build()
    return wise.load()


def test_header_lists_the_binding_exports():
    assert header_functions() == sorted(wise.EXPORTS)


def test_exports(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", wise.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    syms = {ln.split()[-1] for ln in out.splitlines() if ln.strip()}
    for fn in header_functions():
        assert fn in syms, fn
        assert hasattr(lib, fn)


def test_version_and_strings(lib):
    assert wise.wise_abi_version() == 6
    for st, name in wise.STATUS_NAMES.items():
        assert wise.wise_status_string(st).startswith(name)
    assert "unknown" in wise.wise_status_string(99)


def S(**kw):
    base = dict(batch=1, heads=2, seq_len=512, head_dim=64, block=64, scale=0.0)
    base.update(kw)
    return wise.make_shape(**base)


def test_capacity_and_workspace(lib):
    s = S()
    assert wise.wise_support_capacity(s) == 2 * 8 * 9 // 2
    assert wise.wise_select_workspace_bytes(s) > 0
    s4 = S(batch=1, heads=32, seq_len=32768, head_dim=128, block=128)
    assert wise.wise_support_capacity(s4) == 32 * 256 * 257 // 2
    assert wise.wise_support_capacity(S(seq_len=500)) == -1
    assert wise.wise_select_workspace_bytes(S(head_dim=80)) == 0
    assert wise.wise_support_capacity(S(block=32)) == 2 * 16 * 17 // 2
    assert wise.wise_support_capacity(S(block=16)) == 2 * 32 * 33 // 2
    # 512 = 4 tiles of 128 queries; tile t keeps (t+1)*2 spans of 64 keys (4 of 32 keys)
    assert wise.wise_mass_workspace_bytes(S()) == 2 * 128 * 2 * (4 * 5 // 2) * 4
    assert wise.wise_mass_workspace_bytes(S(block=32)) == 2 * 128 * 4 * (4 * 5 // 2) * 4
    assert wise.wise_mass_workspace_bytes(S(block=16)) == 2 * 128 * 8 * (4 * 5 // 2) * 4
    assert wise.wise_mass_workspace_bytes(S(seq_len=320)) == 2 * 64 * 1 * (5 * 6 // 2) * 4
    # head_dim 128: tiles of 256 queries when they divide seq_len
    assert wise.wise_mass_workspace_bytes(S(head_dim=128)) == 2 * 256 * 4 * (2 * 3 // 2) * 4
    assert wise.wise_mass_workspace_bytes(S(head_dim=128, seq_len=384)) == 2 * 128 * 2 * (3 * 4 // 2) * 4
    assert wise.wise_mass_workspace_bytes(S(head_dim=80)) == 0
    # the smallest workspace: one key-value group of heads
    assert wise.wise_mass_workspace_min_bytes(S()) == wise.wise_mass_workspace_bytes(S()) // 2
    g = S(heads=8, kv_heads=2, batch=3)
    assert wise.wise_mass_workspace_min_bytes(g) == wise.wise_mass_workspace_bytes(g) // 24 * 4
    assert wise.wise_mass_workspace_min_bytes(S(head_dim=80)) == 0
    assert wise.wise_mask_words(S()) == 1
    assert wise.wise_mask_words(S(seq_len=64 * 65)) == 2
    assert wise.wise_mask_words(s4) == 4
    assert wise.wise_mask_words(S(seq_len=500)) == -1


FAKE = ctypes.c_void_p(4096)        # aligned, never dereferenced: calls fail validation first
MIS = ctypes.c_void_p(4096 + 2)     # misaligned


def dense(lib, s, q=FAKE, k=FAKE, v=FAKE, o=FAKE, lse=None, acc=None, ws=None, wsb=0):
    return lib.wise_dense_attn_accum(ctypes.byref(s) if s is not None else None, q, k, v, o, lse,
                                     acc, ws, wsb, None)


def select(lib, s, acc=FAKE, tau=0.9, flags=3, rp=FAKE, ci=FAKE, ro=None, ws=FAKE, wsb=1 << 30):
    return lib.wise_select_support(ctypes.byref(s) if s is not None else None, acc,
                                   ctypes.c_float(tau), flags, rp, ci, ro, ws, wsb, None)


def sparse(lib, s, q=FAKE, rp=FAKE, ci=FAKE, o=FAKE):
    return lib.wise_sparse_attn(ctypes.byref(s) if s is not None else None, q, FAKE, FAKE, rp, ci,
                                None, o, None, None)


@pytest.mark.parametrize("case,status", [
    (dict(s=None), 1), (dict(q=None), 1), (dict(o=None), 1), (dict(acc=FAKE), 1),
    (dict(acc=FAKE, ws=FAKE, wsb=16), 5), (dict(acc=FAKE, ws=ctypes.c_void_p(4096 + 16), wsb=1 << 40), 2),
    (dict(s=S(seq_len=500)), 2), (dict(s=S(batch=0)), 2), (dict(s=S(heads=-1)), 2),
    (dict(s=S(head_dim=80)), 3), (dict(s=S(block=8)), 3), (dict(q=MIS), 2),
    (dict(s=S(block=16, seq_len=96)), 2),
    (dict(s=S(block=32, seq_len=96)), 2), (dict(s=S(block=256)), 3),
    (dict(s=S(heads=4, kv_heads=3)), 2), (dict(s=S(kv_heads=-1)), 2), (dict(s=S(kv_heads=4)), 2),
    (dict(s=S(scale=float("inf"))), 4), (dict(s=S(scale=float("nan"))), 4),
    (dict(s=S(batch=4096, heads=4096, seq_len=1024, block=64)), 2),
])
def test_dense_validation(lib, case, status):
    s = case.pop("s", S())
    assert dense(lib, s, **case) == status


@pytest.mark.parametrize("case,status", [
    (dict(s=None), 1), (dict(acc=None), 1), (dict(rp=None), 1), (dict(ws=None), 1),
    (dict(tau=0.0), 4), (dict(tau=1.5), 4), (dict(tau=float("nan")), 4), (dict(tau=-0.1), 4),
    (dict(flags=4), 4), (dict(wsb=16), 5), (dict(s=S(block=96)), 3),
    (dict(s=S(seq_len=64 * 2048)), 3), (dict(ws=ctypes.c_void_p(4096 + 16)), 2),
])
def test_select_validation(lib, case, status):
    s = case.pop("s", S())
    assert select(lib, s, **case) == status


@pytest.mark.parametrize("case,status", [
    (dict(s=None), 1), (dict(q=None), 1), (dict(rp=None), 1), (dict(ci=None), 1),
    (dict(o=None), 1), (dict(s=S(seq_len=100)), 2), (dict(s=S(head_dim=256)), 3),
    (dict(o=MIS), 2),
])
def test_sparse_validation(lib, case, status):
    s = case.pop("s", S())
    assert sparse(lib, s, **dict(case)) == status
    g = dict(case)
    assert lib.wise_sparse_attn_grouped(sh(s), g.get("q", FAKE), FAKE, FAKE, g.get("rp", FAKE),
                                        g.get("ci", FAKE), g.get("o", FAKE), None, None) == status


def test_sparse_group_rows(lib):
    assert wise.wise_sparse_group_rows(S(head_dim=128, seq_len=1024)) == 4   # 256-query groups
    assert wise.wise_sparse_group_rows(S(head_dim=128, seq_len=640)) == 2    # 128 divides, 256 not
    assert wise.wise_sparse_group_rows(S(head_dim=96)) == 2
    assert wise.wise_sparse_group_rows(S(head_dim=64, seq_len=320)) == 0     # 64-query tiles
    assert wise.wise_sparse_group_rows(S(block=32)) == 0
    assert wise.wise_sparse_group_rows(S(block=128)) == 0                    # 128-key rows: d 128 only
    assert wise.wise_sparse_group_rows(S(block=128, head_dim=96)) == 0
    assert wise.wise_sparse_group_rows(S(block=128, head_dim=128)) == 2      # two rows of 4 waves
    assert wise.wise_sparse_group_rows(S(block=128, head_dim=128, seq_len=640)) == 0
    assert wise.wise_sparse_group_rows(S(block=128, head_dim=128, seq_len=128 * 1024)) == 2
    assert wise.wise_sparse_group_rows(S(block=128, head_dim=128, seq_len=128 * 1026)) == 0
    assert wise.wise_sparse_group_rows(S(seq_len=64 * 2048)) == 0            # > 1024 key blocks
    assert wise.wise_sparse_group_rows(S(seq_len=500)) == -1


def test_group_density_covers_every_group_shape(lib):
    """The pipeline's automatic late-kernel choice has a measured break-even
    density (or a measured "never") for every group shape and head_dim the
    library can return."""
    from paper_2609_27373_amd.pipeline import WisePipeline
    seen = set()
    for d in (64, 96, 128):
        for block in (16, 32, 64, 128):
            for n in (128, 256, 384, 512, 640, 4096, 8192, 65536, 131072):
                if n % block:
                    continue
                rows = wise.wise_sparse_group_rows(S(head_dim=d, block=block, seq_len=n))
                if rows > 0:
                    seen.add((block, rows, d))
                    assert (block, rows, d) in WisePipeline.GROUP_DENSITY, (d, block, n, rows)
    assert seen == set(WisePipeline.GROUP_DENSITY)


MIS8 = ctypes.c_void_p(4096 + 4)    # 4-byte but not 8-byte aligned


def sh(s):
    return ctypes.byref(s) if s is not None else None


@pytest.mark.parametrize("case,status", [
    (dict(s=None), 1), (dict(r=None), 1), (dict(mask=None), 1), (dict(tau=0.0), 4),
    (dict(tau=1.01), 4), (dict(tau=float("nan")), 4), (dict(mask=MIS8), 2),
    (dict(s=S(seq_len=64 * 2048)), 3), (dict(s=S(head_dim=80)), 3),
])
def test_select_step_validation(lib, case, status):
    s = case.pop("s", S())
    a = dict(r=FAKE, tau=0.9, mask=FAKE)
    a.update(case)
    assert lib.wise_select_step(sh(s), a["r"], ctypes.c_float(a["tau"]), a["mask"], None) == status


@pytest.mark.parametrize("case,status", [
    (dict(s=None), 1), (dict(masks=None), 1), (dict(rp=None), 1), (dict(ws=None), 1),
    (dict(n=0), 2), (dict(n=-3), 2), (dict(flags=8), 4), (dict(wsb=16), 5),
    (dict(masks=MIS8), 2), (dict(s=S(seq_len=64 * 2048)), 3),
])
def test_support_from_masks_validation(lib, case, status):
    s = case.pop("s", S())
    a = dict(masks=FAKE, n=4, flags=3, rp=FAKE, ci=FAKE, ws=FAKE, wsb=1 << 30)
    a.update(case)
    assert lib.wise_support_from_masks(sh(s), a["masks"], a["n"], a["flags"], a["rp"], a["ci"],
                                       None, a["ws"], a["wsb"], None) == status


@pytest.mark.parametrize("fn,args,status", [
    ("wise_mask_union", (None, 2, FAKE), 1), ("wise_mask_union", (FAKE, 0, FAKE), 2),
    ("wise_mask_union", (FAKE, 2, MIS8), 2), ("wise_mask_union", (FAKE, 1, None), 1),
    ("wise_mask_overlap", (FAKE, None, FAKE), 1), ("wise_mask_overlap", (FAKE, FAKE, MIS8), 2),
    ("wise_support_mass", (FAKE, FAKE, FAKE, None, None), 1),
    ("wise_support_mass", (None, FAKE, FAKE, FAKE, None), 1),
    ("wise_support_mass", (FAKE, FAKE, FAKE, MIS8, None), 2),
    ("wise_support_mass", (FAKE, FAKE, FAKE, FAKE, MIS8), 2),
])
def test_mask_and_mass_validation(lib, fn, args, status):
    assert getattr(lib, fn)(sh(S()), *args, None) == status
    assert getattr(lib, fn)(None, *args, None) == 1
    assert getattr(lib, fn)(sh(S(head_dim=80)), *args, None) == 3


@pytest.mark.parametrize("case,status", [
    (dict(s=None), 1), (dict(acc=None), 1), (dict(rp=None), 1), (dict(ci=None), 1),
    (dict(tau=0.0), 4), (dict(tau=1.5), 4), (dict(flags=4), 4), (dict(s=S(block=96)), 3),
    (dict(s=S(seq_len=64 * 2048)), 3), (dict(rp=MIS8.value + 1), 2),
    # 1024 x 1024 rows of 1024 blocks need 132 MiB of scratch, past the 4 MiB array
    (dict(s=S(batch=16, heads=64, seq_len=32 * 1024, block=32)), 5),
])
def test_select_noalloc_validation(lib, case, status):
    s = case.pop("s", S())
    a = dict(acc=FAKE, tau=0.9, flags=3, rp=FAKE, ci=FAKE)
    a.update(case)
    rp = ctypes.c_void_p(a["rp"]) if isinstance(a["rp"], int) else a["rp"]
    assert lib.wise_select_support_noalloc(sh(s), a["acc"], ctypes.c_float(a["tau"]), a["flags"],
                                           rp, a["ci"], None, None) == status
    if s is not None and status == 5:
        assert wise.wise_select_workspace_bytes(s) > wise.NOALLOC_SCRATCH_BYTES
