"""CPU checks of the C ABI: exported symbols, the host-side partition builder
(bit-exact against the oracle's builder) and argument errors.  No kernel is
launched here; the partition is built with PGCN_SETUP_HOST_ONLY.
"""
import ctypes as C
import os
import re
import subprocess
import sys

import numpy as np
import pytest

from oracle.partition import build_partition
from paper_2203_10428_amd import binding as B
from paper_2203_10428_amd import configs, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "pgcn.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pgcn_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    syms = declared_symbols()
    assert len(syms) >= 14
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB_PATH], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (pgcn_\w+)", out))
    missing = [s for s in syms if s not in exported]
    assert not missing, missing
    assert set(syms) == set(B.SIGNATURES), "binding signatures must cover exactly the header"
    for s in syms:
        assert getattr(B.lib, s) is not None
    header = open(os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "pgcn.h")).read()
    assert B.pgcn_version() == int(re.search(r"#define PGCN_VERSION (\d+)", header).group(1)) == 165


def compare(g_n, rowptr, col, owner, nparts, part, self_loop=True):
    ref = build_partition(g_n, rowptr, col, owner, part, nparts, self_loop=self_loop)
    h = B.pgcn_partition_setup(g_n, rowptr, col, owner, nparts, part, host_only=True, self_loop=self_loop)
    info = B.pgcn_partition_info(h)
    assert info["host_only"] == 1
    assert (info["n_inner"], info["n_bd"], info["nnz"], info["n_send"]) == \
        (ref.n_inner, ref.n_bd, ref.nnz, len(ref.send_idx))
    ex = B.pgcn_partition_export(h)
    for k in ("inner_gid", "bd_gid", "recv_ptr", "rowptr", "col", "rowptr_t", "col_t", "send_ptr", "send_idx",
              "inv_ptr", "inv_k", "deg"):
        a, b = ex[k], getattr(ref, k)
        assert a.shape == b.shape and np.array_equal(a, b.astype(a.dtype)), k
    if ref.n_inner:
        assert info["max_row_len"] == int(np.diff(ref.rowptr).max())
    return info


def random_sym(n, m, nparts, seed):
    rng = np.random.default_rng(seed)
    u, v = rng.integers(0, n, m), rng.integers(0, n, m)
    src, dst = np.concatenate([u, v, u[:5]]), np.concatenate([v, u, v[:5]])   # duplicates + self loops
    o = np.lexsort((dst, src))
    rowptr = np.zeros(n + 1, np.int64)
    np.cumsum(np.bincount(src, minlength=n), out=rowptr[1:])
    return rowptr, dst[o].astype(np.int32), rng.integers(0, nparts, n).astype(np.int32)


@pytest.mark.parametrize("self_loop", [True, False])
@pytest.mark.parametrize("seed", range(6))
def test_setup_bit_exact_small(seed, self_loop):
    n, nparts = [5, 40, 64, 1, 33, 90][seed], [2, 3, 4, 1, 5, 3][seed]
    rowptr, col, owner = random_sym(n, 3 * n, nparts, seed)
    for part in range(nparts):
        compare(n, rowptr, col, owner, nparts, part, self_loop)


@pytest.mark.parametrize("self_loop", [True, False])
def test_setup_bit_exact_tiny_workload(self_loop):
    g = synth.tiny_uniform()
    for part in range(2):
        compare(g.n, g.rowptr, g.col, g.owner, g.nparts, part, self_loop)


def test_setup_empty_partition_and_isolated_nodes():
    # partition 2 owns nothing; node 0 is isolated
    n = 6
    rowptr = np.array([0, 0, 1, 2, 3, 4, 4], np.int64)
    col = np.array([2, 1, 4, 3], np.int32)
    owner = np.array([0, 0, 1, 0, 1, 1], np.int32)
    for part in range(3):
        info = compare(n, rowptr, col, owner, 3, part)
        if part == 2:
            assert info["n_inner"] == 0 and info["nnz"] == 0


def test_setup_chunk_counts_by_row_width(monkeypatch):
    # column chunks: about 8,000 gathered rows each (32,000 for rows of at most
    # 64 floats), while rows keep >= 32 non-zeros per chunk; the overrides set
    # every plan (PGCN_AGG_CHUNKS), those of P_i^T (PGCN_AGG_CHUNKS_T) or the
    # narrow ones (PGCN_AGG_CHUNKS_NARROW, before both)
    from gpu_helpers import random_partition_graph
    n, rowptr, col, owner = random_partition_graph(9000, 3000, 2, 120, 13)
    for k in ("PGCN_AGG_CHUNKS", "PGCN_AGG_CHUNKS_T", "PGCN_AGG_CHUNKS_NARROW"):
        monkeypatch.delenv(k, raising=False)

    def counts():
        info = B.pgcn_partition_info(B.pgcn_partition_setup(n, rowptr, col, owner, 2, 0, host_only=True))
        return info, (info["spmm_chunks"], info["spmm_chunks_narrow"], info["spmmt_chunks"],
                      info["spmmt_chunks_narrow"])

    info, got = counts()
    rows, cols, nnz = info["n_inner"], info["n_inner"] + info["n_bd"], info["nnz"]
    rule = lambda nr, nc, per: max(1, min(-(-nc // per), nnz // nr // 32, 16))
    assert got == (rule(rows, cols, 8000), rule(rows, cols, 32000), rule(cols, rows, 8000), rule(cols, rows, 32000))
    assert got == (2, 1, 2, 1)
    monkeypatch.setenv("PGCN_AGG_CHUNKS", "3")
    assert counts()[1] == (3, 3, 3, 3)
    monkeypatch.setenv("PGCN_AGG_CHUNKS_T", "5")
    assert counts()[1] == (3, 3, 5, 5)
    monkeypatch.setenv("PGCN_AGG_CHUNKS_NARROW", "2")
    assert counts()[1] == (3, 2, 5, 2)


def test_setup_heavy_rows_are_split_into_fixed_segments():
    # a star: the hub's row is longer than the default segment
    n = 1500
    hub_nb = np.arange(1, n, dtype=np.int32)
    rowptr = np.zeros(n + 1, np.int64)
    rowptr[1] = n - 1
    rowptr[2:] = n - 1 + np.arange(1, n)
    col = np.concatenate([hub_nb, np.zeros(n - 1, np.int32)])
    owner = (np.arange(n) % 2).astype(np.int32)
    info = compare(n, rowptr, col, owner, 2, 0)
    assert info["spmm_split_slots"] >= 2


@pytest.mark.parametrize("bad", ["rowptr0", "decreasing", "col_range", "owner_range", "self_range", "asymmetric",
                                 "asymmetric_duplicate"])
def test_setup_rejects_bad_input(bad):
    n = 4
    rowptr = np.array([0, 1, 2, 3, 4], np.int64)
    col = np.array([1, 0, 3, 2], np.int32)
    owner = np.array([0, 0, 1, 1], np.int32)
    nparts, part = 2, 0
    if bad == "rowptr0":
        rowptr = rowptr + 1
    elif bad == "decreasing":
        rowptr = np.array([0, 2, 1, 3, 4], np.int64)
    elif bad == "col_range":
        col = np.array([1, 0, 7, 2], np.int32)
    elif bad == "owner_range":
        owner = np.array([0, 0, 2, 1], np.int32)
    elif bad == "asymmetric":                   # 2 lists 1, 1 does not list 2
        rowptr = np.array([0, 1, 2, 4, 5], np.int64)
        col = np.array([1, 0, 3, 1, 2], np.int32)
    elif bad == "asymmetric_duplicate":         # a repeated entry does not stand in for the reverse edge
        rowptr = np.array([0, 2, 3, 4, 5], np.int64)
        col = np.array([1, 2, 0, 3, 2], np.int32)
    else:
        part = 2
    with pytest.raises(B.PgcnError) as e:
        B.pgcn_partition_setup(n, rowptr, col, owner, nparts, part, host_only=True)
    assert e.value.code == B.PGCN_EINVAL
    assert B.pgcn_last_error()
    if bad.startswith("asymmetric"):
        assert "not symmetric" in B.pgcn_last_error()


def test_setup_accepts_duplicates_and_self_loops():
    # a symmetric graph listed with repeated entries and self loops (both are canonicalised)
    rowptr = np.array([0, 3, 5, 7, 8], np.int64)
    col = np.array([1, 1, 0, 0, 1, 3, 2, 2], np.int32)
    owner = np.array([0, 0, 1, 1], np.int32)
    h = B.pgcn_partition_setup(4, rowptr, col, owner, 2, 0, host_only=True)
    assert B.pgcn_partition_info(h)["nnz"] == 4          # rows {0, 1} and {0, 1} with their self loops


def test_out_of_host_memory_is_a_status_not_an_abort():
    """A host allocation that fails inside set-up comes back as PGCN_ENOMEM (no C++ exception
    crosses the C interface).  Run in a child process whose address space is capped just above
    what it holds, on a graph whose set-up needs a few hundred MB more."""
    import textwrap
    code = textwrap.dedent("""
        import resource, sys
        import numpy as np
        sys.path.insert(0, %r)
        from paper_2203_10428_amd import binding as B
        n = 50_000_000
        rowptr = np.zeros(n + 1, np.int64)
        owner = np.zeros(n, np.int32)
        col = np.zeros(1, np.int32)
        vm = [int(l.split()[1]) for l in open("/proc/self/status") if l.startswith("VmSize:")][0] * 1024
        resource.setrlimit(resource.RLIMIT_AS, (vm + (128 << 20), vm + (128 << 20)))
        try:
            B.pgcn_partition_setup(n, rowptr, col, owner, 1, 0, host_only=True)
            print("no error")
        except B.PgcnError as e:
            print("status", e.code, B.pgcn_last_error())
    """ % os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    assert f"status {B.PGCN_ENOMEM} pgcn_partition_setup: out of host memory" in r.stdout, r.stdout + r.stderr[-2000:]


def test_setup_symmetric_flag():
    g = synth.tiny_uniform()
    h = B.pgcn_partition_setup(g.n, g.rowptr, g.col, g.owner, g.nparts, 0, host_only=True, symmetric=True)
    info = B.pgcn_partition_info(h)
    assert info["symmetric"] == 1 and info["self_loop"] == 1
    ref = build_partition(g.n, g.rowptr, g.col, g.owner, 0, g.nparts)
    assert np.array_equal(B.pgcn_partition_export(h)["deg"], ref.deg)
    with pytest.raises(B.PgcnError, match="self loops"):
        B.pgcn_partition_setup(g.n, g.rowptr, g.col, g.owner, g.nparts, 0, host_only=True, self_loop=False,
                               symmetric=True)
    flags_bad = B.PGCN_SETUP_HOST_ONLY | 64
    csr = B.pgcn_csr(g.n, np.ascontiguousarray(g.rowptr, np.int64).ctypes.data,
                     np.ascontiguousarray(g.col, np.int32).ctypes.data)
    owner = np.ascontiguousarray(g.owner, np.int32)
    bmap = B.pgcn_boundary_map(g.nparts, 0, owner.ctypes.data)
    out = B._vp()
    assert B.lib.pgcn_partition_setup(B.C.byref(csr), B.C.byref(bmap), flags_bad, B.C.byref(out)) == B.PGCN_EINVAL
    assert "unknown flags" in B.pgcn_last_error()


def test_compute_calls_reject_host_only_handle():
    g = synth.tiny_uniform()
    h = B.pgcn_partition_setup(g.n, g.rowptr, g.col, g.owner, 2, 0, host_only=True)
    with pytest.raises(B.PgcnError) as e:
        B.pgcn_pack_boundary(h, B.PGCN_PACK_FEAT, 0, 0, 4, 4)
    assert e.value.code == B.PGCN_EINVAL
    # argument errors are reported without touching the device
    with pytest.raises(B.PgcnError):
        B.pgcn_smooth_ema(0, 0, 10, 8, 6, 0.9)          # ld < cols
    with pytest.raises(B.PgcnError):
        B.pgcn_loss_fwd_bwd(7, 0, 1, 1, 1, None, None, 1, 1.0, 0, 0, 0, 0)
    # the forward that allocates nothing checks its handle and workspace arguments before any device call
    fwd = dict(f_in=8, f_out=4, gemm_dtype=B.PGCN_F32, relu=True, ld_in=8, ld_out=4, H_in=None, H_bd=None, W=None,
               A=None, A_bf16=None, H_out=None)
    with pytest.raises(B.PgcnError, match="host-only") as e:
        B.pgcn_layer_fwd_noalloc(h, **fwd)
    assert e.value.code == B.PGCN_EINVAL


def test_noalloc_scratch_limit_matches_the_header():
    header = open(os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "pgcn.h")).read()
    m = re.search(r"#define PGCN_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", header)
    assert m and int(m.group(1)) << int(m.group(2)) == B.PGCN_NOALLOC_SCRATCH_BYTES


@pytest.mark.slow
@pytest.mark.parametrize("name", ["reddit-like-1of4", "products-like-1of8", "yelp-like-1of3", "stress-rmat-2M"])
def test_setup_bit_exact_full_size(name):
    w = configs.WORKLOADS[name]
    g = configs.make_graph(w)
    compare(g.n, g.rowptr, g.col, g.owner, g.nparts, 0)


def test_binding_structs_match_the_header(tmp_path):
    """Every ctypes structure of the binding has the header's size and, field
    by field, its offsets (a C program compiled against include/pgcn.h prints
    them), so no argument can land in the wrong slot."""
    structs = [B.pgcn_csr, B.pgcn_boundary_map, B.pgcn_info, B.pgcn_arrays, B.pgcn_fwd_args, B.pgcn_bwd_args,
               B.pgcn_sage_fwd_args, B.pgcn_sage_bwd_args]
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "pgcn.h"', "int main(void) {"]
    for cls in structs:
        name = cls.__name__
        lines.append(f'  printf("{name} %zu\\n", sizeof({name}));')
        for field, _ in cls._fields_:
            lines.append(f'  printf("{name}.{field} %zu\\n", offsetof({name}, {field}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    r = subprocess.run(["gcc", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
                        str(src), "-o", str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    c_side = dict(line.split() for line in subprocess.run([str(exe)], capture_output=True, text=True,
                                                          check=True).stdout.splitlines())
    for cls in structs:
        name = cls.__name__
        assert int(c_side[name]) == C.sizeof(cls), name
        for field, _ in cls._fields_:
            assert int(c_side[f"{name}.{field}"]) == getattr(cls, field).offset, f"{name}.{field}"


def test_narrow_plans_share_the_dense_block(monkeypatch):
    """A narrow plan (rows of at most 64 floats, chunks of its own) aggregates with its
    matrix's dense block: a 41-wide layer's workspace holds the block's column images and
    sums, which a partition without the block does not need."""
    from gpu_helpers import random_partition_graph
    n, rowptr, col, owner = random_partition_graph(1500, 900, 3, 30, 4, hub_deg=800)
    for k, v in (("PGCN_HUB_ROWS", "300"), ("PGCN_HUB_COLS", "700"), ("PGCN_AGG_CHUNKS", "3"),
                 ("PGCN_AGG_CHUNKS_NARROW", "2")):
        monkeypatch.setenv(k, v)

    def sizes():
        h = B.pgcn_partition_setup(n, rowptr, col, owner, 3, 0, host_only=True)
        info = B.pgcn_partition_info(h)
        assert (info["spmm_chunks"], info["spmm_chunks_narrow"]) == (3, 2)
        return info, {(f, o): B.pgcn_layer_workspace_size(h, f, f, B.PGCN_F32, o)
                      for f in (41, 256) for o in (B.PGCN_ORDER_AGG, B.PGCN_ORDER_TRANSFORM)}

    info, with_block = sizes()
    assert info["spmm_hub_cols"] == 700
    monkeypatch.setenv("PGCN_HUB", "0")
    _, without = sizes()
    images = (700 + 31) // 32 * 8 * 8192           # column tiles x feature blocks x image bytes
    for key in with_block:
        assert with_block[key] - without[key] >= images, key


def test_dense_block_selection(monkeypatch):
    """PGCN_HUB_ROWS / _COLS force a dense block: the rows with the most non-zeros and the most
    referenced columns (ties by id); its non-zeros counted as set-up counts them, both directions."""
    from gpu_helpers import random_partition_graph
    n, rowptr, col, owner = random_partition_graph(1500, 900, 3, 30, 4, hub_deg=800)
    ref = build_partition(n, rowptr, col, owner, 0, 3)
    monkeypatch.setenv("PGCN_HUB_ROWS", "300")
    monkeypatch.setenv("PGCN_HUB_COLS", "700")
    info = B.pgcn_partition_info(B.pgcn_partition_setup(n, rowptr, col, owner, 3, 0, host_only=True))

    def block_nnz(rp, cl, nrows, ncols, R, C):
        lens = np.diff(rp)
        top_r = np.argsort(-lens, kind="stable")[:R]
        cnt = np.bincount(cl, minlength=ncols)
        top_c = np.zeros(ncols, bool)
        top_c[np.argsort(-cnt, kind="stable")[:C]] = True
        return int(sum(top_c[cl[rp[r]:rp[r + 1]]].sum() for r in top_r))

    nr, nc = ref.n_inner, ref.n_inner + ref.n_bd
    assert (info["spmm_hub_rows"], info["spmm_hub_cols"]) == (300, 700)
    assert info["spmm_hub_nnz"] == block_nnz(ref.rowptr, ref.col, nr, nc, 300, 700) > 0
    assert (info["spmmt_hub_rows"], info["spmmt_hub_cols"]) == (300, 700)
    assert info["spmmt_hub_nnz"] == block_nnz(ref.rowptr_t, ref.col_t, nc, nr, 300, 700) > 0
    # the set-up arrays themselves do not change
    compare(n, rowptr, col, owner, 3, 0)
    monkeypatch.setenv("PGCN_HUB", "0")
    info = B.pgcn_partition_info(B.pgcn_partition_setup(n, rowptr, col, owner, 3, 0, host_only=True))
    assert info["spmm_hub_rows"] == 0 and info["spmmt_hub_rows"] == 0
