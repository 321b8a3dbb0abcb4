"""C-ABI library: loads, exports every declared symbol, and its host-side calls
(partition, mini-batch CSR) match the oracle bit for bit.  No GPU needed:
these entry points run on the host and launch nothing."""

import os
import re

import numpy as np
import pytest

from gist_synth import get_config
from gist_synth.graphs import chung_lu, erdos_renyi, sbm
from oracle import minibatch as MB
from oracle import partition as P

G = pytest.importorskip("paper_2102_10424_amd.gist",
                        reason="libgist.so not built (python -m paper_2102_10424_amd.build)")

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "include", "gist.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gist_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 15
    lib = G._lib
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(G.EXPORTED) == names


def test_status_strings():
    assert G.status_str(0) == "GIST_OK"
    assert G.status_str(-5) == "GIST_E_NONFINITE"


@pytest.mark.parametrize("d,m", [(4, 2), (256, 2), (2048, 4), (4096, 4), (32768, 8),
                                 (2048, 8), (97, 97), (10, 1), (1433, 1)])
def test_partition_bit_exact(d, m):
    for seed in (0, 1, 12345, 2**64 - 1):
        idx, offs = G.gist_partition(d, m, seed)
        oi, oo = P.partition(d, m, seed)
        assert np.array_equal(idx, np.asarray(oi, dtype=np.int32))
        assert np.array_equal(offs, np.asarray(oo, dtype=np.int64))


@pytest.mark.parametrize("d,m", [(64, 4), (1000, 8), (5, 5)])
def test_partition_categorical_bit_exact(d, m):
    for seed in (3, 77):
        idx, offs = G.gist_partition(d, m, seed, G.GIST_PART_CATEGORICAL)
        oi, oo = P.partition(d, m, seed, categorical=True)
        assert np.array_equal(idx, np.asarray(oi, dtype=np.int32))
        assert np.array_equal(offs, np.asarray(oo, dtype=np.int64))


def test_single_hip_runtime():
    """The binding runs on PyTorch's HIP runtime; no second copy is loaded."""
    maps = {line.split()[-1] for line in open("/proc/self/maps") if "libamdhip64" in line}
    assert len(maps) == 1, maps


@pytest.mark.parametrize("d,m,cat", [(64, 4, False), (32768, 8, False), (1000, 8, True),
                                     (7, 1, False)])
def test_partition_inverse(d, m, cat):
    """The rank of index r is its place in the block-ordered list: block b's
    k-th member r has offs[b] + k == rank[r], so rank is a bijection of
    [0, d) that recovers each index's block and position."""
    oi, oo = P.partition(d, m, 9, categorical=cat)
    rank = G.gist_partition_inverse(np.asarray(oi, np.int32), np.asarray(oo, np.int64))
    for b, blk in enumerate(P.blocks_of(oi, oo)):
        for k, r in enumerate(blk):
            assert rank[r] == oo[b] + k
    assert sorted(rank.tolist()) == list(range(d))


def test_partition_inverse_errors():
    with pytest.raises(G.GistError):
        G.gist_partition_inverse(np.array([0, 2, 1, 2], np.int32), np.array([0, 2, 4]))
    with pytest.raises(G.GistError):
        G.gist_partition_inverse(np.arange(4, dtype=np.int32), np.array([0, 3, 2, 4]))
    with pytest.raises(G.GistError):
        G.gist_partition_inverse(np.array([0, 1, 5], np.int32), np.array([0, 3]))


@pytest.mark.parametrize("d,m,flags", [(10, 3, 0), (4, 0, 0), (4, 5, 0), (0, 1, 0), (8, 2, 4)])
def test_partition_errors(d, m, flags):
    with pytest.raises(G.GistError) as e:
        G.gist_partition(d, m, 0, flags)
    assert e.value.status == G.GIST_E_INVAL


def _same_csr(a, b, sage):
    assert a["n"] == b["n"] and a["nnz"] == b["nnz"]
    keys = ["rowptr", "col", "val", "node_map"] + (["t_rowptr", "t_col", "t_val"] if sage else [])
    for k in keys:
        x = np.asarray(a[k])
        y = np.asarray(b[k])
        if k.endswith("val"):
            assert x.dtype == np.float32 and y.dtype == np.float32
            assert np.array_equal(x.view(np.uint32), y.view(np.uint32)), k
        else:
            assert np.array_equal(x.astype(np.int64), y.astype(np.int64)), k


GRAPHS = {
    "er": lambda: erdos_renyi(300, 700, seed=1, clusters=6),
    "er_isolated": lambda: erdos_renyi(50, 20, seed=2, clusters=5),
    "chung_lu": lambda: chung_lu(3000, 2.5, 5.0, seed=3),
    "sbm": lambda: sbm(5000, 40, 25.0, 0.9, seed=4),
}


@pytest.mark.parametrize("gname", sorted(GRAPHS))
@pytest.mark.parametrize("norm", ["gcn", "sage", "theory"])
def test_minibatch_csr_bit_exact(gname, norm):
    g = GRAPHS[gname]()
    sels = [None]
    if g.n_clusters > 1:
        rng = np.random.default_rng(0)
        sels += [[0], list(rng.choice(g.n_clusters, 3, replace=False)),
                 [g.n_clusters - 1, 0, 0, g.n_clusters - 1]]
    for sel in sels:
        _same_csr(G.gist_build_minibatch_csr(g, sel, norm), MB.build(g, sel, norm),
                  norm == "sage")


def test_minibatch_csr_reddit_sized_batch():
    cfg = get_config("c3")
    g = cfg.make_graph()
    sel = cfg.minibatch(0, 0)
    a = G.gist_build_minibatch_csr(g, sel, "sage")
    _same_csr(a, MB.build(g, sel, "sage"), True)
    assert 3000 <= a["n"] <= 3200


def test_minibatch_csr_errors():
    g = erdos_renyi(30, 40, seed=1, clusters=3)
    for sel in ([], [3], [-1]):
        with pytest.raises(G.GistError) as e:
            G.gist_build_minibatch_csr(g, sel, "gcn")
        assert e.value.status == G.GIST_E_INVAL
    with pytest.raises(G.GistError):
        G.gist_build_minibatch_csr(g, None, 7)


def _prototypes():
    """name -> list of parameter texts, for every function the header declares."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    out = {}
    for m in re.finditer(r"\b(gist_[a-z_0-9]+)\s*\(([^;{]*?)\)\s*;", text):
        params = [p.strip() for p in m.group(2).split(",")]
        out[m.group(1)] = [] if params == ["void"] else params
    return out


def _ctype_kind(t):
    import ctypes as C
    if t is None:
        return None
    if t in (C.c_void_p, C.c_char_p) or getattr(t, "_type_", None) is not None and hasattr(t, "contents"):
        return "ptr"
    return {C.c_int64: "i64", C.c_int32: "i32", C.c_uint32: "u32", C.c_uint64: "u64",
            C.c_float: "f32", C.c_double: "f64", C.c_size_t: "u64"}.get(t, repr(t))


def _param_kind(p):
    if "*" in p:
        return "ptr"
    base = p.rsplit(" ", 1)[0].replace("const ", "").strip()
    if base.startswith("gist_"):      # the header's enums are int-sized
        return "i32"
    return {"int64_t": "i64", "int32_t": "i32", "int": "i32", "uint32_t": "u32", "uint64_t": "u64",
            "float": "f32", "double": "f64", "size_t": "u64", "gist_status": "i32"}[base]


def test_binding_signatures_match_header():
    """Every ctypes prototype of the binding has the header's arity and
    parameter kinds (pointer, width and signedness of integers, float)."""
    protos = _prototypes()
    assert sorted(protos) == declared_functions()
    for name, params in protos.items():
        f = getattr(G._lib, name)
        got = [_ctype_kind(t) for t in f.argtypes]
        want = [_param_kind(p) for p in params]
        assert got == want, (name, got, want)


# ---- LADIES sampler ------------------------------------------------------------------

def _same_ladies(lib, ora):
    L = len(ora["layers"])
    assert len(lib["layers"]) == L
    for l in range(L + 1):
        assert np.array_equal(np.asarray(lib["nodes"][l], np.int64),
                              np.asarray(ora["nodes"][l], np.int64)), l
    for l in range(L):
        a, b = lib["layers"][l], ora["layers"][l]
        assert (a["n"], a["n_in"], a["nnz"]) == (b["n"], b["n_in"], b["nnz"]), l
        for k in ("rowptr", "col", "t_rowptr", "t_col"):
            assert np.array_equal(np.asarray(a[k], np.int64), np.asarray(b[k], np.int64)), (l, k)
        for k in ("val", "t_val"):
            assert a[k].dtype == np.float32 and b[k].dtype == np.float32
            assert np.array_equal(a[k].view(np.uint32), b[k].view(np.uint32)), (l, k)


LADIES_GRAPHS = {
    "er": lambda: erdos_renyi(400, 1200, seed=5),
    "chung_lu": lambda: chung_lu(3000, 2.2, 6.0, seed=6),      # hubs: very uneven p
    "sbm": lambda: sbm(5000, 40, 25.0, 0.9, seed=7),
}


@pytest.mark.parametrize("gname", sorted(LADIES_GRAPHS))
@pytest.mark.parametrize("L,s,b", [(1, 64, 16), (2, 128, 40), (3, 50, 9), (2, 0, 12),
                                   (2, 1, 1), (2, 1000, 100)])
def test_ladies_sample_bit_exact(gname, L, s, b):
    from oracle import ladies as LD
    g = LADIES_GRAPHS[gname]()
    A = MB.build(g, None, "gcn")
    h = G.CsrHandle(A)
    rng = np.random.default_rng(L * 1000 + s + b)
    for seed in (0, 77, 2**64 - 1):
        batch = np.sort(rng.choice(g.n, b, replace=False))
        _same_ladies(G.gist_ladies_sample(h, batch, L, s, seed), LD.sample(A, batch, L, s, seed))


def test_ladies_sample_reddit_sized():
    """Batch of 512 output nodes, 512 draws per layer, on the 232,965-node graph."""
    from oracle import ladies as LD
    g = get_config("c3").make_graph()
    A = G.gist_build_minibatch_csr(g, None, "gcn")
    batch = np.sort(np.random.default_rng(11).choice(g.n, 512, replace=False))
    for L in (2, 3):
        lib = G.gist_ladies_sample(A, batch, L, 512, 1234 + L)
        _same_ladies(lib, LD.sample(A, batch, L, 512, 1234 + L))
        assert lib["layers"][0]["n_in"] > 512


def test_ladies_sample_edge_cases_and_errors():
    from oracle import ladies as LD
    g = erdos_renyi(50, 20, seed=2)             # many isolated nodes
    A = MB.build(g, None, "gcn")
    deg = np.diff(g.rowptr)
    iso = int(np.nonzero(deg == 0)[0][0])
    for batch in ([], [iso], sorted({0, iso, 49})):
        _same_ladies(G.gist_ladies_sample(A, batch, 2, 8, 3), LD.sample(A, batch, 2, 8, 3))
    h = G.CsrHandle(A)
    for batch in ([3, 2], [50], [-1], [4, 4]):
        with pytest.raises(G.GistError) as e:
            G.gist_ladies_sample(h, batch, 2, 8, 3)
        assert e.value.status == G.GIST_E_INVAL
    with pytest.raises(G.GistError):
        G.gist_ladies_sample(h, [1], 0, 8, 3)
    with pytest.raises(G.GistError):
        G.gist_ladies_sample(h, [1], 1, -1, 3)
    # capacity too small: NOMEM, and the sizes are still reported
    q, _ = G.ladies_layers(2)
    G.ladies_sample_into(h, [0, 1, 2], 2, 8, 3, q)
    need = [(q[l].n_in, q[l].nnz) for l in range(2)]
    arr, _ = G.ladies_layers(2, [(need[0][0] - 1, need[0][1]), need[1]])
    with pytest.raises(G.GistError) as e:
        G.ladies_sample_into(h, [0, 1, 2], 2, 8, 3, arr)
    assert e.value.status == G.GIST_E_NOMEM
    assert [(arr[l].n_in, arr[l].nnz) for l in range(2)] == need


def test_struct_layouts_match_header(tmp_path):
    """Offsets and sizes of every ctypes structure equal the C compiler's for
    the header's struct of the same name."""
    import ctypes as C
    import subprocess
    structs = [G.gist_graph, G.gist_csr, G.gist_csr_dev, G.gist_layer_desc, G.gist_gat_desc,
               G.gist_slice_set, G.gist_prof_entry, G.gist_ladies_layer]
    lines = ["#include <stdio.h>", "#include <stddef.h>", f'#include "{HEADER}"',
             "int main(void) {"]
    for st in structs:
        lines.append(f'  printf("%zu\\n", sizeof({st.__name__}));')
        for f in st._fields_:
            lines.append(f'  printf("%zu\\n", offsetof({st.__name__}, {f[0]}));')
    lines.append("  return 0; }")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", str(src), "-o", str(exe)], check=True)
    got = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True,
                                          check=True).stdout.split()]
    want = []
    for st in structs:
        want.append(C.sizeof(st))
        want += [getattr(st, f[0]).offset for f in st._fields_]
    assert got == want


def test_replay_and_copy_argument_errors():
    """Host-side checks of the replay / copy / event entry points (no device
    work is reached)."""
    import ctypes as C
    lib = G._lib
    assert lib.gist_capture_begin(None) == G.GIST_E_INVAL
    out = C.c_void_p()
    assert lib.gist_capture_end(None, C.byref(out)) == G.GIST_E_INVAL
    assert lib.gist_replay_launch(None, None, None, None, 0, None) == G.GIST_E_INVAL
    assert lib.gist_copy(None, None, None, 0, None) == G.GIST_E_INVAL
    assert lib.gist_event_create(None) == G.GIST_E_INVAL
    assert lib.gist_event_synchronize(None) == G.GIST_E_INVAL
    assert lib.gist_replay_destroy(None) == G.GIST_OK
    assert lib.gist_event_destroy(None) == G.GIST_OK
    assert lib.gist_softmax_xent_padded(None, 1, 1, None, None, None, None, None, None, 0) == \
        G.GIST_E_INVAL
