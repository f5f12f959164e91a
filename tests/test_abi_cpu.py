"""Host-only checks of the C ABI library: it loads, exports every symbol the
header declares, validates trees, numbers nodes canonically, builds trees
from sequences, and rejects bad arguments before touching a GPU."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle as O
import paper_2607_02525_amd as P
import peek_workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "peek.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(peek_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 11
    out = subprocess.run(["nm", "-D", "--defined-only", P.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (peek_\w+)", out))
    assert set(names) <= exported, set(names) - exported
    bound = {name for name, _, _ in P.EXPORTS}
    assert set(names) == bound


def test_library_is_built_for_gfx950_only():
    blob = open(P.LIB_PATH, "rb").read()
    targets = set(re.findall(rb"amdgcn-amd-amdhsa--(gfx\w+)", blob))
    assert targets == {b"gfx950"}


def test_abi_version():
    assert P.peek_abi_version() == 1


@pytest.mark.parametrize("seed", range(10))
def test_canonical_ids_match_the_oracle(seed):
    w = W.random_tree_case(seed, n_nodes=60, n=4, vocab=7, max_edge=4)
    ours = P.peek_tree_canonical_ids(*w.cache_tree)
    theirs = O.Tree.from_description(*w.cache_tree).canonical_ids(len(w.cache_tree[0]))
    assert np.array_equal(ours, theirs)


def _desc(parent, edges):
    tok, off = W.pack([np.asarray(e, dtype=np.int32) for e in edges])
    return np.asarray(parent, dtype=np.int32), off, tok


@pytest.mark.parametrize("parent,edges", [
    ([-1, 0, 0], [[], [1, 2], [1, 3]]),
    ([-1, 0, 0], [[], [1], []]),
    ([-1, -1], [[], []]),
    ([0, 0], [[1], [2]]),
    ([-1, 2, 1], [[], [1], [2]]),
    ([-1, 5], [[], [1]]),
    ([-1, 0], [[4], [1]]),
])
def test_invalid_trees_are_rejected(parent, edges):
    with pytest.raises(P.PeekError) as e:
        P.peek_tree_canonical_ids(*_desc(parent, edges))
    assert e.value.status == P.PEEK_ERR_INVALID_TREE
    assert P.peek_last_error()


def test_signed_token_order_and_extremes():
    # children ordered by signed first token: INT32_MIN < -1 < 0 < INT32_MAX
    lo, hi = np.iinfo(np.int32).min, np.iinfo(np.int32).max
    parent, off, tok = _desc([-1, 0, 0, 0, 0], [[], [hi, 1], [0], [lo], [-1, 5]])
    assert list(P.peek_tree_canonical_ids(parent, off, tok)) == [0, 4, 3, 1, 2]


def _same_tree(a, b):
    pa, oa, ta = a
    pb, ob, tb = b
    return np.array_equal(pa, pb) and np.array_equal(oa, ob) and np.array_equal(ta, tb)


@pytest.mark.parametrize("seed,vocab", [(s, v) for s in range(8) for v in (2, 3, 50)])
def test_tree_from_sequences_matches_the_oracle(seed, vocab):
    w = W.random_case(seed, n=5, n_cached=30, vocab=vocab, max_len=30)
    ours = P.peek_tree_from_sequences(*w.cache_sequences)
    par, depth, eoff, etok = O.Tree.from_sequences(*w.cache_sequences).export()
    assert _same_tree(ours, (par, eoff, etok))


@pytest.mark.parametrize("name", ["tiny", "rag", "agentic", "nosharing"])
def test_tree_from_sequences_on_workload_caches(name):
    w = W.make(name, 42)
    ours = P.peek_tree_from_sequences(*w.cache_sequences)
    par, depth, eoff, etok = O.Tree.from_sequences(*w.cache_sequences).export()
    assert _same_tree(ours, (par, eoff, etok))


def test_tree_from_sequences_edge_cases():
    # no sequences, only empty ones, duplicates, a prefix of another
    for seqs in ([], [[]], [[], []], [[1, 2], [1, 2]], [[1, 2, 3], [1, 2]], [[5], [5, 6], [5, 6, 7]]):
        tok, off = W.pack([np.asarray(s, np.int32) for s in seqs])
        ours = P.peek_tree_from_sequences(tok, off)
        par, depth, eoff, etok = O.Tree.from_sequences(tok, off).export()
        assert _same_tree(ours, (par, eoff, etok)), seqs


def test_argument_errors_before_any_gpu_work():
    lib = P._lib
    # NULL cache
    assert lib.peek_lpm_batch(None, 1, None, None, 16, None, None, None, None) == P.PEEK_ERR_INVALID_ARGUMENT
    assert "NULL" in P.peek_last_error()
    assert lib.peek_cache_stats(None, None, None, None, None, None) == P.PEEK_ERR_INVALID_ARGUMENT
    assert lib.peek_cache_free(None) == P.PEEK_OK
    # threshold < 1, n < 0, mismatched cluster outputs
    assert lib.peek_queue_signals(None, 4, None, None, None, None, 0, None, None, None, None, 0, None) \
        == P.PEEK_ERR_INVALID_ARGUMENT
    assert lib.peek_queue_signals(None, -1, None, None, None, None, 8, None, None, None, None, 0, None) \
        == P.PEEK_ERR_INVALID_ARGUMENT
    fake = ctypes.c_void_p(0x1000)
    assert lib.peek_queue_signals(None, 4, fake, fake, None, None, 8, fake, None, None, None, 0, None) \
        == P.PEEK_ERR_INVALID_ARGUMENT
    # workspace too small for the cluster pass (checked before any launch)
    need = P.peek_queue_signals_workspace(4, 0)
    assert need > 0
    assert lib.peek_queue_signals(None, 4, fake, fake, None, None, 8, fake, fake, None, fake, need - 1, None) \
        == P.PEEK_ERR_WORKSPACE_TOO_SMALL
    # demand without a cache
    assert lib.peek_queue_signals(None, 4, fake, fake, fake, None, 8, None, None, fake, fake, need, None) \
        == P.PEEK_ERR_INVALID_ARGUMENT
    # cLPM signals: need the cluster outputs, d_h for the section, theta >= 0
    assert lib.peek_clpm_signals(None, 4, fake, fake, fake, None, None, 8, 0, 32, None, None, None, fake, fake,
                                 fake, fake, need, None) == P.PEEK_ERR_INVALID_ARGUMENT
    assert "d_cluster_id" in P.peek_last_error()
    assert lib.peek_clpm_signals(None, 4, fake, fake, None, None, None, 8, 0, 32, fake, fake, None, None, fake,
                                 None, fake, need, None) == P.PEEK_ERR_INVALID_ARGUMENT
    assert "d_h" in P.peek_last_error()
    assert lib.peek_clpm_signals(None, 4, fake, fake, fake, None, None, 8, 0, -1, fake, fake, None, fake, fake,
                                 fake, fake, need, None) == P.PEEK_ERR_INVALID_ARGUMENT
    assert "theta" in P.peek_last_error()
    assert lib.peek_clpm_signals(None, 4, fake, fake, fake, None, None, 8, 0, 32, fake, fake, None, fake, fake,
                                 fake, fake, need - 1, None) == P.PEEK_ERR_WORKSPACE_TOO_SMALL


def test_noalloc_signals_errors_before_any_gpu_work():
    lib = P._lib
    fake = ctypes.c_void_p(0x1000)
    assert lib.peek_queue_signals_noalloc(None, -1, None, None, None, None, 8, None, None, None, None) \
        == P.PEEK_ERR_INVALID_ARGUMENT
    assert lib.peek_queue_signals_noalloc(None, 4, fake, fake, None, None, 0, fake, fake, None, None) \
        == P.PEEK_ERR_INVALID_ARGUMENT
    # a queue whose scratch exceeds the static array is refused with its size
    n = 300000
    assert P.peek_queue_signals_workspace(n, 0) > P.PEEK_NOALLOC_SCRATCH_BYTES
    assert lib.peek_queue_signals_noalloc(None, n, fake, fake, None, None, 8, fake, fake, None, None) \
        == P.PEEK_ERR_WORKSPACE_TOO_SMALL
    assert "static scratch" in P.peek_last_error()
    # the header's maximum and the binding's agree
    with open(HEADER) as f:
        assert "#define PEEK_NOALLOC_SCRATCH_BYTES (32u << 20)" in f.read()
    assert P.PEEK_NOALLOC_SCRATCH_BYTES == 32 << 20


def test_block_table_argument_errors_before_any_gpu_work():
    lib = P._lib
    parent = np.array([-1, 0, 0], dtype=np.int32)
    eoff = np.array([0, 0, 3, 5], dtype=np.int64)
    etok = np.array([1, 2, 3, 4, 5], dtype=np.int32)
    out = ctypes.c_void_p(0x1234)
    args = (3, parent.ctypes.data_as(P._i32p), eoff.ctypes.data_as(P._i64p), etok.ctypes.data_as(P._i32p))
    for bad in (0, 1, 2, 3, 12, 512, -16):
        out = ctypes.c_void_p(0x1234)
        assert lib.peek_block_table_build(*args, bad, None, ctypes.byref(out)) == P.PEEK_ERR_INVALID_ARGUMENT
        assert "block_size" in P.peek_last_error()
        assert out.value is None
    assert lib.peek_block_table_build(*args, 16, None, None) == P.PEEK_ERR_INVALID_ARGUMENT
    # siblings with the same first token: not a radix tree
    etok2 = np.array([1, 2, 3, 1, 5], dtype=np.int32)
    assert lib.peek_block_table_build(3, parent.ctypes.data_as(P._i32p), eoff.ctypes.data_as(P._i64p),
                                      etok2.ctypes.data_as(P._i32p), 16, None, ctypes.byref(out)) \
        == P.PEEK_ERR_INVALID_TREE
    assert lib.peek_block_lpm_batch(None, 1, None, None, None, None) == P.PEEK_ERR_INVALID_ARGUMENT
    assert lib.peek_block_table_stats(None, None, None, None) == P.PEEK_ERR_INVALID_ARGUMENT
    assert lib.peek_block_table_free(None) == P.PEEK_OK


def test_offline_order_argument_errors_before_any_gpu_work():
    lib = P._lib
    fake = ctypes.c_void_p(0x1000)
    need = P.peek_offline_order_workspace(8)
    assert need > 0 and P.peek_offline_order_workspace(0) == 0 and P.peek_offline_order_workspace(-1) == 0
    assert P.peek_offline_order_workspace(64) > need
    assert lib.peek_offline_order(-1, fake, fake, 128, fake, fake, need, None) == P.PEEK_ERR_INVALID_ARGUMENT
    assert lib.peek_offline_order(8, fake, fake, -1, fake, fake, need, None) == P.PEEK_ERR_INVALID_ARGUMENT
    assert "depth_limit" in P.peek_last_error()
    assert lib.peek_offline_order(1 << 30, fake, fake, 128, fake, fake, need, None) == P.PEEK_ERR_INVALID_ARGUMENT
    assert "2^30" in P.peek_last_error()
    assert lib.peek_offline_order(0, None, None, 128, None, None, 0, None) == P.PEEK_OK
    assert lib.peek_offline_order(8, fake, fake, 128, None, fake, need, None) == P.PEEK_ERR_INVALID_ARGUMENT
    assert lib.peek_offline_order(8, fake, fake, 128, fake, None, need, None) == P.PEEK_ERR_INVALID_ARGUMENT
    assert lib.peek_offline_order(8, fake, fake, 128, fake, fake, need - 1, None) == P.PEEK_ERR_WORKSPACE_TOO_SMALL
    assert lib.peek_offline_order(8, fake, fake, 128, fake, ctypes.c_void_p(0x1010), need, None) \
        == P.PEEK_ERR_INVALID_ARGUMENT


def test_workspace_grows_with_the_queue_and_the_cache():
    a = P.peek_queue_signals_workspace(1000, 10)
    assert P.peek_queue_signals_workspace(2000, 10) > a
    assert P.peek_queue_signals_workspace(1000, 100000) > a
    assert P.peek_queue_signals_workspace(-1, 0) == 0


def test_binding_checks_tensors_before_the_call():
    """The binding refuses what the C entry points cannot check: element
    type, contiguity and host-resident tensors (the first argument checked
    here; the GPU tests cover the outputs)."""
    torch = pytest.importorskip("torch")
    import paper_2607_02525_amd as P

    class NoCache:
        handle = None

    tok = torch.zeros(16, dtype=torch.int32)
    off = torch.arange(0, 20, 4, dtype=torch.int64)
    h = torch.zeros(4, dtype=torch.int32)
    with pytest.raises(TypeError, match="offsets"):
        P.peek_lpm_batch(NoCache(), tok, off.to(torch.int32), 4, h)
    with pytest.raises(TypeError, match="tokens"):
        P.peek_lpm_batch(NoCache(), tok.to(torch.int64), off, 4, h)
    with pytest.raises(ValueError, match="contiguous"):
        P.peek_block_lpm_batch(None, torch.zeros(32, dtype=torch.int32)[::2], off, h)
    with pytest.raises(ValueError, match="device tensor"):
        P.peek_offline_order(tok, off, 128, h, None)


def test_one_hip_runtime_per_process():
    # the package binds libpeek.so to torch's HIP runtime; a second runtime
    # loaded beside it finds no device on a GPU machine
    code = ("import paper_2607_02525_amd\n"
            "maps = open('/proc/self/maps').read().splitlines()\n"
            "print(len({l.split()[-1] for l in maps if 'libamdhip64' in l}))\n")
    out = subprocess.run(["python", "-c", code], capture_output=True, text=True, cwd=ROOT, check=True).stdout
    assert out.strip() == "1"
