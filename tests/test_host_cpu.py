"""Host-side checks that need no GPU: the C-ABI library loads and exports every
entry point its header declares, and the HBM block cache bookkeeping (LRU,
never evicting a block of the current request, hit/miss accounting)."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ls_ffn.h")
CSRC = os.path.join(ROOT, "paper_2609_03079_amd", "csrc")


def _declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:ls_status|const char\*)\s+(ls_\w+)\s*\(", text, re.M)))


def test_header_declares_the_boundary():
    names = _declared_functions()
    for required in ("ls_ffn_create", "ls_predict", "ls_select_blocks", "ls_sparse_ffn_step",
                     "ls_stream_weights", "ls_decode_step", "ls_ffn_set_layer", "ls_ffn_destroy",
                     "ls_last_error"):
        assert required in names


def test_library_exports_every_declared_symbol():
    import paper_2609_03079_amd as lsffn
    if not os.path.exists(lsffn.LIB_PATH):
        from paper_2609_03079_amd import build as b
        b.build()
    lib = ctypes.CDLL(lsffn.LIB_PATH)
    for name in _declared_functions():
        assert hasattr(lib, name), name
    assert set(_declared_functions()) == set(lsffn.EXPORTS)
    # the error text for a failed create is available without a context
    lsffn.load()
    desc = lsffn.LsFfnDesc(0, 64, 64, 8, 64, 1, 0, 0, 0, 0, 0, None, 0)
    out = ctypes.c_void_p()
    st = lsffn.load().ls_ffn_create(ctypes.byref(desc), ctypes.byref(out))
    assert st == lsffn.LS_E_INVAL and not out.value
    assert b"n_layers" in lsffn.load().ls_last_error(None)


def test_binding_fails_loudly_without_library(tmp_path, monkeypatch):
    import paper_2609_03079_amd as lsffn
    monkeypatch.setattr(lsffn, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(lsffn, "_lib", None)
    with pytest.raises(RuntimeError):
        lsffn.load()


@pytest.fixture(scope="module")
def bc(tmp_path_factory):
    out = tmp_path_factory.mktemp("bc") / "libbc.so"
    subprocess.run(["g++", "-O1", "-std=c++17", "-shared", "-fPIC", "-o", str(out),
                    os.path.join(CSRC, "block_cache_capi.cpp")], check=True)
    lib = ctypes.CDLL(str(out))
    lib.bc_create.restype = ctypes.c_void_p
    lib.bc_create.argtypes = [ctypes.c_int64, ctypes.c_int, ctypes.c_int]
    lib.bc_destroy.argtypes = [ctypes.c_void_p]
    lib.bc_request.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
                               ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
    lib.bc_slot_table.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
    lib.bc_invalidate_layer.argtypes = [ctypes.c_void_p, ctypes.c_int]
    return lib


class Cache:
    def __init__(self, lib, slots, L, n_blk):
        self.lib, self.L, self.n_blk = lib, L, n_blk
        self.h = lib.bc_create(slots, L, n_blk)

    def request(self, layer, blocks, protect=-1):
        b = np.ascontiguousarray(blocks, np.int32)
        counts = np.zeros(3, np.int64)
        fills = np.zeros(4 * max(1, len(b)), np.int32)
        nf = np.zeros(1, np.int32)
        ok = self.lib.bc_request(self.h, layer, b.ctypes.data, len(b), counts.ctypes.data,
                                 fills.ctypes.data, nf.ctypes.data, protect)
        return ok, counts.tolist(), fills[:4 * nf[0]].reshape(-1, 4).tolist()

    def table(self, layer):
        t = np.zeros(self.n_blk, np.int32)
        self.lib.bc_slot_table(self.h, layer, t.ctypes.data)
        return t


def test_block_cache_accounting_and_lru(bc):
    c = Cache(bc, 4, 2, 10)
    ok, cnt, fills = c.request(0, [3, 1, 4])
    assert ok and cnt == [0, 3, 0]
    assert all(f[3] == -1 for f in fills)  # empty slots: nothing evicted
    assert [f[:2] for f in fills] == [[0, 3], [1, 1], [2, 4]]  # misses in priority order
    ok, cnt, _ = c.request(0, [1, 5])
    assert ok and cnt == [1, 1, 0]
    # cache full: {3,1,4,5}; LRU order oldest -> newest: 3, 4, 1, 5
    ok, cnt, fills = c.request(1, [7])
    assert ok and cnt == [0, 1, 1]
    assert fills[0][3] == 0  # the slot it took held a block of layer 0
    t0 = c.table(0)
    assert t0[3] == -1 and t0[1] >= 0 and t0[4] >= 0 and t0[5] >= 0
    # a request never evicts its own blocks, even when they are the least recent
    ok, cnt, fills = c.request(0, [4, 9, 8])
    assert ok and cnt == [1, 2, 2]
    t0 = c.table(0)
    assert t0[4] >= 0 and t0[9] >= 0 and t0[8] >= 0
    slots = [s for s in t0 if s >= 0] + [s for s in c.table(1) if s >= 0]
    assert len(slots) == len(set(slots)) == 4


def test_block_cache_properties_random(bc):
    rng = np.random.default_rng(0)
    S, L, N = 7, 3, 12
    c = Cache(bc, S, L, N)
    for it in range(400):
        layer = int(rng.integers(L))
        n = int(rng.integers(0, S + 1))
        req = rng.integers(0, N, size=n).astype(np.int32)  # duplicates allowed
        before = c.table(layer).copy()
        ok, (hits, misses, ev), fills = c.request(layer, req)
        assert ok
        assert hits + misses == n
        assert misses == len(fills) == len(set(int(b) for b in req if before[b] < 0))
        t = c.table(layer)
        assert all(t[b] >= 0 for b in req)
        assert [f[0] for f in fills] == sorted(f[0] for f in fills)
        # a fill that evicted reports the layer whose block the slot held
        assert sum(1 for f in fills if f[3] >= 0) == ev and all(-1 <= f[3] < L for f in fills)
        occupied = [s for l in range(L) for s in c.table(l) if s >= 0]
        assert len(occupied) == len(set(occupied)) <= S
    ok, _, _ = c.request(0, list(range(S + 1)))
    assert not ok  # larger than the cache


def test_block_cache_protected_layer_and_failed_request(bc):
    c = Cache(bc, 5, 3, 10)
    assert c.request(0, [0, 1, 2])[0]
    assert c.request(1, [5, 6])[0]          # cache full; layer 0's blocks are the least recent
    ok, cnt, fills = c.request(2, [7, 8], protect=0)
    assert ok and cnt == [0, 2, 2] and all(f[3] == 1 for f in fills)  # only layer 1 gave way
    assert all(c.table(0)[[0, 1, 2]] >= 0)
    before = [c.table(l).copy() for l in range(3)]
    ok, _, _ = c.request(1, [3, 4, 9], protect=0)  # 3 misses, 2 takeable slots: refused
    assert not ok
    assert all(np.array_equal(c.table(l), before[l]) for l in range(3))  # nothing changed hands
    ok, cnt, fills = c.request(1, [3, 4, 9])      # without protection it fits
    assert ok and cnt == [0, 3, 3] and [f[3] for f in fills] == [0, 0, 0]  # the least recent: layer 0


def test_block_cache_invalidate(bc):
    c = Cache(bc, 3, 1, 5)
    c.request(0, [0, 1])
    bc.bc_invalidate_layer(c.h, 0)
    assert np.all(c.table(0) == -1)
    ok, cnt, _ = c.request(0, [0, 1, 2])
    assert ok and cnt == [0, 3, 0]


def test_zero_skip_byte_counts():
    """The bench's zero-skip byte accounting on hand-made activations: no active neuron costs the
    gate rows alone, all active costs the whole blocks, one active neuron adds its up row plus
    one group of V down rows (V = 16 / element size)."""
    import importlib.util
    import lsgen
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    bench = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(bench)
    cfg = lsgen.CONFIGS["llama2_7b_ffn"]
    U, blk, row, V = 3, cfg.block, cfg.d_model * cfg.elem_bytes, 16 // cfg.elem_bytes
    z = np.zeros((2, U * blk), np.float32)
    assert bench.zero_skip_bytes(cfg, z, U) == (3 * U * blk * row, U * blk * row, U * blk * row)
    full = np.ones_like(z)
    assert bench.zero_skip_bytes(cfg, full, U) == (3 * U * blk * row,) * 3
    one = z.copy()
    one[1, blk + 5] = -0.25  # one neuron of the second entry, active for the second token only
    blockb, neuron, kernel = bench.zero_skip_bytes(cfg, one, U)
    assert neuron == U * blk * row + 2 * row
    assert kernel == U * blk * row + row + V * row
    neg_zero = z.copy()
    neg_zero[0, 7] = -0.0  # a signed zero is no activation
    assert bench.zero_skip_bytes(cfg, neg_zero, U)[2] == U * blk * row
    assert bench.zero_skip_bytes(cfg, z[:, :0], 0) == (0, 0, 0)


# ---- sanitizer builds of the host code (CPU only) ----

NATIVE = os.path.join(ROOT, "tests", "native")


def _build_and_run(tmp_path, cmd_build, exe):
    r = subprocess.run(cmd_build, capture_output=True, text=True)
    if r.returncode != 0:
        pytest.skip(f"sanitizer build not available here: {r.stderr[-300:]}")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr


def test_block_cache_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    """The host-resident block cache under random request sequences, built with
    AddressSanitizer and UndefinedBehaviorSanitizer: its invariants hold and no memory or UB
    error is reported."""
    exe = str(tmp_path / "cache_fuzz")
    _build_and_run(tmp_path, ["g++", "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined",
                              "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-o", exe,
                              os.path.join(NATIVE, "cache_fuzz.cpp")], exe)


def test_threaded_oracle_under_thread_sanitizer(tmp_path):
    """The oracle's thread-split layer step (used to time it on every host core), built with
    ThreadSanitizer: no data race is reported and it equals the single-thread step bitwise."""
    exe = str(tmp_path / "oracle_mt_race")
    _build_and_run(tmp_path, ["gcc", "-O1", "-g", "-std=c11", "-fsanitize=thread", "-o", exe,
                              os.path.join(ROOT, "oracle", "ls_oracle.c"),
                              os.path.join(NATIVE, "oracle_mt_race.c"), "-lm", "-lpthread"], exe)
