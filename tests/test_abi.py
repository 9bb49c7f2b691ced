"""The C-ABI library loads, exports every symbol include/evox.h declares, and
rejects invalid arguments on the host side (no GPU needed: validation runs
before any HIP call)."""
import ctypes
import os
import re

import pytest

from conftest import ROOT

HEADER = os.path.join(ROOT, "include", "evox.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(evox_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def evox():
    import paper_2301_12457_amd as m
    if not os.path.exists(m.LIB_PATH):
        from paper_2301_12457_amd import build
        build.build()
    return m


def test_exports_every_declared_symbol(evox):
    L = evox.lib()
    names = declared_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(L, n), n
    assert sorted(evox.EXPORTS) == names


def test_struct_layouts_match_header(evox):
    # evox_params: 2 x int32, 3 x int64, 9 floats, 2 x int32, 8 floats, (pad), uint64
    assert ctypes.sizeof(evox.Params) == 136
    assert evox.Params.x_init.offset == 72
    assert evox.Params.de_f.offset == 84
    assert evox.Params.es_lr.offset == 96
    assert evox.Params.pgpe_max_change.offset == 104
    assert evox.Params.seed.offset == 112
    assert ctypes.sizeof(evox.Buffers) == 14 * 8


def test_row_layout_policy(evox):
    # PSO / evaluation: the fewest lanes that hold a row in <= 2 float4 per lane
    assert evox.row_layout(1) == (4, 1)
    assert evox.row_layout(10) == (4, 1)
    assert evox.row_layout(100) == (16, 2)
    assert evox.row_layout(1000) == (128, 2)
    assert evox.row_layout(1001) == (128, 2)
    assert evox.row_layout(32768) == (1024, 8)
    cap = lambda G: 8 if G == 1024 else 2
    for D in list(range(1, 300)) + [1023, 1024, 1025, 4096, 4097, 16385, 32767]:
        G, nit = evox.row_layout(D)
        c4 = (D + 3) // 4
        assert G * nit >= c4 and nit <= cap(G)
        assert G == 4 or (G // 2) * cap(G // 2) < c4      # no smaller group holds the row
    with pytest.raises(evox.EvoxError):
        evox.row_layout(32769)
    # CSO: one chunk per lane while it fits
    C = evox.LAYOUT_CSO
    assert evox.row_layout(100, C) == (32, 1)
    assert evox.row_layout(10, C) == (4, 1)
    assert evox.row_layout(4096, C) == (1024, 1)
    assert evox.row_layout(4100, C) == (1024, 2)
    assert evox.row_layout(32768, C) == (1024, 8)
    # evox_eval: up to 4 chunks per lane (one wave per row at D = 1000)
    E = evox.LAYOUT_EVAL
    assert evox.row_layout(1000, E) == (64, 4)
    assert evox.row_layout(100, E) == (8, 4)
    assert evox.row_layout(32768, E) == (1024, 8)
    with pytest.raises(evox.EvoxError):
        evox.row_layout(100, 3)


def test_default_pitch_policy(evox):
    L = evox.lib()
    P, C = evox.PSO, evox.CSO
    for D, want in [(1, 4), (10, 12), (100, 100), (511, 512), (512, 512), (1000, 1024), (1025, 1056),
                    (32768, 32768)]:
        assert L.evox_default_ldx(P, D) == want, (D, want)
    for D, want in [(1, 4), (10, 12), (63, 64), (64, 64), (65, 68), (100, 100), (1000, 1000), (1001, 1004)]:
        assert L.evox_default_ldx(C, D) == want, (D, want)
    for D in (10, 100, 1000):
        for algo in (evox.DE, evox.ES, evox.PGPE, evox.MAES, evox.NSGA2):
            assert L.evox_default_ldx(algo, D) == L.evox_default_ldx(P, D)
    for algo, D in [(P, 0), (C, 32769), (7, 10)]:
        assert L.evox_default_ldx(algo, D) == 0
    assert evox.make_params(C, evox.GRIEWANK, 10, 100, -1, 1).ldx == 100
    assert evox.make_params(P, evox.GRIEWANK, 10, 100, -1, 1).ldx == 100
    with pytest.raises(evox.EvoxError):
        evox.pitch(0)


def test_permutation_scratch(evox):
    L = evox.lib()
    assert L.evox_permutation_scratch_bytes(0, 1) == 0
    assert L.evox_permutation_scratch_bytes(2**24 + 1, 1) == 0
    assert L.evox_permutation_scratch_bytes(100, 9) == 0
    one, eight = L.evox_permutation_scratch_bytes(10**6, 1), L.evox_permutation_scratch_bytes(10**6, 8)
    assert one >= 8 * 10**6 and eight >= 8 * one - 8 * 4096


def test_scratch_bytes(evox):
    p = evox.make_params(evox.PSO, evox.SPHERE, 100, 10, -1, 1)
    assert evox.evox_scratch_bytes(p) > 0
    c = evox.make_params(evox.CSO, evox.GRIEWANK, 1_000_000, 100, -600, 600)
    n = evox.evox_scratch_bytes(c)
    assert n >= 3 * 4 * 1_000_000  # keys, indices, permutation
    bad = evox.make_params(evox.PSO, 9, 100, 10, -1, 1)
    assert evox.evox_scratch_bytes(bad) == 0


@pytest.mark.parametrize("algo,field,value", [(0, "N", 0), (0, "D", 0), (0, "D", 40000),
                                              (0, "ldx", 6), (0, "fn_id", 6), (0, "algo", 5),
                                              (1, "N", 1), (1, "N", 2**24 + 1), (0, "x_init", 2),
                                              (1, "x_init", -1), (2, "N", 3), (2, "D", 0),
                                              (3, "N", 7), (3, "N", 16386), (3, "N", 0), (4, "N", 5)])
def test_create_rejects_bad_params(evox, algo, field, value):
    p = evox.make_params(algo, evox.SPHERE, 8, 5, -1, 1)
    setattr(p, field, value)
    b = evox.Buffers()
    h = ctypes.c_void_p()
    rc = evox.lib().evox_state_create(ctypes.byref(p), ctypes.byref(b), None, ctypes.byref(h))
    assert rc == evox.EINVAL
    assert evox.lib().evox_last_error().decode()
    assert not h.value


def test_create_rejects_missing_and_misaligned_buffers(evox):
    p = evox.make_params(evox.PSO, evox.SPHERE, 8, 5, -1, 1)
    b = evox.Buffers()
    h = ctypes.c_void_p()
    L = evox.lib()
    assert L.evox_state_create(ctypes.byref(p), ctypes.byref(b), None, ctypes.byref(h)) == evox.EINVAL
    need = evox.evox_scratch_bytes(p)
    b = evox.Buffers(x=0x1000, v=0x2000, pbest=0x3000, pfit=0x4000, gbest=0x5008, scratch=0x10000,
                     scratch_bytes=need)
    assert L.evox_state_create(ctypes.byref(p), ctypes.byref(b), None, ctypes.byref(h)) == evox.EALIGN
    b.gbest = 0x5000
    b.scratch_bytes = need - 1
    assert L.evox_state_create(ctypes.byref(p), ctypes.byref(b), None, ctypes.byref(h)) == evox.ENOSPC
    c = evox.make_params(evox.CSO, evox.SPHERE, 1, 5, -1, 1)    # CSO needs a pair
    assert L.evox_state_create(ctypes.byref(c), ctypes.byref(b), None, ctypes.byref(h)) == evox.EINVAL


def test_eval_rejects_bad_args(evox):
    L = evox.lib()
    assert L.evox_eval(7, None, 1, 1, None, None) == evox.EINVAL
    assert L.evox_eval(0, None, 1, 0, None, None) == evox.EINVAL
    assert L.evox_eval(0, None, 5, 3, None, None) == evox.EINVAL
    assert L.evox_eval(0, None, 0, 3, None, None) == evox.OK     # empty: nothing to do
    assert L.evox_eval_ld(0, None, 0, 8, 4, None, None) == evox.EINVAL
    assert L.evox_eval_argmin(0, None, 0, 3, 3, None, None, None, None, 0, None) == evox.EINVAL
    assert L.evox_copy(None, None, 0, None) == evox.OK
    assert L.evox_copy(None, None, 5, None) == evox.EINVAL
    assert L.evox_copy(0x1000, 0x2000, -1, None) == evox.EINVAL
    assert L.evox_copy(0x1004, 0x2000, 5, None) == evox.EALIGN
    assert L.evox_pso_stream(None, None, None, 0, None) == evox.OK
    assert L.evox_pso_stream(None, None, None, 8, None) == evox.EINVAL                 # null buffers
    assert L.evox_pso_stream(0x1000, 0x2000, 0x3000, 6, None) == evox.EINVAL         # n % 4
    assert L.evox_pso_stream(0x1000, 0x2000, 0x3000, -4, None) == evox.EINVAL        # n < 0
    assert L.evox_pso_stream(0x1000, 0x2004, 0x3000, 8, None) == evox.EALIGN
    assert L.evox_fill_normal(1, 0, 3, 4, 0.0, 1.0, None, None) == evox.OK     # empty
    assert L.evox_fill_normal(1, 5, 3, 4, 0.0, 1.0, None, None) == evox.EINVAL
    assert L.evox_fill_normal(1, 5, 5, 4, 0.0, 1.0, 0x1000, None) == evox.EINVAL
    assert L.evox_fill_normal(1, 5, 3, 6, 0.0, 1.0, 0x1000, None) == evox.EINVAL
    assert L.evox_fill_normal(1, -1, 3, 4, 0.0, 1.0, 0x1000, None) == evox.EINVAL
    assert L.evox_fill_normal(1, 5, 3, 4, 0.0, 1.0, 0x1004, None) == evox.EALIGN


def test_null_state_is_rejected(evox):
    L = evox.lib()
    assert L.evox_pso_step(None, 1) == evox.EINVAL
    assert L.evox_cso_step(None, 1) == evox.EINVAL
    assert L.evox_de_step(None, 1) == evox.EINVAL
    assert L.evox_es_step(None, 1) == evox.EINVAL
    assert L.evox_pgpe_step(None, 1) == evox.EINVAL
    assert L.evox_best(None, None, None, None) == evox.EINVAL
    assert L.evox_generation(None) == -1
    assert L.evox_set_generation(None, 5) == evox.EINVAL


def test_pair_move_validates_before_any_gpu_call(evox):
    L = evox.lib()
    f = ctypes.c_void_p(0x1000)
    assert L.evox_pair_move(f, f, 1, 10, 12, f, None) == evox.EINVAL               # N < 2
    assert L.evox_pair_move(f, f, 10, 0, 12, f, None) == evox.EINVAL               # D < 1
    assert L.evox_pair_move(f, f, 10, 10, 14, f, None) == evox.EINVAL              # ldx % 4
    assert L.evox_pair_move(f, f, 10, 10, 12, None, None) == evox.EINVAL           # winner_of
    assert L.evox_pair_move(ctypes.c_void_p(0x1004), f, 10, 10, 12, f, None) == evox.EALIGN


def test_noalloc_entry_point_validates_before_any_gpu_call(evox):
    L = evox.lib()
    f = ctypes.c_void_p(0x1000)
    assert L.evox_eval_argmin_noalloc(0, f, 0, 10, 10, f, f, f, None) == evox.EINVAL    # N < 1
    assert L.evox_eval_argmin_noalloc(9, f, 5, 10, 10, f, f, f, None) == evox.EINVAL    # fn_id
    assert L.evox_eval_argmin_noalloc(0, f, 5, 10, 8, f, f, f, None) == evox.EINVAL     # ldx < D
    assert L.evox_eval_argmin_noalloc(0, f, 5, 10, 10, f, None, f, None) == evox.EINVAL  # outputs
    assert L.evox_eval_argmin_noalloc(0, None, 5, 10, 10, f, f, f, None) == evox.EINVAL  # X
    assert "X and out are required" in L.evox_last_error().decode()
    assert L.evox_strerror(evox.ENOSPC).decode() == "scratch buffer too small"
