"""The C-ABI library loads, exports every declared symbol and validates its
arguments on the host before any HIP call (runs without a GPU)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2510_11683_amd", "libbgpo.so")


def _declared():
    names = set()
    for h in ("bgpo.h", "bgpo_testing.h", "bgpo_stats.h"):
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names |= set(re.findall(r"\b(bgpo_\w+)\s*\(", src))
    return names


pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libbgpo.so not built")


def test_exports_every_declared_symbol():
    declared = _declared()
    assert {"bgpo_elbo_fwd", "bgpo_elbo_bwd_accumulate", "bgpo_workspace_size",
            "bgpo_sample_masks", "bgpo_status_string", "bgpo_version"} <= declared
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (bgpo_\w+)", out))
    missing = declared - exported
    assert not missing, missing
    lib = ctypes.CDLL(LIB)
    for n in declared:
        assert hasattr(lib, n)


@pytest.fixture(scope="module")
def b():
    from paper_2510_11683_amd import bgpo
    return bgpo


def _prob(b, **kw):
    base = dict(B=8, L=512, d=4096, V=126464, n_t=64, j_begin=0, j_count=None, seed=1)
    base.update(kw)
    return b.Problem(**base)


def test_status_strings(b):
    for s in (0, -1, -2, -3, -4, -5):
        assert b._lib.bgpo_status_string(s)
    assert b"budget" in b._lib.bgpo_status_string(-5)
    assert b"unknown" in b._lib.bgpo_status_string(-99)


def test_workspace_independent_of_n_t(b):
    sizes = {b.bgpo_workspace_size(_prob(b, n_t=n)) for n in (1, 4, 16, 64, 1000)}
    assert len(sizes) == 1
    assert b.bgpo_workspace_size(_prob(b, B=16)) > b.bgpo_workspace_size(_prob(b))


@pytest.mark.parametrize("kw,status", [
    (dict(d=4000), -4), (dict(V=126000), -4), (dict(d=32), -4), (dict(B=5000, L=1), -4),
    (dict(B=2048, L=1024), -4), (dict(B=0), -1), (dict(L=0), -1), (dict(n_t=0), -1),
    (dict(j_begin=-1), -1), (dict(j_begin=60, j_count=5), -1), (dict(t_mode=2), -1),
    (dict(bound=4), -1), (dict(sample_stride=-8), -1), (dict(sample_stride=12), -1),
    (dict(norm_eps=float("nan")), -1), (dict(norm_eps=-1.0), -1),
    (dict(in_dtype=2), -1), (dict(in_dtype=-1), -1), (dict(vocab_chunk=100), -1),
    (dict(vocab_chunk=-256), -1), (dict(ws_budget=1 << 20), -5),
    (dict(bound=3, retain_samples=1, vocab_chunk=256), -1),
    (dict(bound=3, retain_samples=1, ws_budget=1 << 40), -1),
])
def test_problem_validation(b, kw, status):
    with pytest.raises(b.BgpoError) as e:
        b.bgpo_workspace_size(_prob(b, **kw))
    assert e.value.status == status


def test_null_pointers_and_workspace_rejected_before_hip(b):
    p = _prob(b, B=2, L=64, d=128, V=1024, n_t=4).c()
    lib = b._lib
    fake = ctypes.c_void_p(0x1000)        # never dereferenced: validation fails first
    nbytes = ctypes.c_size_t(0)
    assert lib.bgpo_workspace_size(ctypes.byref(p), ctypes.byref(nbytes)) == 0
    # missing hidden
    assert lib.bgpo_elbo_fwd(ctypes.byref(p), None, fake, fake, fake, fake, fake, None,
                             fake, nbytes.value, None, None) == -1
    # workspace too small / misaligned / missing
    ws_small = ctypes.c_void_p(0x100000)
    assert lib.bgpo_elbo_fwd(ctypes.byref(p), fake, fake, fake, fake, fake, fake, None,
                             ws_small, nbytes.value - 1, None, None) == -2
    assert lib.bgpo_elbo_fwd(ctypes.byref(p), fake, fake, fake, fake, fake, fake, None,
                             ctypes.c_void_p(0x100010), nbytes.value, None, None) == -2
    assert lib.bgpo_elbo_fwd(ctypes.byref(p), fake, fake, fake, fake, fake, fake, None,
                             None, nbytes.value, None, None) == -2
    # backward: missing dW, non-finite loss scale
    assert lib.bgpo_elbo_bwd_accumulate(ctypes.byref(p), fake, fake, fake, fake, fake, None, 0.125,
                                        fake, None, fake, fake, fake, fake, None, None,
                                        ws_small, nbytes.value, None, None) == -1
    assert lib.bgpo_elbo_bwd_accumulate(ctypes.byref(p), fake, fake, fake, fake, fake, None,
                                        float("nan"), fake, fake, fake, fake, fake, fake, None,
                                        None, ws_small, nbytes.value, None, None) == -1
    # sample masks: j out of range
    assert lib.bgpo_sample_masks(ctypes.byref(p), fake, 4, fake, fake, None, None) == -1
    assert lib.bgpo_sample_masks(ctypes.byref(p), fake, -1, fake, fake, None, None) == -1
    # objective mode outside BGPO_BOUND_*
    for bad in (-1, 4):
        q = _prob(b, B=2, L=64, d=128, V=1024, n_t=4).c()
        q.bound = bad
        assert lib.bgpo_workspace_size(ctypes.byref(q), ctypes.byref(nbytes)) == -1
    # the exact objective couples all samples: a partial range is refused
    # before anything is enqueued
    q = _prob(b, B=2, L=64, d=128, V=1024, n_t=4, j_begin=1, j_count=2).c()
    q.bound = b.BGPO_BOUND_EXACT
    assert lib.bgpo_elbo_bwd_accumulate(ctypes.byref(q), fake, fake, fake, fake, fake, None, 0.125,
                                        fake, fake, fake, fake, fake, fake, None, None,
                                        ws_small, nbytes.value, None, None) == -1


def test_gemm_hooks_check_shapes_before_hip(b):
    """The GEMM-core test hooks refuse shapes their layouts cannot hold before
    any device call (the pointers are never dereferenced)."""
    lib = b._lib
    fake = ctypes.c_void_p(0x1000)
    for M, N, K in ((64, 64, 0), (64, 64, 96), (0, 64, 64), (64, 0, 64)):
        assert lib.bgpo_test_gemm_nt(fake, fake, fake, M, N, K, None) == -1
        assert lib.bgpo_test_gemm_tn(fake, fake, fake, M, N, K, None) == -1
    # the dW GEMM's A layout holds whole 64-wide slabs of M
    assert lib.bgpo_test_gemm_tn(fake, fake, fake, 96, 64, 64, None) == -1
    assert lib.bgpo_test_gemm_tn(None, fake, fake, 64, 64, 64, None) == -1
    assert lib.bgpo_test_gemm_split(fake, fake, fake, 64, 64, 64, 0, None) == -1


def test_problem_struct_layout(b):
    # matches the C struct: 8 int32, uint64, uint32, int32, int64, float, 3 int32, uint64
    assert ctypes.sizeof(b._Problem) == 80
    assert b._Problem.seed.offset == 32
    assert b._Problem.bound.offset == 44
    assert b._Problem.sample_stride.offset == 48
    assert b._Problem.norm_eps.offset == 56
    assert b._Problem.retain_samples.offset == 60
    assert b._Problem.in_dtype.offset == 64
    assert b._Problem.vocab_chunk.offset == 68
    assert b._Problem.ws_budget.offset == 72
    src = open(os.path.join(ROOT, "include", "bgpo.h")).read()
    src = src[src.index("typedef struct bgpo_problem {"):src.index("} bgpo_problem;")]
    fields = re.findall(r"^\s+(?:int32_t|uint64_t|uint32_t|int64_t|float)\s+(\w+);", src, flags=re.M)
    assert [f for f in fields if f in dict(b._Problem._fields_)] == [n for n, _ in b._Problem._fields_]


def test_retained_workspace_grows_linearly_with_n_t(b):
    """Retained mode keeps the state of every unit of samples (8 samples per
    unit at this shape, fewer when n_t is smaller): memory grows with n_t,
    by the same amount per added unit."""
    size = {n: b.bgpo_workspace_size(_prob(b, n_t=n, bound=3, retain_samples=1))
            for n in (1, 2, 4, 8, 16, 24, 64)}
    assert size[1] < size[2] < size[4] < size[8]
    per_unit = size[16] - size[8]
    assert per_unit > 8 * 10 ** 9                  # dZ rows, H_c^T columns + state of 8 samples
    assert size[24] - size[16] == per_unit
    assert size[64] - size[16] == 6 * per_unit
    assert b.bgpo_workspace_size(_prob(b, n_t=64, bound=3)) < size[16]   # constant mode, any n_t


def test_every_entry_point_lays_out_what_it_checked(b):
    """One byte short of bgpo_workspace_size() is refused, for the retained
    and the constant layouts alike; the entry points then use the layout they
    checked (workspace_layout with the problem's retain flag, or the fixed
    layout of a branch taken only for that flag), so an accepted workspace is
    never overrun."""
    lib = b._lib
    fake = ctypes.c_void_p(0x1000)
    for retain in (0, 1):
        pr = _prob(b, B=2, L=64, d=128, V=1024, n_t=4, bound=3, retain_samples=retain, j_begin=1,
                   j_count=2).c()
        n = ctypes.c_size_t(0)
        assert lib.bgpo_workspace_size(ctypes.byref(pr), ctypes.byref(n)) == 0
        ws = ctypes.c_void_p(0x100000)
        # one byte short: refused before anything is enqueued
        assert lib.bgpo_elbo_fwd(ctypes.byref(pr), fake, fake, fake, fake, fake, fake, None, ws,
                                 n.value - 1, None, None) == -2
    src = open(os.path.join(ROOT, "paper_2510_11683_amd", "csrc", "api.hip")).read()
    # every layout call lays out a plan (the one plan_problem chose for the
    # problem, which check_workspace measured), never a layout of its own
    calls = re.findall(r"workspace_layout\(([^;]*)\);", src)
    assert calls and all(re.search(r"(^|, )\*?pl, ", c) for c in calls), calls
    assert src.count("plan_problem(prob, &pl)") >= 4


def test_reserved_field_and_rmsnorm_arguments_rejected_before_hip(b):
    lib = b._lib
    fake = ctypes.c_void_p(0x1000)
    nbytes = ctypes.c_size_t(0)
    for bound, retain in ((0, 1), (3, 2), (3, -1)):        # retain needs the exact bound, 0 or 1
        q = _prob(b, B=2, L=64, d=128, V=1024, n_t=4).c()
        q.bound, q.retain_samples = bound, retain
        assert lib.bgpo_workspace_size(ctypes.byref(q), ctypes.byref(nbytes)) == -1
    p = _prob(b, B=2, L=64, d=128, V=1024, n_t=4).c()
    assert lib.bgpo_workspace_size(ctypes.byref(p), ctypes.byref(nbytes)) == 0
    ws = ctypes.c_void_p(0x100000)
    # missing norm weight / its gradient
    assert lib.bgpo_elbo_fwd_rmsnorm(ctypes.byref(p), fake, None, fake, fake, fake, fake, fake,
                                     None, ws, nbytes.value, None, None) == -1
    assert lib.bgpo_elbo_bwd_accumulate_rmsnorm(ctypes.byref(p), fake, fake, fake, fake, fake,
                                                fake, None, 0.125, fake, None, fake, fake, fake,
                                                fake, fake, None, None, ws, nbytes.value, None,
                                                None) == -1
    # misaligned norm weight
    assert lib.bgpo_elbo_fwd_rmsnorm(ctypes.byref(p), fake, ctypes.c_void_p(0x1004), fake, fake,
                                     fake, fake, fake, None, ws, nbytes.value, None, None) == -1


def test_retained_rows_bounded_by_the_column_range(b):
    """H_c^T holds one column and the kept dZ one row per kept row (32-bit
    offsets in the sample records): with every sample retained, the kept rows (whole
    units of samples, B*L rounded up to 256 per sample) must stay at or below
    2^30.  At B*L = 2^20 a unit holds 3 samples: n_t = 1023 keeps 341 units
    (1023 * 2^20 rows), n_t = 1024 one unit more; the constant mode takes any
    n_t."""
    big = dict(B=4096, L=256, d=64, V=128, bound=3)
    assert b.bgpo_workspace_size(_prob(b, n_t=1023, retain_samples=1, **big)) > 0
    for n_t in (1024, 4096):
        with pytest.raises(b.BgpoError) as e:
            b.bgpo_workspace_size(_prob(b, n_t=n_t, retain_samples=1, **big))
        assert e.value.status == -4
    assert b.bgpo_workspace_size(_prob(b, n_t=1000, **big)) == b.bgpo_workspace_size(_prob(b, n_t=1, **big))


GiB = 1 << 30


def test_budget_picks_layouts_that_fit(b):
    """A workspace budget selects the largest stored-exponential layout that
    fits, and below that the recompute layout; the chosen size never exceeds
    the budget and never depends on n_t; a budget below the smallest layout is
    refused with BGPO_ERR_BUDGET."""
    full = b.bgpo_workspace_size(_prob(b))
    assert full > 20 * GiB                                  # default: stored, units of 8
    sizes = {}
    for budget in (2, 3, 4, 6, 8, 16, 24, 32, 64):
        sz = b.bgpo_workspace_size(_prob(b, ws_budget=budget * GiB))
        assert sz <= budget * GiB
        assert {b.bgpo_workspace_size(_prob(b, n_t=n, ws_budget=budget * GiB)) for n in (1, 4, 16, 64)} == {sz}
        sizes[budget] = sz
    assert sizes[64] == full or sizes[64] <= 64 * GiB
    # monotone: a larger budget never gives a smaller layout here
    vals = [sizes[k] for k in sorted(sizes)]
    assert vals == sorted(vals)
    # the smallest layouts hold the transposed head (2 d V bytes) and little else
    dV2 = 2 * 4096 * 126464
    assert dV2 < sizes[2] <= 2 * GiB
    with pytest.raises(b.BgpoError) as e:
        b.bgpo_workspace_size(_prob(b, ws_budget=dV2))
    assert e.value.status == b.BGPO_ERR_BUDGET


def test_budget_above_the_default_raises_the_dw_batch(b):
    """A budget the default layout fits in keeps its units and raises its dW
    batch (fewer read-modify-writes of dW) as far as the budget allows, up to
    four units; without a budget the default batch of two stays."""
    dflt = b.bgpo_workspace_plan(_prob(b))
    assert dflt["dw_batch"] == 2
    seen = []
    for budget in (24, 32, 40, 48, 64):
        plan = b.bgpo_workspace_plan(_prob(b, ws_budget=budget * GiB))
        assert plan["workspace_bytes"] <= budget * GiB
        assert plan["samples_per_unit"] == dflt["samples_per_unit"] and plan["mode"] == "stored"
        seen.append(plan["dw_batch"])
    assert seen == sorted(seen) and seen[0] == 2 and seen[-1] == 4


def test_w_copy_kept_where_it_pays(b):
    """The default layout keeps the slab-major copy of W (2 d V bytes, the dX
    GEMM's operand); a tight budget drops it for bf16 inputs when that buys
    a larger unit (4 GiB at the benchmark shape: units of 2 without it, of 1
    with it), while fp32 inputs, which need a bf16 W anyway, keep it; the
    recompute layouts keep it for fp32 inputs only."""
    assert b.bgpo_workspace_plan(_prob(b))["w_copy"] == 1
    tight = b.bgpo_workspace_plan(_prob(b, ws_budget=4 * GiB))
    assert (tight["mode"], tight["w_copy"], tight["samples_per_unit"]) == ("stored", 0, 2)
    tight32 = b.bgpo_workspace_plan(_prob(b, ws_budget=4 * GiB, in_dtype=b.BGPO_F32))
    assert tight32["w_copy"] == 1 and tight32["samples_per_unit"] == 1
    for dt, wc in ((b.BGPO_BF16, 0), (b.BGPO_F32, 1)):
        assert b.bgpo_workspace_plan(_prob(b, vocab_chunk=4096, in_dtype=dt))["w_copy"] == wc
    assert b.bgpo_workspace_plan(_prob(b, retain_samples=1, bound=3))["w_copy"] == 1


def test_forced_vocab_chunk_and_fp32_copy(b):
    """vocab_chunk > 0 forces the recompute layout (much smaller than the
    stored one at the same unit size).  The stored layout always holds a
    slab-major bf16 copy of W (the dX GEMM's operand), so fp32 inputs cost
    nothing more there; the recompute layout reads a bf16 W in place and
    adds the copy (2 d V bytes) only for fp32 inputs."""
    stored = b.bgpo_workspace_size(_prob(b))
    chunked = b.bgpo_workspace_size(_prob(b, vocab_chunk=8192))
    assert chunked < stored / 4
    small = dict(B=2, L=64, d=128, V=1024, n_t=4)
    w16 = b.bgpo_workspace_size(_prob(b, **small))
    w32 = b.bgpo_workspace_size(_prob(b, in_dtype=b.BGPO_F32, **small))
    assert w32 == w16
    r16 = b.bgpo_workspace_size(_prob(b, vocab_chunk=256, **small))
    r32 = b.bgpo_workspace_size(_prob(b, vocab_chunk=256, in_dtype=b.BGPO_F32, **small))
    assert r32 - r16 >= 2 * 128 * 1024
    assert w16 - r16 >= 2 * 128 * 1024
    # a chunk wider than the vocabulary is the whole vocabulary
    assert (b.bgpo_workspace_size(_prob(b, vocab_chunk=4096, **small)) ==
            b.bgpo_workspace_size(_prob(b, vocab_chunk=1024, **small)))


def test_ell_old_aliasing_rejected_before_hip(b):
    """l is written before l_old is read, so ell_old overlapping ell or g is
    refused (BGPO_ERR_INVALID_ARG) before anything is enqueued; disjoint
    buffers pass that check (and here fail the workspace check instead)."""
    p = _prob(b, B=2, L=64, d=128, V=1024, n_t=4).c()
    lib = b._lib
    n = ctypes.c_size_t(0)
    assert lib.bgpo_workspace_size(ctypes.byref(p), ctypes.byref(n)) == 0
    fake = ctypes.c_void_p(0x1000)
    ws = ctypes.c_void_p(0x100000)
    ell, g = 0x200000, 0x300000
    nbytes = 2 * 4 * 8

    def call(ell_old):
        return lib.bgpo_elbo_bwd_accumulate(ctypes.byref(p), fake, fake, fake, fake, fake,
                                            ctypes.c_void_p(ell_old), 0.125, fake, fake,
                                            ctypes.c_void_p(ell), ctypes.c_void_p(g), fake, fake,
                                            None, None, ws, n.value - 1, None, None)
    for eo in (ell, ell + 8, ell - nbytes + 8, g, g + nbytes - 8):
        assert call(eo) == -1, hex(eo)
    for eo in (ell + nbytes, ell - nbytes, 0x400000):
        assert call(eo) == -2, hex(eo)


def test_noalloc_refuses_problems_beyond_its_scratch_before_hip(b):
    """The allocation-free backward plans the problem within its static
    scratch (128 MiB): a problem whose smallest layout is larger (the LLaDA
    head: W^T alone is 1 GB) is refused with BGPO_ERR_BUDGET, a retained-state
    problem with BGPO_ERR_INVALID_ARG, before any HIP call."""
    lib = b._lib
    assert b.bgpo_noalloc_scratch_bytes() == 128 << 20
    fake = ctypes.c_void_p(0x1000)

    def call(p):
        return lib.bgpo_elbo_bwd_accumulate_noalloc(ctypes.byref(p.c()), *([fake] * 6), 0.125,
                                                    *([fake] * 8), None)
    assert call(_prob(b)) == b.BGPO_ERR_BUDGET
    assert call(_prob(b, bound=3, retain_samples=1, B=2, L=64, d=128, V=1024, n_t=4)) == -1
    assert call(_prob(b, B=0)) == -1
    # a small problem fits the scratch: its plan under that budget exists
    small = _prob(b, B=4, L=200, d=576, V=4288, n_t=3, ws_budget=128 << 20)
    assert b.bgpo_workspace_plan(small)["workspace_bytes"] <= 128 << 20
