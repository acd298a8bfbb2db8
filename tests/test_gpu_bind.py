"""Caller-owned memory (bgmf_query_sizes, bgmf_bind): U, V, the device
workspace and the pinned host arena are PyTorch tensors, and the stream is
PyTorch's.  A bound handle must give bit-identical results to a handle that
owns its memory -- in-core and streamed -- and must allocate nothing in
bgmf_load_coo, bgmf_epoch or bgmf_rmse.

Also the bounds of the streamed load: a budgeted load that buckets the
ratings group by group (many groups, many input batches) is bit-exact
against the oracle's bucketing, and its device memory for ratings peaks
within the budget (or within the bytes needed to bucket the largest block).
"""
import numpy as np
import pytest

import oracle
from workloads import make, make_config

pytestmark = pytest.mark.gpu


def _owned(w, epochs, budget=0):
    from paper_2304_13724_amd import bgmf
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        mdl.set_option(bgmf.BGMF_OPT_RATINGS_BUDGET, budget)
        mdl.set_factors(w.U0, w.V0)
        mdl.load_coo(w.rows, w.cols, w.vals)
        bp, perm = mdl.get_layout()
        hist = []
        for _ in range(epochs):
            mdl.epoch(w.alpha, w.beta)
            hist.append(mdl.rmse())
        U, V = mdl.get_factors()
        info = dict(slots=mdl.get_option(bgmf.BGMF_OPT_STREAM_SLOTS),
                    peak=mdl.get_option(bgmf.BGMF_OPT_LOAD_PEAK))
    return U, V, hist, bp, perm, info


def _bound(w, epochs, ws_bytes=None, pinned=True, budget=0):
    """The same run with every buffer a torch tensor on cuda:0 and torch's
    current stream; returns the results and the allocation counts."""
    import torch
    from paper_2304_13724_amd import bgmf
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        sizes = mdl.query_sizes(w.nnz)
        assert sizes["factor_bytes"] == (w.n + w.m) * w.k * 4
        assert sizes["min_ws_bytes"] <= sizes["incore_ws_bytes"]
        ws_bytes = sizes["incore_ws_bytes"] if ws_bytes is None else ws_bytes
        U_t = torch.from_numpy(w.U0).to("cuda:0")
        V_t = torch.from_numpy(w.V0).to("cuda:0")
        ws_t = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda:0")
        pin_t = (torch.empty(sizes["pinned_bytes"], dtype=torch.uint8, pin_memory=True)
                 if pinned else None)
        torch.cuda.synchronize()
        mdl.set_option(bgmf.BGMF_OPT_RATINGS_BUDGET, budget)
        mdl.bind_tensors(U_t, V_t, ws_t, pin_t, stream.cuda_stream)
        before = mdl.get_option(bgmf.BGMF_OPT_ALLOC_COUNT)
        mdl.load_coo(w.rows, w.cols, w.vals)
        hist = []
        for _ in range(epochs):
            mdl.epoch(w.alpha, w.beta)
            hist.append(mdl.rmse())
        after = mdl.get_option(bgmf.BGMF_OPT_ALLOC_COUNT)
        bp, perm = mdl.get_layout()
        slots = mdl.get_option(bgmf.BGMF_OPT_STREAM_SLOTS)
        # the factors live in the caller's tensors
        U = U_t.cpu().numpy()
        V = V_t.cpu().numpy()
        U2, V2 = mdl.get_factors()
        assert np.array_equal(U, U2) and np.array_equal(V, V2)
        assert bgmf.bgmf_factor_ptrs(mdl.h) == (U_t.data_ptr(), V_t.data_ptr())
    del ws_t, pin_t
    return U, V, hist, bp, perm, dict(allocs=after - before, slots=slots)


CASES = {
    "tiny": lambda: make_config("tiny"),
    "large_shape": lambda: make_config("large", n=48_000, m=1_800, nnz=1_000_000, p=128),
    "k128_ragged": lambda: make("b", n=3_001, m=1_999, nnz=150_000, k=128, p=7, alpha=0.01,
                                beta=0.05, epochs=1, seed=41, structure="uniform",
                                values="int5", rank=4),
}


def _same(a, b, streamed=False):
    assert np.array_equal(a[3], b[3]) and np.array_equal(a[4], b[4])  # layout
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])  # U, V
    if not streamed:
        assert a[2] == b[2]  # RMSE history
    else:
        # the streamed RMSE pass adds the same squares in another fixed order
        for x, y in zip(a[2], b[2]):
            assert abs(x - y) <= 1e-12 * y


@pytest.mark.parametrize("case", sorted(CASES))
def test_bound_incore_bit_identical(case):
    w = CASES[case]()
    own = _owned(w, 2)
    bnd = _bound(w, 2)
    assert bnd[5]["slots"] == 0 and bnd[5]["allocs"] == 0
    _same(bnd, own)


@pytest.mark.parametrize("case", ["large_shape", "k128_ragged"])
def test_bound_streamed_bit_identical(case):
    """A workspace of the tables plus a third of the records: the ratings
    stream from the bound pinned arena, bucketed group by group inside the
    workspace; results equal the in-core library-owned run."""
    from paper_2304_13724_amd import bgmf
    w = CASES[case]()
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        sizes = mdl.query_sizes(w.nnz)
    tables = (w.p * w.p + 1) * 8 + w.p * w.p + 512
    ws = max(tables + w.nnz * 8 // 3, sizes["min_ws_bytes"])
    assert ws < sizes["incore_ws_bytes"]
    own = _owned(w, 2)
    bnd = _bound(w, 2, ws_bytes=ws)
    assert bnd[5]["slots"] in (2, 3) and bnd[5]["allocs"] == 0
    _same(bnd, own, streamed=True)


def test_bound_errors():
    import torch
    from paper_2304_13724_amd import bgmf
    w = CASES["tiny"]()
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        sizes = mdl.query_sizes(w.nnz)
        U_t = torch.from_numpy(w.U0).to("cuda:0")
        V_t = torch.from_numpy(w.V0).to("cuda:0")
        ws_t = torch.empty(sizes["incore_ws_bytes"] + 256, dtype=torch.uint8, device="cuda:0")
        torch.cuda.synchronize()
        # misaligned workspace
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.bind(U_t.data_ptr(), V_t.data_ptr(), ws_t.data_ptr() + 16,
                     sizes["incore_ws_bytes"], 0, 0, None)
        assert ei.value.code == bgmf.BGMF_E_ARG and "256-byte" in str(ei.value)
        # pageable host memory (256-byte aligned) where device memory is needed
        host = np.zeros(w.U0.size + 64, dtype=np.float32)
        off = (-host.ctypes.data % 256) // 4
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.bind(host[off:].ctypes.data, V_t.data_ptr(), ws_t.data_ptr(),
                     sizes["incore_ws_bytes"], 0, 0, None)
        assert ei.value.code == bgmf.BGMF_E_ARG and "device memory" in str(ei.value)
        # a workspace below the block tables
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.bind(U_t.data_ptr(), V_t.data_ptr(), ws_t.data_ptr(), 64, 0, 0, None)
        assert ei.value.code == bgmf.BGMF_E_BUDGET
        # too small to hold the ratings, and no pinned arena to stream them
        mdl.bind(U_t.data_ptr(), V_t.data_ptr(), ws_t.data_ptr(), sizes["min_ws_bytes"], 0, 0,
                 None)
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.load_coo(w.rows, w.cols, w.vals)
        assert ei.value.code == bgmf.BGMF_E_BUDGET
        # a workable binding, then binding again once ratings are loaded
        mdl.bind(U_t.data_ptr(), V_t.data_ptr(), ws_t.data_ptr(), sizes["incore_ws_bytes"], 0,
                 0, None)
        mdl.load_coo(w.rows, w.cols, w.vals)
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.bind(U_t.data_ptr(), V_t.data_ptr(), ws_t.data_ptr(), sizes["incore_ws_bytes"],
                     0, 0, None)
        assert ei.value.code == bgmf.BGMF_E_STATE
        mdl.epoch(w.alpha, w.beta)
        assert np.isfinite(mdl.rmse())


@pytest.mark.parametrize("budget_kib", [256, 1024, 8192])
def test_streamed_load_groups_bit_exact_and_within_budget(budget_kib):
    """1e6 ratings (8 MB of records) under budgets of 0.25 to 8 MiB: the
    bucketing runs in many groups and input batches (down to 4096
    ratings); block_ptr and perm equal the oracle's, two epochs equal the
    in-core run bit for bit, and the load's device memory for ratings peaks
    within the budget, or, when the budget is below it, within the bytes
    needed to bucket the largest block with the smallest batch.  A budget
    below two strata is refused with BGMF_E_BUDGET."""
    w = make_config("large", n=48_000, m=1_800, nnz=1_000_000, p=64)
    budget = budget_kib * 1024
    bp_ref, perm_ref = oracle.bucket(w.n, w.m, w.p, w.rows, w.cols)
    widest = int(np.diff(bp_ref[:: w.p]).max())
    if 2 * (widest + 256) * 8 > budget:
        # the ring needs two strata on the device: below that, a clear error
        from paper_2304_13724_amd import bgmf
        with pytest.raises(bgmf.BgmfError) as ei:
            _owned(w, 1, budget=budget)
        assert ei.value.code == bgmf.BGMF_E_BUDGET and "two strata" in str(ei.value)
        return
    inc = _owned(w, 2)
    ooc = _owned(w, 2, budget=budget)
    assert ooc[5]["slots"] in (2, 3)
    assert np.array_equal(ooc[3], bp_ref) and np.array_equal(ooc[4], perm_ref)
    assert np.array_equal(ooc[0], inc[0]) and np.array_equal(ooc[1], inc[1])
    for x, y in zip(ooc[2], inc[2]):
        assert abs(x - y) <= 1e-12 * y
    biggest = int(np.diff(bp_ref).max())
    slots = w.p * w.p
    # bucketing one block costs some 52 bytes per rating (its COO arrays and
    # input positions, the radix sort's key and value buffers, the sorted
    # records and perm), plus tables of the p^2 slots and one input batch
    floor = 64 * biggest + 48 * (slots + 1) + (1 << 20)
    print(f"budget {budget}, load peak {ooc[5]['peak']}, floor {floor}", flush=True)
    assert 0 < ooc[5]["peak"] <= max(budget, floor)
