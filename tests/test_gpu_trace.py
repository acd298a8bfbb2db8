"""Block trace of the sweep (BGMF_OPT_TRACE, bgmf_get_trace) on the GPU: in
every schedule and V placement, streamed or in-core, no block starts
before its row-block's previous block or its column-block's previous
holder handed its results on (nor, with one launch per stratum, before the
previous stratum ended), every block is traced, and tracing leaves the
results bit-identical."""
import numpy as np
import pytest

from workloads import make_config

pytestmark = pytest.mark.gpu

CASES = {
    # name: options (v_staging, schedule, lds_handover, passes, streamed)
    "lds_persistent": dict(),
    "lds_persistent_global_handover": dict(lds_handover=0),
    "lds_per_stratum": dict(schedule=1),
    "global_v_per_stratum": dict(v_staging=2, schedule=1),
    "global_v_persistent": dict(v_staging=2, schedule=2),
    "two_passes": dict(passes=2),
    "streamed": dict(streamed=True),
}


def _run(w, trace, v_staging=0, schedule=0, lds_handover=1, passes=1, streamed=False):
    from paper_2304_13724_amd import bgmf
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        mdl.set_option(bgmf.BGMF_OPT_V_STAGING, v_staging)
        mdl.set_option(bgmf.BGMF_OPT_SCHEDULE, schedule)
        mdl.set_option(bgmf.BGMF_OPT_LDS_HANDOVER, lds_handover)
        mdl.set_option(bgmf.BGMF_OPT_BLOCK_PASSES, passes)
        if streamed:
            mdl.set_option(bgmf.BGMF_OPT_RATINGS_BUDGET, w.nnz * 8 // 3)
        mdl.set_option(bgmf.BGMF_OPT_TRACE, 1 if trace else 0)
        mdl.set_factors(w.U0, w.V0)
        mdl.load_coo(w.rows, w.cols, w.vals)
        mdl.epoch(w.alpha, w.beta)
        tr = mdl.get_trace() if trace else None
        placement = mdl.get_option(bgmf.BGMF_OPT_PLACEMENT)
        mdl.epoch(w.alpha, w.beta)
        U, V = mdl.get_factors()
    return tr, placement, U, V


@pytest.mark.parametrize("case", sorted(CASES))
def test_trace_order_and_bit_identity(case):
    from paper_2304_13724_amd import trace as T
    w = make_config("medium", n=7_000, m=1_000, nnz=300_000, p=32)
    opts = CASES[case]
    print(f"trace case {case}: {opts}", flush=True)
    (begin, end, tps), placement, U, V = _run(w, True, **opts)
    _, _, U0, V0 = _run(w, False, **opts)
    assert np.array_equal(U, U0) and np.array_equal(V, V0)
    assert 1e6 <= tps <= 1e10
    if not opts.get("streamed"):
        assert np.all(begin > 0) and np.all(end >= begin)
    per_stratum = not (placement & 4)
    bad = T.violations(begin, end, per_stratum=per_stratum)
    assert bad == [], bad[:10]
    out = T.summary(begin, end, tps)
    print(f"{case}: placement {placement}, {out}", flush=True)
    assert out["span_us"] > 0


def test_trace_state_errors():
    from paper_2304_13724_amd import bgmf
    w = make_config("tiny")
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        mdl.set_factors(w.U0, w.V0)
        mdl.load_coo(w.rows, w.cols, w.vals)
        assert mdl.get_option(bgmf.BGMF_OPT_TRACE) == 0
        mdl.epoch(w.alpha, w.beta)
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.get_trace()  # not traced
        assert ei.value.code == bgmf.BGMF_E_STATE
        mdl.set_option(bgmf.BGMF_OPT_TRACE, 1)
        assert mdl.get_option(bgmf.BGMF_OPT_TRACE) == 1
        with pytest.raises(bgmf.BgmfError):
            mdl.get_trace()  # no epoch since the option was set
        mdl.epoch(w.alpha, w.beta)
        begin, end, _ = mdl.get_trace()
        assert begin.shape == (w.p, w.p) and np.all(end >= begin) and np.all(begin > 0)
        mdl.set_option(bgmf.BGMF_OPT_TRACE, 0)
        with pytest.raises(bgmf.BgmfError):
            mdl.get_trace()
        with pytest.raises(bgmf.BgmfError):
            mdl.set_option(bgmf.BGMF_OPT_TRACE, 2)
