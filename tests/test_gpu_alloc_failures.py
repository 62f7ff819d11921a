"""Device allocation failures, injected through the test hook of
include/nmt_debug.h at every position of every call that allocates: the call
must report NMT_ENOMEM, leave none of its allocations behind, and leave the
library usable (the same call then succeeds)."""
import numpy as np
import pytest

from paper_1605_04809_amd.workloads import CONFIGS, make_workload

pytestmark = pytest.mark.gpu


def _torch():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _fail_everywhere(nb, call, cleanup, limit=200):
    """Run call() with allocation n failing, for n = 0, 1, ... until it
    succeeds; every failing run must give NMT_ENOMEM and leak nothing."""
    base = nb.debug_alloc_hook(-1)
    for n in range(limit):
        nb.debug_alloc_hook(n)
        try:
            out = call()
        except nb.NmtError as e:
            live = nb.debug_alloc_hook(-1)
            assert e.status == nb.NMT_ENOMEM, (n, str(e))
            assert live == base, f"allocation {n} failing left {live - base} allocations behind"
            continue
        nb.debug_alloc_hook(-1)
        cleanup(out)
        assert nb.debug_alloc_hook(-1) == base
        return n
    raise AssertionError("the call never succeeded")


def test_every_allocating_call_reports_enomem_and_leaks_nothing():
    torch = _torch()
    from paper_1605_04809_amd import binding as nb
    wl = make_workload(CONFIGS["tiny"].replace(seed=71))
    c = wl.cfg
    cu = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    try:
        n_model = _fail_everywhere(nb, lambda: nb.Model.from_workload(wl), lambda m: m.close())
        model = nb.Model.from_workload(wl)
        n_enc = _fail_everywhere(nb, lambda: nb.nmt_encode(model, cu(wl.src_ids), wl.src_len), lambda s: s.close())
        ctx = torch.randn((c.S, c.Tpad, c.C), device="cuda")
        n_ann = _fail_everywhere(nb, lambda: nb.nmt_source_from_annotations(model, ctx, wl.src_len),
                                 lambda s: s.close())
        n_avg = _fail_everywhere(nb, lambda: nb.nmt_model_average([model, model]), lambda m: m.close())
        s0 = torch.empty((c.S, c.H), device="cuda")
        src = nb.nmt_encode(model, cu(wl.src_ids), wl.src_len, s0)
        n_res = _fail_everywhere(nb, lambda: nb.Rescorer([model], [src], [s0], 64), lambda r: r.close())

        def stack():
            r = nb.Rescorer([model], [src], [s0], 64)
            try:
                r.rescore([0, 0, 0], [[1, 2], [1], []])
            finally:
                r.close()
            return None
        n_stack = _fail_everywhere(nb, stack, lambda _: None)
        # the library is still usable: a normal step
        logp = torch.empty(c.B, device="cuda")
        nb.nmt_score_batch(model, src, cu(wl.s_prev), cu(wl.y_prev), cu(wl.sent_id), cu(wl.req), logp,
                           torch.empty((c.B, c.H), device="cuda"))
        torch.cuda.synchronize()
        assert bool(torch.isfinite(logp).all())
        print(f"allocations before success: model {n_model}, encode {n_enc}, annotations {n_ann}, "
              f"average {n_avg}, rescorer {n_res}, rescore stack {n_stack}", flush=True)
        assert min(n_model, n_enc, n_ann, n_avg, n_res, n_stack) >= 1
        src.close()
        model.close()
    finally:
        nb.debug_alloc_hook(-1)
