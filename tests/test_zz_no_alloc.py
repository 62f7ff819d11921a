"""The allocation-free step (nmt_score_batch_noalloc) against nmt_score_batch.

Both run the same kernels in the same launch shapes; only where the step's
scratch lives differs (the library's per-device array instead of a caller
workspace), so the outputs must be identical.  Two calls in a row, the second
with fewer rows, show that what the first call leaves in the shared array
does not leak into the next; a batch too large for the array is refused on
the host with nothing enqueued.
"""
import numpy as np
import pytest

from paper_1605_04809_amd.workloads import CONFIGS, make_workload

pytestmark = pytest.mark.gpu


def _torch():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


@pytest.mark.parametrize("wtype,B1,B2", [("f32", 2000, 333), ("bf16", 2000, 701)])
def test_noalloc_matches_workspace_step(wtype, B1, B2):
    torch = _torch()
    from paper_1605_04809_amd import binding as nb
    wl = make_workload(CONFIGS["enru_b2000"].replace(wtype=wtype, seed=61))
    c = wl.cfg
    model = nb.Model.from_workload(wl)
    cu = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    src = nb.nmt_encode(model, cu(wl.src_ids), wl.src_len)
    assert nb.nmt_score_workspace_bytes(model, B1) <= nb.NOALLOC_SCRATCH_BYTES
    rng = np.random.default_rng(62)
    for B in (B1, B2):
        rows = np.sort(rng.choice(c.B, size=B, replace=False))
        sp, y, s, r = (cu(a[rows]) for a in (wl.s_prev, wl.y_prev, wl.sent_id, wl.req))
        want = dict(logp=torch.empty(B, device="cuda"), logZ=torch.empty(B, device="cuda"),
                    s_new=torch.empty((B, c.H), device="cuda"))
        got = {k: torch.full_like(v, float("nan")) for k, v in want.items()}
        nb.nmt_score_batch(model, src, sp, y, s, r, want["logp"], want["s_new"], want["logZ"])
        nb.nmt_score_batch_noalloc(model, src, sp, y, s, r, got["logp"], got["s_new"], got["logZ"])
        torch.cuda.synchronize()
        assert nb.nmt_stream_status(model) == nb.NMT_OK
        for k in want:
            np.testing.assert_array_equal(got[k].cpu().numpy(), want[k].cpu().numpy(), err_msg=f"B={B} {k}")
        print(f"{wtype} B={B}: noalloc == workspace step on every output", flush=True)
    # a batch whose scratch exceeds the array is refused before anything runs
    B = 4096
    assert nb.nmt_score_workspace_bytes(model, B) > nb.NOALLOC_SCRATCH_BYTES
    z = torch.zeros(B, dtype=torch.int32, device="cuda")
    st = torch.zeros((B, c.H), device="cuda")
    logp = torch.full((B,), 7.0, device="cuda")
    with pytest.raises(nb.NmtError) as ei:
        nb.nmt_score_batch_noalloc(model, src, st, z, z, z, logp, st)
    assert ei.value.status == nb.NMT_EWORKSPACE and "scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert torch.all(logp == 7.0)
    src.close()
    model.close()
