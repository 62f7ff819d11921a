"""The batched step captured in a HIP graph (torch.cuda.CUDAGraph around
the library's launches on the capture stream) and replayed: the step makes
no allocation and records no memset, so every replay must reproduce the
eagerly launched step bit for bit, also with other eager work and
synchronisations between the replays."""
import numpy as np
import pytest

from paper_1605_04809_amd.workloads import CONFIGS, make_workload

pytestmark = pytest.mark.gpu


def _torch():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


@pytest.mark.parametrize("name,B,wtype,form", [("tiny", 8, "f32", 0), ("enru_b2000", 96, "f32", 0),
                                               ("enru_b2000", 96, "bf16", 1)],
                         ids=["tiny", "enru_b96", "enru_b96_bf16_streamed"])
def test_graph_replays_match_eager_step(name, B, wtype, form):
    """form 1 (nmt_debug.h) makes the bf16 products take the weight-streaming
    kernels at this size, so they are captured too."""
    torch = _torch()
    from paper_1605_04809_amd import binding as nb
    prev = nb.debug_gemm_form(form)
    try:
        _graph_replays(torch, nb, name, B, wtype)
    finally:
        nb.debug_gemm_form(prev)


def _graph_replays(torch, nb, name, B, wtype):
    wl = make_workload(CONFIGS[name].replace(B=B, seed=91, wtype=wtype))
    c = wl.cfg
    model = nb.Model.from_workload(wl)
    cu = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    src = nb.nmt_encode(model, cu(wl.src_ids), wl.src_len)
    s_prev, y_prev, sent_id, req = cu(wl.s_prev), cu(wl.y_prev), cu(wl.sent_id), cu(wl.req)
    ws = torch.empty(nb.nmt_score_workspace_bytes(model, B), dtype=torch.uint8, device="cuda")
    out = lambda: (torch.empty(B, device="cuda"), torch.empty((B, c.H), device="cuda"), torch.empty(B, device="cuda"))
    logp, s_new, logZ = out()
    # eager reference
    e_logp, e_snew, e_logZ = out()
    nb.nmt_score_batch(model, src, s_prev, y_prev, sent_id, req, e_logp, e_snew, e_logZ, workspace=ws)
    torch.cuda.synchronize()
    want = [x.cpu().numpy() for x in (e_logp, e_snew, e_logZ)]
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        nb.nmt_score_batch(model, src, s_prev, y_prev, sent_id, req, logp, s_new, logZ, workspace=ws)
    torch.cuda.current_stream().wait_stream(cap)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        nb.nmt_score_batch(model, src, s_prev, y_prev, sent_id, req, logp, s_new, logZ, workspace=ws)
    for rep in range(4):
        for x in (logp, s_new, logZ):
            x.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        for got, w, name_ in zip((logp, s_new, logZ), want, ("logp", "s_new", "logZ")):
            np.testing.assert_array_equal(got.cpu().numpy(), w, err_msg=f"replay {rep}: {name_}")
        # eager work between replays: an eager step of other rows on the same workspace
        nb.nmt_score_batch(model, src, s_prev.flip(0).contiguous(), y_prev, sent_id, req, e_logp, e_snew,
                           e_logZ, workspace=ws)
        torch.cuda.synchronize()
    assert nb.nmt_stream_status(model) == nb.NMT_OK
    print(f"{name} B={B} {wtype}: 4 graph replays equal the eager step", flush=True)
    src.close()
    model.close()
