"""The library issues only kernel launches on the caller's stream (no allocation, memset,
copy or synchronisation), so a prefill or decode step can be captured into a HIP graph.
Each replay is compared bit for bit with an eager call on the same inputs, with eager work
and synchronisations between the replays."""
import pytest
import torch

from kvp_inputs import device as kd
from paper_2608_15943_amd import binding as kb

from gpu_util import DEV, build_device_model, say, small_workload, workspace

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    kb.lib()


def _capture(run):
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        run()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    torch.cuda.synchronize()
    return g


def test_decode_step_replays_match_eager():
    w = small_workload("graph-dec", 4, 512, 4, 2, [0, 0, 2, 2], seed=41)
    B, cap = 6, 256
    lens = [0, 5, 63, 64, 130, 200]
    say(f"[graph decode] B={B} lens={lens}")
    dm = build_device_model(w, B, 1, cap, fill_cache_npos=max(lens))
    x = torch.empty((B, w.h), dtype=torch.bfloat16, device=DEV)
    kd.fill_decode_x(w, x.data_ptr(), B)
    lens_t = torch.tensor(lens, dtype=torch.int32, device=DEV)
    ws, n = workspace(dm, kb.KVP_PHASE_DECODE, B)
    y = torch.empty_like(x)

    def run():
        dm.model.kvp_decode_step(x.data_ptr(), lens_t.data_ptr(), max(lens), y.data_ptr(), B, ws.data_ptr(), n,
                                 torch.cuda.current_stream().cuda_stream)

    run()
    torch.cuda.synchronize()
    ref = y.clone()
    g = _capture(run)
    for rep in range(4):
        y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, ref), rep
        run()                                   # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(y, ref), rep
    say("  4 replays bit-identical to eager")


def test_prefill_replays_match_eager():
    w = small_workload("graph-pre", 3, 512, 4, 2, [0, 0, 2], seed=42)
    B, S = 2, 200
    say(f"[graph prefill] B={B} S={S}")
    dm = build_device_model(w, B, S, 256)
    x = torch.empty((B, S, w.h), dtype=torch.bfloat16, device=DEV)
    kd.fill_prefill_x(w, x.data_ptr(), B, S)
    ws, n = workspace(dm, kb.KVP_PHASE_PREFILL, B, S)
    y = torch.empty_like(x)

    def run():
        dm.model.kvp_prefill(x.data_ptr(), y.data_ptr(), B, S, ws.data_ptr(), n,
                             torch.cuda.current_stream().cuda_stream)

    run()
    torch.cuda.synchronize()
    ref = y.clone()
    g = _capture(run)
    for rep in range(3):
        y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, ref), rep
        run()
        torch.cuda.synchronize()
    say("  3 replays bit-identical to eager")
