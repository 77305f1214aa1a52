"""Both device entry points enqueue one kernel on the caller's stream and
allocate nothing, so a caller can capture them in a HIP graph.  Each test
captures one call, then replays the graph several times with eager work in
between (the outputs are overwritten before every replay) and checks every
replay against the eager result."""
import pytest

from paper_2609_26219_amd import binding as pb
from paper_2609_26219_amd import workloads as wl
from parity import log, oracle_checkpoint

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as _t
    if not _t.cuda.is_available():
        pytest.skip("no GPU")
    pb.load()
    return _t


def test_restore_replays_from_a_graph(torch):
    from paper_2609_26219_amd.device import DeviceRestore
    log("[gpu] graph capture: pkv_restore on llama8b_1l, 4 replays")
    case = wl.make_case("llama8b_1l")
    dr = DeviceRestore(case, checkpoint=oracle_checkpoint(case))
    dr.run()
    torch.cuda.synchronize()
    want_k, want_v = dr.k_cache.clone(), dr.v_cache.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, capture_error_mode="thread_local"):
        pb.restore_tensors(dr.plan, dr.payload, dr.scales, dr.k_cache, dr.v_cache)
    for _ in range(4):
        dr.prefill()
        torch.cuda.synchronize()
        assert not torch.equal(dr.k_cache, want_k)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(dr.k_cache, want_k) and torch.equal(dr.v_cache, want_v)


def test_checkpoint_write_replays_from_a_graph(torch):
    from paper_2609_26219_amd.device import DeviceCheckpoint, OldCaches
    log("[gpu] graph capture: pkv_quantize_gather on llama8b_1l, 4 replays")
    case = wl.make_case("llama8b_1l")
    ck = DeviceCheckpoint(case, OldCaches(case))
    ck.write()
    torch.cuda.synchronize()
    want_p, want_s = ck.payload.clone(), ck.scales.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, capture_error_mode="thread_local"):
        pb.quantize_gather_tensors(ck.plan, ck.old.k, ck.old.v, ck.payload, ck.scales)
    for i in range(4):
        ck.payload.fill_(0xA0 + i)
        ck.scales.fill_(0x1234 + i)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(ck.payload, want_p) and torch.equal(ck.scales, want_s)
