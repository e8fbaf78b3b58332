"""GPU: the library keeps no state between calls, so calls on different streams may
run at the same time, and a call's kernels can be captured in a HIP graph and
replayed (no allocation, no memset and no synchronous call on the path).  Every
result must equal the eager, single-stream one bit for bit."""
import pytest
import torch

import workloads as W
from tests.gpu_util import gpu_run, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_13126_amd  # noqa: F401  (fails loudly if the library is missing)


def int_view(t):
    return t.view(torch.int32 if t.dtype == torch.float32 else torch.int16)


def test_two_streams_at_once():
    # the 8B RAG tail (split-KV partials in its own workspace) and the decode batch,
    # each written and attended on its own stream, interleaved, several times
    a, b = gpu_run(W.llama3_8b_rag()), gpu_run(W.decode_64req(num_reqs=8, num_spans=4, span_len=128))
    ref_a, ref_b = a.o.clone(), b.o.clone()
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()   # default priority
    torch.cuda.synchronize()
    say("[gpu] streams: 8B RAG tail and decode on two streams, 5 rounds")
    for _ in range(5):
        a.o.zero_()
        b.o.zero_()
        torch.cuda.synchronize()
        with torch.cuda.stream(sa):
            a.write()
            a.attend()
        with torch.cuda.stream(sb):
            b.write()
            b.attend()
        torch.cuda.synchronize()
        assert torch.equal(int_view(a.o), int_view(ref_a))
        assert torch.equal(int_view(b.o), int_view(ref_b))


@pytest.mark.parametrize("name", ["llama3_8b_rag", "decode"])
def test_graph_capture_and_replay(name):
    wl = W.llama3_8b_rag() if name == "llama3_8b_rag" else W.decode_64req(num_reqs=8, num_spans=4, span_len=128)
    db = gpu_run(wl)
    ref = db.o.clone()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    say(f"[gpu] graph: capture kv_write + attention of {wl.name}")
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            db.write()
            db.attend()
    torch.cuda.synchronize()
    for r in range(3):
        # eager work of the program between the replays
        db.o.fill_(7.0)
        junk = torch.randn(1 << 20, device="cuda").sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        say(f"  replay {r}: junk={float(junk):.3f}")
        assert torch.equal(int_view(db.o), int_view(ref))
    # and an eager call afterwards still gives the same result
    db.o.zero_()
    db.attend()
    torch.cuda.synchronize()
    assert torch.equal(int_view(db.o), int_view(ref))
