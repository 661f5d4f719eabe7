"""Library calls captured into a HIP graph (torch.cuda.graph) and replayed.

Once a call has run on a stream, the library's workspace for that stream has
its size, and later calls with the same shapes on that stream neither
allocate nor synchronise, so they can be captured.  The kernels are
deterministic: every replay must reproduce the eager result bit for bit, with
unrelated eager work on the device between replays.
"""
import pytest

from gpu_helpers import log

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2512_04632_amd import _lib as tm  # noqa: E402


def _inputs(case):
    g = torch.Generator(device="cuda")
    g.manual_seed(7)

    def rn(*shape):
        return torch.randn(shape, generator=g, device="cuda")

    if case == "batched_bf16":
        return [rn(3, 256, 640).bfloat16()]
    if case == "tall_bf16":
        return [rn(2, 700, 300).bfloat16()]
    if case == "batched_f32":
        return [rn(2, 192, 320)]
    if case == "fused_bf16":        # k <= 128: the single-launch small-matrix kernel
        return [rn(16, 64, 576).bfloat16()]
    if case == "fused_grouped_bf16":
        return [rn(m, n).bfloat16() for m, n in [(64, 576), (576, 64), (17, 33), (128, 320)]]
    return [rn(m, n).bfloat16() for m, n in [(64, 576), (300, 200), (128, 1152), (768, 768)]]


def _call(xs):
    if len(xs) == 1:
        tm.orthogonalize(xs[0], 4, None, "aol")
    else:
        tm.orthogonalize_grouped(xs, 4, None, "aol")


def _busy_work():
    a = torch.randn(512, 512, device="cuda")
    return float((a @ a).sum().item())


@pytest.mark.parametrize("case", ["batched_bf16", "tall_bf16", "batched_f32", "grouped_bf16",
                                  "fused_bf16", "fused_grouped_bf16"])
def test_replays_match_eager(case):
    log(f"case: graph capture and replay, {case}")
    X0 = _inputs(case)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    ref = [x.clone() for x in X0]
    with torch.cuda.stream(side):      # eager reference on the capture stream
        _call(ref)
    side.synchronize()
    buf = [x.clone() for x in X0]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        _call(buf)
    for r in range(3):
        for b, x in zip(buf, X0):
            b.copy_(x)
        _busy_work()
        graph.replay()
        torch.cuda.synchronize()
        for i, (b, e) in enumerate(zip(buf, ref)):
            assert torch.equal(b, e), (r, i)


def test_optimizer_step_replays_match_eager():
    log("case: graph capture and replay, optimizer step")
    shapes = [(64, 96), (128, 64), (256, 512), (768, 3072)]
    g = torch.Generator(device="cuda")
    g.manual_seed(3)
    W0 = [0.02 * torch.randn(s, generator=g, device="cuda") for s in shapes]
    G = [torch.randn(s, generator=g, device="cuda") for s in shapes]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    Wr, Mr = [w.clone() for w in W0], [torch.zeros_like(w) for w in W0]
    with torch.cuda.stream(side):      # two eager steps on the capture stream
        for _ in range(2):
            tm.muon_step_grouped(Wr, G, Mr, 0.02, 0.95, True, 0.01)
    side.synchronize()
    W, M = [w.clone() for w in W0], [torch.zeros_like(w) for w in W0]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        tm.muon_step_grouped(W, G, M, 0.02, 0.95, True, 0.01)
    # capture does not run the step: two replays are the two eager steps
    for _ in range(2):
        _busy_work()
        graph.replay()
    torch.cuda.synchronize()
    for a, b in zip(W + M, Wr + Mr):
        assert torch.equal(a, b)


def test_larger_call_after_capture_keeps_the_graph_valid():
    """A workspace used under capture keeps its address: a later, larger eager call
    on the same stream gets a new workspace, and the graph's replays stay exact."""
    log("case: graph capture, then a larger eager call on the capture stream")
    X0 = _inputs("batched_bf16")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    ref = [x.clone() for x in X0]
    with torch.cuda.stream(side):
        _call(ref)
    side.synchronize()
    buf = [x.clone() for x in X0]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        _call(buf)
    big = torch.randn((2, 1024, 2048), device="cuda").bfloat16()
    big_ref = big.clone()
    tm.orthogonalize(big_ref, 4, None, "aol")      # default stream
    with torch.cuda.stream(side):                  # grows the capture stream's workspace
        tm.orthogonalize(big, 4, None, "aol", stream=side)
    side.synchronize()
    assert torch.equal(big, big_ref)
    for r in range(2):
        for b, x in zip(buf, X0):
            b.copy_(x)
        _busy_work()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(buf[0], ref[0]), r
    del graph


# the refused call enqueues nothing, so torch reports the captured graph as empty
@pytest.mark.filterwarnings("ignore:The CUDA Graph is empty")
def test_capture_with_too_small_a_workspace_is_refused():
    """Nothing can be allocated during capture: a call whose stream has no workspace
    of that size yet returns TM_ERR_UNSUPPORTED and enqueues nothing."""
    log("case: capture without a sized workspace")
    tm.release_workspaces()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    x = torch.randn((300, 700), device="cuda").bfloat16()
    keep = x.clone()
    graph = torch.cuda.CUDAGraph()
    seen = []
    with torch.cuda.graph(graph, stream=side):
        try:
            tm.orthogonalize(x, 4, None, "aol", stream=side)
        except tm.TurboMuonError as err:
            seen.append(err.status)
    torch.cuda.synchronize()
    assert seen == [tm.TM_ERR_UNSUPPORTED]
    graph.replay()
    torch.cuda.synchronize()
    assert torch.equal(x, keep)
    del graph
