"""tm_orthogonalize_noalloc through the C ABI: the allocation-free entry point
(workspace in the library's static per-GPU scratch array) against
tm_orthogonalize, which plans the same launches over an allocated workspace.

Two calls in a row share the one scratch array, the second on a smaller input,
so the second must not depend on what the first left behind.  Both must equal
the cached-workspace call bit for bit and stay within the bf16 tolerance of the
fp64 oracle."""
import numpy as np
import pytest

from oracle import turbomuon as O
from gpu_helpers import BF16_TOL, from_device, log, make_input, relF, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2512_04632_amd import _lib as tm  # noqa: E402


def _pair(Xs, iters, precond):
    """(no-alloc result, cached-workspace result) of one batched call."""
    a = torch.stack([to_device(X, "bf16") for X in Xs]).contiguous()
    b = a.clone()
    tm.orthogonalize_noalloc(a, iters, None, precond)
    tm.orthogonalize(b, iters, None, precond)
    torch.cuda.synchronize()
    return a, b


@pytest.mark.parametrize("precond,iters", [("aol", 4), ("frobenius", 5)])
def test_noalloc_matches_allocating_call_twice(precond, iters):
    log(f"case: noalloc {precond} t={iters}: 3 x 768 x 3072, then 1 x 520 x 257 (tall)")
    first = [make_input(768, 3072, 0.8, 40 + i, "bf16") for i in range(3)]
    a, b = _pair(first, iters, precond)
    assert torch.equal(a, b)
    second = [make_input(520, 257, 0.8, 50, "bf16")]
    c, d = _pair(second, iters, precond)
    assert torch.equal(c, d)
    for X, G in ((first[0], a[0]), (first[2], a[2]), (second[0], c[0])):
        e = relF(from_device(G), O.orthogonalize(X, iters, None, precond))
        log(f"relF vs oracle {e:.3e}")
        assert e <= BF16_TOL


def test_noalloc_rejects_calls_beyond_the_scratch():
    """A call whose workspace exceeds the static array fails before anything is
    enqueued: the input is left as it was."""
    need = tm.workspace_bytes([(2048, 8192)], 2)
    assert need > tm.TM_NOALLOC_SCRATCH_BYTES
    x = torch.randn((2048, 8192), device="cuda").to(torch.bfloat16)
    keep = x.clone()
    with pytest.raises(tm.TurboMuonError) as err:
        tm.orthogonalize_noalloc(x, 4, None, "aol")
    assert err.value.status == tm.TM_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert torch.equal(x, keep)
    # and the entry point still works afterwards
    X = make_input(64, 576, 1.0, 7, "bf16")
    g, h = _pair([X], 4, "aol")
    assert torch.equal(g, h)


def test_noalloc_graph_replays_match_eager():
    """Captured into a HIP graph (no allocation during capture), replayed three
    times with eager work between the replays: each replay equals the eager call."""
    log("case: noalloc call captured in a graph, 2 x 256 x 1000 AOL t=4")
    Xs = [make_input(256, 1000, 0.8, 60 + i, "bf16") for i in range(2)]
    src = torch.stack([to_device(X, "bf16") for X in Xs]).contiguous()
    ref = src.clone()
    tm.orthogonalize(ref, 4, None, "aol")
    buf = src.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        tm.orthogonalize_noalloc(buf, 4, None, "aol", stream=side)   # warm the code path
    side.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        tm.orthogonalize_noalloc(buf, 4, None, "aol", stream=side)
    torch.cuda.synchronize()
    for r in range(3):
        buf.copy_(src)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(buf, ref), r
        other = to_device(make_input(300, 200, 0.8, 70 + r, "bf16"), "bf16")
        tm.orthogonalize_noalloc(other, 4, None, "aol")   # eager use of the same scratch
        torch.cuda.synchronize()
    del graph
