"""Concurrent calls: different streams (each with its own workspace) and
different host threads, on the tiled kernels and on the fused small-matrix
one.  Results must be bit for bit those of the same calls made one after the
other on one stream."""
import threading

import pytest

from gpu_helpers import log

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2512_04632_amd import _lib as tm  # noqa: E402


def _inputs(seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    batch = torch.randn((4, 512, 1024), generator=g, device="cuda").bfloat16()
    group = [torch.randn(s, generator=g, device="cuda").bfloat16()
             for s in [(64, 576), (768, 300), (256, 2304), (128, 128)]]
    f32 = torch.randn((2, 200, 333), generator=g, device="cuda")
    # k <= 128 only: the fused single-launch kernel
    small = [torch.randn(s, generator=g, device="cuda").bfloat16() for s in [(576, 64), (64, 576), (200, 96)]]
    return batch, group, f32, small


def _run(batch, group, f32, small):
    tm.orthogonalize(batch, 4, None, "aol")
    tm.orthogonalize_grouped(group, 4, None, "aol")
    tm.orthogonalize(f32, 4, None, "frobenius")
    tm.orthogonalize_grouped(small, 4, None, "aol")


def _copy(o):
    b, g, f, sm = o
    return b.clone(), [x.clone() for x in g], f.clone(), [x.clone() for x in sm]


def _sequential(inputs):
    outs = [_copy(o) for o in inputs]
    for o in outs:
        _run(*o)
    torch.cuda.synchronize()
    return outs


def _same(a, b):
    (ba, ga, fa, sa), (bb, gb, fb, sb) = a, b
    return (torch.equal(ba, bb) and torch.equal(fa, fb) and all(torch.equal(x, y) for x, y in zip(ga, gb))
            and all(torch.equal(x, y) for x, y in zip(sa, sb)))


def test_two_streams_match_sequential():
    log("case: calls on two streams at once")
    inputs = [_inputs(1), _inputs(2)]
    ref = _sequential(inputs)
    outs = [_copy(o) for o in inputs]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    for rep in range(3):
        work = [_copy(o) for o in outs]
        for s, w in zip(streams, work):
            s.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s):
                _run(*w)
        torch.cuda.synchronize()
        for w, r in zip(work, ref):
            assert _same(w, r), rep


def test_two_host_threads_match_sequential():
    log("case: calls from two host threads, each on its own stream")
    inputs = [_inputs(3), _inputs(4)]
    ref = _sequential(inputs)
    work = [_copy(o) for o in inputs]
    torch.cuda.synchronize()
    errors = []

    def body(w):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                _run(*w)
            s.synchronize()
        except Exception as e:  # noqa: BLE001
            errors.append(e)

    threads = [threading.Thread(target=body, args=(w,)) for w in work]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=60)
    assert not errors, errors
    assert all(not t.is_alive() for t in threads)
    torch.cuda.synchronize()
    for w, r in zip(work, ref):
        assert _same(w, r)
