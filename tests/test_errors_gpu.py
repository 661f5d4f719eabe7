"""Failure paths on the GPU: a workspace allocation that fails is reported as
TM_ERR_NO_MEMORY before anything is enqueued, and the library recovers.  The
failure is forced from the host (the TM_TEST_FAIL_ALLOC switch of the
workspace cache); every kernel that does run exits normally."""
import pytest

from gpu_helpers import log, make_input, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2512_04632_amd import _lib as tm  # noqa: E402


def test_failed_allocation_reports_no_memory_and_recovers(monkeypatch):
    log("case: forced workspace allocation failure, 512 x 1536 bf16 AOL t=4")
    X = make_input(512, 1536, 0.8, 2, "bf16")
    ref = to_device(X, "bf16")
    tm.orthogonalize(ref, 4, None, "aol")
    torch.cuda.synchronize()
    tm.release_workspaces()            # every cache empty: the next call must allocate
    x = to_device(X, "bf16")
    keep = x.clone()
    monkeypatch.setenv("TM_TEST_FAIL_ALLOC", "1")
    with pytest.raises(tm.TurboMuonError) as err:
        tm.orthogonalize(x, 4, None, "aol")
    assert err.value.status == tm.TM_ERR_NO_MEMORY
    assert "allocation" in tm.last_error()
    torch.cuda.synchronize()
    assert torch.equal(x, keep)        # nothing was enqueued
    # the allocation-free entry point needs no allocation, so it still runs
    y = x.clone()
    tm.orthogonalize_noalloc(y, 4, None, "aol")
    torch.cuda.synchronize()
    assert torch.equal(y, ref)
    monkeypatch.delenv("TM_TEST_FAIL_ALLOC")
    tm.orthogonalize(x, 4, None, "aol")
    torch.cuda.synchronize()
    assert torch.equal(x, ref)
