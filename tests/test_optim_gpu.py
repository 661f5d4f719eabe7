"""The optimizer step (tm_muon_step_grouped) against the fp64 oracle's step."""
import numpy as np
import pytest

from oracle import turbomuon as O
from paper_2512_04632_amd import synth
from gpu_helpers import BF16_TOL, log

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2512_04632_amd import _lib as tm  # noqa: E402
from paper_2512_04632_amd.optim import TurboMuon  # noqa: E402

SHAPES = [(64, 96), (96, 64), (128, 128), (17, 300), (300, 17), (1, 5), (768, 3072), (3072, 768)]
# only matrices the fused small-matrix kernel takes (k <= 128, within one compute unit's LDS)
SMALL_SHAPES = [(64, 96), (96, 64), (128, 128), (17, 300), (300, 17), (1, 5), (64, 576)]


def f32(x):
    return np.asarray(x, dtype=np.float32).astype(np.float64)


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


def host(t):
    return t.detach().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("shapes", [SHAPES, SMALL_SHAPES], ids=["mixed", "small"])
@pytest.mark.parametrize("nesterov", [True, False])
@pytest.mark.parametrize("wd", [0.0, 0.05])
def test_two_grouped_steps_match_the_oracle(nesterov, wd, shapes):
    log(f"case: grouped optimizer steps nesterov={nesterov} wd={wd} shapes={shapes}")
    lr, mu = 0.02, 0.9
    Ws = [f32(0.02 * synth.gaussian_matrix(m, n, 10 + i)) for i, (m, n) in enumerate(shapes)]
    Ms = [f32(0.1 * synth.gaussian_matrix(m, n, 20 + i)) for i, (m, n) in enumerate(shapes)]
    tW, tM = [dev(w) for w in Ws], [dev(m) for m in Ms]
    for step in range(2):
        Gs = [f32(synth.power_law_matrix(m, n, 0.8, 100 * step + i)) for i, (m, n) in enumerate(shapes)]
        tG = [dev(g) for g in Gs]
        tm.muon_step_grouped(tW, tG, tM, lr, mu, nesterov, wd)
        torch.cuda.synchronize()
        for i, (m, n) in enumerate(shapes):
            Wr, Mr, Or = O.muon_step(Ws[i], Gs[i], Ms[i], lr, mu, nesterov, wd)
            Wg, Mg = host(tW[i]), host(tM[i])
            # momentum: one fp32 multiply-add per element
            assert np.max(np.abs(Mg - Mr)) <= 1e-6 * max(1.0, np.max(np.abs(Mr))), (step, i)
            # the step taken, against the oracle's -lr scale O
            D = Wg - Ws[i] * (1 - lr * wd)
            Dr = Wr - Ws[i] * (1 - lr * wd)
            e = O.rel_frobenius(D, Dr)
            assert e <= BF16_TOL, (step, i, e)
            Ws[i], Ms[i] = Wg, Mg        # continue from the GPU's state
    log("ok")


def test_optimizer_class_equals_direct_call():
    log("case: TurboMuon.step vs tm_muon_step_grouped")
    shapes = [(32, 48), (48, 32), (64, 64)]
    torch.manual_seed(0)
    ps = [torch.nn.Parameter(0.02 * torch.randn(m, n, device="cuda")) for m, n in shapes]
    ref = [p.detach().clone() for p in ps]
    bufs = [torch.zeros_like(p) for p in ps]
    opt = TurboMuon(ps, lr=0.05, momentum=0.9, weight_decay=0.01)
    for step in range(3):
        grads = [torch.randn_like(p) for p in ps]
        for p, g in zip(ps, grads):
            p.grad = g.clone()
        opt.step()
        tm.muon_step_grouped(ref, grads, bufs, 0.05, 0.9, True, 0.01)
        torch.cuda.synchronize()
        for p, r in zip(ps, ref):
            assert torch.equal(p.detach(), r), step


def test_zero_gradient_only_decays():
    W = dev(synth.gaussian_matrix(40, 70, 3))
    W0 = W.clone()
    G = torch.zeros_like(W)
    M = torch.zeros_like(W)
    tm.muon_step_grouped([W], [G], [M], 0.5, 0.9, True, 0.1)
    torch.cuda.synchronize()
    assert torch.equal(M, G)
    assert torch.allclose(W, W0 * 0.95, rtol=1e-6, atol=0)


def test_unaligned_and_ragged_sizes():
    """Matrices whose pointers are not 16-byte aligned or whose sizes are not
    multiples of 4 take the scalar path: same values as the vector path."""
    log("case: optimizer scalar path")
    shapes = [(3, 7), (33, 65), (64, 64)]
    ws = [dev(0.02 * synth.gaussian_matrix(m, n, i)) for i, (m, n) in enumerate(shapes)]
    gs = [dev(synth.power_law_matrix(m, n, 1.0, 5 + i)) for i, (m, n) in enumerate(shapes)]
    ms = [torch.zeros_like(w) for w in ws]
    # copies stored 4 bytes past a 16-byte boundary
    def off(t):
        buf = torch.zeros(t.numel() + 4, device="cuda")
        v = buf[1:1 + t.numel()].view(t.shape)
        v.copy_(t)
        return v
    ws2, gs2, ms2 = [off(w) for w in ws], [off(g) for g in gs], [off(m) for m in ms]
    assert ws2[2].data_ptr() % 16 == 4
    tm.muon_step_grouped(ws, gs, ms, 0.1, 0.9, True, 0.01)
    tm.muon_step_grouped(ws2, gs2, ms2, 0.1, 0.9, True, 0.01)
    torch.cuda.synchronize()
    for a, b in zip(ws + ms, ws2 + ms2):
        assert torch.equal(a, b)
