"""Every element of large tensors and lists is written exactly once by the simulate and backward
launches, whatever order the blocks take.  With theta0 = 0, theta = 1 and s = keep (rescale), a
kept coordinate of theta~ is exactly 1 and a dropped one exactly 0; with g~ = 1, grad 0 and
lambda t = 1 the gradient is 1 where kept and 0 where dropped.  Whole tensors spanning many XCD
super-blocks (and a partial one) are compared with the keep mask of smat_debug_draws, which is
bit-exact against the oracle."""
import pytest
import torch

import paper_2609_33437_amd as smat

pytestmark = pytest.mark.gpu
DEV = "cuda"
KEEP = 0.5
P = dict(s=KEEP, keep=KEEP, sigma=0.0, rescale=1)


def kept_mask(n, tid, off, seed=17, step=5):
    kept = torch.empty(n, dtype=torch.uint8, device=DEV)
    smat.smat_debug_draws(n, P, seed, step, tid, off, kept=kept)
    return kept.bool()


def tensors(n):
    theta = torch.ones(n, device=DEV)
    theta0 = torch.zeros(n, dtype=torch.bfloat16, device=DEV)
    out = torch.full((n,), 7.0, dtype=torch.bfloat16, device=DEV)
    gs = torch.ones(n, dtype=torch.bfloat16, device=DEV)
    gt = torch.zeros(n, device=DEV)
    return theta, theta0, out, gs, gt


@pytest.mark.parametrize("n", [(1 << 24) + 4096 + 3, 5 * (1 << 20) + 1])
def test_single_tensor_every_element_once(n):
    theta, theta0, out, gs, gt = tensors(n)
    smat.smat_simulate(theta, theta0, out, P, 17, 5, 3, 0)
    smat.smat_backward_accum(gs, gt, P, 1.0, 17, 5, 3, 0)
    kept = kept_mask(n, 3, 0)
    torch.cuda.synchronize()
    assert torch.equal(out.float(), kept.float())
    assert torch.equal(gt, kept.float())


def test_list_every_element_once():
    sizes = [(1 << 23) + 3, 1, 3 * (1 << 20) + 17, 16384, (1 << 22)]
    ts = [tensors(n) for n in sizes]
    with smat.Plan([t[0] for t in ts], [t[2] for t in ts], [t[1] for t in ts], [t[3] for t in ts],
                   [t[4] for t in ts]) as plan:
        plan.set_params([P] * len(sizes))
        plan.simulate(17, 5)
        plan.switch_storage(smat.SMAT_SIMULATED)
        plan.backward_accum(17, 5, 1.0)
        plan.switch_storage(smat.SMAT_EXPERT)
        torch.cuda.synchronize()
    for i, (n, t) in enumerate(zip(sizes, ts)):
        kept = kept_mask(n, i, 0).float()
        torch.cuda.synchronize()
        assert torch.equal(t[2].float(), kept), f"tensor {i}: theta~"
        assert torch.equal(t[4], kept), f"tensor {i}: grad"


@pytest.mark.parametrize("nbytes", [48, 4096 + 16, (1 << 20) + 48, (1 << 27) + 4080])
def test_stream_copy(nbytes):
    g = torch.Generator(DEV).manual_seed(nbytes % 1000)
    src = torch.randint(0, 255, (nbytes,), dtype=torch.uint8, device=DEV, generator=g)
    dst = torch.zeros(nbytes + 64, dtype=torch.uint8, device=DEV)
    smat.smat_stream_copy(src, dst[:nbytes])
    torch.cuda.synchronize()
    assert torch.equal(dst[:nbytes], src)
    assert int(dst[nbytes:].sum()) == 0          # nothing written past the end
    with pytest.raises(smat.SmatError):
        smat.smat_stream_copy(src[1:33], dst[1:33])   # not 16-byte aligned


def test_backward_overwrite_writes_every_element():
    sizes = [(1 << 23) + 3, 1, 3 * (1 << 20) + 17]
    ts = [tensors(n) for n in sizes]
    for t in ts:
        t[4].fill_(float("nan"))                     # grad_theta is never read in overwrite mode
    with smat.Plan([t[0] for t in ts], [t[2] for t in ts], [t[1] for t in ts], [t[3] for t in ts],
                   [t[4] for t in ts]) as plan:
        plan.set_params([P] * len(sizes))
        plan.backward(17, 5, 1.0, accumulate=False)
        torch.cuda.synchronize()
    for i, (n, t) in enumerate(zip(sizes, ts)):
        kept = kept_mask(n, i, 0).float()
        torch.cuda.synchronize()
        assert torch.equal(t[4], kept), f"tensor {i}"
