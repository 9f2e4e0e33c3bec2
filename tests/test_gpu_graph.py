"""The layer stack captured as a HIP graph: every replay must reproduce the eager
step bit for bit (the kernels are deterministic and every buffer is preallocated),
also with unrelated eager work and synchronisations between the replays."""

import pytest
import torch

from paper_2106_12736_amd import inputs, layers

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("wl", [inputs.LAYER64, inputs.STACK256], ids=lambda w: w.name)
def test_graph_replays_match_eager(wl):
    print(f"graph {wl.name}", flush=True)
    d = inputs.make_cic_stack(wl)
    x = torch.from_numpy(d.x).cuda()
    Ks = [torch.from_numpy(k).cuda() for k in d.kernels]
    g = torch.from_numpy(d.grad).cuda()
    stack = layers.CicStack(wl.batch, wl.sizes, wl.channels)
    gin = torch.empty_like(x)

    def step():
        stack.forward(x, Ks)
        stack.backward(g, Ks, input_grad=gin)

    def outputs():
        return [a.clone() for a in stack.acts] + [k.clone() for k in stack.gks] + [gin.clone()]

    step()
    torch.cuda.synchronize()
    ref = outputs()

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for rep in range(4):
        # unrelated eager work on the same buffers' device between replays
        scratch = torch.randn(1 << 20, device="cuda")
        scratch.mul_(2.0).sum().item()
        for t in stack.acts + stack.gks + [gin]:
            t.zero_()
        graph.replay()
        torch.cuda.synchronize()
        got = outputs()
        for i, (a, b) in enumerate(zip(ref, got)):
            assert torch.equal(a, b), f"replay {rep}: output {i} differs from the eager step"


def test_classifier_graph_replays_follow_eager_steps():
    """A captured training step of the FDCNN classifier advances its own state (the Adam
    step count lives on the device): from the same start, replay r must equal eager step
    r bit for bit, with unrelated eager work between the replays."""
    wl = inputs.LAYER64
    d = inputs.make_cic_stack(wl)
    x = torch.from_numpy(d.x).cuda()
    clf = layers.FdcnnClassifier(wl.batch, wl.sizes, wl.channels, classes=2, lr=1e-3)
    gen = torch.Generator().manual_seed(5)
    W = torch.randn((2, clf.features), generator=gen) * (2.0 / clf.features) ** 0.5
    clf.load([torch.from_numpy(k).cuda() for k in d.kernels], W.cuda(), torch.zeros(2).cuda())
    labels = torch.tensor([0, 1], dtype=torch.int32, device="cuda")
    start = clf.state()

    eager = []
    for _ in range(4):
        clf.train_step(x, labels)
        torch.cuda.synchronize()
        eager.append([t.clone() for t in (clf.loss, clf.params, clf.m, clf.v, clf.step_count)])

    clf.set_state(start)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        clf.train_step(x, labels)
    clf.set_state(start)  # capture ran nothing, but start from a known state anyway
    for rep in range(4):
        scratch = torch.randn(1 << 20, device="cuda")
        scratch.mul_(2.0).sum().item()
        graph.replay()
        torch.cuda.synchronize()
        got = (clf.loss, clf.params, clf.m, clf.v, clf.step_count)
        for a, b in zip(eager[rep], got):
            assert torch.equal(a, b), f"replay {rep}"
    assert int(clf.step_count.item()) == 4
