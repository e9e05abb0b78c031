"""The benchmark's timed single-layer step prefetches the rule book over two streams (the next
step's build queued on a side stream behind the current forward, ordered by fence-free events).
Its results must be bit-identical to the same step with every phase in sequence on one stream:
forward output, input-feature gradient and coefficient gradient of every pipelined step."""
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
P = pytest.importorskip("paper_2111_07383_amd")

import bench  # noqa: E402  (repository root is on sys.path via conftest)

DEV = torch.device("cuda:0")


@pytest.mark.parametrize("config", [4, 2])
def test_pipelined_step_matches_sequential(config, monkeypatch):
    b = bench.SingleLayer(config, DEV)
    grads = []
    backward = P.backward

    def capture(*a, **k):
        gf, gc = backward(*a, **k)
        grads.append((gf.clone(), gc.clone()))  # on the caller's stream, behind the backward
        return gf, gc

    monkeypatch.setattr(P, "backward", capture)
    outs = [b.step().clone() for _ in range(4)]
    torch.cuda.synchronize()
    b.events = []                       # the sequential form of the same step
    ref = b.step().clone()
    torch.cuda.synchronize()
    assert len(grads) == 5
    for i, o in enumerate(outs):
        assert torch.equal(o, ref), f"forward output of pipelined step {i}"
    for i, (gf, gc) in enumerate(grads[:-1]):
        assert torch.equal(gf, grads[-1][0]), f"feature gradient of pipelined step {i}"
        assert torch.equal(gc, grads[-1][1]), f"coefficient gradient of pipelined step {i}"
