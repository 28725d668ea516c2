"""The routed layer captured as a HIP graph: every replay must give the
eager pass's output bit for bit (the kernels are deterministic and the graph
holds no memset nodes), with eager work and synchronisations between the
replays."""
import sys

import pytest
import torch

from paper_2609_23733_amd import synth

pytestmark = pytest.mark.gpu


def log(msg):
    sys.stdout.write("[gpu-case] %s\n" % msg)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_23733_amd import vp
    vp.load_library()


@pytest.mark.parametrize("S,P,dtype,sharp", [(2, 1374, "bf16", False), (1, 1500, "bf16", True),
                                             (2, 700, "f32", True)])
def test_graph_replays_equal_eager(S, P, dtype, sharp):
    from paper_2609_23733_amd import vp
    log("graph S=%d P=%d %s sharp=%d" % (S, P, dtype, sharp))
    modes = torch.tensor([2, 1, 0, 2, 1, 0, 2, 0, 1, 0, 2, 1, 0, 0, 1, 2], dtype=torch.uint8).numpy()
    x = synth.make_layer(S, P, dtype=dtype, key=(80, S), sharp=sharp, modes=modes,
                         qkv_device="cuda")
    layer = vp.RoutedLayer(x, y_dtype=torch.float32)
    Y0 = layer.step().clone()
    modes0 = layer.modes.clone()
    torch.cuda.synchronize()
    g = vp.LayerGraph(layer)
    for k in range(4):
        layer.Y.fill_(float("nan"))            # eager work between replays
        torch.cuda.synchronize()
        Y = g.replay()
        torch.cuda.synchronize()
        assert torch.equal(layer.modes, modes0), k
        assert torch.equal(Y, Y0), (k, (Y - Y0).abs().max().item())
        if k == 1:                             # an eager pass in between
            torch.cuda.synchronize()
            assert torch.equal(layer.step(), Y0)
            torch.cuda.synchronize()
