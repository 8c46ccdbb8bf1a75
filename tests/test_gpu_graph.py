"""HIP graph capture of the library's calls (the capture rules in include/bcpnn.h).

A training sequence -- batches, a structural update and the flush -- captured on the layer's
stream and replayed once leaves the same state, bit for bit, as the same calls made eagerly
(the silent-block sweeps on the layer's second stream join the capture through events).  A
captured forward pass, which keeps no host-side state, replays several times with eager
training between the replays, each replay's activities equal to an eager forward pass from the
state at that point.
"""
import numpy as np
import pytest

from paper_2106_05373_amd import synth

from pairs import bcpnn, workload_config, workload_mask

pytestmark = pytest.mark.gpu

MNIST = synth.WORKLOADS["mnist"]


@pytest.fixture(autouse=True)
def _announce(request):
    print(f"\n[gpu case] {request.node.nodeid}", flush=True)
    yield


def _batches(n):
    px, _ = synth.dataset(MNIST, n=128 * n)
    x = synth.encode_pixels(px)
    import torch
    return torch.from_numpy(x).cuda()


@pytest.mark.parametrize("pairs", [1, 0])
def test_captured_training_replayed_once_equals_eager(pairs):
    import torch
    X = _batches(14)
    cfg = workload_config(MNIST, alpha=0.02, complement_pairs=pairs)
    mask = workload_mask(MNIST)
    states = []
    for mode in ("eager", "graph"):
        stream = torch.cuda.Stream()
        lay = bcpnn().Layer(cfg, mask, stream=stream)
        for k in range(2):                                 # two eager batches first
            lay.train_batch(X[k * 128:(k + 1) * 128])
        torch.cuda.synchronize()

        def seq():
            for k in range(2, 14):                         # sweeps of 8, then the flush
                if k == 9:
                    lay.structural_update(count=False)
                lay.train_batch(X[k * 128:(k + 1) * 128])
            lay.flush()

        if mode == "eager":
            seq()
        else:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=stream):
                seq()
            torch.cuda.synchronize()
            with torch.cuda.stream(stream):
                g.replay()
        torch.cuda.synchronize()
        states.append(lay.get_state())
        lay.close()
    for key in states[0]:
        assert np.array_equal(states[0][key].view(np.uint8), states[1][key].view(np.uint8)), key


def test_captured_forward_replays_with_training_between():
    import torch
    X = _batches(8)
    stream = torch.cuda.Stream()
    lay = bcpnn().Layer(workload_config(MNIST, alpha=0.05), workload_mask(MNIST), stream=stream)
    ref = bcpnn().Layer(workload_config(MNIST, alpha=0.05), workload_mask(MNIST), stream=stream)
    xq = X[:128]
    y_g = torch.empty((128, lay.n_out), device="cuda")
    y_e = torch.empty_like(y_g)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        lay.forward(xq, y_g)
    torch.cuda.synchronize()
    for rep in range(3):
        for k in range(2 * rep + 1, 2 * rep + 3):         # eager training moves both layers
            lay.train_batch(X[k * 128:(k + 1) * 128])
            ref.train_batch(X[k * 128:(k + 1) * 128])
        with torch.cuda.stream(stream):
            g.replay()
            ref.forward(xq, y_e)
        torch.cuda.synchronize()
        assert torch.equal(y_g, y_e), f"replay {rep}"
    lay.close()
    ref.close()
