"""bcpnn_structural_update_static, the structural update for callers that cannot allocate:
through the C ABI, against bcpnn_structural_update on the same state -- masks, weights and the
swap count equal bit for bit -- on two calls in a row, the second on a smaller layer (the
shared static scratch then holds the first call's scores), and its size limit."""
import numpy as np
import pytest

from paper_2106_05373_amd import synth

from pairs import bcpnn, gpu_config, workload_config, workload_mask

pytestmark = pytest.mark.gpu

MNIST = synth.WORKLOADS["mnist"]


@pytest.fixture(autouse=True)
def _announce(request):
    print(f"\n[gpu case] {request.node.nodeid}", flush=True)
    yield


def _trained_pair(cfg, mask, xs):
    """Two layers with the same configuration and mask, trained on the same batches."""
    import torch
    B = bcpnn()
    out = []
    for _ in range(2):
        lay = B.Layer(cfg, mask)
        for x in xs:
            lay.train_batch(torch.from_numpy(np.ascontiguousarray(x)).cuda())
        out.append(lay)
    return out


def _compare(ref, sta):
    import torch
    n_ref = ref.structural_update()
    n_dev = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    sta.structural_update_static(n_dev)
    n_sta = int(n_dev.cpu()[0])
    s_ref, s_sta = ref.get_state(), sta.get_state()
    for key in s_ref:
        assert np.array_equal(s_ref[key].view(np.uint8), s_sta[key].view(np.uint8)), key
    assert n_sta == n_ref, (n_sta, n_ref)
    return n_ref


def test_static_structural_update_matches_the_allocating_one():
    B = bcpnn()
    # first call: the MNIST-shaped layer, trained at a rate that gives real swaps
    px, _ = synth.dataset(MNIST, n=128 * 12)
    X = synth.encode_pixels(px)
    cfg = workload_config(MNIST, alpha=0.05, n_swaps=2)
    ref, sta = _trained_pair(cfg, workload_mask(MNIST), [X[k * 128:(k + 1) * 128] for k in range(12)])
    n1 = _compare(ref, sta)
    with pytest.raises(B.BcpnnError) as ei:          # the scores live in the shared scratch
        sta.get_mi()
    assert ei.value.status == -1
    ref.close()
    sta.close()
    # second call: a smaller layer; the scratch still holds the first call's larger score table
    rng = np.random.default_rng(3)
    hin, hout, mout, k = 40, 6, 20, 17
    mask = np.stack([synth.random_mask(hin, 1, k, 90 + c)[:, 0] for c in range(hout)], 1)
    cfg2 = gpu_config(hin, 2, hout, mout, 48, alpha=0.1, gain=2.0, complement_pairs=1)
    xs = [synth.encode_pixels(rng.random((48, hin)).astype(np.float32)) for _ in range(10)]
    ref, sta = _trained_pair(cfg2, mask, xs)
    n2 = _compare(ref, sta)
    # with no swap configured the count is 0 (not the scratch's last counts)
    cfg3 = gpu_config(hin, 2, hout, mout, 48, alpha=0.1, gain=2.0, n_swaps=0)
    ref3, sta3 = _trained_pair(cfg3, mask, xs[:3])
    assert _compare(ref3, sta3) == 0
    for lay in (ref, sta, ref3, sta3):
        lay.close()
    print(f"swaps: first call {n1}, second call {n2}")
    assert n1 > 0 and n2 > 0


def test_static_structural_update_rejects_a_table_beyond_its_scratch():
    """49152 x 100 HCU pairs need 39 MB of scores, more than the 32 MiB scratch: EINVAL, and the
    layer stays usable."""
    B = bcpnn()
    cfg = gpu_config(49152, 2, 100, 1, 16)
    mask = np.stack([synth.random_mask(49152, 1, 100, 200 + c)[:, 0] for c in range(100)], 1)
    lay = B.Layer(cfg, mask)
    with pytest.raises(B.BcpnnError) as ei:
        lay.structural_update_static(None)
    assert ei.value.status == -1 and "scratch" in str(ei.value)
    assert lay.structural_update() >= 0             # the allocating update still runs
    lay.close()
