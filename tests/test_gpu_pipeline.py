"""The two-layer network (hidden layer + supervised readout) against the oracle.

The readout learns in lockstep with an oracle readout fed the same hidden activities and
targets (traces max-abs 1e-5, weights 1e-4 * max(1, |w|) after every batch); inference from the
trained states must give the oracle's class for every held-out sample whose top two readout
supports are not within rounding of each other.
"""
import numpy as np
import pytest

import oracle
from paper_2106_05373_amd import synth

from pairs import TOL_ACT, assert_weights_close, max_abs, workload_config, workload_mask

pytestmark = pytest.mark.gpu


def test_pipeline_readout_lockstep_and_inference_agree_with_oracle():
    import torch
    from paper_2106_05373_amd.pipeline import Network

    w = synth.WORKLOADS["tiny"]
    L = w.layer
    B = w.batch
    n_classes = 4                                   # the blob prototypes of the tiny workload
    px, labels = synth.dataset(w)
    tx, tlabels = synth.dataset(w, split="test", n=512)
    X = synth.encode_pixels(px)
    Xt = synth.encode_pixels(tx)
    T = synth.one_hot(labels, n_classes)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()

    cfg = workload_config(w)
    net = Network(cfg, workload_mask(w), n_classes)
    per_epoch = w.n_train // B
    for e in range(2):                              # hidden layer, unsupervised
        perm = synth.epoch_permutation(w.n_train, w.seed_shuffle, e)
        xe = dev(X[perm])
        for k in range(per_epoch):
            net.train_hidden(xe[k * B:(k + 1) * B])

    # readout in lockstep: the oracle readout sees the GPU's hidden activities
    rc = net.readout.cfg
    ro = oracle.OracleLayer(oracle.make_params(rc.in_hcu, rc.in_mcu, rc.out_hcu, rc.out_mcu,
                                               alpha=rc.alpha, seed=rc.seed))
    st = net.readout.get_state()
    for key in ("pi", "pj", "pij", "w", "mask"):
        assert np.array_equal(st[key], ro.get_state()[key]), key
    perm = synth.epoch_permutation(w.n_train, w.seed_shuffle, 2)
    xe, te = dev(X[perm]), dev(T[perm])
    y = torch.empty((B, net.hidden.n_out), device="cuda", dtype=torch.float32)
    worst = 0.0
    for k in range(per_epoch):
        net.train_readout(xe[k * B:(k + 1) * B], te[k * B:(k + 1) * B])
        net.hidden.forward(xe[k * B:(k + 1) * B], y)
        ro.train_batch(y.cpu().numpy(), T[perm][k * B:(k + 1) * B])
        sg, so = net.readout.get_state(), ro.get_state()
        for key in ("pi", "pj", "pij"):
            err = max_abs(sg[key], so[key])
            worst = max(worst, err)
            assert err <= TOL_ACT, (k, key, err)
        assert_weights_close(sg["w"], so["w"], f"readout w, batch {k}")
        assert_weights_close(sg["b"], so["b"], f"readout b, batch {k}")
        ro.set_state(sg)                            # re-sync: the next batch starts equal
    print(f"readout lockstep: worst trace error {worst:.2e}")

    # held-out inference from the trained states
    pred = net.predict(dev(Xt)).cpu().numpy()
    ho = oracle.OracleLayer(oracle.make_params(L.in_hcu, L.in_mcu, L.out_hcu, L.out_mcu,
                                               gain=w.gain))
    ho.set_state(net.hidden.get_state())
    ro.set_state(net.readout.get_state())
    _, yo = ho.forward(Xt)
    s = oracle.support(ro.p, yo, ro.w, ro.b)
    ora = oracle.readout(ro.p, s)[:, 0]
    top2 = np.sort(s, axis=1)[:, -2:]
    clear = (top2[:, 1] - top2[:, 0]) > 1e-5 * np.maximum(1.0, np.abs(top2[:, 1]))
    assert np.array_equal(pred[clear], ora[clear]), int(np.sum(pred[clear] != ora[clear]))
    acc = float(np.mean(pred == tlabels))
    print(f"held-out: {int(clear.sum())} of {len(pred)} clear of ties, accuracy {acc:.3f} "
          f"(reported, not asserted: the method's accuracy on this tiny run is not a parity "
          f"property)")
    net.close()


def test_mnist_shaped_readout_lockstep_and_heldout_inference():
    """The readout pipeline at its own shapes: the MNIST-shaped hidden layer (784 x 2 -> 30 x 100,
    10% receptive fields, the pipeline's learning settings) feeding a 1 x 10 readout whose 30
    input HCUs have 100 MCUs each (3000 input units).  After 150 hidden batches on the GPU (one
    structural update), the readout learns 30 batches in lockstep with an oracle readout fed
    the same hidden activities and re-synchronised before each: the change of every readout
    trace, and the weights, per batch.  Then inference on 2000 held-out samples from the trained
    states: the hidden activities against the oracle's, the readout's support over all ten
    classes against the oracle's support of the same activities, and the GPU's class for every
    sample whose top two supports are not within rounding of each other against the oracle's."""
    import torch
    from paper_2106_05373_amd.pipeline import Network
    from pairs import assert_increments_close, assert_support_close, decay

    w = synth.WORKLOADS["mnist_pipeline"]
    L = w.layer
    B = w.batch
    n_hidden, n_read = 150, 30
    px, labels = synth.dataset(w, n=B * (n_hidden + n_read))
    tx, tlabels = synth.dataset(w, split="test", n=2000)
    X = synth.encode_pixels(px)
    Xt = synth.encode_pixels(tx)
    T = synth.one_hot(labels, w.readout_mcu)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()

    net = Network(workload_config(w), workload_mask(w), w.readout_mcu)
    for k in range(n_hidden):
        if (k + 1) % w.period == 0:
            net.hidden.structural_update(count=False)
        net.train_hidden(dev(X[k * B:(k + 1) * B]))

    rc = net.readout.cfg
    assert (rc.in_hcu, rc.in_mcu, rc.out_hcu, rc.out_mcu) == (30, 100, 1, 10)
    ro = oracle.OracleLayer(oracle.make_params(rc.in_hcu, rc.in_mcu, rc.out_hcu, rc.out_mcu,
                                               alpha=rc.alpha, gain=rc.gain,
                                               bias_gain=rc.bias_gain, seed=rc.seed))
    st = net.readout.get_state()
    for key in ("pi", "pj", "pij", "w", "mask"):
        assert np.array_equal(st[key], ro.get_state()[key]), key
    y = torch.empty((B, net.hidden.n_out), device="cuda", dtype=torch.float32)
    for k in range(n_hidden, n_hidden + n_read):
        xb, tb = X[k * B:(k + 1) * B], T[k * B:(k + 1) * B]
        prior = net.readout.get_state()
        ro.set_state(prior)
        net.hidden.forward(dev(xb), y)
        net.train_readout(dev(xb), dev(tb))
        ro.train_batch(y.cpu().numpy(), tb)
        sg, so = net.readout.get_state(), ro.get_state()
        for key in ("pi", "pj", "pij"):
            assert max_abs(sg[key], so[key]) <= TOL_ACT, (k, key)
            assert_increments_close(prior[key], sg[key], so[key], f"readout {key}, batch {k}",
                                    decay(rc), resolved=0.0 if key != "pij" else 0.5)
        assert_weights_close(sg["w"], so["w"], f"readout w, batch {k}")
        assert_weights_close(sg["b"], so["b"], f"readout b, batch {k}")

    # held-out inference: activities, readout support, classes
    xt = dev(Xt)
    yg = torch.empty((len(Xt), net.hidden.n_out), device="cuda", dtype=torch.float32)
    sg = torch.empty((len(Xt), w.readout_mcu), device="cuda", dtype=torch.float32)
    ysink = torch.empty_like(sg)
    for k in range(0, len(Xt), B):
        n = min(B, len(Xt) - k)
        net.hidden.forward(xt[k:k + n], yg[k:k + n])
        net.readout.forward(yg[k:k + n], ysink[k:k + n], sg[k:k + n])
    pred = net.predict(xt).cpu().numpy()
    yg, sg = yg.cpu().numpy(), sg.cpu().numpy()
    ho = oracle.OracleLayer(oracle.make_params(L.in_hcu, L.in_mcu, L.out_hcu, L.out_mcu,
                                               gain=w.gain, bias_gain=w.bias_gain))
    ho.set_state(net.hidden.get_state())
    ro.set_state(net.readout.get_state())
    _, yo = ho.forward(Xt)
    assert max_abs(yg, yo) <= TOL_ACT, max_abs(yg, yo)
    assert_support_close(sg, oracle.support(ro.p, yg, ro.w, ro.b))
    s = oracle.support(ro.p, yo, ro.w, ro.b)
    ora = oracle.readout(ro.p, s)[:, 0]
    top2 = np.sort(s, axis=1)[:, -2:]
    clear = (top2[:, 1] - top2[:, 0]) > 1e-5 * np.maximum(1.0, np.abs(top2[:, 1]))
    assert clear.mean() > 0.95
    assert np.array_equal(pred[clear], ora[clear]), int(np.sum(pred[clear] != ora[clear]))
    print(f"held-out: {int(clear.sum())} of {len(pred)} clear of ties, agreement on them 1.0, "
          f"{len(np.unique(pred))} classes predicted, accuracy "
          f"{float(np.mean(pred == tlabels)):.3f} after {n_hidden} hidden and {n_read} readout "
          f"batches (reported, not asserted)")
    net.close()
