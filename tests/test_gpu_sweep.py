"""The deferred sweep over silent elements.

The library updates the Pij elements of active blocks every batch, and those of silent blocks
(which the support never reads) for several consecutive batches in one sweep on a second
stream, each batch's update applied in order with the same rounding.  Grouping must therefore
be invisible: the state after a run is bitwise the same whether the sweeps cover eight batches
or one (reading the state applies the pending ones), and a multi-batch run without
re-synchronisation agrees with the oracle's per-batch updates.
"""
import numpy as np
import pytest

from paper_2106_05373_amd import synth

from pairs import (TOL_ACT, TOL_ACT_LOWP, TOL_INC_ULPS, Pair, decay, assert_increments_close,
                   assert_state_close, assert_storage_close, assert_weights_close,
                   assert_weights_storage_close, bcpnn, element_mask, max_abs, workload_config,
                   workload_mask)

pytestmark = pytest.mark.gpu

MNIST = synth.WORKLOADS["mnist"]
# 20 batches of mixed sizes (a 17-row batch has a partial 16-row k-step, a 1-row batch a single
# row): run freely, sweeps of 8 and 8 with the rest applied before a structural update or a read
SIZES = [128, 128, 64, 128, 128, 128, 96, 128, 128, 17, 128, 128, 1, 128, 64, 128, 128, 96, 128, 128]
STRUCTURAL_AT = 11


@pytest.fixture(autouse=True)
def _announce(request):
    print(f"\n[gpu case] {request.node.nodeid}", flush=True)
    yield


def _inputs():
    px, _ = synth.dataset(MNIST, n=sum(SIZES))
    X = synth.encode_pixels(px)
    out, k = [], 0
    for b in SIZES:
        out.append(X[k:k + b])
        k += b
    return out


@pytest.mark.parametrize("pairs", [1, 0])
def test_sweep_grouping_is_bitwise_invisible(pairs):
    """The same batches, with a structural update before the twelfth, run freely and with the
    state read after every batch: bitwise identical states."""
    import torch
    xs = [torch.from_numpy(np.ascontiguousarray(x)).cuda() for x in _inputs()]
    states = []
    for read_each in (False, True):
        layer = bcpnn().Layer(workload_config(MNIST, alpha=0.02, complement_pairs=pairs),
                              workload_mask(MNIST))
        for k, x in enumerate(xs):
            if k == STRUCTURAL_AT:
                layer.structural_update(count=False)
            layer.train_batch(x)
            if read_each:
                layer.get_state(("pij",))
        states.append(layer.get_state())
        layer.close()
    for key in states[0]:
        assert np.array_equal(states[0][key].view(np.uint8), states[1][key].view(np.uint8)), key


def test_profile_holds_more_launches_than_one_slot_chunk():
    """More timed launches between two reads than one device allocation of stamp slots holds
    (256): the library adds slots as it goes, and the read returns every launch, each of a
    plausible duration, and leaves none behind."""
    import torch
    xs = [torch.from_numpy(np.ascontiguousarray(x)).cuda() for x in _inputs()[:4]]
    lay = bcpnn().Layer(workload_config(MNIST), workload_mask(MNIST))
    lay.profile_enable(1)
    n = 300
    for k in range(n):
        lay.train_batch(xs[k % len(xs)])
    for kernel in ("support", "active"):
        ms, m = lay.profile_read_kernel(kernel)
        assert m == n, (kernel, m)
        assert 1e-3 < ms / n < 5.0, (kernel, ms)
        assert lay.profile_read_kernel(kernel) == (0.0, 0)
    lay.profile_enable(0)
    lay.close()


@pytest.mark.parametrize("shape,pairs,storage", [("mnist", 1, "f32"), ("mnist", 0, "bf16"),
                                                  ("large", 1, "f32"), ("large", 0, "f32")])
def test_timed_launches_compute_the_same_bits(shape, pairs, storage):
    """The launches that time themselves (the support and active-block kernels with their
    clock stamps, which the profiling pass of the benchmark runs) compute what the untimed ones
    do: the same batches, a structural update among them, with profiling off and with every
    launch timed, give bitwise identical activities and states.  The large layer's support
    takes several chunks of active rows (its lean variant)."""
    import torch
    from pairs import gpu_config
    if shape == "mnist":
        cfg = workload_config(MNIST, alpha=0.02, complement_pairs=pairs, storage=storage)
        mask = workload_mask(MNIST)
        xs = _inputs()[:12]
    else:
        in_hcu, out_hcu, out_mcu = 4100, 21, 100
        cfg = gpu_config(in_hcu, 2, out_hcu, out_mcu, 64, alpha=0.05, complement_pairs=pairs,
                         storage=storage)
        mask = np.stack([synth.random_mask(in_hcu, 1, 104, 70 + c)[:, 0]
                         for c in range(out_hcu)], 1)
        rng = np.random.default_rng(5)
        xs = [synth.encode_pixels(rng.random((B, in_hcu)).astype(np.float32))
              for B in (64, 40, 64, 23, 64, 1, 64, 64, 50, 64, 17, 64)]
    xs = [torch.from_numpy(np.ascontiguousarray(x)).cuda() for x in xs]
    runs = []
    for period in (0, 1):
        layer = bcpnn().Layer(cfg, mask)
        layer.profile_enable(period)
        ys = []
        for k, x in enumerate(xs):
            if k == 7:
                layer.structural_update(count=False)
            y = torch.empty((x.shape[0], layer.n_out), dtype=torch.float32, device="cuda")
            layer.train_batch(x, y=y)
            ys.append(y)
        state = layer.get_state()
        if period:
            assert layer.profile_read_kernel("support")[1] == len(xs)
            assert layer.profile_read_kernel("active")[1] == len(xs)
        layer.profile_enable(0)
        layer.close()
        runs.append(([y.cpu().numpy() for y in ys], state))
    (y0, s0), (y1, s1) = runs
    for k, (a, b) in enumerate(zip(y0, y1)):
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), f"activities of batch {k}"
    for key in s0:
        assert np.array_equal(s0[key].view(np.uint8), s1[key].view(np.uint8)), key


class Moved:
    """Sum over the steps of a run of the oracle's per-step contraction term |P_new - c1 P_old|
    of each trace (what the contraction error of each step is relative to)."""

    def __init__(self, ora, c1):
        self.ora, self.c1 = ora, c1
        self.sum = {k: np.zeros(getattr(ora, k).shape, np.float64) for k in ("pi", "pj", "pij")}
        self.peak = np.abs(ora.pij.astype(np.float64))      # largest |Pij| along the run

    def before(self):
        self.prev = {k: getattr(self.ora, k).astype(np.float64) for k in self.sum}

    def after(self):
        for k in self.sum:
            self.sum[k] += np.abs(getattr(self.ora, k).astype(np.float64) - self.c1 * self.prev[k])
        np.maximum(self.peak, np.abs(self.ora.pij), out=self.peak)


def check_run(prior, sg, so, cfg, storage, where, n_batches, moved):
    """End state of a run of n_batches from a common prior state.  Pi, Pj (fp32 in every
    format) and, with fp32 storage, Pij (silent and active blocks apart): the change over the
    run to the increment bound, its relative part taken on the sum of the oracle's per-step
    contraction terms (with complement pairs, of the pair's two rows together) and its ulp
    allowance that of one step per batch (the roundings of each step add up).  Reduced storage:
    Pij within two storage ulps of the largest value the element reached (a one-ulp difference
    left where a step's result sits at a rounding midpoint persists, decaying with c1, while
    the value may fall into a smaller binade, where rounding can add up to one more of that
    binade's ulps per crossing), and w against the oracle's weights from the GPU's own traces
    (within one storage ulp and the fp32 weight tolerance)."""
    import oracle
    from pairs import oracle_params, pair_total
    ulps = TOL_INC_ULPS * n_batches
    assert np.array_equal(sg["mask"], so["mask"]), f"{where} mask differs"
    for k in ("pi", "pj"):
        assert_increments_close(prior[k], sg[k], so[k], f"{where} {k}", moved.c1, ulps=ulps,
                                resolved=0.0, contraction=moved.sum[k])
    act = element_mask(prior["mask"], cfg.in_mcu, cfg.out_mcu)
    if storage == "f32":
        ct = pair_total(moved.sum["pij"]) if cfg.complement_pairs else moved.sum["pij"]
        for name, sel in (("silent", ~act), ("active", act)):
            assert_increments_close(prior["pij"], sg["pij"], so["pij"], f"{where} pij {name}",
                                    moved.c1, ulps=ulps, select=sel, contraction=ct)
        assert_weights_close(sg["w"], so["w"], f"{where} w")
        assert_weights_close(sg["b"], so["b"], f"{where} b")
    else:
        assert_storage_close(sg["pij"], so["pij"], storage, f"{where} pij", ulps=2,
                             scale=moved.peak)
        w_o, b_o = oracle.update_weights(oracle_params(cfg), sg["mask"], sg["pi"], sg["pj"],
                                         sg["pij"])
        assert_weights_storage_close(sg["w"], w_o, storage, f"{where} w from the GPU's traces")
        assert_weights_close(sg["b"], b_o, f"{where} b")


@pytest.mark.parametrize("storage", ["f32", "bf16", "m10"])
@pytest.mark.parametrize("pairs", [1, 0])
def test_multi_batch_run_matches_oracle(pairs, storage):
    """Target-clamped batches (the traces then depend on the inputs alone, with no feedback
    through the weights), no re-synchronisation: after 20 batches (two sweeps of eight, the
    rest applied by the read) the change of every trace agrees with the oracle's, silent and
    active blocks apart; a forward pass mid-run does not disturb the sweeps."""
    rng = np.random.default_rng(5)
    pair = Pair(workload_config(MNIST, alpha=0.02, complement_pairs=pairs, storage=storage),
                workload_mask(MNIST))
    cfg = pair.cfg
    t = pair.torch
    prior = pair.ora.get_state()
    moved = Moved(pair.ora, decay(cfg))
    for k, x in enumerate(_inputs()):
        win = rng.integers(0, cfg.out_mcu, size=(x.shape[0], cfg.out_hcu))
        target = np.zeros((x.shape[0], cfg.out_hcu, cfg.out_mcu), np.float32)
        np.put_along_axis(target, win[..., None], 1.0, axis=-1)
        moved.before()
        pair.train(x, target.reshape(x.shape[0], -1))
        moved.after()
        if k == 6:
            # (with reduced storage the two runs' weights are storage ulps apart by now, so only
            # the fp32 run's activities are compared; the call must not disturb the queue)
            y = t.empty((x.shape[0], pair.n_out), device="cuda", dtype=t.float32)
            pair.gpu.forward(pair.dev(x), y)
            if storage == "f32":
                _, y_o = pair.ora.forward(x)
                assert max_abs(y.cpu().numpy(), y_o) <= TOL_ACT
    sg, so = pair.gpu.get_state(), pair.ora.get_state()
    where = f"after {len(SIZES)} batches"
    if storage == "f32":
        assert_state_close(sg, so, where=where)
    check_run(prior, sg, so, cfg, storage, where, len(SIZES), moved)
    pair.close()


def test_state_calls_between_batches_see_every_update():
    """Calls that touch the traces, made while a group of silent updates is still queued:
    recompute_weights, readout and set_state in the middle of a run, and destroy right after
    batches, leave the layer as per-batch updates would.  The reference run reads the state
    after every batch; the other interleaves the calls at the same points."""
    import torch
    xs = [torch.from_numpy(np.ascontiguousarray(x)).cuda() for x in _inputs()]
    cfg = workload_config(MNIST, alpha=0.02)
    mask = workload_mask(MNIST)

    ref = bcpnn().Layer(cfg, mask)
    snap = None
    for k, x in enumerate(xs):
        ref.train_batch(x)
        if k == 2:
            snap = ref.get_state()                   # the state set_state re-applies below
        if k == 4:
            ref.recompute_weights()
    st_ref = ref.get_state()
    ref.close()

    lay = bcpnn().Layer(cfg, mask)
    win = torch.empty((xs[0].shape[0], cfg.out_hcu), device="cuda", dtype=torch.int32)
    for k, x in enumerate(xs):
        lay.train_batch(x)
        if k == 1:
            lay.readout(xs[0], win)                  # reads w, b only; the queue stays
        if k == 2:
            lay.set_state(snap)                      # applies the queue, then replaces
        if k == 4:
            lay.recompute_weights()
    st = lay.get_state()
    lay.close()
    for key in st_ref:
        assert np.array_equal(st_ref[key].view(np.uint8), st[key].view(np.uint8)), key

    # destroy with queued silent updates (waits for both streams, no leak, no fault)
    for _ in range(3):
        tmp = bcpnn().Layer(cfg, mask)
        for x in xs[:6]:
            tmp.train_batch(x)
        tmp.close()
    torch.cuda.synchronize()


@pytest.mark.parametrize("storage", ["f32", "bf16", "m10"])
@pytest.mark.parametrize("pairs", [1, 0])
def test_tiled_sweep_on_a_ragged_large_layer(pairs, storage):
    """A layer just past the size at which the library sweeps silent blocks in workgroup tiles
    (257 x 66 blocks of 32: ragged row and column tiles), ten target-clamped batches of mixed
    size (one sweep of eight, two pending), against the oracle: the change of every trace
    (silent and active blocks apart), or Pij and w within storage ulps (the tiled kernels of
    the reduced formats)."""
    from pairs import gpu_config
    in_hcu, out_hcu, out_mcu = 4100, 21, 100
    rng = np.random.default_rng(11)
    mask = np.stack([synth.random_mask(in_hcu, 1, 104, 70 + c)[:, 0] for c in range(out_hcu)], 1)
    pair = Pair(gpu_config(in_hcu, 2, out_hcu, out_mcu, 64, alpha=0.05, complement_pairs=pairs,
                           storage=storage), mask)
    prior = pair.ora.get_state()
    moved = Moved(pair.ora, decay(pair.cfg))
    sizes = (64, 64, 40, 64, 23, 64, 1, 64, 64, 50)
    for B in sizes:
        p = rng.random((B, in_hcu)).astype(np.float32)
        x = synth.encode_pixels(p)
        win = rng.integers(0, out_mcu, size=(B, out_hcu))
        target = np.zeros((B, out_hcu, out_mcu), np.float32)
        np.put_along_axis(target, win[..., None], 1.0, axis=-1)
        moved.before()
        pair.train(x, target.reshape(B, -1))
        moved.after()
    sg, so = pair.gpu.get_state(), pair.ora.get_state()
    if storage == "f32":
        assert_state_close(sg, so, where="tiled sweep")
    check_run(prior, sg, so, pair.cfg, storage, "tiled sweep", len(sizes), moved)
    pair.close()


@pytest.mark.parametrize("storage", ["f32", "bf16"])
def test_tiled_sweep_with_batches_past_sixteen_k_steps(storage):
    """The tiled sweeps of a large paired layer with batches of up to 300 rows (19 k-steps: the
    column totals past the first sixteen tiles taken one by one, chunks past sixteen k-steps),
    mixed with small ones, against the oracle as in the ragged test above."""
    from pairs import gpu_config
    in_hcu, out_hcu, out_mcu = 4100, 21, 100
    rng = np.random.default_rng(13)
    mask = np.stack([synth.random_mask(in_hcu, 1, 104, 110 + c)[:, 0] for c in range(out_hcu)], 1)
    pair = Pair(gpu_config(in_hcu, 2, out_hcu, out_mcu, 300, alpha=0.05, complement_pairs=1,
                           storage=storage), mask)
    prior = pair.ora.get_state()
    moved = Moved(pair.ora, decay(pair.cfg))
    sizes = (300, 17, 272, 300)
    for B in sizes:
        p = rng.random((B, in_hcu)).astype(np.float32)
        x = synth.encode_pixels(p)
        win = rng.integers(0, out_mcu, size=(B, out_hcu))
        target = np.zeros((B, out_hcu, out_mcu), np.float32)
        np.put_along_axis(target, win[..., None], 1.0, axis=-1)
        moved.before()
        pair.train(x, target.reshape(B, -1))
        moved.after()
    sg, so = pair.gpu.get_state(), pair.ora.get_state()
    if storage == "f32":
        assert_state_close(sg, so, where="tiled sweep, batches past 16 k-steps")
    check_run(prior, sg, so, pair.cfg, storage, "tiled sweep, batches past 16 k-steps",
              len(sizes), moved)
    pair.close()


def test_large_layer_sum_form_grouping():
    """A large layer with complement pairs and fp32 storage sweeps its silent blocks in sum
    form (the queued batches' updates regrouped as c1^n P + R): the same batches run freely
    (one sweep of eight, then two) and with the state read after every batch (ten sweeps of
    one) give bitwise the same Pi, Pj, w, b, mask and active-block Pij, and silent-block Pij
    within TOL_INC_ULPS fp32 ulps per batch of each other."""
    import torch
    from pairs import gpu_config, ulp
    in_hcu, out_hcu, out_mcu = 4100, 21, 100
    rng = np.random.default_rng(5)
    mask = np.stack([synth.random_mask(in_hcu, 1, 104, 90 + c)[:, 0] for c in range(out_hcu)], 1)
    cfg = gpu_config(in_hcu, 2, out_hcu, out_mcu, 64, alpha=0.05, complement_pairs=1)
    sizes = (64, 64, 40, 64, 23, 64, 1, 64, 64, 50)
    xs = [torch.from_numpy(synth.encode_pixels(rng.random((B, in_hcu)).astype(np.float32))).cuda()
          for B in sizes]
    states = []
    for read_each in (False, True):
        lay = bcpnn().Layer(cfg, mask)
        for x in xs:
            lay.train_batch(x)
            if read_each:
                lay.get_state(("pij",))
        states.append(lay.get_state())
        lay.close()
    a, b = states
    for key in ("pi", "pj", "w", "b", "mask"):
        assert np.array_equal(a[key].view(np.uint8), b[key].view(np.uint8)), key
    act = element_mask(a["mask"], 2, out_mcu)
    assert np.array_equal(a["pij"][act].view(np.uint32), b["pij"][act].view(np.uint32))
    silent = ~act
    d = np.abs(a["pij"][silent].astype(np.float64) - b["pij"][silent])
    scale = ulp(np.maximum(np.abs(a["pij"][silent]), np.abs(b["pij"][silent])))
    worst = float(np.max(d / scale))
    assert worst <= TOL_INC_ULPS * len(sizes), worst


def test_flush_enqueues_exactly_the_queued_sweep():
    """bcpnn_flush applies the queued silent-block updates on the caller's stream: three
    batches then a flush give one sweep launch, a second flush with nothing queued none, and the
    state equals that of a run read after every batch (grouping stays invisible)."""
    import torch
    xs = [torch.from_numpy(np.ascontiguousarray(x)).cuda() for x in _inputs()[:6]]
    cfg = workload_config(MNIST, alpha=0.02)
    lay = bcpnn().Layer(cfg, workload_mask(MNIST))
    lay.profile_enable(1)
    counts = []
    for x in xs[:3]:
        lay.train_batch(x)
    lay.flush()
    lay.flush()
    torch.cuda.synchronize()
    counts.append(lay.profile_read_kernel("sweep")[1])
    for x in xs[3:]:
        lay.train_batch(x)
        lay.flush()
    counts.append(lay.profile_read_kernel("sweep")[1])
    lay.profile_enable(0)
    st = lay.get_state()
    lay.close()
    assert counts == [1, 3], counts
    ref = bcpnn().Layer(cfg, workload_mask(MNIST))
    for x in xs:
        ref.train_batch(x)
    st_ref = ref.get_state()
    ref.close()
    for key in st_ref:
        assert np.array_equal(st_ref[key].view(np.uint8), st[key].view(np.uint8)), key


@pytest.mark.parametrize("pairs", [1, 0])
def test_inputs_that_are_not_pairs_fail_loudly(pairs):
    """With complement_pairs set, a training batch whose input units are not (x, 1 - x) pairs
    is reported by the next waiting call as BCPNN_EINPUT, and the layer refuses further work
    (BCPNN_ESTATE); true pairs pass, and a layer without the setting accepts any input."""
    import torch
    B = bcpnn()
    cfg = workload_config(MNIST, complement_pairs=pairs)
    good = torch.from_numpy(np.ascontiguousarray(_inputs()[0])).cuda()
    bad = good.clone()
    bad[5, 2 * 300 + 1] += 0.01                   # one pair of one row no longer adds up to 1
    lay = B.Layer(cfg, workload_mask(MNIST))
    lay.train_batch(good)
    lay.get_state(("pi",))
    lay.train_batch(bad)
    if pairs:
        with pytest.raises(B.BcpnnError) as ei:
            lay.get_state(("pi",))
        assert ei.value.status == -5, ei.value
        with pytest.raises(B.BcpnnError) as ei:
            lay.train_batch(good)
        assert ei.value.status == -4
    else:
        lay.get_state(("pi",))
    lay.close()


def test_profile_records_each_kernel():
    """Timing of each train_batch kernel: with period 1, nine batches give nine support and nine
    active-block launches (which stamp their own span) and one sweep (of the first eight;
    reading leaves the ninth batch queued); three more batches read three launches of the same
    order once the slots are read; the flush a second sweep; period 2 every second launch; an
    unknown kernel is rejected."""
    import torch
    xs = [torch.from_numpy(np.ascontiguousarray(x)).cuda() for x in _inputs()[:9]]
    lay = bcpnn().Layer(workload_config(MNIST), workload_mask(MNIST))
    lay.profile_enable(1)
    for x in xs:
        lay.train_batch(x)
    ms_sw, n_sw = lay.profile_read_kernel("sweep")
    ms_su, n_su = lay.profile_read_kernel("support")
    ms_ac, n_ac = lay.profile_read_kernel("active")
    assert (n_sw, n_su, n_ac) == (1, 9, 9)
    assert ms_sw > 0 and ms_su > 0 and ms_ac > 0
    # the support and active-block launches time themselves (device-clock stamps): each a
    # microsecond to a few milliseconds
    assert 1e-3 < ms_su / 9 < 5.0 and 1e-3 < ms_ac / 9 < 5.0, (ms_su, ms_ac)
    assert lay.profile_read_kernel("support") == (0.0, 0)          # reading clears
    # reading leaves the stamp slots blank again: a slot still holding an earlier start would
    # read the whole interval since then
    for x in xs[:3]:
        lay.train_batch(x)
    ms2, n2 = lay.profile_read_kernel("support")
    assert n2 == 3 and 1e-3 < ms2 / 3 < 5.0, (ms2, n2)
    assert lay.profile_read_kernel("active")[1] == 3
    lay.flush()
    assert lay.profile_read_kernel("sweep")[1] == 1                 # the ninth batch's sweep
    lay.profile_enable(2)                                           # every second launch
    for x in xs[:4]:
        lay.train_batch(x)
    assert lay.profile_read_kernel("support")[1] == 2
    assert lay.profile_read_kernel("active")[1] == 2
    B = bcpnn()
    import ctypes
    ms, n = ctypes.c_double(), ctypes.c_int32()
    st = B.lib.bcpnn_profile_read_kernel(lay._h, 7, ctypes.byref(ms), ctypes.byref(n))
    assert st == -1, st
    lay.profile_enable(0)
    lay.close()
