"""Helpers that run the GPU library and the CPU oracle side by side on identical inputs.

The GPU side goes through the C ABI (paper_2106_05373_amd.bcpnn); the oracle side through
oracle/.  Only the seeded input generators (paper_2106_05373_amd.synth) serve both.
"""
from __future__ import annotations

import numpy as np

import oracle
from paper_2106_05373_amd import synth

# Tolerances (per step, from an identical prior state).
TOL_ACT = 1e-5          # activities and traces, max-abs (fp32 storage)
TOL_ACT_LOWP = 1e-2     # traces with bf16 / 10-bit-mantissa storage
TOL_W = 1e-4            # weights and bias: |dw| <= TOL_W * max(1, |w|)
# With reduced-precision storage both sides round w to the storage format; values computed
# a few fp32 ulps apart can round to neighbouring storage values, one storage ulp apart:
# 2^-7 relative for bf16 (7 stored mantissa bits), 2^-10 for the 10-bit format.
TOL_W_STORAGE = {"f32": TOL_W, "bf16": 2.0 ** -7, "m10": 2.0 ** -10}
TOL_S_REL = 1e-6        # support: fp64 sums on both sides, rounded to fp32 (<= a few ulp)
TOL_MI_REL = 1e-12      # fp64 mutual information: summation order and libm differences
# Trace increments from a common prior state (the change a step makes, not the value, so that
# small learning rates are resolved).  A step is P <- c1 P + c2 T (c1 = 1 - alpha_eff); per
# element, |dP_gpu - dP_oracle| <= TOL_INC_REL * |c2 T| + TOL_INC_ULPS fp32 ulps of the value,
# with |c2 T| = |P_new - c1 P_old| from the oracle's states (summed over the steps of a run).
# The relative part covers the split-bf16 contraction: each product carries at most about
# 2^-16 of its value (the dropped lo*lo term and the rounding of the lo parts; all products are
# non-negative, so the sum does too), and 1e-4 is 6.5 times that.  The ulps cover the rounding
# of the stored result on both sides (half an ulp each) and the fp32 rounding of c1 (about half
# an ulp of the value).
TOL_INC_REL = 1e-4
TOL_INC_ULPS = 4
# Stored mantissa bits of the storage formats of Pij and w.
STORAGE_BITS = {"f32": 23, "bf16": 7, "m10": 10}


def bcpnn():
    """The GPU binding (imported lazily so CPU-only collection does not need the library)."""
    from paper_2106_05373_amd import bcpnn as b
    return b


def gpu_config(in_hcu, in_mcu, out_hcu, out_mcu, max_batch, **kw):
    return bcpnn().default_config(in_hcu, in_mcu, out_hcu, out_mcu, max_batch, **kw)


def oracle_params(cfg) -> oracle.Params:
    """Oracle parameters with the same values as a GPU config."""
    return oracle.Params(cfg.in_hcu, cfg.in_mcu, cfg.out_hcu, cfg.out_mcu, cfg.alpha,
                         cfg.n_cycles, cfg.gain, cfg.bias_gain, cfg.eps, cfg.pi_init,
                         cfg.pj_init, cfg.init_noise, cfg.seed, cfg.n_swaps, cfg.storage)


def workload_config(w: synth.Workload, max_batch=None, **kw):
    L = w.layer
    base = dict(alpha=w.alpha, gain=w.gain, bias_gain=w.bias_gain, init_noise=w.init_noise,
                seed=w.seed_noise, storage=w.storage,
                complement_pairs=int(w.complement_pairs))
    base.update(kw)
    return gpu_config(L.in_hcu, L.in_mcu, L.out_hcu, L.out_mcu, max_batch or w.batch, **base)


def workload_mask(w: synth.Workload) -> np.ndarray:
    L = w.layer
    if w.mask_frac >= 1.0:
        return synth.full_mask(L.in_hcu, L.out_hcu)
    return synth.random_mask(L.in_hcu, L.out_hcu, synth.active_count(L.in_hcu, w.mask_frac),
                             w.seed_mask)


class Pair:
    """A GPU layer and an oracle layer created from one configuration and mask."""

    def __init__(self, cfg, mask=None):
        import torch
        self.torch = torch
        self.cfg = cfg
        self.gpu = bcpnn().Layer(cfg, mask)
        self.ora = oracle.OracleLayer(oracle_params(cfg), mask)
        self.n_in, self.n_out = self.gpu.n_in, self.gpu.n_out

    def dev(self, a, dtype=None):
        t = self.torch
        return t.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=dtype or t.float32)

    def sync_gpu_to_oracle(self):
        """Give the GPU layer the oracle's exact state."""
        self.gpu.set_state(self.ora.get_state())

    def train(self, x, target=None):
        """One batch on both sides; returns (y_gpu, y_oracle, s_oracle)."""
        t = self.torch
        xd = self.dev(x)
        td = None if target is None else self.dev(target)
        y = t.empty((x.shape[0], self.n_out), device="cuda", dtype=t.float32)
        self.gpu.train_batch(xd, td, y)
        s_o, y_o = self.ora.train_batch(x, target)
        return y.cpu().numpy(), y_o, s_o

    def forward(self, x):
        t = self.torch
        xd = self.dev(x)
        y = t.empty((x.shape[0], self.n_out), device="cuda", dtype=t.float32)
        s = t.empty_like(y)
        self.gpu.forward(xd, y, s)
        s_o, y_o = self.ora.forward(x)
        return y.cpu().numpy(), s.cpu().numpy(), y_o, s_o

    def forward_gpu_only(self, x):
        """The GPU forward pass alone: (y, s, None, None)."""
        t = self.torch
        xd = self.dev(x)
        y = t.empty((x.shape[0], self.n_out), device="cuda", dtype=t.float32)
        s = t.empty_like(y)
        self.gpu.forward(xd, y, s)
        return y.cpu().numpy(), s.cpu().numpy(), None, None

    def close(self):
        self.gpu.close()


def max_abs(a, b):
    return float(np.max(np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64)))) if np.size(a) else 0.0


def assert_weights_close(w_gpu, w_ora, what="w", tol=TOL_W):
    w_gpu = np.asarray(w_gpu, np.float64)
    w_ora = np.asarray(w_ora, np.float64)
    err = np.abs(w_gpu - w_ora) / np.maximum(1.0, np.abs(w_ora))
    assert err.max() <= tol, f"{what}: max scaled error {err.max():.3g} > {tol}"


def assert_state_close(sg, so, tol=TOL_ACT, where="", storage="f32"):
    for k in ("pi", "pj", "pij"):
        e = max_abs(sg[k], so[k])
        assert e <= tol, f"{where} {k}: max-abs {e:.3g} > {tol}"
    assert_weights_close(sg["w"], so["w"], f"{where} w", TOL_W_STORAGE[storage])
    assert_weights_close(sg["b"], so["b"], f"{where} b")
    assert np.array_equal(sg["mask"], so["mask"]), f"{where} mask differs"


def assert_support_close(s_gpu, s_ora):
    s_gpu = np.asarray(s_gpu, np.float64)
    s_ora = np.asarray(s_ora, np.float64)
    err = np.abs(s_gpu - s_ora) / np.maximum(np.abs(s_ora), 1e-30)
    small = np.abs(s_ora) < 1e-30
    assert np.all(err[~small] <= TOL_S_REL), f"support: max rel error {err[~small].max():.3g}"
    assert np.all(np.abs(s_gpu[small]) < 1e-30)


def ulp(v, bits=23):
    """Spacing of a binary floating-point format with `bits` stored mantissa bits at |v| (fp32:
    23, bf16: 7, the 10-bit format: 10), with fp32's subnormal spacing as the floor."""
    a = np.abs(np.asarray(v, np.float64))
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -126)))
    return np.exp2(e - bits)


def element_mask(block_mask, in_mcu, out_mcu):
    """The (input HCU, hidden HCU) mask expanded to the [N_in][N_out] elements (True = active)."""
    m = np.asarray(block_mask, bool)
    return np.repeat(np.repeat(m, in_mcu, axis=0), out_mcu, axis=1)


def decay(cfg):
    """c1 = (1 - alpha)^n_cycles, the factor a step applies to the previous trace."""
    return (1.0 - float(np.float32(cfg.alpha))) ** int(cfg.n_cycles)


def assert_increments_close(prior, g, o, what, c1, ulps=TOL_INC_ULPS, select=None,
                            resolved=0.5, contraction=None):
    """The change from `prior` to the GPU's value `g` against the oracle's change to `o`:
    |dg - do| <= TOL_INC_REL * |o - c1 prior| + ulps * ulp(value) for every element (of
    `select`, a boolean mask of the elements to check).  For a run of several steps,
    `contraction` replaces |o - c1 prior| by the sum of each step's |P_new - c1 P_old| on the
    oracle side.  `resolved`: the fraction of the checked elements at which a 1% error in the
    change would exceed the bound must reach it, else the case cannot tell a wrong update from a
    right one."""
    p = np.asarray(prior, np.float64).ravel()
    gg = np.asarray(g, np.float64).ravel()
    oo = np.asarray(o, np.float64).ravel()
    ct = None if contraction is None else np.asarray(contraction, np.float64).ravel()
    if select is not None:
        sel = np.asarray(select, bool).ravel()
        p, gg, oo = p[sel], gg[sel], oo[sel]
        ct = None if ct is None else ct[sel]
    if p.size == 0:
        return
    dg, do = gg - p, oo - p
    if ct is None:
        ct = np.abs(oo - c1 * p)
    slack = ulps * ulp(np.maximum(np.abs(gg), np.abs(oo)))
    bound = TOL_INC_REL * ct + slack
    ratio = np.abs(dg - do) / bound
    k = int(np.argmax(ratio))
    frac = float(np.mean(0.01 * np.abs(do) > bound))
    print(f"{what}: {p.size} elements, worst |d err| / bound {ratio[k]:.3g} "
          f"(do {do[k]:.3g}, dg {dg[k]:.3g}), resolved at 1%: {frac:.3f}")
    assert ratio[k] <= 1.0, (f"{what}: increment error {abs(dg[k] - do[k]):.3g} exceeds "
                             f"{bound[k]:.3g} (oracle change {do[k]:.3g}, value {oo[k]:.3g})")
    assert frac >= resolved, f"{what}: only {frac:.3f} of the changes are resolved at 1%"


def pair_total(a):
    """For a [N_in][N_out] array over complementary input pairs (x, 1 - x): each row replaced by
    the sum of its pair's two rows.  With complement pairs the second row's contraction is the
    column total minus the first's, so it carries the first row's absolute error: the error of
    either row is relative to the pair's total."""
    a = np.asarray(a, np.float64)
    t = a.reshape(a.shape[0] // 2, 2, a.shape[1]).sum(axis=1)
    return np.repeat(t, 2, axis=0)


def assert_storage_close(g, o, storage, what, ulps=1, extra=0.0, scale=None):
    """Values both sides round to a reduced storage format from fp32 results that agree to a
    few fp32 ulps: at most `ulps` storage ulps apart (plus `extra` absolute), the ulp taken at
    `scale` (default: the larger of the two values)."""
    gg = np.asarray(g, np.float64)
    oo = np.asarray(o, np.float64)
    big = np.maximum(np.abs(gg), np.abs(oo))
    if scale is not None:
        big = np.maximum(big, np.asarray(scale, np.float64))
    bound = ulps * ulp(big, STORAGE_BITS[storage]) + 4 * ulp(big) + extra
    err = np.abs(gg - oo)
    k = np.unravel_index(int(np.argmax(err - bound)), err.shape) if err.size else None
    if k is not None:
        assert err[k] <= bound[k], (f"{what}: {err[k]:.3g} apart at {k} (values {gg[k]:.6g}, "
                                    f"{oo[k]:.6g}), more than {ulps} {storage} ulp")


def assert_weights_storage_close(w_gpu, w_ora, storage, what="w"):
    """Weights in a reduced storage format: the fp32 weight tolerance (the results before the
    storage rounding) plus one storage ulp (the rounding may then land on neighbours)."""
    wg = np.asarray(w_gpu, np.float64)
    wo = np.asarray(w_ora, np.float64)
    bound = TOL_W * np.maximum(1.0, np.abs(wo)) + ulp(np.maximum(np.abs(wg), np.abs(wo)),
                                                      STORAGE_BITS[storage])
    err = np.abs(wg - wo)
    assert np.all(err <= bound), f"{what}: max excess {float(np.max(err - bound)):.3g}"
