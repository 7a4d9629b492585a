"""Helpers that run the HIP path (through the C ABI binding) and the CPU oracle side by
side on the same seeded inputs and compare them element by element.

Bar: winner, second, d1, d2, acceptance, edge lists, positions and errors all bit-exact:
both sides evaluate the same binary32 expressions in the same order (no contraction), so
no tolerance is needed.  The looser bar of positions within 1e-6 after a run is implied
and reported separately by ``max_position_error``.
"""
from __future__ import annotations

import os

import numpy as np

import oracle

POS_TOL = 1e-6


def oracle_threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def params_pair(n_max, e_max, m_max, eps_b=0.05, eps_n=0.0006, max_age=50, err_alpha=0.5,
                err_beta=0.995, lock_mode=0, key_mode=0):
    from paper_1503_08294_amd import gsn
    g = gsn.make_params(eps_b, eps_n, max_age, err_alpha, err_beta, n_max, e_max, m_max,
                        lock_mode, key_mode)
    o = oracle.Params(eps_b, eps_n, max_age, err_alpha, err_beta, n_max, e_max, m_max,
                      lock_mode=lock_mode, key_mode=key_mode)
    return g, o


class Pair:
    """A GPU network and an oracle network created from the same units and parameters."""

    def __init__(self, units: np.ndarray, n_max=None, e_max=None, m_max=1024, **kw):
        import torch
        from paper_1503_08294_amd import gsn
        n = units.shape[1]
        n_max = n_max or n
        e_max = e_max if e_max is not None else 4 * n_max + 16
        gp, op = params_pair(n_max, e_max, m_max, **kw)
        self.torch = torch
        self.gsn = gsn
        self.net = gsn.Network(gp, torch.from_numpy(np.ascontiguousarray(units)).cuda())
        self.orc = oracle.Oracle(op, units, threads=oracle_threads())

    def to_dev(self, a: np.ndarray):
        return self.torch.from_numpy(np.ascontiguousarray(a)).cuda()

    def find(self, sig: np.ndarray):
        g = [t.cpu().numpy() for t in self.net.find_winners(self.to_dev(sig))]
        o = self.orc.find_winners(sig)
        return g, o

    def iterate(self, sig: np.ndarray, it=0, insert_every=0, grow=False, calls="fused"):
        """One iteration on both sides; calls="fused" runs gsn_iterate, calls="steps" the
        four separate calls (find, resolve, adapt, update_edges)."""
        run = self.net.iterate if calls == "fused" else self.net.iterate_steps
        g = [t.cpu().numpy() for t in run(self.to_dev(sig))]
        if grow:
            self.net.grow(it, insert_every)
        o = self.orc.iterate(sig, it, insert_every, grow)
        return g, o

    def compare_state(self, where=""):
        gs = self.net.export()
        os_ = self.orc.export()
        assert self.net.sizes() == tuple(int(v) for v in self.orc.sizes()), where
        np.testing.assert_array_equal(gs["edges"].numpy(), os_["edges"], err_msg=where)
        np.testing.assert_array_equal(gs["xyz"].numpy(), os_["xyz"], err_msg=where)
        np.testing.assert_array_equal(gs["err"].numpy(), os_["err"], err_msg=where)
        return gs, os_

    def max_position_error(self) -> float:
        """Largest absolute position difference between the two sides."""
        gx = self.net.export()["xyz"].numpy().astype(np.float64)
        ox = self.orc.export()["xyz"].astype(np.float64)
        return float(np.abs(gx - ox).max()) if gx.size else 0.0


def assert_find_equal(g, o, where=""):
    names = ("winner", "second", "d1", "d2")
    for a, b, nm in zip(g, o, names):
        np.testing.assert_array_equal(a, b, err_msg=f"{where} {nm}")


def assert_iter_equal(g, o, where=""):
    names = ("winner", "second", "d1", "d2", "accepted")
    for a, b, nm in zip(g, o, names):
        np.testing.assert_array_equal(a, b, err_msg=f"{where} {nm}")


def run_workload(name, iterations=None, compare_every=1, n_points=None, m=None,
                 n_units=None, calls="fused", **over):
    from paper_1503_08294_amd.clouds import WORKLOADS, SignalStream
    wl = WORKLOADS[name]
    cloud = wl.make_cloud(n_points)
    units = wl.make_units(cloud, n_units)
    m = m or wl.m
    its = iterations or wl.iterations
    cap = wl.capacity(m)
    kw = dict(eps_b=wl.eps_b, eps_n=wl.eps_n, max_age=wl.max_age, err_alpha=wl.err_alpha,
              err_beta=wl.err_beta)
    kw.update(over)
    pair = Pair(units, n_max=max(cap["n_max"], units.shape[1]), e_max=cap["e_max"], m_max=m,
                **kw)
    stream = SignalStream(cloud, wl.signal_seed)
    rejected = 0
    for t in range(1, its + 1):
        sig = stream.next(m)
        g, o = pair.iterate(sig, t, wl.insert_every, wl.grow, calls)
        assert_iter_equal(g, o, f"{name} iteration {t}")
        rejected += int(m - o[4].sum())
        if t % compare_every == 0 or t == its:
            pair.compare_state(f"{name} iteration {t}")
    assert pair.net.check() == 0
    assert pair.max_position_error() <= POS_TOL
    return pair, rejected / (its * m)
