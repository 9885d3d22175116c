"""Checkpoint and resume of the error-feedback state.

The state a worker carries from one iteration to the next is its error
vector e (Algorithm 1 sets e_0 = 0 and carries e_{t+1} = p - Delta); the
gradients are regenerated from (workload, worker, t).  An EF trajectory
saved to disk after step s and resumed in a fresh state object (new
buffers, a new Top-k workspace with no recorded threshold, a new counter)
must produce the same payloads and the same final e, bit for bit, as the
trajectory that ran without interruption.
"""
import os

import numpy as np
import pytest

import oracle
from paper_2108_00951_amd import synth
from tests._checks import assert_bits_equal, canonical

LR = synth.LR
D, K, T, STOP = 200_003, 900, 8, 3


def _gradient(t):
    return synth.small_gradient(800 + t, D)


def _oracle_run(lam, t0, t1, e_ht, e_tk, out):
    for t in range(t0, t1):
        g = _gradient(t)
        ri, rv, e_ht, _ = oracle.ht(g, e_ht, LR, lam)
        ti, tv, e_tk = oracle.topk(g, e_tk, LR, K)
        out.append((ri, rv, ti, tv))
    return e_ht, e_tk


def test_oracle_trajectory_resumes_bit_identically(tmp_path):
    lam = oracle.calibrate_lambda(_gradient(0), 0.01)
    z = np.zeros(D, np.float32)
    whole = []
    e_ht, e_tk = _oracle_run(lam, 0, T, z, z, whole)
    part = []
    a_ht, a_tk = _oracle_run(lam, 0, STOP, z, z, part)
    np.save(os.path.join(tmp_path, "ht.npy"), a_ht, allow_pickle=False)
    np.save(os.path.join(tmp_path, "tk.npy"), a_tk, allow_pickle=False)
    del a_ht, a_tk
    b_ht = np.load(os.path.join(tmp_path, "ht.npy"), allow_pickle=False)
    b_tk = np.load(os.path.join(tmp_path, "tk.npy"), allow_pickle=False)
    b_ht, b_tk = _oracle_run(lam, STOP, T, b_ht, b_tk, part)
    assert_bits_equal(b_ht, e_ht, "hard-threshold e after resume")
    assert_bits_equal(b_tk, e_tk, "Top-k e after resume")
    for t, (x, y) in enumerate(zip(whole, part)):
        for a, b in zip(x, y):
            np.testing.assert_array_equal(a.view(np.uint32), b.view(np.uint32), err_msg="t=%d" % t)


@pytest.mark.gpu
def test_device_trajectory_resumes_bit_identically(tmp_path):
    torch = pytest.importorskip("torch")
    from paper_2108_00951_amd import binding as efs

    lam = oracle.calibrate_lambda(_gradient(0), 0.01)

    class State:
        def __init__(self):
            self.e_ht = torch.zeros(D, device="cuda")
            self.e_tk = torch.zeros(D, device="cuda")
            self.idx = torch.empty(D, dtype=torch.int32, device="cuda")
            self.val = torch.empty(D, device="cuda")
            self.ctr = efs.new_counter("cuda")
            self.tidx = torch.empty(K, dtype=torch.int32, device="cuda")
            self.tval = torch.empty(K, device="cuda")
            self.ws = efs.new_topk_workspace(D, K, "cuda")
            self.ws.zero_()

        def run(self, t0, t1, out):
            for t in range(t0, t1):
                g = torch.from_numpy(_gradient(t)).to("cuda")
                efs.ht_compress(g, self.e_ht, LR, lam, self.idx, self.val, self.ctr)
                efs.topk_compress(g, self.e_tk, LR, K, self.tidx, self.tval, self.ws)
                n = efs.counter_value(self.ctr)
                out.append((canonical(self.idx[:n].cpu().numpy(), self.val[:n].cpu().numpy()),
                            canonical(self.tidx.cpu().numpy(), self.tval.cpu().numpy()),
                            efs.topk_took_bracket_path(self.ws)))

    whole = []
    a = State()
    a.run(0, T, whole)
    part = []
    b = State()
    b.run(0, STOP, part)
    np.save(os.path.join(tmp_path, "ht.npy"), b.e_ht.cpu().numpy(), allow_pickle=False)
    np.save(os.path.join(tmp_path, "tk.npy"), b.e_tk.cpu().numpy(), allow_pickle=False)
    del b
    c = State()   # fresh buffers, workspace and counter: no threshold recorded
    c.e_ht.copy_(torch.from_numpy(np.load(os.path.join(tmp_path, "ht.npy"), allow_pickle=False)))
    c.e_tk.copy_(torch.from_numpy(np.load(os.path.join(tmp_path, "tk.npy"), allow_pickle=False)))
    c.run(STOP, T, part)
    assert_bits_equal(c.e_ht.cpu().numpy(), a.e_ht.cpu().numpy(), "hard-threshold e after resume")
    assert_bits_equal(c.e_tk.cpu().numpy(), a.e_tk.cpu().numpy(), "Top-k e after resume")
    for t, (x, y) in enumerate(zip(whole, part)):
        for (xi, xv), (yi, yv) in zip(x[:2], y[:2]):
            np.testing.assert_array_equal(xi, yi, err_msg="t=%d" % t)
            np.testing.assert_array_equal(xv.view(np.uint32), yv.view(np.uint32), err_msg="t=%d" % t)
    # the resumed run's first Top-k call had no recorded threshold (radix
    # path) where the uninterrupted run could select from its bracket
    assert not part[STOP][2]
    # and the device trajectory is the oracle's
    z = np.zeros(D, np.float32)
    ref = []
    _oracle_run(lam, 0, T, z, z, ref)
    for t, (x, r) in enumerate(zip(whole, ref)):
        np.testing.assert_array_equal(x[0][0], r[0], err_msg="ht t=%d" % t)
        np.testing.assert_array_equal(x[0][1].view(np.uint32), r[1].view(np.uint32))
        np.testing.assert_array_equal(x[1][0], r[2], err_msg="topk t=%d" % t)
        np.testing.assert_array_equal(x[1][1].view(np.uint32), r[3].view(np.uint32))
