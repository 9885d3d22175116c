"""The calls are enqueued on the caller's stream: a side stream made current
with torch.cuda.stream(), or one passed explicitly while another is current.
Results after synchronising that stream match the oracle."""
import numpy as np
import pytest

from paper_2108_00951_amd import synth
from tests._checks import assert_bits_equal, assert_payload_equal

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import oracle  # noqa: E402
from paper_2108_00951_amd import binding as efs  # noqa: E402

DEV = "cuda"
LR = synth.LR


def _step(d, k, lam, g, stream=None):
    gd = torch.from_numpy(g).to(DEV)
    e_ht = torch.zeros(d, device=DEV)
    e_tk = torch.zeros(d, device=DEV)
    idx = torch.empty(d, dtype=torch.int32, device=DEV)
    val = torch.empty(d, device=DEV)
    ctr = efs.new_counter(DEV)
    ti = torch.empty(k, dtype=torch.int32, device=DEV)
    tv = torch.empty(k, device=DEV)
    ws = efs.new_topk_workspace(d, k, DEV)
    out = torch.empty(d, device=DEV)
    aws = efs.new_apply_workspace([(idx, val, ctr)], d, DEV)
    if stream is not None:
        torch.cuda.synchronize()  # the inputs above are ready before the side stream runs
    efs.ht_compress(gd, e_ht, LR, lam, idx, val, ctr, stream=stream)
    efs.topk_compress(gd, e_tk, LR, k, ti, tv, ws, stream=stream)
    efs.sparse_accumulate([(idx, val, ctr)], d, out, aws, stream=stream)
    return e_ht, e_tk, idx, val, ctr, ti, tv, out


def _check(d, k, lam, g, res, sync):
    sync()
    e_ht, e_tk, idx, val, ctr, ti, tv, out = res
    n = efs.counter_value(ctr)
    ri, rv, re, rk = oracle.ht(g, np.zeros(d, np.float32), LR, lam)
    assert n == rk
    assert_payload_equal(idx[:n].cpu().numpy(), val[:n].cpu().numpy(), ri, rv, "ht")
    assert_bits_equal(e_ht.cpu().numpy(), re, "ht e'")
    ti_r, tv_r, te = oracle.topk(g, np.zeros(d, np.float32), LR, k)
    assert_payload_equal(ti.cpu().numpy(), tv.cpu().numpy(), ti_r, tv_r, "topk")
    assert_bits_equal(e_tk.cpu().numpy(), te, "topk e'")
    assert_bits_equal(out.cpu().numpy(), oracle.accumulate([(ri, rv)], d), "average")


def test_calls_run_on_the_current_side_stream():
    d, k = 300_007, 3000
    g = synth.small_gradient(41, d)
    lam = oracle.calibrate_lambda(g, 0.01)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        res = _step(d, k, lam, g)
    _check(d, k, lam, g, res, s.synchronize)


def test_calls_run_on_an_explicit_stream():
    d, k = 300_007, 3000
    g = synth.small_gradient(42, d)
    lam = oracle.calibrate_lambda(g, 0.01)
    s = torch.cuda.Stream()
    res = _step(d, k, lam, g, stream=s)
    _check(d, k, lam, g, res, s.synchronize)
