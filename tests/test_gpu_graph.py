"""The library's calls allocate nothing and issue no memset, so a whole step
(hard threshold, Top-k, average of the hard-threshold payload) can be
captured in a HIP graph and replayed.  Each replay is checked against the
same step run eagerly from the same state, with eager work (the next
gradient copied into the captured input buffer) and synchronisation between
replays."""
import numpy as np
import pytest

import oracle
from paper_2108_00951_amd import synth
from tests._checks import assert_bits_equal

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2108_00951_amd import binding as efs  # noqa: E402

DEV = "cuda"
LR = synth.LR


class Step:
    def __init__(self, d, k, lam):
        self.d, self.k, self.lam = d, k, lam
        self.g = torch.zeros(d, dtype=torch.float32, device=DEV)
        self.e_ht = torch.zeros(d, dtype=torch.float32, device=DEV)
        self.e_tk = torch.zeros(d, dtype=torch.float32, device=DEV)
        self.idx = torch.empty(d, dtype=torch.int32, device=DEV)
        self.val = torch.empty(d, dtype=torch.float32, device=DEV)
        self.ctr = efs.new_counter(DEV)
        self.tidx = torch.empty(k, dtype=torch.int32, device=DEV)
        self.tval = torch.empty(k, dtype=torch.float32, device=DEV)
        self.ws = efs.new_topk_workspace(d, k, DEV)
        self.ws.zero_()
        self.out = torch.empty(d, dtype=torch.float32, device=DEV)
        self.aws = efs.new_apply_workspace([(self.idx, self.val, self.ctr)], d, DEV)

    def run(self):
        efs.ht_compress(self.g, self.e_ht, LR, self.lam, self.idx, self.val, self.ctr)
        efs.topk_compress(self.g, self.e_tk, LR, self.k, self.tidx, self.tval, self.ws)
        efs.sparse_accumulate([(self.idx, self.val, self.ctr)], self.d, self.out, self.aws)

    def result(self):
        n = efs.counter_value(self.ctr)
        hi, hv = self.idx[:n].cpu().numpy(), self.val[:n].cpu().numpy()
        ti, tv = self.tidx.cpu().numpy(), self.tval.cpu().numpy()
        ho, to = np.argsort(hi), np.argsort(ti)
        return {"e_ht": self.e_ht.cpu().numpy(), "e_tk": self.e_tk.cpu().numpy(),
                "out": self.out.cpu().numpy(), "ht_idx": hi[ho], "ht_val": hv[ho],
                "tk_idx": ti[to], "tk_val": tv[to]}


def test_step_replays_in_a_graph():
    d, k, steps = 300_007, 3000, 6
    pool = [synth.small_gradient(700 + t, d) for t in range(steps)]
    lam = oracle.calibrate_lambda(pool[0], 0.01)

    eager = Step(d, k, lam)
    want = []
    for t in range(steps):
        eager.g.copy_(torch.from_numpy(pool[t]))
        eager.run()
        want.append(eager.result())

    graphed = Step(d, k, lam)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        graphed.run()  # recorded only
    torch.cuda.synchronize()
    for t in range(steps):
        graphed.g.copy_(torch.from_numpy(pool[t]))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = graphed.result()
        for name in ("ht_idx", "tk_idx"):
            np.testing.assert_array_equal(got[name], want[t][name], "%s replay %d" % (name, t))
        for name in ("e_ht", "e_tk", "out", "ht_val", "tk_val"):
            assert_bits_equal(got[name], want[t][name], "%s replay %d" % (name, t))


def test_layerwise_step_with_momentum_replays_in_a_graph():
    # layer-wise Top-k over 12 layers, then the momentum update of x from
    # that payload (one worker), captured together
    rng = np.random.default_rng(710)
    d, steps = 250_000, 5
    cuts = np.sort(rng.integers(0, d + 1, size=11))
    off = np.concatenate([[0], cuts, [d]]).astype(np.int64)
    ks = synth.layerwise_k(off, 0.01)
    kt = int(ks.sum())
    pool = [synth.small_gradient(720 + t, d) for t in range(steps)]
    x0 = synth.small_gradient(730, d, scale=1.0)
    beta, gamma = 0.9, 0.05

    def make():
        s = {"g": torch.zeros(d, dtype=torch.float32, device=DEV),
             "e": torch.zeros(d, dtype=torch.float32, device=DEV),
             "idx": torch.empty(kt, dtype=torch.int32, device=DEV),
             "val": torch.empty(kt, dtype=torch.float32, device=DEV),
             "ws": efs.new_topk_segmented_workspace(ks.size, kt, DEV),
             "x": torch.from_numpy(x0.copy()).to(DEV),
             "m": torch.zeros(d, dtype=torch.float32, device=DEV),
             "off": torch.from_numpy(off).to(DEV), "k": torch.from_numpy(ks).to(DEV)}
        s["ws"].zero_()
        s["aws"] = efs.new_apply_workspace([(s["idx"], s["val"])], d, DEV)
        return s

    def run(s):
        # both calls on the current stream (the capture stream when recording)
        efs.topk_segmented_compress(s["g"], s["e"], LR, s["off"], s["k"], s["idx"], s["val"],
                                    s["ws"])
        efs.sparse_apply([(s["idx"], s["val"])], d, efs.APPLY_MOMENTUM, s["x"], s["aws"],
                         m=s["m"], beta=beta, gamma=gamma)

    def result(s):
        i, v = s["idx"].cpu().numpy(), s["val"].cpu().numpy()
        o = np.argsort(i)
        return {"idx": i[o], "val": v[o], "e": s["e"].cpu().numpy(), "x": s["x"].cpu().numpy(),
                "m": s["m"].cpu().numpy()}

    eager = make()
    want = []
    for t in range(steps):
        eager["g"].copy_(torch.from_numpy(pool[t]))
        run(eager)
        want.append(result(eager))

    graphed = make()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run(graphed)  # recorded only
    torch.cuda.synchronize()
    for t in range(steps):
        graphed["g"].copy_(torch.from_numpy(pool[t]))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = result(graphed)
        np.testing.assert_array_equal(got["idx"], want[t]["idx"], "idx replay %d" % t)
        for name in ("val", "e", "x", "m"):
            assert_bits_equal(got[name], want[t][name], "%s replay %d" % (name, t))
