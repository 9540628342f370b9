"""GPU parity of the session predictor (Sec. 3.3) through the C ABI against
the fp64 oracle: the first layer's output (its k slices summed) element by
element and the logits
within 1e-5 (1 + |y|) (fp32 evaluation in blocked and in sequential order
stays within a tenth of it, while a dropped term exceeds it tenfold: both
pinned in tests/test_oracle_predictor.py); predictions
equal wherever the logit is farther than that from 0.  Sizes: the full
d = 4,096 of the workload, a ragged batch, the smallest and largest d, one
row."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from harness import say  # noqa: E402
from oracle import predictor as P  # noqa: E402
from paper_2605_18825_amd import api  # noqa: E402
from synth import predictor as S  # noqa: E402

TOL = 1e-5


def dev(a, dt):
    return torch.as_tensor(np.ascontiguousarray(a)).to(device="cuda", dtype=dt)


def run(n, d, seed):
    h = S.hidden_states(n, d, seed)
    w = S.weights(d, seed + 1)
    wd = dict(w1=dev(w["w1"].view(np.int16), torch.int16), b1=dev(w["b1"], torch.float32),
              w2=dev(w["w2"], torch.float32), b2=dev(w["b2"], torch.float32), w3=dev(w["w3"], torch.float32),
              b3=dev(w["b3"], torch.float32))
    work = torch.full((4, max(n, 1), 256), float("nan"), dtype=torch.float32, device="cuda")
    logit = torch.full((max(n, 1),), float("nan"), dtype=torch.float32, device="cuda")
    pred = torch.full((max(n, 1),), 7, dtype=torch.uint8, device="cuda")
    say("predictor n %d d %d" % (n, d))
    api.sae_predict_sessions(dev(h.view(np.int16), torch.int16).reshape(n, d), wd, work, logit, pred)
    torch.cuda.synchronize()
    y, h1, _ = P.forward(h, w["w1"], w["b1"], w["w2"], w["b2"], w["w3"], w["b3"])
    eb = P.error_bound(h, w["w1"], w["b1"], w["w2"], w["b2"], w["w3"], w["b3"])
    part = work.cpu().numpy()[:, :n].astype(np.float64).sum(axis=0) + w["b1"]
    return y, h1, eb, np.maximum(part, 0), logit.cpu().numpy()[:n], pred.cpu().numpy()[:n]


@pytest.mark.parametrize("n,d", [(4096, 4096), (1000, 4096), (77, 256), (1, 512), (130, 1024), (300, 16384)])
def test_predictor_matches_oracle(n, d):
    y, h1, eb, g1, gy, gp = run(n, d, 900 + n + d)
    assert np.all(np.isfinite(g1)) and np.all(np.isfinite(gy))
    assert np.all(np.abs(g1 - h1) <= TOL * (1 + np.abs(h1))), np.max(np.abs(g1 - h1))
    tol = TOL * (1 + np.abs(y))
    err = np.abs(gy.astype(np.float64) - y)
    assert np.all(err <= tol), (float(err.max()), int(np.argmax(err / tol)))
    assert np.all(err <= eb)
    sure = np.abs(y) > tol
    assert np.array_equal(gp[sure], (y[sure] > 0).astype(np.uint8))
    assert set(np.unique(gp).tolist()) <= {0, 1}
    say("predictor n %d d %d: max |dy| %.3g, max |dh1| / (1 + |h1|) %.3g, %.1f %% predicted to continue"
        % (n, d, err.max(), float(np.max(np.abs(g1 - h1) / (1 + np.abs(h1)))), 100 * gp.mean()))


def test_predictor_argument_checks():
    w = {k: torch.zeros(8, dtype=torch.float32, device="cuda") for k in ("b1", "w2", "b2", "w3", "b3")}
    w["w1"] = torch.zeros((256, 64), dtype=torch.int16, device="cuda")
    h = torch.zeros((4, 320), dtype=torch.int16, device="cuda")
    out = torch.zeros(4, dtype=torch.float32, device="cuda")
    with pytest.raises(api.SaeError, match="multiple of 256"):
        api.sae_predict_sessions(h, w, out, out)
    h = torch.zeros((0, 256), dtype=torch.int16, device="cuda")
    api.sae_predict_sessions(h, w, out, out)  # n = 0: nothing to do
