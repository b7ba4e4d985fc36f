"""The hand-derived examples of tests/golden/ through the library.

Each example's Gram matrix goes through the solve entry point and its task
gradients (one bucket) through the whole resolve, against the values
derived by hand from the method's definitions (Eq. mgda, Eq. pcgrad_proj
with Algorithm 1, Eq. cagrad).  The Gram matrices of these vectors are
exact in floating point (small integers), so the only error allowed is the
fp32 rounding of the weights and of the update.
"""

import json
import os

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

GOLD = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")
CASES = json.load(open(GOLD))["cases"]


def _method(case):
    return case["name"].split("_")[0].rstrip("0123456789")


def _order(case, dev):
    if "order" not in case:
        return None
    return torch.tensor(case["order"], dtype=torch.int8, device=dev)[None].contiguous()


@pytest.mark.parametrize("case", CASES, ids=[c["name"] for c in CASES])
def test_golden_solve(case):
    from paper_2606_05613_amd import bkmoo
    dev = torch.device("cuda", 0)
    g = np.array(case["g"], dtype=np.float64)
    G = torch.from_numpy((g @ g.T)[None].copy()).to(dev)
    m = _method(case)
    w, _ = bkmoo.solve(G, m, 20, case.get("c", 0.5), _order(case, dev))
    want = np.array(case["alpha"] if m == "mgda" else case["weights"])
    got = w.cpu().numpy()[0].astype(np.float64)
    assert np.all(np.abs(got - want) <= 1e-6 * np.maximum(1.0, np.abs(want))), (case["name"], got, want)


@pytest.mark.parametrize("case", CASES, ids=[c["name"] for c in CASES])
def test_golden_resolve(case):
    from paper_2606_05613_amd import bkmoo
    dev = torch.device("cuda", 0)
    g = torch.tensor(case["g"], dtype=torch.float32, device=dev)
    n = g.shape[1]
    offs = torch.tensor([0, n], dtype=torch.int64, device=dev)
    out = bkmoo.resolve(g.contiguous(), offs, _method(case), 20, case.get("c", 0.5), _order(case, dev))
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    want = np.array(case["d"])
    scale = max(1.0, float(np.abs(np.array(case["g"])).max()))
    assert np.all(np.abs(got - want) <= 1e-6 * scale), (case["name"], got, want)
