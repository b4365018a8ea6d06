"""A whole multi-layer step recorded into a HIP graph: every replay equals
the eager step bit for bit, with eager work and synchronisations between
the replays (dense fp32 and bf16 stacks, the low-rank stack, the linear
recurrence)."""

import numpy as np
import pytest
import torch

from helpers import dev, layer_to_dev
from paper_1709_02755_amd import sru
from paper_1709_02755_amd.workloads import WORKLOADS, make_inputs, scaled

pytestmark = pytest.mark.gpu


def _outputs(st):
    out = {}
    for li, o in enumerate(st.fw):
        for k in ("H", "C"):
            if o.get(k) is not None:
                out[f"{k}{li}"] = o[k].clone()
    for li, b in enumerate(st.bw):
        for k, v in b.items():
            if v is not None:
                out[f"{k}{li}"] = v.clone()
    return out


@pytest.mark.parametrize("wi", [1, 3, 6, 7])
def test_graph_replay_equals_eager(wi):
    w = WORKLOADS[wi]
    if w.L * w.B * w.d > 1 << 22:
        w = scaled(w, L=48, B=12, d=256)
    print(f"graph replay {w.name}", flush=True)
    inp = make_inputs(w)
    layers = [layer_to_dev(p) for p in inp["layers"]]
    st = sru.Stack(layers, w.L, w.B, w.d_in, w.d, w.direction, w.gemm_dtype, "cuda",
                   backward=w.backward, linear=w.linear)
    X, dH, mask = dev(inp["X"]), dev(inp["dH"]), dev(inp["mask"])
    st.step(X, dH, mask)
    torch.cuda.synchronize()
    eager = _outputs(st)
    graph = st.capture(X, dH, mask)
    rng = np.random.default_rng(1)
    for rep in range(3):
        # eager work on other inputs between replays overwrites every buffer
        X2 = dev(rng.standard_normal(tuple(X.shape)).astype(np.float32))
        st.step(X2, dH, mask)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = _outputs(st)
        for k, v in eager.items():
            assert torch.equal(got[k], v), (rep, k)


def test_graph_replay_reads_updated_inputs():
    """A replay runs on the inputs' current contents: updating X in place and
    replaying equals an eager step on the new X."""
    w = scaled(WORKLOADS[3], L=32, B=8, d=128)
    inp = make_inputs(w)
    layers = [layer_to_dev(p) for p in inp["layers"]]
    st = sru.Stack(layers, w.L, w.B, w.d_in, w.d, w.direction, w.gemm_dtype, "cuda")
    X, dH = dev(inp["X"]), dev(inp["dH"])
    graph = st.capture(X, dH)
    X_new = dev(np.random.default_rng(2).standard_normal(tuple(X.shape)).astype(np.float32))
    st.step(X_new, dH)
    torch.cuda.synchronize()
    want = _outputs(st)
    X.copy_(X_new)
    graph.replay()
    torch.cuda.synchronize()
    got = _outputs(st)
    for k, v in want.items():
        assert torch.equal(got[k], v), k
