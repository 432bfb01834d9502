"""vqc_train_step captured into a HIP graph (through torch.cuda.graph) and
replayed: the streaming step forks to the library's side stream and joins back
with events, which the capture turns into graph dependencies; the resident
step is one launch.  Every replay, with the program's own eager work and
synchronizations between replays, reproduces the eager step bit for bit
(outputs are cleared before each replay)."""
import numpy as np
import pytest

from paper_2607_11985_amd import workloads as W
from tests.parity_util import note
from tests.test_gpu_parity import torch_mod  # noqa: F401

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("idx,B", [(5, 4), (4, 6), (2, 16)])
def test_train_step_graph_replays(torch_mod, idx, B):
    torch = torch_mod
    from paper_2607_11985_amd import _lib
    from paper_2607_11985_amd.api import Circuit
    w = W.make_config(idx, batch=B)
    n = w.n_qubits
    dev = torch.device("cuda", 0)
    c = Circuit(w.ops, n, w.n_params, w.n_inputs)
    note(f"{w.name} B={B}: graph capture and replays of the training step "
         f"(path {c.info()['path']})")
    p = torch.from_numpy(w.params).to(dev)
    x = torch.from_numpy(w.inputs).to(dev)
    y = torch.from_numpy(w.y).to(dev) if w.y is not None else None
    outs = [torch.zeros((B, n), device=dev), torch.zeros((B, n), device=dev),
            torch.zeros((B, w.n_params), device=dev), torch.zeros((B, w.n_inputs), device=dev)]
    nb = c.workspace_bytes(B, 2)
    ws = torch.empty(max(nb, 1), dtype=torch.uint8, device=dev)

    def step(stream):  # raises on a library error
        _lib.vqc_train_step(c.handle, B, p.data_ptr(), x.data_ptr(), _lib.LOSS[w.loss],
                            y.data_ptr() if y is not None else None, outs[0].data_ptr(),
                            outs[1].data_ptr(), outs[2].data_ptr(), outs[3].data_ptr(),
                            ws.data_ptr() if nb else None, nb, stream)

    side = torch.cuda.Stream(dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        for _ in range(2):  # warm up (creates the library's side stream)
            step(side.cuda_stream)
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize()
    ref = [t.cpu().numpy().copy() for t in outs]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(torch.cuda.current_stream(dev).cuda_stream)
    torch.cuda.synchronize()
    scratch = torch.zeros(1 << 20, device=dev)
    for r in range(3):
        for t in outs:
            t.zero_()
        scratch.add_(1.0)  # the program's own work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, a, b in zip(("E", "g", "dparams", "dinputs"), (t.cpu().numpy() for t in outs),
                              ref):
            assert np.array_equal(a, b), f"replay {r}: {name} differs from the eager step"
    del g
