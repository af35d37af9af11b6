"""The layer's forward and backward calls captured into a HIP graph (through
torch.cuda.graph) and replayed: the calls fork onto the library's helper streams
and join back inside each call, which capture turns into graph edges.  Every
replay, with eager calls and synchronisations between the replays, must match
the eager result bitwise (the same kernels on the same buffers)."""
import pytest
import torch

from paper_2511_07343_amd import inputs, tnt

pytestmark = pytest.mark.gpu
GRADS = ("dq", "dk", "dv", "dlr", "dmom", "ddecay", "dW1", "dW2")


@pytest.mark.parametrize("w", [1, 2])
def test_captured_step_replays_bitwise(w):
    cfg = inputs.WORKLOADS[w]
    dev = torch.device("cuda:0")
    x = tnt.device_inputs(inputs.make_inputs(cfg, w), cfg, device=dev)
    u8 = lambda n: torch.empty(max(n, 16), dtype=torch.uint8, device=dev)
    o = torch.empty_like(x["q"])
    saved = u8(tnt.tnt_mem_saved_size(cfg))
    ws_f = u8(tnt.tnt_mem_workspace_size(cfg, 0))
    ws_b = u8(tnt.tnt_mem_workspace_size(cfg, 1))
    g = {k: torch.empty_like(x[s]) for k, s in (("dq", "q"), ("dk", "k"), ("dv", "v"), ("dlr", "lr"),
                                                 ("dmom", "mom"), ("ddecay", "decay"), ("dW1", "W1"),
                                                 ("dW2", "W2"))}
    st = torch.cuda.Stream(dev)

    def step():
        s1 = tnt.tnt_mem_fwd(cfg, x["q"], x["k"], x["v"], x["lr"], x["mom"], x["decay"], x["W1"],
                             x["W2"], o, None, saved, ws_f, stream=st)
        s2 = tnt.tnt_mem_bwd(cfg, x["q"], x["k"], x["v"], x["lr"], x["mom"], x["decay"], x["W1"],
                             x["W2"], x["dO"], saved, g["dq"], g["dk"], g["dv"], g["dlr"], g["dmom"],
                             g["ddecay"], g["dW1"], g["dW2"], ws_b, stream=st)
        assert s1 == 0 and s2 == 0

    with torch.cuda.stream(st):
        step()
    torch.cuda.synchronize()
    outs = lambda: dict(g, o=o)
    ref = {k: v.clone() for k, v in outs().items()}
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=st):
        step()
    torch.cuda.synchronize()
    for rep in range(3):
        for v in outs().values():
            v.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        bad = [k for k, v in outs().items() if not torch.equal(v, ref[k])]
        assert not bad, f"replay {rep}: {bad} differ from the eager step"
        with torch.cuda.stream(st):
            step()  # eager work between the replays
        torch.cuda.synchronize()
        bad = [k for k, v in outs().items() if not torch.equal(v, ref[k])]
        assert not bad, f"eager step after replay {rep}: {bad} differ"
