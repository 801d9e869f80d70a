"""A whole step captured in a HIP graph (torch.cuda.CUDAGraph around lce_forward_backward, which
allocates nothing and never synchronizes) and replayed: every replay, with eager work and
synchronizations between replays, gives bitwise the eager call's results, and a replay after the
inputs were overwritten in place gives the eager results of the new inputs."""
import pytest
import torch

import workloads

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lce():
    import paper_2603_16428_amd as m
    m.load_library()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return m


@pytest.mark.parametrize("N,H,V,dtype,chunk", [
    (2048, 1024, 32768, "bf16", 512),   # four chunks, split dH, dW carried in bf16
    (700, 136, 4099, "fp16", 128),     # fp16: the dlogits pass, ragged tails
    (300, 132, 2049, "fp32", 64),      # fp32: five chunks, split dH
])
def test_graph_replay_matches_eager(lce, N, H, V, dtype, chunk):
    d = workloads.random_case(N, H, V, dtype=dtype, seed=N + V, w_std=0.3)
    X, W, y = d["hidden"].cuda(), d["weight"].cuda(), d["labels"].cuda()
    print(f"case N={N} H={H} V={V} {dtype} chunk={chunk} plan {lce.plan_info(N, H, V, X.dtype, True, chunk)}",
          flush=True)
    ws = torch.empty(lce.workspace_size(N, H, V, X.dtype, True, chunk), dtype=torch.uint8, device="cuda")
    out = (torch.empty(1, dtype=torch.float32, device="cuda"), torch.empty_like(X), torch.empty_like(W))

    def eager():
        r = lce.forward_backward(X, W, y, d["ignore_index"], d["reduction"], chunk)
        torch.cuda.synchronize()
        return tuple(t.clone() for t in (r[0].reshape(1), r[1], r[2]))

    ref = eager()
    # Warm up on a side stream (as graph capture requires), then capture.
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        lce.forward_backward(X, W, y, d["ignore_index"], d["reduction"], chunk, ws, out)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        lce.forward_backward(X, W, y, d["ignore_index"], d["reduction"], chunk, ws, out)
    torch.cuda.synchronize()
    for k in range(4):
        for t in out:
            t.fill_(float("nan"))     # eager work between replays
        ws.fill_(255)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out[0], ref[0]) and torch.equal(out[1], ref[1]) and torch.equal(out[2], ref[2]), k
    # New inputs in place: the replay computes with them.
    X.mul_(0.5)
    ref2 = eager()
    assert not torch.equal(ref2[1], ref[1])
    g.replay()
    torch.cuda.synchronize()
    assert torch.equal(out[0], ref2[0]) and torch.equal(out[1], ref2[1]) and torch.equal(out[2], ref2[2])
