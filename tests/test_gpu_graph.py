"""A whole sequence (reset, every slice forward and backward, the deferred dW
GEMMs) captured as a HIP graph on the stage's stream and replayed: every replay
must reproduce the eager outputs and gradients bit for bit.  Replays are
separated by eager work on the same stream and by synchronisations."""
import pytest
import torch

from stage_harness import make_inputs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("wgrad", ["deferred", "per_slice"])
def test_graph_replay_matches_eager(wgrad):
    from paper_2102_07988_amd import terapipe as tp
    H, heads, L = 256, 2, 256
    fwd, bwd = [64, 128, 64], [96, 160]
    print(f"case graph replay: H={H} L={L} {wgrad} fwd={fwd} bwd={bwd}", flush=True)
    params, x, dy = make_inputs(2, H, L, "bf16", (41, 42, 43))
    cs = torch.cuda.Stream()
    with torch.cuda.stream(cs):
        dparams = [{k: v.cuda() for k, v in p.items()} for p in params]
        xd, dyd = x.cuda(), dy.cuda()
        st = tp.Stage(dparams, H, heads, L, dtype="bf16", wgrad=wgrad)
        y = torch.empty_like(xd)
        dx = torch.empty_like(dyd)
        fb, bb = [0], [0]
        for n in fwd:
            fb.append(fb[-1] + n)
        for n in bwd:
            bb.append(bb[-1] + n)

        def seq():
            st.reset()
            for i in range(len(fwd)):
                st.forward(fb[i], fb[i + 1], xd[fb[i]:fb[i + 1]], out=y[fb[i]:fb[i + 1]])
            for i in range(len(bwd) - 1, -1, -1):
                st.backward(bb[i], bb[i + 1], dyd[bb[i]:bb[i + 1]], out=dx[bb[i]:bb[i + 1]])

        st.zero_grads()
        seq()
        torch.cuda.synchronize()
        y_e, dx_e = y.clone(), dx.clone()
        g_e = [{k: v.clone() for k, v in g.items()} for g in st.grads]

        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=cs):
            seq()
        scratch = torch.ones(1 << 20, device="cuda")
        for rep in range(3):
            y.zero_()
            dx.zero_()
            st.zero_grads()
            scratch.mul_(1.5)  # eager work on the same stream between replays
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            assert torch.equal(y, y_e), rep
            assert torch.equal(dx, dx_e), rep
            for g, ge in zip(st.grads, g_e):
                for k in g:
                    assert torch.equal(g[k], ge[k]), (rep, k)
        del graph, st
