"""The fused step captured into a HIP graph (what a serving loop or the bench's
--graph mode does to remove host launch gaps) gives, on every replay, exactly
the codes, scales and y of the same launches made eagerly. Between replays the
state is reset by an eager copy and the stream is synchronized."""
import pytest
import torch

from paper_2609_39185_amd import workloads as wl

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


@pytest.mark.parametrize("fmt,rule,group", [("bf16", "weyl", 0), ("e4m3", "sr", 0),
                                            ("int8", "weyl", 128), ("int4", "philox", 128)])
def test_graph_replays_match_eager(fmt, rule, group):
    import paper_2609_39185_amd as m
    b, H, P, N, G, steps = 4, 8, 64, 128, 2, 3
    A, D = (v.to(DEV) for v in wl.layer_params("mamba2", H, N, 90))
    inputs = [tuple(v.to(DEV) for v in wl.step_inputs(b, H, P, N, G, 91 + k)) for k in range(steps)]
    codes0, scale0 = wl.initial_state(fmt, b, H, P, N, 95, group=group, device=DEV)
    ys = [torch.empty((b, H, P), device=DEV) for _ in range(steps)]

    def run(st, sc, stream=None):
        for k, (x, dt, B, C) in enumerate(inputs):
            m.state_update(st, sc, x, dt, A, B, C, D, ys[k], rule=rule, fmt=fmt, dither_block=128,
                           scale_group=group, step=40 + k, layer=2, stream=stream)

    st_e = codes0.clone()
    sc_e = None if scale0 is None else scale0.clone()
    run(st_e, sc_e)
    torch.cuda.synchronize()
    y_e = [y.clone() for y in ys]

    st_g = codes0.clone()
    sc_g = None if scale0 is None else scale0.clone()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run(st_g, sc_g, stream=torch.cuda.current_stream(DEV))
    torch.cuda.synchronize()
    for rep in range(3):
        st_g.copy_(codes0)
        if sc_g is not None:
            sc_g.copy_(scale0)
        for y in ys:
            y.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(st_g, st_e), (fmt, rule, rep)
        if sc_g is not None:
            assert torch.equal(sc_g, sc_e), (fmt, rule, rep)
        assert all(torch.equal(a, c) for a, c in zip(ys, y_e)), (fmt, rule, rep)
