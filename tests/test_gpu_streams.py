"""Calls on different streams and host threads: two layers updated concurrently
(two default-priority streams, two Python threads) give the codes, scales and y of
the same updates run one after the other."""
import threading

import pytest
import torch

from paper_2609_39185_amd import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def ssmq():
    import paper_2609_39185_amd as m
    m.library()
    return m


@pytest.mark.parametrize("fmt,rule", [("bf16", "weyl"), ("e4m3", "sr"), ("int8", "weyl")])
def test_two_streams_two_threads_match_sequential(ssmq, fmt, rule):
    b, H, P, N, G = 8, 16, 64, 128, 2
    group = 128 if fmt == "int8" else 0
    layers = []
    for ell in range(2):
        A, D = wl.layer_params("mamba2", H, N, 40 + ell, device=DEV)
        x, dt, B, C = wl.step_inputs(b, H, P, N, G, 50 + ell, device=DEV)
        codes, scale = wl.initial_state(fmt, b, H, P, N, 60 + ell, group=group, device=DEV)
        layers.append(dict(A=A, D=D, x=x, dt=dt, B=B, C=C, codes=codes, scale=scale))

    def run(L, ell, codes, scale, y, stream=None):
        ssmq.state_update(codes, scale, L["x"], L["dt"], L["A"], L["B"], L["C"], L["D"], y,
                          rule=rule, fmt=fmt, scale_group=group, dither_block=128, step=9,
                          layer=ell, stream=stream)

    # sequential reference on copies
    ref = []
    for ell, L in enumerate(layers):
        c, s = L["codes"].clone(), None if L["scale"] is None else L["scale"].clone()
        y = torch.empty((b, H, P), device=DEV)
        run(L, ell, c, s, y)
        ref.append((c, s, y))
    torch.cuda.synchronize()

    # concurrent: each layer on its own stream, launched from its own host thread
    streams = [torch.cuda.Stream(device=DEV), torch.cuda.Stream(device=DEV)]
    outs = [None, None]

    def worker(ell):
        L = layers[ell]
        c, s = L["codes"].clone(), None if L["scale"] is None else L["scale"].clone()
        y = torch.empty((b, H, P), device=DEV)
        torch.cuda.synchronize()
        with torch.cuda.stream(streams[ell]):
            run(L, ell, c, s, y, stream=streams[ell])
        streams[ell].synchronize()
        outs[ell] = (c, s, y)

    threads = [threading.Thread(target=worker, args=(ell,)) for ell in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    for (c, s, y), (rc, rs, ry) in zip(outs, ref):
        assert torch.equal(c, rc)
        assert (s is None and rs is None) or torch.equal(s, rs)
        assert torch.equal(y, ry)
